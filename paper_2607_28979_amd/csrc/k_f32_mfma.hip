// fp32 translation path on the fp32 matrix cores (v_mfma_f32_16x16x4_f32,
// MI355X's 157.3 TFLOP/s fp32 figure): two launches per call.
//
//   layer 1 (+ router): logits = Wr z + br, g = softmax, Top-K renormalised
//     (paper Sec. 3, Definition "Mixture-of-Translators"), and
//     Hs[u][t][m*hidden+k] = g_m * GELU(W1_m z_t + b1_m)[k]  (erf GELU, App. C.2)
//   layer 2: dst[j][t][o] = sum_{m,k} Hs[u][t][m*hidden+k] W2_m[o][k] + sum_m g_m b2_m[o]
// which equals sum_m g_m (W2_m GELU(W1_m z + b1_m) + b2_m), Eq. mot_definition.
//
// Workgroup = 4 waves, 64 (hidden or output) rows x 64 tokens; wave w owns
// 16 rows x 4 blocks of 16 tokens.  Every workgroup of a unit also computes
// the unit's router logits for its 64 tokens as a 16-row MFMA block (Wr rows,
// zero-padded to 16): wave w takes the k blocks kb = w (mod 4), and the four
// partial sums are added in wave order through LDS.  The logits come out of
// the same instruction sequence in every workgroup, so the gates are
// bit-identical across the unit's workgroups; the one with hidden tile 0
// writes them (dense rows, zeros outside the Top-K set) for layer 2 and adds
// the selections to the usage counts.
//
// Operands come straight from global memory into registers, 16 bytes per
// lane: for a 16-wide k block, lane l holds k = 4*(l/16) .. +3 of its row, and
// k-step s of the block uses k = 4*(l/16) + s (a permutation of the block's
// k values shared by A and B).  Blocks are prefetched kRing deep.
#include "mot_device.h"
#include "mot_internal.h"
#include "../../include/mot.h"

namespace mot {

namespace {

constexpr int kRing = 4;   // k blocks in flight per wave

__device__ __forceinline__ f32x4 mfma_f32_16x16x4(float a, float b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ size_t src_off(const Problem& p, int i, int tok, int c) {
    const size_t layer = (size_t)i * p.n_tok * p.d_in;
    if (p.src_layout == MOT_LAYOUT_BTHD) return layer + (size_t)tok * p.d_in + c;
    const int b = tok / p.T, t = tok % p.T, hh = c / p.D_src, dd = c % p.D_src;
    return layer + (((size_t)b * p.H_src + hh) * p.T + t) * p.D_src + dd;
}

__device__ __forceinline__ f32x4 ld4(const float* ptr) { return *reinterpret_cast<const f32x4*>(ptr); }

// grid: x = (hidden tiles of 64) x (token tiles of 64), hidden fastest; z = unit
__global__ __launch_bounds__(256) void k_f32_mfma_gemm1(Problem p, UnitTab ut) {
    __shared__ float s_gate[64][MOT_MAX_EXPERTS];
    __shared__ f32x4 s_part[4][64][4];   // [wave][token][expert quad] partial logits
    const uint32_t code = ut.code[blockIdx.z];
    const int j = unit_j(code), x = unit_x(code), i = unit_i(code), gs = unit_gslot(code);
    const int E = p.E, EH = E * p.hidden, nA = EH / 64;
    const int at = blockIdx.x % nA, bt = blockIdx.x / nA;
    const int hid0 = at * 64, tok0 = bt * 64;
    const size_t unit = (size_t)j * p.streams + x;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, l16 = lane & 15, q = lane >> 4;
    const float* W1 = reinterpret_cast<const float*>(p.w1) + unit * EH * p.d_in;
    const float* Wr = reinterpret_cast<const float*>(p.wr) + unit * E * p.d_in;
    const float* src = reinterpret_cast<const float*>(p.src[x]);

    // operand rows of this lane: hidden row, router row (< E, else zeros), and
    // the four token rows (clamped into range; those columns are not stored)
    const float* arow = W1 + (size_t)(hid0 + w * 16 + l16) * p.d_in;
    const bool rvalid = l16 < E;
    const float* rrow = Wr + (size_t)(rvalid ? l16 : 0) * p.d_in;
    int tokc[4];
#pragma unroll
    for (int tg = 0; tg < 4; ++tg) tokc[tg] = min(tok0 + tg * 16 + l16, p.n_tok - 1);
    const bool bthd = p.src_layout == MOT_LAYOUT_BTHD;
    const float* brow[4];
#pragma unroll
    for (int tg = 0; tg < 4; ++tg) brow[tg] = src + src_off(p, i, tokc[tg], 0);

    const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
    f32x4 acc[4], racc[4];
#pragma unroll
    for (int tg = 0; tg < 4; ++tg) acc[tg] = racc[tg] = zero;
    const int nb = p.d_in / 16;
    // ring slot s holds k block kb0 + s, and kb = s (mod 4): the router rows
    // are fetched and used only in slot w
    f32x4 ra[kRing], rr[kRing], rb[kRing][4];
    auto fetch = [&](int kb, int slot) {
        const int k = kb * 16 + 4 * q;
        ra[slot] = ld4(arow + k);
        rr[slot] = slot == w && rvalid ? ld4(rrow + k) : zero;
#pragma unroll
        for (int tg = 0; tg < 4; ++tg)
            rb[slot][tg] = bthd ? ld4(brow[tg] + k) : ld4(src + src_off(p, i, tokc[tg], k));
    };
#pragma unroll
    for (int s = 0; s < kRing; ++s)
        if (s < nb) fetch(s, s);
    for (int kb0 = 0; kb0 < nb; kb0 += kRing) {
#pragma unroll
        for (int s = 0; s < kRing; ++s) {
            const int kb = kb0 + s;
            if (kb < nb) {
#pragma unroll
                for (int st = 0; st < 4; ++st) {
#pragma unroll
                    for (int tg = 0; tg < 4; ++tg) acc[tg] = mfma_f32_16x16x4(ra[s][st], rb[s][tg][st], acc[tg]);
                    if (s == w) {
#pragma unroll
                        for (int tg = 0; tg < 4; ++tg) racc[tg] = mfma_f32_16x16x4(rr[s][st], rb[s][tg][st], racc[tg]);
                    }
                }
                if (kb + kRing < nb) fetch(kb + kRing, s);
            }
        }
    }

    // router: racc[tg] holds this wave's partial logits of experts 4q .. 4q+3
    // for token tg*16 + l16; the sum over the waves (in wave order) for token
    // w*16 + l16, all E per lane, softmax + Top-K, gates to LDS (and to
    // global from hidden tile 0, with the usage counts)
#pragma unroll
    for (int tg = 0; tg < 4; ++tg) s_part[w][tg * 16 + l16][q] = racc[tg];
    __syncthreads();
    {
        const int tl = w * 16 + l16;
        f32x4 lg = s_part[0][tl][q];
#pragma unroll
        for (int ww = 1; ww < 4; ++ww) {
            const f32x4 v = s_part[ww][tl][q];
#pragma unroll
            for (int r = 0; r < 4; ++r) lg[r] += v[r];
        }
        float g[MOT_MAX_EXPERTS];
#pragma unroll
        for (int qq = 0; qq < 4; ++qq)
#pragma unroll
            for (int r = 0; r < 4; ++r) g[4 * qq + r] = __shfl(lg[r], 16 * qq + l16, 64);
        const float* br = p.br ? reinterpret_cast<const float*>(p.br) + unit * E : nullptr;
        float mx = -INFINITY;
#pragma unroll
        for (int m = 0; m < MOT_MAX_EXPERTS; ++m)
            if (m < E) {
                g[m] += br ? br[m] : 0.f;
                mx = fmaxf(mx, g[m]);
            }
        float den = 0.f;
#pragma unroll
        for (int m = 0; m < MOT_MAX_EXPERTS; ++m) {
            g[m] = m < E ? expf(g[m] - mx) : 0.f;
            den += g[m];
        }
        const float inv = 1.0f / den;
#pragma unroll
        for (int m = 0; m < MOT_MAX_EXPERTS; ++m) g[m] *= inv;
        const uint32_t taken = topk_renormalise(g, E, p.top_k);
        const int tok = tok0 + tl;
        if (q == 0) {
#pragma unroll
            for (int m = 0; m < MOT_MAX_EXPERTS; ++m)
                if (m < E) s_gate[tl][m] = g[m];
        }
        if (at == 0) {
            if (q == 0 && tok < p.n_tok) {
                float* G = p.gates + ((size_t)gs * p.n_tok_pad + tok) * E;
                for (int m = 0; m < E; ++m) G[m] = g[m];
            }
            if (p.usage)
                count_usage(p.usage + unit * E, E, taken, q == 0 && tok < p.n_tok);
        }
    }
    __syncthreads();

    // epilogue: + b1, GELU, * gate; lane holds hidden rows 4q .. 4q+3 of the
    // wave's 16 for token tg*16 + l16
    const int m = hid0 / p.hidden;   // hidden % 64 == 0: one expert per tile
    const int h = hid0 + w * 16 + 4 * q;
    f32x4 bias = zero;
    if (p.b1) bias = ld4(reinterpret_cast<const float*>(p.b1) + unit * EH + h);
    float* H = reinterpret_cast<float*>(p.hbuf) + (size_t)blockIdx.z * p.n_tok_pad * EH;
#pragma unroll
    for (int tg = 0; tg < 4; ++tg) {
        const int tl = tg * 16 + l16, tok = tok0 + tl;
        if (tok >= p.n_tok) continue;
        const float gate = s_gate[tl][m];
        f32x4 v;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const float a = acc[tg][r] + bias[r];
            v[r] = gate * (p.act == MOT_ACT_GELU ? gelu_erf(a) : a);
        }
        *reinterpret_cast<f32x4*>(H + (size_t)tok * EH + h) = v;
    }
}

// grid: x = (output tiles of 64) x (token tiles of 64), outputs fastest; z = unit
__global__ __launch_bounds__(256) void k_f32_mfma_gemm2(Problem p, UnitTab ut) {
    const uint32_t code = ut.code[blockIdx.z];
    const int j = unit_j(code), x = unit_x(code), gs = unit_gslot(code);
    const int E = p.E, EH = E * p.hidden, nA = (p.d_out + 63) / 64;
    const int at = blockIdx.x % nA, bt = blockIdx.x / nA;
    const int out0 = at * 64, tok0 = bt * 64;
    const size_t unit = (size_t)j * p.streams + x;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, l16 = lane & 15, q = lane >> 4;
    const float* W2 = reinterpret_cast<const float*>(p.w2) + unit * E * p.d_out * p.hidden;
    const float* H = reinterpret_cast<const float*>(p.hbuf) + (size_t)blockIdx.z * p.n_tok_pad * EH;
    const float* G = p.gates + (size_t)gs * p.n_tok_pad * E;
    const int orow = min(out0 + w * 16 + l16, p.d_out - 1);
    int tokc[4];
#pragma unroll
    for (int tg = 0; tg < 4; ++tg) tokc[tg] = min(tok0 + tg * 16 + l16, p.n_tok - 1);
    const f32x4 zero = {0.f, 0.f, 0.f, 0.f};

    // accumulators start at sum_m b2_m[o] g_m[t]: k = m in blocks of four
    f32x4 acc[4];
#pragma unroll
    for (int tg = 0; tg < 4; ++tg) acc[tg] = zero;
    if (p.b2) {
        const float* b2 = reinterpret_cast<const float*>(p.b2) + unit * E * p.d_out;
        for (int m0 = 0; m0 < E; m0 += 4) {
            const int m = m0 + q;
            const float a = m < E ? b2[(size_t)m * p.d_out + orow] : 0.f;
#pragma unroll
            for (int tg = 0; tg < 4; ++tg) {
                const float b = m < E ? G[(size_t)tokc[tg] * E + m] : 0.f;
                acc[tg] = mfma_f32_16x16x4(a, b, acc[tg]);
            }
        }
    }

    const int nb = EH / 16;
    f32x4 ra[kRing], rb[kRing][4];
    auto fetch = [&](int kb, int slot) {
        const int k = kb * 16 + 4 * q, m = k / p.hidden, kk = k - m * p.hidden;
        ra[slot] = ld4(W2 + ((size_t)m * p.d_out + orow) * p.hidden + kk);
#pragma unroll
        for (int tg = 0; tg < 4; ++tg) rb[slot][tg] = ld4(H + (size_t)tokc[tg] * EH + k);
    };
#pragma unroll
    for (int s = 0; s < kRing; ++s)
        if (s < nb) fetch(s, s);
    for (int kb0 = 0; kb0 < nb; kb0 += kRing) {
#pragma unroll
        for (int s = 0; s < kRing; ++s) {
            const int kb = kb0 + s;
            if (kb < nb) {
#pragma unroll
                for (int st = 0; st < 4; ++st)
#pragma unroll
                    for (int tg = 0; tg < 4; ++tg) acc[tg] = mfma_f32_16x16x4(ra[s][st], rb[s][tg][st], acc[tg]);
                if (kb + kRing < nb) fetch(kb + kRing, s);
            }
        }
    }

    // lane holds outputs o .. o+3 (o = out0 + w*16 + 4q) of token tg*16 + l16
    const int o = out0 + w * 16 + 4 * q;
    if (o >= p.d_out) return;   // d_out % 4 == 0
    float* dst = reinterpret_cast<float*>(p.dst[x]) + (size_t)j * p.n_tok * p.d_out;
#pragma unroll
    for (int tg = 0; tg < 4; ++tg) {
        const int tok = tok0 + tg * 16 + l16;
        if (tok >= p.n_tok) continue;
        size_t off;
        if (p.dst_layout == MOT_LAYOUT_BTHD) {
            off = (size_t)tok * p.d_out + o;
        } else {   // D_tgt % 4 == 0: o .. o+3 in one head
            const int b = tok / p.T, t = tok % p.T, hh = o / p.D_tgt, dd = o % p.D_tgt;
            off = (((size_t)b * p.H_tgt + hh) * p.T + t) * p.D_tgt + dd;
        }
        *reinterpret_cast<f32x4*>(dst + off) = acc[tg];
    }
}

}  // namespace

bool f32_mfma_fits(const Problem& p) {
    return p.hidden % 64 == 0 && p.d_in % 16 == 0 && p.d_out % 4 == 0 && p.E <= MOT_MAX_EXPERTS;
}

hipError_t launch_f32_mfma_gemm1(const Problem& p, const UnitTab& ut, hipStream_t stream) {
    if (ut.n == 0 || p.n_tok == 0) return hipSuccess;
    const int EH = p.E * p.hidden;
    dim3 grid((EH / 64) * ((p.n_tok + 63) / 64), 1, ut.n);
    hipLaunchKernelGGL(k_f32_mfma_gemm1, grid, dim3(256), 0, stream, p, ut);
    return hipGetLastError();
}

hipError_t launch_f32_mfma_gemm2(const Problem& p, const UnitTab& ut, hipStream_t stream) {
    if (ut.n == 0 || p.n_tok == 0) return hipSuccess;
    dim3 grid(((p.d_out + 63) / 64) * ((p.n_tok + 63) / 64), 1, ut.n);
    hipLaunchKernelGGL(k_f32_mfma_gemm2, grid, dim3(256), 0, stream, p, ut);
    return hipGetLastError();
}

}  // namespace mot
