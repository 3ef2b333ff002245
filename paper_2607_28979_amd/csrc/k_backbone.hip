// Backbone translator body (paper App. C.2, "Backbone Translator") as the
// experts of the mixture, one channel-window slot per unit.  The host runs,
// per unit and expert, a chain of two generic kernels and the causal
// attention kernel of the replay step:
//   * k_ln_rows: LayerNorm of bf16 rows (fp32 statistics, population
//     variance, eps 1e-5), bf16 out; optionally a second affine pair on the
//     same statistics into a second output (one read for two LayerNorms of
//     one input).  Rows of up to 256 take half a wave each, wider rows a
//     whole wave;
//   * k_linear: out[t][o] = act(sum_k in[t][k] W[o][k] + b[o]) (+ res[t][o]) on
//     v_mfma_f32_32x32x16_bf16, 128 outputs x 128 rows per 256-thread
//     workgroup, K in 64-wide double-buffered XOR-swizzled LDS slices.  The
//     epilogue stages act(acc + b) in fp32 through LDS so that every global
//     access after it (residual, output, fp32 mixture) is a row-contiguous
//     16-byte access; it either stores bf16 rows or adds gate[t][m] * value
//     into the fp32 mixture (the last expert rounds the mixture to bf16 into
//     the target cache).
#include "mot_device.h"
#include "mot_internal.h"
#include "../../include/mot.h"

namespace mot {

namespace {

constexpr int LM = 128, LN_ = 128, LK = 64;
constexpr int kLChunks = LM * LK / 8;   // 16-byte chunks per operand tile

__device__ __forceinline__ int lswz(int row, int c) { return row * 8 + (c ^ (row & 7)); }

// LPR lanes per row (64: w <= 4096, 32: w <= 256); grid: ceil(n / rows per
// workgroup) workgroups of 4 waves.  w % 8 == 0.
template <int LPR>
__global__ __launch_bounds__(256) void k_ln_rows(LnProblem p) {
    constexpr int MAXC = LPR == 64 ? 8 : 1;   // 16-byte chunks per lane
    constexpr int RPW = 64 / LPR;             // rows per wave
    const int lane = threadIdx.x & 63, hl = lane % LPR;
    const int row = (blockIdx.x * 4 + (threadIdx.x >> 6)) * RPW + lane / LPR;
    const bool live = row < p.n;
    const int w = p.w;
    const size_t gy = blockIdx.y;
    const size_t pg = gy * p.p_gs;
    const uint16_t *pg_g = p.g + pg, *pg_b = p.b + pg;
    const uint16_t *pg_g2 = p.out2 ? p.g2 + pg : nullptr, *pg_b2 = p.out2 ? p.b2 + pg : nullptr;
    uint16_t* out = p.out + gy * p.out_gs;
    uint16_t* out2 = p.out2 ? p.out2 + gy * p.out_gs : nullptr;
    const uint16_t* r = p.in + gy * p.in_gs + (size_t)(live ? row : 0) * p.ld_in;
    const u32x4 zero = {0u, 0u, 0u, 0u};
    u32x4 q[MAXC];
#pragma unroll
    for (int c = 0; c < MAXC; ++c) {
        const int e = (hl + LPR * c) * 8;
        q[c] = live && e < w ? *reinterpret_cast<const u32x4*>(r + e) : zero;
    }
    // the affine parameters of the single-chunk form load before the reductions
    u32x4 gq[MAXC], bq[MAXC], gq2[MAXC], bq2[MAXC];
    if (MAXC == 1) {
        const int e = hl * 8;
        gq[0] = e < w ? *reinterpret_cast<const u32x4*>(pg_g + e) : zero;
        bq[0] = e < w ? *reinterpret_cast<const u32x4*>(pg_b + e) : zero;
        if (out2) {
            gq2[0] = e < w ? *reinterpret_cast<const u32x4*>(pg_g2 + e) : zero;
            bq2[0] = e < w ? *reinterpret_cast<const u32x4*>(pg_b2 + e) : zero;
        }
    }
    float v[MAXC][8];
    float sum = 0.f;
#pragma unroll
    for (int c = 0; c < MAXC; ++c)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            v[c][2 * i] = bf16_lo(q[c][i]);
            v[c][2 * i + 1] = bf16_hi(q[c][i]);
            sum += v[c][2 * i] + v[c][2 * i + 1];
        }
#pragma unroll
    for (int off = LPR / 2; off >= 1; off >>= 1) sum += __shfl_xor(sum, off, 64);
    const float mean = sum / (float)w;
    float sq = 0.f;
#pragma unroll
    for (int c = 0; c < MAXC; ++c) {
        if ((hl + LPR * c) * 8 < w) {
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const float d = v[c][i] - mean;
                sq += d * d;
            }
        }
    }
#pragma unroll
    for (int off = LPR / 2; off >= 1; off >>= 1) sq += __shfl_xor(sq, off, 64);
    const float inv = rsqrtf(sq / (float)w + 1e-5f);
    if (!live) return;
#pragma unroll
    for (int c = 0; c < MAXC; ++c) {
        const int e = (hl + LPR * c) * 8;
        if (e < w) {
            if (MAXC > 1) {
                gq[c] = *reinterpret_cast<const u32x4*>(pg_g + e);
                bq[c] = *reinterpret_cast<const u32x4*>(pg_b + e);
            }
            u32x4 o;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float y0 = (v[c][2 * i] - mean) * inv * bf16_lo(gq[c][i]) + bf16_lo(bq[c][i]);
                const float y1 = (v[c][2 * i + 1] - mean) * inv * bf16_hi(gq[c][i]) + bf16_hi(bq[c][i]);
                o[i] = pack_bf16x2(y0, y1);
            }
            *reinterpret_cast<u32x4*>(out + (size_t)row * w + e) = o;
            if (out2) {
                if (MAXC > 1) {
                    gq2[c] = *reinterpret_cast<const u32x4*>(pg_g2 + e);
                    bq2[c] = *reinterpret_cast<const u32x4*>(pg_b2 + e);
                }
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float y0 = (v[c][2 * i] - mean) * inv * bf16_lo(gq2[c][i]) + bf16_lo(bq2[c][i]);
                    const float y1 = (v[c][2 * i + 1] - mean) * inv * bf16_hi(gq2[c][i]) + bf16_hi(bq2[c][i]);
                    o[i] = pack_bf16x2(y0, y1);
                }
                *reinterpret_cast<u32x4*>(out2 + (size_t)row * w + e) = o;
            }
        }
    }
}

// grid: x = row tiles of 128, y = output tiles of 128 of the parts in turn;
// 256 threads
__global__ __launch_bounds__(256) void k_linear(LinearProblem p) {
    __shared__ u32x4 lds[2][2][kLChunks];   // [stage][0 = W rows, 1 = input rows]
    __shared__ u32x4 lnp[2][kLinearLnMaxK / 8];   // fused LayerNorm gamma, beta
    // the part of this output tile, selected field by field (no dynamic
    // indexing into the argument block)
    int y = blockIdx.y, pi = 0;
    const int t0 = (p.part[0].N + LM - 1) / LM, t1 = (p.part[1].N + LM - 1) / LM;
    if (p.nparts > 1 && y >= t0) {
        y -= t0;
        pi = 1;
        if (p.nparts > 2 && y >= t1) {
            y -= t1;
            pi = 2;
        }
    }
#define MOT_PART(f) (pi == 0 ? p.part[0].f : pi == 1 ? p.part[1].f : p.part[2].f)
    const uint16_t* W = MOT_PART(W);
    const uint16_t* bias = MOT_PART(bias);
    const uint16_t* lng = MOT_PART(ln_g);
    const uint16_t* lnb = MOT_PART(ln_b);
    uint16_t* out = MOT_PART(out);
    const int N = MOT_PART(N);
#undef MOT_PART
    // group of a grouped launch
    const int gz = blockIdx.z;
    {
        const size_t wg = (size_t)gz * p.w_gs;
        W += wg;
        bias += wg;
        if (lng) {
            lng += wg;
            lnb += wg;
        }
        out = p.out_tab[0] ? p.out_tab[gz] : out + (size_t)gz * p.out_gs;
    }
    const uint16_t* res = p.res ? p.res + (size_t)gz * p.res_gs : nullptr;
    float* mix_acc = p.mix ? p.mix_acc + (size_t)gz * p.mix_gs : nullptr;
    const float* gates = p.mix ? p.gates + (size_t)gz * p.gate_gs : nullptr;
    const int r0 = blockIdx.x * LN_, o0 = y * LM;
    const int K = p.K;
    const uint16_t* A = p.in_tab[0] ? p.in_tab[gz / p.tab_div] : p.in + (size_t)gz * p.in_gs;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1, g = lane >> 5, l32 = lane & 31;
    const u32x4 zero = {0u, 0u, 0u, 0u};
    // register ring of KD slices: the loads of up to KD slices are in flight
    // at once, so a K of up to 64 * KD costs one memory latency
    constexpr int KD = 4;
    u32x4 ra[KD][4], rb[KD][4];
    auto gload = [&](int k0, u32x4 (&xa)[4], u32x4 (&xb)[4]) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            // rows past the ends read the last row: they only feed outputs that
            // are never stored, and unconditional loads keep the wait counts exact
            const int row = (tid >> 3) + 32 * r, c = tid & 7;
            const int o = min(o0 + row, N - 1), t = min(r0 + row, p.n - 1);
            xa[r] = *reinterpret_cast<const u32x4*>(W + (size_t)o * K + k0 + c * 8);
            xb[r] = *reinterpret_cast<const u32x4*>(A + (size_t)t * p.ld_in + k0 + c * 8);
        }
    };
    auto sstore = [&](int st, const u32x4 (&xa)[4], const u32x4 (&xb)[4]) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int row = (tid >> 3) + 32 * r, c = tid & 7;
            lds[st][0][lswz(row, c)] = xa[r];
            lds[st][1][lswz(row, c)] = xb[r];
        }
    };
    f32x16 acc[2][2];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int bb = 0; bb < 2; ++bb)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[a][bb][e] = 0.f;
    const int nk = K / LK;
    // LayerNorm parameters: issued before the operand ring so that their wait
    // leaves the ring's loads in flight
    u32x4 lnv = zero;
    const bool lnl = lng && tid < 2 * (kLinearLnMaxK / 8) && (tid & 31) * 8 < K;
    if (lnl) lnv = *reinterpret_cast<const u32x4*>((tid < 32 ? lng : lnb) + (tid & 31) * 8);
#pragma unroll
    for (int d = 0; d < KD; ++d)
        if (d < nk) gload(d * LK, ra[d], rb[d]);
    if (lnl) lnp[tid >> 5][tid & 31] = lnv;
    // fused LayerNorm of the input rows (K <= 64 * KD: every row is in the
    // ring).  Thread holds columns 64 d + 8 (tid & 7) .. +7 of rows
    // (tid >> 3) + 32 r; the 8 lanes tid & 7 of a row reduce by shuffles.
    float mean[4], inv[4];
    if (lng) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            float s = 0.f;
#pragma unroll
            for (int d = 0; d < KD; ++d)
                if (d < nk)
#pragma unroll
                    for (int i = 0; i < 4; ++i) s += bf16_lo(rb[d][r][i]) + bf16_hi(rb[d][r][i]);
#pragma unroll
            for (int off = 1; off < 8; off <<= 1) s += __shfl_xor(s, off, 64);
            mean[r] = s / (float)K;
            float q = 0.f;
#pragma unroll
            for (int d = 0; d < KD; ++d)
                if (d < nk)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const float d0 = bf16_lo(rb[d][r][i]) - mean[r], d1 = bf16_hi(rb[d][r][i]) - mean[r];
                        q += d0 * d0 + d1 * d1;
                    }
#pragma unroll
            for (int off = 1; off < 8; off <<= 1) q += __shfl_xor(q, off, 64);
            inv[r] = rsqrtf(q / (float)K + 1e-5f);
        }
        __syncthreads();   // gamma and beta in LDS
    }
    // one barrier per slice: a wave past the barrier of slice kt - 1 knows every
    // wave has finished computing slice kt - 2, whose LDS stage slice kt reuses
    for (int kt0 = 0; kt0 < nk; kt0 += KD) {
#pragma unroll
        for (int d = 0; d < KD; ++d) {
            const int kt = kt0 + d;
            if (kt >= nk) continue;
            const int st = kt & 1;
            if (lng) {   // nk <= KD here: slice kt is ring entry d
                const u32x4 lg = lnp[0][kt * 8 + (tid & 7)], lb = lnp[1][kt * 8 + (tid & 7)];
#pragma unroll
                for (int r = 0; r < 4; ++r)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const float y0 = (bf16_lo(rb[d][r][i]) - mean[r]) * inv[r] * bf16_lo(lg[i]) + bf16_lo(lb[i]);
                        const float y1 = (bf16_hi(rb[d][r][i]) - mean[r]) * inv[r] * bf16_hi(lg[i]) + bf16_hi(lb[i]);
                        rb[d][r][i] = pack_bf16x2(y0, y1);
                    }
            }
            sstore(st, ra[d], rb[d]);
            if (kt + KD < nk) gload((kt + KD) * LK, ra[d], rb[d]);
            __syncthreads();
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                const int c = 2 * s + g;
                u32x4 a[2], bo[2];
#pragma unroll
                for (int bm = 0; bm < 2; ++bm) a[bm] = lds[st][0][lswz(wm * 64 + bm * 32 + l32, c)];
#pragma unroll
                for (int bn = 0; bn < 2; ++bn) bo[bn] = lds[st][1][lswz(wn * 64 + bn * 32 + l32, c)];
#pragma unroll
                for (int bm = 0; bm < 2; ++bm)
#pragma unroll
                    for (int bn = 0; bn < 2; ++bn) acc[bm][bn] = mfma_32x32x16(a[bm], bo[bn], acc[bm][bn]);
            }
        }
    }
    // the last slice's barrier has been passed; reads of its stage must retire
    // before the staging overwrites it
    __syncthreads();
    // epilogue, stage 1: act(acc + b) in fp32 into LDS, token-major, 32
    // chunks of 4 outputs per row, chunk c of row r at r * 32 + (c ^ (r & 31)).
    f32x4* stg = reinterpret_cast<f32x4*>(&lds[0][0][0]);   // 128 x 128 fp32 = 64 KB
    u32x2 bw[2][4];   // bias of outputs o0 + wm*64 + bm*32 + 8*ii + 4*g .. +3, all loads issued at once
#pragma unroll
    for (int bm = 0; bm < 2; ++bm)
#pragma unroll
        for (int ii = 0; ii < 4; ++ii)
            bw[bm][ii] = *reinterpret_cast<const u32x2*>(bias + min(o0 + wm * 64 + bm * 32 + 8 * ii + 4 * g, N - 4));
#pragma unroll
    for (int bm = 0; bm < 2; ++bm) {
        const int ol = wm * 64 + bm * 32;
#pragma unroll
        for (int bn = 0; bn < 2; ++bn) {
            const int tl = wn * 64 + bn * 32 + l32;   // lane holds outputs ol + 8*ii + 4*g + jj of row tl
#pragma unroll
            for (int ii = 0; ii < 4; ++ii) {
                const int c = (ol >> 2) + 2 * ii + g;
                f32x4 v;
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) {
                    const float bj = (jj & 1) ? bf16_hi(bw[bm][ii][jj >> 1]) : bf16_lo(bw[bm][ii][jj >> 1]);
                    const float x = acc[bm][bn][4 * ii + jj] + bj;
                    v[jj] = p.gelu ? gelu_tanh(x) : x;
                }
                stg[tl * 32 + (c ^ (tl & 31))] = v;
            }
        }
    }
    // the epilogue's own global inputs (residual, fp32 mixture, gates) are
    // fetched for every pass at once, after the accumulators are staged: thread ->
    // 8 consecutive outputs of one row, 16 rows per pass
    constexpr int NP = LN_ / 16;
    const int h = tid & 15, oc = o0 + 8 * h;
    u32x4 rres[NP];
    f32x4 rmix[NP][2];
    float rgate[NP];
    const size_t ld_res = p.ld_res ? p.ld_res : (size_t)N, ld_out = p.ld_out ? p.ld_out : (size_t)N;
#pragma unroll
    for (int pass = 0; pass < NP; ++pass) {
        // clamped to the last row / column group: values of lanes that store
        // nothing are never used
        const int t = min(r0 + pass * 16 + (tid >> 4), p.n - 1);
        const size_t at = (size_t)t * N + min(oc, N - 8);
        rres[pass] = res ? *reinterpret_cast<const u32x4*>(res + (size_t)t * ld_res + min(oc, N - 8)) : zero;
        rgate[pass] = p.mix ? gates[(size_t)t * p.gate_ld + p.expert] : 0.f;
#pragma unroll
        for (int i = 0; i < 2; ++i)
            rmix[pass][i] = p.mix && !p.first ? reinterpret_cast<const f32x4*>(mix_acc + at)[i]
                                              : f32x4{0.f, 0.f, 0.f, 0.f};
    }
    __syncthreads();
    // stage 2: add the residual or mix, round, store row-contiguous 16 bytes
    if (oc >= N) return;
#pragma unroll
    for (int pass = 0; pass < NP; ++pass) {
        const int tl = pass * 16 + (tid >> 4), t = r0 + tl;
        if (t >= p.n) break;
        const f32x4 lo = stg[tl * 32 + ((2 * h) ^ (tl & 31))];
        const f32x4 hi = stg[tl * 32 + ((2 * h + 1) ^ (tl & 31))];
        float v[8] = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        const size_t at = (size_t)t * N + oc;   // the fp32 mixture rows are dense
        if (res) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                v[2 * i] += bf16_lo(rres[pass][i]);
                v[2 * i + 1] += bf16_hi(rres[pass][i]);
            }
        }
        if (p.mix) {
            f32x4 m0 = rmix[pass][0], m1 = rmix[pass][1];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                m0[i] += rgate[pass] * v[i];
                m1[i] += rgate[pass] * v[4 + i];
            }
            if (!p.last) {
                f32x4* accp = reinterpret_cast<f32x4*>(mix_acc + at);
                accp[0] = m0;
                accp[1] = m1;
                continue;
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                v[i] = m0[i];
                v[4 + i] = m1[i];
            }
        }
        const u32x4 w4 = {pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]), pack_bf16x2(v[4], v[5]),
                          pack_bf16x2(v[6], v[7])};
        *reinterpret_cast<u32x4*>(out + (size_t)t * ld_out + oc) = w4;
    }
}

}  // namespace

hipError_t launch_ln_rows(const LnProblem& p, hipStream_t stream) {
    if (p.n == 0) return hipSuccess;
    const unsigned gy = p.groups > 1 ? (unsigned)p.groups : 1u;
    if (p.w <= 256)
        hipLaunchKernelGGL(k_ln_rows<32>, dim3((p.n + 7) / 8, gy), dim3(256), 0, stream, p);
    else
        hipLaunchKernelGGL(k_ln_rows<64>, dim3((p.n + 3) / 4, gy), dim3(256), 0, stream, p);
    return hipGetLastError();
}

hipError_t launch_linear(const LinearProblem& p, hipStream_t stream) {
    if (p.n == 0) return hipSuccess;
    int tiles = 0;
    for (int q = 0; q < p.nparts; ++q) tiles += (p.part[q].N + LM - 1) / LM;
    const unsigned gz = p.groups > 1 ? (unsigned)p.groups : 1u;
    hipLaunchKernelGGL(k_linear, dim3((p.n + LN_ - 1) / LN_, tiles, gz), dim3(256), 0, stream, p);
    return hipGetLastError();
}

}  // namespace mot
