// Fused bf16 translation kernel: router + translator layer 1 + GELU + gate +
// translator layer 2 + gated mix + store, in one pass per token tile.  The
// E*hidden activations of a token never leave the chip.
//
// Per (token tile of 128, unit) workgroup, four waves of 32 tokens each:
//   * the wave's source rows (32 x d_in bf16) are held in VGPRs as MFMA B
//     operands for the whole kernel;
//   * router: logits = Wr z on MFMA (Wr zero-padded to 32 rows), fp32
//     softmax -> gates g[m] (paper Sec. 3, Definition "Mixture-of-Translators");
//   * the gated mix of the second-layer biases, sum_m g_m b2_m, seeds the
//     output accumulators (two small MFMAs per output block);
//   * the hidden dimension E*hidden is walked in 32-wide chunks (each inside
//     one translator m):
//       S^T = W1_m[chunk] z^T + b1   (MFMA 32x32x16, A = W1 rows from LDS)
//       A2  = bf16(g_m * GELU(S))    (VALU; S's accumulator fragment is
//                                     already the A-operand fragment of the
//                                     next product because W1's rows are
//                                     staged in a matching permuted order)
//       Y  += A2 . W2_m[:, chunk]^T  (MFMA, B = W2 columns from LDS)
//     so the expert reduction of the gated sum happens inside Y;
//   * W1/b1 chunks are prefetched one chunk ahead and W2 chunks are consumed
//     one chunk late (software pipeline): in iteration c the wave issues
//     layer-1 MFMAs of chunk c, layer-2 MFMAs of chunk c-1 and the GELU of
//     chunk c, so VALU work overlaps matrix-core work.  Weight chunks move
//     global -> LDS with direct-to-LDS 16-byte loads (no VGPR staging).
//   * Y is rounded to bf16 and stored in the target layout.
#include "mot_device.h"
#include "mot_internal.h"
#include "../../include/mot.h"

namespace mot {

namespace {

typedef __attribute__((address_space(3))) void lds_void;

template <int D_IN, int D_OUT>
struct Cfg {
    static constexpr int BM = 128;                // tokens per workgroup
    static constexpr int KS1 = D_IN / 16;         // layer-1 k-steps
    static constexpr int NB = D_OUT / 32;         // layer-2 output blocks
    static constexpr int CPR1 = D_IN / 8;         // 16-byte chunks per W1 row
    static constexpr int W1_CH = 32 * CPR1;       // chunks per W1 stage
    static constexpr int W2_CH = D_OUT * 4;       // chunks per W2 stage (32 hidden = 4 chunks)
    static constexpr int W1_ROUNDS = W1_CH / 256;
    static constexpr int W2_ROUNDS = W2_CH / 256;
    static constexpr int GS = 4 * MOT_MAX_EXPERTS * 32;   // gate floats (4 waves)
    // LDS map in 16-byte units
    static constexpr int OFF_W1 = 0;
    static constexpr int OFF_W2 = OFF_W1 + 2 * W1_CH;
    static constexpr int OFF_B1 = OFF_W2 + 2 * W2_CH;     // 2 stages x 4 chunks
    static constexpr int OFF_G = OFF_B1 + 8;
    static constexpr int TOTAL = OFF_G + GS / 4;
    static_assert(W1_CH % 256 == 0 && W2_CH % 256 == 0, "tile shape");
};

// Row r of a staged 32-row W1 block holds hidden row perm(r) of the chunk, so
// that the layer-1 accumulator fragment (rows 8*i + 4*g + j of lane-half g)
// lists hidden values 8*g .. 8*g+7 (i < 2) and 16+8*g .. 16+8*g+7 (i >= 2):
// exactly the two 16-wide k-slices the lane supplies as layer-2 A operand.
__device__ __forceinline__ int w1_perm(int r) {
    const int i = r >> 3, g = (r >> 2) & 1, jj = r & 3;
    return ((i >> 1) << 4) | (g << 3) | ((i & 1) << 2) | jj;
}

__device__ __forceinline__ void load_lds16(const void* gsrc, u32x4* lds_dst_wave_base) {
    __builtin_amdgcn_global_load_lds(gsrc, (lds_void*)lds_dst_wave_base, 16, 0, 0);
}

// Per-lane choice between two registers as a bitwise blend, so the compiler
// cannot fold it into a dynamically indexed (scratch) array access.
__device__ __forceinline__ float pick(uint32_t mask, float a, float b) {
    return __uint_as_float((__float_as_uint(a) & ~mask) | (__float_as_uint(b) & mask));
}

__device__ __forceinline__ void wait_vm_all() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

template <int D_IN, int D_OUT>
__global__ __launch_bounds__(256, 1) __attribute__((amdgpu_waves_per_eu(1, 1))) void k_bf16_fused(Problem p, UnitTab ut) {
    using C = Cfg<D_IN, D_OUT>;
    __shared__ u32x4 smem[C::TOTAL];
    u32x4* W1s = smem + C::OFF_W1;
    u32x4* W2s = smem + C::OFF_W2;
    u32x4* B1s = smem + C::OFF_B1;
    float* Gs = reinterpret_cast<float*>(smem + C::OFF_G);

    const uint32_t code = ut.code[blockIdx.y];
    const int j = unit_j(code), x = unit_x(code), i = unit_i(code);
    const int E = p.E, hidden = p.hidden, EH = E * hidden;
    const size_t unit = (size_t)j * 2 + x;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int g = lane >> 5, l32 = lane & 31;
    const uint32_t gmask = 0u - (uint32_t)g;   // all ones in the upper lane half
    const int tok0 = blockIdx.x * C::BM;
    const int my_tok = tok0 + 32 * w + l32;

    const uint16_t* W1u = reinterpret_cast<const uint16_t*>(p.w1) + unit * EH * D_IN;
    const uint16_t* W2u = reinterpret_cast<const uint16_t*>(p.w2) + unit * E * D_OUT * hidden;
    const uint16_t* b1u = p.b1 ? reinterpret_cast<const uint16_t*>(p.b1) + unit * EH : nullptr;
    const uint16_t* b2u = p.b2 ? reinterpret_cast<const uint16_t*>(p.b2) + unit * E * D_OUT : nullptr;
    const uint16_t* Wru = reinterpret_cast<const uint16_t*>(p.wr) + unit * E * D_IN;
    float* Gw = Gs + w * (MOT_MAX_EXPERTS * 32);   // this wave's gates [m][32 tokens]

    // ---- stage loaders (each thread issues its share of direct-to-LDS loads)
    auto load_w1 = [&](int c, int st) {
#pragma unroll
        for (int r = 0; r < C::W1_ROUNDS; ++r) {
            const int slot = r * 256 + w * 64 + lane;
            const int row = slot / C::CPR1, pc = slot % C::CPR1, cl = pc ^ (row & 7);
            const uint16_t* src = W1u + (size_t)(c * 32 + w1_perm(row)) * D_IN + cl * 8;
            load_lds16(src, W1s + st * C::W1_CH + r * 256 + w * 64);
        }
        if (b1u && w == 0 && lane < 4)
            load_lds16(b1u + c * 32 + lane * 8, B1s + st * 4);
    };
    auto load_w2 = [&](int c, int st) {
        const int m = (c * 32) / hidden, kk0 = (c * 32) % hidden;
        const uint16_t* base = W2u + (size_t)m * D_OUT * hidden + kk0;
#pragma unroll
        for (int r = 0; r < C::W2_ROUNDS; ++r) {
            const int slot = r * 256 + w * 64 + lane;
            const int o = slot >> 2, pc = slot & 3, cl = pc ^ ((o >> 1) & 3);
            load_lds16(base + (size_t)o * hidden + cl * 8, W2s + st * C::W2_CH + r * 256 + w * 64);
        }
    };

    // ---- source rows -> VGPRs (B operand of layer 1 and of the router)
    u32x4 zf[C::KS1];
    {
        const bool ok = my_tok < p.n_tok;
        const uint16_t* src = reinterpret_cast<const uint16_t*>(p.src[x]) + (size_t)i * p.n_tok * D_IN;
        const int b = ok ? my_tok / p.T : 0, t = ok ? my_tok % p.T : 0;
#pragma unroll
        for (int s = 0; s < C::KS1; ++s) {
            const int k = 16 * s + 8 * g;
            size_t off;
            if (p.src_layout == MOT_LAYOUT_BTHD) {
                off = (size_t)my_tok * D_IN + k;
            } else {
                const int hh = k / p.D_src, dd = k % p.D_src;
                off = (((size_t)b * p.H_src + hh) * p.T + t) * p.D_src + dd;
            }
            const u32x4 zero = {0u, 0u, 0u, 0u};
            zf[s] = ok ? *reinterpret_cast<const u32x4*>(src + off) : zero;
        }
    }

    // ---- router on MFMA: stage Wr (rows >= E zero) in the second W1 stage
    {
        u32x4* Rs = W1s + C::W1_CH;
#pragma unroll
        for (int r = 0; r < C::W1_ROUNDS; ++r) {
            const int slot = r * 256 + tid;
            const int row = slot / C::CPR1, pc = slot % C::CPR1, cl = pc ^ (row & 7);
            const u32x4 zero = {0u, 0u, 0u, 0u};
            Rs[slot] = row < E ? *reinterpret_cast<const u32x4*>(Wru + (size_t)row * D_IN + cl * 8) : zero;
        }
        if (!b1u && tid < 8) {
            const u32x4 zero = {0u, 0u, 0u, 0u};
            B1s[tid] = zero;
        }
    }
    // prefetch the first W1/b1 chunk while the router runs
    load_w1(0, 0);
    __syncthreads();
    float gate_all[MOT_MAX_EXPERTS];
    {
        const u32x4* Rs = W1s + C::W1_CH;
        f32x16 lg;
#pragma unroll
        for (int e = 0; e < 16; ++e) lg[e] = 0.f;
#pragma unroll
        for (int s = 0; s < C::KS1; ++s) {
            const u32x4 a = Rs[l32 * C::CPR1 + ((2 * s + g) ^ (l32 & 7))];
            lg = mfma_32x32x16(a, zf[s], lg);
        }
        // lane half g holds experts 8*ii + 4*g + jj (ii = 0, 1) of token l32;
        // fetch the other half's four-expert groups from lane ^ 32
        float own[8], oth[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            own[e] = lg[e];
            oth[e] = __shfl_xor(lg[e], 32, 64);
        }
        float logit[16];
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
            logit[jj] = pick(gmask, own[jj], oth[jj]);
            logit[4 + jj] = pick(gmask, oth[jj], own[jj]);
            logit[8 + jj] = pick(gmask, own[4 + jj], oth[4 + jj]);
            logit[12 + jj] = pick(gmask, oth[4 + jj], own[4 + jj]);
        }
        const uint16_t* bru = p.br ? reinterpret_cast<const uint16_t*>(p.br) + unit * E : nullptr;
        float mx = -INFINITY;
#pragma unroll
        for (int m = 0; m < MOT_MAX_EXPERTS; ++m) {
            if (m < E) {
                if (bru) logit[m] += bf16_to_f32(bru[m]);
                mx = fmaxf(mx, logit[m]);
            }
        }
        float den = 0.f;
#pragma unroll
        for (int m = 0; m < MOT_MAX_EXPERTS; ++m) {
            gate_all[m] = m < E ? __expf(logit[m] - mx) : 0.f;
            den += gate_all[m];
        }
        const float inv = 1.0f / den;
#pragma unroll
        for (int m = 0; m < MOT_MAX_EXPERTS; ++m) gate_all[m] *= inv;
        if (g == 0) {
#pragma unroll
            for (int m = 0; m < MOT_MAX_EXPERTS; ++m)
                if (m < E) Gw[m * 32 + l32] = gate_all[m];
        }
    }
    __syncthreads();   // gates visible; router stage free again

    // ---- output accumulators seeded with sum_m g_m b2_m[o], on MFMA:
    // A = gates (token rows, k = expert), B = b2 (k = expert, column o).
    // Each gate is split into bf16 hi + lo parts (two products) so the seed
    // carries ~16 mantissa bits of the fp32 gate.
    // acc[nb] fragment: column o = nb*32 + l32, rows (tokens) 8*ii + 4*g + jj
    f32x16 acc[C::NB];
#pragma unroll
    for (int nb = 0; nb < C::NB; ++nb)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[nb][e] = 0.f;
    if (b2u) {
        u32x4 ghi, glo;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const float g0 = pick(gmask, gate_all[2 * q], gate_all[8 + 2 * q]);
            const float g1 = pick(gmask, gate_all[2 * q + 1], gate_all[9 + 2 * q]);
            const uint32_t hi = pack_bf16x2(g0, g1);
            ghi[q] = hi;
            glo[q] = pack_bf16x2(g0 - bf16_lo(hi), g1 - bf16_hi(hi));
        }
#pragma unroll
        for (int nb = 0; nb < C::NB; ++nb) {
            const int o = nb * 32 + l32;
            u32x4 bv;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int m0 = 8 * g + 2 * q;
                const uint32_t v0 = m0 < E ? b2u[(size_t)m0 * D_OUT + o] : 0u;
                const uint32_t v1 = m0 + 1 < E ? b2u[(size_t)(m0 + 1) * D_OUT + o] : 0u;
                bv[q] = v0 | (v1 << 16);
            }
            acc[nb] = mfma_32x32x16(ghi, bv, acc[nb]);
            acc[nb] = mfma_32x32x16(glo, bv, acc[nb]);
        }
    }

    // ---- main loop over 32-wide hidden chunks, layer 2 one chunk behind
    const int nch = EH / 32;
    u32x4 a2_prev[2];
    for (int c = 0; c <= nch; ++c) {
        wait_vm_all();
        __syncthreads();   // chunk c of W1/b1 and chunk c-1 of W2 are in LDS
        if (c + 1 < nch) load_w1(c + 1, (c + 1) & 1);
        if (c < nch) load_w2(c, c & 1);

        u32x4 a2_cur[2];
        f32x16 s_acc;
        if (c < nch) {
            const int st = c & 1;
            const u32x4* W1c = W1s + st * C::W1_CH;
            const u32x4 bv0 = B1s[st * 4 + g], bv1 = B1s[st * 4 + 2 + g];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                s_acc[2 * q] = bf16_lo(bv0[q]);
                s_acc[2 * q + 1] = bf16_hi(bv0[q]);
                s_acc[8 + 2 * q] = bf16_lo(bv1[q]);
                s_acc[8 + 2 * q + 1] = bf16_hi(bv1[q]);
            }
#pragma unroll
            for (int s = 0; s < C::KS1; ++s) {
                const u32x4 a = W1c[l32 * C::CPR1 + ((2 * s + g) ^ (l32 & 7))];
                s_acc = mfma_32x32x16(a, zf[s], s_acc);
            }
        }
        if (c > 0) {
            const u32x4* W2c = W2s + ((c - 1) & 1) * C::W2_CH;
#pragma unroll
            for (int nb = 0; nb < C::NB; ++nb) {
                const int o = nb * 32 + l32;
#pragma unroll
                for (int s2 = 0; s2 < 2; ++s2) {
                    const u32x4 b = W2c[o * 4 + ((2 * s2 + g) ^ ((o >> 1) & 3))];
                    acc[nb] = mfma_32x32x16(a2_prev[s2], b, acc[nb]);
                }
            }
        }
        if (c < nch) {
            const int m = (c * 32) / hidden;
            const float gate = Gw[m * 32 + l32];
            float h[16];
            if (p.act == MOT_ACT_GELU) {
#pragma unroll
                for (int e = 0; e < 16; ++e) h[e] = gate * gelu_fast(s_acc[e]);
            } else {
#pragma unroll
                for (int e = 0; e < 16; ++e) h[e] = gate * s_acc[e];
            }
#pragma unroll
            for (int s2 = 0; s2 < 2; ++s2) {
                u32x4 v;
#pragma unroll
                for (int q = 0; q < 4; ++q) v[q] = pack_bf16x2(h[8 * s2 + 2 * q], h[8 * s2 + 2 * q + 1]);
                a2_cur[s2] = v;
            }
            a2_prev[0] = a2_cur[0];
            a2_prev[1] = a2_cur[1];
        }
    }

    // ---- epilogue: bf16 round and store in the target layout
    uint16_t* dst = reinterpret_cast<uint16_t*>(p.dst[x]) + (size_t)j * p.n_tok * D_OUT;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
        const int tok = tok0 + 32 * w + 8 * (e >> 2) + 4 * g + (e & 3);
        if (tok >= p.n_tok) continue;
        const int b = tok / p.T, t = tok % p.T;
#pragma unroll
        for (int nb = 0; nb < C::NB; ++nb) {
            const int o = nb * 32 + l32;
            size_t off;
            if (p.dst_layout == MOT_LAYOUT_BTHD) {
                off = (size_t)tok * D_OUT + o;
            } else {
                const int hh = o / p.D_tgt, dd = o % p.D_tgt;
                off = (((size_t)b * p.H_tgt + hh) * p.T + t) * p.D_tgt + dd;
            }
            dst[off] = (uint16_t)(pack_bf16x2(acc[nb][e], 0.f) & 0xFFFFu);
        }
    }
}

template <int D_IN, int D_OUT>
hipError_t launch_t(const Problem& p, const UnitTab& ut, hipStream_t stream) {
    dim3 grid(p.n_tok_pad / 128, ut.n);
    hipLaunchKernelGGL((k_bf16_fused<D_IN, D_OUT>), grid, dim3(256), 0, stream, p, ut);
    return hipGetLastError();
}

template <int D_IN>
hipError_t launch_din(const Problem& p, const UnitTab& ut, hipStream_t stream) {
    switch (p.d_out) {
        case 128: return launch_t<D_IN, 128>(p, ut, stream);
        case 256: return launch_t<D_IN, 256>(p, ut, stream);
        case 512: return launch_t<D_IN, 512>(p, ut, stream);
        default: return hipErrorNotSupported;
    }
}

}  // namespace

bool fused_supported(const Problem& p) {
    const bool din = p.d_in == 128 || p.d_in == 256 || p.d_in == 512;
    const bool dout = p.d_out == 128 || p.d_out == 256 || p.d_out == 512;
    return din && dout && p.hidden % 32 == 0 && p.E <= MOT_MAX_EXPERTS;
}

hipError_t launch_bf16_fused(const Problem& p, const UnitTab& ut, hipStream_t stream) {
    if (ut.n == 0 || p.n_tok == 0) return hipSuccess;
    switch (p.d_in) {
        case 128: return launch_din<128>(p, ut, stream);
        case 256: return launch_din<256>(p, ut, stream);
        case 512: return launch_din<512>(p, ut, stream);
        default: return hipErrorNotSupported;
    }
}

}  // namespace mot
