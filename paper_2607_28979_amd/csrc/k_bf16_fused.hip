// Fused bf16 translation kernel: router + translator layer 1 + GELU + gate +
// translator layer 2 + gated mix + store, in one pass per token tile.  The
// E*hidden activations of a token never leave the chip.
//
// Workgroup = one unit (target layer, K or V) x TB token blocks of 32
// (TB = 4, or 3 when d_out = 512 so the output accumulators leave AGPR room
// for layer 1); four waves, one per SIMD.  Wave w:
//   * holds the source rows of token block w (32 x d_in bf16) in VGPRs as
//     MFMA B operands for the whole kernel (with TB = 3, wave 3 runs a
//     discarded layer-1 block on zero rows: it keeps the loop branch-free and
//     costs no time, since waves 0..2 set the pace);
//   * router: logits = Wr z on MFMA (Wr zero-padded to 32 rows), fp32
//     softmax -> gates (paper Sec. 3, Definition "Mixture-of-Translators");
//   * owns output columns [w*d_out/4, (w+1)*d_out/4) for all TB blocks; its
//     accumulators are seeded with sum_m g_m b2_m[o] by small MFMAs;
//   * walks E*hidden in 32-wide chunks (each inside one translator m) as a
//     three-stage software pipeline; iteration c runs, independently,
//       layer 1 of chunk c:   S^T = W1_m[c] z^T + b1   (MFMA, A = W1 from LDS)
//       GELU of chunk c-1:    H = bf16(g_m * GELU(S))  (VALU; written to LDS)
//       layer 2 of chunk c-2: Y += H . W2_m[:, c]^T    (MFMA, A = H, B = W2)
//     so matrix-core and vector work overlap; the expert reduction of the
//     gated sum happens inside Y.
//   W1's 32 rows are staged in a permuted order (w1_perm) that makes each
//   lane's layer-1 accumulator fragment exactly the 16-byte A-operand pieces
//   of layer 2.  Weight chunks move global -> LDS with direct-to-LDS 16-byte
//   loads, one chunk ahead; LDS tiles are XOR-swizzled in 16-byte units so
//   every fragment read is bank-conflict free.
//   * Y is rounded to bf16 and stored in the target layout.
#include <type_traits>

#include "mot_device.h"
#include "mot_internal.h"
#include "../../include/mot.h"

namespace mot {

namespace {

typedef __attribute__((address_space(3))) void lds_void;

template <int D_IN, int D_OUT>
struct Cfg {
    static constexpr int TB = D_OUT == 512 ? 3 : 4;   // token blocks per workgroup
    static constexpr int BM = 32 * TB;            // tokens per workgroup
    static constexpr int KS1 = D_IN / 16;         // layer-1 k-steps
    static constexpr int OUTW = D_OUT / 4;        // output columns per wave
    static constexpr int NBW = OUTW / 32;         // output blocks per wave
    static constexpr int CPR1 = D_IN / 8;         // 16-byte chunks per W1 row
    static constexpr int W1_CH = 32 * CPR1;       // chunks per W1 stage
    static constexpr int W2_CH = D_OUT * 4;       // chunks per W2 stage (32 hidden = 4 chunks)
    static constexpr int H_CH = 4 * 128;          // chunks per hidden stage (4 blocks x 32 tokens x 32)
    static constexpr int W1_ROUNDS = W1_CH / 256;
    static constexpr int W2_ROUNDS = W2_CH / 256;
    static constexpr int GS = 4 * MOT_MAX_EXPERTS * 32;   // gate floats (4 token blocks)
    // LDS map in 16-byte units
    static constexpr int OFF_W1 = 0;
    static constexpr int OFF_W2 = OFF_W1 + 2 * W1_CH;
    static constexpr int OFF_H = OFF_W2 + 2 * W2_CH;
    static constexpr int OFF_G = OFF_H + 2 * H_CH;
    static constexpr int TOTAL = OFF_G + GS / 4;
    static_assert(W1_CH % 256 == 0 && W2_CH % 256 == 0 && NBW >= 1, "tile shape");
};

// Row r of a staged 32-row W1 block holds hidden row w1_perm(r) of the chunk,
// so the layer-1 accumulator fragment (rows 8*i + 4*g + j of lane half g)
// lists hidden values 8g..8g+7 (i < 2) and 16+8g..16+8g+7 (i >= 2): the two
// 16-wide k-slices of the layer-2 A operand.
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

// Compile-time loop: f(std::integral_constant<int, I>) for I in [B, E).
template <int B, int E, class F>
__device__ __forceinline__ void static_for(F&& f) {
    if constexpr (B < E) {
        f(std::integral_constant<int, B>{});
        static_for<B + 1, E>(f);
    }
}

template <int D_IN, int D_OUT, int ACT>
__global__ __launch_bounds__(256, 1) __attribute__((amdgpu_waves_per_eu(1, 1)))
void k_bf16_fused(Problem p, UnitTab ut) {
    using C = Cfg<D_IN, D_OUT>;
    constexpr int TB = C::TB;
    __shared__ u32x4 smem[C::TOTAL];
    u32x4* W1s = smem + C::OFF_W1;
    u32x4* W2s = smem + C::OFF_W2;
    u32x4* Hs = smem + C::OFF_H;
    float* Gs = reinterpret_cast<float*>(smem + C::OFF_G);

    const uint32_t code = ut.code[blockIdx.y];
    const int j = unit_j(code), x = unit_x(code), i = unit_i(code);
    const int E = p.E, hidden = p.hidden, EH = E * hidden;
    const size_t unit = (size_t)j * 2 + x;
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 5, l32 = lane & 31;
    const uint32_t gmask = 0u - (uint32_t)g;   // all ones in the upper lane half
    const int tok0 = blockIdx.x * C::BM;
    const int my_tok = tok0 + 32 * w + l32;

    const uint16_t* W1u = reinterpret_cast<const uint16_t*>(p.w1) + unit * EH * D_IN;
    const uint16_t* W2u = reinterpret_cast<const uint16_t*>(p.w2) + unit * E * D_OUT * hidden;
    // layer-1 bias: without one, read W1 instead and mask the bits to zero
    const uint16_t* b1u = p.b1 ? reinterpret_cast<const uint16_t*>(p.b1) + unit * EH : W1u;
    const uint32_t b1_mask = p.b1 ? 0xFFFFFFFFu : 0u;
    const uint16_t* b2u = p.b2 ? reinterpret_cast<const uint16_t*>(p.b2) + unit * E * D_OUT : nullptr;
    const uint16_t* Wru = reinterpret_cast<const uint16_t*>(p.wr) + unit * E * D_IN;

    // ---- loop-invariant per-lane offsets of the direct-to-LDS loads
    uint32_t off_w1[C::W1_ROUNDS], off_w2[C::W2_ROUNDS];
#pragma unroll
    for (int r = 0; r < C::W1_ROUNDS; ++r) {
        const int slot = r * 256 + w * 64 + lane;
        const int row = slot / C::CPR1, pc = slot % C::CPR1, cl = pc ^ (row & 7);
        off_w1[r] = (uint32_t)(w1_perm(row) * D_IN + cl * 8);
    }
#pragma unroll
    for (int r = 0; r < C::W2_ROUNDS; ++r) {
        const int slot = r * 256 + w * 64 + lane;
        const int o = slot >> 2, pc = slot & 3, cl = pc ^ ((o >> 1) & 3);
        off_w2[r] = (uint32_t)(o * hidden + cl * 8);
    }
    auto load_w1 = [&](int c, int st) {
        const uint16_t* base = W1u + (size_t)c * 32 * D_IN;
#pragma unroll
        for (int r = 0; r < C::W1_ROUNDS; ++r)
            load_lds16(base + off_w1[r], W1s + st * C::W1_CH + r * 256 + w * 64);
    };
    // W2 columns [kk, kk+32) of translator m into stage st
    auto load_w2 = [&](int m, int kk, int st) {
        const uint16_t* base = W2u + (size_t)m * D_OUT * hidden + kk;
#pragma unroll
        for (int r = 0; r < C::W2_ROUNDS; ++r)
            load_lds16(base + off_w2[r], W2s + st * C::W2_CH + r * 256 + w * 64);
    };
    // the two 8-value pieces of b1 lane half g needs for chunk c
    auto load_b1 = [&](int c, u32x4* bv) {
        typedef const __attribute__((address_space(1))) u32x4* gvec;
        const uint16_t* bp = b1u + c * 32;
        bv[0] = *(gvec)(bp + 8 * g) & b1_mask;
        bv[1] = *(gvec)(bp + 16 + 8 * g) & b1_mask;
    };

    // ---- source rows -> VGPRs (B operand of layer 1 and of the router)
    u32x4 zf[C::KS1];
    {
        const bool ok = w < TB && my_tok < p.n_tok;
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
    }
    load_w1(0, 0);   // first W1 chunk in flight while the router runs
    __syncthreads();
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
        float gate_all[MOT_MAX_EXPERTS];
        float den = 0.f;
#pragma unroll
        for (int m = 0; m < MOT_MAX_EXPERTS; ++m) {
            gate_all[m] = m < E ? __expf(logit[m] - mx) : 0.f;
            den += gate_all[m];
        }
        const float inv = 1.0f / den;
        if (g == 0) {
            float* Gw = Gs + w * (MOT_MAX_EXPERTS * 32);
#pragma unroll
            for (int m = 0; m < MOT_MAX_EXPERTS; ++m)
                if (m < E) Gw[m * 32 + l32] = gate_all[m] * inv;
        }
    }
    __syncthreads();   // all gates visible; router stage free again

    // ---- output accumulators, seeded with sum_m g_m b2_m[o] on MFMA:
    // A = gates of a token block (k = translator), B = b2 (k = translator).
    // Gates are split into bf16 high + residual parts (two products) so the
    // seed keeps ~16 mantissa bits of the fp32 gates.
    // acc[tb][nb]: column o = w*OUTW + nb*32 + l32, rows = tokens
    // tb*32 + 8*ii + 4*g + jj (element 4*ii + jj).
    f32x16 acc[TB][C::NBW];
#pragma unroll
    for (int tb = 0; tb < TB; ++tb)
#pragma unroll
        for (int nb = 0; nb < C::NBW; ++nb)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[tb][nb][e] = 0.f;
    if (b2u) {
        u32x4 bv[C::NBW];
#pragma unroll
        for (int nb = 0; nb < C::NBW; ++nb) {
            const int o = w * C::OUTW + nb * 32 + l32;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int m0 = 8 * g + 2 * q;
                const uint32_t v0 = m0 < E ? b2u[(size_t)m0 * D_OUT + o] : 0u;
                const uint32_t v1 = m0 + 1 < E ? b2u[(size_t)(m0 + 1) * D_OUT + o] : 0u;
                bv[nb][q] = v0 | (v1 << 16);
            }
        }
#pragma unroll
        for (int tb = 0; tb < TB; ++tb) {
            const float* Gt = Gs + tb * (MOT_MAX_EXPERTS * 32);
            u32x4 ghi, glo;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int m0 = 8 * g + 2 * q;
                const float g0 = m0 < E ? Gt[m0 * 32 + l32] : 0.f;
                const float g1 = m0 + 1 < E ? Gt[(m0 + 1) * 32 + l32] : 0.f;
                const uint32_t hi = pack_bf16x2(g0, g1);
                ghi[q] = hi;
                glo[q] = pack_bf16x2(g0 - bf16_lo(hi), g1 - bf16_hi(hi));
            }
#pragma unroll
            for (int nb = 0; nb < C::NBW; ++nb) {
                acc[tb][nb] = mfma_32x32x16(ghi, bv[nb], acc[tb][nb]);
                acc[tb][nb] = mfma_32x32x16(glo, bv[nb], acc[tb][nb]);
            }
        }
    }

    // ---- pipeline stages
    const float* Gw = Gs + w * (MOT_MAX_EXPERTS * 32);
    // layer 1 of chunk c from W1 stage c&1, bias bv preloaded into the accumulator
    auto layer1 = [&](int c, const u32x4* bv) -> f32x16 {
        const u32x4* W1c = W1s + (c & 1) * C::W1_CH;
        f32x16 s;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            s[2 * q] = bf16_lo(bv[0][q]);
            s[2 * q + 1] = bf16_hi(bv[0][q]);
            s[8 + 2 * q] = bf16_lo(bv[1][q]);
            s[8 + 2 * q + 1] = bf16_hi(bv[1][q]);
        }
#pragma unroll
        for (int k = 0; k < C::KS1; ++k) {
            const u32x4 a = W1c[l32 * C::CPR1 + ((2 * k + g) ^ (l32 & 7))];
            s = mfma_32x32x16(a, zf[k], s);
        }
        return s;
    };
    // gate-scaled GELU of chunk c (translator m), written to hidden stage c&1
    // in fragment order [token block][k-slice][lane half][token]
    auto gelu_store = [&](int c, int m, const f32x16& s) {
        const float hg = 0.5f * Gw[m * 32 + l32];
        float h[16];
#pragma unroll
        for (int e = 0; e < 16; ++e)
            h[e] = ACT == MOT_ACT_GELU ? gelu_half_scaled(s[e], hg) : 2.0f * hg * s[e];
        u32x4* Hc = Hs + (c & 1) * C::H_CH + w * 128;
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            u32x4 v;
#pragma unroll
            for (int q = 0; q < 4; ++q) v[q] = pack_bf16x2(h[8 * ks + 2 * q], h[8 * ks + 2 * q + 1]);
            Hc[ks * 64 + g * 32 + l32] = v;
        }
    };
    // layer 2 of chunk c: all TB token blocks x this wave's output blocks
    auto layer2 = [&](int c) {
        const u32x4* Hc = Hs + (c & 1) * C::H_CH;
        const u32x4* W2c = W2s + (c & 1) * C::W2_CH;
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            u32x4 bw[C::NBW];
#pragma unroll
            for (int nb = 0; nb < C::NBW; ++nb) {
                const int o = w * C::OUTW + nb * 32 + l32;
                bw[nb] = W2c[o * 4 + ((2 * ks + g) ^ ((o >> 1) & 3))];
            }
#pragma unroll
            for (int tb = 0; tb < TB; ++tb) {
                const u32x4 a = Hc[tb * 128 + ks * 64 + g * 32 + l32];
#pragma unroll
                for (int nb = 0; nb < C::NBW; ++nb) acc[tb][nb] = mfma_32x32x16(a, bw[nb], acc[tb][nb]);
            }
        }
    };
    auto sync_stage = [&]() {
        wait_vm_all();
        __syncthreads();
    };

    // One steady-state iteration as a fixed slot schedule: layer-1 MFMAs of
    // chunk c and layer-2 MFMAs of chunk c-2 are merged proportionally; every
    // LDS operand read is issued LOOK slots before its MFMA; the 16 GELU
    // evaluations of chunk c-1 are spread evenly over the slots; each slot is
    // fenced so the compiler keeps this order.
    auto steady_slots = [&](int c, int m, const u32x4* bv, const f32x16& sp, int cn, int m_w2,
                            int kk_w2, u32x4* bnext_out) -> f32x16 {
        constexpr int NL1 = C::KS1, NL2 = 2 * TB * C::NBW, NM = NL1 + NL2, LOOK = 3;
        // global -> LDS loads of the next W1 chunk and of W2 for chunk c-1,
        // plus the next b1 pieces, spread evenly over the slots
        constexpr int NV = C::W1_ROUNDS + C::W2_ROUNDS + 2;
        const uint16_t* w1_base = W1u + (size_t)cn * 32 * D_IN;
        u32x4* w1_dst = W1s + ((c + 1) & 1) * C::W1_CH + w * 64;
        const uint16_t* w2_base = W2u + (size_t)m_w2 * D_OUT * hidden + kk_w2;
        u32x4* w2_dst = W2s + ((c - 1) & 1) * C::W2_CH + w * 64;
        auto issue_vmem = [&](auto rc) {
            constexpr int r = decltype(rc)::value;
            if constexpr (r < C::W1_ROUNDS) {
                load_lds16(w1_base + off_w1[r], w1_dst + r * 256);
            } else if constexpr (r < C::W1_ROUNDS + C::W2_ROUNDS) {
                constexpr int q = r - C::W1_ROUNDS;
                load_lds16(w2_base + off_w2[q], w2_dst + q * 256);
            } else if constexpr (r == NV - 2) {
                load_b1(cn, bnext_out);
            }
        };
        const u32x4* W1c = W1s + (c & 1) * C::W1_CH;
        const u32x4* Hc = Hs + (c & 1) * C::H_CH;          // chunk c-2 shares c's parity
        const u32x4* W2c = W2s + (c & 1) * C::W2_CH;
        u32x4* Hw = Hs + ((c - 1) & 1) * C::H_CH + w * 128;
        const float hg = 0.5f * Gw[m * 32 + l32];
        f32x16 s;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            s[2 * q] = bf16_lo(bv[0][q]);
            s[2 * q + 1] = bf16_hi(bv[0][q]);
            s[8 + 2 * q] = bf16_lo(bv[1][q]);
            s[8 + 2 * q + 1] = bf16_hi(bv[1][q]);
        }
        u32x4 a1[NL1], hA[2][TB], bW[2][C::NBW];
        float h[16], gx[16], gt[16], gx2[16], gq[16], ge[16];
        constexpr int GD = 2;   // slots between GELU stages
        // operand reads needed by slot k
        auto issue_reads = [&](auto kc) {
            constexpr int k = decltype(kc)::value;
            if constexpr (k < NM) {
                constexpr int n1 = (k * NL1) / NM;
                if constexpr (((k + 1) * NL1) / NM > n1) {
                    a1[n1] = W1c[l32 * C::CPR1 + ((2 * n1 + g) ^ (l32 & 7))];
                } else {
                    constexpr int q = k - n1, ks = q / (TB * C::NBW), tb = (q / C::NBW) % TB,
                                  nb = q % C::NBW;
                    if constexpr (nb == 0) hA[ks][tb] = Hc[tb * 128 + ks * 64 + g * 32 + l32];
                    if constexpr (tb == 0) {
                        const int o = w * C::OUTW + nb * 32 + l32;
                        bW[ks][nb] = W2c[o * 4 + ((2 * ks + g) ^ ((o >> 1) & 3))];
                    }
                }
            }
        };
        static_for<0, LOOK>([&](auto kc) { issue_reads(kc); });
        static_for<0, NM>([&](auto kc) {
            constexpr int k = decltype(kc)::value;
            static_for<0, NV>([&](auto rc) {
                if constexpr ((decltype(rc)::value * NM) / NV == k) issue_vmem(rc);
            });
            issue_reads(std::integral_constant<int, k + LOOK>{});
            constexpr int n1 = (k * NL1) / NM;
            if constexpr (((k + 1) * NL1) / NM > n1) {
                s = mfma_32x32x16(a1[n1], zf[n1], s);
            } else {
                constexpr int q = k - n1, ks = q / (TB * C::NBW), tb = (q / C::NBW) % TB,
                              nb = q % C::NBW;
                acc[tb][nb] = mfma_32x32x16(hA[ks][tb], bW[ks][nb], acc[tb][nb]);
            }
            // GELU of element e runs as three stages in slots g0(e), g0(e)+GD,
            // g0(e)+2*GD, so several independent chains overlap in each slot
            static_for<0, 16>([&](auto ec) {
                constexpr int e = decltype(ec)::value;
                constexpr int g0 = (e * (NM - 2 * GD - 1)) / 15;
                if constexpr (ACT == MOT_ACT_GELU) {
                    if constexpr (k == g0) {
                        float v = sp[e];
                        asm volatile("" : "+v"(v));
                        gx[e] = v;
                        gelu_stage1(v, gt[e], gx2[e]);
                        asm volatile("" : "+v"(gt[e]), "+v"(gx2[e]));
                    } else if constexpr (k == g0 + GD) {
                        gelu_stage2(gt[e], gx2[e], gq[e], ge[e]);
                        asm volatile("" : "+v"(gq[e]), "+v"(ge[e]));
                    } else if constexpr (k == g0 + 2 * GD) {
                        h[e] = gelu_stage3(gx[e], gt[e], gq[e], ge[e], hg);
                    }
                } else if constexpr (k == g0) {
                    float v = sp[e];
                    asm volatile("" : "+v"(v));
                    h[e] = 2.0f * hg * v;
                }
            });
            __builtin_amdgcn_sched_barrier(0);
        });
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            u32x4 v;
#pragma unroll
            for (int q = 0; q < 4; ++q) v[q] = pack_bf16x2(h[8 * ks + 2 * q], h[8 * ks + 2 * q + 1]);
            Hw[ks * 64 + g * 32 + l32] = v;
        }
        return s;
    };

    // ---- prologue (chunks 0, 1), steady state, drain.  (m1, kk1) = the
    // translator and column offset of chunk c-1, advanced by 32 per step.
    const int nch = EH / 32;   // >= 2
    int m1 = 0, kk1 = 0;
    auto advance = [&]() {
        kk1 += 32;
        const bool wrap = kk1 == hidden;
        kk1 = wrap ? 0 : kk1;
        m1 = wrap ? m1 + 1 : m1;
    };
    u32x4 bcur[2], bnext[2];
    load_b1(0, bcur);
    f32x16 s_prev;
    sync_stage();                          // iteration 0
    load_w1(1, 1);
    load_b1(1, bnext);
    s_prev = layer1(0, bcur);
    bcur[0] = bnext[0]; bcur[1] = bnext[1];
    sync_stage();                          // iteration 1
    load_w1(nch > 2 ? 2 : nch - 1, 0);
    load_w2(m1, kk1, 0);
    load_b1(nch > 2 ? 2 : nch - 1, bnext);
    {
        f32x16 s_new = layer1(1, bcur);
        gelu_store(0, m1, s_prev);
        s_prev = s_new;
    }
    advance();
    bcur[0] = bnext[0]; bcur[1] = bnext[1];
    for (int c = 2; c < nch; ++c) {        // steady state: one basic block
        sync_stage();
        const int cn = c + 1 < nch ? c + 1 : nch - 1;
        f32x16 s_new = steady_slots(c, m1, bcur, s_prev, cn, m1, kk1, bnext);
        s_prev = s_new;
        advance();
        bcur[0] = bnext[0]; bcur[1] = bnext[1];
    }
    sync_stage();                          // iteration nch
    load_w2(m1, kk1, (nch - 1) & 1);
    gelu_store(nch - 1, m1, s_prev);
    layer2(nch - 2);
    sync_stage();                          // iteration nch + 1
    layer2(nch - 1);

    // ---- epilogue: bf16 round and store in the target layout
    uint16_t* dst = reinterpret_cast<uint16_t*>(p.dst[x]) + (size_t)j * p.n_tok * D_OUT;
#pragma unroll
    for (int tb = 0; tb < TB; ++tb) {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const int tok = tok0 + tb * 32 + 8 * (e >> 2) + 4 * g + (e & 3);
            if (tok >= p.n_tok) continue;
            const int b = tok / p.T, t = tok % p.T;
#pragma unroll
            for (int nb = 0; nb < C::NBW; ++nb) {
                const int o = w * C::OUTW + nb * 32 + l32;
                size_t off;
                if (p.dst_layout == MOT_LAYOUT_BTHD) {
                    off = (size_t)tok * D_OUT + o;
                } else {
                    const int hh = o / p.D_tgt, dd = o % p.D_tgt;
                    off = (((size_t)b * p.H_tgt + hh) * p.T + t) * p.D_tgt + dd;
                }
                dst[off] = (uint16_t)(pack_bf16x2(acc[tb][nb][e], 0.f) & 0xFFFFu);
            }
        }
    }
}

template <int D_IN, int D_OUT>
hipError_t launch_t(const Problem& p, const UnitTab& ut, hipStream_t stream) {
    using C = Cfg<D_IN, D_OUT>;
    dim3 grid((p.n_tok + C::BM - 1) / C::BM, ut.n);
    if (p.act == MOT_ACT_GELU)
        hipLaunchKernelGGL((k_bf16_fused<D_IN, D_OUT, MOT_ACT_GELU>), grid, dim3(256), 0, stream, p, ut);
    else
        hipLaunchKernelGGL((k_bf16_fused<D_IN, D_OUT, MOT_ACT_IDENTITY>), grid, dim3(256), 0, stream, p, ut);
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
    return din && dout && p.hidden % 32 == 0 && p.E * p.hidden >= 64 && p.E <= MOT_MAX_EXPERTS;
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
