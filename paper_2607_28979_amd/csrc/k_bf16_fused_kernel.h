// Fused bf16 translation kernel: router + translator layer 1 + GELU + gate +
// translator layer 2 + gated mix + store, in one pass per token tile (paper
// Sec. 3, Definition "Mixture-of-Translators", with the Linear-GELU-Linear
// translator body).  The E*hidden activations of a token never leave the chip.
//
// Workgroup = one unit (target layer, K or V) x TB token blocks of 32, with
// fixed wave roles:
//   * waves 0..TB-1: source rows of one token block in VGPRs (MFMA B operand)
//     for the whole kernel; router logits on MFMA, fp32 softmax, Top-K; then
//     per 32-wide chunk of E*hidden: layer 1 (S = W1_m[c] z^T, four
//     independent 16x16x32 accumulators started from the bias) and
//     g_m * GELU(S) -> bf16 hidden tile in LDS;
//   * waves 4..4+L2W-1: d_out/L2W output columns each, for all TB blocks;
//     accumulators seeded with sum_m g_m b2_m; per chunk
//     Y += H . W2_m[:, c]^T (32x32x16); they also issue every global -> LDS
//     weight load (direct-to-LDS, no VGPR staging).  L2W = 8 (two layer-2
//     waves per SIMD, TB = 4, 12 waves) when d_in <= 256 and d_out >= 256,
//     else 4 (8 waves);
//   * wave 3 when TB = 3 (d_in = d_out = 512): no block; evaluates part of
//     the layer-1 waves' GELU (fp32 values handed over through LDS).
// Iteration c runs layer 1 of chunk c, the GELU of chunk c-1 and layer 2 of
// chunk c-2, and fetches W1 of chunk c+1 and W2 of chunk c (three W2 stages)
// or c-1 (two); one workgroup barrier per iteration.  W1's 32 rows are staged
// in a permuted order (w1_perm) that leaves each lane, per token, 8
// consecutive hidden values: exactly a 16-byte piece of the layer-2 A operand.
// LDS tiles are XOR-swizzled in 16-byte units so every 16-lane group of a
// fragment read hits distinct banks.  Y is rounded to bf16 and stored in the
// target layout.
#pragma once

#include <type_traits>

#include "mot_device.h"
#include "mot_internal.h"
#include "../../include/mot.h"

namespace mot {

namespace {

typedef __attribute__((address_space(3))) void lds_void;

// Elements (of 16 per lane and chunk) whose GELU runs as vector-only work
// outside the layer-1 MFMA slots: before them (MOT_FUSED_A_LAST = 0) or after
// them (1)
#ifndef MOT_FUSED_PHASE_A
#define MOT_FUSED_PHASE_A 6
#endif
// The same count for the 12-wave form (two layer-2 waves per SIMD)
#ifndef MOT_FUSED_PHASE_A12
#define MOT_FUSED_PHASE_A12 16
#endif
#ifndef MOT_FUSED_A_LAST
#define MOT_FUSED_A_LAST 0
#endif
// 0: layer-1 waves are the older waves of each SIMD pair; 4: layer-2 waves are
#ifndef MOT_FUSED_ROLE_SHIFT
#define MOT_FUSED_ROLE_SHIFT 0
#endif
// Layer-2 waves per workgroup when d_out >= 256 and d_in <= 256: 4 (one per
// SIMD; d_out = 512 then takes 3 token blocks) or 8 (two per SIMD, each with
// half the output columns, which leaves room for 4 token blocks)
#ifndef MOT_FUSED_L2W
#define MOT_FUSED_L2W 8
#endif
// With TB = 3, wave 3 has no token block: it evaluates the GELU of this many
// of each layer-1 lane's 16 elements (0, 4 or 8: row half 1 of token half 1,
// or of both token halves), handed over through LDS in fp32.
#ifndef MOT_FUSED_OFFLOAD
#define MOT_FUSED_OFFLOAD 4
#endif
// Split iteration (12-wave form, off by default): the layer-1 waves evaluate
// all their GELU elements while the layer-2 waves run their MFMAs, then,
// after a mid-iteration barrier, the layer-1 waves run their MFMAs alone
#ifndef MOT_FUSED_SPLIT
#define MOT_FUSED_SPLIT 0
#endif
// Slots of the layer-2 waves' global -> LDS weight loads within an
// iteration: spread evenly over the MFMA slots (1) or issued in the first
// slots (0)
#ifndef MOT_FUSED_LOAD_SPREAD
#define MOT_FUSED_LOAD_SPREAD 1
#endif
// Wave priority (s_setprio) of the layer-1 waves during their MFMA slots
// (0: the default priority throughout)
#ifndef MOT_FUSED_L2_LOOK
#define MOT_FUSED_L2_LOOK 2   // layer-2 operand reads issued this many MFMA slots ahead
#endif
#ifndef MOT_FUSED_L1_PRIO
#define MOT_FUSED_L1_PRIO 0
#endif

template <int D_IN, int D_OUT>
struct Cfg {
    static constexpr int L2W = (D_OUT >= 256 && D_IN <= 256) ? MOT_FUSED_L2W : 4;   // layer-2 waves
    static constexpr int NW = 4 + L2W;                     // waves per workgroup
    static constexpr int TB = (D_OUT == 512 && L2W == 4) ? 3 : 4;   // token blocks per workgroup
    static constexpr int BM = 32 * TB;            // tokens per workgroup
    static constexpr int KS1 = D_IN / 16;         // layer-1 k-steps
    static constexpr int OUTW = D_OUT / L2W;      // output columns per layer-2 wave
    static constexpr int NBW = OUTW / 32;         // output blocks per wave
    static constexpr int CPR1 = D_IN / 8;         // 16-byte chunks per W1 row
    static constexpr int W1_CH = 32 * CPR1;       // chunks per W1 stage
    static constexpr int W2_CH = D_OUT * 4;       // chunks per W2 stage (32 hidden = 4 chunks)
    static constexpr int H_CH = TB * 128;         // chunks per hidden stage (TB blocks x 32 tokens x 32)
    static constexpr int GS = TB * MOT_MAX_EXPERTS * 32;  // gate floats
    static constexpr int NOFF = TB == 3 ? MOT_FUSED_OFFLOAD : 0;   // GELU elements on wave 3
    static constexpr int X_CH = TB * (NOFF / 4) * 64;   // hand-over stage: f32x4 per lane
    // W2 stages: three (each chunk fetched two iterations before its use)
    // when they fit in the 160 KB of LDS, else two (one iteration ahead)
    static constexpr int NW2 =
        (2 * W1_CH + 3 * W2_CH + 2 * H_CH + GS / 4 + 2 * X_CH) * 16 <= 160 * 1024 ? 3 : 2;
    // LDS map in 16-byte units
    static constexpr int OFF_W1 = 0;
    static constexpr int OFF_W2 = OFF_W1 + 2 * W1_CH;
    static constexpr int OFF_H = OFF_W2 + NW2 * W2_CH;
    static constexpr int OFF_G = OFF_H + 2 * H_CH;
    static constexpr int OFF_X = OFF_G + GS / 4;
    static constexpr int TOTAL = OFF_X + 2 * X_CH;
    static_assert(NOFF == 0 || NOFF == 4 || NOFF == 8, "offloaded GELU elements");
    static_assert(TOTAL * 16 <= 160 * 1024, "LDS");
    static_assert(W1_CH % 256 == 0 && W2_CH % 256 == 0 && NBW >= 1, "tile shape");
    static_assert(TB * NBW * 16 <= 192, "layer-2 accumulators must leave VGPR room");
    static constexpr bool SPLIT = MOT_FUSED_SPLIT && L2W == 8 && NOFF == 0;
};

// Row R of a staged 32-row W1 block holds hidden row w1_perm(R) of the chunk.
// Layer 1 runs as 16x16 MFMA blocks over row halves hh = R / 16; lane group q
// of a block's accumulator holds rows 4q + j, j = 0..3.  Mapping row
// hh*16 + 4q + j to hidden 8q + 4hh + j gives each lane, for one token, the
// eight consecutive hidden values 8q .. 8q+7: one 16-byte unit of the
// layer-2 A-operand tile.
__device__ __forceinline__ int w1_perm(int r) {
    const int hh = r >> 4, q = (r >> 2) & 3, jj = r & 3;
    return 8 * q + 4 * hh + jj;
}

// Weight loads go straight into LDS through a buffer descriptor
// (buffer_load_dwordx4 ... lds): 16 bytes per lane at voff (per lane) + soff
// (wave-uniform).  The MUBUF form, not global_load_lds: a pending FLAT-family
// load makes the compiler's wait insertion drain every outstanding LDS read
// (lgkmcnt(0)) before each use of an LDS operand, which defeats the layer-2
// waves' operand lookahead.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
__device__ __forceinline__ rsrc_t make_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ void load_lds16(rsrc_t r, uint32_t voff, uint32_t soff, u32x4* lds_dst_wave_base) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)lds_dst_wave_base, 16, voff, soff, 0, 0);
}

// 16 zero bytes: the layer-1 bias source when a call has no bias
static __device__ __align__(16) const u32x4 kZero16 = {0u, 0u, 0u, 0u};

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

// ROUTED: the workgroup runs one tile of the routed path: up to BM
// assignments (token, gate) of a single translator, gathered by token index;
// the router is skipped (the gates come with the assignments) and the E*hidden
// walk covers that translator's hidden only.
template <int D_IN, int D_OUT, int ACT, bool ROUTED>
__global__ __attribute__((amdgpu_flat_work_group_size(64 * Cfg<D_IN, D_OUT>::NW, 64 * Cfg<D_IN, D_OUT>::NW)))
void k_bf16_fused(Problem p, UnitTab ut) {
    using C = Cfg<D_IN, D_OUT>;
    constexpr int TB = C::TB;
    // the layer-2 waves issue the global -> LDS weight loads
    constexpr int NLD = C::L2W;
    constexpr int W1_RL = C::W1_CH / (64 * NLD), W2_RL = C::W2_CH / (64 * NLD);
    __shared__ u32x4 smem[C::TOTAL];
    u32x4* W1s = smem + C::OFF_W1;
    u32x4* W2s = smem + C::OFF_W2;
    u32x4* Hs = smem + C::OFF_H;
    float* Gs = reinterpret_cast<float*>(smem + C::OFF_G);
    u32x4* Xs = smem + C::OFF_X;   // fp32 layer-1 results handed to wave 3
    // Translator usage of the tile (non-routed mode): MOT_MAX_EXPERTS
    // counters in the last 64 bytes of W1 stage 1, which holds the router
    // rows during the router and is zeroed there for rows >= E (these words
    // are in row 31); W1 chunk 1 overwrites it only after the counters are
    // flushed.  Kept inside smem: a second LDS object would make the
    // compiler wait for every direct-to-LDS load before each LDS read.
    uint32_t* s_usage = reinterpret_cast<uint32_t*>(W1s + 2 * C::W1_CH) - MOT_MAX_EXPERTS;
    static_assert(C::W1_CH / C::CPR1 == 32 && C::CPR1 * 16 >= MOT_MAX_EXPERTS * 4, "usage counters in row 31");

    const uint32_t code = ut.code[blockIdx.y];
    const int j = unit_j(code), x = unit_x(code), i = unit_i(code);
    const size_t unit = (size_t)j * p.streams + x;
    // routed tile: {translator, first assignment, rows}; tiles beyond the
    // unit's count leave at once (uniform over the workgroup, before any barrier)
    int4 tile = make_int4(0, 0, 0, 0);
    if constexpr (ROUTED) {
        const int gs = unit_gslot(code);
        // Workgroups go to the 8 XCDs round-robin by linear id, and the tiles
        // of one translator are consecutive: give each XCD a contiguous run
        // of tiles (max_tiles is a multiple of 8), so the workgroups an XCD
        // runs together share one translator's weights in its L2.
        const int t = (int)(blockIdx.x % 8) * (p.rt.max_tiles / 8) + (int)(blockIdx.x / 8);
        if (t >= p.rt.ntiles[gs]) return;
        tile = p.rt.tiles[(size_t)gs * p.rt.max_tiles + t];
    }
    const int E = ROUTED ? 1 : p.E, hidden = p.hidden, EH = E * hidden;
    const size_t um = unit * p.E + (ROUTED ? tile.x : 0);   // first translator walked
    const int lane = threadIdx.x & 63;
    // logical wave index: hardware wave h plays role (h + MOT_FUSED_ROLE_SHIFT) % NW
    // (hardware waves h, h + 4, h + 8 share a SIMD)
    const int w = __builtin_amdgcn_readfirstlane(((threadIdx.x >> 6) + MOT_FUSED_ROLE_SHIFT) % C::NW);
    const int tid = w * 64 + lane;   // logical thread index
    const int g = lane >> 5, l32 = lane & 31;
    const uint32_t gmask = 0u - (uint32_t)g;   // all ones in the upper lane half
    const int tok0 = blockIdx.x * C::BM;
    const bool is_l1 = w < TB;                 // layer-1 + GELU wave of token block w
    const bool is_l2 = w >= 4;                 // layer-2 wave q = w - 4
    const int q2 = w - 4;                      // layer-2 column group
    const int lw = q2;                         // index among the loading waves

    const uint16_t* W1u = reinterpret_cast<const uint16_t*>(p.w1) + um * hidden * D_IN;
    const uint16_t* W2u = reinterpret_cast<const uint16_t*>(p.w2) + um * D_OUT * hidden;
    // layer-1 bias: without one, every lane reads the same 16 zero bytes
    // (chunk and lane strides 0), so no mask is needed at the use
    const uint16_t* b1u = p.b1 ? reinterpret_cast<const uint16_t*>(p.b1) + um * hidden
                               : reinterpret_cast<const uint16_t*>(&kZero16);
    const int b1_cstride = p.b1 ? 32 : 0;
    const uint16_t* b2u = p.b2 ? reinterpret_cast<const uint16_t*>(p.b2) + um * D_OUT : nullptr;
    const uint16_t* Wru = reinterpret_cast<const uint16_t*>(p.wr) + unit * E * D_IN;

    // ---- global -> LDS weight loads (the layer-2 waves)
    // Round r of a stage load fills LDS slots [r*256, r*256 + 256); this lane
    // fills slot r*256 + t.  Its global byte offset is a per-lane part plus a
    // part that depends on r only:
    //   W1: staged row r*RS + u (RS = 256/CPR1, u = t/CPR1), chunk t % CPR1;
    //       w1_perm and the (row & 15) swizzle act on the disjoint bits of
    //       r*RS and u, so only (r*RS) & 15 (NV1 values) changes the lane part;
    //   W2: output row 64r + t/4, swizzle ((row >> 2) & 3) the same for all r.
    const int t_ld = lw * 64 + lane;
    constexpr int RS = 64 * NLD / C::CPR1;
    constexpr int NV1 = RS < 16 ? 16 / RS : 1;
    auto w1_lane = [&](int v) -> uint32_t {
        const int u = t_ld / C::CPR1, pc = t_ld % C::CPR1;
        return (uint32_t)(w1_perm(u) * D_IN + ((pc ^ (u & 15)) ^ ((v * RS) & 15)) * 8) * 2u;
    };
    const uint32_t w2_lane = (uint32_t)((t_ld >> 2) * hidden + ((t_ld & 3) ^ ((t_ld >> 4) & 3)) * 8) * 2u;
    // chunk c of W1 (round r) into stage st; the chunk base is wave-uniform,
    // so each load is a scalar base plus a per-lane offset
    const rsrc_t w1buf = make_rsrc(W1u, (uint32_t)EH * D_IN * 2);
    const rsrc_t w2buf = make_rsrc(W2u, (uint32_t)EH * D_OUT * 2);
    auto load_w1_round = [&](int c, int st, int r, uint32_t lane_off) {
        const uint32_t soff = (uint32_t)(c * 32 * D_IN + w1_perm(r * RS) * D_IN) * 2u;
        load_lds16(w1buf, lane_off, soff, W1s + st * C::W1_CH + r * 64 * NLD + lw * 64);
    };
    // W2 columns [kk, kk+32) of translator m (round r) into stage st
    auto load_w2_round = [&](int m, int kk, int st, int r) {
        const uint32_t soff = (uint32_t)((m * D_OUT + 16 * NLD * r) * hidden + kk) * 2u;
        load_lds16(w2buf, w2_lane, soff, W2s + st * C::W2_CH + r * 64 * NLD + lw * 64);
    };
    const int nch = EH / 32;   // >= 2
    // The three roles run the same number of workgroup barriers: two around
    // the router, then one per pipeline iteration c = 0 .. nch+1.  Iteration c
    // runs layer 1 of chunk c, the GELU of chunk c-1 and layer 2 of chunk c-2;
    // the loading wave(s) fetch W1 of chunk c+1 and W2 of chunk c-1.
    // (m1, kk1) = translator and column offset of chunk c-1.
    auto stage_router_weights = [&]() {   // waves 0..3
        u32x4* Rs = W1s + C::W1_CH;
#pragma unroll
        for (int r = 0; r < C::W1_CH / 256; ++r) {
            const int slot = r * 256 + tid;
            const int row = slot / C::CPR1, pc = slot % C::CPR1, cl = pc ^ (row & 15);
            const u32x4 zero = {0u, 0u, 0u, 0u};
            Rs[slot] = row < E ? *reinterpret_cast<const u32x4*>(Wru + (size_t)row * D_IN + cl * 8) : zero;
        }
    };
    // Pipeline barrier.  Each wave first waits for its own LDS traffic and for
    // its global loads except the newest `keep` (LDS data produced by direct
    // loads is written when the load completes), then all waves meet.  No
    // fence: the waits above are all the ordering the pipeline needs, and a
    // fence would drain every outstanding load.
    auto sync_keep = [&](auto keepc) {
        constexpr int keep = decltype(keepc)::value;
        static_assert(keep >= 0 && keep < 64, "vmcnt range");
        __builtin_amdgcn_sched_barrier(0);
        asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)" :: "n"(keep) : "memory");
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        __builtin_amdgcn_sched_barrier(0);
    };
    auto sync_stage = [&]() { sync_keep(std::integral_constant<int, 0>{}); };
    // mid-iteration barrier of the split form: timing only, no data crosses it
    auto mid_barrier = [&]() {
        if constexpr (C::SPLIT) {
            __builtin_amdgcn_sched_barrier(0);
            __builtin_amdgcn_s_barrier();
            __builtin_amdgcn_sched_barrier(0);
        }
    };

    if (is_l1) {
        // ---------------------------------------------------------- layer 1
        // Layer 1 and the router use v_mfma_f32_16x16x32_bf16: the 32-token
        // block is two 16-token halves th, the 32 staged W1 rows two 16-row
        // halves hh, so the chunk's S block is four independent 16x16
        // accumulators (no dependent MFMA chain).  Lane l = 16*q + l16 holds
        // S rows 4q + j of each sub-block for token th*16 + l16.
        constexpr int KS2 = D_IN / 32;
        const int l16 = lane & 15, q4 = lane >> 4;
        u32x4 zf[2][KS2];   // B operand: token th*16 + l16, k = 32s + 8*q4 .. +7
        {
            const uint16_t* src = reinterpret_cast<const uint16_t*>(p.src[x]) + (size_t)i * p.n_tok * D_IN;
#pragma unroll
            for (int th = 0; th < 2; ++th) {
                const int r = 32 * w + 16 * th + l16;   // row of the tile
                const bool ok = ROUTED ? r < tile.z : tok0 + r < p.n_tok;
                const int my_tok = ROUTED ? (ok ? p.rt.list[(size_t)unit_gslot(code) * p.n_tok * p.top_k + tile.y + r] : 0)
                                          : tok0 + r;
                const int b = ok ? my_tok / p.T : 0, t = ok ? my_tok % p.T : 0;
#pragma unroll
                for (int s = 0; s < KS2; ++s) {
                    const int k = 32 * s + 8 * q4;
                    size_t off;
                    if (p.src_layout == MOT_LAYOUT_BTHD) {
                        off = (size_t)my_tok * D_IN + k;
                    } else {
                        const int hh = k / p.D_src, dd = k % p.D_src;
                        off = (((size_t)b * p.H_src + hh) * p.T + t) * p.D_src + dd;
                    }
                    const u32x4 zero = {0u, 0u, 0u, 0u};
                    zf[th][s] = ok ? *reinterpret_cast<const u32x4*>(src + off) : zero;
                }
            }
        }
        if constexpr (!ROUTED) stage_router_weights();
        __syncthreads();                                     // barrier A
        if constexpr (ROUTED) {
            // gates come with the assignments (translator 0 of this walk)
            float* Gw = Gs + w * (MOT_MAX_EXPERTS * 32);
            const float* ag = p.rt.agate + (size_t)unit_gslot(code) * p.n_tok * p.top_k + tile.y;
            if (q4 == 0) {
#pragma unroll
                for (int th = 0; th < 2; ++th) {
                    const int r = 32 * w + 16 * th + l16;
                    Gw[th * 16 + l16] = r < tile.z ? ag[r] : 0.f;
                }
            }
        } else {
            // router on MFMA: logits[expert][token] = Wr z (Wr rows >= E zero)
            const u32x4* Rs = W1s + C::W1_CH;
            const uint16_t* bru = p.br ? reinterpret_cast<const uint16_t*>(p.br) + unit * E : nullptr;
            float* Gw = Gs + w * (MOT_MAX_EXPERTS * 32);
#pragma unroll
            for (int th = 0; th < 2; ++th) {
                f32x4 lg = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int s = 0; s < KS2; ++s) {
                    const u32x4 a = Rs[l16 * C::CPR1 + ((4 * s + q4) ^ l16)];
                    lg = mfma_16x16x32(a, zf[th][s], lg);
                }
                // lane group q4 holds experts 4*q4 .. 4*q4+3 of token l16; the
                // other three groups' experts come from lanes ^ 16, ^ 32, ^ 48
                float src4[4][4];
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) {
                    src4[0][jj] = lg[jj];
                    src4[1][jj] = __shfl_xor(lg[jj], 16, 64);
                    src4[2][jj] = __shfl_xor(lg[jj], 32, 64);
                    src4[3][jj] = __shfl_xor(lg[jj], 48, 64);
                }
                float logit[16];
#pragma unroll
                for (int kq = 0; kq < 4; ++kq) {
                    // experts 4*kq.. live in the source with index q4 ^ kq
                    const uint32_t m0 = 0u - (uint32_t)((q4 ^ kq) & 1), m1 = 0u - (uint32_t)(((q4 ^ kq) >> 1) & 1);
#pragma unroll
                    for (int jj = 0; jj < 4; ++jj) {
                        const float t0 = pick(m0, src4[0][jj], src4[1][jj]);
                        const float t1 = pick(m0, src4[2][jj], src4[3][jj]);
                        logit[4 * kq + jj] = pick(m1, t0, t1);
                    }
                }
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
#pragma unroll
                for (int m = 0; m < MOT_MAX_EXPERTS; ++m) gate_all[m] *= inv;
                const uint32_t taken = topk_renormalise(gate_all, E, p.top_k);
                // translator usage: lanes 0..15 hold this token half's tokens
                if (p.usage && q4 == 0 && tok0 + 32 * w + 16 * th + l16 < p.n_tok) {
                    for (uint32_t t = taken; t; t &= t - 1) atomicAdd(&s_usage[__builtin_ctz(t)], 1u);
                }
                if (q4 == 0) {
#pragma unroll
                    for (int m = 0; m < MOT_MAX_EXPERTS; ++m)
                        if (m < E) Gw[m * 32 + th * 16 + l16] = gate_all[m];
                }
            }
        }
        __syncthreads();                                     // barrier B

        const float* Gw = Gs + w * (MOT_MAX_EXPERTS * 32);
        // layer-1 biases enter as the accumulators' initial values: this lane's
        // rows 4*q4 + j of row half hh are hidden 8*q4 + 4*hh + j of the chunk
        // (w1_perm), i.e. the 16 bytes at hidden 8*q4 of the chunk's b1, loaded
        // one chunk ahead so nothing waits on these loads mid-iteration.
        const int b1_lane = p.b1 ? 8 * q4 : 0;
        auto load_b1 = [&](int c, u32x4& bv) {
            typedef const __attribute__((address_space(1))) u32x4* gu128;
            bv = *(gu128)(b1u + c * b1_cstride + b1_lane);
        };
        // W1 operand of (k-step s, row half hh) sits at W1c[abase[s & 3] +
        // hh*16*CPR1 + 16*(s >> 2)]: the swizzled chunk (4s + q4) ^ l16 splits
        // into a per-lane part and compile-time offsets
        int abase[4];
#pragma unroll
        for (int b = 0; b < 4; ++b) abase[b] = l16 * C::CPR1 + 4 * (b ^ (l16 >> 2)) + (q4 ^ (l16 & 3));
        // One iteration in two phases.  Phase A: GELU of the first NEA of the
        // lane's 16 elements of chunk c-1, vector work only, while the layer-2
        // wave on this SIMD runs its MFMAs.  Phase B: a slot schedule of
        // 16x16x32 MFMAs (KS2 k-steps x 2 row halves x 2 token halves, all on
        // independent accumulators; the first k-step starts from the bias)
        // with the three-stage GELU of the other elements spread
        // over the slots (stage s of element e in slot g0(e) + s*GD); W1
        // operand reads run LOOK slots ahead.
        constexpr int NEA0 = C::L2W == 8 ? MOT_FUSED_PHASE_A12 : MOT_FUSED_PHASE_A;
        constexpr int NEA = NEA0 < 16 - C::NOFF ? NEA0 : 16 - C::NOFF;
        auto l1_iter = [&](auto l1c, auto gc, auto pc, int c, int m, const u32x4& bv,
                           const f32x4 (&sp)[2][2], u32x4& bnext, int c_next,
                           f32x4 (&s)[2][2]) {
            constexpr bool do_l1 = decltype(l1c)::value, do_gelu = decltype(gc)::value;
            // parity of c: a constant (0 or 1), which makes the LDS stage
            // offsets immediates, or -1 for the parity of the run-time c
            constexpr int P0 = decltype(pc)::value;
            const int P = P0 >= 0 ? P0 : (c & 1);
            constexpr int NEAx = C::SPLIT ? 16 : NEA;
            constexpr int NM = 4 * KS2, LOOK = 4, GD = 3, NEB = 16 - C::NOFF - NEAx;
            static_assert(NEB >= 0, "phase split");
            const u32x4* W1c = W1s + P * C::W1_CH;
            u32x4* Hw = Hs + (P ^ 1) * C::H_CH + w * 128;
            // gates of the two token halves; the GELU stages take 1/g, kept
            // finite: for a zero gate (a translator outside the Top-K) it is
            // FLT_MAX, and the element's value is then 0, or below 1e-36 where
            // e underflows (x above ~5)
            const float gv0 = Gw[m * 32 + l16], gv1 = Gw[m * 32 + 16 + l16];
            const float cg0 = fminf(__builtin_amdgcn_rcpf(gv0), 3.4028235e38f),
                        cg1 = fminf(__builtin_amdgcn_rcpf(gv1), 3.4028235e38f);
            if constexpr (do_l1) load_b1(c_next, bnext);
            u32x4 a1[KS2][2];
            float h[2][2][4], gx[16], gt[16], gq[16];
            // A operand of (k-step s, row half hh), first used in slot 4s + 2hh
            auto read_a = [&](auto kc) {
                constexpr int k = decltype(kc)::value;
                if constexpr (k < NM && (k % 2) == 0) {
                    constexpr int s = k / 4, hh = (k / 2) % 2;
                    a1[s][hh] = W1c[abase[s & 3] + hh * 16 * C::CPR1 + 16 * (s >> 2)];
                }
            };
            auto gelu_elem = [&](auto ec, auto stc) {
                constexpr int e = decltype(ec)::value, st = decltype(stc)::value;
                constexpr int hh = e / 8, th = (e / 4) % 2, jj = e % 4;
                if constexpr (ACT == MOT_ACT_GELU) {
                    if constexpr (st == 0) {
                        gx[e] = sp[hh][th][jj];
                        gelu_stage1(gx[e], gt[e]);
                    } else if constexpr (st == 1) {
                        gelu_stage2_gated(gt[e], th ? cg1 : cg0, gq[e]);
                    } else {
                        h[hh][th][jj] = gx[e] * gq[e];
                    }
                } else if constexpr (st == 0) {
                    h[hh][th][jj] = (th ? gv1 : gv0) * sp[hh][th][jj];
                }
            };
            // bias of rows 4*q4 + j of row half hh (zero without a bias)
            f32x4 binit[2];
#pragma unroll
            for (int hh = 0; hh < 2; ++hh) {
                const uint32_t w0 = bv[2 * hh], w1 = bv[2 * hh + 1];
                binit[hh] = f32x4{bf16_lo(w0), bf16_hi(w0), bf16_lo(w1), bf16_hi(w1)};
            }
            // the GELU results of chunk c-1 into this wave's hidden tile
            auto write_h = [&]() {
                // token th*16 + l16: hidden 8*q4 .. 8*q4+3 from row half 0 and
                // 8*q4+4 .. 8*q4+7 from row half 1: one 16-byte fragment unit
                // (the row-half-1 part of token halves >= TH_OFF comes from wave 3)
                constexpr int TH_OFF = 2 - C::NOFF / 4;
#pragma unroll
                for (int th = 0; th < 2; ++th) {
                    u32x4* dst = &Hw[(q4 >> 1) * 64 + (q4 & 1) * 32 + th * 16 + l16];
                    if (th >= TH_OFF) {
                        const u32x2 v = {pack_bf16x2(h[0][th][0], h[0][th][1]), pack_bf16x2(h[0][th][2], h[0][th][3])};
                        *reinterpret_cast<u32x2*>(dst) = v;
                    } else {
                        u32x4 v;
                        v[0] = pack_bf16x2(h[0][th][0], h[0][th][1]);
                        v[1] = pack_bf16x2(h[0][th][2], h[0][th][3]);
                        v[2] = pack_bf16x2(h[1][th][0], h[1][th][1]);
                        v[3] = pack_bf16x2(h[1][th][2], h[1][th][3]);
                        *dst = v;
                    }
                }
            };
            if constexpr (do_l1) static_for<0, LOOK>([&](auto kc) { read_a(kc); });
            if constexpr (do_gelu && C::SPLIT) {
                // all 16 elements, four at a time through the three stages
                static_for<0, 4>([&](auto gc4) {
                    constexpr int g4 = decltype(gc4)::value;
                    static_for<0, 3>([&](auto stc) {
                        static_for<0, 4>([&](auto ec) {
                            gelu_elem(std::integral_constant<int, 4 * g4 + decltype(ec)::value>{}, stc);
                        });
                    });
                });
                write_h();
            } else if constexpr (do_gelu && !MOT_FUSED_A_LAST) {
                static_for<0, 3>([&](auto stc) {
                    static_for<0, NEA>([&](auto ec) { gelu_elem(ec, stc); });
                });
            }
            mid_barrier();
            __builtin_amdgcn_sched_barrier(0);
            if constexpr (MOT_FUSED_L1_PRIO > 0 && do_l1) __builtin_amdgcn_s_setprio(MOT_FUSED_L1_PRIO);
            static_for<0, NM>([&](auto kc) {
                constexpr int k = decltype(kc)::value;
                if constexpr (do_l1) {
                    read_a(std::integral_constant<int, k + LOOK>{});
                    constexpr int st = k / 4, hh = (k / 2) % 2, th = k % 2;
                    s[hh][th] = mfma_16x16x32(a1[st][hh], zf[th][st], st == 0 ? binit[hh] : s[hh][th]);
                }
                if constexpr (do_gelu && NEB > 0) {
                    static_for<0, NEB>([&](auto ec) {
                        constexpr int eb = decltype(ec)::value, e = NEA + eb;
                        constexpr int hh = e / 8, th = (e / 4) % 2, jj = e % 4;
                        constexpr int g0 = NEB > 1 ? (eb * (NM - 2 * GD - 1)) / (NEB - 1) : 0;
                        if constexpr (ACT == MOT_ACT_GELU) {
                            if constexpr (k == g0) {
                                float v = sp[hh][th][jj];
                                asm volatile("" : "+v"(v));
                                gx[e] = v;
                                gelu_stage1(v, gt[e]);
                                asm volatile("" : "+v"(gt[e]));
                            } else if constexpr (k == g0 + GD) {
                                gelu_stage2_gated(gt[e], th ? cg1 : cg0, gq[e]);
                                asm volatile("" : "+v"(gq[e]));
                            } else if constexpr (k == g0 + 2 * GD) {
                                h[hh][th][jj] = gx[e] * gq[e];
                            }
                        } else if constexpr (k == g0) {
                            float v = sp[hh][th][jj];
                            asm volatile("" : "+v"(v));
                            h[hh][th][jj] = (th ? gv1 : gv0) * v;
                        }
                    });
                }
                __builtin_amdgcn_sched_barrier(0);
            });
            if constexpr (MOT_FUSED_L1_PRIO > 0 && do_l1) {
                __builtin_amdgcn_sched_barrier(0);
                __builtin_amdgcn_s_setprio(0);
            }
            if constexpr (do_gelu && MOT_FUSED_A_LAST && !C::SPLIT) {
                static_for<0, 3>([&](auto stc) {
                    static_for<0, NEA>([&](auto ec) { gelu_elem(ec, stc); });
                });
            }
            if constexpr (do_gelu && !C::SPLIT) write_h();
            if constexpr (do_l1 && C::NOFF > 0) {
                // hand row half 1 of the offloaded token halves of chunk c to wave 3
                constexpr int TH_OFF = 2 - C::NOFF / 4;
#pragma unroll
                for (int th = TH_OFF; th < 2; ++th)
                    Xs[P * C::X_CH + (w * (C::NOFF / 4) + th - TH_OFF) * 64 + lane] =
                        __builtin_bit_cast(u32x4, s[1][th]);
            }
        };

        int m1 = 0, kk1 = 0;
        u32x4 bcur, bnext = {0u, 0u, 0u, 0u};
        load_b1(0, bcur);
        f32x4 s_prev[2][2], s_new[2][2];
        auto advance = [&]() {          // (m1, kk1) -> the next chunk
            kk1 += 32;
            const bool wrap = kk1 == hidden;
            kk1 = wrap ? 0 : kk1;
            m1 = wrap ? m1 + 1 : m1;
        };
        auto rotate = [&]() {
#pragma unroll
            for (int a = 0; a < 2; ++a)
#pragma unroll
                for (int b = 0; b < 2; ++b) s_prev[a][b] = s_new[a][b];
            bcur = bnext;
        };
        const std::integral_constant<bool, true> yes{};
        const std::integral_constant<bool, false> no{};
        // c = 0: layer 1 only; 1 .. nch-1: layer 1 and GELU; nch: GELU only;
        // nch+1: barrier only (layer 2 of the last chunk runs on other waves).
        // nch is even (hidden % 64 == 0): after c = 0 the odd/even pairs
        // alternate the bias and accumulator registers, and c = nch - 1 (odd)
        // and c = nch close the walk.
        const std::integral_constant<int, 0> even{};
        const std::integral_constant<int, 1> odd{};
        if constexpr (C::L2W == 8) {
            // 12-wave form: one loop body, stage offsets from the parity of c
            // (the odd/even pairs below measured 1.3 % slower at 256 -> 512)
            sync_stage();
            l1_iter(yes, no, even, 0, m1, bcur, s_prev, bnext, 1, s_new);
            rotate();
            for (int c = 1; c < nch; ++c) {
                sync_stage();
                l1_iter(yes, yes, std::integral_constant<int, -1>{}, c, m1, bcur, s_prev, bnext,
                        c + 1 < nch ? c + 1 : nch - 1, s_new);
                rotate();
                advance();
            }
            sync_stage();
            l1_iter(no, yes, even, nch, m1, bcur, s_prev, bnext, nch - 1, s_new);
            sync_stage();
        } else {
            // 8-wave forms: odd/even pairs with the stage offsets as immediates
            // (2 % faster at 512 -> 512 than the single body)
            sync_stage();
            l1_iter(yes, no, even, 0, m1, bcur, s_prev, bnext, 1, s_new);
            rotate();
            int c = 1;
            for (; c + 1 < nch; c += 2) {
                sync_stage();
                l1_iter(yes, yes, odd, c, m1, bcur, s_prev, bnext, c + 1, s_new);
                advance();
                sync_stage();
                l1_iter(yes, yes, even, c + 1, m1, bnext, s_new, bcur, c + 2 < nch ? c + 2 : nch - 1, s_prev);
                advance();
            }
            sync_stage();
            l1_iter(yes, yes, odd, c, m1, bcur, s_prev, bnext, nch - 1, s_new);
            advance();
            sync_stage();
            l1_iter(no, yes, even, nch, m1, bnext, s_new, bcur, nch - 1, s_prev);
            sync_stage();
        }
        mid_barrier();   // the layer-2 waves' last iteration
    } else if (is_l2) {
        // ---------------------------------------------------------- layer 2
        uint32_t ow1[NV1];
#pragma unroll
        for (int v = 0; v < NV1; ++v) ow1[v] = w1_lane(v);
#pragma unroll
        for (int r = 0; r < W1_RL; ++r) load_w1_round(0, 0, r, ow1[r % NV1]);
        __syncthreads();                                     // barrier A
        __syncthreads();                                     // barrier B
        // the tile's translator usage, counted by the layer-1 waves' router
        if (!ROUTED && p.usage && q2 == 0 && lane < E && s_usage[lane])
            atomicAdd(p.usage + unit * E + lane, s_usage[lane]);
        // accumulators seeded with sum_m g_m b2_m[o] on MFMA: A = gates of a
        // token block (k = translator), B = b2 (k = translator); gates split
        // into bf16 high + residual parts keep ~16 mantissa bits.
        // acc[tb][nb]: column o = q2*OUTW + nb*32 + l32, rows = tokens
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
                const int o = q2 * C::OUTW + nb * 32 + l32;
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

        // One iteration as a slot schedule over this wave's MFMAs, ordered
        // (k-slice, token block, output block): a k-slice's W2 fragments stay
        // live while each H fragment is used by consecutive MFMAs, which keeps
        // the operand registers few enough for the 128 accumulators of
        // TB = 4, NBW = 2 to fit 168 VGPRs without spilling; H and W2 operand
        // reads run LOOK slots ahead, and the weight loads are spread over
        // the slots.
        auto l2_iter = [&](auto l2c, auto w1c, auto w2c, int c, int c_w1, int m_w2, int kk_w2, int st_w2) {
            constexpr bool do_l2 = decltype(l2c)::value, do_w1 = decltype(w1c)::value,
                           do_w2 = decltype(w2c)::value;
            constexpr int NM = 2 * TB * C::NBW, LOOK = MOT_FUSED_L2_LOOK;
            constexpr int NV = W1_RL + W2_RL;
            const u32x4* Hc = Hs + (c & 1) * C::H_CH;          // chunk c-2 shares c's parity
            const u32x4* W2c = W2s + ((c + C::NW2 - 2) % C::NW2) * C::W2_CH;
            u32x4 hA[2][TB], bW[2][C::NBW];
            auto issue_reads = [&](auto kc) {
                constexpr int k = decltype(kc)::value;
                if constexpr (k < NM) {
                    constexpr int ks = k / (TB * C::NBW), nb = k % C::NBW, tb = (k / C::NBW) % TB;
                    if constexpr (nb == 0) hA[ks][tb] = Hc[tb * 128 + ks * 64 + g * 32 + l32];
                    if constexpr (tb == 0) {
                        const int o = q2 * C::OUTW + nb * 32 + l32;
                        bW[ks][nb] = W2c[o * 4 + ((2 * ks + g) ^ ((o >> 2) & 3))];
                    }
                }
            };
            if constexpr (do_l2) static_for<0, LOOK>([&](auto kc) { issue_reads(kc); });
            static_for<0, NM>([&](auto kc) {
                constexpr int k = decltype(kc)::value;
                if constexpr (NV > 0) {
                    static_for<0, NV>([&](auto rc) {
                        constexpr int r = decltype(rc)::value;
                        if constexpr ((MOT_FUSED_LOAD_SPREAD ? (r * NM) / NV : r) == k) {
                            if constexpr (r < W1_RL) {
                                if constexpr (do_w1) load_w1_round(c_w1, (c + 1) & 1, r, ow1[r % NV1]);
                            } else {
                                if constexpr (do_w2) load_w2_round(m_w2, kk_w2, st_w2, r - W1_RL);
                            }
                        }
                    });
                }
                if constexpr (do_l2) {
                    issue_reads(std::integral_constant<int, k + LOOK>{});
                    constexpr int ks = k / (TB * C::NBW), nb = k % C::NBW, tb = (k / C::NBW) % TB;
                    acc[tb][nb] = mfma_32x32x16(hA[ks][tb], bW[ks][nb], acc[tb][nb]);
                }
                __builtin_amdgcn_sched_barrier(0);
            });
            mid_barrier();
        };

        // (m1, kk1): translator and column offset of W2 chunk kw, the one
        // fetched in iteration c: kw = c with three W2 stages, else c - 1
        int m1 = 0, kk1 = 0;
        const std::integral_constant<bool, true> T{};
        const std::integral_constant<bool, false> F{};
        auto advance = [&]() {
            kk1 += 32;
            const bool wrap = kk1 == hidden;
            kk1 = wrap ? 0 : kk1;
            m1 = wrap ? m1 + 1 : m1;
        };
        // Iteration c runs layer 2 of chunk c-2 (c >= 2), fetches W1 of chunk
        // c+1 (c+1 < nch) and W2 of chunk kw (0 <= kw < nch).  The pipeline
        // fill and drain iterations are peeled with their stage flags fixed at
        // compile time (nch >= 2); the steady state runs every stage.
        constexpr bool W2_AT_C = C::NW2 == 3;   // kw = c, else kw = c - 1
        const std::integral_constant<bool, W2_AT_C> W2_FIRST{};
        const std::integral_constant<bool, !W2_AT_C> W2_LAST{};
        auto w2_stage = [&](int c) { return (c - (W2_AT_C ? 0 : 1) + C::NW2) % C::NW2; };
        sync_stage();                                                   // c = 0
        l2_iter(F, T, W2_FIRST, 0, 1, m1, kk1, w2_stage(0));
        if (W2_AT_C) advance();
        sync_stage();                                                   // c = 1
        if (nch > 2) l2_iter(F, T, T, 1, 2, m1, kk1, w2_stage(1));
        else l2_iter(F, F, T, 1, 2, m1, kk1, w2_stage(1));
        advance();
        for (int c = 2; c + 1 < nch; ++c) {                             // steady state
            // after a steady iteration, whose last loads are W2 rounds of a
            // chunk used two iterations later, those stay in flight
            if (C::NW2 == 3 && c > 2) sync_keep(std::integral_constant<int, C::NW2 == 3 ? W2_RL : 0>{});
            else sync_stage();
            l2_iter(T, T, T, c, c + 1, m1, kk1, w2_stage(c));
            advance();
        }
        if (nch >= 3) {                                                 // c = nch - 1
            sync_stage();
            l2_iter(T, F, T, nch - 1, nch, m1, kk1, w2_stage(nch - 1));
            advance();
        }
        sync_stage();                                                   // c = nch
        l2_iter(T, F, W2_LAST, nch, nch + 1, m1, kk1, w2_stage(nch));
        sync_stage();                                                   // c = nch + 1
        l2_iter(T, F, F, nch + 1, nch + 2, m1, kk1, w2_stage(nch + 1));

        // epilogue: bf16 round and store in the target layout
        {
        uint16_t* dst = reinterpret_cast<uint16_t*>(p.dst[x]) + (size_t)j * p.n_tok * D_OUT;
#pragma unroll
        for (int tb = 0; tb < TB; ++tb) {
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int r = tb * 32 + 8 * (e >> 2) + 4 * g + (e & 3);   // row of the tile
                int tok;
                if constexpr (ROUTED) {
                    if (r >= tile.z) continue;
                    const size_t NK = (size_t)p.n_tok * p.top_k;
                    if (p.top_k > 1) {
                        // fp32 row of assignment tile.y + r; the combine sums a token's rows
                        float* prow = p.rt.part + (blockIdx.y * NK + tile.y + r) * D_OUT;
#pragma unroll
                        for (int nb = 0; nb < C::NBW; ++nb)
                            prow[q2 * C::OUTW + nb * 32 + l32] = acc[tb][nb][e];
                        continue;
                    }
                    tok = p.rt.list[(size_t)unit_gslot(code) * NK + tile.y + r];
                } else {
                    tok = tok0 + r;
                    if (tok >= p.n_tok) continue;
                }
                const int b = tok / p.T, t = tok % p.T;
#pragma unroll
                for (int nb = 0; nb < C::NBW; ++nb) {
                    const int o = q2 * C::OUTW + nb * 32 + l32;
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
    } else {
        // wave 3 when TB = 3: no token block; it helps stage the router
        // weights, then (NOFF > 0) evaluates the GELU of the row-half-1
        // elements of the offloaded token halves of every layer-1 wave:
        // iteration c reads chunk c-1's fp32 values from the hand-over stage
        // and writes the upper 8 bytes of those hidden-tile units
        if constexpr (!ROUTED) stage_router_weights();
        __syncthreads();
        __syncthreads();
        const int l16 = lane & 15, q4 = lane >> 4;
        constexpr int NX = C::NOFF / 4, TH_OFF = 2 - NX;
        int m3 = 0, kk3 = 0;
        for (int c = 0; c <= nch + 1; ++c) {
            sync_stage();
            if (C::NOFF > 0 && c >= 1 && c <= nch) {
                const u32x4* Xc = Xs + ((c - 1) & 1) * C::X_CH;
                u32x4* Hc = Hs + ((c - 1) & 1) * C::H_CH;
                f32x4 sv[TB][NX];
                float hg[TB][NX];
#pragma unroll
                for (int wb = 0; wb < TB; ++wb)
#pragma unroll
                    for (int f = 0; f < NX; ++f) {
                        sv[wb][f] = __builtin_bit_cast(f32x4, Xc[(wb * NX + f) * 64 + lane]);
                        hg[wb][f] = 0.5f * Gs[wb * (MOT_MAX_EXPERTS * 32) + m3 * 32 + (TH_OFF + f) * 16 + l16];
                    }
#pragma unroll
                for (int wb = 0; wb < TB; ++wb)
#pragma unroll
                    for (int f = 0; f < NX; ++f) {
                        float hv[4];
#pragma unroll
                        for (int jj = 0; jj < 4; ++jj)
                            hv[jj] = ACT == MOT_ACT_GELU ? gelu_half_scaled(sv[wb][f][jj], hg[wb][f])
                                                         : 2.0f * hg[wb][f] * sv[wb][f][jj];
                        const u32x2 v = {pack_bf16x2(hv[0], hv[1]), pack_bf16x2(hv[2], hv[3])};
                        u32x4* unit16 = &Hc[wb * 128 + (q4 >> 1) * 64 + (q4 & 1) * 32 + (TH_OFF + f) * 16 + l16];
                        reinterpret_cast<u32x2*>(unit16)[1] = v;
                    }
                kk3 += 32;
                const bool wrap = kk3 == hidden;
                kk3 = wrap ? 0 : kk3;
                m3 = wrap ? m3 + 1 : m3;
            }
        }
    }
}

template <int D_IN, int D_OUT, bool ROUTED>
hipError_t launch_t(const Problem& p, const UnitTab& ut, hipStream_t stream) {
    using C = Cfg<D_IN, D_OUT>;
    dim3 grid(ROUTED ? p.rt.max_tiles : (p.n_tok + C::BM - 1) / C::BM, ut.n);
    if (p.act == MOT_ACT_GELU)
        hipLaunchKernelGGL((k_bf16_fused<D_IN, D_OUT, MOT_ACT_GELU, ROUTED>), grid, dim3(64 * C::NW), 0, stream, p,
                           ut);
    else
        hipLaunchKernelGGL((k_bf16_fused<D_IN, D_OUT, MOT_ACT_IDENTITY, ROUTED>), grid, dim3(64 * C::NW), 0, stream,
                           p, ut);
    return hipGetLastError();
}

}  // namespace

}  // namespace mot
