// Two-GEMM bf16 translation path, large-tile form: the same two products as
// k_bf16_unfused.hip (translator layer 1 with its gated GELU epilogue, then
// layer 2 whose K axis runs over every expert's hidden units so the gated sum
// of the mixture, paper Sec. 3 Eq. mot_definition, is reduced inside the
// accumulator), on 256 x 256 output tiles.
//
//   gemm1: Hs[u][t][m*hidden+k] = bf16( g[u][t][m] * GELU((W1_m z_t + b1_m)[k]) )
//          MFMA A = W1 rows (hidden), B = source rows (tokens)
//   gemm2: dst[j][t][o] = bf16( sum_kk W2cat[o][kk] Hs[u][t][kk] + sum_m g_m b2_m[o] )
//          MFMA A = W2cat rows (outputs), B = hidden rows (tokens)
//
// One 256-thread workgroup per CU (128 KB of LDS): four waves in a 2 x 2
// grid, 128 x 128 outputs per wave = 4 x 4 blocks of v_mfma_f32_32x32x16_bf16
// (256 accumulators per lane, held in the AGPR half of the register file).
// Per 32-wide K slice a tile moves 32 KB into LDS for 2 * 256 * 256 * 32
// flops (128 flop/B, twice the 128 x 128 form's).
//
// Operands go global -> LDS directly (buffer_load_dwordx4 ... lds, 16 bytes
// per lane, through a buffer descriptor per operand; the MUBUF form rather
// than global_load_lds, whose FLAT encoding makes the compiler's wait
// insertion treat every later LDS read as out of order and wait for all of
// them): a wave's load fills 1 KB of LDS = 16 rows of four 16-byte chunks,
// and the lane order within those rows is chosen so that row r stores
// logical chunk c at physical chunk c ^ ((r >> 2) & 3).  Sixteen lanes of a
// fragment read (16 consecutive rows, one logical chunk) then hit 16
// distinct 16-byte bank groups.
//
// Five LDS stages (all 160 KB): the loads of slice k+4 are trickled over the
// MFMAs of slice k, one 1 KB load after every four MFMAs.  A wave that issues
// several loads back to back cannot issue its next MFMA until the memory
// pipeline has accepted them, so loads bunched at the start of a slice stall
// the matrix core although they complete asynchronously; one load per four
// MFMAs (32 B per clock per CU, about half of what the path sustains) does
// not.  Every load is a per-lane offset computed once plus the slice's
// uniform offset in a scalar register, so the loop does almost no vector
// address arithmetic.  One barrier per slice.
//
// Bias terms enter through the accumulators' initial values: gemm1 starts
// from b1 (each lane's rows are 4 consecutive hidden units), gemm2 from two
// extra 32x32x16 products B2 . G with the gates split into a bf16 high part
// and a bf16 residual (K = 16 covers E <= 16 experts).
#include "mot_device.h"
#include "mot_internal.h"
#include "../../include/mot.h"

namespace mot {

namespace {

constexpr int kTile = 256;
constexpr int kGroup = 32;              // B tiles per dispatch group

// LDS geometry of a 32-wide K slice: rows of four 16-byte chunks, a wave's
// 1 KB load fills 16 rows, kNI loads per operand and wave, kNST stages of
// kStage slots (A rows then B rows).  Logical chunk c of row r sits at
// c ^ swz(r): 16 consecutive rows of one logical chunk fill 16 distinct
// 16-byte bank groups.
constexpr int kBK = 32, kCPR = kBK / 8, kRPI = 64 / kCPR, kNI = kTile / kRPI / 4;
constexpr int kNST = 5, kStage = 2 * kTile * kCPR;
static_assert(kNST * kStage * 16 == 160 * 1024, "160 KB of LDS");
__device__ __forceinline__ int swz(int r) { return (r >> 2) & 3; }

typedef __attribute__((address_space(3))) void lds_void;

typedef __amdgpu_buffer_rsrc_t rsrc_t;

// Raw buffer over `bytes` bytes at `base` (reads past the end return 0).
__device__ __forceinline__ rsrc_t make_rsrc(const void* base, size_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0,
                                             (int)(bytes < 0xFFFFFFFFu ? bytes : 0xFFFFFFFFu), 0x00020000);
}

// Dispatch order: groups of kGroup consecutive B tiles (tokens), A tiles
// outer within a group.  Workgroups go round-robin to the 8 XCDs, so an XCD's
// 32 resident workgroups cover 4 token tiles x 8 A tiles of one group: 12
// distinct operand tiles per K slice instead of up to 64.
__device__ __forceinline__ void tile_of(int lin, int nA, int nB, int& a_tile, int& b_tile) {
    const int grp = lin / (kGroup * nA);
    const int gsz = min(kGroup, nB - kGroup * grp);
    const int r = lin - grp * kGroup * nA;
    b_tile = kGroup * grp + r % gsz;
    a_tile = r / gsz;
}

__device__ __forceinline__ uint32_t src_row_bytes(const Problem& p, int tok) {
    if (p.src_layout == MOT_LAYOUT_BTHD) return (uint32_t)tok * p.d_in * 2;
    const int b = tok / p.T, t = tok % p.T;
    return ((uint32_t)b * p.H_src * p.T + t) * p.D_src * 2;
}
__device__ __forceinline__ uint32_t src_k_bytes(const Problem& p, int k) {
    if (p.src_layout == MOT_LAYOUT_BTHD) return (uint32_t)k * 2;
    return ((uint32_t)(k / p.D_src) * p.T * p.D_src + k % p.D_src) * 2;
}

// s_waitcnt immediate (gfx9 encoding): vector-memory count n, LDS/scalar
// count 0, export count left at its maximum
constexpr int waitcnt_vm_lgkm0(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4); }

// The K loop shared by both products.  voA / voB: this lane's byte offsets
// into the operands' buffers for its rows of each of its kNI loads per
// operand (rows kRPI*J + lane/kCPR of the tile, J = wave*kNI + q), including
// the column offset of its chunk wherever that offset is the same in every
// slice; slice(kt, sa, sb, vb) gives slice kt's uniform byte offsets sa, sb
// and a per-lane term vb added to voB (zero where B's column offset is
// uniform).  acc holds the initial values on entry.
//
// Register double buffering: the fragments of k-step 1 are read while the
// 16 MFMAs of k-step 0 run; the slice's barrier sits before the MFMAs of
// k-step 1 (whose fragments are already in registers), and the next slice's
// first fragments are read right after it, so the matrix core has queued
// work across the barrier.  Slice indices past the end are clamped (a
// redundant reload into a stage that is no longer read), so every barrier
// waits for the same count.
template <class Slice>
__device__ __forceinline__ void k_loop(u32x4* lds, rsrc_t bufA, rsrc_t bufB, const uint32_t (&voA)[kNI],
                                       const uint32_t (&voB)[kNI], int nk, Slice slice, f32x16 (&acc)[4][4]) {
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 1, wn = wave & 1, g = lane >> 5, l32 = lane & 31;
    const int sw = swz(l32);
    u32x4* const wbase = lds + wave * kNI * 64;
    // load l of the 2 kNI per wave and slice: q-pair l / 2, operand A (even) or B (odd)
    auto ld1 = [&](int st, uint32_t sa, uint32_t sb, uint32_t vb, int l) {
        const int q = l >> 1;
        u32x4* dst = wbase + st * kStage + ((l & 1) ? kTile * kCPR : 0) + q * 64;
        if (l & 1) __builtin_amdgcn_raw_ptr_buffer_load_lds(bufB, (lds_void*)dst, 16, voB[q] + vb, sb, 0, 0);
        else __builtin_amdgcn_raw_ptr_buffer_load_lds(bufA, (lds_void*)dst, 16, voA[q], sa, 0, 0);
    };
    // fragments of k-step s of stage st: rows wm*128 + i*32 + l32 (A) and
    // wn*128 + i*32 + l32 (B), logical chunk 2s + g
    auto read = [&](int st, int s, u32x4 (&a)[4], u32x4 (&b)[4]) {
        const u32x4* la = lds + st * kStage + (wm * 128 + l32) * kCPR;
        const u32x4* lb = lds + st * kStage + kTile * kCPR + (wn * 128 + l32) * kCPR;
        const int c = (2 * s + g) ^ sw;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            a[i] = la[i * 32 * kCPR + c];
            b[i] = lb[i * 32 * kCPR + c];
        }
    };
    // the 16 MFMAs of a k-step with loads 4h .. 4h+3 of slice kt+4, one after
    // every four (sched_barrier fences keep that order, and keep each read
    // group ahead of the MFMAs that precede its use)
    auto mma_ld = [&](const u32x4 (&a)[4], const u32x4 (&b)[4], int st, uint32_t sa, uint32_t sb, uint32_t vb,
                      int h) {
#pragma unroll
        for (int bm = 0; bm < 4; ++bm) {
#pragma unroll
            for (int bn = 0; bn < 4; ++bn) acc[bm][bn] = mfma_32x32x16(a[bm], b[bn], acc[bm][bn]);
            ld1(st, sa, sb, vb, 4 * h + bm);
            __builtin_amdgcn_sched_barrier(0);
        }
    };
    // workgroup barrier after an explicit wait: __syncthreads() would add its
    // own fence, which waits for every load in flight (vmcnt(0)) and so for
    // the later slices' loads too.  The waits are s_waitcnt instructions the
    // compiler sees (it then adds no LDS waits of its own after the barrier).
    auto barrier = [&]() {
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
    };
    // slices 0..3 in flight, wait for slice 0
#pragma unroll
    for (int s0 = 0; s0 < kNST - 1; ++s0) {
        uint32_t sa, sb, vb;
        slice(s0 < nk ? s0 : nk - 1, sa, sb, vb);
#pragma unroll
        for (int l = 0; l < 2 * kNI; ++l) ld1(s0, sa, sb, vb, l);
    }
    __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0((kNST - 2) * 2 * kNI));
    barrier();
    u32x4 a0[4], b0[4], a1[4], b1[4];
    read(0, 0, a0, b0);
    int st = 0, stl = kNST - 1;   // stages of slices kt and kt + 4
    for (int kt = 0; kt < nk; ++kt) {
        const int kl = kt + kNST - 1;
        uint32_t sa, sb, vb;
        slice(kl < nk ? kl : nk - 1, sa, sb, vb);
        read(st, 1, a1, b1);
        __builtin_amdgcn_sched_barrier(0);
        mma_ld(a0, b0, stl, sa, sb, vb, 0);
        // every wave's reads of stage st are in registers and slice kt+1 has
        // landed: slices kt+2, kt+3 and the four loads of slice kt+4 issued
        // above may stay in flight
        __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0((kNST - 3) * 2 * kNI + kNI));
        barrier();
        const int st1 = st + 1 == kNST ? 0 : st + 1;
        if (kt + 1 < nk) read(st1, 0, a0, b0);
        __builtin_amdgcn_sched_barrier(0);
        mma_ld(a1, b1, stl, sa, sb, vb, 1);
        __builtin_amdgcn_sched_barrier(0);
        st = st1;
        stl = stl + 1 == kNST ? 0 : stl + 1;
    }
    // the clamped reloads of the last slices are still in flight
    __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0(0));
}

// Accumulators of block (bm, bn) start at the bias products of a 32-row
// block of A rows and a 32-column block of B columns: D[r][t] = sum_m
// bias_m[r] gate_m[t] over m < nm <= 16, as two 32x32x16 MFMAs with the gates
// split into a bf16 high part and a bf16 residual.  bias(m, r) and gate(m, t)
// return the values for this lane's row r (m = 8*g .. 8*g+7) and column t.
template <class BiasF, class GateF>
__device__ __forceinline__ void seed_bias(f32x16 (&acc)[4][4], int nm, BiasF bias, GateF gate, int row0,
                                          int col0) {
    const int lane = threadIdx.x & 63, g = lane >> 5, l32 = lane & 31;
    u32x4 ghi[4], glo[4];
#pragma unroll
    for (int bn = 0; bn < 4; ++bn) {
        const int t = col0 + bn * 32 + l32;
        float gv[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) gv[e] = 8 * g + e < nm ? gate(8 * g + e, t) : 0.f;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const uint32_t h = pack_bf16x2(gv[2 * e], gv[2 * e + 1]);
            ghi[bn][e] = h;
            glo[bn][e] = pack_bf16x2(gv[2 * e] - bf16_lo(h), gv[2 * e + 1] - bf16_hi(h));
        }
    }
#pragma unroll
    for (int bm = 0; bm < 4; ++bm) {
        const int r = row0 + bm * 32 + l32;
        u32x4 bb;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int m = 8 * g + 2 * e;
            const uint32_t lo = m < nm ? bias(m, r) : 0u;
            const uint32_t hi = m + 1 < nm ? bias(m + 1, r) : 0u;
            bb[e] = lo | (hi << 16);
        }
#pragma unroll
        for (int bn = 0; bn < 4; ++bn) {
            acc[bm][bn] = mfma_32x32x16(bb, ghi[bn], acc[bm][bn]);
            acc[bm][bn] = mfma_32x32x16(bb, glo[bn], acc[bm][bn]);
        }
    }
}

// Rows of the routed path's hidden buffer per unit: assignments rounded up to
// a 32-row fragment group.
__device__ __forceinline__ size_t routed_hidden_elems(const Problem& p) {
    return ((size_t)p.n_tok * p.top_k + 31) / 32 * 32 * p.hidden;
}

// ---------------------------------------------------------------------------
// gemm1.  grid: x = (hidden tiles) x (token tiles) in dispatch order, z = unit
// in the launch.  ROUTED: the token tiles are the routing plan's tiles (up to
// 256 assignments of one translator m); the B rows are gathered by token
// index, A is W1_m, and the hidden rows are stored in assignment order with
// the assignment's gate.
// ---------------------------------------------------------------------------
template <bool ROUTED>
__global__ __launch_bounds__(256, 1) void k_bf16_gemm1_256(Problem p, UnitTab ut) {
    __shared__ u32x4 lds[kNST * kStage];
    const uint32_t code = ut.code[blockIdx.z];
    const int j = unit_j(code), x = unit_x(code), i = unit_i(code), gs = unit_gslot(code);
    // A rows: E*hidden (dense) or the hidden units of one translator (routed)
    const int EH = ROUTED ? p.hidden : p.E * p.hidden;
    const int nA = (EH + kTile - 1) / kTile;
    const int nB = ROUTED ? p.rt.max_tiles : (p.n_tok + kTile - 1) / kTile;
    int at, bt;
    tile_of(blockIdx.x, nA, nB, at, bt);
    int m = 0, first = 0, rows = 0;
    const int32_t* list = nullptr;
    if constexpr (ROUTED) {
        if (bt >= p.rt.ntiles[gs]) return;
        const int4 tl = p.rt.tiles[(size_t)gs * p.rt.max_tiles + bt];
        m = tl.x; first = tl.y; rows = tl.z;
        list = p.rt.list + (size_t)gs * p.n_tok * p.top_k;
    }
    const int hid0 = at * kTile, tok0 = bt * kTile;
    const size_t unit = (size_t)j * p.streams + x;
    const size_t wsel = ROUTED ? unit * p.E + m : unit;   // W1 block: [EH][d_in]
    const rsrc_t bufA = make_rsrc(reinterpret_cast<const char*>(p.w1) + wsel * EH * p.d_in * 2,
                                  (size_t)EH * p.d_in * 2);
    const rsrc_t bufB = make_rsrc(reinterpret_cast<const char*>(p.src[x]) + (size_t)i * p.n_tok * p.d_in * 2,
                                  (size_t)p.n_tok * p.d_in * 2);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int L = lane / kCPR;
    // this lane's logical chunk: the same in each of its loads (their rows
    // differ by multiples of 16, which swz ignores)
    const int c = (lane % kCPR) ^ swz(L);

    uint32_t voA[kNI], voB[kNI];
#pragma unroll
    for (int q = 0; q < kNI; ++q) {
        const int r = kRPI * (wave * kNI + q) + L;
        voA[q] = (uint32_t)min(hid0 + r, EH - 1) * p.d_in * 2 + 16 * c;
        const int tok = ROUTED ? list[first + min(r, rows - 1)] : min(tok0 + r, p.n_tok - 1);
        voB[q] = src_row_bytes(p, tok);
    }
    // W1 columns are uniform; a source row's column offset depends on the
    // layout (BHTD: head-major), so it is a per-lane term, once per slice
    auto slice = [&](int kt, uint32_t& sa, uint32_t& sb, uint32_t& vb) {
        sa = (uint32_t)kt * kBK * 2;
        sb = 0;
        vb = src_k_bytes(p, kt * kBK + 8 * c);
    };

    // accumulators start at b1: lane rows of block bm are hidden
    // hid0 + wm*128 + bm*32 + 8*ii + 4*g + jj
    const int wm = wave >> 1, wn = wave & 1, g = lane >> 5, l32 = lane & 31;
    const uint16_t* b1 = p.b1 ? reinterpret_cast<const uint16_t*>(p.b1) + wsel * EH : nullptr;
    f32x16 acc[4][4];
#pragma unroll
    for (int bm = 0; bm < 4; ++bm) {
        const int hb = min(hid0 + wm * 128 + bm * 32, EH - 32);
        f32x16 init;
#pragma unroll
        for (int ii = 0; ii < 4; ++ii) {
            u32x2 w = {0u, 0u};
            if (b1) w = *reinterpret_cast<const u32x2*>(b1 + hb + 8 * ii + 4 * g);
            init[4 * ii + 0] = bf16_lo(w[0]);
            init[4 * ii + 1] = bf16_hi(w[0]);
            init[4 * ii + 2] = bf16_lo(w[1]);
            init[4 * ii + 3] = bf16_hi(w[1]);
        }
#pragma unroll
        for (int bn = 0; bn < 4; ++bn) acc[bm][bn] = init;
    }

    k_loop(lds, bufA, bufB, voA, voB, p.d_in / kBK, slice, acc);

    // epilogue: GELU, * gate, round to bf16, fragment-native hidden store
    // (16-byte units of 8 hidden values of one row, [r/32][kk/8][r%32]; rows
    // are tokens, or assignments on the routed path)
    uint16_t* H = reinterpret_cast<uint16_t*>(p.hbuf) +
                  blockIdx.z * (ROUTED ? routed_hidden_elems(p) : (size_t)p.n_tok_pad * EH);
    const float* G = ROUTED ? p.rt.agate + (size_t)gs * p.n_tok * p.top_k
                            : p.gates + (size_t)gs * p.n_tok_pad * p.E;
    const int row_end = ROUTED ? first + rows : p.n_tok_pad;
#pragma unroll
    for (int bm = 0; bm < 4; ++bm) {
        const int hbase = hid0 + wm * 128 + bm * 32;
        if (hbase >= EH) continue;
        const int e = hbase / p.hidden;   // hidden % 64 == 0: one expert per 32 rows
#pragma unroll
        for (int bn = 0; bn < 4; ++bn) {
            const int tc = (ROUTED ? first : tok0) + wn * 128 + bn * 32 + l32;
            if (tc >= row_end) continue;
            const float gate = ROUTED ? G[tc] : tc < p.n_tok ? G[(size_t)tc * p.E + e] : 0.f;
            uint16_t* hrow = H + ((size_t)(tc >> 5) * (EH >> 3) + (hbase >> 3)) * 256 + (tc & 31) * 8 + 4 * g;
#pragma unroll
            for (int ii = 0; ii < 4; ++ii) {
                float v[4];
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) {
                    const float a = acc[bm][bn][4 * ii + jj];
                    v[jj] = gate * (p.act == MOT_ACT_GELU ? gelu_tanh(a) : a);
                }
                u32x2 w = {pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
                *reinterpret_cast<u32x2*>(hrow + (size_t)ii * 256) = w;
            }
        }
    }
}

// ---------------------------------------------------------------------------
// gemm2.  grid: x = (output tiles) x (token tiles) in dispatch order, z = unit
// in the launch.  ROUTED: the token tiles are the plan's tiles; A is W2_m
// (K = hidden), the B rows are the tile's assignments (contiguous in the
// hidden buffer), the bias is g * b2_m, and the result goes to the token's
// target row (top_k = 1) or, in fp32, to the assignment's row of the
// per-assignment buffer that the combine kernel sums (top_k > 1).
// ---------------------------------------------------------------------------
template <bool ROUTED>
__global__ __launch_bounds__(256, 1) void k_bf16_gemm2_256(Problem p, UnitTab ut) {
    __shared__ u32x4 lds[kNST * kStage];
    const uint32_t code = ut.code[blockIdx.z];
    const int j = unit_j(code), x = unit_x(code), gs = unit_gslot(code);
    const int EH = ROUTED ? p.hidden : p.E * p.hidden;   // the K axis
    const int nA = (p.d_out + kTile - 1) / kTile;
    const int nB = ROUTED ? p.rt.max_tiles : (p.n_tok + kTile - 1) / kTile;
    int at, bt;
    tile_of(blockIdx.x, nA, nB, at, bt);
    int m = 0, first = 0, rows = 0;
    if constexpr (ROUTED) {
        if (bt >= p.rt.ntiles[gs]) return;
        const int4 tl = p.rt.tiles[(size_t)gs * p.rt.max_tiles + bt];
        m = tl.x; first = tl.y; rows = tl.z;
    }
    const int out0 = at * kTile, tok0 = ROUTED ? first : bt * kTile;
    const int row_end = ROUTED ? first + rows : p.n_tok;
    const size_t unit = (size_t)j * p.streams + x;
    const size_t wsel = ROUTED ? unit * p.E + m : unit;
    const size_t hstride = ROUTED ? routed_hidden_elems(p) : (size_t)p.n_tok_pad * EH;
    const rsrc_t bufA = make_rsrc(reinterpret_cast<const char*>(p.w2) + wsel * EH * p.d_out * 2,
                                  (size_t)EH * p.d_out * 2);
    const rsrc_t bufB = make_rsrc(reinterpret_cast<const char*>(p.hbuf) + blockIdx.z * hstride * 2, hstride * 2);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int L = lane / kCPR;
    const int c = (lane % kCPR) ^ swz(L);   // this lane's logical chunk, the same in each load

    uint32_t voA[kNI], voB[kNI];
#pragma unroll
    for (int q = 0; q < kNI; ++q) {
        const int r = kRPI * (wave * kNI + q) + L;
        const int o = min(out0 + r, p.d_out - 1);
        const int t = min(tok0 + r, row_end - 1);
        voA[q] = (uint32_t)o * p.hidden * 2 + 16 * c;
        voB[q] = ((uint32_t)(t >> 5) * (EH >> 3) * 256 + (t & 31) * 8) * 2 + 512 * c;
    }
    // W2cat is [E][d_out][hidden]: slice kt lies in expert k0 / hidden (hidden
    // is a multiple of 64); the hidden buffer's 16-byte units of a slice are
    // [t/32][k/8][t%32], so both column offsets are uniform
    auto slice = [&](int kt, uint32_t& sa, uint32_t& sb, uint32_t& vb) {
        const int k0 = kt * kBK, e = k0 / p.hidden;
        sa = ((uint32_t)e * p.d_out * p.hidden + (k0 - e * p.hidden)) * 2;
        sb = (uint32_t)(k0 >> 3) * 512;
        vb = 0;
    };

    // accumulators start at sum_e g_e(t) b2_e[o] (routed: g(t) b2_m[o])
    const int wave_m = wave >> 1, wn = wave & 1, g = lane >> 5, l32 = lane & 31;
    f32x16 acc[4][4];
#pragma unroll
    for (int bm = 0; bm < 4; ++bm)
#pragma unroll
        for (int bn = 0; bn < 4; ++bn)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[bm][bn][e] = 0.f;
    if (p.b2) {
        const uint16_t* b2 = reinterpret_cast<const uint16_t*>(p.b2) + wsel * (ROUTED ? 1 : p.E) * p.d_out;
        if constexpr (ROUTED) {
            const float* ag = p.rt.agate + (size_t)gs * p.n_tok * p.top_k;
            seed_bias(
                acc, 1, [&](int, int o) -> uint32_t { return b2[min(o, p.d_out - 1)]; },
                [&](int, int a) -> float { return a < row_end ? ag[a] : 0.f; }, out0 + wave_m * 128,
                tok0 + wn * 128);
        } else {
            const float* G = p.gates + (size_t)gs * p.n_tok_pad * p.E;
            seed_bias(
                acc, p.E, [&](int e, int o) -> uint32_t { return b2[(size_t)e * p.d_out + min(o, p.d_out - 1)]; },
                [&](int e, int t) -> float { return t < p.n_tok ? G[(size_t)t * p.E + e] : 0.f; },
                out0 + wave_m * 128, tok0 + wn * 128);
        }
    }

    k_loop(lds, bufA, bufB, voA, voB, EH / kBK, slice, acc);

    // epilogue: four consecutive outputs of one row per store
    const int32_t* list = ROUTED ? p.rt.list + (size_t)gs * p.n_tok * p.top_k : nullptr;
    float* part = ROUTED && p.top_k > 1 ? p.rt.part + blockIdx.z * (size_t)p.n_tok * p.top_k * p.d_out : nullptr;
    uint16_t* dst = reinterpret_cast<uint16_t*>(p.dst[x]) + (size_t)j * p.n_tok * p.d_out;
#pragma unroll
    for (int bm = 0; bm < 4; ++bm) {
        const int obase = out0 + wave_m * 128 + bm * 32;
        if (obase >= p.d_out) continue;   // d_out % 32 == 0
#pragma unroll
        for (int bn = 0; bn < 4; ++bn) {
            const int r = tok0 + wn * 128 + bn * 32 + l32;   // token, or assignment
            if (r >= row_end) continue;
            if (part) {
#pragma unroll
                for (int ii = 0; ii < 4; ++ii) {
                    const f32x4 v = {acc[bm][bn][4 * ii], acc[bm][bn][4 * ii + 1], acc[bm][bn][4 * ii + 2],
                                     acc[bm][bn][4 * ii + 3]};
                    *reinterpret_cast<f32x4*>(part + (size_t)r * p.d_out + obase + 8 * ii + 4 * g) = v;
                }
                continue;
            }
            const int t = ROUTED ? list[r] : r;
            size_t row;
            int hs = 0;
            if (p.dst_layout == MOT_LAYOUT_BTHD) {
                row = (size_t)t * p.d_out;
            } else {
                const int b = t / p.T, tt = t % p.T;
                row = ((size_t)b * p.H_tgt * p.T + tt) * p.D_tgt;
                hs = p.T * p.D_tgt;
            }
#pragma unroll
            for (int ii = 0; ii < 4; ++ii) {
                const int o = obase + 8 * ii + 4 * g;   // D_tgt % 8 == 0: o .. o+3 in one head
                const size_t off = p.dst_layout == MOT_LAYOUT_BTHD
                                       ? row + o
                                       : row + (size_t)(o / p.D_tgt) * hs + o % p.D_tgt;
                u32x2 w = {pack_bf16x2(acc[bm][bn][4 * ii], acc[bm][bn][4 * ii + 1]),
                           pack_bf16x2(acc[bm][bn][4 * ii + 2], acc[bm][bn][4 * ii + 3])};
                *reinterpret_cast<u32x2*>(dst + off) = w;
            }
        }
    }
}

// ---------------------------------------------------------------------------
// MoT-h restoration (paper App. C.5) on the same tiles: per layer l,
// out[t][o] = sum_k a[l][t][k] W[o][k] + b[o] with W^K rows (o < d_kv) and
// W^V rows side by side.  d_kv % 256 == 0, so an output tile lies in one of
// the two projections.  grid: x = (output tiles) x (token tiles) in dispatch
// order, z = position in the layer list.  MFMA A = projection rows, B =
// activation rows; each lane's four consecutive outputs of one token go to
// the key or value cache as one 8-byte store in the target layout.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256, 1) void k_bf16_project_256(ProjProblem p) {
    __shared__ u32x4 lds[kNST * kStage];
    const int l = p.layers[blockIdx.z];
    const int d_kv = p.d_kv, d_act = p.d_act;
    int at, bt;
    tile_of(blockIdx.x, 2 * d_kv / kTile, (p.n_tok + kTile - 1) / kTile, at, bt);
    const int out0 = at * kTile, tok0 = bt * kTile;
    const bool isv = out0 >= d_kv;
    const int ok0 = isv ? out0 - d_kv : out0;   // first row of the tile in its projection
    const uint16_t* W = reinterpret_cast<const uint16_t*>(isv ? p.wv : p.wk) + (size_t)l * d_kv * d_act;
    const uint16_t* bias = reinterpret_cast<const uint16_t*>(isv ? p.bv : p.bk);
    if (bias) bias += (size_t)l * d_kv;
    const rsrc_t bufA = make_rsrc(W, (size_t)d_kv * d_act * 2);
    const rsrc_t bufB = make_rsrc(reinterpret_cast<const uint16_t*>(p.act) + (size_t)l * p.n_tok * d_act,
                                  (size_t)p.n_tok * d_act * 2);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int L = lane / kCPR;
    const int c = (lane % kCPR) ^ swz(L);   // this lane's logical chunk, the same in each load
    uint32_t voA[kNI], voB[kNI];
#pragma unroll
    for (int q = 0; q < kNI; ++q) {
        const int r = kRPI * (wave * kNI + q) + L;
        voA[q] = (uint32_t)(ok0 + r) * d_act * 2 + 16 * c;
        voB[q] = (uint32_t)min(tok0 + r, p.n_tok - 1) * d_act * 2 + 16 * c;
    }
    auto slice = [&](int kt, uint32_t& sa, uint32_t& sb, uint32_t& vb) {
        sa = (uint32_t)kt * kBK * 2;
        sb = sa;
        vb = 0;
    };
    // accumulators start at the bias: lane rows of block bm are outputs
    // ok0 + wm*128 + bm*32 + 8*ii + 4*g + jj of the projection
    const int wm = wave >> 1, wn = wave & 1, g = lane >> 5, l32 = lane & 31;
    f32x16 acc[4][4];
#pragma unroll
    for (int bm = 0; bm < 4; ++bm) {
        f32x16 init;
#pragma unroll
        for (int ii = 0; ii < 4; ++ii) {
            u32x2 w = {0u, 0u};
            if (bias) w = *reinterpret_cast<const u32x2*>(bias + ok0 + wm * 128 + bm * 32 + 8 * ii + 4 * g);
            init[4 * ii + 0] = bf16_lo(w[0]);
            init[4 * ii + 1] = bf16_hi(w[0]);
            init[4 * ii + 2] = bf16_lo(w[1]);
            init[4 * ii + 3] = bf16_hi(w[1]);
        }
#pragma unroll
        for (int bn = 0; bn < 4; ++bn) acc[bm][bn] = init;
    }

    k_loop(lds, bufA, bufB, voA, voB, d_act / kBK, slice, acc);

    uint16_t* dst = reinterpret_cast<uint16_t*>(isv ? p.dst_v : p.dst_k) + (size_t)l * p.n_tok * d_kv;
#pragma unroll
    for (int bn = 0; bn < 4; ++bn) {
        const int tc = tok0 + wn * 128 + bn * 32 + l32;
        if (tc >= p.n_tok) continue;
        const int b = tc / p.T, t = tc % p.T;
#pragma unroll
        for (int bm = 0; bm < 4; ++bm) {
#pragma unroll
            for (int ii = 0; ii < 4; ++ii) {
                const int ok = ok0 + wm * 128 + bm * 32 + 8 * ii + 4 * g;   // four outputs of one head
                const int hh = ok / p.D_tgt, dd = ok % p.D_tgt;
                const size_t off = p.dst_layout == MOT_LAYOUT_BTHD
                                       ? (size_t)tc * d_kv + ok
                                       : (((size_t)b * p.H_tgt + hh) * p.T + t) * p.D_tgt + dd;
                const u32x2 w = {pack_bf16x2(acc[bm][bn][4 * ii], acc[bm][bn][4 * ii + 1]),
                                 pack_bf16x2(acc[bm][bn][4 * ii + 2], acc[bm][bn][4 * ii + 3])};
                *reinterpret_cast<u32x2*>(dst + off) = w;
            }
        }
    }
}

}  // namespace

// Large tiles pay when a launch has at least one round of workgroups.
bool bf16_gemm256_fits(const Problem& p, int n_units) {
    const int EH = p.E * p.hidden;
    const long t = (p.n_tok + kTile - 1) / kTile;
    const long g1 = t * ((EH + kTile - 1) / kTile) * n_units;
    // every operand region is addressed with 32-bit byte offsets
    const size_t lim = (size_t)1 << 31;
    const size_t w1 = (size_t)EH * p.d_in * 2, src = (size_t)p.n_tok * p.d_in * 2;
    const size_t hb = (size_t)p.n_tok_pad * EH * 2, w2 = (size_t)EH * p.d_out * 2;
    return p.E <= 16 && g1 >= 128 && w1 < lim && src < lim && hb < lim && w2 < lim;
}

hipError_t launch_bf16_gemm1_256(const Problem& p, const UnitTab& ut, hipStream_t stream) {
    if (ut.n == 0 || p.n_tok == 0) return hipSuccess;
    const int EH = p.E * p.hidden;
    dim3 grid(((EH + kTile - 1) / kTile) * ((p.n_tok + kTile - 1) / kTile), 1, ut.n);
    hipLaunchKernelGGL(k_bf16_gemm1_256<false>, grid, dim3(256), 0, stream, p, ut);
    return hipGetLastError();
}

hipError_t launch_bf16_gemm2_256(const Problem& p, const UnitTab& ut, hipStream_t stream) {
    if (ut.n == 0 || p.n_tok == 0) return hipSuccess;
    dim3 grid(((p.d_out + kTile - 1) / kTile) * ((p.n_tok + kTile - 1) / kTile), 1, ut.n);
    hipLaunchKernelGGL(k_bf16_gemm2_256<false>, grid, dim3(256), 0, stream, p, ut);
    return hipGetLastError();
}

bool bf16_routed_gemm_fits(const Problem& p) {
    const size_t lim = (size_t)1 << 31;
    const size_t nk = (size_t)p.n_tok * p.top_k;
    const size_t w1 = (size_t)p.hidden * p.d_in * 2, src = (size_t)p.n_tok * p.d_in * 2;
    const size_t hb = (nk + 31) / 32 * 32 * p.hidden * 2, w2 = (size_t)p.hidden * p.d_out * 2;
    return p.E <= 16 && w1 < lim && src < lim && hb < lim && w2 < lim;
}

bool bf16_project_256_fits(const ProjProblem& p, int n_layers) {
    const size_t lim = (size_t)1 << 31;
    const long wgs = (long)(2 * p.d_kv / kTile) * ((p.n_tok + kTile - 1) / kTile) * n_layers;
    // the biases are read four at a time (8 bytes); the API guarantees 2-byte alignment only
    const bool bias8 = (reinterpret_cast<uintptr_t>(p.bk) & 7) == 0 && (reinterpret_cast<uintptr_t>(p.bv) & 7) == 0;
    return p.d_kv % kTile == 0 && p.d_act % kBK == 0 && p.D_tgt % 4 == 0 && wgs >= 128 && bias8 &&
           (size_t)p.n_tok * p.d_act * 2 < lim && (size_t)p.d_kv * p.d_act * 2 < lim;
}

hipError_t launch_bf16_project_256(const ProjProblem& p, int n_layers, hipStream_t stream) {
    if (n_layers == 0 || p.n_tok == 0) return hipSuccess;
    const dim3 grid((2 * p.d_kv / kTile) * ((p.n_tok + kTile - 1) / kTile), 1, n_layers);
    hipLaunchKernelGGL(k_bf16_project_256, grid, dim3(256), 0, stream, p);
    return hipGetLastError();
}

size_t bf16_routed_hidden_bytes(const Problem& p) {
    return ((size_t)p.n_tok * p.top_k + 31) / 32 * 32 * p.hidden * 2;
}

hipError_t launch_bf16_gemm1_routed(const Problem& p, const UnitTab& ut, hipStream_t stream) {
    if (ut.n == 0 || p.n_tok == 0) return hipSuccess;
    dim3 grid(((p.hidden + kTile - 1) / kTile) * p.rt.max_tiles, 1, ut.n);
    hipLaunchKernelGGL(k_bf16_gemm1_256<true>, grid, dim3(256), 0, stream, p, ut);
    return hipGetLastError();
}

hipError_t launch_bf16_gemm2_routed(const Problem& p, const UnitTab& ut, hipStream_t stream) {
    if (ut.n == 0 || p.n_tok == 0) return hipSuccess;
    dim3 grid(((p.d_out + kTile - 1) / kTile) * p.rt.max_tiles, 1, ut.n);
    hipLaunchKernelGGL(k_bf16_gemm2_256<true>, grid, dim3(256), 0, stream, p, ut);
    return hipGetLastError();
}

}  // namespace mot
