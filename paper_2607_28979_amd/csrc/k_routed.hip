// Routed (Top-K sparse) path, the parts around the fused kernel (paper
// Sec. 3, Definition "Mixture-of-Translators" with K < E: every token runs
// through its K selected translators only).
//
// k_route_plan: one workgroup per unit turns the per-token Top-K lists into
// translator-contiguous assignment lists by a stable counting sort (tokens in
// ascending order within each translator), the tile table of the fused
// kernel (tiles of tile_rows assignments, never straddling two translators)
// and, for top_k > 1, each (token, k)'s assignment index.  No atomics: the
// result is the same on every run.  The translator totals are also added to
// the optional usage counts.
//
// k_routed_combine (top_k > 1): out[token] = sum over k of the fp32
// per-assignment rows, in k order, rounded once to bf16 and stored in the
// target layout.
#include "mot_device.h"
#include "mot_internal.h"
#include "../../include/mot.h"

namespace mot {

namespace {

constexpr int kPlanThreads = 1024;

__global__ __launch_bounds__(kPlanThreads) void k_route_plan(Problem p, UnitTab ut) {
    __shared__ int32_t s_run[MOT_MAX_EXPERTS][kPlanThreads];   // per-thread counts, then cursors
    __shared__ int32_t s_wave[MOT_MAX_EXPERTS][kPlanThreads / 64];
    __shared__ int32_t s_eoff[MOT_MAX_EXPERTS + 1], s_toff[MOT_MAX_EXPERTS + 1];

    const uint32_t code = ut.code[blockIdx.x];
    const int gs = unit_gslot(code);
    // translator usage of this unit (the totals of the counting sort)
    uint32_t* usage = p.usage ? p.usage + ((size_t)unit_j(code) * p.streams + unit_x(code)) * p.E : nullptr;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int N = p.n_tok, K = p.top_k, E = p.E, BM = p.rt.tile_rows;
    const size_t NK = (size_t)N * K;
    const int32_t* sel = p.rt.sel + gs * NK;
    const float* gk = p.rt.gk + gs * NK;
    int32_t* list = p.rt.list + gs * NK;
    float* agate = p.rt.agate + gs * NK;
    int32_t* slot = p.rt.slot ? p.rt.slot + gs * NK : nullptr;

    // contiguous token range of this thread
    const int per = (N + kPlanThreads - 1) / kPlanThreads;
    const int t0 = tid * per < N ? tid * per : N;
    const int t1 = t0 + per < N ? t0 + per : N;

    int cnt[MOT_MAX_EXPERTS];
#pragma unroll
    for (int m = 0; m < MOT_MAX_EXPERTS; ++m) cnt[m] = 0;
    for (int t = t0; t < t1; ++t)
        for (int k = 0; k < K; ++k) {
            const int m = sel[(size_t)t * K + k];
#pragma unroll
            for (int mm = 0; mm < MOT_MAX_EXPERTS; ++mm) cnt[mm] += m == mm ? 1 : 0;
        }

    // exclusive scan of every translator's counts over the threads, in
    // thread (= token) order: inclusive scan inside each wave, then over waves
    int incl[MOT_MAX_EXPERTS];
#pragma unroll
    for (int m = 0; m < MOT_MAX_EXPERTS; ++m) {
        int v = cnt[m];
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const int u = __shfl_up(v, d, 64);
            v += lane >= d ? u : 0;
        }
        incl[m] = v;
        if (lane == 63 && m < E) s_wave[m][wave] = v;
    }
    __syncthreads();
    if (tid < E) {
        int run = 0;
        for (int w = 0; w < kPlanThreads / 64; ++w) {
            const int v = s_wave[tid][w];
            s_wave[tid][w] = run;
            run += v;
        }
        s_run[tid][0] = run;   // translator total, read below before the cursors are written
    }
    __syncthreads();
    if (tid == 0) {
        int a = 0, tl = 0;
        for (int m = 0; m < E; ++m) {
            const int tot = s_run[m][0];
            if (usage && tot) atomicAdd(usage + m, (uint32_t)tot);
            s_eoff[m] = a;
            s_toff[m] = tl;
            a += tot;
            tl += (tot + BM - 1) / BM;
        }
        s_eoff[E] = a;
        s_toff[E] = tl;
        p.rt.ntiles[gs] = tl;
    }
    __syncthreads();
    // cursors: first assignment index of this thread's tokens per translator
#pragma unroll
    for (int m = 0; m < MOT_MAX_EXPERTS; ++m)
        if (m < E) s_run[m][tid] = s_eoff[m] + s_wave[m][wave] + incl[m] - cnt[m];
    __syncthreads();

    for (int t = t0; t < t1; ++t)
        for (int k = 0; k < K; ++k) {
            const size_t tk = (size_t)t * K + k;
            const int m = sel[tk];
            const int a = s_run[m][tid]++;
            list[a] = t;
            agate[a] = gk[tk];
            if (slot) slot[tk] = a;
        }

    // tile table: tiles of translator m cover its assignments in order
    if (tid < E) {
        const int m = tid, first = s_eoff[m], tot = s_eoff[m + 1] - first;
        int4* tiles = p.rt.tiles + (size_t)gs * p.rt.max_tiles + s_toff[m];
        for (int i = 0; i * BM < tot; ++i) {
            const int rows = tot - i * BM < BM ? tot - i * BM : BM;
            tiles[i] = make_int4(m, first + i * BM, rows, 0);
        }
    }
}

// 8 outputs per thread; blockIdx.y = the unit's position in its group
__global__ __launch_bounds__(256) void k_routed_combine(Problem p, UnitTab ut) {
    const uint32_t code = ut.code[blockIdx.y];
    const int j = unit_j(code), x = unit_x(code), gs = unit_gslot(code);
    const int d_out = p.d_out, per_tok = d_out / 8, K = p.top_k;
    const size_t idx = (size_t)blockIdx.x * 256 + threadIdx.x;
    if (idx >= (size_t)p.n_tok * per_tok) return;
    const int tok = (int)(idx / per_tok), o = (int)(idx % per_tok) * 8;
    const size_t NK = (size_t)p.n_tok * K;
    const int32_t* slot = p.rt.slot + gs * NK + (size_t)tok * K;
    const float* part = p.rt.part + blockIdx.y * NK * d_out;
    float s[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) s[e] = 0.f;
    for (int k = 0; k < K; ++k) {
        const float* r = part + (size_t)slot[k] * d_out + o;
        const f32x4 a = *reinterpret_cast<const f32x4*>(r);
        const f32x4 b = *reinterpret_cast<const f32x4*>(r + 4);
        s[0] += a[0]; s[1] += a[1]; s[2] += a[2]; s[3] += a[3];
        s[4] += b[0]; s[5] += b[1]; s[6] += b[2]; s[7] += b[3];
    }
    u32x4 v;
#pragma unroll
    for (int q = 0; q < 4; ++q) v[q] = pack_bf16x2(s[2 * q], s[2 * q + 1]);
    size_t off;
    if (p.dst_layout == MOT_LAYOUT_BTHD) {
        off = (size_t)tok * d_out + o;
    } else {
        const int b = tok / p.T, t = tok % p.T, hh = o / p.D_tgt, dd = o % p.D_tgt;
        off = (((size_t)b * p.H_tgt + hh) * p.T + t) * p.D_tgt + dd;
    }
    uint16_t* dst = reinterpret_cast<uint16_t*>(p.dst[x]) + (size_t)j * p.n_tok * d_out;
    *reinterpret_cast<u32x4*>(dst + off) = v;
}

}  // namespace

hipError_t launch_route_plan(const Problem& p, const UnitTab& ut, hipStream_t stream) {
    if (ut.n == 0 || p.n_tok == 0) return hipSuccess;
    hipLaunchKernelGGL(k_route_plan, dim3(ut.n), dim3(kPlanThreads), 0, stream, p, ut);
    return hipGetLastError();
}

hipError_t launch_routed_combine(const Problem& p, const UnitTab& ut, hipStream_t stream) {
    if (ut.n == 0 || p.n_tok == 0) return hipSuccess;
    const size_t items = (size_t)p.n_tok * (p.d_out / 8);
    dim3 grid((unsigned)((items + 255) / 256), ut.n);
    hipLaunchKernelGGL(k_routed_combine, grid, dim3(256), 0, stream, p, ut);
    return hipGetLastError();
}

}  // namespace mot
