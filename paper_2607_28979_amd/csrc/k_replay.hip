// Context replay after translation (paper App. C.4, "Post-Translation Phase:
// Cache Replay"): Top-S source-guided sparse attention.
//
// * k_topS_select: for each query position u, the S key positions v <= u
//   with the largest head-averaged source attention A[b][u][v] (ties to the
//   lower position), in ascending position order, padded with -1.  Radix
//   select over order-preserving 32-bit keys: a 1024-bin histogram of the
//   top 10 bits finds the bin holding the S-th largest key; that bin's keys
//   (a few dozen on attention rows) are ranked against each other for the
//   exact key, or, past 256 of them, 8-bit radix passes over the lower bits
//   finish the search; then one ordered pass keeps every larger key and the
//   lowest-positioned equal ones.
// * k_sparse_attn: attention of every query head of (b, u) over its key set
//   (grouped-query: query head h reads KV head h / G).  Per KV head the
//   workgroup computes scores^T = K_sel . Q^T on v_mfma_f32_16x16x32_bf16 with
//   the gathered key rows loaded straight into A operands, a softmax over the
//   set, and O^T = V_sel^T . P^T with V_sel staged transposed in LDS.
// * k_causal_attn: the full causal attention of the bottom layers, tiled
//   (128 query positions of one head, two tiles per workgroup paired short
//   with long, 64-key chunks of K and V^T loaded straight into LDS one chunk
//   ahead, online softmax, v_mfma_f32_32x32x16_bf16).
// Scores, softmax and accumulation are fp32; Q, K, V, O are bf16.
#include "mot_device.h"
#include "mot_internal.h"
#include "../../include/mot.h"

namespace mot {

namespace {

constexpr float kLog2e = 1.4426950408889634f;

typedef __attribute__((address_space(3))) void lds_void;
typedef __amdgpu_buffer_rsrc_t rsrc_t;

// Raw buffer over `bytes` bytes at `base` (reads past the end return 0).
__device__ __forceinline__ rsrc_t make_rsrc(const void* base, size_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0,
                                             (int)(bytes < 0xFFFFFFFFu ? bytes : 0xFFFFFFFFu), 0x00020000);
}

// 16 bytes per lane from the buffer straight into this wave's 1 KB of LDS
__device__ __forceinline__ void load_lds16(rsrc_t r, uint32_t off, u32x4* lds_dst_wave_base) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)lds_dst_wave_base, 16, off, 0, 0, 0);
}

// Monotone map float -> uint32 (a < b  <=>  key(a) < key(b) for non-NaN).
__device__ __forceinline__ uint32_t order_key(float a) {
    const uint32_t b = __float_as_uint(a);
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

constexpr int kSelBits = 10, kSelBins = 1 << kSelBits;   // first radix digit
constexpr int kSelCand = 256;                              // boundary-bin keys ranked directly
static_assert(kSelBins == 4 * 256, "four first-digit bins per thread");

// grid (T, B), 256 threads; CACHE: the row's keys live in dynamic LDS (T words)
// ahead of the per-chunk counts
template <bool CACHE>
__global__ __launch_bounds__(256) void k_topS_select(const float* A, int32_t* idx, int T, int S) {
    extern __shared__ uint32_t s_key[];
    __shared__ uint32_t hist[kSelBins];
    __shared__ uint32_t s_cand[kSelCand];
    __shared__ uint32_t s_sel[3], s_wsum[4];
    __shared__ int s_cnt;
    const int u = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
    const int n = u + 1;
    int32_t* out = idx + ((size_t)b * T + u) * S;
    if (n <= S) {   // every causal position is kept (uniform exit, before any barrier)
        for (int c = tid; c < S; c += 256) out[c] = c < n ? c : -1;
        return;
    }
    const float* row = A + ((size_t)b * T + u) * T;
    // dynamic LDS: [CACHE: T keys] then per-chunk counts s_gt, s_eq (T/64 + 1 each)
    int* s_gt = reinterpret_cast<int*>(s_key + (CACHE ? T : 0));
    int* s_eq = s_gt + (T >> 6) + 1;
    if constexpr (CACHE) {
        // fill the key cache with 16-byte loads, several in flight per thread
        // (rows are 16-byte aligned when T % 4 == 0; the last piece may read
        // positions past u, still inside the row, and they are never used)
        if ((T & 3) == 0) {
            const f32x4* row4 = reinterpret_cast<const f32x4*>(row);
            u32x4* key4 = reinterpret_cast<u32x4*>(s_key);
            const int n4 = (n + 3) >> 2;
#pragma unroll 4
            for (int v = tid; v < n4; v += 256) {
                const f32x4 a = row4[v];
                key4[v] = u32x4{order_key(a.x), order_key(a.y), order_key(a.z), order_key(a.w)};
            }
        } else {
#pragma unroll 8
            for (int v = tid; v < n; v += 256) s_key[v] = order_key(row[v]);
        }
        __syncthreads();
    }
    // first digit: the top kSelBits bits (sign, exponent and one mantissa bit)
    constexpr int sh1 = 32 - kSelBits;
    auto key_at = [&](int v) -> uint32_t {
        if constexpr (CACHE) return s_key[v];
        else return order_key(row[v]);
    };
    // 1024 bins: an attention row's keys crowd into a few exponents, and with
    // an 8-bit first digit the boundary bin held ~70 keys and needed another
    // full radix pass; with 10 bits it holds a few dozen, ranked directly.
    if (tid < 64) s_cnt = 0;
#pragma unroll
    for (int i = 0; i < kSelBins / 256; ++i) hist[tid + 256 * i] = 0;
    __syncthreads();
    for (int v = tid; v < n; v += 256) atomicAdd(&hist[key_at(v) >> sh1], 1u);
    __syncthreads();
    {
        // thread t holds bins 4t .. 4t+3: suffix sums over the threads (within
        // each wave by shuffles, then the higher waves' totals) find the bin
        // holding the S-th largest key
        const int lane = tid & 63, wv = tid >> 6;
        const uint32_t h0 = hist[4 * tid], h1 = hist[4 * tid + 1], h2 = hist[4 * tid + 2], h3 = hist[4 * tid + 3];
        const uint32_t c = h0 + h1 + h2 + h3;
        uint32_t suf = c;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const uint32_t t = __shfl_down(suf, off, 64);
            if (lane + off < 64) suf += t;
        }
        if (lane == 0) s_wsum[wv] = suf;
        __syncthreads();
        for (int q = wv + 1; q < 4; ++q) suf += s_wsum[q];
        if (suf >= (uint32_t)S && suf - c < (uint32_t)S) {
            uint32_t cum = suf - c;   // keys in bins above 4t+3
            const uint32_t hb[4] = {h0, h1, h2, h3};
            int d = 4 * tid;
            uint32_t cnt = h0;
#pragma unroll
            for (int q = 3; q >= 0; --q) {
                if (cum + hb[q] >= (uint32_t)S) {
                    d = 4 * tid + q;
                    cnt = hb[q];
                    break;
                }
                cum += hb[q];
            }
            s_sel[0] = (uint32_t)d;
            s_sel[1] = cum;
            s_sel[2] = cnt;
        }
    }
    __syncthreads();
    const uint32_t d1 = s_sel[0], cnt1 = s_sel[2];
    int rem = S - (int)s_sel[1];   // keys still to choose in the boundary bin
    uint32_t prefix = d1 << sh1, mask = ~0u << sh1;
    if (cnt1 != (uint32_t)rem) {   // uniform: not every key of the boundary bin is taken
        if (cnt1 <= (uint32_t)kSelCand) {
            // the boundary bin's keys, ranked against each other: the rem-th
            // largest is the S-th largest of the row, and the keys equal to it
            // that are taken are the first ones in position order
            for (int v = tid; v < n; v += 256) {
                const uint32_t k = key_at(v);
                if ((k >> sh1) == d1) s_cand[atomicAdd(&s_cnt, 1)] = k;
            }
            __syncthreads();
            if (tid < (int)cnt1) {
                const uint32_t ki = s_cand[tid];
                int gt = 0, eq = 0;
                for (int j = 0; j < (int)cnt1; ++j) {
                    const uint32_t kj = s_cand[j];
                    gt += kj > ki;
                    eq += kj == ki;
                }
                if (gt < rem && rem <= gt + eq) {   // every such thread writes the same pair
                    s_sel[0] = ki;
                    s_sel[1] = (uint32_t)(rem - gt);
                }
            }
            __syncthreads();
            prefix = s_sel[0];
            mask = ~0u;
            rem = (int)s_sel[1];
        } else {
            // many keys share the digit: 8-bit radix passes over the bits
            // below it (a last digit that overlaps resolved bits is harmless:
            // the prefix filter fixes them)
            for (int sh = sh1; sh > 0;) {
                sh = sh > 8 ? sh - 8 : 0;
                const int shift = sh;
                hist[tid] = 0;
                __syncthreads();
                for (int v = tid; v < n; v += 256) {
                    const uint32_t k = key_at(v);
                    if ((k & mask) == prefix) atomicAdd(&hist[(k >> shift) & 255u], 1u);
                }
                __syncthreads();
                if (tid < 64) {
                    // lane l holds bins 4l .. 4l+3; suffix sums over lanes find the
                    // bin holding the rem-th largest remaining key
                    const uint32_t h0 = hist[4 * tid], h1 = hist[4 * tid + 1], h2 = hist[4 * tid + 2],
                                   h3 = hist[4 * tid + 3];
                    const uint32_t c = h0 + h1 + h2 + h3;
                    uint32_t suf = c;
#pragma unroll
                    for (int off = 1; off < 64; off <<= 1) {
                        const uint32_t t = __shfl_down(suf, off, 64);
                        if (tid + off < 64) suf += t;
                    }
                    const unsigned long long bal = __ballot(suf >= (uint32_t)rem);   // lanes 0 .. L
                    const int L = 63 - __clzll(bal);
                    if (tid == L) {
                        uint32_t cum = suf - c;   // keys in bins above 4L+3
                        int d = 4 * L;
                        uint32_t cnt = h0;
                        const uint32_t hb[4] = {h0, h1, h2, h3};
#pragma unroll
                        for (int q = 3; q >= 0; --q) {
                            if (cum + hb[q] >= (uint32_t)rem) {
                                d = 4 * L + q;
                                cnt = hb[q];
                                break;
                            }
                            cum += hb[q];
                        }
                        s_sel[0] = (uint32_t)d;
                        s_sel[1] = cum;
                        s_sel[2] = cnt;
                    }
                }
                __syncthreads();
                const uint32_t d = s_sel[0], cnt = s_sel[2];
                rem -= (int)s_sel[1];
                prefix |= d << shift;
                mask |= 255u << shift;
                __syncthreads();
                // every key of the boundary bin is taken: the digits below decide nothing
                if (cnt == (uint32_t)rem) break;
            }
        }
    }
    // prefix is the S-th largest key on the resolved digits (k & mask): take
    // every key larger under the mask and the first rem equal ones in
    // position order (all of them after an early stop).  Rows are cut into
    // 64-position chunks (chunk c: positions 64c + lane, wave c % 4):
    // per-chunk counts of larger and equal keys, one scan over the chunks,
    // then each chunk writes its picks at its offset in ballot order.
    const int lane = tid & 63, wv = tid >> 6, nch = (n + 63) >> 6;
    for (int c = wv; c < nch; c += 4) {
        const int v = 64 * c + lane;
        const uint32_t k = v < n ? key_at(v) & mask : 0u;
        const unsigned long long bg = __ballot(v < n && k > prefix), be = __ballot(v < n && k == prefix);
        if (lane == 0) {
            s_gt[c] = __popcll(bg);
            s_eq[c] = __popcll(be);
        }
    }
    __syncthreads();
    if (tid < 64) {
        // exclusive scans over chunks: lane l owns chunks [l*cpl, l*cpl + cpl)
        const int cpl = (nch + 63) >> 6, c0 = tid * cpl, c1 = min(c0 + cpl, nch);
        int eq_l = 0;
        for (int c = c0; c < c1; ++c) eq_l += s_eq[c];
        int eq_pre = eq_l;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int t = __shfl_up(eq_pre, off, 64);
            if (tid >= off) eq_pre += t;
        }
        eq_pre -= eq_l;   // equal keys before this lane's chunks
        int take_l = 0;
        for (int c = c0; c < c1; ++c) {
            const int e = s_eq[c];
            const int left = rem - eq_pre;   // equal keys still to take when chunk c starts
            const int tk = s_gt[c] + (left <= 0 ? 0 : (left < e ? left : e));
            s_eq[c] = eq_pre;                // now: equal keys before chunk c
            s_gt[c] = tk;                    // now: picks in chunk c
            eq_pre += e;
            take_l += tk;
        }
        int tk_pre = take_l;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int t = __shfl_up(tk_pre, off, 64);
            if (tid >= off) tk_pre += t;
        }
        tk_pre -= take_l;
        for (int c = c0; c < c1; ++c) {
            const int tk = s_gt[c];
            s_gt[c] = tk_pre;                // now: picks before chunk c
            tk_pre += tk;
        }
    }
    __syncthreads();
    for (int c = wv; c < nch; c += 4) {
        const int v = 64 * c + lane;
        const uint32_t k = v < n ? key_at(v) & mask : 0u;
        const bool eq = v < n && k == prefix;
        const unsigned long long be = __ballot(eq);
        const int eq_rank = s_eq[c] + __popcll(be & ((1ull << lane) - 1ull));
        const bool take = (v < n && k > prefix) || (eq && eq_rank < rem);
        const unsigned long long bt = __ballot(take);
        const int pos = s_gt[c] + __popcll(bt & ((1ull << lane) - 1ull));
        if (take && pos < S) out[pos] = v;
    }
}

__device__ __forceinline__ size_t kv_row(const ReplayProblem& p, int b, int t, int kvh) {
    return p.kv_layout == MOT_LAYOUT_BTHD ? (((size_t)b * p.T + t) * p.H_kv + kvh) * p.D
                                          : (((size_t)b * p.H_kv + kvh) * p.T + t) * p.D;
}

// Workgroups are dispatched round-robin over the 8 XCDs, each with its own
// L2.  A grid of 8 * ceil(n / 8) workgroups is remapped so that XCD k walks
// the contiguous range [k * per, (k + 1) * per) of the n work items: items
// that share K/V rows (neighbouring positions, the heads of one KV group)
// meet in one L2.  Items >= n return at once.
__device__ __forceinline__ int xcd_item(int id, int n) { return (id & 7) * ((n + 7) >> 3) + (id >> 3); }
inline int xcd_grid(int n) { return 8 * ((n + 7) / 8); }

__device__ __forceinline__ void wave_lds_sync() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// 8 bf16 of chunk a (keys k0) and c (key k0+1) interleaved into 8 words:
// word i = (a[i], c[i]) for d = 8*chunk + i
__device__ __forceinline__ uint32_t pair_word(const u32x4& a, const u32x4& c, int i) {
    const uint32_t wa = a[i >> 1], wc = c[i >> 1];
    return (i & 1) ? ((wa >> 16) | (wc & 0xFFFF0000u)) : ((wa & 0xFFFFu) | (wc << 16));
}

// grid (xcd_grid(T), B), 256 threads; dynamic LDS: V^T [D][S] + P [16][S] (bf16) + 128 floats
template <int D, int SMAX>
__global__ __launch_bounds__(256) void k_sparse_attn(ReplayProblem p) {
    extern __shared__ u32x4 s_dyn[];
    constexpr int DC = D / 8;               // 16-byte chunks per row of D
    const int S = p.S, SC = S / 8;          // 16-byte chunks per row of S keys
    // XOR swizzle within aligned groups of the largest power of two (<= 16)
    // dividing SC, so that a permuted chunk stays inside its row
    const int swm = replay_swizzle_mask(SC);
    u32x4* Vt = s_dyn;                      // row d: SC chunks, chunk c at (c ^ (d & swm))
    u32x4* Pl = s_dyn + D * SC;             // row = query head slot
    float* red = reinterpret_cast<float*>(Pl + 16 * SC);   // [4 waves][16]: max, then sum
    const int u = xcd_item(blockIdx.x, p.T), b = blockIdx.y;
    if (u >= p.T) return;   // uniform over the workgroup
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, l16 = lane & 15, q4 = lane >> 4;
    const int G = p.H_q / p.H_kv, KB = S / 16;
    const int32_t* keys = p.idx + ((size_t)b * p.T + u) * S;
    const uint16_t* Q = reinterpret_cast<const uint16_t*>(p.q);
    const uint16_t* K = reinterpret_cast<const uint16_t*>(p.k);
    const uint16_t* V = reinterpret_cast<const uint16_t*>(p.v);
    uint16_t* O = reinterpret_cast<uint16_t*>(p.o);
    const float sl2 = kLog2e / sqrtf((float)D);
    const u32x4 zero = {0u, 0u, 0u, 0u};
    // a key entry outside 0..u (the -1 padding) is not attended
    auto key_ok = [&](int kv) { return kv >= 0 && kv <= u; };
    // the set is the same for every KV head: read it once
    __shared__ int s_keys[256];
    for (int i = tid; i < S; i += 256) s_keys[i] = keys[i];
    __syncthreads();
    // per-thread item counts for sets of up to SMAX keys
    constexpr int MAXR = replay_sparse_v_items(D, SMAX);   // V key-pair items
    constexpr int MAXB = replay_sparse_key_blocks(SMAX);   // key blocks per wave
    static_assert(replay_sparse_supported(D, SMAX), "instantiated set size");

    for (int kvh = 0; kvh < p.H_kv; ++kvh) {
        // every gather of this KV head is issued before the first is used:
        // (a) V rows, item = (key pair, d chunk); (b) K rows of this wave's
        // key blocks kb = w, w+4, ...; then the query heads of the group
        u32x4 va[MAXR], vc[MAXR];
#pragma unroll
        for (int r = 0; r < MAXR; ++r) {
            const int it = tid + 256 * r;
            va[r] = zero;
            vc[r] = zero;
            if (it < (S / 2) * DC) {
                const int pr = it % (S / 2), dc = it / (S / 2), k0 = 2 * pr;
                const int v0 = s_keys[k0], v1 = s_keys[k0 + 1];
                if (key_ok(v0)) va[r] = *reinterpret_cast<const u32x4*>(V + kv_row(p, b, v0, kvh) + 8 * dc);
                if (key_ok(v1)) vc[r] = *reinterpret_cast<const u32x4*>(V + kv_row(p, b, v1, kvh) + 8 * dc);
            }
        }
        u32x4 ka[MAXB][D / 32];
#pragma unroll
        for (int i = 0; i < MAXB; ++i) {
            const int kb = w + 4 * i;
            const int kr = kb < KB ? s_keys[kb * 16 + l16] : -1;
            const uint16_t* krow = K + (key_ok(kr) ? kv_row(p, b, kr, kvh) : 0);
#pragma unroll
            for (int ks = 0; ks < D / 32; ++ks)
                ka[i][ks] = key_ok(kr) ? *reinterpret_cast<const u32x4*>(krow + 32 * ks + 8 * q4) : zero;
        }
        const int hq = kvh * G + l16;
        u32x4 qop[D / 32];
#pragma unroll
        for (int ks = 0; ks < D / 32; ++ks)
            qop[ks] = l16 < G ? *reinterpret_cast<const u32x4*>(Q + (((size_t)b * p.T + u) * p.H_q + hq) * D + 32 * ks + 8 * q4)
                              : zero;
        // V_sel^T into LDS
        uint32_t* Vw = reinterpret_cast<uint32_t*>(Vt);
#pragma unroll
        for (int r = 0; r < MAXR; ++r) {
            const int it = tid + 256 * r;
            if (it < (S / 2) * DC) {
                const int pr = it % (S / 2), dc = it / (S / 2), k0 = 2 * pr;
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    const int d = 8 * dc + i;
                    Vw[(d * SC + ((k0 >> 3) ^ (d & swm))) * 4 + ((k0 & 7) >> 1)] = pair_word(va[r], vc[r], i);
                }
            }
        }
        // scores^T[key][head]
        f32x4 sc[MAXB];
        float mx = -INFINITY;
#pragma unroll
        for (int i = 0; i < MAXB; ++i) {
            const int kb = w + 4 * i;
            sc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
            if (kb < KB) {
#pragma unroll
                for (int ks = 0; ks < D / 32; ++ks) sc[i] = mfma_16x16x32(ka[i][ks], qop[ks], sc[i]);
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    sc[i][j] = key_ok(s_keys[kb * 16 + 4 * q4 + j]) ? sc[i][j] : -INFINITY;
                    mx = fmaxf(mx, sc[i][j]);
                }
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j) sc[i][j] = -INFINITY;
            }
        }
        // (c) softmax over the set, per head (lane column l16)
        mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
        mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
        if (q4 == 0) red[w * 16 + l16] = mx;
        __syncthreads();
        mx = fmaxf(fmaxf(red[l16], red[16 + l16]), fmaxf(red[32 + l16], red[48 + l16]));
        float sum = 0.f;
#pragma unroll
        for (int i = 0; i < MAXB; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const float e = sc[i][j] == -INFINITY ? 0.f : exp2f((sc[i][j] - mx) * sl2);
                sc[i][j] = e;
                sum += e;
            }
        sum += __shfl_xor(sum, 16, 64);
        sum += __shfl_xor(sum, 32, 64);
        __syncthreads();   // every wave has read the maxima
        if (q4 == 0) red[w * 16 + l16] = sum;
        __syncthreads();
        sum = red[l16] + red[16 + l16] + red[32 + l16] + red[48 + l16];
        const float inv = sum > 0.f ? 1.0f / sum : 0.f;
        uint32_t* Pw = reinterpret_cast<uint32_t*>(Pl);
#pragma unroll
        for (int i = 0; i < MAXB; ++i) {
            const int kb = w + 4 * i;
            if (kb < KB) {
                const int ch = (2 * kb + (q4 >> 1)) ^ (l16 & swm);
                const int base = (l16 * SC + ch) * 4 + 2 * (q4 & 1);
                Pw[base] = pack_bf16x2(sc[i][0] * inv, sc[i][1] * inv);
                Pw[base + 1] = pack_bf16x2(sc[i][2] * inv, sc[i][3] * inv);
            }
        }
        __syncthreads();
        // (d) O^T[d][head] = V_sel^T . P^T, d blocks db = w, w+4, ...
#pragma unroll
        for (int i = 0; i < D / 64; ++i) {
            const int db = w + 4 * i;
            const int dr = 16 * db + l16;
            f32x4 acc = {0.f, 0.f, 0.f, 0.f};
            for (int ks = 0; ks < S / 32; ++ks) {
                const u32x4 a = Vt[dr * SC + ((4 * ks + q4) ^ (dr & swm))];
                const u32x4 bb = Pl[l16 * SC + ((4 * ks + q4) ^ (l16 & swm))];
                acc = mfma_16x16x32(a, bb, acc);
            }
            if (l16 < G) {
                const u32x2 o2 = {pack_bf16x2(acc[0], acc[1]), pack_bf16x2(acc[2], acc[3])};
                *reinterpret_cast<u32x2*>(O + (((size_t)b * p.T + u) * p.H_q + hq) * D + 16 * db + 4 * q4) = o2;
            }
        }
        __syncthreads();   // V^T and P are rewritten for the next KV head
    }
}

// Two neighbouring positions per workgroup (grouped-query heads G <= 8, sets
// of up to 128 keys): u0 = 2 * item and u0 + 1 attend over the union of
// their two sets, each key gathered once, with a per-position membership
// mask.  The 2G query heads of the pair are the B columns of the score
// product (16 columns), so the two positions share every gathered K and V row
// and every MFMA.  Column c < 2G is position pp = c / G, head c % G.
//
// The union: when both sets are ascending with their -1 padding at the end
// (what the Top-S selection writes), it is set 0 followed by the keys of set 1
// that set 0 lacks (binary search), and a key of set 0 belongs to position 1
// if set 1 holds it.  When the union exceeds kPairKeys keys, or a set is not
// ascending (unordered, duplicates), the workgroup makes two passes instead,
// one per position over that position's set as listed, and stores only that
// position's columns.  A position attends to the entries of its bit that lie
// in 0 .. u0 + pp.
//
// grid (xcd_grid(ceil(T / 2)), B), 256 threads
constexpr int kPairKeys = 192;   // largest union one pass takes (register arrays and LDS are sized for it)

template <int D>
__global__ __launch_bounds__(256, 2) void k_sparse_attn_pair(ReplayProblem p) {
    constexpr int SMAX = 128, UMAX = kPairKeys, DC = D / 8;
    __shared__ u32x4 s_lds[(D * UMAX + 16 * UMAX) / 8];
    __shared__ float red[128];
    __shared__ int s_set[2][SMAX];
    __shared__ int s_keys[UMAX];
    __shared__ int s_mask[UMAX];
    __shared__ int s_cnt[2];
    const int npair = (p.T + 1) / 2;
    const int item = xcd_item(blockIdx.x, npair), b = blockIdx.y;
    if (item >= npair) return;   // uniform over the workgroup
    const int u0 = 2 * item;
    const bool has1 = u0 + 1 < p.T;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, l16 = lane & 15, q4 = lane >> 4;
    const int S = p.S, G = p.H_q / p.H_kv;
    const uint16_t* Q = reinterpret_cast<const uint16_t*>(p.q);
    const uint16_t* K = reinterpret_cast<const uint16_t*>(p.k);
    const uint16_t* V = reinterpret_cast<const uint16_t*>(p.v);
    uint16_t* O = reinterpret_cast<uint16_t*>(p.o);
    const float sl2 = kLog2e / sqrtf((float)D);
    const u32x4 zero = {0u, 0u, 0u, 0u};

    // ---- the two sets, then their union with membership bits
    if (tid < 2 * S) {
        const int pp = tid / S, e = tid % S;
        s_set[pp][e] = pp == 0 || has1 ? p.idx[((size_t)b * p.T + u0 + pp) * S + e] : -1;
    }
    __syncthreads();
    bool bad = false;
    if (tid < 2 * S) {
        const int pp = tid / S, e = tid % S, v = s_set[pp][e], nx = e + 1 < S ? s_set[pp][e + 1] : -1;
        bad = (v < 0 && nx >= 0) || (v >= 0 && nx >= 0 && nx <= v) || v < -1;
    }
    const bool ordered = !__syncthreads_or(bad);
    // nonnegative prefix lengths of the two sets
    const int n0 = __syncthreads_count(tid < S && s_set[0][tid] >= 0);
    const int n1 = __syncthreads_count(tid < S && s_set[1][tid] >= 0);
    // union (one pass) when ordered and small enough; ext = set 1's extra keys
    bool extra = false;
    int v1 = -1;
    if (ordered && tid < S) {
        auto find = [&](const int* set, int n, int v) {
            int lo = 0, hi = n;   // first index with set[i] >= v
            while (lo < hi) {
                const int mid = (lo + hi) >> 1;
                if (set[mid] < v) lo = mid + 1;
                else hi = mid;
            }
            return lo < n && set[lo] == v;
        };
        v1 = s_set[1][tid];
        extra = tid < n1 && !find(s_set[0], n0, v1);
        if (tid < n0) {
            const int v0 = s_set[0][tid];
            s_keys[tid] = v0;
            s_mask[tid] = 1 | (find(s_set[1], n1, v0) ? 2 : 0);
        }
    }
    const unsigned long long bal = __ballot(extra);
    if (lane == 0 && w < 2) s_cnt[w] = __popcll(bal);
    __syncthreads();
    const int n_union = n0 + s_cnt[0] + s_cnt[1];
    const bool one_pass = ordered && n_union <= UMAX;
    if (one_pass && extra) {
        const int pos = n0 + (w == 1 ? s_cnt[0] : 0) + __popcll(bal & ((1ull << lane) - 1ull));
        s_keys[pos] = v1;
        s_mask[pos] = 2;
    }
    // B column of this lane: position pp, head hh (kv head kvh*G + hh)
    const int pp = l16 / G, hh = l16 - pp * G;
    const bool col_ok = l16 < 2 * G && (pp == 0 || has1);
    for (int pass = 0; pass < (one_pass ? 1 : (has1 ? 2 : 1)); ++pass) {
    // keys of this pass: the union, or set `pass` as listed
    int U;
    if (one_pass) {
        U = n_union;
    } else {
        __syncthreads();   // the previous pass has finished with s_keys
        if (tid < S) {
            s_keys[tid] = s_set[pass][tid];
            s_mask[tid] = 1 << pass;
        }
        U = S;
    }
    // the positions whose columns this pass stores
    const int store_mask = one_pass ? 3 : 1 << pass;
    const int UP = U < 32 ? 32 : (U + 31) / 32 * 32;   // rounded up to whole 32-key steps
    for (int e = U + tid; e < UP; e += 256) {
        s_keys[e] = -1;
        s_mask[e] = 0;
    }
    __syncthreads();

    const int SC = UP / 8, KB = UP / 16;
    const int swm = replay_swizzle_mask(SC);
    u32x4* Vt = s_lds;                      // row d: SC chunks, chunk c at (c ^ (d & swm))
    u32x4* Pl = s_lds + D * SC;             // row = B column
    // a key is gathered when some position may attend it
    auto gather_ok = [&](int kv) { return kv >= 0 && kv <= u0 + (has1 ? 1 : 0); };
    constexpr int MAXR = replay_sparse_v_items(D, UMAX);
    constexpr int MAXB = replay_sparse_key_blocks(UMAX);

    for (int kvh = 0; kvh < p.H_kv; ++kvh) {
        u32x4 va[MAXR], vc[MAXR];
#pragma unroll
        for (int r = 0; r < MAXR; ++r) {
            const int it = tid + 256 * r;
            va[r] = zero;
            vc[r] = zero;
            if (it < (UP / 2) * DC) {
                const int pr = it % (UP / 2), dc = it / (UP / 2), k0 = 2 * pr;
                const int v0 = s_keys[k0], v1 = s_keys[k0 + 1];
                if (gather_ok(v0)) va[r] = *reinterpret_cast<const u32x4*>(V + kv_row(p, b, v0, kvh) + 8 * dc);
                if (gather_ok(v1)) vc[r] = *reinterpret_cast<const u32x4*>(V + kv_row(p, b, v1, kvh) + 8 * dc);
            }
        }
        u32x4 ka[MAXB][D / 32];
#pragma unroll
        for (int i = 0; i < MAXB; ++i) {
            const int kb = w + 4 * i;
            const int kr = kb < KB ? s_keys[kb * 16 + l16] : -1;
            const uint16_t* krow = K + (gather_ok(kr) ? kv_row(p, b, kr, kvh) : 0);
#pragma unroll
            for (int ks = 0; ks < D / 32; ++ks)
                ka[i][ks] = gather_ok(kr) ? *reinterpret_cast<const u32x4*>(krow + 32 * ks + 8 * q4) : zero;
        }
        const size_t qrow = (((size_t)b * p.T + u0 + pp) * p.H_q + kvh * G + hh) * D;
        u32x4 qop[D / 32];
#pragma unroll
        for (int ks = 0; ks < D / 32; ++ks)
            qop[ks] = col_ok ? *reinterpret_cast<const u32x4*>(Q + qrow + 32 * ks + 8 * q4) : zero;
        // V^T of the union into LDS
        uint32_t* Vw = reinterpret_cast<uint32_t*>(Vt);
#pragma unroll
        for (int r = 0; r < MAXR; ++r) {
            const int it = tid + 256 * r;
            if (it < (UP / 2) * DC) {
                const int pr = it % (UP / 2), dc = it / (UP / 2), k0 = 2 * pr;
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    const int d = 8 * dc + i;
                    Vw[(d * SC + ((k0 >> 3) ^ (d & swm))) * 4 + ((k0 & 7) >> 1)] = pair_word(va[r], vc[r], i);
                }
            }
        }
        // scores^T[key][column], masked per column to its position's entries
        f32x4 sc[MAXB];
        float mx = -INFINITY;
#pragma unroll
        for (int i = 0; i < MAXB; ++i) {
            const int kb = w + 4 * i;
            sc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
            if (kb < KB) {
#pragma unroll
                for (int ks = 0; ks < D / 32; ++ks) sc[i] = mfma_16x16x32(ka[i][ks], qop[ks], sc[i]);
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int e = kb * 16 + 4 * q4 + j, kv = s_keys[e];
                    const bool ok = col_ok && kv >= 0 && kv <= u0 + pp && ((s_mask[e] >> pp) & 1);
                    sc[i][j] = ok ? sc[i][j] : -INFINITY;
                    mx = fmaxf(mx, sc[i][j]);
                }
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j) sc[i][j] = -INFINITY;
            }
        }
        // softmax over the union, per column (lane column l16)
        mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
        mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
        if (q4 == 0) red[w * 16 + l16] = mx;
        __syncthreads();
        mx = fmaxf(fmaxf(red[l16], red[16 + l16]), fmaxf(red[32 + l16], red[48 + l16]));
        float sum = 0.f;
#pragma unroll
        for (int i = 0; i < MAXB; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const float e = sc[i][j] == -INFINITY ? 0.f : exp2f((sc[i][j] - mx) * sl2);
                sc[i][j] = e;
                sum += e;
            }
        sum += __shfl_xor(sum, 16, 64);
        sum += __shfl_xor(sum, 32, 64);
        __syncthreads();   // every wave has read the maxima
        if (q4 == 0) red[w * 16 + l16] = sum;
        __syncthreads();
        sum = red[l16] + red[16 + l16] + red[32 + l16] + red[48 + l16];
        const float inv = sum > 0.f ? 1.0f / sum : 0.f;
        uint32_t* Pw = reinterpret_cast<uint32_t*>(Pl);
#pragma unroll
        for (int i = 0; i < MAXB; ++i) {
            const int kb = w + 4 * i;
            if (kb < KB) {
                const int ch = (2 * kb + (q4 >> 1)) ^ (l16 & swm);
                const int base = (l16 * SC + ch) * 4 + 2 * (q4 & 1);
                Pw[base] = pack_bf16x2(sc[i][0] * inv, sc[i][1] * inv);
                Pw[base + 1] = pack_bf16x2(sc[i][2] * inv, sc[i][3] * inv);
            }
        }
        __syncthreads();
        // O^T[d][column] = V_union^T . P^T, d blocks db = w, w+4, ...
#pragma unroll
        for (int i = 0; i < D / 64; ++i) {
            const int db = w + 4 * i;
            const int dr = 16 * db + l16;
            f32x4 acc = {0.f, 0.f, 0.f, 0.f};
            for (int ks = 0; ks < UP / 32; ++ks) {
                const u32x4 a = Vt[dr * SC + ((4 * ks + q4) ^ (dr & swm))];
                const u32x4 bb = Pl[l16 * SC + ((4 * ks + q4) ^ (l16 & swm))];
                acc = mfma_16x16x32(a, bb, acc);
            }
            if (col_ok && ((store_mask >> pp) & 1)) {
                const u32x2 o2 = {pack_bf16x2(acc[0], acc[1]), pack_bf16x2(acc[2], acc[3])};
                *reinterpret_cast<u32x2*>(O + qrow + 16 * db + 4 * q4) = o2;
            }
        }
        __syncthreads();   // V^T and P are rewritten for the next KV head
    }
    }   // pass
}

// V transposed for the causal kernel: vt[b][kvh][d][t] (t < replay_tpad(T),
// zero past T).  grid (replay_tpad(T) / 64, H_kv, B), 256 threads: one
// 64-key chunk through LDS (rows padded by 8 elements against bank conflicts).
template <int D>
__global__ __launch_bounds__(256) void k_transpose_v(ReplayProblem p) {
    constexpr int DC = D / 8;
    __shared__ __align__(16) uint16_t tl[64][D + 8];
    const int t0 = blockIdx.x * 64, kvh = blockIdx.y, b = blockIdx.z, tid = threadIdx.x;
    const uint16_t* V = reinterpret_cast<const uint16_t*>(p.v);
    const u32x4 zero = {0u, 0u, 0u, 0u};
    for (int it = tid; it < 64 * DC; it += 256) {
        const int kr = it / DC, c = it % DC, t = t0 + kr;
        const u32x4 x = t < p.T ? *reinterpret_cast<const u32x4*>(V + kv_row(p, b, t, kvh) + 8 * c) : zero;
        *reinterpret_cast<u32x4*>(&tl[kr][8 * c]) = x;
    }
    __syncthreads();
    const int64_t tpad = replay_tpad(p.T);
    uint16_t* out = p.vt + ((size_t)b * p.H_kv + kvh) * D * tpad + t0;
    // chunk c of a row holds keys 16 (c / 2) + 4 (c % 2) + {0..3} and the
    // same + 8: the order in which a 32x32 score block's accumulators hold
    // them, so the causal kernel's P . V operands pair up without a shuffle
    for (int it = tid; it < D * 8; it += 256) {
        const int d = it >> 3, c = it & 7, k0 = 16 * (c >> 1) + 4 * (c & 1);
        u32x4 w;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int k = k0 + (j < 2 ? 2 * j : 8 + 2 * (j - 2));
            w[j] = (uint32_t)tl[k][d] | ((uint32_t)tl[k + 1][d] << 16);
        }
        *reinterpret_cast<u32x4*>(out + (size_t)d * tpad + 8 * c) = w;
    }
}

// grid xcd_grid(npairs * H_q * B) with npairs = ceil(ceil(T/128) / 2), items
// ordered (pair, head, batch row) pair fastest; 256 threads: query positions
// u0 + 32w + l32 of head hq for two query tiles of 128 (a short and a long
// one); 64-key chunks up to the tile's last position.
//
// Per wave and chunk, on v_mfma_f32_32x32x16_bf16: scores^T[key][position]
// for two 32-key blocks (A = K rows from LDS, B = the wave's 32 query rows,
// held in registers), an online softmax per position (column), and
// O^T[d][position] += V^T . P^T with A = V^T rows from LDS and B = the
// probabilities straight from the score accumulators: a lane's accumulator
// holds keys 8i + 4g + {0..3} of its position, and the staged V^T rows keep
// each 16-key group in the matching order (keys 0-3, 8-11, 4-7, 12-15), so k
// step s of the product takes accumulator elements 8 (s % 2) .. +7 of block
// s / 2 as its B operand.  LDS: K chunk [64][D], V^T chunk [D][64] (bf16).
template <int D>
__device__ __forceinline__ int causal_kswz(int r) {   // K rows: D/8 chunks
    return D == 128 ? (r & 15) : ((r >> 1) & 7);
}

template <int D>
__global__ __launch_bounds__(256, 2) void k_causal_attn(ReplayProblem p) {
    constexpr int DC = D / 8;
    constexpr int KS = 64 * DC, VS = D * 8;   // 16-byte slots of a K chunk and a V^T chunk
    // two stages, each: K chunk rows (key: chunk c at c ^ causal_kswz(key)),
    // then V^T rows (d: chunk c at c ^ ((d >> 1) & 7)); filled straight from
    // global memory (buffer loads into LDS) one chunk ahead
    __shared__ u32x4 lds[2 * (KS + VS)];
    // workgroup x runs query tile x and tile ntiles-1-x: every workgroup
    // walks about the same number of key chunks
    const int ntiles = (p.T + 127) / 128, npairs = (ntiles + 1) / 2;
    const int item = xcd_item(blockIdx.x, npairs * p.H_q * p.B);
    if (item >= npairs * p.H_q * p.B) return;   // uniform over the workgroup
    const int px = item % npairs, hq = (item / npairs) % p.H_q, b = item / (npairs * p.H_q);
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, l32 = lane & 31, g = lane >> 5;
    const int G = p.H_q / p.H_kv, kvh = hq / G;
    const uint16_t* Q = reinterpret_cast<const uint16_t*>(p.q);
    uint16_t* O = reinterpret_cast<uint16_t*>(p.o);
    const float sl2 = kLog2e / sqrtf((float)D);
    const u32x4 zero = {0u, 0u, 0u, 0u};
    const int64_t tpad = replay_tpad(p.T);
    // key t of this batch row and KV head sits at row t * ts of the K buffer;
    // the host admits only shapes whose byte offsets (up to (T + 64) * ts * 2)
    // fit in 31 bits; rows past T lie past the descriptor's range and read as zero
    const uint32_t ts = p.kv_layout == MOT_LAYOUT_BTHD ? (uint32_t)(p.H_kv * D) : (uint32_t)D;
    const rsrc_t kbuf = make_rsrc(reinterpret_cast<const uint16_t*>(p.k) + kv_row(p, b, 0, kvh),
                                  ((size_t)(p.T - 1) * ts + D) * 2);
    const rsrc_t vbuf = make_rsrc(p.vt + ((size_t)b * p.H_kv + kvh) * D * tpad, (size_t)D * tpad * 2);
    // this lane's part of the chunk loads: wave load q fills slots
    // (w * NQ + q) * 64 + lane of the K rows (NQ = KS / 256 loads), then of
    // the V^T rows
    constexpr int NQK = KS / 256, NQV = VS / 256;
    uint32_t koff[NQK], voff[NQV];
#pragma unroll
    for (int q = 0; q < NQK; ++q) {
        const int slot = (w * NQK + q) * 64 + lane, kr = slot / DC, c = (slot % DC) ^ causal_kswz<D>(kr);
        koff[q] = ((uint32_t)kr * ts + 8 * c) * 2;
    }
#pragma unroll
    for (int q = 0; q < NQV; ++q) {
        const int slot = (w * NQV + q) * 64 + lane, d = slot >> 3, c = (slot & 7) ^ ((d >> 1) & 7);
        voff[q] = ((uint32_t)d * tpad + 8 * c) * 2;
    }
    auto issue = [&](int kc0, int st) {
        u32x4* kb = lds + st * (KS + VS) + w * NQK * 64;
        u32x4* vb = lds + st * (KS + VS) + KS + w * NQV * 64;
#pragma unroll
        for (int q = 0; q < NQK; ++q) load_lds16(kbuf, koff[q] + (uint32_t)kc0 * ts * 2, kb + q * 64);
#pragma unroll
        for (int q = 0; q < NQV; ++q) load_lds16(vbuf, voff[q] + (uint32_t)kc0 * 2, vb + q * 64);
    };
    auto barrier = [&]() {
        __builtin_amdgcn_s_waitcnt(0x70);   // vmcnt(0) lgkmcnt(0)
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
    };
    for (int pass = 0; pass < 2; ++pass) {
    const int tile = pass == 0 ? px : ntiles - 1 - px;
    if (pass == 1 && tile <= px) break;   // uniform over the workgroup
    const int u0 = tile * 128;
    const int uw = u0 + 32 * w;            // first position of this wave
    const int u = uw + l32;                // this lane's query column
    u32x4 qop[D / 16];                     // k step s: d = 16 s + 8 g .. +7
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks)
        qop[ks] = u < p.T ? *reinterpret_cast<const u32x4*>(Q + (((size_t)b * p.T + u) * p.H_q + hq) * D + 16 * ks + 8 * g)
                          : zero;
    f32x16 acc[D / 32];
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[db][e] = 0.f;
    float m = -INFINITY, l = 0.f;
    const int last = (u0 + 127 < p.T ? u0 + 127 : p.T - 1);
    barrier();   // the previous tile's last chunk is consumed
    issue(0, 0);
    barrier();
    for (int kc0 = 0; kc0 <= last; kc0 += 64) {
        const int st = (kc0 >> 6) & 1;
        if (kc0 + 64 <= last) issue(kc0 + 64, st ^ 1);
        const u32x4* Kl = lds + st * (KS + VS);
        const u32x4* Vt = Kl + KS;
        // keys after every position of this wave add nothing (uniform)
        if (kc0 <= uw + 31 && uw < p.T) {
        // scores^T[key][position], two blocks of 32 keys; only chunks that
        // reach past the wave's first position need the mask
        const bool diag = kc0 + 63 > uw;
        f32x16 sc[2];
        float cm = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
            for (int e = 0; e < 16; ++e) sc[kb][e] = 0.f;
            const int kr = kb * 32 + l32;
#pragma unroll
            for (int ks = 0; ks < D / 16; ++ks)
                sc[kb] = mfma_32x32x16(Kl[kr * DC + ((2 * ks + g) ^ causal_kswz<D>(kr))], qop[ks], sc[kb]);
            if (diag) {
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int key = kc0 + kb * 32 + 8 * (e >> 2) + 4 * g + (e & 3);
                    sc[kb][e] = key <= u ? sc[kb][e] : -INFINITY;
                }
            }
#pragma unroll
            for (int e = 0; e < 16; ++e) cm = fmaxf(cm, sc[kb][e]);
        }
        cm = fmaxf(cm, __shfl_xor(cm, 32, 64));
        const float mn = fmaxf(m, cm);   // finite: chunk 0 holds key 0 <= u
        // v_exp_f32 directly: results below 2^-126 flush to 0, far below the
        // bf16 resolution of P; exp2(-inf) = 0 for masked keys and the first chunk
        const float alpha = __builtin_amdgcn_exp2f((m - mn) * sl2);
        const float mo = mn * sl2;       // e = 2^(s sl2 - mn sl2)
        float rs = 0.f;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const float ex = __builtin_amdgcn_exp2f(fmaf(sc[kb][e], sl2, -mo));
                sc[kb][e] = ex;
                rs += ex;
            }
        rs += __shfl_xor(rs, 32, 64);
        l = l * alpha + rs;
        // alpha is exactly 1 where the running maximum did not move: the
        // accumulators are rescaled only when some position's maximum rose
        if (__builtin_amdgcn_ballot_w64(mn != m)) {
#pragma unroll
            for (int db = 0; db < D / 32; ++db)
#pragma unroll
                for (int e = 0; e < 16; ++e) acc[db][e] *= alpha;
        }
        m = mn;
        // O^T[d][position] += V^T . P^T, four k steps of 16 keys
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            const int kb = ks >> 1, e0 = 8 * (ks & 1);
            const u32x4 pf = {pack_bf16x2(sc[kb][e0], sc[kb][e0 + 1]), pack_bf16x2(sc[kb][e0 + 2], sc[kb][e0 + 3]),
                              pack_bf16x2(sc[kb][e0 + 4], sc[kb][e0 + 5]), pack_bf16x2(sc[kb][e0 + 6], sc[kb][e0 + 7])};
#pragma unroll
            for (int db = 0; db < D / 32; ++db) {
                const int dr = 32 * db + l32;
                acc[db] = mfma_32x32x16(Vt[dr * 8 + ((2 * ks + g) ^ ((dr >> 1) & 7))], pf, acc[db]);
            }
        }
        }
        barrier();   // stage st^1 has landed; every wave is done with stage st
    }
    // lane holds d = 32 db + 8 i + 4 g + {0..3} of position u
    if (u < p.T) {
        const float inv = 1.0f / l;
#pragma unroll
        for (int db = 0; db < D / 32; ++db)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const u32x2 o2 = {pack_bf16x2(acc[db][4 * i] * inv, acc[db][4 * i + 1] * inv),
                                  pack_bf16x2(acc[db][4 * i + 2] * inv, acc[db][4 * i + 3] * inv)};
                *reinterpret_cast<u32x2*>(O + (((size_t)b * p.T + u) * p.H_q + hq) * D + 32 * db + 8 * i + 4 * g) = o2;
            }
    }
    }
}

constexpr int kSelCacheMax = 15872;   // rows up to this length keep their keys in LDS (<= 64 KB with the counts)

}  // namespace

hipError_t launch_topS_select(const float* A, int32_t* idx, int B, int T, int S, hipStream_t stream) {
    if (B == 0 || T == 0) return hipSuccess;
    const dim3 grid(T, B);
    const size_t counts = (size_t)2 * ((T >> 6) + 1) * 4;
    if (T <= kSelCacheMax)
        hipLaunchKernelGGL(k_topS_select<true>, grid, dim3(256), (size_t)T * 4 + counts, stream, A, idx, T, S);
    else
        hipLaunchKernelGGL(k_topS_select<false>, grid, dim3(256), counts, stream, A, idx, T, S);
    return hipGetLastError();
}

hipError_t launch_replay_attention(const ReplayProblem& p, hipStream_t stream) {
    if (p.B == 0 || p.T == 0) return hipSuccess;
    if (p.idx) {
        // the caller's check admits only these sizes; the register arrays of
        // the instantiation below cover every admitted S
        if (!replay_sparse_supported(p.D, p.S)) return hipErrorInvalidValue;
        if (replay_sparse_pair_supported(p.D, p.S, p.H_q / p.H_kv)) {
            const dim3 pgrid(xcd_grid((p.T + 1) / 2), p.B);
            if (p.D == 128) hipLaunchKernelGGL(k_sparse_attn_pair<128>, pgrid, dim3(256), 0, stream, p);
            else hipLaunchKernelGGL(k_sparse_attn_pair<64>, pgrid, dim3(256), 0, stream, p);
            return hipGetLastError();
        }
        const dim3 grid(xcd_grid(p.T), p.B);
        const size_t lds = replay_sparse_lds_bytes(p.D, p.S);
        // register arrays sized for S <= 128, or for the largest S the LDS allows
        if (p.D == 128) {
            if (replay_sparse_instance(128, p.S) == 128)
                hipLaunchKernelGGL((k_sparse_attn<128, 128>), grid, dim3(256), lds, stream, p);
            else hipLaunchKernelGGL((k_sparse_attn<128, replay_sparse_smax(128)>), grid, dim3(256), lds, stream, p);
        } else {
            if (replay_sparse_instance(64, p.S) == 128)
                hipLaunchKernelGGL((k_sparse_attn<64, 128>), grid, dim3(256), lds, stream, p);
            else hipLaunchKernelGGL((k_sparse_attn<64, replay_sparse_smax(64)>), grid, dim3(256), lds, stream, p);
        }
    } else {
        if (!p.vt || !replay_causal_supported(p.T, p.H_kv, p.D, p.kv_layout == MOT_LAYOUT_BTHD))
            return hipErrorInvalidValue;
        const dim3 tgrid((unsigned)(replay_tpad(p.T) / 64), p.H_kv, p.B);
        if (p.D == 128) hipLaunchKernelGGL(k_transpose_v<128>, tgrid, dim3(256), 0, stream, p);
        else hipLaunchKernelGGL(k_transpose_v<64>, tgrid, dim3(256), 0, stream, p);
        const int npairs = ((p.T + 127) / 128 + 1) / 2;
        const dim3 grid(xcd_grid(npairs * p.H_q * p.B));
        if (p.D == 128) hipLaunchKernelGGL(k_causal_attn<128>, grid, dim3(256), 0, stream, p);
        else hipLaunchKernelGGL(k_causal_attn<64>, grid, dim3(256), 0, stream, p);
    }
    return hipGetLastError();
}

}  // namespace mot
