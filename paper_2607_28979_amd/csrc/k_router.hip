// Router GEMV + softmax: gates[unit][token][m] = softmax_m(Wr_unit z + br_unit),
// then Top-K: the top_k largest kept and renormalised, the rest zero.
// Paper Sec. 3, Definition "Mixture-of-Translators": token-level nonnegative
// gate scores; here softmax of a linear map of the source row.
//
// Eight lanes share one token row: lane q reads 16-byte chunks q, q+8, ...
// (coalesced 128-byte runs), accumulates E partial dot products in fp32, and
// the eight partials are combined with cross-lane shuffles.  256 threads =
// 32 tokens per pass, 8 passes per workgroup; grid.y enumerates the units.
#include "mot_device.h"
#include "mot_internal.h"
#include "../../include/mot.h"

namespace mot {

namespace {

constexpr int kLanesPerTok = 8;
constexpr int kTokPerBlock = 256 / kLanesPerTok;   // tokens per pass of a workgroup
constexpr int kGroups = 8;                          // passes per workgroup

template <bool BF16>
struct Vec;
template <>
struct Vec<true> {  // 8 bf16 per 16-byte chunk
    static constexpr int n = 8;
    __device__ static float scalar(const void* base, size_t elem) {
        return bf16_to_f32(reinterpret_cast<const uint16_t*>(base)[elem]);
    }
    typedef u32x4 Raw;
    __device__ static Raw raw(const void* base, size_t elem) {
        return *reinterpret_cast<const u32x4*>(reinterpret_cast<const uint16_t*>(base) + elem);
    }
    // acc + w . z over the 8 values, on packed bf16 dot products (exact
    // products, fp32 sums)
    __device__ static float dot2(uint32_t w, uint32_t z, float acc) {
        return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w), __builtin_bit_cast(bf16x2, z), acc,
                                               false);
    }
    __device__ static float dot(Raw w, Raw z, float acc) {
        acc = dot2(w.x, z.x, acc);
        acc = dot2(w.y, z.y, acc);
        acc = dot2(w.z, z.z, acc);
        return dot2(w.w, z.w, acc);
    }
};
template <>
struct Vec<false> {  // 4 fp32 per 16-byte chunk
    static constexpr int n = 4;
    __device__ static float scalar(const void* base, size_t elem) {
        return reinterpret_cast<const float*>(base)[elem];
    }
    typedef f32x4 Raw;
    __device__ static Raw raw(const void* base, size_t elem) {
        return *reinterpret_cast<const f32x4*>(reinterpret_cast<const float*>(base) + elem);
    }
    __device__ static float dot(const Raw& w, const Raw& z, float acc) {
#pragma unroll
        for (int e = 0; e < 4; ++e) acc = fmaf(w[e], z[e], acc);
        return acc;
    }
};

// LISTS = false: dense gate rows p.gates[gslot][token][E] (zeros outside the
// Top-K set); LISTS = true: the Top-K lists p.rt.sel / p.rt.gk of the routed path.
// WLDS: the unit's router rows (E x d_in) are staged once in LDS (dynamic
// shared memory, when they fit) instead of being re-read per token.
template <bool BF16, bool LISTS, bool WLDS>
__global__ __launch_bounds__(256) void k_router(Problem p, UnitTab ut) {
    using V = Vec<BF16>;
    extern __shared__ u32x4 s_wr[];
    const uint32_t code = ut.code[blockIdx.y];
    const int j = unit_j(code), x = unit_x(code), i = unit_i(code), gs = unit_gslot(code);
    const int q = threadIdx.x % kLanesPerTok;
    const void* wr = p.wr;
    size_t wr_base = ((size_t)j * p.streams + x) * p.E * p.d_in;
    if constexpr (WLDS) {
        const int n16 = p.E * p.d_in / V::n;   // 16-byte chunks
        const u32x4* g = reinterpret_cast<const u32x4*>(reinterpret_cast<const char*>(p.wr) +
                                                        wr_base * (BF16 ? 2 : 4));
        for (int c = threadIdx.x; c < n16; c += 256) s_wr[c] = g[c];
        __syncthreads();
        wr = s_wr;
        wr_base = 0;
    }
    for (int grp = 0; grp < kGroups; ++grp) {
    const int tok = (blockIdx.x * kGroups + grp) * kTokPerBlock + threadIdx.x / kLanesPerTok;
    // the gate rows of the last partial pass are still written by lanes q == 0
    // of valid tokens only; the usage count needs every lane of the wave
    const bool owner = tok < p.n_tok && q == 0;
    const int E = p.E, d_in = p.d_in;
    const size_t unit = (size_t)j * p.streams + x;

    float acc[MOT_MAX_EXPERTS];
#pragma unroll
    for (int m = 0; m < MOT_MAX_EXPERTS; ++m) acc[m] = 0.f;

    if (tok < p.n_tok) {
        const size_t layer = (size_t)i * p.n_tok * d_in;
        const int b = tok / p.T, t = tok % p.T;
        // four 16-byte source chunks in flight per lane before they are used
        constexpr int kStep = kLanesPerTok * V::n;
        for (int c0 = q * V::n; c0 < d_in; c0 += 4 * kStep) {
            typename V::Raw zr[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int c = c0 + u * kStep;
                const int cc = c < d_in ? c : c0;   // in range; unused when c >= d_in
                size_t off;
                if (p.src_layout == MOT_LAYOUT_BTHD) {
                    off = layer + (size_t)tok * d_in + cc;
                } else {
                    const int hh = cc / p.D_src, dd = cc % p.D_src;
                    off = layer + (((size_t)b * p.H_src + hh) * p.T + t) * p.D_src + dd;
                }
                zr[u] = V::raw(p.src[x], off);
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int c = c0 + u * kStep;
                if (c < d_in) {
#pragma unroll
                    for (int m = 0; m < MOT_MAX_EXPERTS; ++m)
                        if (m < E) acc[m] = V::dot(V::raw(wr, wr_base + (size_t)m * d_in + c), zr[u], acc[m]);
                }
            }
        }
    }
    // combine the eight partial sums of each token (lanes of a token are
    // consecutive and aligned to 8)
#pragma unroll
    for (int m = 0; m < MOT_MAX_EXPERTS; ++m) {
        if (m < E) {
            float v = acc[m];
            v += __shfl_xor(v, 1, 64);
            v += __shfl_xor(v, 2, 64);
            v += __shfl_xor(v, 4, 64);
            acc[m] = v;
        }
    }
    // every lane runs the softmax and the selection (lanes without a token
    // work on zeros and write nothing), so the wave can count selections
    float mx = -INFINITY;
#pragma unroll
    for (int m = 0; m < MOT_MAX_EXPERTS; ++m) {
        if (m < E) {
            if (p.br) acc[m] += V::scalar(p.br, unit * E + m);
            mx = fmaxf(mx, acc[m]);
        }
    }
    float den = 0.f;
#pragma unroll
    for (int m = 0; m < MOT_MAX_EXPERTS; ++m) {
        if (m < E) {
            acc[m] = expf(acc[m] - mx);
            den += acc[m];
        }
    }
    const float inv = 1.0f / den;
#pragma unroll
    for (int m = 0; m < MOT_MAX_EXPERTS; ++m) acc[m] = m < E ? acc[m] * inv : 0.f;
    if constexpr (LISTS) {
        // the routed path counts usage in its plan kernel
        if (!owner) continue;
        const size_t base = ((size_t)gs * p.n_tok + tok) * p.top_k;
        topk_list(acc, E, p.top_k, p.rt.sel + base, p.rt.gk + base);
        continue;
    }
    const uint32_t taken = topk_renormalise(acc, E, p.top_k);
    if (p.usage) count_usage(p.usage + unit * E, E, taken, owner);
    if (!owner) continue;
    float* g = p.gates + ((size_t)gs * p.n_tok_pad + tok) * E;
#pragma unroll
    for (int m = 0; m < MOT_MAX_EXPERTS; ++m)
        if (m < E) g[m] = acc[m];
    }
}

// Translator usage statistics (paper Sec. 4, "MoT Architecture Ablation"),
// one thread per row of counts I[E]: CV^2 = population variance over the
// squared mean, entropy = -sum p ln p with p = I / sum I (0 ln 0 = 0), in
// double; NaN for a row of zeros.
__global__ __launch_bounds__(256) void k_usage_stats(const uint32_t* counts, int n, int E, double* cv2,
                                                     double* entropy) {
    const int r = blockIdx.x * 256 + threadIdx.x;
    if (r >= n) return;
    const uint32_t* c = counts + (size_t)r * E;
    double total = 0.0;
    for (int m = 0; m < E; ++m) total += (double)c[m];
    const double mean = total / E;
    double var = 0.0;
    for (int m = 0; m < E; ++m) var += ((double)c[m] - mean) * ((double)c[m] - mean);
    var /= E;
    cv2[r] = var / (mean * mean);
    double h = 0.0;
    for (int m = 0; m < E; ++m) {
        if (c[m] == 0) continue;
        const double q = (double)c[m] / total;
        h -= q * log(q);
    }
    entropy[r] = total > 0.0 ? h : __builtin_nan("");
}

constexpr size_t kWrLdsMax = 64 * 1024;   // router rows staged in LDS up to this size

template <bool BF16, bool LISTS>
hipError_t launch_k(const Problem& p, const UnitTab& ut, hipStream_t stream) {
    if (ut.n == 0 || p.n_tok == 0) return hipSuccess;
    dim3 grid((p.n_tok + kTokPerBlock * kGroups - 1) / (kTokPerBlock * kGroups), ut.n);
    const size_t wr_bytes = (size_t)p.E * p.d_in * (BF16 ? 2 : 4);
    if (wr_bytes <= kWrLdsMax)
        hipLaunchKernelGGL((k_router<BF16, LISTS, true>), grid, dim3(256), wr_bytes, stream, p, ut);
    else
        hipLaunchKernelGGL((k_router<BF16, LISTS, false>), grid, dim3(256), 0, stream, p, ut);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_router(const Problem& p, const UnitTab& ut, bool bf16, hipStream_t stream) {
    return bf16 ? launch_k<true, false>(p, ut, stream) : launch_k<false, false>(p, ut, stream);
}

hipError_t launch_router_lists(const Problem& p, const UnitTab& ut, hipStream_t stream) {
    return launch_k<true, true>(p, ut, stream);
}

hipError_t launch_usage_stats(const uint32_t* counts, int n, int E, double* cv2, double* entropy,
                              hipStream_t stream) {
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(k_usage_stats, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, counts, n, E, cv2,
                       entropy);
    return hipGetLastError();
}

}  // namespace mot
