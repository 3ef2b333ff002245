// Router GEMV + softmax: gates[unit][token][m] = softmax_m(Wr_unit z + br_unit),
// then Top-K: the top_k largest kept and renormalised, the rest zero.
// Paper Sec. 3, Definition "Mixture-of-Translators": token-level nonnegative
// gate scores; here softmax of a linear map of the source row.
//
// Eight lanes share one token row: lane q reads 16-byte chunks q, q+8, ...
// (coalesced 128-byte runs), accumulates E partial dot products in fp32, and
// the eight partials are combined with cross-lane shuffles.  256 threads =
// 32 tokens per workgroup; grid.y enumerates the units.
#include "mot_device.h"
#include "mot_internal.h"
#include "../../include/mot.h"

namespace mot {

namespace {

constexpr int kLanesPerTok = 8;
constexpr int kTokPerBlock = 256 / kLanesPerTok;

template <bool BF16>
struct Vec;
template <>
struct Vec<true> {  // 8 bf16 per 16-byte chunk
    static constexpr int n = 8;
    __device__ static void load(const void* base, size_t elem, float* out) {
        u32x4 w = *reinterpret_cast<const u32x4*>(reinterpret_cast<const uint16_t*>(base) + elem);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            out[2 * q] = bf16_lo(w[q]);
            out[2 * q + 1] = bf16_hi(w[q]);
        }
    }
    __device__ static float scalar(const void* base, size_t elem) {
        return bf16_to_f32(reinterpret_cast<const uint16_t*>(base)[elem]);
    }
};
template <>
struct Vec<false> {  // 4 fp32 per 16-byte chunk
    static constexpr int n = 4;
    __device__ static void load(const void* base, size_t elem, float* out) {
        f32x4 w = *reinterpret_cast<const f32x4*>(reinterpret_cast<const float*>(base) + elem);
        out[0] = w[0]; out[1] = w[1]; out[2] = w[2]; out[3] = w[3];
    }
    __device__ static float scalar(const void* base, size_t elem) {
        return reinterpret_cast<const float*>(base)[elem];
    }
};

// LISTS = false: dense gate rows p.gates[gslot][token][E] (zeros outside the
// Top-K set); LISTS = true: the Top-K lists p.rt.sel / p.rt.gk of the routed path.
template <bool BF16, bool LISTS>
__global__ __launch_bounds__(256) void k_router(Problem p, UnitTab ut) {
    using V = Vec<BF16>;
    const uint32_t code = ut.code[blockIdx.y];
    const int j = unit_j(code), x = unit_x(code), i = unit_i(code), gs = unit_gslot(code);
    const int tok = blockIdx.x * kTokPerBlock + threadIdx.x / kLanesPerTok;
    const int q = threadIdx.x % kLanesPerTok;
    const int E = p.E, d_in = p.d_in;
    const size_t unit = (size_t)j * 2 + x;
    const size_t wr_base = unit * E * d_in;

    float acc[MOT_MAX_EXPERTS];
#pragma unroll
    for (int m = 0; m < MOT_MAX_EXPERTS; ++m) acc[m] = 0.f;

    if (tok < p.n_tok) {
        const size_t layer = (size_t)i * p.n_tok * d_in;
        const int b = tok / p.T, t = tok % p.T;
        for (int c0 = q * V::n; c0 < d_in; c0 += kLanesPerTok * V::n) {
            size_t off;
            if (p.src_layout == MOT_LAYOUT_BTHD) {
                off = layer + (size_t)tok * d_in + c0;
            } else {
                const int hh = c0 / p.D_src, dd = c0 % p.D_src;
                off = layer + (((size_t)b * p.H_src + hh) * p.T + t) * p.D_src + dd;
            }
            float z[V::n];
            V::load(p.src[x], off, z);
#pragma unroll
            for (int m = 0; m < MOT_MAX_EXPERTS; ++m) {
                if (m < E) {
                    float w[V::n];
                    V::load(p.wr, wr_base + (size_t)m * d_in + c0, w);
                    float s = acc[m];
#pragma unroll
                    for (int e = 0; e < V::n; ++e) s = fmaf(w[e], z[e], s);
                    acc[m] = s;
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
    if (tok >= p.n_tok || q != 0) return;
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
        const size_t base = ((size_t)gs * p.n_tok + tok) * p.top_k;
        topk_list(acc, E, p.top_k, p.rt.sel + base, p.rt.gk + base);
        return;
    }
    topk_renormalise(acc, E, p.top_k);
    float* g = p.gates + ((size_t)gs * p.n_tok_pad + tok) * E;
#pragma unroll
    for (int m = 0; m < MOT_MAX_EXPERTS; ++m)
        if (m < E) g[m] = acc[m];
}

}  // namespace

hipError_t launch_router(const Problem& p, const UnitTab& ut, bool bf16, hipStream_t stream) {
    if (ut.n == 0 || p.n_tok == 0) return hipSuccess;
    dim3 grid((p.n_tok + kTokPerBlock - 1) / kTokPerBlock, ut.n);
    if (bf16)
        hipLaunchKernelGGL((k_router<true, false>), grid, dim3(256), 0, stream, p, ut);
    else
        hipLaunchKernelGGL((k_router<false, false>), grid, dim3(256), 0, stream, p, ut);
    return hipGetLastError();
}

hipError_t launch_router_lists(const Problem& p, const UnitTab& ut, hipStream_t stream) {
    if (ut.n == 0 || p.n_tok == 0) return hipSuccess;
    dim3 grid((p.n_tok + kTokPerBlock - 1) / kTokPerBlock, ut.n);
    hipLaunchKernelGGL((k_router<true, true>), grid, dim3(256), 0, stream, p, ut);
    return hipGetLastError();
}

}  // namespace mot
