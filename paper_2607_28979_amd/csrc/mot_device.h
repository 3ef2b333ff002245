// Device helpers for the gfx950 kernels: bf16 packing, MFMA wrappers, GELU.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mot {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }
__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// Two floats -> two bf16 (round to nearest even), packed low = a, high = b.
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
    f32x2 v = {a, b};
    bf16x2 r = __builtin_convertvector(v, bf16x2);
    return __builtin_bit_cast(uint32_t, r);
}

// D(32x32, fp32) += A(32x16, bf16) * B(16x32, bf16).
// Lane l holds A row (l % 32), k = 8*(l/32) .. +7; B column (l % 32), the
// same k; D column (l % 32), rows 8*i + 4*(l/32) + j at element 4*i + j.
__device__ __forceinline__ f32x16 mfma_32x32x16(u32x4 a, u32x4 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// D(16x16, fp32) += A(16x32, bf16) * B(32x16, bf16).
// Lane l holds A row (l % 16), k = 8*(l/16) .. +7; B column (l % 16), the
// same k; D column (l % 16), rows 4*(l/16) + j at element j.
__device__ __forceinline__ f32x4 mfma_16x16x32(u32x4 a, u32x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// Top-K of the E softmax scores g[0..E) (paper Sec. 3, Definition
// "Mixture-of-Translators": the K largest scores, renormalised to sum to one
// over the selected set; the others become zero).  K rounds each take the
// largest score not yet taken; the scan is ascending with a strict '>', so
// ties go to the lower index.  K >= E keeps every score unchanged (the dense
// mixture).  Returns the selected set as a bit mask (bit m = translator m).
template <int EMAX>
__device__ __forceinline__ uint32_t topk_renormalise(float (&g)[EMAX], int E, int K) {
    if (K >= E) return E >= 32 ? 0xFFFFFFFFu : (1u << E) - 1u;
    uint32_t taken = 0;
    float sum = 0.f;
    for (int k = 0; k < K; ++k) {
        int best = -1;
        float bv = 0.f;
#pragma unroll
        for (int m = 0; m < EMAX; ++m) {
            const bool cand = m < E && !((taken >> m) & 1u) && (best < 0 || g[m] > bv);
            best = cand ? m : best;
            bv = cand ? g[m] : bv;
        }
        if (best < 0) break;
        taken |= 1u << best;
        sum += bv;
    }
    const float inv = 1.0f / sum;
#pragma unroll
    for (int m = 0; m < EMAX; ++m) g[m] = ((taken >> m) & 1u) ? g[m] * inv : 0.f;
    return taken;
}

// Translator usage: add, for every translator m < E, the number of lanes of
// the wave whose selected set `taken` holds m (lanes with valid == false
// add nothing) to usage[m].  Called by every lane of the wave.
__device__ __forceinline__ void count_usage(uint32_t* usage, int E, uint32_t taken, bool valid) {
    const int lane = threadIdx.x & 63;
    for (int m = 0; m < E; ++m) {
        const unsigned long long b = __ballot(valid && ((taken >> m) & 1u));
        if (lane == 0 && b) atomicAdd(usage + m, (uint32_t)__popcll(b));
    }
}

// The same Top-K as topk_renormalise, emitted as a list: sel[k], gk[k] for
// k < K in selection order (largest score first, ties to the lower index),
// gates renormalised over the list.  K <= E.  The selection runs twice (sum,
// then emit) so nothing is read back from the output arrays.
template <int EMAX>
__device__ __forceinline__ void topk_list(const float (&g)[EMAX], int E, int K, int32_t* sel,
                                          float* gk) {
    float inv = 0.f;
    for (int pass = 0; pass < 2; ++pass) {
        uint32_t taken = 0;
        float sum = 0.f;
        for (int k = 0; k < K; ++k) {
            int best = -1;
            float bv = 0.f;
#pragma unroll
            for (int m = 0; m < EMAX; ++m) {
                const bool cand = m < E && !((taken >> m) & 1u) && (best < 0 || g[m] > bv);
                best = cand ? m : best;
                bv = cand ? g[m] : bv;
            }
            if (best < 0) best = 0;   // not reached for finite scores
            taken |= 1u << best;
            sum += bv;
            if (pass == 1) {
                sel[k] = best;
                gk[k] = bv * inv;
            }
        }
        inv = 1.0f / sum;
    }
}

// Exact-erf GELU, x * Phi(x), with the device erff.
__device__ __forceinline__ float gelu_erf(float x) {
    return 0.5f * x * (1.0f + erff(x * 0.70710678118654752f));
}

// g * GELU(x) with hg = g / 2, for the fused bf16 kernel, in the tanh form
// of GELU (Hendrycks & Gimpel): GELU(x) ~ x * sigmoid(2u),
// u = sqrt(2/pi) * (x + 0.044715 x^3).  Its largest deviation from the erf
// form is 4.7e-4 absolute (at |x| ~ 2.7); over normal pre-activations its rms
// deviation is ~2e-4 of the rms value, an order below the bf16 rounding the
// result gets next.  With e = 2^(x * (K1 + K3 x^2)) = exp(-2u):
// g * GELU(x) = hg * x * 2 / (1 + e).
#define MOT_GELU_K1 (-2.3022082f)      // -2 sqrt(2/pi) log2(e)
#define MOT_GELU_K3 (-0.10294324f)     // K1 * 0.044715
__device__ __forceinline__ float gelu_half_scaled(float x, float hg) {
    const float e = __builtin_amdgcn_exp2f(x * fmaf(x * x, MOT_GELU_K3, MOT_GELU_K1));
    return (hg * x) * __builtin_amdgcn_rcpf(fmaf(e, 0.5f, 0.5f));
}

// GELU(x) in the same tanh form, x / (1 + e), for the two-GEMM bf16 path's
// layer-1 epilogue and the backbone experts' linear epilogue.
__device__ __forceinline__ float gelu_tanh(float x) {
    const float e = __builtin_amdgcn_exp2f(x * fmaf(x * x, MOT_GELU_K3, MOT_GELU_K1));
    return x * __builtin_amdgcn_rcpf(1.0f + e);
}

// The same function with the gate g folded in, in three dependent stages so
// a software pipeline can overlap the chains of several elements: stage 1
// gives e, stage 2 gives r = g / (1 + e) as the reciprocal of cg (1 + e) with
// cg = 1/g (kept finite), and stage 3 is the product g GELU(x) = x r.
__device__ __forceinline__ void gelu_stage1(float x, float& e) {
    e = __builtin_amdgcn_exp2f(x * fmaf(x * x, MOT_GELU_K3, MOT_GELU_K1));
}
__device__ __forceinline__ void gelu_stage2_gated(float e, float cg, float& r) {
    r = __builtin_amdgcn_rcpf(fmaf(e, cg, cg));
}

}  // namespace mot
