// fp32 translation path for shapes the matrix-core form (k_f32_mfma.hip)
// does not take (hidden not a multiple of 64): two LDS-tiled GEMMs on the
// vector ALUs.  Built without packed fp32 instructions, the vector ALUs peak
// at half of MI355X's 157.3 TFLOP/s fp32 figure (one FMA per lane and cycle).
//
//   gemm1: Hs[u][t][m*hidden+k] = g[u][t][m] * GELU(W1_m z_t + b1_m)[k]
//   gemm2: dst[j][t][o]         = sum_{m,k} Hs[u][t][m*hidden+k] W2_m[o][k]
//                                 + sum_m g[u][t][m] b2_m[o]
// which equals sum_m g_m (W2_m GELU(W1_m z + b1_m) + b2_m): the gated sum of
// the paper's Eq. mot_definition with the gate folded into the hidden row.
//
// Tiles: 64 x 64 outputs per 256-thread workgroup, 4 x 4 per thread, K in
// steps of 16 staged through LDS (k-major so inner-loop reads broadcast).
#include "mot_device.h"
#include "mot_internal.h"
#include "../../include/mot.h"

namespace mot {

namespace {

constexpr int TM = 64, TN = 64, TK = 16;

__device__ __forceinline__ size_t src_offset(const Problem& p, int i, int tok, int c) {
    const size_t layer = (size_t)i * p.n_tok * p.d_in;
    if (p.src_layout == MOT_LAYOUT_BTHD) return layer + (size_t)tok * p.d_in + c;
    const int b = tok / p.T, t = tok % p.T, hh = c / p.D_src, dd = c % p.D_src;
    return layer + (((size_t)b * p.H_src + hh) * p.T + t) * p.D_src + dd;
}

__device__ __forceinline__ size_t dst_offset(const Problem& p, int j, int tok, int o) {
    const size_t layer = (size_t)j * p.n_tok * p.d_out;
    if (p.dst_layout == MOT_LAYOUT_BTHD) return layer + (size_t)tok * p.d_out + o;
    const int b = tok / p.T, t = tok % p.T, hh = o / p.D_tgt, dd = o % p.D_tgt;
    return layer + (((size_t)b * p.H_tgt + hh) * p.T + t) * p.D_tgt + dd;
}

// grid: x = token tiles, y = hidden tiles over E*hidden, z = unit in launch
__global__ __launch_bounds__(256) void k_f32_gemm1(Problem p, UnitTab ut) {
    __shared__ float As[TK][TM + 4];   // tokens
    __shared__ float Bs[TK][TN + 4];   // hidden rows
    const uint32_t code = ut.code[blockIdx.z];
    const int j = unit_j(code), x = unit_x(code), i = unit_i(code), gs = unit_gslot(code);
    const int EH = p.E * p.hidden;
    const int tok0 = blockIdx.x * TM, hid0 = blockIdx.y * TN;
    const size_t unit = (size_t)j * p.streams + x;
    const float* W1 = reinterpret_cast<const float*>(p.w1) + unit * EH * p.d_in;
    const float* src = reinterpret_cast<const float*>(p.src[x]);
    const int tid = threadIdx.x, tx = tid % 16, ty = tid / 16;
    const int lr = tid / 4, lk = (tid % 4) * 4;   // loader: row, k offset

    float acc[4][4] = {};
    for (int k0 = 0; k0 < p.d_in; k0 += TK) {
        f32x4 a = {0.f, 0.f, 0.f, 0.f}, b = {0.f, 0.f, 0.f, 0.f};
        const int tok = tok0 + lr, hid = hid0 + lr, k = k0 + lk;
        if (tok < p.n_tok && k < p.d_in)
            a = *reinterpret_cast<const f32x4*>(src + src_offset(p, i, tok, k));
        if (hid < EH && k < p.d_in)
            b = *reinterpret_cast<const f32x4*>(W1 + (size_t)hid * p.d_in + k);
#pragma unroll
        for (int e = 0; e < 4; ++e) { As[lk + e][lr] = a[e]; Bs[lk + e][lr] = b[e]; }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < TK; ++kk) {
            float av[4], bv[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) { av[e] = As[kk][ty * 4 + e]; bv[e] = Bs[kk][tx * 4 + e]; }
#pragma unroll
            for (int r = 0; r < 4; ++r)
#pragma unroll
                for (int c = 0; c < 4; ++c) acc[r][c] = fmaf(av[r], bv[c], acc[r][c]);
        }
        __syncthreads();
    }
    float* H = reinterpret_cast<float*>(p.hbuf) + (size_t)blockIdx.z * p.n_tok_pad * EH;
    const float* b1 = p.b1 ? reinterpret_cast<const float*>(p.b1) + unit * EH : nullptr;
    const float* g = p.gates + (size_t)gs * p.n_tok_pad * p.E;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int tok = tok0 + ty * 4 + r;
        if (tok >= p.n_tok) continue;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const int hid = hid0 + tx * 4 + c;
            if (hid >= EH) continue;
            float v = acc[r][c] + (b1 ? b1[hid] : 0.f);
            v = p.act == MOT_ACT_GELU ? gelu_erf(v) : v;
            H[(size_t)tok * EH + hid] = g[(size_t)tok * p.E + hid / p.hidden] * v;
        }
    }
}

// grid: x = token tiles, y = output tiles over d_out, z = unit in launch
__global__ __launch_bounds__(256) void k_f32_gemm2(Problem p, UnitTab ut) {
    __shared__ float As[TK][TM + 4];   // tokens (hidden rows of Hs)
    __shared__ float Bs[TK][TN + 4];   // output channels (rows of W2)
    const uint32_t code = ut.code[blockIdx.z];
    const int j = unit_j(code), x = unit_x(code), gs = unit_gslot(code);
    const int EH = p.E * p.hidden;
    const int tok0 = blockIdx.x * TM, out0 = blockIdx.y * TN;
    const size_t unit = (size_t)j * p.streams + x;
    const float* W2 = reinterpret_cast<const float*>(p.w2) + unit * p.E * p.d_out * p.hidden;
    const float* H = reinterpret_cast<const float*>(p.hbuf) + (size_t)blockIdx.z * p.n_tok_pad * EH;
    const int tid = threadIdx.x, tx = tid % 16, ty = tid / 16;
    const int lr = tid / 4, lk = (tid % 4) * 4;

    float acc[4][4] = {};
    for (int k0 = 0; k0 < EH; k0 += TK) {
        f32x4 a = {0.f, 0.f, 0.f, 0.f}, b = {0.f, 0.f, 0.f, 0.f};
        const int tok = tok0 + lr, o = out0 + lr, k = k0 + lk;
        if (tok < p.n_tok && k < EH)
            a = *reinterpret_cast<const f32x4*>(H + (size_t)tok * EH + k);
        if (o < p.d_out && k < EH) {
            const int m = k / p.hidden, kk = k % p.hidden;   // hidden % 4 == 0
            b = *reinterpret_cast<const f32x4*>(W2 + ((size_t)m * p.d_out + o) * p.hidden + kk);
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) { As[lk + e][lr] = a[e]; Bs[lk + e][lr] = b[e]; }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < TK; ++kk) {
            float av[4], bv[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) { av[e] = As[kk][ty * 4 + e]; bv[e] = Bs[kk][tx * 4 + e]; }
#pragma unroll
            for (int r = 0; r < 4; ++r)
#pragma unroll
                for (int c = 0; c < 4; ++c) acc[r][c] = fmaf(av[r], bv[c], acc[r][c]);
        }
        __syncthreads();
    }
    const float* b2 = p.b2 ? reinterpret_cast<const float*>(p.b2) + unit * p.E * p.d_out : nullptr;
    const float* g = p.gates + (size_t)gs * p.n_tok_pad * p.E;
    float* dst = reinterpret_cast<float*>(p.dst[x]);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int tok = tok0 + ty * 4 + r;
        if (tok >= p.n_tok) continue;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const int o = out0 + tx * 4 + c;
            if (o >= p.d_out) continue;
            float v = acc[r][c];
            if (b2)
                for (int m = 0; m < p.E; ++m)
                    v = fmaf(g[(size_t)tok * p.E + m], b2[(size_t)m * p.d_out + o], v);
            dst[dst_offset(p, j, tok, o)] = v;
        }
    }
}

}  // namespace

hipError_t launch_f32_gemm1(const Problem& p, const UnitTab& ut, hipStream_t stream) {
    if (ut.n == 0 || p.n_tok == 0) return hipSuccess;
    const int EH = p.E * p.hidden;
    dim3 grid((p.n_tok + TM - 1) / TM, (EH + TN - 1) / TN, ut.n);
    hipLaunchKernelGGL(k_f32_gemm1, grid, dim3(256), 0, stream, p, ut);
    return hipGetLastError();
}

hipError_t launch_f32_gemm2(const Problem& p, const UnitTab& ut, hipStream_t stream) {
    if (ut.n == 0 || p.n_tok == 0) return hipSuccess;
    dim3 grid((p.n_tok + TM - 1) / TM, (p.d_out + TN - 1) / TN, ut.n);
    hipLaunchKernelGGL(k_f32_gemm2, grid, dim3(256), 0, stream, p, ut);
    return hipGetLastError();
}

}  // namespace mot
