// Key/value restoration for the activation-translation variant MoT-h (paper
// App. C.5): the target model's fixed key and value projections applied to a
// translated intermediate activation,
//     K[l][t] = W^K[l] a[l][t] + b^K[l],    V[l][t] = W^V[l] a[l][t] + b^V[l].
// One bf16 MFMA GEMM per layer with both projections side by side (output
// rows o < d_kv are keys, the rest values): 128 x 128 output tile per
// 256-thread workgroup (2 x 2 waves of 64 x 64, each 2 x 2 blocks of
// v_mfma_f32_32x32x16_bf16), the d_act contraction staged in 64-wide
// double-buffered LDS slices, 16-byte chunks XOR-swizzled by row.  Epilogue:
// + bias, round to bf16, store four consecutive outputs of a token as one
// 8-byte write into the key or value cache in the target layout.
#include "mot_device.h"
#include "mot_internal.h"
#include "../../include/mot.h"

namespace mot {

namespace {

constexpr int PM = 128, PN = 128, PK = 64;
constexpr int kPChunks = PM * PK / 8;   // 16-byte chunks per operand tile

__device__ __forceinline__ int pswz(int row, int c) { return row * 8 + (c ^ (row & 7)); }

// grid: x = token tiles, y = output tiles over 2*d_kv, z = position in the layer list
__global__ __launch_bounds__(256) void k_bf16_project(ProjProblem p) {
    __shared__ u32x4 lds[2][2][kPChunks];   // [stage][0 = W rows, 1 = activation rows]
    const int l = p.layers[blockIdx.z];
    const int tok0 = blockIdx.x * PN, out0 = blockIdx.y * PM;
    const int d_act = p.d_act, d_kv = p.d_kv, n_out = 2 * d_kv;
    const uint16_t* A = reinterpret_cast<const uint16_t*>(p.act) + (size_t)l * p.n_tok * d_act;
    const uint16_t* WK = reinterpret_cast<const uint16_t*>(p.wk) + (size_t)l * d_kv * d_act;
    const uint16_t* WV = reinterpret_cast<const uint16_t*>(p.wv) + (size_t)l * d_kv * d_act;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1, g = lane >> 5, l32 = lane & 31;

    u32x4 ra[4], rb[4];
    const u32x4 zero = {0u, 0u, 0u, 0u};
    auto gload = [&](int k0) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int row = (tid >> 3) + 32 * r, c = tid & 7;
            const int o = out0 + row, tok = tok0 + row;
            const uint16_t* wrow = o < d_kv ? WK + (size_t)o * d_act : WV + (size_t)(o - d_kv) * d_act;
            ra[r] = o < n_out ? *reinterpret_cast<const u32x4*>(wrow + k0 + c * 8) : zero;
            rb[r] = tok < p.n_tok ? *reinterpret_cast<const u32x4*>(A + (size_t)tok * d_act + k0 + c * 8) : zero;
        }
    };
    auto sstore = [&](int st) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int row = (tid >> 3) + 32 * r, c = tid & 7;
            lds[st][0][pswz(row, c)] = ra[r];
            lds[st][1][pswz(row, c)] = rb[r];
        }
    };

    f32x16 acc[2][2];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[a][b][e] = 0.f;

    const int nk = d_act / PK;
    gload(0);
    sstore(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int st = kt & 1;
        if (kt + 1 < nk) gload((kt + 1) * PK);
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            const int c = 2 * s + g;
            u32x4 a[2], b[2];
#pragma unroll
            for (int bm = 0; bm < 2; ++bm) a[bm] = lds[st][0][pswz(wm * 64 + bm * 32 + l32, c)];
#pragma unroll
            for (int bn = 0; bn < 2; ++bn) b[bn] = lds[st][1][pswz(wn * 64 + bn * 32 + l32, c)];
#pragma unroll
            for (int bm = 0; bm < 2; ++bm)
#pragma unroll
                for (int bn = 0; bn < 2; ++bn) acc[bm][bn] = mfma_32x32x16(a[bm], b[bn], acc[bm][bn]);
        }
        if (kt + 1 < nk) sstore(st ^ 1);
        __syncthreads();
    }

    // epilogue: lane holds outputs obase + 8*ii + 4*g + jj (jj = 0..3) of token tc
    const uint16_t* BK = reinterpret_cast<const uint16_t*>(p.bk);
    const uint16_t* BV = reinterpret_cast<const uint16_t*>(p.bv);
#pragma unroll
    for (int bm = 0; bm < 2; ++bm) {
        const int obase = out0 + wm * 64 + bm * 32;
#pragma unroll
        for (int bn = 0; bn < 2; ++bn) {
            const int tc = tok0 + wn * 64 + bn * 32 + l32;
            if (tc >= p.n_tok) continue;
            const int b = tc / p.T, t = tc % p.T;
#pragma unroll
            for (int ii = 0; ii < 4; ++ii) {
                const int o = obase + 8 * ii + 4 * g;   // four outputs o .. o+3, one head, one of K / V
                if (o >= n_out) continue;
                const bool isv = o >= d_kv;
                const int ok = isv ? o - d_kv : o;
                const uint16_t* bias = isv ? BV : BK;
                float v[4];
#pragma unroll
                for (int jj = 0; jj < 4; ++jj)
                    v[jj] = acc[bm][bn][4 * ii + jj] + (bias ? bf16_to_f32(bias[(size_t)l * d_kv + ok + jj]) : 0.f);
                const int hh = ok / p.D_tgt, dd = ok % p.D_tgt;
                size_t off = (size_t)l * p.n_tok * d_kv;
                off += p.dst_layout == MOT_LAYOUT_BTHD ? (size_t)tc * d_kv + ok
                                                       : (((size_t)b * p.H_tgt + hh) * p.T + t) * p.D_tgt + dd;
                uint16_t* dst = reinterpret_cast<uint16_t*>(isv ? p.dst_v : p.dst_k);
                const u32x2 w = {pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
                *reinterpret_cast<u32x2*>(dst + off) = w;
            }
        }
    }
}

}  // namespace

hipError_t launch_bf16_project(const ProjProblem& p, int n_layers, hipStream_t stream) {
    if (n_layers == 0 || p.n_tok == 0) return hipSuccess;
    dim3 grid((p.n_tok + PN - 1) / PN, (2 * p.d_kv + PM - 1) / PM, n_layers);
    hipLaunchKernelGGL(k_bf16_project, grid, dim3(256), 0, stream, p);
    return hipGetLastError();
}

}  // namespace mot
