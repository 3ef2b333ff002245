// bf16 translation path in two grouped MFMA GEMMs (any d_in multiple of 64).
//
//   gemm1 (translator layer 1, all E experts side by side, N = E*hidden):
//     Hs[u][t][m*hidden+k] = bf16( g[u][t][m] * GELU((W1_m z_t + b1_m)[k]) )
//   gemm2 (translator layer 2, K = E*hidden: the reduction over experts of
//     the gated sum happens inside the accumulator):
//     dst[j][t][o] = bf16( sum_kk Hs[u][t][kk] W2cat[o][kk] + sum_m g_m b2_m[o] )
//   with W2cat[o][m*hidden+k] = W2_m[o][k].  In exact arithmetic this is
//   sum_m g_m (W2_m GELU(W1_m z + b1_m) + b2_m), the paper's gated sum
//   (Sec. 3, Eq. mot_definition) with all E translators selected.
//
// Both kernels: 128 x 128 output tile per 256-thread workgroup (four waves in
// a 2 x 2 grid, 64 x 64 per wave = 2 x 2 MFMA 32x32x16 blocks), K staged in
// 64-wide slices through double-buffered LDS (16-byte chunks XOR-swizzled by
// row so the fragment reads are bank-conflict free).
//
// Hidden buffer layout ("fragment-native"): 16-byte units of 8 consecutive
// hidden values of one token, ordered [t/32][kk/8][t%32].  gemm1's MFMA
// result fragments store as full 512-byte runs, and gemm2 stages its A tile
// with 512-byte contiguous reads that land in LDS already in fragment order.
#include "mot_device.h"
#include "mot_internal.h"
#include "../../include/mot.h"

namespace mot {

namespace {

constexpr int BM = 128, BN = 128, BK = 64;
constexpr int kChunks = BM * BK / 8;   // 16-byte chunks per operand tile (1024)

__device__ __forceinline__ int swz(int row, int c) { return row * 8 + (c ^ (row & 7)); }

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

// ---------------------------------------------------------------------------
// gemm1: S^T[hidden][token] = W1[hidden][:] . Z[token][:]
//   MFMA A operand = W1 rows (hidden), B operand = source rows (tokens), so
//   each lane ends with 4 consecutive hidden values of one token per group.
// grid: x = token tiles, y = hidden tiles (E*hidden / 128), z = unit; the
// (x, y) workgroup id is remapped to a grouped order (below)
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_bf16_gemm1(Problem p, UnitTab ut) {
    __shared__ u32x4 lds[2][2][kChunks];   // [stage][0 = W1, 1 = Z]
    const uint32_t code = ut.code[blockIdx.z];
    const int j = unit_j(code), x = unit_x(code), i = unit_i(code), gs = unit_gslot(code);
    const int EH = p.E * p.hidden;
    // grouped dispatch order as in gemm2: 8 token tiles inner, hidden tiles
    // outer, so each XCD keeps one token tile's source rows in its L2 and a W1
    // tile is fetched once per group
    const int lin = blockIdx.x + gridDim.x * blockIdx.y, ny = gridDim.y;
    const int grp = lin / (8 * ny), gsz = min(8, (int)gridDim.x - 8 * grp), r = lin - grp * 8 * ny;
    const int tok0 = (8 * grp + r % gsz) * BN, hid0 = (r / gsz) * BM;
    const size_t unit = (size_t)j * p.streams + x;
    const uint16_t* W1 = reinterpret_cast<const uint16_t*>(p.w1) + unit * EH * p.d_in;
    const uint16_t* src = reinterpret_cast<const uint16_t*>(p.src[x]);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1, g = lane >> 5, l32 = lane & 31;

    u32x4 ra[4], rb[4];
    const u32x4 zero = {0u, 0u, 0u, 0u};
    auto gload = [&](int k0) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int row = (tid >> 3) + 32 * r, c = tid & 7;
            const int hid = hid0 + row, tok = tok0 + row;
            ra[r] = hid < EH ? *reinterpret_cast<const u32x4*>(W1 + (size_t)hid * p.d_in + k0 + c * 8)
                             : zero;
            rb[r] = tok < p.n_tok ? *reinterpret_cast<const u32x4*>(src + src_offset(p, i, tok, k0 + c * 8))
                                  : zero;
        }
    };
    auto sstore = [&](int st) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int row = (tid >> 3) + 32 * r, c = tid & 7;
            lds[st][0][swz(row, c)] = ra[r];
            lds[st][1][swz(row, c)] = rb[r];
        }
    };

    f32x16 acc[2][2];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[a][b][e] = 0.f;

    const int nk = p.d_in / BK;
    gload(0);
    sstore(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int st = kt & 1;
        if (kt + 1 < nk) gload((kt + 1) * BK);
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            const int c = 2 * s + g;
            u32x4 a[2], b[2];
#pragma unroll
            for (int bm = 0; bm < 2; ++bm) {
                const int row = wm * 64 + bm * 32 + l32;
                a[bm] = lds[st][0][swz(row, c)];
            }
#pragma unroll
            for (int bn = 0; bn < 2; ++bn) {
                const int row = wn * 64 + bn * 32 + l32;
                b[bn] = lds[st][1][swz(row, c)];
            }
#pragma unroll
            for (int bm = 0; bm < 2; ++bm)
#pragma unroll
                for (int bn = 0; bn < 2; ++bn) acc[bm][bn] = mfma_32x32x16(a[bm], b[bn], acc[bm][bn]);
        }
        if (kt + 1 < nk) sstore(st ^ 1);
        __syncthreads();
    }

    // epilogue: + b1, GELU, * gate, round to bf16, fragment-native store
    uint16_t* H = reinterpret_cast<uint16_t*>(p.hbuf) + (size_t)blockIdx.z * p.n_tok_pad * EH;
    const uint16_t* b1 = p.b1 ? reinterpret_cast<const uint16_t*>(p.b1) + unit * EH : nullptr;
    const float* G = p.gates + (size_t)gs * p.n_tok_pad * p.E;
#pragma unroll
    for (int bm = 0; bm < 2; ++bm) {
        const int hbase = hid0 + wm * 64 + bm * 32;
        if (hbase >= EH) continue;
        const int e = hbase / p.hidden;   // hidden % 64 == 0: one expert per 32 rows
#pragma unroll
        for (int bn = 0; bn < 2; ++bn) {
            const int tc = tok0 + wn * 64 + bn * 32 + l32;
            const float gate = tc < p.n_tok ? G[(size_t)tc * p.E + e] : 0.f;
            uint16_t* hrow = H + ((size_t)(tc >> 5) * (EH >> 3) + (hbase >> 3)) * 256 + (tc & 31) * 8 + 4 * g;
#pragma unroll
            for (int ii = 0; ii < 4; ++ii) {
                float v[4];
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) {
                    const int hr = hbase + 8 * ii + 4 * g + jj;
                    float a = acc[bm][bn][4 * ii + jj] + (b1 ? bf16_to_f32(b1[hr]) : 0.f);
                    a = p.act == MOT_ACT_GELU ? gelu_tanh(a) : a;
                    v[jj] = gate * a;
                }
                u32x2 w = {pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
                *reinterpret_cast<u32x2*>(hrow + (size_t)ii * 256) = w;
            }
        }
    }
}

// ---------------------------------------------------------------------------
// gemm2: Y[token][out] = Hs[token][:] . W2cat[out][:]  (+ gate-mixed b2)
//   MFMA A operand = hidden rows (tokens), B operand = W2 rows (outputs).
// grid: x = token tiles, y = output tiles (d_out / 128, ragged), z = unit;
// the (x, y) workgroup id is remapped to a grouped order (below)
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_bf16_gemm2(Problem p, UnitTab ut) {
    __shared__ u32x4 lds[2][2][kChunks];   // [stage][0 = Hs, 1 = W2]
    const uint32_t code = ut.code[blockIdx.z];
    const int j = unit_j(code), x = unit_x(code), gs = unit_gslot(code);
    const int EH = p.E * p.hidden;
    // dispatch order in groups of 8 token tiles: output tiles outer, the
    // group's token tiles inner.  Workgroups are dealt round-robin to the 8
    // XCDs, so each XCD keeps one token tile (its A rows, re-read by every
    // output tile) in its L2, and a W2 tile is fetched once per group instead
    // of once per token tile.
    const int lin = blockIdx.x + gridDim.x * blockIdx.y, ny = gridDim.y;
    const int grp = lin / (8 * ny), gsz = min(8, (int)gridDim.x - 8 * grp), r = lin - grp * 8 * ny;
    const int tok0 = (8 * grp + r % gsz) * BM, out0 = (r / gsz) * BN;
    const size_t unit = (size_t)j * p.streams + x;
    const uint16_t* W2 = reinterpret_cast<const uint16_t*>(p.w2) + unit * p.E * p.d_out * p.hidden;
    const uint16_t* H = reinterpret_cast<const uint16_t*>(p.hbuf) + (size_t)blockIdx.z * p.n_tok_pad * EH;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1, g = lane >> 5, l32 = lane & 31;

    u32x4 ra[4], rb[4];
    const u32x4 zero = {0u, 0u, 0u, 0u};
    auto gload = [&](int k0) {
        const int m = k0 / p.hidden, kk = k0 % p.hidden;   // hidden % 64 == 0
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int q = tid + 256 * r;
            // A: fragment-native, q = tb*256 + kc*32 + tl maps to one 16-byte unit
            const int tb = q >> 8, kc = (q >> 5) & 7, tl = q & 31;
            ra[r] = *reinterpret_cast<const u32x4*>(
                H + ((size_t)((tok0 >> 5) + tb) * (EH >> 3) + (k0 >> 3) + kc) * 256 + tl * 8);
            // B: W2 row o, 8 consecutive k
            const int row = q >> 3, c = q & 7, o = out0 + row;
            rb[r] = o < p.d_out
                        ? *reinterpret_cast<const u32x4*>(W2 + ((size_t)m * p.d_out + o) * p.hidden + kk + c * 8)
                        : zero;
        }
    };
    auto sstore = [&](int st) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int q = tid + 256 * r;
            lds[st][0][q] = ra[r];
            lds[st][1][swz(q >> 3, q & 7)] = rb[r];
        }
    };

    f32x16 acc[2][2];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[a][b][e] = 0.f;

    const int nk = EH / BK;
    gload(0);
    sstore(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int st = kt & 1;
        if (kt + 1 < nk) gload((kt + 1) * BK);
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            const int c = 2 * s + g;
            u32x4 a[2], b[2];
#pragma unroll
            for (int bm = 0; bm < 2; ++bm) a[bm] = lds[st][0][(wm * 2 + bm) * 256 + c * 32 + l32];
#pragma unroll
            for (int bn = 0; bn < 2; ++bn) {
                const int row = wn * 64 + bn * 32 + l32;
                b[bn] = lds[st][1][swz(row, c)];
            }
#pragma unroll
            for (int bm = 0; bm < 2; ++bm)
#pragma unroll
                for (int bn = 0; bn < 2; ++bn) acc[bm][bn] = mfma_32x32x16(a[bm], b[bn], acc[bm][bn]);
        }
        if (kt + 1 < nk) sstore(st ^ 1);
        __syncthreads();
    }

    // epilogue: + sum_m g_m b2_m[o], round to bf16, store in the target layout
    const uint16_t* b2 = p.b2 ? reinterpret_cast<const uint16_t*>(p.b2) + unit * p.E * p.d_out : nullptr;
    const float* G = p.gates + (size_t)gs * p.n_tok_pad * p.E;
    uint16_t* dst = reinterpret_cast<uint16_t*>(p.dst[x]);
#pragma unroll
    for (int bn = 0; bn < 2; ++bn) {
        const int o = out0 + wn * 64 + bn * 32 + l32;
        if (o >= p.d_out) continue;
        float bias[MOT_MAX_EXPERTS];
#pragma unroll
        for (int m = 0; m < MOT_MAX_EXPERTS; ++m)
            bias[m] = (b2 && m < p.E) ? bf16_to_f32(b2[(size_t)m * p.d_out + o]) : 0.f;
#pragma unroll
        for (int bm = 0; bm < 2; ++bm) {
#pragma unroll
            for (int ii = 0; ii < 4; ++ii) {
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) {
                    const int tok = tok0 + wm * 64 + bm * 32 + 8 * ii + 4 * g + jj;
                    if (tok >= p.n_tok) continue;
                    float v = acc[bm][bn][4 * ii + jj];
                    if (b2) {
                        const float* gt = G + (size_t)tok * p.E;
#pragma unroll
                        for (int m = 0; m < MOT_MAX_EXPERTS; ++m)
                            if (m < p.E) v = fmaf(gt[m], bias[m], v);
                    }
                    dst[dst_offset(p, j, tok, o)] = (uint16_t)(pack_bf16x2(v, 0.f) & 0xFFFFu);
                }
            }
        }
    }
}

}  // namespace

hipError_t launch_bf16_gemm1(const Problem& p, const UnitTab& ut, hipStream_t stream) {
    if (ut.n == 0 || p.n_tok == 0) return hipSuccess;
    const int EH = p.E * p.hidden;
    dim3 grid(p.n_tok_pad / BN, (EH + BM - 1) / BM, ut.n);
    hipLaunchKernelGGL(k_bf16_gemm1, grid, dim3(256), 0, stream, p, ut);
    return hipGetLastError();
}

hipError_t launch_bf16_gemm2(const Problem& p, const UnitTab& ut, hipStream_t stream) {
    if (ut.n == 0 || p.n_tok == 0) return hipSuccess;
    dim3 grid(p.n_tok_pad / BM, (p.d_out + BN - 1) / BN, ut.n);
    hipLaunchKernelGGL(k_bf16_gemm2, grid, dim3(256), 0, stream, p, ut);
    return hipGetLastError();
}

}  // namespace mot
