// Backbone translator body (paper App. C.2, "Backbone Translator") as the
// experts of the mixture, one channel-window slot per unit.  The host runs,
// per unit and expert, a chain of two generic kernels and the causal
// attention kernel of the replay step:
//   * k_ln_rows: LayerNorm of bf16 rows (one wave per row, fp32 statistics,
//     population variance, eps 1e-5), bf16 out;
//   * k_linear: out[t][o] = act(sum_k in[t][k] W[o][k] + b[o]) (+ res[t][o]) on
//     v_mfma_f32_32x32x16_bf16, 128 outputs x 128 rows per 256-thread
//     workgroup, K in 64-wide double-buffered XOR-swizzled LDS slices; the
//     epilogue either stores bf16 rows or adds gate[t][m] * value into the
//     fp32 mixture (the last expert rounds the mixture to bf16 into the
//     target cache).
#include "mot_device.h"
#include "mot_internal.h"
#include "../../include/mot.h"

namespace mot {

namespace {

constexpr int LM = 128, LN_ = 128, LK = 64;
constexpr int kLChunks = LM * LK / 8;   // 16-byte chunks per operand tile

__device__ __forceinline__ int lswz(int row, int c) { return row * 8 + (c ^ (row & 7)); }

// grid: ceil(n / 4) workgroups of 4 waves, one row per wave; w % 8 == 0, w <= 4096
__global__ __launch_bounds__(256) void k_ln_rows(const uint16_t* in, size_t ld_in, const uint16_t* g,
                                                 const uint16_t* b, uint16_t* out, int n, int w) {
    constexpr int MAXC = 8;   // 16-byte chunks per lane (w <= 64 * 8 * 8)
    const int lane = threadIdx.x & 63, row = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= n) return;
    const uint16_t* r = in + (size_t)row * ld_in;
    float v[MAXC][8];
    float sum = 0.f;
#pragma unroll
    for (int c = 0; c < MAXC; ++c) {
        const int e = (lane + 64 * c) * 8;
        if (e < w) {
            const u32x4 q = *reinterpret_cast<const u32x4*>(r + e);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                v[c][2 * i] = bf16_lo(q[i]);
                v[c][2 * i + 1] = bf16_hi(q[i]);
                sum += v[c][2 * i] + v[c][2 * i + 1];
            }
        }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) sum += __shfl_xor(sum, off, 64);
    const float mean = sum / (float)w;
    float sq = 0.f;
#pragma unroll
    for (int c = 0; c < MAXC; ++c) {
        const int e = (lane + 64 * c) * 8;
        if (e < w) {
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const float d = v[c][i] - mean;
                sq += d * d;
            }
        }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) sq += __shfl_xor(sq, off, 64);
    const float inv = rsqrtf(sq / (float)w + 1e-5f);
#pragma unroll
    for (int c = 0; c < MAXC; ++c) {
        const int e = (lane + 64 * c) * 8;
        if (e < w) {
            const u32x4 gq = *reinterpret_cast<const u32x4*>(g + e);
            const u32x4 bq = *reinterpret_cast<const u32x4*>(b + e);
            u32x4 o;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float y0 = (v[c][2 * i] - mean) * inv * bf16_lo(gq[i]) + bf16_lo(bq[i]);
                const float y1 = (v[c][2 * i + 1] - mean) * inv * bf16_hi(gq[i]) + bf16_hi(bq[i]);
                o[i] = pack_bf16x2(y0, y1);
            }
            *reinterpret_cast<u32x4*>(out + (size_t)row * w + e) = o;
        }
    }
}

// grid: x = row tiles of 128, y = output tiles of 128; 256 threads
__global__ __launch_bounds__(256) void k_linear(LinearProblem p) {
    __shared__ u32x4 lds[2][2][kLChunks];   // [stage][0 = W rows, 1 = input rows]
    const int r0 = blockIdx.x * LN_, o0 = blockIdx.y * LM;
    const int K = p.K, N = p.N;
    const uint16_t* A = p.in;
    const uint16_t* W = p.W;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1, g = lane >> 5, l32 = lane & 31;
    const u32x4 zero = {0u, 0u, 0u, 0u};
    u32x4 ra[4], rb[4];
    auto gload = [&](int k0) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int row = (tid >> 3) + 32 * r, c = tid & 7;
            const int o = o0 + row, t = r0 + row;
            ra[r] = o < N ? *reinterpret_cast<const u32x4*>(W + (size_t)o * K + k0 + c * 8) : zero;
            rb[r] = t < p.n ? *reinterpret_cast<const u32x4*>(A + (size_t)t * p.ld_in + k0 + c * 8) : zero;
        }
    };
    auto sstore = [&](int st) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int row = (tid >> 3) + 32 * r, c = tid & 7;
            lds[st][0][lswz(row, c)] = ra[r];
            lds[st][1][lswz(row, c)] = rb[r];
        }
    };
    f32x16 acc[2][2];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int bb = 0; bb < 2; ++bb)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[a][bb][e] = 0.f;
    const int nk = K / LK;
    gload(0);
    sstore(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int st = kt & 1;
        if (kt + 1 < nk) gload((kt + 1) * LK);
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            const int c = 2 * s + g;
            u32x4 a[2], bo[2];
#pragma unroll
            for (int bm = 0; bm < 2; ++bm) a[bm] = lds[st][0][lswz(wm * 64 + bm * 32 + l32, c)];
#pragma unroll
            for (int bn = 0; bn < 2; ++bn) bo[bn] = lds[st][1][lswz(wn * 64 + bn * 32 + l32, c)];
#pragma unroll
            for (int bm = 0; bm < 2; ++bm)
#pragma unroll
                for (int bn = 0; bn < 2; ++bn) acc[bm][bn] = mfma_32x32x16(a[bm], bo[bn], acc[bm][bn]);
        }
        if (kt + 1 < nk) sstore(st ^ 1);
        __syncthreads();
    }
    // epilogue: lane holds outputs obase + 8*ii + 4*g + jj (jj = 0..3) of row tc
#pragma unroll
    for (int bm = 0; bm < 2; ++bm) {
        const int obase = o0 + wm * 64 + bm * 32;
#pragma unroll
        for (int bn = 0; bn < 2; ++bn) {
            const int tc = r0 + wn * 64 + bn * 32 + l32;
            if (tc >= p.n) continue;
#pragma unroll
            for (int ii = 0; ii < 4; ++ii) {
                const int o = obase + 8 * ii + 4 * g;
                if (o >= N) continue;
                float v[4];
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) {
                    float x = acc[bm][bn][4 * ii + jj] + bf16_to_f32(p.bias[o + jj]);
                    if (p.gelu) x = gelu_fast(x);
                    if (p.res) x += bf16_to_f32(p.res[(size_t)tc * N + o + jj]);
                    v[jj] = x;
                }
                if (!p.mix) {
                    const u32x2 w2 = {pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
                    *reinterpret_cast<u32x2*>(p.out + (size_t)tc * N + o) = w2;
                } else {
                    const float gt = p.gates[(size_t)tc * p.gate_ld + p.expert];
                    f32x4 m = {0.f, 0.f, 0.f, 0.f};
                    float* accp = p.mix_acc + (size_t)tc * N + o;
                    if (!p.first) m = *reinterpret_cast<const f32x4*>(accp);
#pragma unroll
                    for (int jj = 0; jj < 4; ++jj) m[jj] += gt * v[jj];
                    if (p.last) {
                        const u32x2 w2 = {pack_bf16x2(m[0], m[1]), pack_bf16x2(m[2], m[3])};
                        *reinterpret_cast<u32x2*>(p.out + (size_t)tc * N + o) = w2;
                    } else {
                        *reinterpret_cast<f32x4*>(accp) = m;
                    }
                }
            }
        }
    }
}

}  // namespace

hipError_t launch_ln_rows(const uint16_t* in, size_t ld_in, const uint16_t* g, const uint16_t* b, uint16_t* out,
                          int n, int w, hipStream_t stream) {
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(k_ln_rows, dim3((n + 3) / 4), dim3(256), 0, stream, in, ld_in, g, b, out, n, w);
    return hipGetLastError();
}

hipError_t launch_linear(const LinearProblem& p, hipStream_t stream) {
    if (p.n == 0) return hipSuccess;
    hipLaunchKernelGGL(k_linear, dim3((p.n + LN_ - 1) / LN_, (p.N + LM - 1) / LM), dim3(256), 0, stream, p);
    return hipGetLastError();
}

}  // namespace mot
