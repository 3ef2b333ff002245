// Internal launch descriptors shared by the host dispatcher and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "replay_limits.h"

namespace mot {

// Up to 2 * MOT_MAX_LAYERS units can be launched together.
constexpr int kMaxUnits = 512;

// One unit = (target layer j, X in {K=0, V=1}) reading source layer i.
// gslot indexes the gate buffer (all units of a call), the launch position
// indexes the hidden buffer (units of one group).
__host__ __device__ inline uint32_t unit_code(int j, int x, int i, int gslot) {
    return (uint32_t)j | ((uint32_t)x << 8) | ((uint32_t)i << 9) | ((uint32_t)gslot << 17);
}
__host__ __device__ inline int unit_j(uint32_t c) { return (int)(c & 0xFF); }
__host__ __device__ inline int unit_x(uint32_t c) { return (int)((c >> 8) & 1); }
__host__ __device__ inline int unit_i(uint32_t c) { return (int)((c >> 9) & 0xFF); }
__host__ __device__ inline int unit_gslot(uint32_t c) { return (int)((c >> 17) & 0x3FF); }

struct UnitTab {
    int32_t n;
    uint32_t code[kMaxUnits];
};

// Buffers of the routed (Top-K sparse) path, all in the workspace.  Arrays
// marked [units] are indexed by the unit's gslot; part by the launch position
// of the unit within its group.
struct Routing {
    int32_t* sel;       // [units][n_tok][top_k] selected translators, best first
    float* gk;          // [units][n_tok][top_k] their renormalised gates
    int32_t* list;      // [units][n_tok*top_k] token of each assignment, grouped by translator
    float* agate;       // [units][n_tok*top_k] gate of each assignment
    int32_t* slot;      // [units][n_tok][top_k] assignment index of (token, k)
    int4* tiles;        // [units][max_tiles] {translator, first assignment, rows, 0}
    int32_t* ntiles;    // [units]
    float* part;        // [group][n_tok*top_k][d_out] fp32 per-assignment outputs (top_k > 1)
    int32_t max_tiles;  // tiles per unit the launch grid covers
    int32_t tile_rows;  // assignments per tile
};

// Problem description handed to every kernel by value.
struct Problem {
    const void* src[2];   // source K, V: [L_src] x layout
    void* dst[2];         // target K, V: [L_tgt] x layout
    const void* w1;       // [L_tgt][2][E][hidden][d_in]
    const void* b1;       // [L_tgt][2][E][hidden] or null
    const void* w2;       // [L_tgt][2][E][d_out][hidden]
    const void* b2;       // [L_tgt][2][E][d_out] or null
    const void* wr;       // [L_tgt][2][E][d_in]
    const void* br;       // [L_tgt][2][E] or null
    int32_t B, T, H_src, D_src, H_tgt, D_tgt, E, top_k, hidden;
    int32_t d_in, d_out, n_tok, n_tok_pad;   // n_tok_pad: n_tok rounded up to 128
    int32_t src_layout, dst_layout, act;
    int32_t streams;      // 2: keys and values; 1: one activation stream (src[0] -> dst[0])
    uint32_t* usage;      // [L_tgt][streams][E] selection counts to add to, or null
    float* gates;         // workspace: [n_units_total][n_tok_pad][E] fp32
    void* hbuf;           // workspace: [group][n_tok_pad][E*hidden] (layout per path)
    Routing rt;           // routed path only
};

// Key/value restoration (MoT-h): K and V caches from a translated activation.
struct ProjProblem {
    const void* act;      // [L][B*T][d_act]
    const void* wk;       // [L][d_kv][d_act]
    const void* bk;       // [L][d_kv] or null
    const void* wv;
    const void* bv;
    void* dst_k;          // [L] x dst layout, d_kv = H_tgt * D_tgt per token
    void* dst_v;
    int32_t B, T, n_tok, d_act, d_kv, H_tgt, D_tgt, dst_layout;
    int32_t layers[kMaxUnits];   // layers to restore, in launch order
};
hipError_t launch_bf16_project(const ProjProblem& p, int n_layers, hipStream_t stream);
// The same on 256 x 256 tiles (k_bf16_gemm256.hip) when d_kv % 256 == 0 and
// the launch fills at least half a round of the chip
bool bf16_project_256_fits(const ProjProblem& p, int n_layers);
hipError_t launch_bf16_project_256(const ProjProblem& p, int n_layers, hipStream_t stream);

// Context replay attention (Top-S sparse, or full causal when idx == nullptr).
struct ReplayProblem {
    const void* q;        // bf16 [B][T][H_q][D]
    const void* k;        // bf16 [B][T][H_kv][D] (BTHD) or [B][H_kv][T][D] (BHTD)
    const void* v;
    const int32_t* idx;   // [B][T][S] key sets, -1 padded; nullptr = full causal
    void* o;              // bf16 [B][T][H_q][D]
    // full causal path only: scratch for V transposed, bf16
    // [B][H_kv][D][replay_tpad(T)], written by the launch before use
    uint16_t* vt;
    int32_t B, T, H_q, H_kv, D, S, kv_layout;
};
__host__ __device__ inline int64_t replay_tpad(int64_t T) { return (T + 63) / 64 * 64; }
inline size_t replay_vt_bytes(int B, int T, int H_kv, int D) {
    return (size_t)B * H_kv * D * (size_t)replay_tpad(T) * 2;
}

// Generic bf16 linear layer of the backbone translator body.  One launch
// computes up to three output blocks ("parts") that share the input rows:
// part q writes out_q[t][o] = act(sum_k x_q[t][k] W_q[o][k] + b_q[o]), where
// x_q is the input row, or its LayerNorm with (ln_g, ln_b) when ln_g is set
// (then K <= kLinearLnMaxK).
struct LinearPart {
    const uint16_t* W;      // [N][K]
    const uint16_t* bias;   // [N]
    const uint16_t* ln_g;   // [K] or nullptr
    const uint16_t* ln_b;   // [K]
    uint16_t* out;          // [n][N] bf16 (plain output, or the mixture when last)
    int32_t N;
};
constexpr int kLinearLnMaxK = 256;
constexpr int kLinearTab = 64;   // pointer-table entries of a grouped launch
// Grouped launches: blockIdx.z = group g < groups (0 or 1: one group).  The
// input rows, W, bias and LayerNorm parameters, output, residual, mixture and
// gates of group g sit at their pointer plus g times their group stride; a
// non-null in_tab[0] gives the input rows of group g as in_tab[g / tab_div]
// instead, a non-null out_tab[0] the output as out_tab[g].
struct LinearProblem {
    const uint16_t* in;   // [n] rows of K inputs, row stride ld_in elements
    size_t ld_in;
    LinearPart part[3];
    int32_t nparts;
    // residual and mixture apply to a single part
    const uint16_t* res;  // [n] rows of N: residual added after the activation, or nullptr
    size_t ld_res;        // row stride of res in elements (0: N)
    size_t ld_out;        // row stride of the part's plain output in elements (0: N)
    float* mix_acc;       // [n][N] fp32 mixture accumulator (mix)
    const float* gates;   // gate of row t, expert e: gates[t * gate_ld + e] (mix)
    int32_t gate_ld, expert;
    int32_t n, K;
    int32_t gelu, mix, first, last;
    int32_t groups, tab_div;
    size_t in_gs, w_gs, out_gs, res_gs, mix_gs, gate_gs;
    const uint16_t* in_tab[kLinearTab];
    uint16_t* out_tab[kLinearTab];
};

// LayerNorm of n bf16 rows of width w (w % 8 == 0, w <= 4096): out = LN(in; g, b)
// and, when out2 is set, out2 = LN(in; g2, b2) on the same statistics.
struct LnProblem {
    const uint16_t* in;   // [n] rows, row stride ld_in elements
    size_t ld_in;
    const uint16_t *g, *b, *g2, *b2;   // [w] each
    uint16_t *out, *out2;              // [n][w]
    int32_t n, w;
    // grouped launches (blockIdx.y = group g < groups; 0 or 1: one): the rows
    // of group g at in + g * in_gs, its parameters at g, b, g2, b2 + g * p_gs,
    // its outputs at out, out2 + g * out_gs
    int32_t groups;
    size_t in_gs, p_gs, out_gs;
};

hipError_t launch_ln_rows(const LnProblem& p, hipStream_t stream);
hipError_t launch_linear(const LinearProblem& p, hipStream_t stream);
hipError_t launch_topS_select(const float* A, int32_t* idx, int B, int T, int S, hipStream_t stream);
hipError_t launch_replay_attention(const ReplayProblem& p, hipStream_t stream);

// Kernel launchers (each enqueues on `stream`; return hipGetLastError()).
hipError_t launch_router(const Problem& p, const UnitTab& ut, bool bf16, hipStream_t stream);
hipError_t launch_f32_gemm1(const Problem& p, const UnitTab& ut, hipStream_t stream);
hipError_t launch_f32_gemm2(const Problem& p, const UnitTab& ut, hipStream_t stream);
// fp32 on the matrix cores (k_f32_mfma.hip): the router runs inside layer 1,
// which also writes p.gates; used when f32_mfma_fits
bool f32_mfma_fits(const Problem& p);
hipError_t launch_f32_mfma_gemm1(const Problem& p, const UnitTab& ut, hipStream_t stream);
hipError_t launch_f32_mfma_gemm2(const Problem& p, const UnitTab& ut, hipStream_t stream);
hipError_t launch_bf16_gemm1(const Problem& p, const UnitTab& ut, hipStream_t stream);
hipError_t launch_bf16_gemm2(const Problem& p, const UnitTab& ut, hipStream_t stream);
// 256 x 256-tile forms of the same two products (k_bf16_gemm256.hip), used
// when a launch of n_units units fills at least half a round of the chip
bool bf16_gemm256_fits(const Problem& p, int n_units);
hipError_t launch_bf16_gemm1_256(const Problem& p, const UnitTab& ut, hipStream_t stream);
hipError_t launch_bf16_gemm2_256(const Problem& p, const UnitTab& ut, hipStream_t stream);
// Routed (Top-K sparse) two-GEMM path on the same tiles: each plan tile is up
// to 256 assignments of one translator; the hidden buffer of a unit holds
// bf16_routed_hidden_bytes(p) in assignment order.
bool bf16_routed_gemm_fits(const Problem& p);
size_t bf16_routed_hidden_bytes(const Problem& p);
hipError_t launch_bf16_gemm1_routed(const Problem& p, const UnitTab& ut, hipStream_t stream);
hipError_t launch_bf16_gemm2_routed(const Problem& p, const UnitTab& ut, hipStream_t stream);
// Fused single-kernel path (router + both layers + mix + store); returns
// hipErrorNotSupported when the sizes have no fused instantiation.
bool fused_supported(const Problem& p);
hipError_t launch_bf16_fused(const Problem& p, const UnitTab& ut, hipStream_t stream);
// Routed path: router -> per-token Top-K lists; per-unit counting sort of the
// (token, translator) assignments into translator-contiguous lists and row
// tiles; the fused kernel over tiles (one translator each); for top_k > 1, a
// combine of the top_k per-assignment rows of every token.
int fused_tile_rows(const Problem& p);
hipError_t launch_router_lists(const Problem& p, const UnitTab& ut, hipStream_t stream);
hipError_t launch_usage_stats(const uint32_t* counts, int n, int E, double* cv2, double* entropy,
                              hipStream_t stream);
hipError_t launch_route_plan(const Problem& p, const UnitTab& ut, hipStream_t stream);
hipError_t launch_bf16_fused_routed(const Problem& p, const UnitTab& ut, hipStream_t stream);
hipError_t launch_routed_combine(const Problem& p, const UnitTab& ut, hipStream_t stream);

}  // namespace mot
