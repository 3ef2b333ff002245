/*
 * libmot — Mixture-of-Translators KV-cache translation on AMD Instinct MI355X
 * (gfx950).  Plain C ABI: device pointers, host structs of sizes, status codes.
 *
 * Operation (paper Sec. 2.1 "Problem Setup", paragraphs "Translation" and
 * "Communication"; Sec. 3, Definition "Mixture-of-Translators", Eq.
 * mot_definition; translator activation phi = GELU, App. C.2):
 *
 *   A source model's context KV cache is translated into the target model's
 *   cache space.  A channel (i, j) connects source layer i to target layer j;
 *   layer_map[j] = i lists the channels (App. C.3 "Depth-Ratio Mapping" gives
 *   the default map, mot_depth_ratio_map below).  For every channel, for keys
 *   and for values separately, every context token row z (the source cache row
 *   of one token, flattened head-major: index h*D_src + d) is translated as
 *
 *       g      = softmax(Wr z + br)                   (E nonnegative gates)
 *       Tr_m z = W2_m GELU(W1_m z + b1_m) + b2_m     (m = 0..E-1)
 *       S      = the top_k largest g_m (ties: lower index), 1 <= top_k <= E
 *       out    = sum_{m in S} (g_m / sum_{r in S} g_r) Tr_m z
 *
 *   and written into target layer j, un-flattened as (h', d') =
 *   (o / D_tgt, o % D_tgt).  top_k = E is the dense mixture.  GELU is
 *   x * Phi(x) with the exact erf in MOT_F32; every MOT_BF16 kernel evaluates
 *   the tanh form of GELU (Hendrycks & Gimpel), whose largest deviation from
 *   the erf form is 4.7e-4 absolute (at |x| ~ 2.7), well below the bf16
 *   rounding of the hidden activation that follows it.
 *
 * Terms.  d_in = H_src*D_src, d_out = H_tgt*D_tgt, N_tok = B*T.  A "unit" is
 * one (target layer j, X in {K, V}) with layer_map[j] >= 0.
 */
#ifndef MOT_H
#define MOT_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MOT_ABI_VERSION 5
#define MOT_MAX_LAYERS 256   /* L_src, L_tgt <= MOT_MAX_LAYERS               */
#define MOT_MAX_EXPERTS 16   /* E <= MOT_MAX_EXPERTS                         */

typedef enum {
    MOT_OK = 0,
    MOT_ERR_NULL_ARG = 1,            /* a required pointer is NULL                */
    MOT_ERR_BAD_SHAPE = 2,           /* a size is <= 0, too large, or inconsistent */
    MOT_ERR_BAD_LAYER_MAP = 3,       /* layer_map[j] >= L_src or < -1             */
    MOT_ERR_UNSUPPORTED = 4,         /* valid but not implemented (see below)     */
    MOT_ERR_MISALIGNED = 5,          /* a device pointer is not 16-byte aligned   */
    MOT_ERR_WORKSPACE_TOO_SMALL = 6, /* caller workspace below the minimum        */
    MOT_ERR_HIP = 7                  /* a HIP runtime call or launch failed       */
} mot_status;

typedef enum { MOT_F32 = 0, MOT_BF16 = 1 } mot_dtype;
typedef enum { MOT_LAYOUT_BTHD = 0, MOT_LAYOUT_BHTD = 1 } mot_layout;
typedef enum { MOT_ACT_GELU = 0, MOT_ACT_IDENTITY = 1 } mot_act;
typedef enum { MOT_ALGO_AUTO = 0, MOT_ALGO_UNFUSED = 1, MOT_ALGO_FUSED = 2, MOT_ALGO_ROUTED = 3 } mot_algo;

/*
 * Problem sizes and options (host struct, read during the call only).
 *   L_src, L_tgt   source / target layer counts (1..MOT_MAX_LAYERS)
 *   B, T           batch and context tokens (B*T >= 0; 0 is a no-op)
 *   H_src, D_src   source KV heads and head dim
 *   H_tgt, D_tgt   target KV heads and head dim
 *   E              translators per unit (1..MOT_MAX_EXPERTS)
 *   top_k          translators used per token, 1..E: the top_k largest softmax
 *                  scores are kept and renormalised to sum to one, the others
 *                  are zero (ties go to the lower translator index); top_k = E
 *                  is the dense mixture.  MOT_ALGO_ROUTED runs each translator
 *                  only on the tokens that selected it; MOT_ALGO_FUSED and
 *                  MOT_ALGO_UNFUSED evaluate every translator and give the
 *                  unselected ones a gate of exactly zero.
 *   hidden         translator hidden width
 *   dtype          MOT_F32: fp32 storage and math (erf GELU, expf softmax).
 *                  MOT_BF16: bf16 storage; fp32 accumulation; fp32 gates;
 *                  tanh-form GELU (within 4.7e-4 absolute of the erf form);
 *                  the gate-scaled hidden activation is rounded to bf16
 *                  before the second translator layer; outputs rounded to
 *                  nearest even.
 *   src_layout     layout of each source layer: BTHD [B][T][H][D] or BHTD
 *   dst_layout     layout of each target layer, same encoding
 *   act            MOT_ACT_GELU (the method) or MOT_ACT_IDENTITY (tests)
 *   algo           kernel path: MOT_ALGO_AUTO picks (bf16: ROUTED when
 *                  top_k < E, else FUSED when the fused kernel fits, else
 *                  UNFUSED; fp32: UNFUSED); MOT_ALGO_FUSED = one kernel per
 *                  token tile over every translator (bf16 only; d_in and d_out
 *                  in {128, 256, 512}; no workspace); MOT_ALGO_ROUTED = Top-K
 *                  sparse (bf16 only): a router pass writes each token's top_k
 *                  translators, a per-unit counting sort groups the (token,
 *                  translator) pairs by translator, each translator runs only
 *                  on its tokens (the fused kernel over translator tiles where
 *                  it fits, else the two GEMMs over translator tiles of up to
 *                  256 pairs), and for top_k > 1 a combine sums each token's
 *                  top_k rows (workspace needed); MOT_ALGO_UNFUSED = router,
 *                  then two grouped GEMMs over every translator through a
 *                  hidden-activation workspace (the fp32 matrix-core GEMMs,
 *                  used when hidden % 64 == 0, compute the router inside the
 *                  first one).  Requesting an impossible path
 *                  returns MOT_ERR_UNSUPPORTED.  All paths compute the same
 *                  function.
 *   streams        2 (or 0): keys and values, each with its own translators;
 *                  1: one activation stream per layer (the MoT-h variant,
 *                  paper App. C.5): src_k -> dst_k with translators indexed
 *                  [L_tgt][1][E]...; src_v and dst_v are ignored (may be
 *                  NULL).  mot_restore_kv then forms K and V from it.
 *   workspace      optional device scratch; NULL = library-owned buffer
 *   workspace_bytes size of `workspace` in bytes
 *   usage          optional device uint32 [L_tgt][streams][E], 4-byte aligned:
 *                  translator usage (paper Sec. 4, "MoT Architecture
 *                  Ablation": I_m, the cumulative selection count of
 *                  translator m).  For every mapped unit (j, x) and every
 *                  context token, usage[j][x][m] is incremented once for each
 *                  translator m of the token's Top-K set, so each call adds
 *                  top_k * B * T to a unit's row (B * T per translator when
 *                  top_k = E).  Counts accumulate over calls (zero the array
 *                  to start; they wrap at 2^32); rows of unmapped layers are
 *                  not touched; NULL = not counted.  mot_usage_stats turns
 *                  the counts into the paper's usage imbalance and entropy.
 *
 * Supported sizes (others return MOT_ERR_UNSUPPORTED):
 *   MOT_BF16: D_src, D_tgt multiples of 8; d_in multiple of 64;
 *             hidden multiple of 64; d_out multiple of 32.
 *   MOT_F32:  D_src, D_tgt multiples of 4; d_in, hidden multiples of 4.
 */
typedef struct {
    int32_t L_src, L_tgt;
    int32_t B, T;
    int32_t H_src, D_src;
    int32_t H_tgt, D_tgt;
    int32_t E, top_k, hidden;
    int32_t dtype, src_layout, dst_layout, act, algo;
    int32_t streams;
    void* workspace;
    size_t workspace_bytes;
    uint32_t* usage;
} mot_shapes;

/*
 * Translator weights: host struct of device pointers, element type = dtype,
 * nn.Linear layout ([out][in]); index 1 of every array is 0 = keys, 1 = values.
 *   w1 [L_tgt][2][E][hidden][d_in]     b1 [L_tgt][2][E][hidden]   (may be NULL)
 *   w2 [L_tgt][2][E][d_out][hidden]    b2 [L_tgt][2][E][d_out]    (may be NULL)
 * Weights are indexed by TARGET layer: two target layers that read the same
 * source layer still have their own translators.
 */
typedef struct {
    const void* w1;
    const void* b1;
    const void* w2;
    const void* b2;
} mot_translator_weights;

/* Router (gate) weights, element type = dtype:
 *   w [L_tgt][2][E][d_in]    b [L_tgt][2][E] (may be NULL)                   */
typedef struct {
    const void* w;
    const void* b;
} mot_router_weights;

/*
 * mot_translate — translate the source context cache into the target layout.
 *
 *   src_k, src_v  device, [L_src] x (src_layout) of dtype
 *   layer_map     HOST int32[L_tgt]; layer_map[j] in [0, L_src) reads that
 *                 source layer, -1 leaves target layer j untouched
 *   tw, rw        translator / router weights (above)
 *   dst_k, dst_v  device, [L_tgt] x (dst_layout) of dtype; only mapped layers
 *                 are written
 *   shapes        sizes and options (above)
 *   stream        HIP stream the work is enqueued on (0 = default stream)
 *
 * B*T == 0 is a valid no-op that inspects no pointer.
 *
 * Asynchronous with respect to the host; results are ready when `stream`
 * reaches this point.  All argument checks run before anything is enqueued:
 * on any error nothing is launched and the outputs are untouched.  Device
 * pointers must be 16-byte aligned; dst must not overlap src, weights or the
 * workspace.  With workspace == NULL the library uses a per-device buffer it
 * owns (grown with hipMalloc on first need, kept until process exit); calls
 * that overlap in time on different streams of one device must then pass
 * their own workspaces.  No call retains any pointer after it returns.
 */
mot_status mot_translate(const void* src_k, const void* src_v, const int32_t* layer_map,
                         const mot_translator_weights* tw, const mot_router_weights* rw,
                         void* dst_k, void* dst_v, const mot_shapes* shapes,
                         hipStream_t stream);

/*
 * Workspace bytes mot_translate needs for `shapes` (its dtype, sizes and
 * options; the workspace fields are ignored).  0 when the chosen kernels need
 * none.  A smaller caller workspace that is still >= the per-unit minimum is
 * accepted and processed in smaller unit groups.  Returns SIZE_MAX when the
 * shapes are invalid or unsupported (mot_last_error() says why).
 */
size_t mot_workspace_bytes(const mot_shapes* shapes);

/*
 * Depth-ratio channel map (paper App. C.3, "Depth-Ratio Mapping"): target
 * layer j reads source layer floor(j * L_src / L_tgt), in exact integer
 * arithmetic.  out: host int32[L_tgt].
 */
mot_status mot_depth_ratio_map(int32_t L_src, int32_t L_tgt, int32_t* out);

/*
 * Translator usage statistics (paper Sec. 4, "MoT Architecture Ablation",
 * Table "mot_analysis") of n rows of selection counts I[n][E] (as written
 * by mot_translate's usage output; device uint32):
 *     cv2[r]     = Var_m(I[r][m]) / Mean_m(I[r][m])^2   (population variance
 *                  over the E translators: the usage imbalance CV^2)
 *     entropy[r] = -sum_m p_m ln p_m,  p_m = I[r][m] / sum_m I[r][m]
 *                  (natural log, 0 ln 0 = 0: the usage entropy)
 * in double precision; both are NaN for a row of zeros.  cv2 and entropy:
 * device double [n], 8-byte aligned, not overlapping the counts.  1 <= E <=
 * MOT_MAX_EXPERTS; n = 0 is a no-op.  Asynchronous on `stream`; every check
 * runs before the launch.
 */
mot_status mot_usage_stats(const uint32_t* counts, int32_t n, int32_t E, double* cv2, double* entropy,
                           hipStream_t stream);

/* Static text for a status code. */
const char* mot_status_string(mot_status status);

/* Detail of the last error raised on the calling thread ("" if none). */
const char* mot_last_error(void);

/*
 * Key/value restoration for the activation-translation variant MoT-h (paper
 * App. C.5): the target's key and value projections applied to a translated
 * intermediate activation a (as written by mot_translate with streams = 1):
 *     K[l][t] = W^K[l] a[l][t] + b^K[l],    V[l][t] = W^V[l] a[l][t] + b^V[l]
 * for every layer l with layer_map[l] >= 0 (NULL: every layer).
 *
 *   act        device bf16 [L][B][T][d_act]
 *   wk, wv     device bf16 [L][d_kv][d_act], d_kv = H_tgt * D_tgt (nn.Linear layout)
 *   bk, bv     device bf16 [L][d_kv] or NULL (zero)
 *   dst_k/v    device bf16 [L] x dst_layout ([B][T][H_tgt][D_tgt] or [B][H_tgt][T][D_tgt])
 *   layer_map  HOST int32[L] or NULL; layers with a negative entry are not written
 * Requires dtype MOT_BF16, d_act a multiple of 64, D_tgt a multiple of 8
 * (MOT_ERR_UNSUPPORTED otherwise).  Same error discipline as mot_translate:
 * every check runs before anything is enqueued.
 */
typedef struct {
    int32_t L, B, T;
    int32_t d_act;
    int32_t H_tgt, D_tgt;
    int32_t dtype, dst_layout;
} mot_restore_shapes;

mot_status mot_restore_kv(const void* act, const int32_t* layer_map, const void* wk, const void* bk,
                          const void* wv, const void* bv, void* dst_k, void* dst_v,
                          const mot_restore_shapes* shapes, hipStream_t stream);

/*
 * Context replay after translation (paper App. C.4, "Post-Translation Phase:
 * Cache Replay", Top-S source-guided sparse attention).  Query position u of
 * a target layer attends only to the S context positions that the source
 * model attended to most at the guiding source layer (head-averaged map A),
 * or, in the bottom L_Full layers, to every position 0..u.
 *
 *   B, T       batch rows, context tokens
 *   H_q, H_kv  target query heads and KV heads (H_q a multiple of H_kv; query
 *              head h reads KV head h / (H_q / H_kv), at most 16 per KV head;
 *              H_kv * D below 2^20)
 *   D          head dim: 64 or 128
 *   S          Top-S budget: a multiple of 32, 32 .. 256 (at most 192 when
 *              D = 128); the paper uses 128
 *   kv_layout  K and V in MOT_LAYOUT_BTHD ([B][T][H_kv][D]) or MOT_LAYOUT_BHTD
 *   workspace, workspace_bytes
 *              optional device scratch of mot_replay_attention without key
 *              sets (16-byte aligned, at least mot_replay_workspace_bytes);
 *              NULL = the library's per-device buffer (see below)
 */
typedef struct {
    int32_t B, T;
    int32_t H_q, H_kv, D;
    int32_t S;
    int32_t kv_layout;
    void* workspace;
    size_t workspace_bytes;
} mot_replay_shapes;

/*
 * mot_replay_attention for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same operation, arguments and checks, but the full causal
 * path (idx = NULL) stages V in a static 32 MiB array that the library holds
 * on each device it runs on until the process ends, instead of a workspace
 * or a library-allocated buffer; it calls no hipMalloc, hipFree or
 * allocating routine.  shapes->workspace and workspace_bytes are ignored.
 * Shapes whose staged V (mot_replay_workspace_bytes) exceeds 32 MiB return
 * MOT_ERR_WORKSPACE_TOO_SMALL before anything is launched.  All calls on one
 * device share that array (its contents after a call are unspecified): calls
 * that overlap in time on one device race.  With key sets (idx != NULL) no
 * scratch is used.
 */
mot_status mot_replay_attention_noalloc(const void* q, const void* k, const void* v, const int32_t* idx, void* o,
                                        const mot_replay_shapes* shapes, hipStream_t stream);

/* Scratch bytes mot_replay_attention needs for `shapes` with idx = NULL (V
 * staged transposed: B * H_kv * D * T rounded up to 64, bf16); 0 with key
 * sets; SIZE_MAX for invalid or unsupported shapes. */
size_t mot_replay_workspace_bytes(const mot_replay_shapes* shapes, int with_sets);

/*
 * Top-S key sets (App. C.4, N(u) = Top-S of A[u, 1:u]): for every b and u,
 * the S positions v <= u with the largest A[b][u][v] (ties: lower v), written
 * in ascending order to idx[b][u][0..S) and padded with -1 (all of 0..u when
 * u < S).  A: device fp32 [B][T][T] head-averaged source attention (entries
 * v > u are not read); idx: device int32 [B][T][S].  Only B, T and S of
 * `shapes` are used (T at most 65536).  Both pointers 4-byte aligned and
 * non-overlapping.
 */
mot_status mot_topS_select(const float* A, int32_t* idx, const mot_replay_shapes* shapes, hipStream_t stream);

/*
 * Replay attention of one target layer: for every b, u and query head h,
 *     o[b][u][h] = sum_{v in N(u)} softmax_v(q[b][u][h] . k[v] / sqrt(D)) v[v]
 * with N(u) = the entries of idx[b][u] that lie in 0..u (others, such as the
 * -1 padding, are skipped; a set with none gives zeros), or the full causal
 * set 0..u when idx is NULL.  q, o: device bf16 [B][T][H_q][D]; k, v: device
 * bf16 in kv_layout; idx: device int32 [B][T][S] or NULL.  Softmax and
 * accumulation in fp32; o rounded to bf16.  All pointers 16-byte aligned; o
 * must not overlap an input.  With idx NULL the call stages V transposed
 * (mot_replay_workspace_bytes) in shapes->workspace, or, when that is NULL,
 * in the per-device buffer that mot_translate uses without a workspace (so
 * such calls and those of mot_translate or mot_backbone_translate without
 * workspaces that overlap in time on one device race; calls with their own
 * workspaces do not).  A workspace below the need returns
 * MOT_ERR_WORKSPACE_TOO_SMALL; it must not overlap q, k, v or o.  With idx
 * NULL, (T + 64) * row stride * 2 bytes must stay under 2^31 (row stride:
 * H_kv * D in BTHD, D in BHTD), else MOT_ERR_UNSUPPORTED.
 */
mot_status mot_replay_attention(const void* q, const void* k, const void* v, const int32_t* idx, void* o,
                                const mot_replay_shapes* shapes, hipStream_t stream);

/*
 * The backbone translator body (paper App. C.2, "Backbone Translator") as the
 * experts of the mixture, over channel windows of N = dims->n_slots slots (0
 * or 1: one slot per unit).  Window w covers target layers wN .. wN+N-1 (so
 * L_tgt must be a multiple of N); its slot r reads source layer
 * layer_map[wN + r], and a window is either fully mapped or fully -1
 * (skipped).  Keys and values are translated separately; one unit is a
 * (window, K or V).  For each batch row, over the context positions t,
 * expert m computes
 *     z_r = GELU(W_in LN_in(x_r[t]) + b_in)                     r = 1..N (d_h)
 *     h_0 = z_1;  for r = 1..N (block CAB_r, its own parameters):
 *       h~  = h_{r-1} + Wo CausalMHA(Wq LN_Q(h_{r-1}) + bq, Wk LN_C(z_r) + bk,
 *                                    Wv LN_C(z_r) + bv) + bo
 *       h_r = h~ + W_f2 GELU(W_f1 LN_F(h~) + b_f1) + b_f2
 *     y_t = GELU(W_out LN_out(Concat(h_1..h_N)) + b_out)          (N d_out)
 * (n_heads heads of width d_h / n_heads, softmax(q.k / sqrt(width)) over the
 * positions s <= t of the same batch row; LN with population variance,
 * eps 1e-5); the output row is sum_m g~_m y_t^(m) with Top-K gates from a
 * router over the window's concatenated source rows, and its slice
 * [r d_out, (r+1) d_out) is written to target layer wN + r.  One translator
 * stage (one scan) per expert.
 *
 *   params   device bf16 [L_tgt/N][2][E][P], P = mot_backbone_param_count():
 *            per expert, in order: ln_in_g[d_in] ln_in_b[d_in] w_in[d_h][d_in]
 *            b_in[d_h]; then for each slot r = 1..N: ln_q_g[d_h] ln_q_b[d_h]
 *            ln_c_g[d_h] ln_c_b[d_h] wq[d_h][d_h] bq[d_h] wk[d_h][d_h] bk[d_h]
 *            wv[d_h][d_h] bv[d_h] wo[d_h][d_h] bo[d_h] ln_f_g[d_h] ln_f_b[d_h]
 *            w_f1[d_ff][d_h] b_f1[d_ff] w_f2[d_h][d_ff] b_f2[d_h]; then
 *            ln_out_g[N d_h] ln_out_b[N d_h] w_out[N d_out][N d_h]
 *            b_out[N d_out]
 *   router   w [L_tgt/N][2][E][N d_in], b [L_tgt/N][2][E] (bias optional);
 *            with N = 1 the layout of mot_translate's router
 *   shapes   as for mot_translate (including the optional usage counts of
 *            the Top-K selections, here [L_tgt/N][2][E]: one row per
 *            window and K/V); dtype MOT_BF16, both layouts
 *            MOT_LAYOUT_BTHD, streams 2; hidden, act and algo are not used.
 *            workspace: device scratch of at least
 *            mot_backbone_workspace_bytes (16-byte aligned, not overlapping
 *            any other argument), or NULL for the per-device buffer that
 *            mot_translate uses without a workspace (calls of either that
 *            overlap in time on one device then race)
 * Requires d_in and d_h multiples of 64 up to 4096, N d_h up to 4096, d_ff a
 * multiple of 64, D_tgt a multiple of 8, head width d_h / n_heads of 64 or
 * 128, N <= 8, (T + 64) d_h 2 < 2^31 (MOT_ERR_UNSUPPORTED / MOT_ERR_BAD_SHAPE
 * otherwise; a window mixing mapped and unmapped slots is
 * MOT_ERR_BAD_LAYER_MAP).  Every check runs before any enqueue.
 */
typedef struct {
    int32_t d_h;       /* translator width                               */
    int32_t n_heads;   /* attention heads                                */
    int32_t d_ff;      /* feed-forward width                             */
    int32_t n_slots;   /* channel-window slots N (0 or 1: one per unit)  */
} mot_backbone_dims;

/* Elements per expert of the packed parameters (0 for invalid arguments). */
size_t mot_backbone_param_count(const mot_shapes* shapes, const mot_backbone_dims* dims);

/* Scratch bytes mot_backbone_translate needs (the router's gates for every
 * unit, one unit's activations and the attention's staged V); SIZE_MAX for
 * invalid or unsupported arguments. */
size_t mot_backbone_workspace_bytes(const mot_shapes* shapes, const mot_backbone_dims* dims);

mot_status mot_backbone_translate(const void* src_k, const void* src_v, const int32_t* layer_map,
                                  const void* params, const mot_router_weights* router, void* dst_k, void* dst_v,
                                  const mot_shapes* shapes, const mot_backbone_dims* dims, hipStream_t stream);

/* MOT_ABI_VERSION of the loaded library. */
int mot_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* MOT_H */
