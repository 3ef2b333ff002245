/*
 * Plain CPU oracle for the Mixture-of-Translators (MoT) KV-cache translation.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, obviously-correct
 * definition that the HIP library is checked against.  Only the tests, the
 * smoke check and the benchmark's CPU-baseline leg may load it.  It shares no
 * code, header, table or helper with the GPU library, and it never imports it.
 *
 * What it computes (paper: Sec. 3 "Mixture-of-Translators", Definition
 * "Mixture-of-Translators", Eq. (mot_definition); problem statement in
 * Sec. 2.1 "Problem Setup", paragraphs "Translation" and "Communication"):
 *
 *   for every channel (source layer i -> target layer j), i = layer_map[j] >= 0,
 *   for X in {K, V} (keys and values translated independently, App. C.2;
 *                   streams = 1: the single intermediate-activation stream
 *                   of the MoT-h variant, App. C.5),
 *   for every context token u = (b, t):
 *     z_u            = the source cache row of token u in layer i, flattened
 *                      head-major (index h*D_src + d)
 *     l_m            = sum_c Wr[m][c] z_u[c] + br[m]              (gate logits)
 *     g_m            = exp(l_m - max l) / sum_r exp(l_r - max l)  (nonnegative)
 *     TopK(u)        = indices of the top_k largest g_m (ties: lower index)
 *     gt_m           = g_m / sum_{r in TopK(u)} g_r,  m in TopK(u)
 *     Tr_m(z)        = W2_m act(W1_m z + b1_m) + b2_m             (translator)
 *     out_u          = sum_{m in TopK(u), ascending} gt_m Tr_m(z_u)
 *     dst[j] row u   = out_u, un-flattened as (h', d') = (o / D_tgt, o % D_tgt)
 *
 *   Target layers with layer_map[j] < 0 are not written.
 *
 * act is the exact erf GELU, 0.5 a (1 + erf(a / sqrt 2)) (the paper's phi,
 * App. C.2), or the identity (used by closed-form pins).
 *
 * Precision: inputs arrive as float (bf16 values are widened exactly by the
 * caller); every sum, exp and erf is evaluated in double; outputs are double.
 * Sums run in plain index order with no blocking or reordering.
 *
 * Parity pins (each checked by a CPU test, see tests/test_oracle_pins.py):
 * one-hot gate == single translator; E = 1 identity translators pass the
 * mapped source rows through; uniform gate == mean of the translators;
 * identity activation == closed-form matrix product; GELU against tabulated
 * normal-CDF values; brute-force scalar loops on 2-token, 2-dim shapes;
 * token and expert permutation invariance; depth-ratio map properties.
 *
 * Also here: the key/value restoration of the activation-translation variant
 * MoT-h (App. C.5), pinned by hand-computed values, the identity projection,
 * a float64 matrix product and an identity-translator chain; and the context
 * replay step after translation (App. C.4): Top-S source-guided key
 * selection and attention over the selected (or the full causal) key set,
 * pinned by worked examples, sorting, single-key and uniform-score cases and
 * numpy softmax attention; and the backbone translator body (App. C.2) as
 * the experts of the mixture, pinned by a numpy implementation, a closed
 * form (zero output weights), causality and batch-row independence.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* Problem dimensions.  Independent of the GPU library's own struct. */
typedef struct {
    int32_t L_src, L_tgt;   /* source / target layer counts                 */
    int32_t B, T;           /* batch, context tokens                        */
    int32_t H_src, D_src;   /* source KV heads, head dim                    */
    int32_t H_tgt, D_tgt;   /* target KV heads, head dim                    */
    int32_t E;              /* number of translators N_Tr                   */
    int32_t top_k;          /* translators used per token (1..E)            */
    int32_t hidden;         /* translator hidden width                      */
    int32_t src_layout;     /* 0: [L][B][T][H][D]   1: [L][B][H][T][D]      */
    int32_t dst_layout;     /* same encoding for the target cache           */
    int32_t act;            /* 0: exact-erf GELU    1: identity             */
    int32_t streams;        /* 2: keys and values; 1: one activation stream
                               (MoT-h, App. C.5): weights [L_tgt][streams][E] */
} mot_oracle_dims;

enum { OR_OK = 0, OR_BAD_ARG = 1, OR_NO_MEM = 2 };

/* ------------------------------------------------------------------ */
/* index helpers                                                       */
/* ------------------------------------------------------------------ */

static size_t cache_index(const mot_oracle_dims* s, int layout, int32_t H, int32_t D,
                          int32_t layer, int32_t b, int32_t t, int32_t h, int32_t d)
{
    size_t L_stride = (size_t)s->B * s->T * H * D;
    if (layout == 0) /* [L][B][T][H][D] */
        return (size_t)layer * L_stride + (((size_t)b * s->T + t) * H + h) * D + d;
    /* [L][B][H][T][D] */
    return (size_t)layer * L_stride + (((size_t)b * H + h) * s->T + t) * D + d;
}

static double act_fn(int act, double a)
{
    if (act == 1) return a;
    return 0.5 * a * (1.0 + erf(a / sqrt(2.0)));
}

/* ------------------------------------------------------------------ */
/* one token row of one channel, straight from the definition          */
/* ------------------------------------------------------------------ */

typedef struct {
    const float *w1, *b1, *w2, *b2, *wr, *br;   /* b* may be NULL (zero)  */
} oracle_weights;

/* scratch: z[d_in], logits[E], g[E], sel[E], a[hidden], y[d_out] */
static void translate_row(const mot_oracle_dims* s, const oracle_weights* w,
                          int32_t j, int32_t x, const double* z,
                          double* out, double* gates_out,
                          double* logits, double* g, int* sel, double* hid, double* y)
{
    const int32_t d_in = s->H_src * s->D_src;
    const int32_t d_out = s->H_tgt * s->D_tgt;
    const int32_t E = s->E, Hd = s->hidden;
    const size_t unit = (size_t)j * s->streams + x;

    /* gate logits l_m = Wr z + br */
    for (int32_t m = 0; m < E; ++m) {
        const float* wr = w->wr + (unit * E + m) * d_in;
        double acc = 0.0;
        for (int32_t c = 0; c < d_in; ++c) acc += (double)wr[c] * z[c];
        if (w->br) acc += (double)w->br[unit * E + m];
        logits[m] = acc;
    }
    /* softmax: nonnegative scores that sum to one */
    double mx = logits[0];
    for (int32_t m = 1; m < E; ++m) if (logits[m] > mx) mx = logits[m];
    double den = 0.0;
    for (int32_t m = 0; m < E; ++m) { g[m] = exp(logits[m] - mx); den += g[m]; }
    for (int32_t m = 0; m < E; ++m) g[m] /= den;

    /* Top-K selection: repeatedly take the largest remaining score; on a tie
     * the lower index wins because the scan is ascending with strict '>'. */
    for (int32_t m = 0; m < E; ++m) sel[m] = 0;
    for (int32_t k = 0; k < s->top_k; ++k) {
        int32_t best = -1;
        for (int32_t m = 0; m < E; ++m)
            if (!sel[m] && (best < 0 || g[m] > g[best])) best = m;
        sel[best] = 1;
    }
    /* renormalise over the selected set */
    double gsum = 0.0;
    for (int32_t m = 0; m < E; ++m) if (sel[m]) gsum += g[m];

    for (int32_t o = 0; o < d_out; ++o) out[o] = 0.0;
    for (int32_t m = 0; m < E; ++m) {
        double gt = sel[m] ? g[m] / gsum : 0.0;
        if (gates_out) gates_out[m] = gt;
        if (!sel[m]) continue;
        const size_t em = unit * E + m;
        /* hidden = act(W1 z + b1) */
        for (int32_t k = 0; k < Hd; ++k) {
            const float* w1 = w->w1 + (em * Hd + k) * d_in;
            double acc = 0.0;
            for (int32_t c = 0; c < d_in; ++c) acc += (double)w1[c] * z[c];
            if (w->b1) acc += (double)w->b1[em * Hd + k];
            hid[k] = act_fn(s->act, acc);
        }
        /* Tr_m(z) = W2 hidden + b2 */
        for (int32_t o = 0; o < d_out; ++o) {
            const float* w2 = w->w2 + (em * d_out + o) * Hd;
            double acc = 0.0;
            for (int32_t k = 0; k < Hd; ++k) acc += (double)w2[k] * hid[k];
            if (w->b2) acc += (double)w->b2[em * d_out + o];
            y[o] = acc;
        }
        /* gated sum, translators in ascending order */
        for (int32_t o = 0; o < d_out; ++o) out[o] += gt * y[o];
    }
}

static void gather_row(const mot_oracle_dims* s, const float* src, int32_t i,
                       int32_t b, int32_t t, double* z)
{
    for (int32_t h = 0; h < s->H_src; ++h)
        for (int32_t d = 0; d < s->D_src; ++d)
            z[h * s->D_src + d] =
                (double)src[cache_index(s, s->src_layout, s->H_src, s->D_src, i, b, t, h, d)];
}

/* ------------------------------------------------------------------ */
/* work distribution: one item = (unit index, row index)               */
/* ------------------------------------------------------------------ */

typedef struct {
    const mot_oracle_dims* s;
    const oracle_weights* w;
    const float *src_k, *src_v;
    const int32_t* layer_map;
    /* either a full run (dst_k/dst_v) or a sampled run (rows/out) */
    double *dst_k, *dst_v;
    const int32_t *unit_j, *unit_x;
    int32_t n_units;
    const int64_t* rows;
    int64_t n_rows;
    double* out;      /* [n_units][n_rows][d_out]  (sampled)  */
    double* gates;    /* [n_units][n_rows][E] or NULL          */
    int64_t n_items;
    int64_t next;     /* shared counter */
    pthread_mutex_t lock;
    int failed;
} oracle_job;

static void* worker(void* arg)
{
    oracle_job* jb = (oracle_job*)arg;
    const mot_oracle_dims* s = jb->s;
    const int32_t d_in = s->H_src * s->D_src, d_out = s->H_tgt * s->D_tgt;
    double* z = (double*)malloc(sizeof(double) * d_in);
    double* lg = (double*)malloc(sizeof(double) * s->E);
    double* g = (double*)malloc(sizeof(double) * s->E);
    int* sel = (int*)malloc(sizeof(int) * s->E);
    double* hid = (double*)malloc(sizeof(double) * s->hidden);
    double* y = (double*)malloc(sizeof(double) * d_out);
    double* row = (double*)malloc(sizeof(double) * d_out);
    double* gt = (double*)malloc(sizeof(double) * s->E);
    if (!z || !lg || !g || !sel || !hid || !y || !row || !gt) {
        pthread_mutex_lock(&jb->lock);
        jb->failed = 1;
        pthread_mutex_unlock(&jb->lock);
        goto done;
    }
    for (;;) {
        int64_t item;
        pthread_mutex_lock(&jb->lock);
        item = jb->next++;
        pthread_mutex_unlock(&jb->lock);
        if (item >= jb->n_items) break;
        int64_t ui = item / jb->n_rows, ri = item % jb->n_rows;
        int32_t j = jb->unit_j[ui], x = jb->unit_x[ui];
        int32_t i = jb->layer_map[j];
        int64_t r = jb->rows ? jb->rows[ri] : ri;
        int32_t b = (int32_t)(r / s->T), t = (int32_t)(r % s->T);
        gather_row(s, x == 0 ? jb->src_k : jb->src_v, i, b, t, z);
        translate_row(s, jb->w, j, x, z, row, gt, lg, g, sel, hid, y);
        if (jb->out) {
            double* o = jb->out + ((size_t)ui * jb->n_rows + ri) * d_out;
            memcpy(o, row, sizeof(double) * d_out);
            if (jb->gates)
                memcpy(jb->gates + ((size_t)ui * jb->n_rows + ri) * s->E, gt,
                       sizeof(double) * s->E);
        } else {
            double* dst = x == 0 ? jb->dst_k : jb->dst_v;
            for (int32_t o = 0; o < d_out; ++o) {
                int32_t hh = o / s->D_tgt, dd = o % s->D_tgt;
                dst[cache_index(s, s->dst_layout, s->H_tgt, s->D_tgt, j, b, t, hh, dd)] = row[o];
            }
        }
    }
done:
    free(z); free(lg); free(g); free(sel); free(hid); free(y); free(row); free(gt);
    return NULL;
}

static int check_dims(const mot_oracle_dims* s, const int32_t* layer_map)
{
    if (!s || !layer_map) return OR_BAD_ARG;
    if (s->L_src <= 0 || s->L_tgt <= 0 || s->B < 0 || s->T < 0 || s->H_src <= 0 ||
        s->D_src <= 0 || s->H_tgt <= 0 || s->D_tgt <= 0 || s->E <= 0 || s->hidden <= 0)
        return OR_BAD_ARG;
    if (s->top_k < 1 || s->top_k > s->E) return OR_BAD_ARG;
    if ((s->src_layout != 0 && s->src_layout != 1) || (s->dst_layout != 0 && s->dst_layout != 1))
        return OR_BAD_ARG;
    if (s->act != 0 && s->act != 1) return OR_BAD_ARG;
    if (s->streams != 1 && s->streams != 2) return OR_BAD_ARG;
    for (int32_t j = 0; j < s->L_tgt; ++j)
        if (layer_map[j] >= s->L_src) return OR_BAD_ARG;
    return OR_OK;
}

static int run_job(oracle_job* jb, int nthreads)
{
    if (jb->n_items == 0) return OR_OK;
    if (nthreads < 1) nthreads = 1;
    if (nthreads > 256) nthreads = 256;
    pthread_t th[256];
    pthread_mutex_init(&jb->lock, NULL);
    int started = 0;
    for (int k = 0; k < nthreads; ++k)
        if (pthread_create(&th[k], NULL, worker, jb) == 0) ++started;
    if (started == 0) worker(jb);
    for (int k = 0; k < started; ++k) pthread_join(th[k], NULL);
    pthread_mutex_destroy(&jb->lock);
    return jb->failed ? OR_NO_MEM : OR_OK;
}

/* ------------------------------------------------------------------ */
/* public entry points (C ABI, loaded by the test harness via ctypes)  */
/* ------------------------------------------------------------------ */

/* Full translation: writes every row of every target layer j with
 * layer_map[j] >= 0 into dst_k / dst_v (double, laid out per dst_layout);
 * other layers are left untouched. */
int mot_oracle_translate(const float* src_k, const float* src_v, const int32_t* layer_map,
                         const float* w1, const float* b1, const float* w2, const float* b2,
                         const float* wr, const float* br,
                         double* dst_k, double* dst_v, const mot_oracle_dims* s, int nthreads)
{
    int rc = check_dims(s, layer_map);
    if (rc) return rc;
    if (!src_k || !w1 || !w2 || !wr || !dst_k) return OR_BAD_ARG;
    if (s->streams == 2 && (!src_v || !dst_v)) return OR_BAD_ARG;
    oracle_weights w = {w1, b1, w2, b2, wr, br};
    int32_t* uj = (int32_t*)malloc(sizeof(int32_t) * 2 * s->L_tgt);
    int32_t* ux = (int32_t*)malloc(sizeof(int32_t) * 2 * s->L_tgt);
    if (!uj || !ux) { free(uj); free(ux); return OR_NO_MEM; }
    int32_t nu = 0;
    for (int32_t j = 0; j < s->L_tgt; ++j)
        if (layer_map[j] >= 0)
            for (int32_t x = 0; x < s->streams; ++x) { uj[nu] = j; ux[nu] = x; ++nu; }
    oracle_job jb;
    memset(&jb, 0, sizeof jb);
    jb.s = s; jb.w = &w; jb.src_k = src_k; jb.src_v = src_v; jb.layer_map = layer_map;
    jb.dst_k = dst_k; jb.dst_v = dst_v; jb.unit_j = uj; jb.unit_x = ux; jb.n_units = nu;
    jb.rows = NULL; jb.n_rows = (int64_t)s->B * s->T;
    jb.n_items = (int64_t)nu * jb.n_rows;
    rc = run_job(&jb, nthreads);
    free(uj); free(ux);
    return rc;
}

/* Sampled translation: for each listed unit (unit_j[u], unit_x[u]) and each
 * listed flattened token row r = b*T + t, writes out[u][k][0..d_out) and,
 * if gates != NULL, the renormalised gates gates[u][k][0..E) (zero for
 * translators outside the Top-K set).  layer_map[unit_j[u]] must be >= 0. */
int mot_oracle_rows(const float* src_k, const float* src_v, const int32_t* layer_map,
                    const float* w1, const float* b1, const float* w2, const float* b2,
                    const float* wr, const float* br, const mot_oracle_dims* s,
                    const int32_t* unit_j, const int32_t* unit_x, int32_t n_units,
                    const int64_t* rows, int64_t n_rows,
                    double* out, double* gates, int nthreads)
{
    int rc = check_dims(s, layer_map);
    if (rc) return rc;
    if (!src_k || !w1 || !w2 || !wr || !out || !unit_j || !unit_x || !rows) return OR_BAD_ARG;
    if (s->streams == 2 && !src_v) return OR_BAD_ARG;
    for (int32_t u = 0; u < n_units; ++u) {
        if (unit_j[u] < 0 || unit_j[u] >= s->L_tgt || unit_x[u] < 0 || unit_x[u] >= s->streams)
            return OR_BAD_ARG;
        if (layer_map[unit_j[u]] < 0) return OR_BAD_ARG;
    }
    for (int64_t k = 0; k < n_rows; ++k)
        if (rows[k] < 0 || rows[k] >= (int64_t)s->B * s->T) return OR_BAD_ARG;
    oracle_weights w = {w1, b1, w2, b2, wr, br};
    oracle_job jb;
    memset(&jb, 0, sizeof jb);
    jb.s = s; jb.w = &w; jb.src_k = src_k; jb.src_v = src_v; jb.layer_map = layer_map;
    jb.unit_j = unit_j; jb.unit_x = unit_x; jb.n_units = n_units;
    jb.rows = rows; jb.n_rows = n_rows; jb.out = out; jb.gates = gates;
    jb.n_items = (int64_t)n_units * n_rows;
    return run_job(&jb, nthreads);
}

/* Depth-ratio channel map (App. C.3, "Depth-Ratio Mapping"): target layer j
 * reads the source layer at the same relative depth, i = floor(j * L_src / L_tgt),
 * computed in exact integer arithmetic.  Lower target layers read lower source
 * layers and the order is preserved. */
int mot_oracle_depth_ratio_map(int32_t L_src, int32_t L_tgt, int32_t* out)
{
    if (L_src <= 0 || L_tgt <= 0 || !out) return OR_BAD_ARG;
    for (int32_t j = 0; j < L_tgt; ++j) out[j] = (int32_t)(((int64_t)j * L_src) / L_tgt);
    return OR_OK;
}

/* Key/value restoration of the activation-translation variant MoT-h
 * (App. C.5, "Hidden States Translation"): the target's fixed key and value
 * projections applied to a translated intermediate activation,
 *     K[l][u] = W^K[l] a[l][u] + b^K[l],    V[l][u] = W^V[l] a[l][u] + b^V[l],
 * for every layer l with layer_map[l] >= 0 (layer_map NULL: every layer).
 *   act   [L][B][T][d_act]        wk, wv [L][d_kv][d_act], d_kv = H_tgt*D_tgt
 *   bk,bv [L][d_kv] or NULL        dst_k, dst_v [L] x dst_layout, double
 * Sums run over c = 0..d_act-1 in order, in double; the bias is added last.
 * Layers that are not restored are left untouched. */
int mot_oracle_restore_kv(const float* act, const int32_t* layer_map,
                          const float* wk, const float* bk, const float* wv, const float* bv,
                          double* dst_k, double* dst_v, int32_t L, int32_t B, int32_t T,
                          int32_t d_act, int32_t H_tgt, int32_t D_tgt, int32_t dst_layout)
{
    if (!act || !wk || !wv || !dst_k || !dst_v) return OR_BAD_ARG;
    if (L <= 0 || B < 0 || T < 0 || d_act <= 0 || H_tgt <= 0 || D_tgt <= 0) return OR_BAD_ARG;
    if (dst_layout != 0 && dst_layout != 1) return OR_BAD_ARG;
    const size_t d_kv = (size_t)H_tgt * D_tgt, n_tok = (size_t)B * T;
    for (int32_t l = 0; l < L; ++l) {
        if (layer_map && layer_map[l] < 0) continue;
        for (int32_t b = 0; b < B; ++b)
            for (int32_t t = 0; t < T; ++t) {
                const float* a = act + ((size_t)l * n_tok + (size_t)b * T + t) * d_act;
                for (int32_t h = 0; h < H_tgt; ++h)
                    for (int32_t d = 0; d < D_tgt; ++d) {
                        const size_t o = (size_t)h * D_tgt + d;
                        const float* rk = wk + ((size_t)l * d_kv + o) * d_act;
                        const float* rv = wv + ((size_t)l * d_kv + o) * d_act;
                        double sk = 0.0, sv = 0.0;
                        for (int32_t c = 0; c < d_act; ++c) {
                            sk += (double)rk[c] * (double)a[c];
                            sv += (double)rv[c] * (double)a[c];
                        }
                        if (bk) sk += (double)bk[(size_t)l * d_kv + o];
                        if (bv) sv += (double)bv[(size_t)l * d_kv + o];
                        size_t idx = (size_t)l * n_tok * d_kv;
                        idx += dst_layout == 0 ? (((size_t)b * T + t) * H_tgt + h) * D_tgt + d
                                               : (((size_t)b * H_tgt + h) * T + t) * D_tgt + d;
                        dst_k[idx] = sk;
                        dst_v[idx] = sv;
                    }
            }
    }
    return OR_OK;
}

/* ------------------------------------------------------------------ */
/* Context replay with Top-S source-guided sparse attention (App. C.4, */
/* "Post-Translation Phase: Cache Replay")                             */
/* ------------------------------------------------------------------ */

/* Selection: for each batch row b and context query position u, the key
 * set N(u) holds the S positions v in 0..u with the largest head-averaged
 * source attention A[b][u][v] (all of 0..u when u + 1 <= S).  Order of
 * preference: larger A first, then the lower position.  The set is written
 * in ascending position order to idx[b][u][0..S), padded with -1.
 * A: [B][T][T] (entries v > u are never read). */
int mot_oracle_topS_select(const float* A, int32_t B, int32_t T, int32_t S, int32_t* idx)
{
    if (!A || !idx || B < 0 || T < 0 || S < 1) return OR_BAD_ARG;
    char* take = (char*)malloc(T > 0 ? T : 1);
    if (!take) return OR_NO_MEM;
    for (int32_t b = 0; b < B; ++b)
        for (int32_t u = 0; u < T; ++u) {
            const float* row = A + ((size_t)b * T + u) * T;
            const int32_t n = u + 1;
            int32_t* out = idx + ((size_t)b * T + u) * S;
            for (int32_t v = 0; v < n; ++v) take[v] = 0;
            /* S rounds of "the best position not yet taken" (ties: lower v) */
            const int32_t k = n < S ? n : S;
            for (int32_t r = 0; r < k; ++r) {
                int32_t best = -1;
                for (int32_t v = 0; v < n; ++v)
                    if (!take[v] && (best < 0 || row[v] > row[best])) best = v;
                take[best] = 1;
            }
            int32_t c = 0;
            for (int32_t v = 0; v < n; ++v)
                if (take[v]) out[c++] = v;
            for (; c < S; ++c) out[c] = -1;
        }
    free(take);
    return OR_OK;
}

/* Replay attention of one target layer: for batch row b, query position u
 * and query head h (KV head h / (H_q / H_kv)), over the key set N(u):
 *     o[b][u][h] = sum_{v in N(u)} p_v V[v],  p = softmax_v(Q[b][u][h] . K[v] / sqrt(D))
 * N(u) = idx[b][u][0..S) without the -1 entries, or, when idx is NULL, the
 * full causal set 0..u (the bottom L_Full layers).
 *   q, o: [B][T][H_q][D];  k, v: [B][T][H_kv][D] (kv_layout 0) or [B][H_kv][T][D] (1).
 * Dot products, exponentials and sums in double, in index order. */
typedef struct {
    const float *q, *k, *v;
    const int32_t* idx;
    int32_t B, T, H_q, H_kv, D, S, kv_layout;
} replay_args;

/* all heads of (b, u) into orow[H_q][D]; sc, keys: scratch of T entries */
static int replay_row(const replay_args* a, int32_t b, int32_t u, double* orow, double* sc, int32_t* keys)
{
    const int32_t G = a->H_q / a->H_kv, D = a->D, T = a->T;
    const double scale = 1.0 / sqrt((double)D);
    int32_t n = 0;
    if (a->idx) {
        const int32_t* row = a->idx + ((size_t)b * T + u) * a->S;
        for (int32_t c = 0; c < a->S; ++c)
            if (row[c] >= 0) {
                if (row[c] > u) return OR_BAD_ARG;
                keys[n++] = row[c];
            }
    } else {
        for (int32_t t = 0; t <= u; ++t) keys[n++] = t;
    }
    for (int32_t h = 0; h < a->H_q; ++h) {
        const int32_t hk = h / G;
        const float* qr = a->q + (((size_t)b * T + u) * a->H_q + h) * D;
        double* oh = orow + (size_t)h * D;
        double mx = -INFINITY;
        for (int32_t c = 0; c < n; ++c) {
            const size_t kr = a->kv_layout == 0 ? (((size_t)b * T + keys[c]) * a->H_kv + hk) * D
                                                : (((size_t)b * a->H_kv + hk) * T + keys[c]) * D;
            double acc = 0.0;
            for (int32_t d = 0; d < D; ++d) acc += (double)qr[d] * (double)a->k[kr + d];
            sc[c] = acc * scale;
            if (sc[c] > mx) mx = sc[c];
        }
        double den = 0.0;
        for (int32_t c = 0; c < n; ++c) { sc[c] = exp(sc[c] - mx); den += sc[c]; }
        for (int32_t d = 0; d < D; ++d) oh[d] = 0.0;
        for (int32_t c = 0; c < n; ++c) {
            const size_t vr = a->kv_layout == 0 ? (((size_t)b * T + keys[c]) * a->H_kv + hk) * D
                                                : (((size_t)b * a->H_kv + hk) * T + keys[c]) * D;
            const double pr = sc[c] / den;
            for (int32_t d = 0; d < D; ++d) oh[d] += pr * (double)a->v[vr + d];
        }
    }
    return OR_OK;
}

static int replay_check(const replay_args* a)
{
    if (!a->q || !a->k || !a->v || a->B < 0 || a->T < 0 || a->H_q < 1 || a->H_kv < 1 || a->D < 1) return OR_BAD_ARG;
    if (a->H_q % a->H_kv || (a->idx && a->S < 1) || (a->kv_layout != 0 && a->kv_layout != 1)) return OR_BAD_ARG;
    return OR_OK;
}

int mot_oracle_replay_attention(const float* q, const float* k, const float* v, const int32_t* idx,
                                double* o, int32_t B, int32_t T, int32_t H_q, int32_t H_kv, int32_t D,
                                int32_t S, int32_t kv_layout)
{
    replay_args a = {q, k, v, idx, B, T, H_q, H_kv, D, S, kv_layout};
    int rc = replay_check(&a);
    if (rc || !o) return rc ? rc : OR_BAD_ARG;
    double* sc = (double*)malloc(sizeof(double) * (T > 0 ? T : 1));
    int32_t* keys = (int32_t*)malloc(sizeof(int32_t) * (T > 0 ? T : 1));
    if (!sc || !keys) { free(sc); free(keys); return OR_NO_MEM; }
    for (int32_t b = 0; b < B && rc == OR_OK; ++b)
        for (int32_t u = 0; u < T && rc == OR_OK; ++u)
            rc = replay_row(&a, b, u, o + ((size_t)b * T + u) * H_q * D, sc, keys);
    free(sc); free(keys);
    return rc;
}

/* The same for listed positions (rb[i], ru[i]) only: out[i][H_q][D]. */
int mot_oracle_replay_attention_rows(const float* q, const float* k, const float* v, const int32_t* idx,
                                     int32_t B, int32_t T, int32_t H_q, int32_t H_kv, int32_t D,
                                     int32_t S, int32_t kv_layout, const int32_t* rb, const int32_t* ru,
                                     int32_t n_rows, double* out)
{
    replay_args a = {q, k, v, idx, B, T, H_q, H_kv, D, S, kv_layout};
    int rc = replay_check(&a);
    if (rc || !out || !rb || !ru || n_rows < 0) return rc ? rc : OR_BAD_ARG;
    for (int32_t i = 0; i < n_rows; ++i)
        if (rb[i] < 0 || rb[i] >= B || ru[i] < 0 || ru[i] >= T) return OR_BAD_ARG;
    double* sc = (double*)malloc(sizeof(double) * (T > 0 ? T : 1));
    int32_t* keys = (int32_t*)malloc(sizeof(int32_t) * (T > 0 ? T : 1));
    if (!sc || !keys) { free(sc); free(keys); return OR_NO_MEM; }
    for (int32_t i = 0; i < n_rows && rc == OR_OK; ++i)
        rc = replay_row(&a, rb[i], ru[i], out + (size_t)i * H_q * D, sc, keys);
    free(sc); free(keys);
    return rc;
}

/* Top-S sets of listed rows (rb[i], ru[i]) only: out[i][S] (see
 * mot_oracle_topS_select). */
int mot_oracle_topS_rows(const float* A, int32_t B, int32_t T, int32_t S, const int32_t* rb,
                         const int32_t* ru, int32_t n_rows, int32_t* out)
{
    if (!A || !out || !rb || !ru || B < 0 || T < 0 || S < 1 || n_rows < 0) return OR_BAD_ARG;
    char* take = (char*)malloc(T > 0 ? T : 1);
    if (!take) return OR_NO_MEM;
    for (int32_t i = 0; i < n_rows; ++i) {
        const int32_t b = rb[i], u = ru[i];
        if (b < 0 || b >= B || u < 0 || u >= T) { free(take); return OR_BAD_ARG; }
        const float* row = A + ((size_t)b * T + u) * T;
        const int32_t n = u + 1, k = n < S ? n : S;
        int32_t* o = out + (size_t)i * S;
        for (int32_t v = 0; v < n; ++v) take[v] = 0;
        for (int32_t r = 0; r < k; ++r) {
            int32_t best = -1;
            for (int32_t v = 0; v < n; ++v)
                if (!take[v] && (best < 0 || row[v] > row[best])) best = v;
            take[best] = 1;
        }
        int32_t c = 0;
        for (int32_t v = 0; v < n; ++v)
            if (take[v]) o[c++] = v;
        for (; c < S; ++c) o[c] = -1;
    }
    free(take);
    return OR_OK;
}

/* ------------------------------------------------------------------ */
/* Backbone translator body (App. C.2, "Backbone Translator")          */
/* ------------------------------------------------------------------ */

/* One channel-window slot per unit (target layer j, K or V, source layer
 * i = layer_map[j]): for every batch row b, over the context positions t,
 *   x_t  = source row (d_in)
 *   z_t  = GELU(W_in LN_in(x_t) + b_in)                     (d_h)
 *   h0   = z                                                (h_0 = z_1)
 *   a    = CrossAttn(LN_Q(h0), LN_C(z), LN_C(z)):  n_heads heads of width
 *          d_h / n_heads, Q = Wq . + bq, K = Wk . + bk, V = Wv . + bv,
 *          causal softmax(Q_t . K_s / sqrt(width)) over s <= t, Wo . + bo
 *   h1   = h0 + a
 *   h2   = h1 + W_f2 GELU(W_f1 LN_F(h1) + b_f1) + b_f2       (FFN)
 *   y_t  = GELU(W_out LN_out(h2_t) + b_out)                  (d_out)
 * and the mixture out_t = sum over the Top-K experts m of g~_m y_t^(m), with
 * the gates of the translation (softmax of Wr x_t + br, renormalised Top-K).
 * LN(v) = (v - mean) / sqrt(var + 1e-5) * gamma + beta, population variance.
 *
 * Parameters of (unit u = 2j + x, expert m), packed in this order at
 * params + (u * E + m) * P (P = mot_oracle_backbone_param_count):
 *   ln_in_g[d_in] ln_in_b[d_in] w_in[d_h][d_in] b_in[d_h]
 *   ln_q_g[d_h] ln_q_b[d_h] ln_c_g[d_h] ln_c_b[d_h]
 *   wq[d_h][d_h] bq[d_h] wk[d_h][d_h] bk[d_h] wv[d_h][d_h] bv[d_h] wo[d_h][d_h] bo[d_h]
 *   ln_f_g[d_h] ln_f_b[d_h] w_f1[d_ff][d_h] b_f1[d_ff] w_f2[d_h][d_ff] b_f2[d_h]
 *   ln_out_g[d_h] ln_out_b[d_h] w_out[d_out][d_h] b_out[d_out]
 * Everything in double; dst in the dst layout (double), layers with
 * layer_map[j] < 0 untouched. */
size_t mot_oracle_backbone_param_count(int32_t d_in, int32_t d_h, int32_t d_ff, int32_t d_out)
{
    return (size_t)2 * d_in + (size_t)d_h * d_in + d_h + 4 * (size_t)d_h +
           4 * ((size_t)d_h * d_h + d_h) + 2 * (size_t)d_h + (size_t)d_ff * d_h + d_ff +
           (size_t)d_h * d_ff + d_h + 2 * (size_t)d_h + (size_t)d_out * d_h + d_out;
}

static void bb_layernorm(const double* v, int32_t w, const float* g, const float* b, double* out)
{
    double mean = 0.0, var = 0.0;
    for (int32_t c = 0; c < w; ++c) mean += v[c];
    mean /= w;
    for (int32_t c = 0; c < w; ++c) var += (v[c] - mean) * (v[c] - mean);
    var /= w;
    const double inv = 1.0 / sqrt(var + 1e-5);
    for (int32_t c = 0; c < w; ++c) out[c] = (v[c] - mean) * inv * (double)g[c] + (double)b[c];
}

/* out[o] = W[o][:] . v + b[o] (+ act) */
static void bb_linear(const double* v, int32_t n_in, const float* W, const float* b, int32_t n_out, int gelu,
                      double* out)
{
    for (int32_t o = 0; o < n_out; ++o) {
        double acc = 0.0;
        for (int32_t c = 0; c < n_in; ++c) acc += (double)W[(size_t)o * n_in + c] * v[c];
        acc += (double)b[o];
        out[o] = gelu ? act_fn(0, acc) : acc;
    }
}

int mot_oracle_backbone_translate(const float* src_k, const float* src_v, const int32_t* layer_map,
                                  const float* params, const float* wr, const float* br,
                                  double* dst_k, double* dst_v, const mot_oracle_dims* s,
                                  int32_t d_h, int32_t n_heads, int32_t d_ff)
{
    int rc = check_dims(s, layer_map);
    if (rc) return rc;
    if (!src_k || !src_v || !params || !wr || !dst_k || !dst_v || s->streams != 2) return OR_BAD_ARG;
    if (d_h < 1 || n_heads < 1 || d_h % n_heads || d_ff < 1) return OR_BAD_ARG;
    const int32_t d_in = s->H_src * s->D_src, d_out = s->H_tgt * s->D_tgt, E = s->E, T = s->T;
    const int32_t hw = d_h / n_heads;
    const size_t P = mot_oracle_backbone_param_count(d_in, d_h, d_ff, d_out);
    const size_t TT = T > 0 ? (size_t)T : 1;
    double* x = (double*)malloc(sizeof(double) * TT * d_in);
    double* z = (double*)malloc(sizeof(double) * TT * d_h);
    double* Q = (double*)malloc(sizeof(double) * TT * d_h);
    double* K = (double*)malloc(sizeof(double) * TT * d_h);
    double* V = (double*)malloc(sizeof(double) * TT * d_h);
    double* h2 = (double*)malloc(sizeof(double) * TT * d_h);
    double* out = (double*)malloc(sizeof(double) * TT * d_out);
    double* gt = (double*)malloc(sizeof(double) * TT * E);
    double* t1 = (double*)malloc(sizeof(double) * (d_in > d_h ? d_in : d_h));
    double* t2 = (double*)malloc(sizeof(double) * d_h);
    double* att = (double*)malloc(sizeof(double) * d_h);
    double* f = (double*)malloc(sizeof(double) * d_ff);
    double* y = (double*)malloc(sizeof(double) * d_out);
    double* sc = (double*)malloc(sizeof(double) * TT);
    double* lg = (double*)malloc(sizeof(double) * E);
    int* sel = (int*)malloc(sizeof(int) * E);
    if (!x || !z || !Q || !K || !V || !h2 || !out || !gt || !t1 || !t2 || !att || !f || !y || !sc || !lg || !sel) {
        rc = OR_NO_MEM;
        goto done;
    }
    for (int32_t j = 0; j < s->L_tgt; ++j) {
        const int32_t i = layer_map[j];
        if (i < 0) continue;
        for (int32_t xk = 0; xk < 2; ++xk) {
            const size_t unit = (size_t)j * 2 + xk;
            const float* src = xk == 0 ? src_k : src_v;
            double* dst = xk == 0 ? dst_k : dst_v;
            for (int32_t b = 0; b < s->B; ++b) {
                /* source rows and gates */
                for (int32_t t = 0; t < T; ++t) {
                    gather_row(s, src, i, b, t, x + (size_t)t * d_in);
                    const double* xt = x + (size_t)t * d_in;
                    double mx = -INFINITY;
                    for (int32_t m = 0; m < E; ++m) {
                        double acc = 0.0;
                        for (int32_t c = 0; c < d_in; ++c) acc += (double)wr[(unit * E + m) * d_in + c] * xt[c];
                        if (br) acc += (double)br[unit * E + m];
                        lg[m] = acc;
                        if (acc > mx) mx = acc;
                    }
                    double den = 0.0;
                    for (int32_t m = 0; m < E; ++m) { lg[m] = exp(lg[m] - mx); den += lg[m]; }
                    for (int32_t m = 0; m < E; ++m) { lg[m] /= den; sel[m] = 0; }
                    for (int32_t k = 0; k < s->top_k; ++k) {
                        int32_t best = -1;
                        for (int32_t m = 0; m < E; ++m)
                            if (!sel[m] && (best < 0 || lg[m] > lg[best])) best = m;
                        sel[best] = 1;
                    }
                    double gs = 0.0;
                    for (int32_t m = 0; m < E; ++m) if (sel[m]) gs += lg[m];
                    for (int32_t m = 0; m < E; ++m) gt[(size_t)t * E + m] = sel[m] ? lg[m] / gs : 0.0;
                }
                for (size_t c = 0; c < (size_t)T * d_out; ++c) out[c] = 0.0;
                for (int32_t m = 0; m < E; ++m) {
                    int used = 0;
                    for (int32_t t = 0; t < T; ++t) used |= gt[(size_t)t * E + m] != 0.0;
                    if (!used) continue;
                    const float* pp = params + (unit * E + m) * P;
                    const float *ln_in_g = pp, *ln_in_b = ln_in_g + d_in, *w_in = ln_in_b + d_in,
                                *b_in = w_in + (size_t)d_h * d_in, *ln_q_g = b_in + d_h, *ln_q_b = ln_q_g + d_h,
                                *ln_c_g = ln_q_b + d_h, *ln_c_b = ln_c_g + d_h, *wq = ln_c_b + d_h,
                                *bq = wq + (size_t)d_h * d_h, *wk = bq + d_h, *bk = wk + (size_t)d_h * d_h,
                                *wv = bk + d_h, *bv = wv + (size_t)d_h * d_h, *wo = bv + d_h,
                                *bo = wo + (size_t)d_h * d_h, *ln_f_g = bo + d_h, *ln_f_b = ln_f_g + d_h,
                                *w_f1 = ln_f_b + d_h, *b_f1 = w_f1 + (size_t)d_ff * d_h, *w_f2 = b_f1 + d_ff,
                                *b_f2 = w_f2 + (size_t)d_h * d_ff, *ln_out_g = b_f2 + d_h,
                                *ln_out_b = ln_out_g + d_h, *w_out = ln_out_b + d_h,
                                *b_out = w_out + (size_t)d_out * d_h;
                    /* z, then Q (from LN_Q(z)), K and V (from LN_C(z)) */
                    for (int32_t t = 0; t < T; ++t) {
                        bb_layernorm(x + (size_t)t * d_in, d_in, ln_in_g, ln_in_b, t1);
                        bb_linear(t1, d_in, w_in, b_in, d_h, 1, z + (size_t)t * d_h);
                        bb_layernorm(z + (size_t)t * d_h, d_h, ln_q_g, ln_q_b, t1);
                        bb_linear(t1, d_h, wq, bq, d_h, 0, Q + (size_t)t * d_h);
                        bb_layernorm(z + (size_t)t * d_h, d_h, ln_c_g, ln_c_b, t1);
                        bb_linear(t1, d_h, wk, bk, d_h, 0, K + (size_t)t * d_h);
                        bb_linear(t1, d_h, wv, bv, d_h, 0, V + (size_t)t * d_h);
                    }
                    for (int32_t t = 0; t < T; ++t) {
                        /* causal multi-head attention of position t */
                        for (int32_t hh = 0; hh < n_heads; ++hh) {
                            const double* qt = Q + (size_t)t * d_h + hh * hw;
                            double mx = -INFINITY;
                            for (int32_t u = 0; u <= t; ++u) {
                                const double* ku = K + (size_t)u * d_h + hh * hw;
                                double acc = 0.0;
                                for (int32_t d = 0; d < hw; ++d) acc += qt[d] * ku[d];
                                sc[u] = acc / sqrt((double)hw);
                                if (sc[u] > mx) mx = sc[u];
                            }
                            double den = 0.0;
                            for (int32_t u = 0; u <= t; ++u) { sc[u] = exp(sc[u] - mx); den += sc[u]; }
                            for (int32_t d = 0; d < hw; ++d) att[hh * hw + d] = 0.0;
                            for (int32_t u = 0; u <= t; ++u) {
                                const double* vu = V + (size_t)u * d_h + hh * hw;
                                for (int32_t d = 0; d < hw; ++d) att[hh * hw + d] += sc[u] / den * vu[d];
                            }
                        }
                        /* h1 = z + Wo a + bo;  h2 = h1 + FFN(LN_F(h1)) */
                        bb_linear(att, d_h, wo, bo, d_h, 0, t2);
                        for (int32_t c = 0; c < d_h; ++c) t2[c] += z[(size_t)t * d_h + c];
                        bb_layernorm(t2, d_h, ln_f_g, ln_f_b, t1);
                        bb_linear(t1, d_h, w_f1, b_f1, d_ff, 1, f);
                        bb_linear(f, d_ff, w_f2, b_f2, d_h, 0, h2 + (size_t)t * d_h);
                        for (int32_t c = 0; c < d_h; ++c) h2[(size_t)t * d_h + c] += t2[c];
                        bb_layernorm(h2 + (size_t)t * d_h, d_h, ln_out_g, ln_out_b, t1);
                        bb_linear(t1, d_h, w_out, b_out, d_out, 1, y);
                        const double g = gt[(size_t)t * E + m];
                        for (int32_t o = 0; o < d_out; ++o) out[(size_t)t * d_out + o] += g * y[o];
                    }
                }
                for (int32_t t = 0; t < T; ++t)
                    for (int32_t o = 0; o < d_out; ++o)
                        dst[cache_index(s, s->dst_layout, s->H_tgt, s->D_tgt, j, b, t, o / s->D_tgt, o % s->D_tgt)] =
                            out[(size_t)t * d_out + o];
            }
        }
    }
done:
    free(x); free(z); free(Q); free(K); free(V); free(h2); free(out); free(gt); free(t1); free(t2);
    free(att); free(f); free(y); free(sc); free(lg); free(sel);
    return rc;
}

/* ------------------------------------------------------------------ */
/* translator usage (paper Sec. 4, "MoT Architecture Ablation",        */
/* Table "mot_analysis")                                               */
/* ------------------------------------------------------------------ */

/* Selection counts: counts[(j * streams + x) * E + m] += the number of
 * context tokens whose Top-K set (Definition "Mixture-of-Translators": the
 * top_k largest softmax scores, ties to the lower index) holds translator m,
 * for every unit (j, x) with layer_map[j] >= 0.  Counts accumulate: the
 * caller zeroes them to start. */
int mot_oracle_usage(const float* src_k, const float* src_v, const int32_t* layer_map,
                     const float* wr, const float* br, const mot_oracle_dims* s, int64_t* counts)
{
    int rc = check_dims(s, layer_map);
    if (rc) return rc;
    if (!src_k || !wr || !counts || (s->streams == 2 && !src_v)) return OR_BAD_ARG;
    const int32_t d_in = s->H_src * s->D_src, E = s->E;
    double* z = (double*)malloc(sizeof(double) * d_in);
    double* g = (double*)malloc(sizeof(double) * E);
    int* sel = (int*)malloc(sizeof(int) * E);
    if (!z || !g || !sel) { free(z); free(g); free(sel); return OR_NO_MEM; }
    for (int32_t j = 0; j < s->L_tgt; ++j) {
        const int32_t i = layer_map[j];
        if (i < 0) continue;
        for (int32_t x = 0; x < s->streams; ++x) {
            const size_t unit = (size_t)j * s->streams + x;
            for (int32_t b = 0; b < s->B; ++b)
                for (int32_t t = 0; t < s->T; ++t) {
                    gather_row(s, x == 0 ? src_k : src_v, i, b, t, z);
                    /* gate logits, softmax */
                    double mx = -INFINITY;
                    for (int32_t m = 0; m < E; ++m) {
                        double acc = 0.0;
                        for (int32_t c = 0; c < d_in; ++c) acc += (double)wr[(unit * E + m) * d_in + c] * z[c];
                        if (br) acc += (double)br[unit * E + m];
                        g[m] = acc;
                        if (acc > mx) mx = acc;
                    }
                    double den = 0.0;
                    for (int32_t m = 0; m < E; ++m) { g[m] = exp(g[m] - mx); den += g[m]; }
                    for (int32_t m = 0; m < E; ++m) { g[m] /= den; sel[m] = 0; }
                    /* Top-K: the largest remaining score, top_k times; a tie
                     * keeps the lower index (ascending scan, strict '>') */
                    for (int32_t k = 0; k < s->top_k; ++k) {
                        int32_t best = -1;
                        for (int32_t m = 0; m < E; ++m)
                            if (!sel[m] && (best < 0 || g[m] > g[best])) best = m;
                        sel[best] = 1;
                    }
                    for (int32_t m = 0; m < E; ++m) counts[unit * E + m] += sel[m];
                }
        }
    }
    free(z); free(g); free(sel);
    return OR_OK;
}

/* Usage imbalance and entropy of one unit's counts I[0..E):
 *   CV^2    = Var_m(I_m) / Mean_m(I_m)^2   (population variance: the mean of
 *             the squared deviations over the E translators)
 *   entropy = -sum_m p_m ln p_m,  p_m = I_m / sum_r I_r  (0 ln 0 = 0)
 * Both are NaN when every count is zero. */
int mot_oracle_usage_stats(const int64_t* counts, int32_t E, double* cv2, double* entropy)
{
    if (!counts || E < 1 || !cv2 || !entropy) return OR_BAD_ARG;
    double total = 0.0;
    for (int32_t m = 0; m < E; ++m) total += (double)counts[m];
    const double mean = total / E;
    double var = 0.0;
    for (int32_t m = 0; m < E; ++m) var += ((double)counts[m] - mean) * ((double)counts[m] - mean);
    var /= E;
    *cv2 = var / (mean * mean);
    double h = 0.0;
    for (int32_t m = 0; m < E; ++m) {
        if (counts[m] == 0) continue;
        const double p = (double)counts[m] / total;
        h -= p * log(p);
    }
    *entropy = total > 0.0 ? h : NAN;
    return OR_OK;
}

/* ------------------------------------------------------------------ */
/* backbone translator over a multi-slot channel window (App. C.2)     */
/* ------------------------------------------------------------------ */

/* Parameters per (window, X, expert), in order (N = n_slots):
 *   ln_in_g[d_in] ln_in_b[d_in] w_in[d_h][d_in] b_in[d_h]        (shared by the slots)
 *   for each slot r = 1..N (the block CAB_r):
 *     ln_q_g[d_h] ln_q_b[d_h] ln_c_g[d_h] ln_c_b[d_h] wq[d_h][d_h] bq[d_h] wk[d_h][d_h] bk[d_h]
 *     wv[d_h][d_h] bv[d_h] wo[d_h][d_h] bo[d_h] ln_f_g[d_h] ln_f_b[d_h] w_f1[d_ff][d_h] b_f1[d_ff]
 *     w_f2[d_h][d_ff] b_f2[d_h]
 *   ln_out_g[N d_h] ln_out_b[N d_h] w_out[N d_out][N d_h] b_out[N d_out]
 * With N = 1 this is the packing of mot_oracle_backbone_translate. */
size_t mot_oracle_backbone_window_param_count(int32_t d_in, int32_t d_h, int32_t d_ff, int32_t d_out, int32_t N)
{
    const size_t cab = 4 * (size_t)d_h + 4 * ((size_t)d_h * d_h + d_h) + 2 * (size_t)d_h + (size_t)d_ff * d_h +
                       d_ff + (size_t)d_h * d_ff + d_h;
    return 2 * (size_t)d_in + (size_t)d_h * d_in + d_h + (size_t)N * cab + 2 * (size_t)N * d_h +
           (size_t)N * d_out * N * d_h + (size_t)N * d_out;
}

/* Windows w = 0 .. L_tgt/N - 1 cover target layers wN .. wN+N-1; slot r of
 * window w reads source layer layer_map[wN + r].  A window whose entries are
 * all -1 is skipped (its target layers untouched); a window with some -1
 * entries is an error.  For each window, X in {K, V} and batch row b, over
 * the context positions t:
 *   x_r[t]   = source row of slot r (head-major)
 *   gates    = Top-K renormalised softmax of Wr Concat(x_1..x_N)[t] + br
 *              (router weights [L_tgt/N][2][E][N d_in], bias [L_tgt/N][2][E])
 *   expert m:
 *     z_r[t] = GELU(W_in LN_in(x_r[t]) + b_in)
 *     h_0 = z_1;  for r = 1..N:
 *       a     = CausalMHA(LN_Q^r(h_{r-1}), LN_C^r(z_r), LN_C^r(z_r))  (Wq, Wk, Wv, Wo of slot r)
 *       h~    = h_{r-1} + Wo^r a + bo^r
 *       h_r   = h~ + W_f2^r GELU(W_f1^r LN_F^r(h~) + b_f1^r) + b_f2^r
 *     y[t]   = GELU(W_out LN_out(Concat(h_1..h_N)[t]) + b_out)    (N d_out)
 *   out[t] = sum_m g~_m y[t];  target layer wN + r receives out[t][r d_out .. (r+1) d_out).
 * Sums in index order, double throughout. */
int mot_oracle_backbone_window(const float* src_k, const float* src_v, const int32_t* layer_map,
                               const float* params, const float* wr, const float* br,
                               double* dst_k, double* dst_v, const mot_oracle_dims* s,
                               int32_t d_h, int32_t n_heads, int32_t d_ff, int32_t N)
{
    int rc = check_dims(s, layer_map);
    if (rc) return rc;
    if (!src_k || !src_v || !params || !wr || !dst_k || !dst_v || s->streams != 2) return OR_BAD_ARG;
    if (d_h < 1 || n_heads < 1 || d_h % n_heads || d_ff < 1 || N < 1 || s->L_tgt % N) return OR_BAD_ARG;
    const int32_t d_in = s->H_src * s->D_src, d_out = s->H_tgt * s->D_tgt, E = s->E, T = s->T;
    const int32_t hw = d_h / n_heads, W = s->L_tgt / N, Nd_in = N * d_in, Nd_h = N * d_h, Nd_out = N * d_out;
    for (int32_t w = 0; w < W; ++w) {
        int n_neg = 0;
        for (int32_t r = 0; r < N; ++r) n_neg += layer_map[w * N + r] < 0;
        if (n_neg != 0 && n_neg != N) return OR_BAD_ARG;
    }
    const size_t P = mot_oracle_backbone_window_param_count(d_in, d_h, d_ff, d_out, N);
    const size_t cab = 4 * (size_t)d_h + 4 * ((size_t)d_h * d_h + d_h) + 2 * (size_t)d_h + (size_t)d_ff * d_h +
                       d_ff + (size_t)d_h * d_ff + d_h;
    const size_t TT = T > 0 ? (size_t)T : 1;
    double* x = (double*)malloc(sizeof(double) * TT * Nd_in);     /* [t][r][d_in]: the concatenated rows */
    double* z = (double*)malloc(sizeof(double) * TT * Nd_h);      /* [t][r][d_h] */
    double* F = (double*)malloc(sizeof(double) * TT * Nd_h);      /* [t][r][d_h]: h_1..h_N */
    double* Q = (double*)malloc(sizeof(double) * TT * d_h);
    double* K = (double*)malloc(sizeof(double) * TT * d_h);
    double* V = (double*)malloc(sizeof(double) * TT * d_h);
    double* out = (double*)malloc(sizeof(double) * TT * Nd_out);
    double* gt = (double*)malloc(sizeof(double) * TT * E);
    double* t1 = (double*)malloc(sizeof(double) * (Nd_h > d_in ? Nd_h : d_in));
    double* t2 = (double*)malloc(sizeof(double) * d_h);
    double* att = (double*)malloc(sizeof(double) * d_h);
    double* f = (double*)malloc(sizeof(double) * d_ff);
    double* y = (double*)malloc(sizeof(double) * Nd_out);
    double* sc = (double*)malloc(sizeof(double) * TT);
    double* lg = (double*)malloc(sizeof(double) * E);
    int* sel = (int*)malloc(sizeof(int) * E);
    if (!x || !z || !F || !Q || !K || !V || !out || !gt || !t1 || !t2 || !att || !f || !y || !sc || !lg || !sel) {
        rc = OR_NO_MEM;
        goto done;
    }
    for (int32_t w = 0; w < W; ++w) {
        if (layer_map[w * N] < 0) continue;
        for (int32_t xk = 0; xk < 2; ++xk) {
            const size_t unit = (size_t)w * 2 + xk;
            const float* src = xk == 0 ? src_k : src_v;
            double* dst = xk == 0 ? dst_k : dst_v;
            for (int32_t b = 0; b < s->B; ++b) {
                for (int32_t t = 0; t < T; ++t) {
                    for (int32_t r = 0; r < N; ++r)
                        gather_row(s, src, layer_map[w * N + r], b, t, x + (size_t)t * Nd_in + (size_t)r * d_in);
                    const double* xt = x + (size_t)t * Nd_in;
                    double mx = -INFINITY;
                    for (int32_t m = 0; m < E; ++m) {
                        double acc = 0.0;
                        for (int32_t c = 0; c < Nd_in; ++c) acc += (double)wr[(unit * E + m) * Nd_in + c] * xt[c];
                        if (br) acc += (double)br[unit * E + m];
                        lg[m] = acc;
                        if (acc > mx) mx = acc;
                    }
                    double den = 0.0;
                    for (int32_t m = 0; m < E; ++m) { lg[m] = exp(lg[m] - mx); den += lg[m]; }
                    for (int32_t m = 0; m < E; ++m) { lg[m] /= den; sel[m] = 0; }
                    for (int32_t k = 0; k < s->top_k; ++k) {
                        int32_t best = -1;
                        for (int32_t m = 0; m < E; ++m)
                            if (!sel[m] && (best < 0 || lg[m] > lg[best])) best = m;
                        sel[best] = 1;
                    }
                    double gs = 0.0;
                    for (int32_t m = 0; m < E; ++m) if (sel[m]) gs += lg[m];
                    for (int32_t m = 0; m < E; ++m) gt[(size_t)t * E + m] = sel[m] ? lg[m] / gs : 0.0;
                }
                for (size_t c = 0; c < (size_t)T * Nd_out; ++c) out[c] = 0.0;
                for (int32_t m = 0; m < E; ++m) {
                    int used = 0;
                    for (int32_t t = 0; t < T; ++t) used |= gt[(size_t)t * E + m] != 0.0;
                    if (!used) continue;
                    const float* pp = params + (unit * E + m) * P;
                    const float *ln_in_g = pp, *ln_in_b = ln_in_g + d_in, *w_in = ln_in_b + d_in,
                                *b_in = w_in + (size_t)d_h * d_in;
                    const float* cab0 = b_in + d_h;
                    const float *ln_out_g = cab0 + (size_t)N * cab, *ln_out_b = ln_out_g + Nd_h,
                                *w_out = ln_out_b + Nd_h, *b_out = w_out + (size_t)Nd_out * Nd_h;
                    /* z_r = GELU(W_in LN_in(x_r) + b_in) for every slot */
                    for (int32_t t = 0; t < T; ++t)
                        for (int32_t r = 0; r < N; ++r) {
                            bb_layernorm(x + (size_t)t * Nd_in + (size_t)r * d_in, d_in, ln_in_g, ln_in_b, t1);
                            bb_linear(t1, d_in, w_in, b_in, d_h, 1, z + (size_t)t * Nd_h + (size_t)r * d_h);
                        }
                    /* the recurrent scan over the slots */
                    for (int32_t r = 0; r < N; ++r) {
                        const float* cp = cab0 + (size_t)r * cab;
                        const float *ln_q_g = cp, *ln_q_b = ln_q_g + d_h, *ln_c_g = ln_q_b + d_h,
                                    *ln_c_b = ln_c_g + d_h, *wq = ln_c_b + d_h, *bq = wq + (size_t)d_h * d_h,
                                    *wk = bq + d_h, *bk = wk + (size_t)d_h * d_h, *wv = bk + d_h,
                                    *bv = wv + (size_t)d_h * d_h, *wo = bv + d_h, *bo = wo + (size_t)d_h * d_h,
                                    *ln_f_g = bo + d_h, *ln_f_b = ln_f_g + d_h, *w_f1 = ln_f_b + d_h,
                                    *b_f1 = w_f1 + (size_t)d_ff * d_h, *w_f2 = b_f1 + d_ff,
                                    *b_f2 = w_f2 + (size_t)d_h * d_ff;
                        /* h_{r-1}: z_1 before the first block, then the previous block's output */
                        for (int32_t t = 0; t < T; ++t) {
                            const double* hp = r == 0 ? z + (size_t)t * Nd_h : F + (size_t)t * Nd_h + (size_t)(r - 1) * d_h;
                            const double* zr = z + (size_t)t * Nd_h + (size_t)r * d_h;
                            bb_layernorm(hp, d_h, ln_q_g, ln_q_b, t1);
                            bb_linear(t1, d_h, wq, bq, d_h, 0, Q + (size_t)t * d_h);
                            bb_layernorm(zr, d_h, ln_c_g, ln_c_b, t1);
                            bb_linear(t1, d_h, wk, bk, d_h, 0, K + (size_t)t * d_h);
                            bb_linear(t1, d_h, wv, bv, d_h, 0, V + (size_t)t * d_h);
                        }
                        for (int32_t t = 0; t < T; ++t) {
                            for (int32_t hh = 0; hh < n_heads; ++hh) {
                                const double* qt = Q + (size_t)t * d_h + hh * hw;
                                double mx = -INFINITY;
                                for (int32_t u = 0; u <= t; ++u) {
                                    const double* ku = K + (size_t)u * d_h + hh * hw;
                                    double acc = 0.0;
                                    for (int32_t d = 0; d < hw; ++d) acc += qt[d] * ku[d];
                                    sc[u] = acc / sqrt((double)hw);
                                    if (sc[u] > mx) mx = sc[u];
                                }
                                double den = 0.0;
                                for (int32_t u = 0; u <= t; ++u) { sc[u] = exp(sc[u] - mx); den += sc[u]; }
                                for (int32_t d = 0; d < hw; ++d) att[hh * hw + d] = 0.0;
                                for (int32_t u = 0; u <= t; ++u) {
                                    const double* vu = V + (size_t)u * d_h + hh * hw;
                                    for (int32_t d = 0; d < hw; ++d) att[hh * hw + d] += sc[u] / den * vu[d];
                                }
                            }
                            const double* hp = r == 0 ? z + (size_t)t * Nd_h : F + (size_t)t * Nd_h + (size_t)(r - 1) * d_h;
                            double* hr = F + (size_t)t * Nd_h + (size_t)r * d_h;
                            bb_linear(att, d_h, wo, bo, d_h, 0, t2);
                            for (int32_t c = 0; c < d_h; ++c) t2[c] += hp[c];
                            bb_layernorm(t2, d_h, ln_f_g, ln_f_b, t1);
                            bb_linear(t1, d_h, w_f1, b_f1, d_ff, 1, f);
                            bb_linear(f, d_ff, w_f2, b_f2, d_h, 0, hr);
                            for (int32_t c = 0; c < d_h; ++c) hr[c] += t2[c];
                        }
                    }
                    /* y = GELU(W_out LN_out(Concat(h_1..h_N)) + b_out), gated sum */
                    for (int32_t t = 0; t < T; ++t) {
                        bb_layernorm(F + (size_t)t * Nd_h, Nd_h, ln_out_g, ln_out_b, t1);
                        bb_linear(t1, Nd_h, w_out, b_out, Nd_out, 1, y);
                        const double g = gt[(size_t)t * E + m];
                        for (int32_t o = 0; o < Nd_out; ++o) out[(size_t)t * Nd_out + o] += g * y[o];
                    }
                }
                for (int32_t r = 0; r < N; ++r)
                    for (int32_t t = 0; t < T; ++t)
                        for (int32_t o = 0; o < d_out; ++o)
                            dst[cache_index(s, s->dst_layout, s->H_tgt, s->D_tgt, w * N + r, b, t, o / s->D_tgt,
                                            o % s->D_tgt)] = out[(size_t)t * Nd_out + (size_t)r * d_out + o];
            }
        }
    }
done:
    free(x); free(z); free(F); free(Q); free(K); free(V); free(out); free(gt); free(t1); free(t2);
    free(att); free(f); free(y); free(sc); free(lg); free(sel);
    return rc;
}
