// C-ABI entry points of libmot: argument validation, planning, workspace and
// kernel dispatch.  Every check runs before the first enqueue; on error
// nothing is launched and the outputs are untouched.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>

#include "../../include/mot.h"
#include "mot_internal.h"

using namespace mot;

namespace {

thread_local char g_err[512] = "";

mot_status fail(mot_status s, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return s;
}

constexpr size_t kAlign = 256;
constexpr size_t kDefaultHiddenCap = size_t(1) << 30;   // hidden buffer per group, bytes

size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

struct Plan {
    bool bf16 = false;
    bool fused = false;
    bool routed = false;       // Top-K sparse path (fused kernel over translator tiles)
    bool routed2 = false;      // Top-K sparse path on the two-GEMM kernels (shapes the fused kernel lacks)
    int n_units = 0;
    int32_t n_tok = 0, n_tok_pad = 0;
    size_t fixed_bytes = 0;    // workspace for all units of the call
    size_t unit_bytes = 0;     // workspace per unit of a launch group
    int32_t max_tiles = 0, tile_rows = 0;
    uint32_t codes[kMaxUnits];
};

Problem base_problem(const mot_shapes* s);

mot_status check_shapes(const mot_shapes* s) {
    if (!s) return fail(MOT_ERR_NULL_ARG, "shapes is NULL");
    if (s->L_src < 1 || s->L_src > MOT_MAX_LAYERS || s->L_tgt < 1 || s->L_tgt > MOT_MAX_LAYERS)
        return fail(MOT_ERR_BAD_SHAPE, "L_src=%d L_tgt=%d must be in [1, %d]", s->L_src, s->L_tgt,
                    MOT_MAX_LAYERS);
    if (s->B < 0 || s->T < 0)
        return fail(MOT_ERR_BAD_SHAPE, "B=%d T=%d must be >= 0", s->B, s->T);
    if ((int64_t)s->B * s->T > (int64_t)1 << 26)
        return fail(MOT_ERR_BAD_SHAPE, "B*T=%lld exceeds 2^26 tokens", (long long)s->B * s->T);
    if (s->H_src < 1 || s->D_src < 1 || s->H_tgt < 1 || s->D_tgt < 1 || s->hidden < 1)
        return fail(MOT_ERR_BAD_SHAPE, "head counts, head dims and hidden must be >= 1");
    if ((int64_t)s->H_src * s->D_src > 65536 || (int64_t)s->H_tgt * s->D_tgt > 65536 ||
        s->hidden > 65536)
        return fail(MOT_ERR_BAD_SHAPE, "row or hidden width above 65536");
    if (s->E < 1 || s->E > MOT_MAX_EXPERTS)
        return fail(MOT_ERR_BAD_SHAPE, "E=%d must be in [1, %d]", s->E, MOT_MAX_EXPERTS);
    if (s->top_k < 1 || s->top_k > s->E)
        return fail(MOT_ERR_BAD_SHAPE, "top_k=%d must be in [1, E=%d]", s->top_k, s->E);
    if (s->dtype != MOT_F32 && s->dtype != MOT_BF16)
        return fail(MOT_ERR_BAD_SHAPE, "dtype=%d is not MOT_F32 or MOT_BF16", s->dtype);
    if ((s->src_layout != MOT_LAYOUT_BTHD && s->src_layout != MOT_LAYOUT_BHTD) ||
        (s->dst_layout != MOT_LAYOUT_BTHD && s->dst_layout != MOT_LAYOUT_BHTD))
        return fail(MOT_ERR_BAD_SHAPE, "layouts must be MOT_LAYOUT_BTHD or MOT_LAYOUT_BHTD");
    if (s->act != MOT_ACT_GELU && s->act != MOT_ACT_IDENTITY)
        return fail(MOT_ERR_BAD_SHAPE, "act=%d is not MOT_ACT_GELU or MOT_ACT_IDENTITY", s->act);
    if (s->streams < 0 || s->streams > 2)
        return fail(MOT_ERR_BAD_SHAPE, "streams=%d must be 1 (one activation stream) or 2 (keys and values; 0 = 2)",
                    s->streams);
    if (s->algo != MOT_ALGO_AUTO && s->algo != MOT_ALGO_UNFUSED && s->algo != MOT_ALGO_FUSED &&
        s->algo != MOT_ALGO_ROUTED)
        return fail(MOT_ERR_BAD_SHAPE, "algo=%d is not a mot_algo value", s->algo);
    const int d_in = s->H_src * s->D_src, d_out = s->H_tgt * s->D_tgt;
    if (s->algo == MOT_ALGO_FUSED) {
        Problem p = base_problem(s);
        if (s->dtype != MOT_BF16 || !fused_supported(p))
            return fail(MOT_ERR_UNSUPPORTED,
                        "the fused kernel needs bf16, d_in and d_out in {128, 256, 512}, hidden %% 32 == 0");
    }
    if (s->algo == MOT_ALGO_ROUTED) {
        Problem p = base_problem(s);
        if (s->dtype != MOT_BF16 || (!fused_supported(p) && !bf16_routed_gemm_fits(p)))
            return fail(MOT_ERR_UNSUPPORTED,
                        "the routed path needs bf16 and either the fused kernel's shapes or operand regions "
                        "under 2 GiB for the routed two-GEMM kernels");
    }
    if (s->dtype == MOT_BF16) {
        if (s->D_src % 8 || s->D_tgt % 8 || d_in % 64 || s->hidden % 64 || d_out % 32)
            return fail(MOT_ERR_UNSUPPORTED,
                        "bf16 needs D_src, D_tgt %% 8 == 0, d_in %% 64 == 0, hidden %% 64 == 0, d_out %% 32 == 0 "
                        "(got D_src=%d D_tgt=%d d_in=%d hidden=%d d_out=%d)",
                        s->D_src, s->D_tgt, d_in, s->hidden, d_out);
    } else {
        if (s->D_src % 4 || s->D_tgt % 4 || s->hidden % 4)
            return fail(MOT_ERR_UNSUPPORTED,
                        "fp32 needs D_src, D_tgt, hidden %% 4 == 0 (got D_src=%d D_tgt=%d hidden=%d)",
                        s->D_src, s->D_tgt, s->hidden);
    }
    return MOT_OK;
}

Problem base_problem(const mot_shapes* s) {
    Problem p;
    memset(&p, 0, sizeof p);
    p.B = s->B; p.T = s->T; p.H_src = s->H_src; p.D_src = s->D_src;
    p.H_tgt = s->H_tgt; p.D_tgt = s->D_tgt; p.E = s->E; p.top_k = s->top_k; p.hidden = s->hidden;
    p.d_in = s->H_src * s->D_src; p.d_out = s->H_tgt * s->D_tgt;
    p.n_tok = s->B * s->T;
    p.n_tok_pad = (int32_t)round_up((size_t)p.n_tok, 128);
    p.src_layout = s->src_layout; p.dst_layout = s->dst_layout; p.act = s->act;
    p.streams = s->streams == 1 ? 1 : 2;
    p.usage = s->usage;
    return p;
}

// Plan for the given layer map (or the worst case, all 2*L_tgt units).
void make_plan(const mot_shapes* s, const int32_t* layer_map, Plan* pl) {
    Problem p = base_problem(s);
    pl->bf16 = s->dtype == MOT_BF16;
    pl->fused = pl->bf16 && s->algo != MOT_ALGO_UNFUSED && fused_supported(p);
    const bool want_routed = s->algo == MOT_ALGO_ROUTED || (s->algo == MOT_ALGO_AUTO && s->top_k < s->E);
    pl->routed = pl->fused && want_routed;
    pl->routed2 = pl->bf16 && !pl->fused && want_routed && bf16_routed_gemm_fits(p);
    pl->n_tok = p.n_tok;
    pl->n_tok_pad = p.n_tok_pad;
    int n = 0;
    for (int j = 0; j < s->L_tgt; ++j) {
        const int i = layer_map ? layer_map[j] : 0;
        if (i < 0) continue;
        for (int x = 0; x < p.streams; ++x) {
            pl->codes[n] = unit_code(j, x, i, n);
            ++n;
        }
    }
    pl->n_units = n;
    pl->fixed_bytes = 0;
    pl->unit_bytes = 0;
    pl->max_tiles = pl->tile_rows = 0;
    if (pl->routed || pl->routed2) {
        const size_t nk = (size_t)p.n_tok * p.top_k;
        pl->tile_rows = pl->routed ? fused_tile_rows(p) : 256;
        pl->max_tiles = (int32_t)round_up((nk + pl->tile_rows - 1) / pl->tile_rows + p.E, 8);
        const size_t per = round_up(nk * 4, kAlign);   // one int32 / fp32 per assignment
        pl->fixed_bytes = (size_t)n * (5 * per + round_up((size_t)pl->max_tiles * 16, kAlign)) +
                          round_up((size_t)n * 4, kAlign);
        // per unit of a launch group: (two-GEMM) the hidden rows in assignment
        // order, then (top_k > 1) the fp32 per-assignment output rows
        if (pl->routed2) pl->unit_bytes = round_up(bf16_routed_hidden_bytes(p), kAlign);
        if (p.top_k > 1) pl->unit_bytes += round_up(nk * p.d_out * sizeof(float), kAlign);
    } else if (!pl->fused) {
        pl->fixed_bytes = round_up((size_t)n * p.n_tok_pad * p.E * sizeof(float), kAlign);
        pl->unit_bytes = round_up((size_t)p.n_tok_pad * p.E * p.hidden * (pl->bf16 ? 2 : 4), kAlign);
    }
}

int default_group(const Plan& pl) {
    if (pl.unit_bytes == 0) return pl.n_units;
    size_t g = kDefaultHiddenCap / pl.unit_bytes;
    if (g < 1) g = 1;
    if (g > (size_t)pl.n_units) g = pl.n_units;
    return (int)g;
}

size_t plan_bytes(const Plan& pl, int group) {
    if (pl.n_units == 0) return 0;
    return pl.fixed_bytes + (size_t)group * pl.unit_bytes;
}

// Carve the routed path's buffers out of the workspace (layout of make_plan).
void carve_routing(const Plan& pl, const Problem& p, void* ws, Routing* rt) {
    const size_t nk = (size_t)p.n_tok * p.top_k, per = round_up(nk * 4, kAlign);
    const size_t U = (size_t)pl.n_units;
    char* c = reinterpret_cast<char*>(ws);
    rt->sel = reinterpret_cast<int32_t*>(c); c += U * per;
    rt->gk = reinterpret_cast<float*>(c); c += U * per;
    rt->list = reinterpret_cast<int32_t*>(c); c += U * per;
    rt->agate = reinterpret_cast<float*>(c); c += U * per;
    rt->slot = p.top_k > 1 ? reinterpret_cast<int32_t*>(c) : nullptr; c += U * per;
    rt->tiles = reinterpret_cast<int4*>(c); c += U * round_up((size_t)pl.max_tiles * 16, kAlign);
    rt->ntiles = reinterpret_cast<int32_t*>(c); c += round_up(U * 4, kAlign);
    rt->part = p.top_k > 1 ? reinterpret_cast<float*>(c) : nullptr;
    rt->max_tiles = pl.max_tiles;
    rt->tile_rows = pl.tile_rows;
}

// Library-owned workspace, one per device, grown on demand.
struct OwnedBuf {
    void* ptr = nullptr;
    size_t bytes = 0;
};
std::mutex g_buf_mu;
OwnedBuf g_bufs[64];

mot_status owned_workspace(size_t need, void** out) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64)
        return fail(MOT_ERR_HIP, "hipGetDevice failed");
    std::lock_guard<std::mutex> lk(g_buf_mu);
    OwnedBuf& b = g_bufs[dev];
    if (b.bytes < need) {
        if (b.ptr) {
            hipError_t e = hipFree(b.ptr);
            b.ptr = nullptr;
            b.bytes = 0;
            if (e != hipSuccess) return fail(MOT_ERR_HIP, "hipFree: %s", hipGetErrorString(e));
        }
        hipError_t e = hipMalloc(&b.ptr, need);
        if (e != hipSuccess) {
            b.ptr = nullptr;
            return fail(MOT_ERR_HIP, "hipMalloc(%zu): %s", need, hipGetErrorString(e));
        }
        b.bytes = need;
    }
    *out = b.ptr;
    return MOT_OK;
}

bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
    const uintptr_t pa = reinterpret_cast<uintptr_t>(a), pb = reinterpret_cast<uintptr_t>(b);
    return na && nb && pa < pb + nb && pb < pa + na;
}

}  // namespace

extern "C" {

int mot_abi_version(void) { return MOT_ABI_VERSION; }

const char* mot_last_error(void) { return g_err; }

const char* mot_status_string(mot_status s) {
    switch (s) {
        case MOT_OK: return "MOT_OK";
        case MOT_ERR_NULL_ARG: return "MOT_ERR_NULL_ARG";
        case MOT_ERR_BAD_SHAPE: return "MOT_ERR_BAD_SHAPE";
        case MOT_ERR_BAD_LAYER_MAP: return "MOT_ERR_BAD_LAYER_MAP";
        case MOT_ERR_UNSUPPORTED: return "MOT_ERR_UNSUPPORTED";
        case MOT_ERR_MISALIGNED: return "MOT_ERR_MISALIGNED";
        case MOT_ERR_WORKSPACE_TOO_SMALL: return "MOT_ERR_WORKSPACE_TOO_SMALL";
        case MOT_ERR_HIP: return "MOT_ERR_HIP";
    }
    return "MOT_ERR_UNKNOWN";
}

mot_status mot_depth_ratio_map(int32_t L_src, int32_t L_tgt, int32_t* out) {
    g_err[0] = 0;
    if (!out) return fail(MOT_ERR_NULL_ARG, "out is NULL");
    if (L_src < 1 || L_src > MOT_MAX_LAYERS || L_tgt < 1 || L_tgt > MOT_MAX_LAYERS)
        return fail(MOT_ERR_BAD_SHAPE, "L_src=%d L_tgt=%d must be in [1, %d]", L_src, L_tgt, MOT_MAX_LAYERS);
    for (int32_t j = 0; j < L_tgt; ++j) out[j] = (int32_t)(((int64_t)j * L_src) / L_tgt);
    return MOT_OK;
}

size_t mot_workspace_bytes(const mot_shapes* shapes) {
    g_err[0] = 0;
    if (check_shapes(shapes) != MOT_OK) return SIZE_MAX;
    static thread_local Plan pl;
    make_plan(shapes, nullptr, &pl);
    return plan_bytes(pl, default_group(pl));
}

mot_status mot_translate(const void* src_k, const void* src_v, const int32_t* layer_map,
                         const mot_translator_weights* tw, const mot_router_weights* rw,
                         void* dst_k, void* dst_v, const mot_shapes* s, hipStream_t stream) {
    g_err[0] = 0;
    mot_status st = check_shapes(s);
    if (st != MOT_OK) return st;
    if ((int64_t)s->B * s->T == 0) return MOT_OK;   // empty context: nothing is read or written
    const bool two = s->streams != 1;   // keys and values, or one activation stream
    if (!src_k || !layer_map || !tw || !rw || !dst_k || (two && (!src_v || !dst_v)))
        return fail(MOT_ERR_NULL_ARG, "a required argument is NULL");
    if (!tw->w1 || !tw->w2 || !rw->w)
        return fail(MOT_ERR_NULL_ARG, "w1, w2 and the router weight are required (biases may be NULL)");
    for (int j = 0; j < s->L_tgt; ++j)
        if (layer_map[j] < -1 || layer_map[j] >= s->L_src)
            return fail(MOT_ERR_BAD_LAYER_MAP, "layer_map[%d]=%d outside [-1, %d)", j, layer_map[j], s->L_src);
    const void* dev_ptrs[] = {src_k, dst_k, tw->w1, tw->w2, rw->w, two ? src_v : src_k, two ? dst_v : dst_k};
    for (const void* q : dev_ptrs)
        if (!aligned16(q)) return fail(MOT_ERR_MISALIGNED, "device pointer %p is not 16-byte aligned", q);
    if (!two) {
        src_v = nullptr;
        dst_v = nullptr;
    }
    const size_t es = s->dtype == MOT_BF16 ? 2 : 4;
    if (s->usage && (reinterpret_cast<uintptr_t>(s->usage) & 3))
        return fail(MOT_ERR_MISALIGNED, "usage %p is not 4-byte aligned", (void*)s->usage);
    const void* bias_ptrs[] = {tw->b1, tw->b2, rw->b};
    for (const void* q : bias_ptrs)
        if (q && !aligned16(q))   // the fused kernel reads b1 in 16-byte pieces
            return fail(MOT_ERR_MISALIGNED, "bias pointer %p is not 16-byte aligned", q);

    static thread_local Plan pl;
    make_plan(s, layer_map, &pl);
    const size_t n_tok = (size_t)pl.n_tok;
    const int d_in = s->H_src * s->D_src, d_out = s->H_tgt * s->D_tgt;
    const size_t src_bytes = (size_t)s->L_src * n_tok * d_in * es;
    const size_t dst_bytes = (size_t)s->L_tgt * n_tok * d_out * es;
    if (overlaps(dst_k, dst_bytes, src_k, src_bytes) ||
        (two && (overlaps(dst_k, dst_bytes, dst_v, dst_bytes) || overlaps(dst_k, dst_bytes, src_v, src_bytes) ||
                 overlaps(dst_v, dst_bytes, src_k, src_bytes) || overlaps(dst_v, dst_bytes, src_v, src_bytes))))
        return fail(MOT_ERR_BAD_SHAPE, "destination caches overlap each other or the source caches");
    const size_t usage_bytes = (size_t)s->L_tgt * (two ? 2 : 1) * s->E * 4;
    if (s->usage && (overlaps(s->usage, usage_bytes, dst_k, dst_bytes) ||
                     (two && overlaps(s->usage, usage_bytes, dst_v, dst_bytes))))
        return fail(MOT_ERR_BAD_SHAPE, "usage overlaps a destination cache");

    // workspace
    int group = default_group(pl);
    void* ws = nullptr;
    const size_t need_min = plan_bytes(pl, pl.n_units ? 1 : 0);
    if (need_min > 0) {
        if (s->workspace) {
            if (!aligned16(s->workspace))
                return fail(MOT_ERR_MISALIGNED, "workspace %p is not 16-byte aligned", s->workspace);
            if (s->workspace_bytes < need_min)
                return fail(MOT_ERR_WORKSPACE_TOO_SMALL, "workspace of %zu bytes, need at least %zu",
                            s->workspace_bytes, need_min);
            if (pl.unit_bytes) {
                size_t g = (s->workspace_bytes - pl.fixed_bytes) / pl.unit_bytes;
                group = (int)(g < (size_t)pl.n_units ? g : (size_t)pl.n_units);
            }
            ws = s->workspace;
            if (overlaps(ws, s->workspace_bytes, dst_k, dst_bytes) ||
                (two && overlaps(ws, s->workspace_bytes, dst_v, dst_bytes)))
                return fail(MOT_ERR_BAD_SHAPE, "workspace overlaps a destination cache");
        }
    }
    if (pl.n_units == 0 || n_tok == 0) return MOT_OK;   // nothing to translate
    if (need_min > 0 && !s->workspace) {
        st = owned_workspace(plan_bytes(pl, group), &ws);
        if (st != MOT_OK) return st;
    }

    Problem p = base_problem(s);
    p.src[0] = src_k; p.src[1] = src_v;
    p.dst[0] = dst_k; p.dst[1] = dst_v;
    p.w1 = tw->w1; p.b1 = tw->b1; p.w2 = tw->w2; p.b2 = tw->b2;
    p.wr = rw->w; p.br = rw->b;
    if (ws && pl.routed) {
        carve_routing(pl, p, ws, &p.rt);
    } else if (ws && pl.routed2) {
        carve_routing(pl, p, ws, &p.rt);
        // after the routing buffers: the group's hidden buffers, then its fp32 rows
        const size_t hid = round_up(bf16_routed_hidden_bytes(p), kAlign);
        p.hbuf = reinterpret_cast<char*>(ws) + pl.fixed_bytes;
        p.rt.part = p.top_k > 1 ? reinterpret_cast<float*>(reinterpret_cast<char*>(ws) + pl.fixed_bytes +
                                                           (size_t)group * hid)
                                : nullptr;
    } else if (ws) {
        p.gates = reinterpret_cast<float*>(ws);
        p.hbuf = reinterpret_cast<char*>(ws) + pl.fixed_bytes;
    }

    static thread_local UnitTab ut;
    hipError_t e = hipSuccess;
    if (pl.routed) {
        ut.n = pl.n_units;
        memcpy(ut.code, pl.codes, sizeof(uint32_t) * pl.n_units);
        e = launch_router_lists(p, ut, stream);
        if (e == hipSuccess) e = launch_route_plan(p, ut, stream);
        for (int u0 = 0; e == hipSuccess && u0 < pl.n_units; u0 += group) {
            const int n = pl.n_units - u0 < group ? pl.n_units - u0 : group;
            ut.n = n;
            memcpy(ut.code, pl.codes + u0, sizeof(uint32_t) * n);
            e = launch_bf16_fused_routed(p, ut, stream);
            if (e == hipSuccess && p.top_k > 1) e = launch_routed_combine(p, ut, stream);
        }
    } else if (pl.routed2) {
        ut.n = pl.n_units;
        memcpy(ut.code, pl.codes, sizeof(uint32_t) * pl.n_units);
        e = launch_router_lists(p, ut, stream);
        if (e == hipSuccess) e = launch_route_plan(p, ut, stream);
        for (int u0 = 0; e == hipSuccess && u0 < pl.n_units; u0 += group) {
            const int n = pl.n_units - u0 < group ? pl.n_units - u0 : group;
            ut.n = n;
            memcpy(ut.code, pl.codes + u0, sizeof(uint32_t) * n);
            e = launch_bf16_gemm1_routed(p, ut, stream);
            if (e == hipSuccess) e = launch_bf16_gemm2_routed(p, ut, stream);
            if (e == hipSuccess && p.top_k > 1) e = launch_routed_combine(p, ut, stream);
        }
    } else if (pl.fused) {
        ut.n = pl.n_units;
        memcpy(ut.code, pl.codes, sizeof(uint32_t) * pl.n_units);
        e = launch_bf16_fused(p, ut, stream);
    } else if (!pl.bf16 && f32_mfma_fits(p)) {
        for (int u0 = 0; e == hipSuccess && u0 < pl.n_units; u0 += group) {
            const int n = pl.n_units - u0 < group ? pl.n_units - u0 : group;
            ut.n = n;
            memcpy(ut.code, pl.codes + u0, sizeof(uint32_t) * n);
            e = launch_f32_mfma_gemm1(p, ut, stream);
            if (e == hipSuccess) e = launch_f32_mfma_gemm2(p, ut, stream);
        }
    } else {
        ut.n = pl.n_units;
        memcpy(ut.code, pl.codes, sizeof(uint32_t) * pl.n_units);
        e = launch_router(p, ut, pl.bf16, stream);
        for (int u0 = 0; e == hipSuccess && u0 < pl.n_units; u0 += group) {
            const int n = pl.n_units - u0 < group ? pl.n_units - u0 : group;
            ut.n = n;
            memcpy(ut.code, pl.codes + u0, sizeof(uint32_t) * n);
            if (pl.bf16 && bf16_gemm256_fits(p, n)) {
                e = launch_bf16_gemm1_256(p, ut, stream);
                if (e == hipSuccess) e = launch_bf16_gemm2_256(p, ut, stream);
            } else if (pl.bf16) {
                e = launch_bf16_gemm1(p, ut, stream);
                if (e == hipSuccess) e = launch_bf16_gemm2(p, ut, stream);
            } else {
                e = launch_f32_gemm1(p, ut, stream);
                if (e == hipSuccess) e = launch_f32_gemm2(p, ut, stream);
            }
        }
    }
    if (e != hipSuccess) return fail(MOT_ERR_HIP, "kernel launch: %s", hipGetErrorString(e));
    return MOT_OK;
}

mot_status mot_usage_stats(const uint32_t* counts, int32_t n, int32_t E, double* cv2, double* entropy,
                           hipStream_t stream) {
    g_err[0] = 0;
    if (n < 0 || E < 1 || E > MOT_MAX_EXPERTS)
        return fail(MOT_ERR_BAD_SHAPE, "n=%d E=%d: need n >= 0 and 1 <= E <= %d", n, E, MOT_MAX_EXPERTS);
    if (n == 0) return MOT_OK;
    if (!counts || !cv2 || !entropy) return fail(MOT_ERR_NULL_ARG, "counts, cv2 and entropy are required");
    if ((reinterpret_cast<uintptr_t>(counts) & 3) || (reinterpret_cast<uintptr_t>(cv2) & 7) ||
        (reinterpret_cast<uintptr_t>(entropy) & 7))
        return fail(MOT_ERR_MISALIGNED, "counts must be 4-byte, cv2 and entropy 8-byte aligned");
    const size_t cb = (size_t)n * E * 4, ob = (size_t)n * 8;
    if (overlaps(counts, cb, cv2, ob) || overlaps(counts, cb, entropy, ob) || overlaps(cv2, ob, entropy, ob))
        return fail(MOT_ERR_BAD_SHAPE, "counts, cv2 and entropy overlap");
    hipError_t e = launch_usage_stats(counts, n, E, cv2, entropy, stream);
    if (e != hipSuccess) return fail(MOT_ERR_HIP, "kernel launch: %s", hipGetErrorString(e));
    return MOT_OK;
}

mot_status mot_restore_kv(const void* act, const int32_t* layer_map, const void* wk, const void* bk,
                          const void* wv, const void* bv, void* dst_k, void* dst_v,
                          const mot_restore_shapes* s, hipStream_t stream) {
    g_err[0] = 0;
    if (!s) return fail(MOT_ERR_NULL_ARG, "shapes is NULL");
    if (s->L < 1 || s->L > MOT_MAX_LAYERS)
        return fail(MOT_ERR_BAD_SHAPE, "L=%d must be in [1, %d]", s->L, MOT_MAX_LAYERS);
    if (s->B < 0 || s->T < 0 || (int64_t)s->B * s->T > (int64_t)1 << 26)
        return fail(MOT_ERR_BAD_SHAPE, "B=%d T=%d: need B, T >= 0 and B*T <= 2^26", s->B, s->T);
    if (s->d_act < 1 || s->d_act > 65536 || s->H_tgt < 1 || s->D_tgt < 1 || (int64_t)s->H_tgt * s->D_tgt > 65536)
        return fail(MOT_ERR_BAD_SHAPE, "d_act, H_tgt, D_tgt must be >= 1 and rows at most 65536 wide");
    if (s->dtype != MOT_F32 && s->dtype != MOT_BF16)
        return fail(MOT_ERR_BAD_SHAPE, "dtype=%d is not MOT_F32 or MOT_BF16", s->dtype);
    if (s->dst_layout != MOT_LAYOUT_BTHD && s->dst_layout != MOT_LAYOUT_BHTD)
        return fail(MOT_ERR_BAD_SHAPE, "dst_layout must be MOT_LAYOUT_BTHD or MOT_LAYOUT_BHTD");
    if (s->dtype != MOT_BF16 || s->d_act % 64 || s->D_tgt % 8)
        return fail(MOT_ERR_UNSUPPORTED, "restore needs bf16, d_act %% 64 == 0 and D_tgt %% 8 == 0 "
                    "(got dtype=%d d_act=%d D_tgt=%d)", s->dtype, s->d_act, s->D_tgt);
    if ((int64_t)s->B * s->T == 0) return MOT_OK;
    if (!act || !wk || !wv || !dst_k || !dst_v)
        return fail(MOT_ERR_NULL_ARG, "act, wk, wv, dst_k and dst_v are required (biases may be NULL)");
    const void* dev_ptrs[] = {act, wk, wv, dst_k, dst_v};
    for (const void* q : dev_ptrs)
        if (!aligned16(q)) return fail(MOT_ERR_MISALIGNED, "device pointer %p is not 16-byte aligned", q);
    if ((bk && (reinterpret_cast<uintptr_t>(bk) & 1)) || (bv && (reinterpret_cast<uintptr_t>(bv) & 1)))
        return fail(MOT_ERR_MISALIGNED, "bias pointers must be 2-byte aligned");
    const size_t n_tok = (size_t)s->B * s->T, d_kv = (size_t)s->H_tgt * s->D_tgt;
    const size_t act_bytes = (size_t)s->L * n_tok * s->d_act * 2, kv_bytes = (size_t)s->L * n_tok * d_kv * 2;
    if (overlaps(dst_k, kv_bytes, dst_v, kv_bytes) || overlaps(dst_k, kv_bytes, act, act_bytes) ||
        overlaps(dst_v, kv_bytes, act, act_bytes))
        return fail(MOT_ERR_BAD_SHAPE, "destination caches overlap each other or the activation");
    static thread_local ProjProblem p;
    memset(&p, 0, sizeof p);
    p.act = act; p.wk = wk; p.bk = bk; p.wv = wv; p.bv = bv; p.dst_k = dst_k; p.dst_v = dst_v;
    p.B = s->B; p.T = s->T; p.n_tok = (int32_t)n_tok; p.d_act = s->d_act; p.d_kv = (int32_t)d_kv;
    p.H_tgt = s->H_tgt; p.D_tgt = s->D_tgt; p.dst_layout = s->dst_layout;
    int n = 0;
    for (int l = 0; l < s->L; ++l)
        if (!layer_map || layer_map[l] >= 0) p.layers[n++] = l;
    hipError_t e = bf16_project_256_fits(p, n) ? launch_bf16_project_256(p, n, stream)
                                               : launch_bf16_project(p, n, stream);
    if (e != hipSuccess) return fail(MOT_ERR_HIP, "kernel launch: %s", hipGetErrorString(e));
    return MOT_OK;
}

namespace {
// Offsets (elements) of one expert's packed backbone parameters over a
// channel window of N slots, in the order the header documents: the shared
// input projection, N cross-attention blocks of `cab` elements each (the
// block offsets are relative to the block's start), the output projection.
// N = 1 is the single-slot packing.
struct BackboneOffsets {
    size_t ln_in_g, ln_in_b, w_in, b_in, cab0, cab;
    size_t ln_q_g, ln_q_b, ln_c_g, ln_c_b, wq, bq, wk, bk, wv, bv, wo, bo, ln_f_g, ln_f_b, w_f1, b_f1, w_f2, b_f2;
    size_t ln_out_g, ln_out_b, w_out, b_out, total;
};
BackboneOffsets backbone_offsets(size_t d_in, size_t d_h, size_t d_ff, size_t d_out, size_t N) {
    BackboneOffsets o;
    size_t at = 0;
    auto take = [&](size_t n) { const size_t r = at; at += n; return r; };
    o.ln_in_g = take(d_in); o.ln_in_b = take(d_in); o.w_in = take(d_h * d_in); o.b_in = take(d_h);
    o.cab0 = at;
    at = 0;
    o.ln_q_g = take(d_h); o.ln_q_b = take(d_h); o.ln_c_g = take(d_h); o.ln_c_b = take(d_h);
    o.wq = take(d_h * d_h); o.bq = take(d_h); o.wk = take(d_h * d_h); o.bk = take(d_h);
    o.wv = take(d_h * d_h); o.bv = take(d_h); o.wo = take(d_h * d_h); o.bo = take(d_h);
    o.ln_f_g = take(d_h); o.ln_f_b = take(d_h); o.w_f1 = take(d_ff * d_h); o.b_f1 = take(d_ff);
    o.w_f2 = take(d_h * d_ff); o.b_f2 = take(d_h);
    o.cab = at;
    at = o.cab0 + N * o.cab;
    o.ln_out_g = take(N * d_h); o.ln_out_b = take(N * d_h);
    o.w_out = take(N * d_out * N * d_h); o.b_out = take(N * d_out);
    o.total = at;
    return o;
}

mot_status check_replay(const mot_replay_shapes* s, bool need_s) {
    if (!s) return fail(MOT_ERR_NULL_ARG, "shapes is NULL");
    if (s->B < 0 || s->T < 0 || (int64_t)s->B * s->T > (int64_t)1 << 26)
        return fail(MOT_ERR_BAD_SHAPE, "B=%d T=%d: need B, T >= 0 and B*T <= 2^26", s->B, s->T);
    if (s->H_q < 1 || s->H_kv < 1 || s->H_q % s->H_kv || s->D < 1)
        return fail(MOT_ERR_BAD_SHAPE, "H_q=%d H_kv=%d D=%d: need H_q a positive multiple of H_kv and D >= 1",
                    s->H_q, s->H_kv, s->D);
    if (s->kv_layout != MOT_LAYOUT_BTHD && s->kv_layout != MOT_LAYOUT_BHTD)
        return fail(MOT_ERR_BAD_SHAPE, "kv_layout must be MOT_LAYOUT_BTHD or MOT_LAYOUT_BHTD");
    if (need_s && s->S < 1) return fail(MOT_ERR_BAD_SHAPE, "S=%d must be >= 1", s->S);
    if (s->D != 64 && s->D != 128)
        return fail(MOT_ERR_UNSUPPORTED, "D=%d: replay attention supports head dims 64 and 128", s->D);
    if ((int64_t)s->H_kv * s->D >= (1 << 20))
        return fail(MOT_ERR_UNSUPPORTED, "H_kv * D = %lld: at most 2^20 - 1", (long long)s->H_kv * s->D);
    if (s->H_q / s->H_kv > 16)
        return fail(MOT_ERR_UNSUPPORTED, "%d query heads per KV head (at most 16)", s->H_q / s->H_kv);
    if (need_s && !replay_sparse_supported(s->D, s->S))
        return fail(MOT_ERR_UNSUPPORTED, "S=%d: need a multiple of 32 from 32 to %d for D = %d", s->S,
                    replay_sparse_smax(s->D), s->D);
    if (!need_s && !replay_causal_supported(s->T, s->H_kv, s->D, s->kv_layout == MOT_LAYOUT_BTHD))
        return fail(MOT_ERR_UNSUPPORTED, "T=%d: a batch row's K of %lld bytes exceeds the 2 GiB the causal kernel "
                    "addresses", s->T,
                    (long long)s->T * (s->kv_layout == MOT_LAYOUT_BTHD ? s->H_kv * s->D : s->D) * 2);
    return MOT_OK;
}
}  // namespace

mot_status mot_topS_select(const float* A, int32_t* idx, const mot_replay_shapes* s, hipStream_t stream) {
    g_err[0] = 0;
    if (!s) return fail(MOT_ERR_NULL_ARG, "shapes is NULL");
    if (s->B < 0 || s->T < 0 || (int64_t)s->B * s->T > (int64_t)1 << 26 || s->S < 1)
        return fail(MOT_ERR_BAD_SHAPE, "B=%d T=%d S=%d: need B, T >= 0, B*T <= 2^26, S >= 1", s->B, s->T, s->S);
    if (s->T > 65536) return fail(MOT_ERR_UNSUPPORTED, "T=%d: selection supports rows of up to 65536 positions", s->T);
    if ((int64_t)s->B * s->T == 0) return MOT_OK;
    if (!A || !idx) return fail(MOT_ERR_NULL_ARG, "A and idx are required");
    if ((reinterpret_cast<uintptr_t>(A) & 3) || (reinterpret_cast<uintptr_t>(idx) & 3))
        return fail(MOT_ERR_MISALIGNED, "A and idx must be 4-byte aligned");
    if (overlaps(A, (size_t)s->B * s->T * s->T * 4, idx, (size_t)s->B * s->T * s->S * 4))
        return fail(MOT_ERR_BAD_SHAPE, "idx overlaps A");
    hipError_t e = launch_topS_select(A, idx, s->B, s->T, s->S, stream);
    if (e != hipSuccess) return fail(MOT_ERR_HIP, "kernel launch: %s", hipGetErrorString(e));
    return MOT_OK;
}

namespace {
// Scratch of mot_replay_attention_noalloc: the full causal path's V staging
// in a file-scope device array, so that entry point allocates nothing.
// Every device that runs the library holds its own copy until the process
// ends; host code reaches it only through the address hipGetSymbolAddress
// returns for the current device (the array's name is a host stand-in).
constexpr size_t kNoAllocScratchBytes = size_t(32) << 20;
__device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];
std::mutex g_scratch_mu;
void* g_scratch_ptr[64];

// Device address of `scratch` on the current device, looked up on the first
// call per device (with that device current) and kept.
mot_status noalloc_scratch(void** out) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return fail(MOT_ERR_HIP, "hipGetDevice failed");
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* ptr = nullptr;
        const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !ptr)
            return fail(MOT_ERR_HIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
        g_scratch_ptr[dev] = ptr;
    }
    *out = g_scratch_ptr[dev];
    return MOT_OK;
}

enum class ReplayScratch { Caller, Static };

mot_status replay_attention_impl(const void* q, const void* k, const void* v, const int32_t* idx, void* o,
                                 const mot_replay_shapes* s, hipStream_t stream, ReplayScratch mode);
}  // namespace

mot_status mot_replay_attention(const void* q, const void* k, const void* v, const int32_t* idx, void* o,
                                const mot_replay_shapes* s, hipStream_t stream) {
    g_err[0] = 0;
    return replay_attention_impl(q, k, v, idx, o, s, stream, ReplayScratch::Caller);
}

mot_status mot_replay_attention_noalloc(const void* q, const void* k, const void* v, const int32_t* idx, void* o,
                                        const mot_replay_shapes* s, hipStream_t stream) {
    g_err[0] = 0;
    return replay_attention_impl(q, k, v, idx, o, s, stream, ReplayScratch::Static);
}

namespace {
mot_status replay_attention_impl(const void* q, const void* k, const void* v, const int32_t* idx, void* o,
                                 const mot_replay_shapes* s, hipStream_t stream, ReplayScratch mode) {
    mot_status st = check_replay(s, idx != nullptr);
    if (st != MOT_OK) return st;
    if ((int64_t)s->B * s->T == 0) return MOT_OK;
    if (!q || !k || !v || !o) return fail(MOT_ERR_NULL_ARG, "q, k, v and o are required");
    const void* ptrs[] = {q, k, v, o, idx ? static_cast<const void*>(idx) : q};
    for (const void* x : ptrs)
        if (!aligned16(x)) return fail(MOT_ERR_MISALIGNED, "device pointer %p is not 16-byte aligned", x);
    const size_t qo = (size_t)s->B * s->T * s->H_q * s->D * 2, kv = (size_t)s->B * s->T * s->H_kv * s->D * 2;
    if (overlaps(o, qo, q, qo) || overlaps(o, qo, k, kv) || overlaps(o, qo, v, kv) ||
        (idx && overlaps(o, qo, idx, (size_t)s->B * s->T * s->S * 4)))
        return fail(MOT_ERR_BAD_SHAPE, "o overlaps an input");
    ReplayProblem p;
    p.q = q; p.k = k; p.v = v; p.idx = idx; p.o = o; p.vt = nullptr;
    p.B = s->B; p.T = s->T; p.H_q = s->H_q; p.H_kv = s->H_kv; p.D = s->D; p.S = idx ? s->S : 0;
    p.kv_layout = s->kv_layout;
    if (!idx) {   // the full causal path stages V transposed through scratch
        const size_t need = replay_vt_bytes(s->B, s->T, s->H_kv, s->D);
        void* ws = mode == ReplayScratch::Caller ? s->workspace : nullptr;
        if (mode == ReplayScratch::Static) {
            // every position of the staged V is written before it is read
            // (zero past T), so nothing has to be cleared between calls
            if (need > kNoAllocScratchBytes)
                return fail(MOT_ERR_WORKSPACE_TOO_SMALL, "the staged V needs %zu bytes; the static scratch holds %zu",
                            need, kNoAllocScratchBytes);
            st = noalloc_scratch(&ws);
            if (st != MOT_OK) return st;
        } else if (ws) {
            if (!aligned16(ws)) return fail(MOT_ERR_MISALIGNED, "workspace %p is not 16-byte aligned", ws);
            if (s->workspace_bytes < need)
                return fail(MOT_ERR_WORKSPACE_TOO_SMALL, "workspace of %zu bytes, need %zu", s->workspace_bytes,
                            need);
            if (overlaps(ws, need, q, qo) || overlaps(ws, need, k, kv) || overlaps(ws, need, v, kv) ||
                overlaps(ws, need, o, qo))
                return fail(MOT_ERR_BAD_SHAPE, "workspace overlaps q, k, v or o");
        } else {
            st = owned_workspace(need, &ws);
            if (st != MOT_OK) return st;
        }
        p.vt = reinterpret_cast<uint16_t*>(ws);
    }
    hipError_t e = launch_replay_attention(p, stream);
    if (e != hipSuccess) return fail(MOT_ERR_HIP, "kernel launch: %s", hipGetErrorString(e));
    return MOT_OK;
}
}  // namespace

size_t mot_replay_workspace_bytes(const mot_replay_shapes* s, int with_sets) {
    g_err[0] = 0;
    if (check_replay(s, with_sets != 0) != MOT_OK) return SIZE_MAX;
    return with_sets ? 0 : replay_vt_bytes(s->B, s->T, s->H_kv, s->D);
}

constexpr int kMaxSlots = 8;   // channel-window slots of the backbone

int backbone_slots(const mot_backbone_dims* bd) { return bd->n_slots > 1 ? bd->n_slots : 1; }

size_t mot_backbone_param_count(const mot_shapes* s, const mot_backbone_dims* bd) {
    if (!s || !bd || s->H_src < 1 || s->D_src < 1 || s->H_tgt < 1 || s->D_tgt < 1 || bd->d_h < 1 || bd->d_ff < 1 ||
        bd->n_slots < 0 || bd->n_slots > kMaxSlots)
        return 0;
    return backbone_offsets((size_t)s->H_src * s->D_src, bd->d_h, bd->d_ff, (size_t)s->H_tgt * s->D_tgt,
                            backbone_slots(bd)).total;
}

namespace {
// Workspace of the backbone call: the gates of every unit, then the
// activations of one batch of ub units, each with its E experts as groups of
// grouped launches (group g = unit-in-batch * E + expert, every buffer
// group-major), then the attention's transposed V.  Buffers, in order: LN_in
// rows [g][n][d_in], z of the N slots [g][N][n][d_h], LN_Q and LN_C rows, Q,
// K, V, attention, h~, LN_F rows [g][n][d_h], FFN hidden [g][n][d_ff],
// Concat(h_1..h_N) and its LayerNorm [g][n][N d_h], the fp32 mixture
// [unit][N][n][d_out], the window's concatenated source rows [unit][n][N d_in]
// (N > 1: the router's input).
constexpr int kBbBufs = 15;
constexpr size_t kBackboneBatchCap = size_t(8) << 30;   // activation bytes per batch of units
struct BackboneScratch {
    size_t gates;             // bytes of the gates of every unit
    size_t at[kBbBufs];       // offsets of the batch buffers
    size_t at_vt;
    size_t total;
};
// bytes of one unit's share of the batch buffers (its E groups and mixture)
size_t backbone_unit_bytes(const mot_shapes* s, const mot_backbone_dims* bd) {
    const size_t n = (size_t)s->B * s->T, d_in = (size_t)s->H_src * s->D_src, d_out = (size_t)s->H_tgt * s->D_tgt;
    const size_t d_h = bd->d_h, d_ff = bd->d_ff, N = bd->n_slots > 1 ? bd->n_slots : 1, E = s->E;
    const size_t per_group = n * 2 * (d_in + N * d_h + 9 * d_h + d_ff + 2 * N * d_h);
    const size_t vt = replay_vt_bytes(s->B, s->T, bd->n_heads, bd->d_h / bd->n_heads);
    return E * (per_group + vt) + n * N * d_out * 4 + (N > 1 ? n * N * d_in * 2 : 0) + 16 * kAlign;
}
BackboneScratch backbone_scratch(const mot_shapes* s, const mot_backbone_dims* bd, int n_units, int ub) {
    const size_t n = (size_t)s->B * s->T, d_in = (size_t)s->H_src * s->D_src, d_out = (size_t)s->H_tgt * s->D_tgt;
    const size_t d_h = bd->d_h, d_ff = bd->d_ff, N = bd->n_slots > 1 ? bd->n_slots : 1;
    const size_t G = (size_t)ub * s->E;
    const size_t row_b[kBbBufs] = {G * d_in * 2, G * N * d_h * 2, G * d_h * 2, G * d_h * 2, G * d_h * 2,
                                   G * d_h * 2,  G * d_h * 2,     G * d_h * 2, G * d_h * 2, G * d_h * 2,
                                   G * d_ff * 2, G * N * d_h * 2, G * N * d_h * 2,
                                   (size_t)ub * N * d_out * 4, N > 1 ? (size_t)ub * N * d_in * 2 : 0};
    BackboneScratch b;
    b.gates = round_up((size_t)n_units * round_up(n, 128) * s->E * 4, kAlign);
    size_t need = b.gates;
    for (int k = 0; k < kBbBufs; ++k) { b.at[k] = need; need += round_up(n * row_b[k], kAlign); }
    b.at_vt = need;
    need += round_up(replay_vt_bytes((int)(s->B * G), s->T, bd->n_heads, bd->d_h / bd->n_heads), kAlign);
    b.total = need;
    return b;
}
// units per batch: every unit when they fit the cap, at most kLinearTab
int backbone_batch(const mot_shapes* s, const mot_backbone_dims* bd, int n_units) {
    size_t ub = kBackboneBatchCap / backbone_unit_bytes(s, bd);
    if (ub < 1) ub = 1;
    if (ub > (size_t)kLinearTab) ub = kLinearTab;
    if (ub > (size_t)n_units) ub = n_units;
    return (int)ub;
}

mot_status check_backbone(const mot_shapes* s, const mot_backbone_dims* bd) {
    mot_status st = check_shapes(s);
    if (st != MOT_OK) return st;
    if (!bd) return fail(MOT_ERR_NULL_ARG, "backbone dims are NULL");
    const int d_in = s->H_src * s->D_src, d_out = s->H_tgt * s->D_tgt, d_h = bd->d_h, nh = bd->n_heads,
              d_ff = bd->d_ff;
    if (d_h < 1 || nh < 1 || d_ff < 1 || d_h % nh)
        return fail(MOT_ERR_BAD_SHAPE, "d_h=%d n_heads=%d d_ff=%d: need positive sizes, d_h a multiple of n_heads",
                    d_h, nh, d_ff);
    if (bd->n_slots < 0 || bd->n_slots > kMaxSlots)
        return fail(MOT_ERR_BAD_SHAPE, "n_slots=%d must be in [0, %d]", bd->n_slots, kMaxSlots);
    const int N = backbone_slots(bd);
    if (s->L_tgt % N)
        return fail(MOT_ERR_BAD_SHAPE, "L_tgt=%d is not a multiple of the window of %d slots", s->L_tgt, N);
    if (s->dtype != MOT_BF16 || s->src_layout != MOT_LAYOUT_BTHD || s->dst_layout != MOT_LAYOUT_BTHD ||
        s->streams == 1)
        return fail(MOT_ERR_UNSUPPORTED, "the backbone translator needs bf16, BTHD source and target layouts, "
                    "keys and values (streams = 2)");
    if (d_in % 64 || d_in > 4096 || d_h % 64 || d_h > 4096 || N * d_h > 4096 || d_ff % 64 || d_out % 8 ||
        (d_h / nh != 64 && d_h / nh != 128))
        return fail(MOT_ERR_UNSUPPORTED, "backbone sizes: d_in, d_h multiples of 64 up to 4096 (n_slots * d_h too), "
                    "d_ff a multiple of 64, d_out of 8, head width d_h / n_heads 64 or 128 (got d_in=%d d_h=%d "
                    "n_heads=%d d_ff=%d d_out=%d n_slots=%d)", d_in, d_h, nh, d_ff, d_out, N);
    if (!replay_causal_supported(s->T, nh, d_h / nh, true))
        return fail(MOT_ERR_UNSUPPORTED, "T=%d: a batch row's attention keys (%lld bytes) exceed the 2 GiB the "
                    "causal kernel addresses", s->T, (long long)s->T * d_h * 2);
    return MOT_OK;
}
}  // namespace

size_t mot_backbone_workspace_bytes(const mot_shapes* s, const mot_backbone_dims* bd) {
    g_err[0] = 0;
    if (check_backbone(s, bd) != MOT_OK) return SIZE_MAX;
    if ((int64_t)s->B * s->T == 0) return 0;
    const int nu = 2 * s->L_tgt / backbone_slots(bd);
    return backbone_scratch(s, bd, nu, backbone_batch(s, bd, nu)).total;
}

mot_status mot_backbone_translate(const void* src_k, const void* src_v, const int32_t* layer_map, const void* params,
                                  const mot_router_weights* rw, void* dst_k, void* dst_v, const mot_shapes* s,
                                  const mot_backbone_dims* bd, hipStream_t stream) {
    g_err[0] = 0;
    mot_status st = check_backbone(s, bd);
    if (st != MOT_OK) return st;
    const int d_in = s->H_src * s->D_src, d_out = s->H_tgt * s->D_tgt, d_h = bd->d_h, nh = bd->n_heads,
              d_ff = bd->d_ff, N = backbone_slots(bd), W = s->L_tgt / N;
    if ((int64_t)s->B * s->T == 0) return MOT_OK;
    if (!src_k || !src_v || !layer_map || !params || !rw || !rw->w || !dst_k || !dst_v)
        return fail(MOT_ERR_NULL_ARG, "a required argument is NULL");
    for (int j = 0; j < s->L_tgt; ++j)
        if (layer_map[j] < -1 || layer_map[j] >= s->L_src)
            return fail(MOT_ERR_BAD_LAYER_MAP, "layer_map[%d]=%d outside [-1, %d)", j, layer_map[j], s->L_src);
    for (int w = 0; w < W; ++w)
        for (int r = 1; r < N; ++r)
            if ((layer_map[w * N + r] < 0) != (layer_map[w * N] < 0))
                return fail(MOT_ERR_BAD_LAYER_MAP, "window %d (target layers %d..%d) mixes mapped and unmapped slots",
                            w, w * N, w * N + N - 1);
    const void* dev_ptrs[] = {src_k, src_v, params, rw->w, dst_k, dst_v};
    for (const void* q : dev_ptrs)
        if (!aligned16(q)) return fail(MOT_ERR_MISALIGNED, "device pointer %p is not 16-byte aligned", q);
    if (rw->b && (reinterpret_cast<uintptr_t>(rw->b) & 1)) return fail(MOT_ERR_MISALIGNED, "router bias misaligned");
    if (s->usage && (reinterpret_cast<uintptr_t>(s->usage) & 3))
        return fail(MOT_ERR_MISALIGNED, "usage %p is not 4-byte aligned", (void*)s->usage);
    const size_t n = (size_t)s->B * s->T;
    const size_t dst_bytes = (size_t)s->L_tgt * n * d_out * 2, src_bytes = (size_t)s->L_src * n * d_in * 2;
    if (overlaps(dst_k, dst_bytes, dst_v, dst_bytes) || overlaps(dst_k, dst_bytes, src_k, src_bytes) ||
        overlaps(dst_k, dst_bytes, src_v, src_bytes) || overlaps(dst_v, dst_bytes, src_k, src_bytes) ||
        overlaps(dst_v, dst_bytes, src_v, src_bytes))
        return fail(MOT_ERR_BAD_SHAPE, "destination caches overlap each other or the source caches");

    const BackboneOffsets off = backbone_offsets(d_in, d_h, d_ff, d_out, N);
    Problem p = base_problem(s);
    // one unit per (window, X): the window index plays the target layer's
    // part in the unit code (weights, router, usage are per window)
    static thread_local UnitTab ut;
    int nu = 0;
    for (int w = 0; w < W; ++w)
        if (layer_map[w * N] >= 0)
            for (int x = 0; x < 2; ++x) { ut.code[nu] = unit_code(w, x, layer_map[w * N], nu); ++nu; }
    ut.n = nu;
    if (nu == 0) return MOT_OK;
    // workspace: gates, then one batch of units' activations, then V transposed;
    // a caller workspace below the default batch's need gets smaller batches
    int ub = backbone_batch(s, bd, nu);
    BackboneScratch sc = backbone_scratch(s, bd, nu, ub);
    void* ws = s->workspace;
    if (ws) {
        if (!aligned16(ws)) return fail(MOT_ERR_MISALIGNED, "workspace %p is not 16-byte aligned", ws);
        while (ub > 1 && s->workspace_bytes < sc.total) sc = backbone_scratch(s, bd, nu, --ub);
        if (s->workspace_bytes < sc.total)
            return fail(MOT_ERR_WORKSPACE_TOO_SMALL, "workspace of %zu bytes, need at least %zu", s->workspace_bytes,
                        sc.total);
        if (overlaps(ws, sc.total, dst_k, dst_bytes) || overlaps(ws, sc.total, dst_v, dst_bytes) ||
            overlaps(ws, sc.total, src_k, src_bytes) || overlaps(ws, sc.total, src_v, src_bytes))
            return fail(MOT_ERR_BAD_SHAPE, "workspace overlaps a source or destination cache");
    } else {
        st = owned_workspace(sc.total, &ws);
        if (st != MOT_OK) return st;
    }
    char* w8 = reinterpret_cast<char*>(ws);
    auto buf = [&](int k) { return reinterpret_cast<uint16_t*>(w8 + sc.at[k]); };
    uint16_t *xn = buf(0), *z = buf(1), *qn = buf(2), *cn = buf(3), *Q = buf(4), *K = buf(5), *V = buf(6),
             *att = buf(7), *h1 = buf(8), *fn = buf(9), *f1 = buf(10), *F = buf(11), *on = buf(12), *xcat = buf(14);
    float* mix = reinterpret_cast<float*>(w8 + sc.at[13]);   // [unit][N][n][d_out]
    uint16_t* vt = reinterpret_cast<uint16_t*>(w8 + sc.at_vt);

    p.src[0] = src_k; p.src[1] = src_v; p.wr = rw->w; p.br = rw->b;
    p.gates = reinterpret_cast<float*>(ws);
    hipError_t e = hipSuccess;
    if (N == 1) e = launch_router(p, ut, true, stream);   // every unit at once
    const uint16_t* P0 = reinterpret_cast<const uint16_t*>(params);
    const int n_i = (int)n, E = s->E;
    const size_t ldF = (size_t)N * d_h, P = off.total, nz = n * (size_t)d_h, nF = n * ldF;
    const bool fuse_in = d_in <= kLinearLnMaxK, fuse_h = d_h <= kLinearLnMaxK, fuse_out = N * d_h <= kLinearLnMaxK;
    auto pidx = [&](int u) { return unit_j(ut.code[u]) * 2 + unit_x(ut.code[u]); };   // the unit's parameter block

    for (int u0 = 0; u0 < nu && e == hipSuccess;) {
        // a batch: up to ub units whose parameter blocks are consecutive
        int nb = 1;
        while (nb < ub && u0 + nb < nu && pidx(u0 + nb) == pidx(u0) + nb) ++nb;
        const int G = nb * E;
        const uint16_t* Pb = P0 + (size_t)pidx(u0) * E * P;   // group g = (u - u0) * E + m at Pb + g * P
        auto src_slot = [&](int u, int r) {
            const uint32_t code = ut.code[u];
            const uint16_t* sx = reinterpret_cast<const uint16_t*>(unit_x(code) ? src_v : src_k);
            return sx + (size_t)layer_map[unit_j(code) * N + r] * n * d_in;
        };
        if (N > 1) {
            // the router reads each window's concatenated source rows
            static thread_local UnitTab bt;
            bt.n = nb;
            for (int u = 0; u < nb && e == hipSuccess; ++u) {
                const uint32_t code = ut.code[u0 + u];
                for (int r = 0; r < N && e == hipSuccess; ++r)
                    e = hipMemcpy2DAsync(xcat + (size_t)u * n * N * d_in + (size_t)r * d_in, (size_t)N * d_in * 2,
                                         src_slot(u0 + u, r), (size_t)d_in * 2, (size_t)d_in * 2, n,
                                         hipMemcpyDeviceToDevice, stream);
                bt.code[u] = unit_code(unit_j(code), unit_x(code), u, unit_gslot(code));
            }
            Problem pr = p;
            pr.src[0] = pr.src[1] = xcat;
            pr.d_in = N * d_in; pr.H_src = 1; pr.D_src = N * d_in; pr.src_layout = MOT_LAYOUT_BTHD;
            if (e == hipSuccess) e = launch_router(pr, bt, true, stream);
        }
        // grouped launches over the batch's G groups (parameters at stride P)
        auto part = [&](size_t o, int N_, uint16_t* out, size_t ln_g = SIZE_MAX, size_t ln_b = SIZE_MAX) {
            LinearPart q;
            q.W = Pb + o; q.bias = nullptr; q.ln_g = ln_g == SIZE_MAX ? nullptr : Pb + ln_g;
            q.ln_b = ln_b == SIZE_MAX ? nullptr : Pb + ln_b; q.out = out; q.N = N_;
            return q;
        };
        auto lin = [&](const uint16_t* in, size_t ld_in, size_t in_gs, int K_, int gelu, const uint16_t* res,
                       size_t ld_res, size_t res_gs, size_t ld_out, size_t out_gs, int np, LinearPart* ps,
                       const size_t* bias_off) {
            LinearProblem lp;
            memset(&lp, 0, sizeof lp);
            lp.in = in; lp.ld_in = ld_in; lp.in_gs = in_gs; lp.res = res; lp.ld_res = ld_res; lp.res_gs = res_gs;
            lp.ld_out = ld_out; lp.out_gs = out_gs; lp.w_gs = P; lp.groups = G;
            lp.n = n_i; lp.K = K_; lp.gelu = gelu;
            lp.nparts = np;
            for (int q = 0; q < np; ++q) {
                lp.part[q] = ps[q];
                lp.part[q].bias = Pb + bias_off[q];
            }
            return launch_linear(lp, stream);
        };
        // grouped LayerNorm rows (parameters at stride P)
        auto ln = [&](const uint16_t* in, size_t ld_in, size_t in_gs, int wd, size_t g_off, size_t b_off,
                      uint16_t* out, size_t out_gs, size_t g2_off, size_t b2_off, uint16_t* out2) {
            LnProblem q;
            q.in = in; q.ld_in = ld_in; q.g = Pb + g_off; q.b = Pb + b_off; q.out = out;
            q.g2 = out2 ? Pb + g2_off : nullptr; q.b2 = out2 ? Pb + b2_off : nullptr; q.out2 = out2;
            q.n = n_i; q.w = wd; q.groups = G; q.in_gs = in_gs; q.p_gs = P; q.out_gs = out_gs;
            return launch_ln_rows(q, stream);
        };
        // z_r = GELU(W_in LN_in(x_r) + b_in), every slot; the source rows come
        // from each unit's table entry (groups of one unit share them)
        for (int r = 0; r < N && e == hipSuccess; ++r) {
            if (fuse_in) {
                LinearProblem lp;
                memset(&lp, 0, sizeof lp);
                for (int u = 0; u < nb; ++u) lp.in_tab[u] = src_slot(u0 + u, r);
                lp.tab_div = E;
                lp.ld_in = d_in; lp.w_gs = P; lp.groups = G;
                lp.out_gs = N * nz;
                lp.nparts = 1;
                lp.part[0] = part(off.w_in, d_h, z + (size_t)r * nz, off.ln_in_g, off.ln_in_b);
                lp.part[0].bias = Pb + off.b_in;
                lp.n = n_i; lp.K = d_in; lp.gelu = 1;
                e = launch_linear(lp, stream);
            } else {
                // LN_in per unit (its E experts' parameters as groups), then the projection
                for (int u = 0; u < nb && e == hipSuccess; ++u) {
                    LnProblem q;
                    q.in = src_slot(u0 + u, r); q.ld_in = d_in;
                    q.g = Pb + (size_t)u * E * P + off.ln_in_g; q.b = Pb + (size_t)u * E * P + off.ln_in_b;
                    q.g2 = q.b2 = nullptr; q.out2 = nullptr;
                    q.out = xn + (size_t)u * E * n * d_in;
                    q.n = n_i; q.w = d_in; q.groups = E; q.in_gs = 0; q.p_gs = P; q.out_gs = n * d_in;
                    e = launch_ln_rows(q, stream);
                }
                LinearPart q = part(off.w_in, d_h, z + (size_t)r * nz);
                const size_t bo[1] = {off.b_in};
                if (e == hipSuccess) e = lin(xn, d_in, n * d_in, d_in, 1, nullptr, 0, 0, 0, N * nz, 1, &q, bo);
            }
        }
        // the scan h_0 = z_1, h_r = CAB_r(h_{r-1}, z_r); h_r goes to slot r of F
        for (int r = 0; r < N && e == hipSuccess; ++r) {
            const size_t C = off.cab0 + (size_t)r * off.cab;
            const uint16_t* zr = z + (size_t)r * nz;
            const uint16_t* hp = r == 0 ? z : F + (size_t)(r - 1) * d_h;   // h_{r-1}
            const size_t ld_hp = r == 0 ? (size_t)d_h : ldF, hp_gs = r == 0 ? N * nz : nF;
            // Q = Wq LN_Q(h_{r-1}) + bq; K, V = Wk, Wv LN_C(z_r) + bk, bv
            if (fuse_h && r == 0) {
                LinearPart q[3] = {part(C + off.wq, d_h, Q, C + off.ln_q_g, C + off.ln_q_b),
                                   part(C + off.wk, d_h, K, C + off.ln_c_g, C + off.ln_c_b),
                                   part(C + off.wv, d_h, V, C + off.ln_c_g, C + off.ln_c_b)};
                const size_t bo[3] = {C + off.bq, C + off.bk, C + off.bv};
                e = lin(zr, d_h, N * nz, d_h, 0, nullptr, 0, 0, 0, nz, 3, q, bo);
            } else if (fuse_h) {
                LinearPart q = part(C + off.wq, d_h, Q, C + off.ln_q_g, C + off.ln_q_b);
                LinearPart kv[2] = {part(C + off.wk, d_h, K, C + off.ln_c_g, C + off.ln_c_b),
                                    part(C + off.wv, d_h, V, C + off.ln_c_g, C + off.ln_c_b)};
                const size_t bq[1] = {C + off.bq}, bkv[2] = {C + off.bk, C + off.bv};
                e = lin(hp, ld_hp, hp_gs, d_h, 0, nullptr, 0, 0, 0, nz, 1, &q, bq);
                if (e == hipSuccess) e = lin(zr, d_h, N * nz, d_h, 0, nullptr, 0, 0, 0, nz, 2, kv, bkv);
            } else {
                if (r == 0) {
                    e = ln(zr, d_h, N * nz, d_h, C + off.ln_q_g, C + off.ln_q_b, qn, nz, C + off.ln_c_g,
                           C + off.ln_c_b, cn);
                } else {
                    e = ln(hp, ld_hp, hp_gs, d_h, C + off.ln_q_g, C + off.ln_q_b, qn, nz, 0, 0, nullptr);
                    if (e == hipSuccess)
                        e = ln(zr, d_h, N * nz, d_h, C + off.ln_c_g, C + off.ln_c_b, cn, nz, 0, 0, nullptr);
                }
                LinearPart q = part(C + off.wq, d_h, Q);
                LinearPart kv[2] = {part(C + off.wk, d_h, K), part(C + off.wv, d_h, V)};
                const size_t bq[1] = {C + off.bq}, bkv[2] = {C + off.bk, C + off.bv};
                if (e == hipSuccess) e = lin(qn, d_h, nz, d_h, 0, nullptr, 0, 0, 0, nz, 1, &q, bq);
                if (e == hipSuccess) e = lin(cn, d_h, nz, d_h, 0, nullptr, 0, 0, 0, nz, 2, kv, bkv);
            }
            // causal attention of every group at once: (group, batch row) is the batch index
            if (e == hipSuccess) {
                ReplayProblem rp;
                rp.q = Q; rp.k = K; rp.v = V; rp.idx = nullptr; rp.o = att; rp.vt = vt;
                rp.B = s->B * G; rp.T = s->T; rp.H_q = nh; rp.H_kv = nh; rp.D = d_h / nh; rp.S = 0;
                rp.kv_layout = MOT_LAYOUT_BTHD;
                e = launch_replay_attention(rp, stream);
            }
            // h~ = Wo att + bo + h_{r-1}
            if (e == hipSuccess) {
                LinearPart q = part(C + off.wo, d_h, h1);
                const size_t bo[1] = {C + off.bo};
                e = lin(att, d_h, nz, d_h, 0, hp, ld_hp, hp_gs, 0, nz, 1, &q, bo);
            }
            // f1 = GELU(W_f1 LN_F(h~) + b_f1)
            if (e == hipSuccess) {
                const size_t bo[1] = {C + off.b_f1};
                if (fuse_h) {
                    LinearPart q = part(C + off.w_f1, d_ff, f1, C + off.ln_f_g, C + off.ln_f_b);
                    e = lin(h1, d_h, nz, d_h, 1, nullptr, 0, 0, 0, n * d_ff, 1, &q, bo);
                } else {
                    e = ln(h1, d_h, nz, d_h, C + off.ln_f_g, C + off.ln_f_b, fn, nz, 0, 0, nullptr);
                    LinearPart q = part(C + off.w_f1, d_ff, f1);
                    if (e == hipSuccess) e = lin(fn, d_h, nz, d_h, 1, nullptr, 0, 0, 0, n * d_ff, 1, &q, bo);
                }
            }
            // h_r = W_f2 f1 + b_f2 + h~, into slot r of F
            if (e == hipSuccess) {
                LinearPart q = part(C + off.w_f2, d_h, F + (size_t)r * d_h);
                const size_t bo[1] = {C + off.b_f2};
                e = lin(f1, d_ff, n * d_ff, d_ff, 0, h1, d_h, nz, ldF, nF, 1, &q, bo);
            }
        }
        // mixture += gate_m * GELU(W_out LN_out(F) + b_out): one launch per
        // expert (in order) and slot over the batch's units, slot r of unit u
        // into its target layer w N + r
        const uint16_t* out_in = F;
        if (e == hipSuccess && !fuse_out) {
            e = ln(F, ldF, nF, N * d_h, off.ln_out_g, off.ln_out_b, on, nF, 0, 0, nullptr);
            out_in = on;
        }
        for (int m = 0; m < E && e == hipSuccess; ++m) {
            for (int r = 0; r < N && e == hipSuccess; ++r) {
                LinearProblem lp;
                memset(&lp, 0, sizeof lp);
                const uint16_t* Pm = Pb + (size_t)m * P;
                lp.in = out_in + (size_t)m * nF; lp.ld_in = ldF; lp.in_gs = (size_t)E * nF;
                lp.w_gs = (size_t)E * P; lp.groups = nb;
                lp.nparts = 1;
                lp.part[0].W = Pm + off.w_out + (size_t)r * d_out * N * d_h;
                lp.part[0].bias = Pm + off.b_out + (size_t)r * d_out;
                lp.part[0].ln_g = fuse_out ? Pm + off.ln_out_g : nullptr;
                lp.part[0].ln_b = fuse_out ? Pm + off.ln_out_b : nullptr;
                lp.part[0].N = d_out;
                for (int u = 0; u < nb; ++u) {
                    const uint32_t code = ut.code[u0 + u];
                    lp.out_tab[u] = reinterpret_cast<uint16_t*>(unit_x(code) ? dst_v : dst_k) +
                                    (size_t)(unit_j(code) * N + r) * n * d_out;
                }
                lp.part[0].out = lp.out_tab[0];
                lp.mix_acc = mix + (size_t)r * n * d_out; lp.mix_gs = (size_t)N * n * d_out;
                lp.gates = p.gates + (size_t)unit_gslot(ut.code[u0]) * p.n_tok_pad * E;
                lp.gate_gs = (size_t)p.n_tok_pad * E; lp.gate_ld = E; lp.expert = m;
                lp.n = n_i; lp.K = N * d_h; lp.gelu = 1; lp.mix = 1;
                lp.first = m == 0; lp.last = m == E - 1;
                e = launch_linear(lp, stream);
            }
        }
        u0 += nb;
    }
    if (e != hipSuccess) return fail(MOT_ERR_HIP, "launch: %s", hipGetErrorString(e));
    return MOT_OK;
}

}  // extern "C"
