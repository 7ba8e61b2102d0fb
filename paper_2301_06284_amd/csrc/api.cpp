// api.cpp -- C ABI entry points of librgnn: argument checks, plan selection by
// modelled HBM bytes, workspace carving and the kernel sequence of each layer.
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "rgnn_internal.h"

namespace rgnn {

// ------------------------------------------------------------------ profiling
namespace {
struct ProfRec {
    std::string name;
    hipEvent_t a, b;
};
std::mutex g_prof_mu;
bool g_prof_on = false;
std::vector<ProfRec> g_prof;
}  // namespace

LaunchScope::LaunchScope(const char *n, hipStream_t s) : name(n), stream(s), slot(-1)
{
    if (!g_prof_on) return;
    std::lock_guard<std::mutex> lk(g_prof_mu);
    ProfRec r{n, nullptr, nullptr};
    if (hipEventCreate(&r.a) != hipSuccess || hipEventCreate(&r.b) != hipSuccess) return;
    if (hipEventRecord(r.a, s) != hipSuccess) return;
    g_prof.push_back(r);
    slot = (int)g_prof.size() - 1;
}

LaunchScope::~LaunchScope()
{
    if (slot < 0) return;
    std::lock_guard<std::mutex> lk(g_prof_mu);
    if (slot < (int)g_prof.size()) (void)hipEventRecord(g_prof[slot].b, stream);
}

// ------------------------------------------------------------------ helpers
namespace {

inline size_t pad256(size_t b) { return (b + 255) & ~size_t(255); }

struct Carver {
    char *base;
    size_t off = 0;
    explicit Carver(void *b) : base((char *)b) {}
    template <class T>
    T *take(size_t n)
    {
        T *p = base ? (T *)(base + off) : nullptr;
        off += pad256(n * sizeof(T));
        return p;
    }
};

rgnn_status check_graph(const rgnn_graph *g)
{
    if (!g) return fail(RGNN_EINVAL, "graph is NULL");
    if (g->device < 0) return fail(RGNN_EINVAL, "graph was created host-only");
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev != g->device)
        return fail(RGNN_EINVAL, "graph lives on device " + std::to_string(g->device) +
                                     " but the current device is " + std::to_string(dev));
    return RGNN_OK;
}

// feature widths of the RGCN / RGAT layers: 64 and 128 in any combination,
// 32 only as d_in = d_out = 32
bool dims_ok(int d_in, int d_out)
{
    if (d_in == 32 || d_out == 32) return d_in == d_out;
    return (d_in == 64 || d_in == 128) && (d_out == 64 || d_out == 128);
}

// ---- modelled HBM bytes of the two plans (gathered rows counted per edge) ----
void plan_bytes(const rgnn_graph *g, int layer, int d_in, int d_out, int H, double *tf, double *af)
{
    const double E = (double)g->E, N = (double)g->N, U = (double)g->U_src, V = (double)g->V;
    const double bi = 4.0 * d_in, bo = 4.0 * d_out;
    if (layer == RGNN_LAYER_RGCN) {
        *tf = U * (bi + bo) + E * (4 + bo) + V * 12 + N * bo;
        // fused: gathered rows + segment table + T written and read back
        *af = E * (4 + bi) + V * (16 + 2 * bo) + N * bo;
    } else {
        *tf = U * (bi + bo) + E * (4 + bo) + V * (12 + 4 * H) + N * (bi + bo + 8 * H);
        // destination terms (h_v once per destination), fused traversal (rows,
        // segment table, destination term, T, (max, sum)), statistics, reduce
        *af = E * (4 + bi) + N * (bi + 8 + bo) + V * (48 + 2 * bo);
    }
}

int resolve_plan(const rgnn_graph *g, int layer, int d_in, int d_out, int H, int plan)
{
    if (plan != RGNN_PLAN_AUTO) return plan;
    if (layer == RGNN_LAYER_RGAT && H != 1) return RGNN_PLAN_TRANSFORM_FIRST;
    double tf, af;
    plan_bytes(g, layer, d_in, d_out, H, &tf, &af);
    return af < tf ? RGNN_PLAN_AGGREGATE_FIRST : RGNN_PLAN_TRANSFORM_FIRST;
}

// ---- workspace layouts ----
struct RgcnWs { float *M, *partial, *T; };
size_t rgcn_layout(const rgnn_graph *g, int d_in, int d_out, int plan, void *base, RgcnWs *w)
{
    Carver c(base);
    RgcnWs x{};
    if (plan == RGNN_PLAN_TRANSFORM_FIRST) {
        x.M = c.take<float>((size_t)g->U_src * d_out);
        x.partial = c.take<float>((size_t)g->n_slots * (2 + d_out));
    } else {
        x.T = c.take<float>((size_t)g->V * d_out);
    }
    if (w) *w = x;
    return c.off;
}

struct RgatWs { float *M, *wsp, *wtp, *vatt, *partial, *vstat, *vscale, *T; };
size_t rgat_layout(const rgnn_graph *g, int d_in, int d_out, int H, int plan, void *base,
                   RgatWs *w)
{
    Carver c(base);
    RgatWs x{};
    x.wsp = c.take<float>((size_t)g->R * H * d_in);
    x.wtp = c.take<float>((size_t)g->R * H * d_in);
    x.vatt = c.take<float>((size_t)g->V * H);
    if (plan == RGNN_PLAN_TRANSFORM_FIRST || plan == RGNN_PLAN_TRANSFORM_FIRST_UNREORDERED ||
        plan == RGNN_PLAN_TRANSFORM_FIRST_ATTMSG) {
        const int ldm = plan == RGNN_PLAN_TRANSFORM_FIRST_ATTMSG ? att_row_ld(d_out, H) : d_out;
        x.M = c.take<float>((size_t)g->U_src * ldm);
        x.partial = c.take<float>((size_t)g->n_slots * (2 * H + d_out));
        if (plan == RGNN_PLAN_TRANSFORM_FIRST_UNREORDERED)   // h_v W_r per segment
            x.T = c.take<float>((size_t)g->V * d_out);
    } else {
        x.vstat = c.take<float>((size_t)g->V * 2);
        x.vscale = c.take<float>((size_t)g->V);
        x.T = c.take<float>((size_t)g->V * d_out);
    }
    if (w) *w = x;
    return c.off;
}

// RGAT backward workspace: the one-head backward (input space) or the
// several-head backward (message space, backward_heads.hip).
size_t rgat_bwd_layout(const rgnn_graph *g, int d_in, int d_out, int H)
{
    size_t need = 0;
    if (H > 1)
        rgat_backward_heads_impl(g, nullptr, nullptr, nullptr, nullptr, d_out, H, 0.f, 0, nullptr, nullptr,
                                 nullptr, nullptr, nullptr, nullptr, nullptr, 0, nullptr, &need);
    else
        rgat_backward_impl(g, nullptr, nullptr, nullptr, nullptr, d_in, d_out, 0.f, 0, nullptr, nullptr,
                           nullptr, nullptr, nullptr, nullptr, nullptr, 0, nullptr, &need);
    return need;
}

// Aggregate-first with several heads: the one-head aggregate-first workspace
// plus the masked weights, one head's output and its softmax statistics (per
// destination or per (dst, rel) segment).
struct HeadsAfWs { float *Wm, *wsm, *wdm, *outk, *sk; void *inner; size_t inner_bytes; };
size_t rgat_heads_af_layout(const rgnn_graph *g, int d, int H, void *base, HeadsAfWs *w)
{
    const size_t inner = rgat_layout(g, d, d, 1, RGNN_PLAN_AGGREGATE_FIRST, nullptr, nullptr);
    Carver c(base);
    HeadsAfWs x{};
    x.inner = c.take<char>(inner);
    x.inner_bytes = inner;
    (void)H;
    x.Wm = c.take<float>((size_t)g->R * d * d);
    x.wsm = c.take<float>((size_t)g->R * d);
    x.wdm = c.take<float>((size_t)g->R * d);
    x.outk = c.take<float>((size_t)g->N * d);
    x.sk = c.take<float>((size_t)std::max<int64_t>(std::max(g->U_dst, g->N), 1) * 2);
    if (w) *w = x;
    return c.off;
}

struct HgtWs { float *KV, *Q, *QP, *Wqp, *agg, *partial; };
size_t hgt_layout(const rgnn_graph *g, int d, int H, void *base, HgtWs *w)
{
    Carver c(base);
    HgtWs x{};
    x.KV = c.take<float>((size_t)g->N * 2 * d);
    x.Q = c.take<float>((size_t)g->N * d);
    x.QP = c.take<float>((size_t)g->V * d);
    x.Wqp = c.take<float>((size_t)g->R * d * d);
    x.agg = c.take<float>((size_t)g->N * d);
    x.partial = c.take<float>((size_t)g->n_slots * (2 * H + d));
    if (w) *w = x;
    return c.off;
}

size_t segment_gemm_layout(int64_t M, int32_t T, void *base, Tile **tiles, int64_t *ntiles)
{
    // upper bound on the tile count: every type may add one partial tile
    const int64_t n = (M + kGemmTileRows - 1) / kGemmTileRows + T;
    Carver c(base);
    Tile *t = c.take<Tile>((size_t)std::max<int64_t>(n, 1));
    if (tiles) *tiles = t;
    if (ntiles) *ntiles = n;
    return c.off;
}

}  // namespace
}  // namespace rgnn

using namespace rgnn;

extern "C" rgnn_status rgnn_profile_enable(int32_t on)
{
    std::lock_guard<std::mutex> lk(g_prof_mu);
    g_prof_on = on != 0;
    return RGNN_OK;
}

extern "C" rgnn_status rgnn_profile_reset(void)
{
    std::lock_guard<std::mutex> lk(g_prof_mu);
    for (auto &r : g_prof) {
        (void)hipEventSynchronize(r.b);
        (void)hipEventDestroy(r.a);
        (void)hipEventDestroy(r.b);
    }
    g_prof.clear();
    return RGNN_OK;
}

namespace {
struct ProfAgg { std::string name; int64_t n; double ms; };
std::vector<ProfAgg> prof_aggregate(rgnn_status *st)
{
    std::vector<ProfAgg> out;
    *st = RGNN_OK;
    for (auto &r : g_prof) {
        hipError_t e = hipEventSynchronize(r.b);
        float ms = 0.f;
        if (e == hipSuccess) e = hipEventElapsedTime(&ms, r.a, r.b);
        if (e != hipSuccess) { *st = hip_fail(e, "profiling event"); return out; }
        auto it = std::find_if(out.begin(), out.end(), [&](const ProfAgg &p) { return p.name == r.name; });
        if (it == out.end()) out.push_back(ProfAgg{r.name, 1, ms});
        else { it->n++; it->ms += ms; }
    }
    return out;
}
}  // namespace

extern "C" rgnn_status rgnn_profile_count(int32_t *count)
{
    if (!count) return fail(RGNN_EINVAL, "count is NULL");
    std::lock_guard<std::mutex> lk(g_prof_mu);
    rgnn_status st;
    auto agg = prof_aggregate(&st);
    *count = (int32_t)agg.size();
    return st;
}

extern "C" rgnn_status rgnn_profile_read(int32_t i, char *name, size_t name_bytes,
                                         int64_t *launches, double *total_ms)
{
    std::lock_guard<std::mutex> lk(g_prof_mu);
    rgnn_status st;
    auto agg = prof_aggregate(&st);
    if (st != RGNN_OK) return st;
    if (i < 0 || i >= (int)agg.size()) return fail(RGNN_EINVAL, "profile index out of range");
    if (name && name_bytes) {
        std::snprintf(name, name_bytes, "%s", agg[i].name.c_str());
    }
    if (launches) *launches = agg[i].n;
    if (total_ms) *total_ms = agg[i].ms;
    return RGNN_OK;
}

// ------------------------------------------------------------------ planning
extern "C" rgnn_status rgnn_select_plan(const rgnn_graph_t *g, int32_t layer, int32_t d_in,
                                        int32_t d_out, int32_t heads, int32_t *plan,
                                        double *bytes_tf, double *bytes_af)
{
    if (!g) return fail(RGNN_EINVAL, "graph is NULL");
    if (layer != RGNN_LAYER_RGCN && layer != RGNN_LAYER_RGAT)
        return fail(RGNN_EINVAL, "plans exist for RGCN and RGAT only");
    if (heads <= 0) return fail(RGNN_EINVAL, "heads must be positive");
    double tf, af;
    plan_bytes(g, layer, d_in, d_out, heads, &tf, &af);
    if (bytes_tf) *bytes_tf = tf;
    if (bytes_af) *bytes_af = af;
    if (plan) *plan = resolve_plan(g, layer, d_in, d_out, heads, RGNN_PLAN_AUTO);
    return RGNN_OK;
}

extern "C" rgnn_status rgnn_workspace_size(const rgnn_graph_t *g, int32_t layer, int32_t d_in,
                                           int32_t d_out, int32_t heads, int32_t plan,
                                           size_t *bytes)
{
    if (!g || !bytes) return fail(RGNN_EINVAL, "NULL argument");
    if (heads <= 0) return fail(RGNN_EINVAL, "heads must be positive");
    if (plan < 0 || plan > 4) return fail(RGNN_EINVAL, "unknown plan");
    if ((plan == RGNN_PLAN_TRANSFORM_FIRST_UNREORDERED || plan == RGNN_PLAN_TRANSFORM_FIRST_ATTMSG) &&
        layer != RGNN_LAYER_RGAT)
        return fail(RGNN_EINVAL, "the unreordered and attention+message transform-first plans are RGAT plans");
    switch (layer) {
    case RGNN_LAYER_RGCN:
        *bytes = rgcn_layout(g, d_in, d_out, resolve_plan(g, layer, d_in, d_out, 1, plan), nullptr, nullptr);
        return RGNN_OK;
    case RGNN_LAYER_RGAT:
        if (plan == RGNN_PLAN_AGGREGATE_FIRST && heads > 1)   // per-(dst, rel) softmax, several heads
            *bytes = rgat_heads_af_layout(g, d_out, heads, nullptr, nullptr);
        else
            *bytes = rgat_layout(g, d_in, d_out, heads, resolve_plan(g, layer, d_in, d_out, heads, plan),
                                 nullptr, nullptr);
        return RGNN_OK;
    case RGNN_LAYER_HGT:
        *bytes = hgt_layout(g, d_out, heads, nullptr, nullptr);
        return RGNN_OK;
    case RGNN_LAYER_RGAT_BACKWARD:
        *bytes = rgat_bwd_layout(g, d_in, d_out, heads);
        return RGNN_OK;
    case RGNN_LAYER_HGT_BACKWARD: {
        size_t need = 0;
        hgt_backward_impl(g, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, d_out,
                          heads, 0.f, 0, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                          nullptr, nullptr, nullptr, 0, nullptr, &need);
        *bytes = need;
        return RGNN_OK;
    }
    case RGNN_LAYER_RGCN_BACKWARD: {
        size_t need = 0;
        rgcn_backward_impl(g, nullptr, nullptr, nullptr, d_in, d_out, 0, nullptr, nullptr, nullptr,
                           nullptr, nullptr, nullptr, 0, nullptr, &need);
        *bytes = need;
        return RGNN_OK;
    }
    default:
        return fail(RGNN_EINVAL, "unknown layer");
    }
}

// ------------------------------------------------------------------ RGCN
extern "C" rgnn_status rgcn_forward(const rgnn_graph_t *g, const float *h, const float *W,
                                    const float *W0, int32_t d_in, int32_t d_out, int32_t flags,
                                    int32_t plan, float *out, void *ws, size_t ws_bytes,
                                    void *stream)
{
    rgnn_status st = check_graph(g);
    if (st != RGNN_OK) return st;
    if (!h || !W || !out) return fail(RGNN_EINVAL, "NULL tensor pointer");
    if (!dims_ok(d_in, d_out))
        return fail(RGNN_EUNSUPPORTED, "d_in, d_out must be 64 or 128, or both 32");
    if (flags & ~RGNN_FLAG_RELU) return fail(RGNN_EINVAL, "unknown RGCN flag");
    if (plan < 0 || plan > 2) return fail(RGNN_EINVAL, "unknown plan");
    plan = resolve_plan(g, RGNN_LAYER_RGCN, d_in, d_out, 1, plan);
    const size_t need = rgcn_layout(g, d_in, d_out, plan, nullptr, nullptr);
    if (need && (!ws || ws_bytes < need))
        return fail(RGNN_EINVAL, "workspace too small: need " + std::to_string(need) + " bytes");
    RgcnWs w;
    rgcn_layout(g, d_in, d_out, plan, ws, &w);
    hipStream_t s = (hipStream_t)stream;
    const int relu = (flags & RGNN_FLAG_RELU) ? 1 : 0;
    const int relu_in_traversal = relu && !W0;
    if (plan == RGNN_PLAN_TRANSFORM_FIRST) {
        // compact materialization: one message row per unique (src, rel) pair
        GemmArgs ga;
        ga.split_bf16 = 1;
        ga.X = h; ga.ldx = d_in; ga.gather = g->dev.uniq_src;
        ga.W[0] = W; ga.K = d_in; ga.Nc = d_out;
        ga.tiles = g->dev.tiles_pairs; ga.ntiles = g->n_tiles_pairs;
        ga.Y = w.M; ga.ldy = d_out;
        if ((st = launch_typed_gemm(ga, s)) != RGNN_OK) return st;
        TravArgs ta;
        ta.g = g; ta.M = w.M; ta.d = d_out; ta.out = out; ta.partial = w.partial;
        ta.relu = relu_in_traversal;
        if ((st = launch_rgcn_traverse_tf(ta, s)) != RGNN_OK) return st;
        if ((st = launch_merge_partials(g, d_out, 1, 0, w.partial, out, nullptr, ta.relu, s)) != RGNN_OK)
            return st;
    } else {
        // fused gather + per-(dst, rel) mean + W_r per virtual segment, then
        // the segments of each destination summed
        // (a destination with a single virtual segment gets its row from the fused kernel)
        FusedArgs fa;
        fa.g = g; fa.h = h; fa.W = W; fa.d_in = d_in; fa.d_out = d_out; fa.T = w.T;
        fa.out = out; fa.relu = relu_in_traversal;
        if ((st = launch_af_fused(fa, s)) != RGNN_OK) return st;
        if ((st = launch_vseg_reduce(g, w.T, nullptr, d_out, out, 0, relu_in_traversal, s, 0, 1)) != RGNN_OK)
            return st;
    }
    if (W0) {   // virtual self-loop h_v W0, accumulated into out (then the activation)
        GemmArgs ga;
        ga.split_bf16 = 1;
        ga.X = h; ga.ldx = d_in; ga.W[0] = W0; ga.K = d_in; ga.Nc = d_out;
        ga.tiles = g->dev.tiles_all; ga.ntiles = g->n_tiles_all;
        ga.Y = out; ga.ldy = d_out;
        ga.ep.accumulate = 1; ga.ep.relu = relu;
        if ((st = launch_typed_gemm(ga, s)) != RGNN_OK) return st;
    }
    return RGNN_OK;
}

// ------------------------------------------------------------------ RGAT
rgnn_status rgat_forward_impl(const rgnn_graph *g, const float *h, const float *W, const float *w_src,
                              const float *w_dst, int d_in, int d_out, int heads, float neg_slope, bool per_seg,
                              int plan, float *out, float *saved, void *ws, size_t ws_bytes, hipStream_t s);

extern "C" rgnn_status rgat_forward(const rgnn_graph_t *g, const float *h, const float *W,
                                    const float *w_src, const float *w_dst, int32_t d_in,
                                    int32_t d_out, int32_t heads, float neg_slope,
                                    int32_t softmax_scope, int32_t plan, float *out, float *saved,
                                    void *ws, size_t ws_bytes, void *stream)
{
    rgnn_status st = check_graph(g);
    if (st != RGNN_OK) return st;
    if (!h || !W || !w_src || !w_dst || !out) return fail(RGNN_EINVAL, "NULL tensor pointer");
    if (!dims_ok(d_in, d_out))
        return fail(RGNN_EUNSUPPORTED, "d_in, d_out must be 64 or 128, or both 32");
    if (heads <= 0 || d_out % heads) return fail(RGNN_EINVAL, "heads must divide d_out");
    if ((d_out / heads) % 16) return fail(RGNN_EUNSUPPORTED, "d_out / heads must be a multiple of 16");
    if (softmax_scope != RGNN_SOFTMAX_PER_DST && softmax_scope != RGNN_SOFTMAX_PER_DST_REL)
        return fail(RGNN_EINVAL, "unknown softmax scope");
    if (plan < 0 || plan > 4) return fail(RGNN_EINVAL, "unknown plan");
    if (!std::isfinite(neg_slope)) return fail(RGNN_EINVAL, "neg_slope must be finite");
    const bool per_seg = softmax_scope == RGNN_SOFTMAX_PER_DST_REL;
    if (per_seg) {   // normalised per (dst, rel) segment: the aggregate-first plan
        if (plan == RGNN_PLAN_TRANSFORM_FIRST || plan == RGNN_PLAN_TRANSFORM_FIRST_UNREORDERED ||
            plan == RGNN_PLAN_TRANSFORM_FIRST_ATTMSG)
            return fail(RGNN_EUNSUPPORTED, "softmax per (destination, relation) runs aggregate-first");
        plan = RGNN_PLAN_AGGREGATE_FIRST;
    }
    plan = resolve_plan(g, RGNN_LAYER_RGAT, d_in, d_out, heads, plan);
    if (plan != RGNN_PLAN_AGGREGATE_FIRST && d_in != d_out)
        return fail(RGNN_EUNSUPPORTED, "RGAT needs d_in == d_out");
    if (plan == RGNN_PLAN_AGGREGATE_FIRST && d_in != d_out)
        return fail(RGNN_EUNSUPPORTED, "aggregate-first RGAT needs d_in == d_out");
    hipStream_t s = (hipStream_t)stream;
    if (heads == 1 || plan != RGNN_PLAN_AGGREGATE_FIRST)
        return rgat_forward_impl(g, h, W, w_src, w_dst, d_in, d_out, heads, neg_slope, per_seg, plan, out,
                                 saved, ws, ws_bytes, s);
    // aggregate-first with several heads: one masked one-head aggregate-first
    // pass per head (head k reads only its columns of W_r, w_src[r] and
    // w_dst[r], so the masked pass computes exactly head k's logits, softmax
    // and output columns, and zeros elsewhere); outputs summed, statistics
    // interleaved into saved [N or U_dst, heads, 2]
    const size_t need = rgat_heads_af_layout(g, d_out, heads, nullptr, nullptr);
    if (!ws || ws_bytes < need)
        return fail(RGNN_EINVAL, "workspace too small: need " + std::to_string(need) + " bytes");
    HeadsAfWs w;
    rgat_heads_af_layout(g, d_out, heads, ws, &w);
    const int64_t R = g->R, N = g->N, dk = d_out / heads;
    for (int k = 0; k < heads; ++k) {
        const int c0 = (int)(k * dk), c1 = (int)((k + 1) * dk);
        if ((st = launch_mask_cols(W, w.Wm, R * d_in, d_out, c0, c1, s)) != RGNN_OK) return st;
        if ((st = launch_mask_cols(w_src, w.wsm, R, d_out, c0, c1, s)) != RGNN_OK) return st;
        if ((st = launch_mask_cols(w_dst, w.wdm, R, d_out, c0, c1, s)) != RGNN_OK) return st;
        float *ok = k ? w.outk : out;
        if ((st = rgat_forward_impl(g, h, w.Wm, w.wsm, w.wdm, d_in, d_out, 1, neg_slope, per_seg,
                                    RGNN_PLAN_AGGREGATE_FIRST, ok, saved ? w.sk : nullptr, w.inner,
                                    w.inner_bytes, s)) != RGNN_OK)
            return st;
        if (k && (st = launch_add(out, out, w.outk, N * d_out, s)) != RGNN_OK) return st;
        if (saved && (st = launch_head_stats_scatter(w.sk, saved, per_seg ? g->U_dst : N, heads, k, s)) != RGNN_OK)
            return st;
    }
    return RGNN_OK;
}

rgnn_status rgat_forward_impl(const rgnn_graph *g, const float *h, const float *W, const float *w_src,
                              const float *w_dst, int d_in, int d_out, int heads, float neg_slope, bool per_seg,
                              int plan, float *out, float *saved, void *ws, size_t ws_bytes, hipStream_t s)
{
    rgnn_status st;
    const size_t need = rgat_layout(g, d_in, d_out, heads, plan, nullptr, nullptr);
    if (!ws || ws_bytes < need)
        return fail(RGNN_EINVAL, "workspace too small: need " + std::to_string(need) + " bytes");
    RgatWs w;
    rgat_layout(g, d_in, d_out, heads, plan, ws, &w);
    // linear operator reordering: W_r w_dst[r] (and W_r w_src[r]) once per relation,
    // then the destination term h_v . (W_r w_dst[r]) once per (dst, rel) segment
    // (aggregate-first also needs W_r w_src[r]: both in one launch)
    const bool af = plan == RGNN_PLAN_AGGREGATE_FIRST;
    if (plan == RGNN_PLAN_TRANSFORM_FIRST_UNREORDERED) {
        // without reordering: the segment's h_v W_r row is materialized and its
        // dot products with w_dst[r] taken in the GEMM epilogue
        GemmArgs gd;
        gd.split_bf16 = 1;
        gd.X = h; gd.ldx = d_in; gd.gather = g->dev.vsegdst_byrel;
        gd.W[0] = W; gd.K = d_in; gd.Nc = d_out;
        gd.tiles = g->dev.tiles_vsegs; gd.ntiles = g->n_tiles_vsegs;
        gd.Y = w.T; gd.ldy = d_out; gd.scatter = g->dev.vseg_byrel;
        gd.ep.dot_vec = w_dst; gd.ep.dot_out = w.vatt; gd.ep.dot_heads = heads;
        if ((st = launch_typed_gemm(gd, s)) != RGNN_OK) return st;
    } else {
        if ((st = launch_reorder_vec(W, g->R, d_in, d_out, heads, w_dst, w.wtp, af ? w_src : nullptr,
                                     af ? w.wsp : nullptr, s)) != RGNN_OK)
            return st;
        TravArgs ta;
        ta.g = g; ta.h = h; ta.wtp = w.wtp; ta.heads = heads; ta.d = d_in; ta.vatt = w.vatt;
        if ((st = launch_seg_attn(ta, s)) != RGNN_OK) return st;
    }
    if (plan != RGNN_PLAN_AGGREGATE_FIRST) {
        const bool attmsg = plan == RGNN_PLAN_TRANSFORM_FIRST_ATTMSG;
        GemmArgs ga;
        ga.split_bf16 = 1;
        ga.X = h; ga.ldx = d_in; ga.gather = g->dev.uniq_src;
        ga.W[0] = W; ga.K = d_in; ga.Nc = d_out;
        ga.tiles = g->dev.tiles_pairs; ga.ntiles = g->n_tiles_pairs;
        ga.Y = w.M; ga.ldy = attmsg ? att_row_ld(d_out, heads) : d_out;
        if (attmsg) {   // the source terms m . w_src[r] per head, written after each row's message
            ga.ep.dot_vec = w_src; ga.ep.dot_out = w.M + d_out; ga.ep.dot_heads = heads; ga.ep.dot_ld = ga.ldy;
        }
        if ((st = launch_typed_gemm(ga, s)) != RGNN_OK) return st;
        // the per-head source terms are formed in the traversal from the gathered
        // message row itself (no per-pair term is materialized), or read from
        // the attention+message row
        TravArgs ta;
        ta.g = g; ta.h = h; ta.M = w.M; ta.wtp = w.wtp; ta.vatt = w.vatt; ta.wsp = w_src;
        ta.att_in_row = attmsg;
        ta.slope = neg_slope; ta.heads = heads; ta.d = d_out;
        ta.out = out; ta.saved = saved; ta.partial = w.partial;
        if ((st = launch_rgat_traverse_tf(ta, s)) != RGNN_OK) return st;
        if ((st = launch_merge_partials(g, d_out, heads, 1, w.partial, out, saved, 0, s)) != RGNN_OK)
            return st;
    } else {
        // fused gather + per-segment online softmax + W_r per virtual segment;
        // the softmax is finished per destination (or per segment) when the
        // segments are summed
        FusedArgs fa;
        fa.g = g; fa.h = h; fa.W = W; fa.wsp = w.wsp; fa.vatt = w.vatt; fa.slope = neg_slope;
        fa.d_in = d_in; fa.d_out = d_out; fa.softmax = 1; fa.T = w.T; fa.vstat = w.vstat;
        if (!per_seg) {   // destinations with one segment are finished in the fused kernel
            fa.out = out; fa.saved = saved;
        }
        if ((st = launch_af_fused(fa, s)) != RGNN_OK) return st;
        if (per_seg) {
            TravArgs ta;
            ta.g = g; ta.vstat = w.vstat; ta.vscale = w.vscale; ta.saved = saved;   // [U_dst, 2]
            if ((st = launch_seg_softmax_scale(ta, s)) != RGNN_OK) return st;
            if ((st = launch_vseg_reduce(g, w.T, w.vscale, d_out, out, 0, 0, s)) != RGNN_OK) return st;
        } else if ((st = launch_softmax_reduce(g, w.vstat, w.T, d_out, out, saved, w.vscale, 1, s)) != RGNN_OK) {
            return st;
        }
    }
    return RGNN_OK;
}

// ------------------------------------------------------------------ HGT
extern "C" rgnn_status hgt_forward(const rgnn_graph_t *g, const float *h, const float *Wk,
                                   const float *Wq, const float *Wv, const float *Wa,
                                   const float *Watt, const float *Wmsg, const float *mu,
                                   int32_t d, int32_t heads, float att_scale, int32_t flags,
                                   float *out, float *saved, void *ws, size_t ws_bytes, void *stream)
{
    rgnn_status st = check_graph(g);
    if (st != RGNN_OK) return st;
    if (!h || !Wk || !Wq || !Wv || !Watt || !Wmsg || !mu || !out)
        return fail(RGNN_EINVAL, "NULL tensor pointer");
    if ((flags & RGNN_FLAG_A_LINEAR) && !Wa) return fail(RGNN_EINVAL, "Wa is NULL");
    if (flags & ~(RGNN_FLAG_RESIDUAL | RGNN_FLAG_A_LINEAR)) return fail(RGNN_EINVAL, "unknown HGT flag");
    if (d != 32 && d != 64 && d != 128) return fail(RGNN_EUNSUPPORTED, "HGT supports d = 32, 64 or 128");
    if (!(heads == 1 || heads == 2 || heads == 4 || heads == 8) || d / heads < 16)
        return fail(RGNN_EUNSUPPORTED, "HGT heads must be 1, 2, 4 or 8 with d / heads >= 16");
    if (!std::isfinite(att_scale)) return fail(RGNN_EINVAL, "att_scale must be finite");
    const size_t need = hgt_layout(g, d, heads, nullptr, nullptr);
    if (!ws || ws_bytes < need)
        return fail(RGNN_EINVAL, "workspace too small: need " + std::to_string(need) + " bytes");
    HgtWs w;
    hgt_layout(g, d, heads, ws, &w);
    hipStream_t s = (hipStream_t)stream;
    // The segment queries QP = Q_t Wqp[r] need Q only through that product.
    // When every relation's destinations share one node type t(r) (typed
    // relations), Wq[t(r)] folds into the per-relation weight, QP = h_t
    // (Wq[t(r)] Wqp[r]), and Q is never formed; otherwise (and when the
    // traversal forms the queries itself from Q at d = 128) Q is projected
    // with K and V.
    const bool fused_query = d == 128 && hgt_fused_query_fits(g->R, d, heads);
    const bool fold_q = !fused_query && g->rel_dst_typed;
    // K | V (| Q) of every node by node-typed GEMMs (segment MM over node
    // types): one GEMM with the weights side by side at d = 64, one per
    // projection otherwise (a 3d-wide weight tile would not fit LDS at 128)
    GemmArgs ga;
    ga.split_bf16 = 1;
    ga.X = h; ga.ldx = d; ga.gather = g->dev.ntype_perm; ga.scatter = g->dev.ntype_perm;
    ga.K = d;
    ga.tiles = g->dev.tiles_nodes; ga.ntiles = g->n_tiles_nodes;
    if (d == 64 && fold_q) {
        ga.W[0] = Wk; ga.W[1] = Wv; ga.nparts = 2;
        ga.Nc = 2 * d;
        ga.Y = w.KV; ga.ldy = 2 * d;
        if ((st = launch_typed_gemm(ga, s)) != RGNN_OK) return st;
    } else if (d == 64) {
        ga.W[0] = Wk; ga.W[1] = Wv; ga.W[2] = Wq; ga.nparts = 3;
        ga.Nc = 3 * d;
        ga.Y = w.KV; ga.ldy = 2 * d;
        ga.ep.Y2 = w.Q; ga.ep.ldy2 = d; ga.ep.split = 2 * d;
        if ((st = launch_typed_gemm(ga, s)) != RGNN_OK) return st;
    } else {
        ga.Nc = d;
        const float *Wp[3] = {Wk, Wv, Wq};
        float *Yp[3] = {w.KV, w.KV + d, w.Q};
        const int64_t ld[3] = {2 * d, 2 * d, d};
        for (int p = 0; p < (fold_q ? 2 : 3); ++p) {
            ga.W[0] = Wp[p]; ga.Y = Yp[p]; ga.ldy = ld[p];
            if ((st = launch_typed_gemm(ga, s)) != RGNN_OK) return st;
        }
    }
    HgtArgs ha;
    ha.g = g; ha.KV = w.KV; ha.Wmsg = Wmsg;
    if (fused_query) {
        // the traversal forms each segment's reordered query Q_t (mu scale Watt[r]^T)
        // from LDS-resident blocks at the segment's first edge.  Measured on the
        // 1.9M-node graph this wins only at d = 128 (the 128-wide segment-query
        // GEMM it replaces is MFMA-bound); at d = 32 and 64 the per-segment
        // vector-matrix product in the traversal costs more than the GEMM.
        ha.QP = nullptr; ha.Q = w.Q; ha.Watt = Watt; ha.mu = mu; ha.scale = att_scale;
    } else {
        // reordered query of every (dst, rel) segment: QP = Q_t Wqp[r], or
        // h_t (Wq[t(r)] Wqp[r]) with the projection folded in (segment MM over
        // relations; Wqp[r] alone is block-diagonal over the heads)
        if (fold_q) {
            if ((st = launch_hgt_qp_fold(Wq, Watt, mu, att_scale, g->dev.rel_dsttype, g->R, d, heads, w.Wqp, s)) !=
                RGNN_OK)
                return st;
        } else if ((st = launch_hgt_qp_weights(Watt, mu, att_scale, g->R, d, heads, w.Wqp, s)) != RGNN_OK) {
            return st;
        }
        GemmArgs gq;
        gq.split_bf16 = 1;
        gq.X = fold_q ? h : w.Q; gq.ldx = d; gq.gather = g->dev.vsegdst_byrel; gq.scatter = g->dev.vseg_byrel;
        gq.W[0] = w.Wqp; gq.K = d; gq.Nc = d;
        // tiles by destination range: each destination row is gathered by its
        // relations' tiles on one XCD, from L2 after the first
        gq.tiles = g->dev.tiles_vsegs_dst; gq.ntiles = g->n_tiles_vsegs_dst;
        gq.Y = w.QP; gq.ldy = d; gq.ep.diag_blocks = fold_q ? 1 : heads;
        if ((st = launch_typed_gemm(gq, s)) != RGNN_OK) return st;
        ha.QP = w.QP;
    }
    ha.heads = heads; ha.d = d; ha.agg = w.agg; ha.partial = w.partial; ha.saved = saved;
    if ((st = launch_hgt_traverse(ha, s)) != RGNN_OK) return st;
    if ((st = launch_merge_partials(g, d, heads, 1, w.partial, w.agg, saved, 0, s)) != RGNN_OK)
        return st;
    if (flags & RGNN_FLAG_A_LINEAR) {
        GemmArgs gb;
        gb.split_bf16 = 1;
        gb.X = w.agg; gb.ldx = d; gb.gather = g->dev.ntype_perm; gb.scatter = g->dev.ntype_perm;
        gb.W[0] = Wa; gb.K = d; gb.Nc = d;
        gb.tiles = g->dev.tiles_nodes; gb.ntiles = g->n_tiles_nodes;
        gb.Y = out; gb.ldy = d;
        if (flags & RGNN_FLAG_RESIDUAL) { gb.ep.residual = h; gb.ep.ld_res = d; }
        return launch_typed_gemm(gb, s);
    }
    if (flags & RGNN_FLAG_RESIDUAL) return launch_add(out, w.agg, h, g->N * d, s);
    hipError_t e = hipMemcpyAsync(out, w.agg, (size_t)g->N * d * sizeof(float),
                                  hipMemcpyDeviceToDevice, s);
    return e == hipSuccess ? RGNN_OK : hip_fail(e, "hipMemcpyAsync");
}

// ------------------------------------------------------------------ RGAT backward
extern "C" rgnn_status rgat_backward(const rgnn_graph_t *g, const float *h, const float *W,
                                     const float *w_src, const float *w_dst, int32_t d_in,
                                     int32_t d_out, int32_t heads, float neg_slope,
                                     int32_t softmax_scope, const float *saved,
                                     const float *grad_out, float *grad_h,
                                     float *grad_W, float *grad_w_src, float *grad_w_dst,
                                     void *ws, size_t ws_bytes, void *stream)
{
    rgnn_status st = check_graph(g);
    if (st != RGNN_OK) return st;
    if (!h || !W || !w_src || !w_dst || !grad_out || !grad_h || !grad_W || !grad_w_src || !grad_w_dst)
        return fail(RGNN_EINVAL, "NULL tensor pointer");
    if (!saved && (softmax_scope == RGNN_SOFTMAX_PER_DST_REL ? g->U_dst : g->N) > 0)
        return fail(RGNN_EINVAL, "saved is NULL");
    if (d_in != d_out || (d_in != 32 && d_in != 64 && d_in != 128))
        return fail(RGNN_EUNSUPPORTED, "RGAT backward supports d_in = d_out in {32, 64, 128}");
    if (heads <= 0 || d_out % heads || (d_out / heads) % 16)
        return fail(RGNN_EUNSUPPORTED, "RGAT backward heads must give d_out / heads a multiple of 16");
    if (softmax_scope != RGNN_SOFTMAX_PER_DST && softmax_scope != RGNN_SOFTMAX_PER_DST_REL)
        return fail(RGNN_EINVAL, "unknown softmax scope");
    const int per_seg = softmax_scope == RGNN_SOFTMAX_PER_DST_REL;
    if (!std::isfinite(neg_slope)) return fail(RGNN_EINVAL, "neg_slope must be finite");
    hipStream_t s = (hipStream_t)stream;
    const size_t need = rgat_bwd_layout(g, d_in, d_out, heads);
    if (!ws || ws_bytes < need)
        return fail(RGNN_EINVAL, "workspace too small: need " + std::to_string(need) + " bytes");
    if (heads == 1)
        return rgat_backward_impl(g, h, W, w_src, w_dst, d_in, d_out, neg_slope, per_seg, saved, grad_out, grad_h,
                                  grad_W, grad_w_src, grad_w_dst, ws, ws_bytes, s, nullptr);
    return rgat_backward_heads_impl(g, h, W, w_src, w_dst, d_out, heads, neg_slope, per_seg, saved, grad_out,
                                    grad_h, grad_W, grad_w_src, grad_w_dst, ws, ws_bytes, s, nullptr);
}

extern "C" rgnn_status hgt_backward(const rgnn_graph_t *g, const float *h, const float *Wk,
                                    const float *Wq, const float *Wv, const float *Wa,
                                    const float *Watt, const float *Wmsg, const float *mu, int32_t d,
                                    int32_t heads, float att_scale, int32_t flags, const float *grad_out,
                                    const float *saved, float *grad_h, float *grad_Wk, float *grad_Wq,
                                    float *grad_Wv,
                                    float *grad_Wa, float *grad_Watt, float *grad_Wmsg, float *grad_mu,
                                    void *ws, size_t ws_bytes, void *stream)
{
    rgnn_status st = check_graph(g);
    if (st != RGNN_OK) return st;
    if (!h || !Wk || !Wq || !Wv || !Watt || !Wmsg || !mu || !grad_out || !grad_h || !grad_Wk ||
        !grad_Wq || !grad_Wv || !grad_Watt || !grad_Wmsg || !grad_mu)
        return fail(RGNN_EINVAL, "NULL tensor pointer");
    if (flags & ~(RGNN_FLAG_RESIDUAL | RGNN_FLAG_A_LINEAR)) return fail(RGNN_EINVAL, "unknown HGT flag");
    if ((flags & RGNN_FLAG_A_LINEAR) && !Wa) return fail(RGNN_EINVAL, "Wa is NULL");
    if (d != 32 && d != 64 && d != 128) return fail(RGNN_EUNSUPPORTED, "HGT backward supports d = 32, 64 or 128");
    if (!(heads == 1 || heads == 2 || heads == 4 || heads == 8) || d / heads < 16)
        return fail(RGNN_EUNSUPPORTED, "HGT backward heads must be 1, 2, 4 or 8 with d / heads >= 16");
    if (!std::isfinite(att_scale)) return fail(RGNN_EINVAL, "att_scale must be finite");
    return hgt_backward_impl(g, h, Wk, Wq, Wv, Wa, Watt, Wmsg, mu, d, heads, att_scale, flags, grad_out,
                             saved, grad_h, grad_Wk, grad_Wq, grad_Wv, (flags & RGNN_FLAG_A_LINEAR) ? grad_Wa : nullptr,
                             grad_Watt, grad_Wmsg, grad_mu, ws, ws_bytes, (hipStream_t)stream, nullptr);
}

extern "C" rgnn_status rgcn_backward(const rgnn_graph_t *g, const float *h, const float *W,
                                     const float *W0, int32_t d_in, int32_t d_out, int32_t flags,
                                     const float *out, const float *grad_out, float *grad_h,
                                     float *grad_W, float *grad_W0, void *ws, size_t ws_bytes,
                                     void *stream)
{
    rgnn_status st = check_graph(g);
    if (st != RGNN_OK) return st;
    if (!h || !W || !grad_out || !grad_h || !grad_W) return fail(RGNN_EINVAL, "NULL tensor pointer");
    if (flags & ~RGNN_FLAG_RELU) return fail(RGNN_EINVAL, "unknown RGCN flag");
    if (d_in != d_out || (d_in != 32 && d_in != 64 && d_in != 128))
        return fail(RGNN_EUNSUPPORTED, "RGCN backward supports d_in = d_out in {32, 64, 128}");
    if ((flags & RGNN_FLAG_RELU) && !out)
        return fail(RGNN_EINVAL, "RGCN backward with ReLU needs the forward output");
    return rgcn_backward_impl(g, h, W, W0, d_in, d_out, flags, out, grad_out, grad_h, grad_W,
                              W0 ? grad_W0 : nullptr, ws, ws_bytes, (hipStream_t)stream, nullptr);
}

// ------------------------------------------------------------------ segment MM
extern "C" rgnn_status rgnn_segment_gemm_workspace_size(int64_t M, int32_t num_types, size_t *bytes)
{
    if (!bytes || M < 0 || num_types <= 0) return fail(RGNN_EINVAL, "bad argument");
    *bytes = segment_gemm_layout(M, num_types, nullptr, nullptr, nullptr);
    return RGNN_OK;
}

extern "C" rgnn_status rgnn_segment_gemm(const float *X, int64_t ldx, const int32_t *gather,
                                         const int64_t *type_ptr, int32_t num_types,
                                         const float *W, int32_t K, int32_t Nc, float *Y,
                                         int64_t ldy, const int32_t *scatter, void *ws,
                                         size_t ws_bytes, void *stream)
{
    if (!X || !W || !Y || !type_ptr) return fail(RGNN_EINVAL, "NULL pointer");
    if (num_types <= 0) return fail(RGNN_EINVAL, "num_types must be positive");
    if (!dims_ok(K, Nc)) return fail(RGNN_EUNSUPPORTED, "K and Nc must be 64 or 128, or both 32");
    if (ldx < K || ldy < Nc) return fail(RGNN_EINVAL, "leading dimension too small");
    if (type_ptr[0] != 0) return fail(RGNN_EINVAL, "type_ptr[0] must be 0");
    for (int t = 0; t < num_types; ++t)
        if (type_ptr[t + 1] < type_ptr[t]) return fail(RGNN_EINVAL, "type_ptr is not monotone");
    const int64_t M = type_ptr[num_types];
    if (M >= (int64_t(1) << 31) - 1) return fail(RGNN_ERANGE, "too many rows");
    const size_t need = segment_gemm_layout(M, num_types, nullptr, nullptr, nullptr);
    if (!ws || ws_bytes < need)
        return fail(RGNN_EINVAL, "workspace too small: need " + std::to_string(need) + " bytes");
    std::vector<int32_t> tp(num_types + 1);
    for (int t = 0; t <= num_types; ++t) tp[t] = (int32_t)type_ptr[t];
    std::vector<Tile> tiles;
    build_tiles(tp, kGemmTileRows, tiles);
    Tile *dt = nullptr;
    segment_gemm_layout(M, num_types, ws, &dt, nullptr);
    hipStream_t s = (hipStream_t)stream;
    if (tiles.empty()) return RGNN_OK;
    // The tile table is enqueued on the stream; the host vector must outlive the
    // copy, so this call waits for it (a few KB).
    hipError_t e = hipMemcpyAsync(dt, tiles.data(), tiles.size() * sizeof(Tile),
                                  hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(e, "tile table upload");
    GemmArgs ga;
    ga.split_bf16 = 1;
    ga.X = X; ga.ldx = ldx; ga.gather = gather; ga.W[0] = W; ga.K = K; ga.Nc = Nc;
    ga.tiles = dt; ga.ntiles = (int64_t)tiles.size();
    ga.Y = Y; ga.ldy = ldy; ga.scatter = scatter;
    return launch_typed_gemm(ga, s);
}
