/*
 * rgnn_oracle.c -- plain, slow, fp64 CPU reference of the RGCN, RGAT and HGT
 * layers and of their backward passes.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  It shares no code,
 * header or helper with the GPU library.
 *
 * Every function evaluates the defining equations edge by edge, in fp64, from
 * the same float32 inputs the GPU path reads:
 *   - no compact materialization, no linear-operator reordering, no fusion;
 *   - per-edge terms (h_u W_r, h_v W_r, HGT keys/values) are recomputed for
 *     every edge; node-level linears that the definitions state per node
 *     (RGCN self-loop, HGT query and output linears) are computed per node;
 *   - each destination is handled in passes: logits, softmax, aggregation.
 *
 * Conventions (row vectors, y = x W, as in the paper's RGCN equation and its
 * typed-linear formula Y[i,0,j] = sum_k X[i,0,k] W[T[i],k,j]):
 *   h      [N, d_in]              node features
 *   W      [R, d_in, d_out]       one weight per relation
 *   W0     [d_in, d_out]          virtual self-loop weight (may be NULL)
 *   w_src, w_dst [R, d_out]       RGAT attention vectors
 *   outputs are fp64, row-major.
 *
 * OpenMP parallelises over destinations only; each destination's sums are
 * taken in edge-id order, so results do not depend on the thread count.
 *
 * Return value: 0 on success, -1 on invalid arguments, -3 on allocation failure.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* In-edges of every destination, listed in increasing edge id. */
typedef struct {
    int64_t *ptr;   /* [N+1] */
    int64_t *eid;   /* [E]   */
} in_lists;

static int build_in_lists(int64_t N, int64_t E, const int32_t *dst, in_lists *a)
{
    a->ptr = (int64_t *)calloc((size_t)N + 1, sizeof(int64_t));
    a->eid = (int64_t *)malloc((size_t)(E > 0 ? E : 1) * sizeof(int64_t));
    if (!a->ptr || !a->eid) return -3;
    for (int64_t e = 0; e < E; ++e) a->ptr[dst[e] + 1]++;
    for (int64_t v = 0; v < N; ++v) a->ptr[v + 1] += a->ptr[v];
    int64_t *fill = (int64_t *)malloc((size_t)(N > 0 ? N : 1) * sizeof(int64_t));
    if (!fill) return -3;
    memcpy(fill, a->ptr, (size_t)N * sizeof(int64_t));
    for (int64_t e = 0; e < E; ++e) a->eid[fill[dst[e]]++] = e;
    free(fill);
    return 0;
}

static void free_in_lists(in_lists *a) { free(a->ptr); free(a->eid); }

static int check_coo(int64_t N, int64_t E, int32_t R, const int32_t *src,
                     const int32_t *dst, const int32_t *rel)
{
    if (N < 0 || E < 0 || R <= 0) return -1;
    for (int64_t e = 0; e < E; ++e) {
        if (src[e] < 0 || src[e] >= N || dst[e] < 0 || dst[e] >= N) return -1;
        if (rel[e] < 0 || rel[e] >= R) return -1;
    }
    return 0;
}

/* y[0:n] = x[0:k] M, M row-major [k, ldm] starting at column c0 (fp32 M). */
static void vecmat(const double *x, const float *M, int k, int ldm, int c0, int n, double *y)
{
    for (int j = 0; j < n; ++j) y[j] = 0.0;
    for (int i = 0; i < k; ++i) {
        const double xi = x[i];
        const float *row = M + (size_t)i * ldm + c0;
        for (int j = 0; j < n; ++j) y[j] += xi * (double)row[j];
    }
}

static void load_row(const float *h, int64_t n, int d, double *x)
{
    const float *p = h + (size_t)n * d;
    for (int i = 0; i < d; ++i) x[i] = (double)p[i];
}

/* Rows to produce: sel[0:nsel], or every node when sel is NULL. */
static inline int64_t sel_node(const int32_t *sel, int64_t i) { return sel ? sel[i] : i; }

/* Per-destination scratch: per-edge messages and logits of one row. */
typedef struct {
    double *msg, *aux, *z;
    int64_t cap;
    int64_t *cnt;
} row_scratch;

static int scratch_reserve(row_scratch *s, int64_t deg, int d, int H)
{
    if (deg <= s->cap) return 0;
    free(s->msg); free(s->aux); free(s->z);
    s->cap = deg;
    s->msg = (double *)malloc((size_t)deg * d * sizeof(double));
    s->aux = (double *)malloc((size_t)deg * d * sizeof(double));
    s->z = (double *)malloc((size_t)deg * H * sizeof(double));
    if (!s->msg || !s->aux || !s->z) { s->cap = 0; return -3; }
    return 0;
}

static void scratch_free(row_scratch *s) { free(s->msg); free(s->aux); free(s->z); free(s->cnt); }

/* Destinations with more in-edges than this are handled one at a time with
 * the per-edge pass spread over threads; all others one per thread.  The
 * arithmetic and the order of every sum are the same either way. */
#define BIG_ROW 4096

/* ------------------------------------------------------------------------ */
/* RGCN (the paper's RGCN equation):
 *   out_v = act( h_v W0 + sum_r sum_{u in N_v^r} h_u W_r / c_{v,r} )
 * with c_{v,r} the number of in-edges of v with relation r (duplicates counted)
 * and the self-loop term present only when W0 is given.  act = ReLU if relu. */
typedef struct {
    int64_t N, E; int32_t R, d_in, d_out;
    const int32_t *src, *rel; const float *h, *W, *W0; int32_t relu;
    const int32_t *sel; double *out; in_lists a;
} rgcn_ctx;

static int rgcn_row(const rgcn_ctx *c, int64_t i, int inner, row_scratch *sc)
{
    const int64_t v = sel_node(c->sel, i);
    const int64_t p0 = c->a.ptr[v], deg = c->a.ptr[v + 1] - p0;
    const int d_in = c->d_in, d_out = c->d_out;
    if (scratch_reserve(sc, deg, d_out, 1)) return -3;
    double *o = c->out + (size_t)i * d_out;
    for (int j = 0; j < d_out; ++j) o[j] = 0.0;
    if (c->W0) {
        double x[512], m[512];
        load_row(c->h, v, d_in, x);
        vecmat(x, c->W0, d_in, d_out, 0, d_out, m);
        for (int j = 0; j < d_out; ++j) o[j] += m[j];
    }
    for (int r = 0; r < c->R; ++r) sc->cnt[r] = 0;
    for (int64_t p = p0; p < p0 + deg; ++p) sc->cnt[c->rel[c->a.eid[p]]]++;
#pragma omp parallel for schedule(static) if (inner)
    for (int64_t q = 0; q < deg; ++q) {
        double x[512];
        const int64_t e = c->a.eid[p0 + q];
        load_row(c->h, c->src[e], d_in, x);
        vecmat(x, c->W + (size_t)c->rel[e] * d_in * d_out, d_in, d_out, 0, d_out,
               sc->msg + q * d_out);
    }
    for (int64_t q = 0; q < deg; ++q) {
        const double inv_c = 1.0 / (double)sc->cnt[c->rel[c->a.eid[p0 + q]]];
        for (int j = 0; j < d_out; ++j) o[j] += sc->msg[q * d_out + j] * inv_c;
    }
    if (c->relu)
        for (int j = 0; j < d_out; ++j) o[j] = o[j] > 0.0 ? o[j] : 0.0;
    return 0;
}

int oracle_rgcn_forward(int64_t N, int64_t E, int32_t R, int32_t d_in, int32_t d_out,
                        const int32_t *src, const int32_t *dst, const int32_t *rel,
                        const float *h, const float *W, const float *W0, int32_t relu,
                        int64_t nsel, const int32_t *sel, double *out)
{
    if (check_coo(N, E, R, src, dst, rel) || d_in <= 0 || d_out <= 0 || d_in > 512 ||
        d_out > 512)
        return -1;
    rgcn_ctx c = {N, E, R, d_in, d_out, src, rel, h, W, W0, relu, sel, out, {0, 0}};
    int rc = build_in_lists(N, E, dst, &c.a);
    if (rc) { free_in_lists(&c.a); return rc; }
    const int64_t nrows = sel ? nsel : N;
    int err = 0;
#pragma omp parallel reduction(| : err)
    {
        row_scratch sc = {0, 0, 0, 0, (int64_t *)malloc((size_t)R * sizeof(int64_t))};
        if (!sc.cnt) err = 1;
#pragma omp for schedule(dynamic, 16)
        for (int64_t i = 0; i < nrows; ++i) {
            const int64_t v = sel_node(sel, i);
            if (err || c.a.ptr[v + 1] - c.a.ptr[v] > BIG_ROW) continue;
            if (rgcn_row(&c, i, 0, &sc)) err = 1;
        }
        scratch_free(&sc);
    }
    row_scratch sc = {0, 0, 0, 0, (int64_t *)malloc((size_t)R * sizeof(int64_t))};
    if (!sc.cnt) err = 1;
    for (int64_t i = 0; i < nrows && !err; ++i) {
        const int64_t v = sel_node(sel, i);
        if (c.a.ptr[v + 1] - c.a.ptr[v] > BIG_ROW && rgcn_row(&c, i, 1, &sc)) err = 1;
    }
    scratch_free(&sc);
    free_in_lists(&c.a);
    return err ? -3 : 0;
}

/* ------------------------------------------------------------------------ */
/* RGAT (the paper's RGAT listing and the RGAT/HGT figure caption).  For every
 * in-edge e = (u -> v, r) and head k (columns [k*dh, (k+1)*dh) of d_out):
 *   m_e   = h_u W_r                        (edge message)
 *   t_e   = h_v W_r
 *   y_e,k = sum_{j in k} m_e[j] w_src[r][j] + t_e[j] w_dst[r][j]
 *   z_e,k = leakyrelu(y_e,k)  (slope `neg_slope` for y <= 0)
 *   alpha = exp(z_e,k) / sum_{e' in group(e)} exp(z_e',k)
 *   out_v[j in k] = sum_e alpha_e,k m_e[j]   (0 when v has no in-edges)
 * group(e) = all in-edges of v (scope 0) or those of v with relation r (scope 1).
 * Both the numerator and denominator are taken relative to the group maximum,
 * which leaves alpha unchanged.
 * Optional outputs, for scope 0 only: stat_max[v,k] = max z, stat_sum[v,k] =
 * sum exp(z - max); alpha_out[e,k] for every in-edge of a produced row. */
typedef struct {
    int64_t N, E; int32_t R, d_in, d_out, H, scope;
    const int32_t *src, *rel; const float *h, *W, *w_src, *w_dst; double slope;
    const int32_t *sel; double *out, *stat_max, *stat_sum, *alpha_out; in_lists a;
} rgat_ctx;

static int rgat_row(const rgat_ctx *c, int64_t i, int inner, row_scratch *sc, double *mx,
                    double *sm)
{
    const int64_t v = sel_node(c->sel, i);
    const int64_t p0 = c->a.ptr[v], deg = c->a.ptr[v + 1] - p0;
    const int d_in = c->d_in, d_out = c->d_out, H = c->H, dh = d_out / H;
    if (scratch_reserve(sc, deg, d_out, H)) return -3;
    double *o = c->out + (size_t)i * d_out;
    for (int j = 0; j < d_out; ++j) o[j] = 0.0;
    /* pass 1: messages and logits of every in-edge */
#pragma omp parallel for schedule(static) if (inner)
    for (int64_t q = 0; q < deg; ++q) {
        double x[512], xv[512];
        double *msg = sc->msg + q * d_out, *t = sc->aux + q * d_out;
        const int64_t e = c->a.eid[p0 + q];
        const int r = c->rel[e];
        const float *Wr = c->W + (size_t)r * d_in * d_out;
        load_row(c->h, c->src[e], d_in, x);
        load_row(c->h, v, d_in, xv);
        vecmat(x, Wr, d_in, d_out, 0, d_out, msg);
        vecmat(xv, Wr, d_in, d_out, 0, d_out, t);
        for (int k = 0; k < H; ++k) {
            double y = 0.0;
            for (int j = k * dh; j < (k + 1) * dh; ++j)
                y += msg[j] * (double)c->w_src[(size_t)r * d_out + j] +
                     t[j] * (double)c->w_dst[(size_t)r * d_out + j];
            sc->z[q * H + k] = y > 0.0 ? y : c->slope * y;
        }
    }
    /* pass 2: softmax maximum and denominator per group and head */
    const int G = c->scope == 0 ? 1 : c->R;
    for (int q = 0; q < G * H; ++q) { mx[q] = -INFINITY; sm[q] = 0.0; }
    for (int64_t q = 0; q < deg; ++q) {
        const int gi = c->scope == 0 ? 0 : c->rel[c->a.eid[p0 + q]];
        for (int k = 0; k < H; ++k)
            if (sc->z[q * H + k] > mx[gi * H + k]) mx[gi * H + k] = sc->z[q * H + k];
    }
    for (int64_t q = 0; q < deg; ++q) {
        const int gi = c->scope == 0 ? 0 : c->rel[c->a.eid[p0 + q]];
        for (int k = 0; k < H; ++k) sm[gi * H + k] += exp(sc->z[q * H + k] - mx[gi * H + k]);
    }
    /* pass 3: attention-weighted sum of the messages */
    for (int64_t q = 0; q < deg; ++q) {
        const int64_t e = c->a.eid[p0 + q];
        const int gi = c->scope == 0 ? 0 : c->rel[e];
        for (int k = 0; k < H; ++k) {
            const double al = exp(sc->z[q * H + k] - mx[gi * H + k]) / sm[gi * H + k];
            if (c->alpha_out) c->alpha_out[(size_t)e * H + k] = al;
            for (int j = k * dh; j < (k + 1) * dh; ++j) o[j] += al * sc->msg[q * d_out + j];
        }
    }
    if (c->scope == 0) {
        for (int k = 0; k < H; ++k) {
            if (c->stat_max) c->stat_max[(size_t)i * H + k] = deg ? mx[k] : 0.0;
            if (c->stat_sum) c->stat_sum[(size_t)i * H + k] = deg ? sm[k] : 0.0;
        }
    }
    return 0;
}

int oracle_rgat_forward(int64_t N, int64_t E, int32_t R, int32_t d_in, int32_t d_out,
                        int32_t heads, const int32_t *src, const int32_t *dst,
                        const int32_t *rel, const float *h, const float *W,
                        const float *w_src, const float *w_dst, double neg_slope,
                        int32_t scope, int64_t nsel, const int32_t *sel, double *out,
                        double *stat_max, double *stat_sum, double *alpha_out)
{
    if (check_coo(N, E, R, src, dst, rel) || d_in <= 0 || d_out <= 0 || d_in > 512 ||
        d_out > 512 || heads <= 0 || d_out % heads || (scope != 0 && scope != 1))
        return -1;
    rgat_ctx c = {N, E, R, d_in, d_out, heads, scope, src, rel, h, W, w_src, w_dst, neg_slope,
                  sel, out, stat_max, stat_sum, alpha_out, {0, 0}};
    int rc = build_in_lists(N, E, dst, &c.a);
    if (rc) { free_in_lists(&c.a); return rc; }
    const int64_t nrows = sel ? nsel : N;
    const size_t gh = (size_t)R * heads * sizeof(double);
    int err = 0;
#pragma omp parallel reduction(| : err)
    {
        row_scratch sc = {0, 0, 0, 0, 0};
        double *mx = (double *)malloc(gh), *sm = (double *)malloc(gh);
        if (!mx || !sm) err = 1;
#pragma omp for schedule(dynamic, 16)
        for (int64_t i = 0; i < nrows; ++i) {
            const int64_t v = sel_node(sel, i);
            if (err || c.a.ptr[v + 1] - c.a.ptr[v] > BIG_ROW) continue;
            if (rgat_row(&c, i, 0, &sc, mx, sm)) err = 1;
        }
        scratch_free(&sc); free(mx); free(sm);
    }
    row_scratch sc = {0, 0, 0, 0, 0};
    double *mx = (double *)malloc(gh), *sm = (double *)malloc(gh);
    if (!mx || !sm) err = 1;
    for (int64_t i = 0; i < nrows && !err; ++i) {
        const int64_t v = sel_node(sel, i);
        if (c.a.ptr[v + 1] - c.a.ptr[v] > BIG_ROW && rgat_row(&c, i, 1, &sc, mx, sm)) err = 1;
    }
    scratch_free(&sc); free(mx); free(sm);
    free_in_lists(&c.a);
    return err ? -3 : 0;
}

/* ------------------------------------------------------------------------ */
/* HGT (the layer the paper's RGAT/HGT figure shows; equations of the HGT
 * paper it cites).  Heads split d into H blocks of dk = d / H.
 *   K_n = h_n Wk[tau(n)],  Q_n = h_n Wq[tau(n)],  V_n = h_n Wv[tau(n)]
 *   for every in-edge e = (s -> t, r) and head i:
 *     a_e,i   = (K_s,i Watt[r][i]) . Q_t,i * mu[r] * att_scale
 *     msg_e,i = V_s,i Wmsg[r][i]
 *     alpha_e,i = softmax of a_.,i over all in-edges of t
 *   agg_t = concat_i sum_e alpha_e,i msg_e,i      (0 without in-edges)
 *   out_t = agg_t Wa[tau(t)] (if a_linear, else agg_t) + h_t (if residual)
 * K and V are recomputed for every edge from h_s (they depend only on the
 * source node; recomputation gives the same fp64 values). */
typedef struct {
    int64_t N, E; int32_t R, T, d, H;
    const int32_t *src, *rel, *ntype; const float *h, *Wk, *Wq, *Wv, *Wa, *Watt, *Wmsg, *mu;
    double scale; int32_t residual, a_linear;
    const int32_t *sel; double *out; in_lists a;
} hgt_ctx;

static int hgt_row(const hgt_ctx *c, int64_t i, int inner, row_scratch *sc, double *mx,
                   double *sm)
{
    const int64_t t = sel_node(c->sel, i);
    const int64_t p0 = c->a.ptr[t], deg = c->a.ptr[t + 1] - p0;
    const int d = c->d, H = c->H, dk = d / H;
    if (scratch_reserve(sc, deg, d, H)) return -3;
    double q[512], agg[512];
    {
        double x[512];
        load_row(c->h, t, d, x);
        vecmat(x, c->Wq + (size_t)c->ntype[t] * d * d, d, d, 0, d, q);
    }
#pragma omp parallel for schedule(static) if (inner)
    for (int64_t p = 0; p < deg; ++p) {
        double x[512], kk[512], vv[512], kw[512];
        const int64_t e = c->a.eid[p0 + p];
        const int64_t s = c->src[e];
        const int r = c->rel[e];
        load_row(c->h, s, d, x);
        vecmat(x, c->Wk + (size_t)c->ntype[s] * d * d, d, d, 0, d, kk);
        vecmat(x, c->Wv + (size_t)c->ntype[s] * d * d, d, d, 0, d, vv);
        for (int hh = 0; hh < H; ++hh) {
            const float *Wat = c->Watt + ((size_t)r * H + hh) * dk * dk;
            const float *Wms = c->Wmsg + ((size_t)r * H + hh) * dk * dk;
            vecmat(kk + hh * dk, Wat, dk, dk, 0, dk, kw);
            double dot = 0.0;
            for (int j = 0; j < dk; ++j) dot += kw[j] * q[hh * dk + j];
            sc->z[p * H + hh] = dot * (double)c->mu[r] * c->scale;
            vecmat(vv + hh * dk, Wms, dk, dk, 0, dk, sc->msg + p * d + hh * dk);
        }
    }
    for (int hh = 0; hh < H; ++hh) { mx[hh] = -INFINITY; sm[hh] = 0.0; }
    for (int64_t p = 0; p < deg; ++p)
        for (int hh = 0; hh < H; ++hh)
            if (sc->z[p * H + hh] > mx[hh]) mx[hh] = sc->z[p * H + hh];
    for (int64_t p = 0; p < deg; ++p)
        for (int hh = 0; hh < H; ++hh) sm[hh] += exp(sc->z[p * H + hh] - mx[hh]);
    for (int j = 0; j < d; ++j) agg[j] = 0.0;
    for (int64_t p = 0; p < deg; ++p)
        for (int hh = 0; hh < H; ++hh) {
            const double al = exp(sc->z[p * H + hh] - mx[hh]) / sm[hh];
            for (int j = hh * dk; j < (hh + 1) * dk; ++j) agg[j] += al * sc->msg[p * d + j];
        }
    double *o = c->out + (size_t)i * d;
    if (c->a_linear) vecmat(agg, c->Wa + (size_t)c->ntype[t] * d * d, d, d, 0, d, o);
    else for (int j = 0; j < d; ++j) o[j] = agg[j];
    if (c->residual)
        for (int j = 0; j < d; ++j) o[j] += (double)c->h[(size_t)t * d + j];
    return 0;
}

int oracle_hgt_forward(int64_t N, int64_t E, int32_t R, int32_t T, int32_t d,
                       int32_t heads, const int32_t *src, const int32_t *dst,
                       const int32_t *rel, const int32_t *ntype, const float *h,
                       const float *Wk, const float *Wq, const float *Wv, const float *Wa,
                       const float *Watt, const float *Wmsg, const float *mu,
                       double att_scale, int32_t residual, int32_t a_linear,
                       int64_t nsel, const int32_t *sel, double *out)
{
    if (check_coo(N, E, R, src, dst, rel) || T <= 0 || d <= 0 || d > 512 || heads <= 0 ||
        d % heads)
        return -1;
    for (int64_t n = 0; n < N; ++n)
        if (ntype[n] < 0 || ntype[n] >= T) return -1;
    hgt_ctx c = {N, E, R, T, d, heads, src, rel, ntype, h, Wk, Wq, Wv, Wa, Watt, Wmsg, mu,
                 att_scale, residual, a_linear, sel, out, {0, 0}};
    int rc = build_in_lists(N, E, dst, &c.a);
    if (rc) { free_in_lists(&c.a); return rc; }
    const int64_t nrows = sel ? nsel : N;
    const size_t hb = (size_t)heads * sizeof(double);
    int err = 0;
#pragma omp parallel reduction(| : err)
    {
        row_scratch sc = {0, 0, 0, 0, 0};
        double *mx = (double *)malloc(hb), *sm = (double *)malloc(hb);
        if (!mx || !sm) err = 1;
#pragma omp for schedule(dynamic, 16)
        for (int64_t i = 0; i < nrows; ++i) {
            const int64_t t = sel_node(sel, i);
            if (err || c.a.ptr[t + 1] - c.a.ptr[t] > BIG_ROW) continue;
            if (hgt_row(&c, i, 0, &sc, mx, sm)) err = 1;
        }
        scratch_free(&sc); free(mx); free(sm);
    }
    row_scratch sc = {0, 0, 0, 0, 0};
    double *mx = (double *)malloc(hb), *sm = (double *)malloc(hb);
    if (!mx || !sm) err = 1;
    for (int64_t i = 0; i < nrows && !err; ++i) {
        const int64_t t = sel_node(sel, i);
        if (c.a.ptr[t + 1] - c.a.ptr[t] > BIG_ROW && hgt_row(&c, i, 1, &sc, mx, sm)) err = 1;
    }
    scratch_free(&sc); free(mx); free(sm);
    free_in_lists(&c.a);
    return err ? -3 : 0;
}

/* ------------------------------------------------------------------------ */
/* RGAT backward for the loss L = sum(out * G) (G = grad_out), softmax over all
 * in-edges of the destination (scope 0) or over its in-edges of one relation
 * (scope 1; the groups below are then the (v, r) segments).  With the
 * forward's notation and Y_e,k = dL/dy_e,k:
 *   dalpha_e,k = sum_{j in k} G_v[j] m_e[j]
 *   s_g,k      = sum_{e in group g} alpha_e,k dalpha_e,k     (g: e's group)
 *   Y_e,k      = alpha_e,k (dalpha_e,k - s_g,k) * (1 if y_e,k > 0 else slope)
 *   dm_e[j]    = alpha_e,k G_v[j] + Y_e,k w_src[r][j]     (message and atts paths)
 *   dt_e[j]    = Y_e,k w_dst[r][j]                          (attt path)
 *   dW_r      += h_u^T dm_e + h_v^T dt_e
 *   dh_u      += dm_e W_r^T ;   dh_v += dt_e W_r^T
 *   dw_src[r] += Y_e,k m_e ;    dw_dst[r] += Y_e,k t_e
 * node_mask (nullable): compute dh only for nodes with node_mask[n] != 0
 * rel_mask  (nullable): compute dW, dw_src, dw_dst only for those relations.
 * Entries outside the masks are left at zero.  Only destinations that feed a
 * requested entry are visited.
 * kink_flip (nullable, [E, H] by edge id): the leaky ReLU has no derivative at
 * y = 0; where kink_flip[e * H + k] != 0 the derivative is taken from the
 * other side of the kink (1 for y <= 0, slope for y > 0).  A caller flags the
 * edges whose pre-activation lies within rounding of zero, where an fp32
 * evaluation may land on either side and both one-sided derivatives are
 * correct results.
 * Y_out (nullable, [E, H] by edge id): receives Y_e,k = dL/dy_e,k of every edge
 * whose destination was visited (NaN for the others).
 *
 * Every sum over edges runs in one fixed order, the "global edge order":
 * destinations in increasing id, each destination's in-edges in increasing
 * edge id.  The work is spread over threads in three stages, none of which
 * changes that order for any output entry:
 *   A. per destination (threads over destinations): the forward recomputed
 *      edge by edge, the softmax, dalpha, s and Y; alpha and Y are kept per
 *      edge;
 *   B. per requested relation (threads over relations x blocks of output
 *      rows or columns): dW_r, dw_src[r], dw_dst[r] summed over r's edges in
 *      the global order, with m_e and t_e recomputed from h and W_r;
 *   C. per requested node n (threads over nodes): dh_n summed over the edges
 *      that touch n in the global order (an edge that is both an out-edge and
 *      an in-edge of n adds its source term first). */
typedef struct {
    int64_t N, E;
    int32_t R, d_in, d_out, H, scope;
    const int32_t *src, *dst, *rel;
    const float *h, *W, *w_src, *w_dst, *G;
    double slope;
    const in_lists *a;
    double *AL, *YY;   /* [E, H] alpha and Y by edge id */
    const uint8_t *flip;   /* [E, H] or NULL: derivative from the other side of the kink */
} rgat_bwd_ctx;

typedef struct {
    double *msg, *t, *al, *y, *da, *mx, *sm, *sv;
    int64_t cap;
} rgat_bwd_scratch;

static int rgat_bwd_reserve(rgat_bwd_scratch *s, int64_t deg, int d_out, int H, int R)
{
    if (!s->mx) {
        s->mx = (double *)malloc((size_t)R * H * sizeof(double));
        s->sm = (double *)malloc((size_t)R * H * sizeof(double));
        s->sv = (double *)malloc((size_t)R * H * sizeof(double));
        if (!s->mx || !s->sm || !s->sv) return -3;
    }
    if (deg <= s->cap) return 0;
    free(s->msg); free(s->t); free(s->al); free(s->y); free(s->da);
    s->cap = deg;
    s->msg = (double *)malloc((size_t)deg * d_out * sizeof(double));
    s->t = (double *)malloc((size_t)deg * d_out * sizeof(double));
    s->al = (double *)malloc((size_t)deg * H * sizeof(double));
    s->y = (double *)malloc((size_t)deg * H * sizeof(double));
    s->da = (double *)malloc((size_t)deg * H * sizeof(double));
    if (!s->msg || !s->t || !s->al || !s->y || !s->da) { s->cap = 0; return -3; }
    return 0;
}

static void rgat_bwd_scratch_free(rgat_bwd_scratch *s)
{
    free(s->msg); free(s->t); free(s->al); free(s->y); free(s->da);
    free(s->mx); free(s->sm); free(s->sv);
}

/* Stage A for destination v: alpha and Y of its in-edges.  inner: spread the
 * per-edge recomputation over threads (for destinations with many edges). */
static int rgat_bwd_dst(const rgat_bwd_ctx *c, int64_t v, int inner, rgat_bwd_scratch *sc)
{
    const int H = c->H, d_in = c->d_in, d_out = c->d_out, dh_ = d_out / H;
    const int64_t p0 = c->a->ptr[v], deg = c->a->ptr[v + 1] - p0;
    if (deg == 0) return 0;
    if (rgat_bwd_reserve(sc, deg, d_out, H, c->R)) return -3;
    double xv[512];
    load_row(c->h, v, d_in, xv);
    double *msg = sc->msg, *t = sc->t, *al = sc->al, *Y = sc->y, *dal = sc->da;
    /* forward recomputation: messages, t_e, logits */
#pragma omp parallel for schedule(static) if (inner)
    for (int64_t q = 0; q < deg; ++q) {
        double xl[512];
        const int64_t e = c->a->eid[p0 + q];
        const int r = c->rel[e];
        const float *Wr = c->W + (size_t)r * d_in * d_out;
        load_row(c->h, c->src[e], d_in, xl);
        vecmat(xl, Wr, d_in, d_out, 0, d_out, msg + q * d_out);
        vecmat(xv, Wr, d_in, d_out, 0, d_out, t + q * d_out);
        for (int k = 0; k < H; ++k) {
            double y = 0.0;
            for (int j = k * dh_; j < (k + 1) * dh_; ++j)
                y += msg[q * d_out + j] * (double)c->w_src[(size_t)r * d_out + j] +
                     t[q * d_out + j] * (double)c->w_dst[(size_t)r * d_out + j];
            Y[q * H + k] = y;          /* pre-activation, kept for the derivative */
            al[q * H + k] = y > 0.0 ? y : c->slope * y;
        }
    }
    double *mx = sc->mx, *sm = sc->sm, *sv = sc->sv;
#define GRP(q) ((c->scope ? c->rel[c->a->eid[p0 + (q)]] : 0) * H)
    for (int64_t q = 0; q < deg; ++q)
        for (int k = 0; k < H; ++k) { mx[GRP(q) + k] = -INFINITY; sm[GRP(q) + k] = 0.0; sv[GRP(q) + k] = 0.0; }
    for (int64_t q = 0; q < deg; ++q)
        for (int k = 0; k < H; ++k) if (al[q * H + k] > mx[GRP(q) + k]) mx[GRP(q) + k] = al[q * H + k];
    for (int64_t q = 0; q < deg; ++q)
        for (int k = 0; k < H; ++k) sm[GRP(q) + k] += exp(al[q * H + k] - mx[GRP(q) + k]);
    for (int64_t q = 0; q < deg; ++q)
        for (int k = 0; k < H; ++k) al[q * H + k] = exp(al[q * H + k] - mx[GRP(q) + k]) / sm[GRP(q) + k];
    /* dalpha and s (per normalisation group) */
    const float *Gv = c->G + (size_t)v * d_out;
    for (int64_t q = 0; q < deg; ++q)
        for (int k = 0; k < H; ++k) {
            double da = 0.0;
            for (int j = k * dh_; j < (k + 1) * dh_; ++j) da += (double)Gv[j] * msg[q * d_out + j];
            sv[GRP(q) + k] += al[q * H + k] * da;
            dal[q * H + k] = da;
        }
    for (int64_t q = 0; q < deg; ++q) {
        const int64_t e = c->a->eid[p0 + q];
        for (int k = 0; k < H; ++k) {
            const double y = Y[q * H + k];
            const double dz = al[q * H + k] * (dal[q * H + k] - sv[GRP(q) + k]);
            c->AL[e * H + k] = al[q * H + k];
            const int pos = (y > 0.0) != (c->flip && c->flip[e * H + k]);
            c->YY[e * H + k] = dz * (pos ? 1.0 : c->slope);
        }
    }
#undef GRP
    return 0;
}

/* dm_e (message and source-attention paths) and dt_e (destination-attention
 * path) of edge e, from its alpha and Y. */
static void rgat_bwd_edge_grads(const rgat_bwd_ctx *c, int64_t e, double *dm, double *dtv)
{
    const int H = c->H, d_out = c->d_out, dh_ = d_out / H;
    const int r = c->rel[e];
    const float *Gv = c->G + (size_t)c->dst[e] * d_out;
    for (int j = 0; j < d_out; ++j) {
        const int k = j / dh_;
        if (dm) dm[j] = c->AL[e * H + k] * (double)Gv[j] + c->YY[e * H + k] * (double)c->w_src[(size_t)r * d_out + j];
        if (dtv) dtv[j] = c->YY[e * H + k] * (double)c->w_dst[(size_t)r * d_out + j];
    }
}

/* dst_row[i] += sum_j W_r[i][j] g[j] */
static void add_matvec_t(const float *Wr, int d_in, int d_out, const double *g, double *dst_row)
{
    for (int i = 0; i < d_in; ++i) {
        double s = 0.0;
        for (int j = 0; j < d_out; ++j) s += (double)Wr[(size_t)i * d_out + j] * g[j];
        dst_row[i] += s;
    }
}

#define RGAT_BWD_ROWS 8   /* dW rows, or dw columns, per stage-B job */

int oracle_rgat_backward(int64_t N, int64_t E, int32_t R, int32_t d_in, int32_t d_out,
                         int32_t heads, const int32_t *src, const int32_t *dst,
                         const int32_t *rel, const float *h, const float *W,
                         const float *w_src, const float *w_dst, double neg_slope,
                         int32_t scope, const float *G, const uint8_t *node_mask,
                         const uint8_t *rel_mask, const uint8_t *kink_flip, double *dh, double *dW,
                         double *dw_src, double *dw_dst, double *Y_out)
{
    if (check_coo(N, E, R, src, dst, rel) || d_in <= 0 || d_in > 512 || d_out <= 0 ||
        d_out > 512 || heads <= 0 || d_out % heads)
        return -1;
    const int H = heads;
    in_lists a;
    int rc = build_in_lists(N, E, dst, &a);
    if (rc) { free_in_lists(&a); return rc; }
    memset(dh, 0, (size_t)N * d_in * sizeof(double));
    memset(dW, 0, (size_t)R * d_in * d_out * sizeof(double));
    memset(dw_src, 0, (size_t)R * d_out * sizeof(double));
    memset(dw_dst, 0, (size_t)R * d_out * sizeof(double));
    /* destinations whose in-edges contribute to a requested entry */
    const size_t E1 = (size_t)(E > 0 ? E : 1), N1 = (size_t)(N > 0 ? N : 1);
    uint8_t *need = (uint8_t *)calloc(N1, 1);
    double *AL = (double *)malloc(E1 * H * sizeof(double));
    double *YY = (double *)malloc(E1 * H * sizeof(double));
    int64_t *relptr = (int64_t *)calloc((size_t)R + 1, sizeof(int64_t));
    int64_t *reledge = (int64_t *)malloc(E1 * sizeof(int64_t));
    int64_t *outptr = (int64_t *)calloc(N1 + 1, sizeof(int64_t));
    int64_t *outpos = (int64_t *)malloc(E1 * sizeof(int64_t));
    int err = !need || !AL || !YY || !relptr || !reledge || !outptr || !outpos;
    if (!err) {
        for (int64_t e = 0; e < E; ++e) {
            const int want_rel = rel_mask ? rel_mask[rel[e]] != 0 : 1;
            const int want_node = node_mask ? (node_mask[src[e]] || node_mask[dst[e]]) : 1;
            if (want_rel || want_node) need[dst[e]] = 1;
        }
        /* relations' edge lists and sources' out-edge positions, both in the
         * global edge order (positions p index a.eid) */
        for (int64_t e = 0; e < E; ++e) { relptr[rel[e] + 1]++; outptr[src[e] + 1]++; }
        for (int r = 0; r < R; ++r) relptr[r + 1] += relptr[r];
        for (int64_t n = 0; n < N; ++n) outptr[n + 1] += outptr[n];
        int64_t *rf = (int64_t *)malloc((size_t)R * sizeof(int64_t));
        int64_t *of = (int64_t *)malloc(N1 * sizeof(int64_t));
        if (!rf || !of) {
            err = 1;
        } else {
            memcpy(rf, relptr, (size_t)R * sizeof(int64_t));
            memcpy(of, outptr, (size_t)N * sizeof(int64_t));
            for (int64_t p = 0; p < E; ++p) {
                const int64_t e = a.eid[p];
                reledge[rf[rel[e]]++] = e;
                outpos[of[src[e]]++] = p;
            }
        }
        free(rf); free(of);
    }
    rgat_bwd_ctx c = {N, E, R, d_in, d_out, H, scope, src, dst, rel, h, W, w_src, w_dst, G,
                      neg_slope, &a, AL, YY, kink_flip};
    /* stage A */
    if (!err) {
#pragma omp parallel reduction(| : err)
        {
            rgat_bwd_scratch sc = {0};
#pragma omp for schedule(dynamic, 16)
            for (int64_t v = 0; v < N; ++v)
                if (need[v] && a.ptr[v + 1] - a.ptr[v] <= BIG_ROW && rgat_bwd_dst(&c, v, 0, &sc)) err = 1;
            rgat_bwd_scratch_free(&sc);
        }
    }
    if (!err) {
        rgat_bwd_scratch sc = {0};
        for (int64_t v = 0; v < N && !err; ++v)
            if (need[v] && a.ptr[v + 1] - a.ptr[v] > BIG_ROW && rgat_bwd_dst(&c, v, 1, &sc)) err = 1;
        rgat_bwd_scratch_free(&sc);
    }
    if (!err && Y_out)
        for (int64_t e = 0; e < E; ++e)
            for (int k = 0; k < H; ++k)
                Y_out[e * H + k] = need[dst[e]] ? YY[e * H + k] : NAN;
    /* stage B: jobs (relation, block of dW rows) then (relation, block of dw columns) */
    if (!err) {
        const int nbi = (d_in + RGAT_BWD_ROWS - 1) / RGAT_BWD_ROWS;
        const int nbj = (d_out + RGAT_BWD_ROWS - 1) / RGAT_BWD_ROWS;
        const int64_t njobs = (int64_t)R * (nbi + nbj);
#pragma omp parallel for schedule(dynamic, 1)
        for (int64_t job = 0; job < njobs; ++job) {
            const int r = (int)(job / (nbi + nbj)), b = (int)(job % (nbi + nbj));
            if (rel_mask && !rel_mask[r]) continue;
            const float *Wr = W + (size_t)r * d_in * d_out;
            double dm[512], dtv[512], xu[512], xv[512], mb[RGAT_BWD_ROWS], tb[RGAT_BWD_ROWS];
            if (b < nbi) {
                const int i0 = b * RGAT_BWD_ROWS, i1 = i0 + RGAT_BWD_ROWS < d_in ? i0 + RGAT_BWD_ROWS : d_in;
                for (int64_t q = relptr[r]; q < relptr[r + 1]; ++q) {
                    const int64_t e = reledge[q];
                    rgat_bwd_edge_grads(&c, e, dm, dtv);
                    for (int i = i0; i < i1; ++i) {
                        const double hu = (double)h[(size_t)src[e] * d_in + i];
                        const double hv = (double)h[(size_t)dst[e] * d_in + i];
                        double *row = dW + ((size_t)r * d_in + i) * d_out;
                        for (int j = 0; j < d_out; ++j) row[j] += hu * dm[j] + hv * dtv[j];
                    }
                }
            } else {
                const int j0 = (b - nbi) * RGAT_BWD_ROWS;
                const int nj = j0 + RGAT_BWD_ROWS < d_out ? RGAT_BWD_ROWS : d_out - j0;
                const int dh_ = d_out / H;
                for (int64_t q = relptr[r]; q < relptr[r + 1]; ++q) {
                    const int64_t e = reledge[q];
                    load_row(h, src[e], d_in, xu);
                    load_row(h, dst[e], d_in, xv);
                    vecmat(xu, Wr, d_in, d_out, j0, nj, mb);
                    vecmat(xv, Wr, d_in, d_out, j0, nj, tb);
                    for (int jj = 0; jj < nj; ++jj) {
                        const double y = YY[e * H + (j0 + jj) / dh_];
                        dw_src[(size_t)r * d_out + j0 + jj] += y * mb[jj];
                        dw_dst[(size_t)r * d_out + j0 + jj] += y * tb[jj];
                    }
                }
            }
        }
    }
    /* stage C: dh of the requested nodes, merging each node's out-edges and
     * in-edges by their position in the global order */
    if (!err) {
#pragma omp parallel for schedule(dynamic, 64)
        for (int64_t n = 0; n < N; ++n) {
            if (node_mask && !node_mask[n]) continue;
            double g[512];
            double *row = dh + (size_t)n * d_in;
            int64_t po = outptr[n], pi = a.ptr[n];
            const int64_t po1 = outptr[n + 1], pi1 = a.ptr[n + 1];
            while (po < po1 || pi < pi1) {
                if (po < po1 && (pi >= pi1 || outpos[po] <= pi)) {   /* n as the source */
                    const int64_t e = a.eid[outpos[po++]];
                    rgat_bwd_edge_grads(&c, e, g, NULL);
                    add_matvec_t(W + (size_t)rel[e] * d_in * d_out, d_in, d_out, g, row);
                } else {                                             /* n as the destination */
                    const int64_t e = a.eid[pi++];
                    rgat_bwd_edge_grads(&c, e, NULL, g);
                    add_matvec_t(W + (size_t)rel[e] * d_in * d_out, d_in, d_out, g, row);
                }
            }
        }
    }
    free(need); free(AL); free(YY); free(relptr); free(reledge); free(outptr); free(outpos);
    free_in_lists(&a);
    return err ? -3 : 0;
}

/* ------------------------------------------------------------------------ */
/* RGCN backward for the loss L = sum(out * G) (G = grad_out), from the paper's
 * RGCN equation by the chain rule.  With the pre-activation
 *   P_v = h_v W0 + sum_r sum_{u in N_v^r} h_u W_r / c_{v,r}
 * and Gp_v = G_v * act'(P_v) (ReLU: 1 where P_v > 0, else 0; identity: 1):
 *   dW_r += h_u^T Gp_v / c_{v,r},   dh_u += Gp_v W_r^T / c_{v,r}   per in-edge (u -> v, r)
 *   dW0  += h_v^T Gp_v,             dh_v += Gp_v W0^T              per node (W0 given)
 * node_mask / rel_mask (nullable) restrict dh and dW as for the RGAT backward;
 * dW0 is computed when both W0 and dW0 are given.  Destinations are visited in
 * increasing id and their in-edges in edge-id order. */
int oracle_rgcn_backward(int64_t N, int64_t E, int32_t R, int32_t d_in, int32_t d_out,
                         const int32_t *src, const int32_t *dst, const int32_t *rel,
                         const float *h, const float *W, const float *W0, int32_t relu,
                         const float *G, const uint8_t *node_mask, const uint8_t *rel_mask,
                         double *dh, double *dW, double *dW0)
{
    if (check_coo(N, E, R, src, dst, rel) || d_in <= 0 || d_in > 512 || d_out <= 0 || d_out > 512)
        return -1;
    in_lists a;
    int rc = build_in_lists(N, E, dst, &a);
    if (rc) { free_in_lists(&a); return rc; }
    const int want_w0 = W0 && dW0;
    uint8_t *need = (uint8_t *)calloc((size_t)(N > 0 ? N : 1), 1);
    int64_t *cnt = (int64_t *)malloc((size_t)(R > 0 ? R : 1) * sizeof(int64_t));
    double *P = (double *)malloc((size_t)d_out * sizeof(double));
    double *Gp = (double *)malloc((size_t)d_out * sizeof(double));
    double *xv = (double *)malloc((size_t)d_in * sizeof(double));
    double *xu = (double *)malloc((size_t)d_in * sizeof(double));
    double *m = (double *)malloc((size_t)d_out * sizeof(double));
    int err = !need || !cnt || !P || !Gp || !xv || !xu || !m;
    if (!err) {
        for (int64_t v = 0; v < N; ++v)
            if (want_w0 || (W0 && (!node_mask || node_mask[v]))) need[v] = 1;
        for (int64_t e = 0; e < E; ++e)
            if ((!rel_mask || rel_mask[rel[e]]) || (!node_mask || node_mask[src[e]])) need[dst[e]] = 1;
        memset(dh, 0, (size_t)N * d_in * sizeof(double));
        memset(dW, 0, (size_t)R * d_in * d_out * sizeof(double));
        if (want_w0) memset(dW0, 0, (size_t)d_in * d_out * sizeof(double));
    }
    for (int64_t v = 0; v < N && !err; ++v) {
        if (!need[v]) continue;
        const int64_t p0 = a.ptr[v], deg = a.ptr[v + 1] - p0;
        for (int r = 0; r < R; ++r) cnt[r] = 0;
        for (int64_t p = p0; p < p0 + deg; ++p) cnt[rel[a.eid[p]]]++;
        load_row(h, v, d_in, xv);
        const float *Gv = G + (size_t)v * d_out;
        for (int j = 0; j < d_out; ++j) Gp[j] = (double)Gv[j];
        if (relu) {   /* recompute the pre-activation */
            for (int j = 0; j < d_out; ++j) P[j] = 0.0;
            if (W0) {
                vecmat(xv, W0, d_in, d_out, 0, d_out, m);
                for (int j = 0; j < d_out; ++j) P[j] += m[j];
            }
            for (int64_t p = p0; p < p0 + deg; ++p) {
                const int64_t e = a.eid[p];
                load_row(h, src[e], d_in, xu);
                vecmat(xu, W + (size_t)rel[e] * d_in * d_out, d_in, d_out, 0, d_out, m);
                const double inv_c = 1.0 / (double)cnt[rel[e]];
                for (int j = 0; j < d_out; ++j) P[j] += m[j] * inv_c;
            }
            for (int j = 0; j < d_out; ++j) if (!(P[j] > 0.0)) Gp[j] = 0.0;
        }
        if (W0) {
            if (want_w0)
                for (int i = 0; i < d_in; ++i)
                    for (int j = 0; j < d_out; ++j) dW0[(size_t)i * d_out + j] += xv[i] * Gp[j];
            if (!node_mask || node_mask[v])
                for (int i = 0; i < d_in; ++i) {
                    double s = 0.0;
                    for (int j = 0; j < d_out; ++j) s += (double)W0[(size_t)i * d_out + j] * Gp[j];
                    dh[(size_t)v * d_in + i] += s;
                }
        }
        for (int64_t p = p0; p < p0 + deg; ++p) {
            const int64_t e = a.eid[p];
            const int r = rel[e];
            const int64_t u = src[e];
            const double inv_c = 1.0 / (double)cnt[r];
            const float *Wr = W + (size_t)r * d_in * d_out;
            if (!rel_mask || rel_mask[r]) {
                load_row(h, u, d_in, xu);
                for (int i = 0; i < d_in; ++i) {
                    double *row = dW + ((size_t)r * d_in + i) * d_out;
                    for (int j = 0; j < d_out; ++j) row[j] += xu[i] * Gp[j] * inv_c;
                }
            }
            if (!node_mask || node_mask[u])
                for (int i = 0; i < d_in; ++i) {
                    double s = 0.0;
                    for (int j = 0; j < d_out; ++j) s += (double)Wr[(size_t)i * d_out + j] * Gp[j];
                    dh[(size_t)u * d_in + i] += s * inv_c;
                }
        }
    }
    free(need); free(cnt); free(P); free(Gp); free(xv); free(xu); free(m);
    free_in_lists(&a);
    return err ? -3 : 0;
}

/* ------------------------------------------------------------------------ */
/* HGT backward for the loss L = sum(out * G) (G = grad_out): the chain rule of
 * the HGT layer above.  With c_r = mu[r] * att_scale and kw_e,i = K_s,i Watt[r][i]:
 *   dagg_t = G_t Wa[tau(t)]^T (a_linear, else G_t);  dWa[tau(t)] += agg_t^T G_t
 *   dh_t  += G_t                                              (residual)
 *   for every in-edge e = (s -> t, r) and head i:
 *     dalpha = dagg_t,i . msg_e,i;  s_t,i = sum_e alpha dalpha;  da = alpha (dalpha - s_t,i)
 *     dmsg = alpha dagg_t,i:   dWmsg[r][i] += V_s,i^T dmsg;  dV_s,i += dmsg Wmsg[r][i]^T
 *     dkw = da c_r Q_t,i:      dWatt[r][i] += K_s,i^T dkw;   dK_s,i += dkw Watt[r][i]^T
 *     dQ_t,i += da c_r kw_e,i;  dmu[r] += da att_scale (kw_e,i . Q_t,i)
 *   for every node n (X in K, Q, V):
 *     dWx[tau(n)] += h_n^T dX_n;  dh_n += dX_n Wx[tau(n)]^T
 * K, Q, V are computed once per node (node-level linears); every edge term is
 * computed per edge.  Every sum over edges runs in the global edge order
 * (destinations in increasing id, each one's in-edges in increasing edge id),
 * every sum over nodes in increasing node id.  The work is spread over
 * threads in stages that keep those orders for every output entry:
 *   A. per destination: scores, softmax, messages, agg, dagg, s; alpha, da
 *      and kw . Q kept per edge, dQ per destination;
 *   B. per relation (and head, and row of the head block): dWatt, dWmsg,
 *      dmu over the relation's edges; per node type and row: dWa;
 *   C. per source: dK and dV over its out-edges;
 *   D. per node type, projection and row: dWk, dWq, dWv; per node: dh.
 * node_mask (nullable): dh only for those nodes; rel_mask (nullable): dWatt,
 * dWmsg and dmu only for those relations.  With either mask the node-type
 * weight gradients (dWk, dWq, dWv, dWa) are not computed (left zero), and
 * only the destinations that feed a requested entry are visited.  dWa may be
 * NULL when a_linear is 0. */
typedef struct {
    int64_t N, E;
    int32_t R, T, d, H;
    const int32_t *src, *dst, *rel, *ntype;
    const float *Wa, *Watt, *Wmsg, *mu, *G;
    double att_scale;
    int32_t a_linear;
    const in_lists *a;
    const double *K, *Q, *V;
    double *agg, *dagg, *dQ;     /* [N, d] */
    double *AL, *DA, *KQ;        /* [E, H] alpha, da and kw . Q by edge id */
} hgt_bwd_ctx;

static int hgt_bwd_dst(const hgt_bwd_ctx *c, int64_t t, double **kwbuf, double **msgbuf, double **albuf,
                       double **dalbuf, int64_t *cap)
{
    const int H = c->H, d = c->d, dk = d / H;
    const int64_t p0 = c->a->ptr[t], deg = c->a->ptr[t + 1] - p0;
    if (deg > *cap) {
        free(*kwbuf); free(*msgbuf); free(*albuf); free(*dalbuf);
        *cap = deg;
        *kwbuf = (double *)malloc((size_t)deg * d * sizeof(double));
        *msgbuf = (double *)malloc((size_t)deg * d * sizeof(double));
        *albuf = (double *)malloc((size_t)deg * H * sizeof(double));
        *dalbuf = (double *)malloc((size_t)deg * H * sizeof(double));
        if (!*kwbuf || !*msgbuf || !*albuf || !*dalbuf) { *cap = 0; return -3; }
    }
    double *kw = *kwbuf, *msg = *msgbuf, *al = *albuf, *dal = *dalbuf;
    const float *Gt = c->G + (size_t)t * d;
    const double *Qt = c->Q + (size_t)t * d;
    double *agg = c->agg + (size_t)t * d, *dagg = c->dagg + (size_t)t * d, *dQt = c->dQ + (size_t)t * d;
    double mx[64], sm[64], sv[64];
    /* forward: scores, softmax, messages, agg */
    for (int64_t p = 0; p < deg; ++p) {
        const int64_t e = c->a->eid[p0 + p];
        const int64_t sn = c->src[e];
        const int r = c->rel[e];
        for (int i = 0; i < H; ++i) {
            const float *Wat = c->Watt + ((size_t)r * H + i) * dk * dk;
            const float *Wms = c->Wmsg + ((size_t)r * H + i) * dk * dk;
            vecmat(c->K + (size_t)sn * d + i * dk, Wat, dk, dk, 0, dk, kw + p * d + i * dk);
            vecmat(c->V + (size_t)sn * d + i * dk, Wms, dk, dk, 0, dk, msg + p * d + i * dk);
            double dot = 0.0;
            for (int j = 0; j < dk; ++j) dot += kw[p * d + i * dk + j] * Qt[i * dk + j];
            al[p * H + i] = dot * (double)c->mu[r] * c->att_scale;
        }
    }
    for (int i = 0; i < H; ++i) { mx[i] = -INFINITY; sm[i] = 0.0; sv[i] = 0.0; }
    for (int64_t p = 0; p < deg; ++p)
        for (int i = 0; i < H; ++i) if (al[p * H + i] > mx[i]) mx[i] = al[p * H + i];
    for (int64_t p = 0; p < deg; ++p)
        for (int i = 0; i < H; ++i) sm[i] += exp(al[p * H + i] - mx[i]);
    for (int64_t p = 0; p < deg; ++p)
        for (int i = 0; i < H; ++i) al[p * H + i] = exp(al[p * H + i] - mx[i]) / sm[i];
    for (int j = 0; j < d; ++j) agg[j] = 0.0;
    for (int64_t p = 0; p < deg; ++p)
        for (int j = 0; j < d; ++j) agg[j] += al[p * H + j / dk] * msg[p * d + j];
    /* output linear */
    if (c->a_linear) {
        const float *Wat = c->Wa + (size_t)c->ntype[t] * d * d;
        for (int i = 0; i < d; ++i) {
            double s2 = 0.0;
            for (int j = 0; j < d; ++j) s2 += (double)Wat[(size_t)i * d + j] * (double)Gt[j];
            dagg[i] = s2;
        }
    } else {
        for (int j = 0; j < d; ++j) dagg[j] = (double)Gt[j];
    }
    /* softmax backward */
    for (int64_t p = 0; p < deg; ++p)
        for (int i = 0; i < H; ++i) {
            double da = 0.0;
            for (int j = i * dk; j < (i + 1) * dk; ++j) da += dagg[j] * msg[p * d + j];
            dal[p * H + i] = da;
            sv[i] += al[p * H + i] * da;
        }
    for (int j = 0; j < d; ++j) dQt[j] = 0.0;
    for (int64_t p = 0; p < deg; ++p) {
        const int64_t e = c->a->eid[p0 + p];
        const int r = c->rel[e];
        const double cr = (double)c->mu[r] * c->att_scale;
        for (int i = 0; i < H; ++i) {
            const double alpha = al[p * H + i];
            const double da = alpha * (dal[p * H + i] - sv[i]);
            const double *kwe = kw + p * d + i * dk, *Qti = Qt + i * dk;
            for (int j = 0; j < dk; ++j) dQt[i * dk + j] += da * cr * kwe[j];
            double kq = 0.0;
            for (int j = 0; j < dk; ++j) kq += kwe[j] * Qti[j];
            c->AL[e * H + i] = alpha;
            c->DA[e * H + i] = da;
            c->KQ[e * H + i] = kq;
        }
    }
    return 0;
}

int oracle_hgt_backward(int64_t N, int64_t E, int32_t R, int32_t T, int32_t d, int32_t heads,
                        const int32_t *src, const int32_t *dst, const int32_t *rel,
                        const int32_t *ntype, const float *h, const float *Wk, const float *Wq,
                        const float *Wv, const float *Wa, const float *Watt, const float *Wmsg,
                        const float *mu, double att_scale, int32_t residual, int32_t a_linear,
                        const float *G, const uint8_t *node_mask, const uint8_t *rel_mask,
                        double *dh, double *dWk, double *dWq, double *dWv,
                        double *dWa, double *dWatt, double *dWmsg, double *dmu)
{
    if (check_coo(N, E, R, src, dst, rel) || T <= 0 || d <= 0 || d > 512 || heads <= 0 ||
        heads > 64 || d % heads)
        return -1;
    for (int64_t n = 0; n < N; ++n)
        if (ntype[n] < 0 || ntype[n] >= T) return -1;
    const int H = heads, dk = d / heads;
    const int full = !node_mask && !rel_mask;
    in_lists a;
    int rc = build_in_lists(N, E, dst, &a);
    if (rc) { free_in_lists(&a); return rc; }
    const size_t nd = (size_t)(N > 0 ? N : 1) * d, E1 = (size_t)(E > 0 ? E : 1), N1 = (size_t)(N > 0 ? N : 1);
    double *K = (double *)malloc(nd * sizeof(double));
    double *Q = (double *)malloc(nd * sizeof(double));
    double *V = (double *)malloc(nd * sizeof(double));
    double *dK = (double *)calloc(nd, sizeof(double));
    double *dQ = (double *)calloc(nd, sizeof(double));
    double *dV = (double *)calloc(nd, sizeof(double));
    double *agg = (double *)calloc(nd, sizeof(double));
    double *dagg = (double *)calloc(nd, sizeof(double));
    double *AL = (double *)malloc(E1 * H * sizeof(double));
    double *DA = (double *)malloc(E1 * H * sizeof(double));
    double *KQ = (double *)malloc(E1 * H * sizeof(double));
    uint8_t *need = (uint8_t *)calloc(N1, 1);
    int64_t *relptr = (int64_t *)calloc((size_t)R + 1, sizeof(int64_t));
    int64_t *reledge = (int64_t *)malloc(E1 * sizeof(int64_t));
    int64_t *outptr = (int64_t *)calloc(N1 + 1, sizeof(int64_t));
    int64_t *outedge = (int64_t *)malloc(E1 * sizeof(int64_t));
    int err = !K || !Q || !V || !dK || !dQ || !dV || !agg || !dagg || !AL || !DA || !KQ || !need ||
              !relptr || !reledge || !outptr || !outedge;
    if (!err) {
        memset(dh, 0, (size_t)N * d * sizeof(double));
        memset(dWk, 0, (size_t)T * d * d * sizeof(double));
        memset(dWq, 0, (size_t)T * d * d * sizeof(double));
        memset(dWv, 0, (size_t)T * d * d * sizeof(double));
        if (dWa) memset(dWa, 0, (size_t)T * d * d * sizeof(double));
        memset(dWatt, 0, (size_t)R * H * dk * dk * sizeof(double));
        memset(dWmsg, 0, (size_t)R * H * dk * dk * sizeof(double));
        memset(dmu, 0, (size_t)R * sizeof(double));
        for (int64_t e = 0; e < E; ++e) {
            const int want = full || (rel_mask && rel_mask[rel[e]]) ||
                             (node_mask && (node_mask[src[e]] || node_mask[dst[e]]));
            if (want) need[dst[e]] = 1;
        }
        if (node_mask)
            for (int64_t n = 0; n < N; ++n) if (node_mask[n]) need[n] = 1;   /* dQ of n */
        /* relations' edges and sources' out-edges, both in the global order */
        for (int64_t e = 0; e < E; ++e) { relptr[rel[e] + 1]++; outptr[src[e] + 1]++; }
        for (int r = 0; r < R; ++r) relptr[r + 1] += relptr[r];
        for (int64_t n = 0; n < N; ++n) outptr[n + 1] += outptr[n];
        int64_t *rf = (int64_t *)malloc((size_t)R * sizeof(int64_t));
        int64_t *of = (int64_t *)malloc(N1 * sizeof(int64_t));
        if (!rf || !of) {
            err = 1;
        } else {
            memcpy(rf, relptr, (size_t)R * sizeof(int64_t));
            memcpy(of, outptr, (size_t)N * sizeof(int64_t));
            for (int64_t p = 0; p < E; ++p) {
                const int64_t e = a.eid[p];
                reledge[rf[rel[e]]++] = e;
                outedge[of[src[e]]++] = e;
            }
        }
        free(rf); free(of);
    }
    if (!err) {   /* node-level K, Q, V */
#pragma omp parallel for schedule(static)
        for (int64_t n = 0; n < N; ++n) {
            double x[512];
            load_row(h, n, d, x);
            const size_t wo = (size_t)ntype[n] * d * d;
            vecmat(x, Wk + wo, d, d, 0, d, K + (size_t)n * d);
            vecmat(x, Wq + wo, d, d, 0, d, Q + (size_t)n * d);
            vecmat(x, Wv + wo, d, d, 0, d, V + (size_t)n * d);
        }
    }
    hgt_bwd_ctx c = {N, E, R, T, d, H, src, dst, rel, ntype, Wa, Watt, Wmsg, mu, G, att_scale, a_linear,
                     &a, K, Q, V, agg, dagg, dQ, AL, DA, KQ};
    /* stage A */
    if (!err) {
#pragma omp parallel reduction(| : err)
        {
            double *kw = NULL, *msg = NULL, *al = NULL, *dal = NULL;
            int64_t cap = 0;
#pragma omp for schedule(dynamic, 16)
            for (int64_t t = 0; t < N; ++t)
                if (need[t] && hgt_bwd_dst(&c, t, &kw, &msg, &al, &dal, &cap)) err = 1;
            free(kw); free(msg); free(al); free(dal);
        }
    }
    /* stage B: dWatt / dWmsg rows per (relation, head, row), dmu per relation,
     * dWa rows per (node type, row) */
    if (!err) {
        const int64_t n_att = (int64_t)R * H * dk, n_mu = R, n_wa = (full && a_linear && dWa) ? (int64_t)T * d : 0;
#pragma omp parallel for schedule(dynamic, 1)
        for (int64_t job = 0; job < n_att + n_mu + n_wa; ++job) {
            if (job < n_att) {
                const int r = (int)(job / (H * dk)), i = (int)(job / dk % H), j = (int)(job % dk);
                if (rel_mask && !rel_mask[r]) continue;
                const double cr = (double)mu[r] * att_scale;
                double *dWms = dWmsg + (((size_t)r * H + i) * dk + j) * dk;
                double *dWat = dWatt + (((size_t)r * H + i) * dk + j) * dk;
                for (int64_t q = relptr[r]; q < relptr[r + 1]; ++q) {
                    const int64_t e = reledge[q];
                    const double alpha = AL[e * H + i], da = DA[e * H + i];
                    const double Vs = V[(size_t)src[e] * d + i * dk + j], Ks = K[(size_t)src[e] * d + i * dk + j];
                    const double *dg = dagg + (size_t)dst[e] * d + i * dk, *Qti = Q + (size_t)dst[e] * d + i * dk;
                    for (int k = 0; k < dk; ++k) {
                        dWms[k] += Vs * alpha * dg[k];
                        dWat[k] += Ks * da * cr * Qti[k];
                    }
                }
            } else if (job < n_att + n_mu) {
                const int r = (int)(job - n_att);
                if (rel_mask && !rel_mask[r]) continue;
                for (int64_t q = relptr[r]; q < relptr[r + 1]; ++q) {
                    const int64_t e = reledge[q];
                    for (int i = 0; i < H; ++i) dmu[r] += DA[e * H + i] * att_scale * KQ[e * H + i];
                }
            } else {
                const int64_t w = job - n_att - n_mu;
                const int ty = (int)(w / d), i = (int)(w % d);
                double *row = dWa + ((size_t)ty * d + i) * d;
                for (int64_t t = 0; t < N; ++t) {
                    if (ntype[t] != ty) continue;
                    const double ai = agg[(size_t)t * d + i];
                    const float *Gt = G + (size_t)t * d;
                    for (int j = 0; j < d; ++j) row[j] += ai * (double)Gt[j];
                }
            }
        }
    }
    /* stage C: dK and dV per source over its out-edges */
    if (!err) {
#pragma omp parallel for schedule(dynamic, 64)
        for (int64_t sn = 0; sn < N; ++sn) {
            if (!full && !(node_mask && node_mask[sn])) continue;
            for (int64_t q = outptr[sn]; q < outptr[sn + 1]; ++q) {
                const int64_t e = outedge[q], t = dst[e];
                const int r = rel[e];
                const double cr = (double)mu[r] * att_scale;
                for (int i = 0; i < H; ++i) {
                    const double alpha = AL[e * H + i], da = DA[e * H + i];
                    const float *Wat = Watt + ((size_t)r * H + i) * dk * dk;
                    const float *Wms = Wmsg + ((size_t)r * H + i) * dk * dk;
                    const double *dg = dagg + (size_t)t * d + i * dk, *Qti = Q + (size_t)t * d + i * dk;
                    for (int j = 0; j < dk; ++j) {
                        double sv2 = 0.0, sk = 0.0;
                        for (int k = 0; k < dk; ++k) {
                            sv2 += alpha * dg[k] * (double)Wms[(size_t)j * dk + k];
                            sk += da * cr * Qti[k] * (double)Wat[(size_t)j * dk + k];
                        }
                        dV[(size_t)sn * d + i * dk + j] += sv2;
                        dK[(size_t)sn * d + i * dk + j] += sk;
                    }
                }
            }
        }
    }
    /* stage D: node-type weights (per type, projection and row) and dh (per node) */
    if (!err && full) {
#pragma omp parallel for schedule(dynamic, 1)
        for (int64_t job = 0; job < (int64_t)T * 3 * d; ++job) {
            const int ty = (int)(job / (3 * d)), m = (int)(job / d % 3), i = (int)(job % d);
            const double *dX = m == 0 ? dK : (m == 1 ? dQ : dV);
            double *row = (m == 0 ? dWk : (m == 1 ? dWq : dWv)) + ((size_t)ty * d + i) * d;
            for (int64_t n = 0; n < N; ++n) {
                if (ntype[n] != ty) continue;
                const double xi = (double)h[(size_t)n * d + i];
                for (int j = 0; j < d; ++j) row[j] += xi * dX[(size_t)n * d + j];
            }
        }
    }
    if (!err) {
#pragma omp parallel for schedule(static)
        for (int64_t n = 0; n < N; ++n) {
            if (node_mask && !node_mask[n]) continue;
            double *row = dh + (size_t)n * d;
            if (residual)
                for (int j = 0; j < d; ++j) row[j] += (double)G[(size_t)n * d + j];
            const size_t wo = (size_t)ntype[n] * d * d;
            const double *dx[3] = {dK + (size_t)n * d, dQ + (size_t)n * d, dV + (size_t)n * d};
            const float *Wx[3] = {Wk + wo, Wq + wo, Wv + wo};
            for (int m = 0; m < 3; ++m)
                for (int i = 0; i < d; ++i) {
                    double s2 = 0.0;
                    for (int j = 0; j < d; ++j) s2 += dx[m][j] * (double)Wx[m][(size_t)i * d + j];
                    row[i] += s2;
                }
        }
    }
    free(K); free(Q); free(V); free(dK); free(dQ); free(dV); free(agg); free(dagg);
    free(AL); free(DA); free(KQ); free(need); free(relptr); free(reledge); free(outptr); free(outedge);
    free_in_lists(&a);
    return err ? -3 : 0;
}

int oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
