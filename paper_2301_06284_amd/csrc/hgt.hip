// hgt.hip -- HGT edge traversal for d = heads x d_k in {32, 64, 128}.
//
// Keys and values of every node come from node-typed GEMMs (K|V stored side
// by side, 512 bytes per node at d = 64) and are gathered once per edge.
// Both per-relation head matrices are moved to the destination side by linear
// operator reordering (Section "Linear Operator Reordering"):
//   a_e,i = (K_s,i Watt[r,i]) . Q_t,i  =  K_s,i . (Q_t,i Watt[r,i]^T)
//   sum_e alpha_e,i (V_s,i Wmsg[r,i])  =  (sum_e alpha_e,i V_s,i) Wmsg[r,i]
// The reordered query of every (destination, relation) segment, with the
// prior mu[r] and the attention scale folded in, is one typed GEMM over the
// segments (weights built by hgt_qp_weights_kernel); the traversal then only
// dots each key row with its segment's query row.  Wmsg is applied once per
// segment to the attention-weighted value sum, from LDS (shared by a
// 1024-thread workgroup) when it fits.
//
// Work items are those of the RGAT traversal (at most kChunkEdges edges: a
// bundle of small destinations or a piece of a large one), one per group of
// d / 4 lanes; lane l holds features 4l..4l+3, so head i is lanes
// [i*LH, (i+1)*LH) with LH = d_k / 4.  Each item first stages its edge
// sources and segment / destination boundaries in LDS, then streams the
// K|V rows of its edges, kU at a time with the next kU in flight; each
// segment's query row is loaded once, while the segment before it runs.
#include "rgnn_internal.h"
#include "wave_ops.h"

namespace rgnn {

namespace {

__device__ __forceinline__ float4 ld4(const float *p) { return *reinterpret_cast<const float4 *>(p); }
__device__ __forceinline__ void st4(float *p, float4 v) { *reinterpret_cast<float4 *>(p) = v; }
__device__ __forceinline__ float dot4(float4 a, float4 b) { return a.x * b.x + a.y * b.y + a.z * b.z + a.w * b.w; }
__device__ __forceinline__ float4 scale4(float4 a, float s) { return make_float4(a.x * s, a.y * s, a.z * s, a.w * s); }
__device__ __forceinline__ float4 lin4(float4 a, float s, float4 b, float t)
{
    return make_float4(a.x * s + b.x * t, a.y * s + b.y * t, a.z * s + b.z * t, a.w * s + b.w * t);
}
__device__ __forceinline__ float4 add4(float4 a, float4 b) { return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w); }
__device__ __forceinline__ float4 zero4() { return make_float4(0.f, 0.f, 0.f, 0.f); }

constexpr int kE = kChunkEdges, kDst = kMaxDstPerItem;
constexpr int kU = 2;                    // gathered K|V rows per batch

// Launch shape at width D: a group of D/4 lanes per work item; 1024-lane
// workgroups (512 at d = 32, whose 128 item stages would not fit in LDS).
template <int D>
struct HS {
    static constexpr int G = D / 4;
    static constexpr int NTH = D == 32 ? 512 : 1024;
    static constexpr int GPB = NTH / G;
};

template <bool FQ>
struct HStage {
    int eidx[kE];          // source node of each edge
    int vptr[kE + 1];      // item-local edge offset of each virtual segment
    int vrel[kE];
    int dptr[kDst + 1];    // item-local edge offset of each destination
    int vdst[FQ ? kE : 1]; // destination of each virtual segment (queries formed in the kernel)
};

struct HK {
    int64_t n_items;
    const Item *items;
    const int32_t *item_slot, *dst_vsegptr, *vseg_ptr, *vseg_rel, *vseg_dst, *in_src;
    const float *KV, *QP, *Wmsg;
    const float *Q, *Watt, *mu;   // queries formed in the kernel: Q [N, d], Watt, mu, scale
    float scale;
    int R;
    float *agg, *partial;
    float *saved;          // [N, H, 2] per destination and head (max, sum), or NULL
};

// Value of lane jj of this lane's head (LH aligned lanes).  A DPP quad
// broadcast would serve LH = 4 without the LDS crossbar, but it lets the LDS
// matrix rows of several steps be hoisted ahead of their FMAs and the 1024-lane
// launch bound then spills; ds_bpermute keeps one step live at a time.
template <int G>
__device__ __forceinline__ float head_bcast(float v, int jj, int base)
{
    return __shfl(v, base + jj, G);
}

// y[4 values of this lane] = x_head (1 x dk) . Mat (dk x dk), Mat row-major,
// with x_head distributed over the head's LH lanes (4 values each).
// ROLLED: a loop instead of LH unrolled steps (one code copy where several
// call sites are inlined into the unrolled edge loop).
template <int LH, int G, bool ROLLED = false>
__device__ __forceinline__ float4 head_vecmat(float4 x, const float *Mt, int gl)
{
    constexpr int DK = LH * 4;
    const int base = (gl / LH) * LH;     // first lane of this head within the group
    const int c0 = 4 * (gl % LH);
    float4 y = zero4();
#pragma unroll(ROLLED ? 1 : LH)
    for (int jj = 0; jj < LH; ++jj) {
        const float x0 = head_bcast<G>(x.x, jj, base), x1 = head_bcast<G>(x.y, jj, base);
        const float x2 = head_bcast<G>(x.z, jj, base), x3 = head_bcast<G>(x.w, jj, base);
        y = lin4(y, 1.f, ld4(Mt + (4 * jj + 0) * DK + c0), x0);
        y = lin4(y, 1.f, ld4(Mt + (4 * jj + 1) * DK + c0), x1);
        y = lin4(y, 1.f, ld4(Mt + (4 * jj + 2) * DK + c0), x2);
        y = lin4(y, 1.f, ld4(Mt + (4 * jj + 3) * DK + c0), x3);
        __builtin_amdgcn_sched_barrier(0);   // bound the live LDS rows to one step
    }
    return y;
}

// FQ: the reordered query of each segment, Q_t,i (mu[r] scale Watt[r, i]^T),
// is formed in the kernel at the segment's first edge from LDS-resident
// blocks (requires LDSW), with the next segment's Q row already in flight,
// instead of being read from a materialized [V, d] array.
template <int D, int H, bool LDSW, bool FQ>
__global__ __launch_bounds__(HS<D>::NTH) void hgt_kernel(HK k)
{
    static_assert(!FQ || LDSW, "kernel-formed queries keep both weight sets in LDS");
    constexpr int G = HS<D>::G, GPB = HS<D>::GPB, kBlock = HS<D>::NTH;
    constexpr int DK = D / H, LH = DK / 4;
    constexpr int MAT = H * DK * DK;            // floats per relation per matrix
    extern __shared__ float4 smem4[];
    float *smem = reinterpret_cast<float *>(smem4);
    const int nW = LDSW ? k.R * MAT : 0;
    const int nQ = FQ ? k.R * MAT : 0;
    HStage<FQ> *stages = reinterpret_cast<HStage<FQ> *>(smem + nW + nQ);
    const float *Wmsg = k.Wmsg;
    if (LDSW) {
        const int n4 = k.R * MAT / 4;
        for (int i = threadIdx.x; i < n4; i += kBlock) smem4[i] = reinterpret_cast<const float4 *>(k.Wmsg)[i];
        Wmsg = smem;
    }
    float *Wq = smem + nW;   // [R][H][j][n] = mu[r] scale Watt[r, i][n][j]
    if (FQ) {
        for (int idx = threadIdx.x; idx < nQ; idx += kBlock) {
            const int r = idx / MAT, rem = idx % MAT;
            const int i = rem / (DK * DK), j = rem / DK % DK, n = rem % DK;
            Wq[idx] = k.mu[r] * k.scale * k.Watt[(((size_t)r * H + i) * DK + n) * DK + j];
        }
    }
    const int gl = threadIdx.x % G, gi = threadIdx.x / G;
    HStage<FQ> &st = stages[gi];
    const int64_t item = (int64_t)blockIdx.x * GPB + gi;
    const bool valid = item < k.n_items;
    int dst0 = 0, nd = 0, vs0 = 0, nv = 0, e0 = 0, ne = 0, slot = -1;
    if (valid) {
        const Item x = k.items[item];
        dst0 = x.dst0; nd = x.dst1 - x.dst0; vs0 = x.vs0; nv = x.vs1 - x.vs0;
        e0 = k.vseg_ptr[x.vs0]; ne = k.vseg_ptr[x.vs1] - e0;
        slot = k.item_slot[item];
        for (int j = gl; j < nv; j += G) {
            const int a = k.vseg_ptr[vs0 + j] - e0;
            st.vptr[j] = a;
            st.vrel[j] = k.vseg_rel[vs0 + j];
            if (FQ) st.vdst[j] = k.vseg_dst[vs0 + j];
        }
        if (gl == 0) st.vptr[nv] = ne;
        auto dst_edge = [&](int jj) {
            int vs = k.dst_vsegptr[dst0 + jj];
            vs = vs < vs0 ? vs0 : (vs > vs0 + nv ? vs0 + nv : vs);
            return k.vseg_ptr[vs] - e0;
        };
        for (int j = gl; j < nd; j += G) st.dptr[j] = dst_edge(j);
        if (gl == 0) st.dptr[nd] = ne;
        for (int e = gl; e < ne; e += G) st.eidx[e] = k.in_src[e0 + e];
    }
    __syncthreads();
    if (!valid) return;

    const int head = gl / LH;
    float m = -INFINITY, s = 0.f;
    float4 agg = zero4(), vacc = zero4();
    auto flush = [&](int jj) {
        if (slot < 0) {
            st4(k.agg + (size_t)(dst0 + jj) * D + gl * 4, scale4(agg, s > 0.f ? 1.f / s : 0.f));
            if (k.saved && gl % LH == 0)
                *reinterpret_cast<float2 *>(k.saved + ((size_t)(dst0 + jj) * H + head) * 2) =
                    make_float2(s > 0.f ? m : 0.f, s);
        } else {
            float *pr = k.partial + (size_t)slot * (2 * H + D);
            if (gl % LH == 0) { pr[head * 2] = m; pr[head * 2 + 1] = s; }
            st4(pr + 2 * H + gl * 4, agg);
        }
        m = -INFINITY; s = 0.f; agg = zero4();
    };
    int j = 0, jv = 0;
    while (j < nd && st.dptr[j + 1] == st.dptr[j]) { flush(j); ++j; }
    // qcur: FQ, the Q row of segment jv's destination; otherwise segment jv's
    // reordered query row, loaded one segment ahead.  qp: segment jv's query.
    float4 qcur = zero4(), qp = zero4();
    if (ne > 0) qcur = FQ ? ld4(k.Q + (size_t)st.vdst[0] * D + gl * 4) : ld4(k.QP + (size_t)vs0 * D + gl * 4);
    if (ne > 0) {
        // Ping-pong batches: batch A is consumed while batch B is in flight.
        // Each edge brings its K|V row; each segment's query row is read once,
        // at the segment before it.
        float4 Ak[kU], Av[kU], Bk[kU], Bv[kU];
        auto load = [&](float4 (&Xk)[kU], float4 (&Xv)[kU], int base) {
#pragma unroll
            for (int u = 0; u < kU; ++u) {
                const int e = base + u < ne ? base + u : ne - 1;
                const size_t row = (size_t)st.eidx[e] * (2 * D);
                Xk[u] = ld4(k.KV + row + gl * 4);
                Xv[u] = ld4(k.KV + row + D + gl * 4);
            }
        };
        auto consume = [&](const float4 (&Xk)[kU], const float4 (&Xv)[kU], int base) {
#pragma unroll
            for (int u = 0; u < kU; ++u) {
                const int e = base + u;
                if (e < ne) {
                    if (e == st.vptr[jv]) {   // first edge of segment jv: its query
                        if (FQ) {
                            qp = head_vecmat<LH, G, true>(qcur, Wq + (size_t)st.vrel[jv] * MAT + (size_t)head * DK * DK, gl);
                            if (jv + 1 < nv && st.vdst[jv + 1] != st.vdst[jv])
                                qcur = ld4(k.Q + (size_t)st.vdst[jv + 1] * D + gl * 4);
                        } else {
                            qp = qcur;
                            if (jv + 1 < nv) qcur = ld4(k.QP + (size_t)(vs0 + jv + 1) * D + gl * 4);
                        }
                    }
                    const float a = gsum<LH>(dot4(Xk[u], qp));
                    const float mn = fmaxf(m, a);
                    const float c1 = __expf(m - mn), c2 = __expf(a - mn);
                    s = s * c1 + c2;
                    vacc = lin4(vacc, c1, Xv[u], c2);
                    agg = scale4(agg, c1);
                    m = mn;
                    if (e + 1 == st.vptr[jv + 1]) {
                        const size_t off = (size_t)st.vrel[jv] * MAT + (size_t)head * DK * DK;
                        agg = add4(agg, head_vecmat<LH, G>(vacc, Wmsg + off, gl));
                        vacc = zero4();
                        ++jv;
                        if (e + 1 == st.dptr[j + 1]) {
                            flush(j);
                            ++j;
                            while (j < nd && st.dptr[j + 1] == st.dptr[j]) { flush(j); ++j; }
                        }
                    }
                }
            }
        };
        load(Ak, Av, 0);
        __builtin_amdgcn_sched_barrier(0);
        for (int eb = 0; eb < ne; eb += 2 * kU) {
            load(Bk, Bv, eb + kU);
            __builtin_amdgcn_sched_barrier(0);
            consume(Ak, Av, eb);
            load(Ak, Av, eb + 2 * kU);
            __builtin_amdgcn_sched_barrier(0);
            consume(Bk, Bv, eb + kU);
        }
    }
    while (j < nd) { flush(j); ++j; }
}

template <int D, bool FQ>
size_t stage_bytes() { return (size_t)HS<D>::GPB * sizeof(HStage<FQ>); }

size_t weight_bytes(int D, int R, int heads)
{
    const int dk = D / heads;
    return (size_t)R * heads * dk * dk * sizeof(float);
}

// Wqp[r][j][n] = mu[r] * scale * Watt[r, i][n - i dk][j - i dk] when j and n
// both fall in head i's columns, else 0.
__global__ void hgt_qp_weights_kernel(const float *Watt, const float *mu, float scale, int R, int D,
                                      int heads, float *Wqp)
{
    const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (idx >= (int64_t)R * D * D) return;
    const int r = (int)(idx / (D * D)), j = (int)(idx / D % D), n = (int)(idx % D);
    const int dk = D / heads, i = j / dk;
    float v = 0.f;
    if (n / dk == i)
        v = mu[r] * scale * Watt[(((size_t)r * heads + i) * dk + (n - i * dk)) * dk + (j - i * dk)];
    Wqp[idx] = v;
}

// Wc[r][j][n] = sum_k Wq[t][j][k] Wqp[r][k][n], t = rel_dsttype[r]: only the
// k of n's head block contribute (Wqp[r] is block-diagonal), so each entry is
// a dk-term product of a Wq row piece with a row of Watt[r, i].
__global__ void hgt_qp_fold_kernel(const float *Wq, const float *Watt, const float *mu, float scale,
                                   const int32_t *rel_dsttype, int R, int D, int heads, float *Wc)
{
    const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (idx >= (int64_t)R * D * D) return;
    const int r = (int)(idx / (D * D)), j = (int)(idx / D % D), n = (int)(idx % D);
    const int dk = D / heads, i = n / dk;
    const float *wq = Wq + ((size_t)rel_dsttype[r] * D + j) * D + i * dk;
    const float *wa = Watt + (((size_t)r * heads + i) * dk + (n - i * dk)) * dk;
    float acc = 0.f;
    for (int k = 0; k < dk; ++k) acc = fmaf(wq[k], wa[k], acc);
    Wc[idx] = mu[r] * scale * acc;
}

template <int D, int H>
hipError_t launch_hgt_shape(const HK &k, int64_t n_items, int R, hipStream_t s)
{
    const size_t wb = weight_bytes(D, R, H);
    const unsigned nb = (unsigned)((n_items + HS<D>::GPB - 1) / HS<D>::GPB);
    hipError_t e;
#define HGT_LAUNCH(LDSW, FQ, LDS)                                                                          \
    do {                                                                                                   \
        e = hipFuncSetAttribute((const void *)hgt_kernel<D, H, LDSW, FQ>,                                  \
                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)(LDS));                   \
        if (e == hipSuccess)                                                                               \
            hipLaunchKernelGGL((hgt_kernel<D, H, LDSW, FQ>), dim3(nb), dim3(HS<D>::NTH), (LDS), s, k);     \
    } while (0)
    if (!k.QP) {   // queries formed in the kernel (the caller checked that both weight sets fit)
        if constexpr (D == 128) HGT_LAUNCH(true, true, (stage_bytes<D, true>() + 2 * wb));
        else e = hipErrorInvalidValue;
    } else if (wb + stage_bytes<D, false>() <= 160 * 1024) {
        HGT_LAUNCH(true, false, (stage_bytes<D, false>() + wb));
    } else {
        HGT_LAUNCH(false, false, (stage_bytes<D, false>()));
    }
#undef HGT_LAUNCH
    return e;
}

template <int D>
bool fused_query_fits(int R, int heads)
{
    return stage_bytes<D, true>() + 2 * weight_bytes(D, R, heads) <= 160 * 1024;
}

}  // namespace

rgnn_status launch_hgt_traverse(const HgtArgs &a, hipStream_t s)
{
    const rgnn_graph *g = a.g;
    if (g->n_items == 0) return RGNN_OK;
    HK k{};
    k.n_items = g->n_items; k.items = g->dev.items; k.item_slot = g->dev.item_slot;
    k.dst_vsegptr = g->dev.dst_vsegptr; k.vseg_ptr = g->dev.vseg_ptr;
    k.vseg_rel = g->dev.vseg_rel; k.vseg_dst = g->dev.vseg_dst; k.in_src = g->dev.in_src;
    k.KV = a.KV; k.QP = a.QP; k.Wmsg = a.Wmsg;
    k.Q = a.Q; k.Watt = a.Watt; k.mu = a.mu; k.scale = a.scale;
    if (!a.QP && !(a.Q && a.Watt && a.mu && hgt_fused_query_fits(g->R, a.d, a.heads)))
        return fail(RGNN_EINVAL, "HGT traversal without segment queries needs Q, Watt, mu and LDS room");
    k.R = g->R; k.agg = a.agg; k.partial = a.partial; k.saved = a.saved;
    LaunchScope ls("hgt_traverse", s);
    hipError_t e;
    const int64_t n = g->n_items;
    const int R = g->R;
    if (a.d == 32 && a.heads == 1) e = launch_hgt_shape<32, 1>(k, n, R, s);
    else if (a.d == 32 && a.heads == 2) e = launch_hgt_shape<32, 2>(k, n, R, s);
    else if (a.d == 64 && a.heads == 1) e = launch_hgt_shape<64, 1>(k, n, R, s);
    else if (a.d == 64 && a.heads == 2) e = launch_hgt_shape<64, 2>(k, n, R, s);
    else if (a.d == 64 && a.heads == 4) e = launch_hgt_shape<64, 4>(k, n, R, s);
    else if (a.d == 128 && a.heads == 1) e = launch_hgt_shape<128, 1>(k, n, R, s);
    else if (a.d == 128 && a.heads == 2) e = launch_hgt_shape<128, 2>(k, n, R, s);
    else if (a.d == 128 && a.heads == 4) e = launch_hgt_shape<128, 4>(k, n, R, s);
    else if (a.d == 128 && a.heads == 8) e = launch_hgt_shape<128, 8>(k, n, R, s);
    else return fail(RGNN_EUNSUPPORTED, "HGT traversal: unsupported (d, heads)");
    if (e != hipSuccess) return hip_fail(e, "hipFuncSetAttribute (HGT LDS)");
    e = hipGetLastError();
    return e == hipSuccess ? RGNN_OK : hip_fail(e, "hgt traversal launch");
}

bool hgt_fused_query_fits(int R, int d, int heads)
{
    // instantiated at d = 128 only, the width where it beats the segment-query GEMM
    return d == 128 && fused_query_fits<128>(R, heads);
}

rgnn_status launch_hgt_qp_weights(const float *Watt, const float *mu, float scale, int R, int d,
                                  int heads, float *Wqp, hipStream_t s)
{
    if (d != 32 && d != 64 && d != 128) return fail(RGNN_EUNSUPPORTED, "HGT supports d = 32, 64, 128");
    const int64_t n = (int64_t)R * d * d;
    if (n == 0) return RGNN_OK;
    LaunchScope ls("hgt_qp_weights", s);
    hipLaunchKernelGGL(hgt_qp_weights_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, Watt, mu, scale,
                       R, d, heads, Wqp);
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? RGNN_OK : hip_fail(e, "hgt_qp_weights launch");
}

rgnn_status launch_hgt_qp_fold(const float *Wq, const float *Watt, const float *mu, float scale,
                               const int32_t *rel_dsttype, int R, int d, int heads, float *Wc, hipStream_t s)
{
    if (d != 32 && d != 64 && d != 128) return fail(RGNN_EUNSUPPORTED, "HGT supports d = 32, 64, 128");
    const int64_t n = (int64_t)R * d * d;
    if (n == 0) return RGNN_OK;
    LaunchScope ls("hgt_qp_weights", s);
    hipLaunchKernelGGL(hgt_qp_fold_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, Wq, Watt, mu, scale,
                       rel_dsttype, R, d, heads, Wc);
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? RGNN_OK : hip_fail(e, "hgt_qp_fold launch");
}

}  // namespace rgnn
