// traverse.hip -- CSR edge traversal kernels of RGCN and RGAT for gfx950 (the
// paper's traversal template, Section "The GEMM Template and the Traversal
// Template", with the destination loop of its graph-semantic loop
// transformation and loop hoisting).
//
// Work decomposition.  In-edges are sorted by (dst, rel, src) and cut into
// virtual segments (runs of one (dst, rel) pair, at most kChunkEdges long).
// A host-built list of work items gives each group of D/4 lanes either a
// bundle of consecutive small destinations or a piece of one large
// destination, never more than kChunkEdges edges.  Each lane owns four
// consecutive features (one float4), so a gathered 256-byte row is one
// coalesced dwordx4 load per lane of the group.
//
// Each item runs in phases separated by workgroup barriers:
//   1. stage: the item's segment offsets, relations, destination terms and
//      edge indices are read in parallel by the group's lanes into LDS, so no
//      later load depends on another global load except the row gathers;
//   2. logits (RGAT transform-first): per edge, in parallel, from the
//      materialized source term and the segment's destination term;
//   3. softmax: per destination, max and sum by group reductions, turned into
//      edge weights in LDS (unnormalised for a piece of a split destination);
//   4. aggregate: the item's edges are streamed in order with kU gathered rows
//      in flight and the next batch prefetched, flushing at segment or
//      destination boundaries.
// Forward traversals use no atomics: results are bitwise reproducible.
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
__device__ __forceinline__ float4 relu4(float4 a)
{
    return make_float4(fmaxf(a.x, 0.f), fmaxf(a.y, 0.f), fmaxf(a.z, 0.f), fmaxf(a.w, 0.f));
}
__device__ __forceinline__ float4 zero4() { return make_float4(0.f, 0.f, 0.f, 0.f); }

__device__ __forceinline__ float leaky(float y, float slope) { return y > 0.f ? y : slope * y; }

constexpr int kE = kChunkEdges;        // edges per item, at most
constexpr int kDst = kMaxDstPerItem;   // destinations per item, at most
constexpr int kU = 8;                  // gathered rows per batch

struct TK {
    int64_t n_items;
    const Item *items;
    const int32_t *item_slot;
    const int32_t *dst_vsegptr, *vseg_ptr, *vseg_rel, *vseg_cnt;
    const int32_t *e2u;
    const float *h, *M, *wsp, *wtp;
    float *vatt;
    float slope;
    float *out, *saved, *partial;
    int relu;
};

TK make_tk(const TravArgs &a)
{
    const rgnn_graph *g = a.g;
    TK k{};
    k.n_items = g->n_items;
    k.items = g->dev.items; k.item_slot = g->dev.item_slot;
    k.dst_vsegptr = g->dev.dst_vsegptr; k.vseg_ptr = g->dev.vseg_ptr;
    k.vseg_rel = g->dev.vseg_rel; k.vseg_cnt = g->dev.vseg_cnt;
    k.e2u = g->dev.e2u;
    k.h = a.h; k.M = a.M; k.wsp = a.wsp; k.wtp = a.wtp; k.vatt = a.vatt;
    k.slope = a.slope;
    k.out = a.out; k.saved = a.saved; k.partial = a.partial;
    k.relu = a.relu;
    return k;
}

// Per-group LDS staging area.
template <int H>
struct Stage {
    int eidx[kE];          // per edge: message row (transform-first) or source node
    int evs[kE];           // per edge: item-local virtual segment
    float ew[kE * H];      // per edge: logit, then weight
    int dptr[kDst + 1];    // item-local edge offset of each destination's first edge
    int vptr[kE + 1];      // item-local edge offset of each virtual segment's first edge
    int vrel[kE];
    float vw[kE * H];      // per segment: destination attention term, or 1/c
};

struct ItemHdr {
    int dst0, nd, vs0, nv, e0, ne, slot;
    bool valid;
};

__device__ __forceinline__ ItemHdr item_header(const TK &k, int64_t item)
{
    ItemHdr it{0, 0, 0, 0, 0, 0, -1, false};
    if (item >= k.n_items) return it;
    const Item x = k.items[item];
    it.valid = true;
    it.dst0 = x.dst0; it.nd = x.dst1 - x.dst0;
    it.vs0 = x.vs0; it.nv = x.vs1 - x.vs0;
    it.e0 = k.vseg_ptr[x.vs0];
    it.ne = k.vseg_ptr[x.vs1] - it.e0;
    it.slot = k.item_slot[item];
    return it;
}

// Phase 1: segment and destination offsets, relations, per-segment terms and
// edge indices, all loaded lane-parallel.  MODE 0: vw = destination attention
// term (H per segment); MODE 1: vw = 1 / c_{v,r}.
template <int G, int H, int MODE>
__device__ __forceinline__ void stage_item(const TK &k, const ItemHdr &it, Stage<H> &st,
                                           const int32_t *eidx_src, int gl)
{
    if (!it.valid) return;
    for (int j = gl; j < it.nv; j += G) {
        const int a = k.vseg_ptr[it.vs0 + j] - it.e0, b = k.vseg_ptr[it.vs0 + j + 1] - it.e0;
        st.vptr[j] = a;
        st.vrel[j] = k.vseg_rel[it.vs0 + j];
        if (MODE == 0) {
#pragma unroll
            for (int hh = 0; hh < H; ++hh) st.vw[j * H + hh] = k.vatt[(size_t)(it.vs0 + j) * H + hh];
        } else {
            st.vw[j] = 1.f / (float)k.vseg_cnt[it.vs0 + j];
        }
        for (int e = a; e < b; ++e) st.evs[e] = j;
    }
    if (gl == 0) st.vptr[it.nv] = it.ne;
    for (int j = gl; j <= it.nd; j += G) {
        int vs = k.dst_vsegptr[it.dst0 + j];
        vs = vs < it.vs0 ? it.vs0 : (vs > it.vs0 + it.nv ? it.vs0 + it.nv : vs);
        st.dptr[j] = k.vseg_ptr[vs] - it.e0;
    }
    for (int e = gl; e < it.ne; e += G) st.eidx[e] = eidx_src[it.e0 + e];
}

// Phase 4 (destination flush): weighted sums of gathered rows, written per
// destination; pieces of split destinations write (max, sum, acc) partials.
template <int D, int H, bool SOFTMAX>
__device__ __forceinline__ void aggregate_item(const TK &k, const ItemHdr &it, const Stage<H> &st,
                                               const float *rows, int gl, int head, float pm, float ps)
{
    constexpr int REC = SOFTMAX ? 2 * H + D : 2 + D;
    constexpr int OFF = SOFTMAX ? 2 * H : 2;
    constexpr int LH = D / H / 4;
    if (!it.valid) return;
    int j = 0;
    float4 acc = zero4();
    auto flush = [&](int jj) {
        if (it.slot < 0) {
            const size_t v = (size_t)it.dst0 + jj;
            st4(k.out + v * D + gl * 4, k.relu ? relu4(acc) : acc);
        } else {
            float *pr = k.partial + (size_t)it.slot * REC;
            if (SOFTMAX && gl % LH == 0) { pr[head * 2] = pm; pr[head * 2 + 1] = ps; }
            st4(pr + OFF + gl * 4, acc);
        }
        acc = zero4();
    };
    if (it.ne > 0) {
        // Two row buffers in ping-pong: while one batch is consumed the other
        // is in flight.  Loads are unconditional (clamped to the last edge)
        // and no register copies rotate the buffers, so the compiler's waits
        // never drain the batch still in flight.
        float4 A[kU], B[kU];
        auto load = [&](float4 (&X)[kU], int base) {
#pragma unroll
            for (int u = 0; u < kU; ++u) {
                const int e = base + u < it.ne ? base + u : it.ne - 1;
                X[u] = ld4(rows + (size_t)st.eidx[e] * D + gl * 4);
            }
        };
        auto consume = [&](const float4 (&X)[kU], int base) {
#pragma unroll
            for (int u = 0; u < kU; ++u) {
                const int e = base + u;
                if (e < it.ne) {
                    while (e >= st.dptr[j + 1]) { flush(j); ++j; }
                    acc = lin4(acc, 1.f, X[u], st.ew[e * H + head]);
                }
            }
        };
        load(A, 0);
        __builtin_amdgcn_sched_barrier(0);
        for (int e0 = 0; e0 < it.ne; e0 += 2 * kU) {
            load(B, e0 + kU);
            __builtin_amdgcn_sched_barrier(0);
            consume(A, e0);
            load(A, e0 + 2 * kU);
            __builtin_amdgcn_sched_barrier(0);
            consume(B, e0 + kU);
        }
    }
    for (; j < it.nd; ++j) flush(j);
}

// ---------------------------------------------------------------- destination attention terms
// vatt[vs, k] = h_v . (W_r w_dst[r])_k for every virtual segment (v, r): the
// reordered destination term (Section "Linear Operator Reordering"), hoisted
// out of the edge loop to one evaluation per (dst, rel) segment.
// One group of D/4 lanes per kSegPerGroup consecutive segments, all loads of
// a group issued together.
constexpr int kSegPerGroup = 8;

template <int D, int H>
__global__ __launch_bounds__(256) void seg_attn_kernel(TK k, int64_t V, const int32_t *vseg_dst)
{
    constexpr int G = D / 4, GPB = 256 / G;
    constexpr int S = kSegPerGroup;
    const int gl = threadIdx.x % G;
    const int64_t vs0 = ((int64_t)blockIdx.x * GPB + threadIdx.x / G) * S;
    if (vs0 >= V) return;
    int v[S], r[S];
#pragma unroll
    for (int i = 0; i < S; ++i) {
        const int64_t vs = vs0 + i < V ? vs0 + i : V - 1;
        v[i] = vseg_dst[vs];
        r[i] = k.vseg_rel[vs];
    }
    // consecutive segments mostly share their destination: its row is loaded
    // once and reused
    float4 hv[S];
    hv[0] = ld4(k.h + (size_t)v[0] * D + gl * 4);
#pragma unroll
    for (int i = 1; i < S; ++i)
        hv[i] = v[i] == v[i - 1] ? hv[i - 1] : ld4(k.h + (size_t)v[i] * D + gl * 4);
    float4 wt[S][H];
#pragma unroll
    for (int i = 0; i < S; ++i)
#pragma unroll
        for (int hh = 0; hh < H; ++hh) wt[i][hh] = ld4(k.wtp + ((size_t)r[i] * H + hh) * D + gl * 4);
    // every lane ends with all S * H terms; lane l keeps terms l, l + G, ... and
    // stores them (coalesced: the group's terms are contiguous in vatt)
    constexpr int NM = (S * H + G - 1) / G;
    float mine[NM];
#pragma unroll
    for (int m = 0; m < NM; ++m) mine[m] = 0.f;
#pragma unroll
    for (int i = 0; i < S; ++i)
#pragma unroll
        for (int hh = 0; hh < H; ++hh) {
            const float p = gsum<G>(dot4(hv[i], wt[i][hh]));
            const int t = i * H + hh;
            if (gl == t % G) mine[t / G] = p;
        }
#pragma unroll
    for (int m = 0; m < NM; ++m) {
        const int t = m * G + gl;
        if (t < S * H && vs0 * H + t < V * H) k.vatt[(size_t)vs0 * H + t] = mine[m];
    }
}

// ---------------------------------------------------------------- RGAT, transform-first
// One pass per item with an online softmax per head: the source term of head
// k, M[p][k-cols] . w_src[r][k-cols], is formed from the gathered message row
// itself (a sum over the head's lanes), so the attention term rides in the
// message row's own read -- neither a per-pair source term (a random gather
// per edge) nor a logit staging pass is needed.  Each lane's four features
// belong to one head; the running maximum, denominator and weighted row sum of
// that head are rescaled as the maximum grows, and a destination's result is
// written when its last edge is consumed.  k.wsp holds w_src [R, D].
//
// ATT: the rows are attention+message rows (the proposal of Section
// "Discussion and Future Work": the attention term and the message in one
// tensor of width hidden + 1, here hidden + the heads, padded to a 16-byte
// multiple), written by the GEMM epilogue; each lane reads its head's source
// term from the row (same line as the row's tail) instead of forming the dot.
template <int D, int H, bool ATT>
__global__ __launch_bounds__(256) void rgat_tf1_kernel(TK k)
{
    constexpr int G = D / 4, GPB = 256 / G, LH = G / H;
    constexpr int LDM = ATT ? D + 4 * ((H + 3) / 4) : D;   // row stride of M
    constexpr int kU = 4;   // each entry carries two rows: half the batch of the other traversals
    __shared__ Stage<H> stage[GPB];
    const int gl = threadIdx.x % G, gi = threadIdx.x / G;
    const int head = gl / LH;
    Stage<H> &st = stage[gi];
    const ItemHdr it = item_header(k, (int64_t)blockIdx.x * GPB + gi);
    stage_item<G, H, 0>(k, it, st, k.e2u, gl);
    __syncthreads();
    if (!it.valid) return;
    int j = 0;
    float m = -INFINITY, s = 0.f;
    float4 acc = zero4();
    auto flush = [&](int jj) {
        const size_t v = (size_t)it.dst0 + jj;
        if (it.slot < 0) {
            st4(k.out + v * D + gl * 4, scale4(acc, s > 0.f ? 1.f / s : 0.f));
            if (k.saved && gl % LH == 0) {
                k.saved[(v * H + head) * 2] = s > 0.f ? m : 0.f;
                k.saved[(v * H + head) * 2 + 1] = s;
            }
        } else {
            float *pr = k.partial + (size_t)it.slot * (2 * H + D);
            if (gl % LH == 0) { pr[head * 2] = m; pr[head * 2 + 1] = s; }
            st4(pr + 2 * H + gl * 4, acc);
        }
        m = -INFINITY; s = 0.f; acc = zero4();
    };
    if (it.ne > 0) {
        // ping-pong batches of (message row, w_src row) per edge
        float4 A[kU], Aw[kU], B[kU], Bw[kU];
        auto load = [&](float4 (&X)[kU], float4 (&Xw)[kU], int base) {
#pragma unroll
            for (int u = 0; u < kU; ++u) {
                const int e = base + u < it.ne ? base + u : it.ne - 1;
                X[u] = ld4(k.M + (size_t)st.eidx[e] * LDM + gl * 4);
                if (ATT) Xw[u].x = k.M[(size_t)st.eidx[e] * LDM + D + head];
                else Xw[u] = ld4(k.wsp + (size_t)st.vrel[st.evs[e]] * D + gl * 4);
            }
        };
        auto consume = [&](const float4 (&X)[kU], const float4 (&Xw)[kU], int base) {
#pragma unroll
            for (int u = 0; u < kU; ++u) {
                const int e = base + u;
                const float src_term = ATT ? Xw[u].x : gsum<LH>(dot4(X[u], Xw[u]));
                if (e < it.ne) {
                    while (e >= st.dptr[j + 1]) { flush(j); ++j; }
                    const float z = leaky(src_term + st.vw[st.evs[e] * H + head], k.slope);
                    const float mn = fmaxf(m, z);
                    const float c1 = __expf(m - mn), c2 = __expf(z - mn);
                    s = s * c1 + c2;
                    acc = lin4(acc, c1, X[u], c2);
                    m = mn;
                }
            }
        };
        load(A, Aw, 0);
        __builtin_amdgcn_sched_barrier(0);
        for (int e0 = 0; e0 < it.ne; e0 += 2 * kU) {
            load(B, Bw, e0 + kU);
            __builtin_amdgcn_sched_barrier(0);
            consume(A, Aw, e0);
            load(A, Aw, e0 + 2 * kU);
            __builtin_amdgcn_sched_barrier(0);
            consume(B, Bw, e0 + kU);
        }
    }
    for (; j < it.nd; ++j) flush(j);
}

// ---------------------------------------------------------------- RGCN, transform-first
template <int D>
__global__ __launch_bounds__(256) void rgcn_tf_kernel(TK k)
{
    constexpr int G = D / 4, GPB = 256 / G;
    __shared__ Stage<1> stage[GPB];
    const int gl = threadIdx.x % G, gi = threadIdx.x / G;
    Stage<1> &st = stage[gi];
    const ItemHdr it = item_header(k, (int64_t)blockIdx.x * GPB + gi);
    stage_item<G, 1, 1>(k, it, st, k.e2u, gl);
    __syncthreads();
    if (it.valid)
        for (int e = gl; e < it.ne; e += G) st.ew[e] = st.vw[st.evs[e]];
    __syncthreads();
    aggregate_item<D, 1, false>(k, it, st, k.M, gl, 0, 0.f, 0.f);
}

// The same with the reordered vectors of every relation staged in LDS (when
// they fit) and each group taking SB batches of S consecutive segments: the
// workgroup's (destination, relation) pairs are staged in LDS with coalesced
// loads next to the vectors, and the next batch's destination rows are in
// flight while the current batch's dot products are formed.
constexpr int kSegBatches = 4;

// NT threads per workgroup: 256, or 1024 when the vectors of several heads
// take most of the LDS (one workgroup per CU then stages them once for four
// times the segments).
// GW: the vectors too many for LDS (hundreds of relations at d = 128) are read
// from global memory (L2-resident) with each batch's rows, four segments per
// batch.
constexpr int kSegPerGroupGW = 4;
template <int D, int H, int NT, bool GW = false>
__global__ __launch_bounds__(NT) void seg_attn_lds_kernel(TK k, int64_t V, const int32_t *vseg_dst, int R)
{
    constexpr int G = D / 4, GPB = NT / G;
    constexpr int S = GW ? kSegPerGroupGW : kSegPerGroup, SB = kSegBatches, SW = GPB * S * SB;
    extern __shared__ float4 wts[];   // [R, H, D / 4] (not GW)
    __shared__ int2 sidx[SW];         // (destination, relation) of the workgroup's segments
    const int gl = threadIdx.x % G, gi = threadIdx.x / G;
    const int64_t wbase = (int64_t)blockIdx.x * SW;
    if (!GW)
        for (int i = threadIdx.x; i < R * H * G; i += NT) wts[i] = ld4(k.wtp + (size_t)i * 4);
    for (int i = threadIdx.x; i < SW; i += NT) {
        const int64_t vs = wbase + i < V ? wbase + i : V - 1;
        sidx[i] = make_int2(vseg_dst[vs], k.vseg_rel[vs]);
    }
    __syncthreads();
    const int64_t base = wbase + (int64_t)gi * (S * SB);
    if (base >= V) return;
    int v[2][S], r[2][S];
    float4 hv[2][S];
    float4 wr[GW ? 2 : 1][GW ? S : 1][GW ? H : 1];
    auto idx = [&](int slot, int b) {
#pragma unroll
        for (int i = 0; i < S; ++i) {
            const int2 x = sidx[gi * S * SB + b * S + i];
            v[slot][i] = x.x;
            r[slot][i] = x.y;
        }
    };
    auto rows = [&](int slot) {
#pragma unroll
        for (int i = 0; i < S; ++i) hv[slot][i] = ld4(k.h + (size_t)v[slot][i] * D + gl * 4);
        if constexpr (GW) {
#pragma unroll
            for (int i = 0; i < S; ++i)
#pragma unroll
                for (int hh = 0; hh < H; ++hh)
                    wr[slot][i][hh] = ld4(k.wtp + ((size_t)r[slot][i] * H + hh) * D + gl * 4);
        }
    };
    constexpr int NM = (S * H + G - 1) / G;
    auto compute = [&](int slot, int b) {
        const int64_t vs0 = base + b * S;
        float mine[NM];
#pragma unroll
        for (int m = 0; m < NM; ++m) mine[m] = 0.f;
#pragma unroll
        for (int i = 0; i < S; ++i)
#pragma unroll
            for (int hh = 0; hh < H; ++hh) {
                float4 w;
                if constexpr (GW) w = wr[slot][i][hh];
                else w = wts[(r[slot][i] * H + hh) * G + gl];
                const float p = gsum<G>(dot4(hv[slot][i], w));
                const int t = i * H + hh;
                if (gl == t % G) mine[t / G] = p;
            }
#pragma unroll
        for (int m = 0; m < NM; ++m) {
            const int t = m * G + gl;
            if (t < S * H && vs0 * H + t < V * H) k.vatt[(size_t)vs0 * H + t] = mine[m];
        }
    };
    idx(0, 0);
    rows(0);
    idx(1, 1);
#pragma unroll
    for (int b = 0; b < SB; ++b) {
        const int cur = b & 1, nxt = cur ^ 1;
        if (b + 1 < SB) {
            if (base + (b + 1) * S < V) rows(nxt);
        }
        __builtin_amdgcn_sched_barrier(0);
        if (base + b * S < V) compute(cur, b);
        if (b + 2 < SB) idx(cur, b + 2);
    }
}

inline unsigned blocks_for(int64_t n, int per_block) { return (unsigned)((n + per_block - 1) / per_block); }

}  // namespace

rgnn_status launch_seg_attn(const TravArgs &a, hipStream_t s)
{
    if (a.g->V == 0) return RGNN_OK;
    TK k = make_tk(a);
    LaunchScope ls("seg_attn", s);
    const size_t wbytes = (size_t)a.g->R * a.heads * a.d * sizeof(float);
    if (wbytes <= 32768 && a.heads <= 2) {
        const unsigned nbl = blocks_for((a.g->V + kSegPerGroup * kSegBatches - 1) / (kSegPerGroup * kSegBatches),
                                        256 / (a.d / 4));
#define SAL(D, H) hipLaunchKernelGGL((seg_attn_lds_kernel<D, H, 256>), dim3(nbl), dim3(256), wbytes, s, k, \
                                     a.g->V, a.g->dev.vseg_dst, a.g->R)
        bool done = true;
        if (a.d == 32 && a.heads == 1) SAL(32, 1);
        else if (a.d == 32 && a.heads == 2) SAL(32, 2);
        else if (a.d == 64 && a.heads == 1) SAL(64, 1);
        else if (a.d == 64 && a.heads == 2) SAL(64, 2);
        else if (a.d == 128 && a.heads == 1) SAL(128, 1);
        else if (a.d == 128 && a.heads == 2) SAL(128, 2);
        else done = false;
#undef SAL
        if (done) {
            hipError_t e = hipGetLastError();
            return e == hipSuccess ? RGNN_OK : hip_fail(e, "seg_attn launch");
        }
    }
    // larger vector sets (several heads, d = 128): 1024-thread workgroups, one per CU
    const size_t sidx_bytes = (size_t)(1024 / (a.d / 4)) * kSegPerGroup * kSegBatches * sizeof(int2);
    if (wbytes + sidx_bytes <= 160 * 1024) {
        const unsigned nbl = blocks_for((a.g->V + kSegPerGroup * kSegBatches - 1) / (kSegPerGroup * kSegBatches),
                                        1024 / (a.d / 4));
        hipError_t ea = hipSuccess;
#define SAW(D, H)                                                                                          \
    do {                                                                                                   \
        ea = hipFuncSetAttribute((const void *)seg_attn_lds_kernel<D, H, 1024>,                            \
                                 hipFuncAttributeMaxDynamicSharedMemorySize, (int)wbytes);                 \
        if (ea == hipSuccess)                                                                              \
            hipLaunchKernelGGL((seg_attn_lds_kernel<D, H, 1024>), dim3(nbl), dim3(1024), wbytes, s, k, a.g->V, \
                               a.g->dev.vseg_dst, a.g->R);                                                 \
    } while (0)
        bool done = true;
        if (a.d == 32 && a.heads == 1) SAW(32, 1);
        else if (a.d == 32 && a.heads == 2) SAW(32, 2);
        else if (a.d == 64 && a.heads == 1) SAW(64, 1);
        else if (a.d == 64 && a.heads == 2) SAW(64, 2);
        else if (a.d == 64 && a.heads == 4) SAW(64, 4);
        else if (a.d == 128 && a.heads == 1) SAW(128, 1);
        else if (a.d == 128 && a.heads == 2) SAW(128, 2);
        else if (a.d == 128 && a.heads == 8) SAW(128, 8);   // (128, 4) would spill
        else done = false;
#undef SAW
        if (done) {
            if (ea != hipSuccess) return hip_fail(ea, "hipFuncSetAttribute (seg_attn LDS)");
            hipError_t e = hipGetLastError();
            return e == hipSuccess ? RGNN_OK : hip_fail(e, "seg_attn launch");
        }
    }
    if (a.heads <= 2) {   // batches pipelined per group, the vectors read with the rows
        constexpr int SPG = kSegPerGroupGW * kSegBatches;
        const unsigned nbg = blocks_for((a.g->V + SPG - 1) / SPG, 256 / (a.d / 4));
#define SAG(D, H) hipLaunchKernelGGL((seg_attn_lds_kernel<D, H, 256, true>), dim3(nbg), dim3(256), 0, s, k, \
                                     a.g->V, a.g->dev.vseg_dst, a.g->R)
        bool done = true;
        if (a.d == 32 && a.heads == 1) SAG(32, 1);
        else if (a.d == 32 && a.heads == 2) SAG(32, 2);
        else if (a.d == 64 && a.heads == 1) SAG(64, 1);
        else if (a.d == 64 && a.heads == 2) SAG(64, 2);
        else if (a.d == 128 && a.heads == 1) SAG(128, 1);
        else if (a.d == 128 && a.heads == 2) SAG(128, 2);
        else done = false;
#undef SAG
        if (done) {
            hipError_t e = hipGetLastError();
            return e == hipSuccess ? RGNN_OK : hip_fail(e, "seg_attn launch");
        }
    }
    const unsigned nb = blocks_for((a.g->V + kSegPerGroup - 1) / kSegPerGroup, 256 / (a.d / 4));
#define SA(D, H) hipLaunchKernelGGL((seg_attn_kernel<D, H>), dim3(nb), dim3(256), 0, s, k, a.g->V, \
                                    a.g->dev.vseg_dst)
    if (a.d == 32 && a.heads == 1) SA(32, 1);
    else if (a.d == 32 && a.heads == 2) SA(32, 2);
    else if (a.d == 64 && a.heads == 1) SA(64, 1);
    else if (a.d == 64 && a.heads == 2) SA(64, 2);
    else if (a.d == 64 && a.heads == 4) SA(64, 4);
    else if (a.d == 128 && a.heads == 1) SA(128, 1);
    else if (a.d == 128 && a.heads == 2) SA(128, 2);
    else if (a.d == 128 && a.heads == 4) SA(128, 4);
    else if (a.d == 128 && a.heads == 8) SA(128, 8);
    else return fail(RGNN_EUNSUPPORTED, "segment attention: unsupported (d, heads)");
#undef SA
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? RGNN_OK : hip_fail(e, "seg_attn launch");
}

rgnn_status launch_rgat_traverse_tf(const TravArgs &a, hipStream_t s)
{
    if (a.g->n_items == 0) return RGNN_OK;
    TK k = make_tk(a);
    LaunchScope ls("rgat_traverse_tf", s);
    const unsigned nb = blocks_for(a.g->n_items, 256 / (a.d / 4));
    if (!a.wsp && !a.att_in_row) return fail(RGNN_EINVAL, "RGAT traversal needs w_src");
#define RGAT_TF(D, H)                                                                        \
    do {                                                                                     \
        if (a.att_in_row) hipLaunchKernelGGL((rgat_tf1_kernel<D, H, true>), dim3(nb), dim3(256), 0, s, k); \
        else hipLaunchKernelGGL((rgat_tf1_kernel<D, H, false>), dim3(nb), dim3(256), 0, s, k);            \
    } while (0)
    if (a.d == 32 && a.heads == 1) RGAT_TF(32, 1);
    else if (a.d == 32 && a.heads == 2) RGAT_TF(32, 2);
    else if (a.d == 64 && a.heads == 1) RGAT_TF(64, 1);
    else if (a.d == 64 && a.heads == 2) RGAT_TF(64, 2);
    else if (a.d == 64 && a.heads == 4) RGAT_TF(64, 4);
    else if (a.d == 128 && a.heads == 1) RGAT_TF(128, 1);
    else if (a.d == 128 && a.heads == 2) RGAT_TF(128, 2);
    else if (a.d == 128 && a.heads == 4) RGAT_TF(128, 4);
    else if (a.d == 128 && a.heads == 8) RGAT_TF(128, 8);
    else return fail(RGNN_EUNSUPPORTED, "RGAT traversal: unsupported (d, heads)");
#undef RGAT_TF
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? RGNN_OK : hip_fail(e, "rgat_tf launch");
}

rgnn_status launch_rgcn_traverse_tf(const TravArgs &a, hipStream_t s)
{
    if (a.g->n_items == 0) return RGNN_OK;
    TK k = make_tk(a);
    LaunchScope ls("rgcn_traverse_tf", s);
    const unsigned nb = blocks_for(a.g->n_items, 256 / (a.d / 4));
    if (a.d == 32) hipLaunchKernelGGL((rgcn_tf_kernel<32>), dim3(nb), dim3(256), 0, s, k);
    else if (a.d == 64) hipLaunchKernelGGL((rgcn_tf_kernel<64>), dim3(nb), dim3(256), 0, s, k);
    else if (a.d == 128) hipLaunchKernelGGL((rgcn_tf_kernel<128>), dim3(nb), dim3(256), 0, s, k);
    else return fail(RGNN_EUNSUPPORTED, "RGCN traversal: d must be 32, 64 or 128");
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? RGNN_OK : hip_fail(e, "rgcn_tf launch");
}

}  // namespace rgnn
