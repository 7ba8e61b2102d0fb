// traverse.hip -- CSR edge traversal kernels (the paper's traversal template,
// Section "The GEMM Template and the Traversal Template") for gfx950.
//
// Work decomposition.  In-edges are sorted by (dst, rel, src) and cut into
// virtual segments (runs of one (dst, rel) pair, at most kChunkEdges long).  A
// host-built list of work items assigns either a bundle of consecutive small
// destinations, or a piece of one large destination, to a group of D/4 lanes
// (16 lanes for d = 64).  Each lane owns four consecutive features (one float4),
// so one gathered 256-byte row is a single coalesced dwordx4 load of the group,
// and a wave serves 64/G items at once.  The destination-level loop is the
// paper's graph-semantic loop transformation (an edge loop rewritten as a
// destination loop over incoming edges); per-destination and per-segment terms
// are hoisted out of the edge loop (Section "Operator-Specific Schedule").
//
// Softmax.  Attention logits are folded into an online (running-max) softmax:
//   m' = max(m, z);  s' = s e^{m-m'} + e^{z-m'};  acc' = acc e^{m-m'} + row e^{z-m'}
// so every destination is finished in one pass.  Large destinations split over
// several items write (m, s, acc) partials that a merge kernel combines in a
// fixed order; no atomics are used and results are bitwise reproducible.
#include "rgnn_internal.h"

namespace rgnn {

namespace {

__device__ __forceinline__ float4 ld4(const float *p) { return *reinterpret_cast<const float4 *>(p); }
__device__ __forceinline__ void st4(float *p, float4 v) { *reinterpret_cast<float4 *>(p) = v; }
__device__ __forceinline__ float dot4(float4 a, float4 b) { return a.x * b.x + a.y * b.y + a.z * b.z + a.w * b.w; }
__device__ __forceinline__ float4 scale4(float4 a, float s) { return make_float4(a.x * s, a.y * s, a.z * s, a.w * s); }
__device__ __forceinline__ float4 add4(float4 a, float4 b) { return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w); }
// a * s + b * t
__device__ __forceinline__ float4 lin4(float4 a, float s, float4 b, float t)
{
    return make_float4(a.x * s + b.x * t, a.y * s + b.y * t, a.z * s + b.z * t, a.w * s + b.w * t);
}
__device__ __forceinline__ float4 relu4(float4 a)
{
    return make_float4(fmaxf(a.x, 0.f), fmaxf(a.y, 0.f), fmaxf(a.z, 0.f), fmaxf(a.w, 0.f));
}

// Sum over aligned groups of W lanes.
template <int W>
__device__ __forceinline__ float gsum(float x)
{
#pragma unroll
    for (int off = W / 2; off > 0; off >>= 1) x += __shfl_xor(x, off, W);
    return x;
}

__device__ __forceinline__ float leaky(float y, float slope) { return y > 0.f ? y : slope * y; }

// Online softmax step.
__device__ __forceinline__ void osm_step(float z, float4 row, float &m, float &s, float4 &acc)
{
    const float mn = fmaxf(m, z);
    const float c1 = __expf(m - mn), c2 = __expf(z - mn);
    s = s * c1 + c2;
    acc = lin4(acc, c1, row, c2);
    m = mn;
}

constexpr int kUnroll = 4;

struct TK {
    int64_t n_items;
    const Item *items;
    const int32_t *item_slot;
    const int32_t *dst_vsegptr, *vseg_ptr, *vseg_rel, *vseg_cnt;
    const int32_t *in_src, *e2u;
    const float *h, *M, *atts, *wsp, *wtp;
    float slope;
    float *out, *saved, *partial, *S, *vstat;
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
    k.in_src = g->dev.in_src; k.e2u = g->dev.e2u;
    k.h = a.h; k.M = a.M; k.atts = a.atts; k.wsp = a.wsp; k.wtp = a.wtp;
    k.slope = a.slope;
    k.out = a.out; k.saved = a.saved; k.partial = a.partial; k.S = a.S; k.vstat = a.vstat;
    k.relu = a.relu;
    return k;
}

// ---------------------------------------------------------------- RGAT, transform-first
// Messages M[p] = h_u W_r and source terms atts[p] = M[p] . w_src[r] exist once
// per unique (src, rel) pair (compact materialization); the destination term
// is h_v . (W_r w_dst[r]) (linear operator reordering), once per segment.
template <int D, int H>
__global__ __launch_bounds__(256) void rgat_tf_kernel(TK k)
{
    constexpr int G = D / 4, LH = D / H / 4, GPB = 256 / G;
    const int gl = threadIdx.x % G;
    const int64_t item = (int64_t)blockIdx.x * GPB + threadIdx.x / G;
    if (item >= k.n_items) return;
    const Item it = k.items[item];
    const int slot = k.item_slot[item];
    const int head = gl / LH;
    for (int v = it.dst0; v < it.dst1; ++v) {
        const int sb = max(it.vs0, k.dst_vsegptr[v]);
        const int se = min(it.vs1, k.dst_vsegptr[v + 1]);
        float m = -INFINITY, s = 0.f;
        float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
        if (sb < se) {
            const float4 hv = ld4(k.h + (size_t)v * D + gl * 4);
            for (int vs = sb; vs < se; ++vs) {
                const int r = k.vseg_rel[vs];
                float attt = 0.f;
#pragma unroll
                for (int hh = 0; hh < H; ++hh) {
                    const float p = gsum<G>(dot4(hv, ld4(k.wtp + ((size_t)r * H + hh) * D + gl * 4)));
                    if (hh == head) attt = p;
                }
                const int e0 = k.vseg_ptr[vs], e1 = k.vseg_ptr[vs + 1];
                for (int e = e0; e < e1; e += kUnroll) {
                    int p[kUnroll];
                    float4 row[kUnroll];
                    float at[kUnroll];
#pragma unroll
                    for (int u = 0; u < kUnroll; ++u) p[u] = k.e2u[min(e + u, e1 - 1)];
#pragma unroll
                    for (int u = 0; u < kUnroll; ++u) {
                        row[u] = ld4(k.M + (size_t)p[u] * D + gl * 4);
                        at[u] = k.atts[(size_t)p[u] * H + head];
                    }
#pragma unroll
                    for (int u = 0; u < kUnroll; ++u)
                        if (e + u < e1) osm_step(leaky(at[u] + attt, k.slope), row[u], m, s, acc);
                }
            }
        }
        if (slot < 0) {
            const float inv = s > 0.f ? 1.f / s : 0.f;
            st4(k.out + (size_t)v * D + gl * 4, scale4(acc, inv));
            if (k.saved && gl % LH == 0) {
                k.saved[((size_t)v * H + head) * 2] = sb < se ? m : 0.f;
                k.saved[((size_t)v * H + head) * 2 + 1] = s;
            }
        } else {
            float *pr = k.partial + (size_t)slot * (2 * H + D);
            if (gl % LH == 0) { pr[head * 2] = m; pr[head * 2 + 1] = s; }
            st4(pr + 2 * H + gl * 4, acc);
        }
    }
}

// ---------------------------------------------------------------- RGAT, aggregate-first
// Gathers h_u, computes both attention terms from reordered vectors
// (h_u . W_r w_src, h_v . W_r w_dst) and writes, per virtual segment, the
// exp-weighted feature sum S (relative to the segment's own maximum) and the
// segment's (max, sum).  W_r is applied afterwards by the typed GEMM, whose
// per-row scale exp(m_seg - M_v) / Z_v finishes the softmax.
template <int D>
__global__ __launch_bounds__(256) void rgat_af_kernel(TK k)
{
    constexpr int G = D / 4, GPB = 256 / G;
    const int gl = threadIdx.x % G;
    const int64_t item = (int64_t)blockIdx.x * GPB + threadIdx.x / G;
    if (item >= k.n_items) return;
    const Item it = k.items[item];
    for (int v = it.dst0; v < it.dst1; ++v) {
        const int sb = max(it.vs0, k.dst_vsegptr[v]);
        const int se = min(it.vs1, k.dst_vsegptr[v + 1]);
        if (sb >= se) continue;
        const float4 hv = ld4(k.h + (size_t)v * D + gl * 4);
        for (int vs = sb; vs < se; ++vs) {
            const int r = k.vseg_rel[vs];
            const float attt = gsum<G>(dot4(hv, ld4(k.wtp + (size_t)r * D + gl * 4)));
            const float4 ws = ld4(k.wsp + (size_t)r * D + gl * 4);
            float m = -INFINITY, s = 0.f;
            float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
            const int e0 = k.vseg_ptr[vs], e1 = k.vseg_ptr[vs + 1];
            for (int e = e0; e < e1; e += kUnroll) {
                int u_[kUnroll];
                float4 row[kUnroll];
#pragma unroll
                for (int u = 0; u < kUnroll; ++u) u_[u] = k.in_src[min(e + u, e1 - 1)];
#pragma unroll
                for (int u = 0; u < kUnroll; ++u) row[u] = ld4(k.h + (size_t)u_[u] * D + gl * 4);
#pragma unroll
                for (int u = 0; u < kUnroll; ++u) {
                    const float atts = gsum<G>(dot4(row[u], ws));
                    if (e + u < e1) osm_step(leaky(atts + attt, k.slope), row[u], m, s, acc);
                }
            }
            st4(k.S + (size_t)vs * D + gl * 4, acc);
            if (gl == 0) { k.vstat[(size_t)vs * 2] = m; k.vstat[(size_t)vs * 2 + 1] = s; }
        }
    }
}

// Per destination: M_v = max over its segments, Z_v = sum s_seg e^{m_seg - M_v}.
__global__ __launch_bounds__(256) void vseg_stats_kernel(int64_t N, const int32_t *dst_vsegptr,
                                                         const float *vstat, float *saved)
{
    const int64_t v = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (v >= N) return;
    const int b = dst_vsegptr[v], e = dst_vsegptr[v + 1];
    float M = -INFINITY;
    for (int i = b; i < e; ++i) M = fmaxf(M, vstat[(size_t)i * 2]);
    float Z = 0.f;
    for (int i = b; i < e; ++i) Z += vstat[(size_t)i * 2 + 1] * __expf(vstat[(size_t)i * 2] - M);
    saved[v * 2] = b < e ? M : 0.f;
    saved[v * 2 + 1] = Z;
}

// out_v (+)= sum of the transformed segment rows of v (then optional ReLU).
template <int D>
__global__ __launch_bounds__(256) void vseg_reduce_kernel(int64_t N, const int32_t *dst_vsegptr,
                                                          const float *T, float *out,
                                                          int accumulate, int relu)
{
    constexpr int G = D / 4, GPB = 256 / G;
    const int gl = threadIdx.x % G;
    const int64_t v = (int64_t)blockIdx.x * GPB + threadIdx.x / G;
    if (v >= N) return;
    const int b = dst_vsegptr[v], e = dst_vsegptr[v + 1];
    float4 acc = accumulate ? ld4(out + (size_t)v * D + gl * 4) : make_float4(0.f, 0.f, 0.f, 0.f);
    for (int i = b; i < e; ++i) acc = add4(acc, ld4(T + (size_t)i * D + gl * 4));
    st4(out + (size_t)v * D + gl * 4, relu ? relu4(acc) : acc);
}

// ---------------------------------------------------------------- RGCN
// transform-first: out_v = sum over segments of mean of M[pair] rows.
template <int D>
__global__ __launch_bounds__(256) void rgcn_tf_kernel(TK k)
{
    constexpr int G = D / 4, GPB = 256 / G;
    const int gl = threadIdx.x % G;
    const int64_t item = (int64_t)blockIdx.x * GPB + threadIdx.x / G;
    if (item >= k.n_items) return;
    const Item it = k.items[item];
    const int slot = k.item_slot[item];
    for (int v = it.dst0; v < it.dst1; ++v) {
        const int sb = max(it.vs0, k.dst_vsegptr[v]);
        const int se = min(it.vs1, k.dst_vsegptr[v + 1]);
        float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
        for (int vs = sb; vs < se; ++vs) {
            const float inv = 1.f / (float)k.vseg_cnt[vs];
            float4 loc = make_float4(0.f, 0.f, 0.f, 0.f);
            const int e0 = k.vseg_ptr[vs], e1 = k.vseg_ptr[vs + 1];
            for (int e = e0; e < e1; e += kUnroll) {
                int p[kUnroll];
                float4 row[kUnroll];
#pragma unroll
                for (int u = 0; u < kUnroll; ++u) p[u] = k.e2u[min(e + u, e1 - 1)];
#pragma unroll
                for (int u = 0; u < kUnroll; ++u) row[u] = ld4(k.M + (size_t)p[u] * D + gl * 4);
#pragma unroll
                for (int u = 0; u < kUnroll; ++u)
                    if (e + u < e1) loc = add4(loc, row[u]);
            }
            acc = lin4(acc, 1.f, loc, inv);
        }
        if (slot < 0) st4(k.out + (size_t)v * D + gl * 4, k.relu ? relu4(acc) : acc);
        else st4(k.partial + (size_t)slot * (2 + D) + 2 + gl * 4, acc);
    }
}

// aggregate-first: S[vseg] = mean of h_u rows over the vseg's segment.
template <int D>
__global__ __launch_bounds__(256) void rgcn_af_kernel(TK k)
{
    constexpr int G = D / 4, GPB = 256 / G;
    const int gl = threadIdx.x % G;
    const int64_t item = (int64_t)blockIdx.x * GPB + threadIdx.x / G;
    if (item >= k.n_items) return;
    const Item it = k.items[item];
    for (int vs = it.vs0; vs < it.vs1; ++vs) {
        const float inv = 1.f / (float)k.vseg_cnt[vs];
        float4 loc = make_float4(0.f, 0.f, 0.f, 0.f);
        const int e0 = k.vseg_ptr[vs], e1 = k.vseg_ptr[vs + 1];
        for (int e = e0; e < e1; e += kUnroll) {
            int u_[kUnroll];
            float4 row[kUnroll];
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) u_[u] = k.in_src[min(e + u, e1 - 1)];
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) row[u] = ld4(k.h + (size_t)u_[u] * D + gl * 4);
#pragma unroll
            for (int u = 0; u < kUnroll; ++u)
                if (e + u < e1) loc = add4(loc, row[u]);
        }
        st4(k.S + (size_t)vs * D + gl * 4, scale4(loc, inv));
    }
}

// ---------------------------------------------------------------- merges
// Combine the partials of destinations split over several items, in slot
// order.  softmax: partial = (m, s) per head then acc[D]; else acc only.
template <int D, int H, bool SOFTMAX>
__global__ __launch_bounds__(256) void merge_kernel(int64_t n_split, const int32_t *split_dst,
                                                    const int32_t *split_slotptr,
                                                    const float *partial, float *out,
                                                    float *saved, int relu)
{
    constexpr int G = D / 4, GPB = 256 / G, LH = D / H / 4;
    constexpr int REC = SOFTMAX ? 2 * H + D : 2 + D;
    constexpr int OFF = SOFTMAX ? 2 * H : 2;
    const int gl = threadIdx.x % G;
    const int64_t i = (int64_t)blockIdx.x * GPB + threadIdx.x / G;
    if (i >= n_split) return;
    const int v = split_dst[i];
    const int b = split_slotptr[i], e = split_slotptr[i + 1];
    const int head = gl / LH;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    if (SOFTMAX) {
        float M = -INFINITY;
        for (int sl = b; sl < e; ++sl) M = fmaxf(M, partial[(size_t)sl * REC + head * 2]);
        float Z = 0.f;
        for (int sl = b; sl < e; ++sl) {
            const float *pr = partial + (size_t)sl * REC;
            const float c = __expf(pr[head * 2] - M);
            Z += pr[head * 2 + 1] * c;
            acc = lin4(acc, 1.f, ld4(pr + OFF + gl * 4), c);
        }
        acc = scale4(acc, Z > 0.f ? 1.f / Z : 0.f);
        if (saved && gl % LH == 0) {
            saved[((size_t)v * H + head) * 2] = M;
            saved[((size_t)v * H + head) * 2 + 1] = Z;
        }
    } else {
        for (int sl = b; sl < e; ++sl) acc = add4(acc, ld4(partial + (size_t)sl * REC + OFF + gl * 4));
    }
    st4(out + (size_t)v * D + gl * 4, relu ? relu4(acc) : acc);
}

__global__ void fill_kernel(float *p, int64_t n, float v)
{
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < n) p[i] = v;
}

__global__ void relu_kernel(float *p, int64_t n)
{
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < n) p[i] = fmaxf(p[i], 0.f);
}

__global__ void add_kernel(float *out, const float *a, const float *b, int64_t n)
{
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < n) out[i] = a[i] + b[i];
}

// Reordered attention vectors: out[r, k, i] = sum_{j in head k} W[r, i, j] v[r, j].
__global__ __launch_bounds__(256) void reorder_vec_kernel(const float *W, const float *v, int R,
                                                          int d_in, int d_out, int heads,
                                                          float *out)
{
    const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;   // (r, k, i)
    if (idx >= (int64_t)R * heads * d_in) return;
    const int i = (int)(idx % d_in);
    const int k = (int)((idx / d_in) % heads);
    const int r = (int)(idx / ((int64_t)d_in * heads));
    const int dh = d_out / heads;
    const float *Wr = W + ((size_t)r * d_in + i) * d_out + k * dh;
    const float *vr = v + (size_t)r * d_out + k * dh;
    float s = 0.f;
    for (int j = 0; j < dh; ++j) s += Wr[j] * vr[j];
    out[idx] = s;
}

inline unsigned blocks_for(int64_t n, int per_block) { return (unsigned)((n + per_block - 1) / per_block); }

hipError_t last() { return hipGetLastError(); }

}  // namespace

rgnn_status launch_rgat_traverse_tf(const TravArgs &a, hipStream_t s)
{
    if (a.g->n_items == 0) return RGNN_OK;
    TK k = make_tk(a);
    LaunchScope ls("rgat_traverse_tf", s);
    const unsigned nb = blocks_for(a.g->n_items, 256 / (a.d / 4));
#define RGAT_TF(D, H) hipLaunchKernelGGL((rgat_tf_kernel<D, H>), dim3(nb), dim3(256), 0, s, k)
    if (a.d == 64 && a.heads == 1) RGAT_TF(64, 1);
    else if (a.d == 64 && a.heads == 2) RGAT_TF(64, 2);
    else if (a.d == 64 && a.heads == 4) RGAT_TF(64, 4);
    else if (a.d == 128 && a.heads == 1) RGAT_TF(128, 1);
    else if (a.d == 128 && a.heads == 2) RGAT_TF(128, 2);
    else if (a.d == 128 && a.heads == 4) RGAT_TF(128, 4);
    else if (a.d == 128 && a.heads == 8) RGAT_TF(128, 8);
    else return fail(RGNN_EUNSUPPORTED, "RGAT traversal: unsupported (d, heads)");
#undef RGAT_TF
    hipError_t e = last();
    return e == hipSuccess ? RGNN_OK : hip_fail(e, "rgat_tf launch");
}

rgnn_status launch_rgat_traverse_af(const TravArgs &a, hipStream_t s)
{
    if (a.g->n_items == 0) return RGNN_OK;
    TK k = make_tk(a);
    LaunchScope ls("rgat_traverse_af", s);
    const unsigned nb = blocks_for(a.g->n_items, 256 / (a.d / 4));
    if (a.heads != 1) return fail(RGNN_EUNSUPPORTED, "aggregate-first RGAT needs heads == 1");
    if (a.d == 64) hipLaunchKernelGGL((rgat_af_kernel<64>), dim3(nb), dim3(256), 0, s, k);
    else if (a.d == 128) hipLaunchKernelGGL((rgat_af_kernel<128>), dim3(nb), dim3(256), 0, s, k);
    else return fail(RGNN_EUNSUPPORTED, "RGAT traversal: d must be 64 or 128");
    hipError_t e = last();
    return e == hipSuccess ? RGNN_OK : hip_fail(e, "rgat_af launch");
}

rgnn_status launch_rgcn_traverse_tf(const TravArgs &a, hipStream_t s)
{
    if (a.g->n_items == 0) return RGNN_OK;
    TK k = make_tk(a);
    LaunchScope ls("rgcn_traverse_tf", s);
    const unsigned nb = blocks_for(a.g->n_items, 256 / (a.d / 4));
    if (a.d == 64) hipLaunchKernelGGL((rgcn_tf_kernel<64>), dim3(nb), dim3(256), 0, s, k);
    else if (a.d == 128) hipLaunchKernelGGL((rgcn_tf_kernel<128>), dim3(nb), dim3(256), 0, s, k);
    else return fail(RGNN_EUNSUPPORTED, "RGCN traversal: d must be 64 or 128");
    hipError_t e = last();
    return e == hipSuccess ? RGNN_OK : hip_fail(e, "rgcn_tf launch");
}

rgnn_status launch_rgcn_traverse_af(const TravArgs &a, hipStream_t s)
{
    if (a.g->n_items == 0) return RGNN_OK;
    TK k = make_tk(a);
    LaunchScope ls("rgcn_traverse_af", s);
    const unsigned nb = blocks_for(a.g->n_items, 256 / (a.d / 4));
    if (a.d == 64) hipLaunchKernelGGL((rgcn_af_kernel<64>), dim3(nb), dim3(256), 0, s, k);
    else if (a.d == 128) hipLaunchKernelGGL((rgcn_af_kernel<128>), dim3(nb), dim3(256), 0, s, k);
    else return fail(RGNN_EUNSUPPORTED, "RGCN traversal: d must be 64 or 128");
    hipError_t e = last();
    return e == hipSuccess ? RGNN_OK : hip_fail(e, "rgcn_af launch");
}

rgnn_status launch_merge_partials(const TravArgs &a, int softmax, hipStream_t s)
{
    const rgnn_graph *g = a.g;
    if (g->n_split == 0) return RGNN_OK;
    LaunchScope ls("merge_partials", s);
    const unsigned nb = blocks_for(g->n_split, 256 / (a.d / 4));
    const int32_t *sd = g->dev.split_dst, *sp = g->dev.split_slotptr;
#define MERGE(D, H, SM) hipLaunchKernelGGL((merge_kernel<D, H, SM>), dim3(nb), dim3(256), 0, s, \
                                           g->n_split, sd, sp, a.partial, a.out, a.saved, a.relu)
    if (!softmax) {
        if (a.d == 64) MERGE(64, 1, false);
        else if (a.d == 128) MERGE(128, 1, false);
        else return fail(RGNN_EUNSUPPORTED, "merge: d must be 64 or 128");
    } else if (a.d == 64 && a.heads == 1) MERGE(64, 1, true);
    else if (a.d == 64 && a.heads == 2) MERGE(64, 2, true);
    else if (a.d == 64 && a.heads == 4) MERGE(64, 4, true);
    else if (a.d == 128 && a.heads == 1) MERGE(128, 1, true);
    else if (a.d == 128 && a.heads == 2) MERGE(128, 2, true);
    else if (a.d == 128 && a.heads == 4) MERGE(128, 4, true);
    else if (a.d == 128 && a.heads == 8) MERGE(128, 8, true);
    else return fail(RGNN_EUNSUPPORTED, "merge: unsupported (d, heads)");
#undef MERGE
    hipError_t e = last();
    return e == hipSuccess ? RGNN_OK : hip_fail(e, "merge launch");
}

rgnn_status launch_vseg_stats(const TravArgs &a, hipStream_t s)
{
    const rgnn_graph *g = a.g;
    if (g->N == 0) return RGNN_OK;
    LaunchScope ls("vseg_stats", s);
    hipLaunchKernelGGL(vseg_stats_kernel, dim3(blocks_for(g->N, 256)), dim3(256), 0, s, g->N,
                       g->dev.dst_vsegptr, a.vstat, a.saved);
    hipError_t e = last();
    return e == hipSuccess ? RGNN_OK : hip_fail(e, "vseg_stats launch");
}

rgnn_status launch_vseg_reduce(const rgnn_graph *g, const float *T, int d, float *out,
                               int accumulate, int relu, hipStream_t s)
{
    if (g->N == 0) return RGNN_OK;
    LaunchScope ls("vseg_reduce", s);
    const unsigned nb = blocks_for(g->N, 256 / (d / 4));
    if (d == 64)
        hipLaunchKernelGGL((vseg_reduce_kernel<64>), dim3(nb), dim3(256), 0, s, g->N,
                           g->dev.dst_vsegptr, T, out, accumulate, relu);
    else if (d == 128)
        hipLaunchKernelGGL((vseg_reduce_kernel<128>), dim3(nb), dim3(256), 0, s, g->N,
                           g->dev.dst_vsegptr, T, out, accumulate, relu);
    else return fail(RGNN_EUNSUPPORTED, "reduce: d must be 64 or 128");
    hipError_t e = last();
    return e == hipSuccess ? RGNN_OK : hip_fail(e, "vseg_reduce launch");
}

rgnn_status launch_fill(float *p, int64_t n, float v, hipStream_t s)
{
    if (n == 0) return RGNN_OK;
    LaunchScope ls("fill", s);
    hipLaunchKernelGGL(fill_kernel, dim3(blocks_for(n, 256)), dim3(256), 0, s, p, n, v);
    hipError_t e = last();
    return e == hipSuccess ? RGNN_OK : hip_fail(e, "fill launch");
}

rgnn_status launch_relu(float *p, int64_t n, hipStream_t s)
{
    if (n == 0) return RGNN_OK;
    LaunchScope ls("relu", s);
    hipLaunchKernelGGL(relu_kernel, dim3(blocks_for(n, 256)), dim3(256), 0, s, p, n);
    hipError_t e = last();
    return e == hipSuccess ? RGNN_OK : hip_fail(e, "relu launch");
}

rgnn_status launch_add(float *out, const float *a, const float *b, int64_t n, hipStream_t s)
{
    if (n == 0) return RGNN_OK;
    LaunchScope ls("add", s);
    hipLaunchKernelGGL(add_kernel, dim3(blocks_for(n, 256)), dim3(256), 0, s, out, a, b, n);
    hipError_t e = last();
    return e == hipSuccess ? RGNN_OK : hip_fail(e, "add launch");
}

rgnn_status launch_reorder_vec(const float *W, const float *v, int R, int d_in, int d_out,
                               int heads, float *out, hipStream_t s)
{
    const int64_t n = (int64_t)R * heads * d_in;
    LaunchScope ls("reorder_vec", s);
    hipLaunchKernelGGL(reorder_vec_kernel, dim3(blocks_for(n, 256)), dim3(256), 0, s, W, v, R,
                       d_in, d_out, heads, out);
    hipError_t e = last();
    return e == hipSuccess ? RGNN_OK : hip_fail(e, "reorder_vec launch");
}

}  // namespace rgnn
