// rgcn_backward.hip -- RGCN backward pass for the loss L = sum(out * G), the
// chain rule applied to the paper's RGCN equation (Section "Backward
// Propagation" generates it from the forward; here it is written out), for
// d_in = d_out in {32, 64, 128}.  With the pre-activation P and Gp = G * act'(P):
//   dS_seg = Gp_v W_r^T / c_{v,r}            per virtual segment (v, r)
//   dh_u   = sum over u's out-edges of dS_seg(e)  +  Gp_u W0^T
//   dW_r   = sum over r's segments of Sbar_seg^T Gp_v,  Sbar_seg = (1/c) sum_{u in seg} h_u
//   dW0    = sum_v h_v^T Gp_v
//
// Kernel sequence:
//   1. Gp = G masked by out > 0 (ReLU only).
//   2. dS by the typed GEMM (B = W_r^T, row scale 1/c) over the segments in
//      the by-relation order; dh = Gp W0^T by the typed GEMM (or zeros).
//   3. A source-major traversal over the out-edges (sorted by source, then
//      relation) gathers the dS rows and adds their sum to dh with one store
//      per source: the per-edge scatter becomes a gather.  Pieces of sources
//      with more than kChunkEdges out-edges leave their sums in slots that one
//      workgroup per such source adds in slot order (no atomics anywhere).
//   4. Sbar by the fused aggregate-first kernel's sums-only mode; dW_r and dW0
//      by outer-product MFMA chunks (K = segments or nodes) and ordered sums.
#include "rgnn_internal.h"

namespace rgnn {

namespace {

constexpr int kE = kChunkEdges, kDst = kMaxDstPerItem;
constexpr int kU = 4;   // dS rows per prefetch batch

__device__ __forceinline__ float4 ld4(const float *p) { return *reinterpret_cast<const float4 *>(p); }
__device__ __forceinline__ void st4(float *p, float4 v) { *reinterpret_cast<float4 *>(p) = v; }
__device__ __forceinline__ float4 zero4() { return make_float4(0.f, 0.f, 0.f, 0.f); }
__device__ __forceinline__ float4 add4(float4 a, float4 b) { return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w); }

// Gp = G where out > 0, else 0 (ReLU derivative from the forward output).
__global__ __launch_bounds__(256) void relu_mask_kernel(const float *G, const float *out, float *Gp, int64_t n4)
{
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n4) return;
    const float4 g = ld4(G + i * 4), o = ld4(out + i * 4);
    st4(Gp + i * 4, make_float4(o.x > 0.f ? g.x : 0.f, o.y > 0.f ? g.y : 0.f, o.z > 0.f ? g.z : 0.f,
                                o.w > 0.f ? g.w : 0.f));
}

struct RStage {
    int evs[kE];         // dS row (by-relation segment position) of each out-edge
    int enode[kE];       // item-local source of each out-edge
    int optr[kDst + 1];  // item-local first out-edge of each source
};

// dh_u += sum of the dS rows of u's out-edges; one group of D/4 lanes per
// out-edge work item (bundles of small sources or pieces of large ones).
template <int D>
__global__ __launch_bounds__(256) void rgcn_bwd_src_kernel(int64_t n_items, const Item *items,
                                                           const int32_t *item_slot,
                                                           const int32_t *out_ptr, const int32_t *out_vseg,
                                                           const float *dS, float *dh, float *part)
{
    constexpr int G = D / 4, GPB = 256 / G;
    __shared__ RStage stage[GPB];
    const int gl = threadIdx.x % G, gi = threadIdx.x / G;
    RStage &st = stage[gi];
    const int64_t item = (int64_t)blockIdx.x * GPB + gi;
    const bool valid = item < n_items;
    int n0 = 0, nn = 0, q0 = 0, nq = 0;
    bool split = false;   // a piece of a source whose out-edges span several items
    int slot = -1;
    if (valid) {
        const Item x = items[item];
        n0 = x.dst0; nn = x.dst1 - x.dst0; q0 = x.vs0; nq = x.vs1 - x.vs0;
        slot = item_slot[item];
        split = slot >= 0;
        for (int e = gl; e < nq; e += G) st.evs[e] = out_vseg[q0 + e];
        auto opos = [&](int jj) {
            const int q = out_ptr[n0 + jj];
            return (q < q0 ? q0 : (q > q0 + nq ? q0 + nq : q)) - q0;
        };
        for (int j = gl; j < nn; j += G) {
            const int a = opos(j), b = opos(j + 1);
            st.optr[j] = a;
            for (int e = a; e < b; ++e) st.enode[e] = j;
        }
        if (gl == 0) st.optr[nn] = nq;
    }
    __syncthreads();
    if (!valid || nq == 0) return;
    int j = 0;
    while (st.optr[j + 1] == st.optr[j]) ++j;   // first source with out-edges
    float4 acc = zero4();
    // ping-pong batches of (dS row, the source's dh row) per out-edge
    float4 Ad[kU], Ah[kU], Bd[kU], Bh[kU];
    auto load = [&](float4 (&Xd)[kU], float4 (&Xh)[kU], int b0) {
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int e = b0 + u < nq ? b0 + u : nq - 1;
            Xd[u] = ld4(dS + (size_t)st.evs[e] * D + gl * 4);
            Xh[u] = ld4(dh + (size_t)(n0 + st.enode[e]) * D + gl * 4);
        }
    };
    auto consume = [&](const float4 (&Xd)[kU], const float4 (&Xh)[kU], int b0) {
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int e = b0 + u;
            if (e < nq) {
                acc = add4(acc, Xd[u]);
                if (e + 1 == st.optr[j + 1]) {   // the source's last out-edge in this item
                    // a piece of a split source leaves its sum in its slot
                    if (split) st4(part + (size_t)slot * D + gl * 4, acc);
                    else st4(dh + (size_t)(n0 + j) * D + gl * 4, add4(Xh[u], acc));
                    acc = zero4();
                    ++j;
                    while (j < nn && st.optr[j + 1] == st.optr[j]) ++j;
                }
            }
        }
    };
    load(Ad, Ah, 0);
    __builtin_amdgcn_sched_barrier(0);
    for (int eb = 0; eb < nq; eb += 2 * kU) {
        load(Bd, Bh, eb + kU);
        __builtin_amdgcn_sched_barrier(0);
        consume(Ad, Ah, eb);
        load(Ad, Ah, eb + 2 * kU);
        __builtin_amdgcn_sched_barrier(0);
        consume(Bd, Bh, eb + kU);
    }
}

__global__ __launch_bounds__(256) void zero4_kernel(float *p, int64_t n4)
{
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < n4) st4(p + i * 4, zero4());
}

inline unsigned blocks_for(int64_t n, int per_block) { return (unsigned)((n + per_block - 1) / per_block); }
inline size_t pad256(size_t b) { return (b + 255) & ~size_t(255); }

struct RgcnBwdWs { float *Gp, *dS, *Sb, *partial, *part; };

size_t rgcn_bwd_layout(const rgnn_graph *g, int D, void *base, RgcnBwdWs *w)
{
    char *b = (char *)base;
    size_t off = 0;
    auto take = [&](size_t n) {
        float *p = b ? (float *)(b + off) : nullptr;
        off += pad256(n * sizeof(float));
        return p;
    };
    const size_t nchunks = (size_t)std::max<int64_t>(std::max(g->n_tiles_outer, g->n_tiles_nodes_outer), 1);
    RgcnBwdWs x{};
    x.Gp = take((size_t)std::max<int64_t>(g->N, 1) * D);   // masked gradient (ReLU)
    x.dS = take((size_t)std::max<int64_t>(g->V, 1) * D);
    x.Sb = take((size_t)std::max<int64_t>(g->V, 1) * D);
    x.partial = take(nchunks * D * D);
    x.part = take((size_t)std::max<int64_t>(g->n_oslots, 1) * D);
    if (w) *w = x;
    return off;
}

template <int D>
rgnn_status rgcn_backward_d(const rgnn_graph *g, const float *h, const float *W, const float *W0, int relu,
                            const float *out, const float *Gm, float *dh, float *dW, float *dW0, void *ws,
                            hipStream_t s)
{
    constexpr int G = D / 4;
    RgcnBwdWs w;
    rgcn_bwd_layout(g, D, ws, &w);
    rgnn_status st;
    hipError_t e;
    const float *Gp = Gm;
    if (relu && g->N > 0) {
        {
            LaunchScope ls("rgcn_bwd_mask", s);
            hipLaunchKernelGGL(relu_mask_kernel, dim3(blocks_for(g->N * D / 4, 256)), dim3(256), 0, s, Gm, out,
                               w.Gp, g->N * D / 4);
        }
        if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "relu_mask launch");
        Gp = w.Gp;
    }
    if (g->V > 0) {
        // dS = (Gp_v W_r^T) / c per segment, by-relation order
        GemmArgs ga;
        ga.split_bf16 = 1;
        ga.X = Gp; ga.ldx = D; ga.gather = g->dev.vsegdst_byrel;
        ga.W[0] = W; ga.trans_b = 1; ga.K = D; ga.Nc = D;
        ga.tiles = g->dev.tiles_vsegs; ga.ntiles = g->n_tiles_vsegs;
        ga.Y = w.dS; ga.ldy = D;
        ga.ep.row_scale = g->dev.invcnt_byrel;
        if ((st = launch_typed_gemm(ga, s)) != RGNN_OK) return st;
    }
    // dh = Gp W0^T (or zeros), then the relation terms gathered over out-edges
    if (W0) {
        GemmArgs ga;
        ga.split_bf16 = 1;
        ga.X = Gp; ga.ldx = D; ga.W[0] = W0; ga.trans_b = 1; ga.K = D; ga.Nc = D;
        ga.tiles = g->dev.tiles_all; ga.ntiles = g->n_tiles_all;
        ga.Y = dh; ga.ldy = D;
        if ((st = launch_typed_gemm(ga, s)) != RGNN_OK) return st;
    } else if (g->N > 0) {
        {
            LaunchScope ls("zero", s);
            hipLaunchKernelGGL(zero4_kernel, dim3(blocks_for(g->N * D / 4, 256)), dim3(256), 0, s, dh,
                               g->N * D / 4);
        }
        if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "zero launch");
    }
    if (g->n_oitems > 0) {
        {
            LaunchScope ls("rgcn_bwd_src", s);
            hipLaunchKernelGGL(rgcn_bwd_src_kernel<D>, dim3(blocks_for(g->n_oitems, 256 / G)), dim3(256), 0, s,
                               g->n_oitems, g->dev.oitems, g->dev.oitem_slot, g->dev.out_ptr, g->dev.out_vseg, w.dS,
                               dh, w.part);
        }
        if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "rgcn_bwd_src launch");
        if ((st = launch_src_merge(g, w.part, dh, D, s)) != RGNN_OK) return st;
    }
    // dW_r = sum over r's segments of Sbar^T Gp_v
    if (g->V > 0) {
        FusedArgs fa;
        fa.g = g; fa.h = h; fa.d_in = D; fa.d_out = D; fa.S = w.Sb;
        if ((st = launch_af_fused(fa, s)) != RGNN_OK) return st;
        if ((st = launch_outer_chunks(g->dev.tiles_outer, g->n_tiles_outer, g->dev.vsegdst_byrel, 0, w.Sb, D,
                                      Gp, D, w.partial, D, s)) != RGNN_OK)
            return st;
    }
    if ((st = launch_chunk_sum(w.partial, g->dev.rel_chunkptr, g->R, dW, D, s)) != RGNN_OK) return st;
    // dW0 = sum_v h_v^T Gp_v
    if (W0 && dW0) {
        if ((st = launch_outer_chunks(g->dev.tiles_nodes_outer, g->n_tiles_nodes_outer, nullptr, 0, h, D, Gp,
                                      D, w.partial, D, s)) != RGNN_OK)
            return st;
        if ((st = launch_chunk_sum(w.partial, g->dev.nodes_chunkptr, 1, dW0, D, s)) != RGNN_OK) return st;
    }
    return RGNN_OK;
}

}  // namespace

rgnn_status rgcn_backward_impl(const rgnn_graph *g, const float *h, const float *W, const float *W0,
                               int d_in, int d_out, int flags, const float *out, const float *Gm,
                               float *dh, float *dW, float *dW0, void *ws, size_t ws_bytes,
                               hipStream_t s, size_t *need)
{
    const int relu = (flags & RGNN_FLAG_RELU) ? 1 : 0;
    const size_t bytes = rgcn_bwd_layout(g, d_in, nullptr, nullptr);
    if (need) { *need = bytes; return RGNN_OK; }
    if (d_in != d_out || (d_in != 32 && d_in != 64 && d_in != 128))
        return fail(RGNN_EUNSUPPORTED, "RGCN backward supports d_in = d_out in {32, 64, 128}");
    if (relu && !out) return fail(RGNN_EINVAL, "RGCN backward with ReLU needs the forward output");
    if (!ws || ws_bytes < bytes)
        return fail(RGNN_EINVAL, "workspace too small: need " + std::to_string(bytes) + " bytes");
    if (d_in == 32) return rgcn_backward_d<32>(g, h, W, W0, relu, out, Gm, dh, dW, dW0, ws, s);
    if (d_in == 64) return rgcn_backward_d<64>(g, h, W, W0, relu, out, Gm, dh, dW, dW0, ws, s);
    return rgcn_backward_d<128>(g, h, W, W0, relu, out, Gm, dh, dW, dW0, ws, s);
}

}  // namespace rgnn
