// backward.hip -- RGAT backward pass (Section "Backward Propagation") for one
// head and d = 64, softmax over each destination's in-edges.
//
// With G = dL/dout, the forward's per-destination softmax maximum M_v and
// denominator Z_v, and the reordered vectors ws'_r = W_r w_src[r],
// wt'_r = W_r w_dst[r]:
//   alpha_e  = exp(leaky(h_u.ws'_r + h_v.wt'_r) - M_v) / Z_v
//   dalpha_e = G_v . (h_u W_r) = h_u . dS_{v,r},   dS_{v,r} = G_v W_r^T
//   s_v      = sum_e alpha_e dalpha_e
//   Y_e      = alpha_e (dalpha_e - s_v) leaky'(y_e)
//   dh_u    += alpha_e dS_{v,r} + Y_e ws'_r       (atomic scatter)
//   dh_v    += Y_e wt'_r
//   dW_r     = sum_seg (sum_e alpha_e h_u)^T G_v  +  dws'_r^T w_src[r] + dwt'_r^T w_dst[r]
//              with dws'_r = sum_e Y_e h_u,  dwt'_r = sum_e Y_e h_v
//   dw_src[r] = dws'_r W_r,   dw_dst[r] = dwt'_r W_r
// Kernel sequence: dS by the typed GEMM (B = W_r^T) over (dst, rel) segments;
// a traversal that recomputes the attention and scatters dh with float atomics
// after summing within each lane's segment (the paper's partial aggregation
// before atomics); an outer-product MFMA GEMM for dW over K-chunks of
// segments with a deterministic combine; and a per-relation finalize.
#include "rgnn_internal.h"

namespace rgnn {

namespace {

constexpr int D = 64, G = 16;
constexpr int kUnroll = 4;
constexpr int kCopies = 64;       // privatized copies of the per-relation accumulators
constexpr int kOuterRows = 2048;  // segments per outer-product K-chunk

__device__ __forceinline__ float4 ld4(const float *p) { return *reinterpret_cast<const float4 *>(p); }
__device__ __forceinline__ void st4(float *p, float4 v) { *reinterpret_cast<float4 *>(p) = v; }
__device__ __forceinline__ float dot4(float4 a, float4 b) { return a.x * b.x + a.y * b.y + a.z * b.z + a.w * b.w; }
__device__ __forceinline__ float4 lin4(float4 a, float s, float4 b, float t)
{
    return make_float4(a.x * s + b.x * t, a.y * s + b.y * t, a.z * s + b.z * t, a.w * s + b.w * t);
}
__device__ __forceinline__ void atomic_add4(float *p, float4 v)
{
    atomicAdd(p + 0, v.x); atomicAdd(p + 1, v.y); atomicAdd(p + 2, v.z); atomicAdd(p + 3, v.w);
}

template <int W>
__device__ __forceinline__ float gsum(float x)
{
#pragma unroll
    for (int off = W / 2; off > 0; off >>= 1) x += __shfl_xor(x, off, W);
    return x;
}

struct BK {
    int64_t n_items;
    const Item *items;
    const int32_t *item_slot, *dst_vsegptr, *vseg_ptr, *vseg_rel, *in_src;
    const float *h, *wsp, *wtp, *saved, *dS, *sv_in;
    float slope;
    float *Sa, *ssum, *dh, *acc_ws, *acc_wt;
    int copies, R;
};

// PHASE 0: every item; whole destinations run both passes, pieces of split
//          destinations run the first pass and leave their part of s_v.
// PHASE 1: pieces of split destinations only, second pass with the merged s_v.
template <int PHASE>
__global__ __launch_bounds__(256) void rgat_bwd_kernel(BK k)
{
    constexpr int GPB = 256 / G;
    const int gl = threadIdx.x % G;
    const int64_t item = (int64_t)blockIdx.x * GPB + threadIdx.x / G;
    if (item >= k.n_items) return;
    const int slot = k.item_slot[item];
    if (PHASE == 1 && slot < 0) return;
    const Item it = k.items[item];
    const int copy = blockIdx.x % k.copies;
    for (int v = it.dst0; v < it.dst1; ++v) {
        const int sb = max(it.vs0, k.dst_vsegptr[v]);
        const int se = min(it.vs1, k.dst_vsegptr[v + 1]);
        if (sb >= se) continue;
        const float4 hv = ld4(k.h + (size_t)v * D + gl * 4);
        const float Mv = k.saved[(size_t)v * 2];
        const float Zinv = 1.f / k.saved[(size_t)v * 2 + 1];
        float sacc = 0.f;
        if (PHASE == 0) {
            for (int vs = sb; vs < se; ++vs) {
                const int r = k.vseg_rel[vs];
                const float attt = gsum<G>(dot4(hv, ld4(k.wtp + (size_t)r * D + gl * 4)));
                const float4 ws = ld4(k.wsp + (size_t)r * D + gl * 4);
                const float4 ds = ld4(k.dS + (size_t)vs * D + gl * 4);
                float4 sa = make_float4(0.f, 0.f, 0.f, 0.f);
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
                        const float y = gsum<G>(dot4(row[u], ws)) + attt;
                        const float da = gsum<G>(dot4(row[u], ds));
                        if (e + u < e1) {
                            const float z = y > 0.f ? y : k.slope * y;
                            const float al = __expf(z - Mv) * Zinv;
                            sacc += al * da;
                            sa = lin4(sa, 1.f, row[u], al);
                        }
                    }
                }
                st4(k.Sa + (size_t)vs * D + gl * 4, sa);
            }
            if (slot >= 0) {
                if (gl == 0) k.ssum[slot] = sacc;
                continue;
            }
        }
        const float sv = PHASE == 0 ? sacc : k.sv_in[v];
        float4 dhv = make_float4(0.f, 0.f, 0.f, 0.f);
        for (int vs = sb; vs < se; ++vs) {
            const int r = k.vseg_rel[vs];
            const float4 wt = ld4(k.wtp + (size_t)r * D + gl * 4);
            const float attt = gsum<G>(dot4(hv, wt));
            const float4 ws = ld4(k.wsp + (size_t)r * D + gl * 4);
            const float4 ds = ld4(k.dS + (size_t)vs * D + gl * 4);
            float4 P = make_float4(0.f, 0.f, 0.f, 0.f);
            float ysum = 0.f;
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
                    const float y = gsum<G>(dot4(row[u], ws)) + attt;
                    const float da = gsum<G>(dot4(row[u], ds));
                    if (e + u < e1) {
                        const float z = y > 0.f ? y : k.slope * y;
                        const float al = __expf(z - Mv) * Zinv;
                        const float Y = al * (da - sv) * (y > 0.f ? 1.f : k.slope);
                        atomic_add4(k.dh + (size_t)u_[u] * D + gl * 4, lin4(ds, al, ws, Y));
                        P = lin4(P, 1.f, row[u], Y);
                        ysum += Y;
                    }
                }
            }
            atomic_add4(k.acc_ws + ((size_t)copy * k.R + r) * D + gl * 4, P);
            atomic_add4(k.acc_wt + ((size_t)copy * k.R + r) * D + gl * 4,
                        make_float4(hv.x * ysum, hv.y * ysum, hv.z * ysum, hv.w * ysum));
            dhv = lin4(dhv, 1.f, wt, ysum);
        }
        atomic_add4(k.dh + (size_t)v * D + gl * 4, dhv);
    }
}

__global__ __launch_bounds__(256) void merge_s_kernel(int64_t n_split, const int32_t *split_dst,
                                                      const int32_t *split_slotptr,
                                                      const float *ssum, float *sv)
{
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n_split) return;
    if (split_slotptr[i + 1] - split_slotptr[i] > kBigRange) return;
    float s = 0.f;
    for (int sl = split_slotptr[i]; sl < split_slotptr[i + 1]; ++sl) s += ssum[sl];
    sv[split_dst[i]] = s;
}

// One workgroup per split destination with many partials; thread sums are
// added in thread order.
__global__ __launch_bounds__(256) void merge_s_big_kernel(const int32_t *big_split,
                                                          const int32_t *split_dst,
                                                          const int32_t *split_slotptr,
                                                          const float *ssum, float *sv)
{
    __shared__ float part[256];
    const int i = big_split[blockIdx.x];
    float s = 0.f;
    for (int sl = split_slotptr[i] + (int)threadIdx.x; sl < split_slotptr[i + 1]; sl += 256) s += ssum[sl];
    part[threadIdx.x] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
        float t = 0.f;
        for (int j = 0; j < 256; ++j) t += part[j];
        sv[split_dst[i]] = t;
    }
}

typedef float floatx4 __attribute__((ext_vector_type(4)));

// partial[c] = sum over the chunk's segments of Sa[seg]^T (d_in) x G[dst(seg)] (d_out)
__global__ __launch_bounds__(256) void outer_gemm_kernel(const Tile *chunks, const int32_t *vseg_byrel,
                                                         const int32_t *vseg_dst, const float *Sa,
                                                         const float *Gm, float *partial)
{
    constexpr int KB = 64, P = 68;
    __shared__ float As[KB * P];
    __shared__ float Bs[KB * P];
    const Tile t = chunks[blockIdx.x];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int li = lane & 15, q = lane >> 4;
    floatx4 acc[4];
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) acc[cb] = floatx4{0.f, 0.f, 0.f, 0.f};
    for (int k0 = 0; k0 < t.rows; k0 += KB) {
        __syncthreads();
        // 64 rows x 64 floats of each operand: 16 float4 per row, 1024 float4 per operand
        for (int idx = tid; idx < KB * 16; idx += 256) {
            const int rr = idx >> 4, c4 = (idx & 15) * 4;
            float4 a = make_float4(0.f, 0.f, 0.f, 0.f), b = a;
            if (k0 + rr < t.rows) {
                const int vs = vseg_byrel[t.row0 + k0 + rr];
                a = ld4(Sa + (size_t)vs * D + c4);
                b = ld4(Gm + (size_t)vseg_dst[vs] * D + c4);
            }
            *reinterpret_cast<float4 *>(&As[rr * P + c4]) = a;
            *reinterpret_cast<float4 *>(&Bs[rr * P + c4]) = b;
        }
        __syncthreads();
#pragma unroll 4
        for (int kk = 0; kk < KB; kk += 4) {
            const float a = As[(kk + q) * P + w * 16 + li];
#pragma unroll
            for (int cb = 0; cb < 4; ++cb)
                acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, Bs[(kk + q) * P + cb * 16 + li], acc[cb], 0, 0, 0);
        }
    }
    float *out = partial + (size_t)blockIdx.x * D * D;
#pragma unroll
    for (int cb = 0; cb < 4; ++cb)
#pragma unroll
        for (int v = 0; v < 4; ++v) out[(size_t)(w * 16 + q * 4 + v) * D + cb * 16 + li] = acc[cb][v];
}

// Per relation r (one block): combine chunk partials in order, add the rank-1
// attention terms, and finish dw_src, dw_dst.
__global__ __launch_bounds__(256) void bwd_finalize_kernel(const float *partial, const int32_t *rel_chunkptr,
                                                           const float *acc_ws, const float *acc_wt,
                                                           int copies, int R, const float *W,
                                                           const float *w_src, const float *w_dst,
                                                           float *dW, float *dws, float *dwt)
{
    __shared__ float pws[D], pwt[D];
    const int r = blockIdx.x, tid = threadIdx.x;   // blockIdx.y: which 256 entries of dW_r
    if (tid < D) {
        float a = 0.f, b = 0.f;
        for (int c = 0; c < copies; ++c) {
            a += acc_ws[((size_t)c * R + r) * D + tid];
            b += acc_wt[((size_t)c * R + r) * D + tid];
        }
        pws[tid] = a; pwt[tid] = b;
    }
    __syncthreads();
    const int c0 = rel_chunkptr[r], c1 = rel_chunkptr[r + 1];
    {
        const int idx = blockIdx.y * 256 + tid;
        const int i = idx / D, j = idx % D;
        float s = 0.f;
        for (int c = c0; c < c1; ++c) s += partial[(size_t)c * D * D + idx];
        s += pws[i] * w_src[(size_t)r * D + j] + pwt[i] * w_dst[(size_t)r * D + j];
        dW[(size_t)r * D * D + idx] = s;
    }
    if (blockIdx.y == 0 && tid < D) {
        float a = 0.f, b = 0.f;
        for (int i = 0; i < D; ++i) {
            const float wij = W[((size_t)r * D + i) * D + tid];
            a += pws[i] * wij;
            b += pwt[i] * wij;
        }
        dws[(size_t)r * D + tid] = a;
        dwt[(size_t)r * D + tid] = b;
    }
}

__global__ void zero_kernel(float *p, int64_t n)
{
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < n) p[i] = 0.f;
}

inline size_t pad256(size_t b) { return (b + 255) & ~size_t(255); }

struct BwdWs { float *wsp, *wtp, *dS, *Sa, *ssum, *sv, *acc_ws, *acc_wt, *partial; };

size_t bwd_layout(const rgnn_graph *g, void *base, BwdWs *w)
{
    char *b = (char *)base;
    size_t off = 0;
    auto take = [&](size_t n) {
        float *p = b ? (float *)(b + off) : nullptr;
        off += pad256(n * sizeof(float));
        return p;
    };
    BwdWs x;
    x.wsp = take((size_t)g->R * D);
    x.wtp = take((size_t)g->R * D);
    x.dS = take((size_t)g->V * D);
    x.Sa = take((size_t)g->V * D);
    x.ssum = take((size_t)std::max<int64_t>(g->n_slots, 1));
    x.sv = take((size_t)std::max<int64_t>(g->N, 1));
    x.acc_ws = take((size_t)kCopies * g->R * D);
    x.acc_wt = take((size_t)kCopies * g->R * D);
    x.partial = take((size_t)std::max<int64_t>(g->n_tiles_outer, 1) * D * D);
    if (w) *w = x;
    return off;
}

hipError_t zero(float *p, int64_t n, hipStream_t s)
{
    if (n <= 0) return hipSuccess;
    LaunchScope ls("zero", s);
    hipLaunchKernelGGL(zero_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, p, n);
    return hipGetLastError();
}

}  // namespace

int bwd_outer_rows() { return kOuterRows; }

rgnn_status rgat_backward_impl(const rgnn_graph *g, const float *h, const float *W,
                               const float *w_src, const float *w_dst, int d_in, int d_out,
                               float slope, const float *saved, const float *Gm, float *dh,
                               float *dW, float *dws, float *dwt, void *ws, size_t ws_bytes,
                               hipStream_t s, size_t *need)
{
    const size_t bytes = bwd_layout(g, nullptr, nullptr);
    if (need) { *need = bytes; return RGNN_OK; }
    if (d_in != D || d_out != D) return fail(RGNN_EUNSUPPORTED, "RGAT backward supports d = 64");
    if (!ws || ws_bytes < bytes)
        return fail(RGNN_EINVAL, "workspace too small: need " + std::to_string(bytes) + " bytes");
    BwdWs w;
    bwd_layout(g, ws, &w);
    rgnn_status st;
    hipError_t e;
    if ((st = launch_reorder_vec(W, w_src, g->R, D, D, 1, w.wsp, s)) != RGNN_OK) return st;
    if ((st = launch_reorder_vec(W, w_dst, g->R, D, D, 1, w.wtp, s)) != RGNN_OK) return st;
    // dS_{v,r} = G_v W_r^T for every (dst, rel) segment
    GemmArgs ga;
    ga.X = Gm; ga.ldx = D; ga.gather = g->dev.vsegdst_byrel;
    ga.W[0] = W; ga.trans_b = 1; ga.K = D; ga.Nc = D;
    ga.tiles = g->dev.tiles_vsegs; ga.ntiles = g->n_tiles_vsegs;
    ga.Y = w.dS; ga.ldy = D; ga.scatter = g->dev.vseg_byrel;
    if ((st = launch_typed_gemm(ga, s)) != RGNN_OK) return st;
    if ((e = zero(dh, g->N * D, s)) != hipSuccess) return hip_fail(e, "zero launch");
    if ((e = zero(w.acc_ws, (int64_t)kCopies * g->R * D, s)) != hipSuccess) return hip_fail(e, "zero launch");
    if ((e = zero(w.acc_wt, (int64_t)kCopies * g->R * D, s)) != hipSuccess) return hip_fail(e, "zero launch");
    BK k{};
    k.n_items = g->n_items; k.items = g->dev.items; k.item_slot = g->dev.item_slot;
    k.dst_vsegptr = g->dev.dst_vsegptr; k.vseg_ptr = g->dev.vseg_ptr; k.vseg_rel = g->dev.vseg_rel;
    k.in_src = g->dev.in_src; k.h = h; k.wsp = w.wsp; k.wtp = w.wtp; k.saved = saved;
    k.dS = w.dS; k.sv_in = w.sv; k.slope = slope; k.Sa = w.Sa; k.ssum = w.ssum; k.dh = dh;
    k.acc_ws = w.acc_ws; k.acc_wt = w.acc_wt; k.copies = kCopies; k.R = g->R;
    if (g->n_items) {
        const dim3 grid((unsigned)((g->n_items + 15) / 16));
        {
            LaunchScope ls("rgat_bwd_traverse", s);
            hipLaunchKernelGGL((rgat_bwd_kernel<0>), dim3(grid.x, 1), dim3(256), 0, s, k);
        }
        if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "rgat_bwd launch");
        if (g->n_split) {
            {
                LaunchScope ls("rgat_bwd_merge_s", s);
                hipLaunchKernelGGL(merge_s_kernel, dim3((unsigned)((g->n_split + 255) / 256)), dim3(256), 0,
                                   s, g->n_split, g->dev.split_dst, g->dev.split_slotptr, w.ssum, w.sv);
            }
            if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "merge_s launch");
            if (g->n_big_split) {
                LaunchScope ls("rgat_bwd_merge_s_big", s);
                hipLaunchKernelGGL(merge_s_big_kernel, dim3((unsigned)g->n_big_split), dim3(256), 0, s,
                                   g->dev.big_split, g->dev.split_dst, g->dev.split_slotptr, w.ssum, w.sv);
            }
            if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "merge_s_big launch");
            {
                LaunchScope ls("rgat_bwd_traverse", s);
                hipLaunchKernelGGL((rgat_bwd_kernel<1>), dim3(grid.x, 1), dim3(256), 0, s, k);
            }
            if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "rgat_bwd launch");
        }
    }
    if (g->n_tiles_outer) {
        LaunchScope ls("outer_gemm", s);
        hipLaunchKernelGGL(outer_gemm_kernel, dim3((unsigned)g->n_tiles_outer), dim3(256), 0, s,
                           g->dev.tiles_outer, g->dev.vseg_byrel, g->dev.vseg_dst, w.Sa, Gm, w.partial);
    }
    if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "outer_gemm launch");
    {
        LaunchScope ls("rgat_bwd_finalize", s);
        hipLaunchKernelGGL(bwd_finalize_kernel, dim3((unsigned)g->R, D * D / 256), dim3(256), 0, s, w.partial,
                           g->dev.rel_chunkptr, w.acc_ws, w.acc_wt, kCopies, g->R, W, w_src, w_dst,
                           dW, dws, dwt);
    }
    if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "finalize launch");
    return RGNN_OK;
}

}  // namespace rgnn
