// hgt.hip -- HGT edge traversal for d = 64 (heads x d_k = 64).
//
// Keys and values of every node come from one node-typed GEMM (K|V stored
// side by side, 512 bytes per node at d = 64) and are gathered once per edge.
// Both per-relation head matrices are moved to the destination side by linear
// operator reordering (Section "Linear Operator Reordering"):
//   a_e,i = (K_s,i Watt[r,i]) . Q_t,i  =  K_s,i . (Watt[r,i] Q_t,i^T)
//   sum_e alpha_e,i (V_s,i Wmsg[r,i])  =  (sum_e alpha_e,i V_s,i) Wmsg[r,i]
// so Watt is applied once per (destination, relation) segment to the query,
// and Wmsg once per segment to the attention-weighted value sum, instead of
// once per edge.  The per-relation matrices are staged in LDS when they fit.
//
// Lane layout: a group of 16 lanes owns one work item; lane l holds features
// 4l..4l+3, so head i is lanes [i*LH, (i+1)*LH) with LH = d_k / 4 lanes.
#include "rgnn_internal.h"

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

template <int W>
__device__ __forceinline__ float gsum(float x)
{
#pragma unroll
    for (int off = W / 2; off > 0; off >>= 1) x += __shfl_xor(x, off, W);
    return x;
}

constexpr int D = 64, G = 16;
constexpr int kUnroll = 4;

struct HK {
    int64_t n_items;
    const Item *items;
    const int32_t *item_slot, *dst_vsegptr, *vseg_ptr, *vseg_rel, *in_src;
    const float *KV, *Q, *Watt, *Wmsg, *mu;
    float scale;
    int R;
    float *agg, *partial;
};

// y[4 values of this lane] = x_head (1 x dk) . Mat (dk x dk), Mat row-major in
// memory `Mt` (LDS or global), where x_head is distributed over the head's LH
// lanes (4 values each).  Column block of this lane: 4 * (gl % LH).
template <int LH>
__device__ __forceinline__ float4 head_vecmat(float4 x, const float *Mt, int gl)
{
    constexpr int DK = LH * 4;
    const int base = (gl / LH) * LH;     // first lane of this head within the group
    const int c0 = 4 * (gl % LH);
    float4 y = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int jj = 0; jj < LH; ++jj) {
        const float x0 = __shfl(x.x, base + jj, G), x1 = __shfl(x.y, base + jj, G);
        const float x2 = __shfl(x.z, base + jj, G), x3 = __shfl(x.w, base + jj, G);
        const float4 r0 = ld4(Mt + (4 * jj + 0) * DK + c0);
        const float4 r1 = ld4(Mt + (4 * jj + 1) * DK + c0);
        const float4 r2 = ld4(Mt + (4 * jj + 2) * DK + c0);
        const float4 r3 = ld4(Mt + (4 * jj + 3) * DK + c0);
        y = lin4(y, 1.f, r0, x0); y = lin4(y, 1.f, r1, x1);
        y = lin4(y, 1.f, r2, x2); y = lin4(y, 1.f, r3, x3);
    }
    return y;
}

// y[k] = sum_j Mat[k][j] x[j]  (x . Mat^T), same distribution as above.
template <int LH>
__device__ __forceinline__ float4 head_matvec_t(float4 x, const float *Mt, int gl)
{
    constexpr int DK = LH * 4;
    const int base = (gl / LH) * LH;
    const int c0 = 4 * (gl % LH);
    float4 y = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int jj = 0; jj < LH; ++jj) {
        const float4 xj = make_float4(__shfl(x.x, base + jj, G), __shfl(x.y, base + jj, G),
                                      __shfl(x.z, base + jj, G), __shfl(x.w, base + jj, G));
        y.x += dot4(ld4(Mt + (c0 + 0) * DK + 4 * jj), xj);
        y.y += dot4(ld4(Mt + (c0 + 1) * DK + 4 * jj), xj);
        y.z += dot4(ld4(Mt + (c0 + 2) * DK + 4 * jj), xj);
        y.w += dot4(ld4(Mt + (c0 + 3) * DK + 4 * jj), xj);
    }
    return y;
}

template <int H, bool LDS>
__global__ __launch_bounds__(512) void hgt_kernel(HK k)
{
    constexpr int DK = D / H, LH = DK / 4, GPB = 512 / G;
    constexpr int MAT = H * DK * DK;            // floats per relation per matrix
    extern __shared__ float smem[];
    const float *Watt = k.Watt, *Wmsg = k.Wmsg;
    if (LDS) {
        const int n = k.R * MAT;
        for (int i = threadIdx.x; i < n; i += 512) {
            smem[i] = k.Watt[i];
            smem[n + i] = k.Wmsg[i];
        }
        __syncthreads();
        Watt = smem;
        Wmsg = smem + n;
    }
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
        float4 agg = make_float4(0.f, 0.f, 0.f, 0.f);
        if (sb < se) {
            const float4 q = ld4(k.Q + (size_t)v * D + gl * 4);
            for (int vs = sb; vs < se; ++vs) {
                const int r = k.vseg_rel[vs];
                const float *Wa = Watt + (size_t)r * MAT + (size_t)head * DK * DK;
                const float *Wm = Wmsg + (size_t)r * MAT + (size_t)head * DK * DK;
                // query moved through W_att (reordering), with prior and scale folded in
                const float4 qp = scale4(head_matvec_t<LH>(q, Wa, gl), k.mu[r] * k.scale);
                float4 vacc = make_float4(0.f, 0.f, 0.f, 0.f);
                const int e0 = k.vseg_ptr[vs], e1 = k.vseg_ptr[vs + 1];
                for (int e = e0; e < e1; e += kUnroll) {
                    int src[kUnroll];
                    float4 kr[kUnroll], vr[kUnroll];
#pragma unroll
                    for (int u = 0; u < kUnroll; ++u) src[u] = k.in_src[min(e + u, e1 - 1)];
#pragma unroll
                    for (int u = 0; u < kUnroll; ++u) {
                        kr[u] = ld4(k.KV + (size_t)src[u] * (2 * D) + gl * 4);
                        vr[u] = ld4(k.KV + (size_t)src[u] * (2 * D) + D + gl * 4);
                    }
#pragma unroll
                    for (int u = 0; u < kUnroll; ++u) {
                        const float a = gsum<LH>(dot4(kr[u], qp));
                        if (e + u < e1) {
                            const float mn = fmaxf(m, a);
                            const float c1 = __expf(m - mn), c2 = __expf(a - mn);
                            s = s * c1 + c2;
                            vacc = lin4(vacc, c1, vr[u], c2);
                            agg = scale4(agg, c1);
                            m = mn;
                        }
                    }
                }
                agg = add4(agg, head_vecmat<LH>(vacc, Wm, gl));
            }
        }
        if (slot < 0) {
            st4(k.agg + (size_t)v * D + gl * 4, scale4(agg, s > 0.f ? 1.f / s : 0.f));
        } else {
            float *pr = k.partial + (size_t)slot * (2 * H + D);
            if (gl % LH == 0) { pr[head * 2] = m; pr[head * 2 + 1] = s; }
            st4(pr + 2 * H + gl * 4, agg);
        }
    }
}

}  // namespace

size_t hgt_lds_bytes(int R, int heads)
{
    const int dk = D / heads;
    return (size_t)2 * R * heads * dk * dk * sizeof(float);
}

rgnn_status launch_hgt_traverse(const HgtArgs &a, hipStream_t s)
{
    const rgnn_graph *g = a.g;
    if (g->n_items == 0) return RGNN_OK;
    if (a.d != D) return fail(RGNN_EUNSUPPORTED, "HGT traversal supports d = 64");
    HK k{};
    k.n_items = g->n_items; k.items = g->dev.items; k.item_slot = g->dev.item_slot;
    k.dst_vsegptr = g->dev.dst_vsegptr; k.vseg_ptr = g->dev.vseg_ptr;
    k.vseg_rel = g->dev.vseg_rel; k.in_src = g->dev.in_src;
    k.KV = a.KV; k.Q = a.Q; k.Watt = a.Watt; k.Wmsg = a.Wmsg; k.mu = a.mu;
    k.scale = a.scale; k.R = g->R; k.agg = a.agg; k.partial = a.partial;
    const size_t lds = hgt_lds_bytes(g->R, a.heads);
    const bool use_lds = lds <= 64 * 1024;
    const unsigned nb = (unsigned)((g->n_items + 31) / 32);
    LaunchScope ls("hgt_traverse", s);
#define HGT(H) do { if (use_lds) hipLaunchKernelGGL((hgt_kernel<H, true>), dim3(nb), dim3(512), lds, s, k); \
                    else hipLaunchKernelGGL((hgt_kernel<H, false>), dim3(nb), dim3(512), 0, s, k); } while (0)
    if (a.heads == 1) HGT(1);
    else if (a.heads == 2) HGT(2);
    else if (a.heads == 4) HGT(4);
    else return fail(RGNN_EUNSUPPORTED, "HGT traversal supports heads in {1, 2, 4}");
#undef HGT
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? RGNN_OK : hip_fail(e, "hgt traversal launch");
}

}  // namespace rgnn
