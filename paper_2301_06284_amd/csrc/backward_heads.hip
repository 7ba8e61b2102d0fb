// backward_heads.hip -- RGAT backward with several heads in one pass over the
// graph (Section "Backward Propagation"), for d in {32, 64, 128} and
// H = d / d_k heads of d_k >= 16 columns, softmax over each destination's
// in-edges or over each (destination, relation) segment.
//
// With one head the backward runs in the input space (backward.hip: the
// destination-side gradient G_v W_r^T is one d_in-row per segment).  With H
// heads that row becomes H rows, one per head (head k's columns of W_r), and
// the source pass would gather H of them per out-edge.  Here the gradient is
// taken in the message space instead, where every head owns its own columns
// of one d_out-row.  For an in-edge e = (u -> v, r) with message
// m_e = M_p = h_u W_r (p = (u, r), the compact pair of Section "Compact
// Tensor Materialization"), and head k of columns C_k:
//   y_e,k     = m_e[C_k] . w_src[r][C_k] + h_v . wt'_{r,k}
//   q_e,k     = exp(leaky(y_e,k) - M_v,k),   Z'_v,k = sum_e q,   S'_v,k = sum_e q dalpha
//   dalpha_e,k = m_e[C_k] . G_v[C_k],   alpha = q / Z',   s = S' / Z'
//   Y_e,k     = alpha (dalpha - s) leaky'(y_e,k)
//   dM_p      = sum_{e in p} alpha_e (.) G_v + ypair_p (.) w_src[r]      ((.): per head)
//   dh_u     += sum_p dM_p W_r^T              dh_v += sum_seg sum_k ysum_seg,k wt'_{r,k}
//   dW_r      = sum_p h_u^T dM_p + sum_k dwt'_{r,k} (x) w_dst[r][C_k]
//   dw_src[r][C_k] = dws'_{r,k} W_r[:, C_k],  dw_dst[r][C_k] = dwt'_{r,k} W_r[:, C_k]
//   with dws'_{r,k} = sum_p ypair_p,k h_u and dwt'_{r,k} = sum_seg ysum_seg,k h_v.
// Z' and S' are summed here from this pass's own logits (the forward's M only
// shifts the exponent), as in the one-head backward.
//
// Kernels: the messages M by the typed GEMM over the compact pairs; a
// destination-major pass over the forward's work items (alpha, Y per edge and
// head, the per-segment sums of Y, dh_v's destination term); a source-major
// pass over the out-edges that forms dM per pair (a pair's out-edges are
// consecutive); dM W_r^T by the typed GEMM with rows scattered into
// source-major pair order, summed per source into dh; outer-product MFMA
// chunks of h_u^T dM per relation; per-head GEMVs for dws' and dwt'; a
// per-relation finalize.
#include <type_traits>

#include "rgnn_internal.h"
#include "wave_ops.h"

namespace rgnn {

namespace {

constexpr int kE = kChunkEdges, kDst = kMaxDstPerItem;
// threads per workgroup of the item passes: eight items at d = 32 and 64,
// four at d = 128 (their LDS stages hold per-edge and per-destination values
// of every head)
constexpr int mh_threads(int D) { return D == 32 ? 64 : 128; }
constexpr int kU = 4;      // edges per prefetch batch
constexpr int kDstKU = 2;  // edges per prefetch batch of the destination pass

__device__ __forceinline__ float4 ld4(const float *p) { return *reinterpret_cast<const float4 *>(p); }
__device__ __forceinline__ void st4(float *p, float4 v) { *reinterpret_cast<float4 *>(p) = v; }
__device__ __forceinline__ float dot4(float4 a, float4 b) { return a.x * b.x + a.y * b.y + a.z * b.z + a.w * b.w; }
__device__ __forceinline__ float4 zero4() { return make_float4(0.f, 0.f, 0.f, 0.f); }
__device__ __forceinline__ float4 add4(float4 a, float4 b) { return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w); }
__device__ __forceinline__ float4 lin4(float4 a, float s, float4 b, float t)
{
    return make_float4(a.x * s + b.x * t, a.y * s + b.y * t, a.z * s + b.z * t, a.w * s + b.w * t);
}
__device__ __forceinline__ float2 add2(float2 a, float2 b) { return make_float2(a.x + b.x, a.y + b.y); }
__device__ __forceinline__ float leaky(float y, float slope) { return y > 0.f ? y : slope * y; }
__device__ __forceinline__ void atomic_add4(float *p, float4 v)
{
    atomicAdd(p + 0, v.x); atomicAdd(p + 1, v.y); atomicAdd(p + 2, v.z); atomicAdd(p + 3, v.w);
}
// a * b - c and a * b - c * d with every product rounded on its own (never
// fused into an FMA): exactly 0 when c was formed as the rounded product of
// the same two values
__device__ __forceinline__ float mul_sub_exact(float a, float b, float c)
{
#pragma clang fp contract(off)
    return a * b - c;
}
__device__ __forceinline__ float cross_diff(float a, float b, float c, float d)
{
#pragma clang fp contract(off)
    return a * b - c * d;
}

// ---------------------------------------------------------------- destination-major pass
struct HK {
    int64_t n_items;
    const Item *items;
    const int32_t *item_slot, *dst_vsegptr, *vseg_ptr, *vseg_rel, *vseg_pos, *e2u, *vseg_seg;
    const float *M, *w_src, *wtp, *saved, *vatt, *G;
    float2 *sv;              // [N, H] (S', Z') per destination and head: written by pass 1 for
                             // whole destinations, by the merge for split ones
    float2 *ssum;            // [slots, H] (S', Z') of each piece of a split destination
    float2 *svs;             // per-segment softmax: [V, H] (S', Z') per vseg, then per segment
    float slope;
    float *ay;               // [E, H, 2] per sorted in-edge and head: (q, dalpha) from pass 1
                             // (q with the sign bit set where the logit is <= 0), then (alpha, Y)
    float *ysum;             // [V, H] per vseg (by-relation position) and head: sum of Y
    float *dh;               // [N, D] destination terms written here
    float *dpart;            // [slots, D] a split destination's term, per piece (summed after)
    const int32_t *split_items;
    int64_t n_split_items;
};

// Only indices and the forward's maxima live in LDS (about 2 KB per item):
// the per-edge (q, dalpha) and per-destination (S', Z') go to global memory
// (their own outputs' buffers), which keeps occupancy at the register limit.
template <int H, bool SEG>
struct MStage {
    int eidx[kE];            // compact pair of each edge (row of M)
    int evs[kE];             // item-local segment of each edge
    int vptr[kE + 1];
    int vrel[kE];
    int vpos[kE];            // by-relation position of each segment
    int vdj[kE];             // item-local destination of each segment
    int dptr[kDst + 1];
    float dM[SEG ? 1 : kDst * H];   // reference maximum of each destination and head
    float vM[SEG ? kE * H : 1];     // per-segment softmax: reference maximum per segment
};

// PHASE 0: every item; whole destinations run all passes, pieces of split
//          destinations run pass 1 and leave (S', Z') in ssum.
// PHASE 1: pieces of split destinations: the segment sums and pass 2 with the
//          merged (S', Z').
// SEG: PHASE 0 runs pass 1 for every item (per-vseg (S', Z') to svs); PHASE 1
//      runs the rest for every item.
// KU: edges per prefetch batch of pass 1 (two batches in flight).
template <int D, int H, int PHASE, bool SEG, int KU>
__global__ __launch_bounds__(mh_threads(D)) void mh_dst_kernel(HK k)
{
    constexpr int G = D / 4, GPB = mh_threads(D) / G, LH = G / H;
    __shared__ MStage<H, SEG> stage[GPB];
    const int gl = threadIdx.x % G, gi = threadIdx.x / G;
    const int head = gl / LH;
    const bool hl = gl % LH == 0;   // the lane that records its head's scalars
    MStage<H, SEG> &st = stage[gi];
    float2 *ay2 = reinterpret_cast<float2 *>(k.ay);
    const int64_t gidx = (int64_t)blockIdx.x * GPB + gi;
    const int64_t item = PHASE == 1 && !SEG ? (gidx < k.n_split_items ? k.split_items[gidx] : k.n_items) : gidx;
    bool valid = item < k.n_items;
    int dst0 = 0, nd = 0, vs0 = 0, nv = 0, e0 = 0, ne = 0, slot = -1;
    if (valid) {
        const Item x = k.items[item];
        slot = k.item_slot[item];
        dst0 = x.dst0; nd = x.dst1 - x.dst0; vs0 = x.vs0; nv = x.vs1 - x.vs0;
        e0 = k.vseg_ptr[x.vs0]; ne = k.vseg_ptr[x.vs1] - e0;
        if (PHASE == 1 && !SEG && slot < 0) valid = false;
    }
    if (valid) {
        for (int j = gl; j < nv; j += G) {
            const int a = k.vseg_ptr[vs0 + j] - e0, b = k.vseg_ptr[vs0 + j + 1] - e0;
            st.vptr[j] = a;
            st.vrel[j] = k.vseg_rel[vs0 + j];
            st.vpos[j] = k.vseg_pos[vs0 + j];
            for (int e = a; e < b; ++e) st.evs[e] = j;
        }
        if (SEG && PHASE == 0)
            for (int i = gl; i < nv * H; i += G)
                st.vM[i] = k.saved[((size_t)k.vseg_seg[vs0 + i / H] * H + i % H) * 2];
        if (gl == 0) st.vptr[nv] = ne;
        auto dvs = [&](int jj) {
            const int vs = k.dst_vsegptr[dst0 + jj];
            return (vs < vs0 ? vs0 : (vs > vs0 + nv ? vs0 + nv : vs)) - vs0;
        };
        for (int j = gl; j < nd; j += G) {
            const int a = dvs(j), b = dvs(j + 1);
            st.dptr[j] = k.vseg_ptr[vs0 + a] - e0;
            for (int jv = a; jv < b; ++jv) st.vdj[jv] = j;
        }
        if (!SEG && PHASE == 0)
            for (int i = gl; i < nd * H; i += G) st.dM[i] = k.saved[((int64_t)dst0 * H + i) * 2];
        if (gl == 0) st.dptr[nd] = ne;
        if (PHASE == 0)
            for (int e = gl; e < ne; e += G) st.eidx[e] = k.e2u[e0 + e];
    }
    __syncthreads();

    // pass 1: per edge and head the logit, q and dalpha (to ay); (S', Z') per
    // destination (or per vseg)
    if (PHASE == 0 && valid && ne > 0) {
        int j = 0, jv = 0;
        while (st.dptr[j + 1] == st.dptr[j]) ++j;
        float s = 0.f, zs = 0.f;
        // ping-pong batches of (message row, w_src row, G row of the destination,
        // the segment's destination term)
        float4 Am[KU], Aw[KU], Ag[KU], Bm[KU], Bw[KU], Bg[KU];
        float Av[KU], Bv[KU];
        auto load = [&](float4 (&Xm)[KU], float4 (&Xw)[KU], float4 (&Xg)[KU], float (&Xv)[KU], int base) {
#pragma unroll
            for (int u = 0; u < KU; ++u) {
                const int e = base + u < ne ? base + u : ne - 1;
                const int jj = st.evs[e];
                Xm[u] = ld4(k.M + (size_t)st.eidx[e] * D + gl * 4);
                Xw[u] = ld4(k.w_src + (size_t)st.vrel[jj] * D + gl * 4);
                Xg[u] = ld4(k.G + (size_t)(dst0 + st.vdj[jj]) * D + gl * 4);
                Xv[u] = k.vatt[(size_t)(vs0 + jj) * H + head];
            }
        };
        auto consume = [&](const float4 (&Xm)[KU], const float4 (&Xw)[KU], const float4 (&Xg)[KU],
                           const float (&Xv)[KU], int base) {
#pragma unroll
            for (int u = 0; u < KU; ++u) {
                const int e = base + u;
                const float ys = gsum<LH>(dot4(Xm[u], Xw[u]));
                const float da = gsum<LH>(dot4(Xm[u], Xg[u]));
                if (e < ne) {
                    const float y = ys + Xv[u];
                    const float z = leaky(y, k.slope);
                    const float q = __expf(z - (SEG ? st.vM[jv * H + head] : st.dM[j * H + head]));
                    s = __builtin_fmaf(q, da, s);   // the same operation as the segment sums
                    zs += q;
                    if (hl) ay2[(size_t)(e0 + e) * H + head] = make_float2(y > 0.f ? q : -q, da);
                    if (e + 1 == st.vptr[jv + 1]) {
                        if (SEG) {
                            if (hl) k.svs[(size_t)(vs0 + jv) * H + head] = make_float2(s, zs);
                            s = 0.f;
                            zs = 0.f;
                        }
                        ++jv;
                        if (e + 1 == st.dptr[j + 1]) {
                            if (!SEG) {
                                if (hl) {
                                    if (slot < 0) k.sv[(size_t)(dst0 + j) * H + head] = make_float2(s, zs);
                                    else k.ssum[(size_t)slot * H + head] = make_float2(s, zs);
                                }
                                s = 0.f;
                                zs = 0.f;
                            }
                            ++j;
                            while (j < nd && st.dptr[j + 1] == st.dptr[j]) ++j;
                        }
                    }
                }
            }
        };
        load(Am, Aw, Ag, Av, 0);
        __builtin_amdgcn_sched_barrier(0);
        for (int eb = 0; eb < ne; eb += 2 * KU) {
            load(Bm, Bw, Bg, Bv, eb + KU);
            __builtin_amdgcn_sched_barrier(0);
            consume(Am, Aw, Ag, Av, eb);
            load(Am, Aw, Ag, Av, eb + 2 * KU);
            __builtin_amdgcn_sched_barrier(0);
            consume(Bm, Bw, Bg, Bv, eb + KU);
        }
    }
    // the workgroup's global writes of pass 1 are visible to it after the barrier
    __syncthreads();

    const bool fin = valid && (PHASE == 1 || (!SEG && slot < 0));
    auto sz_of = [&](int jv, int hh) {
        return SEG ? k.svs[(size_t)(vs0 + jv) * H + hh] : k.sv[(size_t)(dst0 + st.vdj[jv]) * H + hh];
    };
    // the sum of Y per segment and head, from (q, dalpha) before pass 2
    // replaces them.  A piece of a split destination with few segments (of
    // many edges): the group's lanes take its edges (all in flight) and the
    // four sums per head are reduced over the group; otherwise a lane takes a
    // (segment, head) pair with four edges' pairs in flight.
    if (fin && PHASE == 1 && !SEG && nv * H <= G / 2) {
        constexpr int NPL = (kE + G - 1) / G;   // edges per lane
        for (int jv = 0; jv < nv; ++jv) {
            const int eb = st.vptr[jv], ee = st.vptr[jv + 1];
            float2 p[NPL][H];
#pragma unroll
            for (int u = 0; u < NPL; ++u) {
                const int e = eb + gl + u * G;
#pragma unroll
                for (int hh = 0; hh < H; ++hh)
                    p[u][hh] = e < ee ? ay2[(size_t)(e0 + e) * H + hh] : make_float2(0.f, 0.f);
            }
            float ap[H], bp[H], an[H], bn[H];
#pragma unroll
            for (int hh = 0; hh < H; ++hh) {
                ap[hh] = bp[hh] = an[hh] = bn[hh] = 0.f;
#pragma unroll
                for (int u = 0; u < NPL; ++u) {
                    const float a = p[u][hh].x, q = fabsf(a);
                    if (signbit(a)) {
                        an[hh] = __builtin_fmaf(q, p[u][hh].y, an[hh]);
                        bn[hh] += q;
                    } else {
                        ap[hh] = __builtin_fmaf(q, p[u][hh].y, ap[hh]);
                        bp[hh] += q;
                    }
                }
                ap[hh] = gsum<G>(ap[hh]);
                bp[hh] = gsum<G>(bp[hh]);
                an[hh] = gsum<G>(an[hh]);
                bn[hh] = gsum<G>(bn[hh]);
            }
#pragma unroll
            for (int hh = 0; hh < H; ++hh) {
                if (gl != hh) continue;
                const float2 sz = sz_of(jv, hh);
                const float ys = sz.y > 0.f ? (cross_diff(ap[hh], sz.y, sz.x, bp[hh]) +
                                               k.slope * cross_diff(an[hh], sz.y, sz.x, bn[hh])) /
                                                  (sz.y * sz.y)
                                            : 0.f;
                k.ysum[(size_t)st.vpos[jv] * H + hh] = ys;
            }
        }
    } else if (fin) {
        for (int i = gl; i < nv * H; i += G) {
            const int jv = i / H, hh = i % H;
            const float2 sz = sz_of(jv, hh);
            float ap = 0.f, bp = 0.f, an = 0.f, bn = 0.f;
            const int eb = st.vptr[jv], ee = st.vptr[jv + 1];
            for (int e = eb; e < ee; e += 4) {
                float2 p[4];
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    p[u] = ay2[(size_t)(e0 + (e + u < ee ? e + u : ee - 1)) * H + hh];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    if (e + u >= ee) break;
                    const float a = p[u].x, q = fabsf(a);
                    if (signbit(a)) {
                        an = __builtin_fmaf(q, p[u].y, an);
                        bn += q;
                    } else {
                        ap = __builtin_fmaf(q, p[u].y, ap);
                        bp += q;
                    }
                }
            }
            const float ys = sz.y > 0.f ? (cross_diff(ap, sz.y, sz.x, bp) + k.slope * cross_diff(an, sz.y, sz.x, bn)) /
                                              (sz.y * sz.y)
                                        : 0.f;
            k.ysum[(size_t)st.vpos[jv] * H + hh] = ys;
        }
    }
    __syncthreads();   // every (q, dalpha) of the item has been read; ysum is visible
    // pass 2: (alpha, Y) per edge and head, over the pairs written by pass 1
    if (fin) {
        for (int i = gl; i < ne * H; i += G) {
            const int e = i / H, hh = i % H, jv = st.evs[e];
            const float2 sz = sz_of(jv, hh);
            const float2 p = ay2[(size_t)e0 * H + i];
            const float a = p.x;
            const float al = sz.y > 0.f ? fabsf(a) / sz.y : 0.f;
            const float dz = sz.y > 0.f ? mul_sub_exact(p.y, sz.y, sz.x) / sz.y : 0.f;
            const float Y = al * dz * (signbit(a) ? k.slope : 1.f);
            ay2[(size_t)e0 * H + i] = make_float2(al, Y);
        }
    }
    // pass 3: destination term dh_v = sum over v's segments and heads of ysum * wt'
    // (a piece of a split destination writes its segments' share to its slot)
    if (fin && (slot < 0 ? PHASE == 0 || SEG : PHASE == 1)) {
        float4 acc = zero4();
        int j = 0;
        auto flush_to = [&](int jn) {
            while (j < jn) {
                st4((slot < 0 ? k.dh + (size_t)(dst0 + j) * D : k.dpart + (size_t)slot * D) + gl * 4, acc);
                acc = zero4();
                ++j;
            }
        };
        constexpr int SB = 2;   // segments per batch
        float4 Aw[SB][H], Bw[SB][H];
        float Ay[SB][H], By[SB][H];
        auto load = [&](float4 (&Xw)[SB][H], float (&Xy)[SB][H], int base) {
#pragma unroll
            for (int u = 0; u < SB; ++u) {
                const int jv = base + u < nv ? base + u : (nv > 0 ? nv - 1 : 0);
#pragma unroll
                for (int hh = 0; hh < H; ++hh) {
                    Xw[u][hh] = ld4(k.wtp + ((size_t)st.vrel[jv] * H + hh) * D + gl * 4);
                    Xy[u][hh] = k.ysum[(size_t)st.vpos[jv] * H + hh];
                }
            }
        };
        auto consume = [&](const float4 (&Xw)[SB][H], const float (&Xy)[SB][H], int base) {
#pragma unroll
            for (int u = 0; u < SB; ++u) {
                const int jv = base + u;
                if (jv < nv) {
                    flush_to(st.vdj[jv]);
#pragma unroll
                    for (int hh = 0; hh < H; ++hh) acc = lin4(acc, 1.f, Xw[u][hh], Xy[u][hh]);
                }
            }
        };
        if (nv > 0) {
            load(Aw, Ay, 0);
            __builtin_amdgcn_sched_barrier(0);
            for (int b = 0; b < nv; b += 2 * SB) {
                load(Bw, By, b + SB);
                __builtin_amdgcn_sched_barrier(0);
                consume(Aw, Ay, b);
                load(Aw, Ay, b + 2 * SB);
                __builtin_amdgcn_sched_barrier(0);
                consume(Bw, By, b + SB);
            }
        }
        flush_to(nd);
    }
}

// Per-segment softmax: (S', Z') of a (dst, rel) segment cut into several
// vsegs, summed in vseg order and written back to each of them.
template <int H>
__global__ __launch_bounds__(256) void mh_merge_seg_s_kernel(int64_t U, const int32_t *seg_vsegptr, float2 *svs)
{
    const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (t >= U * H) return;
    const int64_t i = t / H;
    const int hh = (int)(t % H);
    const int b = seg_vsegptr[i], e = seg_vsegptr[i + 1];
    if (e - b <= 1) return;
    float2 s = make_float2(0.f, 0.f);
    for (int vs = b; vs < e; ++vs) s = add2(s, svs[(size_t)vs * H + hh]);
    for (int vs = b; vs < e; ++vs) svs[(size_t)vs * H + hh] = s;
}

// ---------------------------------------------------------------- source-major pass
// dM_p = sum over the out-edges of pair p of alpha (.) G_v, plus ypair_p (.)
// w_src[r]; ypair_p,k = sum of Y_k.  Out-edges are ordered by (src, rel,
// position), so a pair's out-edges are consecutive; a pair lies in one item
// unless its source is split over several, whose pairs are summed with
// atomics into rows zeroed beforehand.
struct PK {
    int64_t n_items;
    const Item *items;
    const int32_t *out_ptr, *out_pos, *out_rel, *out_pair, *out_dst;
    const float *G, *ay, *w_src;
    float *dM;               // [U, D]
    float *ypair;            // [U, H]
};

struct PStage {
    int edst[kE], epos[kE], erel[kE], epair[kE], enode[kE];
    int optr[kDst + 1];
};

template <int D, int H>
__global__ __launch_bounds__(mh_threads(D)) void mh_pair_kernel(PK k)
{
    constexpr int G = D / 4, GPB = mh_threads(D) / G, LH = G / H;
    __shared__ PStage stage[GPB];
    const int gl = threadIdx.x % G, gi = threadIdx.x / G;
    const int head = gl / LH;
    PStage &st = stage[gi];
    const int64_t item = (int64_t)blockIdx.x * GPB + gi;
    const bool valid = item < k.n_items;
    int n0 = 0, nn = 0, q0 = 0, nq = 0;
    bool split = false;
    if (valid) {
        const Item x = k.items[item];
        n0 = x.dst0; nn = x.dst1 - x.dst0; q0 = x.vs0; nq = x.vs1 - x.vs0;
        split = nn == 1 && k.out_ptr[n0 + 1] - k.out_ptr[n0] > nq;
        for (int e = gl; e < nq; e += G) {
            st.edst[e] = k.out_dst[q0 + e];
            st.epos[e] = k.out_pos[q0 + e];
            st.erel[e] = k.out_rel[q0 + e];
            st.epair[e] = k.out_pair[q0 + e];
        }
        auto opos = [&](int jj) {
            const int q = k.out_ptr[n0 + jj];
            return (q < q0 ? q0 : (q > q0 + nq ? q0 + nq : q)) - q0;
        };
        for (int j = gl; j < nn; j += G) {
            const int a = opos(j), b = opos(j + 1);
            for (int e = a; e < b; ++e) st.enode[e] = j;
        }
    }
    __syncthreads();
    if (!valid || nq == 0) return;
    float4 acc = zero4();
    float ysrc = 0.f;
    // ping-pong batches of (G row of the destination, (alpha, Y) of this lane's head)
    float4 Ag[kU], Bg[kU];
    float2 Aa[kU], Ba[kU];
    auto load = [&](float4 (&Xg)[kU], float2 (&Xa)[kU], int b0) {
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int e = b0 + u < nq ? b0 + u : nq - 1;
            Xg[u] = ld4(k.G + (size_t)st.edst[e] * D + gl * 4);
            Xa[u] = reinterpret_cast<const float2 *>(k.ay)[(size_t)st.epos[e] * H + head];
        }
    };
    auto consume = [&](const float4 (&Xg)[kU], const float2 (&Xa)[kU], int b0) {
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int e = b0 + u;
            if (e < nq) {
                acc = lin4(acc, 1.f, Xg[u], Xa[u].x);
                ysrc += Xa[u].y;
                if (e + 1 == nq || st.epair[e + 1] != st.epair[e]) {   // the pair ends here
                    const int p = st.epair[e];
                    const float4 row = lin4(acc, 1.f, ld4(k.w_src + (size_t)st.erel[e] * D + gl * 4), ysrc);
                    float *dst = k.dM + (size_t)p * D + gl * 4;
                    if (split) {
                        atomic_add4(dst, row);
                        if (gl % LH == 0) atomicAdd(k.ypair + (size_t)p * H + head, ysrc);
                    } else {
                        st4(dst, row);
                        if (gl % LH == 0) k.ypair[(size_t)p * H + head] = ysrc;
                    }
                    acc = zero4();
                    ysrc = 0.f;
                }
            }
        }
    };
    load(Ag, Aa, 0);
    __builtin_amdgcn_sched_barrier(0);
    for (int eb = 0; eb < nq; eb += 2 * kU) {
        load(Bg, Ba, eb + kU);
        __builtin_amdgcn_sched_barrier(0);
        consume(Ag, Aa, eb);
        load(Ag, Aa, eb + 2 * kU);
        __builtin_amdgcn_sched_barrier(0);
        consume(Bg, Ba, eb + kU);
    }
}

// Zero the dM rows and ypair entries of the pairs of split sources (summed
// with atomics); one 256-thread workgroup per split source.
template <int D, int H>
__global__ __launch_bounds__(256) void mh_zero_split_pairs_kernel(const int32_t *osplit, const int32_t *out_ptr,
                                                                  const int32_t *out_pair, float *dM, float *ypair)
{
    constexpr int G = D / 4, NG = 256 / G;
    const int gl = threadIdx.x % G, gi = threadIdx.x / G;
    const int u = osplit[blockIdx.x];
    for (int q = out_ptr[u] + gi; q < out_ptr[u + 1]; q += NG) {
        const int p = out_pair[q];
        st4(dM + (size_t)p * D + gl * 4, zero4());
        if (gl < H) ypair[(size_t)p * H + gl] = 0.f;
    }
}

// dh_u += sum of the rows of u's pairs in source-major order (dHp = dM W_r^T).
// ---------------------------------------------------------------- pair-major pass (d <= 64)
// One workgroup per chunk of virtual pairs of one relation r (a compact pair,
// or a piece of at most kPairPiece of its out-edges).  In steps of KB virtual
// pairs, every group of D/4 lanes forms the dM rows of its pairs from their
// out-edges (the alpha-weighted G rows summed in out-edge order, plus the sum
// of Y times w_src[r], per head) and fetches their h_u rows, both into LDS; then
// on the matrix cores
//   dHp rows  = dM W_r^T    (stored at the virtual pair's source-major row)
//   partial  += h^T dM       (the chunk's share of dW_r, 16 rows per wave)
// and per head the chunk's sum of ypair h_u (its share of dws').  The
// per-pair gradient dM and the per-pair Y sums never go to memory.
typedef float floatx4 __attribute__((ext_vector_type(4)));

struct PF {
    const Tile *tiles;
    const int32_t *vpair_oe0, *vpair_ne, *vpair_src, *vpair_smpos;
    const int32_t *out_pos, *out_dst;   // sorted in-edge position and destination of each out-edge
    const float *G, *ay, *w_src, *W, *h;
    float *dHp;              // [NVP, D] rows in source-major order
    float *partial;          // [chunks, D, D]
    float *pvec;             // [chunks, H, D]
};

template <int D, int H>
__global__ __launch_bounds__(256) void mh_pair_fused_kernel(PF k)
{
    static_assert(H <= 4, "the per-head Y sums ride in the four padding floats of an LDS row");
    constexpr int G = D / 4, NG = 256 / G, LH = G / H;
    constexpr int KB = 64, P = D + 4;
    constexpr int RPG = KB / NG;        // pair rows per group and step
    constexpr int NCB = D / 16, KC = D / 16;
    static_assert(RPG * NG == KB, "a step must split evenly over the groups");
    __shared__ float Ws[D * P];         // W_r, row-major: Ws[i * P + j] = W_r[i][j]
    __shared__ float As[KB * P];        // h_u rows of the step's virtual pairs, their sums of Y
                                        // per head in the row padding (H <= 4)
    __shared__ float Bs[KB * P];        // their dM rows
    const Tile t = k.tiles[blockIdx.x];
    const int r = t.type;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int li = lane & 15, q = lane >> 4;
    const int gl = tid % G, gi = tid / G, head = gl / LH;
    const bool hl = gl % LH == 0;
    for (int i = tid; i < D * D / 4; i += 256) {
        const int row = i / (D / 4), c4 = (i % (D / 4)) * 4;
        *reinterpret_cast<float4 *>(&Ws[row * P + c4]) = ld4(k.W + ((size_t)r * D + row) * D + c4);
    }
    const float4 ws = ld4(k.w_src + (size_t)r * D + gl * 4);
    const float2 *ay2 = reinterpret_cast<const float2 *>(k.ay);
    // outer-product accumulators: NCB blocks of h^T dM, and one block of h^T Y
    // (its first H columns: the chunk's dws' share per head)
    floatx4 acc[NCB + 1];
#pragma unroll
    for (int cb = 0; cb <= NCB; ++cb) acc[cb] = floatx4{0.f, 0.f, 0.f, 0.f};
    for (int k0 = 0; k0 < t.rows; k0 += KB) {
        // gather: the group's RPG rows together, two out-edges of each per batch
        int oe[RPG], ne[RPG], us[RPG];
#pragma unroll
        for (int s = 0; s < RPG; ++s) {
            const int rr = gi + NG * s;
            const bool ok = k0 + rr < t.rows;
            const int vp = t.row0 + (ok ? k0 + rr : 0);
            oe[s] = k.vpair_oe0[vp];
            ne[s] = ok ? k.vpair_ne[vp] : 0;
            us[s] = k.vpair_src[vp];
        }
        float4 hr[RPG], am[RPG];
        float ys[RPG];
        int nmax = 0;
#pragma unroll
        for (int s = 0; s < RPG; ++s) {
            hr[s] = ld4(k.h + (size_t)us[s] * D + gl * 4);
            am[s] = zero4();
            ys[s] = 0.f;
            nmax = ne[s] > nmax ? ne[s] : nmax;
        }
        // the wave's largest count (pairs are ordered by count, so a step's
        // pairs mostly share it): batches of two out-edges, one for an odd tail
#pragma unroll
        for (int m = 1; m < 64; m <<= 1) nmax = max(nmax, __shfl_xor(nmax, m));
        nmax = __builtin_amdgcn_readfirstlane(nmax);
        auto batch = [&](auto nu_c, int o) {
            constexpr int NU = decltype(nu_c)::value;
            int pos[RPG][NU], dv[RPG][NU];
#pragma unroll
            for (int s = 0; s < RPG; ++s)
#pragma unroll
                for (int u = 0; u < NU; ++u) {
                    const int e = oe[s] + (o + u < ne[s] ? o + u : 0);
                    pos[s][u] = k.out_pos[e];
                    dv[s][u] = k.out_dst[e];
                }
            float4 gr[RPG][NU];
            float2 a[RPG][NU];
#pragma unroll
            for (int s = 0; s < RPG; ++s)
#pragma unroll
                for (int u = 0; u < NU; ++u) {
                    gr[s][u] = ld4(k.G + (size_t)dv[s][u] * D + gl * 4);
                    a[s][u] = ay2[(size_t)pos[s][u] * H + head];
                }
#pragma unroll
            for (int s = 0; s < RPG; ++s)
#pragma unroll
                for (int u = 0; u < NU; ++u)
                    if (o + u < ne[s]) {
                        am[s] = lin4(am[s], 1.f, gr[s][u], a[s][u].x);
                        ys[s] += a[s][u].y;
                    }
        };
        int o = 0;
        for (; o + 1 < nmax; o += 2) batch(std::integral_constant<int, 2>{}, o);
        if (o < nmax) batch(std::integral_constant<int, 1>{}, o);
#pragma unroll
        for (int s = 0; s < RPG; ++s) {
            const int rr = gi + NG * s;
            const bool ok = ne[s] > 0;
            *reinterpret_cast<float4 *>(&As[rr * P + gl * 4]) = ok ? hr[s] : zero4();
            *reinterpret_cast<float4 *>(&Bs[rr * P + gl * 4]) = ok ? lin4(am[s], 1.f, ws, ys[s]) : zero4();
            if (hl) As[rr * P + D + head] = ok ? ys[s] : 0.f;
        }
        __syncthreads();
        // dHp rows of this wave's 16 virtual pairs (transposed block: lane
        // (li, q) ends with row li, columns 4q .. 4q + 3 of each column block)
        if (wave * 16 < KB) {
            const int p0 = wave * 16;
            floatx4 o4[NCB];
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb) o4[cb] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int c = 0; c < KC; ++c) {
                const float4 b4 = *reinterpret_cast<const float4 *>(&Bs[(p0 + li) * P + c * 16 + q * 4]);
#pragma unroll
                for (int cb = 0; cb < NCB; ++cb) {
                    const float4 a4 = *reinterpret_cast<const float4 *>(&Ws[(cb * 16 + li) * P + c * 16 + q * 4]);
                    o4[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4.x, b4.x, o4[cb], 0, 0, 0);
                    o4[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4.y, b4.y, o4[cb], 0, 0, 0);
                    o4[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4.z, b4.z, o4[cb], 0, 0, 0);
                    o4[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4.w, b4.w, o4[cb], 0, 0, 0);
                }
            }
            const int row = k0 + p0 + li;
            if (row < t.rows) {
                float *dst = k.dHp + (size_t)k.vpair_smpos[t.row0 + row] * D + q * 4;
#pragma unroll
                for (int cb = 0; cb < NCB; ++cb)
                    st4(dst + cb * 16, make_float4(o4[cb][0], o4[cb][1], o4[cb][2], o4[cb][3]));
            }
        }
        // the chunk's dW_r share: rows 16 wave .. of h^T dM, k over the step's pairs
        if (wave * 16 < D) {
#pragma unroll 4
            for (int kk = 0; kk < KB; kk += 4) {
                const float av = As[(kk + q) * P + wave * 16 + li];
#pragma unroll
                for (int cb = 0; cb < NCB; ++cb)
                    acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, Bs[(kk + q) * P + cb * 16 + li], acc[cb], 0, 0, 0);
                const float yv = li < H ? As[(kk + q) * P + D + li] : 0.f;
                acc[NCB] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, yv, acc[NCB], 0, 0, 0);
            }
        }
        __syncthreads();
    }
    if (wave * 16 < D) {
        float *out = k.partial + (size_t)blockIdx.x * D * D;
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
            for (int v = 0; v < 4; ++v) out[(size_t)(wave * 16 + q * 4 + v) * D + cb * 16 + li] = acc[cb][v];
        if (li < H)
#pragma unroll
            for (int v = 0; v < 4; ++v)
                k.pvec[((size_t)blockIdx.x * H + li) * D + wave * 16 + q * 4 + v] = acc[NCB][v];
    }
}

template <int D>
__global__ __launch_bounds__(256) void mh_src_sum_kernel(int64_t N, const int32_t *src_pairptr, const float *dHp,
                                                         float *dh)
{
    constexpr int G = D / 4, GPB = 256 / G;
    const int gl = threadIdx.x % G;
    const int64_t u = (int64_t)blockIdx.x * GPB + threadIdx.x / G;
    if (u >= N) return;
    const int b = src_pairptr[u], e = src_pairptr[u + 1];
    if (b == e) return;
    float4 acc = ld4(dh + (size_t)u * D + gl * 4);
    // rows in batches of four (clamped loads, all in flight together)
    for (int i = b; i < e; i += 4) {
        float4 x[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) x[j] = ld4(dHp + (size_t)(i + j < e ? i + j : e - 1) * D + gl * 4);
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if (i + j < e) acc = add4(acc, x[j]);
    }
    st4(dh + (size_t)u * D + gl * 4, acc);
}

// out[t, k, :] = sum over the rows of tile t of wgt[row, k] * X[idx[row]]
// (groups of D/4 lanes over rows, combined in group order).
template <int D, int H>
__global__ __launch_bounds__(256) void mh_gemv_kernel(const Tile *tiles, const int32_t *idx, const float *wgt,
                                                      const float *X, float *out)
{
    constexpr int G = D / 4, NG = 256 / G;
    __shared__ float4 part[NG][G];
    const Tile t = tiles[blockIdx.x];
    const int gl = threadIdx.x % G, gi = threadIdx.x / G;
    float4 acc[H];
#pragma unroll
    for (int hh = 0; hh < H; ++hh) acc[hh] = zero4();
    for (int i = gi; i < t.rows; i += NG) {
        const int row = t.row0 + i;
        const float4 x = ld4(X + (size_t)idx[row] * D + gl * 4);
#pragma unroll
        for (int hh = 0; hh < H; ++hh) acc[hh] = lin4(acc[hh], 1.f, x, wgt[(size_t)row * H + hh]);
    }
#pragma unroll
    for (int hh = 0; hh < H; ++hh) {
        part[gi][gl] = acc[hh];
        __syncthreads();
        if (gi == 0) {
            float4 s = zero4();
            for (int g = 0; g < NG; ++g) s = add4(s, part[g][gl]);
            st4(out + ((size_t)blockIdx.x * H + hh) * D + gl * 4, s);
        }
        __syncthreads();
    }
}

// Per relation r (blockIdx.x) and 64 entries of its [H, D] vectors
// (blockIdx.y): dws'[r] = sum of its pair chunks' vectors, dwt'[r] = sum of
// its segment chunks' vectors.  16 threads per entry take every 16th chunk
// (four loads in flight); their sums are added in thread order.
template <int D, int H>
__global__ __launch_bounds__(1024) void mh_reduce_kernel(const float *pvec, const int32_t *rel_pairchunkptr,
                                                         const float *yvec, const int32_t *rel_chunkptr, float *dws,
                                                         float *dwt)
{
    constexpr int NS = 16;
    __shared__ float2 red[NS][64];
    const int r = blockIdx.x, li = threadIdx.x % 64, c = threadIdx.x / 64;
    const int i = blockIdx.y * 64 + li;   // entry of [H, D]
    constexpr int U = 4;
    auto strided_sum = [&](const float *vec, int t0, int t1) {
        float acc = 0.f;
        for (int t = t0 + c; t < t1; t += NS * U) {
            float x[U];
#pragma unroll
            for (int u = 0; u < U; ++u) x[u] = t + u * NS < t1 ? vec[(size_t)(t + u * NS) * H * D + i] : 0.f;
#pragma unroll
            for (int u = 0; u < U; ++u) acc += x[u];
        }
        return acc;
    };
    const float a = strided_sum(pvec, rel_pairchunkptr[r], rel_pairchunkptr[r + 1]);
    const float b = strided_sum(yvec, rel_chunkptr[r], rel_chunkptr[r + 1]);
    red[c][li] = make_float2(a, b);
    __syncthreads();
    if (c == 0) {
        float2 s = make_float2(0.f, 0.f);
        for (int cc = 0; cc < NS; ++cc) s = add2(s, red[cc][li]);
        dws[(size_t)r * H * D + i] = s.x;
        dwt[(size_t)r * H * D + i] = s.y;
    }
}

// dW_r (already the ordered sum of the outer-product chunks) += dwt'_{r,k} (x)
// w_dst[r][C_k]; dw_src[r][C_k] = dws'_{r,k} W_r[:, C_k]; dw_dst likewise.
template <int D, int H>
__global__ __launch_bounds__(256) void mh_finalize_kernel(const float *W, const float *w_dst, const float *dws,
                                                          const float *dwt, float *dW, float *dw_src, float *dw_dst)
{
    constexpr int DK = D / H;
    const int r = blockIdx.x;
    const float *Wr = W + (size_t)r * D * D;
    {
        const int idx = blockIdx.y * 256 + threadIdx.x;
        const int i = idx / D, j = idx % D, hh = j / DK;
        dW[(size_t)r * D * D + idx] += dwt[((size_t)r * H + hh) * D + i] * w_dst[(size_t)r * D + j];
    }
    if (blockIdx.y) return;
    // column j: threads (part q, j) take the rows i = q, q + NQ, ... (all loads
    // of a part issued together), the parts are added in order
    constexpr int NQ = 256 / D, RI = D / NQ;
    __shared__ float2 red[NQ][D];
    const int j = threadIdx.x % D, q = threadIdx.x / D, hh = j / DK;
    const float *a = dws + ((size_t)r * H + hh) * D, *b = dwt + ((size_t)r * H + hh) * D;
    float w[RI], av[RI], bv[RI];
#pragma unroll
    for (int t = 0; t < RI; ++t) {
        const int i = q + NQ * t;
        w[t] = Wr[(size_t)i * D + j];
        av[t] = a[i];
        bv[t] = b[i];
    }
    float sa = 0.f, sb = 0.f;
#pragma unroll
    for (int t = 0; t < RI; ++t) {
        sa += av[t] * w[t];
        sb += bv[t] * w[t];
    }
    red[q][j] = make_float2(sa, sb);
    __syncthreads();
    if (q == 0) {
        float2 s = red[0][j];
        for (int qq = 1; qq < NQ; ++qq) s = add2(s, red[qq][j]);
        dw_src[(size_t)r * D + j] = s.x;
        dw_dst[(size_t)r * D + j] = s.y;
    }
}

inline size_t pad256(size_t b) { return (b + 255) & ~size_t(255); }

struct MhWs {
    float *wtp, *vatt, *M, *dHp, *ay, *ysum, *ypair, *partial, *pvec, *yvec, *dws, *dwt, *dpart;
    float2 *ssum, *sv, *svs;
};

size_t mh_layout(const rgnn_graph *g, int D, int H, void *base, MhWs *w)
{
    char *b = (char *)base;
    size_t off = 0;
    auto take = [&](size_t n) {
        float *p = b ? (float *)(b + off) : nullptr;
        off += pad256(std::max<size_t>(n, 1) * sizeof(float));
        return p;
    };
    const size_t R = (size_t)g->R, V = (size_t)g->V, U = (size_t)g->U_src;
    MhWs x;
    x.wtp = take(R * H * D);
    x.vatt = take(V * H);
    const size_t NVP = std::max<size_t>((size_t)g->n_vpairs, U);
    const size_t NCH = std::max<size_t>((size_t)g->n_tiles_vpairs, (size_t)g->n_tiles_outer_pairs);
    x.M = take(U * D);              // messages (then, at d = 128, their gradients dM)
    x.dHp = take(NVP * D);          // dM W_r^T per (virtual) pair, source-major
    x.ay = take((size_t)g->E * H * 2);
    x.ysum = take(V * H);
    x.ypair = take(U * H);
    x.partial = take(NCH * D * D);
    x.pvec = take(NCH * H * D);
    x.yvec = take((size_t)g->n_tiles_outer * H * D);
    x.dws = take(R * H * D);
    x.dwt = take(R * H * D);
    x.ssum = (float2 *)take((size_t)g->n_slots * H * 2);
    x.sv = (float2 *)take((size_t)g->N * H * 2);
    x.svs = (float2 *)take(V * H * 2);
    x.dpart = take((size_t)g->n_slots * D);
    if (w) *w = x;
    return off;
}

template <int D, int H>
rgnn_status mh_backward_dh(const rgnn_graph *g, const float *h, const float *W, const float *w_src,
                           const float *w_dst, float slope, int per_seg, const float *saved, const float *Gm,
                           float *dh, float *dW, float *dws, float *dwt, void *ws, hipStream_t s)
{
    MhWs w;
    mh_layout(g, D, H, ws, &w);
    rgnn_status st;
    hipError_t e;
    const DeviceIndex &x = g->dev;
    // destination terms per segment and head: h_v . wt'_{r,k}
    if ((st = launch_reorder_vec(W, g->R, D, D, H, w_dst, w.wtp, nullptr, nullptr, s)) != RGNN_OK) return st;
    {
        TravArgs ta;
        ta.g = g; ta.h = h; ta.wtp = w.wtp; ta.heads = H; ta.d = D; ta.vatt = w.vatt;
        if ((st = launch_seg_attn(ta, s)) != RGNN_OK) return st;
    }
    {   // messages of the compact pairs
        GemmArgs ga;
        ga.X = h; ga.ldx = D; ga.gather = x.uniq_src;
        ga.W[0] = W; ga.K = D; ga.Nc = D;
        ga.tiles = x.tiles_pairs; ga.ntiles = g->n_tiles_pairs;
        ga.Y = w.M; ga.ldy = D;
        if ((st = launch_typed_gemm(ga, s)) != RGNN_OK) return st;
    }
    HK k{};
    k.n_items = g->n_items; k.items = x.items; k.item_slot = x.item_slot; k.dst_vsegptr = x.dst_vsegptr;
    k.vseg_ptr = x.vseg_ptr; k.vseg_rel = x.vseg_rel; k.vseg_pos = x.vseg_pos; k.e2u = x.e2u;
    k.vseg_seg = x.vseg_seg; k.M = w.M; k.w_src = w_src; k.wtp = w.wtp; k.saved = saved; k.vatt = w.vatt;
    k.G = Gm; k.sv = w.sv; k.ssum = w.ssum; k.svs = w.svs; k.slope = slope; k.ay = w.ay; k.ysum = w.ysum;
    k.dh = dh; k.dpart = w.dpart; k.split_items = x.split_items; k.n_split_items = g->n_split_items;
    constexpr int NTH = mh_threads(D), GPB = NTH / (D / 4);
    if (g->n_items) {
        const dim3 grid((unsigned)((g->n_items + GPB - 1) / GPB));
        if (per_seg) {
            {
                LaunchScope ls("rgat_bwd_heads_dst", s);
                hipLaunchKernelGGL((mh_dst_kernel<D, H, 0, true, kDstKU>), grid, dim3(NTH), 0, s, k);
            }
            if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "mh_dst launch");
            if (g->U_dst) {
                LaunchScope ls("rgat_bwd_heads_merge", s);
                hipLaunchKernelGGL(mh_merge_seg_s_kernel<H>, dim3((unsigned)((g->U_dst * H + 255) / 256)), dim3(256),
                                   0, s, g->U_dst, x.seg_vsegptr, w.svs);
            }
            if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "mh_merge_seg launch");
            {
                LaunchScope ls("rgat_bwd_heads_dst_seg", s);
                hipLaunchKernelGGL((mh_dst_kernel<D, H, 1, true, kDstKU>), grid, dim3(NTH), 0, s, k);
            }
            if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "mh_dst launch");
        } else {
            LaunchScope ls("rgat_bwd_heads_dst", s);
            hipLaunchKernelGGL((mh_dst_kernel<D, H, 0, false, kDstKU>), grid, dim3(NTH), 0, s, k);
            if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "mh_dst launch");
        }
        if (g->n_split) {
            if (!per_seg) {
                // (S', Z') of split destinations: their pieces' parts summed per head
                if ((st = launch_slot_sum(g->n_split, g->n_split_wide, x.split_order, x.split_dst, x.split_slotptr,
                                          reinterpret_cast<const float *>(w.ssum), reinterpret_cast<float *>(w.sv),
                                          2 * H, false, "rgat_bwd_heads_merge", s)) != RGNN_OK)
                    return st;
                if (g->n_split_items) {
                    LaunchScope ls("rgat_bwd_heads_dst_split", s);
                    const dim3 sgrid((unsigned)((g->n_split_items + GPB - 1) / GPB));
                    hipLaunchKernelGGL((mh_dst_kernel<D, H, 1, false, kDstKU>), sgrid, dim3(NTH), 0, s, k);
                }
                if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "mh_dst launch");
            }
            // destination terms of split destinations: the pieces' shares summed
            if ((st = launch_slot_sum(g->n_split, g->n_split_wide, x.split_order, x.split_dst, x.split_slotptr,
                                      w.dpart, dh, D, false, "rgat_bwd_heads_split_dst_term", s)) != RGNN_OK)
                return st;
        }
    }
    const int32_t *pairchunkptr = x.rel_pairchunkptr;
    if constexpr (D <= 64) {
        // one pair-major pass: dM per virtual pair, dHp = dM W_r^T and the
        // chunk shares of dW_r and dws' (dM stays on chip)
        if (g->n_tiles_vpairs) {
            PF p{};
            p.tiles = x.tiles_vpairs; p.vpair_oe0 = x.vpair_oe0; p.vpair_ne = x.vpair_ne;
            p.vpair_src = x.vpair_src; p.vpair_smpos = x.vpair_smpos; p.out_pos = x.out_pos; p.out_dst = x.out_dst;
            p.G = Gm; p.ay = w.ay; p.w_src = w_src; p.W = W; p.h = h;
            p.dHp = w.dHp; p.partial = w.partial; p.pvec = w.pvec;
            LaunchScope ls("rgat_bwd_heads_pair", s);
            hipLaunchKernelGGL((mh_pair_fused_kernel<D, H>), dim3((unsigned)g->n_tiles_vpairs), dim3(256), 0, s, p);
        }
        if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "mh_pair_fused launch");
        if (g->N) {
            LaunchScope ls("rgat_bwd_heads_src_sum", s);
            constexpr int SPB = 256 / (D / 4);
            hipLaunchKernelGGL(mh_src_sum_kernel<D>, dim3((unsigned)((g->N + SPB - 1) / SPB)), dim3(256), 0, s, g->N,
                               x.src_vpairptr, w.dHp, dh);
        }
        if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "mh_src_sum launch");
        if ((st = launch_chunk_sum(w.partial, x.rel_vpairchunkptr, g->R, dW, D, s)) != RGNN_OK) return st;
        pairchunkptr = x.rel_vpairchunkptr;
        {   // dwt' per relation and head
            LaunchScope ls("rgat_bwd_heads_gemv", s);
            if (g->n_tiles_outer)
                hipLaunchKernelGGL((mh_gemv_kernel<D, H>), dim3((unsigned)g->n_tiles_outer), dim3(256), 0, s,
                                   x.tiles_outer, x.vsegdst_byrel, w.ysum, h, w.yvec);
        }
        if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "mh_gemv launch");
    } else {
        // dM per pair (the messages' buffer is reused: M is not read after this)
        float *dM = w.M;
        if (g->n_osplit) {
            LaunchScope ls("zero", s);
            hipLaunchKernelGGL((mh_zero_split_pairs_kernel<D, H>), dim3((unsigned)g->n_osplit), dim3(256), 0, s,
                               x.osplit, x.out_ptr, x.out_pair, dM, w.ypair);
        }
        if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "zero launch");
        if (g->n_oitems) {
            PK p{};
            p.n_items = g->n_oitems; p.items = x.oitems; p.out_ptr = x.out_ptr; p.out_pos = x.out_pos;
            p.out_rel = x.out_rel; p.out_pair = x.out_pair; p.out_dst = x.out_dst; p.G = Gm; p.ay = w.ay;
            p.w_src = w_src; p.dM = dM; p.ypair = w.ypair;
            LaunchScope ls("rgat_bwd_heads_pair", s);
            hipLaunchKernelGGL((mh_pair_kernel<D, H>), dim3((unsigned)((g->n_oitems + GPB - 1) / GPB)), dim3(NTH), 0, s,
                               p);
        }
        if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "mh_pair launch");
        {   // dHp = dM W_r^T, rows in source-major pair order
            GemmArgs ga;
            ga.X = dM; ga.ldx = D; ga.gather = nullptr;
            ga.W[0] = W; ga.trans_b = 1; ga.K = D; ga.Nc = D;
            ga.tiles = x.tiles_pairs; ga.ntiles = g->n_tiles_pairs;
            ga.Y = w.dHp; ga.ldy = D; ga.scatter = x.pair_smpos;
            if ((st = launch_typed_gemm(ga, s)) != RGNN_OK) return st;
        }
        if (g->N) {
            LaunchScope ls("rgat_bwd_heads_src_sum", s);
            constexpr int SPB = 256 / (D / 4);
            hipLaunchKernelGGL(mh_src_sum_kernel<D>, dim3((unsigned)((g->N + SPB - 1) / SPB)), dim3(256), 0, s, g->N,
                               x.src_pairptr, w.dHp, dh);
        }
        if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "mh_src_sum launch");
        // dW: outer products h_u^T dM over the pairs of each relation, summed in order
        if ((st = launch_outer_chunks(x.tiles_outer_pairs, g->n_tiles_outer_pairs, x.uniq_src, 2, h, D, dM, D,
                                      w.partial, D, s)) != RGNN_OK)
            return st;
        if ((st = launch_chunk_sum(w.partial, x.rel_pairchunkptr, g->R, dW, D, s)) != RGNN_OK) return st;
        {   // dws' and dwt' per relation and head
            LaunchScope ls("rgat_bwd_heads_gemv", s);
            if (g->n_tiles_outer_pairs)
                hipLaunchKernelGGL((mh_gemv_kernel<D, H>), dim3((unsigned)g->n_tiles_outer_pairs), dim3(256), 0, s,
                                   x.tiles_outer_pairs, x.uniq_src, w.ypair, h, w.pvec);
            if (g->n_tiles_outer)
                hipLaunchKernelGGL((mh_gemv_kernel<D, H>), dim3((unsigned)g->n_tiles_outer), dim3(256), 0, s,
                                   x.tiles_outer, x.vsegdst_byrel, w.ysum, h, w.yvec);
        }
        if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "mh_gemv launch");
    }
    {
        LaunchScope ls("rgat_bwd_heads_finalize", s);
        hipLaunchKernelGGL((mh_reduce_kernel<D, H>), dim3((unsigned)g->R, H * D / 64), dim3(1024), 0, s, w.pvec,
                           pairchunkptr, w.yvec, x.rel_chunkptr, w.dws, w.dwt);
        hipLaunchKernelGGL((mh_finalize_kernel<D, H>), dim3((unsigned)g->R, D * D / 256), dim3(256), 0, s, W, w_dst,
                           w.dws, w.dwt, dW, dws, dwt);
    }
    if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "mh_finalize launch");
    return RGNN_OK;
}

}  // namespace

rgnn_status rgat_backward_heads_impl(const rgnn_graph *g, const float *h, const float *W, const float *w_src,
                                     const float *w_dst, int d, int heads, float slope, int per_seg,
                                     const float *saved, const float *Gm, float *dh, float *dW, float *dws,
                                     float *dwt, void *ws, size_t ws_bytes, hipStream_t s, size_t *need)
{
    const size_t bytes = mh_layout(g, d, heads, nullptr, nullptr);
    if (need) { *need = bytes; return RGNN_OK; }
    if (!ws || ws_bytes < bytes)
        return fail(RGNN_EINVAL, "workspace too small: need " + std::to_string(bytes) + " bytes");
#define MH(D, H) return mh_backward_dh<D, H>(g, h, W, w_src, w_dst, slope, per_seg, saved, Gm, dh, dW, dws, dwt, ws, s)
    if (d == 32 && heads == 2) MH(32, 2);
    if (d == 64 && heads == 2) MH(64, 2);
    if (d == 64 && heads == 4) MH(64, 4);
    if (d == 128 && heads == 2) MH(128, 2);
    if (d == 128 && heads == 4) MH(128, 4);
    if (d == 128 && heads == 8) MH(128, 8);
#undef MH
    return fail(RGNN_EUNSUPPORTED, "RGAT backward: unsupported (d, heads) for several heads");
}

}  // namespace rgnn
