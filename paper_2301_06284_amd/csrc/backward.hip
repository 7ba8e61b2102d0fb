// backward.hip -- RGAT backward pass (Section "Backward Propagation") for one
// head and d in {32, 64, 128}, softmax over each destination's in-edges, or over each
// (destination, relation) segment (the per-relation variant: M, Z and s below
// are then per segment).
//
// With G = dL/dout, the forward's per-destination softmax maximum M_v and
// denominator Z_v, and the reordered vectors ws'_r = W_r w_src[r],
// wt'_r = W_r w_dst[r]:
//   q_e      = exp(leaky(h_u.ws'_r + h_v.wt'_r) - M_v)
//   Z'_v     = sum_e q_e,   alpha_e = q_e / Z'_v
//   dalpha_e = G_v . (h_u W_r) = h_u . dS_{v,r},   dS_{v,r} = G_v W_r^T
//   s_v      = sum_e alpha_e dalpha_e = S'_v / Z'_v,   S'_v = sum_e q_e dalpha_e
//   Y_e      = alpha_e (dalpha_e - s_v) leaky'(y_e)
//            = alpha_e ((dalpha_e Z'_v - S'_v) / Z'_v) leaky'(y_e)
//   ysum_g   = sum_{e in segment g} Y_e
//            = ((A+_g Z'_v - S'_v B+_g) + slope (A-_g Z'_v - S'_v B-_g)) / Z'_v^2
//            with A+-_g = sum q_e dalpha_e, B+-_g = sum q_e over g's edges with
//            positive (+) and non-positive (-) logits
//   dh_u    += alpha_e dS_{v,r} + Y_e ws'_r       (u as a source)
//   dh_v    += Y_e wt'_r                          (v as a destination)
//   dW_r     = sum_seg (sum_e alpha_e h_u)^T G_v  +  dws'_r^T w_src[r] + dwt'_r^T w_dst[r]
//              with dws'_r = sum_e Y_e h_u,  dwt'_r = sum_e Y_e h_v
//   dw_src[r] = dws'_r W_r,   dw_dst[r] = dwt'_r W_r
//
// The denominator Z'_v is summed here from the backward's own logits rather
// than taken from the forward (whose logits may round differently, e.g. when
// they were formed from the message rows): the alpha that enters Y then sums
// to one in this pass's own arithmetic, and a softmax whose Jacobian vanishes
// exactly (one in-edge: dalpha Z' - S' = dalpha q - q dalpha = 0) gives an
// exact zero.  M_v only shifts the exponent.  Sa (below), which is summed
// before Z'_v is known, takes the forward's Z_v.  The per-segment sum of Y
// is formed from sums accumulated in the same order and with the same
// operations as S' and Z', so that when a segment holds all of a softmax
// group's edges and their logits share a sign (sum Y = 0 exactly: the
// softmax Jacobian's rows sum to zero) A = S' and B = Z' bit for bit and the
// sum is an exact zero, as in exact arithmetic.
//
// Kernel sequence:
//   1. dS by the typed GEMM (B = W_r^T) over the (dst, rel) segments, and the
//      destination attention terms h_v . wt'_r per segment.
//   2. A destination-major traversal over the forward's work items.  Pass 1
//      streams the source rows with the next batch in flight and recomputes
//      alpha, dalpha per edge (kept in LDS), s_v per destination and
//      Sa = sum alpha h_u per segment; pass 2 forms Y per edge and its sum per
//      segment.  Pieces of split destinations finish pass 2 in a second launch
//      once their s_v partials are merged.
//      A third pass writes dh_v's destination term, the sum over v's
//      segments of ysum * wt'_r.  dS, Sa and ysum rows are kept in the
//      by-relation segment order, so the GEMMs over them read and write
//      contiguous rows.
//   3. A source-major traversal over the out-edges (sorted by source, then
//      relation) that gathers dS rows and forms dh_u = (destination term) +
//      sum alpha dS + Y ws'_r with one store per source row: the scatter of
//      the paper's backward becomes a gather, with no per-edge atomics.
//      Pieces of sources with more than kChunkEdges out-edges leave their sums
//      in slots, added to dh in slot order by one workgroup per such source.
//      It also sums Y per (source, relation) pair, the compact rows of the
//      forward.
//   4. dws'_r = sum over r's compact pairs of ysum_pair * h_src, by chunks of
//      pairs; an outer-product MFMA GEMM for dW over K-chunks of segments of
//      one relation (also summing ysum * h_v per chunk for dwt'); then a
//      deterministic combine of the chunks and a per-relation finalize.
#include "rgnn_internal.h"
#include "wave_ops.h"

namespace rgnn {

namespace {

constexpr int kE = kChunkEdges, kDst = kMaxDstPerItem;
// threads per workgroup of the item traversals at width D: 16 items per
// workgroup (their LDS stages), so 128 threads at d = 32
constexpr int item_threads(int D) { return D == 32 ? 128 : 256; }
constexpr int kU = 4;              // rows per prefetch batch in the traversals

__device__ __forceinline__ float4 ld4(const float *p) { return *reinterpret_cast<const float4 *>(p); }
__device__ __forceinline__ void st4(float *p, float4 v) { *reinterpret_cast<float4 *>(p) = v; }
__device__ __forceinline__ float dot4(float4 a, float4 b) { return a.x * b.x + a.y * b.y + a.z * b.z + a.w * b.w; }
__device__ __forceinline__ float4 zero4() { return make_float4(0.f, 0.f, 0.f, 0.f); }
__device__ __forceinline__ float2 add2(float2 a, float2 b) { return make_float2(a.x + b.x, a.y + b.y); }
// a * b - c with the product rounded on its own (never fused into an FMA), so
// that a * b - c is exactly 0 whenever c was formed as the rounded product b * a
__device__ __forceinline__ float mul_sub_exact(float a, float b, float c)
{
#pragma clang fp contract(off)
    return a * b - c;
}
// a * b - c * d with both products rounded on their own: exactly 0 when
// (a, b) and (c, d) are the same pair of values
__device__ __forceinline__ float cross_diff(float a, float b, float c, float d)
{
#pragma clang fp contract(off)
    return a * b - c * d;
}
__device__ __forceinline__ float4 add4(float4 a, float4 b) { return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w); }
__device__ __forceinline__ float4 lin4(float4 a, float s, float4 b, float t)
{
    return make_float4(a.x * s + b.x * t, a.y * s + b.y * t, a.z * s + b.z * t, a.w * s + b.w * t);
}

// ---------------------------------------------------------------- destination-major traversal
struct BK {
    int64_t n_items;
    const Item *items;
    const int32_t *item_slot, *dst_vsegptr, *vseg_ptr, *vseg_rel, *vseg_pos, *in_src;
    const float *h, *wsp, *wtp, *saved, *dS, *vatt;
    const float2 *sv_in;       // [N] merged (S', Z') of split destinations
    const int32_t *vseg_seg;   // per-segment softmax: segment of each vseg (row of saved)
    float2 *svs;               // per-segment softmax: [V] (S', Z') per vseg, then per segment
    float slope;
    float *Sa;       // [V, D]  sum alpha h_u per segment (by-relation order)
    float2 *ssum;    // [slots] (S', Z') partial of each piece of a split destination
    float *ay;       // [E, 2]  per sorted in-edge: (alpha, Y); pieces hold (signed alpha, dalpha) in between
    float *ysum;     // [V]     sum of Y per segment (by-relation order)
    float *dh;       // [N, D]  destination terms written (acc_dh: added) here
    float *dpart;    // [slots, D] a split destination's term, per piece (summed after)
    int acc_dh;
    const int32_t *split_items;   // PHASE 1 without SEG runs over these items only
    int64_t n_split_items;
};

template <bool SEG>
struct BStage {
    int eidx[kE];        // source of each edge
    int evs[kE];         // item-local segment of each edge
    int vptr[kE + 1];    // item-local first edge of each segment
    int vrel[kE];
    int vpos[kE];        // by-relation position of each segment (row of dS, Sa, ysum)
    int vdj[kE];         // item-local destination of each segment
    float vatt[kE];      // h_v . wt'_r of each segment, then its sum of Y
    float ea[kE];        // q of each edge, sign bit set where the logit is <= 0
    float eda[kE];       // dalpha of each edge
    int dptr[kDst + 1];  // item-local first edge of each destination
    float dM[kDst], dZi[kDst];   // per destination: the forward's M_v and 1/Z_v
    float dsv[kDst], dzs[kDst];  // per destination: S'_v and Z'_v of this pass
    float vM[SEG ? kE : 1], vZi[SEG ? kE : 1];   // per segment (per-segment softmax): M, 1/Z
};

// PHASE 0: every item.  Whole destinations run all passes; pieces of split
//          destinations run pass 1, leave their part of (S', Z') in ssum and park
//          (signed q, dalpha) in ay.
// PHASE 1: pieces of split destinations only: pass 2 with the merged s_v and
//          pass 3 for their own segments, written to the piece's slot (the slots
//          of a destination are summed afterwards).
// SEG (softmax per (dst, rel) segment): PHASE 0 runs pass 1 for every item,
//          writing each vseg's part of (S', Z') to svs and parking (q, dalpha);
//          once the parts are summed per segment, PHASE 1 runs passes 2 and 3
//          for every item (pass 3 of a piece to its slot).
template <int D, int PHASE, bool SEG>
__global__ __launch_bounds__(item_threads(D)) void bwd_traverse_kernel(BK k)
{
    constexpr int G = D / 4, GPB = item_threads(D) / G;
    __shared__ BStage<SEG> stage[GPB];
    const int gl = threadIdx.x % G, gi = threadIdx.x / G;
    BStage<SEG> &st = stage[gi];
    const int64_t gidx = (int64_t)blockIdx.x * GPB + gi;
    // the second launch of the per-destination softmax serves only the pieces
    // of split destinations and takes them from their list
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
            st.vatt[j] = k.vatt[vs0 + j];
            if (SEG && PHASE == 0) {
                const float2 sz = *reinterpret_cast<const float2 *>(k.saved + (size_t)k.vseg_seg[vs0 + j] * 2);
                st.vM[j] = sz.x;
                st.vZi[j] = sz.y > 0.f ? 1.f / sz.y : 0.f;
            }
            for (int e = a; e < b; ++e) st.evs[e] = j;
        }
        if (gl == 0) st.vptr[nv] = ne;
        auto dvs = [&](int jj) {   // item-local first segment of destination jj
            const int vs = k.dst_vsegptr[dst0 + jj];
            return (vs < vs0 ? vs0 : (vs > vs0 + nv ? vs0 + nv : vs)) - vs0;
        };
        for (int j = gl; j < nd; j += G) {
            const int a = dvs(j), b = dvs(j + 1);
            st.dptr[j] = k.vseg_ptr[vs0 + a] - e0;
            for (int jv = a; jv < b; ++jv) st.vdj[jv] = j;
            const int64_t v = dst0 + j;
            if (!SEG) {
                const float Z = k.saved[v * 2 + 1];
                st.dM[j] = k.saved[v * 2];
                st.dZi[j] = Z > 0.f ? 1.f / Z : 0.f;
                if (PHASE == 1) {
                    const float2 sz = k.sv_in[v];
                    st.dsv[j] = sz.x;
                    st.dzs[j] = sz.y;
                }
            }
        }
        if (gl == 0) st.dptr[nd] = ne;
        for (int e = gl; e < ne; e += G) {
            if (PHASE == 0) {
                st.eidx[e] = k.in_src[e0 + e];
            } else {
                const float2 p = reinterpret_cast<const float2 *>(k.ay)[e0 + e];
                st.ea[e] = p.x;
                st.eda[e] = p.y;
            }
        }
    }
    __syncthreads();

    // pass 1: alpha, dalpha per edge; s_v per destination; Sa per segment
    if (PHASE == 0 && valid && ne > 0) {
        int j = 0, jv = 0;
        while (st.dptr[j + 1] == st.dptr[j]) ++j;   // first destination with edges
        float s = 0.f, zs = 0.f;
        float4 sa = zero4();
        // ping-pong batches of (source row, ws'_r row, dS row) per edge
        float4 Ah[kU], Aw[kU], Ad[kU], Bh[kU], Bw[kU], Bd[kU];
        auto load = [&](float4 (&Xh)[kU], float4 (&Xw)[kU], float4 (&Xd)[kU], int base) {
#pragma unroll
            for (int u = 0; u < kU; ++u) {
                const int e = base + u < ne ? base + u : ne - 1;
                const int jj = st.evs[e];
                Xh[u] = ld4(k.h + (size_t)st.eidx[e] * D + gl * 4);
                Xw[u] = ld4(k.wsp + (size_t)st.vrel[jj] * D + gl * 4);
                Xd[u] = ld4(k.dS + (size_t)st.vpos[jj] * D + gl * 4);
            }
        };
        auto consume = [&](const float4 (&Xh)[kU], const float4 (&Xw)[kU], const float4 (&Xd)[kU],
                           int base) {
#pragma unroll
            for (int u = 0; u < kU; ++u) {
                const int e = base + u;
                const float ys = gsum<G>(dot4(Xh[u], Xw[u]));
                const float da = gsum<G>(dot4(Xh[u], Xd[u]));
                if (e < ne) {
                    const float y = ys + st.vatt[jv];
                    const float z = y > 0.f ? y : k.slope * y;
                    const float q = SEG ? __expf(z - st.vM[jv]) : __expf(z - st.dM[j]);
                    const float al = q * (SEG ? st.vZi[jv] : st.dZi[j]);   // for Sa only
                    s = __builtin_fmaf(q, da, s);   // same operation as the segment sums of pass 2
                    zs += q;
                    sa = lin4(sa, 1.f, Xh[u], al);
                    if (gl == 0) {
                        st.ea[e] = y > 0.f ? q : -q;
                        st.eda[e] = da;
                    }
                    if (e + 1 == st.vptr[jv + 1]) {
                        st4(k.Sa + (size_t)st.vpos[jv] * D + gl * 4, sa);
                        sa = zero4();
                        if (SEG) {
                            if (gl == 0) k.svs[vs0 + jv] = make_float2(s, zs);
                            s = 0.f;
                            zs = 0.f;
                        }
                        ++jv;
                        if (e + 1 == st.dptr[j + 1]) {
                            if (!SEG) {
                                if (gl == 0) {
                                    if (slot < 0) {
                                        st.dsv[j] = s;
                                        st.dzs[j] = zs;
                                    } else {
                                        k.ssum[slot] = make_float2(s, zs);
                                    }
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
        load(Ah, Aw, Ad, 0);
        __builtin_amdgcn_sched_barrier(0);
        for (int eb = 0; eb < ne; eb += 2 * kU) {
            load(Bh, Bw, Bd, eb + kU);
            __builtin_amdgcn_sched_barrier(0);
            consume(Ah, Aw, Ad, eb);
            load(Ah, Aw, Ad, eb + 2 * kU);
            __builtin_amdgcn_sched_barrier(0);
            consume(Bh, Bw, Bd, eb + kU);
        }
    }
    __syncthreads();

    const bool fin = valid && (PHASE == 1 || (!SEG && slot < 0));   // this launch finishes the item
    if (PHASE == 0 && valid && (SEG || slot >= 0)) {
        for (int e = gl; e < ne; e += G)
            reinterpret_cast<float2 *>(k.ay)[e0 + e] = make_float2(st.ea[e], st.eda[e]);
    }
    // pass 2: Y per edge (edge-parallel over lanes, coalesced (alpha, Y)
    // stores; Y kept in eda), then its sum per segment (segment-parallel,
    // edges in order)
    if (fin) {
        for (int e = gl; e < ne; e += G) {
            const int jv = st.evs[e];
            const float2 sz = SEG ? k.svs[vs0 + jv] : make_float2(st.dsv[st.vdj[jv]], st.dzs[st.vdj[jv]]);
            const float a = st.ea[e];
            const float al = sz.y > 0.f ? fabsf(a) / sz.y : 0.f;
            const float dz = sz.y > 0.f ? mul_sub_exact(st.eda[e], sz.y, sz.x) / sz.y : 0.f;
            const float Y = al * dz * (signbit(a) ? k.slope : 1.f);
            reinterpret_cast<float2 *>(k.ay)[e0 + e] = make_float2(al, Y);
        }
    }
    __syncthreads();
    if (fin) {
        for (int jv = gl; jv < nv; jv += G) {
            const float2 sz = SEG ? k.svs[vs0 + jv] : make_float2(st.dsv[st.vdj[jv]], st.dzs[st.vdj[jv]]);
            float ap = 0.f, bp = 0.f, an = 0.f, bn = 0.f;
            for (int e = st.vptr[jv]; e < st.vptr[jv + 1]; ++e) {
                const float a = st.ea[e], q = fabsf(a);
                if (signbit(a)) {
                    an = __builtin_fmaf(q, st.eda[e], an);
                    bn += q;
                } else {
                    ap = __builtin_fmaf(q, st.eda[e], ap);
                    bp += q;
                }
            }
            const float ys = sz.y > 0.f ? (cross_diff(ap, sz.y, sz.x, bp) + k.slope * cross_diff(an, sz.y, sz.x, bn)) /
                                              (sz.y * sz.y)
                                        : 0.f;
            k.ysum[st.vpos[jv]] = ys;
            st.vatt[jv] = ys;
        }
    }
    __syncthreads();
    // pass 3: destination term dh_v = sum over v's segments of ysum * wt'_r,
    // streaming the wt' rows of the item's segments in ping-pong batches (a
    // piece of a split destination writes its segments' share to its slot)
    if (fin && (slot < 0 ? PHASE == 0 || SEG : PHASE == 1)) {
        float4 acc = zero4();
        int j = 0;
        auto flush_to = [&](int jn) {   // finish destinations [j, jn)
            while (j < jn) {
                if (slot >= 0) {
                    st4(k.dpart + (size_t)slot * D + gl * 4, acc);
                    acc = zero4();
                    ++j;
                    continue;
                }
                float *p = k.dh + (size_t)(dst0 + j) * D + gl * 4;
                st4(p, k.acc_dh ? add4(acc, ld4(p)) : acc);
                acc = zero4();
                ++j;
            }
        };
        float4 Aw[kU], Bw[kU];
        auto load = [&](float4 (&Xw)[kU], int base) {
#pragma unroll
            for (int u = 0; u < kU; ++u) {
                const int jv = base + u < nv ? base + u : (nv > 0 ? nv - 1 : 0);
                Xw[u] = ld4(k.wtp + (size_t)st.vrel[jv] * D + gl * 4);
            }
        };
        auto consume = [&](const float4 (&Xw)[kU], int base) {
#pragma unroll
            for (int u = 0; u < kU; ++u) {
                const int jv = base + u;
                if (jv < nv) {
                    flush_to(st.vdj[jv]);
                    acc = lin4(acc, 1.f, Xw[u], st.vatt[jv]);
                }
            }
        };
        if (nv > 0) {
            load(Aw, 0);
            __builtin_amdgcn_sched_barrier(0);
            for (int b = 0; b < nv; b += 2 * kU) {
                load(Bw, b + kU);
                __builtin_amdgcn_sched_barrier(0);
                consume(Aw, b);
                load(Aw, b + 2 * kU);
                __builtin_amdgcn_sched_barrier(0);
                consume(Bw, b + kU);
            }
        }
        flush_to(nd);
    }
}

// Per-segment softmax: (S', Z') of a (dst, rel) segment cut into several
// vsegs is the sum of its vsegs' parts (in vseg order), written back to each.
__global__ __launch_bounds__(256) void merge_seg_s_kernel(int64_t U, const int32_t *seg_vsegptr, float2 *svs)
{
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= U) return;
    const int b = seg_vsegptr[i], e = seg_vsegptr[i + 1];
    if (e - b <= 1 || e - b > kBigRange) return;
    float2 s = make_float2(0.f, 0.f);
    for (int vs = b; vs < e; ++vs) s = add2(s, svs[vs]);
    for (int vs = b; vs < e; ++vs) svs[vs] = s;
}

// The same for segments with more than kBigRange vsegs: one workgroup each,
// thread parts added in thread order.
__global__ __launch_bounds__(256) void merge_seg_s_big_kernel(const int32_t *big_seg, const int32_t *seg_vsegptr,
                                                              float2 *svs)
{
    __shared__ float2 part[256];
    __shared__ float2 tot;
    const int sg = big_seg[blockIdx.x];
    const int b = seg_vsegptr[sg], e = seg_vsegptr[sg + 1];
    float2 s = make_float2(0.f, 0.f);
    for (int vs = b + (int)threadIdx.x; vs < e; vs += 256) s = add2(s, svs[vs]);
    part[threadIdx.x] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
        float2 t = make_float2(0.f, 0.f);
        for (int i = 0; i < 256; ++i) t = add2(t, part[i]);
        tot = t;
    }
    __syncthreads();
    for (int vs = b + (int)threadIdx.x; vs < e; vs += 256) svs[vs] = tot;
}


// ---------------------------------------------------------------- source-major traversal
struct SK {
    int64_t n_items;
    const Item *items;           // {node0, node1, q0, q1}: nodes and their out-edge range
    const int32_t *out_ptr, *out_pos, *out_vseg, *out_rel, *out_pair;
    const float *wsp, *dS, *ay;
    float *dh;                   // holds the destination terms on entry
    float *ypair;                // [U_src] sum of Y per compact (src, rel) pair, zeroed before
                                 // (written by a store, or by atomics for split sources)
    const int32_t *item_slot;    // slot of each piece of a split source, else -1
    float *part;                 // [slots, D] such pieces' sums, added to dh in slot order later
};

struct SStage {
    int evs[kE];         // dS row (by-relation segment position) of each out-edge
    int erel[kE];
    int epair[kE];       // compact (src, rel) pair of each out-edge
    int enode[kE];       // item-local source of each out-edge
    float ea[kE], ey[kE];
    int optr[kDst + 1];  // item-local first out-edge of each source
};

template <int D>
__global__ __launch_bounds__(item_threads(D)) void bwd_src_kernel(SK k)
{
    constexpr int G = D / 4, GPB = item_threads(D) / G;
    __shared__ SStage stage[GPB];
    const int gl = threadIdx.x % G, gi = threadIdx.x / G;
    SStage &st = stage[gi];
    const int64_t item = (int64_t)blockIdx.x * GPB + gi;
    const bool valid = item < k.n_items;
    int n0 = 0, nn = 0, q0 = 0, nq = 0;
    bool split = false;   // a piece of a source whose out-edges span several items
    int slot = -1;
    if (valid) {
        const Item x = k.items[item];
        n0 = x.dst0; nn = x.dst1 - x.dst0; q0 = x.vs0; nq = x.vs1 - x.vs0;
        slot = k.item_slot[item];
        split = slot >= 0;
        for (int e = gl; e < nq; e += G) {
            const int p = k.out_pos[q0 + e];
            st.evs[e] = k.out_vseg[q0 + e];
            st.erel[e] = k.out_rel[q0 + e];
            st.epair[e] = k.out_pair[q0 + e];
            const float2 a = reinterpret_cast<const float2 *>(k.ay)[p];
            st.ea[e] = a.x;
            st.ey[e] = a.y;
        }
        auto opos = [&](int jj) {
            const int q = k.out_ptr[n0 + jj];
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
    float ysrc = 0.f;
    // ping-pong batches of (dS row, ws'_r row, the source's dh row) per out-edge
    float4 Ad[kU], Aw[kU], Ah[kU], Bd[kU], Bw[kU], Bh[kU];
    auto load = [&](float4 (&Xd)[kU], float4 (&Xw)[kU], float4 (&Xh)[kU], int b0) {
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int e = b0 + u < nq ? b0 + u : nq - 1;
            Xd[u] = ld4(k.dS + (size_t)st.evs[e] * D + gl * 4);
            Xw[u] = ld4(k.wsp + (size_t)st.erel[e] * D + gl * 4);
            Xh[u] = ld4(k.dh + (size_t)(n0 + st.enode[e]) * D + gl * 4);
        }
    };
    auto consume = [&](const float4 (&Xd)[kU], const float4 (&Xw)[kU], const float4 (&Xh)[kU], int b0) {
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int e = b0 + u;
            if (e < nq) {
                const float Y = st.ey[e];
                acc = lin4(acc, 1.f, Xd[u], st.ea[e]);
                acc = lin4(acc, 1.f, Xw[u], Y);
                ysrc += Y;
                const bool node_end = e + 1 == st.optr[j + 1];
                // the last out-edge of the item always ends its source
                if (node_end || st.erel[e + 1] != st.erel[e]) {
                    // a pair's out-edges lie in one item unless its source is
                    // split, so only pieces of split sources need the atomic
                    if (gl == 0) {
                        if (split) atomicAdd(k.ypair + st.epair[e], ysrc);
                        else k.ypair[st.epair[e]] = ysrc;
                    }
                    ysrc = 0.f;
                }
                if (node_end) {
                    if (split) st4(k.part + (size_t)slot * D + gl * 4, acc);
                    else st4(k.dh + (size_t)(n0 + j) * D + gl * 4, add4(acc, Xh[u]));
                    acc = zero4();
                    ++j;
                    while (j < nn && st.optr[j + 1] == st.optr[j]) ++j;
                }
            }
        }
    };
    load(Ad, Aw, Ah, 0);
    __builtin_amdgcn_sched_barrier(0);
    for (int eb = 0; eb < nq; eb += 2 * kU) {
        load(Bd, Bw, Bh, eb + kU);
        __builtin_amdgcn_sched_barrier(0);
        consume(Ad, Aw, Ah, eb);
        load(Ad, Aw, Ah, eb + 2 * kU);
        __builtin_amdgcn_sched_barrier(0);
        consume(Bd, Bw, Bh, eb + kU);
    }
}

// pvec[t] = sum over the compact pairs of tile t (one relation) of
// ypair[pair] * h[src(pair)]; lanes of 16-lane groups over features, groups
// over pairs, combined in group order.
template <int D>
__global__ __launch_bounds__(256) void pair_gemv_kernel(const Tile *tiles, const int32_t *uniq_src,
                                                        const float *ypair, const float *h, float *pvec)
{
    constexpr int G = D / 4, NG = 256 / G;
    __shared__ float4 part[NG][G];
    const Tile t = tiles[blockIdx.x];
    const int gl = threadIdx.x % G, gi = threadIdx.x / G;
    float4 a0 = zero4(), a1 = zero4();
    int i = gi;
    for (; i + NG < t.rows; i += 2 * NG) {
        const int p0 = t.row0 + i, p1 = p0 + NG;
        const float y0 = ypair[p0], y1 = ypair[p1];
        const float4 h0 = ld4(h + (size_t)uniq_src[p0] * D + gl * 4);
        const float4 h1 = ld4(h + (size_t)uniq_src[p1] * D + gl * 4);
        a0 = lin4(a0, 1.f, h0, y0);
        a1 = lin4(a1, 1.f, h1, y1);
    }
    if (i < t.rows) {
        const int p0 = t.row0 + i;
        a0 = lin4(a0, 1.f, ld4(h + (size_t)uniq_src[p0] * D + gl * 4), ypair[p0]);
    }
    part[gi][gl] = add4(a0, a1);
    __syncthreads();
    if (gi == 0) {
        float4 s = zero4();
        for (int g = 0; g < NG; ++g) s = add4(s, part[g][gl]);
        st4(pvec + (size_t)blockIdx.x * D + gl * 4, s);
    }
}

// ---------------------------------------------------------------- dW
typedef float floatx4 __attribute__((ext_vector_type(4)));

// Chunk c covers rows [row0, row0 + rows) of the by-relation segment order:
// partial[c] = sum over its segments of Sa[seg]^T (d_in) x G[dst(seg)] (d_out);
// yvec[c]   = sum over its segments of ysum[seg] * h[dst(seg)].
// YS: also sum ysum[row] * h[v] per chunk (the RGAT dwt' term); GATHER: the
// second operand's row (and h's) is vsegdst[row], else the row itself; GA:
// the first operand's row is vsegdst[row], else the row itself.  lda, ldb:
// row strides.
// A workgroup computes one 64 x 64 tile of the D x D product (blockIdx.y: the
// tile, four at D = 128); at D = 32 the columns past D read as zeros.
template <int D, bool YS, bool GATHER, bool GA>
__global__ __launch_bounds__(256) void outer_gemm_kernel(const Tile *chunks, const int32_t *vsegdst_byrel,
                                                         const float *Sa, int lda,
                                                         const float *Gm, int ldb, const float *h,
                                                         const float *ysum, float *partial,
                                                         float *yvec)
{
    constexpr int KB = 64, P = 68;
    constexpr int SL = KB * 16 / 256;   // float4 slots of each operand per thread and step
    constexpr int NT = D > 64 ? D / 64 : 1;   // tiles per side
    __shared__ float As[KB * P];
    __shared__ float Bs[KB * P];
    __shared__ float4 yred[256];
    const Tile t = chunks[blockIdx.x];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int li = lane & 15, q = lane >> 4;
    const int a0 = NT > 1 ? 64 * ((int)blockIdx.y / NT) : 0;   // tile origin
    const int b0 = NT > 1 ? 64 * ((int)blockIdx.y % NT) : 0;
    const int c4 = (tid & 15) * 4;      // this thread's columns in every slot
    constexpr bool FULL = D >= 64;      // every tile column is a column of the product
    const bool aok = FULL || a0 + c4 < D, bok = FULL || b0 + c4 < D;
    const bool ys = YS && b0 == 0;      // the dwt' sum once per A column range
    floatx4 acc[4];
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) acc[cb] = floatx4{0.f, 0.f, 0.f, 0.f};
    float4 yacc = zero4();
    // Software pipeline over the chunk's 64-row steps: destination indices two
    // steps ahead, rows one step ahead (registers), MFMAs on the LDS copy of
    // the current step.  Rows past the chunk end are clamped to its last row
    // and masked when written to LDS.
    auto row_of = [&](int k0, int sl) {
        const int rr = (tid >> 4) + 16 * sl;
        return t.row0 + min(k0 + rr, t.rows - 1);
    };
    int vi[SL], vn[SL];
    float4 ra[SL], rb[SL], rh[SL];
    float ry[SL];
    auto load_idx = [&](int k0, int (&v)[SL]) {
#pragma unroll
        for (int sl = 0; sl < SL; ++sl) v[sl] = (GATHER || GA) ? vsegdst_byrel[row_of(k0, sl)] : row_of(k0, sl);
    };
    auto load_rows = [&](int k0, const int (&v)[SL]) {
#pragma unroll
        for (int sl = 0; sl < SL; ++sl) {
            const int row = row_of(k0, sl);
            ra[sl] = aok ? ld4(Sa + (size_t)(GA ? v[sl] : row) * lda + a0 + c4) : zero4();
            rb[sl] = bok ? ld4(Gm + (size_t)(GATHER ? v[sl] : row) * ldb + b0 + c4) : zero4();
            if (YS) {
                rh[sl] = ys && aok ? ld4(h + (size_t)v[sl] * D + a0 + c4) : zero4();
                ry[sl] = ysum[row];
            }
        }
    };
    load_idx(0, vi);
    load_rows(0, vi);
    load_idx(KB, vn);
    for (int k0 = 0; k0 < t.rows; k0 += KB) {
#pragma unroll
        for (int sl = 0; sl < SL; ++sl) {
            const int rr = (tid >> 4) + 16 * sl;
            const bool ok = k0 + rr < t.rows;
            *reinterpret_cast<float4 *>(&As[rr * P + c4]) = ok ? ra[sl] : zero4();
            *reinterpret_cast<float4 *>(&Bs[rr * P + c4]) = ok ? rb[sl] : zero4();
            if (YS && ok) yacc = lin4(yacc, 1.f, rh[sl], ry[sl]);
        }
        __syncthreads();
        load_rows(k0 + KB, vn);
        load_idx(k0 + 2 * KB, vn);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll 4
        for (int kk = 0; kk < KB; kk += 4) {
            const float a = As[(kk + q) * P + w * 16 + li];
#pragma unroll
            for (int cb = 0; cb < 4; ++cb)
                acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, Bs[(kk + q) * P + cb * 16 + li], acc[cb], 0, 0, 0);
        }
        __syncthreads();
    }
    float *out = partial + (size_t)blockIdx.x * D * D;
#pragma unroll
    for (int cb = 0; cb < 4; ++cb)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int i = a0 + w * 16 + q * 4 + v, jc = b0 + cb * 16 + li;
            if (FULL || (i < D && jc < D)) out[(size_t)i * D + jc] = acc[cb][v];
        }
    if (ys) {
        yred[tid] = yacc;
        __syncthreads();
        if (tid < 16 && (FULL || a0 + tid * 4 < D)) {
            float4 s = zero4();
            for (int i = tid; i < 256; i += 16) s = add4(s, yred[i]);
            st4(yvec + (size_t)blockIdx.x * D + a0 + tid * 4, s);
        }
    }
}

// The same product at D = 128 with one workgroup per chunk computing all of
// the 128 x 128 partial (the 64 x 64 tiling above reads every row twice).
// The products run on the bf16 matrix cores from exact three-piece splits of
// both operands (x = x1 + x2 + x3, the six piece products of order >= 2^-16
// accumulated in fp32, smallest first; the typed GEMM's split path, which has
// the derivation): 32-row steps, each thread loading one column of 16 rows
// of both operands (every load instruction covers 256 contiguous bytes) and
// writing its column's pieces k-contiguous into three transposed bf16 planes
// per operand, so each MFMA operand fragment is one ds_read_b128; each wave
// computes 32 rows of the product (two row blocks against all eight column
// blocks).
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ void split3_8(const float *x, bf16x8 &hi, bf16x8 &mid, bf16x8 &lo)
{
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const __bf16 a = (__bf16)x[j];
        const float r = x[j] - (float)a;
        const __bf16 b = (__bf16)r;
        hi[j] = a;
        mid[j] = b;
        lo[j] = (__bf16)(r - (float)b);
    }
}

template <bool YS, bool GATHER, bool GA>
__global__ __launch_bounds__(256) void outer_gemm128_kernel(const Tile *chunks, const int32_t *vsegdst_byrel,
                                                            const float *Sa, int lda,
                                                            const float *Gm, int ldb, const float *h,
                                                            const float *ysum, float *partial,
                                                            float *yvec)
{
    constexpr int D = 128, KB = 32, RG = 16;    // rows per step; rows per thread and step
    constexpr int KP = KB + 8;                  // padded bf16 row of a transposed plane
    constexpr int PL = D * KP;                  // bf16 per plane
    __shared__ __attribute__((aligned(16))) __bf16 At[3 * PL];   // At[p][a][k]: pieces of Sa
    __shared__ __attribute__((aligned(16))) __bf16 Bt[3 * PL];   // Bt[p][b][k]: pieces of Gm
    __shared__ float yred[YS ? 256 : 1];
    const Tile t = chunks[blockIdx.x];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int li = lane & 15, q = lane >> 4;
    const int col = tid % D, rg = tid / D;      // this thread's column and row group (16 rows)
    floatx4 acc[2][8];
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int cb = 0; cb < 8; ++cb) acc[rb][cb] = floatx4{0.f, 0.f, 0.f, 0.f};
    float yacc = 0.f;
    auto row_of = [&](int k0, int i) { return t.row0 + min(k0 + rg * RG + i, t.rows - 1); };
    int vi[RG];
    float xa[RG], xb[RG], xh[YS ? RG : 1], xy[YS ? RG : 1];
    auto load_rows = [&](int k0) {
#pragma unroll
        for (int i = 0; i < RG; ++i) vi[i] = (GATHER || GA) ? vsegdst_byrel[row_of(k0, i)] : row_of(k0, i);
#pragma unroll
        for (int i = 0; i < RG; ++i) {
            const int row = row_of(k0, i);
            xa[i] = Sa[(size_t)(GA ? vi[i] : row) * lda + col];
            xb[i] = Gm[(size_t)(GATHER ? vi[i] : row) * ldb + col];
            if (YS) {
                xh[i] = h[(size_t)vi[i] * D + col];
                xy[i] = ysum[row];
            }
        }
    };
    load_rows(0);
    for (int k0 = 0; k0 < t.rows; k0 += KB) {
        // stage this step's pieces (rows past the chunk as zeros)
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
            float va[8], vb[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const int i = 8 * hh + j;
                const bool ok = k0 + rg * RG + i < t.rows;
                va[j] = ok ? xa[i] : 0.f;
                vb[j] = ok ? xb[i] : 0.f;
                if (YS && ok) yacc = fmaf(xy[i], xh[i], yacc);
            }
            bf16x8 p0, p1, p2;
            const int o = col * KP + rg * RG + 8 * hh;
            split3_8(va, p0, p1, p2);
            *reinterpret_cast<bf16x8 *>(&At[o]) = p0;
            *reinterpret_cast<bf16x8 *>(&At[PL + o]) = p1;
            *reinterpret_cast<bf16x8 *>(&At[2 * PL + o]) = p2;
            split3_8(vb, p0, p1, p2);
            *reinterpret_cast<bf16x8 *>(&Bt[o]) = p0;
            *reinterpret_cast<bf16x8 *>(&Bt[PL + o]) = p1;
            *reinterpret_cast<bf16x8 *>(&Bt[2 * PL + o]) = p2;
        }
        __syncthreads();
        if (k0 + KB < t.rows) load_rows(k0 + KB);   // the next step's rows in flight
        __builtin_amdgcn_sched_barrier(0);
        // A = Sa^T (rows a of the product), B = Gm (columns b); lane (li, q)
        // supplies k = 8q .. 8q + 7 of its row / column
        bf16x8 af[2][3];
#pragma unroll
        for (int rb = 0; rb < 2; ++rb)
#pragma unroll
            for (int pl = 0; pl < 3; ++pl)
                af[rb][pl] = *reinterpret_cast<const bf16x8 *>(&At[pl * PL + (w * 32 + rb * 16 + li) * KP + 8 * q]);
#pragma unroll
        for (int cb = 0; cb < 8; ++cb) {
            bf16x8 bfr[3];
#pragma unroll
            for (int pl = 0; pl < 3; ++pl)
                bfr[pl] = *reinterpret_cast<const bf16x8 *>(&Bt[pl * PL + (cb * 16 + li) * KP + 8 * q]);
            // the six piece products, smallest first (planes of A, B)
            constexpr int PA[6] = {0, 2, 1, 1, 0, 0}, PB[6] = {2, 0, 1, 0, 1, 0};
#pragma unroll
            for (int u = 0; u < 6; ++u)
#pragma unroll
                for (int rb = 0; rb < 2; ++rb)
                    acc[rb][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[rb][PA[u]], bfr[PB[u]], acc[rb][cb], 0, 0, 0);
        }
        __syncthreads();
    }
    float *out = partial + (size_t)blockIdx.x * D * D;
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int cb = 0; cb < 8; ++cb)
#pragma unroll
            for (int v = 0; v < 4; ++v)
                out[(size_t)(w * 32 + rb * 16 + q * 4 + v) * D + cb * 16 + li] = acc[rb][cb][v];
    if (YS) {
        yred[tid] = yacc;
        __syncthreads();
        if (tid < D) yvec[(size_t)blockIdx.x * D + tid] = yred[tid] + yred[tid + D];
    }
}

// Per relation r: pws = sum of r's pair-tile vectors, pwt = sum of r's
// segment-chunk vectors, both in a fixed order.
template <int D>
__global__ __launch_bounds__(1024) void bwd_reduce_kernel(const float *pvec, const int32_t *rel_pairtileptr,
                                                          const float *yvec, const int32_t *rel_chunkptr,
                                                          float *pws, float *pwt)
{
    constexpr int NC = 1024 / D;
    __shared__ float red[2][NC][D];
    const int r = blockIdx.x, i = threadIdx.x % D, c = threadIdx.x / D;
    constexpr int U = 4;   // loads in flight per thread
    auto strided_sum = [&](const float *vec, int t0, int t1) {
        float acc = 0.f;
        for (int t = t0 + c; t < t1; t += NC * U) {
            float x[U];
#pragma unroll
            for (int u = 0; u < U; ++u) x[u] = t + u * NC < t1 ? vec[(size_t)(t + u * NC) * D + i] : 0.f;
#pragma unroll
            for (int u = 0; u < U; ++u) acc += x[u];
        }
        return acc;
    };
    const float a = strided_sum(pvec, rel_pairtileptr[r], rel_pairtileptr[r + 1]);
    const float b = strided_sum(yvec, rel_chunkptr[r], rel_chunkptr[r + 1]);
    red[0][c][i] = a;
    red[1][c][i] = b;
    __syncthreads();
    if (c == 0) {
        float x = 0.f, y = 0.f;
        for (int cc = 0; cc < NC; ++cc) { x += red[0][cc][i]; y += red[1][cc][i]; }
        pws[(size_t)r * D + i] = x;
        pwt[(size_t)r * D + i] = y;
    }
}

// Per relation r (blockIdx.x) and 256 entries of dW_r (blockIdx.y): combine
// chunk partials in order, add the rank-1 attention terms; dw_src, dw_dst.
// ATT false: only the ordered sum of the chunk partials (dW of RGCN).
template <int D, bool ATT>
__global__ __launch_bounds__(256) void bwd_finalize_kernel(const float *partial, const int32_t *rel_chunkptr,
                                                           const float *pws_all, const float *pwt_all,
                                                           const float *W, const float *w_src,
                                                           const float *w_dst, float *dW, float *dws,
                                                           float *dwt, int col0, int col1, int acc)
{
    __shared__ float pws[D], pwt[D];
    const int r = blockIdx.x, tid = threadIdx.x;
    if (ATT && tid < D) {
        pws[tid] = pws_all[(size_t)r * D + tid];
        pwt[tid] = pwt_all[(size_t)r * D + tid];
    }
    __syncthreads();
    const int c0 = rel_chunkptr[r], c1 = rel_chunkptr[r + 1];
    {
        const int idx = blockIdx.y * 256 + tid;
        const int i = idx / D, j = idx % D;
        // chunks in order, eight loads in flight
        float s = 0.f;
        for (int c = c0; c < c1; c += 8) {
            float p[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) p[u] = c + u < c1 ? partial[(size_t)(c + u) * D * D + idx] : 0.f;
#pragma unroll
            for (int u = 0; u < 8; ++u) s += p[u];
        }
        if (j < col0 || j >= col1) s = 0.f;
        if (ATT) s += pws[i] * w_src[(size_t)r * D + j] + pwt[i] * w_dst[(size_t)r * D + j];
        if (acc) s += dW[(size_t)r * D * D + idx];
        dW[(size_t)r * D * D + idx] = s;
    }
    if (ATT && blockIdx.y == 0 && tid < D) {
        float a = 0.f, b = 0.f;
        for (int i = 0; i < D; ++i) {
            const float wij = W[((size_t)r * D + i) * D + tid];
            a += pws[i] * wij;
            b += pwt[i] * wij;
        }
        if (acc) {
            a += dws[(size_t)r * D + tid];
            b += dwt[(size_t)r * D + tid];
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

struct BwdWs {
    float *wsp, *wtp, *vatt, *dS, *Sa, *ay, *ysum, *ypair, *pvec, *pws, *pwt, *partial, *yvec, *part, *dpart;
    float2 *ssum, *sv, *svs;
};

size_t bwd_layout(const rgnn_graph *g, int D, void *base, BwdWs *w)
{
    char *b = (char *)base;
    size_t off = 0;
    auto take = [&](size_t n) {
        float *p = b ? (float *)(b + off) : nullptr;
        off += pad256(n * sizeof(float));
        return p;
    };
    const size_t nchunks = (size_t)std::max<int64_t>(g->n_tiles_outer, 1);
    BwdWs x;
    x.wsp = take((size_t)g->R * D);
    x.wtp = take((size_t)g->R * D);
    x.vatt = take((size_t)std::max<int64_t>(g->V, 1));
    x.dS = take((size_t)g->V * D);
    x.Sa = take((size_t)g->V * D);
    x.ssum = (float2 *)take((size_t)std::max<int64_t>(g->n_slots, 1) * 2);
    x.sv = (float2 *)take((size_t)std::max<int64_t>(g->N, 1) * 2);
    x.svs = (float2 *)take((size_t)std::max<int64_t>(g->V, 1) * 2);
    x.ay = take((size_t)g->E * 2);
    x.ysum = take((size_t)std::max<int64_t>(g->V, 1));
    x.ypair = take((size_t)std::max<int64_t>(g->U_src, 1));
    x.pvec = take((size_t)std::max<int64_t>(g->n_tiles_pairs, 1) * D);
    x.pws = take((size_t)g->R * D);
    x.pwt = take((size_t)g->R * D);
    x.partial = take(nchunks * D * D);
    x.yvec = take(nchunks * D);
    x.part = take((size_t)std::max<int64_t>(g->n_oslots, 1) * D);
    x.dpart = take((size_t)std::max<int64_t>(g->n_slots, 1) * D);
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


// 64 x 64 tiles of the D x D outer products
constexpr unsigned outer_tiles(int D) { return D > 64 ? (unsigned)(D / 64) * (D / 64) : 1u; }

}  // namespace


template <int D>
void outer_chunks_d(const Tile *chunks, int64_t nchunks, const int32_t *gather, int gather_x, const float *X,
                    int ldx, const float *Gm, int ldg, float *partial, hipStream_t s)
{
    if constexpr (D == 128) {
        const dim3 grid((unsigned)nchunks);
        if (gather && gather_x == 2)
            hipLaunchKernelGGL((outer_gemm128_kernel<false, false, true>), grid, dim3(256), 0, s,
                               chunks, gather, X, ldx, Gm, ldg, nullptr, nullptr, partial, nullptr);
        else if (gather && gather_x)
            hipLaunchKernelGGL((outer_gemm128_kernel<false, true, true>), grid, dim3(256), 0, s,
                               chunks, gather, X, ldx, Gm, ldg, nullptr, nullptr, partial, nullptr);
        else if (gather)
            hipLaunchKernelGGL((outer_gemm128_kernel<false, true, false>), grid, dim3(256), 0, s,
                               chunks, gather, X, ldx, Gm, ldg, nullptr, nullptr, partial, nullptr);
        else
            hipLaunchKernelGGL((outer_gemm128_kernel<false, false, false>), grid, dim3(256), 0, s,
                               chunks, nullptr, X, ldx, Gm, ldg, nullptr, nullptr, partial, nullptr);
    } else {
        const dim3 grid((unsigned)nchunks, outer_tiles(D));
        if (gather && gather_x == 2)   // only the first operand gathered
            hipLaunchKernelGGL((outer_gemm_kernel<D, false, false, true>), grid, dim3(256), 0, s,
                               chunks, gather, X, ldx, Gm, ldg, nullptr, nullptr, partial, nullptr);
        else if (gather && gather_x)
            hipLaunchKernelGGL((outer_gemm_kernel<D, false, true, true>), grid, dim3(256), 0, s,
                               chunks, gather, X, ldx, Gm, ldg, nullptr, nullptr, partial, nullptr);
        else if (gather)
            hipLaunchKernelGGL((outer_gemm_kernel<D, false, true, false>), grid, dim3(256), 0, s,
                               chunks, gather, X, ldx, Gm, ldg, nullptr, nullptr, partial, nullptr);
        else
            hipLaunchKernelGGL((outer_gemm_kernel<D, false, false, false>), grid, dim3(256), 0, s,
                               chunks, nullptr, X, ldx, Gm, ldg, nullptr, nullptr, partial, nullptr);
    }
}

rgnn_status launch_outer_chunks(const Tile *chunks, int64_t nchunks, const int32_t *gather, int gather_x,
                                const float *X, int ldx, const float *Gm, int ldg, float *partial, int d,
                                hipStream_t s)
{
    if (nchunks == 0) return RGNN_OK;
    {
        LaunchScope ls("outer_gemm", s);
        if (d == 32) outer_chunks_d<32>(chunks, nchunks, gather, gather_x, X, ldx, Gm, ldg, partial, s);
        else if (d == 64) outer_chunks_d<64>(chunks, nchunks, gather, gather_x, X, ldx, Gm, ldg, partial, s);
        else if (d == 128) outer_chunks_d<128>(chunks, nchunks, gather, gather_x, X, ldx, Gm, ldg, partial, s);
        else return fail(RGNN_EUNSUPPORTED, "outer products: d must be 32, 64 or 128");
    }
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? RGNN_OK : hip_fail(e, "outer_gemm launch");
}

namespace {

// Sums of slot rows (rows of W floats, V floats per lane, G = W / V lanes per
// row).  A wave per entry: its 64 / G groups take every (64 / G)-th slot (U
// rows in flight), then the groups' sums are combined by a butterfly over
// the group bits (every lane ends with the same bits).  An entry with more
// than kWaveSlots slots takes a whole 1024-thread workgroup: sixteen waves do
// the same, and their sums are added in wave order.
template <int V>
struct SlotVec;
template <>
struct SlotVec<4> {
    float4 v;
    __device__ void zero() { v = zero4(); }
    __device__ void load(const float *p) { v = ld4(p); }
    __device__ void add(const SlotVec &o) { v = add4(v, o.v); }
    __device__ void xor_add(int m)
    {
        v = add4(v, make_float4(__shfl_xor(v.x, m), __shfl_xor(v.y, m), __shfl_xor(v.z, m), __shfl_xor(v.w, m)));
    }
    __device__ void store(float *p, bool acc) const { st4(p, acc ? add4(ld4(p), v) : v); }
};
template <>
struct SlotVec<2> {
    float2 v;
    __device__ void zero() { v = make_float2(0.f, 0.f); }
    __device__ void load(const float *p) { v = *reinterpret_cast<const float2 *>(p); }
    __device__ void add(const SlotVec &o) { v = make_float2(v.x + o.v.x, v.y + o.v.y); }
    __device__ void xor_add(int m) { v = make_float2(v.x + __shfl_xor(v.x, m), v.y + __shfl_xor(v.y, m)); }
    __device__ void store(float *p, bool acc) const
    {
        float2 *q = reinterpret_cast<float2 *>(p);
        *q = acc ? make_float2(q->x + v.x, q->y + v.y) : v;
    }
};

template <int W, bool ACC>
__global__ __launch_bounds__(1024) void slot_sum_kernel(int64_t n, int64_t nwide, const int32_t *order,
                                                        const int32_t *ids, const int32_t *slotptr,
                                                        const float *part, float *out)
{
    constexpr int V = W % 4 == 0 ? 4 : 2, G = W / V, GW = 64 / G, U = 4;
    static_assert(G >= 1 && G <= 64 && G * V == W, "row width");
    __shared__ SlotVec<V> red[16][G];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const bool wide = (int64_t)blockIdx.x < nwide;
    const int64_t k = wide ? (int64_t)blockIdx.x : nwide + ((int64_t)blockIdx.x - nwide) * 16 + wave;
    if (!wide && k >= n) return;   // whole waves; the narrow path has no barrier
    const int i = order[k];
    const int b = slotptr[i], e = slotptr[i + 1];
    const int gl = lane % G, gw = lane / G;
    const int gi = wide ? wave * GW + gw : gw, ng = wide ? 16 * GW : GW;
    SlotVec<V> acc;
    acc.zero();
    for (int sl = b + gi; sl < e; sl += ng * U) {
        SlotVec<V> x[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (sl + u * ng < e) x[u].load(part + (size_t)(sl + u * ng) * W + gl * V);
            else x[u].zero();
        }
#pragma unroll
        for (int u = 0; u < U; ++u) acc.add(x[u]);
    }
#pragma unroll
    for (int m = G; m < 64; m <<= 1) acc.xor_add(m);
    float *o = out + (size_t)ids[i] * W + gl * V;
    if (!wide) {
        if (gw == 0) acc.store(o, ACC);
        return;
    }
    if (gw == 0) red[wave][gl] = acc;
    __syncthreads();
    if (wave == 0 && gw == 0) {
        SlotVec<V> t = red[0][gl];
        for (int w = 1; w < 16; ++w) t.add(red[w][gl]);
        t.store(o, ACC);
    }
}

// dW[t] = sum of the partials of t's chunks [chunkptr[t], chunkptr[t + 1]),
// per 256 entries (blockIdx.y; four per lane): 16 slices of threads take
// every 16th chunk (eight loads in flight), the slice sums are added in slice
// order.
template <int D>
__global__ __launch_bounds__(1024) void chunk_sum_kernel(const float *partial, const int32_t *chunkptr, float *dW)
{
    constexpr int NS = 16, U = 8;
    __shared__ float4 red[NS][64];
    const int t = blockIdx.x, li = threadIdx.x % 64, c = threadIdx.x / 64;
    const int i = blockIdx.y * 256 + li * 4;
    const int c0 = chunkptr[t], c1 = chunkptr[t + 1];
    float4 s = zero4();
    for (int ch = c0 + c; ch < c1; ch += NS * U) {
        float4 p[U];
#pragma unroll
        for (int u = 0; u < U; ++u) p[u] = ch + u * NS < c1 ? ld4(partial + (size_t)(ch + u * NS) * D * D + i) : zero4();
#pragma unroll
        for (int u = 0; u < U; ++u) s = add4(s, p[u]);
    }
    red[c][li] = s;
    __syncthreads();
    if (c == 0) {
        float4 tot = zero4();
        for (int cc = 0; cc < NS; ++cc) tot = add4(tot, red[cc][li]);
        st4(dW + (size_t)t * D * D + i, tot);
    }
}

}  // namespace

rgnn_status launch_slot_sum(int64_t n, int64_t nwide, const int32_t *order, const int32_t *ids,
                            const int32_t *slotptr, const float *part, float *out, int w, bool accumulate,
                            const char *name, hipStream_t s)
{
    if (n == 0) return RGNN_OK;
    const unsigned nb = (unsigned)(nwide + (n - nwide + 15) / 16);
    {
        LaunchScope ls(name, s);
#define SS(W)                                                                                              \
    do {                                                                                                   \
        if (accumulate)                                                                                    \
            hipLaunchKernelGGL((slot_sum_kernel<W, true>), dim3(nb), dim3(1024), 0, s, n, nwide, order, ids, \
                               slotptr, part, out);                                                        \
        else                                                                                               \
            hipLaunchKernelGGL((slot_sum_kernel<W, false>), dim3(nb), dim3(1024), 0, s, n, nwide, order,    \
                               ids, slotptr, part, out);                                                   \
    } while (0)
        switch (w) {
        case 2: SS(2); break;
        case 4: SS(4); break;
        case 8: SS(8); break;
        case 16: SS(16); break;
        case 32: SS(32); break;
        case 64: SS(64); break;
        case 128: SS(128); break;
        default: return fail(RGNN_EUNSUPPORTED, "slot sums: unsupported row width");
        }
#undef SS
    }
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? RGNN_OK : hip_fail(e, "slot_sum launch");
}

rgnn_status launch_src_merge(const rgnn_graph *g, const float *part, float *dh, int d, hipStream_t s)
{
    if (d != 32 && d != 64 && d != 128) return fail(RGNN_EUNSUPPORTED, "source merge: d must be 32, 64 or 128");
    return launch_slot_sum(g->n_osplit, g->n_osplit_wide, g->dev.osplit_order, g->dev.osplit,
                           g->dev.osplit_slotptr, part, dh, d, true, "src_merge", s);
}

rgnn_status launch_chunk_sum(const float *partial, const int32_t *chunkptr, int R, float *dW, int d,
                             hipStream_t s)
{
    if (R == 0) return RGNN_OK;
    {
        LaunchScope ls("chunk_sum", s);
#define CS(D) hipLaunchKernelGGL((chunk_sum_kernel<D>), dim3((unsigned)R, D * D / 256), dim3(1024), 0, s, \
                                 partial, chunkptr, dW)
        if (d == 32) CS(32);
        else if (d == 64) CS(64);
        else if (d == 128) CS(128);
        else return fail(RGNN_EUNSUPPORTED, "chunk sums: d must be 32, 64 or 128");
#undef CS
    }
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? RGNN_OK : hip_fail(e, "chunk_sum launch");
}

namespace {

template <int D>
rgnn_status rgat_backward_d(const rgnn_graph *g, const float *h, const float *W, const float *w_src,
                            const float *w_dst, float slope, int per_seg, const float *saved, const float *Gm,
                            float *dh, float *dW, float *dws, float *dwt, void *ws, hipStream_t s, BwdHead hd)
{
    BwdWs w;
    bwd_layout(g, D, ws, &w);
    rgnn_status st;
    hipError_t e;
    if ((st = launch_reorder_vec(W, g->R, D, D, 1, w_src, w.wsp, w_dst, w.wtp, s)) != RGNN_OK) return st;
    {   // h_v . wt'_r per segment
        TravArgs ta;
        ta.g = g; ta.h = h; ta.wtp = w.wtp; ta.heads = 1; ta.d = D; ta.vatt = w.vatt;
        if ((st = launch_seg_attn(ta, s)) != RGNN_OK) return st;
    }
    // dS_{v,r} = G_v W_r^T for every (dst, rel) segment
    GemmArgs ga;
    ga.X = Gm; ga.ldx = D; ga.gather = g->dev.vsegdst_byrel;
    ga.W[0] = W; ga.trans_b = 1; ga.K = D; ga.Nc = D;
    ga.tiles = g->dev.tiles_vsegs; ga.ntiles = g->n_tiles_vsegs;
    ga.Y = w.dS; ga.ldy = D; ga.scatter = nullptr;   // dS rows in by-relation order
    if ((st = launch_typed_gemm(ga, s)) != RGNN_OK) return st;

    BK k{};
    k.n_items = g->n_items; k.items = g->dev.items; k.item_slot = g->dev.item_slot;
    k.dst_vsegptr = g->dev.dst_vsegptr; k.vseg_ptr = g->dev.vseg_ptr; k.vseg_rel = g->dev.vseg_rel;
    k.vseg_pos = g->dev.vseg_pos; k.wtp = w.wtp; k.dh = dh;
    k.in_src = g->dev.in_src; k.h = h; k.wsp = w.wsp; k.saved = saved; k.dS = w.dS;
    k.vatt = w.vatt; k.sv_in = w.sv; k.slope = slope; k.Sa = w.Sa; k.ssum = w.ssum; k.ay = w.ay;
    k.ysum = w.ysum; k.vseg_seg = g->dev.vseg_seg; k.svs = w.svs; k.acc_dh = hd.acc;
    k.split_items = g->dev.split_items; k.n_split_items = g->n_split_items; k.dpart = w.dpart;
    if (g->n_items && per_seg) {
        constexpr int GPB = item_threads(D) / (D / 4);
        const dim3 grid((unsigned)((g->n_items + GPB - 1) / GPB));
        {
            LaunchScope ls("rgat_bwd_traverse", s);
            hipLaunchKernelGGL((bwd_traverse_kernel<D, 0, true>), grid, dim3(item_threads(D)), 0, s, k);
        }
        if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "rgat_bwd launch");
        {
            LaunchScope ls("rgat_bwd_merge_seg_s", s);
            if (g->U_dst)
                hipLaunchKernelGGL(merge_seg_s_kernel, dim3((unsigned)((g->U_dst + 255) / 256)), dim3(256), 0,
                                   s, g->U_dst, g->dev.seg_vsegptr, w.svs);
            if (g->n_big_seg)
                hipLaunchKernelGGL(merge_seg_s_big_kernel, dim3((unsigned)g->n_big_seg), dim3(256), 0, s,
                                   g->dev.big_seg, g->dev.seg_vsegptr, w.svs);
        }
        if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "merge_seg_s launch");
        {
            LaunchScope ls("rgat_bwd_traverse_seg", s);
            hipLaunchKernelGGL((bwd_traverse_kernel<D, 1, true>), grid, dim3(item_threads(D)), 0, s, k);
        }
        if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "rgat_bwd launch");
        // split destinations: their pieces' shares of the destination term summed
        if ((st = launch_slot_sum(g->n_split, g->n_split_wide, g->dev.split_order, g->dev.split_dst,
                                  g->dev.split_slotptr, w.dpart, dh, D, hd.acc != 0, "rgat_bwd_split_dst_term",
                                  s)) != RGNN_OK)
            return st;
    } else if (g->n_items) {
        constexpr int GPB = item_threads(D) / (D / 4);
        const dim3 grid((unsigned)((g->n_items + GPB - 1) / GPB));
        {
            LaunchScope ls("rgat_bwd_traverse", s);
            hipLaunchKernelGGL((bwd_traverse_kernel<D, 0, false>), grid, dim3(item_threads(D)), 0, s, k);
        }
        if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "rgat_bwd launch");
        if (g->n_split) {
            // (S', Z') of split destinations: their pieces' parts summed
            if ((st = launch_slot_sum(g->n_split, g->n_split_wide, g->dev.split_order, g->dev.split_dst,
                                      g->dev.split_slotptr, reinterpret_cast<const float *>(w.ssum),
                                      reinterpret_cast<float *>(w.sv), 2, false, "rgat_bwd_merge_s", s)) != RGNN_OK)
                return st;
            {
                LaunchScope ls("rgat_bwd_traverse_split", s);
                const dim3 sgrid((unsigned)((g->n_split_items + GPB - 1) / GPB));
                hipLaunchKernelGGL((bwd_traverse_kernel<D, 1, false>), sgrid, dim3(item_threads(D)), 0, s, k);
            }
            if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "rgat_bwd launch");
            if ((st = launch_slot_sum(g->n_split, g->n_split_wide, g->dev.split_order, g->dev.split_dst,
                                      g->dev.split_slotptr, w.dpart, dh, D, hd.acc != 0, "rgat_bwd_split_dst_term",
                                      s)) != RGNN_OK)
                return st;
        }
    }
    // dh += source terms (dh holds the destination terms); Y sums per compact pair
    if ((e = zero(w.ypair, g->U_src, s)) != hipSuccess) return hip_fail(e, "zero launch");
    if (g->n_oitems) {
        SK sk{};
        sk.n_items = g->n_oitems; sk.items = g->dev.oitems; sk.out_ptr = g->dev.out_ptr;
        sk.out_pos = g->dev.out_pos; sk.out_vseg = g->dev.out_vseg; sk.out_rel = g->dev.out_rel;
        sk.out_pair = g->dev.out_pair; sk.wsp = w.wsp; sk.dS = w.dS; sk.ay = w.ay; sk.dh = dh; sk.ypair = w.ypair;
        sk.item_slot = g->dev.oitem_slot; sk.part = w.part;
        LaunchScope ls("rgat_bwd_src", s);
        constexpr int GPB = item_threads(D) / (D / 4);
        hipLaunchKernelGGL(bwd_src_kernel<D>, dim3((unsigned)((g->n_oitems + GPB - 1) / GPB)), dim3(item_threads(D)),
                           0, s, sk);
    }
    if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "bwd_src launch");
    if ((st = launch_src_merge(g, w.part, dh, D, s)) != RGNN_OK) return st;
    if (g->n_tiles_pairs) {   // dws' per pair tile
        LaunchScope ls("rgat_bwd_pair_gemv", s);
        hipLaunchKernelGGL(pair_gemv_kernel<D>, dim3((unsigned)g->n_tiles_pairs), dim3(256), 0, s,
                           g->dev.tiles_pairs, g->dev.uniq_src, w.ypair, h, w.pvec);
    }
    if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "pair_gemv launch");
    if (g->n_tiles_outer) {
        LaunchScope ls("outer_gemm", s);
        if constexpr (D == 128)
            hipLaunchKernelGGL((outer_gemm128_kernel<true, true, false>), dim3((unsigned)g->n_tiles_outer),
                               dim3(256), 0, s,
                               g->dev.tiles_outer, g->dev.vsegdst_byrel, w.Sa, D, Gm, D, h, w.ysum,
                               w.partial, w.yvec);
        else
            hipLaunchKernelGGL((outer_gemm_kernel<D, true, true, false>), dim3((unsigned)g->n_tiles_outer, outer_tiles(D)),
                               dim3(256), 0, s,
                               g->dev.tiles_outer, g->dev.vsegdst_byrel, w.Sa, D, Gm, D, h, w.ysum,
                               w.partial, w.yvec);
    }
    if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "outer_gemm launch");
    {
        LaunchScope ls("rgat_bwd_reduce", s);
        hipLaunchKernelGGL(bwd_reduce_kernel<D>, dim3((unsigned)g->R), dim3(1024), 0, s, w.pvec,
                           g->dev.rel_pairtileptr, w.yvec, g->dev.rel_chunkptr, w.pws, w.pwt);
    }
    if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "bwd_reduce launch");
    {
        LaunchScope ls("rgat_bwd_finalize", s);
        hipLaunchKernelGGL((bwd_finalize_kernel<D, true>), dim3((unsigned)g->R, D * D / 256), dim3(256), 0, s, w.partial,
                           g->dev.rel_chunkptr, w.pws, w.pwt, W, w_src, w_dst, dW, dws, dwt, hd.col0, hd.col1,
                           hd.acc);
    }
    if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "finalize launch");
    return RGNN_OK;
}

}  // namespace

rgnn_status rgat_backward_impl(const rgnn_graph *g, const float *h, const float *W,
                               const float *w_src, const float *w_dst, int d_in, int d_out,
                               float slope, int per_seg, const float *saved, const float *Gm,
                               float *dh, float *dW, float *dws, float *dwt, void *ws,
                               size_t ws_bytes, hipStream_t s, size_t *need, BwdHead hd)
{
    const size_t bytes = bwd_layout(g, d_in, nullptr, nullptr);
    if (need) { *need = bytes; return RGNN_OK; }
    if (d_in != d_out || (d_in != 32 && d_in != 64 && d_in != 128))
        return fail(RGNN_EUNSUPPORTED, "RGAT backward supports d_in = d_out in {32, 64, 128}");
    if (!ws || ws_bytes < bytes)
        return fail(RGNN_EINVAL, "workspace too small: need " + std::to_string(bytes) + " bytes");
    if (d_in == 32) return rgat_backward_d<32>(g, h, W, w_src, w_dst, slope, per_seg, saved, Gm, dh, dW, dws, dwt, ws, s, hd);
    if (d_in == 64) return rgat_backward_d<64>(g, h, W, w_src, w_dst, slope, per_seg, saved, Gm, dh, dW, dws, dwt, ws, s, hd);
    return rgat_backward_d<128>(g, h, W, w_src, w_dst, slope, per_seg, saved, Gm, dh, dW, dws, dwt, ws, s, hd);
}

}  // namespace rgnn
