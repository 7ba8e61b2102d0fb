// hgt_backward.hip -- HGT backward pass for the loss L = sum(out * G), the
// chain rule of the HGT layer (Section "Backward Propagation" derives the
// backward from the forward; here it is written out), for d in {32, 64, 128}
// and d / heads >= 16.  With the forward's reordered segment queries QP_vs = c_r Q_t
// Watt[r]^T per head (c_r = mu[r] * scale), the per-edge score a_e = K_s . QP_vs,
// alpha_e its softmax over the destination's in-edges (saved max M_t and sum
// Z_t), and dagg = G Wa^T (or G):
//   dP_vs   = dagg_t Wmsg[r]^T                (per head; so dalpha_e = V_s . dP_vs)
//   s_t     = sum_e alpha_e dalpha_e,   da_e = alpha_e (dalpha_e - s_t)
//   dK_s    = sum over s's out-edges of da_e QP_vs
//   dV_s    = sum over s's out-edges of alpha_e dP_vs
//   dQP_vs  = sum_{e in vs} da_e K_s = A_vs - s_t B_vs,
//             A_vs = sum alpha dalpha K_s,  B_vs = sum alpha K_s
//   dQ_t    = sum over t's segments of dQP_vs Wqp[r]^T
//   dWatt[r] = c_r (sum_vs dQP_vs^T Q_t)[head blocks],  dmu[r] = scale <., Watt[r]>
//   dWmsg[r] = (sum_vs Salpha_vs^T dagg_t)[head blocks],  Salpha_vs = sum alpha V_s
//   dWa = sum_t agg_t^T G_t,  dh = dK Wk^T + dV Wv^T + dQ Wq^T (+ G with the residual)
//   dWk = sum_n h_n^T dK_n (per node type), likewise dWv, dWq.
//
// Kernel sequence: the forward (K|V|Q GEMM, segment queries, traversal with
// its softmax statistics) is recomputed; dagg and dWa; the block-diagonal
// W_msg^T and the segment rows dP (typed GEMM); a destination-major pass over
// the forward's work items (per edge alpha and dalpha from the K|V row and the
// segment's QP and dP rows; per segment Salpha, A, B; per destination s); the
// split destinations' s merged in slot order; dQP; dQ by the typed GEMM and
// the segment reduction; the per-relation outer products (MFMA chunks);
// a source-major pass over the out-edge index that recomputes alpha and da per
// out-edge and writes dK|dV once per source (float atomics only for pieces of
// sources with more than kChunkEdges out-edges); dh and the per-type weight
// gradients by typed GEMMs and outer-product chunks.
#include "rgnn_internal.h"
#include "wave_ops.h"

namespace rgnn {

namespace {

constexpr int kE = kChunkEdges, kDst = kMaxDstPerItem;
constexpr int kU = 2;             // edges per prefetch batch

__device__ __forceinline__ float4 ld4(const float *p) { return *reinterpret_cast<const float4 *>(p); }
__device__ __forceinline__ void st4(float *p, float4 v) { *reinterpret_cast<float4 *>(p) = v; }
__device__ __forceinline__ float dot4(float4 a, float4 b) { return a.x * b.x + a.y * b.y + a.z * b.z + a.w * b.w; }
__device__ __forceinline__ float4 zero4() { return make_float4(0.f, 0.f, 0.f, 0.f); }
__device__ __forceinline__ float4 axpy4(float4 y, float a, float4 x)
{
    return make_float4(y.x + a * x.x, y.y + a * x.y, y.z + a * x.z, y.w + a * x.w);
}
__device__ __forceinline__ void atomic_add4(float *p, float4 v)
{
    atomicAdd(p + 0, v.x); atomicAdd(p + 1, v.y); atomicAdd(p + 2, v.z); atomicAdd(p + 3, v.w);
}

// Wmt[r][i dk + b][i dk + a] = Wmsg[r][i][a][b]: block-diagonal W_msg^T per head.
__global__ void hgt_msgT_weights_kernel(const float *Wmsg, int R, int D, int heads, float *Wmt)
{
    const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (idx >= (int64_t)R * D * D) return;
    const int r = (int)(idx / (D * D)), row = (int)(idx / D % D), col = (int)(idx % D);
    const int dk = D / heads, i = row / dk;
    float v = 0.f;
    if (col / dk == i) v = Wmsg[(((size_t)r * heads + i) * dk + (col - i * dk)) * dk + (row - i * dk)];
    Wmt[idx] = v;
}

// ---------------------------------------------------------------- destination-major pass
template <int H>
struct DStage {
    int eidx[kE];                  // source node of each edge
    int vptr[kE + 1];              // item-local first edge of each virtual segment
    int vpos[kE];                  // by-relation position of each virtual segment
    int dptr[kDst + 1];            // item-local first edge of each destination
    float dm[kDst * H];            // per destination and head: softmax max
    float dzi[kDst * H];           // and 1 / sum
};

struct DKArgs {
    int64_t n_items;
    const Item *items;
    const int32_t *item_slot, *dst_vsegptr, *vseg_ptr, *in_src, *vseg_pos;
    const float *KV, *QP, *dP, *saved;
    float *Sal, *Aac, *Bac, *sfin, *spart;
};

template <int D, int H>
__global__ __launch_bounds__(256) void hgt_bwd_dst_kernel(DKArgs k)
{
    constexpr int G = D / 4, GPB = 256 / G;
    constexpr int DKH = D / H, LH = DKH / 4;
    __shared__ DStage<H> stage[GPB];
    const int gl = threadIdx.x % G, gi = threadIdx.x / G;
    DStage<H> &st = stage[gi];
    const int64_t item = (int64_t)blockIdx.x * GPB + gi;
    const bool valid = item < k.n_items;
    int dst0 = 0, nd = 0, vs0 = 0, nv = 0, e0 = 0, ne = 0, slot = -1;
    if (valid) {
        const Item x = k.items[item];
        dst0 = x.dst0; nd = x.dst1 - x.dst0; vs0 = x.vs0; nv = x.vs1 - x.vs0;
        e0 = k.vseg_ptr[x.vs0]; ne = k.vseg_ptr[x.vs1] - e0;
        slot = k.item_slot[item];
        for (int j = gl; j < nv; j += G) {
            st.vptr[j] = k.vseg_ptr[vs0 + j] - e0;
            st.vpos[j] = k.vseg_pos[vs0 + j];
        }
        if (gl == 0) st.vptr[nv] = ne;
        auto dst_edge = [&](int jj) {
            int vs = k.dst_vsegptr[dst0 + jj];
            vs = vs < vs0 ? vs0 : (vs > vs0 + nv ? vs0 + nv : vs);
            return k.vseg_ptr[vs] - e0;
        };
        for (int j = gl; j < nd; j += G) st.dptr[j] = dst_edge(j);
        if (gl == 0) st.dptr[nd] = ne;
        for (int q = gl; q < nd * H; q += G) {
            const float2 sv = *reinterpret_cast<const float2 *>(k.saved + ((size_t)dst0 * H + q) * 2);
            st.dm[q] = sv.x;
            st.dzi[q] = sv.y > 0.f ? 1.f / sv.y : 0.f;
        }
        for (int e = gl; e < ne; e += G) st.eidx[e] = k.in_src[e0 + e];
    }
    __syncthreads();
    if (!valid) return;

    const int head = gl / LH;
    float4 sal = zero4(), aac = zero4(), bac = zero4();
    float sacc = 0.f;
    auto flush_dst = [&](int jj) {
        if (gl % LH == 0) {
            if (slot < 0) k.sfin[(size_t)(dst0 + jj) * H + head] = sacc;
            else k.spart[(size_t)slot * H + head] = sacc;
        }
        sacc = 0.f;
    };
    int j = 0, jv = 0;
    while (j < nd && st.dptr[j + 1] == st.dptr[j]) { flush_dst(j); ++j; }
    if (ne > 0) {
        // ping-pong batches of (K row, V row); each segment's QP and dP rows
        // are read once, while the segment before it runs
        float4 qn = ld4(k.QP + (size_t)vs0 * D + gl * 4), pn = ld4(k.dP + (size_t)vs0 * D + gl * 4);
        float4 qs = zero4(), ps = zero4();
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
                    if (e == st.vptr[jv]) {   // first edge of segment jv
                        qs = qn; ps = pn;
                        if (jv + 1 < nv) {
                            const size_t vrow = (size_t)(vs0 + jv + 1) * D + gl * 4;
                            qn = ld4(k.QP + vrow);
                            pn = ld4(k.dP + vrow);
                        }
                    }
                    const float a = gsum<LH>(dot4(Xk[u], qs));
                    const float da = gsum<LH>(dot4(Xv[u], ps));
                    const float al = __expf(a - st.dm[j * H + head]) * st.dzi[j * H + head];
                    sal = axpy4(sal, al, Xv[u]);
                    bac = axpy4(bac, al, Xk[u]);
                    aac = axpy4(aac, al * da, Xk[u]);
                    sacc += al * da;
                    if (e + 1 == st.vptr[jv + 1]) {
                        const size_t o = (size_t)st.vpos[jv] * D + gl * 4;
                        st4(k.Sal + o, sal);
                        st4(k.Aac + o, aac);
                        st4(k.Bac + o, bac);
                        sal = zero4(); aac = zero4(); bac = zero4();
                        ++jv;
                        if (e + 1 == st.dptr[j + 1]) {
                            flush_dst(j);
                            ++j;
                            while (j < nd && st.dptr[j + 1] == st.dptr[j]) { flush_dst(j); ++j; }
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
    while (j < nd) { flush_dst(j); ++j; }
}

// s of destinations split over several items: their slots summed in order.
__global__ __launch_bounds__(256) void hgt_bwd_merge_s_kernel(int64_t n_split, int heads,
                                                              const int32_t *split_dst,
                                                              const int32_t *split_slotptr,
                                                              const float *spart, float *sfin)
{
    const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (idx >= n_split * heads) return;
    const int64_t i = idx / heads;
    const int hh = (int)(idx % heads);
    float s = 0.f;
    for (int sl = split_slotptr[i]; sl < split_slotptr[i + 1]; ++sl) s += spart[(size_t)sl * heads + hh];
    sfin[(size_t)split_dst[i] * heads + hh] = s;
}

// Per destination and head, (max, 1 / sum, s, 0) in one 16-byte record, so that
// the source-major pass reads one line per out-edge for them instead of two.
__global__ __launch_bounds__(256) void hgt_bwd_pack_kernel(int64_t n, const float *saved, const float *sfin,
                                                           float4 *rec)
{
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n) return;
    const float2 mz = *reinterpret_cast<const float2 *>(saved + i * 2);
    rec[i] = make_float4(mz.x, mz.y > 0.f ? 1.f / mz.y : 0.f, sfin[i], 0.f);
}

// dQP = A - s_t B per by-relation segment row (head blocks of dk features).
__global__ __launch_bounds__(256) void hgt_bwd_dqp_kernel(int64_t V, int D, int heads, const int32_t *vsegdst_byrel,
                                                          const float *A, const float *B,
                                                          const float *sfin, float *dQP)
{
    const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;   // (row, float4)
    if (idx >= V * (D / 4)) return;
    const int64_t row = idx / (D / 4);
    const int f4 = (int)(idx % (D / 4));
    const float sv = sfin[(size_t)vsegdst_byrel[row] * heads + (f4 * 4) / (D / heads)];
    st4(dQP + idx * 4, axpy4(ld4(A + idx * 4), -sv, ld4(B + idx * 4)));
}

// ---------------------------------------------------------------- source-major pass
struct SStageH {
    int ev[kE];          // virtual segment (QP / dP row) of each out-edge
    int et[kE];          // its destination
    int enode[kE];       // item-local source of each out-edge
    int optr[kDst + 1];  // item-local first out-edge of each source
};

struct SKArgs {
    int64_t n_items;
    const Item *items;
    const int32_t *out_ptr;
    const int32_t *out_vs, *out_dst;   // per out-edge: vseg (QP / dP row) and destination, read in order
    const float *KV, *QP, *dP;
    const float4 *rec;   // [N, H] (max, 1 / sum, s, 0) per destination and head
    float *dKV;          // [N, 3D] dK | dV | dQ rows: dK | dV of split sources zero on entry,
                         // of every other source written here
};

template <int D, int H>
__global__ __launch_bounds__(256) void hgt_bwd_src_kernel(SKArgs k)
{
    constexpr int G = D / 4, GPB = 256 / G;
    constexpr int DKH = D / H, LH = DKH / 4;
    __shared__ SStageH stage[GPB];
    const int gl = threadIdx.x % G, gi = threadIdx.x / G;
    SStageH &st = stage[gi];
    const int64_t item = (int64_t)blockIdx.x * GPB + gi;
    const bool valid = item < k.n_items;
    int n0 = 0, nn = 0, q0 = 0, nq = 0;
    bool split = false;   // a piece of a source whose out-edges span several items
    if (valid) {
        const Item x = k.items[item];
        n0 = x.dst0; nn = x.dst1 - x.dst0; q0 = x.vs0; nq = x.vs1 - x.vs0;
        split = nn == 1 && k.out_ptr[n0 + 1] - k.out_ptr[n0] > nq;
        for (int e = gl; e < nq; e += G) {
            st.ev[e] = k.out_vs[q0 + e];
            st.et[e] = k.out_dst[q0 + e];
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
    if (!valid) return;
    // sources of a bundle without out-edges get zero rows
    for (int jj = 0; jj < nn; ++jj)
        if (st.optr[jj + 1] == st.optr[jj]) {
            float *p = k.dKV + (size_t)(n0 + jj) * (3 * D) + gl * 4;
            st4(p, zero4());
            st4(p + D, zero4());
        }
    if (nq == 0) return;
    const int head = gl / LH;
    int j = 0;
    while (st.optr[j + 1] == st.optr[j]) ++j;   // first source with out-edges
    float4 dk = zero4(), dv = zero4();
    // ping-pong batches of (K row, V row of the source, QP and dP rows of the
    // segment, the destination's max, sum and s for this head)
    float4 Ak[kU], Av[kU], Aq[kU], Ap[kU], Bk[kU], Bv[kU], Bq[kU], Bp[kU];
    float4 Am[kU], Bm[kU];
    auto load = [&](float4 (&Xk)[kU], float4 (&Xv)[kU], float4 (&Xq)[kU], float4 (&Xp)[kU],
                    float4 (&Xm)[kU], int b0) {
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int e = b0 + u < nq ? b0 + u : nq - 1;
            const size_t row = (size_t)(n0 + st.enode[e]) * (2 * D);
            const size_t vrow = (size_t)st.ev[e] * D;
            const size_t th = (size_t)st.et[e] * H + head;
            Xk[u] = ld4(k.KV + row + gl * 4);
            Xv[u] = ld4(k.KV + row + D + gl * 4);
            Xq[u] = ld4(k.QP + vrow + gl * 4);
            Xp[u] = ld4(k.dP + vrow + gl * 4);
            Xm[u] = k.rec[th];
        }
    };
    auto consume = [&](const float4 (&Xk)[kU], const float4 (&Xv)[kU], const float4 (&Xq)[kU],
                       const float4 (&Xp)[kU], const float4 (&Xm)[kU], int b0) {
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int e = b0 + u;
            if (e < nq) {
                const float a = gsum<LH>(dot4(Xk[u], Xq[u]));
                const float dal = gsum<LH>(dot4(Xv[u], Xp[u]));
                const float al = __expf(a - Xm[u].x) * Xm[u].y;
                dk = axpy4(dk, al * (dal - Xm[u].z), Xq[u]);
                dv = axpy4(dv, al, Xp[u]);
                if (e + 1 == st.optr[j + 1]) {   // the source's last out-edge in this item
                    float *p = k.dKV + (size_t)(n0 + j) * (3 * D) + gl * 4;
                    if (split) {
                        atomic_add4(p, dk);
                        atomic_add4(p + D, dv);
                    } else {
                        st4(p, dk);
                        st4(p + D, dv);
                    }
                    dk = zero4(); dv = zero4();
                    ++j;
                    while (j < nn && st.optr[j + 1] == st.optr[j]) ++j;
                }
            }
        }
    };
    load(Ak, Av, Aq, Ap, Am, 0);
    __builtin_amdgcn_sched_barrier(0);
    for (int eb = 0; eb < nq; eb += 2 * kU) {
        load(Bk, Bv, Bq, Bp, Bm, eb + kU);
        __builtin_amdgcn_sched_barrier(0);
        consume(Ak, Av, Aq, Ap, Am, eb);
        load(Ak, Av, Aq, Ap, Am, eb + 2 * kU);
        __builtin_amdgcn_sched_barrier(0);
        consume(Bk, Bv, Bq, Bp, Bm, eb + kU);
    }
}

// Per relation: dWatt, dWmsg from the head blocks of OT = sum dQP^T Q and
// M2 = sum Salpha^T dagg, and dmu = scale * <OT head blocks, Watt> (fixed order).
__global__ __launch_bounds__(256) void hgt_bwd_rel_kernel(const float *OT, const float *M2, const float *Watt,
                                                          const float *mu, float scale, int D, int heads,
                                                          float *dWatt, float *dWmsg, float *dmu)
{
    __shared__ float red[256];
    const int r = blockIdx.x, tid = threadIdx.x;
    const int dk = D / heads, n = heads * dk * dk;
    float part = 0.f;
    for (int idx = tid; idx < n; idx += 256) {
        const int i = idx / (dk * dk), p = idx / dk % dk, q = idx % dk;
        const size_t src = ((size_t)r * D + i * dk + p) * D + i * dk + q;
        const float ot = OT[src];
        dWatt[(size_t)r * n + idx] = mu[r] * scale * ot;
        dWmsg[(size_t)r * n + idx] = M2[src];
        part += ot * Watt[(size_t)r * n + idx];
    }
    red[tid] = part;
    __syncthreads();
    if (tid == 0) {
        float s = 0.f;
        for (int t = 0; t < 256; ++t) s += red[t];
        dmu[r] = scale * s;
    }
}

// zero the first w floats (w a multiple of 4) of the rows (stride ld) listed in rows
__global__ __launch_bounds__(256) void zero_rows_kernel(const int32_t *rows, int64_t n, int w, int ld, float *p)
{
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x, q = w / 4;
    if (i < n * q) st4(p + (size_t)rows[i / q] * ld + (i % q) * 4, zero4());
}

// Wc[t][n][j D + k] = W_j[t][n][k] for (W_0, W_1, W_2) = (Wk, Wv, Wq): the three
// transposed weights side by side, so that dh = [dK | dV | dQ] Wc^T is one GEMM.
__global__ __launch_bounds__(256) void hgt_cat_weights_kernel(const float *Wk, const float *Wv, const float *Wq,
                                                              int T, int D, float *Wc)
{
    const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (idx >= (int64_t)T * D * 3 * D) return;
    const int64_t row = idx / (3 * D);
    const int c = (int)(idx % (3 * D)), j = c / D, k = c % D;
    const float *W = j == 0 ? Wk : (j == 1 ? Wv : Wq);
    Wc[idx] = W[row * D + k];
}

inline unsigned blocks_for(int64_t n, int per_block) { return (unsigned)((n + per_block - 1) / per_block); }
inline size_t pad256(size_t b) { return (b + 255) & ~size_t(255); }

struct HgtBwdWs {
    float *KV, *Q, *Wqp, *QP, *agg, *partial, *saved, *dagg, *Wmt, *dP, *Sal, *Aac, *Bac, *sfin,
        *spart, *dQP, *Tq, *dQ, *dKV, *chunks, *OT, *M2, *rec, *Wc, *Wf;
};

size_t hgt_bwd_layout(const rgnn_graph *g, int D, int H, void *base, HgtBwdWs *w)
{
    char *b = (char *)base;
    size_t off = 0;
    auto take = [&](size_t n) {
        float *p = b ? (float *)(b + off) : nullptr;
        off += pad256(std::max<size_t>(n, 1) * sizeof(float));
        return p;
    };
    const size_t N = (size_t)g->N, V = (size_t)g->V, R = (size_t)g->R;
    const size_t slots = (size_t)g->n_slots;
    const size_t nchunks = (size_t)std::max<int64_t>(std::max(g->n_tiles_outer, g->n_tiles_types_outer), 1);
    HgtBwdWs x{};
    x.KV = take(N * 2 * D); x.Q = take(N * D); x.Wqp = take(R * D * D); x.QP = take(V * D);
    x.agg = take(N * D); x.partial = take(slots * (2 * H + D)); x.saved = take(N * H * 2);
    x.dagg = take(N * D); x.Wmt = take(R * D * D); x.dP = take(V * D);
    x.Sal = take(V * D); x.Aac = take(V * D); x.Bac = take(V * D);
    x.sfin = take(N * H); x.spart = take(slots * H);
    x.dQP = take(V * D); x.Tq = take(V * D); x.dKV = take(N * 3 * D);
    x.dQ = x.dKV ? x.dKV + 2 * D : nullptr;   // dK | dV | dQ side by side per node
    x.Wc = take((size_t)g->T * D * 3 * D);
    x.chunks = take(nchunks * D * D); x.OT = take(R * D * D); x.M2 = take(R * D * D);
    x.rec = take(N * H * 4);
    x.Wf = take(R * D * D);
    if (w) *w = x;
    return off;
}

// Y = X W[type]^T over the nodes grouped by type (typed GEMM, B = W^T).
rgnn_status node_gemm_t(const rgnn_graph *g, int D, const float *X, int64_t ldx, const float *W, float *Y,
                        const float *residual, int accumulate, hipStream_t s)
{
    GemmArgs ga;
    ga.split_bf16 = 1;
    ga.X = X; ga.ldx = ldx; ga.gather = g->dev.ntype_perm; ga.scatter = g->dev.ntype_perm;
    ga.W[0] = W; ga.trans_b = 1; ga.K = D; ga.Nc = D;
    ga.tiles = g->dev.tiles_nodes; ga.ntiles = g->n_tiles_nodes;
    ga.Y = Y; ga.ldy = D;
    if (residual) { ga.ep.residual = residual; ga.ep.ld_res = D; }
    ga.ep.accumulate = accumulate;
    return launch_typed_gemm(ga, s);
}

// dW[type] = sum over the nodes n of the type of X[n]^T Y[n].
rgnn_status type_outer(const rgnn_graph *g, int D, const float *X, int ldx, const float *Y, int ldy, float *chunks,
                       float *dW, hipStream_t s)
{
    rgnn_status st = launch_outer_chunks(g->dev.tiles_types_outer, g->n_tiles_types_outer, g->dev.ntype_perm, 1,
                                         X, ldx, Y, ldy, chunks, D, s);
    if (st != RGNN_OK) return st;
    return launch_chunk_sum(chunks, g->dev.types_chunkptr, g->T, dW, D, s);
}

template <int D>
rgnn_status hgt_backward_d(const rgnn_graph *g, const float *h, const float *Wk, const float *Wq,
                           const float *Wv, const float *Wa, const float *Watt, const float *Wmsg,
                           const float *mu, int H, float att_scale, int flags, const float *Gm,
                           const float *saved, float *dh, float *dWk, float *dWq, float *dWv, float *dWa,
                           float *dWatt, float *dWmsg, float *dmu, void *ws, hipStream_t s)
{
    constexpr int G = D / 4, GPB = 256 / G;
    const bool a_linear = (flags & RGNN_FLAG_A_LINEAR) != 0;
    HgtBwdWs w;
    hgt_bwd_layout(g, D, H, ws, &w);
    rgnn_status st;
    hipError_t e;
    // ---- forward recomputation: K | V | Q, the segment queries and, without the
    //      forward's statistics, the traversal that yields them and agg
    const float *stats = saved ? saved : w.saved;
    {
        GemmArgs ga;
        ga.split_bf16 = 1;
        ga.X = h; ga.ldx = D; ga.gather = g->dev.ntype_perm; ga.scatter = g->dev.ntype_perm;
        ga.K = D;
        ga.tiles = g->dev.tiles_nodes; ga.ntiles = g->n_tiles_nodes;
        if (D == 64) {   // K | V | Q in one GEMM
            ga.W[0] = Wk; ga.W[1] = Wv; ga.W[2] = Wq; ga.nparts = 3;
            ga.Nc = 3 * D;
            ga.Y = w.KV; ga.ldy = 2 * D;
            ga.ep.Y2 = w.Q; ga.ep.ldy2 = D; ga.ep.split = 2 * D;
            if ((st = launch_typed_gemm(ga, s)) != RGNN_OK) return st;
        } else {
            ga.Nc = D;
            const float *Wp[3] = {Wk, Wv, Wq};
            float *Yp[3] = {w.KV, w.KV + D, w.Q};
            const int64_t ld[3] = {2 * D, 2 * D, D};
            for (int p = 0; p < 3; ++p) {
                ga.W[0] = Wp[p]; ga.Y = Yp[p]; ga.ldy = ld[p];
                if ((st = launch_typed_gemm(ga, s)) != RGNN_OK) return st;
            }
        }
    }
    if ((st = launch_hgt_qp_weights(Watt, mu, att_scale, g->R, D, H, w.Wqp, s)) != RGNN_OK) return st;
    {
        // the segment queries exactly as the forward forms them (with the query
        // projection folded into the per-relation weight when the relations
        // are typed), so that the recomputed scores match its statistics
        const bool fold_q = g->rel_dst_typed && !(D == 128 && hgt_fused_query_fits(g->R, D, H));
        if (fold_q &&
            (st = launch_hgt_qp_fold(Wq, Watt, mu, att_scale, g->dev.rel_dsttype, g->R, D, H, w.Wf, s)) != RGNN_OK)
            return st;
        GemmArgs gq;
        gq.split_bf16 = 1;
        gq.X = fold_q ? h : w.Q; gq.ldx = D; gq.gather = g->dev.vsegdst_byrel; gq.scatter = g->dev.vseg_byrel;
        gq.W[0] = fold_q ? w.Wf : w.Wqp; gq.K = D; gq.Nc = D;
        gq.tiles = g->dev.tiles_vsegs; gq.ntiles = g->n_tiles_vsegs;
        gq.Y = w.QP; gq.ldy = D; gq.ep.diag_blocks = fold_q ? 1 : H;
        if ((st = launch_typed_gemm(gq, s)) != RGNN_OK) return st;
    }
    if (!saved) {
        HgtArgs ha;
        ha.g = g; ha.KV = w.KV; ha.QP = w.QP; ha.Wmsg = Wmsg;
        ha.heads = H; ha.d = D; ha.agg = w.agg; ha.partial = w.partial; ha.saved = w.saved;
        if ((st = launch_hgt_traverse(ha, s)) != RGNN_OK) return st;
        if ((st = launch_merge_partials(g, D, H, 1, w.partial, w.agg, w.saved, 0, s)) != RGNN_OK) return st;
    }
    // ---- output linear: dagg = G Wa^T, dWa = sum agg^T G per node type (with
    //      the forward's statistics agg is rebuilt after the destination pass)
    const float *dagg = Gm;
    if (a_linear) {
        if ((st = node_gemm_t(g, D, Gm, D, Wa, w.dagg, nullptr, 0, s)) != RGNN_OK) return st;
        dagg = w.dagg;
        if (dWa && !saved && (st = type_outer(g, D, w.agg, D, Gm, D, w.chunks, dWa, s)) != RGNN_OK) return st;
    }
    // ---- dP = dagg_t Wmsg[r]^T per segment (vseg order)
    if (g->V > 0) {
        {
            const int64_t n = (int64_t)g->R * D * D;
            LaunchScope ls("hgt_msgT_weights", s);
            hipLaunchKernelGGL(hgt_msgT_weights_kernel, dim3(blocks_for(n, 256)), dim3(256), 0, s, Wmsg, g->R, D, H,
                               w.Wmt);
        }
        if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "msgT weights launch");
        GemmArgs gp;
        gp.split_bf16 = 1;
        gp.X = dagg; gp.ldx = D; gp.gather = g->dev.vsegdst_byrel; gp.scatter = g->dev.vseg_byrel;
        gp.W[0] = w.Wmt; gp.K = D; gp.Nc = D;
        gp.tiles = g->dev.tiles_vsegs; gp.ntiles = g->n_tiles_vsegs;
        gp.Y = w.dP; gp.ldy = D; gp.ep.diag_blocks = H;
        if ((st = launch_typed_gemm(gp, s)) != RGNN_OK) return st;
    }
    // ---- destination-major pass: Salpha, A, B per segment; s per destination
    if (g->n_items > 0) {
        DKArgs k{};
        k.n_items = g->n_items; k.items = g->dev.items; k.item_slot = g->dev.item_slot;
        k.dst_vsegptr = g->dev.dst_vsegptr; k.vseg_ptr = g->dev.vseg_ptr; k.in_src = g->dev.in_src;
        k.vseg_pos = g->dev.vseg_pos;
        k.KV = w.KV; k.QP = w.QP; k.dP = w.dP; k.saved = stats;
        k.Sal = w.Sal; k.Aac = w.Aac; k.Bac = w.Bac; k.sfin = w.sfin; k.spart = w.spart;
        const unsigned nb = blocks_for(g->n_items, GPB);
        {
            LaunchScope ls("hgt_bwd_dst", s);
            if (H == 1) hipLaunchKernelGGL((hgt_bwd_dst_kernel<D, 1>), dim3(nb), dim3(256), 0, s, k);
            else if (H == 2) hipLaunchKernelGGL((hgt_bwd_dst_kernel<D, 2>), dim3(nb), dim3(256), 0, s, k);
            else if constexpr (D >= 64) {
                if (H == 4) hipLaunchKernelGGL((hgt_bwd_dst_kernel<D, 4>), dim3(nb), dim3(256), 0, s, k);
                else if constexpr (D >= 128) hipLaunchKernelGGL((hgt_bwd_dst_kernel<D, 8>), dim3(nb), dim3(256), 0, s, k);
            }
        }
        if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "hgt_bwd_dst launch");
    }
    if (g->n_split > 0) {
        {
            LaunchScope ls("hgt_bwd_merge_s", s);
            hipLaunchKernelGGL(hgt_bwd_merge_s_kernel, dim3(blocks_for(g->n_split * H, 256)), dim3(256), 0, s,
                               g->n_split, H, g->dev.split_dst, g->dev.split_slotptr, w.spart, w.sfin);
        }
        if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "hgt_bwd_merge_s launch");
    }
    // ---- agg_t = sum over t's segments of Salpha_vs Wmsg[r] (the messages are
    //      linear in V_s, so the alpha-weighted V sums of the destination pass
    //      give the forward's aggregate), then dWa = sum agg^T G per node type
    if (a_linear && dWa && saved) {
        if (g->V > 0) {
            GemmArgs gm;
            gm.split_bf16 = 1;
            gm.X = w.Sal; gm.ldx = D; gm.W[0] = w.Wmt; gm.trans_b = 1; gm.K = D; gm.Nc = D;
            gm.tiles = g->dev.tiles_vsegs; gm.ntiles = g->n_tiles_vsegs;
            gm.Y = w.Tq; gm.ldy = D; gm.scatter = g->dev.vseg_byrel; gm.ep.diag_blocks = H;
            if ((st = launch_typed_gemm(gm, s)) != RGNN_OK) return st;
        }
        if ((st = launch_vseg_reduce(g, w.Tq, nullptr, D, w.agg, 0, 0, s)) != RGNN_OK) return st;
        if ((st = type_outer(g, D, w.agg, D, Gm, D, w.chunks, dWa, s)) != RGNN_OK) return st;
    }
    // ---- dQP, dQ and the per-relation weight gradients
    if (g->V > 0) {
        {
            LaunchScope ls("hgt_bwd_dqp", s);
            hipLaunchKernelGGL(hgt_bwd_dqp_kernel, dim3(blocks_for(g->V * (D / 4), 256)), dim3(256), 0, s, g->V,
                               D, H, g->dev.vsegdst_byrel, w.Aac, w.Bac, w.sfin, w.dQP);
        }
        if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "hgt_bwd_dqp launch");
        GemmArgs gt;
        gt.split_bf16 = 1;
        gt.X = w.dQP; gt.ldx = D; gt.W[0] = w.Wqp; gt.trans_b = 1; gt.K = D; gt.Nc = D;
        gt.tiles = g->dev.tiles_vsegs; gt.ntiles = g->n_tiles_vsegs;
        gt.Y = w.Tq; gt.ldy = D; gt.scatter = g->dev.vseg_byrel; gt.ep.diag_blocks = H;
        if ((st = launch_typed_gemm(gt, s)) != RGNN_OK) return st;
    }
    if ((st = launch_vseg_reduce(g, w.Tq, nullptr, D, w.dQ, 0, 0, s, 3 * D)) != RGNN_OK) return st;
    if (g->V > 0) {
        if ((st = launch_outer_chunks(g->dev.tiles_outer, g->n_tiles_outer, g->dev.vsegdst_byrel, 0, w.dQP, D, w.Q,
                                      D, w.chunks, D, s)) != RGNN_OK)
            return st;
    }
    if ((st = launch_chunk_sum(w.chunks, g->dev.rel_chunkptr, g->R, w.OT, D, s)) != RGNN_OK) return st;
    if (g->V > 0) {
        if ((st = launch_outer_chunks(g->dev.tiles_outer, g->n_tiles_outer, g->dev.vsegdst_byrel, 0, w.Sal, D, dagg,
                                      D, w.chunks, D, s)) != RGNN_OK)
            return st;
    }
    if ((st = launch_chunk_sum(w.chunks, g->dev.rel_chunkptr, g->R, w.M2, D, s)) != RGNN_OK) return st;
    if (g->R > 0) {
        {
            LaunchScope ls("hgt_bwd_rel", s);
            hipLaunchKernelGGL(hgt_bwd_rel_kernel, dim3((unsigned)g->R), dim3(256), 0, s, w.OT, w.M2, Watt, mu,
                               att_scale, D, H, dWatt, dWmsg, dmu);
        }
        if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "hgt_bwd_rel launch");
    }
    if (g->N > 0) {
        {
            LaunchScope ls("hgt_bwd_pack", s);
            hipLaunchKernelGGL(hgt_bwd_pack_kernel, dim3(blocks_for(g->N * H, 256)), dim3(256), 0, s, g->N * H,
                               stats, w.sfin, reinterpret_cast<float4 *>(w.rec));
        }
        if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "hgt_bwd_pack launch");
    }
    // ---- source-major pass: dK | dV per source (the rows of sources split over
    //      several items are summed with atomics and start from zero)
    if (g->n_osplit > 0) {
        {
            LaunchScope ls("zero", s);
            hipLaunchKernelGGL(zero_rows_kernel, dim3(blocks_for(g->n_osplit * (2 * D / 4), 256)), dim3(256), 0, s,
                               g->dev.osplit, g->n_osplit, 2 * D, 3 * D, w.dKV);
        }
        if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "zero launch");
    }
    if (g->n_oitems > 0) {
        SKArgs k{};
        k.n_items = g->n_oitems; k.items = g->dev.oitems; k.out_ptr = g->dev.out_ptr;
        k.out_vs = g->dev.out_vs; k.out_dst = g->dev.out_dst;
        k.KV = w.KV; k.QP = w.QP; k.dP = w.dP; k.rec = reinterpret_cast<const float4 *>(w.rec); k.dKV = w.dKV;
        const unsigned nb = blocks_for(g->n_oitems, GPB);
        {
            LaunchScope ls("hgt_bwd_src", s);
            if (H == 1) hipLaunchKernelGGL((hgt_bwd_src_kernel<D, 1>), dim3(nb), dim3(256), 0, s, k);
            else if (H == 2) hipLaunchKernelGGL((hgt_bwd_src_kernel<D, 2>), dim3(nb), dim3(256), 0, s, k);
            else if constexpr (D >= 64) {
                if (H == 4) hipLaunchKernelGGL((hgt_bwd_src_kernel<D, 4>), dim3(nb), dim3(256), 0, s, k);
                else if constexpr (D >= 128) hipLaunchKernelGGL((hgt_bwd_src_kernel<D, 8>), dim3(nb), dim3(256), 0, s, k);
            }
        }
        if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "hgt_bwd_src launch");
    }
    // ---- node-level linears: dh and the per-type weight gradients
    const float *res = (flags & RGNN_FLAG_RESIDUAL) ? Gm : nullptr;
    if constexpr (D <= 64) {   // dh = [dK | dV | dQ] [Wk | Wv | Wq]^T in one GEMM (K = 3D)
        if (g->T > 0) {
            const int64_t n = (int64_t)g->T * D * 3 * D;
            LaunchScope ls("hgt_cat_weights", s);
            hipLaunchKernelGGL(hgt_cat_weights_kernel, dim3(blocks_for(n, 256)), dim3(256), 0, s, Wk, Wv, Wq, g->T,
                               D, w.Wc);
        }
        if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "cat weights launch");
        GemmArgs ga;
        ga.split_bf16 = 1;
        ga.X = w.dKV; ga.ldx = 3 * D; ga.gather = g->dev.ntype_perm; ga.scatter = g->dev.ntype_perm;
        ga.W[0] = w.Wc; ga.trans_b = 1; ga.K = 3 * D; ga.Nc = D;
        ga.tiles = g->dev.tiles_nodes; ga.ntiles = g->n_tiles_nodes;
        ga.Y = dh; ga.ldy = D;
        if (res) { ga.ep.residual = res; ga.ep.ld_res = D; }
        if ((st = launch_typed_gemm(ga, s)) != RGNN_OK) return st;
    } else {   // a 3D-deep weight tile would not fit LDS at D = 128
        if ((st = node_gemm_t(g, D, w.dKV, 3 * D, Wk, dh, res, 0, s)) != RGNN_OK) return st;
        if ((st = node_gemm_t(g, D, w.dKV + D, 3 * D, Wv, dh, nullptr, 1, s)) != RGNN_OK) return st;
        if ((st = node_gemm_t(g, D, w.dQ, 3 * D, Wq, dh, nullptr, 1, s)) != RGNN_OK) return st;
    }
    if ((st = type_outer(g, D, h, D, w.dKV, 3 * D, w.chunks, dWk, s)) != RGNN_OK) return st;
    if ((st = type_outer(g, D, h, D, w.dKV + D, 3 * D, w.chunks, dWv, s)) != RGNN_OK) return st;
    if ((st = type_outer(g, D, h, D, w.dQ, 3 * D, w.chunks, dWq, s)) != RGNN_OK) return st;
    return RGNN_OK;
}

}  // namespace

rgnn_status hgt_backward_impl(const rgnn_graph *g, const float *h, const float *Wk, const float *Wq,
                              const float *Wv, const float *Wa, const float *Watt, const float *Wmsg,
                              const float *mu, int d, int heads, float att_scale, int flags,
                              const float *Gm, const float *saved, float *dh, float *dWk, float *dWq,
                              float *dWv, float *dWa, float *dWatt, float *dWmsg, float *dmu, void *ws,
                              size_t ws_bytes, hipStream_t s, size_t *need)
{
    const int H = heads;
    const size_t bytes = hgt_bwd_layout(g, d, H > 0 ? H : 1, nullptr, nullptr);
    if (need) { *need = bytes; return RGNN_OK; }
    if (d != 32 && d != 64 && d != 128) return fail(RGNN_EUNSUPPORTED, "HGT backward supports d = 32, 64 or 128");
    if (!(H == 1 || H == 2 || H == 4 || H == 8) || d / H < 16)
        return fail(RGNN_EUNSUPPORTED, "HGT backward heads must be 1, 2, 4 or 8 with d / heads >= 16");
    if (!ws || ws_bytes < bytes)
        return fail(RGNN_EINVAL, "workspace too small: need " + std::to_string(bytes) + " bytes");
#define HB(D) hgt_backward_d<D>(g, h, Wk, Wq, Wv, Wa, Watt, Wmsg, mu, H, att_scale, flags, Gm, saved, dh, dWk, \
                                dWq, dWv, dWa, dWatt, dWmsg, dmu, ws, s)
    if (d == 32) return HB(32);
    if (d == 64) return HB(64);
    return HB(128);
#undef HB
}

}  // namespace rgnn
