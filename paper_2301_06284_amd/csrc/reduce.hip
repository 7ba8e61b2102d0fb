// reduce.hip -- per-destination reductions and small helpers of the layers:
// merging the partial softmax states of destinations split over several work
// items, softmax statistics and sums over (dst, rel) segment rows for the
// aggregate-first plan, the reordered attention vectors
// W_r w[r] (linear operator reordering), fill / ReLU / add.
// Every reduction runs in a fixed order, so results are reproducible bit for bit.
#include "rgnn_internal.h"
#include "wave_ops.h"

namespace rgnn {

namespace {

__device__ __forceinline__ float4 ld4(const float *p) { return *reinterpret_cast<const float4 *>(p); }
__device__ __forceinline__ void st4(float *p, float4 v) { *reinterpret_cast<float4 *>(p) = v; }
__device__ __forceinline__ float4 scale4(float4 a, float s) { return make_float4(a.x * s, a.y * s, a.z * s, a.w * s); }
__device__ __forceinline__ float dot4(float4 a, float4 b) { return a.x * b.x + a.y * b.y + a.z * b.z + a.w * b.w; }
__device__ __forceinline__ float4 add4(float4 a, float4 b) { return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w); }
__device__ __forceinline__ float4 fma4(float4 a, float s, float4 c)
{
    return make_float4(a.x * s + c.x, a.y * s + c.y, a.z * s + c.z, a.w * s + c.w);
}
__device__ __forceinline__ float4 lin4(float4 a, float s, float4 b, float t)
{
    return make_float4(a.x * s + b.x * t, a.y * s + b.y * t, a.z * s + b.z * t, a.w * s + b.w * t);
}
__device__ __forceinline__ float4 relu4(float4 a)
{
    return make_float4(fmaxf(a.x, 0.f), fmaxf(a.y, 0.f), fmaxf(a.z, 0.f), fmaxf(a.w, 0.f));
}

// Softmax per (dst, rel) segment: a segment longer than kChunkEdges is cut into
// several virtual segments, each with its own (max m_i, sum s_i), stored at the
// segment's fused position fpos[i]; per virtual segment the scale
// exp(m_i - M) / Z of its (dst, rel) segment is written, and (M, Z) to
// saved[segment] when saved is not NULL.  Segments with more than kBigRange
// pieces are left to the block kernel.
__global__ __launch_bounds__(256) void vseg_stats_kernel(int64_t N, const int32_t *grp_vsegptr,
                                                         const int32_t *fpos, const float *vstat,
                                                         float *vscale, float *saved)
{
    const int64_t v = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (v >= N) return;
    const int b = grp_vsegptr[v], e = grp_vsegptr[v + 1];
    if (e - b > kBigRange) return;
    float M = -INFINITY;
    for (int i = b; i < e; ++i) M = fmaxf(M, vstat[(size_t)fpos[i] * 2]);
    float Z = 0.f;
    for (int i = b; i < e; ++i) {
        const float2 st = *reinterpret_cast<const float2 *>(vstat + (size_t)fpos[i] * 2);
        Z += st.y * __expf(st.x - M);
    }
    for (int i = b; i < e; ++i) vscale[i] = __expf(vstat[(size_t)fpos[i] * 2] - M) / Z;
    if (saved) *reinterpret_cast<float2 *>(saved + v * 2) = make_float2(M, Z);
}

// One workgroup per group with many segments: strided per-thread partial
// (max, sum), combined in thread order through LDS.
__global__ __launch_bounds__(256) void vseg_stats_big_kernel(const int32_t *big_grp,
                                                             const int32_t *grp_vsegptr,
                                                             const int32_t *fpos, const float *vstat,
                                                             float *vscale, float *saved)
{
    __shared__ float sm[256], ss[256];
    __shared__ float fin[2];
    const int v = big_grp[blockIdx.x];
    const int b = grp_vsegptr[v], e = grp_vsegptr[v + 1];
    float m = -INFINITY, s = 0.f;
    for (int i = b + (int)threadIdx.x; i < e; i += 256) {
        const float2 st = *reinterpret_cast<const float2 *>(vstat + (size_t)fpos[i] * 2);
        const float mi = st.x, si = st.y;
        const float mn = fmaxf(m, mi);
        s = s * __expf(m - mn) + si * __expf(mi - mn);
        m = mn;
    }
    sm[threadIdx.x] = m;
    ss[threadIdx.x] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
        float M = -INFINITY;
        for (int t = 0; t < 256; ++t) M = fmaxf(M, sm[t]);
        float Z = 0.f;
        for (int t = 0; t < 256; ++t)
            if (ss[t] > 0.f) Z += ss[t] * __expf(sm[t] - M);
        fin[0] = M;
        fin[1] = Z;
        if (saved) *reinterpret_cast<float2 *>(saved + (size_t)v * 2) = make_float2(M, Z);
    }
    __syncthreads();
    const float M = fin[0], Zi = 1.f / fin[1];
    for (int i = b + (int)threadIdx.x; i < e; i += 256) vscale[i] = __expf(vstat[(size_t)fpos[i] * 2] - M) * Zi;
}

// Destinations with more than kBigRange segments get one workgroup of NTH
// threads each, at the front of the grid (largest first, so they start
// early and overlap the rest): every group of D/4 lanes sums a strided subset
// of the rows (U in flight), the group sums are then added in group order.
template <int D, int NTH, int U>
__device__ __forceinline__ void vseg_reduce_big(int v, const int32_t *dst_vsegptr, const float *T,
                                                const float *scale, float *out, int64_t ldo, int accumulate,
                                                int relu)
{
    constexpr int G = D / 4, NG = NTH / G;
    __shared__ float4 part[NG * G];
    const int gl = threadIdx.x % G, gi = threadIdx.x / G;
    const int b = dst_vsegptr[v], e = dst_vsegptr[v + 1];
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int i0 = b + gi; i0 < e; i0 += U * NG) {
        float4 t[U];
        float sc[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int i = i0 + u * NG;
            if (i < e) {
                t[u] = ld4(T + (size_t)i * D + gl * 4);
                sc[u] = scale ? scale[i] : 1.f;
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (i0 + u * NG < e) acc = scale ? fma4(t[u], sc[u], acc) : add4(acc, t[u]);
    }
    part[gi * G + gl] = acc;
    __syncthreads();
    if (gi == 0) {
        float4 tot = accumulate ? ld4(out + (size_t)v * ldo + gl * 4) : make_float4(0.f, 0.f, 0.f, 0.f);
        for (int j = 0; j < NG; ++j) tot = add4(tot, part[j * G + gl]);
        st4(out + (size_t)v * ldo + gl * 4, relu ? relu4(tot) : tot);
    }
}

// out_v (+)= sum of the (scaled) transformed segment rows of v (then optional
// ReLU), out rows ldo floats apart.  Blocks [0, nbig) take the destinations of
// big_vdst; the others a group of D/4 lanes per destination: every one of the
// N nodes, or the N listed in vlist (those the fused kernel did not finish).
template <int D>
__global__ __launch_bounds__(256) void vseg_reduce_kernel(int64_t N, int64_t nbig, const int32_t *big_vdst,
                                                          const int32_t *dst_vsegptr,
                                                          const float *T, const float *scale,
                                                          float *out, int64_t ldo, int accumulate, int relu,
                                                          const int32_t *vlist)
{
    if ((int64_t)blockIdx.x < nbig) {
        vseg_reduce_big<D, 256, 8>(big_vdst[blockIdx.x], dst_vsegptr, T, scale, out, ldo, accumulate, relu);
        return;
    }
    constexpr int G = D / 4, GPB = 256 / G;
    const int gl = threadIdx.x % G;
    const int64_t t = ((int64_t)blockIdx.x - nbig) * GPB + threadIdx.x / G;
    if (t >= N) return;
    const int64_t v = vlist ? (int64_t)vlist[t] : t;
    const int b = dst_vsegptr[v], e = dst_vsegptr[v + 1];
    if (e - b > kBigRange) return;
    float4 acc = accumulate ? ld4(out + (size_t)v * ldo + gl * 4) : make_float4(0.f, 0.f, 0.f, 0.f);
    // rows in batches of four (all in flight together), summed in segment order
    for (int i0 = b; i0 < e; i0 += 4) {
        float4 t[4];
        float sc[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            if (i0 + u < e) {
                t[u] = ld4(T + (size_t)(i0 + u) * D + gl * 4);
                sc[u] = scale ? scale[i0 + u] : 1.f;
            }
        }
#pragma unroll
        for (int u = 0; u < 4; ++u)
            if (i0 + u < e) acc = scale ? fma4(t[u], sc[u], acc) : add4(acc, t[u]);
    }
    st4(out + (size_t)v * ldo + gl * 4, relu ? relu4(acc) : acc);
}

// ---------------------------------------------------------------- softmax reduction
// Destinations with more than kBigRange segments: one workgroup of NTH threads
// each, at the front of the grid (largest first); every thread folds its strided share of the (max, sum)
// pairs into one online pair (four loads in flight), the maximum and the
// denominator follow by workgroup reductions; every thread then writes the
// weights exp(m_i - M) / Z of its share to scale[i] (segment order, so the row
// pass reads them without the fused-position indirection); then every group of
// D/4 lanes sums a strided subset of the rows (U in flight) and the group sums
// are added in group order.
template <int D, int NTH, int U>
__device__ __forceinline__ void softmax_reduce_big(int v, const int32_t *dst_vsegptr, const int32_t *fpos,
                                                   const float *vstat, const float *T, float *out,
                                                   float *saved, float *scale)
{
    constexpr int G = D / 4, NG = NTH / G, NWV = NTH / 64;
    __shared__ float red[NWV];
    __shared__ float4 part[NG * G];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int gl = tid % G, gi = tid / G;
    const int b = dst_vsegptr[v], e = dst_vsegptr[v + 1];
    float ml = -INFINITY, zl = 0.f;
    for (int i0 = b + tid; i0 < e; i0 += 4 * NTH) {
        float2 st[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int i = i0 + u * NTH;
            st[u] = i < e ? *reinterpret_cast<const float2 *>(vstat + (size_t)fpos[i] * 2) : make_float2(-INFINITY, 0.f);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            if (st[u].y > 0.f) {
                const float mn = fmaxf(ml, st[u].x);
                zl = zl * __expf(ml - mn) + st[u].y * __expf(st[u].x - mn);
                ml = mn;
            }
        }
    }
    // maximum
    float m = gmax<32>(ml);
    m = fmaxf(m, __shfl_xor(m, 32));
    if (lane == 0) red[wave] = m;
    __syncthreads();
    float M = red[0];
    for (int w = 1; w < NWV; ++w) M = fmaxf(M, red[w]);
    __syncthreads();
    // denominator
    float z = zl > 0.f ? zl * __expf(ml - M) : 0.f;
    z = gsum<32>(z);
    z += __shfl_xor(z, 32);
    if (lane == 0) red[wave] = z;
    __syncthreads();
    float Z = 0.f;
    for (int w = 0; w < NWV; ++w) Z += red[w];
    if (saved && tid == 0) *reinterpret_cast<float2 *>(saved + (size_t)v * 2) = make_float2(M, Z);
    const float inv = 1.f / Z;
    for (int i0 = b + tid; i0 < e; i0 += 4 * NTH) {
        float mu[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int i = i0 + u * NTH;
            mu[u] = i < e ? vstat[(size_t)fpos[i] * 2] : 0.f;
        }
#pragma unroll
        for (int u = 0; u < 4; ++u)
            if (i0 + u * NTH < e) scale[i0 + u * NTH] = __expf(mu[u] - M) * inv;
    }
    __syncthreads();   // the weights are read by other threads of the workgroup
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int i0 = b + gi; i0 < e; i0 += U * NG) {
        float4 t[U];
        float wu[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int i = i0 + u * NG;
            if (i < e) {
                t[u] = ld4(T + (size_t)i * D + gl * 4);
                wu[u] = scale[i];
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (i0 + u * NG < e) acc = fma4(t[u], wu[u], acc);
    }
    part[gi * G + gl] = acc;
    __syncthreads();
    if (gi == 0) {
        float4 tot = make_float4(0.f, 0.f, 0.f, 0.f);
        for (int j = 0; j < NG; ++j) tot = add4(tot, part[j * G + gl]);
        st4(out + (size_t)v * D + gl * 4, tot);
    }
}

// Softmax per destination finished and summed in one pass: per destination v
// with segments i (each with its own logit maximum m_i, sum s_i and
// exp-weighted transformed row T_i relative to m_i; (m_i, s_i) stored at the
// segment's fused position fpos[i]):
//   M = max_i m_i,  Z = sum_i s_i exp(m_i - M),  out_v = sum_i exp(m_i - M) / Z * T_i
// and saved[v] = (M, Z) ((0, 0) without in-edges); with vlist, only the N
// listed destinations (those the fused kernel did not finish).  Blocks [0, nbig) take the
// destinations of big_vdst; the others a group of D/4 lanes per destination,
// the statistics taken over the group's lanes (fixed butterfly), the rows
// summed in segment order.
template <int D>
__global__ __launch_bounds__(256) void softmax_reduce_kernel(int64_t N, int64_t nbig, const int32_t *big_vdst,
                                                             const int32_t *dst_vsegptr,
                                                             const int32_t *fpos, const float *vstat,
                                                             const float *T, float *out, float *saved,
                                                             float *scale, const int32_t *vlist)
{
    if ((int64_t)blockIdx.x < nbig) {
        softmax_reduce_big<D, 256, 8>(big_vdst[blockIdx.x], dst_vsegptr, fpos, vstat, T, out, saved, scale);
        return;
    }
    constexpr int G = D / 4, GPB = 256 / G;
    constexpr int NE = (kBigRange + G - 1) / G;   // statistics entries per lane
    const int gl = threadIdx.x % G;
    const int64_t t = ((int64_t)blockIdx.x - nbig) * GPB + threadIdx.x / G;
    if (t >= N) return;
    const int64_t v = vlist ? (int64_t)vlist[t] : t;
    const int b = dst_vsegptr[v], e = dst_vsegptr[v + 1];
    if (e - b > kBigRange) return;
    // rows in batches of four, two batches in flight; the first goes out before
    // the statistics are gathered (the rows do not depend on them)
    float4 ta[4], tb[4];
    auto load = [&](float4 (&t)[4], int i0) {
#pragma unroll
        for (int u = 0; u < 4; ++u)
            if (i0 + u < e) t[u] = ld4(T + (size_t)(i0 + u) * D + gl * 4);
    };
    load(ta, b);
    // lane gl holds the statistics of segments b + gl + j G
    float mi[NE], si[NE];
#pragma unroll
    for (int j = 0; j < NE; ++j) {
        const int i = b + gl + j * G;
        const float2 st = i < e ? *reinterpret_cast<const float2 *>(vstat + (size_t)fpos[i] * 2)
                                : make_float2(-INFINITY, 0.f);
        mi[j] = st.x;
        si[j] = st.y;
    }
    float M = mi[0];
#pragma unroll
    for (int j = 1; j < NE; ++j) M = fmaxf(M, mi[j]);
    M = gmax<G>(M);
    float z = 0.f;
#pragma unroll
    for (int j = 0; j < NE; ++j) z += si[j] > 0.f ? si[j] * __expf(mi[j] - M) : 0.f;
    const float Z = gsum<G>(z);
    if (saved && gl == 0) *reinterpret_cast<float2 *>(saved + (size_t)v * 2) = make_float2(b < e ? M : 0.f, Z);
    const float inv = Z > 0.f ? 1.f / Z : 0.f;
    float w[NE];
#pragma unroll
    for (int j = 0; j < NE; ++j) w[j] = si[j] > 0.f ? __expf(mi[j] - M) * inv : 0.f;
    // summed in segment order; segment b + r takes its weight from lane r % G
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    auto consume = [&](const float4 (&t)[4], int i0) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int r = i0 + u - b, jr = r / G;
            float x = w[0];
#pragma unroll
            for (int j = 1; j < NE; ++j) x = jr == j ? w[j] : x;
            const float wu = __shfl(x, r % G, G);
            if (i0 + u < e) acc = fma4(t[u], wu, acc);
        }
    };
    for (int i0 = b; i0 < e; i0 += 8) {
        const bool more = i0 + 4 < e;
        if (more) load(tb, i0 + 4);
        consume(ta, i0);
        if (!more) break;
        if (i0 + 8 < e) load(ta, i0 + 8);
        consume(tb, i0 + 4);
    }
    st4(out + (size_t)v * D + gl * 4, acc);
}

// ---------------------------------------------------------------- merges
// Combine the partials of destinations split over several items, in slot
// order (all maxima, then the records eight at a time in flight).  softmax:
// partial = (m, s) per head then acc[D]; else acc only.
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
    if (e - b > kBigRange) return;
    const int head = gl / LH;
    constexpr int U = 8;   // records in flight
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    if (SOFTMAX) {
        // every slot's maximum at once, then the records in batches of U
        float M = -INFINITY;
#pragma unroll
        for (int j = 0; j < kBigRange; ++j)
            M = fmaxf(M, b + j < e ? partial[(size_t)(b + j) * REC + head * 2] : -INFINITY);
        float Z = 0.f;
        for (int sl0 = b; sl0 < e; sl0 += U) {
            float4 a[U];
            float2 ms[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const float *pr = partial + (size_t)(sl0 + u < e ? sl0 + u : sl0) * REC;
                a[u] = ld4(pr + OFF + gl * 4);
                ms[u] = make_float2(pr[head * 2], pr[head * 2 + 1]);
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (sl0 + u >= e) break;
                const float c = __expf(ms[u].x - M);
                Z += ms[u].y * c;
                acc = lin4(acc, 1.f, a[u], c);
            }
        }
        acc = scale4(acc, Z > 0.f ? 1.f / Z : 0.f);
        if (saved && gl % LH == 0) {
            saved[((size_t)v * H + head) * 2] = M;
            saved[((size_t)v * H + head) * 2 + 1] = Z;
        }
    } else {
        for (int sl0 = b; sl0 < e; sl0 += U) {
            float4 a[U];
#pragma unroll
            for (int u = 0; u < U; ++u) a[u] = ld4(partial + (size_t)(sl0 + u < e ? sl0 + u : sl0) * REC + OFF + gl * 4);
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (sl0 + u >= e) break;
                acc = add4(acc, a[u]);
            }
        }
    }
    st4(out + (size_t)v * D + gl * 4, relu ? relu4(acc) : acc);
}

// Destinations split over many items, level 1: a 256-thread workgroup per
// chunk of at most kMergeChunk partials; each group of D/4 lanes merges a
// strided subset (four records in flight), group 0 merges the group states in
// group order and writes the chunk's merged record over its first partial
// (softmax: per head the maximum, the sum relative to it and the row sum;
// sums: the row sum).
template <int D, int H, bool SOFTMAX>
__global__ __launch_bounds__(256) void merge_chunk_kernel(const int32_t *chunk_lo, const int32_t *chunk_hi,
                                                          float *partial)
{
    constexpr int G = D / 4, NG = 256 / G, LH = D / H / 4;
    constexpr int REC = SOFTMAX ? 2 * H + D : 2 + D;
    constexpr int OFF = SOFTMAX ? 2 * H : 2;
    constexpr int U = 4;
    __shared__ float4 pacc[NG * G];
    __shared__ float pm[NG * H], ps[NG * H];
    const int gl = threadIdx.x % G, gi = threadIdx.x / G;
    const int b = chunk_lo[blockIdx.x], e = chunk_hi[blockIdx.x];
    const int head = gl / LH;
    float m = -INFINITY, s = 0.f;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int sl0 = b + gi; sl0 < e; sl0 += U * NG) {
        float4 a[U];
        float mi[U], si[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int sl = sl0 + u * NG;
            if (sl < e) {
                const float *pr = partial + (size_t)sl * REC;
                a[u] = ld4(pr + OFF + gl * 4);
                if (SOFTMAX) { mi[u] = pr[head * 2]; si[u] = pr[head * 2 + 1]; }
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (sl0 + u * NG >= e) break;
            if (SOFTMAX) {
                const float mn = fmaxf(m, mi[u]);
                const float c1 = __expf(m - mn), c2 = __expf(mi[u] - mn);
                s = s * c1 + si[u] * c2;
                acc = lin4(acc, c1, a[u], c2);
                m = mn;
            } else {
                acc = add4(acc, a[u]);
            }
        }
    }
    pacc[gi * G + gl] = acc;
    if (gl % LH == 0) { pm[gi * H + head] = m; ps[gi * H + head] = s; }
    __syncthreads();   // every partial of the chunk has been read
    if (gi != 0) return;
    float4 tot = make_float4(0.f, 0.f, 0.f, 0.f);
    float *pr = partial + (size_t)b * REC;
    if (SOFTMAX) {
        float M = -INFINITY;
        for (int j = 0; j < NG; ++j) M = fmaxf(M, pm[j * H + head]);
        float Z = 0.f;
        for (int j = 0; j < NG; ++j) {
            if (!(ps[j * H + head] > 0.f)) continue;
            const float c = __expf(pm[j * H + head] - M);
            Z += ps[j * H + head] * c;
            tot = lin4(tot, 1.f, pacc[j * G + gl], c);
        }
        if (gl % LH == 0) { pr[head * 2] = M; pr[head * 2 + 1] = Z; }
    } else {
        for (int j = 0; j < NG; ++j) tot = add4(tot, pacc[j * G + gl]);
    }
    st4(pr + OFF + gl * 4, tot);
}

// Level 2: a group of D/4 lanes per split destination merges its chunks'
// records in chunk order (four in flight) and writes the output row (and
// the softmax statistics).
template <int D, int H, bool SOFTMAX>
__global__ __launch_bounds__(256) void merge_chunks_final_kernel(int64_t nbig, const int32_t *big_split,
                                                                 const int32_t *split_dst,
                                                                 const int32_t *big_chunkptr,
                                                                 const int32_t *chunk_lo, const float *partial,
                                                                 float *out, float *saved, int relu)
{
    constexpr int G = D / 4, GPB = 256 / G, LH = D / H / 4;
    constexpr int REC = SOFTMAX ? 2 * H + D : 2 + D;
    constexpr int OFF = SOFTMAX ? 2 * H : 2;
    constexpr int U = 4;
    const int gl = threadIdx.x % G;
    const int64_t j = (int64_t)blockIdx.x * GPB + threadIdx.x / G;
    if (j >= nbig) return;
    const int v = split_dst[big_split[j]];
    const int c0 = big_chunkptr[j], c1 = big_chunkptr[j + 1];
    const int head = gl / LH;
    float m = -INFINITY, s = 0.f;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int cb = c0; cb < c1; cb += U) {
        float4 a[U];
        float mi[U], si[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (cb + u < c1) {
                const float *pr = partial + (size_t)chunk_lo[cb + u] * REC;
                a[u] = ld4(pr + OFF + gl * 4);
                if (SOFTMAX) { mi[u] = pr[head * 2]; si[u] = pr[head * 2 + 1]; }
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (cb + u >= c1) break;
            if (SOFTMAX) {
                if (!(si[u] > 0.f)) continue;
                const float mn = fmaxf(m, mi[u]);
                const float e1 = __expf(m - mn), e2 = __expf(mi[u] - mn);
                s = s * e1 + si[u] * e2;
                acc = lin4(acc, e1, a[u], e2);
                m = mn;
            } else {
                acc = add4(acc, a[u]);
            }
        }
    }
    if (SOFTMAX) {
        acc = scale4(acc, s > 0.f ? 1.f / s : 0.f);
        if (saved && gl % LH == 0) {
            saved[((size_t)v * H + head) * 2] = m;
            saved[((size_t)v * H + head) * 2 + 1] = s;
        }
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

// out[i, j] = in[i, j] for columns c0 <= j < c1, else 0 ([rows, d], row-major)
__global__ void mask_cols_kernel(const float *in, float *out, int64_t n, int d, int c0, int c1)
{
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n) return;
    const int j = (int)(i % d);
    out[i] = (j >= c0 && j < c1) ? in[i] : 0.f;
}

// saved[v, k] = in[v] for the (max, sum) pairs of one head ([N, 2] -> [N, H, 2])
__global__ void head_stats_scatter_kernel(const float *in, float *saved, int64_t N, int H, int k)
{
    const int64_t v = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (v >= N) return;
    *reinterpret_cast<float2 *>(saved + (v * H + k) * 2) = *reinterpret_cast<const float2 *>(in + v * 2);
}

// out[v] = saved[v, k] for the (max, sum) pairs of one head ([N, H, 2] -> [N, 2])
__global__ void head_stats_kernel(const float *saved, float *out, int64_t N, int H, int k)
{
    const int64_t v = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (v >= N) return;
    *reinterpret_cast<float2 *>(out + v * 2) = *reinterpret_cast<const float2 *>(saved + (v * H + k) * 2);
}

// Reordered attention vectors (linear operator reordering): for every row
// (r, i) of W_r, out[r, k, i] = W_r[i, k-cols] . v[r, k-cols] for one or two
// vectors v.  A group of DO/4 lanes reads the W row once (one float4 per
// lane) and reduces per head over DH/4 lanes.
template <int DO, int DH>
__global__ __launch_bounds__(256) void reorder_vec_kernel(const float *W, const float *v1,
                                                          const float *v2, int R, int d_in,
                                                          float *out1, float *out2)
{
    constexpr int G = DO / 4, L = DH / 4, H = DO / DH;
    const int gl = threadIdx.x % G;
    const int64_t row = (int64_t)blockIdx.x * (256 / G) + threadIdx.x / G;   // (r, i)
    if (row >= (int64_t)R * d_in) return;
    const int r = (int)(row / d_in), i = (int)(row % d_in), k = gl / L;
    const float4 w = ld4(W + (size_t)row * DO + gl * 4);
    const float a = gsum<L>(dot4(w, ld4(v1 + (size_t)r * DO + gl * 4)));
    if (gl % L == 0) out1[((size_t)r * H + k) * d_in + i] = a;
    if (v2) {
        const float b = gsum<L>(dot4(w, ld4(v2 + (size_t)r * DO + gl * 4)));
        if (gl % L == 0) out2[((size_t)r * H + k) * d_in + i] = b;
    }
}

inline unsigned blocks_for(int64_t n, int per_block) { return (unsigned)((n + per_block - 1) / per_block); }

hipError_t last() { return hipGetLastError(); }

}  // namespace

rgnn_status launch_merge_partials(const rgnn_graph *g, int d, int heads, int softmax,
                                  float *partial, float *out, float *saved, int relu,
                                  hipStream_t s)
{
    if (g->n_split == 0) return RGNN_OK;
    const int32_t *sd = g->dev.split_dst, *sp = g->dev.split_slotptr, *bs = g->dev.big_split;
    const unsigned nb = blocks_for(g->n_split, 256 / (d / 4));
    const unsigned nbig = (unsigned)g->n_big_split;
    {
        LaunchScope ls("merge_partials", s);
#define MERGE(D, H, SM) hipLaunchKernelGGL((merge_kernel<D, H, SM>), dim3(nb), dim3(256), 0, s, \
                                           g->n_split, sd, sp, partial, out, saved, relu)
        if (!softmax) {
            if (d == 32) MERGE(32, 1, false);
            else if (d == 64) MERGE(64, 1, false);
            else if (d == 128) MERGE(128, 1, false);
            else return fail(RGNN_EUNSUPPORTED, "merge: d must be 32, 64 or 128");
        } else if (d == 32 && heads == 1) MERGE(32, 1, true);
        else if (d == 32 && heads == 2) MERGE(32, 2, true);
        else if (d == 64 && heads == 1) MERGE(64, 1, true);
        else if (d == 64 && heads == 2) MERGE(64, 2, true);
        else if (d == 64 && heads == 4) MERGE(64, 4, true);
        else if (d == 128 && heads == 1) MERGE(128, 1, true);
        else if (d == 128 && heads == 2) MERGE(128, 2, true);
        else if (d == 128 && heads == 4) MERGE(128, 4, true);
        else if (d == 128 && heads == 8) MERGE(128, 8, true);
        else return fail(RGNN_EUNSUPPORTED, "merge: unsupported (d, heads)");
#undef MERGE
    }
    hipError_t e = last();
    if (e != hipSuccess) return hip_fail(e, "merge launch");
    if (nbig == 0) return RGNN_OK;
    {
        LaunchScope ls("merge_partials_big", s);
        const unsigned nc = (unsigned)g->n_big_chunks, nf = blocks_for(nbig, 256 / (d / 4));
        const int32_t *clo = g->dev.chunk_lo, *chi = g->dev.chunk_hi, *cp = g->dev.big_chunkptr;
#define MERGEB(D, H, SM)                                                                             \
    do {                                                                                             \
        hipLaunchKernelGGL((merge_chunk_kernel<D, H, SM>), dim3(nc), dim3(256), 0, s, clo, chi,      \
                           partial);                                                                 \
        hipLaunchKernelGGL((merge_chunks_final_kernel<D, H, SM>), dim3(nf), dim3(256), 0, s, nbig,   \
                           bs, sd, cp, clo, partial, out, saved, relu);                              \
    } while (0)
        if (!softmax) {
            if (d == 32) MERGEB(32, 1, false);
            else if (d == 64) MERGEB(64, 1, false);
            else MERGEB(128, 1, false);
        } else if (d == 32 && heads == 1) MERGEB(32, 1, true);
        else if (d == 32 && heads == 2) MERGEB(32, 2, true);
        else if (d == 64 && heads == 1) MERGEB(64, 1, true);
        else if (d == 64 && heads == 2) MERGEB(64, 2, true);
        else if (d == 64 && heads == 4) MERGEB(64, 4, true);
        else if (d == 128 && heads == 1) MERGEB(128, 1, true);
        else if (d == 128 && heads == 2) MERGEB(128, 2, true);
        else if (d == 128 && heads == 4) MERGEB(128, 4, true);
        else MERGEB(128, 8, true);
#undef MERGEB
    }
    e = last();
    return e == hipSuccess ? RGNN_OK : hip_fail(e, "merge_partials_big launch");
}

rgnn_status launch_seg_softmax_scale(const TravArgs &a, hipStream_t s)
{
    const rgnn_graph *g = a.g;
    if (g->U_dst == 0) return RGNN_OK;
    {
        LaunchScope ls("seg_softmax_scale", s);
        hipLaunchKernelGGL(vseg_stats_kernel, dim3(blocks_for(g->U_dst, 256)), dim3(256), 0, s, g->U_dst,
                           g->dev.seg_vsegptr, g->dev.vseg_fpos, a.vstat, a.vscale, a.saved);
    }
    hipError_t e = last();
    if (e != hipSuccess) return hip_fail(e, "seg_softmax_scale launch");
    if (g->n_big_seg == 0) return RGNN_OK;
    {
        LaunchScope ls("seg_softmax_scale_big", s);
        hipLaunchKernelGGL(vseg_stats_big_kernel, dim3((unsigned)g->n_big_seg), dim3(256), 0, s,
                           g->dev.big_seg, g->dev.seg_vsegptr, g->dev.vseg_fpos, a.vstat, a.vscale, a.saved);
    }
    e = last();
    return e == hipSuccess ? RGNN_OK : hip_fail(e, "seg_softmax_scale_big launch");
}

rgnn_status launch_vseg_reduce(const rgnn_graph *g, const float *T, const float *scale, int d,
                               float *out, int accumulate, int relu, hipStream_t s, int64_t ldo, int skip1)
{
    if (ldo == 0) ldo = d;
    if (g->N == 0) return RGNN_OK;
    if (d != 32 && d != 64 && d != 128) return fail(RGNN_EUNSUPPORTED, "reduce: d must be 32, 64 or 128");
    const int64_t nbig = g->n_big_vdst;
    const int32_t *vlist = skip1 ? g->dev.reduce_dst : nullptr;
    const int64_t n = skip1 ? g->n_reduce_dst : g->N;
    const unsigned nb = (unsigned)nbig + blocks_for(n, 256 / (d / 4));
    if (nb == 0) return RGNN_OK;
    {
        LaunchScope ls("vseg_reduce", s);
#define VR(D) hipLaunchKernelGGL((vseg_reduce_kernel<D>), dim3(nb), dim3(256), 0, s, n, nbig, \
                                 g->dev.big_vdst, g->dev.dst_vsegptr, T, scale, out, ldo, accumulate, relu, \
                                 vlist)
        if (d == 32) VR(32);
        else if (d == 64) VR(64);
        else VR(128);
#undef VR
    }
    hipError_t e = last();
    return e == hipSuccess ? RGNN_OK : hip_fail(e, "vseg_reduce launch");
}

rgnn_status launch_softmax_reduce(const rgnn_graph *g, const float *vstat, const float *T, int d,
                                  float *out, float *saved, float *scale, int skip1, hipStream_t s)
{
    if (g->N == 0) return RGNN_OK;
    if (d != 32 && d != 64 && d != 128) return fail(RGNN_EUNSUPPORTED, "softmax reduce: d must be 32, 64 or 128");
    if (g->n_big_vdst && !scale) return fail(RGNN_EINVAL, "softmax reduce needs its scale scratch");
    const int64_t nbig = g->n_big_vdst;
    const int32_t *vlist = skip1 ? g->dev.reduce_dst : nullptr;
    const int64_t n = skip1 ? g->n_reduce_dst : g->N;
    const unsigned nb = (unsigned)nbig + blocks_for(n, 256 / (d / 4));
    if (nb == 0) return RGNN_OK;
    {
        LaunchScope ls("softmax_reduce", s);
#define SR(D) hipLaunchKernelGGL((softmax_reduce_kernel<D>), dim3(nb), dim3(256), 0, s, n, nbig, \
                                 g->dev.big_vdst, g->dev.dst_vsegptr, g->dev.vseg_fpos, vstat, T, out, \
                                 saved, scale, vlist)
        if (d == 32) SR(32);
        else if (d == 64) SR(64);
        else SR(128);
#undef SR
    }
    hipError_t e = last();
    return e == hipSuccess ? RGNN_OK : hip_fail(e, "softmax_reduce launch");
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

rgnn_status launch_mask_cols(const float *in, float *out, int64_t rows, int d, int c0, int c1, hipStream_t s)
{
    const int64_t n = rows * d;
    if (n == 0) return RGNN_OK;
    LaunchScope ls("mask_cols", s);
    hipLaunchKernelGGL(mask_cols_kernel, dim3(blocks_for(n, 256)), dim3(256), 0, s, in, out, n, d, c0, c1);
    hipError_t e = last();
    return e == hipSuccess ? RGNN_OK : hip_fail(e, "mask_cols launch");
}

rgnn_status launch_head_stats(const float *saved, float *out, int64_t N, int H, int k, hipStream_t s)
{
    if (N == 0) return RGNN_OK;
    LaunchScope ls("head_stats", s);
    hipLaunchKernelGGL(head_stats_kernel, dim3(blocks_for(N, 256)), dim3(256), 0, s, saved, out, N, H, k);
    hipError_t e = last();
    return e == hipSuccess ? RGNN_OK : hip_fail(e, "head_stats launch");
}

rgnn_status launch_head_stats_scatter(const float *in, float *saved, int64_t N, int H, int k, hipStream_t s)
{
    if (N == 0) return RGNN_OK;
    LaunchScope ls("head_stats", s);
    hipLaunchKernelGGL(head_stats_scatter_kernel, dim3(blocks_for(N, 256)), dim3(256), 0, s, in, saved, N, H, k);
    hipError_t e = last();
    return e == hipSuccess ? RGNN_OK : hip_fail(e, "head_stats_scatter launch");
}

rgnn_status launch_reorder_vec(const float *W, int R, int d_in, int d_out, int heads,
                               const float *v1, float *out1, const float *v2, float *out2,
                               hipStream_t s)
{
    const int64_t rows = (int64_t)R * d_in;
    if (rows == 0) return RGNN_OK;
    if (d_out != 32 && d_out != 64 && d_out != 128)
        return fail(RGNN_EUNSUPPORTED, "reorder: d_out must be 32, 64 or 128");
    const unsigned nb = blocks_for(rows, 256 / (d_out / 4));
    bool ok = true;
    {
        LaunchScope ls("reorder_vec", s);
#define RV(DO, DH) hipLaunchKernelGGL((reorder_vec_kernel<DO, DH>), dim3(nb), dim3(256), 0, s, W, v1, v2, R, \
                                      d_in, out1, out2)
        const int dh = d_out / heads;
        if (d_out == 32 && dh == 32) RV(32, 32);
        else if (d_out == 32 && dh == 16) RV(32, 16);
        else if (d_out == 64 && dh == 64) RV(64, 64);
        else if (d_out == 64 && dh == 32) RV(64, 32);
        else if (d_out == 64 && dh == 16) RV(64, 16);
        else if (d_out == 128 && dh == 128) RV(128, 128);
        else if (d_out == 128 && dh == 64) RV(128, 64);
        else if (d_out == 128 && dh == 32) RV(128, 32);
        else if (d_out == 128 && dh == 16) RV(128, 16);
        else ok = false;
#undef RV
    }
    if (!ok) return fail(RGNN_EUNSUPPORTED, "reorder: unsupported heads");
    hipError_t e = last();
    return e == hipSuccess ? RGNN_OK : hip_fail(e, "reorder_vec launch");
}

}  // namespace rgnn
