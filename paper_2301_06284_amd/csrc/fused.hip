// fused.hip -- fused gather -> segment sum -> typed transform for the
// aggregate-first plan (Section "Graph-Semantic Optimizations": linear operator
// reordering moves W_r after the per-(dst, rel) aggregation; Section "The GEMM
// Template and the Traversal Template" gives the two halves fused here).
//
// For every virtual segment (one (dst, rel) pair, at most kChunkEdges in-edges)
// the kernel forms the segment's weighted row sum S of the gathered source
// rows h_u and immediately multiplies it by W_r on the matrix cores, writing
// T = S W_r.  S never goes to memory.
//
// Work decomposition.  Segments are grouped by relation and, inside a
// relation, ordered by edge count (largest first); a host-built tile table
// gives each workgroup up to kFusedTileRows consecutive segments of one
// relation, so W_r is staged once in LDS for the whole tile.  A wave takes 16
// segments at a time -- one 16-row MFMA block.  The rows are gathered with
// eight adjacent lanes per source row (whole 128-byte lines per load
// instruction), summed, and moved into the B-operand layout of
// v_mfma_f32_16x16x4f32 by lane permutes; the products are permuted back to
// the row layout for the stores.  Because the 16 segments of a block have
// nearly equal edge counts, the edge loop wastes few lane-steps, and the first
// gathers of a wave's next block are issued before the current block's
// transform so that loads stay in flight.
//
// RGAT: per edge the source term h_u . (W_r w_src[r]) (reordered) is summed
// over the eight lanes of the row; with the segment's destination term it
// gives the logit, and an online softmax keeps the running maximum m, the sum
// s and the exp-weighted row sum.  T is written per segment (row vs), (m, s)
// per segment in the fused order (sequential stores; the reductions find them
// through vseg_fpos); the per-destination normalisation exp(m - M_v) / Z_v is
// applied when the segments of a destination are summed.  RGCN: plain sums
// scaled by 1 / c_{v,r}.  No atomics: results are bitwise reproducible.
#include "rgnn_internal.h"
#include "wave_ops.h"

namespace rgnn {

namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float4 ld4(const float *p) { return *reinterpret_cast<const float4 *>(p); }
__device__ __forceinline__ void st4(float *p, float4 v) { *reinterpret_cast<float4 *>(p) = v; }
__device__ __forceinline__ float dot4(float4 a, float4 b) { return a.x * b.x + a.y * b.y + a.z * b.z + a.w * b.w; }
__device__ __forceinline__ float leaky(float y, float slope) { return y > 0.f ? y : slope * y; }

enum : int { kModeMean = 0, kModeSoftmax = 1, kModeSum = 2 };

struct FK {
    const FusedRow *rows;
    const Tile *tiles;           // pad = the tile's first position in src
    int64_t ntiles, nedges;
    const int32_t *src;          // source node of every in-edge, in fused order
    const float *h, *W, *wsp, *vatt;
    float slope;
    float *T, *vstat;
    float *out, *saved;          // rows of destinations with one virtual segment (softmax: and
                                 // their statistics)
    int relu;                    // mean: ReLU on those rows
    const int32_t *pos;          // sums only: output row of each virtual segment
    float *S;
};

// DI: input features, DO: output features, NWAVE: waves per workgroup,
// KU: edges per gathered batch (two batches in flight).
//
// Gather layout: lane l serves rows l/8 and l/8 + 8 of the 16-row block, and
// within each the features 32c + 4(l%8) .. +3 (c < DI/32), so one dwordx4
// load instruction covers whole 128-byte lines of eight rows.  The finished
// row sums are moved into the MFMA operand layout by lane permutes.
template <int DI, int DO, int MODE, int NWAVE, int KU, int WPE>
__global__ __launch_bounds__(64 * NWAVE) __attribute__((amdgpu_waves_per_eu(WPE))) void af_fused_kernel(FK k)
{
    constexpr int NT = 64 * NWAVE;
    constexpr int KP = DI + 4;       // padded LDS row (conflict-free b128 reads)
    constexpr int KC = DI / 16;      // MFMA k chunks
    constexpr int CH = DI / 32;      // float4 chunks per lane and gathered row
    constexpr int NCB = DO / 16;     // output column blocks
    constexpr int CBP = 2;           // output column blocks per MFMA pass
    constexpr int NW = DI * DO / 4 / NT;
    constexpr int NR = (kFusedTileRows + NT - 1) / NT;   // segment entries per thread
    constexpr int NS = (kFusedTileEdges + NT - 1) / NT;  // source indices per thread
    static_assert(NW * NT * 4 == DI * DO, "weight tile must split evenly over the workgroup");
    __shared__ float Wt[MODE == kModeSum ? 1 : DO * KP];
    __shared__ float wsl[MODE == kModeSoftmax ? DI : 1];
    __shared__ FusedRow srow[kFusedTileRows];
    __shared__ int32_t ssrc[kFusedTileEdges];

    const Tile tile = k.tiles[blockIdx.x];
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int li = lane & 15, q = lane >> 4;       // MFMA layout
    const int gr = lane >> 3, gp = lane & 7;       // gather layout: rows gr, gr + 8
    const int r = tile.type;
    const int64_t te0 = tile.pad;
    const int tne = (int)((blockIdx.x + 1 < k.ntiles ? (int64_t)k.tiles[blockIdx.x + 1].pad : k.nedges) - te0);

    // Stage: W_r, the tile's segment table and its source indices are all
    // fetched into registers first (independent, coalesced loads), then
    // written to LDS behind one barrier.  After it, the row gathers are the
    // only loads that depend on another load.
    float4 wv[NW];
#pragma unroll
    for (int t = 0; t < NW; ++t) {
        if (MODE == kModeSum) break;
        const int idx = tid + NT * t;
        const int kk = idx / (DO / 4), n4 = (idx % (DO / 4)) * 4;
        wv[t] = ld4(k.W + ((size_t)r * DI + kk) * DO + n4);
    }
    FusedRow rv[NR];
#pragma unroll
    for (int t = 0; t < NR; ++t) {
        const int i = tid + NT * t;
        rv[t] = k.rows[tile.row0 + (i < tile.rows ? i : 0)];
    }
    int sv[NS];
#pragma unroll
    for (int t = 0; t < NS; ++t) {
        const int i = tid + NT * t;
        sv[t] = k.src[te0 + (i < tne ? i : 0)];
    }
    float wsv = 0.f;
    if (MODE == kModeSoftmax && tid < DI) wsv = k.wsp[(size_t)r * DI + tid];
#pragma unroll
    for (int t = 0; t < NW; ++t) {
        if (MODE == kModeSum) break;
        const int idx = tid + NT * t;
        const int kk = idx / (DO / 4), n4 = (idx % (DO / 4)) * 4;
        Wt[(n4 + 0) * KP + kk] = wv[t].x;
        Wt[(n4 + 1) * KP + kk] = wv[t].y;
        Wt[(n4 + 2) * KP + kk] = wv[t].z;
        Wt[(n4 + 3) * KP + kk] = wv[t].w;
    }
#pragma unroll
    for (int t = 0; t < NR; ++t) {
        const int i = tid + NT * t;
        if (i < tile.rows) srow[i] = rv[t];
    }
#pragma unroll
    for (int t = 0; t < NS; ++t) {
        const int i = tid + NT * t;
        if (i < tne) ssrc[i] = sv[t];
    }
    if (MODE == kModeSoftmax && tid < DI) wsl[tid] = wsv;
    __syncthreads();

    const int nrb = (tile.rows + 15) >> 4;
    // One 16-row block's gathered rows, as this lane sees them: rows past the
    // tile's end repeat the block's first row (never longer than the block's
    // longest) and store nothing.
    struct Blk {
        FusedRow fr[2];
        bool valid[2];
        int lso[2];      // first source index of the row in ssrc
        int fp[2];       // position of the row in the fused order
        float va[2];     // destination attention term
        int sid[2];      // output row: vs (a T row), or ~v when the row finishes destination v
        int nmax;        // edge count of the block's longest segment
    };
    auto setup = [&](int rb, Blk &b) {
#pragma unroll
        for (int h2 = 0; h2 < 2; ++h2) {
            const int row = rb * 16 + gr + 8 * h2;
            b.valid[h2] = row < tile.rows;
            b.fp[h2] = (int)tile.row0 + row;
            b.fr[h2] = srow[b.valid[h2] ? row : rb * 16];
            b.lso[h2] = (int)(b.fr[h2].e0 - te0);
            b.va[h2] = MODE == kModeSoftmax ? k.vatt[b.fr[h2].vs] : 0.f;
            b.sid[h2] = MODE != kModeSum && k.out && b.fr[h2].cnt < 0 ? b.fr[h2].cnt : b.fr[h2].vs;
        }
        // rows are sorted by edge count inside a relation (largest first), so
        // the block's first row is its longest
        b.nmax = __builtin_amdgcn_readfirstlane(srow[rb * 16].ne);
    };
    // batches of KU edges of both rows (indices from LDS); a row already
    // finished issues no gathers (most segments are one or two edges long)
    float4 A[KU][2][CH], B[KU][2][CH];
    auto load = [&](const Blk &b, float4 (&X)[KU][2][CH], int t) {
#pragma unroll
        for (int u = 0; u < KU; ++u)
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2) {
                if (t + u < b.fr[h2].ne) {
                    const int i = ssrc[b.lso[h2] + t + u];
#pragma unroll
                    for (int c = 0; c < CH; ++c) X[u][h2][c] = ld4(k.h + (size_t)i * DI + c * 32 + gp * 4);
                } else {
#pragma unroll
                    for (int c = 0; c < CH; ++c) X[u][h2][c] = make_float4(0.f, 0.f, 0.f, 0.f);
                }
            }
    };
    // The first batch of a wave's next block is issued before the current
    // block's transform and stores, so a wave always has gathers in flight
    // (blocks of one- and two-edge segments are a single batch).
    Blk cur;
    if (wave < nrb) {
        setup(wave, cur);
        load(cur, A, 0);
    }
    for (int rb = wave; rb < nrb; rb += NWAVE) {
        const FusedRow (&fr)[2] = cur.fr;
        const bool (&valid)[2] = cur.valid;
        const int nmax = cur.nmax;
        float m[2] = {-INFINITY, -INFINITY}, s[2] = {0.f, 0.f};
        float4 acc[2][CH];
#pragma unroll
        for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
            for (int c = 0; c < CH; ++c) acc[h2][c] = make_float4(0.f, 0.f, 0.f, 0.f);

        auto consume = [&](const float4 (&X)[KU][2][CH], int t) {
#pragma unroll
            for (int u = 0; u < KU; ++u) {
                if (t + u >= nmax) break;   // past every row of the block (uniform)
#pragma unroll
                for (int h2 = 0; h2 < 2; ++h2) {
                    const float4 *x = X[u][h2];
                    if (MODE == kModeSoftmax) {
                        float p = 0.f;
#pragma unroll
                        for (int c = 0; c < CH; ++c)
                            p += dot4(x[c], *reinterpret_cast<const float4 *>(&wsl[c * 32 + gp * 4]));
                        p = gsum<8>(p);   // the row's eight lanes: identical sums
                        if (t + u < fr[h2].ne) {
                            // online update with one exponential: the smaller of
                            // the old maximum and z is scaled by exp(-|z - m|)
                            const float z = leaky(p + cur.va[h2], k.slope);
                            const bool up = z > m[h2];
                            const float ex = __expf(up ? m[h2] - z : z - m[h2]);
                            const float c1 = up ? ex : 1.f, c2 = up ? 1.f : ex;
                            const float mn = up ? z : m[h2];
                            s[h2] = s[h2] * c1 + c2;
#pragma unroll
                            for (int c = 0; c < CH; ++c) {
                                float4 &a = acc[h2][c];
                                a = make_float4(a.x * c1 + x[c].x * c2, a.y * c1 + x[c].y * c2,
                                                a.z * c1 + x[c].z * c2, a.w * c1 + x[c].w * c2);
                            }
                            m[h2] = mn;
                        }
                    } else if (t + u < fr[h2].ne) {
#pragma unroll
                        for (int c = 0; c < CH; ++c) {
                            float4 &a = acc[h2][c];
                            a = make_float4(a.x + x[c].x, a.y + x[c].y, a.z + x[c].z, a.w + x[c].w);
                        }
                    }
                }
            }
        };
        // ping-pong: batch 0 is already in A; batches past the block's
        // longest segment are neither loaded nor consumed (wave-uniform tests)
        __builtin_amdgcn_sched_barrier(0);
        for (int t = 0; t < nmax; t += 2 * KU) {
            const bool more_b = t + KU < nmax;
            if (more_b) load(cur, B, t + KU);
            __builtin_amdgcn_sched_barrier(0);
            consume(A, t);
            if (!more_b) break;
            if (t + 2 * KU < nmax) load(cur, A, t + 2 * KU);
            __builtin_amdgcn_sched_barrier(0);
            consume(B, t + KU);
        }
        // the next block's first batch goes out now
        Blk nxt = cur;
        if (rb + NWAVE < nrb) {
            setup(rb + NWAVE, nxt);
            load(nxt, A, 0);
        }
        __builtin_amdgcn_sched_barrier(0);

        if (MODE == kModeSum) {   // the segment means themselves, in the row layout
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2) {
                if (!valid[h2]) continue;
                const float sc = 1.f / (float)(fr[h2].cnt < 0 ? fr[h2].ne : fr[h2].cnt);
                float *o = k.S + (size_t)k.pos[fr[h2].vs] * DI + gp * 4;
#pragma unroll
                for (int c = 0; c < CH; ++c) {
                    const float4 a = acc[h2][c];
                    st4(o + c * 32, make_float4(a.x * sc, a.y * sc, a.z * sc, a.w * sc));
                }
            }
            cur = nxt;
            continue;
        }
        // A destination with one virtual segment is finished here: its output
        // row is the segment's own transformed row (softmax: its denominator is
        // the segment's own sum, so the row sum is divided by it before the
        // transform, and saved gets (m, s)); every other segment leaves T (and
        // (m, s)) for the reduction.
        bool fin[2];
        float *rowp[2];
#pragma unroll
        for (int h2 = 0; h2 < 2; ++h2) {
            fin[h2] = MODE != kModeSum && cur.sid[h2] < 0;
            rowp[h2] = (fin[h2] ? k.out + (size_t)~cur.sid[h2] * DO : k.T + (size_t)cur.sid[h2] * DO) + gp * 4;
            if (MODE != kModeSum) {
                const float sc = MODE == kModeMean ? 1.f / (float)(fr[h2].cnt < 0 ? fr[h2].ne : fr[h2].cnt)
                                                   : (fin[h2] ? 1.f / s[h2] : 1.f);
#pragma unroll
                for (int c = 0; c < CH; ++c) {
                    float4 &a = acc[h2][c];
                    a = make_float4(a.x * sc, a.y * sc, a.z * sc, a.w * sc);
                }
            }
            if (MODE == kModeSoftmax && valid[h2] && gp == 0) {
                if (!fin[h2])
                    *reinterpret_cast<float2 *>(k.vstat + (size_t)cur.fp[h2] * 2) = make_float2(m[h2], s[h2]);
                else if (k.saved)
                    *reinterpret_cast<float2 *>(k.saved + (size_t)~cur.sid[h2] * 2) = make_float2(m[h2], s[h2]);
            }
        }
        // row sums -> MFMA operand layout by lane permutes: lane (li, q) takes
        // features 16c + 4q .. +3 of row li, held by lane 8 (li % 8) + 4 (c % 2) + q
        // in its chunk c / 2 of row set li / 8
        const bool hi = li >= 8;
        float4 sb[KC];
#pragma unroll
        for (int c = 0; c < KC; ++c) {
            const int sl = 8 * (li & 7) + 4 * (c & 1) + q;
            const float4 a0 = acc[0][c >> 1], a1 = acc[1][c >> 1];
            const float x0 = __shfl(a0.x, sl), x1 = __shfl(a1.x, sl);
            const float y0 = __shfl(a0.y, sl), y1 = __shfl(a1.y, sl);
            const float z0 = __shfl(a0.z, sl), z1 = __shfl(a1.z, sl);
            const float w0 = __shfl(a0.w, sl), w1 = __shfl(a1.w, sl);
            sb[c] = make_float4(hi ? x1 : x0, hi ? y1 : y0, hi ? z1 : z0, hi ? w1 : w0);
        }

        // T = S W_r on the matrix cores: A = W_r^T fragments from LDS, B = the
        // row sums (k-slot q of step (c, j) is feature 16c + 4q + j for both)
#pragma unroll
        for (int c0 = 0; c0 < NCB; c0 += CBP) {
            floatx4 o[CBP];
#pragma unroll
            for (int j = 0; j < CBP; ++j) o[j] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int c = 0; c < KC; ++c) {
                float4 b[CBP];
#pragma unroll
                for (int j = 0; j < CBP; ++j)
                    b[j] = *reinterpret_cast<const float4 *>(&Wt[((c0 + j) * 16 + li) * KP + c * 16 + q * 4]);
#pragma unroll
                for (int j = 0; j < CBP; ++j) o[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(b[j].x, sb[c].x, o[j], 0, 0, 0);
#pragma unroll
                for (int j = 0; j < CBP; ++j) o[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(b[j].y, sb[c].y, o[j], 0, 0, 0);
#pragma unroll
                for (int j = 0; j < CBP; ++j) o[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(b[j].z, sb[c].z, o[j], 0, 0, 0);
#pragma unroll
                for (int j = 0; j < CBP; ++j) o[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(b[j].w, sb[c].w, o[j], 0, 0, 0);
            }
            // back to the row layout for the stores (whole 128-byte lines per
            // instruction): lane (gr, gp) takes features 32c' + 4gp .. +3 of
            // rows gr and gr + 8, held by lane row + 16 (gp % 4) in column
            // block 2c' + gp / 4
#pragma unroll
            for (int cc = 0; cc < CBP / 2; ++cc) {
#pragma unroll
                for (int h2 = 0; h2 < 2; ++h2) {
                    const int sl = gr + 8 * h2 + 16 * (gp & 3);
                    const floatx4 lo = o[2 * cc], hi4 = o[2 * cc + 1];
                    float v[4];
#pragma unroll
                    for (int t = 0; t < 4; ++t) {
                        const float a = __shfl(lo[t], sl), b = __shfl(hi4[t], sl);
                        v[t] = gp >= 4 ? b : a;
                    }
                    if (MODE == kModeMean && fin[h2] && k.relu)
#pragma unroll
                        for (int t = 0; t < 4; ++t) v[t] = fmaxf(v[t], 0.f);
                    if (valid[h2])
                        st4(rowp[h2] + (c0 / 2 + cc) * 32,
                            make_float4(v[0], v[1], v[2], v[3]));
                }
            }
        }
        cur = nxt;
    }
}

template <int DI, int DO, int MODE>
void launch_shape(const FK &k, int64_t ntiles, hipStream_t s)
{
    // d = 128: the 64 KB weight tile is shared by eight waves; one batch of
    // rows per wave in flight keeps the gathered rows within the VGPR budget
    constexpr int NWAVE = (DI == 128 || DO == 128) ? 8 : 4;
    constexpr int KU = DI == 128 ? 1 : 2;
    // waves per SIMD the LDS allows; the 128 x 64 mean shape gets the register
    // budget of three
    constexpr int WPE = (DI == 128 && DO == 64) ? 3 : 4;
    hipLaunchKernelGGL((af_fused_kernel<DI, DO, MODE, NWAVE, KU, WPE>), dim3((unsigned)ntiles),
                       dim3(64 * NWAVE), 0, s, k);
}

template <int MODE>
bool dispatch(int di, int dout, const FK &k, int64_t n, hipStream_t s)
{
    if constexpr (MODE == kModeSum) {   // no transform: the output width is d_in
        if (di == 32) launch_shape<32, 32, MODE>(k, n, s);
        else if (di == 64) launch_shape<64, 64, MODE>(k, n, s);
        else if (di == 128) launch_shape<128, 128, MODE>(k, n, s);
        else return false;
        return true;
    }
    if (di == 32 && dout == 32) launch_shape<32, 32, MODE>(k, n, s);
    else if (di == 64 && dout == 64) launch_shape<64, 64, MODE>(k, n, s);
    else if (di == 128 && dout == 128) launch_shape<128, 128, MODE>(k, n, s);
    else if constexpr (MODE == kModeMean) {   // RGCN only: RGAT needs d_in == d_out
        if (di == 64 && dout == 128) launch_shape<64, 128, MODE>(k, n, s);
        else if (di == 128 && dout == 64) launch_shape<128, 64, MODE>(k, n, s);
        else return false;
    } else {
        return false;
    }
    return true;
}

}  // namespace

rgnn_status launch_af_fused(const FusedArgs &a, hipStream_t s)
{
    const rgnn_graph *g = a.g;
    if (g->n_tiles_fused == 0) return RGNN_OK;
    FK k{};
    k.rows = g->dev.fused_rows; k.tiles = g->dev.tiles_fused;
    k.ntiles = g->n_tiles_fused; k.nedges = g->E; k.src = g->dev.fused_src;
    k.h = a.h; k.W = a.W; k.wsp = a.wsp; k.vatt = a.vatt; k.slope = a.slope;
    k.T = a.T; k.vstat = a.vstat; k.S = a.S; k.pos = g->dev.vseg_pos;
    k.out = a.out; k.saved = a.saved; k.relu = a.relu;
    if (a.softmax && (!a.wsp || !a.vatt || !a.vstat))
        return fail(RGNN_EINVAL, "fused softmax aggregation needs wsp, vatt and vstat");
    if (a.S && a.softmax) return fail(RGNN_EINVAL, "segment means are for the mean aggregation");
    bool ok;
    {
        LaunchScope ls(a.softmax ? "rgat_af_fused" : (a.S ? "segment_means" : "rgcn_af_fused"), s);
        ok = a.softmax ? dispatch<kModeSoftmax>(a.d_in, a.d_out, k, g->n_tiles_fused, s)
             : a.S     ? dispatch<kModeSum>(a.d_in, a.d_out, k, g->n_tiles_fused, s)
                       : dispatch<kModeMean>(a.d_in, a.d_out, k, g->n_tiles_fused, s);
    }
    if (!ok) return fail(RGNN_EUNSUPPORTED, "fused aggregation: unsupported (d_in, d_out)");
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? RGNN_OK : hip_fail(e, "af_fused launch");
}

}  // namespace rgnn
