// gemm.hip -- typed / segment GEMM on fp32 MFMA:  Y[S[i]] = X[G[i]] x W[t(i)].
//
// This is the GEMM template of the paper (Section "The GEMM Template and the
// Traversal Template", Y[S] = X[G] x W[T] with gather list G, scatter list S
// and a per-row type T), written for gfx950:
//   * rows are pre-grouped by type; a host-built tile table gives every
//     workgroup one tile of at most kGemmTileRows rows of a single type, so
//     one launch covers all types (no per-type kernel loop);
//   * the tile's weight W[t] (K x Nc fp32) is staged once in LDS, transposed
//     so that each lane fetches four k-values of one column with ds_read_b128;
//   * each wave computes 16-row blocks with v_mfma_f32_16x16x4f32: the A rows
//     are gathered straight from global memory (each lane reads 64 contiguous
//     bytes of its row per load); the rows of the next block (two ahead for
//     64 x 64 weights) are prefetched while the current block runs on the
//     MFMA units;
//   * the epilogue fuses what the paper's fusion rule allows into the GEMM --
//     a per-row scalar (attention normalisation), a per-row dot product with a
//     per-type vector (the reordered attention term), residual add,
//     accumulation, ReLU, a split of the output columns into two tensors --
//     selected at compile time, with its operand loads issued before the
//     next block's prefetch.
//
// Split-bf16 products (the 64-deep shapes): the fp32 MFMA rate, not HBM,
// bounds these GEMMs (16 flop per byte at d = 64, near the fp32 ridge).  Each
// fp32 operand x is split exactly into three bf16 pieces, x = x1 + x2 + x3
// (x1 = RN_bf16(x), x2 = RN_bf16(x - x1), x3 = x - x1 - x2, which needs at
// most 8 significant bits and so is exact in bf16), and the product is
// accumulated in fp32 from the six piece products whose order of magnitude is
// at least 2^-16 of x.w, smallest first:
//   x.w ~ x3 w1 + x1 w3 + x2 w2 + x2 w1 + x1 w2 + x1 w1.
// Each piece product is exact in fp32; the three dropped ones (x2 w3, x3 w2,
// x3 w3) are below 2^-23 |x||w| together, under the rounding of a single fp32
// multiply-add, so the result keeps fp32 accuracy while the matrix cores run
// at the bf16 rate (v_mfma_f32_16x16x32_bf16: 8 k-steps per instruction in
// half the cycles of four fp32 ones, so six of them cost 0.375 of the fp32
// MFMAs).  The weight tile is split once per workgroup into LDS (three bf16
// planes, 6 bytes per entry); each gathered row is split in registers after
// its load.  Operands must be finite with magnitude below 3.38e38 (the split
// of a larger value rounds to infinity).
//
// Load ordering matters on gfx9: the vector-memory counter retires in issue
// order, so waiting for any load also waits for every older one.  All loads
// are unconditional (out-of-tile rows are clamped to a valid row) and issued
// in the order they are consumed: epilogue operands of block i, then the rows
// of block i+PF, so the MFMAs and the epilogue of block i never wait for the
// prefetches of the blocks after it.
//
// MFMA operand layout used (v_mfma_f32_16x16x4f32, one block): lane l supplies
// A[l%16][l/16] and B[l/16][l%16]; the 4 accumulator VGPRs of lane l hold
// D[4*(l/16)+v][l%16], v = 0..3.  The kernel computes the transposed block
// D = W^T X^T (A = W^T from LDS, B = the gathered rows), so lane l holds row
// l%16 and four consecutive columns 4*(l/16) .. +3: one float4 store per
// column block.  The k-slot q = l/16 of step (c, t) is mapped to the actual
// reduction index kk = 16c + 4q + t, identically for A and B.
#include "rgnn_internal.h"
#include "wave_ops.h"

namespace rgnn {

namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

// x = hi + mid + lo exactly (see the split-bf16 note above), eight values at a time
__device__ __forceinline__ void split3(const float (&x)[8], bf16x8 &hi, bf16x8 &mid, bf16x8 &lo)
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

// Shapes whose products can run on split bf16 (a caller's choice, GemmArgs::
// split_bf16): 64- and 128-deep weights of 64 or 128 columns
template <int K, int NC>
constexpr bool split_shape() { return (K == 64 || K == 128) && (NC == 64 || NC == 128); }

// Waves per workgroup: eight for the split 128 x 128 tile, whose three weight
// planes (104 KB of LDS) allow one workgroup per CU, so that a CU still runs
// two waves per SIMD; four otherwise
template <int K, int NC, bool S3>
constexpr int wg_waves() { return S3 && K * NC > 64 * 128 ? 8 : 4; }

enum : int {
    EP_DOT = 1,      // dot_out[row, head] = Y[row, head cols] . dot_vec[type, head cols]
    EP_SCALE = 2,    // Y[row] = row_scale[row] * (X W)[row]
    EP_RESID = 4,    // Y[row] += residual[row]
    EP_ACC = 8,      // Y[row] += old Y[row]
    EP_RELU = 16,    // max(0, .) last
    EP_SPLIT = 32,   // columns >= split go to Y2
    EP_BDIAG = 64    // W[type] is block-diagonal in DH blocks: off-diagonal products skipped
};

struct GemmK {
    const float *X; int64_t ldx;
    const int32_t *gather;
    const float *W0, *W1, *W2;
    int nparts, trans_b;
    const Tile *tiles;
    float *Y; int64_t ldy;
    const int32_t *scatter;
    const float *row_scale;
    const float *dot_vec; float *dot_out; int64_t dot_ld;
    const float *residual; int64_t ld_res;
    float *Y2; int64_t ldy2; int split;
};

template <int K, int NC, int EP, int DH, bool S3>
__global__ __launch_bounds__((64 * wg_waves<K, NC, S3>())) void typed_gemm_kernel(GemmK a)
{
    constexpr int KP = K + 4;           // padded LDS row (conflict-free b128 reads)
    constexpr int NCB = NC / 16;        // 16-column blocks
    constexpr int KC = K / 16;          // 16-wide k chunks (4 MFMA steps each)
    constexpr int NWV = wg_waves<K, NC, S3>(), NT = 64 * NWV;
    constexpr int MB = kGemmTileRows / (16 * NWV);   // row blocks per wave
    constexpr int CBH = NCB / DH;       // column blocks per dot-product head / diagonal block
    constexpr int KCH = KC / DH;        // k chunks per diagonal block
    static_assert(!S3 || split_shape<K, NC>(), "no split path for this shape");
    constexpr int KC3 = K / 32;         // split path: 32-deep k chunks (one bf16 MFMA each)
    constexpr int KB = K + 8;           // split path: padded bf16 row of a weight plane
    __shared__ float Wt[S3 ? 1 : NC * KP];
    // split path: the three bf16 planes of W^T, plane p at [p * NC * KB]
    __shared__ __attribute__((aligned(16))) __bf16 Wb[S3 ? 3 * NC * KB : 8];
    __shared__ float dvs[(EP & EP_DOT) ? NC : 1];

    const Tile tile = a.tiles[blockIdx.x];
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int li = lane & 15, q = lane >> 4;

    // Prologue, ordered so that its three latencies overlap: the weight tile
    // W[type] is fetched into registers, then the row indices, then the first
    // PF row blocks; W is written to LDS (transposed: Wt[n][k] = B[k][n]) only
    // after all of them are in flight.
    constexpr int NW = K * NC / 4 / NT;     // float4 of W per thread
    static_assert(NW * NT * 4 == K * NC, "weight tile must split evenly over the workgroup");
    // split path: (column n, eight consecutive k) runs of W^T per thread
    constexpr int NP8 = S3 ? K * NC / 8 / NT : 1;
    static_assert(!S3 || NP8 * NT * 8 == K * NC, "weight tile must split evenly over the workgroup");
    float4 wv[S3 ? 1 : NW];
    float w8[NP8][8];
    if constexpr (S3) {
        const int NP = NC / a.nparts;
#pragma unroll
        for (int t = 0; t < NP8; ++t) {
            const int idx = tid + NT * t;
            if (a.trans_b) {               // stored [types][NC][K]: rows of W^T
                const int n = idx / (K / 8), k8 = idx % (K / 8);
                const float *src = a.W0 + ((size_t)tile.type * NC + n) * K + 8 * k8;
                const float4 u0 = *reinterpret_cast<const float4 *>(src);
                const float4 u1 = *reinterpret_cast<const float4 *>(src + 4);
                w8[t][0] = u0.x; w8[t][1] = u0.y; w8[t][2] = u0.z; w8[t][3] = u0.w;
                w8[t][4] = u1.x; w8[t][5] = u1.y; w8[t][6] = u1.z; w8[t][7] = u1.w;
            } else {                       // stored [types][K][NP] per part: lanes walk n
                const int n = idx % NC, k8 = idx / NC;
                const int part = n / NP, nn = n % NP;
                const float *Wp = part == 0 ? a.W0 : (part == 1 ? a.W1 : a.W2);
                const float *src = Wp + ((size_t)tile.type * K + 8 * k8) * NP + nn;
#pragma unroll
                for (int j = 0; j < 8; ++j) w8[t][j] = src[(size_t)j * NP];
            }
        }
    } else {
        const int NP = NC / a.nparts;
#pragma unroll
        for (int t = 0; t < NW; ++t) {
            const int idx = tid + NT * t;
            if (a.trans_b) {               // stored [types][NC][K]: rows of W^T
                const int n = idx / (K / 4), k4 = (idx % (K / 4)) * 4;
                wv[t] = *reinterpret_cast<const float4 *>(a.W0 + ((size_t)tile.type * NC + n) * K + k4);
            } else {                       // stored [types][K][NP] per part
                const int k = idx / (NC / 4), n4 = (idx % (NC / 4)) * 4;
                const int part = n4 / NP, nn = n4 % NP;
                const float *Wp = part == 0 ? a.W0 : (part == 1 ? a.W1 : a.W2);
                wv[t] = *reinterpret_cast<const float4 *>(Wp + ((size_t)tile.type * K + k) * NP + nn);
            }
        }
    }
    // Row blocks of this wave: rb = wave + NWV i, i < MB.  Lane (li, q) owns row
    // 16 rb + li of the block and, per column block cb, columns 16 cb + 4q .. +3.
    const int nrb = (tile.rows + 15) >> 4;
    const int32_t *any_idx = reinterpret_cast<const int32_t *>(a.tiles + blockIdx.x);
    int xr[MB], yr[MB];
#pragma unroll
    for (int i = 0; i < MB; ++i) {
        const int r = (wave + NWV * i) * 16 + li;
        const int grow = tile.row0 + (r < tile.rows ? r : 0);
        const int lg = *(a.gather ? a.gather + grow : any_idx);
        const int ls = *(a.scatter ? a.scatter + grow : any_idx);
        xr[i] = a.gather ? lg : grow;
        yr[i] = a.scatter ? ls : grow;
    }
    // Row blocks are prefetched PF blocks ahead (two for 64 x 64 weights, one
    // for wider ones whose accumulators and B fragments already fill the VGPR
    // budget); the loop is fully unrolled, so each block's registers are live
    // only from its load to its MFMAs.
    constexpr int PF = K * NC <= 64 * 64 || (S3 && K == 64) ? 2 : 1;
    float4 ab[MB][KC];
    // SR: the results leave through a wave-private LDS tile, 32 columns at a
    // time, so that each store instruction writes whole 128-byte lines (eight
    // rows of 32 columns) instead of sixteen half lines; residual and
    // accumulated operands are read in that row layout too.  Not for the
    // 128-deep shapes, whose MFMAs are the limit (the tile made them 1-2 %
    // slower; the 64-deep ones 8-16 % faster).
    constexpr bool SR = NCB % 2 == 0 && K != 128;
    constexpr int TP = 36;   // padded tile row (conflict-free b128 writes and reads)
    __shared__ float Ysm[SR ? NWV * 16 * TP : 1];
    // fp32 path: ab[i][c] holds k = 16c + 4q .. +3; split path: ab[i][2c3 + h]
    // holds k = 32c3 + 8q + 4h .. +3 (eight consecutive k per lane and chunk,
    // the bf16 MFMA's operand layout)
    auto load_block = [&](int i) {
        if constexpr (S3) {
            const float *p = a.X + (int64_t)xr[i] * a.ldx + q * 8;
#pragma unroll
            for (int c = 0; c < KC; ++c)
                ab[i][c] = *reinterpret_cast<const float4 *>(p + (c / 2) * 32 + (c % 2) * 4);
        } else {
            const float *p = a.X + (int64_t)xr[i] * a.ldx + q * 4;
#pragma unroll
            for (int c = 0; c < KC; ++c) ab[i][c] = *reinterpret_cast<const float4 *>(p + c * 16);
        }
    };
#pragma unroll
    for (int i = 0; i < PF && i < MB; ++i) load_block(i);
    if constexpr (S3) {
#pragma unroll
        for (int t = 0; t < NP8; ++t) {
            const int idx = tid + NT * t;
            const int n = a.trans_b ? idx / (K / 8) : idx % NC;
            const int k8 = a.trans_b ? idx % (K / 8) : idx / NC;
            bf16x8 hi, mid, lo;
            split3(w8[t], hi, mid, lo);
            __bf16 *dst = &Wb[n * KB + 8 * k8];
            *reinterpret_cast<bf16x8 *>(dst) = hi;
            *reinterpret_cast<bf16x8 *>(dst + NC * KB) = mid;
            *reinterpret_cast<bf16x8 *>(dst + 2 * NC * KB) = lo;
        }
        if (EP & EP_DOT)
            for (int n = tid; n < NC; n += NT) dvs[n] = a.dot_vec[(size_t)tile.type * NC + n];
    } else {
#pragma unroll
        for (int t = 0; t < NW; ++t) {
            const int idx = tid + NT * t;
            if (a.trans_b) {
                const int n = idx / (K / 4), k4 = (idx % (K / 4)) * 4;
                *reinterpret_cast<float4 *>(&Wt[n * KP + k4]) = wv[t];
            } else {
                const int k = idx / (NC / 4), n4 = (idx % (NC / 4)) * 4;
                Wt[(n4 + 0) * KP + k] = wv[t].x;
                Wt[(n4 + 1) * KP + k] = wv[t].y;
                Wt[(n4 + 2) * KP + k] = wv[t].z;
                Wt[(n4 + 3) * KP + k] = wv[t].w;
            }
        }
        if (EP & EP_DOT)
            for (int n = tid; n < NC; n += NT) dvs[n] = a.dot_vec[(size_t)tile.type * NC + n];
    }
    __syncthreads();   // W staged; the first row blocks are already in flight

#pragma unroll
    for (int i = 0; i < MB; ++i) {
        const int rb = wave + NWV * i;
        if (rb >= nrb) break;
        const int64_t y = yr[i];
        const bool valid = rb * 16 + li < tile.rows;
        // (a) epilogue operands of this block
        float sc = 1.f;
        float4 ex[NCB];
        int64_t y2[2];      // SR: the block rows 8j + lane / 8 this lane stores
        bool ok2[2];
        if (EP & EP_SCALE) sc = a.row_scale[y];
        if constexpr (SR) {
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int r2 = 8 * j + (lane >> 3);
                y2[j] = __shfl(yr[i], r2);
                ok2[j] = rb * 16 + r2 < tile.rows;
            }
            if (EP & (EP_RESID | EP_ACC)) {   // ex[2h + j]: columns 32h + 4 (lane % 8) of row y2[j]
#pragma unroll
                for (int hj = 0; hj < NCB; ++hj) {
                    const int j = hj % 2, col = (hj / 2) * 32 + (lane & 7) * 4;
                    float4 x = make_float4(0.f, 0.f, 0.f, 0.f);
                    if (EP & EP_RESID) {
                        const float4 t = *reinterpret_cast<const float4 *>(a.residual + y2[j] * a.ld_res + col);
                        x = make_float4(x.x + t.x, x.y + t.y, x.z + t.z, x.w + t.w);
                    }
                    if (EP & EP_ACC) {
                        const float4 t = *reinterpret_cast<const float4 *>(a.Y + y2[j] * a.ldy + col);
                        x = make_float4(x.x + t.x, x.y + t.y, x.z + t.z, x.w + t.w);
                    }
                    ex[hj] = x;
                }
            }
        } else if (EP & (EP_RESID | EP_ACC)) {
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb) {
                float4 x = make_float4(0.f, 0.f, 0.f, 0.f);
                if (EP & EP_RESID) {
                    const float4 t = *reinterpret_cast<const float4 *>(a.residual + y * a.ld_res + cb * 16 + q * 4);
                    x = make_float4(x.x + t.x, x.y + t.y, x.z + t.z, x.w + t.w);
                }
                if (EP & EP_ACC) {
                    const float4 t = *reinterpret_cast<const float4 *>(a.Y + y * a.ldy + cb * 16 + q * 4);
                    x = make_float4(x.x + t.x, x.y + t.y, x.z + t.z, x.w + t.w);
                }
                ex[cb] = x;
            }
        }
        // (b) rows of block i + PF
        if (i + PF < MB) load_block(i + PF);
        // (c) MFMAs, with W^T as the A operand and the gathered rows as B, so
        // that the accumulator of lane (li, q) holds row li, columns 4q..4q+3
        // of each column block.  The W fragments are re-read from LDS for every
        // row block (keeping the whole weight tile in VGPRs would cap occupancy).
        // Columns are produced in passes of at most four column blocks against
        // the same loaded rows, which bounds the live accumulators and weight
        // fragments (and so the VGPRs) of the wide shapes; each pass ends with
        // its part of the epilogue.
        constexpr int CBP = NCB < 4 ? NCB : 4;
        const float4 (&acur)[KC] = ab[i];
        // with EP_BDIAG only the k chunks of a column block's own diagonal
        // block contribute (a compile-time test after unrolling)
        auto live = [](int c, int cb) { return !(EP & EP_BDIAG) || c / KCH == cb / CBH; };
        // split path: a 32-deep chunk is live when it meets the block's k range
        auto live3 = [](int c3, int cb) {
            constexpr int KD = K / DH;
            return !(EP & EP_BDIAG) || (32 * c3 < (cb / CBH + 1) * KD && (cb / CBH) * KD < 32 * c3 + 32);
        };
        // split path: this block's row pieces, shared by every column pass
        bf16x8 xs[S3 ? KC3 : 1][3];
        if constexpr (S3) {
#pragma unroll
            for (int c3 = 0; c3 < KC3; ++c3) {
                const float4 u0 = acur[2 * c3], u1 = acur[2 * c3 + 1];
                const float x8[8] = {u0.x, u0.y, u0.z, u0.w, u1.x, u1.y, u1.z, u1.w};
                split3(x8, xs[c3][0], xs[c3][1], xs[c3][2]);
            }
        }
        float dpart[DH];
#pragma unroll
        for (int hh = 0; hh < DH; ++hh) dpart[hh] = 0.f;
#pragma unroll
        for (int c0 = 0; c0 < NCB; c0 += CBP) {
            floatx4 acc[CBP];
#pragma unroll
            for (int j = 0; j < CBP; ++j) acc[j] = floatx4{0.f, 0.f, 0.f, 0.f};
            asm volatile("" ::: "memory");
            if constexpr (S3) {
#pragma unroll
                for (int c3 = 0; c3 < KC3; ++c3) {
                    bf16x8 wp[CBP][3];
#pragma unroll
                    for (int j = 0; j < CBP; ++j)
                        if (live3(c3, c0 + j)) {
                            const __bf16 *src = &Wb[((c0 + j) * 16 + li) * KB + 32 * c3 + 8 * q];
#pragma unroll
                            for (int pl = 0; pl < 3; ++pl)
                                wp[j][pl] = *reinterpret_cast<const bf16x8 *>(src + pl * NC * KB);
                        }
                    // the six piece products, smallest first (plane indices of W, X)
                    constexpr int PW[6] = {0, 2, 1, 1, 0, 0}, PX[6] = {2, 0, 1, 0, 1, 0};
#pragma unroll
                    for (int t = 0; t < 6; ++t)
#pragma unroll
                        for (int j = 0; j < CBP; ++j)
                            if (live3(c3, c0 + j))
                                acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wp[j][PW[t]], xs[c3][PX[t]], acc[j],
                                                                                  0, 0, 0);
                }
            }
#pragma unroll
            for (int c = 0; c < (S3 ? 0 : KC); ++c) {
                float4 b[CBP];
#pragma unroll
                for (int j = 0; j < CBP; ++j)
                    if (live(c, c0 + j))
                        b[j] = *reinterpret_cast<const float4 *>(&Wt[((c0 + j) * 16 + li) * KP + c * 16 + q * 4]);
#pragma unroll
                for (int j = 0; j < CBP; ++j)
                    if (live(c, c0 + j)) acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(b[j].x, acur[c].x, acc[j], 0, 0, 0);
#pragma unroll
                for (int j = 0; j < CBP; ++j)
                    if (live(c, c0 + j)) acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(b[j].y, acur[c].y, acc[j], 0, 0, 0);
#pragma unroll
                for (int j = 0; j < CBP; ++j)
                    if (live(c, c0 + j)) acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(b[j].z, acur[c].z, acc[j], 0, 0, 0);
#pragma unroll
                for (int j = 0; j < CBP; ++j)
                    if (live(c, c0 + j)) acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(b[j].w, acur[c].w, acc[j], 0, 0, 0);
            }
            // (d) epilogue of this pass
#pragma unroll
            for (int j = 0; j < CBP; ++j) {
                const int cb = c0 + j;
                float4 v = make_float4(acc[j][0], acc[j][1], acc[j][2], acc[j][3]);
                if (EP & EP_SCALE) v = make_float4(v.x * sc, v.y * sc, v.z * sc, v.w * sc);
                if (EP & EP_DOT) {
                    const float4 d = *reinterpret_cast<const float4 *>(&dvs[cb * 16 + q * 4]);
                    dpart[cb / CBH] += v.x * d.x + v.y * d.y + v.z * d.z + v.w * d.w;
                }
                if constexpr (SR) {
                    float *ts = Ysm + wave * 16 * TP;
                    *reinterpret_cast<float4 *>(&ts[li * TP + (cb & 1) * 16 + q * 4]) = v;
                    if (cb & 1) {   // a 32-column half is complete: out in the row layout
                        __builtin_amdgcn_wave_barrier();
#pragma unroll
                        for (int jr = 0; jr < 2; ++jr) {
                            float4 w = *reinterpret_cast<const float4 *>(&ts[(8 * jr + (lane >> 3)) * TP + (lane & 7) * 4]);
                            if (!ok2[jr]) continue;
                            const int col = (cb - 1) * 16 + (lane & 7) * 4;
                            if (EP & (EP_RESID | EP_ACC)) {
                                const float4 x = ex[(cb / 2) * 2 + jr];
                                w = make_float4(w.x + x.x, w.y + x.y, w.z + x.z, w.w + x.w);
                            }
                            if (EP & EP_RELU) w = make_float4(fmaxf(w.x, 0.f), fmaxf(w.y, 0.f), fmaxf(w.z, 0.f), fmaxf(w.w, 0.f));
                            if ((EP & EP_SPLIT) && col >= a.split)
                                *reinterpret_cast<float4 *>(a.Y2 + y2[jr] * a.ldy2 + (col - a.split)) = w;
                            else
                                *reinterpret_cast<float4 *>(a.Y + y2[jr] * a.ldy + col) = w;
                        }
                        __builtin_amdgcn_wave_barrier();
                    }
                    continue;
                }
                if (!valid) continue;
                if (EP & (EP_RESID | EP_ACC)) v = make_float4(v.x + ex[cb].x, v.y + ex[cb].y, v.z + ex[cb].z, v.w + ex[cb].w);
                if (EP & EP_RELU) v = make_float4(fmaxf(v.x, 0.f), fmaxf(v.y, 0.f), fmaxf(v.z, 0.f), fmaxf(v.w, 0.f));
                const int col = cb * 16 + q * 4;
                if ((EP & EP_SPLIT) && cb * 16 >= a.split)
                    *reinterpret_cast<float4 *>(a.Y2 + y * a.ldy2 + (col - a.split)) = v;
                else
                    *reinterpret_cast<float4 *>(a.Y + y * a.ldy + col) = v;
            }
        }
        if (EP & EP_DOT) {
#pragma unroll
            for (int hh = 0; hh < DH; ++hh) {
                float part = dpart[hh];
                part += __shfl_xor(part, 16);
                part += __shfl_xor(part, 32);
                if (valid && q == 0) a.dot_out[y * a.dot_ld + hh] = part;
            }
        }
    }
}

template <int K, int NC, int EP, int DH = 1, bool S3 = false>
void launch_k(const GemmK &k, int64_t ntiles, hipStream_t s)
{
    hipLaunchKernelGGL((typed_gemm_kernel<K, NC, EP, DH, S3>), dim3((unsigned)ntiles),
                       dim3(64 * wg_waves<K, NC, S3>()), 0, s, k);
}

// Epilogues instantiated per shape: square shapes (32, 64, 128) serve every layer; the
// rectangular ones serve RGCN with d_in != d_out and the segment-MM entry
// point; 64 x 192 is the fused K|V|Q projection of HGT.
template <int K, int NC, bool S3 = false>
bool dispatch_square(int ep, int heads, const GemmK &k, int64_t n, hipStream_t s)
{
    switch (ep) {
    case 0: launch_k<K, NC, 0, 1, S3>(k, n, s); return true;
    case EP_DOT:
        switch (heads) {
        case 1: launch_k<K, NC, EP_DOT, 1, S3>(k, n, s); return true;
        case 2: launch_k<K, NC, EP_DOT, 2, S3>(k, n, s); return true;
        case 4:
            if constexpr (NC >= 64) { launch_k<K, NC, EP_DOT, 4, S3>(k, n, s); return true; }
            return false;
        case 8:
            if constexpr (NC >= 128) { launch_k<K, NC, EP_DOT, 8, S3>(k, n, s); return true; }
            return false;
        default: return false;
        }
    case EP_SCALE: launch_k<K, NC, EP_SCALE, 1, S3>(k, n, s); return true;
    case EP_ACC: launch_k<K, NC, EP_ACC, 1, S3>(k, n, s); return true;
    case EP_ACC | EP_RELU: launch_k<K, NC, EP_ACC | EP_RELU, 1, S3>(k, n, s); return true;
    case EP_RESID: launch_k<K, NC, EP_RESID, 1, S3>(k, n, s); return true;
    case EP_BDIAG:
        switch (heads) {
        case 1: launch_k<K, NC, 0, 1, S3>(k, n, s); return true;
        case 2: launch_k<K, NC, EP_BDIAG, 2, S3>(k, n, s); return true;
        case 4:
            if constexpr (NC >= 64) { launch_k<K, NC, EP_BDIAG, 4, S3>(k, n, s); return true; }
            return false;
        case 8:
            if constexpr (NC >= 128) { launch_k<K, NC, EP_BDIAG, 8, S3>(k, n, s); return true; }
            return false;
        default: return false;
        }
    default: return false;
    }
}

template <int K, int NC, bool S3 = false>
bool dispatch_rect(int ep, const GemmK &k, int64_t n, hipStream_t s)
{
    switch (ep) {
    case 0: launch_k<K, NC, 0, 1, S3>(k, n, s); return true;
    case EP_ACC: launch_k<K, NC, EP_ACC, 1, S3>(k, n, s); return true;
    case EP_ACC | EP_RELU: launch_k<K, NC, EP_ACC | EP_RELU, 1, S3>(k, n, s); return true;
    default: return false;
    }
}

}  // namespace

rgnn_status launch_typed_gemm(const GemmArgs &a, hipStream_t s)
{
    if (a.ntiles == 0) return RGNN_OK;
    GemmK k{};
    k.X = a.X; k.ldx = a.ldx; k.gather = a.gather;
    k.W0 = a.W[0]; k.W1 = a.W[1]; k.W2 = a.W[2];
    k.nparts = a.nparts; k.trans_b = a.trans_b;
    k.tiles = a.tiles; k.Y = a.Y; k.ldy = a.ldy; k.scatter = a.scatter;
    k.row_scale = a.ep.row_scale;
    k.dot_vec = a.ep.dot_vec; k.dot_out = a.ep.dot_out;
    k.dot_ld = a.ep.dot_ld ? a.ep.dot_ld : a.ep.dot_heads;
    k.residual = a.ep.residual; k.ld_res = a.ep.ld_res;
    k.Y2 = a.ep.Y2; k.ldy2 = a.ep.ldy2; k.split = a.ep.split;
    if (a.trans_b && a.nparts != 1) return fail(RGNN_EINVAL, "transposed B takes one part");
    if (a.Nc % a.nparts) return fail(RGNN_EINVAL, "column parts must split Nc evenly");
    if (a.ep.dot_out && ((a.Nc / 16) % a.ep.dot_heads))
        return fail(RGNN_EUNSUPPORTED, "dot-product heads must own whole 16-column blocks");
    const int ep = (a.ep.dot_out ? EP_DOT : 0) | (a.ep.row_scale ? EP_SCALE : 0) |
                   (a.ep.residual ? EP_RESID : 0) | (a.ep.accumulate ? EP_ACC : 0) |
                   (a.ep.relu ? EP_RELU : 0) | (a.ep.Y2 ? EP_SPLIT : 0) |
                   (a.ep.diag_blocks > 1 ? EP_BDIAG : 0);
    if ((ep & EP_BDIAG) && ep != EP_BDIAG)
        return fail(RGNN_EUNSUPPORTED, "block-diagonal weights take no epilogue");
    const int heads = (ep & EP_BDIAG) ? a.ep.diag_blocks : a.ep.dot_heads;
    bool ok = false;
    {
        LaunchScope ls("typed_gemm", s);
        const bool sp = a.split_bf16;
        if (a.K == 32 && a.Nc == 32) ok = dispatch_square<32, 32>(ep, heads, k, a.ntiles, s);
        else if (a.K == 64 && a.Nc == 64)
            ok = sp ? dispatch_square<64, 64, true>(ep, heads, k, a.ntiles, s)
                    : dispatch_square<64, 64>(ep, heads, k, a.ntiles, s);
        else if (a.K == 128 && a.Nc == 128)
            ok = sp ? dispatch_square<128, 128, true>(ep, heads, k, a.ntiles, s)
                    : dispatch_square<128, 128>(ep, heads, k, a.ntiles, s);
        else if (a.K == 64 && a.Nc == 128)
            ok = sp ? dispatch_rect<64, 128, true>(ep, k, a.ntiles, s) : dispatch_rect<64, 128>(ep, k, a.ntiles, s);
        else if (a.K == 128 && a.Nc == 64)
            ok = sp ? dispatch_rect<128, 64, true>(ep, k, a.ntiles, s) : dispatch_rect<128, 64>(ep, k, a.ntiles, s);
        else if (a.K == 64 && a.Nc == 192 && ep == EP_SPLIT) {
            launch_k<64, 192, EP_SPLIT>(k, a.ntiles, s);
            ok = true;
        } else if (a.K == 192 && a.Nc == 64 && (ep == 0 || ep == EP_RESID)) {   // three weights stacked in K
            if (ep) launch_k<192, 64, EP_RESID>(k, a.ntiles, s);
            else launch_k<192, 64, 0>(k, a.ntiles, s);
            ok = true;
        } else if (a.K == 96 && a.Nc == 32 && (ep == 0 || ep == EP_RESID)) {
            if (ep) launch_k<96, 32, EP_RESID>(k, a.ntiles, s);
            else launch_k<96, 32, 0>(k, a.ntiles, s);
            ok = true;
        }
    }
    if (!ok) return fail(RGNN_EUNSUPPORTED, "typed GEMM: unsupported shape / epilogue combination");
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? RGNN_OK : hip_fail(e, "typed_gemm launch");
}

}  // namespace rgnn
