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
//     bytes of its row per load); the next block's rows are prefetched while
//     the current block runs on the MFMA units;
//   * the epilogue fuses what the paper's fusion rule allows into the GEMM --
//     a per-row scalar (attention normalisation), a per-row dot product with a
//     per-type vector (the reordered attention term), residual add,
//     accumulation, ReLU, a split of the output columns into two tensors --
//     selected at compile time, with its operand loads issued before the
//     next block's prefetch.
//
// Load ordering matters on gfx9: the vector-memory counter retires in issue
// order, so waiting for any load also waits for every older one.  All loads
// are unconditional (out-of-tile rows are clamped to a valid row) and issued
// in the order they are consumed: epilogue operands of block i, then the rows
// of block i+1, so the MFMAs and the epilogue of block i never wait for the
// prefetch of block i+1.
//
// MFMA operand layout used (v_mfma_f32_16x16x4f32, one block): lane l supplies
// A[l%16][l/16] and B[l/16][l%16]; the 4 accumulator VGPRs of lane l hold
// D[4*(l/16)+v][l%16], v = 0..3.  The k-slot q = l/16 of step (c, t) is mapped
// to the actual reduction index kk = 16c + 4q + t, identically for A and B.
#include "rgnn_internal.h"
#include "wave_ops.h"

namespace rgnn {

namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));

enum : int {
    EP_DOT = 1,      // dot_out[row, head] = Y[row, head cols] . dot_vec[type, head cols]
    EP_SCALE = 2,    // Y[row] = row_scale[row] * (X W)[row]
    EP_RESID = 4,    // Y[row] += residual[row]
    EP_ACC = 8,      // Y[row] += old Y[row]
    EP_RELU = 16,    // max(0, .) last
    EP_SPLIT = 32    // columns >= split go to Y2
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
    const float *dot_vec; float *dot_out; int dot_heads;
    const float *residual; int64_t ld_res;
    float *Y2; int64_t ldy2; int split;
};

template <int K, int NC, int EP>
__global__ __launch_bounds__(256) void typed_gemm_kernel(GemmK a)
{
    constexpr int KP = K + 4;           // padded LDS row (conflict-free b128 reads)
    constexpr int NCB = NC / 16;        // 16-column blocks
    constexpr int KC = K / 16;          // 16-wide k chunks (4 MFMA steps each)
    constexpr int MB = kGemmTileRows / 64;
    __shared__ float Wt[NC * KP];

    const Tile tile = a.tiles[blockIdx.x];
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int li = lane & 15, q = lane >> 4;

    // ---- stage W[type] transposed into LDS: Wt[n][k] = B[k][n] (float4 reads) ----
    {
        const int NP = NC / a.nparts;
        for (int idx = tid; idx < K * NC / 4; idx += 256) {
            if (a.trans_b) {               // stored [types][NC][K]: copy rows
                const int n = idx / (K / 4), k4 = (idx % (K / 4)) * 4;
                const float4 w = *reinterpret_cast<const float4 *>(a.W0 + ((size_t)tile.type * NC + n) * K + k4);
                *reinterpret_cast<float4 *>(&Wt[n * KP + k4]) = w;
            } else {                       // stored [types][K][NP] per part
                const int k = idx / (NC / 4), n4 = (idx % (NC / 4)) * 4;
                const int part = n4 / NP, nn = n4 % NP;
                const float *Wp = part == 0 ? a.W0 : (part == 1 ? a.W1 : a.W2);
                const float4 w = *reinterpret_cast<const float4 *>(Wp + ((size_t)tile.type * K + k) * NP + nn);
                Wt[(n4 + 0) * KP + k] = w.x;
                Wt[(n4 + 1) * KP + k] = w.y;
                Wt[(n4 + 2) * KP + k] = w.z;
                Wt[(n4 + 3) * KP + k] = w.w;
            }
        }
    }
    float dv[NCB];
    if (EP & EP_DOT) {
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) dv[cb] = a.dot_vec[(size_t)tile.type * NC + cb * 16 + li];
    }
    __syncthreads();

    // Row blocks of this wave: rb = wave + 4 i, i < MB.
    const int nrb = (tile.rows + 15) >> 4;
    const int32_t *any_idx = reinterpret_cast<const int32_t *>(a.tiles + blockIdx.x);
    int xr[MB];
#pragma unroll
    for (int i = 0; i < MB; ++i) {
        const int r = (wave + 4 * i) * 16 + li;
        const int grow = tile.row0 + (r < tile.rows ? r : 0);
        const int ld = *(a.gather ? a.gather + grow : any_idx);
        xr[i] = a.gather ? ld : grow;
    }
    float4 acur[KC], anext[KC];
    int64_t ycur[4], ynext[4];
    auto load_block = [&](int i, float4 (&dst)[KC], int64_t (&ys)[4]) {
        const float *p = a.X + (int64_t)xr[i] * a.ldx + q * 4;
#pragma unroll
        for (int c = 0; c < KC; ++c) dst[c] = *reinterpret_cast<const float4 *>(p + c * 16);
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int r = (wave + 4 * i) * 16 + q * 4 + v;
            const int grow = tile.row0 + (r < tile.rows ? r : 0);
            const int ld = *(a.scatter ? a.scatter + grow : any_idx);
            ys[v] = a.scatter ? ld : grow;
        }
    };
    load_block(0, acur, ycur);
#pragma unroll
    for (int i = 0; i < MB; ++i) {
        const int rb = wave + 4 * i;
        if (rb >= nrb) break;
        // (a) epilogue operands of this block
        float sc[4];
        float ex[4][NCB];
        if (EP & EP_SCALE) {
#pragma unroll
            for (int v = 0; v < 4; ++v) sc[v] = a.row_scale[ycur[v]];
        }
        if (EP & (EP_RESID | EP_ACC)) {
#pragma unroll
            for (int v = 0; v < 4; ++v)
#pragma unroll
                for (int cb = 0; cb < NCB; ++cb) {
                    const int col = cb * 16 + li;
                    float x = 0.f;
                    if (EP & EP_RESID) x += a.residual[ycur[v] * a.ld_res + col];
                    if (EP & EP_ACC) x += a.Y[ycur[v] * a.ldy + col];
                    ex[v][cb] = x;
                }
        }
        // (b) rows and scatter indices of the next block
        if (i + 1 < MB) load_block(i + 1, anext, ynext);
        // (c) MFMAs; B fragments are re-read from LDS for every row block
        // (keeping the whole weight tile in VGPRs would cap occupancy)
        floatx4 acc[NCB];
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) acc[cb] = floatx4{0.f, 0.f, 0.f, 0.f};
        asm volatile("" ::: "memory");
#pragma unroll
        for (int c = 0; c < KC; ++c) {
            float4 b[NCB];
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb)
                b[cb] = *reinterpret_cast<const float4 *>(&Wt[(cb * 16 + li) * KP + c * 16 + q * 4]);
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb)
                acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(acur[c].x, b[cb].x, acc[cb], 0, 0, 0);
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb)
                acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(acur[c].y, b[cb].y, acc[cb], 0, 0, 0);
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb)
                acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(acur[c].z, b[cb].z, acc[cb], 0, 0, 0);
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb)
                acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(acur[c].w, b[cb].w, acc[cb], 0, 0, 0);
        }
        // (d) epilogue: rows 16*rb + 4q + v, columns 16*cb + li
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int r = rb * 16 + q * 4 + v;
            const bool valid = r < tile.rows;
            const int64_t yr = ycur[v];
            float val[NCB];
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb) val[cb] = (EP & EP_SCALE) ? acc[cb][v] * sc[v] : acc[cb][v];
            if (EP & EP_DOT) {
                const int cbh = NCB / a.dot_heads;     // column blocks per head
                for (int hh = 0; hh < a.dot_heads; ++hh) {
                    float part = 0.f;
#pragma unroll
                    for (int cb = 0; cb < NCB; ++cb)
                        if (cb / cbh == hh) part += val[cb] * dv[cb];
                    part = gsum<16>(part);
                    if (valid && li == 0) a.dot_out[yr * a.dot_heads + hh] = part;
                }
            }
            if (!valid) continue;
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb) {
                const int col = cb * 16 + li;
                float o = val[cb];
                if (EP & (EP_RESID | EP_ACC)) o += ex[v][cb];
                if (EP & EP_RELU) o = fmaxf(o, 0.f);
                if ((EP & EP_SPLIT) && col >= a.split) a.Y2[yr * a.ldy2 + (col - a.split)] = o;
                else a.Y[yr * a.ldy + col] = o;
            }
        }
#pragma unroll
        for (int c = 0; c < KC; ++c) acur[c] = anext[c];
#pragma unroll
        for (int v = 0; v < 4; ++v) ycur[v] = ynext[v];
    }
}

template <int K, int NC, int EP>
void launch_k(const GemmK &k, int64_t ntiles, hipStream_t s)
{
    hipLaunchKernelGGL((typed_gemm_kernel<K, NC, EP>), dim3((unsigned)ntiles), dim3(256), 0, s, k);
}

// Epilogues instantiated per shape: square shapes serve every layer; the
// rectangular ones serve RGCN with d_in != d_out and the segment-MM entry
// point; 64 x 192 is the fused K|V|Q projection of HGT.
template <int K, int NC>
bool dispatch_square(int ep, const GemmK &k, int64_t n, hipStream_t s)
{
    switch (ep) {
    case 0: launch_k<K, NC, 0>(k, n, s); return true;
    case EP_DOT: launch_k<K, NC, EP_DOT>(k, n, s); return true;
    case EP_SCALE: launch_k<K, NC, EP_SCALE>(k, n, s); return true;
    case EP_ACC: launch_k<K, NC, EP_ACC>(k, n, s); return true;
    case EP_ACC | EP_RELU: launch_k<K, NC, EP_ACC | EP_RELU>(k, n, s); return true;
    case EP_RESID: launch_k<K, NC, EP_RESID>(k, n, s); return true;
    default: return false;
    }
}

template <int K, int NC>
bool dispatch_rect(int ep, const GemmK &k, int64_t n, hipStream_t s)
{
    switch (ep) {
    case 0: launch_k<K, NC, 0>(k, n, s); return true;
    case EP_ACC: launch_k<K, NC, EP_ACC>(k, n, s); return true;
    case EP_ACC | EP_RELU: launch_k<K, NC, EP_ACC | EP_RELU>(k, n, s); return true;
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
    k.dot_vec = a.ep.dot_vec; k.dot_out = a.ep.dot_out; k.dot_heads = a.ep.dot_heads;
    k.residual = a.ep.residual; k.ld_res = a.ep.ld_res;
    k.Y2 = a.ep.Y2; k.ldy2 = a.ep.ldy2; k.split = a.ep.split;
    if (a.trans_b && a.nparts != 1) return fail(RGNN_EINVAL, "transposed B takes one part");
    if (a.Nc % a.nparts) return fail(RGNN_EINVAL, "column parts must split Nc evenly");
    if (a.ep.dot_out && ((a.Nc / 16) % a.ep.dot_heads))
        return fail(RGNN_EUNSUPPORTED, "dot-product heads must own whole 16-column blocks");
    const int ep = (a.ep.dot_out ? EP_DOT : 0) | (a.ep.row_scale ? EP_SCALE : 0) |
                   (a.ep.residual ? EP_RESID : 0) | (a.ep.accumulate ? EP_ACC : 0) |
                   (a.ep.relu ? EP_RELU : 0) | (a.ep.Y2 ? EP_SPLIT : 0);
    bool ok = false;
    {
        LaunchScope ls("typed_gemm", s);
        if (a.K == 64 && a.Nc == 64) ok = dispatch_square<64, 64>(ep, k, a.ntiles, s);
        else if (a.K == 128 && a.Nc == 128) ok = dispatch_square<128, 128>(ep, k, a.ntiles, s);
        else if (a.K == 64 && a.Nc == 128) ok = dispatch_rect<64, 128>(ep, k, a.ntiles, s);
        else if (a.K == 128 && a.Nc == 64) ok = dispatch_rect<128, 64>(ep, k, a.ntiles, s);
        else if (a.K == 64 && a.Nc == 192 && ep == EP_SPLIT) {
            launch_k<64, 192, EP_SPLIT>(k, a.ntiles, s);
            ok = true;
        }
    }
    if (!ok) return fail(RGNN_EUNSUPPORTED, "typed GEMM: unsupported shape / epilogue combination");
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? RGNN_OK : hip_fail(e, "typed_gemm launch");
}

}  // namespace rgnn
