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
//     bytes of its row per load), the next block's rows are prefetched while
//     the current block's MFMAs run;
//   * the epilogue fuses what the paper's fusion rule allows into the GEMM:
//     a per-row scalar (attention / normalisation), a per-row dot product with
//     a per-type vector (the reordered attention term), residual add,
//     accumulation, ReLU, and a split of the output columns into two tensors.
//
// MFMA operand layout used (v_mfma_f32_16x16x4f32, one block): lane l supplies
// A[l%16][l/16] and B[l/16][l%16]; the 4 accumulator VGPRs of lane l hold
// D[4*(l/16)+v][l%16], v = 0..3.  The k-slot q = l/16 of step (c, t) is mapped
// to the actual reduction index kk = 16c + 4q + t, identically for A and B.
#include "rgnn_internal.h"

namespace rgnn {

namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));

struct GemmK {
    const float *X; int64_t ldx;
    const int32_t *gather;
    const float *W0, *W1, *W2;
    int nparts, trans_b;
    const Tile *tiles;
    float *Y; int64_t ldy;
    const int32_t *scatter;
    // epilogue
    int scale_mode;
    const float *seg_stat; const int32_t *row_dst; const float *dst_stat;
    const float *dot_vec; float *dot_out; int dot_heads;
    const float *residual; int64_t ld_res;
    int accumulate, relu;
    float *Y2; int64_t ldy2; int split;
};

template <int K, int NC>
__global__ __launch_bounds__(256) void typed_gemm_kernel(GemmK a)
{
    constexpr int KP = K + 4;           // padded LDS row (conflict-free b128 reads)
    constexpr int NCB = NC / 16;        // 16-column blocks
    constexpr int KC = K / 16;          // 16-wide k chunks (4 MFMA steps each)
    __shared__ float Wt[NC * KP];

    const Tile tile = a.tiles[blockIdx.x];
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int li = lane & 15, q = lane >> 4;

    // ---- stage W[type] transposed into LDS: Wt[n][k] = B[k][n] ----
    {
        const int NP = NC / a.nparts;
        for (int idx = tid; idx < K * NC; idx += 256) {
            if (a.trans_b) {               // stored [types][NC][K]: copy rows
                const int n = idx / K, k = idx % K;
                Wt[n * KP + k] = a.W0[((size_t)tile.type * NC + n) * K + k];
            } else {                       // stored [types][K][NP] per part
                const int k = idx / NC, n = idx % NC;
                const int part = n / NP, nn = n % NP;
                const float *Wp = part == 0 ? a.W0 : (part == 1 ? a.W1 : a.W2);
                Wt[n * KP + k] = Wp[((size_t)tile.type * K + k) * NP + nn];
            }
        }
    }
    __syncthreads();

    const int nrb = (tile.rows + 15) >> 4;
    auto xrow_of = [&](int rb) -> const float * {
        const int r = rb * 16 + li;
        const int grow = tile.row0 + (r < tile.rows ? r : 0);
        const int64_t xr = a.gather ? a.gather[grow] : grow;
        return a.X + xr * a.ldx + q * 4;
    };

    float4 acur[KC], anext[KC];
    int rb = wave;
    if (rb < nrb) {
        const float *p = xrow_of(rb);
#pragma unroll
        for (int c = 0; c < KC; ++c) acur[c] = *reinterpret_cast<const float4 *>(p + c * 16);
    }
    for (; rb < nrb; rb += 4) {
        if (rb + 4 < nrb) {
            const float *p = xrow_of(rb + 4);
#pragma unroll
            for (int c = 0; c < KC; ++c) anext[c] = *reinterpret_cast<const float4 *>(p + c * 16);
        }
        floatx4 acc[NCB];
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) acc[cb] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < KC; ++c) {
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb) {
                const float4 b = *reinterpret_cast<const float4 *>(&Wt[(cb * 16 + li) * KP + c * 16 + q * 4]);
                acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(acur[c].x, b.x, acc[cb], 0, 0, 0);
                acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(acur[c].y, b.y, acc[cb], 0, 0, 0);
                acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(acur[c].z, b.z, acc[cb], 0, 0, 0);
                acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(acur[c].w, b.w, acc[cb], 0, 0, 0);
            }
        }
        // ---- epilogue: rows 16*rb + 4q + v, columns 16*cb + li ----
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int r = rb * 16 + q * 4 + v;
            const bool valid = r < tile.rows;
            const int grow = tile.row0 + (valid ? r : 0);
            const int64_t yr = a.scatter ? a.scatter[grow] : grow;
            float scale = 1.f;
            if (a.scale_mode == 1 && valid) {
                const int dst = a.row_dst[yr];
                const float dm = a.dst_stat[(size_t)dst * 2], ds = a.dst_stat[(size_t)dst * 2 + 1];
                scale = __expf(a.seg_stat[yr * 2] - dm) / ds;
            }
            float val[NCB];
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb) val[cb] = acc[cb][v] * scale;
            if (a.dot_out) {
                const int cbh = NCB / a.dot_heads;     // column blocks per head
                for (int hh = 0; hh < a.dot_heads; ++hh) {
                    float part = 0.f;
#pragma unroll
                    for (int cb = 0; cb < NCB; ++cb)
                        if (cb / cbh == hh)
                            part += val[cb] * a.dot_vec[(size_t)tile.type * NC + cb * 16 + li];
                    part += __shfl_xor(part, 8, 16);
                    part += __shfl_xor(part, 4, 16);
                    part += __shfl_xor(part, 2, 16);
                    part += __shfl_xor(part, 1, 16);
                    if (valid && li == 0) a.dot_out[yr * a.dot_heads + hh] = part;
                }
            }
            if (!valid) continue;
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb) {
                const int col = cb * 16 + li;
                float o = val[cb];
                if (a.residual) o += a.residual[yr * a.ld_res + col];
                if (col < a.split) {
                    float *dst = a.Y + yr * a.ldy + col;
                    if (a.accumulate) o += *dst;
                    if (a.relu) o = fmaxf(o, 0.f);
                    *dst = o;
                } else {
                    float *dst = a.Y2 + yr * a.ldy2 + (col - a.split);
                    if (a.accumulate) o += *dst;
                    if (a.relu) o = fmaxf(o, 0.f);
                    *dst = o;
                }
            }
        }
        if (rb + 4 < nrb) {
#pragma unroll
            for (int c = 0; c < KC; ++c) acur[c] = anext[c];
        }
    }
}

template <int K, int NC>
void launch_k(const GemmK &k, int64_t ntiles, hipStream_t s)
{
    hipLaunchKernelGGL((typed_gemm_kernel<K, NC>), dim3((unsigned)ntiles), dim3(256), 0, s, k);
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
    k.scale_mode = a.ep.scale_mode; k.seg_stat = a.ep.seg_stat; k.row_dst = a.ep.row_dst;
    k.dst_stat = a.ep.dst_stat; k.dot_vec = a.ep.dot_vec; k.dot_out = a.ep.dot_out;
    k.dot_heads = a.ep.dot_heads; k.residual = a.ep.residual; k.ld_res = a.ep.ld_res;
    k.accumulate = a.ep.accumulate; k.relu = a.ep.relu;
    k.Y2 = a.ep.Y2; k.ldy2 = a.ep.ldy2; k.split = a.ep.Y2 ? a.ep.split : a.Nc;
    if (a.trans_b && a.nparts != 1) return fail(RGNN_EINVAL, "transposed B takes one part");
    if (a.Nc % a.nparts) return fail(RGNN_EINVAL, "column parts must split Nc evenly");
    if (a.ep.dot_out && ((a.Nc / 16) % a.ep.dot_heads))
        return fail(RGNN_EUNSUPPORTED, "dot-product heads must own whole 16-column blocks");
    LaunchScope ls("typed_gemm", s);
    if (a.K == 64 && a.Nc == 64) launch_k<64, 64>(k, a.ntiles, s);
    else if (a.K == 128 && a.Nc == 128) launch_k<128, 128>(k, a.ntiles, s);
    else if (a.K == 64 && a.Nc == 128) launch_k<64, 128>(k, a.ntiles, s);
    else if (a.K == 128 && a.Nc == 64) launch_k<128, 64>(k, a.ntiles, s);
    else if (a.K == 64 && a.Nc == 192) launch_k<64, 192>(k, a.ntiles, s);
    else return fail(RGNN_EUNSUPPORTED, "typed GEMM supports K in {64,128}, Nc in {64,128,192}");
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? RGNN_OK : hip_fail(e, "typed_gemm launch");
}

}  // namespace rgnn
