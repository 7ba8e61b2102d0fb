// rgnn_internal.h -- shared definitions of librgnn (host + device code).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>
#include <vector>

#include "rgnn.h"

namespace rgnn {

// Maximum in-edges one traversal work item handles.  Destinations with more
// in-edges are split into several items whose partial softmax states are merged.
constexpr int kChunkEdges = 64;
// Maximum destinations bundled into one work item.
constexpr int kMaxDstPerItem = 32;
// Rows of one typed-GEMM tile (a tile never mixes weight types).
constexpr int kGemmTileRows = 512;
// fused aggregate-first tiles: at most this many segments of one relation and,
// beyond the first 16-row block, at most this many in-edges
constexpr int kFusedTileRows = 256;
constexpr int kFusedTileEdges = 4096;
// Reductions over more records than this (partials of a split destination,
// segments of one destination) get a whole workgroup instead of one group.
constexpr int kBigRange = 32;
// Split destinations / sources with more slots than this have their slot sums
// taken by a whole workgroup, the others by a single wave.
constexpr int kWaveSlots = 64;
// the partials of a destination split over more than kBigRange items are
// merged in two levels: chunks of kMergeChunk partials, then the chunks
constexpr int kMergeChunk = 128;
// rows (segments or nodes) per K-chunk of the backward outer-product GEMMs
constexpr int kOuterRows = 2048;
// several-head backward, pair pass: out-edges per virtual pair (longer pairs
// are cut into pieces) and virtual pairs per workgroup chunk
constexpr int kPairPiece = 64;
constexpr int kPairChunkRows = 1024;

struct Tile {          // one typed-GEMM tile: rows [row0, row0 + rows) of type `type`
    int32_t type, row0, rows, pad;
};

struct FusedRow {      // one virtual segment in the fused aggregate-first order
    int32_t vs;           // virtual segment id
    int32_t e0, ne;       // its in-edges' sources at [e0, e0 + ne) of the fused source list
    int32_t cnt;          // edge count of its whole (dst, rel) segment; ~v (negative) when the
                          // segment is the only virtual segment of its destination v (then
                          // the whole segment is this one: its count is ne)
};

struct Item {          // one traversal work item
    int32_t dst0, dst1;   // destinations [dst0, dst1)
    int32_t vs0, vs1;     // virtual segments [vs0, vs1) (subset of the destinations' ones)
};

// Host copy of every index array (kept for host-only graphs and while building).
struct HostIndex {
    std::vector<int32_t> rowptr, in_src, in_rel, in_eid;
    std::vector<int32_t> seg_ptr, seg_rel, dst_segptr;
    std::vector<int32_t> uniq_src, uniq_rel_ptr, e2u;
    std::vector<int32_t> ntype_perm, ntype_ptr;
    std::vector<int32_t> rel_dsttype;   // node type of every relation's destinations (-1: mixed)
    // scheduling
    std::vector<int32_t> vseg_ptr, vseg_rel, vseg_dst, vseg_cnt, dst_vsegptr;
    std::vector<int32_t> vseg_byrel, rel_vsegptr, vsegdst_byrel;
    std::vector<Item> items;
    std::vector<int32_t> item_slot, split_dst, split_slotptr;
    std::vector<int32_t> split_items;   // items that are pieces of split destinations (slot >= 0)
    std::vector<int32_t> big_split;   // indices into split_dst with > kBigRange slots
    std::vector<int32_t> split_order;   // indices into split_dst, most slots first [n_split]
    std::vector<int32_t> big_chunkptr;  // chunks of each big split [n_big_split + 1]
    std::vector<int32_t> chunk_lo, chunk_hi;   // slot range of each chunk [n_big_chunks]
    std::vector<int32_t> reduce_dst;  // destinations with 0 or 2..kBigRange virtual segments
    std::vector<int32_t> big_vdst;    // destinations with > kBigRange virtual segments,
                                      // largest first
    std::vector<int32_t> seg_vsegptr;  // first virtual segment of each (dst, rel) segment [U_dst+1]
    std::vector<int32_t> big_seg;      // (dst, rel) segments with > kBigRange virtual segments
    std::vector<int32_t> osplit;       // sources whose out-edges span several out-edge items
    std::vector<int32_t> oitem_slot;   // per out-edge item: its slot if it is a piece of such a
                                       // source, else -1 [n_oitems]
    std::vector<int32_t> osplit_slotptr;   // slots of each of those sources [n_osplit+1]
    std::vector<int32_t> osplit_order;     // indices into osplit, most slots first [n_osplit]
    std::vector<FusedRow> fused_rows;  // vsegs by (rel, edge count desc, id) [V]
    std::vector<Tile> tiles_fused;     // tiles over fused_rows (pad: first fused_src position)
    std::vector<int32_t> fused_src;    // in-edge sources, segment by segment in fused order [E]
    std::vector<int32_t> vseg_fpos;    // position of each vseg in fused_rows [V]
    std::vector<int32_t> vseg_seg;     // (dst, rel) segment of each vseg [V]
    std::vector<Tile> tiles_pairs, tiles_vsegs, tiles_nodes, tiles_all, tiles_outer;
    std::vector<Tile> tiles_vsegs_dst;   // tiles_vsegs' rows by destination range, XCD-interleaved
    std::vector<int32_t> rel_chunkptr;   // outer-product chunks per relation [R+1]
    std::vector<float> invcnt_byrel;      // 1 / c_{v,r} of each virtual segment, by-relation order
    std::vector<Tile> tiles_nodes_outer;  // outer-product chunks over all nodes
    std::vector<int32_t> nodes_chunkptr;  // {0, number of node chunks}
    std::vector<Tile> tiles_types_outer;  // outer-product chunks over the nodes of each type
    std::vector<int32_t> types_chunkptr;  // chunks per node type [T+1]
    std::vector<int32_t> rel_pairtileptr;   // compact-pair GEMM tiles per relation [R+1]
    // out-edges (source-major view of the sorted in-edges), for the backward pass
    std::vector<int32_t> out_ptr, out_pos, out_vseg, out_rel, out_pair;
    std::vector<int32_t> out_vs, out_dst;   // per out-edge: its in-edge's vseg id and destination
    std::vector<int32_t> vseg_pos;       // position of each vseg in the by-relation order
    std::vector<Item> oitems;            // {node0, node1, q0, q1} over out-edge offsets
    // compact pairs in source-major order (several-head backward)
    std::vector<int32_t> src_pairptr;    // [N+1] pairs of each source in that order
    std::vector<int32_t> pair_smpos;     // [U_src] position of each pair in that order
    std::vector<Tile> tiles_outer_pairs;  // outer-product chunks over the pairs of each relation
    std::vector<int32_t> rel_pairchunkptr;   // those chunks per relation [R+1]
    // virtual pairs: the compact pairs of each relation in (rel, src) order, cut
    // into pieces of at most kPairPiece out-edges
    std::vector<int32_t> vpair_oe0, vpair_ne;   // out-edge range of each virtual pair [NVP]
    std::vector<int32_t> vpair_src;             // its source [NVP]
    std::vector<int32_t> vpair_smpos;           // its row in source-major order [NVP]
    std::vector<int32_t> src_vpairptr;          // virtual pairs of each source in that order [N+1]
    std::vector<Tile> tiles_vpairs;             // chunks of kPairChunkRows virtual pairs of one relation
    std::vector<int32_t> rel_vpairchunkptr;     // those chunks per relation [R+1]
};

// Device copies (one allocation, carved).
struct DeviceIndex {
    void *base = nullptr;
    size_t bytes = 0;
    int32_t *rowptr = nullptr, *in_src = nullptr, *in_rel = nullptr, *in_eid = nullptr;
    int32_t *seg_ptr = nullptr, *seg_rel = nullptr, *dst_segptr = nullptr;
    int32_t *uniq_src = nullptr, *uniq_rel_ptr = nullptr, *e2u = nullptr;
    int32_t *ntype_perm = nullptr, *ntype_ptr = nullptr, *rel_dsttype = nullptr;
    int32_t *vseg_ptr = nullptr, *vseg_rel = nullptr, *vseg_dst = nullptr, *vseg_cnt = nullptr;
    int32_t *dst_vsegptr = nullptr, *vseg_byrel = nullptr, *rel_vsegptr = nullptr;
    int32_t *vsegdst_byrel = nullptr, *rel_chunkptr = nullptr, *rel_pairtileptr = nullptr;
    Item *items = nullptr;
    int32_t *item_slot = nullptr, *split_dst = nullptr, *split_slotptr = nullptr, *split_items = nullptr;
    int32_t *big_split = nullptr, *big_vdst = nullptr, *reduce_dst = nullptr;
    int32_t *big_chunkptr = nullptr, *chunk_lo = nullptr, *chunk_hi = nullptr;
    int32_t *seg_vsegptr = nullptr, *big_seg = nullptr, *osplit = nullptr;
    int32_t *oitem_slot = nullptr, *osplit_slotptr = nullptr;
    int32_t *split_order = nullptr, *osplit_order = nullptr;
    float *invcnt_byrel = nullptr;
    Tile *tiles_nodes_outer = nullptr;
    int32_t *nodes_chunkptr = nullptr;
    Tile *tiles_types_outer = nullptr;
    int32_t *types_chunkptr = nullptr;
    FusedRow *fused_rows = nullptr;
    int32_t *fused_src = nullptr;
    int32_t *vseg_fpos = nullptr;
    int32_t *vseg_seg = nullptr;
    Tile *tiles_fused = nullptr;
    Tile *tiles_vsegs_dst = nullptr;
    Tile *tiles_pairs = nullptr, *tiles_vsegs = nullptr, *tiles_nodes = nullptr,
         *tiles_all = nullptr, *tiles_outer = nullptr;
    int32_t *out_ptr = nullptr, *out_pos = nullptr, *out_vseg = nullptr, *out_rel = nullptr;
    int32_t *out_pair = nullptr, *out_vs = nullptr, *out_dst = nullptr;
    int32_t *vseg_pos = nullptr;
    Item *oitems = nullptr;
    int32_t *src_pairptr = nullptr, *pair_smpos = nullptr, *rel_pairchunkptr = nullptr;
    Tile *tiles_outer_pairs = nullptr;
    int32_t *vpair_oe0 = nullptr, *vpair_ne = nullptr, *vpair_src = nullptr, *vpair_smpos = nullptr;
    int32_t *src_vpairptr = nullptr, *rel_vpairchunkptr = nullptr;
    Tile *tiles_vpairs = nullptr;
};

}  // namespace rgnn

struct rgnn_graph {
    int64_t N = 0, E = 0;
    int32_t R = 0, T = 0;
    int64_t U_src = 0, U_dst = 0, V = 0;
    int64_t n_items = 0, n_split = 0, n_slots = 0;
    int64_t max_in_deg = 0, n_empty = 0;
    int32_t chunk = rgnn::kChunkEdges;
    int32_t device = -1;
    int64_t n_tiles_pairs = 0, n_tiles_vsegs = 0, n_tiles_nodes = 0, n_tiles_all = 0;
    int64_t n_tiles_vsegs_dst = 0;
    int64_t n_tiles_outer = 0, n_tiles_fused = 0, n_tiles_nodes_outer = 0, n_tiles_types_outer = 0;
    int64_t n_big_split = 0, n_big_vdst = 0, n_big_seg = 0, n_big_chunks = 0, n_reduce_dst = 0;
    int64_t n_oitems = 0, n_osplit = 0, n_oslots = 0, n_split_items = 0, n_tiles_outer_pairs = 0;
    int64_t n_vpairs = 0, n_tiles_vpairs = 0;
    int64_t n_split_wide = 0, n_osplit_wide = 0;   // split lists' entries with > kWaveSlots slots
    bool rel_dst_typed = false;   // every relation's destinations share one node type
    rgnn::HostIndex host;
    rgnn::DeviceIndex dev;
};

namespace rgnn {

// ---- error reporting (api.cpp) ----
rgnn_status fail(rgnn_status st, const std::string &msg);
rgnn_status hip_fail(hipError_t e, const char *what);

// ---- graph building (graph.cpp) ----
rgnn_status build_host_index(int64_t N, int32_t T, int32_t R, int64_t E, const int32_t *src,
                             const int32_t *dst, const int32_t *rel, const int32_t *ntype,
                             int32_t flags, rgnn_graph *g);
void build_tiles(const std::vector<int32_t> &type_ptr, int tile_rows, std::vector<Tile> &out);
rgnn_status launch_add(float *out, const float *a, const float *b, int64_t n, hipStream_t s);
// out [rows, d] = in with the columns outside [c0, c1) set to 0
rgnn_status launch_mask_cols(const float *in, float *out, int64_t rows, int d, int c0, int c1, hipStream_t s);
// out [N, 2] = saved [N, H, 2] of head k, and the converse
rgnn_status launch_head_stats(const float *saved, float *out, int64_t N, int H, int k, hipStream_t s);
rgnn_status launch_head_stats_scatter(const float *in, float *saved, int64_t N, int H, int k, hipStream_t s);

// ---- profiling (api.cpp) ----
struct LaunchScope {   // records a hipEvent pair around one kernel launch when profiling
    LaunchScope(const char *name, hipStream_t s);
    ~LaunchScope();
    const char *name;
    hipStream_t stream;
    int slot;
};

// ---- kernel launchers (device .hip files) ----
struct GemmEpilogue {
    // Optional per-row scale of the A rows (Section "Operator-Specific Schedule":
    // a per-row scalar applied to the tiles of matrix A), indexed by scatter id.
    const float *row_scale = nullptr;
    // Optional row dot products of the output with a per-type vector, written to
    // dot_out[scatter_row * dot_ld + head] (heads split the output columns;
    // dot_ld 0 means heads).
    const float *dot_vec = nullptr;    // [types, Nc]
    float *dot_out = nullptr;
    int dot_heads = 1;
    int64_t dot_ld = 0;
    // Optional residual: Y[row] += res[row] (same row index as the output).
    const float *residual = nullptr;
    int64_t ld_res = 0;
    int accumulate = 0;                // Y[row] += result instead of =
    int relu = 0;                      // apply max(0, .) after everything
    // Second output for columns >= split (split == Nc: unused).
    float *Y2 = nullptr;
    int64_t ldy2 = 0;
    int split = 0;
    // W[type] is block-diagonal with this many equal blocks (> 1: the
    // off-diagonal products are skipped; no other epilogue may be set).
    int diag_blocks = 1;
};

struct GemmArgs {
    const float *X = nullptr;   int64_t ldx = 0;
    const int32_t *gather = nullptr;     // row -> X row (NULL: identity)
    const float *W[3] = {nullptr, nullptr, nullptr};   // column parts, each [types, K, Np]
    int nparts = 1;
    int trans_b = 0;                     // B = W[type]^T (W stored [types, Nc, K])
    int K = 0, Nc = 0;
    const Tile *tiles = nullptr;   int64_t ntiles = 0;
    float *Y = nullptr;   int64_t ldy = 0;
    const int32_t *scatter = nullptr;    // row -> Y row (NULL: identity)
    GemmEpilogue ep;
    // Products from exact three-piece bf16 splits on the bf16 matrix cores
    // (fp32-accurate, see gemm.hip) for the 64- and 128-deep shapes.  The
    // forward layers and the RGCN and HGT backward passes take it; the RGAT
    // backward keeps the fp32 matrix cores (its gradients' near-cancelling
    // rows -- softmax Jacobian sums -- are pinned at that rounding).
    int split_bf16 = 0;
};
rgnn_status launch_typed_gemm(const GemmArgs &a, hipStream_t s);

// Reordered attention vectors: out1[r, k, :] = W_r[:, k-cols] v1[r, k-cols]
// and the same for v2 into out2 when v2 is not NULL (one launch).
rgnn_status launch_reorder_vec(const float *W, int R, int d_in, int d_out, int heads,
                               const float *v1, float *out1, const float *v2, float *out2,
                               hipStream_t s);

struct TravArgs {
    const rgnn_graph *g = nullptr;
    const float *h = nullptr;            // node features [N, d_in]
    const float *M = nullptr;            // compact messages [U_src, d_out] (transform-first)
    const float *wsp = nullptr;          // vector dotted with each gathered row for the source
                                         // term: [R, d_in] W_r w_src (aggregate-first), or
                                         // [R, d_out] w_src (transform-first, per head slice)
    const float *wtp = nullptr;          // [R, heads, d_in] reordered w_dst
    float slope = 0.2f;
    int heads = 1;
    int d = 64;
    float *out = nullptr;                // [N, d]
    float *saved = nullptr;              // [N, heads, 2] or NULL
    float *partial = nullptr;            // [slots, 2*heads + d]
    float *vstat = nullptr;              // aggregate-first: [V, 2] per-vseg (max, sum), fused order
    float *vatt = nullptr;               // [V, heads] destination attention term per vseg
    float *vscale = nullptr;             // aggregate-first: [V] softmax scale per vseg
    int relu = 0;
    // transform-first with the attention+message rows: each row of M holds the
    // d_out message features, then the per-head source terms (row stride
    // att_row_ld()); the traversal reads the terms instead of forming them
    int att_in_row = 0;
};
// Row stride (floats) of the attention+message rows: d_out message features,
// then the heads' source terms padded to whole 16-byte groups.
inline int att_row_ld(int d_out, int heads) { return d_out + 4 * ((heads + 3) / 4); }
// vatt[vs, k] = h_v . wtp[r, k] for every virtual segment (v, r).
rgnn_status launch_seg_attn(const TravArgs &a, hipStream_t s);
rgnn_status launch_rgcn_traverse_tf(const TravArgs &a, hipStream_t s);
rgnn_status launch_rgat_traverse_tf(const TravArgs &a, hipStream_t s);
// Finish destinations split over several work items: combine their partials
// (softmax: (max, sum) per head then the D-vector; else the D-vector only).
// The partials of destinations with many pieces are overwritten (the chunk
// records of the two-level merge).
rgnn_status launch_merge_partials(const rgnn_graph *g, int d, int heads, int softmax,
                                  float *partial, float *out, float *saved, int relu,
                                  hipStream_t s);
// Softmax per (dst, rel) segment: per virtual segment the scale
// exp(m_i - M_seg) / Z_seg from the pieces' (max, sum) in a.vstat, to a.vscale.
rgnn_status launch_seg_softmax_scale(const TravArgs &a, hipStream_t s);
// out_v (+)= sum over v's virtual segments of scale[vs] * T[vs] (scale NULL: 1);
// out rows ldo floats apart (0: d).  skip1: destinations with a single virtual
// segment are left alone (the fused kernel wrote their rows).
rgnn_status launch_vseg_reduce(const rgnn_graph *g, const float *T, const float *scale, int d,
                               float *out, int accumulate, int relu, hipStream_t s, int64_t ldo = 0,
                               int skip1 = 0);

// Softmax per destination finished from the per-segment (max, sum) in vstat
// (fused order) and the segments' transformed rows summed: out_v = sum_i
// exp(m_i - M_v) / Z_v * T_i; saved[v] = (M_v, Z_v) when saved is not NULL.
// scale [V]: scratch (the weights of destinations with many segments).
// skip1: destinations with a single virtual segment are left alone (the fused
// kernel wrote their rows and statistics).
rgnn_status launch_softmax_reduce(const rgnn_graph *g, const float *vstat, const float *T, int d,
                                  float *out, float *saved, float *scale, int skip1, hipStream_t s);

// Fused aggregate-first gather + segment sum + transform: per virtual segment
// T[vs] = S_vs W_r with S_vs the segment's mean of h_u (softmax == 0) or its
// exp-weighted sum relative to the segment's own logit maximum (softmax == 1,
// one head; (max, sum) to vstat at the fused position).
struct FusedArgs {
    const rgnn_graph *g = nullptr;
    const float *h = nullptr;     // [N, d_in]
    const float *W = nullptr;     // [R, d_in, d_out]
    const float *wsp = nullptr;   // [R, d_in] W_r w_src[r] (softmax)
    const float *vatt = nullptr;  // [V] destination terms (softmax)
    float slope = 0.2f;
    int d_in = 64, d_out = 64;
    int softmax = 0;
    float *T = nullptr;           // [V, d_out]
    float *vstat = nullptr;       // [V, 2] (softmax), indexed by fused position
    // optional: a destination with a single virtual segment gets its output
    // row [N, d_out] here, not in T (softmax: and its (max, sum) [N, 2] in
    // saved, not in vstat; mean: with ReLU when relu is set)
    float *out = nullptr, *saved = nullptr;
    int relu = 0;
    // S given (softmax == 0): write the segment means S_vs = (1/c) sum h_u
    // themselves, at the segment's by-relation position [V, d_in], no transform
    float *S = nullptr;
};
rgnn_status launch_af_fused(const FusedArgs &a, hipStream_t s);

// Outer-product chunks of the backward: partial[c] (d x d, d in {32, 64, 128})
// = sum over the rows of chunk c of X[x(row)]^T Gm[g(row)], g(row) = gather ?
// gather[row] : row and x(row) = g(row) when gather_x, else row; ldx, ldg: row
// strides.
rgnn_status launch_outer_chunks(const Tile *chunks, int64_t nchunks, const int32_t *gather, int gather_x,
                                const float *X, int ldx, const float *Gm, int ldg, float *partial, int d,
                                hipStream_t s);
// dW[r] = sum of partial[c] for c in [chunkptr[r], chunkptr[r+1]) in order (d x d each).
// Pieces of split sources: dh[osplit[i]] += the partial rows of its slots
// [osplit_slotptr[i], osplit_slotptr[i + 1]) in a fixed order (d in {32, 64, 128}).
rgnn_status launch_src_merge(const rgnn_graph *g, const float *part, float *dh, int d, hipStream_t s);
// out[ids[i] * w ...] = (accumulate: +=) the sum of the w-float rows part[sl], sl in
// [slotptr[i], slotptr[i + 1]), for all n entries, in a fixed order (w in {2, 4, 8,
// 16, 32, 64, 128}).  order lists the entries with the nwide ones holding more than
// kWaveSlots slots first: each of those takes a 1024-thread workgroup, the others a
// wave each (sixteen per workgroup).
rgnn_status launch_slot_sum(int64_t n, int64_t nwide, const int32_t *order, const int32_t *ids,
                            const int32_t *slotptr, const float *part, float *out, int w, bool accumulate,
                            const char *name, hipStream_t s);
rgnn_status launch_chunk_sum(const float *partial, const int32_t *chunkptr, int R, float *dW, int d,
                             hipStream_t s);
// RGAT backward with several heads (2 to 8, d / heads >= 16) in one pass over
// the graph; need != NULL: only the workspace size.
rgnn_status rgat_backward_heads_impl(const rgnn_graph *g, const float *h, const float *W, const float *w_src,
                                     const float *w_dst, int d, int heads, float slope, int per_seg,
                                     const float *saved, const float *Gm, float *dh, float *dW, float *dws,
                                     float *dwt, void *ws, size_t ws_bytes, hipStream_t s, size_t *need);
rgnn_status launch_fill(float *p, int64_t n, float v, hipStream_t s);
rgnn_status launch_relu(float *p, int64_t n, hipStream_t s);

struct HgtArgs {
    const rgnn_graph *g = nullptr;
    const float *KV = nullptr;     // [N, 2d]: K then V per node
    const float *QP = nullptr;     // [V, d]: mu[r] * scale * Q_t Watt[r]^T per virtual segment,
                                   // or NULL: formed in the kernel from Q, Watt, mu, scale
                                   // (when hgt_fused_query_fits)
    const float *Q = nullptr, *Watt = nullptr, *mu = nullptr;
    float scale = 1.f;
    const float *Wmsg = nullptr;
    int heads = 4;
    int d = 64;
    float *agg = nullptr;          // [N, d]
    float *partial = nullptr;      // [slots, 2*heads + d]
    float *saved = nullptr;        // [N, heads, 2] softmax (max, sum) or NULL (split
                                   // destinations: written by the partial merge)
};
rgnn_status launch_hgt_traverse(const HgtArgs &a, hipStream_t s);
// Whether the traversal can form the segment queries itself (d = 128, both
// per-relation weight sets and the work-item stages in one workgroup's LDS).
bool hgt_fused_query_fits(int R, int d, int heads);
// Wqp[r] (d x d) = mu[r] * scale * blockdiag over heads i of Watt[r, i]^T, so
// that Q_t Wqp[r] is the reordered query of segment (t, r).
rgnn_status launch_hgt_qp_weights(const float *Watt, const float *mu, float scale, int R, int d,
                                  int heads, float *Wqp, hipStream_t s);
// Wc[r] (d x d) = Wq[rel_dsttype[r]] Wqp[r]: the query projection folded into
// the reordered query weights, so that h_t Wc[r] is the query of segment (t, r)
// when every destination of r has node type rel_dsttype[r].
rgnn_status launch_hgt_qp_fold(const float *Wq, const float *Watt, const float *mu, float scale,
                               const int32_t *rel_dsttype, int R, int d, int heads, float *Wc, hipStream_t s);

// One head's share of a several-head RGAT backward run as one-head passes:
// only the output columns [col0, col1) of dW take the outer products (the
// weights and attention vectors the pass gets are zero outside them), and with
// acc the pass adds dh, dW, dw_src, dw_dst to what the outputs hold.
struct BwdHead {
    int col0 = 0, col1 = 1 << 30, acc = 0;
};

// RGAT backward (backward.hip), one head.  per_seg: softmax per (dst, rel)
// segment, saved [U_dst, 2]; else per destination, saved [N, 2].  With
// need != NULL only stores the workspace bytes the call needs.
rgnn_status rgat_backward_impl(const rgnn_graph *g, const float *h, const float *W,
                               const float *w_src, const float *w_dst, int d_in, int d_out,
                               float slope, int per_seg, const float *saved, const float *Gm,
                               float *dh, float *dW, float *dws, float *dwt, void *ws,
                               size_t ws_bytes, hipStream_t s, size_t *need, BwdHead hd = BwdHead());

// HGT backward (hgt_backward.hip), the same convention for need.
rgnn_status hgt_backward_impl(const rgnn_graph *g, const float *h, const float *Wk, const float *Wq,
                              const float *Wv, const float *Wa, const float *Watt, const float *Wmsg,
                              const float *mu, int d, int heads, float att_scale, int flags,
                              const float *Gm, const float *saved, float *dh, float *dWk, float *dWq,
                              float *dWv, float *dWa, float *dWatt, float *dWmsg, float *dmu, void *ws,
                              size_t ws_bytes, hipStream_t s, size_t *need);

// RGCN backward (rgcn_backward.hip), the same convention for need.
rgnn_status rgcn_backward_impl(const rgnn_graph *g, const float *h, const float *W, const float *W0,
                               int d_in, int d_out, int flags, const float *out, const float *Gm,
                               float *dh, float *dW, float *dW0, void *ws, size_t ws_bytes,
                               hipStream_t s, size_t *need);

}  // namespace rgnn
