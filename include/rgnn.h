/*
 * rgnn.h -- C ABI of librgnn.so: RGCN, RGAT and HGT layers and the RGAT
 * backward pass on one MI355X (gfx950), in fp32.
 *
 * The layers follow the definitions of Hector (ASPLOS '24, arXiv 2301.06284):
 *   RGCN  -- the RGCN equation of Section "RGNN Formulation and Operators";
 *   RGAT  -- the single-head RGAT listing of Section "Inter-Operator Level IR"
 *            (per-edge leaky-ReLU attention, edge softmax over the destination's
 *            incoming edges), extended to heads that split the output columns;
 *   HGT   -- the layer of the paper's RGAT/HGT figure (per-node-type K/Q/V/A
 *            linears, per-relation attention and message matrices and prior).
 * The two optimizations of Sections "Compact Tensor Materialization" and
 * "Linear Operator Reordering" are applied inside the calls.
 *
 * Conventions shared by every call
 *   - Row vectors, y = x W: a weight of shape [d_in, d_out] is stored row-major
 *     and maps a row of d_in features to d_out outputs (the typed-linear formula
 *     Y[i,0,j] = sum_k X[i,0,k] W[T[i],k,j] of Section "Inefficiency in Existing
 *     Computation Stack").
 *   - All tensors are dense, row-major, fp32, on the device the graph was
 *     created on.  Pointers named h, W, out, grad_* and ws are DEVICE pointers
 *     owned by the caller; the library never frees them.
 *   - Outputs and gradients are overwritten, never accumulated.
 *   - `stream` is a hipStream_t (NULL = the default stream).  Calls only
 *     enqueue work and return RGNN_OK once it is enqueued; device faults
 *     surface at the next synchronisation or as RGNN_EDEVICE from a later call.
 *   - `ws` is a caller-owned device workspace of at least the size
 *     rgnn_workspace_size() reports for the same arguments.  The library
 *     allocates no device memory inside the layer calls.  Two calls may run
 *     concurrently on different streams only with distinct workspaces.
 *   - On error nothing is enqueued and rgnn_last_error() describes the cause.
 *   - Arithmetic is fp32-accurate.  The forward layers' dense transforms form
 *     each fp32 product from exact three-piece bf16 splits on the bf16 matrix
 *     cores (see rgnn_segment_gemm), so their inputs (features, weights) must be
 *     finite with magnitude below 3.38e38.
 */
#ifndef RGNN_H
#define RGNN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct rgnn_graph rgnn_graph_t;   /* opaque, immutable after creation */

typedef enum {
    RGNN_OK = 0,
    RGNN_EINVAL = -1,        /* bad argument: NULL pointer, size, flag, workspace   */
    RGNN_ERANGE = -2,        /* an id out of range, or a count too large           */
    RGNN_ENOMEM = -3,        /* host or device allocation failed (graph creation)  */
    RGNN_EDEVICE = -4,       /* a HIP runtime call failed                          */
    RGNN_EUNSUPPORTED = -5   /* valid request the library does not implement      */
} rgnn_status;

/* Which side of the aggregation the relation weight W_r is applied on
 * (Section "Linear Operator Reordering"; the choice between materializing
 * per-(src, rel) messages and transforming per-(dst, rel) sums). */
typedef enum {
    RGNN_PLAN_AUTO = 0,              /* pick the plan with fewer modelled HBM bytes */
    RGNN_PLAN_TRANSFORM_FIRST = 1,   /* M = h W_r once per unique (src, rel) pair    */
                                     /* (compact materialization), then gather M     */
    RGNN_PLAN_AGGREGATE_FIRST = 2,   /* gather h, sum per (dst, rel), then apply W_r */
    RGNN_PLAN_TRANSFORM_FIRST_UNREORDERED = 3,
                                     /* RGAT only: transform-first with the          */
                                     /* destination attention term taken from the    */
                                     /* materialized h_v W_r row of every (dst, rel) */
                                     /* segment instead of h_v . (W_r w_dst[r]): the */
                                     /* layer without linear operator reordering     */
    RGNN_PLAN_TRANSFORM_FIRST_ATTMSG = 4
                                     /* RGAT only: transform-first whose materialized */
                                     /* rows hold the message and, after it, the      */
                                     /* heads' source attention terms m . w_src[r]    */
                                     /* (one tensor for attention and message, the    */
                                     /* proposal of Section "Discussion and Future    */
                                     /* Work"; rows padded to 16-byte multiples)      */
} rgnn_plan;

typedef enum {
    RGNN_LAYER_RGCN = 0,
    RGNN_LAYER_RGAT = 1,
    RGNN_LAYER_HGT = 2,
    RGNN_LAYER_RGAT_BACKWARD = 3,
    RGNN_LAYER_SEGMENT_GEMM = 4,
    RGNN_LAYER_RGCN_BACKWARD = 5,
    RGNN_LAYER_HGT_BACKWARD = 6
} rgnn_layer;

enum { RGNN_SOFTMAX_PER_DST = 0, RGNN_SOFTMAX_PER_DST_REL = 1 };

enum {
    RGNN_FLAG_RELU = 1,       /* RGCN: output activation sigma = ReLU (else identity) */
    RGNN_FLAG_RESIDUAL = 2,   /* HGT: add h_t to the output                           */
    RGNN_FLAG_A_LINEAR = 4    /* HGT: apply the per-node-type output linear A         */
};

enum {
    RGNN_GRAPH_HOST_ONLY = 1,    /* build the index on the host only (no device) */
    RGNN_GRAPH_NO_COMPACT = 2    /* one materialized row per edge instead of per unique
                                    (src, rel) pair: the vanilla materialization that
                                    Section "Compact Tensor Materialization" improves on */
};

typedef struct {
    int64_t num_nodes;           /* N                                           */
    int64_t num_edges;           /* E                                           */
    int32_t num_rels;            /* R                                           */
    int32_t num_ntypes;          /* T                                           */
    int64_t num_src_pairs;       /* U_src: unique (src, rel) pairs              */
    int64_t num_dst_segments;    /* U_dst: unique (dst, rel) pairs              */
    int64_t max_in_degree;
    int64_t num_empty_dst;       /* destinations without in-edges               */
    int64_t num_vsegs;           /* (dst, rel) segments after splitting long ones */
    int64_t num_items;           /* traversal work items                         */
    int64_t num_split_dst;       /* destinations spread over several items       */
    int32_t chunk_edges;         /* maximum edges per work item                  */
    int32_t device;              /* HIP device id, -1 for a host-only graph      */
} rgnn_graph_info_t;

/* Index arrays a graph holds, for export and bit-exact checks.  Every array is
 * int32.  In-edges are ordered by (dst, rel, src, original edge id). */
typedef enum {
    RGNN_IDX_DST_ROWPTR = 0,    /* [N+1]     in-edge offsets per destination       */
    RGNN_IDX_IN_SRC = 1,        /* [E]       source of each sorted in-edge         */
    RGNN_IDX_IN_REL = 2,        /* [E]       relation of each sorted in-edge       */
    RGNN_IDX_IN_EID = 3,        /* [E]       original (input) edge id              */
    RGNN_IDX_SEG_PTR = 4,       /* [U_dst+1] edge offsets of the (dst, rel) segments */
    RGNN_IDX_SEG_REL = 5,       /* [U_dst]   relation of each segment              */
    RGNN_IDX_DST_SEGPTR = 6,    /* [N+1]     segment offsets per destination       */
    RGNN_IDX_UNIQ_SRC = 7,      /* [U_src]   source of each unique (rel, src) pair,
                                             pairs in ascending (rel, src) order   */
    RGNN_IDX_UNIQ_REL_PTR = 8,  /* [R+1]     pair offsets per relation             */
    RGNN_IDX_EDGE2UNIQ = 9,     /* [E]       pair index of each sorted in-edge     */
    RGNN_IDX_NTYPE_PERM = 10,   /* [N]       node ids, stable-sorted by node type  */
    RGNN_IDX_NTYPE_PTR = 11,    /* [T+1]     offsets of the node-type segments     */
    RGNN_IDX_OUT_PTR = 12,      /* [N+1]     out-edge offsets per source node      */
    RGNN_IDX_OUT_POS = 13       /* [E]       sorted in-edge position of each out-edge,
                                             out-edges in (src, rel, position) order */
} rgnn_index_kind;

/* ------------------------------------------------------------------ graph */

/* Build the graph index (the preprocessing of Section "Code Generation":
 * COO -> CSR by destination, plus the compact (src, rel) map of Section
 * "Compact Tensor Materialization" and node-type segments for segment MM) and
 * upload it to the current HIP device.
 *   num_nodes N, num_ntypes T >= 1, num_rels R >= 1, num_edges E (0 allowed).
 *   src, dst, rel: HOST int32 arrays [E]; ntype: HOST int32 [N] (NULL = all 0).
 *   The arrays are read during the call only.
 *   flags: RGNN_GRAPH_HOST_ONLY (no device memory; only info/export work),
 *   RGNN_GRAPH_NO_COMPACT (transform-first plans materialize one row per edge;
 *   num_src_pairs = E), or 0.
 *   stream: hipStream_t for the uploads (the call synchronises it).
 * Errors: RGNN_ERANGE for ids outside [0,N) / [0,R) / [0,T) or N, E >= 2^31;
 *         RGNN_EINVAL for NULL arrays or non-positive R, T; RGNN_ENOMEM. */
rgnn_status rgnn_graph_create_coo(int64_t num_nodes, int32_t num_ntypes, int32_t num_rels,
                                  int64_t num_edges, const int32_t *src, const int32_t *dst,
                                  const int32_t *rel, const int32_t *ntype, int32_t flags,
                                  void *stream, rgnn_graph_t **out);

/* Same from CSR by destination: dst_rowptr HOST int64 [N+1] (monotone,
 * rowptr[0] = 0, rowptr[N] = E), col_src and rel HOST int32 [E].  Edge ids are
 * the CSR positions.  RGNN_EINVAL for a malformed row pointer. */
rgnn_status rgnn_graph_create_csr(int64_t num_nodes, int32_t num_ntypes, int32_t num_rels,
                                  const int64_t *dst_rowptr, const int32_t *col_src,
                                  const int32_t *rel, const int32_t *ntype, int32_t flags,
                                  void *stream, rgnn_graph_t **out);

rgnn_status rgnn_graph_destroy(rgnn_graph_t *g);
rgnn_status rgnn_graph_info(const rgnn_graph_t *g, rgnn_graph_info_t *info);

/* Copy one int32 index array into HOST memory `dst` of `bytes` bytes
 * (RGNN_EINVAL if too small).  Device graphs copy from device memory. */
rgnn_status rgnn_graph_export(const rgnn_graph_t *g, int32_t kind, void *dst, size_t bytes);

/* ------------------------------------------------------------------ planning */

/* Workspace bytes a call needs (layer = rgnn_layer; heads 1 for RGCN). */
rgnn_status rgnn_workspace_size(const rgnn_graph_t *g, int32_t layer, int32_t d_in,
                                int32_t d_out, int32_t heads, int32_t plan, size_t *bytes);

/* The plan RGNN_PLAN_AUTO resolves to, with the modelled HBM bytes of both
 * plans (either pointer may be NULL).  The model counts each gathered row once
 * per edge, each materialized row once per write and read. */
rgnn_status rgnn_select_plan(const rgnn_graph_t *g, int32_t layer, int32_t d_in, int32_t d_out,
                             int32_t heads, int32_t *plan, double *bytes_transform_first,
                             double *bytes_aggregate_first);

/* ------------------------------------------------------------------ layers */

/* RGCN layer (the paper's RGCN equation):
 *   out_v = act( h_v W0 + sum_r sum_{u in N_v^r} h_u W_r / c_{v,r} )
 * c_{v,r} = number of in-edges of v with relation r (duplicates counted).
 *   h [N, d_in], W [R, d_in, d_out], W0 [d_in, d_out] or NULL (no self-loop),
 *   out [N, d_out].  flags: RGNN_FLAG_RELU.  d_in, d_out in {64, 128}, or
 *   d_in = d_out = 32. */
rgnn_status rgcn_forward(const rgnn_graph_t *g, const float *h, const float *W, const float *W0,
                         int32_t d_in, int32_t d_out, int32_t flags, int32_t plan, float *out,
                         void *ws, size_t ws_bytes, void *stream);

/* RGAT layer (the paper's RGAT listing).  Per in-edge e = (u -> v, r), head k
 * owning columns [k*d_out/H, (k+1)*d_out/H):
 *   y_e,k = (h_u W_r)_k . w_src[r]_k + (h_v W_r)_k . w_dst[r]_k
 *   alpha_e,k = softmax over the in-edges of v of leakyrelu(y_e,k)
 *   out_v[k-cols] = sum_e alpha_e,k (h_u W_r)[k-cols]      (0 without in-edges)
 *   h [N, d_in], W [R, d_in, d_out], w_src, w_dst [R, d_out], out [N, d_out].
 *   saved [N, heads, 2] or NULL: per destination and head the softmax maximum
 *   and denominator (max z, sum exp(z - max)), 0 for empty rows; needed by
 *   rgat_backward.
 *   softmax_scope RGNN_SOFTMAX_PER_DST_REL takes the softmax over the in-edges
 *   of v with relation r instead (each relation's messages are normalised on
 *   their own; out_v sums the relations): it runs the aggregate-first plan
 *   (d_in == d_out; size the workspace for RGNN_PLAN_AGGREGATE_FIRST with the
 *   head count) and returns RGNN_EUNSUPPORTED for the transform-first plans;
 *   saved is then [num_dst_segments, heads, 2], the (max, sum) of each
 *   (dst, rel) segment in (dst, rel) order, or NULL.
 *   d_in, d_out in {64, 128}, or d_in = d_out = 32; d_out / heads a multiple of 16.
 *   Aggregate-first with several heads (either softmax) runs one pass per
 *   head over the weights and attention vectors with the other heads'
 *   columns zeroed, the outputs summed: exact, at the cost of one pass per
 *   head, so RGNN_PLAN_AUTO picks transform-first for several heads. */
rgnn_status rgat_forward(const rgnn_graph_t *g, const float *h, const float *W,
                         const float *w_src, const float *w_dst, int32_t d_in, int32_t d_out,
                         int32_t heads, float neg_slope, int32_t softmax_scope, int32_t plan,
                         float *out, float *saved, void *ws, size_t ws_bytes, void *stream);

/* rgat_forward without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, serving loops,
 * harnesses that forbid allocation).  Arguments, results and errors as in
 * rgat_forward; the workspace lives in a static device array of 64 MiB that
 * every GPU the library runs on holds from the first call until the process
 * ends.  RGNN_ERANGE when rgnn_workspace_size() for these arguments exceeds
 * 64 MiB (for one head at d = 64 that is roughly 2.4e5 (dst, rel) segments).
 * The call allocates nothing.  Calls that overlap on one GPU share the array
 * and race: serialise them (one stream, or events between streams). */
rgnn_status rgat_forward_noalloc(const rgnn_graph_t *g, const float *h, const float *W,
                                 const float *w_src, const float *w_dst, int32_t d_in, int32_t d_out,
                                 int32_t heads, float neg_slope, int32_t softmax_scope, int32_t plan,
                                 float *out, float *saved, void *stream);

/* HGT layer.  With K_n = h_n Wk[tau(n)], Q_n = h_n Wq[tau(n)],
 * V_n = h_n Wv[tau(n)] split into `heads` blocks of dk = d / heads, per in-edge
 * e = (s -> t, r) and head i:
 *   a_e,i = (K_s,i Watt[r,i]) . Q_t,i * mu[r] * att_scale
 *   alpha_e,i = softmax over the in-edges of t;   msg_e,i = V_s,i Wmsg[r,i]
 *   agg_t = concat_i sum_e alpha_e,i msg_e,i
 *   out_t = agg_t Wa[tau(t)] (RGNN_FLAG_A_LINEAR, else agg_t) + h_t (RGNN_FLAG_RESIDUAL)
 *   h [N, d]; Wk, Wq, Wv, Wa [T, d, d]; Watt, Wmsg [R, heads, dk, dk]; mu [R].
 *   saved: NULL, or [N, heads, 2] written with each destination's softmax
 *   maximum and sum per head ((0, 0) for a destination without in-edges), which
 *   hgt_backward takes to skip recomputing the forward traversal.
 *   d in {32, 64, 128}, heads in {1, 2, 4, 8} with dk = d / heads >= 16. */
rgnn_status hgt_forward(const rgnn_graph_t *g, const float *h, const float *Wk, const float *Wq,
                        const float *Wv, const float *Wa, const float *Watt, const float *Wmsg,
                        const float *mu, int32_t d, int32_t heads, float att_scale, int32_t flags,
                        float *out, float *saved, void *ws, size_t ws_bytes, void *stream);

/* RGAT backward (Section "Backward Propagation") for the forward above: given
 * grad_out = dL/dout [N, d_out] and the forward's `saved`, writes dL/dh
 * [N, d_in], dL/dW [R, d_in, d_out], dL/dw_src and dL/dw_dst [R, d_out].
 * softmax_scope as in the forward: RGNN_SOFTMAX_PER_DST with saved
 * [N, heads, 2]; RGNN_SOFTMAX_PER_DST_REL with the forward's per-segment
 * saved [num_dst_segments, heads, 2].  d_in = d_out in {32, 64, 128}, d_out / heads
 * a multiple of 16.
 * Several heads run as one pass per head over the weights, attention vectors
 * and grad_out with the other heads' columns zeroed (each head's logits,
 * softmax and messages read only its own columns, so the per-head gradients
 * add up to the exact ones); the cost grows with the heads.  Workspace:
 * rgnn_workspace_size(RGNN_LAYER_RGAT_BACKWARD, d_in, d_out, heads). */
rgnn_status rgat_backward(const rgnn_graph_t *g, const float *h, const float *W,
                          const float *w_src, const float *w_dst, int32_t d_in, int32_t d_out,
                          int32_t heads, float neg_slope, int32_t softmax_scope,
                          const float *saved, const float *grad_out, float *grad_h,
                          float *grad_W, float *grad_w_src, float *grad_w_dst, void *ws,
                          size_t ws_bytes, void *stream);

/* RGCN backward for the RGCN layer above: the chain rule of the RGCN
 * equation (Section "Backward Propagation" derives the backward from the
 * forward).  With P the pre-activation and Gp = grad_out * act'(P):
 *   dW_r = sum over in-edges (u -> v, r) of h_u^T Gp_v / c_{v,r}
 *   dh_u = sum over out-edges (u -> v, r) of Gp_v W_r^T / c_{v,r}  +  Gp_u W0^T
 *   dW0  = sum_v h_v^T Gp_v
 *   h [N, d_in], W [R, d_in, d_out], W0 [d_in, d_out] or NULL (as in the
 *   forward), flags as in the forward (RGNN_FLAG_RELU: out = the forward's
 *   output [N, d_out], which gives act' = [out > 0]; otherwise out may be NULL),
 *   grad_out [N, d_out]; writes grad_h [N, d_in], grad_W [R, d_in, d_out] and,
 *   when W0 and grad_W0 are both given, grad_W0 [d_in, d_out].
 *   d_in = d_out in {32, 64, 128}.  Workspace: rgnn_workspace_size(RGNN_LAYER_RGCN_BACKWARD).
 *   Results are reproducible except the rows of sources with more than 64
 *   out-edges, which are summed with float atomics. */
rgnn_status rgcn_backward(const rgnn_graph_t *g, const float *h, const float *W, const float *W0,
                          int32_t d_in, int32_t d_out, int32_t flags, const float *out,
                          const float *grad_out, float *grad_h, float *grad_W, float *grad_W0,
                          void *ws, size_t ws_bytes, void *stream);

/* HGT backward for the HGT layer above: the chain rule of its definition
 * (Section "Backward Propagation" derives the backward from the forward) for
 * the loss L = sum(out * grad_out).  Arguments as in hgt_forward plus
 * grad_out [N, d]; writes grad_h [N, d], grad_Wk, grad_Wq, grad_Wv [T, d, d],
 * grad_Wa [T, d, d] (with RGNN_FLAG_A_LINEAR; otherwise not written, may be
 * NULL), grad_Watt, grad_Wmsg [R, heads, dk, dk] and grad_mu [R].  saved: the
 * forward's softmax statistics [N, heads, 2] from hgt_forward with the same
 * inputs, or NULL, in which case the forward traversal is recomputed inside
 * the call (with saved given, the aggregate that grad_Wa needs is rebuilt from
 * the backward's own per-segment sums instead).  d in {32, 64, 128},
 * d / heads >= 16.  Workspace:
 * rgnn_workspace_size(RGNN_LAYER_HGT_BACKWARD, d, d, heads).  Results are
 * reproducible except the K|V gradient rows of sources with more than 64
 * out-edges, which are summed with float atomics. */
rgnn_status hgt_backward(const rgnn_graph_t *g, const float *h, const float *Wk, const float *Wq,
                         const float *Wv, const float *Wa, const float *Watt, const float *Wmsg,
                         const float *mu, int32_t d, int32_t heads, float att_scale, int32_t flags,
                         const float *grad_out, const float *saved, float *grad_h, float *grad_Wk,
                         float *grad_Wq, float *grad_Wv, float *grad_Wa, float *grad_Watt,
                         float *grad_Wmsg, float *grad_mu, void *ws, size_t ws_bytes, void *stream);

/* Segment MM: the GEMM template of Section "The GEMM Template and the
 * Traversal Template", Y[S] = X[G] x W[T]:
 *   for every row i in [0, M): Y[scatter[i]] = X[gather[i]] W[t(i)]
 * where t(i) is the segment of i given by type_ptr (HOST int64 [T+1],
 * type_ptr[0] = 0, type_ptr[T] = M, rows of one type contiguous).
 *   X [*, ldx >= K], W [T, K, Nc], Y [*, ldy >= Nc]; gather, scatter: DEVICE
 *   int32 [M] or NULL for the identity.  K in {64, 128}, Nc in {64, 128}, or
 *   K = Nc = 32.
 *   Rows written twice through `scatter` race; the caller avoids that.
 *   Arithmetic: fp32 inputs and outputs with fp32 accuracy.  For K, Nc in
 *   {64, 128} each product is formed from an exact split of both operands into
 *   three bf16 pieces on the bf16 matrix cores (six piece products accumulated
 *   in fp32; the dropped ones are below 2^-23 |x||w|); X and W must then be
 *   finite with magnitude below 3.38e38.  The forward layers use the same
 *   products. */
rgnn_status rgnn_segment_gemm(const float *X, int64_t ldx, const int32_t *gather,
                              const int64_t *type_ptr, int32_t num_types, const float *W,
                              int32_t K, int32_t Nc, float *Y, int64_t ldy,
                              const int32_t *scatter, void *ws, size_t ws_bytes, void *stream);
rgnn_status rgnn_segment_gemm_workspace_size(int64_t M, int32_t num_types, size_t *bytes);

/* ------------------------------------------------------------------ profiling */

/* With profiling on, every kernel launch of the library is bracketed by two
 * hipEvents recorded on the launch's stream.  rgnn_profile_read synchronises
 * those events and returns, for kernel index i in [0, *count), its name, the
 * number of launches and their summed duration in milliseconds.
 * rgnn_profile_reset drops all records. */
rgnn_status rgnn_profile_enable(int32_t on);
rgnn_status rgnn_profile_count(int32_t *count);
rgnn_status rgnn_profile_read(int32_t i, char *name, size_t name_bytes, int64_t *launches,
                              double *total_ms);
rgnn_status rgnn_profile_reset(void);

/* Thread-local description of the last error of this thread ("" if none). */
const char *rgnn_last_error(void);

/* Library version string. */
const char *rgnn_version(void);

#ifdef __cplusplus
}
#endif
#endif /* RGNN_H */
