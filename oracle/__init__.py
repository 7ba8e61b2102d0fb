"""fp64 CPU oracle for the RGCN / RGAT / HGT layers and the RGAT backward pass.

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the benchmark's
CPU-baseline leg are the only callers.  Nothing here imports, loads or shares
code with the GPU library (`paper_2301_06284_amd`), and the GPU library never
imports this package.

Two parts:
  * `graph_index`  -- the integer preprocessing the GPU library must reproduce
    bit for bit (CSR by destination, (dst, rel) segments, the compact
    (src, rel) map of compact materialization, node-type segments), written
    with numpy sorts in the order the definitions fix;
  * `rgcn_forward`, `rgat_forward`, `hgt_forward`, `rgat_backward` -- thin
    ctypes wrappers over `rgnn_oracle.c`, the edge-by-edge fp64 evaluation of
    the layer equations.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "rgnn_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile the C oracle with gcc (-O2, OpenMP, no fp contraction, no fast-math)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-fPIC",
                               "-shared", "-std=c11", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        _lib = ctypes.CDLL(_LIB)
        i64, i32, vp, f64 = ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p, ctypes.c_double
        _lib.oracle_rgcn_forward.argtypes = [i64, i64, i32, i32, i32, vp, vp, vp, vp, vp, vp,
                                             i32, i64, vp, vp]
        _lib.oracle_rgat_forward.argtypes = [i64, i64, i32, i32, i32, i32, vp, vp, vp, vp, vp,
                                             vp, vp, f64, i32, i64, vp, vp, vp, vp, vp]
        _lib.oracle_hgt_forward.argtypes = [i64, i64, i32, i32, i32, i32, vp, vp, vp, vp, vp,
                                            vp, vp, vp, vp, vp, vp, vp, f64, i32, i32, i64, vp,
                                            vp]
        _lib.oracle_rgat_backward.argtypes = [i64, i64, i32, i32, i32, i32, vp, vp, vp, vp, vp,
                                              vp, vp, f64, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp]
        _lib.oracle_rgcn_backward.argtypes = [i64, i64, i32, i32, i32, vp, vp, vp, vp, vp, vp,
                                              i32, vp, vp, vp, vp, vp, vp]
        _lib.oracle_hgt_backward.argtypes = [i64, i64, i32, i32, i32, i32, vp, vp, vp, vp, vp,
                                             vp, vp, vp, vp, vp, vp, vp, f64, i32, i32, vp, vp,
                                             vp, vp, vp, vp, vp, vp, vp, vp, vp]
        for f in ("oracle_rgcn_forward", "oracle_rgat_forward", "oracle_hgt_forward",
                  "oracle_rgat_backward", "oracle_rgcn_backward", "oracle_hgt_backward",
                  "oracle_num_threads"):
            getattr(_lib, f).restype = ctypes.c_int
    return _lib


def num_threads() -> int:
    return int(_load().oracle_num_threads())


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def _f32(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.float32)


def _sel(sel, N):
    if sel is None:
        return None, N
    sel = _i32(sel)
    return sel, len(sel)


def _check(rc, name):
    if rc != 0:
        raise ValueError(f"{name}: oracle returned {rc}")


# --------------------------------------------------------------------------
# Layers
# --------------------------------------------------------------------------
def rgcn_forward(g, h, W, W0=None, relu=False, sel=None):
    """RGCN equation: out_v = act(h_v W0 + sum_r sum_{u in N_v^r} h_u W_r / c_{v,r})."""
    h, W, W0 = _f32(h), _f32(W), _f32(W0)
    src, dst, rel = _i32(g["src"]), _i32(g["dst"]), _i32(g["rel"])
    sel, n = _sel(sel, g["N"])
    d_in, d_out = W.shape[1], W.shape[2]
    out = np.zeros((n, d_out), np.float64)
    rc = _load().oracle_rgcn_forward(g["N"], g["E"], g["R"], d_in, d_out, _p(src), _p(dst),
                                     _p(rel), _p(h), _p(W), _p(W0), int(relu), n, _p(sel),
                                     _p(out))
    _check(rc, "rgcn_forward")
    return out


def rgat_forward(g, h, W, w_src, w_dst, heads=1, neg_slope=0.2, scope=0, sel=None,
                 want_stats=False, want_alpha=False):
    """RGAT listing: leaky-ReLU attention on m_e . w_src + t_e . w_dst, edge softmax
    over the destination's in-edges (scope 0) or its in-edges of one relation
    (scope 1), attention-weighted sum of the messages m_e = h_u W_r."""
    h, W, w_src, w_dst = _f32(h), _f32(W), _f32(w_src), _f32(w_dst)
    src, dst, rel = _i32(g["src"]), _i32(g["dst"]), _i32(g["rel"])
    sel, n = _sel(sel, g["N"])
    d_in, d_out = W.shape[1], W.shape[2]
    out = np.zeros((n, d_out), np.float64)
    smax = np.zeros((n, heads), np.float64) if want_stats else None
    ssum = np.zeros((n, heads), np.float64) if want_stats else None
    alpha = np.full((g["E"], heads), np.nan, np.float64) if want_alpha else None
    rc = _load().oracle_rgat_forward(g["N"], g["E"], g["R"], d_in, d_out, heads, _p(src),
                                     _p(dst), _p(rel), _p(h), _p(W), _p(w_src), _p(w_dst),
                                     float(neg_slope), int(scope), n, _p(sel), _p(out),
                                     _p(smax), _p(ssum), _p(alpha))
    _check(rc, "rgat_forward")
    res = [out]
    if want_stats:
        res += [smax, ssum]
    if want_alpha:
        res.append(alpha)
    return res[0] if len(res) == 1 else tuple(res)


def hgt_forward(g, h, Wk, Wq, Wv, Wa, Watt, Wmsg, mu, heads, att_scale=None,
                residual=True, a_linear=True, sel=None):
    """HGT layer: per-node-type K/Q/V, per-relation W_att / W_msg and prior mu,
    per-head edge softmax over all in-edges, A-linear and residual."""
    h = _f32(h)
    Wk, Wq, Wv, Wa, Watt, Wmsg, mu = map(_f32, (Wk, Wq, Wv, Wa, Watt, Wmsg, mu))
    src, dst, rel, ntype = (_i32(g[k]) for k in ("src", "dst", "rel", "ntype"))
    sel, n = _sel(sel, g["N"])
    d = h.shape[1]
    if att_scale is None:
        att_scale = 1.0 / np.sqrt(d // heads)
    out = np.zeros((n, d), np.float64)
    rc = _load().oracle_hgt_forward(g["N"], g["E"], g["R"], g["T"], d, heads, _p(src), _p(dst),
                                    _p(rel), _p(ntype), _p(h), _p(Wk), _p(Wq), _p(Wv), _p(Wa),
                                    _p(Watt), _p(Wmsg), _p(mu), float(att_scale), int(residual),
                                    int(a_linear), n, _p(sel), _p(out))
    _check(rc, "hgt_forward")
    return out


def rgat_backward(g, h, W, w_src, w_dst, grad_out, heads=1, neg_slope=0.2, scope=0,
                  node_mask=None, rel_mask=None, kink_flip=None, want_Y=False):
    """Gradients of L = sum(out * grad_out) of the RGAT layer with the softmax
    over each destination's in-edges (scope 0) or over its in-edges of one
    relation (scope 1).  Returns (dh, dW, dw_src, dw_dst); entries outside the
    masks are zero.  kink_flip: None or a boolean [E, heads] array; where set,
    the leaky ReLU's derivative is taken from the other side of its kink (the
    derivative at y = 0 is one-sided: either side is a correct result where y
    lies within rounding of zero, see rgat_preactivations).  want_Y: also
    return Y = dL/dy [E, heads] (NaN for edges whose destination the masks
    left unvisited)."""
    h, W, w_src, w_dst, G = map(_f32, (h, W, w_src, w_dst, grad_out))
    src, dst, rel = _i32(g["src"]), _i32(g["dst"]), _i32(g["rel"])
    N, R = g["N"], g["R"]
    d_in, d_out = W.shape[1], W.shape[2]
    nm = None if node_mask is None else np.ascontiguousarray(node_mask, np.uint8)
    rm = None if rel_mask is None else np.ascontiguousarray(rel_mask, np.uint8)
    kf = None
    if kink_flip is not None:
        kf = np.ascontiguousarray(np.asarray(kink_flip, bool).reshape(g["E"], heads), np.uint8)
    dh = np.zeros((N, d_in)); dW = np.zeros((R, d_in, d_out))
    dws = np.zeros((R, d_out)); dwd = np.zeros((R, d_out))
    Y = np.empty((g["E"], heads)) if want_Y else None
    rc = _load().oracle_rgat_backward(N, g["E"], R, d_in, d_out, heads, _p(src), _p(dst),
                                      _p(rel), _p(h), _p(W), _p(w_src), _p(w_dst),
                                      float(neg_slope), int(scope), _p(G), _p(nm), _p(rm), _p(kf), _p(dh),
                                      _p(dW), _p(dws), _p(dwd), _p(Y))
    _check(rc, "rgat_backward")
    return (dh, dW, dws, dwd, Y) if want_Y else (dh, dW, dws, dwd)


def rgat_preactivations(g, h, W, w_src, w_dst, heads=1, chunk=1 << 20):
    """The RGAT attention logits before the leaky ReLU, edge by edge (Listing 1,
    Section 3.2.1): y_e,k = (h_u W_r)[k] . w_src[r][k] + (h_v W_r)[k] . w_dst[r][k]
    over head k's columns, in fp64.  Also returns each logit's rounding scale,
    sum_j |(h_u W_r)_j w_src_j| + |(h_v W_r)_j w_dst_j| over the same columns:
    an fp32 evaluation can put y on either side of zero where |y| is within a
    small multiple of 2^-24 of that scale.  Returns (y, scale), both [E, heads]."""
    src, dst, rel = (np.asarray(g[k]) for k in ("src", "dst", "rel"))
    E = len(src)
    h = np.asarray(h, np.float64)
    d_out = W.shape[2]
    dk = d_out // heads
    y = np.zeros((E, heads)); scale = np.zeros((E, heads))
    for r in range(W.shape[0]):
        Wr = np.asarray(W[r], np.float64)
        ws, wd = np.asarray(w_src[r], np.float64), np.asarray(w_dst[r], np.float64)
        er = np.nonzero(rel == r)[0]
        for c0 in range(0, len(er), chunk):
            e = er[c0:c0 + chunk]
            ps, pd = (h[src[e]] @ Wr) * ws, (h[dst[e]] @ Wr) * wd
            for k in range(heads):
                cols = slice(k * dk, (k + 1) * dk)
                y[e, k] = ps[:, cols].sum(axis=1) + pd[:, cols].sum(axis=1)
                scale[e, k] = np.abs(ps[:, cols]).sum(axis=1) + np.abs(pd[:, cols]).sum(axis=1)
    return y, scale


def rgcn_backward(g, h, W, W0, grad_out, relu=False, node_mask=None, rel_mask=None,
                  want_dW0=True):
    """Gradients of L = sum(out * grad_out) of the RGCN layer (chain rule on the
    RGCN equation).  Returns (dh, dW, dW0); dW0 is None without W0 or when not
    wanted; entries outside the masks are zero."""
    h, W, G = map(_f32, (h, W, grad_out))
    W0 = None if W0 is None else _f32(W0)
    src, dst, rel = _i32(g["src"]), _i32(g["dst"]), _i32(g["rel"])
    N, R = g["N"], g["R"]
    d_in, d_out = W.shape[1], W.shape[2]
    nm = None if node_mask is None else np.ascontiguousarray(node_mask, np.uint8)
    rm = None if rel_mask is None else np.ascontiguousarray(rel_mask, np.uint8)
    dh = np.zeros((N, d_in)); dW = np.zeros((R, d_in, d_out))
    dW0 = np.zeros((d_in, d_out)) if (W0 is not None and want_dW0) else None
    rc = _load().oracle_rgcn_backward(N, g["E"], R, d_in, d_out, _p(src), _p(dst), _p(rel),
                                      _p(h), _p(W), _p(W0), int(bool(relu)), _p(G), _p(nm),
                                      _p(rm), _p(dh), _p(dW), _p(dW0))
    _check(rc, "rgcn_backward")
    return dh, dW, dW0


def hgt_backward(g, h, Wk, Wq, Wv, Wa, Watt, Wmsg, mu, grad_out, heads, att_scale=None,
                 residual=True, a_linear=True, node_mask=None, rel_mask=None):
    """Gradients of L = sum(out * grad_out) of the HGT layer (chain rule of its
    definition).  Returns a dict with dh, dWk, dWq, dWv, dWa (None without the
    output linear), dWatt, dWmsg, dmu.  node_mask / rel_mask (uint8 [N] / [R],
    optional): dh only for the flagged nodes, dWatt / dWmsg / dmu only for the
    flagged relations; with either mask the node-type weight gradients are
    left zero."""
    h, Wk, Wq, Wv, Wa, Watt, Wmsg, mu, G = map(_f32, (h, Wk, Wq, Wv, Wa, Watt, Wmsg, mu, grad_out))
    src, dst, rel, nt = _i32(g["src"]), _i32(g["dst"]), _i32(g["rel"]), _i32(g["ntype"])
    N, R, T = g["N"], g["R"], g["T"]
    d = h.shape[1]
    dk = d // heads
    if att_scale is None:
        att_scale = 1.0 / np.sqrt(dk)
    out = dict(dh=np.zeros((N, d)), dWk=np.zeros((T, d, d)), dWq=np.zeros((T, d, d)),
               dWv=np.zeros((T, d, d)), dWa=np.zeros((T, d, d)) if a_linear else None,
               dWatt=np.zeros((R, heads, dk, dk)), dWmsg=np.zeros((R, heads, dk, dk)),
               dmu=np.zeros(R))
    nm = None if node_mask is None else np.ascontiguousarray(node_mask, np.uint8)
    rm = None if rel_mask is None else np.ascontiguousarray(rel_mask, np.uint8)
    rc = _load().oracle_hgt_backward(N, g["E"], R, T, d, heads, _p(src), _p(dst), _p(rel), _p(nt),
                                     _p(h), _p(Wk), _p(Wq), _p(Wv), _p(Wa), _p(Watt), _p(Wmsg),
                                     _p(mu), float(att_scale), int(bool(residual)),
                                     int(bool(a_linear)), _p(G), _p(nm), _p(rm), _p(out["dh"]), _p(out["dWk"]),
                                     _p(out["dWq"]), _p(out["dWv"]), _p(out["dWa"]),
                                     _p(out["dWatt"]), _p(out["dWmsg"]), _p(out["dmu"]))
    _check(rc, "hgt_backward")
    return out


# --------------------------------------------------------------------------
# Integer preprocessing (compact materialization map, CSR, segments)
# --------------------------------------------------------------------------
def graph_index(g) -> dict:
    """The index arrays the GPU library exports, in the order they are defined:

    * in-edges sorted by (dst, rel, src, original edge id):
        dst_rowptr [N+1], in_src / in_rel / in_eid [E]
    * (dst, rel) segments of that order: seg_ptr [U_dst+1] (edge offsets),
        seg_rel [U_dst], dst_segptr [N+1] (segment offsets per destination)
    * compact materialization map: the unique (rel, src) pairs in ascending
        (rel, src) order: uniq_src [U_src], uniq_rel_ptr [R+1]; and
        edge2uniq [E], the pair index of each edge in the sorted in-edge order
    * node-type segments: ntype_perm [N] (node ids, stable by type),
        ntype_ptr [T+1]
    * out-edges: out_ptr [N+1] (out-edge offsets per source) and out_pos [E],
        the sorted in-edge positions ordered by (src, rel, position)
    All arrays are int64 here; only their values are compared.
    """
    N, E, R, T = g["N"], g["E"], g["R"], g["T"]
    src = np.asarray(g["src"], np.int64); dst = np.asarray(g["dst"], np.int64)
    rel = np.asarray(g["rel"], np.int64); ntype = np.asarray(g["ntype"], np.int64)
    eid = np.arange(E, dtype=np.int64)
    order = np.lexsort((eid, src, rel, dst))
    in_src, in_rel, in_dst = src[order], rel[order], dst[order]
    dst_rowptr = np.zeros(N + 1, np.int64)
    np.cumsum(np.bincount(dst, minlength=N), out=dst_rowptr[1:])
    if E:
        key = in_dst * R + in_rel
        starts = np.flatnonzero(np.r_[True, key[1:] != key[:-1]])
    else:
        starts = np.zeros(0, np.int64)
    seg_ptr = np.r_[starts, E].astype(np.int64)
    seg_rel = in_rel[starts] if E else np.zeros(0, np.int64)
    seg_dst = in_dst[starts] if E else np.zeros(0, np.int64)
    dst_segptr = np.zeros(N + 1, np.int64)
    np.cumsum(np.bincount(seg_dst, minlength=N), out=dst_segptr[1:])
    pair = rel * N + src
    upair, inv = np.unique(pair, return_inverse=True)
    uniq_src = upair % N if N else upair
    uniq_rel = upair // N if N else upair
    uniq_rel_ptr = np.zeros(R + 1, np.int64)
    np.cumsum(np.bincount(uniq_rel, minlength=R), out=uniq_rel_ptr[1:])
    edge2uniq = inv.reshape(-1)[order]
    ntype_perm = np.argsort(ntype, kind="stable").astype(np.int64)
    ntype_ptr = np.zeros(T + 1, np.int64)
    np.cumsum(np.bincount(ntype, minlength=T), out=ntype_ptr[1:])
    position = np.arange(E, dtype=np.int64)
    out_pos = np.lexsort((position, in_rel, in_src))
    out_ptr = np.zeros(N + 1, np.int64)
    np.cumsum(np.bincount(src, minlength=N), out=out_ptr[1:])
    return dict(out_ptr=out_ptr, out_pos=out_pos,dst_rowptr=dst_rowptr, in_src=in_src, in_rel=in_rel, in_eid=order,
                seg_ptr=seg_ptr, seg_rel=seg_rel, dst_segptr=dst_segptr,
                uniq_src=uniq_src, uniq_rel_ptr=uniq_rel_ptr, edge2uniq=edge2uniq,
                ntype_perm=ntype_perm, ntype_ptr=ntype_ptr,
                U_src=int(len(upair)), U_dst=int(len(starts)))
