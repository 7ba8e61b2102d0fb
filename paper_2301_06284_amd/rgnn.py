"""ctypes binding of librgnn.so (declared in include/rgnn.h).

Argument marshalling only: every computation runs inside the HIP library.
Tensors are torch tensors on the GPU (PyTorch provides device memory and the
stream); index arrays for graph creation are host numpy arrays.  If the built
library is missing, importing this module raises -- there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "librgnn.so")

OK, EINVAL, ERANGE, ENOMEM, EDEVICE, EUNSUPPORTED = 0, -1, -2, -3, -4, -5
PLAN_AUTO, PLAN_TRANSFORM_FIRST, PLAN_AGGREGATE_FIRST = 0, 1, 2
PLAN_TRANSFORM_FIRST_UNREORDERED = 3
PLAN_TRANSFORM_FIRST_ATTMSG = 4
LAYER_RGCN, LAYER_RGAT, LAYER_HGT, LAYER_RGAT_BACKWARD, LAYER_SEGMENT_GEMM = 0, 1, 2, 3, 4
LAYER_RGCN_BACKWARD, LAYER_HGT_BACKWARD = 5, 6
SOFTMAX_PER_DST, SOFTMAX_PER_DST_REL = 0, 1
FLAG_RELU, FLAG_RESIDUAL, FLAG_A_LINEAR = 1, 2, 4
GRAPH_HOST_ONLY, GRAPH_NO_COMPACT = 1, 2

INDEX_KINDS = {
    "dst_rowptr": 0, "in_src": 1, "in_rel": 2, "in_eid": 3, "seg_ptr": 4, "seg_rel": 5,
    "dst_segptr": 6, "uniq_src": 7, "uniq_rel_ptr": 8, "edge2uniq": 9, "ntype_perm": 10,
    "ntype_ptr": 11, "out_ptr": 12, "out_pos": 13,
}

EXPORTED = [
    "rgnn_graph_create_coo", "rgnn_graph_create_csr", "rgnn_graph_destroy", "rgnn_graph_info",
    "rgnn_graph_export", "rgnn_workspace_size", "rgnn_select_plan", "rgcn_forward",
    "rgat_forward", "rgat_forward_noalloc", "hgt_forward", "rgat_backward", "rgcn_backward", "hgt_backward",
    "rgnn_segment_gemm",
    "rgnn_segment_gemm_workspace_size", "rgnn_profile_enable", "rgnn_profile_count",
    "rgnn_profile_read", "rgnn_profile_reset", "rgnn_last_error", "rgnn_version",
]


class RgnnError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"librgnn status {status}: {msg}")
        self.status = status


class GraphInfo(ctypes.Structure):
    _fields_ = [("num_nodes", ctypes.c_int64), ("num_edges", ctypes.c_int64),
                ("num_rels", ctypes.c_int32), ("num_ntypes", ctypes.c_int32),
                ("num_src_pairs", ctypes.c_int64), ("num_dst_segments", ctypes.c_int64),
                ("max_in_degree", ctypes.c_int64), ("num_empty_dst", ctypes.c_int64),
                ("num_vsegs", ctypes.c_int64), ("num_items", ctypes.c_int64),
                ("num_split_dst", ctypes.c_int64), ("chunk_edges", ctypes.c_int32),
                ("device", ctypes.c_int32)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                          "(there is no CPU fallback)")
    lib = ctypes.CDLL(LIB_PATH)
    i32, i64, vp, f32, sz = ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p, ctypes.c_float, ctypes.c_size_t
    P = ctypes.POINTER
    sig = {
        "rgnn_graph_create_coo": [i64, i32, i32, i64, vp, vp, vp, vp, i32, vp, P(vp)],
        "rgnn_graph_create_csr": [i64, i32, i32, vp, vp, vp, vp, i32, vp, P(vp)],
        "rgnn_graph_destroy": [vp],
        "rgnn_graph_info": [vp, P(GraphInfo)],
        "rgnn_graph_export": [vp, i32, vp, sz],
        "rgnn_workspace_size": [vp, i32, i32, i32, i32, i32, P(sz)],
        "rgnn_select_plan": [vp, i32, i32, i32, i32, P(i32), P(ctypes.c_double), P(ctypes.c_double)],
        "rgcn_forward": [vp, vp, vp, vp, i32, i32, i32, i32, vp, vp, sz, vp],
        "rgat_forward": [vp, vp, vp, vp, vp, i32, i32, i32, f32, i32, i32, vp, vp, vp, sz, vp],
        "rgat_forward_noalloc": [vp, vp, vp, vp, vp, i32, i32, i32, f32, i32, i32, vp, vp, vp],
        "hgt_forward": [vp, vp, vp, vp, vp, vp, vp, vp, vp, i32, i32, f32, i32, vp, vp, vp, sz, vp],
        "rgat_backward": [vp, vp, vp, vp, vp, i32, i32, i32, f32, i32, vp, vp, vp, vp, vp, vp, vp, sz, vp],
        "rgcn_backward": [vp, vp, vp, vp, i32, i32, i32, vp, vp, vp, vp, vp, vp, sz, vp],
        "hgt_backward": [vp, vp, vp, vp, vp, vp, vp, vp, vp, i32, i32, f32, i32, vp, vp, vp, vp, vp, vp, vp,
                         vp, vp, vp, vp, sz, vp],
        "rgnn_segment_gemm": [vp, i64, vp, vp, i32, vp, i32, i32, vp, i64, vp, vp, sz, vp],
        "rgnn_segment_gemm_workspace_size": [i64, i32, P(sz)],
        "rgnn_profile_enable": [i32],
        "rgnn_profile_count": [P(i32)],
        "rgnn_profile_read": [i32, ctypes.c_char_p, sz, P(i64), P(ctypes.c_double)],
        "rgnn_profile_reset": [],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = ctypes.c_int
    lib.rgnn_last_error.restype = ctypes.c_char_p
    lib.rgnn_last_error.argtypes = []
    lib.rgnn_version.restype = ctypes.c_char_p
    lib.rgnn_version.argtypes = []
    return lib


_lib = _load()


def lib():
    return _lib


def _check(st: int):
    if st != OK:
        raise RgnnError(st, _lib.rgnn_last_error().decode())


def _ptr(t):
    """Device pointer of a torch tensor (None -> NULL)."""
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors passed to librgnn must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _host(a, dtype):
    return None if a is None else np.ascontiguousarray(a, dtype=dtype)


def _np_ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _stream(stream):
    if stream is None:
        import torch
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return ctypes.c_void_p(stream)
    return ctypes.c_void_p(stream.cuda_stream)


class Graph:
    """A graph index built by rgnn_graph_create_{coo,csr}."""

    def __init__(self, handle):
        self._h = handle

    @classmethod
    def from_coo(cls, N, T, R, src, dst, rel, ntype=None, host_only=False, stream=None,
                 compact=True):
        src, dst, rel = _host(src, np.int32), _host(dst, np.int32), _host(rel, np.int32)
        ntype = _host(ntype, np.int32)
        h = ctypes.c_void_p()
        flags = (GRAPH_HOST_ONLY if host_only else 0) | (0 if compact else GRAPH_NO_COMPACT)
        st = _lib.rgnn_graph_create_coo(int(N), int(T), int(R), len(src), _np_ptr(src),
                                        _np_ptr(dst), _np_ptr(rel), _np_ptr(ntype), flags,
                                        None if host_only else _stream(stream), ctypes.byref(h))
        _check(st)
        return cls(h)

    @classmethod
    def from_csr(cls, N, T, R, rowptr, col_src, rel, ntype=None, host_only=False, stream=None):
        rowptr = _host(rowptr, np.int64)
        col_src, rel, ntype = _host(col_src, np.int32), _host(rel, np.int32), _host(ntype, np.int32)
        h = ctypes.c_void_p()
        st = _lib.rgnn_graph_create_csr(int(N), int(T), int(R), _np_ptr(rowptr), _np_ptr(col_src),
                                        _np_ptr(rel), _np_ptr(ntype),
                                        GRAPH_HOST_ONLY if host_only else 0,
                                        None if host_only else _stream(stream), ctypes.byref(h))
        _check(st)
        return cls(h)

    @classmethod
    def from_dict(cls, g, host_only=False, compact=True):
        return cls.from_coo(g["N"], g["T"], g["R"], g["src"], g["dst"], g["rel"], g["ntype"],
                            host_only=host_only, compact=compact)

    @property
    def handle(self):
        if self._h is None:
            raise ValueError("graph destroyed")
        return self._h

    def info(self) -> dict:
        inf = GraphInfo()
        _check(_lib.rgnn_graph_info(self.handle, ctypes.byref(inf)))
        return {f: getattr(inf, f) for f, _ in GraphInfo._fields_}

    def export(self, kind: str) -> np.ndarray:
        inf = self.info()
        n = {"dst_rowptr": inf["num_nodes"] + 1, "dst_segptr": inf["num_nodes"] + 1,
             "in_src": inf["num_edges"], "in_rel": inf["num_edges"], "in_eid": inf["num_edges"],
             "edge2uniq": inf["num_edges"], "seg_ptr": inf["num_dst_segments"] + 1,
             "seg_rel": inf["num_dst_segments"], "uniq_src": inf["num_src_pairs"],
             "uniq_rel_ptr": inf["num_rels"] + 1, "ntype_perm": inf["num_nodes"],
             "ntype_ptr": inf["num_ntypes"] + 1, "out_ptr": inf["num_nodes"] + 1,
             "out_pos": inf["num_edges"]}[kind]
        out = np.empty(max(n, 1), np.int32)
        _check(_lib.rgnn_graph_export(self.handle, INDEX_KINDS[kind], _np_ptr(out), out.nbytes))
        return out[:n]

    def close(self):
        if self._h is not None:
            _check(_lib.rgnn_graph_destroy(self._h))
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def workspace_size(g: Graph, layer: int, d_in: int, d_out: int, heads: int = 1,
                   plan: int = PLAN_AUTO) -> int:
    n = ctypes.c_size_t()
    _check(_lib.rgnn_workspace_size(g.handle, layer, d_in, d_out, heads, plan, ctypes.byref(n)))
    return n.value


def select_plan(g: Graph, layer: int, d_in: int, d_out: int, heads: int = 1):
    p = ctypes.c_int32()
    tf, af = ctypes.c_double(), ctypes.c_double()
    _check(_lib.rgnn_select_plan(g.handle, layer, d_in, d_out, heads, ctypes.byref(p),
                                 ctypes.byref(tf), ctypes.byref(af)))
    return p.value, tf.value, af.value


def rgcn_forward(g, h, W, W0, out, ws, d_in, d_out, flags=0, plan=PLAN_AUTO, stream=None):
    _check(_lib.rgcn_forward(g.handle, _ptr(h), _ptr(W), _ptr(W0), d_in, d_out, flags, plan,
                             _ptr(out), _ptr(ws), 0 if ws is None else ws.numel() * ws.element_size(),
                             _stream(stream)))


def rgat_forward(g, h, W, w_src, w_dst, out, saved, ws, d_in, d_out, heads=1, neg_slope=0.2,
                 softmax_scope=SOFTMAX_PER_DST, plan=PLAN_AUTO, stream=None):
    _check(_lib.rgat_forward(g.handle, _ptr(h), _ptr(W), _ptr(w_src), _ptr(w_dst), d_in, d_out,
                             heads, float(neg_slope), softmax_scope, plan, _ptr(out), _ptr(saved),
                             _ptr(ws), 0 if ws is None else ws.numel() * ws.element_size(),
                             _stream(stream)))


def rgat_forward_noalloc(g, h, W, w_src, w_dst, out, saved, d_in, d_out, heads=1, neg_slope=0.2,
                         softmax_scope=SOFTMAX_PER_DST, plan=PLAN_AUTO, stream=None):
    """rgat_forward with the workspace in the library's static device scratch."""
    _check(_lib.rgat_forward_noalloc(g.handle, _ptr(h), _ptr(W), _ptr(w_src), _ptr(w_dst), d_in, d_out,
                                     heads, float(neg_slope), softmax_scope, plan, _ptr(out), _ptr(saved),
                                     _stream(stream)))


def hgt_forward(g, h, Wk, Wq, Wv, Wa, Watt, Wmsg, mu, out, ws, d, heads, att_scale,
                flags=FLAG_RESIDUAL | FLAG_A_LINEAR, stream=None, saved=None):
    """saved: None or a [N, heads, 2] tensor for the softmax statistics."""
    _check(_lib.hgt_forward(g.handle, _ptr(h), _ptr(Wk), _ptr(Wq), _ptr(Wv), _ptr(Wa), _ptr(Watt),
                            _ptr(Wmsg), _ptr(mu), d, heads, float(att_scale), flags, _ptr(out),
                            _ptr(saved), _ptr(ws), 0 if ws is None else ws.numel() * ws.element_size(),
                            _stream(stream)))


def hgt_backward(g, h, Wk, Wq, Wv, Wa, Watt, Wmsg, mu, grad_out, grads, ws, d, heads, att_scale,
                 flags=FLAG_RESIDUAL | FLAG_A_LINEAR, stream=None, saved=None):
    """grads: dict of output tensors dh, dWk, dWq, dWv, dWa (or None), dWatt, dWmsg, dmu.
    saved: the forward's statistics (hgt_forward's saved), or None to recompute them."""
    _check(_lib.hgt_backward(g.handle, _ptr(h), _ptr(Wk), _ptr(Wq), _ptr(Wv), _ptr(Wa), _ptr(Watt),
                             _ptr(Wmsg), _ptr(mu), d, heads, float(att_scale), flags, _ptr(grad_out),
                             _ptr(saved), _ptr(grads["dh"]), _ptr(grads["dWk"]), _ptr(grads["dWq"]), _ptr(grads["dWv"]),
                             _ptr(grads.get("dWa")), _ptr(grads["dWatt"]), _ptr(grads["dWmsg"]),
                             _ptr(grads["dmu"]), _ptr(ws), 0 if ws is None else ws.numel() * ws.element_size(),
                             _stream(stream)))


def rgcn_backward(g, h, W, W0, out, grad_out, grad_h, grad_W, grad_W0, ws, d_in, d_out, flags=0,
                  stream=None):
    _check(_lib.rgcn_backward(g.handle, _ptr(h), _ptr(W), _ptr(W0), d_in, d_out, flags, _ptr(out),
                              _ptr(grad_out), _ptr(grad_h), _ptr(grad_W), _ptr(grad_W0), _ptr(ws),
                              0 if ws is None else ws.numel() * ws.element_size(), _stream(stream)))


def rgat_backward(g, h, W, w_src, w_dst, saved, grad_out, grad_h, grad_W, grad_w_src,
                  grad_w_dst, ws, d_in, d_out, heads=1, neg_slope=0.2,
                  softmax_scope=SOFTMAX_PER_DST, stream=None):
    _check(_lib.rgat_backward(g.handle, _ptr(h), _ptr(W), _ptr(w_src), _ptr(w_dst), d_in, d_out,
                              heads, float(neg_slope), softmax_scope, _ptr(saved), _ptr(grad_out),
                              _ptr(grad_h),
                              _ptr(grad_W), _ptr(grad_w_src), _ptr(grad_w_dst), _ptr(ws),
                              0 if ws is None else ws.numel() * ws.element_size(),
                              _stream(stream)))


def segment_gemm_workspace_size(M: int, num_types: int) -> int:
    n = ctypes.c_size_t()
    _check(_lib.rgnn_segment_gemm_workspace_size(M, num_types, ctypes.byref(n)))
    return n.value


def segment_gemm(X, gather, type_ptr, W, Y, scatter, ws, K, Nc, stream=None):
    tp = _host(type_ptr, np.int64)
    _check(_lib.rgnn_segment_gemm(_ptr(X), X.shape[1], _ptr(gather), _np_ptr(tp), len(tp) - 1,
                                  _ptr(W), K, Nc, _ptr(Y), Y.shape[1], _ptr(scatter), _ptr(ws),
                                  0 if ws is None else ws.numel() * ws.element_size(),
                                  _stream(stream)))


def profile_enable(on: bool):
    _check(_lib.rgnn_profile_enable(1 if on else 0))


def profile_reset():
    _check(_lib.rgnn_profile_reset())


def profile_read() -> dict:
    """{kernel name: (launches, total ms)} of the launches recorded while enabled."""
    n = ctypes.c_int32()
    _check(_lib.rgnn_profile_count(ctypes.byref(n)))
    out = {}
    buf = ctypes.create_string_buffer(128)
    for i in range(n.value):
        cnt, ms = ctypes.c_int64(), ctypes.c_double()
        _check(_lib.rgnn_profile_read(i, buf, 128, ctypes.byref(cnt), ctypes.byref(ms)))
        out[buf.value.decode()] = (cnt.value, ms.value)
    return out


def version() -> str:
    return _lib.rgnn_version().decode()
