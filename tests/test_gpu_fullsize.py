"""GPU parity at the workloads' full sizes, in the launch configuration the
benchmark times.  Every forward output row is compared with the fp64 oracle
(which evaluates each destination edge by edge over the whole graph), every
index array is compared bit for bit, and the RGAT backward on workload 5 is
compared in full (every dh row, every relation's dW, dw_src and dw_dst).
The HGT and RGCN backward at full size, and the RGAT backward at d = 128,
are compared on node and relation samples that include the largest hubs
(the oracle visits only the destinations that feed the sampled entries).
Properties that hold at any size are checked on every row: empty
destinations give exact zeros, softmax denominators are >= 1, outputs are
finite.

Workloads (seeded, see workloads/synth.py):
  1  RGCN   2 000 nodes / 20 000 edges / 8 relations, d = 64
  2  RGAT   880 000 nodes / 5.7 M edges / 96 relations, d = 64
  3  HGT    1.9 M nodes / 21 M edges / 7 relations, d = 64 = 4 x 16
  4  RGCN, RGAT at d = 128 on 2.5 M nodes / 16 M edges / 535 relations
  5  RGAT and RGCN backward on workload 2's graph
Workload 2's graph also runs at d = 32 (the hidden-size sweep), workload 3's
at d = 32 and 128.
"""
import numpy as np
import pytest

import oracle
import workloads
from helpers import TOL, Runner, rgat_backward_ref, row_err

pytestmark = pytest.mark.gpu

_cache = {}
_refs = {}


def load(k):
    if k not in _cache:
        _cache.clear()
        _refs.clear()
        g = workloads.make_graph(k)
        layer = workloads.CONFIGS[k]["layers"][0]
        t = workloads.make_tensors(k, g, layer)
        _cache[k] = (g, t, Runner(g, t))
    return _cache[k]


def ref(key, fn):
    """fp64 oracle output, computed once per key while its workload is loaded."""
    if key not in _refs:
        print(f"  oracle {key}", flush=True)
        _refs[key] = fn()
    return _refs[key]


@pytest.fixture(scope="module", autouse=True)
def gpu():
    import torch
    assert torch.cuda.is_available()
    torch.cuda.set_device(0)
    yield
    _cache.clear()
    _refs.clear()


def check_properties(g, out, saved=None):
    deg = np.bincount(g["dst"], minlength=g["N"])
    assert np.isfinite(out).all()
    if saved is not None:
        s = saved.cpu().numpy().reshape(g["N"], -1, 2)
        assert (s[deg == 0] == 0).all()
        assert (s[deg > 0][..., 1] >= 1 - 1e-5).all()
        assert np.isfinite(s).all()


def hub_nodes(g, n_random, seed, n_top=4):
    """Sampled nodes for the backward checks: the largest in- and out-degrees,
    nodes without in-edges or without out-edges, and a random sample."""
    indeg = np.bincount(g["dst"], minlength=g["N"])
    outdeg = np.bincount(g["src"], minlength=g["N"])
    rng = np.random.default_rng(seed)
    return np.unique(np.r_[np.argsort(-indeg, kind="stable")[:n_top], np.argsort(-outdeg, kind="stable")[:n_top],
                           np.flatnonzero(indeg == 0)[:4], np.flatnonzero(outdeg == 0)[:4],
                           rng.choice(g["N"], n_random, replace=False)]).astype(np.int64)


def masks(g, nodes, rels):
    nm = np.zeros(g["N"], np.uint8); nm[nodes] = 1
    rm = np.zeros(g["R"], np.uint8); rm[rels] = 1
    return nm, rm


def isolated(g):
    return (np.bincount(g["src"], minlength=g["N"]) + np.bincount(g["dst"], minlength=g["N"])) == 0


def check_index(k):
    """Every exported index array of the device graph equals the oracle's
    numpy construction, bit for bit."""
    g, t, run = load(k)
    print(f"workload {k} index", flush=True)
    ix = oracle.graph_index(g)
    for name in run.rgnn.INDEX_KINDS:
        np.testing.assert_array_equal(run.G.export(name), ix[name], err_msg=name)
    info = run.G.info()
    assert info["num_src_pairs"] == ix["U_src"] and info["num_dst_segments"] == ix["U_dst"]


# ------------------------------------------------------------------ workload 1
@pytest.mark.parametrize("plan", [1, 2])
def test_workload1_rgcn_all_rows(plan):
    g, t, run = load(1)
    print(f"workload 1 rgcn plan={plan}", flush=True)
    got = run.rgcn(W0=True, plan=plan)
    r = ref("rgcn", lambda: oracle.rgcn_forward(g, t["h"], t["W"], t["W0"]))
    assert row_err(got, r) <= TOL


@pytest.mark.parametrize("relu", [False, True])
def test_workload1_rgcn_backward_all_rows(relu):
    g, t, run = load(1)
    print(f"workload 1 rgcn backward relu={relu}", flush=True)
    out = oracle.rgcn_forward(g, t["h"], t["W"], t["W0"], relu=True) if relu else None
    gh, gW, gW0 = run.rgcn_backward(W0=True, relu=relu, out=out)
    dh, dW, dW0 = oracle.rgcn_backward(g, t["h"], t["W"], t["W0"], t["grad_out"], relu=relu)
    assert row_err(gh, dh) <= TOL
    assert row_err(gW.reshape(-1, 64), dW.reshape(-1, 64)) <= TOL
    assert row_err(gW0, dW0) <= TOL


def test_workload1_graph_index_bit_exact():
    check_index(1)


# ------------------------------------------------------------------ workload 2
@pytest.mark.parametrize("plan", [1, 2, 4])
def test_workload2_rgat(plan):
    """Every plan (4: attention+message rows), every output row and every
    destination's softmax statistics."""
    g, t, run = load(2)
    print(f"workload 2 rgat plan={plan}", flush=True)
    got, saved = run.rgat(plan=plan, want_saved=True)
    check_properties(g, got, saved)
    r, mx, sm = ref("rgat", lambda: oracle.rgat_forward(g, t["h"], t["W"], t["w_src"], t["w_dst"],
                                                        want_stats=True))
    assert row_err(got, r) <= TOL
    s = saved.cpu().numpy()[:, 0]
    has = np.bincount(g["dst"], minlength=g["N"]) > 0
    np.testing.assert_allclose(s[has, 0], mx[has, 0], rtol=1e-4, atol=1e-4)
    np.testing.assert_allclose(s[has, 1], sm[has, 0], rtol=1e-4)


@pytest.mark.parametrize("plan", [1, 2])
def test_workload2_rgat_four_heads(plan):
    """Four heads of 16 columns on the 880k-node graph, transform-first and
    aggregate-first, every output row."""
    g, t, run = load(2)
    print(f"workload 2 rgat 4 heads plan={plan}", flush=True)
    got, saved = run.rgat(heads=4, plan=plan, want_saved=True)
    check_properties(g, got, saved)
    r = ref("rgat4", lambda: oracle.rgat_forward(g, t["h"], t["W"], t["w_src"], t["w_dst"], heads=4))
    assert row_err(got, r) <= TOL


def test_workload2_rgat_per_relation_softmax():
    g, t, run = load(2)
    print("workload 2 rgat per-relation softmax", flush=True)
    got = run.rgat(scope=1)
    assert np.isfinite(got).all()
    r = oracle.rgat_forward(g, t["h"], t["W"], t["w_src"], t["w_dst"], scope=1)
    assert row_err(got, r) <= TOL


@pytest.mark.parametrize("layer", ["rgat", "rgcn"])
def test_workload2_graph_d32(layer):
    """The hidden-size sweep's narrow end: workload 2's graph with d = 32
    tensors, both plans, every row."""
    g, _, _ = load(2)
    t = workloads.make_tensors(2, g, "rgat", 32)
    run = Runner(g, t)
    if layer == "rgat":
        r = oracle.rgat_forward(g, t["h"], t["W"], t["w_src"], t["w_dst"])
    else:
        r = oracle.rgcn_forward(g, t["h"], t["W"], t["W0"])
    for plan in (1, 2):
        print(f"workload 2 graph d=32 {layer} plan={plan}", flush=True)
        got = run.rgat(plan=plan) if layer == "rgat" else run.rgcn(W0=True, plan=plan)
        assert np.isfinite(got).all()
        assert row_err(got, r) <= TOL
    run.close()


def test_workload2_graph_index_bit_exact():
    check_index(2)


# ------------------------------------------------------------------ workload 3
def test_workload3_hgt():
    g, t, run = load(3)
    print("workload 3 hgt", flush=True)
    got, saved = run.hgt(4, 0.25, want_saved=True)
    check_properties(g, got, saved)
    plain = run.hgt(4, 0.25)
    np.testing.assert_array_equal(got, plain)   # saving the statistics leaves the output unchanged
    r = oracle.hgt_forward(g, t["h"], t["Wk"], t["Wq"], t["Wv"], t["Wa"], t["Watt"], t["Wmsg"],
                           t["mu"], heads=4, att_scale=0.25)
    assert row_err(got, r) <= TOL


@pytest.mark.parametrize("use_saved", [True, False])
def test_workload3_hgt_backward(use_saved):
    """The HGT backward on the 21 M-edge graph against the oracle: dh on
    sampled nodes (largest in- and out-degrees included), dWatt, dWmsg and
    dmu of the smallest and the largest cross-type relations; both from the
    forward's saved statistics and recomputing them."""
    g, t, run = load(3)
    print(f"workload 3 hgt backward saved={use_saved}", flush=True)
    got = run.hgt_backward(4, 0.25, use_saved=use_saved)
    for k in ("dh", "dWk", "dWq", "dWv", "dWa", "dWatt", "dWmsg", "dmu"):
        assert np.isfinite(got[k]).all(), k
    relcount = np.bincount(g["rel"], minlength=g["R"])
    rels = np.r_[np.argmin(relcount), [3]]
    nodes = hub_nodes(g, 200, 31)
    nm, rm = masks(g, nodes, rels)
    r = ref("hgt_bwd", lambda: oracle.hgt_backward(g, t["h"], t["Wk"], t["Wq"], t["Wv"], t["Wa"], t["Watt"],
                                                   t["Wmsg"], t["mu"], t["grad_out"], heads=4, att_scale=0.25,
                                                   node_mask=nm, rel_mask=rm))
    assert row_err(got["dh"][nodes], r["dh"][nodes]) <= TOL
    for k in ("dWatt", "dWmsg"):
        assert row_err(got[k][rels].reshape(-1, 16), r[k][rels].reshape(-1, 16)) <= TOL, k
    assert row_err(got["dmu"][rels].reshape(1, -1), r["dmu"][rels].reshape(1, -1)) <= TOL


@pytest.mark.parametrize("d,heads", [(32, 2), (128, 8)])
def test_workload3_graph_hgt_hidden_sizes(d, heads):
    """HGT on workload 3's graph with d = 32 and 128 tensors (the
    hidden-size sweep), every row."""
    g, _, _ = load(3)
    H = heads
    dk = d // H
    t = workloads.make_tensors(3, g, "hgt", d, heads=H)
    run = Runner(g, t)
    scale = 1.0 / np.sqrt(dk)
    print(f"workload 3 graph hgt d={d} heads={H}", flush=True)
    got = run.hgt(H, scale)
    run.close()
    assert np.isfinite(got).all()
    r = oracle.hgt_forward(g, t["h"], t["Wk"], t["Wq"], t["Wv"], t["Wa"], t["Watt"], t["Wmsg"],
                           t["mu"], heads=H, att_scale=scale)
    assert row_err(got, r) <= TOL


def test_workload3_graph_index_bit_exact():
    check_index(3)


# ------------------------------------------------------------------ workload 4
@pytest.mark.parametrize("plan", [1, 2])
def test_workload4_rgcn(plan):
    g, t, run = load(4)
    print(f"workload 4 rgcn plan={plan}", flush=True)
    got = run.rgcn(W0=True, plan=plan)
    assert np.isfinite(got).all()
    r = ref("rgcn", lambda: oracle.rgcn_forward(g, t["h"], t["W"], t["W0"]))
    assert row_err(got, r) <= TOL


@pytest.mark.parametrize("plan", [1, 2])
def test_workload4_rgat(plan):
    g, t, run = load(4)
    print(f"workload 4 rgat plan={plan}", flush=True)
    got, saved = run.rgat(plan=plan, want_saved=True)
    check_properties(g, got, saved)
    r = ref("rgat", lambda: oracle.rgat_forward(g, t["h"], t["W"], t["w_src"], t["w_dst"]))
    assert row_err(got, r) <= TOL


@pytest.mark.parametrize("layer", ["rgat", "rgcn"])
def test_workload4_backward_d128(layer):
    """RGAT and RGCN backward at d = 128 on the 2.5M-node graph (hubs of up
    to 5e5 in-edges, 535 relations): dh on sampled nodes with the largest in-
    and out-degrees, dW (and dw_src, dw_dst) of the three rarest relations and
    of two mid-frequency ones."""
    g, t, run = load(4)
    print(f"workload 4 {layer} backward d=128", flush=True)
    order = np.argsort(np.bincount(g["rel"], minlength=g["R"]), kind="stable")
    rels = np.r_[order[:3], order[-20], order[-100]]
    nodes = hub_nodes(g, 60, 41)
    nm, rm = masks(g, nodes, rels)
    iso = isolated(g)[nodes]
    if layer == "rgat":
        gh, gW, gs, gt = run.rgat_backward()
        dh, dW, dws, dwt = rgat_backward_ref(g, t, node_mask=nm, rel_mask=rm)
        assert row_err(gs[rels], dws[rels], cancel_floor=1e-6) <= TOL
        assert row_err(gt[rels], dwt[rels], cancel_floor=1e-6) <= TOL
    else:
        gh, gW, _ = run.rgcn_backward(W0=True)
        dh, dW, _ = oracle.rgcn_backward(g, t["h"], t["W"], t["W0"], t["grad_out"], node_mask=nm,
                                         rel_mask=rm, want_dW0=False)
    assert np.isfinite(gh).all() and np.isfinite(gW).all()
    assert row_err(gh[nodes], dh[nodes], structural_zero=iso, cancel_floor=1e-6) <= TOL
    assert row_err(gW[rels].reshape(-1, 128), dW[rels].reshape(-1, 128), cancel_floor=1e-6) <= TOL


def test_workload4_graph_index_bit_exact():
    check_index(4)


# ------------------------------------------------------------------ workload 5
@pytest.mark.parametrize("scope", [0, 1])
def test_workload5_rgat_backward(scope):
    """The RGAT training step on the 880k-node graph, every gradient in full:
    dh of all 880 000 nodes, dW, dw_src and dw_dst of all 96 relations; the
    softmax over each destination's in-edges (scope 0) or over each
    (destination, relation) segment (scope 1)."""
    g, t, run = load(5)
    print(f"workload 5 rgat backward scope={scope}", flush=True)
    gh, gW, gs, gt = run.rgat_backward(scope=scope)
    for a in (gh, gW, gs, gt):
        assert np.isfinite(a).all()
    dh, dW, dws, dwt = rgat_backward_ref(g, t, scope=scope)
    assert row_err(gh, dh, structural_zero=isolated(g), cancel_floor=1e-6) <= TOL
    assert row_err(gW.reshape(-1, 64), dW.reshape(-1, 64), cancel_floor=1e-6) <= TOL
    assert row_err(gs, dws, cancel_floor=1e-6) <= TOL
    assert row_err(gt, dwt, cancel_floor=1e-6) <= TOL


def test_workload5_rgcn_backward():
    """RGCN backward (with self-loop, identity activation) on the 880k-node
    graph: dh at sampled nodes with the largest in- and out-degrees, dW of the
    three rarest and the three most frequent relations, dW0 in full."""
    g, t, run = load(5)
    print("workload 5 rgcn backward", flush=True)
    W0 = t["W0"]
    gh, gW, gW0 = run.rgcn_backward(W0=True, relu=False)
    for a in (gh, gW, gW0):
        assert np.isfinite(a).all()
    order = np.argsort(np.bincount(g["rel"], minlength=g["R"]), kind="stable")
    rels = np.r_[order[:3], order[-3:]]
    nodes = hub_nodes(g, 400, 56)
    nm, rm = masks(g, nodes, rels)
    dh, dW, dW0 = oracle.rgcn_backward(g, t["h"], t["W"], W0, t["grad_out"], node_mask=nm, rel_mask=rm)
    assert row_err(gh[nodes], dh[nodes]) <= TOL
    assert row_err(gW[rels].reshape(-1, 64), dW[rels].reshape(-1, 64)) <= TOL
    assert row_err(gW0, dW0) <= TOL


# ------------------------------------------------------------------ mid-size HGT backward
@pytest.mark.parametrize("kind,heads,use_saved", [("random", 4, False), ("hub", 2, False), ("random", 4, True),
                                                   ("hub", 2, True)])
def test_hgt_backward_mid_size(kind, heads, use_saved):
    """HGT backward on a 20 000-node / 300 000-edge graph with 7 relations and
    4 node types (thousands of work items and GEMM tiles, split destinations
    for the hub kind), every gradient in full against the oracle, including
    the node-type weight gradients that the full-size test leaves out."""
    g = workloads.tiny_graph(36, N=20000, E=300000, R=7, T=4, kind=kind)
    t = workloads.tiny_tensors(36, g, 64, 64, heads=heads)
    t["mu"] = (1.0 + 0.25 * np.arange(7)).astype(np.float32)
    scale = 1.0 / np.sqrt(64 // heads)
    print(f"hgt backward mid-size {kind} heads={heads} saved={use_saved}", flush=True)
    run = Runner(g, t)
    got = run.hgt_backward(heads, scale, use_saved=use_saved)
    run.close()
    r = oracle.hgt_backward(g, t["h"], t["Wk"], t["Wq"], t["Wv"], t["Wa"], t["Watt"], t["Wmsg"],
                            t["mu"], t["grad_out"], heads=heads, att_scale=scale)
    dk = 64 // heads
    assert row_err(got["dh"], r["dh"]) <= TOL
    for k in ("dWk", "dWq", "dWv", "dWa"):
        assert row_err(got[k].reshape(-1, 64), r[k].reshape(-1, 64)) <= TOL, k
    for k in ("dWatt", "dWmsg"):
        assert row_err(got[k].reshape(-1, dk), r[k].reshape(-1, dk)) <= TOL, k
    assert row_err(got["dmu"].reshape(1, -1), r["dmu"].reshape(1, -1)) <= TOL
