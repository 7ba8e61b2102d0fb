"""GPU parity at the workloads' full sizes, in the launch configuration the
benchmark times.  The whole output is computed on the GPU; the fp64 oracle
recomputes sampled destinations one by one (the largest hubs, destinations
without in-edges and a random sample).  Properties that hold at any size are
checked on every row: empty destinations give exact zeros, softmax
denominators are >= 1, outputs are finite.

Workloads (seeded, see workloads/synth.py):
  1  RGCN   2 000 nodes / 20 000 edges / 8 relations, d = 64
  2  RGAT   880 000 nodes / 5.7 M edges / 96 relations, d = 64
  3  HGT    1.9 M nodes / 21 M edges / 7 relations, d = 64 = 4 x 16
  4  RGCN, RGAT at d = 128 on 2.5 M nodes / 16 M edges / 535 relations
  5  RGAT and RGCN backward on workload 2's graph
Workload 2's graph also runs at d = 32 (the hidden-size sweep).
"""
import numpy as np
import pytest

import oracle
import workloads
from helpers import TOL, Runner, row_err, sample_rows

pytestmark = pytest.mark.gpu

_cache = {}


def load(k):
    if k not in _cache:
        _cache.clear()
        g = workloads.make_graph(k)
        layer = workloads.CONFIGS[k]["layers"][0]
        t = workloads.make_tensors(k, g, layer)
        _cache[k] = (g, t, Runner(g, t))
    return _cache[k]


@pytest.fixture(scope="module", autouse=True)
def gpu():
    import torch
    assert torch.cuda.is_available()
    torch.cuda.set_device(0)
    yield
    _cache.clear()


def check_properties(g, out, saved=None):
    deg = np.bincount(g["dst"], minlength=g["N"])
    assert np.isfinite(out).all()
    if saved is not None:
        s = saved.cpu().numpy().reshape(g["N"], -1, 2)
        assert (s[deg == 0] == 0).all()
        assert (s[deg > 0][..., 1] >= 1 - 1e-5).all()
        assert np.isfinite(s).all()


@pytest.mark.parametrize("plan", [1, 2])
def test_workload1_rgcn_all_rows(plan):
    g, t, run = load(1)
    print(f"workload 1 rgcn plan={plan}", flush=True)
    got = run.rgcn(W0=True, plan=plan)
    ref = oracle.rgcn_forward(g, t["h"], t["W"], t["W0"])
    assert row_err(got, ref) <= TOL


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
    g, t, run = load(1)
    ix = oracle.graph_index(g)
    for k in run.rgnn.INDEX_KINDS:
        np.testing.assert_array_equal(run.G.export(k), ix[k], err_msg=k)


def test_workload2_graph_index_bit_exact():
    g, t, run = load(2)
    print("workload 2 index", flush=True)
    ix = oracle.graph_index(g)
    for k in run.rgnn.INDEX_KINDS:
        np.testing.assert_array_equal(run.G.export(k), ix[k], err_msg=k)


@pytest.mark.parametrize("plan", [1, 2])
def test_workload2_rgat(plan):
    g, t, run = load(2)
    print(f"workload 2 rgat plan={plan}", flush=True)
    got, saved = run.rgat(plan=plan, want_saved=True)
    check_properties(g, got, saved)
    sel = sample_rows(g, 300, seed=plan)
    ref, mx, sm = oracle.rgat_forward(g, t["h"], t["W"], t["w_src"], t["w_dst"], sel=sel,
                                      want_stats=True)
    assert row_err(got[sel], ref) <= TOL
    s = saved.cpu().numpy()[sel, 0]
    np.testing.assert_allclose(s[:, 0], mx[:, 0], rtol=1e-4, atol=1e-4)
    np.testing.assert_allclose(s[:, 1], sm[:, 0], rtol=1e-4)


def test_workload2_rgat_per_relation_softmax():
    g, t, run = load(2)
    print("workload 2 rgat per-relation softmax", flush=True)
    got = run.rgat(scope=1)
    assert np.isfinite(got).all()
    sel = sample_rows(g, 300, seed=5)
    ref = oracle.rgat_forward(g, t["h"], t["W"], t["w_src"], t["w_dst"], scope=1, sel=sel)
    assert row_err(got[sel], ref) <= TOL


@pytest.mark.parametrize("layer", ["rgat", "rgcn"])
def test_workload2_graph_d32(layer):
    """The hidden-size sweep's narrow end: workload 2's graph with d = 32
    tensors, both plans."""
    g, _, _ = load(2)
    t = workloads.make_tensors(2, g, "rgat", 32)
    run = Runner(g, t)
    sel = sample_rows(g, 200, seed=32)
    if layer == "rgat":
        ref = oracle.rgat_forward(g, t["h"], t["W"], t["w_src"], t["w_dst"], sel=sel)
    else:
        ref = oracle.rgcn_forward(g, t["h"], t["W"], t["W0"], sel=sel)
    for plan in (1, 2):
        print(f"workload 2 graph d=32 {layer} plan={plan}", flush=True)
        got = run.rgat(plan=plan) if layer == "rgat" else run.rgcn(W0=True, plan=plan)
        assert np.isfinite(got).all()
        assert row_err(got[sel], ref) <= TOL
    run.close()


def test_workload3_hgt():
    g, t, run = load(3)
    print("workload 3 hgt", flush=True)
    got = run.hgt(4, 0.25)
    assert np.isfinite(got).all()
    sel = sample_rows(g, 300)
    ref = oracle.hgt_forward(g, t["h"], t["Wk"], t["Wq"], t["Wv"], t["Wa"], t["Watt"], t["Wmsg"],
                             t["mu"], heads=4, att_scale=0.25, sel=sel)
    assert row_err(got[sel], ref) <= TOL


def test_workload3_hgt_saved_and_backward():
    """The full 21 M-edge HGT layer: the forward's saved softmax statistics
    leave its output unchanged and satisfy the per-destination properties, and
    the backward from them agrees with the backward that recomputes them
    (a property at any size; the oracle checks both on the mid-size graphs)."""
    g, t, run = load(3)
    print("workload 3 hgt saved statistics and backward", flush=True)
    plain = run.hgt(4, 0.25)
    out, saved = run.hgt(4, 0.25, want_saved=True)
    np.testing.assert_array_equal(out, plain)
    check_properties(g, out, saved)
    del saved
    a = run.hgt_backward(4, 0.25, use_saved=True)
    b = run.hgt_backward(4, 0.25, use_saved=False)
    for k in ("dh", "dWk", "dWq", "dWv", "dWa"):
        assert np.isfinite(a[k]).all(), k
        assert row_err(a[k].reshape(-1, 64), b[k].reshape(-1, 64)) <= 1e-5, k
    for k in ("dWatt", "dWmsg"):
        assert row_err(a[k].reshape(-1, 16), b[k].reshape(-1, 16)) <= 1e-5, k
    assert row_err(a["dmu"].reshape(1, -1), b["dmu"].reshape(1, -1)) <= 1e-5


@pytest.mark.parametrize("d,heads", [(32, 2), (128, 8)])
def test_workload3_graph_hgt_hidden_sizes(d, heads):
    """HGT on workload 3's graph with d = 32 and 128 tensors (the
    hidden-size sweep), sampled rows."""
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
    sel = sample_rows(g, 200, seed=d)
    ref = oracle.hgt_forward(g, t["h"], t["Wk"], t["Wq"], t["Wv"], t["Wa"], t["Watt"], t["Wmsg"],
                             t["mu"], heads=H, att_scale=scale, sel=sel)
    assert row_err(got[sel], ref) <= TOL


@pytest.mark.parametrize("plan", [1, 2])
def test_workload4_rgcn(plan):
    g, t, run = load(4)
    print(f"workload 4 rgcn plan={plan}", flush=True)
    got = run.rgcn(W0=True, plan=plan)
    assert np.isfinite(got).all()
    sel = sample_rows(g, 200, seed=plan)
    ref = oracle.rgcn_forward(g, t["h"], t["W"], t["W0"], sel=sel)
    assert row_err(got[sel], ref) <= TOL


@pytest.mark.parametrize("plan", [1, 2])
def test_workload4_rgat(plan):
    g, t, run = load(4)
    print(f"workload 4 rgat plan={plan}", flush=True)
    got, saved = run.rgat(plan=plan, want_saved=True)
    check_properties(g, got, saved)
    sel = sample_rows(g, 150, seed=10 + plan)
    ref = oracle.rgat_forward(g, t["h"], t["W"], t["w_src"], t["w_dst"], sel=sel)
    assert row_err(got[sel], ref) <= TOL


@pytest.mark.parametrize("layer", ["rgat", "rgcn"])
def test_workload4_backward_d128(layer):
    """RGAT and RGCN backward at d = 128 on the 2.5M-node graph (hubs of up
    to 5e5 in-edges, 535 relations), sampled like workload 5's."""
    g, t, run = load(4)
    print(f"workload 4 {layer} backward d=128", flush=True)
    rng = np.random.default_rng(41)
    relcount = np.bincount(g["rel"], minlength=g["R"])
    rels = np.r_[np.argsort(relcount)[:3], [7]]
    nodes = rng.choice(g["N"], 40, replace=False)
    nm = np.zeros(g["N"], np.uint8); nm[nodes] = 1
    rm = np.zeros(g["R"], np.uint8); rm[rels] = 1
    isolated = (np.bincount(g["src"], minlength=g["N"]) + np.bincount(g["dst"], minlength=g["N"])) == 0
    if layer == "rgat":
        gh, gW, gs, gt = run.rgat_backward()
        dh, dW, dws, dwt = oracle.rgat_backward(g, t["h"], t["W"], t["w_src"], t["w_dst"], t["grad_out"],
                                                node_mask=nm, rel_mask=rm)
        assert row_err(gs[rels], dws[rels], cancel_floor=1e-6) <= TOL
        assert row_err(gt[rels], dwt[rels], cancel_floor=1e-6) <= TOL
    else:
        gh, gW, _ = run.rgcn_backward(W0=True)
        dh, dW, _ = oracle.rgcn_backward(g, t["h"], t["W"], t["W0"], t["grad_out"], node_mask=nm,
                                         rel_mask=rm, want_dW0=False)
    assert np.isfinite(gh).all() and np.isfinite(gW).all()
    assert row_err(gh[nodes], dh[nodes], structural_zero=isolated[nodes], cancel_floor=1e-6) <= TOL
    assert row_err(gW[rels].reshape(-1, 128), dW[rels].reshape(-1, 128), cancel_floor=1e-6) <= TOL


def test_workload5_rgat_backward():
    g, t, run = load(5)
    print("workload 5 rgat backward", flush=True)
    gh, gW, gs, gt = run.rgat_backward()
    for a in (gh, gW, gs, gt):
        assert np.isfinite(a).all()
    rng = np.random.default_rng(5)
    relcount = np.bincount(g["rel"], minlength=g["R"])
    rels = np.r_[np.argsort(relcount)[:3], [20]]
    nodes = rng.choice(g["N"], 60, replace=False)
    nm = np.zeros(g["N"], np.uint8); nm[nodes] = 1
    rm = np.zeros(g["R"], np.uint8); rm[rels] = 1
    dh, dW, dws, dwt = oracle.rgat_backward(g, t["h"], t["W"], t["w_src"], t["w_dst"],
                                            t["grad_out"], node_mask=nm, rel_mask=rm)
    isolated = (np.bincount(g["src"], minlength=g["N"]) + np.bincount(g["dst"], minlength=g["N"])) == 0
    assert row_err(gh[nodes], dh[nodes], structural_zero=isolated[nodes], cancel_floor=1e-6) <= TOL
    assert row_err(gW[rels].reshape(-1, 64), dW[rels].reshape(-1, 64)) <= TOL
    assert row_err(gs[rels], dws[rels]) <= TOL
    assert row_err(gt[rels], dwt[rels]) <= TOL


def test_workload5_rgat_backward_per_relation_softmax():
    """The per-(dst, rel) softmax backward on the 880k-node graph, sampled as
    above (the oracle visits only the destinations that feed the sample)."""
    g, t, run = load(5)
    print("workload 5 rgat backward per-relation softmax", flush=True)
    gh, gW, gs, gt = run.rgat_backward(scope=1)
    for a in (gh, gW, gs, gt):
        assert np.isfinite(a).all()
    rng = np.random.default_rng(6)
    relcount = np.bincount(g["rel"], minlength=g["R"])
    rels = np.r_[np.argsort(relcount)[:3], [17]]
    nodes = rng.choice(g["N"], 60, replace=False)
    nm = np.zeros(g["N"], np.uint8); nm[nodes] = 1
    rm = np.zeros(g["R"], np.uint8); rm[rels] = 1
    dh, dW, dws, dwt = oracle.rgat_backward(g, t["h"], t["W"], t["w_src"], t["w_dst"],
                                            t["grad_out"], scope=1, node_mask=nm, rel_mask=rm)
    isolated = (np.bincount(g["src"], minlength=g["N"]) + np.bincount(g["dst"], minlength=g["N"])) == 0
    assert row_err(gh[nodes], dh[nodes], structural_zero=isolated[nodes], cancel_floor=1e-6) <= TOL
    assert row_err(gW[rels].reshape(-1, 64), dW[rels].reshape(-1, 64), cancel_floor=1e-6) <= TOL
    assert row_err(gs[rels], dws[rels], cancel_floor=1e-6) <= TOL
    assert row_err(gt[rels], dwt[rels], cancel_floor=1e-6) <= TOL


def test_workload5_rgcn_backward():
    """RGCN backward (with self-loop, identity activation) on the 880k-node
    graph: dh at sampled sources, dW at sampled relations, dW0 in full."""
    g, t, run = load(5)
    print("workload 5 rgcn backward", flush=True)
    W0 = t["W0"]
    gh, gW, gW0 = run.rgcn_backward(W0=True, relu=False)
    for a in (gh, gW, gW0):
        assert np.isfinite(a).all()
    rng = np.random.default_rng(56)
    relcount = np.bincount(g["rel"], minlength=g["R"])
    rels = np.r_[np.argsort(relcount)[:3], [20]]
    outdeg = np.bincount(g["src"], minlength=g["N"])
    nodes = np.unique(np.r_[rng.choice(g["N"], 60, replace=False), np.argsort(-outdeg)[:4],
                            np.flatnonzero(outdeg == 0)[:4]])
    nm = np.zeros(g["N"], np.uint8); nm[nodes] = 1
    rm = np.zeros(g["R"], np.uint8); rm[rels] = 1
    dh, dW, dW0 = oracle.rgcn_backward(g, t["h"], t["W"], W0, t["grad_out"], node_mask=nm, rel_mask=rm)
    assert row_err(gh[nodes], dh[nodes]) <= TOL
    assert row_err(gW[rels].reshape(-1, 64), dW[rels].reshape(-1, 64)) <= TOL
    assert row_err(gW0, dW0) <= TOL


@pytest.mark.parametrize("kind,heads,use_saved", [("random", 4, False), ("hub", 2, False), ("random", 4, True),
                                                   ("hub", 2, True)])
def test_hgt_backward_mid_size(kind, heads, use_saved):
    """HGT backward on a 20 000-node / 300 000-edge graph with 7 relations and
    4 node types (thousands of work items and GEMM tiles, split destinations
    for the hub kind), checked in full against the oracle (the 21 M-edge
    workload itself is beyond the fp64 oracle's budget; bench.py runs it)."""
    g = workloads.tiny_graph(36, N=20000, E=300000, R=7, T=4, kind=kind)
    t = workloads.tiny_tensors(36, g, 64, 64, heads=heads)
    t["mu"] = (1.0 + 0.25 * np.arange(7)).astype(np.float32)
    scale = 1.0 / np.sqrt(64 // heads)
    print(f"hgt backward mid-size {kind} heads={heads} saved={use_saved}", flush=True)
    run = Runner(g, t)
    got = run.hgt_backward(heads, scale, use_saved=use_saved)
    run.close()
    ref = oracle.hgt_backward(g, t["h"], t["Wk"], t["Wq"], t["Wv"], t["Wa"], t["Watt"], t["Wmsg"],
                              t["mu"], t["grad_out"], heads=heads, att_scale=scale)
    dk = 64 // heads
    assert row_err(got["dh"], ref["dh"]) <= TOL
    for k in ("dWk", "dWq", "dWv", "dWa"):
        assert row_err(got[k].reshape(-1, 64), ref[k].reshape(-1, 64)) <= TOL, k
    for k in ("dWatt", "dWmsg"):
        assert row_err(got[k].reshape(-1, dk), ref[k].reshape(-1, dk)) <= TOL, k
    assert row_err(got["dmu"].reshape(1, -1), ref["dmu"].reshape(1, -1)) <= TOL
