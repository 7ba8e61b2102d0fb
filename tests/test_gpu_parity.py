"""GPU parity on small graphs: every layer and plan through the C ABI against
the fp64 oracle, element by element, on graphs that still span many work
items, split hub destinations, empty destinations, duplicate edges and
ragged GEMM tiles.  Index arrays are compared bit for bit."""
import numpy as np
import pytest

import oracle
import workloads
from helpers import TOL, Runner, rgat_backward_ref, row_err

pytestmark = pytest.mark.gpu

KINDS = ["random", "hub", "srchub", "dups", "isolated", "empty"]


@pytest.fixture(scope="module", autouse=True)
def gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2301_06284_amd import rgnn  # noqa: F401  (fails loudly if not built)
    torch.cuda.set_device(0)


def graph(kind, seed=5, N=300, E=4000, R=6, T=3):
    return workloads.tiny_graph(seed, N=N, E=E, R=R, T=T, kind=kind)


@pytest.mark.parametrize("kind", KINDS + ["complete"])
def test_device_graph_index_bit_exact(kind):
    from paper_2301_06284_amd import rgnn
    g = graph(kind, N=120 if kind == "complete" else 300)
    print(f"graph index {kind}", flush=True)
    G = rgnn.Graph.from_dict(g)
    ix = oracle.graph_index(g)
    for k in rgnn.INDEX_KINDS:
        np.testing.assert_array_equal(G.export(k), ix[k], err_msg=k)
    G.close()


@pytest.mark.parametrize("K,Nc", [(32, 32), (64, 64), (128, 128), (64, 128), (128, 64)])
def test_segment_gemm(K, Nc):
    import torch
    from paper_2301_06284_amd import rgnn
    rng = np.random.default_rng(K + Nc)
    type_ptr = np.array([0, 5, 5, 200, 201, 777, 1000], np.int64)   # empty and 1-row types
    M, T = int(type_ptr[-1]), len(type_ptr) - 1
    X = rng.standard_normal((1500, K)).astype(np.float32)
    W = rng.standard_normal((T, K, Nc)).astype(np.float32)
    gather = rng.integers(0, 1500, M).astype(np.int32)
    scatter = rng.permutation(1200)[:M].astype(np.int32)
    print(f"segment_gemm {K}x{Nc}", flush=True)
    dev = torch.device("cuda:0")
    Xd, Wd = torch.from_numpy(X).to(dev), torch.from_numpy(W).to(dev)
    gd, sd = torch.from_numpy(gather).to(dev), torch.from_numpy(scatter).to(dev)
    Y = torch.zeros(1200, Nc, device=dev)
    ws = torch.empty(rgnn.segment_gemm_workspace_size(M, T), dtype=torch.uint8, device=dev)
    rgnn.segment_gemm(Xd, gd, type_ptr, Wd, Y, sd, ws, K, Nc)
    torch.cuda.synchronize()
    ref = np.zeros((1200, Nc))
    for t in range(T):
        rows = np.arange(type_ptr[t], type_ptr[t + 1])
        ref[scatter[rows]] = X[gather[rows]].astype(np.float64) @ W[t].astype(np.float64)
    assert row_err(Y.cpu().numpy(), ref) <= TOL


@pytest.mark.parametrize("K,Nc", [(32, 32), (64, 64), (128, 128), (64, 128), (128, 64)])
def test_segment_gemm_fp32_grade(K, Nc):
    """Every output entry within a few fp32 unit roundoffs of the exact product,
    relative to sum_k |x_k w_k| (a sequential fp32 dot product is bounded by K of
    them): the 64-deep shapes, whose products run on split bf16 pieces, must be
    as accurate as the fp32 MFMA ones.  Rows span twelve decades of scale, and
    a plain bf16 (or two-piece bf16) product would miss the bound by far."""
    import torch
    from paper_2301_06284_amd import rgnn
    rng = np.random.default_rng(1000 + K + Nc)
    type_ptr = np.array([0, 700, 701, 1500, 2048], np.int64)
    M, T = int(type_ptr[-1]), len(type_ptr) - 1
    X = (rng.standard_normal((M, K)) * 10.0 ** rng.uniform(-6, 6, (M, 1))).astype(np.float32)
    W = (rng.standard_normal((T, K, Nc)) * 10.0 ** rng.uniform(-3, 3, (T, 1, Nc))).astype(np.float32)
    gather = np.arange(M, dtype=np.int32)
    scatter = rng.permutation(M).astype(np.int32)
    print(f"segment_gemm fp32 grade {K}x{Nc}", flush=True)
    dev = torch.device("cuda:0")
    Y = torch.zeros(M, Nc, device=dev)
    ws = torch.empty(rgnn.segment_gemm_workspace_size(M, T), dtype=torch.uint8, device=dev)
    rgnn.segment_gemm(torch.from_numpy(X).to(dev), torch.from_numpy(gather).to(dev), type_ptr,
                      torch.from_numpy(W).to(dev), Y, torch.from_numpy(scatter).to(dev), ws, K, Nc)
    torch.cuda.synchronize()
    got = Y.cpu().numpy().astype(np.float64)
    u = 2.0 ** -24
    worst = 0.0
    for t in range(T):
        rows = np.arange(type_ptr[t], type_ptr[t + 1])
        x, w = X[rows].astype(np.float64), W[t].astype(np.float64)
        exact = x @ w
        scale = np.abs(x) @ np.abs(w)
        worst = max(worst, float((np.abs(got[scatter[rows]] - exact) / (u * scale)).max()))
    print(f"  max error / (u sum |x w|) = {worst:.2f}", flush=True)
    assert worst <= 8.0


@pytest.mark.parametrize("d,heads", [(128, 1), (128, 2), (64, 1)])
def test_rgat_many_relations(d, heads):
    """More relations than the segment-term kernel can stage in LDS (their
    reordered w_dst vectors: 700 x d floats per head): the vectors are read
    with the rows instead.  Forward (both plans) and backward."""
    g = graph("random", seed=9, N=600, E=6000, R=700, T=2)
    t = workloads.tiny_tensors(9, g, d, d, heads=heads, att_var=1.0)
    print(f"rgat many relations d={d} heads={heads}", flush=True)
    run = Runner(g, t)
    ref = oracle.rgat_forward(g, t["h"], t["W"], t["w_src"], t["w_dst"], heads=heads)
    for plan in (1, 2) if heads == 1 else (1,):
        assert row_err(run.rgat(heads=heads, plan=plan), ref) <= TOL
    gh, gW, gs, gt = run.rgat_backward(heads=heads)
    run.close()
    dh, dW, dws, dwt = rgat_backward_ref(g, t, heads=heads)
    isolated = (np.bincount(g["src"], minlength=g["N"]) + np.bincount(g["dst"], minlength=g["N"])) == 0
    assert row_err(gh, dh, structural_zero=isolated, cancel_floor=1e-6) <= TOL
    assert row_err(gW.reshape(-1, d), dW.reshape(-1, d), cancel_floor=1e-6) <= TOL
    assert row_err(gs, dws, cancel_floor=1e-6) <= TOL
    assert row_err(gt, dwt, cancel_floor=1e-6) <= TOL


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("plan", [1, 2])
@pytest.mark.parametrize("W0,relu", [(True, False), (False, False), (True, True), (False, True)])
def test_rgcn_small(kind, plan, W0, relu):
    g = graph(kind)
    t = workloads.tiny_tensors(1, g, 64, 64)
    print(f"rgcn {kind} plan={plan} W0={W0} relu={relu}", flush=True)
    run = Runner(g, t)
    got = run.rgcn(W0=W0, relu=relu, plan=plan)
    ref = oracle.rgcn_forward(g, t["h"], t["W"], t["W0"] if W0 else None, relu=relu)
    run.close()
    assert row_err(got, ref) <= TOL


@pytest.mark.parametrize("d_in,d_out", [(128, 128), (64, 128), (128, 64)])
@pytest.mark.parametrize("plan", [1, 2])
def test_rgcn_dims(d_in, d_out, plan):
    g = graph("hub", seed=9)
    t = workloads.tiny_tensors(9, g, d_in, d_out)
    print(f"rgcn dims {d_in}->{d_out} plan={plan}", flush=True)
    run = Runner(g, t)
    got = run.rgcn(plan=plan)
    ref = oracle.rgcn_forward(g, t["h"], t["W"], t["W0"])
    run.close()
    assert row_err(got, ref) <= TOL


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("plan,heads", [(1, 1), (2, 1), (1, 2), (1, 4), (2, 2), (2, 4), (4, 1), (4, 2), (4, 4)])
def test_rgat_small(kind, plan, heads):
    """Plans 1 (transform-first), 2 (aggregate-first; several heads as one
    masked pass per head) and 4 (transform-first with attention+message
    rows), 1 to 4 heads: output and saved statistics against the oracle."""
    g = graph(kind)
    t = workloads.tiny_tensors(2, g, 64, 64, heads=heads, att_var=1.0)
    print(f"rgat {kind} plan={plan} heads={heads}", flush=True)
    run = Runner(g, t)
    got, saved = run.rgat(heads=heads, plan=plan, want_saved=True)
    ref, mx, sm = oracle.rgat_forward(g, t["h"], t["W"], t["w_src"], t["w_dst"], heads=heads,
                                      want_stats=True)
    run.close()
    assert row_err(got, ref) <= TOL
    sv = saved.cpu().numpy()
    np.testing.assert_allclose(sv[..., 0], mx, rtol=1e-4, atol=1e-4)
    np.testing.assert_allclose(sv[..., 1], sm, rtol=1e-4, atol=1e-5)


@pytest.mark.parametrize("plan,heads", [(1, 1), (2, 1), (1, 8), (2, 8), (4, 8), (4, 1)])
def test_rgat_d128(plan, heads):
    g = graph("hub", seed=4)
    t = workloads.tiny_tensors(4, g, 128, 128, heads=heads, att_var=1.0)
    print(f"rgat d128 plan={plan} heads={heads}", flush=True)
    run = Runner(g, t)
    got = run.rgat(heads=heads, plan=plan)
    ref = oracle.rgat_forward(g, t["h"], t["W"], t["w_src"], t["w_dst"], heads=heads)
    run.close()
    assert row_err(got, ref) <= TOL


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("plan", [1, 2])
@pytest.mark.parametrize("W0,relu", [(True, True), (False, False)])
def test_rgcn_d32(kind, plan, W0, relu):
    """Hidden size 32 (the narrow end of the hidden-size sweep)."""
    g = graph(kind, seed=41)
    t = workloads.tiny_tensors(41, g, 32, 32)
    print(f"rgcn d32 {kind} plan={plan} W0={W0} relu={relu}", flush=True)
    run = Runner(g, t)
    got = run.rgcn(W0=W0, relu=relu, plan=plan)
    ref = oracle.rgcn_forward(g, t["h"], t["W"], t["W0"] if W0 else None, relu=relu)
    run.close()
    assert row_err(got, ref) <= TOL


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("plan,heads", [(1, 1), (2, 1), (3, 1), (1, 2)])
def test_rgat_d32(kind, plan, heads):
    g = graph(kind, seed=42)
    t = workloads.tiny_tensors(42, g, 32, 32, heads=heads, att_var=1.0)
    print(f"rgat d32 {kind} plan={plan} heads={heads}", flush=True)
    run = Runner(g, t)
    got, saved = run.rgat(heads=heads, plan=plan, want_saved=True)
    ref, mx, sm = oracle.rgat_forward(g, t["h"], t["W"], t["w_src"], t["w_dst"], heads=heads,
                                      want_stats=True)
    run.close()
    assert row_err(got, ref) <= TOL
    sv = saved.cpu().numpy()
    np.testing.assert_allclose(sv[..., 0], mx, rtol=1e-4, atol=1e-4)
    np.testing.assert_allclose(sv[..., 1], sm, rtol=1e-4, atol=1e-5)


def test_d32_huge_hub():
    """d = 32 through the 256- and 1024-thread reductions and the split
    destination merges (a hub with thousands of in-edges)."""
    g = graph("hub", seed=43, N=200, E=70000, R=3)
    t = workloads.tiny_tensors(43, g, 32, 32, att_var=1.0)
    print("d32 huge hub", flush=True)
    run = Runner(g, t)
    ref_gcn = oracle.rgcn_forward(g, t["h"], t["W"], t["W0"])
    ref_gat = oracle.rgat_forward(g, t["h"], t["W"], t["w_src"], t["w_dst"])
    for plan in (1, 2):
        assert row_err(run.rgcn(plan=plan), ref_gcn) <= TOL
        assert row_err(run.rgat(plan=plan), ref_gat) <= TOL
    ref_rel = oracle.rgat_forward(g, t["h"], t["W"], t["w_src"], t["w_dst"], scope=1)
    assert row_err(run.rgat(scope=1), ref_rel) <= TOL
    run.close()


def test_d32_rejects_mixed_widths():
    import torch
    from paper_2301_06284_amd import rgnn
    g = graph("random", seed=44)
    t = workloads.tiny_tensors(44, g, 32, 64)
    print("d32 mixed widths rejected", flush=True)
    run = Runner(g, t)
    T = run.T
    out = torch.empty(g["N"], 64, device="cuda:0")
    ws = run.ws(0, 32, 64, 1, 1)
    with pytest.raises(rgnn.RgnnError) as e:
        rgnn.rgcn_forward(run.G, T["h"], T["W"], None, out, ws, 32, 64, plan=rgnn.PLAN_TRANSFORM_FIRST)
    assert e.value.status == rgnn.EUNSUPPORTED
    run.close()


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("d", [32, 64, 128])
def test_rgat_per_relation_softmax(kind, d):
    """Softmax over the in-edges of one (destination, relation) segment."""
    g = graph(kind)
    t = workloads.tiny_tensors(21, g, d, d, att_var=1.0)
    print(f"rgat per-relation softmax {kind} d={d}", flush=True)
    run = Runner(g, t)
    got = run.rgat(plan=0, scope=1)
    again = run.rgat(plan=2, scope=1)
    run.close()
    ref = oracle.rgat_forward(g, t["h"], t["W"], t["w_src"], t["w_dst"], scope=1)
    assert row_err(got, ref) <= TOL
    assert np.array_equal(got, again)


def test_rgat_per_relation_softmax_big_segment():
    """One (destination, relation) segment cut into more pieces than one
    thread reduces (the workgroup-per-segment statistics path)."""
    g = graph("hub", seed=22, N=200, E=6000, R=1)
    t = workloads.tiny_tensors(22, g, 64, 64, att_var=1.0)
    print("rgat per-relation softmax big segment", flush=True)
    run = Runner(g, t)
    got = run.rgat(scope=1)
    run.close()
    ref = oracle.rgat_forward(g, t["h"], t["W"], t["w_src"], t["w_dst"], scope=1)
    assert row_err(got, ref) <= TOL


@pytest.mark.parametrize("R", [1, 3])
def test_huge_hub(R):
    """Destinations with hundreds to thousands of virtual segments (the
    workgroup-per-destination reductions at the front of the reduction grid)
    beside ordinary ones, through every plan of RGCN and RGAT."""
    g = graph("hub", seed=24, N=200, E=70000, R=R)
    t = workloads.tiny_tensors(24, g, 64, 64, att_var=1.0)
    print(f"huge hub R={R}", flush=True)
    run = Runner(g, t)
    ref_gcn = oracle.rgcn_forward(g, t["h"], t["W"], t["W0"])
    ref_gat = oracle.rgat_forward(g, t["h"], t["W"], t["w_src"], t["w_dst"])
    for plan in (1, 2):
        assert row_err(run.rgcn(plan=plan), ref_gcn) <= TOL
        assert row_err(run.rgat(plan=plan), ref_gat) <= TOL
    ref_rel = oracle.rgat_forward(g, t["h"], t["W"], t["w_src"], t["w_dst"], scope=1)
    assert row_err(run.rgat(scope=1), ref_rel) <= TOL
    run.close()


def test_rgat_per_relation_softmax_rejects():
    import torch
    from paper_2301_06284_amd import rgnn
    g = graph("random", seed=23)
    t = workloads.tiny_tensors(23, g, 64, 64)
    print("rgat per-relation softmax argument checks", flush=True)
    run = Runner(g, t)
    T = run.T
    out = torch.empty(g["N"], 64, device="cuda:0")
    saved = torch.empty(g["N"], 1, 2, device="cuda:0")
    ws = run.ws(1, 64, 64, 1, 2)
    with pytest.raises(rgnn.RgnnError, match="aggregate-first"):
        rgnn.rgat_forward(run.G, T["h"], T["W"], T["w_src"], T["w_dst"], out, None, ws, 64, 64,
                          softmax_scope=rgnn.SOFTMAX_PER_DST_REL, plan=rgnn.PLAN_TRANSFORM_FIRST)
    run.close()


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("heads", [1, 2, 4])
def test_hgt_small(kind, heads):
    g = graph(kind, T=4, R=7)
    t = workloads.tiny_tensors(3, g, 64, 64, heads=heads)
    scale = 1.0 / np.sqrt(64 // heads)
    print(f"hgt {kind} heads={heads}", flush=True)
    run = Runner(g, t)
    got = run.hgt(heads, scale)
    ref = oracle.hgt_forward(g, t["h"], t["Wk"], t["Wq"], t["Wv"], t["Wa"], t["Watt"], t["Wmsg"],
                             t["mu"], heads=heads, att_scale=scale)
    run.close()
    assert row_err(got, ref) <= TOL


@pytest.mark.parametrize("kind", ["random", "hub", "dups", "empty"])
@pytest.mark.parametrize("d,heads", [(32, 1), (32, 2), (128, 1), (128, 2), (128, 4), (128, 8)])
def test_hgt_hidden_sizes(kind, d, heads):
    """HGT at d = 32 and 128 (the hidden-size sweep), every head count with
    d_k >= 16; R = 7 keeps W_msg in LDS except at d = 128 with one or two
    heads (global reads)."""
    g = graph(kind, T=4, R=7)
    t = workloads.tiny_tensors(49, g, d, d, heads=heads)
    scale = 1.0 / np.sqrt(d // heads)
    print(f"hgt d={d} {kind} heads={heads}", flush=True)
    run = Runner(g, t)
    got = run.hgt(heads, scale)
    ref = oracle.hgt_forward(g, t["h"], t["Wk"], t["Wq"], t["Wv"], t["Wa"], t["Watt"], t["Wmsg"],
                             t["mu"], heads=heads, att_scale=scale)
    run.close()
    assert row_err(got, ref) <= TOL


@pytest.mark.parametrize("kind", ["typed", "typedhub"])
@pytest.mark.parametrize("d,heads", [(32, 1), (32, 2), (64, 1), (64, 2), (64, 4), (128, 2), (128, 8)])
def test_hgt_typed_relations(kind, d, heads):
    """Relations that each join one source type to one destination type: the
    forward folds the query projection into the segment-query weights (all
    widths where the traversal does not form the queries itself)."""
    g = graph(kind, T=4, R=7)
    t = workloads.tiny_tensors(51, g, d, d, heads=heads)
    t["mu"] = (1.0 + 0.25 * np.arange(7)).astype(np.float32)
    scale = 1.0 / np.sqrt(d // heads)
    print(f"hgt typed d={d} {kind} heads={heads}", flush=True)
    run = Runner(g, t)
    got = run.hgt(heads, scale)
    ref = oracle.hgt_forward(g, t["h"], t["Wk"], t["Wq"], t["Wv"], t["Wa"], t["Watt"], t["Wmsg"],
                             t["mu"], heads=heads, att_scale=scale)
    run.close()
    assert row_err(got, ref) <= TOL


@pytest.mark.parametrize("heads,R", [(2, 12), (4, 24)])
def test_hgt_many_relations(heads, R):
    """Enough relations that the per-relation message matrices no longer fit
    in LDS beside the staged items (the traversal reads them from memory)."""
    g = graph("random", T=3, R=R, E=5000)
    t = workloads.tiny_tensors(4, g, 64, 64, heads=heads)
    scale = 1.0 / np.sqrt(64 // heads)
    print(f"hgt heads={heads} R={R}", flush=True)
    run = Runner(g, t)
    got = run.hgt(heads, scale)
    ref = oracle.hgt_forward(g, t["h"], t["Wk"], t["Wq"], t["Wv"], t["Wa"], t["Watt"], t["Wmsg"],
                             t["mu"], heads=heads, att_scale=scale)
    run.close()
    assert row_err(got, ref) <= TOL


@pytest.mark.parametrize("flags", [0, 2, 4])
def test_hgt_flags(flags):
    g = graph("hub", T=2, R=3)
    t = workloads.tiny_tensors(6, g, 64, 64, heads=4)
    print(f"hgt flags={flags}", flush=True)
    run = Runner(g, t)
    got = run.hgt(4, 0.3, flags=flags)
    ref = oracle.hgt_forward(g, t["h"], t["Wk"], t["Wq"], t["Wv"], t["Wa"], t["Watt"], t["Wmsg"],
                             t["mu"], heads=4, att_scale=0.3, residual=bool(flags & 2),
                             a_linear=bool(flags & 4))
    run.close()
    assert row_err(got, ref) <= TOL


@pytest.mark.parametrize("kind", KINDS)
def test_rgat_backward_small(kind):
    g = graph(kind, E=3000)
    t = workloads.tiny_tensors(8, g, 64, 64, att_var=1.0)
    print(f"rgat backward {kind}", flush=True)
    run = Runner(g, t)
    gh, gW, gs, gt = run.rgat_backward()
    run.close()
    dh, dW, dws, dwt = rgat_backward_ref(g, t)
    isolated = (np.bincount(g["src"], minlength=g["N"]) + np.bincount(g["dst"], minlength=g["N"])) == 0
    assert row_err(gh, dh, structural_zero=isolated, cancel_floor=1e-6) <= TOL
    assert row_err(gW.reshape(-1, 64), dW.reshape(-1, 64)) <= TOL
    assert row_err(gs, dws) <= TOL
    assert row_err(gt, dwt) <= TOL


@pytest.mark.parametrize("kind", KINDS)
def test_rgat_backward_per_relation_softmax(kind):
    """Softmax per (dst, rel) segment: the forward's per-segment (max, sum)
    feed the backward; s is summed per segment."""
    g = graph(kind, E=3000)
    t = workloads.tiny_tensors(47, g, 64, 64, att_var=1.0)
    print(f"rgat backward per-relation softmax {kind}", flush=True)
    run = Runner(g, t)
    gh, gW, gs, gt = run.rgat_backward(scope=1)
    run.close()
    dh, dW, dws, dwt = rgat_backward_ref(g, t, scope=1)
    isolated = (np.bincount(g["src"], minlength=g["N"]) + np.bincount(g["dst"], minlength=g["N"])) == 0
    assert row_err(gh, dh, structural_zero=isolated, cancel_floor=1e-6) <= TOL
    # a relation whose segments each repeat one (src, rel) pair has uniform
    # attention, Y = 0 on all its edges and zero w_dst / w_src gradients by
    # cancellation (fp64 ~1e-17, fp32 ~1e-8)
    assert row_err(gW.reshape(-1, 64), dW.reshape(-1, 64), cancel_floor=1e-6) <= TOL
    assert row_err(gs, dws, cancel_floor=1e-6) <= TOL
    assert row_err(gt, dwt, cancel_floor=1e-6) <= TOL


@pytest.mark.parametrize("kind", ["random", "hub", "dups", "empty"])
@pytest.mark.parametrize("heads", [2, 4])
def test_rgat_per_relation_softmax_multihead(kind, heads):
    """Softmax per (dst, rel) segment with several heads: the forward as one
    masked one-head pass per head, the backward in one pass over all heads,
    against the oracle."""
    g = graph(kind, E=3000)
    t = workloads.tiny_tensors(50, g, 64, 64, heads=heads, att_var=1.0)
    print(f"rgat per-relation softmax {kind} heads={heads}", flush=True)
    run = Runner(g, t)
    got, saved = run.rgat(heads=heads, scope=1, want_saved=True)
    ref = oracle.rgat_forward(g, t["h"], t["W"], t["w_src"], t["w_dst"], heads=heads, scope=1)
    assert row_err(got, ref) <= TOL
    sv = saved.cpu().numpy()
    if len(sv):
        assert np.isfinite(sv).all() and (sv[..., 1] >= 1 - 1e-5).all()
    gh, gW, gs, gt = run.rgat_backward(heads=heads, scope=1)
    run.close()
    dh, dW, dws, dwt = rgat_backward_ref(g, t, heads=heads, scope=1)
    isolated = (np.bincount(g["src"], minlength=g["N"]) + np.bincount(g["dst"], minlength=g["N"])) == 0
    assert row_err(gh, dh, structural_zero=isolated, cancel_floor=1e-6) <= TOL
    assert row_err(gW.reshape(-1, 64), dW.reshape(-1, 64), cancel_floor=1e-6) <= TOL
    assert row_err(gs, dws, cancel_floor=1e-6) <= TOL
    assert row_err(gt, dwt, cancel_floor=1e-6) <= TOL


def test_rgat_backward_per_relation_softmax_hub_segments():
    """Segments cut into many pieces (one relation, a 5000-edge hub: more
    than 32 pieces in one segment) and destinations split over work items."""
    g = graph("hub", seed=48, N=400, E=12000, R=1)
    t = workloads.tiny_tensors(48, g, 64, 64, att_var=1.0)
    print("rgat backward per-relation softmax hub segments", flush=True)
    run = Runner(g, t)
    _, saved = run.rgat(scope=1, want_saved=True)
    sv = saved.cpu().numpy()
    assert np.isfinite(sv).all() and (sv[..., 1] >= 1 - 1e-5).all()
    gh, gW, gs, gt = run.rgat_backward(scope=1)
    run.close()
    dh, dW, dws, dwt = rgat_backward_ref(g, t, scope=1)
    isolated = (np.bincount(g["src"], minlength=g["N"]) + np.bincount(g["dst"], minlength=g["N"])) == 0
    assert row_err(gh, dh, structural_zero=isolated, cancel_floor=1e-6) <= TOL
    # a relation whose segments each repeat one (src, rel) pair has uniform
    # attention, Y = 0 on all its edges and zero w_dst / w_src gradients by
    # cancellation (fp64 ~1e-17, fp32 ~1e-8)
    assert row_err(gW.reshape(-1, 64), dW.reshape(-1, 64), cancel_floor=1e-6) <= TOL
    assert row_err(gs, dws, cancel_floor=1e-6) <= TOL
    assert row_err(gt, dwt, cancel_floor=1e-6) <= TOL


@pytest.mark.parametrize("kind", ["random", "hub", "srchub", "dups", "empty"])
@pytest.mark.parametrize("d,heads,scope", [(32, 1, 0), (32, 2, 0), (32, 2, 1), (32, 1, 1), (64, 2, 1), (64, 4, 1),
                                           (128, 1, 0), (128, 2, 0), (128, 4, 1), (128, 8, 0), (128, 8, 1),
                                           (128, 1, 1)])
def test_rgat_backward_hidden_sizes(kind, d, heads, scope):
    """RGAT backward at d = 32, 64 and 128, one to eight heads, both softmax
    scopes (the outer products as 64 x 64 tiles: one zero-padded tile at 32,
    four at 128)."""
    g = graph(kind, E=3000)
    t = workloads.tiny_tensors(51, g, d, d, heads=heads, att_var=1.0)
    print(f"rgat backward d={d} heads={heads} scope={scope} {kind}", flush=True)
    run = Runner(g, t)
    gh, gW, gs, gt = run.rgat_backward(heads=heads, scope=scope)
    run.close()
    dh, dW, dws, dwt = rgat_backward_ref(g, t, heads=heads, scope=scope)
    isolated = (np.bincount(g["src"], minlength=g["N"]) + np.bincount(g["dst"], minlength=g["N"])) == 0
    assert row_err(gh, dh, structural_zero=isolated, cancel_floor=1e-6) <= TOL
    assert row_err(gW.reshape(-1, d), dW.reshape(-1, d), cancel_floor=1e-6) <= TOL
    assert row_err(gs, dws, cancel_floor=1e-6) <= TOL
    assert row_err(gt, dwt, cancel_floor=1e-6) <= TOL


@pytest.mark.parametrize("kind", ["random", "hub", "srchub", "dups", "empty"])
@pytest.mark.parametrize("d", [32, 128])
@pytest.mark.parametrize("W0,relu", [(True, True), (False, False)])
def test_rgcn_backward_hidden_sizes(kind, d, W0, relu):
    g = graph(kind, seed=52)
    t = workloads.tiny_tensors(52, g, d, d)
    print(f"rgcn backward d={d} {kind} W0={W0} relu={relu}", flush=True)
    run = Runner(g, t)
    out = oracle.rgcn_forward(g, t["h"], t["W"], t["W0"] if W0 else None, relu=True) if relu else None
    gh, gW, gW0 = run.rgcn_backward(W0=W0, relu=relu, out=out)
    run.close()
    dh, dW, dW0 = oracle.rgcn_backward(g, t["h"], t["W"], t["W0"] if W0 else None, t["grad_out"], relu=relu)
    isolated = (np.bincount(g["src"], minlength=g["N"]) + np.bincount(g["dst"], minlength=g["N"])) == 0
    assert row_err(gh, dh, structural_zero=None if W0 else isolated, cancel_floor=1e-6) <= TOL
    assert row_err(gW.reshape(-1, d), dW.reshape(-1, d), cancel_floor=1e-6) <= TOL
    if W0:
        assert row_err(gW0, dW0) <= TOL


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("heads", [2, 4])
def test_rgat_backward_multihead(kind, heads):
    """Several heads in one backward pass (gradients in the message space)."""
    g = graph(kind, E=3000)
    t = workloads.tiny_tensors(45, g, 64, 64, heads=heads, att_var=1.0)
    print(f"rgat backward {kind} heads={heads}", flush=True)
    run = Runner(g, t)
    gh, gW, gs, gt = run.rgat_backward(heads=heads)
    run.close()
    dh, dW, dws, dwt = rgat_backward_ref(g, t, heads=heads)
    isolated = (np.bincount(g["src"], minlength=g["N"]) + np.bincount(g["dst"], minlength=g["N"])) == 0
    assert row_err(gh, dh, structural_zero=isolated, cancel_floor=1e-6) <= TOL
    assert row_err(gW.reshape(-1, 64), dW.reshape(-1, 64)) <= TOL
    assert row_err(gs, dws) <= TOL
    assert row_err(gt, dwt) <= TOL


@pytest.mark.parametrize("d,heads,kind", [(64, 2, "hub"), (64, 4, "hub"), (128, 8, "hub"), (64, 4, "srchub"),
                                         (32, 2, "srchub"), (128, 4, "srchub")])
def test_rgat_backward_multihead_mid_size(d, heads, kind):
    """Several heads on a 200k-edge graph with hubs (split destinations and
    sources with many out-edges), every gradient in full, at the standard
    cancellation floor.

    The multi-head forward (transform-first) forms its logits from the message
    rows, the backward from h . (W_r w_src): the two round differently.  The
    backward sums its own softmax denominator, so its alpha sums to one in its
    own arithmetic.  This graph has sources whose only out-edges enter the
    10^5-edge hub (dh norm ~1e-5 of the median) and whose one in-edge forms a
    one-edge softmax, whose Jacobian is exactly zero: with alpha normalised by
    the forward's denominator instead, that zero came out as ~1e-7 |dalpha|,
    a 3e-4 row error.
    With a source hub (half the edges leave node 0: pairs of ~8 000 out-edges,
    cut into 64-edge pieces over several workgroup chunks at d <= 64, and a
    source split over ~1 500 out-edge items) the same checks hold."""
    g = workloads.tiny_graph(46, N=20000, E=200000, R=12, T=2, kind=kind)
    t = workloads.tiny_tensors(46, g, d, d, heads=heads, att_var=1.0)
    print(f"rgat backward d={d} heads={heads} {kind} mid size", flush=True)
    run = Runner(g, t)
    gh, gW, gs, gt = run.rgat_backward(heads=heads)
    run.close()
    dh, dW, dws, dwt = rgat_backward_ref(g, t, heads=heads)
    isolated = (np.bincount(g["src"], minlength=g["N"]) + np.bincount(g["dst"], minlength=g["N"])) == 0
    assert row_err(gh, dh, structural_zero=isolated, cancel_floor=1e-6) <= TOL
    assert row_err(gW.reshape(-1, d), dW.reshape(-1, d)) <= TOL
    assert row_err(gs, dws) <= TOL
    assert row_err(gt, dwt) <= TOL


@pytest.mark.parametrize("plan", [1, 2])
def test_rgat_backward_mid_size_one_head(plan):
    """The graph above with one head, from the saved statistics of either
    forward plan (transform-first forms the source logit from the message
    row, aggregate-first from h . (W_r w_src)), standard cancellation floor."""
    g = workloads.tiny_graph(46, N=20000, E=200000, R=12, T=2, kind="hub")
    t = workloads.tiny_tensors(46, g, 64, 64, heads=1, att_var=1.0)
    print(f"rgat backward heads=1 mid size forward plan={plan}", flush=True)
    run = Runner(g, t)
    gh, gW, gs, gt = run.rgat_backward(heads=1, plan=plan)
    run.close()
    dh, dW, dws, dwt = rgat_backward_ref(g, t)
    isolated = (np.bincount(g["src"], minlength=g["N"]) + np.bincount(g["dst"], minlength=g["N"])) == 0
    assert row_err(gh, dh, structural_zero=isolated, cancel_floor=1e-6) <= TOL
    assert row_err(gW.reshape(-1, 64), dW.reshape(-1, 64)) <= TOL
    assert row_err(gs, dws) <= TOL
    assert row_err(gt, dwt) <= TOL


@pytest.mark.parametrize("d", [64, 128])
def test_backward_mid_size_source_hub(d):
    """One-head RGAT and RGCN backward on a 200k-edge graph whose node 0 sends
    half the edges: its out-edges span ~1 500 work items, whose sums are added
    to its row in slot order."""
    g = workloads.tiny_graph(47, N=20000, E=200000, R=12, T=2, kind="srchub")
    t = workloads.tiny_tensors(47, g, d, d, heads=1, att_var=1.0)
    print(f"rgat/rgcn backward d={d} source hub mid size", flush=True)
    run = Runner(g, t)
    gh, gW, gs, gt = run.rgat_backward(heads=1)
    rh, rW, rW0 = run.rgcn_backward(W0=True, relu=False)
    run.close()
    dh, dW, dws, dwt = rgat_backward_ref(g, t)
    isolated = (np.bincount(g["src"], minlength=g["N"]) + np.bincount(g["dst"], minlength=g["N"])) == 0
    assert row_err(gh, dh, structural_zero=isolated, cancel_floor=1e-6) <= TOL
    assert row_err(gW.reshape(-1, d), dW.reshape(-1, d)) <= TOL
    assert row_err(gs, dws) <= TOL
    assert row_err(gt, dwt) <= TOL
    eh, eW, eW0 = oracle.rgcn_backward(g, t["h"], t["W"], t["W0"], t["grad_out"], relu=False)
    assert row_err(rh, eh) <= TOL
    assert row_err(rW.reshape(-1, d), eW.reshape(-1, d)) <= TOL
    assert row_err(rW0, eW0) <= TOL


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("W0,relu", [(True, False), (False, False), (True, True), (False, True)])
def test_rgcn_backward_small(kind, W0, relu):
    g = graph(kind, E=3000)
    t = workloads.tiny_tensors(31, g, 64, 64)
    w0 = t["W0"] if W0 else None
    print(f"rgcn backward {kind} W0={W0} relu={relu}", flush=True)
    # the ReLU derivative is read from the oracle's forward output, so both
    # sides take the same mask
    out = oracle.rgcn_forward(g, t["h"], t["W"], w0, relu=True) if relu else None
    run = Runner(g, t)
    gh, gW, gW0 = run.rgcn_backward(W0=W0, relu=relu, out=out)
    run.close()
    dh, dW, dW0 = oracle.rgcn_backward(g, t["h"], t["W"], w0, t["grad_out"], relu=relu)
    assert row_err(gh, dh) <= TOL
    assert row_err(gW.reshape(-1, 64), dW.reshape(-1, 64)) <= TOL
    if W0:
        assert row_err(gW0, dW0) <= TOL


def test_rgcn_backward_after_forward():
    """Forward then backward through this library (the mask from its own output)."""
    g = graph("hub", seed=32, E=3000)
    t = workloads.tiny_tensors(32, g, 64, 64)
    print("rgcn forward + backward", flush=True)
    run = Runner(g, t)
    gh, gW, gW0 = run.rgcn_backward(W0=True, relu=True)
    run.close()
    dh, dW, dW0 = oracle.rgcn_backward(g, t["h"], t["W"], t["W0"], t["grad_out"], relu=True)
    assert row_err(gh, dh) <= TOL
    assert row_err(gW.reshape(-1, 64), dW.reshape(-1, 64)) <= TOL
    assert row_err(gW0, dW0) <= TOL


def check_hgt_grads(got, ref, heads, d=64):
    dk = d // heads
    assert row_err(got["dh"], ref["dh"]) <= TOL
    for k in ("dWk", "dWq", "dWv", "dWa"):
        if ref[k] is None:
            continue
        assert row_err(got[k].reshape(-1, d), ref[k].reshape(-1, d)) <= TOL, k
    for k in ("dWatt", "dWmsg"):
        assert row_err(got[k].reshape(-1, dk), ref[k].reshape(-1, dk)) <= TOL, k
    assert row_err(got["dmu"].reshape(1, -1), ref["dmu"].reshape(1, -1)) <= TOL


def hgt_case(kind, heads, seed, flags=None, R=7, T=4, E=4000, scale=None):
    g = graph(kind, seed=seed, T=T, R=R, E=E)
    t = workloads.tiny_tensors(seed, g, 64, 64, heads=heads)
    t["mu"] = (1.0 + 0.25 * np.arange(R)).astype(np.float32)   # distinct priors
    scale = 1.0 / np.sqrt(64 // heads) if scale is None else scale
    return g, t, scale


@pytest.mark.parametrize("use_saved", [False, True])
@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("heads", [1, 2, 4])
def test_hgt_backward_small(kind, heads, use_saved):
    g, t, scale = hgt_case(kind, heads, 33)
    print(f"hgt backward {kind} heads={heads} saved={use_saved}", flush=True)
    run = Runner(g, t)
    got = run.hgt_backward(heads, scale, use_saved=use_saved)
    run.close()
    ref = oracle.hgt_backward(g, t["h"], t["Wk"], t["Wq"], t["Wv"], t["Wa"], t["Watt"], t["Wmsg"],
                              t["mu"], t["grad_out"], heads=heads, att_scale=scale)
    check_hgt_grads(got, ref, heads)


@pytest.mark.parametrize("use_saved", [False, True])
@pytest.mark.parametrize("kind", ["random", "hub", "dups", "empty"])
@pytest.mark.parametrize("d,heads", [(32, 1), (32, 2), (128, 2), (128, 8)])
def test_hgt_backward_hidden_sizes(kind, d, heads, use_saved):
    g = graph(kind, T=4, R=7, E=3000)
    t = workloads.tiny_tensors(53, g, d, d, heads=heads)
    t["mu"] = (1.0 + 0.25 * np.arange(7)).astype(np.float32)   # distinct priors
    scale = 1.0 / np.sqrt(d // heads)
    print(f"hgt backward d={d} heads={heads} {kind} saved={use_saved}", flush=True)
    run = Runner(g, t)
    got = run.hgt_backward(heads, scale, use_saved=use_saved)
    run.close()
    ref = oracle.hgt_backward(g, t["h"], t["Wk"], t["Wq"], t["Wv"], t["Wa"], t["Watt"], t["Wmsg"],
                              t["mu"], t["grad_out"], heads=heads, att_scale=scale)
    check_hgt_grads(got, ref, heads, d)


@pytest.mark.parametrize("use_saved", [False, True])
@pytest.mark.parametrize("kind", ["typed", "typedhub"])
@pytest.mark.parametrize("d,heads", [(32, 2), (64, 4), (128, 8)])
def test_hgt_backward_typed_relations(kind, d, heads, use_saved):
    """Typed relations: the backward recomputes the folded segment queries the
    forward used, so the saved statistics match its scores."""
    g = graph(kind, T=4, R=7, E=3000)
    t = workloads.tiny_tensors(57, g, d, d, heads=heads)
    t["mu"] = (1.0 + 0.25 * np.arange(7)).astype(np.float32)
    scale = 1.0 / np.sqrt(d // heads)
    print(f"hgt backward typed d={d} heads={heads} {kind} saved={use_saved}", flush=True)
    run = Runner(g, t)
    got = run.hgt_backward(heads, scale, use_saved=use_saved)
    run.close()
    ref = oracle.hgt_backward(g, t["h"], t["Wk"], t["Wq"], t["Wv"], t["Wa"], t["Watt"], t["Wmsg"],
                              t["mu"], t["grad_out"], heads=heads, att_scale=scale)
    check_hgt_grads(got, ref, heads, d)


@pytest.mark.parametrize("use_saved", [False, True])
@pytest.mark.parametrize("flags", [0, 2, 4])
def test_hgt_backward_flags(flags, use_saved):
    g, t, scale = hgt_case("hub", 4, 34, R=3, T=2)
    print(f"hgt backward flags={flags} saved={use_saved}", flush=True)
    run = Runner(g, t)
    got = run.hgt_backward(4, 0.3, flags=flags, use_saved=use_saved)
    run.close()
    ref = oracle.hgt_backward(g, t["h"], t["Wk"], t["Wq"], t["Wv"], t["Wa"], t["Watt"], t["Wmsg"],
                              t["mu"], t["grad_out"], heads=4, att_scale=0.3,
                              residual=bool(flags & 2), a_linear=bool(flags & 4))
    check_hgt_grads(got, ref, 4)
    if not flags & 4:
        assert got["dWa"] is None


@pytest.mark.parametrize("heads,R", [(2, 12), (4, 24)])
def test_hgt_backward_many_relations(heads, R):
    g, t, scale = hgt_case("random", heads, 35, R=R, T=3, E=5000)
    print(f"hgt backward heads={heads} R={R}", flush=True)
    run = Runner(g, t)
    got = run.hgt_backward(heads, scale)
    run.close()
    ref = oracle.hgt_backward(g, t["h"], t["Wk"], t["Wq"], t["Wv"], t["Wa"], t["Watt"], t["Wmsg"],
                              t["mu"], t["grad_out"], heads=heads, att_scale=scale)
    check_hgt_grads(got, ref, heads)


@pytest.mark.parametrize("kind", ["random", "hub", "isolated", "empty"])
@pytest.mark.parametrize("d,heads", [(64, 4), (128, 8), (32, 2)])
def test_hgt_forward_saved_statistics(kind, d, heads):
    """The forward's optional softmax statistics: the output is the same with
    and without them; per destination and head, the maximum is the largest
    logit (a_e of the layer's definition, formed here in fp64 from the same
    inputs) and the sum is sum_e exp(a_e - max); (0, 0) without in-edges."""
    g = graph(kind, T=4, R=7, E=3000)
    t = workloads.tiny_tensors(54, g, d, d, heads=heads)
    t["mu"] = (1.0 + 0.25 * np.arange(7)).astype(np.float32)
    scale = 1.0 / np.sqrt(d // heads)
    print(f"hgt forward saved d={d} heads={heads} {kind}", flush=True)
    run = Runner(g, t)
    plain = run.hgt(heads, scale)
    out, saved = run.hgt(heads, scale, want_saved=True)
    sv = saved.cpu().numpy()
    run.close()
    np.testing.assert_array_equal(out, plain)
    # logits of the definition: (K_s,i Watt[r,i]) . Q_t,i * mu[r] * scale
    dk = d // heads
    h = t["h"].astype(np.float64)
    nt = g["ntype"]
    K = np.einsum("nd,nde->ne", h, t["Wk"].astype(np.float64)[nt]).reshape(-1, heads, dk)
    Q = np.einsum("nd,nde->ne", h, t["Wq"].astype(np.float64)[nt]).reshape(-1, heads, dk)
    src, dst, rel = g["src"], g["dst"], g["rel"]
    KW = np.einsum("ehk,ehkl->ehl", K[src], t["Watt"].astype(np.float64)[rel])
    a = (KW * Q[dst]).sum(-1) * t["mu"].astype(np.float64)[rel][:, None] * scale   # [E, heads]
    M = np.full((g["N"], heads), -np.inf)
    np.maximum.at(M, dst, a)
    Z = np.zeros((g["N"], heads))
    np.add.at(Z, dst, np.exp(a - M[dst]))
    has = np.bincount(dst, minlength=g["N"]) > 0
    assert np.all(sv[~has] == 0)
    np.testing.assert_allclose(sv[has, :, 0], M[has], rtol=1e-5, atol=1e-5)
    np.testing.assert_allclose(sv[has, :, 1], Z[has], rtol=1e-4)


@pytest.mark.parametrize("kind", ["random", "hub", "dups", "empty"])
@pytest.mark.parametrize("heads", [1, 2])
def test_rgat_ablation_plans(kind, heads):
    """Transform-first with and without compact materialization (graph flag)
    and with and without linear operator reordering of the destination term
    and with the attention term carried in the message rows all give the
    layer's output."""
    g = graph(kind, seed=37)
    t = workloads.tiny_tensors(37, g, 64, 64, heads=heads, att_var=1.0)
    ref = oracle.rgat_forward(g, t["h"], t["W"], t["w_src"], t["w_dst"], heads=heads)
    for compact in (True, False):
        print(f"rgat ablation {kind} heads={heads} compact={compact}", flush=True)
        run = Runner(g, t, compact=compact)
        if not compact:
            assert run.G.info()["num_src_pairs"] == g["E"]
        for plan in (1, 3, 4):
            assert row_err(run.rgat(heads=heads, plan=plan), ref) <= TOL, (compact, plan)
        run.close()


@pytest.mark.parametrize("kind", ["random", "hub"])
def test_rgcn_without_compaction(kind):
    g = graph(kind, seed=38)
    t = workloads.tiny_tensors(38, g, 64, 64)
    print(f"rgcn no compaction {kind}", flush=True)
    run = Runner(g, t, compact=False)
    got = run.rgcn(plan=1)
    run.close()
    assert row_err(got, oracle.rgcn_forward(g, t["h"], t["W"], t["W0"])) <= TOL


def test_forward_bitwise_deterministic():
    g = graph("hub", seed=12)
    t = workloads.tiny_tensors(12, g, 64, 64, heads=4, att_var=1.0)
    print("determinism", flush=True)
    run = Runner(g, t)
    for fn in (lambda: run.rgcn(plan=1), lambda: run.rgcn(plan=2), lambda: run.rgat(plan=1),
               lambda: run.rgat(plan=2), lambda: run.hgt(4, 0.25)):
        a, b = fn(), fn()
        assert np.array_equal(a, b)
    run.close()


def test_plans_agree():
    g = graph("dups", seed=13)
    t = workloads.tiny_tensors(13, g, 64, 64, att_var=1.0)
    print("plans agree", flush=True)
    run = Runner(g, t)
    for fn in (run.rgcn, run.rgat):
        a, b = fn(plan=1), fn(plan=2)
        assert row_err(a, b.astype(np.float64)) <= 1e-5
    run.close()
