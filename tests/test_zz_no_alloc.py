"""rgat_forward_noalloc (the RGAT forward with its workspace in the library's
static device scratch) against rgat_forward with a caller workspace, through
the C ABI: two calls in a row, the second on a smaller graph, both plans and
both softmax scopes; every output and saved statistic bit for bit (both
calls run the same kernels on the same inputs), and the outputs within the
oracle tolerance.  A graph whose workspace exceeds the scratch is rejected
before anything is enqueued."""
import numpy as np
import pytest

import oracle
import workloads
from helpers import TOL, row_err

pytestmark = pytest.mark.gpu


def run_both(g, t, heads, plan, scope):
    import torch
    from paper_2301_06284_amd import rgnn
    dev = torch.device("cuda:0")
    G = rgnn.Graph.from_dict(g)
    T = {k: torch.from_numpy(np.ascontiguousarray(v)).to(dev) for k, v in t.items()}
    d = T["W"].shape[2]
    nsaved = g["N"] if scope == 0 else G.info()["num_dst_segments"]
    res = []
    for noalloc in (False, True):
        out = torch.full((g["N"], d), float("nan"), device=dev)
        saved = torch.full((nsaved, heads, 2), float("nan"), device=dev)
        if noalloc:
            rgnn.rgat_forward_noalloc(G, T["h"], T["W"], T["w_src"], T["w_dst"], out, saved, d, d, heads,
                                      0.2, scope, plan)
        else:
            n = rgnn.workspace_size(G, rgnn.LAYER_RGAT, d, d, heads, 2 if scope == 1 else plan)
            ws = torch.empty(max(n, 256), dtype=torch.uint8, device=dev)
            rgnn.rgat_forward(G, T["h"], T["W"], T["w_src"], T["w_dst"], out, saved, ws, d, d, heads,
                              0.2, scope, plan)
        torch.cuda.synchronize()
        res.append((out.cpu().numpy(), saved.cpu().numpy()))
    G.close()
    return res


@pytest.mark.parametrize("heads,plan,scope", [(1, 0, 0), (1, 1, 0), (1, 2, 0), (4, 1, 0), (1, 0, 1), (2, 0, 1)])
def test_noalloc_matches_workspace_call(heads, plan, scope):
    sizes = [(20000, 200000, "hub"), (3000, 30000, "random")]   # the second call on a smaller graph
    for N, E, kind in sizes:
        g = workloads.tiny_graph(81, N=N, E=E, R=12, T=2, kind=kind)
        t = workloads.tiny_tensors(81, g, 64, 64, heads=heads)
        print(f"noalloc N={N} E={E} heads={heads} plan={plan} scope={scope}", flush=True)
        (o1, s1), (o2, s2) = run_both(g, t, heads, plan, scope)
        np.testing.assert_array_equal(o2, o1)
        np.testing.assert_array_equal(s2, s1)
        ref = oracle.rgat_forward(g, t["h"], t["W"], t["w_src"], t["w_dst"], heads=heads, scope=scope)
        assert row_err(o2, ref) <= TOL


def test_noalloc_rejects_graph_beyond_scratch():
    import torch
    from paper_2301_06284_amd import rgnn
    g = workloads.tiny_graph(82, N=400000, E=800000, R=96, T=2, kind="random")
    t = workloads.tiny_tensors(82, g, 64, 64)
    dev = torch.device("cuda:0")
    G = rgnn.Graph.from_dict(g)
    assert rgnn.workspace_size(G, rgnn.LAYER_RGAT, 64, 64, 1, 0) > 64 << 20
    T = {k: torch.from_numpy(np.ascontiguousarray(v)).to(dev) for k, v in t.items()}
    out = torch.zeros(g["N"], 64, device=dev)
    with pytest.raises(rgnn.RgnnError) as e:
        rgnn.rgat_forward_noalloc(G, T["h"], T["W"], T["w_src"], T["w_dst"], out, None, 64, 64)
    assert e.value.status == rgnn.ERANGE and "scratch" in str(e.value)
    torch.cuda.synchronize()
    assert (out.cpu().numpy() == 0).all()   # nothing was enqueued
    G.close()
