"""Host check of the kink-aware RGAT gradient reference used by the GPU tests:
every combination of one-sided derivatives on the flagged logits is accepted,
a flip of an unflagged logit is not."""
import numpy as np

import helpers
import oracle
import workloads
from helpers import TOL, rgat_backward_ref, row_err


def test_kink_ref_accepts_flagged_flips_only(monkeypatch):
    g = workloads.tiny_graph(60, N=40, E=300, R=3, T=2, kind="random")
    t = workloads.tiny_tensors(60, g, 16, 16, heads=2, att_var=1.0)
    y, scale = oracle.rgat_preactivations(g, t["h"], t["W"], t["w_src"], t["w_dst"], heads=2)
    rel = np.abs(y) / scale
    # flag the three logits nearest the kink by widening the band to them
    order = np.argsort(rel, axis=None)
    monkeypatch.setattr(helpers, "KINK_REL", float(rel.ravel()[order[2]]) * (1 + 1e-9))
    ref = rgat_backward_ref(g, t, heads=2)
    args = (g, t["h"], t["W"], t["w_src"], t["w_dst"], t["grad_out"])
    flagged = [np.unravel_index(i, y.shape) for i in order[:3]]
    for subset in range(8):
        flip = np.zeros(y.shape, bool)
        for j in range(3):
            if subset >> j & 1:
                flip[flagged[j]] = True
        got = oracle.rgat_backward(*args, heads=2, kink_flip=flip)
        for a, b in zip(got, ref):
            assert row_err(a.reshape(len(a), -1), b.reshape(len(b), -1)) <= 1e-12
        # dW compared row by row of each relation's matrix, as the GPU tests do
        assert row_err(got[1].reshape(-1, 16), ref[1].reshape(-1, 16)) <= 1e-12
    # an unflagged logit differentiated from the wrong side is caught
    flip = np.zeros(y.shape, bool)
    flip[np.unravel_index(order[-1], y.shape)] = True
    got = oracle.rgat_backward(*args, heads=2, kink_flip=flip)
    assert max(row_err(a.reshape(len(a), -1), b.reshape(len(b), -1)) for a, b in zip(got, ref)) > TOL



def test_kink_ref_many_deltas_on_one_row():
    """More than twelve kink choices on one row: the row may lie anywhere
    within base +- the sum of the deltas' magnitudes, and not beyond."""
    from helpers import KinkRef
    rng = np.random.default_rng(3)
    base = rng.standard_normal((3, 8))
    deltas = [(np.array([1]), 1e-3 * rng.standard_normal((1, 8))) for _ in range(20)]
    ref = KinkRef(base, deltas)
    pick = base.copy()
    pick[1] += sum(d[1][0] for d in deltas[::3])
    assert row_err(pick, ref) <= 1e-12
    off = pick.copy()
    off[1, 0] += 25e-3 * 20
    assert row_err(off, ref) > TOL
