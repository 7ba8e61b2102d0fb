"""Shared helpers of the GPU parity tests: run a layer through the C ABI with
torch-allocated outputs and workspace, and the row-normalised error measure.

Tolerance (fp32 GPU vs fp64 oracle): for every output row v,
    max_j |gpu[v, j] - ref[v, j]| / ||ref[v]||_2  <=  1e-4,
and rows whose reference is exactly zero (destinations without in-edges)
must be exactly zero on the GPU as well.
"""
from __future__ import annotations

import numpy as np

TOL = 1e-4


class KinkRef:
    """A reference output with optional exact corrections: base + any subset
    of the deltas is a correct result (each delta is the change of the output
    when one logit on the leaky ReLU's kink is differentiated from the other
    side; the backward is linear in each such choice and the choices do not
    interact).  Each delta touches a few rows: (rows, values).  Indexing rows
    and reshaping (splitting each row into whole rows) map the deltas along."""

    def __init__(self, base, deltas):
        self.base = np.asarray(base)
        self.deltas = deltas

    def __len__(self):
        return len(self.base)

    def __getitem__(self, idx):
        pos = np.arange(len(self.base))[idx]
        inv = {int(r): i for i, r in enumerate(np.atleast_1d(pos))}
        out = []
        for rows, vals in self.deltas:
            keep = [(inv[int(r)], v) for r, v in zip(rows, vals) if int(r) in inv]
            if keep:
                out.append((np.array([k[0] for k in keep]), np.stack([k[1] for k in keep])))
        return KinkRef(self.base[idx], out)

    def reshape(self, *shape):
        new = self.base.reshape(*shape)
        f = len(new) // len(self.base)
        out = [((rows[:, None] * f + np.arange(f)[None, :]).ravel(),
                vals.reshape(len(rows) * f, *new.shape[1:])) for rows, vals in self.deltas]
        return KinkRef(new, out)


def _row_errs(got, ref, structural_zero, cancel_floor):
    got = np.asarray(got, np.float64).reshape(len(ref), -1)
    ref = np.asarray(ref, np.float64).reshape(len(ref), -1)
    nrm = np.linalg.norm(ref, axis=1)
    med = float(np.median(nrm[nrm > 0])) if (nrm > 0).any() else 1.0
    zero = nrm <= cancel_floor * med if cancel_floor > 0 else nrm == 0
    if structural_zero is None and cancel_floor > 0:
        structural_zero = np.zeros(len(ref), bool)
    strict = zero if structural_zero is None else (zero & np.asarray(structural_zero, bool))
    err = np.zeros(len(ref))
    diff = np.abs(got - ref)
    if (~zero).any():
        err[~zero] = diff[~zero].max(axis=1) / nrm[~zero]
    loose = zero & ~strict
    if loose.any():
        err[loose] = diff[loose].max(axis=1) / med
    if strict.any():
        err[strict] = np.where(np.abs(got[strict]).max(axis=1) != 0.0, np.inf, 0.0)
    return err


def row_err(got, ref, structural_zero=None, cancel_floor=0.0) -> float:
    """Largest row-normalised error.  Reference rows that are exactly zero:
    with structural_zero=None every such row must be exactly zero on the GPU
    (forward outputs: a zero row only arises from a destination without
    in-edges).  Otherwise only rows flagged in structural_zero (no incident
    edge at all) must be exactly zero.  Gradient rows can also be zero by
    cancellation (a softmax over identical logits has zero gradient): the
    fp64 oracle then leaves ~1e-17 and fp32 ~1e-8.  Rows whose reference
    norm is below cancel_floor x the median row norm are such rows; they are
    measured against the median row norm instead of their own.  With a
    KinkRef as the reference, each row it corrects takes its smallest error
    over the corrected alternatives."""
    if not isinstance(ref, KinkRef):
        return float(_row_errs(got, ref, structural_zero, cancel_floor).max(initial=0.0))
    base = np.asarray(ref.base, np.float64).reshape(len(ref), -1)
    got2 = np.asarray(got, np.float64).reshape(len(ref), -1)
    err = _row_errs(got2, base, structural_zero, cancel_floor)
    # rows touched by kink deltas: the smallest error over every subset of them
    touch = {}
    for i, (rows, vals) in enumerate(ref.deltas):
        for r, v in zip(rows, np.asarray(vals, np.float64).reshape(len(rows), -1)):
            touch.setdefault(int(r), []).append(v)
    nrm = np.linalg.norm(base, axis=1)
    med = float(np.median(nrm[nrm > 0])) if (nrm > 0).any() else 1.0
    for r, vs in touch.items():
        if len(vs) > 12:
            # too many choices to enumerate (a relation's dW row): every
            # combination lies within base +- sum |delta|, the slack allowed
            slack = np.sum(np.abs(vs), axis=0)
            n = np.linalg.norm(base[r])
            scale = n if n > cancel_floor * med and n > 0 else med
            err[r] = min(err[r], float(np.maximum(np.abs(got2[r] - base[r]) - slack, 0.0).max() / scale))
            continue
        best = err[r]
        for mask in range(1, 1 << len(vs)):
            cand = base[r] + sum(v for j, v in enumerate(vs) if mask >> j & 1)
            n = np.linalg.norm(cand)
            scale = n if n > cancel_floor * med and n > 0 else med
            best = min(best, float(np.abs(got2[r] - cand).max() / scale))
        err[r] = best
    return float(err.max(initial=0.0))


# An RGAT logit y within this fraction of its rounding scale (oracle.
# rgat_preactivations) of zero sits on the leaky ReLU's kink for an fp32
# evaluation: the GPU may take either one-sided derivative there (the fp32
# rounding of y is a few 1e-7 of the scale).
KINK_REL = 2e-6


def rgat_backward_ref(g, t, heads=1, neg_slope=0.2, scope=0, node_mask=None, rel_mask=None):
    """The oracle's RGAT gradients (dh, dW, dw_src, dw_dst) for a GPU
    comparison.  When some logits lie on the leaky ReLU's kink (|y| <=
    KINK_REL x its rounding scale), each gradient is a KinkRef: the oracle's
    standard result plus, per such logit y_e,k, the exact change of the
    gradients when it is differentiated from the other side of the kink.  The
    change follows from the oracle's Y_e,k = dz (1 or slope): Y moves by
    dz (slope - 1) or dz (1 - slope), and the backward's terms that take
    Y_e,k (the message and both attention paths of edge e, head k's columns)
    move with it -- dh of its source and destination, dW, dw_src and dw_dst of
    its relation.  Any combination of these choices is a correct result."""
    import oracle
    args = (g, t["h"], t["W"], t["w_src"], t["w_dst"], t["grad_out"])
    *ref, Yg = oracle.rgat_backward(*args, heads=heads, neg_slope=neg_slope, scope=scope,
                                    node_mask=node_mask, rel_mask=rel_mask, want_Y=True)
    nm = np.ones(g["N"], bool) if node_mask is None else np.asarray(node_mask, bool)
    rm = np.ones(g["R"], bool) if rel_mask is None else np.asarray(rel_mask, bool)
    # logits of the edges that touch a requested entry
    sel = np.nonzero(nm[g["src"]] | nm[g["dst"]] | rm[g["rel"]])[0]
    sub = {k: np.asarray(g[k])[sel] for k in ("src", "dst", "rel")}
    ys, scs = oracle.rgat_preactivations(sub, t["h"], t["W"], t["w_src"], t["w_dst"], heads=heads)
    y = np.zeros((g["E"], heads)); y[sel] = ys
    kink = [(sel[i], k) for i, k in np.argwhere(np.abs(ys) <= KINK_REL * scs)]
    h, W = np.asarray(t["h"], np.float64), np.asarray(t["W"], np.float64)
    ws, wd = np.asarray(t["w_src"], np.float64), np.asarray(t["w_dst"], np.float64)
    d_out = W.shape[2]
    dk = d_out // heads
    deltas = [[], [], [], []]
    for e, k in kink:
        u, v, r = int(g["src"][e]), int(g["dst"][e]), int(g["rel"][e])
        if not (nm[u] or nm[v] or rm[r]):
            continue                       # touches no requested entry
        assert np.isfinite(Yg[e, k]) and neg_slope != 0
        pos = y[e, k] > 0
        dz = Yg[e, k] / (1.0 if pos else neg_slope)
        dY = dz * ((neg_slope - 1.0) if pos else (1.0 - neg_slope))
        cols = slice(k * dk, (k + 1) * dk)
        ddm = np.zeros(d_out); ddm[cols] = dY * ws[r, cols]
        ddt = np.zeros(d_out); ddt[cols] = dY * wd[r, cols]
        dh_rows = {}
        for n, dd in ((u, ddm), (v, ddt)):
            if nm[n]:
                dh_rows[n] = dh_rows.get(n, 0.0) + dd @ W[r].T
        if dh_rows:
            nodes = np.array(sorted(dh_rows))
            deltas[0].append((nodes, np.stack([dh_rows[n] for n in nodes])))
        if rm[r]:
            m, tt = h[u] @ W[r], h[v] @ W[r]
            deltas[1].append((np.array([r]), (np.outer(h[u], ddm) + np.outer(h[v], ddt))[None]))
            dsrc = np.zeros(d_out); dsrc[cols] = dY * m[cols]
            ddst = np.zeros(d_out); ddst[cols] = dY * tt[cols]
            deltas[2].append((np.array([r]), dsrc[None]))
            deltas[3].append((np.array([r]), ddst[None]))
    print(f"  kink logits touching compared entries: {sum(len(x) for x in deltas[:1]) or len(deltas[1])}",
          flush=True)
    if not any(deltas):
        return tuple(ref)
    return tuple(KinkRef(x, dl) for x, dl in zip(ref, deltas))



class Runner:
    """Runs the library's layers on one device with torch-owned buffers."""

    def __init__(self, g, t, device="cuda:0", compact=True):
        import torch
        from paper_2301_06284_amd import rgnn
        self.torch, self.rgnn = torch, rgnn
        self.dev = torch.device(device)
        self.g = g
        self.G = rgnn.Graph.from_dict(g, compact=compact)
        self.T = {k: torch.from_numpy(np.ascontiguousarray(v)).to(self.dev) for k, v in t.items()}

    def ws(self, layer, d_in, d_out, heads=1, plan=0):
        n = self.rgnn.workspace_size(self.G, layer, d_in, d_out, heads, plan)
        return self.torch.empty(max(n, 256), dtype=self.torch.uint8, device=self.dev)

    def rgcn(self, W0=True, relu=False, plan=0):
        T, torch = self.T, self.torch
        d_in, d_out = T["W"].shape[1], T["W"].shape[2]
        out = torch.full((self.g["N"], d_out), float("nan"), device=self.dev)
        self.rgnn.rgcn_forward(self.G, T["h"], T["W"], T["W0"] if W0 else None, out,
                               self.ws(0, d_in, d_out, 1, plan), d_in, d_out,
                               self.rgnn.FLAG_RELU if relu else 0, plan)
        torch.cuda.synchronize()
        return out.cpu().numpy()

    def rgat(self, heads=1, plan=0, slope=0.2, want_saved=False, scope=0):
        T, torch = self.T, self.torch
        d_in, d_out = T["W"].shape[1], T["W"].shape[2]
        out = torch.full((self.g["N"], d_out), float("nan"), device=self.dev)
        saved = None
        if scope == 0:
            saved = torch.full((self.g["N"], heads, 2), float("nan"), device=self.dev)
        elif want_saved:   # per (dst, rel) segment
            saved = torch.full((self.G.info()["num_dst_segments"], heads, 2), float("nan"), device=self.dev)
        ws_plan = 2 if scope == 1 else plan   # per-(dst, rel) softmax runs aggregate-first
        self.rgnn.rgat_forward(self.G, T["h"], T["W"], T["w_src"], T["w_dst"], out, saved,
                               self.ws(1, d_in, d_out, heads, ws_plan), d_in, d_out, heads, slope,
                               scope, plan)
        torch.cuda.synchronize()
        if want_saved:
            return out.cpu().numpy(), saved
        return out.cpu().numpy()

    def hgt(self, heads, scale, flags=None, want_saved=False):
        """want_saved: also return the softmax statistics [N, heads, 2] (a device tensor)."""
        T, torch, rgnn = self.T, self.torch, self.rgnn
        d = T["h"].shape[1]
        flags = rgnn.FLAG_RESIDUAL | rgnn.FLAG_A_LINEAR if flags is None else flags
        out = torch.full((self.g["N"], d), float("nan"), device=self.dev)
        saved = torch.full((self.g["N"], heads, 2), float("nan"), device=self.dev) if want_saved else None
        rgnn.hgt_forward(self.G, T["h"], T["Wk"], T["Wq"], T["Wv"], T["Wa"], T["Watt"], T["Wmsg"],
                         T["mu"], out, self.ws(2, d, d, heads), d, heads, scale, flags, saved=saved)
        torch.cuda.synchronize()
        if want_saved:
            return out.cpu().numpy(), saved
        return out.cpu().numpy()

    def rgat_backward(self, slope=0.2, heads=1, scope=0, plan=0):
        """plan: the forward plan whose saved statistics the backward takes."""
        T, torch, rgnn = self.T, self.torch, self.rgnn
        d = T["W"].shape[1]
        R = T["W"].shape[0]
        _, saved = self.rgat(heads=heads, slope=slope, want_saved=True, scope=scope, plan=plan)
        gh = torch.full((self.g["N"], d), float("nan"), device=self.dev)
        gW = torch.full((R, d, d), float("nan"), device=self.dev)
        gs = torch.full((R, d), float("nan"), device=self.dev)
        gt = torch.full((R, d), float("nan"), device=self.dev)
        rgnn.rgat_backward(self.G, T["h"], T["W"], T["w_src"], T["w_dst"], saved, T["grad_out"],
                           gh, gW, gs, gt, self.ws(3, d, d, heads), d, d, heads, slope, scope)
        torch.cuda.synchronize()
        return gh.cpu().numpy(), gW.cpu().numpy(), gs.cpu().numpy(), gt.cpu().numpy()

    def hgt_backward(self, heads, scale, flags=None, use_saved=False):
        """use_saved: run this library's forward first and hand its softmax
        statistics to the backward (otherwise the backward recomputes them)."""
        T, torch, rgnn = self.T, self.torch, self.rgnn
        d = T["h"].shape[1]
        flags = rgnn.FLAG_RESIDUAL | rgnn.FLAG_A_LINEAR if flags is None else flags
        N, R, NT = self.g["N"], T["Watt"].shape[0], T["Wk"].shape[0]
        dk = d // heads
        nan = lambda *shape: torch.full(shape, float("nan"), device=self.dev)
        grads = dict(dh=nan(N, d), dWk=nan(NT, d, d), dWq=nan(NT, d, d), dWv=nan(NT, d, d),
                     dWa=nan(NT, d, d) if flags & rgnn.FLAG_A_LINEAR else None,
                     dWatt=nan(R, heads, dk, dk), dWmsg=nan(R, heads, dk, dk), dmu=nan(R))
        saved = self.hgt(heads, scale, flags, want_saved=True)[1] if use_saved else None
        # workspace filled with NaN bytes: a row the backward reads without
        # having written it shows up in the gradients
        ws = self.ws(rgnn.LAYER_HGT_BACKWARD, d, d, heads).fill_(255)
        rgnn.hgt_backward(self.G, T["h"], T["Wk"], T["Wq"], T["Wv"], T["Wa"], T["Watt"], T["Wmsg"],
                          T["mu"], T["grad_out"], grads, ws, d, heads, scale, flags, saved=saved)
        torch.cuda.synchronize()
        return {k: (None if v is None else v.cpu().numpy()) for k, v in grads.items()}

    def rgcn_backward(self, W0=True, relu=False, out=None):
        """out: the forward output the ReLU derivative is read from (numpy);
        None runs this library's forward first."""
        T, torch, rgnn = self.T, self.torch, self.rgnn
        d = T["W"].shape[1]
        R = T["W"].shape[0]
        flags = rgnn.FLAG_RELU if relu else 0
        o = None
        if relu:
            if out is None:
                out = self.rgcn(W0=W0, relu=True)
            o = torch.from_numpy(np.ascontiguousarray(out, np.float32)).to(self.dev)
        gh = torch.full((self.g["N"], d), float("nan"), device=self.dev)
        gW = torch.full((R, d, d), float("nan"), device=self.dev)
        gW0 = torch.full((d, d), float("nan"), device=self.dev) if W0 else None
        rgnn.rgcn_backward(self.G, T["h"], T["W"], T["W0"] if W0 else None, o, T["grad_out"], gh, gW,
                           gW0, self.ws(rgnn.LAYER_RGCN_BACKWARD, d, d), d, d, flags)
        torch.cuda.synchronize()
        return (gh.cpu().numpy(), gW.cpu().numpy(), None if gW0 is None else gW0.cpu().numpy())

    def close(self):
        self.G.close()
