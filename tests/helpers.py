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


def row_err(got, ref, structural_zero=None, cancel_floor=0.0) -> float:
    """Largest row-normalised error.  Reference rows that are exactly zero:
    with structural_zero=None every such row must be exactly zero on the GPU
    (forward outputs: a zero row only arises from a destination without
    in-edges).  Otherwise only rows flagged in structural_zero (no incident
    edge at all) must be exactly zero.  Gradient rows can also be zero by
    cancellation (a softmax over identical logits has zero gradient): the
    fp64 oracle then leaves ~1e-17 and fp32 ~1e-8.  Rows whose reference
    norm is below cancel_floor x the median row norm are such rows; they are
    measured against the median row norm instead of their own."""
    got = np.asarray(got, np.float64).reshape(len(ref), -1)
    ref = np.asarray(ref, np.float64).reshape(len(ref), -1)
    nrm = np.linalg.norm(ref, axis=1)
    med = float(np.median(nrm[nrm > 0])) if (nrm > 0).any() else 1.0
    zero = nrm <= cancel_floor * med if cancel_floor > 0 else nrm == 0
    if structural_zero is None and cancel_floor > 0:
        structural_zero = np.zeros(len(ref), bool)
    strict = zero if structural_zero is None else (zero & np.asarray(structural_zero, bool))
    if strict.any() and np.abs(got[strict]).max(initial=0.0) != 0.0:
        return float("inf")
    err = 0.0
    if (~zero).any():
        err = float((np.abs(got - ref)[~zero].max(axis=1) / nrm[~zero]).max())
    loose = zero & ~strict
    if loose.any():
        err = max(err, float(np.abs(got[loose] - ref[loose]).max() / med))
    return err


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
