"""Benchmark of the RGNN layer hot path on one MI355X.

Headline (`value`): edges/s of one RGAT layer forward (all of its kernels:
reordered attention vectors, destination terms, the fused gather-transform
traversal or the typed GEMM and traversal, softmax statistics, reductions and
merges, per the plan the library selects) on the am-like
workload -- 880 000 nodes, 7 node types, 96 relations (Zipf 1.2), 5.7 M edges
(power-law in-degree, exponent 2.1), d = 64, one head -- with every input
resident in HBM.  One step = one layer forward; K steps are timed between two
device synchronisations, after W warm-up steps.  The line also carries:
  roofline      the dominant kernel's algorithmic bytes (or flops) per launch
                over its average duration, measured with hipEvents the library
                records around its own launches on the launch stream;
  cpu_baseline  the fp64 oracle timed on the host's cores on a bounded sample
                of destinations of the same workload;
  layers        edges/s of the other layers and workloads (RGCN, HGT, RGCN and
                RGAT at d = 128, RGAT, RGCN and HGT backward, both RGAT plans).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
FP32_PEAK_TFLOPS = 157.3
METRIC = "edges/sec per RGNN layer fwd (RGAT, HGT) on 1 MI355X; achieved HBM GB/s"


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    # 100 timed steps of the headline layer (~60 ms): a mean that a few slow
    # steps do not move
    p.add_argument("--steps", type=int, default=100)
    # the first ~30 ms of continuous work run slower (the device's clocks
    # ramp up): 50 warm-up steps of the headline layer cover that
    p.add_argument("--warmup", type=int, default=50)
    p.add_argument("--only", choices=["headline", "all"], default="all",
                   help="headline: time only the RGAT workload of the headline")
    p.add_argument("--no-cpu", action="store_true", help="skip the CPU baseline leg")
    p.add_argument("--sweep", action="store_true",
                   help="instead of the benchmark line: the optimization ablation (compact "
                        "materialization x linear operator reordering, and the fused "
                        "aggregate-first plan) for RGAT and RGCN at d = 64 and d = 128")
    p.add_argument("--calibrate-copy", action="store_true",
                   help="also run a 1 GiB device copy (reference for HBM byte counters)")
    p.add_argument("--cpu-seconds", type=float, default=12.0,
                   help="target wall time of the CPU-baseline sample")
    return p.parse_args()


class Ctx:
    def __init__(self, k):
        import torch
        import workloads
        from paper_2301_06284_amd import rgnn
        self.torch, self.rgnn, self.k = torch, rgnn, k
        self.dev = torch.device("cuda:0")
        self.g = workloads.make_graph(k)
        self.t = workloads.make_tensors(k, self.g, workloads.CONFIGS[k]["layers"][0])
        self.G = rgnn.Graph.from_dict(self.g)
        self.T = {n: torch.from_numpy(v).to(self.dev) for n, v in self.t.items()}
        self.info = self.G.info()

    def ws(self, layer, d_in, d_out, heads=1, plan=0):
        n = self.rgnn.workspace_size(self.G, layer, d_in, d_out, heads, plan)
        return self.torch.empty(max(n, 256), dtype=self.torch.uint8, device=self.dev)

    def close(self):
        self.G.close()
        self.T.clear()
        self.torch.cuda.empty_cache()


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def time_steps(torch, fn, steps, warmup, per_step=False):
    """Mean ms per step over `steps` timed steps (events on the current stream,
    which the library launches on); with per_step, also the list of step times."""
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    ev[0].record()
    for i in range(steps):
        fn()
        ev[i + 1].record()
    torch.cuda.synchronize()
    each = [ev[i].elapsed_time(ev[i + 1]) for i in range(steps)]
    mean = ev[0].elapsed_time(ev[steps]) / steps
    return (mean, each) if per_step else mean


def kernel_profile(rgnn, torch, fn, steps):
    """Per-kernel (launches, mean ms) from the library's own event pairs."""
    torch.cuda.synchronize()
    rgnn.profile_reset()
    rgnn.profile_enable(True)
    for _ in range(steps):
        fn()
    torch.cuda.synchronize()
    rgnn.profile_enable(False)
    prof = rgnn.profile_read()
    rgnn.profile_reset()
    return {k: (n // steps, ms / n) for k, (n, ms) in prof.items()}


# ---------------------------------------------------------------- algorithmic traffic
def rgat_tf_model(info, d, H):
    """Algorithmic bytes / flops per launch of the transform-first RGAT kernels.
    Gathered rows count once per edge, node rows once per node, index arrays once."""
    E, N, U, V = info["num_edges"], info["num_nodes"], info["num_src_pairs"], info["num_vsegs"]
    R, I = info["num_rels"], info["num_items"]
    return {
        # per pair: gather index, h row read, message row write; W_r once per relation
        "typed_gemm": dict(bytes=U * (4 + 4 * d + 4 * d) + R * 4 * d * d, flops=2.0 * U * d * d),
        # per edge: pair index, message row (the per-head source terms are formed
        # from it with w_src); per destination: output row, (max, sum) per head;
        # per segment: offset, relation and destination terms; per item:
        # descriptor and slot; w_src once per relation
        "rgat_traverse_tf": dict(bytes=E * (4 + 4 * d) + N * (4 * d + 8 * H + 4)
                                 + V * (8 + 4 * H) + I * 20 + R * d * 4,
                                 flops=E * (4.0 * d + 10 * H)),
    }


def single_segment_dsts(G):
    """Destinations whose in-edges form one virtual segment (one relation, at
    most chunk_edges edges): the fused kernel finishes them itself."""
    import numpy as np
    inf = G.info()
    dseg = np.diff(G.export("dst_segptr").astype(np.int64))
    sptr = G.export("seg_ptr").astype(np.int64)
    first = G.export("dst_segptr")[:-1].astype(np.int64)
    one = dseg == 1
    cnt = sptr[np.minimum(first + 1, len(sptr) - 1)] - sptr[np.minimum(first, len(sptr) - 1)]
    return int(np.count_nonzero(one & (cnt <= inf["chunk_edges"])))


def rgat_af_model(info, d, n_single=0):
    """Algorithmic bytes / flops per launch of the aggregate-first RGAT kernels.
    n_single: destinations with a single virtual segment, finished by the fused
    kernel (their output row and statistics replace the T row and (max, sum))."""
    E, N, V, R = info["num_edges"], info["num_nodes"], info["num_vsegs"], info["num_rels"]
    return {
        # per edge: source index and gathered h row; per segment: its table
        # entry, destination term, T row and (max, sum) written; W_r and
        # W_r w_src once per relation.  Flops: the segment transform on the
        # matrix cores plus the per-edge dot and weighted accumulation.
        "rgat_af_fused": dict(bytes=E * (4 + 4 * d) + V * (16 + 4 + 4 * d + 8) + R * (4 * d * d + 4 * d),
                              flops=2.0 * V * d * d + E * 4.0 * d),
        # all destinations (groups of lanes, and whole workgroups for hubs):
        # per segment T row and scale read, per destination offsets and output row
        "vseg_reduce": dict(bytes=V * (4 * d + 4) + N * (4 + 4 * d), flops=2.0 * V * d),
        # per segment T row, fused position and (max, sum); per destination
        # offsets, output row and saved (max, sum) -- except the segments and
        # rows of the destinations the fused kernel finished (offsets only)
        "softmax_reduce": dict(bytes=(V - n_single) * (4 * d + 4 + 8) + N * 4 + (N - n_single) * (4 * d + 8),
                               flops=2.0 * (V - n_single) * d),
        # per destination its h row (consecutive segments share it); per
        # segment its destination, relation and term written; W_r w_dst per relation
        "seg_attn": dict(bytes=N * 4 * d + V * 12 + R * 4 * d, flops=2.0 * V * d),
    }


def roofline_of(kernels, model):
    """Dominant kernel (largest time) among those with a traffic model."""
    best = None
    for name, (launches, ms) in kernels.items():
        if name in model and (best is None or ms * launches > best[1] * best[2]):
            best = (name, ms, launches)
    name, ms, _ = best
    m = model[name]
    gbs = m["bytes"] / (ms * 1e-3) / 1e9
    tfl = m["flops"] / (ms * 1e-3) / 1e12
    return name, ms, gbs, tfl, m


def counter_traffic(tag, kernel):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 counter
    summary (FETCH_SIZE + WRITE_SIZE, scaled by a copy of known size), or None
    when there is none or the kernel's source changed since it was taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"{tag}_hbm_counters.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))["kernels"].get(kernel)
    if not rec or not rec.get("source"):
        return None
    src = os.path.join(ROOT, rec["source"])
    if not os.path.exists(src) or hashlib.sha256(open(src, "rb").read()).hexdigest()[:16] != rec["source_sha256_16"]:
        return None
    return rec["bytes_per_launch"]


def cpu_baseline(ctx, target_s):
    import oracle
    g, t = ctx.g, ctx.t
    deg = np.bincount(g["dst"], minlength=g["N"])
    rng = np.random.default_rng(2301)
    order = rng.permutation(g["N"]).astype(np.int32)
    # calibrate on a small slice, then size the sample for ~target_s seconds
    probe = order[:5000]
    t0 = time.perf_counter()
    oracle.rgat_forward(g, t["h"], t["W"], t["w_src"], t["w_dst"], sel=probe)
    dt = time.perf_counter() - t0
    rate = max(1.0, deg[probe].sum()) / max(dt, 1e-6)
    want_edges = rate * target_s
    csum = np.cumsum(deg[order])
    n = int(min(len(order), max(5000, np.searchsorted(csum, want_edges) + 1)))
    sel = order[:n]
    t0 = time.perf_counter()
    oracle.rgat_forward(g, t["h"], t["W"], t["w_src"], t["w_dst"], sel=sel)
    dt = time.perf_counter() - t0
    edges = int(deg[sel].sum())
    return {"value": edges / dt, "unit": "edges/s", "cores": oracle.num_threads(), "kind": "oracle",
            "sample": (f"fp64 RGAT layer forward (edge-by-edge definition) for {n} random "
                       f"destinations of the 880000-node workload, {edges} in-edges, {dt:.1f} s")}


def sweep(args):
    """The analogue of the paper's optimization table and hidden-size curve on
    the synthetic graphs (the 880k-node graph at d = 32, 64, 128; the 2.5M-node
    graph at d = 128): per layer and hidden size, the ms per forward of
    transform-first without and
    with compact materialization (graph flag) and without and with linear
    operator reordering of the attention's destination term (RGAT plan 3 vs 1),
    with the attention term carried in the message rows (plan 4), and of the
    fused aggregate-first plan, with the plan the model selects."""
    import torch
    from paper_2301_06284_amd import rgnn
    torch.cuda.set_device(0)
    import workloads
    K, W = args.steps, args.warmup
    rows = []
    runs = [(2, d, "am_like_880k") for d in (32, 64, 128)] + [(4, 128, "wikikg2_like_2p5m")]
    c = Gn = None
    for wk, d, name in runs:
        log(f"sweep: workload {wk}, d = {d}")
        if c is None or c.k != wk:
            if c is not None:
                Gn.close()
                c.close()
            c = Ctx(wk)
            Gn = rgnn.Graph.from_dict(c.g, compact=False)
        # the hidden-size sweep: same graph, tensors of width d
        c.T = {n: torch.from_numpy(v).to(c.dev) for n, v in workloads.make_tensors(wk, c.g, "rgat", d).items()}
        E = c.info["num_edges"]
        out = torch.empty(c.info["num_nodes"], d, device=c.dev)
        for lname, layer in (("rgat", rgnn.LAYER_RGAT), ("rgcn", rgnn.LAYER_RGCN)):
            auto = rgnn.select_plan(c.G, layer, d, d, 1)[0]
            cases = [("vanilla", False, 3), ("compact", True, 3), ("reorder", False, 1),
                     ("compact+reorder", True, 1), ("compact+reorder, attention+message rows", True, 4),
                     ("aggregate-first fused", True, 2)]
            if layer == rgnn.LAYER_RGCN:
                cases = [("vanilla", False, 1), ("compact", True, 1), ("aggregate-first fused", True, 2)]
            for label, compact, plan in cases:
                G = c.G if compact else Gn
                ws = torch.empty(max(rgnn.workspace_size(G, layer, d, d, 1, plan), 256),
                                 dtype=torch.uint8, device=c.dev)
                if layer == rgnn.LAYER_RGAT:
                    fn = lambda: rgnn.rgat_forward(G, c.T["h"], c.T["W"], c.T["w_src"], c.T["w_dst"], out, None,
                                                   ws, d, d, 1, 0.2, 0, plan)
                else:
                    fn = lambda: rgnn.rgcn_forward(G, c.T["h"], c.T["W"], c.T["W0"], out, ws, d, d, 0, plan)
                ms = time_steps(torch, fn, K, W)
                rows.append({"workload": name, "d": d, "layer": lname, "variant": label,
                             "plan": plan, "compact": compact, "ms": round(ms, 4),
                             "edges_per_s": E / (ms * 1e-3), "auto_selects": plan == auto and compact})
                log(f"  {lname} {label}: {ms:.3f} ms")
                del ws
        if wk == 2:   # training: the backward passes at this width
            N2, R2 = c.info["num_nodes"], c.info["num_rels"]
            saved = torch.empty(N2, 1, 2, device=c.dev)
            ws = torch.empty(max(rgnn.workspace_size(c.G, rgnn.LAYER_RGAT, d, d, 1), 256), dtype=torch.uint8,
                             device=c.dev)
            rgnn.rgat_forward(c.G, c.T["h"], c.T["W"], c.T["w_src"], c.T["w_dst"], out, saved, ws, d, d)
            del ws
            Gd = torch.from_numpy(workloads.make_tensors(5, c.g, "rgat_bwd", d)["grad_out"]).to(c.dev)
            gh = torch.empty(N2, d, device=c.dev)
            gW, gs, gt, gW0 = (torch.empty(R2, d, d, device=c.dev), torch.empty(R2, d, device=c.dev),
                               torch.empty(R2, d, device=c.dev), torch.empty(d, d, device=c.dev))
            for lname, layer in (("rgat", rgnn.LAYER_RGAT_BACKWARD), ("rgcn", rgnn.LAYER_RGCN_BACKWARD)):
                ws = torch.empty(max(rgnn.workspace_size(c.G, layer, d, d, 1), 256), dtype=torch.uint8,
                                 device=c.dev)
                if lname == "rgat":
                    fn = lambda: rgnn.rgat_backward(c.G, c.T["h"], c.T["W"], c.T["w_src"], c.T["w_dst"], saved,
                                                    Gd, gh, gW, gs, gt, ws, d, d)
                else:
                    fn = lambda: rgnn.rgcn_backward(c.G, c.T["h"], c.T["W"], c.T["W0"], None, Gd, gh, gW, gW0,
                                                    ws, d, d, 0)
                ms = time_steps(torch, fn, K, W)
                rows.append({"workload": name, "d": d, "layer": lname, "variant": "backward", "ms": round(ms, 4),
                             "edges_per_s": E / (ms * 1e-3)})
                log(f"  {lname} backward: {ms:.3f} ms")
                del ws
            del saved, Gd, gh, gW, gs, gt, gW0
        del out
    Gn.close()
    c.close()
    # HGT on the 1.9M-node graph at d = 32, 64, 128 with d_k = 16 (2, 4, 8 heads)
    c = Ctx(3)
    E = c.info["num_edges"]
    for d in (32, 64, 128):
        H = d // 16
        log(f"sweep: workload 3, HGT d = {d}, {H} heads")
        c.T = {n: torch.from_numpy(v).to(c.dev) for n, v in workloads.make_tensors(3, c.g, "hgt", d, heads=H).items()}
        out = torch.empty(c.info["num_nodes"], d, device=c.dev)
        saved = torch.empty(c.info["num_nodes"], H, 2, device=c.dev)
        ws = torch.empty(max(rgnn.workspace_size(c.G, rgnn.LAYER_HGT, d, d, H), 256), dtype=torch.uint8,
                         device=c.dev)
        T = c.T
        fn = lambda: rgnn.hgt_forward(c.G, T["h"], T["Wk"], T["Wq"], T["Wv"], T["Wa"], T["Watt"], T["Wmsg"],
                                      T["mu"], out, ws, d, H, 0.25, rgnn.FLAG_RESIDUAL | rgnn.FLAG_A_LINEAR,
                                      saved=saved)
        ms = time_steps(torch, fn, K, W)
        rows.append({"workload": "mag_like_1p9m", "d": d, "layer": "hgt", "heads": H,
                     "variant": "reordered segment queries", "ms": round(ms, 4), "edges_per_s": E / (ms * 1e-3)})
        log(f"  hgt d={d}: {ms:.3f} ms")
        del ws
        # backward from the forward's softmax statistics
        Nn, R3, T3, dk = c.info["num_nodes"], c.info["num_rels"], c.info["num_ntypes"], d // H
        grads = dict(dh=torch.empty(Nn, d, device=c.dev),
                     **{k: torch.empty(T3, d, d, device=c.dev) for k in ("dWk", "dWq", "dWv", "dWa")},
                     dWatt=torch.empty(R3, H, dk, dk, device=c.dev), dWmsg=torch.empty(R3, H, dk, dk, device=c.dev),
                     dmu=torch.empty(R3, device=c.dev))
        ws = torch.empty(max(rgnn.workspace_size(c.G, rgnn.LAYER_HGT_BACKWARD, d, d, H), 256), dtype=torch.uint8,
                         device=c.dev)
        fb = lambda: rgnn.hgt_backward(c.G, T["h"], T["Wk"], T["Wq"], T["Wv"], T["Wa"], T["Watt"], T["Wmsg"],
                                       T["mu"], T["grad_out"], grads, ws, d, H, 0.25, saved=saved)
        ms = time_steps(torch, fb, K, W)
        rows.append({"workload": "mag_like_1p9m", "d": d, "layer": "hgt", "heads": H, "variant": "backward",
                     "ms": round(ms, 4), "edges_per_s": E / (ms * 1e-3)})
        log(f"  hgt backward d={d}: {ms:.3f} ms")
        del ws, out, grads, saved
    c.close()
    print(json.dumps({"sweep": rows}))


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the multi-GPU sharding "
              "of this path is a design note, not an implementation.", file=sys.stderr)
        sys.exit(2)
    if args.sweep:
        sweep(args)
        return
    import torch
    from paper_2301_06284_amd import rgnn
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    K, W = args.steps, args.warmup
    layers = {}

    # ------------------------------------------------ headline: RGAT forward, workload 2
    log("workload 2: generating and building the graph")
    c = Ctx(2)
    d, H = 64, 1
    inf = c.info
    plan, b_tf, b_af = rgnn.select_plan(c.G, rgnn.LAYER_RGAT, d, d, H)
    out = torch.empty(inf["num_nodes"], d, device=c.dev)
    saved = torch.empty(inf["num_nodes"], H, 2, device=c.dev)
    plans = {}
    other = rgnn.PLAN_AGGREGATE_FIRST if plan == rgnn.PLAN_TRANSFORM_FIRST else rgnn.PLAN_TRANSFORM_FIRST
    for p in ((plan,) if args.only == "headline" else (plan, other)):
        log(f"workload 2: RGAT forward plan {p}")
        ws = c.ws(rgnn.LAYER_RGAT, d, d, H, p)
        fn = (lambda ws=ws, p=p: rgnn.rgat_forward(c.G, c.T["h"], c.T["W"], c.T["w_src"],
                                                   c.T["w_dst"], out, saved, ws, d, d, H, 0.2,
                                                   0, p))
        ms, each = time_steps(torch, fn, K, W, per_step=True)
        # per-kernel durations: K more steps right after the timed ones, each
        # launch bracketed by the library's events (kept out of the timed steps,
        # whose time the event records would stretch)
        kern = kernel_profile(rgnn, torch, fn, K)
        plans[p] = (ms, kern, fn, each)
        del ws
    ms, kern, fn, each = plans[plan]
    model = (rgat_tf_model(inf, d, H) if plan == rgnn.PLAN_TRANSFORM_FIRST
             else rgat_af_model(inf, d, single_segment_dsts(c.G)))
    kname, kms, kgbs, ktfl, km = roofline_of(kern, model)
    E = inf["num_edges"]
    value = E / (ms * 1e-3)
    names = {1: "transform_first", 2: "aggregate_first"}
    if args.only == "all":
        # several heads (transform-first; the per-head source terms come from the
        # gathered message rows)
        log("workload 2: RGAT forward, 4 heads")
        ws4 = c.ws(rgnn.LAYER_RGAT, d, d, 4, rgnn.PLAN_TRANSFORM_FIRST)
        sv4 = torch.empty(inf["num_nodes"], 4, 2, device=c.dev)
        fn4 = lambda: rgnn.rgat_forward(c.G, c.T["h"], c.T["W"], c.T["w_src"], c.T["w_dst"], out, sv4, ws4,
                                        d, d, 4, 0.2, 0, rgnn.PLAN_TRANSFORM_FIRST)
        m4h = time_steps(torch, fn4, K, W)
        k4h = kernel_profile(rgnn, torch, fn4, max(3, K // 2))
        layers["rgat_fwd_am_like_880k_4heads"] = {"edges_per_s": inf["num_edges"] / (m4h * 1e-3), "ms": m4h,
                                                  "kernels_ms": {k: round(v[1], 4) for k, v in k4h.items()}}
        del ws4
        # the same with aggregate-first (one masked pass per head)
        ws4 = c.ws(rgnn.LAYER_RGAT, d, d, 4, rgnn.PLAN_AGGREGATE_FIRST)
        fn4a = lambda: rgnn.rgat_forward(c.G, c.T["h"], c.T["W"], c.T["w_src"], c.T["w_dst"], out, sv4, ws4,
                                         d, d, 4, 0.2, 0, rgnn.PLAN_AGGREGATE_FIRST)
        m4a = time_steps(torch, fn4a, K, W)
        layers["rgat_fwd_am_like_880k_4heads_aggregate_first"] = {"edges_per_s": inf["num_edges"] / (m4a * 1e-3),
                                                                  "ms": m4a}
        del ws4, sv4
    if other in plans:
        layers["rgat_fwd_am_like_880k_" + names[other]] = {
            "edges_per_s": E / (plans[other][0] * 1e-3), "ms": plans[other][0],
            "kernels_ms": {k: round(v[1], 4) for k, v in plans[other][1].items()}}
    if args.calibrate_copy:
        # a plain device copy of known size, for scaling the FETCH_SIZE /
        # WRITE_SIZE counters of a profiling run (1 GiB read + 1 GiB written)
        log("copy calibration")
        src = torch.ones(1 << 28, device=c.dev)
        dst = torch.empty_like(src)
        for _ in range(2):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    log("cpu baseline")
    cpu = None if args.no_cpu else cpu_baseline(c, args.cpu_seconds)
    line_kernels = {k: {"launches_per_step": n, "mean_ms": round(m, 4)} for k, (n, m) in kern.items()}
    # every modelled kernel of the headline: algorithmic and counter GB/s against
    # the HBM peak, and the GEMM's MFMA utilisation against the fp32 dense peak
    for k, m in model.items():
        if k not in kern:
            continue
        kms_k = kern[k][1]
        ent = line_kernels[k]
        ent["model_bytes"] = m["bytes"]
        ent["model_gbs"] = round(m["bytes"] / (kms_k * 1e-3) / 1e9, 1)
        ent["model_frac"] = round(ent["model_gbs"] / HBM_PEAK_GBS, 4)
        tr = counter_traffic("rgat_am_like_880k", k)
        ent["counter_bytes"] = tr
        ent["counter_gbs"] = None if tr is None else round(tr / (kms_k * 1e-3) / 1e9, 1)
        if k in ("typed_gemm", "rgat_af_fused"):
            ent["mfma_tflops"] = round(m["flops"] / (kms_k * 1e-3) / 1e12, 2)
            ent["mfma_frac"] = round(ent["mfma_tflops"] / FP32_PEAK_TFLOPS, 4)
    c.close()
    del out, saved

    if args.only == "all":
        # ------------------------------------------------ RGAT backward (workload 5 = graph 2)
        log("workload 5: RGAT backward")
        c = Ctx(5)
        out = torch.empty(inf["num_nodes"], d, device=c.dev)
        saved = torch.empty(inf["num_nodes"], 1, 2, device=c.dev)
        wsf = c.ws(rgnn.LAYER_RGAT, d, d, 1)
        rgnn.rgat_forward(c.G, c.T["h"], c.T["W"], c.T["w_src"], c.T["w_dst"], out, saved, wsf, d, d)
        R = inf["num_rels"]
        gh = torch.empty(inf["num_nodes"], d, device=c.dev)
        gW, gs, gt = (torch.empty(R, d, d, device=c.dev), torch.empty(R, d, device=c.dev),
                      torch.empty(R, d, device=c.dev))
        wsb = c.ws(rgnn.LAYER_RGAT_BACKWARD, d, d)
        fnb = lambda: rgnn.rgat_backward(c.G, c.T["h"], c.T["W"], c.T["w_src"], c.T["w_dst"], saved,
                                         c.T["grad_out"], gh, gW, gs, gt, wsb, d, d)
        msb = time_steps(torch, fnb, K, W)
        kb = kernel_profile(rgnn, torch, fnb, max(3, K // 2))
        layers["rgat_bwd_am_like_880k"] = {"edges_per_s": E / (msb * 1e-3), "ms": msb,
                                           "kernels_ms": {k: round(v[1], 4) for k, v in kb.items()}}
        del wsb
        # softmax per (dst, rel) segment: forward (aggregate-first) and backward
        savedr = torch.empty(inf["num_dst_segments"], 2, device=c.dev)
        wsr1 = c.ws(rgnn.LAYER_RGAT, d, d, 1, rgnn.PLAN_AGGREGATE_FIRST)
        rgnn.rgat_forward(c.G, c.T["h"], c.T["W"], c.T["w_src"], c.T["w_dst"], out, savedr, wsr1, d, d,
                          softmax_scope=rgnn.SOFTMAX_PER_DST_REL)
        del wsr1
        wsbr = c.ws(rgnn.LAYER_RGAT_BACKWARD, d, d)
        fnbr = lambda: rgnn.rgat_backward(c.G, c.T["h"], c.T["W"], c.T["w_src"], c.T["w_dst"], savedr,
                                          c.T["grad_out"], gh, gW, gs, gt, wsbr, d, d,
                                          softmax_scope=rgnn.SOFTMAX_PER_DST_REL)
        msbr = time_steps(torch, fnbr, K, W)
        layers["rgat_bwd_am_like_880k_per_relation_softmax"] = {"edges_per_s": E / (msbr * 1e-3), "ms": msbr}
        del wsbr, savedr
        # four heads: one pass over all heads (gradients in the message space)
        saved4 = torch.empty(inf["num_nodes"], 4, 2, device=c.dev)
        ws4 = c.ws(rgnn.LAYER_RGAT, d, d, 4)
        rgnn.rgat_forward(c.G, c.T["h"], c.T["W"], c.T["w_src"], c.T["w_dst"], out, saved4, ws4, d, d, 4)
        del ws4
        wsb4 = c.ws(rgnn.LAYER_RGAT_BACKWARD, d, d, 4)
        fnb4 = lambda: rgnn.rgat_backward(c.G, c.T["h"], c.T["W"], c.T["w_src"], c.T["w_dst"], saved4,
                                          c.T["grad_out"], gh, gW, gs, gt, wsb4, d, d, 4)
        msb4 = time_steps(torch, fnb4, K, W)
        kb4 = kernel_profile(rgnn, torch, fnb4, max(3, K // 2))
        layers["rgat_bwd_am_like_880k_4heads"] = {"edges_per_s": E / (msb4 * 1e-3), "ms": msb4,
                                                  "kernels_ms": {k: round(v[1], 4) for k, v in kb4.items()}}
        del wsb4, saved4
        # RGCN forward (with self-loop) and backward on the same graph
        log("workload 5: RGCN forward and backward")
        pr = rgnn.select_plan(c.G, rgnn.LAYER_RGCN, d, d, 1)[0]
        wsr = c.ws(rgnn.LAYER_RGCN, d, d, 1, pr)
        fnr = lambda: rgnn.rgcn_forward(c.G, c.T["h"], c.T["W"], c.T["W0"], out, wsr, d, d, 0, pr)
        msr = time_steps(torch, fnr, K, W)
        kr = kernel_profile(rgnn, torch, fnr, max(3, K // 2))
        layers["rgcn_fwd_am_like_880k"] = {"edges_per_s": E / (msr * 1e-3), "ms": msr, "plan": names[pr],
                                           "kernels_ms": {k: round(v[1], 4) for k, v in kr.items()}}
        gW0 = torch.empty(d, d, device=c.dev)
        wsrb = c.ws(rgnn.LAYER_RGCN_BACKWARD, d, d)
        fnrb = lambda: rgnn.rgcn_backward(c.G, c.T["h"], c.T["W"], c.T["W0"], None, c.T["grad_out"], gh, gW,
                                          gW0, wsrb, d, d, 0)
        msrb = time_steps(torch, fnrb, K, W)
        krb = kernel_profile(rgnn, torch, fnrb, max(3, K // 2))
        layers["rgcn_bwd_am_like_880k"] = {"edges_per_s": E / (msrb * 1e-3), "ms": msrb,
                                           "kernels_ms": {k: round(v[1], 4) for k, v in krb.items()}}
        c.close()
        del out, saved, wsf, gh, gW, gs, gt, wsr, wsrb, gW0

        # ------------------------------------------------ HGT forward, workload 3
        log("workload 3: HGT forward")
        c = Ctx(3)
        d3 = 64
        out = torch.empty(c.info["num_nodes"], d3, device=c.dev)
        saved3 = torch.empty(c.info["num_nodes"], 4, 2, device=c.dev)
        ws = c.ws(rgnn.LAYER_HGT, d3, d3, 4)
        # the layer forward (inference: no softmax statistics kept), then the
        # same keeping them for the backward (training)
        fnh = lambda: rgnn.hgt_forward(c.G, c.T["h"], c.T["Wk"], c.T["Wq"], c.T["Wv"], c.T["Wa"],
                                       c.T["Watt"], c.T["Wmsg"], c.T["mu"], out, ws, d3, 4, 0.25)
        msh = time_steps(torch, fnh, K, W)
        kh = kernel_profile(rgnn, torch, fnh, max(3, K // 2))
        layers["hgt_fwd_mag_like_1p9m"] = {"edges_per_s": c.info["num_edges"] / (msh * 1e-3), "ms": msh,
                                           "kernels_ms": {k: round(v[1], 4) for k, v in kh.items()}}
        fnhs = lambda: rgnn.hgt_forward(c.G, c.T["h"], c.T["Wk"], c.T["Wq"], c.T["Wv"], c.T["Wa"],
                                        c.T["Watt"], c.T["Wmsg"], c.T["mu"], out, ws, d3, 4, 0.25,
                                        saved=saved3)
        mshs = time_steps(torch, fnhs, K, W)
        layers["hgt_fwd_mag_like_1p9m_keeping_softmax_stats"] = {
            "edges_per_s": c.info["num_edges"] / (mshs * 1e-3), "ms": mshs}
        # HGT backward from the forward's softmax statistics (the forward above
        # wrote them), and without them (the forward traversal recomputed inside)
        log("workload 3: HGT backward")
        N3, R3, T3 = c.info["num_nodes"], c.info["num_rels"], c.g["T"]
        grads = dict(dh=torch.empty(N3, d3, device=c.dev), dWk=torch.empty(T3, d3, d3, device=c.dev),
                     dWq=torch.empty(T3, d3, d3, device=c.dev), dWv=torch.empty(T3, d3, d3, device=c.dev),
                     dWa=torch.empty(T3, d3, d3, device=c.dev), dWatt=torch.empty(R3, 4, 16, 16, device=c.dev),
                     dWmsg=torch.empty(R3, 4, 16, 16, device=c.dev), dmu=torch.empty(R3, device=c.dev))
        wsb3 = c.ws(rgnn.LAYER_HGT_BACKWARD, d3, d3, 4)
        fnhb = lambda: rgnn.hgt_backward(c.G, c.T["h"], c.T["Wk"], c.T["Wq"], c.T["Wv"], c.T["Wa"], c.T["Watt"],
                                         c.T["Wmsg"], c.T["mu"], c.T["grad_out"], grads, wsb3, d3, 4, 0.25,
                                         saved=saved3)
        mshb = time_steps(torch, fnhb, K, W)
        khb = kernel_profile(rgnn, torch, fnhb, max(3, K // 2))
        layers["hgt_bwd_mag_like_1p9m"] = {"edges_per_s": c.info["num_edges"] / (mshb * 1e-3), "ms": mshb,
                                           "kernels_ms": {k: round(v[1], 4) for k, v in khb.items()}}
        fnhr = lambda: rgnn.hgt_backward(c.G, c.T["h"], c.T["Wk"], c.T["Wq"], c.T["Wv"], c.T["Wa"], c.T["Watt"],
                                         c.T["Wmsg"], c.T["mu"], c.T["grad_out"], grads, wsb3, d3, 4, 0.25)
        mshr = time_steps(torch, fnhr, K, W)
        layers["hgt_bwd_mag_like_1p9m_forward_recomputed"] = {"edges_per_s": c.info["num_edges"] / (mshr * 1e-3),
                                                               "ms": mshr}
        del grads, wsb3, saved3
        c.close()
        del out, ws

        # ------------------------------------------------ RGCN and RGAT at d = 128, workload 4
        log("workload 4: RGCN and RGAT at d = 128")
        c = Ctx(4)
        d4 = 128
        out = torch.empty(c.info["num_nodes"], d4, device=c.dev)
        for lname, layer in (("rgcn", rgnn.LAYER_RGCN), ("rgat", rgnn.LAYER_RGAT)):
            p4 = rgnn.select_plan(c.G, layer, d4, d4, 1)[0]
            ws = c.ws(layer, d4, d4, 1, p4)
            if layer == rgnn.LAYER_RGCN:
                f4 = lambda ws=ws, p4=p4: rgnn.rgcn_forward(c.G, c.T["h"], c.T["W"], c.T["W0"], out, ws,
                                                            d4, d4, 0, p4)
            else:
                f4 = lambda ws=ws, p4=p4: rgnn.rgat_forward(c.G, c.T["h"], c.T["W"], c.T["w_src"],
                                                            c.T["w_dst"], out, None, ws, d4, d4, 1,
                                                            0.2, 0, p4)
            m4 = time_steps(torch, f4, K, W)
            k4 = kernel_profile(rgnn, torch, f4, max(3, K // 2))
            layers[f"{lname}_fwd_wikikg2_like_2p5m_d128"] = {
                "edges_per_s": c.info["num_edges"] / (m4 * 1e-3), "ms": m4, "plan": names[p4],
                "kernels_ms": {k: round(v[1], 4) for k, v in k4.items()}}
            del ws
        # backward at d = 128 (the loss weight of the workload's generator)
        N4, R4 = c.info["num_nodes"], c.info["num_rels"]
        saved4 = torch.empty(N4, 1, 2, device=c.dev)
        ws = c.ws(rgnn.LAYER_RGAT, d4, d4, 1)
        rgnn.rgat_forward(c.G, c.T["h"], c.T["W"], c.T["w_src"], c.T["w_dst"], out, saved4, ws, d4, d4)
        del ws
        gh = torch.empty(N4, d4, device=c.dev)
        gW, gs, gt = (torch.empty(R4, d4, d4, device=c.dev), torch.empty(R4, d4, device=c.dev),
                      torch.empty(R4, d4, device=c.dev))
        ws = c.ws(rgnn.LAYER_RGAT_BACKWARD, d4, d4)
        fb4 = lambda: rgnn.rgat_backward(c.G, c.T["h"], c.T["W"], c.T["w_src"], c.T["w_dst"], saved4,
                                         c.T["grad_out"], gh, gW, gs, gt, ws, d4, d4)
        mb4 = time_steps(torch, fb4, K, W)
        layers["rgat_bwd_wikikg2_like_2p5m_d128"] = {"edges_per_s": c.info["num_edges"] / (mb4 * 1e-3), "ms": mb4}
        del ws
        gW0 = torch.empty(d4, d4, device=c.dev)
        ws = c.ws(rgnn.LAYER_RGCN_BACKWARD, d4, d4)
        fr4 = lambda: rgnn.rgcn_backward(c.G, c.T["h"], c.T["W"], c.T["W0"], None, c.T["grad_out"], gh, gW,
                                         gW0, ws, d4, d4, 0)
        mr4 = time_steps(torch, fr4, K, W)
        layers["rgcn_bwd_wikikg2_like_2p5m_d128"] = {"edges_per_s": c.info["num_edges"] / (mr4 * 1e-3), "ms": mr4}
        del ws, gh, gW, gs, gt, gW0, saved4
        c.close()
        del out

        # ------------------------------------------------ RGCN, workload 1 (small, launch-bound)
        log("workload 1: RGCN")
        c = Ctx(1)
        out = torch.empty(c.info["num_nodes"], 64, device=c.dev)
        ws = c.ws(rgnn.LAYER_RGCN, 64, 64)
        f1 = lambda: rgnn.rgcn_forward(c.G, c.T["h"], c.T["W"], c.T["W0"], out, ws, 64, 64)
        m1 = time_steps(torch, f1, K, W)
        layers["rgcn_fwd_uniform_2k"] = {"edges_per_s": c.info["num_edges"] / (m1 * 1e-3), "ms": m1}
        c.close()

    line = {
        "metric": METRIC,
        "value": value,
        "unit": "edges/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": ms,
        "ms_median": float(np.median(each)),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": "rgat_am_like_880k: RGAT layer forward, 880000 nodes / 7 node types / "
                        "96 relations (Zipf 1.2) / 5700000 edges (power-law in-degree, gamma 2.1), "
                        "d_in = d_out = 64, 1 head, softmax per destination",
            "plan": names[plan],
            "modelled_bytes": {"transform_first": b_tf, "aggregate_first": b_af},
            "U_src": inf["num_src_pairs"], "U_dst": inf["num_dst_segments"],
            "max_in_degree": inf["max_in_degree"],
        },
        "roofline": {
            "bound": "hbm",
            "kernel": kname,
            "achieved": kgbs,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": kgbs / HBM_PEAK_GBS,
            "traffic": counter_traffic("rgat_am_like_880k", kname),
            "mean_ms": kms,
            "algorithmic_bytes": km["bytes"],
            "algorithmic_tflops": ktfl,
        },
        "kernels": line_kernels,
        "cpu_baseline": cpu,
        "layers": layers,
    }
    print(json.dumps(line))


if __name__ == "__main__":
    main()
