"""Seeded synthetic heterogeneous graphs and layer tensors.

The paper evaluates single RGNN layers (in/out dimension 64, one head) on DGL/OGB
heterogeneous graphs (Section "Methodology", Table "tab:datasets").  Those
datasets are not available here, so every input is drawn from numpy's PCG64 with
a fixed seed, with the sizes, type counts and degree / relation-frequency shapes
of the five workloads this library is measured on:

  1  RGCN   2 000 nodes, 3 node types, 8 relations, 20 000 edges, uniform ends.
  2  RGAT   880 000 nodes, 7 node types, 96 relations, 5.7 M edges; relation
            frequencies Zipf(1.2); destinations power-law (Chung-Lu, gamma 2.1);
            sources uniform  (an am-like graph).
  3  HGT    1.9 M nodes in 4 types (1 102 000 / 722 000 / 9 500 / 66 500),
            7 relations: 4 forward ones with sizes 1:5:10:5 units plus exact
            transposes of the three that join different node types; 21 M edges
            (a mag-like graph).
  4  RGCN+RGAT, d=128: 2.5 M nodes, 1 node type, 535 relations (Zipf 1.1),
            16 M edges, power-law sources and destinations (a wikikg2-like graph).
  5  RGAT forward+backward on workload 2's graph plus a N(0,1) loss weight.

Nothing here computes any part of a layer: the module only draws index arrays and
random tensors, so both the CPU oracle and the GPU path can consume the same bytes.
"""
from __future__ import annotations

import numpy as np

BASE_SEED = 230106284

# Units of workload 3: one relation "unit" of edges.
_HGT_UNIT = 656_250
_HGT_NTYPE_COUNTS = (1_102_000, 722_000, 9_500, 66_500)   # A, P, I, F
# (src type, dst type, units) of the forward relations r0..r3, then the
# relations r4..r6 that are exact transposes of r0, r1, r3.
_HGT_FWD = ((0, 2, 1), (0, 1, 5), (1, 1, 10), (1, 3, 5))
_HGT_REV_OF = (0, 1, 3)

CONFIGS = {
    1: dict(name="rgcn_uniform_2k", layers=("rgcn",), N=2000, T=3, R=8, E=20_000,
            d=64, heads=1, graph="uniform"),
    2: dict(name="rgat_am_like_880k", layers=("rgat",), N=880_000, T=7, R=96,
            E=5_700_000, d=64, heads=1, graph="powerlaw_dst", rel_zipf=1.2, gamma=2.1),
    3: dict(name="hgt_mag_like_1p9m", layers=("hgt",), N=1_900_000, T=4, R=7,
            E=21_000_000, d=64, heads=4, graph="typed_blocks"),
    4: dict(name="rgcn_rgat_wikikg2_like_2p5m", layers=("rgcn", "rgat"), N=2_500_000,
            T=1, R=535, E=16_000_000, d=128, heads=1, graph="powerlaw_both",
            rel_zipf=1.1, gamma=2.1),
    5: dict(name="rgat_train_am_like_880k", layers=("rgat_bwd",), N=880_000, T=7,
            R=96, E=5_700_000, d=64, heads=1, graph="powerlaw_dst", rel_zipf=1.2,
            gamma=2.1),
}


def _streams(k: int, n: int = 6):
    # workload 5 is workload 2's graph and tensors plus a loss weight
    ss = np.random.SeedSequence(BASE_SEED + (2 if k == 5 else k))
    return [np.random.Generator(np.random.PCG64(c)) for c in ss.spawn(n)]


def _categorical(rng, weights: np.ndarray, size: int) -> np.ndarray:
    cdf = np.cumsum(weights, dtype=np.float64)
    cdf /= cdf[-1]
    idx = np.searchsorted(cdf, rng.random(size), side="right")
    return np.minimum(idx, len(weights) - 1)


def _zipf_rel(rng, R: int, s: float, E: int) -> np.ndarray:
    w = np.arange(1, R + 1, dtype=np.float64) ** (-s)
    return _categorical(rng, w, E).astype(np.int32)


def _chung_lu(rng, N: int, E: int, gamma: float) -> np.ndarray:
    """Endpoints with a power-law expected degree: rank k has weight k^(-1/(gamma-1));
    ranks are mapped to node ids by a seeded random permutation."""
    w = np.arange(1, N + 1, dtype=np.float64) ** (-1.0 / (gamma - 1.0))
    ranks = _categorical(rng, w, E)
    perm = rng.permutation(N).astype(np.int32)
    return perm[ranks]


def _uniform_types(rng, N: int, T: int) -> np.ndarray:
    return rng.integers(0, T, size=N, dtype=np.int32)


def make_graph(k: int, scale: float = 1.0) -> dict:
    """COO graph of workload k.  `scale` < 1 shrinks node and edge counts
    proportionally while keeping the shape (used for mid-size parity tests)."""
    c = CONFIGS[k]
    g_rng, t_rng = _streams(k)[:2]
    R, T = c["R"], c["T"]
    if c["graph"] == "typed_blocks":
        counts = [max(1, int(round(n * scale))) for n in _HGT_NTYPE_COUNTS]
        N = int(sum(counts))
        ntype = np.repeat(np.arange(T, dtype=np.int32), counts)
        ntype = ntype[t_rng.permutation(N)]
        members = [np.flatnonzero(ntype == t).astype(np.int32) for t in range(T)]
        unit = max(1, int(round(_HGT_UNIT * scale)))
        srcs, dsts, rels = [], [], []
        fwd = []
        for r, (ts, td, units) in enumerate(_HGT_FWD):
            ne = units * unit
            s = members[ts][g_rng.integers(0, len(members[ts]), ne)]
            d = members[td][g_rng.integers(0, len(members[td]), ne)]
            fwd.append((s, d))
            srcs.append(s); dsts.append(d); rels.append(np.full(ne, r, np.int32))
        for j, r_of in enumerate(_HGT_REV_OF):
            s, d = fwd[r_of]
            srcs.append(d); dsts.append(s)
            rels.append(np.full(len(s), len(_HGT_FWD) + j, np.int32))
        src = np.concatenate(srcs); dst = np.concatenate(dsts); rel = np.concatenate(rels)
        order = g_rng.permutation(len(src))
        src, dst, rel = src[order], dst[order], rel[order]
    else:
        N = max(2, int(round(c["N"] * scale)))
        E = max(1, int(round(c["E"] * scale)))
        ntype = _uniform_types(t_rng, N, T)
        if c["graph"] == "uniform":
            src = g_rng.integers(0, N, E, dtype=np.int32)
            dst = g_rng.integers(0, N, E, dtype=np.int32)
            rel = g_rng.integers(0, R, E, dtype=np.int32)
        else:
            rel = _zipf_rel(g_rng, R, c["rel_zipf"], E)
            dst = _chung_lu(g_rng, N, E, c["gamma"])
            if c["graph"] == "powerlaw_both":
                src = _chung_lu(g_rng, N, E, c["gamma"])
            else:
                src = g_rng.integers(0, N, E, dtype=np.int32)
    return dict(N=int(N), E=int(len(src)), R=R, T=T,
                src=np.ascontiguousarray(src, np.int32),
                dst=np.ascontiguousarray(dst, np.int32),
                rel=np.ascontiguousarray(rel, np.int32),
                ntype=np.ascontiguousarray(ntype, np.int32))


def _normal(rng, shape, var: float) -> np.ndarray:
    return (rng.standard_normal(shape, dtype=np.float32) * np.float32(np.sqrt(var)))


def make_tensors(k: int, g: dict, layer: str | None = None, d: int | None = None,
                 heads: int | None = None) -> dict:
    """Features, weights and (workloads 1 to 5) the loss weight for workload k.
    Variances: features and weights 1/fan_in, attention vectors 0.1, HGT head
    blocks 1/d_k, loss weight 1.  `d` and `heads` override the workload's
    hidden size and HGT head count (the hidden-size sweep)."""
    c = CONFIGS[k]
    _, _, f_rng, w_rng, a_rng, l_rng = _streams(k)
    layer = layer or c["layers"][0]
    N, R, T, d = g["N"], c["R"], c["T"], d or c["d"]
    out = dict(h=_normal(f_rng, (N, d), 1.0 / d))
    if layer in ("rgcn", "rgat", "rgat_bwd"):
        out["W"] = _normal(w_rng, (R, d, d), 1.0 / d)
        out["W0"] = _normal(w_rng, (d, d), 1.0 / d)
        out["w_src"] = _normal(a_rng, (R, d), 0.1)
        out["w_dst"] = _normal(a_rng, (R, d), 0.1)
        if layer == "rgat_bwd" or k in (1, 2, 4, 5):
            out["grad_out"] = _normal(l_rng, (N, d), 1.0)
    if layer == "hgt":
        H = heads or c["heads"]
        dk = d // H
        for name in ("Wk", "Wq", "Wv", "Wa"):
            out[name] = _normal(w_rng, (T, d, d), 1.0 / d)
        out["Watt"] = _normal(a_rng, (R, H, dk, dk), 1.0 / dk)
        out["Wmsg"] = _normal(a_rng, (R, H, dk, dk), 1.0 / dk)
        out["mu"] = np.ones(R, np.float32)
        out["grad_out"] = _normal(l_rng, (N, d), 1.0)
    return out


def tiny_graph(seed: int, N: int, E: int, R: int, T: int = 1, kind: str = "random") -> dict:
    """Small graphs for oracle pins and edge cases.

    kind: "random"   uniform ends and relations (self-edges and duplicates occur);
          "hub"      half the edges point at node 0;
          "srchub"   half the edges leave node 0;
          "complete" every ordered pair (s, t) once, including s == t, relation 0;
          "isolated" destinations drawn from the first half of the nodes only;
          "dups"     a few (u, v, r) triples repeated many times;
          "typed"    every relation joins one source node type to one
                     destination node type (as in heterogeneous graphs);
          "typedhub" the same with half the edges at the first node of
                     their relation's destination type;
          "empty"    no edges at all.
    """
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed)))
    ntype = rng.integers(0, T, N, dtype=np.int32)
    if kind == "empty" or (E == 0 and kind != "complete"):
        src = dst = rel = np.zeros(0, np.int32)
    elif kind == "complete":
        s, t = np.meshgrid(np.arange(N), np.arange(N), indexing="ij")
        src = s.ravel().astype(np.int32); dst = t.ravel().astype(np.int32)
        rel = np.zeros(len(src), np.int32)
        perm = rng.permutation(len(src))
        src, dst = src[perm], dst[perm]
    else:
        src = rng.integers(0, N, E, dtype=np.int32)
        dst = rng.integers(0, N, E, dtype=np.int32)
        rel = rng.integers(0, R, E, dtype=np.int32)
        if kind in ("hub", "srchub"):
            (dst if kind == "hub" else src)[: E // 2] = 0
            perm = rng.permutation(E)
            src, dst, rel = src[perm], dst[perm], rel[perm]
        elif kind == "isolated":
            dst = rng.integers(0, max(1, N // 2), E, dtype=np.int32)
        elif kind == "dups":
            k = max(1, E // 8)
            pick = rng.integers(0, k, E)
            src, dst, rel = src[pick], dst[pick], rel[pick]
        elif kind in ("typed", "typedhub"):
            ntype[: min(T, N)] = np.arange(min(T, N), dtype=np.int32)   # no empty type
            members = [np.flatnonzero(ntype == t).astype(np.int32) for t in range(T)]
            dtype_r = np.arange(R) % T
            stype_r = (np.arange(R) * 3 + 1) % T
            for r in range(R):
                m = rel == r
                ds, ss = members[dtype_r[r]], members[stype_r[r]]
                dst[m] = ds[rng.integers(0, len(ds), int(m.sum()))]
                src[m] = ss[rng.integers(0, len(ss), int(m.sum()))]
                if kind == "typedhub":
                    hub = m & (np.arange(E) % 2 == 0)
                    dst[hub] = ds[0]
    return dict(N=int(N), E=int(len(src)), R=int(R), T=int(T),
                src=np.ascontiguousarray(src, np.int32),
                dst=np.ascontiguousarray(dst, np.int32),
                rel=np.ascontiguousarray(rel, np.int32),
                ntype=ntype)


def tiny_tensors(seed: int, g: dict, d_in: int, d_out: int, heads: int = 1,
                 att_var: float = 0.1) -> dict:
    """All tensors any layer may need on a tiny graph (float32)."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 7])))
    N, R, T = g["N"], g["R"], g["T"]
    dk = d_out // heads
    return dict(
        h=_normal(rng, (N, d_in), 1.0 / d_in),
        W=_normal(rng, (R, d_in, d_out), 1.0 / d_in),
        W0=_normal(rng, (d_in, d_out), 1.0 / d_in),
        w_src=_normal(rng, (R, d_out), att_var),
        w_dst=_normal(rng, (R, d_out), att_var),
        Wk=_normal(rng, (T, d_in, d_out), 1.0 / d_in),
        Wq=_normal(rng, (T, d_in, d_out), 1.0 / d_in),
        Wv=_normal(rng, (T, d_in, d_out), 1.0 / d_in),
        Wa=_normal(rng, (T, d_out, d_out), 1.0 / d_out),
        Watt=_normal(rng, (R, heads, dk, dk), 1.0 / dk),
        Wmsg=_normal(rng, (R, heads, dk, dk), 1.0 / dk),
        mu=(1.0 + 0.5 * rng.random(R)).astype(np.float32),
        grad_out=_normal(rng, (N, d_out), 1.0),
    )


def degree_stats(g: dict) -> dict:
    """Counts used in documentation: unique (src, rel) and (dst, rel) pairs,
    maximum in-degree and the number of destinations without in-edges."""
    N, R = g["N"], g["R"]
    src = g["src"].astype(np.int64); dst = g["dst"].astype(np.int64)
    rel = g["rel"].astype(np.int64)
    indeg = np.bincount(dst, minlength=N)
    return dict(
        N=N, E=g["E"], R=R,
        U_src=int(len(np.unique(rel * N + src))),
        U_dst=int(len(np.unique(dst * R + rel))),
        max_in_deg=int(indeg.max()) if N else 0,
        zero_in_deg=int((indeg == 0).sum()),
    )
