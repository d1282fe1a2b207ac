"""Seeded synthetic decoding graphs and log-likelihood matrices.

This module only draws random numbers and lays them out as a CSR graph and a
frames x pdfs matrix.  It performs none of the decoder's arithmetic, so both
the CPU oracle (test infrastructure) and the GPU library can be fed from it.

The workloads stand in for the paper's Switchboard / NIST 2000 setup
(Sec. 4.1: a 30k-word tri-gram HCLG, sub-sampled frame rate, beam 14; Sec. 4.3:
HCLG sizes from 13 MB up to an 11 GB graph), which is not available here.
Every graph has start state 0 and no final weights (every state final with
cost 0) unless a test asks for finals.

Graph layout (CSR, arc id = position in the arrays):
  row_ptr[S+1] u32, dst[A] u32, ilabel[A] i32 (0 = epsilon, k >= 1 -> pdf
  column k-1), olabel[A] i32 (0 = no word), weight[A] f32 (>= 0).
"""
from __future__ import annotations

import numpy as np

__all__ = ["WORKLOADS", "workload", "make_graph", "make_loglikes", "make_batch",
           "tiny_graph", "tiny_loglikes", "zipf_exponent"]

# Decoding workloads.  `index` fixes the seeds: graph seed 1000*index + 1,
# log-likelihood seed 1000*index + 2 (+ 100 + i for utterance i of a batch).
WORKLOADS = {
    # 10k states, ~30k arcs (1 + Poisson(2) out-degree), 20% epsilon arcs to
    # higher state ids, 500 pdfs, 1000 words, weights Exp(mean 2); 300 frames
    # of N(-12, 3) with one N(-2, 1) peak per frame.
    "tiny_10k": dict(index=1, family="forward_eps", S=10_000, eps_frac=0.2, P=500,
                     V=1000, wmean=2.0, T=300, ll_mean=-12.0, ll_std=3.0,
                     peaks=(1, 1), beam=10.0, max_active=2000, lattice_beam=6.0),
    # HCLG-shaped: 5M states, 12M arcs, Zipf out-degree on 1..200, 15% epsilon
    # arcs in chains of depth <= 4, 6000 pdfs, 30k words, Exp(mean 3);
    # 1000 frames of N(-15, 4) with 3-5 N(-2, 1) peaks per frame.
    "hclg_5m": dict(index=2, family="zipf_levels", S=5_000_000, A=12_000_000,
                    eps_frac=0.15, depth=4, P=6000, V=30_000, wmean=3.0, T=1000,
                    ll_mean=-15.0, ll_std=4.0, peaks=(3, 5), beam=15.0,
                    max_active=7000, lattice_beam=8.0),
    # Large-LM graph: 30M states, 80M arcs, 10% epsilon (depth <= 4),
    # 100k words; 1500 frames as hclg_5m.
    "lm_30m": dict(index=3, family="zipf_levels", S=30_000_000, A=80_000_000,
                   eps_frac=0.10, depth=4, P=6000, V=100_000, wmean=3.0, T=1500,
                   ll_mean=-15.0, ll_std=4.0, peaks=(3, 5), beam=15.0,
                   max_active=10000, lattice_beam=8.0),
    # 64 utterances of U{500..1500} frames against the hclg_5m graph.
    "batch64_hclg_5m": dict(index=4, family="zipf_levels", graph_of="hclg_5m",
                            S=5_000_000, A=12_000_000, eps_frac=0.15, depth=4,
                            P=6000, V=30_000, wmean=3.0, batch=64, T_range=(500, 1500),
                            ll_mean=-15.0, ll_std=4.0, peaks=(3, 5), beam=15.0,
                            max_active=7000, lattice_beam=8.0),
    # Wide beam: 2M states, 6M arcs, 40% epsilon (depth <= 8), 3000 pdfs,
    # 800 frames of flat N(-8, 1), beam 20, no max-active limit.
    "wide_2m": dict(index=5, family="zipf_levels", S=2_000_000, A=6_000_000,
                    eps_frac=0.40, depth=8, P=3000, V=30_000, wmean=3.0, T=800,
                    ll_mean=-8.0, ll_std=1.0, peaks=(0, 0), beam=20.0,
                    max_active=0, lattice_beam=10.0),
}
# Same as wide_2m with weights and log-likelihoods rounded to multiples of
# 2^-4, so that every cost sum is exact in fp32 and ties are real.
WORKLOADS["wide_2m_dyadic"] = dict(WORKLOADS["wide_2m"], dyadic=True)


def workload(name: str) -> dict:
    if name not in WORKLOADS:
        raise KeyError(f"unknown workload {name!r}; known: {sorted(WORKLOADS)}")
    return dict(WORKLOADS[name], name=name)


def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def zipf_exponent(mean: float, kmax: int = 200) -> float:
    """Exponent s of a Zipf law truncated to 1..kmax whose mean is `mean`."""
    k = np.arange(1, kmax + 1, dtype=np.float64)
    lo, hi = 0.5, 8.0
    for _ in range(200):
        s = 0.5 * (lo + hi)
        p = k ** -s
        m = float((k * p).sum() / p.sum())
        if m > mean:
            lo = s
        else:
            hi = s
    return 0.5 * (lo + hi)


def _quantize(x: np.ndarray) -> np.ndarray:
    return (np.round(x.astype(np.float64) * 16.0) / 16.0).astype(np.float32)


def _graph_forward_eps(cfg: dict, rng: np.random.Generator) -> dict:
    S = cfg["S"]
    deg = 1 + rng.poisson(2.0, S)
    row_ptr = np.zeros(S + 1, dtype=np.int64)
    np.cumsum(deg, out=row_ptr[1:])
    A = int(row_ptr[-1])
    src = np.repeat(np.arange(S, dtype=np.int64), deg)
    is_eps = (rng.random(A) < cfg["eps_frac"]) & (src < S - 1)
    dst = rng.integers(0, S, A, dtype=np.int64)
    u = rng.random(A)
    # epsilon destination uniform over the higher state ids (src, S)
    eps_dst = src + 1 + np.minimum((u * (S - 1 - src)).astype(np.int64), S - 2 - src)
    dst = np.where(is_eps, eps_dst, dst)
    ilabel = np.where(is_eps, 0, rng.integers(1, cfg["P"] + 1, A))
    olabel = np.where(rng.random(A) < 0.9, 0, rng.integers(1, cfg["V"] + 1, A))
    weight = rng.exponential(cfg["wmean"], A).astype(np.float32)
    return dict(row_ptr=row_ptr, dst=dst, ilabel=ilabel, olabel=olabel, weight=weight)


def _graph_zipf_levels(cfg: dict, rng: np.random.Generator) -> dict:
    S, A, depth = cfg["S"], cfg["A"], cfg["depth"]
    # out-degree: Zipf truncated to 1..200, exponent fitted to the mean A/S,
    # then nudged by +-1 on random states so the arc count is exactly A.
    kmax = 200
    s = zipf_exponent(A / S, kmax)
    k = np.arange(1, kmax + 1, dtype=np.float64)
    cdf = np.cumsum(k ** -s)
    cdf /= cdf[-1]
    deg = (np.searchsorted(cdf, rng.random(S), side="right") + 1).astype(np.int64)
    deg = np.minimum(deg, kmax)
    # the start state fans out widely, as an HCLG start state does
    deg[0] = kmax
    diff = A - int(deg.sum())
    while diff != 0:
        if diff > 0:
            cand = np.flatnonzero(deg < kmax)
            cand = cand[cand != 0]
            pick = rng.choice(cand, size=min(diff, cand.size), replace=False)
            deg[pick] += 1
        else:
            cand = np.flatnonzero(deg > 1)
            cand = cand[cand != 0]
            pick = rng.choice(cand, size=min(-diff, cand.size), replace=False)
            deg[pick] -= 1
        diff = A - int(deg.sum())
    row_ptr = np.zeros(S + 1, dtype=np.int64)
    np.cumsum(deg, out=row_ptr[1:])
    src = np.repeat(np.arange(S, dtype=np.int64), deg)
    first = np.zeros(A, dtype=bool)
    first[row_ptr[:-1]] = True
    # epsilon levels 0..depth, geometric sizes (half the states at level 0);
    # an epsilon arc always climbs to a strictly higher level, so the epsilon
    # subgraph is acyclic and its longest chain has at most `depth` arcs.
    lw = 0.5 ** np.arange(depth + 1)
    lw /= lw.sum()
    level = np.searchsorted(np.cumsum(lw), rng.random(S), side="right").clip(0, depth)
    by_level = [np.flatnonzero(level == l) for l in range(depth + 1)]
    # the first arc of every state is emitting; epsilon arcs are drawn among
    # the other arcs of states below the top level
    eligible = (~first) & (level[src] < depth)
    q = cfg["eps_frac"] * A / max(1, int(eligible.sum()))
    is_eps = eligible & (rng.random(A) < q)
    dst = rng.integers(0, S, A, dtype=np.int64)
    # HMM-like self-loop on the first arc, only where another arc leaves the
    # state (a lone self-loop would be a trap) and never on the start state
    selfloop = first & (rng.random(A) < 0.5) & (deg[src] >= 2) & (src != 0)
    dst = np.where(selfloop, src, dst)
    eidx = np.flatnonzero(is_eps)
    lsrc = level[src[eidx]]
    # destination level uniform over (level(src), depth], state uniform in it
    tl = lsrc + 1 + (rng.random(eidx.size) * (depth - lsrc)).astype(np.int64)
    tl = np.minimum(tl, depth)
    u = rng.random(eidx.size)
    edst = np.empty(eidx.size, dtype=np.int64)
    for l in range(1, depth + 1):
        m = tl == l
        pool = by_level[l]
        if m.any():
            if pool.size == 0:
                raise RuntimeError("empty epsilon level; enlarge the graph")
            edst[m] = pool[np.minimum((u[m] * pool.size).astype(np.int64), pool.size - 1)]
    dst[eidx] = edst
    ilabel = np.where(is_eps, 0, rng.integers(1, cfg["P"] + 1, A))
    olabel = np.where(rng.random(A) < 0.9, 0, rng.integers(1, cfg["V"] + 1, A))
    weight = rng.exponential(cfg["wmean"], A).astype(np.float32)
    return dict(row_ptr=row_ptr, dst=dst, ilabel=ilabel, olabel=olabel, weight=weight)


def _pack(g: dict, S: int, final=None) -> dict:
    return dict(num_states=S, start_state=0,
                row_ptr=np.ascontiguousarray(g["row_ptr"], dtype=np.uint32),
                dst=np.ascontiguousarray(g["dst"], dtype=np.uint32),
                ilabel=np.ascontiguousarray(g["ilabel"], dtype=np.int32),
                olabel=np.ascontiguousarray(g["olabel"], dtype=np.int32),
                weight=np.ascontiguousarray(g["weight"], dtype=np.float32),
                final_weight=None if final is None else np.ascontiguousarray(final, dtype=np.float32))


def make_graph(cfg) -> dict:
    """Graph of a workload (dict or name), deterministic in its seed."""
    if isinstance(cfg, str):
        cfg = workload(cfg)
    gcfg = workload(cfg["graph_of"]) if "graph_of" in cfg else cfg
    rng = _rng(1000 * gcfg["index"] + 1)
    if gcfg["family"] == "forward_eps":
        g = _graph_forward_eps(gcfg, rng)
    else:
        g = _graph_zipf_levels(gcfg, rng)
    if cfg.get("dyadic"):
        g["weight"] = _quantize(g["weight"])
    return _pack(g, gcfg["S"])


def _loglikes(cfg: dict, T: int, rng: np.random.Generator) -> np.ndarray:
    P = cfg["P"]
    L = rng.standard_normal((T, P), dtype=np.float32)
    L *= np.float32(cfg["ll_std"])
    L += np.float32(cfg["ll_mean"])
    lo, hi = cfg["peaks"]
    if hi > 0:
        npk = rng.integers(lo, hi + 1, T)
        for t in range(T):
            cols = rng.choice(P, size=int(npk[t]), replace=False)
            L[t, cols] = rng.normal(-2.0, 1.0, cols.size).astype(np.float32)
    if cfg.get("dyadic"):
        L = _quantize(L)
    return np.ascontiguousarray(L)


def make_loglikes(cfg, utt: int | None = None) -> np.ndarray:
    """T x P float32 log-likelihoods of a workload (utterance `utt` of a batch)."""
    if isinstance(cfg, str):
        cfg = workload(cfg)
    seed = 1000 * cfg["index"] + 2
    if "batch" in cfg:
        if utt is None:
            raise ValueError("batch workload: pass utt")
        T = batch_lengths(cfg)[utt]
        seed += 100 + utt
    else:
        T = cfg["T"]
    return _loglikes(cfg, T, _rng(seed))


def batch_lengths(cfg) -> list[int]:
    if isinstance(cfg, str):
        cfg = workload(cfg)
    lo, hi = cfg["T_range"]
    rng = _rng(1000 * cfg["index"] + 3)
    return [int(x) for x in rng.integers(lo, hi + 1, cfg["batch"])]


def make_batch(cfg) -> list[np.ndarray]:
    if isinstance(cfg, str):
        cfg = workload(cfg)
    return [make_loglikes(cfg, i) for i in range(cfg["batch"])]


def tiny_graph(seed: int, S: int = 6, A: int = 14, eps_frac: float = 0.3, P: int = 4,
               V: int = 5, finals: bool = False, dyadic: bool = False,
               wmean: float = 1.0) -> dict:
    """Small random graph for exhaustive checks.  Epsilon arcs go to higher
    state ids (acyclic); every state gets at least one arc when A >= S."""
    rng = _rng(seed)
    src = np.concatenate([np.arange(min(S, A)), rng.integers(0, S, max(0, A - S))])
    src.sort()
    deg = np.bincount(src, minlength=S)
    row_ptr = np.zeros(S + 1, dtype=np.int64)
    np.cumsum(deg, out=row_ptr[1:])
    is_eps = (rng.random(A) < eps_frac) & (src < S - 1)
    dst = rng.integers(0, S, A)
    eps_dst = src + 1 + (rng.random(A) * (S - 1 - src)).astype(np.int64)
    dst = np.where(is_eps, np.minimum(eps_dst, S - 1), dst)
    ilabel = np.where(is_eps, 0, rng.integers(1, P + 1, A))
    olabel = np.where(rng.random(A) < 0.5, 0, rng.integers(1, V + 1, A))
    weight = rng.exponential(wmean, A).astype(np.float32)
    if dyadic:
        weight = _quantize(weight)
        # keep a fair share of exact ties
        weight = np.where(rng.random(A) < 0.3, np.float32(0.5), weight).astype(np.float32)
    final = None
    if finals:
        final = np.where(rng.random(S) < 0.5, rng.exponential(wmean, S), np.inf).astype(np.float32)
        if dyadic:
            final = np.where(np.isfinite(final), _quantize(final), final).astype(np.float32)
    return _pack(dict(row_ptr=row_ptr, dst=dst, ilabel=ilabel, olabel=olabel, weight=weight),
                 S, final)


def tiny_loglikes(seed: int, T: int, P: int, dyadic: bool = False) -> np.ndarray:
    rng = _rng(seed)
    L = rng.normal(-2.0, 1.5, (T, P)).astype(np.float32)
    if dyadic:
        L = _quantize(L)
        L = np.where(rng.random((T, P)) < 0.3, np.float32(-1.0), L).astype(np.float32)
    return np.ascontiguousarray(L)
