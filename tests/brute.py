"""Exhaustive path enumeration on tiny graphs: an independent check of the
oracle with infinite beams.

Every complete path (one emitting arc per frame, any acyclic run of epsilon
arcs inside a frame) is costed in fp32 in the fixed per-arc order
x = fl(fl(c + ac) + w) (emitting) / fl(c + w) (epsilon).  From whole paths this
derives the best cost, each token's best cost and predecessor (lowest arc id
among the candidates reaching that cost), link extra costs (best complete path
through the link minus the best overall) and fp64 posteriors (path sums).
"""
from __future__ import annotations

import math
from collections import defaultdict

import numpy as np

f32 = np.float32


def _canon(x):
    return f32(0.0) if x == 0 else x


def enumerate_paths(g: dict, L: np.ndarray, limit: int = 300_000):
    """All complete paths as lists of (t, arc, x) with x the fp32 cost after
    the arc; the first element is the start token (0, None, 0.0)."""
    S = g["num_states"]
    rp, dst, il, w = g["row_ptr"], g["dst"], g["ilabel"], g["weight"]
    T = L.shape[0]
    out = []

    def rec(t, s, c, path):
        if len(out) > limit:
            raise RuntimeError("too many paths")
        if t == T:
            out.append(list(path))
        for a in range(int(rp[s]), int(rp[s + 1])):
            if il[a] == 0:
                x = _canon(f32(c + w[a]))
                if not np.isfinite(x):
                    continue
                path.append((t, a, x))
                rec(t, int(dst[a]), x, path)
                path.pop()
            elif t < T:
                ac = f32(-L[t, il[a] - 1])
                x = f32(c + ac)
                x = _canon(f32(x + w[a]))
                if not np.isfinite(x):
                    continue
                path.append((t + 1, a, x))
                rec(t + 1, int(dst[a]), x, path)
                path.pop()

    s0 = int(g.get("start_state", 0))
    rec(0, s0, f32(0.0), [(0, None, f32(0.0))])
    del S
    return out


def arc_src(g, a):
    return int(np.searchsorted(g["row_ptr"], a, side="right") - 1)


def brute_decode(g: dict, L: np.ndarray, lattice_beam: float = math.inf):
    """Infinite-beam decode by enumeration.  Returns a dict with cost, words,
    node costs, links {(t, arc): (src, dst, x, extra)}, kept set and fp64
    posteriors of the kept links."""
    paths = enumerate_paths(g, L)
    if not paths:
        raise RuntimeError("no complete path")
    il, ol, dst, w = g["ilabel"], g["olabel"], g["dst"], g["weight"]
    fw = g.get("final_weight")
    s0 = int(g.get("start_state", 0))
    T = L.shape[0]

    def end_state(p):
        t, a, x = p[-1]
        return s0 if a is None else int(dst[a])

    # final costs: finals are used when some reachable end state is final
    final_used = False
    if fw is not None:
        for p in paths:
            s = end_state(p)
            if np.isfinite(fw[s]) and np.isfinite(f32(p[-1][2] + fw[s])):
                final_used = True
                break

    def F(p):
        s = end_state(p)
        c = p[-1][2]
        return _canon(f32(c + fw[s])) if final_used else c

    Fs = [F(p) for p in paths]
    best = min(Fs)

    # token costs: min prefix cost reaching (t, s)
    node_cost = {}
    for p in paths:
        s = s0
        for (t, a, x) in p:
            if a is not None:
                s = int(dst[a])
            key = (t, s)
            if key not in node_cost or x < node_cost[key]:
                node_cost[key] = x
    # predecessor: lowest arc id among candidates reaching the token's cost
    # (candidates from the best costs of the source tokens)
    cands = defaultdict(list)
    for p in paths:
        s = s0
        for (t, a, x) in p:
            if a is None:
                continue
            src_t = t if il[a] == 0 else t - 1
            src = arc_src(g, a)
            cs = node_cost[(src_t, src)]
            if il[a] == 0:
                xc = _canon(f32(cs + w[a]))
            else:
                xc = _canon(f32(f32(cs + f32(-L[t - 1, il[a] - 1])) + w[a]))
            cands[(t, int(dst[a]))].append((xc, a, src_t, src))
    pred = {}
    for key, lst in cands.items():
        c = node_cost[key]
        ok = [e for e in lst if e[0] == c]
        assert ok, "token cost must be reached by a candidate"
        e = min(ok, key=lambda e: e[1])
        pred[key] = e
    # best end state: lowest state id among the argmin
    ends = sorted({end_state(p) for p, f in zip(paths, Fs) if f == best})
    b = ends[0]
    words = []
    key = (T, b)
    while key in pred:
        xc, a, src_t, src = pred[key]
        if ol[a] != 0:
            words.append(int(ol[a]))
        key = (src_t, src)
    assert key == (0, s0)
    words.reverse()

    # links: (t, arc) of every candidate from a reachable source (x from the
    # source's best cost); extra = best complete path through it minus best
    links = {}
    for key, lst in cands.items():
        for (xc, a, src_t, src) in lst:
            links[(key[0], a)] = (src, key[1], xc)
    through = {}
    for p, f in zip(paths, Fs):
        if not np.isfinite(f):
            continue
        for (t, a, x) in p:
            if a is None:
                continue
            k = (t, a)
            if k not in through or f < through[k]:
                through[k] = f
    extra = {k: (float(through[k]) - float(best)) if k in through else math.inf for k in links}
    kept = {k for k, e in extra.items() if e <= lattice_beam and np.isfinite(e)}

    # posteriors over complete paths made only of kept links (fp64)
    def pcost(p):
        tot = 0.0
        for (t, a, x) in p:
            if a is None:
                continue
            tot += float(w[a])
            if il[a] != 0:
                tot += -float(L[t - 1, il[a] - 1])
        s = end_state(p)
        tot += float(fw[s]) if final_used else 0.0
        return tot

    kp = [p for p in paths if all(a is None or (t, a) in kept for (t, a, x) in p)]
    kp = [p for p in kp if np.isfinite(pcost(p))]
    post = {}
    if kp:
        costs = np.array([pcost(p) for p in kp])
        m = costs.min()
        wts = np.exp(-(costs - m))
        Z = wts.sum()
        acc = defaultdict(float)
        for p, wt in zip(kp, wts):
            for (t, a, x) in p:
                if a is not None:
                    acc[(t, a)] += wt
        post = {k: acc[k] / Z for k in kept}
    return dict(cost=best, words=words, node_cost=node_cost, pred=pred, links=links,
                extra=extra, kept=kept, post=post, final_used=final_used, npaths=len(paths))
