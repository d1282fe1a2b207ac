"""Checks a decode result against the conditions that define it, frame by
frame, from the result's own dump of surviving tokens (per frame sorted by
state), cutoffs and raw lattice.  None of this recomputes the decode: each
frame is checked given the previous frame's surviving set, so a wrong term,
sign, index or cutoff anywhere in the decoder breaks one of the equalities.

Used on the oracle (its debug output) and, with the same arrays, on the GPU
library.
"""
from __future__ import annotations

import numpy as np

f32 = np.float32
NONE = np.uint32(0xFFFFFFFF)


def _canon(x):
    x = np.asarray(x, dtype=f32).copy()
    x[x == 0] = f32(0.0)
    return x


def _bits(x):
    return np.asarray(x, dtype=f32).view(np.uint32)


class Graph:
    def __init__(self, g):
        self.S = int(g["num_states"])
        self.s0 = int(g.get("start_state", 0))
        self.rp = g["row_ptr"].astype(np.int64)
        self.dst = g["dst"].astype(np.int64)
        self.il = g["ilabel"].astype(np.int64)
        self.ol = g["olabel"].astype(np.int64)
        self.w = g["weight"].astype(f32)
        self.fw = g.get("final_weight")
        self.deg = np.diff(self.rp)
        self.src = np.repeat(np.arange(self.S), self.deg)

    def out_arcs(self, states):
        """Arc ids of all out-arcs of `states` and the index of their state."""
        states = np.asarray(states, dtype=np.int64)
        d = self.deg[states]
        owner = np.repeat(np.arange(states.size), d)
        start = np.repeat(self.rp[states], d)
        first = np.repeat(np.cumsum(d) - d, d)
        arcs = start + (np.arange(owner.size) - first)
        return arcs, owner


def frame_slices(toks, T):
    return np.searchsorted(toks["t"], np.arange(T + 2), side="left")


def lexmin(dst, x, arc):
    """Per destination: the candidate with the smallest (x, arc)."""
    if dst.size == 0:
        return np.zeros(0, np.int64), np.zeros(0, f32), np.zeros(0, np.int64)
    o = np.lexsort((arc, x, dst))
    d, xx, aa = dst[o], x[o], arc[o]
    first = np.ones(d.size, bool)
    first[1:] = d[1:] != d[:-1]
    return d[first], xx[first], aa[first]


def emitting_candidates(G, L, t, prev):
    arcs, owner = G.out_arcs(prev["state"])
    em = G.il[arcs] != 0
    arcs, owner = arcs[em], owner[em]
    c = prev["cost"][owner].astype(f32)
    ac = (-L[t - 1, G.il[arcs] - 1]).astype(f32)
    x = _canon((c + ac).astype(f32) + G.w[arcs])
    return arcs, owner, x


def eps_candidates(G, cur):
    arcs, owner = G.out_arcs(cur["state"])
    ep = G.il[arcs] == 0
    arcs, owner = arcs[ep], owner[ep]
    x = _canon(cur["cost"][owner].astype(f32) + G.w[arcs])
    return arcs, owner, x


def check_frames(g, L, beam, max_active, toks, best, cutb, cut):
    """Surviving sets: optimality of every token and its predecessor, the beam
    and max-active cutoffs, completeness of every set."""
    G = Graph(g)
    T = L.shape[0]
    off = frame_slices(toks, T)
    assert off[T + 1] == toks.size
    for t in range(T + 1):
        A = toks[off[t]:off[t + 1]]
        assert A.size > 0, f"frame {t}: empty surviving set"
        assert np.all(np.diff(A["state"]) > 0), f"frame {t}: not sorted by state"
        if t == 0:
            d0 = np.array([G.s0]), np.array([f32(0.0)]), np.array([int(NONE)])
            assert best[0] == f32(0.0)
        else:
            P = toks[off[t - 1]:off[t]]
            arcs, owner, x = emitting_candidates(G, L, t, P)
            fin = np.isfinite(x)
            assert fin.any()
            assert best[t] == x[fin].min(), f"frame {t}: best"
            d0 = G.dst[arcs[fin]], x[fin], arcs[fin]
        assert cutb[t] == f32(best[t] + f32(beam)), f"frame {t}: beam cutoff"
        earcs, eowner, ex = eps_candidates(G, A)
        ok = np.isfinite(ex) & (ex <= cutb[t])
        dd = np.concatenate([d0[0], G.dst[earcs[ok]]])
        xx = np.concatenate([np.asarray(d0[1], f32), ex[ok]])
        aa = np.concatenate([np.asarray(d0[2], np.int64), earcs[ok]])
        ds, xs, as_ = lexmin(dd, xx, aa)
        inside = xs <= cut[t]
        assert np.array_equal(ds[inside], A["state"]), f"frame {t}: surviving set"
        assert np.array_equal(_bits(xs[inside]), _bits(A["cost"])), f"frame {t}: token costs"
        assert np.array_equal(as_[inside].astype(np.uint32), A["pred_arc"]), f"frame {t}: preds"
        # cutoffs
        c = A["cost"]
        assert cut[t] <= cutb[t]
        assert np.all(c <= cut[t])
        if max_active > 0 and cut[t] < cutb[t]:
            assert np.any(c == cut[t]), f"frame {t}: max-active cutoff is no token cost"
            assert (c < cut[t]).sum() < max_active <= c.size, f"frame {t}: max-active rank"
        elif max_active > 0:
            assert c.size <= max_active or (c < cutb[t]).sum() < max_active, f"frame {t}: max-active"
        else:
            assert cut[t] == cutb[t]
    return off


def check_links(g, L, toks, cut, raw):
    """The raw lattice is exactly the candidates of surviving sources whose
    cost lies within the frame's final cutoff."""
    G = Graph(g)
    T = L.shape[0]
    off = frame_slices(toks, T)
    exp = []
    for t in range(T + 1):
        A = toks[off[t]:off[t + 1]]
        if t > 0:
            P = toks[off[t - 1]:off[t]]
            arcs, owner, x = emitting_candidates(G, L, t, P)
            k = np.isfinite(x) & (x <= cut[t])
            exp.append(np.stack([np.full(k.sum(), t), arcs[k], P["state"][owner[k]], G.dst[arcs[k]],
                                 _bits(x[k]).astype(np.int64)], 1))
        arcs, owner, x = eps_candidates(G, A)
        k = np.isfinite(x) & (x <= cut[t])
        exp.append(np.stack([np.full(k.sum(), t), arcs[k], A["state"][owner[k]], G.dst[arcs[k]],
                             _bits(x[k]).astype(np.int64)], 1))
    e = np.concatenate(exp) if exp else np.zeros((0, 5), np.int64)
    e = e[np.lexsort((e[:, 1], e[:, 0]))]
    got = np.stack([raw["t"], raw["arc_id"], raw["src_state"], raw["dst_state"],
                    _bits(raw["fwd_cost"]).astype(np.int64)], 1).astype(np.int64)
    assert got.shape == e.shape, f"raw link count {got.shape[0]} != {e.shape[0]}"
    assert np.array_equal(got, e), "raw lattice"
    # per-link fields
    assert np.array_equal(raw["ilabel"], G.il[raw["arc_id"]])
    assert np.array_equal(raw["olabel"], G.ol[raw["arc_id"]])
    assert np.array_equal(_bits(raw["graph_cost"]), _bits(G.w[raw["arc_id"]]))
    em = raw["ilabel"] != 0
    ac = np.zeros(raw.size, f32)
    ac[em] = -L[raw["t"][em] - 1, raw["ilabel"][em] - 1]
    assert np.array_equal(_bits(raw["ac_cost"]), _bits(ac))


def node_index(toks, off, t, states):
    idx = np.searchsorted(toks["state"][off[t]:off[t + 1]], states) + off[t]
    return idx


def check_pruning(g, L, toks, raw, cost, final_reached, lattice_beam, links):
    """Extra costs are the fixpoint of Sec. 3.5's update and the kept links
    are exactly those within the lattice beam."""
    G = Graph(g)
    T = L.shape[0]
    off = frame_slices(toks, T)
    n = toks.size
    src_t = np.where(raw["ilabel"] != 0, raw["t"] - 1, raw["t"])
    si = np.empty(raw.size, np.int64)
    di = np.empty(raw.size, np.int64)
    for t in range(T + 1):
        m = src_t == t
        si[m] = node_index(toks, off, t, raw["src_state"][m])
        m = raw["t"] == t
        di[m] = node_index(toks, off, t, raw["dst_state"][m])
    assert np.array_equal(toks["state"][si], raw["src_state"])
    assert np.array_equal(toks["state"][di], raw["dst_state"])
    E = np.full(n, np.inf, f32)
    AT = toks[off[T]:off[T + 1]]
    if final_reached:
        F = _canon(AT["cost"] + G.fw[AT["state"]].astype(f32))
    else:
        F = AT["cost"].astype(f32)
    fin = np.isfinite(F)
    assert cost == F[fin].min()
    E[off[T]:off[T + 1]][fin] = (F[fin] - f32(cost)).astype(f32)
    np.minimum.at(E, si, raw["extra"].astype(f32))
    le = (E[di] + (raw["fwd_cost"] - toks["cost"][di]).astype(f32)).astype(f32)
    assert np.array_equal(_bits(le), _bits(raw["extra"])), "link extra cost fixpoint"
    keep = np.isfinite(le) & (le <= f32(lattice_beam))
    kk = raw[keep]
    assert kk.size == links.size, f"kept {links.size} != {kk.size}"
    for f in ("t", "arc_id", "src_state", "dst_state"):
        assert np.array_equal(kk[f], links[f]), f
    for f in ("fwd_cost", "extra", "graph_cost", "ac_cost"):
        assert np.array_equal(_bits(kk[f]), _bits(links[f])), f
    return E, si, di, keep


def check_traceback(g, toks, T, cost, final_reached, words):
    G = Graph(g)
    off = frame_slices(toks, T)
    AT = toks[off[T]:off[T + 1]]
    F = _canon(AT["cost"] + G.fw[AT["state"]].astype(f32)) if final_reached else AT["cost"]
    assert cost == F.min()
    b = int(np.flatnonzero(F == F.min())[0])   # lowest state id among the argmin
    t, i = T, off[T] + b
    out = []
    while toks["pred_arc"][i] != NONE:
        a = int(toks["pred_arc"][i])
        if G.ol[a] != 0:
            out.append(int(G.ol[a]))
        if G.il[a] != 0:
            t -= 1
        s = int(G.src[a])
        j = np.searchsorted(toks["state"][off[t]:off[t + 1]], s) + off[t]
        assert j < off[t + 1] and toks["state"][j] == s
        i = j
    assert t == 0 and toks["state"][i] == G.s0
    out.reverse()
    assert list(words) == out, "1-best words"


def check_posteriors(links, T, atol=1e-9):
    em = links["ilabel"] != 0
    sums = np.bincount(links["t"][em], weights=links["posterior"][em], minlength=T + 1)
    assert np.allclose(sums[1:], 1.0, atol=atol, rtol=0), f"posterior sums {sums[1:].min()} {sums[1:].max()}"
    assert np.all(links["posterior"] >= 0) and np.all(links["posterior"] <= 1 + atol)


def check_nodes(toks, links, E, nodes, s0, T):
    off = frame_slices(toks, T)
    keys = set(zip(links["t"].tolist(), links["dst_state"].tolist()))
    src_t = np.where(links["ilabel"] != 0, links["t"] - 1, links["t"])
    keys |= set(zip(src_t.tolist(), links["src_state"].tolist()))
    keys.add((0, s0))
    exp = sorted(keys)
    got = list(zip(nodes["t"].tolist(), nodes["state"].tolist()))
    assert got == exp, "lattice node set"
    idx = np.array([node_index(toks, off, t, np.array([s]))[0] for t, s in exp], np.int64)
    assert np.array_equal(_bits(nodes["cost"]), _bits(toks["cost"][idx]))
    assert np.array_equal(_bits(nodes["extra"]), _bits(E[idx]))


def check_all(g, L, beam, max_active, lattice_beam, r):
    """Every check above on a debug decode result `r` (oracle or library)."""
    T = L.shape[0]
    check_frames(g, L, beam, max_active, r.tokens, r.best, r.cutoff_beam, r.cutoff)
    check_links(g, L, r.tokens, r.cutoff, r.raw_links)
    E, _, _, _ = check_pruning(g, L, r.tokens, r.raw_links, r.cost, r.stats["final_reached"],
                               lattice_beam, r.links)
    check_traceback(g, r.tokens, T, r.cost, r.stats["final_reached"], r.words)
    check_posteriors(r.links, T)
    check_nodes(r.tokens, r.links, E, r.nodes, int(g.get("start_state", 0)), T)
