"""Helpers for the determinised-lattice tests: load lattices from a fixture,
enumerate the paths of a determinised lattice, check its structure, and
compare it with the oracle's best path per word sequence."""
from __future__ import annotations

import json
import math
import os
from types import SimpleNamespace

import numpy as np

import oracle
from oracle import lattice_paths as lp

HERE = os.path.dirname(os.path.abspath(__file__))


def load_fixture(name):
    d = json.load(open(os.path.join(HERE, "golden", name)))
    links = np.zeros(len(d["links"]), oracle.LINK_DTYPE)
    for i, l in enumerate(d["links"]):
        for k, v in l.items():
            links[i][k] = v
    nodes = np.zeros(len(d["nodes"]), oracle.NODE_DTYPE)
    for i, (t, s) in enumerate(d["nodes"]):
        nodes[i]["t"], nodes[i]["state"] = t, s
    nf = np.array([np.inf if v is None else v for v in d["node_final"]], np.float64)
    return d, links, nodes, nf


def paths(c, max_paths=1_000_000):
    """{words: (g, a, string)} of every path of determinised lattice c; a
    word sequence seen twice fails (the lattice would not be deterministic)."""
    by = {}
    for a in c.arcs:
        by.setdefault(int(a["src"]), []).append(a)
    fin = {int(f["state"]): f for f in c.finals}
    al = c.align
    out, stack = {}, [(0, 0.0, 0.0, (), ())] if c.states else []
    while stack:
        u, g, a, s, w = stack.pop()
        if u in fin:
            f = fin[u]
            o, n = int(f["align_off"]), int(f["align_len"])
            assert w not in out, ("word sequence twice", w)
            out[w] = (g + float(f["graph_cost"]), a + float(f["ac_cost"]), s + tuple(int(x) for x in al[o:o + n]))
            assert len(out) <= max_paths
        for e in by.get(u, []):
            o, n = int(e["align_off"]), int(e["align_len"])
            stack.append((int(e["dst"]), g + float(e["graph_cost"]), a + float(e["ac_cost"]),
                          s + tuple(int(x) for x in al[o:o + n]), w + (int(e["word"]),)))
    return out


def check_structure(c):
    """Deterministic on words, no word 0, arcs sorted by (src, word), every
    state reachable from state 0 and leading to a final state."""
    if c.states == 0:
        assert len(c.arcs) == 0 and len(c.finals) == 0
        return
    a = c.arcs
    assert np.all(a["word"] > 0)
    key = a["src"].astype(np.int64) * (1 << 32) + a["word"]
    assert np.all(np.diff(key) > 0), "arcs not sorted by (src, word) or a word repeats"
    assert np.all((a["src"] >= 0) & (a["src"] < c.states) & (a["dst"] >= 0) & (a["dst"] < c.states))
    fwd = {0}
    adj, radj = {}, {}
    for s, d in zip(a["src"], a["dst"]):
        adj.setdefault(int(s), []).append(int(d))
        radj.setdefault(int(d), []).append(int(s))
    todo = [0]
    while todo:
        u = todo.pop()
        for v in adj.get(u, []):
            if v not in fwd:
                fwd.add(v)
                todo.append(v)
    assert len(fwd) == c.states, "unreachable states"
    back = set(int(f["state"]) for f in c.finals)
    todo = list(back)
    while todo:
        u = todo.pop()
        for v in radj.get(u, []):
            if v not in back:
                back.add(v)
                todo.append(v)
    assert len(back) == c.states, "states that reach no final state"


def assert_matches(got, best, exact=True, rtol=1e-9):
    """got, best: {words: (g, a, string)}.  exact: dyadic inputs, every sum
    is exact.  Otherwise totals within rtol and strings equal."""
    assert set(got) == set(best), (len(got), len(best), sorted(set(got) ^ set(best))[:5])
    for w, (g, a, s) in best.items():
        gg, ga, gs = got[w]
        if exact:
            assert (gg, ga, gs) == (g, a, s), (w, got[w], best[w])
        else:
            assert math.isclose(gg + ga, g + a, rel_tol=rtol, abs_tol=1e-9), (w, got[w], best[w])
            assert gs == s, (w, gs, s)


def lattice_of(result, start_state, final_weight):
    return SimpleNamespace(links=result.links, nodes=result.nodes, start=int(start_state),
                           node_final=lp.node_final_costs(result, final_weight))
