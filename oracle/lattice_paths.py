"""Oracle of lattice determinisation (test infrastructure, like the rest of
this package: only tests, the smoke check and the CPU baseline use it).

The compact "exact lattice" of Sec. 3.4 (after Povey et al. 2012) keeps, for
every word sequence of the pruned state-level lattice, the best path with
that word sequence: its weight (graph cost, acoustic cost) and its string
(the ilabels of its emitting links in frame order).  This module writes that
definition out directly, with no determinisation at all:

* `best_by_words` enumerates every path from the start node to a final node
  (pure Python; small lattices only) and keeps the best per word sequence;
* `best_for_words` finds the best path carrying one given word sequence by
  dynamic programming over (lattice node, words consumed), for lattices of
  any size.

Path weights are sums in double in path order.  "Best": lower total (graph +
acoustic), then the lexicographically smaller string, then the lower graph
cost.  Every path reaching a node of frame t has exactly t emitting links, so
strings compared at one node have equal length and the order survives
extension, which is what makes the dynamic programme exact.  A link runs from
node (t-1, src_state) when its ilabel is nonzero, else from (t, src_state),
to (t, dst_state); the start node is (0, start_state).
"""
from __future__ import annotations

import math

import numpy as np


class TooManyPaths(RuntimeError):
    pass


def _graph(links, nodes):
    index = {(int(t), int(s)): i for i, (t, s) in enumerate(zip(nodes["t"], nodes["state"]))}
    out = [[] for _ in range(len(nodes))]
    for l in links:
        t = int(l["t"])
        il = int(l["ilabel"])
        u = index[(t - 1 if il != 0 else t, int(l["src_state"]))]
        v = index[(t, int(l["dst_state"]))]
        out[u].append((v, int(l["olabel"]), il, float(l["graph_cost"]), float(l["ac_cost"])))
    return index, out


def _better(x, y):
    """x, y: (g, a, string); True if x is better than y."""
    tx, ty = x[0] + x[1], y[0] + y[1]
    if tx != ty:
        return tx < ty
    if x[2] != y[2]:
        return x[2] < y[2]
    return x[0] < y[0]


def best_by_words(links, nodes, start_state, node_final, max_paths=200_000):
    """{word tuple: (g, a, string tuple)} over every start-to-final path, and
    the number of such paths.  node_final[i]: final graph cost of node i
    (+inf: not final)."""
    if len(nodes) == 0:
        return {}, 0
    index, out = _graph(links, nodes)
    start = index[(0, int(start_state))]
    best, count = {}, 0
    # iterative depth-first search: (node, g, a, string, words, next arc)
    stack = [(start, 0.0, 0.0, (), (), 0)]
    while stack:
        u, g, a, s, w, k = stack.pop()
        if k == 0 and math.isfinite(float(node_final[u])):
            count += 1
            if count > max_paths:
                raise TooManyPaths(f"more than {max_paths} paths")
            cand = (g + float(node_final[u]), a, s)
            if w not in best or _better(cand, best[w]):
                best[w] = cand
        if k < len(out[u]):
            stack.append((u, g, a, s, w, k + 1))
            v, word, il, ag, aa = out[u][k]
            stack.append((v, g + ag, a + aa, s + ((il,) if il else ()), w + ((word,) if word else ()), 0))
    return best, count


def best_for_words(links, nodes, start_state, node_final, words):
    """(g, a, string tuple) of the best start-to-final path whose nonzero
    olabels are exactly `words`, or None."""
    words = tuple(int(x) for x in words)
    if len(nodes) == 0:
        return None
    index, out = _graph(links, nodes)
    n = len(nodes)
    # topological order: frames ascend; inside a frame, Kahn's algorithm
    indeg = [0] * n
    for u in range(n):
        for v, *_ in out[u]:
            indeg[v] += 1
    order = [u for u in range(n) if indeg[u] == 0]
    for u in order:
        for v, *_ in out[u]:
            indeg[v] -= 1
            if indeg[v] == 0:
                order.append(v)
    if len(order) != n:
        raise ValueError("lattice has a cycle")
    K = len(words)
    best = [dict() for _ in range(n)]  # node -> {k: (g, a, string)}
    best[index[(0, int(start_state))]][0] = (0.0, 0.0, ())
    result = None
    for u in order:
        for k, (g, a, s) in best[u].items():
            if k == K and math.isfinite(float(node_final[u])):
                cand = (g + float(node_final[u]), a, s)
                if result is None or _better(cand, result):
                    result = cand
            for v, word, il, ag, aa in out[u]:
                k2 = k
                if word:
                    if k == K or words[k] != word:
                        continue
                    k2 = k + 1
                cand = (g + ag, a + aa, s + ((il,) if il else ()))
                if k2 not in best[v] or _better(cand, best[v][k2]):
                    best[v][k2] = cand
    return result


def node_final_costs(result, final_weight=None):
    """Final graph cost per node of a decode result: the last frame's nodes
    are final with the graph's final weights when the decode used them,
    else with cost 0; other nodes are not final."""
    nodes = result.nodes
    T = int(result.stats["frames"])
    nf = np.full(len(nodes), np.inf)
    last = nodes["t"] == T
    if final_weight is not None and result.stats["final_reached"]:
        nf[last] = np.asarray(final_weight, np.float32)[nodes["state"][last]].astype(np.float64)
    else:
        nf[last] = 0.0
    return nf
