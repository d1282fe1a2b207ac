"""Properties of a decode result that hold at any size and need only the
result itself (kept lattice, nodes, words, cost), the graph and the
log-likelihoods — no per-frame token dump and no oracle run.  Used where the
oracle is too slow for the whole utterance (the wide-beam 2M-state graph at
full length), and pinned on the CPU by running it on oracle results.

What is checked (Sec. 3.4-3.5 of the paper, readings as in the oracle):
* every kept link is an arc of the graph between the right states, with the
  graph cost and the acoustic cost -L[t-1][ilabel-1] bit for bit;
* its forward cost is the fp32 sum of its source node's cost and its costs,
  and is not below its destination node's cost (that node is the minimum);
* its extra cost is fl(extra(dst) + fl(x - cost(dst))) bit for bit, within
  the lattice beam;
* every node's extra cost is the minimum over its kept out-links (and, in
  the last frame, its final extra cost);
* the node list is the set of link endpoints plus the start node, in
  (t, state) order;
* per frame, the posteriors of the emitting links sum to 1;
* the best cost is the best final cost of the last frame, and the links with
  extra cost 0 carry the 1-best words from the start node to the end.
"""
from __future__ import annotations

import numpy as np

f32 = np.float32


def _canon(x):
    x = np.asarray(x, dtype=f32).copy()
    x[x == 0] = f32(0.0)
    return x


def _bits(x):
    return np.ascontiguousarray(x, dtype=f32).view(np.uint32)


def check(g, L, lattice_beam, r, post_atol=1e-6):
    links, nodes = r.links, r.nodes
    T = L.shape[0]
    S = int(g["num_states"])
    s0 = int(g.get("start_state", 0))
    row = np.asarray(g["row_ptr"], np.int64)
    src_of = np.repeat(np.arange(S, dtype=np.int64), np.diff(row))
    dst = np.asarray(g["dst"], np.int64)
    il = np.asarray(g["ilabel"], np.int64)
    ol = np.asarray(g["olabel"], np.int64)
    w = np.asarray(g["weight"], f32)
    fw = g.get("final_weight")

    assert r.stats["kept_links"] == len(links) and r.stats["nodes"] == len(nodes)
    # ---- nodes: sorted, unique, the endpoints of the links plus the start
    nkey = nodes["t"].astype(np.int64) * S + nodes["state"]
    assert np.all(np.diff(nkey) > 0), "nodes not in (t, state) order"
    lt = links["t"].astype(np.int64)
    a = links["arc_id"].astype(np.int64)
    emit = il[a] != 0
    src_t = np.where(emit, lt - 1, lt)
    skey = src_t * S + links["src_state"]
    dkey = lt * S + links["dst_state"]
    ends = np.unique(np.concatenate([skey, dkey, [s0]]))
    assert np.array_equal(ends, nkey), "node set != link endpoints + start"
    si = np.searchsorted(nkey, skey)
    di = np.searchsorted(nkey, dkey)
    # ---- links: order, graph fields
    lkey = lt * (1 << 32) + a
    assert np.all(np.diff(lkey) > 0), "links not in (t, arc id) order"
    assert np.array_equal(links["src_state"], src_of[a]) and np.array_equal(links["dst_state"], dst[a])
    assert np.array_equal(links["ilabel"], il[a]) and np.array_equal(links["olabel"], ol[a])
    assert np.array_equal(_bits(links["graph_cost"]), _bits(w[a]))
    ac = np.zeros(len(links), f32)
    ac[emit] = -L[lt[emit] - 1, il[a][emit] - 1]
    assert np.array_equal(_bits(links["ac_cost"]), _bits(ac)), "acoustic costs"
    assert np.all(lt[emit] >= 1)
    # ---- forward costs from the source node
    cs = nodes["cost"][si]
    x = np.where(emit, _canon((cs + ac).astype(f32) + w[a]), _canon(cs + w[a]))
    assert np.array_equal(_bits(links["fwd_cost"]), _bits(x)), "forward costs"
    cd = nodes["cost"][di]
    assert np.all(links["fwd_cost"] >= cd), "a link below its destination token"
    # ---- extra costs
    le = _canon(nodes["extra"][di] + _canon(links["fwd_cost"] - cd))
    assert np.array_equal(_bits(links["extra"]), _bits(le)), "link extra costs"
    assert np.all(links["extra"] <= f32(lattice_beam)) and np.all(np.isfinite(links["extra"]))
    best_out = np.full(len(nodes), np.inf, f32)
    np.minimum.at(best_out, si, links["extra"])
    last = nodes["t"] == T
    final_used = bool(r.stats["final_reached"])
    c_last = nodes["cost"][last]
    if final_used:
        F = _canon(c_last + np.asarray(fw, f32)[nodes["state"][last]])
    else:
        F = c_last
    assert float(r.cost) == float(F.min()), "best cost"
    fin = np.where(np.isfinite(F), _canon(F - f32(r.cost)), np.inf).astype(f32)
    exp = best_out.copy()
    exp[last] = np.minimum(exp[last], fin)
    assert np.array_equal(_bits(nodes["extra"]), _bits(exp)), "node extra = min over kept out-links"
    # ---- posteriors
    sums = np.bincount(lt[emit], weights=links["posterior"][emit], minlength=T + 1)
    assert np.allclose(sums[1:], 1.0, atol=post_atol, rtol=0), (sums[1:].min(), sums[1:].max())
    # ---- the zero-extra path from the start carries the words
    zero = links["extra"] == 0
    order = np.argsort(si[zero], kind="stable")
    zs, zd, zo = si[zero][order], di[zero][order], links["olabel"][zero][order]
    start = int(np.searchsorted(nkey, s0))
    assert nodes["extra"][start] == 0
    out, n, unique = [], start, True
    while True:
        lo, hi = np.searchsorted(zs, n), np.searchsorted(zs, n, side="right")
        if hi == lo:
            break
        if hi - lo > 1:
            unique = False  # tied best paths: words are one of them, not checked
            break
        if zo[lo] != 0:
            out.append(int(zo[lo]))
        n = int(zd[lo])
    if unique:
        assert nodes["t"][n] == T and fin[np.flatnonzero(last).tolist().index(n)] == 0
        assert list(r.words) == out, "1-best words along the zero-extra path"
    return unique
