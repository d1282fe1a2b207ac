"""Lattice determinisation (wd_lattice_determinize, host code of the
library) against its oracle: every word sequence of the input once, with the
best input path's weight and string.  Inputs are lattices from the CPU
oracle decoder (the GPU decoder's lattices are identical to them, which the
GPU parity tests check; tests/test_gpu_determinize.py repeats these checks
on GPU lattices)."""
import math

import numpy as np
import pytest

import oracle
import synth
from lattice_det import assert_matches, check_structure, load_fixture, paths
from oracle import lattice_paths as lp


@pytest.fixture(scope="module")
def wf():
    from paper_1804_03243_amd import wfstdec
    wfstdec.lib()
    return wfstdec


def test_hand_worked(wf):
    d, links, nodes, nf = load_fixture("det_hand_1.json")
    c = wf.wd_lattice_determinize(links, nodes, d["start_state"], nf)
    check_structure(c)
    exp = {tuple(e["words"]): (e["graph_cost"], e["ac_cost"], tuple(e["string"])) for e in d["expect"]}
    assert paths(c) == exp


@pytest.mark.parametrize("dyadic", [True, False])
@pytest.mark.parametrize("seed", range(40))
def test_tiny_random(wf, seed, dyadic):
    g = synth.tiny_graph(seed, dyadic=dyadic, finals=seed % 2 == 1)
    L = synth.tiny_loglikes(seed, 6 + seed % 5, 4, dyadic=dyadic)
    try:
        o = oracle.decode(g, L, 8.0, 0, 5.0)
    except oracle.OracleError:
        pytest.skip("no surviving path")
    s0, fw = g.get("start_state", 0), g.get("final_weight")
    nf = lp.node_final_costs(o, fw)
    try:
        best, _ = lp.best_by_words(o.links, o.nodes, s0, nf)
    except lp.TooManyPaths:
        best = None
    c = wf.determinize(o, s0, fw)
    check_structure(c)
    got = paths(c)
    if best is None:
        # too many input paths to enumerate: each output sequence against the
        # best input path with exactly those words (a DP over the lattice),
        # and the decode's 1-best among them
        best = {w: lp.best_for_words(o.links, o.nodes, s0, nf, w) for w in got}
        assert tuple(int(x) for x in o.words) in got
    assert_matches(got, best, exact=dyadic)


@pytest.mark.parametrize("T", [5, 15, 40])
def test_tiny_10k_prefix(wf, T):
    cfg = synth.workload("tiny_10k")
    g = synth.make_graph(cfg)
    L = synth.make_loglikes(cfg)[:T]
    o = oracle.decode(g, L, cfg["beam"], cfg["max_active"], 3.0)
    s0, fw = g.get("start_state", 0), g.get("final_weight")
    nf = lp.node_final_costs(o, fw)
    best, count = lp.best_by_words(o.links, o.nodes, s0, nf)
    c = wf.determinize(o, s0, fw)
    check_structure(c)
    assert_matches(paths(c), best, exact=False)


def best_path(c):
    """(total, words) of the best path of a determinised lattice (DP over a
    topological order)."""
    n = c.states
    indeg = np.zeros(n, np.int64)
    np.add.at(indeg, c.arcs["dst"], 1)
    by = {}
    for a in c.arcs:
        by.setdefault(int(a["src"]), []).append(a)
    order = [u for u in range(n) if indeg[u] == 0]
    for u in order:
        for a in by.get(u, []):
            indeg[int(a["dst"])] -= 1
            if indeg[int(a["dst"])] == 0:
                order.append(int(a["dst"]))
    assert len(order) == n
    best = {0: (0.0, ())}
    fin = {int(f["state"]): float(f["graph_cost"] + f["ac_cost"]) for f in c.finals}
    out = None
    for u in order:
        if u not in best:
            continue
        cu, wu = best[u]
        if u in fin and (out is None or cu + fin[u] < out[0]):
            out = (cu + fin[u], wu)
        for a in by.get(u, []):
            v, cv = int(a["dst"]), cu + float(a["graph_cost"] + a["ac_cost"])
            if v not in best or cv < best[v][0]:
                best[v] = (cv, wu + (int(a["word"]),))
    return out


def random_paths(c, k, seed):
    """k random start-to-final paths of a determinised lattice: (words, g, a,
    string)."""
    rng = np.random.default_rng(seed)
    by = {}
    for a in c.arcs:
        by.setdefault(int(a["src"]), []).append(a)
    fin = {int(f["state"]): f for f in c.finals}
    out = []
    for _ in range(k):
        u, g, a, s, w = 0, 0.0, 0.0, (), ()
        while True:
            arcs = by.get(u, [])
            if u in fin and (not arcs or rng.random() < 1.0 / (len(arcs) + 1)):
                f = fin[u]
                o, n = int(f["align_off"]), int(f["align_len"])
                out.append((w, g + float(f["graph_cost"]), a + float(f["ac_cost"]),
                            s + tuple(int(x) for x in c.align[o:o + n])))
                break
            e = arcs[int(rng.integers(len(arcs)))]
            o, n = int(e["align_off"]), int(e["align_len"])
            u, g, a = int(e["dst"]), g + float(e["graph_cost"]), a + float(e["ac_cost"])
            s, w = s + tuple(int(x) for x in c.align[o:o + n]), w + (int(e["word"]),)
    return out


def check_large(c, result, s0, fw, k=12, seed=0):
    """Lattices too large to enumerate: structure; the best path is the
    decoder's 1-best; sampled paths carry the best weight and string for
    their words (the oracle's dynamic programme, one sequence at a time)."""
    check_structure(c)
    total, words = best_path(c)
    assert math.isclose(total, float(result.cost), rel_tol=1e-5, abs_tol=1e-3)
    assert list(words) == list(result.words)
    nf = lp.node_final_costs(result, fw)
    for w, g, a, s in random_paths(c, k, seed):
        b = lp.best_for_words(result.links, result.nodes, s0, nf, w)
        assert b is not None
        assert math.isclose(g + a, b[0] + b[1], rel_tol=1e-9, abs_tol=1e-9), (w, g + a, b)
        assert s == b[2]


def test_tiny_10k_full(wf):
    cfg = synth.workload("tiny_10k")
    g = synth.make_graph(cfg)
    L = synth.make_loglikes(cfg)
    o = oracle.decode(g, L, cfg["beam"], cfg["max_active"], cfg["lattice_beam"])
    s0, fw = g.get("start_state", 0), g.get("final_weight")
    c = wf.determinize(o, s0, fw)
    check_large(c, o, s0, fw)


def test_errors(wf):
    d, links, nodes, nf = load_fixture("det_hand_1.json")
    with pytest.raises(wf.WdError) as e:
        wf.wd_lattice_determinize(links, nodes[::-1].copy(), 0, nf[::-1].copy())
    assert e.value.status == wf.WD_EINVAL                 # nodes not sorted
    bad = links.copy()
    bad[0]["dst_state"] = 99
    with pytest.raises(wf.WdError) as e:
        wf.wd_lattice_determinize(bad, nodes, 0, nf)
    assert e.value.status == wf.WD_EINVAL                 # a link to no node
    cyc = np.concatenate([links, links[2:3]])
    cyc[-1]["src_state"], cyc[-1]["dst_state"] = 4, 1     # epsilon link back: a cycle
    with pytest.raises(wf.WdError) as e:
        wf.wd_lattice_determinize(cyc, nodes, 0, nf)
    assert e.value.status == wf.WD_EINVAL
    with pytest.raises(wf.WdError) as e:
        wf.wd_lattice_determinize(links, nodes, 0, nf, max_states=1)
    assert e.value.status == wf.WD_ECAPACITY
    with pytest.raises(wf.WdError) as e:
        wf.wd_lattice_determinize(links, nodes, 7, nf)   # no start node
    assert e.value.status == wf.WD_EINVAL
    c = wf.wd_lattice_determinize(links[:0], nodes[:0], 0, nf[:0])
    assert c.states == 0 and len(c.arcs) == 0


@pytest.mark.parametrize("beam", [0.0, 0.5, 2.0, 5.0])
@pytest.mark.parametrize("seed", range(20))
def test_beam_keeps_every_sequence_within_it(wf, seed, beam):
    """Pruned determinisation: every word sequence whose best path is within
    the beam of the best path is kept, with that best path (dyadic inputs:
    exact); a sequence beyond the beam may appear, with a path beyond it."""
    g = synth.tiny_graph(seed, dyadic=True, finals=seed % 2 == 1)
    L = synth.tiny_loglikes(seed, 6 + seed % 5, 4, dyadic=True)
    try:
        o = oracle.decode(g, L, 8.0, 0, 5.0)
    except oracle.OracleError:
        pytest.skip("no surviving path")
    s0, fw = g.get("start_state", 0), g.get("final_weight")
    nf = lp.node_final_costs(o, fw)
    try:
        best, _ = lp.best_by_words(o.links, o.nodes, s0, nf)
    except lp.TooManyPaths:
        best = None
    c = wf.determinize(o, s0, fw, beam=beam)
    check_structure(c)
    got = paths(c)
    if best is None:
        # too many input paths to enumerate: the 1-best sequence is kept, and
        # each kept sequence is checked against the best input path of its
        # words (a DP over the lattice) as below
        one = tuple(int(x) for x in o.words)
        assert one in got
        b1 = lp.best_for_words(o.links, o.nodes, s0, nf, one)
        top = b1[0] + b1[1]
        for w, v in got.items():
            bw = lp.best_for_words(o.links, o.nodes, s0, nf, w)
            if bw[0] + bw[1] <= top + beam:
                assert v == bw, (w, v, bw)
            else:
                assert v[0] + v[1] > top + beam and v[0] + v[1] >= bw[0] + bw[1]
        return
    top = min(v[0] + v[1] for v in best.values())
    within = {w for w, v in best.items() if v[0] + v[1] <= top + beam}
    assert within <= set(got)
    for w, v in got.items():
        if w in within:
            assert v == best[w], (w, v, best[w])
        else:
            assert v[0] + v[1] > top + beam and v[0] + v[1] >= best[w][0] + best[w][1]


def test_beam_on_a_longer_lattice(wf):
    cfg = synth.workload("tiny_10k")
    g = synth.make_graph(cfg)
    L = synth.make_loglikes(cfg)
    o = oracle.decode(g, L, cfg["beam"], cfg["max_active"], cfg["lattice_beam"])
    s0, fw = g.get("start_state", 0), g.get("final_weight")
    c = wf.determinize(o, s0, fw, beam=1.0)
    check_structure(c)
    total, words = best_path(c)
    assert list(words) == list(o.words)
    assert math.isclose(total, float(o.cost), rel_tol=1e-5, abs_tol=1e-3)


def test_beam_errors(wf):
    d, links, nodes, nf = load_fixture("det_hand_1.json")
    for beam in (-1.0, float("nan")):
        with pytest.raises(wf.WdError) as e:
            wf.wd_lattice_determinize(links, nodes, 0, nf, beam=beam)
        assert e.value.status == wf.WD_EINVAL
    # beam 0 on the hand-worked lattice: (10, 11) costs 4.25, (10,) 5.5
    c = wf.wd_lattice_determinize(links, nodes, 0, nf, beam=0.0)
    assert set(paths(c)) >= {(10, 11)}
