"""Pins of the lattice-determinisation oracle (oracle/lattice_paths.py): the
hand-worked lattice, path enumeration against the word-constrained dynamic
programme (two independent routes to the same definition), and the best
word sequence against the decoder's 1-best."""
import math

import numpy as np
import pytest

import oracle
import synth
from lattice_det import load_fixture
from oracle import lattice_paths as lp


def test_hand_worked():
    d, links, nodes, nf = load_fixture("det_hand_1.json")
    best, count = lp.best_by_words(links, nodes, d["start_state"], nf)
    assert count == d["paths"]
    exp = {tuple(e["words"]): (e["graph_cost"], e["ac_cost"], tuple(e["string"])) for e in d["expect"]}
    assert best == exp
    for w, v in exp.items():
        assert lp.best_for_words(links, nodes, d["start_state"], nf, w) == v
    assert lp.best_for_words(links, nodes, d["start_state"], nf, (11,)) is None
    assert lp.best_for_words(links, nodes, d["start_state"], nf, (10, 10)) is None


def _decoded(seed, dyadic):
    g = synth.tiny_graph(seed, dyadic=dyadic)
    L = synth.tiny_loglikes(seed, 6, 4, dyadic=dyadic)
    try:
        o = oracle.decode(g, L, 8.0, 0, 5.0)
    except oracle.OracleError:
        return None
    return g, o, lp.node_final_costs(o, g.get("final_weight"))


@pytest.mark.parametrize("dyadic", [True, False])
@pytest.mark.parametrize("seed", range(16))
def test_enumeration_equals_dynamic_programme(seed, dyadic):
    got = _decoded(seed, dyadic)
    if got is None:
        pytest.skip("no surviving path")
    g, o, nf = got
    s0 = g.get("start_state", 0)
    best, count = lp.best_by_words(o.links, o.nodes, s0, nf)
    assert count >= len(best) >= 1
    for w, v in best.items():
        assert lp.best_for_words(o.links, o.nodes, s0, nf, w) == v


@pytest.mark.parametrize("seed", range(16))
def test_best_sequence_is_the_one_best(seed):
    """The best word sequence of the lattice is the decoder's 1-best, and its
    total cost is the 1-best cost up to fp32 rounding of the decoder's sums."""
    got = _decoded(seed, False)
    if got is None:
        pytest.skip("no surviving path")
    g, o, nf = got
    best, _ = lp.best_by_words(o.links, o.nodes, g.get("start_state", 0), nf)
    ranked = sorted(best.items(), key=lambda kv: kv[1][0] + kv[1][1])
    w, (gc, ac, _) = ranked[0]
    assert math.isclose(gc + ac, float(o.cost), rel_tol=1e-5, abs_tol=1e-4)
    if len(ranked) == 1 or (ranked[1][1][0] + ranked[1][1][1]) - (gc + ac) > 1e-3:
        assert list(w) == list(o.words)


def test_no_nodes():
    e = np.zeros(0, oracle.LINK_DTYPE)
    n = np.zeros(0, oracle.NODE_DTYPE)
    assert lp.best_by_words(e, n, 0, []) == ({}, 0)
    assert lp.best_for_words(e, n, 0, [], ()) is None
