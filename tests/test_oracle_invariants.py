"""The oracle with finite beam and max-active: every frame is checked against
the conditions that define it (token optimality and predecessor tie-break,
beam and max-active cutoffs, completeness, the raw-lattice definition, the
extra-cost fixpoint, the traceback, posterior normalisation)."""
import math

import numpy as np
import pytest

import invariants
import synth

INF = math.inf


@pytest.mark.parametrize("beam,max_active,lattice_beam", [
    (10.0, 2000, 6.0),      # the tiny_10k workload's own settings
    (10.0, 40, 6.0),        # max-active binds
    (4.0, 0, 2.0),
    (25.0, 150, INF),
    (2.0, 5, 0.0),          # very narrow
])
def test_tiny_10k(oracle_mod, beam, max_active, lattice_beam):
    cfg = synth.workload("tiny_10k")
    g = synth.make_graph(cfg)
    L = synth.make_loglikes(cfg)[:120]
    r = oracle_mod.decode(g, L, beam, max_active, lattice_beam, debug=True)
    invariants.check_all(g, L, beam, max_active, lattice_beam, r)


@pytest.mark.parametrize("seed", range(12))
def test_random_medium(oracle_mod, seed):
    rng = np.random.default_rng(seed)
    dyadic = seed % 3 == 0
    g = synth.tiny_graph(500 + seed, S=150, A=520, eps_frac=0.25, P=12, V=20,
                         finals=seed % 2 == 1, dyadic=dyadic)
    L = synth.tiny_loglikes(600 + seed, 40, 12, dyadic=dyadic)
    beam = float(rng.choice([2.0, 5.0, 9.0, INF]))
    max_active = int(rng.choice([0, 5, 30]))
    lb = float(rng.choice([0.0, 1.0, 4.0, INF]))
    r = oracle_mod.decode(g, L, beam, max_active, lb, debug=True)
    invariants.check_all(g, L, beam, max_active, lb, r)


def test_wide_2m_dyadic_prefix(oracle_mod):
    """A few frames of the wide-beam workload with dyadic inputs: tens of
    thousands of tokens, exact cost ties, depth-8 epsilon chains."""
    cfg = synth.workload("wide_2m_dyadic")
    g = synth.make_graph(cfg)
    L = synth.make_loglikes(cfg)[:3]
    r = oracle_mod.decode(g, L, cfg["beam"], cfg["max_active"], cfg["lattice_beam"], debug=True)
    assert r.stats["max_tokens"] > 10000
    invariants.check_all(g, L, cfg["beam"], cfg["max_active"], cfg["lattice_beam"], r)


def test_hclg_5m_prefix_max_active(oracle_mod):
    cfg = synth.workload("hclg_5m")
    g = synth.make_graph(cfg)
    L = synth.make_loglikes(cfg)[:25]
    r = oracle_mod.decode(g, L, cfg["beam"], 60, cfg["lattice_beam"], debug=True)
    invariants.check_all(g, L, cfg["beam"], 60, cfg["lattice_beam"], r)


def test_zero_frames(oracle_mod):
    """T = 0: the result is the epsilon closure of the start state."""
    g = synth.tiny_graph(77, S=6, A=14, eps_frac=0.6, P=3, finals=True)
    L = np.zeros((0, 3), np.float32)
    r = oracle_mod.decode(g, L, INF, 0, INF, debug=True)
    assert r.stats["frames"] == 0
    invariants.check_all(g, L, INF, 0, INF, r)


def test_beam_monotone(oracle_mod):
    """A wider beam keeps a superset of each frame's tokens when nothing else
    prunes and the narrower decode's tokens keep their costs."""
    g = synth.tiny_graph(91, S=120, A=400, eps_frac=0.2, P=8)
    L = synth.tiny_loglikes(92, 25, 8)
    a = oracle_mod.decode(g, L, 3.0, 0, INF, debug=True)
    b = oracle_mod.decode(g, L, 30.0, 0, INF, debug=True)
    assert float(b.cost) <= float(a.cost)
    ka = set(zip(a.tokens["t"].tolist(), a.tokens["state"].tolist()))
    kb = set(zip(b.tokens["t"].tolist(), b.tokens["state"].tolist()))
    assert ka <= kb
