"""The size-independent lattice property checker (used on the GPU at full
size) holds on oracle results, and fails on a lattice with a planted fault."""
import math

import numpy as np
import pytest

import lattice_props
import synth

INF = math.inf


@pytest.mark.parametrize("seed", range(6))
def test_props_on_oracle_medium(oracle_mod, seed):
    rng = np.random.default_rng(seed)
    g = synth.tiny_graph(500 + seed, S=150, A=520, eps_frac=0.25, P=12, V=20, finals=seed % 2 == 1)
    L = synth.tiny_loglikes(600 + seed, 40, 12)
    beam = float(rng.choice([5.0, 9.0, INF]))
    lb = float(rng.choice([1.0, 4.0, INF]))
    o = oracle_mod.decode(g, L, beam, 0, lb)
    lattice_props.check(g, L, lb, o)


@pytest.mark.parametrize("beam,ma,lb", [(10.0, 2000, 6.0), (4.0, 0, 2.0), (25.0, 150, INF)])
def test_props_on_oracle_tiny_10k(oracle_mod, beam, ma, lb):
    cfg = synth.workload("tiny_10k")
    g = synth.make_graph(cfg)
    L = synth.make_loglikes(cfg)
    o = oracle_mod.decode(g, L, beam, ma, lb)
    assert lattice_props.check(g, L, lb, o)


@pytest.mark.parametrize("field,delta", [("fwd_cost", 1e-3), ("extra", 1e-3), ("posterior", 1e-3),
                                         ("ac_cost", 1e-3)])
def test_props_catch_a_planted_fault(oracle_mod, field, delta):
    cfg = synth.workload("tiny_10k")
    g = synth.make_graph(cfg)
    L = synth.make_loglikes(cfg)
    o = oracle_mod.decode(g, L, 10.0, 2000, 6.0)
    links = o.links.copy()
    k = len(links) // 2
    links[field][k] += delta
    o.links = links
    with pytest.raises(AssertionError):
        lattice_props.check(g, L, 6.0, o)


def test_props_catch_a_missing_node(oracle_mod):
    cfg = synth.workload("tiny_10k")
    g = synth.make_graph(cfg)
    L = synth.make_loglikes(cfg)
    o = oracle_mod.decode(g, L, 10.0, 2000, 6.0)
    o.nodes = np.delete(o.nodes, len(o.nodes) // 2)
    o.stats = dict(o.stats, nodes=len(o.nodes))
    with pytest.raises(AssertionError):
        lattice_props.check(g, L, 6.0, o)
