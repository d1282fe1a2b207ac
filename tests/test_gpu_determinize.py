"""Determinisation of lattices the GPU decoder produced: identical to the
determinisation of the oracle's lattice (the lattices are bit-identical),
and checked against the oracle's definition (every word sequence once, with
its best path) by enumeration where feasible, else on sampled paths."""
import numpy as np
import pytest

import oracle
import synth
from lattice_det import assert_matches, check_structure, paths
from oracle import lattice_paths as lp
from test_determinize import check_large

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def wf():
    import torch
    from paper_1804_03243_amd import wfstdec
    assert torch.cuda.is_available()
    wfstdec.lib()
    return wfstdec


def same_clat(a, b):
    assert a.states == b.states
    for f in ("arcs", "finals", "align"):
        assert np.array_equal(getattr(a, f), getattr(b, f)), f


@pytest.mark.parametrize("mode", ["workgroup", "chip"])
@pytest.mark.parametrize("T,lb", [(15, 3.0), (40, 3.0), (300, 6.0)])
def test_tiny_10k(wf, mode, T, lb):
    import torch
    cfg = synth.workload("tiny_10k")
    g = synth.make_graph(cfg)
    L = synth.make_loglikes(cfg)[:T]
    graph = wf.Graph(g, cfg["P"])
    s0, fw = g.get("start_state", 0), g.get("final_weight")
    print(f"\n[gpu case] determinise tiny_10k T={T} lattice_beam={lb} mode={mode}", flush=True)
    r = wf.decode(graph, torch.from_numpy(np.ascontiguousarray(L)).to(graph.device), cfg["beam"],
                  cfg["max_active"], lb, mode=mode)
    o = oracle.decode(g, L, cfg["beam"], cfg["max_active"], lb)
    c = wf.determinize(r, s0, fw)
    same_clat(c, wf.determinize(o, s0, fw))
    if T <= 40:
        best, _ = lp.best_by_words(r.links, r.nodes, s0, lp.node_final_costs(r, fw))
        check_structure(c)
        assert_matches(paths(c), best, exact=False)
    else:
        check_large(c, r, s0, fw)


def test_hclg_5m(wf):
    import torch
    cfg = synth.workload("hclg_5m")
    g = synth.make_graph(cfg)
    L = synth.make_loglikes(cfg)
    graph = wf.Graph(g, cfg["P"])
    s0, fw = g.get("start_state", 0), g.get("final_weight")
    print("\n[gpu case] determinise hclg_5m", flush=True)
    r = wf.decode(graph, torch.from_numpy(L).to(graph.device), cfg["beam"], cfg["max_active"],
                  cfg["lattice_beam"])
    c = wf.determinize(r, s0, fw)
    check_large(c, r, s0, fw, k=20)
