"""The pins catch plausible mistakes: each mutant is the oracle's C source
with one mistake planted (on the CPU, in a temporary copy), and at least one
pin (brute force, closed forms, frame invariants) must reject it."""
import math
import os
import subprocess

import numpy as np
import pytest

import golden_cases
import invariants
import oracle as oracle_pkg
import synth
from brute import brute_decode

INF = math.inf

MUTANTS = {
    "dropped_acoustic_term": ("        float x = c + ac;\n        x = canon(x + g->weight[a]);\n        if (isinf(x)) continue;\n        recombine(",
                              "        float x = c;\n        x = canon(x + g->weight[a]);\n        if (isinf(x)) continue;\n        recombine("),
    "acoustic_sign": ("        float ac = -row[g->ilabel[a] - 1];\n        float x = c + ac;\n        x = canon(x + g->weight[a]);\n        if (isinf(x)) continue;\n        recombine(",
                      "        float ac = row[g->ilabel[a] - 1];\n        float x = c + ac;\n        x = canon(x + g->weight[a]);\n        if (isinf(x)) continue;\n        recombine("),
    "summation_order": ("        float x = c + ac;\n        x = canon(x + g->weight[a]);\n        if (isinf(x)) continue;\n        recombine(",
                        "        float x = c + (ac + g->weight[a]);\n        x = canon(x);\n        if (isinf(x)) continue;\n        recombine("),
    "tie_break_reversed": ("return x < y || (x == y && a < b);", "return x < y || (x == y && a > b);"),
    "eps_cutoff_exclusive": ("if (isinf(x) || !(x <= cutb)) continue;\n        if (recombine", "if (isinf(x) || !(x < cutb)) continue;\n        if (recombine"),
    "max_active_off_by_one": ("float v = d->sortbuf[d->p.max_active - 1];", "float v = d->sortbuf[d->p.max_active];"),
    "eps_single_sweep": ("        if (recombine(d, g->dst[a], x, a)) changed = 1;", "        recombine(d, g->dst[a], x, a);"),
    "link_cutoff_is_beam": ("const float cut = d->cut[t];", "const float cut = d->cutb[t];"),
    "prune_wrong_node": ("float le = ex[l->dst] + (l->x - d->toks[l->dst].cost);\n        if (le < ex[l->src]) ex[l->src] = le;",
                         "float le = ex[l->dst] + (l->x - d->toks[l->src].cost);\n        if (le < ex[l->src]) ex[l->src] = le;"),
    "final_weight_dropped": ("F[i] = final_used ? canon(tk->cost + g->final_weight[tk->state]) : tk->cost;",
                             "F[i] = tk->cost;"),
    "posterior_sign": ("post[k] = exp(Z - lse_val(&al[l->src]) - (double)g->weight[l->arc] - ac - lse_val(&be[l->dst]));",
                       "post[k] = exp(Z - lse_val(&al[l->src]) - (double)g->weight[l->arc] + ac - lse_val(&be[l->dst]));"),
    "beam_cutoff_from_zero": ("float cutb = best + d->p.beam;", "float cutb = d->p.beam + 0.0f * best;"),
    "eps_arcs_not_counted": ("    d->st.arcs_expanded += eps_deg(g, d->list[i]);\n", "\n"),
}


def _pins(oracle_mod):
    """Run a small battery of pins; raise on the first failure."""
    for name in ("hand_worked_1.json", "hand_worked_2.json"):
        d, g, L = golden_cases.load(name)
        r = oracle_mod.decode(g, L, d["beam"], d["max_active"], d["lattice_beam"])
        e = d["expect"]
        assert float(r.cost) == e["cost"] and list(r.words) == e["words"]
        assert r.stats["arcs_expanded"] == e["arcs_expanded"]
        assert len(r.links) == len(e["links"])
        for got, exp in zip(r.links, e["links"]):
            assert abs(got["posterior"] - exp["posterior"]) < 1e-12
            assert float(got["extra"]) == exp["extra"]
    for seed in range(30):
        dy = seed % 2 == 0
        g = synth.tiny_graph(3000 + seed, S=4 + seed % 4, A=10 + seed % 7, eps_frac=0.35, P=3,
                             finals=seed % 3 == 0, dyadic=dy)
        L = synth.tiny_loglikes(3100 + seed, 1 + seed % 4, 3, dyadic=dy)
        try:
            b = brute_decode(g, L)
        except RuntimeError:
            continue
        r = oracle_mod.decode(g, L, INF, 0, INF)
        assert r.cost == np.float32(b["cost"]) and list(r.words) == b["words"]
    cfg = synth.workload("tiny_10k")
    g = synth.make_graph(cfg)
    L = synth.make_loglikes(cfg)[:60]
    for beam, ma, lb in [(10.0, 40, 6.0), (6.0, 0, 3.0)]:
        r = oracle_mod.decode(g, L, beam, ma, lb, debug=True)
        invariants.check_all(g, L, beam, ma, lb, r)
    for seed in range(4):
        g = synth.tiny_graph(700 + seed, S=100, A=330, eps_frac=0.3, P=8, finals=True,
                             dyadic=seed % 2 == 0)
        L = synth.tiny_loglikes(710 + seed, 20, 8, dyadic=seed % 2 == 0)
        r = oracle_mod.decode(g, L, 6.0, 10, 3.0, debug=True)
        invariants.check_all(g, L, 6.0, 10, 3.0, r)


def test_unmutated_passes(oracle_mod):
    _pins(oracle_mod)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(oracle_mod, tmp_path, name):
    src = open(oracle_pkg.SRC_PATH).read()
    old, new = MUTANTS[name]
    assert src.count(old) == 1, f"mutation site for {name} not unique / not found"
    msrc = tmp_path / "wfst_oracle.c"
    msrc.write_text(src.replace(old, new))
    hdr = os.path.join(os.path.dirname(oracle_pkg.SRC_PATH), "wfst_oracle.h")
    (tmp_path / "wfst_oracle.h").write_text(open(hdr).read())
    so = tmp_path / "libmut.so"
    subprocess.check_call(["gcc", *oracle_pkg.CFLAGS, "-o", str(so), str(msrc), "-lm"])
    saved_lib, saved_path = oracle_pkg._LIB, oracle_pkg.LIB_PATH
    oracle_pkg._LIB, oracle_pkg.LIB_PATH = None, str(so)
    try:
        with pytest.raises((AssertionError, oracle_pkg.OracleError, KeyError, IndexError)):
            _pins(oracle_pkg)
    finally:
        oracle_pkg._LIB, oracle_pkg.LIB_PATH = saved_lib, saved_path
