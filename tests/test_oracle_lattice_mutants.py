"""The pins of the determinisation oracle catch plausible mistakes: each
mutant is oracle/lattice_paths.py with one mistake planted (a text edit of a
temporary copy, loaded as its own module), and the pins of
test_oracle_lattice_paths must reject it."""
import importlib.util
import os
import sys

import pytest

import test_oracle_lattice_paths as pins

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle", "lattice_paths.py")

MUTANTS = {
    "final_cost_dropped": ("cand = (g + float(node_final[u]), a, s)\n            if w not in best",
                           "cand = (g, a, s)\n            if w not in best"),
    "graph_cost_before_string": ("    if x[2] != y[2]:\n        return x[2] < y[2]\n    return x[0] < y[0]",
                                 "    if x[0] != y[0]:\n        return x[0] < y[0]\n    return x[2] < y[2]"),
    "emitting_source_same_frame": ("u = index[(t - 1 if il != 0 else t, int(l[\"src_state\"]))]",
                                   "u = index[(t, int(l[\"src_state\"]))]"),
    "epsilon_ilabel_in_string": ("s + ((il,) if il else ()), w + ((word,) if word else ()), 0))",
                                 "s + (il,), w + ((word,) if word else ()), 0))"),
    "zero_olabel_is_a_word": ("s + ((il,) if il else ()), w + ((word,) if word else ()), 0))",
                              "s + ((il,) if il else ()), w + (word,), 0))"),
    "dp_accepts_prefix": ("            if k == K and math.isfinite(float(node_final[u])):",
                          "            if math.isfinite(float(node_final[u])):"),
    "acoustic_cost_dropped": ("stack.append((v, g + ag, a + aa, s +", "stack.append((v, g + ag, a, s +"),
}


def _load(text, name):
    spec = importlib.util.spec_from_loader(name, loader=None)
    mod = importlib.util.module_from_spec(spec)
    exec(compile(text, name, "exec"), mod.__dict__)
    return mod


def _run_pins(lp):
    old = pins.lp
    pins.lp = lp
    try:
        pins.test_hand_worked()
        for dy in (True, False):
            for seed in range(16):
                try:
                    pins.test_enumeration_equals_dynamic_programme(seed, dy)
                except pytest.skip.Exception:
                    pass
        for seed in range(16):
            try:
                pins.test_best_sequence_is_the_one_best(seed)
            except pytest.skip.Exception:
                pass
    finally:
        pins.lp = old


def test_unmutated_passes():
    _run_pins(_load(open(SRC).read(), "lattice_paths_copy"))


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name):
    old, new = MUTANTS[name]
    text = open(SRC).read()
    assert text.count(old) == 1, f"mutation anchor for {name} not found once"
    mod = _load(text.replace(old, new), f"lattice_paths_{name}")
    with pytest.raises(Exception):
        _run_pins(mod)
