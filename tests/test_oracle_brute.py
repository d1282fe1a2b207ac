"""The oracle against exhaustive path enumeration on tiny random graphs,
with infinite beams (the decode is then exact Viterbi plus the full lattice).

With generic real inputs the best cost must match bit for bit: min commutes
with monotone fp32 addition, so the frame recursion equals the minimum over
all paths costed in the same order.  With dyadic inputs (multiples of 2^-4)
every sum is exact, so ties are real and the tie-break (lowest arc id, then
lowest final state), the link extras and the kept set match exactly.
"""
import math

import numpy as np
import pytest

import synth
from brute import brute_decode

INF = math.inf


def _decode(oracle_mod, g, L, lattice_beam=INF):
    return oracle_mod.decode(g, L, INF, 0, lattice_beam, debug=True)


def _cases(n, dyadic, finals):
    out = []
    for seed in range(n):
        S = 3 + seed % 5
        A = S + 2 + seed % 9
        T = 1 + seed % 5
        out.append((seed, S, A, T, dyadic, finals))
    return out


def _check_against_brute(oracle_mod, seed, S, A, T, dyadic, finals, lattice_beam, exact_extra):
    g = synth.tiny_graph(seed, S=S, A=A, eps_frac=0.3, P=3, V=4, finals=finals, dyadic=dyadic)
    L = synth.tiny_loglikes(seed + 7, T, 3, dyadic=dyadic)
    try:
        b = brute_decode(g, L, lattice_beam)
    except RuntimeError:
        pytest.skip("no complete path / too many paths")
    r = _decode(oracle_mod, g, L, lattice_beam)
    assert r.cost.view(np.uint32) == np.float32(b["cost"]).view(np.uint32), (r.cost, b["cost"])
    assert bool(r.stats["final_reached"]) == b["final_used"]
    # token costs of every token on a complete path
    toks = {(int(t), int(s)): (c, p) for t, s, c, p in zip(r.tokens["t"], r.tokens["state"],
                                                           r.tokens["cost"], r.tokens["pred_arc"])}
    for key, c in b["node_cost"].items():
        assert key in toks, key
        assert toks[key][0].view(np.uint32) == np.float32(c).view(np.uint32), key
        if key in b["pred"]:
            assert int(toks[key][1]) == b["pred"][key][1], ("pred", key)
    # kept lattice links and their extra costs
    kept = {(int(t), int(a)) for t, a in zip(r.links["t"], r.links["arc_id"])}
    if exact_extra:
        assert kept == b["kept"]
        for l in r.links:
            assert float(l["extra"]) == b["extra"][(int(l["t"]), int(l["arc_id"]))]
    else:
        for k in kept ^ b["kept"]:   # only links on the lattice-beam boundary may differ
            assert abs(b["extra"][k] - lattice_beam) < 1e-3, k
        for l in r.links:
            assert abs(float(l["extra"]) - b["extra"][(int(l["t"]), int(l["arc_id"]))]) < 1e-3
    if kept == b["kept"]:
        for l in r.links:
            k = (int(l["t"]), int(l["arc_id"]))
            assert abs(l["posterior"] - b["post"][k]) < 1e-9, (k, l["posterior"], b["post"][k])
    return r, b


@pytest.mark.parametrize("seed,S,A,T,dyadic,finals", _cases(40, False, False) + _cases(40, False, True))
def test_generic_inputs(oracle_mod, seed, S, A, T, dyadic, finals):
    r, b = _check_against_brute(oracle_mod, seed, S, A, T, dyadic, finals, INF, exact_extra=False)
    assert list(r.words) == b["words"]


@pytest.mark.parametrize("seed,S,A,T,dyadic,finals", _cases(60, True, False) + _cases(60, True, True))
def test_dyadic_ties(oracle_mod, seed, S, A, T, dyadic, finals):
    r, b = _check_against_brute(oracle_mod, 1000 + seed, S, A, T, dyadic, finals, INF,
                                exact_extra=True)
    assert list(r.words) == b["words"]


@pytest.mark.parametrize("lb", [0.0, 0.5, 1.5, 3.0])
@pytest.mark.parametrize("seed", range(25))
def test_dyadic_lattice_beam(oracle_mod, seed, lb):
    _check_against_brute(oracle_mod, 2000 + seed, 5, 12, 4, True, seed % 2 == 1, lb,
                         exact_extra=True)


def test_ties_are_exercised():
    """The dyadic cases must contain tokens whose minimum cost is reached by
    several candidates, so that the lowest-arc-id rule is what decides."""
    ties = 0
    for seed in range(60):
        g = synth.tiny_graph(1000 + seed, S=3 + seed % 5, A=3 + seed % 5 + 2 + seed % 9,
                             eps_frac=0.3, P=3, V=4, dyadic=True)
        L = synth.tiny_loglikes(1000 + seed + 7, 1 + seed % 5, 3, dyadic=True)
        try:
            b = brute_decode(g, L)
        except RuntimeError:
            continue
        for key, c in b["node_cost"].items():
            n = sum(1 for (t, a), v in b["links"].items()
                    if t == key[0] and v[1] == key[1] and v[2] == c)
            ties += n > 1
    assert ties >= 10
