"""Input validation and failure statuses of the oracle."""
import math

import numpy as np
import pytest

import synth

INF = math.inf


def _base():
    g = synth.tiny_graph(5, S=6, A=14, eps_frac=0.3, P=3)
    L = synth.tiny_loglikes(6, 4, 3)
    return g, L


def _err(oracle_mod, g, L, beam=10.0, ma=0, lb=5.0):
    with pytest.raises(oracle_mod.OracleError) as e:
        oracle_mod.decode(g, L, beam, ma, lb)
    return e.value.code


@pytest.mark.parametrize("mutate", [
    lambda g, L: g["row_ptr"].__setitem__(2, g["row_ptr"][3] + 1),
    lambda g, L: g["dst"].__setitem__(0, 6),
    lambda g, L: g["ilabel"].__setitem__(0, 4),
    lambda g, L: g["ilabel"].__setitem__(0, -1),
    lambda g, L: g["olabel"].__setitem__(0, -1),
    lambda g, L: g["weight"].__setitem__(0, -1.0),
    lambda g, L: g["weight"].__setitem__(0, np.nan),
    lambda g, L: g["weight"].__setitem__(0, np.inf),
    lambda g, L: L.__setitem__((1, 1), np.nan),
    lambda g, L: L.__setitem__((1, 1), np.inf),
    lambda g, L: L.__setitem__((1, 1), 2e30),
    lambda g, L: g.__setitem__("final_weight", np.full(6, np.nan, np.float32)),
    lambda g, L: g.__setitem__("final_weight", np.full(6, -1.0, np.float32)),
    lambda g, L: g.__setitem__("start_state", 6),
])
def test_einval(oracle_mod, mutate):
    g, L = _base()
    mutate(g, L)
    assert _err(oracle_mod, g, L) == oracle_mod.EINVAL


@pytest.mark.parametrize("beam,ma,lb", [(0.0, 0, 1.0), (-1.0, 0, 1.0), (np.nan, 0, 1.0),
                                        (1.0, -1, 1.0), (1.0, 0, -1.0), (1.0, 0, np.nan)])
def test_bad_params(oracle_mod, beam, ma, lb):
    g, L = _base()
    assert _err(oracle_mod, g, L, beam, ma, lb) == oracle_mod.EINVAL


def test_epsilon_cycle(oracle_mod):
    g = dict(num_states=3, start_state=0, row_ptr=np.array([0, 2, 3, 4], np.uint32),
             dst=np.array([1, 0, 2, 1], np.uint32), ilabel=np.array([0, 1, 0, 0], np.int32),
             olabel=np.zeros(4, np.int32), weight=np.ones(4, np.float32), final_weight=None)
    L = np.zeros((2, 1), np.float32)
    assert _err(oracle_mod, g, L) == oracle_mod.ECYCLE


def test_no_path(oracle_mod):
    """Every pdf impossible (-inf) at one frame: no token survives it."""
    g, L = _base()
    L[2, :] = -np.inf
    assert _err(oracle_mod, g, L, beam=INF) == oracle_mod.ENOPATH


def test_impossible_pdf_is_skipped(oracle_mod):
    """-inf log-likelihood makes those arcs unusable but the decode proceeds."""
    g, L = _base()
    L[1, 0] = -np.inf
    r = oracle_mod.decode(g, L, INF, 0, INF)
    assert np.isfinite(r.cost)
    assert not np.any((r.links["t"] == 2) & (r.links["ilabel"] == 1))
