"""The oracle on cases whose answer has a closed form or a library routine:
a hand-worked example, a single-state graph (per-frame argmax and softmax),
a linear chain, and the shortest path through graph x trellis (scipy)."""
import math

import numpy as np
import pytest
import scipy.sparse as sp
from scipy.sparse.csgraph import shortest_path
from scipy.special import softmax

import golden_cases
import synth

INF = math.inf
f32 = np.float32


@pytest.mark.parametrize("name", ["hand_worked_1.json", "hand_worked_2.json"])
def test_hand_worked_example(oracle_mod, name):
    d, g, L = golden_cases.load(name)
    r = oracle_mod.decode(g, L, d["beam"], d["max_active"], d["lattice_beam"])
    e = d["expect"]
    assert float(r.cost) == e["cost"]
    assert list(r.words) == e["words"]
    assert r.stats["arcs_expanded"] == e["arcs_expanded"]
    assert len(r.links) == len(e["links"])
    for got, exp in zip(r.links, e["links"]):
        for k in ("t", "arc_id", "src_state", "dst_state"):
            assert int(got[k]) == exp[k], k
        assert float(got["fwd_cost"]) == exp["fwd_cost"]
        assert float(got["extra"]) == exp["extra"]
        assert abs(got["posterior"] - exp["posterior"]) < 1e-12
    assert len(r.nodes) == len(e["nodes"])
    for got, exp in zip(r.nodes, e["nodes"]):
        assert (int(got["t"]), int(got["state"])) == (exp["t"], exp["state"])
        assert float(got["cost"]) == exp["cost"] and float(got["extra"]) == exp["extra"]


def _single_state(P):
    return dict(num_states=1, start_state=0, row_ptr=np.array([0, P], np.uint32),
                dst=np.zeros(P, np.uint32), ilabel=np.arange(1, P + 1, dtype=np.int32),
                olabel=np.arange(1, P + 1, dtype=np.int32), weight=np.zeros(P, np.float32),
                final_weight=None)


@pytest.mark.parametrize("seed", range(4))
def test_single_state_argmax_and_softmax(oracle_mod, seed):
    """One state with a zero-weight self-loop per pdf: the best path takes the
    per-frame argmax pdf (lowest pdf on ties), its cost is the sequential fp32
    sum of the per-frame minima of -loglike, and every link's posterior is the
    per-frame softmax of the log-likelihoods."""
    rng = np.random.default_rng(seed)
    T, P = 40, 17
    L = rng.normal(-3, 2, (T, P)).astype(f32)
    if seed == 3:  # exact ties between pdfs
        L = (np.round(L * 2) / 2).astype(f32)
    r = oracle_mod.decode(_single_state(P), L, INF, 0, INF)
    assert list(r.words) == list(np.argmax(L, axis=1) + 1)
    c = f32(0)
    for t in range(T):
        c = f32(f32(c + f32(-L[t].max())) + f32(0))
    assert r.cost.view(np.uint32) == c.view(np.uint32)
    sm = softmax(L.astype(np.float64), axis=1)
    assert len(r.links) == T * P
    for l in r.links:
        assert abs(l["posterior"] - sm[l["t"] - 1, l["arc_id"]]) < 1e-12


def test_single_state_max_active_one(oracle_mod):
    """max_active = 1 cannot change a single-state decode."""
    rng = np.random.default_rng(9)
    L = rng.normal(-3, 2, (30, 8)).astype(f32)
    a = oracle_mod.decode(_single_state(8), L, INF, 0, INF)
    b = oracle_mod.decode(_single_state(8), L, INF, 1, INF)
    assert list(a.words) == list(b.words) and a.cost == b.cost


def test_linear_chain(oracle_mod):
    """A chain 0 -> 1 -> ... -> T: the only path; its cost is the fixed
    sequential sum and every link has posterior 1 and extra 0."""
    T, P = 25, 6
    rng = np.random.default_rng(5)
    il = rng.integers(1, P + 1, T).astype(np.int32)
    w = rng.exponential(1.0, T).astype(f32)
    g = dict(num_states=T + 1, start_state=0, row_ptr=np.r_[np.arange(T + 1), T].astype(np.uint32),
             dst=np.arange(1, T + 1, dtype=np.uint32), ilabel=il,
             olabel=np.arange(1, T + 1, dtype=np.int32), weight=w, final_weight=None)
    L = rng.normal(-2, 1, (T, P)).astype(f32)
    r = oracle_mod.decode(g, L, INF, 0, 0.0)
    c = f32(0)
    for t in range(T):
        c = f32(f32(c + f32(-L[t, il[t] - 1])) + w[t])
    assert r.cost.view(np.uint32) == c.view(np.uint32)
    assert list(r.words) == list(range(1, T + 1))
    assert len(r.links) == T
    assert np.all(r.links["extra"] == 0) and np.allclose(r.links["posterior"], 1.0, atol=1e-12)


@pytest.mark.parametrize("seed", range(6))
def test_shortest_path_through_trellis(oracle_mod, seed):
    """With infinite beams the best cost equals the shortest path through the
    graph x trellis (fp64 library routine; fp32 rounding tolerance)."""
    g = synth.tiny_graph(300 + seed, S=25, A=70, eps_frac=0.2, P=5, V=6, finals=seed % 2 == 1)
    T = 10
    L = synth.tiny_loglikes(400 + seed, T, 5)
    r = oracle_mod.decode(g, L, INF, 0, INF)
    S = g["num_states"]
    N = S * (T + 1) + 1
    # shortest path without shifting: Bellman-Ford handles negative edges
    rp = g["row_ptr"].astype(np.int64)
    src = np.repeat(np.arange(S), np.diff(rp))
    il, dst, w = g["ilabel"], g["dst"].astype(np.int64), g["weight"].astype(np.float64)
    best = {}
    rows, cols, vals = [], [], []
    for t in range(T + 1):
        for a in range(dst.size):
            if il[a] == 0:
                u, v, c = t * S + src[a], t * S + dst[a], w[a]
            elif t < T:
                u, v, c = t * S + src[a], (t + 1) * S + dst[a], w[a] - float(L[t, il[a] - 1])
            else:
                continue
            if (u, v) not in best or c < best[(u, v)]:
                best[(u, v)] = c
    fw = g.get("final_weight")
    final_used = fw is not None and bool(np.isfinite(fw).any())
    for s in range(S):
        if fw is None or not final_used:
            best[(T * S + s, N - 1)] = 0.0
        elif np.isfinite(fw[s]):
            best[(T * S + s, N - 1)] = float(fw[s])
    keys = list(best)
    m = sp.csr_matrix(([best[k] for k in keys], ([k[0] for k in keys], [k[1] for k in keys])),
                      shape=(N, N))
    # a zero-weight edge must stay an edge: scipy keeps explicit entries
    d = shortest_path(m, method="BF", directed=True, indices=[0])[0, N - 1]
    if not np.isfinite(d):
        pytest.skip("no complete path")
    if r.stats["final_reached"] != int(final_used):
        pytest.skip("final states unreachable")
    assert abs(float(r.cost) - d) < 1e-3 * max(1.0, abs(d)), (r.cost, d)
