"""GPU library (through its C ABI) against the CPU oracle on the same seeded
inputs: 1-best words, cost, every lattice link and node bit for bit,
posteriors within 1e-4; with the debug flag also every frame's surviving
tokens, cutoffs and the raw lattice.  Sizes span several tiles of the
1024-thread workgroup, both compaction paths (LDS rank sort, state bitmap)
and ragged frames.  Every case runs in every execution mode: one workgroup
per utterance, chip-wide kernels per frame, and chip-wide with dynamic load
balancing of the emitting arcs; the one-workgroup mode both with the
epsilon closure over the graph's enumerated epsilon paths (its default) and
level by level."""
import math

import numpy as np
import pytest

import golden_cases
import invariants
import synth
from gpu_compare import assert_same

pytestmark = pytest.mark.gpu
INF = math.inf
MODES = ["workgroup", "workgroup_levels", "chip", "chip_dyn"]


@pytest.fixture(scope="module")
def wf():
    import torch
    from paper_1804_03243_amd import wfstdec
    assert torch.cuda.is_available()
    wfstdec.lib()
    return wfstdec


def _run(wf, oracle_mod, g, L, P, beam, ma, lb, debug=True, graph=None, case="", mode="auto"):
    import torch
    print(f"\n[gpu case] {case} S={g['num_states']} A={g['dst'].size} T={L.shape[0]} "
          f"beam={beam} max_active={ma} lattice_beam={lb} debug={debug} mode={mode}", flush=True)
    graph = graph or wf.Graph(g, P)
    x = torch.from_numpy(np.ascontiguousarray(L)).to(graph.device)
    r = wf.decode(graph, x, beam, ma, lb, debug=debug, mode=mode)
    o = oracle_mod.decode(g, L, beam, ma, lb, debug=debug)
    assert_same(r, o, debug=debug)
    return r, o, graph


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("name", ["hand_worked_1.json", "hand_worked_2.json"])
def test_golden(wf, oracle_mod, name, mode):
    d, g, L = golden_cases.load(name)
    r, o, _ = _run(wf, oracle_mod, g, L, L.shape[1], d["beam"], d["max_active"], d["lattice_beam"],
                   case=name, mode=mode)
    e = d["expect"]
    assert float(r.cost) == e["cost"] and list(r.words) == e["words"]
    assert r.stats["arcs_expanded"] == e["arcs_expanded"]


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("seed", range(24))
def test_tiny_random(wf, oracle_mod, seed, mode):
    dy = seed % 2 == 0
    g = synth.tiny_graph(4000 + seed, S=4 + seed % 6, A=12 + seed % 11, eps_frac=0.35, P=3,
                         finals=seed % 3 == 0, dyadic=dy)
    L = synth.tiny_loglikes(4100 + seed, 1 + seed % 6, 3, dyadic=dy)
    beam = [INF, 3.0, 1.5][seed % 3]
    ma = [0, 2, 0, 1][seed % 4]
    lb = [INF, 1.0, 0.0][seed % 3]
    try:
        oracle_mod.decode(g, L, beam, ma, lb)
    except oracle_mod.OracleError as e:
        # no token survives some frame: the GPU must report the same status
        assert e.code == oracle_mod.ENOPATH, e
        import torch
        print(f"\n[gpu case] tiny seed {seed} (no path) mode={mode}", flush=True)
        graph = wf.Graph(g, 3)
        x = torch.from_numpy(np.ascontiguousarray(L)).to(graph.device)
        with pytest.raises(wf.WdError) as err:
            wf.decode(graph, x, beam, ma, lb, mode=mode)
        assert err.value.status == wf.WD_ENOPATH
        return
    _run(wf, oracle_mod, g, L, 3, beam, ma, lb, case=f"tiny seed {seed}", mode=mode)


@pytest.mark.parametrize("mode", MODES)
def test_zero_frames(wf, oracle_mod, mode):
    g = synth.tiny_graph(77, S=6, A=14, eps_frac=0.6, P=3, finals=True)
    L = np.zeros((0, 3), np.float32)
    _run(wf, oracle_mod, g, L, 3, INF, 0, INF, case="T=0", mode=mode)


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("seed", range(8))
def test_medium_random(wf, oracle_mod, seed, mode):
    rng = np.random.default_rng(seed)
    dy = seed % 3 == 0
    g = synth.tiny_graph(500 + seed, S=150, A=520, eps_frac=0.25, P=12, V=20,
                         finals=seed % 2 == 1, dyadic=dy)
    L = synth.tiny_loglikes(600 + seed, 40, 12, dyadic=dy)
    beam = float(rng.choice([2.0, 5.0, 9.0, INF]))
    ma = int(rng.choice([0, 5, 30]))
    lb = float(rng.choice([0.0, 1.0, 4.0, INF]))
    r, _, _ = _run(wf, oracle_mod, g, L, 12, beam, ma, lb, case=f"medium seed {seed}", mode=mode)
    invariants.check_all(g, L, beam, ma, lb, r)


TINY_PARAMS = [(10.0, 2000, 6.0), (10.0, 40, 6.0), (4.0, 0, 2.0), (25.0, 150, INF), (2.0, 5, 0.0),
               (INF, 0, 3.0)]


@pytest.fixture(scope="module")
def tiny10k(wf):
    cfg = synth.workload("tiny_10k")
    g = synth.make_graph(cfg)
    return cfg, g, synth.make_loglikes(cfg), wf.Graph(g, cfg["P"])


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("beam,ma,lb", TINY_PARAMS)
def test_tiny_10k(wf, oracle_mod, tiny10k, beam, ma, lb, mode):
    cfg, g, L, graph = tiny10k
    r, _, _ = _run(wf, oracle_mod, g, L, cfg["P"], beam, ma, lb, graph=graph,
                   case=f"tiny_10k {beam}/{ma}/{lb}", mode=mode)
    invariants.check_all(g, L, beam, ma, lb, r)


@pytest.mark.parametrize("mode", ["workgroup", "workgroup_levels", "chip"])
@pytest.mark.parametrize("T", [1800, 2100])
def test_long_utterance(wf, oracle_mod, tiny10k, T, mode):
    """Utterances past the lattice pass's LDS limits: 1800 frames keep ~2.9k
    lattice links (more than the LDS posteriors hold: their per-frame
    windowed form runs, the staged sweep still fits), 2100 frames are longer
    than its frame tables (the frame-by-frame sweep and the windowed
    posteriors)."""
    cfg, g, _, graph = tiny10k
    L = synth.make_loglikes(dict(cfg, T=T))
    r, o, _ = _run(wf, oracle_mod, g, L, cfg["P"], cfg["beam"], cfg["max_active"], cfg["lattice_beam"],
                   graph=graph, case=f"tiny_10k T={T}", mode=mode)
    assert o.stats["kept_links"] > 2560


@pytest.mark.parametrize("mode", ["chip", "chip_noprune", "chip_dyn"])
@pytest.mark.parametrize("beam,ma,lb", TINY_PARAMS)
def test_incremental_prune(wf, oracle_mod, tiny10k, beam, ma, lb, mode):
    """Chip-wide decodes without the debug flag prune the lattice every 32
    frames while decoding (conservatively); the result still equals the
    oracle's, and with a finite lattice beam the link store peaks below the
    raw lattice."""
    cfg, g, L, graph = tiny10k
    r, o, _ = _run(wf, oracle_mod, g, L, cfg["P"], beam, ma, lb, debug=False, graph=graph,
                   case=f"tiny_10k incremental prune {beam}/{ma}/{lb}", mode=mode)
    assert r.stats["raw_links"] == o.stats["raw_links"]
    if mode == "chip_noprune" or math.isinf(lb):
        assert r.needed["links"] <= r.stats["raw_links"]
    else:
        assert r.needed["links"] < r.stats["raw_links"]


@pytest.mark.parametrize("mode", ["chip", "chip_dyn"])
def test_incremental_prune_batch(wf, oracle_mod, tiny10k, mode):
    """Pruning windows of 32 frames with utterances of different lengths in
    one batch: shorter than a window, ending on a window's last frame (that
    window is never pruned), one frame into the next window, several windows.
    Every lane equals the oracle and its own single decode."""
    import torch
    cfg, g, L, graph = tiny10k
    lens = [0, 1, 31, 32, 33, 63, 64, 95, 120]
    Ls = [np.ascontiguousarray(synth.tiny_loglikes(700 + i, n, cfg["P"]) * 3 - 10, dtype=np.float32)
          for i, n in enumerate(lens)]
    xs = [torch.from_numpy(x).to(graph.device) for x in Ls]
    print(f"\n[gpu case] incremental prune batch lens={lens} mode={mode}", flush=True)
    rb = wf.decode_batch(graph, xs, 10.0, 40, 6.0, mode=mode)
    for i, x in enumerate(xs):
        rs = wf.decode(graph, x, 10.0, 40, 6.0, mode=mode)
        o = oracle_mod.decode(g, Ls[i], 10.0, 40, 6.0)
        assert_same(rb[i], o)
        assert_same(rs, o)
        assert rb[i].stats["raw_links"] == o.stats["raw_links"]


@pytest.mark.parametrize("mode", MODES)
def test_determinism(wf, oracle_mod, tiny10k, mode):
    import torch
    cfg, g, L, graph = tiny10k
    x = torch.from_numpy(L).to(graph.device)
    print(f"\n[gpu case] determinism tiny_10k x3 mode={mode}", flush=True)
    rs = [wf.decode(graph, x, 10.0, 40, 6.0, debug=True, mode=mode) for _ in range(3)]
    for r in rs[1:]:
        assert r.cost == rs[0].cost and list(r.words) == list(rs[0].words)
        assert np.array_equal(r.links[["t", "arc_id", "fwd_cost", "extra"]],
                              rs[0].links[["t", "arc_id", "fwd_cost", "extra"]])
        assert np.array_equal(r.tokens, rs[0].tokens)
        assert np.abs(r.links["posterior"] - rs[0].links["posterior"]).max(initial=0) < 1e-12


@pytest.mark.parametrize("mode", MODES)
def test_batch_lanes_equal_single(wf, oracle_mod, tiny10k, mode):
    """Lane i of a batch equals a single decode of utterance i, bit for bit,
    for utterances of different lengths."""
    import torch
    cfg, g, L, graph = tiny10k
    rng = np.random.default_rng(3)
    Ls = [synth.tiny_loglikes(900 + i, int(n), cfg["P"]) * 3 - 10 for i, n in
          enumerate([50, 1, 120, 0, 77])]
    Ls = [np.ascontiguousarray(x, dtype=np.float32) for x in Ls]
    xs = [torch.from_numpy(x).to(graph.device) for x in Ls]
    print(f"\n[gpu case] batch of 5 tiny_10k utterances mode={mode}", flush=True)
    rb = wf.decode_batch(graph, xs, 10.0, 40, 6.0, debug=True, mode=mode)
    for i, x in enumerate(xs):
        rs = wf.decode(graph, x, 10.0, 40, 6.0, debug=True, mode=mode)
        o = oracle_mod.decode(g, Ls[i], 10.0, 40, 6.0, debug=True)
        assert_same(rb[i], o, debug=True)
        assert_same(rs, o, debug=True)
    del rng


def test_batch_more_lanes_than_cus(wf, oracle_mod, tiny10k):
    """300 utterances in one call (more workgroups than the chip's 256 CUs),
    lengths 0..80 frames, results through the packed single transfer: every
    lane equals the oracle's decode of its utterance."""
    import torch
    cfg, g, L, graph = tiny10k
    rng = np.random.default_rng(17)
    lens = [0, 1] + [int(n) for n in rng.integers(2, 81, 298)]
    Ls = [np.ascontiguousarray(synth.tiny_loglikes(5000 + i, n, cfg["P"]) * 3 - 10, dtype=np.float32)
          for i, n in enumerate(lens)]
    xs = [torch.from_numpy(x).to(graph.device) for x in Ls]
    args = (10.0, 200, 6.0)
    print(f"\n[gpu case] batch of {len(lens)} tiny_10k utterances, {sum(lens)} frames, mode=workgroup",
          flush=True)
    rb = wf.decode_batch(graph, xs, *args, mode="workgroup")
    assert len(rb) == len(lens)
    for i, x in enumerate(Ls):
        assert_same(rb[i], oracle_mod.decode(g, x, *args))


@pytest.mark.parametrize("mode", MODES)
def test_wide_2m_dyadic_prefix(wf, oracle_mod, mode):
    """Tens of thousands of tokens per frame (state-bitmap compaction), exact
    ties, epsilon chains of depth 8."""
    cfg = synth.workload("wide_2m_dyadic")
    g = synth.make_graph(cfg)
    L = synth.make_loglikes(cfg)[:3]
    r, _, _ = _run(wf, oracle_mod, g, L, cfg["P"], cfg["beam"], cfg["max_active"], cfg["lattice_beam"],
                   case="wide_2m_dyadic T=3", mode=mode)
    assert r.stats["max_tokens"] > 2048


def test_lds_table_spill_and_reuse(wf, oracle_mod, hclg5m):
    """Frames whose expansion touches more states than the LDS token table
    records (2048): each is redone on the global slot array, and the next
    one, small again after the max-active cut, starts in the table, which
    must have been emptied of every slot the spilled frame claimed."""
    cfg, g, L, graph, _ = hclg5m
    r, _, _ = _run(wf, oracle_mod, g, L[:30], cfg["P"], 40.0, 1500, 6.0, graph=graph,
                   case="hclg_5m T=30 beam=40 max_active=1500 (table spills)", mode="workgroup")
    assert r.needed["frame_tokens"] > 2048
    assert r.stats["max_tokens"] == 1500


@pytest.fixture(scope="module")
def hclg5m(wf, oracle_mod):
    cfg = synth.workload("hclg_5m")
    g = synth.make_graph(cfg)
    L = synth.make_loglikes(cfg)
    o = oracle_mod.decode(g, L, cfg["beam"], cfg["max_active"], cfg["lattice_beam"])
    return cfg, g, L, wf.Graph(g, cfg["P"]), o


@pytest.mark.parametrize("mode", MODES)
def test_hclg_5m(wf, hclg5m, mode):
    import torch
    cfg, g, L, graph, o = hclg5m
    print(f"\n[gpu case] hclg_5m full mode={mode}", flush=True)
    x = torch.from_numpy(L).to(graph.device)
    r = wf.decode(graph, x, cfg["beam"], cfg["max_active"], cfg["lattice_beam"], mode=mode)
    assert_same(r, o)


@pytest.mark.parametrize("mode", MODES)
def test_invalid_loglikes(wf, tiny10k, mode):
    import torch
    cfg, g, L, graph = tiny10k
    bad = L[:20].copy()
    bad[7, 3] = np.nan
    print(f"\n[gpu case] NaN log-likelihood mode={mode}", flush=True)
    with pytest.raises(wf.WdError) as e:
        wf.decode(graph, torch.from_numpy(bad).to(graph.device), 10.0, 0, 5.0, mode=mode)
    assert e.value.status == wf.WD_EINVAL


@pytest.mark.parametrize("mode", MODES)
def test_no_path(wf, tiny10k, mode):
    import torch
    cfg, g, L, graph = tiny10k
    bad = L[:20].copy()
    bad[5, :] = -np.inf
    print(f"\n[gpu case] all pdfs impossible at one frame mode={mode}", flush=True)
    with pytest.raises(wf.WdError) as e:
        wf.decode(graph, torch.from_numpy(bad).to(graph.device), INF, 0, 5.0, mode=mode)
    assert e.value.status == wf.WD_ENOPATH


@pytest.mark.parametrize("mode", MODES)
def test_capacity_retry(wf, oracle_mod, tiny10k, mode):
    """Deliberately small capacities: the decode reports WD_ECAPACITY with the
    sizes it needs, and the retries end with the oracle's result."""
    import torch
    cfg, g, L, graph = tiny10k
    x = torch.from_numpy(L[:80]).to(graph.device)
    small = wf.wd_caps(64, 64, 500, 500, 16, 40)
    print(f"\n[gpu case] capacity retry mode={mode}", flush=True)
    p = wf.wd_params(10.0, 2000, 6.0, wf._MODE_FLAGS[mode])
    ws, nbytes, used = graph.workspace(1, 80, p, small)
    st, res = wf.wd_decode(graph.handle, x.data_ptr(), 80, p, used, ws, nbytes,
                           torch.cuda.current_stream().cuda_stream)
    assert st == wf.WD_ECAPACITY and res
    r0 = wf.wd_result_read(res)
    wf.wd_result_free(res)
    assert any(r0.needed[f] > getattr(used, f) for f, _ in wf.wd_caps._fields_), r0.needed
    r = wf.decode(graph, x, 10.0, 2000, 6.0, caps=small, mode=mode)
    o = oracle_mod.decode(g, L[:80], 10.0, 2000, 6.0)
    assert_same(r, o)


def test_mode_flags_exclusive(wf, tiny10k):
    import torch
    cfg, g, L, graph = tiny10k
    x = torch.from_numpy(L[:10]).to(graph.device)
    p = wf.wd_params(10.0, 40, 6.0, wf.WD_FLAG_ONE_WORKGROUP | wf.WD_FLAG_CHIP_WIDE)
    ws, nbytes, used = graph.workspace(1, 10, wf.wd_params(10.0, 40, 6.0, 0), None)
    print("\n[gpu case] both mode flags", flush=True)
    st, res = wf.wd_decode(graph.handle, x.data_ptr(), 10, p, used, ws, nbytes,
                           torch.cuda.current_stream().cuda_stream)
    assert st == wf.WD_EINVAL and not res


def fanin_graph(n_spread: int, n_hub: int = 8, P: int = 16, seed: int = 0) -> dict:
    """Start state -> n_spread states by emitting arcs; each of those has an
    epsilon arc to every one of n_hub hub states; each hub goes back to the
    start by an emitting arc.  Every other frame, the epsilon closure has
    one level of n_spread * n_hub work items over only n_spread + n_hub
    table entries."""
    rng = np.random.default_rng(seed)
    S = 1 + n_spread + n_hub
    src, dst, il = [], [], []
    for i in range(n_spread):
        src.append(0), dst.append(1 + i), il.append(1 + i % P)
    for i in range(n_spread):
        for h in range(n_hub):
            src.append(1 + i), dst.append(1 + n_spread + h), il.append(0)
    for h in range(n_hub):
        src.append(1 + n_spread + h), dst.append(0), il.append(1 + h % P)
    src = np.asarray(src)
    A = src.size
    row_ptr = np.zeros(S + 1, np.int64)
    np.cumsum(np.bincount(src, minlength=S), out=row_ptr[1:])
    olabel = np.where(rng.random(A) < 0.3, rng.integers(1, 50, A), 0)
    return synth._pack(dict(row_ptr=row_ptr, dst=np.asarray(dst), ilabel=np.asarray(il), olabel=olabel,
                            weight=rng.exponential(1.0, A).astype(np.float32)), S)


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("n_spread", [500, 600])
def test_epsilon_fanin_level(wf, oracle_mod, n_spread, mode):
    """One epsilon level with 4000 (500 x 8) and 4800 (600 x 8) work items:
    in one-workgroup mode below and above the number whose owners fit the
    owner array (4096), so both the owner lookup and the search fallback run."""
    g = fanin_graph(n_spread)
    L = synth.tiny_loglikes(31 + n_spread, 7, 16) * 3 - 6
    _run(wf, oracle_mod, g, L, 16, INF, 2000, 4.0, case=f"epsilon fan-in {n_spread}", mode=mode)


def test_phase_profile(wf, oracle_mod, tiny10k):
    """WD_FLAG_PHASES runs the profiled copy of the forward kernel: the same
    result, and per frame non-decreasing wall-clock stamps at the step
    boundaries and the frame's token and link counts; chip-wide mode rejects
    the flag."""
    import torch
    cfg, g, L, graph = tiny10k
    args = (cfg["beam"], cfg["max_active"], cfg["lattice_beam"])
    x = torch.from_numpy(L[:120]).to(graph.device)
    print("\n[gpu case] step profile tiny_10k 120 frames", flush=True)
    r = wf.decode(graph, x, *args, debug=True, mode="workgroup", flags=wf.WD_FLAG_PHASES)
    o = oracle_mod.decode(g, L[:120], *args, debug=True)
    assert_same(r, o, debug=True)
    ph = r.phases
    assert ph.shape == (121, wf.WD_PHASE_SLOTS) and r.phase_tick_hz > 0
    st = ph[:, :wf.WD_PHASE_STAMPS].astype(np.int64)
    assert np.all(np.diff(st, axis=1) >= 0)
    assert np.all(st[1:, 0] >= st[:-1, wf.WD_PHASE_STAMPS - 1])
    ntok = (ph[:, wf.WD_PHASE_STAMPS] >> 8) & 0xffffff
    counts = np.bincount(o.tokens["t"], minlength=121)
    assert np.array_equal(ntok, counts)
    nlink = ph[:, wf.WD_PHASE_STAMPS] >> 32
    assert np.array_equal(nlink, np.bincount(o.raw_links["t"], minlength=121))
    lp = r.lattice_phases.astype(np.int64)
    assert lp.shape == (wf.WD_LATTICE_PHASE_STAMPS,) and np.all(np.diff(lp) >= 0)
    assert lp[0] >= st[-1, wf.WD_PHASE_STAMPS - 1]  # the lattice pass runs after the last frame
    plain = wf.decode(graph, x, *args, mode="workgroup")
    assert plain.phases.shape[0] == 0 and plain.lattice_phases.shape[0] == 0
    with pytest.raises(wf.WdError) as e:
        wf.decode(graph, x, *args, mode="chip", flags=wf.WD_FLAG_PHASES)
    assert e.value.status == wf.WD_EINVAL
