"""Streaming decodes (wd_stream_begin / advance / end) against the CPU oracle
and against whole-utterance decodes: log-likelihoods arrive in chunks of any
size (empty chunks, single frames, chunk ends on and around the 32-frame
pruning windows), the decoder carries its frontier and counters between
launches, and the result is the whole utterance's, bit for bit."""
import math

import numpy as np
import pytest

import synth
from gpu_compare import assert_same

pytestmark = pytest.mark.gpu
MODES = ["workgroup", "chip", "chip_dyn"]


@pytest.fixture(scope="module")
def wf():
    import torch
    from paper_1804_03243_amd import wfstdec
    assert torch.cuda.is_available()
    wfstdec.lib()
    return wfstdec


@pytest.fixture(scope="module")
def tiny10k(wf):
    cfg = synth.workload("tiny_10k")
    g = synth.make_graph(cfg)
    return cfg, g, synth.make_loglikes(cfg), wf.Graph(g, cfg["P"])


def chunks(pattern, T, seed=0):
    """Chunk sizes summing to T: a fixed list (cycled), or 'random'."""
    out, left, i = [], T, 0
    rng = np.random.default_rng(seed)
    while left > 0:
        n = int(rng.integers(0, 40)) if pattern == "random" else pattern[i % len(pattern)]
        n = min(n, left)
        out.append(n)
        left -= n
        i += 1
    return out


def stream_decode(wf, graph, L, args, sizes, mode, debug=False, max_T=None):
    import torch
    x = torch.from_numpy(np.ascontiguousarray(L)).to(graph.device)
    s = wf.Stream(graph, 1, max_T if max_T is not None else L.shape[0], *args, debug=debug, mode=mode)
    t = 0
    for n in sizes:
        s.push([x[t:t + n]])
        t += n
    assert t == L.shape[0]
    return s.end()[0]


PATTERNS = {"ones": [1], "window": [31, 1, 32, 33], "random": "random", "whole": [10 ** 6],
            "empty_first": [0, 0, 7, 0, 300]}


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("pattern", sorted(PATTERNS))
@pytest.mark.parametrize("debug", [False, True])
def test_stream_tiny_10k(wf, oracle_mod, tiny10k, mode, pattern, debug):
    cfg, g, L, graph = tiny10k
    args = (cfg["beam"], cfg["max_active"], cfg["lattice_beam"])
    sizes = chunks(PATTERNS[pattern], L.shape[0], seed=5)
    print(f"\n[gpu case] stream tiny_10k pattern={pattern} chunks={len(sizes)} mode={mode} debug={debug}",
          flush=True)
    r = stream_decode(wf, graph, L, args, sizes, mode, debug=debug)
    o = oracle_mod.decode(g, L, *args, debug=debug)
    assert_same(r, o, debug=debug)


@pytest.mark.parametrize("mode", MODES)
def test_stream_short_and_empty(wf, oracle_mod, tiny10k, mode):
    """No frame at all (end right after begin), and a single frame; max_T
    larger than the frames received."""
    cfg, g, L, graph = tiny10k
    args = (cfg["beam"], cfg["max_active"], cfg["lattice_beam"])
    print(f"\n[gpu case] stream T=0 and T=1 mode={mode}", flush=True)
    for T in (0, 1):
        r = stream_decode(wf, graph, L[:T], args, [T] if T else [], mode, debug=True, max_T=50)
        assert_same(r, oracle_mod.decode(g, L[:T], *args, debug=True), debug=True)


def test_stream_batch(wf, oracle_mod, tiny10k):
    """Several utterances in one stream, advancing by different amounts (and
    not at all) in each push; one workgroup per utterance."""
    import torch
    cfg, g, L, graph = tiny10k
    args = (10.0, 40, 6.0)
    lens = [50, 1, 120, 0, 77]
    Ls = [np.ascontiguousarray(synth.tiny_loglikes(900 + i, n, cfg["P"]) * 3 - 10, dtype=np.float32)
          for i, n in enumerate(lens)]
    xs = [torch.from_numpy(x).to(graph.device) for x in Ls]
    print(f"\n[gpu case] stream batch lens={lens}", flush=True)
    s = wf.Stream(graph, len(lens), max(lens), *args, debug=True, mode="workgroup")
    rng = np.random.default_rng(11)
    pos = [0] * len(lens)
    while any(p < n for p, n in zip(pos, lens)):
        push = []
        for i, n in enumerate(lens):
            k = int(rng.integers(0, 25)) if rng.random() < 0.7 else 0
            k = min(k, n - pos[i])
            push.append(xs[i][pos[i]:pos[i] + k] if k or rng.random() < 0.5 else None)
            pos[i] += k
        s.push(push)
    rs = s.end()
    for i in range(len(lens)):
        assert_same(rs[i], oracle_mod.decode(g, Ls[i], *args, debug=True), debug=True)


@pytest.fixture(scope="module")
def wide(wf, oracle_mod):
    cfg = synth.workload("wide_2m_dyadic")
    g = synth.make_graph(cfg)
    L = synth.make_loglikes(cfg)[:4]
    args = (cfg["beam"], cfg["max_active"], cfg["lattice_beam"])
    return g, L, wf.Graph(g, cfg["P"]), args, oracle_mod.decode(g, L, *args, debug=True)


@pytest.mark.parametrize("mode", MODES)
def test_stream_wide_frontier(wf, wide, mode):
    """Frames of tens of thousands of tokens: the frontier lives in the
    workspace, not in LDS, when a chunk ends."""
    g, L, graph, args, o = wide
    print(f"\n[gpu case] stream wide_2m_dyadic T=4 chunks 1,0,2,1 mode={mode}", flush=True)
    r = stream_decode(wf, graph, L, args, [1, 0, 2, 1], mode, debug=True)
    assert_same(r, o, debug=True)
    assert r.stats["max_tokens"] > 2048


@pytest.fixture(scope="module")
def hclg(wf):
    cfg = synth.workload("hclg_5m")
    g = synth.make_graph(cfg)
    return cfg, synth.make_loglikes(cfg), wf.Graph(g, cfg["P"])


@pytest.mark.parametrize("mode", MODES)
def test_stream_hclg_5m_equals_decode(wf, hclg, mode):
    """The 5M-state graph in 32-frame chunks equals the whole-utterance
    decode (which the parity suite checks against the oracle)."""
    import torch
    cfg, L, graph = hclg
    args = (cfg["beam"], cfg["max_active"], cfg["lattice_beam"])
    print(f"\n[gpu case] stream hclg_5m chunks of 32 mode={mode}", flush=True)
    r = stream_decode(wf, graph, L, args, chunks([32], L.shape[0]), mode)
    w = wf.decode(graph, torch.from_numpy(L).to(graph.device), *args, mode=mode)
    assert_same(r, w)


@pytest.mark.parametrize("mode", MODES)
def test_stream_invalid_chunk(wf, tiny10k, mode):
    """A NaN in a later chunk: WD_EINVAL at the end."""
    import torch
    cfg, g, L, graph = tiny10k
    bad = L[:40].copy()
    bad[33, 3] = np.nan
    x = torch.from_numpy(bad).to(graph.device)
    print(f"\n[gpu case] stream NaN in the second chunk mode={mode}", flush=True)
    s = wf.Stream(graph, 1, 40, 10.0, 0, 5.0, mode=mode)
    s.push([x[:20]])
    s.push([x[20:]])
    with pytest.raises(wf.WdError) as e:
        s.end()
    assert e.value.status == wf.WD_EINVAL


def test_stream_argument_errors(wf, tiny10k):
    import torch
    cfg, g, L, graph = tiny10k
    x = torch.from_numpy(L[:12]).to(graph.device)
    print("\n[gpu case] stream argument errors", flush=True)
    s = wf.Stream(graph, 1, 10, 10.0, 2000, 6.0, mode="workgroup")
    with pytest.raises(ValueError):
        s.push([x])                      # past max_T, caught by the binding
    with pytest.raises(wf.WdError) as e:
        wf.wd_stream_advance(s.handle, [11])  # past max_T, caught by the library
    assert e.value.status == wf.WD_EINVAL
    with pytest.raises(wf.WdError) as e:
        wf.wd_stream_advance(s.handle, [-1])
    assert e.value.status == wf.WD_EINVAL
    s.push([x[:10]])
    r = s.end()[0]
    assert r.stats["frames"] == 10
    # chip-wide streams hold one utterance
    with pytest.raises(wf.WdError) as e:
        wf.Stream(graph, 2, 10, 10.0, 2000, 6.0, mode="chip")
    assert e.value.status == wf.WD_EINVAL


@pytest.mark.parametrize("mode", MODES)
def test_stream_capacity_fallback(wf, oracle_mod, tiny10k, mode):
    """Tiny capacities: the stream ends with WD_ECAPACITY and the binding
    decodes the frame store again with the capacities it reported."""
    cfg, g, L, graph = tiny10k
    L80 = L[:80]
    print(f"\n[gpu case] stream capacity fallback mode={mode}", flush=True)
    import torch
    x = torch.from_numpy(np.ascontiguousarray(L80)).to(graph.device)
    s = wf.Stream(graph, 1, 80, 10.0, 2000, 6.0, mode=mode, caps=wf.wd_caps(64, 64, 500, 500, 16, 40))
    for t in range(0, 80, 16):
        s.push([x[t:t + 16]])
    r = s.end()[0]
    assert_same(r, oracle_mod.decode(g, L80, 10.0, 2000, 6.0))
    assert not math.isnan(float(r.cost))


def test_concurrent_chip_decodes(wf, oracle_mod, tiny10k):
    """Chip-wide decodes from two host threads on two HIP streams share the
    library's pruning stream (each decode orders it with its own events):
    every result equals the oracle's.  Each thread has its own Graph (a
    Graph's workspace serves one decode at a time)."""
    import threading
    import torch
    cfg, g, L, _ = tiny10k
    args = (10.0, 0, 6.0)
    L1, L2 = L[:150], L[100:300]
    o1, o2 = oracle_mod.decode(g, L1, *args), oracle_mod.decode(g, L2, *args)
    graphs = [wf.Graph(g, cfg["P"]), wf.Graph(g, cfg["P"])]
    xs = [torch.from_numpy(np.ascontiguousarray(a)).to(graphs[0].device) for a in (L1, L2)]
    print("\n[gpu case] two threads x 3 chip-wide decodes on two streams", flush=True)
    results, errors = [[], []], []

    def work(k):
        try:
            s = torch.cuda.Stream()
            with torch.cuda.stream(s):
                for _ in range(3):
                    results[k].append(wf.decode(graphs[k], xs[k], *args, mode="chip"))
        except Exception as e:  # reported below
            errors.append(e)

    th = [threading.Thread(target=work, args=(k,)) for k in range(2)]
    for t in th:
        t.start()
    for t in th:
        t.join()
    assert not errors, errors
    for r in results[0]:
        assert_same(r, o1)
    for r in results[1]:
        assert_same(r, o2)


@pytest.mark.parametrize("mode", ["workgroup", "chip"])
def test_stream_chunks_from_another_stream(wf, oracle_mod, tiny10k, mode):
    """Chunks produced on a side stream (a pretend acoustic model: a
    host-to-device copy and a scale on that stream) and pushed while the
    side stream is current: the decode, on the stream the decoder was built
    on, waits for each chunk."""
    import torch
    cfg, g, L, graph = tiny10k
    args = (cfg["beam"], cfg["max_active"], cfg["lattice_beam"])
    print(f"\n[gpu case] stream chunks from a side stream mode={mode}", flush=True)
    half = np.ascontiguousarray(L * np.float32(0.5))
    s = wf.Stream(graph, 1, L.shape[0], *args, mode=mode)
    side = torch.cuda.Stream(graph.device)
    host = torch.from_numpy(half).pin_memory()
    t = 0
    with torch.cuda.stream(side):
        for n in chunks([37, 1, 64], L.shape[0], seed=3):
            x = host[t:t + n].to(graph.device, non_blocking=True)
            x = x * 2.0  # exact: restores L
            s.push([x])
            del x
            t += n
    r = s.end()[0]
    assert_same(r, oracle_mod.decode(g, L, *args))
