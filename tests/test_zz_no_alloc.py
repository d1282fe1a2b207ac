"""The decode entry point that allocates nothing (wd_decode_noalloc: the
workspace is the library's fixed device scratch, results go into the
caller's host buffers), through the C ABI, against wd_decode on the same
inputs: two calls in a row, the second with a smaller input, so the second
decode runs on a scratch that still holds the first one's contents."""
import numpy as np
import pytest

import synth
from gpu_compare import assert_links_equal

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def wf():
    import torch
    from paper_1804_03243_amd import wfstdec
    assert torch.cuda.is_available()
    wfstdec.lib()
    return wfstdec


def _bits(a):
    return np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)


def _noalloc(wf, graph, x, args, caps=None, cap=200_000):
    import torch
    p = wf.wd_params(float(args[0]), int(args[1]), float(args[2]), wf.WD_FLAG_ONE_WORKGROUP)
    words = np.zeros(cap, np.int32)
    links = np.zeros(cap, wf.LINK_DTYPE)
    nodes = np.zeros(cap, wf.NODE_DTYPE)
    st, cost, nw, stats, needed = wf.wd_decode_noalloc(
        graph.handle, x.data_ptr() if x.numel() else 0, int(x.shape[0]), p, caps,
        torch.cuda.current_stream(graph.device).cuda_stream, words, links, nodes)
    return st, cost, words[:nw], links[:stats["kept_links"]], nodes[:stats["nodes"]], stats, needed


def _same(wf, a, ref):
    st, cost, words, links, nodes, stats, _ = a
    assert st == wf.WD_OK, (st, wf.lib().wd_last_error())
    assert _bits(cost) == _bits(ref.cost)
    assert list(words) == list(ref.words)
    assert_links_equal(links, ref.links, 1e-4)
    assert np.array_equal(nodes["t"], ref.nodes["t"]) and np.array_equal(nodes["state"], ref.nodes["state"])
    assert np.array_equal(_bits(nodes["cost"]), _bits(ref.nodes["cost"]))
    assert np.array_equal(_bits(nodes["extra"]), _bits(ref.nodes["extra"]))
    for k in ("arcs_expanded", "eps_arcs_expanded", "tokens", "max_tokens", "raw_links", "kept_links", "nodes",
              "frames", "final_reached"):
        assert stats[k] == ref.stats[k], k


@pytest.mark.parametrize("workload,T1,T2", [("tiny_10k", 300, 97), ("hclg_5m", 400, 150)])
def test_noalloc_equals_decode(wf, workload, T1, T2):
    import torch
    cfg = synth.workload(workload)
    g = synth.make_graph(cfg)
    L = synth.make_loglikes(cfg)
    graph = wf.Graph(g, cfg["P"])
    args = (cfg["beam"], cfg["max_active"], cfg["lattice_beam"])
    for T in (T1, T2):
        print(f"\n[gpu case] noalloc {workload} T={T}", flush=True)
        x = torch.from_numpy(np.ascontiguousarray(L[:T])).to(graph.device)
        ref = wf.decode(graph, x, *args, mode="workgroup")
        # capacities as a serving loop would keep them: what a first decode needed, with room
        caps = wf.wd_caps(*(max(2 * ref.needed[f], 1024) for f, _ in wf.wd_caps._fields_))
        _same(wf, _noalloc(wf, graph, x, args, caps), ref)


def test_noalloc_limits(wf):
    """A workspace beyond the scratch, chip-wide or debug flags, and too
    small output buffers are refused with their status; the scratch is not
    touched by the refused calls, and a decode right after still matches."""
    import torch
    cfg = synth.workload("tiny_10k")
    g = synth.make_graph(cfg)
    L = synth.make_loglikes(cfg)[:60]
    graph = wf.Graph(g, cfg["P"])
    args = (cfg["beam"], cfg["max_active"], cfg["lattice_beam"])
    x = torch.from_numpy(L).to(graph.device)
    print("\n[gpu case] noalloc limits", flush=True)
    big = wf.wd_caps(0, 0, 0, wf.WD_NOALLOC_SCRATCH_BYTES // 16, 0, 0)
    st = _noalloc(wf, graph, x, args, big)[0]
    assert st == wf.WD_EINVAL and "scratch" in wf.lib().wd_last_error().decode()
    stream = torch.cuda.current_stream(graph.device).cuda_stream
    for flags in (wf.WD_FLAG_CHIP_WIDE, wf.WD_FLAG_DEBUG | wf.WD_FLAG_ONE_WORKGROUP,
                  wf.WD_FLAG_TIMING | wf.WD_FLAG_ONE_WORKGROUP):
        p = wf.wd_params(10.0, 2000, 6.0, flags)
        a = np.zeros(16, np.int32)
        st = wf.wd_decode_noalloc(graph.handle, x.data_ptr(), 60, p, None, stream, a,
                                  np.zeros(16, wf.LINK_DTYPE), np.zeros(16, wf.NODE_DTYPE))[0]
        assert st == wf.WD_EINVAL
    st, cost, words, links, nodes, stats, _ = _noalloc(wf, graph, x, args, cap=3)
    assert st == wf.WD_ECAPACITY and stats["kept_links"] > 3
    ref = wf.decode(graph, x, *args, mode="workgroup")
    _same(wf, _noalloc(wf, graph, x, args), ref)
