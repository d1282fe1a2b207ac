"""Comparison of a GPU decode result with the oracle's, field by field."""
import numpy as np

STATS = ("final_reached", "arcs_expanded", "eps_arcs_expanded", "tokens", "max_tokens", "raw_links",
         "kept_links", "nodes")


def _bits(a):
    return np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)


def assert_links_equal(g, o, post_tol, what="links"):
    assert g.size == o.size, f"{what}: {g.size} != {o.size}"
    for f in ("t", "arc_id", "src_state", "dst_state", "ilabel", "olabel"):
        if not np.array_equal(g[f], o[f]):
            i = int(np.flatnonzero(g[f] != o[f])[0])
            raise AssertionError(f"{what}.{f} differs first at {i}: gpu {g[i]} oracle {o[i]}")
    for f in ("graph_cost", "ac_cost", "fwd_cost", "extra"):
        if not np.array_equal(_bits(g[f]), _bits(o[f])):
            i = int(np.flatnonzero(_bits(g[f]) != _bits(o[f]))[0])
            raise AssertionError(f"{what}.{f} differs first at {i}: gpu {g[i]} oracle {o[i]}")
    d = np.abs(g["posterior"] - o["posterior"])
    assert d.size == 0 or d.max() <= post_tol, f"{what}.posterior max diff {d.max()}"


def assert_same(gpu, orc, debug=False, post_tol=1e-4):
    assert gpu.cost.view(np.uint32) == np.float32(orc.cost).view(np.uint32), (gpu.cost, orc.cost)
    assert list(gpu.words) == list(orc.words), "words"
    for k in STATS:
        assert gpu.stats[k] == orc.stats[k], (k, gpu.stats[k], orc.stats[k])
    assert_links_equal(gpu.links, orc.links, post_tol)
    assert np.array_equal(gpu.nodes["t"], orc.nodes["t"])
    assert np.array_equal(gpu.nodes["state"], orc.nodes["state"])
    assert np.array_equal(_bits(gpu.nodes["cost"]), _bits(orc.nodes["cost"]))
    assert np.array_equal(_bits(gpu.nodes["extra"]), _bits(orc.nodes["extra"]))
    if debug:
        for f in ("best", "cutoff_beam", "cutoff"):
            assert np.array_equal(_bits(getattr(gpu, f)), _bits(getattr(orc, f))), f
        gt, ot = gpu.tokens, orc.tokens
        assert gt.size == ot.size, ("tokens", gt.size, ot.size)
        for f in ("t", "state", "pred_arc"):
            assert np.array_equal(gt[f], ot[f]), f"tokens.{f}"
        assert np.array_equal(_bits(gt["cost"]), _bits(ot["cost"])), "tokens.cost"
        assert_links_equal(gpu.raw_links, orc.raw_links, post_tol, "raw_links")
