"""Store the oracle's result for a prefix of the wide-beam 2M-state workload.

The CPU oracle needs several seconds per frame on this graph (650k tokens and
1.1M candidate links per frame), too slow to run inside a GPU test, so its
canonical result for the first T frames is computed here once and committed
as tests/golden/wide_2m_<T>.npz and tests/golden/wide_2m_dyadic_<T>.npz:
  - the 1-best words, the cost bits and the decode statistics;
  - sha256 digests of every exact field of the lattice (each kept link's
    t, arc id, states, labels and graph/acoustic/forward/extra cost bits;
    each node's t, state, cost and extra cost bits): one per frame, so a
    mismatch names its first frame, and one over the whole lattice;
  - every kept link's posterior (float32; the parity bound is 1e-4).

Only synth/ (inputs) and oracle/ (the CPU decoder) are called.  The decode
is a whole utterance of T frames (beam 20, no max-active limit, lattice beam
10), so its lattice is pruned exactly at its last frame (Sec. 3.5); T = 200
spans six 32-frame windows of the GPU's incremental pruning and part of a
seventh.

  python tests/golden/make_wide_2m.py [--frames 200] [--names wide_2m,wide_2m_dyadic]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import synth  # noqa: E402

LINK_EXACT = ("t", "arc_id", "src_state", "dst_state", "ilabel", "olabel", "graph_cost", "ac_cost",
              "fwd_cost", "extra")
NODE_EXACT = ("t", "state", "cost", "extra")
STATS = ("frames", "final_reached", "arcs_expanded", "eps_arcs_expanded", "tokens", "max_tokens",
         "raw_links", "kept_links", "nodes")


def _digest(arrs) -> str:
    h = hashlib.sha256()
    for a in arrs:
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()


def frame_digests(links, nodes, T: int) -> tuple[list, list]:
    """Per frame t = 0..T: sha256 of the exact link fields and of the node
    fields of that frame (records in canonical order, floats as bits)."""
    lf = np.searchsorted(links["t"], np.arange(T + 2))
    nf = np.searchsorted(nodes["t"], np.arange(T + 2))
    dl = [_digest([np.ascontiguousarray(links[f][lf[t]:lf[t + 1]]) for f in LINK_EXACT]) for t in range(T + 1)]
    dn = [_digest([np.ascontiguousarray(nodes[f][nf[t]:nf[t + 1]]) for f in NODE_EXACT]) for t in range(T + 1)]
    return dl, dn


def exact_digest(words, cost, links, nodes) -> str:
    """sha256 over the fields that must match bit for bit (floats as bits)."""
    return _digest([np.ascontiguousarray(words, np.int32), np.float32(cost).view(np.uint32)] +
                   [links[f] for f in LINK_EXACT] + [nodes[f] for f in NODE_EXACT])


def path(name: str, T: int) -> str:
    return os.path.join(HERE, f"{name}_{T}.npz")


def make(name: str, T: int) -> str:
    cfg = synth.workload(name)
    g = synth.make_graph(cfg)
    L = synth.make_loglikes(cfg)[:T]
    t0 = time.time()
    o = oracle.decode(g, L, cfg["beam"], cfg["max_active"], cfg["lattice_beam"])
    dt = time.time() - t0
    dl, dn = frame_digests(o.links, o.nodes, T)
    meta = dict(workload=name, frames=T, beam=cfg["beam"], max_active=cfg["max_active"],
                lattice_beam=cfg["lattice_beam"], stats={k: int(o.stats[k]) for k in STATS},
                words=[int(w) for w in o.words], cost_bits=int(np.float32(o.cost).view(np.uint32)),
                n_links=int(o.links.size), n_nodes=int(o.nodes.size),
                digest=exact_digest(o.words, o.cost, o.links, o.nodes),
                link_digests=dl, node_digests=dn, oracle_seconds=round(dt, 1))
    out = path(name, T)
    np.savez_compressed(out, meta=np.array(json.dumps(meta)),
                        posterior=o.links["posterior"].astype(np.float32))
    print(f"{name} T={T}: {dt:.0f} s, {o.links.size} links, {o.nodes.size} nodes, "
          f"{os.path.getsize(out) / 1e6:.2f} MB -> {out}", flush=True)
    return out


def load(name: str, T: int):
    """(meta, posteriors) of a stored result."""
    with np.load(path(name, T), allow_pickle=False) as z:
        return json.loads(str(z["meta"])), z["posterior"].astype(np.float64)


def compare(meta: dict, post: np.ndarray, words, cost, links, nodes, stats: dict, tol: float = 1e-4) -> None:
    """Raise AssertionError naming the first difference between a decode
    result (links, nodes in the canonical record layout) and a stored one."""
    T = meta["frames"]
    assert [int(w) for w in words] == meta["words"], "words"
    assert int(np.float32(cost).view(np.uint32)) == meta["cost_bits"], ("cost", float(cost))
    for k in STATS:
        if k in stats:
            assert int(stats[k]) == meta["stats"][k], (k, int(stats[k]), meta["stats"][k])
    assert links.size == meta["n_links"], ("kept links", links.size, meta["n_links"])
    assert nodes.size == meta["n_nodes"], ("nodes", nodes.size, meta["n_nodes"])
    dl, dn = frame_digests(links, nodes, T)
    for t in range(T + 1):
        assert dl[t] == meta["link_digests"][t], f"lattice links of frame {t} differ"
        assert dn[t] == meta["node_digests"][t], f"lattice nodes of frame {t} differ"
    assert exact_digest(words, cost, links, nodes) == meta["digest"], "whole-lattice digest"
    d = np.abs(links["posterior"] - post)
    assert d.size == 0 or d.max() <= tol, f"posterior max diff {d.max()}"


if __name__ == "__main__":
    ap = argparse.ArgumentParser()
    ap.add_argument("--frames", type=int, default=200)
    ap.add_argument("--names", default="wide_2m,wide_2m_dyadic")
    a = ap.parse_args()
    oracle.build()
    for n in a.names.split(","):
        make(n, a.frames)
