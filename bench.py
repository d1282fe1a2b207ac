"""Benchmark: decoded frames/s (and arcs expanded/s, RTF, HBM fraction) of the
GPU decoder on the 5M-state HCLG-shaped workload, one MI355X.

One step = one full decode of the 1000-frame utterance: token passing with
recombination, epsilon closure, beam and max-active pruning, lattice links,
lattice pruning, posteriors and the final merge, results copied to the host.
Inputs (graph and log-likelihoods) are resident in GPU memory before timing.

Prints one JSON line.  `python bench.py [--gpus 1] [--steps K] [--warmup W]`.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

WORKLOAD = "hclg_5m"
HBM_PEAK_GBS = 8000.0       # MI355X HBM3E
FRAME_RATE = 100.0 / 3.0    # sub-sampled frame rate (frames per second of audio)
METRIC = "decoded frames/sec + arcs expanded/sec at 1 GPU; % of HBM peak"

# Algorithmic bytes the token-passing kernel must move (not what a dense
# Viterbi would): per expanded arc its 16-byte record and the 8-byte slot
# atomic, plus the 4-byte log-likelihood gather for emitting arcs; per
# surviving token 8 bytes of offsets, 12 read and 12 written; per lattice
# link 16 bytes written.
BYTES_ARC = 16 + 8
BYTES_LOGLIKE = 4
BYTES_TOKEN = 8 + 12 + 12
BYTES_LINK = 16


def algorithmic_bytes(stats: dict) -> int:
    emit = stats["arcs_expanded"] - stats["eps_arcs_expanded"]
    return (stats["arcs_expanded"] * BYTES_ARC + emit * BYTES_LOGLIKE +
            stats["tokens"] * BYTES_TOKEN + stats["raw_links"] * BYTES_LINK)


def cpu_baseline(g, L, cfg, min_seconds: float = 10.0) -> dict:
    """The CPU oracle (plain sequential C, one thread) on the same utterance,
    repeated until about `min_seconds` of CPU work."""
    import oracle
    oracle.build()
    runs, t0 = 0, time.perf_counter()
    while True:
        oracle.decode(g, L, cfg["beam"], cfg["max_active"], cfg["lattice_beam"])
        runs += 1
        dt = time.perf_counter() - t0
        if dt >= min_seconds:
            break
    return {"value": round(runs * L.shape[0] / dt, 2), "unit": "frames/s", "cores": 1, "kind": "oracle",
            "sample": f"{WORKLOAD} full utterance ({L.shape[0]} frames) x {runs} runs, one thread, "
                      f"{dt:.1f} s"}


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this decoder runs on one GPU; --gpus {args.gpus} is not supported "
              "(utterances shard across GPUs with no exchange, see DESIGN.md)", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    import synth
    from paper_1804_03243_amd import wfstdec

    cfg = synth.workload(WORKLOAD)
    g = synth.make_graph(cfg)
    L = synth.make_loglikes(cfg)
    dev = torch.device("cuda:0")
    graph = wfstdec.Graph(g, cfg["P"], "cuda:0")
    x = torch.from_numpy(L).to(dev)
    beam, ma, lb = cfg["beam"], cfg["max_active"], cfg["lattice_beam"]

    for _ in range(max(1, args.warmup)):
        r = wfstdec.decode(graph, x, beam, ma, lb, timing=True)
    torch.cuda.synchronize()
    fwd_ms, lat_ms = [], []
    t0 = time.perf_counter()
    for _ in range(args.steps):
        r = wfstdec.decode(graph, x, beam, ma, lb, timing=True)
        fwd_ms.append(r.stats["forward_ms"])
        lat_ms.append(r.stats["lattice_ms"])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    T = L.shape[0]
    ms_step = 1e3 * wall / args.steps
    fps = T * args.steps / wall
    st = r.stats
    fwd = float(np.mean(fwd_ms))
    bytes_launch = algorithmic_bytes(st)
    achieved = bytes_launch / (fwd * 1e-3) / 1e9
    out = {
        "metric": METRIC,
        "value": round(fps, 2),
        "unit": "frames/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": WORKLOAD, "states": cfg["S"], "arcs": cfg["A"], "frames": T,
                   "pdfs": cfg["P"], "beam": beam, "max_active": ma, "lattice_beam": lb,
                   "utterances_per_step": 1},
        "arcs_expanded_per_s": round(st["arcs_expanded"] * args.steps / wall, 1),
        "rtf": round((wall / args.steps) / (T / FRAME_RATE), 7),
        "tokens_per_frame": round(st["tokens"] / (T + 1), 1),
        "kernel_ms": {"forward": round(fwd, 3), "lattice": round(float(np.mean(lat_ms)), 3)},
        "roofline": {"bound": "hbm", "kernel": "k_forward", "achieved": round(achieved, 3),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 6),
                     "traffic": None, "algorithmic_bytes_per_launch": int(bytes_launch)},
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(g, L, cfg)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
