"""Benchmark: decoded frames/s (and arcs expanded/s, RTF, HBM fraction) of the
GPU decoder on the 5M-state HCLG-shaped workload, one MI355X.

One step = one full decode of the 1000-frame utterance: token passing with
recombination, epsilon closure, beam and max-active pruning, lattice links,
lattice pruning, posteriors and the final merge, results copied to the host.
Inputs (graph and log-likelihoods) are resident in GPU memory before timing.

Prints one JSON line.  `python bench.py [--gpus 1] [--steps K] [--warmup W]`.

Besides the headline line's fields: `roofline.traffic` is the HBM traffic of
one k_forward launch measured with hardware counters (FETCH_SIZE + WRITE_SIZE,
each scaled by what the same counter reads for a plain device copy of known
size), reported only while the kernel sources hash to the ones the counters
were taken on; `other_workloads` times the same utterance streamed in chunks
of 32 and 8 frames, the host determinisation of its lattice, the
64-utterance batch on the same graph (with its own roofline), and the
chip-wide mode on the wide-beam 2M-state graph (with and without incremental
lattice pruning, and with dynamic load balancing); `roofline.copy_ceiling_gbs`
is what a plain device copy reaches.  `--copy-kernel-bytes N` only runs a plain N-byte device copy
(the counter calibration run) and exits.
"""
from __future__ import annotations

import argparse
import hashlib
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
BYTES_ARC_RECORD = 16
BYTES_ARC = BYTES_ARC_RECORD + 8
BYTES_LOGLIKE = 4
BYTES_TOKEN = 8 + 12 + 12
BYTES_LINK = 16


# HBM traffic of one k_forward launch on this workload, from rocprofv3 --pmc
# runs of this script (FETCH_SIZE, then WRITE_SIZE, KiB per dispatch), each
# divided by the counter's reading per byte of a plain device copy of known
# size (bench.py --copy-kernel-bytes).  Valid while k_forward's sources hash to this.
TRAFFIC = {"sources_sha256": "939d545fec9ffe3ba92d01c1a49c7271ec731bb32f90926100672b7b1ed07a56",
           "bytes_per_launch": 65999327}


# what k_forward is built from, and the device graph layout it reads
FORWARD_SOURCES = ("wd_block.h", "wd_common.h", "wd_forward.hip", "wd_graph.hip")


def sources_sha256() -> str:
    d = os.path.join(ROOT, "paper_1804_03243_amd", "csrc")
    h = hashlib.sha256()
    for name in FORWARD_SOURCES:
        with open(os.path.join(d, name), "rb") as f:
            h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()


def copy_kernel(nbytes: int) -> int:
    """A plain device-to-device copy of nbytes, five times (counter calibration)."""
    import torch
    src = torch.ones(nbytes, dtype=torch.uint8, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_kernel_bytes": nbytes, "launches": 5}), flush=True)
    return 0


def wide_chip(wfstdec, steps: int = 3, mode: str = "chip", cpu: bool = False, cpu_frames: int = 10) -> dict:
    """Chip-wide mode on the wide-beam 2M-state graph (800 frames, beam 20,
    no max-active): full decodes, lattice and posteriors included.
    mode "chip_dyn": the same with dynamic load balancing of the emitting
    arcs (the A/B against the prefix-sum work space)."""
    import synth
    import torch
    cfg = synth.workload("wide_2m")
    g = synth.make_graph(cfg)
    L = synth.make_loglikes(cfg)
    graph = wfstdec.Graph(g, cfg["P"], "cuda:0")
    x = torch.from_numpy(L).to(graph.device)
    args = (cfg["beam"], cfg["max_active"], cfg["lattice_beam"])
    r = wfstdec.decode(graph, x, *args, timing=True, mode=mode)  # sizes the workspace
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    fwd, lat = [], []
    for _ in range(steps):
        r = wfstdec.decode(graph, x, *args, timing=True, mode=mode)
        fwd.append(r.stats["forward_ms"])
        lat.append(r.stats["lattice_ms"])
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) / steps
    T = L.shape[0]
    st = r.stats
    out = {"workload": "wide_2m", "mode": mode, "frames": T, "steps": steps,
           "frames_per_s": round(T / wall, 1), "ms_per_step": round(1e3 * wall, 2),
           "arcs_expanded_per_s": round(st["arcs_expanded"] / wall, 1),
           "tokens_per_frame": round(st["tokens"] / (T + 1), 1),
           "raw_links": st["raw_links"], "kept_links": st["kept_links"], "link_store_links": r.needed["links"] + 2 * r.needed["window_links"],
           "kernel_ms": {"forward": round(sum(fwd) / steps, 2), "lattice": round(sum(lat) / steps, 2)}}
    # the forward pass is ~25 kernels per frame; their summed time (HIP events
    # around the decode's forward part on its stream) against its bytes
    nbytes = algorithmic_bytes(st)
    f_ms = sum(fwd) / steps
    achieved = nbytes / (f_ms * 1e-3) / 1e9
    out["roofline"] = {"bound": "hbm", "kernel": "chip-wide forward kernels (all launches of the forward pass)",
                       "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                       "frac": round(achieved / HBM_PEAK_GBS, 5), "algorithmic_bytes_per_launch": int(nbytes)}
    if cpu:
        out["cpu_baseline"] = cpu_prefix_baseline(g, L, cfg, "wide_2m", cpu_frames)
    if mode == "chip":
        # host determinisation of this lattice, pruned to a beam of 6 (the
        # lattice beam is 10; at 10 the compact lattice keeps ~450 arcs/frame)
        t0 = time.perf_counter()
        c = wfstdec.determinize(r, int(g.get("start_state", 0)), g.get("final_weight"), beam=6.0)
        out["determinize"] = {"where": "host, one thread", "beam": 6.0,
                              "ms": round(1e3 * (time.perf_counter() - t0), 1),
                              "lattice_arcs_per_frame": round(len(r.links) / T, 1),
                              "compact_arcs_per_frame": round(len(c.arcs) / T, 2)}
    del graph
    torch.cuda.empty_cache()
    return out


def stream_hclg(wfstdec, graph, x, cfg, chunk: int, steps: int = 3) -> dict:
    """The headline utterance streamed in chunks of `chunk` frames
    (wd_stream_*): throughput with every chunk pushed without waiting (begin
    to end, lattice included), and the latency of one chunk's decode when
    each push is waited for."""
    import numpy as np
    import torch
    T = int(x.shape[0])
    args = (cfg["beam"], cfg["max_active"], cfg["lattice_beam"])

    def run(wait: bool):
        s = wfstdec.Stream(graph, 1, T, *args, mode="workgroup")
        lat = []
        for t0 in range(0, T, chunk):
            a = time.perf_counter()
            s.push([x[t0:t0 + chunk]])
            if wait:
                torch.cuda.synchronize()
                lat.append(1e3 * (time.perf_counter() - a))
        return s.end()[0], lat

    run(False)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        r, _ = run(False)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) / steps
    _, lat = run(True)
    return {"workload": f"{WORKLOAD}_stream", "chunk_frames": chunk, "frames": T, "steps": steps,
            "frames_per_s": round(T / wall, 1), "ms_per_utterance": round(1e3 * wall, 2),
            "chunk_latency_ms": {"mean": round(float(np.mean(lat)), 3),
                                 "p95": round(float(np.percentile(lat, 95)), 3)},
            "cost": float(r.cost)}


def determinize_hclg(wfstdec, r, g, T: int, reps: int = 20) -> dict:
    """Host determinisation of the headline utterance's lattice (the compact
    exact lattice), timed over `reps` runs; lattice density (arcs per frame)
    before and after."""
    s0, fw = int(g.get("start_state", 0)), g.get("final_weight")
    t0 = time.perf_counter()
    for _ in range(reps):
        c = wfstdec.determinize(r, s0, fw)
    dt = (time.perf_counter() - t0) / reps
    return {"workload": f"{WORKLOAD}_determinize", "where": "host, one thread", "ms": round(1e3 * dt, 3),
            "lattice_arcs_per_frame": round(len(r.links) / T, 3),
            "compact_arcs_per_frame": round(len(c.arcs) / T, 3), "compact_states": int(c.states)}


_CPU_GRAPH = None


def _cpu_init(workload: str) -> None:
    global _CPU_GRAPH
    import oracle
    import synth
    oracle.build()
    cfg = synth.workload(workload)
    _CPU_GRAPH = (cfg, synth.make_graph(cfg))


def _cpu_decode(i: int) -> tuple:
    import oracle
    import synth
    cfg, g = _CPU_GRAPH
    if i < 0:
        return (0, os.getpid(), 0.0)  # warm-up task: the worker is initialised
    L = synth.make_loglikes(cfg, i)
    t0 = time.perf_counter()
    oracle.decode(g, L, cfg["beam"], cfg["max_active"], cfg["lattice_beam"])
    return (int(L.shape[0]), os.getpid(), time.perf_counter() - t0)


def cpu_batch_baseline(workload: str, n_utts: int) -> dict:
    """The CPU oracle on the batch, one utterance per task over a pool of
    processes (started fresh, they never touch the GPU), one per host core.
    Throughput = frames / the longest per-process sum of decode times (the
    log-likelihood generation of each task is not counted)."""
    import multiprocessing as mp
    n = os.cpu_count() or 1
    with mp.get_context("spawn").Pool(n, initializer=_cpu_init, initargs=(workload,)) as pool:
        pool.map(_cpu_decode, [-1] * n, chunksize=1)
        res = pool.map(_cpu_decode, range(n_utts), chunksize=1)
    frames = sum(r[0] for r in res)
    busy = {}
    for _, pid, dt in res:
        busy[pid] = busy.get(pid, 0.0) + dt
    span = max(busy.values())
    return {"value": round(frames / span, 1), "unit": "frames/s", "cores": len(busy), "kind": "oracle",
            "sample": f"all {n_utts} utterances of {workload} ({frames} frames) over {len(busy)} processes; "
                      f"longest per-process decode time {span:.1f} s, {sum(busy.values()):.1f} s of CPU work"}


def batch(wfstdec, graph, n_utts: int = 64, steps: int = 3, cpu: bool = True) -> dict:
    """A batch of utterances on the same graph (one workgroup per utterance,
    one launch for the batch): aggregate frames/s (median step) and the
    roofline of the batch's k_forward launch.  n_utts = 64 is the batch
    workload; 256 (one workgroup per CU) draws more utterances from the same
    distribution.  Algorithmic bytes credit an arc record once per unique
    (step, arc) over the lanes (`unique_arc_bytes`); the per-lane sum is
    reported beside it."""
    import numpy as np
    import synth
    import torch
    cfg = dict(synth.workload("batch64_hclg_5m"))
    cfg["batch"] = n_utts
    name = f"batch{n_utts}_hclg_5m"
    xs = [torch.from_numpy(synth.make_loglikes(cfg, i)).to(graph.device) for i in range(n_utts)]
    args = (cfg["beam"], cfg["max_active"], cfg["lattice_beam"])
    wfstdec.decode_batch(graph, xs, *args, timing=True)
    torch.cuda.synchronize()
    fwd, lat, walls = [], [], []
    for _ in range(steps):
        t0 = time.perf_counter()
        rs = wfstdec.decode_batch(graph, xs, *args, timing=True)
        torch.cuda.synchronize()
        walls.append(time.perf_counter() - t0)
        fwd.append(rs[0].stats["forward_ms"])
        lat.append(rs[0].stats["lattice_ms"])
    wall = float(np.median(walls))
    frames = sum(int(x.shape[0]) for x in xs)
    f_ms = float(np.median(fwd))
    lane_sum = sum(algorithmic_bytes(r.stats) for r in rs)
    uq = unique_arc_bytes(wfstdec, graph, xs, args, rs)
    nbytes = lane_sum - uq["duplicate_arc_records"] * BYTES_ARC_RECORD
    achieved = nbytes / (f_ms * 1e-3) / 1e9
    out = {"workload": name, "utterances": len(xs), "frames": frames, "steps": steps,
           "frames_per_s": round(frames / wall, 1), "ms_per_step": round(1e3 * wall, 2),
           "arcs_expanded_per_s": round(sum(r.stats["arcs_expanded"] for r in rs) / wall, 1),
           "kernel_ms": {"forward": round(f_ms, 3), "lattice": round(float(np.median(lat)), 3)},
           "roofline": {"bound": "hbm", "kernel": f"k_forward ({n_utts} workgroups)",
                        "achieved": round(achieved, 3), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                        "frac": round(achieved / HBM_PEAK_GBS, 6), "algorithmic_bytes_per_launch": int(nbytes),
                        "per_lane_sum_bytes": int(lane_sum), "unique_arcs": uq}}
    del xs, rs
    graph._ws = None  # the batch's workspace (~0.4 GB per utterance)
    torch.cuda.empty_cache()
    if cpu:
        out["cpu_baseline"] = cpu_batch_baseline(name, n_utts)
    return out


PHASE_NAMES = ("expand", "eps_closure", "survivors", "max_active", "compact", "degrees",
               "owners_warming", "bookkeeping", "frame_end")


LATTICE_PHASE_NAMES = ("final_costs", "pruning_sweep", "kept_links", "kept_offsets_records", "posteriors",
                       "merge", "node_list")


def phase_profile(wfstdec, workload: str, reps: int = 3) -> dict:
    """Step profile of the one-workgroup forward pass (WD_FLAG_PHASES): per
    frame the device wall clock at each step boundary, summarised as the mean
    microseconds per frame spent in each step (frames 1..T, all `reps`
    decodes), with the frames whose token table went to device memory
    counted apart.  The profiled kernel is a separate copy; its total is
    compared with the plain kernel's time in the same run."""
    import numpy as np
    import synth
    import torch
    cfg = synth.workload(workload)
    g = synth.make_graph(cfg)
    L = synth.make_loglikes(cfg)
    graph = wfstdec.Graph(g, cfg["P"], "cuda:0")
    x = torch.from_numpy(L).to(graph.device)
    args = (cfg["beam"], cfg["max_active"], cfg["lattice_beam"])
    plain = [wfstdec.decode(graph, x, *args, timing=True, mode="workgroup").stats["forward_ms"]
             for _ in range(reps + 1)][1:]
    rows, fwd, lat = [], [], []
    for _ in range(reps + 1):
        r = wfstdec.decode(graph, x, *args, timing=True, mode="workgroup", flags=wfstdec.WD_FLAG_PHASES)
        rows.append(r.phases[1:])
        fwd.append(r.stats["forward_ms"])
        lat.append(np.diff(r.lattice_phases.astype(np.int64)))
    rows, fwd, lat = rows[1:], fwd[1:], lat[1:]
    ph = np.concatenate(rows).astype(np.int64)
    hz = r.phase_tick_hz
    S = wfstdec.WD_PHASE_STAMPS
    st = ph[:, :S]
    # a step the frame skipped (no max-active cut, ...) has the previous stamp's value
    d = np.diff(st, axis=1).astype(np.float64) * 1e6 / hz
    frame_us = (st[:, S - 1] - st[:, 0]) * 1e6 / hz
    lds = (ph[:, S] & 1).astype(bool)
    ntok = (ph[:, S] >> 8) & 0xffffff
    nlink = ph[:, S] >> 32
    W = ph[:, S + 1] & 0xffffffff
    nbk = ph[:, S + 1] >> 32
    # frame end -> next frame's start, within each decode
    gap = np.concatenate([r[1:, 0].astype(np.int64) - r[:-1, S - 1].astype(np.int64) for r in rows]) * 1e6 / hz

    def summary(sel):
        if not sel.any():
            return None
        return {"frames": int(sel.sum()), "frame_us": round(float(frame_us[sel].mean()), 3),
                "step_us": {n: round(float(d[sel, i].mean()), 3) for i, n in enumerate(PHASE_NAMES)},
                "tokens": round(float(ntok[sel].mean()), 1), "emitting_items": round(float(W[sel].mean()), 1),
                "eps_bucket_entries": round(float(nbk[sel].mean()), 1), "links": round(float(nlink[sel].mean()), 1)}

    out = {"workload": workload, "kernel": "k_forward_phases (WD_FLAG_PHASES copy of k_forward)",
           "frames_per_decode": int(L.shape[0]), "decodes": reps, "tick_hz": hz,
           "forward_ms_plain": round(float(np.mean(plain)), 3),
           "forward_ms_profiled": round(float(np.mean(fwd)), 3),
           "all": summary(np.ones(len(lds), bool)), "lds_table": summary(lds),
           "device_table": summary(~lds),
           "between_frames_us": round(float(gap.mean()), 3) if gap.size else None,
           # the lattice pass of the same decodes (k_lattice, one workgroup)
           "lattice_us": {n: round(float(np.mean([v[i] for v in lat])) * 1e6 / hz, 1)
                          for i, n in enumerate(LATTICE_PHASE_NAMES)}}
    del graph
    torch.cuda.empty_cache()
    return out


def unique_arc_bytes(wfstdec, graph, xs, args, rs) -> dict:
    """Arc records a batch step shares between lanes.  Step t expands the
    emitting arcs of every lane's surviving tokens of frame t-1 and the
    epsilon arcs of its epsilon closure at frame t; an arc that several
    lanes expand in the same step is one record read, so the algorithmic
    bytes credit it once.  The closure's token set is taken as the frame's
    surviving tokens, which is exact while max-active does not cut (checked:
    the per-lane counts must reproduce each lane's arcs_expanded).  One
    debug decode of the batch (not timed) lists every lane's tokens."""
    import numpy as np
    dbg = wfstdec.decode_batch(graph, xs, *args, debug=True, mode="workgroup")
    edeg, xdeg = graph.degrees()
    keys_e, keys_x, lane_ok, total = [], [], True, 0
    for r, x in zip(dbg, xs):
        T = int(x.shape[0])
        t = r.tokens["t"].astype(np.int64)
        s_ = r.tokens["state"].astype(np.int64)
        n_lane = int(edeg[s_[t < T]].sum() + xdeg[s_].sum())
        lane_ok &= n_lane == r.stats["arcs_expanded"]
        total += n_lane
        keys_e.append((t[t < T] << 32) | s_[t < T])
        keys_x.append((t << 32) | s_)
    ue = np.unique(np.concatenate(keys_e)) & 0xffffffff
    ux = np.unique(np.concatenate(keys_x)) & 0xffffffff
    unique = int(edeg[ue].sum() + xdeg[ux].sum())
    return {"arcs_summed_over_lanes": total, "unique_step_arcs": unique,
            "duplicate_arc_records": total - unique if lane_ok else 0, "lane_counts_match": bool(lane_ok)}


def single(wfstdec, workload: str, steps: int = 5, cpu_seconds: float = 10.0, cpu: bool = True) -> dict:
    """One utterance of `workload` in the library's default mode: frames/s
    (median step), kernel times, the forward launch's roofline and the
    oracle on the host (the whole utterance, repeated for about
    `cpu_seconds`)."""
    import numpy as np
    import synth
    import torch
    cfg = synth.workload(workload)
    g = synth.make_graph(cfg)
    L = synth.make_loglikes(cfg)
    graph = wfstdec.Graph(g, cfg["P"], "cuda:0")
    x = torch.from_numpy(L).to(graph.device)
    args = (cfg["beam"], cfg["max_active"], cfg["lattice_beam"])
    wfstdec.decode(graph, x, *args, timing=True)
    torch.cuda.synchronize()
    walls, fwd, lat = [], [], []
    for _ in range(steps):
        t0 = time.perf_counter()
        r = wfstdec.decode(graph, x, *args, timing=True)
        torch.cuda.synchronize()
        walls.append(time.perf_counter() - t0)
        fwd.append(r.stats["forward_ms"])
        lat.append(r.stats["lattice_ms"])
    wall, f_ms = float(np.median(walls)), float(np.median(fwd))
    T = L.shape[0]
    nbytes = algorithmic_bytes(r.stats)
    achieved = nbytes / (f_ms * 1e-3) / 1e9
    out = {"workload": workload, "states": cfg["S"], "arcs": int(g["dst"].size), "frames": T, "steps": steps,
           "frames_per_s": round(T / wall, 1), "ms_per_step": round(1e3 * wall, 3),
           "arcs_expanded_per_s": round(r.stats["arcs_expanded"] / wall, 1),
           "rtf": round(wall / (T / FRAME_RATE), 7), "tokens_per_frame": round(r.stats["tokens"] / (T + 1), 1),
           "kernel_ms": {"forward": round(f_ms, 3), "lattice": round(float(np.median(lat)), 3)},
           "roofline": {"bound": "hbm", "kernel": "k_forward", "achieved": round(achieved, 3),
                        "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 7),
                        "algorithmic_bytes_per_launch": int(nbytes)}}
    del graph, x
    torch.cuda.empty_cache()
    if cpu:
        out["cpu_baseline"] = cpu_baseline(g, L, cfg, workload, min_seconds=cpu_seconds)
    return out


def copy_ceiling(nbytes: int = 1 << 30, reps: int = 10) -> float:
    """GB/s (bytes read + written) of a plain device-to-device copy: the
    bandwidth a streaming kernel reaches on this GPU."""
    import torch
    src = torch.ones(nbytes, dtype=torch.uint8, device="cuda:0")
    dst = torch.empty_like(src)
    dst.copy_(src)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    gbs = 2 * nbytes * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del src, dst
    torch.cuda.empty_cache()
    return round(gbs, 1)


def host_info() -> dict:
    import torch
    model = ""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    props = torch.cuda.get_device_properties(0)
    return {"nproc": os.cpu_count(), "cpu": model, "gpu": torch.cuda.get_device_name(0),
            "gpu_arch": getattr(props, "gcnArchName", ""), "gpu_cus": props.multi_processor_count,
            "gpu_mem_gib": round(props.total_memory / 2 ** 30, 1)}


def algorithmic_bytes(stats: dict) -> int:
    emit = stats["arcs_expanded"] - stats["eps_arcs_expanded"]
    return (stats["arcs_expanded"] * BYTES_ARC + emit * BYTES_LOGLIKE +
            stats["tokens"] * BYTES_TOKEN + stats["raw_links"] * BYTES_LINK)


def cpu_baseline(g, L, cfg, workload, min_seconds: float = 10.0) -> dict:
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
            "sample": f"{workload} full utterance ({L.shape[0]} frames) x {runs} runs, one thread, "
                      f"{dt:.1f} s"}


def cpu_prefix_baseline(g, L, cfg, workload, frames: int) -> dict:
    """The oracle (one thread) on the first `frames` frames of a workload
    whose whole utterance takes the oracle far too long (the wide-beam graph:
    seconds per frame).  The early frames hold fewer tokens than later ones,
    so the arcs-expanded rate is the comparable figure."""
    import oracle
    oracle.build()
    t0 = time.perf_counter()
    o = oracle.decode(g, L[:frames], cfg["beam"], cfg["max_active"], cfg["lattice_beam"])
    dt = time.perf_counter() - t0
    return {"value": round(frames / dt, 3), "unit": "frames/s", "cores": 1, "kind": "oracle",
            "arcs_expanded_per_s": round(o.stats["arcs_expanded"] / dt, 1),
            "sample": f"{workload} first {frames} frames (whole decode of that prefix, lattice included), "
                      f"one thread, {dt:.1f} s; {o.stats['tokens'] / (frames + 1):.0f} tokens per frame "
                      f"on average in the sample"}


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extra", action="store_true", help="skip other_workloads")
    ap.add_argument("--copy-kernel-bytes", type=int, default=0)
    ap.add_argument("--workload", default=WORKLOAD,
                    help="workload timed (the headline line is hclg_5m; others are for profiling)")
    ap.add_argument("--mode", default="auto", help="execution mode of the timed decodes (for profiling)")
    ap.add_argument("--frames", type=int, default=0,
                    help="decode only the first N frames of --workload (for profiling runs)")
    ap.add_argument("--phases", action="store_true",
                    help="only print the step profile of the one-workgroup forward pass on --workload")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this decoder runs on one GPU; --gpus {args.gpus} is not supported "
              "(utterances would shard across GPUs with no exchange between them)", file=sys.stderr)
        return 2

    if args.copy_kernel_bytes:
        return copy_kernel(args.copy_kernel_bytes)
    if args.phases:
        from paper_1804_03243_amd import wfstdec
        print(json.dumps(phase_profile(wfstdec, args.workload)), flush=True)
        return 0

    import numpy as np
    import torch

    import synth
    from paper_1804_03243_amd import wfstdec

    workload = args.workload
    cfg = synth.workload(workload)
    g = synth.make_graph(cfg)
    L = synth.make_loglikes(cfg)
    if args.frames:
        L = np.ascontiguousarray(L[:args.frames])
    dev = torch.device("cuda:0")
    graph = wfstdec.Graph(g, cfg["P"], "cuda:0")
    x = torch.from_numpy(L).to(dev)
    beam, ma, lb = cfg["beam"], cfg["max_active"], cfg["lattice_beam"]

    for _ in range(max(1, args.warmup)):
        r = wfstdec.decode(graph, x, beam, ma, lb, timing=True, mode=args.mode)
    torch.cuda.synchronize()
    fwd_ms, lat_ms = [], []
    t0 = time.perf_counter()
    for _ in range(args.steps):
        r = wfstdec.decode(graph, x, beam, ma, lb, timing=True, mode=args.mode)
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
    traffic = (TRAFFIC["bytes_per_launch"]
               if TRAFFIC and workload == WORKLOAD and TRAFFIC["sources_sha256"] == sources_sha256()
               else None)
    chip = args.mode.startswith("chip") or (args.mode == "auto" and (
        cfg["max_active"] == 0 or cfg["max_active"] >= wfstdec.WD_CHIP_WIDE_MAX_ACTIVE))
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
        "config": {"workload": workload, "states": cfg["S"], "arcs": cfg["A"], "frames": T,
                   "pdfs": cfg["P"], "beam": beam, "max_active": ma, "lattice_beam": lb,
                   "utterances_per_step": 1, "mode": args.mode},
        "arcs_expanded_per_s": round(st["arcs_expanded"] * args.steps / wall, 1),
        "rtf": round((wall / args.steps) / (T / FRAME_RATE), 7),
        "tokens_per_frame": round(st["tokens"] / (T + 1), 1),
        "kernel_ms": {"forward": round(fwd, 3), "lattice": round(float(np.mean(lat_ms)), 3)},
        "roofline": {"bound": "hbm", "kernel": "chip-wide forward kernels" if chip else "k_forward", "achieved": round(achieved, 3),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 6),
                     "traffic": traffic, "algorithmic_bytes_per_launch": int(bytes_launch)},
    }
    if not args.no_extra and workload == WORKLOAD:
        streamed = [stream_hclg(wfstdec, graph, x, cfg, chunk) for chunk in (32, 8)]
        streamed.append(determinize_hclg(wfstdec, r, g, T))
        streamed.append(batch(wfstdec, graph, 64, cpu=not args.no_cpu_baseline))
        streamed.append(batch(wfstdec, graph, 256, steps=5, cpu=False))
        del graph, x
        torch.cuda.empty_cache()
        out["other_workloads"] = streamed + [wide_chip(wfstdec, mode=m, cpu=m == "chip" and not args.no_cpu_baseline)
                                             for m in ("chip", "chip_noprune", "chip_dyn")]
        out["other_workloads"] += [single(wfstdec, w, cpu=not args.no_cpu_baseline)
                                   for w in ("tiny_10k", "lm_30m")]
    if not args.no_extra:
        out["roofline"]["copy_ceiling_gbs"] = copy_ceiling()
    out["host"] = host_info()
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(g, L, cfg, workload)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
