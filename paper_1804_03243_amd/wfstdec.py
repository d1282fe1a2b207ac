"""ctypes binding of libwfstdec.so (include/wfstdec.h).

The functions named wd_* mirror the C ABI one to one and only marshal
arguments.  Graph, decode(), decode_batch(), Stream and determinize() add the
bookkeeping a Python caller needs: device buffers come from torch (torch is
used for device memory and streams only), and a decode that reports
WD_ECAPACITY is run again with the capacities it reported as needed (growing
at least fourfold per attempt).  A Graph keeps one workspace for its decodes,
so decodes on one Graph object must not run from several threads at once.
Every step of the decoder runs in the library's HIP kernels; if the library
is missing this module raises.
"""
from __future__ import annotations

import ctypes
import os
from types import SimpleNamespace

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libwfstdec.so")

WD_OK, WD_EINVAL, WD_ECYCLE, WD_ENOPATH, WD_ECAPACITY, WD_EDEVICE = range(6)
WD_FLAG_DEBUG = 1
WD_FLAG_TIMING = 2
WD_FLAG_ONE_WORKGROUP = 4
WD_FLAG_CHIP_WIDE = 8
WD_CHIP_WIDE_MAX_ACTIVE = 32768
WD_FLAG_DYNAMIC_LB = 16
WD_FLAG_NO_INCREMENTAL_PRUNE = 32
WD_FLAG_PHASES = 64
WD_FLAG_EPS_LEVELS = 128
WD_PHASE_STAMPS = 10
WD_PHASE_SLOTS = 12
WD_LATTICE_PHASE_STAMPS = 8
_MODE_FLAGS = {"auto": 0, "workgroup": WD_FLAG_ONE_WORKGROUP, "chip": WD_FLAG_CHIP_WIDE,
               "chip_dyn": WD_FLAG_CHIP_WIDE | WD_FLAG_DYNAMIC_LB,
               "chip_noprune": WD_FLAG_CHIP_WIDE | WD_FLAG_NO_INCREMENTAL_PRUNE,
               "workgroup_levels": WD_FLAG_ONE_WORKGROUP | WD_FLAG_EPS_LEVELS}
STATUS_NAMES = {0: "WD_OK", 1: "WD_EINVAL", 2: "WD_ECYCLE", 3: "WD_ENOPATH", 4: "WD_ECAPACITY",
                5: "WD_EDEVICE"}

LINK_DTYPE = np.dtype([("t", "<i4"), ("arc_id", "<u4"), ("src_state", "<i4"), ("dst_state", "<i4"),
                       ("ilabel", "<i4"), ("olabel", "<i4"), ("graph_cost", "<f4"),
                       ("ac_cost", "<f4"), ("fwd_cost", "<f4"), ("extra", "<f4"),
                       ("posterior", "<f8")], align=True)
CLAT_ARC_DTYPE = np.dtype([("src", "<i4"), ("dst", "<i4"), ("word", "<i4"), ("align_len", "<i4"),
                           ("graph_cost", "<f8"), ("ac_cost", "<f8"), ("align_off", "<i8")], align=True)
CLAT_FINAL_DTYPE = np.dtype([("state", "<i4"), ("align_len", "<i4"), ("graph_cost", "<f8"),
                             ("ac_cost", "<f8"), ("align_off", "<i8")], align=True)
NODE_DTYPE = np.dtype([("t", "<i4"), ("state", "<i4"), ("cost", "<f4"), ("extra", "<f4")], align=True)
TOKEN_DTYPE = np.dtype([("t", "<i4"), ("state", "<i4"), ("cost", "<f4"), ("pred_arc", "<u4")],
                       align=True)


class WdError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


class wd_graph_desc(ctypes.Structure):
    _fields_ = [("num_states", ctypes.c_int32), ("num_arcs", ctypes.c_int64),
                ("start_state", ctypes.c_int32), ("row_ptr", ctypes.c_void_p),
                ("dst", ctypes.c_void_p), ("ilabel", ctypes.c_void_p), ("olabel", ctypes.c_void_p),
                ("weight", ctypes.c_void_p), ("final_weight", ctypes.c_void_p),
                ("num_pdfs", ctypes.c_int32)]


class wd_params(ctypes.Structure):
    _fields_ = [("beam", ctypes.c_float), ("max_active", ctypes.c_int32),
                ("lattice_beam", ctypes.c_float), ("flags", ctypes.c_uint32)]


class wd_caps(ctypes.Structure):
    _fields_ = [("frame_tokens", ctypes.c_int64), ("frame_arcs", ctypes.c_int64),
                ("nodes", ctypes.c_int64), ("links", ctypes.c_int64), ("kept_links", ctypes.c_int64),
                ("window_links", ctypes.c_int64)]


class wd_stats(ctypes.Structure):
    _fields_ = [("frames", ctypes.c_int32), ("final_reached", ctypes.c_int32),
                ("arcs_expanded", ctypes.c_int64), ("tokens", ctypes.c_int64),
                ("max_tokens", ctypes.c_int64), ("raw_links", ctypes.c_int64),
                ("kept_links", ctypes.c_int64), ("nodes", ctypes.c_int64),
                ("eps_arcs_expanded", ctypes.c_int64), ("forward_ms", ctypes.c_float),
                ("lattice_ms", ctypes.c_float), ("needed", wd_caps)]


EXPORTS = ["wd_graph_bytes", "wd_graph_load", "wd_graph_free", "wd_graph_eps_levels", "wd_graph_eps_paths",
           "wd_workspace_bytes", "wd_decode", "wd_decode_batch", "wd_decode_noalloc", "wd_stream_begin",
           "wd_stream_advance", "wd_stream_end", "wd_stream_free", "wd_lattice_determinize",
           "wd_clat_states", "wd_clat_arcs", "wd_clat_finals", "wd_clat_alignment", "wd_clat_free",
           "wd_result_status",
           "wd_result_cost", "wd_result_words", "wd_result_lattice", "wd_result_nodes",
           "wd_result_tokens", "wd_result_raw_lattice", "wd_result_cutoffs", "wd_result_phases",
           "wd_result_lattice_phases",
           "wd_result_stats",
           "wd_result_free", "wd_last_error"]

_LIB = None


def lib():
    """The loaded library; raises if it has not been built."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with "
                              "`python -c 'import __graft_entry__ as g; g.build()'`")
        L = ctypes.CDLL(LIB_PATH)
        P, VP = ctypes.POINTER, ctypes.c_void_p
        sig = {
            "wd_graph_bytes": ([P(wd_graph_desc), P(ctypes.c_size_t)], ctypes.c_int),
            "wd_graph_load": ([P(wd_graph_desc), VP, ctypes.c_size_t, VP, P(VP)], ctypes.c_int),
            "wd_graph_free": ([VP], None),
            "wd_graph_eps_levels": ([VP], ctypes.c_int32),
            "wd_graph_eps_paths": ([VP], ctypes.c_int64),
            "wd_workspace_bytes": ([VP, ctypes.c_int32, ctypes.c_int32, P(wd_params), P(wd_caps),
                                    P(ctypes.c_size_t), P(wd_caps)], ctypes.c_int),
            "wd_decode": ([VP, VP, ctypes.c_int32, P(wd_params), P(wd_caps), VP, ctypes.c_size_t, VP,
                           P(VP)], ctypes.c_int),
            "wd_decode_noalloc": ([VP, VP, ctypes.c_int32, P(wd_params), P(wd_caps), VP, P(ctypes.c_float),
                                   VP, ctypes.c_int32, P(ctypes.c_int32), VP, ctypes.c_int64, VP, ctypes.c_int64,
                                   P(wd_stats)], ctypes.c_int),
            "wd_decode_batch": ([VP, ctypes.c_int32, P(VP), P(ctypes.c_int32), P(wd_params),
                                 P(wd_caps), VP, ctypes.c_size_t, VP, P(VP)], ctypes.c_int),
            "wd_stream_begin": ([VP, ctypes.c_int32, P(VP), ctypes.c_int32, P(wd_params), P(wd_caps),
                                 VP, ctypes.c_size_t, VP, P(VP)], ctypes.c_int),
            "wd_stream_advance": ([VP, P(ctypes.c_int32)], ctypes.c_int),
            "wd_stream_end": ([VP, P(VP)], ctypes.c_int),
            "wd_stream_free": ([VP], None),
            "wd_lattice_determinize": ([VP, ctypes.c_int64, VP, ctypes.c_int64, ctypes.c_int32, VP,
                                        ctypes.c_double, ctypes.c_int64, P(VP)], ctypes.c_int),
            "wd_clat_states": ([VP], ctypes.c_int32),
            "wd_clat_arcs": ([VP, P(VP)], ctypes.c_int64),
            "wd_clat_finals": ([VP, P(VP)], ctypes.c_int64),
            "wd_clat_alignment": ([VP, P(VP)], ctypes.c_int64),
            "wd_clat_free": ([VP], None),
            "wd_result_status": ([VP], ctypes.c_int),
            "wd_result_cost": ([VP], ctypes.c_float),
            "wd_result_words": ([VP, P(VP)], ctypes.c_int32),
            "wd_result_lattice": ([VP, P(VP)], ctypes.c_int64),
            "wd_result_nodes": ([VP, P(VP)], ctypes.c_int64),
            "wd_result_tokens": ([VP, P(VP)], ctypes.c_int64),
            "wd_result_raw_lattice": ([VP, P(VP)], ctypes.c_int64),
            "wd_result_cutoffs": ([VP, P(VP), P(VP), P(VP)], ctypes.c_int32),
            "wd_result_phases": ([VP, P(VP), P(ctypes.c_double)], ctypes.c_int32),
            "wd_result_lattice_phases": ([VP, P(VP)], ctypes.c_int32),
            "wd_result_stats": ([VP, P(wd_stats)], None),
            "wd_result_free": ([VP], None),
            "wd_last_error": ([], ctypes.c_char_p),
        }
        for name, (args, res) in sig.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = res
        _LIB = L
    return _LIB


def _check(st: int):
    if st != WD_OK:
        raise WdError(st, lib().wd_last_error().decode())


# ------------------------------------------------------------ one-to-one ABI

def wd_graph_bytes(desc: wd_graph_desc) -> int:
    n = ctypes.c_size_t()
    _check(lib().wd_graph_bytes(ctypes.byref(desc), ctypes.byref(n)))
    return n.value


def wd_graph_load(desc: wd_graph_desc, dev_buf: int, dev_bytes: int, stream: int) -> int:
    h = ctypes.c_void_p()
    _check(lib().wd_graph_load(ctypes.byref(desc), dev_buf, dev_bytes, stream, ctypes.byref(h)))
    return h.value


def wd_graph_free(handle: int) -> None:
    lib().wd_graph_free(handle)


def wd_graph_eps_levels(handle: int) -> int:
    return lib().wd_graph_eps_levels(handle)


def wd_graph_eps_paths(handle: int) -> int:
    return lib().wd_graph_eps_paths(handle)


def wd_workspace_bytes(handle: int, lanes: int, max_T: int, params: wd_params,
                       caps: wd_caps | None = None) -> tuple[int, wd_caps]:
    n = ctypes.c_size_t()
    out = wd_caps()
    _check(lib().wd_workspace_bytes(handle, lanes, max_T, ctypes.byref(params),
                                    ctypes.byref(caps) if caps is not None else None,
                                    ctypes.byref(n), ctypes.byref(out)))
    return n.value, out


def wd_decode(handle: int, loglikes_ptr: int, T: int, params: wd_params, caps: wd_caps | None,
              ws: int, ws_bytes: int, stream: int) -> tuple[int, int]:
    """Returns (status, result handle or 0)."""
    r = ctypes.c_void_p()
    st = lib().wd_decode(handle, loglikes_ptr, T, ctypes.byref(params),
                         ctypes.byref(caps) if caps is not None else None, ws, ws_bytes, stream,
                         ctypes.byref(r))
    return st, r.value or 0


def wd_decode_batch(handle: int, loglikes_ptrs: list[int], Ts: list[int], params: wd_params,
                    caps: wd_caps | None, ws: int, ws_bytes: int, stream: int) -> tuple[int, list[int]]:
    B = len(Ts)
    ptrs = (ctypes.c_void_p * B)(*loglikes_ptrs)
    ts = (ctypes.c_int32 * B)(*Ts)
    outs = (ctypes.c_void_p * B)()
    st = lib().wd_decode_batch(handle, B, ptrs, ts, ctypes.byref(params),
                               ctypes.byref(caps) if caps is not None else None, ws, ws_bytes, stream,
                               outs)
    return st, [o or 0 for o in outs]


WD_NOALLOC_SCRATCH_BYTES = 256 << 20


def wd_decode_noalloc(handle: int, loglikes_ptr: int, T: int, params: wd_params, caps: wd_caps | None,
                      stream: int, words: np.ndarray, links: np.ndarray, nodes: np.ndarray):
    """The no-allocation decode: results into the given host arrays (int32,
    LINK_DTYPE, NODE_DTYPE; their sizes are the capacities).  Returns
    (status, cost, n_words, stats dict, needed dict); on WD_OK the first
    n_words words, stats['kept_links'] links and stats['nodes'] nodes are
    filled."""
    for a, dt, what in ((words, np.dtype("<i4"), "words"), (links, LINK_DTYPE, "links"), (nodes, NODE_DTYPE, "nodes")):
        if a.dtype != dt or a.ndim != 1 or not a.flags.c_contiguous:
            raise ValueError(f"{what} must be a contiguous 1-d array of {dt}")
    cost, nw, st_ = ctypes.c_float(), ctypes.c_int32(), wd_stats()
    st = lib().wd_decode_noalloc(handle, loglikes_ptr, T, ctypes.byref(params),
                                 ctypes.byref(caps) if caps is not None else None, stream, ctypes.byref(cost),
                                 words.ctypes.data, words.size, ctypes.byref(nw), links.ctypes.data, links.size,
                                 nodes.ctypes.data, nodes.size, ctypes.byref(st_))
    stats = {f: getattr(st_, f) for f, _ in wd_stats._fields_ if f != "needed"}
    needed = {f: getattr(st_.needed, f) for f, _ in wd_caps._fields_}
    return st, np.float32(cost.value), nw.value, stats, needed


def wd_stream_begin(handle: int, frame_ptrs: list[int], max_T: int, params: wd_params,
                    caps: wd_caps | None, ws: int, ws_bytes: int, stream: int) -> int:
    """Returns the stream handle; raises WdError on a non-OK status."""
    B = len(frame_ptrs)
    ptrs = (ctypes.c_void_p * B)(*frame_ptrs)
    h = ctypes.c_void_p()
    _check(lib().wd_stream_begin(handle, B, ptrs, max_T, ctypes.byref(params),
                                 ctypes.byref(caps) if caps is not None else None, ws, ws_bytes, stream,
                                 ctypes.byref(h)))
    return h.value


def wd_stream_advance(sh: int, n_frames: list[int]) -> None:
    ns = (ctypes.c_int32 * len(n_frames))(*n_frames)
    _check(lib().wd_stream_advance(sh, ns))


def wd_stream_end(sh: int, B: int) -> tuple[int, list[int]]:
    """Returns (status, result handles or 0); frees the stream."""
    outs = (ctypes.c_void_p * B)()
    st = lib().wd_stream_end(sh, outs)
    return st, [o or 0 for o in outs]


def wd_stream_free(sh: int) -> None:
    lib().wd_stream_free(sh)


def wd_lattice_determinize(links, nodes, start_state: int, node_final=None, beam: float = float("inf"),
                           max_states: int = 0) -> SimpleNamespace:
    """Host lattice determinisation of (links, nodes) arrays; returns
    states, arcs (CLAT_ARC_DTYPE), finals (CLAT_FINAL_DTYPE) and the
    alignment label pool."""
    L = lib()
    la = np.zeros(len(links), LINK_DTYPE)
    for f in LINK_DTYPE.names:
        la[f] = links[f]
    na = np.zeros(len(nodes), NODE_DTYPE)
    for f in NODE_DTYPE.names:
        na[f] = nodes[f]
    nf = None if node_final is None else np.ascontiguousarray(node_final, dtype=np.float32)
    if nf is not None and nf.size != len(nodes):
        raise ValueError("node_final needs one value per node")
    h = ctypes.c_void_p()
    _check(L.wd_lattice_determinize(la.ctypes.data if la.size else None, la.size,
                                    na.ctypes.data if na.size else None, na.size, int(start_state),
                                    None if nf is None else nf.ctypes.data, float(beam), int(max_states),
                                    ctypes.byref(h)))
    try:
        out = SimpleNamespace(states=L.wd_clat_states(h))
        for name, acc, dt in (("arcs", L.wd_clat_arcs, CLAT_ARC_DTYPE),
                              ("finals", L.wd_clat_finals, CLAT_FINAL_DTYPE),
                              ("align", L.wd_clat_alignment, np.dtype("<i4"))):
            vp = ctypes.c_void_p()
            n = acc(h, ctypes.byref(vp))
            setattr(out, name, _copy(vp.value, n, dt))
    finally:
        L.wd_clat_free(h)
    return out


def determinize(result, start_state: int = 0, final_weight=None, beam: float = float("inf"),
                max_states: int = 0) -> SimpleNamespace:
    """The compact lattice of a decode result (this library's or the
    oracle's): the last frame's nodes are final with the graph's final
    weights when the decode used them (stats final_reached), else cost 0."""
    nodes = result.nodes
    T = int(result.stats["frames"])
    nf = np.full(len(nodes), np.inf, np.float32)
    last = nodes["t"] == T
    if final_weight is not None and result.stats["final_reached"]:
        nf[last] = np.asarray(final_weight, np.float32)[nodes["state"][last]]
    else:
        nf[last] = 0.0
    return wd_lattice_determinize(result.links, nodes, start_state, nf, beam, max_states)


def _copy(ptr, n, dtype):
    """n records of `dtype` at host address ptr, copied into a new array."""
    out = np.empty(max(int(n), 0), dtype=dtype)
    if out.size and ptr:
        ctypes.memmove(out.ctypes.data, ptr, out.nbytes)
    return out


class _ResultOwner:
    """Frees a result handle once no array viewing its memory is left."""
    __slots__ = ("r",)

    def __init__(self, r: int):
        self.r = r

    def __del__(self):
        r, self.r = self.r, None
        if r:
            try:
                lib().wd_result_free(r)
            except Exception:  # (interpreter shutdown)
                pass


def _view(ptr, n, dtype, owner: _ResultOwner):
    """n records of `dtype` at host address ptr, viewed in place; the view
    keeps `owner` (and with it the result handle) alive."""
    n = max(int(n), 0)
    if n == 0 or not ptr:
        return np.empty(0, dtype=dtype)
    buf = (ctypes.c_char * (n * dtype.itemsize)).from_address(ptr)
    buf._owner = owner
    return np.frombuffer(buf, dtype=dtype, count=n)


def wd_result_read(r: int, debug: bool = True, phases: bool = True,
                   owner: _ResultOwner | None = None) -> SimpleNamespace:
    """Copy everything out of a result handle (wd_result_* accessors).
    `debug` / `phases` false: the outputs only WD_FLAG_DEBUG / WD_FLAG_PHASES
    produce (tokens, raw lattice, cutoffs / step profile) are left empty
    without asking the library for them.  With `owner` (which then owns r)
    the words, lattice and nodes are views of the handle's memory instead of
    copies, and the handle is freed when the last of them is gone."""
    L = lib()
    out = SimpleNamespace()
    out.status = L.wd_result_status(r)
    out.cost = np.float32(L.wd_result_cost(r))
    def get(accessor, dtype, view=False):
        vp = ctypes.c_void_p()
        n = accessor(r, ctypes.byref(vp))   # sets vp; read it only afterwards
        return _view(vp.value, n, dtype, owner) if view and owner is not None else _copy(vp.value, n, dtype)

    out.words = get(L.wd_result_words, np.dtype("<i4"), True)
    out.links = get(L.wd_result_lattice, LINK_DTYPE, True)
    out.nodes = get(L.wd_result_nodes, NODE_DTYPE, True)
    f4 = np.dtype("<f4")
    if debug:
        out.tokens = get(L.wd_result_tokens, TOKEN_DTYPE)
        out.raw_links = get(L.wd_result_raw_lattice, LINK_DTYPE)
        b, cb, c = ctypes.c_void_p(), ctypes.c_void_p(), ctypes.c_void_p()
        n = L.wd_result_cutoffs(r, ctypes.byref(b), ctypes.byref(cb), ctypes.byref(c))
        out.best, out.cutoff_beam, out.cutoff = (_copy(b.value, n, f4), _copy(cb.value, n, f4),
                                                 _copy(c.value, n, f4))
    else:
        out.tokens = np.zeros(0, TOKEN_DTYPE)
        out.raw_links = np.zeros(0, LINK_DTYPE)
        out.best, out.cutoff_beam, out.cutoff = (np.zeros(0, f4), np.zeros(0, f4), np.zeros(0, f4))
    if phases:
        vp, hz = ctypes.c_void_p(), ctypes.c_double()
        n = L.wd_result_phases(r, ctypes.byref(vp), ctypes.byref(hz))
        out.phases = _copy(vp.value, n * WD_PHASE_SLOTS, np.dtype("<u8")).reshape(n, WD_PHASE_SLOTS)
        out.phase_tick_hz = hz.value
        lp = ctypes.c_void_p()
        n = L.wd_result_lattice_phases(r, ctypes.byref(lp))
        out.lattice_phases = _copy(lp.value, n, np.dtype("<u8"))
    else:
        out.phases = np.zeros((0, WD_PHASE_SLOTS), np.dtype("<u8"))
        out.phase_tick_hz = 0.0
        out.lattice_phases = np.zeros(0, np.dtype("<u8"))
    st = wd_stats()
    L.wd_result_stats(r, ctypes.byref(st))
    out.stats = {f: getattr(st, f) for f, _ in wd_stats._fields_ if f != "needed"}
    out.needed = {f: getattr(st.needed, f) for f, _ in wd_caps._fields_}
    return out


def wd_result_free(r: int) -> None:
    lib().wd_result_free(r)


# ---------------------------------------------------------------- helpers

def _torch():
    import torch
    if not torch.cuda.is_available():
        raise RuntimeError("wfstdec needs a GPU (torch.cuda.is_available() is False)")
    return torch


def _stream(torch):
    return torch.cuda.current_stream().cuda_stream


class Graph:
    """A decoding graph resident in GPU memory (buffer owned by a torch tensor)."""

    def __init__(self, g: dict, num_pdfs: int, device: str = "cuda:0"):
        torch = _torch()
        self._arrs = dict(row_ptr=np.ascontiguousarray(g["row_ptr"], dtype=np.uint32),
                          dst=np.ascontiguousarray(g["dst"], dtype=np.uint32),
                          ilabel=np.ascontiguousarray(g["ilabel"], dtype=np.int32),
                          olabel=np.ascontiguousarray(g["olabel"], dtype=np.int32),
                          weight=np.ascontiguousarray(g["weight"], dtype=np.float32))
        fw = g.get("final_weight")
        self._fw = None if fw is None else np.ascontiguousarray(fw, dtype=np.float32)
        a = self._arrs
        self.desc = wd_graph_desc(int(g["num_states"]), int(a["dst"].size), int(g.get("start_state", 0)),
                                  a["row_ptr"].ctypes.data, a["dst"].ctypes.data,
                                  a["ilabel"].ctypes.data, a["olabel"].ctypes.data,
                                  a["weight"].ctypes.data,
                                  None if self._fw is None else self._fw.ctypes.data, int(num_pdfs))
        self.num_pdfs = int(num_pdfs)
        self.device = torch.device(device)
        with torch.cuda.device(self.device):
            nbytes = wd_graph_bytes(self.desc)
            self.buf = torch.empty(nbytes + 256, dtype=torch.uint8, device=self.device)
            base = (self.buf.data_ptr() + 255) // 256 * 256
            self.handle = wd_graph_load(self.desc, base, nbytes, _stream(torch))
        self.nbytes = nbytes
        self.eps_levels = wd_graph_eps_levels(self.handle)
        self.eps_paths = wd_graph_eps_paths(self.handle)
        self._ws = None
        self._caps = {}

    def __del__(self):
        h = getattr(self, "handle", None)
        if h:
            try:
                wd_graph_free(h)
            except Exception:
                pass
            self.handle = None

    def degrees(self):
        """Per-state (emitting, epsilon) out-degrees of the graph (host numpy
        arrays, from the CSR this graph was loaded from)."""
        rp = self._arrs["row_ptr"].astype(np.int64)
        S = rp.size - 1
        src = np.repeat(np.arange(S), np.diff(rp))
        eps = self._arrs["ilabel"] == 0
        return np.bincount(src[~eps], minlength=S), np.bincount(src[eps], minlength=S)

    def workspace(self, lanes: int, max_T: int, params: wd_params, caps: wd_caps | None):
        """(pointer, bytes) of a workspace large enough; reuses one buffer."""
        torch = _torch()
        nbytes, used = wd_workspace_bytes(self.handle, lanes, max_T, params, caps)
        if self._ws is None or self._ws.numel() < nbytes + 256:
            self._ws = None
            self._ws = torch.empty(nbytes + 256, dtype=torch.uint8, device=self.device)
        base = (self._ws.data_ptr() + 255) // 256 * 256
        return base, nbytes, used


def _params(beam, max_active, lattice_beam, debug, timing=False, mode="auto", flags=0):
    if mode not in _MODE_FLAGS:
        raise ValueError(f"mode must be one of {sorted(_MODE_FLAGS)}")
    return wd_params(float(beam), int(max_active), float(lattice_beam),
                     (WD_FLAG_DEBUG if debug else 0) | (WD_FLAG_TIMING if timing else 0) |
                     _MODE_FLAGS[mode] | int(flags))


def _grow(caps: wd_caps, needed: dict) -> wd_caps:
    """Capacities for the next attempt: at least what was needed, and a fast
    geometric step (an attempt only reveals the first capacity it outgrew)."""
    c = wd_caps(*(getattr(caps, f) for f, _ in wd_caps._fields_))
    for f, _ in wd_caps._fields_:
        need = needed[f]
        if need > getattr(c, f):
            setattr(c, f, int(max(need, 4 * getattr(c, f))))
    return c


def decode_batch(graph: Graph, loglikes: list, beam: float, max_active: int, lattice_beam: float,
                 debug: bool = False, caps: wd_caps | None = None, max_retries: int = 12,
                 timing: bool = False, mode: str = "auto", flags: int = 0):
    """Decode utterances (device float32 tensors, T_i x P) concurrently.
    `mode`: "workgroup" (one workgroup per utterance), "chip" (chip-wide
    kernels per frame), "chip_dyn" (chip-wide with dynamic load balancing of
    the emitting arcs), "chip_noprune" (chip-wide without incremental lattice
    pruning), "workgroup_levels" (one workgroup, epsilon closure level by
    level instead of by the graph's epsilon paths) or "auto" (the library's
    choice).  `flags`: further WD_FLAG_*
    bits (e.g. WD_FLAG_PHASES).  Returns one result namespace per utterance."""
    torch = _torch()
    for x in loglikes:
        if x.dtype != torch.float32 or not x.is_contiguous() or x.device != graph.device:
            raise ValueError("log-likelihoods must be contiguous float32 tensors on the graph's device")
        if x.dim() != 2 or x.shape[1] != graph.num_pdfs:
            raise ValueError(f"log-likelihoods must be T x {graph.num_pdfs}")
    p = _params(beam, max_active, lattice_beam, debug, timing, mode, flags)
    Ts = [int(x.shape[0]) for x in loglikes]
    key = (len(Ts), max(Ts), float(beam), int(max_active), float(lattice_beam), bool(debug), int(flags))
    if caps is None:
        caps = graph._caps.get(key)
    for attempt in range(max_retries + 1):
        with torch.cuda.device(graph.device):
            ws, nbytes, used = graph.workspace(len(Ts), max(Ts), p, caps)
            st, res = wd_decode_batch(graph.handle, [x.data_ptr() for x in loglikes], Ts, p, used, ws,
                                      nbytes, _stream(torch))
        outs = []
        err = lib().wd_last_error().decode() if st != WD_OK else ""
        want_phases = bool(p.flags & WD_FLAG_PHASES)
        for r in res:
            # views of the handle's memory, freed with the last of them
            outs.append(wd_result_read(r, debug, want_phases, _ResultOwner(r)) if r else None)
        if st == WD_ECAPACITY and attempt < max_retries:
            need = {f: max(o.needed[f] for o in outs if o is not None) for f, _ in wd_caps._fields_}
            caps = _grow(used, need)
            continue
        if st != WD_OK:
            raise WdError(st, err)
        graph._caps[key] = used
        return outs
    raise WdError(WD_ECAPACITY, "capacity retries exhausted")


def decode(graph: Graph, loglikes, beam: float, max_active: int, lattice_beam: float,
           debug: bool = False, caps: wd_caps | None = None, timing: bool = False,
           mode: str = "auto", flags: int = 0):
    """Decode one utterance (device float32 tensor, T x P)."""
    return decode_batch(graph, [loglikes], beam, max_active, lattice_beam, debug, caps,
                        timing=timing, mode=mode, flags=flags)[0]


class Stream:
    """Streaming decode of B utterances whose log-likelihoods arrive in chunks
    (wd_stream_begin / wd_stream_advance / wd_stream_end).  `frames[i]` is
    utterance i's frame store (max_T x P device tensor); `push` copies chunks
    into it on the current stream and decodes them.  `end` returns the same
    results as decode_batch of the complete utterances; if the workspace
    turns out too small it decodes them again from the frame stores with the
    capacities the stream reported (decode_batch's retry)."""

    def __init__(self, graph: Graph, B: int, max_T: int, beam: float, max_active: int,
                 lattice_beam: float, debug: bool = False, timing: bool = False, mode: str = "auto",
                 caps: wd_caps | None = None):
        torch = _torch()
        self.graph, self.B, self.max_T = graph, int(B), int(max_T)
        self.args = (beam, max_active, lattice_beam)
        self.debug, self.timing, self.mode = debug, timing, mode
        self.params = _params(beam, max_active, lattice_beam, debug, timing, mode)
        self.T = [0] * self.B
        with torch.cuda.device(graph.device):
            self.frames = torch.empty((self.B, max(self.max_T, 1), graph.num_pdfs), dtype=torch.float32,
                                      device=graph.device)
            nbytes, used = wd_workspace_bytes(graph.handle, self.B, self.max_T, self.params, caps)
            self._ws = torch.empty(nbytes + 256, dtype=torch.uint8, device=graph.device)
            ws = (self._ws.data_ptr() + 255) // 256 * 256
            # the stream every advance decodes on (wd_stream_begin keeps it)
            self._stream = torch.cuda.current_stream(graph.device)
            self.handle = wd_stream_begin(graph.handle, [self.frames[i].data_ptr() for i in range(self.B)],
                                          self.max_T, self.params, used, ws, nbytes,
                                          self._stream.cuda_stream)
        self.caps = used

    def push(self, chunks: list) -> None:
        """chunks[i]: None or a device float32 tensor (n_i x P) of utterance
        i's next frames, produced on the caller's current stream.  The copies
        into the frame stores run on the decoding stream (the one current at
        construction) after it has waited for the current stream, so the
        decode never reads a row before its chunk is complete."""
        torch = _torch()
        counts = [0] * self.B
        for i, x in enumerate(chunks):
            if x is None:
                continue
            if x.dim() != 2 or x.shape[1] != self.graph.num_pdfs or x.dtype != torch.float32:
                raise ValueError(f"chunk {i} must be n x {self.graph.num_pdfs} float32")
            if self.T[i] + int(x.shape[0]) > self.max_T:
                raise ValueError(f"utterance {i} would pass max_T = {self.max_T}")
        with torch.cuda.device(self.graph.device):
            cur = torch.cuda.current_stream(self.graph.device)
            if cur != self._stream:
                self._stream.wait_stream(cur)
            with torch.cuda.stream(self._stream):
                for i, x in enumerate(chunks):
                    if x is None:
                        continue
                    n = int(x.shape[0])
                    if n:
                        self.frames[i, self.T[i]:self.T[i] + n].copy_(x)
                        if cur != self._stream:
                            x.record_stream(self._stream)  # x may be freed on `cur` meanwhile
                    counts[i] = n
            wd_stream_advance(self.handle, counts)
        for i, n in enumerate(counts):
            self.T[i] += n

    def end(self) -> list:
        torch = _torch()
        with torch.cuda.device(self.graph.device):
            st, res = wd_stream_end(self.handle, self.B)
        self.handle = None
        outs, err = [], lib().wd_last_error().decode() if st != WD_OK else ""
        for r in res:
            outs.append(wd_result_read(r, self.debug, False) if r else None)
            if r:
                wd_result_free(r)
        if st == WD_ECAPACITY:
            need = {f: max(o.needed[f] for o in outs if o is not None) for f, _ in wd_caps._fields_}
            xs = [self.frames[i, :self.T[i]] for i in range(self.B)]
            return decode_batch(self.graph, xs, *self.args, debug=self.debug, caps=_grow(self.caps, need),
                                timing=self.timing, mode=self.mode)
        if st != WD_OK:
            raise WdError(st, err)
        return outs

    def __del__(self):
        h = getattr(self, "handle", None)
        if h:
            try:
                wd_stream_free(h)
            except Exception:
                pass
            self.handle = None
