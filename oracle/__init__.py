"""CPU oracle of the decoder (test infrastructure).

A plain sequential C implementation (wfst_oracle.c) of frame-synchronous
Viterbi token passing with exact lattice generation, lattice pruning and fp64
arc posteriors, wrapped with ctypes.  Only the tests, the smoke check and the
CPU-baseline leg of the benchmark may use this package; the GPU library neither
imports it nor shares any code with it.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from types import SimpleNamespace

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libwfst_oracle.so")
SRC_PATH = os.path.join(_HERE, "wfst_oracle.c")
CFLAGS = ["-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
          "-Wall", "-Wextra"]

OK, EINVAL, ECYCLE, ENOPATH, ENOMEM = 0, 1, 2, 3, 6

LINK_DTYPE = np.dtype([("t", "<i4"), ("arc_id", "<u4"), ("src_state", "<i4"), ("dst_state", "<i4"),
                       ("ilabel", "<i4"), ("olabel", "<i4"), ("graph_cost", "<f4"),
                       ("ac_cost", "<f4"), ("fwd_cost", "<f4"), ("extra", "<f4"),
                       ("posterior", "<f8")], align=True)
NODE_DTYPE = np.dtype([("t", "<i4"), ("state", "<i4"), ("cost", "<f4"), ("extra", "<f4")], align=True)
TOKEN_DTYPE = np.dtype([("t", "<i4"), ("state", "<i4"), ("cost", "<f4"), ("pred_arc", "<u4")],
                       align=True)
assert LINK_DTYPE.itemsize == 48 and NODE_DTYPE.itemsize == 16 and TOKEN_DTYPE.itemsize == 16


class OracleError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"oracle status {code}: {msg}")
        self.code = code


class _Graph(ctypes.Structure):
    _fields_ = [("num_states", ctypes.c_int32), ("num_arcs", ctypes.c_int64),
                ("start_state", ctypes.c_int32), ("row_ptr", ctypes.c_void_p),
                ("dst", ctypes.c_void_p), ("ilabel", ctypes.c_void_p),
                ("olabel", ctypes.c_void_p), ("weight", ctypes.c_void_p),
                ("final_weight", ctypes.c_void_p)]


class _Params(ctypes.Structure):
    _fields_ = [("beam", ctypes.c_float), ("max_active", ctypes.c_int32),
                ("lattice_beam", ctypes.c_float), ("debug", ctypes.c_int32)]


class _Stats(ctypes.Structure):
    _fields_ = [("frames", ctypes.c_int32), ("final_reached", ctypes.c_int32),
                ("arcs_expanded", ctypes.c_int64), ("tokens", ctypes.c_int64),
                ("max_tokens", ctypes.c_int64), ("raw_links", ctypes.c_int64),
                ("kept_links", ctypes.c_int64), ("nodes", ctypes.c_int64),
                ("eps_arcs_expanded", ctypes.c_int64)]


def build(force: bool = False) -> str:
    """Compile the oracle with gcc into oracle/libwfst_oracle.so."""
    if force or not os.path.exists(LIB_PATH) or \
            os.path.getmtime(LIB_PATH) < os.path.getmtime(SRC_PATH):
        tmp = LIB_PATH + ".tmp"
        subprocess.check_call(["gcc", *CFLAGS, "-o", tmp, SRC_PATH, "-lm"])
        os.replace(tmp, LIB_PATH)
    return LIB_PATH


_LIB = None


def _lib():
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            build()
        lib = ctypes.CDLL(LIB_PATH)
        P, VP = ctypes.POINTER, ctypes.c_void_p
        lib.wdo_decode.argtypes = [P(_Graph), VP, ctypes.c_int32, ctypes.c_int32, P(_Params), P(VP)]
        lib.wdo_decode.restype = ctypes.c_int
        lib.wdo_result_cost.argtypes = [VP]
        lib.wdo_result_cost.restype = ctypes.c_float
        for name, rt in [("wdo_result_words", ctypes.c_int32), ("wdo_result_links", ctypes.c_int64),
                         ("wdo_result_nodes", ctypes.c_int64), ("wdo_result_tokens", ctypes.c_int64),
                         ("wdo_result_raw_links", ctypes.c_int64)]:
            f = getattr(lib, name)
            f.argtypes = [VP, P(VP)]
            f.restype = rt
        lib.wdo_result_cutoffs.argtypes = [VP, P(VP), P(VP), P(VP)]
        lib.wdo_result_cutoffs.restype = ctypes.c_int32
        lib.wdo_result_stats.argtypes = [VP, P(_Stats)]
        lib.wdo_result_stats.restype = None
        lib.wdo_result_free.argtypes = [VP]
        lib.wdo_result_free.restype = None
        lib.wdo_error_message.argtypes = [ctypes.c_int]
        lib.wdo_error_message.restype = ctypes.c_char_p
        _LIB = lib
    return _LIB


def _ptr(a):
    return None if a is None else a.ctypes.data


def _copy(ptr, n, dtype):
    if n <= 0 or not ptr:
        return np.zeros(0, dtype=dtype)
    buf = (ctypes.c_char * (int(n) * dtype.itemsize)).from_address(ptr)
    return np.frombuffer(bytes(buf), dtype=dtype).copy()


def decode(graph: dict, loglikes: np.ndarray, beam: float, max_active: int, lattice_beam: float,
           debug: bool = False) -> SimpleNamespace:
    """Decode one utterance on the CPU.  Returns words, cost, links (sorted by
    (t, arc_id)), nodes (sorted by (t, state)), stats and, with debug, the
    per-frame token sets, the raw lattice and the per-frame cutoffs."""
    lib = _lib()
    L = np.ascontiguousarray(loglikes, dtype=np.float32)
    if L.ndim != 2:
        raise ValueError("loglikes must be T x P")
    arrs = dict(row_ptr=np.ascontiguousarray(graph["row_ptr"], dtype=np.uint32),
                dst=np.ascontiguousarray(graph["dst"], dtype=np.uint32),
                ilabel=np.ascontiguousarray(graph["ilabel"], dtype=np.int32),
                olabel=np.ascontiguousarray(graph["olabel"], dtype=np.int32),
                weight=np.ascontiguousarray(graph["weight"], dtype=np.float32))
    fw = graph.get("final_weight")
    fw = None if fw is None else np.ascontiguousarray(fw, dtype=np.float32)
    g = _Graph(int(graph["num_states"]), int(arrs["dst"].size), int(graph.get("start_state", 0)),
               _ptr(arrs["row_ptr"]), _ptr(arrs["dst"]), _ptr(arrs["ilabel"]), _ptr(arrs["olabel"]),
               _ptr(arrs["weight"]), _ptr(fw))
    p = _Params(float(beam), int(max_active), float(lattice_beam), 1 if debug else 0)
    res = ctypes.c_void_p()
    rc = lib.wdo_decode(ctypes.byref(g), _ptr(L) if L.size else None, L.shape[0], L.shape[1],
                        ctypes.byref(p), ctypes.byref(res))
    if rc != OK:
        raise OracleError(rc, lib.wdo_error_message(rc).decode())
    try:
        out = SimpleNamespace()
        out.cost = np.float32(lib.wdo_result_cost(res))
        vp = ctypes.c_void_p()
        n = lib.wdo_result_words(res, ctypes.byref(vp))
        out.words = _copy(vp.value, n, np.dtype("<i4"))
        n = lib.wdo_result_links(res, ctypes.byref(vp))
        out.links = _copy(vp.value, n, LINK_DTYPE)
        n = lib.wdo_result_nodes(res, ctypes.byref(vp))
        out.nodes = _copy(vp.value, n, NODE_DTYPE)
        st = _Stats()
        lib.wdo_result_stats(res, ctypes.byref(st))
        out.stats = {f: getattr(st, f) for f, _ in _Stats._fields_}
        if debug:
            n = lib.wdo_result_tokens(res, ctypes.byref(vp))
            out.tokens = _copy(vp.value, n, TOKEN_DTYPE)
            n = lib.wdo_result_raw_links(res, ctypes.byref(vp))
            out.raw_links = _copy(vp.value, n, LINK_DTYPE)
            b, cb, c = ctypes.c_void_p(), ctypes.c_void_p(), ctypes.c_void_p()
            n = lib.wdo_result_cutoffs(res, ctypes.byref(b), ctypes.byref(cb), ctypes.byref(c))
            f4 = np.dtype("<f4")
            out.best, out.cutoff_beam, out.cutoff = (_copy(b.value, n, f4), _copy(cb.value, n, f4),
                                                     _copy(c.value, n, f4))
        return out
    finally:
        lib.wdo_result_free(res)
