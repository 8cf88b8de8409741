"""ctypes wrapper of the serial C oracle (TEST INFRASTRUCTURE ONLY).

``build()`` compiles ``oracle_wfst.c`` with gcc (-O2, no FP contraction, no
fast-math) into ``liboracle_wfst.so`` next to this file; ``decode()`` runs one
utterance and returns its outputs as numpy arrays.
"""
from __future__ import annotations

import ctypes as C
import dataclasses
import os
import subprocess
import threading
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "oracle_wfst.c")
LIB = os.path.join(HERE, "liboracle_wfst.so")

ORACLE_OK = 0
ORACLE_EINVAL = -1
ORACLE_ENOMEM = -2
ORACLE_ENOPATH = -3
ORACLE_EINTERNAL = -9


class _Result(C.Structure):
    _fields_ = [
        ("status", C.c_int32),
        ("cost", C.c_float),
        ("final_state", C.c_int32),
        ("reached_final", C.c_int32),
        ("path_len", C.c_int32),
        ("path_arcs", C.POINTER(C.c_int32)),
        ("path_frames", C.POINTER(C.c_int32)),
        ("num_frames", C.c_int32),
        ("num_decoded", C.c_int32),
        ("kept", C.POINTER(C.c_int32)),
        ("tok_off", C.POINTER(C.c_int64)),
        ("tok_state", C.POINTER(C.c_int32)),
        ("tok_cost_bits", C.POINTER(C.c_uint32)),
        ("tok_arc", C.POINTER(C.c_int32)),
        ("cut_key", C.POINTER(C.c_uint32)),
        ("lat_raw", C.c_int64),
        ("lat_n", C.c_int64),
        ("lat_frame", C.POINTER(C.c_int32)),
        ("lat_arc", C.POINTER(C.c_int32)),
        ("lat_cost", C.POINTER(C.c_float)),
        ("lat_extra", C.POINTER(C.c_float)),
        ("arcs_expanded", C.c_int64),
        ("eps_arcs", C.c_int64),
        ("tokens", C.c_int64),
        ("seconds", C.c_double),
    ]


@dataclasses.dataclass
class OracleResult:
    status: int
    cost: float = float("nan")
    final_state: int = -1
    reached_final: int = 0
    path_arcs: Optional[np.ndarray] = None
    path_frames: Optional[np.ndarray] = None
    num_frames: int = 0
    num_decoded: int = 0
    kept: Optional[np.ndarray] = None
    tok_off: Optional[np.ndarray] = None
    tok_state: Optional[np.ndarray] = None
    tok_cost_bits: Optional[np.ndarray] = None
    tok_arc: Optional[np.ndarray] = None
    cut_key: Optional[np.ndarray] = None
    lat_raw: int = 0
    lat_frame: Optional[np.ndarray] = None
    lat_arc: Optional[np.ndarray] = None
    lat_cost: Optional[np.ndarray] = None
    lat_extra: Optional[np.ndarray] = None
    arcs_expanded: int = 0
    eps_arcs: int = 0
    tokens: int = 0
    seconds: float = 0.0

    def token_set(self, j: int):
        """(state, cost bits, back-pointer arc) of token set j, sorted by state."""
        a, b = int(self.tok_off[j]), int(self.tok_off[j + 1])
        return self.tok_state[a:b], self.tok_cost_bits[a:b], self.tok_arc[a:b]

    def token_cost(self, j: int) -> np.ndarray:
        return self.token_set(j)[1].view(np.float32)


_lib = None
_lock = threading.Lock()


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (always when force, else only if missing
    or older than its source)."""
    if force or not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
        tmp = LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-std=c11",
                               "-D_POSIX_C_SOURCE=200809L", "-shared", "-fPIC", "-o", tmp, SRC,
                               "-lm"])
        os.replace(tmp, LIB)
    return LIB


def _load():
    global _lib
    with _lock:
        if _lib is None:
            # WFST_ORACLE_LIB lets the mutation tests load a deliberately
            # broken build of this same source
            path = os.environ.get("WFST_ORACLE_LIB")
            if not path:
                path = build()
            lib = C.CDLL(path)
            i32p = C.POINTER(C.c_int32)
            f32p = C.POINTER(C.c_float)
            lib.oracle_decode.restype = C.POINTER(_Result)
            lib.oracle_decode.argtypes = [C.c_int32, C.c_int64, i32p, i32p, i32p, i32p, f32p,
                                          C.c_int32, f32p, f32p, C.c_int32, C.c_int32,
                                          C.c_float, C.c_int32, C.c_float, C.c_float, C.c_int32]
            lib.oracle_decode_ext.restype = C.POINTER(_Result)
            lib.oracle_decode_ext.argtypes = [C.c_int32, C.c_int64, i32p, i32p, i32p, i32p, f32p,
                                              C.c_int32, f32p, f32p, C.c_int32, C.c_int32,
                                              C.c_float, C.c_int32, C.c_float, C.c_float, i32p,
                                              C.c_int32, C.c_int32]
            lib.oracle_validate_graph.restype = C.c_int
            lib.oracle_validate_graph.argtypes = [C.c_int32, C.c_int64, i32p, i32p, i32p, i32p,
                                                  f32p, C.c_int32, f32p]
            lib.oracle_free.argtypes = [C.POINTER(_Result)]
            lib.oracle_free.restype = None
            _lib = lib
    return _lib


def _p(a, ct):
    if a is None:
        return None
    return a.ctypes.data_as(C.POINTER(ct))


def _arr(ptr, n, dt):
    if n <= 0 or not ptr:
        return np.zeros(0, dtype=dt)
    return np.ctypeslib.as_array(ptr, shape=(n,)).astype(dt, copy=True)


def _graph_arrays(g):
    src = np.ascontiguousarray(g.src, dtype=np.int32)
    dst = np.ascontiguousarray(g.dst, dtype=np.int32)
    il = np.ascontiguousarray(g.ilabel, dtype=np.int32)
    ol = np.ascontiguousarray(g.olabel, dtype=np.int32)
    w = np.ascontiguousarray(g.weight, dtype=np.float32)
    fw = None if g.final is None else np.ascontiguousarray(g.final, dtype=np.float32)
    return src, dst, il, ol, w, fw


def validate_graph(g) -> int:
    lib = _load()
    src, dst, il, ol, w, fw = _graph_arrays(g)
    return int(lib.oracle_validate_graph(g.num_states, src.shape[0], _p(src, C.c_int32),
                                         _p(dst, C.c_int32), _p(il, C.c_int32),
                                         _p(ol, C.c_int32), _p(w, C.c_float), g.start,
                                         _p(fw, C.c_float)))


def decode(g, loglikes: np.ndarray, beam: float, max_active: int = 0,
           lattice_beam: float = -1.0, blank_threshold: float = 2.0,
           blank_id: int = 0, blank_ids=None, frame_stride: int = 1) -> OracleResult:
    """Decode one utterance on the CPU.  ``g`` has the fields of
    ``workloads.Graph``; ``loglikes`` is float32 [T x L].  ``blank_ids``
    (a set of blank-like units) replaces ``blank_id`` when given;
    ``frame_stride`` decodes every frame_stride-th frame only."""
    lib = _load()
    src, dst, il, ol, w, fw = _graph_arrays(g)
    ll = np.ascontiguousarray(loglikes, dtype=np.float32)
    if ll.ndim != 2:
        raise ValueError("loglikes must be [T x L]")
    T, L = ll.shape
    ids = np.ascontiguousarray([blank_id] if blank_ids is None else blank_ids, dtype=np.int32)
    rp = lib.oracle_decode_ext(g.num_states, src.shape[0], _p(src, C.c_int32), _p(dst, C.c_int32),
                               _p(il, C.c_int32), _p(ol, C.c_int32), _p(w, C.c_float), g.start,
                               _p(fw, C.c_float), _p(ll, C.c_float), T, L, beam, max_active,
                               lattice_beam, blank_threshold, _p(ids, C.c_int32), ids.shape[0],
                               frame_stride)
    if not rp:
        raise MemoryError("oracle_decode returned NULL")
    try:
        r = rp.contents
        out = OracleResult(status=int(r.status))
        if r.status != ORACLE_OK:
            return out
        tp = int(r.num_decoded)
        out.cost = float(np.float32(r.cost))
        out.final_state = int(r.final_state)
        out.reached_final = int(r.reached_final)
        out.path_arcs = _arr(r.path_arcs, r.path_len, np.int32)
        out.path_frames = _arr(r.path_frames, r.path_len, np.int32)
        out.num_frames = int(r.num_frames)
        out.num_decoded = tp
        out.kept = _arr(r.kept, tp, np.int32)
        out.tok_off = _arr(r.tok_off, tp + 2, np.int64)
        nt = int(out.tok_off[-1])
        out.tok_state = _arr(r.tok_state, nt, np.int32)
        out.tok_cost_bits = _arr(r.tok_cost_bits, nt, np.uint32)
        out.tok_arc = _arr(r.tok_arc, nt, np.int32)
        out.cut_key = _arr(r.cut_key, tp + 1, np.uint32)
        out.lat_raw = int(r.lat_raw)
        out.lat_frame = _arr(r.lat_frame, r.lat_n, np.int32)
        out.lat_arc = _arr(r.lat_arc, r.lat_n, np.int32)
        out.lat_cost = _arr(r.lat_cost, r.lat_n, np.float32)
        out.lat_extra = _arr(r.lat_extra, r.lat_n, np.float32)
        out.arcs_expanded = int(r.arcs_expanded)
        out.eps_arcs = int(r.eps_arcs)
        out.tokens = int(r.tokens)
        out.seconds = float(r.seconds)
        return out
    finally:
        lib.oracle_free(rp)
