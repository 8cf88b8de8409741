"""Thin Python binding of libwfstdec.so (the C ABI in include/wfstdec.h).

The functions keep the C names (``wfst_load``, ``wfst_decode``,
``wfst_decode_batch``, ...) and only marshal arguments: every step of the
decode runs in the library's HIP kernels.  PyTorch supplies device memory
and streams; inputs may be torch tensors on the GPU (the normal case) or
numpy arrays (copied by the library, WFST_LOGLIKES_HOST).

If the library has not been built this module raises on import: there is no
CPU fallback.
"""
from __future__ import annotations

import ctypes as C
import dataclasses
import os
from typing import List, Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libwfstdec.so")

WFST_OK = 0
WFST_EINVAL = -1
WFST_ENOMEM = -2
WFST_ENOPATH = -3
WFST_ECAPACITY = -4
WFST_EDEVICE = -5

WFST_RECORD_TOKENS = 1
WFST_LOGLIKES_HOST = 2
WFST_PROFILE = 4
WFST_PROFILE_STEPS = 8
WFST_WORD_LATTICE = 16
WFST_INCREMENTAL_LATTICE = 32


class WfstError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__("wfstdec error %d: %s" % (code, msg))
        self.code = code


class _Opts(C.Structure):
    _fields_ = [("beam", C.c_float), ("max_active", C.c_int32), ("lattice_beam", C.c_float),
                ("blank_threshold", C.c_float), ("blank_id", C.c_int32), ("flags", C.c_uint32),
                ("capacity_hint", C.c_int64), ("blank_ids", C.c_void_p), ("num_blank_ids", C.c_int32),
                ("frame_stride", C.c_int32)]


class _Info(C.Structure):
    _fields_ = [("num_states", C.c_int32), ("num_arcs", C.c_int64), ("num_emitting", C.c_int64),
                ("num_epsilon", C.c_int64), ("max_ilabel", C.c_int32), ("epsilon_depth", C.c_int32),
                ("device_bytes", C.c_int64), ("num_closure_states", C.c_int64)]


class _Stats(C.Structure):
    _fields_ = [("frames", C.c_int32), ("frames_decoded", C.c_int32), ("tokens", C.c_int64),
                ("tokens_last", C.c_int64), ("arcs_expanded", C.c_int64), ("eps_arcs", C.c_int64), ("lattice_raw", C.c_int64),
                ("lattice_kept", C.c_int64), ("decode_ms", C.c_double), ("search_ms", C.c_double),
                ("record_ms", C.c_double), ("final_ms", C.c_double), ("search_launches", C.c_int32),
                ("search_phase_ms", C.c_double * 7), ("backtrace_ms", C.c_double),
                ("lattice_prune_ms", C.c_double), ("search_span_ms", C.c_double),
                ("word_sequences", C.c_int64), ("lattice_incremental", C.c_int64),
                ("workspace_bytes", C.c_int64)]


_STAT_FIELDS = tuple(f for f, _ in _Stats._fields_ if f != "search_phase_ms")


class _DebugOpts(C.Structure):
    _fields_ = [("lds_fill", C.c_int32), ("queue_cap", C.c_int32), ("record_fill", C.c_int32),
                ("record_big_fill", C.c_int32), ("lattice_lds", C.c_int32), ("permute", C.c_int32),
                ("fail_lattice_alloc", C.c_int32), ("lattice_chunk", C.c_int32), ("lattice_ring", C.c_int32),
                ("record_groups", C.c_int32), ("record_publish", C.c_int32),
                ("lattice_pipe", C.c_int32), ("lattice_spin", C.c_int32)]


class _LatArc(C.Structure):
    _fields_ = [("frame", C.c_int32), ("arc", C.c_int32), ("cost", C.c_float), ("extra", C.c_float)]


class _Summary(C.Structure):
    _fields_ = [("status", C.c_int32), ("num_frames", C.c_int32), ("num_decoded", C.c_int32),
                ("path_len", C.c_int32), ("cost", C.c_float), ("final_state", C.c_int32),
                ("reached_final", C.c_int32), ("reserved", C.c_int32),
                ("orig_frame", C.POINTER(C.c_int32)), ("path_arcs", C.POINTER(C.c_int32)),
                ("path_frames", C.POINTER(C.c_int32)), ("lattice_n", C.c_int64),
                ("lattice", C.POINTER(_LatArc)), ("stats", _Stats)]


class _NoallocOut(C.Structure):
    _fields_ = [("path_arcs", C.c_void_p), ("path_frames", C.c_void_p), ("path_cap", C.c_int32),
                ("lattice", C.c_void_p), ("lattice_cap", C.c_int64), ("kept", C.c_void_p), ("kept_cap", C.c_int32),
                ("status", C.c_int32), ("cost", C.c_float), ("final_state", C.c_int32),
                ("reached_final", C.c_int32), ("path_len", C.c_int32), ("num_decoded", C.c_int32),
                ("lattice_n", C.c_int64), ("lattice_raw", C.c_int64), ("tokens", C.c_int64),
                ("arcs_expanded", C.c_int64), ("eps_arcs", C.c_int64)]


def _load_lib():
    if not os.path.exists(LIB_PATH):
        raise ImportError("libwfstdec.so is not built (run __graft_entry__.build() or "
                          "python -m paper_1808_00687_amd.csrc.build)")
    lib = C.CDLL(LIB_PATH)
    i32p, f32p, vp = C.POINTER(C.c_int32), C.POINTER(C.c_float), C.c_void_p
    lib.wfst_load.argtypes = [C.c_int32, C.c_int64, i32p, i32p, i32p, i32p, f32p, C.c_int32, f32p,
                              C.POINTER(vp)]
    lib.wfst_load.restype = C.c_int
    lib.wfst_graph_free.argtypes = [vp]
    lib.wfst_graph_free.restype = None
    lib.wfst_graph_get_info.argtypes = [vp, C.POINTER(_Info)]
    lib.wfst_graph_get_info.restype = C.c_int
    lib.wfst_default_opts.argtypes = [C.POINTER(_Opts)]
    lib.wfst_default_opts.restype = None
    lib.wfst_decode.argtypes = [vp, vp, C.c_int32, C.c_int32, C.POINTER(_Opts), vp, C.POINTER(vp)]
    lib.wfst_decode.restype = C.c_int
    lib.wfst_decode_batch.argtypes = [vp, C.c_int32, C.POINTER(vp), i32p, C.c_int32,
                                      C.POINTER(_Opts), vp, C.POINTER(vp)]
    lib.wfst_decode_batch.restype = C.c_int
    lib.wfst_result_status.argtypes = [vp]
    lib.wfst_result_status.restype = C.c_int
    lib.wfst_result_best.argtypes = [vp, f32p, i32p, i32p, i32p, C.POINTER(i32p), C.POINTER(i32p)]
    lib.wfst_result_best.restype = C.c_int
    lib.wfst_result_frames.argtypes = [vp, i32p, i32p, C.POINTER(i32p)]
    lib.wfst_result_frames.restype = C.c_int
    lib.wfst_result_lattice.argtypes = [vp, C.POINTER(C.c_int64), C.POINTER(C.POINTER(_LatArc))]
    lib.wfst_result_lattice.restype = C.c_int
    lib.wfst_result_lattice_device.argtypes = [vp, C.POINTER(C.c_int64), C.POINTER(vp)]
    lib.wfst_result_lattice_device.restype = C.c_int
    lib.wfst_result_tokens.argtypes = [vp, C.c_int32, i32p, C.POINTER(i32p), C.POINTER(f32p),
                                       C.POINTER(i32p)]
    lib.wfst_result_tokens.restype = C.c_int
    lib.wfst_result_words.argtypes = [vp, C.POINTER(C.c_int64), C.POINTER(C.POINTER(C.c_int64)),
                                      C.POINTER(i32p), C.POINTER(f32p)]
    lib.wfst_result_words.restype = C.c_int
    lib.wfst_result_stats.argtypes = [vp, C.POINTER(_Stats)]
    lib.wfst_result_stats.restype = C.c_int
    lib.wfst_result_summaries.argtypes = [C.POINTER(vp), C.c_int32, C.c_int32, C.POINTER(_Summary)]
    lib.wfst_result_summaries.restype = C.c_int
    lib.wfst_result_free.argtypes = [vp]
    lib.wfst_result_free.restype = None
    lib.wfst_decode_noalloc.argtypes = [vp, vp, C.c_int32, C.c_int32, C.POINTER(_Opts), vp, C.POINTER(_NoallocOut)]
    lib.wfst_decode_noalloc.restype = C.c_int
    lib.wfst_set_debug_opts.argtypes = [C.POINTER(_DebugOpts)]
    lib.wfst_set_debug_opts.restype = C.c_int
    lib.wfst_last_error.argtypes = []
    lib.wfst_last_error.restype = C.c_char_p
    return lib


_lib = _load_lib()


def wfst_last_error() -> str:
    return _lib.wfst_last_error().decode(errors="replace")


def _check(rc: int, what: str):
    if rc != WFST_OK:
        raise WfstError(rc, "%s: %s" % (what, wfst_last_error()))


def wfst_set_debug_opts(**fields) -> None:
    """Process-wide test and debugging switches (wfst_set_debug_opts in
    include/wfstdec.h); no arguments restores the defaults."""
    if not fields:
        _check(_lib.wfst_set_debug_opts(None), "wfst_set_debug_opts")
        return
    o = _DebugOpts()
    for k, v in fields.items():
        setattr(o, k, int(v))
    _check(_lib.wfst_set_debug_opts(C.byref(o)), "wfst_set_debug_opts")


class debug_opts:
    """Context manager: wfst_set_debug_opts(**fields) inside, defaults after."""

    def __init__(self, **fields):
        self.fields = fields

    def __enter__(self):
        wfst_set_debug_opts(**self.fields)
        return self

    def __exit__(self, *exc):
        wfst_set_debug_opts()


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def _p(a, ct):
    return None if a is None else a.ctypes.data_as(C.POINTER(ct))


# --------------------------------------------------------------------------
# graphs
# --------------------------------------------------------------------------

class WfstGraph:
    """Owns a wfst_graph handle (device layout of one WFST)."""

    def __init__(self, handle):
        self._h = handle

    @property
    def handle(self):
        return self._h

    def info(self) -> dict:
        i = _Info()
        _check(_lib.wfst_graph_get_info(self._h, C.byref(i)), "wfst_graph_get_info")
        return {f: getattr(i, f) for f, _ in _Info._fields_}

    def free(self):
        if self._h:
            _lib.wfst_graph_free(self._h)
            self._h = None

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass


def wfst_load(num_states: int, src, dst, ilabel, olabel, weight, start_state: int = 0,
              final_weight=None) -> WfstGraph:
    """Validate and upload a WFST (arc arrays sorted by src); see wfst_load in
    include/wfstdec.h."""
    src, dst, il, ol = _i32(src), _i32(dst), _i32(ilabel), _i32(olabel)
    w = np.ascontiguousarray(weight, dtype=np.float32)
    fw = None if final_weight is None else np.ascontiguousarray(final_weight, dtype=np.float32)
    e = src.shape[0]
    if not (dst.shape[0] == il.shape[0] == ol.shape[0] == w.shape[0] == e):
        raise ValueError("arc arrays differ in length")
    if fw is not None and fw.shape[0] != num_states:
        raise ValueError("final_weight must have num_states entries")
    h = C.c_void_p()
    rc = _lib.wfst_load(num_states, e, _p(src, C.c_int32), _p(dst, C.c_int32), _p(il, C.c_int32),
                        _p(ol, C.c_int32), _p(w, C.c_float), start_state, _p(fw, C.c_float),
                        C.byref(h))
    _check(rc, "wfst_load")
    return WfstGraph(h)


def load_graph(g) -> WfstGraph:
    """wfst_load from an object with the fields of workloads.Graph."""
    return wfst_load(g.num_states, g.src, g.dst, g.ilabel, g.olabel, g.weight, g.start, g.final)


# --------------------------------------------------------------------------
# results
# --------------------------------------------------------------------------

@dataclasses.dataclass
class WfstResult:
    status: int
    num_frames: int = 0
    num_decoded: int = 0
    kept: Optional[np.ndarray] = None
    cost: float = float("nan")
    final_state: int = -1
    reached_final: int = 0
    path_arcs: Optional[np.ndarray] = None
    path_frames: Optional[np.ndarray] = None
    lat_frame: Optional[np.ndarray] = None
    lat_arc: Optional[np.ndarray] = None
    lat_cost: Optional[np.ndarray] = None
    lat_extra: Optional[np.ndarray] = None
    tok_off: Optional[np.ndarray] = None
    tok_state: Optional[np.ndarray] = None
    tok_cost: Optional[np.ndarray] = None
    tok_arc: Optional[np.ndarray] = None
    stats: Optional[dict] = None
    words: Optional[list] = None          # word-level lattice: [(word tuple, float32 cost)] sorted by cost

    def token_set(self, j: int):
        """(state, cost bits, back-pointer arc) of token set j, sorted by state."""
        a, b = int(self.tok_off[j]), int(self.tok_off[j + 1])
        return self.tok_state[a:b], self.tok_cost[a:b].view(np.uint32), self.tok_arc[a:b]


def _arr(ptr, n, dt):
    """Copy of n elements of type dt at a library pointer (one memmove: a
    ctypes array view per call costs more than the copy)."""
    if n <= 0 or not ptr:
        return np.zeros(0, dtype=dt)
    a = np.empty(n, dtype=dt)
    C.memmove(a.ctypes.data, ptr, a.nbytes)
    return a


def _lattice_views(outs, spans=None) -> list:
    """Each result's lattice as an [n x 4] int32 view of one host copy: the
    lattices of a batch lie in one host buffer the results share, copied here
    once instead of once per result.  spans: (address, arcs) of each result's
    lattice when the caller has them already."""
    if spans is None:
        spans = []
        for h in outs:
            ln = C.c_int64()
            la = C.POINTER(_LatArc)()
            _check(_lib.wfst_result_lattice(h, C.byref(ln), C.byref(la)), "wfst_result_lattice")
            spans.append((C.cast(la, C.c_void_p).value or 0, ln.value))
    live = [(p, m) for p, m in spans if m > 0 and p]
    if not live:
        return [np.zeros((0, 4), np.int32)] * len(spans)
    base = min(p for p, _ in live)
    end = max(p + 16 * m for p, m in live)
    big = np.ctypeslib.as_array(C.cast(C.c_void_p(base), C.POINTER(C.c_int32)), shape=((end - base) // 16, 4)).copy()
    views = []
    for p, m in spans:
        i = (p - base) // 16 if m > 0 and p else 0
        views.append(big[i:i + m] if m > 0 and p else np.zeros((0, 4), np.int32))
    return views


def _collect(h, lattice: bool, tokens: bool, lat=None, words: bool = False, sm=None) -> WfstResult:
    """The result behind handle h; sm: its wfst_result_summaries entry, when
    the caller has fetched those for the batch (else per-result calls)."""
    if sm is None:
        st = _lib.wfst_result_status(h)
        nf, nd = C.c_int32(), C.c_int32()
        kp = C.POINTER(C.c_int32)()
        _check(_lib.wfst_result_frames(h, C.byref(nf), C.byref(nd), C.byref(kp)), "wfst_result_frames")
        num_frames, num_decoded = nf.value, nd.value
        s = _Stats()
        _check(_lib.wfst_result_stats(h, C.byref(s)), "wfst_result_stats")
    else:
        st, num_frames, num_decoded, kp, s = sm.status, sm.num_frames, sm.num_decoded, sm.orig_frame, sm.stats
    r = WfstResult(status=st)
    r.num_frames, r.num_decoded = num_frames, num_decoded
    r.kept = _arr(kp, num_decoded, np.int32)
    r.stats = {f: getattr(s, f) for f in _STAT_FIELDS}
    r.stats["search_phase_ms"] = list(s.search_phase_ms)
    if st != WFST_OK:
        return r
    if sm is None:
        cost, fs, rf, n = C.c_float(), C.c_int32(), C.c_int32(), C.c_int32()
        pa, pf = C.POINTER(C.c_int32)(), C.POINTER(C.c_int32)()
        _check(_lib.wfst_result_best(h, C.byref(cost), C.byref(fs), C.byref(rf), C.byref(n),
                                     C.byref(pa), C.byref(pf)), "wfst_result_best")
        cost, fs, rf, n = cost.value, fs.value, rf.value, n.value
    else:
        cost, fs, rf, n, pa, pf = sm.cost, sm.final_state, sm.reached_final, sm.path_len, sm.path_arcs, sm.path_frames
    r.cost, r.final_state, r.reached_final = float(np.float32(cost)), fs, rf
    r.path_arcs = _arr(pa, n, np.int32)
    r.path_frames = _arr(pf, n, np.int32)
    if lattice:
        if lat is None:
            lat = _lattice_views([h])[0]
        fl = lat.view(np.float32)
        r.lat_frame = lat[:, 0]
        r.lat_arc = lat[:, 1]
        r.lat_cost = fl[:, 2]
        r.lat_extra = fl[:, 3]
    if words:
        wn = C.c_int64()
        wo = C.POINTER(C.c_int64)()
        ww, wc = C.POINTER(C.c_int32)(), C.POINTER(C.c_float)()
        _check(_lib.wfst_result_words(h, C.byref(wn), C.byref(wo), C.byref(ww), C.byref(wc)), "wfst_result_words")
        off = _arr(wo, wn.value + 1, np.int64)
        wl = _arr(ww, int(off[-1]) if wn.value else 0, np.int32)
        cs = _arr(wc, wn.value, np.float32)
        r.words = [(tuple(int(x) for x in wl[off[k]:off[k + 1]]), np.float32(cs[k])) for k in range(wn.value)]
    if tokens:
        offs = [0]
        states, costs, arcs = [], [], []
        for j in range(r.num_decoded + 1):
            tn = C.c_int32()
            sp, cp, ap = C.POINTER(C.c_int32)(), C.POINTER(C.c_float)(), C.POINTER(C.c_int32)()
            _check(_lib.wfst_result_tokens(h, j, C.byref(tn), C.byref(sp), C.byref(cp), C.byref(ap)),
                   "wfst_result_tokens")
            states.append(_arr(sp, tn.value, np.int32))
            costs.append(_arr(cp, tn.value, np.float32))
            arcs.append(_arr(ap, tn.value, np.int32))
            offs.append(offs[-1] + tn.value)
        r.tok_off = np.array(offs, np.int64)
        r.tok_state = np.concatenate(states)
        r.tok_cost = np.concatenate(costs)
        r.tok_arc = np.concatenate(arcs)
    return r


# --------------------------------------------------------------------------
# decode
# --------------------------------------------------------------------------

def _opts(beam, max_active, lattice_beam, blank_threshold, blank_id, flags, capacity_hint,
          blank_ids=None, frame_stride=1, keep=None) -> _Opts:
    o = _Opts()
    _lib.wfst_default_opts(C.byref(o))
    o.beam = beam
    o.max_active = max_active
    o.lattice_beam = lattice_beam
    o.blank_threshold = blank_threshold
    o.blank_id = blank_id
    o.flags = flags
    o.capacity_hint = capacity_hint
    if blank_ids is not None:
        ids = np.ascontiguousarray(blank_ids, dtype=np.int32)
        if keep is not None:
            keep.append(ids)
        o.blank_ids = ids.ctypes.data if ids.size else None
        o.num_blank_ids = ids.size if ids.size else -1   # an empty set is an error
    o.frame_stride = frame_stride
    return o


def _ll_ptr(x, keep: list):
    """Device pointer of a CUDA float32 tensor, or host pointer of numpy."""
    if isinstance(x, np.ndarray):
        a = np.ascontiguousarray(x, dtype=np.float32)
        keep.append(a)
        return a.ctypes.data, a.shape, True
    import torch
    if not isinstance(x, torch.Tensor):
        raise TypeError("loglikes must be a torch tensor or a numpy array")
    if x.dtype != torch.float32 or x.dim() != 2:
        raise ValueError("loglikes must be a 2-D float32 tensor [T x L]")
    if not x.is_contiguous():
        x = x.contiguous()
    keep.append(x)
    return x.data_ptr(), tuple(x.shape), not x.is_cuda


def _stream_handle(stream):
    if stream is None:
        try:
            import torch
            if torch.cuda.is_available():
                return torch.cuda.current_stream().cuda_stream
        except Exception:
            pass
        return None
    return getattr(stream, "cuda_stream", stream)


def wfst_decode_batch(graph: WfstGraph, loglikes: Sequence, beam: float, max_active: int = 0,
                      lattice_beam: float = -1.0, blank_threshold: float = 2.0, blank_id: int = 0,
                      record_tokens: bool = False, profile: bool = False, capacity_hint: int = 0,
                      stream=None, profile_steps: bool = False, blank_ids=None,
                      frame_stride: int = 1, word_lattice: bool = False,
                      incremental_lattice: bool = False) -> List[WfstResult]:
    """Decode a batch of utterances (wfst_decode_batch).  ``loglikes`` are
    [T_u x L] float32 tensors on the graph's device (or numpy arrays)."""
    keep: list = []
    ptrs, Ts, L, host = [], [], None, None
    for x in loglikes:
        ptr, shape, is_host = _ll_ptr(x, keep)
        if L is None:
            L, host = shape[1], is_host
        if shape[1] != L or is_host != host:
            raise ValueError("all utterances need the same L and memory kind")
        ptrs.append(ptr)
        Ts.append(shape[0])
    n = len(ptrs)
    flags = (WFST_RECORD_TOKENS if record_tokens else 0) | (WFST_LOGLIKES_HOST if host else 0) | \
        (WFST_PROFILE if profile else 0) | (WFST_PROFILE_STEPS if profile_steps else 0) | \
        (WFST_WORD_LATTICE if word_lattice else 0) | (WFST_INCREMENTAL_LATTICE if incremental_lattice else 0)
    o = _opts(beam, max_active, lattice_beam, blank_threshold, blank_id, flags, capacity_hint,
              blank_ids, frame_stride, keep)
    parr = (C.c_void_p * n)(*ptrs)
    tarr = np.array(Ts, np.int32)
    outs = (C.c_void_p * n)()
    rc = _lib.wfst_decode_batch(graph.handle, n, parr, _p(tarr, C.c_int32), L, C.byref(o),
                                _stream_handle(stream), outs)
    _check(rc, "wfst_decode_batch")
    res = []
    try:
        # the results' fields in one call (per-result calls cost more than
        # their work for a batch of short results)
        summ = (_Summary * n)()
        want_lat = lattice_beam >= 0
        _check(_lib.wfst_result_summaries(outs, n, 1 if want_lat else 0, summ), "wfst_result_summaries")
        sms = list(summ)
        if want_lat:
            lats = _lattice_views(outs, [(C.cast(sm.lattice, C.c_void_p).value or 0, sm.lattice_n) for sm in sms])
        else:
            lats = [None] * n
        for h, lat, sm in zip(outs, lats, sms):
            res.append(_collect(h, want_lat, record_tokens, lat, word_lattice, sm))
    finally:
        for h in outs:
            _lib.wfst_result_free(h)
    return res


def wfst_decode(graph: WfstGraph, loglikes, beam: float, max_active: int = 0,
                lattice_beam: float = -1.0, blank_threshold: float = 2.0, blank_id: int = 0,
                record_tokens: bool = False, profile: bool = False, capacity_hint: int = 0,
                stream=None, profile_steps: bool = False, blank_ids=None,
                frame_stride: int = 1, word_lattice: bool = False,
                incremental_lattice: bool = False) -> WfstResult:
    """Decode one utterance (wfst_decode).  Returns the result also when the
    status is WFST_ENOPATH; other errors raise WfstError."""
    keep: list = []
    ptr, shape, host = _ll_ptr(loglikes, keep)
    flags = (WFST_RECORD_TOKENS if record_tokens else 0) | (WFST_LOGLIKES_HOST if host else 0) | \
        (WFST_PROFILE if profile else 0) | (WFST_PROFILE_STEPS if profile_steps else 0) | \
        (WFST_WORD_LATTICE if word_lattice else 0) | (WFST_INCREMENTAL_LATTICE if incremental_lattice else 0)
    o = _opts(beam, max_active, lattice_beam, blank_threshold, blank_id, flags, capacity_hint,
              blank_ids, frame_stride, keep)
    out = C.c_void_p()
    rc = _lib.wfst_decode(graph.handle, ptr, shape[0], shape[1], C.byref(o), _stream_handle(stream),
                          C.byref(out))
    if rc not in (WFST_OK, WFST_ENOPATH) or not out:
        raise WfstError(rc, "wfst_decode: %s" % wfst_last_error())
    try:
        return _collect(out, lattice_beam >= 0, record_tokens, None, word_lattice)
    finally:
        _lib.wfst_result_free(out)


WFST_NOALLOC_SCRATCH_BYTES = 512 << 20


@dataclasses.dataclass
class NoallocResult:
    """Outputs of wfst_decode_noalloc: the host fields of the descriptor and
    the caller-owned device buffers (torch tensors) it wrote."""
    rc: int
    status: int
    cost: float
    final_state: int
    reached_final: int
    path_len: int
    num_decoded: int
    lattice_n: int
    lattice_raw: int
    tokens: int
    arcs_expanded: int
    eps_arcs: int
    path_arcs: object       # int32 tensor [path_cap] on the device
    path_frames: object
    lattice: object         # int32 tensor [lattice_cap, 4] on the device
    kept: object            # int32 tensor [kept_cap] on the device


def wfst_decode_noalloc(graph: WfstGraph, loglikes, beam: float, max_active: int = 0,
                        lattice_beam: float = -1.0, blank_threshold: float = 2.0, blank_id: int = 0,
                        path_cap: int = 4096, lattice_cap: int = 1 << 16, kept_cap: int = 0,
                        capacity_hint: int = 0, stream=None, blank_ids=None, frame_stride: int = 1,
                        outputs=None) -> NoallocResult:
    """Decode one utterance with wfst_decode_noalloc.  ``loglikes`` is a
    [T x L] float32 tensor on the graph's device.  The output buffers are
    torch tensors: ``outputs`` = (path_arcs, path_frames, lattice, kept) to
    reuse existing ones, else they are created here (by the caller's side,
    as the C call itself allocates nothing).  Returns the return code with
    the outputs; a WfstError is raised only for WFST_EINVAL and
    WFST_EDEVICE."""
    import torch
    keep: list = []
    ptr, shape, host = _ll_ptr(loglikes, keep)
    if host:
        raise ValueError("wfst_decode_noalloc takes device log-likelihoods")
    dev = loglikes.device
    if outputs is None:
        pa = torch.empty(max(path_cap, 1), dtype=torch.int32, device=dev)
        pf = torch.empty(max(path_cap, 1), dtype=torch.int32, device=dev)
        lat = torch.empty((max(lattice_cap, 1), 4), dtype=torch.int32, device=dev)
        kp = torch.empty(max(kept_cap, 1), dtype=torch.int32, device=dev)
    else:
        pa, pf, lat, kp = outputs
        path_cap, lattice_cap, kept_cap = pa.numel(), lat.shape[0], kp.numel()
    o = _opts(beam, max_active, lattice_beam, blank_threshold, blank_id, 0, capacity_hint, blank_ids,
              frame_stride, keep)
    d = _NoallocOut()
    d.path_arcs, d.path_frames, d.path_cap = pa.data_ptr(), pf.data_ptr(), path_cap
    d.lattice, d.lattice_cap = lat.data_ptr(), lattice_cap
    d.kept, d.kept_cap = (kp.data_ptr(), kept_cap) if kept_cap > 0 else (None, 0)
    rc = _lib.wfst_decode_noalloc(graph.handle, ptr, shape[0], shape[1], C.byref(o), _stream_handle(stream),
                                  C.byref(d))
    if rc in (WFST_EINVAL, WFST_EDEVICE):
        raise WfstError(rc, "wfst_decode_noalloc: %s" % wfst_last_error())
    return NoallocResult(rc=rc, status=d.status, cost=float(np.float32(d.cost)), final_state=d.final_state,
                         reached_final=d.reached_final, path_len=d.path_len, num_decoded=d.num_decoded,
                         lattice_n=d.lattice_n, lattice_raw=d.lattice_raw, tokens=d.tokens,
                         arcs_expanded=d.arcs_expanded, eps_arcs=d.eps_arcs, path_arcs=pa, path_frames=pf,
                         lattice=lat, kept=kp)
