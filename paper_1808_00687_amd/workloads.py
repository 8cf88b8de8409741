"""Seeded synthetic workloads for the WFST Viterbi / LSD decoder.

This module only draws random inputs (graphs, acoustic log-likelihoods and
decode options).  It holds none of the decoding arithmetic: the serial CPU
oracle and the HIP path both receive the same arrays from here and share
nothing else.

The paper measures on Switchboard / hub5e-swb with trained CTC and hybrid
acoustic models and n-gram LMs (Sec. 2, Fig. 1; Sec. 3, Fig. 3).  None of
those assets exist here, so five synthetic workloads of the same structure
stand in for them:

1. tiny random WFST (2,000 states), 50 frames, beam 12;
2. medium WFST (200k states, 1M arcs, Zipf-like out-degree), 500 frames,
   max-active 7,000, lattice beam 8;
3. LVCSR-scale HCLG-like WFST (10M states, 25M arcs, 6,000 senones,
   olabels on 10% of arcs), 1,000 frames, max-active 10,000, lattice beam 8;
4. the graph of (3) shared by 64 utterances of 300-1,500 frames;
5. a CTC-style graph (5M states, 15M arcs, a blank self-loop on every state)
   with blank-dominated frames, decoded frame-synchronously and
   label-synchronously (Sec. 2, Alg. 1).

Recipe (every draw comes from ``numpy.random.default_rng`` seeded with
``SeedSequence([1808, 687, cfg, purpose, utt])``; purpose 0 = graph,
1 = log-likelihoods):

* arcs are generated state by state, so ``src`` is sorted; the start state is
  0; no final weights;
* an emitting arc has ``dst`` uniform in [0, N) and ``ilabel`` uniform in
  [1, L] (ilabel i reads log-likelihood column i-1; 0 is epsilon);
* an epsilon arc has ``dst`` uniform in (s, N), so the epsilon subgraph is
  acyclic; an epsilon arc drawn on the last state is made emitting;
* weights are Exp(mean) drawn in float64 and cast to float32;
* log-likelihoods are ``z - logsumexp(z)`` per row with ``z ~ N(0, sigma)``
  drawn in float64, cast to float32, row-major [T x L].

The Zipf-like out-degree of configs 2, 3 and 5 is a rank law
``deg(r) = clip(floor(C * r**-1.2), 1, 200)`` for ranks r = 1..N with C the
largest constant whose total does not exceed the arc budget; the residual
arcs go, one each, to randomly chosen degree-1 states, and a seeded random
permutation maps ranks to states.  (An i.i.d. Zipf(1.2) draw cannot give a
mean degree of 2.5-5 at a cap of 200, so the rank law is used instead.)
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional

import numpy as np

GRAPH = 0
LOGLIKES = 1


def rng_for(cfg: int, purpose: int, utt: int = 0) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([1808, 687, cfg, purpose, utt]))


@dataclasses.dataclass
class Graph:
    num_states: int
    src: np.ndarray      # int32 [E], sorted ascending
    dst: np.ndarray      # int32 [E]
    ilabel: np.ndarray   # int32 [E], 0 = epsilon, i >= 1 reads column i-1
    olabel: np.ndarray   # int32 [E], 0 = no output
    weight: np.ndarray   # float32 [E]
    start: int = 0
    final: Optional[np.ndarray] = None  # float32 [N] or None (all final, cost 0)

    @property
    def num_arcs(self) -> int:
        return int(self.src.shape[0])


@dataclasses.dataclass
class DecodeOpts:
    beam: float
    max_active: int = 0            # <= 0: unlimited
    lattice_beam: float = -1.0     # < 0: no lattice
    blank_threshold: float = 2.0   # > 1: frame synchronous
    blank_id: int = 0
    blank_ids: Optional[tuple] = None   # a set of blank-like units instead of blank_id
    frame_stride: int = 1               # decode every frame_stride-th frame


@dataclasses.dataclass
class Workload:
    cfg: int
    name: str
    graph: Graph
    num_labels: int
    loglikes: List[np.ndarray]  # one float32 [T x L] array per utterance
    opts: DecodeOpts


# --------------------------------------------------------------------------
# graph pieces
# --------------------------------------------------------------------------

def _rank_law_total(c: float, n: int, s: float, cap: int, r: np.ndarray) -> int:
    """sum over ranks 1..n of clip(floor(c * r**-s), 1, cap), evaluating only
    the ranks strictly between the capped head and the degree-1 tail."""
    r_cap = int(np.floor((c / cap) ** (1.0 / s)))          # c r^-s >= cap for r <= r_cap
    r_one = int(np.ceil(c ** (1.0 / s))) + 1               # c r^-s < 1 beyond this
    lo = max(min(r_cap - 2, n), 0)
    hi = max(min(r_one, n), lo)
    mid = np.clip(np.floor(c * r[lo:hi] ** (-s)), 1, cap).sum()
    return int(lo * cap + mid + (n - hi))


def rank_law_degrees(n: int, total: int, s: float, cap: int,
                     rng: np.random.Generator) -> np.ndarray:
    """Out-degree per state from the rank law, permuted onto states."""
    r = np.arange(1, n + 1, dtype=np.float64)
    lo, hi = 1.0, 1e13
    for _ in range(80):
        mid = np.sqrt(lo * hi)
        if _rank_law_total(mid, n, s, cap, r) <= total:
            lo = mid
        else:
            hi = mid
    deg = np.clip(np.floor(lo * r ** (-s)), 1, cap).astype(np.int64)
    resid = total - int(deg.sum())
    assert resid >= 0
    if resid:
        ones = np.flatnonzero(deg == 1)
        pick = ones[rng.choice(ones.size, size=resid, replace=False)]
        deg[pick] += 1
    perm = rng.permutation(n)
    out = np.empty(n, dtype=np.int64)
    out[perm] = deg
    return out


def arcs_from_degrees(n: int, deg: np.ndarray, eps_frac: float, num_labels: int,
                      mean_w: float, rng: np.random.Generator,
                      first_label: int = 1) -> dict:
    """Arcs state by state; epsilon arcs only to higher-index states."""
    src = np.repeat(np.arange(n, dtype=np.int32), deg)
    e = src.shape[0]
    is_eps = rng.random(e) < eps_frac
    is_eps &= src < n - 1
    eps = np.flatnonzero(is_eps)
    del is_eps
    dst = rng.integers(0, n, size=e, dtype=np.int32)
    dst[eps] = rng.integers(src[eps] + 1, n, dtype=np.int32)
    il = rng.integers(first_label, num_labels + 1, size=e, dtype=np.int32)
    il[eps] = 0
    w = rng.exponential(mean_w, size=e).astype(np.float32)
    return dict(src=src, dst=dst, ilabel=il, weight=w)


def graph_cfg1() -> Graph:
    rng = rng_for(1, GRAPH)
    n = 2000
    deg = 1 + rng.poisson(3.0, size=n)
    a = arcs_from_degrees(n, deg, 0.15, 64, 1.5, rng)
    return Graph(n, a["src"], a["dst"], a["ilabel"], np.zeros_like(a["src"]), a["weight"])


def graph_rank_law(cfg: int, n: int, e: int, eps_frac: float, num_labels: int,
                   mean_w: float, olabel_frac: float = 0.0, vocab: int = 0) -> Graph:
    rng = rng_for(cfg, GRAPH)
    deg = rank_law_degrees(n, e, 1.2, 200, rng)
    a = arcs_from_degrees(n, deg, eps_frac, num_labels, mean_w, rng)
    if olabel_frac > 0:
        has = rng.random(e) < olabel_frac
        ol = np.where(has, rng.integers(1, vocab + 1, size=e), 0).astype(np.int32)
    else:
        ol = np.zeros(e, dtype=np.int32)
    return Graph(n, a["src"], a["dst"], a["ilabel"], ol, a["weight"])


def graph_cfg2() -> Graph:
    return graph_rank_law(2, 200_000, 1_000_000, 0.12, 2000, 2.0)


def graph_cfg3() -> Graph:
    return graph_rank_law(3, 10_000_000, 25_000_000, 0.20, 6000, 2.5, 0.10, 100_000)


def graph_cfg5() -> Graph:
    """CTC-style: a blank self-loop (ilabel 1 = column 0) on every state,
    plus 10M rank-law arcs with non-blank labels 2..80, 15% of them epsilon
    (about 10% of all 15M arcs)."""
    rng = rng_for(5, GRAPH)
    n = 5_000_000
    deg = rank_law_degrees(n, 10_000_000, 1.2, 200, rng)
    a = arcs_from_degrees(n, deg, 0.15, 80, 2.0, rng, first_label=2)
    loop_w = rng.exponential(2.0, size=n).astype(np.float32)
    # interleave: state s owns [self-loop, its rank-law arcs...]
    tot = n + a["src"].shape[0]
    rows = np.zeros(n + 1, dtype=np.int64)
    rows[1:] = np.cumsum(deg + 1)
    loop_pos = rows[:-1]
    other_pos = np.ones(tot, dtype=bool)
    other_pos[loop_pos] = False
    src = np.empty(tot, np.int32); dst = np.empty(tot, np.int32)
    il = np.empty(tot, np.int32); w = np.empty(tot, np.float32)
    src[loop_pos] = np.arange(n, dtype=np.int32); dst[loop_pos] = np.arange(n, dtype=np.int32)
    il[loop_pos] = 1; w[loop_pos] = loop_w
    src[other_pos] = a["src"]; dst[other_pos] = a["dst"]
    il[other_pos] = a["ilabel"]; w[other_pos] = a["weight"]
    return Graph(n, src, dst, il, np.zeros(tot, np.int32), w)


HMM_BLANK_UNITS = 8   # blank-like units of the HMM-topology stand-in (columns 0..7)


def graph_cfg6() -> Graph:
    """HMM-topology stand-in for the LSD variant the paper extends to HMM
    models whose topology has a blank-like state (Sec. 2): the config-5
    shape, but each state's self-loop reads one of HMM_BLANK_UNITS blank-like
    units (ilabels 1..8, one per "phone" group, drawn per state), and the
    rank-law arcs read the labels 9..80."""
    rng = rng_for(6, GRAPH)
    n = 5_000_000
    k = HMM_BLANK_UNITS
    deg = rank_law_degrees(n, 10_000_000, 1.2, 200, rng)
    a = arcs_from_degrees(n, deg, 0.15, 80, 2.0, rng, first_label=k + 1)
    loop_w = rng.exponential(2.0, size=n).astype(np.float32)
    loop_il = rng.integers(1, k + 1, size=n).astype(np.int32)
    tot = n + a["src"].shape[0]
    rows = np.zeros(n + 1, dtype=np.int64)
    rows[1:] = np.cumsum(deg + 1)
    loop_pos = rows[:-1]
    other_pos = np.ones(tot, dtype=bool)
    other_pos[loop_pos] = False
    src = np.empty(tot, np.int32); dst = np.empty(tot, np.int32)
    il = np.empty(tot, np.int32); w = np.empty(tot, np.float32)
    src[loop_pos] = np.arange(n, dtype=np.int32); dst[loop_pos] = np.arange(n, dtype=np.int32)
    il[loop_pos] = loop_il; w[loop_pos] = loop_w
    src[other_pos] = a["src"]; dst[other_pos] = a["dst"]
    il[other_pos] = a["ilabel"]; w[other_pos] = a["weight"]
    return Graph(n, src, dst, il, np.zeros(tot, np.int32), w)


# --------------------------------------------------------------------------
# log-likelihoods
# --------------------------------------------------------------------------

def log_softmax_rows(z: np.ndarray) -> np.ndarray:
    m = z.max(axis=1, keepdims=True)
    lse = m + np.log(np.exp(z - m).sum(axis=1, keepdims=True))
    return (z - lse).astype(np.float32)


def loglikes_gauss(cfg: int, utt: int, t: int, num_labels: int, sigma: float) -> np.ndarray:
    rng = rng_for(cfg, LOGLIKES, utt)
    z = rng.normal(0.0, sigma, size=(t, num_labels))
    return np.ascontiguousarray(log_softmax_rows(z))


def loglikes_ctc(cfg: int, utt: int, t: int, num_labels: int, boost: float = 8.0,
                 p_blank: float = 0.85) -> np.ndarray:
    rng = rng_for(cfg, LOGLIKES, utt)
    z = rng.normal(0.0, 1.0, size=(t, num_labels))
    m = rng.random(t) < p_blank
    z[m, 0] += boost
    return np.ascontiguousarray(log_softmax_rows(z))


def loglikes_hmm(cfg: int, utt: int, t: int, num_labels: int, k: int, boost: float = 8.0,
                 p_blank: float = 0.85) -> np.ndarray:
    """Logits N(0, 1); on frames drawn with probability p_blank one of the k
    blank-like units, drawn per frame, is raised by ``boost``."""
    rng = rng_for(cfg, LOGLIKES, utt)
    z = rng.normal(0.0, 1.0, size=(t, num_labels))
    m = np.flatnonzero(rng.random(t) < p_blank)
    z[m, rng.integers(0, k, size=t)[m]] += boost
    return np.ascontiguousarray(log_softmax_rows(z))


def batch_lengths(n_utt: int = 64, lo: int = 300, hi: int = 1500) -> np.ndarray:
    rng = rng_for(4, LOGLIKES, 10_000)
    return rng.integers(lo, hi + 1, size=n_utt)


# --------------------------------------------------------------------------
# the five workloads
# --------------------------------------------------------------------------

_graph_cache: dict = {}


def graph_for(cfg: int) -> Graph:
    key = 3 if cfg == 4 else cfg
    if key not in _graph_cache:
        _graph_cache[key] = {1: graph_cfg1, 2: graph_cfg2, 3: graph_cfg3, 5: graph_cfg5, 6: graph_cfg6}[key]()
    return _graph_cache[key]


def workload(cfg: int, n_utt: Optional[int] = None, lsd: bool = True, frame_stride: int = 1) -> Workload:
    """Config ``cfg`` (1..6).  For cfg 4, ``n_utt`` limits the number of
    utterances (default 64); for cfg 5 and 6, ``lsd`` selects label-synchronous
    (threshold 0.95) or frame-synchronous (threshold 2) decoding; cfg 6 is
    the HMM-topology stand-in (a set of blank-like units), decoded every
    ``frame_stride``-th frame."""
    g = graph_for(cfg)
    if cfg == 1:
        ll = [loglikes_gauss(1, 0, 50, 64, 2.0)]
        return Workload(1, "tiny-fsd", g, 64, ll, DecodeOpts(beam=12.0))
    if cfg == 2:
        ll = [loglikes_gauss(2, 0, 500, 2000, 3.0)]
        return Workload(2, "medium-fsd-lattice", g, 2000, ll,
                        DecodeOpts(beam=13.0, max_active=7000, lattice_beam=8.0))
    if cfg == 3:
        ll = [loglikes_gauss(3, 0, 1000, 6000, 3.0)]
        return Workload(3, "lvcsr-25m", g, 6000, ll,
                        DecodeOpts(beam=15.0, max_active=10000, lattice_beam=8.0))
    if cfg == 4:
        n = 64 if n_utt is None else n_utt
        # (a longer draw starts with the same 64 lengths)
        lens = batch_lengths(max(64, n))
        ll = [loglikes_gauss(4, u, int(lens[u]), 6000, 3.0) for u in range(n)]
        return Workload(4, "lvcsr-25m-batch%d" % n, g, 6000, ll,
                        DecodeOpts(beam=15.0, max_active=10000, lattice_beam=8.0))
    if cfg == 5:
        ll = [loglikes_ctc(5, 0, 2000, 80)]
        thr = 0.95 if lsd else 2.0
        return Workload(5, "ctc-lsd" if lsd else "ctc-fsd", g, 80, ll,
                        DecodeOpts(beam=14.0, max_active=8000, lattice_beam=8.0,
                                   blank_threshold=thr, blank_id=0))
    if cfg == 6:
        k = HMM_BLANK_UNITS
        ll = [loglikes_hmm(6, 0, 2000, 80, k)]
        thr = 0.95 if lsd else 2.0
        name = ("hmm-lsd" if lsd else "hmm-fsd") + ("-stride%d" % frame_stride if frame_stride > 1 else "")
        return Workload(6, name, g, 80, ll,
                        DecodeOpts(beam=14.0, max_active=8000, lattice_beam=8.0, blank_threshold=thr,
                                   blank_ids=tuple(range(k)), frame_stride=frame_stride))
    raise ValueError("cfg must be 1..6")


# --------------------------------------------------------------------------
# small graphs for pins, fuzz and tie forcing
# --------------------------------------------------------------------------

# float32 values at the edges of the number format: signed zeros, the
# smallest subnormal, a mid subnormal, the largest subnormal, the smallest
# normal, and small dyadics (so sums of them tie exactly)
EDGE_WEIGHTS = np.array([0.0, -0.0, 1e-45, -1e-45, 2.9e-39, 1.1754942e-38, 1.17549435e-38, 0.5, 1.0, 0.0],
                        np.float32)
EDGE_LOGLIKES = np.array([0.0, -0.0, -1e-45, 1e-45, -2.9e-39, -1.1754942e-38, -1.17549435e-38, -0.5, -1.0,
                          -np.inf], np.float32)


def random_small_graph(seed: int, n: int, mean_deg: float = 2.0, eps_frac: float = 0.2,
                       num_labels: int = 4, weights: str = "exp",
                       final: bool = False) -> Graph:
    """Small random WFST.  ``weights``: "exp" (Exp(1) float32), "int"
    (integers 0..3, forcing cost ties), "dyadic" (multiples of 1/16 in
    [0, 4), exact in float32 sums of modest length) or "edge" (float32
    special values: signed zeros, subnormals, the smallest normal and a few
    small dyadics; epsilon arcs draw only the non-negative ones)."""
    rng = np.random.default_rng(np.random.SeedSequence([1808, 687, 99, seed]))
    deg = rng.poisson(mean_deg, size=n)
    src = np.repeat(np.arange(n), deg)
    e = src.shape[0]
    is_eps = (rng.random(e) < eps_frac) & (src < n - 1)
    u = rng.random(e)
    dst = np.where(is_eps, src + 1 + (u * (n - 1 - src)).astype(np.int64),
                   (u * n).astype(np.int64))
    dst = np.minimum(dst, n - 1)
    il = np.where(is_eps, 0, rng.integers(1, num_labels + 1, size=e))
    if weights == "exp":
        w = rng.exponential(1.0, size=e).astype(np.float32)
    elif weights == "int":
        w = rng.integers(0, 4, size=e).astype(np.float32)
    elif weights == "dyadic":
        w = (rng.integers(0, 64, size=e) / 16.0).astype(np.float32)
    elif weights == "edge":
        w = EDGE_WEIGHTS[rng.integers(0, EDGE_WEIGHTS.size, size=e)]
        w = np.where(is_eps & (w < 0), -w, w).astype(np.float32)
    else:
        raise ValueError(weights)
    fw = None
    if final:
        fw = np.where(rng.random(n) < 0.5, rng.integers(0, 4, size=n).astype(np.float32),
                      np.float32(np.inf)).astype(np.float32)
    return Graph(n, src.astype(np.int32), dst.astype(np.int32), il.astype(np.int32),
                 np.zeros(e, np.int32), w, 0, fw)


def closure_shapes_graph(seed: int, num_labels: int = 5) -> Graph:
    """A graph of epsilon structures around the sizes where a decoder may
    switch between precomputed closure lists and arc-by-arc relaxation:
    epsilon chains of 1 to 12 arcs, and two-level fans whose heads have 2 to
    300 epsilon paths (k arcs to states with m epsilon arcs each, k (m + 1)
    paths), some with chains behind their leaves.  Epsilon arcs go to higher
    state ids (the graph is epsilon-acyclic); every state also has one to
    three emitting arcs to uniformly drawn states, and the start state has an
    emitting arc to every structure's head.  Weights are Exp(1) in float32."""
    rng = np.random.default_rng(np.random.SeedSequence([1808, 687, 95, seed]))
    eps_arcs = []   # (src, dst)
    heads = []
    nxt = [1]       # state 0 is the start state

    def new_state():
        nxt[0] += 1
        return nxt[0] - 1

    def chain(length, head=None):
        a = new_state() if head is None else head
        h = a
        for _ in range(length):
            b = new_state()
            eps_arcs.append((a, b))
            a = b
        return h

    for length in (1, 2, 5, 6, 8, 9, 10, 12):
        heads.append(chain(length))
    for k, m, tail in ((1, 1, 0), (16, 15, 0), (16, 16, 0), (8, 31, 0), (2, 127, 0), (1, 255, 0), (1, 256, 0),
                       (3, 4, 7), (4, 2, 6), (20, 14, 0)):
        a = new_state()
        heads.append(a)
        for _ in range(k):
            b = new_state()
            eps_arcs.append((a, b))
            for _ in range(m):
                c = new_state()
                eps_arcs.append((b, c))
                if tail:
                    chain(tail, head=c)
    n = nxt[0]
    src = [np.asarray([e[0] for e in eps_arcs], np.int64)]
    dst = [np.asarray([e[1] for e in eps_arcs], np.int64)]
    il = [np.zeros(len(eps_arcs), np.int64)]
    deg = rng.integers(1, 4, size=n)
    es = np.repeat(np.arange(n), deg)
    src.append(es)
    dst.append(rng.integers(0, n, size=es.size))
    il.append(rng.integers(1, num_labels + 1, size=es.size))
    hs = np.asarray(heads, np.int64)
    src.append(np.zeros(hs.size, np.int64))
    dst.append(hs)
    il.append(rng.integers(1, num_labels + 1, size=hs.size))
    src, dst, il = np.concatenate(src), np.concatenate(dst), np.concatenate(il)
    w = rng.exponential(1.0, size=src.size).astype(np.float32)
    order = np.argsort(src, kind="stable")
    return Graph(n, src[order].astype(np.int32), dst[order].astype(np.int32), il[order].astype(np.int32),
                 np.zeros(src.size, np.int32), w[order])


def random_small_hmm_graph(seed: int, k: int, n: int = 400) -> Graph:
    """A small graph whose every state has a self-loop on one of k
    blank-like units (columns 0..k-1, one per phone of an HMM topology);
    its other emitting arcs read columns k..k+5."""
    g = random_small_graph(seed, n, mean_deg=2.0, eps_frac=0.1, num_labels=6)
    rng = np.random.default_rng(np.random.SeedSequence([1808, 687, 97, seed]))
    src = np.concatenate([np.arange(n), g.src]).astype(np.int32)
    dst = np.concatenate([np.arange(n), g.dst]).astype(np.int32)
    il = np.concatenate([rng.integers(1, k + 1, size=n), np.where(g.ilabel == 0, 0, g.ilabel + k)]).astype(np.int32)
    w = np.concatenate([np.full(n, 0.5), g.weight]).astype(np.float32)
    order = np.argsort(src, kind="stable")
    return Graph(n, src[order], dst[order], il[order], np.zeros_like(src), w[order])


def random_small_hmm_loglikes(seed: int, t: int, k: int) -> np.ndarray:
    """log-softmax rows over k + 6 units; on about 70% of the frames one
    blank-like unit, drawn at random, is raised by 7."""
    rng = np.random.default_rng(np.random.SeedSequence([1808, 687, 96, seed]))
    z = rng.normal(0.0, 1.0, size=(t, k + 6))
    hot = rng.random(t) < 0.7
    z[np.flatnonzero(hot), rng.integers(0, k, size=t)[hot]] += 7.0
    return np.ascontiguousarray(log_softmax_rows(z))


def random_small_loglikes(seed: int, t: int, num_labels: int, kind: str = "gauss",
                          blank_boost: float = 0.0) -> np.ndarray:
    """``kind``: "gauss" (log-softmax of N(0,2)), "int" (negative integers
    0..-3, forcing ties), "dyadic" (multiples of -1/16 in (-4, 0]) or "edge"
    (float32 special values, -inf included, and one column that is -inf on
    every frame)."""
    rng = np.random.default_rng(np.random.SeedSequence([1808, 687, 98, seed]))
    if kind == "gauss":
        z = rng.normal(0.0, 2.0, size=(t, num_labels))
        if blank_boost:
            m = rng.random(t) < 0.6
            z[m, 0] += blank_boost
        return np.ascontiguousarray(log_softmax_rows(z))
    if kind == "int":
        return np.ascontiguousarray(-rng.integers(0, 4, size=(t, num_labels)).astype(np.float32))
    if kind == "dyadic":
        return np.ascontiguousarray((-rng.integers(0, 64, size=(t, num_labels)) / 16.0).astype(np.float32))
    if kind == "edge":
        x = EDGE_LOGLIKES[rng.integers(0, EDGE_LOGLIKES.size, size=(t, num_labels))]
        if num_labels > 1:
            x[:, int(rng.integers(0, num_labels))] = -np.inf
        return np.ascontiguousarray(x.astype(np.float32))
    raise ValueError(kind)
