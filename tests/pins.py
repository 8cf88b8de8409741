"""Independent checkers that pin the oracle to the mathematics.

Nothing here calls the oracle or the GPU decoder; the tests compare their
outputs with these:

* ``brute_force``: enumerates every path of a tiny WFST (epsilon arcs
  acyclic) and accumulates costs in float32 in path order.  Because
  x -> fl(x + w) and x -> fl(x - l) are monotone, the minimum over paths of
  the forward-accumulated cost equals the dynamic-programming value bit for
  bit, so with an infinite beam the best cost of a Viterbi decoder must
  match it exactly.
* ``dense_viterbi``: exact Viterbi (no pruning) over all states at once with
  numpy float32 min-plus, epsilon arcs relaxed level by level in
  topological order of the acyclic epsilon subgraph.
* ``f32`` helpers for float32 ordered keys.
"""
from __future__ import annotations

import numpy as np

EMPTY = np.uint64(0xFFFFFFFFFFFFFFFF)


def okeys(c: np.ndarray) -> np.ndarray:
    """float32 array -> uint32 keys whose unsigned order is the numeric order."""
    u = np.ascontiguousarray(c, dtype=np.float32).view(np.uint32)
    return np.where(u >> np.uint32(31), ~u, u | np.uint32(0x80000000)).astype(np.uint32)


def okey_value(k: np.ndarray) -> np.ndarray:
    k = np.asarray(k, dtype=np.uint32)
    u = np.where(k >> np.uint32(31), k & np.uint32(0x7FFFFFFF), ~k).astype(np.uint32)
    return u.view(np.float32)


def f32(x) -> np.float32:
    return np.float32(x)


# --------------------------------------------------------------------------
# brute force
# --------------------------------------------------------------------------

def _adjacency(g):
    n = g.num_states
    out = [[] for _ in range(n)]
    for a in range(g.num_arcs):
        out[int(g.src[a])].append(a)
    return out


def brute_force(g, ll_kept: np.ndarray, max_paths: int = 2_000_000):
    """Enumerate all paths from the start state through T' = len(ll_kept)
    emitting arcs (epsilon arcs anywhere).

    Returns dict with:
      ``prefix``: {(j, s): min float32 cost of reaching s at token set j}
      ``complete``: list of (total float32 cost incl. final weight, arcs tuple,
                    frames tuple (token set index of each arc's source))
    """
    out = _adjacency(g)
    Tp = ll_kept.shape[0]
    prefix = {}
    complete = []
    fw = g.final
    count = [0]

    def visit(j, s, c, arcs, frames):
        count[0] += 1
        if count[0] > max_paths:
            raise RuntimeError("too many paths")
        k = (j, s)
        if k not in prefix or okeys(np.array([c]))[0] < okeys(np.array([prefix[k]]))[0]:
            prefix[k] = c
        if j == Tp:
            f = f32(0.0) if fw is None else f32(fw[s])
            complete.append((f32(c + f), arcs, frames))
        for a in out[s]:
            il = int(g.ilabel[a])
            w = f32(g.weight[a])
            d = int(g.dst[a])
            if il == 0:
                visit(j, d, f32(c + w), arcs + (a,), frames + (j,))
            elif j < Tp:
                t1 = f32(c + w)
                visit(j + 1, d, f32(t1 - f32(ll_kept[j, il - 1])), arcs + (a,), frames + (j,))

    visit(0, int(g.start), f32(0.0), (), ())
    return dict(prefix=prefix, complete=complete)


def path_cost(g, arcs, ll_kept) -> np.float32:
    """Forward-accumulated float32 cost of an arc sequence (no final weight)."""
    c = f32(0.0)
    j = 0
    for a in arcs:
        w = f32(g.weight[a])
        il = int(g.ilabel[a])
        if il == 0:
            c = f32(c + w)
        else:
            t1 = f32(c + w)
            c = f32(t1 - f32(ll_kept[j, il - 1]))
            j += 1
    return c


def is_valid_path(g, arcs, n_emit: int, end_state: int) -> bool:
    s = int(g.start)
    ne = 0
    for a in arcs:
        if int(g.src[a]) != s:
            return False
        if int(g.ilabel[a]) != 0:
            ne += 1
        s = int(g.dst[a])
    return ne == n_emit and s == end_state


# --------------------------------------------------------------------------
# exact dense Viterbi
# --------------------------------------------------------------------------

def eps_levels(g):
    """Topological levels of the epsilon subgraph: every epsilon arc goes
    from a lower level to a higher one.  Returns a list of arc-index arrays,
    the epsilon arcs leaving the states of each level."""
    n = g.num_states
    eps = np.flatnonzero(g.ilabel == 0)
    src = g.src[eps].astype(np.int64)
    dst = g.dst[eps].astype(np.int64)
    indeg = np.bincount(dst, minlength=n)
    level = np.full(n, -1, dtype=np.int64)
    frontier = np.flatnonzero(indeg == 0)
    order = np.argsort(src, kind="stable")
    src_s, dst_s = src[order], dst[order]
    starts = np.searchsorted(src_s, np.arange(n + 1))
    lv = 0
    remaining = indeg.copy()
    while frontier.size:
        level[frontier] = lv
        # arcs out of the frontier
        seg = [np.arange(starts[s], starts[s + 1]) for s in frontier if starts[s + 1] > starts[s]]
        if not seg:
            break
        idx = np.concatenate(seg)
        d = dst_s[idx]
        np.subtract.at(remaining, d, 1)
        cand = np.unique(d)
        frontier = cand[remaining[cand] == 0]
        lv += 1
    assert (level >= 0).all(), "epsilon subgraph has a cycle"
    arc_level = level[src]
    return [eps[arc_level == k] for k in range(lv)]


def _pack(c: np.ndarray, arcs: np.ndarray) -> np.ndarray:
    return (okeys(c).astype(np.uint64) << np.uint64(32)) | (arcs.astype(np.uint64) + np.uint64(1))


def _cost(tok: np.ndarray) -> np.ndarray:
    return okey_value((tok >> np.uint64(32)).astype(np.uint32))


def dense_viterbi(g, ll_kept: np.ndarray):
    """Exact Viterbi with no pruning.  Returns a list over token sets
    j = 0..T' of (states, cost float32, back-pointer arc) sorted by state."""
    n = g.num_states
    levels = eps_levels(g)
    emit = np.flatnonzero(g.ilabel != 0)
    e_src = g.src[emit]
    e_dst = g.dst[emit]
    e_w = g.weight[emit].astype(np.float32)
    e_col = g.ilabel[emit].astype(np.int64) - 1

    def close(tok):
        for arcs in levels:
            s = g.src[arcs]
            have = tok[s] != EMPTY
            arcs = arcs[have]
            if arcs.size == 0:
                continue
            c = _cost(tok[g.src[arcs]])
            cand = (c + g.weight[arcs].astype(np.float32)).astype(np.float32)
            np.minimum.at(tok, g.dst[arcs], _pack(cand, arcs))
        return tok

    def export(tok):
        st = np.flatnonzero(tok != EMPTY)
        t = tok[st]
        c = _cost(t)
        fin = np.isfinite(c)
        st, t, c = st[fin], t[fin], c[fin]
        return st.astype(np.int32), c, ((t & np.uint64(0xFFFFFFFF)).astype(np.int64) - 1).astype(np.int32)

    tok = np.full(n, EMPTY, dtype=np.uint64)
    tok[g.start] = np.uint64(okeys(np.array([0.0], np.float32))[0]) << np.uint64(32)
    tok = close(tok)
    sets = [export(tok)]
    for j in range(ll_kept.shape[0]):
        prev = tok
        have = prev[e_src] != EMPTY
        c = _cost(prev[e_src[have]])
        t1 = (c + e_w[have]).astype(np.float32)
        cand = (t1 - ll_kept[j][e_col[have]]).astype(np.float32)
        tok = np.full(n, EMPTY, dtype=np.uint64)
        np.minimum.at(tok, e_dst[have], _pack(cand, emit[have]))
        tok = close(tok)
        sets.append(export(tok))
    return sets
