"""Word sequences of a state-level lattice and their best costs (TEST
INFRASTRUCTURE ONLY, like the rest of oracle/).

The paper decodes into exact lattices (Sec. 1, after Povey et al. 2012,
which it cites): a lattice from which, for every word sequence it holds, the
best path with that word sequence can be read.  The word-level lattice that
determinisation over the output labels produces is therefore fixed by one
function, and this module writes that function out by brute force, for small
cases only:

  word_costs(lattice)  maps each word sequence (the non-zero output labels
                       along a complete path, in order) to the smallest cost
                       of a complete path of the lattice that outputs it.

Costs follow the decoder's arithmetic step by step in float32: an emitting
arc read in decoded frame j turns cost c into fl(fl(c + w) - ll[kept[j]][i-1]),
an epsilon arc into fl(c + w), and a path ends with fl(c + f(s)) (f = 0
without final weights, and when final weights exist but the last token set
holds no final state).  ``graph_word_costs`` computes the same map from the
graph alone, by enumerating every path, so the two check each other.
"""
from __future__ import annotations

from typing import Dict, Optional, Tuple

import numpy as np

f32 = np.float32


def _final_costs(g, states, costs):
    """Final cost of each (state, cost) at the end of the utterance, by the
    decoder's rule (Alg. 1's final transition, with the all-final fallback)."""
    fw = getattr(g, "final", None)
    if fw is None:
        return [f32(c) + f32(0.0) for c in costs], True
    tot = [f32(c) + f32(fw[s]) for s, c in zip(states, costs)]
    if any(np.isfinite(t) for t in tot):
        return tot, True
    return [f32(c) + f32(0.0) for c in costs], False


def word_costs(g, loglikes: np.ndarray, res, max_paths: int = 200000) -> Dict[Tuple[int, ...], np.float32]:
    """Best cost of each word sequence of the pruned lattice of ``res`` (an
    oracle decode result with a lattice).  Nodes are (token set j, state);
    an emitting lattice arc of set j goes to set j + 1, an epsilon arc stays
    in set j; complete paths start at (0, start) and end in the last set."""
    ll = np.asarray(loglikes, dtype=np.float32)
    Tp = int(res.num_decoded)
    kept = np.arange(Tp, dtype=np.int64) if res.kept is None else np.asarray(res.kept, np.int64)
    out_arcs: Dict[Tuple[int, int], list] = {}
    for j, a in zip(np.asarray(res.lat_frame).tolist(), np.asarray(res.lat_arc).tolist()):
        s = int(g.src[a])
        out_arcs.setdefault((j, s), []).append(a)
    best: Dict[Tuple[int, ...], np.float32] = {}
    ends = []   # (state, cost, words) of complete paths
    stack = [(0, int(g.start), f32(0.0), ())]
    n_paths = 0
    while stack:
        j, s, c, words = stack.pop()
        if j == Tp:
            ends.append((s, c, words))
            n_paths += 1
            if n_paths > max_paths:
                raise ValueError("too many paths for the brute-force word map")
        for a in out_arcs.get((j, s), ()):
            w = f32(g.weight[a])
            il = int(g.ilabel[a])
            ol = int(g.olabel[a])
            nw = words + ((ol,) if ol != 0 else ())
            if il == 0:
                stack.append((j, int(g.dst[a]), f32(c + w), nw))
            elif j < Tp:
                stack.append((j + 1, int(g.dst[a]), f32(f32(c + w) - ll[kept[j], il - 1]), nw))
    # whether final weights apply was decided over the whole last token set
    fw = getattr(g, "final", None)
    if fw is None or res.reached_final == 0:
        tot = [f32(e[1]) + f32(0.0) for e in ends]
    else:
        tot = [f32(e[1]) + f32(fw[e[0]]) for e in ends]
    for (s, c, words), t in zip(ends, tot):
        if not np.isfinite(t):
            continue
        if words not in best or t < best[words]:
            best[words] = f32(t)
    return best


def graph_word_costs(g, loglikes: np.ndarray, frames: Optional[np.ndarray] = None,
                     max_paths: int = 200000) -> Dict[Tuple[int, ...], np.float32]:
    """The same map over every path of the graph itself (no beam, no
    pruning): ``frames`` lists the decoded frames (all frames by default).
    A path reads one decoded frame per emitting arc, with epsilon arcs
    anywhere in between and after the last frame."""
    ll = np.asarray(loglikes, dtype=np.float32)
    kept = np.arange(ll.shape[0], dtype=np.int64) if frames is None else np.asarray(frames, np.int64)
    Tp = kept.shape[0]
    order = np.argsort(g.src, kind="stable")
    out_arcs: Dict[int, list] = {}
    for a in order.tolist():
        out_arcs.setdefault(int(g.src[a]), []).append(a)
    ends = []
    stack = [(0, int(g.start), f32(0.0), ())]
    n_paths = 0
    while stack:
        j, s, c, words = stack.pop()
        if j == Tp:
            ends.append((s, c, words))
            n_paths += 1
            if n_paths > max_paths:
                raise ValueError("too many paths for the brute-force word map")
        for a in out_arcs.get(s, ()):
            w = f32(g.weight[a])
            il = int(g.ilabel[a])
            ol = int(g.olabel[a])
            nw = words + ((ol,) if ol != 0 else ())
            if il == 0:
                stack.append((j, int(g.dst[a]), f32(c + w), nw))
            elif j < Tp:
                stack.append((j + 1, int(g.dst[a]), f32(f32(c + w) - ll[kept[j], il - 1]), nw))
    tot, _ = _final_costs(g, [e[0] for e in ends], [e[1] for e in ends])
    best: Dict[Tuple[int, ...], np.float32] = {}
    for (s, c, words), t in zip(ends, tot):
        if not np.isfinite(t):
            continue
        if words not in best or t < best[words]:
            best[words] = f32(t)
    return best
