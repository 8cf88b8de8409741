"""The word-sequence map of a lattice (oracle/word_lattice.py), pinned:
its best entry is the decode's best cost and path, and on lattices kept
whole it equals the same map computed over every path of the graph."""
import numpy as np
import pytest

import oracle
from oracle import word_lattice as WL
from paper_1808_00687_amd import workloads as W

INF = float("inf")


def tiny(seed, n=9, final=False):
    g = W.random_small_graph(3000 + seed, n, mean_deg=2.2, eps_frac=0.25, num_labels=3, final=final)
    rng = np.random.default_rng(3000 + seed)
    # words on about half of the arcs, from a small vocabulary so that
    # different paths share word sequences
    g.olabel = np.where(rng.random(g.src.size) < 0.5, rng.integers(1, 4, size=g.src.size), 0).astype(np.int32)
    return g


def bits(x):
    return np.float32(x).view(np.uint32)


@pytest.mark.parametrize("seed", range(12))
def test_best_word_sequence_is_the_decode_best_path(seed):
    g = tiny(seed, final=seed % 3 == 2)
    ll = W.random_small_loglikes(3100 + seed, 4, 3)
    for beam, lb in ((INF, INF), (4.0, 2.0)):
        o = oracle.decode(g, ll, beam, 0, lb)
        if o.status != 0:
            continue
        m = WL.word_costs(g, ll, o)
        words = tuple(int(g.olabel[a]) for a in o.path_arcs if g.olabel[a] != 0)
        assert words in m
        assert bits(m[words]) == bits(o.cost)
        assert bits(min(m.values())) == bits(o.cost)


@pytest.mark.parametrize("seed", range(12))
def test_whole_lattice_holds_every_path_of_the_graph(seed):
    g = tiny(seed, final=seed % 4 == 1)
    ll = W.random_small_loglikes(3200 + seed, 3 + seed % 3, 3)
    o = oracle.decode(g, ll, INF, 0, INF)
    full = WL.graph_word_costs(g, ll)
    if o.status != 0:
        assert not full
        return
    m = WL.word_costs(g, ll, o)
    assert set(m) == set(full)
    for k in m:
        assert bits(m[k]) == bits(full[k]), k


def test_kept_frames_of_label_synchronous_decoding():
    g = tiny(5)
    ll = W.random_small_loglikes(3300, 6, 3, blank_boost=6.0)
    o = oracle.decode(g, ll, INF, 0, INF, blank_threshold=0.9)
    assert o.status == 0 and 0 < o.num_decoded < 6
    m = WL.word_costs(g, ll, o)
    full = WL.graph_word_costs(g, ll, frames=o.kept)
    assert set(m) == set(full)
    assert all(bits(m[k]) == bits(full[k]) for k in m)


def test_without_output_labels_one_empty_sequence():
    g = tiny(7)
    g.olabel = np.zeros_like(g.olabel)
    ll = W.random_small_loglikes(3400, 4, 3)
    o = oracle.decode(g, ll, INF, 0, INF)
    assert o.status == 0
    m = WL.word_costs(g, ll, o)
    assert list(m) == [()]
    assert bits(m[()]) == bits(o.cost)


def test_pruned_lattice_is_a_subset():
    # lattice-beam pruning drops paths, never invents them or lowers a cost
    g = tiny(3)
    ll = W.random_small_loglikes(3500, 5, 3)
    whole = WL.word_costs(g, ll, oracle.decode(g, ll, INF, 0, INF))
    pruned = WL.word_costs(g, ll, oracle.decode(g, ll, INF, 0, 1.0))
    assert set(pruned) <= set(whole)
    assert all(pruned[k] >= whole[k] for k in pruned)
    assert len(pruned) < len(whole)
