"""Word-level lattice on the GPU (WFST_WORD_LATTICE) against the oracle's
brute-force word-sequence map (oracle/word_lattice.py): the same word
sequences, each with the same float32 cost bit for bit, on small graphs
(beams finite and infinite, final weights, label-synchronous frame
skipping, batches) and on the medium 1M-arc graph with output labels on
30% of its arcs (500 frames, lattice beam 8: 285,120 word sequences)."""
import numpy as np
import pytest

from oracle import word_lattice as WL
from paper_1808_00687_amd import workloads as W
import parity

pytestmark = pytest.mark.gpu

INF = float("inf")


def say(*a):
    print(*a, flush=True)


@pytest.fixture(scope="module")
def dec():
    import torch
    assert torch.cuda.is_available(), "no GPU"
    from paper_1808_00687_amd import wfstdec
    return wfstdec


def _dev(ll):
    import torch
    return torch.from_numpy(np.ascontiguousarray(ll)).to("cuda:0")


def _tiny(seed, n=9, final=False):
    g = W.random_small_graph(3000 + seed, n, mean_deg=2.2, eps_frac=0.25, num_labels=3, final=final)
    rng = np.random.default_rng(3000 + seed)
    g.olabel = np.where(rng.random(g.src.size) < 0.5, rng.integers(1, 4, size=g.src.size), 0).astype(np.int32)
    return g


def _same_map(exp, got, tag):
    """exp: {words: float32} from the oracle; got: [(words, float32)] from the GPU."""
    gm = {}
    for w, c in got:
        assert w not in gm, (tag, "sequence listed twice", w)
        gm[w] = c
    assert set(gm) == set(exp), (tag, len(gm), len(exp), sorted(set(exp) ^ set(gm))[:5])
    for w, c in exp.items():
        assert parity.bits(gm[w]) == parity.bits(c), (tag, w, gm[w], c)
    # sorted by cost key, then by the sequence
    keys = [(int(np.uint32(parity.bits(c))) ^ (0xFFFFFFFF if parity.bits(c) >> 31 else 0x80000000), w)
            for w, c in got]
    assert keys == sorted(keys), tag


@pytest.mark.parametrize("seed", range(16))
def test_small_lattices(dec, oracle_mod, seed):
    g = _tiny(seed, n=[9, 12, 20, 40][seed % 4], final=seed % 3 == 2)
    ll = W.random_small_loglikes(3100 + seed, 3 + seed % 5, 3)
    gh = dec.load_graph(g)
    for beam, ma, lb in ((INF, 0, INF), (4.0, 0, 2.0), (6.0, 5, 3.0), (3.0, 0, 0.0)):
        o = oracle_mod.decode(g, ll, beam, ma, lb)
        r = dec.wfst_decode(gh, _dev(ll), beam, ma, lb, word_lattice=True)
        assert r.status == o.status
        if o.status != 0:
            continue
        exp = WL.word_costs(g, ll, o)
        _same_map(exp, r.words, "seed %d beam %g lb %g" % (seed, beam, lb))
        # the best sequence is the best path's
        best_words = tuple(int(g.olabel[a]) for a in r.path_arcs if g.olabel[a] != 0)
        assert r.words[0][0] == best_words and parity.bits(r.words[0][1]) == parity.bits(r.cost)
        assert r.stats["word_sequences"] == len(exp)
    gh.free()


def test_whole_lattice_is_the_graph_map_and_lsd(dec, oracle_mod):
    # infinite beams keep every path: the map of the graph itself; with
    # label-synchronous decoding, the graph's map over the kept frames
    for seed in range(6):
        g = _tiny(20 + seed, final=seed % 2 == 1)
        ll = W.random_small_loglikes(3200 + seed, 3 + seed % 3, 3)
        gh = dec.load_graph(g)
        r = dec.wfst_decode(gh, _dev(ll), INF, 0, INF, word_lattice=True)
        full = WL.graph_word_costs(g, ll)
        if r.status != 0:
            assert not full
        else:
            _same_map(full, r.words, "whole lattice seed %d" % seed)
        gh.free()
    g = _tiny(5)
    ll = W.random_small_loglikes(3300, 6, 3, blank_boost=6.0)
    gh = dec.load_graph(g)
    r = dec.wfst_decode(gh, _dev(ll), INF, 0, INF, blank_threshold=0.9, word_lattice=True)
    assert 0 < r.num_decoded < 6
    _same_map(WL.graph_word_costs(g, ll, frames=r.kept), r.words, "lsd")
    gh.free()


def test_batch_and_no_output_labels(dec, oracle_mod):
    # a batch of 40 utterances (length groups on several streams) on one
    # graph; and a graph without output labels: one empty sequence
    g = _tiny(31, n=60, final=True)
    gh = dec.load_graph(g)
    rng = np.random.default_rng(77)
    lls = [W.random_small_loglikes(3400 + u, int(rng.integers(0, 9)), 3) for u in range(40)]
    res = dec.wfst_decode_batch(gh, [_dev(x) for x in lls], 5.0, 30, 2.5, word_lattice=True)
    for u, (x, r) in enumerate(zip(lls, res)):
        o = oracle_mod.decode(g, x, 5.0, 30, 2.5)
        assert r.status == o.status
        if o.status == 0:
            _same_map(WL.word_costs(g, x, o), r.words, "batch utt %d" % u)
    gh.free()
    g = _tiny(7)
    g.olabel = np.zeros_like(g.olabel)
    ll = W.random_small_loglikes(3500, 4, 3)
    gh = dec.load_graph(g)
    r = dec.wfst_decode(gh, _dev(ll), INF, 0, INF, word_lattice=True)
    assert [w for w, _ in r.words] == [()] and parity.bits(r.words[0][1]) == parity.bits(r.cost)
    gh.free()


def test_medium_graph_word_lattice(dec, oracle_mod):
    # the 1M-arc graph of the medium configuration with output labels on 30%
    # of its arcs (a vocabulary of 49 words): 500 frames, beam 13,
    # max-active 7,000, lattice beam 8, and shorter cases
    wl = W.workload(2)
    g = wl.graph
    rng = np.random.default_rng(5)
    g.olabel = np.where(rng.random(g.src.size) < 0.3, rng.integers(1, 50, size=g.src.size), 0).astype(np.int32)
    gh = dec.load_graph(g)
    for T, lb in ((40, 4.0), (200, 8.0), (500, 8.0)):
        ll = wl.loglikes[0][:T]
        r = dec.wfst_decode(gh, _dev(ll), 13.0, 7000, lb, word_lattice=True)
        o = oracle_mod.decode(g, ll, 13.0, 7000, lb)
        say("medium graph T=%d lattice beam %g: %d word sequences, %d lattice arcs" % (
            T, lb, len(r.words), r.stats["lattice_kept"]))
        exp = WL.word_costs(g, ll, o, max_paths=2_000_000)
        _same_map(exp, r.words, "medium T=%d lb %g" % (T, lb))
    gh.free()


def test_word_lattice_needs_a_lattice(dec):
    g = _tiny(1)
    gh = dec.load_graph(g)
    with pytest.raises(dec.WfstError) as e:
        dec.wfst_decode(gh, _dev(W.random_small_loglikes(1, 3, 3)), 5.0, 0, -1.0, word_lattice=True)
    assert e.value.code == dec.WFST_EINVAL
    gh.free()
