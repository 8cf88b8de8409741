"""The allocation-free entry point (wfst_decode_noalloc) against wfst_decode.

The no-allocation call decodes into a fixed workspace and caller-owned
buffers; its outputs must be bit-identical to those of wfst_decode on the
same inputs: best path, frames, cost, final state, counters and the pruned
lattice.  Two calls in a row on one device share the workspace, the second
with a smaller input, so whatever the first left behind must not leak into
the second.
"""
import os
import sys

import numpy as np
import pytest

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


def _same(ref, got, tag):
    """wfst_decode's result against wfst_decode_noalloc's outputs."""
    assert got.rc == ref.status == got.status, (tag, got.rc, ref.status, got.status)
    if ref.status != 0:
        return
    assert got.num_decoded == ref.num_decoded, tag
    assert parity.bits(got.cost) == parity.bits(ref.cost), (tag, got.cost, ref.cost)
    assert got.final_state == ref.final_state and got.reached_final == ref.reached_final, tag
    n = got.path_len
    assert n == ref.path_arcs.size, tag
    np.testing.assert_array_equal(got.path_arcs[:n].cpu().numpy(), ref.path_arcs, err_msg=tag)
    np.testing.assert_array_equal(got.path_frames[:n].cpu().numpy(), ref.path_frames, err_msg=tag)
    if got.kept.numel() >= ref.num_decoded and ref.num_decoded:
        np.testing.assert_array_equal(got.kept[:ref.num_decoded].cpu().numpy(), ref.kept, err_msg=tag)
    for f in ("tokens", "arcs_expanded", "eps_arcs"):
        assert getattr(got, f) == ref.stats[f], (tag, f)
    if ref.lat_arc is not None:
        assert got.lattice_raw == ref.stats["lattice_raw"], tag
        m = got.lattice_n
        assert m == ref.lat_arc.size, tag
        lat = got.lattice[:m].cpu().numpy()
        np.testing.assert_array_equal(lat[:, 0], ref.lat_frame, err_msg=tag)
        np.testing.assert_array_equal(lat[:, 1], ref.lat_arc, err_msg=tag)
        np.testing.assert_array_equal(lat[:, 2].view(np.uint32), parity.bits(ref.lat_cost), err_msg=tag)
        np.testing.assert_array_equal(lat[:, 3].view(np.uint32), parity.bits(ref.lat_extra), err_msg=tag)


def test_noalloc_matches_decode_two_calls(dec):
    # the medium graph (1M arcs, max-active 7,000, lattice beam 8): a call of
    # 120 frames, then one of 45 frames into the same output buffers
    wl = W.workload(2)
    o = wl.opts
    gh = dec.load_graph(wl.graph)
    outs = None
    for T in (120, 45):
        x = _dev(wl.loglikes[0][:T])
        say("config 2, %d frames" % T)
        ref = dec.wfst_decode(gh, x, o.beam, o.max_active, o.lattice_beam)
        got = dec.wfst_decode_noalloc(gh, x, o.beam, o.max_active, o.lattice_beam, path_cap=2048,
                                      lattice_cap=1 << 18, kept_cap=4096, outputs=outs)
        _same(ref, got, "config 2 T=%d" % T)
        outs = (got.path_arcs, got.path_frames, got.lattice, got.kept)
    gh.free()


def test_noalloc_matches_decode_lsd_and_small_graphs(dec):
    # label-synchronous decoding (kept frames) on a small CTC-like graph, then
    # small random graphs with final weights and ties, each call smaller than
    # the one before
    g = W.random_small_graph(950, 5000, mean_deg=2.0, eps_frac=0.1, num_labels=30)
    n = g.num_states
    src = np.concatenate([np.arange(n), g.src]).astype(np.int32)
    dst = np.concatenate([np.arange(n), g.dst]).astype(np.int32)
    il = np.concatenate([np.ones(n), np.where(g.ilabel == 0, 0, np.maximum(g.ilabel, 2))]).astype(np.int32)
    w = np.concatenate([np.full(n, 0.3), g.weight]).astype(np.float32)
    order = np.argsort(src, kind="stable")
    g2 = W.Graph(n, src[order], dst[order], il[order], np.zeros_like(src), w[order])
    gh = dec.load_graph(g2)
    ll = W.random_small_loglikes(951, 300, 30, blank_boost=7.0)
    for T, thr in ((300, 0.95), (120, 0.5), (40, 2.0)):
        x = _dev(ll[:T])
        ref = dec.wfst_decode(gh, x, 10.0, 400, 6.0, blank_threshold=thr)
        got = dec.wfst_decode_noalloc(gh, x, 10.0, 400, 6.0, blank_threshold=thr, kept_cap=T)
        _same(ref, got, "lsd T=%d thr %g" % (T, thr))
    gh.free()
    for seed in range(6):
        gs = W.random_small_graph(1500 + seed, 300, mean_deg=3.0, eps_frac=0.3, num_labels=5, weights="int",
                                  final=seed % 2 == 0)
        h = dec.load_graph(gs)
        for T in (40, 13):
            x = _dev(W.random_small_loglikes(1500 + seed, T, 5, kind="int"))
            ref = dec.wfst_decode(h, x, 9.0, [0, 11][seed % 2], 3.0)
            got = dec.wfst_decode_noalloc(h, x, 9.0, [0, 11][seed % 2], 3.0, kept_cap=T)
            _same(ref, got, "small seed %d T=%d" % (seed, T))
        h.free()


def test_noalloc_limits(dec):
    # an output buffer that is too small: WFST_ECAPACITY with the size needed;
    # more frames than the fixed workspace holds: WFST_ECAPACITY; a forbidden
    # flag: WFST_EINVAL
    wl = W.workload(1)
    o = wl.opts
    gh = dec.load_graph(wl.graph)
    x = _dev(wl.loglikes[0])
    ref = dec.wfst_decode(gh, x, o.beam, 300, 6.0)
    got = dec.wfst_decode_noalloc(gh, x, o.beam, 300, 6.0, path_cap=3, lattice_cap=1 << 16)
    assert got.rc == dec.WFST_ECAPACITY and got.path_len == ref.path_arcs.size
    got = dec.wfst_decode_noalloc(gh, x, o.beam, 300, 6.0, path_cap=4096, lattice_cap=2)
    assert got.rc == dec.WFST_ECAPACITY and got.lattice_n == ref.lat_arc.size
    got = dec.wfst_decode_noalloc(gh, x, o.beam, 300, 6.0, path_cap=4096, lattice_cap=1 << 16)
    _same(ref, got, "config 1 after the refused calls")
    # a workspace for this many frames does not fit (a check on the host,
    # before anything runs)
    import torch
    big = torch.zeros((1 << 20, 64), dtype=torch.float32, device="cuda:0")
    got = dec.wfst_decode_noalloc(gh, big, o.beam, 300, -1.0)
    assert got.rc == dec.WFST_ECAPACITY
    del big
    gh.free()
