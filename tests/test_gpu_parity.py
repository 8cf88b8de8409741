"""GPU decoder (HIP, through the C ABI) against the CPU oracle.

Every case compares token sets (states, float32 cost bits, back-pointers),
best path, cost, counters and lattice (arcs, prefix costs, extra costs)
exactly.  Sizes span many 64-token wave chunks and ragged tails; the
workloads include the medium and LVCSR-scale graphs decoded in the same
launch configuration as the benchmark.
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
    sys.stdout.flush()


@pytest.fixture(scope="module")
def dec():
    import torch
    assert torch.cuda.is_available(), "no GPU"
    from paper_1808_00687_amd import wfstdec
    return wfstdec


@pytest.fixture(scope="module")
def torch_mod():
    import torch
    return torch


def to_dev(torch_mod, ll):
    return torch_mod.from_numpy(np.ascontiguousarray(ll)).to("cuda:0")


def both(dec, torch_mod, oracle_mod, g, ll, gh=None, tokens=True, **o):
    ro = oracle_mod.decode(g, ll, o.get("beam", INF), o.get("max_active", 0), o.get("lattice_beam", -1.0),
                           o.get("blank_threshold", 2.0), o.get("blank_id", 0), o.get("blank_ids"),
                           o.get("frame_stride", 1))
    own = gh is None
    if own:
        gh = dec.load_graph(g)
    rg = dec.wfst_decode(gh, to_dev(torch_mod, ll), beam=o.get("beam", INF), max_active=o.get("max_active", 0),
                         lattice_beam=o.get("lattice_beam", -1.0),
                         blank_threshold=o.get("blank_threshold", 2.0), blank_id=o.get("blank_id", 0),
                         record_tokens=tokens, blank_ids=o.get("blank_ids"), frame_stride=o.get("frame_stride", 1))
    if own:
        gh.free()
    return ro, rg


SMALL = []
for seed in range(60):
    kind = ["exp", "int", "dyadic"][seed % 3]
    SMALL.append((seed, kind))


@pytest.mark.parametrize("seed,kind", SMALL)
def test_small_random_graphs(dec, torch_mod, oracle_mod, seed, kind):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(5, 400))
    g = W.random_small_graph(700 + seed, n, mean_deg=float(rng.uniform(1.2, 4.0)),
                             eps_frac=float(rng.uniform(0.0, 0.4)), num_labels=5,
                             weights=kind, final=bool(seed % 4 == 1))
    T = int(rng.integers(0, 40))
    ll = W.random_small_loglikes(700 + seed, T, 5, kind={"exp": "gauss", "int": "int", "dyadic": "dyadic"}[kind])
    beam = [INF, 3.0, 6.5, 12.0][seed % 4]
    max_active = [0, 0, 5, 37, 120][seed % 5]
    lb = [-1.0, 0.0, 2.5, INF][seed % 4]
    ro, rg = both(dec, torch_mod, oracle_mod, g, ll, beam=beam, max_active=max_active, lattice_beam=lb)
    parity.assert_same(ro, rg, lattice=lb >= 0, tag="seed %d" % seed)


@pytest.mark.parametrize("L", [6145, 9000])
def test_wide_label_rows(dec, torch_mod, oracle_mod, L):
    # more log-likelihood columns than the search keeps in LDS: the emitting
    # expansion reads the row from device memory (labels spread over the
    # whole row)
    for seed in range(6):
        rng = np.random.default_rng(900 + seed)
        g = W.random_small_graph(900 + seed, int(rng.integers(20, 300)), mean_deg=2.5, eps_frac=0.3,
                                 num_labels=5, weights=["exp", "dyadic"][seed % 2], final=seed % 3 == 0)
        g.ilabel = np.where(g.ilabel > 0, rng.integers(1, L + 1, size=g.ilabel.size), 0).astype(np.int32)
        ll = rng.normal(0.0, 2.0, size=(int(rng.integers(1, 30)), L)).astype(np.float32)
        ro, rg = both(dec, torch_mod, oracle_mod, g, ll, beam=[INF, 5.0, 9.0][seed % 3],
                      max_active=[0, 20][seed % 2], lattice_beam=[3.0, INF][seed % 2])
        parity.assert_same(ro, rg, lattice=True, tag="L %d seed %d" % (L, seed))


def listed_closure_states(g, max_paths, max_len):
    """States whose epsilon closure is at most max_paths paths of at most
    max_len arcs, every child with epsilon arcs being such a state too
    (epsilon arcs of these graphs go to higher state ids)."""
    eps = g.ilabel == 0
    kids = {}
    for s, d in zip(g.src[eps].tolist(), g.dst[eps].tolist()):
        kids.setdefault(s, []).append(d)
    size, depth, listed = {}, {}, {}
    for s in sorted(kids, reverse=True):
        sz = sum(1 + size.get(d, 0) for d in kids[s])
        dp = max(1 + depth.get(d, 0) for d in kids[s])
        ok = all(listed.get(d, True) for d in kids[s])
        size[s], depth[s] = min(sz, max_paths + 1), min(dp, max_len + 1)
        listed[s] = sz <= max_paths and dp <= max_len and ok
    return sum(listed.values())


@pytest.mark.parametrize("seed", range(4))
def test_epsilon_closure_shapes(dec, torch_mod, oracle_mod, seed):
    # epsilon chains and fans just inside and just outside the sizes and
    # lengths of precomputed closure lists, with float32 weights whose sums
    # depend on the order of the additions
    g = W.closure_shapes_graph(seed)
    gh = dec.load_graph(g)
    # the library lists closures up to 256 paths of up to 9 arcs (the
    # results do not show it: they are the same either way)
    n_listed = gh.info()["num_closure_states"]
    assert n_listed == listed_closure_states(g, 256, 9)
    assert n_listed > listed_closure_states(g, 64, 5)
    ll = W.random_small_loglikes(60 + seed, 12, 5)
    for beam, max_active, lb in ((INF, 0, INF), (6.0, 400, 3.0), (2.5, 0, 1.0)):
        ro, rg = both(dec, torch_mod, oracle_mod, g, ll, gh=gh, beam=beam, max_active=max_active, lattice_beam=lb)
        parity.assert_same(ro, rg, lattice=True, tag="closure shapes %d beam %g" % (seed, beam))
    gh.free()
    say("closure shapes", seed, "listed", n_listed, "tokens", rg.stats["tokens"])


def test_config1_full(dec, torch_mod, oracle_mod):
    wl = W.workload(1)
    o = wl.opts
    for lb in (-1.0, 8.0):
        ro, rg = both(dec, torch_mod, oracle_mod, wl.graph, wl.loglikes[0], beam=o.beam,
                      max_active=o.max_active, lattice_beam=lb)
        parity.assert_same(ro, rg, lattice=lb >= 0, tag="config 1 lb %g" % lb)
        say("config 1: cost", rg.cost, "tokens", rg.stats["tokens"], "lattice", rg.stats["lattice_kept"])


@pytest.fixture(scope="module")
def cfg2(dec):
    wl = W.workload(2)
    return wl, dec.load_graph(wl.graph)


def test_config2_full(dec, torch_mod, oracle_mod, cfg2):
    wl, gh = cfg2
    o = wl.opts
    ro, rg = both(dec, torch_mod, oracle_mod, wl.graph, wl.loglikes[0], gh=gh, beam=o.beam,
                  max_active=o.max_active, lattice_beam=o.lattice_beam)
    parity.assert_same(ro, rg, lattice=True, tag="config 2")
    parity.assert_path_consistent(wl.graph, rg, wl.loglikes[0])
    say("config 2: cost", rg.cost, "arcs", rg.stats["arcs_expanded"], "lattice raw", rg.stats["lattice_raw"],
        "kept", rg.stats["lattice_kept"])


def test_config2_raw_lattice_and_infinite_beam_prefix(dec, torch_mod, oracle_mod, cfg2):
    wl, gh = cfg2
    ll = wl.loglikes[0][:30]
    ro, rg = both(dec, torch_mod, oracle_mod, wl.graph, ll, gh=gh, beam=13.0, max_active=7000,
                  lattice_beam=INF)
    parity.assert_same(ro, rg, lattice=True, tag="config 2 raw lattice")
    ro, rg = both(dec, torch_mod, oracle_mod, wl.graph, ll[:6], gh=gh, beam=INF, max_active=0,
                  lattice_beam=4.0, tokens=True)
    parity.assert_same(ro, rg, lattice=True, tag="config 2 infinite beam")


def test_epsilon_queue_overflow_path(dec, torch_mod, oracle_mod, cfg2):
    # two epsilon items per generation in LDS: the rest of the closure goes
    # through the device-memory spill lists
    wl, gh = cfg2
    with dec.debug_opts(queue_cap=2):
        ro, rg = both(dec, torch_mod, oracle_mod, wl.graph, wl.loglikes[0][:80], gh=gh, beam=13.0,
                      max_active=7000, lattice_beam=8.0)
    parity.assert_same(ro, rg, lattice=True, tag="overflow queue")


@pytest.mark.parametrize("fill", [1, 40, 700])
def test_device_memory_table_path(dec, torch_mod, oracle_mod, cfg2, fill):
    # frames reaching more than `fill` states are redone with the token table
    # in device memory (every frame for fill = 1, a mix for the others)
    wl, gh = cfg2
    with dec.debug_opts(lds_fill=fill):
        ro, rg = both(dec, torch_mod, oracle_mod, wl.graph, wl.loglikes[0][:60], gh=gh, beam=13.0,
                      max_active=7000 if fill != 40 else 300, lattice_beam=8.0)
    parity.assert_same(ro, rg, lattice=True, tag="device table fill %d" % fill)
    for seed in range(6):
        g = W.random_small_graph(900 + seed, 300, mean_deg=3.0, eps_frac=0.3, num_labels=5, weights="int",
                                 final=seed % 2 == 0)
        ll = W.random_small_loglikes(900 + seed, 25, 5, kind="int")
        with dec.debug_opts(lds_fill=fill, queue_cap=2):
            ro, rg = both(dec, torch_mod, oracle_mod, g, ll, beam=9.0, max_active=[0, 11][seed % 2],
                          lattice_beam=3.0)
        parity.assert_same(ro, rg, lattice=True, tag="device table fill %d seed %d" % (fill, seed))


@pytest.mark.parametrize("cap", [-1, 25, 3900])
def test_lattice_device_memory_path(dec, torch_mod, oracle_mod, cfg2, cap):
    # the lattice backward pass keeps token sets of at most `cap` survivors in
    # LDS and does larger ones in device memory: every set for cap = -1 (none
    # in LDS), a mix of both (and the hand-overs between them) for the others
    wl, gh = cfg2
    with dec.debug_opts(lattice_lds=cap):
        ro, rg = both(dec, torch_mod, oracle_mod, wl.graph, wl.loglikes[0][:80], gh=gh, beam=13.0,
                      max_active=7000, lattice_beam=8.0)
    parity.assert_same(ro, rg, lattice=True, tag="lattice lds %d" % cap)
    for seed in range(6):
        g = W.random_small_graph(950 + seed, 300, mean_deg=3.0, eps_frac=0.3, num_labels=5, weights="int",
                                 final=seed % 2 == 0)
        ll = W.random_small_loglikes(950 + seed, 25, 5, kind="int")
        with dec.debug_opts(lattice_lds=cap):
            ro, rg = both(dec, torch_mod, oracle_mod, g, ll, beam=9.0, max_active=[0, 11][seed % 2],
                          lattice_beam=3.0)
        parity.assert_same(ro, rg, lattice=True, tag="lattice lds %d seed %d" % (cap, seed))


@pytest.mark.parametrize("mode", [-1, 1])
def test_lattice_streamed_pass(dec, torch_mod, oracle_mod, cfg2, mode):
    # lattice pruning's streamed pass (one wave computes the nodes' extra
    # costs from an LDS ring of records that the block's other waves fill),
    # forced on wherever it fits (1) and off (-1): sets of thousands of
    # records that wrap around the ring every few sets, with epsilon rounds
    # over several pieces, and random graphs with epsilon-heavy sets of a few
    # hundred tokens
    wl, gh = cfg2
    with dec.debug_opts(lattice_pipe=mode):
        ro, rg = both(dec, torch_mod, oracle_mod, wl.graph, wl.loglikes[0][:120], gh=gh, beam=13.0,
                      max_active=7000, lattice_beam=8.0)
    parity.assert_same(ro, rg, lattice=True, tag="streamed pass %d" % mode)
    assert rg.stats["lattice_raw"] > 8192 * 4
    for seed in range(8):
        g = W.random_small_graph(1300 + seed, 600 + 200 * seed, mean_deg=3.0, eps_frac=0.35, num_labels=5,
                                 weights=["int", "exp"][seed % 2], final=seed % 3 == 0)
        ll = W.random_small_loglikes(1300 + seed, 30, 5, kind=["int", "gauss"][seed % 2])
        with dec.debug_opts(lattice_pipe=mode):
            ro, rg = both(dec, torch_mod, oracle_mod, g, ll, beam=[INF, 9.0][seed % 2],
                          max_active=[0, 300][seed % 2 if seed < 4 else 0], lattice_beam=[3.0, INF][seed % 2])
        parity.assert_same(ro, rg, lattice=True, tag="streamed pass %d seed %d" % (mode, seed))


@pytest.mark.parametrize("seed", range(30))
def test_lattice_passes_on_random_graphs(dec, torch_mod, oracle_mod, seed):
    # random graphs of 40-2,500 states with up to 45% epsilon arcs, finite
    # and infinite beams: the streamed lattice pass forced wherever it fits,
    # and the passes the rules pick otherwise, against the oracle
    rng = np.random.default_rng(seed)
    n = int(rng.integers(40, 2500))
    g = W.random_small_graph(5000 + seed, n, mean_deg=float(rng.uniform(1.5, 4.0)),
                             eps_frac=float(rng.uniform(0.0, 0.45)), num_labels=5,
                             weights=["int", "exp", "dyadic"][seed % 3], final=bool(seed % 4 == 1))
    ll = W.random_small_loglikes(5000 + seed, int(rng.integers(1, 60)), 5,
                                 kind={0: "int", 1: "gauss", 2: "dyadic"}[seed % 3])
    kw = dict(beam=[INF, 6.0, 10.0, 14.0][seed % 4], max_active=[0, 0, 50, 400][(seed // 4) % 4],
              lattice_beam=[2.0, 5.0, INF][seed % 3])
    gh = dec.load_graph(g)
    for mode in (1, 0):
        with dec.debug_opts(lattice_pipe=mode):
            ro, rg = both(dec, torch_mod, oracle_mod, g, ll, gh=gh, **kw)
        parity.assert_same(ro, rg, lattice=True, tag="seed %d lattice_pipe %d" % (seed, mode))
    gh.free()


@pytest.mark.parametrize("form", ["one-wave", "streamed"])
def test_lattice_pass_gives_up(dec, torch_mod, oracle_mod, cfg2, form):
    # the lattice passes' hand-over waits are bounded: with one poll allowed
    # (set from the host) the pass gives up, every kernel ends and the call
    # reports a device error; the next call, with the library's own limit,
    # decodes as before
    if form == "one-wave":
        g = W.random_small_graph(1500, 40, mean_deg=2.0, eps_frac=0.2, num_labels=5, weights="int")
        ll = W.random_small_loglikes(1500, 30, 5, kind="int")
        gh, kw = None, dict(beam=INF, lattice_beam=INF)
        opts = dict()
    else:
        wl, gh = cfg2
        g, ll = wl.graph, wl.loglikes[0][:60]
        kw = dict(beam=13.0, max_active=7000, lattice_beam=8.0)
        opts = dict(lattice_pipe=1)
    own = gh is None
    if own:
        gh = dec.load_graph(g)
    with dec.debug_opts(lattice_spin=1, **opts):
        with pytest.raises(dec.WfstError) as e:
            dec.wfst_decode(gh, to_dev(torch_mod, ll), kw["beam"], kw.get("max_active", 0), kw["lattice_beam"])
    assert e.value.code == dec.WFST_EDEVICE and "lattice pass stopped waiting" in str(e.value)
    with dec.debug_opts(**opts):
        ro, rg = both(dec, torch_mod, oracle_mod, g, ll, gh=gh, **kw)
    parity.assert_same(ro, rg, lattice=True, tag="after a pass that gave up (%s)" % form)
    if own:
        gh.free()


def test_lattice_output_large_sets(dec, torch_mod, oracle_mod):
    # token sets with more kept arcs than the output pass sorts in LDS (512
    # per set): every raw record kept (infinite beams) on a graph with
    # thousands of arcs per set, against the oracle
    g = W.random_small_graph(1400, 1500, mean_deg=3.0, eps_frac=0.2, num_labels=5, weights="int")
    ll = W.random_small_loglikes(1400, 12, 5, kind="int")
    ro, rg = both(dec, torch_mod, oracle_mod, g, ll, beam=INF, lattice_beam=INF)
    parity.assert_same(ro, rg, lattice=True, tag="large kept sets")
    per_set = np.bincount(np.asarray(rg.lat_frame))
    assert per_set.max() > 512 and per_set.min() >= 0


@pytest.mark.parametrize("fill,big", [(1, 1), (900, 1), (1, 1 << 20), (900, 1500)])
def test_record_large_set_path(dec, torch_mod, oracle_mod, cfg2, fill, big):
    # token sets of more than `fill` survivors get their back-pointers and
    # lattice records from the large-set pass: with its LDS table up to `big`
    # survivors, beyond that with the utterance's device-memory table (every
    # set for fill = 1, a mix for 900), alone and in a batch
    wl, gh = cfg2
    with dec.debug_opts(record_fill=fill, record_big_fill=big):
        ro, rg = both(dec, torch_mod, oracle_mod, wl.graph, wl.loglikes[0][:60], gh=gh, beam=13.0,
                      max_active=7000, lattice_beam=8.0)
        parity.assert_same(ro, rg, lattice=True, tag="record fill %d/%d" % (fill, big))
        lls = [wl.loglikes[0][:40], wl.loglikes[0][10:35]]
        res = dec.wfst_decode_batch(gh, [to_dev(torch_mod, x) for x in lls], 13.0, 7000, 8.0, record_tokens=True)
        for i, x in enumerate(lls):
            ro = oracle_mod.decode(wl.graph, x, 13.0, 7000, 8.0)
            parity.assert_same(ro, res[i], lattice=True, tag="record fill %d/%d batch %d" % (fill, big, i))


def test_capacity_retry(dec, torch_mod, oracle_mod, cfg2):
    # a capacity hint of 8 tokens per frame overflows the survivor, lattice,
    # table and candidate buffers: the library grows them and decodes again
    wl, gh = cfg2
    ll = wl.loglikes[0][:50]
    ro = oracle_mod.decode(wl.graph, ll, 13.0, 7000, 8.0)
    rg = dec.wfst_decode(gh, to_dev(torch_mod, ll), beam=13.0, max_active=7000, lattice_beam=8.0,
                         record_tokens=True, capacity_hint=8)
    parity.assert_same(ro, rg, lattice=True, tag="capacity retry")


def test_determinism(dec, torch_mod, cfg2):
    wl, gh = cfg2
    o = wl.opts
    x = to_dev(torch_mod, wl.loglikes[0][:120])
    a = dec.wfst_decode(gh, x, o.beam, o.max_active, o.lattice_beam, record_tokens=True)
    b = dec.wfst_decode(gh, x, o.beam, o.max_active, o.lattice_beam, record_tokens=True)
    for f in ("tok_off", "tok_state", "tok_arc", "path_arcs", "lat_arc", "lat_frame"):
        np.testing.assert_array_equal(getattr(a, f), getattr(b, f))
    np.testing.assert_array_equal(parity.bits(a.tok_cost), parity.bits(b.tok_cost))
    np.testing.assert_array_equal(parity.bits(a.lat_extra), parity.bits(b.lat_extra))


def test_order_permutation_is_bit_identical(dec, torch_mod, oracle_mod, cfg2):
    # another hash multiplier (other slots, claim order, probe sequences and
    # survivor order) and the arc chunks of every set expanded last to first:
    # every output must be bit-identical, and the oracle's
    wl, gh = cfg2
    o = wl.opts
    x = to_dev(torch_mod, wl.loglikes[0][:150])
    a = dec.wfst_decode(gh, x, o.beam, o.max_active, o.lattice_beam, record_tokens=True)
    with dec.debug_opts(permute=1):
        b = dec.wfst_decode(gh, x, o.beam, o.max_active, o.lattice_beam, record_tokens=True)
        with dec.debug_opts(permute=1, lds_fill=300, queue_cap=3, record_fill=200, lattice_lds=100):
            c = dec.wfst_decode(gh, x, o.beam, o.max_active, o.lattice_beam, record_tokens=True)
    ro = oracle_mod.decode(wl.graph, wl.loglikes[0][:150], o.beam, o.max_active, o.lattice_beam)
    for r, tag in ((a, "plain"), (b, "permuted"), (c, "permuted, small tables")):
        parity.assert_same(ro, r, lattice=True, tag=tag)
    for seed in range(8):
        g = W.random_small_graph(1200 + seed, 400, mean_deg=3.0, eps_frac=0.3, num_labels=5, weights="int",
                                 final=seed % 2 == 0)
        lls = [W.random_small_loglikes(1200 + 10 * seed + u, 10 + 7 * u, 5, kind="int") for u in range(5)]
        gs = dec.load_graph(g)
        with dec.debug_opts(permute=1):
            res = dec.wfst_decode_batch(gs, [to_dev(torch_mod, y) for y in lls], 9.0, [0, 13][seed % 2], 4.0,
                                        record_tokens=True)
        gs.free()
        for u, (y, r) in enumerate(zip(lls, res)):
            parity.assert_same(oracle_mod.decode(g, y, 9.0, [0, 13][seed % 2], 4.0), r, lattice=True,
                               tag="permuted seed %d utt %d" % (seed, u))


def test_incremental_lattice_pass_is_exact(dec, torch_mod, oracle_mod, cfg2):
    # WFST_INCREMENTAL_LATTICE: a pass beside the search prunes every chunk
    # of token sets against its frontier (extra cost 0 there) and keeps the
    # survivors for the final pass.  The result must be bit-identical to
    # pruning the whole lattice after the search, and the oracle's; chunks of
    # 1 and 3 sets and rings too small for a chunk (chunks end early, records
    # wrap around the ring) included.
    wl, gh = cfg2
    o = wl.opts
    ll = wl.loglikes[0][:160]
    x = to_dev(torch_mod, ll)
    ro = oracle_mod.decode(wl.graph, ll, o.beam, o.max_active, o.lattice_beam)
    whole = dec.wfst_decode(gh, x, o.beam, o.max_active, o.lattice_beam, record_tokens=True)
    parity.assert_same(ro, whole, lattice=True, tag="after the search")
    for chunk, ring in ((0, 0), (1, 0), (3, 0), (3, 90000), (32, 150000)):
        with dec.debug_opts(lattice_chunk=chunk, lattice_ring=ring):
            r = dec.wfst_decode(gh, x, o.beam, o.max_active, o.lattice_beam, record_tokens=True,
                                incremental_lattice=True)
        parity.assert_same(ro, r, lattice=True, tag="chunk %d ring %d" % (chunk, ring))
        assert r.stats["lattice_incremental"] < whole.stats["lattice_raw"]
        say("chunk %d ring %d: raw %d, kept by the incremental pass %d, final %d" % (
            chunk, ring, r.stats["lattice_raw"], r.stats["lattice_incremental"], r.stats["lattice_kept"]))
    # the switch that turns the pass off gives the one-shot path
    with dec.debug_opts(lattice_chunk=-1):
        r = dec.wfst_decode(gh, x, o.beam, o.max_active, o.lattice_beam, incremental_lattice=True)
    assert r.stats["lattice_incremental"] == r.stats["lattice_raw"]
    for seed in range(8):
        g = W.random_small_graph(1300 + seed, 300, mean_deg=3.0, eps_frac=0.3, num_labels=5, weights="int",
                                 final=seed % 2 == 0)
        lls = [W.random_small_loglikes(1300 + 10 * seed + u, 5 + 9 * u, 5, kind="int") for u in range(6)]
        gs = dec.load_graph(g)
        for chunk, ring in ((1, 0), (2, 3000), (5, 0)):
            with dec.debug_opts(lattice_chunk=chunk, lattice_ring=ring):
                res = dec.wfst_decode_batch(gs, [to_dev(torch_mod, y) for y in lls], 9.0, [0, 13][seed % 2],
                                            [INF, 2.5][seed % 2], record_tokens=True, incremental_lattice=True)
            for u, (y, r) in enumerate(zip(lls, res)):
                parity.assert_same(oracle_mod.decode(g, y, 9.0, [0, 13][seed % 2], [INF, 2.5][seed % 2]), r,
                                   lattice=True, tag="seed %d chunk %d ring %d utt %d" % (seed, chunk, ring, u))
        gs.free()


def test_lattice_alloc_failure_returns_enomem(dec, torch_mod, oracle_mod, cfg2):
    # the lattice output cannot be allocated: the call fails with WFST_ENOMEM,
    # and the next decode works
    wl, gh = cfg2
    o = wl.opts
    ll = wl.loglikes[0][:40]
    x = to_dev(torch_mod, ll)
    with dec.debug_opts(fail_lattice_alloc=1):
        with pytest.raises(dec.WfstError) as e:
            dec.wfst_decode(gh, x, o.beam, o.max_active, o.lattice_beam)
        assert e.value.code == dec.WFST_ENOMEM
        with pytest.raises(dec.WfstError) as e:
            dec.wfst_decode_batch(gh, [x, x], o.beam, o.max_active, o.lattice_beam)
        assert e.value.code == dec.WFST_ENOMEM
        # without a lattice nothing is allocated
        r = dec.wfst_decode(gh, x, o.beam, o.max_active, -1.0)
        assert r.status == 0
    r = dec.wfst_decode(gh, x, o.beam, o.max_active, o.lattice_beam, record_tokens=True)
    parity.assert_same(oracle_mod.decode(wl.graph, ll, o.beam, o.max_active, o.lattice_beam), r, lattice=True,
                       tag="after the failed allocation")


def _golden_graph(fx):
    a = np.array(fx["arcs_src_dst_ilabel_olabel_weight"], np.float64).reshape(-1, 5)
    return W.Graph(fx["num_states"], a[:, 0].astype(np.int32), a[:, 1].astype(np.int32), a[:, 2].astype(np.int32),
                   a[:, 3].astype(np.int32), a[:, 4].astype(np.float32), fx.get("start", 0))


def test_golden_cases(dec, torch_mod, oracle_mod):
    # the hand-computed cases of tests/golden on the GPU: the token sets of
    # the recombination example (and its tie variant), and the raw lattice
    # with an epsilon arc above the cutoff and two exactly at it
    import json
    here = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
    fx = json.load(open(os.path.join(here, "fig2_recombination.json")))
    ll = np.array(fx["loglikes"], np.float32)
    for variant in ("base", "tie"):
        if variant == "tie":
            fx["arcs_src_dst_ilabel_olabel_weight"][3][4] = fx["tie_variant"]["arc3_weight"]
        g = _golden_graph(fx)
        ro, rg = both(dec, torch_mod, oracle_mod, g, ll, beam=fx["beam"], lattice_beam=INF)
        parity.assert_same(ro, rg, lattice=True, tag="fig2 " + variant)
        exp = fx["tie_variant"] if variant == "tie" else fx["expected"]
        assert list(rg.path_arcs) == exp["best_path"]
        st, cb, bp = rg.token_set(2)
        assert {str(int(s)): [float(c), int(b)] for s, c, b in zip(st, cb.view(np.float32), bp)} == \
            exp["token_set_2"]
    fx = json.load(open(os.path.join(here, "eps_lattice_cutoff.json")))
    g = _golden_graph(fx)
    ll = np.array(fx["loglikes"], np.float32)
    ro, rg = both(dec, torch_mod, oracle_mod, g, ll, beam=fx["beam"], lattice_beam=INF)
    parity.assert_same(ro, rg, lattice=True, tag="epsilon cutoff")
    raw = fx["expected"]["raw_lattice_frame_arc_cost_extra"]
    assert rg.stats["lattice_raw"] == len(raw)
    assert [[int(f), int(a), float(c), float(e)] for f, a, c, e in
            zip(rg.lat_frame, rg.lat_arc, rg.lat_cost, rg.lat_extra)] == raw


@pytest.mark.parametrize("seed", range(30))
def test_fp32_edge_values(dec, torch_mod, oracle_mod, seed):
    # signed zeros, subnormal weights and log-likelihoods (a flush to zero
    # would change cost bits), -inf log-likelihood columns, +inf final
    # weights, subnormal beams (ties at the beam edge) and exact ties
    rng = np.random.default_rng(3000 + seed)
    n = int(rng.integers(5, 300))
    g = W.random_small_graph(3000 + seed, n, mean_deg=3.0, eps_frac=0.3, num_labels=4, weights="edge",
                             final=seed % 2 == 1)
    ll = W.random_small_loglikes(3000 + seed, int(rng.integers(1, 30)), 4, kind="edge")
    beam = [INF, 1e-45, 2.9e-39, 1.17549435e-38, 0.5, 1.0][seed % 6]
    max_active = [0, 0, 1, 3, 17][seed % 5]
    lb = [INF, 0.0, 1e-45, 0.5][seed % 4]
    ro, rg = both(dec, torch_mod, oracle_mod, g, ll, beam=beam, max_active=max_active, lattice_beam=lb)
    parity.assert_same(ro, rg, lattice=True, tag="edge values seed %d" % seed)


def test_batch_matches_single_and_oracle(dec, torch_mod, oracle_mod):
    g = W.random_small_graph(901, 3000, mean_deg=3.0, eps_frac=0.2, num_labels=20)
    gh = dec.load_graph(g)
    lls = [W.random_small_loglikes(910 + u, T, 20) for u, T in enumerate([0, 1, 17, 64, 65, 130, 3])]
    res = dec.wfst_decode_batch(gh, [to_dev(torch_mod, x) for x in lls], beam=9.0, max_active=150,
                                lattice_beam=5.0, record_tokens=True)
    for u, (x, r) in enumerate(zip(lls, res)):
        ro = oracle_mod.decode(g, x, 9.0, 150, 5.0)
        parity.assert_same(ro, r, lattice=True, tag="batch utt %d" % u)
    gh.free()


def test_batch_groups_match_oracle(dec, torch_mod, oracle_mod):
    # 70 utterances of mixed lengths, in caller order unlike their length
    # order: the batch runs as four length groups on separate streams, and
    # every result must still be the oracle's for its own utterance
    g = W.random_small_graph(931, 2000, mean_deg=3.0, eps_frac=0.2, num_labels=16)
    gh = dec.load_graph(g)
    rng = np.random.default_rng(931)
    lens = [int(x) for x in rng.integers(0, 90, size=70)]
    lls = [W.random_small_loglikes(940 + u, T, 16) for u, T in enumerate(lens)]
    res = dec.wfst_decode_batch(gh, [to_dev(torch_mod, x) for x in lls], beam=9.0, max_active=120,
                                lattice_beam=4.0, record_tokens=True)
    for u, (x, r) in enumerate(zip(lls, res)):
        ro = oracle_mod.decode(g, x, 9.0, 120, 4.0)
        parity.assert_same(ro, r, lattice=True, tag="grouped batch utt %d (T=%d)" % (u, lens[u]))
    gh.free()


@pytest.mark.parametrize("groups,publish,fill", [(-1, 0, 0), (0, 0, 0), (1, 1, 0), (2, 3, 0), (5, 1, 8),
                                                   (64, 7, 0)])
def test_record_workgroups_beside_search(dec, torch_mod, oracle_mod, groups, publish, fill):
    # The record pass of the last length group runs in workgroups appended to
    # its search launch, which wait for the search's progress reports (every
    # `publish` token sets); -1 leaves it to the record kernel after the
    # search.  One workgroup reporting every set, a few, and more workgroups
    # than items per report; sets beyond a small record table (fill) go to the
    # large-set pass after the launch.  A 70-utterance batch (four length
    # groups), a 12-utterance one (a single group: record workgroups only
    # with an explicit count) and a 36-utterance label-synchronous batch
    # whose decoded frames are fewer than its frames: every result is the
    # oracle's.
    g = W.random_small_graph(990, 2500, mean_deg=3.0, eps_frac=0.25, num_labels=16)
    gh = dec.load_graph(g)
    rng = np.random.default_rng(991)
    batches = [[int(x) for x in rng.integers(0, 90, size=70)], [int(x) for x in rng.integers(1, 140, size=12)]]
    with dec.debug_opts(record_groups=groups, record_publish=publish, record_fill=fill):
        for b, lens in enumerate(batches):
            lls = [W.random_small_loglikes(1000 + 100 * b + u, T, 16) for u, T in enumerate(lens)]
            res = dec.wfst_decode_batch(gh, [to_dev(torch_mod, x) for x in lls], beam=9.0, max_active=140,
                                        lattice_beam=4.0, record_tokens=True)
            for u, (x, r) in enumerate(zip(lls, res)):
                ro = oracle_mod.decode(g, x, 9.0, 140, 4.0)
                parity.assert_same(ro, r, lattice=True, tokens=True,
                                   tag="batch %d utt %d (T=%d) groups %d publish %d" % (b, u, lens[u], groups,
                                                                                        publish))
        lls = [W.random_small_loglikes(1300 + u, 30 + 3 * u, 16, blank_boost=6.0) for u in range(36)]
        res = dec.wfst_decode_batch(gh, [to_dev(torch_mod, x) for x in lls], beam=9.0, max_active=140,
                                    lattice_beam=4.0, blank_threshold=0.9, blank_id=0, record_tokens=True)
        for u, (x, r) in enumerate(zip(lls, res)):
            ro = oracle_mod.decode(g, x, 9.0, 140, 4.0, 0.9, 0)
            parity.assert_same(ro, r, lattice=True, tokens=True, tag="lsd utt %d groups %d" % (u, groups))
        assert sum(r.num_decoded for r in res) < sum(x.shape[0] for x in lls)
    gh.free()


def test_concurrent_decodes_match(dec, torch_mod, oracle_mod):
    # Three host threads decode the same batch at once: the calls that find
    # the device's workspace, staging buffer or waiting-launch flag taken use
    # their own or decode without record workgroups, and every result is the
    # sequential decode's, bit for bit (and the oracle's for a sample).
    from concurrent.futures import ThreadPoolExecutor
    g = W.random_small_graph(1400, 2500, mean_deg=3.0, eps_frac=0.25, num_labels=16)
    gh = dec.load_graph(g)
    lens = [20 + (7 * u) % 60 for u in range(40)]
    lls = [W.random_small_loglikes(1410 + u, T, 16) for u, T in enumerate(lens)]
    xs = [to_dev(torch_mod, x) for x in lls]

    def run(_):
        return dec.wfst_decode_batch(gh, xs, beam=9.0, max_active=140, lattice_beam=4.0, record_tokens=True)

    ref = run(None)
    for u in (0, 17, 39):
        parity.assert_same(oracle_mod.decode(g, lls[u], 9.0, 140, 4.0), ref[u], lattice=True, tokens=True,
                           tag="sequential utt %d" % u)
    with ThreadPoolExecutor(max_workers=3) as ex:
        outs = list(ex.map(run, range(6)))
    for k, res in enumerate(outs):
        for u, (a, b) in enumerate(zip(ref, res)):
            tag = "call %d utt %d" % (k, u)
            assert a.status == b.status and a.num_decoded == b.num_decoded, tag
            assert np.float32(a.cost).view(np.uint32) == np.float32(b.cost).view(np.uint32), tag
            np.testing.assert_array_equal(a.path_arcs, b.path_arcs, err_msg=tag)
            for f in ("lat_frame", "lat_arc", "lat_cost", "lat_extra", "tok_state", "tok_cost", "tok_arc"):
                x, y = getattr(a, f), getattr(b, f)
                if x is not None and x.dtype == np.float32:
                    x, y = x.view(np.uint32), y.view(np.uint32)
                np.testing.assert_array_equal(x, y, err_msg=tag + " " + f)
            assert a.stats["lattice_raw"] == b.stats["lattice_raw"], tag
    gh.free()


def test_lsd_small_ctc(dec, torch_mod, oracle_mod):
    g = W.random_small_graph(950, 5000, mean_deg=2.0, eps_frac=0.1, num_labels=30)
    n = g.num_states
    src = np.concatenate([np.arange(n), g.src]).astype(np.int32)
    dst = np.concatenate([np.arange(n), g.dst]).astype(np.int32)
    il = np.concatenate([np.ones(n), np.where(g.ilabel == 0, 0, np.maximum(g.ilabel, 2))]).astype(np.int32)
    w = np.concatenate([np.full(n, 0.3), g.weight]).astype(np.float32)
    o = np.argsort(src, kind="stable")
    g2 = W.Graph(n, src[o], dst[o], il[o], np.zeros_like(src), w[o])
    ll = W.random_small_loglikes(951, 300, 30, blank_boost=7.0)
    for thr in (0.5, 0.95, 2.0):
        ro, rg = both(dec, torch_mod, oracle_mod, g2, ll, beam=10.0, max_active=400, lattice_beam=6.0,
                      blank_threshold=thr, blank_id=0)
        parity.assert_same(ro, rg, lattice=True, tag="lsd thr %g" % thr)


@pytest.mark.parametrize("thr,stride", [(0.95, 1), (0.5, 1), (0.9, 2), (2.0, 3), (0.95, 4)])
def test_lsd_blank_unit_set_and_stride(dec, torch_mod, oracle_mod, thr, stride):
    # HMM topology: several blank-like units; a lower frame rate by a stride
    k = 3
    g = W.random_small_hmm_graph(960, k, n=2000)
    gh = dec.load_graph(g)
    for seed in range(4):
        ll = W.random_small_hmm_loglikes(970 + seed, 120, k)
        ro, rg = both(dec, torch_mod, oracle_mod, g, ll, gh=gh, beam=10.0, max_active=300, lattice_beam=5.0,
                      blank_threshold=thr, blank_ids=[2, 0, 1], frame_stride=stride)
        parity.assert_same(ro, rg, lattice=True, tag="hmm thr %g stride %d seed %d" % (thr, stride, seed))
    # the batch path (length groups) with the same options
    lls = [W.random_small_hmm_loglikes(980 + u, 20 + 3 * u, k) for u in range(36)]
    res = dec.wfst_decode_batch(gh, [to_dev(torch_mod, x) for x in lls], beam=10.0, max_active=300,
                                lattice_beam=5.0, blank_threshold=thr, record_tokens=True, blank_ids=[0, 1, 2],
                                frame_stride=stride)
    for u, (x, r) in enumerate(zip(lls, res)):
        ro = oracle_mod.decode(g, x, 10.0, 300, 5.0, thr, 0, [0, 1, 2], stride)
        parity.assert_same(ro, r, lattice=True, tag="hmm batch utt %d" % u)
    gh.free()


def test_edge_cases(dec, torch_mod, oracle_mod):
    def gr(n, arcs, final=None):
        a = np.array(arcs, np.float64).reshape(-1, 5)
        return W.Graph(n, a[:, 0].astype(np.int32), a[:, 1].astype(np.int32), a[:, 2].astype(np.int32),
                       a[:, 3].astype(np.int32), a[:, 4].astype(np.float32), 0,
                       None if final is None else np.asarray(final, np.float32))
    # dead end -> ENOPATH
    ro, rg = both(dec, torch_mod, oracle_mod, gr(2, [[0, 1, 1, 0, 0.0]]), np.zeros((2, 1), np.float32), beam=5.0)
    assert ro.status == rg.status == -3
    # T = 0: the closure of the start state
    g = gr(3, [[0, 1, 0, 0, 0.5], [0, 0, 1, 0, 0.0], [1, 2, 0, 0, 1.0]])
    ro, rg = both(dec, torch_mod, oracle_mod, g, np.zeros((0, 1), np.float32), beam=5.0, lattice_beam=INF)
    parity.assert_same(ro, rg, lattice=True, tag="T=0")
    # all frames blank
    ll = np.log(np.array([[0.99, 0.01]] * 7, np.float32))
    ro, rg = both(dec, torch_mod, oracle_mod, g, ll, beam=5.0, blank_threshold=0.9)
    parity.assert_same(ro, rg, lattice=False, tag="all blank")
    # final weights with no final state reached (fallback)
    g = gr(2, [[0, 1, 1, 0, 0.5]], final=[0.0, INF])
    ro, rg = both(dec, torch_mod, oracle_mod, g, np.array([[-0.25]], np.float32), beam=INF, lattice_beam=3.0)
    parity.assert_same(ro, rg, lattice=True, tag="final fallback")
    assert rg.reached_final == 0


def test_long_utterance(dec, torch_mod, oracle_mod):
    # more frames than a 16-bit index holds: frame offsets, per-frame launch
    # grids and the lattice pass's chain over the sets all span them
    # a small graph whose states all have a self-loop, so no path dies out
    b = W.random_small_graph(990, 60, mean_deg=3.0, eps_frac=0.2, num_labels=5)
    n = b.num_states
    src = np.concatenate([np.arange(n), b.src]).astype(np.int32)
    order = np.argsort(src, kind="stable")
    g = W.Graph(n, src[order], np.concatenate([np.arange(n), b.dst]).astype(np.int32)[order],
                np.concatenate([np.full(n, 1), b.ilabel]).astype(np.int32)[order], np.zeros(src.size, np.int32),
                np.concatenate([np.full(n, 1.5), b.weight]).astype(np.float32)[order])
    ll = W.random_small_loglikes(990, 70000, 5)
    ro, rg = both(dec, torch_mod, oracle_mod, g, ll, beam=8.0, max_active=12, lattice_beam=3.0)
    assert ro.status == 0
    parity.assert_same(ro, rg, lattice=True, tag="70k frames")
    say("70k frames: cost", rg.cost, "tokens", rg.stats["tokens"], "lattice", rg.stats["lattice_kept"])


def test_argument_errors(dec, torch_mod):
    g = W.Graph(2, np.array([0], np.int32), np.array([1], np.int32), np.array([3], np.int32),
                np.array([0], np.int32), np.array([1.0], np.float32))
    gh = dec.load_graph(g)
    x = to_dev(torch_mod, np.zeros((1, 3), np.float32))
    assert dec.wfst_decode(gh, x, 1.0).status == 0
    for kw in (dict(beam=0.0), dict(beam=float("nan")), dict(beam=1.0, blank_id=3),
               dict(beam=1.0, blank_threshold=0.0), dict(beam=1.0, lattice_beam=float("nan")),
               dict(beam=1.0, blank_ids=[0, 3]), dict(beam=1.0, blank_ids=[-1]), dict(beam=1.0, blank_ids=[]),
               dict(beam=1.0, frame_stride=-1)):
        with pytest.raises(dec.WfstError) as e:
            dec.wfst_decode(gh, x, **kw)
        assert e.value.code == dec.WFST_EINVAL
    with pytest.raises(dec.WfstError) as e:
        dec.wfst_decode(gh, to_dev(torch_mod, np.zeros((1, 2), np.float32)), 1.0)
    assert e.value.code == dec.WFST_EINVAL
    gh.free()


# ---------------------------------------------------------------------------
# full-size workloads
# ---------------------------------------------------------------------------

@pytest.fixture(scope="module")
def cfg3(dec):
    say("generating the 25M-arc graph ...")
    g = W.graph_for(3)
    say("uploading")
    return g, dec.load_graph(g)


def test_config3_full(dec, torch_mod, oracle_mod, cfg3):
    g, gh = cfg3
    wl = W.workload(3)
    o = wl.opts
    say("oracle on config 3 ...")
    ro, rg = both(dec, torch_mod, oracle_mod, g, wl.loglikes[0], gh=gh, beam=o.beam,
                  max_active=o.max_active, lattice_beam=o.lattice_beam)
    say("oracle %.1fs; comparing" % ro.seconds)
    parity.assert_same(ro, rg, lattice=True, tag="config 3")
    parity.assert_path_consistent(g, rg, wl.loglikes[0])


def test_config4_batch_full(dec, torch_mod, oracle_mod, cfg3):
    # the benchmark's batch (64 utterances on the 25M-arc graph, one batched
    # call in the launch configuration the benchmark times): every utterance
    # against the oracle, token sets of every frame included
    from concurrent.futures import ThreadPoolExecutor
    g, gh = cfg3
    wl = W.workload(4)
    o = wl.opts
    xs = [to_dev(torch_mod, x) for x in wl.loglikes]
    say("batch decode of %d utterances" % len(xs))
    res = dec.wfst_decode_batch(gh, xs, o.beam, o.max_active, o.lattice_beam, record_tokens=True)
    del xs
    threads = max(1, min(16, len(os.sched_getaffinity(0))))
    say("oracle on %d utterances, %d threads" % (len(res), threads))

    def check(u):
        ro = oracle_mod.decode(g, wl.loglikes[u], o.beam, o.max_active, o.lattice_beam)
        parity.assert_same(ro, res[u], lattice=True, tokens=True, tag="config 4 utt %d" % u)
        parity.assert_path_consistent(g, res[u], wl.loglikes[u])
        return ro.tokens

    with ThreadPoolExecutor(max_workers=threads) as ex:
        toks = list(ex.map(check, range(len(res))))
    say("config 4: %d utterances, %d tokens compared" % (len(res), sum(toks)))


def test_config4_streamed_lattice_pass(dec, torch_mod, oracle_mod, cfg3):
    # the benchmark's batch with lattice pruning's streamed pass forced on
    # (by default its utterances, of about 1,200 records per set, take the
    # block pass): the same lattice, extra costs and kept counts as the
    # default call, and the oracle's on two utterances
    g, gh = cfg3
    wl = W.workload(4)
    o = wl.opts
    xs = [to_dev(torch_mod, x) for x in wl.loglikes]
    a = dec.wfst_decode_batch(gh, xs, o.beam, o.max_active, o.lattice_beam)
    with dec.debug_opts(lattice_pipe=1):
        b = dec.wfst_decode_batch(gh, xs, o.beam, o.max_active, o.lattice_beam)
    del xs
    for u, (ra, rb) in enumerate(zip(a, b)):
        for f in ("lat_frame", "lat_arc", "path_arcs"):
            np.testing.assert_array_equal(getattr(ra, f), getattr(rb, f), err_msg="utt %d %s" % (u, f))
        np.testing.assert_array_equal(parity.bits(ra.lat_cost), parity.bits(rb.lat_cost), err_msg="utt %d" % u)
        np.testing.assert_array_equal(parity.bits(ra.lat_extra), parity.bits(rb.lat_extra), err_msg="utt %d" % u)
    for u in (0, 37):
        ro = oracle_mod.decode(g, wl.loglikes[u], o.beam, o.max_active, o.lattice_beam)
        parity.assert_same(ro, b[u], lattice=True, tokens=False, tag="config 4 streamed utt %d" % u)


def test_config4_wide_rows(dec, torch_mod, oracle_mod, cfg3):
    # the benchmark batch with its rows widened past what the search keeps in
    # LDS (6,000 columns padded to 6,400): rows read from device memory, the
    # same results as the oracle, token sets included
    from concurrent.futures import ThreadPoolExecutor
    g, gh = cfg3
    wl = W.workload(4)
    o = wl.opts
    rng = np.random.default_rng(44)
    lls = [np.concatenate([x, rng.normal(0.0, 1.0, size=(x.shape[0], 400)).astype(np.float32)], axis=1)
           for x in wl.loglikes]
    xs = [to_dev(torch_mod, x) for x in lls]
    say("batch decode of %d widened utterances" % len(xs))
    res = dec.wfst_decode_batch(gh, xs, o.beam, o.max_active, o.lattice_beam, record_tokens=True)
    del xs
    threads = max(1, min(16, len(os.sched_getaffinity(0))))

    def check(u):
        ro = oracle_mod.decode(g, lls[u], o.beam, o.max_active, o.lattice_beam)
        parity.assert_same(ro, res[u], lattice=True, tokens=True, tag="wide config 4 utt %d" % u)

    with ThreadPoolExecutor(max_workers=threads) as ex:
        list(ex.map(check, range(len(res))))


def test_config4_incremental_lattice(dec, torch_mod, oracle_mod, cfg3):
    # the benchmark's batch with the incremental lattice pass: every
    # utterance's lattice, path and token sets bit-identical to the one-shot
    # pass, with a smaller workspace
    g, gh = cfg3
    wl = W.workload(4)
    o = wl.opts
    xs = [to_dev(torch_mod, x) for x in wl.loglikes]
    one = dec.wfst_decode_batch(gh, xs, o.beam, o.max_active, o.lattice_beam, record_tokens=True)
    inc = dec.wfst_decode_batch(gh, xs, o.beam, o.max_active, o.lattice_beam, record_tokens=True,
                                incremental_lattice=True)
    for u, (a, b) in enumerate(zip(one, inc)):
        assert a.status == b.status == 0
        for f in ("tok_off", "tok_state", "tok_arc", "path_arcs", "path_frames", "lat_frame", "lat_arc"):
            np.testing.assert_array_equal(getattr(a, f), getattr(b, f), err_msg="utt %d %s" % (u, f))
        for f in ("tok_cost", "lat_cost", "lat_extra"):
            np.testing.assert_array_equal(parity.bits(getattr(a, f)), parity.bits(getattr(b, f)),
                                          err_msg="utt %d %s" % (u, f))
        assert parity.bits(a.cost) == parity.bits(b.cost)
        assert a.stats["lattice_raw"] == b.stats["lattice_raw"]
    raw = sum(r.stats["lattice_raw"] for r in one)
    kept = sum(r.stats["lattice_incremental"] for r in inc)
    ws_one, ws_inc = one[0].stats["workspace_bytes"], inc[0].stats["workspace_bytes"]
    say("config 4: raw lattice %d arcs, %d left by the incremental pass; workspace %.2f GiB one-shot, "
        "%.2f GiB incremental" % (raw, kept, ws_one / 2**30, ws_inc / 2**30))
    assert kept < raw and ws_inc < ws_one


def test_config6_hmm_lsd_and_stride(dec, torch_mod, oracle_mod):
    # the HMM-topology stand-in at full size: eight blank-like units, with and
    # without a frame stride of 3
    wl = W.workload(6, lsd=True)
    g = wl.graph
    gh = dec.load_graph(g)
    o = wl.opts
    for thr, stride in ((0.95, 1), (0.95, 3), (2.0, 3)):
        say("config 6 threshold", thr, "stride", stride)
        ro, rg = both(dec, torch_mod, oracle_mod, g, wl.loglikes[0], gh=gh, beam=o.beam,
                      max_active=o.max_active, lattice_beam=o.lattice_beam, blank_threshold=thr,
                      blank_ids=list(o.blank_ids), frame_stride=stride)
        parity.assert_same(ro, rg, lattice=True, tag="config 6 thr %g stride %d" % (thr, stride))
        say("decoded", rg.num_decoded, "of", rg.num_frames, "arcs", rg.stats["arcs_expanded"])
    gh.free()


def test_config5_lsd_and_fsd(dec, torch_mod, oracle_mod):
    wl = W.workload(5, lsd=True)
    g = wl.graph
    gh = dec.load_graph(g)
    o = wl.opts
    for thr in (0.95, 2.0):
        say("config 5 threshold", thr)
        ro, rg = both(dec, torch_mod, oracle_mod, g, wl.loglikes[0], gh=gh, beam=o.beam,
                      max_active=o.max_active, lattice_beam=o.lattice_beam, blank_threshold=thr, blank_id=0)
        parity.assert_same(ro, rg, lattice=True, tag="config 5 thr %g" % thr)
        say("decoded", rg.num_decoded, "of", rg.num_frames, "arcs", rg.stats["arcs_expanded"])
    gh.free()
