"""Element-by-element comparison of a GPU decode with the CPU oracle.

The bar is exact equality: integer outputs (states, arcs, frames, counts) and
float32 costs compared bit for bit (0 ULP), since both sides compute
(cost + weight) - loglike with the same two roundings and take every
decision on ordered float32 keys.
"""
import numpy as np


def bits(x):
    return np.asarray(x, np.float32).view(np.uint32)


def assert_same(o, r, lattice: bool, tokens: bool = True, tag: str = ""):
    """o: oracle.OracleResult, r: wfstdec.WfstResult."""
    assert r.status == o.status, "%s status gpu %d oracle %d" % (tag, r.status, o.status)
    if o.status != 0:
        return
    assert r.num_decoded == o.num_decoded, tag
    np.testing.assert_array_equal(r.kept, o.kept, err_msg=tag + " kept frames")
    if tokens:
        np.testing.assert_array_equal(r.tok_off, o.tok_off, err_msg=tag + " token set sizes")
        np.testing.assert_array_equal(r.tok_state, o.tok_state, err_msg=tag + " token states")
        np.testing.assert_array_equal(r.tok_cost.view(np.uint32), o.tok_cost_bits, err_msg=tag + " token costs")
        np.testing.assert_array_equal(r.tok_arc, o.tok_arc, err_msg=tag + " back-pointers")
    assert bits(r.cost) == bits(o.cost), "%s cost gpu %r oracle %r" % (tag, r.cost, o.cost)
    assert r.final_state == o.final_state, tag
    assert r.reached_final == o.reached_final, tag
    np.testing.assert_array_equal(r.path_arcs, o.path_arcs, err_msg=tag + " best path")
    np.testing.assert_array_equal(r.path_frames, o.path_frames, err_msg=tag + " path frames")
    assert r.stats["arcs_expanded"] == o.arcs_expanded, tag
    assert r.stats["eps_arcs"] == o.eps_arcs, tag
    assert r.stats["tokens"] == o.tokens, tag
    if lattice:
        assert r.stats["lattice_raw"] == o.lat_raw, "%s raw lattice gpu %d oracle %d" % (
            tag, r.stats["lattice_raw"], o.lat_raw)
        np.testing.assert_array_equal(r.lat_frame, o.lat_frame, err_msg=tag + " lattice frames")
        np.testing.assert_array_equal(r.lat_arc, o.lat_arc, err_msg=tag + " lattice arcs")
        np.testing.assert_array_equal(bits(r.lat_cost), bits(o.lat_cost), err_msg=tag + " lattice costs")
        np.testing.assert_array_equal(bits(r.lat_extra), bits(o.lat_extra), err_msg=tag + " lattice extras")


def assert_path_consistent(g, r, ll):
    """Properties that hold at any size: the best path is a path of the graph
    from the start state to the final state, it consumes the decoded frames in
    order, and its float32 cost (plus final cost) reproduces the reported
    cost bit for bit."""
    s = int(g.start)
    c = np.float32(0.0)
    j = 0
    for a, f in zip(r.path_arcs, r.path_frames):
        assert int(g.src[a]) == s
        il = int(g.ilabel[a])
        if il == 0:
            assert f == -1
            c = np.float32(c + g.weight[a])
        else:
            assert f == r.kept[j]
            c = np.float32(np.float32(c + g.weight[a]) - ll[f, il - 1])
            j += 1
        s = int(g.dst[a])
    assert j == r.num_decoded and s == r.final_state
    if g.final is not None and r.reached_final:
        c = np.float32(c + g.final[s])
    else:
        c = np.float32(c + np.float32(0.0))
    assert bits(c) == bits(r.cost)
