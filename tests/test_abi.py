"""The C-ABI library loads, exports every declared entry point, and its graph
validation agrees with the oracle's (no GPU needed: validation runs on the
host before any device call)."""
import os
import re

import numpy as np
import pytest

from paper_1808_00687_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "wfstdec.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(wfst_\w+)\s*\(", text)))


def test_header_declares_the_api():
    names = declared_functions()
    for n in ("wfst_load", "wfst_decode", "wfst_decode_batch", "wfst_result_best",
              "wfst_result_lattice", "wfst_result_tokens", "wfst_result_free", "wfst_last_error"):
        assert n in names


def test_library_exports_every_declared_symbol():
    from paper_1808_00687_amd import wfstdec
    import ctypes
    lib = ctypes.CDLL(wfstdec.LIB_PATH)
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing


def _graph(n, arcs, start=0, final=None):
    a = np.array(arcs, dtype=np.float64).reshape(-1, 5)
    return W.Graph(n, a[:, 0].astype(np.int32), a[:, 1].astype(np.int32), a[:, 2].astype(np.int32),
                   a[:, 3].astype(np.int32), a[:, 4].astype(np.float32), start,
                   None if final is None else np.asarray(final, np.float32))


BASE = [[0, 1, 1, 0, 1.0], [1, 2, 0, 0, 0.5], [2, 0, 2, 0, 0.0]]


def _cases():
    def mod(**kw):
        g = _graph(3, BASE)
        for k, v in kw.items():
            getattr(g, k)[:] = v
        return g
    yield "ok", _graph(3, BASE)
    yield "unsorted", mod(src=[1, 0, 2])
    yield "dst_range", mod(dst=[0, 3, 0])
    yield "src_range", mod(src=[0, 1, 3])
    yield "neg_label", mod(ilabel=[1, 0, -1])
    yield "neg_olabel", mod(olabel=[0, -2, 0])
    yield "nan_weight", mod(weight=[np.nan, 0.5, 0.0])
    yield "inf_weight", mod(weight=[np.inf, 0.5, 0.0])
    yield "neg_eps_weight", mod(weight=[1.0, -0.5, 0.0])
    yield "neg_emit_weight_ok", mod(weight=[-1.0, 0.5, 0.0])
    yield "eps_path_ok", mod(ilabel=[1, 0, 0])
    yield "eps_cycle", mod(ilabel=[0, 0, 0])
    yield "eps_selfloop", mod(src=[0, 1, 2], dst=[1, 2, 2], ilabel=[1, 0, 0])
    yield "start_range", _graph(3, BASE, start=3)
    yield "final_nan", _graph(3, BASE, final=[0.0, np.nan, 0.0])
    yield "final_neginf", _graph(3, BASE, final=[0.0, -np.inf, 0.0])
    yield "final_inf_ok", _graph(3, BASE, final=[0.0, np.inf, 1.0])
    yield "no_arcs_ok", W.Graph(2, np.zeros(0, np.int32), np.zeros(0, np.int32), np.zeros(0, np.int32),
                                np.zeros(0, np.int32), np.zeros(0, np.float32))


@pytest.mark.parametrize("name,g", list(_cases()))
def test_validation_agrees_with_oracle(oracle_mod, name, g):
    from paper_1808_00687_amd import wfstdec
    want = oracle_mod.validate_graph(g)
    assert (want == 0) == name.endswith("ok")
    try:
        h = wfstdec.load_graph(g)
        got = 0
        h.free()
    except wfstdec.WfstError as e:
        got = e.code
    if want == 0:
        # valid: loads on a GPU, or reaches the device step without one
        assert got in (0, wfstdec.WFST_EDEVICE)
    else:
        assert got == wfstdec.WFST_EINVAL


def test_ctypes_structs_match_the_header(tmp_path):
    # the binding's ctypes mirrors of the header's structs: same size, same
    # field offsets (read from a C program compiled against the header)
    import ctypes
    import subprocess
    from paper_1808_00687_amd import wfstdec
    mirrors = {"wfst_decode_opts": wfstdec._Opts, "wfst_stats": wfstdec._Stats,
               "wfst_graph_info": wfstdec._Info, "wfst_lat_arc": wfstdec._LatArc,
               "wfst_debug_opts": wfstdec._DebugOpts, "wfst_noalloc_out": wfstdec._NoallocOut,
               "wfst_result_summary": wfstdec._Summary}
    lines = ["#include <stdio.h>", "#include <stddef.h>", '#include "wfstdec.h"', "int main(void) {"]
    for cname, py in mirrors.items():
        lines.append('printf("%s size %%zu\\n", sizeof(%s));' % (cname, cname))
        for f, _ in py._fields_:
            lines.append('printf("%s %s %%zu\\n", offsetof(%s, %s));' % (cname, f, cname, f))
    lines += ["return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    subprocess.check_call(["gcc", "-std=c11", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)])
    got = {}
    for ln in subprocess.check_output([str(exe)], text=True).splitlines():
        a, b, c = ln.split()
        got[(a, b)] = int(c)
    for cname, py in mirrors.items():
        assert got[(cname, "size")] == ctypes.sizeof(py), cname
        for f, _ in py._fields_:
            assert got[(cname, f)] == getattr(py, f).offset, (cname, f)


def test_debug_opts_validation():
    # host-side only: the switches are checked and stored without a device call
    from paper_1808_00687_amd import wfstdec
    wfstdec.wfst_set_debug_opts(lds_fill=5, lattice_lds=-1, permute=1, lattice_pipe=-1)
    wfstdec.wfst_set_debug_opts(lattice_pipe=1)
    for bad in (dict(lds_fill=-1), dict(lattice_lds=-2), dict(permute=-3), dict(fail_lattice_alloc=-1),
                dict(lattice_pipe=-2), dict(lattice_spin=-1)):
        with pytest.raises(wfstdec.WfstError) as e:
            wfstdec.wfst_set_debug_opts(**bad)
        assert e.value.code == wfstdec.WFST_EINVAL
    wfstdec.wfst_set_debug_opts()


def test_noalloc_rejects_bad_arguments_on_the_host():
    # argument checks come before any device call
    import ctypes
    from paper_1808_00687_amd import wfstdec
    lib = wfstdec._lib
    o = wfstdec._Opts()
    lib.wfst_default_opts(ctypes.byref(o))
    d = wfstdec._NoallocOut()
    assert lib.wfst_decode_noalloc(None, None, 0, 1, ctypes.byref(o), None, ctypes.byref(d)) == wfstdec.WFST_EINVAL
    assert lib.wfst_decode_noalloc(None, None, 0, 1, None, None, None) == wfstdec.WFST_EINVAL


def test_result_summaries_reject_bad_arguments_on_the_host():
    # the batched result accessor checks its arguments before touching a result
    import ctypes
    from paper_1808_00687_amd import wfstdec
    s = (wfstdec._Summary * 1)()
    lib = wfstdec._lib
    assert lib.wfst_result_summaries(None, 1, 0, s) == wfstdec.WFST_EINVAL
    outs = (ctypes.c_void_p * 1)()
    assert lib.wfst_result_summaries(outs, 1, 0, s) == wfstdec.WFST_EINVAL
    assert lib.wfst_result_summaries(outs, -1, 0, s) == wfstdec.WFST_EINVAL
    assert lib.wfst_result_summaries(outs, 0, 1, None) == wfstdec.WFST_OK
