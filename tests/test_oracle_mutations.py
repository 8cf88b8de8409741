"""The pins must catch plausible mistakes in the oracle.

Each case plants one mistake in a copy of the oracle's C source (on the CPU,
in a temporary directory), builds it, and runs the pin suite against it in a
subprocess; the pin suite must fail.  The committed oracle is not touched.
"""
import os
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "oracle_wfst.c")

MUTATIONS = {
    "loglike_sign": ("float cand = t1 - row[ilabel[a] - 1];", "float cand = t1 + row[ilabel[a] - 1];"),
    "loglike_column": ("float cand = t1 - row[ilabel[a] - 1];", "float cand = t1 - row[ilabel[a] % L];"),
    "add_order": ("float t1 = c + weight[a];\n                float cand = t1 - row[ilabel[a] - 1];",
                  "float t1 = weight[a] - row[ilabel[a] - 1];\n                float cand = c + t1;"),
    "subnormal_flush": ("float cand = t1 - row[ilabel[a] - 1];\n                touch",
                        "float cand = t1 - row[ilabel[a] - 1];\n                if (fabsf(cand) < FLT_MIN) cand = 0.0f;\n                touch"),
    "dropped_weight": ("float t1 = c + weight[a];\n                float cand", "float t1 = c;\n                float cand"),
    "tie_break_reversed": ("| (uint32_t)(arc + 1);", "| (uint32_t)(0x7fffffff - arc);"),
    "beam_exclusive": ("if (k <= lim) scratch[nk++] = k;", "if (k < lim) scratch[nk++] = k;"),
    "max_active_off_by_one": ("uint32_t theta = scratch[max_active - 1];", "uint32_t theta = scratch[max_active];"),
    "closure_no_repush": ("if (touch(w, d, make_tok(cand, a)) && !w->inq[d]) {", "if (touch(w, d, make_tok(cand, a)) && 0) {"),
    "eps_weight_dropped": ("float cand = c + g->w[a];", "float cand = c;"),
    "final_weight_ignored": ("float f = final_weight ? final_weight[S[i].state] : 0.0f;", "float f = 0.0f;"),
    "blank_test_inverted": ("if (ll[(int64_t)t * L + blank_ids[i]] > thr) blank = 1;",
                            "if (ll[(int64_t)t * L + blank_ids[i]] < thr) blank = 1;"),
    "blank_set_first_unit_only": ("for (int32_t i = 0; i < nb; i++)\n            if (ll",
                                  "for (int32_t i = 0; i < 1; i++)\n            if (ll"),
    "frame_stride_ignored": ("for (int32_t t = 0; t < T; t += stride) {", "for (int32_t t = 0; t < T; t++) {"),
    "lattice_extra_sign": ("R[k].ex = d1 + e_node[R[k].gd];", "R[k].ex = d1 - e_node[R[k].gd];"),
    "lattice_prefix_swapped": ("float d1 = R[k].p - tok_cost(S[R[k].gd].tok);\n                    R[k].ex",
                               "float d1 = tok_cost(S[R[k].gd].tok) - R[k].p;\n                    R[k].ex"),
    "lattice_eps_not_iterated": ("if (okey(ex) < okey(e_node[R[k].gs])) { e_node[R[k].gs] = ex; changed = 1; }",
                                 "if (okey(ex) < okey(e_node[R[k].gs])) { e_node[R[k].gs] = ex; }"),
    "lattice_cut_strict": ("if (okey(p) > cuts[j + 1]) continue;", "if (okey(p) >= cuts[j + 1]) continue;"),
    "eps_lattice_cut_dropped": ("if (okey(p) > cuts[j]) continue;", "if (0) continue;"),
    "eps_lattice_cut_strict": ("if (okey(p) > cuts[j]) continue;", "if (okey(p) >= cuts[j]) continue;"),
    "final_tie_highest_state": ("if (okey(tot[i - lo]) < okey(tot[best - lo])) best = i;",
                                "if (okey(tot[i - lo]) <= okey(tot[best - lo])) best = i;"),
}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_catch_mutation(name, tmp_path):
    old, new = MUTATIONS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, "mutation anchor not found: %s" % name
    mdir = tmp_path / "o"
    mdir.mkdir()
    mc = mdir / "oracle_wfst.c"
    mc.write_text(src.replace(old, new))
    hdr = os.path.join(ROOT, "oracle", "oracle_wfst.h")
    (mdir / "oracle_wfst.h").write_text(open(hdr).read())
    lib = mdir / "liboracle_wfst.so"
    subprocess.check_call(["gcc", "-O2", "-ffp-contract=off", "-std=c11", "-D_POSIX_C_SOURCE=200809L",
                           "-shared", "-fPIC", "-o", str(lib), str(mc), "-lm"])
    env = dict(os.environ, WFST_ORACLE_LIB=str(lib))
    p = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_pins.py")],
                       env=env, cwd=ROOT, capture_output=True, text=True, timeout=600)
    assert p.returncode != 0, "pins did not catch mutation %s:\n%s" % (name, p.stdout[-2000:])
