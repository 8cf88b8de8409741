"""bench.py's host-side tools on synthetic rocprofv3 output (no GPU): the
kernel-trace and counter summaries, the overlap summary of the incremental
lattice mode, and the refusal of more than one GPU."""
import csv
import importlib.util
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture()
def bench(tmp_path, monkeypatch):
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    b = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(b)
    monkeypatch.setattr(b, "PROFILES", str(tmp_path))
    monkeypatch.setattr(b, "OVERLAP", str(tmp_path / "overlap.txt"))
    return b


def kname(k, tmpl=""):
    return "wfd::(anonymous namespace)::%s%s(wfd::Params)" % (k, tmpl)


def write_csv(path, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=list(rows[0]))
        w.writeheader()
        w.writerows(rows)


def test_overlap_summary(bench, tmp_path):
    # three batches: clearing and classification, the search, the lattice pass
    # beside it (starting 1 ms later, ending 10 ms after the search), finish
    rows = []
    for b in range(3):
        o = b * 100_000_000
        for k, a, e in (("zero_kernel", 0, 1_000), ("classify_kernel", 2_000, 3_000),
                        ("search_kernel<false>", 5_000, 30_005_000), ("lattice_stream_kernel", 1_005_000, 40_005_000),
                        ("finish_kernel", 40_010_000, 43_010_000)):
            rows.append({"Kernel_Name": kname(k), "Start_Timestamp": o + a, "End_Timestamp": o + e})
    trace = tmp_path / "trace.csv"
    write_csv(trace, rows)
    bench.write_overlap_profile(str(trace))
    text = (tmp_path / "overlap.txt").read_text()
    # overlap 29 ms (1 ms after the search starts until it ends), 10 ms after it
    assert "overlap 29.00 ms (97% of the search)" in text
    assert "lattice pass after the search 10.00 ms" in text
    assert "batch 43.01 ms" in text
    # template arguments do not split a kernel's line
    assert "\nsearch_kernel " in text


def test_trace_and_counter_summaries(bench, tmp_path):
    G = bench.GROUP_LAUNCHES
    d = tmp_path / "prof"
    d.mkdir()
    # 3 batches of G concurrent search launches; spans 30, 20 and 22 ms
    rows = []
    for b, span in enumerate((30_000_000, 20_000_000, 22_000_000)):
        o = b * 100_000_000
        for g in range(G):
            rows.append({"Kernel_Name": kname("search_kernel", "<false>"), "Start_Timestamp": o + g * 1000,
                         "End_Timestamp": o + span if g == G - 1 else o + span // 2})
    write_csv(d / "run_kernel_trace.csv", rows)
    write_csv(d / "run_kernel_stats.csv", [{"Name": kname("search_kernel", "<false>"), "Calls": 3 * G,
                                            "TotalDurationNs": 1, "AverageNs": 1, "Percentage": 100}])
    # counters: the copy of CALIBRATION_MIB reads half its bytes on FETCH_SIZE
    # (scale 2) and all of them on WRITE_SIZE; G dispatches of 1000 KiB each
    cal_kib = bench.CALIBRATION_MIB * 1024.0
    for tag, name, reading in (("fetch", "FETCH_SIZE", cal_kib / 2), ("write", "WRITE_SIZE", cal_kib)):
        rr = [{"Kernel_Name": "__amd_rocclr_copyBuffer", "Counter_Name": name, "Counter_Value": reading}] * 3
        rr += [{"Kernel_Name": kname("search_kernel", "<false>"), "Counter_Name": name, "Counter_Value": 1000.0}] * G
        write_csv(d / ("%s.csv" % tag), rr)
    bench.write_profiles(str(d / "run_kernel_stats.csv"), str(d / "fetch.csv"), str(d / "write.csv"))
    trace = open(bench.profile_path("cfg4", "trace")).read()
    # the warm-up batch (30 ms) is left out of the average: (20 + 22) / 2
    assert "average over the 2 batches after the warm-up: 21000.0 us" in trace
    counters = open(bench.profile_path("cfg4", "counters")).read()
    kv = dict(l.split(": ", 1) for l in counters.splitlines() if ": " in l and not l.startswith("#"))
    assert float(kv["fetch_scale"]) == pytest.approx(2.0)
    assert float(kv["write_scale"]) == pytest.approx(1.0)
    per_batch = G * 1000.0 * 1024.0
    assert float(kv["hbm_bytes_per_batch"]) == pytest.approx(per_batch * 2.0 + per_batch)
    # the summary holds for the sources it was taken on
    assert bench.read_traffic("cfg4") == pytest.approx(per_batch * 3.0)
    with open(bench.profile_path("cfg4", "counters"), "a") as f:
        f.write("kernel_source_sha256: 0\n")
    assert bench.read_traffic("cfg4") is None
    assert bench.read_traffic("cfg5") is None


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=60)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
