#!/usr/bin/env python3
"""Benchmark of WFST Viterbi beam decoding with lattice generation on one
MI355X: decoded frames/s (with RTF, arcs expanded/s and the HBM roofline of
the search kernel) on the 25M-arc LVCSR-scale graph, 64 utterances of
300-1,500 frames decoded in one batched call.

One step = one wfst_decode_batch call over the whole batch: label-synchronous
classification, every decoded frame (expansion + epsilon closure, pruning,
lattice recording), final costs, backtrace, lattice-beam pruning and the
sorted lattice.  Log-likelihoods are resident in device memory before the
timed region; graph generation and upload are outside it.

Prints one JSON line.  --gpus N with N > 1 is rejected: the decoder runs on
one GPU; batches of utterances would shard across GPUs with no per-frame
communication, which this build does not do.
"""
import argparse
import gc
import hashlib
import json
import os
import re
import sys
import time
from concurrent.futures import ThreadPoolExecutor

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "decoded frames/sec (RTF) + arcs expanded/sec + % HBM peak, 25M-arc graph"
HBM_PEAK_GBS = 8000.0
FRAME_SHIFT_S = 0.010
PROFILES = os.path.join(ROOT, "profiles")
SQ = os.path.join(PROFILES, "search_kernel_lvcsr-25m-batch64_sq.txt")
# the workloads with kernel-trace and HBM-counter summaries in profiles/
PROFILED = {"cfg4": "lvcsr-25m-batch64", "cfg4x256": "lvcsr-25m-batch256"}


def profile_path(workload: str, kind: str) -> str:
    return os.path.join(PROFILES, "search_kernel_%s_%s.txt" % (PROFILED[workload], kind))


def wl_flag(workload: str) -> str:
    return "" if workload == "cfg4" else " --workload " + workload
CSRC = os.path.join(ROOT, "paper_1808_00687_amd", "csrc")
KERNEL_SOURCES = [os.path.join(CSRC, f) for f in ("search_body.h", "search_kernel.hip", "search_record_kernel.hip",
                                                   "record_set.h", "device_util.h", "internal.h")]
KERNEL_NAME = "search_kernel"
# the 64-utterance batch's search is this many concurrent launches (the
# library's length groups: at most four, of at least 16 utterances each)
GROUP_LAUNCHES = 4
CALIBRATION_MIB = 1024
TRACE_CMD = ("rocprofv3 --kernel-trace --stats --output-format csv -d gpurun_out/prof_search -o run -- "
             "python3 bench.py --steps 3 --warmup 1 --no-cpu-baseline{wl}")
# The counter passes run with the record workgroups off (--record-groups -1):
# the last length group's search launch then holds its search alone, and the
# counters count the search's work only.
PMC_CMD = ("timeout -s KILL 180 rocprofv3 --pmc {counter} --output-format csv -d gpurun_out/pmc_{tag} -o run -- "
           "python3 bench.py --steps 1 --warmup 0 --no-cpu-baseline --no-profile --record-groups -1 "
           "--copy-calibration-mib %d{wl}" % CALIBRATION_MIB)
SQ_PASSES = (("a", "SQ_WAVE_CYCLES SQ_BUSY_CYCLES SQ_WAIT_ANY SQ_WAIT_INST_ANY SQ_ACTIVE_INST_ANY SQ_INSTS_VALU "
                   "SQ_INSTS_LDS SQ_INSTS_SALU"),
             ("b", "SQ_INSTS_VMEM_RD SQ_INSTS_VMEM_WR SQ_INSTS_BRANCH SQ_WAIT_INST_LDS SQ_ACTIVE_INST_VALU "
                   "SQ_ACTIVE_INST_LDS SQ_LDS_BANK_CONFLICT SQ_INSTS_LDS_ATOMIC"))
SQ_CMD = ("timeout -s KILL 120 rocprofv3 --pmc {counters} --output-format csv -d gpurun_out/sq{tag} -o run -- "
          "python3 bench.py --steps 1 --warmup 0 --no-cpu-baseline --no-profile --record-groups -1")
OVERLAP = os.path.join(PROFILES, "lattice_stream_kernel_lvcsr-25m-batch64_overlap.txt")
OVERLAP_CMD = ("rocprofv3 --kernel-trace --stats --output-format csv -d gpurun_out/prof_incr -o run -- "
               "python3 bench.py --steps 3 --warmup 1 --no-cpu-baseline --no-profile --incremental-lattice")

# name: (config, label-synchronous, frame stride, utterances); cfg6 is the
# HMM-topology stand-in (a set of blank-like units), not one of the five
# listed configs; cfg4x256 is config 4's workload at the batch that fills
# every CU with a search workgroup (the same 64 utterances first)
WORKLOADS = {
    "cfg1": (1, True, 1, None), "cfg2": (2, True, 1, None), "cfg3": (3, True, 1, None),
    "cfg4": (4, True, 1, None), "cfg4x256": (4, True, 1, 256),
    "cfg5": (5, True, 1, None), "cfg5fsd": (5, False, 1, None),
    "cfg6": (6, True, 1, None), "cfg6fsd": (6, False, 1, None), "cfg6stride3": (6, True, 3, None),
}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def search_bytes(stats_list):
    """Algorithmic device-memory bytes of the search over one batch, per the
    method's own traffic: per surviving token expanded 16 B (its state, cost
    and the two emitting row offsets), per emitting arc expanded 24 B
    (destination, input label, weight, log-likelihood and the 8-byte token
    of the recombination), per epsilon out-arc of a surviving token 16 B
    (destination, weight and the 8-byte token)."""
    tok = sum(s["tokens"] for s in stats_list)
    arcs = sum(s["arcs_expanded"] for s in stats_list)
    eps = sum(s["eps_arcs"] for s in stats_list)
    return 16 * tok + 24 * arcs + 16 * eps


def kernel_sha() -> str:
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        h.update(open(f, "rb").read())
    return h.hexdigest()


def read_traffic(workload: str):
    """HBM bytes of a batch's search launches from the committed rocprofv3 counter
    summary of the workload, if it was taken on the current kernel sources."""
    if workload not in PROFILED or not os.path.exists(profile_path(workload, "counters")):
        return None
    kv = {}
    for line in open(profile_path(workload, "counters")):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("kernel_source_sha256") != kernel_sha():
        return None
    try:
        return float(kv["hbm_bytes_per_batch"])
    except (KeyError, ValueError):
        return None


def write_profiles(stats_csv: str, fetch_csv: str, write_csv: str, workload: str = "cfg4"):
    """Summaries of the rocprofv3 runs for profiles/: the kernel-trace
    statistics and the HBM counters of the search kernel, each counter scaled
    by what it reads for the plain device copy of known size that bench.py
    runs first (--copy-calibration-mib)."""
    import csv
    rows = list(csv.DictReader(open(stats_csv)))
    wl = wl_flag(workload)
    n_utt = WORKLOADS[workload][3] or 64
    lines = ["# rocprofv3 kernel-trace statistics, workload %s (%d utterances, 25M-arc graph)"
             % (PROFILED[workload], n_utt),
             "# command: " + TRACE_CMD.format(wl=wl),
             "# summary written by: python3 bench.py --write-profiles gpurun_out/prof_search/run_kernel_stats.csv "
             "gpurun_out/pmc_fetch/run_counter_collection.csv gpurun_out/pmc_write/run_counter_collection.csv" + wl,
             "%-62s %6s %14s %14s %7s" % ("kernel", "calls", "total_ms", "average_us", "pct")]
    for r in rows:
        lines.append("%-62s %6s %14.3f %14.1f %7s" % (r["Name"][:62], r["Calls"], float(r["TotalDurationNs"]) / 1e6,
                                                      float(r["AverageNs"]) / 1e3, r["Percentage"]))
    # the batch's search launches run side by side: their span per batch,
    # first start to last end, from the trace of the same run
    trace_csv = os.path.join(os.path.dirname(stats_csv), "run_kernel_trace.csv")
    if os.path.exists(trace_csv):
        ks = sorted((int(r["Start_Timestamp"]), int(r["End_Timestamp"])) for r in csv.DictReader(open(trace_csv))
                    if KERNEL_NAME in r["Kernel_Name"])
        spans = [max(e for _, e in ks[i:i + GROUP_LAUNCHES]) - ks[i][0]
                 for i in range(0, len(ks) - GROUP_LAUNCHES + 1, GROUP_LAUNCHES)]
        if spans:
            # the first batch is the untimed warm-up
            timed = spans[1:] or spans
            lines.append("# %s: %d concurrent launches per batch; span per batch (first start to last end): %s us; "
                         "average over the %d batches after the warm-up: %.1f us"
                         % (KERNEL_NAME, GROUP_LAUNCHES, " ".join("%.0f" % (x / 1e3) for x in spans), len(timed),
                            sum(timed) / len(timed) / 1e3))
    open(profile_path(workload, "trace"), "w").write("\n".join(lines) + "\n")
    out = ["# HBM traffic of %s per batch (its %d concurrent launches summed), workload %s"
           % (KERNEL_NAME, GROUP_LAUNCHES, PROFILED[workload]),
           "# fetch command: " + PMC_CMD.format(counter="FETCH_SIZE", tag="fetch", wl=wl),
           "# write command: " + PMC_CMD.format(counter="WRITE_SIZE", tag="write", wl=wl),
           "# counters are KiB per dispatch; each is scaled by bytes/reading of a %d MiB device copy" % CALIBRATION_MIB,
           "# taken with the record workgroups off (--record-groups -1): the search's own traffic"]
    total = 0.0
    for tag, path in (("fetch", fetch_csv), ("write", write_csv)):
        rows = list(csv.DictReader(open(path)))
        copies = sorted(float(r["Counter_Value"]) for r in rows if "copyBuffer" in r["Kernel_Name"])[-3:]
        cal = sorted(copies)[len(copies) // 2]
        factor = CALIBRATION_MIB * (1 << 20) / (cal * 1024.0)
        vals = [float(r["Counter_Value"]) for r in rows if KERNEL_NAME in r["Kernel_Name"]]
        kib = sum(vals) / len(vals) * GROUP_LAUNCHES
        byts = kib * 1024.0 * factor
        total += byts
        out += ["%s_counter: %s" % (tag, rows[0]["Counter_Name"]),
                "%s_copy_reading_kib: %.1f" % (tag, cal),
                "%s_scale: %.4f" % (tag, factor),
                "%s_kib_per_batch: %.1f" % (tag, kib),
                "%s_bytes_per_batch: %.0f" % (tag, byts)]
    out += ["hbm_bytes_per_batch: %.0f" % total, "kernel_source_sha256: %s" % kernel_sha()]
    open(profile_path(workload, "counters"), "w").write("\n".join(out) + "\n")
    print(profile_path(workload, "trace"))
    print(profile_path(workload, "counters"))


def write_sq_profile(csv_a: str, csv_b: str):
    """Summary of the two SQ counter passes (SQ_PASSES) over the search
    kernel for profiles/: counts summed over the batch's launches, and per
    wave and decoded frame (a utterance's 16 waves run all its frames)."""
    import csv
    from paper_1808_00687_amd import workloads
    wl = workloads.workload(4)
    frames = sum(x.shape[0] for x in wl.loglikes)
    waves = 16 * len(wl.loglikes)
    per = waves * frames / len(wl.loglikes)
    tot = {}
    for path in (csv_a, csv_b):
        for r in csv.DictReader(open(path)):
            if KERNEL_NAME in r["Kernel_Name"]:
                tot[r["Counter_Name"]] = tot.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    lines = ["# SQ counters of %s, workload lvcsr-25m-batch64 (64 utterances, 25M-arc graph), summed over the "
             "batch's %d concurrent launches (%d waves)" % (KERNEL_NAME, GROUP_LAUNCHES, waves)]
    for tag, counters in SQ_PASSES:
        lines.append("# pass %s: %s" % (tag, SQ_CMD.format(counters=counters, tag=tag)))
    lines += ["# summary written by: python3 bench.py --write-sq-profile gpurun_out/sqa/run_counter_collection.csv "
              "gpurun_out/sqb/run_counter_collection.csv",
              "# the cycle counters count in units of four cycles; per_wave_frame = count / (waves x frames per "
              "utterance), %d decoded frames" % frames,
              "%-24s %14s %16s" % ("counter", "count", "per_wave_frame")]
    for name in sorted(tot):
        lines.append("%-24s %14.4g %16.1f" % (name, tot[name], tot[name] / per))
    w = tot.get("SQ_WAVE_CYCLES", 0.0)
    if w:
        for name in ("SQ_WAIT_ANY", "SQ_ACTIVE_INST_ANY", "SQ_WAIT_INST_ANY"):
            if name in tot:
                lines.append("%s / SQ_WAVE_CYCLES: %.2f" % (name, tot[name] / w))
    if "SQ_INSTS_VALU" in tot and w:
        # four waves share a SIMD; a wave64 VALU instruction holds it for one
        # four-cycle unit
        lines.append("SIMD busy with VALU, share of wave time: %.2f" % (4.0 * tot["SQ_INSTS_VALU"] / w))
    lines.append("kernel_source_sha256: %s" % kernel_sha())
    open(SQ, "w").write("\n".join(lines) + "\n")
    print(SQ)


def write_overlap_profile(trace_csv: str):
    """Summary of a kernel trace of the incremental lattice mode for
    profiles/: per batch, the interval of the search launch and of the
    lattice pass beside it on the library's second stream, how long the two
    ran at the same time, and the kernels that follow the search."""
    import csv
    rows = sorted(((int(r["Start_Timestamp"]), int(r["End_Timestamp"]), r["Kernel_Name"])
                   for r in csv.DictReader(open(trace_csv)) if "wfd::" in r["Kernel_Name"]))
    # a batch starts with the kernels the decode launches before its search
    # (clearing and frame classification)
    starts, first = [], 0
    for si, r in enumerate(rows):
        if KERNEL_NAME in r[2]:
            i = si
            while i > first and any(k in rows[i - 1][2] for k in ("zero_kernel", "classify_kernel")):
                i -= 1
            starts.append((i, si))
            first = si + 1
    lines = ["# kernel trace of the incremental lattice mode, workload lvcsr-25m-batch64 (64 utterances, "
             "25M-arc graph): one search launch per batch on the decode stream, one lattice_stream_kernel "
             "launch beside it on a second stream",
             "# command: " + OVERLAP_CMD,
             "# summary written by: python3 bench.py --write-overlap-profile gpurun_out/prof_incr/run_kernel_trace.csv",
             "# times in ms relative to the batch's first kernel start; overlap = time both kernels ran",
             "%5s %9s %9s %9s %9s %9s %9s %9s" % ("batch", "search0", "search1", "lat0", "lat1", "overlap",
                                                 "lat_after", "batch_end")]
    agg = []
    for b, (i, si) in enumerate(starts):
        window = rows[i:starts[b + 1][0] if b + 1 < len(starts) else len(rows)]
        t0 = min(r[0] for r in window)
        s0, s1 = rows[si][0], rows[si][1]
        lat = [r for r in window if "lattice_stream_kernel" in r[2]]
        if not lat:
            continue
        l0, l1 = lat[0][0], lat[0][1]
        ov = max(0, min(s1, l1) - max(s0, l0))
        end = max(r[1] for r in window)
        vals = [(x - t0) / 1e6 for x in (s0, s1, l0, l1)] + [ov / 1e6, max(0, l1 - s1) / 1e6, (end - t0) / 1e6]
        agg.append(vals)
        lines.append("%5d " % b + " ".join("%9.2f" % v for v in vals))
    if len(agg) > 1:
        tail = agg[1:]
        mean = [sum(v[j] for v in tail) / len(tail) for j in range(len(tail[0]))]
        lines.append("mean over batches 1..%d: search %.2f ms, lattice pass %.2f ms, overlap %.2f ms (%.0f%% of "
                     "the search), lattice pass after the search %.2f ms, batch %.2f ms"
                     % (len(agg) - 1, mean[1] - mean[0], mean[3] - mean[2], mean[4],
                        100.0 * mean[4] / max(mean[1] - mean[0], 1e-9), mean[5], mean[6]))
    names = {}
    for r in rows[starts[min(1, len(starts) - 1)][0]:] if starts else []:
        k = re.findall(r"(\w+)(?:<[^>]*>)?\(", r[2])
        names.setdefault(k[0] if k else r[2], []).append((r[1] - r[0]) / 1e6)
    lines.append("%-28s %6s %12s" % ("kernel (batches 1..)", "calls", "mean_ms"))
    for k in sorted(names, key=lambda k: -sum(names[k])):
        lines.append("%-28s %6d %12.3f" % (k, len(names[k]), sum(names[k]) / len(names[k])))
    open(OVERLAP, "w").write("\n".join(lines) + "\n")
    print(OVERLAP)


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


# A GPU machine grants one process at most this many host threads, whatever the
# affinity mask shows.
HOST_THREAD_SHARE = 16


def cpu_baseline(wl):
    """The oracle as it stands, on the host cores, over the same workload:
    every utterance, one oracle call per thread of a pool over the usable
    cores, rate = decoded frames / wall seconds of the pool.  A batch
    workload also gets a one-core rate over its first four utterances (run
    one after another), so the figure can be scaled per core."""
    import oracle
    oracle.build()
    visible = len(os.sched_getaffinity(0))
    cores = max(1, min(visible, HOST_THREAD_SHARE))
    o = wl.opts
    g = wl.graph
    n_utt = len(wl.loglikes)

    def run(u):
        return oracle.decode(g, wl.loglikes[u], o.beam, o.max_active, o.lattice_beam, o.blank_threshold,
                             o.blank_id, o.blank_ids, o.frame_stride)

    threads = min(cores, n_utt)
    t0 = time.perf_counter()
    with ThreadPoolExecutor(max_workers=threads) as ex:
        res = list(ex.map(run, range(n_utt)))
    wall = time.perf_counter() - t0
    frames = sum(r.num_decoded for r in res)
    out = {
        "value": frames / wall,
        "unit": "frames/s",
        "cores": threads,
        "kind": "oracle",
        "sample": "all %d utterance(s) of the workload (%d decoded frames), one oracle call per thread of a "
                  "%d-thread pool, rate = decoded frames / wall seconds (%.2f s)" % (n_utt, frames, threads, wall),
        "cpu_model": cpu_model(),
        "cores_visible": visible,
    }
    if n_utt > 1:
        k = min(4, n_utt)
        t0 = time.perf_counter()
        one = [run(u) for u in range(k)]
        w1 = time.perf_counter() - t0
        out["one_core"] = {"value": sum(r.num_decoded for r in one) / w1, "unit": "frames/s",
                           "sample": "utterances 0..%d one after another on one thread (%.2f s)" % (k - 1, w1)}
    return out


def copy_bandwidth(torch, mib: int = 2048, reps: int = 5):
    """Achievable HBM bandwidth: a plain device-to-device copy of `mib` MiB,
    timed with HIP events; bytes moved = read + write."""
    n = mib * (1 << 20) // 4
    a = torch.ones(n, dtype=torch.float32, device="cuda:0")
    b = torch.empty_like(a)
    b.copy_(a)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        b.copy_(a)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del a, b
    torch.cuda.empty_cache()
    return 2.0 * mib * (1 << 20) / (ms / 1e3) / 1e9


def copy_calibration(torch, mib: int):
    """A plain device copy of known size, for scaling HBM counters."""
    n = mib * (1 << 20) // 4
    a = torch.ones(n, dtype=torch.float32, device="cuda:0")
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    log("copy calibration: 3 copies of %d MiB" % mib)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="cfg4", choices=sorted(WORKLOADS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration-mib", type=int, default=0)
    ap.add_argument("--no-profile", action="store_true",
                    help="do not time kernel phases with HIP events")
    ap.add_argument("--write-profiles", nargs=3, metavar=("STATS_CSV", "FETCH_CSV", "WRITE_CSV"),
                    help="write the profiles/ summaries from rocprofv3 CSV output and exit")
    ap.add_argument("--incremental-lattice", action="store_true",
                    help="decode with the incremental lattice pass beside the search (not the benchmark line)")
    ap.add_argument("--word-lattice", action="store_true",
                    help="also build the word-level lattice (not the benchmark line)")
    ap.add_argument("--write-sq-profile", nargs=2, metavar=("PASS_A_CSV", "PASS_B_CSV"),
                    help="write the SQ counter summary for profiles/ and exit")
    ap.add_argument("--record-groups", type=int, default=0,
                    help="record workgroups in the last length group's search launch (-1: none, the record "
                         "kernel runs after that search; 0: the library's default)")
    ap.add_argument("--write-overlap-profile", metavar="TRACE_CSV",
                    help="write the incremental-mode overlap summary for profiles/ and exit")
    args = ap.parse_args()
    if args.write_overlap_profile:
        write_overlap_profile(args.write_overlap_profile)
        return
    if args.write_profiles:
        write_profiles(*args.write_profiles, workload=args.workload)
        return
    if args.write_sq_profile:
        write_sq_profile(*args.write_sq_profile)
        return

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py: this decoder runs on one GPU; --gpus %d is not supported (utterance batches "
              "would shard across GPUs with no per-frame traffic, which this build does not do)"
              % max(args.gpus, world), file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_1808_00687_amd import wfstdec, workloads

    if not torch.cuda.is_available():
        print("bench.py: no GPU", file=sys.stderr)
        sys.exit(1)
    cfg, lsd, stride, n_utt = WORKLOADS[args.workload]
    t = time.time()
    wl = workloads.workload(cfg, n_utt=n_utt, lsd=lsd, frame_stride=stride)
    log("workload %s generated in %.1fs (%d states, %d arcs, %d utterances)" % (
        wl.name, time.time() - t, wl.graph.num_states, wl.graph.num_arcs, len(wl.loglikes)))
    if args.copy_calibration_mib:
        copy_calibration(torch, args.copy_calibration_mib)
    t = time.time()
    gh = wfstdec.load_graph(wl.graph)
    torch.cuda.synchronize()
    load_s = time.time() - t
    xs = [torch.from_numpy(x).to("cuda:0") for x in wl.loglikes]
    torch.cuda.synchronize()
    o = wl.opts
    stream = torch.cuda.current_stream()

    def step(profile, steps=False):
        return wfstdec.wfst_decode_batch(gh, xs, o.beam, o.max_active, o.lattice_beam, o.blank_threshold,
                                         o.blank_id, profile=profile, stream=stream, profile_steps=steps,
                                         blank_ids=o.blank_ids, frame_stride=o.frame_stride,
                                         incremental_lattice=args.incremental_lattice,
                                         word_lattice=args.word_lattice)

    if args.record_groups:
        wfstdec.wfst_set_debug_opts(record_groups=args.record_groups)
    for i in range(args.warmup):
        res = step(False)
        log("warmup %d done" % i)
    torch.cuda.synchronize()
    profile = not args.no_profile
    # the process's long-lived objects (torch's, the workload's) go to the
    # permanent generation: a full collection over them would otherwise land
    # inside a step now and then (tens of ms); each step's own garbage is
    # still collected
    gc.collect()
    gc.freeze()
    t0 = time.perf_counter()
    res = None
    for i in range(args.steps):
        res = step(profile)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_per_step = (t1 - t0) * 1e3 / max(args.steps, 1)
    bad = [r.status for r in res if r.status != 0]
    if bad:
        log("warning: %d utterances without a path" % len(bad))
    stats = [r.stats for r in res]
    frames_dec = sum(s["frames_decoded"] for s in stats)
    frames = sum(s["frames"] for s in stats)
    arcs = sum(s["arcs_expanded"] for s in stats)
    sec = ms_per_step / 1e3
    out = {
        "metric": METRIC,
        "value": frames_dec / sec,
        "unit": "frames/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": wl.name,
            "graph_states": wl.graph.num_states,
            "graph_arcs": wl.graph.num_arcs,
            "utterances": len(wl.loglikes),
            "frames": frames,
            "decoded_frames": frames_dec,
            "labels": wl.num_labels,
            "beam": o.beam,
            "max_active": o.max_active,
            "lattice_beam": o.lattice_beam,
            "blank_threshold": o.blank_threshold,
            "blank_units": len(o.blank_ids) if o.blank_ids else 1,
            "frame_stride": o.frame_stride,
            "parallelism": "utterance batch of %d on 1 GPU" % len(wl.loglikes),
            "lattice_mode": ("incremental" if args.incremental_lattice else "one-shot")
                            + (" + word lattice" if args.word_lattice else ""),
            "record_pass": ("beside the search (incremental pass)" if args.incremental_lattice else
                            "after each length group's search" if args.record_groups < 0 else
                            "beside the last length group's search, after the others'"),
        },
        "rtf": sec / (frames * FRAME_SHIFT_S),
        "original_frames_per_s": frames / sec,
        "arcs_expanded_per_s": arcs / sec,
        "tokens_per_decoded_frame": sum(s["tokens"] for s in stats) / max(frames_dec, 1),
        "lattice_arcs_kept": sum(s["lattice_kept"] for s in stats),
        "graph_load_s": load_s,
    }
    if profile:
        s0 = stats[0]
        launches = s0["search_launches"]
        search_ms = s0["search_ms"]
        # A batch's search is one launch per length group, the groups' launches
        # running at the same time on separate streams: they are measured as
        # one launch of the batch, from the first one's start to the last
        # one's end (HIP events on the launch streams).
        alg = search_bytes(stats)
        dur_s = s0["search_span_ms"] / 1e3
        achieved = alg / dur_s / 1e9 if dur_s > 0 else None
        traffic = read_traffic(args.workload)
        copy_gbs = copy_bandwidth(torch)
        out["roofline"] = {
            "kernel": "search_kernel",
            "bound": "hbm",
            "achieved": achieved,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS if achieved else None,
            "copy_gbs": copy_gbs,
            "frac_of_copy": achieved / copy_gbs if achieved and copy_gbs else None,
            "traffic": traffic,
            "algorithmic_bytes_per_launch": alg,
            "avg_launch_us": dur_s * 1e6,
            "launches": 1,
            "concurrent_group_launches": launches,
            "group_launch_ms_sum": search_ms,
        }
        out["kernel_ms"] = {"search": search_ms, "record": s0["record_ms"], "final": s0["final_ms"]}
        # the utterance with the most decoded frames sets the search kernel's
        # duration: its workgroup's time per step of a frame, from one more
        # call (after the timed ones) that reads the device clock per step
        steps_res = step(True, True)
        torch.cuda.synchronize()
        crit = max((r.stats for r in steps_res), key=lambda s: s["frames_decoded"])
        names = ["expand+queue_closure", "spill_closure", "prune", "compact", "wave0_expand", "between_frames",
                 "abandoned_lds_attempts"]
        out["search_steps_ms_longest_utt"] = {n: round(v, 3) for n, v in zip(names, crit["search_phase_ms"])}
        out["finish_ms_longest_utt"] = {"backtrace": round(crit["backtrace_ms"], 3),
                                        "lattice_prune": round(crit["lattice_prune_ms"], 3)}
    if not args.no_cpu_baseline:
        log("oracle baseline ...")
        out["cpu_baseline"] = cpu_baseline(wl)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
