"""Benchmark of the in-memory snapshot hot path on one MI355X.

    python bench.py [--steps K] [--warmup W] [--no-overlap] [--no-cpu] [--no-gating]

One step is one pass of the whole path over one rank's state shard -- by
default the 7B LLaMA shard (32 layers, hidden 4096, FFN 11008: 1164
fragments, 94.3 GB of bf16 params, fp32 master weights and Adam moments,
64 MiB chunks), whose two host images are pageable memory behind 8 GiB
pinned bounce rings:
  update   = an optimizer-like update of every fragment, in buckets, each
             behind the wait on exactly the chunks it overwrites
                                                        (paper Sec. VI-A)
  snapshot = triggered right after the update: pack + chunk sums (HBM ->
             HBM staging) -> chunked D2H -> commit     (paper Sec. V-B, VI-A)
  verify   = H2D + re-check every chunk sum, of the previous step's
             committed snapshot, after this step's has committed (the
             snapshot has the host link to itself, as in training; the first
             step verifies its own)
  restore  = H2D + scatter into the tensors + re-check every chunk sum
The state is generated on the GPU before timing starts.  Prints one JSON
line; `value` is the snapshot rate: payload bytes over the trigger-to-commit
time of the timed steps' snapshots.

Also measured: the pack kernel against the HBM roofline (HIP events that the
library records on its own pack stream around every launch) and against the
same kernel over one contiguous fragment; the pack stream's whole span (pack
launches, release kernels, chunk-sum reduce); D2H against the host link's
measured peak (plain pinned 1 GiB copies in the same process);
restore/verify rates; the step-time overhead of a snapshot every step for 50
steps under the shard's bf16 GEMM load (8192x4096x11008), timed per the
paper's Sec. VII-B per-iteration statistic, with the snapshots in direct D2H
mode (no device staging: the DMA engines copy the fragments into host memory
and the kernels only sum them; --overlap-mode full for the staged pack); and
the CPU oracle on a bounded sample, and the comparison of per-bucket and
whole-range waits before the update with a staging ring (one rank of a 65B
model under TP=8 x PP=8).
"""
import argparse
import json
import math
import os
import subprocess
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "snapshot GB/s (HBM pack+checksum, D2H) + % step overhead under overlap"
HBM_PEAK_GBPS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", type=int, default=4,
                    help="shard of the timed steps (default 4: the 7B LLaMA shard, the largest single-GPU one)")
    ap.add_argument("--no-overlap", action="store_true")
    ap.add_argument("--overlap-steps", type=int, default=50)
    ap.add_argument("--overlap-workload", type=int, default=0, help="0 = the --workload shard (its context reused)")
    ap.add_argument("--overlap-base-steps", type=int, default=20,
                    help="steps of each of the two no-snapshot runs (0 = --overlap-steps)")
    ap.add_argument("--overlap-ratios", default="1.5",
                    help="compute window / standalone snapshot time ratios to run, comma-separated (first = "
                         "headline); each entry also gives the floor max(0, T_snapshot - base step) / base step")
    ap.add_argument("--overlap-gating", choices=["buckets", "whole"], default="buckets",
                    help="the update's gate: one ckpt_wait per optimizer bucket on its own fragments, or one wait "
                         "on every fragment")
    ap.add_argument("--overlap-only", action="store_true",
                    help="run only the overlap leg and print its JSON")
    ap.add_argument("--no-gating", action="store_true",
                    help="skip the gate-granularity comparison (per-bucket against whole-range waits with a "
                         "staging ring)")
    ap.add_argument("--gating-only", action="store_true", help="run only the gate-granularity comparison")
    ap.add_argument("--gemm-beside-only", action="store_true",
                    help="time the load's GEMM alone, beside host-to-device copies and beside a snapshot's "
                         "device-to-host copies (workload 3)")
    ap.add_argument("--gating-workload", type=int, default=3)
    ap.add_argument("--gating-direct", action="store_true",
                    help="gate comparison in direct D2H mode instead of with a staging ring")
    ap.add_argument("--gating-ratios", default="0.75",
                    help="compute window / snapshot time ratios of the gate comparison (the full sweep: "
                         "0.5,0.75,1.0,1.5)")
    ap.add_argument("--gating-steps", type=int, default=20)
    ap.add_argument("--gating-base-steps", type=int, default=12)
    ap.add_argument("--gating-staging-bytes", type=int, default=256 << 20,
                    help="staging ring of the gate comparison (default: four one-chunk slots)")
    ap.add_argument("--bounce-bytes", type=int, default=-1,
                    help="pageable host images behind pinned bounce rings of this many bytes; 0 = pinned images; "
                         "-1 = 8 GiB rings for workload 4 (two 94.3 GB images exceed the pinned memory the host "
                         "grants), pinned otherwise")
    ap.add_argument("--host-threads", type=int, default=0, help="bounce mode: host copy threads (0 = library default)")
    ap.add_argument("--group-bytes", type=int, default=0,
                    help="bytes per pack launch and DMA request (whole chunks); 0 = the library default (1 GiB, or "
                         "a quarter of the staging ring), except for the timed steps with pageable images, which "
                         "default to 256 MiB groups in 1 GiB pack launches")
    ap.add_argument("--staging-bytes", type=int, default=0,
                    help="device staging: 0 = a full-size image (default); else a ring of slots of one chunk group "
                         "each, at most this many bytes in all, the next pack of a slot waiting for its copy (main "
                         "and overlap legs)")
    ap.add_argument("--pack-launch-bytes", type=int, default=0,
                    help="full-image staging: bytes per pack launch (whole groups); 0 = the library default (one group)")
    ap.add_argument("--d2h-engines", type=int, default=0, help="DMA engines of the snapshot copies (0 = library default)")
    ap.add_argument("--direct", action="store_true",
                    help="direct D2H (ckpt_config.direct_d2h) in the timed steps: no device staging, the DMA engines "
                         "copy the fragments and the kernels only sum")
    ap.add_argument("--overlap-mode", choices=["direct", "full"], default="direct",
                    help="snapshot mode of the overlap leg: direct D2H (default; the mode for a compute window "
                         "longer than the snapshot) or full-image staging with the pack kernel")
    ap.add_argument("--overlap-R", type=int, default=0, help="overlap leg: GEMMs per step (0 = from the ratio)")
    ap.add_argument("--ceiling-bytes", type=int, default=8 << 30,
                    help="size of the contiguous fragment the pack ceiling is measured on")
    ap.add_argument("--image-file", default="",
                    help="bounce mode: keep the host images in this file (crash-surviving; removed at the end)")
    ap.add_argument("--grid-blocks", type=int, default=0,
                    help="overlap leg: cap on the tile kernels' workgroups per launch (0 = one per tile)")
    ap.add_argument("--h2h-only", action="store_true",
                    help="run only the H2H replication leg (ring peer in this process, TCP over 127.0.0.1)")
    ap.add_argument("--h2h-workload", type=int, default=3)
    ap.add_argument("--h2h-steps", type=int, default=5)
    ap.add_argument("--h2h-peers", type=int, default=1,
                    help="replicate each snapshot to this many peers (k of Sec. V-C), all in this process")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--cpu-sample-bytes", type=int, default=10 << 30)
    ap.add_argument("--traffic", type=str, default=os.path.join(ROOT, "profiles", "pack_checksum_llama7b_traffic.txt"),
                    help="rocprofv3 FETCH_SIZE/WRITE_SIZE summary written by --pmc-summary")
    ap.add_argument("--pmc-run", action="store_true",
                    help="short run for counter collection: a 1 GiB plain copy, then two snapshots of --workload, "
                         "a restore and a verify")
    ap.add_argument("--pmc-summary", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="summarize two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE) of --pmc-run")
    ap.add_argument("--stats-summary", metavar="DIR", help="summarize a rocprofv3 --kernel-trace --stats run")
    ap.add_argument("--gemm-inflation", metavar="DIR",
                    help="summarize GEMM durations of a rocprofv3 --kernel-trace --memory-copy-trace run of the "
                         "overlap leg: beside a pack launch, beside a D2H copy, and alone")
    ap.add_argument("--gemm-pmc-run", action="store_true",
                    help="short run for the GEMM counter study: phases of the load's GEMM alone and beside a "
                         "snapshot's device-to-host copies (workload 3); prints the phases as JSON")
    ap.add_argument("--counters-summary", nargs="+", metavar=("KIND", "DIR"),
                    help="KIND pack|gemm, then rocprofv3 --pmc --kernel-trace output folders of --pmc-run (pack) or "
                         "--gemm-pmc-run (gemm; each folder also holds that run's printed JSON as run.json)")
    ap.add_argument("--command", default="", help="command line recorded in a summary")
    ap.add_argument("--bench-json", default="", help="with --stats-summary: the JSON line bench.py printed in that run")
    return ap.parse_args()


DEFAULT_BOUNCE = 8 << 30


PACK_KERNEL = "tile_kernel<0"  # PACK instantiation of the tile kernel
SCATTER_KERNEL = "tile_kernel<1"
VERIFY_KERNEL = "tile_kernel<2"
SUMS_KERNEL = "sums_run_kernel"  # direct D2H
COPY_KERNEL = "__amd_rocclr_copyBuffer"
CALIBRATION_BYTES = 1 << 30


def kernel_source_sha():
    import hashlib

    h = hashlib.sha256()
    for f in ["ckpt_kernels.hip", "ckpt_internal.h"]:
        h.update(open(os.path.join(ROOT, "paper_2607_01646_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


def read_counter_csv(d):
    import csv
    import glob

    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit("no counter_collection.csv under %s" % d)
    rows = []
    for f in files:
        rows += list(csv.DictReader(open(f)))
    return rows


def pmc_summary(fetch_dir, write_dir, command):
    """Per-dispatch FETCH_SIZE / WRITE_SIZE of the pack kernel, scaled by the
    same counters on a plain copy kernel of known size (1 GiB read, 1 GiB
    written), into HBM bytes per launch."""
    out = {"kernel_source_sha": kernel_source_sha(), "command": command}
    others = {"scatter": SCATTER_KERNEL, "verify": VERIFY_KERNEL, "sums": SUMS_KERNEL}
    for name, d in [("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)]:
        rows = [r for r in read_counter_csv(d) if r["Counter_Name"] == name]
        copy = [float(r["Counter_Value"]) for r in rows if COPY_KERNEL in r["Kernel_Name"]
                and int(r["Grid_Size"]) > 1024]
        pack = [float(r["Counter_Value"]) for r in rows if PACK_KERNEL in r["Kernel_Name"]]
        if not copy or not pack:
            raise SystemExit("%s: missing dispatches (copy %d, pack %d)" % (name, len(copy), len(pack)))
        copy_kib = max(copy)  # the 1 GiB calibration copy
        factor = CALIBRATION_BYTES / (copy_kib * 1024.0)
        key = name.split("_")[0].lower()
        out[key + "_kib_per_pack_dispatch"] = sum(pack) / len(pack)
        out[key + "_pack_dispatches"] = len(pack)
        out[key + "_kib_calibration_copy"] = copy_kib
        out[key + "_scale"] = factor
        out[key + "_bytes_per_pack_dispatch"] = sum(pack) / len(pack) * 1024.0 * factor
        for kind, kname in others.items():  # restore and verify passes of the same run, when present
            v = [float(r["Counter_Value"]) for r in rows if kname in r["Kernel_Name"]]
            if v:
                out["%s_%s_dispatches" % (key, kind)] = len(v)
                out["%s_bytes_per_%s_dispatch" % (key, kind)] = sum(v) / len(v) * 1024.0 * factor
    out["traffic_bytes_per_pack_dispatch"] = out["fetch_bytes_per_pack_dispatch"] + out["write_bytes_per_pack_dispatch"]
    for kind in others:
        f, w = out.get("fetch_bytes_per_%s_dispatch" % kind), out.get("write_bytes_per_%s_dispatch" % kind)
        if f is not None and w is not None:
            out["traffic_bytes_per_%s_dispatch" % kind] = f + w
    return out


def write_summary(path, d, header):
    with open(path, "w") as f:
        f.write(header.rstrip() + "\n\n")
        for k, v in d.items():
            f.write("%s: %s\n" % (k, v))


def read_summary(path):
    d = {}
    if not os.path.exists(path):
        return d
    for line in open(path):
        if ": " in line and not line.startswith("#"):
            k, v = line.rstrip("\n").split(": ", 1)
            d[k.strip()] = v.strip()
    return d


def timed_pack_average(d, bench):
    """Average duration (ms) of the pack dispatches of the bench's timed steps,
    from the kernel trace: after the ceiling's passes, (warmup + steps)
    passes of `launches / steps` dispatches each."""
    import csv
    import glob

    files = glob.glob(os.path.join(d, "**", "*kernel_trace.csv"), recursive=True)
    rows = []
    for f in files:
        rows += [r for r in csv.DictReader(open(f)) if PACK_KERNEL in r["Kernel_Name"]]
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    rows = rows[bench["components"]["pack_ceiling"]["launches_total"]:]  # the ceiling's passes come first
    per = bench["roofline"]["launches"] // bench["steps"]
    timed = rows[bench["warmup"] * per:(bench["warmup"] + bench["steps"]) * per]
    durs = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e6 for r in timed]
    return sum(durs) / len(durs), len(durs)


def timed_d2h_from_trace(d, bench):
    """Per timed snapshot of the bench's workload-2 steps: image bytes / (last
    group copy's end - first group copy's start), from the memory-copy trace.
    The group copies are the device-to-host copies longer than 1 ms, in time
    order: (warmup + steps) snapshots of one copy per chunk group each come
    first (the calibration copies before them are blit kernels, not copies)."""
    import csv
    import glob
    import statistics

    copies = []
    for f in glob.glob(os.path.join(d, "**", "*memory_copy_trace.csv"), recursive=True):
        for r in csv.DictReader(open(f)):
            kind = " ".join(str(v) for k, v in r.items() if k and ("Direction" in k or "Kind" in k))
            a, b = int(r["Start_Timestamp"]), int(r["End_Timestamp"])
            if "DEVICE_TO_HOST" in kind and b - a > 1_000_000:
                copies.append((a, b))
    copies.sort()
    per = bench["config"].get("groups_per_snapshot") or bench["roofline"]["launches"] // bench["steps"]
    image = bench["config"]["image_bytes"]
    rates = []
    for k in range(bench["warmup"], bench["warmup"] + bench["steps"]):
        grp = copies[k * per:(k + 1) * per]
        if len(grp) < per:
            break
        span = max(b for _, b in grp) - min(a for a, _ in grp)
        rates.append(image / span)  # bytes per ns = GB/s
    return rates, (statistics.median(rates) if rates else float("nan"))


def stats_summary(d, command):
    """Markdown table of our kernels and copies from a --kernel-trace --stats run."""
    import csv
    import glob

    ks = glob.glob(os.path.join(d, "**", "*kernel_stats.csv"), recursive=True)
    ms = glob.glob(os.path.join(d, "**", "*memory_copy_stats.csv"), recursive=True)
    lines = ["| name | calls | average (us) | min (us) | max (us) | total (ms) |", "|---|---|---|---|---|---|"]
    for f in ks + ms:
        for r in csv.DictReader(open(f)):
            n = r["Name"]
            if "ckpt::" in n or "MEMORY_COPY" in n or COPY_KERNEL in n:
                short = n.replace("void ckpt::(anonymous namespace)::", "").replace("(ckpt::(anonymous namespace)::Args)", "")
                short = short.replace("ckpt::(anonymous namespace)::", "").split("(")[0]
                lines.append("| %s | %s | %.1f | %.1f | %.1f | %.2f |" % (
                    short, r["Calls"], float(r["AverageNs"]) / 1e3, float(r["MinNs"]) / 1e3, float(r["MaxNs"]) / 1e3,
                    float(r["TotalDurationNs"]) / 1e6))
    return "\n".join(lines)


def gemm_inflation(d, command):
    """GEMM dispatch durations of an overlap run, split by what ran beside
    them: a pack (or, in direct D2H mode, sums) launch of the library, a
    device-to-host copy, or neither; and the GEMM time each adds over the
    median of the GEMMs that ran alone."""
    import bisect
    import csv
    import glob
    import statistics

    kt = glob.glob(os.path.join(d, "**", "*kernel_trace.csv"), recursive=True)
    mt = glob.glob(os.path.join(d, "**", "*memory_copy_trace.csv"), recursive=True)
    gemms, packs, sums, copies = [], [], [], []
    for f in kt:
        for r in csv.DictReader(open(f)):
            a, b, n = int(r["Start_Timestamp"]), int(r["End_Timestamp"]), r["Kernel_Name"]
            if PACK_KERNEL in n:
                packs.append((a, b))
            elif SUMS_KERNEL in n:
                sums.append((a, b))
            elif "Cijk" in n or "gemm" in n.lower():
                gemms.append((a, b))
    for f in mt:
        for r in csv.DictReader(open(f)):
            kind = " ".join(str(v) for k, v in r.items() if k and ("Direction" in k or "Kind" in k))
            if "DEVICE_TO_HOST" in kind:
                copies.append((int(r["Start_Timestamp"]), int(r["End_Timestamp"])))

    def overlaps(iv, lst, starts):
        k = bisect.bisect_left(starts, iv[1])  # intervals starting before the GEMM ends
        for j in range(max(0, k - 64), k):
            if lst[j][1] > iv[0]:
                return True
        return False

    sides = [("beside_pack", sorted(packs)), ("beside_sums", sorted(sums)), ("beside_d2h", sorted(copies))]
    starts = {k: [iv[0] for iv in lst] for k, lst in sides}
    groups = {k: [] for k, _ in sides}
    groups["alone"] = []
    for g in gemms:
        key = next((k for k, lst in sides if overlaps(g, lst, starts[k])), "alone")
        groups[key].append((g[1] - g[0]) / 1e3)
    base = statistics.median(groups["alone"]) if groups["alone"] else float("nan")
    lines = ["# GEMM durations under snapshots (rocprofv3 kernel + memory-copy trace)", "",
             "command: `%s`" % command, "",
             "%d GEMM dispatches, %d pack launches, %d sums launches, %d device-to-host copies in the trace." % (
                 len(gemms), len(packs), len(sums), len(copies)), "",
             "| GEMMs | count | median (us) | mean (us) | median vs alone | added over the alone median, in all (ms) |",
             "|---|---|---|---|---|---|"]
    for k, v in groups.items():
        if v:
            lines.append("| %s | %d | %.1f | %.1f | %+.2f%% | %.1f |" % (
                k, len(v), statistics.median(v), statistics.mean(v), 100 * (statistics.median(v) / base - 1),
                sum(x - base for x in v) / 1e3))
    return "\n".join(lines)


def counter_dispatches(d):
    """Per-dispatch counters of one rocprofv3 --pmc --kernel-trace run:
    {dispatch_id: {"name", "grid", "ns", counter: value}} (duration from the
    kernel trace, else from the counter file's own timestamps)."""
    import csv
    import glob

    out = {}
    for r in read_counter_csv(d):
        k = int(r["Dispatch_Id"])
        e = out.setdefault(k, {"name": r["Kernel_Name"], "grid": int(r["Grid_Size"]), "ns": 0})
        e[r["Counter_Name"]] = e.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
        if r.get("Start_Timestamp") and r.get("End_Timestamp"):
            e["ns"] = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
    for f in glob.glob(os.path.join(d, "**", "*kernel_trace.csv"), recursive=True):
        for r in csv.DictReader(open(f)):
            k = int(r["Dispatch_Id"])
            if k in out:
                out[k]["ns"] = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
    return out


def counter_totals(rows):
    """Sum of every counter and of the durations over a list of dispatches."""
    t = {"dispatches": len(rows), "ns": sum(r["ns"] for r in rows)}
    for r in rows:
        for k, v in r.items():
            if k not in ("name", "grid", "ns"):
                t[k] = t.get(k, 0.0) + v
    return t


def counter_readings(t):
    """Derived figures of a class of dispatches whose counters may come from
    several runs (each counter from the run that collected it; every run
    repeats the same dispatches).  Ratios of counters of one clock domain:
    the TCC's (L2 channel) counters among themselves, GRBM among itself."""
    g = t.get
    n = t["dispatches"]
    out = {"dispatches": n, "mean duration (us)": t["ns"] / n / 1e3}
    if g("clock"):
        out["GRBM_COUNT per ns (clock, summed over the counter's instances)"] = t["clock"]
    if g("GRBM_GUI_ACTIVE") and g("GRBM_COUNT"):
        out["GRBM_GUI_ACTIVE / GRBM_COUNT"] = t["GRBM_GUI_ACTIVE"] / t["GRBM_COUNT"]
    if g("TCC_EA0_RDREQ_sum") and g("TCC_EA0_RDREQ_128B_sum") is not None and g("TCC_EA0_RDREQ_64B_sum") is not None:
        n32 = g("TCC_EA0_RDREQ_32B_sum", 0.0)
        by_size = 32 * n32 + 64 * t["TCC_EA0_RDREQ_64B_sum"] + 128 * t["TCC_EA0_RDREQ_128B_sum"]
        out["read requests per dispatch (32/64/128 B)"] = "%.0f / %.0f / %.0f" % (
            n32 / n, t["TCC_EA0_RDREQ_64B_sum"] / n, t["TCC_EA0_RDREQ_128B_sum"] / n)
        out["read bytes per dispatch from request sizes"] = by_size / n
        out["read requests not of 32/64/128 B"] = (t["TCC_EA0_RDREQ_sum"] - n32 - t["TCC_EA0_RDREQ_64B_sum"]
                                                    - t["TCC_EA0_RDREQ_128B_sum"]) / n
    if g("TCC_BUBBLE_sum") is not None and g("TCC_EA0_RDREQ_sum") and g("TCC_EA0_RDREQ_32B_sum") is not None:
        b, rq, n32 = t["TCC_BUBBLE_sum"], t["TCC_EA0_RDREQ_sum"], t["TCC_EA0_RDREQ_32B_sum"]
        out["TCC_BUBBLE (128-byte requests by FETCH_SIZE's count) per dispatch"] = b / n
        out["read bytes per dispatch by FETCH_SIZE's formula"] = (128 * b + 64 * (rq - b - n32) + 32 * n32) / n
    if g("TCC_EA0_WRREQ_sum") and g("TCC_EA0_WRREQ_64B_sum") is not None:
        w, w64 = t["TCC_EA0_WRREQ_sum"], t["TCC_EA0_WRREQ_64B_sum"]
        out["write bytes per dispatch (WRITE_SIZE's formula)"] = (64 * w64 + 32 * (w - w64)) / n
    if g("TCC_EA0_RDREQ_LEVEL_sum") and g("TCC_EA0_RDREQ_sum"):
        out["EA read latency (TCC cycles, in-flight level / requests)"] = (t["TCC_EA0_RDREQ_LEVEL_sum"]
                                                                           / t["TCC_EA0_RDREQ_sum"])
    if g("TCC_EA0_WRREQ_LEVEL_sum") and g("TCC_EA0_WRREQ_sum"):
        out["EA write latency (TCC cycles)"] = t["TCC_EA0_WRREQ_LEVEL_sum"] / t["TCC_EA0_WRREQ_sum"]
    busy = g("TCC_BUSY_sum")
    if busy:
        if g("TCC_BUSY_avr"):
            out["TCC channels (TCC_BUSY_sum / TCC_BUSY_avr)"] = busy / t["TCC_BUSY_avr"]
        for k, label in [("TCC_EA0_RDREQ_LEVEL_sum", "reads in flight per channel per busy cycle"),
                         ("TCC_EA0_WRREQ_LEVEL_sum", "writes in flight per channel per busy cycle"),
                         ("TCC_EA0_RDREQ_DRAM_CREDIT_STALL_sum", "read DRAM-credit stall cycles / busy cycles"),
                         ("TCC_EA0_WRREQ_DRAM_CREDIT_STALL_sum", "write DRAM-credit stall cycles / busy cycles"),
                         ("TCC_EA0_WRREQ_STALL_sum", "write-request stall cycles / busy cycles"),
                         ("TCC_TAG_STALL_sum", "tag stall cycles / busy cycles")]:
            if g(k) is not None:
                out[label] = t[k] / busy
        if g("TCC_WRREQ_STALL_max") is not None and g("TCC_EA0_WRREQ_STALL_sum") and g("TCC_BUSY_avr"):
            ch = busy / t["TCC_BUSY_avr"]
            out["write stalls: busiest channel / channel mean"] = t["TCC_WRREQ_STALL_max"] / (
                t["TCC_EA0_WRREQ_STALL_sum"] / ch)
    if g("TCC_HIT_sum") is not None and g("TCC_MISS_sum") is not None and t["TCC_HIT_sum"] + t["TCC_MISS_sum"] > 0:
        out["L2 hit rate"] = t["TCC_HIT_sum"] / (t["TCC_HIT_sum"] + t["TCC_MISS_sum"])
    if g("TCC_EA0_RDREQ_sum"):
        out["EA read requests per dispatch"] = t["TCC_EA0_RDREQ_sum"] / n
    if g("TCC_EA0_RDREQ_DRAM_sum") is not None and g("TCC_EA0_RDREQ_sum"):
        out["read requests to DRAM / all read requests"] = t["TCC_EA0_RDREQ_DRAM_sum"] / t["TCC_EA0_RDREQ_sum"]
    if g("TCC_EA0_WRREQ_DRAM_sum") is not None and g("TCC_EA0_WRREQ_sum"):
        out["write requests to DRAM / all write requests"] = t["TCC_EA0_WRREQ_DRAM_sum"] / t["TCC_EA0_WRREQ_sum"]
    if g("TA_BUSY_avr") and g("TA_BUSY_max"):
        # (the least busy TA belongs to a compute unit that the part does not enable, so it reads 0)
        out["TA busy: mean / busiest instance"] = t["TA_BUSY_avr"] / t["TA_BUSY_max"]
    if g("TA_BUSY_avr") and g("GRBM_GUI_ACTIVE"):
        out["TA_BUSY_avr per dispatch (cycles)"] = t["TA_BUSY_avr"] / n
    if g("TD_TD_BUSY_sum"):
        out["TD_TD_BUSY_sum per dispatch (cycles)"] = t["TD_TD_BUSY_sum"] / n
    if g("TCP_TCC_READ_REQ_LATENCY_sum") and g("TCP_TCC_READ_REQ_sum"):
        out["TCP->TCC read latency (cycles)"] = t["TCP_TCC_READ_REQ_LATENCY_sum"] / t["TCP_TCC_READ_REQ_sum"]
    if g("TCP_PENDING_STALL_CYCLES_sum") is not None:
        out["TCP_PENDING_STALL_CYCLES_sum per dispatch"] = t["TCP_PENDING_STALL_CYCLES_sum"] / n
    if g("TCP_TCR_TCP_STALL_CYCLES_sum") is not None:
        out["TCP_TCR_TCP_STALL_CYCLES_sum per dispatch"] = t["TCP_TCR_TCP_STALL_CYCLES_sum"] / n
    for k, label in [("SQ_BUSY_CYCLES", "SQ_BUSY_CYCLES per dispatch"),
                     ("SQ_VALU_MFMA_BUSY_CYCLES", "SQ_VALU_MFMA_BUSY_CYCLES per dispatch"),
                     ("SQ_WAVE_CYCLES", "SQ_WAVE_CYCLES per dispatch"),
                     ("SQ_INSTS_VALU_MFMA_MOPS_BF16", "SQ_INSTS_VALU_MFMA_MOPS_BF16 per dispatch"),
                     ("GRBM_GUI_ACTIVE", "GRBM_GUI_ACTIVE per dispatch")]:
        if g(k) is not None:
            out[label] = t[k] / n
    if g("SQ_VALU_MFMA_BUSY_CYCLES") and g("GRBM_GUI_ACTIVE"):
        out["SQ_VALU_MFMA_BUSY_CYCLES / GRBM_GUI_ACTIVE"] = t["SQ_VALU_MFMA_BUSY_CYCLES"] / t["GRBM_GUI_ACTIVE"]
    return out


def merge_totals(parts):
    """One class's totals from several runs: each counter from the first run
    that collected it, scaled to the first run's dispatch count (a GEMM
    phase's length differs between runs), and the durations from the first
    run.  The clock comes from the run that counted GRBM_COUNT, over that
    run's own durations."""
    t = dict(parts[0])
    for p in parts[1:]:
        for k, v in p.items():
            if k not in ("dispatches", "ns") and k not in t:
                t[k] = v * t["dispatches"] / p["dispatches"]
    for p in parts:
        if p.get("GRBM_COUNT") and p["ns"]:
            t["clock"] = p["GRBM_COUNT"] / p["ns"]
            break
    return t


def pack_classes(disp):
    """The pack run's dispatches by kernel: the 1 GiB calibration copy, the
    pack, scatter and verify tile kernels."""
    rows = [disp[k] for k in sorted(disp)]
    copies = [r for r in rows if COPY_KERNEL in r["name"] and r["grid"] > 1024]  # the run's first large copy
    return {"calibration copy (1 GiB)": copies[:1],
            "pack": [r for r in rows if PACK_KERNEL in r["name"]],
            "scatter": [r for r in rows if SCATTER_KERNEL in r["name"]],
            "verify": [r for r in rows if VERIFY_KERNEL in r["name"]]}


def gemm_classes(d, disp):
    """The GEMM run's dispatches by phase, from the phase list the run
    printed (run.json in the same folder): the GEMM kernel's dispatches in
    order, cut by the phases' counts."""
    lines = [x for x in open(os.path.join(d, "run.json")).read().splitlines() if x.startswith('{"workload"')]
    phases = json.loads(lines[-1])["phases"]
    names = {}
    for r in disp.values():
        names[r["name"]] = names.get(r["name"], 0) + 1
    gemm = max(names, key=names.get)
    rows = [disp[k] for k in sorted(disp) if disp[k]["name"] == gemm]
    if len(rows) != sum(c for _, c in phases):
        raise SystemExit("%s: %d GEMM dispatches, phases list %d" % (d, len(rows), sum(c for _, c in phases)))
    out, i = {}, 0
    for name, c in phases:
        out.setdefault(name, []).extend(rows[i:i + c])
        i += c
    out.pop("warmup", None)
    return out


def counters_summary(kind, dirs, command):
    """Markdown table of counter readings per kernel class (pack run) or per
    phase (GEMM run), over one or more rocprofv3 --pmc runs."""
    per_dir = []
    for d in dirs:
        disp = counter_dispatches(d)
        cls = pack_classes(disp) if kind == "pack" else gemm_classes(d, disp)
        per_dir.append({k: counter_totals(v) for k, v in cls.items() if v})
    names = [k for k in per_dir[0]]
    tables = {k: counter_readings(merge_totals([p[k] for p in per_dir if k in p])) for k in names}
    # GEMM phases: also each phase against the GEMMs alone
    rel = [c for c in names if c != "alone"] if "alone" in tables else []
    keys = list(tables[names[0]])
    keys += sorted({k for c in names for k in tables[c]} - set(keys))
    rows = []
    for k in keys:
        vals = []
        for c in names:
            v = tables[c].get(k)
            vals.append("" if v is None else v if isinstance(v, str) else "%.4g" % v)
        for c in rel:
            a, v = tables["alone"].get(k), tables[c].get(k)
            ok = isinstance(a, float) and isinstance(v, float) and a != 0 and k != "dispatches"
            vals.append("%+.2f%%" % (100 * (v / a - 1)) if ok else "")
        rows.append("| %s | %s |" % (k, " | ".join(vals)))
    cols = names + ["%s vs alone" % c for c in rel]
    head = ["command: `%s`" % command, "", "| | %s |" % " | ".join(cols), "|---|%s" % ("---|" * len(cols))]
    return "\n".join(head + rows)


def gemm_pmc_run(torch, P, W, wid=3, reps=3):
    """Short run for the counter study of the load's GEMM: phases of GEMMs
    alone and beside a snapshot's device-to-host copies after its pack has
    finished.  GEMMs go in batches of 10 with a host synchronisation after
    each, and the 'beside' phase stops once the snapshot has committed: every
    GEMM of that phase but those of its last batch ran beside the copies, also
    when a counter tool serializes the dispatches.  Prints the phases (name,
    GEMM dispatches) as JSON."""
    M, K, N = W.OVERLAP_GEMM[wid]
    x = torch.randn(M, K, device="cuda", dtype=torch.bfloat16)
    w = torch.randn(K, N, device="cuda", dtype=torch.bfloat16)
    tensors, plan = W.make_state(wid, device="cuda")
    ck = P.Checkpointer(tensors, chunk_bytes=W.WORKLOADS[wid]["chunk"])
    for k in range(2):
        s = ck.snapshot(step=k)
        ck.wait_committed(s)
    phases = []

    def run(name, busy, cap):
        n = 0
        while n < cap and busy():
            for _ in range(10):
                torch.matmul(x, w)
            torch.cuda.synchronize()
            n += 10
        phases.append([name, n])
        return n

    run("warmup", lambda: True, 20)
    for rep in range(reps):
        run("alone", lambda: True, 200)
        s = ck.snapshot(step=10 + rep)
        ck.wait_captured(s)
        torch.cuda.synchronize()  # the pack has finished; the copies run
        run("beside_d2h", lambda: ck.state(s) == P.CKPT_SNAP_IN_FLIGHT, 2000)
        ck.wait_committed(s)
        log("gemm pmc run: rep %d, phases %s" % (rep, phases[-2:]))
    ck.close()
    print(json.dumps({"workload": W.WORKLOADS[wid]["name"], "gemm_mkn": [M, K, N], "phases": phases}), flush=True)


_T0 = time.perf_counter()


def log(*a):
    print("[bench +%.0fs]" % (time.perf_counter() - _T0), *a, file=sys.stderr, flush=True)


def trimmed_mean(xs, warm=10, drop=0.05):
    """Paper Sec. VII-B (per-iteration overhead): discard the first 10 iterations, drop the slowest 5%
    of the rest, average."""
    xs = list(xs[warm:]) if len(xs) > warm else list(xs)
    xs.sort()
    keep = len(xs) - int(math.floor(len(xs) * drop))
    xs = xs[:max(keep, 1)]
    return sum(xs) / len(xs)


def link_peak(torch):
    """Plain pinned 1 GiB D2H / H2D copies: the host link's measured peak,
    the best of one 1 GiB copy and of 2 or 4 concurrent copies of its parts
    on their own streams (wall time from the first start to the last end)."""
    n = 1 << 30
    h = torch.empty(n, dtype=torch.uint8, pin_memory=True)
    d = torch.empty(n, dtype=torch.uint8, device="cuda")
    d.fill_(7)
    streams = [torch.cuda.Stream() for _ in range(4)]
    out = {}
    for name in ("d2h", "h2d"):
        best = 1e9
        for parts in (1, 2, 4):
            per = n // parts
            dst, src = (h, d) if name == "d2h" else (d, h)

            def run():
                start = torch.cuda.Event(enable_timing=True)
                start.record()
                ends = []
                for k in range(parts):
                    st = streams[k]
                    st.wait_event(start)
                    with torch.cuda.stream(st):
                        dst[k * per:(k + 1) * per].copy_(src[k * per:(k + 1) * per], non_blocking=True)
                        e = torch.cuda.Event(enable_timing=True)
                        e.record(st)
                        ends.append(e)
                for e in ends:
                    e.synchronize()
                return max(start.elapsed_time(e) for e in ends)

            run()
            for _ in range(5):
                best = min(best, run())
        out[name] = n / best / 1e6
    torch.cuda.synchronize()
    del h, d
    return out


def host_cpus():
    """Cores the oracle may use here (this process's CPU affinity, capped by a
    cgroup CPU quota when one is set) and what the host reports about itself."""
    aff = len(os.sched_getaffinity(0))
    quota = None
    try:
        q, per = open("/sys/fs/cgroup/cpu.max").read().split()
        if q != "max":
            quota = int(q) / int(per)
    except (OSError, ValueError):
        pass
    usable = aff if quota is None else max(1, min(aff, int(quota)))
    topo = {}
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            k, _, v = line.partition(":")
            if k.strip() in ("Model name", "Socket(s)", "Core(s) per socket", "Thread(s) per core", "CPU(s)",
                             "NUMA node(s)"):
                topo[k.strip()] = v.strip()
    except (OSError, subprocess.SubprocessError):
        pass
    return usable, {"os_cpu_count": os.cpu_count(), "affinity_cpus": aff, "cgroup_quota_cpus": quota,
                    "threads_used": usable, "lscpu": topo}


def cpu_baseline(tensors, chunk, target_bytes):
    """The oracle as it stands, on the first fragments of the shard up to
    target_bytes: pack + chunk sums + restore + verify (the GPU step's
    kernels' work, without the host-link copies a CPU does not need).  Timed
    with the image split by whole chunks over every core this process may use
    (the oracle's C calls run outside the interpreter lock), and on one
    thread."""
    from concurrent.futures import ThreadPoolExecutor

    import numpy as np
    import torch

    import oracle as O

    frags, total = [], 0
    for t in tensors:
        nb = t.numel() * t.element_size()
        if total and total + nb > target_bytes:
            break
        frags.append(t.detach().cpu().reshape(-1).view(torch.uint8).numpy())
        total += nb
    sizes = [f.size for f in frags]
    O.lib()
    off, I, nc = O.layout(sizes, 256, chunk)

    def cycle(lo, hi):
        t0 = time.perf_counter()
        win = O.pack_window(frags, off, lo, hi)
        sums = O.chunk_sums(win, lo, hi, chunk)
        t1 = time.perf_counter()
        back = O.restore_window(win, lo, hi, off, sizes)
        bad = O.verify(win, lo, hi, chunk, sums)
        t2 = time.perf_counter()
        return t1 - t0, t2 - t1, bad, back

    nthr, host = host_cpus()
    per = (nc + nthr - 1) // nthr
    parts = [(k * per * chunk, min((k + 1) * per * chunk, I)) for k in range(nthr) if k * per * chunk < I]
    t0 = time.perf_counter()
    with ThreadPoolExecutor(len(parts)) as ex:
        res = list(ex.map(lambda r: cycle(*r)[2], parts))
    dtn = time.perf_counter() - t0
    assert all(r == [] for r in res)
    t0 = time.perf_counter()
    t_pack, t_rest, bad, back = cycle(0, I)
    dt1 = time.perf_counter() - t0
    assert bad == [] and all(np.array_equal(a, b) for a, b in zip(frags[:3], back[:3]))
    del back
    return {"value": round(total / dtn / 1e9, 3), "unit": "GB/s", "cores": len(parts), "kind": "oracle",
            "sample": "first %d of %d fragments of the shard (%d bytes, %d chunks of %d MiB): pack + chunk sums + "
                      "restore + verify, split by whole chunks over %d threads (%.2f s), and on one thread (%.1f s)"
                      % (len(frags), len(tensors), total, nc, chunk >> 20, len(parts), dtn, dt1),
            "host": host,
            "single_thread": {"value": round(total / dt1 / 1e9, 3), "cores": 1, "seconds": round(dt1, 2),
                              "pack_checksum_GBps": round(2 * total / t_pack / 1e9, 3),
                              "restore_verify_GBps": round(total / t_rest / 1e9, 3)}}


def buckets_of(plan, n_buckets):
    """Contiguous runs of whole parameters (4 fragments each: param, master,
    m, v) of about equal bytes: the optimizer's buckets, in registration order."""
    sizes = [sum(p[1] for p in plan[i:i + 4]) for i in range(0, len(plan), 4)]
    total, out, lo, acc = sum(sizes), [], 0, 0
    for j, z in enumerate(sizes):
        acc += z
        if acc >= total * (len(out) + 1) / n_buckets or j == len(sizes) - 1:
            out.append((lo * 4, (j + 1) * 4))
            lo = j + 1
    return out


class Optimizer:
    """An in-place optimizer-like update of every registered fragment (read
    and write of all 14 bytes per parameter, like an Adam step): m *= 0.9,
    v *= 0.999, master -= 1e-3 * m, param = master.  update(lo, hi) touches
    fragments [lo, hi) only; each bucket can be gated by ckpt_wait(CAPTURED)
    on exactly the fragments it overwrites."""

    def __init__(self, torch, tensors):
        self.torch = torch
        self.t = tensors

    def update(self, lo, hi):
        T = self.torch
        p, w, m, v = self.t[lo:hi:4], self.t[lo + 1:hi:4], self.t[lo + 2:hi:4], self.t[lo + 3:hi:4]
        T._foreach_mul_(m, 0.9)
        T._foreach_mul_(v, 0.999)
        T._foreach_add_(w, m, alpha=-1e-3)
        for a, b in zip(p, w):
            a.copy_(b)


def pack_ceiling(torch, P, nbytes, chunk, launch=0):
    """The same pack kernel over one contiguous, 16-byte-aligned fragment of
    nbytes (1 GiB launches, as for the shard): pack-only passes (the offload
    is cut before its first copy, so the link stays idle), each right after
    an in-place update of the fragment (as a snapshot follows the optimizer
    step), and each after a host synchronisation with the GPU idle."""
    buf = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    buf.view(torch.int32).random_()
    ck = P.Checkpointer([buf], chunk_bytes=chunk, pack_launch_bytes=launch)
    P.ckpt_set_timing(ck.ctx, True)

    def one(update):
        if update:
            buf.view(torch.int32).add_(0)
        else:
            torch.cuda.synchronize()
        P.ckpt_debug_interrupt_next(ck.ctx, 0)
        s = ck.snapshot()
        ck.wait_captured(s, 0, 1)
        torch.cuda.current_stream().synchronize()
        return P.ckpt_last_timing(ck.ctx, P.CKPT_OP_PACK)

    one(True)
    out = {}
    for name, update in (("after_update", True), ("idle", False)):
        ts = [one(update) for _ in range(3)]
        ms = sum(t["kernel_ms"] for t in ts)
        out[name + "_GBps"] = round(2 * nbytes * 3 / ms / 1e6, 1)
        out[name + "_avg_launch_ms"] = round(ms / sum(t["kernels"] for t in ts), 4)
    out["bytes"] = nbytes
    out["launches_per_pass"] = ts[0]["kernels"]
    out["launches_total"] = 7 * ts[0]["kernels"]  # the first pass, then three after an update and three idle
    ck.close()
    del buf
    torch.cuda.empty_cache()
    return out


def standalone_snapshot(P, ck, link_d2h_gbps, runs=3, warm=1):
    """Snapshot time alone, trigger to commit: the median of `runs` snapshots
    after `warm` warm-up snapshots (the first snapshots of a context also set
    up its records).  Returns (median ms, [runs ms], [DMA spans ms], pack
    launches per snapshot, [kernel GB/s of each run: the snapshot's
    algorithmic kernel bytes over its launches' summed durations])."""
    P.ckpt_set_timing(ck.ctx, True)
    t_runs, copy_runs, kernel_runs = [], [], []
    for k in range(warm + runs):
        s = ck.snapshot(step=k)
        ck.wait_committed(s)
        tm = P.ckpt_last_timing(ck.ctx, P.CKPT_OP_SNAPSHOT)
        t = tm["total_ms"]
        if t <= 0:  # engine timestamps unavailable (a copy tracer owns the signals)
            t = ck.image_bytes / link_d2h_gbps / 1e6
        if k >= warm:
            t_runs.append(t)
            copy_runs.append(tm["copy_ms"])
            kernel_runs.append(tm["kernel_bytes"] / tm["kernel_ms"] / 1e6 if tm["kernel_ms"] > 0 else None)
    P.ckpt_set_timing(ck.ctx, False)
    return sorted(t_runs)[len(t_runs) // 2], t_runs, copy_runs, tm["kernels"], kernel_runs


def overlap_leg(torch, P, W, wid, steps, link_d2h_gbps, ratios=(1.5,), base_steps=0, bounce=0, threads=0,
                grid_blocks=0, staging=0, group=0, shared=None, gating="buckets", n_buckets=8, launch=0,
                snap=None, engines=0, fixed_R=0, direct=False, state=None):
    """Step-time overhead of per-step snapshots under a bf16 GEMM load.

    One step: R back-to-back GEMMs on the compute stream, then the optimizer
    update in buckets, each gated by ckpt_wait(CAPTURED) on exactly the
    fragments it overwrites (gating="buckets"; "whole": one wait on every
    fragment before the first bucket); the snapshot is issued right after
    the previous update.  R is fixed before measuring as
    ceil(ratio * T_D2H / T_GEMM) from the standalone snapshot time (trigger
    to commit) and the GEMM time; the headline uses the first ratio.
    Overhead compares the mean step (paper Sec. VII-B per-iteration
    statistic) with and without snapshots; the no-snapshot runs bracket the
    snapshot run.  shared = (tensors, plan, checkpointer) reuses a registered
    state instead of making one; state = (tensors, plan) registers existing
    tensors in a context of this leg's own."""
    base_steps = base_steps or steps
    if shared is None:
        tensors, plan = state if state is not None else W.make_state(wid, device="cuda")
        ck = P.Checkpointer(tensors, [p[2] for p in plan], [p[3] for p in plan],
                            chunk_bytes=W.WORKLOADS[wid]["chunk"], bounce_bytes=bounce, host_threads=threads,
                            grid_blocks=grid_blocks, device_staging_bytes=staging, group_bytes=group,
                            pack_launch_bytes=launch, d2h_engines=engines, direct=direct)
    else:
        tensors, plan, ck = shared
    n = len(tensors)
    M, K, N = W.OVERLAP_GEMM[wid]
    x = torch.randn(M, K, device="cuda", dtype=torch.bfloat16)
    w = torch.randn(K, N, device="cuda", dtype=torch.bfloat16)
    for _ in range(5):
        torch.matmul(x, w)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(50):
        torch.matmul(x, w)
    e1.record()
    e1.synchronize()
    t_gemm = e0.elapsed_time(e1) / 50
    # Standalone snapshot (trigger to commit), unless the caller measured it
    t_d2h, d2h_runs, copy_runs, ck_groups, kernel_runs = snap or standalone_snapshot(P, ck, link_d2h_gbps)
    opt = Optimizer(torch, tensors)
    bks = buckets_of(plan, n_buckets)
    calls = []  # host time of each snapshot call

    def run(with_snap, R, steps, mode):
        times = []
        snap = None
        for k in range(steps):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            if with_snap:
                if snap is not None:  # one snapshot in flight: a D2H longer than the step shows up here
                    ck.wait_committed(snap)
                tc = time.perf_counter()
                snap = ck.snapshot(step=k)
                calls.append((time.perf_counter() - tc) * 1e3)
            for _ in range(R):
                torch.matmul(x, w)
            if with_snap and mode == "whole":
                ck.wait_captured(snap, 0, n)
            for lo, hi in bks:
                if with_snap and mode == "buckets":
                    ck.wait_captured(snap, lo, hi)
                opt.update(lo, hi)
            torch.cuda.synchronize()
            times.append((time.perf_counter() - t0) * 1e3)
            if (k + 1) % 10 == 0:
                log("overlap: %s, %d/%d steps, last %.1f ms" % (
                    ("snapshots, %s gating" % mode) if with_snap else "baseline", k + 1, steps, times[-1]))
        return times

    sweep = []
    for ratio in ratios:
        R = fixed_R or int(math.ceil(ratio * t_d2h / t_gemm))
        log("overlap: ratio %.2f, R = %d GEMMs per step" % (ratio, R))
        base1 = run(False, R, base_steps, None)
        withs = run(True, R, steps, gating)
        base2 = run(False, R, base_steps, None)
        b = trimmed_mean(base1 + base2[10:], warm=10)
        wv = trimmed_mean(withs, warm=10)
        sweep.append({"window_over_d2h": ratio, "R": R, "base_ms": round(b, 2), "with_snapshot_ms": round(wv, 2),
                      "overhead_pct": round(100 * (wv - b) / b, 3),
                      "floor_pct": round(100 * max(0.0, t_d2h - b) / b, 3)})
    # The recovery side in this context's mode: verify, then restore, of the
    # newest committed snapshot (the tensors already hold its bytes).
    recovery = None
    if ck.latest()[0]:
        P.ckpt_set_timing(ck.ctx, True)
        bad = ck.verify(0)
        tv = P.ckpt_last_timing(ck.ctx, P.CKPT_OP_VERIFY)
        bad += ck.restore(0)
        tr = P.ckpt_last_timing(ck.ctx, P.CKPT_OP_RESTORE)
        P.ckpt_set_timing(ck.ctx, False)
        if bad:
            raise RuntimeError("checksum mismatch after the overlap run: %s" % bad)
        recovery = {"verify_GBps": round(tv["copy_bytes"] / tv["total_ms"] / 1e6, 2),
                    "restore_GBps": round(tr["copy_bytes"] / tr["total_ms"] / 1e6, 2),
                    "scatter_GBps": round(tr["kernel_bytes"] / tr["kernel_ms"] / 1e6, 1),
                    "note": "H2D + checks (+ scatter) of the newest committed snapshot, after the overlap run"}
    if shared is None:
        ck.close()
        del tensors
    del x, w
    torch.cuda.empty_cache()
    mode = ("direct D2H: no device staging; the DMA engines copy the fragments into host memory and the kernels only "
            "sum them (ckpt_config.direct_d2h)" if direct else
            "pack into device staging, then DMA from the staging")
    head = sweep[0]
    out = {"workload": W.WORKLOADS[wid]["name"], "snapshot_mode": mode,
           "payload_bytes": sum(p[1] for p in plan), "gemm_mkn": [M, K, N],
           "host_images": "pageable, %d-byte pinned bounce rings" % bounce if bounce else "pinned",
           "device_staging": ("none (direct D2H: the engines copy the fragments, the kernels only sum)"
                              if direct
                              else staging_text(staging, W.WORKLOADS[wid]["chunk"])),
           "pack_launches_per_snapshot": ck_groups,
           "tile_kernel_workgroups": grid_blocks or "one per tile",
           "gating": "%d buckets, each behind ckpt_wait(CAPTURED) on its own fragments" % len(bks)
                     if gating == "buckets" else "one ckpt_wait(CAPTURED) on every fragment",
           "gemm_ms": round(t_gemm, 4), "snapshot_ms": round(t_d2h, 2),
           "snapshot_runs_ms": [round(t, 2) for t in d2h_runs],
           "snapshot_kernel_GBps": [round(g, 1) if g else None for g in kernel_runs],
           "snapshot_kernel_note": ("the standalone snapshots' kernels: algorithmic bytes (%s) over the launches' "
                                    "summed durations (HIP events), HBM peak 8000 GB/s"
                                    % ("S, the sums read the fragments" if direct else "2 S, the pack")),
           "snapshot_alone_GBps": round(sum(p[1] for p in plan) / t_d2h / 1e6, 2),
           "d2h_alone_GBps": round(ck.image_bytes / sorted(copy_runs)[1] / 1e6, 2) if min(copy_runs) > 0 else None,
           "d2h_link_peak_GBps": round(link_d2h_gbps, 2),
           "R": head["R"], "steps": steps,
           "base_steps": base_steps, "base_ms": head["base_ms"], "with_snapshot_ms": head["with_snapshot_ms"],
           "overhead_pct": head["overhead_pct"],
           "snapshot_call_ms": round(sorted(calls)[len(calls) // 2], 3) if calls else None,
           "statistic": "mean after dropping 10 warm-up steps and the slowest 5%"}
    if out["d2h_alone_GBps"]:
        out["d2h_alone_frac_of_link"] = round(out["d2h_alone_GBps"] / link_d2h_gbps, 4)
    if recovery:
        out["recovery"] = recovery
    if len(sweep) > 1:
        out["sweep"] = sweep
    return out


class ClockSampler:
    """Background reader of the GPU's own telemetry (amdsmi GPU metrics, read
    only): graphics clock per XCD, socket power and memory clock, every
    `period` s, so that a phase's GEMM durations can be set against the
    clock they ran at.  `error` holds the reason when the metrics cannot be
    read; the phases then report no telemetry."""

    def __init__(self, torch, period=0.01):
        import threading

        self.samples, self.error, self.period = [], None, period
        self._stop = threading.Event()
        try:
            import amdsmi

            amdsmi.amdsmi_init()
            self._smi = amdsmi
            p = torch.cuda.get_device_properties(torch.cuda.current_device())
            want = "%04x:%02x:%02x" % (p.pci_domain_id, p.pci_bus_id, p.pci_device_id)
            handles = amdsmi.amdsmi_get_processor_handles()
            match = [h for h in handles if amdsmi.amdsmi_get_gpu_device_bdf(h).lower().startswith(want)]
            if not match and len(handles) != 1:
                raise RuntimeError("no amdsmi device at %s among %d" % (want, len(handles)))
            self._h = (match or handles)[0]
            self._read()
        except Exception as e:  # telemetry is optional: the timing stands without it
            self.error = "%s: %s" % (type(e).__name__, e)
            return
        self._t = threading.Thread(target=self._run, daemon=True)
        self._t.start()

    def _read(self):
        m = self._smi.amdsmi_get_gpu_metrics_info(self._h)
        clks = [c for c in (m.get("current_gfxclks") or []) if isinstance(c, (int, float)) and c > 0]
        num = lambda k: m.get(k) if isinstance(m.get(k), (int, float)) else None  # noqa: E731
        return {"t": time.perf_counter(), "gfxclk": sum(clks) / len(clks) if clks else num("current_gfxclk"),
                "power": num("current_socket_power"), "uclk": num("current_uclk"),
                "throttle": m.get("indep_throttle_status")}

    def _run(self):
        while not self._stop.is_set():
            try:
                self.samples.append(self._read())
            except Exception as e:
                self.error = "%s: %s" % (type(e).__name__, e)
                return
            self._stop.wait(self.period)

    def stop(self):
        self._stop.set()
        if self.error is None:
            self._t.join()
            try:
                self._smi.amdsmi_shut_down()
            except Exception:
                pass

    def window(self, t0, t1):
        """Mean clock (MHz), socket power (W) and memory clock over [t0, t1]."""
        s = [x for x in self.samples if t0 <= x["t"] <= t1]
        out = {"samples": len(s)}
        for k in ("gfxclk", "power", "uclk"):
            v = [x[k] for x in s if x[k] is not None]
            out[k] = sum(v) / len(v) if v else None
        out["throttled_samples"] = sum(1 for x in s if x["throttle"] not in (None, 0, False, "N/A"))
        return out


def gemm_beside_leg(torch, P, W, wid=3, reps=5):
    """Where the step overhead under snapshots comes from: the load's GEMM
    timed alone, beside host -> device copies on the DMA engines (torch's
    pinned copies, 3 x 8 GiB), and beside a snapshot's device -> host copies
    (the library, after its pack).  Alternating, median of the middle runs."""
    M, K, N = W.OVERLAP_GEMM[wid]
    x = torch.randn(M, K, device="cuda", dtype=torch.bfloat16)
    w = torch.randn(K, N, device="cuda", dtype=torch.bfloat16)
    tensors, plan = W.make_state(wid, device="cuda")
    ck = P.Checkpointer(tensors, chunk_bytes=W.WORKLOADS[wid]["chunk"])
    for k in range(2):
        s = ck.snapshot(step=k)
        ck.wait_committed(s)
    host = torch.empty(8 << 30, dtype=torch.uint8, pin_memory=True)
    dev = torch.empty(8 << 30, dtype=torch.uint8, device="cuda")
    side = torch.cuda.Stream()

    def gemms(n):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(n):
            torch.matmul(x, w)
        e1.record()
        e1.synchronize()
        return e0.elapsed_time(e1) / n

    gemms(50)
    res = {"alone": [], "beside_h2d": [], "beside_d2h": []}
    clock = ClockSampler(torch)
    windows = {k: [] for k in res}

    def timed(kind, n):
        t0 = time.perf_counter()
        res[kind].append(gemms(n))
        windows[kind].append((t0, time.perf_counter()))

    for rep in range(reps):
        torch.cuda.synchronize()
        timed("alone", 300)
        torch.cuda.synchronize()
        with torch.cuda.stream(side):
            for _ in range(3):
                dev.copy_(host, non_blocking=True)
        timed("beside_h2d", 300)
        torch.cuda.synchronize()
        s = ck.snapshot(step=10 + rep)
        time.sleep(0.01)  # past the pack (a few ms), into the copies (~250 ms)
        timed("beside_d2h", 250)
        ck.wait_committed(s)
        log("gemm beside: rep %d" % rep)
    clock.stop()
    ck.close()
    del tensors, host, dev, x, w
    torch.cuda.empty_cache()

    def mid(v):
        v = sorted(v)
        return sum(v[1:-1]) / len(v[1:-1])

    def telemetry(kind):  # sample-weighted over every window of the phase
        parts = [clock.window(a, b) for a, b in windows[kind]]
        out = {"samples": sum(p["samples"] for p in parts),
               "throttled_samples": sum(p["throttled_samples"] for p in parts)}
        for k in ("gfxclk", "power", "uclk"):
            num = sum(p[k] * p["samples"] for p in parts if p[k] is not None)
            den = sum(p["samples"] for p in parts if p[k] is not None)
            out[k] = round(num / den, 1) if den else None
        return out

    a = mid(res["alone"])
    out = {"workload": W.WORKLOADS[wid]["name"], "gemm_mkn": [M, K, N],
           "gemm_ms": {k: [round(t, 4) for t in v] for k, v in res.items()},
           "beside_h2d_pct": round(100 * (mid(res["beside_h2d"]) / a - 1), 2),
           "beside_d2h_pct": round(100 * (mid(res["beside_d2h"]) / a - 1), 2),
           "statistic": "mean of the runs left after dropping the fastest and the slowest"}
    if clock.error:
        out["telemetry_error"] = clock.error
    else:
        out["telemetry"] = {k: telemetry(k) for k in res}
        out["telemetry_note"] = ("amdsmi GPU metrics sampled every 10 ms during each phase: graphics clock (MHz, "
                                 "mean over the XCDs), socket power (W), memory clock (MHz)")
    return out


def gating_leg(torch, P, W, wid, ratios, steps, base_steps, staging, n_buckets=8, direct=False):
    """Does waiting only on the chunks each bucket overwrites pay?  With a
    staging ring (or direct D2H) the capture of the later chunks is paced by
    the D2H, so a single wait on every fragment holds the whole update back
    until the last chunk is captured, while per-bucket waits let each bucket
    go as soon as its own chunks are.  Same loop as the overlap leg, for each
    window/D2H ratio: no snapshots, snapshots with one whole-range wait,
    snapshots with per-bucket waits (each run on the same registered
    state)."""
    tensors, plan = W.make_state(wid, device="cuda")
    ck = P.Checkpointer(tensors, [p[2] for p in plan], [p[3] for p in plan], chunk_bytes=W.WORKLOADS[wid]["chunk"],
                        device_staging_bytes=0 if direct else staging, direct=direct)
    shared = (tensors, plan, ck)
    rows = []
    link = link_peak(torch)["d2h"]
    snap = standalone_snapshot(P, ck, link, runs=3, warm=2)  # one R for both modes
    for ratio in ratios:
        res = {}
        for mode in ("whole", "buckets"):
            res[mode] = overlap_leg(torch, P, W, wid, steps, link, (ratio,), base_steps, shared=shared, gating=mode,
                                    n_buckets=n_buckets, snap=snap, direct=direct)
        rows.append({"window_over_d2h": ratio, "R": res["whole"]["R"], "gemm_ms": res["whole"]["gemm_ms"],
                     "update_ms": round(res["whole"]["base_ms"] - res["whole"]["R"] * res["whole"]["gemm_ms"], 2),
                     "base_ms": res["whole"]["base_ms"],
                     "whole_range_ms": res["whole"]["with_snapshot_ms"],
                     "whole_range_overhead_pct": res["whole"]["overhead_pct"],
                     "per_bucket_base_ms": res["buckets"]["base_ms"],
                     "per_bucket_ms": res["buckets"]["with_snapshot_ms"],
                     "per_bucket_overhead_pct": res["buckets"]["overhead_pct"],
                     "per_bucket_saves_ms": round(res["whole"]["with_snapshot_ms"]
                                                  - res["buckets"]["with_snapshot_ms"], 2),
                     "snapshot_ms": res["whole"]["snapshot_ms"]})
        log("gating: ratio %.2f: whole range %+.2f%%, per bucket %+.2f%%" % (
            ratio, rows[-1]["whole_range_overhead_pct"], rows[-1]["per_bucket_overhead_pct"]))
    ck.close()
    del tensors, shared
    torch.cuda.empty_cache()
    return {"workload": W.WORKLOADS[wid]["name"], "payload_bytes": sum(p[1] for p in plan),
            "device_staging": ("none (direct D2H: the gate waits for the copies)" if direct
                               else staging_text(staging, W.WORKLOADS[wid]["chunk"])), "buckets": n_buckets,
            "gemm_mkn": list(W.OVERLAP_GEMM[wid]), "steps": steps, "base_steps": base_steps, "rows": rows}


def staging_text(staging, chunk):
    return "full image" if not staging else "ring of at most %d bytes (%d chunks)" % (staging, staging // chunk)


def loopback_peak(nbytes=4 << 30, piece=256 << 20):
    """One TCP stream over 127.0.0.1 with the library's socket settings: the
    emulated network's own ceiling."""
    import socket
    import threading

    ls = socket.socket(socket.AF_INET, socket.SOCK_STREAM)
    ls.bind(("127.0.0.1", 0))
    ls.listen(1)
    tx = socket.create_connection(ls.getsockname())
    rx, _ = ls.accept()
    for s in (tx, rx):
        s.setsockopt(socket.IPPROTO_TCP, socket.TCP_NODELAY, 1)
        s.setsockopt(socket.SOL_SOCKET, socket.SO_SNDBUF, 16 << 20)
        s.setsockopt(socket.SOL_SOCKET, socket.SO_RCVBUF, 16 << 20)
    src = bytearray(piece)
    dst = memoryview(bytearray(piece))

    def send():
        for _ in range(nbytes // piece):
            tx.sendall(src)

    t = threading.Thread(target=send)
    t0 = time.perf_counter()
    t.start()
    got = 0
    while got < nbytes:
        k = rx.recv_into(dst[:min(piece, nbytes - got)])
        if not k:
            break
        got += k
    t.join()
    dt = time.perf_counter() - t0
    for s in (tx, rx, ls):
        s.close()
    return got / dt / 1e9


def h2h_leg(torch, P, W, wid, steps, n_peers=1, bounce_bytes=0, host_threads=0):
    """H2H replication (paper Sec. V-B): the optimizer-state chunks of each
    snapshot go to n_peers ring peers (k of Sec. V-C) in this process over
    TCP on 127.0.0.1; each peer re-checks every chunk sum on the GPU before it
    commits.  The state is registered class-major so that the optimizer
    classes fill a run of chunks."""
    tensors, plan = W.make_state(wid, device="cuda")
    order = sorted(range(len(plan)), key=lambda i: (plan[i][3], i))
    tensors = [tensors[i] for i in order]
    dtypes, classes = [plan[i][2] for i in order], [plan[i][3] for i in order]
    torch.cuda.synchronize()
    mask = (1 << W.CLS_MASTER) | (1 << W.CLS_ADAM_M) | (1 << W.CLS_ADAM_V)
    log("h2h: loopback peak")
    loop = loopback_peak()
    peers = [P.Peer() for _ in range(n_peers)]
    peer = peers[0]
    # (pageable images behind bounce rings keep the pinned total under the
    # host's limit when several peers hold pinned replicas)
    ck = P.Checkpointer(tensors, dtypes, classes, chunk_bytes=W.WORKLOADS[wid]["chunk"], bounce_bytes=bounce_bytes,
                        host_threads=host_threads)
    for p in peers:
        ck.replicate_to(p.port, mask)
    ids, rbytes = P.ckpt_replica_chunks(ck.ctx)
    rows = []
    for k in range(steps):
        s = ck.snapshot(step=k)
        ck.wait_replicated(s)
        send_ms, ack_ms = P.ckpt_replica_timing(ck.ctx)
        recv_ms, check_ms = peer.timing()
        rows.append((send_ms, ack_ms, recv_ms, check_ms))
        log("h2h: snapshot %d: sent in %.1f ms, acknowledged after %.1f ms (peer check done %.1f ms after the "
            "last byte)" % (k, send_ms, ack_ms, check_ms))
    image_bytes = int(ck.image_bytes)
    ck.close()  # the rank is lost; its peer keeps the replica
    # A replacement rank with the same layout takes the optimizer state back
    # from the peer (Sec. V-C, third recovery stage): fetch over TCP, then
    # host -> device, scatter and the chunk-sum check on the GPU.
    fresh = [torch.empty_like(t) for t in tensors]
    for t in fresh:
        t.view(-1).view(torch.uint8).fill_(0x3C)
    torch.cuda.synchronize()
    rk = P.Checkpointer(fresh, dtypes, classes, chunk_bytes=W.WORKLOADS[wid]["chunk"], bounce_bytes=bounce_bytes,
                        host_threads=host_threads)
    rest = []
    for k in range(3):
        _, _, bad = rk.restore_from_peer(peer.port)
        torch.cuda.synchronize()
        if bad:
            raise RuntimeError("peer restore: chunks %s failed their sums" % bad)
        info = rk.peer_restore_info()
        rest.append((info["fetch_ms"], info["check_ms"]))
        log("h2h: replacement restore %d: last byte after %.1f ms, restored and checked %.1f ms later"
            % (k, info["fetch_ms"], info["check_ms"]))
    for i, c in enumerate(classes):  # every optimizer fragment is back, byte for byte
        if (mask >> c) & 1 and not torch.equal(fresh[i].view(-1).view(torch.uint8),
                                                tensors[i].view(-1).view(torch.uint8)):
            raise RuntimeError("peer restore: fragment %d differs from the lost rank's" % i)
    rk.close()
    for p in peers:
        p.close()
    del tensors, fresh
    torch.cuda.empty_cache()
    import statistics

    med = [statistics.median(r[i] for r in rows[1:] or rows) for i in range(4)]
    f_ms = statistics.median(r[0] for r in rest)
    c_ms = statistics.median(r[1] for r in rest)
    t_ms = statistics.median(r[0] + r[1] for r in rest)
    return {"workload": W.WORKLOADS[wid]["name"], "classes": "master, Adam m, Adam v (params stay local)",
            "peers": n_peers, "host_images": "pageable + bounce" if bounce_bytes else "pinned",
            "image_bytes": image_bytes, "replica_bytes": int(rbytes),
            "replica_chunks": int(len(ids)),
            "snapshots": steps, "send_ms": round(med[0], 1), "ack_ms": round(med[1], 1),
            "peer_recv_ms": round(med[2], 1), "peer_check_after_last_byte_ms": round(med[3], 1),
            "h2h_GBps": round(n_peers * rbytes / med[0] / 1e6, 2),
            "h2h_with_check_GBps": round(n_peers * rbytes / med[1] / 1e6, 2),
            "loopback_peak_GBps": round(loop, 2),
            "statistic": "median over snapshots after the first; rates count the bytes sent to all peers",
            "replacement_restore": {"to_last_byte_ms": round(f_ms, 1), "after_last_byte_ms": round(c_ms, 1),
                                    "total_ms": round(t_ms, 1), "total_GBps": round(rbytes / t_ms / 1e6, 2),
                                    "runs": len(rest), "statistic": "median of the runs"}}


def pmc_run(torch, P, W, wid, bounce):
    """Short run whose dispatches the counter summary reads: a 1 GiB plain
    device copy (calibration), then two snapshots of workload wid, one
    restore and one verify, then one snapshot in direct D2H mode (its sums
    kernel)."""
    a = torch.empty(CALIBRATION_BYTES, dtype=torch.uint8, device="cuda")
    b = torch.empty(CALIBRATION_BYTES, dtype=torch.uint8, device="cuda")
    a.fill_(1)
    b.copy_(a)
    torch.cuda.synchronize()
    del a, b
    tensors, plan = W.make_state(wid, device="cuda")
    ck = P.Checkpointer(tensors, chunk_bytes=W.WORKLOADS[wid]["chunk"], bounce_bytes=bounce)
    for k in range(2):
        s = ck.snapshot(step=k)
        ck.wait_committed(s)
        print("pmc run: snapshot %d committed" % k, flush=True)
    if ck.restore(s) or ck.verify(s):  # one pass of the scatter and of the verify kernel
        raise SystemExit("checksum mismatch in the counter run")
    image_bytes = ck.image_bytes
    ck.close()
    ck = P.Checkpointer(tensors, chunk_bytes=W.WORKLOADS[wid]["chunk"], bounce_bytes=bounce, direct=True)
    s = ck.snapshot(step=2)
    ck.wait_committed(s)
    print("pmc run: direct snapshot committed", flush=True)
    ck.close()
    print("pmc run done: %s, %d payload bytes, %d-byte image" % (W.WORKLOADS[wid]["name"], sum(p[1] for p in plan),
                                                                  image_bytes), flush=True)


def main():
    args = parse()
    if args.pmc_summary:
        d = pmc_summary(args.pmc_summary[0], args.pmc_summary[1], args.command)
        import workloads as W

        wid = args.workload
        plan = W.fragment_plan(wid)
        S = sum(p[1] for p in plan)
        import oracle as O

        _, I, _ = O.layout([p[1] for p in plan], 256, W.WORKLOADS[wid]["chunk"])
        per = (I + (1 << 30) - 1) >> 30
        header = ("# HBM traffic of the pack kernel (tile_kernel<PACK>) on the %s shard\n"
                  "# (%d payload bytes, 1 GiB launches), from two rocprofv3 --pmc runs of\n"
                  "# `python bench.py --pmc-run`: FETCH_SIZE, then WRITE_SIZE (KiB per dispatch), each scaled by\n"
                  "# the same counter on a plain 1 GiB device copy (__amd_rocclr_copyBuffer).  The same run's\n"
                  "# restore (tile_kernel<SCATTER>), verify (tile_kernel<VERIFY>) and direct D2H snapshot\n"
                  "# (sums_run_kernel) passes are summarized too.\n"
                  "# Algorithmic bytes per dispatch (%d per pass, the last one short): pack and scatter\n"
                  "# %d (read + write), verify %d (read), sums %d (read)." % (W.WORKLOADS[wid]["name"], S, per,
                                                                              2 * S // per, I // per, S // per))
        out = args.traffic
        write_summary(out, d, header)
        print(open(out).read())
        return
    if args.counters_summary:
        print(counters_summary(args.counters_summary[0], args.counters_summary[1:], args.command))
        return
    if args.gemm_inflation:
        print(gemm_inflation(args.gemm_inflation, args.command))
        return
    if args.stats_summary:
        print("# rocprofv3 --kernel-trace --memory-copy-trace --stats\n\ncommand: `%s`\n" % args.command)
        print(stats_summary(args.stats_summary, args.command))
        if args.bench_json:
            b = json.loads(open(args.bench_json).read().strip().splitlines()[-1])
            avg, n = timed_pack_average(args.stats_summary, b)
            rl = b["roofline"]
            print("\nPack kernel over the bench's timed steps (%d dispatches, taken from the kernel trace in order):"
                  % n)
            print("- rocprofv3 average duration: %.4f ms" % avg)
            print("- bench.py HIP events on the pack stream, same run: %.4f ms (achieved %.1f GB/s, frac %.4f)"
                  % (rl["avg_launch_ms"], rl["achieved"], rl["frac"]))
            print("- algorithmic bytes per launch %d -> %.1f GB/s from the rocprofv3 average"
                  % (rl["algorithmic_bytes_per_launch"], rl["algorithmic_bytes_per_launch"] / avg / 1e6))
            rates, med = timed_d2h_from_trace(args.stats_summary, b)
            c = b["components"]
            print("\nD2H of the bench's timed snapshots (image bytes / first group copy start to last group copy end, "
                  "from the memory-copy trace):")
            print("- per snapshot: %s GB/s; median %.2f GB/s = %.1f%% of the link measured in the run (%.2f GB/s)"
                  % (", ".join("%.2f" % x for x in rates), med, 100 * med / c["d2h_link_peak_GBps"],
                     c["d2h_link_peak_GBps"]))
            print("- bench.py's own figure from the engines' completion timestamps, same run: %s"
                  % ("%.2f GB/s" % c["d2h_GBps"] if c["d2h_GBps"] else "not available (the copy tracer owns the "
                     "completion signals)"))
        return
    if args.gpus != 1:
        print("bench.py measures one GPU: each rank packs and offloads its own shard, with no step across GPUs, "
              "so more GPUs would only repeat the one-GPU figure (--gpus %d requested)" % args.gpus, file=sys.stderr)
        sys.exit(2)
    import torch

    import paper_2607_01646_amd as P
    import workloads as W

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    P.lib()  # fails loudly when libckpt.so is missing
    if args.pmc_run:
        wid = args.workload
        pmc_run(torch, P, W, wid, args.bounce_bytes if args.bounce_bytes >= 0 else (DEFAULT_BOUNCE if wid == 4 else 0))
        return
    ratios = [float(r) for r in args.overlap_ratios.split(",") if r]
    wid = args.workload
    bounce = args.bounce_bytes if args.bounce_bytes >= 0 else (DEFAULT_BOUNCE if wid == 4 else 0)
    owid = args.overlap_workload or wid
    if args.h2h_only:
        print(json.dumps({"h2h": h2h_leg(torch, P, W, args.h2h_workload, args.h2h_steps, args.h2h_peers,
                                         max(args.bounce_bytes, 0), args.host_threads)}), flush=True)
        return
    if args.gemm_pmc_run:
        gemm_pmc_run(torch, P, W)
        return
    if args.gemm_beside_only:
        print(json.dumps({"gemm_beside": gemm_beside_leg(torch, P, W)}), flush=True)
        return
    if args.gating_only:
        g = gating_leg(torch, P, W, args.gating_workload, [float(r) for r in args.gating_ratios.split(",") if r],
                       args.gating_steps, args.gating_base_steps, args.gating_staging_bytes, direct=args.gating_direct)
        print(json.dumps({"gating": g}), flush=True)
        return
    if args.overlap_only:
        log("link peak")
        link = link_peak(torch)
        ob = bounce if owid == wid else max(args.bounce_bytes, 0)
        ov = overlap_leg(torch, P, W, owid, args.overlap_steps, link["d2h"], ratios, args.overlap_base_steps, ob,
                         args.host_threads, args.grid_blocks, args.staging_bytes, args.group_bytes,
                         gating=args.overlap_gating, launch=args.pack_launch_bytes, engines=args.d2h_engines,
                         fixed_R=args.overlap_R, direct=args.overlap_mode == "direct")
        print(json.dumps({"overlap": ov, "d2h_link_peak_GBps": round(link["d2h"], 2)}), flush=True)
        return
    wl = W.WORKLOADS[wid]
    gating = None
    if not args.no_gating:  # first: its host memory is freed again before the shard's images are made
        log("gating leg")
        gating = gating_leg(torch, P, W, args.gating_workload, [float(r) for r in args.gating_ratios.split(",") if r],
                            args.gating_steps, args.gating_base_steps, args.gating_staging_bytes)
    log("link peak")
    link = link_peak(torch)
    log("pack ceiling: one contiguous %d-byte fragment" % args.ceiling_bytes)
    ceiling = pack_ceiling(torch, P, args.ceiling_bytes, wl["chunk"], args.pack_launch_bytes)
    log("generating workload", wl["name"])
    tensors, plan = W.make_state(wid, device="cuda")
    torch.cuda.synchronize()
    S = sum(p[1] for p in plan)
    n = len(tensors)
    cpu = None
    if not args.no_cpu:  # before the host images take their share of host memory
        log("cpu baseline")
        cpu = cpu_baseline(tensors, wl["chunk"], args.cpu_sample_bytes)
    log("registering %d fragments (%d payload bytes; host images %s)" % (
        n, S, "pageable behind %d-byte bounce rings" % bounce if bounce else "pinned"))
    # Pageable images: 256 MiB DMA groups, packed four to a 1 GiB launch.  The
    # host copy of each landed group (bounce slot -> image) overlaps the DMA of
    # the next one, so the commit waits for a quarter of a gigabyte after the
    # last copy instead of a whole one; the pack keeps its 1 GiB launches.
    group_bytes, launch_bytes = args.group_bytes, args.pack_launch_bytes
    if bounce and not (args.staging_bytes or args.direct or group_bytes or launch_bytes):
        group_bytes, launch_bytes = 256 << 20, 1 << 30
    ck = P.Checkpointer(tensors, [p[2] for p in plan], [p[3] for p in plan], chunk_bytes=wl["chunk"],
                        bounce_bytes=bounce, host_threads=args.host_threads,
                        image_file=args.image_file or None, device_staging_bytes=args.staging_bytes,
                        group_bytes=group_bytes, pack_launch_bytes=launch_bytes,
                        d2h_engines=args.d2h_engines, direct=args.direct)
    P.ckpt_set_timing(ck.ctx, True)
    opt = Optimizer(torch, tensors)
    bks = buckets_of(plan, 8)
    compute = torch.cuda.current_stream()
    prev = [None]

    def step(k):
        # Optimizer step k-1: each bucket waits (on the compute stream) only
        # for the previous snapshot's capture of the chunks it overwrites.
        for lo, hi in bks:
            if prev[0] is not None:
                ck.wait_captured(prev[0], lo, hi)
            opt.update(lo, hi)
        # Snapshot k, triggered on the compute stream right after the update,
        # with the host link to itself (as in training); once it has
        # committed, the previous committed snapshot is verified (H2D) and
        # snapshot k restored.
        snap = ck.snapshot(step=k, meta=b"step=%d" % k)
        ck.wait_committed(snap)
        bad = ck.verify(prev[0] if prev[0] is not None else snap)
        bad += ck.restore(snap)  # the tensors already hold these bytes: every chunk must check
        if bad:
            raise RuntimeError("checksum mismatch in chunks %s" % bad)
        prev[0] = snap

    log("warmup")
    for k in range(args.warmup):
        step(k)
    torch.cuda.synchronize()
    timings = {"snapshot": [], "restore": [], "verify": []}
    t0 = time.perf_counter()
    for k in range(args.steps):
        step(args.warmup + k)
        timings["snapshot"].append(P.ckpt_last_timing(ck.ctx, P.CKPT_OP_SNAPSHOT))
        timings["restore"].append(P.ckpt_last_timing(ck.ctx, P.CKPT_OP_RESTORE))
        timings["verify"].append(P.ckpt_last_timing(ck.ctx, P.CKPT_OP_VERIFY))
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    ms_per_step = dt * 1e3 / args.steps
    log("timed %d steps: %.1f ms/step" % (args.steps, ms_per_step))

    def agg(kind, key):
        return sum(t[key] for t in timings[kind])

    sn = timings["snapshot"][0]
    K = args.steps
    # trigger to commit; the engines' timestamps are unavailable while a copy
    # tracer owns the completion signals (the trace summary then gives D2H)
    traced = any(t["total_ms"] <= 0 for t in timings["snapshot"])
    snap_ms = None if traced else agg("snapshot", "total_ms") / K
    pack_ms = agg("snapshot", "kernel_ms")
    launches = sum(t["kernels"] for t in timings["snapshot"])
    KB = sn["kernel_bytes"]  # algorithmic bytes of a snapshot's kernels: 2 S (pack), S (direct D2H: sums)
    pack_gbps = KB * K / pack_ms / 1e6
    span_gbps = KB * K / agg("snapshot", "span_ms") / 1e6
    d2h_ms = agg("snapshot", "copy_ms")
    d2h_gbps = sn["copy_bytes"] * K / d2h_ms / 1e6 if d2h_ms > 0 else None
    restore_gbps = sn["copy_bytes"] * K / agg("restore", "total_ms") / 1e6
    scatter_gbps = 2 * S * K / agg("restore", "kernel_ms") / 1e6
    h2d_gbps = sn["copy_bytes"] * K / agg("restore", "copy_ms") / 1e6
    verify_gbps = sn["copy_bytes"] * K / agg("verify", "total_ms") / 1e6
    verify_kernel_gbps = sn["copy_bytes"] * K / agg("verify", "kernel_ms") / 1e6
    # HBM bytes per pack launch from the committed counter summary, unless
    # the kernel source changed since the counters were taken.
    traffic = None
    summ = read_summary(args.traffic)
    if (not args.direct and summ.get("kernel_source_sha") == kernel_source_sha()
            and "traffic_bytes_per_pack_dispatch" in summ):
        traffic = round(float(summ["traffic_bytes_per_pack_dispatch"]))
    roofline = {"kernel": "sums (tile_kernel<SUMS>, direct D2H)" if args.direct else "pack_checksum (tile_kernel<PACK>)",
                "bound": "hbm", "achieved": round(pack_gbps, 1),
                "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(pack_gbps / HBM_PEAK_GBPS, 4),
                "traffic": traffic, "launches": launches, "avg_launch_ms": round(pack_ms / launches, 4),
                "algorithmic_bytes_per_launch": int(KB * K / launches),
                "ceiling": "the same kernel over one contiguous 16-byte-aligned %d-byte fragment, right after an "
                           "in-place update of it: %.1f GB/s" % (ceiling["bytes"], ceiling["after_update_GBps"]),
                "frac_of_ceiling": round(pack_gbps / ceiling["after_update_GBps"], 4),
                "a3_span_GBps": round(span_gbps, 1), "a3_span_frac": round(span_gbps / HBM_PEAK_GBPS, 4)}

    # Pack-only passes over the shard (outside the timed steps): snapshots
    # whose offload is cut before their first copy, so the kernels run with
    # the host link idle; each right after the optimizer update, and each
    # after a host synchronisation with the GPU idle.  Such a snapshot is
    # aborted and never committed.
    def pack_only(update, reps=3):
        ms, cnt = 0.0, 0
        for k in range(reps):
            if update:
                for lo, hi in bks:
                    opt.update(lo, hi)
            else:
                torch.cuda.synchronize()
            P.ckpt_debug_interrupt_next(ck.ctx, 0)
            s_cut = ck.snapshot(step=10_000 + k)
            ck.wait_captured(s_cut, 0, n)
            compute.synchronize()
            t = P.ckpt_last_timing(ck.ctx, P.CKPT_OP_PACK)
            ms += t["kernel_ms"]
        return KB * reps / ms / 1e6

    pack_after_update_gbps = pack_only(True)
    pack_idle_gbps = pack_only(False)
    # The pack stream's span without the per-launch timing events (which
    # lengthen the gaps between launches): snapshots like the timed steps'
    # (update, then snapshot), timed around the first launch and after the
    # chunk-sum reduce only.
    P.ckpt_set_timing(ck.ctx, 2)
    spans = []
    for k in range(3):
        for lo, hi in bks:
            opt.update(lo, hi)
        s_k = ck.snapshot(step=30_000 + k)
        ck.wait_committed(s_k)
        spans.append(P.ckpt_last_timing(ck.ctx, P.CKPT_OP_SNAPSHOT)["span_ms"])
        prev[0] = s_k
    P.ckpt_set_timing(ck.ctx, True)
    span_plain_gbps = KB * len(spans) / sum(spans) / 1e6
    roofline["a3_span_without_launch_events_GBps"] = round(span_plain_gbps, 1)
    roofline["a3_span_without_launch_events_frac"] = round(span_plain_gbps / HBM_PEAK_GBPS, 4)
    roofline["a3_span_note"] = ("2 x payload over the pack stream's whole span: every pack launch, the release "
                                "kernel, the chunk-sum reduce and the gaps between them; in the timed steps (with an "
                                "event pair around every launch) and in three more such snapshots timed around the "
                                "first launch and the end only")
    overlap = None
    if not args.no_overlap:
        log("overlap leg")
        odirect = args.overlap_mode == "direct"
        shared = state = None
        # The overlap leg keeps the library's group sizes (or the ones given):
        # it shares the timed steps' context only when that has them too.
        same_groups = (group_bytes, launch_bytes) == (args.group_bytes, args.pack_launch_bytes)
        if owid == wid and odirect == args.direct and same_groups:
            shared = (tensors, plan, ck)
        elif owid == wid:  # the same tensors in a context of the overlap's mode; its images replace these
            ck.close()
            state = (tensors, plan)
        overlap = overlap_leg(torch, P, W, owid, args.overlap_steps, link["d2h"], ratios, args.overlap_base_steps,
                              bounce if owid == wid else 0, args.host_threads, args.grid_blocks, args.staging_bytes,
                              args.group_bytes, shared=shared, gating=args.overlap_gating,
                              launch=args.pack_launch_bytes, engines=args.d2h_engines, fixed_R=args.overlap_R,
                              direct=odirect, state=state)
    ck.close()
    if overlap and args.overlap_mode == "direct":
        # The overlap's snapshot kernel (direct D2H: sums only) against the
        # same HBM roofline, from the overlap leg's standalone snapshots.
        ks = sorted(g for g in overlap["snapshot_kernel_GBps"] if g)
        if ks:
            per = -(-int(sn["copy_bytes"]) // (1 << 30))  # 1 GiB launches
            st = None
            if summ.get("kernel_source_sha") == kernel_source_sha() and "traffic_bytes_per_sums_dispatch" in summ:
                st = round(float(summ["traffic_bytes_per_sums_dispatch"]))
            overlap["sums_roofline"] = {"kernel": "sums_run_kernel (direct D2H)", "bound": "hbm",
                                        "achieved": ks[len(ks) // 2], "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                                        "frac": round(ks[len(ks) // 2] / HBM_PEAK_GBPS, 4),
                                        "algorithmic_bytes_per_launch": S // per, "traffic": st}
    if args.image_file and os.path.exists(args.image_file):
        os.unlink(args.image_file)
    del tensors
    torch.cuda.empty_cache()
    try:
        sha = subprocess.run(["git", "rev-parse", "--short", "HEAD"], cwd=ROOT, capture_output=True,
                             text=True).stdout.strip() or None
    except Exception:
        sha = None
    out = {
        "metric": METRIC, "value": round(S / snap_ms / 1e6, 3) if snap_ms else None, "unit": "GB/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 2), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "u64", "data": "synthetic",
        "config": {"workload": "%s shard: %d fragments, %d payload bytes, %d MiB chunks; per step: optimizer update "
                               "(per-bucket gate), snapshot (pack + sums + D2H + commit), verify of the previous "
                               "snapshot, restore" % (wl["name"], n, S, wl["chunk"] >> 20),
                   "value": "snapshot GB/s: payload bytes / trigger-to-commit time of the timed steps' snapshots "
                            "(pack + chunk sums + D2H into host memory + commit)",
                   "payload_bytes": S, "image_bytes": int(sn["copy_bytes"]), "chunk_bytes": wl["chunk"],
                   "host_images": ("image file %s behind %d-byte pinned bounce rings" % (args.image_file, bounce)
                                   if args.image_file else
                                   "pageable, %d-byte pinned bounce rings" % bounce if bounce else "pinned"),
                   "device_staging": ("none (direct D2H)" if args.direct
                                      else staging_text(args.staging_bytes, wl["chunk"])),
                   "groups_per_snapshot": int(sn["copies"]), "pack_launches_per_snapshot": int(sn["kernels"]),
                   "group_bytes": group_bytes or None, "pack_launch_bytes": launch_bytes or None,
                   "parallelism": "one rank, one GPU"},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "components": {"snapshot_ms": round(snap_ms, 2) if snap_ms else None,
                       "cycle_GBps": round(S / ms_per_step / 1e6, 3),
                       "pack_GBps": round(pack_gbps, 1),
                       "pack_ceiling": ceiling,
                       "pack_after_update_GBps": round(pack_after_update_gbps, 1),
                       "pack_after_update_frac": round(pack_after_update_gbps / HBM_PEAK_GBPS, 4),
                       "pack_after_update_frac_of_ceiling": round(pack_after_update_gbps
                                                                  / ceiling["after_update_GBps"], 4),
                       "pack_idle_GBps": round(pack_idle_gbps, 1),
                       "pack_idle_frac": round(pack_idle_gbps / HBM_PEAK_GBPS, 4),
                       "d2h_GBps": d2h_gbps and round(d2h_gbps, 2),
                       "d2h_link_peak_GBps": round(link["d2h"], 2),
                       "d2h_frac_of_link": d2h_gbps and round(d2h_gbps / link["d2h"], 4),
                       "d2h_note": "DMA span of the timed snapshots (alone on the host link)",
                       "h2d_GBps": round(h2d_gbps, 2), "h2d_link_peak_GBps": round(link["h2d"], 2),
                       "restore_GBps": round(restore_gbps, 2), "scatter_verify_GBps": round(scatter_gbps, 1),
                       "verify_GBps": round(verify_gbps, 2), "verify_kernel_GBps": round(verify_kernel_gbps, 1)},
        "overlap": overlap,
        "gating": gating,
        "git": sha,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
