"""rocprofv3 summaries of the benchmark kernels.

    python -m paper_1903_01814_amd.counters pmc --config c4 --op bwd --kernel wgrad32_k
    python -m paper_1903_01814_amd.counters stats --config c4 --csv <kernel_stats.csv> \
        --command "<the rocprofv3 command line>" [--bench-live <bench.py output>]

`stats` turns a `rocprofv3 --kernel-trace --stats` kernel_stats.csv into
profiles/kernels_<workload>.txt (one row per kernel instantiation: calls,
average, min, max duration, share of GPU time).

`pmc` measures one kernel while one op of a workload runs alone: bench.py
--counter-op <op> (eager launches, after one warm-up step) under four
rocprofv3 --pmc passes, each a run of its own:
  1. FETCH_SIZE and 2. WRITE_SIZE -- HBM bytes.  The run ends with a plain
     device-to-device copy of known size (bench.py --calib-copy-mib); its
     bytes over its counter readings give one scale factor per counter,
     applied to the kernel's per-dispatch average.
  3. SQ_VALU_MFMA_BUSY_CYCLES, SQ_INSTS_VALU_MFMA_MOPS_BF16,
     SQ_INSTS_VALU_MFMA_MOPS_F32, GRBM_GUI_ACTIVE -- matrix-core busy
     cycles over (active cycles x 1024 SIMDs) is the MFMA utilisation;
     MOPS x 512 is the matrix-core FLOP count.
  4. SQ_INSTS_LDS, SQ_LDS_BANK_CONFLICT, SQ_LDS_IDX_ACTIVE, SQ_INSTS_MFMA,
     GRBM_GUI_ACTIVE -- LDS instructions issued and cycles lost to bank
     conflicts.
rocprofv3 writes one row per counter and dispatch, summed over the
counter's instances; GRBM_GUI_ACTIVE, counted per XCD, is divided by the 8
XCDs to give the dispatch's active cycles.  The summary goes to
profiles/counters_<workload>_<op>_<kernel>.txt with the exact kernel
instantiation and the hash of the kernel sources; bench.py attaches it to
its roofline entry only for the same workload, op, kernel and sources.
rocprofv3 is started as a child process with the Python interpreter
directly after `--`.
"""
from __future__ import annotations

import argparse
import csv
import glob
import os
import subprocess
import sys
import tempfile

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

COPY_KERNEL = "__amd_rocclr_copyBuffer"
COPY_MIB = 1024
SIMDS = 1024
XCDS = 8           # GRBM_GUI_ACTIVE comes summed over the 8 XCDs

PASSES = [
    ("fetch", ["FETCH_SIZE"]),
    ("write", ["WRITE_SIZE"]),
    ("mfma", ["SQ_VALU_MFMA_BUSY_CYCLES", "SQ_INSTS_VALU_MFMA_MOPS_BF16",
              "SQ_INSTS_VALU_MFMA_MOPS_F32", "GRBM_GUI_ACTIVE"]),
    ("lds", ["SQ_INSTS_LDS", "SQ_LDS_BANK_CONFLICT", "SQ_LDS_IDX_ACTIVE", "SQ_INSTS_MFMA",
             "GRBM_GUI_ACTIVE"]),
]


def run_pass(tag, counters, cfg, op, regex, out_dir, steps, reuse=False):
    """One rocprofv3 --pmc pass (or, with reuse, the CSV an earlier run of
    the same command left in out_dir)."""
    d = os.path.join(out_dir, tag)
    cmd = ["rocprofv3", "--pmc"] + counters + [
        "--kernel-include-regex", regex, "--output-format", "csv", "-d", d, "-o", "pmc", "--",
        "python3", os.path.join(ROOT, "bench.py"), "--config", cfg, "--counter-op", op,
        "--steps", str(steps), "--calib-copy-mib", str(COPY_MIB)]
    rc = 0
    if not reuse:
        env = dict(os.environ, TMPDIR=os.environ.get("TMPDIR", "/tmp"))
        print("counters: running", " ".join(cmd), flush=True)
        rc = subprocess.run([sys.executable if c == "python3" else c for c in cmd], cwd="/tmp",
                            env=env, timeout=180).returncode
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if rc != 0 and not files:
        raise SystemExit("counters: rocprofv3 --pmc %s exited with %d" % (tag, rc))
    if not files:
        raise SystemExit("counters: no counter_collection.csv under " + d)
    return files[0], " ".join(cmd)


def per_dispatch(path):
    """{(kernel base name, counter): {dispatch: value}} (rows of one
    dispatch and counter summed) and {dispatch: full instantiation name}."""
    acc, inst = {}, {}
    for row in csv.DictReader(open(path)):
        full = short_name(row["Kernel_Name"])
        base = full.split("<")[0].strip()
        cn = row.get("Counter_Name")
        disp = int(row.get("Dispatch_Id") or row.get("Correlation_Id"))
        inst[disp] = full
        slot = acc.setdefault((base, cn), {})
        slot[disp] = slot.get(disp, 0.0) + float(row["Counter_Value"])
    return acc, inst


def short_name(name):
    """Kernel name without namespaces, argument list and return type, with
    template arguments kept."""
    n = name.replace("void ", "", 1) if name.startswith("void ") else name
    for ns in ("hexk::(anonymous namespace)::", "hexk::"):
        n = n.replace(ns, "")
    depth, cut = 0, len(n)
    for i, ch in enumerate(n):
        if ch == "<":
            depth += 1
        elif ch == ">":
            depth -= 1
        elif ch == "(" and depth == 0 and i > 0:
            cut = i
            break
    return n[:cut]


def stats(args):
    from paper_1903_01814_amd import inputs as gen
    import json
    workload = gen.CONFIGS[args.config]["name"]
    rows = list(csv.DictReader(open(args.csv)))
    total = sum(float(r["TotalDurationNs"]) for r in rows)
    dst = os.path.join(args.dest, "kernels_%s.txt" % workload)
    with open(dst, "w") as fo:
        fo.write("# rocprofv3 kernel statistics, workload %s\n" % workload)
        fo.write("# command (run from /tmp): %s\n" % args.command)
        fo.write("# MI355X (gfx950), durations in microseconds; source_hash %s\n"
                 % __import__("bench").source_hash())
        fo.write("kernel | calls | avg_us | min_us | max_us | share_%\n")
        for r in sorted(rows, key=lambda r: -float(r["TotalDurationNs"])):
            fo.write("%s | %s | %.2f | %.2f | %.2f | %.2f\n" % (
                short_name(r["Name"]), r["Calls"], float(r["AverageNs"]) / 1e3,
                float(r["MinNs"]) / 1e3, float(r["MaxNs"]) / 1e3,
                100.0 * float(r["TotalDurationNs"]) / total))
        # an instantiation launched with several grids (a stack's layers
        # sharing a kernel) is split by grid from the per-dispatch trace
        if args.trace:
            by = {}
            for r in csv.DictReader(open(args.trace)):
                if r.get("Kind") != "KERNEL_DISPATCH":
                    continue
                grid = (int(r["Grid_Size_X"]) * int(r["Grid_Size_Y"]) * int(r["Grid_Size_Z"])
                        // max(1, int(r["Workgroup_Size_X"]) * int(r["Workgroup_Size_Y"])
                               * int(r["Workgroup_Size_Z"])))
                d = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
                by.setdefault(short_name(r["Kernel_Name"]), {}).setdefault(grid, []).append(d)
            split = {k: v for k, v in by.items() if len(v) > 1}
            if split:
                fo.write("# launches by grid (blocks) for instantiations with several grids "
                         "(from the per-dispatch trace)\n")
                fo.write("kernel | blocks | calls | avg_us | min_us | max_us\n")
                for k in sorted(split):
                    for grid, ds in sorted(split[k].items(), key=lambda kv: -sum(kv[1])):
                        fo.write("%s | %d | %d | %.2f | %.2f | %.2f\n" % (
                            k, grid, len(ds), sum(ds) / len(ds), min(ds), max(ds)))
        # the unprofiled bench.py run of the same GPU session (its live
        # timing: the profiler delays the library's own events on short
        # kernels, so the profiled run's bench line is not quoted)
        if args.bench_live:
            lines = [l for l in open(args.bench_live) if l.startswith("{")]
            rec = None
            if lines:
                b = json.loads(lines[-1])
                if b.get("config", {}).get("workload") == workload:
                    rec = b
                else:
                    rec = b.get("others", {}).get(workload)
            if rec is not None:
                roof = rec.get("roofline", {})
                fo.write("# bench.py without the profiler, same session: %s %s, %.5f ms per "
                         "step; dominant kernel %s (op %s) at %.2f us per launch (library "
                         "timing: events attached to the launch), roofline %s frac %s\n"
                         % (rec["value"], rec["unit"], rec["ms_per_step"], roof.get("kernel"),
                            roof.get("op"), 1e3 * roof.get("kernel_ms", 0.0), roof.get("bound"),
                            roof.get("frac")))
    print(open(dst).read())


def pmc(args):
    from paper_1903_01814_amd import inputs as gen
    import bench
    workload = gen.CONFIGS[args.config]["name"]
    regex = "%s|%s" % (args.kernel, COPY_KERNEL)
    cmds, vals, insts = [], {}, set()
    for tag, counters in PASSES:
        path, cmd = run_pass(tag, counters, args.config, args.op, regex,
                             os.path.join(args.out_dir, "%s_%s" % (args.config, args.op)),
                             args.steps, reuse=args.reuse)
        cmds.append(cmd)
        acc, inst = per_dispatch(path)
        for cn in counters:
            k = acc.get((args.kernel, cn))
            if not k:
                raise SystemExit("counters: %s of %s missing from %s" % (cn, args.kernel, path))
            disp = sorted(k)[-args.steps:]                # the op's launches
            insts |= {inst[i] for i in disp}
            d = [k[i] for i in disp]
            vals[cn] = sum(d) / len(d)
            if tag in ("fetch", "write"):
                c = acc.get((COPY_KERNEL, cn))
                if not c:
                    raise SystemExit("counters: calibration copy missing from %s" % path)
                vals["copy_" + cn] = max(c.values())
    copy_bytes = COPY_MIB * 1024.0 * 1024.0
    f_scale = copy_bytes / vals["copy_FETCH_SIZE"]       # bytes per counted unit
    w_scale = copy_bytes / vals["copy_WRITE_SIZE"]
    read_b = vals["FETCH_SIZE"] * f_scale
    write_b = vals["WRITE_SIZE"] * w_scale
    gui = vals["GRBM_GUI_ACTIVE"] / XCDS
    mfma_util = vals["SQ_VALU_MFMA_BUSY_CYCLES"] / (gui * SIMDS) if gui > 0 else 0.0
    mflop = 512.0 * (vals["SQ_INSTS_VALU_MFMA_MOPS_BF16"] + vals["SQ_INSTS_VALU_MFMA_MOPS_F32"])
    lds_idx = vals["SQ_LDS_IDX_ACTIVE"]
    conflict_frac = vals["SQ_LDS_BANK_CONFLICT"] / lds_idx if lds_idx > 0 else 0.0
    dst = os.path.join(args.dest, "counters_%s_%s_%s.txt" % (workload, args.op, args.kernel))
    with open(dst, "w") as fo:
        fo.write("# rocprofv3 counters per launch of %s while op %s of workload %s runs alone\n"
                 % (args.kernel, args.op, workload))
        fo.write("# commands (run from /tmp, one pass each):\n")
        for c in cmds:
            fo.write("#   %s\n" % c)
        fo.write("# calibration: a %d MiB device-to-device copy (%s) reads and writes %d bytes\n"
                 % (COPY_MIB, COPY_KERNEL, int(copy_bytes)))
        fo.write("# one value per counter and dispatch (summed over instances); active cycles "
                 "= GRBM_GUI_ACTIVE / %d XCDs; mfma_util = SQ_VALU_MFMA_BUSY_CYCLES / (active "
                 "cycles x %d SIMDs); lds_bank_conflict_frac = SQ_LDS_BANK_CONFLICT / "
                 "SQ_LDS_IDX_ACTIVE\n" % (XCDS, SIMDS))
        fo.write("workload: %s\n" % workload)
        fo.write("op: %s\n" % args.op)
        fo.write("kernel: %s\n" % args.kernel)
        fo.write("instantiation: %s\n" % " ; ".join(sorted(insts)))
        fo.write("source_hash: %s\n" % bench.source_hash())
        fo.write("launches_averaged: %d (the op's last launches in each pass)\n" % args.steps)
        for cn in sorted(k for k in vals if not k.startswith("copy_")):
            fo.write("raw_%s: %.1f\n" % (cn, vals[cn]))
        fo.write("copy_fetch_size_raw: %.1f\n" % vals["copy_FETCH_SIZE"])
        fo.write("copy_write_size_raw: %.1f\n" % vals["copy_WRITE_SIZE"])
        fo.write("fetch_scale_bytes_per_unit: %.4f\n" % f_scale)
        fo.write("write_scale_bytes_per_unit: %.4f\n" % w_scale)
        fo.write("hbm_read_bytes_per_launch: %.0f\n" % read_b)
        fo.write("hbm_write_bytes_per_launch: %.0f\n" % write_b)
        fo.write("hbm_bytes_per_launch: %.0f\n" % (read_b + write_b))
        fo.write("active_cycles_per_launch: %.0f\n" % gui)
        fo.write("mfma_util: %.4f\n" % mfma_util)
        fo.write("mfma_flop_per_launch: %.0f\n" % mflop)
        fo.write("lds_insts_per_launch: %.0f\n" % vals["SQ_INSTS_LDS"])
        fo.write("lds_bank_conflict_cycles_per_launch: %.0f\n" % vals["SQ_LDS_BANK_CONFLICT"])
        fo.write("lds_bank_conflict_frac: %.4f\n" % conflict_frac)
    print(open(dst).read())


def main():
    p = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    sub = p.add_subparsers(dest="cmd", required=True)
    q = sub.add_parser("pmc")
    q.add_argument("--config", required=True, choices=["c2", "c3", "c4", "c5", "c6"])
    q.add_argument("--op", required=True, help="op of the workload, as bench.py names it")
    q.add_argument("--kernel", required=True, help="kernel base name, as bench.py reports it")
    q.add_argument("--out-dir", default=os.path.join(tempfile.gettempdir(), "hexconv_pmc"),
                   help="where rocprofv3 writes its raw CSVs")
    q.add_argument("--steps", type=int, default=3)
    q.add_argument("--dest", default=os.path.join(ROOT, "profiles"))
    q.add_argument("--reuse", action="store_true",
                   help="summarise the CSVs an earlier run left under --out-dir")
    q = sub.add_parser("stats")
    q.add_argument("--dest", default=os.path.join(ROOT, "profiles"))
    q.add_argument("--config", required=True, choices=["c1", "c2", "c3", "c4", "c5", "c6"])
    q.add_argument("--csv", required=True)
    q.add_argument("--command", required=True)
    q.add_argument("--trace", default=None,
                   help="kernel_trace.csv of the same run (splits instantiations by grid)")
    q.add_argument("--bench-live", default=None,
                   help="JSON line of an unprofiled bench.py run (its live timing is quoted)")
    args = p.parse_args()
    if args.cmd == "stats":
        stats(args)
    else:
        pmc(args)


if __name__ == "__main__":
    main()
