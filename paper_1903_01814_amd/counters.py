"""rocprofv3 summaries of the benchmark kernels.

    python -m paper_1903_01814_amd.counters pmc --config c2 --kernel bwd_f32_k
    python -m paper_1903_01814_amd.counters stats --config c2 --csv <kernel_stats.csv> \
        --command "<the rocprofv3 command line>" [--bench-json <bench output>]

`stats` turns a `rocprofv3 --kernel-trace --stats` kernel_stats.csv into
profiles/kernels_<workload>.txt (one row per kernel: calls, average, min,
max duration, share of GPU time).

`pmc` measures the HBM traffic of one kernel:
runs bench.py (eager launches, a few steps) twice under
`rocprofv3 --pmc FETCH_SIZE` and `--pmc WRITE_SIZE`, each time followed by a
plain device-to-device copy of known size (bench.py --calib-copy-mib).  The
copy calibrates the counters: its bytes read and written over its FETCH_SIZE
and WRITE_SIZE readings give one scale factor per counter, applied to the
kernel's per-dispatch average.  The summary goes to
profiles/counters_<workload>.txt, stamped with the hash of the kernel
sources; bench.py reports it as roofline.traffic only while the sources are
unchanged.  rocprofv3 is started as a child process with the Python
interpreter directly after `--`.
"""
from __future__ import annotations

import argparse
import csv
import glob
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

COPY_KERNEL = "__amd_rocclr_copyBuffer"
COPY_MIB = 1024


def run_pmc(counter, cfg, regex, out_dir, steps):
    d = os.path.join(out_dir, counter.lower())
    cmd = ["rocprofv3", "--pmc", counter, "--kernel-include-regex", regex,
           "--output-format", "csv", "-d", d, "-o", "pmc", "--",
           sys.executable, os.path.join(ROOT, "bench.py"), "--config", cfg, "--eager",
           "--steps", str(steps), "--warmup", "1", "--no-cpu-baseline",
           "--calib-copy-mib", str(COPY_MIB)]
    env = dict(os.environ, TMPDIR=os.environ.get("TMPDIR", "/tmp"))
    print("counters: running", " ".join(cmd), flush=True)
    r = subprocess.run(cmd, cwd="/tmp", env=env, timeout=240)
    if r.returncode != 0:
        raise SystemExit("counters: rocprofv3 --pmc %s exited with %d" % (counter, r.returncode))
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit("counters: no counter_collection.csv under " + d)
    return files[0], " ".join(cmd)


def per_dispatch(path, counter):
    """{kernel base name: [per-dispatch values in dispatch order]} of one
    counter (summed over the dimension rows of a dispatch)."""
    acc = {}
    for row in csv.DictReader(open(path)):
        if row.get("Counter_Name") != counter:
            continue
        key = short_name(row["Kernel_Name"]).split("<")[0].split("::")[-1].strip()
        disp = row.get("Dispatch_Id") or row.get("Correlation_Id")
        acc.setdefault(key, {}).setdefault(int(disp), 0.0)
        acc[key][int(disp)] += float(row["Counter_Value"])
    return {k: [v[d] for d in sorted(v)] for k, v in acc.items()}


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
        if args.bench_json:
            lines = [l for l in open(args.bench_json) if l.startswith("{")]
            if lines:
                b = json.loads(lines[-1])
                roof = b.get("roofline", {})
                fo.write("# bench line of the same run: %s %s %s, %.5f ms per step; dominant "
                         "kernel %s at %.2f us per launch (library event timing)\n"
                         % (b["metric"], b["value"], b["unit"], b["ms_per_step"],
                            roof.get("kernel"), 1e3 * roof.get("kernel_ms", 0.0)))
    print(open(dst).read())


def main():
    p = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    sub = p.add_subparsers(dest="cmd", required=True)
    q = sub.add_parser("pmc")
    q.add_argument("--config", required=True, choices=["c2", "c3", "c4", "c5"])
    q.add_argument("--kernel", required=True, help="kernel base name, as bench.py reports it")
    q.add_argument("--out-dir", default=os.path.join(ROOT, "gpurun_out", "pmc"))
    q.add_argument("--steps", type=int, default=3)
    q.add_argument("--dest", default=os.path.join(ROOT, "profiles"))
    q = sub.add_parser("stats")
    q.add_argument("--dest", default=os.path.join(ROOT, "profiles"))
    q.add_argument("--config", required=True, choices=["c2", "c3", "c4", "c5"])
    q.add_argument("--csv", required=True)
    q.add_argument("--command", required=True)
    q.add_argument("--bench-json", default=None)
    args = p.parse_args()
    if args.cmd == "stats":
        stats(args)
        return
    from paper_1903_01814_amd import inputs as gen
    import bench
    workload = gen.CONFIGS[args.config]["name"]
    regex = "%s|%s" % (args.kernel, COPY_KERNEL)
    out = {}
    cmds = []
    for counter in ("FETCH_SIZE", "WRITE_SIZE"):
        path, cmd = run_pmc(counter, args.config, regex, os.path.join(args.out_dir, args.config),
                            args.steps)
        cmds.append(cmd)
        vals = per_dispatch(path, counter)
        if args.kernel not in vals or COPY_KERNEL not in vals:
            raise SystemExit("counters: %s or %s missing from %s (found %s)"
                             % (args.kernel, COPY_KERNEL, path, sorted(vals)))
        # the last `steps` dispatches of the kernel are bench.py's timing pass
        # of the dominant op (the last launches before the calibration copy),
        # so they have that op's shape even where the kernel serves others
        k = vals[args.kernel][-args.steps:]
        c = max(vals[COPY_KERNEL])   # the calibration copy is the largest copy
        out[counter] = (sum(k) / len(k), len(k), c)
    copy_bytes = COPY_MIB * 1024.0 * 1024.0
    f_kib, n_f, f_copy = out["FETCH_SIZE"]
    w_kib, n_w, w_copy = out["WRITE_SIZE"]
    f_scale = copy_bytes / f_copy          # bytes per counted KiB unit
    w_scale = copy_bytes / w_copy
    read_b = f_kib * f_scale
    write_b = w_kib * w_scale
    dst = os.path.join(args.dest, "counters_%s.txt" % workload)
    with open(dst, "w") as fo:
        fo.write("# HBM traffic per launch of %s, workload %s, from rocprofv3 counters\n"
                 % (args.kernel, workload))
        fo.write("# commands (run from /tmp):\n#   %s\n#   %s\n" % (cmds[0], cmds[1]))
        fo.write("# calibration: a %d MiB device-to-device copy (%s) read and wrote %d bytes\n"
                 % (COPY_MIB, COPY_KERNEL, int(copy_bytes)))
        fo.write("kernel: %s\n" % args.kernel)
        fo.write("source_hash: %s\n" % bench.source_hash())
        fo.write("dispatches: %d (FETCH_SIZE), %d (WRITE_SIZE): the last ones of the run, "
                 "from bench.py's timing pass of the dominant op\n" % (n_f, n_w))
        fo.write("fetch_size_raw_per_launch: %.1f\n" % f_kib)
        fo.write("write_size_raw_per_launch: %.1f\n" % w_kib)
        fo.write("copy_fetch_size_raw: %.1f\n" % f_copy)
        fo.write("copy_write_size_raw: %.1f\n" % w_copy)
        fo.write("fetch_scale_bytes_per_unit: %.4f\n" % f_scale)
        fo.write("write_scale_bytes_per_unit: %.4f\n" % w_scale)
        fo.write("hbm_read_bytes_per_launch: %.0f\n" % read_b)
        fo.write("hbm_write_bytes_per_launch: %.0f\n" % write_b)
        fo.write("hbm_bytes_per_launch: %.0f\n" % (read_b + write_b))
    print(open(dst).read())


if __name__ == "__main__":
    main()
