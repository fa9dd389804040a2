"""Collect and summarise rocprofv3 runs of bench.py (kernel timing and HBM traffic).

    python -m paper_2609_13846_amd.rocprof collect --out gpurun_out/prof
    python -m paper_2609_13846_amd.rocprof summarize --dir gpurun_out/prof --profiles profiles

``collect`` runs five rocprofv3 passes of ``bench.py``, each in its own process with its
own time limit, writing CSV output (no database files):

* ``trace``: ``--kernel-trace --stats`` of a timed bench run;
* ``fetch`` / ``write``: ``--pmc FETCH_SIZE`` and ``--pmc WRITE_SIZE`` of a short run;
* ``copyf`` / ``copyw``: the same counters on a plain 1 GiB device copy, which fixes the
  scale of each counter on this GPU (bytes the copy moves / bytes the counter reports).

``summarize`` writes a markdown summary of the kernel trace and the traffic of the
affinity kernel (bytes per launch, counter scales applied) to ``profiles/``, plus the
JSON record ``bench.py`` reads for its roofline ``traffic`` field.  That record carries a
hash of the kernel source, so it is ignored once the kernel changes.
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
KERNEL_SRC = os.path.join(ROOT, "paper_2609_13846_amd", "csrc", "affinity.hip")
COPY_MIB = 1024


def kernel_sha() -> str:
    return hashlib.sha256(open(KERNEL_SRC, "rb").read()).hexdigest()[:16]


def _passes(out: str, steps: int):
    bench = [sys.executable, os.path.join(ROOT, "bench.py")]
    timed = bench + ["--steps", str(steps), "--warmup", "2", "--no-cpu-baseline"]
    short = bench + ["--steps", "2", "--warmup", "1", "--no-cpu-baseline"]
    copy = bench + ["--copy-calibration", str(COPY_MIB)]
    return [
        ("trace", ["--kernel-trace", "--stats"], timed, 300),
        ("fetch", ["--pmc", "FETCH_SIZE"], short, 180),
        ("write", ["--pmc", "WRITE_SIZE"], short, 180),
        ("copyf", ["--pmc", "FETCH_SIZE"], copy, 120),
        ("copyw", ["--pmc", "WRITE_SIZE"], copy, 120),
    ]


def collect(out: str, steps: int) -> int:
    out = os.path.abspath(out)
    os.makedirs(out, exist_ok=True)
    env = dict(os.environ, TMPDIR="/tmp")
    for name, opts, cmd, limit in _passes(out, steps):
        full = ["timeout", "-s", "KILL", str(limit), "rocprofv3", *opts, "--output-format", "csv",
                "-d", os.path.join(out, name), "-o", "run", "--", *cmd]
        print(f"[rocprof] pass {name}: {' '.join(full)}", flush=True)
        with open(os.path.join(out, f"{name}.log"), "w") as log:
            rc = subprocess.run(full, cwd="/tmp", env=env, stdout=log, stderr=subprocess.STDOUT).returncode
        if rc != 0:
            print(f"[rocprof] pass {name} failed with {rc}", flush=True)
            return rc
    with open(os.path.join(out, "commands.txt"), "w") as f:
        for name, opts, cmd, limit in _passes(out, steps):
            shown = ["python3" if c == sys.executable else
                     (os.path.relpath(c, ROOT) if c.startswith(ROOT) else c) for c in cmd]
            f.write(f"{name}: rocprofv3 {' '.join(opts)} --output-format csv -d <dir>/{name} -o run -- "
                    f"{' '.join(shown)}\n")
    return 0


def _one(pattern):
    hits = glob.glob(pattern, recursive=True)
    if not hits:
        raise FileNotFoundError(pattern)
    return hits[0]


def _counter(dirname, kernel_sub):
    """{kernel name: [values]} of the single counter in a --pmc pass."""
    vals = {}
    for row in csv.DictReader(open(_one(os.path.join(dirname, "**", "*counter_collection.csv")))):
        if kernel_sub in row["Kernel_Name"]:
            vals.setdefault(row["Kernel_Name"], []).append(float(row["Counter_Value"]))
    return vals


def summarize(d: str, profiles: str, workload: str, bench_cmd: str) -> None:
    stats = list(csv.DictReader(open(_one(os.path.join(d, "trace", "**", "*kernel_stats.csv")))))
    stats.sort(key=lambda r: -float(r["TotalDurationNs"]))
    aff = [r for r in stats if "affinity_bf16_kernel" in r["Name"]]
    fetch = _counter(os.path.join(d, "fetch"), "affinity_bf16_kernel")
    write = _counter(os.path.join(d, "write"), "affinity_bf16_kernel")
    cf = _counter(os.path.join(d, "copyf"), "copyBuffer")
    cw = _counter(os.path.join(d, "copyw"), "copyBuffer")
    copy_kib = COPY_MIB * 1024.0
    f_scale = copy_kib / (sum(sum(v) for v in cf.values()) / sum(len(v) for v in cf.values()))
    w_scale = copy_kib / (sum(sum(v) for v in cw.values()) / sum(len(v) for v in cw.values()))
    fk = [x for v in fetch.values() for x in v]
    wk = [x for v in write.values() for x in v]
    fetch_b = sum(fk) / len(fk) * 1024 * f_scale
    write_b = sum(wk) / len(wk) * 1024 * w_scale
    os.makedirs(profiles, exist_ok=True)
    name = f"affinity_bf16_{workload}"
    lines = [f"# rocprofv3 summary: affinity kernel, {workload} workload", "",
             "Commands (run from the repository root on one MI355X):", "", "```"]
    lines += [l.rstrip() for l in open(os.path.join(d, "commands.txt"))]
    lines += ["```", "", f"Summarised with `python -m paper_2609_13846_amd.rocprof summarize --dir <dir> "
              f"--profiles profiles` (kernel source sha256 prefix `{kernel_sha()}`).", "",
              "## Kernel trace (--kernel-trace --stats), top kernels", "",
              "| kernel | calls | avg (us) | total (ms) | share |", "|---|---:|---:|---:|---:|"]
    for r in stats[:12]:
        nm = r["Name"]
        nm = nm if len(nm) < 90 else nm[:87] + "..."
        lines.append(f"| `{nm}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                     f"{float(r['TotalDurationNs']) / 1e6:.2f} | {float(r['Percentage']):.1f}% |")
    if aff:
        a = aff[0]
        lines += ["", f"Affinity kernel: {a['Calls']} launches, average {float(a['AverageNs']) / 1e3:.1f} us, "
                  f"min {float(a['MinNs']) / 1e3:.1f} us, max {float(a['MaxNs']) / 1e3:.1f} us."]
    lines += ["", "## HBM traffic of the affinity kernel (--pmc FETCH_SIZE, WRITE_SIZE)", "",
              f"Counter scale from a plain {COPY_MIB} MiB device copy: FETCH_SIZE x{f_scale:.3f}, "
              f"WRITE_SIZE x{w_scale:.3f} (copy bytes / counter bytes).", "",
              f"- FETCH_SIZE: {sum(fk) / len(fk):.0f} KiB per launch raw, {fetch_b / 1e9:.3f} GB scaled",
              f"- WRITE_SIZE: {sum(wk) / len(wk):.0f} KiB per launch raw, {write_b / 1e9:.3f} GB scaled",
              f"- total: {(fetch_b + write_b) / 1e9:.3f} GB per launch ({len(fk)} launches sampled)"]
    open(os.path.join(profiles, name + ".md"), "w").write("\n".join(lines) + "\n")
    rec = {"kernel": "affinity_bf16_kernel", "workload": workload, "kernel_sha": kernel_sha(),
           "fetch_bytes_per_launch": fetch_b, "write_bytes_per_launch": write_b,
           "bytes_per_launch": fetch_b + write_b, "fetch_scale": f_scale, "write_scale": w_scale,
           "avg_launch_us": float(aff[0]["AverageNs"]) / 1e3 if aff else None}
    json.dump(rec, open(os.path.join(profiles, "affinity_traffic.json"), "w"), indent=1)
    print(f"wrote {os.path.join(profiles, name + '.md')} and affinity_traffic.json")


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    sub = ap.add_subparsers(dest="cmd", required=True)
    c = sub.add_parser("collect")
    c.add_argument("--out", required=True)
    c.add_argument("--steps", type=int, default=5)
    s = sub.add_parser("summarize")
    s.add_argument("--dir", required=True)
    s.add_argument("--profiles", default=os.path.join(ROOT, "profiles"))
    s.add_argument("--workload", default="qwen3-0.6b-layer")
    args = ap.parse_args()
    if args.cmd == "collect":
        sys.exit(collect(args.out, args.steps))
    summarize(args.dir, args.profiles, args.workload, "")


if __name__ == "__main__":
    main()
