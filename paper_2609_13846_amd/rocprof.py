"""Collect and summarise rocprofv3 runs of bench.py (kernel timing and HBM traffic).

    python -m paper_2609_13846_amd.rocprof collect --out <dir> [--workload NAME]
    python -m paper_2609_13846_amd.rocprof summarize --dir <dir> --profiles profiles [--workload NAME]

(NAME: a workload of ``synth.WORKLOADS``, the Qwen3-0.6B-shaped layer by default.)

``collect`` runs seven rocprofv3 passes of ``bench.py``, each in its own process with its
own time limit, writing CSV output (no database files):

* ``trace``: ``--kernel-trace --stats`` of a timed bench run;
* ``fetch`` / ``write``: ``--pmc FETCH_SIZE`` and ``--pmc WRITE_SIZE`` of a short run;
* ``copyf`` / ``copyw``: the same counters on a plain 1 GiB device copy, which fixes the
  scale of each counter on this GPU (bytes the copy moves / bytes the counter reports);
* ``mfma``: ``--kernel-trace`` with the SQ and GRBM counters of MFMA and VALU work:
  SQ_VALU_MFMA_BUSY_CYCLES sums the matrix-core cycles of every SIMD (16 per
  ``v_mfma_f32_16x16x32_bf16``, 32 per ``32x32x16``), GRBM_GUI_ACTIVE the GPU cycles of each
  of the 8 XCDs, so the MFMA busy fraction is MFMA_BUSY / (GRBM_GUI_ACTIVE / 8 * 1024 SIMDs)
  and GRBM_GUI_ACTIVE / 8 over the launch's duration is the clock it ran at;
* ``stall``: ``--kernel-trace`` with the SQ counters of where a wave's cycles go, all over
  the wave cycles (SQ_WAVE_CYCLES, same units): issuing an instruction (VALU with the
  MFMAs, LDS and scalar apart), ready with an instruction that its unit does not take yet
  (SQ_WAIT_INST_ANY, and LDS instructions alone), and waiting at ``s_waitcnt`` or a
  barrier (SQ_WAIT_ANY).  The three states cover the wave cycles.

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
MFMA_COUNTERS = ["SQ_VALU_MFMA_BUSY_CYCLES", "SQ_BUSY_CYCLES", "SQ_INSTS_MFMA", "SQ_INSTS_VALU",
                 "SQ_INSTS_LDS", "SQ_LDS_BANK_CONFLICT", "SQ_LDS_IDX_ACTIVE", "SQ_WAVE_CYCLES",
                 "GRBM_GUI_ACTIVE"]
STALL_COUNTERS = ["SQ_WAVE_CYCLES", "SQ_ACTIVE_INST_VALU", "SQ_ACTIVE_INST_LDS", "SQ_ACTIVE_INST_SCA",
                  "SQ_ACTIVE_INST_ANY", "SQ_WAIT_INST_ANY", "SQ_WAIT_INST_LDS", "SQ_WAIT_ANY",
                  "GRBM_GUI_ACTIVE"]
N_XCD = 8
N_SIMD = 1024


def kernel_sha() -> str:
    return hashlib.sha256(open(KERNEL_SRC, "rb").read()).hexdigest()[:16]


DEFAULT_WORKLOAD = "qwen3-0.6b-layer"


def traffic_file(profiles: str, workload: str) -> str:
    """The JSON record of one workload's affinity-kernel counters."""
    return os.path.join(profiles, f"affinity_traffic_{workload}.json")


def _passes(out: str, steps: int, workload: str = DEFAULT_WORKLOAD):
    bench = [sys.executable, os.path.join(ROOT, "bench.py")]
    quiet = ["--no-cpu-baseline", "--no-library-gemm", "--no-full-model"]
    if workload != DEFAULT_WORKLOAD:
        quiet += ["--workload", workload]
    timed = bench + ["--steps", str(steps), "--warmup", "2", *quiet]
    short = bench + ["--steps", "2", "--warmup", "1", *quiet]
    copy = bench + ["--copy-calibration", str(COPY_MIB)]
    return [
        ("trace", ["--kernel-trace", "--stats"], timed, 300),
        ("fetch", ["--pmc", "FETCH_SIZE"], short, 180),
        ("write", ["--pmc", "WRITE_SIZE"], short, 180),
        ("copyf", ["--pmc", "FETCH_SIZE"], copy, 120),
        ("copyw", ["--pmc", "WRITE_SIZE"], copy, 120),
        ("mfma", ["--kernel-trace", "--pmc", *MFMA_COUNTERS], short, 180),
        ("stall", ["--kernel-trace", "--pmc", *STALL_COUNTERS], short, 180),
    ]


def collect(out: str, steps: int, workload: str = DEFAULT_WORKLOAD) -> int:
    out = os.path.abspath(out)
    os.makedirs(out, exist_ok=True)
    env = dict(os.environ, TMPDIR="/tmp")
    for name, opts, cmd, limit in _passes(out, steps, workload):
        full = ["timeout", "-s", "KILL", str(limit), "rocprofv3", *opts, "--output-format", "csv",
                "-d", os.path.join(out, name), "-o", "run", "--", *cmd]
        print(f"[rocprof] pass {name}: {' '.join(full)}", flush=True)
        with open(os.path.join(out, f"{name}.log"), "w") as log:
            rc = subprocess.run(full, cwd="/tmp", env=env, stdout=log, stderr=subprocess.STDOUT).returncode
        if rc != 0:
            print(f"[rocprof] pass {name} failed with {rc}", flush=True)
            return rc
    with open(os.path.join(out, "commands.txt"), "w") as f:
        for name, opts, cmd, limit in _passes(out, steps, workload):
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


def _counters(dirname, kernel_sub):
    """{counter: mean per dispatch} over the dispatches of kernels matching kernel_sub, and
    the mean duration (ns) of those dispatches from the pass's kernel trace."""
    acc = {}
    for row in csv.DictReader(open(_one(os.path.join(dirname, "**", "*counter_collection.csv")))):
        if kernel_sub in row["Kernel_Name"]:
            acc.setdefault(row["Counter_Name"], []).append(float(row["Counter_Value"]))
    durs = [int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
            for r in csv.DictReader(open(_one(os.path.join(dirname, "**", "*kernel_trace.csv"))))
            if kernel_sub in r["Kernel_Name"]]
    return {k: sum(v) / len(v) for k, v in acc.items()}, (sum(durs) / len(durs) if durs else 0.0)


def _timed_region(d: str):
    """(launches, bench average ms, rocprofv3 average us) of the trace pass's timed region:
    the bench's JSON line in the pass's log gives its launch count and HIP-event average,
    which the last that many traced launches of the kernel are compared with."""
    try:
        line = [l for l in open(os.path.join(d, "trace.log")) if l.startswith("{")][-1]
        roof = json.loads(line)["roofline"]
        n, bench_ms = int(roof["launches"]), float(roof["avg_launch_ms"])
        rows = [r for r in csv.DictReader(open(_one(os.path.join(d, "trace", "**", "*kernel_trace.csv"))))
                if "affinity_bf16_kernel" in r["Kernel_Name"]]
    except (OSError, ValueError, KeyError, IndexError, FileNotFoundError):
        return None
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    last = rows[-n:] if 0 < n <= len(rows) else []
    if not last:
        return None
    traced = sum(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]) for r in last) / len(last) / 1e3
    return n, bench_ms, traced


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
    wl_opt = f" --workload {workload}" if workload != DEFAULT_WORKLOAD else ""
    lines += ["```", "", f"Summarised with `python -m paper_2609_13846_amd.rocprof summarize --dir <dir> "
              f"--profiles profiles{wl_opt}` (kernel source sha256 prefix `{kernel_sha()}`).", "",
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
        timed = _timed_region(d)
        if timed:
            n, bench_ms, traced_us = timed
            lines += ["", f"The traced bench run's timed region: {n} launches, average "
                      f"{bench_ms * 1e3:.1f} us by the bench's HIP events on the launch stream, "
                      f"{traced_us:.1f} us by rocprofv3 over the same (last {n}) launches; the "
                      f"average above also counts the warm-up, serial and breakdown passes."]
    lines += ["", "## HBM traffic of the affinity kernel (--pmc FETCH_SIZE, WRITE_SIZE)", "",
              f"Counter scale from a plain {COPY_MIB} MiB device copy: FETCH_SIZE x{f_scale:.3f}, "
              f"WRITE_SIZE x{w_scale:.3f} (copy bytes / counter bytes).", "",
              f"- FETCH_SIZE: {sum(fk) / len(fk):.0f} KiB per launch raw, {fetch_b / 1e9:.3f} GB scaled",
              f"- WRITE_SIZE: {sum(wk) / len(wk):.0f} KiB per launch raw, {write_b / 1e9:.3f} GB scaled",
              f"- total: {(fetch_b + write_b) / 1e9:.3f} GB per launch ({len(fk)} launches sampled)"]
    if aff:
        gbs = (fetch_b + write_b) / (float(aff[0]["AverageNs"]) * 1e-9) / 1e9
        lines += [f"- at the traced average duration: {gbs:.0f} GB/s, {gbs / 8000:.1%} of the 8 TB/s HBM peak"]
    mdir = os.path.join(d, "mfma")
    if os.path.isdir(mdir):
        m, dur_ns = _counters(mdir, "affinity_bf16_kernel")
        cyc = m["GRBM_GUI_ACTIVE"] / N_XCD
        busy = m["SQ_VALU_MFMA_BUSY_CYCLES"] / (cyc * N_SIMD)
        clock = cyc / dur_ns if dur_ns else 0.0
        lines += ["", "## MFMA and VALU work of the affinity kernel (--pmc, one pass)", "",
                  f"Counters: {', '.join(MFMA_COUNTERS)}; means per dispatch.", "",
                  f"- MFMA busy: {busy:.1%} of the SIMD cycles "
                  f"(SQ_VALU_MFMA_BUSY_CYCLES {m['SQ_VALU_MFMA_BUSY_CYCLES']:.4g} / "
                  f"(GRBM_GUI_ACTIVE / {N_XCD} = {cyc:.4g} cycles x {N_SIMD} SIMDs))",
                  f"- clock during the launch: {clock:.2f} GHz (GRBM_GUI_ACTIVE / {N_XCD} over "
                  f"{dur_ns / 1e3:.0f} us)",
                  f"- MFMA instructions: {m['SQ_INSTS_MFMA']:.4g} per launch; VALU instructions "
                  f"{m['SQ_INSTS_VALU']:.4g}; LDS instructions {m['SQ_INSTS_LDS']:.4g}",
                  f"- LDS bank conflicts: {m['SQ_LDS_BANK_CONFLICT'] / max(m['SQ_LDS_IDX_ACTIVE'], 1):.1%} "
                  f"of the LDS active cycles"]
    sdir = os.path.join(d, "stall")
    stall = {}
    if os.path.isdir(sdir):
        m2, _ = _counters(sdir, "affinity_bf16_kernel")
        wc = m2["SQ_WAVE_CYCLES"]
        stall = {k: m2[c] / wc for k, c in (("valu_issue", "SQ_ACTIVE_INST_VALU"),
                                             ("lds_issue", "SQ_ACTIVE_INST_LDS"),
                                             ("scalar_issue", "SQ_ACTIVE_INST_SCA"),
                                             ("any_issue", "SQ_ACTIVE_INST_ANY"),
                                             ("issue_wait", "SQ_WAIT_INST_ANY"),
                                             ("issue_wait_lds", "SQ_WAIT_INST_LDS"),
                                             ("wait_any", "SQ_WAIT_ANY"))}
        lines += ["", "## Where a wave's cycles go (--pmc, one pass)", "",
                  f"Counters: {', '.join(STALL_COUNTERS)}; each as a share of SQ_WAVE_CYCLES "
                  f"({wc:.4g} per launch).", "",
                  f"- issuing VALU instructions (MFMAs included): {stall['valu_issue']:.1%}",
                  f"- issuing LDS instructions: {stall['lds_issue']:.1%}; scalar: {stall['scalar_issue']:.1%}; "
                  f"any: {stall['any_issue']:.1%}",
                  f"- ready but not issued (SQ_WAIT_INST_ANY; an instruction waiting for its unit, "
                  f"e.g. behind the other wave's MFMA): {stall['issue_wait']:.1%} "
                  f"(LDS instructions: {stall['issue_wait_lds']:.1%})",
                  f"- waiting at s_waitcnt or a barrier (SQ_WAIT_ANY): {stall['wait_any']:.1%}",
                  f"- the three states (issuing, ready, waiting) add to "
                  f"{stall['any_issue'] + stall['issue_wait'] + stall['wait_any']:.1%} of the wave cycles"]
    open(os.path.join(profiles, name + ".md"), "w").write("\n".join(lines) + "\n")
    mf = {}
    if os.path.isdir(mdir):
        mf = {"mfma_busy": busy, "clock_ghz": clock, "mfma_insts_per_launch": m["SQ_INSTS_MFMA"]}
    if stall:
        mf["wave_cycles"] = stall
    rec = {"kernel": "affinity_bf16_kernel", "workload": workload, "kernel_sha": kernel_sha(),
           "fetch_bytes_per_launch": fetch_b, "write_bytes_per_launch": write_b,
           "bytes_per_launch": fetch_b + write_b, "fetch_scale": f_scale, "write_scale": w_scale,
           "avg_launch_us": float(aff[0]["AverageNs"]) / 1e3 if aff else None, **mf}
    json.dump(rec, open(traffic_file(profiles, workload), "w"), indent=1)
    print(f"wrote {os.path.join(profiles, name + '.md')} and {os.path.basename(traffic_file(profiles, workload))}")


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    sub = ap.add_subparsers(dest="cmd", required=True)
    c = sub.add_parser("collect")
    c.add_argument("--out", required=True)
    c.add_argument("--steps", type=int, default=5)
    c.add_argument("--workload", default=DEFAULT_WORKLOAD)
    s = sub.add_parser("summarize")
    s.add_argument("--dir", required=True)
    s.add_argument("--profiles", default=os.path.join(ROOT, "profiles"))
    s.add_argument("--workload", default=DEFAULT_WORKLOAD)
    args = ap.parse_args()
    if args.cmd == "collect":
        sys.exit(collect(args.out, args.steps, args.workload))
    summarize(args.dir, args.profiles, args.workload, "")


if __name__ == "__main__":
    main()
