"""Summaries of rocprofv3 runs of the FlashNorm kernels (kept as text under profiles/).

A summary records, for one kernel and workload: the commands that produced it,
the kernel's average duration from ``--kernel-trace --stats`` (over all its dispatches,
and over the last ``--timed-steps`` ones, the bench's timed region), the FETCH_SIZE and
WRITE_SIZE counters per dispatch (KiB) scaled by the factors a plain device copy
of known size yields on the same machine, the matrix-core busy fraction, and a
SHA-256 of the kernel's source file and the shared headers.  bench.py reports the
measured HBM traffic only while that hash still matches the sources.

  python -m paper_2407_09577_amd.profiling --workload smollm2_prefill --kernel prefill_bf16_kernel \
      --trace DIR --fetch DIR --write DIR --mfma DIR --cal-fetch DIR --cal-write DIR --copy-bytes N \
      --command "..." --out profiles/NAME.txt
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import os
import re

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
PROFILES = os.path.join(ROOT, "profiles")


def kernel_source(kernel: str) -> str:
    """The csrc/*.hip file that defines the __global__ function ``kernel`` (a name such as
    ``fn::f32_few_rows_kernel<...>`` or ``f32_few_rows_kernel``)."""
    base = re.split(r"[<(]", kernel)[0].split("::")[-1].split()[-1]
    if not base.endswith("_kernel"):
        raise ValueError(f"not a kernel name: {kernel}")
    pat = re.compile(r"__global__[^;{]*?\b" + re.escape(base) + r"\s*\(", re.S)
    for src in sorted(glob.glob(os.path.join(HERE, "csrc", "*.hip"))):
        if pat.search(open(src).read()):
            return src
    raise ValueError(f"no source defines {base}")


def kernel_sources_sha256(kernel: str) -> str:
    """SHA-256 over the source file that defines ``kernel`` and every shared header and
    generated include, i.e. everything its code is built from."""
    src = kernel_source(kernel)
    h = hashlib.sha256()
    shared = sorted(glob.glob(os.path.join(HERE, "csrc", "*.h")) + glob.glob(os.path.join(HERE, "csrc", "*.inc")))
    for path in [src] + shared:
        h.update(os.path.basename(path).encode())
        h.update(open(path, "rb").read())
    return h.hexdigest()


def _rows(d, name):
    """Rows of rocprofv3's CSV ``name`` under output directory ``d`` (at its top level, or in
    the per-host/per-process subdirectories rocprofv3 may create)."""
    path = os.path.join(d, name)
    if not os.path.exists(path):
        found = sorted(glob.glob(os.path.join(d, "**", "*" + name), recursive=True))
        if not found:
            raise FileNotFoundError(f"no {name} under {d}")
        path = found[0]
    with open(path) as f:
        return list(csv.DictReader(f))


def counter_mean(d, kernel, counter):
    vals = [float(r["Counter_Value"]) for r in _rows(d, "run_counter_collection.csv")
            if kernel in r["Kernel_Name"] and r["Counter_Name"] == counter]
    if not vals:
        raise ValueError(f"no {counter} rows for {kernel} in {d}")
    return sum(vals) / len(vals), len(vals)


def kernel_stats(d, kernel):
    for r in _rows(d, "run_kernel_stats.csv"):
        if kernel in r["Name"]:
            return r["Name"], int(r["Calls"]), float(r["AverageNs"])
    raise ValueError(f"{kernel} not in {d}")


def timed_avg_ns(d, name, last):
    """Mean duration of the last `last` dispatches of kernel `name` (full name) in the
    kernel trace: bench.py ends with timed graph replays of `steps` calls each."""
    durs = [int(r["End_Timestamp"]) - int(r["Start_Timestamp"]) for r in _rows(d, "run_kernel_trace.csv")
            if r["Kernel_Name"] == name]
    if len(durs) < last:
        raise ValueError(f"{name}: {len(durs)} dispatches in the trace, fewer than {last}")
    return sum(durs[-last:]) / last


def summarize(a) -> str:
    name, calls, avg_ns = kernel_stats(a.trace, a.kernel) if a.trace else (a.kernel, 0, float("nan"))
    timed_ns = timed_avg_ns(a.trace, name, a.timed_steps) if a.trace else float("nan")
    fetch_kib, nf = counter_mean(a.fetch, a.kernel, "FETCH_SIZE")
    write_kib, nw = counter_mean(a.write, a.kernel, "WRITE_SIZE")
    cal_fetch, _ = counter_mean(a.cal_fetch, "copyBuffer", "FETCH_SIZE")
    cal_write, _ = counter_mean(a.cal_write, "copyBuffer", "WRITE_SIZE")
    f_fetch = a.copy_bytes / (cal_fetch * 1024)
    f_write = a.copy_bytes / (cal_write * 1024)
    busy, _ = counter_mean(a.mfma, a.kernel, "SQ_VALU_MFMA_BUSY_CYCLES")
    active, _ = counter_mean(a.mfma, a.kernel, "GRBM_GUI_ACTIVE")
    # GRBM_GUI_ACTIVE is summed over the 8 XCDs; MFMA busy cycles over all SIMDs.
    util = busy / (active / a.xcds * a.simds)
    traffic = fetch_kib * 1024 * f_fetch + write_kib * 1024 * f_write
    lines = [
        f"# rocprofv3 summary: {a.kernel} on workload {a.workload}",
        "# commands (run from /tmp with TMPDIR=/tmp; R = repository root):",
        *[f"#   {c}" for c in a.command],
        f"kernel: {name}",
        f"kernel_trace_calls: {calls}",
        f"kernel_avg_duration_us: {avg_ns / 1e3:.3f}  (all {calls} dispatches, warm-up included)",
        f"kernel_timed_avg_duration_us: {timed_ns / 1e3:.3f}  (the last {a.timed_steps} dispatches: "
        f"bench.py's last timed graph replay)",
        f"fetch_size_kib_per_dispatch: {fetch_kib:.1f}  (mean of {nf} dispatches)",
        f"write_size_kib_per_dispatch: {write_kib:.1f}  (mean of {nw} dispatches)",
        f"copy_calibration: {a.copy_bytes} bytes copied; FETCH_SIZE {cal_fetch:.1f} KiB -> factor {f_fetch:.4f}; "
        f"WRITE_SIZE {cal_write:.1f} KiB -> factor {f_write:.4f}",
        f"hbm_fetch_bytes_per_launch: {fetch_kib * 1024 * f_fetch:.0f}",
        f"hbm_write_bytes_per_launch: {write_kib * 1024 * f_write:.0f}",
        f"traffic_bytes_per_launch: {traffic:.0f}",
        f"mfma_busy_fraction: {util:.4f}  (SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE/{a.xcds} x {a.simds} SIMDs))",
        f"kernel_sources_sha256: {kernel_sources_sha256(a.kernel)}",
    ]
    return "\n".join(lines) + "\n"


def read_summary(workload: str):
    """Parsed summary for a workload if present and taken with the current kernel sources."""
    paths = glob.glob(os.path.join(PROFILES, f"*_{workload}.txt"))
    for p in paths:
        kv = {}
        for line in open(p):
            m = re.match(r"^([a-z_0-9]+):\s*(\S+)", line)
            if m:
                kv[m.group(1)] = m.group(2)
        m = re.search(r"^kernel: .*?fn::(\w+_kernel)", open(p).read(), flags=re.M)
        if ("traffic_bytes_per_launch" in kv and m
                and kv.get("kernel_sources_sha256") == kernel_sources_sha256(m.group(1))):
            kv["path"] = os.path.relpath(p, ROOT)
            return kv
    return None


def main():
    p = argparse.ArgumentParser()
    p.add_argument("--workload", required=True)
    p.add_argument("--kernel", required=True)
    for k in ("fetch", "write", "mfma", "cal-fetch", "cal-write"):
        p.add_argument(f"--{k}", required=True)
    p.add_argument("--trace", default=None, help="--kernel-trace --stats output of the same command")
    p.add_argument("--copy-bytes", type=int, required=True)
    p.add_argument("--timed-steps", type=int, default=100, help="bench.py --steps of the traced command")
    p.add_argument("--xcds", type=int, default=8)
    p.add_argument("--simds", type=int, default=1024)
    p.add_argument("--command", action="append", default=[])
    p.add_argument("--out", required=True)
    a = p.parse_args()
    text = summarize(a)
    with open(a.out, "w") as f:
        f.write(text)
    print(text)


if __name__ == "__main__":
    main()
