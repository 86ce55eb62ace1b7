"""Text summaries of rocprofv3 CSV output for the kernels of libjarq.

    python3 -m paper_2609_38599_amd.profiling stats RUN_kernel_stats.csv --sweeps K
        per-kernel calls, average, time per sweep and share of libjarq GPU time

    python3 -m paper_2609_38599_amd.profiling traffic --fetch F.csv --write W.csv \
        --copy-fetch CF.csv --copy-write CW.csv --copy-bytes N \
        --kernel split3_kernel --source paper_2609_38599_amd/csrc/sgemm.hip
        HBM bytes per dispatch from the FETCH_SIZE / WRITE_SIZE counters (KiB per
        dispatch), each scaled by the factor that makes the same counter read N
        bytes for a plain device copy of N bytes; prints key = value lines for
        the named kernel (read by bench.py) and a table for every kernel.

Reads CSV written by rocprofv3 --output-format csv; nothing here touches the GPU.
"""

from __future__ import annotations

import argparse
import collections
import csv
import hashlib
import os
import re
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def short_name(name: str) -> str:
    """Readable kernel name: the jarq:: function with its template arguments."""
    m = re.match(r"_ZN4jarq\d+(\w+?)I((?:Li\d+E)+)E", name)
    if m:
        args = re.findall(r"Li(\d+)E", m.group(2))
        return f"{m.group(1)}<{','.join(args)}>"
    m = re.match(r"_ZN4jarq\d+(\w+?)E", name)
    if m:
        return m.group(1)
    m = re.match(r"(?:void )?jarq::(\w+)(<[^>]*>)?", name)
    if m:
        return m.group(1) + (m.group(2) or "")
    return name[:48]


def stats(path: str, sweeps: int) -> str:
    """libjarq kernels only (the rest of the process is input generation)."""
    rows = [r for r in csv.DictReader(open(path)) if "jarq" in r["Name"]]
    gpu_total = sum(float(r["TotalDurationNs"]) for r in rows)
    out = [f"{'kernel':28s} {'calls':>6s} {'avg us':>9s} {'ms/sweep':>9s} {'share':>7s}"]
    for r in sorted(rows, key=lambda r: -float(r["TotalDurationNs"])):
        tot = float(r["TotalDurationNs"])
        out.append(f"{short_name(r['Name']):28s} {int(r['Calls']):6d} "
                   f"{float(r['AverageNs']) / 1e3:9.2f} {tot / 1e6 / sweeps:9.4f} "
                   f"{100 * tot / gpu_total:6.2f}%")
    return "\n".join(out)


def per_kernel_mean(path: str) -> dict:
    acc = collections.defaultdict(list)
    for r in csv.DictReader(open(path)):
        acc[r["Kernel_Name"]].append(float(r["Counter_Value"]))
    return {k: sum(v) / len(v) for k, v in acc.items()}


def copy_factor(path: str, nbytes: int) -> float:
    """True KiB / counter KiB for the copy dispatches (the largest-reading kernel)."""
    means = per_kernel_mean(path)
    name = max((k for k in means if "copy" in k.lower()), key=lambda k: means[k])
    return (nbytes / 1024.0) / means[name]


def traffic(a) -> str:
    ff = copy_factor(a.copy_fetch, a.copy_bytes)
    fw = copy_factor(a.copy_write, a.copy_bytes)
    fetch, write = per_kernel_mean(a.fetch), per_kernel_mean(a.write)
    lines = [f"# FETCH_SIZE scale {ff:.4f}, WRITE_SIZE scale {fw:.4f} (plain copy of {a.copy_bytes} bytes)",
             f"# {'kernel':34s} {'fetch MiB':>10s} {'write MiB':>10s}   per dispatch"]
    target = None
    for k in fetch:
        fb = fetch[k] * ff * 1024
        wb = write.get(k, 0.0) * fw * 1024
        lines.append(f"# {short_name(k):34s} {fb / 2**20:10.2f} {wb / 2**20:10.2f}")
        if a.kernel in k:
            target = (k, fb, wb)
    if target is None:
        raise SystemExit(f"kernel {a.kernel} not in {a.fetch}")
    src = os.path.join(ROOT, a.source)
    digest = hashlib.sha256(open(src, "rb").read()).hexdigest()
    k, fb, wb = target
    kv = [f"kernel = {short_name(k)}",
          f"source = {a.source}",
          f"source_sha256 = {digest}",
          f"fetch_size_kib_per_dispatch = {fetch[k]:.1f}",
          f"write_size_kib_per_dispatch = {write.get(k, 0.0):.1f}",
          f"fetch_scale = {ff:.4f}",
          f"write_scale = {fw:.4f}",
          f"hbm_fetch_bytes_per_launch = {fb:.0f}",
          f"hbm_write_bytes_per_launch = {wb:.0f}",
          f"hbm_bytes_per_launch = {fb + wb:.0f}"]
    return "\n".join(kv + lines)


def main(argv=None):
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    s = sub.add_parser("stats")
    s.add_argument("csv")
    s.add_argument("--sweeps", type=int, required=True,
                   help="sweeps in the profiled run (per-sweep column; one-off kernels show /sweeps too)")
    t = sub.add_parser("traffic")
    for name in ("fetch", "write", "copy_fetch", "copy_write", "kernel", "source"):
        t.add_argument("--" + name.replace("_", "-"), dest=name, required=True)
    t.add_argument("--copy-bytes", dest="copy_bytes", type=int, required=True)
    a = ap.parse_args(argv)
    print(stats(a.csv, a.sweeps) if a.cmd == "stats" else traffic(a))


if __name__ == "__main__":
    main(sys.argv[1:])
