"""Text summaries of rocprofv3 CSV output for the kernels of libjarq.

    python3 -m paper_2609_38599_amd.profiling stats RUN_kernel_stats.csv --sweeps K
        per-kernel calls, average, time per sweep and share of libjarq GPU time

    python3 -m paper_2609_38599_amd.profiling traffic --fetch F.csv --write W.csv \
        --copy-fetch CF.csv --copy-write CW.csv --copy-bytes N \
        --kernel resid_kernel --source paper_2609_38599_amd/csrc/sgemm.hip
        HBM bytes per dispatch from the FETCH_SIZE / WRITE_SIZE counters (KiB per
        dispatch), each scaled by the factor that makes the same counter read N
        bytes for a plain device copy of N bytes; prints key = value lines for
        the named kernel (read by bench.py) and a table for every kernel.

    python3 -m paper_2609_38599_amd.profiling counters --fetch F.csv --write W.csv \
        --copy-fetch CF.csv --copy-write CW.csv --copy-bytes N \
        --lds L.csv --probe-lds PL.csv --probe-read-bytes R --probe-write-bytes S \
        --kernel gram_kernel=paper_2609_38599_amd/csrc/gram.hip [--kernel ...]
        per named kernel and dispatch: HBM bytes (FETCH_SIZE / WRITE_SIZE scaled
        by the plain copy) and LDS bytes (SQ_INSTS_LDS_LOAD_BANDWIDTH /
        SQ_INSTS_LDS_STORE_BANDWIDTH, 64-byte units, scaled so that the LDS
        probe kernel reads R and writes S bytes per dispatch), with the LDS
        bank-conflict cycles; key = value lines (read by bench.py) keyed by
        the kernel source's sha256.

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


def per_kernel_mean(path: str, counter: str = None) -> dict:
    """Mean counter value per dispatch for each kernel (one counter name, or
    the only one the file holds)."""
    acc = collections.defaultdict(list)
    for r in csv.DictReader(open(path)):
        if counter is not None and r.get("Counter_Name") != counter:
            continue
        acc[r["Kernel_Name"]].append(float(r["Counter_Value"]))
    return {k: sum(v) / len(v) for k, v in acc.items()}


def _find(means: dict, name: str):
    """The kernel whose name, or short name (template arguments demangled),
    contains `name` (the first by sorted name)."""
    keys = sorted(k for k in means if name in k or name in short_name(k))
    return keys[0] if keys else None


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


def counters(a) -> str:
    ff = copy_factor(a.copy_fetch, a.copy_bytes)
    fw = copy_factor(a.copy_write, a.copy_bytes)
    fetch, write = per_kernel_mean(a.fetch), per_kernel_mean(a.write)
    ld = per_kernel_mean(a.lds, "SQ_INSTS_LDS_LOAD_BANDWIDTH")
    st = per_kernel_mean(a.lds, "SQ_INSTS_LDS_STORE_BANDWIDTH")
    bank = per_kernel_mean(a.lds, "SQ_LDS_BANK_CONFLICT")
    active = per_kernel_mean(a.lds, "SQ_LDS_IDX_ACTIVE")
    pld = per_kernel_mean(a.probe_lds, "SQ_INSTS_LDS_LOAD_BANDWIDTH")
    pst = per_kernel_mean(a.probe_lds, "SQ_INSTS_LDS_STORE_BANDWIDTH")
    probe = _find(pld, "lds_probe")
    if probe is None:
        raise SystemExit(f"lds_probe_kernel not in {a.probe_lds}")
    fl = a.probe_read_bytes / (64.0 * pld[probe])
    fs = a.probe_write_bytes / (64.0 * pst[probe])
    lines = [f"# FETCH_SIZE scale {ff:.4f}, WRITE_SIZE scale {fw:.4f} (plain copy of {a.copy_bytes} bytes)",
             f"# LDS load scale {fl:.4f}, store scale {fs:.4f} (probe: {a.probe_read_bytes} bytes "
             f"read, {a.probe_write_bytes} written per dispatch; counters in 64-byte units)"]
    kv = [f"fetch_scale = {ff:.4f}", f"write_scale = {fw:.4f}",
          f"lds_load_scale = {fl:.4f}", f"lds_store_scale = {fs:.4f}"]
    lines.append(f"# {'kernel':30s} {'fetch MiB':>10s} {'write MiB':>10s} {'LDS rd MiB':>11s} "
                 f"{'LDS wr MiB':>11s} {'bank confl':>11s} {'LDS active':>11s}   per dispatch")
    for spec in a.kernel:
        name, src = spec.split("=", 1)
        k = _find(fetch, name)
        kl = _find(ld, name)
        if k is None or kl is None:
            raise SystemExit(f"kernel {name} missing from the counter files")
        fb = fetch[k] * ff * 1024
        wb = write.get(_find(write, name), 0.0) * fw * 1024
        lr = ld[kl] * 64.0 * fl
        lw = st.get(_find(st, name), 0.0) * 64.0 * fs
        digest = hashlib.sha256(open(os.path.join(ROOT, src), "rb").read()).hexdigest()
        kv += [f"{name}.source = {src}", f"{name}.source_sha256 = {digest}",
               f"{name}.hbm_fetch_bytes = {fb:.0f}", f"{name}.hbm_write_bytes = {wb:.0f}",
               f"{name}.lds_read_bytes = {lr:.0f}", f"{name}.lds_write_bytes = {lw:.0f}",
               f"{name}.lds_bank_conflict_cycles = {bank.get(_find(bank, name), 0.0):.0f}",
               f"{name}.lds_idx_active_cycles = {active.get(_find(active, name), 0.0):.0f}"]
        lines.append(f"# {short_name(k):30s} {fb / 2**20:10.2f} {wb / 2**20:10.2f} {lr / 2**20:11.2f} "
                     f"{lw / 2**20:11.2f} {bank.get(_find(bank, name), 0.0):11.0f} "
                     f"{active.get(_find(active, name), 0.0):11.0f}")
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
    c = sub.add_parser("counters")
    for name in ("fetch", "write", "copy_fetch", "copy_write", "lds", "probe_lds"):
        c.add_argument("--" + name.replace("_", "-"), dest=name, required=True)
    c.add_argument("--copy-bytes", dest="copy_bytes", type=int, required=True)
    c.add_argument("--probe-read-bytes", dest="probe_read_bytes", type=float, required=True)
    c.add_argument("--probe-write-bytes", dest="probe_write_bytes", type=float, required=True)
    c.add_argument("--kernel", action="append", required=True,
                   help="name=source: a kernel (substring of its name) and its source file")
    a = ap.parse_args(argv)
    if a.cmd == "stats":
        print(stats(a.csv, a.sweeps))
    elif a.cmd == "traffic":
        print(traffic(a))
    else:
        print(counters(a))


if __name__ == "__main__":
    main(sys.argv[1:])
