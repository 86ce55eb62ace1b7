"""Benchmark of the JARQ refinement sweep on one MI355X.

A step is one sweep of the hot path over the whole layer: Gram matrices and
joint scale solve, residual product with the row objectives, and the
Gauss-Seidel Babai code update.  The workload is the 4096 x 4096 attention
projection layer (Student-t weights, AR(1)-correlated calibration inputs with
outlier channels, RTN 3-bit host, g = 128), with every input resident in HBM
before the timed region.  W untimed warm-up sweeps run on a copy of the host
state; then R repetitions (--reps, default 5) of K sweeps from the host state
are timed, each as one call bracketed by device synchronisation, and the
reported value is the median over the repetitions of the time per sweep (the
interquartile range beside it).  K defaults to the layer's own sweep count
(10 for the headline layer); when another K is asked for, the layer's own K is
timed the same way and reported beside it.  Inside the timed calls the library
times the residual product only (the roofline kernel), with HIP events
attached to its dispatch (they take the kernel's own start and end times; no
marker is added to the stream).  The per-stage breakdown comes from a
separate, untimed call of the same K sweeps from the host state with events
around every stage.

The roofline fraction counts the method's own work: 2 rows d^2 FLOP per
residual product, against the dense fp16 matrix-core peak (the product runs
on fp16 matrix cores as W M^T - What M^T: the layer's W M^T is formed once,
and each sweep multiplies the exact codes minus zero points by M held as two
fp16 terms, with the scales applied to each group's partial sum; the two fp16
products executed per sweep are reported separately as the executed rate).

After the sweeps, a set-up leg (not part of a sweep; --no-setup skips it)
times the per-layer set-up on the GPU: the Hessian from the layer's 262,144
calibration tokens (fp32 chunks resident in HBM, then the same tokens in
bf16), its finalisation with the layer's damping, and the RTN host.

Prints one JSON line.  --gpus above 1 is refused: the path runs on one GPU.
--copy-probe runs only a plain device copy of known size (used to calibrate
the HBM byte counters of rocprofv3) and prints nothing else; --lds-probe runs
only the library's LDS calibration kernel (known LDS bytes, for the LDS
counters) and logs the rate it reaches.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "ms per JARQ sweep, 4096x4096 G128 3-bit layer; MFMA% and HBM GB/s of peak"
PEAK_FP16_MFMA_TFLOPS = 2500.0   # dense
PEAK_FP32_MFMA_TFLOPS = 157.3
PEAK_FP64_TFLOPS = 78.6
PEAK_HBM_GBS = 8000.0
# LDS: 256 CUs x 256 bytes per clock x 2.4 GHz (the library's LDS probe reads
# 124 TB/s, above the 78.6 TB/s that 128 bytes per clock would allow)
PEAK_LDS_GBS = 256 * 256 * 2.4
COPY_PROBE_BYTES = 256 << 20
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic_residual_product_4096x4096.txt")
STAGE_COUNTERS_FILE = os.path.join(ROOT, "profiles",
                                   "stage_counters_attn_proj_4096x4096_first_sweep.txt")


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def stage_work(cfg, rows, corr_blocks):
    """Executed FLOP of each stage for one sweep (per row: residual product 2 d^2 as two fp16
    products, Gram (d^2 + d g)/2 MACs on two planes, objective two products over the
    triangle of each group, Babai core 2 d g plus corrections)."""
    d, g = cfg.cols, cfg.group_size
    G = d // g
    return {
        "gram": 2.0 * 2.0 * rows * (d * d + d * g) / 2.0,   # two fp16 planes x (d^2+dg)/2 MACs
        "solve": rows * (G ** 3 / 3.0 + 4 * G * G + 2 * d),
        "residual": 2 * 2.0 * rows * d * d,                 # two fp16 products of What M^T
        "objective": 2 * 2.0 * rows * d * g / 2.0,          # cz R_i^T per group, triangular
        "babai": 2.0 * rows * d * g + 2.0 * 16 * g * g * 2 * corr_blocks,
        "panel": 0.0,                                       # in proportion to the rows that changed
    }


def workload_text(cfg, rows, cols, steps):
    """The synthetic layer in words (weights, calibration recipe, host)."""
    wdist = {"normal": "normal", "student_t5": "Student-t(5)"}[cfg.w_dist]
    xdesc = {"zl": "correlated Gaussian", "ar1": "AR(1)", "silu_gate": "SiLU-gated AR(1)",
             "block_equi": "block-equicorrelated"}[cfg.x_recipe]
    outl = f" with {cfg.n_outliers} outlier channels" if cfg.n_outliers else ""
    return (f"{cfg.name}: W {rows}x{cols} {wdist} std {cfg.w_std}, H from {cfg.n_tokens} "
            f"{xdesc} tokens{outl}, {cfg.host.upper()} {cfg.bits}-bit host, g {cfg.group_size}, "
            f"{steps} sweeps from the host state")


def traffic_from_profile():
    """Per-launch HBM bytes of the residual product kernel from rocprofv3 counters.

    Read from the committed summary; None once the kernel source has changed
    since the counters were taken."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    try:
        kv = {}
        for line in open(TRAFFIC_FILE):
            if "=" in line and not line.lstrip().startswith("#"):
                k, v = line.split("=", 1)
                kv[k.strip()] = v.strip()
        src = os.path.join(ROOT, kv["source"])
        digest = hashlib.sha256(open(src, "rb").read()).hexdigest()
        if digest != kv["source_sha256"]:
            return None
        return float(kv["hbm_bytes_per_launch"])
    except Exception:
        return None


def _host_description():
    """CPU model, sockets, logical CPUs and the BLAS NumPy runs on."""
    model, sockets = None, set()
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name") and model is None:
                model = line.split(":", 1)[1].strip()
            elif line.startswith("physical id"):
                sockets.add(line.split(":", 1)[1].strip())
    except OSError:
        pass
    blas = None
    try:
        from threadpoolctl import threadpool_info
        info = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        if info:
            blas = f"{info[0].get('internal_api')} {info[0].get('version')}"
    except Exception:
        pass
    return {"cpu_model": model, "sockets": len(sockets) or None, "logical_cpus": os.cpu_count(),
            "blas": blas}


def _oracle_sweeps(jarq, cfg, H, R, Ws, qs, ss, zs, sweeps):
    g, bits = cfg.group_size, cfg.bits
    t0 = time.perf_counter()
    for _ in range(sweeps):
        ss, _ = jarq.scale_step(Ws, H, qs, zs, g)
        jarq.objective_rows(Ws, H, qs, ss, zs, g)
        qs = jarq.code_step(Ws, H, R, qs, ss, zs, g, bits)
    return time.perf_counter() - t0


def stage_counters():
    """Per-dispatch HBM and LDS bytes of the sweep's kernels in the first sweep
    of a run, from rocprofv3 counters (the committed summary); a kernel whose
    source has changed since is left out."""
    if not os.path.exists(STAGE_COUNTERS_FILE):
        return {}
    kv = {}
    for line in open(STAGE_COUNTERS_FILE):
        if "=" in line and not line.lstrip().startswith("#"):
            k, v = line.split("=", 1)
            kv[k.strip()] = v.strip()
    out = {}
    for key in kv:
        if not key.endswith(".source"):
            continue
        name = key[:-len(".source")]
        try:
            digest = hashlib.sha256(open(os.path.join(ROOT, kv[key]), "rb").read()).hexdigest()
            if digest != kv[name + ".source_sha256"]:
                continue
            out[name] = {f: float(kv[f"{name}.{f}"]) for f in
                         ("hbm_fetch_bytes", "hbm_write_bytes", "lds_read_bytes", "lds_write_bytes",
                          "lds_bank_conflict_cycles")}
        except (OSError, KeyError, ValueError):
            continue
    return out


def stage_rooflines(cfg, rows, stb, npan):
    """HBM and LDS rates of the Gram, Babai and panel-update kernels in the
    first sweep (full Gram build, every row changes), from the per-launch
    time of that sweep (HIP events) and the counted bytes per dispatch."""
    from paper_2609_38599_amd.binding import STAGE_NAMES
    d, g = cfg.cols, cfg.group_size
    G, pg = d // g, min(512 // g, 16)
    sm = stb["stage_ms"][0]
    launch = {"gram_kernel": sm[STAGE_NAMES.index("gram")],
              "babai_kernel": sm[STAGE_NAMES.index("babai")] / npan,
              "panel_update_kernel": sm[STAGE_NAMES.index("panel")] / max(npan - 1, 1)}
    # the method's own work per launch (FLOP as in the residual product's
    # roofline: fp32-equivalent, against the fp16 peak the kernel runs on)
    flop = {"gram_kernel": float(rows) * (d * d + d * g),
            "babai_kernel": 2.0 * rows * pg * g * g,
            "panel_update_kernel": None}
    counted = stage_counters()
    out = {}
    for k, ms in launch.items():
        e = {"launch_ms": ms, "scope": "first sweep of a run"}
        c = counted.get(k)
        if c is not None and ms > 0:
            hbm = c["hbm_fetch_bytes"] + c["hbm_write_bytes"]
            lds = c["lds_read_bytes"] + c["lds_write_bytes"]
            e.update({"hbm_bytes": hbm, "hbm_gbs": hbm / (ms * 1e-3) / 1e9,
                      "hbm_frac": hbm / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS,
                      "lds_bytes": lds, "lds_gbs": lds / (ms * 1e-3) / 1e9,
                      "lds_frac": lds / (ms * 1e-3) / 1e9 / PEAK_LDS_GBS,
                      "lds_bank_conflict_cycles": c["lds_bank_conflict_cycles"]})
        else:
            e.update({"hbm_bytes": None, "lds_bytes": None})
        if flop[k] is not None and ms > 0:
            e["algorithmic_flop"] = flop[k]
            e["frac_of_fp16_peak"] = flop[k] / (ms * 1e-3) / 1e12 / PEAK_FP16_MFMA_TFLOPS
        out[k] = e
    return out


def cpu_baseline(cfg, W, H, q, s, z, rows, sweeps, st_rows=256):
    """The float64 oracle on the host cores, over a bounded sample of the workload,
    with every BLAS thread, then on one thread over a smaller sample."""
    import numpy  # noqa: F401  (loads the BLAS before it is inspected)
    from oracle import jarq
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threadpool_limits = None
        threads = os.cpu_count() or 1
    rows = min(rows, W.shape[0])
    R = jarq.group_factors(H, cfg.group_size)      # per-layer set-up, not timed
    dt = _oracle_sweeps(jarq, cfg, H, R, W[:rows], q[:rows].copy(), s[:rows].copy(), z[:rows],
                        sweeps)
    ms = dt * 1e3 / sweeps * (W.shape[0] / rows)
    out = {"value": ms, "unit": "ms/sweep", "cores": int(threads), "kind": "oracle",
           "sample": f"{sweeps} sweeps (scale update, objective, code update) from the "
                     f"{cfg.host.upper()} host "
                     f"over rows 0..{rows - 1} of {W.shape[0]}, float64 NumPy, {dt:.1f} s wall"
                     + ("" if rows == W.shape[0] else ", scaled by rows (rows are independent)")}
    out.update(_host_description())
    if threadpool_limits is not None:
        st_rows = min(st_rows, W.shape[0])
        with threadpool_limits(limits=1):
            dt1 = _oracle_sweeps(jarq, cfg, H, R, W[:st_rows], q[:st_rows].copy(),
                                 s[:st_rows].copy(), z[:st_rows], 1)
        out["single_thread"] = {"value": dt1 * 1e3 * (W.shape[0] / st_rows), "unit": "ms/sweep",
                                "sample": f"1 sweep over rows 0..{st_rows - 1}, one BLAS thread, "
                                          f"{dt1:.1f} s wall, scaled by rows"}
    return out


def lds_probe(workgroups=4096, passes=128, reps=5):
    import torch
    import paper_2609_38599_amd as jq
    out = torch.empty(workgroups * 256, dtype=torch.float32, device="cuda")
    for _ in range(2):
        jq.binding.lds_probe(workgroups, passes, out)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    torch.cuda.synchronize()
    ev[0].record()
    for _ in range(reps):
        n, _ = jq.binding.lds_probe(workgroups, passes, out)
    ev[1].record()
    torch.cuda.synchronize()
    ms = ev[0].elapsed_time(ev[1]) / reps
    log(f"[bench] LDS probe: {workgroups} work-groups x {passes} passes, {n} LDS bytes per dispatch "
        f"({workgroups * 32768} written, {workgroups * 32768 * passes} read), {ms:.4f} ms, "
        f"{n / (ms * 1e-3) / 1e12:.2f} TB/s")


def copy_probe():
    import torch
    n = COPY_PROBE_BYTES // 4
    a = torch.rand(n, device="cuda")
    b = torch.empty_like(a)
    for _ in range(5):
        b.copy_(a)
    torch.cuda.synchronize()
    log(f"[bench] copy probe: 5 copies of {COPY_PROBE_BYTES} bytes")


def setup_leg(cfg, jq, H_ref, W_dev):
    """Per-layer set-up on the GPU, timed with events on the current stream:
    the calibration Hessian from the layer's full token set (fp32 chunks of
    8192 tokens resident in HBM), its finalisation with the layer's damping,
    and the RTN host.  Not part of a sweep."""
    import torch
    from synth import calibration_chunks
    d = cfg.cols
    chunks = [xc.to(torch.float32).contiguous()
              for xc in calibration_chunks(cfg, device="cuda", chunk=8192)]
    n = sum(int(x.shape[0]) for x in chunks)
    Hacc = torch.zeros(d, d, dtype=torch.float64, device="cuda")
    jq.binding.hessian_accumulate(chunks[0], Hacc, 1.0 / n)      # warm-up
    Hacc.zero_()
    p = jq.make_params(W_dev.shape[0], d, cfg.group_size, cfg.bits, 1)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    torch.cuda.synchronize()
    ev[0].record()
    for X in chunks:
        jq.binding.hessian_accumulate(X, Hacc, 1.0 / n)
    ev[1].record()
    H = jq.binding.hessian_finalize(Hacc, cfg.damping, 0.0)
    ev[2].record()
    jq.binding.rtn(p, W_dev)
    ev[3].record()
    torch.cuda.synchronize()
    t_h, t_f, t_r = (ev[i].elapsed_time(ev[i + 1]) for i in range(3))
    flops = float(n) * d * (d + 1)                 # the d (d + 1) / 2 distinct entries, 2 n each
    dg = torch.sqrt(torch.diagonal(H_ref).double())
    dev_rel = float(((H.double() - H_ref.double()).abs() / torch.outer(dg, dg)).max())
    # the same tokens held in bf16 (the dtype a model would capture them in)
    chunks = [x.to(torch.bfloat16) for x in chunks]
    Hacc.zero_()
    jq.binding.hessian_accumulate(chunks[0], Hacc, 1.0 / n)      # warm-up
    Hacc.zero_()
    torch.cuda.synchronize()
    ev[0].record()
    for X in chunks:
        jq.binding.hessian_accumulate(X, Hacc, 1.0 / n)
    ev[1].record()
    torch.cuda.synchronize()
    t_b = ev[0].elapsed_time(ev[1])
    Hb = jq.binding.hessian_finalize(Hacc, cfg.damping, 0.0)
    dev_rel_b = float(((Hb.double() - H_ref.double()).abs() / torch.outer(dg, dg)).max())
    del chunks, Hacc, H, Hb
    torch.cuda.empty_cache()
    tflops = flops / (t_h * 1e-3) / 1e12
    return {"tokens": n, "chunk_tokens": 8192, "launches": (n + 8191) // 8192,
            "hessian_ms": t_h, "hessian_tflops": tflops,
            "hessian_frac_of_fp32_mfma_peak": tflops / PEAK_FP32_MFMA_TFLOPS,
            "finalize_ms": t_f, "rtn_ms": t_r,
            "rtn_hbm_gbs": (W_dev.numel() * 5 + 8 * W_dev.numel() // cfg.group_size) / (t_r * 1e-3) / 1e9,
            "max_rel_dev_from_fp64_build": dev_rel,
            "hessian_bf16_ms": t_b, "hessian_bf16_tflops": flops / (t_b * 1e-3) / 1e12,
            "hessian_bf16_frac_of_bf16_mfma_peak": flops / (t_b * 1e-3) / 1e12 / PEAK_FP16_MFMA_TFLOPS,
            "bf16_inputs_max_rel_dev_from_fp64_build": dev_rel_b}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None,
                    help="sweeps per timed run (default: the layer's own sweep count)")
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--reps", type=int, default=5, help="timed runs of --steps sweeps")
    ap.add_argument("--no-own-k", action="store_true",
                    help="do not also time the layer's own sweep count when --steps differs")
    ap.add_argument("--config", type=int, default=1)
    ap.add_argument("--tau", type=float, default=-1.0,
                    help="early-stopping threshold (App. E.2 uses 1e-5); negative = off (default)")
    ap.add_argument("--cpu-rows", type=int, default=4096)
    ap.add_argument("--cpu-sweeps", type=int, default=2)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-probe", action="store_true")
    ap.add_argument("--lds-probe", action="store_true")
    ap.add_argument("--no-setup", action="store_true",
                    help="skip the timed per-layer set-up leg (Hessian from tokens, RTN host)")
    ap.add_argument("--inputs", default=None,
                    help="cache file (.npz) of the synthetic layer: loaded if present, else written")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py runs on one GPU only: the refinement path is single-GPU "
              "(rows would shard across GPUs with no per-sweep exchange; not implemented).",
              file=sys.stderr)
        sys.exit(2)
    if args.copy_probe:
        copy_probe()
        return
    if args.lds_probe:
        lds_probe()
        return

    import torch
    import paper_2609_38599_amd as jq
    from paper_2609_38599_amd.binding import STAGE_NAMES
    if not os.path.exists(jq.LIB_PATH):
        from paper_2609_38599_amd.build import build
        build()
    from synth import CONFIGS, make_hessian, make_weights, rtn_quantize

    cfg = CONFIGS[args.config]
    g, bits = cfg.group_size, cfg.bits
    if args.steps is None:
        args.steps = cfg.sweeps
    if args.inputs and os.path.exists(args.inputs):
        log(f"[bench] loading inputs for {cfg.name} from {args.inputs}")
        with np.load(args.inputs, allow_pickle=False) as f:
            W, H, q, s, z = (f[k] for k in ("W", "H", "q", "s", "z"))
    else:
        log(f"[bench] building inputs for {cfg.name}")
        W = make_weights(cfg)
        H = make_hessian(cfg, device="cuda")
        if cfg.host == "gptq":
            # the layer's GPTQ-style host state, built by the library on the GPU
            ph = jq.make_params(W.shape[0], W.shape[1], g, bits, 1)
            qg, sg, zg = jq.binding.gptq(ph, torch.from_numpy(W).cuda(), torch.from_numpy(H).cuda())
            q, s, z = qg.cpu().numpy(), sg.cpu().numpy(), zg.cpu().numpy()
            del qg, sg, zg
        else:
            q, s, z = rtn_quantize(W, g, bits)
        if args.inputs:
            np.savez(args.inputs, W=W, H=H, q=q, s=s, z=z)
    dev = torch.device("cuda:0")
    Wd, Hd = torch.from_numpy(W).to(dev), torch.from_numpy(H).to(dev)
    qh, sh, zd = torch.from_numpy(q).to(dev), torch.from_numpy(s).to(dev), torch.from_numpy(z).to(dev)
    rows, cols = W.shape

    p = jq.make_params(rows, cols, g, bits, args.steps, args.tau)
    ws = jq.alloc_workspace(p, dev)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    jq.prepare(p, Wd, Hd, ws)
    torch.cuda.synchronize()
    prep_ms = (time.perf_counter() - t0) * 1e3
    log(f"[bench] prepare {prep_ms:.2f} ms")

    if args.warmup > 0:
        pw = jq.make_params(rows, cols, g, bits, args.warmup, args.tau)
        qw, sw = qh.clone(), sh.clone()
        jq.sweeps(pw, Wd, Hd, qw, sw, zd, ws)
        del qw, sw
    res_stage = STAGE_NAMES.index("residual")

    def timed_runs(K, reps):
        """reps runs of K sweeps from the host state, each bracketed by device
        synchronisation; per run (ms per sweep, stats)."""
        pk = jq.make_params(rows, cols, g, bits, K, args.tau)
        out = []
        for _ in range(reps):
            qd, sd = qh.clone(), sh.clone()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            st = jq.sweeps(pk, Wd, Hd, qd, sd, zd, ws, stage_mask=1 << res_stage)
            torch.cuda.synchronize()
            wall_ms = (time.perf_counter() - t0) * 1e3
            # With early stopping a run can end before its budget (every row
            # stopped): the time is per sweep run.
            out.append((wall_ms / max(st["sweeps_run"], 1), st))
            del qd, sd
        return out

    runs = timed_runs(args.steps, args.reps)
    per_sweep = np.array([r[0] for r in runs])
    ms_per_step = float(np.median(per_sweep))
    q25, q75 = (float(v) for v in np.percentile(per_sweep, [25, 75]))
    st = runs[0][1]
    log(f"[bench] {args.reps} runs of {args.steps} sweeps: {per_sweep.round(4).tolist()} ms per sweep")
    n = min(args.steps, len(st["stage_ms"]))
    res_ms = float(np.mean([r[1]["stage_ms"][k][res_stage] for r in runs
                            for k in range(min(r[1]["sweeps_run"], len(r[1]["stage_ms"])))]))
    own_k = None
    if args.steps != cfg.sweeps and not args.no_own_k:
        own = np.array([r[0] for r in timed_runs(cfg.sweeps, args.reps)])
        own_k = {"sweeps": cfg.sweeps, "ms_per_sweep_median": float(np.median(own)),
                 "ms_per_sweep_iqr": [float(v) for v in np.percentile(own, [25, 75])]}
        log(f"[bench] the layer's own {cfg.sweeps} sweeps: {own.round(4).tolist()} ms per sweep")

    # Per-stage breakdown: the same sweeps again, untimed, with every stage's events.
    qb, sb = qh.clone(), sh.clone()
    stb = jq.sweeps(p, Wd, Hd, qb, sb, zd, ws, stage_mask=0)
    torch.cuda.synchronize()
    del qb, sb
    stage_ms = {name: float(np.mean([stb["stage_ms"][k][j] for k in range(n)]))
                for j, name in enumerate(STAGE_NAMES)}
    blocks = float(np.mean(st["correction_blocks"][:n]))
    work = stage_work(cfg, rows, blocks)

    # Roofline of the residual product kernel (resid_kernel, one launch per
    # sweep, timed by events attached to its dispatch inside the timed calls): the
    # single kernel with the largest time per sweep.  achieved = the method's
    # own work, 2 rows d^2 FLOP per launch, over the average launch time,
    # against the dense fp16 matrix-core peak (the dtype the contraction runs
    # in).  The two fp16 products it executes are reported as the executed
    # rate and fraction.
    t_res = res_ms * 1e-3
    algorithmic = 2.0 * rows * cols * cols
    achieved = algorithmic / t_res / 1e12
    executed = work["residual"] / t_res / 1e12
    roofline = {"bound": "mfma", "kernel": "resid_kernel", "achieved": achieved,
                "peak": PEAK_FP16_MFMA_TFLOPS, "unit": "TFLOP/s",
                "frac": achieved / PEAK_FP16_MFMA_TFLOPS, "traffic": traffic_from_profile(),
                "launch_ms": res_ms, "algorithmic_flop_per_launch": algorithmic,
                "executed_fp16_tflops": executed,
                "executed_frac_of_fp16_peak": executed / PEAK_FP16_MFMA_TFLOPS,
                "frac_of_fp32_mfma_peak": achieved / PEAK_FP32_MFMA_TFLOPS}
    out = {
        "metric": METRIC,
        "value": ms_per_step,
        "unit": "ms/sweep",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16-codes x f16x2-split/f32acc",
        "data": "synthetic",
        "config": {"workload": workload_text(cfg, rows, cols, args.steps),
                   "rows": rows, "cols": cols, "group_size": g, "bits": bits,
                   "tau": args.tau if args.tau >= 0 else None},
        "rows_per_s": rows / (ms_per_step * 1e-3),
        "reps": args.reps,
        "ms_per_sweep_runs": per_sweep.tolist(),
        "ms_per_sweep_iqr": [q25, q75],
        "own_sweep_count": own_k,
        "dtype_note": "contractions on fp16 matrix cores: exact codes minus zero points (fp16) "
                      "times fp32 operands split into two fp16 terms (22-bit products), fp32 "
                      "accumulation, group scales applied to each group's partial sum; the "
                      "layer's W M^T formed once with three such products; scale solves in fp64",
        "prep_ms": prep_ms,
        "stage_ms": stage_ms,
        "stage_ms_note": "separate untimed run of the same sweeps with HIP events around every stage",
        "stage_ms_per_sweep": {name: [round(stb["stage_ms"][k][j], 5) for k in range(n)]
                               for j, name in enumerate(STAGE_NAMES)},
        "gram_listed": stb["gram_listed"][:n],
        "accepted_groups": st["accepted_groups"][:n],
        "rows_active": st["rows_active"][:n],
        "sweeps_run": st["sweeps_run"],
        "objective_after_scales": st["objective_after_scales"][:n],
        "roofline": roofline,
        "stage_rates_tflops": {name: (work[name] / (stage_ms[name] * 1e-3) / 1e12
                                      if stage_ms[name] > 0 else None) for name in STAGE_NAMES},
        "stage_rooflines": stage_rooflines(cfg, rows, stb, (cols // g + min(512 // g, 16) - 1)
                                           // min(512 // g, 16)),
        "peaks": {"fp16_mfma_tflops": PEAK_FP16_MFMA_TFLOPS, "hbm_gbs": PEAK_HBM_GBS,
                  "lds_gbs": PEAK_LDS_GBS},
    }
    if not args.no_setup:
        log("[bench] per-layer set-up leg (Hessian from calibration tokens, RTN host)")
        out["setup"] = setup_leg(cfg, jq, Hd, Wd)
    if not args.no_cpu_baseline:
        log("[bench] timing the float64 oracle on the host")
        out["cpu_baseline"] = cpu_baseline(cfg, W, H, q, s, z, args.cpu_rows, args.cpu_sweeps)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
