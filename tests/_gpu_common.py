"""Shared helpers of the GPU parity tests (HIP path vs the float64 oracle)."""

from __future__ import annotations

import functools
import sys

import numpy as np
import torch

import paper_2609_38599_amd as jq
from oracle import hosts, jarq
from oracle.replay import forced_refine, replay_code_step
from synth import CONFIGS, make_hessian, make_weights, rtn_quantize

SCALE_RTOL = 1e-4          # scales within 1e-4 relative (parity bar)
SCALE_FLOOR = 1e-3         # ... of max(|s_oracle|, 1e-3 * rms(s_row))
OBJ_RTOL = 1e-5            # final objective within 1e-5 relative
EXEMPT_FRAC = 1e-3         # at most 0.1% of codes within 1e-4 of a rounding boundary


def say(*args):
    print(*args, flush=True)
    sys.stdout.flush()


def to_dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.cuda()


def host_state(cfg, W, H):
    if cfg.host == "gptq":
        return hosts.gptq_host(W, H, cfg.group_size, cfg.bits)
    return rtn_quantize(W, cfg.group_size, cfg.bits)


@functools.lru_cache(maxsize=2)
def layer(cfg_id: int):
    """(cfg, W, H, codes, scales, zeros) as numpy arrays (the canonical inputs)."""
    cfg = CONFIGS[cfg_id]
    say(f"[inputs] building config {cfg_id} ({cfg.name})")
    W = make_weights(cfg)
    H = make_hessian(cfg, device="cuda" if cfg_id else None)
    q, s, z = host_state(cfg, W, H)
    say(f"[inputs] config {cfg_id} ready")
    return cfg, W, H, q, s, z


def random_layer(rows, cols, g, bits, seed, corr=0.5):
    """Small random layer with correlated inputs (for edge-case shapes)."""
    rng = np.random.default_rng(seed)
    n = max(2 * cols, 256)
    X = rng.standard_normal((n, cols))
    for c in range(1, cols):
        X[:, c] = corr * X[:, c - 1] + np.sqrt(1 - corr * corr) * X[:, c]
    H = X.T @ X / n
    H += 0.01 * np.mean(np.diag(H)) * np.eye(cols)
    W = (0.02 * rng.standard_normal((rows, cols))).astype(np.float32)
    H32 = np.ascontiguousarray(H.astype(np.float32))
    q, s, z = rtn_quantize(W, g, bits)
    return W, H32, q, s, z


class GpuLayer:
    """Device copies of one layer plus a prepared workspace."""

    def __init__(self, W, H, q, s, z, g, bits, sweeps=1, tau=-1.0, prepare=True,
                 ridge_accept=False):
        self.rows, self.cols = W.shape
        self.g, self.bits = g, bits
        self.p = jq.make_params(self.rows, self.cols, g, bits, sweeps, tau,
                                ridge_accept=ridge_accept)
        self.W = to_dev(W)
        self.H = to_dev(H)
        self.codes = to_dev(q)
        self.scales = to_dev(s)
        self.zeros = to_dev(z)
        self.ws = jq.alloc_workspace(self.p)
        if prepare:
            jq.prepare(self.p, self.W, self.H, self.ws)

    def state(self):
        torch.cuda.synchronize()
        return self.codes.cpu().numpy(), self.scales.cpu().numpy()

    def scale_step(self):
        jq.scale_step(self.p, self.H, self.codes, self.scales, self.zeros, self.ws)

    def code_step(self, trace=True):
        cand = dec = None
        if trace:
            cand = torch.empty_like(self.codes)
            dec = torch.empty(self.rows, self.cols // self.g, dtype=torch.uint8, device="cuda")
        jq.code_step(self.p, self.W, self.H, self.codes, self.scales, self.zeros, self.ws, cand, dec)
        if trace:
            torch.cuda.synchronize()
            return cand.cpu().numpy(), dec.cpu().numpy()
        return None

    def objective(self):
        out = jq.objective(self.p, self.W, self.H, self.codes, self.scales, self.zeros, self.ws)
        torch.cuda.synchronize()
        return out.cpu().numpy()


def check_scales(s_gpu, s_ref, label=""):
    s_gpu = np.asarray(s_gpu, np.float64)
    s_ref = np.asarray(s_ref, np.float64)
    rms = np.sqrt(np.mean(s_ref * s_ref, axis=1, keepdims=True))
    tol = SCALE_RTOL * np.maximum(np.abs(s_ref), SCALE_FLOOR * rms)
    err = np.abs(s_gpu - s_ref)
    worst = float(np.max(err / np.maximum(tol, 1e-300) * SCALE_RTOL))
    say(f"[scales{label}] worst scaled error {worst:.3e} (bar {SCALE_RTOL:g})")
    assert np.all(err <= tol), f"scales differ: worst {worst:.3e}"


def check_code_step(W, H, R, q0, s, z, g, bits, cand, dec, label=""):
    rep = replay_code_step(W, H, R, q0, s, z, g, bits, cand, dec)
    say(f"[codes{label}] positions {rep.n_codes} mismatch {rep.code_mismatch} "
        f"exempt {rep.code_exempt} near-boundary {rep.near_boundary} | groups {rep.n_groups} "
        f"decision mismatch {rep.decision_mismatch} exempt {rep.decision_exempt} "
        f"skip mismatch {rep.skip_mismatch} worst gap {rep.worst_x_gap:.2e}")
    assert rep.skip_mismatch == 0
    assert rep.code_mismatch == 0, rep
    assert rep.decision_mismatch == 0, rep
    assert rep.code_exempt + rep.decision_exempt <= max(1, EXEMPT_FRAC * rep.n_codes), rep
    return rep


def rel(a, b):
    return abs(a - b) / max(abs(b), 1e-300)


def traced_sweeps(gl, K, rows=None):
    """K sweeps of the step entry points on a GpuLayer, with traces.

    Returns per sweep the proposals and decisions (restricted to `rows` if
    given) and the state (codes, scales) after every sweep, states[0] being
    the start.  The step entry points run the same kernels as jarq_sweeps
    with every row active."""
    sel = slice(None) if rows is None else rows
    cands, decs = [], []
    q, s = gl.state()
    states = [(q[sel].copy(), s[sel].copy())]
    for _ in range(K):
        gl.scale_step()
        cand, dec = gl.code_step()
        cands.append(cand[sel].copy())
        decs.append(dec[sel].copy())
        q, s = gl.state()
        states.append((q[sel].copy(), s[sel].copy()))
    return cands, decs, states


def check_forced(W, H, R, q0, s0, z, g, bits, K, cands, decs, q_gpu, s_gpu, label="",
                 tau=None, stop_at=None, rows_active=None):
    """The oracle's own K iterations, deferring to the GPU only inside the bands
    (oracle.replay.forced_refine), must reach the GPU's codes exactly and each
    row's final objective within OBJ_RTOL; at most EXEMPT_FRAC of the proposal
    positions may be deferred."""
    qf, sf, rep = forced_refine(W, H, q0, s0, z, g, bits, K, cands, decs, tau=tau,
                                stop_at=stop_at, R=R)
    F_gpu = jarq.objective_rows(W, H, q_gpu, s_gpu, z, g)
    F_f = jarq.objective_rows(W, H, qf, sf, z, g)
    row_rel = np.abs(F_gpu - F_f) / np.maximum(np.abs(F_f), 1e-300)
    forced = rep.code_forced + rep.decision_forced + rep.stop_forced
    say(f"[forced{label}] {rep.sweeps} sweeps, positions {rep.n_codes}: deferred codes "
        f"{rep.code_forced} decisions {rep.decision_forced} stops {rep.stop_forced} of {rep.n_stops}; "
        f"mismatches codes {rep.code_mismatch} decisions {rep.decision_mismatch} "
        f"skips {rep.skip_mismatch} stops {rep.stop_mismatch}; codes equal "
        f"{np.array_equal(qf, q_gpu)}; F rel total {rel(F_gpu.sum(), F_f.sum()):.2e} "
        f"worst row {float(np.max(row_rel)):.2e}")
    assert rep.ok, rep
    assert forced <= max(1, EXEMPT_FRAC * rep.n_codes), rep
    assert np.array_equal(qf, q_gpu)
    assert np.all(row_rel <= OBJ_RTOL), float(np.max(row_rel))
    if rows_active is not None:
        assert [int(a.sum()) for a in rep.active][:len(rows_active)] == list(rows_active)
    return rep


__all__ = ["jq", "jarq", "torch", "np", "CONFIGS", "layer", "random_layer", "GpuLayer",
           "check_scales", "check_code_step", "check_forced", "traced_sweeps", "rel", "say",
           "OBJ_RTOL", "to_dev"]
