"""Synthetic linear layers shaped like LLaMA projections.

The paper calibrates on 128 WikiText-2 sequences of 2048 tokens (Appendix A.1)
and refines LLaMA/Qwen projection weights with g = 128 at 3 and 4 bits.  Those
datasets and checkpoints are not available here, so each layer below is a
seeded synthetic stand-in with the same shapes and the structure that matters
to the method: heavy-tailed or Gaussian weights, correlated input channels,
outlier channels, and a damped Hessian H = X^T X / n + 0.01 mean(diag) I.

Every random stream is derived from numpy.random.SeedSequence([0, cfg_id]),
seed 0 following the paper's calibration seed.  The heavy Hessian builds run
in float64 with torch on the requested device (the GPU when one is present),
chunked over tokens; the result is stored as float32, the canonical input that
both the HIP path and the oracle read.
"""

from __future__ import annotations

import dataclasses
import math

import numpy as np

try:  # torch is only needed for the large token-streaming Hessian builds
    import torch
except Exception:  # pragma: no cover - torch is present in this image
    torch = None


@dataclasses.dataclass(frozen=True)
class LayerConfig:
    cfg_id: int
    name: str
    rows: int            # d_out: output channels (rows of W)
    cols: int            # d_in: input channels (order of H)
    group_size: int
    bits: int
    sweeps: int
    w_dist: str          # "normal" or "student_t5"
    w_std: float
    x_recipe: str        # "zl", "ar1", "silu_gate", "block_equi"
    n_tokens: int
    rho: float
    n_outliers: int
    outlier_scale: float
    damping: float
    host: str            # "rtn" or "gptq"

    @property
    def groups(self) -> int:
        return self.cols // self.group_size


CONFIGS = {
    0: LayerConfig(0, "tiny", 64, 256, 64, 3, 5, "normal", 0.02, "zl",
                   512, 0.0, 4, 20.0, 0.01, "rtn"),
    1: LayerConfig(1, "attn_proj_4096x4096", 4096, 4096, 128, 3, 10,
                   "student_t5", 0.02, "ar1", 2048 * 128, 0.6,
                   round(0.01 * 4096), 20.0, 0.01, "rtn"),
    2: LayerConfig(2, "mlp_up_11008x4096", 11008, 4096, 128, 4, 10,
                   "normal", 0.02, "ar1", 2048 * 128, 0.6,
                   round(0.01 * 4096), 20.0, 0.01, "rtn"),
    3: LayerConfig(3, "mlp_down_4096x11008", 4096, 11008, 128, 3, 10,
                   "student_t5", 0.02, "silu_gate", 2048 * 128, 0.6,
                   0, 1.0, 0.01, "rtn"),
    4: LayerConfig(4, "wide_mlp_14336x4096", 14336, 4096, 64, 3, 20,
                   "normal", 0.015, "block_equi", 2048 * 128, 0.8,
                   round(0.005 * 4096), 50.0, 0.01, "gptq"),
}


def _streams(cfg_id: int):
    ss = np.random.SeedSequence([0, cfg_id])
    w_ss, x_ss, o_ss, extra_ss = ss.spawn(4)
    return w_ss, x_ss, o_ss, extra_ss


def _torch_seed(ss: np.random.SeedSequence) -> int:
    return int(ss.generate_state(1, dtype=np.uint64)[0] & ((1 << 63) - 1))


def make_weights(cfg: LayerConfig) -> np.ndarray:
    """W [rows, cols] float32 with the configured distribution and std."""
    w_ss, _, _, _ = _streams(cfg.cfg_id)
    rng = np.random.Generator(np.random.PCG64(w_ss))
    shape = (cfg.rows, cfg.cols)
    if cfg.w_dist == "normal":
        w = rng.standard_normal(shape) * cfg.w_std
    elif cfg.w_dist == "student_t5":
        # Student-t with 5 degrees of freedom has variance 5/3.
        w = rng.standard_t(5, size=shape) * (cfg.w_std / math.sqrt(5.0 / 3.0))
    else:
        raise ValueError(cfg.w_dist)
    return np.ascontiguousarray(w.astype(np.float32))


def _outlier_channels(cfg: LayerConfig) -> np.ndarray:
    _, _, o_ss, _ = _streams(cfg.cfg_id)
    rng = np.random.Generator(np.random.PCG64(o_ss))
    if cfg.n_outliers == 0:
        return np.zeros(0, dtype=np.int64)
    return np.sort(rng.choice(cfg.cols, size=cfg.n_outliers, replace=False))


def _ar1_block_matrix(rho: float, n: int, first: bool, dtype, device):
    """Lower-triangular M with x_blk = eps_blk @ M^T + carry * rho^(1..n).

    AR(1) across channels with unit stationary variance:
    x_0 = eps_0, x_c = rho x_{c-1} + sqrt(1 - rho^2) eps_c.
    """
    t = torch.arange(n, device=device, dtype=dtype)
    diff = t[:, None] - t[None, :]
    m = torch.where(diff >= 0, rho ** diff.clamp(min=0), torch.zeros((), dtype=dtype, device=device))
    m = m * math.sqrt(1.0 - rho * rho)
    if first:
        m[:, 0] = rho ** t
    return m


def _ar1(eps, rho: float, block: int = 256):
    """Exact AR(1) recurrence across the columns of eps, blocked over channels."""
    n_tok, d = eps.shape
    out = torch.empty_like(eps)
    carry = None
    for b0 in range(0, d, block):
        b1 = min(d, b0 + block)
        nb = b1 - b0
        m = _ar1_block_matrix(rho, nb, b0 == 0, eps.dtype, eps.device)
        x = eps[:, b0:b1] @ m.T
        if carry is not None:
            powers = rho ** torch.arange(1, nb + 1, device=eps.device, dtype=eps.dtype)
            x = x + carry[:, None] * powers[None, :]
        out[:, b0:b1] = x
        carry = x[:, -1]
    return out


def _token_chunks(cfg: LayerConfig, n_tokens: int, device: str, chunk: int):
    """Yield float64 activation chunks X_c [chunk, cols] for the recipe."""
    _, x_ss, _, _ = _streams(cfg.cfg_id)
    gen = torch.Generator(device=device)
    gen.manual_seed(_torch_seed(x_ss))
    d = cfg.cols
    for t0 in range(0, n_tokens, chunk):
        nt = min(chunk, n_tokens - t0)
        if cfg.x_recipe == "ar1":
            eps = torch.randn(nt, d, generator=gen, device=device, dtype=torch.float64)
            yield _ar1(eps, cfg.rho)
        elif cfg.x_recipe == "silu_gate":
            a = _ar1(torch.randn(nt, d, generator=gen, device=device, dtype=torch.float64), cfg.rho)
            b = _ar1(torch.randn(nt, d, generator=gen, device=device, dtype=torch.float64), cfg.rho)
            yield torch.nn.functional.silu(a) * b
        elif cfg.x_recipe == "block_equi":
            nblk = (d + 63) // 64
            f = torch.randn(nt, nblk, generator=gen, device=device, dtype=torch.float64)
            e = torch.randn(nt, d, generator=gen, device=device, dtype=torch.float64)
            fb = f.repeat_interleave(64, dim=1)[:, :d]
            yield math.sqrt(cfg.rho) * fb + math.sqrt(1.0 - cfg.rho) * e
        else:
            raise ValueError(cfg.x_recipe)


def _tiny_x(cfg: LayerConfig) -> np.ndarray:
    """Activations of the tiny 64 x 256 layer: X = Z L (Z standard normal, L unit lower-triangular)."""
    _, x_ss, _, _ = _streams(cfg.cfg_id)
    rng = np.random.Generator(np.random.PCG64(x_ss))
    z = rng.standard_normal((cfg.n_tokens, cfg.cols))
    low = np.tril(rng.standard_normal((cfg.cols, cfg.cols)) * 0.1, k=-1)
    low += np.eye(cfg.cols)
    x = z @ low
    x[:, _outlier_channels(cfg)] *= cfg.outlier_scale
    return x


def calibration_chunks(cfg: LayerConfig, device: str | None = None,
                       n_tokens: int | None = None, chunk: int = 8192):
    """Yield the calibration activations X_c [<= chunk, cols] (float64, on
    ``device``) whose Gram matrix make_hessian forms: the recipe's tokens with
    the outlier channels scaled.  sum_c X_c^T X_c / n plus the damping is H."""
    if cfg.x_recipe == "zl":
        x = _tiny_x(cfg)
        n = x.shape[0] if n_tokens is None else int(n_tokens)
        for t0 in range(0, n, chunk):
            yield x[t0:min(n, t0 + chunk)]
        return
    if torch is None:
        raise RuntimeError("torch is required for the token-streaming activations")
    if device is None:
        device = "cuda" if torch.cuda.is_available() else "cpu"
    n = cfg.n_tokens if n_tokens is None else int(n_tokens)
    scale = torch.ones(cfg.cols, dtype=torch.float64, device=device)
    out = torch.as_tensor(_outlier_channels(cfg), device=device)
    if out.numel():
        scale[out] = cfg.outlier_scale
    for xc in _token_chunks(cfg, n, device, chunk):
        yield xc * scale[None, :]


def propagated_inputs(x: np.ndarray, seed: int, rel: float = 0.1, add: float = 0.02):
    """Stand-in for the inputs a layer receives once the layers before it are
    quantized: x~ = x (1 + rel xi) + add rms(x) eta, xi and eta independent
    standard normal (seeded), rms over the whole chunk.  float32 in, float32 out."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([0, 1000 + seed])))
    x64 = np.asarray(x, np.float64)
    rms = float(np.sqrt(np.mean(x64 * x64)))
    xi = rng.standard_normal(x64.shape)
    eta = rng.standard_normal(x64.shape)
    return (x64 * (1.0 + rel * xi) + add * rms * eta).astype(np.float32)


def make_hessian(cfg: LayerConfig, device: str | None = None,
                 n_tokens: int | None = None, chunk: int = 8192,
                 return_x: bool = False):
    """H [cols, cols] float32 (and, for the tiny 64 x 256 layer, X as float64 if asked).

    H = X^T X / n with outlier channels of X scaled, plus damping
    0.01 * mean(diag(X^T X / n)) * I.  ``n_tokens`` overrides the token count
    (used only to keep CPU-side experiments small).
    """
    if cfg.x_recipe == "zl":
        x = _tiny_x(cfg)
        h = x.T @ x / x.shape[0]
        h += cfg.damping * np.mean(np.diag(h)) * np.eye(cfg.cols)
        h32 = np.ascontiguousarray(h.astype(np.float32))
        if return_x:
            return h32, x, h
        return h32
    if torch is None:
        raise RuntimeError("torch is required for the token-streaming Hessian build")
    if device is None:
        device = "cuda" if torch.cuda.is_available() else "cpu"
    n = cfg.n_tokens if n_tokens is None else int(n_tokens)
    acc = torch.zeros(cfg.cols, cfg.cols, dtype=torch.float64, device=device)
    for xc in _token_chunks(cfg, n, device, chunk):
        acc += xc.T @ xc
    acc /= n
    out = torch.as_tensor(_outlier_channels(cfg), device=device)
    if out.numel():
        scale = torch.ones(cfg.cols, dtype=torch.float64, device=device)
        scale[out] = cfg.outlier_scale
        acc *= scale[:, None] * scale[None, :]
    acc += cfg.damping * torch.diagonal(acc).mean() * torch.eye(cfg.cols, dtype=torch.float64, device=device)
    acc = 0.5 * (acc + acc.T)
    h32 = acc.to(torch.float32).cpu().numpy()
    del acc
    if device.startswith("cuda"):
        torch.cuda.empty_cache()
    return np.ascontiguousarray(h32)


def make_layer(cfg_id: int, device: str | None = None, n_tokens: int | None = None,
               rows: int | None = None):
    """(cfg, W, H) for a configuration; ``rows`` keeps only the leading rows."""
    cfg = CONFIGS[cfg_id]
    w = make_weights(cfg)
    if rows is not None:
        w = np.ascontiguousarray(w[:rows])
    h = make_hessian(cfg, device=device, n_tokens=n_tokens)
    return cfg, w, h
