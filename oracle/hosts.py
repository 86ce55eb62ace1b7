"""Host quantizers: round-to-nearest, and GPTQ-style for the wide-MLP layer
(test oracle side).

TEST INFRASTRUCTURE ONLY.  It produces the starting state (S0, Q0, Z) of a
refinement run whose codes come from sequential error compensation rather
than from plain rounding (the paper's GPTQ host, App. A.1; the relation of
that recursion to Babai's algorithm is Remark "Relation to GPTQ", App. G.7).

Recursion (GPTQ, written from its published mathematics): let U be the upper
Cholesky factor of H^{-1} (H^{-1} = U^T U).  Visit the columns k = 0..d-1 in
their natural order (no activation ordering, so groups stay contiguous).  At
the first column of each group, fix the group's asymmetric grid by the
min/max rule on the current, already compensated, weights of that group.
Quantize column k on that grid and push its scaled error
err_k = (w_k - what_k) / U_kk into the later columns: w_m -= err_k U_km for
m > k.  Updates to columns after the current group are deferred and applied
once per group as one matrix product; the result is the same recursion.
"""

from __future__ import annotations

import numpy as np


def _grid(wg, qmax):
    """Asymmetric min/max grid with 0 inside the range: (scale float32, zero)."""
    lo = np.minimum(wg.min(axis=1), 0.0)
    hi = np.maximum(wg.max(axis=1), 0.0)
    s = np.where(hi > lo, (hi - lo) / qmax, 1.0).astype(np.float32).astype(np.float64)
    z = np.clip(np.rint(-lo / s), 0, qmax)
    return s, z


def rtn_host(W, g, bits):
    """Asymmetric group-wise round-to-nearest host (App. A.1; the min/max reading
    with 0 inside each group's range): every group gets the grid of `_grid` on
    its own weights and each weight its nearest code, clipped to [0, 2^b - 1].
    Returns (codes uint8 [rows, cols], scales float32 [rows, G], zeros int32 [rows, G])."""
    W = np.asarray(W, dtype=np.float64)
    rows, d = W.shape
    G = d // g
    qmax = (1 << bits) - 1
    codes = np.zeros((rows, d), dtype=np.uint8)
    scales = np.zeros((rows, G), dtype=np.float32)
    zeros = np.zeros((rows, G), dtype=np.int32)
    for i in range(G):
        wg = W[:, i * g:(i + 1) * g]
        s, z = _grid(wg, qmax)
        codes[:, i * g:(i + 1) * g] = np.clip(np.rint(wg / s[:, None]) + z[:, None], 0, qmax)
        scales[:, i] = s.astype(np.float32)
        zeros[:, i] = z.astype(np.int32)
    return codes, scales, zeros


def gptq_host(W, H, g, bits, return_pre=False):
    """Return (codes uint8 [rows, cols], scales float32 [rows, G], zeros int32 [rows, G]);
    with return_pre also the value each code was rounded from (w_k / s + z, float64
    [rows, cols]) and the value each zero point was rounded from (-lo / s, [rows, G])."""
    W = np.array(W, dtype=np.float64, copy=True)
    H = np.asarray(H, dtype=np.float64)
    rows, d = W.shape
    G = d // g
    qmax = (1 << bits) - 1
    Hinv = np.linalg.inv(H)
    Hinv = 0.5 * (Hinv + Hinv.T)
    U = np.linalg.cholesky(Hinv).T          # Hinv = U^T U, U upper triangular
    codes = np.zeros((rows, d), dtype=np.uint8)
    scales = np.zeros((rows, G), dtype=np.float32)
    zeros = np.zeros((rows, G), dtype=np.int32)
    pre = np.zeros((rows, d))
    zpre = np.zeros((rows, G))
    for i in range(G):
        b0, b1 = i * g, (i + 1) * g
        s, z = _grid(W[:, b0:b1], qmax)
        zpre[:, i] = -np.minimum(W[:, b0:b1].min(axis=1), 0.0) / s
        scales[:, i] = s.astype(np.float32)
        zeros[:, i] = z.astype(np.int32)
        err = np.zeros((rows, g))
        for k in range(b0, b1):
            wk = W[:, k]
            pre[:, k] = wk / s + z
            qk = np.clip(np.rint(wk / s) + z, 0, qmax)
            codes[:, k] = qk.astype(np.uint8)
            e = (wk - s * (qk - z)) / U[k, k]
            W[:, k + 1:b1] -= e[:, None] * U[k, k + 1:b1][None, :]
            err[:, k - b0] = e
        if b1 < d:
            W[:, b1:] -= err @ U[b0:b1, b1:]
    if return_pre:
        return codes, scales, zeros, pre, zpre
    return codes, scales, zeros


__all__ = ["rtn_host", "gptq_host"]
