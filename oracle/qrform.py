"""JARQ in the paper's least-squares form, one row at a time (test oracle).

TEST INFRASTRUCTURE ONLY.

This follows the paper's notation directly where the calibration design is
available: A = [X; nu I] and y_j = A w_j (eq. (3), main target), B_j with
columns A_i (q_i - z_i 1) (eq. (5)), the normal equations eq. (6) with the
ridge rule of App. E.2, the conditional target y^(i,k) of eq. (7), a thin QR
A_i = U_i R_i without column permutation (eq. (9)), v = U_i^T y^(i,k) / s_i, the
bounded back substitution eq. (10), and acceptance on the group residual of
eq. (8) evaluated as written (no reduction).  It never forms H, so agreement
with the Hessian-form oracle pins that reformulation.
"""

from __future__ import annotations

import numpy as np
from scipy.linalg import solve_triangular

FP32_EPS = 2.0 ** -23
RIDGE_LAMBDA = 1e-4
RIDGE_RCOND = 1e-10


def design(X, nu):
    """A = [X; nu I] (eq. (3))."""
    X = np.asarray(X, dtype=np.float64)
    return np.vstack([X, nu * np.eye(X.shape[1])])


def _ridge_solve(Gm, rhs, lam, rcond):
    Gs = 0.5 * (Gm + Gm.T)
    trigger = not np.all(np.isfinite(Gs))
    if not trigger:
        ev = np.linalg.eigvalsh(Gs)
        trigger = (not np.all(np.isfinite(ev))) or ev[0] <= rcond * max(abs(ev[-1]), FP32_EPS)
    if not trigger:
        try:
            L = np.linalg.cholesky(Gs)
        except np.linalg.LinAlgError:
            trigger = True
    if trigger:
        L = np.linalg.cholesky(Gs + lam * np.eye(Gs.shape[0]))
    y = solve_triangular(L, rhs, lower=True)
    return solve_triangular(L.T, y, lower=False), trigger


def refine_row(A, w, q0, s0, z, g, bits, K, lam=RIDGE_LAMBDA, rcond=RIDGE_RCOND):
    """Refine one row (output channel) for K iterations without early stopping.

    Returns (codes, scales, list of (objective after scales, objective after codes)).
    """
    A = np.asarray(A, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    y = A @ w                                   # main target, eq. (3)
    d = A.shape[1]
    G = d // g
    qmax = (1 << bits) - 1
    q = np.asarray(q0).astype(np.float64).copy()
    s = np.asarray(s0, dtype=np.float64).copy()
    z = np.asarray(z, dtype=np.float64)
    blocks = [slice(i * g, (i + 1) * g) for i in range(G)]
    factors = []
    for b in blocks:
        U, R = np.linalg.qr(A[:, b], mode="reduced")   # eq. (9)
        factors.append((U, R))

    def what(q_, s_):
        return np.concatenate([s_[i] * (q_[b] - z[i]) for i, b in enumerate(blocks)])

    def objective(q_, s_):
        r = y - A @ what(q_, s_)
        return float(r @ r)

    hist = []
    for _ in range(K):
        # eqs. (5)-(6): B_j = [A_i (q_i - z_i 1)], normal equations, Cholesky.
        B = np.stack([A[:, b] @ (q[b] - z[i]) for i, b in enumerate(blocks)], axis=1)
        s, _ = _ridge_solve(B.T @ B, B.T @ y, lam, rcond)
        f_scale = objective(q, s)
        for i, b in enumerate(blocks):
            if abs(s[i]) <= FP32_EPS:
                continue
            # eq. (7): subtract the latest contributions of every other group.
            t = y.copy()
            for h, bh in enumerate(blocks):
                if h != i:
                    t -= s[h] * (A[:, bh] @ (q[bh] - z[h]))
            U, R = factors[i]
            v = U.T @ t / s[i]
            cand = np.zeros(g)
            for l in range(g - 1, -1, -1):          # eq. (10), l = d_i..1
                x = z[i] + (v[l] - R[l, l + 1:] @ (cand[l + 1:] - z[i])) / R[l, l]
                cand[l] = np.clip(np.rint(x), 0, qmax)
            # eq. (8): accept only a finite, strictly smaller residual.
            r_new = t - s[i] * (A[:, b] @ (cand - z[i]))
            r_old = t - s[i] * (A[:, b] @ (q[b] - z[i]))
            e_new = float(r_new @ r_new)
            e_old = float(r_old @ r_old)
            if np.isfinite(e_new) and e_new < e_old:
                q[b] = cand
        hist.append((f_scale, objective(q, s)))
    return q.astype(np.uint8), s, hist


__all__ = ["design", "refine_row"]
