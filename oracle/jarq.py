"""JARQ per-layer refinement in float64, Hessian form (test oracle).

TEST INFRASTRUCTURE ONLY: used by the tests, the smoke check and the
CPU-baseline leg of the benchmark; never by the product path.

Problem (Sec. 3.1-3.2).  Row j of W (one output channel, the paper's column
w_j) is represented by eq. (1): what_j = D_{s_j}(q_j - z_j), with G groups of g
consecutive weights, one signed scale and one integer zero point per group and
codes in B = {0, ..., 2^b - 1}.  The objective eq. (4) is separable over rows:
F_j = ||y_j - A what_j||^2 with A = [X; nu I], y_j = A w_j.  With H = A^T A this
is F_j = (w_j - what_j)^T H (w_j - what_j); the constant of the QR reduction is
zero for this target (App. E.1), so nothing is dropped.

One iteration k (Sec. 3.3; the missing Algorithm 1 is read from Sec. 3.3 and
App. E.2 as "refit all scales of the row, then visit the groups in order"):

* scale update (eqs. (5)-(6), App. E.2): B_j has columns A_i (q_i - z_i 1);
  the Gram matrix B_j^T B_j has entries c_i^T H_ih c_h and the right-hand side
  B_j^T y_j has entries c_i^T (H w)_i, where c_i = q_i - z_i 1.  Symmetrise,
  add 1e-4 I when the spectrum is nonfinite, the smallest eigenvalue is at
  most 1e-10 max(|lambda_max|, eps_fp32) or Cholesky fails; a second failure
  is a numerical error.
  Optionally (the remark on ridge acceptance, App. G.5) a ridge solution is
  kept only when it does not increase F_j against the previous scales.
* early stopping (App. E.2, eq. (strict_stopping)), optional.
* code update (eqs. (7)-(10)): for i = 1..G, the conditional target
  y^(i,k) subtracts the latest contributions of every other group; with
  A_i = U_i R_i (eq. (9)), v = U_i^T y^(i,k) / s_i, and U_i^T y = R_i^{-T} A_i^T y
  because U_i = A_i R_i^{-1}; A_i^T y^(i,k) = (H w)_i - sum_{h != i} s_h H_ih c_h.
  Back substitution eq. (10) runs l = g..1 with round-half-to-even and a clip
  to B.  The proposal is kept only if the residual of eq. (8) is finite and
  strictly smaller (Sec. 3.3.2, App. E.2); by App. G.4 that residual is
  s_i^2 ||v - R_i (q - z 1)||^2 plus a term that does not depend on q.  Groups
  with |s_i| <= eps_fp32 keep their codes (App. E.2, "Small scales").

R_i is obtained from H_ii = A_i^T A_i = R_i^T R_i as its upper Cholesky factor
(the Babai proposal does not depend on the row signs of R_i).
"""

from __future__ import annotations

import dataclasses

import numpy as np
from scipy.linalg import solve_triangular

FP32_EPS = 2.0 ** -23        # "FP32 machine epsilon", App. E.2
RIDGE_LAMBDA = 1e-4          # lambda of the stabilised scale solve, App. E.2
RIDGE_RCOND = 1e-10          # r_cond of the spectrum test, App. E.2
STOP_TAU = 1e-5              # tau of eq. (strict_stopping), App. E.2

DEC_REJECT, DEC_ACCEPT, DEC_SKIP = 0, 1, 2


class NotSPDError(ValueError):
    """A diagonal block H_ii is not positive definite (eq. (9) needs R_i nonsingular)."""


class ScaleSolveError(ArithmeticError):
    """The Gram matrix of some row failed Cholesky even after the ridge (App. E.2)."""

    def __init__(self, rows):
        super().__init__(f"scale solve failed after ridge for rows {list(rows)[:8]}")
        self.rows = list(rows)


def _f64(a):
    return np.asarray(a, dtype=np.float64)


def code_offsets(codes, zeros, g):
    """c = q - z per group, shape [rows, G, g] (eq. (1))."""
    codes = np.asarray(codes)
    rows, cols = codes.shape
    G = cols // g
    return codes.reshape(rows, G, g).astype(np.float64) - _f64(zeros)[:, :, None]


def dequantize(codes, scales, zeros, g):
    """what = D_s (q - z) as [rows, cols] float64 (eq. (1))."""
    c = code_offsets(codes, zeros, g)
    rows = c.shape[0]
    return (_f64(scales)[:, :, None] * c).reshape(rows, -1)


def objective_rows(W, H, codes, scales, zeros, g):
    """F_j = (w_j - what_j)^T H (w_j - what_j) for every row (eq. (4), Hessian form)."""
    E = _f64(W) - dequantize(codes, scales, zeros, g)
    return np.einsum("jc,jc->j", E @ _f64(H).T, E)


def group_factors(H, g):
    """R_i, upper triangular with R_i^T R_i = H_ii, for every group (eq. (9))."""
    H = _f64(H)
    G = H.shape[0] // g
    R = np.empty((G, g, g))
    for i in range(G):
        blk = slice(i * g, (i + 1) * g)
        Hii = H[blk, blk]
        try:
            L = np.linalg.cholesky(Hii)
        except np.linalg.LinAlgError as exc:
            raise NotSPDError(f"H block {i} is not positive definite") from exc
        if not np.all(np.isfinite(L)):
            raise NotSPDError(f"H block {i} is not finite")
        R[i] = L.T
    return R


def gram_system(W, H, codes, zeros, g):
    """Gram matrices B_j^T B_j [rows, G, G] and right-hand sides B_j^T y_j [rows, G].

    Entry (i, h) of the Gram matrix is c_i^T H_ih c_h and entry i of the
    right-hand side is c_i^T (H w)_i (eq. (5) with H = A^T A, y_j = A w_j).
    """
    W = _f64(W)
    H = _f64(H)
    c = code_offsets(codes, zeros, g)
    rows, G, _ = c.shape
    cflat = c.reshape(rows, -1)
    Hw = W @ H.T                       # row j holds (H w_j)^T
    rhs = (cflat * Hw).reshape(rows, G, g).sum(axis=2)
    gram = np.empty((rows, G, G))
    for h in range(G):
        blk = slice(h * g, (h + 1) * g)
        Hc_h = c[:, h, :] @ H[:, blk].T    # row j holds (H_{:,h} c_h)^T
        gram[:, :, h] = (cflat * Hc_h).reshape(rows, G, g).sum(axis=2)
    return gram, rhs


def _needs_ridge(Gs, rcond):
    """Trigger of the stabilised solve (App. E.2): nonfinite spectrum, small eigenvalue."""
    if not np.all(np.isfinite(Gs)):
        return True
    ev = np.linalg.eigvalsh(Gs)
    if not np.all(np.isfinite(ev)):
        return True
    return ev[0] <= rcond * max(abs(ev[-1]), FP32_EPS)


def _cholesky_or_none(M):
    try:
        L = np.linalg.cholesky(M)
    except np.linalg.LinAlgError:
        return None
    if not np.all(np.isfinite(L)):
        return None
    return L


def scale_objective_change(gram, rhs, s_new, s_old):
    """F_j(s_new) - F_j(s_old) at fixed codes, per row.

    F_j(s) = ||y_j - B_j s||^2 = y_j^T y_j - 2 s^T B_j^T y_j + s^T B_j^T B_j s
    (eq. (5)), so the difference needs only the Gram matrix and the right-hand
    side: q(s_new) - q(s_old) with q(s) = s^T (B^T B) s - 2 (B^T y)^T s.
    """
    gram = _f64(gram)
    rhs = _f64(rhs)
    Gs = 0.5 * (gram + np.swapaxes(gram, 1, 2))

    def q(s):
        s = _f64(s)
        return np.einsum("ji,jih,jh->j", s, Gs, s) - 2.0 * np.einsum("ji,ji->j", rhs, s)

    return q(s_new) - q(s_old)


def solve_scales(gram, rhs, lam=RIDGE_LAMBDA, rcond=RIDGE_RCOND, prev=None):
    """Solve every row's normal equations eq. (6) with the ridge rule of App. E.2.

    Returns (scales [rows, G], ridge [rows] bool).  Raises ScaleSolveError if a
    row's factorisation fails again after adding lam * I.  With ``prev`` (the
    row's previous scales) a ridge solution that would increase F_j is
    replaced by ``prev`` (ridge acceptance, the remark of App. G.5); the ridge
    flag stays set either way.
    """
    gram = _f64(gram)
    rhs = _f64(rhs)
    rows, G, _ = gram.shape
    s = np.empty((rows, G))
    ridge = np.zeros(rows, dtype=bool)
    failed = []
    for j in range(rows):
        Gs = 0.5 * (gram[j] + gram[j].T)
        L = None
        if not _needs_ridge(Gs, rcond):
            L = _cholesky_or_none(Gs)
        if L is None:
            ridge[j] = True
            L = _cholesky_or_none(Gs + lam * np.eye(G))
            if L is None:
                failed.append(j)
                s[j] = np.nan
                continue
        y = solve_triangular(L, rhs[j], lower=True, check_finite=False)
        s[j] = solve_triangular(L.T, y, lower=False, check_finite=False)
    if failed:
        raise ScaleSolveError(failed)
    if prev is not None and np.any(ridge):
        ir = np.nonzero(ridge)[0]
        worse = scale_objective_change(gram[ir], rhs[ir], s[ir], _f64(prev)[ir]) > 0.0
        s[ir[worse]] = _f64(prev)[ir[worse]]
    return s, ridge


def scale_step(W, H, codes, zeros, g, lam=RIDGE_LAMBDA, rcond=RIDGE_RCOND, prev=None):
    """Joint scale update of Sec. 3.3.1: (scales, ridge flags) for the given codes.

    ``prev`` (previous scales) turns on ridge acceptance (see solve_scales).
    """
    gram, rhs = gram_system(W, H, codes, zeros, g)
    return solve_scales(gram, rhs, lam, rcond, prev)


@dataclasses.dataclass
class CodeTrace:
    """What one code sweep decided, per row and group (for tests and parity)."""
    x: np.ndarray          # [rows, cols] pre-rounding values of eq. (10)
    cand: np.ndarray       # [rows, cols] proposals (old codes where skipped)
    decision: np.ndarray   # [rows, G] DEC_REJECT / DEC_ACCEPT / DEC_SKIP
    err_old: np.ndarray    # [rows, G] s^2 ||v - R(q_old - z)||^2
    err_new: np.ndarray    # [rows, G] s^2 ||v - R(q_cand - z)||^2


def babai_group(v, R, z, qmax):
    """Bounded Babai back substitution eq. (10) for a batch of rows.

    v [rows, g] (already divided by the scale), R [g, g] upper triangular,
    z [rows] integer zero points.  Returns (candidate codes, pre-rounding values).
    """
    rows, g = v.shape
    cand = np.zeros((rows, g))
    x = np.zeros((rows, g))
    for l in range(g - 1, -1, -1):
        tail = (cand[:, l + 1:] - z[:, None]) @ R[l, l + 1:]
        x[:, l] = z + (v[:, l] - tail) / R[l, l]
        cand[:, l] = np.clip(np.rint(x[:, l]), 0, qmax)
    return cand, x


def code_step(W, H, R, codes, scales, zeros, g, bits, record=False):
    """One Gauss-Seidel sweep of bounded Babai proposals over the groups (Sec. 3.3.2).

    Returns the new codes (uint8) and, if ``record``, a CodeTrace.
    """
    W = _f64(W)
    H = _f64(H)
    s = _f64(scales)
    zf = _f64(zeros)
    qmax = (1 << bits) - 1
    rows, cols = W.shape
    G = cols // g
    q = np.asarray(codes).astype(np.int64).copy()
    if record:
        tr = CodeTrace(np.full((rows, cols), np.nan), q.astype(np.uint8).copy(),
                       np.full((rows, G), DEC_SKIP, dtype=np.uint8),
                       np.full((rows, G), np.nan), np.full((rows, G), np.nan))
    for i in range(G):
        blk = slice(i * g, (i + 1) * g)
        # eq. (7): every other group at its latest codes (new for h < i, previous
        # for h > i), all at the new scales.
        what = dequantize(q, s, zeros, g)
        what[:, blk] = 0.0
        aty = (W - what) @ H[blk, :].T          # A_i^T y^(i,k) = (H w)_i - sum_{h!=i} s_h H_ih c_h
        si = s[:, i]
        active = np.abs(si) > FP32_EPS
        if not np.any(active):
            continue
        rows_a = np.nonzero(active)[0]
        # v = U_i^T y^(i,k) / s_i = R_i^{-T} A_i^T y^(i,k) / s_i
        v = solve_triangular(R[i].T, aty[rows_a].T, lower=True, check_finite=False).T / si[rows_a, None]
        za = zf[rows_a, i]
        cand, x = babai_group(v, R[i], za, qmax)
        qold = q[rows_a, blk].astype(np.float64)
        r_old = v - (qold - za[:, None]) @ R[i].T
        r_new = v - (cand - za[:, None]) @ R[i].T
        e_old = si[rows_a] ** 2 * np.sum(r_old * r_old, axis=1)
        e_new = si[rows_a] ** 2 * np.sum(r_new * r_new, axis=1)
        with np.errstate(invalid="ignore"):
            acc = np.isfinite(e_new) & (e_new < e_old)
        q[rows_a[acc], blk] = cand[acc].astype(np.int64)
        if record:
            tr.x[rows_a, blk] = x
            cand_u8 = np.where(np.isfinite(cand), cand, 0).astype(np.uint8)
            tr.cand[rows_a, blk] = cand_u8
            tr.decision[rows_a, i] = np.where(acc, DEC_ACCEPT, DEC_REJECT)
            tr.err_old[rows_a, i] = e_old
            tr.err_new[rows_a, i] = e_new
    q8 = q.astype(np.uint8)
    return (q8, tr) if record else q8


def stop_rows(L_prev, L, tau):
    """Early-stopping test of eq. (strict_stopping), App. E.2, per row.

    L_prev holds L_j^(k-1) and L holds L_j^(k), the objective right after the
    scale updates of two consecutive iterations k - 1 and k (k >= 2; there is
    no test at k = 1).  A row stops when its decrease L^(k-1) - L^(k) is at
    most tau relative to max(|L^(k-1)|, eps_fp32), or at most tau in absolute
    value.  A negative decrease (the objective went up, e.g. after a ridge
    solve) therefore always stops the row.  The stopped row keeps the new
    scales s^(k) and skips the code update of iteration k.
    """
    L_prev = _f64(L_prev)
    L = _f64(L)
    dec = L_prev - L
    rel = dec / np.maximum(np.abs(L_prev), FP32_EPS)
    return (rel <= tau) | (np.abs(dec) <= tau)


@dataclasses.dataclass
class SweepRecord:
    L: np.ndarray            # objective right after the scale update, per row
    F_after: np.ndarray      # objective after the code update, per row
    ridge: np.ndarray        # rows that took the stabilised branch
    accepted: int            # accepted group proposals
    changed: int             # codes changed
    active: np.ndarray       # rows that ran the code update this sweep


def refine(W, H, codes, scales, zeros, g, bits, K, tau=None,
           lam=RIDGE_LAMBDA, rcond=RIDGE_RCOND, R=None, ridge_accept=False):
    """Alternate scale and code updates for K iterations (Sec. 3.3, App. E.2).

    ``tau`` None disables early stopping; otherwise a row stops before its
    code update at iteration k >= 2 when the decrease of L between consecutive
    scale updates is at most tau, relatively or absolutely, keeping the new
    scales.  ``ridge_accept`` keeps a ridge solution only when it does not
    increase F_j (the remark of App. G.5).  Returns (codes uint8, scales
    float64, list of SweepRecord).
    """
    W = _f64(W)
    H = _f64(H)
    if R is None:
        R = group_factors(H, g)
    q = np.asarray(codes).astype(np.uint8).copy()
    s = _f64(scales).copy()
    rows = W.shape[0]
    active = np.ones(rows, dtype=bool)
    L_prev = None
    history = []
    for k in range(1, K + 1):
        if not np.any(active):
            break
        ia = np.nonzero(active)[0]
        s_new, ridge_a = scale_step(W[ia], H, q[ia], zeros[ia], g, lam, rcond,
                                    prev=s[ia] if ridge_accept else None)
        s[ia] = s_new
        ridge = np.zeros(rows, dtype=bool)
        ridge[ia] = ridge_a
        L = np.full(rows, np.nan)
        L[ia] = objective_rows(W[ia], H, q[ia], s[ia], zeros[ia], g)
        if tau is not None and k >= 2:
            stop = stop_rows(L_prev[ia], L[ia], tau)
            active[ia[stop]] = False
            ia = np.nonzero(active)[0]
        if L_prev is None:
            L_prev = L.copy()
        else:
            L_prev = np.where(np.isnan(L), L_prev, L)
        q_old = q.copy()
        accepted = 0
        if ia.size:
            q_new, tr = code_step(W[ia], H, R, q[ia], s[ia], zeros[ia], g, bits, record=True)
            q[ia] = q_new
            accepted = int(np.sum(tr.decision == DEC_ACCEPT))
        F_after = np.full(rows, np.nan)
        F_after[ia] = objective_rows(W[ia], H, q[ia], s[ia], zeros[ia], g) if ia.size else F_after[ia]
        history.append(SweepRecord(L, F_after, ridge, accepted,
                                   int(np.sum(q != q_old)), active.copy()))
    return q, s, history
