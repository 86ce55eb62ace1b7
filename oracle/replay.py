"""Teacher-forced re-evaluation of a code sweep (test oracle).

TEST INFRASTRUCTURE ONLY.

Another implementation (the HIP path) reports, for one code sweep started
from codes q0 at scales s, its proposal for every group (``cand``) and its
decision per group (accept / reject / skip).  A single decision that falls
the other way near a rounding boundary changes every later decision of that
row, so the decisions are checked one at a time, each conditioned on the
other implementation's earlier decisions:

* group i is evaluated at the state in which groups h < i hold the other
  implementation's final codes and groups h >= i hold q0 (eq. (7));
* position l of the back substitution eq. (10) uses the other
  implementation's proposal for the positions m > l of the same group;
* the accept test eq. (8) is evaluated on the other implementation's proposal.

Every quantity is then computed in float64 from the definitions, as in
``oracle.jarq``.  A proposal position disagrees legitimately only when the
float64 pre-rounding value lies within ``x_tol`` of a rounding boundary
m + 1/2 with 0 <= m < 2^b - 1, and an accept decision only when the float64
change of the objective is within ``f_tol`` of zero relative to the size of
its terms.

``forced_refine`` runs K whole iterations of the oracle (scale step,
objective, stopping test of eq. (strict_stopping), code sweep) on its own
state and takes the other implementation's decision only where the two may
legitimately differ by the same bands (and, for a stopping decision, where
the test flips under a small relative change of either objective).  A single
near-boundary split early in a run changes every later decision of the row;
forcing those splits lets the end-to-end objective of the two
implementations be compared on the same trajectory.
"""

from __future__ import annotations

import dataclasses

import numpy as np
from scipy.linalg import solve_triangular

from . import jarq
from .jarq import DEC_ACCEPT, DEC_REJECT, DEC_SKIP, FP32_EPS, dequantize


@dataclasses.dataclass
class ReplayReport:
    n_codes: int               # proposal positions checked
    code_mismatch: int         # disagreeing positions outside the boundary band
    code_exempt: int           # disagreeing positions inside the band
    near_boundary: int         # positions whose float64 value is inside the band
    n_groups: int              # group decisions checked
    decision_mismatch: int     # accept/reject disagreements outside the margin
    decision_exempt: int       # accept/reject disagreements inside the margin
    skip_mismatch: int         # skip decisions that differ (must be zero)
    worst_x_gap: float         # largest |x - boundary| among non-exempt mismatches

    @property
    def ok(self) -> bool:
        return self.code_mismatch == 0 and self.decision_mismatch == 0 and self.skip_mismatch == 0


def _band(x, qmax, x_tol):
    """True where x is within x_tol of a boundary m + 1/2, 0 <= m < qmax."""
    nearest = np.floor(x) + 0.5          # the closest half-integer to x
    inside = (nearest >= 0.5) & (nearest <= qmax - 0.5)
    return inside & (np.abs(x - nearest) <= x_tol)


def replay_code_step(W, H, R, q0, scales, zeros, g, bits, cand, decision,
                     x_tol=1e-4, f_tol=1e-5):
    """Check another implementation's sweep decision by decision (see module doc)."""
    W = np.asarray(W, dtype=np.float64)
    H = np.asarray(H, dtype=np.float64)
    s = np.asarray(scales, dtype=np.float64)
    zf = np.asarray(zeros, dtype=np.float64)
    q0 = np.asarray(q0).astype(np.int64)
    cand = np.asarray(cand).astype(np.int64)
    decision = np.asarray(decision)
    qmax = (1 << bits) - 1
    rows, cols = W.shape
    G = cols // g
    # The other implementation's state after its own decisions.
    final = q0.copy()
    for i in range(G):
        blk = slice(i * g, (i + 1) * g)
        acc = decision[:, i] == DEC_ACCEPT
        final[acc, blk] = cand[acc, blk]
    n_codes = code_mismatch = code_exempt = near = 0
    n_groups = dec_mismatch = dec_exempt = skip_mismatch = 0
    worst = 0.0
    for i in range(G):
        blk = slice(i * g, (i + 1) * g)
        cond = np.concatenate([final[:, :i * g], q0[:, i * g:]], axis=1)
        si = s[:, i]
        skip = ~(np.abs(si) > FP32_EPS)
        skip_mismatch += int(np.sum(skip != (decision[:, i] == DEC_SKIP)))
        rows_a = np.nonzero(~skip & (decision[:, i] != DEC_SKIP))[0]
        if rows_a.size == 0:
            continue
        what = dequantize(cond[rows_a], s[rows_a], zeros[rows_a], g)
        what[:, blk] = 0.0
        aty = (W[rows_a] - what) @ H[blk, :].T
        Ri = R[i]
        v = solve_triangular(Ri.T, aty.T, lower=True, check_finite=False).T / si[rows_a, None]
        za = zf[rows_a, i]
        cg = cand[rows_a, blk].astype(np.float64)
        x = np.empty_like(v)
        for l in range(g - 1, -1, -1):
            tail = (cg[:, l + 1:] - za[:, None]) @ Ri[l, l + 1:]
            x[:, l] = za + (v[:, l] - tail) / Ri[l, l]
        mine = np.clip(np.rint(x), 0, qmax)
        band = _band(x, qmax, x_tol)
        diff = mine != cg
        n_codes += x.size
        near += int(np.sum(band))
        code_exempt += int(np.sum(diff & band))
        bad = diff & ~band
        code_mismatch += int(np.sum(bad))
        if np.any(bad):
            m = np.floor(x[bad])
            gap = np.min(np.abs(x[bad] - (m + 0.5)))
            worst = max(worst, float(gap))
        # Accept test on the other implementation's proposal.
        qold = cond[rows_a, blk].astype(np.float64)
        r_old = v - (qold - za[:, None]) @ Ri.T
        r_new = v - (cg - za[:, None]) @ Ri.T
        e_old = si[rows_a] ** 2 * np.sum(r_old * r_old, axis=1)
        e_new = si[rows_a] ** 2 * np.sum(r_new * r_new, axis=1)
        with np.errstate(invalid="ignore"):
            acc = np.isfinite(e_new) & (e_new < e_old)
        theirs = decision[rows_a, i] == DEC_ACCEPT
        # Size of the terms of dF = delta^T H_ii delta - 2 delta^T (H e)_i.
        delta = si[rows_a, None] * (cg - qold)
        dHd = np.einsum("rg,gh,rh->r", delta, H[blk, blk], delta)
        e_cur = W[rows_a] - dequantize(cond[rows_a], s[rows_a], zeros[rows_a], g)
        he = e_cur @ H[blk, :].T
        dhe = np.einsum("rg,rg->r", delta, he)
        margin = f_tol * (np.abs(dHd) + 2 * np.abs(dhe))
        dF = e_new - e_old
        n_groups += rows_a.size
        differ = acc != theirs
        ex = differ & (np.abs(dF) <= margin)
        dec_exempt += int(np.sum(ex))
        dec_mismatch += int(np.sum(differ & ~ex))
    return ReplayReport(n_codes, code_mismatch, code_exempt, near, n_groups,
                        dec_mismatch, dec_exempt, skip_mismatch, worst)


__all__ = ["ReplayReport", "replay_code_step", "DEC_ACCEPT", "DEC_REJECT", "DEC_SKIP"]


# ---------------------------------------------------------------------------
# K iterations that defer to another implementation only inside the bands
# ---------------------------------------------------------------------------

@dataclasses.dataclass
class ForcedReport:
    sweeps: int                # iterations run
    n_codes: int               # proposal positions evaluated
    code_forced: int           # positions where the other's proposal was taken (inside the band)
    code_mismatch: int         # positions where they differ outside the band (own value kept)
    n_groups: int              # accept decisions evaluated
    decision_forced: int       # accept decisions taken from the other (inside the margin)
    decision_mismatch: int     # accept decisions that differ outside the margin (own kept)
    skip_mismatch: int         # small-scale skips that differ
    n_stops: int               # stopping tests evaluated
    stop_forced: int           # stopping decisions taken from the other (inside the band)
    stop_mismatch: int         # stopping decisions that differ outside the band (own kept)
    active: list               # rows that ran the code update, per iteration

    @property
    def ok(self) -> bool:
        return (self.code_mismatch == 0 and self.decision_mismatch == 0 and self.skip_mismatch == 0
                and self.stop_mismatch == 0)


def stop_band(L_prev, L, tau, l_tol):
    """True where the stopping test of eq. (strict_stopping) changes its answer
    when L^(k-1) or L^(k) moves by a relative l_tol (the test at the four
    corners is not unanimous)."""
    L_prev = np.asarray(L_prev, dtype=np.float64)
    L = np.asarray(L, dtype=np.float64)
    answers = [jarq.stop_rows(L_prev * (1 + a * l_tol), L * (1 + b * l_tol), tau)
               for a in (-1, 1) for b in (-1, 1)]
    first = answers[0]
    return np.logical_or.reduce([ans != first for ans in answers[1:]])


def forced_refine(W, H, q0, s0, zeros, g, bits, K, cand, decision, tau=None, stop_at=None,
                  R=None, x_tol=1e-4, f_tol=1e-5, l_tol=1e-6,
                  lam=jarq.RIDGE_LAMBDA, rcond=jarq.RIDGE_RCOND):
    """The oracle's own K iterations, taking another implementation's decision
    only where the two may legitimately differ.

    ``cand[k]``, ``decision[k]`` ([rows, cols] and [rows, G]) are the other
    implementation's proposals and decisions in iteration k + 1, as
    ``replay_code_step`` reads them; ``stop_at[r]`` (with ``tau``) is the
    iteration at which it stopped row r, 0 if never.  Every iteration runs the
    oracle's scale step, objective and stopping test on its own state, then a
    Gauss-Seidel code sweep in the oracle's float64 arithmetic.  Where the
    oracle's value of a decision lies inside the band of ``replay_code_step``
    (a pre-rounding value within x_tol of a rounding boundary, an objective
    change within f_tol of zero relative to its terms) or of ``stop_band``
    (the stopping test flips when either objective moves by a relative l_tol)
    and the other decided differently, the other's decision is taken and
    counted; every other disagreement is counted as a mismatch and the oracle
    keeps its own decision.  With no mismatch, the returned state follows the
    other implementation's trajectory exactly in its codes and the oracle's
    own float64 scale solves.

    Returns (codes uint8, scales float64, ForcedReport).
    """
    W = np.asarray(W, dtype=np.float64)
    H = np.asarray(H, dtype=np.float64)
    zf = np.asarray(zeros, dtype=np.float64)
    if R is None:
        R = jarq.group_factors(H, g)
    qmax = (1 << bits) - 1
    rows, cols = W.shape
    G = cols // g
    q = np.asarray(q0).astype(np.int64).copy()
    s = np.asarray(s0, dtype=np.float64).copy()
    active = np.ones(rows, dtype=bool)
    L_prev = np.full(rows, np.nan)
    n_codes = code_forced = code_mismatch = 0
    n_groups = dec_forced = dec_mismatch = skip_mismatch = 0
    n_stops = stop_forced = stop_mismatch = 0
    active_hist = []
    run = 0
    for k in range(1, K + 1):
        if not np.any(active):
            break
        run += 1
        ia = np.nonzero(active)[0]
        s[ia], _ = jarq.scale_step(W[ia], H, q[ia].astype(np.uint8), zeros[ia], g, lam, rcond)
        L = jarq.objective_rows(W[ia], H, q[ia], s[ia], zeros[ia], g)
        if tau is not None and k >= 2:
            own = jarq.stop_rows(L_prev[ia], L, tau)
            theirs = np.asarray(stop_at)[ia] == k
            band = stop_band(L_prev[ia], L, tau, l_tol)
            differ = own != theirs
            n_stops += ia.size
            stop_forced += int(np.sum(differ & band))
            stop_mismatch += int(np.sum(differ & ~band))
            stop = np.where(differ & band, theirs, own)
            L_prev[ia] = L
            active[ia[stop]] = False
            ia = np.nonzero(active)[0]
        else:
            L_prev[ia] = L
        active_hist.append(active.copy())
        if ia.size == 0:
            continue
        cand_k = np.asarray(cand[k - 1]).astype(np.int64)
        dec_k = np.asarray(decision[k - 1])
        for i in range(G):
            blk = slice(i * g, (i + 1) * g)
            si = s[ia, i]
            own_skip = ~(np.abs(si) > jarq.FP32_EPS)
            their_skip = dec_k[ia, i] == DEC_SKIP
            skip_mismatch += int(np.sum(own_skip != their_skip))
            sel = np.nonzero(~own_skip)[0]
            if sel.size == 0:
                continue
            rr = ia[sel]
            comparable = ~their_skip[sel]
            what = jarq.dequantize(q[rr], s[rr], zeros[rr], g)
            e_cur = W[rr] - what
            what[:, blk] = 0.0
            aty = (W[rr] - what) @ H[blk, :].T
            Ri = R[i]
            sr = s[rr, i]
            v = solve_triangular(Ri.T, aty.T, lower=True, check_finite=False).T / sr[:, None]
            za = zf[rr, i]
            other = cand_k[rr, blk]
            cg = np.zeros((rr.size, g))
            for l in range(g - 1, -1, -1):
                tail = (cg[:, l + 1:] - za[:, None]) @ Ri[l, l + 1:]
                x = za + (v[:, l] - tail) / Ri[l, l]
                mine = np.clip(np.rint(x), 0, qmax)
                differ = comparable & (mine != other[:, l])
                band = _band(x, qmax, x_tol)
                code_forced += int(np.sum(differ & band))
                code_mismatch += int(np.sum(differ & ~band))
                cg[:, l] = np.where(differ & band, other[:, l], mine)
            n_codes += int(np.sum(comparable)) * g
            qold = q[rr, blk].astype(np.float64)
            r_old = v - (qold - za[:, None]) @ Ri.T
            r_new = v - (cg - za[:, None]) @ Ri.T
            e_old = sr ** 2 * np.sum(r_old * r_old, axis=1)
            e_new = sr ** 2 * np.sum(r_new * r_new, axis=1)
            with np.errstate(invalid="ignore"):
                acc = np.isfinite(e_new) & (e_new < e_old)
            theirs = dec_k[rr, i] == DEC_ACCEPT
            delta = sr[:, None] * (cg - qold)
            dHd = np.einsum("rg,gh,rh->r", delta, H[blk, blk], delta)
            dhe = np.einsum("rg,rg->r", delta, e_cur @ H[blk, :].T)
            margin = f_tol * (np.abs(dHd) + 2 * np.abs(dhe))
            differ = comparable & (acc != theirs)
            inside = np.abs(e_new - e_old) <= margin
            n_groups += int(np.sum(comparable))
            dec_forced += int(np.sum(differ & inside))
            dec_mismatch += int(np.sum(differ & ~inside))
            acc = np.where(differ & inside, theirs, acc)
            q[rr[acc], blk] = cg[acc].astype(np.int64)
    rep = ForcedReport(run, n_codes, code_forced, code_mismatch, n_groups, dec_forced,
                       dec_mismatch, skip_mismatch, n_stops, stop_forced, stop_mismatch,
                       active_hist)
    return q.astype(np.uint8), s, rep


__all__ += ["ForcedReport", "forced_refine", "stop_band"]
