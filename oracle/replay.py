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
"""

from __future__ import annotations

import dataclasses

import numpy as np
from scipy.linalg import solve_triangular

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
