"""Plausible mistakes planted in the oracle (on the CPU) must trip a pin.

Each mutation replaces one piece of ``oracle.jarq`` with a wrong variant (a
transposed operand, a dropped term, a wrong sign or index, a wrong rounding,
Jacobi instead of Gauss-Seidel, ...).  The pin battery below re-runs the
pins of tests/test_oracle_pins.py against the mutated oracle; at least one
of them must fail for every mutation.
"""

import numpy as np
import pytest
from scipy.linalg import solve_triangular

from oracle import jarq
from tests import test_oracle_pins as pins

_ORIG = {name: getattr(jarq, name) for name in
         ("babai_group", "code_step", "gram_system", "solve_scales",
          "group_factors", "objective_rows", "dequantize", "refine")}


def _battery():
    """Run the pins; return the names of those that fail."""
    mc = pins.build_multicode()
    st = pins.build_staleness()
    tl = pins.build_tiny_layer()
    checks = [
        ("multicode_refit", lambda: pins.test_multicode_scale_refit(mc)),
        ("multicode_nbrs", lambda: [pins.test_multicode_single_code_neighbours(mc, c, k) for c, k in
                                    [((0, 2), "nbr_0_2"), ((3, 2), "nbr_3_2"), ((1, 3), "nbr_1_3")]]),
        ("multicode_babai", lambda: pins.test_multicode_babai_step(mc)),
        ("staleness_trace", lambda: pins.test_staleness_full_trace(st)),
        ("staleness_host", lambda: pins.test_staleness_babai_at_host_scale_keeps_host(st)),
        ("bruteforce_g1", lambda: pins.test_babai_vs_bruteforce(1, 3, False)),
        ("bruteforce_diag", lambda: pins.test_babai_vs_bruteforce(3, 2, True)),
        ("bruteforce_full", lambda: pins.test_babai_vs_bruteforce(3, 3, False)),
        ("lstsq", lambda: pins.test_scale_step_matches_lstsq(tl)),
        ("independent", lambda: pins.test_block_diagonal_hessian_gives_independent_fits()),
        ("ridge", lambda: pins.test_ridge_branch_on_singular_gram()),
        ("ridge_large_pivots", pins.test_ridge_trigger_is_the_spectrum_not_the_pivots),
        ("qr_form", lambda: pins.test_qr_form_equals_hessian_form(tl)),
        ("monotone", lambda: pins.test_monotone_descent_and_host_bound(tl)),
        ("babai_bound", lambda: pins.test_unclipped_babai_residual_bound(tl)),
        ("stop_sequences", pins.test_stopping_rule_on_hand_built_sequences),
        ("stop_counts", pins.test_stopping_rule_active_counts),
        ("stop_idle_rows", lambda: pins.test_row_without_accepts_stops_at_the_next_iteration(tl)),
    ]
    failed = []
    for name, fn in checks:
        try:
            with np.errstate(all="ignore"):
                fn()
        except Exception:       # an assertion or a crash both count as a catch
            failed.append(name)
    return failed


# --- mutated pieces --------------------------------------------------------

def _babai_factory(tail_transposed=False, drop_zero=False, rounding=np.rint, clip_hi=0):
    def babai_group(v, R, z, qmax):
        rows, g = v.shape
        cand = np.zeros((rows, g))
        x = np.zeros((rows, g))
        for l in range(g - 1, -1, -1):
            coef = R[l + 1:, l] if tail_transposed else R[l, l + 1:]
            off = 0.0 if drop_zero else z[:, None]
            tail = (cand[:, l + 1:] - off) @ coef
            base = 0.0 if drop_zero else z
            x[:, l] = base + (v[:, l] - tail) / R[l, l]
            cand[:, l] = np.clip(rounding(x[:, l]), 0, qmax - clip_hi)
        return cand, x
    return babai_group


def _code_step_factory(jacobi=False, residual_sign=-1.0, divide_by_scale=True, accept_inverted=False):
    def code_step(W, H, R, codes, scales, zeros, g, bits, record=False):
        W = np.asarray(W, dtype=np.float64)
        H = np.asarray(H, dtype=np.float64)
        s = np.asarray(scales, dtype=np.float64)
        zf = np.asarray(zeros, dtype=np.float64)
        qmax = (1 << bits) - 1
        rows, cols = W.shape
        G = cols // g
        q = np.asarray(codes).astype(np.int64).copy()
        q_start = q.copy()
        tr = jarq.CodeTrace(np.full((rows, cols), np.nan), q.astype(np.uint8).copy(),
                            np.full((rows, G), jarq.DEC_SKIP, dtype=np.uint8),
                            np.full((rows, G), np.nan), np.full((rows, G), np.nan))
        for i in range(G):
            blk = slice(i * g, (i + 1) * g)
            what = jarq.dequantize(q_start if jacobi else q, s, zeros, g)
            what[:, blk] = 0.0
            aty = (W + residual_sign * what) @ H[blk, :].T
            si = s[:, i]
            rows_a = np.nonzero(np.abs(si) > jarq.FP32_EPS)[0]
            v = solve_triangular(R[i].T, aty[rows_a].T, lower=True, check_finite=False).T
            if divide_by_scale:
                v = v / si[rows_a, None]
            za = zf[rows_a, i]
            cand, x = jarq.babai_group(v, R[i], za, qmax)
            qold = q[rows_a, blk].astype(np.float64)
            r_old = v - (qold - za[:, None]) @ R[i].T
            r_new = v - (cand - za[:, None]) @ R[i].T
            e_old = si[rows_a] ** 2 * np.sum(r_old * r_old, axis=1)
            e_new = si[rows_a] ** 2 * np.sum(r_new * r_new, axis=1)
            acc = np.isfinite(e_new) & ((e_new > e_old) if accept_inverted else (e_new < e_old))
            q[rows_a[acc], blk] = cand[acc].astype(np.int64)
            tr.x[rows_a, blk] = x
            tr.cand[rows_a, blk] = np.clip(cand, 0, 255).astype(np.uint8)
            tr.decision[rows_a, i] = np.where(acc, jarq.DEC_ACCEPT, jarq.DEC_REJECT)
            tr.err_old[rows_a, i] = e_old
            tr.err_new[rows_a, i] = e_new
        q8 = q.astype(np.uint8)
        return (q8, tr) if record else q8
    return code_step


def _gram_factory(rhs_without_h=False, no_coupling=False, rhs_sign=1.0):
    def gram_system(W, H, codes, zeros, g):
        gram, rhs = _ORIG["gram_system"](W, H, codes, zeros, g)
        if rhs_without_h:
            c = jarq.code_offsets(codes, zeros, g)
            rows, G, _ = c.shape
            rhs = (c.reshape(rows, -1) * np.asarray(W, np.float64)).reshape(rows, G, g).sum(axis=2)
        if no_coupling:
            gram = gram * np.eye(gram.shape[1])[None]
        return gram, rhs_sign * rhs
    return gram_system


def _solve_factory(always_ridge=False, never_ridge=False):
    def solve_scales(gram, rhs, lam=jarq.RIDGE_LAMBDA, rcond=jarq.RIDGE_RCOND):
        gram = np.asarray(gram, dtype=np.float64)
        rows, G, _ = gram.shape
        if always_ridge:
            gram = gram + lam * np.eye(G)[None]
            s, ridge = _ORIG["solve_scales"](gram, rhs, lam=0.0, rcond=-1.0)
            return s, np.ones(rows, dtype=bool)
        if never_ridge:
            s = np.stack([np.linalg.lstsq(gram[j], rhs[j], rcond=None)[0] for j in range(rows)])
            return s, np.zeros(rows, dtype=bool)
        return _ORIG["solve_scales"](gram, rhs, lam, rcond)
    return solve_scales


def _needs_ridge_from_pivots(Gs, rcond):
    """The trigger taken from the Cholesky pivots instead of the spectrum."""
    if not np.all(np.isfinite(Gs)):
        return True
    try:
        L = np.linalg.cholesky(Gs)
    except np.linalg.LinAlgError:
        return True
    return np.min(np.diag(L)) ** 2 <= rcond * max(np.max(np.diag(Gs)), jarq.FP32_EPS)


def _factors_lower(H, g):
    return np.transpose(_ORIG["group_factors"](H, g), (0, 2, 1))


def _objective_without_h(W, H, codes, scales, zeros, g):
    E = np.asarray(W, np.float64) - jarq.dequantize(codes, scales, zeros, g)
    return np.sum(E * E, axis=1)


def _dequantize_no_zero(codes, scales, zeros, g):
    return _ORIG["dequantize"](codes, scales, np.zeros_like(zeros), g)


def _refine_factory(and_not_or=False, first_k=2, keep_old_scales=False, denom_current=False):
    """refine() with a planted mistake in the early-stopping rule.

    and_not_or: both tests of eq. (strict_stopping) must hold; first_k = 1:
    the test also runs at k = 1, against the host state's objective;
    keep_old_scales: a stopped row goes back to its previous scales;
    denom_current: the relative decrease is divided by L^(k), not L^(k-1).
    """
    def refine(W, H, codes, scales, zeros, g, bits, K, tau=None, lam=jarq.RIDGE_LAMBDA,
               rcond=jarq.RIDGE_RCOND, R=None, ridge_accept=False):
        W = np.asarray(W, dtype=np.float64)
        H = np.asarray(H, dtype=np.float64)
        if R is None:
            R = jarq.group_factors(H, g)
        q = np.asarray(codes).astype(np.uint8).copy()
        s = np.asarray(scales, dtype=np.float64).copy()
        rows = W.shape[0]
        active = np.ones(rows, dtype=bool)
        L_prev = jarq.objective_rows(W, H, q, s, zeros, g) if first_k == 1 else None
        history = []
        for k in range(1, K + 1):
            if not np.any(active):
                break
            ia = np.nonzero(active)[0]
            s_old = s.copy()
            s_new, ridge_a = jarq.scale_step(W[ia], H, q[ia], zeros[ia], g, lam, rcond)
            s[ia] = s_new
            L = np.full(rows, np.nan)
            L[ia] = jarq.objective_rows(W[ia], H, q[ia], s[ia], zeros[ia], g)
            if tau is not None and k >= first_k:
                dec = L_prev[ia] - L[ia]
                base = np.abs(L[ia]) if denom_current else np.abs(L_prev[ia])
                rel = dec / np.maximum(base, jarq.FP32_EPS)
                stop = ((rel <= tau) & (np.abs(dec) <= tau)) if and_not_or else \
                    ((rel <= tau) | (np.abs(dec) <= tau))
                active[ia[stop]] = False
                if keep_old_scales:
                    s[ia[stop]] = s_old[ia[stop]]
                ia = np.nonzero(active)[0]
            L_prev = L.copy() if L_prev is None else np.where(np.isnan(L), L_prev, L)
            q_old = q.copy()
            accepted = 0
            if ia.size:
                q_new, tr = jarq.code_step(W[ia], H, R, q[ia], s[ia], zeros[ia], g, bits, record=True)
                q[ia] = q_new
                accepted = int(np.sum(tr.decision == jarq.DEC_ACCEPT))
            F_after = np.full(rows, np.nan)
            if ia.size:
                F_after[ia] = jarq.objective_rows(W[ia], H, q[ia], s[ia], zeros[ia], g)
            history.append(jarq.SweepRecord(L, F_after, np.zeros(rows, bool), accepted,
                                            int(np.sum(q != q_old)), active.copy()))
        return q, s, history
    return refine


MUTATIONS = {
    "babai_tail_transposed": ("babai_group", _babai_factory(tail_transposed=True)),
    "babai_drops_zero_point": ("babai_group", _babai_factory(drop_zero=True)),
    "babai_floor_not_round": ("babai_group", _babai_factory(rounding=np.floor)),
    "babai_clip_one_short": ("babai_group", _babai_factory(clip_hi=1)),
    "jacobi_not_gauss_seidel": ("code_step", _code_step_factory(jacobi=True)),
    "residual_sign_flipped": ("code_step", _code_step_factory(residual_sign=+1.0)),
    "v_not_divided_by_scale": ("code_step", _code_step_factory(divide_by_scale=False)),
    "accept_test_inverted": ("code_step", _code_step_factory(accept_inverted=True)),
    "rhs_without_hessian": ("gram_system", _gram_factory(rhs_without_h=True)),
    "gram_without_coupling": ("gram_system", _gram_factory(no_coupling=True)),
    "rhs_sign_flipped": ("gram_system", _gram_factory(rhs_sign=-1.0)),
    "ridge_always": ("solve_scales", _solve_factory(always_ridge=True)),
    "ridge_never": ("solve_scales", _solve_factory(never_ridge=True)),
    "ridge_from_pivots": ("_needs_ridge", _needs_ridge_from_pivots),
    "factor_lower_not_upper": ("group_factors", _factors_lower),
    "objective_without_hessian": ("objective_rows", _objective_without_h),
    "dequantize_drops_zero_point": ("dequantize", _dequantize_no_zero),
    "stop_and_not_or": ("refine", _refine_factory(and_not_or=True)),
    "stop_from_first_iteration": ("refine", _refine_factory(first_k=1)),
    "stop_keeps_old_scales": ("refine", _refine_factory(keep_old_scales=True)),
    "stop_relative_to_current": ("refine", _refine_factory(denom_current=True)),
}


def test_refine_factory_without_mistakes_passes_the_stopping_pins(monkeypatch):
    # the mutated copies differ from the oracle only in the planted mistake
    monkeypatch.setattr(jarq, "refine", _refine_factory())
    assert _battery() == []


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutation_is_caught(name, monkeypatch):
    attr, fn = MUTATIONS[name]
    monkeypatch.setattr(jarq, attr, fn)
    failed = _battery()
    assert failed, f"mutation {name} passed every pin"


def test_unmutated_oracle_passes_battery():
    assert _battery() == []
