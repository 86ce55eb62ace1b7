"""Pins of the float64 oracle against values the paper fixes.

Worked examples (App. G.2, G.3), brute-force enumeration of small boxes,
closed forms of the scale step (eq. (6), App. G.1), the QR-form / Hessian-form
equivalence (App. E.1), and the invariants of Theorem 1, Corollary 1 and the
propositions of App. G.4 and G.6.
"""

import itertools

import numpy as np
import pytest

from oracle import jarq, qrform
from tests import _golden

EPS = 1e-12


def _single_group(w, H):
    W = np.asarray(w, dtype=np.float64)[None, :]
    Hm = np.asarray(H, dtype=np.float64)
    z = np.zeros((1, 1), dtype=np.int32)
    return W, Hm, z


def _refit_error(W, H, q, z, g):
    """phi(q) = min_s F(s, q): scale step, then the objective."""
    s, _ = jarq.scale_step(W, H, q, z, g)
    return float(jarq.objective_rows(W, H, q, s, z, g)[0]), s


# ---------------------------------------------------------------------------
# Proposition "Descent beyond single-code updates", App. G.2
# ---------------------------------------------------------------------------

def build_multicode():
    gv = _golden.load("prop_multicode_descent.txt")
    R = np.array([[float(x) for x in gv["R_row0"]], [float(x) for x in gv["R_row1"]]])
    y = np.array([float(x) for x in gv["y"]])
    w = np.linalg.solve(R, y)               # y = R w (main target)
    H = R.T @ R                             # A^T A in the reduced form
    return gv, R, w, H


@pytest.fixture(scope="module")
def multicode():
    return build_multicode()


def test_multicode_scale_refit(multicode):
    gv, R, w, H = multicode
    W, Hm, z = _single_group(w, H)
    q0 = np.array([[int(v) for v in gv["q0"]]], dtype=np.uint8)
    phi, s = _refit_error(W, Hm, q0, z, 2)
    assert abs(s[0, 0] - float(gv["s0"])) < EPS
    assert abs(phi - float(gv["phi_q0"])) < EPS


@pytest.mark.parametrize("codes,key", [((0, 2), "nbr_0_2"), ((2, 2), "nbr_2_2"),
                                       ((3, 2), "nbr_3_2"), ((1, 0), "nbr_1_0"),
                                       ((1, 1), "nbr_1_1"), ((1, 3), "nbr_1_3")])
def test_multicode_single_code_neighbours(multicode, codes, key):
    gv, R, w, H = multicode
    W, Hm, z = _single_group(w, H)
    phi, _ = _refit_error(W, Hm, np.array([codes], dtype=np.uint8), z, 2)
    assert abs(phi - float(gv[key])) < EPS
    assert phi > float(gv["phi_q0"])


def test_multicode_figure_grid(multicode):
    gv, R, w, H = multicode
    raw = _golden.load("prop_multicode_descent.txt", raw=True)
    W, Hm, z = _single_group(w, H)
    for q1 in range(4):
        printed = raw[f"grid_q1_{q1}"]
        for q2 in range(4):
            phi, _ = _refit_error(W, Hm, np.array([[q1, q2]], dtype=np.uint8), z, 2)
            tol = 1e-12 if printed[q2] == "0" else _golden.printed_tolerance(printed[q2])
            assert abs(phi - float(_golden._num(printed[q2]))) <= tol + 1e-12, (q1, q2, phi)


def test_multicode_babai_step(multicode):
    gv, R, w, H = multicode
    W, Hm, z = _single_group(w, H)
    q0 = np.array([[1, 2]], dtype=np.uint8)
    s0 = np.array([[float(gv["s0"])]])
    Rg = jarq.group_factors(Hm, 2)
    qn, tr = jarq.code_step(W, Hm, Rg, q0, s0, z, 2, 2, record=True)
    assert abs(tr.x[0, 1] - float(gv["babai_x2"])) < EPS
    assert abs(tr.x[0, 0] - float(gv["babai_x1"])) < EPS
    assert list(qn[0]) == [int(v) for v in gv["q_plus"]]
    assert tr.decision[0, 0] == jarq.DEC_ACCEPT
    f_plus = jarq.objective_rows(W, Hm, qn, s0, z, 2)[0]
    assert abs(f_plus - float(gv["f_s0_qplus"])) < EPS
    # reduced-form error of the proposal (App. G.4) equals the full objective here
    assert abs(tr.err_new[0, 0] - float(gv["f_s0_qplus"])) < EPS
    phi, s = _refit_error(W, Hm, qn, z, 2)
    assert abs(s[0, 0] - float(gv["s_plus"])) < EPS
    assert abs(phi - float(gv["f_plus"])) < EPS


def test_multicode_refine_two_sweeps(multicode):
    gv, R, w, H = multicode
    W, Hm, z = _single_group(w, H)
    q, s, hist = jarq.refine(W, Hm, np.array([[1, 2]], dtype=np.uint8),
                             np.array([[1.0]]), z, 2, 2, 2)
    assert list(q[0]) == [2, 3]
    assert abs(hist[0].L[0] - 1 / 104) < EPS
    assert abs(hist[0].F_after[0] - 109 / 270400) < EPS
    assert abs(s[0, 0] - 1.0) < EPS and hist[1].L[0] < EPS


# ---------------------------------------------------------------------------
# Proposition "Refitting the grid unlocks descent", App. G.3
# ---------------------------------------------------------------------------

def build_staleness():
    gv = _golden.load("prop_grid_staleness.txt")
    rho = float(gv["rho"])
    H = np.array([[1.0, rho], [rho, 1.0]])
    w = np.array([float(x) for x in gv["w"]])
    return gv, w, H


@pytest.fixture(scope="module")
def staleness():
    return build_staleness()


def test_staleness_host_is_box_optimal(staleness):
    gv, w, H = staleness
    W, Hm, z = _single_group(w, H)
    s0 = np.array([[float(gv["s0"])]])
    errs = {}
    for q in itertools.product(range(4), repeat=2):
        errs[q] = float(jarq.objective_rows(W, Hm, np.array([q], dtype=np.uint8), s0, z, 2)[0])
    order = sorted(errs, key=errs.get)
    assert order[0] == (1, 1)
    assert abs(errs[(1, 1)] - float(gv["f_s0_q0"])) < EPS
    assert order[1] == tuple(int(v) for v in gv["q_second"])
    assert abs(errs[order[1]] - float(gv["f_s0_second"])) < EPS


def test_staleness_babai_at_host_scale_keeps_host(staleness):
    gv, w, H = staleness
    W, Hm, z = _single_group(w, H)
    q0 = np.array([[1, 1]], dtype=np.uint8)
    s0 = np.array([[float(gv["s0"])]])
    qn, tr = jarq.code_step(W, Hm, jarq.group_factors(Hm, 2), q0, s0, z, 2, 2, record=True)
    assert abs(tr.x[0, 1] - float(gv["babai_s0_x2"])) < EPS
    assert abs(tr.x[0, 0] - float(gv["babai_s0_x1"])) < EPS
    assert list(qn[0]) == [1, 1] and tr.decision[0, 0] == jarq.DEC_REJECT


def test_staleness_full_trace(staleness):
    gv, w, H = staleness
    W, Hm, z = _single_group(w, H)
    q0 = np.array([[1, 1]], dtype=np.uint8)
    s_host = np.array([[float(gv["s0"])]])
    Rg = jarq.group_factors(Hm, 2)
    # iteration 1: refit, then Babai
    s1, _ = jarq.scale_step(W, Hm, q0, z, 2)
    assert abs(s1[0, 0] - float(gv["s1"])) < EPS
    assert abs(jarq.objective_rows(W, Hm, q0, s1, z, 2)[0] - float(gv["f_s1_q0"])) < EPS
    q1, tr = jarq.code_step(W, Hm, Rg, q0, s1, z, 2, 2, record=True)
    assert abs(tr.x[0, 1] - float(gv["babai_s1_x2"])) < EPS
    assert abs(tr.x[0, 0] - float(gv["babai_s1_x1"])) < EPS
    assert list(q1[0]) == [int(v) for v in gv["q_plus"]]
    assert abs(jarq.objective_rows(W, Hm, q1, s1, z, 2)[0] - float(gv["f_s1_qplus"])) < EPS
    # iteration 2: refit, Babai proposes q+ again -> fixed point
    q, s, hist = jarq.refine(W, Hm, q0, s_host, z, 2, 2, 3)
    assert list(q[0]) == [0, 2]
    assert abs(s[0, 0] - float(gv["s2"])) < EPS
    assert abs(hist[1].L[0] - float(gv["f_s2_qplus"])) < EPS
    assert hist[1].accepted == 0 and hist[2].accepted == 0
    # 75% reduction from the host state
    assert hist[-1].F_after[0] < 0.26 * float(gv["f_s0_q0"])


# ---------------------------------------------------------------------------
# Brute force over small boxes (eq. (8)); Babai is exact where it must be.
# ---------------------------------------------------------------------------

def _random_problem(rng, g, diag=False):
    X = rng.standard_normal((3 * g + 2, g)) @ (np.eye(g) + 0.6 * np.triu(rng.standard_normal((g, g)), 1))
    H = X.T @ X / X.shape[0] + 0.05 * np.eye(g)
    if diag:
        H = np.diag(np.diag(H))
    return H


def _box_optimum(W, H, s, z, g, bits):
    best, arg = np.inf, None
    for q in itertools.product(range(1 << bits), repeat=g):
        f = jarq.objective_rows(W, H, np.array([q], dtype=np.uint8), s, z, g)[0]
        if f < best:
            best, arg = f, q
    return best, arg


@pytest.mark.parametrize("g,bits,diag", [(1, 3, False), (1, 2, False), (2, 2, True),
                                         (3, 2, True), (4, 2, True), (2, 3, False),
                                         (3, 2, False), (4, 2, False), (3, 3, False)])
def test_babai_vs_bruteforce(g, bits, diag):
    rng = np.random.default_rng(100 * g + 10 * bits + diag)
    qmax = (1 << bits) - 1
    gaps = []
    for trial in range(25):
        H = _random_problem(rng, g, diag)
        z = np.array([[rng.integers(0, qmax + 1)]], dtype=np.int32)
        s = np.array([[rng.uniform(0.3, 1.2)]])
        # targets that reach past the box so clipping is exercised too
        w = s[0, 0] * (rng.uniform(-1.0, qmax + 1.0, size=g) - z[0, 0])
        W = w[None, :]
        q_start = np.array([rng.integers(0, qmax + 1, size=g)], dtype=np.uint8)
        Rg = jarq.group_factors(H, g)
        qn, tr = jarq.code_step(W, H, Rg, q_start, s, z, g, bits, record=True)
        f_babai = jarq.objective_rows(W, H, tr.cand.astype(np.uint8), s, z, g)[0]
        f_best, _ = _box_optimum(W, H, s, z, g, bits)
        f_start = jarq.objective_rows(W, H, q_start, s, z, g)[0]
        f_new = jarq.objective_rows(W, H, qn, s, z, g)[0]
        assert f_best <= f_babai + 1e-12
        assert f_new <= f_start + 1e-12          # accept test never increases F
        if g == 1 or diag:
            assert abs(f_babai - f_best) <= 1e-12 * max(1.0, f_best)
        gaps.append(f_babai - f_best)
    assert np.all(np.asarray(gaps) >= -1e-12)


# ---------------------------------------------------------------------------
# Scale step: closed forms and identities (eq. (6), App. G.1)
# ---------------------------------------------------------------------------

def build_tiny_layer():
    from synth import CONFIGS, make_weights, make_hessian, rtn_quantize
    cfg = CONFIGS[0]
    W = make_weights(cfg)
    H32, X, H64 = make_hessian(cfg, return_x=True)
    codes, scales, zeros = rtn_quantize(W, cfg.group_size, cfg.bits)
    n = X.shape[0]
    lam_d = H64[0, 0] - (X[:, 0] @ X[:, 0]) / n
    A = np.vstack([X / np.sqrt(n), np.sqrt(lam_d) * np.eye(cfg.cols)])
    return cfg, W, H32, H64, A, codes, scales, zeros


@pytest.fixture(scope="module")
def tiny_layer():
    return build_tiny_layer()


def test_scale_step_matches_lstsq(tiny_layer):
    cfg, W, H32, H64, A, codes, scales, zeros = tiny_layer
    g = cfg.group_size
    assert np.allclose(A.T @ A, H64, rtol=1e-12, atol=1e-12)
    s, ridge = jarq.scale_step(W, A.T @ A, codes, zeros, g)
    assert not ridge.any()
    c = jarq.code_offsets(codes, zeros, g)
    for j in range(W.shape[0]):
        B = np.stack([A[:, i * g:(i + 1) * g] @ c[j, i] for i in range(cfg.groups)], axis=1)
        s_ls, *_ = np.linalg.lstsq(B, A @ W[j].astype(np.float64), rcond=None)
        assert np.allclose(s[j], s_ls, rtol=1e-9, atol=1e-12)


def test_scale_step_newton_form(tiny_layer):
    cfg, W, H32, H64, A, codes, scales, zeros = tiny_layer
    g = cfg.group_size
    s, _ = jarq.scale_step(W, H32, codes, zeros, g)
    gram, _ = jarq.gram_system(W, H32, codes, zeros, g)
    E = W.astype(np.float64) - jarq.dequantize(codes, scales, zeros, g)
    He = E @ H32.astype(np.float64).T
    c = jarq.code_offsets(codes, zeros, g).reshape(W.shape[0], -1)
    BtHe = (c * He).reshape(W.shape[0], cfg.groups, g).sum(axis=2)
    s_newton = scales.astype(np.float64) + np.linalg.solve(gram, BtHe[:, :, None])[:, :, 0]
    assert np.allclose(s, s_newton, rtol=1e-9, atol=1e-12)


def test_joint_scale_gap_identity(tiny_layer):
    cfg, W, H32, H64, A, codes, scales, zeros = tiny_layer
    g = cfg.group_size
    s_star, _ = jarq.scale_step(W, H32, codes, zeros, g)
    gram, _ = jarq.gram_system(W, H32, codes, zeros, g)
    rng = np.random.default_rng(7)
    s_tilde = s_star * (1 + 0.1 * rng.standard_normal(s_star.shape))
    f_t = jarq.objective_rows(W, H32, codes, s_tilde, zeros, g)
    f_s = jarq.objective_rows(W, H32, codes, s_star, zeros, g)
    d = s_tilde - s_star
    quad = np.einsum("ji,jih,jh->j", d, gram, d)
    assert np.allclose(f_t - f_s, quad, rtol=1e-8, atol=1e-15)
    assert np.all(f_t >= f_s)


def test_block_diagonal_hessian_gives_independent_fits():
    rng = np.random.default_rng(3)
    g, G, rows = 8, 3, 5
    blocks = [_random_problem(rng, g) for _ in range(G)]
    H = np.zeros((g * G, g * G))
    for i, b in enumerate(blocks):
        H[i * g:(i + 1) * g, i * g:(i + 1) * g] = b
    W = 0.1 * rng.standard_normal((rows, g * G))
    from synth import rtn_quantize
    codes, scales, zeros = rtn_quantize(W, g, 3)
    s, _ = jarq.scale_step(W, H, codes, zeros, g)
    c = jarq.code_offsets(codes, zeros, g)
    for j in range(rows):
        for i in range(G):
            Hi = blocks[i]
            ci, wi = c[j, i], W[j, i * g:(i + 1) * g]
            s_ind = (ci @ Hi @ wi) / (ci @ Hi @ ci)      # eq. (independent-fit)
            assert abs(s[j, i] - s_ind) <= 1e-10 * abs(s_ind) + 1e-14


def test_ridge_branch_on_singular_gram():
    """A group whose codes all equal its zero point makes B_j rank deficient."""
    rng = np.random.default_rng(11)
    g, G = 4, 3
    H = _random_problem(rng, g * G)
    W = 0.1 * rng.standard_normal((2, g * G))
    from synth import rtn_quantize
    codes, scales, zeros = rtn_quantize(W, g, 3)
    codes[0, g:2 * g] = zeros[0, 1]
    s, ridge = jarq.scale_step(W, H, codes, zeros, g)
    assert ridge[0] and not ridge[1]
    assert s[0, 1] == 0.0
    gram, rhs = jarq.gram_system(W, H, codes, zeros, g)
    expect = np.linalg.solve(gram[0] + 1e-4 * np.eye(G), rhs[0])
    assert np.allclose(s[0], expect, rtol=1e-10)


def kahan_gram(G):
    """R^T R with R unit upper triangular, -1 above the diagonal.

    Its Cholesky factor is R^T itself, so every pivot is exactly 1, while
    sigma_min(R) falls like 2^-G: from G = 16 on its smallest eigenvalue is
    below 1e-10 of its largest.  A trigger that looked only at the pivots
    would never fire on it."""
    R = np.eye(G) + np.triu(-np.ones((G, G)), 1)
    return R.T @ R


def test_ridge_trigger_is_the_spectrum_not_the_pivots():
    """App. E.2 tests the smallest eigenvalue, not the factorisation's pivots."""
    G = 20
    Gt = kahan_gram(G)
    assert np.array_equal(np.diag(np.linalg.cholesky(Gt)), np.ones(G))   # every pivot is 1
    ev = np.linalg.eigvalsh(Gt)
    assert ev[0] <= jarq.RIDGE_RCOND * ev[-1]
    rhs = np.arange(1.0, G + 1.0)
    s, ridge = jarq.solve_scales(Gt[None], rhs[None])
    assert ridge[0]
    expect = np.linalg.solve(Gt + jarq.RIDGE_LAMBDA * np.eye(G), rhs)
    assert np.allclose(s[0], expect, rtol=1e-8)
    # a well-conditioned neighbour is solved exactly
    s2, ridge2 = jarq.solve_scales((Gt + np.eye(G))[None], rhs[None])
    assert not ridge2[0]
    assert np.allclose(s2[0], np.linalg.solve(Gt + np.eye(G), rhs), rtol=1e-10)


def _ridge_worse_layer(h_scale=1e-8, seed=23):
    """A layer whose row 0 takes the ridge branch (one group at its zero point,
    so B_0 is rank deficient).  With H scaled by 1e-8, lambda = 1e-4 dominates
    the Gram entries (largest eigenvalue ~ 4e-6): the ridge solution shrinks
    every scale toward zero and raises F_0 above the host's."""
    rng = np.random.default_rng(seed)
    g, G = 4, 3
    H = h_scale * _random_problem(rng, g * G)
    W = 0.1 * rng.standard_normal((3, g * G))
    from synth import rtn_quantize
    codes, scales, zeros = rtn_quantize(W, g, 3)
    codes[0, g:2 * g] = zeros[0, 1]
    return W, H, codes, scales.astype(np.float64), zeros, g


def test_scale_objective_change_matches_the_objective():
    """F(s_new) - F(s_old) from the Gram system equals the objective eq. (4) evaluated directly."""
    rng = np.random.default_rng(29)
    g, G = 4, 3
    H = _random_problem(rng, g * G)
    W = 0.1 * rng.standard_normal((5, g * G))
    from synth import rtn_quantize
    codes, scales, zeros = rtn_quantize(W, g, 3)
    gram, rhs = jarq.gram_system(W, H, codes, zeros, g)
    s_old = scales.astype(np.float64)
    s_new = s_old * (1.0 + 0.3 * rng.standard_normal(s_old.shape))
    got = jarq.scale_objective_change(gram, rhs, s_new, s_old)
    want = (jarq.objective_rows(W, H, codes, s_new, zeros, g)
            - jarq.objective_rows(W, H, codes, s_old, zeros, g))
    assert np.allclose(got, want, rtol=1e-9, atol=1e-14)


def test_ridge_acceptance_keeps_previous_scales_when_worse():
    """Remark of App. G.5: a ridge solution that raises F_j is not kept."""
    W, H, codes, s_prev, zeros, g = _ridge_worse_layer()
    s_plain, ridge = jarq.scale_step(W, H, codes, zeros, g)
    assert ridge[0] and not ridge[1:].any()
    F = lambda s: jarq.objective_rows(W, H, codes, s, zeros, g)
    assert F(s_plain)[0] > F(s_prev)[0]                 # the failure the remark describes
    s_acc, ridge_acc = jarq.scale_step(W, H, codes, zeros, g, prev=s_prev)
    assert np.array_equal(ridge_acc, ridge)
    assert np.array_equal(s_acc[0], s_prev[0])          # previous scales retained
    assert np.array_equal(s_acc[1:], s_plain[1:])       # ordinary solves untouched
    assert np.all(F(s_acc) <= F(s_prev) * (1 + 1e-12))


def test_ridge_acceptance_keeps_a_better_ridge_solution():
    """On the unscaled problem the ridge solution of the same row lowers F and is kept."""
    W, H, codes, s_prev, zeros, g = _ridge_worse_layer(h_scale=1.0)
    s_plain, ridge = jarq.scale_step(W, H, codes, zeros, g)
    F = lambda s: jarq.objective_rows(W, H, codes, s, zeros, g)
    assert ridge[0] and F(s_plain)[0] < F(s_prev)[0]
    s_acc, _ = jarq.scale_step(W, H, codes, zeros, g, prev=s_prev)
    assert np.array_equal(s_acc, s_plain)


def test_ridge_acceptance_makes_the_objective_monotone():
    """With ridge acceptance L_j^(k) (after each scale update) never increases (Thm. 1 (i))."""
    W, H, codes, s_prev, zeros, g = _ridge_worse_layer()
    F0 = jarq.objective_rows(W, H, codes, s_prev, zeros, g)
    _, _, hist = jarq.refine(W, H, codes, s_prev, zeros, g, 3, 4, ridge_accept=True)
    L = np.stack([h.L for h in hist])
    assert np.all(L[0] <= F0 * (1 + 1e-12))
    assert np.all(np.diff(L, axis=0) <= 1e-12 * np.abs(L[:-1]))
    _, _, hist_plain = jarq.refine(W, H, codes, s_prev, zeros, g, 3, 1)
    assert hist_plain[0].L[0] > F0[0]                   # without it the first update goes up


def test_ridge_second_failure_raises():
    """A nonfinite coupling block makes the Gram matrix nonfinite: ridge, then failure."""
    g = 2
    H = np.eye(4)
    H[0, 2] = H[2, 0] = np.nan
    W = np.array([[0.5, 1.0, 2.0, 3.0]])
    codes = np.array([[1, 2, 3, 1]], dtype=np.uint8)
    zeros = np.zeros((1, 2), dtype=np.int32)
    jarq.group_factors(H, g)                     # diagonal blocks are fine
    with pytest.raises(jarq.ScaleSolveError):
        jarq.scale_step(W, H, codes, zeros, g)


def test_nonfinite_weights_give_nonfinite_scales_and_skipped_groups():
    """NaN in w leaves the Gram finite; the scales become NaN and no proposal is made."""
    g = 2
    H = np.eye(4) + 0.1
    W = np.array([[np.nan, 1.0, 2.0, 3.0]])
    codes = np.array([[1, 2, 3, 1]], dtype=np.uint8)
    zeros = np.zeros((1, 2), dtype=np.int32)
    s, ridge = jarq.scale_step(W, H, codes, zeros, g)
    assert not ridge.any() and np.all(np.isnan(s))
    qn, tr = jarq.code_step(W, H, jarq.group_factors(H, g), codes, s, zeros, g, 2, record=True)
    assert np.array_equal(qn, codes) and np.all(tr.decision == jarq.DEC_SKIP)


def test_not_spd_block_raises():
    H = np.eye(4)
    H[2, 2] = -1.0
    with pytest.raises(jarq.NotSPDError):
        jarq.group_factors(H, 2)


# ---------------------------------------------------------------------------
# QR form (paper notation) == Hessian form (App. E.1) on the tiny layer
# ---------------------------------------------------------------------------

def test_qr_form_equals_hessian_form(tiny_layer):
    cfg, W, H32, H64, A, codes, scales, zeros = tiny_layer
    g, bits, K = cfg.group_size, cfg.bits, cfg.sweeps
    Hh = A.T @ A
    qh, sh, hist = jarq.refine(W, Hh, codes, scales, zeros, g, bits, K)
    for j in range(0, W.shape[0], 4):
        qq, sq, hq = qrform.refine_row(A, W[j], codes[j], scales[j], zeros[j], g, bits, K)
        assert np.array_equal(qq, qh[j]), j
        assert np.allclose(sq, sh[j], rtol=1e-9, atol=1e-12)
        for k in range(K):
            assert abs(hq[k][0] - hist[k].L[j]) <= 1e-9 * hist[k].L[j]
            assert abs(hq[k][1] - hist[k].F_after[j]) <= 1e-9 * hist[k].F_after[j]


# ---------------------------------------------------------------------------
# Invariants: Theorem 1, Corollary 1, K = 0, fixed points, App. G.4 / G.6
# ---------------------------------------------------------------------------

def test_monotone_descent_and_host_bound(tiny_layer):
    cfg, W, H32, H64, A, codes, scales, zeros = tiny_layer
    g = cfg.group_size
    F_host = jarq.objective_rows(W, H32, codes, scales, zeros, g)
    q, s, hist = jarq.refine(W, H32, codes, scales, zeros, g, cfg.bits, 8)
    prev = F_host
    for h in hist:
        assert not h.ridge.any()
        assert np.all(h.L <= prev * (1 + 1e-12) + 1e-300)
        assert np.all(h.F_after <= h.L * (1 + 1e-12) + 1e-300)
        prev = h.F_after
    assert np.all(jarq.objective_rows(W, H32, q, s, zeros, g) <= F_host)
    assert hist[0].accepted > 0


def test_zero_budget_returns_host(tiny_layer):
    cfg, W, H32, H64, A, codes, scales, zeros = tiny_layer
    q, s, hist = jarq.refine(W, H32, codes, scales, zeros, cfg.group_size, cfg.bits, 0)
    assert np.array_equal(q, codes) and np.array_equal(s, scales.astype(np.float64))
    assert hist == []


def test_fixed_point_after_a_sweep_without_accepts(tiny_layer):
    cfg, W, H32, H64, A, codes, scales, zeros = tiny_layer
    g = cfg.group_size
    q, s, hist = jarq.refine(W, H32, codes, scales, zeros, g, cfg.bits, 30)
    quiet = [k for k, h in enumerate(hist) if h.accepted == 0]
    assert quiet, "no sweep without accepts within 30 iterations"
    k = quiet[0]
    q2, s2, h2 = jarq.refine(W, H32, codes, scales, zeros, g, cfg.bits, k + 1)
    q3, s3, h3 = jarq.refine(W, H32, q2, s2, zeros, g, cfg.bits, 1)
    assert np.array_equal(q3, q2)
    assert np.allclose(s3, s2, rtol=1e-10, atol=0)
    assert h3[0].accepted == 0


def test_resume_equals_uninterrupted(tiny_layer):
    cfg, W, H32, H64, A, codes, scales, zeros = tiny_layer
    g = cfg.group_size
    qa, sa, _ = jarq.refine(W, H32, codes, scales, zeros, g, cfg.bits, 4)
    q1, s1, _ = jarq.refine(W, H32, codes, scales, zeros, g, cfg.bits, 2)
    qb, sb, _ = jarq.refine(W, H32, q1, s1, zeros, g, cfg.bits, 2)
    assert np.array_equal(qa, qb) and np.array_equal(sa, sb)


def test_unclipped_babai_residual_bound(tiny_layer):
    """App. G.4 (a): |(v - R(q^B - z))_l| <= |R_ll| / 2 when nothing clips."""
    cfg, W, H32, H64, A, codes, scales, zeros = tiny_layer
    g, bits = cfg.group_size, cfg.bits
    qmax = (1 << bits) - 1
    H = H32.astype(np.float64)
    Rg = jarq.group_factors(H, g)
    s, _ = jarq.scale_step(W, H, codes, zeros, g)
    _, tr = jarq.code_step(W, H, Rg, codes, s, zeros, g, bits, record=True)
    checked = 0
    q_cur = codes.astype(np.int64).copy()
    for i in range(cfg.groups):
        blk = slice(i * g, (i + 1) * g)
        unclipped = np.all((np.rint(tr.x[:, blk]) >= 0) & (np.rint(tr.x[:, blk]) <= qmax), axis=1)
        what = jarq.dequantize(q_cur, s, zeros, g)
        what[:, blk] = 0
        aty = (W - what) @ H[blk, :].T
        v = np.linalg.solve(Rg[i].T, aty.T).T / s[:, i:i + 1]
        r = v - (tr.cand[:, blk].astype(np.float64) - zeros[:, i:i + 1]) @ Rg[i].T
        bound = np.abs(np.diag(Rg[i])) / 2
        assert np.all(np.abs(r[unclipped]) <= bound[None, :] * (1 + 1e-9) + 1e-12)
        checked += int(unclipped.sum())
        acc = tr.decision[:, i] == jarq.DEC_ACCEPT
        q_cur[acc, blk] = tr.cand[acc, blk]
    assert checked > 0


def test_stable_point_quality_bound(tiny_layer):
    """App. G.6: at a scale-optimal, Babai-stable point each unclipped group is
    within s^2/4 sum R_ll^2 of its best real-valued fit."""
    cfg, W, H32, H64, A, codes, scales, zeros = tiny_layer
    g, bits = cfg.group_size, cfg.bits
    qmax = (1 << bits) - 1
    H = H32.astype(np.float64)
    Rg = jarq.group_factors(H, g)
    q, s, hist = jarq.refine(W, H, codes, scales, zeros, g, bits, 40)
    assert hist[-1].accepted == 0
    s, _ = jarq.scale_step(W, H, q, zeros, g)
    _, tr = jarq.code_step(W, H, Rg, q, s, zeros, g, bits, record=True)
    checked = 0
    for i in range(cfg.groups):
        blk = slice(i * g, (i + 1) * g)
        unclipped = np.all((np.rint(tr.x[:, blk]) >= 0) & (np.rint(tr.x[:, blk]) <= qmax), axis=1)
        what = jarq.dequantize(q, s, zeros, g)
        E = W - what
        he = E @ H[blk, :].T
        u = np.linalg.solve(Rg[i].T, he.T).T          # R^{-T} (H e)_i
        # group error above the best real fit = ||R^{-T}(H e)_i||^2 (reduced form)
        excess = np.sum(u * u, axis=1)
        bound = s[:, i] ** 2 / 4 * np.sum(np.diag(Rg[i]) ** 2)
        ok = excess <= bound * (1 + 1e-9) + 1e-15
        assert np.all(ok[unclipped])
        checked += int(unclipped.sum())
    assert checked > 0


def test_early_stopping_freezes_rows(tiny_layer):
    cfg, W, H32, H64, A, codes, scales, zeros = tiny_layer
    g = cfg.group_size
    q, s, hist = jarq.refine(W, H32, codes, scales, zeros, g, cfg.bits, 10, tau=1e-5)
    stopped = ~hist[-1].active
    assert stopped.any()
    for h in hist:
        assert np.all(np.isnan(h.F_after[~h.active]))


def test_code_step_two_forms_agree(tiny_layer):
    """The reduced-norm change equals delta^T H_ii delta - 2 delta^T (H e)_i."""
    cfg, W, H32, H64, A, codes, scales, zeros = tiny_layer
    g, bits = cfg.group_size, cfg.bits
    H = H32.astype(np.float64)
    Rg = jarq.group_factors(H, g)
    s, _ = jarq.scale_step(W, H, codes, zeros, g)
    q_cur = codes.astype(np.int64).copy()
    _, tr = jarq.code_step(W, H, Rg, codes, s, zeros, g, bits, record=True)
    for i in range(cfg.groups):
        blk = slice(i * g, (i + 1) * g)
        E = W - jarq.dequantize(q_cur, s, zeros, g)
        he = E @ H[blk, :].T
        delta = s[:, i:i + 1] * (tr.cand[:, blk].astype(np.float64) - q_cur[:, blk])
        dF = np.einsum("rg,gh,rh->r", delta, H[blk, blk], delta) - 2 * np.einsum("rg,rg->r", delta, he)
        scale = np.abs(tr.err_old[:, i]) + np.abs(tr.err_new[:, i]) + 1e-30
        assert np.all(np.abs(dF - (tr.err_new[:, i] - tr.err_old[:, i])) <= 1e-9 * scale)
        acc = tr.decision[:, i] == jarq.DEC_ACCEPT
        q_cur[acc, blk] = tr.cand[acc, blk]


# ---------------------------------------------------------------------------
# Early stopping, eq. (strict_stopping) of App. E.2
# ---------------------------------------------------------------------------
#
# The stopping rule is pinned on hand-built objective sequences: the scale
# step, the objective and the code step are replaced by scripted stand-ins so
# that L_j^(k) (the objective right after the scale update of iteration k)
# follows a table chosen per row, and refine() decides when each row stops.
# tau = 2^-16 keeps every quotient below exact.

STOP_TAU_EXACT = 2.0 ** -16
_BIG = 2.0 ** 20
# rows x (host, k = 1..4); the host column is what a row's objective is at
# the host state (the scripted objective of scales marked 0)
STOP_TABLE = np.array([
    [2 * _BIG, _BIG, _BIG - 16.0, _BIG - 8.0, _BIG - 4.0],      # relative decrease exactly tau at k = 2
    [2 * _BIG, _BIG, _BIG - 32.0, _BIG - 64.0, _BIG - 96.0],    # relative decrease 2 tau: never stops
    [2.0 ** -9, 2.0 ** -10, 2.0 ** -10 - STOP_TAU_EXACT, 0.0, 0.0],  # absolute decrease exactly tau at k = 2
    [4.0, 1.0, 1.5, 1.0, 0.5],                                  # the objective went up at k = 2
    [_BIG, _BIG, _BIG / 2, _BIG / 4, _BIG / 8],                 # no decrease at k = 1: k = 1 never stops
    [8.0, 4.0, 2.0, 1.0, 1.0 - 2.0 ** -20],                     # stops at k = 4 on L^(3) - L^(4)
    [3 * _BIG, 3 * _BIG / 4, 3 * _BIG / 4 - 12.0, 0.0, 0.0],    # relative exactly tau of L^(k-1) (not of L^(k))
])
STOP_EXPECT = [2, None, 2, 2, None, 4, 2]     # iteration at which each row stops (None: never)


class _Scripted:
    """Scripted scale step, objective and code step for refine().

    Row r of W carries r in column 0.  The scale step of iteration k (its k-th
    call) returns scales equal to k; the objective returns STOP_TABLE[r, k] for scales equal
    to k (k = 0 is the host); the code step writes k into column 1 of the codes
    of the rows it updates.
    """

    def __init__(self, table):
        self.table = table
        self.k = 0
        self.saved = {}

    def scale_step(self, W, H, codes, zeros, g, lam=None, rcond=None, prev=None):
        self.k += 1
        return np.full((W.shape[0], zeros.shape[1]), float(self.k)), np.zeros(W.shape[0], bool)

    def objective_rows(self, W, H, codes, scales, zeros, g):
        r = np.asarray(W[:, 0], dtype=np.int64)
        k = np.asarray(scales[:, 0], dtype=np.int64)
        return self.table[r, k].astype(np.float64)

    def code_step(self, W, H, R, codes, scales, zeros, g, bits, record=False):
        q = np.asarray(codes).copy()
        q[:, 1] = np.asarray(scales[:, 0], dtype=np.uint8)
        G = zeros.shape[1]
        tr = jarq.CodeTrace(None, None, np.full((q.shape[0], G), jarq.DEC_REJECT, np.uint8), None, None)
        return (q, tr) if record else q

    def __enter__(self):
        for name in ("scale_step", "objective_rows", "code_step"):
            self.saved[name] = getattr(jarq, name)
            setattr(jarq, name, getattr(self, name))
        return self

    def __exit__(self, *exc):
        for name, fn in self.saved.items():
            setattr(jarq, name, fn)
        return False


def _run_scripted(table, K, tau):
    rows = table.shape[0]
    W = np.zeros((rows, 4))
    W[:, 0] = np.arange(rows)
    codes = np.zeros((rows, 4), dtype=np.uint8)
    scales = np.zeros((rows, 2))
    zeros = np.zeros((rows, 2), dtype=np.int32)
    with _Scripted(table):
        q, s, hist = jarq.refine(W, np.eye(4), codes, scales, zeros, 2, 3, K, tau=tau,
                                 R=np.zeros((2, 2, 2)))
    return q, s, hist


def stopping_sweeps(hist, rows):
    """Iteration at which each row stopped (None if it never did)."""
    out = [None] * rows
    was = np.ones(rows, dtype=bool)
    for k, h in enumerate(hist, start=1):
        for r in np.nonzero(was & ~h.active)[0]:
            out[r] = k
        was = h.active.copy()
    return out


def test_stopping_rule_on_hand_built_sequences():
    q, s, hist = _run_scripted(STOP_TABLE, 4, STOP_TAU_EXACT)
    assert stopping_sweeps(hist, STOP_TABLE.shape[0]) == STOP_EXPECT
    for r, k_stop in enumerate(STOP_EXPECT):
        k_last = 4 if k_stop is None else k_stop
        # a stopped row keeps the scales of the iteration that stopped it and
        # the codes of the iteration before (its code update is skipped)
        assert np.all(s[r] == k_last), (r, s[r])
        assert q[r, 1] == (4 if k_stop is None else k_stop - 1), (r, q[r])


def test_stopping_rule_active_counts():
    _, _, hist = _run_scripted(STOP_TABLE, 4, STOP_TAU_EXACT)
    expect = [sum(1 for e in STOP_EXPECT if e is None or e > k) for k in range(1, 5)]
    assert [int(h.active.sum()) for h in hist] == expect == [7, 3, 3, 2]


def test_stop_rows_branches():
    t = STOP_TAU_EXACT
    # relative branch at exactly tau, and just above it (absolute branch silent)
    assert jarq.stop_rows([_BIG], [_BIG - 16.0], t)[0]
    assert not jarq.stop_rows([_BIG], [_BIG - 17.0], t)[0]
    # absolute branch at exactly tau, relative decrease large
    assert jarq.stop_rows([2.0 ** -10], [2.0 ** -10 - t], t)[0]
    assert not jarq.stop_rows([2.0 ** -10], [2.0 ** -10 - 2 * t], t)[0]
    # an increase stops; tau = 0 stops exactly on no decrease
    assert jarq.stop_rows([1.0], [1.25], t)[0]
    assert jarq.stop_rows([1.0], [1.0], 0.0)[0]
    assert not jarq.stop_rows([1.0], [1.0 - 2.0 ** -40], 0.0)[0]


def test_row_without_accepts_stops_at_the_next_iteration(tiny_layer):
    """After an iteration that changes no code, L^(k) = L^(k-1) and the rule
    stops the row (the remark after the proof of Theorem 1); with tau = 0 a
    row stops exactly then, since every accepted proposal lowers F strictly."""
    cfg, W, H32, H64, A, codes, scales, zeros = tiny_layer
    g, bits, K = cfg.group_size, cfg.bits, 8
    H = H32.astype(np.float64)
    R = jarq.group_factors(H, g)
    # the changes of every sweep without stopping
    q, s = codes.copy(), scales.copy()
    first_idle = [None] * cfg.rows
    for k in range(1, K + 1):
        s, _ = jarq.scale_step(W, H, q, zeros, g)
        q_new = jarq.code_step(W, H, R, q, s, zeros, g, bits)
        idle = np.all(q_new == q, axis=1)
        for r in np.nonzero(idle)[0]:
            if first_idle[r] is None:
                first_idle[r] = k
        q = q_new
    _, _, hist = jarq.refine(W, H, codes, scales, zeros, g, bits, K, tau=0.0, R=R)
    got = stopping_sweeps(hist, cfg.rows)
    expect = [None if f is None or f + 1 > K else f + 1 for f in first_idle]
    assert any(e is not None for e in expect)
    assert got == expect
