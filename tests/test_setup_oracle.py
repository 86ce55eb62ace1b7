"""Pins of the per-layer set-up oracles (CPU): the calibration Hessian and the
round-to-nearest host."""

import numpy as np

from oracle import hessian, hosts, post, qep
from synth import CONFIGS, make_hessian, rtn_quantize


# --------------------------------------------------------------------------
# Hessian H = X~^T X~ + nu^2 I (App. E.1)
# --------------------------------------------------------------------------

def test_hessian_is_the_sum_of_token_outer_products():
    rng = np.random.default_rng(3)
    X = rng.standard_normal((7, 5))
    brute = np.zeros((5, 5))
    for t in range(7):
        for a in range(5):
            for b in range(5):
                brute[a, b] += 0.25 * X[t, a] * X[t, b]
    H = hessian.hessian([X], 5, alpha=0.25)
    assert np.allclose(H, brute, rtol=0, atol=1e-14)


def test_hessian_is_the_gram_matrix_of_the_stacked_design():
    # A = [X~; nu I] with X~ = sqrt(alpha) X: H = A^T A
    rng = np.random.default_rng(4)
    X = rng.standard_normal((40, 12))
    alpha, nu = 1.0 / 40, 0.6
    A = np.vstack([np.sqrt(alpha) * X, nu * np.eye(12)])
    H = hessian.hessian([X], 12, alpha=alpha, nu2=nu * nu)
    assert np.allclose(H, A.T @ A, rtol=1e-13, atol=1e-14)
    assert np.all(np.linalg.eigvalsh(H) >= nu * nu * (1 - 1e-12))


def test_hessian_does_not_depend_on_chunking():
    rng = np.random.default_rng(5)
    X = rng.standard_normal((333, 20))
    whole = hessian.hessian([X], 20, alpha=1 / 333, damp=0.01)
    parts = hessian.hessian([X[:1], X[1:100], X[100:]], 20, alpha=1 / 333, damp=0.01)
    assert np.allclose(whole, parts, rtol=1e-13, atol=1e-15)
    assert np.array_equal(parts, parts.T)


def test_hessian_damping_adds_the_stated_diagonal():
    rng = np.random.default_rng(6)
    X = rng.standard_normal((50, 8)) * np.arange(1, 9)
    base = hessian.hessian([X], 8)
    H = hessian.hessian([X], 8, damp=0.01, nu2=0.36)
    add = 0.01 * np.trace(X.T @ X) / 8 + 0.36
    assert np.allclose(np.diag(H) - np.diag(base), add, rtol=1e-14)
    off = ~np.eye(8, dtype=bool)
    assert np.array_equal(H[off], base[off])
    assert np.isclose(np.trace(base), np.sum(X * X), rtol=1e-14)


def test_hessian_reproduces_the_tiny_synthetic_layer():
    cfg = CONFIGS[0]
    _, X, H64 = make_hessian(cfg, return_x=True)
    H = hessian.hessian([X[:200], X[200:]], cfg.cols, alpha=1 / X.shape[0], damp=cfg.damping)
    assert np.allclose(H, H64, rtol=1e-12, atol=1e-14)


def test_fp32_error_bound_covers_a_simulated_fp32_path():
    # products rounded to fp32, fp32 sums of 256, fp64 sum of the partials
    rng = np.random.default_rng(7)
    m = 1500
    x = (rng.standard_normal((m, 2)) * [1.0, 30.0]).astype(np.float32)
    exact = float(np.dot(x[:, 0].astype(np.float64), x[:, 1].astype(np.float64)))
    prods = (x[:, 0] * x[:, 1]).astype(np.float32)
    tot = 0.0
    for s0 in range(0, m, 256):
        acc = np.float32(0)
        for p in prods[s0:s0 + 256]:
            acc = np.float32(acc + p)
        tot += float(acc)
    absg = float(np.dot(np.abs(x[:, 0]).astype(np.float64), np.abs(x[:, 1]).astype(np.float64)))
    assert abs(tot - exact) <= hessian.fp32_error_bound(absg, 1.0)
    # the bound is not vacuous: it is far below the size of the terms
    assert hessian.fp32_error_bound(absg, 1.0) < 1e-4 * absg


# --------------------------------------------------------------------------
# Round-to-nearest host (App. A.1, min/max reading)
# --------------------------------------------------------------------------

def test_rtn_worked_examples():
    # b = 2 (codes 0..3), one group of four per row, values worked by hand:
    # [-1, 0, 0.5, 2]: lo = -1, hi = 2, s = 1, z = 1, q = rint(w) + 1 (0.5 -> 0, half to even)
    # [0.25, 0.5, 0.75, 1]: lo = 0, hi = 1, s = fp32(1/3) = 0.3333333432674408, z = 0,
    #   w / s = 0.74999998, 1.49999996, 2.24999993, 2.99999991 -> 1, 1, 2, 3
    # [0, 0, 0, 0]: hi == lo, s = 1, z = 0, q = 0
    # [-3, -1, -2, -0.5]: lo = -3, hi = 0, s = 1, z = 3, q = rint(w) + 3 (-0.5 -> -0 -> 3)
    W = np.array([[-1, 0, 0.5, 2], [0.25, 0.5, 0.75, 1], [0, 0, 0, 0], [-3, -1, -2, -0.5]],
                 dtype=np.float32)
    q, s, z = hosts.rtn_host(W, 4, 2)
    assert q.tolist() == [[0, 1, 1, 3], [1, 1, 2, 3], [0, 0, 0, 0], [0, 2, 1, 3]]
    assert s[:, 0].tolist() == [1.0, np.float32(1 / 3), 1.0, 1.0]
    assert z[:, 0].tolist() == [1, 0, 0, 3]


def test_rtn_oracle_equals_the_host_generator():
    # two independent writings of the same rule agree bit for bit
    rng = np.random.default_rng(8)
    W = (0.02 * rng.standard_t(5, size=(33, 384))).astype(np.float32)
    W[0, :32] = 0.0
    W[1, 32:64] = np.abs(W[1, 32:64])
    W[2, 64:96] = -np.abs(W[2, 64:96])
    for g in (32, 64, 128):
        for bits in (1, 2, 3, 4, 8):
            a = hosts.rtn_host(W, g, bits)
            b = rtn_quantize(W, g, bits)
            for x, y in zip(a, b):
                assert x.dtype == y.dtype and np.array_equal(x, y), (g, bits)


def test_rtn_error_is_at_most_half_a_step_inside_the_range():
    rng = np.random.default_rng(9)
    W = (0.03 * rng.standard_normal((20, 256))).astype(np.float32)
    W[:, 5] = 0.0
    q, s, z = hosts.rtn_host(W, 64, 3)
    s64 = np.repeat(s.astype(np.float64), 64, axis=1)
    z64 = np.repeat(z.astype(np.float64), 64, axis=1)
    err = np.abs(W - s64 * (q - z64))
    assert np.all(err <= s64 / 2 * (1 + 1e-6) + 1e-12)
    # 0 lies in every group's range, so a weight of 0 gets the zero point's
    # code and is represented exactly
    assert np.array_equal(q[:, 5].astype(np.int64), z[:, 0].astype(np.int64))


def test_calibration_chunks_form_the_synthetic_hessian():
    # the streamed activations (outlier channels scaled) give make_hessian's H
    import torch
    from synth import calibration_chunks
    cfg = CONFIGS[1]
    n = 1024
    chunks = [c.numpy() for c in calibration_chunks(cfg, device="cpu", n_tokens=n, chunk=300)]
    assert sum(c.shape[0] for c in chunks) == n and chunks[0].shape[1] == cfg.cols
    H = hessian.hessian(chunks, cfg.cols, alpha=1 / n, damp=cfg.damping)
    H32 = make_hessian(cfg, device="cpu", n_tokens=n, chunk=300)
    assert np.max(np.abs(H.astype(np.float32) - H32)) <= 1e-6 * np.max(np.abs(H))
    del torch


# --------------------------------------------------------------------------
# GPTQ-style host (App. A.1 host; its recursion is the nearest-plane relation
# of App. G.7)
# --------------------------------------------------------------------------

def test_gptq_two_columns_follow_the_optimal_brain_surgeon_update():
    # One group of two columns: the grid comes from both raw weights; column 0
    # is rounded as is; column 1 is rounded from the value that minimises the
    # objective once column 0 is fixed, w_1 + (H_01 / H_11) e_0 (set the
    # derivative of e^T H e in e_1 to zero).
    rng = np.random.default_rng(12)
    for _ in range(50):
        w = rng.standard_normal((1, 2)).astype(np.float32)
        B = rng.standard_normal((2, 2))
        H = B @ B.T + 0.1 * np.eye(2)
        q, s, z = hosts.gptq_host(w, H, 2, 3)
        qmax = 7
        w64 = w.astype(np.float64)
        lo, hi = min(w64.min(), 0.0), max(w64.max(), 0.0)
        s0 = np.float64(np.float32((hi - lo) / qmax))
        z0 = np.clip(np.rint(-lo / s0), 0, qmax)
        q0 = np.clip(np.rint(w64[0, 0] / s0) + z0, 0, qmax)
        e0 = w64[0, 0] - s0 * (q0 - z0)
        x1 = w64[0, 1] + H[0, 1] / H[1, 1] * e0
        q1 = np.clip(np.rint(x1 / s0) + z0, 0, qmax)
        assert s[0, 0] == np.float32(s0) and z[0, 0] == z0
        assert q[0].tolist() == [q0, q1]


def test_gptq_with_a_diagonal_hessian_is_rtn():
    rng = np.random.default_rng(13)
    W = (0.02 * rng.standard_normal((9, 192))).astype(np.float32)
    H = np.diag(rng.uniform(0.5, 3.0, 192))
    for x, y in zip(hosts.gptq_host(W, H, 64, 3), hosts.rtn_host(W, 64, 3)):
        assert np.array_equal(x, y)


def _gptq_lower_factor_form(W, H, g, bits):
    """The recursion with M lower, M^T M = H (M = J C^T J, J H J = C C^T), no
    inverse: group grids from w_G + M_GG^{-1} M_GP e_P, columns rounded from
    w_k + (sum_{i<k} M_ki e_i) / M_kk (the formulation of the GPU host)."""
    W = np.asarray(W, np.float64)
    rows, d = W.shape
    qmax = (1 << bits) - 1
    J = np.arange(d)[::-1]
    C = np.linalg.cholesky(np.asarray(H, np.float64)[np.ix_(J, J)])
    M = C.T[np.ix_(J, J)]
    E = np.zeros_like(W)
    q = np.zeros((rows, d), np.uint8)
    for b0 in range(0, d, g):
        b1 = b0 + g
        c = E[:, :b0] @ M[b0:b1, :b0].T
        y = np.linalg.solve(M[b0:b1, b0:b1], c.T).T
        lo = np.minimum((W[:, b0:b1] + y).min(axis=1), 0.0)
        hi = np.maximum((W[:, b0:b1] + y).max(axis=1), 0.0)
        s = np.where(hi > lo, (hi - lo) / qmax, 1.0).astype(np.float32).astype(np.float64)
        z = np.clip(np.rint(-lo / s), 0, qmax)
        for k in range(b0, b1):
            x = W[:, k] + (E[:, :k] @ M[k, :k]) / M[k, k]
            qk = np.clip(np.rint(x / s) + z, 0, qmax)
            q[:, k] = qk
            E[:, k] = W[:, k] - s * (qk - z)
    return q


def test_gptq_lower_factor_form_equals_the_inverse_factor_recursion():
    cfg = CONFIGS[0]
    from synth import make_weights
    W = make_weights(cfg)
    H = make_hessian(cfg)
    q_ref, _, _, pre, _ = hosts.gptq_host(W, H, cfg.group_size, cfg.bits, return_pre=True)
    q = _gptq_lower_factor_form(W, H, cfg.group_size, cfg.bits)
    differ = q != q_ref
    near = np.abs(pre - np.floor(pre) - 0.5) < 1e-6
    assert np.all(near[differ]) and differ.mean() <= 1e-3


# --------------------------------------------------------------------------
# Propagation-corrected target (App. E.5)
# --------------------------------------------------------------------------

def _qep_problem(seed, n=60, d=10, dout=7, nu=0.6):
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((n, d))
    Xq = X + 0.1 * rng.standard_normal((n, d))
    W = rng.standard_normal((dout, d))              # rows = output channels
    H = Xq.T @ Xq + nu * nu * np.eye(d)
    D = Xq.T @ (X - Xq)
    return X, Xq, W, H, D, nu


def test_qep_corrected_weights_solve_the_mixed_target():
    # least squares of Y(mu) = [(1 - mu) X W_p + mu X~ W_p; nu W_p] on A = [X~; nu I]
    X, Xq, W, H, D, nu = _qep_problem(14)
    Wp = W.T
    A = np.vstack([Xq, nu * np.eye(X.shape[1])])
    for mu in (0.0, 0.3, 0.5, 1.0):
        Y = np.vstack([(1 - mu) * X @ Wp + mu * Xq @ Wp, nu * Wp])
        ls = np.linalg.lstsq(A, Y, rcond=None)[0]
        assert np.allclose(qep.corrected_weights(W, H, D, mu), ls.T, rtol=1e-10, atol=1e-12)


def test_qep_objective_splits_into_the_main_problem_plus_a_constant():
    X, Xq, W, H, D, nu = _qep_problem(15)
    mu = 0.5
    Wp = W.T
    A = np.vstack([Xq, nu * np.eye(X.shape[1])])
    Y = np.vstack([(1 - mu) * X @ Wp + mu * Xq @ Wp, nu * Wp])
    Wc = qep.corrected_weights(W, H, D, mu).T
    const = np.sum((Y - A @ Wc) ** 2)
    rng = np.random.default_rng(16)
    for _ in range(5):
        What = Wp + 0.3 * rng.standard_normal(Wp.shape)
        lhs = np.sum((Y - A @ What) ** 2)
        rhs = np.sum((A @ (Wc - What)) ** 2) + const
        assert np.isclose(lhs, rhs, rtol=1e-11)


def test_qep_special_cases():
    X, Xq, W, H, D, nu = _qep_problem(17)
    assert np.array_equal(qep.corrected_weights(W, H, D, 1.0), W)
    assert np.array_equal(qep.corrected_weights(W, H, np.zeros_like(D), 0.0), W)
    Dc = qep.cross([Xq[:20], Xq[20:]], [X[:20], X[20:]], X.shape[1])
    assert np.allclose(Dc, D, rtol=1e-13, atol=1e-13)


# --------------------------------------------------------------------------
# After refinement (App. E.3; packing, activation ordering)
# --------------------------------------------------------------------------

def test_canonicalization_keeps_the_weights_and_makes_scales_positive():
    rng = np.random.default_rng(30)
    rows, cols, g, bits = 6, 96, 32, 3
    codes = rng.integers(0, 8, size=(rows, cols)).astype(np.uint8)
    scales = (rng.standard_normal((rows, cols // g)) * 0.01).astype(np.float32)
    zeros = rng.integers(0, 8, size=(rows, cols // g)).astype(np.int32)
    q, s, z = post.canonicalize(codes, scales, zeros, g, bits)
    assert np.all(s >= 0) and q.max() <= 7 and z.min() >= 0 and z.max() <= 7
    # eq. (canonicalization_equivalence), exactly in fp32
    assert np.array_equal(post.dequantize(q, s, z, g), post.dequantize(codes, scales, zeros, g))
    # a second pass changes nothing
    q2, s2, z2 = post.canonicalize(q, s, z, g, bits)
    assert np.array_equal(q2, q) and np.array_equal(s2, s) and np.array_equal(z2, z)
    # hand-worked group: s = -0.5, z = 2, q = [0, 7] (3 bits) -> s = 0.5, z = 5, q = [7, 0]
    q3, s3, z3 = post.canonicalize(np.array([[0, 7]], np.uint8), np.array([[-0.5]], np.float32),
                                   np.array([[2]], np.int32), 2, 3)
    assert q3.tolist() == [[7, 0]] and s3.tolist() == [[0.5]] and z3.tolist() == [[5]]


def test_dequantize_dtypes():
    import torch
    rng = np.random.default_rng(31)
    codes = rng.integers(0, 16, size=(5, 64)).astype(np.uint8)
    scales = (rng.standard_normal((5, 2)) * 0.03).astype(np.float32)
    zeros = rng.integers(0, 16, size=(5, 2)).astype(np.int32)
    w32 = post.dequantize(codes, scales, zeros, 32)
    assert w32.dtype == np.float32
    assert w32[0, 0] == np.float32(scales[0, 0]) * np.float32(int(codes[0, 0]) - int(zeros[0, 0]))
    # library conversions (round to nearest even) agree with the oracle's
    assert np.array_equal(post.dequantize(codes, scales, zeros, 32, "f16"), w32.astype(np.float16))
    ref_bf16 = torch.from_numpy(w32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(post.dequantize(codes, scales, zeros, 32, "bf16"), ref_bf16)
    # hand-worked bf16 roundings: 1 -> 0x3F80; 1 + 2^-8 (a tie) -> even 0x3F80;
    # 1 + 3 2^-8 (a tie) -> even 0x3F82; 1 + 2^-8 + 2^-20 -> up 0x3F81
    x = np.array([1.0, 1 + 2 ** -8, 1 + 3 * 2 ** -8, 1 + 2 ** -8 + 2 ** -20], np.float32)
    assert post.bf16_bits(x).tolist() == [0x3F80, 0x3F80, 0x3F82, 0x3F81]


def test_dequantize_restores_the_original_column_order():
    rng = np.random.default_rng(32)
    W = rng.standard_normal((3, 8)).astype(np.float32)
    perm = np.array([5, 2, 7, 0, 1, 6, 3, 4])
    codes = np.arange(24, dtype=np.uint8).reshape(3, 8) % 8
    s = np.ones((3, 1), np.float32)
    z = np.zeros((3, 1), np.int32)
    out = post.dequantize(codes, s, z, 8, perm=perm)
    for k in range(8):
        assert np.array_equal(out[:, perm[k]], codes[:, k].astype(np.float32))
    Wp, _ = post.permute(W, np.eye(8), perm)
    assert np.array_equal(Wp[:, 3], W[:, 0])


def test_pack_worked_example_and_round_trip():
    # 3-bit codes 1..7, 0, 1, 2, 3: code k sits at bits 3k; the last code
    # (3 = 0b011) straddles the two words: bits 30, 31 of word 0 hold its low
    # bits (1, 1), bit 0 of word 1 its high bit (0).
    codes = np.array([[1, 2, 3, 4, 5, 6, 7, 0, 1, 2, 3]], np.uint8)
    w0 = (1 + (2 << 3) + (3 << 6) + (4 << 9) + (5 << 12) + (6 << 15) + (7 << 18) + (0 << 21)
          + (1 << 24) + (2 << 27) + (3 << 30)) & 0xFFFFFFFF
    packed = post.pack(codes, 3)
    assert packed.shape == (1, 2) and packed[0, 0] == w0 and packed[0, 1] == 0
    rng = np.random.default_rng(33)
    for bits in range(1, 9):
        c = rng.integers(0, 1 << bits, size=(4, 77)).astype(np.uint8)
        p = post.pack(c, bits)
        assert p.shape == (4, (77 * bits + 31) // 32)
        assert np.array_equal(post.unpack(p, 77, bits), c)
        # every set bit of the stream belongs to some code
        assert sum(bin(int(v)).count("1") for v in p.ravel()) == \
            sum(bin(int(v)).count("1") for v in c.ravel())


def test_act_order_sorts_the_diagonal_stably():
    H = np.diag(np.array([2.0, 5.0, 2.0, 7.0, 5.0], np.float32))
    assert post.act_order(H).tolist() == [3, 1, 4, 0, 2]
