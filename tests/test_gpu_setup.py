"""Per-layer set-up on the GPU vs the float64 oracle (needs an MI355X).

The calibration Hessian (fp32 products on the matrix cores, fp32 sums of at
most 256 tokens added in fp64) must lie within the fp32 summation bound of the
exact Hessian of the same fp32 inputs, be exactly symmetric, and be exact when
every partial sum is an integer below 2^24.  The round-to-nearest host must
reproduce the oracle's codes, scales and zero points bit for bit.
"""

import time

import numpy as np
import pytest
import torch

from oracle import hessian as ohess
from oracle import hosts
from oracle import post as opost
from oracle import qep as oqep
from synth import CONFIGS, calibration_chunks, make_weights, propagated_inputs
from tests._gpu_common import jq, say, to_dev

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

U32 = 2.0 ** -24


def _gpu_hessian(chunks, d, alpha, damp=0.0, nu2=0.0):
    Hacc = torch.zeros(d, d, dtype=torch.float64, device="cuda")
    for X in chunks:
        jq.binding.hessian_accumulate(X, Hacc, alpha)
    H = jq.binding.hessian_finalize(Hacc, damp, nu2)
    torch.cuda.synchronize()
    return Hacc.cpu().numpy(), H.cpu().numpy()


def _bound(X32, alpha, Href):
    """fp32 path bound around the exact Hessian of the fp32 inputs, plus the
    final rounding to fp32."""
    ax = np.abs(X32.astype(np.float64))
    return ohess.fp32_error_bound(ax.T @ ax, alpha) + 2 * U32 * np.abs(Href) + 1e-300


@pytest.mark.parametrize("m,d,splits", [(1000, 260, (333,)), (31, 128, ()), (1, 4, ()),
                                        (600, 516, (64, 65, 300))])
def test_hessian_integer_inputs_are_exact(m, d, splits):
    rng = np.random.default_rng(m + d)
    X = rng.integers(-3, 4, size=(m, d)).astype(np.float32)
    say(f"[hessian-int] m={m} d={d} splits={splits}")
    cuts = [0, *splits, m]
    chunks = [to_dev(X[a:b]) for a, b in zip(cuts[:-1], cuts[1:])]
    Hacc, H = _gpu_hessian(chunks, d, 0.5)
    ref = ohess.hessian([X], d, alpha=0.5)
    assert np.array_equal(Hacc, ref)
    assert np.array_equal(H, ref.astype(np.float32))


@pytest.mark.parametrize("m,d,damp,nu2", [(700, 260, 0.01, 0.0), (257, 516, 0.0, 0.36),
                                          (2048, 384, 0.01, 0.36), (5, 132, 0.0, 1.0)])
def test_hessian_matches_oracle_within_fp32_bound(m, d, damp, nu2):
    rng = np.random.default_rng(d)
    X = rng.standard_normal((m, d))
    for c in range(1, d):
        X[:, c] = 0.6 * X[:, c - 1] + 0.8 * X[:, c]
    X[:, rng.choice(d, 3, replace=False)] *= 20.0
    X32 = X.astype(np.float32)
    say(f"[hessian] m={m} d={d} damp={damp} nu2={nu2}")
    half = m // 2
    Hacc, H = _gpu_hessian([to_dev(X32[:half]), to_dev(X32[half:])], d, 1.0 / m, damp, nu2)
    ref_acc = ohess.hessian([X32], d, alpha=1.0 / m)
    ref = ohess.finalize(ref_acc, damp, nu2)
    bound = _bound(X32, 1.0 / m, ref)
    worst = np.max(np.abs(H - ref) / bound)
    say(f"[hessian] worst error / bound {worst:.3e}")
    assert worst <= 1.0
    assert np.array_equal(H, H.T) and np.array_equal(Hacc, Hacc.T)


def test_hessian_zero_tokens_leave_the_accumulator():
    Hacc = torch.full((8, 8), 2.5, dtype=torch.float64, device="cuda")
    jq.binding.hessian_accumulate(torch.zeros(0, 8, dtype=torch.float32, device="cuda"), Hacc)
    torch.cuda.synchronize()
    assert torch.all(Hacc == 2.5)


def test_hessian_full_size_sampled():
    """4096 channels, 262,144 tokens in chunks of 8192 (the headline layer's
    calibration set): sampled entries against the oracle's exact dot products
    of the same fp32 columns, exact symmetry everywhere."""
    cfg = CONFIGS[1]
    d, n = cfg.cols, cfg.n_tokens
    rng = np.random.default_rng(11)
    idx = np.unique(np.concatenate([rng.choice(d, 40, replace=False), [0, 1, d - 1]]))
    cols = []
    Hacc = torch.zeros(d, d, dtype=torch.float64, device="cuda")
    say(f"[hessian-full] d={d} n={n}")
    t_acc = 0.0
    for c, xc in enumerate(calibration_chunks(cfg, device="cuda", chunk=8192)):
        X = xc.to(torch.float32).contiguous()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        jq.binding.hessian_accumulate(X, Hacc, 1.0 / n)
        torch.cuda.synchronize()
        t_acc += time.perf_counter() - t0
        cols.append(X[:, torch.as_tensor(idx, device="cuda")].double().cpu().numpy())
        if c % 8 == 0:
            say(f"[hessian-full] chunk {c}")
    H = jq.binding.hessian_finalize(Hacc, cfg.damping, 0.0)
    torch.cuda.synchronize()
    say(f"[hessian-full] accumulate {1e3 * t_acc:.1f} ms over {n} tokens")
    Xs = np.concatenate(cols)
    Hs = H[torch.as_tensor(idx, device="cuda")][:, torch.as_tensor(idx, device="cuda")].cpu().numpy()
    assert torch.equal(H, H.T)
    diag = torch.diagonal(Hacc).double()
    shift = cfg.damping * float(diag.mean())
    ref = ohess.finalize(ohess.accumulate(np.zeros((len(idx),) * 2), Xs, 1.0 / n), 0.0, 0.0)
    ref[np.arange(len(idx)), np.arange(len(idx))] += shift
    ax = np.abs(Xs)
    bound = ohess.fp32_error_bound(ax.T @ ax, 1.0 / n) + 2 * U32 * np.abs(ref)
    worst = np.max(np.abs(Hs - ref) / bound)
    rel = np.max(np.abs(Hs - ref) / np.sqrt(np.outer(np.diag(ref), np.diag(ref))))
    say(f"[hessian-full] sampled worst error / bound {worst:.3e}, worst rel {rel:.3e}")
    assert worst <= 1.0


def _edge_weights(rows, cols, g, seed):
    rng = np.random.default_rng(seed)
    W = 0.02 * rng.standard_t(5, size=(rows, cols))
    W[0, :g] = 0.0                        # constant group: s = 1, z = 0
    W[1, :g] = np.abs(W[1, :g])           # lo = 0
    W[2, :g] = -np.abs(W[2, :g])          # hi = 0
    W[3, :g] = 0.01 * np.round(W[3, :g] / 0.01 * 2) / 2   # many ties of w / s
    W[4, g:2 * g] = 7.0                   # one-signed constant group
    return W.astype(np.float32)


@pytest.mark.parametrize("g", [32, 64, 128])
@pytest.mark.parametrize("bits", [1, 2, 3, 4, 8])
def test_rtn_matches_oracle_exactly(g, bits):
    rows, cols = 37, 4 * 128
    W = _edge_weights(rows, cols, g, 100 * g + bits)
    say(f"[rtn] g={g} bits={bits}")
    p = jq.binding.make_params(rows, cols, g, bits, 1)
    q, s, z = jq.binding.rtn(p, to_dev(W))
    torch.cuda.synchronize()
    rq, rs, rz = hosts.rtn_host(W, g, bits)
    assert np.array_equal(q.cpu().numpy(), rq)
    assert np.array_equal(s.cpu().numpy().view(np.uint32), rs.view(np.uint32))
    assert np.array_equal(z.cpu().numpy(), rz)


@pytest.mark.parametrize("cfg_id", [1, 2])
def test_rtn_full_size_exact(cfg_id):
    cfg = CONFIGS[cfg_id]
    W = make_weights(cfg)
    say(f"[rtn-full] config {cfg.name}")
    p = jq.binding.make_params(cfg.rows, cfg.cols, cfg.group_size, cfg.bits, 1)
    Wd = to_dev(W)
    q, s, z = jq.binding.rtn(p, Wd)
    torch.cuda.synchronize()
    rq, rs, rz = hosts.rtn_host(W, cfg.group_size, cfg.bits)
    assert np.array_equal(q.cpu().numpy(), rq)
    assert np.array_equal(s.cpu().numpy().view(np.uint32), rs.view(np.uint32))
    assert np.array_equal(z.cpu().numpy(), rz)


def _correlated_hessian(d, seed, rho=0.7, n=None):
    rng = np.random.default_rng(seed)
    n = n or 3 * d
    X = rng.standard_normal((n, d))
    for c in range(1, d):
        X[:, c] = rho * X[:, c - 1] + np.sqrt(1 - rho * rho) * X[:, c]
    H = X.T @ X / n
    H += 0.01 * np.mean(np.diag(H)) * np.eye(d)
    return H.astype(np.float32)


def _check_gptq(W, H, g, bits, q, s, z, rows_idx=None):
    """Codes identical except where the oracle's pre-rounding value lies within
    1e-6 of a rounding boundary (at most 0.1% of codes); scales within 1e-6
    relative; zero points identical except near-boundary groups."""
    Wr = W if rows_idx is None else W[rows_idx]
    rq, rs, rz, pre, zpre = hosts.gptq_host(Wr, H, g, bits, return_pre=True)
    if rows_idx is not None:
        q, s, z = q[rows_idx], s[rows_idx], z[rows_idx]
    dz = z != rz
    znear = np.abs(zpre - np.floor(zpre) - 0.5) < 1e-6
    assert np.all(znear[dz]) and dz.mean() <= 1e-3
    srel = np.abs(s.astype(np.float64) - rs) / np.abs(rs.astype(np.float64))
    say(f"[gptq] worst scale rel {srel.max():.3e}, zero-point mismatches {int(dz.sum())}")
    # groups whose grid differs cascade into their codes: judge codes elsewhere
    ok_groups = np.repeat(~dz & (srel <= 1e-6), g, axis=1)
    differ = (q != rq) & ok_groups
    near = np.abs(pre - np.floor(pre) - 0.5) < 1e-6
    say(f"[gptq] code mismatches {int(differ.sum())} of {q.size}")
    assert np.all(near[differ]) and differ.mean() <= 1e-3
    assert np.mean(srel <= 1e-6) >= 1 - 1e-3


@pytest.mark.parametrize("rows,cols,g,bits", [(100, 256, 64, 3), (67, 384, 128, 4),
                                              (130, 320, 32, 2), (64, 128, 128, 8)])
def test_gptq_matches_oracle(rows, cols, g, bits):
    rng = np.random.default_rng(rows + cols)
    W = (0.02 * rng.standard_t(5, size=(rows, cols))).astype(np.float32)
    H = _correlated_hessian(cols, cols)
    say(f"[gptq] rows={rows} cols={cols} g={g} bits={bits}")
    p = jq.binding.make_params(rows, cols, g, bits, 1)
    q, s, z = jq.binding.gptq(p, to_dev(W), to_dev(H))
    torch.cuda.synchronize()
    _check_gptq(W, H, g, bits, q.cpu().numpy(), s.cpu().numpy(), z.cpu().numpy())


def test_gptq_full_size_sampled_rows():
    """The wide-MLP layer (14336 x 4096, g = 64, 3 bits) with its own Hessian:
    512 sampled rows against the oracle (rows are independent)."""
    from synth import make_hessian
    cfg = CONFIGS[4]
    say(f"[gptq-full] building {cfg.name}")
    W = make_weights(cfg)
    H = make_hessian(cfg, device="cuda")
    p = jq.binding.make_params(cfg.rows, cfg.cols, cfg.group_size, cfg.bits, 1)
    Wd, Hd = to_dev(W), to_dev(H)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    q, s, z = jq.binding.gptq(p, Wd, Hd)
    torch.cuda.synchronize()
    say(f"[gptq-full] GPU host {1e3 * (time.perf_counter() - t0):.1f} ms")
    idx = np.sort(np.random.default_rng(4).choice(cfg.rows, 512, replace=False))
    _check_gptq(W, H, cfg.group_size, cfg.bits, q.cpu().numpy(), s.cpu().numpy(),
                z.cpu().numpy(), rows_idx=idx)


def test_gptq_rejects_an_indefinite_hessian():
    rng = np.random.default_rng(5)
    W = (0.02 * rng.standard_normal((32, 128))).astype(np.float32)
    H = _correlated_hessian(128, 3)
    H[70, 70] = -1.0
    p = jq.binding.make_params(32, 128, 64, 3, 1)
    with pytest.raises(jq.binding.JarqError) as ei:
        jq.binding.gptq(p, to_dev(W), to_dev(H))
    assert ei.value.status == jq.binding.JARQ_ENOT_SPD


# --------------------------------------------------------------------------
# Propagation-corrected target (App. E.5)
# --------------------------------------------------------------------------

def test_cross_integer_inputs_are_exact():
    rng = np.random.default_rng(21)
    m, d = 700, 196
    X = rng.integers(-3, 4, size=(m, d)).astype(np.float32)
    Xq = (X + rng.integers(-1, 2, size=(m, d))).astype(np.float32)
    D = torch.zeros(d, d, dtype=torch.float64, device="cuda")
    for a, b in ((0, 300), (300, m)):
        jq.binding.cross_accumulate(to_dev(Xq[a:b]), to_dev(X[a:b]), D, 0.5)
    torch.cuda.synchronize()
    assert np.array_equal(D.cpu().numpy(), oqep.cross([Xq], [X], d, 0.5))


@pytest.mark.parametrize("m,d", [(900, 260), (33, 128)])
def test_cross_matches_oracle_within_fp32_bound(m, d):
    rng = np.random.default_rng(m)
    X = rng.standard_normal((m, d)).astype(np.float32)
    X[:, 3] *= 20.0
    Xq = propagated_inputs(X, m)
    D = torch.zeros(d, d, dtype=torch.float64, device="cuda")
    jq.binding.cross_accumulate(to_dev(Xq), to_dev(X), D, 1.0 / m)
    torch.cuda.synchronize()
    ref = oqep.cross([Xq], [X], d, 1.0 / m)
    diff32 = (X - Xq).astype(np.float64)
    absg = np.abs(Xq.astype(np.float64)).T @ np.abs(diff32)
    # one more rounding than the Hessian: X - X~ is formed in fp32
    bound = ohess.fp32_error_bound(absg, 1.0 / m, segment=257) + 1e-300
    worst = np.max(np.abs(D.cpu().numpy() - ref) / bound)
    say(f"[cross] m={m} d={d} worst error / bound {worst:.3e}")
    assert worst <= 1.0


def _qep_inputs(rows, d, seed, n=None):
    rng = np.random.default_rng(seed)
    n = n or 4 * d
    X = rng.standard_normal((n, d))
    for c in range(1, d):
        X[:, c] = 0.6 * X[:, c - 1] + 0.8 * X[:, c]
    X = X.astype(np.float32)
    Xq = propagated_inputs(X, seed)
    H = ohess.hessian([Xq], d, alpha=1.0 / n, damp=0.01).astype(np.float32)
    D = oqep.cross([Xq], [X], d, alpha=1.0 / n)
    W = (0.02 * rng.standard_t(5, size=(rows, d))).astype(np.float32)
    return W, H, D


def _check_qep(Wc, ref, W):
    corr = np.max(np.abs(ref - W))
    err = np.abs(Wc.astype(np.float64) - ref)
    bound = 2.0 ** -24 * np.abs(ref) + 1e-9 * corr
    say(f"[qep] max |correction| {corr:.3e}, worst error / bound {np.max(err / bound):.3e}")
    assert np.all(err <= bound)


@pytest.mark.parametrize("rows,d,mu", [(100, 256, 0.5), (67, 320, 0.0), (64, 192, 0.25)])
def test_qep_correct_matches_oracle(rows, d, mu):
    W, H, D = _qep_inputs(rows, d, rows + d)
    p = jq.binding.make_params(rows, d, 64, 3, 1)
    Wc = jq.binding.qep_correct(p, to_dev(W), to_dev(H), to_dev(D), mu)
    torch.cuda.synchronize()
    _check_qep(Wc.cpu().numpy(), oqep.corrected_weights(W, H, D, mu), W.astype(np.float64))


def test_qep_mu_one_returns_the_weights():
    W, H, D = _qep_inputs(40, 128, 9)
    p = jq.binding.make_params(40, 128, 64, 3, 1)
    Wc = jq.binding.qep_correct(p, to_dev(W), to_dev(H), to_dev(D), 1.0)
    torch.cuda.synchronize()
    assert np.array_equal(Wc.cpu().numpy(), W)


def test_qep_full_size_sampled_rows():
    """The 4096 x 4096 attention projection with its Hessian and a cross term
    from 8192 calibration tokens and their propagated counterparts: 64 sampled
    rows against the oracle (rows are independent)."""
    cfg = CONFIGS[1]
    W = make_weights(cfg)
    from synth import make_hessian
    H = make_hessian(cfg, device="cuda")
    X = next(calibration_chunks(cfg, device="cuda", n_tokens=8192, chunk=8192))
    X = X.to(torch.float32).cpu().numpy()
    Xq = propagated_inputs(X, 1)
    D = oqep.cross([Xq], [X], cfg.cols, alpha=1.0 / X.shape[0])
    say("[qep-full] inputs ready")
    p = jq.binding.make_params(cfg.rows, cfg.cols, cfg.group_size, cfg.bits, 1)
    Wd, Hd, Dd = to_dev(W), to_dev(H), to_dev(D)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    Wc = jq.binding.qep_correct(p, Wd, Hd, Dd, 0.5)
    torch.cuda.synchronize()
    say(f"[qep-full] GPU correction {1e3 * (time.perf_counter() - t0):.1f} ms")
    idx = np.sort(np.random.default_rng(6).choice(cfg.rows, 64, replace=False))
    ref = oqep.corrected_weights(W[idx], H, D, 0.5)
    _check_qep(Wc.cpu().numpy()[idx], ref, W[idx].astype(np.float64))


def test_qep_rejects_an_indefinite_hessian():
    W, H, D = _qep_inputs(32, 128, 10)
    H[5, 5] = -1.0
    p = jq.binding.make_params(32, 128, 64, 3, 1)
    with pytest.raises(jq.binding.JarqError) as ei:
        jq.binding.qep_correct(p, to_dev(W), to_dev(H), to_dev(D), 0.5)
    assert ei.value.status == jq.binding.JARQ_ENOT_SPD


# --------------------------------------------------------------------------
# After refinement: canonical scales, dequantized weights, packed codes,
# activation ordering
# --------------------------------------------------------------------------

def _random_state(rows, cols, g, bits, seed):
    rng = np.random.default_rng(seed)
    codes = rng.integers(0, 1 << bits, size=(rows, cols)).astype(np.uint8)
    scales = (rng.standard_normal((rows, cols // g)) * 0.02).astype(np.float32)
    scales[0, 0] = 0.0
    zeros = rng.integers(0, 1 << bits, size=(rows, cols // g)).astype(np.int32)
    return codes, scales, zeros


@pytest.mark.parametrize("g,bits", [(32, 2), (64, 3), (128, 4), (64, 8)])
def test_canonicalize_matches_oracle(g, bits):
    rows, cols = 45, 384
    codes, scales, zeros = _random_state(rows, cols, g, bits, g + bits)
    p = jq.binding.make_params(rows, cols, g, bits, 1)
    q, s, z = to_dev(codes), to_dev(scales), to_dev(zeros)
    jq.binding.canonicalize(p, q, s, z)
    torch.cuda.synchronize()
    rq, rs, rz = opost.canonicalize(codes, scales, zeros, g, bits)
    assert np.array_equal(q.cpu().numpy(), rq)
    assert np.array_equal(s.cpu().numpy().view(np.uint32), rs.view(np.uint32))
    assert np.array_equal(z.cpu().numpy(), rz)


@pytest.mark.parametrize("dtype,name", [(torch.float32, "f32"), (torch.float16, "f16"),
                                        (torch.bfloat16, "bf16")])
def test_dequantize_matches_oracle(dtype, name):
    rows, cols, g, bits = 37, 256, 64, 4
    codes, scales, zeros = _random_state(rows, cols, g, bits, 40)
    scales[3, 1] = 7e4          # overflows fp16
    p = jq.binding.make_params(rows, cols, g, bits, 1)
    perm = np.random.default_rng(41).permutation(cols).astype(np.int32)
    for pm in (None, perm):
        out = jq.binding.dequantize(p, to_dev(codes), to_dev(scales), to_dev(zeros), dtype,
                                    None if pm is None else to_dev(pm))
        torch.cuda.synchronize()
        ref = opost.dequantize(codes, scales, zeros, g, name, pm)
        got = out.cpu()
        got = got.view(torch.int16).numpy().view(np.uint16) if name == "bf16" else got.numpy()
        assert np.array_equal(got.view(np.uint8), ref.view(np.uint8))


@pytest.mark.parametrize("bits", [1, 2, 3, 4, 5, 6, 7, 8])
def test_pack_and_unpack_match_oracle(bits):
    rows, cols = 19, 352
    codes = np.random.default_rng(bits).integers(0, 1 << bits, size=(rows, cols)).astype(np.uint8)
    p = jq.binding.make_params(rows, cols, 32, bits, 1)
    packed = jq.binding.pack_codes(p, to_dev(codes))
    back = jq.binding.unpack_codes(p, packed)
    torch.cuda.synchronize()
    ref = opost.pack(codes, bits)
    assert np.array_equal(packed.cpu().numpy().view(np.uint32), ref)
    assert np.array_equal(back.cpu().numpy(), codes)


def test_act_order_flow_matches_oracle():
    """GPTQ with activation ordering: order the channels, gather the layer,
    build the host in the permuted coordinates, write the weights back."""
    rows, cols, g, bits = 96, 320, 64, 3
    rng = np.random.default_rng(50)
    W = (0.02 * rng.standard_normal((rows, cols))).astype(np.float32)
    Dg = rng.uniform(0.5, 2.0, cols)
    H = _correlated_hessian(cols, 51).astype(np.float64) * Dg[:, None] * Dg[None, :]
    t = max(H[7, 7], H[8, 8])               # a tie, made by raising a diagonal entry
    H[7, 7] = H[8, 8] = t
    H = H.astype(np.float32)
    p = jq.binding.make_params(rows, cols, g, bits, 1)
    perm = jq.binding.act_order(to_dev(H))
    Wp, Hp = jq.binding.permute(p, perm, to_dev(W), to_dev(H))
    q, s, z = jq.binding.gptq(p, Wp, Hp)
    out = jq.binding.dequantize(p, q, s, z, torch.float32, perm)
    torch.cuda.synchronize()
    rperm = opost.act_order(H)
    assert np.array_equal(perm.cpu().numpy(), rperm)
    rWp, rHp = opost.permute(W, H, rperm)
    assert np.array_equal(Wp.cpu().numpy(), rWp) and np.array_equal(Hp.cpu().numpy(), rHp)
    _check_gptq(rWp, rHp, g, bits, q.cpu().numpy(), s.cpu().numpy(), z.cpu().numpy())
    rq, rs, rz = (x.cpu().numpy() for x in (q, s, z))
    assert np.array_equal(out.cpu().numpy(), opost.dequantize(rq, rs, rz, g, "f32", rperm))


# --------------------------------------------------------------------------
# The widest layer (4096 x 11008, G = 86): set-up entry points at full width
# --------------------------------------------------------------------------

def _wide_inputs(n_tokens=8192):
    cfg = CONFIGS[3]
    X = next(calibration_chunks(cfg, device="cuda", n_tokens=n_tokens, chunk=n_tokens))
    return cfg, X.to(torch.float32).contiguous()


def test_hessian_widest_layer_sampled():
    cfg, X = _wide_inputs()
    d, n = cfg.cols, X.shape[0]
    say(f"[wide-hessian] d={d} n={n}")
    Hacc = torch.zeros(d, d, dtype=torch.float64, device="cuda")
    jq.binding.hessian_accumulate(X[:5000], Hacc, 1.0 / n)
    jq.binding.hessian_accumulate(X[5000:], Hacc, 1.0 / n)
    H = jq.binding.hessian_finalize(Hacc, cfg.damping, 0.0)
    torch.cuda.synchronize()
    assert torch.equal(H, H.T)
    idx = np.unique(np.concatenate([np.random.default_rng(3).choice(d, 40, replace=False),
                                    [0, d - 1]]))
    ti = torch.as_tensor(idx, device="cuda")
    Xs = X[:, ti].double().cpu().numpy()
    ref = ohess.accumulate(np.zeros((len(idx),) * 2), Xs, 1.0 / n)
    ref[np.arange(len(idx)), np.arange(len(idx))] += cfg.damping * float(torch.diagonal(Hacc).mean())
    ax = np.abs(Xs)
    bound = ohess.fp32_error_bound(ax.T @ ax, 1.0 / n) + 2 * U32 * np.abs(ref)
    Hs = H[ti][:, ti].double().cpu().numpy()
    worst = np.max(np.abs(Hs - ref) / bound)
    say(f"[wide-hessian] sampled worst error / bound {worst:.3e}")
    assert worst <= 1.0


def test_gptq_and_qep_widest_layer_sampled_rows():
    from synth import make_hessian
    cfg = CONFIGS[3]
    say(f"[wide] building {cfg.name}")
    W = make_weights(cfg)
    H = make_hessian(cfg, device="cuda")
    p = jq.binding.make_params(cfg.rows, cfg.cols, cfg.group_size, cfg.bits, 1)
    Wd, Hd = to_dev(W), to_dev(H)
    t0 = time.perf_counter()
    q, s, z = jq.binding.gptq(p, Wd, Hd)
    torch.cuda.synchronize()
    say(f"[wide] GPTQ host {1e3 * (time.perf_counter() - t0):.1f} ms")
    idx = np.sort(np.random.default_rng(8).choice(cfg.rows, 32, replace=False))
    _check_gptq(W, H, cfg.group_size, cfg.bits, q.cpu().numpy(), s.cpu().numpy(),
                z.cpu().numpy(), rows_idx=idx)
    _, X = _wide_inputs(4096)
    Xn = X.cpu().numpy()
    Xq = propagated_inputs(Xn, 3)
    D = oqep.cross([Xq], [Xn], cfg.cols, alpha=1.0 / Xn.shape[0])
    t0 = time.perf_counter()
    Wc = jq.binding.qep_correct(p, Wd, Hd, to_dev(D), 0.5)
    torch.cuda.synchronize()
    say(f"[wide] W_corr {1e3 * (time.perf_counter() - t0):.1f} ms")
    _check_qep(Wc.cpu().numpy()[idx], oqep.corrected_weights(W[idx], H, D, 0.5),
               W[idx].astype(np.float64))


def test_layer_flow_end_to_end():
    """One layer through every step on the GPU: Hessian from its tokens, RTN
    host, refinement (App. E.2 early stopping), canonical positive scales,
    dequantized and packed output.  Canonicalization must leave the weights
    unchanged bit for bit (eq. (canonicalization_equivalence)); the packed
    codes must unpack to the canonical codes; the refined objective must not
    exceed the host's (Cor. 1)."""
    from oracle import jarq as ojarq
    cfg = CONFIGS[0]
    W = make_weights(cfg)
    from synth import make_hessian
    _, X, _ = make_hessian(cfg, return_x=True)
    X32 = to_dev(X.astype(np.float32))
    H = jq.binding.hessian([X32[:300], X32[300:]], cfg.cols, alpha=1.0 / X.shape[0],
                           damp=cfg.damping)
    Wd = to_dev(W)
    p = jq.binding.make_params(cfg.rows, cfg.cols, cfg.group_size, cfg.bits, 20, tau=1e-5)
    q, s, z = jq.binding.rtn(p, Wd)
    q0, s0, z0 = q.clone(), s.clone(), z.clone()
    ws = jq.binding.alloc_workspace(p)
    st = jq.binding.refine(p, Wd, H, q, s, z, ws)
    torch.cuda.synchronize()
    Hn = H.cpu().numpy()
    f_host = ojarq.objective_rows(W, Hn, q0.cpu().numpy(), s0.cpu().numpy(), z0.cpu().numpy(),
                                  cfg.group_size).sum()
    f_ref = ojarq.objective_rows(W, Hn, q.cpu().numpy(), s.cpu().numpy(), z.cpu().numpy(),
                                 cfg.group_size).sum()
    say(f"[flow] sweeps {st['sweeps_run']}, objective {f_host:.6e} -> {f_ref:.6e}")
    assert f_ref <= f_host
    # Every other group of the refined state rewritten in its negative-scale
    # form (s -> -s, q -> qmax - q, z -> qmax - z, the same weights), plus the
    # groups refinement itself left negative: canonicalization must restore
    # positive scales without changing a weight.
    qmax = (1 << cfg.bits) - 1
    qn, sn, zn = q.cpu().numpy().copy(), s.cpu().numpy().copy(), z.cpu().numpy().copy()
    flip = (np.arange(sn.size).reshape(sn.shape) % 2 == 0) & (sn > 0)
    sn[flip] = -sn[flip]
    zn[flip] = qmax - zn[flip]
    fc = np.repeat(flip, cfg.group_size, axis=1)
    qn[fc] = qmax - qn[fc]
    qd, sd, zd = to_dev(qn), to_dev(sn), to_dev(zn)
    before = jq.binding.dequantize(p, qd, sd, zd, torch.float32)
    ref = jq.binding.dequantize(p, q, s, z, torch.float32)
    jq.binding.canonicalize(p, qd, sd, zd)
    after = jq.binding.dequantize(p, qd, sd, zd, torch.float32)
    packed = jq.binding.pack_codes(p, qd)
    torch.cuda.synchronize()
    say(f"[flow] groups with negative scales: {int(flip.sum())} planted, "
        f"{int((s < 0).sum())} from refinement")
    assert torch.all(sd >= 0)
    # equal values (a weight of 0 is -0.0 in the negative form: compared by value)
    assert torch.equal(before, ref)
    # and after canonicalization equal bit for bit
    assert torch.equal(after.view(torch.int32), ref.view(torch.int32))
    pos = (s >= 0)
    assert torch.equal(sd[pos], s[pos]) and torch.equal(zd[pos], z[pos])
    assert torch.equal(jq.binding.unpack_codes(p, packed), qd)


# --------------------------------------------------------------------------
# Hessian from bf16 inputs
# --------------------------------------------------------------------------

@pytest.mark.parametrize("m,d,splits", [(1000, 264, (333,)), (64, 128, ()), (1, 8, ()),
                                        (700, 520, (63, 64, 300))])
def test_hessian_bf16_integer_inputs_are_exact(m, d, splits):
    rng = np.random.default_rng(m + d + 1)
    X = rng.integers(-3, 4, size=(m, d)).astype(np.float32)
    say(f"[hessian-bf16-int] m={m} d={d} splits={splits}")
    Xb = to_dev(X).to(torch.bfloat16)
    cuts = [0, *splits, m]
    Hacc = torch.zeros(d, d, dtype=torch.float64, device="cuda")
    for a, b in zip(cuts[:-1], cuts[1:]):
        jq.binding.hessian_accumulate(Xb[a:b].contiguous(), Hacc, 0.5)
    torch.cuda.synchronize()
    assert np.array_equal(Hacc.cpu().numpy(), ohess.hessian([X], d, alpha=0.5))


@pytest.mark.parametrize("m,d", [(900, 264), (2048, 384), (33, 128)])
def test_hessian_bf16_matches_oracle_within_fp32_bound(m, d):
    rng = np.random.default_rng(d + 7)
    X = rng.standard_normal((m, d))
    for c in range(1, d):
        X[:, c] = 0.6 * X[:, c - 1] + 0.8 * X[:, c]
    X[:, 5] *= 20.0
    Xb = to_dev(X.astype(np.float32)).to(torch.bfloat16)
    Xv = Xb.float().cpu().numpy().astype(np.float64)     # the bf16 values the GPU sees
    Hacc = torch.zeros(d, d, dtype=torch.float64, device="cuda")
    jq.binding.hessian_accumulate(Xb, Hacc, 1.0 / m)
    torch.cuda.synchronize()
    H = Hacc.cpu().numpy()
    ref = ohess.hessian([Xv], d, alpha=1.0 / m)
    ax = np.abs(Xv)
    bound = ohess.fp32_error_bound(ax.T @ ax, 1.0 / m) + 1e-300
    worst = np.max(np.abs(H - ref) / bound)
    say(f"[hessian-bf16] m={m} d={d} worst error / bound {worst:.3e}")
    assert worst <= 1.0
    assert np.array_equal(H, H.T)


def test_hessian_bf16_full_size_sampled():
    cfg = CONFIGS[1]
    d, n = cfg.cols, cfg.n_tokens
    rng = np.random.default_rng(12)
    idx = np.unique(np.concatenate([rng.choice(d, 40, replace=False), [0, d - 1]]))
    ti = torch.as_tensor(idx, device="cuda")
    cols = []
    Hacc = torch.zeros(d, d, dtype=torch.float64, device="cuda")
    t_acc = 0.0
    for xc in calibration_chunks(cfg, device="cuda", chunk=8192):
        X = xc.to(torch.bfloat16).contiguous()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        jq.binding.hessian_accumulate(X, Hacc, 1.0 / n)
        torch.cuda.synchronize()
        t_acc += time.perf_counter() - t0
        cols.append(X[:, ti].double().cpu().numpy())
    say(f"[hessian-bf16-full] accumulate {1e3 * t_acc:.1f} ms over {n} tokens")
    Xs = np.concatenate(cols)
    Hs = Hacc[ti][:, ti].cpu().numpy()
    ref = ohess.accumulate(np.zeros((len(idx),) * 2), Xs, 1.0 / n)
    ax = np.abs(Xs)
    worst = np.max(np.abs(Hs - ref) / (ohess.fp32_error_bound(ax.T @ ax, 1.0 / n) + 1e-300))
    say(f"[hessian-bf16-full] sampled worst error / bound {worst:.3e}")
    assert worst <= 1.0
    assert torch.equal(Hacc, Hacc.T)
