"""Input generators and host quantizers (CPU)."""

import numpy as np
import pytest

from oracle import hosts, jarq
from synth import CONFIGS, make_hessian, make_weights, rtn_quantize


def test_rtn_codes_are_rounded_on_the_stored_grid():
    rng = np.random.default_rng(0)
    W = (0.02 * rng.standard_normal((16, 256))).astype(np.float32)
    for bits in (2, 3, 4, 8):
        q, s, z = rtn_quantize(W, 64, bits)
        qmax = (1 << bits) - 1
        assert q.dtype == np.uint8 and s.dtype == np.float32 and z.dtype == np.int32
        assert q.max() <= qmax and z.min() >= 0 and z.max() <= qmax
        s64 = np.repeat(s.astype(np.float64), 64, axis=1)
        z64 = np.repeat(z.astype(np.float64), 64, axis=1)
        expect = np.clip(np.rint(W.astype(np.float64) / s64) + z64, 0, qmax)
        assert np.array_equal(q, expect.astype(np.uint8))
        err = np.abs(W - s64 * (q - z64))
        inside = (q > 0) & (q < qmax)
        assert np.all(err[inside] <= s64[inside] / 2 * (1 + 1e-6))


def test_gptq_host_with_identity_hessian_is_rtn():
    rng = np.random.default_rng(1)
    W = (0.02 * rng.standard_normal((8, 128))).astype(np.float32)
    q, s, z = hosts.gptq_host(W, np.eye(128) * 3.0, 32, 3)
    q2, s2, z2 = rtn_quantize(W, 32, 3)
    assert np.array_equal(q, q2) and np.array_equal(s, s2) and np.array_equal(z, z2)


def test_gptq_host_beats_rtn_on_correlated_inputs():
    cfg = CONFIGS[0]
    W = make_weights(cfg)
    H = make_hessian(cfg)
    qr, sr, zr = rtn_quantize(W, cfg.group_size, cfg.bits)
    qg, sg, zg = hosts.gptq_host(W, H, cfg.group_size, cfg.bits)
    f_rtn = jarq.objective_rows(W, H, qr, sr, zr, cfg.group_size).sum()
    f_gptq = jarq.objective_rows(W, H, qg, sg, zg, cfg.group_size).sum()
    assert f_gptq < 0.8 * f_rtn


def test_tiny_config_shapes_and_hessian():
    cfg = CONFIGS[0]
    W = make_weights(cfg)
    H, X, H64 = make_hessian(cfg, return_x=True)
    assert W.shape == (64, 256) and W.dtype == np.float32
    assert abs(W.std() - 0.02) < 0.002
    assert H.shape == (256, 256) and H.dtype == np.float32
    assert np.array_equal(H, H.T)
    assert np.all(np.linalg.eigvalsh(H64) > 0)
    d = np.diag(H64)
    # four outlier channels scaled by 20 stand out on the diagonal
    assert np.sum(d > 50 * np.median(d)) == 4


def test_generators_are_deterministic():
    cfg = CONFIGS[0]
    assert np.array_equal(make_weights(cfg), make_weights(cfg))
    assert np.array_equal(make_hessian(cfg), make_hessian(cfg))


def test_ar1_recipe_small_on_cpu():
    """Config-1 recipe with few tokens: AR(1) correlation and outliers show up in H."""
    cfg = CONFIGS[1]
    H = make_hessian(cfg, device="cpu", n_tokens=4096, chunk=2048)
    assert H.shape == (4096, 4096)
    d = np.diag(H).astype(np.float64)
    assert np.sum(d > 100 * np.median(d)) == cfg.n_outliers
    normal = np.nonzero(d < 10 * np.median(d))[0]
    i = normal[(normal[:-1] + 1 == normal[1:]).nonzero()[0][0]]
    corr = H[i, i + 1] / np.sqrt(H[i, i] * H[i + 1, i + 1])
    assert abs(corr - 0.6) < 0.1


@pytest.mark.parametrize("cfg_id", [1, 2, 3, 4])
def test_config_table(cfg_id):
    cfg = CONFIGS[cfg_id]
    assert cfg.cols % cfg.group_size == 0
    assert cfg.n_tokens == 2048 * 128
