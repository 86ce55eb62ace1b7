"""HIP path vs the float64 oracle (needs an MI355X and the built libjarq.so).

Per stage: the objective, the scale step (scales within 1e-4 relative) and the
code step checked decision by decision against the oracle conditioned on the
GPU's earlier decisions (codes identical except within 1e-4 of a rounding
boundary, at most 0.1% of codes).  End to end: K sweeps, final objective
within 1e-5 relative; on the small layers against the free-running oracle, on
the full-size layers and with early stopping against the oracle's own K
iterations that defer to the GPU only at decisions inside those bands (a
single near-boundary split changes every later decision of a row, so the
free-running comparison there is reported, not asserted).  Shapes cover
several tiles with ragged tails, every group size and bit width, the
degenerate cases of the method, and the full-size layers (checked on sampled
rows, rows being independent).
"""

import numpy as np
import pytest
import torch

from synth import rtn_quantize
from tests._gpu_common import (CONFIGS, OBJ_RTOL, GpuLayer, check_code_step, check_forced,
                               check_scales, jarq, jq, layer, random_layer, rel, say,
                               traced_sweeps)

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]


def _oracle_final_objective(W, H, q, s, z, g):
    return jarq.objective_rows(W, H, q, s, z, g)


# --------------------------------------------------------------------------
# tiny layer (64 x 256, g = 64, 3 bits, 5 sweeps)
# --------------------------------------------------------------------------

def test_objective_tiny():
    cfg, W, H, q, s, z = layer(0)
    gl = GpuLayer(W, H, q, s, z, cfg.group_size, cfg.bits)
    F = gl.objective()
    F_ref = jarq.objective_rows(W, H, q, s, z, cfg.group_size)
    say(f"[objective] worst rel {np.max(np.abs(F - F_ref) / F_ref):.3e}")
    assert np.all(np.abs(F - F_ref) <= OBJ_RTOL * F_ref)


def test_scale_step_tiny():
    cfg, W, H, q, s, z = layer(0)
    gl = GpuLayer(W, H, q, s, z, cfg.group_size, cfg.bits)
    gl.scale_step()
    _, s_gpu = gl.state()
    s_ref, ridge = jarq.scale_step(W, H, q, z, cfg.group_size)
    assert not ridge.any()
    check_scales(s_gpu, s_ref)


def test_code_step_tiny_teacher_forced():
    cfg, W, H, q, s, z = layer(0)
    g, bits = cfg.group_size, cfg.bits
    gl = GpuLayer(W, H, q, s, z, g, bits)
    R = jarq.group_factors(H, g)
    for sweep in range(3):
        gl.scale_step()
        q0, s1 = gl.state()
        cand, dec = gl.code_step()
        q1, _ = gl.state()
        check_code_step(W, H, R, q0, s1, z, g, bits, cand, dec, f" sweep {sweep + 1}")
        expect = q0.copy()
        for i in range(cfg.groups):
            acc = dec[:, i] == jq.DEC_ACCEPT
            expect[acc, i * g:(i + 1) * g] = cand[acc, i * g:(i + 1) * g]
        assert np.array_equal(q1, expect)
        if sweep == 0:
            assert (dec == jq.DEC_ACCEPT).sum() > 0


def test_refine_tiny_end_to_end():
    cfg, W, H, q, s, z = layer(0)
    g, bits, K = cfg.group_size, cfg.bits, cfg.sweeps
    gl = GpuLayer(W, H, q, s, z, g, bits, sweeps=K)
    st = jq.sweeps(gl.p, gl.W, gl.H, gl.codes, gl.scales, gl.zeros, gl.ws)
    qg, sg = gl.state()
    qo, so, hist = jarq.refine(W, H, q, s, z, g, bits, K)
    F_gpu = _oracle_final_objective(W, H, qg, sg, z, g).sum()
    F_or = _oracle_final_objective(W, H, qo, so, z, g).sum()
    F_host = jarq.objective_rows(W, H, q, s, z, g).sum()
    agree = np.mean(qg == qo)
    say(f"[e2e tiny] F_host {F_host:.6e} F_gpu {F_gpu:.9e} F_oracle {F_or:.9e} "
        f"rel {rel(F_gpu, F_or):.2e} code agreement {agree:.6f} stats {st['accepted_groups']}")
    assert st["sweeps_run"] == K
    assert rel(F_gpu, F_or) <= OBJ_RTOL
    assert F_gpu < F_host
    L = st["objective_after_scales"]
    for k in range(K):
        assert rel(L[k], np.nansum(hist[k].L)) <= OBJ_RTOL
    # the GPU objective of its own final state
    F_dev = gl.objective()
    F_dev_ref = jarq.objective_rows(W, H, qg, sg, z, g)
    assert np.all(np.abs(F_dev - F_dev_ref) <= OBJ_RTOL * F_dev_ref)


def test_zero_sweeps_is_identity():
    cfg, W, H, q, s, z = layer(0)
    gl = GpuLayer(W, H, q, s, z, cfg.group_size, cfg.bits, sweeps=0)
    st = jq.sweeps(gl.p, gl.W, gl.H, gl.codes, gl.scales, gl.zeros, gl.ws)
    qg, sg = gl.state()
    assert st["sweeps_run"] == 0
    assert np.array_equal(qg, q) and np.array_equal(sg, s)


def test_deterministic():
    cfg, W, H, q, s, z = layer(0)
    outs = []
    for _ in range(2):
        gl = GpuLayer(W, H, q, s, z, cfg.group_size, cfg.bits, sweeps=cfg.sweeps)
        jq.sweeps(gl.p, gl.W, gl.H, gl.codes, gl.scales, gl.zeros, gl.ws)
        outs.append(gl.state())
    assert np.array_equal(outs[0][0], outs[1][0])
    assert np.array_equal(outs[0][1].view(np.uint32), outs[1][1].view(np.uint32))


def test_stage_mask_times_only_the_selected_stages():
    # Stage timing is instrumentation: the selected stages report time, the
    # others 0, and the results are bit-identical to a run timing every stage.
    # (the tiny layer's four groups form one panel: no panel update runs)
    cfg, W, H, q, s, z = layer(0)
    res = jq.binding.STAGE_NAMES.index("residual")
    panel = jq.binding.STAGE_NAMES.index("panel")
    outs = []
    for mask in (1 << res, 0):
        gl = GpuLayer(W, H, q, s, z, cfg.group_size, cfg.bits, sweeps=3)
        st = jq.sweeps(gl.p, gl.W, gl.H, gl.codes, gl.scales, gl.zeros, gl.ws, stage_mask=mask)
        outs.append(gl.state())
        for k in range(st["sweeps_run"]):
            for j, ms in enumerate(st["stage_ms"][k]):
                if (mask == 0 and j != panel) or j == res:
                    assert ms > 0.0, (mask, k, j)
                else:
                    assert ms == 0.0, (mask, k, j)
    assert np.array_equal(outs[0][0], outs[1][0])
    assert np.array_equal(outs[0][1].view(np.uint32), outs[1][1].view(np.uint32))


def test_refine_entry_equals_prepare_plus_sweeps():
    cfg, W, H, q, s, z = layer(0)
    a = GpuLayer(W, H, q, s, z, cfg.group_size, cfg.bits, sweeps=3)
    jq.sweeps(a.p, a.W, a.H, a.codes, a.scales, a.zeros, a.ws)
    b = GpuLayer(W, H, q, s, z, cfg.group_size, cfg.bits, sweeps=3, prepare=False)
    st = jq.refine(b.p, b.W, b.H, b.codes, b.scales, b.zeros, b.ws)
    assert st["prep_ms"] > 0
    qa, sa = a.state()
    qb, sb = b.state()
    assert np.array_equal(qa, qb) and np.array_equal(sa, sb)


def _check_stopping_run(W, H, q, s, z, g, bits, K, tau, label):
    """Early stopping on the GPU against the oracle.

    A row that stops at iteration k holds the scales of iteration k and the
    codes of iteration k - 1, and rows are independent, so each row of the
    stopping run (jarq_sweeps) must equal, bit for bit, the same row of a run
    without stopping (the traced step entry points) cut at the iteration
    jarq_stop_sweeps reports.  The oracle then runs its own K iterations with
    the stopping rule, deferring to the GPU only inside the bands: its codes
    must equal the GPU's, every row's objective must agree within 1e-5, and
    the number of active rows must agree in every sweep."""
    rows = W.shape[0]
    R = jarq.group_factors(H, g)
    tr = GpuLayer(W, H, q, s, z, g, bits)
    cands, decs, states = traced_sweeps(tr, K)
    del tr
    gl = GpuLayer(W, H, q, s, z, g, bits, sweeps=K, tau=tau)
    st = jq.sweeps(gl.p, gl.W, gl.H, gl.codes, gl.scales, gl.zeros, gl.ws)
    qg, sg = gl.state()
    stop_at = jq.stop_sweeps(gl.p, gl.ws).cpu().numpy()
    say(f"[stopping{label}] gpu active per sweep {st['rows_active']}, stopped rows "
        f"{int(np.count_nonzero(stop_at))} of {rows}")
    assert np.all((stop_at == 0) | ((stop_at >= 2) & (stop_at <= st["sweeps_run"])))
    for r in range(rows):
        k = int(stop_at[r])
        qk = states[k - 1][0][r] if k else states[K][0][r]
        sk = states[k][1][r] if k else states[K][1][r]
        assert np.array_equal(qg[r], qk), (r, k)
        assert np.array_equal(sg[r].view(np.uint32), sk.view(np.uint32)), (r, k)
    check_forced(W, H, R, q, s, z, g, bits, K, cands, decs, qg, sg, label, tau=tau,
                 stop_at=stop_at, rows_active=st["rows_active"])
    return st, qg, sg


def test_early_stopping_tiny():
    cfg, W, H, q, s, z = layer(0)
    st, _, _ = _check_stopping_run(W, H, q, s, z, cfg.group_size, cfg.bits, 12, 1e-5, " tiny")
    assert st["rows_active_end"] < cfg.rows


def test_active_set_compaction_is_exact():
    # With early stopping each sweep runs on the rows still active, compacted.
    # Every row's computation depends on that row alone, so running the layer
    # in three uneven chunks (each compacting at its own times, each row at a
    # different position) must give bit-identical codes and scales.  Rows stop
    # at spread-out sweeps here (300 active for three sweeps, 62 at the end).
    W, H, q, s, z = random_layer(300, 512, 64, 3, seed=7)
    K, tau = 8, 1e-5
    st, qf, sf = _check_stopping_run(W, H, q, s, z, 64, 3, K, tau, " compaction")
    assert st["rows_active"][0] == 300 and st["rows_active"][-1] < 150
    for lo, hi in ((0, 97), (97, 228), (228, 300)):
        part = GpuLayer(W[lo:hi], H, q[lo:hi], s[lo:hi], z[lo:hi], 64, 3, sweeps=K, tau=tau)
        jq.sweeps(part.p, part.W, part.H, part.codes, part.scales, part.zeros, part.ws)
        qp, sp = part.state()
        assert np.array_equal(qp, qf[lo:hi]), (lo, hi)
        assert np.array_equal(sp.view(np.uint32), sf[lo:hi].view(np.uint32)), (lo, hi)


# --------------------------------------------------------------------------
# shapes: ragged row tiles, every group size, several bit widths
# --------------------------------------------------------------------------

@pytest.mark.parametrize("rows,cols,g,bits", [
    (37, 96, 32, 2), (50, 192, 64, 4), (129, 384, 128, 3), (16, 128, 128, 8),
    (1, 64, 32, 1), (200, 256, 64, 3), (65, 640, 128, 4)])
def test_shapes(rows, cols, g, bits):
    W, H, q, s, z = random_layer(rows, cols, g, bits, seed=rows * 7 + cols + bits)
    say(f"[shape] rows {rows} cols {cols} g {g} bits {bits}")
    gl = GpuLayer(W, H, q, s, z, g, bits)
    F = gl.objective()
    F_ref = jarq.objective_rows(W, H, q, s, z, g)
    assert np.all(np.abs(F - F_ref) <= OBJ_RTOL * F_ref)
    R = jarq.group_factors(H, g)
    for sweep in range(2):
        q_before, _ = gl.state()
        gl.scale_step()
        q0, s1 = gl.state()
        assert np.array_equal(q0, q_before)
        s_ref, _ = jarq.scale_step(W, H, q0, z, g)
        check_scales(s1, s_ref, f" {rows}x{cols} sweep {sweep + 1}")
        cand, dec = gl.code_step()
        check_code_step(W, H, R, q0, s1, z, g, bits, cand, dec, f" {rows}x{cols} sweep {sweep + 1}")
    K = 4
    gk = GpuLayer(W, H, q, s, z, g, bits, sweeps=K)
    jq.sweeps(gk.p, gk.W, gk.H, gk.codes, gk.scales, gk.zeros, gk.ws)
    qg, sg = gk.state()
    qo, so, _ = jarq.refine(W, H, q, s, z, g, bits, K)
    F_gpu = jarq.objective_rows(W, H, qg, sg, z, g).sum()
    F_or = jarq.objective_rows(W, H, qo, so, z, g).sum()
    say(f"[shape e2e] rel {rel(F_gpu, F_or):.2e} agreement {np.mean(qg == qo):.6f}")
    assert rel(F_gpu, F_or) <= OBJ_RTOL


def test_widest_accepted_layer():
    """The most columns a layer may have: 128 groups of 128 (16384 columns).

    H is the AR(1) covariance 0.5^|i-j| plus damping (closed form, so no token
    build is needed at this width); 48 rows (a ragged row tile).  One sweep is
    checked teacher-forced; two sweeps end to end against the oracle deferring
    to the GPU only inside the bands (as for the full-size layers), with the
    free-running oracle reported.
    """
    from scipy.linalg import toeplitz
    rows, cols, g, bits = 48, 16384, 128, 3
    H = toeplitz(0.5 ** np.arange(cols)).astype(np.float32)
    H += np.float32(0.01) * np.eye(cols, dtype=np.float32)
    rng = np.random.default_rng(16384)
    W = (0.02 * rng.standard_normal((rows, cols))).astype(np.float32)
    q, s, z = rtn_quantize(W, g, bits)
    say(f"[widest] rows {rows} cols {cols} g {g} bits {bits}")
    gl = GpuLayer(W, H, q, s, z, g, bits)
    R = jarq.group_factors(H, g)
    q0, _ = gl.state()
    gl.scale_step()
    q1, s1 = gl.state()
    assert np.array_equal(q0, q1)
    s_ref, _ = jarq.scale_step(W, H, q0, z, g)
    check_scales(s1, s_ref, " widest sweep 1")
    cand, dec = gl.code_step()
    check_code_step(W, H, R, q0, s1, z, g, bits, cand, dec, " widest sweep 1")
    del gl
    K = 2
    tr = GpuLayer(W, H, q, s, z, g, bits)
    cands, decs, states = traced_sweeps(tr, K)
    del tr
    gk = GpuLayer(W, H, q, s, z, g, bits, sweeps=K)
    jq.sweeps(gk.p, gk.W, gk.H, gk.codes, gk.scales, gk.zeros, gk.ws)
    qg, sg = gk.state()
    del gk
    torch.cuda.empty_cache()
    # the benchmark's entry point and the step entry points agree bit for bit
    assert np.array_equal(qg, states[K][0]) and np.array_equal(sg, states[K][1])
    check_forced(W, H, R, q, s, z, g, bits, K, cands, decs, qg, sg, " widest")
    qo, so, _ = jarq.refine(W, H, q, s, z, g, bits, K, R=R)
    F_gpu = jarq.objective_rows(W, H, qg, sg, z, g).sum()
    F_or = jarq.objective_rows(W, H, qo, so, z, g).sum()
    say(f"[widest e2e] free-running oracle: F rel {rel(F_gpu, F_or):.2e} "
        f"(gpu {'lower' if F_gpu <= F_or else 'higher'}), code agreement {np.mean(qg == qo):.6f}")


# --------------------------------------------------------------------------
# degenerate cases of the method
# --------------------------------------------------------------------------

def test_ridge_branch_matches_oracle():
    W, H, q, s, z = random_layer(40, 256, 64, 3, seed=5)
    q = q.copy()
    q[3, 64:128] = z[3, 1]           # group 1 of row 3 all at its zero point: B_j rank deficient
    q[17, 0:64] = z[17, 0]
    gl = GpuLayer(W, H, q, s, z, 64, 3, sweeps=1)
    gl.scale_step()
    _, s_gpu = gl.state()
    s_ref, ridge = jarq.scale_step(W, H, q, z, 64)
    assert ridge[3] and ridge[17] and ridge.sum() == 2
    check_scales(s_gpu, s_ref, " ridge")
    assert s_gpu[3, 1] == 0.0 and s_gpu[17, 0] == 0.0
    g2 = GpuLayer(W, H, q, s, z, 64, 3, sweeps=1)
    st = jq.sweeps(g2.p, g2.W, g2.H, g2.codes, g2.scales, g2.zeros, g2.ws)
    assert st["ridge_rows"][0] == 2


def _near_singular_layer(rows, cols, g, kahan_rows, seed):
    """Rows in kahan_rows get a nearly singular Gram matrix whose Cholesky pivots are all 1.

    H = E K E^T + D: K = R^T R (R unit upper triangular, -1 above the
    diagonal: every pivot 1, smallest eigenvalue below 1e-10 of the largest
    from G = 16 on) on the first weight of every group, D = 1 on every other
    weight.  A row whose codes minus zero points are 1 on each group's first
    weight and 0 elsewhere has Gram matrix K exactly (eq. (5)); the other rows
    have random codes and well-conditioned Gram matrices.  The first weights
    of W are multiples of 1/8, so W H and every right-hand side are exact."""
    rng = np.random.default_rng(seed)
    G = cols // g
    R = np.eye(G) + np.triu(-np.ones((G, G)), 1)
    first = np.arange(G) * g
    H = np.eye(cols)
    H[first, first] = 0.0
    H[np.ix_(first, first)] = R.T @ R
    W = 0.02 * rng.standard_normal((rows, cols))
    W[:, first] = rng.integers(-8, 9, size=(rows, G)) / 8.0
    W = W.astype(np.float32)
    q, s, z = rtn_quantize(W, g, 3)
    q, z = q.copy(), z.copy()
    for j in kahan_rows:
        z[j] = 3
        q[j] = 3
        q[j, first] = 4
    return W, np.ascontiguousarray(H.astype(np.float32)), q, s, z


@pytest.mark.parametrize("cols,g", [(512, 32), (1024, 32), (4608, 64), (3200, 32), (3840, 32)])
def test_ridge_trigger_on_large_pivots_matches_oracle(cols, g):
    # G = 16 and 32 (register solve, two rows per wavefront: rows 1 and 6
    # share theirs with a well-conditioned row), 72 and 100 (tile solve), 120
    # (LDS solve).  The pivot test alone would miss rows 1 and 6; the
    # eigenvalue bound and the factorisation of A - t I must catch them.
    W, H, q, s, z = _near_singular_layer(8, cols, g, (1, 6), seed=cols)
    gl = GpuLayer(W, H, q, s, z, g, 3)
    gl.scale_step()
    _, s_gpu = gl.state()
    s_ref, ridge = jarq.scale_step(W, H, q, z, g)
    assert list(np.nonzero(ridge)[0]) == [1, 6]
    check_scales(s_gpu, s_ref, f" near-singular G {cols // g}")
    g2 = GpuLayer(W, H, q, s, z, g, 3, sweeps=1)
    st = jq.sweeps(g2.p, g2.W, g2.H, g2.codes, g2.scales, g2.zeros, g2.ws)
    assert st["ridge_rows"][0] == 2


@pytest.mark.parametrize("cols,g", [(256, 64), (4608, 64)])
def test_ridge_acceptance_matches_oracle(cols, g):
    # Rows 3 and 17 have a group at its zero point (rank-deficient B_j).  With H
    # scaled by 1e-8 the ridge term dominates and the ridge solution raises F_j:
    # ridge acceptance keeps those rows' scales; unscaled, it keeps the ridge
    # solution.  G = 4 and G = 72 cover both solve kernels.
    W, H, q, s, z = random_layer(40, cols, g, 3, seed=5)
    q = q.copy()
    q[3, g:2 * g] = z[3, 1]
    q[17, 0:g] = z[17, 0]
    for h_scale, keeps_old in ((1e-8, True), (1.0, False)):
        Hs = np.ascontiguousarray((H.astype(np.float64) * h_scale).astype(np.float32))
        gl = GpuLayer(W, Hs, q, s, z, g, 3, ridge_accept=True)
        gl.scale_step()
        _, s_gpu = gl.state()
        s_ref, ridge = jarq.scale_step(W, Hs, q, z, g, prev=s)
        assert ridge[3] and ridge[17] and ridge.sum() == 2
        for j in (3, 17):
            assert np.array_equal(s_gpu[j], s[j]) == keeps_old, (h_scale, j)
        check_scales(s_gpu, s_ref, f" ridge accept h_scale {h_scale}")


def test_small_scale_groups_are_skipped():
    W, H, q, s, z = random_layer(20, 256, 64, 3, seed=6)
    gl = GpuLayer(W, H, q, s, z, 64, 3)
    gl.scale_step()
    s_t = gl.scales
    s_t[2, 1] = 1e-9
    s_t[5, 3] = 0.0
    q0, s1 = gl.state()
    cand, dec = gl.code_step()
    q1, _ = gl.state()
    assert dec[2, 1] == jq.DEC_SKIP and dec[5, 3] == jq.DEC_SKIP
    assert np.array_equal(q1[2, 64:128], q0[2, 64:128])
    assert np.array_equal(q1[5, 192:256], q0[5, 192:256])
    check_code_step(W, H, jarq.group_factors(H, 64), q0, s1, z, 64, 3, cand, dec, " skip")


def test_failed_scale_solve_reports_and_keeps_scales():
    W, H, q, s, z = random_layer(24, 128, 64, 3, seed=7)
    H = H.copy()
    H[0, 64] = H[64, 0] = np.nan     # nonfinite coupling block: Gram nonfinite, ridge fails too
    gl = GpuLayer(W, H, q, s, z, 64, 3, sweeps=2)
    status, _ = jq.sweeps(gl.p, gl.W, gl.H, gl.codes, gl.scales, gl.zeros, gl.ws, check=False)
    assert status == jq.JARQ_ESCALE_SOLVE
    qg, sg = gl.state()
    assert np.array_equal(sg, s)


def test_not_spd_block_is_reported():
    W, H, q, s, z = random_layer(8, 128, 64, 3, seed=8)
    H = H.copy()
    H[70, 70] = -1.0
    gl = GpuLayer(W, H, q, s, z, 64, 3, prepare=False)
    with pytest.raises(jq.JarqError) as ei:
        jq.prepare(gl.p, gl.W, gl.H, gl.ws)
    assert ei.value.status == jq.JARQ_ENOT_SPD


def test_out_of_range_codes_are_rejected_untouched():
    W, H, q, s, z = random_layer(8, 128, 64, 3, seed=9)
    q = q.copy()
    q[4, 10] = 9
    gl = GpuLayer(W, H, q, s, z, 64, 3, sweeps=2)
    status, _ = jq.sweeps(gl.p, gl.W, gl.H, gl.codes, gl.scales, gl.zeros, gl.ws, check=False)
    assert status == jq.JARQ_EINVAL
    qg, sg = gl.state()
    assert np.array_equal(qg, q) and np.array_equal(sg, s)


# --------------------------------------------------------------------------
# full-size layers, checked on sampled rows
# --------------------------------------------------------------------------

@pytest.mark.parametrize("cfg_id", [1, 2, 3, 4])
def test_full_size_layer(cfg_id):
    """Every sweep of the benchmark's run, checked on a 128-row sample.

    The K sweeps run on the GPU over the whole layer one at a time with traces
    (the same kernels as jarq_sweeps).  For the sampled rows, each sweep's
    scales are compared with the oracle's scale step on the GPU's codes and each
    sweep's decisions are replayed by the oracle conditioned on the GPU's
    earlier decisions.  End to end, the oracle runs its own K iterations from
    the host state and defers to the GPU only at decisions inside the rounding
    and accept bands: it must reach the GPU's codes exactly and every sampled
    row's final objective within 1e-5 relative.  The free-running oracle
    (which leaves the GPU's trajectory at the first such decision) is
    reported for information.
    """
    cfg, W, H, q, s, z = layer(cfg_id)
    g, bits, K = cfg.group_size, cfg.bits, cfg.sweeps
    rng = np.random.default_rng(cfg_id)
    wide = np.unique(np.concatenate([[0, cfg.rows - 1], rng.choice(cfg.rows, 126, replace=False)]))
    R = jarq.group_factors(H, g)
    gl = GpuLayer(W, H, q, s, z, g, bits, sweeps=1)
    exempt = positions = 0
    cands, decs = [], []
    for k in range(K):
        qk, _ = gl.state()
        gl.scale_step()
        qk2, sk = gl.state()
        assert np.array_equal(qk, qk2)
        s_ref, _ = jarq.scale_step(W[wide], H, qk[wide], z[wide], g)
        check_scales(sk[wide], s_ref, f" cfg{cfg_id} sweep {k + 1}")
        cand, dec = gl.code_step()
        rep = check_code_step(W[wide], H, R, qk[wide], sk[wide], z[wide], g, bits, cand[wide],
                              dec[wide], f" cfg{cfg_id} sweep {k + 1}")
        cands.append(cand[wide].copy())
        decs.append(dec[wide].copy())
        exempt += rep.code_exempt + rep.decision_exempt
        positions += rep.n_codes
    qt, st_ = gl.state()
    del gl
    torch.cuda.empty_cache()
    # the benchmark's entry point reaches the same state
    gk = GpuLayer(W, H, q, s, z, g, bits, sweeps=K)
    st = jq.sweeps(gk.p, gk.W, gk.H, gk.codes, gk.scales, gk.zeros, gk.ws)
    qg, sg = gk.state()
    F_dev = gk.objective()
    assert np.array_equal(qg, qt) and np.array_equal(sg, st_)
    say(f"[cfg{cfg_id}] L per sweep {['%.6e' % v for v in st['objective_after_scales']]}")
    say(f"[cfg{cfg_id}] accepted {st['accepted_groups']} stage ms {st['stage_ms'][-1]} "
        f"Gram from the changed groups only {st['gram_listed']}")
    # the late sweeps rebuild only the changed groups' Gram entries, and the
    # state is bit-identical to the step entry points' full rebuilds (above)
    assert st["gram_listed"][0] == 0 and any(st["gram_listed"])
    del gk
    torch.cuda.empty_cache()
    # end to end on the GPU's trajectory: the oracle deferring only inside the bands
    check_forced(W[wide], H, R, q[wide], s[wide], z[wide], g, bits, K, cands, decs,
                 qg[wide], sg[wide], f" cfg{cfg_id}")
    F_gpu = jarq.objective_rows(W[wide], H, qg[wide], sg[wide], z[wide], g)
    # free-running oracle on the same rows, for information
    qo, so, _ = jarq.refine(W[wide], H, q[wide], s[wide], z[wide], g, bits, K, R=R)
    F_or = jarq.objective_rows(W[wide], H, qo, so, z[wide], g)
    same = np.all(qg[wide] == qo, axis=1)
    say(f"[cfg{cfg_id}] free-running oracle: {wide.size} rows, {int((~same).sum())} on another "
        f"trajectory (band exemptions over the {K} sweeps: {exempt} of {positions} positions); "
        f"F rel all rows {rel(F_gpu.sum(), F_or.sum()):.2e} "
        f"(gpu {'lower' if F_gpu.sum() <= F_or.sum() else 'higher'}), "
        f"agreeing rows {rel(F_gpu[same].sum(), F_or[same].sum()):.2e}")
    assert np.all(np.abs(F_dev[wide] - F_gpu) <= OBJ_RTOL * F_gpu)
    L = st["objective_after_scales"]
    assert all(L[k + 1] <= L[k] * (1 + 1e-6) for k in range(len(L) - 1))
