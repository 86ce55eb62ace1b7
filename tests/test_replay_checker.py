"""The teacher-forced replay accepts a correct trace and flags wrong decisions."""

import numpy as np

from oracle import jarq
from oracle.replay import replay_code_step
from tests.test_oracle_pins import build_tiny_layer


def _trace():
    cfg, W, H32, H64, A, codes, scales, zeros = build_tiny_layer()
    H = H32.astype(np.float64)
    g, bits = cfg.group_size, cfg.bits
    R = jarq.group_factors(H, g)
    s, _ = jarq.scale_step(W, H, codes, zeros, g)
    _, tr = jarq.code_step(W, H, R, codes, s, zeros, g, bits, record=True)
    return W, H, R, codes, s, zeros, g, bits, tr


def test_oracle_trace_replays_clean():
    W, H, R, q0, s, z, g, bits, tr = _trace()
    rep = replay_code_step(W, H, R, q0, s, z, g, bits, tr.cand, tr.decision)
    assert rep.ok and rep.code_exempt == 0 and rep.decision_exempt == 0
    assert rep.n_codes == q0.size and rep.n_groups == q0.shape[0] * (q0.shape[1] // g)


def test_planted_wrong_proposal_is_flagged():
    W, H, R, q0, s, z, g, bits, tr = _trace()
    cand = tr.cand.copy()
    # flip the last position of row 5, group 2 (evaluated first, far from a boundary)
    j, pos = 5, 2 * g + g - 1
    x = tr.x[j, pos]
    assert abs(x - np.floor(x) - 0.5) > 1e-3
    cand[j, pos] = (cand[j, pos] + 1) % (1 << bits)
    rep = replay_code_step(W, H, R, q0, s, z, g, bits, cand, tr.decision)
    assert rep.code_mismatch >= 1


def test_planted_wrong_decision_is_flagged():
    W, H, R, q0, s, z, g, bits, tr = _trace()
    dec = tr.decision.copy()
    j, i = np.argwhere(dec == jarq.DEC_ACCEPT)[0]
    dec[j, i] = jarq.DEC_REJECT
    rep = replay_code_step(W, H, R, q0, s, z, g, bits, tr.cand, dec)
    assert rep.decision_mismatch >= 1
    dec2 = tr.decision.copy()
    dec2[j, i] = jarq.DEC_SKIP
    rep2 = replay_code_step(W, H, R, q0, s, z, g, bits, tr.cand, dec2)
    assert rep2.skip_mismatch >= 1


# ---------------------------------------------------------------------------
# forced_refine: the oracle's own K iterations, deferring only inside the bands
# ---------------------------------------------------------------------------

from oracle.replay import forced_refine  # noqa: E402


def _traced_run(W, H, R, q, s, z, g, bits, K, scale_factor=1.0, tau=None):
    """K oracle iterations recording every sweep's proposals and decisions,
    optionally with every solved scale multiplied by scale_factor (a stand-in
    for an implementation whose scale solve is slightly off)."""
    cands, decs, states = [], [], [(q.copy(), s.copy())]
    for _ in range(K):
        s, _ = jarq.scale_step(W, H, q, z, g)
        s = s * scale_factor
        q, tr = jarq.code_step(W, H, R, q, s, z, g, bits, record=True)
        cands.append(tr.cand)
        decs.append(tr.decision)
        states.append((q.copy(), s.copy()))
    return cands, decs, states


def _tiny():
    cfg, W, H32, H64, A, codes, scales, zeros = build_tiny_layer()
    H = H32.astype(np.float64)
    return cfg, W, H, jarq.group_factors(H, cfg.group_size), codes, scales, zeros


def test_forced_refine_on_own_trace_is_the_oracle():
    cfg, W, H, R, q0, s0, z = _tiny()
    g, bits, K = cfg.group_size, cfg.bits, cfg.sweeps
    cands, decs, _ = _traced_run(W, H, R, q0, s0, z, g, bits, K)
    qf, sf, rep = forced_refine(W, H, q0, s0, z, g, bits, K, cands, decs, R=R)
    qo, so, _ = jarq.refine(W, H, q0, s0, z, g, bits, K, R=R)
    assert rep.ok and rep.code_forced == 0 and rep.decision_forced == 0
    assert rep.n_codes == K * q0.size
    assert np.array_equal(qf, qo) and np.array_equal(sf, so)


def test_forced_refine_follows_a_slightly_perturbed_implementation():
    # An "other" implementation whose scales are 8e-6 too small (relative)
    # leaves the oracle's trajectory at a few decisions that lie close to a
    # rounding boundary; the forced run takes exactly those decisions and
    # ends on the other's codes, with the oracle's own scales.
    cfg, W, H, R, q0, s0, z = _tiny()
    g, bits, K = cfg.group_size, cfg.bits, cfg.sweeps
    cands, decs, states = _traced_run(W, H, R, q0, s0, z, g, bits, K, scale_factor=1 - 8e-6)
    q_other = states[-1][0]
    qo, so, _ = jarq.refine(W, H, q0, s0, z, g, bits, K, R=R)
    assert not np.array_equal(qo, q_other)           # free-running, the trajectories split
    qf, sf, rep = forced_refine(W, H, q0, s0, z, g, bits, K, cands, decs, R=R)
    assert rep.ok, rep
    assert rep.code_forced + rep.decision_forced >= 1
    assert np.array_equal(qf, q_other)
    F_other = jarq.objective_rows(W, H, q_other, states[-1][1], z, g).sum()
    F_forced = jarq.objective_rows(W, H, qf, sf, z, g).sum()
    assert abs(F_forced - F_other) <= 1e-5 * F_forced


def test_forced_refine_flags_a_wrong_decision_outside_the_band():
    cfg, W, H, R, q0, s0, z = _tiny()
    g, bits, K = cfg.group_size, cfg.bits, cfg.sweeps
    cands, decs, _ = _traced_run(W, H, R, q0, s0, z, g, bits, K)
    # an accepted group of the second sweep reported as rejected
    j, i = np.argwhere(decs[1] == jarq.DEC_ACCEPT)[0]
    decs = [d.copy() for d in decs]
    decs[1][j, i] = jarq.DEC_REJECT
    qf, _, rep = forced_refine(W, H, q0, s0, z, g, bits, K, cands, decs, R=R)
    assert rep.decision_mismatch >= 1 and not rep.ok
    # the oracle kept its own decision
    qo, _, _ = jarq.refine(W, H, q0, s0, z, g, bits, K, R=R)
    assert np.array_equal(qf, qo)


def test_forced_refine_flags_a_wrong_proposal_outside_the_band():
    cfg, W, H, R, q0, s0, z = _tiny()
    g, bits, K = cfg.group_size, cfg.bits, cfg.sweeps
    cands, decs, _ = _traced_run(W, H, R, q0, s0, z, g, bits, K)
    cands = [c.copy() for c in cands]
    j, pos = 7, 3 * g + g - 1                 # the first position evaluated in group 3, sweep 3
    cands[2][j, pos] = (cands[2][j, pos] + 1) % (1 << bits)
    _, _, rep = forced_refine(W, H, q0, s0, z, g, bits, K, cands, decs, R=R)
    assert rep.code_mismatch >= 1 and not rep.ok


def test_forced_refine_stopping():
    cfg, W, H, R, q0, s0, z = _tiny()
    g, bits, K, tau = cfg.group_size, cfg.bits, 8, 1e-5
    cands, decs, _ = _traced_run(W, H, R, q0, s0, z, g, bits, K)
    qo, so, hist = jarq.refine(W, H, q0, s0, z, g, bits, K, tau=tau, R=R)
    stop_at = np.zeros(cfg.rows, dtype=np.int64)
    was = np.ones(cfg.rows, dtype=bool)
    for k, h in enumerate(hist, start=1):
        stop_at[was & ~h.active] = k
        was = h.active.copy()
    assert np.count_nonzero(stop_at) >= 4
    qf, sf, rep = forced_refine(W, H, q0, s0, z, g, bits, K, cands, decs, tau=tau,
                                stop_at=stop_at, R=R)
    assert rep.ok and rep.stop_forced == 0 and rep.n_stops > 0
    assert np.array_equal(qf, qo) and np.array_equal(sf, so)
    assert [int(a.sum()) for a in rep.active] == [int(h.active.sum()) for h in hist]
    # a row reported as stopping one iteration late, far from the band, is flagged
    r = int(np.nonzero(stop_at)[0][0])
    late = stop_at.copy()
    late[r] += 1
    _, _, rep2 = forced_refine(W, H, q0, s0, z, g, bits, K, cands, decs, tau=tau,
                               stop_at=late, R=R)
    assert rep2.stop_mismatch >= 1


def test_stop_band_marks_only_decisions_near_tau():
    from oracle.replay import stop_band
    tau, l_tol = 1e-5, 1e-6
    L_prev = np.array([1.0, 1.0, 1.0, 1.0])
    L = np.array([1.0 - 1e-5, 1.0 - 1.0000005e-5, 1.0 - 2e-5, 1.0 - 1e-9])
    band = stop_band(L_prev, L, tau, l_tol)
    assert band.tolist() == [True, True, False, False]
