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
