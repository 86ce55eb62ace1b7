"""The entry point that allocates nothing (jarq_refine_static) against jarq_refine.

Both run the same kernels; jarq_refine_static runs them on the library's
static device workspace.  Two calls in a row on one GPU, the second on a
smaller layer (with early stopping, so the stopping state left by the first
call must not leak), must each give codes and scales bit-identical to
jarq_refine on the same inputs.
"""

import numpy as np
import pytest
import torch

from tests._gpu_common import GpuLayer, jq, random_layer, say, to_dev

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]


def _reference(W, H, q, s, z, g, bits, K, tau):
    gl = GpuLayer(W, H, q, s, z, g, bits, sweeps=K, tau=tau, prepare=False)
    st = jq.refine(gl.p, gl.W, gl.H, gl.codes, gl.scales, gl.zeros, gl.ws)
    qg, sg = gl.state()
    return qg, sg, st


def _static(W, H, q, s, z, g, bits, K, tau):
    rows, cols = W.shape
    p = jq.make_params(rows, cols, g, bits, K, tau)
    Wd, Hd, qd, sd, zd = to_dev(W), to_dev(H), to_dev(q), to_dev(s), to_dev(z)
    st = jq.binding.refine_static(p, Wd, Hd, qd, sd, zd)
    torch.cuda.synchronize()
    return qd.cpu().numpy(), sd.cpu().numpy(), st


@pytest.mark.parametrize("order", ["large_then_small"])
def test_static_refine_matches_refine_on_two_calls(order):
    cases = [(300, 1024, 128, 3, 4, -1.0, 11),     # larger layer, every row active
             (37, 256, 64, 4, 6, 1e-5, 12),        # smaller layer, early stopping on
             # every row stops by sweep 6 of 40: jarq_refine ends the run when
             # its look at the active count (pinned memory, no wait) has landed,
             # jarq_refine_static with its blocking read; same results
             (48, 384, 128, 3, 40, 2e-4, 14)]
    for rows, cols, g, bits, K, tau, seed in cases:
        W, H, q, s, z = random_layer(rows, cols, g, bits, seed=seed)
        say(f"[no-alloc] rows {rows} cols {cols} g {g} bits {bits} K {K} tau {tau}")
        q_ref, s_ref, st_ref = _reference(W, H, q, s, z, g, bits, K, tau)
        q_st, s_st, st = _static(W, H, q, s, z, g, bits, K, tau)
        assert np.array_equal(q_st, q_ref)
        assert np.array_equal(s_st.view(np.uint32), s_ref.view(np.uint32))
        assert st["sweeps_run"] == st_ref["sweeps_run"]
        assert st["rows_active"] == st_ref["rows_active"]
        assert st["objective_after_scales"] == st_ref["objective_after_scales"]
        assert all(ms == 0.0 for row in st["stage_ms"] for ms in row)
        assert not np.array_equal(q_st, q)          # the call did refine the layer
        if K == 40:
            assert st["sweeps_run"] < K


def test_static_refine_rejects_a_layer_beyond_the_limit():
    p = jq.make_params(4096, 11008, 128, 3, 1)
    dummy = torch.zeros(64, dtype=torch.float32, device="cuda")
    codes = torch.zeros(64, dtype=torch.uint8, device="cuda")
    zeros = torch.zeros(64, dtype=torch.int32, device="cuda")
    status, _ = jq.binding.refine_static(p, dummy, dummy, codes, dummy, zeros, check=False)
    assert status == jq.binding.JARQ_ESTATIC_LIMIT
    torch.cuda.synchronize()
    assert int(codes.sum()) == 0
