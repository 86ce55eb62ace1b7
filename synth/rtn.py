"""Asymmetric group-wise round-to-nearest host quantizer.

The paper's RTN host "rounds weights to the quantization grid" with
asymmetric group-wise quantization (Appendix A.1) and gives no formula.  The
reading used here is the usual min/max one, with 0 forced into each group's
range so the zero point lands in [0, 2^b - 1]:

    lo = min(min_group, 0), hi = max(max_group, 0)
    s  = (hi - lo) / (2^b - 1)            (s = 1 when hi == lo)
    z  = rint(-lo / s)
    q  = clip(rint(w / s) + z, 0, 2^b - 1)

The result is the host state (S0, Q0, Z) of eq. (1) that refinement starts
from; refinement never changes Z, the bit width or the groups.
"""

from __future__ import annotations

import numpy as np


def rtn_quantize(w: np.ndarray, group_size: int, bits: int):
    """Return (codes uint8 [rows, cols], scales float32 [rows, G], zeros int32 [rows, G])."""
    w = np.asarray(w, dtype=np.float64)
    rows, cols = w.shape
    if cols % group_size:
        raise ValueError("cols must be a multiple of group_size")
    qmax = (1 << bits) - 1
    G = cols // group_size
    wg = w.reshape(rows, G, group_size)
    lo = np.minimum(wg.min(axis=2), 0.0)
    hi = np.maximum(wg.max(axis=2), 0.0)
    s = (hi - lo) / qmax
    s = np.where(hi > lo, s, 1.0)
    # Store the scale in float32 first so codes are rounded on the stored grid.
    s32 = s.astype(np.float32)
    s64 = s32.astype(np.float64)
    z = np.rint(-lo / s64)
    z = np.clip(z, 0, qmax)
    q = np.clip(np.rint(wg / s64[:, :, None]) + z[:, :, None], 0, qmax)
    return (np.ascontiguousarray(q.reshape(rows, cols).astype(np.uint8)),
            np.ascontiguousarray(s32),
            np.ascontiguousarray(z.astype(np.int32)))
