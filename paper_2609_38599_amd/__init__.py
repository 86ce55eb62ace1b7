"""MI355X-native JARQ refinement sweep.

The per-layer hot path of JARQ (joint alternating refinement of a group-wise
quantized weight matrix against a calibration Hessian) as hand-written HIP for
gfx950 behind the C ABI of include/jarq.h, with a thin ctypes binding.
"""

from .binding import (DEC_ACCEPT, DEC_REJECT, DEC_SKIP, DEC_STOPPED, EXPORTED, JARQ_EHIP,
                      JARQ_EINVAL, JARQ_ENOT_SPD, JARQ_ESCALE_SOLVE, JARQ_EWORKSPACE, JARQ_OK,
                      LIB_PATH, MAX_RECORDED_SWEEPS, JarqError, Params, Stats, abi_version,
                      alloc_workspace, code_step, load_library, make_params, objective, prepare,
                      refine, scale_step, status_string, stop_sweeps, sweeps, workspace_bytes)

__all__ = [
    "DEC_ACCEPT", "DEC_REJECT", "DEC_SKIP", "DEC_STOPPED", "EXPORTED", "JARQ_EHIP",
    "JARQ_EINVAL", "JARQ_ENOT_SPD", "JARQ_ESCALE_SOLVE", "JARQ_EWORKSPACE", "JARQ_OK",
    "LIB_PATH", "MAX_RECORDED_SWEEPS", "JarqError", "Params", "Stats", "abi_version",
    "alloc_workspace", "code_step", "load_library", "make_params", "objective", "prepare",
    "refine", "scale_step", "status_string", "stop_sweeps", "sweeps", "workspace_bytes",
]
