"""ctypes binding of libjarq (include/jarq.h).

Argument marshalling only: every step of the refinement runs in the HIP
library.  torch provides device memory and the current stream.  Loading
fails loudly when the library has not been built.
"""

from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libjarq.so")

MAX_RECORDED_SWEEPS = 64
NUM_STAGES = 6           # Gram, scale solve, residual product, objective, Babai, panel update
STAGE_NAMES = ("gram", "solve", "residual", "objective", "babai", "panel")
ABI_VERSION = 9
(JARQ_OK, JARQ_EINVAL, JARQ_ENOT_SPD, JARQ_ESCALE_SOLVE, JARQ_EHIP, JARQ_EWORKSPACE,
 JARQ_ESTATIC_LIMIT) = range(7)
STATIC_WORKSPACE_BYTES = 512 << 20
DEC_REJECT, DEC_ACCEPT, DEC_SKIP, DEC_STOPPED = 0, 1, 2, 3


class JarqError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {status_string(status)} (status {status})")
        self.status = status


class Params(ctypes.Structure):
    _fields_ = [("rows", ctypes.c_int32), ("cols", ctypes.c_int32),
                ("group_size", ctypes.c_int32), ("bits", ctypes.c_int32),
                ("sweeps", ctypes.c_int32), ("tau", ctypes.c_float),
                ("ridge_lambda", ctypes.c_float), ("ridge_rcond", ctypes.c_float),
                ("ridge_accept", ctypes.c_int32)]


class Stats(ctypes.Structure):
    _fields_ = [("stage_mask", ctypes.c_uint32),
                ("sweeps_run", ctypes.c_int32), ("rows_active_end", ctypes.c_int32),
                ("objective_after_scales", ctypes.c_double * MAX_RECORDED_SWEEPS),
                ("accepted_groups", ctypes.c_int64 * MAX_RECORDED_SWEEPS),
                ("codes_changed", ctypes.c_int64 * MAX_RECORDED_SWEEPS),
                ("skipped_groups", ctypes.c_int64 * MAX_RECORDED_SWEEPS),
                ("ridge_rows", ctypes.c_int32 * MAX_RECORDED_SWEEPS),
                ("rows_active", ctypes.c_int32 * MAX_RECORDED_SWEEPS),
                ("correction_blocks", ctypes.c_int64 * MAX_RECORDED_SWEEPS),
                ("gram_listed", ctypes.c_int32 * MAX_RECORDED_SWEEPS),
                ("stage_ms", (ctypes.c_float * NUM_STAGES) * MAX_RECORDED_SWEEPS),
                ("prep_ms", ctypes.c_float)]

    def to_dict(self):
        n = min(self.sweeps_run, MAX_RECORDED_SWEEPS)
        return {
            "stage_mask": self.stage_mask,
            "sweeps_run": self.sweeps_run,
            "rows_active_end": self.rows_active_end,
            "objective_after_scales": [self.objective_after_scales[k] for k in range(n)],
            "accepted_groups": [self.accepted_groups[k] for k in range(n)],
            "codes_changed": [self.codes_changed[k] for k in range(n)],
            "skipped_groups": [self.skipped_groups[k] for k in range(n)],
            "ridge_rows": [self.ridge_rows[k] for k in range(n)],
            "rows_active": [self.rows_active[k] for k in range(n)],
            "correction_blocks": [self.correction_blocks[k] for k in range(n)],
            "gram_listed": [self.gram_listed[k] for k in range(n)],
            "stage_ms": [list(self.stage_ms[k]) for k in range(n)],
            "prep_ms": self.prep_ms,
        }


_vp = ctypes.c_void_p
_SIGNATURES = {
    "jarq_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(Params)]),
    "jarq_prepare": (ctypes.c_int, [ctypes.POINTER(Params), _vp, _vp, _vp, ctypes.c_size_t, _vp]),
    "jarq_scale_step": (ctypes.c_int, [ctypes.POINTER(Params), _vp, _vp, _vp, _vp, _vp,
                                       ctypes.c_size_t, _vp]),
    "jarq_code_step": (ctypes.c_int, [ctypes.POINTER(Params), _vp, _vp, _vp, _vp, _vp, _vp,
                                      ctypes.c_size_t, _vp, _vp, _vp]),
    "jarq_sweeps": (ctypes.c_int, [ctypes.POINTER(Params), _vp, _vp, _vp, _vp, _vp, _vp,
                                   ctypes.c_size_t, _vp, ctypes.POINTER(Stats)]),
    "jarq_refine": (ctypes.c_int, [ctypes.POINTER(Params), _vp, _vp, _vp, _vp, _vp, _vp,
                                   ctypes.c_size_t, _vp, ctypes.POINTER(Stats)]),
    "jarq_refine_static": (ctypes.c_int, [ctypes.POINTER(Params), _vp, _vp, _vp, _vp, _vp, _vp,
                                          ctypes.POINTER(Stats)]),
    "jarq_objective": (ctypes.c_int, [ctypes.POINTER(Params), _vp, _vp, _vp, _vp, _vp, _vp,
                                      ctypes.c_size_t, _vp, _vp]),
    "jarq_stop_sweeps": (ctypes.c_int, [ctypes.POINTER(Params), _vp, ctypes.c_size_t, _vp, _vp]),
    "jarq_hessian_accumulate": (ctypes.c_int, [_vp, ctypes.c_int64, ctypes.c_int32, ctypes.c_double,
                                               _vp, _vp]),
    "jarq_hessian_accumulate_bf16": (ctypes.c_int, [_vp, ctypes.c_int64, ctypes.c_int32,
                                                    ctypes.c_double, _vp, _vp]),
    "jarq_hessian_finalize": (ctypes.c_int, [_vp, ctypes.c_int32, ctypes.c_double, ctypes.c_double,
                                             _vp, _vp]),
    "jarq_rtn": (ctypes.c_int, [ctypes.POINTER(Params), _vp, _vp, _vp, _vp, _vp]),
    "jarq_cross_accumulate": (ctypes.c_int, [_vp, _vp, ctypes.c_int64, ctypes.c_int32,
                                             ctypes.c_double, _vp, _vp]),
    "jarq_qep_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(Params)]),
    "jarq_qep_correct": (ctypes.c_int, [ctypes.POINTER(Params), _vp, _vp, _vp, ctypes.c_double,
                                        _vp, _vp, ctypes.c_size_t, _vp]),
    "jarq_canonicalize": (ctypes.c_int, [ctypes.POINTER(Params), _vp, _vp, _vp, _vp]),
    "jarq_dequantize": (ctypes.c_int, [ctypes.POINTER(Params), _vp, _vp, _vp, _vp, ctypes.c_int32,
                                       _vp, _vp]),
    "jarq_pack_codes": (ctypes.c_int, [ctypes.POINTER(Params), _vp, _vp, _vp]),
    "jarq_unpack_codes": (ctypes.c_int, [ctypes.POINTER(Params), _vp, _vp, _vp]),
    "jarq_act_order": (ctypes.c_int, [_vp, ctypes.c_int32, _vp, _vp]),
    "jarq_permute": (ctypes.c_int, [ctypes.POINTER(Params), _vp, _vp, _vp, _vp, _vp, _vp]),
    "jarq_gptq_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(Params)]),
    "jarq_gptq": (ctypes.c_int, [ctypes.POINTER(Params), _vp, _vp, _vp, _vp, _vp, _vp,
                                 ctypes.c_size_t, _vp]),
    "jarq_lds_probe": (ctypes.c_int64, [ctypes.c_int32, ctypes.c_int32, _vp, _vp]),
    "jarq_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "jarq_abi_version": (ctypes.c_int32, []),
}
EXPORTED = tuple(_SIGNATURES)

_lib = None


def load_library(path: str = LIB_PATH):
    """Load libjarq.so; raises ImportError if it is missing (no fallback exists)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"libjarq.so not built at {path}; run paper_2609_38599_amd/build.py")
    lib = ctypes.CDLL(path)
    for name, (res, args) in _SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    if lib.jarq_abi_version() != ABI_VERSION:
        raise ImportError(f"{path} has ABI version {lib.jarq_abi_version()}, this binding expects "
                          f"{ABI_VERSION}; rebuild with paper_2609_38599_amd/build.py")
    _lib = lib
    return lib


def status_string(status: int) -> str:
    return load_library().jarq_status_string(int(status)).decode()


def make_params(rows, cols, group_size, bits, sweeps=1, tau=-1.0, ridge_lambda=1e-4,
                ridge_rcond=1e-10, ridge_accept=False) -> Params:
    return Params(int(rows), int(cols), int(group_size), int(bits), int(sweeps), float(tau),
                  float(ridge_lambda), float(ridge_rcond), int(bool(ridge_accept)))


def workspace_bytes(p: Params) -> int:
    return int(load_library().jarq_workspace_bytes(ctypes.byref(p)))


def alloc_workspace(p: Params, device=None) -> torch.Tensor:
    n = workspace_bytes(p)
    if n == 0:
        raise JarqError(JARQ_EINVAL, "workspace_bytes")
    ws = torch.empty(n + 256, dtype=torch.uint8, device=device or "cuda")
    off = (-ws.data_ptr()) % 256
    return ws[off:off + n]


def _ptr(t, dtype, name):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _check(status, what):
    if status != JARQ_OK:
        raise JarqError(status, what)


def prepare(p: Params, W, H, ws, stream=None):
    lib = load_library()
    _check(lib.jarq_prepare(ctypes.byref(p), _ptr(W, torch.float32, "W"),
                            _ptr(H, torch.float32, "H"), _ptr(ws, torch.uint8, "workspace"),
                            ws.numel(), _stream(stream)), "jarq_prepare")


def scale_step(p: Params, H, codes, scales, zeros, ws, stream=None):
    lib = load_library()
    _check(lib.jarq_scale_step(ctypes.byref(p), _ptr(H, torch.float32, "H"),
                               _ptr(codes, torch.uint8, "codes"),
                               _ptr(scales, torch.float32, "scales"),
                               _ptr(zeros, torch.int32, "zeros"),
                               _ptr(ws, torch.uint8, "workspace"), ws.numel(), _stream(stream)),
           "jarq_scale_step")


def code_step(p: Params, W, H, codes, scales, zeros, ws, cand=None, decision=None, stream=None):
    lib = load_library()
    _check(lib.jarq_code_step(ctypes.byref(p), _ptr(W, torch.float32, "W"),
                              _ptr(H, torch.float32, "H"), _ptr(codes, torch.uint8, "codes"),
                              _ptr(scales, torch.float32, "scales"),
                              _ptr(zeros, torch.int32, "zeros"),
                              _ptr(ws, torch.uint8, "workspace"), ws.numel(), _stream(stream),
                              _ptr(cand, torch.uint8, "cand"),
                              _ptr(decision, torch.uint8, "decision")), "jarq_code_step")


def sweeps(p: Params, W, H, codes, scales, zeros, ws, stream=None, want_stats=True, check=True,
           stage_mask=0):
    """jarq_sweeps; stage_mask selects the stages timed with HIP events (0 = all)."""
    lib = load_library()
    st = Stats() if want_stats else None
    if st is not None:
        st.stage_mask = stage_mask
    status = lib.jarq_sweeps(ctypes.byref(p), _ptr(W, torch.float32, "W"),
                             _ptr(H, torch.float32, "H"), _ptr(codes, torch.uint8, "codes"),
                             _ptr(scales, torch.float32, "scales"),
                             _ptr(zeros, torch.int32, "zeros"),
                             _ptr(ws, torch.uint8, "workspace"), ws.numel(), _stream(stream),
                             ctypes.byref(st) if st is not None else None)
    if check:
        _check(status, "jarq_sweeps")
    return (st.to_dict() if st is not None else None) if check else (status, st)


def refine(p: Params, W, H, codes, scales, zeros, ws, stream=None, want_stats=True, check=True,
           stage_mask=0):
    lib = load_library()
    st = Stats() if want_stats else None
    if st is not None:
        st.stage_mask = stage_mask
    status = lib.jarq_refine(ctypes.byref(p), _ptr(W, torch.float32, "W"),
                             _ptr(H, torch.float32, "H"), _ptr(codes, torch.uint8, "codes"),
                             _ptr(scales, torch.float32, "scales"),
                             _ptr(zeros, torch.int32, "zeros"),
                             _ptr(ws, torch.uint8, "workspace"), ws.numel(), _stream(stream),
                             ctypes.byref(st) if st is not None else None)
    if check:
        _check(status, "jarq_refine")
    return (st.to_dict() if st is not None else None) if check else (status, st)


def refine_static(p: Params, W, H, codes, scales, zeros, stream=None, want_stats=True,
                  check=True):
    """jarq_refine_static: jarq_refine on the library's static workspace (no allocation)."""
    lib = load_library()
    st = Stats() if want_stats else None
    status = lib.jarq_refine_static(ctypes.byref(p), _ptr(W, torch.float32, "W"),
                                    _ptr(H, torch.float32, "H"), _ptr(codes, torch.uint8, "codes"),
                                    _ptr(scales, torch.float32, "scales"),
                                    _ptr(zeros, torch.int32, "zeros"), _stream(stream),
                                    ctypes.byref(st) if st is not None else None)
    if check:
        _check(status, "jarq_refine_static")
    return (st.to_dict() if st is not None else None) if check else (status, st)


def objective(p: Params, W, H, codes, scales, zeros, ws, out=None, stream=None):
    lib = load_library()
    if out is None:
        out = torch.empty(p.rows, dtype=torch.float64, device=W.device)
    _check(lib.jarq_objective(ctypes.byref(p), _ptr(W, torch.float32, "W"),
                              _ptr(H, torch.float32, "H"), _ptr(codes, torch.uint8, "codes"),
                              _ptr(scales, torch.float32, "scales"),
                              _ptr(zeros, torch.int32, "zeros"),
                              _ptr(ws, torch.uint8, "workspace"), ws.numel(), _stream(stream),
                              _ptr(out, torch.float64, "row_objective")), "jarq_objective")
    return out


def stop_sweeps(p: Params, ws, out=None, stream=None):
    """Per row, the iteration at which the last sweeps call stopped it (0 = never)."""
    lib = load_library()
    if out is None:
        out = torch.empty(p.rows, dtype=torch.int32, device=ws.device)
    _check(lib.jarq_stop_sweeps(ctypes.byref(p), _ptr(ws, torch.uint8, "workspace"), ws.numel(),
                                _ptr(out, torch.int32, "stop_sweep"), _stream(stream)),
           "jarq_stop_sweeps")
    return out


def hessian_accumulate(X, Hacc, alpha=1.0, stream=None):
    """Hacc += alpha X^T X for one chunk X [m, d] fp32 or bf16 (Hacc [d, d] fp64)."""
    lib = load_library()
    if X.dim() != 2 or Hacc.shape != (X.shape[1], X.shape[1]):
        raise ValueError("X must be [m, d] and Hacc [d, d]")
    if X.dtype == torch.bfloat16:
        _check(lib.jarq_hessian_accumulate_bf16(_ptr(X, torch.bfloat16, "X"), X.shape[0],
                                                X.shape[1], float(alpha),
                                                _ptr(Hacc, torch.float64, "Hacc"), _stream(stream)),
               "jarq_hessian_accumulate_bf16")
        return
    _check(lib.jarq_hessian_accumulate(_ptr(X, torch.float32, "X"), X.shape[0], X.shape[1],
                                       float(alpha), _ptr(Hacc, torch.float64, "Hacc"),
                                       _stream(stream)), "jarq_hessian_accumulate")


def hessian_finalize(Hacc, damp=0.0, nu2=0.0, out=None, stream=None):
    """H = Hacc + (damp mean(diag Hacc) + nu2) I as fp32."""
    lib = load_library()
    d = Hacc.shape[0]
    if Hacc.dim() != 2 or Hacc.shape[1] != d:
        raise ValueError("Hacc must be square")
    if out is None:
        out = torch.empty(d, d, dtype=torch.float32, device=Hacc.device)
    _check(lib.jarq_hessian_finalize(_ptr(Hacc, torch.float64, "Hacc"), d, float(damp),
                                     float(nu2), _ptr(out, torch.float32, "H"), _stream(stream)),
           "jarq_hessian_finalize")
    return out


def hessian(chunks, d, alpha=1.0, damp=0.0, nu2=0.0, device=None, stream=None):
    """The fp32 Hessian of a stream of fp32 device chunks [m_c, d]."""
    Hacc = torch.zeros(d, d, dtype=torch.float64, device=device or "cuda")
    for X in chunks:
        hessian_accumulate(X, Hacc, alpha, stream)
    return hessian_finalize(Hacc, damp, nu2, stream=stream)


def rtn(p: Params, W, codes=None, scales=None, zeros=None, stream=None):
    """Round-to-nearest host state (codes, scales, zeros) of W."""
    lib = load_library()
    G = p.cols // p.group_size
    dev = W.device
    if codes is None:
        codes = torch.empty(p.rows, p.cols, dtype=torch.uint8, device=dev)
    if scales is None:
        scales = torch.empty(p.rows, G, dtype=torch.float32, device=dev)
    if zeros is None:
        zeros = torch.empty(p.rows, G, dtype=torch.int32, device=dev)
    _check(lib.jarq_rtn(ctypes.byref(p), _ptr(W, torch.float32, "W"),
                        _ptr(codes, torch.uint8, "codes"), _ptr(scales, torch.float32, "scales"),
                        _ptr(zeros, torch.int32, "zeros"), _stream(stream)), "jarq_rtn")
    return codes, scales, zeros


DTYPES = {torch.float32: 0, torch.float16: 1, torch.bfloat16: 2}


def canonicalize(p: Params, codes, scales, zeros, stream=None):
    """In place: groups with a negative scale get s' = -s, q' = qmax - q, z' = qmax - z."""
    lib = load_library()
    _check(lib.jarq_canonicalize(ctypes.byref(p), _ptr(codes, torch.uint8, "codes"),
                                 _ptr(scales, torch.float32, "scales"),
                                 _ptr(zeros, torch.int32, "zeros"), _stream(stream)),
           "jarq_canonicalize")


def dequantize(p: Params, codes, scales, zeros, dtype=torch.float32, perm=None, out=None,
               stream=None):
    """s (q - z) as `dtype`; with perm, written back in the original column order."""
    lib = load_library()
    if out is None:
        out = torch.empty(p.rows, p.cols, dtype=dtype, device=codes.device)
    _check(lib.jarq_dequantize(ctypes.byref(p), _ptr(codes, torch.uint8, "codes"),
                               _ptr(scales, torch.float32, "scales"),
                               _ptr(zeros, torch.int32, "zeros"), _ptr(perm, torch.int32, "perm"),
                               DTYPES[out.dtype], _ptr(out, out.dtype, "out"), _stream(stream)),
           "jarq_dequantize")
    return out


def packed_words_per_row(p: Params) -> int:
    return (p.cols * p.bits + 31) // 32


def pack_codes(p: Params, codes, out=None, stream=None):
    lib = load_library()
    if out is None:
        out = torch.empty(p.rows, packed_words_per_row(p), dtype=torch.int32, device=codes.device)
    _check(lib.jarq_pack_codes(ctypes.byref(p), _ptr(codes, torch.uint8, "codes"),
                               _ptr(out, torch.int32, "packed"), _stream(stream)),
           "jarq_pack_codes")
    return out


def unpack_codes(p: Params, packed, out=None, stream=None):
    lib = load_library()
    if out is None:
        out = torch.empty(p.rows, p.cols, dtype=torch.uint8, device=packed.device)
    _check(lib.jarq_unpack_codes(ctypes.byref(p), _ptr(packed, torch.int32, "packed"),
                                 _ptr(out, torch.uint8, "codes"), _stream(stream)),
           "jarq_unpack_codes")
    return out


def act_order(H, out=None, stream=None):
    lib = load_library()
    d = H.shape[0]
    if out is None:
        out = torch.empty(d, dtype=torch.int32, device=H.device)
    _check(lib.jarq_act_order(_ptr(H, torch.float32, "H"), d, _ptr(out, torch.int32, "perm"),
                              _stream(stream)), "jarq_act_order")
    return out


def permute(p: Params, perm, W, H, stream=None):
    lib = load_library()
    Wp, Hp = torch.empty_like(W), torch.empty_like(H)
    _check(lib.jarq_permute(ctypes.byref(p), _ptr(perm, torch.int32, "perm"),
                            _ptr(W, torch.float32, "W"), _ptr(H, torch.float32, "H"),
                            _ptr(Wp, torch.float32, "Wp"), _ptr(Hp, torch.float32, "Hp"),
                            _stream(stream)), "jarq_permute")
    return Wp, Hp


def _scratch(n, dev):
    raw = torch.empty(n + 256, dtype=torch.uint8, device=dev)
    off = (-raw.data_ptr()) % 256
    return raw[off:off + n]


def cross_accumulate(Xq, X, Dacc, alpha=1.0, stream=None):
    """Dacc += alpha Xq^T (X - Xq) for one chunk of tokens (Dacc [d, d] fp64)."""
    lib = load_library()
    if Xq.shape != X.shape or Xq.dim() != 2 or Dacc.shape != (X.shape[1], X.shape[1]):
        raise ValueError("Xq and X must be [m, d] and Dacc [d, d]")
    _check(lib.jarq_cross_accumulate(_ptr(Xq, torch.float32, "Xq"), _ptr(X, torch.float32, "X"),
                                     X.shape[0], X.shape[1], float(alpha),
                                     _ptr(Dacc, torch.float64, "Dacc"), _stream(stream)),
           "jarq_cross_accumulate")


def qep_correct(p: Params, W, H, D, mu, out=None, ws=None, stream=None):
    """W_corr = W + (1 - mu) (W D^T) H^{-1} (fp32)."""
    lib = load_library()
    if out is None:
        out = torch.empty_like(W)
    n = int(lib.jarq_qep_workspace_bytes(ctypes.byref(p)))
    if n == 0:
        raise JarqError(JARQ_EINVAL, "jarq_qep_workspace_bytes")
    if ws is None:
        ws = _scratch(n, W.device)
    _check(lib.jarq_qep_correct(ctypes.byref(p), _ptr(W, torch.float32, "W"),
                                _ptr(H, torch.float32, "H"), _ptr(D, torch.float64, "D"),
                                float(mu), _ptr(out, torch.float32, "Wcorr"),
                                _ptr(ws, torch.uint8, "workspace"), ws.numel(), _stream(stream)),
           "jarq_qep_correct")
    return out


def gptq(p: Params, W, H, codes=None, scales=None, zeros=None, ws=None, stream=None):
    """GPTQ-style host state (codes, scales, zeros) of W under H."""
    lib = load_library()
    G = p.cols // p.group_size
    dev = W.device
    if codes is None:
        codes = torch.empty(p.rows, p.cols, dtype=torch.uint8, device=dev)
    if scales is None:
        scales = torch.empty(p.rows, G, dtype=torch.float32, device=dev)
    if zeros is None:
        zeros = torch.empty(p.rows, G, dtype=torch.int32, device=dev)
    n = int(lib.jarq_gptq_workspace_bytes(ctypes.byref(p)))
    if n == 0:
        raise JarqError(JARQ_EINVAL, "jarq_gptq_workspace_bytes")
    if ws is None:
        raw = torch.empty(n + 256, dtype=torch.uint8, device=dev)
        off = (-raw.data_ptr()) % 256
        ws = raw[off:off + n]
    _check(lib.jarq_gptq(ctypes.byref(p), _ptr(W, torch.float32, "W"), _ptr(H, torch.float32, "H"),
                         _ptr(codes, torch.uint8, "codes"), _ptr(scales, torch.float32, "scales"),
                         _ptr(zeros, torch.int32, "zeros"), _ptr(ws, torch.uint8, "workspace"),
                         ws.numel(), _stream(stream)), "jarq_gptq")
    return codes, scales, zeros


def lds_probe(workgroups, passes, out=None, stream=None):
    """Run the LDS calibration kernel; returns (LDS bytes moved, out)."""
    lib = load_library()
    if out is None:
        out = torch.empty(workgroups * 256, dtype=torch.float32, device="cuda")
    n = int(lib.jarq_lds_probe(int(workgroups), int(passes), _ptr(out, torch.float32, "out"),
                               _stream(stream)))
    if n < 0:
        raise JarqError(JARQ_EINVAL, "jarq_lds_probe")
    return n, out


def abi_version() -> int:
    return int(load_library().jarq_abi_version())
