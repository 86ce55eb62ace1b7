"""The C-ABI library loads and exports what include/jarq.h declares (CPU only).

Only calls that return before touching the GPU are made here: workspace
sizing, status strings, the ABI version and argument checks.
"""

import ctypes
import os
import re

import pytest

from paper_2609_38599_amd import binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "jarq.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(jarq_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    return binding.load_library()


def test_every_declared_symbol_is_exported(lib):
    names = _declared_functions()
    assert "jarq_refine" in names and "jarq_code_step" in names
    for name in names:
        assert hasattr(lib, name), name
        assert name in binding.EXPORTED, name


def test_abi_version_and_status_strings(lib):
    assert binding.abi_version() == binding.ABI_VERSION == 9
    for s in range(7):
        assert binding.status_string(s)
    assert binding.status_string(99) == "unknown status"


def test_workspace_bytes_valid_and_invalid():
    p = binding.make_params(4096, 4096, 128, 3, 10)
    n = binding.workspace_bytes(p)
    # W H, W M^T, P, the accepted changes, q - z and the fp16 planes of H, M
    # and E dominate
    assert 5 * 64 * 2**20 < n < 512 * 2**20
    for bad in [dict(rows=0), dict(cols=100), dict(group_size=48), dict(bits=0), dict(bits=9),
                dict(sweeps=-1), dict(cols=128 * 129), dict(ridge_lambda=-1.0)]:
        kw = dict(rows=64, cols=256, group_size=64, bits=3, sweeps=5)
        kw.update(bad)
        assert binding.workspace_bytes(binding.make_params(**kw)) == 0, bad


def _vp(x):
    return ctypes.c_void_p(x)


def test_argument_errors_return_before_any_launch(lib):
    p = binding.make_params(64, 256, 64, 3, 5)
    fake = _vp(1 << 20)          # aligned, never dereferenced: every call below fails its checks
    bad = binding.make_params(64, 250, 64, 3, 5)
    P = ctypes.POINTER(binding.Params)
    assert lib.jarq_prepare(ctypes.byref(bad), fake, fake, fake, 1 << 30, None) == binding.JARQ_EINVAL
    assert lib.jarq_prepare(ctypes.byref(p), None, fake, fake, 1 << 30, None) == binding.JARQ_EINVAL
    assert lib.jarq_prepare(ctypes.byref(p), _vp((1 << 20) + 4), fake, fake, 1 << 30, None) == binding.JARQ_EINVAL
    assert lib.jarq_prepare(ctypes.byref(p), fake, fake, None, 1 << 30, None) == binding.JARQ_EWORKSPACE
    assert lib.jarq_prepare(ctypes.byref(p), fake, fake, _vp((1 << 20) + 128), 1 << 30, None) == binding.JARQ_EWORKSPACE
    assert lib.jarq_prepare(ctypes.byref(p), fake, fake, fake, 1024, None) == binding.JARQ_EWORKSPACE
    assert lib.jarq_sweeps(ctypes.byref(p), fake, fake, _vp((1 << 20) + 2), fake, fake, fake, 1 << 30,
                           None, None) == binding.JARQ_EINVAL
    # codes are read and written 16 bytes at a time
    assert lib.jarq_sweeps(ctypes.byref(p), fake, fake, _vp((1 << 20) + 4), fake, fake, fake, 1 << 30,
                           None, None) == binding.JARQ_EINVAL
    assert lib.jarq_code_step(ctypes.byref(bad), fake, fake, fake, fake, fake, fake, 1 << 30, None,
                              None, None) == binding.JARQ_EINVAL
    assert lib.jarq_scale_step(ctypes.byref(p), fake, fake, _vp((1 << 20) + 8), fake, fake, 1 << 30,
                               None) == binding.JARQ_EINVAL
    assert lib.jarq_objective(ctypes.byref(p), fake, fake, fake, fake, fake, fake, 1 << 30, None,
                              None) == binding.JARQ_EINVAL
    assert lib.jarq_refine(None, fake, fake, fake, fake, fake, fake, 1 << 30, None, None) == binding.JARQ_EINVAL
    del P


def test_static_refine_rejects_before_any_launch(lib):
    fake = _vp(1 << 20)          # aligned, never dereferenced
    big = binding.make_params(4096, 11008, 128, 3, 10)
    assert binding.workspace_bytes(big) > binding.STATIC_WORKSPACE_BYTES
    assert lib.jarq_refine_static(ctypes.byref(big), fake, fake, fake, fake, fake, None,
                                  None) == binding.JARQ_ESTATIC_LIMIT
    bad = binding.make_params(64, 250, 64, 3, 5)
    assert lib.jarq_refine_static(ctypes.byref(bad), fake, fake, fake, fake, fake, None,
                                  None) == binding.JARQ_EINVAL
    p = binding.make_params(64, 256, 64, 3, 5)
    assert lib.jarq_refine_static(ctypes.byref(p), fake, fake, _vp((1 << 20) + 4), fake, fake,
                                  None, None) == binding.JARQ_EINVAL
    # the headline layer fits
    assert binding.workspace_bytes(binding.make_params(4096, 4096, 128, 3, 10)) <= \
        binding.STATIC_WORKSPACE_BYTES


def test_setup_entry_points_check_arguments(lib):
    fake = _vp(1 << 20)
    st = None
    acc = lib.jarq_hessian_accumulate
    assert acc(fake, 10, 130, 1.0, fake, st) == binding.JARQ_EINVAL          # d % 4
    assert acc(fake, -1, 128, 1.0, fake, st) == binding.JARQ_EINVAL          # m < 0
    assert acc(_vp((1 << 20) + 4), 10, 128, 1.0, fake, st) == binding.JARQ_EINVAL
    assert acc(fake, 10, 128, float("nan"), fake, st) == binding.JARQ_EINVAL
    assert acc(fake, 10, 0, 1.0, fake, st) == binding.JARQ_EINVAL
    assert acc(fake, 0, 128, 1.0, fake, st) == binding.JARQ_OK              # nothing to do
    assert acc(None, 0, 128, 1.0, fake, st) == binding.JARQ_OK
    fin = lib.jarq_hessian_finalize
    assert fin(fake, 128, -0.1, 0.0, _vp(1 << 30), st) == binding.JARQ_EINVAL
    assert fin(fake, 128, 0.0, float("inf"), _vp(1 << 30), st) == binding.JARQ_EINVAL
    assert fin(fake, 128, 0.0, 0.0, _vp((1 << 20) + 64), st) == binding.JARQ_EINVAL  # overlap
    p = binding.make_params(64, 256, 64, 3, 5)
    bad = binding.make_params(64, 250, 64, 3, 5)
    assert lib.jarq_rtn(ctypes.byref(bad), fake, fake, fake, fake, st) == binding.JARQ_EINVAL
    assert lib.jarq_rtn(ctypes.byref(p), fake, _vp((1 << 20) + 8), fake, fake, st) == binding.JARQ_EINVAL


def test_gptq_workspace_and_argument_errors(lib):
    p = binding.make_params(14336, 4096, 64, 3, 1)
    n = lib.jarq_gptq_workspace_bytes(ctypes.byref(p))
    # two 4096^2 fp64 matrices and the 14336 x 4096 fp64 errors dominate
    assert 2 * 8 * 4096 ** 2 + 8 * 14336 * 4096 < n < 1.2 * (2 * 8 * 4096 ** 2 + 8 * 14336 * 4096) + (64 << 20)
    assert lib.jarq_gptq_workspace_bytes(ctypes.byref(binding.make_params(64, 250, 64, 3, 1))) == 0
    fake = _vp(1 << 20)
    q = binding.make_params(64, 256, 64, 3, 1)
    assert lib.jarq_gptq(ctypes.byref(q), fake, fake, fake, fake, fake, None, 1 << 30, None) == binding.JARQ_EWORKSPACE
    assert lib.jarq_gptq(ctypes.byref(q), fake, fake, fake, fake, fake, fake, 1024, None) == binding.JARQ_EWORKSPACE
    assert lib.jarq_gptq(ctypes.byref(q), _vp((1 << 20) + 4), fake, fake, fake, fake, fake, 1 << 30,
                         None) == binding.JARQ_EINVAL


def test_qep_entry_points_check_arguments(lib):
    fake = _vp(1 << 20)
    acc = lib.jarq_cross_accumulate
    assert acc(fake, fake, 10, 130, 1.0, fake, None) == binding.JARQ_EINVAL
    assert acc(None, None, 0, 128, 1.0, fake, None) == binding.JARQ_OK
    assert acc(fake, _vp((1 << 20) + 4), 10, 128, 1.0, fake, None) == binding.JARQ_EINVAL
    p = binding.make_params(64, 256, 64, 3, 1)
    n = lib.jarq_qep_workspace_bytes(ctypes.byref(p))
    assert n >= 8 * (256 * 256 + 2 * 64 * 256)
    cor = lib.jarq_qep_correct
    assert cor(ctypes.byref(p), fake, fake, fake, 1.5, fake, fake, 1 << 30, None) == binding.JARQ_EINVAL
    assert cor(ctypes.byref(p), fake, fake, fake, float("nan"), fake, fake, 1 << 30, None) == binding.JARQ_EINVAL
    assert cor(ctypes.byref(p), fake, fake, fake, 0.5, fake, fake, 16, None) == binding.JARQ_EWORKSPACE


def test_binding_rejects_host_tensors_and_wrong_types():
    import torch
    p = binding.make_params(8, 64, 32, 3, 1)
    W = torch.zeros(8, 64, dtype=torch.float32)          # host memory
    with pytest.raises(ValueError):
        binding.rtn(p, W, codes=torch.zeros(8, 64, dtype=torch.uint8),
                    scales=torch.zeros(8, 2), zeros=torch.zeros(8, 2, dtype=torch.int32))
    with pytest.raises(TypeError):
        binding.rtn(p, W.double(), codes=torch.zeros(8, 64, dtype=torch.uint8),
                    scales=torch.zeros(8, 2), zeros=torch.zeros(8, 2, dtype=torch.int32))
    with pytest.raises(ValueError):
        binding.hessian_accumulate(torch.zeros(5, 8), torch.zeros(4, 4, dtype=torch.float64))
    with pytest.raises(ValueError):
        binding.cross_accumulate(torch.zeros(5, 8), torch.zeros(6, 8),
                                 torch.zeros(8, 8, dtype=torch.float64))
    with pytest.raises(ValueError):
        binding.hessian_finalize(torch.zeros(4, 5, dtype=torch.float64))
    assert binding.packed_words_per_row(binding.make_params(2, 96, 32, 3, 1)) == 9
    assert binding.DTYPES[torch.bfloat16] == 2


def test_bf16_hessian_checks_arguments(lib):
    fake = _vp(1 << 20)
    acc = lib.jarq_hessian_accumulate_bf16
    assert acc(fake, 10, 132, 1.0, fake, None) == binding.JARQ_EINVAL     # d % 8
    assert acc(_vp((1 << 20) + 8), 10, 128, 1.0, fake, None) == binding.JARQ_EINVAL
    assert acc(None, 0, 128, 1.0, fake, None) == binding.JARQ_OK


def test_bench_refuses_more_than_one_gpu():
    """The benchmark runs on one GPU; asking for more exits with a message."""
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    res = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=120)
    assert res.returncode != 0
    assert "one GPU" in (res.stdout + res.stderr)
    assert res.stdout.strip() == "" or not res.stdout.strip().startswith("{")
