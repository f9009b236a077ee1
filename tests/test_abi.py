"""The C-ABI library loads, exports what the header declares, and rejects bad
arguments before touching the GPU (CPU only: no compute call is made)."""
import ctypes
import os
import re
import subprocess

import pytest

from paper_2101_09808_amd import conv as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "conv_fwd.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(conv_\w+)\s*\(", text, flags=re.M)))


def test_header_declares_the_boundary():
    fns = declared_functions()
    for name in ("conv_fwd", "conv_fwd_bf16", "conv_fwd_plan", "conv_fwd_strerror",
                 "conv_fwd_with_plan", "conv_fwd_candidates", "conv_model_volume", "conv_fwd_tune",
                 "conv_fwd_ex", "conv_fwd_ex_inner_shape", "conv_fwd_bf16_out"):
        assert name in fns


def test_library_exports_every_declared_symbol():
    lib = B.lib()
    for name in declared_functions():
        assert hasattr(lib, name), f"missing export {name}"
    nm = subprocess.run(["nm", "-D", "--defined-only", B.LIB_PATH], capture_output=True, text=True)
    if nm.returncode == 0:
        for name in declared_functions():
            assert re.search(rf"\bT {name}$", nm.stdout, flags=re.M), name


def test_plan_struct_layout_matches_header():
    # conv_plan_t: 14 ints, int64, 4 ints, 4+4+1+1+1+4 doubles (no padding)
    assert ctypes.sizeof(B.ConvPlan) == 14 * 4 + 8 + 4 * 4 + 15 * 8
    assert B.ConvPlan.num_wg.offset == 14 * 4


VALID = (1, 4, 8, 6, 6, 3, 3)


@pytest.mark.parametrize("shape,status", [
    ((0, 4, 8, 6, 6, 3, 3), B.CONV_EINVAL),
    ((1, 0, 8, 6, 6, 3, 3), B.CONV_EINVAL),
    ((1, 4, -1, 6, 6, 3, 3), B.CONV_EINVAL),
    ((1, 4, 8, 2, 6, 3, 3), B.CONV_EINVAL),   # R > H
    ((1, 4, 8, 6, 2, 3, 3), B.CONV_EINVAL),   # S > W
    ((1, 4, 8, 6, 6, 0, 3), B.CONV_EINVAL),
    ((4096, 4096, 8, 64, 64, 3, 3), B.CONV_ERANGE),   # In has 2^36 elements
    ((1, 65536, 65536, 6, 6, 1, 1), B.CONV_ERANGE),   # Ker has 2^32 elements
])
def test_bad_shapes_rejected(shape, status):
    L = B.lib()
    fake = ctypes.c_void_p(0x1000)  # never dereferenced: validation fails first
    assert L.conv_fwd(*shape, fake, fake, fake, None) == status
    assert L.conv_fwd_bf16(*shape, fake, fake, fake, None) == status
    p = B.ConvPlan()
    assert L.conv_fwd_plan(*shape, 0, ctypes.byref(p)) == status


@pytest.mark.parametrize("which", [0, 1, 2])
def test_null_pointers_rejected(which):
    L = B.lib()
    ptrs = [ctypes.c_void_p(0x1000)] * 3
    ptrs[which] = None
    assert L.conv_fwd(*VALID, *ptrs, None) == B.CONV_ENULL
    assert L.conv_fwd_bf16(*VALID, *ptrs, None) == B.CONV_ENULL
    assert L.conv_fwd_bf16_out(*VALID, *ptrs, None) == B.CONV_ENULL
    assert L.conv_fwd_with_plan(*VALID, *ptrs, ctypes.byref(B.ConvPlan()), None) == B.CONV_ENULL
    assert L.conv_fwd_plan(*VALID, 0, None) == B.CONV_ENULL


def test_bad_plan_rejected_without_launch():
    L = B.lib()
    fake = ctypes.c_void_p(0x1000)
    p = B.ConvPlan.from_dict(B.conv_fwd_plan(*VALID))
    p.tile_k = 48  # not 16 * wave blocks * waves
    assert L.conv_fwd_with_plan(*VALID, fake, fake, fake, ctypes.byref(p), None) == B.CONV_EINVAL
    p = B.ConvPlan.from_dict(B.conv_fwd_plan(*VALID))
    p.variant = 999
    assert L.conv_fwd_with_plan(*VALID, fake, fake, fake, ctypes.byref(p), None) == B.CONV_EINVAL
    assert L.conv_fwd_plan(*VALID, 7, ctypes.byref(B.ConvPlan())) == B.CONV_EINVAL


def test_tune_arguments_rejected_without_launch():
    L = B.lib()
    fake = ctypes.c_void_p(0x1000)
    p = B.ConvPlan()
    t = (ctypes.c_float * 8)()
    assert L.conv_fwd_tune(*VALID, 0, fake, fake, None, 5, 3, None, ctypes.byref(p), t) == B.CONV_ENULL
    assert L.conv_fwd_tune(*VALID, 0, fake, fake, fake, 5, 3, None, None, t) == B.CONV_ENULL
    assert L.conv_fwd_tune(*VALID, 2, fake, fake, fake, 5, 3, None, ctypes.byref(p), t) == B.CONV_EINVAL
    for top_n, reps in ((0, 3), (B.CONV_TUNE_MAX + 1, 3), (5, 0), (5, 1001)):
        assert L.conv_fwd_tune(*VALID, 0, fake, fake, fake, top_n, reps, None, ctypes.byref(p), t) == B.CONV_EINVAL
    assert L.conv_fwd_tune(0, *VALID[1:], 0, fake, fake, fake, 5, 3, None, ctypes.byref(p), t) == B.CONV_EINVAL


@pytest.mark.parametrize("args,status", [
    ((0, 1, 0, 0), B.CONV_EINVAL),    # stride 0
    ((1, 1, -1, 0), B.CONV_EINVAL),   # negative pad
    ((65, 1, 0, 0), B.CONV_EINVAL),   # stride above 64
    ((2, 2, 0, 0), B.CONV_OK),
])
def test_ex_arguments(args, status):
    L = B.lib()
    inner = (ctypes.c_int32 * 9)()
    assert L.conv_fwd_ex_inner_shape(*VALID, *args, inner) == status
    if status == B.CONV_OK:
        assert list(inner)[7:] == [(6 - 3) // 2 + 1] * 2
    fake = ctypes.c_void_p(0x1000)
    if status != B.CONV_OK:
        assert L.conv_fwd_ex(*VALID, *args, 0, fake, fake, fake, None) == status
    # kernel larger than the padded input; null pointers; bad dtype
    assert L.conv_fwd_ex(1, 4, 8, 2, 6, 5, 3, 1, 1, 1, 0, 0, fake, fake, fake, None) == B.CONV_EINVAL
    assert L.conv_fwd_ex(*VALID, 2, 2, 1, 1, 0, None, fake, fake, None) == B.CONV_ENULL
    assert L.conv_fwd_ex(*VALID, 2, 2, 1, 1, 5, fake, fake, fake, None) == B.CONV_EINVAL
    assert L.conv_fwd_ex_inner_shape(*VALID, 1, 1, 0, 0, None) == B.CONV_ENULL


def test_strerror():
    for st in (B.CONV_OK, B.CONV_EINVAL, B.CONV_ENULL, B.CONV_ERANGE, B.CONV_ENOPLAN, B.CONV_EHIP):
        assert B.strerror(st)
    assert "unknown" in B.strerror(12345)


def test_python_binding_refuses_cpu_tensors():
    import torch
    x = torch.zeros(1, 2, 4, 4)
    k = torch.zeros(3, 2, 3, 3)
    with pytest.raises(ValueError):
        B.conv_fwd(x, k)
