"""The allocation-free entry point conv_fwd_ex_noalloc, through the C ABI.

It runs the plans and kernels of conv_fwd_ex with every workspace carved from
the library's static per-GPU scratch array instead of allocated.  Each case
makes two calls in a row, the second with a smaller input (the array keeps
the first call's contents), and checks each result bit for bit against
conv_fwd_ex on the same inputs (same plans, same fixed summation order) and
against the oracle at the fp32 / bf16 tolerance.  The cases cover every kind
of workspace: the rearranged Ker of a strided layer, phase images of In, the
split reduction's partial sums, and the exact fp32 widening of bf16 inputs
for taps without a bf16 kernel.
"""
import numpy as np
import pytest
import torch

from oracle import conv as oconv
from paper_2101_09808_amd import conv as B
from paper_2101_09808_amd.workloads import ConvShape, make_inputs

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-5, "bf16": 1e-2}
DEV = "cuda:0"


def say(*a):
    print(*a, flush=True)


def host(x):
    return x.float().cpu().numpy()


def rel_err(out, ref):
    m = float(np.max(np.abs(ref)))
    e = float(np.max(np.abs(out.astype(np.float64) - ref)))
    return e / m if m > 0 else e


# (larger call, smaller call) per workspace kind
CASES = {
    "f32_strided_ker_rearranged": (
        ConvShape("na_s2p1_big", 2, 16, 32, 30, 30, 3, 3, "f32", 501, 2, 1),
        ConvShape("na_s2p1_small", 1, 8, 16, 12, 12, 3, 3, "f32", 502, 2, 1)),
    "f32_phase_images": (
        ConvShape("na_s3p2_5x5_big", 2, 6, 10, 23, 19, 5, 5, "f32", 503, 3, 2),
        ConvShape("na_s3p2_5x5_small", 1, 6, 10, 17, 14, 5, 5, "f32", 504, 3, 2)),
    "f32_7x7_s2_register_staged": (
        ConvShape("na_r1_batch1", 1, 3, 64, 224, 224, 7, 7, "f32", 505, 2, 3),
        ConvShape("na_7x7_small", 1, 3, 16, 30, 30, 7, 7, "f32", 506, 2, 3)),
    "f32_split_partial_sums": (
        ConvShape("na_r9_batch1", 1, 256, 256, 14, 14, 3, 3, "f32", 507, 1, 1),
        ConvShape("na_r12_batch1", 1, 512, 512, 7, 7, 3, 3, "f32", 508, 1, 1)),
    "f32_split_valid": (
        ConvShape("na_split_valid_big", 1, 256, 256, 16, 16, 3, 3, "f32", 509),
        ConvShape("na_split_valid_small", 1, 512, 512, 9, 9, 3, 3, "f32", 510)),
    "bf16_strided_phase_images": (
        ConvShape("na_bf16_s2_c32", 1, 32, 64, 34, 34, 3, 3, "bf16", 511, 2, 1),
        ConvShape("na_bf16_s2_c16", 1, 16, 32, 22, 22, 3, 3, "bf16", 512, 2, 1)),
    "bf16_widened_padded": (
        ConvShape("na_bf16_2x3_big", 2, 12, 24, 9, 10, 2, 3, "bf16", 513, 1, 1),
        ConvShape("na_bf16_2x3_small", 1, 5, 7, 6, 6, 2, 3, "bf16", 514, 1, 1)),
    "f32_no_workspace": (
        ConvShape("na_1x1_c256", 2, 256, 64, 56, 56, 1, 1, "f32", 515),
        ConvShape("na_3x3_c64", 1, 64, 64, 58, 58, 3, 3, "f32", 516)),
}


def run_pair(shape):
    In, Ker = make_inputs(shape)
    In_d, Ker_d = In.to(DEV), Ker.to(DEV)
    st, pd = (shape.stride,) * 2, (shape.pad,) * 2
    P, Q = shape.P, shape.Q
    # poisoned outputs: every element must be written
    out_na = torch.full((shape.N, shape.K, P, Q), float("nan"), device=DEV)
    out_ex = torch.full_like(out_na, float("nan"))
    say(f"[gpu] noalloc {shape.name} {shape.key()} stride={shape.stride} pad={shape.pad} {shape.dtype}")
    B.conv_fwd_ex_noalloc(In_d, Ker_d, st, pd, out=out_na)
    torch.cuda.synchronize()
    B.conv_fwd_ex(In_d, Ker_d, st, pd, out=out_ex)
    torch.cuda.synchronize()
    assert torch.equal(out_na, out_ex), f"{shape.name}: allocation-free result differs from conv_fwd_ex"
    ref = oconv.conv_fwd_ex(host(In), host(Ker), st, pd)
    err = rel_err(host(out_na), ref)
    assert err <= TOL[shape.dtype], f"{shape.name}: rel err {err:.3e}"


@pytest.mark.parametrize("case", sorted(CASES), ids=str)
def test_noalloc_matches_conv_fwd_ex_two_calls(case):
    big, small = CASES[case]
    run_pair(big)
    run_pair(small)


def test_noalloc_rejects_oversized_scratch_and_leaves_out_untouched():
    """Phase images of this 5x5 stride-3 layer need about 130 MB of scratch,
    beyond CONV_NOALLOC_SCRATCH_BYTES: the call returns CONV_ESCRATCH before
    launching anything, and conv_fwd_ex still runs it."""
    shape = ConvShape("na_too_big", 8, 64, 16, 256, 256, 5, 5, "f32", 517, 3, 2)
    plan, direct = B.conv_fwd_ex_plan(*shape.key(), shape.stride, shape.pad)
    assert not direct
    In, Ker = make_inputs(shape)
    In_d, Ker_d = In.to(DEV), Ker.to(DEV)
    out = torch.full((shape.N, shape.K, shape.P, shape.Q), 7.0, device=DEV)
    torch.cuda.synchronize()
    say(f"[gpu] noalloc oversized {shape.key()}")
    with pytest.raises(B.ConvError) as ei:
        B.conv_fwd_ex_noalloc(In_d, Ker_d, shape.stride, shape.pad, out=out)
    assert ei.value.status == B.CONV_ESCRATCH
    torch.cuda.synchronize()
    assert (out == 7.0).all()
