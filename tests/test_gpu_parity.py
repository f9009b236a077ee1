"""Parity of the HIP path (through the C ABI) with the fp64 oracle of Eq. (1).

Bar: max|Out - ref| / max|ref| <= 1e-5 for fp32 inputs and <= 1e-2 for bf16
inputs (products of bf16 values are exact in fp32, so the bf16 path is in
practice as accurate as fp32); bitwise equality where every partial sum is an
exact integer (integer-valued inputs, all-ones and one-hot kernels), since
then the result does not depend on the summation order.
"""
import numpy as np
import pytest
import torch

from oracle import conv as oconv
from paper_2101_09808_amd import conv as B
from paper_2101_09808_amd.workloads import CONFIGS, ConvShape, make_inputs

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-5, "bf16": 1e-2}
DEV = "cuda:0"


def say(*a):
    print(*a, flush=True)


def gpu_conv(shape, In, Ker, plan=None, out=None):
    In_d, Ker_d = In.to(DEV), Ker.to(DEV)
    if plan is not None:
        o = B.conv_fwd_with_plan(In_d, Ker_d, plan, out=out)
    elif shape.dtype == "bf16":
        o = B.conv_fwd_bf16(In_d, Ker_d, out=out)
    else:
        o = B.conv_fwd(In_d, Ker_d, out=out)
    torch.cuda.synchronize()
    return o


def host(x):
    return x.float().cpu().numpy()


def rel_err(out, ref):
    m = float(np.max(np.abs(ref)))
    e = float(np.max(np.abs(out.astype(np.float64) - ref)))
    return e / m if m > 0 else e


def check_full(shape, kind="uniform", seed=None, plan=None):
    In, Ker = make_inputs(shape, seed=seed, kind=kind)
    say(f"[gpu] {shape.name} {shape.key()} {shape.dtype} kind={kind} plan={plan and plan.get('variant')}")
    out = host(gpu_conv(shape, In, Ker, plan))
    ref = oconv.conv_fwd(host(In), host(Ker))
    assert out.shape == ref.shape
    if kind == "int":
        assert np.array_equal(out.astype(np.float64), ref), f"{shape.name}: integer result not exact"
    else:
        err = rel_err(out, ref)
        assert err <= TOL[shape.dtype], f"{shape.name}: rel err {err:.3e}"
    return out, ref


def small_version(c, n=2):
    return ConvShape(c.name + f"_n{min(c.N, n)}", min(c.N, n), c.C, c.K, c.H, c.W, c.R, c.S, c.dtype, c.seed)


# ----------------------------------------------------------------- configs

@pytest.mark.parametrize("cfg", CONFIGS, ids=lambda c: c.name)
def test_config_reduced_batch_full_compare(cfg):
    """Each layer at batch <= 2: every output against the oracle."""
    check_full(small_version(cfg, 1 if cfg.dtype == "bf16" else 2))


@pytest.mark.parametrize("cfg", CONFIGS, ids=lambda c: c.name)
def test_config_full_size_full_compare(cfg):
    """Full layer size, the plan the benchmark times: every output against the
    oracle (which runs the whole layer on the host cores in about a second),
    plus the 16 corners of the output tensor checked point by point as a
    second, independent route through the oracle."""
    In, Ker = make_inputs(cfg)
    say(f"[gpu] full {cfg.name} plan={B.conv_fwd_plan(*cfg.key(), dtype=int(cfg.dtype == 'bf16'))}")
    out = host(gpu_conv(cfg, In, Ker))
    ref = oconv.conv_fwd(host(In), host(Ker))
    assert out.shape == ref.shape
    assert np.all(np.isfinite(out))
    err = rel_err(out, ref)
    assert err <= TOL[cfg.dtype], f"{cfg.name}: rel err {err:.3e}"
    P, Q = cfg.P, cfg.Q
    corners = [((n * cfg.K + k) * P + p) * Q + q for n in (0, cfg.N - 1) for k in (0, cfg.K - 1)
               for p in (0, P - 1) for q in (0, Q - 1)]
    idx = np.array(corners, np.int64)
    pts = oconv.conv_fwd_points(host(In), host(Ker), idx)
    assert np.array_equal(pts, ref.reshape(-1)[idx])


def test_smallest_config_full_size_full_compare():
    check_full(CONFIGS[0])


# ----------------------------------------------------------------- edges

EDGE = [
    ConvShape("primes_3x3", 2, 3, 5, 13, 13, 3, 3, "f32", 11),
    ConvShape("rect_taps", 2, 7, 33, 11, 17, 2, 4, "f32", 12),
    ConvShape("pointwise_odd", 3, 5, 17, 9, 7, 1, 1, "f32", 13),
    ConvShape("one_pixel_out", 2, 9, 20, 3, 3, 3, 3, "f32", 14),
    ConvShape("single_everything", 1, 1, 1, 1, 1, 1, 1, "f32", 15),
    ConvShape("tall_thin", 1, 6, 16, 40, 3, 3, 3, "f32", 16),
    ConvShape("wide_row", 1, 4, 16, 3, 300, 3, 3, "f32", 17),
    ConvShape("k_tail_c_tail", 2, 13, 70, 10, 12, 3, 3, "f32", 18),
    ConvShape("big_taps_5x5", 2, 6, 24, 14, 12, 5, 5, "f32", 19),
    ConvShape("r_eq_h", 2, 8, 32, 3, 9, 3, 1, "f32", 20),
    ConvShape("many_images_small", 37, 8, 16, 5, 5, 3, 3, "f32", 21),
    ConvShape("pointwise_many_k", 2, 32, 200, 7, 7, 1, 1, "f32", 22),
]


@pytest.mark.parametrize("shape", EDGE, ids=lambda s: s.name)
def test_edge_shapes(shape):
    check_full(shape)


EDGE_BF16 = [
    ConvShape("bf16_multi_chunk_ktail", 2, 40, 72, 11, 13, 3, 3, "bf16", 41),
    ConvShape("bf16_one_chunk", 1, 32, 64, 20, 22, 3, 3, "bf16", 42),
    ConvShape("bf16_pointwise", 3, 16, 20, 7, 9, 1, 1, "bf16", 43),
    ConvShape("bf16_odd_width", 1, 8, 16, 6, 9, 3, 3, "bf16", 44),
    ConvShape("bf16_rect_taps_generic", 2, 12, 24, 9, 10, 2, 3, "bf16", 45),
]


@pytest.mark.parametrize("shape", EDGE_BF16, ids=lambda s: s.name)
def test_bf16_edge_shapes(shape):
    """Taps without a bf16 kernel instance (2x3) have no bf16 plan; conv_fwd_bf16
    then widens In and Ker exactly to fp32 in a workspace and runs the fp32
    plan, which this checks too."""
    try:
        B.conv_fwd_plan(*shape.key(), dtype=B.CONV_DTYPE_BF16)
    except B.ConvError as e:
        if e.status != B.CONV_ENOPLAN:
            raise
        assert shape.name == "bf16_rect_taps_generic"
    check_full(shape)


@pytest.mark.parametrize("shape", EDGE_BF16[:2], ids=lambda s: s.name)
def test_bf16_integer_inputs_bitwise(shape):
    check_full(shape, kind="int", seed=shape.seed + 1)


@pytest.mark.parametrize("shape", [EDGE[0], EDGE[7], small_version(CONFIGS[2]), small_version(CONFIGS[3]),
                                   small_version(CONFIGS[1])], ids=lambda s: s.name)
def test_integer_inputs_bitwise(shape):
    check_full(shape, kind="int", seed=shape.seed + 1)


def test_closed_forms_bitwise():
    s = ConvShape("ones", 2, 12, 40, 15, 11, 3, 3, "f32", 0)
    say("[gpu] all-ones")
    In = torch.ones(s.N, s.C, s.H, s.W)
    Ker = torch.ones(s.K, s.C, s.R, s.S)
    out = host(gpu_conv(s, In, Ker))
    assert np.all(out == s.C * s.R * s.S)
    say("[gpu] one-hot kernel")
    g = torch.Generator().manual_seed(5)
    In = torch.rand(s.N, s.C, s.H, s.W, generator=g) * 2 - 1
    Ker = torch.zeros(s.K, s.C, s.R, s.S)
    sel = [((3 * k + 1) % s.C, k % s.R, (k // s.R + 1) % s.S) for k in range(s.K)]
    for k, (c0, r0, s0) in enumerate(sel):
        Ker[k, c0, r0, s0] = 1.0
    out = host(gpu_conv(s, In, Ker))
    for k, (c0, r0, s0) in enumerate(sel):
        assert np.array_equal(out[:, k], In[:, c0, r0:r0 + s.P, s0:s0 + s.Q].numpy())


def test_deterministic_and_overwrites_poisoned_output_with_guards():
    s = small_version(CONFIGS[2])
    In, Ker = make_inputs(s)
    In_d, Ker_d = In.to(DEV), Ker.to(DEV)
    n_out = s.N * s.K * s.P * s.Q
    guard = 4096
    buf = torch.full((n_out + 2 * guard,), float("nan"), device=DEV)
    buf[:guard] = 7.0
    buf[-guard:] = 7.0
    out = buf[guard:guard + n_out].view(s.N, s.K, s.P, s.Q)
    say("[gpu] poisoned output run 1")
    B.conv_fwd(In_d, Ker_d, out=out)
    torch.cuda.synchronize()
    first = out.clone()
    assert torch.isfinite(first).all(), "some outputs were not written"
    assert (buf[:guard] == 7.0).all() and (buf[-guard:] == 7.0).all(), "write outside Out"
    say("[gpu] poisoned output run 2")
    out.fill_(float("nan"))
    B.conv_fwd(In_d, Ker_d, out=out)
    torch.cuda.synchronize()
    assert torch.equal(out, first), "two runs differ"


def test_side_stream():
    s = EDGE[7]
    In, Ker = make_inputs(s)
    ref = oconv.conv_fwd(host(In), host(Ker))
    st = torch.cuda.Stream()
    In_d, Ker_d = In.to(DEV), Ker.to(DEV)
    torch.cuda.synchronize()
    say("[gpu] side stream")
    with torch.cuda.stream(st):
        out = B.conv_fwd(In_d, Ker_d)
    st.synchronize()
    assert rel_err(host(out), ref) <= TOL["f32"]


def test_error_leaves_output_untouched():
    """Argument and plan validation errors launch nothing: a poisoned Out
    keeps its values after an unknown plan variant, R > H and a null In."""
    s = EDGE[7]
    In, Ker = make_inputs(s)
    In_d, Ker_d = In.to(DEV), Ker.to(DEV)
    out = torch.full((s.N, s.K, s.P, s.Q), 7.0, device=DEV)
    torch.cuda.synchronize()
    bad = B.conv_fwd_plan(*s.key())
    bad["variant"] = 99999
    with pytest.raises(B.ConvError) as ei:
        B.conv_fwd_with_plan(In_d, Ker_d, bad, out=out)
    assert ei.value.status == B.CONV_EINVAL
    L = B.lib()
    stream = torch.cuda.current_stream().cuda_stream
    assert L.conv_fwd(s.N, s.C, s.K, 2, s.W, 3, 3, In_d.data_ptr(), Ker_d.data_ptr(), out.data_ptr(),
                      stream) == B.CONV_EINVAL
    assert L.conv_fwd(*s.key(), None, Ker_d.data_ptr(), out.data_ptr(), stream) == B.CONV_ENULL
    torch.cuda.synchronize()
    assert (out == 7.0).all()


# ----------------------------------------------------------------- every kernel variant

def _plans_per_variant(dims, dtype=B.CONV_DTYPE_F32, per_variant=3):
    n = B.lib().conv_fwd_candidates(*dims, dtype, None, 0)
    cands = B.conv_fwd_candidates(*dims, dtype=dtype, cap=max(n, 1))
    chosen = {}
    for p in cands:
        key = (p["variant"], p["waves_k"], p["grid_order"], p.get("split_c", 1) > 1)
        chosen.setdefault(key, p)
    by_var = {}
    for key, p in sorted(chosen.items()):
        by_var.setdefault(key[0], [])
        if len(by_var[key[0]]) < per_variant:
            by_var[key[0]].append(p)
    return [p for ps in by_var.values() for p in ps]


VARIANT_SHAPES = [
    ConvShape("var3x3", 2, 20, 72, 15, 19, 3, 3, "f32", 31),
    ConvShape("var1x1", 3, 40, 72, 13, 11, 1, 1, "f32", 32),
    ConvShape("var2x4", 2, 9, 40, 12, 13, 2, 4, "f32", 33),
    # 2x2 and 4x4 taps: the inner problems of stride-2 layers
    ConvShape("var2x2", 2, 40, 72, 11, 13, 2, 2, "f32", 38),
    ConvShape("var4x4", 2, 24, 72, 12, 14, 4, 4, "f32", 39),
    # pointwise layers whose channel count has a fully unrolled streaming kernel
    ConvShape("var1x1_c64", 2, 64, 72, 13, 11, 1, 1, "f32", 34),
    ConvShape("var1x1_c128", 3, 128, 64, 7, 9, 1, 1, "f32", 35),
    ConvShape("var1x1_c256", 2, 256, 80, 8, 10, 1, 1, "f32", 36),
    ConvShape("var1x1_c512", 1, 512, 64, 7, 7, 1, 1, "f32", 37),
    # 792 pixels: shares of 396, 264 and 132 pixels per workgroup, i.e. 3, 2
    # and 1 blocks of 32 per wave plus a tail, for the balanced pointwise
    # kernel (K = 80: a second, partial k tile)
    ConvShape("var1x1_bal_c64", 2, 64, 80, 18, 22, 1, 1, "f32", 40),
    ConvShape("var1x1_bal_c128", 2, 128, 64, 18, 22, 1, 1, "f32", 41),
    ConvShape("var1x1_bal_c256", 2, 256, 80, 18, 22, 1, 1, "f32", 42),
    ConvShape("var1x1_bal_c512", 2, 512, 64, 18, 22, 1, 1, "f32", 43),
    ConvShape("var1x1_bal_c384", 2, 384, 64, 18, 22, 1, 1, "f32", 44),
]


@pytest.mark.parametrize("shape", VARIANT_SHAPES, ids=lambda s: s.name)
def test_every_variant(shape):
    In, Ker = make_inputs(shape)
    ref = oconv.conv_fwd(host(In), host(Ker))
    plans = _plans_per_variant(shape.key())
    assert plans
    for p in plans:
        say(f"[gpu] {shape.name} variant={p['variant']} tile={p['tile_k']}x{p['tile_rows']}x{p['tile_cols']} "
            f"waves={p['waves_k']}x{p['waves_px']} order={p['grid_order']} split={p['split_c']}")
        out = host(gpu_conv(shape, In, Ker, plan=p))
        err = rel_err(out, ref)
        assert err <= TOL["f32"], (p, err)


BF16_VARIANT_SHAPES = [
    ConvShape("bf16_var3x3", 1, 40, 72, 11, 13, 3, 3, "bf16", 51),
    ConvShape("bf16_var1x1", 2, 64, 80, 10, 12, 1, 1, "bf16", 52),
    # C = 32: the transposing-read kernel (tiles of 8 x 32, 4 x 64, 7 x 64)
    ConvShape("bf16_var_c32", 2, 32, 48, 18, 42, 3, 3, "bf16", 53),
    ConvShape("bf16_c32_k64", 1, 32, 64, 58, 66, 3, 3, "bf16", 54),
    # Q % 4 != 0: 4-byte stores; K < 64
    ConvShape("bf16_c32_q42", 1, 32, 40, 10, 44, 3, 3, "bf16", 55),
    # 2x2 and 4x4 taps (inner problems of stride-2 layers)
    ConvShape("bf16_var2x2", 2, 40, 72, 11, 13, 2, 2, "bf16", 56),
    ConvShape("bf16_var4x4", 1, 24, 40, 12, 14, 4, 4, "bf16", 57),
]
# kernel families each shape is there for (others are covered by the shapes before)
BF16_SHAPE_FAMILIES = {"bf16_var_c32": {6}, "bf16_c32_k64": {6}, "bf16_c32_q42": {6}}


def bf16_variant_plans(shape):
    plans = _plans_per_variant(shape.key(), dtype=B.CONV_DTYPE_BF16)
    fams = BF16_SHAPE_FAMILIES.get(shape.name)
    if fams:
        plans = [p for p in plans if B.conv_fwd_geometry(*shape.key(), p)["family"] in fams]
    return plans


def test_bf16_transposing_kernel_unaligned_out():
    """Out 4 bytes past a 16-byte boundary: the transposing-read kernel falls
    back from 16-byte to 4-byte stores."""
    shape = BF16_VARIANT_SHAPES[2]
    In, Ker = make_inputs(shape)
    ref = oconv.conv_fwd(host(In), host(Ker))
    plans = [p for p in bf16_variant_plans(shape) if B.conv_fwd_geometry(*shape.key(), p)["family"] == 6]
    assert plans
    buf = torch.full((shape.N * shape.K * shape.P * shape.Q + 4,), 7.0, device=DEV)
    out = buf[1:1 + shape.N * shape.K * shape.P * shape.Q].view(shape.N, shape.K, shape.P, shape.Q)
    assert out.data_ptr() % 16 == 4
    for p in plans:
        say(f"[gpu] {shape.name} unaligned Out variant={p['variant']}")
        buf.fill_(7.0)
        B.conv_fwd_with_plan(In.to(DEV), Ker.to(DEV), p, out=out)
        torch.cuda.synchronize()
        assert rel_err(host(out), ref) <= TOL["bf16"], p
        assert buf[0].item() == 7.0 and (buf[-3:] == 7.0).all()


@pytest.mark.parametrize("shape", BF16_VARIANT_SHAPES, ids=lambda s: s.name)
def test_every_bf16_variant(shape):
    In, Ker = make_inputs(shape)
    ref = oconv.conv_fwd(host(In), host(Ker))
    plans = bf16_variant_plans(shape)
    assert plans
    for p in plans:
        say(f"[gpu] {shape.name} variant={p['variant']} tile={p['tile_k']}x{p['tile_rows']}x{p['tile_cols']} "
            f"waves={p['waves_k']}x{p['waves_px']} order={p['grid_order']}")
        out = host(gpu_conv(shape, In, Ker, plan=p))
        err = rel_err(out, ref)
        assert err <= TOL["bf16"], (p, err)


@pytest.mark.parametrize("shape", [
    ConvShape("misaligned_1x1_vec_in", 2, 30, 40, 8, 10, 1, 1, "f32", 61),
    ConvShape("misaligned_3x3_vec_ker", 2, 24, 64, 14, 16, 3, 3, "f32", 62),
], ids=lambda s: s.name)
def test_misaligned_tensors(shape):
    """In and Ker starting 4 bytes past a 16-byte boundary: the library picks
    a kernel whose loads suit them, and an explicit plan with vector loads is
    refused without a launch."""
    In, Ker = make_inputs(shape)
    ref = oconv.conv_fwd(host(In), host(Ker))
    aligned_plan = B.conv_fwd_plan(*shape.key())
    bi = torch.zeros(In.numel() + 4, device=DEV)
    bk = torch.zeros(Ker.numel() + 4, device=DEV)
    In_d = bi[1:1 + In.numel()].view(In.shape)
    Ker_d = bk[1:1 + Ker.numel()].view(Ker.shape)
    In_d.copy_(In.to(DEV))
    Ker_d.copy_(Ker.to(DEV))
    assert In_d.data_ptr() % 16 == 4 and Ker_d.data_ptr() % 16 == 4
    say(f"[gpu] {shape.name} misaligned, aligned-case plan {aligned_plan['variant']}")
    out = B.conv_fwd(In_d, Ker_d)
    torch.cuda.synchronize()
    assert rel_err(host(out), ref) <= TOL["f32"]
    g = B.conv_fwd_geometry(*shape.key(), aligned_plan)
    if g["in_vec"] > 1 or g["ker_vec"] > 1:
        poison = torch.full_like(out, 7.0)
        with pytest.raises(B.ConvError) as ei:
            B.conv_fwd_with_plan(In_d, Ker_d, aligned_plan, out=poison)
        assert ei.value.status == B.CONV_EINVAL
        torch.cuda.synchronize()
        assert (poison == 7.0).all()


SPLIT_SHAPE = ConvShape("split_ranges", 1, 40, 64, 12, 12, 3, 3, "f32", 71)


def split_plans(shape):
    """Every split factor the selector offers for the shape, one plan each."""
    plans = {}
    for p in B.conv_fwd_candidates(*shape.key()):
        if p["split_c"] > 1:
            plans.setdefault(p["split_c"], p)
    return [plans[k] for k in sorted(plans)]


def test_split_reduction_parity_and_determinism():
    """Channel ranges reduced by the second pass (uneven ranges included):
    parity with the oracle, bitwise equality of two runs, and exact sums on
    integer inputs."""
    s = SPLIT_SHAPE
    plans = split_plans(s)
    assert len(plans) >= 2
    In, Ker = make_inputs(s)
    ref = oconv.conv_fwd(host(In), host(Ker))
    In_i, Ker_i = make_inputs(s, seed=s.seed + 1, kind="int")
    ref_i = oconv.conv_fwd(host(In_i), host(Ker_i))
    for p in plans:
        g = B.conv_fwd_geometry(*s.key(), p)
        say(f"[gpu] split={p['split_c']} steps={g['nchunks']} per range={g['cps']} variant={p['variant']}")
        a = gpu_conv(s, In, Ker, plan=p)
        b = gpu_conv(s, In, Ker, plan=p)
        assert torch.equal(a, b), "two runs differ"
        assert rel_err(host(a), ref) <= TOL["f32"]
        assert np.array_equal(host(gpu_conv(s, In_i, Ker_i, plan=p)).astype(np.float64), ref_i)


PLAN_KEYS = ("variant", "tile_k", "tile_rows", "tile_cols", "tile_c", "wave_k", "wave_px", "waves_k",
             "waves_px", "grid_order", "split_c")


def _same_plan(a, b):
    return all(a[k] == b[k] for k in PLAN_KEYS)


TUNE_SHAPES = [
    ConvShape("tune_f32_3x3", 2, 24, 40, 14, 16, 3, 3, "f32", 81),
    ConvShape("tune_bf16_c32", 1, 32, 48, 18, 34, 3, 3, "bf16", 82),
]


@pytest.mark.parametrize("shape", TUNE_SHAPES, ids=lambda s: s.name)
def test_tune_keeps_fastest_of_model_top_plans(shape):
    """Empirical pick among the model's best plans (Sec. 10): Out is Eq. (1),
    the plan kept is one of the first top_n candidates with the least time,
    and later calls for the shape run it."""
    In, Ker = make_inputs(shape)
    ref = oconv.conv_fwd(host(In), host(Ker))
    dt = B.CONV_DTYPE_BF16 if shape.dtype == "bf16" else B.CONV_DTYPE_F32
    In_d, Ker_d = In.to(DEV), Ker.to(DEV)
    say(f"[gpu] tune {shape.name}")
    out, plan, times = B.conv_fwd_tune(In_d, Ker_d, top_n=4, reps=2)
    torch.cuda.synchronize()
    assert rel_err(host(out), ref) <= TOL[shape.dtype]
    cands = B.conv_fwd_candidates(*shape.key(), dtype=dt)[:len(times)]
    assert 1 <= len(times) <= 4 and all(t > 0 for t in times)
    idx = [i for i, c in enumerate(cands) if _same_plan(c, plan)]
    assert idx and times[idx[0]] == min(times)
    assert _same_plan(B.conv_fwd_plan(*shape.key(), dtype=dt), plan)
    again = (B.conv_fwd_bf16 if dt == B.CONV_DTYPE_BF16 else B.conv_fwd)(In_d, Ker_d)
    torch.cuda.synchronize()
    assert rel_err(host(again), ref) <= TOL[shape.dtype]


# ---------------------------------------------------------------------------
# Strided, zero-padded convolution (conv_fwd_ex)

STRIDED_SHAPES = [
    ConvShape("s2p1_3x3", 2, 3, 4, 9, 7, 3, 3, "f32", 91, 2, 1),
    ConvShape("s2p1_3x3_c16", 2, 16, 32, 20, 20, 3, 3, "f32", 92, 2, 1),
    ConvShape("s2_1x1", 2, 24, 40, 15, 17, 1, 1, "f32", 93, 2, 0),
    ConvShape("s2p3_7x7_c3", 1, 3, 16, 30, 30, 7, 7, "f32", 94, 2, 3),
    ConvShape("s1p1_3x3", 2, 8, 16, 12, 12, 3, 3, "f32", 95, 1, 1),
    ConvShape("s3p2_5x5", 1, 6, 10, 17, 14, 5, 5, "f32", 96, 3, 2),
    ConvShape("s2p1_3x3_bf16", 1, 16, 32, 22, 22, 3, 3, "bf16", 97, 2, 1),
    ConvShape("s2p1_3x3_c32_bf16", 1, 32, 64, 34, 34, 3, 3, "bf16", 98, 2, 1),
]


@pytest.mark.parametrize("shape", STRIDED_SHAPES, ids=lambda s: s.name)
def test_strided_padded_parity(shape):
    In, Ker = make_inputs(shape)
    ref = oconv.conv_fwd_ex(host(In), host(Ker), (shape.stride,) * 2, (shape.pad,) * 2)
    say(f"[gpu] strided {shape.name} inner {B.conv_fwd_ex_inner_shape(*shape.key(), shape.stride, shape.pad)}")
    out = B.conv_fwd_ex(In.to(DEV), Ker.to(DEV), shape.stride, shape.pad)
    torch.cuda.synchronize()
    assert out.shape == ref.shape
    assert rel_err(host(out), ref) <= TOL[shape.dtype]


def test_strided_asymmetric_stride_and_pad():
    shape = ConvShape("s23p10", 1, 8, 12, 13, 10, 3, 2, "f32", 99)
    In, Ker = make_inputs(shape)
    ref = oconv.conv_fwd_ex(host(In), host(Ker), (2, 3), (1, 0))
    out = B.conv_fwd_ex(In.to(DEV), Ker.to(DEV), (2, 3), (1, 0))
    torch.cuda.synchronize()
    assert rel_err(host(out), ref) <= TOL["f32"]


@pytest.mark.parametrize("cfg", __import__("paper_2101_09808_amd.workloads", fromlist=["x"]).STRIDED_CONFIGS,
                         ids=lambda c: c.name)
def test_strided_full_config_full_compare(cfg):
    """Table 1 strided layers at batch 32: every output against the oracle."""
    In, Ker = make_inputs(cfg)
    say(f"[gpu] strided full {cfg.name}")
    out = host(B.conv_fwd_ex(In.to(DEV), Ker.to(DEV), cfg.stride, cfg.pad))
    ref = oconv.conv_fwd_ex(host(In), host(Ker), (cfg.stride,) * 2, (cfg.pad,) * 2)
    assert out.shape == ref.shape
    assert rel_err(out, ref) <= TOL["f32"]


@pytest.mark.parametrize("shape", [
    ConvShape("s2p0_3x3_c18_partial_chunk", 2, 18, 40, 113, 113, 3, 3, "f32", 91, 2, 0),
    ConvShape("s2p1_3x3_c30", 2, 30, 64, 112, 112, 3, 3, "f32", 92, 2, 1),
    ConvShape("s2p1_3x3_c16_k128", 1, 16, 128, 112, 112, 3, 3, "f32", 93, 2, 1),
], ids=lambda s: s.name)
def test_phase_skip_full_compare(shape):
    """Stride-2 3x3 layers whose plan is the phase-skip variant of the
    direct-to-LDS kernel (zero taps of the phases left out, In read through
    the phase mapping; one with a partial last chunk of input channels):
    every output against the oracle."""
    p, direct = B.conv_fwd_ex_plan(*shape.key(), shape.stride, shape.pad)
    g = B.conv_fwd_ex_geometry(*shape.key(), (2, 2), (shape.pad,) * 2, p)
    assert direct and g["phase_skip"] == 1
    In, Ker = make_inputs(shape)
    say(f"[gpu] phase skip {shape.name} v{p['variant']}")
    out = host(B.conv_fwd_ex(In.to(DEV), Ker.to(DEV), 2, shape.pad))
    ref = oconv.conv_fwd_ex(host(In), host(Ker), (2, 2), (shape.pad,) * 2)
    assert out.shape == ref.shape
    assert rel_err(out, ref) <= TOL["f32"]


def test_strided_padded_1x1_direct_full_compare():
    """A padded stride-2 1x1 layer whose plan is the balanced pointwise
    kernel reading In through the phase mapping (border pixels read zeros
    and are still stored): every output against the oracle."""
    shape = ConvShape("s2p1_1x1_n8_c64_k64_in56", 8, 64, 64, 56, 56, 1, 1, "f32", 75, 2, 1)
    p, direct = B.conv_fwd_ex_plan(*shape.key(), shape.stride, shape.pad)
    assert direct and B.conv_fwd_ex_geometry(*shape.key(), (2, 2), (1, 1), p)["family"] == 7
    In, Ker = make_inputs(shape)
    say(f"[gpu] strided padded 1x1 {shape.name} v{p['variant']}")
    out = host(B.conv_fwd_ex(In.to(DEV), Ker.to(DEV), 2, 1))
    ref = oconv.conv_fwd_ex(host(In), host(Ker), (2, 2), (1, 1))
    assert out.shape == ref.shape
    assert rel_err(out, ref) <= TOL["f32"]


@pytest.mark.parametrize("cfg", __import__("paper_2101_09808_amd.workloads", fromlist=["x"]).TABLE1,
                         ids=lambda c: c.name)
def test_table1_layer_full_compare(cfg):
    """Table 1 layers at batch 1 with stride and same padding: every output
    against the strided oracle."""
    In, Ker = make_inputs(cfg)
    say(f"[gpu] {cfg.name}")
    out = host(B.conv_fwd_ex(In.to(DEV), Ker.to(DEV), cfg.stride, cfg.pad))
    assert out.shape == (cfg.N, cfg.K, cfg.P, cfg.Q)
    ref = oconv.conv_fwd_ex(host(In), host(Ker), (cfg.stride,) * 2, (cfg.pad,) * 2)
    assert rel_err(out, ref) <= TOL["f32"]


# ---------------------------------------------------------------------------
# bf16 output (conv_fwd_bf16_out)

@pytest.mark.parametrize("shape_index", [0, 2], ids=["fallback_c40", "fallback_c32"])
def test_bf16_out_parity_and_rounding(shape_index):
    """bf16 Out through the fallback (fp32 workspace, then rounded): within
    one bf16 rounding of the oracle, and bit-equal to the fp32-Out result of
    the same plan rounded to nearest even by torch."""
    shape = BF16_VARIANT_SHAPES[shape_index]
    In, Ker = make_inputs(shape)
    ref = oconv.conv_fwd(host(In), host(Ker))
    In_d, Ker_d = In.to(DEV), Ker.to(DEV)
    say(f"[gpu] bf16 out {shape.name}")
    ob = B.conv_fwd_bf16_out(In_d, Ker_d)
    of = B.conv_fwd_bf16(In_d, Ker_d)
    torch.cuda.synchronize()
    assert ob.dtype == torch.bfloat16 and ob.shape == of.shape
    assert torch.equal(ob.view(torch.int16), of.to(torch.bfloat16).view(torch.int16))
    got = host(ob.float())
    scale = np.max(np.abs(ref))
    assert np.all(np.abs(got - ref) <= 2.0 ** -8 * np.abs(ref) + TOL["f32"] * scale)


def test_bf16_out_transposing_kernel_full_layer():
    """The 226x226 bf16 layer (transposing-read kernel, bf16 written by the
    kernel itself): bit-equal to the fp32-Out result rounded by torch, and
    every output within one bf16 rounding of the oracle."""
    cfg = CONFIGS[4]
    In, Ker = make_inputs(cfg)
    In_d, Ker_d = In.to(DEV), Ker.to(DEV)
    plan = B.conv_fwd_plan(*cfg.key(), dtype=B.CONV_DTYPE_BF16)
    assert B.conv_fwd_geometry(*cfg.key(), plan)["family"] == 6
    say(f"[gpu] bf16 out {cfg.name} v{plan['variant']}")
    ob = B.conv_fwd_bf16_out(In_d, Ker_d)
    of = B.conv_fwd_bf16(In_d, Ker_d)
    torch.cuda.synchronize()
    assert torch.equal(ob.view(torch.int16), of.to(torch.bfloat16).view(torch.int16))
    got = host(ob.float())
    ref = oconv.conv_fwd(host(In), host(Ker))
    assert np.all(np.abs(got - ref) <= 2.0 ** -8 * np.abs(ref) + TOL["f32"] * np.max(np.abs(ref)))


def test_bf16_out_transposing_kernel_unaligned_out():
    """The 226x226 layer's transposing kernel with Out 2 bytes past an 8-byte
    boundary: 2-byte stores, bit-equal to the fp32 result rounded by torch,
    nothing written outside Out."""
    shape = CONFIGS[4]
    In, Ker = make_inputs(shape)
    In_d, Ker_d = In.to(DEV), Ker.to(DEV)
    n = shape.N * shape.K * shape.P * shape.Q
    buf = torch.zeros(n + 8, dtype=torch.bfloat16, device=DEV)
    out = buf[1:1 + n].view(shape.N, shape.K, shape.P, shape.Q)
    assert out.data_ptr() % 8 == 2
    say(f"[gpu] bf16 out unaligned {shape.name}")
    B.conv_fwd_bf16_out(In_d, Ker_d, out=out)
    ref = B.conv_fwd_bf16(In_d, Ker_d).to(torch.bfloat16)
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16), ref.view(torch.int16))
    assert buf[0].item() == 0 and (buf[1 + n:] == 0).all()


def test_bf16_out_unaligned():
    """bf16 Out 2 bytes past an 8-byte boundary: 2-byte stores."""
    shape = BF16_VARIANT_SHAPES[2]
    In, Ker = make_inputs(shape)
    In_d, Ker_d = In.to(DEV), Ker.to(DEV)
    n = shape.N * shape.K * shape.P * shape.Q
    buf = torch.zeros(n + 8, dtype=torch.bfloat16, device=DEV)
    out = buf[1:1 + n].view(shape.N, shape.K, shape.P, shape.Q)
    assert out.data_ptr() % 8 == 2
    B.conv_fwd_bf16_out(In_d, Ker_d, out=out)
    ref = B.conv_fwd_bf16(In_d, Ker_d).to(torch.bfloat16)
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16), ref.view(torch.int16))
    assert buf[0].item() == 0 and (buf[1 + n:] == 0).all()



# ---------------------------------------------------------------------------
# Random shapes (seeded): every entry point against the oracle

def random_shapes(n=24, seed=2024):
    """Small seeded random layers: taps 1-5 (not only the compiled 1/2/3/4),
    odd extents, channel counts off every tile size, fp32 and bf16; every
    third one strided and/or padded."""
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        R, S = int(rng.integers(1, 6)), int(rng.integers(1, 6))
        H, W = int(rng.integers(R, R + 22)), int(rng.integers(S, S + 26))
        N, C, K = int(rng.integers(1, 4)), int(rng.integers(1, 41)), int(rng.integers(1, 81))
        dt = "bf16" if rng.random() < 0.35 else "f32"
        st, pd = (int(rng.integers(1, 4)), int(rng.integers(0, 3))) if i % 3 == 2 else (1, 0)
        if H + 2 * pd < R or W + 2 * pd < S:
            pd = max(R, S)
        out.append(ConvShape(f"rand{i}_{dt}", N, C, K, H, W, R, S, dt, 300 + i, st, pd))
    return out


RANDOM_SHAPES = random_shapes()


@pytest.mark.parametrize("shape", RANDOM_SHAPES, ids=lambda s: s.name)
def test_random_shape_parity(shape):
    In, Ker = make_inputs(shape)
    In_d, Ker_d = In.to(DEV), Ker.to(DEV)
    say(f"[gpu] random {shape}")
    if shape.stride != 1 or shape.pad != 0:
        ref = oconv.conv_fwd_ex(host(In), host(Ker), (shape.stride,) * 2, (shape.pad,) * 2)
        out = B.conv_fwd_ex(In_d, Ker_d, shape.stride, shape.pad)
    else:
        ref = oconv.conv_fwd(host(In), host(Ker))
        out = (B.conv_fwd_bf16 if shape.dtype == "bf16" else B.conv_fwd)(In_d, Ker_d)
    torch.cuda.synchronize()
    assert rel_err(host(out), ref) <= TOL[shape.dtype]
    if shape.dtype == "bf16" and shape.stride == 1 and shape.pad == 0:
        ob = B.conv_fwd_bf16_out(In_d, Ker_d)
        torch.cuda.synchronize()
        assert torch.equal(ob.view(torch.int16), out.to(torch.bfloat16).view(torch.int16))


@pytest.mark.gpu
def test_workspaces_reused_across_calls_and_streams():
    """The per-stream workspaces: a strided layer (rearranged Ker), then a
    split plan (partial sums), each on two streams in turn, a larger call
    growing the buffer and a smaller one reusing it; every result against
    the oracle."""
    big = ConvShape("ws_s2p1_big", 2, 16, 32, 30, 30, 3, 3, "f32", 81, 2, 1)
    small = ConvShape("ws_s2p1_small", 1, 8, 16, 12, 12, 3, 3, "f32", 82, 2, 1)
    split_shape = ConvShape("ws_split", 2, 40, 72, 11, 13, 3, 3, "f32", 83)
    split_plan = next(p for p in B.conv_fwd_candidates(*split_shape.key()) if p["split_c"] > 1
                      and B.conv_fwd_geometry(*split_shape.key(), p)["family"] == 2)
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    runs = []
    for rep in range(2):
        for si, st in enumerate(streams):
            for shape in (big, small):
                In, Ker = make_inputs(shape, seed=shape.seed + 10 * rep + si)
                In_d, Ker_d = In.to(DEV), Ker.to(DEV)
                torch.cuda.synchronize()
                with torch.cuda.stream(st):
                    out = B.conv_fwd_ex(In_d, Ker_d, shape.stride, shape.pad, stream=st)
                runs.append((shape, In, Ker, out, (shape.stride, shape.stride), (shape.pad, shape.pad), In_d, Ker_d))
            In, Ker = make_inputs(split_shape, seed=split_shape.seed + 10 * rep + si)
            In_d, Ker_d = In.to(DEV), Ker.to(DEV)
            torch.cuda.synchronize()
            with torch.cuda.stream(st):
                out = B.conv_fwd_with_plan(In_d, Ker_d, split_plan, stream=st)
            runs.append((split_shape, In, Ker, out, (1, 1), (0, 0), In_d, Ker_d))
    torch.cuda.synchronize()
    for shape, In, Ker, out, st, pd, _, _ in runs:  # (device inputs kept alive until here)
        say(f"[gpu] workspace reuse {shape.name} stride={st} pad={pd}")
        ref = oconv.conv_fwd_ex(host(In), host(Ker), st, pd)
        assert rel_err(host(out), ref) <= TOL["f32"], shape.name


def test_release_workspaces_then_reuse():
    """conv_fwd_release_workspaces frees the buffers kept for a stream; the
    next call on that stream takes a new one and gives the same result."""
    shape = ConvShape("rel_s2p1", 2, 16, 32, 30, 30, 3, 3, "f32", 85, 2, 1)
    In, Ker = make_inputs(shape)
    In_d, Ker_d = In.to(DEV), Ker.to(DEV)
    st = torch.cuda.Stream()
    torch.cuda.synchronize()
    say("[gpu] release workspaces")
    with torch.cuda.stream(st):
        a = B.conv_fwd_ex(In_d, Ker_d, shape.stride, shape.pad, stream=st)
        B.release_workspaces(st)
        b = B.conv_fwd_ex(In_d, Ker_d, shape.stride, shape.pad, stream=st)
        B.release_workspaces(st)
    st.synchronize()
    assert torch.equal(a, b)
    ref = oconv.conv_fwd_ex(host(In), host(Ker), (2, 2), (1, 1))
    assert rel_err(host(a), ref) <= TOL["f32"]
