"""Host-side emulation of the kernel's index arithmetic for the plans the
library launches (CPU only): every access in bounds, every output stored
exactly once, and the emulated result equal to the oracle."""
import numpy as np
import pytest

from oracle import conv as oconv
from paper_2101_09808_amd import conv as B
from paper_2101_09808_amd.workloads import CONFIGS, ConvShape, make_inputs
from tests.kernel_emulator import emulate
from tests.test_gpu_parity import BF16_VARIANT_SHAPES, EDGE, bf16_variant_plans, VARIANT_SHAPES, _plans_per_variant, small_version


def _run(shape, plan, wgs=None):
    g = B.conv_fwd_geometry(*shape.key(), plan)
    In, Ker = make_inputs(shape)
    In = In.float().numpy().astype(np.float64)
    Ker = Ker.float().numpy().astype(np.float64)
    out, written = emulate(g, In.reshape(-1), Ker.reshape(-1), wgs)
    return g, In, Ker, out, written


def _check_all(shape, plan):
    g, In, Ker, out, written = _run(shape, plan)
    assert np.all(written == 1), "outputs not stored exactly once"
    ref = oconv.conv_fwd(In.astype(np.float32), Ker.astype(np.float32)).reshape(-1)
    assert np.max(np.abs(out - ref)) <= 1e-9 * max(1.0, np.max(np.abs(ref)))


SMALL = EDGE + [small_version(c, 1) for c in CONFIGS if c.dtype == "f32" and c.N * c.K * c.P * c.Q <= 400000]


@pytest.mark.parametrize("shape", SMALL, ids=lambda s: s.name)
def test_selected_plan_indexing(shape):
    _check_all(shape, B.conv_fwd_plan(*shape.key()))


def _variant_cases():
    cases = []
    for shape in VARIANT_SHAPES:
        plans = _plans_per_variant(shape.key())
        if shape.name.startswith("var1x1_bal"):
            # these shapes are there for the balanced pointwise family; the
            # others are emulated on the shapes before
            plans = [p for p in plans if B.conv_fwd_geometry(*shape.key(), p)["family"] == 7]
        for v in sorted({p["variant"] for p in plans}):
            cases.append(pytest.param(shape, v, id=f"{shape.name}-v{v}"))
    return cases


@pytest.mark.parametrize("shape,variant", _variant_cases())
def test_every_variant_indexing(shape, variant):
    """The plans the GPU test runs for every kernel variant."""
    plans = [p for p in _plans_per_variant(shape.key()) if p["variant"] == variant]
    assert plans
    for p in plans:
        _check_all(shape, p)


@pytest.mark.parametrize("cfg", [c for c in CONFIGS if c.dtype == "f32"], ids=lambda c: c.name)
def test_full_config_sampled_workgroups(cfg):
    """Full-size plans: emulate the first, last and some middle workgroups;
    their outputs must equal the oracle at those points."""
    plan = B.conv_fwd_plan(*cfg.key())
    G = B.conv_fwd_geometry(*cfg.key(), plan)["num_tiles"]  # output tiles (all channel ranges of each)
    rng = np.random.default_rng(1)
    wgs = sorted(set([0, 7, G // 2, G - 1] + list(rng.integers(0, G, 2))))
    wgs = [w for w in wgs if 0 <= w < G]
    g, In, Ker, out, written = _run(cfg, plan, wgs)
    assert written.max() <= 1
    idx = np.nonzero(written)[0]
    assert idx.size > 0
    ref = oconv.conv_fwd_points(In.astype(np.float32), Ker.astype(np.float32), idx)
    assert np.max(np.abs(out[idx] - ref)) <= 1e-9 * max(1.0, np.max(np.abs(ref)))


BF16_SHAPES = [
    ConvShape("bf16_multi_chunk_ktail", 2, 40, 72, 11, 13, 3, 3, "bf16", 1),
    ConvShape("bf16_one_chunk", 1, 32, 64, 20, 22, 3, 3, "bf16", 2),
    ConvShape("bf16_pointwise", 3, 16, 20, 7, 9, 1, 1, "bf16", 3),
    ConvShape("bf16_odd_width", 1, 8, 16, 6, 9, 3, 3, "bf16", 4),
]


@pytest.mark.parametrize("shape", BF16_SHAPES, ids=lambda s: s.name)
def test_bf16_plans_indexing(shape):
    from tests.kernel_emulator import emulate_bf16
    In, Ker = make_inputs(shape)
    In64 = In.float().numpy().astype(np.float64)
    Ker64 = Ker.float().numpy().astype(np.float64)
    ref = oconv.conv_fwd(In64.astype(np.float32), Ker64.astype(np.float32)).reshape(-1)
    for p in B.conv_fwd_candidates(*shape.key(), dtype=B.CONV_DTYPE_BF16)[:2]:
        g = B.conv_fwd_geometry(*shape.key(), p)
        out, written = emulate_bf16(g, In64.reshape(-1), Ker64.reshape(-1))
        assert np.all(written == 1)
        assert np.max(np.abs(out - ref)) <= 1e-9 * max(1.0, np.max(np.abs(ref)))


def test_bf16_full_config_sampled_workgroups():
    from tests.kernel_emulator import emulate_bf16
    cfg = [c for c in CONFIGS if c.dtype == "bf16"][0]
    plan = B.conv_fwd_plan(*cfg.key(), dtype=B.CONV_DTYPE_BF16)
    g = B.conv_fwd_geometry(*cfg.key(), plan)
    In, Ker = make_inputs(cfg)
    In64 = In.float().numpy().astype(np.float64).reshape(-1)
    Ker64 = Ker.float().numpy().astype(np.float64).reshape(-1)
    out, written = emulate_bf16(g, In64, Ker64, [0, g["grid"] - 1])
    assert written.max() == 1
    idx = np.nonzero(written)[0]
    ref = oconv.conv_fwd_points(In.float().numpy(), Ker.float().numpy(), idx)
    assert np.max(np.abs(out[idx] - ref)) <= 1e-9 * max(1.0, np.max(np.abs(ref)))


def _bf16_variant_cases():
    cases = []
    for shape in BF16_VARIANT_SHAPES:
        for v in sorted({p["variant"] for p in bf16_variant_plans(shape)}):
            cases.append(pytest.param(shape, v, id=f"{shape.name}-v{v}"))
    return cases


@pytest.mark.parametrize("shape,variant", _bf16_variant_cases())
def test_every_bf16_variant_indexing(shape, variant):
    """The plans the GPU test runs for every bf16 kernel variant."""
    from tests.kernel_emulator import emulate_bf16
    In, Ker = make_inputs(shape)
    In64 = In.float().numpy().astype(np.float64)
    Ker64 = Ker.float().numpy().astype(np.float64)
    ref = oconv.conv_fwd(In64.astype(np.float32), Ker64.astype(np.float32)).reshape(-1)
    plans = [p for p in bf16_variant_plans(shape) if p["variant"] == variant]
    assert plans
    for p in plans:
        g = B.conv_fwd_geometry(*shape.key(), p)
        if shape.name == "bf16_c32_k64":
            # the largest shape: the first, middle and last workgroups
            G = g["grid"]
            out, written = emulate_bf16(g, In64.reshape(-1), Ker64.reshape(-1), sorted({0, G // 2, G - 1}))
            assert written.max() == 1
            idx = np.nonzero(written)[0]
            assert np.max(np.abs(out[idx] - ref[idx])) <= 1e-9 * max(1.0, np.max(np.abs(ref)))
            continue
        out, written = emulate_bf16(g, In64.reshape(-1), Ker64.reshape(-1))
        assert np.all(written == 1)
        assert np.max(np.abs(out - ref)) <= 1e-9 * max(1.0, np.max(np.abs(ref)))


@pytest.mark.parametrize("shape_index", [2, 4])
def test_bf16_transposing_unaligned_out_indexing(shape_index):
    """Family 6 with Out off a 16-byte boundary: 4-byte stores, each output
    once."""
    from tests.kernel_emulator import emulate_bf16
    shape = BF16_VARIANT_SHAPES[shape_index]
    In, Ker = make_inputs(shape)
    In64 = In.float().numpy().astype(np.float64)
    Ker64 = Ker.float().numpy().astype(np.float64)
    ref = oconv.conv_fwd(In64.astype(np.float32), Ker64.astype(np.float32)).reshape(-1)
    plans = [p for p in bf16_variant_plans(shape) if B.conv_fwd_geometry(*shape.key(), p)["family"] == 6]
    assert plans
    g = B.conv_fwd_geometry(*shape.key(), plans[0])
    out, written = emulate_bf16(g, In64.reshape(-1), Ker64.reshape(-1), out_aligned=False)
    assert np.all(written == 1)
    assert np.max(np.abs(out - ref)) <= 1e-9 * max(1.0, np.max(np.abs(ref)))


@pytest.mark.parametrize("shape", [
    ConvShape("misaligned_1x1_vec_in", 2, 30, 40, 8, 10, 1, 1, "f32", 61),
    ConvShape("misaligned_3x3_vec_ker", 2, 24, 64, 14, 16, 3, 3, "f32", 62),
], ids=lambda s: s.name)
def test_misaligned_fallback_plan_indexing(shape):
    """The plan a call with In and Ker off 16-byte boundaries runs: the best
    candidate without vector loads of In (direct-to-LDS family) or Ker."""
    for p in B.conv_fwd_candidates(*shape.key()):
        g = B.conv_fwd_geometry(*shape.key(), p)
        if g["ker_vec"] == 1 and not (g["family"] == 2 and g["in_vec"] > 1):
            break
    else:
        pytest.fail("no plan without vector loads")
    _check_all(shape, p)


def test_split_plans_indexing():
    """The split plans the GPU test runs: every range's partial output stored
    once into its workspace slice, and the fixed-order sum equal to the oracle."""
    from tests.test_gpu_parity import SPLIT_SHAPE, split_plans
    plans = split_plans(SPLIT_SHAPE)
    assert len(plans) >= 2
    for p in plans:
        _check_all(SPLIT_SHAPE, p)


def test_tune_plans_indexing():
    """The plans the tuning GPU test times: the first four candidates of
    each of its shapes, every workgroup emulated."""
    from tests.test_gpu_parity import TUNE_SHAPES
    from tests.kernel_emulator import emulate_bf16
    for shape in TUNE_SHAPES:
        dt = B.CONV_DTYPE_BF16 if shape.dtype == "bf16" else B.CONV_DTYPE_F32
        for p in B.conv_fwd_candidates(*shape.key(), dtype=dt)[:4]:
            if dt == B.CONV_DTYPE_BF16:
                In, Ker = make_inputs(shape)
                In64 = In.float().numpy().astype(np.float64)
                Ker64 = Ker.float().numpy().astype(np.float64)
                ref = oconv.conv_fwd(In64.astype(np.float32), Ker64.astype(np.float32)).reshape(-1)
                g = B.conv_fwd_geometry(*shape.key(), p)
                out, written = emulate_bf16(g, In64.reshape(-1), Ker64.reshape(-1))
                assert np.all(written == 1)
                assert np.max(np.abs(out - ref)) <= 1e-9 * max(1.0, np.max(np.abs(ref)))
            else:
                _check_all(shape, p)



def test_phase_split_rewrite_equals_strided_definition():
    """conv_fwd_ex's rewrite (the two kernels' index maps, emulated) followed
    by Eq. (1) equals the strided, padded oracle; the library reports the
    same inner problem."""
    from tests.kernel_emulator import emulate_phase_split
    from tests.test_gpu_parity import STRIDED_SHAPES
    for shape in STRIDED_SHAPES + [ConvShape("s23p10", 1, 8, 12, 13, 10, 3, 2, "f32", 99)]:
        st = (shape.stride, shape.stride) if shape.name != "s23p10" else (2, 3)
        pd = (shape.pad, shape.pad) if shape.name != "s23p10" else (1, 0)
        In, Ker = make_inputs(shape)
        In64, Ker64 = In.float().numpy().astype(np.float64), Ker.float().numpy().astype(np.float64)
        Inp, Kp, inner = emulate_phase_split(In64, Ker64, st, pd)
        assert tuple(B.conv_fwd_ex_inner_shape(*shape.key(), st, pd)) == inner
        ref = oconv.conv_fwd_ex(In64.astype(np.float32), Ker64.astype(np.float32), st, pd)
        got = oconv.conv_fwd(Inp.astype(np.float32), Kp.astype(np.float32))
        assert got.shape == ref.shape
        assert np.max(np.abs(got - ref)) <= 1e-12 * max(1.0, np.max(np.abs(ref)))


def test_strided_inner_plans_indexing():
    """The plans the strided GPU tests run (conv_fwd_ex_plan): on the inner
    stride-1 problem, or reading In through the phase mapping."""
    from tests.kernel_emulator import emulate_bf16, emulate_phase_split
    from tests.test_gpu_parity import STRIDED_SHAPES
    for shape in STRIDED_SHAPES:
        inner = B.conv_fwd_ex_inner_shape(*shape.key(), shape.stride, shape.pad)
        ish = ConvShape(shape.name + "_inner", *inner[:7], shape.dtype, shape.seed)
        dt = B.CONV_DTYPE_BF16 if shape.dtype == "bf16" else B.CONV_DTYPE_F32
        p, direct = B.conv_fwd_ex_plan(*shape.key(), shape.stride, shape.pad, dtype=dt)
        g = B.conv_fwd_ex_geometry(*shape.key(), shape.stride, shape.pad, p)
        assert bool(g["nph"]) == direct
        if direct:
            In, Ker = make_inputs(shape)
            In64, Ker64 = In.float().numpy().astype(np.float64), Ker.float().numpy().astype(np.float64)
            st, pd = (shape.stride, shape.stride), (shape.pad, shape.pad)
            _, Kp, _ = emulate_phase_split(In64, Ker64, st, pd)
            ref = oconv.conv_fwd_ex(In64.astype(np.float32), Ker64.astype(np.float32), st, pd).reshape(-1)
            out, written = emulate(g, In64.reshape(-1), Kp.reshape(-1))
            assert np.all(written == 1)
            assert np.max(np.abs(out - ref)) <= 1e-9 * max(1.0, np.max(np.abs(ref)))
        elif dt == B.CONV_DTYPE_BF16:
            In, Ker = make_inputs(ish)
            In64 = In.float().numpy().astype(np.float64)
            Ker64 = Ker.float().numpy().astype(np.float64)
            ref = oconv.conv_fwd(In64.astype(np.float32), Ker64.astype(np.float32)).reshape(-1)
            out, written = emulate_bf16(B.conv_fwd_geometry(*ish.key(), p), In64.reshape(-1), Ker64.reshape(-1))
            assert np.all(written == 1)
            assert np.max(np.abs(out - ref)) <= 1e-9 * max(1.0, np.max(np.abs(ref)))
        else:
            _check_all(ish, p)



def _direct_cases():
    from tests.test_gpu_parity import STRIDED_SHAPES
    cases = [s for s in STRIDED_SHAPES if s.dtype == "f32"]
    # stride 1 with same padding, and a 1x1 stride-2 layer on a channel-group kernel
    cases += [ConvShape("pad1_3x3", 2, 24, 40, 13, 11, 3, 3, "f32", 71, 1, 1),
              ConvShape("s2_1x1_c64", 1, 64, 72, 14, 12, 1, 1, "f32", 72, 2, 0),
              # a padded 1x1 layer: the balanced pointwise kernel reads zeros
              # for the border pixels and still stores them
              ConvShape("s2p1_1x1_c128", 2, 128, 40, 15, 13, 1, 1, "f32", 73, 2, 1)]
    return cases


@pytest.mark.parametrize("shape", _direct_cases(), ids=lambda s: s.name)
def test_direct_phase_addressing_indexing(shape):
    """conv_fwd_ex's direct path: the inner plan's direct-to-LDS kernel reads
    the caller's In through the phase mapping (zero outside the image) and the
    rearranged Ker; every inner plan of that family which takes the mapping,
    one per variant, against the strided, padded oracle."""
    from tests.kernel_emulator import emulate_phase_split
    In, Ker = make_inputs(shape)
    In64, Ker64 = In.float().numpy().astype(np.float64), Ker.float().numpy().astype(np.float64)
    st, pd = (shape.stride, shape.stride), (shape.pad, shape.pad)
    _, Kp, inner = emulate_phase_split(In64, Ker64, st, pd)
    ref = oconv.conv_fwd_ex(In64.astype(np.float32), Ker64.astype(np.float32), st, pd).reshape(-1)
    plans, seen = [], set()
    for p in B.conv_fwd_candidates(*inner[:7]):
        g = B.conv_fwd_ex_geometry(*shape.key(), st, pd, p)
        if g["nph"] and p["variant"] not in seen:
            seen.add(p["variant"])
            plans.append((p, g))
    if shape.name == "s3p2_5x5":
        # nine phases per channel: no pipeline step holds whole channels, so
        # conv_fwd_ex phase-splits In first
        assert not plans and B.conv_fwd_ex_geometry(*shape.key(), st, pd, B.conv_fwd_plan(*inner[:7]))["nph"] == 0
        return
    assert plans
    for p, g in plans:
        out, written = emulate(g, In64.reshape(-1), Kp.reshape(-1))
        assert np.all(written == 1), p
        assert np.max(np.abs(out - ref)) <= 1e-9 * max(1.0, np.max(np.abs(ref))), p
    sel = B.conv_fwd_plan(*inner[:7])
    if B.conv_fwd_geometry(*inner[:7], sel)["family"] == 2:
        assert B.conv_fwd_ex_geometry(*shape.key(), st, pd, sel)["nph"] in (0, inner[1] // shape.C)


@pytest.mark.parametrize("shape", [
    ConvShape("s2_1x1_n32_c64_k128_in56", 32, 64, 128, 56, 56, 1, 1, "f32", 74, 2, 0),
    ConvShape("s2p1_1x1_n8_c64_k64_in56", 8, 64, 64, 56, 56, 1, 1, "f32", 75, 2, 1),
], ids=lambda s: s.name)
def test_bal_direct_phase_addressing_indexing(shape):
    """conv_fwd_ex's plan for strided (and padded) 1x1 layers of this size:
    the balanced pointwise kernel reading the caller's In through the phase
    mapping; the first, a middle and the last workgroups, every output they
    store against the strided, padded oracle (the others store nothing)."""
    p, direct = B.conv_fwd_ex_plan(*shape.key(), shape.stride, shape.pad)
    st, pd = (shape.stride, shape.stride), (shape.pad, shape.pad)
    g = B.conv_fwd_ex_geometry(*shape.key(), st, pd, p)
    assert direct and g["family"] == 7 and g["nph"] == 1
    In, Ker = make_inputs(shape)
    In64, Ker64 = In.numpy().astype(np.float64), Ker.numpy().astype(np.float64)
    ref = oconv.conv_fwd_ex(In.numpy(), Ker.numpy(), st, pd).reshape(-1)
    G = g["grid"]
    out, written = emulate(g, In64.reshape(-1), Ker64.reshape(-1), wgs=[0, G // 2, G - 1])
    assert written.max() == 1 and written.sum() > 0
    hit = written == 1
    assert np.max(np.abs(out[hit] - ref[hit])) <= 1e-9 * max(1.0, np.max(np.abs(ref)))
    # every output of those workgroups' pixels (128-pixel block j at
    # (j G + p) 128, the 16-pixel tail at NB G 128 + 16 p) and 64-row k
    # tiles is stored
    PQ = ref.size // (shape.N * shape.K)
    i = np.arange(ref.size)
    px, k = i % PQ + (i // (shape.K * PQ)) * PQ, (i // PQ) % shape.K
    GP, NB = g["tiles_rows"], g["max_ni"]
    mine = np.zeros(ref.size, bool)
    for b in (0, G // 2, G - 1):
        kt, pg = b % g["tiles_k"], b // g["tiles_k"]
        own = (px >= NB * GP * 128 + 16 * pg) & (px < NB * GP * 128 + 16 * pg + 16)
        for j in range(NB):
            own |= (px >= (j * GP + pg) * 128) & (px < (j * GP + pg + 1) * 128)
        mine |= own & (k // 64 == kt)
    assert np.array_equal(hit, mine)


PS_TWINS = {118: 192, 111: 192}  # regular variant -> phase-skip variant, same wave tile


@pytest.mark.parametrize("shape", [
    ConvShape("s2p1_3x3_c16", 2, 16, 32, 20, 20, 3, 3, "f32", 81, 2, 1),
    ConvShape("s2p0_3x3_c12_odd", 1, 12, 24, 17, 15, 3, 3, "f32", 82, 2, 0),
    ConvShape("s2p1_3x3_c36", 2, 36, 40, 13, 16, 3, 3, "f32", 83, 2, 1),
    ConvShape("s2p0_3x3_c18_partial_chunk", 1, 18, 24, 21, 21, 3, 3, "f32", 84, 2, 0),
], ids=lambda s: s.name)
def test_phase_skip_indexing(shape):
    """Phase-skip variants (stride-2 odd-tap layers through conv_fwd_ex):
    each tiling of the inner problem's candidates on the twin with four input
    channels per step, phase-major LDS chunks and the zero-tap steps left
    out, against the strided, padded oracle (a wrongly skipped tap, or a
    channel or phase mixed up, changes the result)."""
    from tests.kernel_emulator import emulate_phase_split
    In, Ker = make_inputs(shape)
    In64, Ker64 = In.float().numpy().astype(np.float64), Ker.float().numpy().astype(np.float64)
    st, pd = (shape.stride, shape.stride), (shape.pad, shape.pad)
    _, Kp, inner = emulate_phase_split(In64, Ker64, st, pd)
    ref = oconv.conv_fwd_ex(In64.astype(np.float32), Ker64.astype(np.float32), st, pd).reshape(-1)
    done = set()
    for p in B.conv_fwd_candidates(*inner[:7]):
        ps = PS_TWINS.get(p["variant"])
        key = (ps, p["tile_rows"], p["tile_cols"], p["waves_k"], p["split_c"])
        if ps is None or key in done:
            continue
        q = dict(p, variant=ps)
        try:
            g = B.conv_fwd_ex_geometry(*shape.key(), st, pd, q)
        except B.ConvError:
            continue
        done.add(key)
        assert g["phase_skip"] == 1 and g["nph"] == 4
        with pytest.raises(B.ConvError):
            B.conv_fwd_geometry(*inner[:7], q)  # never on the plain problem
        out, written = emulate(g, In64.reshape(-1), Kp.reshape(-1))
        assert np.all(written == 1), q
        assert np.max(np.abs(out - ref)) <= 1e-9 * max(1.0, np.max(np.abs(ref))), q
    assert {k[0] for k in done} == {192}, done


def test_phase_skip_selected_for_the_strided_3x3_layer():
    """conv_fwd_ex's plan for the 3x3 stride-2 layer at batch 32 is a
    phase-skip variant reading In directly; three of its workgroups emulated
    against the oracle."""
    from tests.kernel_emulator import emulate_phase_split
    from paper_2101_09808_amd.workloads import BY_NAME
    shape = BY_NAME["conv3x3s2p1_n32_c64_k128_in56"]
    p, direct = B.conv_fwd_ex_plan(*shape.key(), shape.stride, shape.pad)
    st, pd = (shape.stride,) * 2, (shape.pad,) * 2
    g = B.conv_fwd_ex_geometry(*shape.key(), st, pd, p)
    assert direct and g["phase_skip"] == 1
    In, Ker = make_inputs(shape)
    In64, Ker64 = In.numpy().astype(np.float64), Ker.numpy().astype(np.float64)
    _, Kp, _ = emulate_phase_split(In64[:1], Ker64, st, pd)  # the rearranged Ker (batch-independent)
    ref = oconv.conv_fwd_ex(In.numpy(), Ker.numpy(), st, pd).reshape(-1)
    T = g["num_tiles"]
    out, written = emulate(g, In64.reshape(-1), Kp.reshape(-1), wgs=[0, T // 2, T - 1])
    hit = written == 1
    assert written.max() == 1 and hit.sum() > 0
    assert np.max(np.abs(out[hit] - ref[hit])) <= 1e-9 * max(1.0, np.max(np.abs(ref)))


@pytest.mark.parametrize("shape_index,aligned", [(2, True), (4, True), (2, False)])
def test_bf16_transposing_bf16_out_indexing(shape_index, aligned):
    """Family 6 writing bf16 Out: 16-byte stores of eight pixels from lane
    pairs of neighbouring blocks (2-byte stores when Q % 8 != 0, Out is not
    16-byte aligned or the blocks do not pair), each output once."""
    from tests.kernel_emulator import emulate_bf16
    shape = BF16_VARIANT_SHAPES[shape_index]
    In, Ker = make_inputs(shape)
    In64 = In.float().numpy().astype(np.float64)
    Ker64 = Ker.float().numpy().astype(np.float64)
    ref = oconv.conv_fwd(In64.astype(np.float32), Ker64.astype(np.float32)).reshape(-1)
    for p in [p for p in bf16_variant_plans(shape) if B.conv_fwd_geometry(*shape.key(), p)["family"] == 6]:
        out, written = emulate_bf16(B.conv_fwd_geometry(*shape.key(), p), In64.reshape(-1), Ker64.reshape(-1),
                                    out_aligned=aligned, out_bf16=True)
        assert np.all(written == 1)
        assert np.max(np.abs(out - ref)) <= 1e-9 * max(1.0, np.max(np.abs(ref)))



def test_random_shapes_emulated():
    """The plans the random-shape GPU test runs (the selected plan of each
    layer, or of its inner stride-1 problem; bf16 layers without a bf16
    kernel run the fp32 plan on widened inputs), every workgroup emulated."""
    from tests.kernel_emulator import emulate_bf16, emulate_phase_split
    from tests.test_gpu_parity import RANDOM_SHAPES
    for shape in RANDOM_SHAPES:
        In, Ker = make_inputs(shape)
        In64, Ker64 = In.float().numpy().astype(np.float64), Ker.float().numpy().astype(np.float64)
        st, pd = (shape.stride,) * 2, (shape.pad,) * 2
        if shape.stride != 1 or shape.pad != 0:
            In64, Ker64, inner = emulate_phase_split(In64, Ker64, st, pd)
            key = inner[:7]
        else:
            key = shape.key()
        ref = oconv.conv_fwd(In64.astype(np.float32), Ker64.astype(np.float32)).reshape(-1)
        dt = B.CONV_DTYPE_BF16 if shape.dtype == "bf16" else B.CONV_DTYPE_F32
        try:
            p = B.conv_fwd_plan(*key, dtype=dt)
        except B.ConvError as e:
            assert dt == B.CONV_DTYPE_BF16 and e.status == B.CONV_ENOPLAN
            dt, p = B.CONV_DTYPE_F32, B.conv_fwd_plan(*key)  # widened to fp32
        g = B.conv_fwd_geometry(*key, p)
        if g["family"] in (3, 6):
            out, written = emulate_bf16(g, In64.reshape(-1), Ker64.reshape(-1))
        else:
            out, written = emulate(g, In64.reshape(-1), Ker64.reshape(-1))
        assert np.all(written == 1), shape
        assert np.max(np.abs(out - ref)) <= 1e-9 * max(1.0, np.max(np.abs(ref))), shape
