"""The library's tile selector (host C++) against the cost-model oracle and its
own invariants (CPU only)."""
import itertools
import random
from fractions import Fraction

import pytest

from oracle import cost_model as cm
from paper_2101_09808_amd import conv as B
from paper_2101_09808_amd.workloads import CONFIGS


def divisors(n):
    return [d for d in range(1, n + 1) if n % d == 0]


def test_model_volume_matches_oracle_exactly():
    """The C++ rule of Sec. 3.2 equals the exact-rational oracle on random
    permutations and divisible tile sizes (all values are integers < 2^53)."""
    rng = random.Random(21)
    allp = list(itertools.permutations(cm.ITERS))
    for _ in range(400):
        N = {j: rng.randint(1, 64) for j in cm.ITERS}
        T = {j: rng.choice(divisors(N[j])) for j in cm.ITERS}
        p = rng.choice(allp)
        for of in (1, 2):
            got = B.conv_model_volume(p, N, T, of)
            ref = cm.volumes(p, N, T, of)
            for a in cm.ARRAYS:
                assert Fraction(got[a]) == ref[a], (a, p, N, T, of)


def test_model_volume_non_divisible_tiles():
    """Ratios N/T that are not integers are still the oracle's rationals (to
    double rounding)."""
    rng = random.Random(22)
    allp = list(itertools.permutations(cm.ITERS))
    for _ in range(300):
        N = {j: rng.randint(1, 50) for j in cm.ITERS}
        T = {j: rng.randint(1, N[j]) for j in cm.ITERS}
        p = rng.choice(allp)
        got = B.conv_model_volume(p, N, T, 2)
        ref = cm.volumes(p, N, T, 2)
        for a in cm.ARRAYS:
            assert abs(got[a] - float(ref[a])) <= 1e-12 * float(ref[a])


def test_model_volume_rejects_bad_input():
    with pytest.raises(B.ConvError):
        B.conv_model_volume("nkcrshh", dict(n=1, k=1, c=1, r=1, s=1, h=1, w=1),
                            dict(n=1, k=1, c=1, r=1, s=1, h=1, w=1))
    with pytest.raises(B.ConvError):
        B.conv_model_volume("nkcrshw", dict(n=1, k=1, c=1, r=1, s=1, h=1, w=1),
                            dict(n=2, k=1, c=1, r=1, s=1, h=1, w=1))


SHAPES = [c.key() + ((B.CONV_DTYPE_BF16 if c.dtype == "bf16" else B.CONV_DTYPE_F32),) for c in CONFIGS] + [
    (1, 3, 5, 13, 13, 3, 3, 0), (2, 7, 33, 11, 17, 2, 4, 0), (3, 16, 16, 9, 9, 1, 1, 0),
    (1, 1, 1, 1, 1, 1, 1, 0), (1, 64, 64, 58, 58, 3, 3, 0),
]


@pytest.mark.parametrize("shape", SHAPES, ids=str)
def test_plan_invariants(shape):
    *dims, dtype = shape
    N, C, K, H, W, R, S = dims
    try:
        plan = B.conv_fwd_plan(*dims, dtype=dtype)
    except B.ConvError as e:
        if dtype == B.CONV_DTYPE_BF16 and e.status == B.CONV_ENOPLAN:
            pytest.skip("no bf16 kernel variant built")
        raise
    assert plan["dtype"] == dtype
    assert 0 < plan["lds_bytes"] <= 160 * 1024
    assert plan["tile_k"] == plan["wave_k"] * plan["waves_k"]
    assert plan["wave_px"] % 16 == 0 and plan["wave_k"] % 16 == 0
    assert plan["tile_rows"] * plan["tile_cols"] <= plan["wave_px"] * plan["waves_px"]
    e = 2 if dtype == B.CONV_DTYPE_BF16 else 4
    P, Q = H - R + 1, W - S + 1
    compulsory = (N * C * H * W + K * C * R * S) * e + N * K * P * Q * 4
    assert plan["pred_bytes"]["hbm"] >= compulsory * (1 - 1e-12)
    # each level moves at least the bytes it must deliver once
    assert plan["pred_bytes"]["lds"] >= (N * C * H * W + K * C * R * S) * e * (1 - 1e-12) or R * S == 1
    # the slowest level (Sec. 5 min-max) plus the pipeline's fill and drain
    # (and a split plan's second pass)
    slowest = max(list(plan["pred_us"].values()) + [plan["pred_mfma_us"]])
    assert plan["pred_total_us"] > slowest
    # deterministic and cached
    assert B.conv_fwd_plan(*dims, dtype=dtype) == plan
    cands = B.conv_fwd_candidates(*dims, dtype=dtype)
    assert cands[0] == plan
    # ranked by predicted time times the measured factor of the kernel
    # variant (one factor per variant: every plan of a variant has the same
    # ratio of rank time to predicted time)
    assert all(x["rank_us"] <= y["rank_us"] * (1 + 1e-12) for x, y in zip(cands, cands[1:]))
    ratio = {}
    for c in cands:
        r = c["rank_us"] / c["pred_total_us"]
        assert r == pytest.approx(ratio.setdefault(c["variant"], r), rel=1e-12)


def test_enumeration_rules_for_channel_groups_and_narrow_steps():
    """Candidate-set rules of the enumerator: channel-group plans (groups of
    waves splitting each step's channels) only on grids of at most 256
    workgroups and never with a split reduction; pipeline steps of four
    channels only for layers with fewer than 16 channels."""
    from paper_2101_09808_amd.workloads import TABLE1
    shapes = [c.key() for c in CONFIGS if c.dtype == "f32"]
    shapes += [tuple(B.conv_fwd_ex_inner_shape(*c.key(), c.stride, c.pad))[:7] for c in TABLE1]
    seen_groups = seen_narrow = False
    for key in shapes:
        for p in B.conv_fwd_candidates(*key):
            g = B.conv_fwd_geometry(*key, p)
            if g["nwc"] > 1:
                seen_groups = True
                assert g["family"] == 2 and p["split_c"] == 1 and p["num_wg"] <= 256, (key, p)
                assert g["nwk"] * g["nwp"] * g["nwc"] * 64 == g["threads"]
            if g["family"] == 2 and g["tc"] < 8:
                seen_narrow = True
                assert key[1] < 16, (key, p)
    assert seen_groups and seen_narrow


def test_bf16_out_plan_pairs_its_stores():
    """conv_fwd_bf16_out's plan for a layer whose selected fp32-Out tiling
    (here 7 x 64) cannot pair bf16 stores into 16-byte pieces: the best
    candidate whose wave tile pairs them (an even number of 16-pixel blocks
    per part, in rows of an even number of blocks), as the transposing kernel
    does."""
    dims = (8, 32, 48, 226, 226, 3, 3)

    def pairs(p):
        g = B.conv_fwd_geometry(*dims, p)
        if g["family"] != 6:
            return True
        cbr = p["tile_cols"] // 16
        wp = p["tile_rows"] * cbr // 4
        pb = wp // (2 if wp % 2 == 0 else 1)
        return pb % 2 == 0 and cbr % 2 == 0

    sel = B.conv_fwd_plan(*dims, dtype=B.CONV_DTYPE_BF16)
    out = B.conv_fwd_bf16_out_plan(*dims)
    assert not pairs(sel)
    assert pairs(out)
    first = next(p for p in B.conv_fwd_candidates(*dims, dtype=B.CONV_DTYPE_BF16) if pairs(p))
    assert (out["variant"], out["tile_rows"], out["tile_cols"]) == (first["variant"], first["tile_rows"],
                                                                    first["tile_cols"])
    # a shape whose selected plan pairs keeps it
    dims2 = (2, 32, 48, 18, 42, 3, 3)
    if pairs(B.conv_fwd_plan(*dims2, dtype=B.CONV_DTYPE_BF16)):
        assert B.conv_fwd_bf16_out_plan(*dims2)["variant"] == B.conv_fwd_plan(*dims2, dtype=B.CONV_DTYPE_BF16)["variant"]
