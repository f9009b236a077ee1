"""Host logic of the benchmark's counter passes: copy calibration and the
per-layer grouping of dispatches (synthetic counter files, CPU only)."""
import csv
import os

import pytest

import bench
from paper_2101_09808_amd.workloads import CONFIGS


def _write(d, rows, counter):
    os.makedirs(d, exist_ok=True)
    with open(os.path.join(d, "x_counter_collection.csv"), "w", newline="") as fh:
        w = csv.writer(fh)
        w.writerow(["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        for i, (name, vals) in enumerate(rows):
            for v in vals:  # several hardware instances per dispatch
                w.writerow([i + 1, name, counter, v])


def test_calibrated_scales_by_the_copy_and_groups_layers(tmp_path):
    layers = list(CONFIGS[:2])
    launches = 3
    unit = 1024.0
    copy_counter = bench.COPY_BYTES / unit / 2.0  # the counter sees half the copy's bytes
    rows = [("uniform_kernel", [1.0])]
    rows += [("__runtime_copyBuffer", [copy_counter / 2, copy_counter / 2])] * bench.COPY_REPS
    for li, _ in enumerate(layers):
        rows.append(("void convfwd::k<1>", [999.0]))  # first launch: left out
        rows += [("void convfwd::k<1>", [100.0 * (li + 1), 100.0 * (li + 1)])] * (launches - 1)
        rows.append(("bfloat16_copy_kernel", [5.0]))  # a later copy of unknown size is ignored
    _write(tmp_path / "c", rows, "FETCH_SIZE")
    factor, copy_per, per = bench.calibrated(str(tmp_path / "c"), "FETCH_SIZE", unit, layers, launches)
    assert factor == pytest.approx(2.0)
    assert copy_per == pytest.approx(copy_counter)
    for li, c in enumerate(layers):
        assert per[c.name]["per_dispatch"] == pytest.approx(200.0 * (li + 1))
        assert per[c.name]["bytes_per_launch"] == pytest.approx(200.0 * (li + 1) * unit * 2.0)


def test_calibrated_rejects_a_wrong_dispatch_count(tmp_path):
    rows = [("__runtime_copyBuffer", [1.0])] * bench.COPY_REPS + [("void convfwd::k<1>", [1.0])] * 2
    _write(tmp_path / "c", rows, "WRITE_SIZE")
    with pytest.raises(SystemExit):
        bench.calibrated(str(tmp_path / "c"), "WRITE_SIZE", 1024.0, list(CONFIGS[:1]), 3)


def test_instruction_counters_are_not_scaled(tmp_path):
    rows = [("__runtime_copyBuffer", [0.0])] * bench.COPY_REPS + [("void convfwd::k<1>", [7.0])] * 3
    _write(tmp_path / "c", rows, "SQ_INSTS_LDS")
    factor, _, per = bench.calibrated(str(tmp_path / "c"), "SQ_INSTS_LDS", 1.0, list(CONFIGS[:1]), 3)
    assert factor == 1.0 and per[CONFIGS[0].name]["per_dispatch"] == 7.0


def test_split_plan_reduction_counts_with_its_launch(tmp_path):
    """A split plan's second dispatch (the range reduction) is added to the
    main kernel's counts for that launch."""
    layers = list(CONFIGS[:1])
    launches = 3
    rows = [("__runtime_copyBuffer", [10.0])] * bench.COPY_REPS
    for _ in range(launches):
        rows.append(("void convfwd::conv_f32_dma_kernel<1>", [40.0]))
        rows.append(("void convfwd::splitk_reduce_kernel<true>", [2.0]))
    _write(tmp_path / "c", rows, "WRITE_SIZE")
    _, _, per = bench.calibrated(str(tmp_path / "c"), "WRITE_SIZE", 1.0, layers, launches)
    assert per[layers[0].name]["per_dispatch"] == pytest.approx(42.0)


def test_plan_kernel_hash_follows_the_launched_kernel_and_plan():
    """The traffic figures are keyed to the launched kernel's source, its
    instance line, the geometry struct and the plan: the same plan hashes
    the same, another tile of the same variant or another variant does not."""
    from paper_2101_09808_amd import conv as B
    from paper_2101_09808_amd.workloads import BY_NAME
    c = BY_NAME[bench.HEADLINE]
    cands = B.conv_fwd_candidates(*c.key())
    p0 = cands[0]
    h0 = bench.plan_kernel_hash(c, p0)
    assert len(h0) == 16 and h0 == bench.plan_kernel_hash(c, dict(p0))
    other_tile = next(p for p in cands if p["variant"] == p0["variant"] and p["tile_cols"] != p0["tile_cols"])
    other_variant = next(p for p in cands if p["variant"] != p0["variant"])
    assert bench.plan_kernel_hash(c, other_tile) != h0
    assert bench.plan_kernel_hash(c, other_variant) != h0


def test_buffer_sets_put_twice_the_last_level_cache_of_in_behind_every_launch():
    """Out's streaming stores do not stay in the last-level cache, so the
    rotation is sized by In alone: at least 2 x 256 MB of In across the sets
    (a launch then reads In that the cache has evicted), within the cap on
    device memory."""
    mall = bench.MALL_BYTES
    for in_b, out_b in [(52_301_824, 205_520_896), (102_760_448, 25_690_112), (861_184, 802_816),
                        (14_745_600, 12_845_056)]:
        n = bench.buffer_sets(in_b, out_b)
        assert n * in_b >= 2 * mall + in_b, (in_b, n)
        assert (n - 1) * in_b < 2 * mall + in_b, (in_b, n)  # no more than needed
        assert n * (in_b + out_b) <= bench.SETS_MAX_BYTES
    # a huge Out caps the count (and never below two sets)
    assert bench.buffer_sets(1 << 20, 4 << 30) == 3  # 16 GB / (4 GB + 1 MB)
    assert bench.buffer_sets(1 << 30, 8 << 30) == 2


def test_bf16_calibration_layers_admit_every_transposing_tiling():
    """The bf16 first layers of the training and held-out sets have Out rows
    divisible by every transposing tiling's rows, so each tiling is timed on
    each of them."""
    from paper_2101_09808_amd import conv as B

    for seed in (bench.TRAIN_SEED, bench.HELDOUT_SEED):
        layers = [c for c in bench.heldout_layers(seed=seed) if c.dtype == "bf16"]
        assert len(layers) == (4 if seed == bench.TRAIN_SEED else 3)
        for c in layers:
            assert c.C == 32 and c.R == c.S == 3 and c.P % 56 == 0
            n = B.lib().conv_fwd_candidates(*c.key(), B.CONV_DTYPE_BF16, None, 0)
            cands = B.conv_fwd_candidates(*c.key(), dtype=B.CONV_DTYPE_BF16, cap=n)
            assert {211, 212, 213, 214, 215, 216} <= {p["variant"] for p in cands}, c


def _selected(c):
    from paper_2101_09808_amd import conv as B
    dt = B.CONV_DTYPE_BF16 if c.dtype == "bf16" else B.CONV_DTYPE_F32
    return B.conv_fwd_plan(*c.key(), dtype=dt)


def test_committed_counter_profiles_match_the_selected_kernels():
    """The committed counter figures (model vs counters, the headline's HBM
    traffic) were taken on the kernels and plans that the current sources
    select: a change to a selected kernel, its instance or its plan leaves
    them stale, and this fails until they are measured again."""
    import json
    from paper_2101_09808_amd.workloads import BY_NAME
    prof = os.path.join(bench.ROOT, "profiles")
    mv = json.load(open(os.path.join(prof, "model_vs_counters.json")))
    assert {l["workload"] for l in mv["layers"]} == {c.name for c in CONFIGS}
    for l in mv["layers"]:
        c = BY_NAME[l["workload"]]
        p = _selected(c)
        assert (p["variant"], bench.plan_kernel_hash(c, p)) == (l["plan_variant"], l["plan_kernel_sha"]), c.name
    t = json.load(open(bench.TRAFFIC_FILE))
    c = BY_NAME[bench.HEADLINE]
    p = _selected(c)
    assert (p["variant"], bench.plan_kernel_hash(c, p)) == (t["plan_variant"], t["kernel_sha"])


def test_model_levels_bracket_the_measured_traffic():
    """Acceptance band of the per-level model against the counters (the paper
    validates rank only; this band is the build's own): for every layer the
    fabric bytes measured (FETCH_SIZE + WRITE_SIZE, copy-scaled) lie between
    the model's compulsory bytes (its HBM level, less 2% for counter
    rounding) and 1.3x its L2 level plus Out, the traffic if no tile's
    operands were shared through the L2; and the L2->CU read requests lie
    within 0.7-1.3x the model's LDS level in 128-byte lines."""
    import json
    mv = json.load(open(os.path.join(bench.ROOT, "profiles", "model_vs_counters.json")))
    for l in mv["layers"]:
        assert l["hbm_meas"] >= 0.98 * l["hbm_pred"], l["workload"]
        assert l["hbm_meas"] <= 1.3 * max(l["l2_pred"], l["hbm_pred"]), l["workload"]
        assert 0.7 <= l["l2cu_meas"] / l["l2cu_pred"] <= 1.3, l["workload"]
