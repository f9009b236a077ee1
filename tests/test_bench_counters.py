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
