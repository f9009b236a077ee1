"""The layer lists against the paper's Table 1 (CPU only)."""
import csv
import os

from paper_2101_09808_amd.workloads import STRIDED_CONFIGS, TABLE1

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "table1_layers.csv")


def _table():
    with open(GOLDEN) as fh:
        rows = [ln for ln in fh if not ln.startswith("#")]
    return {r["layer"]: r for r in csv.DictReader(rows)}


def test_table1_layers_match_the_table():
    t = _table()
    assert len(TABLE1) == len(t) == 23
    for c in TABLE1:
        r = t[c.name.split("_")[1]]
        assert (c.K, c.C, c.H, c.W, c.R, c.S, c.stride) == (
            int(r["K"]), int(r["C"]), int(r["HW"]), int(r["HW"]), int(r["RS"]), int(r["RS"]), int(r["stride"]))
        assert c.N == 1 and c.pad == c.R // 2 and c.dtype == "f32"


def test_strided_configs_are_table1_layers_at_batch_32():
    t = _table()
    for c, name in zip(STRIDED_CONFIGS, ("R1", "R4", "R5")):
        r = t[name]
        assert (c.K, c.C, c.H, c.R, c.stride) == (int(r["K"]), int(r["C"]), int(r["HW"]), int(r["RS"]),
                                                   int(r["stride"]))
        assert c.N == 32 and c.pad == c.R // 2


def test_same_padding_output_extents():
    for c in TABLE1:
        assert c.P == -(-c.H // c.stride) and c.Q == -(-c.W // c.stride)
