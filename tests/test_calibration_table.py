"""The selector's per-variant calibration table is the one its committed
measurements give: ``csrc/variant_calibration.inc`` equals what
``calibrate.py`` computes from ``calibration/ratios.txt`` (CPU only)."""
import re

from paper_2101_09808_amd import calibrate


def compiled_table():
    text = open(calibrate.OUT).read()
    return {int(a): (float(b), int(c)) for a, b, c in re.findall(r"\{(-?\d+), ([0-9.]+), (\d+)\}", text)}


def test_table_matches_the_committed_ratios():
    ratios, _ = calibrate.read_ratios()
    f, fam, counts = calibrate.factors(ratios)
    table = compiled_table()
    assert set(table) == set(f) | {-k for k in fam}
    for v, x in f.items():
        assert abs(table[v][0] - x) < 5e-5 and table[v][1] == counts[v], v
    for k, x in fam.items():
        assert abs(table[-k][0] - x) < 5e-5


def test_small_variants_take_their_family_median():
    ratios = {1: (2, [1.0, 1.25, 1.75, 2.0]), 2: (2, [2.0, 2.0, 2.5, 3.0, 3.5]), 3: (2, [9.0]), 4: (5, [3.0])}
    f, fam, counts = calibrate.factors(ratios)
    assert f[1] == 1.5 and f[2] == 2.5  # medians of four and five plans
    assert fam[2] == 2.0 and f[3] == 2.0  # one plan: the family's median of its variants' medians
    assert f[4] == 1.0  # no family median: the neutral factor
    assert counts == {1: 4, 2: 5, 3: 1, 4: 1}
