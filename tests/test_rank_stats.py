"""Host statistics of the model-validation sweep (Sec. 9): rank correlation,
top-k loss and the plan sample (CPU only)."""
import random

import numpy as np
import pytest
from scipy import stats

import bench


@pytest.mark.parametrize("seed", range(5))
def test_spearman_matches_scipy_with_ties(seed):
    rng = random.Random(seed)
    x = [rng.choice([1.0, 2.0, 2.0, 3.5, 4.0, 7.0]) for _ in range(40)]
    y = [rng.random() for _ in range(40)]
    y[3] = y[7]  # a tie in y as well
    assert bench.spearman(x, y) == pytest.approx(stats.spearmanr(x, y).correlation, abs=1e-12)


def test_spearman_extremes():
    assert bench.spearman([1, 2, 3, 4], [10, 20, 30, 40]) == pytest.approx(1.0)
    assert bench.spearman([1, 2, 3, 4], [4, 3, 2, 1]) == pytest.approx(-1.0)
    assert np.isnan(bench.spearman([1, 1, 1], [1, 2, 3]))


def test_ranks_average_ties():
    assert bench.ranks([5.0, 1.0, 5.0, 3.0]) == [3.5, 1.0, 3.5, 2.0]


def test_topk_loss():
    t = [12.0, 10.0, 15.0, 8.0, 9.0, 20.0]
    assert bench.topk_loss(t, 1) == pytest.approx(12.0 / 8.0 - 1)
    assert bench.topk_loss(t, 2) == pytest.approx(10.0 / 8.0 - 1)
    assert bench.topk_loss(t, 5) == 0.0


def test_rank_sample_keeps_top5_and_is_uniform_without_replacement():
    cands = list(range(1000))
    idx = bench.rank_sample(cands, n=100, seed=7)
    assert len(idx) == 100 and len(set(idx)) == 100 and idx == sorted(idx)
    assert idx[:5] == [0, 1, 2, 3, 4]
    assert bench.rank_sample(cands, n=100, seed=7) == idx
    small = bench.rank_sample(list(range(30)), n=100, seed=1)
    assert small == list(range(30))
    # the sampled tail covers the range evenly (mean index near the middle)
    tails = [np.mean(bench.rank_sample(cands, n=100, seed=s)[5:]) for s in range(20)]
    assert abs(np.mean(tails) - 502) < 40
