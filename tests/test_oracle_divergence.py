"""Pins of the oracle's per-window divergence count (Sec. 2, divergence map).

Checked against numpy's unique per window, and against the special cases the
definition fixes: one decoder gives exactly 1 per block, a decoder-sorted order
padded to the window size gives exactly 1, all-distinct ids give the window's
occupancy.  The metric of Eq. (normalized_ones_metric) is recomputed from the
per-window counts.
"""
import numpy as np
import pytest

PAD = 0xFFFFFFFF


@pytest.mark.parametrize("wave", [64, 32, 7])
def test_divergence_vs_unique(oracle, wave):
    rng = np.random.default_rng(11)
    T, D, n = 40, 9, 3000
    t2d = rng.integers(0, D + 1, size=T).astype(np.uint32)  # decoder D is invalid
    tex = rng.integers(0, T + 1, size=n).astype(np.uint32)  # texture T is invalid
    order = rng.permutation(n + 200).astype(np.uint32)      # entries >= n are skipped
    order[rng.random(order.size) < 0.05] = PAD
    per, tot = oracle.divergence(tex, t2d, D, order=order, wave=wave)
    exp = []
    for w in range(0, order.size, wave):
        ids = [t2d[tex[q]] for q in order[w:w + wave]
               if q < n and tex[q] < T and t2d[tex[q]] < D]
        exp.append(len(np.unique(np.array(ids, dtype=np.int64))))
    exp = np.array(exp)
    assert np.array_equal(per, exp)
    kept = exp[exp > 0]
    assert tot.tolist() == [kept.size, kept.sum(), int((kept > 1).sum()), kept.max()]


def test_single_decoder_gives_one_per_window(oracle):
    rng = np.random.default_rng(3)
    tex = rng.integers(0, 50, size=5000).astype(np.uint32)
    t2d = np.zeros(50, np.uint32)
    for order in (None, rng.permutation(5000).astype(np.uint32)):
        per, tot = oracle.divergence(tex, t2d, 1, order=order)
        assert np.all(per == 1)
        # the metric of Eq. (normalized_ones_metric) is zero iff all entries are one
        assert tot[1] - tot[0] == 0


def test_binned_order_gives_one_per_window(oracle):
    rng = np.random.default_rng(4)
    T, D = 300, 37
    t2d = rng.integers(0, D, size=T).astype(np.uint32)
    tex = rng.integers(0, T, size=20000).astype(np.uint32)
    _, _, perm, _ = oracle.build_bins(tex, t2d, D, 64)
    per, tot = oracle.divergence(tex, t2d, D, order=perm)
    assert np.all(per == 1)
    per_s, tot_s = oracle.divergence(tex, t2d, D)
    assert tot_s[1] / tot_s[0] > 10  # random stream order is highly divergent


def test_all_distinct_gives_occupancy(oracle):
    n = 64 * 5 + 13
    tex = np.arange(n, dtype=np.uint32)
    per, tot = oracle.divergence(tex, np.arange(n, dtype=np.uint32), n)
    assert per.tolist() == [64] * 5 + [13]
    assert tot.tolist() == [6, n, 6, 64]


def test_metric_equals_mean_excess(oracle):
    rng = np.random.default_rng(8)
    tex = rng.integers(0, 20, size=6400).astype(np.uint32)
    t2d = rng.integers(0, 5, size=20).astype(np.uint32)
    per, tot = oracle.divergence(tex, t2d, 5)
    metric = np.mean(np.abs(per.astype(np.float64) - 1.0))  # Eq. (normalized_ones_metric)
    assert metric == pytest.approx(tot[1] / tot[0] - 1.0, abs=1e-15)
