"""Pins of the oracle's clustering (Stage 2 of Alg. "Overall texture processing
pipeline", Sec. 3.3) and of the gradual-freezing factor (Sec. 3.2), and the
library's host-side freezing factor against the oracle (no GPU needed)."""
import math

import numpy as np
import pytest

from oracle import oracle as O
from paper_2608_27888_amd import workloads as W


def test_kmeans_hand_worked_1d():
    # points 0, 1, 10, 11 seeded at 0 and 1: iteration 1 labels {0}, {1, 10, 11}
    # (centroids 0 and 22/3); iteration 2 labels {0, 1}, {10, 11} (0.5 and 10.5);
    # iteration 3 changes nothing.
    labels, c, sizes, it, conv = O.kmeans(np.array([[0.0], [1.0], [10.0], [11.0]]), [0, 1])
    assert labels.tolist() == [0, 0, 1, 1]
    assert c[:, 0].tolist() == [0.5, 10.5]
    assert sizes.tolist() == [2, 2] and it == 3 and conv


def test_kmeans_ties_and_empty_group():
    # two seeds on one point (1): every distance ties and goes to group 0, which
    # becomes {1, 1, 6} with mean 8/3 while group 1 is empty and keeps its
    # centroid 1; then both 1s move to group 1 (0 < 25/9) and 6 stays
    # (100/9 < 25); the next iteration changes nothing.
    labels, c, sizes, it, conv = O.kmeans(np.array([[1.0], [1.0], [6.0]]), [0, 1])
    assert labels.tolist() == [1, 1, 0]
    assert c[:, 0].tolist() == [6.0, 1.0]
    assert sizes.tolist() == [1, 2] and it == 3 and conv
    # stopped after one iteration: the tie rule and the kept centroid alone decide
    labels, c, sizes, it, conv = O.kmeans(np.array([[1.0], [1.0], [6.0]]), [0, 1], max_iter=1)
    assert labels.tolist() == [0, 0, 0] and sizes.tolist() == [3, 0]
    assert c[:, 0].tolist() == [8.0 / 3.0, 1.0] and it == 1 and not conv


def test_kmeans_single_group_is_the_mean():
    f, _ = W.texture_features(3, 50, 4, 16)
    labels, c, sizes, it, conv = O.kmeans(f, [7])
    assert np.all(labels == 0) and sizes.tolist() == [50] and it == 2 and conv
    assert np.allclose(c[0], f.astype(np.float64).mean(axis=0), rtol=0, atol=1e-12)


def test_kmeans_recovers_separated_groups():
    # one seed inside every generating group: the partition found is the
    # generating one, group g being the group of seed g
    f, group = W.texture_features(1, 300, 8, 64, spread=0.2)
    seeds = [int(np.nonzero(group == g)[0][0]) for g in range(8)]
    labels, _, sizes, _, conv = O.kmeans(f, seeds)
    assert conv
    assert np.array_equal(group[seeds][labels], group)
    assert sizes.tolist() == np.bincount(group, minlength=8)[group[seeds]].tolist()


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_kmeans_converged_result_is_a_fixed_point(seed):
    f, _ = W.texture_features(seed, 256, 16, 128, spread=0.8)
    seeds = W.kmeans_seeds(seed, 256, 12)
    labels, c, sizes, it, conv, inertia = O.kmeans(f, seeds, history=True)
    assert conv and it >= 2
    x = f.astype(np.float64)
    d = ((x[:, None, :] - c[None, :, :]) ** 2).sum(-1)
    assert np.array_equal(labels, d.argmin(axis=1))           # nearest centroid
    for g in range(12):
        if sizes[g]:
            assert np.allclose(c[g], x[labels == g].mean(axis=0), rtol=0, atol=1e-12)
    assert sizes.sum() == 256 and np.array_equal(sizes, np.bincount(labels, minlength=12))
    # Lloyd's steps never increase the within-group sum of squares
    assert all(b <= a + 1e-9 for a, b in zip(inertia, inertia[1:]))


def test_freeze_scale_values():
    lam = O.freeze_scale
    s, T = 50.0, 30.0
    assert lam(0.0, None, T) == 1.0 and lam(1e6, None, T) == 1.0      # never frozen
    assert lam(s - 1, s, T) == 1.0 and lam(s, s, T) == 1.0
    assert lam(s + T, s, T) == 0.0 and lam(s + T + 5, s, T) == 0.0
    # cos(pi/3) = 1/2, cos(pi/2) = 0, cos(2 pi/3) = -1/2
    assert lam(s + T / 3, s, T) == pytest.approx(0.75, abs=1e-15)
    assert lam(s + T / 2, s, T) == pytest.approx(0.5, abs=1e-15)
    assert lam(s + 2 * T / 3, s, T) == pytest.approx(0.25, abs=1e-15)
    e = np.linspace(s - 10, s + T + 10, 401)
    v = np.array([lam(x, s, T) for x in e])
    assert np.all(np.diff(v) <= 1e-15) and v.min() >= 0 and v.max() <= 1
    # half-cosine symmetry about the middle of the window
    u = np.linspace(0, T, 31)
    assert np.allclose([lam(s + a, s, T) + lam(s + T - a, s, T) for a in u], 1.0, atol=1e-15)


def test_library_freeze_scale_matches_oracle():
    from paper_2608_27888_amd import ntc

    for s, T in [(50.0, 30.0), (0.0, 1.0), (10.0, 0.0), (10.0, -3.0), (75.0, 25.0)]:
        for e in np.linspace(-5, 120, 251):
            assert ntc.freeze_scale(e, s, T) == pytest.approx(O.freeze_scale(e, s, T), abs=1e-15)
    assert ntc.freeze_scale(3.0, None, 10.0) == 1.0
    assert math.isclose(ntc.freeze_scale(60.0, 50.0, 20.0), 0.5, abs_tol=1e-15)
