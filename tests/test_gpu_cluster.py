"""GPU parity of the clustering stage (Alg. "Overall texture processing
pipeline", Stage 2, Sec. 3.3) against the oracle, and the map it produces
driving the decode path.

Both sides run Lloyd's iteration in float64 with the same seeds; the centroid
means sum members in the same (ascending) order, so labels, group sizes,
iteration counts and centroids must agree bit for bit.  Distances are summed in
different orders (lane-strided with a butterfly on the GPU, numpy on the host),
so a label decided by a near-exact tie could differ: the tests check that the
oracle's margin between the nearest and second-nearest centroid is far above
float64 rounding before they require identical labels.
"""
import sys

import numpy as np
import pytest
import torch

from paper_2608_27888_amd import ntc
from paper_2608_27888_amd import workloads as W

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    ntc.lib()
    return torch.device("cuda:0")


def margins_ok(f, centroids, labels):
    x = f.astype(np.float64)
    d = ((x[:, None, :] - centroids[None, :, :]) ** 2).sum(-1)
    part = np.sort(d, axis=1)
    if d.shape[1] < 2:
        return True
    return bool(np.all(part[:, 1] - part[:, 0] > 1e-9 * np.maximum(part[:, 1], 1e-300)))


def check(dev, oracle, f, seeds, max_iter=100):
    g = ntc.kmeans(torch.from_numpy(f).to(dev), seeds, max_iter)
    labels, c, sizes, it, conv = oracle.kmeans(f, seeds, max_iter)
    say(f"    iterations {g.iterations} (oracle {it}), converged {g.converged}")
    assert margins_ok(f, c, labels)
    assert np.array_equal(g.assign.cpu().numpy().view(np.uint32), labels)
    assert np.array_equal(g.counts.cpu().numpy().view(np.uint32), sizes)
    assert (g.iterations, g.converged) == (it, conv)
    assert np.array_equal(g.centroids.cpu().numpy(), c)
    return g


@pytest.mark.parametrize("seed,n,m,dim,spread", [
    (0, 512, 16, 512, 0.35),    # the 4K clustered frame's 512 textures into 16 decoders
    (1, 512, 8, 512, 0.35),     # Wide + trilinear: 8 shared decoders
    (2, 1000, 37, 96, 0.9),     # overlapping groups, many iterations
    (3, 64, 64, 512, 0.35),     # one group per texture
    (4, 130, 1, 7, 0.5),        # one group: its mean
])
def test_kmeans_matches_oracle(dev, oracle, seed, n, m, dim, spread):
    f, _ = W.texture_features(seed, n, max(m, 1), dim, spread=spread)
    seeds = W.kmeans_seeds(seed, n, m)
    say(f"[kmeans] n={n} m={m} dim={dim} spread={spread}")
    check(dev, oracle, f, seeds)


def test_kmeans_hand_worked_and_ties(dev, oracle):
    say("[kmeans] 1-D hand-worked, ties and an empty group, unconverged stop")
    g = check(dev, oracle, np.array([[0.0], [1.0], [10.0], [11.0]], np.float32), [0, 1])
    assert g.assign.tolist() == [0, 0, 1, 1] and g.iterations == 3
    g = check(dev, oracle, np.array([[1.0], [1.0], [6.0]], np.float32), [0, 1])
    assert g.assign.tolist() == [1, 1, 0]
    g = check(dev, oracle, np.array([[1.0], [1.0], [6.0]], np.float32), [0, 1], max_iter=1)
    assert g.counts.tolist() == [3, 0] and not g.converged
    assert g.centroids[:, 0].tolist() == [8.0 / 3.0, 1.0]  # the empty group kept its seed


def test_kmeans_map_drives_the_decode(dev, oracle):
    """Features -> k-means labels -> texture -> decoder map -> bins + decode."""
    w = W.small("clustered4k")
    f, _ = W.texture_features(5, w.n_textures, w.n_decoders, 512)
    seeds = W.kmeans_seeds(5, w.n_textures, w.n_decoders)
    say(f"[kmeans->decode] T={w.n_textures} D={w.n_decoders} n={w.n}")
    g = check(dev, oracle, f, seeds)
    w = w.with_decoders(w.n_decoders, g.assign.cpu().numpy().view(np.uint32))
    model, q = ntc.upload(w, dev)
    bins = ntc.build_bins(q.tex_id, model.tex_to_dec, w.n_decoders)
    out = ntc.decode(model, q, bins)
    cnt, off, perm, _ = oracle.build_bins(w.tex_id, w.tex_to_dec, w.n_decoders, 64)
    assert np.array_equal(bins.perm.cpu().numpy().view(np.uint32)[: off[-1]], perm)
    assert np.abs(out.cpu().numpy() - oracle.decode(w)).max() <= 2e-3
