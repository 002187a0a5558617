"""GPU parity of the gather step alone (ntc_gather_features): the feature vector
of every query, the bilinear samples of its texture's latent levels (Sec. 1,
"latent pyramids or grids"), concatenated finest first, levels blended by mip.

Pinned two ways.  At the texel centres of a power-of-two level (mip 0) the
bilinear weights are exactly (1, 0, 0, 0), so that slot must equal the stored
latents bit for bit: the definition itself, no oracle involved.  Elsewhere the
rows are checked against the oracle's float64 features within a bound that the
fp16 arithmetic fixes: with the four weights (summing to one) rounded to fp16
and every product and sum rounded once, a feature is off by at most
6 u max|T| (u = 2^-11, T the four taps); with a mip blend (two interpolations,
a subtraction, t rounded to fp16, one fused multiply-add) by at most
12 u max|T|.  The tests take max|T| over the whole latent pool.
"""
import dataclasses
import sys

import numpy as np
import pytest
import torch

from paper_2608_27888_amd import ntc
from paper_2608_27888_amd import workloads as W

pytestmark = pytest.mark.gpu

U = 2.0 ** -11
SHAPES = {"tiny": (2, 8), "single": (2, 16), "clustered4k": (2, 16), "wide_trilinear": (3, 16)}


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    ntc.lib()
    return torch.device("cuda:0")


def bound(w):
    lat = np.abs(W.bits_to_f32(w.latents)).max()
    return (12.0 if w.mip is not None else 6.0) * U * float(lat) * 1.0001


@pytest.mark.parametrize("name", sorted(SHAPES))
def test_gather_matches_oracle(dev, oracle, name):
    w = W.small(name)
    assert (w.n_levels, w.channels[0]) == SHAPES[name]
    say(f"[gather] {name} n={w.n} levels={list(zip(w.res, w.channels))} mip={w.mip is not None}")
    model, q = ntc.upload(w, dev)
    f32 = ntc.gather_features(model, q)
    ref = oracle.features(w, pe_octaves=0)
    err = np.abs(f32.cpu().numpy().astype(np.float64) - ref).max()
    say(f"    max abs err {err:.3e}, bound {bound(w):.3e}")
    assert err <= bound(w)
    # fp16 rows are the same values: the fp32 rows are them widened exactly
    f16 = ntc.gather_features(model, q, out_dtype=torch.float16)
    assert torch.equal(f32.half().view(torch.int16), f16.view(torch.int16))


@pytest.mark.parametrize("name", ["tiny", "clustered4k"])
def test_gather_texel_centres_are_the_latents(dev, name):
    """uv at the centres of level l's texels (power-of-two resolutions): slot l
    is the stored latent, bit for bit."""
    w = W.small(name)
    rng = np.random.default_rng(7)
    n = 4099
    tex = rng.integers(0, w.n_textures, n).astype(np.uint32)
    offs = W.level_offsets(w.res, w.channels)
    for l, (r, c) in enumerate(zip(w.res, w.channels)):
        assert r & (r - 1) == 0
        i, j = rng.integers(0, r, n), rng.integers(0, r, n)
        uv = np.stack([(i + 0.5) / r, (j + 0.5) / r], axis=1).astype(np.float32)
        ww = dataclasses.replace(w, tex_id=tex, uv=uv, mip=None, screen=None)
        model, q = ntc.upload(ww, dev)
        out = ntc.gather_features(model, q, out_dtype=torch.float16).cpu().numpy().view(np.uint16)
        F = sum(w.channels)
        lat = w.latents.reshape(w.n_textures, -1)
        idx = offs[l] + (j * r + i)[:, None] * c + np.arange(c)[None, :]
        want = lat[tex[:, None], idx]
        say(f"[gather-centres] {name} level {l} res {r}")
        assert np.array_equal(out.reshape(n, F)[:, l * c:(l + 1) * c], want)


@pytest.mark.parametrize("n", [1, 63, 64, 65, 1000, 4097])
def test_gather_ragged_sizes_and_invalid_rows(dev, n):
    """Any n: the rows equal those of the whole stream; rows of queries with an
    out-of-range texture stay untouched."""
    w = W.small("wide_trilinear")
    model, q = ntc.upload(w, dev)
    full = ntc.gather_features(model, q)
    tex = w.tex_id[:n].copy()
    bad = np.arange(n) % 7 == 3
    tex[bad] = w.n_textures + 5
    ww = dataclasses.replace(w, tex_id=tex, uv=w.uv[:n], mip=w.mip[:n], screen=None)
    model_n, q_n = ntc.upload(ww, dev)
    out = torch.full((n, sum(w.channels)), 7.25, dtype=torch.float32, device=dev)
    ntc.gather_features(model_n, q_n, out=out)
    say(f"[gather-ragged] n={n}")
    o = out.cpu().numpy()
    assert np.all(o[bad] == 7.25)
    assert np.array_equal(o[~bad], full[:n].cpu().numpy()[~bad])
