"""The seeded input recipes have the structure they claim."""
import numpy as np
import pytest

from paper_2608_27888_amd import workloads as W


def test_zipf_cluster_sizes():
    s = W.zipf_sizes(512, 16, 1.1)
    assert s.tolist() == [169, 79, 50, 37, 29, 24, 20, 17, 15, 13, 12, 11, 10, 9, 9, 8]
    m = W.clustered_map(0, 512, s)
    assert np.array_equal(np.bincount(m, minlength=16), s)


def test_small_workloads_structure():
    t = W.small("tiny")
    assert t.tex_to_dec.tolist() == [0, 1, 0, 1] and t.n % 64 != 0
    d = W.small("divergent")
    w, h, _ = d.screen
    tex = d.tex_id.reshape(h, w)
    for y in range(0, h, 8):
        for x in range(0, w, 8):
            blk = tex[y:y + 8, x:x + 8]
            assert np.all(blk == blk[0, 0])
    for name in ("single", "divergent", "clustered4k", "wide_trilinear"):
        wl = W.small(name)
        assert wl.uv.dtype == np.float32 and np.all(wl.uv >= 0) and np.all(wl.uv < 1)
        assert wl.latents.size == wl.n_textures * wl.texture_stride
        assert wl.params.size == wl.n_decoders * wl.decoder_stride
        assert wl.dims[0] == sum(wl.channels)
        assert np.all(wl.tex_id < wl.n_textures) and np.all(wl.tex_to_dec < wl.n_decoders)
    wt = W.small("wide_trilinear")
    assert wt.mip is not None and np.all((wt.mip >= 0) & (wt.mip < 2))
    assert wt.n == 161 * 97 * 4 and np.bincount(wt.tex_to_dec).tolist() == [2] * 8


def test_reproducible():
    a, b = W.small("clustered4k", seed=3), W.small("clustered4k", seed=3)
    assert np.array_equal(a.uv, b.uv) and np.array_equal(a.latents, b.latents)
    c = W.small("clustered4k_d512", seed=3)  # same queries and grids, other decoders
    assert np.array_equal(a.tex_id, c.tex_id) and np.array_equal(a.latents, c.latents)


@pytest.mark.parametrize("k", [1, 5, 10])
def test_k_per_wave_has_k_decoders_in_every_wave(oracle, k):
    """The timing-study layout of Sec. 4.4: every 64-query wave holds exactly k decoders."""
    w = W.k_per_wave(0, 96, k)
    per, tot = oracle.divergence(w.tex_id, w.tex_to_dec, w.n_decoders, wave=64)
    full = per[: w.n // 64]
    assert np.all(full == k)
    assert w.screen == (96, 96, 1) and w.n == 96 * 96


def test_cache_round_trip(tmp_path):
    a = W.cached("divergent", 3, str(tmp_path), width=131, height=67)
    b = W.cached("divergent", 3, str(tmp_path), width=131, height=67)
    ref = W.make("divergent", 3, width=131, height=67)
    for w in (a, b):
        for k in ("latents", "params", "tex_to_dec", "tex_id", "uv"):
            assert np.array_equal(getattr(w, k), getattr(ref, k)), k
            assert getattr(w, k).dtype == getattr(ref, k).dtype, k
        assert w.mip is None and w.screen == ref.screen and w.dims == ref.dims
        assert (w.name, w.n_textures, w.res, w.channels, w.n_decoders) == \
            (ref.name, ref.n_textures, ref.res, ref.channels, ref.n_decoders)
    # another seed or size is another entry
    c = W.cached("divergent", 4, str(tmp_path), width=131, height=67)
    assert not np.array_equal(c.tex_id, a.tex_id)
    assert len(list(tmp_path.iterdir())) == 2
    m = W.cached("wide_trilinear", 0, str(tmp_path), width=17, height=9, spp=2, n_decoders=4,
                 n_textures=8)
    assert np.array_equal(m.mip, W.make("wide_trilinear", 0, width=17, height=9, spp=2,
                                        n_decoders=4, n_textures=8).mip)
