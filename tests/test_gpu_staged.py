"""GPU parity of the LDS-staged gather (ntc_decode_options.gather = staged).

The staged path computes the same function as the direct gather (Sec. 1:
bilinear taps of each query's latent levels, then its decoder's MLP) with the
taps of a tile read once into LDS and the MLP on 16x16x32 MFMAs.  Every case is
checked against the oracle's float64 values within max-abs 2e-3; fp16 rows must
be the staged fp32 rows rounded to nearest even; rows of invalid queries and
rows past the last query stay untouched.  At full size the sampled outputs are
checked against the oracle and the whole frame against the direct gather.
"""
import sys

import numpy as np
import pytest
import torch

from paper_2608_27888_amd import ntc
from paper_2608_27888_amd import workloads as W

pytestmark = pytest.mark.gpu

TOL = 2e-3
SMALL = ["tiny", "single", "divergent", "clustered4k", "clustered4k_d512", "k5_per_wave",
         "k10_per_wave"]


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    ntc.lib()
    return torch.device("cuda:0")


_cache = {}


def small(name):
    if name not in _cache:
        _cache[name] = W.small(name)
    return _cache[name]


def staged_vs_oracle(dev, oracle, w, slope=None, dtype=torch.float32, align=64):
    model, q = ntc.upload(w, dev)
    bins = ntc.build_bins(q.tex_id, model.tex_to_dec, w.n_decoders, align=align)
    out = ntc.decode(model, q, bins, leaky_slope=slope, out_dtype=dtype, gather="staged")
    ref = oracle.decode(w, leaky_slope=slope or 0.0)
    y = out.cpu().numpy().astype(np.float64)
    err = np.abs(y - ref).max()
    direct = ntc.decode(model, q, bins, leaky_slope=slope, out_dtype=dtype)
    dd = np.abs(y - direct.cpu().numpy()).max()
    say(f"    max abs err {err:.3e} (vs direct gather {dd:.2e})")
    assert err <= TOL
    assert np.all((y >= 0) & (y <= 1))
    if dtype == torch.float16:
        f32 = ntc.decode(model, q, bins, leaky_slope=slope, gather="staged")
        assert torch.equal(f32.half().view(torch.int16), out.view(torch.int16))
    return model, q, bins, out


@pytest.mark.parametrize("name", SMALL)
def test_staged_matches_oracle(dev, oracle, name):
    w = small(name)
    say(f"[staged] {name} n={w.n} D={w.n_decoders} dims={w.dims} res={w.res}x{w.channels}")
    staged_vs_oracle(dev, oracle, w)


VARIANTS = [  # (config, MLP widths or None, LeakyReLU slope or None, output dtype)
    ("clustered4k", None, 0.01, torch.float32),
    ("clustered4k", None, None, torch.float16),
    ("clustered4k", [32, 64, 64, 3], 0.01, torch.float16),   # RGB rows
    ("clustered4k", [32, 64, 64, 4], None, torch.float32),
    ("clustered4k", [32, 64, 64, 5], 0.2, torch.float32),
    ("clustered4k", [32, 64, 64, 1], None, torch.float32),
    ("single", [32, 64, 64, 64, 8], 0.05, torch.float16),    # two hidden->hidden layers
    ("single", [32, 128, 128, 8], None, torch.float32),      # hidden width 128
    ("divergent", [32, 128, 128, 128, 3], 0.01, torch.float32),
    ("tiny", [16, 64, 64, 3], 0.01, torch.float16),          # 2 levels x 8 channels
    ("tiny", [16, 128, 128, 7], None, torch.float32),
    ("tiny", [16, 64, 64, 64, 2], None, torch.float16),
]


@pytest.mark.parametrize("name,dims,slope,dtype", VARIANTS)
def test_staged_variants(dev, oracle, name, dims, slope, dtype):
    w = small(name)
    if dims is not None:
        w = w.with_dims(dims, seed=3)
    say(f"[staged variant] {name} dims={w.dims} slope={slope} {dtype}")
    staged_vs_oracle(dev, oracle, w, slope, dtype)


@pytest.mark.parametrize("name,octaves,dims,slope", [
    ("clustered4k", 4, None, None),
    ("clustered4k", 8, None, 0.01),
    ("clustered4k", 4, [48, 64, 64, 3], 0.01),
    ("tiny", 4, None, None),
    ("tiny", 8, [48, 64, 64, 8], 0.01),
])
def test_staged_positional_encoding(dev, oracle, name, octaves, dims, slope):
    w = small(name).with_pe(octaves, dims, seed=7)
    w.uv = w.uv.copy()
    w.uv[5::97] = np.array([[1000.3, -3.7e5]], np.float32)
    say(f"[staged pe] {name} octaves={octaves} dims={w.dims} slope={slope}")
    staged_vs_oracle(dev, oracle, w, slope)


@pytest.mark.parametrize("align", [128, 256])
def test_staged_other_alignments(dev, oracle, align):
    w = small("clustered4k_d512")
    say(f"[staged align] align={align}")
    staged_vs_oracle(dev, oracle, w, align=align)


def test_staged_edges_and_far_uv(dev, oracle):
    """Texel centres, the unit square's edges and uv far outside [0, 1): clamped
    quads collapse onto the edge texels, which the staging plan must share."""
    w = W.small("single")
    rng = np.random.default_rng(2)
    n = 20000
    r = w.res[0]
    ix, iy = rng.integers(0, r, n), rng.integers(0, r, n)
    uv = np.stack([(ix + 0.5) / r, (iy + 0.5) / r], 1).astype(np.float32)
    uv[:3000] = rng.uniform(-50, 50, (3000, 2)).astype(np.float32)
    uv[3000:3400] = np.array([0.0, 1.0], np.float32)[rng.integers(0, 2, (400, 2))]
    uv[3400:3800] = np.float32(-1e30)
    uv = uv[np.argsort(uv[:, 1] * 4096 + uv[:, 0], kind="stable")]  # coherent runs
    w.uv, w.tex_id = np.ascontiguousarray(uv), np.zeros(n, np.uint32)
    say("[staged edges]")
    staged_vs_oracle(dev, oracle, w)


def test_staged_invalid_queries_untouched(dev, oracle):
    w = W.small("tiny").with_dims([16, 64, 64, 3], seed=1)
    w.tex_id = w.tex_id.copy()
    w.tex_id[::13] = 7                               # past the last texture
    w.tex_to_dec = np.array([0, 1, 0, 9], np.uint32)  # texture 3 maps past the last decoder
    say("[staged invalid] tiny with bad ids")
    model, q = ntc.upload(w, dev)
    bins = ntc.build_bins(q.tex_id, model.tex_to_dec, w.n_decoders)
    ref = oracle.decode(w)
    bad = np.isnan(ref[:, 0])
    assert bad.sum() > 0 and ntc.device_error(bins) == int(bad.sum())
    for dtype in (torch.float32, torch.float16):
        out = torch.full((w.n, 3), -7.0, dtype=dtype, device=dev)
        ntc.decode(model, q, bins, out=out, out_dtype=dtype, gather="staged")
        o = out.cpu().numpy()
        assert np.all(o[bad] == -7.0)
        assert np.abs(o[~bad].astype(np.float64) - ref[~bad]).max() <= TOL


@pytest.mark.parametrize("n", [1, 2, 63, 64, 65, 127, 255, 257, 4097])
def test_staged_ragged_sizes(dev, oracle, n):
    """Bins of every fill, one-query tiles and a last tile of one query; nothing
    is written past the last row (the kernel stores each tile's rows one tile late)."""
    w = small("clustered4k")
    w = W.Workload(f"ragged{n}", w.n_textures, w.res, w.channels, w.latents, w.n_decoders,
                   w.dims, w.params, w.tex_to_dec, w.tex_id[:n].copy(), w.uv[:n].copy(), None)
    say(f"[staged ragged] n={n}")
    model, q = ntc.upload(w, dev)
    bins = ntc.build_bins(q.tex_id, model.tex_to_dec, w.n_decoders)
    out = torch.full((n + 7, w.out_dim), -3.0, device=dev)
    ntc.decode(model, q, bins, out=out[:n], gather="staged")
    o = out.cpu().numpy()
    assert np.abs(o[:n] - oracle.decode(w)).max() <= TOL
    assert np.all(o[n:] == -3.0)


def test_staged_is_deterministic(dev):
    w = small("clustered4k")
    say("[staged determinism]")
    model, q = ntc.upload(w, dev)
    bins = ntc.build_bins(q.tex_id, model.tex_to_dec, w.n_decoders)
    o1 = ntc.decode(model, q, bins, gather="staged").clone()
    o2 = ntc.decode(model, q, bins, gather="staged")
    assert torch.equal(o1.view(torch.int32), o2.view(torch.int32))


def test_staged_unsupported_shapes_raise(dev):
    w = small("wide_trilinear")  # 3 levels with mip
    model, q = ntc.upload(w, dev)
    bins = ntc.build_bins(q.tex_id, model.tex_to_dec, w.n_decoders)
    with pytest.raises(ntc.NtcError) as e:
        ntc.decode(model, q, bins, gather="staged")
    assert e.value.status == ntc.NTC_ERR_UNSUPPORTED
    w = small("tiny")
    model, q = ntc.upload(w, dev)
    with pytest.raises(ntc.NtcError) as e:
        ntc.decode(model, q, gather="staged")  # stream mode
    assert e.value.status == ntc.NTC_ERR_UNSUPPORTED


@pytest.mark.slow
@pytest.mark.parametrize("decoders", [16, 512])
def test_staged_full_clustered4k(dev, oracle, decoders):
    """The 4K frame with 16 (clustered map) or 512 decoders (one per texture)."""
    w = W.clustered4k()
    if decoders != w.n_decoders:
        w = w.with_decoders(decoders, np.arange(decoders, dtype=np.uint32))
    say(f"[staged full] clustered4k D={w.n_decoders} n={w.n}")
    model, q = ntc.upload(w, dev)
    bins = ntc.alloc_bins(w.n, w.n_decoders, 64, dev)
    ntc.build_bins(q.tex_id, model.tex_to_dec, w.n_decoders, bins=bins)
    out = torch.empty((w.n, w.out_dim), dtype=torch.float32, device=dev)
    ntc.decode(model, q, bins, out=out, gather="staged")
    direct = ntc.decode(model, q, bins)
    y = out.cpu().numpy()
    assert np.all(np.isfinite(y)) and np.all((y >= 0) & (y <= 1))
    s = np.unique(np.concatenate([np.linspace(0, w.n - 1, 32768).round().astype(np.int64),
                                  np.arange(97), np.arange(w.n - 97, w.n)]))
    err = np.abs(y[s].astype(np.float64) - oracle.decode(w, subset=s)).max()
    dd = np.abs(y - direct.cpu().numpy()).max()
    say(f"    sampled max abs err {err:.3e}; whole frame vs direct {dd:.2e}")
    assert err <= TOL
    assert dd <= 2 * TOL  # both within TOL of the exact values
