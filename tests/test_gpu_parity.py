"""GPU parity: the HIP library against the CPU oracle on the same seeded inputs.

Binning (counts, offsets, permutation) and per-wave divergence counts must be
bit-exact; decoded channels must lie within max-abs 2e-3 of the oracle's
float64 values (the tolerance of the decode path: fp16 operands and fp16
activations, fp32 accumulation).  Stream mode and binned mode must agree bit
for bit, since a query's output depends on that query alone.
"""
import sys

import numpy as np
import pytest
import torch

from paper_2608_27888_amd import ntc
from paper_2608_27888_amd import workloads as W

pytestmark = pytest.mark.gpu

TOL = 2e-3
SMALL = ["tiny", "single", "divergent", "clustered4k", "clustered4k_d512", "wide_trilinear",
         "wide_trilinear_d512", "k5_per_wave", "k10_per_wave"]


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


def u32(t):
    return t.cpu().numpy().view(np.uint32)


@pytest.mark.parametrize("name", SMALL)
def test_bins_bit_exact(dev, oracle, name):
    w = small(name)
    say(f"[bins] {name} n={w.n} D={w.n_decoders}")
    model, q = ntc.upload(w, dev)
    bins = ntc.build_bins(q.tex_id, model.tex_to_dec, w.n_decoders)
    cnt, off, perm, bad = oracle.build_bins(w.tex_id, w.tex_to_dec, w.n_decoders, 64)
    torch.cuda.synchronize()
    assert np.array_equal(u32(bins.bin_count), cnt)
    assert np.array_equal(u32(bins.bin_offset), off)
    assert np.array_equal(u32(bins.perm)[: off[-1]], perm)
    assert ntc.device_error(bins) == bad == 0


@pytest.mark.parametrize("align", [1, 8, 64, 256])
def test_bins_invalid_ids_and_alignments(dev, oracle, align):
    rng = np.random.default_rng(align)
    T, D, n = 37, 11, 70001
    t2d = rng.integers(0, D + 1, T).astype(np.uint32)     # some textures map past D
    tex = rng.integers(0, T + 3, n).astype(np.uint32)     # some ids past T
    say(f"[bins-invalid] align={align} n={n}")
    bins = ntc.build_bins(torch.from_numpy(tex.view(np.int32)).to(dev),
                          torch.from_numpy(t2d.view(np.int32)).to(dev), D, align=align,
                          n_textures=T)
    cnt, off, perm, bad = oracle.build_bins(tex, t2d, D, align)
    assert np.array_equal(u32(bins.bin_count), cnt)
    assert np.array_equal(u32(bins.bin_offset), off)
    assert np.array_equal(u32(bins.perm)[: off[-1]], perm)
    assert bad > 0 and ntc.device_error(bins) == bad


@pytest.mark.parametrize("n", [0, 1, 3, 63, 64, 65, 2047, 2049, 4097, 8191, 8192, 8193,
                               16385, 100003])
def test_bins_edge_sizes(dev, oracle, n):
    rng = np.random.default_rng(n)
    T, D = 9, 5
    t2d = rng.integers(0, D, T).astype(np.uint32)
    tex = rng.integers(0, T, n).astype(np.uint32)
    say(f"[bins-edge] n={n}")
    tex_d = torch.from_numpy(tex.view(np.int32)).to(dev) if n else torch.zeros(0, dtype=torch.int32, device=dev)
    bins = ntc.build_bins(tex_d, torch.from_numpy(t2d.view(np.int32)).to(dev), D)
    cnt, off, perm, _ = oracle.build_bins(tex, t2d, D, 64)
    assert np.array_equal(u32(bins.bin_count), cnt)
    assert np.array_equal(u32(bins.bin_offset), off)
    assert np.array_equal(u32(bins.perm)[: off[-1]], perm)


@pytest.mark.parametrize("D", [1, 63, 64, 65])
def test_bins_register_and_lds_paths(dev, oracle, D):
    """Both sides of the 64-decoder boundary between the two-kernel path (register
    tables) and the three-kernel path (LDS tables), over several workgroups with a
    ragged last one, some ids out of range."""
    rng = np.random.default_rng(900 + D)
    T, n = 200, 3 * 16384 + 77
    t2d = rng.integers(0, D + 1, T).astype(np.uint32)     # some textures map past D
    tex = rng.integers(0, T + 2, n).astype(np.uint32)     # some ids past T
    say(f"[bins-paths] D={D} n={n}")
    bins = ntc.build_bins(torch.from_numpy(tex.view(np.int32)).to(dev),
                          torch.from_numpy(t2d.view(np.int32)).to(dev), D, n_textures=T)
    cnt, off, perm, bad = oracle.build_bins(tex, t2d, D, 64, n_textures=T)
    assert np.array_equal(u32(bins.bin_count), cnt)
    assert np.array_equal(u32(bins.bin_offset), off)
    assert np.array_equal(u32(bins.perm)[: off[-1]], perm)
    assert bad > 0 and ntc.device_error(bins) == bad


@pytest.mark.parametrize("D", [16, 512])
def test_bins_every_query_invalid(dev, oracle, D):
    """No query lands in a bin: counts and offsets all zero, every query counted."""
    n, T = 20001, 10
    t2d = np.full(T, D, dtype=np.uint32)                  # every texture maps past D
    tex = np.arange(n, dtype=np.uint32) % T
    say(f"[bins-all-invalid] D={D}")
    bins = ntc.build_bins(torch.from_numpy(tex.view(np.int32)).to(dev),
                          torch.from_numpy(t2d.view(np.int32)).to(dev), D, n_textures=T)
    assert not u32(bins.bin_count).any() and not u32(bins.bin_offset).any()
    assert ntc.device_error(bins) == n


def _bins_inputs(seed, n, T, D):
    rng = np.random.default_rng(seed)
    t2d = rng.integers(0, D + 1, T).astype(np.uint32)     # some textures map past D
    # runs of one texture (screen-coherent regions) with some ids past T
    runs = rng.integers(1, 300, n // 50 + 2)
    ids = rng.integers(0, T + 2, runs.size).astype(np.uint32)
    tex = np.repeat(ids, runs)[:n]
    if tex.size < n:
        tex = np.concatenate([tex, rng.integers(0, T, n - tex.size).astype(np.uint32)])
    return tex, t2d


@pytest.mark.parametrize("n,D", [(1_000_003, 15), (3_000_017, 16), (8_388_608, 64),
                                 (8_388_609, 5)])
def test_bins_workgroup_shapes(dev, oracle, n, D):
    """Binning at 4-, 8- and 16-wave workgroups (two kernels), at the last size
    where every wave's slice is one batch of 1024 queries (8,388,608; with 64
    decoders the three-kernel path) and one past it, with runs of one texture
    and some ids out of range."""
    T = 300
    tex, t2d = _bins_inputs(4000 + n % 1000, n, T, D)
    say(f"[bins-shapes] n={n} D={D}")
    bins = ntc.build_bins(torch.from_numpy(tex.view(np.int32)).to(dev),
                          torch.from_numpy(t2d.view(np.int32)).to(dev), D, n_textures=T)
    cnt, off, perm, bad = oracle.build_bins(tex, t2d, D, 64, n_textures=T)
    assert np.array_equal(u32(bins.bin_count), cnt)
    assert np.array_equal(u32(bins.bin_offset), off)
    assert np.array_equal(u32(bins.perm)[: off[-1]], perm)
    assert bad > 0 and ntc.device_error(bins) == bad


@pytest.mark.parametrize("shift", [1, 2, 3])
def test_bins_unaligned_ids(dev, oracle, shift):
    """tex_id that does not start on a 16-byte boundary (a slice of a larger array)."""
    rng = np.random.default_rng(shift)
    T, D, n = 23, 7, 50021
    t2d = rng.integers(0, D, T).astype(np.uint32)
    tex = rng.integers(0, T, n + shift).astype(np.uint32)
    say(f"[bins-unaligned] shift={shift}")
    tex_d = torch.from_numpy(tex.view(np.int32)).to(dev)[shift:]
    assert tex_d.data_ptr() % 16 != 0
    bins = ntc.build_bins(tex_d, torch.from_numpy(t2d.view(np.int32)).to(dev), D)
    cnt, off, perm, _ = oracle.build_bins(tex[shift:], t2d, D, 64)
    assert np.array_equal(u32(bins.bin_count), cnt)
    assert np.array_equal(u32(bins.bin_offset), off)
    assert np.array_equal(u32(bins.perm)[: off[-1]], perm)


@pytest.mark.parametrize("name", SMALL)
@pytest.mark.parametrize("wave", [64, 32])
def test_divergence_bit_exact(dev, oracle, name, wave):
    w = small(name)
    say(f"[divergence] {name} wave={wave}")
    model, q = ntc.upload(w, dev)
    per, tot = ntc.divergence_stats(q.tex_id, model.tex_to_dec, w.n_decoders, wave=wave)
    per_o, tot_o = oracle.divergence(w.tex_id, w.tex_to_dec, w.n_decoders, wave=wave)
    assert np.array_equal(u32(per), per_o)
    assert np.array_equal(tot.cpu().numpy().astype(np.uint64), tot_o)
    bins = ntc.build_bins(q.tex_id, model.tex_to_dec, w.n_decoders)
    P = int(u32(bins.bin_offset)[-1])
    perm_d = bins.perm[:P]
    per_b, tot_b = ntc.divergence_stats(q.tex_id, model.tex_to_dec, w.n_decoders, order=perm_d,
                                        wave=wave)
    per_bo, tot_bo = oracle.divergence(w.tex_id, w.tex_to_dec, w.n_decoders,
                                       order=u32(perm_d), wave=wave)
    assert np.array_equal(u32(per_b), per_bo)
    assert np.array_equal(tot_b.cpu().numpy().astype(np.uint64), tot_bo)
    assert int(tot_b[3]) == 1  # binned order: one decoder per wave


@pytest.mark.parametrize("name", ["single", "divergent", "clustered4k", "clustered4k_d512",
                                  "wide_trilinear"])
@pytest.mark.parametrize("block", [(8, 8), (16, 16), (5, 3), (64, 1)])
def test_divergence_map_bit_exact(dev, oracle, name, block):
    w = small(name)
    W_, H_, spp = w.screen
    bw, bh = block
    say(f"[divergence-map] {name} {W_}x{H_}x{spp} block {bw}x{bh}")
    model, q = ntc.upload(w, dev)
    dmap, hist, tot = ntc.divergence_map(q.tex_id, W_, H_, model.tex_to_dec, w.n_decoders,
                                         spp=spp, block_w=bw, block_h=bh, hist_len=9)
    dmap_o, hist_o, tot_o = oracle.divergence_map(w.tex_id, W_, H_, w.tex_to_dec, w.n_decoders,
                                                  spp=spp, block_w=bw, block_h=bh, hist_len=9)
    assert np.array_equal(u32(dmap), dmap_o)
    assert np.array_equal(u32(hist), hist_o)
    assert np.array_equal(tot.cpu().numpy().astype(np.uint64), tot_o)


def test_divergence_map_invalid_ids(dev, oracle):
    rng = np.random.default_rng(4)
    W_, H_, T, D = 61, 29, 17, 5
    t2d = rng.integers(0, D + 2, T).astype(np.uint32)
    tex = rng.integers(0, T + 3, W_ * H_).astype(np.uint32)
    say("[divergence-map] invalid ids")
    dmap, hist, tot = ntc.divergence_map(torch.from_numpy(tex.view(np.int32)).to(dev), W_, H_,
                                         torch.from_numpy(t2d.view(np.int32)).to(dev), D,
                                         block_w=4, block_h=4, hist_len=3, n_textures=T)
    dmap_o, hist_o, tot_o = oracle.divergence_map(tex, W_, H_, t2d, D, block_w=4, block_h=4,
                                                  hist_len=3, n_textures=T)
    assert np.array_equal(u32(dmap), dmap_o)
    assert np.array_equal(u32(hist), hist_o)
    assert np.array_equal(tot.cpu().numpy().astype(np.uint64), tot_o)


@pytest.mark.parametrize("name", SMALL)
def test_decode_matches_oracle(dev, oracle, name):
    w = small(name)
    say(f"[decode] {name} n={w.n} dims={w.dims} levels={w.res}x{w.channels} mip={w.mip is not None}")
    model, q = ntc.upload(w, dev)
    bins = ntc.build_bins(q.tex_id, model.tex_to_dec, w.n_decoders)
    out_b = ntc.decode(model, q, bins)
    out_s = ntc.decode(model, q)
    ref = oracle.decode(w)
    yb, ys = out_b.cpu().numpy(), out_s.cpu().numpy()
    err = np.abs(yb.astype(np.float64) - ref).max()
    say(f"    max abs err {err:.3e}")
    assert err <= TOL
    assert np.array_equal(yb.view(np.uint32), ys.view(np.uint32))  # modes agree bit for bit
    assert np.all((yb >= 0) & (yb <= 1))


VARIANTS = [  # (config, MLP widths or None, LeakyReLU slope or None, output dtype)
    ("clustered4k", None, 0.01, torch.float32),
    ("clustered4k", None, None, torch.float16),
    ("clustered4k", [32, 64, 64, 3], 0.01, torch.float32),
    ("clustered4k", [32, 64, 64, 3], 0.01, torch.float16),
    ("clustered4k", [32, 64, 64, 5], None, torch.float32),
    ("single", [32, 64, 64, 64, 12], 0.05, torch.float16),
    ("tiny", [16, 64, 64, 3], 0.01, torch.float16),
    ("wide_trilinear", [48, 128, 128, 128, 3], 0.01, torch.float16),
]


@pytest.mark.parametrize("name,dims,slope,dtype", VARIANTS)
def test_decode_variants(dev, oracle, name, dims, slope, dtype):
    """LeakyReLU hidden layers, RGB and other widths, fp16 output rows (Sec. 4 setup)."""
    w = small(name)
    if dims is not None:
        w = w.with_dims(dims, seed=3)
    say(f"[variant] {name} dims={w.dims} slope={slope} {dtype}")
    model, q = ntc.upload(w, dev)
    bins = ntc.build_bins(q.tex_id, model.tex_to_dec, w.n_decoders)
    out_b = ntc.decode(model, q, bins, leaky_slope=slope, out_dtype=dtype)
    out_s = ntc.decode(model, q, leaky_slope=slope, out_dtype=dtype)
    ref = oracle.decode(w, leaky_slope=slope or 0.0)
    yb = out_b.cpu().numpy()
    err = np.abs(yb.astype(np.float64) - ref).max()
    say(f"    max abs err {err:.3e}")
    assert err <= TOL
    assert torch.equal(out_b.view(torch.int16 if dtype == torch.float16 else torch.int32),
                       out_s.view(torch.int16 if dtype == torch.float16 else torch.int32))
    if dtype == torch.float16:
        # fp16 rows are the fp32 rows rounded to nearest even
        f32 = ntc.decode(model, q, bins, leaky_slope=slope, out_dtype=torch.float32)
        assert torch.equal(f32.half().view(torch.int16), out_b.view(torch.int16))


@pytest.mark.parametrize("align", [128, 256, 4096])
def test_decode_binned_other_alignments(dev, oracle, align):
    """Bins padded to 2, 4 or 64 tiles: the pad tiles hold no queries and are
    skipped; every row matches the oracle and the align-64 decode bit for bit."""
    w = small("clustered4k_d512")
    say(f"[decode align] align={align}")
    model, q = ntc.upload(w, dev)
    bins = ntc.build_bins(q.tex_id, model.tex_to_dec, w.n_decoders, align=align)
    out = ntc.decode(model, q, bins)
    bins64 = ntc.build_bins(q.tex_id, model.tex_to_dec, w.n_decoders)
    out64 = ntc.decode(model, q, bins64)
    assert np.abs(out.cpu().numpy().astype(np.float64) - oracle.decode(w)).max() <= TOL
    assert torch.equal(out.view(torch.int32), out64.view(torch.int32))


def test_decode_4096_decoders(dev, oracle):
    """The largest decoder count: 4096 textures of small grids, each with its own
    decoder (ids scattered over [0, 4096)), about three queries per bin."""
    rng = np.random.default_rng(11)
    T = D = 4096
    res, ch, dims = [16, 8], [16, 16], [32, 64, 64, 8]
    n = 3 * T + 17
    lat = W.draw_latents(11, T, res, ch)
    params = W.draw_decoders(11, D, dims)
    t2d = rng.permutation(D).astype(np.uint32)
    tex = rng.integers(0, T, n).astype(np.uint32)
    uv = rng.random((n, 2), dtype=np.float32)
    w = W.Workload("d4096", T, res, ch, lat, D, dims, params, t2d, tex, uv, None)
    say(f"[decode D=4096] n={n}")
    model, q = ntc.upload(w, dev)
    bins = ntc.build_bins(q.tex_id, model.tex_to_dec, D)
    out_b = ntc.decode(model, q, bins)
    out_s = ntc.decode(model, q)
    ref = oracle.decode(w)
    err = np.abs(out_b.cpu().numpy().astype(np.float64) - ref).max()
    say(f"    max abs err {err:.3e}")
    assert err <= TOL
    assert torch.equal(out_b.view(torch.int32), out_s.view(torch.int32))
    out_g = ntc.decode(model, q, bins, gather="staged")
    assert np.abs(out_g.cpu().numpy().astype(np.float64) - ref).max() <= TOL


def test_decode_fp16_rows_untouched_for_invalid_queries(dev, oracle):
    w = W.small("tiny").with_dims([16, 64, 64, 3], seed=1)
    w.tex_id = w.tex_id.copy()
    w.tex_id[::11] = 9
    say("[variant] invalid queries, fp16 rows")
    model, q = ntc.upload(w, dev)
    bins = ntc.build_bins(q.tex_id, model.tex_to_dec, w.n_decoders)
    out = torch.full((w.n, 3), -7.0, dtype=torch.float16, device=dev)
    ntc.decode(model, q, bins, out=out, leaky_slope=0.01, out_dtype=torch.float16)
    ref = oracle.decode(w, leaky_slope=0.01)
    bad = np.isnan(ref[:, 0])
    o = out.cpu().numpy()
    assert bad.sum() > 0 and np.all(o[bad] == -7.0)
    assert np.abs(o[~bad].astype(np.float64) - ref[~bad]).max() <= TOL


def test_decode_is_deterministic(dev):
    w = small("clustered4k")
    say("[determinism] clustered4k")
    model, q = ntc.upload(w, dev)
    b1 = ntc.build_bins(q.tex_id, model.tex_to_dec, w.n_decoders)
    o1 = ntc.decode(model, q, b1).clone()
    b2 = ntc.build_bins(q.tex_id, model.tex_to_dec, w.n_decoders)
    o2 = ntc.decode(model, q, b2)
    P = int(u32(b1.bin_offset)[-1])
    assert torch.equal(b1.bin_offset, b2.bin_offset)
    assert torch.equal(b1.perm[:P], b2.perm[:P])  # slots past P are never written
    assert torch.equal(o1.view(torch.int32), o2.view(torch.int32))


def test_decode_invalid_queries_untouched(dev, oracle):
    w = W.small("tiny")
    w.tex_id = w.tex_id.copy()
    w.tex_id[::13] = 7                         # past the last texture
    w.tex_to_dec = np.array([0, 1, 0, 9], np.uint32)  # texture 3 maps past the last decoder
    say("[invalid] tiny with bad ids")
    model, q = ntc.upload(w, dev)
    sentinel = -12345.0
    out_s = torch.full((w.n, w.out_dim), sentinel, device=dev)
    ntc.decode(model, q, out=out_s)
    bins = ntc.build_bins(q.tex_id, model.tex_to_dec, w.n_decoders)
    out_b = torch.full((w.n, w.out_dim), sentinel, device=dev)
    ntc.decode(model, q, bins, out=out_b)
    ref = oracle.decode(w)
    bad = np.isnan(ref[:, 0])
    assert bad.sum() > 0 and ntc.device_error(bins) == int(bad.sum())
    for o in (out_s.cpu().numpy(), out_b.cpu().numpy()):
        assert np.all(o[bad] == sentinel)
        assert np.abs(o[~bad] - ref[~bad]).max() <= TOL


def test_decode_texel_centres_and_far_uv(dev, oracle):
    """Queries exactly at texel centres, on edges and far outside [0, 1)."""
    w = W.small("single")
    rng = np.random.default_rng(1)
    n = 5000
    r = w.res[0]
    ix, iy = rng.integers(0, r, n), rng.integers(0, r, n)
    uv = np.stack([(ix + 0.5) / r, (iy + 0.5) / r], 1).astype(np.float32)
    uv[:500] = rng.uniform(-50, 50, (500, 2)).astype(np.float32)
    uv[500:600] = np.array([0.0, 1.0], np.float32)[rng.integers(0, 2, (100, 2))]
    w.uv, w.tex_id = np.ascontiguousarray(uv), np.zeros(n, np.uint32)
    say("[texel-centres]")
    model, q = ntc.upload(w, dev)
    out = ntc.decode(model, q).cpu().numpy()
    assert np.abs(out - oracle.decode(w)).max() <= TOL


@pytest.mark.parametrize("name,octaves,dims,slope,dtype", [
    ("clustered4k", 4, None, None, torch.float32),
    ("clustered4k", 8, None, 0.01, torch.float32),
    ("clustered4k", 4, [48, 64, 64, 3], 0.01, torch.float16),  # the Sec. 4 setup's decoder
    ("tiny", 4, None, None, torch.float32),
    ("tiny", 8, [48, 64, 64, 3], 0.01, torch.float32),
    ("single", 4, None, 0.05, torch.float32),
])
def test_decode_positional_encoding(dev, oracle, name, octaves, dims, slope, dtype):
    """Decoder input = latent features + positional encoding of (u, v) (Sec. 4
    setup), binned and stream order, against the oracle; a few queries far
    outside [0, 1) exercise the angle reduction."""
    w = small(name).with_pe(octaves, dims, seed=7)
    w.uv = w.uv.copy()
    w.uv[5::97] = np.array([[1000.3, -3.7e5]], np.float32)
    w.uv[11::131] = np.array([[-17.25, 2.0e6]], np.float32)
    say(f"[pe] {name} octaves={octaves} dims={w.dims} slope={slope} {dtype} n={w.n}")
    model, q = ntc.upload(w, dev)
    assert model.pe_octaves == octaves
    bins = ntc.build_bins(q.tex_id, model.tex_to_dec, w.n_decoders)
    out_b = ntc.decode(model, q, bins, leaky_slope=slope, out_dtype=dtype)
    out_s = ntc.decode(model, q, leaky_slope=slope, out_dtype=dtype)
    ref = oracle.decode(w, leaky_slope=slope or 0.0)
    err = np.abs(out_b.cpu().numpy().astype(np.float64) - ref).max()
    say(f"    max abs err {err:.3e}")
    assert err <= TOL
    iv = torch.int16 if dtype == torch.float16 else torch.int32
    assert torch.equal(out_b.view(iv), out_s.view(iv))


FMA_CASES = [  # (config, MLP widths or None, LeakyReLU slope or None, output dtype, PE octaves)
    ("tiny", None, None, torch.float32, 0),
    ("single", None, None, torch.float32, 0),
    ("divergent", None, None, torch.float32, 0),
    ("clustered4k_d512", None, 0.01, torch.float16, 0),
    ("k10_per_wave", None, None, torch.float32, 0),
    ("wide_trilinear", None, None, torch.float32, 0),           # mip blending, 128 wide
    ("wide_trilinear_d512", None, 0.05, torch.float16, 0),
    ("single", [32, 64, 64, 64, 16], None, torch.float32, 0),   # two hidden->hidden layers
    ("tiny", [16, 128, 128, 8], None, torch.float16, 0),
    ("clustered4k", None, 0.01, torch.float32, 4),              # positional encoding
    ("tiny", [48, 64, 64, 8], 0.01, torch.float16, 8),
]


@pytest.mark.parametrize("name,dims,slope,dtype,pe", FMA_CASES)
def test_decode_fma_engine(dev, oracle, name, dims, slope, dtype, pe):
    """The per-lane vector-FMA engine (the paper's Non-Shared FMA, Sec. 4.4)
    against the oracle, in stream order with every decoder mix of the small
    configurations (tiles with more distinct decoders than the LDS cache holds
    included); it computes the same function as the MFMA engine within
    rounding, and the cached and direct weight paths agree bit for bit."""
    w = small(name)
    if pe:
        w = w.with_pe(pe, dims, seed=7)
    elif dims is not None:
        w = w.with_dims(dims, seed=3)
    say(f"[fma] {name} dims={w.dims} slope={slope} {dtype} pe={pe} n={w.n} D={w.n_decoders}")
    model, q = ntc.upload(w, dev)
    out_f = ntc.decode(model, q, leaky_slope=slope, out_dtype=dtype, engine="fma")
    out_g = ntc.decode(model, q, leaky_slope=slope, out_dtype=dtype, engine="fma_direct")
    out_m = ntc.decode(model, q, leaky_slope=slope, out_dtype=dtype)
    ref = oracle.decode(w, leaky_slope=slope or 0.0)
    yf = out_f.cpu().numpy().astype(np.float64)
    err = np.abs(yf - ref).max()
    say(f"    max abs err {err:.3e} (vs MFMA engine {np.abs(yf - out_m.cpu().numpy()).max():.2e})")
    assert err <= TOL
    assert np.all((yf >= 0) & (yf <= 1))
    iv = torch.int16 if dtype == torch.float16 else torch.int32
    assert torch.equal(out_f.view(iv), out_g.view(iv))


@pytest.mark.parametrize("engine", ["fma", "fma_direct"])
def test_decode_fma_invalid_queries_untouched(dev, oracle, engine):
    w = W.small("tiny")
    w.tex_id = w.tex_id.copy()
    w.tex_id[::13] = 7
    w.tex_to_dec = np.array([0, 1, 0, 9], np.uint32)
    say(f"[fma-invalid] tiny with bad ids, {engine}")
    model, q = ntc.upload(w, dev)
    out = torch.full((w.n, w.out_dim), -12345.0, device=dev)
    ntc.decode(model, q, out=out, engine=engine)
    ref = oracle.decode(w)
    bad = np.isnan(ref[:, 0])
    o = out.cpu().numpy()
    assert bad.sum() > 0 and np.all(o[bad] == -12345.0)
    assert np.abs(o[~bad] - ref[~bad]).max() <= TOL


@pytest.mark.parametrize("engine", ["fma", "fma_direct"])
@pytest.mark.parametrize("n", [1, 63, 65, 255, 257, 1023, 1025, 4097])
def test_decode_fma_ragged_sizes(dev, oracle, n, engine):
    w = W.small("clustered4k")
    w.tex_id, w.uv = w.tex_id[:n].copy(), w.uv[:n].copy()
    say(f"[fma-ragged] n={n} {engine}")
    model, q = ntc.upload(w, dev)
    out = torch.full((n + 7, w.out_dim), -3.0, device=dev)
    ntc.decode(model, q, out=out[:n], engine=engine)
    o = out.cpu().numpy()
    assert np.abs(o[:n] - oracle.decode(w)).max() <= TOL
    assert np.all(o[n:] == -3.0)  # nothing written past the last row


def test_decode_fma_cache_many_decoders_per_tile(dev, oracle):
    """Every query of a 1024-query tile on its own decoder (far more distinct
    decoders than the LDS cache holds): each tile takes many passes, and every
    pass evicts slots of the previous one."""
    rng = np.random.default_rng(21)
    T = D = 300
    res, ch, dims = [16, 8], [16, 16], [32, 64, 64, 8]
    n = 5000
    lat = W.draw_latents(21, T, res, ch)
    params = W.draw_decoders(21, D, dims)
    t2d = rng.permutation(D).astype(np.uint32)
    tex = rng.integers(0, T, n).astype(np.uint32)
    uv = rng.random((n, 2), dtype=np.float32)
    w = W.Workload("fma_many", T, res, ch, lat, D, dims, params, t2d, tex, uv, None)
    say("[fma-cache] 300 decoders, random per query")
    model, q = ntc.upload(w, dev)
    out_f = ntc.decode(model, q, engine="fma")
    out_g = ntc.decode(model, q, engine="fma_direct")
    assert np.abs(out_f.cpu().numpy().astype(np.float64) - oracle.decode(w)).max() <= TOL
    assert torch.equal(out_f.view(torch.int32), out_g.view(torch.int32))
