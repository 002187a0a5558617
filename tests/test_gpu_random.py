"""Seeded random sweep of GPU parity against the oracle: binning and divergence
over random sizes, decoder counts (up to the 4096 limit), alignments, wave
widths, invalid ids and texture layouts; the decode over random combinations
of every supported decoder shape and variant (levels x channels, hidden width,
depth, output width, mip blending, LeakyReLU, fp16 rows, small and odd level
resolutions, uv far outside [0, 1)), with the LDS-staged gather where it
applies; the 2-D divergence map over random screens, samples per pixel, block
shapes, decoder counts and invalid ids.  Bins and divergence must be bit-exact, decoded channels within 2e-3,
stream and binned order bit-identical."""
import sys

import numpy as np
import pytest
import torch

from paper_2608_27888_amd import ntc
from paper_2608_27888_amd import workloads as W

pytestmark = pytest.mark.gpu

TOL = 2e-3


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    ntc.lib()
    return torch.device("cuda:0")


def u32(t):
    return t.cpu().numpy().view(np.uint32)


def texture_stream(rng, n, T):
    """Runs of one texture (screen-coherent materials) mixed with scattered ids."""
    runs = rng.integers(1, 400, size=n // 8 + 2)
    ids = rng.integers(0, T, size=runs.size)
    tex = np.repeat(ids, runs)[:n]
    if tex.size < n:
        tex = np.concatenate([tex, rng.integers(0, T, n - tex.size)])
    scatter = rng.random(n) < rng.uniform(0.0, 0.3)
    tex[scatter] = rng.integers(0, T, int(scatter.sum()))
    return tex.astype(np.uint32)


@pytest.mark.parametrize("seed", range(16))
def test_random_bins_and_divergence(dev, oracle, seed):
    rng = np.random.default_rng(5000 + seed)
    n = int(rng.choice([int(rng.integers(1, 5000)), int(rng.integers(5000, 400_000))]))
    T = int(rng.integers(1, 700))
    D = int(rng.choice([int(rng.integers(1, 80)), int(rng.integers(80, 4097))]))
    align = int(2 ** rng.integers(0, 13))
    bad = seed % 3 == 0                     # some ids out of range
    t2d = rng.integers(0, D + (1 if bad else 0), T).astype(np.uint32)
    tex = texture_stream(rng, n, T + (2 if bad else 0))
    say(f"[random bins] seed={seed} n={n} T={T} D={D} align={align} bad={bad}")
    tex_d = torch.from_numpy(tex.view(np.int32)).to(dev)
    t2d_d = torch.from_numpy(t2d.view(np.int32)).to(dev)
    bins = ntc.build_bins(tex_d, t2d_d, D, align=align, n_textures=T)
    cnt, off, perm, nbad = oracle.build_bins(tex, t2d, D, align, n_textures=T)
    assert np.array_equal(u32(bins.bin_count), cnt)
    assert np.array_equal(u32(bins.bin_offset), off)
    assert np.array_equal(u32(bins.perm)[: off[-1]], perm)
    assert ntc.device_error(bins) == nbad
    wave = int(rng.integers(1, 65))
    for order in (None, perm):
        per, tot = ntc.divergence_stats(tex_d, t2d_d, D, wave=wave, n_textures=T,
                                        order=None if order is None else
                                        torch.from_numpy(order.view(np.int32)).to(dev))
        per_o, tot_o = oracle.divergence(tex, t2d, D, order=order, wave=wave, n_textures=T)
        assert np.array_equal(u32(per), per_o)
        assert tot.cpu().numpy().astype(np.uint64).tolist() == tot_o.tolist()


SHAPES = [(2, 8), (2, 16), (3, 16)]


def random_workload(rng, seed):
    nl, ch = SHAPES[int(rng.integers(0, 3))]
    hid = int(rng.choice([64, 128]))
    depth = int(rng.integers(1, 3))                       # hidden -> hidden layers
    out = int(rng.integers(1, 17))
    dims = [nl * ch] + [hid] * (depth + 1) + [out]
    res = sorted((int(2 ** rng.integers(1, 9)) for _ in range(nl)), reverse=True)
    if rng.random() < 0.3:
        res = [int(rng.integers(2, 300)) for _ in range(nl)]  # odd resolutions
    T = int(rng.integers(1, 40))
    D = int(rng.integers(1, 12))
    n = int(rng.integers(1, 6000))
    lat = W.draw_latents(seed, T, res, [ch] * nl)
    params = W.draw_decoders(seed, D, dims)
    t2d = rng.integers(0, D, T).astype(np.uint32)
    tex = texture_stream(rng, n, T)
    uv = rng.random((n, 2), dtype=np.float32)
    far = rng.random(n) < 0.05
    uv[far] = rng.uniform(-20, 20, (int(far.sum()), 2)).astype(np.float32)
    mip = None
    if nl == 3 and rng.random() < 0.6:
        mip = rng.uniform(-0.5, 2.5, n).astype(np.float32)
        mip[rng.random(n) < 0.2] = np.float32(rng.integers(0, 3))  # integer levels
    return W.Workload(f"random{seed}", T, res, [ch] * nl, lat, D, dims, params, t2d, tex,
                      np.ascontiguousarray(uv), mip)


@pytest.mark.parametrize("seed", range(16))
def test_random_decode(dev, oracle, seed):
    rng = np.random.default_rng(7000 + seed)
    w = random_workload(rng, seed)
    slope = float(rng.choice([0.0, 0.01, 0.2])) or None
    dtype = torch.float16 if rng.random() < 0.3 else torch.float32
    say(f"[random decode] seed={seed} dims={w.dims} res={w.res} T={w.n_textures} "
        f"D={w.n_decoders} n={w.n} mip={w.mip is not None} slope={slope} {dtype}")
    model, q = ntc.upload(w, dev)
    bins = ntc.build_bins(q.tex_id, model.tex_to_dec, w.n_decoders)
    out_b = ntc.decode(model, q, bins, leaky_slope=slope, out_dtype=dtype)
    out_s = ntc.decode(model, q, leaky_slope=slope, out_dtype=dtype)
    ref = oracle.decode(w, leaky_slope=slope or 0.0)
    err = np.abs(out_b.cpu().numpy().astype(np.float64) - ref).max()
    say(f"    max abs err {err:.3e}")
    assert err <= TOL
    iv = torch.int16 if dtype == torch.float16 else torch.int32
    assert torch.equal(out_b.view(iv), out_s.view(iv))
    if w.out_dim % 8 == 0:
        out_f = ntc.decode(model, q, leaky_slope=slope, out_dtype=dtype, engine="fma")
        assert np.abs(out_f.cpu().numpy().astype(np.float64) - ref).max() <= TOL
        out_g = ntc.decode(model, q, leaky_slope=slope, out_dtype=dtype, engine="fma_direct")
        assert torch.equal(out_f.view(iv), out_g.view(iv))
    if len(w.res) == 2 and w.mip is None and w.out_dim <= 8:
        out_g = ntc.decode(model, q, bins, leaky_slope=slope, out_dtype=dtype, gather="staged")
        err_g = np.abs(out_g.cpu().numpy().astype(np.float64) - ref).max()
        say(f"    staged gather max abs err {err_g:.3e}")
        assert err_g <= TOL


def _map_case(rng, seed):
    """Random screen, samples per pixel, block shape (both kernel paths: power-of-two
    row segments up to 64 samples and at most 16 rows, and any other shape), texture
    layout, decoder count (bitmaps of several words) and invalid ids."""
    spp = int(rng.choice([1, 1, 2, 3, 4, 8]))
    W_ = int(rng.integers(1, 300))
    H_ = int(rng.integers(1, 200))
    if rng.random() < 0.5:  # a tiled shape: block_w * spp a power of two <= 64
        g = int(rng.choice([g for g in (1, 2, 4, 8, 16, 32, 64) if g % spp == 0] or [spp]))
        bw, bh = max(1, g // spp), int(rng.integers(1, 17))
    else:
        bw, bh = int(rng.integers(1, 40)), int(rng.integers(1, 40))
    T = int(rng.integers(1, 200))
    D = int(rng.choice([int(rng.integers(1, 30)), int(rng.integers(33, 300))]))
    bad = seed % 2 == 0
    t2d = rng.integers(0, D + (2 if bad else 0), T).astype(np.uint32)
    tex = texture_stream(rng, W_ * H_ * spp, T + (3 if bad else 0))
    hist_len = int(rng.integers(1, 20))
    return W_, H_, spp, bw, bh, T, D, t2d, tex, hist_len


def _check_map(dev, oracle, W_, H_, spp, bw, bh, T, D, t2d, tex, hist_len):
    tex_d = torch.from_numpy(tex.view(np.int32)).to(dev)
    t2d_d = torch.from_numpy(t2d.view(np.int32)).to(dev)
    dmap, hist, tot = ntc.divergence_map(tex_d, W_, H_, t2d_d, D, spp=spp, block_w=bw,
                                         block_h=bh, hist_len=hist_len, n_textures=T)
    dmap_o, hist_o, tot_o = oracle.divergence_map(tex, W_, H_, t2d, D, spp=spp, block_w=bw,
                                                  block_h=bh, hist_len=hist_len, n_textures=T)
    assert np.array_equal(u32(dmap), dmap_o)
    assert np.array_equal(u32(hist), hist_o)
    assert np.array_equal(tot.cpu().numpy().astype(np.uint64), tot_o)


@pytest.mark.parametrize("seed", range(24))
def test_random_divergence_map(dev, oracle, seed):
    rng = np.random.default_rng(9000 + seed)
    case = _map_case(rng, seed)
    W_, H_, spp, bw, bh, T, D = case[:7]
    say(f"[random map] seed={seed} {W_}x{H_}x{spp} block {bw}x{bh} T={T} D={D} "
        f"blocks={((W_ + bw - 1) // bw) * ((H_ + bh - 1) // bh)} hist_len={case[-1]}")
    _check_map(dev, oracle, *case)


def test_divergence_map_one_block_of_2_20_samples(dev, oracle):
    """One block of 1024 x 1024 samples (the integer-division branch of the sample
    walk) with ids over many bitmap words, beside a second, partial block."""
    rng = np.random.default_rng(77)
    W_, H_, spp, T, D = 1500, 1024, 1, 700, 600
    t2d = rng.integers(0, D + 1, T).astype(np.uint32)
    tex = texture_stream(rng, W_ * H_ * spp, T + 2)
    say("[map] 2^20-sample block")
    _check_map(dev, oracle, W_, H_, spp, 1024, 1024, T, D, t2d, tex, 40)


@pytest.mark.parametrize("W_,H_,spp,bw,bh", [(3840, 2160, 1, 8, 8), (1920, 1080, 4, 16, 16),
                                            (999, 777, 2, 32, 1), (1000, 1000, 1, 64, 16)])
def test_divergence_map_large_frames(dev, oracle, W_, H_, spp, bw, bh):
    """Frame-sized maps, block counts that are not multiples of 16 waves."""
    rng = np.random.default_rng(W_ + H_)
    T, D = 512, 16
    t2d = rng.integers(0, D, T).astype(np.uint32)
    tex = texture_stream(rng, W_ * H_ * spp, T)
    say(f"[map] {W_}x{H_}x{spp} block {bw}x{bh}")
    _check_map(dev, oracle, W_, H_, spp, bw, bh, T, D, t2d, tex, 17)
