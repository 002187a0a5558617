"""GPU parity at the full configuration sizes, in the launch configuration bench.py times.

Binning, permutation and divergence counts are compared bit for bit with the
oracle over the whole frame (the oracle's counting sort and window counts are
cheap); decoded channels are compared on an evenly spaced sample of queries plus
both ends of the frame, which the oracle decodes one by one in float64 (and the
gather step's feature vectors on the same sample).  Every
output row must be finite and in [0, 1], and the stream-order decode must equal
the binned decode bit for bit on the whole frame.
"""
import sys

import numpy as np
import pytest
import torch

from paper_2608_27888_amd import ntc
from paper_2608_27888_amd import workloads as W

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

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


def sample(n, k):
    s = np.unique(np.linspace(0, n - 1, k).round().astype(np.int64))
    return np.unique(np.concatenate([s, np.arange(min(n, 97)), np.arange(max(0, n - 97), n)]))


def check_frame(dev, oracle, w, n_sample, check_stream=True):
    say(f"[full] {w.name}: n={w.n} T={w.n_textures} D={w.n_decoders} dims={w.dims} "
        f"mip={w.mip is not None}")
    model, q = ntc.upload(w, dev)
    bins = ntc.alloc_bins(w.n, w.n_decoders, 64, dev)
    ntc.build_bins(q.tex_id, model.tex_to_dec, w.n_decoders, bins=bins)
    out = torch.empty((w.n, w.out_dim), dtype=torch.float32, device=dev)
    ntc.decode(model, q, bins, out=out)
    torch.cuda.synchronize()
    say("    bins vs oracle")
    cnt, off, perm, bad = oracle.build_bins(w.tex_id, w.tex_to_dec, w.n_decoders, 64)
    assert np.array_equal(u32(bins.bin_count), cnt)
    assert np.array_equal(u32(bins.bin_offset), off)
    P = int(off[-1])
    assert np.array_equal(u32(bins.perm)[:P], perm)
    assert ntc.device_error(bins) == bad == 0
    say("    divergence vs oracle")
    per, tot = ntc.divergence_stats(q.tex_id, model.tex_to_dec, w.n_decoders)
    per_o, tot_o = oracle.divergence(w.tex_id, w.tex_to_dec, w.n_decoders)
    assert np.array_equal(u32(per), per_o)
    assert np.array_equal(tot.cpu().numpy().astype(np.uint64), tot_o)
    per_b, tot_b = ntc.divergence_stats(q.tex_id, model.tex_to_dec, w.n_decoders,
                                        order=bins.perm[:P])
    assert int(tot_b[3]) == 1
    if w.screen is not None:
        W_, H_, spp = w.screen
        dmap, hist, tot_m = ntc.divergence_map(q.tex_id, W_, H_, model.tex_to_dec, w.n_decoders,
                                               spp=spp)
        dmap_o, hist_o, tot_mo = oracle.divergence_map(w.tex_id, W_, H_, w.tex_to_dec,
                                                       w.n_decoders, spp=spp)
        assert np.array_equal(u32(dmap), dmap_o)
        assert np.array_equal(u32(hist), hist_o)
        assert np.array_equal(tot_m.cpu().numpy().astype(np.uint64), tot_mo)
    y = out.cpu().numpy()
    assert np.all(np.isfinite(y)) and np.all((y >= 0) & (y <= 1))
    sub = sample(w.n, n_sample)
    say(f"    decode vs oracle on {sub.size} queries")
    ref = oracle.decode(w, subset=sub)
    err = np.abs(y[sub].astype(np.float64) - ref).max()
    say(f"    max abs err {err:.3e}")
    assert err <= TOL
    if check_stream:
        say("    stream order vs binned")
        out_s = ntc.decode(model, q)
        assert torch.equal(out_s.view(torch.int32), out.view(torch.int32))
        del out_s
    # the gather step alone, on the same sample: within the fp16 arithmetic's
    # bound of the oracle's features (see tests/test_gpu_gather.py)
    feats = ntc.gather_features(model, q)
    f_ref = oracle.features(w, subset=sub, pe_octaves=0)
    f_err = np.abs(feats[torch.from_numpy(sub).to(dev)].cpu().numpy().astype(np.float64)
                   - f_ref).max()
    f_tol = (12.0 if w.mip is not None else 6.0) * 2.0 ** -11 \
        * float(np.abs(W.bits_to_f32(w.latents)).max()) * 1.0001
    say(f"    features: max abs err {f_err:.3e}, bound {f_tol:.3e}")
    assert f_err <= f_tol
    del model, q, bins, out, feats
    torch.cuda.empty_cache()


def test_full_tiny(dev, oracle):
    check_frame(dev, oracle, W.tiny(), 65536)


def test_full_single(dev, oracle):
    check_frame(dev, oracle, W.single(), 32768)


def test_full_divergent(dev, oracle):
    check_frame(dev, oracle, W.divergent(), 32768)


@pytest.fixture(scope="module")
def clustered(dev):
    return W.clustered4k()


def test_full_clustered4k_d16(dev, oracle, clustered):
    check_frame(dev, oracle, clustered, 32768)


def test_full_clustered4k_d512(dev, oracle, clustered):
    w = clustered.with_decoders(512, np.arange(512, dtype=np.uint32))
    check_frame(dev, oracle, w, 32768)


@pytest.mark.parametrize("width,height", [(600, 400), (640, 420), (1100, 700)])
def test_full_clustered_grid_fill(dev, oracle, width, height):
    """Binned decode around the size where its grid fills every CU with two
    workgroups (4096 tiles of 64 slots): 600x400 stays below it (equal tile
    ranges), 640x420 just fills it and 1100x700 holds three times as many tiles
    (the first workgroup on each CU then takes two thirds of the CU's tiles).
    Binned equals stream bit for bit; the oracle on a sample."""
    w = W.clustered4k(0, width, height, n_decoders=16, n_textures=64)
    check_frame(dev, oracle, w, 32768)


@pytest.fixture(scope="module")
def wide(dev):
    return W.wide_trilinear()


def test_full_wide_trilinear_d8(dev, oracle, wide):
    check_frame(dev, oracle, wide, 8192)


def test_full_wide_trilinear_d512(dev, oracle, wide):
    w = wide.with_decoders(512, np.arange(512, dtype=np.uint32))
    check_frame(dev, oracle, w, 8192, check_stream=False)


def test_full_output_past_2gib(dev, oracle):
    """8192^2 queries x 8 fp32 channels = 2 GiB of output: byte offsets past 2^31."""
    check_frame(dev, oracle, W.k_per_wave(0, 8192, 5), 8192)
