"""Pins of the oracle's 2-D divergence map (Sec. 2: D(i,j) = distinct ids per
screen block; Eq. (normalized_ones_metric) from the totals).

Checked against numpy's unique over each block cut out of the screen array
(partial edge blocks, several samples per pixel), against the per-window count
when a block is one 64-pixel row run (the same set of queries), and against the
special cases the definition fixes: one decoder gives exactly 1 per block, a
constant texture per block gives 1, all-distinct ids give the block's size.
"""
import numpy as np
import pytest


def brute(tex, t2d, D, W, H, spp, bw, bh):
    T = t2d.size
    scr = tex.reshape(H, W, spp)
    by, bx = -(-H // bh), -(-W // bw)
    out = np.zeros((by, bx), np.int64)
    for i in range(by):
        for j in range(bx):
            ids = scr[i * bh:(i + 1) * bh, j * bw:(j + 1) * bw].ravel().astype(np.int64)
            ids = ids[ids < T]
            d = t2d[ids].astype(np.int64)
            out[i, j] = np.unique(d[d < D]).size
    return out


@pytest.mark.parametrize("W,H,spp,bw,bh", [(37, 23, 1, 8, 8), (40, 16, 4, 8, 4), (33, 9, 2, 5, 3),
                                           (64, 3, 1, 64, 1), (7, 5, 1, 16, 16)])
def test_map_vs_unique(oracle, W, H, spp, bw, bh):
    rng = np.random.default_rng(W * H + spp)
    T, D = 30, 7
    t2d = rng.integers(0, D + 1, size=T).astype(np.uint32)     # decoder D is invalid
    tex = rng.integers(0, T + 2, size=W * H * spp).astype(np.uint32)  # ids >= T invalid
    dmap, hist, tot = oracle.divergence_map(tex, W, H, t2d, D, spp=spp, block_w=bw, block_h=bh,
                                            hist_len=6)
    exp = brute(tex, t2d, D, W, H, spp, bw, bh)
    assert np.array_equal(dmap, exp)
    assert hist.sum() == exp.size
    assert np.array_equal(hist, np.bincount(np.minimum(exp.ravel(), 5), minlength=6))
    kept = exp[exp > 0]
    assert tot.tolist() == [kept.size, kept.sum(), int((kept > 1).sum()), kept.max()]


def test_row_blocks_equal_stream_windows(oracle):
    """A 64 x 1 block with one sample per pixel is the window of 64 consecutive queries."""
    rng = np.random.default_rng(5)
    W, H, T, D = 256, 11, 50, 13
    t2d = rng.integers(0, D, size=T).astype(np.uint32)
    tex = np.repeat(rng.integers(0, T, size=W * H // 8), 8).astype(np.uint32)
    dmap, _, tot = oracle.divergence_map(tex, W, H, t2d, D, block_w=64, block_h=1)
    per, tot_w = oracle.divergence(tex, t2d, D, wave=64)
    assert np.array_equal(dmap.ravel(), per)
    assert np.array_equal(tot, tot_w)


def test_special_cases(oracle):
    rng = np.random.default_rng(9)
    W, H = 48, 40
    tex = rng.integers(0, 20, size=W * H).astype(np.uint32)
    # one decoder: exactly one per block
    dmap, hist, tot = oracle.divergence_map(tex, W, H, np.zeros(20, np.uint32), 1)
    assert np.all(dmap == 1) and tot[1] == tot[0] == dmap.size and tot[2] == 0
    assert hist[1] == dmap.size
    # texture constant per 8x8 block: one per block even with per-texture decoders
    blk = rng.integers(0, 20, size=(H // 8, W // 8))
    tex2 = np.repeat(np.repeat(blk, 8, 0), 8, 1).ravel().astype(np.uint32)
    dmap, _, _ = oracle.divergence_map(tex2, W, H, np.arange(20, dtype=np.uint32), 20)
    assert np.all(dmap == 1)
    # all distinct: the block size
    tex3 = np.arange(W * H, dtype=np.uint32)
    dmap, _, tot = oracle.divergence_map(tex3, W, H, np.arange(W * H, dtype=np.uint32), W * H,
                                         block_w=8, block_h=4)
    assert np.all(dmap == 32) and tot[3] == 32
    # the metric of Eq. (normalized_ones_metric): mean |D - 1| over kept blocks
    dmap, _, tot = oracle.divergence_map(tex, W, H, np.arange(20, dtype=np.uint32), 20)
    assert tot[1] / tot[0] - 1 == pytest.approx(np.abs(dmap.astype(float) - 1).mean())
