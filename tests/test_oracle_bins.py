"""Pins of the oracle's binning (stable counting sort by decoder id).

Checked against brute force on small inputs, numpy's stable argsort and the
single-decoder special case, none of which share code with the oracle.
"""
import numpy as np
import pytest

PAD = 0xFFFFFFFF


def brute_force_bins(tex_id, tex_to_dec, D, align):
    """Position of each valid query, from its definition: offset of its bin plus
    the number of earlier queries of the same decoder."""
    T = len(tex_to_dec)
    dec = [None if t >= T or tex_to_dec[t] >= D else int(tex_to_dec[t]) for t in tex_id]
    count = [sum(1 for d in dec if d == k) for k in range(D)]
    offset = [0]
    for k in range(D):
        offset.append(offset[-1] + -(-count[k] // align) * align)
    perm = [PAD] * offset[-1]
    for q, d in enumerate(dec):
        if d is None:
            continue
        rank = sum(1 for qq in range(q) if dec[qq] == d)
        perm[offset[d] + rank] = q
    return count, offset, perm, sum(1 for d in dec if d is None)


@pytest.mark.parametrize("align", [1, 4, 64])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_bins_brute_force(oracle, align, seed):
    rng = np.random.default_rng(seed)
    T, D, n = 11, 7, 400
    t2d = rng.integers(0, D + 2, size=T).astype(np.uint32)  # some textures map past D
    tex = rng.integers(0, T + 2, size=n).astype(np.uint32)  # some ids past T
    cnt, off, perm, bad = oracle.build_bins(tex, t2d, D, align)
    c2, o2, p2, b2 = brute_force_bins(tex.tolist(), t2d.tolist(), D, align)
    assert cnt.tolist() == c2
    assert off.tolist() == o2
    assert perm.tolist() == p2
    assert bad == b2 and bad > 0


def test_bins_match_stable_argsort(oracle):
    rng = np.random.default_rng(5)
    T, D, n = 64, 16, 20000
    t2d = rng.integers(0, D, size=T).astype(np.uint32)
    tex = rng.integers(0, T, size=n).astype(np.uint32)
    cnt, off, perm, bad = oracle.build_bins(tex, t2d, D, 64)
    dec = t2d[tex]
    unpadded = perm[perm != PAD]
    assert np.array_equal(unpadded, np.argsort(dec, kind="stable").astype(np.uint32))
    assert np.array_equal(cnt, np.bincount(dec, minlength=D))
    sizes = np.diff(off.astype(np.int64))
    assert np.all(sizes % 64 == 0) and np.all(sizes >= cnt) and np.all(sizes - cnt < 64)
    for d in range(D):  # valid entries first inside each bin, then padding
        seg = perm[off[d]:off[d + 1]]
        assert np.all(seg[: cnt[d]] != PAD) and np.all(seg[cnt[d]:] == PAD)
    assert bad == 0


def test_bins_single_decoder_is_identity(oracle):
    n = 1000
    tex = np.zeros(n, np.uint32)
    cnt, off, perm, _ = oracle.build_bins(tex, np.zeros(1, np.uint32), 1, 64)
    assert off.tolist() == [0, 1024]
    assert np.array_equal(perm[:n], np.arange(n, dtype=np.uint32))
    assert np.all(perm[n:] == PAD)


def test_bins_empty_and_capacity(oracle):
    cnt, off, perm, bad = oracle.build_bins(np.zeros(0, np.uint32), np.arange(3, dtype=np.uint32), 3)
    assert off.tolist() == [0, 0, 0, 0] and perm.size == 0 and bad == 0
    with pytest.raises(oracle.OracleError):
        oracle.build_bins(np.arange(3, dtype=np.uint32), np.arange(3, dtype=np.uint32), 3,
                          align=64, capacity=64)
