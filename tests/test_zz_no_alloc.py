"""GPU: ntc_build_bins_noalloc (the library's own device scratch, no workspace)
gives the same bins as ntc_build_bins, bit for bit, on two calls in a row, the
second on a smaller input; the invalid-query count it writes equals the one
ntc_get_device_error reads for ntc_build_bins."""
import numpy as np
import pytest
import torch

from paper_2608_27888_amd import ntc
from paper_2608_27888_amd import workloads as W

pytestmark = pytest.mark.gpu


def _inputs(seed, n, T, D, n_bad):
    rng = np.random.default_rng(seed)
    # screen-coherent runs (what binning sees in a frame) mixed with random ids
    tex = np.repeat(rng.integers(0, T, n // 37 + 1), 37)[:n].astype(np.uint32)
    flip = rng.random(n) < 0.2
    tex[flip] = rng.integers(0, T, int(flip.sum()))
    t2d = rng.integers(0, D, T).astype(np.uint32)
    if n_bad:
        tex[rng.choice(n, n_bad, replace=False)] = T + 5   # texture out of range
        t2d[0] = D + 1                                      # decoder out of range
    return tex, t2d


def _noalloc(tex_id, t2d, D, align, dev):
    n = tex_id.numel()
    cap = ntc.perm_capacity(n, D, align)
    cnt = torch.full((D,), -7, dtype=torch.int32, device=dev)
    off = torch.full((D + 1,), -7, dtype=torch.int32, device=dev)
    perm = torch.full((max(cap, 1),), -7, dtype=torch.int32, device=dev)
    inv = torch.full((1,), -7, dtype=torch.int32, device=dev)
    ntc.build_bins_noalloc(tex_id, t2d, D, cnt, off, perm, align=align, n_invalid=inv)
    return cnt, off, perm, inv


@pytest.mark.parametrize("sizes", [((1_000_003, 512, 16, 64, 0), (70_001, 64, 7, 64, 3)),
                                   ((300_000, 40, 33, 256, 11), (5_000, 40, 33, 128, 0)),
                                   ((8_294_400, 512, 16, 64, 5), (2_000_000, 64, 63, 64, 0))])
def test_noalloc_matches_workspace_path(sizes):
    dev = torch.device("cuda:0")
    for k, (n, T, D, align, n_bad) in enumerate(sizes):
        tex, t2d = _inputs(100 + k, n, T, D, n_bad)
        tex_d = torch.from_numpy(tex.view(np.int32)).to(dev)
        t2d_d = torch.from_numpy(t2d.view(np.int32)).to(dev)
        ref = ntc.build_bins(tex_d, t2d_d, D, align)
        cnt, off, perm, inv = _noalloc(tex_d, t2d_d, D, align, dev)
        torch.cuda.synchronize()
        assert torch.equal(cnt, ref.bin_count)
        assert torch.equal(off, ref.bin_offset)
        P = int(ref.bin_offset[-1].item())
        assert torch.equal(perm[:P], ref.perm[:P])
        # entries past the padded total are untouched
        assert bool((perm[P:] == -7).all())
        assert int(inv.item()) == ntc.device_error(ref)
        if n_bad:
            assert int(inv.item()) > 0


def test_noalloc_largest_sizes_fit():
    """The scratch holds the workspace of every valid call: 40M queries with the
    largest decoder count, then a small call, both equal to ntc_build_bins."""
    dev = torch.device("cuda:0")
    for k, (n, T, D, align) in enumerate(((40_000_000, 4096, 4096, 64), (1000, 3, 4096, 1))):
        tex, t2d = _inputs(300 + k, n, T, D, 0)
        tex_d = torch.from_numpy(tex.view(np.int32)).to(dev)
        t2d_d = torch.from_numpy(t2d.view(np.int32)).to(dev)
        assert ntc.workspace_bytes(n, D) <= ntc.NOALLOC_SCRATCH_BYTES
        ref = ntc.build_bins(tex_d, t2d_d, D, align)
        cnt, off, perm, inv = _noalloc(tex_d, t2d_d, D, align, dev)
        torch.cuda.synchronize()
        assert torch.equal(cnt, ref.bin_count) and torch.equal(off, ref.bin_offset)
        P = int(ref.bin_offset[-1].item())
        assert torch.equal(perm[:P], ref.perm[:P])
        assert int(inv.item()) == 0
        del tex_d, ref, perm
        torch.cuda.empty_cache()
