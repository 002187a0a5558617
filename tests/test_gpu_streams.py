"""Calls on different HIP streams are independent: two frames, each with its own
binning workspace and outputs, binned, decoded (binned and stream order) and
counted on two side streams with their launches interleaved, give bit for bit
what the same calls give one after another on the default stream."""
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


def frame_steps(w, model, q, dev, res):
    """Binning, binned decode, stream decode and divergence counts of one frame, one
    library call per step on the current stream; the results go into `res`."""
    bins = ntc.alloc_bins(w.n, w.n_decoders, 64, dev)
    ntc.build_bins(q.tex_id, model.tex_to_dec, w.n_decoders, bins=bins)
    yield
    out_b = torch.empty((w.n, w.out_dim), dtype=torch.float32, device=dev)
    ntc.decode(model, q, bins, out=out_b)
    yield
    out_s = torch.empty((w.n, w.out_dim), dtype=torch.float32, device=dev)
    ntc.decode(model, q, out=out_s)
    yield
    per, tot = ntc.divergence_stats(q.tex_id, model.tex_to_dec, w.n_decoders)
    res.extend([bins, out_b, out_s, per, tot])


def run_frame(w, model, q, dev):
    res = []
    for _ in frame_steps(w, model, q, dev, res):
        pass
    return res


def same(a, b):
    """Bitwise equality of two frames' results (perm compared up to its last bin)."""
    (ba, *ra), (bb, *rb) = a, b
    assert torch.equal(ba.bin_count, bb.bin_count)
    assert torch.equal(ba.bin_offset, bb.bin_offset)
    used = int(ba.bin_offset[-1].item())
    assert torch.equal(ba.perm[:used], bb.perm[:used])
    for x, y in zip(ra, rb):
        if x.dtype == torch.float32:
            x, y = x.view(torch.int32), y.view(torch.int32)
        assert torch.equal(x, y)


def test_two_streams_match_default_stream(dev):
    ws = [W.small("clustered4k"), W.small("divergent")]
    ups = [ntc.upload(w, dev) for w in ws]
    torch.cuda.synchronize()
    ref = [run_frame(w, m, q, dev) for w, (m, q) in zip(ws, ups)]
    torch.cuda.synchronize()
    side = [torch.cuda.Stream(device=dev), torch.cuda.Stream(device=dev)]
    for s in side:
        s.wait_stream(torch.cuda.current_stream())
    for rep in range(3):
        got = [[], []]
        steps = [frame_steps(ws[i], *ups[i], dev, got[i]) for i in (0, 1)]
        live = [True, True]
        while any(live):  # one library call of each frame in turn
            for i in (0, 1):
                if live[i]:
                    with torch.cuda.stream(side[i]):
                        live[i] = next(steps[i], StopIteration) is not StopIteration
        for i in (0, 1):
            side[i].synchronize()
            same(ref[i], got[i])
        say(f"[streams] pass {rep}: both frames equal to the default-stream results")
    torch.cuda.synchronize()
