"""Stream-mode decode over query layouts built to walk every state of a workgroup's
shared decoder: groups whose waves all hold one decoder (staged once and read from
LDS), groups that disagree (the odd wave reads its decoder's fragments itself),
waves holding two or many decoders (the staged one from LDS, the others from the
parameter blocks), waves with invalid lanes or no live lane at all, and random runs.
The layout is cut into segments of 8 groups (one vote interval), 8 kinds in turn,
so a workgroup that walks 16 or 64 consecutive groups meets the transitions between
kinds.  Stream order must equal binned order bit for bit on every row (the rows of
invalid queries left untouched by both), and both must match the oracle on a sample
of queries (Sec. 4.4: the non-shared decoder computes the same per-query MLP)."""
import dataclasses
import sys

import numpy as np
import pytest
import torch

from paper_2608_27888_amd import ntc
from paper_2608_27888_amd import workloads as W

pytestmark = pytest.mark.gpu

TOL = 2e-3
WAVE = 64
SEG = 8  # groups per segment


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    ntc.lib()
    return torch.device("cuda:0")


def layout(w, waves, n_groups, seed):
    """Texture id per query: segment s of SEG groups (each group `waves` tiles of 64
    queries) follows kind s % 8."""
    rng = np.random.default_rng(seed)
    t2d = np.asarray(w.tex_to_dec)
    rep = {}
    for t, d in enumerate(t2d):
        rep.setdefault(int(d), t)
    decs = sorted(rep)
    assert len(decs) >= 4
    A, B, C, D = (rep[d] for d in decs[:4])
    many = np.array([rep[d] for d in decs], np.uint32)
    bad = w.n_textures  # an invalid texture id
    per_group = waves * WAVE
    n = n_groups * per_group
    tex = np.empty(n, np.uint32)
    lane = np.arange(WAVE)
    for g in range(n_groups):
        kind = (g // SEG) % 8
        for t in range(waves):
            if kind == 0:
                ids = np.full(WAVE, A)
            elif kind == 1:
                ids = np.full(WAVE, B if t == 0 else A)
            elif kind == 2:
                ids = np.where(lane % 2 == 0, A, B)
            elif kind == 3:
                ids = np.full(WAVE, C)
            elif kind == 4:
                ids = many[lane % many.size]
            elif kind == 5:
                ids = np.where(lane == 5, bad, C)
            elif kind == 6:
                ids = np.full(WAVE, bad if t % 2 == 0 else D)
            else:
                ids = np.repeat(rng.choice([A, B, C, D], WAVE // 16), 16)
            s = (g * waves + t) * WAVE
            tex[s:s + WAVE] = ids
    return tex


CASES = [  # (small workload, waves per stream group of its decoder width, groups)
    ("k5_per_wave", 4, 16384),
    ("wide_trilinear", 8, 16384),
]


@pytest.mark.parametrize("name,waves,n_groups", CASES)
def test_stream_vote_layouts(dev, oracle, name, waves, n_groups):
    base = W.small(name)
    tex = layout(base, waves, n_groups, seed=7)
    n = tex.size
    w = dataclasses.replace(
        base, name=f"{name}_vote_layout", tex_id=tex,
        uv=np.resize(base.uv, (n, 2)).astype(np.float32),
        mip=None if base.mip is None else np.resize(base.mip, n).astype(np.float32),
        screen=None)
    say(f"[stream layouts] {w.name}: n={n} D={w.n_decoders} dims={w.dims} waves/group={waves}")
    model, q = ntc.upload(w, dev)
    sentinel = -777.0
    out_s = torch.full((n, w.out_dim), sentinel, device=dev)
    ntc.decode(model, q, out=out_s)
    bins = ntc.build_bins(q.tex_id, model.tex_to_dec, w.n_decoders)
    out_b = torch.full((n, w.out_dim), sentinel, device=dev)
    ntc.decode(model, q, bins, out=out_b)
    torch.cuda.synchronize()
    invalid = tex >= w.n_textures
    assert ntc.device_error(bins) == int(invalid.sum()) > 0
    ys, yb = out_s.cpu().numpy(), out_b.cpu().numpy()
    assert np.array_equal(ys.view(np.uint32), yb.view(np.uint32))
    assert np.all(ys[invalid] == sentinel)
    # sample: the first two segment cycles in full plus an even spread over the rest
    per_cycle = 8 * SEG * waves * WAVE
    sub = np.unique(np.concatenate([np.arange(0, n, 7)[: 2 * per_cycle // 7],
                                    np.linspace(0, n - 1, 20000).round().astype(np.int64)]))
    sub = sub[~invalid[sub]]
    say(f"    oracle on {sub.size} queries")
    ref = oracle.decode(w, subset=sub)
    err = np.abs(ys[sub].astype(np.float64) - ref).max()
    say(f"    max abs err {err:.3e}")
    assert err <= TOL
    del model, q, bins, out_s, out_b
    torch.cuda.empty_cache()
