"""Pins of the oracle's decode: latent sampling and the MLP decoder.

Sampling is checked against torch's grid_sample (bilinear, border padding,
align_corners=False, float64), against the exact value at texel centres and on
constant grids.  Level blending by mip is checked through properties of the
linear mipmap filter (single levels at integer mips, continuity, betweenness,
clamping, affine on constant levels), each against grid_sample of one level.  The MLP is checked against a float64 chain of
torch.nn.functional.linear, and against zero-weight and identity decoders.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as Fn

from paper_2608_27888_amd import workloads as W


def make_workload(res, ch, T, dims, D, n, seed=0, latents=None, params=None, uv=None, mip=None,
                  tex=None, t2d=None):
    rng = np.random.default_rng(seed)
    stride = W.texture_stride(res, ch)
    if latents is None:
        latents = W.fp16_bits(rng.standard_normal(T * stride))
    if params is None:
        blob = []
        for _ in range(D):
            for a, b in zip(dims[:-1], dims[1:]):
                blob += [rng.uniform(-1, 1, (b, a)).ravel() * np.sqrt(3.0 / a), rng.uniform(-.1, .1, b)]
        params = W.fp16_bits(np.concatenate(blob))
    if tex is None:
        tex = rng.integers(0, T, n).astype(np.uint32)
    if t2d is None:
        t2d = (np.arange(T) % D).astype(np.uint32)
    if uv is None:
        uv = rng.uniform(-0.2, 1.2, (n, 2)).astype(np.float32)
    return W.Workload("t", T, list(res), list(ch), np.ascontiguousarray(latents, np.uint16), D,
                      list(dims), np.ascontiguousarray(params, np.uint16),
                      np.ascontiguousarray(t2d, np.uint32), np.ascontiguousarray(tex, np.uint32),
                      np.ascontiguousarray(uv, np.float32),
                      None if mip is None else np.ascontiguousarray(mip, np.float32))


def level_grid(w, t, l):
    """Level l of texture t as a float64 [C, H, W] tensor."""
    off = W.level_offsets(w.res, w.channels)[l] + t * w.texture_stride
    r, c = w.res[l], w.channels[l]
    a = W.bits_to_f32(w.latents[off:off + r * r * c]).astype(np.float64).reshape(r, r, c)
    return torch.from_numpy(a).permute(2, 0, 1).contiguous()


def grid_sample_level(w, l, tex, uv):
    out = np.zeros((uv.shape[0], w.channels[l]))
    for t in np.unique(tex):
        sel = np.nonzero(tex == t)[0]
        g = torch.from_numpy(uv[sel].astype(np.float64) * 2.0 - 1.0).view(1, 1, -1, 2)
        s = Fn.grid_sample(level_grid(w, int(t), l)[None], g, mode="bilinear",
                           padding_mode="border", align_corners=False)
        out[sel] = s[0, :, 0, :].T.numpy()
    return out


def test_half_to_double(oracle):
    vals = np.array([0.0, -0.0, 1.0, -2.5, 65504.0, 6.1035156e-05, 5.9604645e-08, 0.333],
                    np.float16)
    for v in vals:
        assert oracle.half_to_double(int(v.view(np.uint16))) == float(v)
    assert np.isinf(oracle.half_to_double(0x7C00))
    every = np.arange(0, 0x7C00, 97, dtype=np.uint16)
    got = np.array([oracle.half_to_double(int(b)) for b in every])
    assert np.array_equal(got, every.view(np.float16).astype(np.float64))


@pytest.mark.parametrize("res,ch", [([16, 8], [8, 8]), ([13, 7, 4], [16, 16, 16]), ([32], [4])])
def test_features_match_grid_sample(oracle, res, ch):
    w = make_workload(res, ch, T=3, dims=[sum(ch), 8], D=1, n=3000, seed=1)
    f = oracle.features(w)
    pos = 0
    for l in range(len(res)):
        ref = grid_sample_level(w, l, w.tex_id, w.uv)
        np.testing.assert_allclose(f[:, pos:pos + ch[l]], ref, rtol=0, atol=1e-12)
        pos += ch[l]


def test_texel_centres_return_stored_latent(oracle):
    res, ch = [64, 32], [16, 16]
    rng = np.random.default_rng(2)
    n = 2000
    for l in range(2):
        ix, iy = rng.integers(0, res[l], n), rng.integers(0, res[l], n)
        uv = np.stack([(ix + 0.5) / res[l], (iy + 0.5) / res[l]], 1).astype(np.float32)
        w = make_workload(res, ch, T=5, dims=[32, 8], D=1, n=n, seed=3, uv=uv)
        f = oracle.features(w)[:, 16 * l:16 * l + 16]
        off = W.level_offsets(res, ch)[l]
        idx = ((w.tex_id.astype(np.int64) * w.texture_stride + off
                + (iy * res[l] + ix) * 16)[:, None] + np.arange(16))
        stored = W.bits_to_f32(w.latents[idx]).astype(np.float64)
        assert np.array_equal(f, stored)  # exact, not approximate


def test_constant_latents_give_constant_output(oracle):
    res, ch, dims = [32, 16], [8, 8], [16, 64, 64, 8]
    c = np.float16(0.7109375)
    lat = np.full(2 * W.texture_stride(res, ch), c.view(np.uint16), np.uint16)
    w = make_workload(res, ch, T=2, dims=dims, D=1, n=500, seed=4, latents=lat,
                      uv=np.random.default_rng(0).uniform(-3, 4, (500, 2)).astype(np.float32))
    assert np.all(oracle.features(w) == float(c))
    y = oracle.decode(w)
    assert np.all(y == y[0])
    # the constant output is the MLP applied to the constant vector, in float64 numpy
    p = W.bits_to_f32(w.params).astype(np.float64)
    h, o = np.full(16, float(c)), 0
    for i, (a, b) in enumerate(zip(dims[:-1], dims[1:])):
        Wm = p[o:o + a * b].reshape(b, a); o += a * b
        bb = p[o:o + b]; o += b
        z = Wm @ h + bb
        h = np.maximum(z, 0) if i < len(dims) - 2 else 1 / (1 + np.exp(-z))
    np.testing.assert_allclose(y[0], h, rtol=0, atol=1e-14)


# Level blending by mip (the wide trilinear configuration).  The reading is
# the linear mipmap filter of the graphics APIs (OpenGL 4.6 core profile,
# Sec. 8.14.3 "Mipmapping", LINEAR_MIPMAP_LINEAR; Vulkan's
# VK_SAMPLER_MIPMAP_MODE_LINEAR): the two levels around the level of detail
# are each filtered bilinearly and mixed by the fractional part of the level
# of detail, which is clamped to the pyramid; slot l of the feature vector
# is never finer than level l.  The pins below are properties that filter
# must have, each checked against grid_sample of single levels; none of them
# recomputes the blend.

MIP_RES, MIP_CH = [32, 16, 8], [4, 4, 4]


def _mip_workload(mipval, n=600, seed=5, latents=None):
    mip = np.broadcast_to(np.asarray(mipval, np.float32), (n,)).copy()
    return make_workload(MIP_RES, MIP_CH, T=2, dims=[12, 8], D=1, n=n, seed=seed, mip=mip,
                         latents=latents)


def _slot(f, l):
    return f[:, 4 * l:4 * l + 4]


@pytest.mark.parametrize("k", [0, 1, 2])
def test_mip_integer_levels_are_single_levels(oracle, k):
    # at an integer mip k, slot l samples level max(l, k) alone
    w = _mip_workload(float(k))
    f = oracle.features(w)
    for l in range(3):
        ref = grid_sample_level(w, max(l, k), w.tex_id, w.uv)
        np.testing.assert_allclose(_slot(f, l), ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("k", [1, 2])
@pytest.mark.parametrize("eps", [1.0 / 64, 1.0 / 1024])
def test_mip_continuous_at_integer_levels(oracle, k, eps):
    # approaching level k from either side the finest slot tends to level k's
    # sample, at a rate set by the difference to the neighbouring level: a
    # filter weighted the wrong way round, or one that never reaches the next
    # level, jumps at k
    lo = _mip_workload(k - eps)
    f_lo = _slot(oracle.features(lo), 0)
    a = grid_sample_level(lo, k - 1, lo.tex_id, lo.uv)
    b = grid_sample_level(lo, k, lo.tex_id, lo.uv)
    assert np.all(np.abs(f_lo - b) <= eps * np.abs(b - a) + 1e-12)
    if k < 2:
        hi = _mip_workload(k + eps)
        f_hi = _slot(oracle.features(hi), 0)
        c = grid_sample_level(hi, k + 1, hi.tex_id, hi.uv)
        assert np.all(np.abs(f_hi - b) <= eps * np.abs(c - b) + 1e-12)


@pytest.mark.parametrize("mipval", [0.25, 0.5, 0.999, 1.25, 1.75])
def test_mip_blend_lies_between_its_levels(oracle, mipval):
    # a fractional level of detail lies between floor and floor + 1, and the
    # blended value between the two levels' samples (strictly inside where they
    # differ)
    w = _mip_workload(mipval)
    f = oracle.features(w)
    m = float(np.float32(mipval))
    for l in range(3):
        lod = max(l, m)
        k0 = int(np.floor(lod))
        a = grid_sample_level(w, k0, w.tex_id, w.uv)
        b = grid_sample_level(w, min(k0 + 1, 2), w.tex_id, w.uv)
        s = _slot(f, l)
        assert np.all(s >= np.minimum(a, b) - 1e-12) and np.all(s <= np.maximum(a, b) + 1e-12)
        if lod != k0:
            differ = np.abs(a - b) > 1e-9
            inside = (s > np.minimum(a, b)) & (s < np.maximum(a, b))
            assert differ.any() and np.all(inside[differ])


@pytest.mark.parametrize("mipval", [-3.0, -0.5, 0.0, 0.3, 0.9999, 1.0, 1.5])
def test_mip_below_a_slot_does_not_change_it(oracle, mipval):
    # slot l is level l whenever mip <= l: coarser slots are never refined by a
    # small mip, and negative mips clamp to 0
    w = _mip_workload(mipval)
    f = oracle.features(w)
    m = float(np.float32(mipval))
    for l in range(3):
        if m <= l:
            ref = grid_sample_level(w, l, w.tex_id, w.uv)
            np.testing.assert_allclose(_slot(f, l), ref, rtol=0, atol=1e-12)


def test_mip_beyond_the_pyramid_clamps_to_the_coarsest(oracle):
    w = _mip_workload(7.5)
    f = oracle.features(w)
    ref = grid_sample_level(w, 2, w.tex_id, w.uv)
    for l in range(3):
        np.testing.assert_allclose(_slot(f, l), ref, rtol=0, atol=1e-12)


def test_mip_on_constant_levels_is_affine_and_monotone(oracle):
    # levels holding the constants 0, 1, 3: the finest slot is a function of the
    # mip alone, non-decreasing, affine on each whole level interval (its
    # quarter points average to the interval's ends) and equal to the
    # constants at the integers
    consts = [0.0, 1.0, 3.0]
    stride = W.texture_stride(MIP_RES, MIP_CH)
    offs = W.level_offsets(MIP_RES, MIP_CH)
    lat = np.zeros(2 * stride, np.uint16)
    for t in range(2):
        for l, c in enumerate(consts):
            n_l = MIP_RES[l] ** 2 * MIP_CH[l]
            lat[t * stride + offs[l]:t * stride + offs[l] + n_l] = np.float16(c).view(np.uint16)
    mips = np.arange(0, 2.0 + 1e-9, 1.0 / 32)
    vals = []
    for m in mips:
        s = _slot(oracle.features(_mip_workload(m, n=64, latents=lat)), 0)
        assert np.all(s == s[0, 0])
        vals.append(s[0, 0])
    vals = np.array(vals)
    assert np.all(np.diff(vals) >= 0) and np.all(np.diff(vals)[:32] > 0)
    for k in range(3):
        assert vals[32 * k] == consts[k]
    for k in range(2):
        q1, mid, q3 = vals[32 * k + 8], vals[32 * k + 16], vals[32 * k + 24]
        ends = vals[32 * k] + vals[32 * k + 32]
        assert abs(q1 + q3 - ends) < 1e-12 and abs(2 * mid - ends) < 1e-12


def test_mip_zero_equals_no_mip(oracle):
    w = make_workload([32, 16], [8, 8], T=2, dims=[16, 8], D=1, n=600, seed=6,
                      mip=np.zeros(600))
    f_mip = oracle.features(w)
    w.mip = None
    assert np.array_equal(f_mip, oracle.features(w))


@pytest.mark.parametrize("dims", [[16, 64, 64, 8], [32, 64, 64, 8], [48, 128, 128, 128, 8],
                                  [16, 5, 3]])
def test_mlp_matches_linear_chain(oracle, dims):
    F = dims[0]
    res, ch = ([16, 8], [F // 2, F // 2]) if F % 2 == 0 else ([16], [F])
    if F == 48:
        res, ch = [16, 8, 4], [16, 16, 16]
    w = make_workload(res, ch, T=6, dims=dims, D=3, n=1500, seed=7)
    x = torch.from_numpy(oracle.features(w))
    y = oracle.decode(w)
    p = W.bits_to_f32(w.params).astype(np.float64)
    stride = W.decoder_stride(dims)
    dec = w.tex_to_dec[w.tex_id]
    ref = np.zeros_like(y)
    for d in range(w.n_decoders):
        o = d * stride
        h = x[dec == d]
        for i, (a, b) in enumerate(zip(dims[:-1], dims[1:])):
            Wm = torch.from_numpy(p[o:o + a * b].reshape(b, a)); o += a * b
            bb = torch.from_numpy(p[o:o + b]); o += b
            z = Fn.linear(h, Wm, bb)
            h = torch.relu(z) if i < len(dims) - 2 else torch.sigmoid(z)
        ref[dec == d] = h.numpy()
    np.testing.assert_allclose(y, ref, rtol=0, atol=1e-13)
    assert np.all((y > 0) & (y < 1))


def test_zero_weights_give_sigmoid_of_bias(oracle):
    dims = [16, 64, 64, 8]
    w = make_workload([16, 8], [8, 8], T=2, dims=dims, D=1, n=300, seed=8)
    p = W.bits_to_f32(w.params).astype(np.float64)
    o = 0
    for a, b in zip(dims[:-1], dims[1:]):
        p[o:o + a * b] = 0.0; o += a * b
        last_b = p[o:o + b].copy(); o += b
    w.params = W.fp16_bits(p)
    y = oracle.decode(w)
    np.testing.assert_allclose(y, np.broadcast_to(1.0 / (1.0 + np.exp(-last_b)), y.shape),
                               rtol=4e-16, atol=0)
    assert np.all(y == y[0])


def test_identity_decoder_gives_sigmoid_of_features(oracle):
    dims = [8, 8]
    p = np.concatenate([np.eye(8).ravel(), np.zeros(8)])
    w = make_workload([16], [8], T=2, dims=dims, D=1, n=400, seed=9, params=W.fp16_bits(p))
    x = oracle.features(w)
    # equal up to the last-bit differences between libm's and numpy's exp
    np.testing.assert_allclose(oracle.decode(w), 1.0 / (1.0 + np.exp(-x)), rtol=4e-16, atol=0)


def test_invalid_queries_leave_rows_untouched(oracle):
    w = make_workload([16, 8], [8, 8], T=4, dims=[16, 32, 8], D=2, n=200, seed=10)
    w.tex_id[::7] = 4                      # past the last texture
    w.tex_to_dec = np.array([0, 1, 5, 1], np.uint32)  # texture 2 maps past the last decoder
    y = oracle.decode(w)
    bad = (w.tex_id >= 4) | np.isin(w.tex_id, [2])
    assert np.all(np.isnan(y[bad])) and not np.any(np.isnan(y[~bad]))


def test_subset_matches_full(oracle):
    w = make_workload([16, 8], [8, 8], T=4, dims=[16, 32, 8], D=2, n=500, seed=12)
    full = oracle.decode(w)
    sub = np.array([499, 0, 17, 17, 250])
    assert np.array_equal(oracle.decode(w, subset=sub), full[sub])


@pytest.mark.parametrize("slope", [0.01, 0.2])
def test_leaky_identity_chain_gives_sigmoid_of_leaky_features(oracle, slope):
    """Two identity layers around one LeakyReLU (the Sec. 4 setup's activation):
    y = sigmoid(x) where x > 0 and sigmoid(slope * x) elsewhere."""
    dims = [8, 8, 8]
    eye = np.concatenate([np.eye(8).ravel(), np.zeros(8)])
    w = make_workload([16], [8], T=2, dims=dims, D=1, n=400, seed=19,
                      params=W.fp16_bits(np.concatenate([eye, eye])))
    x = oracle.features(w)
    h = np.where(x > 0, x, slope * x)
    np.testing.assert_allclose(oracle.decode(w, leaky_slope=slope), 1.0 / (1.0 + np.exp(-h)),
                               rtol=4e-16, atol=0)
    assert np.any(x < 0)


def test_leaky_slope_zero_is_relu(oracle):
    w = make_workload([16, 8], [8, 8], T=4, dims=[16, 32, 32, 3], D=2, n=300, seed=21)
    assert np.array_equal(oracle.decode(w, leaky_slope=0.0), oracle.decode(w))
    assert not np.array_equal(oracle.decode(w, leaky_slope=0.1), oracle.decode(w))


# ------------------------------------------------------------ positional encoding
# The Sec. 4 setup concatenates a positional encoding to the encoder output; its
# form is a reading (octave k: sin, cos of 2^k pi u, then of 2^k pi v).  The pins
# below fix the order of the four values, the octave scaling and the placement
# after the latent features, and relate the decoder with encoding to the pinned
# decoder without it.

def pe_columns(oracle, w, K):
    F = int(sum(w.channels))
    f = oracle.features(w, pe_octaves=K)
    assert f.shape[1] == F + 4 * K
    np.testing.assert_array_equal(f[:, :F], oracle.features(w, pe_octaves=0))
    return f[:, F:]


def test_pe_special_points(oracle):
    """u = 1/2, v = 0 and u = 1/4, v = 3/4: values fixed by the unit circle."""
    uv = np.array([[0.5, 0.0], [0.25, 0.75]], np.float32)
    w = make_workload([16], [8], T=1, dims=[8, 8], D=1, n=2, seed=30, uv=uv,
                      tex=np.zeros(2, np.uint32))
    pe = pe_columns(oracle, w, 4)
    r2 = np.sqrt(0.5)
    # octave k of (u, v): sin(2^k pi u), cos(2^k pi u), sin(2^k pi v), cos(2^k pi v)
    want0 = [1, 0, 0, 1,  0, -1, 0, 1,  0, 1, 0, 1,  0, 1, 0, 1]
    want1 = [r2, r2, r2, -r2,  1, 0, -1, 0,  0, -1, 0, -1,  0, 1, 0, 1]
    np.testing.assert_allclose(pe[0], want0, atol=1e-15)
    np.testing.assert_allclose(pe[1], want1, atol=1e-15)
    # u = v = 0: every sine exactly 0, every cosine exactly 1
    w0 = make_workload([16], [8], T=1, dims=[8, 8], D=1, n=1, seed=31,
                       uv=np.zeros((1, 2), np.float32), tex=np.zeros(1, np.uint32))
    assert np.array_equal(pe_columns(oracle, w0, 8)[0], np.tile([0.0, 1.0, 0.0, 1.0], 8))


def test_pe_octaves_double_the_angle(oracle):
    """sin(2a) = 2 sin(a) cos(a), cos(2a) = cos^2(a) - sin^2(a) between octaves
    k and k+1, and sin^2 + cos^2 = 1, for random coordinates inside and outside
    [0, 1)."""
    w = make_workload([16], [8], T=2, dims=[8, 8], D=1, n=300, seed=32)
    pe = pe_columns(oracle, w, 8).reshape(-1, 8, 4)
    for c in (0, 2):  # u, v
        s, co = pe[:, :, c], pe[:, :, c + 1]
        np.testing.assert_allclose(s ** 2 + co ** 2, 1.0, atol=1e-14)
        np.testing.assert_allclose(s[:, 1:], 2 * s[:, :-1] * co[:, :-1], atol=1e-12)
        np.testing.assert_allclose(co[:, 1:], co[:, :-1] ** 2 - s[:, :-1] ** 2, atol=1e-12)
    # octave 0 against the coordinate itself
    np.testing.assert_allclose(pe[:, 0, 0], np.sin(np.pi * w.uv[:, 0].astype(np.float64)),
                               atol=1e-15)


def test_pe_zero_columns_equal_decoder_without_pe(oracle):
    """A decoder whose weights on the encoding are zero gives the output of the
    same decoder restricted to the latent features (the pinned path)."""
    base = make_workload([16, 8], [8, 8], T=4, dims=[16, 32, 32, 3], D=2, n=300, seed=33)
    K = 4
    rng = np.random.default_rng(34)
    blob_pe, blob = [], []
    for _ in range(2):
        w0 = rng.uniform(-0.5, 0.5, (32, 16))
        w0pe = np.concatenate([w0, np.zeros((32, 4 * K))], axis=1)
        rest = [rng.uniform(-0.1, 0.1, 32), rng.uniform(-0.3, 0.3, (32, 32)),
                rng.uniform(-0.1, 0.1, 32), rng.uniform(-0.3, 0.3, (3, 32)), rng.uniform(-0.1, 0.1, 3)]
        blob_pe += [w0pe.ravel()] + [r.ravel() for r in rest]
        blob += [w0.ravel()] + [r.ravel() for r in rest]
    w_no = W.Workload("t", base.n_textures, base.res, base.channels, base.latents, 2, [16, 32, 32, 3],
                      W.fp16_bits(np.concatenate(blob)), base.tex_to_dec, base.tex_id, base.uv, None)
    w_pe = W.Workload("t", base.n_textures, base.res, base.channels, base.latents, 2,
                      [16 + 4 * K, 32, 32, 3], W.fp16_bits(np.concatenate(blob_pe)),
                      base.tex_to_dec, base.tex_id, base.uv, None, pe_octaves=K)
    assert np.array_equal(oracle.decode(w_pe), oracle.decode(w_no))


def test_pe_only_decoder_ignores_latents(oracle):
    """With zero weights on the latent features the output depends on (u, v)
    only: redrawing the latents leaves it unchanged, moving u changes it."""
    K = 4
    w = make_workload([16, 8], [8, 8], T=4, dims=[16 + 4 * K, 32, 32, 8], D=2, n=300, seed=35)
    w.pe_octaves = K
    p = W.bits_to_f32(w.params).astype(np.float64).copy()
    stride = W.decoder_stride(w.dims)
    for d in range(2):
        W0 = p[d * stride: d * stride + 32 * (16 + 4 * K)].reshape(32, 16 + 4 * K)
        W0[:, :16] = 0.0
    w.params = W.fp16_bits(p)
    y = oracle.decode(w)
    w2 = make_workload([16, 8], [8, 8], T=4, dims=w.dims, D=2, n=300, seed=36, params=w.params,
                       tex=w.tex_id, t2d=w.tex_to_dec, uv=w.uv)
    w2.pe_octaves = K
    assert not np.array_equal(w2.latents, w.latents)
    assert np.array_equal(oracle.decode(w2), y)
    w2.uv = (w.uv + np.float32(0.125)).astype(np.float32)
    assert not np.allclose(oracle.decode(w2), y)
