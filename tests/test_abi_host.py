"""The C-ABI library loads, exports every entry point its header declares, and
rejects malformed arguments on the host before any device work (no GPU needed)."""
import ctypes
import os
import re

import pytest

from paper_2608_27888_amd import ntc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ntc.h")

FAKE = ctypes.c_void_p(0x100000)  # never dereferenced: validation fails first

# A call that passes validation goes on to launch kernels on FAKE pointers.  That
# only happens here without a device (the launch then fails with NTC_ERR_HIP);
# with a device those checks are skipped.  Counting devices does not initialise
# them.
HAS_DEVICE = __import__("torch").cuda.device_count() > 0


def declared_functions():
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    return sorted(set(re.findall(r"^[A-Za-z_][\w \*]*?\b(ntc_\w+)\s*\(", text, flags=re.M)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(ntc.LIB_PATH):
        from paper_2608_27888_amd import build
        build.build()
    return ntc.lib()


def test_exports_every_declared_symbol(L):
    names = declared_functions()
    assert {"ntc_build_bins", "ntc_decode", "ntc_divergence_stats"} <= set(names)
    for name in names:
        assert hasattr(L, name), name


def test_status_strings(L):
    assert ntc.status_string(0) == "ok"
    for s in (-1, -2, -3, -4, -5):
        assert ntc.status_string(s) not in ("ok", "unknown status")
    assert ntc.status_string(7) == "unknown status"


def test_sizes(L):
    assert ntc.workspace_bytes(-1, 4) == 0
    assert ntc.workspace_bytes(10, 0) == 0
    assert ntc.workspace_bytes(10, 4097) == 0
    assert ntc.workspace_bytes(1 << 23, 16) > 16 * 4
    assert ntc.workspace_bytes(0, 1) > 0
    assert ntc.perm_capacity(100, 16, 64) == 100 + 16 * 63
    assert ntc.perm_capacity(100, 16, 1) == 100
    assert ntc.perm_capacity(100, 16, 3) == -1
    assert ntc.perm_capacity(100, 16, 8192) == -1


def _bins(L, **kw):
    a = dict(tex_id=FAKE, n=100, tex_to_dec=FAKE, T=4, D=2, align=64, cnt=FAKE, off=FAKE,
             perm=FAKE, cap=100 + 2 * 63, ws=FAKE, wsb=1 << 20)
    a.update(kw)
    return L.ntc_build_bins(a["tex_id"], a["n"], a["tex_to_dec"], a["T"], a["D"], a["align"],
                            a["cnt"], a["off"], a["perm"], a["cap"], a["ws"], a["wsb"], None)


def test_build_bins_validation(L):
    assert _bins(L, n=-1) == ntc.NTC_ERR_ARG
    assert _bins(L, tex_id=None) == ntc.NTC_ERR_ARG
    assert _bins(L, perm=None) == ntc.NTC_ERR_ARG
    assert _bins(L, ws=None) == ntc.NTC_ERR_ARG
    assert _bins(L, D=0) == ntc.NTC_ERR_ARG
    assert _bins(L, D=4097) == ntc.NTC_ERR_ARG
    assert _bins(L, T=0) == ntc.NTC_ERR_ARG
    assert _bins(L, align=48) == ntc.NTC_ERR_ARG
    assert _bins(L, cap=100 + 2 * 63 - 1) == ntc.NTC_ERR_CAPACITY
    assert _bins(L, wsb=8) == ntc.NTC_ERR_CAPACITY
    assert _bins(L, n=1 << 32) == ntc.NTC_ERR_ARG
    assert _bins(L, ws=ctypes.c_void_p(0x100000 + 8)) == ntc.NTC_ERR_ARG  # not 16-byte aligned


def _decode(L, res=(256, 128), ch=(16, 16), dims=(32, 64, 64, 8), n=100, D=4, binned=False,
            align=64, cap=None, nulls=(), ptrs=None):
    g = ntc.Grids()
    g.n_textures, g.n_levels = 4, len(res)
    for i, (r, c) in enumerate(zip(res, ch)):
        g.res[i], g.channels[i] = r, c
    g.latents = None if "latents" in nulls else FAKE
    d = ntc.Decoders()
    d.n_decoders, d.n_layers = D, len(dims) - 1
    for i, v in enumerate(dims):
        d.dims[i] = v
    d.params = None if "params" in nulls else FAKE
    q = ntc.Queries()
    q.tex_id, q.uv, q.mip, q.n = FAKE, FAKE, None, n
    out = None if "out" in nulls else FAKE
    for k, v in (ptrs or {}).items():
        if k == "latents":
            g.latents = v
        elif k == "out":
            out = v
        else:
            setattr(q, k, v)
    if cap is None:
        cap = ntc.perm_capacity(max(n, 0), D, 64)
    return L.ntc_decode(ctypes.byref(g), ctypes.byref(d), FAKE, ctypes.byref(q),
                        FAKE if binned else None, FAKE if binned else None, cap, align,
                        out, None)


def test_decode_validation(L):
    assert _decode(L, n=-5) == ntc.NTC_ERR_ARG
    assert _decode(L, nulls=("latents",)) == ntc.NTC_ERR_ARG
    assert _decode(L, nulls=("out",)) == ntc.NTC_ERR_ARG
    assert _decode(L, dims=(31, 64, 64, 8)) == ntc.NTC_ERR_ARG          # dims[0] != channels
    assert _decode(L, dims=(32, 64, 48, 8)) == ntc.NTC_ERR_UNSUPPORTED  # unequal hidden widths
    assert _decode(L, dims=(32, 96, 96, 8)) == ntc.NTC_ERR_UNSUPPORTED  # width not built
    assert _decode(L, dims=(32, 64, 64, 20)) == ntc.NTC_ERR_UNSUPPORTED  # too many outputs
    assert _decode(L, n=1 << 27, dims=(32, 64, 64, 8)) == ntc.NTC_ERR_UNSUPPORTED  # > 4 GiB
    if not HAS_DEVICE:
        assert _decode(L, dims=(32, 64, 64, 3)) == ntc.NTC_ERR_HIP   # RGB rows are built
        assert _decode(L, n=(1 << 27) - 16, dims=(32, 64, 64, 4)) == ntc.NTC_ERR_HIP  # 2 GiB
    assert _decode(L, dims=(32, 8)) == ntc.NTC_ERR_UNSUPPORTED          # no hidden layer
    assert _decode(L, res=(256, 128), ch=(16, 8), dims=(24, 64, 8)) == ntc.NTC_ERR_UNSUPPORTED
    assert _decode(L, res=(0, 128)) == ntc.NTC_ERR_ARG
    assert _decode(L, binned=True, align=32) == ntc.NTC_ERR_ARG
    assert _decode(L, binned=True, cap=10) == ntc.NTC_ERR_CAPACITY
    assert _decode(L, n=0) == ntc.NTC_OK  # nothing to do, nothing launched


def test_divergence_validation(L):
    f = L.ntc_divergence_stats
    assert f(FAKE, 10, FAKE, 4, 2, None, 10, 0, FAKE, FAKE, None) == ntc.NTC_ERR_ARG
    assert f(FAKE, 10, FAKE, 4, 2, None, 10, 65, FAKE, FAKE, None) == ntc.NTC_ERR_ARG
    assert f(FAKE, 10, FAKE, 4, 2, None, 11, 64, FAKE, FAKE, None) == ntc.NTC_ERR_ARG
    assert f(FAKE, 10, FAKE, 4, 2, None, 10, 64, FAKE, None, None) == ntc.NTC_ERR_ARG
    assert f(FAKE, -1, FAKE, 4, 2, None, 0, 64, FAKE, FAKE, None) == ntc.NTC_ERR_ARG


def test_divergence_map_validation(L):
    f = L.ntc_divergence_map
    ok = dict(tex=FAKE, W=10, H=10, spp=1, t2d=FAKE, T=4, D=2, bw=8, bh=8, map=FAKE, hist=FAKE,
              hl=9, tot=FAKE)

    def call(**kw):
        a = dict(ok)
        a.update(kw)
        return f(a["tex"], a["W"], a["H"], a["spp"], a["t2d"], a["T"], a["D"], a["bw"], a["bh"],
                 a["map"], a["hist"], a["hl"], a["tot"], None)

    assert call(tex=None) == ntc.NTC_ERR_ARG
    assert call(t2d=None) == ntc.NTC_ERR_ARG
    assert call(W=0) == ntc.NTC_ERR_ARG
    assert call(spp=65) == ntc.NTC_ERR_ARG
    assert call(bw=0) == ntc.NTC_ERR_ARG
    assert call(D=4097) == ntc.NTC_ERR_ARG
    assert call(hl=0) == ntc.NTC_ERR_ARG
    assert call(hl=4097) == ntc.NTC_ERR_ARG
    assert call(W=1 << 16, H=1 << 16, spp=2) == ntc.NTC_ERR_ARG


def test_decode_pointer_alignment(L):
    """Taps are 16-byte loads from latents, (u, v) one 8-byte load: misaligned
    pointers are argument errors, whatever the mode; with no queries nothing is
    read."""
    off = lambda b: ctypes.c_void_p(0x100000 + b)  # noqa: E731
    for binned in (False, True):
        for b in (2, 4, 8):
            assert _decode(L, binned=binned, ptrs={"latents": off(b)}) == ntc.NTC_ERR_ARG
        assert _decode(L, binned=binned, ptrs={"uv": off(4)}) == ntc.NTC_ERR_ARG
        assert _decode(L, binned=binned, ptrs={"tex_id": off(2)}) == ntc.NTC_ERR_ARG
        assert _decode(L, binned=binned, ptrs={"mip": off(1)}) == ntc.NTC_ERR_ARG
        assert _decode(L, binned=binned, ptrs={"out": off(2)}) == ntc.NTC_ERR_ARG
        assert _decode(L, binned=binned, n=0, ptrs={"latents": off(8)}) == ntc.NTC_OK
        if not HAS_DEVICE:  # aligned but not 16-byte-multiple offsets are accepted
            assert _decode(L, binned=binned, ptrs={"latents": off(16), "uv": off(8),
                                                   "tex_id": off(4), "out": off(4)}) \
                == ntc.NTC_ERR_HIP


def test_decode_gather_validation(L):
    """The LDS-staged gather: binned MFMA decode of 2 levels without mip and at
    most 8 output channels; an unknown gather is an argument error."""
    def call(gather, binned=True, dims=(32, 64, 64, 8), res=(256, 128), ch=(16, 16),
             engine=ntc.NTC_ENGINE_MFMA, mip=False, n=100):
        g = ntc.Grids()
        g.n_textures, g.n_levels = 4, len(res)
        for i, (r, c) in enumerate(zip(res, ch)):
            g.res[i], g.channels[i] = r, c
        g.latents = FAKE
        d = ntc.Decoders()
        d.n_decoders, d.n_layers = 4, len(dims) - 1
        for i, v in enumerate(dims):
            d.dims[i] = v
        d.params = FAKE
        q = ntc.Queries()
        q.tex_id, q.uv, q.mip, q.n = FAKE, FAKE, FAKE if mip else None, n
        o = ntc.DecodeOptions(ntc.NTC_ACT_RELU, 0.0, ntc.NTC_OUT_F32, 0, engine, gather)
        cap = ntc.perm_capacity(n, 4, 64)
        return L.ntc_decode_ex(ctypes.byref(g), ctypes.byref(d), FAKE, ctypes.byref(q),
                               FAKE if binned else None, FAKE if binned else None, cap,
                               64 if binned else 0, ctypes.byref(o), FAKE, None)

    S = ntc.NTC_GATHER_STAGED
    assert call(2) == ntc.NTC_ERR_ARG
    assert call(-1) == ntc.NTC_ERR_ARG
    assert call(S, binned=False) == ntc.NTC_ERR_UNSUPPORTED
    assert call(S, engine=ntc.NTC_ENGINE_FMA) == ntc.NTC_ERR_UNSUPPORTED
    assert call(S, mip=True) == ntc.NTC_ERR_UNSUPPORTED
    assert call(S, dims=(32, 64, 64, 12)) == ntc.NTC_ERR_UNSUPPORTED
    assert call(S, res=(256, 128, 64), ch=(16, 16, 16), dims=(48, 64, 64, 8)) \
        == ntc.NTC_ERR_UNSUPPORTED
    assert call(ntc.NTC_GATHER_DIRECT, dims=(32, 64, 64, 12), n=0) == ntc.NTC_OK
    if not HAS_DEVICE:  # accepted shapes reach the launch
        for dims, ch in (((32, 64, 64, 8), (16, 16)), ((16, 64, 64, 3), (8, 8)),
                         ((32, 128, 128, 5), (16, 16)), ((32, 64, 64, 64, 8), (16, 16))):
            assert call(S, dims=dims, ch=ch) == ntc.NTC_ERR_HIP


def test_gather_features_validation(L):
    """ntc_gather_features: the decode's grid shapes, an output format, and
    aligned pointers (latents and out 16 bytes, uv 8, tex_id and mip 4); with no
    queries nothing is read."""
    off = lambda b: ctypes.c_void_p(0x100000 + b)  # noqa: E731

    def call(res=(256, 128), ch=(16, 16), fmt=ntc.NTC_OUT_F32, n=100, mip=False, ptrs=None,
             n_textures=4):
        p = {"latents": FAKE, "tex_id": FAKE, "uv": FAKE, "mip": FAKE if mip else None,
             "out": FAKE}
        p.update(ptrs or {})
        g = ntc.Grids()
        g.n_textures, g.n_levels = n_textures, len(res)
        for i, (r, c) in enumerate(zip(res, ch)):
            g.res[i], g.channels[i] = r, c
        g.latents = p["latents"]
        q = ntc.Queries()
        q.tex_id, q.uv, q.mip, q.n = p["tex_id"], p["uv"], p["mip"], n
        return L.ntc_gather_features(ctypes.byref(g), ctypes.byref(q), p["out"], fmt, None)

    assert L.ntc_gather_features(None, None, FAKE, 0, None) == ntc.NTC_ERR_ARG
    assert call(fmt=2) == ntc.NTC_ERR_ARG
    assert call(fmt=-1) == ntc.NTC_ERR_ARG
    assert call(n=-1) == ntc.NTC_ERR_ARG
    assert call(n_textures=0) == ntc.NTC_ERR_ARG
    assert call(res=(256, 0)) == ntc.NTC_ERR_ARG
    assert call(ptrs={"out": None}) == ntc.NTC_ERR_ARG
    assert call(ptrs={"uv": None}) == ntc.NTC_ERR_ARG
    for b in (2, 4, 8):
        assert call(ptrs={"latents": off(b)}) == ntc.NTC_ERR_ARG
        assert call(ptrs={"out": off(b)}) == ntc.NTC_ERR_ARG
    assert call(ptrs={"uv": off(4)}) == ntc.NTC_ERR_ARG
    assert call(ptrs={"tex_id": off(2)}) == ntc.NTC_ERR_ARG
    assert call(mip=True, ptrs={"mip": off(2)}) == ntc.NTC_ERR_ARG
    # shapes the decode does not take
    assert call(res=(256, 128), ch=(16, 8)) == ntc.NTC_ERR_UNSUPPORTED
    assert call(res=(256, 1)) == ntc.NTC_ERR_UNSUPPORTED
    assert call(res=(256,), ch=(16,)) == ntc.NTC_ERR_UNSUPPORTED
    assert call(res=(256, 128), ch=(4, 4)) == ntc.NTC_ERR_UNSUPPORTED
    assert call(res=(256, 128), ch=(4, 4), n=0) == ntc.NTC_ERR_UNSUPPORTED
    for res, ch in (((256, 128), (16, 16)), ((64, 32), (8, 8)), ((512, 256, 128), (16,) * 3)):
        assert call(res=res, ch=ch, n=0) == ntc.NTC_OK
        if not HAS_DEVICE:  # accepted shapes reach the launch
            assert call(res=res, ch=ch, fmt=ntc.NTC_OUT_F16, mip=True) == ntc.NTC_ERR_HIP


def test_decode_options_validation(L):
    g = ntc.Grids()
    g.n_textures, g.n_levels = 4, 2
    for i, (r, c) in enumerate(zip((256, 128), (16, 16))):
        g.res[i], g.channels[i] = r, c
    g.latents = FAKE
    d = ntc.Decoders()
    d.n_decoders, d.n_layers = 4, 3
    for i, v in enumerate((32, 64, 64, 8)):
        d.dims[i] = v
    d.params = FAKE
    q = ntc.Queries()
    q.tex_id, q.uv, q.mip, q.n = FAKE, FAKE, None, 100

    def call(act, slope, fmt, pe=0):
        o = ntc.DecodeOptions(act, slope, fmt, pe)
        return L.ntc_decode_ex(ctypes.byref(g), ctypes.byref(d), FAKE, ctypes.byref(q), None,
                               None, 0, 0, ctypes.byref(o), FAKE, None)

    assert call(2, 0.0, 0) == ntc.NTC_ERR_ARG                 # unknown activation
    assert call(ntc.NTC_ACT_LEAKY_RELU, 0.0, 0) == ntc.NTC_ERR_ARG
    assert call(ntc.NTC_ACT_LEAKY_RELU, 1.0, 0) == ntc.NTC_ERR_ARG
    assert call(ntc.NTC_ACT_RELU, 0.0, 2) == ntc.NTC_ERR_ARG  # unknown output format
    if not HAS_DEVICE:
        assert call(ntc.NTC_ACT_LEAKY_RELU, 0.01, ntc.NTC_OUT_F16) == ntc.NTC_ERR_HIP
    # positional encoding: 0, 4 or 8 octaves; dims[0] must include its 4K values
    assert call(ntc.NTC_ACT_RELU, 0.0, 0, pe=3) == ntc.NTC_ERR_ARG
    assert call(ntc.NTC_ACT_RELU, 0.0, 0, pe=-4) == ntc.NTC_ERR_ARG
    assert call(ntc.NTC_ACT_RELU, 0.0, 0, pe=4) == ntc.NTC_ERR_ARG   # dims[0] is still 32
    d.dims[0] = 48
    if not HAS_DEVICE:
        assert call(ntc.NTC_ACT_LEAKY_RELU, 0.01, 0, pe=4) == ntc.NTC_ERR_HIP  # built: launches
    assert call(ntc.NTC_ACT_RELU, 0.0, 0, pe=8) == ntc.NTC_ERR_ARG   # 32 + 32 != 48
    d.n_layers = 4
    for i, v in enumerate((48, 64, 64, 64, 8)):
        d.dims[i] = v
    assert call(ntc.NTC_ACT_RELU, 0.0, 0, pe=4) == ntc.NTC_ERR_UNSUPPORTED  # two hidden->hidden


def test_decode_engine_validation(L):
    """The FMA engine (the paper's Non-Shared FMA, Sec. 4.4): stream mode only,
    8- or 16-wide outputs, 16-byte aligned parameters; an unknown engine is an
    argument error."""
    g = ntc.Grids()
    g.n_textures, g.n_levels = 4, 2
    for i, (r, c) in enumerate(zip((256, 128), (16, 16))):
        g.res[i], g.channels[i] = r, c
    g.latents = FAKE
    d = ntc.Decoders()
    d.n_decoders, d.n_layers = 4, 3
    for i, v in enumerate((32, 64, 64, 8)):
        d.dims[i] = v
    d.params = FAKE
    q = ntc.Queries()
    q.tex_id, q.uv, q.mip, q.n = FAKE, FAKE, None, 100

    def call(engine, binned=False, n=100):
        q.n = n
        o = ntc.DecodeOptions(ntc.NTC_ACT_RELU, 0.0, ntc.NTC_OUT_F32, 0, engine)
        cap = ntc.perm_capacity(n, 4, 64)
        return L.ntc_decode_ex(ctypes.byref(g), ctypes.byref(d), FAKE, ctypes.byref(q),
                               FAKE if binned else None, FAKE if binned else None, cap,
                               64 if binned else 0, ctypes.byref(o), FAKE, None)

    assert call(3) == ntc.NTC_ERR_ARG
    assert call(-1) == ntc.NTC_ERR_ARG
    assert call(ntc.NTC_ENGINE_FMA, binned=True) == ntc.NTC_ERR_UNSUPPORTED
    assert call(ntc.NTC_ENGINE_FMA_DIRECT, binned=True) == ntc.NTC_ERR_UNSUPPORTED
    assert call(ntc.NTC_ENGINE_FMA, n=0) == ntc.NTC_OK
    if not HAS_DEVICE:
        assert call(ntc.NTC_ENGINE_FMA) == ntc.NTC_ERR_HIP  # built: launches on FAKE
    d.params = ctypes.c_void_p(0x100000 + 8)
    assert call(ntc.NTC_ENGINE_FMA) == ntc.NTC_ERR_ARG     # not 16-byte aligned
    assert call(ntc.NTC_ENGINE_MFMA, n=0) == ntc.NTC_OK    # the MFMA engine has no such need
    d.params = FAKE
    for out_dim in (3, 4, 12):
        d.dims[3] = out_dim
        assert call(ntc.NTC_ENGINE_FMA) == ntc.NTC_ERR_UNSUPPORTED
        assert call(ntc.NTC_ENGINE_FMA_DIRECT) == ntc.NTC_ERR_UNSUPPORTED
    d.dims[3] = 16
    if not HAS_DEVICE:
        assert call(ntc.NTC_ENGINE_FMA) == ntc.NTC_ERR_HIP


def test_kmeans_validation(L):
    ws = ctypes.c_void_p(0x100000)
    seeds = (ctypes.c_uint32 * 4)(0, 5, 9, 2)
    dup = (ctypes.c_uint32 * 4)(0, 5, 5, 2)
    big = (ctypes.c_uint32 * 4)(0, 5, 10, 2)
    wsb = L.ntc_kmeans_workspace_bytes(4, 20)
    assert wsb == (4 + 20) * 4
    assert L.ntc_kmeans_workspace_bytes(0, 20) == 0
    assert L.ntc_kmeans_workspace_bytes(4, 0) == 0

    def call(n=10, dim=8, m=4, init=seeds, it=20, ws=ws, wsb=wsb, feats=FAKE):
        return L.ntc_kmeans(feats, n, dim, m, init, it, FAKE, FAKE, FAKE, ws, wsb, None)

    assert call(feats=None) == ntc.NTC_ERR_ARG
    assert call(init=None) == ntc.NTC_ERR_ARG
    assert call(ws=None) == ntc.NTC_ERR_ARG
    assert call(n=0) == ntc.NTC_ERR_ARG
    assert call(dim=0) == ntc.NTC_ERR_ARG
    assert call(n=3) == ntc.NTC_ERR_ARG           # more groups than textures
    assert call(it=0) == ntc.NTC_ERR_ARG
    assert call(init=dup) == ntc.NTC_ERR_ARG      # seeds must be distinct
    assert call(init=big) == ntc.NTC_ERR_ARG      # seed past the last texture
    assert call(ws=ctypes.c_void_p(0x100002)) == ntc.NTC_ERR_ARG
    assert call(wsb=wsb - 4) == ntc.NTC_ERR_CAPACITY
    assert L.ntc_kmeans_result(None, 4, 20, None, None, None) == ntc.NTC_ERR_ARG
    if not HAS_DEVICE:
        assert call() == ntc.NTC_ERR_HIP  # valid: its seed copy fails without a device


def _bins_noalloc(L, **kw):
    a = dict(tex_id=FAKE, n=100, tex_to_dec=FAKE, T=4, D=2, align=64, cnt=FAKE, off=FAKE,
             perm=FAKE, cap=100 + 2 * 63, inv=None)
    a.update(kw)
    return L.ntc_build_bins_noalloc(a["tex_id"], a["n"], a["tex_to_dec"], a["T"], a["D"],
                                    a["align"], a["cnt"], a["off"], a["perm"], a["cap"],
                                    a["inv"], None)


def test_build_bins_noalloc_validation(L):
    assert _bins_noalloc(L, n=-1) == ntc.NTC_ERR_ARG
    assert _bins_noalloc(L, tex_id=None) == ntc.NTC_ERR_ARG
    assert _bins_noalloc(L, perm=None) == ntc.NTC_ERR_ARG
    assert _bins_noalloc(L, cnt=None) == ntc.NTC_ERR_ARG
    assert _bins_noalloc(L, D=4097) == ntc.NTC_ERR_ARG
    assert _bins_noalloc(L, align=48) == ntc.NTC_ERR_ARG
    assert _bins_noalloc(L, cap=100 + 2 * 63 - 1) == ntc.NTC_ERR_CAPACITY
    # the scratch bound: the workspace is one count per (slice, decoder) plus the
    # invalid row, at most 1 Mi words whatever n, so every valid call fits
    limit = ntc.NOALLOC_SCRATCH_BYTES
    for n in (0, 1, 65536, 3840 * 2160 * 4, 40_000_000, (1 << 32) - 2):
        for D in (1, 2, 16, 63, 64, 512, 1023, 4096):
            ws = ntc.workspace_bytes(n, D)
            assert 0 < ws <= 16 + 4 * (1 << 20) <= limit


def test_noalloc_scratch_size_matches_header():
    text = open(HEADER).read()
    m = re.search(r"#define NTC_NOALLOC_SCRATCH_BYTES \((\d+)u << (\d+)\)", text)
    assert m and int(m.group(1)) << int(m.group(2)) == ntc.NOALLOC_SCRATCH_BYTES
