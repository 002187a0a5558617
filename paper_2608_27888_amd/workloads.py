"""Seeded synthetic inputs for neural texture decode.

This module only *draws* inputs: latent grids, decoder parameters, the
texture -> decoder map and the texel query stream.  It holds none of the decode
arithmetic (no sampling, no MLP, no binning), so both the HIP path and the CPU
oracle can be fed from it without sharing any of the method's code.

Shapes follow the neural-texture-compression setting of the paper (Sec. 1 and
Sec. 4 "Results"): every texture owns a small multi-resolution latent grid, a
decoder MLP is chosen per texture through the map c(i) (Alg. "Overall texture
processing pipeline", Stage 2), and the renderer issues one query per pixel
sample.  The paper's data (Polyhaven textures, the three rendered scenes, the
trained networks) is not available, so every array here is synthetic:

* latents ~ N(0, 1), stored as fp16 (the paper decodes in FP16, Sec. 4.4);
* weights Kaiming-uniform, bound sqrt(6 / fan_in); biases U(-0.1, 0.1); fp16;
* screen-space query streams in row-major pixel order with per-sample jitter;
* material layouts either per 8x8 tile or a Voronoi map of seeded regions.

Every component draws from its own child of ``numpy.random.SeedSequence(seed)``
(latents, decoders, map, queries), so a variant with a different decoder count
shares latents and queries with its base workload.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional

import numpy as np

# Child-stream indices of the seed sequence, one per drawn component.
(_STREAM_LATENTS, _STREAM_DECODERS, _STREAM_MAP, _STREAM_QUERIES, _STREAM_LAYOUT,
 _STREAM_FEATURES, _STREAM_SEEDS) = range(7)

F32_BELOW_ONE = np.nextafter(np.float32(1.0), np.float32(0.0))


def _rng(seed: int, stream: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence(seed).spawn(8)[stream])


@dataclass
class Workload:
    """One decode problem: grids, decoders, map and queries (host arrays)."""

    name: str
    # latent grids (uniform across textures)
    n_textures: int
    res: list                    # per level: square resolution
    channels: list               # per level: channels per texel
    latents: np.ndarray          # uint16 fp16 bits, [T * texture_stride]
    # decoders
    n_decoders: int
    dims: list                   # layer widths d_0 .. d_L (d_0 = sum(channels))
    params: np.ndarray           # uint16 fp16 bits, [D * decoder_stride]
    tex_to_dec: np.ndarray       # uint32 [T]
    # queries
    tex_id: np.ndarray           # uint32 [N]
    uv: np.ndarray               # float32 [N, 2]
    mip: Optional[np.ndarray]    # float32 [N] or None (=> 0)
    screen: Optional[tuple] = None  # (width, height, samples per pixel)
    meta: dict = field(default_factory=dict)
    pe_octaves: int = 0          # positional-encoding octaves of the decoder input

    @property
    def n(self) -> int:
        return int(self.tex_id.shape[0])

    @property
    def n_levels(self) -> int:
        return len(self.res)

    @property
    def n_layers(self) -> int:
        return len(self.dims) - 1

    @property
    def out_dim(self) -> int:
        return int(self.dims[-1])

    @property
    def texture_stride(self) -> int:
        return texture_stride(self.res, self.channels)

    @property
    def decoder_stride(self) -> int:
        return decoder_stride(self.dims)

    def flops_per_query(self) -> int:
        """Multiply-adds x 2 of the MLP, unpadded."""
        return int(sum(2 * a * b for a, b in zip(self.dims[:-1], self.dims[1:])))

    def with_dims(self, dims, seed: int = 0) -> "Workload":
        """Same grids, map and queries; decoders redrawn with layer widths `dims`
        (dims[0] must stay the feature count)."""
        assert dims[0] == self.dims[0]
        params = draw_decoders(seed, self.n_decoders, dims)
        return Workload(f"{self.name}_mlp{'-'.join(map(str, dims))}", self.n_textures,
                        list(self.res), list(self.channels), self.latents, self.n_decoders,
                        list(dims), params, self.tex_to_dec, self.tex_id, self.uv, self.mip,
                        self.screen, dict(self.meta), self.pe_octaves)

    def with_pe(self, octaves: int, dims=None, seed: int = 0) -> "Workload":
        """Same grids, map and queries; decoders redrawn for an input of the
        latent features followed by `octaves` positional-encoding octaves
        (dims[0] = sum(channels) + 4 * octaves; the other widths as given, or
        the workload's)."""
        d0 = int(sum(self.channels)) + 4 * int(octaves)
        dims = [d0] + list(self.dims[1:] if dims is None else dims[1:])
        params = draw_decoders(seed, self.n_decoders, dims)
        return Workload(f"{self.name}_pe{octaves}", self.n_textures, list(self.res),
                        list(self.channels), self.latents, self.n_decoders, dims, params,
                        self.tex_to_dec, self.tex_id, self.uv, self.mip, self.screen,
                        dict(self.meta), int(octaves))

    def with_decoders(self, n_decoders: int, tex_to_dec: np.ndarray, seed: int = 0,
                      name: Optional[str] = None) -> "Workload":
        """Same grids and queries, a different decoder set and map."""
        params = draw_decoders(seed, n_decoders, self.dims)
        return Workload(name or f"{self.name}_d{n_decoders}", self.n_textures, list(self.res),
                        list(self.channels), self.latents, n_decoders, list(self.dims), params,
                        np.ascontiguousarray(tex_to_dec, dtype=np.uint32), self.tex_id, self.uv,
                        self.mip, self.screen, dict(self.meta), self.pe_octaves)


def texture_stride(res, channels) -> int:
    return int(sum(int(r) * int(r) * int(c) for r, c in zip(res, channels)))


def decoder_stride(dims) -> int:
    return int(sum(int(b) * int(a) + int(b) for a, b in zip(dims[:-1], dims[1:])))


def level_offsets(res, channels) -> list:
    """Offset (in fp16 elements) of each level inside one texture's block."""
    offs, acc = [], 0
    for r, c in zip(res, channels):
        offs.append(acc)
        acc += int(r) * int(r) * int(c)
    return offs


def fp16_bits(a: np.ndarray) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.float32).astype(np.float16).view(np.uint16))


def bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return np.asarray(bits, dtype=np.uint16).view(np.float16).astype(np.float32)


# ----------------------------------------------------------------------------- drawing


def draw_latents(seed: int, n_textures: int, res, channels) -> np.ndarray:
    rng = _rng(seed, _STREAM_LATENTS)
    total = n_textures * texture_stride(res, channels)
    out = np.empty(total, dtype=np.uint16)
    chunk = 1 << 26
    for s in range(0, total, chunk):
        e = min(total, s + chunk)
        out[s:e] = rng.standard_normal(e - s, dtype=np.float32).astype(np.float16).view(np.uint16)
    return out


def draw_decoders(seed: int, n_decoders: int, dims) -> np.ndarray:
    """Per decoder, contiguous: W0[d1][d0], b0[d1], W1[d2][d1], b1[d2], ...

    All weights are drawn first (decoder-major, layer-major), then all biases.
    """
    rng = _rng(seed, _STREAM_DECODERS)
    ws = []
    for _ in range(n_decoders):
        per = []
        for a, b in zip(dims[:-1], dims[1:]):
            bound = np.sqrt(6.0 / a)
            per.append(rng.uniform(-bound, bound, size=(b, a)))
        ws.append(per)
    bs = [[rng.uniform(-0.1, 0.1, size=(b,)) for b in dims[1:]] for _ in range(n_decoders)]
    blob = []
    for d in range(n_decoders):
        for w, bb in zip(ws[d], bs[d]):
            blob.append(w.ravel())
            blob.append(bb)
    return fp16_bits(np.concatenate(blob))


def zipf_sizes(total: int, parts: int, s: float) -> np.ndarray:
    """Largest-remainder apportionment of `total` items with weights k^-s."""
    w = np.arange(1, parts + 1, dtype=np.float64) ** (-s)
    q = total * w / w.sum()
    f = np.floor(q).astype(np.int64)
    rem = total - int(f.sum())
    order = np.argsort(-(q - f), kind="stable")
    f[order[:rem]] += 1
    return f


def clustered_map(seed: int, n_textures: int, sizes) -> np.ndarray:
    """Textures, visited in a seeded random order, fill clusters 0, 1, ... by size."""
    rng = _rng(seed, _STREAM_MAP)
    order = rng.permutation(n_textures)
    m = np.empty(n_textures, dtype=np.uint32)
    pos = 0
    for d, sz in enumerate(sizes):
        m[order[pos:pos + sz]] = d
        pos += sz
    assert pos == n_textures
    return m


def equal_map(seed: int, n_textures: int, n_decoders: int) -> np.ndarray:
    rng = _rng(seed, _STREAM_MAP)
    return (rng.permutation(n_textures) % n_decoders).astype(np.uint32)


def _jittered_uv(rng, width, height, spp, base_x, base_y):
    """Pixel (x, y) sample s -> ((x + U) / W, (y + U) / H); one U per coordinate."""
    n = base_x.shape[0]
    jx = rng.random(n)
    jy = rng.random(n)
    u = (base_x + jx) / width
    v = (base_y + jy) / height
    return u, v


def _pixels(width, height, spp):
    """Row-major pixel coordinates, repeated per sample: q = (y * W + x) * spp + s."""
    ys, xs = np.divmod(np.arange(width * height, dtype=np.int64), width)
    if spp > 1:
        xs = np.repeat(xs, spp)
        ys = np.repeat(ys, spp)
    return xs.astype(np.float64), ys.astype(np.float64)


def voronoi_regions(rng, width, height, n_sites) -> np.ndarray:
    """Region index of every pixel centre: nearest of n_sites uniform sites."""
    from scipy.spatial import cKDTree

    sites = np.stack([rng.uniform(0, width, n_sites), rng.uniform(0, height, n_sites)], 1)
    ys, xs = np.divmod(np.arange(width * height, dtype=np.int64), width)
    pts = np.stack([xs + 0.5, ys + 0.5], 1)
    _, idx = cKDTree(sites).query(pts, k=1)
    return idx.astype(np.int64)


def _to_f32_uv(u, v):
    uv = np.stack([u, v], 1).astype(np.float32)
    np.minimum(uv, F32_BELOW_ONE, out=uv)
    np.maximum(uv, np.float32(0.0), out=uv)
    return np.ascontiguousarray(uv)


# ----------------------------------------------------------------------------- configs

# Full-size parameters of the five workloads.  Each entry is (generator, kwargs).
CONFIG_NAMES = ("tiny", "single", "divergent", "clustered4k", "wide_trilinear")


def tiny(seed: int = 0, n: int = 65536) -> Workload:
    """4 textures (64^2x8 + 32^2x8), 2 decoders (t % 2), 16->64->64->8, random queries."""
    res, ch, dims = [64, 32], [8, 8], [16, 64, 64, 8]
    lat = draw_latents(seed, 4, res, ch)
    par = draw_decoders(seed, 2, dims)
    t2d = (np.arange(4) % 2).astype(np.uint32)
    rng = _rng(seed, _STREAM_QUERIES)
    tex = rng.integers(0, 4, size=n).astype(np.uint32)
    uv = np.ascontiguousarray(rng.random((n, 2), dtype=np.float32))
    return Workload("tiny", 4, res, ch, lat, 2, dims, par, t2d, tex, uv, None, None)


def single(seed: int = 0, width: int = 1920, height: int = 1080) -> Workload:
    """1 texture (512^2x16 + 256^2x16), 1 decoder, 32->64->64->8, screen-coherent uv."""
    res, ch, dims = [512, 256], [16, 16], [32, 64, 64, 8]
    lat = draw_latents(seed, 1, res, ch)
    par = draw_decoders(seed, 1, dims)
    rng = _rng(seed, _STREAM_QUERIES)
    xs, ys = _pixels(width, height, 1)
    u, v = _jittered_uv(rng, width, height, 1, xs, ys)
    tex = np.zeros(width * height, dtype=np.uint32)
    return Workload("single", 1, res, ch, lat, 1, dims, par, np.zeros(1, np.uint32), tex,
                    _to_f32_uv(u, v), None, (width, height, 1))


def divergent(seed: int = 0, width: int = 1920, height: int = 1080) -> Workload:
    """64 textures, one decoder each; texture fixed per 8x8 pixel tile, uniform in [0, 64)."""
    res, ch, dims = [256, 128], [16, 16], [32, 64, 64, 8]
    T = 64
    lat = draw_latents(seed, T, res, ch)
    par = draw_decoders(seed, T, dims)
    t2d = np.arange(T, dtype=np.uint32)
    lay = _rng(seed, _STREAM_LAYOUT)
    tw, th = (width + 7) // 8, (height + 7) // 8
    tile_tex = lay.integers(0, T, size=(th, tw)).astype(np.uint32)
    rng = _rng(seed, _STREAM_QUERIES)
    xs, ys = _pixels(width, height, 1)
    u, v = _jittered_uv(rng, width, height, 1, xs, ys)
    tex = tile_tex[(ys.astype(np.int64) >> 3), (xs.astype(np.int64) >> 3)]
    return Workload("divergent", T, res, ch, lat, T, dims, par, t2d,
                    np.ascontiguousarray(tex, dtype=np.uint32), _to_f32_uv(u, v), None,
                    (width, height, 1))


def _voronoi_queries(seed, width, height, spp, n_sites, n_textures, with_mip):
    lay = _rng(seed, _STREAM_LAYOUT)
    region = voronoi_regions(lay, width, height, n_sites)
    region_tex = lay.integers(0, n_textures, size=n_sites)
    off = lay.random((n_sites, 2))
    scale = 2.0 ** lay.uniform(-1.0, 2.0, size=n_sites)
    rng = _rng(seed, _STREAM_QUERIES)
    xs, ys = _pixels(width, height, spp)
    reg = np.repeat(region, spp) if spp > 1 else region
    jx = rng.random(xs.shape[0])
    jy = rng.random(xs.shape[0])
    u = np.mod(off[reg, 0] + scale[reg] * (xs + jx) / width, 1.0)
    v = np.mod(off[reg, 1] + scale[reg] * (ys + jy) / height, 1.0)
    mip = None
    if with_mip:
        mip = np.ascontiguousarray(rng.uniform(0.0, 2.0, size=xs.shape[0]).astype(np.float32))
    tex = np.ascontiguousarray(region_tex[reg], dtype=np.uint32)
    return tex, _to_f32_uv(u, v), mip


def _scaled_sites(width, height, full=(3840, 2160), sites=2000):
    return max(4, int(round(sites * (width * height) / (full[0] * full[1]))))


def clustered4k(seed: int = 0, width: int = 3840, height: int = 2160,
                n_decoders: int = 16, n_textures: int = 512) -> Workload:
    """512 textures, 16 Zipf(1.1)-sized decoder clusters, Voronoi material map.

    ``n_decoders == n_textures`` gives the per-texture-decoder comparison
    (identity map).
    """
    res, ch, dims = [256, 128], [16, 16], [32, 64, 64, 8]
    T = n_textures
    lat = draw_latents(seed, T, res, ch)
    if n_decoders == T:
        t2d = np.arange(T, dtype=np.uint32)
    else:
        t2d = clustered_map(seed, T, zipf_sizes(T, n_decoders, 1.1))
    par = draw_decoders(seed, n_decoders, dims)
    n_sites = _scaled_sites(width, height)
    tex, uv, _ = _voronoi_queries(seed, width, height, 1, n_sites, T, False)
    return Workload(f"clustered4k_d{n_decoders}", T, res, ch, lat, n_decoders, dims, par, t2d,
                    tex, uv, None, (width, height, 1), {"voronoi_sites": n_sites})


def wide_trilinear(seed: int = 0, width: int = 3840, height: int = 2160, spp: int = 4,
                   n_decoders: int = 8, n_textures: int = 512) -> Workload:
    """512 textures with 3-level pyramids, 48->128->128->128->8, 4 spp, mip ~ U[0, 2)."""
    res, ch, dims = [512, 256, 128], [16, 16, 16], [48, 128, 128, 128, 8]
    T = n_textures
    lat = draw_latents(seed, T, res, ch)
    if n_decoders == T:
        t2d = np.arange(T, dtype=np.uint32)
    else:
        t2d = equal_map(seed, T, n_decoders)
    par = draw_decoders(seed, n_decoders, dims)
    n_sites = _scaled_sites(width, height)
    tex, uv, mip = _voronoi_queries(seed, width, height, spp, n_sites, T, True)
    return Workload(f"wide_trilinear_d{n_decoders}", T, res, ch, lat, n_decoders, dims, par, t2d,
                    tex, uv, mip, (width, height, spp), {"voronoi_sites": n_sites})


def k_per_wave(seed: int = 0, side: int = 512, k: int = 5, n_textures: int = 10) -> Workload:
    """The layout of the paper's timing study (Sec. 4.4, Tables performance_5dec and
    performance_10dec): a side x side output image, one query per pixel in row-major
    order, and k decoders spread uniformly over every 64-query wave (lane l of a wave
    uses decoder l mod k; k = 1 is the shared decoder).  Each decoder has its own
    texture; grids and MLP as the clustered 4K workload (256^2x16 + 128^2x16,
    32->64->64->8); uv screen-coherent over the image.
    """
    if not 1 <= k <= n_textures:
        raise ValueError("need 1 <= k <= n_textures")
    res, ch, dims = [256, 128], [16, 16], [32, 64, 64, 8]
    T = n_textures
    lat = draw_latents(seed, T, res, ch)
    par = draw_decoders(seed, T, dims)
    t2d = np.arange(T, dtype=np.uint32)
    rng = _rng(seed, _STREAM_QUERIES)
    xs, ys = _pixels(side, side, 1)
    u, v = _jittered_uv(rng, side, side, 1, xs, ys)
    tex = (np.arange(side * side, dtype=np.int64) % kWaveLanes % k).astype(np.uint32)
    return Workload(f"k{k}_per_wave_{side}", T, res, ch, lat, T, dims, par, t2d, tex,
                    _to_f32_uv(u, v), None, (side, side, 1), {"k": k})


kWaveLanes = 64  # queries per wave of the decode kernels


def make(name: str, seed: int = 0, **kw) -> Workload:
    gens = {"tiny": tiny, "single": single, "divergent": divergent,
            "clustered4k": clustered4k, "wide_trilinear": wide_trilinear}
    return gens[name](seed=seed, **kw)


def cached(name: str, seed: int = 0, cache_dir: Optional[str] = None, **kw) -> Workload:
    """make(name, seed, **kw) through an on-disk cache of .npy files.

    The key is the workload's name, seed and keyword arguments together with a
    hash of this module's source, so a changed generator never reads a stale
    entry.  Arrays are written with numpy.save and read back with numpy.load
    (no pickling); the scalar fields go to a JSON file.  Without cache_dir this
    is make().
    """
    if not cache_dir:
        return make(name, seed, **kw)
    import hashlib
    import json
    import os

    with open(__file__, "rb") as fh:
        src = hashlib.sha256(fh.read()).hexdigest()[:16]
    key = hashlib.sha256(json.dumps([name, seed, sorted(kw.items()), src]).encode()).hexdigest()[:24]
    d = os.path.join(cache_dir, f"{name}_s{seed}_{key}")
    arrays = ("latents", "params", "tex_to_dec", "tex_id", "uv", "mip")
    meta_path = os.path.join(d, "workload.json")
    if os.path.exists(meta_path):
        with open(meta_path) as fh:
            m = json.load(fh)
        a = {k: (np.load(os.path.join(d, k + ".npy")) if m["has"][k] else None) for k in arrays}
        return Workload(m["name"], m["n_textures"], m["res"], m["channels"], a["latents"],
                        m["n_decoders"], m["dims"], a["params"], a["tex_to_dec"], a["tex_id"],
                        a["uv"], a["mip"], tuple(m["screen"]) if m["screen"] else None,
                        m["meta"], m["pe_octaves"])
    w = make(name, seed, **kw)
    tmp = d + ".tmp%d" % os.getpid()
    os.makedirs(tmp, exist_ok=True)
    for k in arrays:
        v = getattr(w, k)
        if v is not None:
            np.save(os.path.join(tmp, k + ".npy"), v)
    with open(os.path.join(tmp, "workload.json"), "w") as fh:
        json.dump({"name": w.name, "n_textures": w.n_textures, "res": list(w.res),
                   "channels": list(w.channels), "n_decoders": w.n_decoders,
                   "dims": list(w.dims), "screen": list(w.screen) if w.screen else None,
                   "meta": w.meta, "pe_octaves": w.pe_octaves,
                   "has": {k: getattr(w, k) is not None for k in arrays}}, fh)
    try:
        os.rename(tmp, d)
    except OSError:  # another process stored it first
        import shutil

        shutil.rmtree(tmp, ignore_errors=True)
    return w


def small(name: str, seed: int = 0) -> Workload:
    """Reduced-screen version of a workload: same structure, oracle-friendly size.

    The screen sizes are chosen to span many 64-query tiles and to leave a
    ragged tail (N is not a multiple of 64 or 256).
    """
    if name == "tiny":
        return tiny(seed, n=65536 + 37)
    if name == "single":
        return single(seed, 333, 121)
    if name == "divergent":
        return divergent(seed, 331, 123)
    # Fewer textures keep the latent pools small; the decoder maps keep their
    # structure (Zipf-sized clusters, equal clusters, or one decoder per texture).
    if name == "clustered4k":
        return clustered4k(seed, 397, 223, n_decoders=16, n_textures=64)
    if name == "clustered4k_d512":
        return clustered4k(seed, 397, 223, n_decoders=64, n_textures=64)
    if name == "wide_trilinear":
        return wide_trilinear(seed, 161, 97, 4, n_decoders=8, n_textures=16)
    if name == "wide_trilinear_d512":
        return wide_trilinear(seed, 161, 97, 4, n_decoders=16, n_textures=16)
    if name in ("k5_per_wave", "k10_per_wave"):
        return k_per_wave(seed, 99, int(name[1:name.index("_")]))
    raise KeyError(name)


# ------------------------------------------------------------------ clustering inputs


def texture_features(seed: int = 0, n_textures: int = 512, n_groups: int = 16, dim: int = 512,
                     spread: float = 0.35):
    """Synthetic stand-ins for the per-texture CLIP embeddings of Stage 1 (Sec. 3.3;
    the textures and the CLIP model are not available): n_groups "semantic" centres
    drawn uniformly on the unit sphere of R^dim, group sizes Zipf(1.1) by largest
    remainder, textures dealt to groups in a seeded random order, and each feature
    vector its centre plus isotropic noise of norm about `spread`, scaled back to
    unit length as CLIP embeddings are.  Returns (features float32 [n][dim], the
    generating group of each texture)."""
    rng = _rng(seed, _STREAM_FEATURES)
    centres = rng.standard_normal((n_groups, dim))
    centres /= np.linalg.norm(centres, axis=1, keepdims=True)
    sizes = zipf_sizes(n_textures, n_groups, 1.1)
    group = np.repeat(np.arange(n_groups), sizes)[rng.permutation(n_textures)]
    f = centres[group] + rng.standard_normal((n_textures, dim)) * (spread / np.sqrt(dim))
    f /= np.linalg.norm(f, axis=1, keepdims=True)
    return f.astype(np.float32), group.astype(np.uint32)


def kmeans_seeds(seed: int, n_textures: int, m: int) -> np.ndarray:
    """Seed textures of the clustering: m distinct textures drawn uniformly (the
    paper does not state a seeding)."""
    rng = _rng(seed, _STREAM_SEEDS)
    return np.sort(rng.choice(n_textures, size=m, replace=False)).astype(np.uint32)
