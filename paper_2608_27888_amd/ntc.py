"""Python binding of libntc (ctypes): argument marshalling only.

Every step of the decode path runs in the HIP kernels of ``libntc.so``; this
module passes device pointers (``tensor.data_ptr()``) and the current HIP
stream.  PyTorch is used for device memory and streams only.  There is no
fallback: if the library is missing the import of the binding fails loudly.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

import numpy as np
import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libntc.so")

NTC_OK = 0
NTC_ERR_ARG = -1
NTC_ERR_UNSUPPORTED = -2
NTC_ERR_CAPACITY = -3
NTC_ERR_HIP = -4
NTC_ERR_INDEX = -5
NTC_PAD = 0xFFFFFFFF
MAX_LEVELS = 4
MAX_LAYERS = 8


class NtcError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__(f"{fn} failed: {status} ({status_string(status)})")
        self.status = status


class Grids(ctypes.Structure):
    _fields_ = [("n_textures", ctypes.c_int32), ("n_levels", ctypes.c_int32),
                ("res", ctypes.c_int32 * MAX_LEVELS), ("channels", ctypes.c_int32 * MAX_LEVELS),
                ("latents", ctypes.c_void_p)]


class Decoders(ctypes.Structure):
    _fields_ = [("n_decoders", ctypes.c_int32), ("n_layers", ctypes.c_int32),
                ("dims", ctypes.c_int32 * (MAX_LAYERS + 1)), ("params", ctypes.c_void_p)]


class Queries(ctypes.Structure):
    _fields_ = [("tex_id", ctypes.c_void_p), ("uv", ctypes.c_void_p), ("mip", ctypes.c_void_p),
                ("n", ctypes.c_int64)]


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2608_27888_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        P, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
        L.ntc_status_string.argtypes = [ctypes.c_int]
        L.ntc_status_string.restype = ctypes.c_char_p
        L.ntc_bins_workspace_bytes.argtypes = [i64, i32]
        L.ntc_bins_workspace_bytes.restype = sz
        L.ntc_bins_capacity.argtypes = [i64, i32, i32]
        L.ntc_bins_capacity.restype = i64
        L.ntc_build_bins.argtypes = [P, i64, P, i32, i32, i32, P, P, P, i64, P, sz, P]
        L.ntc_build_bins_noalloc.argtypes = [P, i64, P, i32, i32, i32, P, P, P, i64, P, P]
        L.ntc_get_device_error.argtypes = [P, P, P]
        L.ntc_decode.argtypes = [ctypes.POINTER(Grids), ctypes.POINTER(Decoders), P,
                                 ctypes.POINTER(Queries), P, P, i64, i32, P, P]
        L.ntc_decode_ex.argtypes = [ctypes.POINTER(Grids), ctypes.POINTER(Decoders), P,
                                    ctypes.POINTER(Queries), P, P, i64, i32, P, P, P]
        L.ntc_gather_features.argtypes = [ctypes.POINTER(Grids), ctypes.POINTER(Queries), P, i32,
                                          P]
        L.ntc_divergence_stats.argtypes = [P, i64, P, i32, i32, P, i64, i32, P, P, P]
        L.ntc_divergence_map.argtypes = [P, i32, i32, i32, P, i32, i32, i32, i32, P, P, i32, P, P]
        L.ntc_kmeans_workspace_bytes.argtypes = [i32, i32]
        L.ntc_kmeans_workspace_bytes.restype = sz
        L.ntc_kmeans.argtypes = [P, i32, i32, i32, P, i32, P, P, P, P, sz, P]
        L.ntc_kmeans_result.argtypes = [P, i32, i32, P, P, P]
        d = ctypes.c_double
        L.ntc_freeze_scale.argtypes = [d, d, d]
        L.ntc_freeze_scale.restype = d
        for f in ("ntc_build_bins", "ntc_build_bins_noalloc", "ntc_get_device_error", "ntc_decode", "ntc_decode_ex",
                  "ntc_gather_features",
                  "ntc_divergence_stats", "ntc_divergence_map", "ntc_kmeans",
                  "ntc_kmeans_result"):
            getattr(L, f).restype = ctypes.c_int
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().ntc_status_string(int(status)).decode()


def _check(fn: str, status: int):
    if status != NTC_OK:
        raise NtcError(fn, status)


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("libntc takes device tensors")
    if not t.is_contiguous():
        raise ValueError("libntc takes contiguous tensors")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream: Optional[torch.cuda.Stream]):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


# ----------------------------------------------------------------------------- binning


def workspace_bytes(n: int, n_decoders: int) -> int:
    return int(lib().ntc_bins_workspace_bytes(n, n_decoders))


def perm_capacity(n: int, n_decoders: int, align: int = 64) -> int:
    return int(lib().ntc_bins_capacity(n, n_decoders, align))


@dataclass
class Bins:
    """Outputs of ntc_build_bins (device tensors, uint32 stored as int32)."""

    bin_count: torch.Tensor
    bin_offset: torch.Tensor
    perm: torch.Tensor
    workspace: torch.Tensor
    align: int

    @property
    def capacity(self) -> int:
        return int(self.perm.numel())


def alloc_bins(n: int, n_decoders: int, align: int = 64, device="cuda") -> Bins:
    cap = perm_capacity(n, n_decoders, align)
    ws = workspace_bytes(n, n_decoders)
    if cap < 0 or ws == 0:
        raise NtcError("alloc_bins", NTC_ERR_ARG)
    return Bins(torch.empty(n_decoders, dtype=torch.int32, device=device),
                torch.empty(n_decoders + 1, dtype=torch.int32, device=device),
                torch.empty(max(cap, 1), dtype=torch.int32, device=device),
                torch.empty(ws, dtype=torch.uint8, device=device), align)


def build_bins(tex_id: torch.Tensor, tex_to_dec: torch.Tensor, n_decoders: int, align: int = 64,
               n_textures: Optional[int] = None, bins: Optional[Bins] = None,
               stream=None) -> Bins:
    n = int(tex_id.numel())
    T = int(tex_to_dec.numel()) if n_textures is None else int(n_textures)
    if bins is None:
        bins = alloc_bins(n, n_decoders, align, tex_id.device)
    _check("ntc_build_bins", lib().ntc_build_bins(
        _ptr(tex_id), n, _ptr(tex_to_dec), T, n_decoders, align, _ptr(bins.bin_count),
        _ptr(bins.bin_offset), _ptr(bins.perm), bins.capacity, _ptr(bins.workspace),
        int(bins.workspace.numel()), _stream(stream)))
    return bins


NOALLOC_SCRATCH_BYTES = 5 << 20  # NTC_NOALLOC_SCRATCH_BYTES


def build_bins_noalloc(tex_id: torch.Tensor, tex_to_dec: torch.Tensor, n_decoders: int,
                       bin_count: torch.Tensor, bin_offset: torch.Tensor, perm: torch.Tensor,
                       align: int = 64, n_textures: Optional[int] = None,
                       n_invalid: Optional[torch.Tensor] = None, stream=None) -> None:
    """ntc_build_bins_noalloc: binning into caller-owned outputs with the library's
    own device scratch (no workspace); n_invalid (one int32 on the device, or
    None) receives the count of queries left out of every bin."""
    n = int(tex_id.numel())
    T = int(tex_to_dec.numel()) if n_textures is None else int(n_textures)
    _check("ntc_build_bins_noalloc", lib().ntc_build_bins_noalloc(
        _ptr(tex_id), n, _ptr(tex_to_dec), T, n_decoders, align, _ptr(bin_count),
        _ptr(bin_offset), _ptr(perm), int(perm.numel()), _ptr(n_invalid), _stream(stream)))


def device_error(bins: Bins, stream=None) -> int:
    """Synchronises; returns the number of queries left out of every bin."""
    v = ctypes.c_uint64(0)
    st = lib().ntc_get_device_error(_ptr(bins.workspace), ctypes.byref(v), _stream(stream))
    if st not in (NTC_OK, NTC_ERR_INDEX):
        raise NtcError("ntc_get_device_error", st)
    return int(v.value)


# ----------------------------------------------------------------------------- decode


@dataclass
class DeviceModel:
    """Latent grids, decoders and the texture -> decoder map, resident on the device."""

    n_textures: int
    res: list
    channels: list
    latents: torch.Tensor      # int16 view of fp16 bits
    n_decoders: int
    dims: list
    params: torch.Tensor       # int16 view of fp16 bits
    tex_to_dec: torch.Tensor   # int32 view of uint32
    pe_octaves: int = 0        # positional-encoding octaves of the decoder input

    def grids(self) -> Grids:
        g = Grids()
        g.n_textures = self.n_textures
        g.n_levels = len(self.res)
        for i, (r, c) in enumerate(zip(self.res, self.channels)):
            g.res[i] = r
            g.channels[i] = c
        g.latents = _ptr(self.latents)
        return g

    def decoders(self) -> Decoders:
        d = Decoders()
        d.n_decoders = self.n_decoders
        d.n_layers = len(self.dims) - 1
        for i, v in enumerate(self.dims):
            d.dims[i] = v
        d.params = _ptr(self.params)
        return d

    @property
    def out_dim(self) -> int:
        return int(self.dims[-1])


@dataclass
class DeviceQueries:
    tex_id: torch.Tensor          # int32 view of uint32 [n]
    uv: torch.Tensor              # float32 [n, 2]
    mip: Optional[torch.Tensor]   # float32 [n] or None

    @property
    def n(self) -> int:
        return int(self.tex_id.numel())

    def struct(self) -> Queries:
        q = Queries()
        q.tex_id = _ptr(self.tex_id)
        q.uv = _ptr(self.uv)
        q.mip = _ptr(self.mip)
        q.n = self.n
        return q


def _dev(a: np.ndarray, dtype, device) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a).view(dtype)).to(device)


def upload(w, device="cuda"):
    """Host workload (paper_2608_27888_amd.workloads.Workload) -> (DeviceModel, DeviceQueries)."""
    model = DeviceModel(w.n_textures, list(w.res), list(w.channels),
                        _dev(w.latents, np.int16, device), w.n_decoders, list(w.dims),
                        _dev(w.params, np.int16, device), _dev(w.tex_to_dec, np.int32, device),
                        int(getattr(w, "pe_octaves", 0)))
    queries = DeviceQueries(_dev(w.tex_id, np.int32, device), _dev(w.uv, np.float32, device),
                            None if w.mip is None else _dev(w.mip, np.float32, device))
    return model, queries


NTC_ACT_RELU, NTC_ACT_LEAKY_RELU = 0, 1
NTC_OUT_F32, NTC_OUT_F16 = 0, 1
NTC_ENGINE_MFMA, NTC_ENGINE_FMA, NTC_ENGINE_FMA_DIRECT = 0, 1, 2
ENGINES = {"mfma": NTC_ENGINE_MFMA, "fma": NTC_ENGINE_FMA, "fma_direct": NTC_ENGINE_FMA_DIRECT}
NTC_GATHER_DIRECT, NTC_GATHER_STAGED = 0, 1
GATHERS = {"direct": NTC_GATHER_DIRECT, "staged": NTC_GATHER_STAGED}


class DecodeOptions(ctypes.Structure):
    _fields_ = [("hidden_activation", ctypes.c_int32), ("leaky_slope", ctypes.c_float),
                ("output_format", ctypes.c_int32), ("pe_octaves", ctypes.c_int32),
                ("engine", ctypes.c_int32), ("gather", ctypes.c_int32)]


def decode(model: DeviceModel, queries: DeviceQueries, bins: Optional[Bins] = None,
           out: Optional[torch.Tensor] = None, stream=None, leaky_slope: Optional[float] = None,
           out_dtype: torch.dtype = torch.float32, engine: str = "mfma",
           gather: str = "direct") -> torch.Tensor:
    """Binned mode when `bins` is given, stream (divergent) mode otherwise.  Hidden
    activation ReLU, or LeakyReLU max(x, slope x) when leaky_slope is given; output
    rows float32 or float16; the model's positional-encoding octaves extend the
    decoder input.  engine "mfma" (tensor path), "fma" (per-lane vector FMA with
    the LDS decoder cache) or "fma_direct" (per-lane vector FMA, weights through
    the caches); the FMA engines take stream mode only.  gather "direct" or "staged" (taps staged in LDS, binned
    MFMA decode only)."""
    if engine not in ENGINES:
        raise ValueError("engine must be 'mfma', 'fma' or 'fma_direct'")
    if gather not in GATHERS:
        raise ValueError("gather must be 'direct' or 'staged'")
    if out_dtype not in (torch.float32, torch.float16):
        raise ValueError("out_dtype must be float32 or float16")
    if out is None:
        out = torch.empty((queries.n, model.out_dim), dtype=out_dtype,
                          device=queries.tex_id.device)
    elif out.dtype != out_dtype:
        raise ValueError("out has the wrong dtype")
    g, d, q = model.grids(), model.decoders(), queries.struct()
    opt = DecodeOptions(NTC_ACT_RELU if leaky_slope is None else NTC_ACT_LEAKY_RELU,
                        0.0 if leaky_slope is None else float(leaky_slope),
                        NTC_OUT_F16 if out_dtype == torch.float16 else NTC_OUT_F32,
                        int(model.pe_octaves), ENGINES[engine], GATHERS[gather])
    if bins is not None:
        st = lib().ntc_decode_ex(ctypes.byref(g), ctypes.byref(d), _ptr(model.tex_to_dec),
                                 ctypes.byref(q), _ptr(bins.bin_offset), _ptr(bins.perm),
                                 bins.capacity, bins.align, ctypes.byref(opt), _ptr(out),
                                 _stream(stream))
    else:
        st = lib().ntc_decode_ex(ctypes.byref(g), ctypes.byref(d), _ptr(model.tex_to_dec),
                                 ctypes.byref(q), None, None, 0, 0, ctypes.byref(opt), _ptr(out),
                                 _stream(stream))
    _check("ntc_decode_ex", st)
    return out


def gather_features(model: DeviceModel, queries: DeviceQueries, out: Optional[torch.Tensor] = None,
                    out_dtype: torch.dtype = torch.float32, stream=None) -> torch.Tensor:
    """ntc_gather_features: the feature vector of every query (the decode's gather
    step without the MLP), rows [n][n_levels * channels] of float32 or float16."""
    if out_dtype not in (torch.float32, torch.float16):
        raise ValueError("out_dtype must be float32 or float16")
    F = sum(model.channels)
    if out is None:
        out = torch.empty((queries.n, F), dtype=out_dtype, device=queries.tex_id.device)
    elif out.dtype != out_dtype:
        raise ValueError("out has the wrong dtype")
    g, q = model.grids(), queries.struct()
    _check("ntc_gather_features", lib().ntc_gather_features(
        ctypes.byref(g), ctypes.byref(q), _ptr(out),
        NTC_OUT_F16 if out_dtype == torch.float16 else NTC_OUT_F32, _stream(stream)))
    return out


# ----------------------------------------------------------------------------- divergence


def divergence_stats(tex_id: torch.Tensor, tex_to_dec: torch.Tensor, n_decoders: int,
                     order: Optional[torch.Tensor] = None, wave: int = 64,
                     n_textures: Optional[int] = None, stream=None):
    """-> (per_wave_distinct int32 tensor, totals int64 tensor [4])."""
    n = int(tex_id.numel())
    T = int(tex_to_dec.numel()) if n_textures is None else int(n_textures)
    ln = n if order is None else int(order.numel())
    per = torch.empty(max(1, (ln + wave - 1) // wave), dtype=torch.int32, device=tex_id.device)
    tot = torch.empty(4, dtype=torch.int64, device=tex_id.device)
    _check("ntc_divergence_stats", lib().ntc_divergence_stats(
        _ptr(tex_id), n, _ptr(tex_to_dec), T, n_decoders, _ptr(order), ln, wave, _ptr(per),
        _ptr(tot), _stream(stream)))
    return per[: (ln + wave - 1) // wave], tot


def divergence_map(tex_id: torch.Tensor, width: int, height: int, tex_to_dec: torch.Tensor,
                   n_decoders: int, spp: int = 1, block_w: int = 8, block_h: int = 8,
                   hist_len: int = 65, n_textures: Optional[int] = None, stream=None):
    """Distinct decoders per screen block -> (map int32 [Hb, Wb], histogram int32
    [hist_len], totals int64 [4])."""
    T = int(tex_to_dec.numel()) if n_textures is None else int(n_textures)
    if int(tex_id.numel()) != width * height * spp:
        raise ValueError("tex_id must hold width * height * spp queries")
    bx, by = (width + block_w - 1) // block_w, (height + block_h - 1) // block_h
    dmap = torch.empty((by, bx), dtype=torch.int32, device=tex_id.device)
    hist = torch.empty(hist_len, dtype=torch.int32, device=tex_id.device)
    tot = torch.empty(4, dtype=torch.int64, device=tex_id.device)
    _check("ntc_divergence_map", lib().ntc_divergence_map(
        _ptr(tex_id), width, height, spp, _ptr(tex_to_dec), T, n_decoders, block_w, block_h,
        _ptr(dmap), _ptr(hist), hist_len, _ptr(tot), _stream(stream)))
    return dmap, hist, tot


# ----------------------------------------------------------------------------- clustering


@dataclass
class Clusters:
    assign: torch.Tensor     # int32 [n]: c(i), the texture -> decoder map
    centroids: torch.Tensor  # float64 [m][dim]
    counts: torch.Tensor     # int32 [m]: k_g
    iterations: int
    converged: bool


def kmeans(features: torch.Tensor, init, max_iter: int = 100, stream=None) -> Clusters:
    """k-means of per-texture feature vectors (float32 [n][dim] on the device) into
    m = len(init) groups seeded by the textures `init` (host integers); the labels
    are a texture -> decoder map.  Synchronises to read the iteration count."""
    if features.dtype != torch.float32 or features.dim() != 2 or not features.is_contiguous():
        raise ValueError("features must be a contiguous float32 [n][dim] tensor")
    n, dim = features.shape
    seeds = np.ascontiguousarray(np.asarray(init, dtype=np.uint32))
    m = int(seeds.size)
    dev = features.device
    assign = torch.empty(n, dtype=torch.int32, device=dev)
    centroids = torch.empty((m, dim), dtype=torch.float64, device=dev)
    counts = torch.empty(m, dtype=torch.int32, device=dev)
    wsb = lib().ntc_kmeans_workspace_bytes(m, int(max_iter))
    ws = torch.empty(max(wsb, 4), dtype=torch.uint8, device=dev)
    st = lib().ntc_kmeans(_ptr(features), n, dim, m, seeds.ctypes.data_as(ctypes.c_void_p),
                          int(max_iter), _ptr(assign), _ptr(centroids), _ptr(counts), _ptr(ws),
                          wsb, _stream(stream))
    _check("ntc_kmeans", st)
    it, conv = ctypes.c_int32(0), ctypes.c_int32(0)
    _check("ntc_kmeans_result", lib().ntc_kmeans_result(_ptr(ws), m, int(max_iter), ctypes.byref(it),
                                                        ctypes.byref(conv), _stream(stream)))
    return Clusters(assign, centroids, counts, int(it.value), bool(conv.value))


def freeze_scale(epoch: float, freeze_start: Optional[float], freeze_duration: float) -> float:
    """Gradual decoder-freezing factor lambda(epoch); freeze_start None = never."""
    start = float("nan") if freeze_start is None else float(freeze_start)
    return float(lib().ntc_freeze_scale(float(epoch), start, float(freeze_duration)))
