"""ctypes wrapper of the CPU oracle library ``libntc_oracle.so``.

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg.  The product package never imports this module.
Each wrapper restates the definition it evaluates; the C source cites the
paper passages.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "ntc_oracle.c")
LIB = os.path.join(HERE, "libntc_oracle.so")
PAD = 0xFFFFFFFF


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (IEEE double, no contraction, OpenMP)."""
    if force or not os.path.exists(LIB):
        tmp = LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
                               "-ffp-contract=off", "-fno-fast-math", "-Wall", "-o", tmp, SRC,
                               "-lm"])
        os.replace(tmp, LIB)
    return LIB


_lib = None


def lib():
    """The oracle library; NTC_ORACLE_LIB names another build of the same source
    (the sanitizer test loads one built with AddressSanitizer and UBSan)."""
    global _lib
    if _lib is None:
        path = os.environ.get("NTC_ORACLE_LIB")
        if not path:
            if not os.path.exists(LIB):
                build(force=False)
            path = LIB
        L = ctypes.CDLL(path)
        P = ctypes.c_void_p
        i32, i64 = ctypes.c_int32, ctypes.c_int64
        L.ntc_oracle_build_bins.argtypes = [P, i64, P, i32, i32, i32, P, P, P, i64, P]
        L.ntc_oracle_divergence.argtypes = [P, i64, P, i32, i32, P, i64, i32, P, P]
        L.ntc_oracle_divergence_map.argtypes = [P, i32, i32, i32, P, i32, i32, i32, i32, P, P,
                                                i32, P]
        L.ntc_oracle_features.argtypes = [P, i32, i32, P, P, P, P, P, i64, P, i64, i32, i32, P]
        L.ntc_oracle_decode.argtypes = [P, i32, i32, P, P, P, i32, i32, P, P, P, P, P, i64, P,
                                        i64, i32, ctypes.c_double, i32, P]
        L.ntc_oracle_half_to_double.argtypes = [ctypes.c_uint16]
        L.ntc_oracle_half_to_double.restype = ctypes.c_double
        for f in ("ntc_oracle_build_bins", "ntc_oracle_divergence", "ntc_oracle_divergence_map",
                  "ntc_oracle_features", "ntc_oracle_decode"):
            getattr(L, f).restype = ctypes.c_int
        _lib = L
    return _lib


def _p(a):
    return None if a is None else ctypes.c_void_p(a.ctypes.data)


def _u32(a):
    return np.ascontiguousarray(a, dtype=np.uint32)


def default_threads() -> int:
    return len(os.sched_getaffinity(0))


class OracleError(RuntimeError):
    pass


def build_bins(tex_id, tex_to_dec, n_decoders, align=64, n_textures=None, capacity=None):
    """Stable counting sort of queries by decoder id -> (bin_count, bin_offset, perm, n_invalid).

    perm is trimmed to bin_offset[-1] entries.
    """
    tex_id, tex_to_dec = _u32(tex_id), _u32(tex_to_dec)
    n = tex_id.shape[0]
    T = tex_to_dec.shape[0] if n_textures is None else n_textures
    cap = n + n_decoders * (align - 1) if capacity is None else capacity
    cnt = np.zeros(n_decoders, np.uint32)
    off = np.zeros(n_decoders + 1, np.uint32)
    perm = np.zeros(max(cap, 1), np.uint32)
    bad = np.zeros(1, np.int64)
    rc = lib().ntc_oracle_build_bins(_p(tex_id), n, _p(tex_to_dec), T, n_decoders, align,
                                     _p(cnt), _p(off), _p(perm), cap, _p(bad))
    if rc != 0:
        raise OracleError("ntc_oracle_build_bins -> %d" % rc)
    return cnt, off, perm[: int(off[-1])].copy(), int(bad[0])


def divergence(tex_id, tex_to_dec, n_decoders, order=None, wave=64, n_textures=None):
    """Distinct decoder ids per window of `wave` entries -> (per_wave, totals[4])."""
    tex_id, tex_to_dec = _u32(tex_id), _u32(tex_to_dec)
    n = tex_id.shape[0]
    T = tex_to_dec.shape[0] if n_textures is None else n_textures
    if order is not None:
        order = _u32(order)
    ln = n if order is None else order.shape[0]
    per = np.zeros(max(1, (ln + wave - 1) // wave), np.uint32)
    tot = np.zeros(4, np.uint64)
    rc = lib().ntc_oracle_divergence(_p(tex_id), n, _p(tex_to_dec), T, n_decoders, _p(order), ln,
                                     wave, _p(per), _p(tot))
    if rc != 0:
        raise OracleError("ntc_oracle_divergence -> %d" % rc)
    return per[: (ln + wave - 1) // wave], tot


def divergence_map(tex_id, width, height, tex_to_dec, n_decoders, spp=1, block_w=8, block_h=8,
                   hist_len=65, n_textures=None):
    """Distinct decoder ids per screen block -> (map [Hb, Wb], histogram, totals[4])."""
    tex_id, tex_to_dec = _u32(tex_id), _u32(tex_to_dec)
    assert tex_id.shape[0] == width * height * spp
    T = tex_to_dec.shape[0] if n_textures is None else n_textures
    bx, by = (width + block_w - 1) // block_w, (height + block_h - 1) // block_h
    dmap = np.zeros((by, bx), np.uint32)
    hist = np.zeros(hist_len, np.uint32)
    tot = np.zeros(4, np.uint64)
    rc = lib().ntc_oracle_divergence_map(_p(tex_id), width, height, spp, _p(tex_to_dec), T,
                                         n_decoders, block_w, block_h, _p(dmap), _p(hist),
                                         hist_len, _p(tot))
    if rc != 0:
        raise OracleError("ntc_oracle_divergence_map -> %d" % rc)
    return dmap, hist, tot


def _grid_args(w):
    res = np.ascontiguousarray(w.res, dtype=np.int32)
    ch = np.ascontiguousarray(w.channels, dtype=np.int32)
    return res, ch


def features(w, subset=None, threads=None, fill=np.nan, pe_octaves=None):
    """Concatenated per-level latent samples of each query, followed by the
    positional encoding when pe_octaves (default: the workload's) is > 0
    (rows of invalid queries = fill)."""
    res, ch = _grid_args(w)
    K = int(getattr(w, "pe_octaves", 0) if pe_octaves is None else pe_octaves)
    F = int(sum(w.channels)) + 4 * K
    sub = None if subset is None else np.ascontiguousarray(subset, dtype=np.int64)
    n_sel = w.n if sub is None else sub.shape[0]
    out = np.full((n_sel, F), fill, np.float64)
    rc = lib().ntc_oracle_features(_p(w.latents), w.n_textures, w.n_levels, _p(res), _p(ch),
                                   _p(w.tex_id), _p(w.uv), _p(w.mip), w.n, _p(sub), n_sel,
                                   threads or default_threads(), K, _p(out))
    if rc != 0:
        raise OracleError("ntc_oracle_features -> %d" % rc)
    return out


def decode(w, subset=None, threads=None, fill=np.nan, leaky_slope=0.0):
    """Decoded channels of each query (rows of invalid queries = fill); hidden
    activation ReLU, or LeakyReLU with 0 < leaky_slope < 1; the decoder input
    carries the workload's positional-encoding octaves (w.pe_octaves)."""
    res, ch = _grid_args(w)
    dims = np.ascontiguousarray(w.dims, dtype=np.int32)
    sub = None if subset is None else np.ascontiguousarray(subset, dtype=np.int64)
    n_sel = w.n if sub is None else sub.shape[0]
    out = np.full((n_sel, w.out_dim), fill, np.float64)
    rc = lib().ntc_oracle_decode(_p(w.latents), w.n_textures, w.n_levels, _p(res), _p(ch),
                                 _p(w.params), w.n_decoders, w.n_layers, _p(dims),
                                 _p(w.tex_to_dec), _p(w.tex_id), _p(w.uv), _p(w.mip), w.n,
                                 _p(sub), n_sel, threads or default_threads(),
                                 float(leaky_slope), int(getattr(w, "pe_octaves", 0)), _p(out))
    if rc != 0:
        raise OracleError("ntc_oracle_decode -> %d" % rc)
    return out


def half_to_double(bits: int) -> float:
    return lib().ntc_oracle_half_to_double(bits)


# ----------------------------------------------------------------------------- clustering


def kmeans(features, init, max_iter=100, history=False):
    """Stage 2 of Alg. "Overall texture processing pipeline" (Sec. 3.3): k-means of
    the per-texture feature rows into m = len(init) groups, Lloyd's iteration in
    float64.  Centroid g starts at the features of texture init[g].  Each iteration
    labels every texture with its nearest centroid (squared Euclidean distance,
    the lowest index among equals); when no label changes (after the first
    iteration) it stops, otherwise each centroid moves to the mean of its
    textures, summed one texture after another in ascending index; a group left
    empty keeps its centroid.  Returns (labels, centroids, sizes k_g, iterations,
    converged) and, with history=True, the within-group sum of squared distances
    after each assignment."""
    x = np.asarray(features, dtype=np.float64)
    n, dim = x.shape
    seeds = [int(i) for i in init]
    m = len(seeds)
    c = x[seeds].copy()
    labels = np.full(n, -1, dtype=np.int64)
    inertia = []
    iterations, converged = max_iter, False
    for t in range(max_iter):
        # distances of every texture to every centroid, one texture at a time
        new = np.empty(n, dtype=np.int64)
        total = 0.0
        for i in range(n):
            d = ((x[i][None, :] - c) ** 2).sum(axis=1)
            new[i] = int(np.argmin(d))  # first minimum: lowest index among equals
            total += float(d[new[i]])
        inertia.append(total)
        changed = t == 0 or bool(np.any(new != labels))
        labels = new
        if not changed:
            iterations, converged = t + 1, True
            break
        for g in range(m):
            members = np.nonzero(labels == g)[0]
            if members.size == 0:
                continue
            acc = np.zeros(dim, dtype=np.float64)
            for i in members:  # ascending texture index
                acc = acc + x[i]
            c[g] = acc / members.size
    sizes = np.bincount(labels, minlength=m)
    out = (labels.astype(np.uint32), c, sizes.astype(np.uint32), iterations, converged)
    return out + (inertia,) if history else out


def freeze_scale(epoch, freeze_start, freeze_duration):
    """Gradual decoder freezing of Sec. 3.2 (Alg. SelfFreezeDecoderGradually): the
    decoder's update factor is 1 until the freezing epoch, 0 once the freezing
    window of freeze_duration epochs has passed, and in between follows half a
    cosine period from 1 down to 0 over the fraction of the window elapsed.
    freeze_start None means the decoder is never frozen."""
    import math

    if freeze_start is None or epoch < freeze_start:
        return 1.0
    if epoch >= freeze_start + freeze_duration:
        return 0.0
    elapsed = (epoch - freeze_start) / freeze_duration
    return 0.5 * (1.0 + math.cos(math.pi * elapsed))
