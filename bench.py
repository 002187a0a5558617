"""Throughput of neural texture decode with per-wave decoder binning on one MI355X.

One step = one pass of the hot path over one frame of queries, inputs resident
in HBM: ntc_build_bins (histogram, scan, stable scatter) followed by the binned
ntc_decode (gather + MFMA MLP + sigmoid + store).  Default workload: the 4K
clustered frame (3840x2160 queries, 512 textures, 16 Zipf-sized decoder
clusters, Voronoi material map).

Prints one JSON line.  Besides the headline it reports the decode kernel's
roofline position (HIP events over the timed region), the CPU oracle timed on a
bounded sample of the same frame, mean decoders per wave in stream and binned
order, and (unless --no-compare) the divergent-vs-clustered 2x2: {512
per-texture decoders, 16 clusters} x {stream order, binned}.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0       # MI355X HBM3E, GB/s
MFMA_F16_PEAK_TFLOPS = 2500.0  # MI355X dense fp16 MFMA, TFLOP/s


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    # the clocks are settled before the warm-up (--settle-ms), so a few warm-up
    # steps suffice
    p.add_argument("--steps", type=int, default=100)
    p.add_argument("--warmup", type=int, default=10)
    p.add_argument("--workload", default="clustered4k",
                   choices=["clustered4k", "single", "divergent", "wide_trilinear"])
    p.add_argument("--seed", type=int, default=0)
    p.add_argument("--no-compare", action="store_true",
                   help="skip the stream/binned x 16/512-decoder comparison runs")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-sample", type=int, default=1 << 20,
                   help="queries of the frame the CPU oracle decodes")
    p.add_argument("--settle-ms", type=float, default=400.0,
                   help="untimed steps run for this much wall time before the warm-up, so the "
                        "GPU clocks reach their steady state whatever --warmup is")
    p.add_argument("--cache-dir", default=os.environ.get("NTC_INPUT_CACHE", ""),
                   help="directory of the seeded inputs saved as .npy (drawn once, then read)")
    p.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                   help="first run a plain device-to-device copy of this many MiB three times, "
                        "so that a counter profile of this run also holds the copy's HBM bytes")
    return p.parse_args()


def unique_latent_bytes(w) -> int:
    """Bytes of distinct latent texels a frame touches (bilinear taps, mip 0 only)."""
    if w.mip is not None:
        return 0  # not counted for blended levels
    total = 0
    u = w.uv[:, 0].astype(np.float32)
    v = w.uv[:, 1].astype(np.float32)
    tex = w.tex_id.astype(np.int64)
    for l, (r, c) in enumerate(zip(w.res, w.channels)):
        x0 = np.floor(u * np.float32(r) - np.float32(0.5)).astype(np.int64)
        y0 = np.floor(v * np.float32(r) - np.float32(0.5)).astype(np.int64)
        keys = []
        for dx in (0, 1):
            for dy in (0, 1):
                xx = np.clip(x0 + dx, 0, r - 1)
                yy = np.clip(y0 + dy, 0, r - 1)
                keys.append((tex * r + yy) * r + xx)
        total += np.unique(np.concatenate(keys)).size * c * 2
    return int(total)


TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "decode_binned_clustered4k_hbm_traffic.md")
DECODE_SOURCES = [os.path.join(ROOT, "paper_2608_27888_amd", "csrc", f)
                  for f in ("ntc_decode_kernels.h", "ntc_decode_launch.h", "ntc_decode_l2c16.hip")]


def decode_source_hash() -> str:
    import hashlib

    h = hashlib.sha256()
    for f in DECODE_SOURCES:
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


COUNTER_PROFILE = os.path.join(ROOT, "profiles", "decode_binned_clustered4k_sq_counters.md")


def profile_fields(path: str, workload: str):
    """The "- key: value" fields of a committed counter profile, or None when the
    profile covers another workload or the decode sources changed since it was taken."""
    try:
        with open(path) as fh:
            fields = dict(line[2:].split(":", 1) for line in fh if line.startswith("- ") and ":" in line)
    except OSError:
        return None
    fields = {k.strip(): v.strip().strip("`") for k, v in fields.items()}
    if fields.get("workload") != workload or fields.get("decode_source_sha256") != decode_source_hash():
        return None
    return fields


def profiled_traffic(workload: str):
    """HBM bytes per decode launch from the committed counter profile (FETCH_SIZE and
    WRITE_SIZE scaled by a device copy's), or None when it does not apply."""
    fields = profile_fields(TRAFFIC_PROFILE, workload)
    try:
        return int(fields["traffic_bytes_per_launch"]) if fields else None
    except (KeyError, ValueError):
        return None


def profiled_mfma_busy(workload: str):
    """MFMA busy cycles over SIMD-cycles (%) of the decode from the committed SQ counter
    profile, or None when it does not apply."""
    fields = profile_fields(COUNTER_PROFILE, workload)
    try:
        return float(fields["mfma_busy_pct"]) if fields else None
    except (KeyError, ValueError):
        return None


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, args, W):
    """The CPU oracle (float64 C, OpenMP over queries) timed on this host: the
    median of three runs over a bounded sample of the frame (binning of the whole
    frame scaled to the sample), plus one single-thread run of the tiny
    configuration for context."""
    from oracle import oracle as O

    threads = O.default_threads()
    n = w.n
    m = min(n, args.cpu_sample)
    sub = np.unique(np.linspace(0, n - 1, m).round().astype(np.int64))  # spread over the frame
    runs = []
    for _ in range(3):
        tb = time.perf_counter()
        O.build_bins(w.tex_id, w.tex_to_dec, w.n_decoders, 64)
        tb = time.perf_counter() - tb
        td = time.perf_counter()
        O.decode(w, subset=sub, threads=threads)
        td = time.perf_counter() - td
        runs.append(td + tb * sub.size / n)
    t_sample = float(np.median(runs))
    tiny = W.tiny(args.seed)
    t1 = time.perf_counter()
    O.build_bins(tiny.tex_id, tiny.tex_to_dec, tiny.n_decoders, 64)
    O.decode(tiny, threads=1)
    t1 = time.perf_counter() - t1
    return {
        "value": round(sub.size / t_sample / 1e9, 6), "unit": "Gtexel/s", "cores": threads,
        "kind": "oracle", "cpu": cpu_model(),
        "runs_s": [round(r, 3) for r in runs],
        "sample": f"{sub.size} queries evenly spaced over the frame decoded in float64, plus "
                  f"binning of the whole frame scaled to the sample; median of 3 runs "
                  f"({t_sample:.2f} s)",
        "tiny_single_thread": {"queries": tiny.n, "s": round(t1, 3),
                               "gtexel_s": round(tiny.n / t1 / 1e9, 6)},
    }


def timed(fn, steps, warmup, torch):
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        fn()
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) / steps


def event_ms(fn, reps, warmup, stream, torch, pre=None, settle_ms=0.0):
    """Mean kernel time of fn in ms: HIP events recorded on `stream` around each of
    `reps` calls, after at least `warmup` untimed calls and `settle_ms` of wall
    time spent in them (the clocks ramp down while the GPU idles and need some
    milliseconds of load to come back).  pre (untimed) runs on the same stream
    before each call, as the binning runs before the headline's decode: the host
    enqueues the timed call while the GPU is still busy, so the events do not take
    in the host's own time per call."""
    t0, done = time.perf_counter(), 0
    while done < warmup or (time.perf_counter() - t0) * 1e3 < settle_ms:
        if pre:
            pre()
        fn()
        done += 1
        if done % 10 == 0:
            torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(reps)]
    for a, b in ev:
        if pre:
            pre()
        a.record(stream)
        fn()
        b.record(stream)
    torch.cuda.synchronize()
    return float(np.mean([a.elapsed_time(b) for a, b in ev]))


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(on several GPUs each would decode its own screen slab, with no exchange between them)",
              file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_2608_27888_amd import ntc
    from paper_2608_27888_amd import workloads as W
    from paper_2608_27888_amd.report import divergence_metric, paper_speedup_percent

    dev = torch.device("cuda:0")
    ntc.lib()
    t0 = time.time()
    w = W.cached(args.workload, seed=args.seed, cache_dir=args.cache_dir)
    log(f"[bench] workload {w.name}: n={w.n} T={w.n_textures} D={w.n_decoders} dims={w.dims} "
        f"levels={w.res}x{w.channels} ({time.time() - t0:.1f} s to draw)")
    model, q = ntc.upload(w, dev)
    n = w.n
    bins = ntc.alloc_bins(n, w.n_decoders, 64, dev)
    out = torch.empty((n, w.out_dim), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()

    if args.copy_calibration > 0:  # reference kernel of known size for HBM byte counters
        src = torch.ones(args.copy_calibration << 18, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        log(f"[bench] copied {args.copy_calibration} MiB three times for counter calibration")
        del src, dst

    # ---------------------------------------------------------------- headline
    # one event pair per timed step, made before the timed region
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]

    def step(i=None):
        ntc.build_bins(q.tex_id, model.tex_to_dec, w.n_decoders, bins=bins, stream=stream)
        if i is not None:
            ev[i][0].record(stream)
        ntc.decode(model, q, bins, out=out, stream=stream)
        if i is not None:
            ev[i][1].record(stream)

    # Clock settling: the GPU needs several milliseconds of sustained load before
    # its clocks stop ramping; untimed steps for a fixed wall time, then the
    # warm-up steps, then the timed region.
    settle_steps = 0
    t_settle = time.perf_counter()
    while (time.perf_counter() - t_settle) * 1e3 < args.settle_ms:
        for _ in range(10):
            step()
        settle_steps += 10
        torch.cuda.synchronize()
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for i in range(args.steps):
        step(i)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    ms_step = wall * 1e3 / args.steps
    decode_ms = float(np.mean([a.elapsed_time(b) for a, b in ev]))
    log(f"[bench] {settle_steps} settling steps, then step {ms_step:.4f} ms, "
        f"decode kernel {decode_ms:.4f} ms")
    assert ntc.device_error(bins) == 0

    # bins alone, for the breakdown
    bins_ms = timed(lambda: ntc.build_bins(q.tex_id, model.tex_to_dec, w.n_decoders, bins=bins,
                                           stream=stream), args.steps, args.warmup, torch) * 1e3

    # ---------------------------------------------------------------- roofline
    flops_q = w.flops_per_query()
    stream_bytes_q = 4 + 4 + 8 + 4 * w.out_dim + (4 if w.mip is not None else 0)
    lat_bytes = unique_latent_bytes(w)
    used = np.unique(w.tex_to_dec[w.tex_id])
    param_bytes = int(used.size * w.decoder_stride * 2)
    decode_bytes = n * stream_bytes_q + lat_bytes + param_bytes
    decode_flops = n * flops_q
    t_hbm = decode_bytes / (HBM_PEAK_GBS * 1e9)
    t_mfma = decode_flops / (MFMA_F16_PEAK_TFLOPS * 1e12)
    dsec = decode_ms * 1e-3
    if t_hbm >= t_mfma:
        roof = {"bound": "hbm", "achieved": round(decode_bytes / dsec / 1e9, 1),
                "peak": HBM_PEAK_GBS, "unit": "GB/s"}
    else:
        roof = {"bound": "mfma", "achieved": round(decode_flops / dsec / 1e12, 1),
                "peak": MFMA_F16_PEAK_TFLOPS, "unit": "TFLOP/s"}
    roof["frac"] = round(roof["achieved"] / roof["peak"], 4)
    roof["traffic"] = profiled_traffic(w.name)
    roof["mfma_busy_pct_counters"] = profiled_mfma_busy(w.name)
    roof["kernel"] = "decode_binned"
    roof["algorithmic_bytes_per_launch"] = int(decode_bytes)
    roof["algorithmic_flops_per_launch"] = int(decode_flops)
    # end-to-end: binning adds 12 B per query (read ids twice, write the permutation)
    e2e_bytes = decode_bytes + 12 * n
    e2e_roof_ms = max(e2e_bytes / (HBM_PEAK_GBS * 1e9), t_mfma) * 1e3

    # ---------------------------------------------------------------- decoder variants
    # The Sec. 4 setup's decoder (LeakyReLU, positional encoding, RGB rows) and
    # its parts, on the same frame and bins: binned decode kernel time of each
    # (HIP events on the decode stream, as for the headline's decode_ms).
    variants = None
    if not args.no_compare and w.mip is None:
        # right after the headline (clocks settled), each with its own warm-up
        reps = max(10, args.steps // 2)
        variants = {}
        for tag, ww, slope, dt in (
                ("relu_f32x8", w, None, torch.float32),
                ("leaky_f32x8", w, 0.01, torch.float32),
                ("pe4_f32x8", w.with_pe(4, seed=args.seed), None, torch.float32),
                ("f16x8", w, None, torch.float16),
                ("sec4_setup_pe4_leaky_f16x3", w.with_pe(4, [0, 64, 64, 3], seed=args.seed), 0.01,
                 torch.float16)):
            # same latents, map and queries on the device; only the decoders differ
            mv = model if ww is w else ntc.DeviceModel(
                model.n_textures, model.res, model.channels, model.latents, ww.n_decoders,
                list(ww.dims), torch.from_numpy(ww.params.view(np.int16)).to(dev),
                model.tex_to_dec, ww.pe_octaves)
            ov = torch.empty((n, ww.out_dim), dtype=dt, device=dev)
            variants[tag] = round(event_ms(
                lambda: ntc.decode(mv, q, bins, out=ov, stream=stream, leaky_slope=slope,
                                   out_dtype=dt), reps, reps, stream, torch,
                pre=lambda: ntc.build_bins(q.tex_id, model.tex_to_dec, w.n_decoders, bins=bins,
                                           stream=stream), settle_ms=args.settle_ms / 4), 4)
            del ov
        log(f"[bench] decode variants {variants}")

    # ---------------------------------------------------------------- divergence
    per_s, tot_s = ntc.divergence_stats(q.tex_id, model.tex_to_dec, w.n_decoders)
    P = int(bins.bin_offset[-1].item())
    per_b, tot_b = ntc.divergence_stats(q.tex_id, model.tex_to_dec, w.n_decoders,
                                        order=bins.perm[:P])
    tot_s, tot_b = tot_s.cpu().tolist(), tot_b.cpu().tolist()

    result = {
        "metric": "decoded texels/sec (Gtexel/s) on 1 MI355X; MFMA util %; mean decoders/wave",
        "value": round(n / (ms_step * 1e-3) / 1e9, 3),
        "unit": "Gtexel/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic",
        "config": {"workload": w.name, "queries": n, "screen": list(w.screen or []),
                   "textures": w.n_textures, "decoders": w.n_decoders, "mlp": list(w.dims),
                   "latent_levels": [[r, r, c] for r, c in zip(w.res, w.channels)],
                   "parallelism": "single GPU", "step": "build_bins + binned decode"},
        "decode_only_gtexel_s": round(n / dsec / 1e9, 3),
        "decode_ms": round(decode_ms, 5),
        "build_bins_ms": round(bins_ms, 5),
        "mfma_util_pct": round(100.0 * decode_flops / dsec / (MFMA_F16_PEAK_TFLOPS * 1e12), 2),
        "roofline": roof,
        "end_to_end_roofline_frac": round(e2e_roof_ms / ms_step, 4),
        "mean_decoders_per_wave": {"stream": round(tot_s[1] / max(tot_s[0], 1), 4),
                                   "binned": round(tot_b[1] / max(tot_b[0], 1), 4),
                                   "divergence_metric_stream": round(divergence_metric(tot_s), 4),
                                   "divergence_metric_binned": round(divergence_metric(tot_b), 4)},
    }

    if variants:
        result["decode_variants_ms"] = variants

    # ---------------------------------------------------------------- divergence map (Sec. 2)
    if w.screen is not None:
        W_, H_, spp = w.screen
        ident = torch.arange(w.n_textures, dtype=torch.int32, device=dev)
        maps = {}
        for tag, t2d, D in ((f"d{w.n_decoders}", model.tex_to_dec, w.n_decoders),
                            (f"d{w.n_textures}_per_texture", ident, w.n_textures)):
            _, hist, tot = ntc.divergence_map(q.tex_id, W_, H_, t2d, D, spp=spp, block_w=8,
                                              block_h=8, hist_len=17)
            tot = tot.cpu().tolist()
            maps[tag] = {"metric": round(divergence_metric(tot), 4),
                         "divergent_blocks_pct": round(100.0 * tot[2] / max(tot[0], 1), 2),
                         "max": int(tot[3]), "histogram": hist.cpu().tolist()}
        result["divergence_map_8x8"] = maps

    # ---------------------------------------------------------------- 2x2 comparison
    if not args.no_compare and w.name.startswith(("clustered4k", "wide_trilinear")):
        T = w.n_textures
        w512 = w.with_decoders(T, np.arange(T, dtype=np.uint32), seed=args.seed)
        m512, _ = ntc.upload(w512, dev)
        bins512 = ntc.alloc_bins(n, T, 64, dev)
        reps = max(3, args.steps // 4)

        def run(m, D, b, binned):
            def f():
                if binned:
                    ntc.build_bins(q.tex_id, m.tex_to_dec, D, bins=b, stream=stream)
                    ntc.decode(m, q, b, out=out, stream=stream)
                else:
                    ntc.decode(m, q, None, out=out, stream=stream)
            return timed(f, reps, max(2, reps // 2), torch) * 1e3

        t = {f"d{w.n_decoders}_binned": ms_step,
             f"d{w.n_decoders}_stream": run(model, w.n_decoders, bins, False),
             f"d{T}_binned": run(m512, T, bins512, True),
             f"d{T}_stream": run(m512, T, bins512, False)}
        _, ts512 = ntc.divergence_stats(q.tex_id, m512.tex_to_dec, T)
        ts512 = ts512.cpu().tolist()
        result["compare_ms"] = {k: round(v, 4) for k, v in t.items()}
        result["compare_decoders_per_wave_stream"] = {
            f"d{w.n_decoders}": result["mean_decoders_per_wave"]["stream"],
            f"d{T}": round(ts512[1] / max(ts512[0], 1), 4)}
        result["speedup_divergent_vs_clustered_binned"] = round(t[f"d{T}_stream"] / ms_step, 3)
        result["speedup_paper_percent_form"] = round(
            paper_speedup_percent([ms_step], [t[f"d{T}_stream"]]), 2)
        result["paper_context"] = ("paper: up to 8.48x (848.49 %) shared vs non-shared WMMA, "
                                   "10 decoders per wave, RX 9070 XT at 1.6 GHz")
        log(f"[bench] compare {result['compare_ms']}")
    elif not args.no_compare:
        # one decoder set only (Divergent: one decoder per texture; Single: one
        # decoder): stream order against the binned step
        reps = max(3, args.steps // 4)
        t_stream = timed(lambda: ntc.decode(model, q, None, out=out, stream=stream), reps,
                         max(2, reps // 2), torch) * 1e3
        result["compare_ms"] = {f"d{w.n_decoders}_binned": round(ms_step, 4),
                                f"d{w.n_decoders}_stream": round(t_stream, 4)}
        result["speedup_stream_vs_binned"] = round(t_stream / ms_step, 3)
        log(f"[bench] compare {result['compare_ms']}")

    # ---------------------------------------------------------------- CPU oracle
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(w, args, W)
        log(f"[bench] cpu oracle {result['cpu_baseline']}")

    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
