"""The paper's decoder-divergence timing study (Sec. 4.4, Tables performance_5dec and
performance_10dec) re-run on one MI355X with this library's kernels.

For an output image of side^2 queries whose 64-query waves each hold k decoders
spread uniformly over the lanes, it times
  shared     : k = 1, every wave runs one decoder (the paper's Shared-Decoder);
  non_shared : k decoders per wave in stream order, each wave running one MFMA
               MLP pass per decoder present (the paper's Non-Shared WMMA column);
  fma        : the same stream on the per-lane vector-FMA engine, every lane
               evaluating its own decoder (the paper's Non-Shared FMA column),
               its weights read from a per-CU LDS cache of whole decoders;
  fma_direct : the same engine with every lane loading its weight rows through
               the L1/L2 caches;
  binned     : the same k-decoder stream binned by decoder id first
               (ntc_build_bins + binned ntc_decode), so each wave runs one pass.
Times are HIP-event medians of one launch sequence, in microseconds; inputs are
resident in HBM.  The summary repeats the paper's "average speedup" form,
mean over sizes of (T_non_shared / T_shared - 1) x 100.

    python -m paper_2608_27888_amd.microbench [--sides 512 1024 2048 4096 8192] [--ks 5 10]
"""
from __future__ import annotations

import argparse
import json
import sys

import numpy as np


def median_us(fn, torch, reps=7, warmup=2):
    for _ in range(warmup):
        fn()
    ts = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        fn()
        e1.record()
        e1.synchronize()
        ts.append(e0.elapsed_time(e1) * 1e3)
    return float(np.median(ts))


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--sides", type=int, nargs="+", default=[512, 1024, 2048, 4096, 8192])
    ap.add_argument("--ks", type=int, nargs="+", default=[5, 10])
    args = ap.parse_args(argv)
    import torch

    from paper_2608_27888_amd import ntc
    from paper_2608_27888_amd import workloads as W
    from paper_2608_27888_amd.report import paper_speedup_percent

    dev = torch.device("cuda:0")
    ntc.lib()
    rows = []
    for side in args.sides:
        row = {"side": side, "queries": side * side}
        for k in [1] + list(args.ks):
            w = W.k_per_wave(0, side, k)
            model, q = ntc.upload(w, dev)
            out = torch.empty((w.n, w.out_dim), dtype=torch.float32, device=dev)
            bins = ntc.alloc_bins(w.n, w.n_decoders, 64, dev)
            per, tot = ntc.divergence_stats(q.tex_id, model.tex_to_dec, w.n_decoders)
            assert int(tot[3]) == k and int(tot[1]) == k * int(tot[0])

            def stream():
                ntc.decode(model, q, None, out=out)

            def binned():
                ntc.build_bins(q.tex_id, model.tex_to_dec, w.n_decoders, bins=bins)
                ntc.decode(model, q, bins, out=out)

            def fma():
                ntc.decode(model, q, None, out=out, engine="fma")

            def fma_direct():
                ntc.decode(model, q, None, out=out, engine="fma_direct")

            row[f"k{k}_stream_us"] = round(median_us(stream, torch), 1)
            row[f"k{k}_binned_us"] = round(median_us(binned, torch), 1)
            row[f"k{k}_fma_us"] = round(median_us(fma, torch), 1)
            row[f"k{k}_fma_direct_us"] = round(median_us(fma_direct, torch, reps=3, warmup=1), 1)
            print(f"[microbench] side {side} k {k}: stream {row[f'k{k}_stream_us']} us, "
                  f"binned {row[f'k{k}_binned_us']} us, fma {row[f'k{k}_fma_us']} us, "
                  f"fma_direct {row[f'k{k}_fma_direct_us']} us", file=sys.stderr, flush=True)
            del model, q, out, bins
            torch.cuda.empty_cache()
        rows.append(row)
    summary = {}
    for k in args.ks:
        shared = [r["k1_stream_us"] for r in rows]
        summary[f"k{k}"] = {
            "non_shared_vs_shared_percent": round(
                paper_speedup_percent(shared, [r[f"k{k}_stream_us"] for r in rows]), 2),
            "non_shared_vs_binned_percent": round(
                paper_speedup_percent([r[f"k{k}_binned_us"] for r in rows],
                                      [r[f"k{k}_stream_us"] for r in rows]), 2),
            "non_shared_fma_vs_shared_percent": round(
                paper_speedup_percent(shared, [r[f"k{k}_fma_us"] for r in rows]), 2),
            "non_shared_fma_vs_binned_percent": round(
                paper_speedup_percent([r[f"k{k}_binned_us"] for r in rows],
                                      [r[f"k{k}_fma_us"] for r in rows]), 2),
            "non_shared_mfma_vs_fma_percent": round(
                paper_speedup_percent([r[f"k{k}_fma_us"] for r in rows],
                                      [r[f"k{k}_stream_us"] for r in rows]), 2)}
    print(json.dumps({"rows": rows, "summary": summary}), flush=True)


if __name__ == "__main__":
    main()
