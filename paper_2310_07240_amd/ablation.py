"""Codec ablation in bits per element on one GPU (CacheGen Sec. 7.5 "Ablation Study", which
starts from uniform quantization with a default arithmetic coder and adds the encoder's ideas
one by one; Sec. 5.2 "Arithmetic coding", which compares per channel-layer distributions with
one global distribution).

Every configuration runs the codec's kernels through the C ABI on a resident synthetic cache:
fit (per (layer, K/V, channel), or pooled into one global distribution), encode, decode. It
reports the payload bits per element and the error of the decoded cache. The configurations:

  1. uniform quantization, one global distribution: every token quantized on its own at the
     8-bit vectorwise step s (group size 1), coded with one pooled table;
  2. + per-(layer, K/V, channel) distributions;
  3. + change-based encoding: groups of 10, deltas against the anchor at the same step
     (bin 1.0 s in every layer), so the error bound s/2 of configurations 1-2 is kept;
  4. + layer-wise quantization: the workload's per-layer bins (0.5 / 1 / 1.5 s by layer group),
     i.e. CacheGen's encoder;
  5. CacheGen's encoder with one global distribution instead of per channel-layer ones;
  6. CacheGen's encoder with per channel-layer distributions fitted on another context of the
     same model (the same generator with another seed): the paper profiles the distributions
     offline per model and reuses them for every context (Sec. 5.2), while its implementation
     counts them per context (Sec. 6).

Chunks are all coded at the first encoding level (multiplier level_mult[0]).

Usage: python -m paper_2310_07240_amd.ablation [--workload NAME ...]  (one JSON line each)
"""
from __future__ import annotations

import argparse
import dataclasses
import json
import sys

import numpy as np

LADDER = (
    ("uniform quantization, one global distribution", 1, "uniform", "global"),
    ("+ per-(layer, K/V, channel) distributions", 1, "uniform", "channel"),
    ("+ change-based encoding (anchor + delta)", 10, "uniform", "channel"),
    ("+ layer-wise quantization (CacheGen)", 10, "layer", "channel"),
    ("CacheGen with one global distribution", 10, "layer", "global"),
    ("CacheGen with distributions of another context", 10, "layer", "other"),
)


def run(w, device="cuda"):
    """Returns a list of dicts, one per configuration of LADDER, for workload `w`."""
    import torch
    from paper_2310_07240_amd import workloads as W
    from paper_2310_07240_amd.cachegen import (CG_FIT_GLOBAL_WORKSPACE_BYTES, Codec, CodecParams,
                                               cg_fit_cdf, cg_fit_cdf_global)
    kv_np = W.generate(w)
    kv = torch.from_numpy(kv_np.view(np.int16)).to(device)
    x = kv.view(torch.float16).float()
    x_rms = float(torch.sqrt(torch.mean(x * x)))
    out_rows = []
    for name, group, bins, fit in LADDER:
        lb = tuple(1.0 for _ in w.layer_bin) if bins == "uniform" else tuple(w.layer_bin)
        wc = dataclasses.replace(w, group_size=group, layer_bin=lb,
                                 level_mult=(w.level_mult[0],))
        p = CodecParams.of(wc)
        codec = Codec(p, device=device)
        L, C = wc.n_layers, wc.n_channels
        ca = torch.empty((L, 2, C, 256), dtype=torch.int16, device=device)
        cd = torch.empty((1, L, 2, C, 256), dtype=torch.int16, device=device)
        if fit == "global":
            ws = torch.empty((CG_FIT_GLOBAL_WORKSPACE_BYTES,), dtype=torch.uint8, device=device)
            cg_fit_cdf_global(p, kv, 0, ca, cd[0], ws)
        elif fit == "other":
            other = W.generate(dataclasses.replace(wc, seed=wc.seed + 1000))
            kv_other = torch.from_numpy(other.view(np.int16)).to(device)
            cg_fit_cdf(p, kv_other, 0, ca, cd[0])
            torch.cuda.synchronize()
            del kv_other
        else:
            cg_fit_cdf(p, kv, 0, ca, cd[0])
        cl = torch.zeros((wc.n_ctx, codec.n_chunks), dtype=torch.uint8, device=device)
        words, offsets, scales = codec.encode(kv, cl, ca, cd)
        out = codec.decode(words, offsets, scales, cl, ca, cd)
        err = out.view(torch.float16).float() - x
        total_words = int(offsets[-1].item())
        n = w.n_elem
        out_rows.append({
            "config": name, "group_size": group, "bins": list(lb), "distributions": fit,
            "payload_bits_per_element": round(total_words * 32 / n, 4),
            "side_bits_per_element": round(codec.n_streams * 12 * 8 / n, 4),
            "rel_rms_error": round(float(torch.sqrt(torch.mean(err * err))) / x_rms, 6),
            "max_abs_error": round(float(err.abs().max()), 6),
        })
        del words, out, err
        torch.cuda.synchronize()
    return out_rows


def main(argv=None):
    from paper_2310_07240_amd import workloads as W
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--workload", action="append",
                    help="workload name (repeatable); default: every workload")
    args = ap.parse_args(argv)
    names = args.workload or list(W.WORKLOADS)
    for nm in names:
        rows = run(W.WORKLOADS[nm])
        base = rows[0]["payload_bits_per_element"]
        for r in rows:
            r["vs_first"] = round(r["payload_bits_per_element"] / base, 4)
        print(json.dumps({"workload": nm, "rows": rows}), flush=True)


if __name__ == "__main__":
    sys.exit(main())
