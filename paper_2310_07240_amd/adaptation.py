"""Streaming adaptation study on one GPU (CacheGen Sec. 5.3 "KV cache streaming adaptation",
App. B Alg. 1; the evaluation of Sec. 7.4 samples every chunk's bandwidth from 0.1-10 Gb/s and
reports the rate of SLO violations).

1. A Mistral-7B-shaped synthetic cache of 9216 tokens (six 1536-token chunks, about a LongChat
   context) is fitted and encoded at seven levels whose delta bins are 0.5, 1, 2, 4, 8, 16 and 32
   times the paper's default bins (level 1 is the default, "medium" level), all with the codec's kernels
   through the C ABI; each chunk's payload size per level comes from the offsets, each level's
   reconstruction error from a decode.
2. For seeded bandwidth traces (one rate per chunk, log-uniform in [0.1, 10] Gb/s) and a set of
   SLOs, the chunks are planned and their transfer simulated by cg_adapt_schedule (host code
   in the library), against three fixed policies: the default level for every chunk (CacheGen
   without adaptation), the smallest level, and the 8-bit quantization baseline (one byte per
   element, no entropy coding).

Text recompute time per chunk is a parameter (no model runs here); quality is reported only as
the decoded cache's relative RMS error of the chosen levels (text counts as exact).

Usage: python -m paper_2310_07240_amd.adaptation [--traces 100] [--recompute-ms 60]
"""
from __future__ import annotations

import argparse
import dataclasses
import json
import sys

import numpy as np

LEVELS = (0.5, 1.0, 2.0, 4.0, 8.0, 16.0, 32.0)
DEFAULT_LEVEL = 1


def level_sizes(w, device="cuda"):
    """Per-chunk payload bytes [NC][levels] and per-level relative RMS error of the decoded
    cache, for workload `w` coded at every level of w.level_mult."""
    import torch
    from paper_2310_07240_amd import workloads as W
    from paper_2310_07240_amd.cachegen import Codec, CodecParams
    p = CodecParams.of(w)
    codec = Codec(p, device=device)
    kv = torch.from_numpy(W.generate(w).view(np.int16)).to(device)
    x = kv.view(torch.float16).float()
    x_rms = float(torch.sqrt(torch.mean(x * x)))
    ca, cd = codec.fit(kv)
    NC, NLV = codec.n_chunks, p.n_levels
    per_chunk = w.n_layers * 2 * w.n_channels
    sizes = np.zeros((NC, NLV))
    errs = []
    for lv in range(NLV):
        cl = torch.full((w.n_ctx, NC), lv, dtype=torch.uint8, device=device)
        words, offsets, scales = codec.encode(kv, cl, ca, cd)
        out = codec.decode(words, offsets, scales, cl, ca, cd)
        off = offsets.cpu().numpy().view(np.uint64).astype(np.int64)
        for c in range(NC):
            for b in range(w.n_ctx):
                s0 = (b * NC + c) * per_chunk
                sizes[c, lv] += 4.0 * (off[s0 + per_chunk] - off[s0])
        e = out.view(torch.float16).float() - x
        errs.append(float(torch.sqrt(torch.mean(e * e))) / x_rms)
    return sizes, errs


def study(sizes, errs, n_elem_per_chunk, slos_ms, traces=100, recompute_ms=60.0,
          text_bytes=6144.0, seed=0):
    """SLO-violation rates of the adaptive plan and the fixed policies."""
    from paper_2310_07240_amd.cachegen import cg_adapt_schedule
    NC, NLV = sizes.shape
    rng = np.random.default_rng(seed)
    bws = np.exp(rng.uniform(np.log(0.1), np.log(10.0), size=(traces, NC)))
    tb = np.full(NC, text_bytes)
    rc = np.full(NC, recompute_ms)
    quant = np.full(NC, float(n_elem_per_chunk))          # 8-bit baseline: 1 byte per element
    res = []
    for slo in slos_ms:
        row = {"slo_ms": slo}
        pol = {"adaptive (text + levels)": [], "adaptive (levels only)": [],
               "fixed default level": [], "fixed smallest level": [], "8-bit quantization": []}
        err = {k: [] for k in pol}
        for bw in bws:
            for name, use_text in (("adaptive (text + levels)", True),
                                   ("adaptive (levels only)", False)):
                ch, t = cg_adapt_schedule(sizes, tb, rc if use_text else None, slo, 0.0,
                                          DEFAULT_LEVEL, bw)
                pol[name].append(t)
                err[name].append(np.mean([0.0 if c < 0 else errs[c] for c in ch]))
            for name, per, e in (("fixed default level", sizes[:, DEFAULT_LEVEL], errs[DEFAULT_LEVEL]),
                                 ("fixed smallest level", sizes[:, NLV - 1], errs[NLV - 1]),
                                 ("8-bit quantization", quant, None)):
                t = float(np.sum(per * 8.0 / (bw * 1e6)))
                pol[name].append(t)
                err[name].append(e if e is not None else float("nan"))
        for name in pol:
            ttft = np.asarray(pol[name])
            row[name] = {"slo_violation_rate": round(float(np.mean(ttft > slo)), 4),
                         "mean_ttft_ms": round(float(np.mean(ttft)), 2),
                         "mean_rel_rms_error": (None if np.isnan(np.mean(err[name]))
                                                else round(float(np.mean(err[name])), 6))}
        res.append(row)
    return res


def main(argv=None):
    from paper_2310_07240_amd import workloads as W
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--traces", type=int, default=100)
    ap.add_argument("--recompute-ms", type=float, default=60.0,
                    help="time to recompute one 1536-token chunk's KV from its text")
    ap.add_argument("--slo-ms", type=float, action="append")
    args = ap.parse_args(argv)
    w = dataclasses.replace(W.MISTRAL_7B_4K, name="mistral7b_gqa_t9216_4levels", n_tokens=9216,
                            level_mult=LEVELS, random_levels=False)
    sizes, errs = level_sizes(w)
    nc = sizes.shape[0]
    per_chunk_elems = w.n_elem // nc
    slos = args.slo_ms or [250.0, 500.0, 1000.0, 2000.0]
    res = study(sizes, errs, per_chunk_elems, slos, args.traces, args.recompute_ms)
    print(json.dumps({"workload": w.name, "levels": LEVELS, "default_level": DEFAULT_LEVEL,
                      "chunk_MB_per_level": [round(float(v) / 1e6, 2) for v in sizes.mean(axis=0)],
                      "rel_rms_error_per_level": [round(e, 6) for e in errs],
                      "recompute_ms_per_chunk": args.recompute_ms, "traces": args.traces,
                      "results": res}), flush=True)


if __name__ == "__main__":
    sys.exit(main())
