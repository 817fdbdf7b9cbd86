#!/usr/bin/env python
"""Benchmark of the KV codec on one MI355X: arithmetic-decode throughput in GB/s of fp16 KV,
plus encode throughput and bits per element.

One step = the whole codec over one KV cache resident in HBM: fit the distributions of every
level (cg_fit_cdf), encode (cg_encode), decode (cg_decode). `value` is the decode throughput
(fp16 bytes of KV produced per second of cg_decode, HIP events on the launch stream).

Prints ONE JSON line. Also reports the roofline of the decode kernel, the HBM fraction, and the
CPU oracle timed on the host's cores on the same workload (a baseline, not the target).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "AC decode GB/s of fp16 KV (+ encode GB/s, bits/element), 1 MI355X"
HBM_PEAK_GBPS = 8000.0
# Integer / fp32 vector issue rate: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz = 39.3 T lane-ops/s.
VALU_PEAK_TOPS = 256 * 4 * 16 * 2.4e9 / 1e12
# Algorithmic 32-bit operations of one decode step (one symbol): target 5, binary search over
# 255 symbols 8, interval update 10, one-step renormalisation with bit refill 20, dequantize 5.
DECODE_OPS_PER_SYMBOL = 48


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "decode_traffic_mistral7b_t4096.json")
DECODE_SRC = os.path.join(ROOT, "paper_2310_07240_amd", "csrc", "cg_decode.hip")


def decode_source_hash() -> str:
    """Hash of the decode kernels' source without comments and blank space, so a profile stays
    valid across comment edits and goes stale on any code change."""
    with open(DECODE_SRC) as f:
        src = f.read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    src = re.sub(r"//[^\n]*", "", src)
    src = re.sub(r"\s+", " ", src).strip()
    return hashlib.sha256(src.encode()).hexdigest()[:16]


def measured_traffic(workload: str):
    """HBM bytes per decode launch from the committed FETCH_SIZE / WRITE_SIZE profile, scaled
    by the same counters on a plain copy of known size; None if the decode kernel's source has
    changed since those counters were taken (or no profile exists for this workload)."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("workload") != workload or t.get("decode_source_sha256_16") != decode_source_hash():
        return None
    return t.get("decode_bytes_per_launch")


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="mistral7b_gqa_t4096")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-threads", type=int, default=0, help="0 = all host cores")
    ap.add_argument("--no-streamed", action="store_true",
                    help="skip the chunk-pipelined decode (payload copied from pinned host memory "
                         "chunk by chunk while earlier chunks decode), run after the timed region")
    ap.add_argument("--no-repeated", action="store_true",
                    help="skip the decode repeated back to back, run after the timed region")
    ap.add_argument("--no-calib-copy", action="store_true",
                    help="skip the plain copy of known size run after the timed region (it "
                         "calibrates rocprofv3's FETCH_SIZE / WRITE_SIZE counters)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the codec has no multi-GPU path (its streams "
              "are independent, so a second GPU would simply take other chunks or layers). "
              "Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2310_07240_amd import workloads as W
    from paper_2310_07240_amd.cachegen import (Codec, CodecParams, cg_decode, cg_encode,
                                               cg_fit_cdf)

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    w = W.WORKLOADS[args.workload]
    p = CodecParams.of(w)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    t = time.time()
    kv_np = W.generate(w)
    log(f"generated {w.name}: {w.n_elem} elements in {time.time() - t:.1f}s")
    codec = Codec(p, device=dev)
    kv = torch.from_numpy(kv_np.view(np.int16)).to(dev)
    cl_np = w.chunk_levels()
    cl = torch.from_numpy(cl_np).to(dev)
    L, C, NLV = w.n_layers, w.n_channels, w.n_levels
    ca = torch.empty((L, 2, C, 256), dtype=torch.int16, device=dev)
    cd = torch.empty((NLV, L, 2, C, 256), dtype=torch.int16, device=dev)
    words = torch.empty((codec.bound_words,), dtype=torch.int32, device=dev)
    offsets = torch.empty((codec.n_streams + 1,), dtype=torch.int64, device=dev)
    scales = torch.empty((codec.n_streams,), dtype=torch.float32, device=dev)
    ws = torch.empty((codec.ws_bytes,), dtype=torch.uint8, device=dev)
    out = torch.zeros(w.kv_shape, dtype=torch.int16, device=dev)
    stream = torch.cuda.current_stream()

    def step(ev=None):
        if ev:
            ev[0].record(stream)
        for lv in range(NLV):
            cg_fit_cdf(p, kv, lv, ca if lv == 0 else None, cd[lv], stream)
        if ev:
            ev[1].record(stream)
        cg_encode(p, kv, cl, ca, cd, words, offsets, scales, ws, stream)
        if ev:
            ev[2].record(stream)
        cg_decode(p, words, offsets, scales, cl, ca, cd, 0, codec.n_chunks, out, stream)
        if ev:
            ev[3].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(events[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    if not args.no_calib_copy:
        # outside the timed region: a plain device-to-device copy of exactly fp16-KV bytes, so a
        # counter profile of this run can scale FETCH_SIZE / WRITE_SIZE to bytes
        calib = torch.empty_like(kv)
        calib.copy_(kv)
        torch.cuda.synchronize()
        del calib
    repeated = None
    if not args.no_repeated:
        # outside the timed region: the same decode repeated back to back, after one untimed run
        # (the decode's own steady state; inside a step it follows the encode)
        cg_decode(p, words, offsets, scales, cl, ca, cd, 0, codec.n_chunks, out, stream)
        rep = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(10)]
        for e0, e1 in rep:
            e0.record(stream)
            cg_decode(p, words, offsets, scales, cl, ca, cd, 0, codec.n_chunks, out, stream)
            e1.record(stream)
        torch.cuda.synchronize()
        rep_ms = sorted(e0.elapsed_time(e1) for e0, e1 in rep)
        repeated = rep_ms[len(rep_ms) // 2]
    fit_ms = [e[0].elapsed_time(e[1]) for e in events]
    enc_ms = [e[1].elapsed_time(e[2]) for e in events]
    dec_ms = [e[2].elapsed_time(e[3]) for e in events]
    dec_avg = sum(dec_ms) / len(dec_ms)
    enc_avg = sum(enc_ms) / len(enc_ms)
    fit_avg = sum(fit_ms) / len(fit_ms)

    n_elem = w.n_elem
    fp16_bytes = 2 * n_elem
    off_np = offsets.cpu().numpy().view(np.uint64)
    total_words = int(off_np[-1])
    S = codec.n_streams
    payload_bits = total_words * 32
    side_bits = S * (4 + 8) * 8                       # fp32 scale + uint64 offset per stream
    cdf_bytes = (L * 2 * C * 512) * (1 + NLV)
    decode_gbps = fp16_bytes / (dec_avg * 1e-3) / 1e9
    encode_gbps = fp16_bytes / (enc_avg * 1e-3) / 1e9
    # decode kernel: algorithmic bytes = fp16 written + payload + side info + the CDF tables of
    # the levels the chunks use (each table counted once)
    levels_used = len(set(int(v) for v in cl_np.reshape(-1)))
    dec_bytes = fp16_bytes + total_words * 4 + S * (4 + 8) + L * 2 * C * 512 * (1 + levels_used)
    hbm_gbps = dec_bytes / (dec_avg * 1e-3) / 1e9
    ops = DECODE_OPS_PER_SYMBOL * n_elem
    alu_tops = ops / (dec_avg * 1e-3) / 1e12

    result = {
        "metric": METRIC,
        "value": round(decode_gbps, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall * 1e3 / args.steps, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u32",
        "data": "synthetic (seeded random-walk KV shaped like the model; no real cache)",
        "config": {"workload": w.name, "n_ctx": w.n_ctx, "n_layers": L, "n_tokens": w.n_tokens,
                   "n_channels_per_kv": C, "group_size": w.group_size, "chunk_len": w.chunk_len,
                   "n_levels": NLV, "streams": S},
        "decode_ms": round(dec_avg, 4),
        "encode_ms": round(enc_avg, 4),
        "fit_ms": round(fit_avg, 4),
        "encode_GBps": round(encode_gbps, 2),
        "bits_per_element": {"payload": round(payload_bits / n_elem, 4),
                             "side_info": round(side_bits / n_elem, 4),
                             "cdf_tables": round(cdf_bytes * 8 / n_elem, 4)},
        "roofline": {"bound": "alu", "achieved": round(alu_tops, 3), "peak": round(VALU_PEAK_TOPS, 1),
                     "unit": "Tops/s", "frac": round(alu_tops / VALU_PEAK_TOPS, 4),
                     "ops_per_symbol": DECODE_OPS_PER_SYMBOL,
                     "traffic": measured_traffic(w.name),
                     "kernel": "decode_g10_kernel" if w.group_size == 10 else "decode_kernel"},
        "hbm": {"achieved": round(hbm_gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                "frac": round(hbm_gbps / HBM_PEAK_GBPS, 4),
                "bytes_per_launch": dec_bytes},
    }

    if repeated is not None:
        result["decode_repeated"] = {
            "ms": round(repeated, 4), "GBps": round(fp16_bytes / (repeated * 1e-3) / 1e9, 2),
            "runs": 10, "what": "median of 10 decodes back to back after the timed steps; "
                                "`value` is the decode inside each step, right after the encode"}
    if not args.no_streamed:
        result["streamed"] = streamed(p, codec, words, offsets, scales, cl, ca, cd, total_words)
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(w, kv_np, args.cpu_threads)
    print(json.dumps(result), flush=True)


def streamed(p, codec, words, offsets, scales, cl, ca, cd, total_words):
    """Chunk-pipelined decode (cg_decode_streamed): the payload arrives chunk by chunk in pinned
    host memory and is copied to the GPU on one stream while the chunks already copied decode on
    another. Reported for the host-to-device bus alone and for a 100 Gb/s link; outside the timed
    region."""
    import torch
    from paper_2310_07240_amd.cachegen import cg_decode_streamed
    tail = 8
    words_host = torch.empty((total_words + tail,), dtype=torch.int32, pin_memory=True)
    words_host.copy_(words[:total_words + tail].cpu())
    off_host = offsets.cpu()
    words_dev = torch.zeros((total_words + tail,), dtype=torch.int32, device=words.device)
    out = torch.empty(codec.p.kv_shape, dtype=torch.int16, device=words.device)
    dec_s, copy_s = torch.cuda.Stream(), torch.cuda.Stream()
    res = {"payload_MB": round(total_words * 4 / 1e6, 2)}
    for name, gbps in (("host_to_device", 0.0), ("link_100gbps", 100.0)):
        cg_decode_streamed(p, words_host, off_host, words_dev, offsets, scales, cl, ca, cd, out,
                           gbps, dec_s, copy_s)          # warm-up
        st = cg_decode_streamed(p, words_host, off_host, words_dev, offsets, scales, cl, ca, cd,
                                out, gbps, dec_s, copy_s)
        res[name] = {k: (round(v, 4) if isinstance(v, float) else v) for k, v in st.items()}
    return res


def cpu_baseline(w, kv_np, threads):
    """The CPU oracle's decode of the same workload on the host's cores (it fits and encodes
    with its own code first, untimed)."""
    import oracle
    threads = threads or oracle.default_threads()
    shape = oracle.shape_from(w)
    cl = w.chunk_levels()
    t = time.time()
    ca, cd = oracle.fit_all_levels(kv_np, shape, threads)
    words, offsets, scales = oracle.encode(kv_np, shape, cl, ca, cd, threads)
    log(f"oracle fit+encode {time.time() - t:.1f}s on {threads} threads")
    t = time.perf_counter()
    oracle.decode(words, offsets, scales, shape, cl, ca, cd, threads=threads)
    dt = time.perf_counter() - t
    cpu_model = ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    cpu_model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"value": round(2 * w.n_elem / dt / 1e9, 4), "unit": "GB/s", "cores": threads,
            "kind": "oracle", "seconds": round(dt, 2), "cpu": cpu_model,
            "sample": f"the whole {w.name} cache ({w.n_elem} fp16 elements) decoded by the "
                      f"oracle from its own payload"}


if __name__ == "__main__":
    main()
