#!/usr/bin/env python
"""Benchmark of the KV codec on one MI355X: arithmetic-decode throughput in GB/s of fp16 KV,
plus encode throughput and bits per element.

One step = the whole codec over one KV cache resident in HBM: fit the distributions of every
level and the streams' scales (cg_fit_cdf_levels), encode with those scales
(cg_encode_with_scales), decode (cg_decode). `value` is the decode throughput
(fp16 bytes of KV produced per second of cg_decode, HIP events on the launch stream) on the
Mistral-7B-shaped 4K-token cache.

The timed region (the warm-up steps, then the timed steps) follows one run of the same steps
(`cold_start`): an MI355X out of idle raises its clock over its first ~20-30 ms of work (the
decode's cycle count stays the same while its time falls by up to 15 %), and five warm-up steps
take about 7 ms. --no-cold-start skips that run.

Prints ONE JSON line. Also reports the roofline of the decode kernel, the HBM fraction, the
other four workloads (`per_workload`: a few steps each, same kernels), and the CPU oracle timed
on the host's cores on the same workload (a baseline, not the target). The oracle's payload and
decoded cache are compared bit for bit with the GPU's (`parity`); a mismatch makes the run exit
with status 3 after printing the line.
"""
from __future__ import annotations

import argparse
import gc
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
# A model, not a measurement: algorithmic 32-bit operations of one decode step (one symbol):
# target 5, binary search over 255 symbols 8, interval update 10, one-step renormalisation with
# bit refill 20, dequantize 5. The measured instruction count comes from the counter profile.
DECODE_OPS_PER_SYMBOL = 48

MAIN_WORKLOAD = "mistral7b_gqa_t4096"
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


def decode_profile(workload: str):
    """The committed counter profile of the decode kernel (HBM bytes per launch from FETCH_SIZE
    / WRITE_SIZE scaled by a plain copy of known size; VALU instructions per symbol step), or
    None if the decode kernel's source has changed since the counters were taken or no profile
    exists for this workload."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("workload") != workload or t.get("decode_source_sha256_16") != decode_source_hash():
        return None
    return t


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


class Run:
    """One workload resident on the GPU with its codec buffers."""

    def __init__(self, w, dev, kv_np=None):
        import torch
        from paper_2310_07240_amd import workloads as W
        from paper_2310_07240_amd.cachegen import Codec, CodecParams
        self.torch = torch
        self.w = w
        self.p = CodecParams.of(w)
        t = time.time()
        if kv_np is None:
            kv_np = W.generate(w)
        log(f"{w.name}: {w.n_elem} elements generated in {time.time() - t:.1f}s")
        self.codec = Codec(self.p, device=dev)
        self.kv = torch.from_numpy(kv_np.view(np.int16)).to(dev)
        self.cl_np = w.chunk_levels()
        self.cl = torch.from_numpy(self.cl_np).to(dev)
        L, C, NLV = w.n_layers, w.n_channels, w.n_levels
        self.ca = torch.empty((L, 2, C, 256), dtype=torch.int16, device=dev)
        self.cd = torch.empty((NLV, L, 2, C, 256), dtype=torch.int16, device=dev)
        self.words = torch.empty((self.codec.bound_words,), dtype=torch.int32, device=dev)
        self.offsets = torch.empty((self.codec.n_streams + 1,), dtype=torch.int64, device=dev)
        self.scales = torch.empty((self.codec.n_streams,), dtype=torch.float32, device=dev)
        self.ws = torch.empty((self.codec.ws_bytes,), dtype=torch.uint8, device=dev)
        self.out = torch.zeros(w.kv_shape, dtype=torch.int16, device=dev)
        self.stream = torch.cuda.current_stream()

    def fit(self):
        # the tables of every level, and the streams' scales from the same maxima
        from paper_2310_07240_amd.cachegen import cg_fit_cdf_levels
        cg_fit_cdf_levels(self.p, self.kv, self.ca, self.cd, None, self.stream, self.scales)

    def encode(self):
        # the encoder takes the fit's scales instead of finding the maxima again
        from paper_2310_07240_amd.cachegen import cg_encode_with_scales
        cg_encode_with_scales(self.p, self.kv, self.cl, self.ca, self.cd, self.scales,
                              self.words, self.offsets, self.ws, self.stream)

    def decode(self):
        from paper_2310_07240_amd.cachegen import cg_decode
        cg_decode(self.p, self.words, self.offsets, self.scales, self.cl, self.ca, self.cd, 0,
                  self.codec.n_chunks, self.out, self.stream)

    def step(self, ev=None):
        if ev:
            ev[0].record(self.stream)
        self.fit()
        if ev:
            ev[1].record(self.stream)
        self.encode()
        if ev:
            ev[2].record(self.stream)
        self.decode()
        if ev:
            ev[3].record(self.stream)

    def timed(self, steps, warmup):
        """Warm-up steps, then `steps` timed steps; per-stage times (ms) and the wall time."""
        torch = self.torch
        for _ in range(warmup):
            self.step()
        torch.cuda.synchronize()
        events = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(steps):
            self.step(events[i])
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        fit = [e[0].elapsed_time(e[1]) for e in events]
        enc = [e[1].elapsed_time(e[2]) for e in events]
        dec = [e[2].elapsed_time(e[3]) for e in events]
        return fit, enc, dec, wall

    def warm(self, seconds):
        """Steps, each waited for, until `seconds` of wall time have passed (the clock of a GPU
        out of idle ramps up over its first ~20-30 ms of work); returns the number of steps."""
        t0 = time.perf_counter()
        n = 0
        while n == 0 or time.perf_counter() - t0 < seconds:
            self.step()
            self.torch.cuda.synchronize()
            n += 1
        return n

    def summary(self, fit, enc, dec):
        """Throughputs, bits per element and the decode's HBM fraction."""
        w = self.w
        L, C = w.n_layers, w.n_channels
        dec_avg, enc_avg, fit_avg = (sum(x) / len(x) for x in (dec, enc, fit))
        fp16_bytes = 2 * w.n_elem
        total_words = int(self.offsets[-1].item())
        S = self.codec.n_streams
        levels_used = len(set(int(v) for v in self.cl_np.reshape(-1)))
        table_bytes = L * 2 * C * 512
        # decode kernel: algorithmic bytes = fp16 written + payload + side info + the tables of
        # the levels the chunks use (each table counted once)
        dec_bytes = fp16_bytes + total_words * 4 + S * (4 + 8) + table_bytes * (1 + levels_used)
        hbm_gbps = dec_bytes / (dec_avg * 1e-3) / 1e9
        return {
            "decode_ms": round(dec_avg, 4),
            "decode_GBps": round(fp16_bytes / (dec_avg * 1e-3) / 1e9, 2),
            "encode_ms": round(enc_avg, 4),
            "encode_GBps": round(fp16_bytes / (enc_avg * 1e-3) / 1e9, 2),
            "fit_ms": round(fit_avg, 4),
            "fit_levels": w.n_levels,
            "bits_per_element": {"payload": round(total_words * 32 / w.n_elem, 4),
                                 "side_info": round(S * 12 * 8 / w.n_elem, 4),
                                 "cdf_tables": round(table_bytes * (1 + w.n_levels) * 8
                                                     / w.n_elem, 4)},
            "hbm": {"achieved": round(hbm_gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                    "frac": round(hbm_gbps / HBM_PEAK_GBPS, 4), "bytes_per_launch": dec_bytes},
            "alu_frac_model": round(DECODE_OPS_PER_SYMBOL * w.n_elem / (dec_avg * 1e-3) / 1e12
                                    / VALU_PEAK_TOPS, 4),
        }

    def host_results(self):
        """Tables, offsets, scales, payload and decoded cache as numpy bit patterns."""
        off = self.offsets.cpu().numpy().view(np.uint64)
        return dict(ca=self.ca.cpu().numpy().view(np.uint16),
                    cd=self.cd.cpu().numpy().view(np.uint16), offsets=off,
                    scales=self.scales.cpu().numpy().view(np.uint32),
                    words=self.words[: int(off[-1])].cpu().numpy().view(np.uint32),
                    out=self.out.cpu().numpy().view(np.uint16))

    def release(self):
        for name in ("kv", "cl", "ca", "cd", "words", "offsets", "scales", "ws", "out"):
            setattr(self, name, None)
        self.torch.cuda.empty_cache()


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=MAIN_WORKLOAD)
    ap.add_argument("--no-cpu-baseline", action="store_true",
                    help="skip the oracle (and with it the bit-exactness check of the run)")
    ap.add_argument("--cpu-threads", type=int, default=0, help="0 = all host cores")
    ap.add_argument("--no-streamed", action="store_true",
                    help="skip the chunk-pipelined decode (payload copied from pinned host memory "
                         "chunk by chunk while earlier chunks decode), run after the timed region")
    ap.add_argument("--no-repeated", action="store_true",
                    help="skip the decode repeated back to back, run after the timed region")
    ap.add_argument("--no-calib-copy", action="store_true",
                    help="skip the plain copy of known size run after the timed region (it "
                         "calibrates rocprofv3's FETCH_SIZE / WRITE_SIZE counters)")
    ap.add_argument("--no-per-workload", action="store_true",
                    help="skip the other workloads (run after the main one, a few steps each)")
    ap.add_argument("--per-workload-steps", type=int, default=3)
    ap.add_argument("--no-cold-start", action="store_true",
                    help="skip the run of the same steps before the timed region (reported as "
                         "cold_start; without it the timed region starts on a GPU out of idle)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the codec has no multi-GPU path (its streams "
              "are independent, so a second GPU would simply take other chunks or layers). "
              "Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2310_07240_amd import workloads as W

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    w = W.WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    kv_np = W.generate(w)
    run = Run(w, dev, kv_np)
    cold = None
    # no garbage collection from here to the end of the timed region: a full collection holds
    # the host for tens of milliseconds, in which the GPU runs dry and its clock drops
    gc.collect()
    gc.disable()
    try:
        if not args.no_cold_start:
            # the same warm-up and timed steps once before the timed region, as the process's
            # first GPU work: reported as `cold_start` (the clock is still ramping up from idle)
            cold = run.timed(args.steps, args.warmup)[:3]
        # the timed region: W warm-up steps, then K timed steps
        fit, enc, dec, wall = run.timed(args.steps, args.warmup)
    finally:
        gc.enable()
    if cold is not None:
        cold = run.summary(*cold)
    if not args.no_calib_copy:
        # outside the timed region: a plain device-to-device copy of exactly fp16-KV bytes, so a
        # counter profile of this run can scale FETCH_SIZE / WRITE_SIZE to bytes
        calib = torch.empty_like(run.kv)
        calib.copy_(run.kv)
        torch.cuda.synchronize()
        del calib
    repeated = None
    if not args.no_repeated:
        # outside the timed region: the same decode repeated back to back, after one untimed run
        # (the decode's own steady state; inside a step it follows the encode)
        run.decode()
        rep = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(10)]
        for e0, e1 in rep:
            e0.record(run.stream)
            run.decode()
            e1.record(run.stream)
        torch.cuda.synchronize()
        rep_ms = sorted(e0.elapsed_time(e1) for e0, e1 in rep)
        repeated = rep_ms[len(rep_ms) // 2]

    s = run.summary(fit, enc, dec)
    dec_avg = s["decode_ms"]
    fp16_bytes = 2 * w.n_elem
    alu_tops = DECODE_OPS_PER_SYMBOL * w.n_elem / (dec_avg * 1e-3) / 1e12
    prof = decode_profile(w.name)
    roofline = {"bound": "alu", "achieved": round(alu_tops, 3), "peak": round(VALU_PEAK_TOPS, 1),
                "unit": "Tops/s", "frac": round(alu_tops / VALU_PEAK_TOPS, 4),
                "ops_per_symbol": DECODE_OPS_PER_SYMBOL,
                "ops_per_symbol_is": "an algorithmic model (not a measurement)",
                "traffic": prof.get("decode_bytes_per_launch") if prof else None,
                "kernel": "decode_g10_kernel" if w.group_size == 10 else "decode_kernel"}
    if prof:
        roofline["overfetch"] = round(prof["decode_bytes_per_launch"]
                                      / s["hbm"]["bytes_per_launch"], 3)
        for k in ("valu_insts_per_symbol_step", "valu_busy", "waves_per_simd"):
            if k in prof:
                roofline[k + "_measured"] = prof[k]

    result = {
        "metric": METRIC,
        "value": s["decode_GBps"],
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
        "config": {"workload": w.name, "n_ctx": w.n_ctx, "n_layers": w.n_layers,
                   "n_tokens": w.n_tokens, "n_channels_per_kv": w.n_channels,
                   "group_size": w.group_size, "chunk_len": w.chunk_len,
                   "n_levels": w.n_levels, "streams": run.codec.n_streams},
        "decode_ms": s["decode_ms"],
        "encode_ms": s["encode_ms"],
        "fit_ms": s["fit_ms"],
        "encode_GBps": s["encode_GBps"],
        "bits_per_element": s["bits_per_element"],
        "roofline": roofline,
        "hbm": s["hbm"],
    }
    if cold is not None:
        result["cold_start"] = {
            k: cold[k] for k in ("decode_ms", "decode_GBps", "encode_ms", "encode_GBps", "fit_ms")}
        result["cold_start"]["what"] = (
            "the same warm-up and timed steps run once right before the timed region, as the "
            "process's first GPU work: an MI355X out of idle raises its clock over the first "
            "~20-30 ms of work (same cycle count per decode, 2.1 -> 2.35 GHz)")
    if repeated is not None:
        result["decode_repeated"] = {
            "ms": round(repeated, 4), "GBps": round(fp16_bytes / (repeated * 1e-3) / 1e9, 2),
            "runs": 10, "what": "median of 10 decodes back to back after the timed steps; "
                                "`value` is the decode inside each step, right after the encode"}
    if not args.no_streamed:
        result["streamed"] = streamed(run)
    gpu_res = run.host_results() if not args.no_cpu_baseline else None
    run.release()
    del run

    if not args.no_per_workload:
        per = {}
        for name, wo in W.WORKLOADS.items():
            if name == w.name:
                continue
            r = Run(wo, dev)
            gc.collect()
            gc.disable()
            try:
                nwarm = r.warm(0.05)   # 50 ms of steps, then the timed ones
                f2, e2, d2, _ = r.timed(args.per_workload_steps, 1)
            finally:
                gc.enable()
            per[name] = r.summary(f2, e2, d2)
            per[name]["steps"] = args.per_workload_steps
            per[name]["warmup_steps"] = nwarm + 1
            log(f"{name}: decode {per[name]['decode_GBps']} GB/s, "
                f"encode {per[name]['encode_GBps']} GB/s, fit {per[name]['fit_ms']} ms")
            r.release()
            del r
        result["per_workload"] = per

    ok = True
    if not args.no_cpu_baseline:
        cpu, parity = cpu_baseline(w, kv_np, args.cpu_threads, gpu_res)
        result["cpu_baseline"] = cpu
        result["parity"] = parity
        ok = parity["bit_exact"]
    print(json.dumps(result), flush=True)
    if not ok:
        log("GPU results differ from the oracle's: " + json.dumps(parity["mismatches"]))
        sys.exit(3)


def streamed(run):
    """Chunk-pipelined decode (cg_decode_streamed): the payload arrives chunk by chunk in pinned
    host memory and is copied to the GPU on one stream while the chunks already copied decode on
    another. Reported for the host-to-device bus alone and for a 100 Gb/s link; outside the timed
    region. `last_chunk_exposed_ms` is the decode time left after the last byte has arrived."""
    import torch
    from paper_2310_07240_amd.cachegen import cg_decode_streamed
    tail = 8
    total_words = int(run.offsets[-1].item())
    words_host = torch.empty((total_words + tail,), dtype=torch.int32, pin_memory=True)
    words_host.copy_(run.words[:total_words + tail].cpu())
    off_host = run.offsets.cpu()
    words_dev = torch.zeros((total_words + tail,), dtype=torch.int32, device=run.words.device)
    out = torch.empty(run.w.kv_shape, dtype=torch.int16, device=run.words.device)
    dec_s, copy_s = torch.cuda.Stream(), torch.cuda.Stream()
    res = {"payload_MB": round(total_words * 4 / 1e6, 2)}
    for name, gbps in (("host_to_device", 0.0), ("link_100gbps", 100.0)):
        args = (run.p, words_host, off_host, words_dev, run.offsets, run.scales, run.cl, run.ca,
                run.cd, out, gbps, dec_s, copy_s)
        cg_decode_streamed(*args)          # warm-up
        st = cg_decode_streamed(*args)
        d = {k: (round(v, 4) if isinstance(v, float)
                 else [round(x, 4) for x in v] if isinstance(v, list) else v)
             for k, v in st.items()}
        d["last_chunk_exposed_ms"] = round(st["total_ms"] - st["transfer_ms"], 4)
        res[name] = d
    return res


def _mismatch(name, a, b):
    a = np.asarray(a).reshape(-1)
    b = np.asarray(b).reshape(-1)
    if a.shape != b.shape:
        return {"what": name, "shape": [list(a.shape), list(b.shape)]}
    n = int(np.count_nonzero(a != b))
    return {"what": name, "count": n} if n else None


def cpu_baseline(w, kv_np, threads, gpu_res):
    """The CPU oracle's decode of the same workload on the host's cores (it fits and encodes
    with its own code first, untimed), one core's rate on a two-layer sample, and the
    comparison of the oracle's tables, payload and decoded cache with the GPU's."""
    import oracle
    threads = threads or oracle.default_threads()
    shape = oracle.shape_from(w)
    cl = w.chunk_levels()
    t = time.time()
    ca, cd = oracle.fit_all_levels(kv_np, shape, threads)
    words, offsets, scales = oracle.encode(kv_np, shape, cl, ca, cd, threads)
    log(f"oracle fit+encode {time.time() - t:.1f}s on {threads} threads")
    t = time.perf_counter()
    out = oracle.decode(words, offsets, scales, shape, cl, ca, cd, threads=threads)
    dt = time.perf_counter() - t
    mism = [m for m in (_mismatch("cdf_anchor", gpu_res["ca"], ca),
                        _mismatch("cdf_delta", gpu_res["cd"], cd),
                        _mismatch("offsets", gpu_res["offsets"], offsets),
                        _mismatch("scales", gpu_res["scales"], scales.view(np.uint32)),
                        _mismatch("words", gpu_res["words"], words),
                        _mismatch("decoded fp16", gpu_res["out"], out)) if m]
    parity = {"bit_exact": not mism, "mismatches": mism,
              "compared": "tables, offsets, scales, payload words and the decoded fp16 cache of "
                          "the timed run against the oracle's, bit for bit"}
    del out, words
    # one core: the oracle decodes a sample of the first two layers, from its own payload
    n_l = min(2, w.n_layers)
    sub = w.with_(name=w.name + "_sample", n_layers=n_l, layer_bin=tuple(w.layer_bin[:n_l]))
    sub_kv = np.ascontiguousarray(kv_np[:, :n_l])
    ssh = oracle.shape_from(sub)
    sca, scd = oracle.fit_all_levels(sub_kv, ssh, threads)
    sw, so, ss = oracle.encode(sub_kv, ssh, cl, sca, scd, threads)
    t = time.perf_counter()
    oracle.decode(sw, so, ss, ssh, cl, sca, scd, threads=1)
    dt1 = time.perf_counter() - t
    cpu_model = ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    cpu_model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    cpu = {"value": round(2 * w.n_elem / dt / 1e9, 4), "unit": "GB/s", "cores": threads,
           "kind": "oracle", "seconds": round(dt, 2), "cpu": cpu_model,
           "sample": f"the whole {w.name} cache ({w.n_elem} fp16 elements) decoded by the "
                     f"oracle from its own payload",
           "single_thread": {"value": round(2 * sub.n_elem / dt1 / 1e9, 4), "unit": "GB/s",
                             "cores": 1, "seconds": round(dt1, 2),
                             "sample": f"layers 0-{n_l - 1} of {w.name} ({sub.n_elem} "
                                       f"elements), decoded on one thread"}}
    return cpu, parity


if __name__ == "__main__":
    main()
