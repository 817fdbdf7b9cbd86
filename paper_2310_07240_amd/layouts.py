"""Stream layouts compared on one GPU: the channel streams of this codec (one arithmetic-coder
stream per (context, chunk, layer, K/V, channel)) against the paper's token-parallel layout
(its GPU decoder runs one thread per token, Sec. 6): one stream per (context, layer, K/V,
token) over the token's channels. Both code the same quantized symbols under the same
per-(layer, K/V, channel) tables and decode to the same fp16 cache; they differ in how many
streams there are, how long, and what a decoding lane has to touch per symbol.

For a workload it fits the tables, encodes the resident cache in both layouts through the C
ABI, checks that both decodes agree bit for bit, and reports per layout:
  * decode time (HIP events around cg_decode / cg_decode_tokens, the median of `reps` runs
    after a warm-up) and fp16 GB/s;
  * bits per element: payload, and side information (offsets 8 bytes per stream, scales 4
    bytes per channel stream; the tables are the same for both and not counted);
  * stream count and mean symbols per stream.

Usage: python -m paper_2310_07240_amd.layouts [--workload NAME ...] [--reps N]  (one JSON line
each)
"""
from __future__ import annotations

import argparse
import json
import statistics
import sys

import numpy as np


def _time(fn, reps, torch):
    fn()
    torch.cuda.synchronize()
    times = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        fn()
        e1.record()
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1))
    return statistics.median(times)


def run(w, reps=10, device="cuda"):
    """Returns a dict with one entry per layout for workload `w`."""
    import torch
    from paper_2310_07240_amd import workloads as W
    from paper_2310_07240_amd.cachegen import Codec, CodecParams, cg_decode_tokens_workspace_bytes
    p = CodecParams.of(w)
    codec = Codec(p, device)
    kv = torch.from_numpy(W.generate(w).view(np.int16)).to(device)
    cl = torch.from_numpy(w.chunk_levels()).to(device)
    ca, cd = codec.fit(kv)
    words, offsets, scales = codec.encode(kv, cl, ca, cd)
    twords, toffsets, tscales = codec.encode_tokens(kv, cl, ca, cd)
    torch.cuda.synchronize()
    del kv
    out = torch.empty(p.kv_shape, dtype=torch.int16, device=device)
    tout = torch.empty_like(out)
    ws = torch.empty((cg_decode_tokens_workspace_bytes(p),), dtype=torch.uint8, device=device)
    ms_c = _time(lambda: codec.decode(words, offsets, scales, cl, ca, cd, out=out), reps, torch)
    ms_t = _time(lambda: codec.decode_tokens(twords, toffsets, tscales, cl, ca, cd, out=tout,
                                             workspace=ws), reps, torch)
    same = bool(torch.equal(out, tout))
    n_elem = w.n_elem
    fp16_gb = 2.0 * n_elem / 1e9
    res = {"workload": w.name, "n_elem": n_elem, "decodes_equal": same}
    for name, ms, off, n_streams in (("channel", ms_c, offsets, codec.n_streams),
                                     ("token", ms_t, toffsets, toffsets.numel() - 1)):
        total = int(off[-1].item())
        res[name] = {
            "streams": n_streams,
            "symbols_per_stream": round(n_elem / n_streams, 1),
            "decode_ms": round(ms, 4),
            "decode_GBps": round(fp16_gb / (ms * 1e-3), 2),
            "payload_bits_per_element": round(total * 32 / n_elem, 4),
            "side_bits_per_element": round((8 * (n_streams + 1) + 4 * codec.n_streams) * 8
                                           / n_elem, 4),
        }
    res["token_over_channel_decode_time"] = round(ms_t / ms_c, 3)
    return res


def main(argv=None):
    from paper_2310_07240_amd import workloads as W
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--workload", action="append", default=None, choices=sorted(W.WORKLOADS))
    ap.add_argument("--reps", type=int, default=10)
    args = ap.parse_args(argv)
    for name in args.workload or ["mistral7b_gqa_t4096"]:
        print(json.dumps(run(W.WORKLOADS[name], args.reps)), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
