"""Helpers for the GPU parity tests: run the HIP codec and the CPU oracle on the same seeded
input and return numpy arrays (uint bit patterns) for exact comparison."""
from __future__ import annotations

import sys
import time

import numpy as np

import oracle
from paper_2310_07240_amd import workloads as W


def say(*a):
    print("[gpu-test]", *a, flush=True)
    sys.stdout.flush()


def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch


def run_gpu(w: W.Workload, kv_np: np.ndarray, decode_oracle_payload=None):
    """Fit, encode and decode on the GPU. Returns a dict of numpy arrays."""
    torch = torch_cuda()
    from paper_2310_07240_amd.cachegen import Codec, CodecParams
    p = CodecParams.of(w)
    codec = Codec(p)
    say(f"{w.name}: upload {kv_np.nbytes / 2**20:.1f} MiB")
    kv = torch.from_numpy(np.ascontiguousarray(kv_np).view(np.int16)).cuda()
    cl = torch.from_numpy(w.chunk_levels()).cuda()
    say(f"{w.name}: fit")
    ca, cd = codec.fit(kv)
    torch.cuda.synchronize()
    say(f"{w.name}: encode")
    words, offsets, scales = codec.encode(kv, cl, ca, cd)
    torch.cuda.synchronize()
    say(f"{w.name}: decode")
    out = codec.decode(words, offsets, scales, cl, ca, cd)
    torch.cuda.synchronize()
    off = offsets.cpu().numpy().view(np.uint64)
    total = int(off[-1])
    res = dict(ca=ca.cpu().numpy().view(np.uint16), cd=cd.cpu().numpy().view(np.uint16),
               offsets=off, scales=scales.cpu().numpy(),
               words=words[:total].cpu().numpy().view(np.uint32),
               out=out.cpu().numpy().view(np.uint16))
    if decode_oracle_payload is not None:
        ow, oo, osc, oca, ocd = decode_oracle_payload
        say(f"{w.name}: decode the oracle's payload")
        # the decoder may read CG_TAIL_WORDS (8) words past the payload: pad the exact-size array
        padded = np.concatenate([np.asarray(ow, np.uint32), np.zeros(8, np.uint32)])
        tw = torch.from_numpy(padded.view(np.int32)).cuda()
        to = torch.from_numpy(np.ascontiguousarray(oo).view(np.int64)).cuda()
        ts = torch.from_numpy(np.ascontiguousarray(osc)).cuda()
        tca = torch.from_numpy(np.ascontiguousarray(oca).view(np.int16)).cuda()
        tcd = torch.from_numpy(np.ascontiguousarray(ocd).view(np.int16)).cuda()
        o2 = codec.decode(tw, to, ts, cl, tca, tcd)
        torch.cuda.synchronize()
        res["out_from_oracle_payload"] = o2.cpu().numpy().view(np.uint16)
    del kv, words, out
    return res


def run_oracle(w: W.Workload, kv_np: np.ndarray, threads=None):
    shape = oracle.shape_from(w)
    cl = w.chunk_levels()
    t = time.time()
    ca, cd = oracle.fit_all_levels(kv_np, shape, threads)
    words, offsets, scales = oracle.encode(kv_np, shape, cl, ca, cd, threads)
    out = oracle.decode(words, offsets, scales, shape, cl, ca, cd, threads=threads)
    say(f"{w.name}: oracle {time.time() - t:.1f}s")
    return dict(ca=ca, cd=cd, words=words, offsets=offsets, scales=scales, out=out)


def assert_same(name, a, b):
    a = np.asarray(a)
    b = np.asarray(b)
    assert a.shape == b.shape, f"{name}: shape {a.shape} vs {b.shape}"
    if a.dtype.kind == "f":
        a = a.view(np.uint32 if a.itemsize == 4 else np.uint16)
        b = b.view(a.dtype)
    bad = np.flatnonzero(a.reshape(-1) != b.reshape(-1))
    assert bad.size == 0, (f"{name}: {bad.size} of {a.size} differ; first at flat index "
                           f"{bad[:5].tolist()}: {a.reshape(-1)[bad[:5]].tolist()} vs "
                           f"{b.reshape(-1)[bad[:5]].tolist()}")


def compare_full(w, g, o):
    assert_same("cdf_anchor", g["ca"], o["ca"])
    assert_same("cdf_delta", g["cd"], o["cd"])
    assert_same("scales", g["scales"], o["scales"])
    assert_same("offsets", g["offsets"], o["offsets"])
    assert_same("words", g["words"], o["words"])
    assert_same("decoded fp16", g["out"], o["out"])
