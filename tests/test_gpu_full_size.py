"""GPU parity at the benchmark workloads' full sizes, in the launch configuration bench.py times.

The Mistral-7B-shaped cache (268M elements) is compared in full. The three larger caches run in
full on the GPU; the oracle recomputes every stream of three sampled layers (first, middle and
last: one per layer group) from a sub-cache holding only those layers. Streams of a layer depend
only on that layer's slab, its bin width and the chunk levels, so the sub-cache's streams, tables
and decoded values must equal the full run's, bit for bit.
"""
import time

import numpy as np
import pytest

import oracle
from paper_2310_07240_amd import workloads as W
from gpu_helpers import assert_same, compare_full, run_gpu, run_oracle, say, torch_cuda

pytestmark = pytest.mark.gpu


@pytest.mark.timeout(600)
def test_mistral7b_4k_full_bit_exact():
    w = W.MISTRAL_7B_4K
    t = time.time()
    kv = W.generate(w)
    say(f"{w.name}: generated in {time.time() - t:.1f}s")
    g = run_gpu(w, kv)
    o = run_oracle(w, kv)
    compare_full(w, g, o)
    say(f"{w.name}: bits/element {g['words'].size * 32 / w.n_elem:.3f}")


def _gpu_full_run(w, kv_np, layers):
    torch = torch_cuda()
    from paper_2310_07240_amd.cachegen import Codec, CodecParams
    codec = Codec(CodecParams.of(w))
    say(f"{w.name}: upload {kv_np.nbytes / 2**30:.2f} GiB")
    kv = torch.from_numpy(kv_np.view(np.int16)).cuda()
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
    del kv
    say(f"{w.name}: copy back")
    off = offsets.cpu().numpy().view(np.uint64)
    idx = torch.tensor(layers, device=out.device)
    res = dict(ca=ca[idx].cpu().numpy().view(np.uint16),
               cd=cd[:, idx].cpu().numpy().view(np.uint16),
               offsets=off, scales=scales.cpu().numpy(),
               words=words[: int(off[-1])].cpu().numpy().view(np.uint32),
               out=out[:, idx].cpu().numpy().view(np.uint16))
    del out, words
    torch.cuda.empty_cache()
    return res


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["llama2_7b_mha_t8192", "llama2_70b_gqa_t16384",
                                  "concurrency_32x_mistral_t2048"])
def test_large_workload_sampled_layers_bit_exact(name):
    w = W.WORKLOADS[name]
    layers = [0, w.n_layers // 2, w.n_layers - 1]
    t = time.time()
    kv = W.generate(w)
    say(f"{w.name}: generated in {time.time() - t:.1f}s")
    g = _gpu_full_run(w, kv, layers)
    sub = w.with_(name=w.name + "_sampled_layers", n_layers=len(layers),
                  layer_bin=tuple(w.layer_bin[l] for l in layers))
    kv_sub = np.ascontiguousarray(kv[:, layers])
    del kv
    o = run_oracle(sub, kv_sub)
    assert np.array_equal(sub.chunk_levels(), w.chunk_levels())
    assert_same("cdf_anchor (sampled layers)", g["ca"], o["ca"])
    assert_same("cdf_delta (sampled layers)", g["cd"], o["cd"])
    assert_same("decoded fp16 (sampled layers)", g["out"], o["out"])
    B, NC, L, C = w.n_ctx, w.n_chunks, w.n_layers, w.n_channels
    goff, ooff = g["offsets"].astype(np.int64), o["offsets"].astype(np.int64)
    for b in range(B):
        for c in range(NC):
            for li, l in enumerate(layers):
                for k in range(2):
                    s_full = (((b * NC + c) * L + l) * 2 + k) * C
                    s_sub = (((b * NC + c) * len(layers) + li) * 2 + k) * C
                    assert_same("stream lengths", np.diff(goff[s_full:s_full + C + 1]),
                                np.diff(ooff[s_sub:s_sub + C + 1]))
                    assert_same("scales", g["scales"][s_full:s_full + C], o["scales"][s_sub:s_sub + C])
                    assert_same(f"words b{b} c{c} l{l} k{k}",
                                g["words"][goff[s_full]:goff[s_full + C]],
                                o["words"][ooff[s_sub]:ooff[s_sub + C]])
    total_bits = int(goff[-1]) * 32
    say(f"{w.name}: bits/element {total_bits / w.n_elem:.3f}")
