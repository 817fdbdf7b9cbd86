"""GPU parity at the benchmark workloads' full sizes, in the launch configuration bench.py times.

Every workload runs in full on the GPU (fit of every level, encode, decode of the whole cache)
and every result is compared with the oracle: tables, scales, per-stream lengths and offsets,
payload words and decoded fp16 bit patterns. The Mistral-7B-shaped cache is compared in one
piece. For the three larger caches the oracle runs on slabs of consecutive layers, so that host
memory stays bounded: the streams of a layer depend only on that layer's values, its bin width
and the chunk levels, and the tables of a (layer, K/V, channel) only on that layer's values, so
a sub-cache holding layers [l0, l1) must reproduce the full run's tables, scales, stream words
and decoded rows of those layers bit for bit. Together the slabs cover every layer.
"""
import time

import numpy as np
import pytest

import oracle
from paper_2310_07240_amd import workloads as W
from gpu_helpers import assert_same, compare_full, run_gpu, run_oracle, say, torch_cuda

pytestmark = pytest.mark.gpu

SLAB_LAYERS = 8


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


def _gpu_full_run(w, kv_np):
    """Fit, encode and decode the whole cache on the GPU; every result back as numpy."""
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
    del kv
    say(f"{w.name}: decode")
    out = codec.decode(words, offsets, scales, cl, ca, cd)
    torch.cuda.synchronize()
    say(f"{w.name}: copy back")
    off = offsets.cpu().numpy().view(np.uint64)
    res = dict(ca=ca.cpu().numpy().view(np.uint16), cd=cd.cpu().numpy().view(np.uint16),
               offsets=off, scales=scales.cpu().numpy(),
               words=words[: int(off[-1])].cpu().numpy().view(np.uint32))
    res["out"] = out.cpu().numpy().view(np.uint16)
    del out, words, offsets, scales, ca, cd
    torch.cuda.empty_cache()
    return res


def _compare_slab(w, g, o, l0, l1):
    """The oracle's results on the sub-cache of layers [l0, l1) against the full GPU run."""
    B, NC, L, C = w.n_ctx, w.n_chunks, w.n_layers, w.n_channels
    Ls = l1 - l0
    tag = f"layers {l0}-{l1 - 1}"
    assert_same(f"cdf_anchor ({tag})", g["ca"][l0:l1], o["ca"])
    assert_same(f"cdf_delta ({tag})", g["cd"][:, l0:l1], o["cd"])
    assert_same(f"decoded fp16 ({tag})", g["out"][:, l0:l1], o["out"])
    goff, ooff = g["offsets"].astype(np.int64), o["offsets"].astype(np.int64)
    per = Ls * 2 * C                       # streams of one (context, chunk) in the slab
    for b in range(B):
        for c in range(NC):
            s_full = ((b * NC + c) * L + l0) * 2 * C
            s_sub = (b * NC + c) * per
            assert_same(f"stream lengths b{b} c{c} ({tag})",
                        np.diff(goff[s_full:s_full + per + 1]),
                        np.diff(ooff[s_sub:s_sub + per + 1]))
            assert_same(f"scales b{b} c{c} ({tag})", g["scales"][s_full:s_full + per],
                        o["scales"][s_sub:s_sub + per])
            assert_same(f"words b{b} c{c} ({tag})", g["words"][goff[s_full]:goff[s_full + per]],
                        o["words"][ooff[s_sub]:ooff[s_sub + per]])


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["llama2_7b_mha_t8192", "llama2_70b_gqa_t16384",
                                  "concurrency_32x_mistral_t2048"])
def test_large_workload_every_layer_bit_exact(name):
    w = W.WORKLOADS[name]
    t = time.time()
    kv = W.generate(w)
    say(f"{w.name}: generated in {time.time() - t:.1f}s")
    g = _gpu_full_run(w, kv)
    goff = g["offsets"]
    assert goff[0] == 0 and np.all(np.diff(goff.astype(np.int64)) > 0)
    covered = 0
    for l0 in range(0, w.n_layers, SLAB_LAYERS):
        l1 = min(w.n_layers, l0 + SLAB_LAYERS)
        sub = w.with_(name=f"{w.name}_layers_{l0}_{l1}", n_layers=l1 - l0,
                      layer_bin=tuple(w.layer_bin[l0:l1]))
        assert np.array_equal(sub.chunk_levels(), w.chunk_levels())
        kv_sub = np.ascontiguousarray(kv[:, l0:l1])
        o = run_oracle(sub, kv_sub)
        del kv_sub
        _compare_slab(w, g, o, l0, l1)
        covered += l1 - l0
        say(f"{w.name}: layers {l0}-{l1 - 1} bit-exact")
        del o
    assert covered == w.n_layers
    say(f"{w.name}: every layer bit-exact; bits/element {int(goff[-1]) * 32 / w.n_elem:.3f}")
