"""GPU parity of the token-parallel stream layout (CacheGen Sec. 6: one decoder thread per
token) against the oracle, bit for bit: payload words, offsets, scales and decoded fp16, on the
same seeded inputs and the same tables (the oracle's fit, which the channel-layout tests pin to
the GPU fit). The decoded cache must also equal the channel-layout decode. Every call goes
through the C ABI (cg_encode_tokens, cg_decode_tokens)."""
import time

import numpy as np
import pytest

import oracle
from paper_2310_07240_amd import workloads as W
from gpu_helpers import assert_same, say, torch_cuda

pytestmark = pytest.mark.gpu

CASES = [
    W.small(),                                                     # C=70: a ragged 64-channel block
    W.small(name="tok_c130_ctx2_heavy", n_ctx=2, n_tokens=61, chunk_len=20, n_channels=130,
            heavy_ctx=(1,)),
    W.small(name="tok_g1", group_size=1, n_tokens=40, chunk_len=16),
    W.small(name="tok_l1_c1_t1", n_layers=1, n_channels=1, n_tokens=1, chunk_len=7),
    W.small(name="tok_g7_levels3", group_size=7, n_tokens=200, chunk_len=64, n_channels=96,
            level_mult=(1.0, 2.0, 4.0)),
    # 150 tokens per chunk: three 64-token blocks, the last one partial
    W.small(name="tok_chunk150_c64", n_layers=2, n_tokens=300, chunk_len=150, n_channels=64),
    W.small(name="tok_c128_chunk1536", n_layers=1, n_tokens=1600, chunk_len=1536,
            n_channels=128, level_mult=(1.0, 8.0)),
    # groups longer than a 64-token block: some blocks hold no anchor token at all
    W.small(name="tok_g100", group_size=100, n_tokens=250, chunk_len=200, n_channels=64),
]


def _run(w, kv_np):
    torch = torch_cuda()
    from paper_2310_07240_amd.cachegen import Codec, CodecParams
    shape = oracle.shape_from(w)
    cl_np = w.chunk_levels()
    t = time.time()
    ca, cd = oracle.fit_all_levels(kv_np, shape)
    ow, oo, osc = oracle.encode_tokens(kv_np, shape, cl_np, ca, cd)
    oout = oracle.decode_tokens(ow, oo, osc, shape, cl_np, ca, cd)
    cw, co, cs = oracle.encode(kv_np, shape, cl_np, ca, cd)
    cout = oracle.decode(cw, co, cs, shape, cl_np, ca, cd)
    say(f"{w.name}: oracle {time.time() - t:.1f}s")
    assert_same("oracle: token layout vs channel layout decode", oout, cout)

    codec = Codec(CodecParams.of(w))
    kv = torch.from_numpy(np.ascontiguousarray(kv_np).view(np.int16)).cuda()
    cl = torch.from_numpy(cl_np).cuda()
    tca = torch.from_numpy(np.ascontiguousarray(ca).view(np.int16)).cuda()
    tcd = torch.from_numpy(np.ascontiguousarray(cd).view(np.int16)).cuda()
    say(f"{w.name}: token-layout encode")
    words, offsets, scales = codec.encode_tokens(kv, cl, tca, tcd)
    torch.cuda.synchronize()
    say(f"{w.name}: token-layout decode")
    out = codec.decode_tokens(words, offsets, scales, cl, tca, tcd)
    torch.cuda.synchronize()
    off = offsets.cpu().numpy().view(np.uint64)
    total = int(off[-1])
    assert_same("offsets", off, oo)
    assert_same("scales", scales.cpu().numpy(), osc)
    assert_same("words", words[:total].cpu().numpy().view(np.uint32), ow)
    assert_same("decoded fp16", out.cpu().numpy().view(np.uint16), oout)
    say(f"{w.name}: decode the oracle's payload")
    padded = np.concatenate([np.asarray(ow, np.uint32), np.zeros(8, np.uint32)])
    tw = torch.from_numpy(padded.view(np.int32)).cuda()
    to = torch.from_numpy(np.ascontiguousarray(oo).view(np.int64)).cuda()
    ts = torch.from_numpy(np.ascontiguousarray(osc)).cuda()
    o2 = codec.decode_tokens(tw, to, ts, cl, tca, tcd)
    torch.cuda.synchronize()
    assert_same("decode of the oracle's payload", o2.cpu().numpy().view(np.uint16), oout)
    return words, total


@pytest.mark.parametrize("w", CASES, ids=lambda w: w.name)
def test_token_layout_bit_exact(w):
    _run(w, W.generate(w))


@pytest.mark.timeout(600)
def test_token_layout_mistral7b_4k_full_bit_exact():
    w = W.MISTRAL_7B_4K
    kv = W.generate(w)
    _, total = _run(w, kv)
    say(f"{w.name}: token layout {total * 32 / w.n_elem:.4f} payload bits/element")
