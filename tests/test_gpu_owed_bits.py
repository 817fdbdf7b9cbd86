"""GPU parity where the coder owes long runs of bits. The delta tables give q = 0 the two-count
interval centred on the midpoint of the range (every other symbol about 258 counts), and the
coarse levels quantize most deltas to 0: each such delta is one more middle-half straddle of
about 15 steps, so the owed bits pile up over a run of zeros and a following nonzero delta
emits more than 32 of them at once. That takes the encoder's branching path and its direct
output, and the stream ends with long runs of owed bits. Channel and token layouts, both
through the C ABI, bit for bit against the oracle under the same tables."""
import numpy as np
import pytest

import oracle
from paper_2310_07240_amd import workloads as W
from gpu_helpers import assert_same, say, torch_cuda

pytestmark = pytest.mark.gpu


def midpoint_table() -> np.ndarray:
    cum = np.zeros(256, np.uint16)
    cum[:128] = np.round(np.arange(128) * 32767 / 127).astype(np.uint16)        # cum[127] = 32767
    cum[128:255] = (32769 + np.round(np.arange(127) * 32767 / 127)).astype(np.uint16)
    return cum                                                                   # cum[255]: padding


CASES = [
    W.small(name="owed_c70", n_layers=2, n_tokens=300, chunk_len=150, n_channels=70,
            level_mult=(8.0, 32.0)),
    W.small(name="owed_c64_chunk1536", n_layers=1, n_tokens=1536, chunk_len=1536,
            n_channels=64, level_mult=(16.0,), random_levels=False),
]


@pytest.mark.parametrize("w", CASES, ids=lambda w: w.name)
def test_owed_bit_runs_bit_exact(w):
    torch = torch_cuda()
    from paper_2310_07240_amd.cachegen import Codec, CodecParams
    kv_np = W.generate(w)
    shape = oracle.shape_from(w)
    cl_np = w.chunk_levels()
    ca, cd = oracle.fit_all_levels(kv_np, shape)
    cd = np.broadcast_to(midpoint_table(), cd.shape).copy()
    t = np.diff(midpoint_table()[:255].astype(np.int64))
    assert t.min() >= 2 and midpoint_table()[127] == 32767 and midpoint_table()[128] == 32769

    codec = Codec(CodecParams.of(w))
    kv = torch.from_numpy(np.ascontiguousarray(kv_np).view(np.int16)).cuda()
    cl = torch.from_numpy(cl_np).cuda()
    tca = torch.from_numpy(np.ascontiguousarray(ca).view(np.int16)).cuda()
    tcd = torch.from_numpy(np.ascontiguousarray(cd).view(np.int16)).cuda()

    ow, oo, osc = oracle.encode(kv_np, shape, cl_np, ca, cd)
    oout = oracle.decode(ow, oo, osc, shape, cl_np, ca, cd)
    # the payload is far above the entropy of mostly-zero deltas: the owed runs are there
    bits = 32.0 * int(oo[-1]) / kv_np.size
    say(f"{w.name}: oracle payload {bits:.2f} bits/element")
    assert bits > 8.0
    say(f"{w.name}: channel-layout encode and decode")
    words, offsets, scales = codec.encode(kv, cl, tca, tcd)
    out = codec.decode(words, offsets, scales, cl, tca, tcd)
    torch.cuda.synchronize()
    off = offsets.cpu().numpy().view(np.uint64)
    assert_same("offsets", off, oo)
    assert_same("scales", scales.cpu().numpy(), osc)
    assert_same("words", words[:int(off[-1])].cpu().numpy().view(np.uint32), ow)
    assert_same("decoded fp16", out.cpu().numpy().view(np.uint16), oout)

    tw_, to_, ts_ = oracle.encode_tokens(kv_np, shape, cl_np, ca, cd)
    say(f"{w.name}: token-layout encode and decode")
    words, offsets, scales = codec.encode_tokens(kv, cl, tca, tcd)
    out = codec.decode_tokens(words, offsets, scales, cl, tca, tcd)
    torch.cuda.synchronize()
    off = offsets.cpu().numpy().view(np.uint64)
    assert_same("token offsets", off, to_)
    assert_same("token words", words[:int(off[-1])].cpu().numpy().view(np.uint32), tw_)
    assert_same("token-layout decoded fp16", out.cpu().numpy().view(np.uint16), oout)
