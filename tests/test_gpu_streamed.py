"""GPU: decoding chunk by chunk while the payload arrives (cg_decode_streamed) gives exactly the
oracle's decode, unthrottled and over a slow simulated link, and its timings are consistent.
Calls go through the C ABI."""
import numpy as np
import pytest

from paper_2310_07240_amd import workloads as W
from gpu_helpers import assert_same, run_oracle, say, torch_cuda

pytestmark = pytest.mark.gpu

CG_TAIL_WORDS = 8


def _setup(w):
    torch = torch_cuda()
    from paper_2310_07240_amd.cachegen import Codec, CodecParams
    codec = Codec(CodecParams.of(w))
    kv_np = W.generate(w)
    kv = torch.from_numpy(kv_np.view(np.int16)).cuda()
    cl = torch.from_numpy(w.chunk_levels()).cuda()
    ca, cd = codec.fit(kv)
    words, offsets, scales = codec.encode(kv, cl, ca, cd)
    torch.cuda.synchronize()
    return torch, codec, kv_np, cl, ca, cd, words, offsets, scales


@pytest.mark.parametrize("link_gbps", [0.0, 0.02])
def test_streamed_decode_equals_oracle(link_gbps):
    w = W.small(name="streamed", n_ctx=2, n_tokens=130, chunk_len=40, n_channels=100)
    torch, codec, kv_np, cl, ca, cd, words, offsets, scales = _setup(w)
    from paper_2310_07240_amd.cachegen import cg_decode_streamed
    off_host = offsets.cpu()
    total = int(off_host[-1])
    words_host = torch.empty((total + CG_TAIL_WORDS,), dtype=torch.int32, pin_memory=True)
    words_host.copy_(words[:total + CG_TAIL_WORDS].cpu())
    words_dev = torch.zeros((total + CG_TAIL_WORDS,), dtype=torch.int32, device="cuda")
    out = torch.zeros(w.kv_shape, dtype=torch.int16, device="cuda")
    dec_s, copy_s = torch.cuda.Stream(), torch.cuda.Stream()
    say(f"streamed decode, link {link_gbps} Gb/s, {total} words")
    st = cg_decode_streamed(codec.p, words_host, off_host, words_dev, offsets, scales, cl, ca, cd,
                            out, link_gbps, dec_s, copy_s)
    say(f"stats {st}")
    o = run_oracle(w, kv_np)
    assert_same("streamed decode", out.cpu().numpy().view(np.uint16), o["out"])
    assert st["n_chunks"] == codec.n_chunks == 4
    assert 0.0 <= st["transfer_ms"] <= st["total_ms"]
    assert st["decode_sum_ms"] > 0.0 and 0.0 <= st["hidden_fraction"] <= 1.0
    _check_event_order(st)
    if link_gbps > 0:
        link_ms = total * 32 / (link_gbps * 1e6)
        assert st["transfer_ms"] >= 0.9 * link_ms
        # overlap by event order: every chunk but the last is decoded before the next chunk's
        # payload has arrived (the link is far slower than a chunk's decode)
        for c in range(st["n_chunks"] - 1):
            assert st["chunk_decode_end_ms"][c] <= st["chunk_copy_done_ms"][c + 1]


def _check_event_order(st):
    """Per chunk: its decode starts after its payload is on the device and ends after it
    starts; decodes run in chunk order; the totals match the per-chunk times."""
    nc = st["n_chunks"]
    cp, db, de = st["chunk_copy_done_ms"], st["chunk_decode_begin_ms"], st["chunk_decode_end_ms"]
    for c in range(nc):
        assert cp[c] <= db[c] + 1e-3 <= de[c] + 2e-3
        if c:
            assert cp[c - 1] <= cp[c] + 1e-3 and de[c - 1] <= db[c] + 1e-3
    assert abs(st["transfer_ms"] - cp[-1]) < 1e-3 and abs(st["total_ms"] - de[-1]) < 1e-3
    assert abs(st["decode_sum_ms"] - sum(de[c] - db[c] for c in range(nc))) < 1e-2


@pytest.mark.timeout(300)
def test_streamed_decode_overlaps_at_mistral_size():
    """The Mistral-7B-shaped 4K cache (three chunks, 158 MB payload) arriving over the
    host-to-device bus: decoding chunk c starts before chunk c + 1's payload has arrived, so only
    the last chunk's decode remains after the transfer; the result equals cg_decode's."""
    w = W.MISTRAL_7B_4K
    torch, codec, kv_np, cl, ca, cd, words, offsets, scales = _setup(w)
    from paper_2310_07240_amd.cachegen import cg_decode_streamed
    ref = codec.decode(words, offsets, scales, cl, ca, cd)
    off_host = offsets.cpu()
    total = int(off_host[-1])
    words_host = torch.empty((total + CG_TAIL_WORDS,), dtype=torch.int32, pin_memory=True)
    words_host.copy_(words[:total + CG_TAIL_WORDS].cpu())
    words_dev = torch.zeros((total + CG_TAIL_WORDS,), dtype=torch.int32, device="cuda")
    out = torch.zeros(w.kv_shape, dtype=torch.int16, device="cuda")
    dec_s, copy_s = torch.cuda.Stream(), torch.cuda.Stream()
    args = (codec.p, words_host, off_host, words_dev, offsets, scales, cl, ca, cd, out, 0.0,
            dec_s, copy_s)
    cg_decode_streamed(*args)   # warm-up
    out.zero_()
    st = cg_decode_streamed(*args)
    say(f"mistral streamed: {st}")
    assert torch.equal(out, ref)
    _check_event_order(st)
    assert st["n_chunks"] == 3
    for c in range(2):
        assert st["chunk_decode_begin_ms"][c] < st["chunk_copy_done_ms"][c + 1]
    # what remains after the last byte is about one chunk's decode, not the whole decode
    exposed = st["total_ms"] - st["transfer_ms"]
    assert exposed <= 1.25 * (st["chunk_decode_end_ms"][2] - st["chunk_decode_begin_ms"][2]) + 0.05
    assert st["hidden_fraction"] >= 0.5


def test_streamed_decode_rejects_bad_arguments():
    torch = torch_cuda()
    from paper_2310_07240_amd.cachegen import CodecError, CodecParams, cg_decode_streamed
    w = W.small(name="streamed_args", n_tokens=20, chunk_len=10)
    p = CodecParams.of(w)
    x = torch.zeros(16, dtype=torch.int64, device="cuda")
    s = torch.cuda.current_stream()
    with pytest.raises(CodecError):
        cg_decode_streamed(p, None, x.cpu(), x, x, x, x, x, x, x, 0.0, s, s)
