"""GPU: cg_encode_noalloc, the encoder for callers that cannot allocate device memory, against
cg_encode through the C ABI: identical payload words, offsets, scales and status on two calls
in a row (the second with a smaller cache, so the shared static scratch holds the first call's
contents), plus the rejection of a cache whose scratch exceeds the static buffer."""
import ctypes

import numpy as np
import pytest

from paper_2310_07240_amd import workloads as W
from gpu_helpers import assert_same, say, torch_cuda

pytestmark = pytest.mark.gpu


def _inputs(torch, w):
    from paper_2310_07240_amd.cachegen import Codec, CodecParams
    codec = Codec(CodecParams.of(w))
    kv = torch.from_numpy(W.generate(w).view(np.int16)).cuda()
    cl = torch.from_numpy(w.chunk_levels()).cuda()
    ca, cd = codec.fit(kv)
    return codec, kv, cl, ca, cd


def _encode_both(torch, codec, kv, cl, ca, cd):
    from paper_2310_07240_amd.cachegen import cg_encode, cg_encode_noalloc
    p = codec.p
    n = codec.bound_words
    S = codec.n_streams
    w_ref = torch.zeros(n, dtype=torch.int32, device="cuda")
    o_ref = torch.zeros(S + 1, dtype=torch.int64, device="cuda")
    s_ref = torch.zeros(S, dtype=torch.float32, device="cuda")
    ws = torch.empty(codec.ws_bytes, dtype=torch.uint8, device="cuda")
    cg_encode(p, kv, cl, ca, cd, w_ref, o_ref, s_ref, ws)
    w_na = torch.full((n,), 0x5A5A5A5A, dtype=torch.int32, device="cuda")
    o_na = torch.full((S + 1,), -1, dtype=torch.int64, device="cuda")
    s_na = torch.full((S,), -1.0, dtype=torch.float32, device="cuda")
    st = torch.full((1,), 7, dtype=torch.int32, device="cuda")
    cg_encode_noalloc(p, kv, cl, ca, cd, w_na, o_na, s_na, st)
    torch.cuda.synchronize()
    off = o_ref.cpu().numpy()
    total = int(off[-1])
    assert_same("offsets", o_na.cpu().numpy(), off)
    assert_same("scales", s_na.cpu().numpy(), s_ref.cpu().numpy())
    assert_same("words", w_na[:total].cpu().numpy(), w_ref[:total].cpu().numpy())
    from paper_2310_07240_amd.cachegen import cg_get_status
    return int(st.item()), cg_get_status(ws)


def test_noalloc_encode_equals_encode_on_two_calls():
    torch = torch_cuda()
    first = W.TINY
    second = W.small(name="noalloc_second", n_layers=2, n_tokens=61, chunk_len=25,
                     n_channels=70)
    assert first.n_elem > second.n_elem
    for w in (first, second):
        say(f"noalloc: {w.name}")
        codec, kv, cl, ca, cd = _inputs(torch, w)
        st, ref_status = _encode_both(torch, codec, kv, cl, ca, cd)
        assert st == 0 and ref_status == 0


def test_noalloc_reports_nonfinite_and_rejects_oversized():
    torch = torch_cuda()
    from paper_2310_07240_amd import cachegen as cg
    w = W.small(name="noalloc_nan", n_layers=2, n_tokens=61, chunk_len=25, n_channels=70)
    codec, kv, cl, ca, cd = _inputs(torch, w)
    bad = kv.clone()
    bad.view(-1)[1234] = 0x7E00      # NaN
    st, ref_status = _encode_both(torch, codec, bad, cl, ca, cd)
    assert st != 0 and ref_status == -4
    # a cache whose scratch exceeds the static buffer: rejected on the host, nothing launched
    big = cg.CodecParams.of(W.MISTRAL_7B_4K)
    assert cg.cg_encode_workspace_bytes(big) > cg.CG_NOALLOC_SCRATCH_BYTES
    s, keep = big.c()
    fake = ctypes.c_void_p(1 << 20)
    rc = cg.lib().cg_encode_noalloc(ctypes.byref(s), fake, fake, fake, fake, fake,
                                    cg.cg_encode_bound_words(big), fake, fake, None, None)
    assert rc == -7
    assert "static buffer" in cg.strerror(-7)
