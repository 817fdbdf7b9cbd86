"""GPU: the one-global-distribution fit (cg_fit_cdf_global, the ablation baseline) equals the
oracle's pooled fit bit for bit, and a cache coded with it round-trips exactly as the oracle
codes it. Calls go through the C ABI."""
import numpy as np
import pytest

import oracle
from paper_2310_07240_amd import workloads as W
from gpu_helpers import assert_same, say, torch_cuda

pytestmark = pytest.mark.gpu

CASES = [
    W.small(name="global_c70", n_ctx=2, n_tokens=100, chunk_len=48, n_channels=70),
    W.small(name="global_g7_c130", group_size=7, n_tokens=61, chunk_len=20, n_channels=130,
            level_mult=(1.0, 2.0, 4.0)),
]


@pytest.mark.parametrize("w", CASES, ids=lambda w: w.name)
def test_global_fit_and_round_trip_bit_exact(w):
    torch = torch_cuda()
    from paper_2310_07240_amd.cachegen import (CG_FIT_GLOBAL_WORKSPACE_BYTES, Codec, CodecParams,
                                               cg_fit_cdf_global)
    kv_np = W.generate(w)
    shape = oracle.shape_from(w)
    codec = Codec(CodecParams.of(w))
    kv = torch.from_numpy(kv_np.view(np.int16)).cuda()
    L, C, NLV = w.n_layers, w.n_channels, len(w.level_mult)
    ca = torch.full((L, 2, C, 256), -1, dtype=torch.int16, device="cuda")
    cd = torch.full((NLV, L, 2, C, 256), -1, dtype=torch.int16, device="cuda")
    ws = torch.full((CG_FIT_GLOBAL_WORKSPACE_BYTES,), 0x5A, dtype=torch.uint8, device="cuda")
    for lv in range(NLV):
        say(f"{w.name}: global fit level {lv}")
        cg_fit_cdf_global(codec.p, kv, lv, ca if lv == 0 else None, cd[lv], ws)
    torch.cuda.synchronize()
    oa = None
    od = np.zeros((NLV, L, 2, C, 256), np.uint16)
    for lv in range(NLV):
        a, d = oracle.fit_cdf_global(kv_np, shape, lv)
        oa = a if lv == 0 else oa
        od[lv] = d
    assert_same("global anchor tables", ca.cpu().numpy().view(np.uint16), oa)
    assert_same("global delta tables", cd.cpu().numpy().view(np.uint16), od)
    cl_np = w.chunk_levels()
    cl = torch.from_numpy(cl_np).cuda()
    say(f"{w.name}: encode / decode with the global tables")
    words, offsets, scales = codec.encode(kv, cl, ca, cd)
    out = codec.decode(words, offsets, scales, cl, ca, cd)
    torch.cuda.synchronize()
    ow, oo, osc = oracle.encode(kv_np, shape, cl_np, oa, od)
    off = offsets.cpu().numpy().view(np.uint64)
    assert_same("offsets", off, oo)
    assert_same("words", words[:int(off[-1])].cpu().numpy().view(np.uint32), ow)
    oout = oracle.decode(ow, oo, osc, shape, cl_np, oa, od)
    assert_same("decoded fp16", out.cpu().numpy().view(np.uint16), oout)


def test_global_fit_rejects_a_small_workspace():
    torch = torch_cuda()
    from paper_2310_07240_amd.cachegen import CodecError, CodecParams, cg_fit_cdf_global
    w = W.small(name="global_ws")
    p = CodecParams.of(w)
    kv = torch.zeros(w.kv_shape, dtype=torch.int16, device="cuda")
    cd = torch.zeros((w.n_layers, 2, w.n_channels, 256), dtype=torch.int16, device="cuda")
    ws = torch.zeros((1024,), dtype=torch.uint8, device="cuda")
    with pytest.raises(CodecError):
        cg_fit_cdf_global(p, kv, 0, None, cd, ws)
