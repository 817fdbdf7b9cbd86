"""GPU parity: the HIP codec against the CPU oracle, bit for bit (tables, scales, offsets,
payload words, decoded fp16), on small seeded workloads that span several 64-channel blocks,
ragged chunks and groups, and the codec's degenerate inputs. Every test calls the C ABI."""
import numpy as np
import pytest

from paper_2310_07240_amd import workloads as W
from gpu_helpers import compare_full, run_gpu, run_oracle, say, assert_same, torch_cuda

pytestmark = pytest.mark.gpu

SMALL = [
    W.small(),                                                     # C=70: a ragged channel block
    W.small(name="c130_ctx2_heavy", n_ctx=2, n_tokens=61, chunk_len=20, n_channels=130,
            heavy_ctx=(1,)),
    W.small(name="g1_all_anchors", group_size=1, n_tokens=40, chunk_len=16),
    W.small(name="one_chunk", n_tokens=37, chunk_len=1536, level_mult=(1.0,), random_levels=False),
    W.small(name="l1_c1_t1", n_layers=1, n_channels=1, n_tokens=1, chunk_len=7),
    W.small(name="l1_c64_t23", n_layers=1, n_channels=64, n_tokens=23, chunk_len=7),
    W.small(name="g7_levels3", group_size=7, n_tokens=200, chunk_len=64, n_channels=96,
            level_mult=(1.0, 2.0, 4.0)),
    W.small(name="long_chunk_1536", n_layers=2, n_tokens=1600, chunk_len=1536, n_channels=65,
            level_mult=(1.0, 8.0)),
    # whole 64-channel blocks and the paper's 1536-token chunks: the fit's register path with
    # full halves (G = 10: 50 tokens per lane; G = 7: 49), and G = 64, which is too long for it
    W.small(name="c128_chunk_1536", n_layers=1, n_tokens=1600, chunk_len=1536, n_channels=128,
            level_mult=(1.0, 8.0)),
    W.small(name="c64_chunk_1536_g7", n_layers=1, n_tokens=1536, chunk_len=1536, n_channels=64,
            group_size=7),
    W.small(name="c64_chunk_1536_g64", n_layers=1, n_tokens=1536, chunk_len=1536, n_channels=64,
            group_size=64),
    # eight levels over sixteen chunks: a workgroup's worst-case table sets exceed the LDS of a
    # CU at sixteen waves, so the launchers use fewer waves per workgroup
    W.small(name="levels8_chunks16", n_layers=2, n_tokens=160, chunk_len=10, n_channels=64,
            level_mult=(1.0, 2.0, 4.0, 8.0, 16.0, 32.0, 64.0, 128.0)),
    W.small(name="levels8_chunks16_g7", n_layers=2, n_tokens=160, chunk_len=10, n_channels=64,
            group_size=7, level_mult=(1.0, 2.0, 4.0, 8.0, 16.0, 32.0, 64.0, 128.0)),
]


@pytest.mark.parametrize("w", SMALL, ids=lambda w: w.name)
def test_small_workloads_bit_exact(w):
    kv = W.generate(w)
    o = run_oracle(w, kv)
    g = run_gpu(w, kv, decode_oracle_payload=(o["words"], o["offsets"], o["scales"], o["ca"], o["cd"]))
    compare_full(w, g, o)
    assert_same("decode of oracle payload", g["out_from_oracle_payload"], o["out"])


# Every remainder of a chunk's token count modulo the group size of 10 (the decoder's last,
# partial group has its own code path): chunk lengths 12, 13, 15, 19 leave 2, 3, 5, 9 tokens,
# and the last chunks of these caches leave 1, 6, 7, 8 (0 and 4 come from the cases above).
TAILS = [
    W.small(name="tail_c12_t61", n_tokens=61, chunk_len=12, n_channels=64, n_layers=2),
    W.small(name="tail_c13_t45", n_tokens=45, chunk_len=13, n_channels=65, n_layers=2),
    W.small(name="tail_c15_t52", n_tokens=52, chunk_len=15, n_channels=64, n_layers=2),
    W.small(name="tail_c19_t46", n_tokens=46, chunk_len=19, n_channels=64, n_layers=2, n_ctx=2),
    # a last group of only its anchor after full groups (its q has no delta row to stay in)
    W.small(name="tail_c21_t63", n_tokens=63, chunk_len=21, n_channels=70, n_layers=2),
    W.small(name="tail_g7_c15_t57", group_size=7, n_tokens=57, chunk_len=15, n_channels=64,
            n_layers=2),
]


# Grids large enough for several (layer, K/V, channel block) units per workgroup: 512, 768 and
# 1024 units give 2, 3 and 4 units per workgroup in the encoder and the decoder; with 4 the
# encoder's absmax is shared by the four waves of a pair (channel-contiguous units).
UNITS = [
    W.small(name="units2_l8_c2048", n_layers=8, n_channels=2048, n_tokens=40, chunk_len=40),
    W.small(name="units3_l12_c2048", n_layers=12, n_channels=2048, n_tokens=30, chunk_len=30),
    W.small(name="units4_l16_c2048_2chunks", n_layers=16, n_channels=2048, n_tokens=47,
            chunk_len=25, level_mult=(1.0,), random_levels=False),   # one table set per unit
]


@pytest.mark.parametrize("w", UNITS, ids=lambda w: w.name)
def test_units_per_workgroup_bit_exact(w):
    kv = W.generate(w)
    o = run_oracle(w, kv)
    g = run_gpu(w, kv)
    compare_full(w, g, o)


@pytest.mark.parametrize("w", TAILS, ids=lambda w: w.name)
def test_group_tails_bit_exact(w):
    kv = W.generate(w)
    o = run_oracle(w, kv)
    g = run_gpu(w, kv)
    compare_full(w, g, o)


@pytest.mark.parametrize("kind", ["zeros", "constant", "subnormal", "ties", "clamp", "signs"])
def test_edge_inputs_bit_exact(kind):
    w = W.small(name=f"edge_{kind}", n_tokens=64, chunk_len=25, n_channels=80)
    kv = W.edge_case_kv(w, kind)
    o = run_oracle(w, kv)
    g = run_gpu(w, kv)
    compare_full(w, g, o)


def test_tiny_config_bit_exact():
    w = W.TINY
    kv = W.generate(w)
    o = run_oracle(w, kv)
    g = run_gpu(w, kv, decode_oracle_payload=(o["words"], o["offsets"], o["scales"], o["ca"], o["cd"]))
    compare_full(w, g, o)
    assert_same("decode of oracle payload", g["out_from_oracle_payload"], o["out"])


def test_chunk_range_decode_and_determinism():
    torch = torch_cuda()
    from paper_2310_07240_amd.cachegen import Codec, CodecParams
    w = W.small(name="ranges", n_ctx=2, n_tokens=130, chunk_len=40, n_channels=100)
    kv_np = W.generate(w)
    codec = Codec(CodecParams.of(w))
    kv = torch.from_numpy(kv_np.view(np.int16)).cuda()
    cl = torch.from_numpy(w.chunk_levels()).cuda()
    ca, cd = codec.fit(kv)
    words, offsets, scales = codec.encode(kv, cl, ca, cd)
    full = codec.decode(words, offsets, scales, cl, ca, cd).cpu().numpy()
    again = codec.decode(words, offsets, scales, cl, ca, cd).cpu().numpy()
    assert_same("decode twice", full, again)
    w2, o2, s2 = codec.encode(kv, cl, ca, cd, words=torch.empty_like(words))
    n = int(offsets[-1])
    assert_same("encode twice", w2[:n].cpu().numpy(), words[:n].cpu().numpy())
    for c0, c1 in [(0, 1), (1, 3), (3, 4), (2, 2)]:
        say(f"ranges: decode chunks [{c0}, {c1})")
        part = codec.decode(words, offsets, scales, cl, ca, cd, c0, c1).cpu().numpy()
        t0, t1 = c0 * w.chunk_len, min(c1 * w.chunk_len, w.n_tokens)
        assert_same(f"chunks {c0}:{c1}", part[..., t0:t1, :], full[..., t0:t1, :])
        mask = np.ones(w.n_tokens, bool)
        mask[t0:t1] = False
        assert np.all(part[..., mask, :] == 0)


@pytest.mark.parametrize("kind", ["random", "ones", "zeros"])
def test_corrupt_payload_decodes_within_bounds(kind):
    """The decoder's documented error behaviour: with valid tables and offsets, a corrupt
    payload gives wrong values but the decode finishes, stays in bounds (the tail after the
    payload is all it may read) and is deterministic; values are those of some symbols, so they
    stay finite. Both layouts."""
    torch = torch_cuda()
    from paper_2310_07240_amd.cachegen import Codec, CodecParams
    w = W.small(name=f"corrupt_{kind}", n_tokens=120, chunk_len=50, n_channels=70)
    codec = Codec(CodecParams.of(w))
    kv = torch.from_numpy(W.generate(w).view(np.int16)).cuda()
    cl = torch.from_numpy(w.chunk_levels()).cuda()
    ca, cd = codec.fit(kv)
    words, offsets, scales = codec.encode(kv, cl, ca, cd)
    twords, toffsets, tscales = codec.encode_tokens(kv, cl, ca, cd)
    rng = np.random.default_rng(5)
    for name, wds, off, sc, dec in (
            ("channel", words, offsets, scales,
             lambda x: codec.decode(x, offsets, scales, cl, ca, cd)),
            ("token", twords, toffsets, tscales,
             lambda x: codec.decode_tokens(x, toffsets, tscales, cl, ca, cd))):
        n = wds.numel()
        if kind == "random":
            bad = torch.from_numpy(rng.integers(0, 2**32, n, dtype=np.uint64).astype(np.uint32)
                                   .view(np.int32)).cuda()
        elif kind == "ones":
            bad = torch.full((n,), -1, dtype=torch.int32, device="cuda")
        else:
            bad = torch.zeros((n,), dtype=torch.int32, device="cuda")
        say(f"corrupt payload ({kind}), {name} layout")
        a = dec(bad).clone()
        b = dec(bad)
        torch.cuda.synchronize()
        assert torch.equal(a, b)
        assert bool(torch.isfinite(a.view(torch.float16).float()).all())


# Four levels over six chunks with enough (layer, K/V, channel block) units for two per
# workgroup: the group-of-10 decoder then stages the delta tables as windows of their 16-entry
# blocks (closed forms outside them). With heavy-tailed values the windows of one unit's four
# sets exceed the unit's LDS region and are staged in two rounds.
COMPACT = [
    W.small(name="compact_l4_c4096", n_layers=4, n_channels=4096, n_tokens=120, chunk_len=20,
            level_mult=(1.0, 2.0, 4.0, 8.0), seed=21),
    W.small(name="compact_heavy_rounds", n_layers=4, n_channels=4096, n_tokens=120,
            chunk_len=20, level_mult=(1.0, 2.0, 4.0, 8.0), heavy_ctx=(0,), seed=22),
    W.small(name="compact_c4100_tail", n_layers=4, n_channels=4100, n_tokens=117, chunk_len=20,
            level_mult=(1.0, 2.0, 4.0, 8.0), seed=23),
]
# the decoder's region per unit with two units of six 10-row waves: an LDS budget of 159 KB
# halved, less the rows (6 x 1280 B) and the window descriptors (4 sets x 64 x 4 B)
REGION_BYTES = 159 * 1024 // 2 - 6 * 1280 - 4 * 64 * 4


def _window_rounds(w, cd):
    """Staging rounds the windowed decoder needs per unit (computed from the oracle's tables the
    way the kernel lays them out), to show which cases exercise more than one round."""
    cum = cd.astype(np.int64).copy()
    cum[..., 255] = 65536
    nonflat = np.diff(cum, axis=-1) != 1                       # [lv, L, 2, C, 255]
    idx = np.arange(255)
    lo = np.where(nonflat, idx, 255).min(-1)
    hi = np.where(nonflat, idx, -1).max(-1)
    g0 = np.maximum(lo // 16 - 1, 0)
    g1 = np.minimum(hi // 16 + 1, 15)
    size = (g1 - g0 + 1) * 32 + 8
    levels = sorted(set(int(v) for v in w.chunk_levels().reshape(-1)))
    rounds = []
    for l in range(w.n_layers):
        for k in range(2):
            for cb in range(0, w.n_channels, 64):
                acc, r = 0, 0
                for lv in levels:
                    tot = int(size[lv, l, k, cb:cb + 64].sum())
                    if acc > 0 and acc + tot > REGION_BYTES:
                        r, acc = r + 1, 0
                    acc += tot
                rounds.append(r + 1)
    return max(rounds)


@pytest.mark.parametrize("w", COMPACT, ids=lambda w: w.name)
def test_windowed_delta_tables_bit_exact(w):
    kv = W.generate(w)
    o = run_oracle(w, kv)
    assert len(set(w.chunk_levels().reshape(-1).tolist())) > 1
    rounds = _window_rounds(w, o["cd"])
    say(f"{w.name}: windowed tables, {rounds} staging round(s)")
    if w.name == "compact_heavy_rounds":
        assert rounds > 1
    g = run_gpu(w, kv, decode_oracle_payload=(o["words"], o["offsets"], o["scales"], o["ca"], o["cd"]))
    compare_full(w, g, o)
    assert_same("decode of oracle payload", g["out_from_oracle_payload"], o["out"])


def test_windowed_tables_chunk_ranges():
    """Chunk-range decodes of a windowed case (fewer pairs per workgroup, other unit counts):
    each range equals the oracle's rows and leaves every other row untouched."""
    torch = torch_cuda()
    from paper_2310_07240_amd.cachegen import Codec, CodecParams
    w = COMPACT[1]
    kv_np = W.generate(w)
    o = run_oracle(w, kv_np)
    codec = Codec(CodecParams.of(w))
    kv = torch.from_numpy(kv_np.view(np.int16)).cuda()
    cl = torch.from_numpy(w.chunk_levels()).cuda()
    ca, cd = codec.fit(kv)
    words, offsets, scales = codec.encode(kv, cl, ca, cd)
    for c0, c1 in [(1, 5), (0, 3), (5, 6), (2, 6)]:
        say(f"{w.name}: decode chunks [{c0}, {c1})")
        part = codec.decode(words, offsets, scales, cl, ca, cd, c0, c1).cpu().numpy().view(np.uint16)
        t0, t1 = c0 * w.chunk_len, min(c1 * w.chunk_len, w.n_tokens)
        assert_same(f"chunks {c0}:{c1}", part[..., t0:t1, :], o["out"][..., t0:t1, :])
        mask = np.ones(w.n_tokens, bool)
        mask[t0:t1] = False
        assert np.all(part[..., mask, :] == 0)


FIT_CASES = [
    W.MISTRAL_7B_4K.with_(name="fit_mistral_l3", n_layers=3, layer_bin=(0.5, 1.0, 1.5)),
    W.small(name="fit_levels4_regs", n_layers=2, n_channels=128, n_tokens=1600, chunk_len=1536,
            level_mult=(1.0, 2.0, 4.0, 8.0)),
    W.small(name="fit_levels8_c70", n_layers=2, n_channels=70, n_tokens=300, chunk_len=64,
            level_mult=(1.0, 2.0, 4.0, 8.0, 16.0, 32.0, 64.0, 128.0)),
    W.small(name="fit_levels5_g7", group_size=7, n_layers=2, n_channels=64, n_tokens=200,
            chunk_len=50, level_mult=(1.0, 1.5, 2.0, 3.0, 5.0)),
    # 64-channel blocks, eight levels in two passes of four, three contexts; chunks of 7 groups
    # leave most of the 32 slices of a chunk empty, the last chunk has 5 tokens
    W.small(name="fit_levels8_b3_c128", n_ctx=3, n_layers=2, n_channels=128, n_tokens=205,
            chunk_len=64, level_mult=(1.0, 1.25, 1.5, 2.0, 3.0, 4.0, 6.0, 8.0)),
    # three levels in one pass; one level with another group size (the generic group loop)
    W.small(name="fit_levels3_c192", n_layers=2, n_channels=192, n_tokens=700, chunk_len=320,
            level_mult=(1.0, 2.0, 4.0)),
    W.small(name="fit_level1_g7_c128", group_size=7, n_layers=2, n_channels=128, n_tokens=500,
            chunk_len=200, level_mult=(1.0,)),
    # a chunk of 4 groups per slice and a ragged group inside the last slice
    W.small(name="fit_levels2_t2995", n_layers=1, n_channels=192, n_tokens=2995, chunk_len=1280,
            level_mult=(1.0, 2.0)),
    # five levels at G = 10: the second pass fits one level without the anchors (the one-read
    # kernel's with_anchor = 0 case)
    W.small(name="fit_levels5_g10_c128", n_layers=2, n_channels=128, n_tokens=700, chunk_len=320,
            level_mult=(1.0, 2.0, 4.0, 8.0, 16.0)),
    # 270 (block, layer, K/V) items, more than the one-read kernel's resident workgroups (one
    # per CU): some workgroups take two items, the next item's first slice loaded across
    W.small(name="fit_level1_items270", n_layers=3, n_channels=2880, n_tokens=300, chunk_len=128,
            level_mult=(1.0,)),
    # more than 2^16 deltas of one channel: the 32-bit per-level path
    W.small(name="fit_long_t76000", n_layers=1, n_channels=64, n_tokens=76000, chunk_len=1536,
            level_mult=(1.0, 4.0)),
]


@pytest.mark.parametrize("w", FIT_CASES, ids=lambda w: w.name)
def test_fit_all_levels_equals_oracle_and_per_level(w):
    """cg_fit_cdf_levels (every level in one call) against the oracle's per-level fit and
    against cg_fit_cdf level by level, bit for bit; its status word reports NaN."""
    torch = torch_cuda()
    import oracle
    from paper_2310_07240_amd.cachegen import Codec, CodecParams, cg_get_status
    kv_np = W.generate(w)
    oca, ocd = oracle.fit_all_levels(kv_np, oracle.shape_from(w))
    codec = Codec(CodecParams.of(w))
    kv = torch.from_numpy(kv_np.view(np.int16)).cuda()
    st = torch.full((1,), 7, dtype=torch.int32, device="cuda")
    ca, cd = codec.fit(kv, status=st)
    ca1, cd1 = codec.fit_per_level(kv)
    torch.cuda.synchronize()
    assert cg_get_status(st) == 0
    assert_same("anchor tables", ca.cpu().numpy().view(np.uint16), oca)
    assert_same("delta tables", cd.cpu().numpy().view(np.uint16), ocd)
    assert_same("per-level anchor tables", ca1.cpu().numpy(), ca.cpu().numpy())
    assert_same("per-level delta tables", cd1.cpu().numpy(), cd.cpu().numpy())
    bad = kv.clone()
    bad.view(-1)[bad.numel() // 3] = 0x7C00     # +Inf
    codec.fit(bad, status=st)
    assert cg_get_status(st) == -4


SCALE_CASES = [
    FIT_CASES[0],   # one level, 64-channel blocks
    W.small(name="scales_one_level_c70", n_tokens=37, chunk_len=1536, level_mult=(1.0,),
            random_levels=False),   # one level, ragged channels: the 32-bit fit kernel
    W.small(name="scales_levels8_c70", n_layers=2, n_channels=70, n_tokens=300, chunk_len=64,
            level_mult=(1.0, 2.0, 4.0, 8.0, 16.0, 32.0, 64.0, 128.0)),   # a lane per channel
    COMPACT[0],     # windowed delta tables in the encoder, coop absmax path in cg_encode
    FIT_CASES[-1],  # more than 2^16 deltas per channel: the per-level 32-bit path
]


@pytest.mark.parametrize("w", SCALE_CASES, ids=lambda w: w.name)
def test_fit_scales_feed_the_encoder(w):
    """cg_fit_cdf_levels' scales equal cg_encode's, and cg_encode_with_scales on them gives
    cg_encode's words and offsets, bit for bit."""
    torch = torch_cuda()
    from paper_2310_07240_amd.cachegen import Codec, CodecParams
    codec = Codec(CodecParams.of(w))
    kv_np = W.generate(w)
    o = run_oracle(w, kv_np)
    kv = torch.from_numpy(kv_np.view(np.int16)).cuda()
    cl = torch.from_numpy(w.chunk_levels()).cuda()
    sc = torch.full((codec.n_streams,), float("nan"), dtype=torch.float32, device="cuda")
    ca, cd = codec.fit(kv, scales=sc)
    assert_same("fit scales vs oracle", sc.cpu().numpy(), o["scales"])
    words, offsets, scales = codec.encode(kv, cl, ca, cd)
    assert codec.status() == 0
    assert_same("fit scales vs encode", sc.cpu().numpy(), scales.cpu().numpy())
    w2, o2 = codec.encode_with_scales(kv, cl, ca, cd, sc)
    assert codec.status() == 0
    n = int(offsets[-1].item())
    assert_same("offsets", o2.cpu().numpy().view(np.uint64), o["offsets"].view(np.uint64))
    assert_same("words", w2[:n].cpu().numpy().view(np.uint32), o["words"][:n].view(np.uint32))
