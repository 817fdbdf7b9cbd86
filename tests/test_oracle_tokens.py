"""Pins of the oracle's token-parallel layout (CacheGen Sec. 6: the decoder runs one thread per
token). The layout groups the same quantized symbols differently: one stream per (context,
layer, K/V, token) over the token's channels, each symbol under its channel's table. So:

* its decode equals the channel-layout decode of the same cache, bit for bit;
* every token stream, decoded on its own with the generic coder and the tables the layout names
  (anchor table on a group's first token, the chunk level's delta table otherwise), returns the
  quantizer's symbols of that token row, built here from the channel streams one by one;
* its scales are the channel streams' scales (same side information);
* every stream's length is within the coder's 2-bit termination of the ideal length."""
import math

import numpy as np
import pytest

import oracle
from paper_2310_07240_amd import workloads as W

CASES = [
    W.small(),
    W.small(name="ctx2_heavy", n_ctx=2, n_tokens=61, chunk_len=20, n_channels=33, heavy_ctx=(1,)),
    W.small(name="g1", group_size=1, n_tokens=40, chunk_len=16),
    W.small(name="g7_levels3", group_size=7, n_tokens=90, chunk_len=32, n_channels=40,
            level_mult=(1.0, 2.0, 4.0)),
    W.small(name="l1_c1", n_layers=1, n_channels=1, n_tokens=23, chunk_len=7),
]


def _setup(w):
    kv = W.generate(w)
    shape = oracle.shape_from(w)
    ca, cd = oracle.fit_all_levels(kv, shape, 4)
    cl = w.chunk_levels()
    return kv, shape, ca, cd, cl


def _symbol_cube(kv, shape, cl):
    """Quantizer symbols [B, L, 2, T, C] assembled from the channel streams one by one."""
    sym = np.zeros(shape.kv_shape(), np.uint8)
    C, L, NC = shape.n_channels, shape.n_layers, shape.n_chunks
    for s in range(shape.n_streams):
        _, ss, _ = oracle.stream_symbols(kv, shape, cl, s)
        ch = s % C; r = s // C; k = r % 2; r //= 2; l = r % L; r //= L; c = r % NC; b = r // NC
        t0 = c * shape.chunk_len
        sym[b, l, k, t0:t0 + ss.size, ch] = ss
    return sym


def _token_streams(shape):
    """(b, c, l, k, t) of every token stream, in stream order."""
    out = []
    for b in range(shape.n_ctx):
        for c in range(shape.n_chunks):
            t0 = c * shape.chunk_len
            n = min(shape.chunk_len, shape.n_tokens - t0)
            for l in range(shape.n_layers):
                for k in range(2):
                    for j in range(n):
                        out.append((b, c, l, k, t0 + j))
    return out


@pytest.mark.parametrize("w", CASES, ids=lambda w: w.name)
def test_token_layout_decode_equals_channel_layout(w):
    kv, shape, ca, cd, cl = _setup(w)
    words, offsets, scales = oracle.encode(kv, shape, cl, ca, cd, 4)
    ref = oracle.decode(words, offsets, scales, shape, cl, ca, cd, threads=4)
    tw, toff, tsc = oracle.encode_tokens(kv, shape, cl, ca, cd, 4)
    assert np.array_equal(tsc, scales)
    assert toff.size == oracle.n_token_streams(shape) + 1
    assert np.all(np.diff(toff.astype(np.int64)) >= 1)
    out = oracle.decode_tokens(tw, toff, tsc, shape, cl, ca, cd, 4)
    assert np.array_equal(out, ref)


@pytest.mark.parametrize("w", CASES, ids=lambda w: w.name)
def test_each_token_stream_holds_its_row(w):
    kv, shape, ca, cd, cl = _setup(w)
    cube = _symbol_cube(kv, shape, cl)
    tw, toff, _ = oracle.encode_tokens(kv, shape, cl, ca, cd, 4)
    cl2 = np.asarray(cl, np.uint8).reshape(shape.n_ctx, shape.n_chunks)
    streams = _token_streams(shape)
    assert len(streams) == oracle.n_token_streams(shape)
    for s, (b, c, l, k, t) in enumerate(streams):
        lv = min(int(cl2[b, c]), shape.n_levels - 1)
        anchor = (t - c * shape.chunk_len) % shape.group_size == 0
        tabs = [ca[l, k, ch] if anchor else cd[lv, l, k, ch] for ch in range(shape.n_channels)]
        got = oracle.ac_decode(tw[int(toff[s]):int(toff[s + 1])], shape.n_channels, tabs)
        assert np.array_equal(got, cube[b, l, k, t]), (s, b, c, l, k, t)
        # length: at least the ideal code length, at most that plus the 2-bit termination
        # (and the coder's 1e-4 per symbol of integer rounding), padded to a word
        row = cube[b, l, k, t].astype(np.int64)
        p = np.array([(oracle.cum32(tabs[ch])[row[ch] + 1] - oracle.cum32(tabs[ch])[row[ch]])
                      / 65536.0 for ch in range(shape.n_channels)])
        ideal = float(-np.log2(p).sum())
        nw = int(toff[s + 1] - toff[s])
        assert nw * 32 >= ideal - 1.0, (s, nw, ideal)
        assert nw <= math.ceil((ideal + 2.0 + 1e-4 * shape.n_channels) / 32.0), (s, nw, ideal)
