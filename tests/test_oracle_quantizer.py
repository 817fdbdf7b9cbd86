"""Pins of the oracle's quantizer and fp16 conversions (CacheGen Sec. 5.2 "Change-based
encoding" and "Layer-wise quantization"), against library routines and closed forms."""
import numpy as np
import pytest

import oracle


def test_half_to_float_all_patterns_match_numpy():
    lib = oracle._lib()
    bits = np.arange(65536, dtype=np.uint16)
    ref = bits.view(np.float16).astype(np.float32)
    got = np.array([lib.cgo_half_to_float(int(b)) for b in bits], np.float32)
    finite = np.isfinite(ref)
    assert np.array_equal(got[finite].view(np.uint32), ref[finite].view(np.uint32))
    assert np.array_equal(np.isnan(got), np.isnan(ref))
    assert np.array_equal(got[np.isinf(ref)], ref[np.isinf(ref)])


def test_float_to_half_matches_numpy_rne():
    lib = oracle._lib()
    rng = np.random.default_rng(0)
    # random bit patterns across the whole float32 range plus every halfway point between
    # adjacent fp16 values (the ties) and their neighbours
    raw = rng.integers(0, 2**32, size=200_000, dtype=np.uint64).astype(np.uint32).view(np.float32)
    h = np.arange(0, 0x7c00, dtype=np.uint16).view(np.float16).astype(np.float64)
    mids = ((h[:-1] + h[1:]) / 2).astype(np.float32)           # exact in fp32
    near = np.concatenate([mids, np.nextafter(mids, np.float32(np.inf)),
                           np.nextafter(mids, np.float32(0))])
    vals = np.concatenate([raw, near, -near, np.float32([65504, 65519.99, 65520, 1e-8, 0.0,
                                                         -0.0, 2.0**-24, 2.0**-25, 3 * 2.0**-26])])
    vals = vals[~np.isnan(vals)]
    ref = vals.astype(np.float16).view(np.uint16)
    got = np.array([lib.cgo_float_to_half(float(v)) for v in vals], np.uint16)
    bad = np.nonzero(got != ref)[0]
    assert bad.size == 0, [(float(vals[i]), hex(got[i]), hex(ref[i])) for i in bad[:5]]



def test_anchor_value_has_no_double_rounding_hazard():
    """An anchor reconstructs as fp16(fp32(q * s)) with s = fp32(m / 127), m an fp16 magnitude
    (Sec. 5.2, vectorwise 8-bit anchors). For every finite m and every q in [-127, 127] this
    equals the single rounding of the exact product q * s to fp16: q * m / 127 lies at least
    2^-18 (relative) from every fp16 midpoint while fp32 rounding moves it by at most 2^-24, so
    a GPU instruction that converts the exact product to fp16 in one step gives the same bits."""
    m = np.arange(0, 0x7c00, dtype=np.uint16).view(np.float16).astype(np.float32)
    s = (m / np.float32(127)).astype(np.float32)
    s[m == 0] = 1.0
    q = np.arange(-127, 128, dtype=np.float64)
    for i in range(0, s.size, 4096):
        exact = s[i:i + 4096].astype(np.float64)[:, None] * q[None, :]   # exact: <= 31 bits
        twice = exact.astype(np.float32).astype(np.float16).view(np.uint16)
        once = exact.astype(np.float16).view(np.uint16)
        assert np.array_equal(twice, once), i

def _smooth(n, C, seed=1, scale=1.0):
    rng = np.random.default_rng(seed)
    sc = np.exp(rng.uniform(np.log(0.1), np.log(4), size=C)) * scale
    x = sc * rng.standard_normal(C) + np.cumsum(rng.standard_normal((n, C)) * 0.05 * sc, axis=0)
    return x.astype(np.float16)


def test_group_size_one_is_per_channel_absmax_int8():
    """With every token an anchor, the codec is vectorwise (per-channel absmax) int8
    quantization as in LLM.int8: q = round(x * 127 / absmax)."""
    x = _smooth(300, 16)
    for ch in range(16):
        col = x[:, ch]
        s = oracle.stream_scale(col)
        sym, rec = oracle.quantize_stream(col, 1, s, 123.0)
        x32 = col.astype(np.float32)
        m = np.float32(np.abs(x32).max())
        s_ref = np.float32(m / np.float32(127.0))
        assert np.float32(s) == s_ref
        q_ref = np.round(np.clip(x32 / s_ref, -127, 127))          # numpy rounds half to even
        assert np.array_equal(sym.astype(np.int64) - 127, q_ref.astype(np.int64))
        rec_ref = (q_ref.astype(np.int64).astype(np.float32) * s_ref).astype(np.float16).view(np.uint16)
        assert np.array_equal(rec, rec_ref)


def test_negation_symmetry():
    x = _smooth(200, 8, seed=2)
    for ch in range(8):
        col = x[:, ch]
        s = oracle.stream_scale(col)
        w = float(np.float32(1.5) * np.float32(s))
        a, _ = oracle.quantize_stream(col, 10, s, w)
        b, _ = oracle.quantize_stream(-col, 10, s, w)
        assert np.array_equal(a.astype(int) - 127, -(b.astype(int) - 127))


@pytest.mark.parametrize("k", [-3, -1, 1, 4])
def test_power_of_two_scaling_leaves_symbols_unchanged(k):
    # keep every value (and every scaled value) in the normal fp16 range so scaling is exact
    x = _smooth(200, 8, seed=3).astype(np.float32)
    x = (np.sign(x) * (np.abs(x) + 0.5)).astype(np.float16)
    y = (x.astype(np.float32) * np.float32(2.0 ** k)).astype(np.float16)
    assert np.array_equal(y.astype(np.float32), x.astype(np.float32) * np.float32(2.0 ** k))
    for ch in range(8):
        s1 = oracle.stream_scale(x[:, ch]); s2 = oracle.stream_scale(y[:, ch])
        w1 = float(np.float32(s1) * np.float32(0.5)); w2 = float(np.float32(s2) * np.float32(0.5))
        a, _ = oracle.quantize_stream(x[:, ch], 10, s1, w1)
        b, _ = oracle.quantize_stream(y[:, ch], 10, s2, w2)
        assert np.array_equal(a, b)


def test_error_bounds():
    """Anchors are within half a step of the input; unclamped deltas within half a bin (plus
    the fp16 rounding of the output)."""
    x = _smooth(1000, 32, seed=4)
    for ch in range(32):
        col = x[:, ch]
        s = oracle.stream_scale(col)
        w = float(np.float32(np.float32(1.0) * np.float32(s)))
        sym, rec = oracle.quantize_stream(col, 10, s, w)
        xv = col.astype(np.float64)
        rv = rec.view(np.float16).astype(np.float64)
        ulp = np.abs(np.spacing(rec.view(np.float16))).astype(np.float64)
        q = sym.astype(int) - 127
        anchors = np.arange(len(col)) % 10 == 0
        assert np.all(np.abs(rv - xv)[anchors] <= s / 2 * (1 + 1e-6) + ulp[anchors] / 2)
        unclamped = (~anchors) & (np.abs(q) < 127)
        assert np.all(np.abs(rv - xv)[unclamped] <= w / 2 * (1 + 1e-5) + ulp[unclamped] / 2)


def test_constant_channel_gives_zero_deltas():
    col = np.full(97, 3.1416, np.float16)
    s = oracle.stream_scale(col)
    sym, rec = oracle.quantize_stream(col, 10, s, float(np.float32(s)))
    assert np.all(sym[np.arange(97) % 10 != 0] == 127)
    assert np.all(sym[np.arange(97) % 10 == 0] == 254)          # absmax maps to +127


def test_zero_channel_scale_falls_back_to_one():
    col = np.zeros(30, np.float16)
    assert oracle.stream_scale(col) == 1.0
    sym, rec = oracle.quantize_stream(col, 10, 1.0, 0.5)
    assert np.all(sym == 127) and np.all(rec == 0)


def test_dequantize_inverts_symbols():
    x = _smooth(333, 4, seed=5)
    for ch in range(4):
        s = oracle.stream_scale(x[:, ch])
        w = float(np.float32(np.float32(0.5) * np.float32(s)))
        sym, rec = oracle.quantize_stream(x[:, ch], 10, s, w)
        assert np.array_equal(oracle.dequantize_stream(sym, 10, s, w), rec)


def test_deltas_more_concentrated_than_values():
    """Token-wise locality (Sec. 5.1.1): on a slowly drifting channel, delta symbols have lower
    empirical entropy than the anchor (8-bit) symbols of the same data."""
    x = _smooth(1536, 64, seed=6)
    ha, hd = [], []
    for ch in range(64):
        s = oracle.stream_scale(x[:, ch])
        w = float(np.float32(np.float32(0.5) * np.float32(s)))
        sym, _ = oracle.quantize_stream(x[:, ch], 1, s, w)      # all tokens 8-bit coded
        sd, _ = oracle.quantize_stream(x[:, ch], 10, s, w)
        def H(v):
            c = np.bincount(v, minlength=255); p = c[c > 0] / c.sum()
            return -(p * np.log2(p)).sum()
        ha.append(H(sym)); hd.append(H(sd[np.arange(1536) % 10 != 0]))
    assert np.mean(hd) < np.mean(ha)


def test_hand_worked_groups_of_ten():
    """Hand-worked streams (tests/golden/quant_g10_hand.txt, Sec. 5.2): anchors at 8 bits,
    deltas against the reconstructed anchor, ties to even, the +-127 clamp."""
    from conftest import golden_rows
    rows = golden_rows("quant_g10_hand.txt")
    for name, bw in (("A", 0.5), ("B", 1.5)):
        r = [x for x in rows if x[0] == name]
        assert [int(x[1]) for x in r] == list(range(len(r)))
        x = np.array([float(v[2]) for v in r], np.float16)
        assert np.array_equal(x.astype(np.float64), [float(v[2]) for v in r])   # exact fp16
        s = oracle.stream_scale(x)
        w = float(np.float32(np.float32(bw) * np.float32(s)))
        sym, rec = oracle.quantize_stream(x, 10, s, w)
        assert (sym.astype(int) - 127).tolist() == [int(v[3]) for v in r]
        assert rec.view(np.float16).astype(np.float64).tolist() == [float(v[4]) for v in r]


def _numpy_quantize_g10(x16, s, w):
    """Group-of-10 quantization in numpy fp32, vectorised over the groups: anchors
    q = rint(clip(x / s)), a = q * s; deltas q = rint(clip((x - a) / w)); reconstruction
    fp16(a + q * w) with the product and the sum each rounded to fp32 (numpy never fuses them)."""
    n = x16.size
    x = x16.astype(np.float32)
    s = np.float32(s)
    w = np.float32(w)
    j = np.arange(n)
    g0 = j - j % 10                                    # the group's anchor token
    # the quantized value is an integer: -0.0 from the rounding becomes 0 (reading of Sec. 5.2:
    # a decoder sees only q)
    qa = np.round(np.clip(x[g0] / s, np.float32(-127), np.float32(127))).astype(np.int64)
    a = (qa.astype(np.float32) * s).astype(np.float32)
    d = (x - a).astype(np.float32)
    qd = np.round(np.clip(d / w, np.float32(-127), np.float32(127)))
    anchor = j % 10 == 0
    q = np.where(anchor, qa, qd).astype(np.int64)
    prod = (q.astype(np.float32) * w).astype(np.float32)
    out = np.where(anchor, a, (a + prod).astype(np.float32))
    return q, out.astype(np.float16).view(np.uint16)


@pytest.mark.parametrize("bw", [0.5, 1.0, 1.5, 4.0, 12.0])
def test_group_of_ten_reconstruction_matches_numpy_fp32(bw):
    """Bit-exact against an independent numpy fp32 evaluation on random streams whose scales
    make the products inexact (a fused multiply-add or another summation order would differ)."""
    rng = np.random.default_rng(int(bw * 10))
    for trial in range(40):
        n = int(rng.integers(1, 400))
        sc = np.float32(np.exp(rng.uniform(np.log(0.01), np.log(300.0))))
        x = (sc * (rng.standard_normal() + np.cumsum(rng.standard_normal(n) * 0.2))).astype(np.float16)
        if trial % 5 == 0:
            x[rng.integers(0, n, size=max(1, n // 20))] *= np.float16(-30)     # clamped deltas
        s = oracle.stream_scale(x)
        w = float(np.float32(np.float32(bw) * np.float32(s)))
        sym, rec = oracle.quantize_stream(x, 10, s, w)
        q_ref, rec_ref = _numpy_quantize_g10(x, s, w)
        assert np.array_equal(sym.astype(np.int64) - 127, q_ref)
        assert np.array_equal(rec, rec_ref)
