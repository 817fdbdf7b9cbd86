"""CPU oracle of the CacheGen KV-cache codec (CacheGen, SIGCOMM '24, Sec. 5.2 and Sec. 6).

TEST INFRASTRUCTURE ONLY. Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg
of ``bench.py`` may import this package. The product (``paper_2310_07240_amd``) never does, and
this package imports nothing from it: the two share no code.

The arithmetic lives in ``cachegen_oracle.c`` (plain C, one stream and one bit at a time);
this module compiles it with gcc and marshals numpy arrays through ctypes.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "cachegen_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_LOCK = threading.Lock()
_LIB = None

NSYM = 255


_FLAGS = ["-std=c11", "-ffp-contract=off", "-fno-fast-math", "-msse2", "-mfpmath=sse", "-fPIC",
          "-shared", "-pthread"]


def build(force: bool = True) -> str:
    """Compile the oracle (gcc, -O2, no fused multiply-add, SSE arithmetic)."""
    if not force and os.path.exists(_LIB_PATH):
        return _LIB_PATH
    tmp = _LIB_PATH + ".tmp%d" % os.getpid()
    subprocess.run(["gcc", "-O2", *_FLAGS, _SRC, "-o", tmp, "-lm"], check=True)
    os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def build_sanitized(path: str) -> str:
    """Compile the oracle with AddressSanitizer and UndefinedBehaviorSanitizer (incl. float to
    integer conversions out of range) into `path`; load it by setting CG_ORACLE_LIB to that path
    in a process that preloads the ASan runtime."""
    subprocess.run(["gcc", "-O1", "-g", "-fno-omit-frame-pointer",
                    "-fsanitize=address,undefined,float-cast-overflow",
                    "-fno-sanitize-recover=all", *_FLAGS, _SRC, "-o", path, "-lm"], check=True)
    return path


class _Params(ctypes.Structure):
    _fields_ = [("n_ctx", ctypes.c_int32), ("n_layers", ctypes.c_int32),
                ("n_tokens", ctypes.c_int32), ("n_channels", ctypes.c_int32),
                ("group_size", ctypes.c_int32), ("chunk_len", ctypes.c_int32),
                ("n_levels", ctypes.c_int32),
                ("layer_bin", ctypes.POINTER(ctypes.c_float)),
                ("level_mult", ctypes.POINTER(ctypes.c_float))]


_P = ctypes.c_void_p
_I64 = ctypes.c_int64
_U64 = ctypes.c_uint64


def _lib():
    global _LIB
    with _LOCK:
        if _LIB is None:
            path = os.environ.get("CG_ORACLE_LIB") or _LIB_PATH
            if path == _LIB_PATH and (not os.path.exists(_LIB_PATH) or (
                    os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC))):
                build()
            L = ctypes.CDLL(path)
            L.cgo_half_to_float.argtypes = [ctypes.c_uint16]
            L.cgo_half_to_float.restype = ctypes.c_float
            L.cgo_float_to_half.argtypes = [ctypes.c_float]
            L.cgo_float_to_half.restype = ctypes.c_uint16
            L.cgo_num_streams.argtypes = [_P]
            L.cgo_num_streams.restype = _I64
            L.cgo_stream_scale.argtypes = [_P, _I64, _I64]
            L.cgo_stream_scale.restype = ctypes.c_float
            L.cgo_quantize_stream.argtypes = [_P, _I64, _I64, ctypes.c_int32, ctypes.c_float,
                                              ctypes.c_float, _P, _P]
            L.cgo_quantize_stream.restype = None
            L.cgo_dequantize_stream.argtypes = [_P, _I64, ctypes.c_int32, ctypes.c_float,
                                                ctypes.c_float, _P, _I64]
            L.cgo_dequantize_stream.restype = None
            L.cgo_normalize.argtypes = [_P, _P]
            L.cgo_normalize.restype = None
            L.cgo_ac_encode.argtypes = [_P, _I64, _P, _P, _U64]
            L.cgo_ac_encode.restype = _U64
            L.cgo_ac_decode.argtypes = [_P, _U64, _I64, _P, _P]
            L.cgo_ac_decode.restype = None
            L.cgo_stream_bound_words.argtypes = [_I64]
            L.cgo_stream_bound_words.restype = _U64
            L.cg_fit_cdf_ref.argtypes = [_P, _P, ctypes.c_int, _P, _P, ctypes.c_int]
            L.cg_fit_cdf_ref.restype = ctypes.c_int
            L.cg_fit_cdf_global_ref.argtypes = [_P, _P, ctypes.c_int, _P, _P, ctypes.c_int]
            L.cg_fit_cdf_global_ref.restype = ctypes.c_int
            L.cg_encode_ref.argtypes = [_P, _P, _P, _P, _P, _P, _U64, _P, _P, ctypes.c_int]
            L.cg_encode_ref.restype = _I64
            L.cg_decode_ref.argtypes = [_P, _P, _P, _P, _P, _P, _P, _I64, _I64, _P, ctypes.c_int]
            L.cg_decode_ref.restype = ctypes.c_int
            L.cgo_encode_stream.argtypes = [_P, _P, _P, _P, _P, _I64, _P, _U64, _P, _P]
            L.cgo_encode_stream.restype = _U64
            L.cgo_decode_stream.argtypes = [_P, _P, _U64, ctypes.c_float, _P, _P, _P, _I64, _P,
                                            _P, _P]
            L.cgo_decode_stream.restype = None
            L.cgo_encode_streams.argtypes = [_P, _P, _P, _P, _P, _P, _I64, _P, _U64, _P, _P,
                                             ctypes.c_int]
            L.cgo_encode_streams.restype = _I64
            L.cgo_num_token_streams.argtypes = [_P]
            L.cgo_num_token_streams.restype = _I64
            L.cg_encode_tokens_ref.argtypes = [_P, _P, _P, _P, _P, _P, _U64, _P, _P,
                                               ctypes.c_int]
            L.cg_encode_tokens_ref.restype = _I64
            L.cg_decode_tokens_ref.argtypes = [_P, _P, _P, _P, _P, _P, _P, _P, ctypes.c_int]
            L.cg_decode_tokens_ref.restype = ctypes.c_int
            _LIB = L
    return _LIB


def _ptr(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"], "oracle arrays must be C-contiguous"
    return ctypes.c_void_p(a.ctypes.data)


def default_threads() -> int:
    try:
        return max(1, len(os.sched_getaffinity(0)))
    except AttributeError:  # pragma: no cover
        return max(1, os.cpu_count() or 1)


@dataclass
class Shape:
    """Codec parameters as the oracle sees them (same meaning as cg_params of the C ABI)."""
    n_ctx: int
    n_layers: int
    n_tokens: int
    n_channels: int
    group_size: int
    chunk_len: int
    layer_bin: np.ndarray
    level_mult: np.ndarray

    @property
    def n_levels(self) -> int:
        return int(len(self.level_mult))

    @property
    def n_chunks(self) -> int:
        return -(-self.n_tokens // self.chunk_len)

    @property
    def n_streams(self) -> int:
        return self.n_ctx * self.n_chunks * self.n_layers * 2 * self.n_channels

    def kv_shape(self):
        return (self.n_ctx, self.n_layers, 2, self.n_tokens, self.n_channels)

    def _c(self):
        lb = np.ascontiguousarray(self.layer_bin, dtype=np.float32)
        lm = np.ascontiguousarray(self.level_mult, dtype=np.float32)
        s = _Params(self.n_ctx, self.n_layers, self.n_tokens, self.n_channels,
                    self.group_size, self.chunk_len, len(lm),
                    lb.ctypes.data_as(ctypes.POINTER(ctypes.c_float)),
                    lm.ctypes.data_as(ctypes.POINTER(ctypes.c_float)))
        return s, (lb, lm)  # keep the arrays alive with the struct


def shape_from(cfg) -> Shape:
    """Build a Shape from any object with the codec-parameter attributes."""
    return Shape(cfg.n_ctx, cfg.n_layers, cfg.n_tokens, cfg.n_channels, cfg.group_size,
                 cfg.chunk_len, np.asarray(cfg.layer_bin, np.float32),
                 np.asarray(cfg.level_mult, np.float32))


# --------------------------------------------------------------------------------------------
# fp16 conversions
# --------------------------------------------------------------------------------------------
def half_to_float(h: int) -> float:
    return float(_lib().cgo_half_to_float(int(h)))


def float_to_half(f: float) -> int:
    return int(_lib().cgo_float_to_half(float(f)))


# --------------------------------------------------------------------------------------------
# single-stream steps
# --------------------------------------------------------------------------------------------
def stream_scale(x_f16: np.ndarray) -> float:
    x = np.ascontiguousarray(x_f16.view(np.uint16))
    return float(_lib().cgo_stream_scale(_ptr(x), 1, x.size))


def quantize_stream(x_f16: np.ndarray, group_size: int, scale: float, width: float):
    """Symbols (uint8, q + 127) and fp16 reconstruction (uint16 bit patterns) of one stream."""
    x = np.ascontiguousarray(x_f16.view(np.uint16))
    sym = np.zeros(x.size, np.uint8)
    rec = np.zeros(x.size, np.uint16)
    _lib().cgo_quantize_stream(_ptr(x), 1, x.size, group_size, scale, width, _ptr(sym), _ptr(rec))
    return sym, rec


def dequantize_stream(sym: np.ndarray, group_size: int, scale: float, width: float):
    sym = np.ascontiguousarray(sym, np.uint8)
    out = np.zeros(sym.size, np.uint16)
    _lib().cgo_dequantize_stream(_ptr(sym), sym.size, group_size, scale, width, _ptr(out), 1)
    return out


def normalize(counts) -> np.ndarray:
    """Integer counts [255] -> uint16 cumulative table [256] (entry 255 is padding)."""
    c = np.ascontiguousarray(np.asarray(counts, dtype=np.uint64))
    assert c.size == NSYM
    out = np.zeros(256, np.uint16)
    _lib().cgo_normalize(_ptr(c), _ptr(out))
    return out


def cum32(table: np.ndarray) -> np.ndarray:
    """Cumulative table with the implicit top: uint32 [256] with entry 255 = 65536."""
    t = np.asarray(table, np.uint32).copy()
    t[255] = 65536
    return t


def ac_encode(symbols, tables) -> tuple[np.ndarray, int]:
    """Arithmetic-code a symbol sequence. `tables` is one uint16 [256] table for every symbol,
    or a list with one table per symbol. Returns (words, bit count before padding)."""
    sym = np.ascontiguousarray(np.asarray(symbols, dtype=np.uint8))
    n = sym.size
    tabs, keep = _table_ptrs(tables, n)
    cap = int(_lib().cgo_stream_bound_words(n))
    out = np.zeros(max(cap, 1), np.uint32)
    nbits = int(_lib().cgo_ac_encode(_ptr(sym), n, tabs, _ptr(out), cap))
    assert nbits != 2**64 - 1
    return out[: (nbits + 31) // 32].copy(), nbits


def ac_decode(words, n: int, tables) -> np.ndarray:
    w = np.ascontiguousarray(np.asarray(words, dtype=np.uint32))
    tabs, keep = _table_ptrs(tables, n)
    sym = np.zeros(max(n, 1), np.uint8)
    _lib().cgo_ac_decode(_ptr(w) if w.size else None, w.size, n, tabs, _ptr(sym))
    return sym[:n]


def _table_ptrs(tables, n):
    if isinstance(tables, np.ndarray) and tables.ndim == 1:
        tables = [tables] * max(n, 1)
    keep = [np.ascontiguousarray(np.asarray(t, dtype=np.uint16)) for t in tables]
    assert len(keep) >= n
    arr = (ctypes.c_void_p * max(len(keep), 1))(*[t.ctypes.data for t in keep])
    return ctypes.cast(arr, ctypes.c_void_p), (keep, arr)


# --------------------------------------------------------------------------------------------
# whole codec
# --------------------------------------------------------------------------------------------
def fit_cdf(kv: np.ndarray, shape: Shape, level: int, threads: int | None = None):
    """cg_fit_cdf at one level: (cdf_anchor [L,2,C,256], cdf_delta_level [L,2,C,256])."""
    kvu = np.ascontiguousarray(kv.view(np.uint16)).reshape(shape.kv_shape())
    L, C = shape.n_layers, shape.n_channels
    ca = np.zeros((L, 2, C, 256), np.uint16)
    cd = np.zeros((L, 2, C, 256), np.uint16)
    ps, keep = shape._c()
    _lib().cg_fit_cdf_ref(ctypes.byref(ps), _ptr(kvu), level, _ptr(ca), _ptr(cd),
                          threads or default_threads())
    return ca, cd


def fit_cdf_global(kv: np.ndarray, shape: Shape, level: int, threads: int | None = None):
    """The ablation baseline: one anchor and one delta distribution pooled over every layer,
    K/V and channel, written to every table slot: (cdf_anchor, cdf_delta_level)."""
    kvu = np.ascontiguousarray(kv.view(np.uint16)).reshape(shape.kv_shape())
    L, C = shape.n_layers, shape.n_channels
    ca = np.zeros((L, 2, C, 256), np.uint16)
    cd = np.zeros((L, 2, C, 256), np.uint16)
    ps, keep = shape._c()
    _lib().cg_fit_cdf_global_ref(ctypes.byref(ps), _ptr(kvu), level, _ptr(ca), _ptr(cd),
                                 threads or default_threads())
    return ca, cd


def fit_all_levels(kv, shape: Shape, threads=None):
    """Anchor tables plus the delta tables of every level [n_levels, L, 2, C, 256]."""
    ca = None
    ds = []
    for lv in range(shape.n_levels):
        a, d = fit_cdf(kv, shape, lv, threads)
        ca = a if ca is None else ca
        ds.append(d)
    return ca, np.stack(ds)


def bound_words(shape: Shape) -> int:
    total = 0
    per = shape.n_ctx * shape.n_layers * 2 * shape.n_channels
    for c in range(shape.n_chunks):
        n = min(shape.chunk_len, shape.n_tokens - c * shape.chunk_len)
        total += per * int(_lib().cgo_stream_bound_words(n))
    return total


def encode(kv, shape: Shape, chunk_level, cdf_anchor, cdf_delta, threads=None):
    """cg_encode: returns (words uint32 [total], offsets uint64 [S+1], scales fp32 [S])."""
    kvu = np.ascontiguousarray(kv.view(np.uint16)).reshape(shape.kv_shape())
    cl = np.ascontiguousarray(np.asarray(chunk_level, np.uint8).reshape(shape.n_ctx, shape.n_chunks))
    ca = np.ascontiguousarray(cdf_anchor, np.uint16)
    cd = np.ascontiguousarray(cdf_delta, np.uint16)
    S = shape.n_streams
    cap = bound_words(shape)
    words = np.zeros(max(cap, 1), np.uint32)
    offsets = np.zeros(S + 1, np.uint64)
    scales = np.zeros(S, np.float32)
    ps, keep = shape._c()
    total = _lib().cg_encode_ref(ctypes.byref(ps), _ptr(kvu), _ptr(cl), _ptr(ca), _ptr(cd),
                                 _ptr(words), cap, _ptr(offsets), _ptr(scales),
                                 threads or default_threads())
    assert total >= 0, "oracle encode overflowed its bound"
    return words[:total].copy(), offsets, scales


def decode(words, offsets, scales, shape: Shape, chunk_level, cdf_anchor, cdf_delta,
           chunk_begin=0, chunk_end=None, out=None, threads=None):
    """cg_decode: fp16 bit patterns [B, L, 2, T, C] (uint16); rows outside the chunk range
    keep the contents of `out` (zeros when not given)."""
    if chunk_end is None:
        chunk_end = shape.n_chunks
    w = np.ascontiguousarray(words, np.uint32)
    if w.size == 0:
        w = np.zeros(1, np.uint32)
    off = np.ascontiguousarray(offsets, np.uint64)
    sc = np.ascontiguousarray(scales, np.float32)
    cl = np.ascontiguousarray(np.asarray(chunk_level, np.uint8).reshape(shape.n_ctx, shape.n_chunks))
    ca = np.ascontiguousarray(cdf_anchor, np.uint16)
    cd = np.ascontiguousarray(cdf_delta, np.uint16)
    if out is None:
        out = np.zeros(shape.kv_shape(), np.uint16)
    ps, keep = shape._c()
    _lib().cg_decode_ref(ctypes.byref(ps), _ptr(w), _ptr(off), _ptr(sc), _ptr(cl), _ptr(ca),
                         _ptr(cd), chunk_begin, chunk_end, _ptr(out), threads or default_threads())
    return out


def n_token_streams(shape: Shape) -> int:
    """Streams of the token-parallel layout: one per (context, layer, K/V, token)."""
    return shape.n_ctx * shape.n_layers * 2 * shape.n_tokens


def encode_tokens(kv, shape: Shape, chunk_level, cdf_anchor, cdf_delta, threads=None):
    """Encode in the token-parallel layout (one stream per (context, layer, K/V, token) over
    the token's channels). Returns (words uint32, offsets uint64 [St+1], scales fp32 [S])."""
    kvu = np.ascontiguousarray(kv.view(np.uint16)).reshape(shape.kv_shape())
    cl = np.ascontiguousarray(np.asarray(chunk_level, np.uint8).reshape(shape.n_ctx, shape.n_chunks))
    ca = np.ascontiguousarray(cdf_anchor, np.uint16)
    cd = np.ascontiguousarray(cdf_delta, np.uint16)
    St = n_token_streams(shape)
    cap = St * int(_lib().cgo_stream_bound_words(shape.n_channels))
    words = np.zeros(max(cap, 1), np.uint32)
    offsets = np.zeros(St + 1, np.uint64)
    scales = np.zeros(shape.n_streams, np.float32)
    ps, keep = shape._c()
    total = _lib().cg_encode_tokens_ref(ctypes.byref(ps), _ptr(kvu), _ptr(cl), _ptr(ca),
                                        _ptr(cd), _ptr(words), cap, _ptr(offsets),
                                        _ptr(scales), threads or default_threads())
    assert total >= 0, "oracle token-layout encode overflowed its bound"
    return words[:total].copy(), offsets, scales


def decode_tokens(words, offsets, scales, shape: Shape, chunk_level, cdf_anchor, cdf_delta,
                  threads=None):
    """Decode the token-parallel layout: fp16 bit patterns [B, L, 2, T, C] (uint16)."""
    w = np.ascontiguousarray(words, np.uint32)
    if w.size == 0:
        w = np.zeros(1, np.uint32)
    off = np.ascontiguousarray(offsets, np.uint64)
    sc = np.ascontiguousarray(scales, np.float32)
    cl = np.ascontiguousarray(np.asarray(chunk_level, np.uint8).reshape(shape.n_ctx, shape.n_chunks))
    ca = np.ascontiguousarray(cdf_anchor, np.uint16)
    cd = np.ascontiguousarray(cdf_delta, np.uint16)
    out = np.zeros(shape.kv_shape(), np.uint16)
    ps, keep = shape._c()
    _lib().cg_decode_tokens_ref(ctypes.byref(ps), _ptr(w), _ptr(off), _ptr(sc), _ptr(cl),
                                _ptr(ca), _ptr(cd), _ptr(out), threads or default_threads())
    return out


def encode_streams(kv, shape: Shape, chunk_level, cdf_anchor, cdf_delta, stream_ids,
                   threads=None):
    """Encode only the listed streams. Returns (list of uint32 word arrays, scales fp32)."""
    kvu = np.ascontiguousarray(kv.view(np.uint16)).reshape(shape.kv_shape())
    cl = np.ascontiguousarray(np.asarray(chunk_level, np.uint8).reshape(shape.n_ctx, shape.n_chunks))
    ca = np.ascontiguousarray(cdf_anchor, np.uint16)
    cd = np.ascontiguousarray(cdf_delta, np.uint16)
    ids = np.ascontiguousarray(np.asarray(stream_ids, np.int64))
    n = ids.size
    per = int(_lib().cgo_stream_bound_words(min(shape.chunk_len, shape.n_tokens)))
    cap = max(n * per, 1)
    out = np.zeros(cap, np.uint32)
    lens = np.zeros(max(n, 1), np.uint64)
    scales = np.zeros(max(n, 1), np.float32)
    ps, keep = shape._c()
    total = _lib().cgo_encode_streams(ctypes.byref(ps), _ptr(kvu), _ptr(cl), _ptr(ca), _ptr(cd),
                                      _ptr(ids), n, _ptr(out), cap, _ptr(lens), _ptr(scales),
                                      threads or default_threads())
    assert total >= 0
    res, pos = [], 0
    for i in range(n):
        k = int(lens[i])
        res.append(out[pos:pos + k].copy())
        pos += k
    return res, scales[:n].copy()


def decode_stream(words, scale, shape: Shape, chunk_level, cdf_anchor, cdf_delta, stream_id):
    """Decode one stream: (fp16 values uint16 [n], symbols uint8 [n])."""
    w = np.ascontiguousarray(np.asarray(words, np.uint32))
    if w.size == 0:
        w_ptr, nw = None, 0
    else:
        w_ptr, nw = _ptr(w), w.size
    cl = np.ascontiguousarray(np.asarray(chunk_level, np.uint8).reshape(shape.n_ctx, shape.n_chunks))
    ca = np.ascontiguousarray(cdf_anchor, np.uint16)
    cd = np.ascontiguousarray(cdf_delta, np.uint16)
    c = (stream_id // (shape.n_channels * 2 * shape.n_layers)) % shape.n_chunks
    n = min(shape.chunk_len, shape.n_tokens - c * shape.chunk_len)
    rec = np.zeros(n, np.uint16)
    sym = np.zeros(n, np.uint8)
    ps, keep = shape._c()
    _lib().cgo_decode_stream(ctypes.byref(ps), w_ptr, nw, float(scale), _ptr(cl), _ptr(ca),
                             _ptr(cd), int(stream_id), None, _ptr(rec), _ptr(sym))
    return rec, sym


def stream_symbols(kv, shape: Shape, chunk_level, stream_id):
    """Scale, symbols and fp16 reconstruction of one stream straight from the quantizer."""
    kvu = np.ascontiguousarray(kv.view(np.uint16)).reshape(shape.kv_shape())
    C, L, NC = shape.n_channels, shape.n_layers, shape.n_chunks
    s = int(stream_id)
    ch = s % C; s //= C
    k = s % 2; s //= 2
    l = s % L; s //= L
    c = s % NC; b = s // NC
    t0 = c * shape.chunk_len
    x = np.ascontiguousarray(kvu[b, l, k, t0:t0 + shape.chunk_len, ch])
    sc = stream_scale(x)
    lv = int(np.asarray(chunk_level, np.uint8).reshape(shape.n_ctx, NC)[b, c])
    lv = min(lv, shape.n_levels - 1)
    bw = np.float32(np.float32(shape.layer_bin[l]) * np.float32(shape.level_mult[lv]))
    w = float(np.float32(bw * np.float32(sc)))
    sym, rec = quantize_stream(x, shape.group_size, sc, w)
    return sc, sym, rec


# --------------------------------------------------------------------------------------------
# Streaming adaptation (Sec. 5.3 "KV cache streaming adaptation"; App. B, Alg. 1), plain Python.
# --------------------------------------------------------------------------------------------
def adapt_schedule(level_bytes, text_bytes, recompute_ms, slo_ms, prior_gbps, default_level,
                   bandwidth_gbps):
    """The streaming adapter of Alg. 1, one chunk at a time, in the algorithm's terms:
    remaining_time = SLO - time_elapsed; text if time_recompute (of the chunks still to send)
    fits in remaining_time; else the encoding level with the least compression loss whose size
    of the chunks still to send, divided by the throughput (the previous chunk's measured one),
    fits; else the smallest one. The first chunk without a throughput takes the default level.
    Returns (choices, ttft_ms) with choice -1 for text."""
    chunks_to_send = list(range(len(text_bytes)))
    n_levels = len(level_bytes[0])
    time_elapsed = 0.0
    throughput = prior_gbps if prior_gbps > 0 else None
    choices = []
    while chunks_to_send:
        c = chunks_to_send[0]
        remaining_time = slo_ms - time_elapsed
        choice = None
        if recompute_ms is not None:
            time_recompute = 0.0
            for i in chunks_to_send:
                time_recompute += recompute_ms[i]
            if time_recompute <= remaining_time:
                choice = -1
        if choice is None:
            if throughput is None:
                choice = default_level
            else:
                for level in range(n_levels):          # level 0 loses least
                    size = 0.0
                    for i in chunks_to_send:
                        size += level_bytes[i][level]
                    if size * 8.0 / (throughput * 1.0e6) <= remaining_time:
                        choice = level
                        break
                if choice is None:
                    choice = n_levels - 1
        sent = text_bytes[c] if choice < 0 else level_bytes[c][choice]
        time_elapsed += sent * 8.0 / (bandwidth_gbps[c] * 1.0e6)
        if choice < 0:
            time_elapsed += recompute_ms[c]
        choices.append(choice)
        throughput = bandwidth_gbps[c]
        chunks_to_send = chunks_to_send[1:]
    return choices, time_elapsed
