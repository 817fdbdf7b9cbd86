"""Python binding of the codec's C ABI (include/cachegen.h).

Argument marshalling only: every step of the codec runs in the HIP kernels of
``libcachegen.so``. torch supplies device buffers and the HIP stream handle. There is no CPU
fallback: if the library is missing or no GPU is present, the calls raise.

Names follow the C ABI: ``cg_fit_cdf``, ``cg_encode``, ``cg_decode`` (plus the size queries);
``Codec`` bundles the parameters and allocates outputs for the common whole-cache calls.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libcachegen.so")

CG_OK = 0
ERRORS = {-1: "CG_ERR_ARG", -2: "CG_ERR_SHAPE", -3: "CG_ERR_CAPACITY", -4: "CG_ERR_NONFINITE",
          -5: "CG_ERR_HIP", -6: "CG_ERR_PARAM", -7: "CG_ERR_SCRATCH"}

EXPORTS = ("cg_num_chunks", "cg_num_streams", "cg_encode_bound_words",
           "cg_encode_workspace_bytes", "cg_fit_cdf", "cg_fit_cdf_global", "cg_encode",
           "cg_decode", "cg_decode_streamed", "cg_adapt_schedule", "cg_check_finite",
           "cg_num_token_streams", "cg_encode_tokens_bound_words",
           "cg_encode_tokens_workspace_bytes", "cg_decode_tokens_workspace_bytes",
           "cg_encode_tokens", "cg_decode_tokens", "cg_get_status", "cg_encode_noalloc",
           "cg_fit_cdf_levels", "cg_encode_with_scales", "cg_strerror")
CG_FIT_GLOBAL_WORKSPACE_BYTES = 8192
CG_NOALLOC_SCRATCH_BYTES = 64 << 20


class CodecError(RuntimeError):
    def __init__(self, code: int, what: str):
        self.code = code
        super().__init__(f"{what}: {ERRORS.get(code, code)} ({strerror(code)})")


class _CParams(ctypes.Structure):
    _fields_ = [("n_ctx", ctypes.c_int32), ("n_layers", ctypes.c_int32),
                ("n_tokens", ctypes.c_int32), ("n_channels", ctypes.c_int32),
                ("group_size", ctypes.c_int32), ("chunk_len", ctypes.c_int32),
                ("n_levels", ctypes.c_int32),
                ("layer_bin", ctypes.POINTER(ctypes.c_float)),
                ("level_mult", ctypes.POINTER(ctypes.c_float))]


class _AdaptParams(ctypes.Structure):
    _fields_ = [("n_chunks", ctypes.c_int32), ("n_levels", ctypes.c_int32),
                ("level_bytes", ctypes.c_void_p), ("text_bytes", ctypes.c_void_p),
                ("recompute_ms", ctypes.c_void_p), ("slo_ms", ctypes.c_double),
                ("prior_gbps", ctypes.c_double), ("default_level", ctypes.c_int32)]


class StreamStats(ctypes.Structure):
    """cg_stream_stats: timings of one cg_decode_streamed call (milliseconds)."""
    _fields_ = [("n_chunks", ctypes.c_int32), ("transfer_ms", ctypes.c_double),
                ("total_ms", ctypes.c_double), ("decode_sum_ms", ctypes.c_double),
                ("hidden_fraction", ctypes.c_double),
                ("chunk_copy_done_ms", ctypes.POINTER(ctypes.c_double)),
                ("chunk_decode_begin_ms", ctypes.POINTER(ctypes.c_double)),
                ("chunk_decode_end_ms", ctypes.POINTER(ctypes.c_double))]
    SCALARS = ("n_chunks", "transfer_ms", "total_ms", "decode_sum_ms", "hidden_fraction")

    def as_dict(self):
        return {f: getattr(self, f) for f in self.SCALARS}


_LIB = None
_P = ctypes.c_void_p


def lib():
    """Load libcachegen.so (raises if it has not been built)."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2310_07240_amd.build` (no CPU fallback exists)")
        L = ctypes.CDLL(LIB_PATH)
        PP = ctypes.POINTER(_CParams)
        L.cg_num_chunks.argtypes = [PP]; L.cg_num_chunks.restype = ctypes.c_int64
        L.cg_num_streams.argtypes = [PP]; L.cg_num_streams.restype = ctypes.c_int64
        L.cg_encode_bound_words.argtypes = [PP]; L.cg_encode_bound_words.restype = ctypes.c_uint64
        L.cg_encode_workspace_bytes.argtypes = [PP]
        L.cg_encode_workspace_bytes.restype = ctypes.c_uint64
        L.cg_fit_cdf.argtypes = [PP, _P, ctypes.c_int32, _P, _P, _P]
        L.cg_fit_cdf.restype = ctypes.c_int
        L.cg_fit_cdf_levels.argtypes = [PP, _P, _P, _P, _P, _P, _P]
        L.cg_fit_cdf_levels.restype = ctypes.c_int
        L.cg_fit_cdf_global.argtypes = [PP, _P, ctypes.c_int32, _P, _P, _P, ctypes.c_uint64, _P]
        L.cg_fit_cdf_global.restype = ctypes.c_int
        L.cg_encode.argtypes = [PP, _P, _P, _P, _P, _P, ctypes.c_uint64, _P, _P, _P,
                                ctypes.c_uint64, _P]
        L.cg_encode.restype = ctypes.c_int
        L.cg_encode_with_scales.argtypes = [PP, _P, _P, _P, _P, _P, _P, ctypes.c_uint64, _P, _P,
                                            ctypes.c_uint64, _P]
        L.cg_encode_with_scales.restype = ctypes.c_int
        L.cg_decode.argtypes = [PP, _P, _P, _P, _P, _P, _P, ctypes.c_int32, ctypes.c_int32, _P, _P]
        L.cg_decode.restype = ctypes.c_int
        L.cg_decode_streamed.argtypes = [PP, _P, _P, _P, ctypes.c_uint64, _P, _P, _P, _P, _P, _P,
                                         ctypes.c_double, _P, _P, ctypes.POINTER(StreamStats)]
        L.cg_decode_streamed.restype = ctypes.c_int
        L.cg_adapt_schedule.argtypes = [ctypes.POINTER(_AdaptParams), _P, _P, _P]
        L.cg_adapt_schedule.restype = ctypes.c_int
        L.cg_check_finite.argtypes = [PP, _P, _P, _P]
        L.cg_check_finite.restype = ctypes.c_int
        L.cg_get_status.argtypes = [_P, _P]
        L.cg_get_status.restype = ctypes.c_int
        L.cg_encode_noalloc.argtypes = [PP, _P, _P, _P, _P, _P, ctypes.c_uint64, _P, _P, _P, _P]
        L.cg_encode_noalloc.restype = ctypes.c_int
        for name in ("cg_encode_tokens_bound_words", "cg_encode_tokens_workspace_bytes",
                     "cg_decode_tokens_workspace_bytes"):
            getattr(L, name).argtypes = [PP]
            getattr(L, name).restype = ctypes.c_uint64
        L.cg_num_token_streams.argtypes = [PP]; L.cg_num_token_streams.restype = ctypes.c_int64
        L.cg_encode_tokens.argtypes = [PP, _P, _P, _P, _P, _P, ctypes.c_uint64, _P, _P, _P,
                                       ctypes.c_uint64, _P]
        L.cg_encode_tokens.restype = ctypes.c_int
        L.cg_decode_tokens.argtypes = [PP, _P, _P, _P, _P, _P, _P, _P, _P, ctypes.c_uint64, _P]
        L.cg_decode_tokens.restype = ctypes.c_int
        L.cg_strerror.argtypes = [ctypes.c_int]
        L.cg_strerror.restype = ctypes.c_char_p
        _LIB = L
    return _LIB


def strerror(code: int) -> str:
    return lib().cg_strerror(int(code)).decode()


@dataclass
class CodecParams:
    """cg_params: shape of the KV cache and the quantizer's tables (host memory)."""
    n_ctx: int
    n_layers: int
    n_tokens: int
    n_channels: int
    layer_bin: tuple
    level_mult: tuple
    group_size: int = 10
    chunk_len: int = 1536

    @classmethod
    def of(cls, obj) -> "CodecParams":
        return cls(obj.n_ctx, obj.n_layers, obj.n_tokens, obj.n_channels, tuple(obj.layer_bin),
                   tuple(obj.level_mult), obj.group_size, obj.chunk_len)

    @property
    def n_levels(self) -> int:
        return len(self.level_mult)

    @property
    def kv_shape(self):
        return (self.n_ctx, self.n_layers, 2, self.n_tokens, self.n_channels)

    def c(self):
        """The C struct plus the arrays it points into (keep both alive for the call)."""
        lb = np.ascontiguousarray(self.layer_bin, np.float32)
        lm = np.ascontiguousarray(self.level_mult, np.float32)
        s = _CParams(self.n_ctx, self.n_layers, self.n_tokens, self.n_channels, self.group_size,
                     self.chunk_len, len(lm), lb.ctypes.data_as(ctypes.POINTER(ctypes.c_float)),
                     lm.ctypes.data_as(ctypes.POINTER(ctypes.c_float)))
        return s, (lb, lm)


def _ptr(t):
    if t is None:
        return None
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _check(rc: int, what: str):
    if rc != CG_OK:
        raise CodecError(rc, what)


# --------------------------------------------------------------------------------------------
# size queries (host only)
# --------------------------------------------------------------------------------------------
def cg_num_chunks(p: CodecParams) -> int:
    s, keep = p.c()
    return int(lib().cg_num_chunks(ctypes.byref(s)))


def cg_num_streams(p: CodecParams) -> int:
    s, keep = p.c()
    return int(lib().cg_num_streams(ctypes.byref(s)))


def cg_encode_bound_words(p: CodecParams) -> int:
    s, keep = p.c()
    return int(lib().cg_encode_bound_words(ctypes.byref(s)))


def cg_encode_workspace_bytes(p: CodecParams) -> int:
    s, keep = p.c()
    return int(lib().cg_encode_workspace_bytes(ctypes.byref(s)))


# --------------------------------------------------------------------------------------------
# the three codec calls
# --------------------------------------------------------------------------------------------
def cg_fit_cdf(p: CodecParams, kv, level: int, cdf_anchor, cdf_delta_level, stream=None):
    s, keep = p.c()
    _check(lib().cg_fit_cdf(ctypes.byref(s), _ptr(kv), int(level), _ptr(cdf_anchor),
                            _ptr(cdf_delta_level), _stream(stream)), "cg_fit_cdf")


def cg_fit_cdf_levels(p: CodecParams, kv, cdf_anchor, cdf_delta, status=None, stream=None,
                      scales=None):
    """Every level's tables in one call (cdf_delta [n_levels, L, 2, C, 256]); `status` is an
    optional device int32 tensor of one element (0, or non-zero for NaN / Inf in kv);
    `scales`, an optional device float32 tensor [S], receives every stream's scale."""
    s, keep = p.c()
    _check(lib().cg_fit_cdf_levels(ctypes.byref(s), _ptr(kv), _ptr(cdf_anchor), _ptr(cdf_delta),
                                   _ptr(status), _ptr(scales), _stream(stream)),
           "cg_fit_cdf_levels")


def cg_fit_cdf_global(p: CodecParams, kv, level: int, cdf_anchor, cdf_delta_level, workspace,
                      stream=None):
    """The one-global-distribution baseline: pooled tables written to every slot."""
    s, keep = p.c()
    _check(lib().cg_fit_cdf_global(ctypes.byref(s), _ptr(kv), int(level), _ptr(cdf_anchor),
                                   _ptr(cdf_delta_level), _ptr(workspace),
                                   workspace.numel() * workspace.element_size(),
                                   _stream(stream)), "cg_fit_cdf_global")


def cg_encode(p: CodecParams, kv, chunk_level, cdf_anchor, cdf_delta, words, offsets, scales,
              workspace, stream=None):
    s, keep = p.c()
    _check(lib().cg_encode(ctypes.byref(s), _ptr(kv), _ptr(chunk_level), _ptr(cdf_anchor),
                           _ptr(cdf_delta), _ptr(words), words.numel(), _ptr(offsets),
                           _ptr(scales), _ptr(workspace), workspace.numel() * workspace.element_size(),
                           _stream(stream)), "cg_encode")


def cg_encode_with_scales(p: CodecParams, kv, chunk_level, cdf_anchor, cdf_delta, scales, words,
                          offsets, workspace, stream=None):
    """cg_encode with the streams' scales as an input (as cg_fit_cdf_levels wrote them)."""
    s, keep = p.c()
    _check(lib().cg_encode_with_scales(ctypes.byref(s), _ptr(kv), _ptr(chunk_level),
                                       _ptr(cdf_anchor), _ptr(cdf_delta), _ptr(scales),
                                       _ptr(words), words.numel(), _ptr(offsets),
                                       _ptr(workspace),
                                       workspace.numel() * workspace.element_size(),
                                       _stream(stream)), "cg_encode_with_scales")


def cg_encode_noalloc(p: CodecParams, kv, chunk_level, cdf_anchor, cdf_delta, words, offsets,
                      scales, status=None, stream=None):
    """cg_encode with the library's static per-GPU scratch instead of a workspace (no device
    allocation); `status` is an optional device int32 tensor of one element."""
    s, keep = p.c()
    _check(lib().cg_encode_noalloc(ctypes.byref(s), _ptr(kv), _ptr(chunk_level),
                                   _ptr(cdf_anchor), _ptr(cdf_delta), _ptr(words), words.numel(),
                                   _ptr(offsets), _ptr(scales), _ptr(status), _stream(stream)),
           "cg_encode_noalloc")


def cg_decode(p: CodecParams, words, offsets, scales, chunk_level, cdf_anchor, cdf_delta,
              chunk_begin: int, chunk_end: int, kv_out, stream=None):
    s, keep = p.c()
    _check(lib().cg_decode(ctypes.byref(s), _ptr(words), _ptr(offsets), _ptr(scales),
                           _ptr(chunk_level), _ptr(cdf_anchor), _ptr(cdf_delta), int(chunk_begin),
                           int(chunk_end), _ptr(kv_out), _stream(stream)), "cg_decode")


def cg_decode_streamed(p: CodecParams, words_host, offsets_host, words_dev, offsets_dev, scales,
                       chunk_level, cdf_anchor, cdf_delta, kv_out, link_gbps: float,
                       decode_stream, copy_stream) -> dict:
    """Decode chunk by chunk while the payload is copied from (pinned) host memory; returns
    the call's timings (cg_stream_stats as a dict, with the per-chunk event times as lists).
    Synchronous."""
    s, keep = p.c()
    nc = cg_num_chunks(p)
    per = [np.zeros(max(nc, 1), np.float64) for _ in range(3)]
    st = StreamStats()
    dp = ctypes.POINTER(ctypes.c_double)
    st.chunk_copy_done_ms = per[0].ctypes.data_as(dp)
    st.chunk_decode_begin_ms = per[1].ctypes.data_as(dp)
    st.chunk_decode_end_ms = per[2].ctypes.data_as(dp)
    _check(lib().cg_decode_streamed(ctypes.byref(s), _ptr(words_host), _ptr(offsets_host),
                                    _ptr(words_dev), words_dev.numel(), _ptr(offsets_dev),
                                    _ptr(scales),
                                    _ptr(chunk_level), _ptr(cdf_anchor), _ptr(cdf_delta),
                                    _ptr(kv_out), float(link_gbps), _stream(decode_stream),
                                    _stream(copy_stream), ctypes.byref(st)), "cg_decode_streamed")
    d = st.as_dict()
    d["chunk_copy_done_ms"] = per[0][:nc].tolist()
    d["chunk_decode_begin_ms"] = per[1][:nc].tolist()
    d["chunk_decode_end_ms"] = per[2][:nc].tolist()
    return d


def cg_adapt_schedule(level_bytes, text_bytes, recompute_ms, slo_ms: float, prior_gbps: float,
                      default_level: int, bandwidth_gbps):
    """Streaming adaptation plan for one context (host only): returns (choices, ttft_ms), a
    choice being the encoding level or -1 for text. level_bytes is [n_chunks][n_levels]."""
    lb = np.ascontiguousarray(level_bytes, np.float64)
    tb = np.ascontiguousarray(text_bytes, np.float64)
    rc = None if recompute_ms is None else np.ascontiguousarray(recompute_ms, np.float64)
    bw = np.ascontiguousarray(bandwidth_gbps, np.float64)
    n, v = lb.shape
    a = _AdaptParams(n, v, lb.ctypes.data, tb.ctypes.data, None if rc is None else rc.ctypes.data,
                     float(slo_ms), float(prior_gbps), int(default_level))
    choices = np.zeros(n, np.int32)
    ttft = ctypes.c_double(0.0)
    _check(lib().cg_adapt_schedule(ctypes.byref(a), bw.ctypes.data, choices.ctypes.data,
                                   ctypes.byref(ttft)), "cg_adapt_schedule")
    return choices.tolist(), ttft.value


def cg_get_status(workspace, stream=None) -> int:
    """Status word of the last cg_encode into `workspace`: 0 (CG_OK) or -4 (CG_ERR_NONFINITE).
    Synchronises the stream."""
    rc = lib().cg_get_status(_ptr(workspace), _stream(stream))
    if rc not in (CG_OK, -4):
        _check(rc, "cg_get_status")
    return rc


def cg_check_finite(p: CodecParams, kv, flag, stream=None) -> bool:
    s, keep = p.c()
    rc = lib().cg_check_finite(ctypes.byref(s), _ptr(kv), _ptr(flag), _stream(stream))
    if rc == -4:
        return False
    _check(rc, "cg_check_finite")
    return True


# --------------------------------------------------------------------------------------------
# token-parallel stream layout (one stream per context, layer, K/V and token)
# --------------------------------------------------------------------------------------------
def cg_num_token_streams(p: CodecParams) -> int:
    s, keep = p.c()
    return int(lib().cg_num_token_streams(ctypes.byref(s)))


def cg_encode_tokens_bound_words(p: CodecParams) -> int:
    s, keep = p.c()
    return int(lib().cg_encode_tokens_bound_words(ctypes.byref(s)))


def cg_encode_tokens_workspace_bytes(p: CodecParams) -> int:
    s, keep = p.c()
    return int(lib().cg_encode_tokens_workspace_bytes(ctypes.byref(s)))


def cg_decode_tokens_workspace_bytes(p: CodecParams) -> int:
    s, keep = p.c()
    return int(lib().cg_decode_tokens_workspace_bytes(ctypes.byref(s)))


def cg_encode_tokens(p: CodecParams, kv, chunk_level, cdf_anchor, cdf_delta, words, offsets,
                     scales, workspace, stream=None):
    s, keep = p.c()
    _check(lib().cg_encode_tokens(ctypes.byref(s), _ptr(kv), _ptr(chunk_level), _ptr(cdf_anchor),
                                  _ptr(cdf_delta), _ptr(words), words.numel(), _ptr(offsets),
                                  _ptr(scales), _ptr(workspace),
                                  workspace.numel() * workspace.element_size(), _stream(stream)),
           "cg_encode_tokens")


def cg_decode_tokens(p: CodecParams, words, offsets, scales, chunk_level, cdf_anchor, cdf_delta,
                     kv_out, workspace, stream=None):
    s, keep = p.c()
    _check(lib().cg_decode_tokens(ctypes.byref(s), _ptr(words), _ptr(offsets), _ptr(scales),
                                  _ptr(chunk_level), _ptr(cdf_anchor), _ptr(cdf_delta),
                                  _ptr(kv_out), _ptr(workspace),
                                  workspace.numel() * workspace.element_size(), _stream(stream)),
           "cg_decode_tokens")


# --------------------------------------------------------------------------------------------
# convenience: allocate outputs with torch and call the above
# --------------------------------------------------------------------------------------------
class Codec:
    """Whole-cache codec on one GPU. Buffers are torch tensors on `device`."""

    def __init__(self, params: CodecParams, device="cuda"):
        import torch
        self.torch = torch
        self.p = params
        self.device = torch.device(device)
        self.n_chunks = cg_num_chunks(params)
        self.n_streams = cg_num_streams(params)
        if self.n_streams == 0:
            raise CodecError(-2, "Codec")
        self.bound_words = cg_encode_bound_words(params)
        self.ws_bytes = cg_encode_workspace_bytes(params)
        self._ws = None

    def _empty(self, shape, dtype):
        return self.torch.empty(shape, dtype=dtype, device=self.device)

    def fit(self, kv, stream=None, status=None, scales=None):
        """Anchor tables [L,2,C,256] and delta tables of every level [NLV,L,2,C,256], in one
        cg_fit_cdf_levels call (which also writes the streams' scales into `scales` [S] if
        given)."""
        t = self.torch
        L, C = self.p.n_layers, self.p.n_channels
        ca = self._empty((L, 2, C, 256), t.int16)
        cd = self._empty((self.p.n_levels, L, 2, C, 256), t.int16)
        cg_fit_cdf_levels(self.p, kv, ca, cd, status, stream, scales)
        return ca, cd

    def fit_per_level(self, kv, stream=None):
        """The same tables from one cg_fit_cdf call per level."""
        t = self.torch
        L, C = self.p.n_layers, self.p.n_channels
        ca = self._empty((L, 2, C, 256), t.int16)
        cd = self._empty((self.p.n_levels, L, 2, C, 256), t.int16)
        for lv in range(self.p.n_levels):
            cg_fit_cdf(self.p, kv, lv, ca if lv == 0 else None, cd[lv], stream)
        return ca, cd

    def workspace(self):
        if self._ws is None:
            self._ws = self._empty((self.ws_bytes,), self.torch.uint8)
        return self._ws

    def status(self, stream=None) -> int:
        """Status of the last encode: 0 (CG_OK) or -4 (CG_ERR_NONFINITE); synchronises."""
        return cg_get_status(self.workspace(), stream)

    def encode(self, kv, chunk_level, cdf_anchor, cdf_delta, stream=None, words=None):
        """Returns (words [bound], offsets [S+1], scales [S]); offsets[S] is the payload length.
        Every call returns new tensors: the payload goes into `words` when given (the caller
        then owns its reuse), else into a fresh buffer. The encode workspace is kept and
        reused across calls (its contents do not outlive a call)."""
        t = self.torch
        if words is None:
            words = self._empty((self.bound_words,), t.int32)
        offsets = self._empty((self.n_streams + 1,), t.int64)
        scales = self._empty((self.n_streams,), t.float32)
        cg_encode(self.p, kv, chunk_level, cdf_anchor, cdf_delta, words, offsets, scales,
                  self.workspace(), stream)
        return words, offsets, scales

    def encode_with_scales(self, kv, chunk_level, cdf_anchor, cdf_delta, scales, stream=None,
                           words=None):
        """(words, offsets) from cg_encode_with_scales, `scales` [S] being the fit's."""
        t = self.torch
        if words is None:
            words = self._empty((self.bound_words,), t.int32)
        offsets = self._empty((self.n_streams + 1,), t.int64)
        cg_encode_with_scales(self.p, kv, chunk_level, cdf_anchor, cdf_delta, scales, words,
                              offsets, self.workspace(), stream)
        return words, offsets

    def decode(self, words, offsets, scales, chunk_level, cdf_anchor, cdf_delta,
               chunk_begin=0, chunk_end=None, out=None, stream=None):
        if chunk_end is None:
            chunk_end = self.n_chunks
        if out is None:
            out = self.torch.zeros(self.p.kv_shape, dtype=self.torch.int16, device=self.device)
        cg_decode(self.p, words, offsets, scales, chunk_level, cdf_anchor, cdf_delta,
                  chunk_begin, chunk_end, out, stream)
        return out

    def encode_tokens(self, kv, chunk_level, cdf_anchor, cdf_delta, stream=None):
        """Token-parallel layout: (words [bound], offsets [St+1], scales [S])."""
        t = self.torch
        words = self._empty((cg_encode_tokens_bound_words(self.p),), t.int32)
        offsets = self._empty((cg_num_token_streams(self.p) + 1,), t.int64)
        scales = self._empty((self.n_streams,), t.float32)
        ws = self._empty((cg_encode_tokens_workspace_bytes(self.p),), t.uint8)
        cg_encode_tokens(self.p, kv, chunk_level, cdf_anchor, cdf_delta, words, offsets, scales,
                         ws, stream)
        return words, offsets, scales

    def decode_tokens(self, words, offsets, scales, chunk_level, cdf_anchor, cdf_delta, out=None,
                      workspace=None, stream=None):
        if out is None:
            out = self.torch.zeros(self.p.kv_shape, dtype=self.torch.int16, device=self.device)
        if workspace is None:
            workspace = self._empty((cg_decode_tokens_workspace_bytes(self.p),), self.torch.uint8)
        cg_decode_tokens(self.p, words, offsets, scales, chunk_level, cdf_anchor, cdf_delta, out,
                         workspace, stream)
        return out
