"""Seeded synthetic KV caches and the codec parameters of the benchmark workloads.

This module only makes inputs: it holds none of the codec's arithmetic, and both the HIP path
and the CPU oracle take their inputs from it. No real model or dataset is available, so the
KV tensors are random with the structure the paper reports for real caches: values of one
(layer, channel) drift slowly along the tokens (Sec. 5.1.1, token-wise locality), channels
differ in scale and a few are outliers, and deeper layers get coarser delta bins in three
equal layer groups (Sec. 5.1.2, App. C.2).

Generator (per context b, layer l, K/V k, channel ch):
  scale ~ LogUniform(0.1, 4); 2 % of channels of a (layer, K/V) (the same channels in every
  context) get scale x20 where the workload has outliers.
  smooth:  x_t = scale * base + W_t, base ~ N(0, 1), W_0 = 0, W_t = W_{t-1} + N(0, (0.05 scale)^2)
  heavy:   x_t = scale * (beta + W_t), beta ~ t_3, W steps 0.5 * z with z ~ t_3 / sqrt(3)
Values are rounded to fp16 (nearest even) after clipping to the finite fp16 range.
Every slab (b, l, k) has its own generator seeded from (seed, b, l, k), so slabs can be made
in parallel and in any order.
"""
from __future__ import annotations

import math
import zlib
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field
import os
import threading

import numpy as np

FP16_MAX = 65504.0


def _groups(n_layers: int, bounds, bins=(0.5, 1.0, 1.5)):
    """Per-layer bin table from layer-group start indices, e.g. bounds=(0, 10, 20)."""
    out = []
    for l in range(n_layers):
        g = sum(1 for b in bounds if l >= b) - 1
        out.append(bins[g])
    return tuple(out)


@dataclass(frozen=True)
class Workload:
    name: str
    n_ctx: int
    n_layers: int
    n_tokens: int
    n_channels: int
    layer_bin: tuple
    level_mult: tuple
    seed: int
    group_size: int = 10
    chunk_len: int = 1536
    outlier_frac: float = 0.0
    heavy_ctx: tuple = ()          # contexts drawn from the heavy-tailed generator
    random_levels: bool = False    # per-(context, chunk) level drawn from the seed
    description: str = ""

    @property
    def n_levels(self) -> int:
        return len(self.level_mult)

    @property
    def n_chunks(self) -> int:
        return -(-self.n_tokens // self.chunk_len)

    @property
    def n_streams(self) -> int:
        return self.n_ctx * self.n_chunks * self.n_layers * 2 * self.n_channels

    @property
    def n_elem(self) -> int:
        return self.n_ctx * self.n_layers * 2 * self.n_tokens * self.n_channels

    @property
    def kv_shape(self):
        return (self.n_ctx, self.n_layers, 2, self.n_tokens, self.n_channels)

    def chunk_levels(self) -> np.ndarray:
        """uint8 [B, NC]: the encoding level of every (context, chunk)."""
        if not self.random_levels:
            return np.zeros((self.n_ctx, self.n_chunks), np.uint8)
        rng = np.random.default_rng([self.seed, 7_000_001])
        return rng.integers(0, self.n_levels, size=(self.n_ctx, self.n_chunks)).astype(np.uint8)

    def with_(self, **kw) -> "Workload":
        d = dict(self.__dict__)
        d.update(kw)
        return Workload(**d)


LEVELS4 = (1.0, 2.0, 4.0, 8.0)

# The five workloads. Shapes follow the models the paper evaluates (Sec. 7.1): K and V channels
# are kv_heads * head_dim; chunks are 1.5K tokens (Sec. 5.3); groups are 10 tokens (Sec. 5.2).
TINY = Workload(
    "tiny_l4_t256_c128", 1, 4, 256, 128, layer_bin=(0.5, 1.0, 1.0, 1.5), level_mult=(1.0,),
    seed=1, description="4 layers, 256 tokens, 2 heads x 64; one 256-token chunk; one level")
MISTRAL_7B_4K = Workload(
    "mistral7b_gqa_t4096", 1, 32, 4096, 1024, layer_bin=_groups(32, (0, 10, 20)),
    level_mult=(1.0,), seed=2, outlier_frac=0.02,
    description="Mistral-7B-shaped GQA KV: 32 layers, 4096 tokens, 8 kv-heads x 128, "
                "2% outlier channels, one level")
LLAMA2_7B_8K = Workload(
    "llama2_7b_mha_t8192", 1, 32, 8192, 4096, layer_bin=_groups(32, (0, 10, 20)),
    level_mult=LEVELS4, seed=3, random_levels=True,
    description="Llama-2-7B-shaped MHA KV: 32 layers, 8192 tokens, 32 heads x 128, "
                "1536-token chunks at 4 levels drawn per chunk")
LLAMA2_70B_16K = Workload(
    "llama2_70b_gqa_t16384", 1, 80, 16384, 1024, layer_bin=_groups(80, (0, 20, 50)),
    level_mult=LEVELS4, seed=4, random_levels=True,
    description="Llama-2-70B-shaped GQA KV: 80 layers, 16384 tokens, 8 kv-heads x 128, "
                "1536-token chunks at mixed levels")
CONCURRENCY_32X2K = Workload(
    "concurrency_32x_mistral_t2048", 32, 32, 2048, 1024, layer_bin=_groups(32, (0, 10, 20)),
    level_mult=LEVELS4, seed=5, outlier_frac=0.02, heavy_ctx=tuple(range(16, 32)),
    random_levels=True,
    description="32 Mistral-7B-shaped contexts of 2048 tokens decoded in one batch; contexts "
                "16-31 heavy-tailed (Student-t 3) with weak locality; per-chunk levels random")

WORKLOADS = {w.name: w for w in (TINY, MISTRAL_7B_4K, LLAMA2_7B_8K, LLAMA2_70B_16K,
                                 CONCURRENCY_32X2K)}


def small(name="small", n_ctx=1, n_layers=3, n_tokens=100, n_channels=70, group_size=10,
          chunk_len=48, level_mult=(1.0, 2.0), seed=11, outlier_frac=0.05, heavy_ctx=(),
          random_levels=True, layer_bin=None) -> Workload:
    """A small workload for parity tests: ragged chunks, channel count off the wave size."""
    if layer_bin is None:
        layer_bin = tuple([0.5, 1.0, 1.5][min(2, 3 * l // max(n_layers, 1))]
                          for l in range(n_layers))
    return Workload(name, n_ctx, n_layers, n_tokens, n_channels, layer_bin=tuple(layer_bin),
                    level_mult=tuple(level_mult), seed=seed, group_size=group_size,
                    chunk_len=chunk_len, outlier_frac=outlier_frac, heavy_ctx=tuple(heavy_ctx),
                    random_levels=random_levels)


def _outlier_channels(w: Workload, l: int, k: int) -> np.ndarray:
    n = int(round(w.outlier_frac * w.n_channels))
    if n == 0:
        return np.zeros(0, np.int64)
    rng = np.random.default_rng([w.seed, 9_000_011, l, k])
    return rng.choice(w.n_channels, size=n, replace=False)


_TLS = threading.local()


def _scratch(T: int, C: int) -> tuple[np.ndarray, np.ndarray]:
    """Two reusable float64 [T, C] buffers per thread (first-touch page faults are costly)."""
    key = (T, C)
    if getattr(_TLS, "key", None) != key:
        _TLS.key = key
        _TLS.a = np.empty((T, C), np.float64)
        _TLS.b = np.empty((T, C), np.float64)
    return _TLS.a, _TLS.b


def _student_t3(rng, shape, out=None, tmp=None):
    """Student-t with 3 degrees of freedom as z / sqrt(chi2_3 / 3) from four normals."""
    if out is None:
        out = np.empty(shape, np.float64)
    if tmp is None:
        tmp = np.empty(shape, np.float64)
    rng.standard_normal(out=tmp)
    np.square(tmp, out=tmp)
    acc = tmp.copy() if tmp.size < 4096 else tmp          # chi2 accumulator
    for _ in range(2):
        rng.standard_normal(out=out)
        np.square(out, out=out)
        acc += out
    acc /= 3.0
    np.sqrt(acc, out=acc)
    rng.standard_normal(out=out)
    out /= acc
    return out


def slab_into(w: Workload, b: int, l: int, k: int, out: np.ndarray) -> np.ndarray:
    """Fill out (fp16 view, [T', C] with T' <= T) with context b, layer l, K/V k."""
    T, C = out.shape
    rng = np.random.default_rng([w.seed, b, l, k])
    scale = np.exp(rng.uniform(math.log(0.1), math.log(4.0), size=C))
    oc = _outlier_channels(w, l, k)
    scale[oc] *= 20.0
    x, z = _scratch(T, C)
    x[0] = 0.0
    if b in w.heavy_ctx:
        beta = _student_t3(rng, (C,))
        _student_t3(rng, (T - 1, C), out=z[: T - 1], tmp=x[1:])
        z[: T - 1] *= 0.5 / math.sqrt(3.0)
        np.cumsum(z[: T - 1], axis=0, out=x[1:])
        x += beta
        x *= scale
    else:
        base = rng.standard_normal(C)
        rng.standard_normal(out=z[: T - 1])
        z[: T - 1] *= 0.05 * scale
        np.cumsum(z[: T - 1], axis=0, out=x[1:])
        x += scale * base
    np.clip(x, -FP16_MAX, FP16_MAX, out=x)
    np.copyto(out, x, casting="unsafe")          # float64 -> float16, round to nearest even
    return out


def slab(w: Workload, b: int, l: int, k: int, n_tokens: int | None = None) -> np.ndarray:
    """fp16 values [T, C] of context b, layer l, K/V k (first n_tokens rows if given)."""
    out = np.empty((w.n_tokens, w.n_channels), np.float16)
    slab_into(w, b, l, k, out)
    return out if n_tokens is None else out[:n_tokens].copy()


def generate(w: Workload, out: np.ndarray | None = None, threads: int | None = None) -> np.ndarray:
    """The whole KV cache as fp16 [B, L, 2, T, C]; fills `out` (fp16 or uint16 view) if given."""
    if out is None:
        out = np.empty(w.kv_shape, np.float16)
    o = out.view(np.float16).reshape(w.kv_shape)
    jobs = [(b, l, k) for b in range(w.n_ctx) for l in range(w.n_layers) for k in range(2)]

    def run(j):
        b, l, k = j
        slab_into(w, b, l, k, o[b, l, k])

    threads = threads or min(16, max(1, len(os.sched_getaffinity(0))))
    if threads == 1 or len(jobs) == 1:
        for j in jobs:
            run(j)
    else:
        with ThreadPoolExecutor(threads) as ex:
            list(ex.map(run, jobs))
    return out


def edge_case_kv(w: Workload, kind: str) -> np.ndarray:
    """Inputs for the codec's degenerate cases, on the shape of workload w:
    'zeros'      every value 0 (scale falls back to 1, every symbol is 127);
    'constant'   every channel constant over the tokens (every delta symbol is 127);
    'subnormal'  tiny values including fp16 subnormals;
    'ties'       values at exact half-bin points of the anchor quantizer;
    'clamp'      a spike per group that drives deltas into the +-127 clamp;
    'signs'      alternating signs and +-0."""
    rng = np.random.default_rng([w.seed, 5_555, zlib.crc32(kind.encode())])
    shape = w.kv_shape
    if kind == "zeros":
        return np.zeros(shape, np.float16)
    if kind == "constant":
        v = rng.standard_normal((w.n_ctx, w.n_layers, 2, 1, w.n_channels))
        return np.broadcast_to(v, shape).astype(np.float16)
    if kind == "subnormal":
        bits = rng.integers(0, 0x0400, size=shape, dtype=np.uint16)      # subnormals and 0
        sign = rng.integers(0, 2, size=shape, dtype=np.uint16) << 15
        bits = bits | sign
        normal = rng.random(shape) < 0.1
        bits[normal] = (rng.integers(0x0400, 0x0800, size=int(normal.sum()), dtype=np.uint16)
                        | sign[normal])
        return bits.view(np.float16)
    if kind == "ties":
        # integers scaled so that absmax = 127: x / s lands on n + 0.5 for many tokens
        q = rng.integers(-126, 126, size=shape).astype(np.float64) + 0.5
        q[..., 0, :] = 127.0
        return q.astype(np.float16)
    if kind == "clamp":
        x = rng.standard_normal(shape) * 0.01
        x[..., 5::10, :] += 100.0                                  # mid-group spikes
        x[..., 0, :] = 100.0
        return x.astype(np.float16)
    if kind == "signs":
        x = rng.standard_normal(shape)
        x[..., ::2, :] *= -1
        x[..., 3::7, :] = -0.0
        return x.astype(np.float16)
    raise ValueError(kind)
