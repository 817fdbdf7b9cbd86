// cg_api.hip — the C ABI (include/cachegen.h): argument and shape validation on the host,
// then kernel launches on the caller's stream. Nothing here allocates device memory.
#include <math.h>
#include <string.h>

#include "../../include/cachegen.h"
#include "cg_device.h"

namespace {

// Validate cg_params and fill the kernel-side view. Returns CG_OK or an error code.
int make_kparams(const cg_params* p, KParams* K) {
  if (!p) return CG_ERR_ARG;
  if (p->n_ctx <= 0 || p->n_layers <= 0 || p->n_tokens <= 0 || p->n_channels <= 0)
    return CG_ERR_SHAPE;
  if (p->group_size < 1 || p->chunk_len < 1) return CG_ERR_SHAPE;
  if (p->n_levels < 1 || p->n_levels > CG_MAX_LEVELS) return CG_ERR_SHAPE;
  if (p->n_layers > CG_MAX_LAYERS) return CG_ERR_SHAPE;
  if (!p->layer_bin || !p->level_mult) return CG_ERR_ARG;
  // index space: element and stream counts must fit comfortably in 63 bits, and the
  // per-workgroup grids in 32 bits
  const double elems = (double)p->n_ctx * p->n_layers * 2.0 * p->n_tokens * p->n_channels;
  if (elems > 9.0e15) return CG_ERR_SHAPE;
  for (int l = 0; l < p->n_layers; ++l)
    if (!(isfinite(p->layer_bin[l]) && p->layer_bin[l] > 0.0f)) return CG_ERR_PARAM;
  for (int v = 0; v < p->n_levels; ++v)
    if (!(isfinite(p->level_mult[v]) && p->level_mult[v] > 0.0f)) return CG_ERR_PARAM;
  memset(K, 0, sizeof(*K));
  K->B = p->n_ctx;
  K->L = p->n_layers;
  K->T = p->n_tokens;
  K->C = p->n_channels;
  K->G = p->group_size;
  K->CL = p->chunk_len;
  K->NC = (int32_t)(((int64_t)p->n_tokens + p->chunk_len - 1) / p->chunk_len);
  K->NLV = p->n_levels;
  K->nblk = (p->n_channels + 63) / 64;
  K->S = (int64_t)K->B * K->NC * K->L * 2 * K->C;
  const int64_t waves = (int64_t)K->B * K->NC * K->L * 2 * K->nblk;
  if (waves > 0x7fffffffLL) return CG_ERR_SHAPE;
  for (int l = 0; l < p->n_layers; ++l) K->layer_bin[l] = p->layer_bin[l];
  for (int v = 0; v < p->n_levels; ++v) K->level_mult[v] = p->level_mult[v];
  return CG_OK;
}

// Largest slot (in words) any stream can need: ceil((18 n + 2) / 32) for its token count n.
uint32_t slot_words_for(const KParams& K) {
  const int64_t n = K.CL < K.T ? K.CL : K.T;
  return (uint32_t)((18ull * (uint64_t)n + 2ull + 31ull) / 32ull);
}

bool aligned(const void* ptr, size_t a) { return ((uintptr_t)ptr % a) == 0; }

}  // namespace

extern "C" {

int64_t cg_num_chunks(const cg_params* p) {
  KParams K;
  return make_kparams(p, &K) == CG_OK ? K.NC : 0;
}

int64_t cg_num_streams(const cg_params* p) {
  KParams K;
  return make_kparams(p, &K) == CG_OK ? K.S : 0;
}

uint64_t cg_encode_bound_words(const cg_params* p) {
  KParams K;
  if (make_kparams(p, &K) != CG_OK) return 0;
  const int64_t per_chunk = (int64_t)K.B * K.L * 2 * K.C;
  uint64_t total = 0;
  for (int c = 0; c < K.NC; ++c) {
    const int64_t n = (c + 1) * (int64_t)K.CL <= K.T ? K.CL : K.T - (int64_t)c * K.CL;
    total += (uint64_t)per_chunk * ((18ull * (uint64_t)n + 2ull + 31ull) / 32ull);
  }
  return total + CG_TAIL_WORDS;
}

uint64_t cg_encode_workspace_bytes(const cg_params* p) {
  KParams K;
  if (make_kparams(p, &K) != CG_OK) return 0;
  return cg_encode_ws_layout(K, slot_words_for(K)).total;
}

int cg_fit_cdf(const cg_params* p, const uint16_t* kv_f16, int32_t level, uint16_t* cdf_anchor,
               uint16_t* cdf_delta_level, hipStream_t stream) {
  KParams K;
  int rc = make_kparams(p, &K);
  if (rc != CG_OK) return rc;
  if (!kv_f16 || !cdf_delta_level) return CG_ERR_ARG;
  if (level < 0 || level >= K.NLV) return CG_ERR_ARG;
  if (!aligned(cdf_delta_level, 8) || (cdf_anchor && !aligned(cdf_anchor, 8)) ||
      !aligned(kv_f16, 2))
    return CG_ERR_ARG;
  return cg_launch_fit(K, kv_f16, level, cdf_anchor, cdf_delta_level, stream) == hipSuccess
             ? CG_OK
             : CG_ERR_HIP;
}

int cg_encode(const cg_params* p, const uint16_t* kv_f16, const uint8_t* chunk_level,
              const uint16_t* cdf_anchor, const uint16_t* cdf_delta, uint32_t* words,
              uint64_t words_cap, uint64_t* offsets, float* scales, void* workspace,
              uint64_t workspace_bytes, hipStream_t stream) {
  KParams K;
  int rc = make_kparams(p, &K);
  if (rc != CG_OK) return rc;
  if (!kv_f16 || !chunk_level || !cdf_anchor || !cdf_delta || !words || !offsets || !scales ||
      !workspace)
    return CG_ERR_ARG;
  if (!aligned(workspace, 256) || !aligned(offsets, 8) || !aligned(words, 4) ||
      !aligned(scales, 4))
    return CG_ERR_ARG;
  if (words_cap < cg_encode_bound_words(p)) return CG_ERR_CAPACITY;
  const uint32_t slot = slot_words_for(K);
  if (workspace_bytes < cg_encode_ws_layout(K, slot).total) return CG_ERR_CAPACITY;
  return cg_launch_encode(K, kv_f16, chunk_level, cdf_anchor, cdf_delta, words, offsets, scales,
                          workspace, slot, stream) == hipSuccess
             ? CG_OK
             : CG_ERR_HIP;
}

int cg_decode(const cg_params* p, const uint32_t* words, const uint64_t* offsets,
              const float* scales, const uint8_t* chunk_level, const uint16_t* cdf_anchor,
              const uint16_t* cdf_delta, int32_t chunk_begin, int32_t chunk_end,
              uint16_t* kv_out_f16, hipStream_t stream) {
  KParams K;
  int rc = make_kparams(p, &K);
  if (rc != CG_OK) return rc;
  if (!words || !offsets || !scales || !chunk_level || !cdf_anchor || !cdf_delta || !kv_out_f16)
    return CG_ERR_ARG;
  if (chunk_begin < 0 || chunk_end > K.NC || chunk_begin > chunk_end) return CG_ERR_ARG;
  if (!aligned(cdf_anchor, 16) || !aligned(cdf_delta, 16) || !aligned(offsets, 8) ||
      !aligned(words, 4) || !aligned(kv_out_f16, 2))
    return CG_ERR_ARG;
  if (chunk_begin == chunk_end) return CG_OK;
  return cg_launch_decode(K, words, offsets, scales, chunk_level, cdf_anchor, cdf_delta,
                          chunk_begin, chunk_end, kv_out_f16, stream) == hipSuccess
             ? CG_OK
             : CG_ERR_HIP;
}

int cg_check_finite(const cg_params* p, const uint16_t* kv_f16, uint32_t* flag_dev,
                    hipStream_t stream) {
  KParams K;
  int rc = make_kparams(p, &K);
  if (rc != CG_OK) return rc;
  if (!kv_f16 || !flag_dev) return CG_ERR_ARG;
  const int64_t n = (int64_t)K.B * K.L * 2 * K.T * K.C;
  if (cg_launch_check_finite(kv_f16, n, flag_dev, stream) != hipSuccess) return CG_ERR_HIP;
  uint32_t h = 0;
  if (hipMemcpyAsync(&h, flag_dev, 4, hipMemcpyDeviceToHost, stream) != hipSuccess)
    return CG_ERR_HIP;
  if (hipStreamSynchronize(stream) != hipSuccess) return CG_ERR_HIP;
  return h ? CG_ERR_NONFINITE : CG_OK;
}

const char* cg_strerror(int code) {
  switch (code) {
    case CG_OK: return "ok";
    case CG_ERR_ARG: return "invalid argument (null or misaligned pointer, level or chunk range)";
    case CG_ERR_SHAPE: return "invalid shape (a dimension, group size, chunk length or level count)";
    case CG_ERR_CAPACITY: return "output or workspace capacity too small";
    case CG_ERR_NONFINITE: return "KV input holds NaN or Inf";
    case CG_ERR_HIP: return "HIP runtime error";
    case CG_ERR_PARAM: return "a layer bin width or level multiplier is not finite and positive";
    default: return "unknown error code";
  }
}

}  // extern "C"

// ---- finiteness scan ----------------------------------------------------------------------
namespace {
__global__ __launch_bounds__(256) void zero_flag(uint32_t* flag) { *flag = 0u; }

__global__ __launch_bounds__(256) void finite_kernel(const uint16_t* __restrict__ kv, int64_t n,
                                                     uint32_t* flag) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  uint32_t bad = 0;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
    bad |= ((kv[i] & 0x7c00u) == 0x7c00u) ? 1u : 0u;
  if (__any(bad) && (threadIdx.x & 63) == 0) atomicOr(flag, 1u);
}
}  // namespace

hipError_t cg_launch_check_finite(const uint16_t* kv, int64_t n, uint32_t* flag,
                                  hipStream_t st) {
  hipLaunchKernelGGL(zero_flag, dim3(1), dim3(1), 0, st, flag);
  int64_t blocks = (n + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(finite_kernel, dim3((unsigned)blocks), dim3(256), 0, st, kv, n, flag);
  return hipGetLastError();
}
