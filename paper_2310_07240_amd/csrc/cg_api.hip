// cg_api.hip — the C ABI (include/cachegen.h): argument and shape validation on the host,
// then kernel launches on the caller's stream. Nothing here allocates device memory.
#include <math.h>
#include <string.h>

#include <chrono>
#include <mutex>
#include <thread>
#include <vector>

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
  return (uint32_t)(((18ull * (uint64_t)n + 2ull + 31ull) / 32ull + 3ull) & ~3ull);   // whole 16-byte chunks
}

bool aligned(const void* ptr, size_t a) { return ((uintptr_t)ptr % a) == 0; }

// Scratch of cg_encode_noalloc: one static device buffer per GPU (each device holds its own copy
// of the array, at its own address, for the life of the process). Host code never uses the
// array's name as an address: the device address of each GPU's copy is looked up once per
// device with hipGetSymbolAddress and kept here.
static __device__ __align__(256) uint8_t scratch[CG_NOALLOC_SCRATCH_BYTES];
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's scratch, or nullptr if it cannot be found.
void* scratch_of_current_device() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return nullptr;
    g_scratch_ptr[dev] = ptr;
  }
  return g_scratch_ptr[dev];
}

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
  if (!aligned(cdf_delta_level, 16) || (cdf_anchor && !aligned(cdf_anchor, 16)) ||
      !aligned(kv_f16, 2))
    return CG_ERR_ARG;
  return cg_launch_fit(K, kv_f16, level, cdf_anchor, cdf_delta_level, stream) == hipSuccess
             ? CG_OK
             : CG_ERR_HIP;
}

int cg_fit_cdf_levels(const cg_params* p, const uint16_t* kv_f16, uint16_t* cdf_anchor,
                      uint16_t* cdf_delta, uint32_t* status, float* scales, hipStream_t stream) {
  KParams K;
  int rc = make_kparams(p, &K);
  if (rc != CG_OK) return rc;
  if (!kv_f16 || !cdf_anchor || !cdf_delta) return CG_ERR_ARG;
  if (!aligned(cdf_anchor, 16) || !aligned(cdf_delta, 16) || !aligned(kv_f16, 2) ||
      (status && !aligned(status, 4)) || (scales && !aligned(scales, 4)))
    return CG_ERR_ARG;
  return cg_launch_fit_levels(K, kv_f16, cdf_anchor, cdf_delta, status, scales, stream) ==
                 hipSuccess
             ? CG_OK
             : CG_ERR_HIP;
}

int cg_fit_cdf_global(const cg_params* p, const uint16_t* kv_f16, int32_t level,
                      uint16_t* cdf_anchor, uint16_t* cdf_delta_level, void* workspace,
                      uint64_t workspace_bytes, hipStream_t stream) {
  KParams K;
  int rc = make_kparams(p, &K);
  if (rc != CG_OK) return rc;
  if (!kv_f16 || !cdf_delta_level || !workspace) return CG_ERR_ARG;
  if (level < 0 || level >= K.NLV) return CG_ERR_ARG;
  if (!aligned(cdf_delta_level, 16) || (cdf_anchor && !aligned(cdf_anchor, 16)) ||
      !aligned(kv_f16, 2) || !aligned(workspace, 256))
    return CG_ERR_ARG;
  if (workspace_bytes < CG_FIT_GLOBAL_WORKSPACE_BYTES) return CG_ERR_CAPACITY;
  return cg_launch_fit_global(K, kv_f16, level, cdf_anchor, cdf_delta_level, workspace,
                              stream) == hipSuccess
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
      !aligned(scales, 4) || !aligned(kv_f16, 2) || !aligned(cdf_anchor, 16) ||
      !aligned(cdf_delta, 16))
    return CG_ERR_ARG;
  if (words_cap < cg_encode_bound_words(p)) return CG_ERR_CAPACITY;
  const uint32_t slot = slot_words_for(K);
  if (workspace_bytes < cg_encode_ws_layout(K, slot).total) return CG_ERR_CAPACITY;
  return cg_launch_encode(K, kv_f16, chunk_level, cdf_anchor, cdf_delta, words, offsets, scales,
                          workspace, slot, stream) == hipSuccess
             ? CG_OK
             : CG_ERR_HIP;
}

int cg_encode_with_scales(const cg_params* p, const uint16_t* kv_f16, const uint8_t* chunk_level,
                          const uint16_t* cdf_anchor, const uint16_t* cdf_delta,
                          const float* scales, uint32_t* words, uint64_t words_cap,
                          uint64_t* offsets, void* workspace, uint64_t workspace_bytes,
                          hipStream_t stream) {
  KParams K;
  int rc = make_kparams(p, &K);
  if (rc != CG_OK) return rc;
  if (!kv_f16 || !chunk_level || !cdf_anchor || !cdf_delta || !words || !offsets || !scales ||
      !workspace)
    return CG_ERR_ARG;
  if (!aligned(workspace, 256) || !aligned(offsets, 8) || !aligned(words, 4) ||
      !aligned(scales, 4) || !aligned(kv_f16, 2) || !aligned(cdf_anchor, 16) ||
      !aligned(cdf_delta, 16))
    return CG_ERR_ARG;
  if (words_cap < cg_encode_bound_words(p)) return CG_ERR_CAPACITY;
  const uint32_t slot = slot_words_for(K);
  if (workspace_bytes < cg_encode_ws_layout(K, slot).total) return CG_ERR_CAPACITY;
  // the kernels only read `scales` in this mode
  return cg_launch_encode(K, kv_f16, chunk_level, cdf_anchor, cdf_delta, words, offsets,
                          const_cast<float*>(scales), workspace, slot, stream, nullptr,
                          true) == hipSuccess
             ? CG_OK
             : CG_ERR_HIP;
}

int cg_encode_noalloc(const cg_params* p, const uint16_t* kv_f16, const uint8_t* chunk_level,
                      const uint16_t* cdf_anchor, const uint16_t* cdf_delta, uint32_t* words,
                      uint64_t words_cap, uint64_t* offsets, float* scales, uint32_t* status,
                      hipStream_t stream) {
  KParams K;
  int rc = make_kparams(p, &K);
  if (rc != CG_OK) return rc;
  if (!kv_f16 || !chunk_level || !cdf_anchor || !cdf_delta || !words || !offsets || !scales)
    return CG_ERR_ARG;
  if (!aligned(offsets, 8) || !aligned(words, 4) || !aligned(scales, 4) || !aligned(kv_f16, 2) ||
      !aligned(cdf_anchor, 16) || !aligned(cdf_delta, 16) || (status && !aligned(status, 4)))
    return CG_ERR_ARG;
  if (words_cap < cg_encode_bound_words(p)) return CG_ERR_CAPACITY;
  const uint32_t slot = slot_words_for(K);
  if (cg_encode_ws_layout(K, slot).total > (uint64_t)CG_NOALLOC_SCRATCH_BYTES)
    return CG_ERR_SCRATCH;
  void* ws = scratch_of_current_device();
  if (!ws) return CG_ERR_HIP;
  return cg_launch_encode(K, kv_f16, chunk_level, cdf_anchor, cdf_delta, words, offsets, scales,
                          ws, slot, stream, status) == hipSuccess
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
      !aligned(words, 4) || !aligned(scales, 4) || !aligned(kv_out_f16, 2))
    return CG_ERR_ARG;
  if (chunk_begin == chunk_end) return CG_OK;
  return cg_launch_decode(K, words, offsets, scales, chunk_level, cdf_anchor, cdf_delta,
                          chunk_begin, chunk_end, kv_out_f16, stream) == hipSuccess
             ? CG_OK
             : CG_ERR_HIP;
}

int64_t cg_num_token_streams(const cg_params* p) {
  KParams K;
  return make_kparams(p, &K) == CG_OK ? cg_token_streams(K) : 0;
}

uint64_t cg_encode_tokens_bound_words(const cg_params* p) {
  KParams K;
  if (make_kparams(p, &K) != CG_OK) return 0;
  return (uint64_t)cg_token_streams(K) * cg_token_slot_words(K) + CG_TAIL_WORDS;
}

uint64_t cg_encode_tokens_workspace_bytes(const cg_params* p) {
  KParams K;
  if (make_kparams(p, &K) != CG_OK) return 0;
  return cg_encode_tokens_ws_layout(K).total;
}

uint64_t cg_decode_tokens_workspace_bytes(const cg_params* p) {
  KParams K;
  if (make_kparams(p, &K) != CG_OK) return 0;
  return (uint64_t)cg_token_streams(K) * (uint64_t)K.C;
}

int cg_encode_tokens(const cg_params* p, const uint16_t* kv_f16, const uint8_t* chunk_level,
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
      !aligned(scales, 4) || !aligned(kv_f16, 2) || !aligned(cdf_anchor, 16) ||
      !aligned(cdf_delta, 16))
    return CG_ERR_ARG;
  if (words_cap < cg_encode_tokens_bound_words(p)) return CG_ERR_CAPACITY;
  if (workspace_bytes < cg_encode_tokens_ws_layout(K).total) return CG_ERR_CAPACITY;
  return cg_launch_encode_tokens(K, kv_f16, chunk_level, cdf_anchor, cdf_delta, words, offsets,
                                 scales, workspace, stream) == hipSuccess
             ? CG_OK
             : CG_ERR_HIP;
}

int cg_decode_tokens(const cg_params* p, const uint32_t* words, const uint64_t* offsets,
                     const float* scales, const uint8_t* chunk_level,
                     const uint16_t* cdf_anchor, const uint16_t* cdf_delta,
                     uint16_t* kv_out_f16, void* workspace, uint64_t workspace_bytes,
                     hipStream_t stream) {
  KParams K;
  int rc = make_kparams(p, &K);
  if (rc != CG_OK) return rc;
  if (!words || !offsets || !scales || !chunk_level || !cdf_anchor || !cdf_delta ||
      !kv_out_f16 || !workspace)
    return CG_ERR_ARG;
  if (!aligned(cdf_anchor, 16) || !aligned(cdf_delta, 16) || !aligned(offsets, 8) ||
      !aligned(words, 4) || !aligned(scales, 4) || !aligned(kv_out_f16, 2) ||
      !aligned(workspace, 256))
    return CG_ERR_ARG;
  if (workspace_bytes < cg_decode_tokens_workspace_bytes(p)) return CG_ERR_CAPACITY;
  return cg_launch_decode_tokens(K, words, offsets, scales, chunk_level, cdf_anchor, cdf_delta,
                                 static_cast<uint8_t*>(workspace), kv_out_f16,
                                 stream) == hipSuccess
             ? CG_OK
             : CG_ERR_HIP;
}

int cg_decode_streamed(const cg_params* p, const uint32_t* words_host,
                       const uint64_t* offsets_host, uint32_t* words_dev, uint64_t words_cap,
                       const uint64_t* offsets_dev, const float* scales_dev,
                       const uint8_t* chunk_level_dev, const uint16_t* cdf_anchor_dev,
                       const uint16_t* cdf_delta_dev, uint16_t* kv_out_dev, double link_gbps,
                       hipStream_t decode_stream, hipStream_t copy_stream,
                       cg_stream_stats* stats) {
  KParams K;
  int rc = make_kparams(p, &K);
  if (rc != CG_OK) return rc;
  if (!words_host || !offsets_host || !words_dev || !offsets_dev || !scales_dev ||
      !chunk_level_dev || !cdf_anchor_dev || !cdf_delta_dev || !kv_out_dev)
    return CG_ERR_ARG;
  if (!aligned(cdf_anchor_dev, 16) || !aligned(cdf_delta_dev, 16) || !aligned(offsets_dev, 8) ||
      !aligned(words_dev, 4) || !aligned(scales_dev, 4) || !aligned(kv_out_dev, 2) ||
      !aligned(words_host, 4) || !aligned(offsets_host, 8))
    return CG_ERR_ARG;
  const int NC = K.NC;
  const int64_t per_chunk = (int64_t)K.L * 2 * K.C;   // streams of one (context, chunk)
  // the copies follow offsets_host: check every boundary they use before issuing anything
  if (offsets_host[0] != 0) return CG_ERR_ARG;
  for (int64_t i = 0; i < (int64_t)K.B * NC; ++i)
    if (offsets_host[(i + 1) * per_chunk] < offsets_host[i * per_chunk]) return CG_ERR_ARG;
  if (words_cap < CG_TAIL_WORDS || offsets_host[K.S] > words_cap - CG_TAIL_WORDS)
    return CG_ERR_CAPACITY;
  const double bits_per_ms = link_gbps > 0.0 ? link_gbps * 1.0e6 : 0.0;

  // events: start, then per chunk copy done, decode start, decode done
  std::vector<hipEvent_t> ev(1 + 3 * (size_t)NC, nullptr);
  auto cleanup = [&]() {
    for (hipEvent_t e : ev)
      if (e) (void)hipEventDestroy(e);
  };
  for (hipEvent_t& e : ev)
    if (hipEventCreate(&e) != hipSuccess) { e = nullptr; cleanup(); return CG_ERR_HIP; }
  hipEvent_t ev0 = ev[0];
  auto ev_copy = [&](int c) { return ev[1 + 3 * c]; };
  auto ev_dbeg = [&](int c) { return ev[2 + 3 * c]; };
  auto ev_dend = [&](int c) { return ev[3 + 3 * c]; };

  bool ok = hipEventRecord(ev0, copy_stream) == hipSuccess;
  const auto t0 = std::chrono::steady_clock::now();
  uint64_t sent_words = 0;
  for (int c = 0; ok && c < NC; ++c) {
    uint64_t chunk_words = 0;
    for (int b = 0; b < K.B; ++b) {
      const int64_t s0 = ((int64_t)b * NC + c) * per_chunk;
      chunk_words += offsets_host[s0 + per_chunk] - offsets_host[s0];
    }
    if (bits_per_ms > 0.0) {   // the chunk's last byte arrives over the link
      const double due_ms = (double)(sent_words + chunk_words) * 32.0 / bits_per_ms;
      std::this_thread::sleep_until(
          t0 + std::chrono::duration_cast<std::chrono::steady_clock::duration>(
                   std::chrono::duration<double, std::milli>(due_ms)));
    }
    for (int b = 0; ok && b < K.B; ++b) {
      const int64_t s0 = ((int64_t)b * NC + c) * per_chunk;
      const uint64_t w0 = offsets_host[s0], w1 = offsets_host[s0 + per_chunk];
      if (w1 > w0)
        ok = hipMemcpyAsync(words_dev + w0, words_host + w0, (w1 - w0) * sizeof(uint32_t),
                            hipMemcpyHostToDevice, copy_stream) == hipSuccess;
    }
    ok = ok && hipEventRecord(ev_copy(c), copy_stream) == hipSuccess &&
         hipStreamWaitEvent(decode_stream, ev_copy(c), 0) == hipSuccess &&
         hipEventRecord(ev_dbeg(c), decode_stream) == hipSuccess &&
         cg_launch_decode(K, words_dev, offsets_dev, scales_dev, chunk_level_dev, cdf_anchor_dev,
                          cdf_delta_dev, c, c + 1, kv_out_dev, decode_stream) == hipSuccess &&
         hipEventRecord(ev_dend(c), decode_stream) == hipSuccess;
    sent_words += chunk_words;
  }
  // wait for everything issued, whether or not a step failed
  const bool synced = hipStreamSynchronize(copy_stream) == hipSuccess &&
                      hipStreamSynchronize(decode_stream) == hipSuccess;
  bool timed = true;
  if (ok && synced && stats) {
    float tx = 0.0f, tot = 0.0f, d = 0.0f;
    double dsum = 0.0;
    timed = hipEventElapsedTime(&tx, ev0, ev_copy(NC - 1)) == hipSuccess &&
            hipEventElapsedTime(&tot, ev0, ev_dend(NC - 1)) == hipSuccess;
    for (int c = 0; timed && c < NC; ++c) {
      timed = hipEventElapsedTime(&d, ev_dbeg(c), ev_dend(c)) == hipSuccess;
      dsum += d;
      float tc = 0.0f, tb = 0.0f, te = 0.0f;
      timed = timed && hipEventElapsedTime(&tc, ev0, ev_copy(c)) == hipSuccess &&
              hipEventElapsedTime(&tb, ev0, ev_dbeg(c)) == hipSuccess &&
              hipEventElapsedTime(&te, ev0, ev_dend(c)) == hipSuccess;
      if (stats->chunk_copy_done_ms) stats->chunk_copy_done_ms[c] = tc;
      if (stats->chunk_decode_begin_ms) stats->chunk_decode_begin_ms[c] = tb;
      if (stats->chunk_decode_end_ms) stats->chunk_decode_end_ms[c] = te;
    }
    stats->n_chunks = NC;
    stats->transfer_ms = tx;
    stats->total_ms = tot;
    stats->decode_sum_ms = dsum;
    double h = dsum > 0.0 ? 1.0 - ((double)tot - (double)tx) / dsum : 1.0;
    stats->hidden_fraction = h < 0.0 ? 0.0 : (h > 1.0 ? 1.0 : h);
  }
  cleanup();
  return ok && synced && timed ? CG_OK : CG_ERR_HIP;
}

int cg_adapt_schedule(const cg_adapt_params* a, const double* bandwidth_gbps,
                      int32_t* choice_out, double* ttft_ms_out) {
  if (!a || !bandwidth_gbps || !choice_out || !ttft_ms_out || !a->level_bytes || !a->text_bytes)
    return CG_ERR_ARG;
  const int N = a->n_chunks, V = a->n_levels;
  if (N <= 0 || V <= 0 || a->default_level < 0 || a->default_level >= V) return CG_ERR_ARG;
  for (int c = 0; c < N; ++c)
    if (!(bandwidth_gbps[c] > 0.0)) return CG_ERR_ARG;
  // milliseconds to move `bytes` at `gbps`
  auto ms_at = [](double bytes, double gbps) { return bytes * 8.0 / (gbps * 1.0e6); };
  double elapsed = 0.0;
  bool have_est = a->prior_gbps > 0.0;
  double est = a->prior_gbps;
  for (int c = 0; c < N; ++c) {
    const double remaining = a->slo_ms - elapsed;
    int choice = -2;
    if (a->recompute_ms) {   // text: the receiver recomputes the remaining chunks' KV
      double t_text = 0.0;
      for (int i = c; i < N; ++i) t_text += a->recompute_ms[i];
      if (t_text <= remaining) choice = -1;
    }
    if (choice == -2) {
      if (!have_est) {
        choice = a->default_level;
      } else {
        for (int v = 0; v < V && choice == -2; ++v) {   // lowest compression loss first
          double bytes = 0.0;
          for (int i = c; i < N; ++i) bytes += a->level_bytes[(size_t)i * V + v];
          if (ms_at(bytes, est) <= remaining) choice = v;
        }
        if (choice == -2) choice = V - 1;
      }
    }
    const double bytes = choice < 0 ? a->text_bytes[c] : a->level_bytes[(size_t)c * V + choice];
    elapsed += ms_at(bytes, bandwidth_gbps[c]);
    if (choice < 0) elapsed += a->recompute_ms[c];
    choice_out[c] = choice;
    est = bandwidth_gbps[c];   // the next chunk's estimate: this chunk's measured throughput
    have_est = true;
  }
  *ttft_ms_out = elapsed;
  return CG_OK;
}

int cg_get_status(const void* workspace, hipStream_t stream) {
  if (!workspace || !aligned(workspace, 4)) return CG_ERR_ARG;
  uint32_t h = 0;
  if (hipMemcpyAsync(&h, workspace, 4, hipMemcpyDeviceToHost, stream) != hipSuccess)
    return CG_ERR_HIP;
  if (hipStreamSynchronize(stream) != hipSuccess) return CG_ERR_HIP;
  return h ? CG_ERR_NONFINITE : CG_OK;
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
    case CG_ERR_SCRATCH:
      return "the cache needs more scratch than the static buffer of cg_encode_noalloc holds";
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
