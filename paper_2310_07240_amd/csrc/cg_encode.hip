// cg_encode.hip — encoder (CacheGen Sec. 5.2: change-based encoding, layer-wise quantization,
// arithmetic coding; Sec. 5.3: each chunk coded independently at its own level).
//
// Launches:
//   encode_kernel   one lane per stream (64 consecutive channels of one (b, c, l, kv) per
//                   wave, so every token row is one coalesced 128-byte load): absmax scale,
//                   quantize, arithmetic-code into a worst-case slot of the workspace, record
//                   the stream's word count;
//   scan_reduce     per-block totals of the word counts (4096 streams per block);
//   scan_top        exclusive scan of the block totals (one workgroup);
//   scan_finish     block-local exclusive scan (wave prefix sums + LDS) plus the block's
//                   carry -> offsets[S + 1];
//   compact         one wave per stream copies its words from the slot to offsets[s].
//
// Arithmetic coder: Witten-Neal-Cleary integer coder, 32-bit registers, 16-bit frequencies.
// Renormalisation is done in one step per symbol instead of one bit at a time:
//   * the leading bits on which low and high agree are shifted out together: their count is
//     clz(low ^ high), and they are output (the first followed by the pending opposite bits);
//   * the "middle half" case that follows (low = 01..., high = 10...) deletes bit 30 of both
//     registers once per step; the number of steps is the run of positions from bit 30 down
//     where low has a 1 and high a 0, i.e. the leading ones of (low & ~high) << 1, and each
//     step adds one pending bit;
//   * high - low grows as rm1 -> (rm1 << n) | (2^n - 1) for n shifts in total.
// This produces exactly the bits of the one-bit-at-a-time definition.
#include "cg_device.h"

namespace {

constexpr int kEncThreads = 256;
constexpr int kScanThreads = 256;
constexpr int kScanItems = 16;
constexpr int kScanBlock = kScanThreads * kScanItems;  // 4096 streams per scan block

struct BitSink {
  uint32_t* out;    // slot base
  uint32_t cap;     // slot capacity in words
  uint32_t nwords;  // words produced
  uint64_t acc;     // output bits not yet in a word, right-aligned
  uint32_t nacc;    // number of bits in acc, < 32 between calls

  __device__ __forceinline__ void put(uint32_t bits, uint32_t nb) {  // nb <= 32
    acc = (acc << nb) | bits;
    nacc += nb;
    if (nacc >= 32) {
      nacc -= 32;
      const uint32_t w = (uint32_t)(acc >> nacc);
      if (nwords < cap) out[nwords] = w;
      ++nwords;
      acc &= (1ull << nacc) - 1ull;
    }
  }
  __device__ __forceinline__ void run(uint32_t bit, uint32_t count) {
    const uint32_t ones = bit ? 0xFFFFFFFFu : 0u;
    while (count >= 32) { put(ones, 32); count -= 32; }
    if (count) put(ones & ((1u << count) - 1u), count);
  }
};

struct EncState {
  uint32_t low;      // low end of the interval
  uint32_t rm1;      // high - low
  uint32_t pending;  // bits owed after the next output bit (opposite value)
};

__device__ __forceinline__ void enc_symbol(EncState& e, BitSink& o, uint32_t clo, uint32_t chi) {
  // R = rm1 + 1 (up to 2^32); new high - old low = (R*chi >> 16) - 1, new low - old low =
  // R*clo >> 16. rm1*c + c = R*c fits in 48 bits.
  const uint32_t lo_off = (uint32_t)(((uint64_t)e.rm1 * clo + clo) >> 16);
  const uint32_t hm1 = (uint32_t)((((uint64_t)e.rm1 * chi + chi) >> 16) - 1ull);
  const uint32_t low = e.low + lo_off;
  const uint32_t rm1 = hm1 - lo_off;
  const uint32_t high = low + rm1;
  const uint32_t n1 = __clz(low ^ high);  // high > low, so n1 <= 31
  if (n1) {
    const uint32_t b0 = low >> 31;
    o.put(b0, 1);
    if (e.pending) { o.run(b0 ^ 1u, e.pending); e.pending = 0; }
    if (n1 > 1) o.put((low << 1) >> (33 - n1), n1 - 1);
  }
  const uint32_t L1 = low << n1, H1 = high << n1;
  const uint32_t m = L1 & ~H1;
  const uint32_t n3 = __clz(~(m << 1));
  e.pending += n3;
  e.low = (L1 & 0x80000000u) | ((L1 << n3) & 0x7FFFFFFFu);
  const uint32_t n = n1 + n3;  // at most 18 (the new range is at least 2^14)
  e.rm1 = (rm1 << n) | ((1u << n) - 1u);
}

__device__ __forceinline__ void enc_finish(EncState& e, BitSink& o) {
  e.pending += 1;
  const uint32_t b = e.low >= 0x40000000u ? 1u : 0u;
  o.put(b, 1);
  o.run(b ^ 1u, e.pending);
  if (o.nacc) o.put(0u, 32 - o.nacc);  // zero-pad to a whole word
}

__global__ __launch_bounds__(kEncThreads) void encode_kernel(
    KParams P, const uint16_t* __restrict__ kv, const uint8_t* __restrict__ chunk_level,
    const uint16_t* __restrict__ cdfA, const uint16_t* __restrict__ cdfD,
    uint32_t* __restrict__ slots, uint32_t slot_words, uint32_t* __restrict__ lens,
    float* __restrict__ scales) {
  const int64_t gw = (int64_t)blockIdx.x * (kEncThreads / 64) + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int64_t nrows = (int64_t)P.B * P.NC * P.L * 2;
  const int64_t bclk = gw / P.nblk;
  const int cb = (int)(gw % P.nblk);
  if (bclk >= nrows) return;
  const int ch = cb * 64 + lane;
  if (ch >= P.C) return;
  const int k = (int)(bclk & 1);
  int64_t r = bclk >> 1;
  const int l = (int)(r % P.L);
  r /= P.L;
  const int c = (int)(r % P.NC);
  const int b = (int)(r / P.NC);
  const int lv = min((int)chunk_level[(int64_t)b * P.NC + c], P.NLV - 1);
  const int t0 = c * P.CL;
  const int n = min(P.CL, P.T - t0);
  const int64_t sidx = cg_stream(P, bclk, ch);
  const uint16_t* x = kv + cg_elem(P, b, l, k, t0, ch);

  float mx = 0.0f;
  for (int j = 0; j < n; ++j) mx = fmaxf(mx, fabsf(cg_h2f(x[(int64_t)j * P.C])));
  const float s = (mx == 0.0f) ? 1.0f : mx / 127.0f;
  scales[sidx] = s;
  const float bw = P.layer_bin[l] * P.level_mult[lv];
  const float w = bw * s;

  const uint16_t* tabA = cdfA + ((int64_t)(l * 2 + k) * P.C + ch) * 256;
  const uint16_t* tabD = cdfD + ((((int64_t)lv * P.L + l) * 2 + k) * P.C + ch) * 256;
  EncState e{0u, 0xFFFFFFFFu, 0u};
  BitSink o{slots + (uint64_t)sidx * slot_words, slot_words, 0u, 0ull, 0u};
  float a = 0.0f;
  int g = 0;
  for (int j = 0; j < n; ++j) {
    const float v = cg_h2f(x[(int64_t)j * P.C]);
    int q;
    const uint16_t* tab;
    if (g == 0) {
      q = cg_quant(v, s);
      a = (float)q * s;
      tab = tabA;
    } else {
      q = cg_quant(v - a, w);
      tab = tabD;
    }
    const int sym = q + 127;
    const uint32_t clo = tab[sym];
    const uint32_t chi = sym == 254 ? CG_TOTAL : (uint32_t)tab[sym + 1];
    enc_symbol(e, o, clo, chi);
    g = (g + 1 == P.G) ? 0 : g + 1;
  }
  enc_finish(e, o);
  // the coder's bound for n symbols; the compaction never writes past the sum of these
  const uint32_t own_bound = (uint32_t)((18ull * (uint64_t)n + 2ull + 31ull) / 32ull);
  lens[sidx] = min(o.nwords, min(own_bound, slot_words));
}

// Block reduction helper: sum of one value per thread of a 256-thread block.
__device__ __forceinline__ uint64_t block_sum(uint64_t v, uint64_t* sh) {
  v = cg_wave_sum<uint64_t>(v);
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) sh[wave] = v;
  __syncthreads();
  uint64_t t = 0;
  for (int i = 0; i < kScanThreads / 64; ++i) t += sh[i];
  __syncthreads();
  return t;
}

__global__ __launch_bounds__(kScanThreads) void scan_reduce(const uint32_t* __restrict__ lens,
                                                            int64_t S,
                                                            uint64_t* __restrict__ partial) {
  __shared__ uint64_t sh[kScanThreads / 64];
  const int64_t base = (int64_t)blockIdx.x * kScanBlock + threadIdx.x * kScanItems;
  uint64_t v = 0;
#pragma unroll
  for (int i = 0; i < kScanItems; ++i) {
    const int64_t idx = base + i;
    if (idx < S) v += lens[idx];
  }
  const uint64_t t = block_sum(v, sh);
  if (threadIdx.x == 0) partial[blockIdx.x] = t;
}

// Exclusive scan of nb block totals in place, by one workgroup.
__global__ __launch_bounds__(kScanThreads) void scan_top(uint64_t* __restrict__ partial,
                                                         int64_t nb) {
  __shared__ uint64_t sh[kScanThreads / 64];
  const int64_t per = (nb + kScanThreads - 1) / kScanThreads;
  const int64_t begin = threadIdx.x * per;
  const int64_t end = min(begin + per, nb);
  uint64_t local = 0;
  for (int64_t i = begin; i < end; ++i) local += partial[i];
  // exclusive scan of the thread totals across the block
  const uint64_t incl = cg_wave_incl_scan64(local);
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 63) sh[wave] = incl;
  __syncthreads();
  uint64_t carry = 0;
  for (int i = 0; i < wave; ++i) carry += sh[i];
  uint64_t run = carry + incl - local;
  for (int64_t i = begin; i < end; ++i) {
    const uint64_t v = partial[i];
    partial[i] = run;
    run += v;
  }
}

__global__ __launch_bounds__(kScanThreads) void scan_finish(const uint32_t* __restrict__ lens,
                                                            int64_t S,
                                                            const uint64_t* __restrict__ partial,
                                                            uint64_t* __restrict__ offsets) {
  __shared__ uint64_t sh[kScanThreads / 64];
  const int64_t base = (int64_t)blockIdx.x * kScanBlock + threadIdx.x * kScanItems;
  uint32_t v[kScanItems];
  uint64_t local = 0;
#pragma unroll
  for (int i = 0; i < kScanItems; ++i) {
    const int64_t idx = base + i;
    v[i] = idx < S ? lens[idx] : 0u;
    local += v[i];
  }
  const uint64_t incl = cg_wave_incl_scan64(local);
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 63) sh[wave] = incl;
  __syncthreads();
  uint64_t run = partial[blockIdx.x] + incl - local;
  for (int i = 0; i < wave; ++i) run += sh[i];
#pragma unroll
  for (int i = 0; i < kScanItems; ++i) {
    const int64_t idx = base + i;
    if (idx < S) offsets[idx] = run;
    run += v[i];
    if (idx == S - 1) offsets[S] = run;
  }
}

__global__ __launch_bounds__(256) void compact_kernel(const uint32_t* __restrict__ slots,
                                                      uint32_t slot_words,
                                                      const uint32_t* __restrict__ lens,
                                                      const uint64_t* __restrict__ offsets,
                                                      int64_t S, uint32_t* __restrict__ words) {
  const int64_t s = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (s >= S) return;
  const int lane = threadIdx.x & 63;
  const uint32_t* src = slots + (uint64_t)s * slot_words;
  uint32_t* dst = words + offsets[s];
  const uint32_t n = lens[s];
  for (uint32_t i = lane; i < n; i += 64) dst[i] = src[i];
}

inline uint64_t align256(uint64_t x) { return (x + 255) & ~(uint64_t)255; }

}  // namespace

EncWorkspace cg_encode_ws_layout(int64_t S, uint32_t slot_words) {
  EncWorkspace w;
  const int64_t nb = (S + kScanBlock - 1) / kScanBlock;
  w.slots_off = 0;
  w.lens_off = align256((uint64_t)S * slot_words * 4ull);
  w.partial_off = align256(w.lens_off + (uint64_t)S * 4ull);
  w.total = align256(w.partial_off + (uint64_t)(nb > 0 ? nb : 1) * 8ull);
  return w;
}

hipError_t cg_launch_encode(const KParams& P, const uint16_t* kv, const uint8_t* chunk_level,
                            const uint16_t* cdf_anchor, const uint16_t* cdf_delta,
                            uint32_t* words, uint64_t* offsets, float* scales, void* ws,
                            uint32_t slot_words, hipStream_t st) {
  const EncWorkspace lay = cg_encode_ws_layout(P.S, slot_words);
  uint8_t* base = static_cast<uint8_t*>(ws);
  uint32_t* slots = reinterpret_cast<uint32_t*>(base + lay.slots_off);
  uint32_t* lens = reinterpret_cast<uint32_t*>(base + lay.lens_off);
  uint64_t* partial = reinterpret_cast<uint64_t*>(base + lay.partial_off);

  const int64_t waves = (int64_t)P.B * P.NC * P.L * 2 * P.nblk;
  const int64_t g1 = (waves + 3) / 4;
  hipLaunchKernelGGL(encode_kernel, dim3((unsigned)g1), dim3(kEncThreads), 0, st, P, kv,
                     chunk_level, cdf_anchor, cdf_delta, slots, slot_words, lens, scales);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t nb = (P.S + kScanBlock - 1) / kScanBlock;
  hipLaunchKernelGGL(scan_reduce, dim3((unsigned)nb), dim3(kScanThreads), 0, st, lens, P.S,
                     partial);
  hipLaunchKernelGGL(scan_top, dim3(1), dim3(kScanThreads), 0, st, partial, nb);
  hipLaunchKernelGGL(scan_finish, dim3((unsigned)nb), dim3(kScanThreads), 0, st, lens, P.S,
                     partial, offsets);
  const int64_t g4 = (P.S + 3) / 4;
  hipLaunchKernelGGL(compact_kernel, dim3((unsigned)g4), dim3(256), 0, st, slots, slot_words,
                     lens, offsets, P.S, words);
  return hipGetLastError();
}
