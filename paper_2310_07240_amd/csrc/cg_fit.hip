// cg_fit.hip — symbol-distribution fit (CacheGen Sec. 5.2 "Arithmetic coding": one
// distribution per channel-layer for deltas and one for anchors; Sec. 6: frequencies counted
// over the context's quantized symbols).
//
// One workgroup of 16 waves per (layer, K/V, 64-channel block). The workgroup takes the
// (context, chunk) pairs of that block one after the other and splits each chunk's groups across
// its waves: every wave first reduces the absmax of its token slice, the slices are combined in
// LDS into the chunk's scale, then every wave quantizes its slice (groups are independent once
// the scale is known) and counts the symbols into LDS histograms. Rows are read 64 channels
// (128 B) at a time, so every load is one coalesced line.
//
// fit_kernel fits one level with 32-bit counts. When the channel count is a multiple of 64 and
// half of a wave's slice is at most kHalf tokens (the paper's 1.5K-token chunks: 48-50), a lane
// takes two neighbouring channels (one dword per token) over half of the wave's groups; the
// slice is read once, into registers, with all its loads in flight together, and both passes
// work from the registers. Otherwise the rows are read once per pass, a lane per channel.
// fit_pass_kernel (whole 64-channel blocks) and fit_levels_kernel (any channel count) fit the
// anchors and several levels from one quantization with 16-bit counts; fit_hold_kernel is
// fit_pass_kernel's one-level case at G = 10 with the slice held in registers between its
// maxima and its count (the cache read once) and resident workgroups that walk the blocks.
//
// Histograms use an odd row stride so lanes that count the same symbol hit different banks. At
// the end each wave normalises histograms to 16-bit cumulative tables: per-lane partial sums, a
// wave reduction for the total, the argmax and the frequency sum, and a wave prefix scan.
#include "cg_device.h"

namespace {

constexpr int kFitWaves = 16;
constexpr int kFitThreads = kFitWaves * 64;
constexpr int kHist = 257;  // 255 symbols, padded; odd stride spreads lanes over the banks
constexpr int kHalf = 56;   // longest half slice per lane held in registers (one dword per token)

// Normalise one histogram [255] into cum[256] (entry 255 = 0) with one wave. With shift >= 0
// the counts are the 16-bit fields at that bit position of 32-bit words. Frequencies are
// 1 + floor(c (2^16 - 255) / N) for the symbol counts c over their total N, the rest of 2^16
// going to the most frequent symbol (the lowest index on ties).
template <typename CountT>
__device__ void normalize_wave(const CountT* cnt, uint16_t* out, int shift = -1) {
  const int lane = threadIdx.x & 63;
  uint64_t c[4];
  uint64_t local = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    int i = lane * 4 + j;
    const uint64_t v = i < CG_NSYM ? (uint64_t)cnt[i] : 0u;
    c[j] = shift < 0 ? v : (v >> shift) & 0xFFFFu;
    local += c[j];
  }
  uint64_t N = cg_wave_sum<uint64_t>(local);
  if (N == 0) {
#pragma unroll
    for (int j = 0; j < 4; ++j) c[j] = (lane * 4 + j) < CG_NSYM ? 1u : 0u;
    N = CG_NSYM;
  }
  constexpr uint32_t kSpread = CG_TOTAL - CG_NSYM;
  uint32_t f[4];
  uint32_t fl = 0;
  int besti = 0x7fffffff;
  if (N <= 0xFFFFFFFFull) {   // wave-uniform: every count and the total fit 32 bits
    // argmax with the lowest index on ties
    uint32_t best = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int i = lane * 4 + j;
      if (i < CG_NSYM && (besti == 0x7fffffff || (uint32_t)c[j] > best)) {
        best = (uint32_t)c[j];
        besti = i;
      }
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
      const uint32_t ob = __shfl_xor(best, o, 64);
      const int oi = __shfl_xor(besti, o, 64);
      if (ob > best || (ob == best && oi < besti)) { best = ob; besti = oi; }
    }
    // floor(c kSpread / N) without a 64-bit division: a float estimate within 0.016 of the
    // quotient (four roundings of 2^-24 each), so its truncation is within one of the floor,
    // then one exact correction step with the 64-bit products
    const uint32_t Nu = (uint32_t)N;
    const float ratio = (float)kSpread / (float)Nu;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t cj = (uint32_t)c[j];
      uint32_t q = (uint32_t)((float)cj * ratio);
      const uint64_t num = (uint64_t)cj * kSpread;
      const uint64_t pq = (uint64_t)q * Nu;
      if (pq > num) q -= 1u;
      else if (num - pq >= Nu) q += 1u;
      f[j] = lane * 4 + j < CG_NSYM ? 1u + q : 0u;
      fl += f[j];
    }
  } else {
    uint64_t best = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int i = lane * 4 + j;
      if (i < CG_NSYM && (besti == 0x7fffffff || c[j] > best)) { best = c[j]; besti = i; }
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
      uint64_t ob = __shfl_xor(best, o, 64);
      int oi = __shfl_xor(besti, o, 64);
      if (ob > best || (ob == best && oi < besti)) { best = ob; besti = oi; }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      int i = lane * 4 + j;
      f[j] = i < CG_NSYM ? 1u + (uint32_t)((c[j] * kSpread) / N) : 0u;
      fl += f[j];
    }
  }
  uint32_t sumf = cg_wave_sum<uint32_t>(fl);
  uint32_t rem = CG_TOTAL - sumf;
#pragma unroll
  for (int j = 0; j < 4; ++j)
    if (lane * 4 + j == besti) { f[j] += rem; fl += rem; }
  uint32_t incl = cg_wave_incl_scan(fl);
  uint32_t run = incl - fl;  // exclusive prefix of this lane's first symbol
  uint16_t o[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    int i = lane * 4 + j;
    o[j] = i < CG_NSYM ? (uint16_t)run : (uint16_t)0;
    run += f[j];
  }
  // 4 consecutive u16 per lane: one 8-byte store, the wave writes the 512-byte table at once
  uint64_t packed = (uint64_t)o[0] | ((uint64_t)o[1] << 16) | ((uint64_t)o[2] << 32) |
                    ((uint64_t)o[3] << 48);
  reinterpret_cast<uint64_t*>(out)[lane] = packed;
}

// Inclusive prefix of v over the 64 lanes with DPP moves (no LDS): a Hillis-Steele scan inside
// each row of 16 lanes (row_shr 1, 2, 4, 8, zero from outside the row), then lane 15 of rows 0
// and 2 into rows 1 and 3 (row_bcast:15) and lane 31 into rows 2 and 3 (row_bcast:31). kMax
// takes the running maximum instead of the sum (values must be non-negative). Lane 63 ends with
// the whole wave's sum or maximum.
template <bool kMax>
__device__ __forceinline__ uint32_t dpp_incl_scan(uint32_t v) {
  auto op = [](uint32_t a, uint32_t b) { return kMax ? max(a, b) : a + b; };
  v = op(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xf, 0xf, true));
  v = op(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xf, 0xf, true));
  v = op(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xf, 0xf, true));
  v = op(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xf, 0xf, true));
  v = op(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xa, 0xf, false));
  v = op(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xc, 0xf, false));
  return v;
}

// normalize_wave for 16-bit counts (the 16-bit field at bit `shift` of each word) whose total
// is below 2^16, as the fit's 16-bit kernels guarantee: the same tables from 32-bit arithmetic.
// Every product c (2^16 - 255) and q N stays below 2^32 (c, N <= 65535; q <= 2^16 - 254), so the
// floor comes from the float estimate and one exact correction with 24-bit multiplies; the total,
// the argmax (key count << 8 | 255 - index: the largest count, then the lowest index) and the
// frequency prefix are DPP scans.
__device__ void normalize16_wave(const uint32_t* cnt, uint16_t* out, int shift) {
  const int lane = threadIdx.x & 63;
  uint32_t c[4];
  uint32_t local = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int i = lane * 4 + j;
    c[j] = i < CG_NSYM ? (cnt[i] >> shift) & 0xFFFFu : 0u;
    local += c[j];
  }
  uint32_t N = (uint32_t)__builtin_amdgcn_readlane((int)dpp_incl_scan<false>(local), 63);
  if (N == 0) {
#pragma unroll
    for (int j = 0; j < 4; ++j) c[j] = (lane * 4 + j) < CG_NSYM ? 1u : 0u;
    N = CG_NSYM;
  }
  constexpr uint32_t kSpread = CG_TOTAL - CG_NSYM;
  uint32_t key = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int i = lane * 4 + j;
    if (i < CG_NSYM) key = max(key, (c[j] << 8) | (uint32_t)(255 - i));
  }
  const uint32_t kmax = (uint32_t)__builtin_amdgcn_readlane((int)dpp_incl_scan<true>(key), 63);
  const int besti = 255 - (int)(kmax & 0xFFu);
  const float ratio = (float)kSpread / (float)N;
  uint32_t f[4];
  uint32_t fl = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    uint32_t q = (uint32_t)((float)c[j] * ratio);
    const uint32_t num = __umul24(c[j], kSpread);
    const uint32_t pq = __umul24(q, N);
    if (pq > num) q -= 1u;
    else if (num - pq >= N) q += 1u;
    f[j] = lane * 4 + j < CG_NSYM ? 1u + q : 0u;
    fl += f[j];
  }
  const uint32_t sumf = (uint32_t)__builtin_amdgcn_readlane((int)dpp_incl_scan<false>(fl), 63);
  const uint32_t rem = CG_TOTAL - sumf;
#pragma unroll
  for (int j = 0; j < 4; ++j)
    if (lane * 4 + j == besti) { f[j] += rem; fl += rem; }
  uint32_t run = dpp_incl_scan<false>(fl) - fl;
  uint16_t o[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    o[j] = lane * 4 + j < CG_NSYM ? (uint16_t)run : (uint16_t)0;
    run += f[j];
  }
  const uint64_t packed = (uint64_t)o[0] | ((uint64_t)o[1] << 16) | ((uint64_t)o[2] << 32) |
                          ((uint64_t)o[3] << 48);
  reinterpret_cast<uint64_t*>(out)[lane] = packed;
}

// x - a for the fp16 value in the low (kHi false) or high half of w: one v_fma_mix_f32 computing
// x * 1 - a with the widening fused in. x * 1 is exact and the sum is rounded once, so the result
// is bit for bit the f32 subtraction of the widened value.
template <bool kHi>
__device__ __forceinline__ float sub_half(uint32_t w, float a) {
  float d;
  if constexpr (kHi)
    asm("v_fma_mix_f32 %0, %1, 1.0, -%2 op_sel:[1,0,0] op_sel_hi:[1,0,0]"
        : "=v"(d) : "v"(w), "v"(a));
  else
    asm("v_fma_mix_f32 %0, %1, 1.0, -%2 op_sel_hi:[1,0,0]"
        : "=v"(d) : "v"(w), "v"(a));
  return d;
}

// kPool: instead of normalising per channel, add the workgroup's counts (summed over its 64
// channels) to the global counts pool[2][256] (anchor, delta): the one-distribution baseline.
// Count one quantized token of a slice: the anchor (group position g == 0) under the 8-bit
// step s, the others as the delta to the dequantized anchor under step w.
// is = 1 / s and iw = 1 / w (correctly rounded).
__device__ __forceinline__ void fit_count(float v, int g, float s, float w, float is, float iw,
                                          float& a, uint32_t* ha, uint32_t* hd) {
  if (g == 0) {
    const int q = cg_quant_inv(v, s, is);
    a = (float)q * s;
    atomicAdd(&ha[q + 127], 1u);
  } else {
    const int q = cg_quant_inv(v - a, w, iw);
    atomicAdd(&hd[q + 127], 1u);
  }
}

// The scale s of the stream (context b, chunk c, layer l, K/V k, channel ch), the value the
// encoder computes from the same maxima, into scales[S].
__device__ __forceinline__ void put_scale(float* scales, const KParams& P, int b, int c, int l,
                                          int k, int ch, float s) {
  scales[cg_stream(P, (((int64_t)b * P.NC + c) * P.L + l) * 2 + k, ch)] = s;
}

template <bool kPool, bool kRegs>
__global__ __launch_bounds__(kFitThreads) void fit_kernel(KParams P, const uint16_t* __restrict__ kv,
                                                         int level, uint16_t* __restrict__ cdf_anchor,
                                                         uint16_t* __restrict__ cdf_delta,
                                                         unsigned long long* __restrict__ pool,
                                                         uint32_t* __restrict__ status,
                                                         float* __restrict__ scales) {
  extern __shared__ uint32_t cnt[];  // [2 kinds][64 channels][kHist]
  // partial absolute maxima as magnitude bits (x & 0x7fff): for finite halves they order like
  // |x|, and NaN or Inf gives at least 0x7c00
  __shared__ uint32_t part[kFitWaves][64];
  __shared__ uint32_t s_bad;
  const int cb = blockIdx.x % P.nblk;
  const int lk = blockIdx.x / P.nblk;
  const int l = lk >> 1, k = lk & 1;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;

  for (int i = threadIdx.x; i < 2 * 64 * kHist; i += kFitThreads) cnt[i] = 0;
  if (threadIdx.x == 0) s_bad = 0u;
  __syncthreads();

  const int ch = cb * 64 + lane;
  const bool act = ch < P.C;
  const float wfac = P.layer_bin[l] * P.level_mult[level];
  uint32_t bad = 0u;
  uint32_t* ha = cnt + lane * kHist;
  uint32_t* hd = cnt + (64 + lane) * kHist;
  const int pairs = P.B * P.NC;
  const int64_t rs = P.C;
  for (int pr = 0; pr < pairs; ++pr) {
    const int b = pr / P.NC, c = pr % P.NC;
    const int t0 = c * P.CL;
    const int n = min(P.CL, P.T - t0);
    const int ng = (n + P.G - 1) / P.G;                 // groups in the chunk
    const int gpw = (ng + kFitWaves - 1) / kFitWaves;   // groups per wave
    const int j0 = min(n, wave * gpw * P.G), j1 = min(n, (wave + 1) * gpw * P.G);
    const uint16_t* x = kv + cg_elem(P, b, l, k, t0, act ? ch : cb * 64);
    if constexpr (kRegs) {
      // lane = (channel pair cp, token half th): channels cb*64 + 2 cp and + 1, read as one
      // dword per token (64-channel blocks are whole and dword aligned on this path), over the
      // th-th half of the wave's groups; each half (at most kHalf tokens, each half's own
      // length) goes into registers with every load in flight at once
      const int cp = lane & 31, th = lane >> 5;
      const int gh = (gpw + 1) >> 1;
      const int h0 = min(j1, j0 + th * gh * P.G), h1 = min(j1, j0 + (th + 1) * gh * P.G);
      const int len = h1 - h0;
      typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
      const half2_t* xw = reinterpret_cast<const half2_t*>(kv + cg_elem(P, b, l, k, t0, cb * 64)) + cp;
      const int64_t rw = P.C >> 1;
      half2_t pk[kHalf];
#pragma unroll
      for (int u = 0; u < kHalf; ++u) pk[u] = xw[(int64_t)min(h0 + u, n - 1) * rw];
      uint32_t b0 = 0u, b1 = 0u;
#pragma unroll
      for (int u = 0; u < kHalf; ++u) {
        if (u < len) {
          const uint32_t bits = __builtin_bit_cast(uint32_t, pk[u]);
          b0 = max(b0, bits & 0x7FFFu);
          b1 = max(b1, (bits >> 16) & 0x7FFFu);
        }
      }
      b0 = max(b0, (uint32_t)__shfl_xor((int)b0, 32, 64));
      b1 = max(b1, (uint32_t)__shfl_xor((int)b1, 32, 64));
      if (th == 0) {
        part[wave][2 * cp] = b0;
        part[wave][2 * cp + 1] = b1;
      }
      __syncthreads();
      b0 = 0u;
      b1 = 0u;
#pragma unroll
      for (int v = 0; v < kFitWaves; ++v) {
        b0 = max(b0, part[v][2 * cp]);
        b1 = max(b1, part[v][2 * cp + 1]);
      }
      bad |= (b0 >= 0x7C00u) | (b1 >= 0x7C00u);
      const float m0 = cg_h2f((uint16_t)b0), m1 = cg_h2f((uint16_t)b1);
      const float s0 = (m0 == 0.0f) ? 1.0f : m0 / 127.0f;
      const float s1 = (m1 == 0.0f) ? 1.0f : m1 / 127.0f;
      if (scales && wave == 0 && th == 0) {   // every wave holds the same maxima
        put_scale(scales, P, b, c, l, k, cb * 64 + 2 * cp, s0);
        put_scale(scales, P, b, c, l, k, cb * 64 + 2 * cp + 1, s1);
      }
      const float w0 = wfac * s0, w1 = wfac * s1;
      const float is0 = 1.0f / s0, is1 = 1.0f / s1, iw0 = 1.0f / w0, iw1 = 1.0f / w1;
      uint32_t* ha0 = cnt + (2 * cp) * kHist;
      uint32_t* hd0 = cnt + (64 + 2 * cp) * kHist;
      float a0 = 0.0f, a1 = 0.0f;
      int g = 0;
#pragma unroll
      for (int u = 0; u < kHalf; ++u) {
        if (u < len) {
          fit_count((float)pk[u].x, g, s0, w0, is0, iw0, a0, ha0, hd0);
          fit_count((float)pk[u].y, g, s1, w1, is1, iw1, a1, ha0 + kHist, hd0 + kHist);
        }
        g = (g + 1 == P.G) ? 0 : g + 1;
      }
    } else {
      // pass 1: absmax of this wave's slice, combined over the waves in LDS
      uint32_t mb = 0u;
#pragma unroll 8
      for (int j = j0; j < j1; ++j) mb = max(mb, (uint32_t)x[(int64_t)j * rs] & 0x7FFFu);
      part[wave][lane] = mb;
      __syncthreads();
      mb = 0u;
#pragma unroll
      for (int v = 0; v < kFitWaves; ++v) mb = max(mb, part[v][lane]);
      bad |= act && mb >= 0x7C00u;
      const float m = cg_h2f((uint16_t)mb);
      const float s = (m == 0.0f) ? 1.0f : m / 127.0f;
      if (scales && wave == 0 && act) put_scale(scales, P, b, c, l, k, ch, s);
      const float w = wfac * s;
      const float is = 1.0f / s, iw = 1.0f / w;
      // pass 2: quantize the slice (it starts on a group boundary) and count
      if (act) {
        float a = 0.0f;
        int g = 0;
#pragma unroll 4
        for (int j = j0; j < j1; ++j) {
          fit_count(cg_h2f(x[(int64_t)j * rs]), g, s, w, is, iw, a, ha, hd);
          g = (g + 1 == P.G) ? 0 : g + 1;
        }
      }
    }
    __syncthreads();   // `part` is reused by the next pair
  }
  if (status) {
    if (bad) s_bad = 1u;   // benign race: every writer stores 1
    __syncthreads();
    if (threadIdx.x == 0 && s_bad) atomicOr(status, 1u);
  }

  if constexpr (kPool) {
    for (int i = threadIdx.x; i < 2 * CG_NSYM; i += kFitThreads) {
      const int kind = i / CG_NSYM, sym = i - kind * CG_NSYM;
      unsigned long long sum = 0;
      for (int c2 = 0; c2 < 64; ++c2) sum += cnt[(kind * 64 + c2) * kHist + sym];
      if (sum) atomicAdd(&pool[kind * 256 + sym], sum);
    }
    return;
  }
  for (int tb = wave; tb < 128; tb += kFitWaves) {
    const int kind = tb >> 6, cl = tb & 63;
    const int chx = cb * 64 + cl;
    if (chx >= P.C) continue;
    if (kind == 0 && cdf_anchor == nullptr) continue;
    uint16_t* dst = (kind == 0 ? cdf_anchor : cdf_delta) +
                    ((int64_t)(l * 2 + k) * P.C + chx) * 256;
    normalize_wave<uint32_t>(cnt + tb * kHist, dst);
  }
}

__global__ __launch_bounds__(256) void pool_zero(unsigned long long* pool) {
  for (int i = threadIdx.x; i < 2 * 256; i += 256) pool[i] = 0ull;
}

// the two pooled tables (wave 0: anchor, wave 1: delta) into tab[2][256]
__global__ __launch_bounds__(128) void pool_normalize(const unsigned long long* pool,
                                                      uint16_t* tab) {
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  normalize_wave<unsigned long long>(pool + wave * 256, tab + wave * 256);
}

// copy the pooled tables into every (layer, K/V, channel) slot: one wave per slot and kind
__global__ __launch_bounds__(256) void pool_broadcast(const uint16_t* __restrict__ tab,
                                                      int64_t n_tables,
                                                      uint16_t* __restrict__ cdf_anchor,
                                                      uint16_t* __restrict__ cdf_delta) {
  const int64_t w = (int64_t)blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (w >= 2 * n_tables) return;
  const int kind = (int)(w / n_tables);
  const int64_t t = w - kind * n_tables;
  uint16_t* dst = kind == 0 ? cdf_anchor : cdf_delta;
  if (!dst) return;
  const uint64_t v = reinterpret_cast<const uint64_t*>(tab + kind * 256)[lane];
  reinterpret_cast<uint64_t*>(dst + t * 256)[lane] = v;
}


// ---- several levels in one pass ---------------------------------------------------------------
// Both kernels fit the anchors (with_anchor) and kNl consecutive levels lv0 .. from one
// quantization of each slice: the chunk's scale, the anchors and the deltas to them are found
// once for all those levels. Counts are 16-bit: the two neighbouring channels 2 cp and 2 cp + 1
// sit in the low and high half of one 32-bit LDS word, so a kind takes the LDS of half a 32-bit
// histogram; the host uses these kernels only when no count can reach 2^16. A slice whose
// absolute maximum has the exponent bits all ones (NaN or Inf) sets *status.
constexpr int kLevelKinds = 4;   // fit_levels_kernel: anchor + levels, or levels, per workgroup
constexpr int kPassKinds = 5;    // fit_pass_kernel: anchor + four levels, 255-word rows
constexpr int kHistP = 255;      // 255 symbols, no padding (odd, so rows fall on other banks)
constexpr int kHoldGroups = 5;   // fit_hold_kernel: groups of a slice held (1536-token chunks: 5)
constexpr int kBufWord3 = 0x00020000;   // raw buffer descriptor: 32-bit data format

// fit_pass_kernel: whole 64-channel blocks. A lane takes a channel pair cp (one dword per
// token) over one of 32 slices of each chunk's groups (slice = 2 wave + lane / 32). The slice is
// read twice: first for the magnitude maximum (combined over the slices in LDS into the chunk's
// scale), then group by group from the last one back, so that the rows read last, the likeliest
// to be still in the L2, are read again first. The rows come through a buffer descriptor of the
// (context, layer, K/V) slab: a row outside the slab reads as zero and such tokens are never
// counted. kG = 10: the group's loads are issued together and the group is unrolled; kG = 0 takes
// the group size from P. With several levels the next group's rows and the next pair's maxima
// are loaded while a group is counted; with one level two workgroups share a CU instead.
template <int kNl, int kG>
__global__ __launch_bounds__(kFitThreads, kNl == 1 ? 8 : 4) void fit_pass_kernel(
    KParams P, const uint16_t* __restrict__ kv, int lv0, int with_anchor,
    uint16_t* __restrict__ cdf_anchor, uint16_t* __restrict__ cdf_delta,
    uint32_t* __restrict__ status, float* __restrict__ scales) {
  extern __shared__ uint32_t cnt[];   // [kinds][32 channel pairs][kHistP]
  // chunk maxima: (pair index + 1) << 16 | magnitude bits, per channel, alternating buffers (a
  // wave can only reach pair pr + 2 once every wave has read pair pr's buffer)
  __shared__ uint32_t s_max[2][64];
  __shared__ uint32_t s_bad;
  const int cb = blockIdx.x % P.nblk;
  const int lk = blockIdx.x / P.nblk;
  const int l = lk >> 1, k = lk & 1;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int cp = lane & 31;
  const int slice = wave * 2 + (lane >> 5);
  const int nk = with_anchor + kNl;
  for (int i = threadIdx.x; i < nk * 32 * kHistP; i += kFitThreads) cnt[i] = 0;
  if (threadIdx.x < 128) s_max[threadIdx.x >> 6][threadIdx.x & 63] = 0u;
  if (threadIdx.x == 0) s_bad = 0u;
  __syncthreads();

  const int G = kG > 0 ? kG : P.G;
  float wfac[kNl];
#pragma unroll
  for (int v = 0; v < kNl; ++v) wfac[v] = P.layer_bin[l] * P.level_mult[lv0 + v];
  // bin of symbol q in this lane's row of a kind: row[q], q in [-127, 127]
  uint32_t* const ha = cnt + cp * kHistP + 127;
  uint32_t* hrow[kNl];
#pragma unroll
  for (int v = 0; v < kNl; ++v) hrow[v] = cnt + ((with_anchor + v) * 32 + cp) * kHistP + 127;
  const int rowb = P.C * 2;                          // bytes per token row (host: slab < 2^31)
  const int slab_bytes = P.T * rowb;
  const int pairs = P.B * P.NC;
  uint32_t bad = 0u;
  typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
  // this lane's slice of pair pr: buffer of the slab, byte offset of its first token, its
  // length in tokens and the groups per slice
  struct Slice {
    __amdgpu_buffer_rsrc_t rs;
    int voff, len, gps;
  };
  auto slice_of = [&](int pr) __attribute__((always_inline)) {
    Slice q;
    const int b = pr / P.NC, c = pr % P.NC;
    const int t0 = c * P.CL;
    const int n = min(P.CL, P.T - t0);
    q.gps = ((n + G - 1) / G + 31) >> 5;
    const int s0 = min(n, slice * q.gps * G);
    q.len = min(n, (slice + 1) * q.gps * G) - s0;
    q.rs = __builtin_amdgcn_make_buffer_rsrc((void*)(kv + cg_elem(P, b, l, k, 0, 0)), (short)0,
                                             slab_bytes, kBufWord3);
    q.voff = (t0 + s0) * rowb + (cb * 64 + 2 * cp) * 2;
    return q;
  };
  auto load = [&](const Slice& q, int u) __attribute__((always_inline)) {
    return __builtin_amdgcn_raw_buffer_load_b32(q.rs, q.voff + u * rowb, 0, 0);
  };
  // magnitude bits of both channels of token u of slice q into the running maxima m
  const u16x2 mag = {0x7FFF, 0x7FFF};
  auto max_in = [&](u16x2& m, uint32_t x, int u, int len) __attribute__((always_inline)) {
    const u16x2 xm = __builtin_bit_cast(u16x2, x) & mag;
    m = u < len ? __builtin_elementwise_max(m, xm) : m;
  };
  // One level: the maxima of pair pr from 16-byte pieces of the chunk's rows. Lane (r = lane >> 3,
  // o = lane & 7) takes channels 8o .. 8o + 7 of the block in rows 8 wave + r + 128 i, four loads
  // in flight together; mw[j] holds channels 8o + 2j and 8o + 2j + 1. Past the chunk's last round
  // the last round is read again (the maxima do not change).
  constexpr bool kWide = kNl == 1 && kG > 0;
  typedef unsigned int u32x4 __attribute__((vector_size(16)));
  u16x2 mw[4];
  auto max_wide = [&](int pr) __attribute__((always_inline)) {
    const int b = pr / P.NC, c = pr % P.NC;
    const int t0 = c * P.CL;
    const int n = min(P.CL, P.T - t0);
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(kv + cg_elem(P, b, l, k, 0, 0)), (short)0, slab_bytes, kBufWord3);
    const int r0 = wave * 8 + (lane >> 3);
    const int voff = (t0 + r0) * rowb + cb * 128 + (lane & 7) * 16;
    const int last = (n - 1) >> 7;   // last round holding a row of the chunk
#pragma unroll
    for (int j = 0; j < 4; ++j) mw[j] = u16x2{0, 0};
    for (int i = 0; i <= last; i += 4) {
      u32x4 v[4];
#pragma unroll
      for (int e = 0; e < 4; ++e)
        v[e] = __builtin_amdgcn_raw_buffer_load_b128(rs, voff + min(i + e, last) * 128 * rowb, 0, 0);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const bool in = r0 + min(i + e, last) * 128 < n;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          // the element is copied out first: a bit cast of the vector element itself read
          // element 0 for every j
          const uint32_t w = v[e][j];
          mw[j] = in ? __builtin_elementwise_max(mw[j], __builtin_bit_cast(u16x2, w) & mag) : mw[j];
        }
      }
    }
  };
  // pass 1 of the first pair; that of every further pair runs inside or after the previous
  // pair's pass 2
  Slice cur = slice_of(0);
  u16x2 m = {0, 0};
  if constexpr (kWide) {
    max_wide(0);
  } else {
#pragma unroll 8
    for (int u = 0; u < cur.gps * G; ++u) max_in(m, load(cur, u), u, cur.len);
  }
  for (int pr = 0; pr < pairs; ++pr) {
    uint32_t* const sm = s_max[pr & 1];
    const uint32_t tag = (uint32_t)(pr + 1) << 16;
    if constexpr (kWide) {
      // the wave's eight rows of each octet combined, then the first row's lanes publish
#pragma unroll
      for (int o = 8; o < 64; o <<= 1) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
          mw[j] = __builtin_elementwise_max(
              mw[j], __builtin_bit_cast(u16x2, __shfl_xor(__builtin_bit_cast(uint32_t, mw[j]), o, 64)));
      }
      if (lane < 8) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          atomicMax(&sm[8 * lane + 2 * j], tag | mw[j].x);
          atomicMax(&sm[8 * lane + 2 * j + 1], tag | mw[j].y);
        }
      }
    } else {
      atomicMax(&sm[2 * cp], tag | m.x);
      atomicMax(&sm[2 * cp + 1], tag | m.y);
    }
    __syncthreads();
    const uint32_t b0 = sm[2 * cp] & 0xFFFFu, b1 = sm[2 * cp + 1] & 0xFFFFu;
    bad |= (b0 >= 0x7C00u) | (b1 >= 0x7C00u);
    const float m0 = cg_h2f((uint16_t)b0), m1 = cg_h2f((uint16_t)b1);
    const float sc0 = (m0 == 0.0f) ? 1.0f : m0 / 127.0f;
    const float sc1 = (m1 == 0.0f) ? 1.0f : m1 / 127.0f;
    if (scales && with_anchor && wave == 0 && lane < 32) {   // every wave holds the maxima
      put_scale(scales, P, pr / P.NC, pr % P.NC, l, k, cb * 64 + 2 * cp, sc0);
      put_scale(scales, P, pr / P.NC, pr % P.NC, l, k, cb * 64 + 2 * cp + 1, sc1);
    }
    const float is0 = 1.0f / sc0, is1 = 1.0f / sc1;
    float w0[kNl], w1[kNl], iw0[kNl], iw1[kNl];
#pragma unroll
    for (int v = 0; v < kNl; ++v) {
      w0[v] = wfac[v] * sc0;
      w1[v] = wfac[v] * sc1;
      iw0[v] = 1.0f / w0[v];
      iw1[v] = 1.0f / w1[v];
    }
    // one token of both channels: the anchor (u == 0) or the deltas to the group's anchors
    float a0 = 0.0f, a1 = 0.0f;
    auto token = [&](uint32_t x, bool anchor) __attribute__((always_inline)) {
      if (anchor) {
        const u16x2 h = __builtin_bit_cast(u16x2, x);
        const float x0 = cg_h2f(h.x), x1 = cg_h2f(h.y);
        const int q0 = cg_quant_inv(x0, sc0, is0), q1 = cg_quant_inv(x1, sc1, is1);
        a0 = (float)q0 * sc0;
        a1 = (float)q1 * sc1;
        if (with_anchor) {
          atomicAdd(&ha[q0], 1u);
          atomicAdd(&ha[q1], 0x10000u);
        }
      } else {
        const float d0 = sub_half<false>(x, a0), d1 = sub_half<true>(x, a1);
#pragma unroll
        for (int v = 0; v < kNl; ++v) {
          atomicAdd(&hrow[v][cg_quant_inv(d0, w0[v], iw0[v])], 1u);
          atomicAdd(&hrow[v][cg_quant_inv(d1, w1[v], iw1[v])], 0x10000u);
        }
      }
    };
    // pass 2: the slice's groups, last first, and pass 1 of the next pair alongside
    const bool more = pr + 1 < pairs;
    const Slice nxt = more ? slice_of(pr + 1) : cur;
    const int span_n = more ? nxt.gps * G : 0;
    u16x2 mn = {0, 0};
    int covered = 0;   // tokens of the next slice already in mn
    if constexpr (kG > 0 && kNl == 1) {
      // one level (the anchors and one delta kind: 65 KB of counts): no prefetch and no
      // interleaved maxima, so that a lane stays within 64 registers and two workgroups share a
      // CU, whose waves hide each other's load latency instead (measured faster)
      for (int gi = cur.gps - 1; gi >= 0; --gi) {
        const int base = gi * kG;
        uint32_t xc[kG];
#pragma unroll
        for (int u = 0; u < kG; ++u) xc[u] = load(cur, base + u);
        if (__builtin_amdgcn_ballot_w64(base + kG > cur.len) == 0) {
#pragma unroll
          for (int u = 0; u < kG; ++u) token(xc[u], u == 0);
        } else if (base < cur.len) {
#pragma unroll
          for (int u = 0; u < kG; ++u)
            if (base + u < cur.len) token(xc[u], u == 0);
        }
      }
    } else if constexpr (kG > 0) {
      uint32_t xc[kG], xn[kG], y[kG];
#pragma unroll
      for (int u = 0; u < kG; ++u) xc[u] = load(cur, (cur.gps - 1) * kG + u);
      for (int gi = cur.gps - 1; gi >= 0; --gi) {
        const int base = gi * kG;
        if (base < span_n) {
#pragma unroll
          for (int u = 0; u < kG; ++u) y[u] = load(nxt, base + u);
        }
        if (gi > 0) {
#pragma unroll
          for (int u = 0; u < kG; ++u) xn[u] = load(cur, base - kG + u);
        }
        if (__builtin_amdgcn_ballot_w64(base + kG > cur.len) == 0) {
          // every lane of the wave has the whole group
#pragma unroll
          for (int u = 0; u < kG; ++u) token(xc[u], u == 0);
        } else if (base < cur.len) {
#pragma unroll
          for (int u = 0; u < kG; ++u)
            if (base + u < cur.len) token(xc[u], u == 0);
        }
        if (base < span_n) {
#pragma unroll
          for (int u = 0; u < kG; ++u) max_in(mn, y[u], base + u, nxt.len);
        }
#pragma unroll
        for (int u = 0; u < kG; ++u) xc[u] = xn[u];
      }
      covered = min(cur.gps * kG, span_n);
    } else {
      for (int gi = cur.gps - 1; gi >= 0; --gi) {
        const int base = gi * G;
        if (base >= cur.len) continue;
        const int e = min(G, cur.len - base);
        for (int u = 0; u < e; ++u) token(load(cur, base + u), u == 0);
      }
    }
    if constexpr (kWide) {
      if (more) max_wide(pr + 1);
    } else {
#pragma unroll 8
      for (int u = covered; u < span_n; ++u) max_in(mn, load(nxt, u), u, nxt.len);
      m = mn;
    }
    cur = nxt;
  }
  if (bad) s_bad = 1u;   // benign race: every writer stores 1
  __syncthreads();
  if (threadIdx.x == 0 && s_bad && status) atomicOr(status, 1u);

  for (int tb = wave; tb < nk * 64; tb += kFitWaves) {
    const int kind = tb >> 6, cl = tb & 63;
    const int chx = cb * 64 + cl;
    uint16_t* dst = (with_anchor && kind == 0)
                        ? cdf_anchor + ((int64_t)lk * P.C + chx) * 256
                        : cdf_delta + (((int64_t)(lv0 + kind - with_anchor) * P.L * 2 + lk) * P.C +
                                       chx) * 256;
    normalize16_wave(cnt + (kind * 32 + (cl >> 1)) * kHistP, dst, 16 * (cl & 1));
  }
}

// fit_hold_kernel: one level, G = 10, whole 64-channel blocks, at most kH groups per slice (the
// paper's 1536-token chunks: 5). The lanes and slices of fit_pass_kernel, but a slice stays in
// registers from its maxima to its count, so the cache is read once: as each group is counted,
// its registers take the same rows of the next slice, whose maxima are taken one group later.
// The workgroups stay resident (one per CU) and take the (64-channel block, layer, K/V) items
// in turn, so the next item's first slice loads while the finished item's tables are
// normalised. Slice maxima meet in LDS under a tag that counts the workgroup's steps.
template <int kH>
__global__ __launch_bounds__(kFitThreads, 4) void fit_hold_kernel(
    KParams P, const uint16_t* __restrict__ kv, int lv0, int with_anchor,
    uint16_t* __restrict__ cdf_anchor, uint16_t* __restrict__ cdf_delta,
    uint32_t* __restrict__ status, float* __restrict__ scales) {
  constexpr int kG = 10, kHR = kH * kG;
  extern __shared__ uint32_t cnt[];   // [kinds][32 channel pairs][kHistP]
  __shared__ uint32_t s_max[2][64];   // (step + 1) << 16 | magnitude bits, alternating buffers
  __shared__ uint32_t s_bad;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int cp = lane & 31;
  const int slice = wave * 2 + (lane >> 5);
  const int nk = with_anchor + 1;
  const int n_items = P.L * 2 * P.nblk;
  if ((int)blockIdx.x >= n_items) return;   // uniform; the host launches at most n_items
  for (int i = threadIdx.x; i < nk * 32 * kHistP; i += kFitThreads) cnt[i] = 0;
  if (threadIdx.x < 128) s_max[threadIdx.x >> 6][threadIdx.x & 63] = 0u;
  if (threadIdx.x == 0) s_bad = 0u;
  __syncthreads();
  uint32_t* const ha = cnt + cp * kHistP + 127;
  uint32_t* const hd = cnt + (with_anchor * 32 + cp) * kHistP + 127;
  const int rowb = P.C * 2;
  const int slab_bytes = P.T * rowb;
  const int pairs = P.B * P.NC;
  uint32_t bad = 0u;
  typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
  struct Slice {
    __amdgpu_buffer_rsrc_t rs;
    int voff, len;
  };
  // this lane's slice of pair pr of item it (block it % nblk of layer-K/V it / nblk)
  auto slice_of = [&](int it, int pr) __attribute__((always_inline)) {
    Slice q;
    const int cb = it % P.nblk, lk = it / P.nblk;
    const int b = pr / P.NC, c = pr % P.NC;
    const int t0 = c * P.CL;
    const int n = min(P.CL, P.T - t0);
    const int gps = ((n + kG - 1) / kG + 31) >> 5;
    const int s0 = min(n, slice * gps * kG);
    q.len = min(n, (slice + 1) * gps * kG) - s0;
    q.rs = __builtin_amdgcn_make_buffer_rsrc((void*)(kv + cg_elem(P, b, lk >> 1, lk & 1, 0, 0)),
                                             (short)0, slab_bytes, kBufWord3);
    q.voff = (t0 + s0) * rowb + (cb * 64 + 2 * cp) * 2;
    return q;
  };
  auto load = [&](const Slice& q, int u) __attribute__((always_inline)) {
    return __builtin_amdgcn_raw_buffer_load_b32(q.rs, q.voff + u * rowb, 0, 0);
  };
  const u16x2 mag = {0x7FFF, 0x7FFF};
  auto max_in = [&](u16x2& mm, uint32_t x, int u, int len) __attribute__((always_inline)) {
    const u16x2 xm = __builtin_bit_cast(u16x2, x) & mag;
    mm = u < len ? __builtin_elementwise_max(mm, xm) : mm;
  };
  int it = blockIdx.x, pr = 0;
  Slice cur = slice_of(it, 0);
  uint32_t xs[kHR];   // rows past the slice are loaded too (another slice's, or zero) and skipped
#pragma unroll
  for (int u = 0; u < kHR; ++u) xs[u] = load(cur, u);
  u16x2 m = {0, 0};
#pragma unroll
  for (int u = 0; u < kHR; ++u) max_in(m, xs[u], u, cur.len);
  for (int step = 0;; ++step) {
    const int cb = it % P.nblk, lk = it / P.nblk;
    const int l = lk >> 1, k = lk & 1;
    int nit = it, npr = pr + 1;
    if (npr == pairs) {
      npr = 0;
      nit = it + (int)gridDim.x;
    }
    const bool more = nit < n_items;
    const Slice nxt = more ? slice_of(nit, npr) : cur;
    uint32_t* const sm = s_max[step & 1];
    const uint32_t tag = (uint32_t)(step + 1) << 16;
    atomicMax(&sm[2 * cp], tag | m.x);
    atomicMax(&sm[2 * cp + 1], tag | m.y);
    __syncthreads();
    const uint32_t b0 = sm[2 * cp] & 0xFFFFu, b1 = sm[2 * cp + 1] & 0xFFFFu;
    bad |= (b0 >= 0x7C00u) | (b1 >= 0x7C00u);
    const float m0 = cg_h2f((uint16_t)b0), m1 = cg_h2f((uint16_t)b1);
    const float sc0 = (m0 == 0.0f) ? 1.0f : m0 / 127.0f;
    const float sc1 = (m1 == 0.0f) ? 1.0f : m1 / 127.0f;
    if (scales && with_anchor && wave == 0 && lane < 32) {
      put_scale(scales, P, pr / P.NC, pr % P.NC, l, k, cb * 64 + 2 * cp, sc0);
      put_scale(scales, P, pr / P.NC, pr % P.NC, l, k, cb * 64 + 2 * cp + 1, sc1);
    }
    const float is0 = 1.0f / sc0, is1 = 1.0f / sc1;
    const float wf = P.layer_bin[l] * P.level_mult[lv0];
    const float w0 = wf * sc0, w1 = wf * sc1;
    const float iw0 = 1.0f / w0, iw1 = 1.0f / w1;
    float a0 = 0.0f, a1 = 0.0f;
    auto token = [&](uint32_t x, bool anchor) __attribute__((always_inline)) {
      if (anchor) {
        const u16x2 h = __builtin_bit_cast(u16x2, x);
        const int q0 = cg_quant_inv(cg_h2f(h.x), sc0, is0), q1 = cg_quant_inv(cg_h2f(h.y), sc1, is1);
        a0 = (float)q0 * sc0;
        a1 = (float)q1 * sc1;
        if (with_anchor) {
          atomicAdd(&ha[q0], 1u);
          atomicAdd(&ha[q1], 0x10000u);
        }
      } else {
        const float d0 = sub_half<false>(x, a0), d1 = sub_half<true>(x, a1);
        atomicAdd(&hd[cg_quant_inv(d0, w0, iw0)], 1u);
        atomicAdd(&hd[cg_quant_inv(d1, w1, iw1)], 0x10000u);
      }
    };
    u16x2 mn = {0, 0};
#pragma unroll
    for (int g = 0; g < kH; ++g) {
      const int base = g * kG;
      if (__builtin_amdgcn_ballot_w64(base + kG > cur.len) == 0) {
#pragma unroll
        for (int u = 0; u < kG; ++u) token(xs[base + u], u == 0);
      } else if (base < cur.len) {
#pragma unroll
        for (int u = 0; u < kG; ++u)
          if (base + u < cur.len) token(xs[base + u], u == 0);
      }
      if (more) {
#pragma unroll
        for (int u = 0; u < kG; ++u) xs[base + u] = load(nxt, base + u);
        if (g > 0) {
#pragma unroll
          for (int u = base - kG; u < base; ++u) max_in(mn, xs[u], u, nxt.len);
        }
      }
    }
    if (more) {
#pragma unroll
      for (int u = kHR - kG; u < kHR; ++u) max_in(mn, xs[u], u, nxt.len);
    }
    m = mn;
    if (npr == 0 || !more) {   // the item's last pair is counted: its tables
      __syncthreads();
      for (int tb = wave; tb < nk * 64; tb += kFitWaves) {
        const int kind = tb >> 6, cl = tb & 63;
        const int chx = cb * 64 + cl;
        uint16_t* dst = (with_anchor && kind == 0)
                            ? cdf_anchor + ((int64_t)lk * P.C + chx) * 256
                            : cdf_delta + (((int64_t)(lv0 + kind - with_anchor) * P.L * 2 + lk) *
                                               P.C + chx) * 256;
        normalize16_wave(cnt + (kind * 32 + (cl >> 1)) * kHistP, dst, 16 * (cl & 1));
      }
      if (!more) break;
      __syncthreads();
      // the next step's barrier orders these stores before any count of the next item
      for (int i = threadIdx.x; i < nk * 32 * kHistP; i += kFitThreads) cnt[i] = 0;
    }
    it = nit;
    pr = npr;
    cur = nxt;
  }
  if (bad) s_bad = 1u;   // benign race: every writer stores 1
  __syncthreads();
  if (threadIdx.x == 0 && s_bad && status) atomicOr(status, 1u);
}

// fit_levels_kernel: any channel count, a lane per channel (channel lane of the block is half
// lane & 1 of pair lane / 2 of the counts); each pass reads the slice from memory.
template <int kNl>
__global__ __launch_bounds__(kFitThreads) void fit_levels_kernel(
    KParams P, const uint16_t* __restrict__ kv, int lv0, int with_anchor,
    uint16_t* __restrict__ cdf_anchor, uint16_t* __restrict__ cdf_delta,
    uint32_t* __restrict__ status, float* __restrict__ scales) {
  extern __shared__ uint32_t cnt[];   // [kinds][32 channel pairs][kHist]
  __shared__ uint32_t part[kFitWaves][64];
  __shared__ uint32_t s_bad;
  const int cb = blockIdx.x % P.nblk;
  const int lk = blockIdx.x / P.nblk;
  const int l = lk >> 1, k = lk & 1;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int nk = with_anchor + kNl;
  for (int i = threadIdx.x; i < nk * 32 * kHist; i += kFitThreads) cnt[i] = 0;
  if (threadIdx.x == 0) s_bad = 0u;
  __syncthreads();

  float wfac[kNl];
#pragma unroll
  for (int v = 0; v < kNl; ++v) wfac[v] = P.layer_bin[l] * P.level_mult[lv0 + v];
  uint32_t* const hist_d = cnt + with_anchor * 32 * kHist;   // kind v: hist_d + v * 32 * kHist
  const int pairs = P.B * P.NC;
  const int64_t rs = P.C;
  uint32_t bad = 0u;
  const int ch = cb * 64 + lane;
  const bool act = ch < P.C;
  const int h = lane >> 1;
  const uint32_t inc = (lane & 1) ? 0x10000u : 1u;
  for (int pr = 0; pr < pairs; ++pr) {
    const int b = pr / P.NC, c = pr % P.NC;
    const int t0 = c * P.CL;
    const int n = min(P.CL, P.T - t0);
    const int ng = (n + P.G - 1) / P.G;                 // groups in the chunk
    const int gpw = (ng + kFitWaves - 1) / kFitWaves;   // groups per wave
    const int j0 = min(n, wave * gpw * P.G), j1 = min(n, (wave + 1) * gpw * P.G);
    const uint16_t* x = kv + cg_elem(P, b, l, k, t0, act ? ch : cb * 64);
    uint32_t m = 0u;
#pragma unroll 8
    for (int j = j0; j < j1; ++j) m = max(m, (uint32_t)x[(int64_t)j * rs] & 0x7FFFu);
    part[wave][lane] = m;
    __syncthreads();
    m = 0u;
#pragma unroll
    for (int v = 0; v < kFitWaves; ++v) m = max(m, part[v][lane]);
    bad |= act && m >= 0x7C00u;
    const float mx = cg_h2f((uint16_t)m);
    const float s = (mx == 0.0f) ? 1.0f : mx / 127.0f;
    if (scales && with_anchor && wave == 0 && act) put_scale(scales, P, b, c, l, k, ch, s);
    const float is = 1.0f / s;
    float w[kNl], iw[kNl];
#pragma unroll
    for (int v = 0; v < kNl; ++v) {
      w[v] = wfac[v] * s;
      iw[v] = 1.0f / w[v];
    }
    if (act) {
      float a = 0.0f;
      int g = 0;
#pragma unroll 4
      for (int j = j0; j < j1; ++j) {
        const float xv = cg_h2f(x[(int64_t)j * rs]);
        if (g == 0) {
          const int q = cg_quant_inv(xv, s, is);
          a = (float)q * s;
          if (with_anchor) atomicAdd(&cnt[h * kHist + q + 127], inc);
        } else {
          const float d = xv - a;
#pragma unroll
          for (int v = 0; v < kNl; ++v) {
            const int q = cg_quant_inv(d, w[v], iw[v]);
            atomicAdd(&hist_d[(v * 32 + h) * kHist + q + 127], inc);
          }
        }
        g = (g + 1 == P.G) ? 0 : g + 1;
      }
    }
    __syncthreads();   // `part` is reused by the next pair
  }
  if (bad) s_bad = 1u;   // benign race: every writer stores 1
  __syncthreads();
  if (threadIdx.x == 0 && s_bad && status) atomicOr(status, 1u);

  for (int tb = wave; tb < nk * 64; tb += kFitWaves) {
    const int kind = tb >> 6, cl = tb & 63;
    const int chx = cb * 64 + cl;
    if (chx >= P.C) continue;
    uint16_t* dst = (with_anchor && kind == 0)
                        ? cdf_anchor + ((int64_t)lk * P.C + chx) * 256
                        : cdf_delta + (((int64_t)(lv0 + kind - with_anchor) * P.L * 2 + lk) * P.C +
                                       chx) * 256;
    normalize16_wave(cnt + (kind * 32 + (cl >> 1)) * kHist, dst, 16 * (cl & 1));
  }
}

__global__ __launch_bounds__(64) void zero_word(uint32_t* w) {
  if (threadIdx.x == 0) *w = 0u;
}

}  // namespace

namespace {
// Whether the register path applies: whole 64-channel blocks, and half of every wave's slice
// within kHalf tokens (the longest chunk has ceil(n / G) groups, a wave takes ceil(groups / 16)
// of them, a lane half of those).
bool fit_slice_in_registers(const KParams& P) {
  const int64_t n = P.CL < P.T ? P.CL : P.T;
  const int64_t ng = (n + P.G - 1) / P.G;
  const int64_t gpw = (ng + kFitWaves - 1) / kFitWaves;
  return P.C % 64 == 0 && ((gpw + 1) / 2) * P.G <= kHalf;
}

template <bool kPool, bool kRegs>
hipError_t launch_fit_kernel(const KParams& P, const uint16_t* kv, int level,
                             uint16_t* cdf_anchor, uint16_t* cdf_delta_level,
                             unsigned long long* pool, hipStream_t st,
                             uint32_t* status = nullptr, float* scales = nullptr) {
  const size_t lds = 2 * 64 * kHist * sizeof(uint32_t);
  hipError_t e = hipFuncSetAttribute((const void*)fit_kernel<kPool, kRegs>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  const int64_t grid = (int64_t)P.L * 2 * P.nblk;
  hipLaunchKernelGGL((fit_kernel<kPool, kRegs>), dim3((unsigned)grid), dim3(kFitThreads), lds,
                     st, P, kv, level, cdf_anchor, cdf_delta_level, pool, status, scales);
  return hipGetLastError();
}
}  // namespace

hipError_t cg_launch_fit(const KParams& P, const uint16_t* kv, int level, uint16_t* cdf_anchor,
                         uint16_t* cdf_delta_level, hipStream_t st, float* scales) {
  return fit_slice_in_registers(P)
             ? launch_fit_kernel<false, true>(P, kv, level, cdf_anchor, cdf_delta_level,
                                              nullptr, st, nullptr, scales)
             : launch_fit_kernel<false, false>(P, kv, level, cdf_anchor, cdf_delta_level,
                                               nullptr, st, nullptr, scales);
}

hipError_t cg_launch_fit_global(const KParams& P, const uint16_t* kv, int level,
                                uint16_t* cdf_anchor, uint16_t* cdf_delta_level, void* ws,
                                hipStream_t st) {
  unsigned long long* pool = static_cast<unsigned long long*>(ws);           // [2][256]
  uint16_t* tab = reinterpret_cast<uint16_t*>(static_cast<uint8_t*>(ws) + 4096);  // [2][256]
  hipLaunchKernelGGL(pool_zero, dim3(1), dim3(256), 0, st, pool);
  hipError_t e = fit_slice_in_registers(P)
                     ? launch_fit_kernel<true, true>(P, kv, level, cdf_anchor, cdf_delta_level,
                                                     pool, st)
                     : launch_fit_kernel<true, false>(P, kv, level, cdf_anchor,
                                                      cdf_delta_level, pool, st);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(pool_normalize, dim3(1), dim3(128), 0, st, pool, tab);
  const int64_t n_tables = (int64_t)P.L * 2 * P.C;
  const int64_t blocks = (2 * n_tables + 3) / 4;
  hipLaunchKernelGGL(pool_broadcast, dim3((unsigned)blocks), dim3(256), 0, st, tab, n_tables,
                     cdf_anchor, cdf_delta_level);
  return hipGetLastError();
}

namespace {
hipError_t launch_fit_levels(const KParams& P, const uint16_t* kv, int lv0, int nl,
                             int with_anchor, uint16_t* cdf_anchor, uint16_t* cdf_delta,
                             uint32_t* status, float* scales, hipStream_t st) {
  const size_t lds = (size_t)(with_anchor + nl) * 32 * kHist * sizeof(uint32_t);
  const void* fn = nl == 1 ? (const void*)fit_levels_kernel<1>
                 : nl == 2 ? (const void*)fit_levels_kernel<2>
                 : nl == 3 ? (const void*)fit_levels_kernel<3>
                           : (const void*)fit_levels_kernel<4>;
  hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  const dim3 grid((unsigned)((int64_t)P.L * 2 * P.nblk)), block(kFitThreads);
  switch (nl) {
    case 1: hipLaunchKernelGGL((fit_levels_kernel<1>), grid, block, lds, st, P, kv, lv0, with_anchor, cdf_anchor, cdf_delta, status, scales); break;
    case 2: hipLaunchKernelGGL((fit_levels_kernel<2>), grid, block, lds, st, P, kv, lv0, with_anchor, cdf_anchor, cdf_delta, status, scales); break;
    case 3: hipLaunchKernelGGL((fit_levels_kernel<3>), grid, block, lds, st, P, kv, lv0, with_anchor, cdf_anchor, cdf_delta, status, scales); break;
    default: hipLaunchKernelGGL((fit_levels_kernel<4>), grid, block, lds, st, P, kv, lv0, with_anchor, cdf_anchor, cdf_delta, status, scales); break;
  }
  return hipGetLastError();
}

// fit_hold_kernel's grid (one workgroup per CU, at most one per item), or 0 where it does not
// apply: G = 10, the longest chunk's groups in 32 slices of at most kHoldGroups groups, and
// under 2^16 steps per workgroup (the maxima tag)
int fit_hold_grid(const KParams& P) {
  if (P.G != 10) return 0;
  const int64_t n = P.CL < P.T ? P.CL : P.T;
  if ((((n + 9) / 10 + 31) >> 5) > kHoldGroups) return 0;
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      cus <= 0)
    return 0;
  const int64_t items = (int64_t)P.L * 2 * P.nblk;
  const int64_t grid = items < cus ? items : cus;
  const int64_t steps = (items + grid - 1) / grid * P.B * P.NC;
  return steps < 65535 ? (int)grid : 0;
}

template <int kNl>
hipError_t launch_fit_pass_nl(const KParams& P, const uint16_t* kv, int lv0, int with_anchor,
                              uint16_t* cdf_anchor, uint16_t* cdf_delta, uint32_t* status,
                              float* scales, hipStream_t st) {
  const size_t lds = (size_t)(with_anchor + kNl) * 32 * kHistP * sizeof(uint32_t);
  const bool g10 = P.G == 10;
  if constexpr (kNl == 1) {
    if (const int grid = fit_hold_grid(P)) {
      const void* fn = (const void*)fit_hold_kernel<kHoldGroups>;
      hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
      if (e != hipSuccess) return e;
      hipLaunchKernelGGL((fit_hold_kernel<kHoldGroups>), dim3((unsigned)grid), dim3(kFitThreads),
                         lds, st, P, kv, lv0, with_anchor, cdf_anchor, cdf_delta, status, scales);
      return hipGetLastError();
    }
  }
  const void* fn = g10 ? (const void*)fit_pass_kernel<kNl, 10> : (const void*)fit_pass_kernel<kNl, 0>;
  hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  const dim3 grid((unsigned)((int64_t)P.L * 2 * P.nblk)), block(kFitThreads);
  if (g10)
    hipLaunchKernelGGL((fit_pass_kernel<kNl, 10>), grid, block, lds, st, P, kv, lv0, with_anchor,
                       cdf_anchor, cdf_delta, status, scales);
  else
    hipLaunchKernelGGL((fit_pass_kernel<kNl, 0>), grid, block, lds, st, P, kv, lv0, with_anchor,
                       cdf_anchor, cdf_delta, status, scales);
  return hipGetLastError();
}

hipError_t launch_fit_pass(const KParams& P, const uint16_t* kv, int lv0, int nl, int with_anchor,
                           uint16_t* cdf_anchor, uint16_t* cdf_delta, uint32_t* status,
                           float* scales, hipStream_t st) {
  switch (nl) {
    case 1: return launch_fit_pass_nl<1>(P, kv, lv0, with_anchor, cdf_anchor, cdf_delta, status, scales, st);
    case 2: return launch_fit_pass_nl<2>(P, kv, lv0, with_anchor, cdf_anchor, cdf_delta, status, scales, st);
    case 3: return launch_fit_pass_nl<3>(P, kv, lv0, with_anchor, cdf_anchor, cdf_delta, status, scales, st);
    default: return launch_fit_pass_nl<4>(P, kv, lv0, with_anchor, cdf_anchor, cdf_delta, status, scales, st);
  }
}

// fit_pass_kernel's conditions: whole 64-channel blocks, and byte offsets inside one (context,
// layer, K/V) slab, plus the reads past the last token (a slice's: under 1/32 of a chunk and a
// group; the one-level maxima pass's: under 128 rows), that stay below 2^31
bool fit_pass_applies(const KParams& P) {
  return P.C % 64 == 0 && (int64_t)P.T * P.C * 2 < ((int64_t)1 << 30) &&
         (int64_t)(P.T + 128) * P.C * 2 < ((int64_t)1 << 31);
}
}  // namespace

// Largest count any (channel, kind, symbol) of the fit can reach: the anchors or the deltas of
// one channel over every chunk of every context.
int64_t cg_fit_max_count(const KParams& P) {
  int64_t na = 0, nd = 0;
  for (int c = 0; c < P.NC; ++c) {
    const int64_t n = (int64_t)(c + 1) * P.CL <= P.T ? P.CL : P.T - (int64_t)c * P.CL;
    const int64_t a = (n + P.G - 1) / P.G;
    na += a;
    nd += n - a;
  }
  return (int64_t)P.B * (na > nd ? na : nd);
}

hipError_t cg_launch_fit_levels(const KParams& P, const uint16_t* kv, uint16_t* cdf_anchor,
                                uint16_t* cdf_delta, uint32_t* status, float* scales,
                                hipStream_t st) {
  if (cg_fit_max_count(P) >= 65536) {
    // 16-bit counts could overflow: one 32-bit pass per level, and the finiteness scan
    for (int v = 0; v < P.NLV; ++v) {
      hipError_t e = cg_launch_fit(P, kv, v, v == 0 ? cdf_anchor : nullptr,
                                   cdf_delta + (size_t)v * P.L * 2 * P.C * 256, st,
                                   v == 0 ? scales : nullptr);
      if (e != hipSuccess) return e;
    }
    return status ? cg_launch_check_finite(kv, (int64_t)P.B * P.L * 2 * P.T * P.C, status, st)
                  : hipSuccess;
  }
  if (status) hipLaunchKernelGGL(zero_word, dim3(1), dim3(64), 0, st, status);
  const bool pass = fit_pass_applies(P);
  if (P.NLV == 1 && !pass)   // one level, any channel count: the 32-bit kernel of cg_fit_cdf
    return fit_slice_in_registers(P)
               ? launch_fit_kernel<false, true>(P, kv, 0, cdf_anchor, cdf_delta, nullptr, st,
                                                status, scales)
               : launch_fit_kernel<false, false>(P, kv, 0, cdf_anchor, cdf_delta, nullptr, st,
                                                 status, scales);
  // fit_pass_kernel: the anchors and up to four levels in the first pass, up to four levels in
  // each further one; fit_levels_kernel: up to four kinds per pass
  for (int lv0 = 0, i = 0; lv0 < P.NLV; ++i) {
    const int wa = i == 0 ? 1 : 0;
    const int nl = min(P.NLV - lv0, pass ? kPassKinds - 1 : kLevelKinds - wa);
    hipError_t e =
        pass ? launch_fit_pass(P, kv, lv0, nl, wa, cdf_anchor, cdf_delta, status, scales, st)
             : launch_fit_levels(P, kv, lv0, nl, wa, cdf_anchor, cdf_delta, status, scales, st);
    if (e != hipSuccess) return e;
    lv0 += nl;
  }
  return hipSuccess;
}
