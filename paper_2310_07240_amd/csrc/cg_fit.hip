// cg_fit.hip — symbol-distribution fit (CacheGen Sec. 5.2 "Arithmetic coding": one
// distribution per channel-layer for deltas and one for anchors; Sec. 6: frequencies counted
// over the context's quantized symbols).
//
// One workgroup of 16 waves per (layer, K/V, 64-channel block); a lane owns one channel. The
// workgroup takes the (context, chunk) pairs of that block one after the other and splits each
// chunk's groups across its waves: every wave first reduces the absmax of its token slice, the
// slices are combined in LDS into the chunk's scale, then every wave quantizes its slice (groups
// are independent once the scale is known) and counts the symbols into LDS histograms. Rows
// are read 64 channels (128 B) at a time, so every load is one coalesced line. When the channel
// count is a multiple of 64 and half of a wave's slice is at most kHalf tokens (the paper's
// 1.5K-token chunks: 48-50), a lane takes two neighbouring channels (one dword per token) over
// half of the wave's groups; the slice is read once, into registers, with all its loads in
// flight together, and both passes work from the registers. Otherwise the rows are read once
// per pass, a lane per channel. Histograms use a
// 257-word stride so lanes that count the same symbol hit different banks. At the end each
// wave normalises histograms to 16-bit cumulative tables: per-lane partial sums, a wave
// reduction for the total, the argmax and the frequency sum, and a wave prefix scan.
#include "cg_device.h"

namespace {

constexpr int kFitWaves = 16;
constexpr int kFitThreads = kFitWaves * 64;
constexpr int kHist = 257;  // 255 symbols, padded; odd stride spreads lanes over the banks
constexpr int kHalf = 56;   // longest half slice per lane held in registers (one dword per token)

// Normalise one histogram [255] into cum[256] (entry 255 = 0) with one wave.
template <typename CountT>
__device__ void normalize_wave(const CountT* cnt, uint16_t* out) {
  const int lane = threadIdx.x & 63;
  uint64_t c[4];
  uint64_t local = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    int i = lane * 4 + j;
    c[j] = i < CG_NSYM ? cnt[i] : 0u;
    local += c[j];
  }
  uint64_t N = cg_wave_sum<uint64_t>(local);
  if (N == 0) {
#pragma unroll
    for (int j = 0; j < 4; ++j) c[j] = (lane * 4 + j) < CG_NSYM ? 1u : 0u;
    N = CG_NSYM;
  }
  // argmax with the lowest index on ties
  uint64_t best = 0;
  int besti = 0x7fffffff;
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
  uint32_t f[4];
  uint32_t fl = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    int i = lane * 4 + j;
    f[j] = i < CG_NSYM ? 1u + (uint32_t)((c[j] * (CG_TOTAL - CG_NSYM)) / N) : 0u;
    fl += f[j];
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

template <bool kPool, bool kRegs>
__global__ __launch_bounds__(kFitThreads) void fit_kernel(KParams P, const uint16_t* __restrict__ kv,
                                                         int level, uint16_t* __restrict__ cdf_anchor,
                                                         uint16_t* __restrict__ cdf_delta,
                                                         unsigned long long* __restrict__ pool) {
  extern __shared__ uint32_t cnt[];  // [2 kinds][64 channels][kHist]
  __shared__ float part[kFitWaves][64];
  const int cb = blockIdx.x % P.nblk;
  const int lk = blockIdx.x / P.nblk;
  const int l = lk >> 1, k = lk & 1;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;

  for (int i = threadIdx.x; i < 2 * 64 * kHist; i += kFitThreads) cnt[i] = 0;
  __syncthreads();

  const int ch = cb * 64 + lane;
  const bool act = ch < P.C;
  const float wfac = P.layer_bin[l] * P.level_mult[level];
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
      float m0 = 0.0f, m1 = 0.0f;
#pragma unroll
      for (int u = 0; u < kHalf; ++u) {
        if (u < len) {
          m0 = fmaxf(m0, fabsf((float)pk[u].x));
          m1 = fmaxf(m1, fabsf((float)pk[u].y));
        }
      }
      m0 = fmaxf(m0, __shfl_xor(m0, 32, 64));
      m1 = fmaxf(m1, __shfl_xor(m1, 32, 64));
      if (th == 0) {
        part[wave][2 * cp] = m0;
        part[wave][2 * cp + 1] = m1;
      }
      __syncthreads();
      m0 = 0.0f;
      m1 = 0.0f;
#pragma unroll
      for (int v = 0; v < kFitWaves; ++v) {
        m0 = fmaxf(m0, part[v][2 * cp]);
        m1 = fmaxf(m1, part[v][2 * cp + 1]);
      }
      const float s0 = (m0 == 0.0f) ? 1.0f : m0 / 127.0f;
      const float s1 = (m1 == 0.0f) ? 1.0f : m1 / 127.0f;
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
      float m = 0.0f;
#pragma unroll 8
      for (int j = j0; j < j1; ++j) m = fmaxf(m, fabsf(cg_h2f(x[(int64_t)j * rs])));
      part[wave][lane] = m;
      __syncthreads();
      m = 0.0f;
#pragma unroll
      for (int v = 0; v < kFitWaves; ++v) m = fmaxf(m, part[v][lane]);
      const float s = (m == 0.0f) ? 1.0f : m / 127.0f;
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
                             unsigned long long* pool, hipStream_t st) {
  const size_t lds = 2 * 64 * kHist * sizeof(uint32_t);
  hipError_t e = hipFuncSetAttribute((const void*)fit_kernel<kPool, kRegs>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  const int64_t grid = (int64_t)P.L * 2 * P.nblk;
  hipLaunchKernelGGL((fit_kernel<kPool, kRegs>), dim3((unsigned)grid), dim3(kFitThreads), lds,
                     st, P, kv, level, cdf_anchor, cdf_delta_level, pool);
  return hipGetLastError();
}
}  // namespace

hipError_t cg_launch_fit(const KParams& P, const uint16_t* kv, int level, uint16_t* cdf_anchor,
                         uint16_t* cdf_delta_level, hipStream_t st) {
  return fit_slice_in_registers(P)
             ? launch_fit_kernel<false, true>(P, kv, level, cdf_anchor, cdf_delta_level,
                                              nullptr, st)
             : launch_fit_kernel<false, false>(P, kv, level, cdf_anchor, cdf_delta_level,
                                               nullptr, st);
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
