// cg_decode.hip — GPU arithmetic decoding back to fp16 KV (CacheGen Sec. 5.2 "Arithmetic
// coding"; Sec. 6 "Speed optimization": decoding runs on the GPU, chunk by chunk).
//
// One lane per stream; a wave decodes the 64 consecutive channels of one (context, chunk,
// layer, K/V), so each decoded token row is one coalesced 128-byte store. The wave's 64 anchor
// tables and 64 delta tables are staged in LDS before the token loop.
//
// Decoder state per lane (Witten-Neal-Cleary decoder, rewritten on differences):
//   low  - low end of the interval
//   rm1  - high - low
//   D    - code value - low (always <= rm1)
// Per symbol:
//   1. target t = floor(((D + 1) * 2^16 - 1) / (rm1 + 1)); a float estimate (reciprocal,
//      relative error < 2^-21, so within one of t) picks a candidate symbol by binary search;
//   2. the candidate is checked exactly with the two products the interval update needs
//      anyway: symbol i is right iff (R*cum[i]) >> 16 <= D <= (R*cum[i+1] >> 16) - 1; a wrong
//      candidate moves one symbol towards the target and is checked again;
//   3. renormalisation in one step: n1 = clz(low ^ high) shared leading bits, then n3
//      "middle half" steps (run of low = 1 / high = 0 from bit 30 down); D and rm1 both shift
//      left by n = n1 + n3 taking in n stream bits (D) or ones (rm1).
#include "cg_device.h"

namespace {

constexpr int kDecThreads = 64;  // one wave per workgroup

struct BitSource {
  const uint32_t* p;    // next word
  const uint32_t* end;  // one past the stream's last word
  uint64_t buf;         // unread bits, left-aligned
  uint32_t avail;       // number of valid bits in buf (>= 32 between calls)

  __device__ __forceinline__ uint32_t next_word() {
    uint32_t w = 0;
    if (p < end) w = *p;
    ++p;
    return w;
  }
  // Take n <= 31 bits (n may be 0).
  __device__ __forceinline__ uint32_t take(uint32_t n) {
    const uint32_t bits = n ? (uint32_t)(buf >> (64 - n)) : 0u;
    buf <<= n;
    avail -= n;
    if (avail < 32) {
      buf |= (uint64_t)next_word() << (32 - avail);
      avail += 32;
    }
    return bits;
  }
};

__device__ __forceinline__ uint32_t cum_at(const uint16_t* tab, int i) {
  return i >= CG_NSYM ? CG_TOTAL : (uint32_t)tab[i];
}

__global__ __launch_bounds__(kDecThreads) void decode_kernel(
    KParams P, const uint32_t* __restrict__ words, const uint64_t* __restrict__ offsets,
    const float* __restrict__ scales, const uint8_t* __restrict__ chunk_level,
    const uint16_t* __restrict__ cdfA, const uint16_t* __restrict__ cdfD, int c_begin,
    int c_end, uint16_t* __restrict__ out) {
  __shared__ uint64_t lds64[2 * 64 * 64];  // [2 kinds][64 tables][256 u16]
  uint16_t* lds = reinterpret_cast<uint16_t*>(lds64);
  const int lane = threadIdx.x;
  const int64_t gw = blockIdx.x;
  const int ncr = c_end - c_begin;
  const int64_t bclk_r = gw / P.nblk;  // row index within the requested chunk range
  const int cb = (int)(gw % P.nblk);
  const int k = (int)(bclk_r & 1);
  int64_t r = bclk_r >> 1;
  const int l = (int)(r % P.L);
  r /= P.L;
  const int c = c_begin + (int)(r % ncr);
  const int b = (int)(r / ncr);
  const int64_t bclk = (((int64_t)b * P.NC + c) * P.L + l) * 2 + k;
  const int lv = min((int)chunk_level[(int64_t)b * P.NC + c], P.NLV - 1);

  // Stage the tables: table i of a kind is 512 bytes = 64 lanes x 8 bytes.
  const int nch = min(64, P.C - cb * 64);
  const uint64_t* gA = reinterpret_cast<const uint64_t*>(cdfA + ((int64_t)(l * 2 + k) * P.C + cb * 64) * 256);
  const uint64_t* gD = reinterpret_cast<const uint64_t*>(
      cdfD + ((((int64_t)lv * P.L + l) * 2 + k) * P.C + cb * 64) * 256);
  for (int t = 0; t < nch; ++t) {
    lds64[t * 64 + lane] = gA[t * 64 + lane];
    lds64[(64 + t) * 64 + lane] = gD[t * 64 + lane];
  }
  __syncthreads();

  const int ch = cb * 64 + lane;
  if (ch >= P.C) return;
  const int64_t sidx = cg_stream(P, bclk, ch);
  const int t0 = c * P.CL;
  const int n = min(P.CL, P.T - t0);
  const float s = scales[sidx];
  const float bw = P.layer_bin[l] * P.level_mult[lv];
  const float w = bw * s;
  const uint16_t* tabA = lds + lane * 256;
  const uint16_t* tabD = lds + (64 + lane) * 256;

  const uint64_t o0 = offsets[sidx], o1 = offsets[sidx + 1];
  BitSource src{words + o0, words + (o1 > o0 ? o1 : o0), 0ull, 0u};
  uint32_t D = src.next_word();
  src.buf = (uint64_t)src.next_word() << 32;
  src.avail = 32;
  uint32_t low = 0u, rm1 = 0xFFFFFFFFu;

  uint16_t* dst = out + cg_elem(P, b, l, k, t0, ch);
  float a = 0.0f;
  int g = 0;
  for (int j = 0; j < n; ++j) {
    const uint16_t* tab = (g == 0) ? tabA : tabD;
    // 1. estimate of the target and candidate symbol
    const float fr = (float)rm1 + 1.0f;
    const float fd = (float)D + 1.0f;
    const float te = fd * (65536.0f * __builtin_amdgcn_rcpf(fr));
    const uint32_t ti = min((uint32_t)te, 65535u);
    int i = 0;
#pragma unroll
    for (int step = 128; step >= 1; step >>= 1) {
      const int jn = i + step;
      if (jn <= CG_NSYM - 1 && (uint32_t)tab[jn] <= ti) i = jn;
    }
    // 2. exact check, moving one symbol at a time if the estimate was off
    uint32_t lo_off, hm1;
    for (int guard = 0; guard < CG_NSYM; ++guard) {
      const uint32_t clo = cum_at(tab, i), chi = cum_at(tab, i + 1);
      lo_off = (uint32_t)(((uint64_t)rm1 * clo + clo) >> 16);
      hm1 = (uint32_t)((((uint64_t)rm1 * chi + chi) >> 16) - 1ull);
      if (D < lo_off) { i = max(i - 1, 0); continue; }
      if (D > hm1) { i = min(i + 1, CG_NSYM - 1); continue; }
      break;
    }
    // 3. interval update and one-step renormalisation
    low += lo_off;
    rm1 = hm1 - lo_off;
    D -= lo_off;
    const uint32_t high = low + rm1;
    const uint32_t n1 = __clz(low ^ high);
    const uint32_t L1 = low << n1, H1 = high << n1;
    const uint32_t m = L1 & ~H1;
    const uint32_t n3 = __clz(~(m << 1));
    low = (L1 & 0x80000000u) | ((L1 << n3) & 0x7FFFFFFFu);
    const uint32_t nsh = n1 + n3;
    rm1 = (rm1 << nsh) | ((1u << nsh) - 1u);
    D = (D << nsh) | src.take(nsh);

    // dequantize (step a7) and store
    const int q = i - 127;
    float v;
    if (g == 0) {
      a = (float)q * s;
      v = a;
    } else {
      const float qw = (float)q * w;
      v = a + qw;
    }
    dst[(int64_t)j * P.C] = cg_f2h(v);
    g = (g + 1 == P.G) ? 0 : g + 1;
  }
}

}  // namespace

hipError_t cg_launch_decode(const KParams& P, const uint32_t* words, const uint64_t* offsets,
                            const float* scales, const uint8_t* chunk_level,
                            const uint16_t* cdf_anchor, const uint16_t* cdf_delta, int c_begin,
                            int c_end, uint16_t* out, hipStream_t st) {
  const int64_t waves = (int64_t)P.B * (c_end - c_begin) * P.L * 2 * P.nblk;
  if (waves == 0) return hipSuccess;
  hipLaunchKernelGGL(decode_kernel, dim3((unsigned)waves), dim3(kDecThreads), 0, st, P, words,
                     offsets, scales, chunk_level, cdf_anchor, cdf_delta, c_begin, c_end, out);
  return hipGetLastError();
}
