// cg_decode.hip — GPU arithmetic decoding back to fp16 KV (CacheGen Sec. 5.2 "Arithmetic
// coding"; Sec. 6 "Speed optimization": decoding runs on the GPU, chunk by chunk).
//
// Work layout
//   One lane per stream. A wave decodes the 64 consecutive channels of one (context, chunk,
//   layer, K/V), so each decoded token row is one coalesced 128-byte store. A workgroup holds
//   up to 16 such waves that share (layer, K/V, channel block) and therefore share their
//   distribution tables, which are staged in LDS once per workgroup:
//     * delta tables (9 of 10 symbols): the whole 16-bit cumulative table, 256 entries, at a
//       516-byte stride so the 64 lanes' tables start in different banks; entry 255 holds a
//       0xFFFF sentinel. Search: a fixed 8-step binary search (every lane takes the same steps,
//       no divergence), each probe an LDS read with an immediate offset.
//     * anchor tables (1 of 10 symbols; broad distributions): only 16 fences cum[16 f] per
//       table stay in LDS (36-byte stride). A 4-step fence search picks the block of 16
//       symbols, one 32-byte global load brings that block (L2-resident), and a 4-step binary
//       search over registers finishes. This keeps a workgroup of the Mistral-7B-shaped cache
//       at 35 KB so every wave of the grid is resident at once.
//
// Decoder state per lane (Witten-Neal-Cleary decoder, rewritten on differences):
//   low  - low end of the interval;  rm1 - high - low;  D - code value - low (<= rm1)
// Per symbol:
//   1. target t = floor(((D + 1) * 2^16 - 1) / (rm1 + 1)); a float estimate (reciprocal,
//      relative error < 2^-21, so within one of t) drives the table search;
//   2. the candidate is checked exactly with the two products the interval update needs
//      anyway: symbol i is right iff (R*cum[i]) >> 16 <= D <= (R*cum[i+1] >> 16) - 1; a wrong
//      candidate (the estimate fell on the other side of a boundary) moves one symbol toward
//      the target and is checked again;
//   3. renormalisation in one step: n1 = clz(low ^ high) shared leading bits, then n3
//      "middle half" steps (run of low = 1 / high = 0 from bit 30 down); D and rm1 both shift
//      left by n = n1 + n3 taking in n stream bits (D) or ones (rm1).
// The payload is read through a 64-bit bit buffer with two words prefetched ahead, so the
// global load latency is covered by the symbols decoded in between.
#include "cg_device.h"

namespace {

constexpr int kMaxWaves = 16;
constexpr int kTabStride = 258;    // u16 per delta table in LDS (256 + 2 pad -> 516 bytes)
constexpr int kFenceStride = 18;   // u16 per anchor fence row (16 + 2 pad -> 36 bytes)

struct BitIn {
  uint64_t buf;         // unread bits, left-aligned
  uint32_t avail;       // valid bits in buf, >= 32 between symbols
  uint32_t w1, w2;      // the next two payload words (already requested)
  const uint32_t* p;    // next word to request
  const uint32_t* end;  // one past the stream's last word

  __device__ __forceinline__ uint32_t fetch() {
    uint32_t w = 0;
    if (p < end) w = *p;
    ++p;
    return w;
  }
  // Take n bits, 0 <= n <= 31.
  __device__ __forceinline__ uint32_t take(uint32_t n) {
    const uint32_t bits = n ? (uint32_t)(buf >> (64 - n)) : 0u;
    buf <<= n;
    avail -= n;
    if (avail < 32) {
      buf |= (uint64_t)w1 << (32 - avail);
      avail += 32;
      w1 = w2;
      w2 = fetch();
    }
    return bits;
  }
};

// Cumulative frequency of symbol i (0..255) in an LDS delta table / a global anchor table.
__device__ __forceinline__ uint32_t cum_lds(const uint16_t* t, int i) {
  return i >= CG_NSYM ? CG_TOTAL : (uint32_t)t[i];
}
__device__ __forceinline__ uint32_t cum_glb(const uint16_t* t, int i) {
  return i >= CG_NSYM ? CG_TOTAL : (uint32_t)t[i];
}

__global__ __launch_bounds__(1024) void decode_kernel(
    KParams P, const uint32_t* __restrict__ words, const uint64_t* __restrict__ offsets,
    const float* __restrict__ scales, const uint8_t* __restrict__ chunk_level,
    const uint16_t* __restrict__ cdfA, const uint16_t* __restrict__ cdfD, int c_begin,
    int c_end, int nw, uint16_t* __restrict__ out) {
  extern __shared__ uint16_t smem[];
  __shared__ uint32_t s_mask;
  __shared__ int s_set_of_level[CG_MAX_LEVELS];
  __shared__ int s_level_of_set[CG_MAX_LEVELS];
  __shared__ int s_nsets;
  uint16_t* fences = smem;                       // [64][kFenceStride]
  uint16_t* tabs = smem + 64 * kFenceStride;     // [nsets][64][kTabStride]

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int nwaves = blockDim.x >> 6;
  const int ncr = c_end - c_begin;
  const int n_pairs = P.B * ncr;
  const int n_groups = (n_pairs + nw - 1) / nw;
  const int grp = blockIdx.x % n_groups;
  int rest = blockIdx.x / n_groups;
  const int cb = rest % P.nblk;
  rest /= P.nblk;
  const int k = rest & 1, l = rest >> 1;

  const int pair = grp * nw + wave;
  const bool active = pair < n_pairs;
  const int b = active ? pair / ncr : 0;
  const int c = active ? c_begin + pair % ncr : 0;
  const int lv = active ? min((int)chunk_level[(int64_t)b * P.NC + c], P.NLV - 1) : 0;

  if (threadIdx.x == 0) s_mask = 0u;
  __syncthreads();
  if (active && lane == 0) atomicOr(&s_mask, 1u << lv);
  __syncthreads();
  if (threadIdx.x == 0) {
    int n = 0;
    for (int v = 0; v < P.NLV; ++v)
      if ((s_mask >> v) & 1u) { s_set_of_level[v] = n; s_level_of_set[n] = v; ++n; }
    s_nsets = n;
  }
  __syncthreads();
  const int nsets = s_nsets;

  // ---- stage the delta tables of every level present: one 512-byte table per wave step ----
  for (int idx = wave; idx < nsets * 64; idx += nwaves) {
    const int s = idx >> 6, t = idx & 63;
    const int ch = cb * 64 + t;
    if (ch >= P.C) continue;
    const uint32_t* src = reinterpret_cast<const uint32_t*>(
        cdfD + ((((int64_t)s_level_of_set[s] * P.L + l) * 2 + k) * P.C + ch) * 256);
    uint32_t* dst = reinterpret_cast<uint32_t*>(tabs + (s * 64 + t) * kTabStride);
    const uint32_t v0 = src[lane];
    uint32_t v1 = src[lane + 64];
    if (lane == 63) v1 = (v1 & 0xFFFFu) | 0xFFFF0000u;  // entry 255: sentinel above any target
    dst[lane] = v0;
    dst[lane + 64] = v1;
  }
  // ---- anchor fences cum[16 f] ----
  for (int idx = threadIdx.x; idx < 64 * 16; idx += blockDim.x) {
    const int t = idx >> 4, f = idx & 15;
    const int ch = cb * 64 + t;
    if (ch < P.C) fences[t * kFenceStride + f] = cdfA[((int64_t)(l * 2 + k) * P.C + ch) * 256 + 16 * f];
  }
  __syncthreads();

  const int ch = cb * 64 + lane;
  if (!active || ch >= P.C) return;

  const int64_t bclk = (((int64_t)b * P.NC + c) * P.L + l) * 2 + k;
  const int64_t sidx = cg_stream(P, bclk, ch);
  const int t0 = c * P.CL;
  const int n = min(P.CL, P.T - t0);
  const float s = scales[sidx];
  const float bw = P.layer_bin[l] * P.level_mult[lv];
  const float w = bw * s;
  const uint16_t* dtab = tabs + (s_set_of_level[lv] * 64 + lane) * kTabStride;
  const uint16_t* ftab = fences + lane * kFenceStride;
  const uint16_t* gA = cdfA + ((int64_t)(l * 2 + k) * P.C + ch) * 256;

  const uint64_t o0 = offsets[sidx], o1 = offsets[sidx + 1];
  BitIn in;
  in.p = words + o0;
  in.end = words + (o1 > o0 ? o1 : o0);
  uint32_t D = in.fetch();
  in.buf = (uint64_t)in.fetch() << 32;
  in.avail = 32;
  in.w1 = in.fetch();
  in.w2 = in.fetch();
  uint32_t low = 0u, rm1 = 0xFFFFFFFFu;

  uint16_t* row = out + cg_elem(P, b, l, k, t0, cb * 64);  // wave-uniform row pointer
  float a = 0.0f;
  int g = 0;
  for (int j = 0; j < n; ++j) {
    // 1. estimate of the target
    const float fr = (float)rm1 + 1.0f;
    const float fd = (float)D + 1.0f;
    const float te = fd * (65536.0f * __builtin_amdgcn_rcpf(fr));
    const uint32_t ti = min((uint32_t)te, 65535u);

    int sym;
    uint32_t clo, chi;
    const bool anchor = (g == 0);
    if (anchor) {
      // fences in LDS: largest f with cum[16 f] <= ti
      int f = 0;
      if ((uint32_t)ftab[f + 8] <= ti) f += 8;
      if ((uint32_t)ftab[f + 4] <= ti) f += 4;
      if ((uint32_t)ftab[f + 2] <= ti) f += 2;
      if ((uint32_t)ftab[f + 1] <= ti) f += 1;
      const uint4* blk = reinterpret_cast<const uint4*>(gA + 16 * f);
      const uint4 q0 = blk[0], q1 = blk[1];
      uint32_t v[16] = {q0.x & 0xFFFFu, q0.x >> 16, q0.y & 0xFFFFu, q0.y >> 16,
                        q0.z & 0xFFFFu, q0.z >> 16, q0.w & 0xFFFFu, q0.w >> 16,
                        q1.x & 0xFFFFu, q1.x >> 16, q1.y & 0xFFFFu, q1.y >> 16,
                        q1.z & 0xFFFFu, q1.z >> 16, q1.w & 0xFFFFu, q1.w >> 16};
      if (f == 15) v[15] = CG_TOTAL;   // symbol 255 does not exist: cum[255] is the implicit top
      uint32_t lo_v = v[0];
      uint32_t hi_v = (f == 15) ? CG_TOTAL : (uint32_t)ftab[f + 1];
      int jj = 0;
      {  // largest jj in [0, 15] with v[jj] <= ti; track v[jj] and the next value
        uint32_t cand = v[8];
        if (cand <= ti) { jj = 8; lo_v = cand; } else { hi_v = cand; }
        cand = jj ? v[12] : v[4];
        if (cand <= ti) { jj += 4; lo_v = cand; } else { hi_v = cand; }
        cand = (jj & 8) ? ((jj & 4) ? v[14] : v[10]) : ((jj & 4) ? v[6] : v[2]);
        if (cand <= ti) { jj += 2; lo_v = cand; } else { hi_v = cand; }
        const uint32_t c8 = (jj & 8) ? ((jj & 4) ? ((jj & 2) ? v[15] : v[13]) : ((jj & 2) ? v[11] : v[9]))
                                     : ((jj & 4) ? ((jj & 2) ? v[7] : v[5]) : ((jj & 2) ? v[3] : v[1]));
        if (c8 <= ti) { jj += 1; lo_v = c8; } else { hi_v = c8; }
      }
      sym = 16 * f + jj;
      clo = lo_v;
      chi = hi_v;
    } else {
      // delta: fixed 8-step binary search in LDS for the largest i with cum[i] <= ti
      const uint16_t* q = dtab;
      if ((uint32_t)q[128] <= ti) q += 128;
      if ((uint32_t)q[64] <= ti) q += 64;
      if ((uint32_t)q[32] <= ti) q += 32;
      if ((uint32_t)q[16] <= ti) q += 16;
      if ((uint32_t)q[8] <= ti) q += 8;
      if ((uint32_t)q[4] <= ti) q += 4;
      if ((uint32_t)q[2] <= ti) q += 2;
      if ((uint32_t)q[1] <= ti) q += 1;
      sym = min((int)(q - dtab), CG_NSYM - 1);
      clo = dtab[sym];
      chi = sym == CG_NSYM - 1 ? CG_TOTAL : (uint32_t)dtab[sym + 1];
    }

    // 2. exact check: (R*clo) >> 16 <= D <= (R*chi >> 16) - 1
    uint32_t lo_off = (uint32_t)(((uint64_t)rm1 * clo + clo) >> 16);
    uint32_t hm1 = (uint32_t)((((uint64_t)rm1 * chi + chi) >> 16) - 1ull);
    if (D < lo_off || D > hm1) {
      for (int guard = 0; guard < CG_NSYM; ++guard) {
        sym = (D < lo_off) ? max(sym - 1, 0) : min(sym + 1, CG_NSYM - 1);
        clo = anchor ? cum_glb(gA, sym) : cum_lds(dtab, sym);
        chi = anchor ? cum_glb(gA, sym + 1) : cum_lds(dtab, sym + 1);
        lo_off = (uint32_t)(((uint64_t)rm1 * clo + clo) >> 16);
        hm1 = (uint32_t)((((uint64_t)rm1 * chi + chi) >> 16) - 1ull);
        if (D >= lo_off && D <= hm1) break;
      }
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
    D = (D << nsh) | in.take(nsh);

    // dequantize (step a7) and store
    const int q = sym - 127;
    float v;
    if (anchor) {
      a = (float)q * s;
      v = a;
    } else {
      const float qw = (float)q * w;
      v = a + qw;
    }
    row[lane] = cg_f2h(v);
    row += P.C;
    g = (g + 1 == P.G) ? 0 : g + 1;
  }
}

}  // namespace

hipError_t cg_launch_decode(const KParams& P, const uint32_t* words, const uint64_t* offsets,
                            const float* scales, const uint8_t* chunk_level,
                            const uint16_t* cdf_anchor, const uint16_t* cdf_delta, int c_begin,
                            int c_end, uint16_t* out, hipStream_t st) {
  const int64_t n_pairs = (int64_t)P.B * (c_end - c_begin);
  if (n_pairs == 0) return hipSuccess;
  const int nw = (int)(n_pairs < kMaxWaves ? n_pairs : kMaxWaves);
  const int64_t n_groups = (n_pairs + nw - 1) / nw;
  const int nsets_max = nw < P.NLV ? nw : P.NLV;
  const size_t lds = (size_t)(64 * kFenceStride + nsets_max * 64 * kTabStride) * sizeof(uint16_t);
  hipError_t e = hipFuncSetAttribute((const void*)decode_kernel,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  const int64_t grid = (int64_t)P.L * 2 * P.nblk * n_groups;
  hipLaunchKernelGGL(decode_kernel, dim3((unsigned)grid), dim3(64 * nw), lds, st, P, words,
                     offsets, scales, chunk_level, cdf_anchor, cdf_delta, c_begin, c_end, nw,
                     out);
  return hipGetLastError();
}
