// cg_decode.hip — GPU arithmetic decoding back to fp16 KV (CacheGen Sec. 5.2 "Arithmetic
// coding"; Sec. 6 "Speed optimization": decoding runs on the GPU, chunk by chunk).
//
// Work layout
//   One lane per stream. A wave decodes the 64 consecutive channels of one (context, chunk,
//   layer, K/V), so each decoded token row is one coalesced 128-byte store. A workgroup holds
//   up to 16 such waves that share (layer, K/V, channel block) and therefore share their
//   distribution tables, which are staged in LDS once per workgroup:
//     * delta tables (9 of 10 symbols): the whole 16-bit cumulative table, 256 entries, at a
//       520-byte stride (8-byte aligned; neighbouring lanes start in different banks), entries
//       255..259 holding 0xFFFF sentinels. Search: a 4-ary search over four levels (three
//       probes per level, the same steps in every lane, no divergence), the last level a single
//       aligned 8-byte read of four neighbouring entries.
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
// The payload is read through a 64-bit bit buffer fed from words requested one epoch (four
// tokens) ahead (see the reader state in the kernel). The words buffer must be readable
// CG_TAIL_WORDS words past offsets[S].
#include "../../include/cachegen.h"
#include "cg_device.h"

namespace {

constexpr int kMaxWaves = 16;
constexpr int kTabStride = 260;    // u16 per delta table in LDS (256 + 4 pad -> 520 bytes)
constexpr int kFenceStride = 18;   // u16 per anchor fence row (16 + 2 pad -> 36 bytes)
constexpr int kEpoch = 4;          // tokens between bitstream requests
constexpr int kRows = 8;           // decoded token rows staged in LDS per wave before a store

__device__ __forceinline__ int uni(int v) { return __builtin_amdgcn_readfirstlane(v); }

// x * c + c2 >> 16 as one 32x32+64 multiply-add. The addend passes through an empty asm so the
// compiler cannot fold x*c + c into a 64-bit (x + 1) * c.
__device__ __forceinline__ uint32_t scaled_off(uint32_t x, uint32_t c) {
  uint32_t c2 = c;
  asm volatile("" : "+v"(c2));
  return (uint32_t)(((uint64_t)x * c + c2) >> 16);
}

// Make the compiler wait here for a register produced by a load (once, outside the loop).
__device__ __forceinline__ void settle(uint32_t v) { asm volatile("" ::"v"(v)); }

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
  uint16_t* obuf_all = smem + 64 * kFenceStride; // [nw][kRows][64] decoded rows per wave
  uint16_t* tabs = obuf_all + nw * kRows * 64;   // [nsets][64][kTabStride]

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

  const int pair = uni(grp * nw + wave);
  const bool active = pair < n_pairs;
  const int b = uni(active ? pair / ncr : 0);
  const int c = uni(active ? c_begin + pair % ncr : 0);
  const int lv = uni(active ? min((int)chunk_level[(int64_t)b * P.NC + c], P.NLV - 1) : 0);

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
    if (lane < 2) dst[128 + lane] = 0xFFFFFFFFu;        // entries 256..259: sentinels
  }
  // ---- anchor fences cum[16 f] ----
  for (int idx = threadIdx.x; idx < 64 * 16; idx += blockDim.x) {
    const int t = idx >> 4, f = idx & 15;
    const int ch = cb * 64 + t;
    if (ch < P.C) fences[t * kFenceStride + f] = cdfA[((int64_t)(l * 2 + k) * P.C + ch) * 256 + 16 * f];
  }
  __syncthreads();

  if (!active) return;
  const int ch = cb * 64 + lane;
  const bool valid = ch < P.C;     // lanes past the last channel only help write rows
  const int chv = valid ? ch : cb * 64;

  const int64_t bclk = (((int64_t)b * P.NC + c) * P.L + l) * 2 + k;
  const int64_t sidx = cg_stream(P, bclk, chv);
  const int tok0 = c * P.CL;
  const int n = uni(min(P.CL, P.T - tok0));
  const float s = scales[sidx];
  const float bw = P.layer_bin[l] * P.level_mult[lv];
  const float w = bw * s;
  const uint16_t* dtab = tabs + (s_set_of_level[lv] * 64 + lane) * kTabStride;
  const uint16_t* ftab = fences + lane * kFenceStride;
  const uint16_t* gA = cdfA + ((int64_t)(l * 2 + k) * P.C + chv) * 256;

  const uint64_t total = offsets[P.S];
  if (total == 0) return;  // no payload at all: nothing can be decoded (uniform)
  // Bitstream reader state (plain locals so everything stays in registers). The lane consumes
  // bits from `buf`; whole words move into it from the four-word shift register s0..s3 (always
  // from s0). Every kEpoch tokens (the same tokens for the whole wave) the h words used since
  // the last epoch are replaced by the next ones, requested one epoch earlier into t0..t3, and
  // t0..t3 are requested again. A symbol takes at most 18 bits, so at most one word moves per
  // token and the shift register never runs dry inside an epoch. Requests are unconditional
  // loads (reading at most CG_TAIL_WORDS past the payload, which never affects a result), so
  // every epoch issues the same memory operations and the wait for t0..t3 comes one epoch
  // after the request instead of at once.
  const uint64_t o0 = offsets[sidx];
  const uint32_t* sbase = words + (o0 < total ? o0 : total);
  uint32_t D = sbase[0];
  uint64_t buf = (uint64_t)sbase[1] << 32;
  uint32_t avail = 32;
  uint32_t s0 = sbase[2], s1 = sbase[3], s2 = sbase[4], s3 = sbase[5];
  uint32_t hcnt = 0;
  uint64_t wpos = (o0 < total ? o0 : total) + 6;        // payload index of t0
  const uint64_t wcap = total;                          // requests start at most here
  const uint32_t* tq0 = words + (wpos < wcap ? wpos : wcap);
  uint32_t t0 = tq0[0], t1 = tq0[1], t2 = tq0[2], t3 = tq0[3];
  settle(D); settle(s0); settle(s1); settle(s2); settle(s3);
  settle((uint32_t)(buf >> 32));
  uint32_t low = 0u, rm1 = 0xFFFFFFFFu;

  uint16_t* row = out + cg_elem(P, b, l, k, tok0, cb * 64);  // wave-uniform row pointer
  const int64_t rstride = P.C;
  uint16_t* obuf = obuf_all + wave * kRows * 64;
  int r = 0;
  float a = 0.0f;
  int g = 0;
  int ep = 0;
  for (int j = 0; j < n; ++j) {
    const bool anchor = (g == 0);
    if (valid) {
      if (ep == kEpoch) {
        // s0..s(3-h) are still unread; positions 4-h..3 take t0..t(h-1)
        const bool g1 = hcnt >= 1, g2 = hcnt >= 2, g3 = hcnt >= 3, g4 = hcnt >= 4;
        const uint32_t n3 = g4 ? t3 : (g3 ? t2 : (g2 ? t1 : (g1 ? t0 : s3)));
        const uint32_t n2 = g4 ? t2 : (g3 ? t1 : (g2 ? t0 : s2));
        const uint32_t n1 = g4 ? t1 : (g3 ? t0 : s1);
        const uint32_t n0 = g4 ? t0 : s0;
        s0 = n0; s1 = n1; s2 = n2; s3 = n3;
        wpos += hcnt;
        hcnt = 0;
        // keep the new requests after the slide: the old t registers are dead by then, so
        // the loads can write them in place instead of through a copy that would wait
        __builtin_amdgcn_sched_barrier(0);
        const uint32_t* tq = words + (wpos < wcap ? wpos : wcap);
        t0 = tq[0]; t1 = tq[1]; t2 = tq[2]; t3 = tq[3];
        ep = 0;
      }
      ++ep;
      // 1. estimate of the target t = floor(((D + 1) * 2^16 - 1) / (rm1 + 1)); within one
      const float te = (float)D * (65536.0f * __builtin_amdgcn_rcpf((float)rm1));
      const uint32_t ti = min((uint32_t)te, 65534u);

      int sym;
      uint32_t clo, chi;
      if (anchor) {
        // fences in LDS: largest f with cum[16 f] <= ti, then the block from global memory
        int f = 0;
        if ((uint32_t)ftab[f + 8] <= ti) f += 8;
        if ((uint32_t)ftab[f + 4] <= ti) f += 4;
        if ((uint32_t)ftab[f + 2] <= ti) f += 2;
        if ((uint32_t)ftab[f + 1] <= ti) f += 1;
        const uint4* blk = reinterpret_cast<const uint4*>(gA + 16 * f);
        const uint4 q0 = blk[0], q1 = blk[1];
        const uint32_t v0 = q0.x & 0xFFFFu, v1 = q0.x >> 16, v2 = q0.y & 0xFFFFu, v3 = q0.y >> 16;
        const uint32_t v4 = q0.z & 0xFFFFu, v5 = q0.z >> 16, v6 = q0.w & 0xFFFFu, v7 = q0.w >> 16;
        const uint32_t v8 = q1.x & 0xFFFFu, v9 = q1.x >> 16, v10 = q1.y & 0xFFFFu, v11 = q1.y >> 16;
        const uint32_t v12 = q1.z & 0xFFFFu, v13 = q1.z >> 16, v14 = q1.w & 0xFFFFu;
        const uint32_t v15 = f == 15 ? CG_TOTAL : q1.w >> 16;  // symbol 255 does not exist
        const uint32_t v16 = f == 15 ? CG_TOTAL : (uint32_t)ftab[f + 1];
        // largest j in [0, 15] with v_j <= ti (v_0 <= ti holds), by selects only
        const bool c3 = v8 <= ti;
        const uint32_t x2 = c3 ? v12 : v4;
        const bool c2 = x2 <= ti;
        const uint32_t x1 = c3 ? (c2 ? v14 : v10) : (c2 ? v6 : v2);
        const bool c1 = x1 <= ti;
        const uint32_t x0 = c3 ? (c2 ? (c1 ? v15 : v13) : (c1 ? v11 : v9))
                               : (c2 ? (c1 ? v7 : v5) : (c1 ? v3 : v1));
        const bool c0 = x0 <= ti;
        const int jj = (c3 ? 8 : 0) + (c2 ? 4 : 0) + (c1 ? 2 : 0) + (c0 ? 1 : 0);
        // v_jj and v_jj+1: the last probe at or below ti and the last one above it
        uint32_t lo_v = v0, hi_v = v16;
        lo_v = c3 ? v8 : lo_v;  hi_v = c3 ? hi_v : v8;
        lo_v = c2 ? x2 : lo_v;  hi_v = c2 ? hi_v : x2;
        lo_v = c1 ? x1 : lo_v;  hi_v = c1 ? hi_v : x1;
        lo_v = c0 ? x0 : lo_v;  hi_v = c0 ? hi_v : x0;
        sym = 16 * f + jj;
        clo = lo_v;
        chi = hi_v;
      } else {
        // delta: 4-ary search in LDS for the largest i with cum[i] <= ti (sorted table; three
        // probes per level, the last level one aligned 8-byte read of cum[i .. i+3])
        int i;
        {
          const uint32_t p1 = dtab[64], p2 = dtab[128], p3 = dtab[192];
          i = 64 * ((p1 <= ti) + (p2 <= ti) + (p3 <= ti));
        }
        {
          const uint16_t* q = dtab + i;
          const uint32_t p1 = q[16], p2 = q[32], p3 = q[48];
          i += 16 * ((p1 <= ti) + (p2 <= ti) + (p3 <= ti));
        }
        {
          const uint16_t* q = dtab + i;
          const uint32_t p1 = q[4], p2 = q[8], p3 = q[12];
          i += 4 * ((p1 <= ti) + (p2 <= ti) + (p3 <= ti));
        }
        const uint2 quad = *reinterpret_cast<const uint2*>(dtab + i);   // cum[i .. i+3]
        const uint32_t x0 = quad.x & 0xFFFFu, x1 = quad.x >> 16;
        const uint32_t x2 = quad.y & 0xFFFFu, x3 = quad.y >> 16;
        const uint32_t x4 = dtab[i + 4];
        const bool b1 = x1 <= ti, b2 = x2 <= ti, b3 = x3 <= ti;
        sym = i + (int)b1 + (int)b2 + (int)b3;
        clo = b3 ? x3 : (b2 ? x2 : (b1 ? x1 : x0));
        chi = b3 ? x4 : (b2 ? x3 : (b1 ? x2 : x1));
        chi = sym == CG_NSYM - 1 ? CG_TOTAL : chi;
      }

      // 2. exact check: (R*clo) >> 16 <= D <= (R*chi >> 16) - 1; a miss means the estimate
      //    fell on the other side of a boundary: walk to the neighbour until the check holds
      uint32_t lo_off = scaled_off(rm1, clo);
      uint32_t hm1 = scaled_off(rm1, chi) - 1u;
      if (D < lo_off || D > hm1) {
        for (int guard = 0; guard < CG_NSYM; ++guard) {
          sym = (D < lo_off) ? max(sym - 1, 0) : min(sym + 1, CG_NSYM - 1);
          clo = anchor ? (uint32_t)gA[sym] : (uint32_t)dtab[sym];
          chi = sym + 1 >= CG_NSYM ? CG_TOTAL
                                   : (anchor ? (uint32_t)gA[sym + 1] : (uint32_t)dtab[sym + 1]);
          lo_off = scaled_off(rm1, clo);
          hm1 = scaled_off(rm1, chi) - 1u;
          if (D >= lo_off && D <= hm1) break;
        }
      }

      // 3. interval update and one-step renormalisation
      low += lo_off;
      rm1 = hm1 - lo_off;
      D -= lo_off;
      const uint32_t high = low + rm1;
      const uint32_t n1 = (uint32_t)__builtin_clz(low ^ high);   // low != high
      const uint32_t L1 = low << n1, H1 = high << n1;
      const uint32_t m = L1 & ~H1;
      const uint32_t n3 = (uint32_t)__builtin_clz(~(m << 1));    // ~(m << 1) is odd
      low = (L1 & 0x80000000u) | ((L1 << n3) & 0x7FFFFFFFu);
      const uint32_t nsh = n1 + n3;
      rm1 = (rm1 << nsh) | ((1u << nsh) - 1u);
      const uint32_t bits = nsh ? (uint32_t)(buf >> (64 - nsh)) : 0u;
      buf <<= nsh;
      avail -= nsh;
      if (avail < 32) {
        buf |= (uint64_t)s0 << (32 - avail);
        avail += 32;
        s0 = s1; s1 = s2; s2 = s3;
        ++hcnt;
      }
      D = (D << nsh) | bits;

      // dequantize (step a7) into the wave's row buffer
      const float qf = (float)(sym - 127);
      float v;
      if (anchor) {
        a = qf * s;
        v = a;
      } else {
        const float qw = qf * w;
        v = a + qw;
      }
      obuf[r * 64 + lane] = cg_f2h(v);
    }
    g = (g + 1 == P.G) ? 0 : g + 1;
    if (++r == kRows || j + 1 == n) {
      // write the staged rows: lane L stores 16 bytes (8 channels) of row L / 8
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      const int rr = lane >> 3, cc = (lane & 7) * 8;
      if (rr < r && cb * 64 + cc < P.C) {
        const uint4 vals = *reinterpret_cast<const uint4*>(obuf + rr * 64 + cc);
        uint16_t* dst = row + rr * rstride + cc;
        if (cb * 64 + cc + 8 <= P.C && (reinterpret_cast<uintptr_t>(dst) & 15) == 0) {
          *reinterpret_cast<uint4*>(dst) = vals;
        } else {
          const uint16_t hv[8] = {(uint16_t)(vals.x & 0xFFFFu), (uint16_t)(vals.x >> 16),
                                  (uint16_t)(vals.y & 0xFFFFu), (uint16_t)(vals.y >> 16),
                                  (uint16_t)(vals.z & 0xFFFFu), (uint16_t)(vals.z >> 16),
                                  (uint16_t)(vals.w & 0xFFFFu), (uint16_t)(vals.w >> 16)};
          for (int e = 0; e < 8; ++e)
            if (cb * 64 + cc + e < P.C) dst[e] = hv[e];
        }
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      row += r * rstride;
      r = 0;
    }
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
  const size_t lds =
      (size_t)(64 * kFenceStride + nw * kRows * 64 + nsets_max * 64 * kTabStride) * sizeof(uint16_t);
  hipError_t e = hipFuncSetAttribute((const void*)decode_kernel,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  const int64_t grid = (int64_t)P.L * 2 * P.nblk * n_groups;
  hipLaunchKernelGGL(decode_kernel, dim3((unsigned)grid), dim3(64 * nw), lds, st, P, words,
                     offsets, scales, chunk_level, cdf_anchor, cdf_delta, c_begin, c_end, nw,
                     out);
  return hipGetLastError();
}
