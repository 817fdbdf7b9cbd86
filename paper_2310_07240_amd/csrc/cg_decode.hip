// cg_decode.hip — GPU arithmetic decoding back to fp16 KV (CacheGen Sec. 5.2 "Arithmetic
// coding"; Sec. 6 "Speed optimization": decoding runs on the GPU, chunk by chunk).
//
// Work layout (both kernels)
//   One lane per stream. A wave decodes the 64 consecutive channels of one (context, chunk,
//   layer, K/V), so each decoded token row is one coalesced 128-byte store. A workgroup holds
//   up to 16 such waves that share (layer, K/V, channel block) and therefore share their
//   distribution tables. decode_kernel stages the delta tables (9 of 10 symbols) of the levels
//   present in LDS once per workgroup: the whole 16-bit cumulative table, 256 entries, at a
//   520-byte stride (8-byte aligned; neighbouring lanes start in different banks), entries
//   255..259 holding 0xFFFF sentinels; its anchor tables (1 of 10 symbols) stay in global
//   memory, a symbol reading one 32-byte block of 16 entries and finishing with a select search
//   in registers. decode_g10_kernel stages the anchor tables, then the delta tables, in a column
//   layout (entry i of the lane in column L at u16 64 i + L, so that a wave's 64 lookups fall in
//   different banks), or the delta tables of several levels as windows of contiguous entries
//   (see the kernel's comment). Fewer waves per workgroup when the worst-case table sets would
//   not fit in a CU's LDS.
//   decode_g10_kernel puts several such units (layer, K/V, channel block) in one workgroup
//   while the grid still covers every CU: a CU then runs one workgroup, whose waves the
//   hardware spreads evenly over the four SIMDs (several small workgroups per CU can land four
//   waves on one SIMD and two on another, and the kernel waits for the most loaded SIMD). Wave
//   w of a workgroup decodes pair slot w / units of unit w % units, so each SIMD gets one wave
//   of every slot; slots are chunk-major (pair p = chunk p / B of context p % B), so the waves
//   of a workgroup share a chunk length, and with one context the last, shorter chunk is
//   decoded by the youngest waves (older waves issue first).
//
// decode_kernel (any group size): anchor fences cum[16 f] in LDS; the delta search is a 4-ary
//   search over four levels in LDS (three probes per level, the last level one aligned 8-byte
//   read of four neighbouring entries); bitstream epochs every four tokens.
// decode_g10_kernel (group size 10, the paper's): the token schedule of a group is fixed at
//   compile time and the fences of both tables sit in registers (see the kernel's comment).
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
// The payload is read from words requested one epoch (three or four tokens) ahead: decode_kernel
// keeps a 64-bit bit buffer refilled from a four-word shift register, decode_g10_kernel and the
// token-layout decoder a four-word window with a bit position (see G10Lane). The words buffer
// must be readable CG_TAIL_WORDS words past offsets[S].
//
// tok_decode_kernel / tok_dequant_kernel decode the token-parallel layout (one stream per
// context, layer, K/V and token; see their comment).
#include "../../include/cachegen.h"
#include <type_traits>

#include "cg_device.h"

namespace {

constexpr int kMaxWaves = 16;
constexpr int kMaxUnits = 16;   // (layer, K/V, channel block) units per workgroup
// static LDS of the kernel with several units (masks, level maps, SIMD ids, remaining counts);
// the dynamic LDS budget leaves 1 KB for it
static_assert(4 * kMaxUnits + 3 * kMaxUnits * CG_MAX_LEVELS + kMaxWaves + 4 * kMaxWaves <= 1024 - 64,
              "static LDS exceeds the reserve");
constexpr int kStageBatch = 8;  // table-staging loads in flight per lane
constexpr int kDeltaPre = 8;
constexpr int kAnchorPre = 12;  // anchor-table loads per lane issued first   // delta-table loads per lane issued before the phase barrier
constexpr size_t kLdsBudget = 160 * 1024 - 1024;   // dynamic LDS per workgroup (CDNA4: 160 KB)
constexpr int kTabStride = 260;    // u16 per delta table in LDS (256 + 4 pad -> 520 bytes)
constexpr int kColSet = 260 * 64;  // u16 of a 64-table set in the column layout (rows of 64)
constexpr int kFenceStride = 18;   // u16 per anchor fence row (16 + 2 pad -> 36 bytes)
constexpr int kEpoch = 4;          // tokens between bitstream requests
constexpr int kRows = 8;           // decoded token rows staged in LDS per wave before a store

__device__ __forceinline__ int uni(int v) { return __builtin_amdgcn_readfirstlane(v); }

// (x * c + c) >> 16 = (x + 1) * c >> 16 with x + 1 up to 2^32, as one 32x32+64 multiply-add
// (written out so that it is not rewritten as a 64-bit product of x + 1, and so that c can be
// both the multiplier and the low half of the addend).
__device__ __forceinline__ uint32_t scaled_off(uint32_t x, uint32_t c) {
  uint64_t r, carry;
  // c as a plain 32-bit value: a table entry loaded as 16 bits would otherwise be masked to
  // 16 bits again before it is widened for the addend
  asm("" : "+v"(c));
  asm("v_mad_u64_u32 %0, %1, %2, %3, %4" : "=v"(r), "=s"(carry) : "v"(x), "v"(c), "v"((uint64_t)c));
  return (uint32_t)(r >> 16);
}

// Make the compiler wait here for a register produced by a load (once, outside the loop).
__device__ __forceinline__ void settle(uint32_t v) { asm volatile("" ::"v"(v)); }

// Number of middle-half (E3) steps after the shared leading bits are shifted out: L1 = low and
// H1 = high shifted left by those bits (so L1 < 2^31 <= H1); the steps are the run of bit
// positions 30, 29, ... where low has a one and high a zero. With the top bit of (L1 & ~H1)
// set, that run is the count of bits after the sign bit equal to it, which v_ffbh_i32 gives
// plus one.
__device__ __forceinline__ uint32_t e3_run(uint32_t L1, uint32_t H1) {
  uint32_t n;
  asm("v_ffbh_i32 %0, %1" : "=v"(n) : "v"((L1 & ~H1) | 0x80000000u));
  return n - 1u;
}

// 16-byte store of decoded fp16 that is not read again by this kernel (non-temporal, so the
// output stream does not push the anchor tables out of the L2).
__device__ __forceinline__ void store_row16(uint16_t* dst, const uint4& v) {
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
  const u32x4 vv = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(vv, reinterpret_cast<u32x4*>(dst));
}

// Last level of the delta search. q points at cum[i] (8-byte aligned) with cum[i] <= ti; the
// symbol is i + c with c in [0, 3]. cum[i .. i+3] come in one 8-byte read (x = cum[i] |
// cum[i+1] << 16, y = cum[i+2] | cum[i+3] << 16), cum[i+4] in a second. The count of entries
// <= ti uses packed 16-bit math: (ti + 1) - cum saturates to zero exactly when cum > ti,
// min(., 1) turns each half into 0 / 1 and a dot product with (1, 1) adds the halves; cum[i]
// always counts, so c = count - 1. Returns c; `pair` = cum[i + c] | cum[i + c + 1] << 16.
__device__ __forceinline__ uint32_t delta_leaf(const uint16_t* q, uint32_t ti, uint32_t& pair) {
  const uint2 xy = *reinterpret_cast<const uint2*>(q);
  const uint32_t x4 = q[4];
  const uint32_t tt = (ti + 1u) * 0x00010001u;
  const uint32_t one2 = 0x00010001u;
  uint32_t ia, ib, c;
  asm("v_pk_sub_u16 %0, %1, %2 clamp" : "=v"(ia) : "v"(tt), "v"(xy.x));
  asm("v_pk_sub_u16 %0, %1, %2 clamp" : "=v"(ib) : "v"(tt), "v"(xy.y));
  asm("v_pk_min_u16 %0, %1, %2" : "=v"(ia) : "v"(ia), "v"(one2));
  asm("v_pk_min_u16 %0, %1, %2" : "=v"(ib) : "v"(ib), "v"(one2));
  asm("v_dot2_u32_u16 %0, %1, %2, %3" : "=v"(c) : "v"(ia), "v"(one2), "v"(0xFFFFFFFFu));
  asm("v_dot2_u32_u16 %0, %1, %2, %3" : "=v"(c) : "v"(ib), "v"(one2), "v"(c));
  // (cum[i + c], cum[i + c + 1]) is the 32-bit window at 16 c bits of x : y : x4
  const uint32_t hi2 = (c & 2u) ? x4 : xy.y;
  const uint32_t lo2 = (c & 2u) ? xy.y : xy.x;
  pair = __builtin_amdgcn_alignbit(hi2, lo2, (c & 1u) << 4);
  return c;
}

// 16 j - 127 for the largest j in [0, 15] with v[j] <= ti (sorted v, v[0] <= ti < v[16]): a
// binary search by selects on registers, each decision also picking the candidates of the
// later levels (a chain of four compare / select steps), its index scaled and biased so that
// adding the offset of the symbol inside the block gives the quantized value.
__device__ __forceinline__ int fence_q(const uint32_t (&v)[17], uint32_t ti) {
  const bool c3 = v[8] <= ti;
  const uint32_t p4 = c3 ? v[12] : v[4];
  const uint32_t p2a = c3 ? v[10] : v[2], p2b = c3 ? v[14] : v[6];
  const uint32_t p1a = c3 ? v[9] : v[1], p1b = c3 ? v[11] : v[3];
  const uint32_t p1c = c3 ? v[13] : v[5], p1d = c3 ? v[15] : v[7];
  const bool c2 = p4 <= ti;
  const uint32_t p2 = c2 ? p2b : p2a;
  const uint32_t p1e = c2 ? p1c : p1a, p1f = c2 ? p1d : p1b;
  const bool c1 = p2 <= ti;
  const uint32_t p1 = c1 ? p1f : p1e;
  const bool c0 = p1 <= ti;
  return (c3 ? 1 : -127) + (c2 ? 64 : 0) + (c1 ? 32 : 0) + (c0 ? 16 : 0);
}

__global__ __launch_bounds__(1024) void decode_kernel(
    KParams P, const uint32_t* __restrict__ words, const uint64_t* __restrict__ offsets,
    const float* __restrict__ scales, const uint8_t* __restrict__ chunk_level,
    const uint16_t* __restrict__ cdfA, const uint16_t* __restrict__ cdfD, int c_begin,
    int c_end, int nw, uint16_t* __restrict__ out) {
  extern __shared__ __attribute__((aligned(16))) uint16_t smem[];
  __shared__ uint32_t s_mask;
  __shared__ int s_set_of_level[CG_MAX_LEVELS];
  __shared__ int s_level_of_set[CG_MAX_LEVELS];
  __shared__ int s_nsets;
  uint16_t* fences = smem;                       // [64][kFenceStride]
  uint16_t* obuf_all = smem + 64 * kFenceStride; // [nw][kRows][64] decoded rows per wave
  uint16_t* tabs = obuf_all + nw * kRows * 64;   // [nsets][64][kTabStride]

  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int nwaves = blockDim.x >> 6;
  const int ncr = c_end - c_begin;
  const int n_pairs = P.B * ncr;
  const int n_groups = (n_pairs + nw - 1) / nw;
  int rest, grp;
  cg_xcd_map(P.L * 2 * P.nblk, n_groups, rest, grp);
  if (rest >= P.L * 2 * P.nblk) return;   // past the last unit (uniform over the workgroup)
  const int cb = rest % P.nblk;
  rest /= P.nblk;
  const int k = rest & 1, l = rest >> 1;

  const int pair = uni(grp * nw + wave);
  const bool active = pair < n_pairs;
  // pairs chunk-major: the waves of a workgroup decode the same chunk of consecutive contexts,
  // so they have the same token count and finish together
  const int b = uni(active ? pair % P.B : 0);
  const int c = uni(active ? c_begin + pair / P.B : 0);
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
  const bool valid = ch < P.C;
  // Lanes past the last channel (only when C is not a multiple of 64) decode a copy of the
  // block's first channel, so the whole wave runs the same code; their rows are never stored.
  const int lsrc = valid ? lane : 0;
  const int chv = cb * 64 + lsrc;

  const int64_t bclk = (((int64_t)b * P.NC + c) * P.L + l) * 2 + k;
  const int64_t sidx = cg_stream(P, bclk, chv);
  const int tok0 = c * P.CL;
  const int n = uni(min(P.CL, P.T - tok0));
  const float s = scales[sidx];
  const float bw = P.layer_bin[l] * P.level_mult[lv];
  const float w = bw * s;
  const uint16_t* dtab = tabs + (s_set_of_level[lv] * 64 + lsrc) * kTabStride;
  const uint16_t* ftab = fences + lsrc * kFenceStride;
  const uint16_t* gA = cdfA + ((int64_t)(l * 2 + k) * P.C + chv) * 256;
  cg_glb_u16* gA1 = (cg_glb_u16*)gA;
  cg_lds_u16* dtab3 = (cg_lds_u16*)dtab;

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
  int nsym = 0;   // symbols decoded so far (the bitstream epochs come every kEpoch symbols)

  // One symbol under the lane's anchor (global blocks, fences in LDS) or delta (LDS) table.
  auto decode_symbol = [&](bool anchor) __attribute__((always_inline)) -> int {
    if ((nsym & (kEpoch - 1)) == 0 && nsym != 0) {
      // s0..s(3-h) are still unread; positions 4-h..3 take t0..t(h-1). Selects between
      // register copies (selects between the captured variables themselves could become
      // selects of their addresses, which would move the state to scratch memory).
      const bool g1 = hcnt >= 1, g2 = hcnt >= 2, g3 = hcnt >= 3, g4 = hcnt >= 4;
      uint32_t T0 = t0, T1 = t1, T2 = t2, T3 = t3, S0 = s0, S1 = s1, S2 = s2, S3 = s3;
      asm("" : "+v"(T0), "+v"(T1), "+v"(T2), "+v"(T3), "+v"(S0), "+v"(S1), "+v"(S2), "+v"(S3));
      const uint32_t n3 = g4 ? T3 : (g3 ? T2 : (g2 ? T1 : (g1 ? T0 : S3)));
      const uint32_t n2 = g4 ? T2 : (g3 ? T1 : (g2 ? T0 : S2));
      const uint32_t n1 = g4 ? T1 : (g3 ? T0 : S1);
      const uint32_t n0 = g4 ? T0 : S0;
      s0 = n0; s1 = n1; s2 = n2; s3 = n3;
      wpos += hcnt;
      hcnt = 0;
      // keep the new requests after the slide: the old t registers are dead by then, so
      // the loads can write them in place instead of through a copy that would wait
      __builtin_amdgcn_sched_barrier(0);
      const uint32_t* tq = words + (wpos < wcap ? wpos : wcap);
      t0 = tq[0]; t1 = tq[1]; t2 = tq[2]; t3 = tq[3];
    }
    ++nsym;
    // 1. estimate of the target t = floor(((D + 1) * 2^16 - 1) / (rm1 + 1)); within one
    const float te = (float)D * (65536.0f * __builtin_amdgcn_rcpf((float)rm1));
    const uint32_t ti = min((uint32_t)te, 65534u);
    const uint32_t kneg = ~ti;   // p + kneg has its top bit set exactly when p <= ti

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
      // probes per level counted by sign bits, the last level one aligned 8-byte read)
      const uint16_t* q = dtab;
      q += 64 * ((((uint32_t)q[64] + kneg) >> 31) + (((uint32_t)q[128] + kneg) >> 31) +
                 (((uint32_t)q[192] + kneg) >> 31));
      q += 16 * ((((uint32_t)q[16] + kneg) >> 31) + (((uint32_t)q[32] + kneg) >> 31) +
                 (((uint32_t)q[48] + kneg) >> 31));
      q += 4 * ((((uint32_t)q[4] + kneg) >> 31) + (((uint32_t)q[8] + kneg) >> 31) +
                (((uint32_t)q[12] + kneg) >> 31));
      uint32_t pr;
      const uint32_t cc = delta_leaf(q, ti, pr);
      sym = (int)((((uint32_t)(uintptr_t)q - (uint32_t)(uintptr_t)dtab) >> 1) + cc);
      clo = pr & 0xFFFFu;
      chi = sym == CG_NSYM - 1 ? CG_TOTAL : pr >> 16;
    }

    // 2. exact check: (R*clo) >> 16 <= D <= (R*chi >> 16) - 1; a miss means the estimate
    //    fell on the other side of a boundary: walk to the neighbour until the check holds
    uint32_t lo_off = scaled_off(rm1, clo);
    uint32_t hm1 = scaled_off(rm1, chi) - 1u;
    if (D < lo_off || D > hm1) {
      for (int guard = 0; guard < CG_NSYM; ++guard) {
        sym = (D < lo_off) ? max(sym - 1, 0) : min(sym + 1, CG_NSYM - 1);
        const int s1 = min(sym + 1, CG_NSYM - 1);
        clo = anchor ? (uint32_t)gA1[sym] : (uint32_t)dtab3[sym];
        chi = anchor ? (uint32_t)gA1[s1] : (uint32_t)dtab3[s1];
        chi = sym + 1 >= CG_NSYM ? CG_TOTAL : chi;
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
    const uint32_t n3 = e3_run(L1, H1);
    low = (L1 << n3) & 0x7FFFFFFFu;   // L1 has a clear top bit
    const uint32_t nsh = n1 + n3;
    rm1 = (rm1 << nsh) | ((1u << nsh) - 1u);
    // D takes the next nsh bits: a funnel shift of (D : top word of buf); nsh = 0 keeps D
    const uint32_t dsh = __builtin_amdgcn_alignbit(D, (uint32_t)(buf >> 32), 32u - nsh);
    D = nsh ? dsh : D;
    buf <<= nsh;
    avail -= nsh;
    if (avail < 32) {
      buf |= (uint64_t)s0 << (32 - avail);
      avail += 32;
      s0 = s1; s1 = s2; s2 = s3;
      ++hcnt;
    }
    return sym - 127;
  };

  // anchor phase: the chunk's anchors come first in the stream. Each one's fp16 value goes to
  // its row; its quantized value q goes to the group's first delta row (when there is one),
  // where the delta phase reads it back before the decoded delta replaces it.
  uint16_t* col = row + lsrc;
  const int na = (n + P.G - 1) / P.G;
  for (int g = 0; g < na; ++g) {
    const int qi = decode_symbol(true);
    uint16_t* ra = col + (int64_t)g * P.G * rstride;
    if (g * P.G + 1 < n && P.G > 1) ra[rstride] = (uint16_t)qi;
    ra[0] = cg_f2h((float)qi * s);
  }
  if (P.G == 1) return;   // every token is an anchor

  // delta phase: rows are staged in LDS as before; an anchor row takes the value the anchor
  // phase stored (read back from its row)
  int r = 0;
  float a = 0.0f;
  int g = 0;
  for (int j = 0; j < n; ++j) {
    float v;
    if (g == 0) {
      const uint16_t* ra = col + (int64_t)j * rstride;
      if (j + 1 < n) a = (float)(int)(int16_t)ra[rstride] * s;
      v = cg_h2f(ra[0]);
    } else {
      const int qi = decode_symbol(false);
      v = a + (float)qi * w;
    }
    obuf[r * 64 + lane] = cg_f2h(v);
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
          store_row16(dst, vals);
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


// ---- group size 10: the schedule of a group is fixed at compile time -------------------------
// Same decoder, same results, for the paper's group of 10 tokens (one anchor, nine deltas). A
// stream holds its chunk's anchors first, then its deltas, so the kernel runs in two phases:
//   * anchor phase: the anchor tables of the workgroup's units are staged in LDS; each wave
//     decodes its anchors, kAnchorRun per bitstream epoch, and keeps each anchor's quantized
//     value q in the anchor's own row;
//   * delta phase: the delta tables replace the anchor tables in LDS; each group reads back its
//     anchor's q (requested a group ahead), decodes its nine deltas with epochs before deltas
//     1 and 6, and stores rows 0..9 (the anchor's fp16 value over the kept q).
// Both searches start from the 15 fences cum[16 f] of the table in registers (a 4-step select
// search, no memory round trip), then take three LDS round trips: one 4-ary level and the
// leaf (each two compare / select steps over entries read together), and the candidate's two
// bounds, read from its address.
constexpr int kG10 = 10;
constexpr int kAnchorRun = 5;   // anchors per bitstream epoch (a symbol takes <= 18 bits)

// Per-lane decoder state of the group-of-10 kernel (plain scalars: it lives in registers).
// Bitstream reader: the next stream bits are the last `avail` bits of w0 (0..31; 0 when w0 is
// used up), then w1, w2, w3. A token takes n <= 18 bits (the interval is wider than 2^30
// before a symbol and at least 2^14 after it, and renormalisation doubles it to at most 2^32),
// so it crosses at most one word boundary and w0 moves up by at most one word; five tokens take
// at most 90 bits, which from an epoch start never reach past w3 (90 < 96), so at most three
// words leave between two epoch boundaries. (Bits that the 32-bit window read takes past the
// token's own come from words already moved and are shifted out unused.)
struct G10Lane {
  // low is kept as the value before its last renormalisation shift by lsh, and only its low 31
  // bits are kept exact: the interval update reads low << lsh + lo_off, and renormalisation
  // uses that sum's bits below the top one (its top bit and that of high = low + hoff - 1 are
  // both off by the same amount, which the xor cancels and the run count masks)
  uint32_t D, low, lsh, rm1;     // code value - low, low (see above), high - low
  uint32_t w0, w1, w2, w3;       // the next stream words, w0 partly consumed
  uint32_t avail;                // bits of w0 not yet taken (< 32)
  uint32_t t0, t1, t2, t3;       // the four words after w3, requested one epoch ahead
  uint32_t hcnt;                 // words moved out of w0 since the last epoch (<= 3)
  uint32_t widx;                 // index of t0's word from the stream's first word
  float a;                       // dequantized anchor of the current group
};

// Epoch boundary, in two halves: g10_epoch_take replaces the hcnt words dropped from the front
// of w0..w3 since the last boundary at the back by as many requested words (it waits for the
// previous request); g10_epoch_request requests the next four. A caller may issue stores
// between the two, so that the next boundary's wait (for this request) covers them long after.
__device__ __forceinline__ void g10_epoch_take(G10Lane& st) {
  const uint32_t h = st.hcnt;
  // register copies behind an empty asm: selects between the fields themselves could be
  // turned into a select of their addresses, which would move the state to scratch memory
  uint32_t t0 = st.t0, t1 = st.t1, t2 = st.t2;
  uint32_t w1 = st.w1, w2 = st.w2, w3 = st.w3;
  asm("" : "+v"(t0), "+v"(t1), "+v"(t2), "+v"(w1), "+v"(w2), "+v"(w3));
  const bool g1 = h >= 1, g2 = h >= 2, g3 = h >= 3;
  w3 = g3 ? t2 : (g2 ? t1 : (g1 ? t0 : w3));
  w2 = g3 ? t1 : (g2 ? t0 : w2);
  w1 = g3 ? t0 : w1;
  // materialise the window here (else the selects are folded into every token's word shift)
  asm("" : "+v"(w1), "+v"(w2), "+v"(w3));
  st.w1 = w1;
  st.w2 = w2;
  st.w3 = w3;
  st.widx += h;
  st.hcnt = 0;
}
__device__ __forceinline__ void g10_epoch_request(G10Lane& st, const uint32_t* __restrict__ sbase,
                                                  uint32_t cap) {
  __builtin_amdgcn_sched_barrier(0);
  const uint32_t* tq = sbase + (st.widx < cap ? st.widx : cap);
  st.t0 = tq[0];
  st.t1 = tq[1];
  st.t2 = tq[2];
  st.t3 = tq[3];
}
__device__ __forceinline__ void g10_epoch(G10Lane& st, const uint32_t* __restrict__ sbase,
                                          uint32_t cap) {
  g10_epoch_take(st);
  g10_epoch_request(st, sbase, cap);
}

// Interval update after the symbol [lo_off, hoff) (offsets from low; d = D - lo_off, rsz =
// hoff - lo_off): one-step renormalisation and the refill of D from the word window.
__device__ __forceinline__ void g10_advance(G10Lane& st, uint32_t lo_off, uint32_t hoff,
                                            uint32_t d, uint32_t rsz) {
  // renormalisation: n1 shared leading bits of low and high, then the middle-half run of
  // f - 1 steps, read as in e3_run from (low & ~high) << n1 (the same bits as L1 & ~H1, with
  // L1 = low << n1 and H1 = high << n1); in all nsh = n1 + f - 1 shifts, after which the new
  // low is low << nsh without its top bit (the shift waits for the next symbol)
  const uint32_t low = (st.low << st.lsh) + lo_off;
  const uint32_t high = low + rsz - 1u;
  const uint32_t n1 = (uint32_t)__builtin_clz(low ^ high);
  uint32_t e, f;
  asm("v_bfi_b32 %0, %1, 0, %2" : "=v"(e) : "v"(high), "v"(low));   // low & ~high
  asm("v_ffbh_i32 %0, %1" : "=v"(f) : "v"((e << n1) | 0x80000000u));   // run + 1
  const uint32_t nsh = n1 + f - 1u;
  st.low = low;
  st.lsh = nsh;
  // high - low + 1 scales by 2^nsh (a result of 2^32 wraps to 0, giving rm1 = 2^32 - 1)
  st.rm1 = (rsz << nsh) - 1u;
  // D takes the next nsh stream bits: the 32 bits after the taken ones of w0:w1, then a 64-bit
  // shift
  const uint32_t win = __builtin_amdgcn_alignbit(st.w0, st.w1, st.avail);
  uint32_t Dn = (uint32_t)(((((uint64_t)d) << 32) | win) << nsh >> 32);
  asm("" : "+v"(Dn));   // keep D a 32-bit value (not the top half of a 64-bit one)
  st.D = Dn;
  // the borrow of avail - nsh is the word advance (one subtract with carry out, no compare)
  uint32_t a2;
  const bool adv = __builtin_sub_overflow(st.avail, nsh, &a2);
  st.w0 = adv ? st.w1 : st.w0;
  st.w1 = adv ? st.w2 : st.w1;
  st.w2 = adv ? st.w3 : st.w2;
  st.avail = a2 & 31u;
  st.hcnt += adv ? 1u : 0u;
}

// LDS byte addresses as plain 32-bit integers, so that offsets can be added without the
// compiler rebuilding a generic pointer.
typedef __attribute__((address_space(3))) const uint16_t lds_cu16;
typedef __attribute__((address_space(3))) const uint64_t lds_cu64;
__device__ __forceinline__ uint32_t lds_addr(const uint16_t* p) {
  return (uint32_t)(uintptr_t)(lds_cu16*)p;
}
__device__ __forceinline__ uint32_t lds_ld16(uint32_t a) { return *(lds_cu16*)(uintptr_t)a; }
__device__ __forceinline__ uint2 lds_ld2x32(uint32_t a) {   // dwords at a and a + 16
  const uint32_t x = *(__attribute__((address_space(3))) const uint32_t*)(uintptr_t)a;
  const uint32_t y = *(__attribute__((address_space(3))) const uint32_t*)(uintptr_t)(a + 16u);
  return make_uint2(x, y);
}
__device__ __forceinline__ uint2 lds_ld64(uint32_t a) {
  const uint64_t v = *(lds_cu64*)(uintptr_t)a;
  return make_uint2((uint32_t)v, (uint32_t)(v >> 32));
}

// Views of a staged table. kS is the distance in bytes between consecutive entries of one
// lane's table: 2 for a table stored contiguously, 128 for the column layout, where entry i of
// the lane in column L of a 64-column block sits at u16 index 64 i + L. In the column layout a
// lane's LDS bank depends on its column only, so a wave's 64 lookups at 64 different entries do
// not collide in the banks (contiguous tables put them in random banks). tb is the byte address
// of the lane's entry 0; cum(i) reads entry i for the rare correction walk after a missed
// candidate, first() gives the first symbol the walk tries; q2f / q_of turn the address of
// the decoded symbol's entry into 2 q (as a float, for the dequantization) or q.
struct ColTab {   // all 256 entries in LDS, column layout
  static constexpr uint32_t kS = 128;
  const uint16_t* tab;   // the lane's column
  uint32_t tb;
  int kqi;               // -((tb >> 7) + 127)
  float kc;              // -(tb / 64 + 254), exact
  __device__ __forceinline__ ColTab(const uint16_t* t)
      : tab(t), tb((uint32_t)(uintptr_t)(__attribute__((address_space(3))) const uint16_t*)t),
        kqi(-(int)((tb >> 7) + 127u)), kc(-((float)tb * 0.015625f + 254.0f)) {}
  __device__ __forceinline__ uint32_t cum(int i) const { return tab[64 * i]; }
  __device__ __forceinline__ int first(int sym, uint32_t, bool down) const {
    return down ? max(sym - 1, 0) : min(sym + 1, CG_NSYM - 1);
  }
  // the entry's address is tb + 128 sym: pa / 64 - tb / 64 - 254 = 2 sym - 254 exactly
  __device__ __forceinline__ float q2f(uint32_t pa) const {
    return __builtin_fmaf((float)pa, 0.015625f, kc);
  }
  __device__ __forceinline__ int q_of(uint32_t pa) const { return (int)(pa >> 7) + kqi; }
};

// Fence registers of a whole table: cum[16 f] << 16 in the high half, and in the low half the
// byte offset 16 kS (f - 1) of block f - 1 from the lane's entry 0, compared against the
// target's fixed-point form ti << 16 | fraction; the fence the search ends on carries the
// block address with it.
// Entries 0 and 16 (cum[0] = 0 and the total) are never compared and stay zero.
template <class Tab>
__device__ __forceinline__ void g10_fences(uint32_t (&fT)[17], const Tab& T) {
  fT[0] = 0u;
  fT[16] = 0u;
#pragma unroll
  for (int f = 1; f < 16; ++f) fT[f] = (T.cum(16 * f) << 16) | (16u * Tab::kS * (f - 1));
}

// A table of which only entries k0 .. k1 are in LDS (entry i at byte address rb + 2 i), the
// rest following closed forms: every frequency below the first one that differs from 1 is 1,
// so cum[i] = i there, and every frequency above the last one that differs from 1 is 1, so
// cum[i] = 65536 - (255 - i) = 65281 + i there. k0 = 16 g0 and k1 = 16 (g1 + 1) bound the
// stored 16-entry blocks g0 .. g1, which extend the blocks holding those two frequencies by one
// block on each side. A target in a flat region jumps straight to its symbol.
struct WinTab {
  static constexpr uint32_t kS = 2;
  uint32_t rb;
  int k0, k1;
  uint32_t tb;   // = rb
  int kq2;       // -(rb + 254)
  __device__ __forceinline__ WinTab(uint32_t r, int a, int b)
      : rb(r), k0(a), k1(b), tb(r), kq2(-(int)(r + 254u)) {}
  __device__ __forceinline__ float q2f(uint32_t pa) const { return (float)(int)(pa + kq2); }
  __device__ __forceinline__ int q_of(uint32_t pa) const { return (int)(pa + kq2) >> 1; }
  __device__ __forceinline__ uint32_t cum(int i) const {
    return i < k0 ? (uint32_t)i
                  : (i > k1 ? 65281u + (uint32_t)i : lds_ld16(rb + 2u * (uint32_t)i));
  }
  __device__ __forceinline__ int first(int sym, uint32_t ti, bool down) const {
    if (ti < (uint32_t)k0) return (int)ti;
    if (ti >= 65281u + (uint32_t)k1) return min((int)(ti - 65281u), CG_NSYM - 1);
    return down ? max(sym - 1, 0) : min(sym + 1, CG_NSYM - 1);
  }
};

// Fences of a window table (blocks g0 .. g1 stored; g1 > g0). The tag of fence f addresses
// block f - 1 clamped to [g0, g1 - 1], so that the search, which reads block f - 1 or f of the
// fence it ends on, stays inside the stored blocks. A tag is clamped only when both blocks lie
// in a flat region (blocks below g0 + 1 and above g1 - 1 hold no frequency other than 1), and a
// target there misses its candidate and is resolved by the walk's jump.
__device__ __forceinline__ void g10_fences_win(uint32_t (&fT)[17], const WinTab& T, int g0,
                                               int g1) {
  fT[0] = 0u;
  fT[16] = 0u;
#pragma unroll
  for (int f = 1; f < 16; ++f) {
    const int blk = min(max(f - 1, g0), g1 - 1);
    fT[f] = (T.cum(16 * f) << 16) | (32u * (uint32_t)blk);
  }
}

// One symbol under the table T whose entry 0 sits (really, or for a window table virtually) at
// LDS byte address T.tb, entries T.kS bytes apart, with tagged fences fT. Returns the byte
// address of the decoded symbol's entry after the interval update and the refill of D.
template <class Tab>
__device__ __forceinline__ uint32_t g10_symbol(G10Lane& st, const uint32_t (&fT)[17],
                                               const Tab& T) {
  constexpr uint32_t kS = Tab::kS;
  const uint32_t tb = T.tb;
  // th = ti << 16 | (16 fraction bits) from one conversion, ti = th >> 16 the target. The scale
  // is 2^32 less 5 ulps (5 * 2^8): with D <= rm1, the reciprocal within 1 ulp and two roundings,
  // te stays below 2^32, so ti <= 65535 needs no clamp. The staged entries 255..259 repeat
  // cum[254], so a target at or above cum[254] (the top symbol, whose upper bound, the total,
  // does not fit 16 bits) selects candidate 255, of empty width, and the walk resolves it with
  // the exact bound. The scale's shortfall of 3e-7 moves ti down by at most 0.02. The entries below
  // compare against ti as the high half of th (SDWA word selects, no shift); a tagged fence
  // (cum << 16 | tag) is <= th iff cum < ti, or cum == ti and tag <= the fraction (a tag is at
  // most 448, so a target exactly on a fence goes to the block below at most once in 146, and
  // the walk takes the one step up).
  const float te = (float)st.D * (4294966016.0f * __builtin_amdgcn_rcpf((float)st.rm1));
  const uint32_t th = (uint32_t)te;
  const uint32_t ti = th >> 16;
  // binary search over the fences by selects (four compare / select steps)
  const bool c3 = fT[8] <= th;
  const uint32_t p4 = c3 ? fT[12] : fT[4];
  const uint32_t p2a = c3 ? fT[10] : fT[2], p2b = c3 ? fT[14] : fT[6];
  const uint32_t p1a = c3 ? fT[9] : fT[1], p1b = c3 ? fT[11] : fT[3];
  const uint32_t p1c = c3 ? fT[13] : fT[5], p1d = c3 ? fT[15] : fT[7];
  const bool c2 = p4 <= th;
  const uint32_t p2 = c2 ? p2b : p2a;
  const uint32_t p1e = c2 ? p1c : p1a, p1f = c2 ? p1d : p1b;
  const bool c1 = p2 <= th;
  const uint32_t p1 = c1 ? p1f : p1e;
  const bool c0 = p1 <= th;
  // block f = (index of p1) - 1 + c0 starts at byte 16 kS f
  uint32_t qa;
  asm("v_add_u32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:WORD_0 "
      "src1_sel:DWORD" : "=v"(qa) : "v"(p1), "v"(c0 ? tb + 16u * kS : tb));
  // 4-ary level: cum[16 f + 4 m], m = 1..3
  // two steps over the three sorted entries: cum[16 f + 8], then cum[16 f + 12] or cum[16 f + 4]
  bool b8, b4;
  if constexpr (kS == 2) {
    // (cum[16 f + 4] and cum[16 f + 12] in the low halves of one two-dword read)
    const uint2 c412 = lds_ld2x32(qa + 8u);
    const uint32_t c8 = lds_ld16(qa + 16u);
    b8 = c8 <= ti;
    b4 = ((b8 ? c412.y : c412.x) & 0xFFFFu) <= ti;
  } else {
    const uint32_t c4 = lds_ld16(qa + 4u * kS), c8 = lds_ld16(qa + 8u * kS),
                   c12 = lds_ld16(qa + 12u * kS);
    b8 = c8 <= ti;
    b4 = (b8 ? c12 : c4) <= ti;
  }
  const uint32_t qb = qa + (b8 ? 8u * kS : 0u) + (b4 ? 4u * kS : 0u);
  // leaf: cum[i .. i+3], i = (qb - tb) / kS; the candidate i + c (c = the number of
  // cum[i+1 .. i+3] <= ti, two steps as above) and the bounds cum[i + c], cum[i + c + 1] are
  // read from its address (contiguous tables: x = cum[i] | cum[i+1] << 16 and y = cum[i+2] |
  // cum[i+3] << 16 from one 8-byte read)
  bool b2, b1;
  if constexpr (kS == 2) {
    const uint2 xy = lds_ld64(qb);
    b2 = (xy.y & 0xFFFFu) <= ti;
    b1 = ((b2 ? xy.y : xy.x) >> 16) <= ti;
  } else {
    const uint32_t x1 = lds_ld16(qb + kS), x2 = lds_ld16(qb + 2u * kS),
                   x3 = lds_ld16(qb + 3u * kS);
    b2 = x2 <= ti;
    b1 = (b2 ? x3 : x1) <= ti;
  }
  // one three-input add (the compiler would merge the two disjoint constants with an OR first)
  uint32_t pa;
  asm("v_add3_u32 %0, %1, %2, %3" : "=v"(pa) : "v"(qb), "v"(b2 ? 2u * kS : 0u), "v"(b1 ? kS : 0u));
  uint32_t clo = lds_ld16(pa);
  const uint32_t chr = lds_ld16(pa + kS);
  // (the candidate is never the top symbol)
  uint32_t chi = chr;
  const uint32_t D = st.D, rm1 = st.rm1;
  // offsets of the candidate's interval from low: [lo_off, hoff) (hoff mod 2^32). The candidate
  // is the symbol iff D - lo_off < hoff - lo_off (unsigned): below lo_off the difference wraps
  // past the interval's size, which is below 2^32 - lo_off.
  uint32_t lo_off = scaled_off(rm1, clo);
  uint32_t hoff = scaled_off(rm1, chi);
  uint32_t d = D - lo_off;
  uint32_t rsz = hoff - lo_off;
  if (d >= rsz) {
    int sym = (int)((pa - tb) / kS);
    int nxt = T.first(sym, ti, D < lo_off);
    for (int guard = 0; guard < CG_NSYM; ++guard) {
      sym = nxt;
      const int s1 = min(sym + 1, CG_NSYM - 1);
      clo = T.cum(sym);
      chi = T.cum(s1);
      chi = sym + 1 >= CG_NSYM ? CG_TOTAL : chi;
      lo_off = scaled_off(rm1, clo);
      hoff = scaled_off(rm1, chi);
      d = D - lo_off;
      rsz = hoff - lo_off;
      if (d < rsz) break;
      nxt = (D < lo_off) ? max(sym - 1, 0) : min(sym + 1, CG_NSYM - 1);
    }
    pa = tb + kS * (uint32_t)sym;
  }
  g10_advance(st, lo_off, hoff, d, rsz);
  return pa;
}

// One delta token: its symbol under the delta table, dequantized against the group's anchor
// into row r of the wave's staging buffer.
// w2 = w / 2 (exact), so 2 q times w2 is the same real number as q times w.
template <class Tab>
__device__ __forceinline__ void g10_delta(G10Lane& st, const uint32_t (&fD)[17], const Tab& T,
                                          float w2, uint16_t* obuf, int r, int lane) {
  const uint32_t pa = g10_symbol(st, fD, T);
  obuf[r * 64 + lane] = cg_f2h(st.a + T.q2f(pa) * w2);
}

// Store rows first .. rows-1 of the staged group: lane L stores 16 bytes (8 channels) of row
// first + L / 8, then lanes 0..15 rows first + 8 and first + 9.
__device__ __forceinline__ void g10_flush(const uint16_t* obuf, uint16_t* row, int64_t rstride,
                                          int first, int rows, int lane, int cbase, int C) {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
  for (int part = 0; part < 2; ++part) {
    const int rr = first + part * 8 + (lane >> 3), cc = (lane & 7) * 8;
    if (rr < rows && cbase + cc < C) {
      const uint4 vals = *reinterpret_cast<const uint4*>(obuf + rr * 64 + cc);
      uint16_t* dst = row + rr * rstride + cc;
      if (cbase + cc + 8 <= C && (reinterpret_cast<uintptr_t>(dst) & 15) == 0) {
        store_row16(dst, vals);
      } else {
        const uint16_t hv[8] = {(uint16_t)(vals.x & 0xFFFFu), (uint16_t)(vals.x >> 16),
                                (uint16_t)(vals.y & 0xFFFFu), (uint16_t)(vals.y >> 16),
                                (uint16_t)(vals.z & 0xFFFFu), (uint16_t)(vals.z >> 16),
                                (uint16_t)(vals.w & 0xFFFFu), (uint16_t)(vals.w >> 16)};
        for (int e = 0; e < 8; ++e)
          if (cbase + cc + e < C) dst[e] = hv[e];
      }
    }
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Rows 0..9 of a whole group of a full, 16-byte aligned 64-channel block: two unconditional
// 16-byte stores per lane (rows 0..7, then rows 8 and 9, which lanes 16..63 store again with the
// same bytes as lanes 0..15). With the same two stores on every path, the wait at the next
// epoch covers only the words it needs, not the stores just issued.
__device__ __forceinline__ void g10_flush_full(const uint16_t* obuf, uint16_t* row,
                                               int64_t rstride, int lane) {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  const int cc = (lane & 7) * 8;
  const int r0 = lane >> 3, r1 = 8 + ((lane >> 3) & 1);
  const uint4 v0 = *reinterpret_cast<const uint4*>(obuf + r0 * 64 + cc);
  const uint4 v1 = *reinterpret_cast<const uint4*>(obuf + r1 * 64 + cc);
  store_row16(row + r0 * rstride + cc, v0);
  store_row16(row + r1 * rstride + cc, v1);
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// kCompact: the delta tables are staged as windows (see WinTab): every unit has a region of
// ustride u16 (at least one whole table set), which holds its anchor tables in the anchor phase
// and then the windows of its delta tables, packed; sets that do not fit together are staged in
// rounds, one after the other. Otherwise the region holds min(nw, levels) whole sets.
template <bool kCompact>
__global__ __launch_bounds__(1024) void decode_g10_kernel(
    KParams P, const uint32_t* __restrict__ words, const uint64_t* __restrict__ offsets,
    const float* __restrict__ scales, const uint8_t* __restrict__ chunk_level,
    const uint16_t* __restrict__ cdfA, const uint16_t* __restrict__ cdfD, int c_begin,
    int c_end, int nw, int nu, int ustride, uint16_t* __restrict__ out) {
  extern __shared__ __attribute__((aligned(16))) uint16_t smem[];
  __shared__ int s_wlv[kMaxWaves];               // bit of the level of each wave's pair (0: none)
  __shared__ uint8_t s_set_of_level[kMaxUnits][CG_MAX_LEVELS];
  __shared__ uint8_t s_level_of_set[kMaxUnits][CG_MAX_LEVELS];
  __shared__ uint8_t s_nsets[kMaxUnits];
  __shared__ uint8_t s_round[kMaxUnits][CG_MAX_LEVELS];   // staging round of each set (compact)
  __shared__ uint8_t s_nrounds[kMaxUnits];
  __shared__ uint8_t s_simd[kMaxWaves];             // SIMD of each wave
  __shared__ int s_left[kMaxWaves];             // symbols each wave has left in this phase
  const int msets = nw < P.NLV ? nw : P.NLV;          // table sets a unit may need
  uint16_t* obuf_all = smem;                          // [nu * nw][kG10][64] rows per wave
  uint16_t* tabs = obuf_all + nu * nw * kG10 * 64;    // [nu][ustride]
  // window descriptors of the delta tables [nu][msets][64] (compact): size / offset, g0, g1
  uint32_t* desc = reinterpret_cast<uint32_t*>(tabs + (size_t)nu * ustride);

  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int nwaves = blockDim.x >> 6;
  const int u = wave % nu, j = wave / nu;             // unit and pair slot of this wave
  const int ncr = c_end - c_begin;
  const int n_pairs = P.B * ncr;
  const int n_groups = (n_pairs + nw - 1) / nw;
  const int n_units = P.L * 2 * P.nblk;
  int ublk, grp;
  cg_xcd_map((n_units + nu - 1) / nu, n_groups, ublk, grp);
  if (ublk * nu >= n_units) return;   // past the last unit block (uniform over the workgroup)
  const int unit = ublk * nu + u;
  const int cb = unit % P.nblk;
  const int k = (unit / P.nblk) & 1, l = (unit / P.nblk) >> 1;

  // Stage whole tables into LDS in the column layout (entry i of channel cb * 64 + L at u16
  // 64 i + L of its set): the anchor tables of every unit (set 0), or the delta tables of the
  // levels each unit's pairs use. The nw waves of a unit stage that unit's tables; a load
  // instruction covers the 16 columns of one residue mod 4, four neighbouring lanes taking four
  // consecutive 16-byte pieces (entries 8 p .. 8 p + 7) of one table, so it touches 16 half
  // cache lines and its column stores put four lanes on a bank (with one lane per table the
  // 64 cache lines of every load made the staging slower, with eight the stores conflicted
  // eight ways). Instruction z of a set (32 of them) takes the columns c with c mod 4 = z mod 4
  // and pieces 4 ((z mod 32) / 4) + (0 .. 3); wave slot j takes instructions j, j + nw, ... of
  // the unit's sets (set and instruction uniform). stage_issue
  // loads batch i0 .. i0 + N - 1 into registers, stage_put writes them (eight 2-byte stores a
  // piece); the first anchor batch
  // goes out before any other load of the kernel, the first delta batch before the barrier
  // that ends the anchor phase. Entries 255..259 repeat cum[254] (candidates past the top
  // symbol have empty intervals, and the walk resolves the top symbol).
  const int half = lane >> 5, piece = lane & 31;
  const bool unit_ok = unit < n_units;
  const int64_t lk_row = (int64_t)(l * 2 + k) * P.C + cb * 64;   // table row of channel cb*64
  const int pcol = ((lane >> 2) << 2);   // the first column of the lane's group of four
  // levels used by this wave's unit, a bit per level (set after the first barrier); the set of
  // a level is its rank among them
  uint32_t umask = 0u;
  auto level_of_set = [&](int st) __attribute__((always_inline)) {
    uint32_t m = umask;
    for (int i = 0; i < st; ++i) m &= m - 1u;
    return (int)__builtin_ctz(m | (1u << 31));
  };
  auto stage_issue = [&](bool anchors, int i0, auto& v, auto& dsto)
                         __attribute__((always_inline)) {
    constexpr int N = sizeof(dsto) / sizeof(dsto[0]);
    const int sets = anchors ? 1 : __builtin_popcount(umask);
    const uint16_t* srcbase = anchors ? cdfA : cdfD;
#pragma unroll
    for (int i = 0; i < N; ++i) {
      // unconditional loads (a piece that is not staged reads the first table instead), so
      // that all of them are in flight before the first store waits
      const int z = uni(j + nw * (i0 + i));      // load instruction of the unit's sets
      const int st = uni(z >> 5);
      const int col = pcol + (z & 3), pc = ((z & 31) >> 2) * 4 + (lane & 3);
      const int lset = anchors ? 0 : level_of_set(st);
      const bool ok = (st < sets) & unit_ok & (cb * 64 + col < P.C);
      const int64_t trow = lk_row + col + (anchors ? 0 : (int64_t)lset * P.L * 2 * P.C);
      v[i] = reinterpret_cast<const uint4*>(srcbase + (ok ? trow : 0) * 256)[pc];
      dsto[i] = ok ? u * ustride + st * kColSet + pc * 8 * 64 + col : -1;
    }
  };
  auto stage_put = [&](const auto& v, const auto& dsto) __attribute__((always_inline)) {
    constexpr int N = sizeof(dsto) / sizeof(dsto[0]);
#pragma unroll
    for (int i = 0; i < N; ++i) {
      if (dsto[i] < 0) continue;
      uint16_t* dst = tabs + dsto[i];
      const uint4 x = v[i];
      const bool last = ((dsto[i] - u * ustride) % kColSet) >= 31 * 8 * 64;   // entries 248..
      const uint32_t top = x.w & 0xFFFFu;   // cum[254] in piece 31
      dst[0 * 64] = (uint16_t)x.x;
      dst[1 * 64] = (uint16_t)(x.x >> 16);
      dst[2 * 64] = (uint16_t)x.y;
      dst[3 * 64] = (uint16_t)(x.y >> 16);
      dst[4 * 64] = (uint16_t)x.z;
      dst[5 * 64] = (uint16_t)(x.z >> 16);
      dst[6 * 64] = (uint16_t)x.w;
      dst[7 * 64] = (uint16_t)(last ? top : x.w >> 16);
      if (last) {
#pragma unroll
        for (int e = 8; e < 12; ++e) dst[e * 64] = (uint16_t)top;   // entries 256..259
      }
    }
  };
  // the batches from i0 on
  auto stage_rest = [&](bool anchors, int i0) __attribute__((always_inline)) {
    const int pairs = (anchors ? 1 : __builtin_popcount(umask)) * 32;
    for (int i = i0; j + nw * i < pairs; i += kStageBatch) {
      uint4 v[kStageBatch];
      int dsto[kStageBatch];
      stage_issue(anchors, i, v, dsto);
      stage_put(v, dsto);
    }
  };

  uint4 anc_v[kAnchorPre];
  int anc_d[kAnchorPre];
  stage_issue(true, 0, anc_v, anc_d);
  // a call without payload decodes nothing (uniform over the grid; checked after the staging)
  const uint64_t total = offsets[P.S];

  const int pair = uni(grp * nw + j);
  const bool active = unit_ok && pair < n_pairs;
  // pairs chunk-major: the waves of a workgroup decode the same chunk of consecutive contexts,
  // so they have the same token count and finish together
  const int b = uni(active ? pair % P.B : 0);
  const int c = uni(active ? c_begin + pair / P.B : 0);
  const int lv = P.NLV == 1 ? 0
                            : uni(active ? min((int)chunk_level[(int64_t)b * P.NC + c], P.NLV - 1)
                                         : 0);
  const int tok0 = c * P.CL;
  const int n = uni(active ? min(P.CL, P.T - tok0) : 0);
  const int na = (n + kG10 - 1) / kG10;               // anchors (coded first)

  const int simd = (int)((__builtin_amdgcn_s_getreg((31 << 11) | 4) >> 4) & 3u);   // HW_ID
  if (lane == 0) {
    s_simd[wave] = simd;
    lds_put(&s_left[wave], na);
    lds_put(&s_wlv[wave], active ? (1 << lv) : 0);
  }
  stage_put(anc_v, anc_d);
  stage_rest(true, kAnchorPre);
  __syncthreads();   // anchor tables, SIMDs, levels and counts of every wave
  for (int jj = 0; jj < nw; ++jj) umask |= (uint32_t)uni(lds_get(&s_wlv[u + jj * nu]));
  // the (up to three) other waves of this workgroup on this wave's SIMD
  int p0 = wave, p1 = wave, p2 = wave, np = 0;
  for (int w2 = 0; w2 < nwaves; ++w2) {
    if (w2 == wave || uni(s_simd[w2]) != simd) continue;
    if (np == 0) p0 = w2; else if (np == 1) p1 = w2; else if (np == 2) p2 = w2;
    ++np;
  }
  // issue priority by what is left among the waves of this SIMD (most left first), so that
  // they finish a phase together instead of the oldest first
  auto set_priority = [&](int left) __attribute__((always_inline)) {
    const int l0 = uni(lds_get(&s_left[p0])), l1 = uni(lds_get(&s_left[p1])),
              l2 = uni(lds_get(&s_left[p2]));
    lds_put(&s_left[wave], left);
    const int rank = (p0 != wave && (l0 > left || (l0 == left && p0 < wave))) +
                     (p1 != wave && (l1 > left || (l1 == left && p1 < wave))) +
                     (p2 != wave && (l2 > left || (l2 == left && p2 < wave)));
    if (rank == 0) __builtin_amdgcn_s_setprio(3);
    else if (rank == 1) __builtin_amdgcn_s_setprio(2);
    else if (rank == 2) __builtin_amdgcn_s_setprio(1);
    else __builtin_amdgcn_s_setprio(0);
  };
  // the windowed kernel's passes read the level sets of every unit of the workgroup
  if constexpr (kCompact) {
    if (threadIdx.x < nu) {
      const int uu = threadIdx.x;
      uint32_t mk = 0u;
      for (int jj = 0; jj < nw; ++jj) mk |= (uint32_t)lds_get(&s_wlv[uu + jj * nu]);
      int m = 0;
      for (int v = 0; v < P.NLV; ++v)
        if ((mk >> v) & 1u) { s_set_of_level[uu][v] = m; s_level_of_set[uu][m] = v; ++m; }
      s_nsets[uu] = m;
    }
    __syncthreads();
  }

  // Compact staging of the delta tables. Pass 1 (window): each table's first and last
  // frequency other than 1 (i0, i1), from the 8 entries a lane holds and the next lane's first;
  // blocks g0 = max(i0 / 16 - 1, 0) .. g1 = min(i1 / 16 + 1, 15) are kept, entries 16 g0 ..
  // 16 (g1 + 1) + 3 (8-byte multiple). Pass 2 (layout, one wave per unit): offsets of the
  // windows, set after set, and a new round whenever a set does not fit the region any more.
  // Pass 3 (per round): the windows of the round's sets are written, with entries 255..259
  // repeating cum[254] as in the full tables.
  auto window_pass = [&]() __attribute__((always_inline)) {
    const int n_rows = nu * msets * 64;
    for (int base = wave; base * 2 < n_rows; base += nwaves * kStageBatch) {
      uint4 v[kStageBatch];
      int rows[kStageBatch];
#pragma unroll
      for (int i = 0; i < kStageBatch; ++i) {
        const int rr = (base + i * nwaves) * 2 + half;
        const int t = rr & 63, st = (rr >> 6) % msets, uu = min((rr >> 6) / msets, nu - 1);
        const int unit2 = ublk * nu + uu;
        const int ch = (unit2 % P.nblk) * 64 + t;
        const int lset = s_level_of_set[uu][st];
        const bool ok = (rr < n_rows) & (unit2 < n_units) & (st < (int)s_nsets[uu]) & (ch < P.C);
        const int64_t trow = ((int64_t)lset * P.L * 2 + unit2 / P.nblk) * P.C + ch;
        v[i] = reinterpret_cast<const uint4*>(cdfD + (ok ? trow : 0) * 256)[piece];
        rows[i] = ok ? rr : -1;
      }
#pragma unroll
      for (int i = 0; i < kStageBatch; ++i) {
        int lo, hi;
        cg_table_window(v[i], piece, lo, hi);
        if (rows[i] >= 0 && piece == 0) desc[rows[i]] = cg_window_desc(lo, hi);
      }
    }
  };
  auto layout_pass = [&]() __attribute__((always_inline)) {
    if (wave >= nu) return;   // one wave per unit (uniform)
    const int uu = wave;
    const int unit2 = ublk * nu + uu;
    const int pool = 2 * ustride;
    const bool chok = unit2 < n_units && (unit2 % P.nblk) * 64 + lane < P.C;
    int round = 0, acc = 0;
    for (int st = 0; st < msets; ++st) {
      const int idx = (uu * msets + st) * 64 + lane;
      const bool ok = chok && st < (int)s_nsets[uu];
      const uint32_t d = ok ? desc[idx] : 0u;
      const uint32_t sz = d >> 8;
      const uint32_t incl = cg_wave_incl_scan(sz);
      const int tot = uni((int)__shfl(incl, 63, 64));
      if (acc > 0 && acc + tot > pool) { ++round; acc = 0; }
      if (ok) desc[idx] = (uint32_t)(acc + (int)(incl - sz)) | ((d & 0xFFu) << 20);
      if (lane == 0) s_round[uu][st] = (uint8_t)round;
      acc += tot;
    }
    if (lane == 0) s_nrounds[uu] = (uint8_t)(round + 1);
  };
  auto stage_round = [&](int rd) __attribute__((always_inline)) {
    const int n_rows = nu * msets * 64;
    for (int base = wave; base * 2 < n_rows; base += nwaves * kStageBatch) {
      uint4 v[kStageBatch];
      int dsto[kStageBatch], k0s[kStageBatch], kends[kStageBatch];
#pragma unroll
      for (int i = 0; i < kStageBatch; ++i) {
        const int rr = (base + i * nwaves) * 2 + half;
        const int t = rr & 63, st = (rr >> 6) % msets, uu = min((rr >> 6) / msets, nu - 1);
        const int unit2 = ublk * nu + uu;
        const int ch = (unit2 % P.nblk) * 64 + t;
        const int lset = s_level_of_set[uu][st];
        const bool ok = (rr < n_rows) & (unit2 < n_units) & (st < (int)s_nsets[uu]) &
                        (ch < P.C) && (int)s_round[uu][st] == rd;
        const int64_t trow = ((int64_t)lset * P.L * 2 + unit2 / P.nblk) * P.C + ch;
        v[i] = reinterpret_cast<const uint4*>(cdfD + (ok ? trow : 0) * 256)[piece];
        const uint32_t d = ok ? desc[min(rr, n_rows - 1)] : 0u;
        const int g0 = (int)((d >> 20) & 15u), g1 = (int)((d >> 24) & 15u);
        dsto[i] = ok ? uu * ustride + (int)((d & 0xFFFFFu) >> 1) : -1;
        k0s[i] = 16 * g0;
        kends[i] = 16 * (g1 + 1) + 4;
      }
#pragma unroll
      for (int i = 0; i < kStageBatch; ++i) {
        if (dsto[i] < 0) continue;
        uint16_t* dst = tabs + dsto[i] - k0s[i];   // entry k of the table at dst[k]
        const int e = 8 * piece;
        uint4 x = v[i];
        if (piece == 31) x.w = (x.w & 0xFFFFu) * 0x10001u;   // entry 255 = cum[254]
        if (e >= k0s[i] && e < kends[i])
          *reinterpret_cast<uint2*>(dst + e) = make_uint2(x.x, x.y);
        if (e + 4 >= k0s[i] && e + 4 < kends[i])
          *reinterpret_cast<uint2*>(dst + e + 4) = make_uint2(x.z, x.w);
        if (piece == 31 && kends[i] > 256)   // entries 256..259 = cum[254]
          *reinterpret_cast<uint2*>(dst + 256) = make_uint2(x.w, x.w);
      }
    }
  };

  if constexpr (kCompact) {
    window_pass();
    __syncthreads();
  }
  if (total == 0) return;
  if constexpr (kCompact) {
    layout_pass();
    __syncthreads();
  }

  const int ch = cb * 64 + lane;
  const bool valid = ch < P.C;
  // Lanes past the last channel (only when C is not a multiple of 64) decode a copy of the
  // block's first channel, so the whole wave runs the same code; they store into that
  // channel's column the values its own lane stores, and their staged rows are never stored.
  const int lsrc = valid ? lane : 0;
  const int chv = cb * 64 + lsrc;
  const int64_t rstride = P.C;
  uint16_t* row0 = out + cg_elem(P, b, l, k, tok0, cb * 64);   // token tok0, channel cb * 64
  const uint16_t* tab0 = tabs + u * ustride + lsrc;   // anchor table of the lane (column)
  G10Lane st;
  const uint32_t* sbase = words;
  uint32_t cap = 0;
  float s = 1.0f, w = 1.0f;

  // ---- anchor phase: the chunk's anchors, first in the stream ----------------------------
  if (active) {
    const int64_t bclk = (((int64_t)b * P.NC + c) * P.L + l) * 2 + k;
    const int64_t sidx = cg_stream(P, bclk, chv);
    s = scales[sidx];
    w = P.layer_bin[l] * P.level_mult[lv] * s;
    uint32_t fA[17];   // tagged fences of the anchor table
    const ColTab TA(tab0);
    g10_fences(fA, TA);
    // bitstream reader: the code value, w1..w3 and the four requested words t0..t3 are the
    // stream's first 8 words; every read stays below offsets[S] + 4 (the requests are clamped
    // to it), inside the readable tail
    const uint64_t o0 = offsets[sidx];
    const uint64_t ob = o0 < total ? o0 : total;
    sbase = words + ob;
    cap = (uint32_t)((total - ob) < 0xFFFFFFF0ull ? (total - ob) : 0xFFFFFFF0ull);
    st.D = sbase[0];
    st.w0 = 0u;   // used up: the stream continues with w1
    st.w1 = sbase[1];
    st.w2 = sbase[2];
    st.w3 = sbase[3];
    st.avail = 0;
    st.hcnt = 0;
    st.widx = 4;
    const uint32_t* tq0 = sbase + (4u < cap ? 4u : cap);
    st.t0 = tq0[0];
    st.t1 = tq0[1];
    st.t2 = tq0[2];
    st.t3 = tq0[3];
    settle(st.D); settle(st.w0); settle(st.w1); settle(st.w2); settle(st.w3);
    st.low = 0u;
    st.lsh = 0u;
    st.rm1 = 0xFFFFFFFFu;
    st.a = 0.0f;

    // kAnchorRun anchors per epoch. The quantized value q of each anchor goes into the anchor's
    // own row, where the delta phase reads it back and its flush then writes the anchor's fp16
    // value. A run's q values are stored at the next epoch, between the wait for the words
    // requested one epoch earlier and the next request, so that no wait for words also waits
    // for stores just issued.
    int qrun[kAnchorRun];
    // row of anchor gs, advanced by whole runs (uniform; the rows of a run at fixed offsets)
    const int64_t astep = (int64_t)kG10 * rstride;
    uint16_t* qrow = row0;
    auto store_run = [&](int gs) __attribute__((always_inline)) {
#pragma unroll
      for (int r = 0; r < kAnchorRun; ++r)
        if (gs + r < na) (qrow + r * astep)[lsrc] = (uint16_t)qrun[r];
    };
    for (int g0 = 0; g0 < na; g0 += kAnchorRun) {
      g10_epoch_take(st);
      if (g0 > 0) {
        store_run(g0 - kAnchorRun);
        qrow += kAnchorRun * astep;
      }
      g10_epoch_request(st, sbase, cap);
#pragma unroll
      for (int r = 0; r < kAnchorRun; ++r)
        if (g0 + r < na) qrun[r] = TA.q_of(g10_symbol(st, fA, TA));
      // every other run (the ranking reads three LDS words and takes a dozen scalar
      // instructions)
      if ((g0 / kAnchorRun) & 1) set_priority(max(na - g0 - kAnchorRun, 0));
    }
    const int glast = (na - 1) / kAnchorRun * kAnchorRun;   // first anchor of the last run
    store_run(glast);   // qrow is the row of anchor glast
    // a last group without deltas (n = 1 mod 10) has no flush: its anchor row takes the value
    if ((na - 1) * kG10 + 1 >= n) {
      const int rl = na - 1 - glast;
      int ql = qrun[0];
#pragma unroll
      for (int r = 1; r < kAnchorRun; ++r) ql = rl == r ? qrun[r] : ql;
      (row0 + (int64_t)(na - 1) * kG10 * rstride)[lsrc] = cg_f2h((float)ql * s);
    }
  }

  auto delta_groups = [&](const auto& T, const uint32_t (&fD)[17])
                          __attribute__((always_inline)) {
  set_priority(n - na);
  const float w2 = w * 0.5f;

  uint16_t* obuf = obuf_all + wave * kG10 * 64;
  const int cbase = cb * 64;
  const int ngr = n / kG10;
  const int gmax = (n - 2) / kG10;                    // last group with a delta
  // the anchor's q of group g (kept in the anchor's row until the group's flush)
  auto q_of = [&](int g) __attribute__((always_inline)) {
    const uint16_t* rq = row0 + (int64_t)min(g, gmax) * kG10 * rstride;   // uniform
    return (uint32_t)rq[lsrc];
  };
  // the anchor value of the next group, carried as a float so that the loop head uses no
  // register a load may still be filling
  float anext = (float)(int)(int16_t)q_of(0) * s;
  uint16_t* row = row0;
  // whole groups: the loop is written out twice, for full aligned blocks and for the rest
  const bool full = cbase + 64 <= P.C && (P.C & 7) == 0 && (reinterpret_cast<uintptr_t>(out) & 15) == 0;
  auto groups = [&](auto kFull) __attribute__((always_inline)) {
  for (int gi = 0; gi < ngr; ++gi) {
    st.a = anext;
    obuf[lane] = cg_f2h(anext);   // row 0: the anchor's value
    g10_epoch(st, sbase, cap);
    g10_delta(st, fD, T, w2, obuf, 1, lane);
    g10_delta(st, fD, T, w2, obuf, 2, lane);
    g10_delta(st, fD, T, w2, obuf, 3, lane);
    g10_delta(st, fD, T, w2, obuf, 4, lane);
    g10_delta(st, fD, T, w2, obuf, 5, lane);
    g10_epoch(st, sbase, cap);
    const uint32_t qnext = q_of(gi + 1);   // requested a group ahead
    g10_delta(st, fD, T, w2, obuf, 6, lane);
    g10_delta(st, fD, T, w2, obuf, 7, lane);
    g10_delta(st, fD, T, w2, obuf, 8, lane);
    g10_delta(st, fD, T, w2, obuf, 9, lane);
    if constexpr (decltype(kFull)::value) g10_flush_full(obuf, row, rstride, lane);
    else g10_flush(obuf, row, rstride, 0, kG10, lane, cbase, P.C);
    row += kG10 * rstride;
    anext = (float)(int)(int16_t)qnext * s;
    // every other group: the ranking reads three LDS words and takes a dozen scalar
    // instructions; updating after every group measured 1-3 % slower
    if (gi & 1) set_priority((ngr - gi - 1) * (kG10 - 1));
  }
  };
  if (full) groups(std::integral_constant<bool, true>{});
  else groups(std::integral_constant<bool, false>{});
  const int rem = n - ngr * kG10;   // last, partial group (uniform)
  if (rem > 1) {
    st.a = anext;
    obuf[lane] = cg_f2h(anext);
    g10_epoch(st, sbase, cap);
    for (int r = 1; r < rem; ++r) {
      if (r == 6) g10_epoch(st, sbase, cap);
      g10_delta(st, fD, T, w2, obuf, r, lane);
    }
    g10_flush(obuf, row, rstride, 0, rem, lane, cbase, P.C);
  }
  };

  // ---- delta phase: the delta tables replace the anchor tables --------------------------
  // (in rounds when compact windows of all sets do not fit a unit's region at once; every wave
  // takes part in every round's staging and barriers, and decodes in its set's round). Whole
  // tables: the first kDeltaPre loads per lane go out before the barrier.
  uint4 dpre_v[kCompact ? 1 : kDeltaPre];
  int dpre_d[kCompact ? 1 : kDeltaPre];
  if constexpr (!kCompact) stage_issue(false, 0, dpre_v, dpre_d);
  __syncthreads();
  int nrounds = 1;
  if constexpr (kCompact) {
    for (int uu = 0; uu < nu; ++uu) nrounds = max(nrounds, (int)s_nrounds[uu]);
    nrounds = uni(nrounds);
  }
  // this wave's round (past the last one: nothing to decode); the rounds before and after it
  // only stage and wait, so that the decoding runs outside any loop
  const int set = !active ? 0
                  : kCompact ? (int)s_set_of_level[u][lv]
                             : __builtin_popcount(umask & ((1u << lv) - 1u));
  const int myr = uni(!active || n < 2 ? nrounds : (kCompact ? (int)s_round[u][set] : 0));
  auto round_stage = [&](int rd) __attribute__((always_inline)) {
    if (rd > 0) __syncthreads();   // the previous round's readers are done
    if constexpr (kCompact) {
      stage_round(rd);
    } else {
      stage_put(dpre_v, dpre_d);
      stage_rest(false, kDeltaPre);
    }
    __syncthreads();
  };
  for (int rd = 0; rd < myr; ++rd) round_stage(rd);
  if (myr >= nrounds) return;
  round_stage(myr);
  {
    if constexpr (kCompact) {
      const uint32_t d = desc[(u * msets + set) * 64 + lsrc];
      const int g0 = (int)((d >> 20) & 15u), g1 = (int)((d >> 24) & 15u);
      const WinTab T(lds_addr(tabs + u * ustride) + (d & 0xFFFFFu) - 32u * (uint32_t)g0, 16 * g0,
                     16 * (g1 + 1));
      uint32_t fD[17];
      g10_fences_win(fD, T, g0, g1);
      delta_groups(T, fD);
    } else {
      const ColTab T(tabs + u * ustride + set * kColSet + lsrc);
      uint32_t fD[17];
      g10_fences(fD, T);
      delta_groups(T, fD);
    }
  }
  for (int rd = myr + 1; rd < nrounds; ++rd) round_stage(rd);
}

// ---- token-parallel layout (Sec. 6: the paper's decoder runs one thread per token) -----------
// A wave decodes 64 consecutive token streams of one (context, chunk, layer, K/V), a lane per
// token, symbol by symbol over the channels. Every lane codes channel ch under the tables of
// (layer, K/V, ch), so per channel the wave stages that channel's anchor and delta tables in LDS
// (512 bytes each, 16 bytes per lane; the next channel's are loaded while the current one is
// decoded) and searches them with the channel layout's delta search from the top: three 4-ary
// levels and the leaf. There are no per-table fences in registers and no table reuse across
// symbols: that is the price of this layout. Symbols collect in a lane-private LDS row and go
// to the symbol array [B][L][2][T][C] every 64 channels; tok_dequant_kernel then reconstructs
// the channel streams exactly as the channel layout does.
constexpr int kTokTab = 264;   // u16 per staged table: 256 entries + 8 sentinels (528 bytes)
constexpr int kTokRow = 68;    // bytes per lane's symbol row (64 + 4: rows start in other banks)

// One symbol of a token stream under the staged table `tab` (sentinels from entry 255 on).
__device__ __forceinline__ uint32_t tok_symbol(G10Lane& st, const uint16_t* tab) {
  const float te = (float)st.D * (65536.0f * __builtin_amdgcn_rcpf((float)st.rm1));
  const uint32_t ti = min((uint32_t)te, 65534u);
  const uint32_t kneg = ~ti;
  const uint16_t* q = tab;
  q += 64 * ((((uint32_t)q[64] + kneg) >> 31) + (((uint32_t)q[128] + kneg) >> 31) +
             (((uint32_t)q[192] + kneg) >> 31));
  q += 16 * ((((uint32_t)q[16] + kneg) >> 31) + (((uint32_t)q[32] + kneg) >> 31) +
             (((uint32_t)q[48] + kneg) >> 31));
  q += 4 * ((((uint32_t)q[4] + kneg) >> 31) + (((uint32_t)q[8] + kneg) >> 31) +
            (((uint32_t)q[12] + kneg) >> 31));
  uint32_t pr;
  const uint32_t cc = delta_leaf(q, ti, pr);
  int sym = (int)((((uint32_t)(uintptr_t)q - (uint32_t)(uintptr_t)tab) >> 1) + cc);
  uint32_t clo = pr & 0xFFFFu;
  uint32_t chi = sym == CG_NSYM - 1 ? CG_TOTAL : pr >> 16;
  const uint32_t D = st.D, rm1 = st.rm1;
  uint32_t lo_off = scaled_off(rm1, clo);
  uint32_t hoff = scaled_off(rm1, chi);
  uint32_t d = D - lo_off;
  uint32_t rsz = hoff - lo_off;
  if (d >= rsz) {
    for (int guard = 0; guard < CG_NSYM; ++guard) {
      sym = (D < lo_off) ? max(sym - 1, 0) : min(sym + 1, CG_NSYM - 1);
      clo = tab[sym];
      chi = sym + 1 >= CG_NSYM ? CG_TOTAL : (uint32_t)tab[sym + 1];
      lo_off = scaled_off(rm1, clo);
      hoff = scaled_off(rm1, chi);
      d = D - lo_off;
      rsz = hoff - lo_off;
      if (d < rsz) break;
    }
  }
  g10_advance(st, lo_off, hoff, d, rsz);
  return (uint32_t)sym;
}

__device__ __forceinline__ void wave_sync_lds() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__global__ __launch_bounds__(256) void tok_decode_kernel(
    KParams P, const uint32_t* __restrict__ words, const uint64_t* __restrict__ offsets,
    const uint8_t* __restrict__ chunk_level, const uint16_t* __restrict__ cdfA,
    const uint16_t* __restrict__ cdfD, int nbj, int64_t n_groups, uint8_t* __restrict__ sym) {
  __shared__ __attribute__((aligned(16))) uint16_t tabs[4][2][2][kTokTab];  // [wave][buffer][anchor, delta]
  __shared__ __attribute__((aligned(16))) uint8_t rows[4][64 * kTokRow];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int64_t grp = (int64_t)blockIdx.x * 4 + wave;
  if (grp >= n_groups) return;   // per wave; only wave-level synchronisation below
  const TokGroup g = tok_group(P, grp, nbj);
  if (g.jb * 64 >= g.n) return;  // a block past a short last chunk: no streams
  const int l = g.lk >> 1, k = g.lk & 1;
  const int t0 = g.c * P.CL;
  const int j = g.jb * 64 + lane;
  const bool valid = j < g.n;
  const int jl = valid ? j : g.n - 1;   // lanes past the chunk decode a copy of its last token
  const bool anchor = jl % P.G == 0;
  const int lv = uni(min((int)chunk_level[(int64_t)g.b * P.NC + g.c], P.NLV - 1));
  const int64_t sidx = tok_stream(P, g.b, g.c, g.lk, jl, g.n);
  const int64_t St = (int64_t)P.B * P.L * 2 * P.T;
  uint16_t* tw = &tabs[wave][0][0][0];
  // sentinels: entries 256..263 of the four staged tables (never overwritten)
  if (lane < 16) reinterpret_cast<uint32_t*>(tw + (lane >> 2) * kTokTab + 256)[lane & 3] = 0xFFFFFFFFu;
  // staging: lane L copies bytes 16 (L % 32) .. +16 of table L / 32 (0 anchor, 1 delta); the
  // lane holding entry 255 replaces it with a sentinel
  const int kind = lane >> 5, part = lane & 31;
  const uint16_t* src = (kind ? cdfD + ((int64_t)lv * 2 * P.L + g.lk) * P.C * 256
                              : cdfA + (int64_t)g.lk * P.C * 256) + part * 8;
  uint4 v = *reinterpret_cast<const uint4*>(src);
  if (part == 31) v.w = (v.w & 0xFFFFu) | 0xFFFF0000u;
  *reinterpret_cast<uint4*>(tw + kind * kTokTab + part * 8) = v;
  wave_sync_lds();

  const uint64_t total = offsets[St];
  if (total == 0) return;
  G10Lane st;
  const uint64_t o0 = offsets[sidx];
  const uint64_t ob = o0 < total ? o0 : total;
  const uint32_t* sbase = words + ob;
  const uint32_t cap = (uint32_t)((total - ob) < 0xFFFFFFF0ull ? (total - ob) : 0xFFFFFFF0ull);
  st.D = sbase[0];
  st.w0 = 0u;   // used up: the stream continues with w1
  st.w1 = sbase[1];
  st.w2 = sbase[2];
  st.w3 = sbase[3];
  st.avail = 0;
  st.hcnt = 0;
  st.widx = 4;
  const uint32_t* tq0 = sbase + (4u < cap ? 4u : cap);
  st.t0 = tq0[0];
  st.t1 = tq0[1];
  st.t2 = tq0[2];
  st.t3 = tq0[3];
  settle(st.D); settle(st.w0); settle(st.w1); settle(st.w2); settle(st.w3);
  st.low = 0u;
  st.lsh = 0u;
  st.rm1 = 0xFFFFFFFFu;
  st.a = 0.0f;

  uint8_t* myrow = &rows[wave][lane * kTokRow];
  uint8_t* gout = sym + cg_elem(P, g.b, l, k, t0 + jl, 0);
  for (int ch = 0; ch < P.C; ++ch) {
    // bitstream epochs every four symbols (at most 72 bits between two)
    if ((ch & 3) == 0 && ch != 0) g10_epoch(st, sbase, cap);
    const bool more = ch + 1 < P.C;
    if (more) v = *reinterpret_cast<const uint4*>(src + (int64_t)(ch + 1) * 256);
    const uint32_t sy = tok_symbol(st, tw + ((ch & 1) * 2 + (anchor ? 0 : 1)) * kTokTab);
    myrow[ch & 63] = (uint8_t)sy;
    if ((ch & 63) == 63 || !more) {
      // this lane's row of up to 64 symbols to the symbol array
      const int c0 = ch & ~63, cnt = ch - c0 + 1;
      if (valid) {
        if (cnt == 64 && (reinterpret_cast<uintptr_t>(gout + c0) & 3) == 0) {
#pragma unroll
          for (int i = 0; i < 16; ++i)
            reinterpret_cast<uint32_t*>(gout + c0)[i] = reinterpret_cast<const uint32_t*>(myrow)[i];
        } else {
          for (int i = 0; i < cnt; ++i) gout[c0 + i] = myrow[i];
        }
      }
    }
    if (more) {
      if (part == 31) v.w = (v.w & 0xFFFFu) | 0xFFFF0000u;
      *reinterpret_cast<uint4*>(tw + (((ch + 1) & 1) * 2 + kind) * kTokTab + part * 8) = v;
      wave_sync_lds();
    }
  }
}

// Reconstruct the channel streams from the symbol array (the channel layout's dequantization):
// one wave per (context, chunk, layer, K/V, 64-channel block), a lane per channel.
__global__ __launch_bounds__(256) void tok_dequant_kernel(KParams P, const uint8_t* __restrict__ sym,
                                                          const float* __restrict__ scales,
                                                          const uint8_t* __restrict__ chunk_level,
                                                          uint16_t* __restrict__ out) {
  const int64_t item = (int64_t)blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (item >= (int64_t)P.B * P.NC * P.L * 2 * P.nblk) return;
  const int cb = (int)(item % P.nblk);
  int64_t r = item / P.nblk;
  const int k = (int)(r & 1);
  r >>= 1;
  const int l = (int)(r % P.L);
  r /= P.L;
  const int c = (int)(r % P.NC);
  const int b = (int)(r / P.NC);
  const int ch = cb * 64 + lane;
  if (ch >= P.C) return;
  const int t0 = c * P.CL;
  const int n = min(P.CL, P.T - t0);
  const float s = scales[cg_stream(P, (((int64_t)b * P.NC + c) * P.L + l) * 2 + k, ch)];
  const int lv = min((int)chunk_level[(int64_t)b * P.NC + c], P.NLV - 1);
  const float w = P.layer_bin[l] * P.level_mult[lv] * s;
  const uint8_t* x = sym + cg_elem(P, b, l, k, t0, ch);
  uint16_t* y = out + cg_elem(P, b, l, k, t0, ch);
  const int64_t rs = P.C;
  float a = 0.0f;
  int g = 0;
  for (int j = 0; j < n; ++j) {
    const float qf = (float)((int)x[(int64_t)j * rs] - 127);
    float v;
    if (g == 0) {
      a = qf * s;
      v = a;
    } else {
      v = a + qf * w;
    }
    y[(int64_t)j * rs] = cg_f2h(v);
    g = (g + 1 == P.G) ? 0 : g + 1;
  }
}

}  // namespace

hipError_t cg_launch_decode_tokens(const KParams& P, const uint32_t* words,
                                   const uint64_t* offsets, const float* scales,
                                   const uint8_t* chunk_level, const uint16_t* cdf_anchor,
                                   const uint16_t* cdf_delta, uint8_t* sym, uint16_t* out,
                                   hipStream_t st) {
  const TokEncWorkspace lay = cg_encode_tokens_ws_layout(P);
  hipLaunchKernelGGL(tok_decode_kernel, dim3((unsigned)((lay.n_groups + 3) / 4)), dim3(256), 0,
                     st, P, words, offsets, chunk_level, cdf_anchor, cdf_delta, lay.nbj,
                     lay.n_groups, sym);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t items = (int64_t)P.B * P.NC * P.L * 2 * P.nblk;
  hipLaunchKernelGGL(tok_dequant_kernel, dim3((unsigned)((items + 3) / 4)), dim3(256), 0, st, P,
                     sym, scales, chunk_level, out);
  return hipGetLastError();
}

hipError_t cg_launch_decode(const KParams& P, const uint32_t* words, const uint64_t* offsets,
                            const float* scales, const uint8_t* chunk_level,
                            const uint16_t* cdf_anchor, const uint16_t* cdf_delta, int c_begin,
                            int c_end, uint16_t* out, hipStream_t st) {
  const int64_t n_pairs = (int64_t)P.B * (c_end - c_begin);
  if (n_pairs == 0) return hipSuccess;
  // LDS of a workgroup of w waves: row buffers plus one delta table set per level its pairs
  // may use (sized for the worst case, min(w, levels) sets); fewer waves per workgroup when
  // that exceeds what a CU offers
  const bool g10 = P.G == kG10;
  auto lds_for = [&](int w, int nu) {
    const size_t sets = (size_t)(w < P.NLV ? w : P.NLV);
    const size_t rows = g10 ? (size_t)nu * w * kG10 * 64
                            : (size_t)64 * kFenceStride + (size_t)w * kRows * 64;
    return (rows + (size_t)nu * sets * 64 * kTabStride) * sizeof(uint16_t);
  };
  int nw = (int)(n_pairs < kMaxWaves ? n_pairs : kMaxWaves);
  while (nw > 1 && lds_for(nw, 1) > kLdsBudget) --nw;
  const int64_t n_groups = (n_pairs + nw - 1) / nw;
  const int64_t n_units = (int64_t)P.L * 2 * P.nblk;
  if (g10) {
    // several units per workgroup while the grid still covers every CU: one workgroup then
    // holds all of a CU's waves, which the hardware spreads evenly over the SIMDs
    int nu = 1;
    while (nu < kMaxUnits && (nu + 1) * nw <= kMaxWaves && lds_for(nw, nu + 1) <= kLdsBudget &&
           (n_units + nu) / (nu + 1) * n_groups >= 256)
      ++nu;
    const int msets = nw < P.NLV ? nw : P.NLV;
    // With several levels, the delta tables can instead be staged as windows (decode_g10_kernel
    // <true>): a unit then needs a region of one table set (its anchor tables) plus window
    // descriptors, so more units fit a workgroup. Used when that allows more units.
    const size_t rows = (size_t)nw * kG10 * 64 * sizeof(uint16_t);   // per unit
    const size_t set_bytes = (size_t)64 * kTabStride * sizeof(uint16_t);
    const size_t desc_bytes = (size_t)msets * 64 * sizeof(uint32_t);
    int nuc = 1;
    while (nuc < kMaxUnits && (nuc + 1) * nw <= kMaxWaves &&
           (size_t)(nuc + 1) * (rows + set_bytes + desc_bytes) <= kLdsBudget &&
           (n_units + nuc) / (nuc + 1) * n_groups >= 256)
      ++nuc;
    const bool compact = msets > 1 && nuc > nu;
    int units = nu, ustride = (int)((size_t)msets * 64 * kTabStride);
    size_t lds = lds_for(nw, nu);
    if (compact) {
      units = nuc;
      // each unit's region: what the LDS budget leaves, in 16-byte multiples
      const size_t per_unit = kLdsBudget / (size_t)nuc - rows - desc_bytes;
      ustride = (int)((per_unit & ~(size_t)15) / sizeof(uint16_t));
      lds = (size_t)nuc * (rows + desc_bytes) + (size_t)nuc * ustride * sizeof(uint16_t);
    }
    const int64_t grid = cg_xcd_grid((n_units + units - 1) / units, n_groups);
    const void* kfn = compact ? (const void*)decode_g10_kernel<true>
                              : (const void*)decode_g10_kernel<false>;
    hipError_t e = hipFuncSetAttribute(kfn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    if (compact)
      hipLaunchKernelGGL(decode_g10_kernel<true>, dim3((unsigned)grid), dim3(64 * nw * units), lds,
                         st, P, words, offsets, scales, chunk_level, cdf_anchor, cdf_delta,
                         c_begin, c_end, nw, units, ustride, out);
    else
      hipLaunchKernelGGL(decode_g10_kernel<false>, dim3((unsigned)grid), dim3(64 * nw * units),
                         lds, st, P, words, offsets, scales, chunk_level, cdf_anchor, cdf_delta,
                         c_begin, c_end, nw, units, ustride, out);
    return hipGetLastError();
  }
  const int64_t grid = cg_xcd_grid(n_units, n_groups);
  const size_t lds = lds_for(nw, 1);
  hipError_t e = hipFuncSetAttribute((const void*)decode_kernel,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(decode_kernel, dim3((unsigned)grid), dim3(64 * nw), lds, st, P, words,
                     offsets, scales, chunk_level, cdf_anchor, cdf_delta, c_begin, c_end, nw,
                     out);
  return hipGetLastError();
}
