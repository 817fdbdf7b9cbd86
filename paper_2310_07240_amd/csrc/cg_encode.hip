// cg_encode.hip — encoder (CacheGen Sec. 5.2: change-based encoding, layer-wise quantization,
// arithmetic coding; Sec. 5.3: each chunk coded independently at its own level).
//
// Launches:
//   encode_kernel   workgroup = (layer, K/V, 64-channel block) x up to 16 (context, chunk)
//                   pairs, one wave per pair and one lane per stream (every token row is one
//                   coalesced 128-byte load); the delta tables of the levels in use sit in LDS.
//                   Absmax scale, quantize, arithmetic-code into a worst-case slot of the
//                   workspace, record the stream's word count;
//   scan_reduce     per-block totals of the word counts (4096 streams per block);
//   scan_top        exclusive scan of the block totals (one workgroup);
//   scan_finish     block-local exclusive scan (wave prefix sums + LDS) plus the block's
//                   carry -> offsets[S + 1];
//   compact         one workgroup per (row, 64-channel block) moves its 64 streams' words
//                   from the slots (interleaved by 16-byte chunk) to their offsets, through an
//                   LDS transpose.
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
#include <type_traits>

#include "cg_device.h"

namespace {

constexpr int kEncMaxWaves = 16;
constexpr int kEncMaxUnits = 16;   // (layer, K/V, channel block) units per workgroup
// waves per workgroup with windowed delta tables: their lookups need more registers than 16
// waves per CU leave (at 12, three waves per SIMD, each may hold 168)
constexpr int kEncWinWaves = 12;
constexpr int kEncStageBatch = 8;  // table-staging loads in flight per lane
constexpr int kCompactRows = 128;  // slot rows per pass of the compaction
// static LDS of the kernel with several units (masks, level maps, SIMD ids, remaining counts);
// the dynamic LDS budget leaves 1 KB for it
static_assert(4 * kEncMaxUnits + 4 * kEncMaxUnits * CG_MAX_LEVELS + 2 * kEncMaxUnits + kEncMaxWaves +
                  4 * kEncMaxWaves + 4 <= 1024 - 64,
              "static LDS exceeds the reserve");
constexpr size_t kEncLdsBudget = 160 * 1024 - 1024;   // dynamic LDS per workgroup (CDNA4: 160 KB)
constexpr int kEncTabStride = 258;   // u16 per delta table in LDS (odd word stride: lanes spread over banks)
constexpr int kScanThreads = 256;
constexpr int kScanItems = 16;
constexpr int kScanBlock = kScanThreads * kScanItems;  // 4096 streams per scan block

// Output of one stream. Finished words go to a lane-private ring of kRing words in LDS and reach
// the stream's slot in global memory as whole 16-byte chunks (four words, 16-byte aligned): a
// flush stores the oldest four pending words once they are all there. A slot group of 64
// streams is interleaved by chunk (chunk m of lane L at words (64 m + L) * 4 of the group), so
// a lane's store is one 16-byte write and a row of chunks is 1 KB for the compaction. Flushes
// are issued right after a step's row values were consumed and between runs of at most five
// symbols: stores issued between the pipeline's loads would make every later wait for those
// loads wait for the stores too (loads and stores share one in-order counter).
//
// Ring bound: a run starts with at most 3 pending words. On the common path a symbol emits at
// most 32 bits and at most 32 + 18 k bits over k symbols (the owed bits it starts with, which
// are at most 32 when any of them is emitted there, plus at most 18 shifts per symbol), so a
// run of at most five symbols adds at most 4 words: never more than 7 are pending, and the slot
// after the last pending word, which the branch-free coder always writes, is free. The rare
// paths (long runs of owed bits, the end of the stream) put one word at a time and flush after
// each.
constexpr int kRing = 8;

struct BitSink {
  uint32_t* out;    // chunk column of this lane: word k at out[256 (k / 4) + k % 4]
  uint32_t cap;     // slot capacity in words (a multiple of 4)
  uint32_t nwords;  // words produced
  uint32_t flushed; // words already in the slot (a multiple of 4)
  uint64_t acc;     // output bits not yet in a word: the low nacc bits (higher bits ignored)
  uint32_t nacc;    // number of bits in acc, < 32 between calls
  uint32_t* ring;   // this lane's kRing words in LDS, 64 words apart (bank-conflict free)

  // a finished word
  __device__ __forceinline__ void word(uint32_t w) {
    ring[(nwords & (kRing - 1)) * 64] = w;
    ++nwords;
  }
  // the oldest four pending words as one chunk, once they are all there
  __device__ __forceinline__ void flush() {
    const uint32_t* r = ring + (flushed & (kRing - 1)) * 64;   // flushed % 8 is 0 or 4
    const uint4 v = make_uint4(r[0], r[64], r[128], r[192]);
    const bool full = nwords - flushed >= 4u;
    if (full && flushed < cap) *reinterpret_cast<uint4*>(out + (uint64_t)(flushed >> 2) * 256) = v;
    flushed += full ? 4u : 0u;
  }
  // a flush in two halves: the ring read first, the store later (after the waits for loads
  // that were issued before it, which then do not cover the store)
  __device__ __forceinline__ uint4 flush_read(bool& full) const {
    const uint32_t* r = ring + (flushed & (kRing - 1)) * 64;
    full = nwords - flushed >= 4u;
    return make_uint4(r[0], r[64], r[128], r[192]);
  }
  __device__ __forceinline__ void flush_store(const uint4& v, bool full) {
    if (full && flushed < cap) *reinterpret_cast<uint4*>(out + (uint64_t)(flushed >> 2) * 256) = v;
    flushed += full ? 4u : 0u;
  }
  // the last chunk, partly filled (its words past nwords are never read)
  __device__ __forceinline__ void flush_last() {
    flush();
    if (nwords > flushed) {
      const uint32_t* r = ring + (flushed & (kRing - 1)) * 64;
      const uint4 v = make_uint4(r[0], r[64], r[128], r[192]);
      if (flushed < cap) *reinterpret_cast<uint4*>(out + (uint64_t)(flushed >> 2) * 256) = v;
      flushed = nwords;
    }
  }
  // output of the rare paths: bit by bit into words, a flush after each word
  __device__ __forceinline__ void put(uint32_t bits, uint32_t nb) {  // nb <= 32
    acc = (acc << nb) | bits;
    nacc += nb;
    if (nacc >= 32) {
      nacc -= 32;
      word((uint32_t)(acc >> nacc));
      flush();
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
  const uint32_t P = e.pending;
  if (n1 != 0 && P + n1 <= 32) {
    // the n1 shared leading bits H, the first of them followed by P opposite bits: as one
    // number of P + n1 bits this is H + ((2^P - 1) << (n1 - 1))
    const uint32_t H = low >> (32 - n1);
    const uint32_t E = P + n1;
    const uint32_t val = H + ((uint32_t)((1ull << P) - 1ull) << (n1 - 1));
    o.acc = (o.acc << E) | val;   // bits above the nacc valid ones are never read
    o.nacc += E;
    if (o.nacc >= 32) {
      o.nacc -= 32;
      o.word((uint32_t)(o.acc >> o.nacc));
    }
    e.pending = 0;
  } else if (n1 != 0) {   // more than 32 bits owed (long middle-half runs): bit by bit
    o.flush();
    const uint32_t b0 = low >> 31;
    o.put(b0, 1);
    o.run(b0 ^ 1u, P);
    e.pending = 0;
    if (n1 > 1) o.put((low << 1) >> (33 - n1), n1 - 1);
  }
  const uint32_t L1 = low << n1, H1 = high << n1;
  const uint32_t m = L1 & ~H1;
  const uint32_t n3 = __clz(~(m << 1));
  e.pending += n3;
  e.low = (L1 << n3) & 0x7FFFFFFFu;   // L1 has a clear top bit
  const uint32_t n = n1 + n3;  // at most 18 (the new range is at least 2^14)
  e.rm1 = (rm1 << n) | ((1u << n) - 1u);
}

// The same symbol without branches, for the steps where no lane owes more than 32 bits: the
// E = P + n1 output bits (none when n1 = 0) go into acc unconditionally, and the ring slot of
// the next word is always written (with the finished word, or with bits a later word
// overwrites: that slot holds no pending word, since at most kRing - 1 are pending). `rare` is
// set when P + n1 > 32; the step is then coded again from its saved state with enc_symbol.
__device__ __forceinline__ void enc_symbol_fast(EncState& e, BitSink& o, uint32_t clo,
                                                uint32_t chi, bool& rare) {
  const uint32_t lo_off = (uint32_t)(((uint64_t)e.rm1 * clo + clo) >> 16);
  // the new interval's size (2^32 wraps to 0, which the shift below turns into the full range)
  const uint32_t rsz = (uint32_t)(((uint64_t)e.rm1 * chi + chi) >> 16) - lo_off;
  const uint32_t low = e.low + lo_off;
  const uint32_t high = low + rsz - 1u;
  const uint32_t n1 = (uint32_t)__builtin_clz(low ^ high);   // high > low
  const uint32_t P = e.pending;
  const bool emit = n1 != 0;
  const uint32_t E = emit ? P + n1 : 0u;
  rare |= E > 32u;
  const uint32_t H = low >> ((32u - n1) & 31u);
  // ((1 << P) - 1) << (n1 - 1), both amounts mod 32, as one bitfield-mask instruction
  uint32_t runb;
  asm("v_bfm_b32 %0, %1, %2" : "=v"(runb) : "v"(P), "v"(n1 - 1u));
  const uint32_t val = emit ? H + runb : 0u;
  o.acc = (o.acc << E) | val;   // bits above the nacc valid ones are never read
  const uint32_t t = o.nacc + E;   // < 64
  const bool full = t >= 32u;
  o.nacc = t & 31u;
  // ring slot (nwords mod kRing) * 64 words: kept as an index and a shift-add (else the compiler
  // turns it into a shift, a mask and an add)
  uint32_t slot = o.nwords & (kRing - 1);
  asm("" : "+v"(slot));
  o.ring[slot * 64] = (uint32_t)(o.acc >> o.nacc);
  o.nwords += full ? 1u : 0u;
  // the middle-half run: f - 1 leading ones of (low & ~high) << (n1 + 1), from v_ffbh_i32 (the
  // count of leading bits equal to the sign bit) of (low & ~high) << n1 with its top bit set
  uint32_t lh, f;
  asm("v_bfi_b32 %0, %1, 0, %2" : "=v"(lh) : "v"(high), "v"(low));   // low & ~high
  asm("v_ffbh_i32 %0, %1" : "=v"(f) : "v"((lh << n1) | 0x80000000u));
  e.pending = (emit ? 0u : P) + f - 1u;
  const uint32_t n = n1 + f - 1u;
  e.low = (low << n) & 0x7FFFFFFFu;
  e.rm1 = (rsz << n) - 1u;
}

__device__ __forceinline__ void enc_finish(EncState& e, BitSink& o) {
  o.flush();
  e.pending += 1;
  const uint32_t b = e.low >= 0x40000000u ? 1u : 0u;
  o.put(b, 1);
  o.run(b ^ 1u, e.pending);
  if (o.nacc) o.put(0u, 32 - o.nacc);  // zero-pad to a whole word
  o.flush_last();
}

// Token pipeline of the encoder: the symbols and their table entries do not depend on the
// coder state, so they are produced ahead of it. Per step of kPipe tokens, the row values of
// the tokens two steps ahead are requested, the tokens one step ahead are quantized and their
// (cum[sym], cum[sym + 1]) requested from the tables, and the tokens of this step are coded
// with the entries requested one step earlier. With the paper's group of 10 a step is one
// group (kG = 10: the anchor is always the step's first token, so every step issues the same
// memory operations); other group sizes use steps of 8 tokens (kG = 0).

// kWin: the delta tables are staged as windows of their 16-entry blocks (cg_table_window):
// each unit has a region of ustride u16 (at least one whole table set), holding its anchor
// tables for the anchor pass and then the packed windows of its delta tables; sets that do not
// fit together are staged in rounds. Entries outside a window follow the flat closed forms.
// Otherwise the region holds nsets_lds whole sets.
template <int kG, bool kWin>
__global__ __launch_bounds__(kWin ? 64 * kEncWinWaves : 1024) void encode_kernel(
    KParams P, const uint16_t* __restrict__ kv, const uint8_t* __restrict__ chunk_level,
    const uint16_t* __restrict__ cdfA, const uint16_t* __restrict__ cdfD,
    uint32_t* __restrict__ slots, uint32_t slot_words, uint32_t* __restrict__ lens,
    float* __restrict__ scales, uint32_t* __restrict__ wflags, int nw, int nu, int nsets_lds,
    int ustride, int scales_given) {
  // workgroup = nu units (layer, K/V, 64-channel block) x nw (context, chunk) pairs; wave w
  // codes pair slot w / nu of unit w % nu (one workgroup per CU where the grid allows, so the
  // hardware spreads its waves evenly over the SIMDs). The anchor tables of the units are
  // staged in LDS for the anchor pass, then the delta tables of the levels their pairs use for
  // the delta pass.
  extern __shared__ __attribute__((aligned(16))) uint16_t tabs[];   // [nu][ustride], then words [nu * nw][kRing][64], then window descriptors [nu][nsets][64] (kWin)
  __shared__ uint32_t s_mask[kEncMaxUnits];
  __shared__ uint8_t s_set_of_level[kEncMaxUnits][CG_MAX_LEVELS];
  __shared__ uint8_t s_level_of_set[kEncMaxUnits][CG_MAX_LEVELS];
  __shared__ uint8_t s_nsets[kEncMaxUnits];
  __shared__ uint8_t s_simd[kEncMaxWaves];   // SIMD of each wave
  __shared__ int s_left[kEncMaxWaves];   // symbols each wave has left to code
  __shared__ uint32_t s_bad;               // some stream of the workgroup holds NaN or Inf
  __shared__ uint8_t s_round[kEncMaxUnits][CG_MAX_LEVELS];   // staging round of each set (kWin)
  __shared__ uint8_t s_nrounds[kEncMaxUnits];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int nwaves = blockDim.x >> 6;
  const int u = wave % nu, j = wave / nu;
  const int n_pairs = P.B * P.NC;
  const int n_groups = (n_pairs + nw - 1) / nw;
  const int n_units = P.L * 2 * P.nblk;
  int ublk, grp;
  cg_xcd_map((n_units + nu - 1) / nu, n_groups, ublk, grp);
  if (ublk * nu >= n_units) {   // past the last unit block (uniform over the workgroup)
    if (threadIdx.x == 0) wflags[blockIdx.x] = 0u;
    return;
  }
  const int unit = ublk * nu + u;
  const int cb = unit % P.nblk;
  const int k = (unit / P.nblk) & 1, l = (unit / P.nblk) >> 1;
  const int pair = __builtin_amdgcn_readfirstlane(grp * nw + j);
  const bool active = unit < n_units && pair < n_pairs;
  // pairs chunk-major: the waves of a workgroup code the same chunk of consecutive contexts
  const int b = active ? pair % P.B : 0;
  const int c = active ? pair / P.B : 0;
  const int lv = active ? min((int)chunk_level[(int64_t)b * P.NC + c], P.NLV - 1) : 0;
  const int n = active ? min(P.CL, P.T - c * P.CL) : 0;

  const int simd = (int)((__builtin_amdgcn_s_getreg((31 << 11) | 4) >> 4) & 3u);   // HW_ID
  if (threadIdx.x < nu) s_mask[threadIdx.x] = 0u;
  if (threadIdx.x == 0) s_bad = 0u;
  if (lane == 0) {
    s_simd[wave] = simd;
    lds_put(&s_left[wave], n);
  }
  __syncthreads();
  if (active && lane == 0) atomicOr(&s_mask[u], 1u << lv);
  __syncthreads();
  if (threadIdx.x < nu) {
    const int uu = threadIdx.x;
    int m = 0;
    for (int v = 0; v < P.NLV; ++v)
      if ((s_mask[uu] >> v) & 1u) { s_set_of_level[uu][v] = m; s_level_of_set[uu][m] = v; ++m; }
    s_nsets[uu] = m;
  }
  __syncthreads();
  // Stage tables into LDS: the anchor table of every unit (set 0; the anchor pass), or the
  // delta tables of the levels each unit's pairs use (the delta pass). A row (one table, 512
  // bytes) is 32 lanes x 16 bytes, so a wave moves two rows per load instruction;
  // kEncStageBatch unconditional loads per lane (a row that is not staged reads the first
  // table instead) are in flight before their stores.
  const int half = lane >> 5, piece = lane & 31;
  auto stage = [&](bool anchors) __attribute__((always_inline)) {
    const int sets = anchors ? 1 : nsets_lds;
    const int n_rows = nu * sets * 64;
    const uint16_t* srcbase = anchors ? cdfA : cdfD;
    for (int base = wave; base * 2 < n_rows; base += nwaves * kEncStageBatch) {
      uint4 v[kEncStageBatch];
      int dsto[kEncStageBatch];
#pragma unroll
      for (int i = 0; i < kEncStageBatch; ++i) {
        const int rr = (base + i * nwaves) * 2 + half;
        const int t = rr & 63, st = (rr >> 6) % sets;
        const int uu = min((rr >> 6) / sets, nu - 1);
        const int unit2 = ublk * nu + uu;
        const int chs = (unit2 % P.nblk) * 64 + t;
        const int lset = s_level_of_set[uu][st];   // in bounds for any rr
        const int nset = anchors ? 1 : (int)s_nsets[uu];
        const bool ok = (rr < n_rows) & (unit2 < n_units) & (st < nset) & (chs < P.C);
        const int lk = unit2 / P.nblk;   // l * 2 + k
        const int64_t trow = anchors ? (int64_t)lk * P.C + chs
                                     : ((int64_t)lset * P.L * 2 + lk) * P.C + chs;
        v[i] = reinterpret_cast<const uint4*>(srcbase + (ok ? trow : 0) * 256)[piece];
        dsto[i] = ok ? uu * ustride + (st * 64 + t) * kEncTabStride + piece * 8 : -1;
      }
#pragma unroll
      for (int i = 0; i < kEncStageBatch; ++i) {
        if (dsto[i] < 0) continue;
        uint32_t* dst = reinterpret_cast<uint32_t*>(tabs + dsto[i]);   // 4-byte aligned rows
        dst[0] = v[i].x;
        dst[1] = v[i].y;
        dst[2] = v[i].z;
        dst[3] = v[i].w;
      }
    }
  };
  uint32_t* const rings_base = reinterpret_cast<uint32_t*>(tabs + (size_t)nu * ustride);
  uint32_t* const desc = rings_base + (size_t)nu * nw * kRing * 64;   // kWin
  // Window staging of the delta tables (kWin): pass 1 finds each table's window, pass 2 (one
  // wave per unit) lays the windows out set after set with a new round whenever a set does not
  // fit the region any more, and stage_round writes the windows of one round's sets.
  auto window_pass = [&]() __attribute__((always_inline)) {
    const int n_rows = nu * nsets_lds * 64;
    for (int base = wave; base * 2 < n_rows; base += nwaves * kEncStageBatch) {
      uint4 v[kEncStageBatch];
      int rows[kEncStageBatch];
#pragma unroll
      for (int i = 0; i < kEncStageBatch; ++i) {
        const int rr = (base + i * nwaves) * 2 + half;
        const int t = rr & 63, st = (rr >> 6) % nsets_lds;
        const int uu = min((rr >> 6) / nsets_lds, nu - 1);
        const int unit2 = ublk * nu + uu;
        const int chs = (unit2 % P.nblk) * 64 + t;
        const int lset = s_level_of_set[uu][st];
        const bool ok = (rr < n_rows) & (unit2 < n_units) & (st < (int)s_nsets[uu]) & (chs < P.C);
        const int64_t trow = ((int64_t)lset * P.L * 2 + unit2 / P.nblk) * P.C + chs;
        v[i] = reinterpret_cast<const uint4*>(cdfD + (ok ? trow : 0) * 256)[piece];
        rows[i] = ok ? rr : -1;
      }
#pragma unroll
      for (int i = 0; i < kEncStageBatch; ++i) {
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
    for (int st = 0; st < nsets_lds; ++st) {
      const int idx = (uu * nsets_lds + st) * 64 + lane;
      const bool ok = chok && st < (int)s_nsets[uu];
      const uint32_t d = ok ? desc[idx] : 0u;
      const uint32_t sz = d >> 8;
      const uint32_t incl = cg_wave_incl_scan(sz);
      const int tot = __builtin_amdgcn_readfirstlane((int)__shfl(incl, 63, 64));
      if (acc > 0 && acc + tot > pool) { ++round; acc = 0; }
      if (ok) desc[idx] = (uint32_t)(acc + (int)(incl - sz)) | ((d & 0xFFu) << 20);
      if (lane == 0) s_round[uu][st] = (uint8_t)round;
      acc += tot;
    }
    if (lane == 0) s_nrounds[uu] = (uint8_t)(round + 1);
  };
  auto stage_round = [&](int rd) __attribute__((always_inline)) {
    const int n_rows = nu * nsets_lds * 64;
    for (int base = wave; base * 2 < n_rows; base += nwaves * kEncStageBatch) {
      uint4 v[kEncStageBatch];
      int dsto[kEncStageBatch], k0s[kEncStageBatch], kends[kEncStageBatch];
#pragma unroll
      for (int i = 0; i < kEncStageBatch; ++i) {
        const int rr = (base + i * nwaves) * 2 + half;
        const int t = rr & 63, st = (rr >> 6) % nsets_lds;
        const int uu = min((rr >> 6) / nsets_lds, nu - 1);
        const int unit2 = ublk * nu + uu;
        const int chs = (unit2 % P.nblk) * 64 + t;
        const int lset = s_level_of_set[uu][st];
        const bool ok = (rr < n_rows) & (unit2 < n_units) & (st < (int)s_nsets[uu]) &
                        (chs < P.C) && (int)s_round[uu][st] == rd;
        const int64_t trow = ((int64_t)lset * P.L * 2 + unit2 / P.nblk) * P.C + chs;
        v[i] = reinterpret_cast<const uint4*>(cdfD + (ok ? trow : 0) * 256)[piece];
        const uint32_t d = ok ? desc[min(rr, n_rows - 1)] : 0u;
        dsto[i] = ok ? uu * ustride + (int)((d & 0xFFFFFu) >> 1) : -1;
        k0s[i] = 16 * (int)((d >> 20) & 15u);
        kends[i] = 16 * ((int)((d >> 24) & 15u) + 1) + 4;
      }
#pragma unroll
      for (int i = 0; i < kEncStageBatch; ++i) {
        if (dsto[i] < 0) continue;
        uint16_t* dst = tabs + dsto[i] - k0s[i];   // entry k of the table at dst[k]
        const int e = 8 * piece;
        if (e >= k0s[i] && e < kends[i])
          *reinterpret_cast<uint2*>(dst + e) = make_uint2(v[i].x, v[i].y);
        if (e + 4 >= k0s[i] && e + 4 < kends[i])
          *reinterpret_cast<uint2*>(dst + e + 4) = make_uint2(v[i].z, v[i].w);
      }
    }
  };
  stage(true);
  if constexpr (kWin) window_pass();
  __syncthreads();
  if constexpr (kWin) {
    layout_pass();
    __syncthreads();
  }

  // Absmax of the streams. When the workgroup holds four channel-contiguous units of one
  // (layer, K/V) and all its pairs are valid (uniform over the workgroup), the four waves of a
  // pair split the chunk's rows (wave u takes rows u, u + 4, ...) and read all 256 channels of
  // a row, 8 bytes (4 channels) per lane; the partial maxima meet in LDS, in the ring area
  // that coding uses only later. Otherwise every wave reads its own 64 channels row by row.
  const int cb0 = (ublk * nu) % P.nblk;
  const bool coop = !scales_given && nu == 4 && (ublk + 1) * nu <= n_units &&
                    cb0 + nu <= P.nblk && (cb0 + nu) * 64 <= P.C && (grp + 1) * nw <= n_pairs &&
                    (P.C & 3) == 0 &&
                    (reinterpret_cast<uintptr_t>(kv) & 7) == 0;   // 8-byte aligned row loads
  // The maximum is taken over the magnitude bits (x & 0x7fff) as integers: for finite halves
  // their order is the order of |x|, and NaN or Inf (exponent all ones) gives a maximum of at
  // least 0x7c00, which flags the stream as outside the quantizer's domain.
  uint32_t mx_coop = 0u;
  if (coop) {
    uint32_t* part = rings_base;
    const uint16_t* xr = kv + cg_elem(P, b, l, k, c * P.CL, cb0 * 64) + 4 * lane;
    const int64_t rs4 = P.C;
    const int nr = (n - u + 3) / 4;   // rows u, u + 4, ... below n
    uint32_t m0 = 0u, m1 = 0u, m2 = 0u, m3 = 0u;
    for (int i0 = 0; i0 < nr; i0 += 16) {
      uint2 v[16];
#pragma unroll
      for (int q = 0; q < 16; ++q)
        v[q] = *reinterpret_cast<const uint2*>(xr + (int64_t)(u + 4 * min(i0 + q, nr - 1)) * rs4);
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        m0 = max(m0, v[q].x & 0x7FFFu);
        m1 = max(m1, (v[q].x >> 16) & 0x7FFFu);
        m2 = max(m2, v[q].y & 0x7FFFu);
        m3 = max(m3, (v[q].y >> 16) & 0x7FFFu);
      }
    }
    *reinterpret_cast<uint4*>(part + (j * nu + u) * 256 + 4 * lane) = make_uint4(m0, m1, m2, m3);
    __syncthreads();
#pragma unroll
    for (int u2 = 0; u2 < 4; ++u2) mx_coop = max(mx_coop, part[(j * nu + u2) * 256 + u * 64 + lane]);
    __syncthreads();   // the ring area is free again before any wave codes
  }

  // the (up to three) other waves of this workgroup on this wave's SIMD
  int p0 = wave, p1 = wave, p2 = wave, np = 0;
  for (int w2 = 0; w2 < nwaves; ++w2) {
    if (w2 == wave || __builtin_amdgcn_readfirstlane(s_simd[w2]) != simd) continue;
    if (np == 0) p0 = w2; else if (np == 1) p1 = w2; else if (np == 2) p2 = w2;
    ++np;
  }
  // issue priority by what is left among the waves of this SIMD (most left first), so that
  // they finish together instead of the oldest first
  auto set_priority = [&](int left) __attribute__((always_inline)) {
    const int l0 = __builtin_amdgcn_readfirstlane(lds_get(&s_left[p0]));
    const int l1 = __builtin_amdgcn_readfirstlane(lds_get(&s_left[p1]));
    const int l2 = __builtin_amdgcn_readfirstlane(lds_get(&s_left[p2]));
    lds_put(&s_left[wave], left);
    const int rank = (p0 != wave && (l0 > left || (l0 == left && p0 < wave))) +
                     (p1 != wave && (l1 > left || (l1 == left && p1 < wave))) +
                     (p2 != wave && (l2 > left || (l2 == left && p2 < wave)));
    if (rank == 0) __builtin_amdgcn_s_setprio(3);
    else if (rank == 1) __builtin_amdgcn_s_setprio(2);
    else if (rank == 2) __builtin_amdgcn_s_setprio(1);
    else __builtin_amdgcn_s_setprio(0);
  };
  const int ch = cb * 64 + lane;
  // lanes that code a stream (the others take part in the barriers between the passes only)
  const bool lane_ok = active && ch < P.C;
  const int64_t bclk = (((int64_t)b * P.NC + c) * P.L + l) * 2 + k;
  const int t0 = c * P.CL;
  const int64_t sidx = cg_stream(P, bclk, ch);
  const uint16_t* x = kv + cg_elem(P, b, l, k, t0, ch);
  const int64_t rs = P.C;

  uint32_t mbits = mx_coop;
  if (!coop && !scales_given && lane_ok) {
#pragma unroll 16
    for (int t = 0; t < n; ++t) mbits = max(mbits, (uint32_t)x[(int64_t)t * rs] & 0x7FFFu);
  }
  if (__builtin_amdgcn_ballot_w64(lane_ok && mbits >= 0x7C00u) != 0ull && lane == 0)
    atomicOr(&s_bad, 1u);
  const float mx = cg_h2f((uint16_t)mbits);
  // with scales_given the stream's scale comes in (from the fit's maxima of the same rows)
  const float s = scales_given ? (lane_ok ? scales[sidx] : 1.0f)
                               : (mx == 0.0f) ? 1.0f : mx / 127.0f;
  if (lane_ok && !scales_given) scales[sidx] = s;
  constexpr int kPipe = kG > 0 ? kG : 8;
  const float bw = P.layer_bin[l] * P.level_mult[lv];
  const float w = bw * s;
  const float is = 1.0f / s, iw = 1.0f / w;
  float one;   // 1.0 that the compiler cannot fold away
  asm volatile("s_mov_b32 %0, 1.0" : "=s"(one));

  cg_lds_u16* tabA = (cg_lds_u16*)(tabs + u * ustride + lane * kEncTabStride);   // anchors
  // the lane's delta table: the whole table (entry i at tabD[i]), or its window (entries wk0
  // .. wk1 + 3 at tabD[i], the rest by the closed forms); set for the delta pass
  cg_lds_u16* tabD = nullptr;
  int wk0 = 0, wk1 = 0;
  EncState e{0u, 0xFFFFFFFFu, 0u};
  uint32_t* rings = rings_base;
  // the slots of a wave's 64 streams, interleaved by 16-byte chunk
  const uint64_t slot_group = (uint64_t)bclk * P.nblk + cb;
  BitSink o{slots + slot_group * slot_words * 64 + lane * 4, slot_words, 0u, 0u, 0ull, 0u,
            rings + wave * kRing * 64 + lane};

  // Pipeline buffers, used in turn (steps alternate between set 0 and set 1, and the loop
  // body is written out for both so no buffer is ever copied: a copy of a register that a
  // load is still filling would make the copy wait for that load and for every memory
  // operation issued after it). xr*: row values; lo* / hi*: the table entries of a step.
  const int last = n - 1;
  float a = 0.0f;
  int gq = 0;   // group position of the next token to quantize (uniform)
  // quantize the next kPipe tokens from xv[] and request their table entries. Tokens past the
  // chunk end (rows clamped to the last one) are quantized too but never coded, so every step
  // issues the same memory operations.
  auto quantize_step = [&](const uint32_t (&xv)[kPipe], uint32_t (&clo)[kPipe],
                           uint32_t (&chi)[kPipe]) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < kPipe; ++u) {
      const float v = cg_h2f((uint16_t)xv[u]);
      const bool anc = kG > 0 ? u == 0 : gq == 0;
      // v - a as fma(v, 1, -a): the same value (v * 1 exact, one rounding), and with the 1 in a
      // register the compiler fuses the fp16 widening into it (one v_fma_mix_f32)
      const int q = anc ? cg_quant_inv(v, s, is) : cg_quant_inv(__builtin_fmaf(v, one, -a), w, iw);
      const int sym = q + 127;
      if (anc) {   // coded in the anchor pass; here only the base of the group's deltas
        a = (float)q * s;
        clo[u] = 0u;
        chi[u] = 0u;
      } else if constexpr (kWin) {
        // sc = sym clamped so that sc and sc + 1 lie in the window. Every frequency from sc
        // out to sym is 1 (below the window cum[i] = i up to the first other frequency, above
        // it cum[i] = 65281 + i from past the last one), so cum[sym] = cum[sc] + (sym - sc) and
        // cum[sym + 1] = cum[sc + 1] + (sym - sc) exactly, inside the window too (sym = sc)
        const int sc = min(max(sym, wk0), wk1 - 1);
        const uint32_t dsym = (uint32_t)(sym - sc);
        clo[u] = (uint32_t)tabD[sc] + dsym;
        chi[u] = (uint32_t)tabD[sc + 1] + dsym;
        chi[u] = sym == CG_NSYM - 1 ? CG_TOTAL : chi[u];
      } else {
        // entry 255 of a staged table is its padding: read for the top symbol, then replaced
        clo[u] = tabD[sym];
        chi[u] = tabD[sym + 1];
        chi[u] = sym == CG_NSYM - 1 ? CG_TOTAL : chi[u];
      }
      if (kG == 0) gq = (gq + 1 == P.G) ? 0 : gq + 1;
    }
  };
  auto load_rows = [&](uint32_t (&xv)[kPipe], int step) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < kPipe; ++u) xv[u] = x[(int64_t)min(step * kPipe + u, last) * rs];
  };
  // a step without branches per symbol; if a lane of the wave owed more than 32 bits at some
  // symbol, the wave codes the step again from the saved state with the branching coder
  // code[u] (uniform) says whether position u of the buffer is coded in this step
  // positions [B, E) of the buffers (at most five symbols: the ring bound)
  auto code_run = [&](const auto& clo, const auto& chi, const bool* code, auto B, auto E)
                      __attribute__((always_inline)) {
    constexpr int kB = decltype(B)::value, kE = decltype(E)::value;
    static_assert(kE - kB <= 5, "a run codes at most five symbols");
    const EncState e0 = e;
    const uint64_t acc0 = o.acc;
    const uint32_t nacc0 = o.nacc, nwords0 = o.nwords;
    bool rare = false;
#pragma unroll
    for (int u = kB; u < kE; ++u)
      if (code[u]) enc_symbol_fast(e, o, clo[u], chi[u], rare);
    if (__builtin_amdgcn_ballot_w64(rare) != 0ull) {
      e = e0;
      o.acc = acc0;
      o.nacc = nacc0;
      o.nwords = nwords0;
#pragma unroll
      for (int u = kB; u < kE; ++u)
        if (code[u]) enc_symbol(e, o, clo[u], chi[u]);
    }
  };
  // a whole buffer of K positions in two runs, with a flush between them
  auto code_halves = [&](const auto& clo, const auto& chi, const bool* code)
                         __attribute__((always_inline)) {
    constexpr int K = sizeof(clo) / sizeof(clo[0]);
    constexpr int H = K / 2;
    code_run(clo, chi, code, std::integral_constant<int, 0>{}, std::integral_constant<int, H>{});
    o.flush();
    code_run(clo, chi, code, std::integral_constant<int, H>{}, std::integral_constant<int, K>{});
  };
  // the deltas of a step of the token pipeline (its anchors were coded in the anchor pass)
  auto code_step = [&](const uint32_t (&clo)[kPipe], const uint32_t (&chi)[kPipe], int step)
                       __attribute__((always_inline)) {
    bool code[kPipe];
    const int g0 = kG > 0 ? 0 : (step * kPipe) % P.G;
#pragma unroll
    for (int u = 0; u < kPipe; ++u) {
      const bool anc = kG > 0 ? u == 0 : (g0 + u) % P.G == 0;
      code[u] = step * kPipe + u < n && !anc;
    }
    code_halves(clo, chi, code);
  };

  // Anchor pass: the anchors of the chunk in token order (they come first in the stream), in
  // steps of kPipeA with the same two-step pipeline (rows two steps ahead, anchor-table
  // entries, from the anchor tables staged in LDS, one step ahead)
  if (lane_ok) {
    constexpr int kPipeA = 8;
    const int G = kG > 0 ? kG : P.G;
    const int na = (n + G - 1) / G;
    uint32_t ya0[kPipeA], ya1[kPipeA], la0[kPipeA], ha0[kPipeA], la1[kPipeA], ha1[kPipeA];
    auto load_anchor_rows = [&](uint32_t (&xv)[kPipeA], int step) __attribute__((always_inline)) {
#pragma unroll
      for (int u = 0; u < kPipeA; ++u)
        xv[u] = x[(int64_t)min(step * kPipeA + u, na - 1) * G * rs];
    };
    auto quantize_anchors = [&](const uint32_t (&xv)[kPipeA], uint32_t (&clo)[kPipeA],
                                uint32_t (&chi)[kPipeA]) __attribute__((always_inline)) {
#pragma unroll
      for (int u = 0; u < kPipeA; ++u) {
        const int sym = cg_quant_inv(cg_h2f((uint16_t)xv[u]), s, is) + 127;
        // both entries loaded unconditionally (a load under a condition would be waited for
        // at once), the top symbol's upper bound selected afterwards
        clo[u] = tabA[sym];
        chi[u] = tabA[sym + 1];   // entry 255 (padding) for the top symbol, then replaced
        chi[u] = sym == CG_NSYM - 1 ? CG_TOTAL : chi[u];
      }
    };
    auto code_anchors = [&](const uint32_t (&clo)[kPipeA], const uint32_t (&chi)[kPipeA],
                            int step) __attribute__((always_inline)) {
      bool code[kPipeA];
#pragma unroll
      for (int u = 0; u < kPipeA; ++u) code[u] = step * kPipeA + u < na;
      code_halves(clo, chi, code);
    };
    load_anchor_rows(ya0, 0);
    load_anchor_rows(ya1, 1);
    quantize_anchors(ya0, la0, ha0);
    load_anchor_rows(ya0, 2);
    for (int st = 0; st * kPipeA < na; st += 2) {
      bool ff;
      uint4 fv = o.flush_read(ff);
      quantize_anchors(ya1, la1, ha1);
      o.flush_store(fv, ff);
      load_anchor_rows(ya1, st + 3);
      code_anchors(la0, ha0, st);
      set_priority(max(na - (st + 1) * kPipeA, 0));
      if ((st + 1) * kPipeA >= na) break;
      fv = o.flush_read(ff);
      quantize_anchors(ya0, la0, ha0);
      o.flush_store(fv, ff);
      load_anchor_rows(ya0, st + 4);
      code_anchors(la1, ha1, st + 1);
      set_priority(max(na - (st + 2) * kPipeA, 0));
    }
  }
  // the delta pass: a software pipeline over steps of kPipe tokens (rows two steps ahead,
  // table entries one step ahead), then the termination and the stream's word count
  auto delta_pass = [&]() __attribute__((always_inline)) {
  uint32_t xr0[kPipe], xr1[kPipe], lo0[kPipe], hi0[kPipe], lo1[kPipe], hi1[kPipe];
  load_rows(xr0, 0);
  load_rows(xr1, 1);
  quantize_step(xr0, lo0, hi0);
  load_rows(xr0, 2);
  for (int st = 0; st * kPipe < n; st += 2) {
    // step st: quantize step st+1, request the rows of step st+3, code step st
    bool ff;
    uint4 fv = o.flush_read(ff);
    quantize_step(xr1, lo1, hi1);
    o.flush_store(fv, ff);
    load_rows(xr1, st + 3);
    code_step(lo0, hi0, st);
    if ((st + 1) * kPipe >= n) break;
    // step st+1: the same with the sets exchanged
    fv = o.flush_read(ff);
    quantize_step(xr0, lo0, hi0);
    o.flush_store(fv, ff);
    load_rows(xr0, st + 4);
    code_step(lo1, hi1, st + 1);
    set_priority(max(n - (st + 2) * kPipe, 0));   // once per two steps (every step: ~1.5 % slower)
  }
  enc_finish(e, o);
  // the coder's bound for n symbols; the compaction never writes past the sum of these
  const uint32_t own_bound = (uint32_t)((18ull * (uint64_t)n + 2ull + 31ull) / 32ull);
  lens[sidx] = min(o.nwords, min(own_bound, slot_words));
  };

  // the delta tables replace the anchor tables (in rounds when windows of all sets do not fit a
  // unit's region at once: every wave takes part in every round's staging and barriers, and
  // codes in its set's round)
  __syncthreads();
  if (threadIdx.x == 0) wflags[blockIdx.x] = s_bad;   // every workgroup writes its flag
  int nrounds = 1;
  if constexpr (kWin) {
    for (int uu = 0; uu < nu; ++uu) nrounds = max(nrounds, (int)s_nrounds[uu]);
    nrounds = __builtin_amdgcn_readfirstlane(nrounds);
  }
  const int set = active ? (int)s_set_of_level[u][lv] : 0;
  // this wave's round (past the last one: no coding); the rounds before and after it only
  // stage and wait, so that the coding runs outside any loop
  const int myr = __builtin_amdgcn_readfirstlane(
      !active ? nrounds : (kWin ? (int)s_round[u][set] : 0));
  auto round_stage = [&](int rd) __attribute__((always_inline)) {
    if (rd > 0) __syncthreads();   // the previous round's readers are done
    if constexpr (kWin) stage_round(rd);
    else stage(false);
    __syncthreads();
  };
  for (int rd = 0; rd < myr; ++rd) round_stage(rd);
  if (myr >= nrounds) return;
  round_stage(myr);
  if constexpr (kWin) {
    const uint32_t d = desc[(u * nsets_lds + set) * 64 + (lane_ok ? lane : 0)];
    wk0 = 16 * (int)((d >> 20) & 15u);
    wk1 = 16 * ((int)((d >> 24) & 15u) + 1);
    tabD = (cg_lds_u16*)(tabs + u * ustride + (d & 0xFFFFFu) / 2) - wk0;
  } else {
    tabD = (cg_lds_u16*)(tabs + u * ustride + (set * 64 + lane) * kEncTabStride);
  }
  if (lane_ok) delta_pass();
  for (int rd = myr + 1; rd < nrounds; ++rd) round_stage(rd);
}

// Block reduction helper: sum of one value per thread of a 256-thread block.
__device__ __forceinline__ uint64_t block_sum(uint64_t v, uint64_t* sh) {
  v = cg_wave_sum<uint64_t>(v);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
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

// Exclusive scan of nb block totals in place, by one workgroup. With `status` given, also the
// OR of the encode workgroups' n_wg non-finite flags into *status (written unconditionally, so
// no clearing is needed between calls).
__global__ __launch_bounds__(kScanThreads) void scan_top(uint64_t* __restrict__ partial,
                                                         int64_t nb,
                                                         const uint32_t* __restrict__ wflags,
                                                         int64_t n_wg,
                                                         uint32_t* __restrict__ status) {
  __shared__ uint64_t sh[kScanThreads / 64];
  if (status) {
    uint32_t bad = 0u;
    for (int64_t i = threadIdx.x; i < n_wg; i += kScanThreads) bad |= wflags[i];
    bad = __syncthreads_or(bad != 0u);
    if (threadIdx.x == 0) *status = bad ? 1u : 0u;
  }
  const int64_t per = (nb + kScanThreads - 1) / kScanThreads;
  const int64_t begin = threadIdx.x * per;
  const int64_t end = min(begin + per, nb);
  uint64_t local = 0;
  for (int64_t i = begin; i < end; ++i) local += partial[i];
  // exclusive scan of the thread totals across the block
  const uint64_t incl = cg_wave_incl_scan64(local);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
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
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
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

// ---- token-parallel layout (Sec. 6: the paper's decoder runs one thread per token) -----------
// One stream per (context, layer, K/V, token) over the token's channels, each symbol coded under
// its channel's table (anchor table on a group's first token, the chunk level's delta table
// otherwise). Quantization and scales are those of the channel layout. Inside context b, chunk
// c (first token t0, n tokens) holds the streams (b T + t0) 2L + (2 l + k) n + (t - t0).

// Symbols of every channel stream (the channel layout's quantizer and scales) into
// sym [B][L][2][T][C]: one wave per (context, chunk, layer, K/V, 64-channel block), a lane per
// channel; each token row is one coalesced 128-byte read and 64-byte write.
__global__ __launch_bounds__(256) void tok_quantize_kernel(KParams P, const uint16_t* __restrict__ kv,
                                                           const uint8_t* __restrict__ chunk_level,
                                                           uint8_t* __restrict__ sym,
                                                           float* __restrict__ scales) {
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
  const int64_t rs = P.C;
  const uint16_t* x = kv + cg_elem(P, b, l, k, t0, ch);
  float m = 0.0f;
  for (int j = 0; j < n; ++j) m = fmaxf(m, fabsf(cg_h2f(x[(int64_t)j * rs])));
  const float s = (m == 0.0f) ? 1.0f : m / 127.0f;
  scales[cg_stream(P, (((int64_t)b * P.NC + c) * P.L + l) * 2 + k, ch)] = s;
  const int lv = min((int)chunk_level[(int64_t)b * P.NC + c], P.NLV - 1);
  const float bw = P.layer_bin[l] * P.level_mult[lv];
  const float w = bw * s;
  const float is = 1.0f / s, iw = 1.0f / w;
  uint8_t* out = sym + cg_elem(P, b, l, k, t0, ch);
  float a = 0.0f;
  int g = 0;
  for (int j = 0; j < n; ++j) {
    const float v = cg_h2f(x[(int64_t)j * rs]);
    int q;
    if (g == 0) {
      q = cg_quant_inv(v, s, is);
      a = (float)q * s;
    } else {
      q = cg_quant_inv(v - a, w, iw);
    }
    out[(int64_t)j * rs] = (uint8_t)(q + 127);
    g = (g + 1 == P.G) ? 0 : g + 1;
  }
}

// Code the token streams: one wave per slot group (64 consecutive tokens of one context, chunk,
// layer and K/V), a lane per token, the channel layout's coder over the token's channels. Lanes
// past the chunk's last token code a copy of the last token (read in bounds, never recorded).
__global__ __launch_bounds__(256) void tok_encode_kernel(KParams P, const uint8_t* __restrict__ sym,
                                                         const uint8_t* __restrict__ chunk_level,
                                                         const uint16_t* __restrict__ cdfA,
                                                         const uint16_t* __restrict__ cdfD,
                                                         uint32_t* __restrict__ slots,
                                                         uint32_t slot_words,
                                                         uint32_t* __restrict__ lens, int nbj,
                                                         int64_t n_groups) {
  __shared__ uint32_t rings[4][kRing * 64];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int64_t grp = (int64_t)blockIdx.x * 4 + wave;
  if (grp >= n_groups) return;   // per wave; no workgroup barriers below
  const TokGroup g = tok_group(P, grp, nbj);
  if (g.jb * 64 >= g.n) return;  // a block past a short last chunk: no streams
  const int l = g.lk >> 1, k = g.lk & 1;
  const int t0 = g.c * P.CL;
  const int j = g.jb * 64 + lane;
  const bool valid = j < g.n;
  const int jl = valid ? j : g.n - 1;
  const bool anchor = jl % P.G == 0;
  const int lv = min((int)chunk_level[(int64_t)g.b * P.NC + g.c], P.NLV - 1);
  const uint8_t* row = sym + cg_elem(P, g.b, l, k, t0 + jl, 0);
  const uint16_t* tab = anchor ? cdfA + (int64_t)g.lk * P.C * 256
                               : cdfD + ((int64_t)lv * P.L * 2 + g.lk) * P.C * 256;
  EncState e{0u, 0xFFFFFFFFu, 0u};
  BitSink o{slots + (uint64_t)grp * slot_words * 64 + lane * 4, slot_words, 0u, 0u, 0ull, 0u,
            rings[wave] + lane};
  // steps of 8 symbols, flushed after every 4 (the ring bound of BitSink)
  constexpr int kStep = 8;
  for (int c0 = 0; c0 < P.C; c0 += kStep) {
    uint32_t lo[kStep], hi[kStep];
#pragma unroll
    for (int u = 0; u < kStep; ++u) {
      const int ch = min(c0 + u, P.C - 1);
      const int sy = row[ch];
      const uint16_t* t = tab + (int64_t)ch * 256;
      lo[u] = t[sy];
      hi[u] = sy == CG_NSYM - 1 ? CG_TOTAL : (uint32_t)t[sy + 1];
    }
#pragma unroll
    for (int u = 0; u < kStep; ++u) {
      if (c0 + u < P.C) enc_symbol(e, o, lo[u], hi[u]);
      if (u == kStep / 2 - 1) o.flush();   // runs of at most four symbols between flushes
    }
    o.flush();
  }
  enc_finish(e, o);
  const uint32_t own_bound = (uint32_t)((18ull * (uint64_t)P.C + 2ull + 31ull) / 32ull);
  if (valid) lens[tok_stream(P, g.b, g.c, g.lk, j, g.n)] = min(o.nwords, min(own_bound, slot_words));
}

// Copy every stream's words from its slot to their place in the payload. One workgroup per slot
// group of 64 streams: the slots of its streams are interleaved by 16-byte chunk, so tiles of
// chunks x 64 streams are read as whole 1 KB rows, transposed through LDS, and written as 16
// consecutive words per stream. Channel layout (kTok false): group = (row, 64-channel block),
// streams row * C + block * 64 + i. Token layout: group = (context, chunk, layer and K/V,
// 64-token block), streams tok_stream(...) of the block's tokens.
template <bool kTok>
__global__ __launch_bounds__(256) void compact_kernel(KParams P, const uint32_t* __restrict__ slots,
                                                      uint32_t slot_words,
                                                      const uint32_t* __restrict__ lens,
                                                      const uint64_t* __restrict__ offsets,
                                                      int nbj, uint32_t* __restrict__ words) {
  __shared__ uint32_t ctile[kCompactRows][65];
  __shared__ uint32_t s_len[64];
  __shared__ uint64_t s_off[64];
  __shared__ uint32_t s_max;
  const int64_t grp = blockIdx.x;
  int64_t base;   // stream of the group's lane 0
  int count;      // streams in the group
  if constexpr (kTok) {
    const TokGroup g = tok_group(P, grp, nbj);
    base = tok_stream(P, g.b, g.c, g.lk, g.jb * 64, g.n);
    count = min(64, g.n - g.jb * 64);
  } else {
    const int64_t row = grp / P.nblk;
    const int cb = (int)(grp - row * P.nblk);
    base = row * P.C + cb * 64;
    count = min(64, P.C - cb * 64);
  }
  const int t = threadIdx.x;
  if (t == 0) s_max = 0u;
  __syncthreads();
  if (t < 64) {
    uint32_t n = 0;
    uint64_t o = 0;
    if (t < count) {
      n = lens[base + t];
      o = offsets[base + t];
    }
    s_len[t] = n;
    s_off[t] = o;
    atomicMax(&s_max, n);
  }
  __syncthreads();
  const uint32_t K = s_max;
  const uint32_t* src = slots + (uint64_t)grp * slot_words * 64;
  // kCompactRows words of every stream per pass (kCompactRows / 4 chunk rows of 1 KB, a wave
  // reading whole rows): every thread has eight 16-byte loads in flight
  for (uint32_t k0 = 0; k0 < K; k0 += kCompactRows) {
    uint4 v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const uint32_t cr = (t >> 6) + 4 * i;   // chunk row of this pass: words 4 cr .. 4 cr + 3
      const uint32_t m = (k0 >> 2) + cr;      // chunk index in the slots
      v[i] = 4 * m < K ? *reinterpret_cast<const uint4*>(src + ((uint64_t)m * 64 + (t & 63)) * 4)
                       : make_uint4(0u, 0u, 0u, 0u);
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int cr = (t >> 6) + 4 * i;
      ctile[4 * cr + 0][t & 63] = v[i].x;
      ctile[4 * cr + 1][t & 63] = v[i].y;
      ctile[4 * cr + 2][t & 63] = v[i].z;
      ctile[4 * cr + 3][t & 63] = v[i].w;
    }
    __syncthreads();
#pragma unroll
    for (int pass = 0; pass < 32; ++pass) {   // 16 lanes write 16 consecutive words of a stream
      const int L = (pass & 3) * 16 + (t >> 4);
      const uint32_t kr = (pass >> 2) * 16 + (t & 15), k = k0 + kr;
      if (k < s_len[L]) words[s_off[L] + k] = ctile[kr][L];
    }
    __syncthreads();
  }
}

inline uint64_t align256(uint64_t x) { return (x + 255) & ~(uint64_t)255; }


// Launch geometry of encode_kernel: nw (context, chunk) pairs x nu units per workgroup, g1
// workgroups, lds bytes of dynamic LDS, nsets delta-table sets per unit.
struct EncGeom {
  int nw, nu, nsets;
  int64_t n_groups, g1;
  size_t lds;
  bool win;      // delta tables staged as windows (encode_kernel<kG, true>)
  int ustride;   // u16 per unit region
};

EncGeom enc_geometry(const KParams& P) {
  EncGeom g;
  const int64_t n_pairs = (int64_t)P.B * P.NC;
  int nw = (int)(n_pairs < kEncMaxWaves ? n_pairs : kEncMaxWaves);
  auto lds_for = [&](int w, int nu) {
    const int sets = w < P.NLV ? w : P.NLV;
    return (size_t)nu * sets * 64 * kEncTabStride * sizeof(uint16_t) +
           (size_t)nu * w * kRing * 64 * sizeof(uint32_t);
  };
  while (nw > 1 && lds_for(nw, 1) > kEncLdsBudget) --nw;
  const int64_t n_groups = (n_pairs + nw - 1) / nw;
  const int64_t n_units = (int64_t)P.L * 2 * P.nblk;
  // several units per workgroup while the grid still covers every CU
  int nu = 1;
  while (nu < kEncMaxUnits && (nu + 1) * nw <= kEncMaxWaves &&
         lds_for(nw, nu + 1) <= kEncLdsBudget && (n_units + nu) / (nu + 1) * n_groups >= 256)
    ++nu;
  g.nw = nw;
  g.nsets = nw < P.NLV ? nw : P.NLV;
  g.n_groups = n_groups;
  // With several levels the delta tables can be staged as windows: a unit then needs a region
  // of one whole table set (its anchor tables) plus its rings and window descriptors, so more
  // units fit a workgroup. Used when that allows more units.
  const size_t rings = (size_t)nw * kRing * 64 * sizeof(uint32_t);   // per unit
  const size_t set_bytes = (size_t)64 * kEncTabStride * sizeof(uint16_t);
  const size_t desc_bytes = (size_t)g.nsets * 64 * sizeof(uint32_t);
  int nuc = 1;
  while (nuc < kEncMaxUnits && (nuc + 1) * nw <= kEncWinWaves &&
         (size_t)(nuc + 1) * (rings + set_bytes + desc_bytes) <= kEncLdsBudget &&
         (n_units + nuc) / (nuc + 1) * n_groups >= 256)
    ++nuc;
  g.win = g.nsets > 1 && nuc > nu;
  if (g.win) {
    g.nu = nuc;
    const size_t per_unit = kEncLdsBudget / (size_t)nuc - rings - desc_bytes;
    g.ustride = (int)((per_unit & ~(size_t)15) / sizeof(uint16_t));
    g.lds = (size_t)nuc * (rings + desc_bytes) + (size_t)nuc * g.ustride * sizeof(uint16_t);
  } else {
    g.nu = nu;
    g.ustride = g.nsets * 64 * kEncTabStride;
    g.lds = lds_for(nw, nu);
  }
  g.g1 = cg_xcd_grid((n_units + g.nu - 1) / g.nu, n_groups);
  return g;
}

}  // namespace

// Workspace: the status word (offset 0, read by cg_get_status), the encode workgroups'
// non-finite flags, one worst-case slot per lane of every (row, 64-channel block) wave (lanes
// past C included), per-stream word counts, and the scan's block totals.
EncWorkspace cg_encode_ws_layout(const KParams& P, uint32_t slot_words) {
  EncWorkspace w;
  const int64_t S = P.S;
  const int64_t nb = (S + kScanBlock - 1) / kScanBlock;
  const uint64_t slot_lanes = (uint64_t)P.B * P.NC * P.L * 2 * P.nblk * 64;
  w.status_off = 0;
  w.wflags_off = 256;
  w.slots_off = align256(w.wflags_off + (uint64_t)enc_geometry(P).g1 * 4ull);
  w.lens_off = align256(w.slots_off + slot_lanes * slot_words * 4ull);
  w.partial_off = align256(w.lens_off + (uint64_t)S * 4ull);
  w.total = align256(w.partial_off + (uint64_t)(nb > 0 ? nb : 1) * 8ull);
  return w;
}

hipError_t cg_launch_encode(const KParams& P, const uint16_t* kv, const uint8_t* chunk_level,
                            const uint16_t* cdf_anchor, const uint16_t* cdf_delta,
                            uint32_t* words, uint64_t* offsets, float* scales, void* ws,
                            uint32_t slot_words, hipStream_t st, uint32_t* status_out,
                            bool scales_given) {
  const EncWorkspace lay = cg_encode_ws_layout(P, slot_words);
  uint8_t* base = static_cast<uint8_t*>(ws);
  uint32_t* status =
      status_out ? status_out : reinterpret_cast<uint32_t*>(base + lay.status_off);
  uint32_t* wflags = reinterpret_cast<uint32_t*>(base + lay.wflags_off);
  uint32_t* slots = reinterpret_cast<uint32_t*>(base + lay.slots_off);
  uint32_t* lens = reinterpret_cast<uint32_t*>(base + lay.lens_off);
  uint64_t* partial = reinterpret_cast<uint64_t*>(base + lay.partial_off);

  const EncGeom g = enc_geometry(P);
  const void* kfn = P.G == 10 ? (g.win ? (const void*)encode_kernel<10, true>
                                       : (const void*)encode_kernel<10, false>)
                              : (g.win ? (const void*)encode_kernel<0, true>
                                       : (const void*)encode_kernel<0, false>);
  hipError_t e =
      hipFuncSetAttribute(kfn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)g.lds);
  if (e != hipSuccess) return e;
  const dim3 grid((unsigned)g.g1), block(64 * g.nw * g.nu);
#define CG_ENCODE_LAUNCH(KG, KW)                                                              \
  hipLaunchKernelGGL((encode_kernel<KG, KW>), grid, block, g.lds, st, P, kv, chunk_level,     \
                     cdf_anchor, cdf_delta, slots, slot_words, lens, scales, wflags, g.nw,    \
                     g.nu, g.nsets, g.ustride, scales_given ? 1 : 0)
  if (P.G == 10) {
    if (g.win) CG_ENCODE_LAUNCH(10, true);
    else CG_ENCODE_LAUNCH(10, false);
  } else {
    if (g.win) CG_ENCODE_LAUNCH(0, true);
    else CG_ENCODE_LAUNCH(0, false);
  }
#undef CG_ENCODE_LAUNCH
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t nb = (P.S + kScanBlock - 1) / kScanBlock;
  hipLaunchKernelGGL(scan_reduce, dim3((unsigned)nb), dim3(kScanThreads), 0, st, lens, P.S,
                     partial);
  hipLaunchKernelGGL(scan_top, dim3(1), dim3(kScanThreads), 0, st, partial, nb,
                     (const uint32_t*)wflags, g.g1, status);
  hipLaunchKernelGGL(scan_finish, dim3((unsigned)nb), dim3(kScanThreads), 0, st, lens, P.S,
                     partial, offsets);
  const int64_t groups = (int64_t)P.B * P.NC * P.L * 2 * P.nblk;
  hipLaunchKernelGGL(compact_kernel<false>, dim3((unsigned)groups), dim3(256), 0, st, P, slots,
                     slot_words, lens, offsets, 0, words);
  return hipGetLastError();
}

// ---- token-parallel layout ----------------------------------------------------------------

int64_t cg_token_streams(const KParams& P) { return (int64_t)P.B * P.L * 2 * P.T; }

uint32_t cg_token_slot_words(const KParams& P) {   // whole 16-byte chunks
  return (uint32_t)(((18ull * (uint64_t)P.C + 2ull + 31ull) / 32ull + 3ull) & ~3ull);
}

TokEncWorkspace cg_encode_tokens_ws_layout(const KParams& P) {
  TokEncWorkspace w;
  const int64_t St = cg_token_streams(P);
  const int64_t nb = (St + kScanBlock - 1) / kScanBlock;
  const int nbj = (int)(((P.CL < P.T ? P.CL : P.T) + 63) / 64);
  w.nbj = nbj;
  w.n_groups = (int64_t)P.B * P.NC * 2 * P.L * nbj;
  w.sym_off = 0;
  w.slots_off = align256((uint64_t)St * P.C);
  w.lens_off = align256(w.slots_off + (uint64_t)w.n_groups * 64 * cg_token_slot_words(P) * 4ull);
  w.partial_off = align256(w.lens_off + (uint64_t)St * 4ull);
  w.total = align256(w.partial_off + (uint64_t)(nb > 0 ? nb : 1) * 8ull);
  return w;
}

hipError_t cg_launch_encode_tokens(const KParams& P, const uint16_t* kv,
                                   const uint8_t* chunk_level, const uint16_t* cdf_anchor,
                                   const uint16_t* cdf_delta, uint32_t* words, uint64_t* offsets,
                                   float* scales, void* ws, hipStream_t st) {
  const TokEncWorkspace lay = cg_encode_tokens_ws_layout(P);
  uint8_t* base = static_cast<uint8_t*>(ws);
  uint8_t* sym = base + lay.sym_off;
  uint32_t* slots = reinterpret_cast<uint32_t*>(base + lay.slots_off);
  uint32_t* lens = reinterpret_cast<uint32_t*>(base + lay.lens_off);
  uint64_t* partial = reinterpret_cast<uint64_t*>(base + lay.partial_off);
  const uint32_t slot_words = cg_token_slot_words(P);
  const int64_t items = (int64_t)P.B * P.NC * P.L * 2 * P.nblk;
  hipLaunchKernelGGL(tok_quantize_kernel, dim3((unsigned)((items + 3) / 4)), dim3(256), 0, st, P,
                     kv, chunk_level, sym, scales);
  hipLaunchKernelGGL(tok_encode_kernel, dim3((unsigned)((lay.n_groups + 3) / 4)), dim3(256), 0,
                     st, P, sym, chunk_level, cdf_anchor, cdf_delta, slots, slot_words, lens,
                     lay.nbj, lay.n_groups);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t St = cg_token_streams(P);
  const int64_t nb = (St + kScanBlock - 1) / kScanBlock;
  hipLaunchKernelGGL(scan_reduce, dim3((unsigned)nb), dim3(kScanThreads), 0, st, lens, St,
                     partial);
  hipLaunchKernelGGL(scan_top, dim3(1), dim3(kScanThreads), 0, st, partial, nb,
                     (const uint32_t*)nullptr, (int64_t)0, (uint32_t*)nullptr);
  hipLaunchKernelGGL(scan_finish, dim3((unsigned)nb), dim3(kScanThreads), 0, st, lens, St,
                     partial, offsets);
  hipLaunchKernelGGL(compact_kernel<true>, dim3((unsigned)lay.n_groups), dim3(256), 0, st, P,
                     slots, slot_words, lens, offsets, lay.nbj, words);
  return hipGetLastError();
}
