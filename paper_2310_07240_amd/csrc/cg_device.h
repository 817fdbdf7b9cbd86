// cg_device.h — device-side definitions shared by the codec's HIP kernels (gfx950).
//
// Kernel-side view of the codec parameters and the small helpers every kernel uses: fp16
// conversion, the quantizer (CacheGen Sec. 5.2, "Change-based encoding" and "Layer-wise
// quantization"), wave-level reductions, and the launchers the C ABI calls.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#define CG_MAX_LAYERS 512
#define CG_MAX_LEVELS 8
#define CG_NSYM 255
#define CG_TOTAL 65536u

// Table pointers typed by address space. Where one expression may read either an LDS table or a
// global one, the loads stay separate LDS and global loads instead of being merged into one
// generic (flat) load through a selected pointer: such a load costs more, and its base (before
// the instruction's immediate offset) can fall outside the LDS aperture, which faults.
typedef __attribute__((address_space(3))) const uint16_t cg_lds_u16;
typedef __attribute__((address_space(1))) const uint16_t cg_glb_u16;

// Parameters as the kernels see them. Passed by value (kernel argument segment, < 4 KiB).
struct KParams {
  int32_t B, L, T, C;      // contexts, layers, tokens, channels per K and per V
  int32_t G, CL, NC, NLV;  // group size, chunk length, chunks, levels
  int32_t nblk;            // 64-channel blocks per (b, c, l, kv) = ceil(C / 64)
  int32_t pad_;
  int64_t S;               // streams
  float layer_bin[CG_MAX_LAYERS];
  float level_mult[CG_MAX_LEVELS];
};

// Relaxed LDS accesses of a value other waves of the workgroup update (no ordering, no wait
// beyond the LDS access itself).
__device__ __forceinline__ int lds_get(int* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ void lds_put(int* p, int v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

__device__ __forceinline__ float cg_h2f(uint16_t h) {
  return (float)__builtin_bit_cast(_Float16, h);               // exact widening
}

__device__ __forceinline__ uint16_t cg_f2h(float f) {
  return __builtin_bit_cast(uint16_t, (_Float16)f);            // round to nearest even
}

// Quantize v by step `step` to an integer in [-127, 127]: rint(clamp(v / step)). The division
// is the correctly rounded IEEE one (the library is built without fast-math), rint rounds half
// to even.
__device__ __forceinline__ int cg_quant(float v, float step) {
  float r = v / step;
  r = fminf(fmaxf(r, -127.0f), 127.0f);
  return (int)__builtin_rintf(r);
}

// The same quantizer through a reciprocal: inv = 1 / step, correctly rounded (computed once
// per stream). r = v * inv is within |q|(2^-23 + 2^-48) of the exact quotient q = v / step,
// and the correctly rounded quotient within |q| 2^-24 of q, so below |r| = 127 they differ by
// less than 2.3e-5. rint(clamp(.)) only changes value at the half-integers k + 0.5 inside
// (-127, 127) (ties round to even), so when the clamped r is farther than 2^-14 from every
// half-integer, r and the correctly rounded quotient give the same integer; otherwise (about
// one value in 8000) the division is done as above. Clamped values (|r| >= 127) are 0.5 from
// the nearest half-integer and give +-127 either way. The distance to the nearest half-integer
// is 0.5 - |r - rint(r)| (exact: |r| < 2^23). The division sits behind a wave-uniform test, so
// the wave branches over it unless one of its lanes is that close to a half-integer (under 1 %
// of the waves); written as a plain branch, the compiler evaluates it on every call.
__device__ __forceinline__ int cg_quant_inv(float v, float step, float inv) {
  const float r = __builtin_amdgcn_fmed3f(v * inv, -127.0f, 127.0f);
  const float rn = __builtin_rintf(r);
  int q = (int)rn;
  const bool near_half = __builtin_fabsf(r - rn) >= 0.5f - 0x1p-14f;
  if (__builtin_expect(__builtin_amdgcn_ballot_w64(near_half) != 0, 0)) {
    if (near_half) q = cg_quant(v, step);
  }
  return q;
}

// Stream index of (b, c, l, kv, ch): chunk-major so each chunk's streams are contiguous.
__device__ __forceinline__ int64_t cg_stream(const KParams& P, int64_t bclk, int ch) {
  return bclk * P.C + ch;
}

// Element offset of token t, channel ch in the [B][L][2][T][C] tensor for row group (b, l, kv).
__device__ __forceinline__ int64_t cg_elem(const KParams& P, int b, int l, int k, int64_t t,
                                           int ch) {
  return ((((int64_t)b * P.L + l) * 2 + k) * P.T + t) * P.C + ch;
}

// Token-parallel layout: a group of 64 consecutive token streams is (context b, chunk c,
// lk = 2 l + k, block jb of 64 tokens), nbj blocks per (b, c, lk) (enough for the longest
// chunk); n = tokens of chunk c. Inside context b, chunk c (first token t0) holds the streams
// (b T + t0) 2L + lk n + (t - t0).
struct TokGroup {
  int b, c, lk, jb, n;
};

__device__ __forceinline__ TokGroup tok_group(const KParams& P, int64_t grp, int nbj) {
  TokGroup g;
  g.jb = (int)(grp % nbj);
  int64_t r = grp / nbj;
  g.lk = (int)(r % (2 * P.L));
  r /= 2 * P.L;
  g.c = (int)(r % P.NC);
  g.b = (int)(r / P.NC);
  g.n = P.CL < P.T - g.c * P.CL ? P.CL : P.T - g.c * P.CL;
  return g;
}

__device__ __forceinline__ int64_t tok_stream(const KParams& P, int b, int c, int lk, int j,
                                              int n) {
  return ((int64_t)b * P.T + (int64_t)c * P.CL) * (2 * P.L) + (int64_t)lk * n + j;
}

// Workgroup -> (unit block, pair group) for grids of n_ublk unit blocks x n_groups pair groups.
// Workgroups are dispatched in block order, each as soon as a CU of its XCD can take it, and the
// hardware deals them to the 8 XCDs in turn (block i to XCD i mod 8). Blocks go pair group by
// pair group: pair groups follow chunk order, so the workgroups of the long chunks start first
// and those of a short last chunk fill in at the end (with the pair group as the fastest index,
// a CU that finished a short workgroup waited for the next long one ahead of its own in the
// queue). Unit blocks are numbered to a multiple of 8 per pair group, so all pair groups of a
// unit block run on one XCD (its tables stay in that XCD's L2); blocks past n_ublk must leave.
__device__ __forceinline__ void cg_xcd_map(int n_ublk, int n_groups, int& ublk, int& grp) {
  const int pad = n_groups == 1 ? n_ublk : (n_ublk + 7) / 8 * 8;
  const int b = (int)blockIdx.x;
  grp = b / pad;
  ublk = b - grp * pad;
}
inline int64_t cg_xcd_grid(int64_t n_ublk, int64_t n_groups) {
  return n_groups == 1 ? n_ublk : (n_ublk + 7) / 8 * 8 * n_groups;
}

// Window of a cumulative table held by 32 lanes of a wave, 16 bytes (8 entries) each: piece p
// holds cum[8 p .. 8 p + 7] in v (the other half of the wave may hold another table). Returns
// in lo / hi the first and the last symbol i in [0, 254] whose frequency cum[i + 1] - cum[i] is
// not 1 (entry 255 is padding; the total 65536 stands in for it), the same in all 32 lanes. A
// table without such a frequency (not a valid table) gives [0, 254]. Every frequency outside
// [lo, hi] is 1, so cum[i] = i for i <= lo and cum[i] = 65281 + i for i > hi.
__device__ __forceinline__ void cg_table_window(const uint4& v, int piece, int& lo, int& hi) {
  const uint32_t e0 = v.x & 0xFFFFu, e1 = v.x >> 16, e2 = v.y & 0xFFFFu, e3 = v.y >> 16;
  const uint32_t e4 = v.z & 0xFFFFu, e5 = v.z >> 16, e6 = v.w & 0xFFFFu;
  const uint32_t e7 = piece == 31 ? CG_TOTAL : v.w >> 16;
  const uint32_t e8 = (uint32_t)__shfl_down((int)e0, 1, 32);   // the next lane's first entry
  const uint32_t e[9] = {e0, e1, e2, e3, e4, e5, e6, e7, e8};
  lo = 255;
  hi = -1;
#pragma unroll
  for (int jj = 7; jj >= 0; --jj)
    if (8 * piece + jj < CG_NSYM && e[jj + 1] - e[jj] != 1u) lo = 8 * piece + jj;
#pragma unroll
  for (int jj = 0; jj < 8; ++jj)
    if (8 * piece + jj < CG_NSYM && e[jj + 1] - e[jj] != 1u) hi = 8 * piece + jj;
#pragma unroll
  for (int o = 16; o >= 1; o >>= 1) {
    lo = min(lo, __shfl_xor(lo, o, 32));
    hi = max(hi, __shfl_xor(hi, o, 32));
  }
  if (hi < lo) {
    lo = 0;
    hi = CG_NSYM - 1;
  }
}

// The 16-entry blocks g0 .. g1 a window keeps: the blocks holding lo and hi extended by one
// block on each side (g1 > g0), and its size in bytes: entries 16 g0 .. 16 (g1 + 1) + 3.
__device__ __forceinline__ uint32_t cg_window_desc(int lo, int hi) {
  const int g0 = max(lo / 16 - 1, 0), g1 = min(hi / 16 + 1, 15);
  return (uint32_t)g0 | ((uint32_t)g1 << 4) | ((uint32_t)((g1 - g0 + 1) * 32 + 8) << 8);
}

template <typename T>
__device__ __forceinline__ T cg_wave_sum(T v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Inclusive prefix sum across the 64 lanes of a wave.
__device__ __forceinline__ uint32_t cg_wave_incl_scan(uint32_t v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    uint32_t n = __shfl_up(v, o, 64);
    if (lane >= o) v += n;
  }
  return v;
}

__device__ __forceinline__ uint64_t cg_wave_incl_scan64(uint64_t v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    uint64_t n = __shfl_up(v, o, 64);
    if (lane >= o) v += n;
  }
  return v;
}

// Launchers (return hipError_t of the launch).
// scales, if not null: receives every stream's scale s (the encoder's value for the same KV).
hipError_t cg_launch_fit(const KParams& P, const uint16_t* kv, int level, uint16_t* cdf_anchor,
                         uint16_t* cdf_delta_level, hipStream_t st, float* scales = nullptr);
// Every level's tables in as few passes as 16-bit counts allow (see cg_fit.hip); status, if not
// null, receives 0 or 1 (NaN or Inf in the KV); scales as for cg_launch_fit.
hipError_t cg_launch_fit_levels(const KParams& P, const uint16_t* kv, uint16_t* cdf_anchor,
                                uint16_t* cdf_delta, uint32_t* status, float* scales,
                                hipStream_t st);
int64_t cg_fit_max_count(const KParams& P);
hipError_t cg_launch_fit_global(const KParams& P, const uint16_t* kv, int level,
                                uint16_t* cdf_anchor, uint16_t* cdf_delta_level, void* ws,
                                hipStream_t st);
// status_out: where the non-finite status word goes (nullptr: the workspace's first word).
// scales_given: scales holds every stream's scale on entry (the encoder then takes no absolute
// maxima and checks no finiteness); otherwise it receives them.
hipError_t cg_launch_encode(const KParams& P, const uint16_t* kv, const uint8_t* chunk_level,
                            const uint16_t* cdf_anchor, const uint16_t* cdf_delta,
                            uint32_t* words, uint64_t* offsets, float* scales, void* ws,
                            uint32_t slot_words, hipStream_t st, uint32_t* status_out = nullptr,
                            bool scales_given = false);
hipError_t cg_launch_decode(const KParams& P, const uint32_t* words, const uint64_t* offsets,
                            const float* scales, const uint8_t* chunk_level,
                            const uint16_t* cdf_anchor, const uint16_t* cdf_delta, int c_begin,
                            int c_end, uint16_t* out, hipStream_t st);
hipError_t cg_launch_check_finite(const uint16_t* kv, int64_t n, uint32_t* flag, hipStream_t st);

// Workspace layout of cg_encode (byte offsets, 256-aligned). The status word sits at offset 0.
struct EncWorkspace {
  uint64_t status_off, wflags_off, slots_off, lens_off, partial_off, total;
};
EncWorkspace cg_encode_ws_layout(const KParams& P, uint32_t slot_words);

// Token-parallel stream layout: one stream per (context, layer, K/V, token) over the token's
// channels (streams in chunk-major order; see cg_encode.hip).
int64_t cg_token_streams(const KParams& P);
uint32_t cg_token_slot_words(const KParams& P);   // worst-case words of one token stream
struct TokEncWorkspace {
  uint64_t sym_off, slots_off, lens_off, partial_off, total;
  int64_t n_groups;   // slot groups of 64 token streams
  int nbj;            // 64-token blocks per (context, chunk, layer, K/V)
};
TokEncWorkspace cg_encode_tokens_ws_layout(const KParams& P);
hipError_t cg_launch_encode_tokens(const KParams& P, const uint16_t* kv,
                                   const uint8_t* chunk_level, const uint16_t* cdf_anchor,
                                   const uint16_t* cdf_delta, uint32_t* words, uint64_t* offsets,
                                   float* scales, void* ws, hipStream_t st);
hipError_t cg_launch_decode_tokens(const KParams& P, const uint32_t* words,
                                   const uint64_t* offsets, const float* scales,
                                   const uint8_t* chunk_level, const uint16_t* cdf_anchor,
                                   const uint16_t* cdf_delta, uint8_t* sym, uint16_t* out,
                                   hipStream_t st);
