/*
 * cachegen.h — C ABI of the CacheGen KV-cache codec for AMD Instinct MI355X (gfx950).
 *
 * The codec (CacheGen, SIGCOMM '24, Sec. 5.2 "KV cache encoding") turns an fp16 KV cache into
 * compact bitstreams in four steps, and decodes them back:
 *   1. token groups of G consecutive tokens; the first token of a group is the anchor and is
 *      quantized on its own at 8 bits, the others are coded as a delta against that anchor
 *      (Sec. 5.2 "Change-based encoding"; 8-bit anchors: Sec. 5.2 "Layer-wise quantization");
 *   2. vectorwise quantization whose delta bin width grows with layer depth
 *      (Sec. 5.2 "Layer-wise quantization"; default bins 0.5 / 1 / 1.5: App. C.2), with an
 *      encoding level chosen per context chunk (Sec. 5.3 "Workflow");
 *   3. one symbol distribution per (layer, K/V, channel) for deltas and one for anchors,
 *      counted over the context (Sec. 5.2 "Arithmetic coding"; Sec. 6 "Speed optimization");
 *   4. arithmetic coding of the symbols into bitstreams, and GPU arithmetic decoding back to
 *      fp16 KV (Sec. 5.2 "Arithmetic coding"; Sec. 6 "Speed optimization").
 *
 * Conventions shared by every call
 * --------------------------------
 *  B = n_ctx contexts, L = n_layers, T = n_tokens, C = n_channels per K and per V.
 *  KV layout (fp16 bit patterns, uint16_t): kv[b][l][kv][t][ch], kv = 0 for K and 1 for V,
 *  channel fastest. Element count n_elem = B*L*2*T*C (64-bit).
 *  Chunks: tokens are split into NC = ceil(T/chunk_len) chunks; the last may be partial.
 *  Token groups restart at every chunk start (chunks decode independently, Sec. 5.3).
 *  One arithmetic-coder stream per (b, c, l, kv, ch) with stream index
 *      s = (((b*NC + c)*L + l)*2 + kv)*C + ch        (S = B*NC*L*2*C streams)
 *  so every chunk's streams are contiguous in the payload. Inside a stream the chunk's anchor
 *  symbols come first, in token order, then its delta symbols, in token order (Sec. 5.2 fixes
 *  what is coded and under which distribution, not the order inside one bitstream; anchors
 *  first lets a decoder take every anchor, then every delta, with one table set at hand).
 *  Symbols: a quantized value q in [-127, 127] is symbol q + 127 in [0, 254] (255 symbols).
 *  Scale (per stream): m = max |x| over the chunk's tokens; s = (m == 0) ? 1 : m / 127 (fp32).
 *  Anchor (token j of a chunk with j % G == 0): q = rint(clamp(x / s, -127, 127)); a = q * s.
 *  Delta (other tokens): w = (layer_bin[l] * level_mult[level]) * s; d = x - a;
 *                        q = rint(clamp(d / w, -127, 127)).
 *  Reconstruction: anchor fp16(a); delta fp16(a + q * w). All fp32 arithmetic is IEEE
 *  binary32, round-to-nearest-even, no fused multiply-add; fp16 conversion rounds to nearest even.
 *
 *  CDF tables: uint16_t cum[256] per distribution with cum[0] = 0, cum[i+1] = cum[i] + freq[i]
 *  for i in [0, 253], every freq >= 1, total 65536. Entry 255 is padding (written 0); the
 *  top of the last interval, 65536, is implicit.
 *    cdf_anchor[l][kv][ch][256]                       (level independent)
 *    cdf_delta [level][l][kv][ch][256]                (one table set per encoding level)
 *
 *  Bitstreams: integer arithmetic coder with 32-bit code registers (Witten, Neal and Cleary,
 *  CACM 30(6), 1987), bitwise renormalisation, 2-bit termination. Bits are written MSB-first
 *  into uint32_t words; each stream is zero-padded to a whole word. offsets[0] = 0 and
 *  offsets[s+1] = offsets[s] + (words of stream s), uint64_t, so stream s occupies
 *  words[offsets[s] .. offsets[s+1]).
 *
 *  Memory: every array argument is a DEVICE pointer owned by the caller, except cg_params and
 *  the arrays it points to, which are HOST memory read during the call only. The library
 *  keeps no state between calls and never allocates device memory; scratch comes from the
 *  caller's workspace argument. Calls are asynchronous on the given HIP stream unless a
 *  description says otherwise; a non-zero return means nothing was launched, except
 *  CG_ERR_HIP, which reports a failed launch.
 */
#ifndef CACHEGEN_H
#define CACHEGEN_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Return codes. */
enum {
  CG_OK = 0,
  CG_ERR_ARG = -1,        /* null or misaligned pointer (tables need 16-byte alignment,
                             offsets 8, words and scales 4, the workspace 256), level or
                             chunk range out of range                                       */
  CG_ERR_SHAPE = -2,      /* a dimension <= 0, group_size < 1, chunk_len < 1, n_levels not
                             in [1, 8], or a size whose index space overflows 64 bits       */
  CG_ERR_CAPACITY = -3,   /* words_cap or workspace_bytes below what the call needs        */
  CG_ERR_NONFINITE = -4,  /* the KV input holds NaN or +-Inf (reported by cg_get_status after
                             cg_encode or cg_fit_cdf_levels, and by cg_check_finite)        */
  CG_ERR_HIP = -5,        /* a HIP runtime call or kernel launch failed                     */
  CG_ERR_PARAM = -6,      /* a layer_bin or level_mult entry is not finite and > 0          */
  CG_ERR_SCRATCH = -7     /* cg_encode_noalloc: the cache needs more scratch than
                             CG_NOALLOC_SCRATCH_BYTES                                       */
};

/* cg_decode may read (but never uses) up to this many words past offsets[S]: a words buffer
 * handed to cg_decode must be readable that far. A buffer sized by cg_encode_bound_words is. */
#define CG_TAIL_WORDS 8

typedef struct cg_params {
  int32_t n_ctx;          /* B */
  int32_t n_layers;       /* L */
  int32_t n_tokens;       /* T */
  int32_t n_channels;     /* C = kv_heads * head_dim, the same for K and V */
  int32_t group_size;     /* G, tokens per group, 10 in the paper (Sec. 5.2) */
  int32_t chunk_len;      /* tokens per chunk, 1.5K in the paper (Sec. 5.3); 1536 here */
  int32_t n_levels;       /* number of encoding levels, 1..8 */
  const float* layer_bin; /* [L] base delta bin width per layer in units of the scale s
                             (three layer groups 0.5 / 1 / 1.5 by default, App. C.2)    */
  const float* level_mult;/* [n_levels] multiplier of the bin width per encoding level */
} cg_params;

/* Number of chunks NC and of streams S for these parameters; 0 if the shape is invalid. */
int64_t cg_num_chunks(const cg_params* p);
int64_t cg_num_streams(const cg_params* p);

/* Capacity (in words) that cg_encode requires for its payload buffer: the sum over streams of
 * ceil((18 * n_s + 2) / 32), n_s being the stream's token count (each symbol costs at most 18
 * renormalisation shifts and the termination 2 bits), plus CG_TAIL_WORDS. 0 if the shape is
 * invalid. */
uint64_t cg_encode_bound_words(const cg_params* p);

/* Device scratch that cg_encode needs (bytes): the status word, per-workgroup non-finite
 * flags, a worst-case slot per stream, per-stream lengths and the scan's partial sums. 0 if the
 * shape is invalid. */
uint64_t cg_encode_workspace_bytes(const cg_params* p);

/* Fit the symbol distributions at encoding level `level` (Sec. 5.2 "Arithmetic coding":
 * one distribution per layer-channel for deltas and one for anchors; Sec. 6: counted over the
 * symbols of the context being coded).
 *   kv_f16          [B][L][2][T][C] fp16, device.
 *   level           0 <= level < n_levels: deltas of EVERY chunk are quantized with
 *                   level_mult[level] for this fit.
 *   cdf_anchor      out [L][2][C][256], device; may be NULL to skip the anchor tables.
 *   cdf_delta_level out [L][2][C][256], device: the delta tables of this level, i.e. the
 *                   slice cdf_delta[level] of the layout above.
 * Counts c_i (i in [0, 254]) are taken over all B*NC chunks; with N = sum c_i,
 * freq_i = 1 + floor(c_i * 65281 / N), and the remainder 65536 - sum freq_i is added to the
 * symbol with the largest count (lowest index on ties); N = 0 gives the uniform table.
 * Returns CG_OK, or an error before anything is launched. Does not scan for non-finite input
 * (cg_check_finite does). */
int cg_fit_cdf(const cg_params* p, const uint16_t* kv_f16, int32_t level,
               uint16_t* cdf_anchor, uint16_t* cdf_delta_level, hipStream_t stream);

/* Fit the tables of every encoding level at once (Sec. 5.2 "Arithmetic coding": one
 * distribution per channel-layer for deltas and one for anchors; Sec. 6: counted over the
 * symbols of the context being coded; Sec. 5.3: one table set per encoding level). The result
 * equals cg_fit_cdf at every level (anchor tables from any of them), but the scale and the
 * anchors of each chunk are found once for up to four levels, so the cache is read once per
 * four levels instead of once per level.
 *   kv_f16       [B][L][2][T][C] fp16, device.
 *   cdf_anchor   out [L][2][C][256], device.
 *   cdf_delta    out [n_levels][L][2][C][256], device.
 *   status       NULL, or a device uint32_t (4-byte aligned) that receives 0, or a non-zero
 *                value when the KV holds NaN or +-Inf (the tables are then meaningless);
 *                cg_get_status(status, stream) reads it.
 *   scales       NULL, or out [S] fp32, device (4-byte aligned): every stream's scale s
 *                (Sec. 5.2 "Layer-wise quantization": absmax / 127, 1 for an all-zero stream),
 *                taken from the same maxima the fit quantizes with; these are the scales
 *                cg_encode computes for the same KV, for cg_encode_with_scales.
 * Asynchronous. */
int cg_fit_cdf_levels(const cg_params* p, const uint16_t* kv_f16, uint16_t* cdf_anchor,
                      uint16_t* cdf_delta, uint32_t* status, float* scales,
                      hipStream_t stream);

/* Device scratch that cg_fit_cdf_global needs (bytes). */
#define CG_FIT_GLOBAL_WORKSPACE_BYTES 8192

/* The ablation baseline "one global symbol distribution" (Sec. 5.2 "Arithmetic coding" measures
 * the per channel-layer distributions against it; the ablation of Sec. 7.5 starts from it):
 * like cg_fit_cdf, but the counts of every layer, K/V and channel are pooled into one anchor
 * histogram and one delta histogram, normalised the same way, and that one table is written to
 * every [l][kv][ch] slot of cdf_anchor (may be NULL) and cdf_delta_level, so cg_encode and
 * cg_decode use it unchanged.
 *   workspace    device scratch of workspace_bytes >= CG_FIT_GLOBAL_WORKSPACE_BYTES, 256-byte
 *                aligned; its contents on entry do not matter.
 * Asynchronous. */
int cg_fit_cdf_global(const cg_params* p, const uint16_t* kv_f16, int32_t level,
                      uint16_t* cdf_anchor, uint16_t* cdf_delta_level, void* workspace,
                      uint64_t workspace_bytes, hipStream_t stream);

/* Encode the whole KV cache (Sec. 5.2: delta, layer-wise quantization, arithmetic coding;
 * Sec. 5.3: each chunk at its own level).
 *   kv_f16       [B][L][2][T][C] fp16, device.
 *   chunk_level  [B][NC] uint8, device: level of every (context, chunk); all equal for a
 *                single-level encode.
 *   cdf_anchor   [L][2][C][256], cdf_delta [n_levels][L][2][C][256], device (from cg_fit_cdf).
 *   words        out, device, capacity words_cap >= cg_encode_bound_words(p).
 *   offsets      out [S + 1] uint64, device; offsets[S] is the payload length in words.
 *   scales       out [S] fp32, device: the per-stream scale s.
 *   workspace    device scratch of workspace_bytes >= cg_encode_workspace_bytes(p), 256-byte
 *                aligned; its contents on entry do not matter. After the call its first word
 *                is the call's status: cg_get_status(workspace, stream) reads it.
 * chunk_level values must be < n_levels (an out-of-range level is clamped to n_levels - 1 on
 * the device). Non-finite input (NaN or +-Inf) is outside the quantizer's domain: the encoder
 * detects it on the device while it takes the streams' absolute maxima (no extra pass) and
 * records it in the status word; the payload is then meaningless but every write stays within
 * the buffers above. Asynchronous. */
int cg_encode(const cg_params* p, const uint16_t* kv_f16, const uint8_t* chunk_level,
              const uint16_t* cdf_anchor, const uint16_t* cdf_delta,
              uint32_t* words, uint64_t words_cap, uint64_t* offsets, float* scales,
              void* workspace, uint64_t workspace_bytes, hipStream_t stream);

/* cg_encode with the streams' scales as an input instead of an output (the vectorwise scale of
 * Sec. 5.2 is found once for fit and encode): `scales` [S] fp32, device (4-byte aligned), as
 * cg_fit_cdf_levels wrote them for the same KV. The encoder then takes no absolute maxima, and
 * words and offsets equal those of cg_encode. Other scales code the cache under those scales
 * (a valid payload; its values are whatever they give). Non-finite input is not looked for:
 * the fit's status reports it, and the status word in the workspace is 0. Other arguments,
 * errors and asynchrony as for cg_encode. */
int cg_encode_with_scales(const cg_params* p, const uint16_t* kv_f16, const uint8_t* chunk_level,
                          const uint16_t* cdf_anchor, const uint16_t* cdf_delta,
                          const float* scales, uint32_t* words, uint64_t words_cap,
                          uint64_t* offsets, void* workspace, uint64_t workspace_bytes,
                          hipStream_t stream);

/* Bytes of the static device scratch of cg_encode_noalloc (held by every GPU the library runs
 * on until the process ends). */
#define CG_NOALLOC_SCRATCH_BYTES (64u << 20)

/* cg_encode without any device allocation by the library or the caller beyond the inputs and
 * outputs, for callers that cannot allocate: code being captured into a HIP graph, tight
 * serving loops, harnesses that forbid hipMalloc. Same arguments, results and errors as
 * cg_encode, except:
 *   - no workspace: the encoder's scratch (status word, per-workgroup flags, worst-case slots,
 *     word counts, scan partials) is one static device buffer of CG_NOALLOC_SCRATCH_BYTES per
 *     GPU; a cache whose scratch (cg_encode_workspace_bytes(p)) exceeds it is rejected with
 *     CG_ERR_SCRATCH before anything is launched (e.g. a whole 1536-token chunk of 32 layers
 *     x 1024 channels needs about 227 MB; one such layer about 7 MB);
 *   - status: NULL, or a caller-owned device uint32_t (4-byte aligned) that receives the call's
 *     status word (0, or non-zero if the KV held NaN or +-Inf), written unconditionally.
 * Every call on a GPU shares that GPU's scratch, and nothing in it needs to start at any value;
 * calls that overlap on one GPU (on different streams, or from different host threads without
 * ordering) race and must not be issued. The first call on a device looks up the address of
 * that device's buffer (hipGetSymbolAddress, no allocation). Asynchronous. */
int cg_encode_noalloc(const cg_params* p, const uint16_t* kv_f16, const uint8_t* chunk_level,
                      const uint16_t* cdf_anchor, const uint16_t* cdf_delta, uint32_t* words,
                      uint64_t words_cap, uint64_t* offsets, float* scales, uint32_t* status,
                      hipStream_t stream);

/* Decode chunks [chunk_begin, chunk_end) of every context back to fp16 KV (Sec. 5.2; the
 * GPU decoder of Sec. 6; chunk ranges allow decoding a chunk as soon as it arrives, Sec. 6).
 *   words, offsets [S + 1], scales [S], chunk_level [B][NC], cdf_anchor, cdf_delta: device,
 *                as produced by cg_encode / cg_fit_cdf.
 *   kv_out_f16   out [B][L][2][T][C] fp16, device; only the token rows of the requested
 *                chunks are written.
 * The words buffer must be readable up to offsets[S] + CG_TAIL_WORDS. Bits after a stream's
 * codeword never change its decoded symbols (whatever follows, the code value stays inside the
 * coder's final interval), so the decoder may read into the next stream or the tail. Every
 * loop is bounded by the stream's token count: a corrupt payload yields wrong values but never
 * an out-of-range access, provided offsets is non-decreasing and offsets[S] + CG_TAIL_WORDS
 * words are readable. Asynchronous. */
int cg_decode(const cg_params* p, const uint32_t* words, const uint64_t* offsets,
              const float* scales, const uint8_t* chunk_level,
              const uint16_t* cdf_anchor, const uint16_t* cdf_delta,
              int32_t chunk_begin, int32_t chunk_end, uint16_t* kv_out_f16,
              hipStream_t stream);

/* Timings of one cg_decode_streamed call (milliseconds from the call's first copy). */
typedef struct cg_stream_stats {
  int32_t n_chunks;        /* chunks decoded (NC) */
  double transfer_ms;      /* until the last chunk's payload is on the device */
  double total_ms;         /* until the last chunk is decoded */
  double decode_sum_ms;    /* sum of the per-chunk decode durations */
  double hidden_fraction;  /* 1 - (total_ms - transfer_ms) / decode_sum_ms, clamped to [0, 1]:
                              the share of decoding done while the payload still arrived */
  /* Optional per-chunk event times, host arrays of n_chunks doubles supplied by the caller
   * (NULL: not reported), in milliseconds from the call's first copy: */
  double* chunk_copy_done_ms;     /* chunk c's payload is on the device          */
  double* chunk_decode_begin_ms;  /* chunk c's decode starts                     */
  double* chunk_decode_end_ms;    /* chunk c's decode ends                       */
} cg_stream_stats;

/* Decode the whole cache chunk by chunk while its payload arrives (Sec. 5.3: the cache is
 * split into chunks that are sent and decoded independently; Sec. 6: decoding is pipelined with
 * the transmission so that it adds little delay).
 *   words_host    [offsets[S]] uint32, HOST memory (page-locked, e.g. from hipHostMalloc, or
 *                 the copies cannot overlap the decode): the payload as cg_encode produced it.
 *   offsets_host  [S + 1] uint64, HOST memory: the same offsets (the side information that
 *                 precedes the payload).
 *   words_dev     device buffer of words_cap words, words_cap >= offsets[S] + CG_TAIL_WORDS,
 *                 that receives the payload; the other device arguments are as for cg_decode.
 * offsets_host is checked on the host before anything is issued: it must start at 0, be
 * non-decreasing at every chunk boundary used for a copy and end within words_cap -
 * CG_TAIL_WORDS (else CG_ERR_ARG / CG_ERR_CAPACITY).
 *   link_gbps     rate of the simulated link the payload arrives over, in gigabits per second:
 *                 chunk c's copy is issued when the bytes of chunks 0..c would have arrived
 *                 (the host waits). 0 or less: every copy is issued at once (the host-to-device
 *                 bus is the link).
 *   decode_stream, copy_stream   two HIP streams (the copies overlap the decodes only if they
 *                 differ); chunk c's decode waits for chunk c's copy through an event.
 *   stats         out, host, may be NULL; its chunk_* pointers are read (NULL or arrays of NC
 *                 doubles that receive the per-chunk times).
 * Chunk c of every context is copied (one copy per context: chunk c's streams of context b are
 * contiguous) and decoded with the cg_decode kernels. Creates and destroys HIP events, and
 * returns after the last decode has finished (synchronous). The result equals cg_decode over
 * all chunks. */
int cg_decode_streamed(const cg_params* p, const uint32_t* words_host,
                       const uint64_t* offsets_host, uint32_t* words_dev, uint64_t words_cap,
                       const uint64_t* offsets_dev, const float* scales_dev,
                       const uint8_t* chunk_level_dev, const uint16_t* cdf_anchor_dev,
                       const uint16_t* cdf_delta_dev, uint16_t* kv_out_dev, double link_gbps,
                       hipStream_t decode_stream, hipStream_t copy_stream,
                       cg_stream_stats* stats);

/* Streaming adaptation (Sec. 5.3 "KV cache streaming adaptation"; App. B, Alg. 1): the
 * configuration of each chunk — text (the receiver recomputes its KV) or one encoding level — is
 * chosen while the chunks are sent, so the transfer stays within a time-to-first-token SLO.
 * Host-only logic; it plans and simulates one context's transfer over a given bandwidth trace.
 * Levels are ordered by compression loss: level 0 loses least (largest payload). */
typedef struct cg_adapt_params {
  int32_t n_chunks;
  int32_t n_levels;
  const double* level_bytes;   /* [n_chunks][n_levels] payload bytes of chunk c at level v */
  const double* text_bytes;    /* [n_chunks] bytes of the chunk's text */
  const double* recompute_ms;  /* [n_chunks] time to recompute the chunk's KV from its text;
                                  NULL: text is never chosen */
  double slo_ms;               /* time-to-first-token objective for the whole context */
  double prior_gbps;           /* throughput known before the first chunk; <= 0: unknown */
  int32_t default_level;       /* level of the first chunk when no throughput is known */
} cg_adapt_params;

/* Plan and simulate: for every chunk in order, with the throughput estimate (the previous
 * chunk's measured throughput, or prior_gbps / none for the first) and remaining = slo_ms -
 * elapsed, choose text if the remaining chunks' recompute time fits in remaining (and
 * recompute_ms is given), else the lowest-loss level whose remaining chunks' bytes at that level
 * would arrive within remaining at the estimated throughput, else the most compressed level;
 * the first chunk without an estimate takes default_level (or text if its rule holds). The
 * chunk is then sent at bandwidth_gbps[c] (its actual rate), which is also the next chunk's
 * estimate; elapsed grows by its transfer time, plus its recompute time when sent as text.
 *   bandwidth_gbps  [n_chunks] host, the link rate each chunk experiences (> 0).
 *   choice_out      [n_chunks] host out: the chosen level, or -1 for text.
 *   ttft_ms_out     host out: elapsed time after the last chunk (the simulated TTFT).
 * Returns CG_OK, or CG_ERR_ARG for a null pointer or a non-positive count or rate. */
int cg_adapt_schedule(const cg_adapt_params* a, const double* bandwidth_gbps,
                      int32_t* choice_out, double* ttft_ms_out);

/* Read a status word on the device: the first word of a cg_encode workspace (the status of
 * the last cg_encode that used it), or the status argument of cg_fit_cdf_levels or
 * cg_encode_noalloc. Waits for `stream` (synchronous), then returns CG_OK, or CG_ERR_NONFINITE
 * if the KV of that call held NaN or +-Inf; CG_ERR_ARG for a null or not 4-byte aligned
 * pointer, CG_ERR_HIP if the copy fails. Every call writes its word, so it never needs
 * clearing; calls that share one on different streams race. */
int cg_get_status(const void* workspace, hipStream_t stream);

/* Scan kv_f16 [n_elem] for NaN / Inf (fp16 exponent field all ones), using flag_dev, one
 * caller-owned device uint32_t, as scratch. Synchronises `stream`. Returns CG_OK,
 * CG_ERR_NONFINITE, or an error code. The quantizer is defined for finite input only;
 * callers that cannot vouch for their input run this first. */
int cg_check_finite(const cg_params* p, const uint16_t* kv_f16, uint32_t* flag_dev,
                    hipStream_t stream);

/* ---- Token-parallel stream layout (Sec. 6: the paper's GPU decoder runs one thread per
 * token), for comparison with the channel streams above. One stream per (context, layer,
 * K/V, token) over the token's C channels in order; the symbol of channel ch is coded under the
 * (layer, K/V, ch) tables: cdf_anchor on the first token of each group, the chunk level's delta
 * table otherwise. The quantized symbols and the scales are exactly those of the channel layout
 * (the same fp16 output comes back); only their grouping into streams changes. Stream order:
 * inside context b, chunk c (first token t0, n tokens) holds streams
 * (b T + t0) 2L + (2 l + k) n + (t - t0), so each chunk's streams are contiguous. */

/* Token streams: B * L * 2 * T. 0 if p is invalid. */
int64_t cg_num_token_streams(const cg_params* p);

/* Capacity of the token-layout payload (words): every token stream at its worst case
 * ceil((18 C + 2) / 32), plus CG_TAIL_WORDS. */
uint64_t cg_encode_tokens_bound_words(const cg_params* p);

/* Device scratch of cg_encode_tokens (bytes): the symbol array (one byte per element), a
 * worst-case slot per token stream, per-stream word counts and scan partials. */
uint64_t cg_encode_tokens_workspace_bytes(const cg_params* p);

/* Device scratch of cg_decode_tokens (bytes): the symbol array, one byte per element. */
uint64_t cg_decode_tokens_workspace_bytes(const cg_params* p);

/* Encode in the token layout. Arguments as for cg_encode, except offsets [St + 1] for the St
 * token streams, words_cap >= cg_encode_tokens_bound_words(p) and workspace_bytes >=
 * cg_encode_tokens_workspace_bytes(p); scales [S] are the channel streams' (as cg_encode).
 * Asynchronous. */
int cg_encode_tokens(const cg_params* p, const uint16_t* kv_f16, const uint8_t* chunk_level,
                     const uint16_t* cdf_anchor, const uint16_t* cdf_delta, uint32_t* words,
                     uint64_t words_cap, uint64_t* offsets, float* scales, void* workspace,
                     uint64_t workspace_bytes, hipStream_t stream);

/* Decode the token layout to fp16 KV [B][L][2][T][C] (every chunk). words, offsets [St + 1],
 * scales [S], chunk_level, tables: device, as cg_encode_tokens / cg_fit_cdf produced them; the
 * words buffer must be readable up to offsets[St] + CG_TAIL_WORDS (as for cg_decode: a corrupt
 * payload gives wrong values, never an out-of-range access). workspace_bytes >=
 * cg_decode_tokens_workspace_bytes(p). Asynchronous. */
int cg_decode_tokens(const cg_params* p, const uint32_t* words, const uint64_t* offsets,
                     const float* scales, const uint8_t* chunk_level,
                     const uint16_t* cdf_anchor, const uint16_t* cdf_delta,
                     uint16_t* kv_out_f16, void* workspace, uint64_t workspace_bytes,
                     hipStream_t stream);

/* Static description of a return code; never NULL. */
const char* cg_strerror(int code);

#ifdef __cplusplus
}
#endif

#endif /* CACHEGEN_H */
