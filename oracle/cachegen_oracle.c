/*
 * cachegen_oracle.c — CPU ORACLE of the CacheGen KV-cache codec.
 *
 * TEST INFRASTRUCTURE ONLY. Nothing in the product (the HIP library and its Python binding)
 * links, loads or calls this file; only the tests, the smoke check and the benchmark's CPU
 * baseline do. It shares no source with the GPU path.
 *
 * It is written to be read against the paper (CacheGen, SIGCOMM '24), not to be fast: every
 * step is the plain definition, one stream at a time, one bit at a time. Where the paper
 * leaves a detail open, the reading taken is named at the step. The only concession to speed
 * is that independent streams are spread over POSIX threads.
 *
 * Floating point: the quantizer decides integer symbols from fp32 arithmetic (the kernel's
 * precision, so both sides take the same decisions); every fp32 operation below is a single
 * IEEE binary32 operation rounded to nearest even. Build with -ffp-contract=off (no fused
 * multiply-add) on an SSE target (no excess precision).
 *
 * Parity pins (see tests/): hand-worked coder streams, brute force over short sequences,
 * the Shannon bound, Kraft's inequality, a closed-form fit, fp16 conversion against numpy,
 * and quantizer special cases (group size 1 is per-channel absmax int8 quantization).
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define NSYM 255          /* symbols q + 127 for q in [-127, 127] */
#define TOTAL 65536u      /* frequency total: 16-bit cumulative tables */

/* ------------------------------------------------------------------------------------------
 * binary16 <-> binary32 (IEEE 754-2008 interchange formats). Plain definitions.
 * ---------------------------------------------------------------------------------------- */
float cgo_half_to_float(uint16_t h) {
  unsigned sign = h >> 15, e = (h >> 10) & 31u, man = h & 1023u;
  float mag;
  if (e == 0) mag = ldexpf((float)man, -24);                    /* zero / subnormal: man * 2^-24 */
  else if (e == 31) mag = man ? NAN : INFINITY;
  else mag = ldexpf((float)(man + 1024u), (int)e - 25);          /* (1024 + man) * 2^(e - 15 - 10) */
  return sign ? -mag : mag;
}

/* Round to nearest, ties to even. Values at or above 65520 (halfway between the largest
 * finite half 65504 and 2^16) round to infinity. */
uint16_t cgo_float_to_half(float f) {
  uint16_t sign = signbit(f) ? 0x8000u : 0u;
  float a = fabsf(f);
  if (isnan(f)) return sign | 0x7e00u;
  if (a >= 65520.0f) return sign | 0x7c00u;
  if (a < 6.103515625e-05f) {                                   /* below 2^-14: step 2^-24 */
    float r = rintf(a * 16777216.0f);                           /* exact scaling, then RNE */
    return sign | (uint16_t)r;                                  /* r == 1024 is 2^-14 itself */
  }
  int e;
  frexpf(a, &e);                                                /* a in [2^(e-1), 2^e) */
  float r = rintf(ldexpf(a, 11 - e));                           /* significand in [1024, 2048] */
  unsigned m = (unsigned)r;
  int be = e - 1 + 15;
  if (m == 2048u) { m = 1024u; be += 1; }
  if (be >= 31) return sign | 0x7c00u;
  return sign | (uint16_t)((unsigned)be << 10) | (uint16_t)(m - 1024u);
}

/* ------------------------------------------------------------------------------------------
 * Shapes. Mirrors cg_params of the C ABI (a separate declaration: nothing is shared).
 * ---------------------------------------------------------------------------------------- */
typedef struct {
  int32_t n_ctx, n_layers, n_tokens, n_channels;
  int32_t group_size, chunk_len, n_levels;
  const float* layer_bin;
  const float* level_mult;
} cgo_params;

static int64_t n_chunks(const cgo_params* p) {
  return ((int64_t)p->n_tokens + p->chunk_len - 1) / p->chunk_len;
}

int64_t cgo_num_streams(const cgo_params* p) {
  return (int64_t)p->n_ctx * n_chunks(p) * p->n_layers * 2 * p->n_channels;
}

/* A stream is one (context b, chunk c, layer l, K/V k, channel ch): the unit the arithmetic
 * coder runs over. Stream order puts each chunk's streams together (reading 15). */
typedef struct {
  int64_t b, c, l, k, ch;
  int64_t t0, n;          /* first token of the chunk, tokens in the chunk */
  const uint16_t* x;      /* first element of the stream in the KV tensor */
  int64_t stride;         /* elements between consecutive tokens (= C) */
} stream_t;

static stream_t locate(const cgo_params* p, const uint16_t* kv, int64_t s) {
  stream_t r;
  int64_t C = p->n_channels, L = p->n_layers, NC = n_chunks(p), T = p->n_tokens;
  r.ch = s % C; s /= C;
  r.k = s % 2; s /= 2;
  r.l = s % L; s /= L;
  r.c = s % NC; s /= NC;
  r.b = s;
  r.t0 = r.c * p->chunk_len;
  r.n = (r.t0 + p->chunk_len <= T) ? p->chunk_len : T - r.t0;
  r.stride = C;
  r.x = kv ? kv + (((r.b * L + r.l) * 2 + r.k) * T + r.t0) * C + r.ch : NULL;
  return r;
}

/* ------------------------------------------------------------------------------------------
 * Steps a1-a3 and a7: scale, anchor / delta quantization, reconstruction.
 * Sec. 5.2 "Change-based encoding" (groups of tokens, first token the anchor, deltas against
 * that same anchor), "Layer-wise quantization" (bin width by layer group, vectorwise
 * quantization, 8-bit anchors); App. C.2 (default bins 0.5 / 1 / 1.5).
 * Readings: the vectorwise scale is the absmax of one stream (one channel of one layer and
 * K/V over one chunk) divided by 127; the bin width is layer_bin * level_mult in units of that
 * scale; deltas are taken against the reconstructed anchor; groups restart at each chunk.
 * ---------------------------------------------------------------------------------------- */
static float clamp127(float v) { return v < -127.0f ? -127.0f : (v > 127.0f ? 127.0f : v); }

float cgo_stream_scale(const uint16_t* x, int64_t stride, int64_t n) {
  float m = 0.0f;
  for (int64_t j = 0; j < n; ++j) {
    float a = fabsf(cgo_half_to_float(x[j * stride]));
    if (a > m) m = a;
  }
  return m == 0.0f ? 1.0f : m / 127.0f;
}

/* Quantize one stream: symbols (q + 127) and the fp16 values the decoder must reproduce. */
void cgo_quantize_stream(const uint16_t* x, int64_t stride, int64_t n, int32_t G,
                         float s, float w, uint8_t* sym, uint16_t* recon) {
  /* The symbol is the integer q; reconstruction starts from that integer (so a value that
   * rounds to -0.0 reconstructs as +0, exactly as a decoder that only sees q). */
  float anchor = 0.0f;
  for (int64_t j = 0; j < n; ++j) {
    float v = cgo_half_to_float(x[j * stride]);
    int q;
    float out;
    if (j % G == 0) {                          /* anchor: 8-bit, on its own */
      q = (int)rintf(clamp127(v / s));
      anchor = (float)q * s;
      out = anchor;
    } else {                                   /* delta against the group's anchor */
      float d = v - anchor;
      q = (int)rintf(clamp127(d / w));
      float qw = (float)q * w;
      out = anchor + qw;
    }
    if (sym) sym[j] = (uint8_t)(q + 127);
    if (recon) recon[j] = cgo_float_to_half(out);
  }
}

/* The inverse of the quantizer for one stream: symbols -> fp16 values (step a7). */
void cgo_dequantize_stream(const uint8_t* sym, int64_t n, int32_t G, float s, float w,
                           uint16_t* out, int64_t stride) {
  float anchor = 0.0f;
  for (int64_t j = 0; j < n; ++j) {
    float q = (float)((int)sym[j] - 127);
    float v;
    if (j % G == 0) {
      anchor = q * s;
      v = anchor;
    } else {
      float qw = q * w;
      v = anchor + qw;
    }
    out[j * stride] = cgo_float_to_half(v);
  }
}

static float bin_width(const cgo_params* p, int64_t l, int level, float s) {
  float bw = p->layer_bin[l] * p->level_mult[level];
  return bw * s;
}

/* ------------------------------------------------------------------------------------------
 * Step a4: distribution fit. Sec. 5.2 "Arithmetic coding" (one distribution per channel-layer
 * for deltas, another for anchors), Sec. 6 (frequencies counted over the context's symbols).
 * Reading: 16-bit frequency total, every symbol at least 1 so any table codes any input,
 * remainder to the most frequent symbol (lowest index on ties).
 * ---------------------------------------------------------------------------------------- */
void cgo_normalize(const uint64_t* counts /*[255]*/, uint16_t* cum_out /*[256]*/) {
  uint64_t c[NSYM], N = 0;
  for (int i = 0; i < NSYM; ++i) { c[i] = counts[i]; N += c[i]; }
  if (N == 0) { for (int i = 0; i < NSYM; ++i) c[i] = 1; N = NSYM; }
  uint64_t freq[NSYM], sum = 0;
  for (int i = 0; i < NSYM; ++i) {
    freq[i] = 1 + (c[i] * (uint64_t)(TOTAL - NSYM)) / N;
    sum += freq[i];
  }
  int top = 0;
  for (int i = 1; i < NSYM; ++i) if (c[i] > c[top]) top = i;
  freq[top] += TOTAL - sum;
  uint64_t cum = 0;
  for (int i = 0; i < NSYM; ++i) { cum_out[i] = (uint16_t)cum; cum += freq[i]; }
  cum_out[255] = 0;                            /* padding; the implicit top is 65536 */
}

typedef struct {
  const cgo_params* p; const uint16_t* kv; int level;
  uint16_t* cdf_anchor; uint16_t* cdf_delta;
  int64_t lk_begin, lk_end;                    /* range of (l, k) pairs for this thread */
} fit_job;

static void* fit_worker(void* arg) {
  fit_job* J = (fit_job*)arg;
  const cgo_params* p = J->p;
  int64_t C = p->n_channels, NC = n_chunks(p), L = p->n_layers;
  uint64_t* ca = (uint64_t*)calloc((size_t)C * NSYM, sizeof(uint64_t));
  uint64_t* cd = (uint64_t*)calloc((size_t)C * NSYM, sizeof(uint64_t));
  uint8_t* sym = (uint8_t*)malloc((size_t)p->chunk_len);
  for (int64_t lk = J->lk_begin; lk < J->lk_end; ++lk) {
    int64_t l = lk / 2, k = lk % 2;
    memset(ca, 0, (size_t)C * NSYM * sizeof(uint64_t));
    memset(cd, 0, (size_t)C * NSYM * sizeof(uint64_t));
    for (int64_t b = 0; b < p->n_ctx; ++b)
      for (int64_t c = 0; c < NC; ++c)
        for (int64_t ch = 0; ch < C; ++ch) {
          int64_t s = (((b * NC + c) * L + l) * 2 + k) * C + ch;
          stream_t st = locate(p, J->kv, s);
          float sc = cgo_stream_scale(st.x, st.stride, st.n);
          float w = bin_width(p, l, J->level, sc);
          cgo_quantize_stream(st.x, st.stride, st.n, p->group_size, sc, w, sym, NULL);
          for (int64_t j = 0; j < st.n; ++j) {
            if (j % p->group_size == 0) ca[ch * NSYM + sym[j]] += 1;
            else cd[ch * NSYM + sym[j]] += 1;
          }
        }
    for (int64_t ch = 0; ch < C; ++ch) {
      size_t t = (size_t)((l * 2 + k) * C + ch) * 256;
      if (J->cdf_anchor) cgo_normalize(ca + ch * NSYM, J->cdf_anchor + t);
      cgo_normalize(cd + ch * NSYM, J->cdf_delta + t);
    }
  }
  free(ca); free(cd); free(sym);
  return NULL;
}

static int clamp_threads(int threads, int64_t work) {
  if (threads < 1) threads = 1;
  if (threads > 256) threads = 256;
  if (work < threads) threads = (int)(work > 0 ? work : 1);
  return threads;
}

/* cg_fit_cdf: counts at one encoding level over every chunk of every context. */
int cg_fit_cdf_ref(const cgo_params* p, const uint16_t* kv, int level, uint16_t* cdf_anchor,
                   uint16_t* cdf_delta_level, int threads) {
  int64_t pairs = (int64_t)p->n_layers * 2;
  threads = clamp_threads(threads, pairs);
  pthread_t th[256];
  fit_job jobs[256];
  for (int i = 0; i < threads; ++i) {
    jobs[i] = (fit_job){p, kv, level, cdf_anchor, cdf_delta_level,
                        pairs * i / threads, pairs * (i + 1) / threads};
    pthread_create(&th[i], NULL, fit_worker, &jobs[i]);
  }
  for (int i = 0; i < threads; ++i) pthread_join(th[i], NULL);
  return 0;
}

/* ------------------------------------------------------------------------------------------
 * Ablation baseline: one global symbol distribution (Sec. 5.2 "Arithmetic coding" compares the
 * per channel-layer distributions against this strawman; Sec. 7.5 "Ablation Study" starts from
 * it). The counts of every (layer, K/V, channel) are summed into one anchor histogram and one
 * delta histogram, normalised once like any other table, and the resulting table is written to
 * every (layer, K/V, channel) slot so the coder uses it everywhere.
 * ---------------------------------------------------------------------------------------- */
typedef struct {
  const cgo_params* p; const uint16_t* kv; int level;
  int64_t s_begin, s_end;                      /* range of streams for this thread */
  uint64_t ca[NSYM], cd[NSYM];                 /* this thread's counts */
} global_job;

static void* global_worker(void* arg) {
  global_job* J = (global_job*)arg;
  const cgo_params* p = J->p;
  int64_t C = p->n_channels, L = p->n_layers;
  uint8_t* sym = (uint8_t*)malloc((size_t)p->chunk_len);
  for (int64_t s = J->s_begin; s < J->s_end; ++s) {
    int64_t l = (s / (2 * C)) % L;
    stream_t st = locate(p, J->kv, s);
    float sc = cgo_stream_scale(st.x, st.stride, st.n);
    float w = bin_width(p, l, J->level, sc);
    cgo_quantize_stream(st.x, st.stride, st.n, p->group_size, sc, w, sym, NULL);
    for (int64_t j = 0; j < st.n; ++j) {
      if (j % p->group_size == 0) J->ca[sym[j]] += 1;
      else J->cd[sym[j]] += 1;
    }
  }
  free(sym);
  return NULL;
}

int cg_fit_cdf_global_ref(const cgo_params* p, const uint16_t* kv, int level,
                          uint16_t* cdf_anchor, uint16_t* cdf_delta_level, int threads) {
  int64_t S = cgo_num_streams(p);
  threads = clamp_threads(threads, S);
  pthread_t th[256];
  global_job* jobs = (global_job*)calloc((size_t)threads, sizeof(global_job));
  for (int i = 0; i < threads; ++i) {
    jobs[i].p = p; jobs[i].kv = kv; jobs[i].level = level;
    jobs[i].s_begin = S * i / threads; jobs[i].s_end = S * (i + 1) / threads;
    pthread_create(&th[i], NULL, global_worker, &jobs[i]);
  }
  uint64_t ca[NSYM] = {0}, cd[NSYM] = {0};
  for (int i = 0; i < threads; ++i) {
    pthread_join(th[i], NULL);
    for (int k = 0; k < NSYM; ++k) { ca[k] += jobs[i].ca[k]; cd[k] += jobs[i].cd[k]; }
  }
  free(jobs);
  uint16_t ta[256], td[256];
  cgo_normalize(ca, ta);
  cgo_normalize(cd, td);
  int64_t tables = (int64_t)p->n_layers * 2 * p->n_channels;
  for (int64_t t = 0; t < tables; ++t) {
    if (cdf_anchor) memcpy(cdf_anchor + t * 256, ta, sizeof(ta));
    memcpy(cdf_delta_level + t * 256, td, sizeof(td));
  }
  return 0;
}

/* ------------------------------------------------------------------------------------------
 * Steps a5 / a6: arithmetic coding (Sec. 5.2 "Arithmetic coding"; GPU coding in Sec. 6).
 * The paper names no variant. Reading: the integer arithmetic coder of Witten, Neal and
 * Cleary (CACM 30(6), 1987) with 32-bit code registers and 16-bit cumulative frequencies:
 *   range update   R = high - low + 1, high = low + R*cum[i+1]/2^16 - 1, low = low + R*cum[i]/2^16
 *   renormalise    high < 1/2 : output 0 then the pending 1s
 *                  low >= 1/2 : output 1 then the pending 0s, subtract 1/2
 *                  1/4 <= low, high < 3/4 : one more pending bit, subtract 1/4
 *                  after each case double both ends (high gets a 1 shifted in)
 *   termination    one more pending bit, then 0 (and pending 1s) if low < 1/4, else 1 (and 0s)
 * Bits go MSB-first into 32-bit words; a stream is zero-padded to a whole word.
 * ---------------------------------------------------------------------------------------- */
#define HALF 0x80000000ull
#define QTR 0x40000000ull
#define Q3 0xC0000000ull

static uint64_t cum_at(const uint16_t* cum, int i) { return i >= NSYM ? TOTAL : cum[i]; }

typedef struct { uint32_t* w; uint64_t cap_bits; uint64_t nbits; int overflow; } bitwriter;

static void put_bit(bitwriter* bw, int bit) {
  if (bw->nbits >= bw->cap_bits) { bw->overflow = 1; return; }
  if (bit) bw->w[bw->nbits >> 5] |= 0x80000000u >> (bw->nbits & 31);
  bw->nbits++;
}

static void put_bit_plus_pending(bitwriter* bw, int bit, uint64_t* pending) {
  put_bit(bw, bit);
  for (; *pending > 0; --*pending) put_bit(bw, !bit);
}

/* Encode n symbols; symbol j uses the table tabs[j] (anchor or delta). Returns the bit count
 * (before padding), or UINT64_MAX if cap_words is too small. `out` must be zeroed. */
uint64_t cgo_ac_encode(const uint8_t* sym, int64_t n, const uint16_t* const* tabs,
                       uint32_t* out, uint64_t cap_words) {
  bitwriter bw = {out, cap_words * 32, 0, 0};
  uint64_t low = 0, high = 0xFFFFFFFFull, pending = 0;
  for (int64_t j = 0; j < n; ++j) {
    const uint16_t* cum = tabs[j];
    int i = sym[j];
    uint64_t R = high - low + 1;
    high = low + ((R * cum_at(cum, i + 1)) >> 16) - 1;
    low = low + ((R * cum_at(cum, i)) >> 16);
    for (;;) {
      if (high < HALF) {
        put_bit_plus_pending(&bw, 0, &pending);
      } else if (low >= HALF) {
        put_bit_plus_pending(&bw, 1, &pending);
        low -= HALF; high -= HALF;
      } else if (low >= QTR && high < Q3) {
        pending++;
        low -= QTR; high -= QTR;
      } else {
        break;
      }
      low = 2 * low;
      high = 2 * high + 1;
    }
  }
  pending++;
  if (low < QTR) put_bit_plus_pending(&bw, 0, &pending);
  else put_bit_plus_pending(&bw, 1, &pending);
  return bw.overflow ? UINT64_MAX : bw.nbits;
}

typedef struct { const uint32_t* w; uint64_t nwords; uint64_t pos; } bitreader;

static int get_bit(bitreader* br) {
  uint64_t p = br->pos++;
  if ((p >> 5) >= br->nwords) return 0;        /* past the end: zeros */
  return (br->w[p >> 5] >> (31 - (p & 31))) & 1u;
}

/* Decode n symbols from nwords words; symbol j uses tabs[j]. */
void cgo_ac_decode(const uint32_t* words, uint64_t nwords, int64_t n,
                   const uint16_t* const* tabs, uint8_t* sym) {
  bitreader br = {words, nwords, 0};
  uint64_t low = 0, high = 0xFFFFFFFFull, value = 0;
  for (int i = 0; i < 32; ++i) value = 2 * value + (uint64_t)get_bit(&br);
  for (int64_t j = 0; j < n; ++j) {
    const uint16_t* cum = tabs[j];
    uint64_t R = high - low + 1;
    uint64_t t = (((value - low + 1) << 16) - 1) / R;
    int i = 0;
    while (i + 1 < NSYM && cum_at(cum, i + 1) <= t) ++i;   /* cum[i] <= t < cum[i+1] */
    sym[j] = (uint8_t)i;
    high = low + ((R * cum_at(cum, i + 1)) >> 16) - 1;
    low = low + ((R * cum_at(cum, i)) >> 16);
    for (;;) {
      if (high < HALF) {
        /* nothing to subtract */
      } else if (low >= HALF) {
        low -= HALF; high -= HALF; value -= HALF;
      } else if (low >= QTR && high < Q3) {
        low -= QTR; high -= QTR; value -= QTR;
      } else {
        break;
      }
      low = 2 * low;
      high = 2 * high + 1;
      value = 2 * value + (uint64_t)get_bit(&br);
    }
  }
}

/* ------------------------------------------------------------------------------------------
 * Whole codec: encode / decode every stream of a KV cache.
 * ---------------------------------------------------------------------------------------- */
static const uint16_t* anchor_table(const cgo_params* p, const uint16_t* cdf_anchor,
                                    const stream_t* st) {
  return cdf_anchor + (size_t)((st->l * 2 + st->k) * p->n_channels + st->ch) * 256;
}

static const uint16_t* delta_table(const cgo_params* p, const uint16_t* cdf_delta, int level,
                                   const stream_t* st) {
  size_t per_level = (size_t)p->n_layers * 2 * p->n_channels * 256;
  return cdf_delta + per_level * (size_t)level +
         (size_t)((st->l * 2 + st->k) * p->n_channels + st->ch) * 256;
}

static int level_of(const cgo_params* p, const uint8_t* chunk_level, const stream_t* st) {
  int lv = chunk_level[st->b * n_chunks(p) + st->c];
  return lv < p->n_levels ? lv : p->n_levels - 1;
}

/* The order in which a stream's symbols are coded (reading 14): order[i] is the token (within
 * the chunk) of the i-th coded symbol. First every anchor (tokens 0, G, 2G, ...), then every
 * other token, each part in token order. The paper fixes what is coded and under which
 * distribution (Sec. 5.2), not the order of the symbols inside one bitstream. */
static void coded_order(int64_t n, int64_t G, int64_t* order) {
  int64_t i = 0;
  for (int64_t j = 0; j < n; j += G) order[i++] = j;
  for (int64_t j = 0; j < n; ++j)
    if (j % G != 0) order[i++] = j;
}

uint64_t cgo_stream_bound_words(int64_t n) { return (18ull * (uint64_t)n + 2 + 31) / 32; }

/* Encode one stream s into out (zeroed, cap_words). Also returns its scale and symbols.
 * Returns the word count, or UINT64_MAX on overflow. */
uint64_t cgo_encode_stream(const cgo_params* p, const uint16_t* kv, const uint8_t* chunk_level,
                           const uint16_t* cdf_anchor, const uint16_t* cdf_delta, int64_t s,
                           uint32_t* out, uint64_t cap_words, float* scale_out,
                           uint8_t* sym_out) {
  stream_t st = locate(p, kv, s);
  int lv = level_of(p, chunk_level, &st);
  float sc = cgo_stream_scale(st.x, st.stride, st.n);
  float w = bin_width(p, st.l, lv, sc);
  uint8_t* sym = sym_out ? sym_out : (uint8_t*)malloc((size_t)st.n);
  const uint16_t** tabs = (const uint16_t**)malloc((size_t)st.n * sizeof(*tabs));
  cgo_quantize_stream(st.x, st.stride, st.n, p->group_size, sc, w, sym, NULL);
  const uint16_t* ta = anchor_table(p, cdf_anchor, &st);
  const uint16_t* td = delta_table(p, cdf_delta, lv, &st);
  /* coded order (reading 14): the anchors in token order, then the deltas in token order */
  int64_t* order = (int64_t*)malloc((size_t)st.n * sizeof(int64_t));
  coded_order(st.n, p->group_size, order);
  uint8_t* csym = (uint8_t*)malloc((size_t)st.n);
  for (int64_t i = 0; i < st.n; ++i) {
    csym[i] = sym[order[i]];
    tabs[i] = (order[i] % p->group_size == 0) ? ta : td;
  }
  uint64_t bits = cgo_ac_encode(csym, st.n, tabs, out, cap_words);
  free(csym);
  free(order);
  free(tabs);
  if (!sym_out) free(sym);
  if (scale_out) *scale_out = sc;
  return bits == UINT64_MAX ? UINT64_MAX : (bits + 31) / 32;
}

/* Decode one stream s from its words into the fp16 KV tensor (or, when kv_out is NULL, into
 * recon[n] contiguous). Symbols are returned in sym_out when non-NULL. */
void cgo_decode_stream(const cgo_params* p, const uint32_t* words, uint64_t nwords, float scale,
                       const uint8_t* chunk_level, const uint16_t* cdf_anchor,
                       const uint16_t* cdf_delta, int64_t s, uint16_t* kv_out,
                       uint16_t* recon, uint8_t* sym_out) {
  stream_t st = locate(p, NULL, s);
  int lv = level_of(p, chunk_level, &st);
  float w = bin_width(p, st.l, lv, scale);
  uint8_t* sym = sym_out ? sym_out : (uint8_t*)malloc((size_t)st.n);
  const uint16_t** tabs = (const uint16_t**)malloc((size_t)st.n * sizeof(*tabs));
  const uint16_t* ta = anchor_table(p, cdf_anchor, &st);
  const uint16_t* td = delta_table(p, cdf_delta, lv, &st);
  int64_t* order = (int64_t*)malloc((size_t)st.n * sizeof(int64_t));
  coded_order(st.n, p->group_size, order);
  uint8_t* csym = (uint8_t*)malloc((size_t)st.n);
  for (int64_t i = 0; i < st.n; ++i) tabs[i] = (order[i] % p->group_size == 0) ? ta : td;
  cgo_ac_decode(words, nwords, st.n, tabs, csym);
  for (int64_t i = 0; i < st.n; ++i) sym[order[i]] = csym[i];
  free(csym);
  free(order);
  if (kv_out) {
    int64_t C = p->n_channels, L = p->n_layers, T = p->n_tokens;
    uint16_t* dst = kv_out + (((st.b * L + st.l) * 2 + st.k) * T + st.t0) * C + st.ch;
    cgo_dequantize_stream(sym, st.n, p->group_size, scale, w, dst, C);
  }
  if (recon) cgo_dequantize_stream(sym, st.n, p->group_size, scale, w, recon, 1);
  free(tabs);
  if (!sym_out) free(sym);
}

typedef struct {
  const cgo_params* p; const uint16_t* kv; const uint8_t* chunk_level;
  const uint16_t* cdf_anchor; const uint16_t* cdf_delta;
  int64_t s_begin, s_end;
  uint32_t* buf; uint64_t buf_words;           /* this thread's streams, back to back */
  uint64_t* lens;                              /* [S] words per stream */
  float* scales;
  int failed;
} enc_job;

static void* enc_worker(void* arg) {
  enc_job* J = (enc_job*)arg;
  uint64_t used = 0, cap = 1 << 16;
  J->buf = (uint32_t*)calloc(cap, sizeof(uint32_t));
  for (int64_t s = J->s_begin; s < J->s_end; ++s) {
    stream_t st = locate(J->p, NULL, s);
    uint64_t need = cgo_stream_bound_words(st.n);
    if (used + need > cap) {
      uint64_t ncap = cap;
      while (used + need > ncap) ncap *= 2;
      J->buf = (uint32_t*)realloc(J->buf, ncap * sizeof(uint32_t));
      memset(J->buf + cap, 0, (ncap - cap) * sizeof(uint32_t));
      cap = ncap;
    }
    uint64_t nw = cgo_encode_stream(J->p, J->kv, J->chunk_level, J->cdf_anchor, J->cdf_delta,
                                    s, J->buf + used, need, &J->scales[s], NULL);
    if (nw == UINT64_MAX) { J->failed = 1; break; }
    J->lens[s] = nw;
    used += nw;
  }
  J->buf_words = used;
  return NULL;
}

/* cg_encode: all streams. words must hold the payload (cap_words); offsets [S+1]; scales [S].
 * Returns the total word count, or -1 if cap_words is too small. */
int64_t cg_encode_ref(const cgo_params* p, const uint16_t* kv, const uint8_t* chunk_level,
                      const uint16_t* cdf_anchor, const uint16_t* cdf_delta, uint32_t* words,
                      uint64_t cap_words, uint64_t* offsets, float* scales, int threads) {
  int64_t S = cgo_num_streams(p);
  threads = clamp_threads(threads, S);
  uint64_t* lens = (uint64_t*)calloc((size_t)S, sizeof(uint64_t));
  pthread_t th[256];
  enc_job jobs[256];
  for (int i = 0; i < threads; ++i) {
    jobs[i] = (enc_job){p, kv, chunk_level, cdf_anchor, cdf_delta,
                        S * i / threads, S * (i + 1) / threads, NULL, 0, lens, scales, 0};
    pthread_create(&th[i], NULL, enc_worker, &jobs[i]);
  }
  for (int i = 0; i < threads; ++i) pthread_join(th[i], NULL);
  int failed = 0;
  for (int i = 0; i < threads; ++i) failed |= jobs[i].failed;
  uint64_t total = 0;
  offsets[0] = 0;
  for (int64_t s = 0; s < S; ++s) { total += lens[s]; offsets[s + 1] = total; }
  if (!failed && total <= cap_words) {
    for (int i = 0; i < threads; ++i)       /* thread ranges are contiguous in stream order */
      memcpy(words + offsets[jobs[i].s_begin], jobs[i].buf, jobs[i].buf_words * sizeof(uint32_t));
  }
  for (int i = 0; i < threads; ++i) free(jobs[i].buf);
  free(lens);
  return (failed || total > cap_words) ? -1 : (int64_t)total;
}

typedef struct {
  const cgo_params* p; const uint32_t* words; const uint64_t* offsets; const float* scales;
  const uint8_t* chunk_level; const uint16_t* cdf_anchor; const uint16_t* cdf_delta;
  uint16_t* kv_out; int64_t s_begin, s_end; int64_t c_begin, c_end;
} dec_job;

static void* dec_worker(void* arg) {
  dec_job* J = (dec_job*)arg;
  for (int64_t s = J->s_begin; s < J->s_end; ++s) {
    stream_t st = locate(J->p, NULL, s);
    if (st.c < J->c_begin || st.c >= J->c_end) continue;
    cgo_decode_stream(J->p, J->words + J->offsets[s], J->offsets[s + 1] - J->offsets[s],
                      J->scales[s], J->chunk_level, J->cdf_anchor, J->cdf_delta, s, J->kv_out,
                      NULL, NULL);
  }
  return NULL;
}

/* cg_decode: chunks [c_begin, c_end) of every context into kv_out. */
int cg_decode_ref(const cgo_params* p, const uint32_t* words, const uint64_t* offsets,
                  const float* scales, const uint8_t* chunk_level, const uint16_t* cdf_anchor,
                  const uint16_t* cdf_delta, int64_t c_begin, int64_t c_end, uint16_t* kv_out,
                  int threads) {
  int64_t S = cgo_num_streams(p);
  threads = clamp_threads(threads, S);
  pthread_t th[256];
  dec_job jobs[256];
  for (int i = 0; i < threads; ++i) {
    jobs[i] = (dec_job){p, words, offsets, scales, chunk_level, cdf_anchor, cdf_delta, kv_out,
                        S * i / threads, S * (i + 1) / threads, c_begin, c_end};
    pthread_create(&th[i], NULL, dec_worker, &jobs[i]);
  }
  for (int i = 0; i < threads; ++i) pthread_join(th[i], NULL);
  return 0;
}

/* Scales and symbols of a list of streams, plus their words, without a whole-cache encode:
 * the sampled parity check at full size. out_words gets the streams back to back; lens[i]
 * the word count of stream ids[i]. Returns total words, or -1 on overflow of cap_words. */
typedef struct {
  const cgo_params* p; const uint16_t* kv; const uint8_t* chunk_level;
  const uint16_t* cdf_anchor; const uint16_t* cdf_delta;
  const int64_t* ids; int64_t i_begin, i_end;
  uint32_t* slots; uint64_t slot_words; uint64_t* lens; float* scales; int failed;
} sample_job;

static void* sample_worker(void* arg) {
  sample_job* J = (sample_job*)arg;
  for (int64_t i = J->i_begin; i < J->i_end; ++i) {
    uint64_t nw = cgo_encode_stream(J->p, J->kv, J->chunk_level, J->cdf_anchor, J->cdf_delta,
                                    J->ids[i], J->slots + (uint64_t)i * J->slot_words,
                                    J->slot_words, &J->scales[i], NULL);
    if (nw == UINT64_MAX) { J->failed = 1; return NULL; }
    J->lens[i] = nw;
  }
  return NULL;
}

int64_t cgo_encode_streams(const cgo_params* p, const uint16_t* kv, const uint8_t* chunk_level,
                           const uint16_t* cdf_anchor, const uint16_t* cdf_delta,
                           const int64_t* ids, int64_t n_ids, uint32_t* out_words,
                           uint64_t cap_words, uint64_t* lens, float* scales, int threads) {
  uint64_t slot = cgo_stream_bound_words(p->chunk_len < p->n_tokens ? p->chunk_len : p->n_tokens);
  uint32_t* slots = (uint32_t*)calloc((size_t)(n_ids > 0 ? n_ids : 1) * slot, sizeof(uint32_t));
  threads = clamp_threads(threads, n_ids);
  pthread_t th[256];
  sample_job jobs[256];
  for (int i = 0; i < threads; ++i) {
    jobs[i] = (sample_job){p, kv, chunk_level, cdf_anchor, cdf_delta, ids,
                           n_ids * i / threads, n_ids * (i + 1) / threads,
                           slots, slot, lens, scales, 0};
    pthread_create(&th[i], NULL, sample_worker, &jobs[i]);
  }
  int failed = 0;
  for (int i = 0; i < threads; ++i) { pthread_join(th[i], NULL); failed |= jobs[i].failed; }
  uint64_t total = 0;
  if (!failed) {
    for (int64_t i = 0; i < n_ids; ++i) {
      if (total + lens[i] > cap_words) { failed = 1; break; }
      memcpy(out_words + total, slots + (uint64_t)i * slot, lens[i] * sizeof(uint32_t));
      total += lens[i];
    }
  }
  free(slots);
  return failed ? -1 : (int64_t)total;
}

/* ------------------------------------------------------------------------------------------
 * Token-parallel stream layout (Sec. 6: the paper's GPU decoder runs one thread per token).
 * Reading: one stream per (context, layer, K/V, token) over that token's channels in order;
 * the symbol of channel ch is coded under the (layer, K/V, ch) tables (the anchor table for the
 * anchor token of a group, the chunk level's delta table otherwise). Quantization, scales and
 * tables are those of the channel-stream layout above: only the grouping of the same symbols
 * into streams differs. Stream order keeps each chunk's streams together: inside context b,
 * chunk c (first token t0, n_c tokens) holds streams (b T + t0) 2L + (2 l + k) n_c + (t - t0).
 * ---------------------------------------------------------------------------------------- */
int64_t cgo_num_token_streams(const cgo_params* p) {
  return (int64_t)p->n_ctx * p->n_layers * 2 * p->n_tokens;
}

typedef struct { int64_t b, c, l, k, t, t0, n; } tok_stream_t;

static tok_stream_t locate_token(const cgo_params* p, int64_t s) {
  tok_stream_t r;
  int64_t L2 = 2 * (int64_t)p->n_layers, T = p->n_tokens;
  r.b = s / (T * L2);
  int64_t rem = s - r.b * T * L2;
  r.c = rem / ((int64_t)p->chunk_len * L2);
  r.t0 = r.c * p->chunk_len;
  r.n = (r.t0 + p->chunk_len <= T) ? p->chunk_len : T - r.t0;
  rem -= r.t0 * L2;
  int64_t lk = rem / r.n;
  r.t = r.t0 + (rem - lk * r.n);
  r.l = lk / 2;
  r.k = lk % 2;
  return r;
}

/* Symbols of the whole cache in [b][l][k][t][ch] order plus the channel streams' scales. */
typedef struct {
  const cgo_params* p; const uint16_t* kv; const uint8_t* chunk_level;
  int64_t s_begin, s_end; uint8_t* sym; float* scales;
} qall_job;

static void* qall_worker(void* arg) {
  qall_job* J = (qall_job*)arg;
  const cgo_params* p = J->p;
  uint8_t* col = (uint8_t*)malloc((size_t)p->chunk_len);
  for (int64_t s = J->s_begin; s < J->s_end; ++s) {
    stream_t st = locate(p, J->kv, s);
    int lv = level_of(p, J->chunk_level, &st);
    float sc = cgo_stream_scale(st.x, st.stride, st.n);
    cgo_quantize_stream(st.x, st.stride, st.n, p->group_size, sc, bin_width(p, st.l, lv, sc),
                        col, NULL);
    J->scales[s] = sc;
    uint8_t* dst = J->sym + (((st.b * p->n_layers + st.l) * 2 + st.k) * p->n_tokens + st.t0) *
                                p->n_channels + st.ch;
    for (int64_t j = 0; j < st.n; ++j) dst[j * p->n_channels] = col[j];
  }
  free(col);
  return NULL;
}

static void quantize_all(const cgo_params* p, const uint16_t* kv, const uint8_t* chunk_level,
                         uint8_t* sym, float* scales, int threads) {
  int64_t S = cgo_num_streams(p);
  threads = clamp_threads(threads, S);
  pthread_t th[256];
  qall_job jobs[256];
  for (int i = 0; i < threads; ++i) {
    jobs[i] = (qall_job){p, kv, chunk_level, S * i / threads, S * (i + 1) / threads, sym, scales};
    pthread_create(&th[i], NULL, qall_worker, &jobs[i]);
  }
  for (int i = 0; i < threads; ++i) pthread_join(th[i], NULL);
}

/* The tables of the C symbols of token stream ts. */
static void token_tables(const cgo_params* p, const uint8_t* chunk_level,
                         const uint16_t* cdf_anchor, const uint16_t* cdf_delta,
                         const tok_stream_t* ts, const uint16_t** tabs) {
  int lv = chunk_level[ts->b * n_chunks(p) + ts->c];
  lv = lv < p->n_levels ? lv : p->n_levels - 1;
  int anchor = (ts->t - ts->t0) % p->group_size == 0;
  for (int64_t ch = 0; ch < p->n_channels; ++ch) {
    stream_t st = {ts->b, ts->c, ts->l, ts->k, ch, ts->t0, ts->n, NULL, p->n_channels};
    tabs[ch] = anchor ? anchor_table(p, cdf_anchor, &st) : delta_table(p, cdf_delta, lv, &st);
  }
}

typedef struct {
  const cgo_params* p; const uint8_t* sym; const uint8_t* chunk_level;
  const uint16_t* cdf_anchor; const uint16_t* cdf_delta;
  int64_t s_begin, s_end;
  uint32_t* buf; uint64_t buf_words; uint64_t* lens; int failed;
} tenc_job;

static void* tenc_worker(void* arg) {
  tenc_job* J = (tenc_job*)arg;
  const cgo_params* p = J->p;
  int64_t C = p->n_channels;
  uint64_t need = cgo_stream_bound_words(C);
  uint64_t cap = (uint64_t)(J->s_end - J->s_begin) * need + 1;
  J->buf = (uint32_t*)calloc((size_t)cap, sizeof(uint32_t));
  const uint16_t** tabs = (const uint16_t**)malloc((size_t)C * sizeof(*tabs));
  uint64_t used = 0;
  for (int64_t s = J->s_begin; s < J->s_end; ++s) {
    tok_stream_t ts = locate_token(p, s);
    token_tables(p, J->chunk_level, J->cdf_anchor, J->cdf_delta, &ts, tabs);
    const uint8_t* row = J->sym + (((ts.b * p->n_layers + ts.l) * 2 + ts.k) * p->n_tokens + ts.t) * C;
    uint64_t bits = cgo_ac_encode(row, C, tabs, J->buf + used, need);
    if (bits == UINT64_MAX) { J->failed = 1; break; }
    J->lens[s] = (bits + 31) / 32;
    used += J->lens[s];
  }
  free(tabs);
  J->buf_words = used;
  return NULL;
}

/* Encode in the token layout. offsets [St + 1] (St token streams); scales [S] of the channel
 * streams (the side information is the same as in the channel layout). Returns the total word
 * count, or -1 if cap_words is too small. */
int64_t cg_encode_tokens_ref(const cgo_params* p, const uint16_t* kv, const uint8_t* chunk_level,
                             const uint16_t* cdf_anchor, const uint16_t* cdf_delta,
                             uint32_t* words, uint64_t cap_words, uint64_t* offsets,
                             float* scales, int threads) {
  int64_t St = cgo_num_token_streams(p);
  int64_t n_elem = St * p->n_channels;
  uint8_t* sym = (uint8_t*)malloc((size_t)(n_elem > 0 ? n_elem : 1));
  quantize_all(p, kv, chunk_level, sym, scales, threads);
  threads = clamp_threads(threads, St);
  uint64_t* lens = (uint64_t*)calloc((size_t)(St > 0 ? St : 1), sizeof(uint64_t));
  pthread_t th[256];
  tenc_job jobs[256];
  for (int i = 0; i < threads; ++i) {
    jobs[i] = (tenc_job){p, sym, chunk_level, cdf_anchor, cdf_delta,
                         St * i / threads, St * (i + 1) / threads, NULL, 0, lens, 0};
    pthread_create(&th[i], NULL, tenc_worker, &jobs[i]);
  }
  for (int i = 0; i < threads; ++i) pthread_join(th[i], NULL);
  int failed = 0;
  for (int i = 0; i < threads; ++i) failed |= jobs[i].failed;
  uint64_t total = 0;
  offsets[0] = 0;
  for (int64_t s = 0; s < St; ++s) { total += lens[s]; offsets[s + 1] = total; }
  if (!failed && total <= cap_words) {
    for (int i = 0; i < threads; ++i)
      memcpy(words + offsets[jobs[i].s_begin], jobs[i].buf, jobs[i].buf_words * sizeof(uint32_t));
  }
  for (int i = 0; i < threads; ++i) free(jobs[i].buf);
  free(lens);
  free(sym);
  return (failed || total > cap_words) ? -1 : (int64_t)total;
}

typedef struct {
  const cgo_params* p; const uint32_t* words; const uint64_t* offsets;
  const uint8_t* chunk_level; const uint16_t* cdf_anchor; const uint16_t* cdf_delta;
  int64_t s_begin, s_end; uint8_t* sym;
} tdec_job;

static void* tdec_worker(void* arg) {
  tdec_job* J = (tdec_job*)arg;
  const cgo_params* p = J->p;
  int64_t C = p->n_channels;
  const uint16_t** tabs = (const uint16_t**)malloc((size_t)C * sizeof(*tabs));
  for (int64_t s = J->s_begin; s < J->s_end; ++s) {
    tok_stream_t ts = locate_token(p, s);
    token_tables(p, J->chunk_level, J->cdf_anchor, J->cdf_delta, &ts, tabs);
    uint8_t* row = J->sym + (((ts.b * p->n_layers + ts.l) * 2 + ts.k) * p->n_tokens + ts.t) * C;
    cgo_ac_decode(J->words + J->offsets[s], J->offsets[s + 1] - J->offsets[s], C, tabs, row);
  }
  free(tabs);
  return NULL;
}

typedef struct {
  const cgo_params* p; const uint8_t* sym; const float* scales; const uint8_t* chunk_level;
  int64_t s_begin, s_end; uint16_t* kv_out;
} tdq_job;

static void* tdq_worker(void* arg) {
  tdq_job* J = (tdq_job*)arg;
  const cgo_params* p = J->p;
  uint8_t* col = (uint8_t*)malloc((size_t)p->chunk_len);
  for (int64_t s = J->s_begin; s < J->s_end; ++s) {
    stream_t st = locate(p, NULL, s);
    int lv = level_of(p, J->chunk_level, &st);
    int64_t base = (((st.b * p->n_layers + st.l) * 2 + st.k) * p->n_tokens + st.t0) *
                   p->n_channels + st.ch;
    for (int64_t j = 0; j < st.n; ++j) col[j] = J->sym[base + j * p->n_channels];
    float sc = J->scales[s];
    cgo_dequantize_stream(col, st.n, p->group_size, sc, bin_width(p, st.l, lv, sc),
                          J->kv_out + base, p->n_channels);
  }
  free(col);
  return NULL;
}

/* Decode every token stream, then reconstruct each channel stream from its symbols. */
int cg_decode_tokens_ref(const cgo_params* p, const uint32_t* words, const uint64_t* offsets,
                         const float* scales, const uint8_t* chunk_level,
                         const uint16_t* cdf_anchor, const uint16_t* cdf_delta,
                         uint16_t* kv_out, int threads) {
  int64_t St = cgo_num_token_streams(p);
  int64_t n_elem = St * p->n_channels;
  uint8_t* sym = (uint8_t*)malloc((size_t)(n_elem > 0 ? n_elem : 1));
  int tt = clamp_threads(threads, St);
  pthread_t th[256];
  tdec_job jobs[256];
  for (int i = 0; i < tt; ++i) {
    jobs[i] = (tdec_job){p, words, offsets, chunk_level, cdf_anchor, cdf_delta,
                         St * i / tt, St * (i + 1) / tt, sym};
    pthread_create(&th[i], NULL, tdec_worker, &jobs[i]);
  }
  for (int i = 0; i < tt; ++i) pthread_join(th[i], NULL);
  int64_t S = cgo_num_streams(p);
  int tq = clamp_threads(threads, S);
  tdq_job qj[256];
  for (int i = 0; i < tq; ++i) {
    qj[i] = (tdq_job){p, sym, scales, chunk_level, S * i / tq, S * (i + 1) / tq, kv_out};
    pthread_create(&th[i], NULL, tdq_worker, &qj[i]);
  }
  for (int i = 0; i < tq; ++i) pthread_join(th[i], NULL);
  free(sym);
  return 0;
}
