/*
 * wc_oracle.c -- CPU ORACLE for the chunked rANS weight codec.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow, single-threaded
 * statement of what the GPU decode path must reproduce.  Only the tests, the
 * package smoke check and the benchmark's CPU-baseline leg load it.  It shares
 * no code, header, table or constant with the HIP library; everything below
 * is written out from the paper and from the format readings documented next
 * to each function.
 *
 * Paper: "Approaching Shannon Bound with Lossless LLM Weight Compression".
 *   Sec. II-B   per-tensor empirical entropy over format-defined symbols,
 *               element-weighted model entropy.
 *   Sec. IV-A   tile-partitioned, independently decodable ANS substreams with
 *               an offset index table.
 *   Sec. V-B    offline compression: static frequency table, independent
 *               initial state per tile.
 *   Alg. 2      lane-parallel rANS decode: slot = state mod 2^b, table
 *               lookup (symbol, freq, cumfreq), state <- f*floor(s/2^b)+slot-c,
 *               renormalise from the interleaved stream.
 *   Sec. VI-F   metadata closed form 4 B * N_tiles + 2^b * 4 B (Table 3).
 *
 * Every arithmetic step is integer except the entropy (fp64).  Nothing here
 * is blocked, fused or reordered beyond what the definitions state.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------ */
/* Constants of the format (own copy; see the format readings).              */

#define ORC_DT_BF16 1
#define ORC_DT_FP16 2
#define ORC_DT_U8 3
#define ORC_DT_U4 4
#define ORC_DT_FP8_E4M3 5   /* 1-byte codes: coded as byte symbols, like ORC_DT_U8 */
#define ORC_DT_FP8_E5M2 6
#define ORC_DT_FP4_E2M1 7   /* packed 4-bit codes: nibble symbols, like ORC_DT_U4 */

#define ORC_PROB_BITS 12u
#define ORC_M (1u << ORC_PROB_BITS)   /* table total 2^12 (Sec. VI-F, b = 12) */
#define ORC_STATE_LOW (1u << 16)       /* rANS lower bound of the state        */
#define ORC_MAGIC 0x31424357u          /* bytes 'W','C','B','1'                */
#define ORC_VERSION 5u

#define ORC_OK 0
#define ORC_EINVAL (-1)
#define ORC_ENOMEM (-2)
#define ORC_ECORRUPT (-3)

/* ------------------------------------------------------------------------ */
/* Little-endian byte access, written out so the layout is explicit.         */

static void put16(uint8_t* p, uint32_t v) { p[0] = (uint8_t)v; p[1] = (uint8_t)(v >> 8); }
static void put32(uint8_t* p, uint32_t v) {
  for (int i = 0; i < 4; i++) p[i] = (uint8_t)(v >> (8 * i));
}
static void put64(uint8_t* p, uint64_t v) {
  for (int i = 0; i < 8; i++) p[i] = (uint8_t)(v >> (8 * i));
}
static uint32_t get16(const uint8_t* p) { return (uint32_t)p[0] | ((uint32_t)p[1] << 8); }
static uint32_t get32(const uint8_t* p) {
  uint32_t v = 0;
  for (int i = 3; i >= 0; i--) v = (v << 8) | p[i];
  return v;
}
static uint64_t get64(const uint8_t* p) {
  uint64_t v = 0;
  for (int i = 7; i >= 0; i--) v = (v << 8) | p[i];
  return v;
}
static uint64_t round16(uint64_t x) { return (x + 15) / 16 * 16; }

/* ------------------------------------------------------------------------ */
/* Field split (Sec. II-B: symbols are determined by the numeric format).    */
/*
 * A 16-bit float word w (bf16, or fp16 with the same bit positions) is split
 * into a coded byte -- bits 14..7, i.e. the bf16 exponent -- and a raw byte
 * holding the sign (bit 15) in its top bit and bits 6..0 below it.  The split
 * is a bit permutation, so every pattern (NaN, Inf, subnormal, -0) survives.
 */
uint8_t orc_coded16(uint16_t w) { return (uint8_t)((w >> 7) & 0xFF); }
uint8_t orc_raw16(uint16_t w) { return (uint8_t)(((w >> 15) & 1) << 7 | (w & 0x7F)); }
uint16_t orc_merge16(uint8_t coded, uint8_t raw) {
  uint32_t sign = (raw >> 7) & 1;
  uint32_t low7 = raw & 0x7F;
  return (uint16_t)((sign << 15) | ((uint32_t)coded << 7) | low7);
}

static int dtype_ok(uint32_t dt) { return dt >= ORC_DT_BF16 && dt <= ORC_DT_FP4_E2M1; }
static int has_raw(uint32_t dt) { return dt == ORC_DT_BF16 || dt == ORC_DT_FP16; }
/* Every byte of the tensor is one symbol (int8, fp8). */
static int is_byte(uint32_t dt) {
  return dt == ORC_DT_U8 || dt == ORC_DT_FP8_E4M3 || dt == ORC_DT_FP8_E5M2;
}
/* Every nibble is one symbol, low nibble first (int4, fp4). */
static int is_nibble(uint32_t dt) { return dt == ORC_DT_U4 || dt == ORC_DT_FP4_E2M1; }
static uint32_t alphabet_of(uint32_t dt) { return is_nibble(dt) ? 16u : 256u; }
/* Symbols per lane-group: a lane-group always covers 16 output bytes. */
static uint32_t group_of(uint32_t dt) {
  return is_nibble(dt) ? 32u : (is_byte(dt) ? 16u : 8u);
}

/* Number of coded symbols of a tensor of `nbytes` storage bytes. */
static uint64_t n_symbols_of(uint32_t dt, uint64_t nbytes) {
  if (is_nibble(dt)) return 2 * nbytes;
  if (is_byte(dt)) return nbytes;
  return nbytes / 2;
}

/* ---- 2-D tiles (Sec. IV-A: each tile of the weight matrix is its own     */
/* substream).  A tensor is tiled when it has a shape the tile divides       */
/* exactly, the tile width is a power of two covering whole lane-groups, and */
/* a tile's bytes are a valid chunk size.  Its symbols are then coded in     */
/* tile-major order (tiles row by row, each tile row-major) with one chunk   */
/* per tile; the raw bytes follow the same order.                            */

static int pow2(uint64_t x) { return x && !(x & (x - 1)); }

/* Within a tile, order 0 is row-major.  Order 1 (column blocks) lists the   */
/* tile's lane-groups of W elements k-block by k-block, every row of the     */
/* tile per block: lane-group g is row g mod tile_r, columns                 */
/* [(g div tile_r) W, (g div tile_r) W + W).  With tile_r rANS lanes, lane l */
/* then always decodes row l, which lets a decoder form whole dot products   */
/* per lane.  Order 1 needs tile_r to be a power of two.                     */
static int tile_ok(uint32_t dt, uint64_t rows, uint64_t cols, uint32_t tr, uint32_t tc,
                   uint32_t order) {
  if (!tr || !tc || !rows || !cols || order > 1) return 0;
  if (rows % tr || cols % tc || !pow2(tc) || tc < group_of(dt)) return 0;
  if (order == 1 && !pow2(tr)) return 0;
  uint64_t cb = (uint64_t)tr * tc * 16 / group_of(dt); /* 16 bytes per lane-group */
  return cb >= 256 && cb <= (1u << 20) && cb % 256 == 0;
}

/* Element index (row-major in the tensor) of tile-major symbol k. */
static uint64_t tile_element(uint64_t k, uint64_t cols, uint32_t tr, uint32_t tc, uint32_t order,
                             uint32_t W) {
  uint64_t per = (uint64_t)tr * tc, t = k / per, in = k % per;
  uint64_t ntc = cols / tc, a = t / ntc, bcol = t % ntc;
  if (order == 0) return (a * tr + in / tc) * cols + bcol * tc + in % tc;
  uint64_t g = in / W, kb = g / tr, n = g % tr;
  return (a * tr + n) * cols + bcol * tc + kb * W + in % W;
}

/*
 * Coded symbol stream (and raw bytes for 16-bit types) of a tensor.
 * int8 / fp8: one symbol per byte.  int4 / fp4: two symbols per byte, low
 * nibble first.
 */
int orc_symbols(uint32_t dt, const uint8_t* data, uint64_t nbytes, uint8_t* coded,
                uint8_t* raw) {
  if (!dtype_ok(dt)) return ORC_EINVAL;
  if (has_raw(dt) && (nbytes % 2) != 0) return ORC_EINVAL;
  uint64_t n = n_symbols_of(dt, nbytes);
  for (uint64_t i = 0; i < n; i++) {
    if (is_byte(dt)) {
      coded[i] = data[i];
    } else if (is_nibble(dt)) {
      uint8_t byte = data[i / 2];
      coded[i] = (i % 2 == 0) ? (byte & 0x0F) : (byte >> 4);
    } else {
      uint16_t w = (uint16_t)(data[2 * i] | (data[2 * i + 1] << 8));
      coded[i] = orc_coded16(w);
      raw[i] = orc_raw16(w);
    }
  }
  return ORC_OK;
}

/* Inverse of orc_symbols: write tensor bytes for symbol range [s0, s0+n). */
/* Symbol s0 + k is written to element map(s0 + k): the identity, or the     */
/* tile order when cols > 0.                                                 */
static void put_symbols(uint32_t dt, const uint8_t* coded, const uint8_t* raw, uint64_t s0,
                        uint64_t n, uint8_t* out, uint64_t cols, uint32_t tr, uint32_t tc,
                        uint32_t order) {
  for (uint64_t k = 0; k < n; k++) {
    uint64_t i = cols ? tile_element(s0 + k, cols, tr, tc, order, group_of(dt)) : s0 + k;
    if (is_byte(dt)) {
      out[i] = coded[k];
    } else if (is_nibble(dt)) {
      if (i % 2 == 0)
        out[i / 2] = (uint8_t)((out[i / 2] & 0xF0) | (coded[k] & 0x0F));
      else
        out[i / 2] = (uint8_t)((out[i / 2] & 0x0F) | ((coded[k] & 0x0F) << 4));
    } else {
      uint16_t w = orc_merge16(coded[k], raw[k]);
      out[2 * i] = (uint8_t)(w & 0xFF);
      out[2 * i + 1] = (uint8_t)(w >> 8);
    }
  }
}

/* ------------------------------------------------------------------------ */
/* Histogram and empirical Shannon entropy (Sec. II-B).                      */

void orc_histogram(const uint8_t* sym, uint64_t n, uint64_t* hist /*[256]*/) {
  for (int s = 0; s < 256; s++) hist[s] = 0;
  for (uint64_t i = 0; i < n; i++) hist[sym[i]]++;
}

/* H = -sum_i p_i log2 p_i with p_i = count_i / n, over `alphabet` bins. */
double orc_entropy(const uint64_t* hist, uint32_t alphabet) {
  uint64_t n = 0;
  for (uint32_t s = 0; s < alphabet; s++) n += hist[s];
  if (n == 0) return 0.0;
  double h = 0.0;
  for (uint32_t s = 0; s < alphabet; s++) {
    if (hist[s] == 0) continue;
    double p = (double)hist[s] / (double)n;
    h -= p * log2(p);
  }
  return h;
}

/* Per-field statistics of one tensor. */
typedef struct {
  uint32_t n_fields;       /* 1 (int8/int4) or 2 (coded byte + raw byte) */
  uint32_t alphabet[2];
  uint64_t count[2];
  uint64_t hist[2][256];
  double H[2];             /* bits per symbol */
  double H_joint16;        /* over whole 16-bit words; NaN for 8/4-bit types */
  double bound_bytes;      /* sum over fields of count * H / 8 */
  double bound_bytes_raw8; /* coded field at H, raw field at 8 bits */
} orc_stats;

int orc_analyze(uint32_t dt, const uint8_t* data, uint64_t nbytes, orc_stats* st) {
  if (!dtype_ok(dt) || !st) return ORC_EINVAL;
  if (has_raw(dt) && nbytes % 2) return ORC_EINVAL;
  memset(st, 0, sizeof(*st));
  uint64_t n = n_symbols_of(dt, nbytes);
  uint8_t* coded = (uint8_t*)malloc(n ? n : 1);
  uint8_t* raw = (uint8_t*)malloc(n ? n : 1);
  if (!coded || !raw) {
    free(coded);
    free(raw);
    return ORC_ENOMEM;
  }
  orc_symbols(dt, data, nbytes, coded, raw);
  st->n_fields = has_raw(dt) ? 2 : 1;
  st->alphabet[0] = alphabet_of(dt);
  st->count[0] = n;
  orc_histogram(coded, n, st->hist[0]);
  st->H[0] = orc_entropy(st->hist[0], st->alphabet[0]);
  st->bound_bytes = (double)n * st->H[0] / 8.0;
  st->bound_bytes_raw8 = st->bound_bytes;
  st->H_joint16 = NAN;
  if (has_raw(dt)) {
    st->alphabet[1] = 256;
    st->count[1] = n;
    orc_histogram(raw, n, st->hist[1]);
    st->H[1] = orc_entropy(st->hist[1], 256);
    st->bound_bytes += (double)n * st->H[1] / 8.0;
    st->bound_bytes_raw8 += (double)n;
    uint64_t* h16 = (uint64_t*)calloc(65536, sizeof(uint64_t));
    if (!h16) {
      free(coded);
      free(raw);
      return ORC_ENOMEM;
    }
    for (uint64_t i = 0; i < n; i++) h16[data[2 * i] | (data[2 * i + 1] << 8)]++;
    st->H_joint16 = 0.0;
    for (uint32_t w = 0; w < 65536; w++) {
      if (!h16[w]) continue;
      double p = (double)h16[w] / (double)n;
      st->H_joint16 -= p * log2(p);
    }
    free(h16);
  }
  free(coded);
  free(raw);
  return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Normalisation of counts to a 2^12 total (Sec. VI-F: b = 12 probability    */
/* bits).  The paper does not give the rounding rule; the reading used is an */
/* integer largest-remainder rule:                                           */
/*   f_s = floor(c_s * 4096 / n), remainder r_s = c_s * 4096 mod n;          */
/*   a present symbol rounded to 0 is forced to 1;                           */
/*   a shortfall d > 0 is handed out +1 each to the d non-forced symbols     */
/*   with the largest remainder (ties: lower symbol first);                  */
/*   an excess is removed -1 at a time from the largest f (ties: lower).     */

int orc_normalise(const uint64_t* hist, uint32_t alphabet, uint32_t* freq) {
  if (alphabet == 0 || alphabet > 256) return ORC_EINVAL;
  uint64_t n = 0;
  for (uint32_t s = 0; s < alphabet; s++) n += hist[s];
  for (uint32_t s = 0; s < alphabet; s++) freq[s] = 0;
  if (n == 0) return ORC_OK; /* empty field: no table */
  uint64_t rem[256];
  int forced[256], chosen[256];
  int64_t total = 0;
  for (uint32_t s = 0; s < alphabet; s++) {
    /* c * 4096 fits in 64 bits for any c < 2^52 */
    freq[s] = (uint32_t)((hist[s] * ORC_M) / n);
    rem[s] = (hist[s] * ORC_M) % n;
    forced[s] = 0;
    chosen[s] = 0;
    if (hist[s] > 0 && freq[s] == 0) {
      freq[s] = 1;
      forced[s] = 1;
    }
    total += freq[s];
  }
  int64_t d = (int64_t)ORC_M - total;
  while (d > 0) {
    int best = -1;
    for (uint32_t s = 0; s < alphabet; s++) {
      if (hist[s] == 0 || forced[s] || chosen[s]) continue;
      if (best < 0 || rem[s] > rem[best]) best = (int)s;
    }
    if (best < 0) return ORC_EINVAL;
    freq[best] += 1;
    chosen[best] = 1; /* each symbol receives at most one extra unit */
    d--;
  }
  while (d < 0) {
    int best = 0;
    for (uint32_t s = 1; s < alphabet; s++)
      if (freq[s] > freq[best]) best = (int)s;
    freq[best] -= 1;
    d++;
  }
  return ORC_OK;
}

/* cum_s = sum_{t < s} f_t */
static void cumulative(const uint32_t* freq, uint32_t alphabet, uint32_t* cum) {
  uint32_t c = 0;
  for (uint32_t s = 0; s < alphabet; s++) {
    cum[s] = c;
    c += freq[s];
  }
}

/* ------------------------------------------------------------------------ */
/* Lane interleave of one chunk (Sec. V-C-3: R substreams, one per lane;    */
/* indices follow the interleaved decode order).  Reading used: symbol i of */
/* a chunk belongs to lane (i mod L*W) div W, at step                        */
/* (i div L*W) * W + (i mod W).  So W consecutive symbols (16 output bytes) */
/* belong to one lane, and a row of L*W symbols is spread over the lanes.   */

static uint64_t symbol_at(uint64_t t, uint32_t lane, uint32_t L, uint32_t W) {
  return (t / W) * (uint64_t)L * W + (uint64_t)lane * W + (t % W);
}

static uint64_t steps_of(uint64_t n, uint32_t L, uint32_t W) {
  uint64_t rows = (n + (uint64_t)L * W - 1) / ((uint64_t)L * W);
  return rows * W;
}

static uint32_t states_of(uint64_t n, uint32_t L, uint32_t W) {
  uint64_t groups = (n + W - 1) / W;
  return (uint32_t)(groups < L ? groups : L);
}

/* ------------------------------------------------------------------------ */
/* Lane states that carry data (format version 4; a reading of ours, the     */
/* paper's encoder starts every lane from the same fixed state, Sec. V-B).   */
/* The encoder's start state is information the decoder gets back for free  */
/* at the end of the lane, so an untiled chunk spends it: lane l starts at   */
/* 2^S + D, D packing the lane's first K_l = min(K, its symbols) symbols     */
/* (step t's symbol in bits [b t, b t + b)), and those steps are not coded.   */
/*   exponent bytes of a 16-bit format   K = 2, b = 8, S = 16                */
/*   byte symbols                        K = 3, b = 8, S = 24                */
/*   nibble symbols                      K = 7, b = 4, S = 28                */
/* K b <= S and 2^S + D < 2^32, so the start state is a valid state; a       */
/* decoded lane must end with x div 2^S = 1 and D below 2^(b K_l).  Tiled     */
/* chunks (the fused products' input) keep the plain start 2^16, K = 0.      */

typedef struct {
  uint32_t K, b, S;
} orc_carry;

static orc_carry carry_of(uint32_t dt, int tiled) {
  orc_carry c = {0, 8, 16};
  if (tiled) return c;
  if (has_raw(dt)) {
    c.K = 2;
  } else if (is_nibble(dt)) {
    c.K = 7;
    c.b = 4;
    c.S = 28;
  } else {
    c.K = 3;
    c.S = 24;
  }
  return c;
}

/* start state of lane l of a chunk of n symbols (sym in coding order) */
static uint32_t carry_state(orc_carry c, const uint8_t* sym, uint64_t n, uint32_t l, uint32_t L,
                            uint32_t W) {
  if (c.K == 0) return ORC_STATE_LOW;
  uint32_t D = 0;
  for (uint32_t t = 0; t < c.K; t++) {
    uint64_t i = symbol_at(t, l, L, W);
    if (i < n) D |= (uint32_t)sym[i] << (c.b * t);
  }
  return (1u << c.S) + D;
}

/* the carried symbols back from lane l's end state; ORC_ECORRUPT if the
   state is not 2^S + D with D inside the lane's K_l symbols */
static int carry_read(orc_carry c, uint32_t x, uint8_t* sym, uint64_t n, uint32_t l, uint32_t L,
                      uint32_t W) {
  if (c.K == 0) return x == ORC_STATE_LOW ? ORC_OK : ORC_ECORRUPT;
  if ((x >> c.S) != 1) return ORC_ECORRUPT;
  uint32_t D = x - (1u << c.S);
  uint32_t used = 0;
  for (uint32_t t = 0; t < c.K; t++) {
    uint64_t i = symbol_at(t, l, L, W);
    if (i >= n) continue;
    sym[i] = (uint8_t)((D >> (c.b * t)) & ((1u << c.b) - 1));
    used += c.b;
  }
  if (used < 32 && (D >> used) != 0) return ORC_ECORRUPT;
  return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* rANS coding of one chunk.                                                 */
/*
 * State x is a 32-bit integer kept in [2^16, 2^32); 16-bit words are moved
 * in and out; probabilities are f_s / 2^12.
 *   encode s:  if x >= f_s * 2^20: emit x mod 2^16, x = floor(x / 2^16)
 *              x = floor(x / f_s) * 2^12 + (x mod f_s) + cum_s
 *   decode:    slot = x mod 2^12; s = the symbol with cum_s <= slot < cum_s+f_s
 *              x = f_s * floor(x / 2^12) + slot - cum_s          (Alg. 2)
 *              if x < 2^16: x = x * 2^16 + next word
 * Lane l starts the encoder at init[l] (2^16 when init is NULL), any value in
 * [2^16, 2^32); decoding lane l ends in that same state, so a correct decode
 * ends with every lane back at its start and the whole word stream consumed.
 * Steps t < skip of every lane are left out of the coding on both sides.
 *
 * Word order: the encoder runs steps T-1..0 and, within a step, lanes L-1..0,
 * pushing words on a stack; the stream is that stack read from the top, so
 * the decoder, running steps 0..T-1 and lanes 0..L-1, meets the words in
 * stream order.
 */

int orc_encode_stream(const uint8_t* sym, uint64_t n, const uint32_t* freq, uint32_t alphabet,
                      uint32_t L, uint32_t W, const uint32_t* init /*[L] or NULL*/,
                      uint32_t skip, uint32_t* states /*[L]*/, uint16_t* words,
                      uint64_t words_cap, uint64_t* n_words, uint32_t* n_states) {
  if (L == 0 || W == 0) return ORC_EINVAL;
  uint32_t cum[256];
  cumulative(freq, alphabet, cum);
  uint32_t A = states_of(n, L, W);
  uint64_t T = steps_of(n, L, W);
  for (uint32_t l = 0; l < A; l++) {
    states[l] = init ? init[l] : ORC_STATE_LOW;
    if (states[l] < ORC_STATE_LOW) return ORC_EINVAL;
  }
  /* the stack is written top-down at the end of `words` and moved later */
  uint64_t pushed = 0;
  for (uint64_t tt = T; tt-- > skip;) {
    for (uint32_t l = A; l-- > 0;) {
      uint64_t i = symbol_at(tt, l, L, W);
      if (i >= n) continue;
      uint32_t s = sym[i];
      if (s >= alphabet || freq[s] == 0) return ORC_EINVAL;
      uint64_t x = states[l];
      uint64_t f = freq[s];
      if (x >= (f << 20)) {
        if (pushed >= words_cap) return ORC_ENOMEM;
        words[words_cap - 1 - pushed] = (uint16_t)(x & 0xFFFF);
        pushed++;
        x >>= 16;
      }
      x = (x / f) * ORC_M + (x % f) + cum[s];
      states[l] = (uint32_t)x;
    }
  }
  /* stack top (last pushed) is at words[words_cap - pushed]: stream order */
  memmove(words, words + (words_cap - pushed), pushed * sizeof(uint16_t));
  *n_words = pushed;
  *n_states = A;
  return ORC_OK;
}

/* Decodes steps skip..T-1 of every lane.  With final == NULL every lane must
   end at 2^16; otherwise the end states are returned there for the caller to
   check.  Either way the whole word stream must be consumed. */
int orc_decode_stream(const uint32_t* states_in, uint32_t n_states, const uint16_t* words,
                      uint64_t n_words, uint64_t n, const uint32_t* freq, uint32_t alphabet,
                      uint32_t L, uint32_t W, uint32_t skip, uint32_t* final /*[L] or NULL*/,
                      uint8_t* sym_out) {
  if (L == 0 || W == 0 || L > 4096) return ORC_EINVAL;
  uint32_t A = states_of(n, L, W);
  if (n_states != A) return ORC_ECORRUPT;
  uint32_t cum[256];
  cumulative(freq, alphabet, cum);
  uint32_t total = 0;
  for (uint32_t s = 0; s < alphabet; s++) total += freq[s];
  if (n > 0 && total != ORC_M) return ORC_EINVAL;
  /* slot -> symbol: symbol s owns slots cum_s .. cum_s + f_s - 1 */
  uint8_t slot_sym[ORC_M];
  memset(slot_sym, 0, sizeof(slot_sym));
  for (uint32_t s = 0; s < alphabet; s++)
    for (uint32_t k = 0; k < freq[s] && cum[s] + k < ORC_M; k++) slot_sym[cum[s] + k] = (uint8_t)s;
  uint32_t x[4096];
  for (uint32_t l = 0; l < A; l++) x[l] = states_in[l];
  uint64_t cursor = 0;
  uint64_t T = steps_of(n, L, W);
  int bad = 0;
  for (uint64_t t = skip; t < T; t++) {
    for (uint32_t l = 0; l < A; l++) {
      uint64_t i = symbol_at(t, l, L, W);
      if (i >= n) continue;
      uint32_t slot = x[l] & (ORC_M - 1);
      uint32_t s = slot_sym[slot];
      sym_out[i] = (uint8_t)s;
      x[l] = freq[s] * (x[l] >> ORC_PROB_BITS) + slot - cum[s];
      if (x[l] < ORC_STATE_LOW) {
        uint32_t w = 0;
        if (cursor < n_words)
          w = words[cursor];
        else
          bad = 1;
        cursor++;
        x[l] = (x[l] << 16) | w;
      }
    }
  }
  for (uint32_t l = 0; l < A; l++) {
    if (final)
      final[l] = x[l];
    else if (x[l] != ORC_STATE_LOW)
      bad = 1;
  }
  if (cursor != n_words) bad = 1;
  return bad ? ORC_ECORRUPT : ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Blob: header, tensor descriptors, tables, chunk index, the raw bytes and  */
/* the chunk records (layout readings in the design notes; Sec. IV-A / V-B   */
/* give per-tile substreams plus an offset table).                           */

typedef struct {
  const uint8_t* data;
  uint64_t nbytes;
  uint32_t dtype;
  uint64_t rows, cols; /* shape in symbol elements (0, 0 = none) */
} orc_tensor;

#define ORC_DESC 96u /* bytes per tensor descriptor */



static uint64_t symbols_per_chunk(uint32_t dt, uint32_t chunk_bytes) {
  return n_symbols_of(dt, chunk_bytes);
}

static uint64_t chunks_of(uint64_t n_sym, uint64_t per) { return (n_sym + per - 1) / per; }

void orc_free(void* p) { free(p); }

int orc_encode_blob(const orc_tensor* ts, uint32_t n_tensors, uint32_t chunk_bytes, uint32_t L,
                    uint32_t tile_r, uint32_t tile_c, uint32_t tile_order, uint32_t shared_tables,
                    uint8_t** blob_out, uint64_t* size_out) {
  if (!ts || !blob_out || !size_out) return ORC_EINVAL;
  if (n_tensors == 0 || n_tensors > 4096) return ORC_EINVAL;
  if (chunk_bytes < 256 || chunk_bytes > (1u << 20) || chunk_bytes % 256) return ORC_EINVAL;
  if (L < 1 || L > 64) return ORC_EINVAL;
  if ((tile_r == 0) != (tile_c == 0) || (tile_c && !pow2(tile_c)) || tile_order > 1)
    return ORC_EINVAL;

  for (uint32_t t = 0; t < n_tensors; t++) {
    uint32_t dt = ts[t].dtype;
    if (!dtype_ok(dt)) return ORC_EINVAL;
    if (has_raw(dt) && ts[t].nbytes % 2) return ORC_EINVAL;
    if ((ts[t].rows || ts[t].cols) && ts[t].rows * ts[t].cols != n_symbols_of(dt, ts[t].nbytes))
      return ORC_EINVAL;
  }

  /* pass 0: per tensor, chunk size (tile or flat) and chunk count */
  uint64_t n_chunks = 0;
  uint32_t* cbytes = (uint32_t*)calloc(n_tensors, sizeof(uint32_t));
  uint8_t* tiled = (uint8_t*)calloc(n_tensors, 1);
  if (!cbytes || !tiled) {
    free(cbytes);
    free(tiled);
    return ORC_ENOMEM;
  }
  for (uint32_t t = 0; t < n_tensors; t++) {
    uint32_t dt = ts[t].dtype;
    uint64_t n = n_symbols_of(dt, ts[t].nbytes);
    tiled[t] = (uint8_t)tile_ok(dt, ts[t].rows, ts[t].cols, tile_r, tile_c, tile_order);
    cbytes[t] = tiled[t] ? (uint32_t)((uint64_t)tile_r * tile_c * 16 / group_of(dt)) : chunk_bytes;
    n_chunks += chunks_of(n, symbols_per_chunk(dt, cbytes[t]));
  }
  int rc = n_chunks > 0xFFFFFFFEull ? ORC_EINVAL : ORC_OK;

  uint8_t** rec = (uint8_t**)calloc(n_chunks ? n_chunks : 1, sizeof(uint8_t*));
  uint64_t* rec_size = (uint64_t*)calloc(n_chunks ? n_chunks : 1, sizeof(uint64_t));
  uint32_t* freqs = (uint32_t*)calloc((size_t)n_tensors * 256, sizeof(uint32_t));
  uint8_t** raws = (uint8_t**)calloc(n_tensors, sizeof(uint8_t*));
  uint8_t** codeds = (uint8_t**)calloc(n_tensors, sizeof(uint8_t*));
  uint32_t* table_of = (uint32_t*)calloc(n_tensors, sizeof(uint32_t)); /* tensor -> table */
  uint64_t(*hist)[256] = (uint64_t(*)[256])calloc(n_tensors, sizeof(uint64_t[256]));
  if (!rec || !rec_size || !freqs || !raws || !codeds || !table_of || !hist) rc = ORC_ENOMEM;
  if (rc != ORC_OK) n_chunks = 0; /* nothing to free per chunk */

  /* pass 1: symbols in coding order (tile-major when tiled), histograms */
  for (uint32_t t = 0; t < n_tensors && rc == ORC_OK; t++) {
    uint32_t dt = ts[t].dtype;
    uint64_t n = n_symbols_of(dt, ts[t].nbytes);
    uint8_t* coded = (uint8_t*)malloc(n ? n : 1);
    uint8_t* raw = (uint8_t*)malloc(n ? n : 1);
    if (!coded || !raw) {
      free(coded);
      free(raw);
      rc = ORC_ENOMEM;
      break;
    }
    orc_symbols(dt, ts[t].data, ts[t].nbytes, coded, raw);
    if (tiled[t]) {
      uint8_t* c2 = (uint8_t*)malloc(n ? n : 1);
      uint8_t* r2 = (uint8_t*)malloc(n ? n : 1);
      if (!c2 || !r2) {
        free(c2);
        free(r2);
        free(coded);
        free(raw);
        rc = ORC_ENOMEM;
        break;
      }
      for (uint64_t k = 0; k < n; k++) {
        uint64_t e = tile_element(k, ts[t].cols, tile_r, tile_c, tile_order, group_of(dt));
        c2[k] = coded[e];
        r2[k] = raw[e];
      }
      free(coded);
      free(raw);
      coded = c2;
      raw = r2;
    }
    orc_histogram(coded, n, hist[t]);
    codeds[t] = coded;
    raws[t] = raw;
  }

  /* tables: one per tensor, or (layer codebook) one per dtype, normalised
     from the summed histogram of every tensor of that dtype */
  uint32_t n_tables = 0;
  for (uint32_t t = 0; t < n_tensors && rc == ORC_OK; t++) {
    uint32_t owner = t;
    if (shared_tables)
      for (uint32_t u = 0; u < t; u++)
        if (ts[u].dtype == ts[t].dtype) {
          owner = u;
          break;
        }
    if (owner == t) {
      uint64_t sum[256];
      memcpy(sum, hist[t], sizeof(sum));
      if (shared_tables)
        for (uint32_t u = t + 1; u < n_tensors; u++)
          if (ts[u].dtype == ts[t].dtype)
            for (int k = 0; k < 256; k++) sum[k] += hist[u][k];
      orc_normalise(sum, alphabet_of(ts[t].dtype), freqs + (size_t)t * 256);
      table_of[t] = n_tables++;
    } else {
      memcpy(freqs + (size_t)t * 256, freqs + (size_t)owner * 256, 256 * sizeof(uint32_t));
      table_of[t] = table_of[owner];
    }
  }

  /* pass 2: chunk records */
  uint64_t c_glob = 0;
  for (uint32_t t = 0; t < n_tensors && rc == ORC_OK; t++) {
    uint32_t dt = ts[t].dtype;
    uint64_t n = n_symbols_of(dt, ts[t].nbytes);
    uint32_t alpha = alphabet_of(dt), W = group_of(dt);
    uint64_t per = symbols_per_chunk(dt, cbytes[t]);
    uint64_t nc = chunks_of(n, per);
    for (uint64_t c = 0; c < nc; c++, c_glob++) {
      uint64_t s0 = c * per;
      uint64_t len = (n - s0) < per ? (n - s0) : per;
      /* each symbol pushes at most one word */
      uint64_t cap = len + 1;
      uint16_t* words = (uint16_t*)malloc(cap * sizeof(uint16_t));
      uint32_t states[64], init[64];
      uint64_t nw = 0;
      uint32_t A = 0;
      if (!words) {
        rc = ORC_ENOMEM;
        break;
      }
      orc_carry cy = carry_of(dt, tiled[t]);
      for (uint32_t l = 0; l < L; l++) init[l] = carry_state(cy, codeds[t] + s0, len, l, L, W);
      rc = orc_encode_stream(codeds[t] + s0, len, freqs + (size_t)t * 256, alpha, L, W, init,
                             cy.K, states, words, cap, &nw, &A);
      if (rc != ORC_OK) {
        free(words);
        break;
      }
      uint64_t sz = 16 + round16(4ull * A) + round16(2ull * nw);
      uint8_t* r = (uint8_t*)calloc(sz, 1);
      if (!r) {
        free(words);
        rc = ORC_ENOMEM;
        break;
      }
      put32(r + 0, (uint32_t)nw);
      put32(r + 4, A);
      put32(r + 8, (uint32_t)len);
      put32(r + 12, 0);
      for (uint32_t l = 0; l < A; l++) put32(r + 16 + 4 * l, states[l]);
      uint8_t* wp = r + 16 + round16(4ull * A);
      for (uint64_t k = 0; k < nw; k++) put16(wp + 2 * k, words[k]);
      free(words);
      rec[c_glob] = r;
      rec_size[c_glob] = sz;
    }
  }

  /* pass 3: lay out the blob */
  uint64_t off_desc = 64;
  uint64_t off_tables = off_desc + (uint64_t)ORC_DESC * n_tensors;
  uint64_t* freq_off = (uint64_t*)calloc(n_tensors, sizeof(uint64_t));
  uint64_t* raw_off_t = (uint64_t*)calloc(n_tensors, sizeof(uint64_t));
  if (!freq_off || !raw_off_t) rc = ORC_ENOMEM;
  uint64_t pos = off_tables;
  for (uint32_t t = 0; t < n_tensors && rc == ORC_OK; t++) {
    uint32_t owner = t;
    for (uint32_t u = 0; u < t; u++)
      if (table_of[u] == table_of[t]) {
        owner = u;
        break;
      }
    if (owner == t) {
      freq_off[t] = pos;
      pos += round16(2ull * alphabet_of(ts[t].dtype));
    } else {
      freq_off[t] = freq_off[owner];
    }
  }
  /* the raw regions come before the records (format 5): their places depend
     on the tensor sizes only, not on how well the chunks code */
  uint64_t off_index = round16(pos);
  uint64_t off_raw = round16(off_index + 4ull * (n_chunks + 1));
  pos = off_raw;
  for (uint32_t t = 0; t < n_tensors && rc == ORC_OK; t++) {
    if (has_raw(ts[t].dtype)) {
      raw_off_t[t] = pos;
      pos += round16(n_symbols_of(ts[t].dtype, ts[t].nbytes));
    }
  }
  uint64_t off_records = pos;
  for (uint64_t c = 0; c < n_chunks && rc == ORC_OK; c++) pos += rec_size[c];
  uint64_t total = pos;
  if (rc == ORC_OK && total / 16 > 0xFFFFFFFFull) rc = ORC_EINVAL;

  uint8_t* b = NULL;
  if (rc == ORC_OK) {
    b = (uint8_t*)calloc(total, 1);
    if (!b) rc = ORC_ENOMEM;
  }
  if (rc == ORC_OK) {
    put32(b + 0, ORC_MAGIC);
    put16(b + 4, ORC_VERSION);
    put16(b + 6, 64);
    put32(b + 8, n_tensors);
    put32(b + 12, ORC_DESC);
    put64(b + 16, n_chunks);
    put64(b + 24, total);
    put64(b + 32, off_index);
    put64(b + 40, off_records);
    put64(b + 48, off_raw);
    put64(b + 56, 0);
    uint64_t first = 0;
    for (uint32_t t = 0; t < n_tensors; t++) {
      uint32_t dt = ts[t].dtype;
      uint64_t n = n_symbols_of(dt, ts[t].nbytes);
      uint64_t nc = chunks_of(n, symbols_per_chunk(dt, cbytes[t]));
      uint8_t* d = b + off_desc + (uint64_t)ORC_DESC * t;
      put32(d + 0, dt);
      put32(d + 4, cbytes[t]);
      put64(d + 8, n);
      put64(d + 16, ts[t].nbytes);
      put64(d + 24, first);
      put64(d + 32, nc);
      put16(d + 40, L);
      d[42] = (uint8_t)group_of(dt);
      d[43] = (uint8_t)ORC_PROB_BITS;
      put16(d + 44, alphabet_of(dt));
      put16(d + 46, 0);
      put64(d + 48, freq_off[t]);
      put64(d + 56, raw_off_t[t]);
      put64(d + 64, ts[t].rows);
      put64(d + 72, ts[t].cols);
      put32(d + 80, tiled[t] ? tile_r : 0);
      put32(d + 84, tiled[t] ? tile_c : 0);
      put32(d + 88, tiled[t] ? tile_order : 0);
      put32(d + 92, 0);
      for (uint32_t s = 0; s < alphabet_of(dt); s++)
        put16(b + freq_off[t] + 2 * s, freqs[(size_t)t * 256 + s]);
      if (has_raw(dt)) memcpy(b + raw_off_t[t], raws[t], n);
      first += nc;
    }
    pos = off_records;
    for (uint64_t c = 0; c < n_chunks; c++) {
      put32(b + off_index + 4 * c, (uint32_t)(pos / 16));
      memcpy(b + pos, rec[c], rec_size[c]);
      pos += rec_size[c];
    }
    put32(b + off_index + 4 * n_chunks, (uint32_t)(pos / 16));
  }

  for (uint64_t c = 0; rec && c < n_chunks; c++) free(rec[c]);
  for (uint32_t t = 0; t < n_tensors; t++) {
    if (raws) free(raws[t]);
    if (codeds) free(codeds[t]);
  }
  free(rec);
  free(rec_size);
  free(freqs);
  free(raws);
  free(codeds);
  free(hist);
  free(table_of);
  free(cbytes);
  free(tiled);
  free(freq_off);
  free(raw_off_t);
  if (rc != ORC_OK) {
    free(b);
    return rc;
  }
  *blob_out = b;
  *size_out = total;
  return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Blob reading and validation.                                              */

typedef struct {
  uint32_t dtype, chunk_bytes, L, W, prob_bits, alphabet, tile_r, tile_c, tile_order;
  uint64_t n_sym, out_bytes, first_chunk, n_chunks, freq_off, raw_off, rows, cols;
} orc_desc;

static int read_desc(const uint8_t* b, uint64_t size, uint32_t t, orc_desc* d) {
  uint32_t n_t = get32(b + 8);
  if (t >= n_t) return ORC_EINVAL;
  const uint8_t* p = b + 64 + (uint64_t)ORC_DESC * t;
  d->dtype = get32(p + 0);
  d->chunk_bytes = get32(p + 4);
  d->n_sym = get64(p + 8);
  d->out_bytes = get64(p + 16);
  d->first_chunk = get64(p + 24);
  d->n_chunks = get64(p + 32);
  d->L = get16(p + 40);
  d->W = p[42];
  d->prob_bits = p[43];
  d->alphabet = get16(p + 44);
  d->freq_off = get64(p + 48);
  d->raw_off = get64(p + 56);
  d->rows = get64(p + 64);
  d->cols = get64(p + 72);
  d->tile_r = get32(p + 80);
  d->tile_c = get32(p + 84);
  d->tile_order = get32(p + 88);
  if (!dtype_ok(d->dtype)) return ORC_EINVAL;
  if (d->prob_bits != ORC_PROB_BITS) return ORC_EINVAL;
  if (d->W != group_of(d->dtype) || d->alphabet != alphabet_of(d->dtype)) return ORC_EINVAL;
  if (d->L < 1 || d->L > 64) return ORC_EINVAL;
  if (d->chunk_bytes < 256 || d->chunk_bytes > (1u << 20) || d->chunk_bytes % 256)
    return ORC_EINVAL;
  if (d->n_sym != n_symbols_of(d->dtype, d->out_bytes)) return ORC_EINVAL;
  if (has_raw(d->dtype) && d->out_bytes % 2) return ORC_EINVAL;
  if (d->n_chunks != chunks_of(d->n_sym, symbols_per_chunk(d->dtype, d->chunk_bytes)))
    return ORC_EINVAL;
  if ((d->rows || d->cols) && d->rows * d->cols != d->n_sym) return ORC_EINVAL;
  if (!(d->tile_r || d->tile_c) && d->tile_order) return ORC_EINVAL;
  if (d->tile_r || d->tile_c) {
    if (!tile_ok(d->dtype, d->rows, d->cols, d->tile_r, d->tile_c, d->tile_order))
      return ORC_EINVAL;
    if (n_symbols_of(d->dtype, d->chunk_bytes) != (uint64_t)d->tile_r * d->tile_c)
      return ORC_EINVAL;
  }
  if (d->freq_off + 2ull * d->alphabet > size) return ORC_EINVAL;
  if (has_raw(d->dtype) && (d->raw_off > size || d->n_sym > size - d->raw_off))
    return ORC_EINVAL;
  return ORC_OK;
}

static int check_header(const uint8_t* b, uint64_t size) {
  if (!b || size < 64) return ORC_EINVAL;
  if (get32(b) != ORC_MAGIC || get16(b + 4) != ORC_VERSION || get16(b + 6) != 64 ||
      get32(b + 12) != ORC_DESC)
    return ORC_EINVAL;
  if (get64(b + 24) != size) return ORC_EINVAL;
  uint32_t n_t = get32(b + 8);
  uint64_t n_c = get64(b + 16);
  uint64_t off_index = get64(b + 32), off_rec = get64(b + 40), off_raw = get64(b + 48);
  if (n_t == 0 || 64 + (uint64_t)ORC_DESC * n_t > size) return ORC_EINVAL;
  if (off_index > size || n_c + 1 > (size - off_index) / 4) return ORC_EINVAL;
  if (off_index + 4 * (n_c + 1) > off_raw || off_raw > off_rec || off_rec > size)
    return ORC_EINVAL;
  uint64_t first = 0;
  for (uint32_t t = 0; t < n_t; t++) {
    orc_desc d;
    int rc = read_desc(b, size, t, &d);
    if (rc) return rc;
    if (d.first_chunk != first) return ORC_EINVAL;
    if (has_raw(d.dtype) && (d.raw_off < off_raw || d.n_sym > off_rec - d.raw_off))
      return ORC_EINVAL;
    first += d.n_chunks;
    if (d.n_sym > 0) {
      uint32_t sum = 0;
      for (uint32_t s = 0; s < d.alphabet; s++) sum += get16(b + d.freq_off + 2 * s);
      if (sum != ORC_M) return ORC_EINVAL;
    }
  }
  if (first != n_c) return ORC_EINVAL;
  for (uint64_t c = 0; c <= n_c; c++) {
    uint64_t o = 16ull * get32(b + off_index + 4 * c);
    if (o < off_rec || o > size) return ORC_EINVAL;
    if (c > 0 && o < 16ull * get32(b + off_index + 4 * (c - 1))) return ORC_EINVAL;
  }
  return ORC_OK;
}

/* Decode chunk `c` (index within tensor `t`) into the tensor buffer `out`. */
static int decode_one(const uint8_t* b, uint64_t size, const orc_desc* d, uint64_t c,
                      uint8_t* out) {
  uint64_t off_index = get64(b + 32);
  uint64_t g = d->first_chunk + c;
  uint64_t o0 = 16ull * get32(b + off_index + 4 * g);
  uint64_t o1 = 16ull * get32(b + off_index + 4 * (g + 1));
  if (o1 < o0 + 16 || o1 > size) return ORC_ECORRUPT;
  const uint8_t* r = b + o0;
  uint64_t per = symbols_per_chunk(d->dtype, d->chunk_bytes);
  uint64_t s0 = c * per;
  uint64_t len = (d->n_sym - s0) < per ? (d->n_sym - s0) : per;
  uint32_t nw = get32(r + 0), A = get32(r + 4), nsym = get32(r + 8);
  if (nsym != len || A != states_of(len, d->L, d->W)) return ORC_ECORRUPT;
  if (16 + round16(4ull * A) + round16(2ull * nw) != o1 - o0) return ORC_ECORRUPT;
  uint32_t states[64];
  for (uint32_t l = 0; l < A; l++) states[l] = get32(r + 16 + 4 * l);
  const uint8_t* wp = r + 16 + round16(4ull * A);
  uint16_t* words = (uint16_t*)malloc((nw ? nw : 1) * sizeof(uint16_t));
  uint8_t* sym = (uint8_t*)malloc(len ? len : 1);
  if (!words || !sym) {
    free(words);
    free(sym);
    return ORC_ENOMEM;
  }
  for (uint32_t k = 0; k < nw; k++) words[k] = (uint16_t)get16(wp + 2 * k);
  uint32_t freq[256];
  for (uint32_t s = 0; s < d->alphabet; s++) freq[s] = get16(b + d->freq_off + 2 * s);
  orc_carry cy = carry_of(d->dtype, d->tile_r != 0);
  uint32_t fin[64];
  memset(sym, 0, len ? len : 1);
  int rc = orc_decode_stream(states, A, words, nw, len, freq, d->alphabet, d->L, d->W, cy.K, fin,
                             sym);
  if (rc == ORC_OK || rc == ORC_ECORRUPT) {
    for (uint32_t l = 0; l < A; l++)
      if (carry_read(cy, fin[l], sym, len, l, d->L, d->W) != ORC_OK) rc = ORC_ECORRUPT;
    const uint8_t* raw = has_raw(d->dtype) ? b + d->raw_off + s0 : NULL;
    put_symbols(d->dtype, sym, raw, s0, len, out, d->tile_r ? d->cols : 0, d->tile_r, d->tile_c,
                d->tile_order);
  }
  free(words);
  free(sym);
  return rc;
}

int orc_blob_tensors(const uint8_t* b, uint64_t size, uint32_t* n_tensors) {
  int rc = check_header(b, size);
  if (rc) return rc;
  *n_tensors = get32(b + 8);
  return ORC_OK;
}

/* out_bytes, dtype and chunk count of tensor t */
int orc_blob_tensor_info(const uint8_t* b, uint64_t size, uint32_t t, uint64_t* out_bytes,
                         uint32_t* dtype, uint64_t* n_chunks, uint32_t* tile) {
  int rc = check_header(b, size);
  if (rc) return rc;
  orc_desc d;
  rc = read_desc(b, size, t, &d);
  if (rc) return rc;
  *out_bytes = d.out_bytes;
  *dtype = d.dtype;
  *n_chunks = d.n_chunks;
  if (tile) {
    tile[0] = d.tile_r;
    tile[1] = d.tile_c;
    tile[2] = d.chunk_bytes;
    tile[3] = d.tile_order;
  }
  return ORC_OK;
}

/* Decode every tensor; outs[t] must hold out_bytes of tensor t. */
int orc_decode_blob(const uint8_t* b, uint64_t size, uint8_t* const* outs) {
  int rc = check_header(b, size);
  if (rc) return rc;
  uint32_t n_t = get32(b + 8);
  int worst = ORC_OK;
  for (uint32_t t = 0; t < n_t; t++) {
    orc_desc d;
    read_desc(b, size, t, &d);
    for (uint64_t c = 0; c < d.n_chunks; c++) {
      rc = decode_one(b, size, &d, c, outs[t]);
      if (rc != ORC_OK) worst = rc;
    }
  }
  return worst;
}

/* Decode chunks [c0, c1) of tensor t into `out` (the whole tensor buffer). */
int orc_decode_chunks(const uint8_t* b, uint64_t size, uint32_t t, uint64_t c0, uint64_t c1,
                      uint8_t* out) {
  int rc = check_header(b, size);
  if (rc) return rc;
  orc_desc d;
  rc = read_desc(b, size, t, &d);
  if (rc) return rc;
  if (c0 > c1 || c1 > d.n_chunks) return ORC_EINVAL;
  int worst = ORC_OK;
  for (uint64_t c = c0; c < c1; c++) {
    rc = decode_one(b, size, &d, c, out);
    if (rc != ORC_OK) worst = rc;
  }
  return worst;
}

/* ------------------------------------------------------------------------ */
/* Metadata closed form (Sec. VI-F): a 4-byte offset per tile plus one      */
/* shared codebook of 2^b entries of 4 bytes, for a rows x cols matrix cut   */
/* into tile_r x tile_c tiles.                                               */

double orc_metadata_bytes(uint64_t rows, uint64_t cols, uint64_t tile_r, uint64_t tile_c,
                          uint32_t b) {
  double tiles = ((double)rows / (double)tile_r) * ((double)cols / (double)tile_c);
  return 4.0 * tiles + (double)(1ull << b) * 4.0;
}

/* ------------------------------------------------------------------------ */
/* What the fused decode-GEMM path computes (Alg. 1 / 3: the decoded tile is */
/* multiplied with the activations): y[m][n] = sum_k x[m][k] * w[n][k] for  */
/* bf16 w (rows x cols, row-major storage words) and bf16 x (M x cols), in  */
/* fp64, summed in k order.  abs_out[m][n] = sum_k |x[m][k] * w[n][k]|, the */
/* scale of any floating-point summation error.                             */

static double bf16_value(uint16_t h) {
  uint32_t u = (uint32_t)h << 16;
  float f;
  memcpy(&f, &u, 4);
  return (double)f;
}

int orc_gemv_bf16(const uint16_t* w, uint64_t rows, uint64_t cols, const uint16_t* x, uint32_t M,
                  double* y, double* abs_out) {
  if (!w || !x || !y || M == 0) return ORC_EINVAL;
  for (uint32_t m = 0; m < M; m++)
    for (uint64_t n = 0; n < rows; n++) {
      double s = 0.0, a = 0.0;
      for (uint64_t k = 0; k < cols; k++) {
        double p = bf16_value(x[(uint64_t)m * cols + k]) * bf16_value(w[n * cols + k]);
        s += p;
        a += fabs(p);
      }
      y[(uint64_t)m * rows + n] = s;
      if (abs_out) abs_out[(uint64_t)m * rows + n] = a;
    }
  return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* What the fused int8 decode-GEMM computes (W8A8, the sq8 format of Sec.    */
/* VI-A; Alg. 1 / 3): y[m][n] = sum_k x[m][k] * w[n][k] for int8 w (rows x   */
/* cols, row-major) and int8 x (M x cols), exactly, in 64-bit integers.      */

int orc_gemm_i8(const int8_t* w, uint64_t rows, uint64_t cols, const int8_t* x, uint32_t M,
                int64_t* y) {
  if (!w || !x || !y || M == 0) return ORC_EINVAL;
  for (uint32_t m = 0; m < M; m++)
    for (uint64_t n = 0; n < rows; n++) {
      int64_t s = 0;
      for (uint64_t k = 0; k < cols; k++)
        s += (int64_t)x[(uint64_t)m * cols + k] * (int64_t)w[n * cols + k];
      y[(uint64_t)m * rows + n] = s;
    }
  return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* What the fused decode-GEMM computes for fp8 weights with bf16 activations */
/* (the fp8 weight formats of Sec. VI-A): y[m][n] = sum_k x[m][k] *          */
/* fp8(w[n][k]), in fp64, summed in k order; abs_out as for orc_gemv_bf16.   */
/* e4m3 (OCP 8-bit float, E4M3): sign, 4 exponent bits with bias 7, 3        */
/* mantissa bits; exponent 0 is subnormal (m/8 * 2^-6); no infinities; the  */
/* two patterns with all exponent and mantissa bits set are NaN.             */
/* e5m2 (OCP 8-bit float, E5M2, the paper's FP8-E5M2): sign, 5 exponent bits */
/* with bias 15, 2 mantissa bits; exponent 0 is subnormal (m/4 * 2^-14);     */
/* exponent 31 is infinity (mantissa 0) or NaN (mantissa not 0).             */

double orc_e4m3_value(uint8_t v) {
  const int s = v >> 7, e = (v >> 3) & 15, m = v & 7;
  if (e == 15 && m == 7) return NAN;
  const double mag = e ? ldexp(1.0 + m / 8.0, e - 7) : ldexp(m / 8.0, -6);
  return s ? -mag : mag;
}

double orc_e5m2_value(uint8_t v) {
  const int s = v >> 7, e = (v >> 2) & 31, m = v & 3;
  double mag;
  if (e == 31) mag = m ? NAN : INFINITY;
  else mag = e ? ldexp(1.0 + m / 4.0, e - 15) : ldexp(m / 4.0, -14);
  return s ? -mag : mag;
}

/* ------------------------------------------------------------------------ */
/* MXFP4 weights (OCP microscaling; the paper's fp4 format, Sec. VI-A):      */
/* e2m1 codes (sign, 2 exponent bits with bias 1, 1 mantissa bit: 0, 0.5, 1, */
/* 1.5, 2, 3, 4, 6), two per byte with the even element in the low nibble,   */
/* and one e8m0 scale byte E per 32 consecutive weights of a row, worth      */
/* 2^(E - 127) (E = 255 is NaN).  What the fused decode-GEMM computes:       */
/* y[m][n] = sum_k x[m][k] * e2m1(w[n][k]) * 2^(E[n][k / 32] - 127), in fp64, */
/* summed in k order; abs_out as for orc_gemv_bf16.                         */

double orc_e2m1_value(uint8_t nibble) {
  const int s = (nibble >> 3) & 1, e = (nibble >> 1) & 3, m = nibble & 1;
  const double mag = e ? ldexp(1.0 + m / 2.0, e - 1) : m / 2.0;
  return s ? -mag : mag;
}

double orc_e8m0_value(uint8_t e) { return e == 255 ? NAN : ldexp(1.0, (int)e - 127); }

int orc_gemv_mxfp4(const uint8_t* w, const uint8_t* scales, uint64_t rows, uint64_t cols,
                   const uint16_t* x, uint32_t M, double* y, double* abs_out) {
  if (!w || !scales || !x || !y || M == 0 || cols % 32) return ORC_EINVAL;
  for (uint32_t m = 0; m < M; m++)
    for (uint64_t n = 0; n < rows; n++) {
      double s = 0.0, a = 0.0;
      for (uint64_t k = 0; k < cols; k++) {
        const uint8_t byte = w[(n * cols + k) / 2];
        const uint8_t code = (k & 1) ? byte >> 4 : byte & 15;
        const double v = orc_e2m1_value(code) * orc_e8m0_value(scales[n * (cols / 32) + k / 32]);
        double p = bf16_value(x[(uint64_t)m * cols + k]) * v;
        s += p;
        a += fabs(p);
      }
      y[(uint64_t)m * rows + n] = s;
      if (abs_out) abs_out[(uint64_t)m * rows + n] = a;
    }
  return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Group-quantised int4 weights (the paper's int4 and awq4 formats, Sec.     */
/* VI-A): codes two per byte (even element in the low nibble), one fp16      */
/* scale per 128 consecutive weights of a row, and either a zero point per   */
/* group (unsigned codes q, weight s (q - z); zeros one byte per group) or   */
/* none (two's-complement codes, weight s q).  What the fused decode-GEMM    */
/* computes: y[m][n] = sum_k x[m][k] * w[n][k], in fp64, summed in k order;  */
/* abs_out as for orc_gemv_bf16.                                             */

double orc_fp16_value(uint16_t h) {
  const int s = h >> 15, e = (h >> 10) & 31, m = h & 1023;
  double mag;
  if (e == 31) mag = m ? NAN : INFINITY;
  else mag = e ? ldexp(1.0 + m / 1024.0, e - 15) : ldexp(m / 1024.0, -14);
  return s ? -mag : mag;
}

int orc_gemv_int4(const uint8_t* w, const uint16_t* scales, const uint8_t* zeros, uint64_t rows,
                  uint64_t cols, const uint16_t* x, uint32_t M, double* y, double* abs_out) {
  if (!w || !scales || !x || !y || M == 0 || cols % 128) return ORC_EINVAL;
  for (uint32_t m = 0; m < M; m++)
    for (uint64_t n = 0; n < rows; n++) {
      double s = 0.0, a = 0.0;
      for (uint64_t k = 0; k < cols; k++) {
        const uint8_t byte = w[(n * cols + k) / 2];
        const int code = (k & 1) ? byte >> 4 : byte & 15;
        const uint64_t g = n * (cols / 128) + k / 128;
        const int q = zeros ? code - (int)zeros[g] : (code ^ 8) - 8;
        double p = bf16_value(x[(uint64_t)m * cols + k]) * (orc_fp16_value(scales[g]) * q);
        s += p;
        a += fabs(p);
      }
      y[(uint64_t)m * rows + n] = s;
      if (abs_out) abs_out[(uint64_t)m * rows + n] = a;
    }
  return ORC_OK;
}

/* fmt: 0 = e4m3, 1 = e5m2 */
int orc_gemv_fp8(const uint8_t* w, uint64_t rows, uint64_t cols, const uint16_t* x, uint32_t M,
                 uint32_t fmt, double* y, double* abs_out) {
  if (!w || !x || !y || M == 0 || fmt > 1) return ORC_EINVAL;
  for (uint32_t m = 0; m < M; m++)
    for (uint64_t n = 0; n < rows; n++) {
      double s = 0.0, a = 0.0;
      for (uint64_t k = 0; k < cols; k++) {
        const uint8_t c = w[n * cols + k];
        double p = bf16_value(x[(uint64_t)m * cols + k]) *
                   (fmt ? orc_e5m2_value(c) : orc_e4m3_value(c));
        s += p;
        a += fabs(p);
      }
      y[(uint64_t)m * rows + n] = s;
      if (abs_out) abs_out[(uint64_t)m * rows + n] = a;
    }
  return ORC_OK;
}
