// wc_host.cpp -- host half of libwc: field split, analysis, normalisation,
// chunk-parallel rANS encoder, blob assembly and validation.
//
// Paper: Sec. II-B (symbols defined by the numeric format, per-tensor
// empirical entropy), Sec. V-B (offline compression into independently addressable tiles, with a
// static table and independently initialised states), Sec. VI-F (b = 12
// probability bits; an offset entry per independently decodable unit).
#include <math.h>
#include <string.h>

#include <algorithm>
#include <array>
#include <atomic>
#include <memory>
#include <new>
#include <thread>
#include <vector>

#include "wc_internal.h"

namespace wc {
namespace {

// ---------------------------------------------------------------------------
// Little-endian field access.

inline void st16(uint8_t* p, uint32_t v) { memcpy(p, &v, 2); }
inline void st32(uint8_t* p, uint32_t v) { memcpy(p, &v, 4); }
inline void st64(uint8_t* p, uint64_t v) { memcpy(p, &v, 8); }
inline uint32_t ld16(const uint8_t* p) { uint16_t v; memcpy(&v, p, 2); return v; }
inline uint32_t ld32(const uint8_t* p) { uint32_t v; memcpy(&v, p, 4); return v; }
inline uint64_t ld64(const uint8_t* p) { uint64_t v; memcpy(&v, p, 8); return v; }

unsigned thread_count(uint32_t requested) {
  if (requested) return requested;
  unsigned h = std::thread::hardware_concurrency();
  return h ? h : 1;
}

// Run fn(i) for i in [0, n) on `threads` workers pulling indices from a counter.
template <class F>
void parallel_for(uint64_t n, unsigned threads, F&& fn) {
  if (n == 0) return;
  threads = (unsigned)std::min<uint64_t>(threads, n);
  if (threads <= 1) {
    for (uint64_t i = 0; i < n; i++) fn(i);
    return;
  }
  std::atomic<uint64_t> next{0};
  std::vector<std::thread> pool;
  pool.reserve(threads);
  for (unsigned t = 0; t < threads; t++)
    pool.emplace_back([&] {
      for (uint64_t i; (i = next.fetch_add(1, std::memory_order_relaxed)) < n;) fn(i);
    });
  for (auto& th : pool) th.join();
}

// ---------------------------------------------------------------------------
// Field split (Sec. II-B): 16-bit words -> coded byte (bits 14..7) and raw
// byte (bit 15 -> bit 7, bits 6..0); int8 / fp8 -> byte; int4 / fp4 -> nibbles,
// low first.

// Symbols [s0, s1) of the tensor at `src`; coded[k] / raw[k] receive symbol s0 + k.
void split_range(uint32_t dt, const uint8_t* src, uint64_t s0, uint64_t s1, uint8_t* coded,
                 uint8_t* raw) {
  if (is_byte(dt)) {
    memcpy(coded, src + s0, s1 - s0);
  } else if (is_nibble(dt)) {
    for (uint64_t i = s0; i < s1; i++) {
      uint8_t b = src[i >> 1];
      coded[i - s0] = (i & 1) ? (b >> 4) : (b & 15);
    }
  } else {
    const uint8_t* w = src + 2 * s0;
    for (uint64_t k = 0; k < s1 - s0; k++, w += 2) {
      uint32_t v = w[0] | (uint32_t(w[1]) << 8);
      coded[k] = uint8_t(v >> 7);
      raw[k] = uint8_t(((v >> 8) & 0x80) | (v & 0x7F));
    }
  }
}

constexpr uint64_t kSplitBlock = 1u << 20;

void split_tensor(uint32_t dt, const uint8_t* src, uint64_t n, uint8_t* coded, uint8_t* raw,
                  unsigned threads) {
  uint64_t blocks = (n + kSplitBlock - 1) / kSplitBlock;
  parallel_for(blocks, threads, [&](uint64_t b) {
    uint64_t s0 = b * kSplitBlock, s1 = std::min(n, s0 + kSplitBlock);
    split_range(dt, src, s0, s1, coded + s0, raw ? raw + s0 : nullptr);
  });
}

void histogram(const uint8_t* sym, uint64_t n, uint64_t* hist, unsigned threads) {
  uint64_t blocks = (n + kSplitBlock - 1) / kSplitBlock;
  std::vector<uint64_t> part(blocks * 256, 0);
  parallel_for(blocks, threads, [&](uint64_t b) {
    uint64_t s0 = b * kSplitBlock, s1 = std::min(n, s0 + kSplitBlock);
    uint64_t* h = part.data() + b * 256;
    for (uint64_t i = s0; i < s1; i++) h[sym[i]]++;
  });
  for (int s = 0; s < 256; s++) hist[s] = 0;
  for (uint64_t b = 0; b < blocks; b++)
    for (int s = 0; s < 256; s++) hist[s] += part[b * 256 + s];
}

double entropy_bits(const uint64_t* hist, uint32_t bins) {
  uint64_t n = 0;
  for (uint32_t s = 0; s < bins; s++) n += hist[s];
  if (!n) return 0.0;
  double h = 0.0, inv = 1.0 / double(n);
  for (uint32_t s = 0; s < bins; s++)
    if (hist[s]) {
      double p = double(hist[s]) * inv;
      h -= p * log2(p);
    }
  return h;
}

// ---------------------------------------------------------------------------
// Normalisation to a 2^12 total (Sec. VI-F, b = 12).  Integer largest
// remainder: floor shares, present symbols at least 1, the shortfall to the
// largest remainders (lower symbol on ties, one unit each), an excess taken
// one unit at a time from the largest frequency (lower symbol on ties).

void normalise(const uint64_t* hist, uint32_t alpha, uint32_t* freq) {
  uint64_t n = 0;
  for (uint32_t s = 0; s < alpha; s++) n += hist[s];
  std::fill(freq, freq + alpha, 0u);
  if (!n) return;
  struct Cand { uint64_t rem; uint32_t sym; };
  std::vector<Cand> cands;
  int64_t sum = 0;
  for (uint32_t s = 0; s < alpha; s++) {
    if (!hist[s]) continue;
    uint64_t scaled = hist[s] * uint64_t(kTableSize);
    uint32_t f = uint32_t(scaled / n);
    if (f == 0) {
      f = 1;  // forced; not a candidate for the shortfall
    } else {
      cands.push_back({scaled % n, s});
    }
    freq[s] = f;
    sum += f;
  }
  int64_t d = int64_t(kTableSize) - sum;
  if (d > 0) {
    std::stable_sort(cands.begin(), cands.end(),
                     [](const Cand& a, const Cand& b) { return a.rem > b.rem; });
    for (int64_t k = 0; k < d && k < int64_t(cands.size()); k++) freq[cands[k].sym] += 1;
  }
  while (d < 0) {
    uint32_t best = 0;
    for (uint32_t s = 1; s < alpha; s++)
      if (freq[s] > freq[best]) best = s;
    freq[best] -= 1;
    d++;
  }
}

// ---------------------------------------------------------------------------
// rANS chunk encoder.  Lanes are encoded back to front (steps T-1..0, lanes
// A-1..0) from the state 2^16; words are pushed on a stack whose top is the
// start of the chunk's stream.  Division by the frequency uses a 64-bit
// reciprocal: for 2 <= f <= 4096 and x < 2^32, floor(x * ceil(2^64/f) / 2^64)
// equals floor(x / f) because the rounding error x * (ceil - 2^64/f) / 2^64
// is below 2^-32 <= 1/f (division by invariant integers, Granlund &
// Montgomery 1994).

struct EncSym {
  uint64_t recip;  // ceil(2^64 / f); 0 marks f == 1
  uint32_t f, cum;
  uint64_t x_max;  // f << 20: states at or above it emit a word first
};

struct Record {
  std::vector<uint8_t> bytes;
  uint32_t n_words = 0, n_states = 0;
};

void encode_chunk(const uint8_t* sym, uint64_t n, const EncSym* tab, uint32_t L, uint32_t W,
                  Carry cy, Record& rec, std::vector<uint16_t>& stack) {
  uint32_t A = uint32_t(std::min<uint64_t>(L, (n + W - 1) / W));
  uint32_t x[kMaxLanes];
  for (uint32_t l = 0; l < A; l++) {
    // the lane's first K symbols (row 0, steps 0..K-1) ride in its start state
    uint32_t D = 0;
    for (uint32_t k = 0; k < cy.K; k++)
      if (uint64_t(l) * W + k < n) D |= uint32_t(sym[uint64_t(l) * W + k]) << (cy.b * k);
    x[l] = cy.K ? (1u << cy.S) + D : kStateLow;
  }
  stack.resize(n + 1);
  uint16_t* top = stack.data() + stack.size();  // grows downwards
  const uint64_t LW = uint64_t(L) * W;
  const uint64_t rows = (n + LW - 1) / LW;
  for (uint64_t r = rows; r-- > 0;) {
    for (uint32_t k = W; k-- > (r == 0 ? cy.K : 0u);) {
      for (uint32_t l = A; l-- > 0;) {
        uint64_t i = r * LW + uint64_t(l) * W + k;
        if (i >= n) continue;
        const EncSym& e = tab[sym[i]];
        uint32_t v = x[l];
        if (uint64_t(v) >= e.x_max) {
          *--top = uint16_t(v);
          v >>= 16;
        }
        uint32_t q = e.recip ? uint32_t((unsigned __int128)v * e.recip >> 64) : v;
        x[l] = (q << kProbBits) + (v - q * e.f) + e.cum;
      }
    }
  }
  uint32_t nw = uint32_t(stack.data() + stack.size() - top);
  uint64_t sz = 16 + pad16(4ull * A) + pad16(2ull * nw);
  rec.bytes.assign(sz, 0);
  uint8_t* p = rec.bytes.data();
  st32(p + 0, nw);
  st32(p + 4, A);
  st32(p + 8, uint32_t(n));
  for (uint32_t l = 0; l < A; l++) st32(p + 16 + 4 * l, x[l]);
  memcpy(p + 16 + pad16(4ull * A), top, 2ull * nw);
  rec.n_words = nw;
  rec.n_states = A;
}

wc_blob* make_handle(BlobPriv&& bp) {
  BlobHandle* h = new (std::nothrow) BlobHandle();
  if (!h) return nullptr;
  h->priv = std::move(bp);
  BlobPriv& P = h->priv;
  wc_blob& b = h->pub;
  memset(&b, 0, sizeof(b));
  b.data = P.bytes.data();
  b.size = P.bytes.size();
  b.n_tensors = uint32_t(P.tensors.size());
  b.n_chunks = P.n_chunks;
  b.out_bytes = P.out_bytes.data();
  b.priv = h;
  // size breakdown
  const uint8_t* base = P.bytes.data();
  b.meta_bytes = P.raw_off;  // header, descriptors, tables and index
  for (uint64_t c = 0; c < P.n_chunks; c++) {
    uint64_t o0 = 16ull * ld32(base + P.index_off + 4 * c);
    uint64_t o1 = 16ull * ld32(base + P.index_off + 4 * (c + 1));
    uint32_t nw = ld32(base + o0), A = ld32(base + o0 + 4);
    b.record_hdr_bytes += 16;
    b.state_bytes += 4ull * A;
    b.word_bytes += 2ull * nw;
    b.pad_bytes += (o1 - o0) - 16 - 4ull * A - 2ull * nw;
  }
  b.raw_bytes = P.records_off - P.raw_off;
  return &b;
}

}  // namespace

// ---------------------------------------------------------------------------
// Statistics from histograms (Sec. II-B).

void finish_stats(uint32_t dt, uint64_t n, const uint64_t* joint16, wc_stats* out) {
  out->n_fields = has_raw(dt) ? 2 : 1;
  out->alphabet[0] = alphabet_of(dt);
  out->alphabet[1] = has_raw(dt) ? 256 : 0;
  out->count[0] = n;
  out->count[1] = has_raw(dt) ? n : 0;
  double bound = 0.0;
  for (uint32_t f = 0; f < out->n_fields; f++) {
    out->H[f] = entropy_bits(out->hist[f], out->alphabet[f]);
    bound += double(n) * out->H[f] / 8.0;
  }
  out->bound_bytes = bound;
  out->bound_bytes_raw8 = double(n) * out->H[0] / 8.0 + (has_raw(dt) ? double(n) : 0.0);
  out->H_joint16 = joint16 ? entropy_bits(joint16, 65536) : NAN;
}

void split_word_counts(const uint64_t* joint16, wc_stats* out) {
  for (uint32_t w = 0; w < 65536; w++) {
    if (!joint16[w]) continue;
    out->hist[0][(w >> 7) & 0xFF] += joint16[w];
    out->hist[1][((w >> 8) & 0x80) | (w & 0x7F)] += joint16[w];
  }
}

// ---------------------------------------------------------------------------
// Blob layout (everything the data does not decide).

wc_status plan_blob(const wc_tensor* ts, uint32_t n, const wc_params* prm, Plan& out) {
  if (!ts || !prm || n == 0 || n > 65536) return WC_EINVAL;
  const uint32_t CB = prm->chunk_bytes, L = prm->lanes;
  const uint32_t TR = prm->tile_rows, TC = prm->tile_cols, TO = prm->tile_order;
  if (CB < 256 || CB > (1u << 20) || CB % 256 || L < 1 || L > kMaxLanes ||
      prm->prob_bits != kProbBits)
    return WC_EINVAL;
  if ((TR == 0) != (TC == 0) || (TC && !pow2(TC)) || prm->codebook > WC_CODEBOOK_LAYER ||
      TO > WC_TILE_COLUMN_BLOCKS)
    return WC_EINVAL;
  for (uint32_t t = 0; t < n; t++) {
    uint32_t dt = uint32_t(ts[t].dtype);
    if (!dtype_ok(dt)) return WC_EINVAL;
    if (has_raw(dt) && ts[t].nbytes % 2) return WC_EINVAL;
    if ((ts[t].rows || ts[t].cols) && ts[t].rows * ts[t].cols != symbols_of(dt, ts[t].nbytes))
      return WC_EINVAL;
  }
  const bool shared = prm->codebook == WC_CODEBOOK_LAYER;
  out = Plan();
  out.tensors.resize(n);
  out.owner.resize(n);
  uint64_t nc_total = 0;
  for (uint32_t t = 0; t < n; t++) {
    TensorInfo& T = out.tensors[t];
    T.dtype = uint32_t(ts[t].dtype);
    T.rows = ts[t].rows;
    T.cols = ts[t].cols;
    if (tile_ok(T.dtype, T.rows, T.cols, TR, TC, TO)) {
      T.tile_r = TR;
      T.tile_c = TC;
      T.tile_order = TO;
    }
    T.chunk_bytes = T.tile_r ? uint32_t(tile_bytes(T.dtype, TR, TC)) : CB;
    T.lanes = L;
    T.group = group_of(T.dtype);
    T.alphabet = alphabet_of(T.dtype);
    T.out_bytes = ts[t].nbytes;
    T.n_sym = symbols_of(T.dtype, T.out_bytes);
    const uint64_t per = T.sym_per_chunk();
    T.n_chunks = (T.n_sym + per - 1) / per;
    T.first_chunk = nc_total;
    nc_total += T.n_chunks;
    // a full chunk's record, times the full chunks, plus the last one's
    if (T.n_chunks)
      out.worst_record_bytes += (T.n_chunks - 1) * worst_record(T, per) +
                                worst_record(T, chunk_symbols(T, T.n_chunks - 1));
  }
  if (nc_total >= 0xFFFFFFFFull) return WC_EINVAL;
  // tables: one per tensor, or the first tensor of each dtype owns its
  // dtype's table (layer codebook)
  uint64_t pos = kHeaderBytes + uint64_t(kDescBytes) * n;
  for (uint32_t t = 0; t < n; t++) {
    out.owner[t] = t;
    if (shared)
      for (uint32_t u = 0; u < t; u++)
        if (out.tensors[u].dtype == out.tensors[t].dtype) {
          out.owner[t] = u;
          break;
        }
    TensorInfo& T = out.tensors[t];
    if (out.owner[t] != t) {
      T.freq_off = out.tensors[out.owner[t]].freq_off;
      continue;
    }
    T.freq_off = pos;
    pos += pad16(2ull * T.alphabet);
  }
  out.n_chunks = nc_total;
  out.index_off = pad16(pos);
  // the raw regions follow the index; their places depend on the sizes only
  out.raw_start = pad16(out.index_off + 4 * (nc_total + 1));
  for (uint32_t t = 0; t < n; t++) {
    TensorInfo& T = out.tensors[t];
    if (!has_raw(T.dtype)) continue;
    T.raw_off = out.raw_region_bytes;
    out.raw_region_bytes += pad16(T.n_sym);
  }
  out.records_off = out.raw_start + out.raw_region_bytes;
  return WC_OK;
}

// ---------------------------------------------------------------------------
// Blob validation.

wc_status parse_blob(const uint8_t* p, uint64_t size, BlobPriv& out) {
  if (!p || size < kHeaderBytes) return WC_EINVAL;
  if (ld32(p) != kMagic || ld16(p + 4) != kVersion || ld16(p + 6) != kHeaderBytes ||
      ld32(p + 12) != kDescBytes || ld64(p + 24) != size)
    return WC_EINVAL;
  uint32_t nt = ld32(p + 8);
  uint64_t nc = ld64(p + 16);
  uint64_t idx = ld64(p + 32), rec = ld64(p + 40), raw = ld64(p + 48);
  if (nt == 0 || kHeaderBytes + uint64_t(kDescBytes) * nt > size) return WC_EINVAL;
  if (idx % 16 || rec % 16 || raw % 16) return WC_EINVAL;
  if (idx > size || nc >= (size - idx) / 4) return WC_EINVAL;
  if (raw < idx + 4 * (nc + 1) || raw > rec || rec > size) return WC_EINVAL;
  out.tensors.assign(nt, TensorInfo());
  out.out_bytes.assign(nt, 0);
  uint64_t first = 0, raw_pos = raw;
  for (uint32_t t = 0; t < nt; t++) {
    const uint8_t* d = p + kHeaderBytes + uint64_t(kDescBytes) * t;
    TensorInfo& T = out.tensors[t];
    T.dtype = ld32(d);
    T.chunk_bytes = ld32(d + 4);
    T.n_sym = ld64(d + 8);
    T.out_bytes = ld64(d + 16);
    T.first_chunk = ld64(d + 24);
    T.n_chunks = ld64(d + 32);
    T.lanes = ld16(d + 40);
    T.group = d[42];
    uint32_t pb = d[43];
    T.alphabet = ld16(d + 44);
    T.freq_off = ld64(d + 48);
    T.raw_off = ld64(d + 56);
    T.rows = ld64(d + 64);
    T.cols = ld64(d + 72);
    T.tile_r = ld32(d + 80);
    T.tile_c = ld32(d + 84);
    T.tile_order = ld32(d + 88);
    if (!dtype_ok(T.dtype) || ld32(d + 92)) return WC_EINVAL;
    if (pb != kProbBits || T.group != group_of(T.dtype) || T.alphabet != alphabet_of(T.dtype))
      return WC_EINVAL;
    if (T.lanes < 1 || T.lanes > kMaxLanes) return WC_EINVAL;
    if (T.chunk_bytes < 256 || T.chunk_bytes > (1u << 20) || T.chunk_bytes % 256)
      return WC_EINVAL;
    if (has_raw(T.dtype) && T.out_bytes % 2) return WC_EINVAL;
    if (T.n_sym != symbols_of(T.dtype, T.out_bytes)) return WC_EINVAL;
    if ((T.rows || T.cols) && T.rows * T.cols != T.n_sym) return WC_EINVAL;
    if (!(T.tile_r || T.tile_c) && T.tile_order) return WC_EINVAL;
    if ((T.tile_r || T.tile_c) &&
        (!tile_ok(T.dtype, T.rows, T.cols, T.tile_r, T.tile_c, T.tile_order) ||
         T.chunk_bytes != tile_bytes(T.dtype, T.tile_r, T.tile_c)))
      return WC_EINVAL;
    uint64_t per = T.sym_per_chunk();
    if (T.n_chunks != (T.n_sym + per - 1) / per || T.first_chunk != first) return WC_EINVAL;
    if (T.freq_off < kHeaderBytes + uint64_t(kDescBytes) * nt ||
        T.freq_off + 2ull * T.alphabet > idx)
      return WC_EINVAL;
    if (T.n_sym) {
      uint32_t sum = 0;
      for (uint32_t s = 0; s < T.alphabet; s++) sum += ld16(p + T.freq_off + 2 * s);
      if (sum != kTableSize) return WC_EINVAL;
    }
    if (has_raw(T.dtype)) {
      if (T.raw_off != raw_pos || T.raw_off + T.n_sym > rec) return WC_EINVAL;
      raw_pos += pad16(T.n_sym);
    }
    first += T.n_chunks;
    out.out_bytes[t] = T.out_bytes;
  }
  if (first != nc || raw_pos != rec) return WC_EINVAL;
  // index and chunk records
  uint64_t prev = rec;
  for (uint32_t t = 0; t < nt; t++) {
    const TensorInfo& T = out.tensors[t];
    uint64_t per = T.sym_per_chunk();
    for (uint64_t c = 0; c < T.n_chunks; c++) {
      uint64_t g = T.first_chunk + c;
      uint64_t o0 = 16ull * ld32(p + idx + 4 * g), o1 = 16ull * ld32(p + idx + 4 * (g + 1));
      if (o0 != prev || o1 < o0 + 16 || o1 > size) return WC_EINVAL;
      uint64_t n_c = std::min(per, T.n_sym - c * per);
      uint32_t nw = ld32(p + o0), A = ld32(p + o0 + 4), ns = ld32(p + o0 + 8);
      uint32_t wantA = uint32_t(std::min<uint64_t>(T.lanes, (n_c + T.group - 1) / T.group));
      if (ns != n_c || A != wantA || 16 + pad16(4ull * A) + pad16(2ull * nw) != o1 - o0)
        return WC_EINVAL;
      prev = o1;
    }
  }
  if (prev != size || 16ull * ld32(p + idx + 4 * nc) != size) return WC_EINVAL;
  out.n_chunks = nc;
  out.index_off = idx;
  out.records_off = rec;
  out.raw_off = raw;
  out.size = size;
  return WC_OK;
}

}  // namespace wc

using namespace wc;

extern "C" {

int32_t wc_version(void) { return 12; }

wc_status wc_analyze(const wc_tensor* t, wc_stats* out) {
  if (!t || !out || (!t->host_ptr && t->nbytes)) return WC_EINVAL;
  uint32_t dt = uint32_t(t->dtype);
  if (!dtype_ok(dt)) return WC_EINVAL;
  if (has_raw(dt) && t->nbytes % 2) return WC_EINVAL;
  try {
    memset(out, 0, sizeof(*out));
    const uint8_t* src = static_cast<const uint8_t*>(t->host_ptr);
    uint64_t n = symbols_of(dt, t->nbytes);
    std::vector<uint64_t> h16;
    if (has_raw(dt)) h16.assign(65536, 0);
    const uint64_t B = 1u << 16;
    uint8_t cbuf[1u << 16], rbuf[1u << 16];
    for (uint64_t s0 = 0; s0 < n; s0 += B) {
      uint64_t s1 = std::min(n, s0 + B);
      split_range(dt, src, s0, s1, cbuf, rbuf);
      for (uint64_t i = 0; i < s1 - s0; i++) out->hist[0][cbuf[i]]++;
      if (has_raw(dt)) {
        for (uint64_t i = 0; i < s1 - s0; i++) out->hist[1][rbuf[i]]++;
        for (uint64_t i = s0; i < s1; i++) h16[src[2 * i] | (uint32_t(src[2 * i + 1]) << 8)]++;
      }
    }
    finish_stats(dt, n, has_raw(dt) ? h16.data() : nullptr, out);
    return WC_OK;
  } catch (const std::bad_alloc&) {
    return WC_ENOMEM;
  } catch (...) {
    return WC_EINVAL;
  }
}

wc_status wc_encode(const wc_tensor* ts, uint32_t n, const wc_params* prm, wc_blob** out) {
  if (!ts || !prm || !out) return WC_EINVAL;
  *out = nullptr;
  for (uint32_t t = 0; t < n; t++)
    if (!ts[t].host_ptr && ts[t].nbytes) return WC_EINVAL;
  const uint32_t L = prm->lanes;
  const unsigned threads = thread_count(prm->n_threads);
  try {
    Plan plan;
    wc_status prc = plan_blob(ts, n, prm, plan);
    if (prc != WC_OK) return prc;
    BlobPriv P;
    P.tensors = plan.tensors;
    const std::vector<uint32_t>& owner = plan.owner;
    const uint64_t nc_total = plan.n_chunks;
    std::vector<std::vector<uint32_t>> freqs(n);
    std::vector<std::vector<uint8_t>> raws(n);
    std::vector<Record> recs(nc_total);

    // symbols in coding order (tile-major for tiled tensors) and histograms
    std::vector<std::vector<uint8_t>> codeds(n);
    std::vector<std::array<uint64_t, 256>> hists(n);
    for (uint32_t t = 0; t < n; t++) {
      TensorInfo& T = P.tensors[t];
      const uint8_t* src = static_cast<const uint8_t*>(ts[t].host_ptr);
      std::vector<uint8_t>& coded = codeds[t];
      coded.resize(T.n_sym);
      if (has_raw(T.dtype)) raws[t].resize(T.n_sym);
      split_tensor(T.dtype, src, T.n_sym, coded.data(),
                   has_raw(T.dtype) ? raws[t].data() : nullptr, threads);
      if (T.tile_r) {
        // tile (a, b) is chunk a * (cols / tile_c) + b; its rows follow each other
        const uint64_t ntc = T.cols / T.tile_c, per = uint64_t(T.tile_r) * T.tile_c;
        std::vector<uint8_t> c2(T.n_sym), r2(has_raw(T.dtype) ? T.n_sym : 0);
        const uint32_t W = T.group;
        parallel_for(T.n_chunks, threads, [&](uint64_t tile) {
          const uint64_t a = tile / ntc, bcol = tile % ntc;
          // a run is tile_c elements of one tile row (row-major order) or one
          // lane-group of W elements (column blocks: k-block kb, row i at
          // position kb * tile_r + i)
          const bool rows_order = T.tile_order == WC_TILE_ROWS;
          const uint64_t runs = rows_order ? T.tile_r : per / W;
          const uint32_t len = rows_order ? T.tile_c : W;
          for (uint64_t g = 0; g < runs; g++) {
            const uint64_t i = rows_order ? g : g % T.tile_r, kb = rows_order ? 0 : g / T.tile_r;
            const uint64_t e = (a * T.tile_r + i) * T.cols + bcol * T.tile_c + kb * W;
            const uint64_t k = tile * per + g * len;
            memcpy(c2.data() + k, coded.data() + e, len);
            if (!r2.empty()) memcpy(r2.data() + k, raws[t].data() + e, len);
          }
        });
        coded.swap(c2);
        if (!r2.empty()) raws[t].swap(r2);
      }
      histogram(coded.data(), T.n_sym, hists[t].data(), threads);
    }

    // tables: one per tensor, or one per dtype normalised from the summed
    // histogram of every tensor of that dtype (layer codebook)
    const bool shared = prm->codebook == WC_CODEBOOK_LAYER;
    for (uint32_t t = 0; t < n; t++) {
      if (owner[t] != t) {
        freqs[t] = freqs[owner[t]];
        continue;
      }
      uint64_t sum[256];
      memcpy(sum, hists[t].data(), sizeof(sum));
      if (shared)
        for (uint32_t u = t + 1; u < n; u++)
          if (P.tensors[u].dtype == P.tensors[t].dtype)
            for (int k = 0; k < 256; k++) sum[k] += hists[u][k];
      freqs[t].assign(P.tensors[t].alphabet, 0);
      normalise(sum, P.tensors[t].alphabet, freqs[t].data());
    }

    for (uint32_t t = 0; t < n; t++) {
      TensorInfo& T = P.tensors[t];
      const std::vector<uint8_t>& coded = codeds[t];
      EncSym tab[256];
      uint32_t cum = 0;
      for (uint32_t s = 0; s < 256; s++) {
        uint32_t f = s < T.alphabet ? freqs[t][s] : 0;
        tab[s].f = f;
        tab[s].cum = cum;
        tab[s].x_max = uint64_t(f) << 20;
        // ceil(2^64 / f) == floor((2^64 - 1) / f) + 1 for every f >= 2
        tab[s].recip = f > 1 ? ~uint64_t(0) / f + 1 : 0;
        cum += f;
      }
      const uint64_t per = T.sym_per_chunk();
      parallel_for(T.n_chunks, threads, [&](uint64_t c) {
        thread_local std::vector<uint16_t> stack;
        uint64_t s0 = c * per, len = std::min(per, T.n_sym - s0);
        encode_chunk(coded.data() + s0, len, tab, L, T.group, carry_of(T.dtype, T.tile_r != 0),
                     recs[T.first_chunk + c], stack);
      });
      std::vector<uint8_t>().swap(codeds[t]);
    }

    // layout: the plan fixed everything up to the records (the raw regions
    // sit between the index and the records); the records follow in order
    const uint64_t idx = plan.index_off;
    const uint64_t raw = plan.raw_start;
    const uint64_t rec = plan.records_off;
    for (uint32_t t = 0; t < n; t++)
      if (has_raw(P.tensors[t].dtype)) P.tensors[t].raw_off += raw;
    uint64_t pos = rec;
    for (auto& r : recs) pos += r.bytes.size();
    const uint64_t total = pos;
    if (total / 16 >= 0xFFFFFFFFull) return WC_EINVAL;

    std::vector<uint8_t> B(total, 0);
    uint8_t* b = B.data();
    st32(b, kMagic);
    st16(b + 4, kVersion);
    st16(b + 6, kHeaderBytes);
    st32(b + 8, n);
    st32(b + 12, kDescBytes);
    st64(b + 16, nc_total);
    st64(b + 24, total);
    st64(b + 32, idx);
    st64(b + 40, rec);
    st64(b + 48, raw);
    for (uint32_t t = 0; t < n; t++) {
      const TensorInfo& T = P.tensors[t];
      uint8_t* d = b + kHeaderBytes + uint64_t(kDescBytes) * t;
      st32(d, T.dtype);
      st32(d + 4, T.chunk_bytes);
      st64(d + 8, T.n_sym);
      st64(d + 16, T.out_bytes);
      st64(d + 24, T.first_chunk);
      st64(d + 32, T.n_chunks);
      st16(d + 40, T.lanes);
      d[42] = uint8_t(T.group);
      d[43] = uint8_t(kProbBits);
      st16(d + 44, T.alphabet);
      st64(d + 48, T.freq_off);
      st64(d + 56, T.raw_off);
      st64(d + 64, T.rows);
      st64(d + 72, T.cols);
      st32(d + 80, T.tile_r);
      st32(d + 84, T.tile_c);
      st32(d + 88, T.tile_order);
      for (uint32_t s = 0; s < T.alphabet; s++) st16(b + T.freq_off + 2 * s, freqs[t][s]);
    }
    std::vector<uint64_t> rec_off(nc_total + 1);
    pos = rec;
    for (uint64_t c = 0; c < nc_total; c++) {
      rec_off[c] = pos;
      st32(b + idx + 4 * c, uint32_t(pos / 16));
      pos += recs[c].bytes.size();
    }
    st32(b + idx + 4 * nc_total, uint32_t(pos / 16));
    parallel_for(nc_total, threads, [&](uint64_t c) {
      memcpy(b + rec_off[c], recs[c].bytes.data(), recs[c].bytes.size());
      std::vector<uint8_t>().swap(recs[c].bytes);
    });
    for (uint32_t t = 0; t < n; t++)
      if (has_raw(P.tensors[t].dtype) && P.tensors[t].n_sym)
        memcpy(b + P.tensors[t].raw_off, raws[t].data(), P.tensors[t].n_sym);

    BlobPriv Q;
    Q.bytes = std::move(B);
    wc_status rc = parse_blob(Q.bytes.data(), Q.bytes.size(), Q);
    if (rc != WC_OK) return rc;
    wc_blob* h = make_handle(std::move(Q));
    if (!h) return WC_ENOMEM;
    *out = h;
    return WC_OK;
  } catch (const std::bad_alloc&) {
    return WC_ENOMEM;
  } catch (...) {
    return WC_EINVAL;
  }
}

wc_status wc_open(const void* data, uint64_t size, wc_blob** out) {
  if (!data || !out) return WC_EINVAL;
  *out = nullptr;
  try {
    BlobPriv Q;
    Q.bytes.assign(static_cast<const uint8_t*>(data), static_cast<const uint8_t*>(data) + size);
    wc_status rc = parse_blob(Q.bytes.data(), Q.bytes.size(), Q);
    if (rc != WC_OK) return rc;
    wc_blob* h = make_handle(std::move(Q));
    if (!h) return WC_ENOMEM;
    *out = h;
    return WC_OK;
  } catch (const std::bad_alloc&) {
    return WC_ENOMEM;
  } catch (...) {
    return WC_EINVAL;
  }
}

void wc_free(wc_blob* b) {
  if (!b) return;
  delete static_cast<BlobHandle*>(b->priv);
}

}  // extern "C"
