// wc_encode.hip -- device half of libwc's encoder and analysis for CDNA4 (gfx950).
//
// Paper: Sec. II-B (per-tensor histograms and empirical entropy over symbols
// the numeric format defines), Sec. V-B (offline compression: a static table
// per tensor or layer, every tile an independently decodable ANS substream
// from its own initial state, an offset index), Sec. VI-F (b = 12).
//
// wc_encode_device writes, on the GPU, the same blob bytes as the host
// encoder.  Its launches, in stream order:
//   1. zero the histograms;
//   2. histograms of the coded symbols (workgroup-private LDS histograms,
//      replicated so that lanes with the same symbol hit different banks,
//      flushed with 64-bit atomics), into the table each tensor uses;
//   3. normalisation to 2^12 (one workgroup per table, integer largest
//      remainder exactly as the host does it), the u16 tables written into the
//      blob, and per symbol {2^12 - f, cum, ceil(2^64 / f)} for the encoder;
//   4. the chunk encoder: one wave per chunk, one rANS lane per wave lane,
//      steps in reverse.  Within a step the lanes that emit a word push it in
//      decreasing lane order (ballot; a lane's place is the number of emitting
//      lanes above it), so the word stack, written downwards from the end of
//      the chunk's worst-case workspace slot, is the chunk's stream in order.
//      The raw sign|mantissa bytes of 16-bit formats go straight to their
//      place in the blob;
//   5. the offset index: one workgroup scans the record sizes and writes the
//      index and the header;
//   6. the descriptors (copied from the host's layout plan);
//   7. packing: every chunk's record copied from its slot to its place.
// The symbols' loads follow the decoder's layout: a lane-group of W symbols
// is 16 bytes of the source, wherever the tiling puts it.
#include <hip/hip_runtime.h>

#include <string.h>

#include <algorithm>
#include <mutex>
#include <type_traits>
#include <vector>

#include "wc_internal.h"

namespace {

constexpr int kWaves = 8;  // chunks (waves) per encoder / packer workgroup
constexpr int kThreads = kWaves * 64;
constexpr int kHistThreads = 1024;           // 16 waves share one set of lane histograms
constexpr int kHistLoads = 2;                // 16-byte loads in flight per lane
constexpr uint64_t kHistSpan = 256u << 10;   // source bytes per histogram workgroup
constexpr int kMaxLaunch = 16;               // tensors per launch
constexpr int kScanThreads = 1024;
constexpr int kScanPer = 32;  // record sizes per scan thread and round
constexpr uint32_t kFarOffset = 0x7FFFFF00u;  // past any slot: buffer stores are dropped

enum Kind : uint32_t { kSplit16 = 0, kByte = 1, kNibble = 2 };

struct EncTensor {
  uint64_t src;             // device pointer of the tensor's bytes
  uint64_t src_bytes;
  uint64_t n_sym;
  uint64_t slot_off;        // workspace offset of chunk 0's slot
  uint64_t raw_rel;         // raw region, relative to the first raw region
  uint64_t pitch;           // tiled: bytes of one matrix row
  uint64_t tile_row_bytes;  // tiled: bytes of one tile row
  uint32_t slot_bytes;      // bytes of one chunk's slot
  uint32_t first_chunk, n_chunks, per, chunk_bytes;
  uint32_t kind, logW, lanes;
  uint32_t table;           // table index in the workspace
  uint32_t wg0;             // first workgroup of the tensor in this launch
  uint32_t tiled, tile_r, log_tc, ntc, order, log_tr;
};

struct EncArgs {
  uint64_t blob, ws;
  uint64_t hist_off, tab_off, rsz_off;
  uint64_t index_off;  // blob offset of the chunk index
  uint64_t raw_start;  // blob offset of the raw regions (after the index)
  uint32_t n_tensors, pad;
  EncTensor t[kMaxLaunch];
};

__device__ __forceinline__ uint64_t dpad16(uint64_t x) { return (x + 15) & ~uint64_t(15); }

typedef uint32_t v4u __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(1))) const v4u gu4;     // global memory: no flat access
typedef __attribute__((address_space(1))) const uint8_t gu8;

// 16 source bytes at `off`, zeros past `bytes`.
__device__ __forceinline__ uint4 load16(const uint8_t* base, uint64_t bytes, uint64_t off) {
  if (off + 16 <= bytes) {
    const v4u v = *(gu4*)(uint64_t)(base + off);
    return make_uint4(v.x, v.y, v.z, v.w);
  }
  uint32_t d[4] = {0u, 0u, 0u, 0u};
  for (uint32_t b = 0; b < 16; b++)
    if (off + b < bytes) d[b >> 2] |= uint32_t(((gu8*)(uint64_t)base)[off + b]) << (8 * (b & 3));
  return make_uint4(d[0], d[1], d[2], d[3]);
}

__device__ __forceinline__ uint32_t dword(const uint4& v, uint32_t j) {
  return j == 0 ? v.x : (j == 1 ? v.y : (j == 2 ? v.z : v.w));
}

// m's lane bit ? a : b, as one v_cndmask.  Written out because the compiler
// turns the equivalent conditional expression around a store into a branch,
// whose skipped path leaves the number of stores in flight unknown to it.
__device__ __forceinline__ uint32_t lane_select(uint64_t m, uint32_t a, uint32_t b) {
  uint32_t r;
  asm("v_cndmask_b32_e64 %0, %1, %2, %3" : "=v"(r) : "v"(b), "v"(a), "s"(m));
  return r;
}

// Coded symbol k of a lane-group (k a compile-time constant after unrolling).
template <uint32_t K>
__device__ __forceinline__ uint32_t symbol(const uint4& v, uint32_t k) {
  if constexpr (K == kSplit16) return (dword(v, k >> 1) >> (16 * (k & 1) + 7)) & 0xFFu;
  else if constexpr (K == kByte) return (dword(v, k >> 2) >> (8 * (k & 3))) & 0xFFu;
  else return (dword(v, k >> 3) >> (4 * (k & 7))) & 0xFu;
}

// Byte offsets in the source of the lane-groups of one chunk: a byte run, or
// a lane-group's place in its tile (row-major or column blocks).  The chunk's
// part is worked out once; at(i0) is the lane-group that starts at symbol i0.
struct GroupAddr {
  uint64_t base, pitch;
  uint32_t mode, logW, log_tc, log_tr;
  __device__ __forceinline__ GroupAddr(const EncTensor& T, uint32_t c)
      : pitch(T.pitch), logW(T.logW), log_tc(T.log_tc), log_tr(T.log_tr) {
    if (!T.tiled) {
      mode = 0;
      base = uint64_t(c) * T.chunk_bytes;
    } else {
      mode = T.order == 0 ? 1u : 2u;
      base = uint64_t(c / T.ntc) * T.tile_r * T.pitch + uint64_t(c % T.ntc) * T.tile_row_bytes;
    }
  }
  __device__ __forceinline__ uint64_t at(uint32_t i0) const {
    if (mode == 0) return base + (uint64_t(i0 >> logW) << 4);
    if (mode == 1)
      return base + uint64_t(i0 >> log_tc) * pitch +
             (uint64_t((i0 & ((1u << log_tc) - 1u)) >> logW) << 4);
    const uint32_t g = i0 >> logW;  // row g mod tile_r of k-block g div tile_r
    return base + uint64_t(g & ((1u << log_tr) - 1u)) * pitch + (uint64_t(g >> log_tr) << 4);
  }
};

// Workgroup b runs on XCD b mod 8; renumbered so that each XCD takes one
// contiguous block of the launch's workgroups (a bijection of [0, n)).  The
// chunk encoder uses it (about 3 % faster); the histogram and pack passes
// measured no better or worse with it.
__device__ __forceinline__ uint32_t xcd_order(uint32_t b, uint32_t n) {
  const uint32_t x = b % 8u, k = b / 8u, q = n / 8u, r = n % 8u;
  return x * q + min(x, r) + k;
}

__device__ __forceinline__ uint32_t tensor_of(const EncArgs& a, uint32_t wg) {
  uint32_t ti = 0;
  for (uint32_t k = 1; k < a.n_tensors; k++)
    if (wg >= a.t[k].wg0) ti = k;
  return ti;
}

// ---------------------------------------------------------------------------
// 1. zero fill (no memset node, so a captured graph can replay it)

__global__ void zero_kernel(uint4* p, uint64_t n16) {
  for (uint64_t i = blockIdx.x * uint64_t(blockDim.x) + threadIdx.x; i < n16;
       i += uint64_t(gridDim.x) * blockDim.x)
    p[i] = make_uint4(0u, 0u, 0u, 0u);
}

// ---------------------------------------------------------------------------
// 2. coded-symbol histograms.  Workgroup w of a tensor counts source bytes
// [w * kHistSpan, +kHistSpan); symbol order does not matter here.  Every wave
// lane has its own histogram in LDS, laid out bin-major (bin * 64 + lane):
// the lanes of one atomic add never share an address, each lane stays in its
// own bank, and the waves of the workgroup share the 64 histograms.

template <uint32_t K>
__device__ void count_span(const EncTensor& T, uint64_t off0, uint64_t off1, uint32_t* h) {
  const uint8_t* src = reinterpret_cast<const uint8_t*>(T.src);
  const uint32_t lane = threadIdx.x & 63u;
  constexpr uint32_t W = K == kSplit16 ? 8u : (K == kByte ? 16u : 32u);
  constexpr uint64_t kStep = kHistThreads * 16ull;
  // whole lane-groups, kHistLoads loads in flight; then the tensor's last bytes
  const uint64_t full_end = off0 + (off1 - off0) / 16 * 16;
  uint64_t off = off0 + threadIdx.x * 16ull;
  for (; off + (kHistLoads - 1) * kStep < full_end; off += kHistLoads * kStep) {
    uint4 v[kHistLoads];
#pragma unroll
    for (int u = 0; u < kHistLoads; u++) v[u] = load16(src, full_end, off + u * kStep);
#pragma unroll
    for (int u = 0; u < kHistLoads; u++)
#pragma unroll
      for (uint32_t k = 0; k < W; k++) atomicAdd(&h[symbol<K>(v[u], k) * 64u + lane], 1u);
  }
  for (; off < off1; off += kStep) {
    const uint4 v = load16(src, T.src_bytes, off);
    // symbols whose bytes lie inside the tensor
    const uint64_t left = T.src_bytes - off;
    const uint32_t nv = left >= 16 ? W : uint32_t(left * W / 16);
#pragma unroll
    for (uint32_t k = 0; k < W; k++)
      if (k < nv) atomicAdd(&h[symbol<K>(v, k) * 64u + lane], 1u);
  }
}

__global__ __launch_bounds__(kHistThreads) void hist_kernel(EncArgs a) {
  __shared__ uint32_t h[256 * 64];
  for (uint32_t i = threadIdx.x; i < 256 * 64; i += kHistThreads) h[i] = 0;
  __syncthreads();
  const EncTensor& T = a.t[tensor_of(a, blockIdx.x)];
  const uint64_t off0 = uint64_t(blockIdx.x - T.wg0) * kHistSpan;
  const uint64_t off1 = min<uint64_t>(off0 + kHistSpan, T.src_bytes);
  if (T.kind == kSplit16) count_span<kSplit16>(T, off0, off1, h);
  else if (T.kind == kByte) count_span<kByte>(T, off0, off1, h);
  else count_span<kNibble>(T, off0, off1, h);
  __syncthreads();
  if (threadIdx.x < 256) {
    // bin threadIdx.x over the 64 lanes, starting at a different lane in
    // every thread so that the wave's reads fall in different banks
    uint32_t c = 0;
    for (uint32_t r = 0; r < 64; r++) c += h[threadIdx.x * 64u + ((r + threadIdx.x) & 63u)];
    unsigned long long* g =
        reinterpret_cast<unsigned long long*>(a.ws + a.hist_off) + uint64_t(T.table) * 256u;
    if (c) atomicAdd(g + threadIdx.x, (unsigned long long)c);
  }
}

// Whole 16-bit words of a 16-bit tensor, bins [part * 16384, +16384) counted
// in LDS (the 65 536 bins of the joint histogram take four passes).
__global__ __launch_bounds__(1024) void word_hist_kernel(uint64_t src, uint64_t bytes,
                                                         uint64_t hist, uint32_t part) {
  __shared__ uint32_t wh[16384];
  for (uint32_t i = threadIdx.x; i < 16384; i += blockDim.x) wh[i] = 0;
  __syncthreads();
  const uint8_t* p = reinterpret_cast<const uint8_t*>(src);
  const uint64_t stride = uint64_t(gridDim.x) * blockDim.x * 16;
  for (uint64_t off = (uint64_t(blockIdx.x) * blockDim.x + threadIdx.x) * 16; off < bytes;
       off += stride) {
    const uint4 v = load16(p, bytes, off);
    const uint32_t nw = bytes - off >= 16 ? 8u : uint32_t((bytes - off) / 2);
#pragma unroll
    for (uint32_t k = 0; k < 8; k++) {
      const uint32_t w = (dword(v, k >> 1) >> (16 * (k & 1))) & 0xFFFFu;
      if (k < nw && (w >> 14) == part) atomicAdd(&wh[w & 0x3FFFu], 1u);
    }
  }
  __syncthreads();
  unsigned long long* g = reinterpret_cast<unsigned long long*>(hist) + part * 16384u;
  for (uint32_t i = threadIdx.x; i < 16384; i += blockDim.x)
    if (wh[i]) atomicAdd(g + i, (unsigned long long)wh[i]);
}

// ---------------------------------------------------------------------------
// 3. normalisation to 2^12 (Sec. VI-F): f = floor(c * 4096 / n); present
// symbols at least 1 (forced); a shortfall d goes +1 each to the d largest
// remainders among the unforced (lower symbol on ties); an excess comes off
// the largest f one unit at a time (lower symbol on ties).

struct NormTable {
  uint64_t freq_off;  // blob offset of the u16 table
  uint32_t table, alphabet;
};

struct NormArgs {
  uint64_t blob, ws, hist_off, tab_off;
  uint32_t n_tables, pad;
  NormTable t[64];
};

__global__ __launch_bounds__(256) void norm_kernel(NormArgs a) {
  __shared__ unsigned long long rem[256];
  __shared__ uint32_t cand[256];
  __shared__ uint32_t red[256];
  __shared__ unsigned long long nsum;
  const NormTable& NT = a.t[blockIdx.x];
  const uint32_t s = threadIdx.x;
  const unsigned long long* hg =
      reinterpret_cast<const unsigned long long*>(a.ws + a.hist_off) + uint64_t(NT.table) * 256u;
  const unsigned long long c = s < NT.alphabet ? hg[s] : 0ull;
  if (s == 0) nsum = 0;
  __syncthreads();
  atomicAdd(&nsum, c);
  __syncthreads();
  const unsigned long long n = nsum;
  uint32_t f = 0;
  bool forced = false;
  unsigned long long r = 0;
  if (n && c) {
    const unsigned long long scaled = c * wc::kTableSize;
    f = uint32_t(scaled / n);
    r = scaled % n;
    if (f == 0) {
      f = 1;
      forced = true;
    }
  }
  rem[s] = r;
  cand[s] = (c && !forced) ? 1u : 0u;
  red[s] = f;
  __syncthreads();
  for (uint32_t w = 128; w > 0; w >>= 1) {
    if (s < w) red[s] += red[s + w];
    __syncthreads();
  }
  int d = n ? int(wc::kTableSize) - int(red[0]) : 0;
  __syncthreads();
  if (d > 0 && cand[s]) {
    // place of this candidate in (remainder descending, symbol ascending)
    uint32_t rank = 0;
    for (uint32_t t = 0; t < 256; t++)
      rank += cand[t] && (rem[t] > r || (rem[t] == r && t < s)) ? 1u : 0u;
    if (rank < uint32_t(d)) f += 1;
  }
  while (d < 0) {
    // the largest f, lowest symbol on ties: reduce (f << 8 | 255 - s)
    red[s] = (f << 8) | (255u - s);
    __syncthreads();
    for (uint32_t w = 128; w > 0; w >>= 1) {
      if (s < w) red[s] = max(red[s], red[s + w]);
      __syncthreads();
    }
    if (s == 255u - (red[0] & 0xFFu)) f -= 1;
    d++;
    __syncthreads();
  }
  // u16 table into the blob; g = 2^12 - f, cum and 1/f for the encoder
  if (s < NT.alphabet) reinterpret_cast<uint16_t*>(a.blob + NT.freq_off)[s] = uint16_t(f);
  red[s] = f;
  __syncthreads();
  uint32_t cum = 0;
  for (uint32_t t = 0; t < s; t++) cum += red[t];
  // 1/f rounded up to a double: the correctly rounded quotient, raised by one
  // unit in the last place when it is below 1/f (the sign of the exact
  // fma(r, f, -1) says which)
  double rcp = 0.0;
  if (f) {
    rcp = 1.0 / double(f);
    if (fma(rcp, double(f), -1.0) < 0.0)
      rcp = __longlong_as_double(__double_as_longlong(rcp) + 1);
  }
  const uint32_t g = f ? wc::kTableSize - f : 0u;
  const unsigned long long rb = __double_as_longlong(rcp);
  uint4* tab = reinterpret_cast<uint4*>(a.ws + a.tab_off) + uint64_t(NT.table) * 256u;
  tab[s] = make_uint4(g, cum, uint32_t(rb), uint32_t(rb >> 32));
}

// ---------------------------------------------------------------------------
// 4. chunk encoder.  Symbol i of a chunk is lane (i mod L*W) div W's symbol at
// step (i div L*W)*W + i mod W.  Steps run from the last to the first; in a
// step every active lane with x >= f * 2^20 emits its low 16 bits (x >>= 16)
// and then x = floor(x / f) * 2^12 + x mod f + cum.  The step works from
// Q = floor(x / f), computed as x * r in double precision with r = 1/f
// rounded up, truncated: the product is never below x / f (so not below Q,
// an integer), and it exceeds x / f by at most (x / f) * 2^-52 < 2^-20,
// while x / f is at least 1/f >= 2^-12 below Q + 1, so it stays below Q + 1.
//   * x >= f * 2^20 exactly when Q >= 2^20; the emitting lane then codes
//     from x >> 16, whose quotient is Q >> 16;
//   * with g = 2^12 - f and q the quotient of the value coded from, the new
//     state is that value + cum + q * g (q < 2^20, g < 2^12: a 24-bit
//     multiply-add).
// A row in which every lane codes all W
// symbols takes a step without any masks; the chunk's last row (row 0, whose
// first symbols the start states carry) and a ragged final row mask inactive
// lanes.

template <uint32_t K>
__device__ void encode_chunk(const EncArgs& a, const EncTensor& T, uint32_t c, uint32_t lane,
                             const uint4* __restrict__ tab) {
  constexpr uint32_t W = K == kSplit16 ? 8u : (K == kByte ? 16u : 32u);
  const uint8_t* src = reinterpret_cast<const uint8_t*>(T.src);
  const uint64_t src_bytes = T.src_bytes;
  const uint64_t s0 = uint64_t(c) * T.per;
  const uint32_t n_c = uint32_t(min<uint64_t>(T.per, T.n_sym - s0));
  const uint32_t L = T.lanes;
  const uint32_t A = min(L, (n_c + W - 1) / W);
  const uint32_t LW = L * W;
  const uint32_t rows = (n_c + LW - 1) / LW;
  // rows [1, full) have every lane coding all W symbols
  const uint32_t full = L == 64 ? n_c / LW : 0u;
  const GroupAddr ga(T, c);
  const uint32_t slot_bytes = T.slot_bytes;
  uint8_t* slot = reinterpret_cast<uint8_t*>(a.ws + T.slot_off) + uint64_t(c) * slot_bytes;
  // the slot as a buffer: word k from its end sits at byte slot_bytes - 2k
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(slot, (short)0, (int)slot_bytes, 0x00020000);
  // this lane's lane-group of row r (zeros past the chunk's symbols)
  auto load_row = [&](uint32_t r) {
    const uint32_t i0 = r * LW + lane * W;
    uint4 v = make_uint4(0u, 0u, 0u, 0u);
    if (lane < L && i0 < n_c) v = load16(src, src_bytes, ga.at(i0));
    return v;
  };
  // an untiled chunk's lane starts at 2^S + D, D its first ck symbols (cb
  // bits each, the first lowest), which are not coded; tiled chunks at 2^16
  const uint32_t ck = T.tiled ? 0u : (K == kSplit16 ? 2u : (K == kByte ? 3u : 7u));
  constexpr uint32_t cb = K == kNibble ? 4u : 8u;
  constexpr uint32_t cs = K == kSplit16 ? 16u : (K == kByte ? 24u : 28u);
  const uint4 zero = make_uint4(0u, 0u, 0u, 0u);
  const uint4 first = rows ? load_row(0) : zero;  // row 0, kept for the last row coded
  uint32_t x = wc::kStateLow;
  if (ck) {
    const uint32_t nv0 = lane < L && lane * W < n_c ? min(W, n_c - lane * W) : 0u;
    uint32_t D = 0;
#pragma unroll
    for (uint32_t k = 0; k < 7; k++)
      if (k < ck && k < nv0) D |= symbol<K>(first, k) << (cb * k);
    x = (1u << cs) + D;
  }
  uint32_t top = 0;  // words pushed
  // 16-bit formats: the raw byte of every word goes straight to its
  // coding-order place in the raw region, which precedes the records.  The
  // stores go through a buffer descriptor: a flat store would also hold the
  // LDS counter that every step's table read waits on.
  const __amdgpu_buffer_rsrc_t rr = __builtin_amdgcn_make_buffer_rsrc(
      reinterpret_cast<uint8_t*>(a.blob) + a.raw_start + T.raw_rel + s0, (short)0,
      K == kSplit16 ? (int)n_c : 0, 0x00020000);
  // One step: symbol k of every lane in `active` (all lanes when kAll).
  auto step = [&](auto all, const uint4& v, uint32_t k, bool active) {
    constexpr bool kAll = decltype(all)::value;
    const uint4 e = tab[symbol<K>(v, k)];  // {g, cum, 1/f rounded up (double)}
    const uint32_t Q = uint32_t(double(x) * __hiloint2double(int(e.w), int(e.z)));
    bool emit = Q >= (1u << 20);
    if constexpr (!kAll) emit = emit && active;
    const uint64_t m = __ballot(emit);
    const uint32_t below = __builtin_amdgcn_mbcnt_hi(
        uint32_t(m >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(m), 0u));
    const uint32_t total = uint32_t(__popcll(m));
    // pushed after the emitting lanes above this one (total - below - 1)
    // Every lane stores (a lane that emits nothing past the slot, where the
    // buffer range check drops it), so that each row issues a fixed number of
    // stores and the wait for the next row's load counts exactly.
    const uint32_t base = __builtin_amdgcn_readfirstlane(slot_bytes - 2u * (top + total));
    __builtin_amdgcn_raw_buffer_store_b16(uint16_t(x), rs,
                                          lane_select(m, base + 2u * below, kFarOffset), 0, 0);
    top += total;
    const uint32_t v2 = emit ? x >> 16 : x;
    const uint32_t q = emit ? Q >> 16 : Q;
    const uint32_t xn = __umul24(q, e.x) + v2 + e.y;
    if constexpr (kAll) x = xn;
    else x = active ? xn : x;
  };
  // A row in which every lane codes all W symbols (every row of a 64-lane
  // chunk but row 0 and a ragged last row).
  auto code_full = [&](uint32_t r, const uint4& cur) {
    if constexpr (K == kSplit16) {
      // raw byte of a word: bit 15 -> bit 7, bits 6..0 kept; the high and the
      // low bytes of four words gathered, then merged bit by bit
      typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
      const uint32_t h0 = __builtin_amdgcn_perm(cur.y, cur.x, 0x07050301u);
      const uint32_t l0 = __builtin_amdgcn_perm(cur.y, cur.x, 0x06040200u);
      const uint32_t h1 = __builtin_amdgcn_perm(cur.w, cur.z, 0x07050301u);
      const uint32_t l1 = __builtin_amdgcn_perm(cur.w, cur.z, 0x06040200u);
      const uint32_t m8 = 0x80808080u;
      __builtin_amdgcn_raw_buffer_store_b64(
          u32x2{(h0 & m8) | (l0 & ~m8), (h1 & m8) | (l1 & ~m8)}, rr, r * LW + lane * W, 0, 0);
    }
#pragma unroll
    for (uint32_t kk = 0; kk < W; kk++) step(std::true_type{}, cur, W - 1 - kk, true);
  };
  // Any row: lanes past the chunk's symbols, and in row 0 the symbols the
  // start states carry, are inactive.
  auto code_any = [&](uint32_t r, const uint4& cur) {
    const uint32_t i0 = r * LW + lane * W;
    const uint32_t nv = lane < L && i0 < n_c ? min(W, n_c - i0) : 0u;
    if constexpr (K == kSplit16) {
      uint32_t rb[2] = {0u, 0u};
#pragma unroll
      for (uint32_t k = 0; k < 8; k++) {
        const uint32_t w = (dword(cur, k >> 1) >> (16 * (k & 1))) & 0xFFFFu;
        rb[k >> 2] |= (((w >> 8) & 0x80u) | (w & 0x7Fu)) << (8 * (k & 3));
      }
#pragma unroll
      for (uint32_t k = 0; k < 8; k++)
        __builtin_amdgcn_raw_buffer_store_b8(uint8_t(rb[k >> 2] >> (8 * (k & 3))), rr,
                                             k < nv ? i0 + k : kFarOffset, 0, 0);
    }
#pragma unroll
    for (uint32_t kk = 0; kk < W; kk++) {
      const uint32_t k = W - 1 - kk;
      step(std::false_type{}, cur, k, k < nv && (r != 0 || k >= ck));
    }
  };
  // Rows are coded from the last to the first, in three runs: rows that are
  // not full (from the top down to row 1), the full rows, row 0.  Each row's
  // successor is loaded before the row is coded.  The empty statement after
  // that load keeps the compiler from merging it with the load before the
  // loop into one load at the top of the loop, which would wait for each
  // row's data as it is needed; the explicit vmcnt(0) before the runs
  // leaves, inside them, only the wait for the next row's load at the end of
  // each row.  Every row issues a fixed number of stores, so that wait counts
  // exactly.
  auto next_row = [&](uint32_t r) { return r > 1 ? load_row(r - 1) : (r == 1 ? first : zero); };
  // the same for a row below `full` (every lane-group inside the tensor): a
  // plain load, with no branch for the tensor's end
  auto next_full = [&](uint32_t r) {
    if (r > 1) {
      const v4u v = *(gu4*)(uint64_t)(src + ga.at((r - 1) * LW + lane * W));
      return make_uint4(v.x, v.y, v.z, v.w);
    }
    return r == 1 ? first : zero;
  };
  uint4 cur = rows > 1 ? load_row(rows - 1) : first;
  __builtin_amdgcn_s_waitcnt(0x0F70);
  uint32_t r = rows;
  const uint32_t lo = max(full, 1u);
  for (; r > lo; r--) {
    const uint4 nxt = next_row(r - 1);
    asm volatile("" ::: "memory");
    code_any(r - 1, cur);
    cur = nxt;
  }
  for (; r > 1; r--) {
    const uint4 nxt = next_full(r - 1);
    asm volatile("" ::: "memory");
    code_full(r - 1, cur);
    cur = nxt;
  }
  if (r == 1) code_any(0, cur);
  if (K == kSplit16 && c + 1 == T.n_chunks) {
    // the raw region's zero padding to 16 bytes
    uint8_t* end = reinterpret_cast<uint8_t*>(a.blob) + a.raw_start + T.raw_rel;
    if (lane < dpad16(T.n_sym) - T.n_sym) end[T.n_sym + lane] = 0;
  }
  // record header, states and their padding at the slot's start
  uint32_t* hdr = reinterpret_cast<uint32_t*>(slot);
  if (lane == 0) *reinterpret_cast<uint4*>(hdr) = make_uint4(top, A, n_c, 0u);
  const uint32_t padA = uint32_t(dpad16(4ull * A) / 4);
  if (lane < padA) hdr[4 + lane] = lane < A ? x : 0u;
  if (lane == 0) {
    const uint32_t bytes = 16u + 4u * padA + uint32_t(dpad16(2ull * top));
    reinterpret_cast<uint32_t*>(a.ws + a.rsz_off)[T.first_chunk + c] = bytes / 16u;
  }
}

__global__ __launch_bounds__(kThreads) void encode_kernel(EncArgs a) {
  __shared__ uint4 tab[256];
  const uint32_t wg = xcd_order(blockIdx.x, gridDim.x);
  const EncTensor& T = a.t[tensor_of(a, wg)];
  const uint4* tg = reinterpret_cast<const uint4*>(a.ws + a.tab_off) + uint64_t(T.table) * 256u;
  if (threadIdx.x < 256) tab[threadIdx.x] = tg[threadIdx.x];
  __syncthreads();
  const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const uint32_t c = (wg - T.wg0) * kWaves + wave;
  if (c >= T.n_chunks) return;
  const uint32_t lane = __lane_id();
  if (T.kind == kSplit16) encode_chunk<kSplit16>(a, T, c, lane, tab);
  else if (T.kind == kByte) encode_chunk<kByte>(a, T, c, lane, tab);
  else encode_chunk<kNibble>(a, T, c, lane, tab);
}

// ---------------------------------------------------------------------------
// 5. offset index: exclusive scan of the record sizes (16-byte units) from the
// records' start; then the header, with the size it implies.

struct ScanArgs {
  uint64_t blob, ws, rsz_off, size_out;
  uint64_t index_off, raw_start, records_off, n_chunks;
  uint32_t header[16];  // the header with the size still 0
};

__global__ __launch_bounds__(kScanThreads) void scan_kernel(ScanArgs a) {
  __shared__ uint32_t wsum[kScanThreads / 64];
  __shared__ uint64_t carry_s;
  const uint32_t tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const uint32_t* rsz = reinterpret_cast<const uint32_t*>(a.ws + a.rsz_off);
  uint32_t* index = reinterpret_cast<uint32_t*>(a.blob + a.index_off);
  const uint64_t rec16 = a.records_off / 16;
  const uint64_t n = a.n_chunks;
  if (tid == 0) carry_s = 0;
  __syncthreads();
  // rounds of kScanThreads * kScanPer sizes; thread tid takes kScanPer
  // consecutive ones, all loaded before any is added
  constexpr uint64_t kRound = uint64_t(kScanThreads) * kScanPer;
  for (uint64_t base = 0; base < n; base += kRound) {
    const uint64_t g0 = base + uint64_t(tid) * kScanPer;
    uint32_t v[kScanPer];
    if (g0 + kScanPer <= n) {
      const uint4* r4 = reinterpret_cast<const uint4*>(rsz + g0);  // 128-byte aligned
#pragma unroll
      for (int j = 0; j < kScanPer / 4; j++) {
        const uint4 q = r4[j];
        v[4 * j] = q.x, v[4 * j + 1] = q.y, v[4 * j + 2] = q.z, v[4 * j + 3] = q.w;
      }
    } else {
#pragma unroll
      for (int j = 0; j < kScanPer; j++) v[j] = g0 + j < n ? rsz[g0 + j] : 0u;
    }
    uint32_t sum = 0;
#pragma unroll
    for (int j = 0; j < kScanPer; j++) sum += v[j];
    uint32_t incl = sum;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const uint32_t u = __shfl_up(incl, d, 64);
      if ((int)lane >= d) incl += u;
    }
    if (lane == 63) wsum[wave] = incl;
    __syncthreads();
    uint32_t before = 0;
    for (uint32_t w = 0; w < wave; w++) before += wsum[w];
    const uint64_t carry = carry_s;
    uint64_t run = rec16 + carry + before + incl - sum;
#pragma unroll
    for (int j = 0; j < kScanPer; j++) {
      if (g0 + j < n) index[g0 + j] = uint32_t(run);
      run += v[j];
    }
    __syncthreads();
    if (tid == kScanThreads - 1) carry_s = carry + before + incl;
    __syncthreads();
  }
  const uint64_t size = a.records_off + 16 * carry_s;
  if (tid == 0) {
    index[a.n_chunks] = uint32_t(size / 16);
    *reinterpret_cast<uint64_t*>(a.size_out) = size;
  }
  // zeros between the index and the raw regions
  uint8_t* b = reinterpret_cast<uint8_t*>(a.blob);
  for (uint64_t o = a.index_off + 4 * (a.n_chunks + 1) + tid; o < a.raw_start; o += kScanThreads)
    b[o] = 0;
  if (tid < 16) {
    uint32_t h = a.header[tid];
    if (tid == 6) h = uint32_t(size);  // bytes 24..31: size
    if (tid == 7) h = uint32_t(size >> 32);
    reinterpret_cast<uint32_t*>(a.blob)[tid] = h;
  }
}

// ---------------------------------------------------------------------------
// 6. descriptors: 96 bytes per tensor, as the host wrote them.

struct DescArgs {
  uint64_t blob;
  uint32_t first, n;
  uint32_t d[kMaxLaunch * 2][24];
};

__global__ void desc_kernel(DescArgs a) {
  const uint32_t t = threadIdx.x / 24, j = threadIdx.x % 24;
  if (t >= a.n) return;
  reinterpret_cast<uint32_t*>(a.blob + wc::kHeaderBytes + uint64_t(wc::kDescBytes) * (a.first + t))[j] =
      a.d[t][j];
}

// ---------------------------------------------------------------------------
// 7. packing: one wave per chunk moves its record from the slot to the offset
// the index gives (words re-based from the stack's end, zero padding).

template <uint32_t K>
__device__ void pack_chunk(const EncArgs& a, const EncTensor& T, uint32_t c, uint32_t lane) {
  const uint32_t g = T.first_chunk + c;
  uint8_t* blob = reinterpret_cast<uint8_t*>(a.blob);
  const uint64_t o = 16ull * reinterpret_cast<const uint32_t*>(a.blob + a.index_off)[g];
  const uint8_t* slot = reinterpret_cast<const uint8_t*>(a.ws + T.slot_off) + uint64_t(c) * T.slot_bytes;
  const uint4 hdr = *reinterpret_cast<const uint4*>(slot);
  const uint32_t nw = hdr.x, A = hdr.y;
  const uint32_t head = 16u + uint32_t(dpad16(4ull * A));
  // header and states (16-byte units)
  for (uint32_t j = lane; j < head / 16; j += 64)
    *reinterpret_cast<uint4*>(blob + o + 16ull * j) = reinterpret_cast<const uint4*>(slot)[j];
  // words: the stack's last nw u16 of the slot, then zeros to 16 bytes.  They
  // start 2 bytes into a dword when nw is odd: five dword loads through the
  // slot's buffer descriptor, realigned by 16 bits; the bytes past the slot's
  // end (the padding) read as zero.
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(slot), (short)0, (int)T.slot_bytes, 0x00020000);
  const uint32_t start = T.slot_bytes - 2u * nw;
  const uint32_t a0 = start & ~3u, sh = (start & 2u) * 8u;
  const uint32_t units = uint32_t(dpad16(2ull * nw) / 16);
  for (uint32_t j = lane; j < units; j += 64) {
    uint32_t d[5];
#pragma unroll
    for (uint32_t q = 0; q < 5; q++)
      d[q] = __builtin_amdgcn_raw_buffer_load_b32(rs, a0 + 16u * j + 4u * q, 0, 0);
    uint32_t w[4];
#pragma unroll
    for (uint32_t q = 0; q < 4; q++) w[q] = sh ? __builtin_amdgcn_alignbit(d[q + 1], d[q], 16) : d[q];
    *reinterpret_cast<uint4*>(blob + o + head + 16ull * j) = make_uint4(w[0], w[1], w[2], w[3]);
  }
}

__global__ __launch_bounds__(kThreads) void pack_kernel(EncArgs a) {
  const EncTensor& T = a.t[tensor_of(a, blockIdx.x)];
  const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const uint32_t c = (blockIdx.x - T.wg0) * kWaves + wave;
  if (c >= T.n_chunks) return;
  const uint32_t lane = __lane_id();
  if (T.kind == kSplit16) pack_chunk<kSplit16>(a, T, c, lane);
  else if (T.kind == kByte) pack_chunk<kByte>(a, T, c, lane);
  else pack_chunk<kNibble>(a, T, c, lane);
}

}  // namespace

// ---------------------------------------------------------------------------
// Host side.

namespace {

using wc::Plan;
using wc::TensorInfo;

struct WsLayout {
  uint64_t hist_off, tab_off, rsz_off, slots_off, total;
  std::vector<uint64_t> slot_off;     // per tensor
  std::vector<uint32_t> table_of;     // per tensor: its table's index
  uint32_t n_tables;
};

inline uint64_t up256(uint64_t x) { return (x + 255) & ~uint64_t(255); }

uint32_t slot_bytes_of(const TensorInfo& T) { return uint32_t(wc::worst_record(T, T.sym_per_chunk())); }

void layout_ws(const Plan& P, WsLayout& L) {
  const uint32_t n = uint32_t(P.tensors.size());
  L.table_of.assign(n, 0);
  L.n_tables = 0;
  for (uint32_t t = 0; t < n; t++)
    L.table_of[t] = P.owner[t] == t ? L.n_tables++ : L.table_of[P.owner[t]];
  uint64_t pos = 0;
  L.hist_off = pos;
  pos = up256(pos + 8ull * 256 * L.n_tables);
  L.tab_off = pos;
  pos = up256(pos + 16ull * 256 * L.n_tables);
  L.rsz_off = pos;
  pos = up256(pos + 4 * (P.n_chunks + 1));
  L.slots_off = pos;
  L.slot_off.assign(n, 0);
  for (uint32_t t = 0; t < n; t++) {
    L.slot_off[t] = pos;
    pos = up256(pos + P.tensors[t].n_chunks * uint64_t(slot_bytes_of(P.tensors[t])));
  }
  L.total = pos;
}

uint32_t kind_of(uint32_t dt) {
  return wc::is_nibble(dt) ? kNibble : (wc::is_byte(dt) ? kByte : kSplit16);
}

void fill_enc(EncTensor& E, const TensorInfo& T, const wc_dtensor& D, const WsLayout& L,
              uint32_t t) {
  E = EncTensor{};
  E.src = reinterpret_cast<uint64_t>(D.dev_ptr);
  E.src_bytes = T.out_bytes;
  E.n_sym = T.n_sym;
  E.slot_off = L.slot_off[t];
  E.raw_rel = T.raw_off;  // relative in the plan
  E.slot_bytes = slot_bytes_of(T);
  E.first_chunk = uint32_t(T.first_chunk);
  E.n_chunks = uint32_t(T.n_chunks);
  E.per = uint32_t(T.sym_per_chunk());
  E.chunk_bytes = T.chunk_bytes;
  E.kind = kind_of(T.dtype);
  E.logW = uint32_t(__builtin_ctz(T.group));
  E.lanes = T.lanes;
  E.table = L.table_of[t];
  E.tiled = T.tile_r ? 1u : 0u;
  if (E.tiled) {
    E.tile_r = T.tile_r;
    E.log_tc = uint32_t(__builtin_ctz(T.tile_c));
    E.ntc = uint32_t(T.cols / T.tile_c);
    E.pitch = T.cols * 16 / T.group;
    E.tile_row_bytes = uint64_t(T.tile_c) * 16 / T.group;
    E.order = T.tile_order;
    E.log_tr = T.tile_order == WC_TILE_COLUMN_BLOCKS ? uint32_t(__builtin_ctz(T.tile_r)) : 0u;
  }
}

void put32(uint32_t* d, uint32_t byte, uint32_t v) { d[byte / 4] = v; }
void put64(uint32_t* d, uint32_t byte, uint64_t v) {
  d[byte / 4] = uint32_t(v);
  d[byte / 4 + 1] = uint32_t(v >> 32);
}

// The 96-byte descriptor of T as dwords (raw_off relative to raw_start).
void descriptor(const TensorInfo& T, uint64_t raw_start, uint32_t* d) {
  memset(d, 0, 96);
  put32(d, 0, T.dtype);
  put32(d, 4, T.chunk_bytes);
  put64(d, 8, T.n_sym);
  put64(d, 16, T.out_bytes);
  put64(d, 24, T.first_chunk);
  put64(d, 32, T.n_chunks);
  d[10] = T.lanes | (T.group << 16) | (wc::kProbBits << 24);
  d[11] = T.alphabet;
  put64(d, 48, T.freq_off);
  put64(d, 56, wc::has_raw(T.dtype) ? raw_start + T.raw_off : 0);
  put64(d, 64, T.rows);
  put64(d, 72, T.cols);
  put32(d, 80, T.tile_r);
  put32(d, 84, T.tile_c);
  put32(d, 88, T.tile_order);
}

wc_status plan_device(const wc_dtensor* t, uint32_t n, const wc_params* p, Plan& P,
                      std::vector<wc_tensor>& hs) {
  if (!t || !p || n == 0 || n > 65536) return WC_EINVAL;
  hs.resize(n);
  for (uint32_t i = 0; i < n; i++)
    hs[i] = wc_tensor{t[i].dev_ptr, t[i].nbytes, t[i].dtype, 0, t[i].rows, t[i].cols};
  return wc::plan_blob(hs.data(), n, p, P);
}

uint64_t capacity_of(const Plan& P) { return P.records_off + P.worst_record_bytes; }

// Launch `kern` over the tensors in groups of kMaxLaunch, each tensor getting
// `wgs_of(T)` workgroups.
template <class WgsOf, class Launch>
bool launch_groups(const Plan& P, const wc_dtensor* dt, const WsLayout& L, EncArgs& args,
                   WgsOf wgs_of, Launch launch) {
  const uint32_t n = uint32_t(P.tensors.size());
  uint32_t t = 0;
  while (t < n) {
    uint32_t nt = 0, wgs = 0;
    for (; t < n && nt < kMaxLaunch; t++) {
      const TensorInfo& T = P.tensors[t];
      const uint32_t w = wgs_of(T);
      if (!w) continue;
      fill_enc(args.t[nt], T, dt[t], L, t);
      args.t[nt].wg0 = wgs;
      nt++;
      wgs += w;
    }
    if (!nt) break;
    args.n_tensors = nt;
    launch(wgs);
    if (hipGetLastError() != hipSuccess) return false;
  }
  return true;
}

}  // namespace

extern "C" wc_status wc_encode_device_bounds(const wc_dtensor* t, uint32_t n, const wc_params* p,
                                             uint64_t* blob_capacity, uint64_t* workspace_bytes) {
  if (!blob_capacity || !workspace_bytes) return WC_EINVAL;
  try {
    Plan P;
    std::vector<wc_tensor> hs;
    wc_status rc = plan_device(t, n, p, P, hs);
    if (rc != WC_OK) return rc;
    const uint64_t cap = capacity_of(P);
    if (cap / 16 >= 0xFFFFFFFFull) return WC_EINVAL;
    WsLayout L;
    layout_ws(P, L);
    *blob_capacity = cap;
    *workspace_bytes = L.total;
    return WC_OK;
  } catch (...) {
    return WC_ENOMEM;
  }
}

extern "C" wc_status wc_encode_device(const wc_dtensor* t, uint32_t n, const wc_params* p,
                                      void* dev_blob, uint64_t blob_capacity, void* dev_workspace,
                                      uint64_t workspace_bytes, void* stream, uint64_t* dev_size) {
  if (!dev_blob || !dev_workspace || !dev_size) return WC_EINVAL;
  if (reinterpret_cast<uintptr_t>(dev_blob) % 16 || reinterpret_cast<uintptr_t>(dev_workspace) % 16 ||
      reinterpret_cast<uintptr_t>(dev_size) % 8)
    return WC_EINVAL;
  try {
    Plan P;
    std::vector<wc_tensor> hs;
    wc_status rc = plan_device(t, n, p, P, hs);
    if (rc != WC_OK) return rc;
    for (uint32_t i = 0; i < n; i++)
      if (t[i].nbytes && (!t[i].dev_ptr || reinterpret_cast<uintptr_t>(t[i].dev_ptr) % 16))
        return WC_EINVAL;
    const uint64_t cap = capacity_of(P);
    if (cap / 16 >= 0xFFFFFFFFull || blob_capacity < cap) return WC_EINVAL;
    WsLayout L;
    layout_ws(P, L);
    if (workspace_bytes < L.total) return WC_EINVAL;
    const hipStream_t st = reinterpret_cast<hipStream_t>(stream);
    const uint64_t blob = reinterpret_cast<uint64_t>(dev_blob);
    const uint64_t ws = reinterpret_cast<uint64_t>(dev_workspace);

    // 1. histograms to zero
    {
      const uint64_t n16 = 8ull * 256 * L.n_tables / 16;
      hipLaunchKernelGGL(zero_kernel, dim3(uint32_t(std::min<uint64_t>((n16 + 255) / 256, 4096))),
                         dim3(256), 0, st, reinterpret_cast<uint4*>(ws + L.hist_off), n16);
      if (hipGetLastError() != hipSuccess) return WC_EHIP;
    }
    EncArgs args{};
    args.blob = blob;
    args.ws = ws;
    args.hist_off = L.hist_off;
    args.tab_off = L.tab_off;
    args.rsz_off = L.rsz_off;
    args.index_off = P.index_off;
    args.raw_start = P.raw_start;
    // 2. histograms
    if (!launch_groups(
            P, t, L, args,
            [](const TensorInfo& T) {
              return uint32_t((T.out_bytes + kHistSpan - 1) / kHistSpan);
            },
            [&](uint32_t wgs) {
              hipLaunchKernelGGL(hist_kernel, dim3(wgs), dim3(kHistThreads), 0, st, args);
            }))
      return WC_EHIP;
    // 3. tables
    {
      NormArgs na{};
      na.blob = blob;
      na.ws = ws;
      na.hist_off = L.hist_off;
      na.tab_off = L.tab_off;
      uint32_t k = 0;
      for (uint32_t i = 0; i <= n; i++) {
        // every table is written, all zeros when no symbol reaches it
        if (i < n && P.owner[i] == i)
          na.t[k++] = NormTable{P.tensors[i].freq_off, L.table_of[i], P.tensors[i].alphabet};
        if (k == 64 || (i == n && k)) {
          na.n_tables = k;
          hipLaunchKernelGGL(norm_kernel, dim3(k), dim3(256), 0, st, na);
          if (hipGetLastError() != hipSuccess) return WC_EHIP;
          k = 0;
        }
      }
    }
    // 4. chunk encoder (and the raw bytes of 16-bit formats)
    if (!launch_groups(
            P, t, L, args,
            [](const TensorInfo& T) { return uint32_t((T.n_chunks + kWaves - 1) / kWaves); },
            [&](uint32_t wgs) {
              hipLaunchKernelGGL(encode_kernel, dim3(wgs), dim3(kThreads), 0, st, args);
            }))
      return WC_EHIP;
    // 5. index and header
    {
      ScanArgs sa{};
      sa.blob = blob;
      sa.ws = ws;
      sa.rsz_off = L.rsz_off;
      sa.size_out = reinterpret_cast<uint64_t>(dev_size);
      sa.index_off = P.index_off;
      sa.raw_start = P.raw_start;
      sa.records_off = P.records_off;
      sa.n_chunks = P.n_chunks;
      uint32_t* h = sa.header;
      put32(h, 0, wc::kMagic);
      h[1] = wc::kVersion | (wc::kHeaderBytes << 16);
      put32(h, 8, n);
      put32(h, 12, wc::kDescBytes);
      put64(h, 16, P.n_chunks);
      put64(h, 32, P.index_off);
      put64(h, 40, P.records_off);
      put64(h, 48, P.raw_start);
      hipLaunchKernelGGL(scan_kernel, dim3(1), dim3(kScanThreads), 0, st, sa);
      if (hipGetLastError() != hipSuccess) return WC_EHIP;
    }
    // 6. descriptors
    for (uint32_t t0 = 0; t0 < n; t0 += 2 * kMaxLaunch) {
      DescArgs da{};
      da.blob = blob;
      da.first = t0;
      da.n = std::min<uint32_t>(2 * kMaxLaunch, n - t0);
      for (uint32_t i = 0; i < da.n; i++) descriptor(P.tensors[t0 + i], P.raw_start, da.d[i]);
      hipLaunchKernelGGL(desc_kernel, dim3(1), dim3(24 * 2 * kMaxLaunch), 0, st, da);
      if (hipGetLastError() != hipSuccess) return WC_EHIP;
    }
    // 7. records
    if (!launch_groups(
            P, t, L, args,
            [](const TensorInfo& T) { return uint32_t((T.n_chunks + kWaves - 1) / kWaves); },
            [&](uint32_t wgs) {
              hipLaunchKernelGGL(pack_kernel, dim3(wgs), dim3(kThreads), 0, st, args);
            }))
      return WC_EHIP;
    return WC_OK;
  } catch (...) {
    return WC_ENOMEM;
  }
}

namespace {

// The histograms of one tensor counted into device memory at dev_workspace
// (65 536 u64 bins, cleared first by a kernel), copied back into `counts` on
// the host (as many bins as the format has) and turned into wc_stats.  The
// caller has checked the arguments.
wc_status analyze_device_into(const wc_dtensor* t, void* dev_workspace, void* stream,
                              wc_stats* out, uint64_t* counts) {
  const uint32_t dt = uint32_t(t->dtype);
  {
    const hipStream_t st = reinterpret_cast<hipStream_t>(stream);
    const uint64_t ws = reinterpret_cast<uint64_t>(dev_workspace);
    const bool words = wc::has_raw(dt);
    const uint64_t bins = words ? 65536 : 256;
    hipLaunchKernelGGL(zero_kernel, dim3(uint32_t((bins * 8 / 16 + 255) / 256)), dim3(256), 0, st,
                       reinterpret_cast<uint4*>(ws), bins * 8 / 16);
    if (hipGetLastError() != hipSuccess) return WC_EHIP;
    if (t->nbytes) {
      if (words) {
        const uint32_t grid =
            uint32_t(std::min<uint64_t>(std::max<uint64_t>((t->nbytes + kHistSpan - 1) / kHistSpan, 1), 1024));
        for (uint32_t part = 0; part < 4; part++) {
          hipLaunchKernelGGL(word_hist_kernel, dim3(grid), dim3(1024), 0, st,
                             reinterpret_cast<uint64_t>(t->dev_ptr), t->nbytes, ws, part);
          if (hipGetLastError() != hipSuccess) return WC_EHIP;
        }
      } else {
        EncArgs a{};
        a.ws = ws;
        a.hist_off = 0;
        a.n_tensors = 1;
        EncTensor& E = a.t[0];
        E.src = reinterpret_cast<uint64_t>(t->dev_ptr);
        E.src_bytes = t->nbytes;
        E.kind = kind_of(dt);
        E.table = 0;
        E.wg0 = 0;
        hipLaunchKernelGGL(hist_kernel, dim3(uint32_t((t->nbytes + kHistSpan - 1) / kHistSpan)),
                           dim3(kHistThreads), 0, st, a);
        if (hipGetLastError() != hipSuccess) return WC_EHIP;
      }
    }
    if (hipMemcpyAsync(counts, dev_workspace, bins * 8, hipMemcpyDeviceToHost, st) != hipSuccess)
      return WC_EHIP;
    if (hipStreamSynchronize(st) != hipSuccess) return WC_EHIP;
    memset(out, 0, sizeof(*out));
    const uint64_t n_sym = wc::symbols_of(dt, t->nbytes);
    if (words) {
      wc::split_word_counts(counts, out);
    } else {
      for (uint32_t s = 0; s < 256; s++) out->hist[0][s] = counts[s];
    }
    wc::finish_stats(dt, n_sym, words ? counts : nullptr, out);
    return WC_OK;
  }
}

// Arguments both analysis entry points check the same way.
bool analyze_args_ok(const wc_dtensor* t, const wc_stats* out) {
  if (!t || !out) return false;
  const uint32_t dt = uint32_t(t->dtype);
  if (!wc::dtype_ok(dt) || (wc::has_raw(dt) && t->nbytes % 2)) return false;
  return !(t->nbytes && (!t->dev_ptr || reinterpret_cast<uintptr_t>(t->dev_ptr) % 16));
}

}  // namespace

extern "C" wc_status wc_analyze_device(const wc_dtensor* t, void* dev_workspace,
                                       uint64_t workspace_bytes, void* stream, wc_stats* out) {
  if (!analyze_args_ok(t, out) || !dev_workspace || workspace_bytes < WC_ANALYZE_WORKSPACE_BYTES)
    return WC_EINVAL;
  if (reinterpret_cast<uintptr_t>(dev_workspace) % 16) return WC_EINVAL;
  try {
    std::vector<uint64_t> counts(WC_ANALYZE_WORKSPACE_BYTES / 8);
    return analyze_device_into(t, dev_workspace, stream, out, counts.data());
  } catch (...) {
    return WC_ENOMEM;
  }
}

// ---------------------------------------------------------------------------
// wc_analyze_device_static: wc_analyze_device for callers that cannot
// allocate.  Its bins live in `scratch`, a device array of the library's own
// (each GPU holds one copy, at its own address, until the process ends); its
// host side copies the counts into a static host array.  One mutex serialises
// the calls of a process, so two calls never share the bins at once.

namespace {

constexpr uint64_t kStaticBins = WC_ANALYZE_WORKSPACE_BYTES / 8;
constexpr int kMaxStaticDevices = 64;

static __device__ __align__(256) uint64_t scratch[kStaticBins];

std::mutex g_static_mu;
void* g_scratch_ptr[kMaxStaticDevices] = {};  // device address of `scratch`, per device
uint64_t g_static_counts[kStaticBins];

}  // namespace

extern "C" wc_status wc_analyze_device_static(const wc_dtensor* t, void* stream, wc_stats* out) {
  if (!analyze_args_ok(t, out)) return WC_EINVAL;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return WC_EHIP;
  if (dev < 0 || dev >= kMaxStaticDevices) return WC_EUNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_static_mu);
  if (!g_scratch_ptr[dev]) {
    // the array's name is a host-side stand-in: only this address is the
    // device's copy, and only it may reach a kernel or a copy
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return WC_EHIP;
    g_scratch_ptr[dev] = p;
  }
  return analyze_device_into(t, g_scratch_ptr[dev], stream, out, g_static_counts);
}
