#pragma once

// wc_decoder.h -- the chunked rANS decoder shared by the decode and the fused
// decode-GEMM kernels of libwc (device code for CDNA4, gfx950), and the launch
// arguments their host sides fill.  Included by wc_decode.hip and wc_gemm.hip.
//
// Paper: Alg. 2 (lane-parallel rANS tile decode: per-lane state, slot = state
// mod 2^b, on-chip table lookup of (symbol, freq, cumfreq), state update
// f * floor(x / 2^b) + slot - cum, renormalisation reads that are coalesced
// because the lanes' words are interleaved in one stream), Sec. V-C-3, and
// Sec. IV-A / V-B (independently decodable units located by an offset index).
//
// Mapping onto the MI355X:
//  * a workgroup of kWaves wave64s decodes chunks of one tensor, one rANS lane
//    per wave lane: a wave decodes one 64-lane chunk, or two adjacent 32-lane
//    chunks, one per half-wave (each half keeps its own word ring and cursor;
//    a lane's rank within its half is the wave's mbcnt minus the lower half's
//    popcount);
//  * the workgroup shares one 4096-entry decode table in LDS, built from the
//    tensor's 2^12-normalised frequencies; an entry is {f | symbol << 24,
//    slot - cum}, so the state update is one v_mad_u32_u24 (the 24-bit multiply
//    ignores the symbol byte);
//  * words reach a per-chunk 2 KiB LDS ring through a fixed-rate pipeline: every
//    four decode steps a chain commits the 256-word unit (8 bytes per lane) it
//    loaded eight steps earlier and issues one new bounds-checked buffer load
//    (the next unit, or a load past the record that returns zeros when the ring
//    is full).  Four steps consume at most 256 words, so the decoder never waits
//    for a unit, and the fixed load pattern gives the compiler exact vmcnt
//    waits.  The ring's first 64 words are mirrored past its end, so a lane's
//    word address is one scalar base plus its rank (two 32-lane chunks per wave move
//    one dword per lane of a half every two steps);
//  * renormalisation: ballot of the lanes whose state fell below 2^16, mbcnt
//    gives each of them its rank, the cursor advances by the popcount -- the
//    lanes' words are consecutive in the stream;
//  * a lane-group is 16 decoded bytes: every G steps a lane assembles a dword
//    (two bf16 rebuilt from their coded and raw bytes with v_perm / v_bfi,
//    four int8 or eight int4), and every 4G steps it stores the four with one
//    16-byte non-temporal (streaming) store, so a wave writes a 1 KiB row;
//  * the raw sign|mantissa bytes of bf16/fp16 rows (8 per lane per row) are
//    loaded two rows ahead with one 8-byte load per lane.
// The decode itself uses no MFMA: it is integer table decoding, not a
// contraction.  The fused decode-GEMM kernels (wc_gemm.hip, Alg. 1 / 3) run the
// same decoder and feed the decoded lane-groups to the VALU dot products or to
// MFMA operands instead of storing them: bf16 as decoded, int8 to
// v_mfma_i32_16x16x64_i8, and fp8, MXFP4 and int4 weights after an exact
// conversion to bf16 (hardware conversions for fp8 / fp4, bit operations for
// int4).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <utility>

#include "wc_internal.h"

namespace {

constexpr int kWaves = 8;                  // waves (chunks) per workgroup
constexpr int kThreads = kWaves * 64;
constexpr int kWaveRingWords = 1024;       // words of a wave's ring (2 KiB)
constexpr int kWaveMirrorWords = 64;       // a ring's first 64 words, mirrored past its end
constexpr int kPipeSteps = 8;              // decode steps between a unit's load and its commit
constexpr int kRawRows = 2;                // raw-byte rows in flight (16-bit formats)
constexpr uint32_t kNoUnit = 0xFFFFFFFFu;
// Offsets that can fall outside a buffer are always passed as the vector
// offset, which the hardware range-checks against num_records; the scalar
// offset carries only offsets that are in range by construction.
constexpr uint32_t kFarOffset = 0x7FFFFF00u;  // past any record: loads return zeros
constexpr int kMaxLaunchTensors = 32;
constexpr int kStreamStore = 2;            // buffer-store cache policy: non-temporal

enum Kind : uint32_t { kSplit16 = 0, kByte = 1, kNibble = 2 };

struct DevTensor {
  uint64_t dst;          // device pointer of the decoded tensor
  uint64_t freq_off;     // u16 frequency table (blob offset)
  union {
    uint64_t raw_off;    // raw bytes (blob offset), 16-bit formats only
    uint64_t zeros;      // fused int4 GEMM: device zero points, [N][K / 128] bytes, or 0
  };
  uint64_t n_sym;        // coded symbols in the tensor
  union {
    uint64_t raw_padded;  // bytes of the (16-B padded) raw region, 16-bit formats only
    uint64_t scales;      // fused MXFP4 GEMM: device e8m0 scales, [N][K / 32] bytes
  };
  uint64_t out_bytes;    // decoded bytes of the tensor
  uint32_t first_chunk;  // global index of the tensor's first chunk
  uint32_t n_chunks;
  uint32_t wg0;          // first workgroup of the tensor in this launch
  uint32_t per;          // symbols per chunk
  uint32_t chunk_bytes;  // decoded bytes per full chunk
  uint32_t kind;
  uint32_t alphabet;
  uint32_t lanes;        // rANS lanes per chunk: 64, or 32 (two chunks per wave)
  uint32_t tiled;        // 1: chunk c is tile (c / ntc, c % ntc) of a row-major matrix
  uint32_t tile_r;       // tile rows
  uint32_t log_tc;       // log2 of the tile columns (symbols)
  uint32_t ntc;          // tiles per band of tile_r rows
  uint32_t pitch;        // decoded bytes of one matrix row
  uint32_t tile_row_bytes;  // decoded bytes of one tile row
  uint32_t order;        // tile order: 0 row-major, 1 column blocks
  uint32_t log_tr;       // log2 of the tile rows (column-block order)
  uint64_t x;            // fused GEMM: const bf16 x[M][K]; y[M][N] is float* dst
};

struct LaunchArgs {
  uint64_t blob;
  uint64_t index_off;
  uint64_t records_off;
  uint64_t records_end;
  uint64_t err;          // int32_t* or 0
  uint32_t n_tensors;
  uint32_t m;            // fused GEMM: rows of x (and of y) in every job
  DevTensor t[kMaxLaunchTensors];
};

constexpr uint32_t wc_ring_words() { return kWaveRingWords + kWaveMirrorWords; }

// Workgroup b of a launch runs on XCD b mod 8 (the eight dies take workgroups
// round-robin, each with its own L2).  Renumber them so that each XCD gets one
// contiguous block of the launch's workgroups: consecutive chunks, whose
// records, raw bytes and outputs are adjacent, then share an XCD.  A
// bijection of [0, n).
__device__ __forceinline__ uint32_t xcd_order(uint32_t b, uint32_t n) {
  const uint32_t x = b % 8u, k = b / 8u, q = n / 8u, r = n % 8u;
  return x * q + min(x, r) + k;
}

__device__ __forceinline__ uint64_t dpad16(uint64_t x) { return (x + 15) & ~uint64_t(15); }

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  // raw buffer: stride 0, num_records in bytes, default data format for gfx9-class parts
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           0x00020000);
}

__device__ __forceinline__ void report(const LaunchArgs& a, uint32_t bits) {
  if (a.err && bits) atomicOr(reinterpret_cast<int32_t*>(a.err), (int32_t)bits);
}

// Decode table of one tensor: slot -> {f | sym << 24, slot - cum_sym}, built
// by a workgroup of kT threads.
template <int kT = kThreads>
__device__ void build_table(const LaunchArgs& a, const DevTensor& T, uint2* tab, uint32_t* cum,
                            uint32_t tid) {
  const uint16_t* fr = reinterpret_cast<const uint16_t*>(a.blob + T.freq_off);
  if (tid < 64) {
    uint32_t f[4];
#pragma unroll
    for (int k = 0; k < 4; k++) {
      uint32_t s = tid * 4 + k;
      f[k] = s < T.alphabet ? fr[s] : 0u;
    }
    uint32_t local = f[0] + f[1] + f[2] + f[3];
    uint32_t incl = local;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      uint32_t v = __shfl_up(incl, d, 64);
      if ((int)tid >= d) incl += v;
    }
    uint32_t base = incl - local;
    cum[tid * 4 + 0] = base;
    cum[tid * 4 + 1] = base + f[0];
    cum[tid * 4 + 2] = base + f[0] + f[1];
    cum[tid * 4 + 3] = base + f[0] + f[1] + f[2];
    if (tid == 63) {
      cum[256] = incl;
      if (incl != wc::kTableSize) report(a, WC_DERR_TABLE);
    }
  }
  __syncthreads();
  constexpr uint32_t kPer = wc::kTableSize / kT;
  const uint32_t j0 = tid * kPer;
  uint32_t lo = 0, hi = 256;  // largest s with cum[s] <= j0
  while (hi - lo > 1) {
    uint32_t mid = (lo + hi) >> 1;
    if (cum[mid] <= j0) lo = mid; else hi = mid;
  }
  uint32_t s = lo;
#pragma unroll
  for (uint32_t j = j0; j < j0 + kPer; j++) {
    while (s < 255 && cum[s + 1] <= j) s++;
    uint32_t f = cum[s + 1] - cum[s];
    tab[j] = make_uint2(f | (s << 24), j - cum[s]);
  }
}

// One decoded dword (G symbols) from the table entries' low words (symbol in
// byte 3) and, for 16-bit formats, its two raw bytes.
template <int G>
__device__ __forceinline__ uint32_t assemble(const uint32_t (&lo)[G], uint32_t raw2) {
  if constexpr (G == 2) {
    // word = raw bit 7 -> bit 15 | coded byte -> bits 14..7 | raw bits 6..0
    const uint32_t E = __builtin_amdgcn_perm(lo[1], lo[0], 0x0C070C03u);  // e0 | e1 << 16
    const uint32_t P = __builtin_amdgcn_perm(0u, raw2, 0x01010000u);       // r0 r0 r1 r1
    const uint32_t M = 0x807F807Fu;
    return (P & M) | ((E << 7) & ~M);
  } else if constexpr (G == 4) {
    const uint32_t b01 = __builtin_amdgcn_perm(lo[1], lo[0], 0x0C0C0703u);
    const uint32_t b23 = __builtin_amdgcn_perm(lo[3], lo[2], 0x0C0C0703u);
    return b01 | (b23 << 16);
  } else {
    // nibbles: even symbols gathered into bytes, odd ones shifted in above them
    const uint32_t e01 = __builtin_amdgcn_perm(lo[2], lo[0], 0x0C0C0703u);
    const uint32_t e23 = __builtin_amdgcn_perm(lo[6], lo[4], 0x0C0C0703u);
    const uint32_t o01 = __builtin_amdgcn_perm(lo[3], lo[1], 0x0C0C0703u);
    const uint32_t o23 = __builtin_amdgcn_perm(lo[7], lo[5], 0x0C0C0703u);
    return (e01 | (e23 << 16)) | ((o01 | (o23 << 16)) << 4);
  }
}

// Everything a wave keeps about the kH chunks it decodes (kH = 64 / L: one
// 64-lane chunk, or two adjacent 32-lane chunks, one per half-wave).  The
// chunks' records, raw bytes and outputs are adjacent, so one buffer
// descriptor spans both and a lane adds its half's base as a vector offset.
template <int L>
struct Chain {
  static constexpr int kH = 64 / L;
  __amdgpu_buffer_rsrc_t rs;  // the chunks' records
  __amdgpu_buffer_rsrc_t rr;  // the chunks' raw bytes (16-bit formats)
  __amdgpu_buffer_rsrc_t os;  // the chunks' decoded bytes
  uint32_t* ring;             // LDS word rings, one per half (kHalfRing32 u32 each)
  uint32_t x;                 // this lane's rANS state
  uint32_t cursor[kH];        // words consumed, per half
  uint32_t issued[kH];        // units loaded or in flight, per half
  uint32_t nunits[kH], nw[kH], A[kH], n_c[kH], wbase[kH];
  uint32_t rec1, raw1, out1;  // half 1's byte offsets within rs / rr / os
  uint32_t n_exist;           // halves with a chunk
  bool ok;
};

// The word pipeline of a wave.  One chunk per wave: a unit is two dwords per
// lane (256 words), loaded and committed every two groups (four steps, which
// read at most 256 words).  Two chunks per wave: a unit is one dword per lane
// of a half (64 words of that half), every group (two steps, at most 64 words
// of a half).  Either way a unit is committed kPipeSteps steps after its load,
// and the ring keeps two spare units.
template <int L>
struct Shape {
  static constexpr int kH = 64 / L;
  static constexpr int kDw = kH == 1 ? 2 : 1;                 // dwords per lane per unit
  static constexpr int kEvery = kDw;                          // groups per pipeline slot
  static constexpr uint32_t kUnitWords = 2 * L * kDw;         // words per unit (per half)
  static constexpr uint32_t kRingWords = kWaveRingWords / kH; // per half
  static constexpr uint32_t kRingUnits = kRingWords / kUnitWords;
  static constexpr int kPipe = kPipeSteps / (2 * kEvery);     // slots between load and commit
  static constexpr uint32_t kMirrorWords = 64 / kH;           // a step reads at most L words
  // a step's reads run at most 64 / kH words past a half's ring: mirrored
  static_assert(kH * (kRingWords + kMirrorWords) <= wc_ring_words(), "ring shape");
  static constexpr uint32_t kHalfRing32 = (kRingWords + kMirrorWords) / 2;
  static_assert(kPipe >= 1 && kPipe <= int(kRingUnits) - 2, "two spare ring units");
  static_assert(2 * kEvery * 64 <= kUnitWords * kH, "a slot's steps read at most one unit");
};

// The index entries of a wave's chunks: g, g + 1 and (two chunks per wave)
// g + 2, clamped to the tensor's chunks.  Loaded before the table build so
// that their latency overlaps it.
struct IndexPre {
  uint32_t v[3];
};

__device__ __forceinline__ IndexPre load_index(const LaunchArgs& a, const DevTensor& T,
                                               uint32_t chunk0, uint32_t per_wave) {
  IndexPre p{};
  if (chunk0 < T.n_chunks) {
    const uint32_t* index = reinterpret_cast<const uint32_t*>(a.blob + a.index_off);
    const uint32_t g = T.first_chunk + chunk0;
    const uint32_t n_exist = min<uint32_t>(per_wave, T.n_chunks - chunk0);
#pragma unroll
    for (uint32_t h = 0; h < 3; h++)
      p.v[h] = __builtin_amdgcn_readfirstlane(index[g + min<uint32_t>(h, n_exist)]);
  }
  return p;
}

template <int L>
__device__ __forceinline__ Chain<L> open_chain(const LaunchArgs& a, const DevTensor& T,
                                               uint32_t chunk0, uint32_t W, uint32_t lane,
                                               uint32_t* ring, const IndexPre& pre) {
  constexpr int kH = Chain<L>::kH;
  Chain<L> c;
  const uint8_t* blob = reinterpret_cast<const uint8_t*>(a.blob);
  c.n_exist = min<uint32_t>(kH, T.n_chunks - chunk0);
  // per-chunk values are wave-uniform; readfirstlane keeps them (and the
  // buffer descriptors built from them) in scalar registers
  uint64_t o[kH + 1];
#pragma unroll
  for (int h = 0; h <= kH; h++) o[h] = 16ull * pre.v[h];
  c.ring = ring;
  c.ok = true;
  uint64_t end = o[0];
#pragma unroll
  for (int h = 0; h < kH; h++) {
    c.cursor[h] = c.issued[h] = 0;
    c.nw[h] = c.nunits[h] = c.wbase[h] = c.A[h] = c.n_c[h] = 0;
    if ((uint32_t)h >= c.n_exist) continue;
    const uint64_t s0 = uint64_t(chunk0 + h) * T.per;
    c.n_c[h] = (uint32_t)min<uint64_t>(T.per, T.n_sym - s0);
    c.A[h] = min<uint32_t>(L, (c.n_c[h] + W - 1) / W);
    bool ok = o[h] >= a.records_off && o[h + 1] <= a.records_end && o[h + 1] >= o[h] + 16;
    if (ok) {
      const uint32_t* rec = reinterpret_cast<const uint32_t*>(blob + o[h]);
      c.nw[h] = __builtin_amdgcn_readfirstlane(rec[0]);
      const uint32_t recA = __builtin_amdgcn_readfirstlane(rec[1]);
      const uint32_t recN = __builtin_amdgcn_readfirstlane(rec[2]);
      c.wbase[h] = (uint32_t)(o[h] - o[0]) + 16u + (uint32_t)dpad16(4ull * c.A[h]);
      ok = recA == c.A[h] && recN == c.n_c[h] &&
           c.wbase[h] + dpad16(2ull * c.nw[h]) == o[h + 1] - o[0];
    }
    c.nunits[h] = ok ? (c.nw[h] + Shape<L>::kUnitWords - 1) / Shape<L>::kUnitWords : 0u;
    c.ok = c.ok && ok;
    end = o[h + 1];
  }
  c.rs = make_rsrc(blob + o[0], c.ok ? (uint32_t)(end - o[0]) : 0u);
  c.rec1 = kH == 2 ? (uint32_t)(o[1] - o[0]) : 0u;
  // lane -> half h, lane within the half
  const uint32_t h = kH == 2 ? lane / L : 0u;
  const uint32_t sub = lane % L;
  const uint32_t A_h = kH == 2 && h ? c.A[kH - 1] : c.A[0];
  c.x = __builtin_amdgcn_raw_buffer_load_b32(c.rs, (h ? c.rec1 : 0u) + 16u + 4u * sub, 0, 0);
  if (sub >= A_h) c.x = wc::kStateLow;  // lanes without symbols keep the initial state
  const uint64_t s0 = uint64_t(chunk0) * T.per;
  if (T.tiled) {
    // a tile's bytes start at its band's first row plus its column offset;
    // the descriptor spans from the first tile's start to the last one's end
    auto base = [&](uint32_t ch) {
      return uint64_t(ch / T.ntc) * T.tile_r * T.pitch + uint64_t(ch % T.ntc) * T.tile_row_bytes;
    };
    const uint64_t out0 = base(chunk0);
    c.out1 = c.n_exist == 2 ? (uint32_t)(base(chunk0 + 1) - out0) : 0u;
    const uint32_t span = c.out1 + (T.tile_r - 1) * T.pitch + T.tile_row_bytes;
    c.os = make_rsrc(reinterpret_cast<const void*>(T.dst + out0), span);
  } else {
    const uint64_t out0 = uint64_t(chunk0) * T.chunk_bytes;
    const uint32_t out_len =
        (uint32_t)min<uint64_t>(uint64_t(kH) * T.chunk_bytes, T.out_bytes - out0);
    c.os = make_rsrc(reinterpret_cast<const void*>(T.dst + out0), out_len);
    c.out1 = T.chunk_bytes;
  }
  const uint32_t raw_len = T.kind == kSplit16
                               ? (uint32_t)min<uint64_t>(uint64_t(kH) * T.per, T.raw_padded - s0)
                               : 0u;
  c.rr = make_rsrc(blob + T.raw_off + s0, raw_len);
  c.raw1 = T.per;
  return c;
}

// Next unit of half h to issue, or kNoUnit when its stream is done or its
// ring is full.
template <int L>
__device__ __forceinline__ uint32_t next_unit(Chain<L>& c, int h) {
  if (c.issued[h] < c.nunits[h] &&
      c.issued[h] < c.cursor[h] / Shape<L>::kUnitWords + Shape<L>::kRingUnits)
    return c.issued[h]++;
  return kNoUnit;
}

// The unit load of one pipeline slot, per lane: unit `u` of the lane's half,
// or (kNoUnit) a load past the records that returns zeros and touches no memory.
template <int L>
__device__ __forceinline__ uint32_t load_unit(const Chain<L>& c, uint32_t u, uint32_t wb,
                                              uint32_t sub) {
  const uint32_t off = u == kNoUnit ? kFarOffset : wb + u * (4u * L);
  return __builtin_amdgcn_raw_buffer_load_b32(c.rs, sub * 4u + off, 0, 0);
}

// One pipeline slot: the unit of each half issued together (one load).
template <int L>
struct Slot {
  uint32_t u;                  // this lane's unit (its half's), or kNoUnit
  uint32_t v[Shape<L>::kDw];   // the loaded dwords
};

template <int L>
__device__ __forceinline__ void commit_unit(const Chain<L>& c, const Slot<L>& s, uint32_t h,
                                            uint32_t sub) {
  const uint32_t u = s.u;
  if (u == kNoUnit) return;
  const uint32_t slot = u % Shape<L>::kRingUnits;
  if constexpr (Chain<L>::kH == 1) {
    // u is wave-uniform here, so both unit tests are scalar branches; the
    // mirror takes the unit's first 64 words (lanes 0..15), all the reads need
    uint2* r = reinterpret_cast<uint2*>(c.ring);
    const uint2 v = make_uint2(s.v[0], s.v[1]);
    r[slot * L + sub] = v;
    if (slot == 0 && sub < Shape<L>::kMirrorWords / 4) r[Shape<L>::kRingWords / 4 + sub] = v;
  } else {
    uint32_t* r = c.ring + h * Shape<L>::kHalfRing32;
    r[slot * L + sub] = s.v[0];
    if (slot == 0 && sub < Shape<L>::kMirrorWords / 2) r[Shape<L>::kRingWords / 2 + sub] = s.v[0];
  }
}

template <int L>
__device__ __forceinline__ Slot<L> issue(Chain<L>& c, uint32_t h, uint32_t sub) {
  Slot<L> s;
  if constexpr (Chain<L>::kH == 1) {
    // wave-uniform, in integer arithmetic (no boolean, which the compiler
    // would carry as a lane mask): the next unit while the stream has one and
    // the ring room.  issued <= lim always: both only grow, issued only below lim.
    using S = Shape<L>;
    const uint32_t lim = min(c.nunits[0], c.cursor[0] / S::kUnitWords + S::kRingUnits);
    const uint32_t take = (c.issued[0] - lim) >> 31;  // lim - issued < 2^31
    const uint32_t none = take - 1u;  // 0, or all ones when nothing is issued
    s.u = c.issued[0] | none;         // the unit, or kNoUnit
    // the unit's offset (below 2^31), or one at least kFarOffset: zeros, no access
    const uint32_t off = (c.wbase[0] + c.issued[0] * (2u * S::kUnitWords)) | (none & kFarOffset);
    c.issued[0] += take;
    const uint2 v = __builtin_bit_cast(
        uint2, __builtin_amdgcn_raw_buffer_load_b64(c.rs, sub * 8u + off, 0, 0));
    s.v[0] = v.x;
    s.v[1] = v.y;
  } else {
    const uint32_t u0 = next_unit(c, 0), u1 = next_unit(c, 1);
    s.u = h ? u1 : u0;
    s.v[0] = load_unit(c, s.u, h ? c.wbase[1] : c.wbase[0], sub);
  }
  return s;
}

// One decode step for the lanes with `active` set; returns the table entry's
// low word (symbol in byte 3).  Branch-free: every lane reads a word and
// v_perm either shifts it in or keeps the state, so a group of steps stays
// one basic block.
// kFoldBase: the ring position of the step's first word rides in the mbcnt
// (its second operand is added to the count), which saves two scalar
// instructions a step and costs one vector move to put the position in a
// VGPR (gfx9 reads one scalar operand per vector instruction).  The decode
// takes it; the fused products, which are bound by their vector instruction
// count, add the position afterwards instead.
template <bool kAll, int L, bool kFoldBase = true>
__device__ __forceinline__ uint32_t step(Chain<L>& c, const uint2* __restrict__ tab, bool active,
                                         uint32_t h) {
  using S = Shape<L>;
  const uint2 e = tab[c.x & (wc::kTableSize - 1)];
  uint32_t xn = __umul24(e.x, c.x >> wc::kProbBits) + e.y;
  uint32_t lo = e.x;
  if (!kAll) {
    xn = active ? xn : c.x;
    lo = active ? lo : 0u;
  }
  const bool need = (kAll || active) && xn < wc::kStateLow;
  const uint64_t m = __ballot(need);
  // the lane's rank among the renormalising lanes (with kFoldBase, on top of
  // the ring position of the step's first word)
  const uint32_t fold = kFoldBase && Chain<L>::kH == 1 ? c.cursor[0] & (S::kRingWords - 1) : 0u;
  const uint32_t rank =
      __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, fold));
  const uint16_t* words = reinterpret_cast<const uint16_t*>(c.ring);
  uint32_t idx;
  if constexpr (Chain<L>::kH == 1) {
    idx = kFoldBase ? rank : (c.cursor[0] & (S::kRingWords - 1)) + rank;
    c.cursor[0] += (uint32_t)__popcll(m);
  } else {
    // the upper half's rank counts the lower half's lanes too: subtract them
    const uint32_t p0 = (uint32_t)__popc((uint32_t)m);
    const uint32_t b0 = c.cursor[0] & (S::kRingWords - 1);
    const uint32_t b1 = 2 * S::kHalfRing32 + (c.cursor[1] & (S::kRingWords - 1)) - p0;
    idx = (h ? b1 : b0) + rank;
    c.cursor[0] += p0;
    c.cursor[1] += (uint32_t)__popc((uint32_t)(m >> 32));
  }
  const uint32_t w = words[idx];
  // bytes {w0, w1, x0, x1} = (x << 16) | w, or {x0, x1, x2, x3} = x
  c.x = __builtin_amdgcn_perm(xn, w, need ? 0x05040100u : 0x07060504u);
  return lo;
}

typedef __attribute__((ext_vector_type(4))) unsigned int u32x4;
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;

// The shared fused GEMM, for many rows of x on column-block tiles of 64 rows:
// the waves of a workgroup decode up to kWaves consecutive tiles of one band
// of 64 W rows (one tile each), so every weight is decoded once per pass over
// the rows of x.  After each pair of wave rows a decoding wave leaves its two
// v_mfma_f32_32x32x16_bf16 B operands (64 W rows x 16 columns) in LDS, and
// every wave multiplies all of them by its own kXB blocks of 32 x rows.
struct Share {
  u32x4* frag;     // LDS [kWaves][2][64]: each wave's B operands of the current pair
  uint32_t wave;   // this wave's slot
  uint32_t n_act;  // waves of the workgroup that decode a tile (operands per pair)
  uint32_t xoff;   // this lane's byte offset in packed x: tile 0, pair 0, x block 0
  uint32_t xtile;  // packed x bytes between two consecutive tiles
  uint32_t xblk;   // packed x bytes between blocks of 32 rows
  uint32_t mrows;  // rows of x from this wave's first (0: none)
  uint32_t first;  // this wave's first row of x (and of y)
  uint32_t n0;     // first W row of the band (column of y)
  uint32_t pairs;  // pairs of wave rows per tile
  uint64_t N;      // columns of y (rows of W)
};

// LDS writes of every wave before the barrier are seen by every wave after it;
// global loads in flight stay in flight.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// A operands of one pair for every decoding wave's tile, from packed x: lane l
// holds x row (first + l mod 32), columns 16 pair + 8 (l div 32) .. of the
// tile; absent tiles and x blocks load nothing.
template <int kXB>
__device__ __forceinline__ void share_load_x(const Share& s, __amdgpu_buffer_rsrc_t xrs,
                                             uint32_t pair, u32x4 (&xs)[kWaves][kXB]) {
#pragma unroll
  for (int f = 0; f < kWaves; f++)
#pragma unroll
    for (int xb = 0; xb < kXB; xb++) {
      const bool use = uint32_t(f) < s.n_act && 32u * xb < s.mrows;
      const uint32_t off = use ? s.xoff + f * s.xtile + xb * s.xblk + pair * 1024u : kFarOffset;
      xs[f][xb] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(xrs, off, 0, 0));
    }
}

// acc[xb][nb] += x block xb times W rows 32 nb .. 32 nb + 31 of every tile's pair
template <int kXB>
__device__ __forceinline__ void share_mma(const Share& s, uint32_t lane,
                                          const u32x4 (&xs)[kWaves][kXB],
                                          f32x16 (&acc)[kXB][2]) {
  if (s.mrows == 0) return;  // no rows of x in this pass: no operand to read
#pragma unroll
  for (int f = 0; f < kWaves; f++) {
    if (uint32_t(f) >= s.n_act) break;
    const bf16x8 b0 = __builtin_bit_cast(bf16x8, s.frag[(2 * f) * 64 + lane]);
    const bf16x8 b1 = __builtin_bit_cast(bf16x8, s.frag[(2 * f + 1) * 64 + lane]);
#pragma unroll
    for (int xb = 0; xb < kXB; xb++) {
      if (32u * xb >= s.mrows) break;
      const bf16x8 A = __builtin_bit_cast(bf16x8, xs[f][xb]);
      acc[xb][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(A, b0, acc[xb][0], 0, 0, 0);
      acc[xb][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(A, b1, acc[xb][1], 0, 0, 0);
    }
  }
}

// y[first + row][n0 + 32 nb + l mod 32] += acc: lane l holds rows
// 8 (i div 4) + 4 (l div 32) + i mod 4 of each 32 x 32 block
template <int kXB>
__device__ __forceinline__ void share_store(const Share& s, uint32_t lane,
                                            const f32x16 (&acc)[kXB][2], float* y) {
#pragma unroll
  for (int xb = 0; xb < kXB; xb++)
#pragma unroll
    for (int nb = 0; nb < 2; nb++)
#pragma unroll
      for (int i = 0; i < 16; i++) {
        const uint32_t row = 32u * xb + 8u * (i >> 2) + 4u * (lane >> 5) + (i & 3);
        if (row < s.mrows)
          unsafeAtomicAdd(y + uint64_t(s.first + row) * s.N + s.n0 + 32u * nb + (lane & 31u),
                          acc[xb][nb][i]);
      }
}

// A wave of the workgroup with no tile to decode (or whose tile's index entry
// is bad): it takes part in every pair's barriers and multiplies the decoding
// waves' operands by its own rows of x.
template <int kXB>
__device__ void share_idle_wave(const LaunchArgs& a, const DevTensor& T, const Share& s,
                                uint32_t lane) {
  const uint32_t K = T.ntc << T.log_tc;
  const __amdgpu_buffer_rsrc_t xrs =
      make_rsrc(reinterpret_cast<const void*>(T.x), ((a.m + 31u) & ~31u) * K * 2u);
  f32x16 acc[kXB][2];
#pragma unroll
  for (int xb = 0; xb < kXB; xb++) acc[xb][0] = acc[xb][1] = f32x16{};
  u32x4 xs[kWaves][kXB];
  for (uint32_t p = 0; p < s.pairs; p++) {
    share_load_x<kXB>(s, xrs, p, xs);
    lds_barrier();
    share_mma<kXB>(s, lane, xs, acc);
    lds_barrier();
  }
  share_store<kXB>(s, lane, acc, reinterpret_cast<float*>(T.dst));
}

// Decode the chunk(s) of one wave, one rANS lane per wave lane.  G symbols
// make one output dword; a lane-group is 4G symbols, 16 output bytes, so a
// lane's share of a row is stored with one 16-byte store.
//
// kGemv: instead of storing a row, multiply it into y (the fused decode-GEMM,
// Alg. 1 / 3).  It needs column-block tiles of 64 rows decoded by 64 lanes:
// lane l then holds 8 consecutive weights of tile row l in every wave row r
// (columns b * tile_c + 8 r ..), so each lane accumulates whole dot products
// of its row with v_dot2_f32_bf16, reading the matching x columns as scalar
// (wave-uniform) loads, and adds them to y once per tile (fp32 atomics: the
// tiles of one row band split K).
//
// kMB: the fused GEMM on the matrix cores, for up to kMR kMB rows of x.  It
// needs column-block tiles of kMR (16 or 32) rows decoded by 64 lanes: lane l
// then holds, in every wave row r, the 8 weights of tile row l mod kMR at
// columns b * tile_c + (512 / kMR) r + 8 (l div kMR) .., which is exactly the
// B operand of v_mfma_f32_16x16x32_bf16 (kMR = 16) or
// v_mfma_f32_32x32x16_bf16 (kMR = 32): B[k][n] = W[n][k], lane l holding
// column n = l mod kMR, rows 8 (l div kMR) ...  Each lane loads the matching
// 8 x values of row l mod kMR of every block of kMR x rows (the A operand;
// rows past M read as zeros through the buffer range check) at the start of
// the wave row, and every wave row issues one MFMA per x block.  At the end
// of the tile each lane adds its kMR * kMR / 64 accumulators per block to y
// (fp32 atomics): lane l holds D[row][l mod kMR] with row = 4 (l div 16) + i
// (kMR = 16) or 8 (i div 4) + 4 (l div 32) + i mod 4 (kMR = 32).
//
// kMR = 64: the same on column-block tiles of 64 rows (the dot-product
// layout: lane l holds row l, columns 8 r ..).  Two wave rows r, r + 1 hold
// 64 rows x 16 columns; one v_permlane32_swap per dword turns them into two
// B operands of v_mfma_f32_32x32x16_bf16 (rows 0..31 and 32..63: lanes 0..31
// keep row r, lanes 32..63 take row r + 1 of the same W rows), which share
// one A operand of x, so every x value loaded feeds 64 W rows.
//
// kShare (with kMR = 64): the shared fused GEMM.  The two B operands of each
// pair go to this wave's slot in LDS instead, and after a workgroup barrier
// every wave multiplies all decoding waves' operands by its own rows of packed
// x (see Share).
template <int G, int L, bool kTiled, int kM = 0, int kMB = 0, int kMR = 16, bool kShare = false,
          int kWF = 0>
__device__ __forceinline__ void decode_chunks(const LaunchArgs& a, const DevTensor& T,
                                              uint32_t chunk0, uint32_t lane,
                                              const uint2* __restrict__ tab, uint32_t* ring,
                                              const IndexPre& pre, const Share* sh = nullptr) {
  constexpr bool kGemv = kM > 0;   // fused GEMM with kM rows of x, dot products
  constexpr bool kMfma = kMB > 0;  // fused GEMM with kMB blocks of x rows, MFMA
  static_assert(!kShare || (kMfma && kMR == 64), "shared fused GEMM: 64-row tiles");
  static_assert(!kGemv || (G == 2 && L == 64 && kTiled), "fused GEMM: bf16, 64-lane tiles");
  static_assert(!kMfma || (L == 64 && kTiled && !kGemv &&
                           (G == 2 || ((G == 4 || (G == 8 && (kWF == 3 || kWF == 4))) &&
                                       kMR == 16 && !kShare))),
                "MFMA GEMM: bf16 tiles, or int8 / fp8 / MXFP4 / int4 tiles of 16 rows");
  // kWF, the weight format the MFMA path converts to bf16 (bf16 x, fp32 sums):
  // 0 none (bf16 weights, or int8 with int8 x); 1 fp8 e4m3; 2 fp8 e5m2;
  // 3 MXFP4 (e2m1 codes, an e8m0 scale per 32-weight lane-group);
  // 4 group-quantised int4 (fp16 scale per 128, zero points or signed codes)
  static_assert(kWF == 0 || ((kWF == 1 || kWF == 2) && kMfma && G == 4) ||
                    (kWF == 3 && kMfma && (G == 8 || G == 4) && kMR == 16 && !kShare) ||
                    (kWF == 4 && kMfma && (G == 4 || G == 8) && kMR == 16 && !kShare),
                "fp8 weights: the byte MFMA path; MXFP4 and int4: nibbles or bytes");
  constexpr bool kInt8 = kMfma && G == 4 && kWF == 0;  // int8 W and x, int32 sums (W8A8)
  constexpr bool kFp8W = kMfma && G == 4 && (kWF == 1 || kWF == 2);  // fp8 W as bf16, bf16 x
  // MXFP4 W as bf16, bf16 x: e2m1 nibble symbols (G = 8), or the packed bytes
  // of two codes as byte symbols (G = 4: two x columns per symbol)
  constexpr bool kMx = kMfma && kWF == 3;
  // int4 W (two codes per byte symbol) as bf16 16 + t, bf16 x, fp32 sums corrected
  // per 128-column group: y += s (sum x (16 + t) - c sum x), c = 16 + z or 24
  constexpr bool kI4 = kMfma && kWF == 4;
  constexpr uint32_t kEPS = (kMx || kI4) && G == 4 ? 2u : 1u;  // x columns per symbol
  static_assert(kMR == 16 || kMR == 32 || kMR == 64, "MFMA tiles of 16, 32 or 64 rows");
  constexpr int kMM = kMR == 64 ? 32 : kMR;   // x rows per MFMA block
  constexpr int kNB = kMR == 64 ? 2 : 1;      // MFMA output blocks of W rows per tile
  constexpr int kH = Chain<L>::kH;
  constexpr int W = 4 * G;                    // symbols per lane-group
  constexpr int kGroupsPerRow = W / 2;        // groups of two steps in a row
  constexpr int kUnroll = G == 2 ? kGroupsPerRow * kRawRows : kGroupsPerRow;  // groups per body
  constexpr uint32_t kRowSym = L * W;          // symbols of one half-row
  constexpr uint32_t kRowBytes = 16u * L;      // decoded bytes of one half-row
  constexpr uint32_t kRawRowBytes = 8u * L;    // raw bytes of one half-row (16-bit formats)
  constexpr uint32_t kLogW = G == 2 ? 3 : (G == 4 ? 4 : 5);
  constexpr int kPipe = Shape<L>::kPipe, kEvery = Shape<L>::kEvery;
  static_assert(!kMfma || kMR != 64 || kUnroll == 2 * kGroupsPerRow, "row pairs per body");
  // Start states that carry data (untiled chunks): a lane's first kCK
  // symbols (kCB bits each, the first lowest) are not coded; the lane ends at
  // 2^kCS + D and they are read back from D.  They all lie in the lane's first
  // output dword.  Tiled chunks (every fused GEMM) carry nothing.
  constexpr uint32_t kCK = kTiled ? 0u : (G == 2 ? 2u : (G == 4 ? 3u : 7u));
  constexpr uint32_t kCB = G == 8 ? 4u : 8u;
  constexpr uint32_t kCS = G == 2 ? 16u : (G == 4 ? 24u : 28u);
  static_assert(kCK <= uint32_t(G) && kCK * kCB <= kCS, "carried symbols fit the first dword");
  static_assert(kUnroll % (kPipe * kEvery) == 0 && kUnroll % kGroupsPerRow == 0,
                "pipeline shape");

  Chain<L> c = open_chain<L>(a, T, chunk0, W, lane, ring, pre);
  if (!c.ok) {
    if (lane == 0) report(a, WC_DERR_INDEX);
    if constexpr (kShare) share_idle_wave<kMB>(a, T, *sh, lane);
    return;
  }
  const uint32_t h = kH == 2 ? lane / L : 0u;
  const uint32_t sub = lane % L;
  // rows every lane of every half decodes in full, and rows in total
  uint32_t rows_full = c.n_c[0] / kRowSym, rows = (c.n_c[0] + kRowSym - 1) / kRowSym;
  if constexpr (kH == 2) {
    rows_full = min(rows_full, c.n_c[1] / kRowSym);
    rows = max(rows, (c.n_c[1] + kRowSym - 1) / kRowSym);
  }
  const uint32_t n_lane = kH == 2 && h ? c.n_c[kH - 1] : c.n_c[0];  // symbols of this lane's chunk
  const uint32_t groups = rows * kGroupsPerRow;
  const uint32_t out_v = (kH == 2 && h ? c.out1 : 0u) + sub * 16u;  // lane's output offset
  const uint32_t half_v = kH == 2 && h ? c.out1 : 0u;                // tiled: half's base
  const uint32_t tc_mask = (1u << T.log_tc) - 1u;
  // output offset (voffset, soffset) of this lane's lane-group in row r: a
  // byte run, or the lane-group's place in the tile of a row-major matrix
  auto out_at = [&](uint32_t r, uint32_t& vo, uint32_t& so) {
    if constexpr (kTiled) {
      const uint32_t i0 = r * kRowSym + sub * W;
      if (T.order == 0) {
        vo = half_v + (i0 >> T.log_tc) * T.pitch + ((i0 & tc_mask) >> kLogW) * 16u;
      } else {
        // lane-group g = i0 / W is row g mod tile_r of k-block g div tile_r
        const uint32_t g = i0 >> kLogW;
        vo = half_v + (g & ((1u << T.log_tr) - 1u)) * T.pitch + (g >> T.log_tr) * 16u;
      }
      so = 0;
    } else {
      vo = out_v;
      so = r * kRowBytes;
    }
  };
  const uint32_t raw_v = (kH == 2 && h ? c.raw1 : 0u) + sub * 8u;   // lane's raw offset

  // prologue: unit 0 committed now, then kPipe units in flight
  Slot<L> pipe[kPipe];
  {
    const Slot<L> s0 = issue(c, h, sub);
    commit_unit(c, s0, h, sub);
  }
#pragma unroll
  for (int j = 0; j < kPipe; j++) pipe[j] = issue(c, h, sub);
  __builtin_amdgcn_wave_barrier();

  // raw bytes (8 per lane per row) of the first kRawRows rows (16-bit formats)
  uint2 rq[G == 2 ? kRawRows : 1];
  if constexpr (G == 2) {
#pragma unroll
    for (int j = 0; j < kRawRows; j++)
      rq[j] = __builtin_bit_cast(
          uint2, __builtin_amdgcn_raw_buffer_load_b64(c.rr, j * kRawRowBytes + raw_v, 0, 0));
  }
  uint32_t lo[G];   // entries of the dword being assembled
  uint32_t ow[4];   // the row's four output dwords
  uint32_t first_dw = 0;  // row 0's first dword without the carried symbols
  float acc[kGemv ? kM : 1];
  // x columns of this tile (fused GEMM), read through the constant address
  // space: the addresses are wave-uniform, so the loads are scalar
  typedef __attribute__((address_space(4))) const uint32_t cu32;
  uint64_t xrow = 0;
  if constexpr (kGemv) {
#pragma unroll
    for (int m = 0; m < kM; m++) acc[m] = 0.0f;
    xrow = T.x + 2ull * (chunk0 % T.ntc) * (1u << T.log_tc);
  }
  typedef __attribute__((ext_vector_type(8))) __bf16 bf8;
  typedef __attribute__((ext_vector_type(kMM * kMM / 64))) float facc;
  typedef __attribute__((ext_vector_type(4))) unsigned int u4v;
  constexpr uint32_t kXB = (G == 2 || kFp8W || kMx || kI4) ? 2u : 1u;  // bytes of an x element
  // bytes of an x row one wave row covers: 64 lane-groups of W columns over kMR rows
  constexpr uint32_t kRowXBytes = 64u * W * kEPS / kMR * kXB;
  typedef __attribute__((ext_vector_type(4))) int i32x4;
  facc macc[kMfma && !kShare && !kInt8 ? kMB : 1][kNB];
  i32x4 iacc[kInt8 ? kMB : 1];                   // int8 GEMM: 16 x 16 int32 sums per block
  f32x16 sacc[kShare ? kMB : 1][2];        // shared GEMM: this wave's x blocks x 64 W rows
  u32x4 xs[kShare ? kWaves : 1][kShare ? kMB : 1];  // shared GEMM: A operands of the pair
  uint32_t prev[kMR == 64 ? 4 : 1];             // 64-row tiles: the even row's dwords
  u4v xa[kMfma ? kMB : 1];
  u4v xa2[kFp8W ? kMB : 1];  // fp8 weights: x columns 8..15 of the lane's 16
  u4v xm[kMx || kI4 ? kMB : 1][3];  // MXFP4 / int4 weights: x columns 8..31 of the lane's 32
  uint32_t mxe = 0;   // MXFP4: the e8m0 scale byte of this lane's lane-group
  uint32_t i4s = 0;   // int4: the fp16 scale of this lane's W row in this wave row's group
  uint32_t i4z = 0;   // int4: its zero point
  // the x rows (fused GEMM on the matrix cores): a.m rows of K bf16
  const uint32_t K = (T.ntc << T.log_tc) * kEPS;  // columns of W = length of an x row
  // (the shared GEMM reads packed x: rows rounded up to blocks of 32)
  const __amdgpu_buffer_rsrc_t xrs = make_rsrc(
      reinterpret_cast<const void*>(T.x),
      kShare ? ((a.m + 31u) & ~31u) * K * 2u : (kMfma ? a.m * K * kXB : 0u));
  uint32_t xoff = 0, xblk = 0;
  if constexpr (kShare) {
#pragma unroll
    for (int xb = 0; xb < kMB; xb++) sacc[xb][0] = sacc[xb][1] = f32x16{};
  } else if constexpr (kMfma) {
#pragma unroll
    for (int mb = 0; mb < kMB; mb++) {
      iacc[kInt8 ? mb : 0] = i32x4{};
#pragma unroll
      for (int nb = 0; nb < kNB; nb++) macc[kInt8 ? 0 : mb][nb] = facc{};
    }
    // this lane's W x values of wave row 0: row sub mod kMM, columns W (sub div kMM) ..
    xoff = ((sub % kMM) * K + (chunk0 % T.ntc) * (kEPS << T.log_tc) + W * kEPS * (sub / kMM)) *
           kXB;
    xblk = kXB * kMM * K;  // bytes of kMM rows of x
  }
  // MXFP4: the scales of W row n, one per 32 columns; the lane-group of this
  // lane in wave row r is k-block (chunk0 mod ntc) tile_c / 32 + 4 r + sub div 16
  const __amdgpu_buffer_rsrc_t mrs = make_rsrc(
      reinterpret_cast<const void*>(kMx ? T.scales : 0ull),
      kMx ? (T.n_chunks / T.ntc) * 16u * (K / 32u) : 0u);
  const uint32_t moff = kMx ? ((chunk0 / T.ntc) * 16u + sub % 16u) * (K / 32u) +
                                  (chunk0 % T.ntc) * ((kEPS << T.log_tc) / 32u) + sub / 16u
                            : 0u;
  // int4: fp16 scales and zero points of W row n, one per 128 columns; wave row r
  // of tile (band, column c) is group c tile_c / 128 + r of the row
  const bool i4zp = kI4 && T.zeros != 0;
  const uint32_t i4n = kI4 ? (T.n_chunks / T.ntc) * 16u * (K / 128u) : 0u;  // groups of W
  const __amdgpu_buffer_rsrc_t srs =
      make_rsrc(reinterpret_cast<const void*>(kI4 ? T.scales : 0ull), 2u * i4n);
  const __amdgpu_buffer_rsrc_t zrs =
      make_rsrc(reinterpret_cast<const void*>(kI4 ? T.zeros : 0ull), i4zp ? i4n : 0u);
  const uint32_t ioff = kI4 ? ((chunk0 / T.ntc) * 16u + sub % 16u) * (K / 128u) +
                                  (chunk0 % T.ntc) * ((kEPS << T.log_tc) / 128u)
                            : 0u;

  // group g of the chunk, j = g mod kUnroll (static)
  auto group = [&](uint32_t g, auto jc, auto tailc, auto firstc) {
    constexpr int j = decltype(jc)::value;
    constexpr bool kTail = decltype(tailc)::value;
    // the first body of full rows: row 0's carried steps are known here
    constexpr bool kFirst = decltype(firstc)::value && j < kGroupsPerRow;
    constexpr int k0 = (j % kGroupsPerRow) * 2;  // first step of this group in its lane-group
    if constexpr (j % kEvery == 0) {
      // every kEvery groups: commit the unit loaded kPipe slots ago, load the next
      constexpr int slot = (j / kEvery) % kPipe;
      commit_unit(c, pipe[slot], h, sub);
      pipe[slot] = issue(c, h, sub);
    }
    __builtin_amdgcn_wave_barrier();
    const uint32_t r = g / kGroupsPerRow;
    if constexpr (kShare) {
      if constexpr (j == 0) share_load_x<kMB>(*sh, xrs, r >> 1, xs);
    }
    if constexpr (kMfma && !kShare && j % kGroupsPerRow == 0 &&
                  (kMR != 64 || j < kGroupsPerRow)) {
      // the A operands of this wave row (512 / kMR columns of each x row; for
      // 64-row tiles, of the even row of a pair: 16 columns)
#pragma unroll
      for (int mb = 0; mb < kMB; mb++) {
        xa[mb] = __builtin_bit_cast(
            u4v, __builtin_amdgcn_raw_buffer_load_b128(xrs, xoff + mb * xblk + r * kRowXBytes,
                                                       0, 0));
        if constexpr (kFp8W)
          xa2[mb] = __builtin_bit_cast(
              u4v, __builtin_amdgcn_raw_buffer_load_b128(
                       xrs, xoff + mb * xblk + r * kRowXBytes + 16u, 0, 0));
        if constexpr (kMx || kI4) {
#pragma unroll
          for (int q = 0; q < 3; q++)
            xm[mb][q] = __builtin_bit_cast(
                u4v, __builtin_amdgcn_raw_buffer_load_b128(
                         xrs, xoff + mb * xblk + r * kRowXBytes + 16u * (q + 1), 0, 0));
        }
      }
      if constexpr (kMx) mxe = __builtin_amdgcn_raw_buffer_load_b8(mrs, moff + 4u * r, 0, 0);
      if constexpr (kI4) {
        i4s = __builtin_amdgcn_raw_buffer_load_b16(srs, 2u * (ioff + r), 0, 0);
        i4z = __builtin_amdgcn_raw_buffer_load_b8(zrs, ioff + r, 0, 0);
      }
    }
    const int nv = kTail ? max(0, min<int>(W, (int)n_lane - (int)(r * kRowSym + sub * W))) : W;
    // in the tail, a runtime row: its carried steps are masked off
    const int kc = kTail && kCK > 0 && r == 0 ? int(kCK) : 0;
#pragma unroll
    for (int k = k0; k < k0 + 2; k++) {
      if (kFirst && uint32_t(k) < kCK)
        lo[k % G] = 0u;  // carried in the start state: not coded
      else
        lo[k % G] = step<!kTail, L, !(kGemv || kMfma)>(c, tab, k < nv && k >= kc, h);
    }
    if constexpr ((k0 + 2) % G == 0) {
      constexpr int d = (k0 + 1) / G;             // the dword these G steps complete
      uint32_t raw2 = 0;
      if constexpr (G == 2) {
        const uint2 rv = rq[(j / kGroupsPerRow) % kRawRows];
        const uint32_t src = d < 2 ? rv.x : rv.y;
        raw2 = d & 1 ? src >> 16 : src;
      }
      ow[d] = assemble<G>(lo, raw2);
      if constexpr (kCK > 0 && d == 0) {
        if (kFirst || (kTail && r == 0)) first_dw = ow[0];
      }
    }
    if constexpr (j % kGroupsPerRow == kGroupsPerRow - 1) {
      if constexpr (G == 2) {
        rq[(j / kGroupsPerRow) % kRawRows] = __builtin_bit_cast(
            uint2, __builtin_amdgcn_raw_buffer_load_b64(c.rr, (r + kRawRows) * kRawRowBytes + raw_v,
                                                        0, 0));
      }
      if constexpr (kMfma && kMR == 64) {
        if constexpr (j < kGroupsPerRow) {
#pragma unroll
          for (int d = 0; d < 4; d++) prev[d] = ow[d];  // the even row waits for its pair
        } else {
          uint32_t b0[4], b1[4];
#pragma unroll
          for (int d = 0; d < 4; d++) {
            const auto sw = __builtin_amdgcn_permlane32_swap(prev[d], ow[d], false, false);
            b0[d] = sw[0];  // W rows 0..31: lanes 0..31 row r, lanes 32..63 row r + 1
            b1[d] = sw[1];  // W rows 32..63
          }
          if constexpr (kShare) {
            // this wave's operands to every wave of the workgroup, then all of them
            // times this wave's rows of x; the second barrier frees the slots
            sh->frag[(2 * sh->wave) * 64 + lane] = u32x4{b0[0], b0[1], b0[2], b0[3]};
            sh->frag[(2 * sh->wave + 1) * 64 + lane] = u32x4{b1[0], b1[1], b1[2], b1[3]};
            lds_barrier();
            share_mma<kMB>(*sh, lane, xs, sacc);
            lds_barrier();
            return;
          }
          const bf8 B0 = __builtin_bit_cast(bf8, u4v{b0[0], b0[1], b0[2], b0[3]});
          const bf8 B1 = __builtin_bit_cast(bf8, u4v{b1[0], b1[1], b1[2], b1[3]});
#pragma unroll
          for (int mb = 0; mb < kMB; mb++) {
            const bf8 A = __builtin_bit_cast(bf8, xa[mb]);
            macc[mb][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(A, B0, macc[mb][0], 0, 0, 0);
            macc[mb][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(A, B1, macc[mb][1], 0, 0, 0);
          }
        }
        return;
      }
      if constexpr (kI4) {
        // 32 int4 codes -> 32 bf16 16 + t (t = q, or the signed code + 8; exact:
        // t sits in the top 4 fraction bits of 2^4), four B operands of 8
        // against x columns 8 q .. of the lane's 32, and four more against ones,
        // which give the group's sums of x in the same layout.  Then
        // y += s (sum x (16 + t) - c sum x) with c = 16 + z, or 24 for signed codes.
        const uint32_t flip = i4zp ? 0u : 0x88888888u;
        uint32_t bw[16];
#pragma unroll
        for (int d = 0; d < 4; d++) {
          const uint32_t v = ow[d] ^ flip;
          const uint32_t lo = v & 0x0F0F0F0Fu, hi = (v >> 4) & 0x0F0F0F0Fu;
#pragma unroll
          for (int b = 0; b < 4; b++) {
            // bytes {lo.b, 0, hi.b, 0}: codes 8 d + 2 b and 8 d + 2 b + 1
            const uint32_t pr = __builtin_amdgcn_perm(hi, lo, 0x0C000C00u | ((4u + b) << 16) | b);
            bw[4 * d + b] = (pr << 3) | 0x41804180u;
          }
        }
        const bf8 ones = __builtin_bit_cast(bf8, u4v{0x3F803F80u, 0x3F803F80u, 0x3F803F80u,
                                                     0x3F803F80u});
        const float sc = (float)__builtin_bit_cast(_Float16, (uint16_t)(i4s & 0xFFFFu));
        const float cc = i4zp ? 16.0f + (float)(i4z & 0xFFu) : 24.0f;
#pragma unroll
        for (int mb = 0; mb < kMB; mb++) {
          facc t{}, u{};
#pragma unroll
          for (int q = 0; q < 4; q++) {
            const bf8 b =
                __builtin_bit_cast(bf8, u4v{bw[4 * q], bw[4 * q + 1], bw[4 * q + 2], bw[4 * q + 3]});
            const bf8 xq = __builtin_bit_cast(bf8, q == 0 ? xa[mb] : xm[mb][q > 0 ? q - 1 : 0]);
            t = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xq, b, t, 0, 0, 0);
            u = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xq, ones, u, 0, 0, 0);
          }
#pragma unroll
          for (int i = 0; i < 4; i++) macc[mb][0][i] += sc * (t[i] - cc * u[i]);
        }
        return;
      }
      if constexpr (kMx) {
        // 32 e2m1 weights -> 32 bf16 times the block's scale 2^(E - 127) (exact
        // while the products stay in bf16's range); byte b of dword d holds
        // weights 8 d + 2 b (low nibble) and 8 d + 2 b + 1.  Four B operands
        // of 8 weights, against x columns 8 q .. 8 q + 7 of the lane's 32.
        const uint32_t e = mxe & 0xFFu;
        const float sc =
            __builtin_bit_cast(float, e == 255u ? 0x7FC00000u : (e ? e << 23 : 0x00400000u));
        uint32_t bw[16];
#pragma unroll
        for (int d = 0; d < 4; d++) {
          bw[4 * d] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(ow[d], sc, 0));
          bw[4 * d + 1] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(ow[d], sc, 1));
          bw[4 * d + 2] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(ow[d], sc, 2));
          bw[4 * d + 3] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(ow[d], sc, 3));
        }
#pragma unroll
        for (int q = 0; q < 4; q++) {
          const bf8 b =
              __builtin_bit_cast(bf8, u4v{bw[4 * q], bw[4 * q + 1], bw[4 * q + 2], bw[4 * q + 3]});
#pragma unroll
          for (int mb = 0; mb < kMB; mb++)
            macc[mb][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf8, q == 0 ? xa[mb] : xm[mb][q > 0 ? q - 1 : 0]), b, macc[mb][0], 0,
                0, 0);
        }
        return;
      }
      if constexpr (kFp8W) {
        // 16 fp8 weights -> 16 bf16 (exact: every e4m3 and e5m2 value is a bf16
        // value; scale 1), two B operands of 8: weights 0..7 and 8..15 of the
        // lane-group, against x columns 0..7 and 8..15 of its 16
        uint32_t bw[8];
#pragma unroll
        for (int d = 0; d < 4; d++) {
          if constexpr (kWF == 1) {
            bw[2 * d] = __builtin_bit_cast(
                uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(ow[d], 1.0f, false));
            bw[2 * d + 1] = __builtin_bit_cast(
                uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(ow[d], 1.0f, true));
          } else {
            bw[2 * d] = __builtin_bit_cast(
                uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_bf8(ow[d], 1.0f, false));
            bw[2 * d + 1] = __builtin_bit_cast(
                uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_bf8(ow[d], 1.0f, true));
          }
        }
        const bf8 b0 = __builtin_bit_cast(bf8, u4v{bw[0], bw[1], bw[2], bw[3]});
        const bf8 b1 = __builtin_bit_cast(bf8, u4v{bw[4], bw[5], bw[6], bw[7]});
#pragma unroll
        for (int mb = 0; mb < kMB; mb++) {
          macc[mb][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf8, xa[mb]),
                                                                b0, macc[mb][0], 0, 0, 0);
          macc[mb][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf8, xa2[mb]),
                                                                b1, macc[mb][0], 0, 0, 0);
        }
        return;
      }
      if constexpr (kInt8) {
        // the lane-group's 16 int8 weights are the B operand as decoded
        const i32x4 b = {int(ow[0]), int(ow[1]), int(ow[2]), int(ow[3])};
#pragma unroll
        for (int mb = 0; mb < kMB; mb++)
          iacc[mb] = __builtin_amdgcn_mfma_i32_16x16x64_i8(__builtin_bit_cast(i32x4, xa[mb]), b,
                                                           iacc[mb], 0, 0, 0);
        return;
      }
      if constexpr (kMfma) {
        const bf8 b = __builtin_bit_cast(bf8, u4v{ow[0], ow[1], ow[2], ow[3]});
#pragma unroll
        for (int mb = 0; mb < kMB; mb++) {
          if constexpr (kMR == 16)
            macc[mb][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf8, xa[mb]),
                                                                  b, macc[mb][0], 0, 0, 0);
          else
            macc[mb][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf8, xa[mb]),
                                                                  b, macc[mb][0], 0, 0, 0);
        }
        return;
      }
      if constexpr (kGemv) {
        // this lane: weights [8 r, 8 r + 8) of its tile row; x rows m < M
        typedef __attribute__((ext_vector_type(2))) __bf16 bf2;
        uint32_t xv[kM][4];
#pragma unroll
        for (int m = 0; m < kM; m++) {
          cu32* xp = reinterpret_cast<cu32*>(
              xrow + 2ull * (uint64_t(m) * (T.ntc << T.log_tc) + r * 8u));
#pragma unroll
          for (int d = 0; d < 4; d++) xv[m][d] = xp[d];
        }
#pragma unroll
        for (int m = 0; m < kM; m++)
#pragma unroll
          for (int d = 0; d < 4; d++)
            acc[m] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf2, ow[d]),
                                                     __builtin_bit_cast(bf2, xv[m][d]), acc[m],
                                                     false);
        return;
      }
      using v4u = __attribute__((ext_vector_type(4))) unsigned int;
      const v4u o = {ow[0], ow[1], ow[2], ow[3]};
      const int nb = nv * 4 / G;  // valid output bytes of this lane
      uint32_t vo, so;
      out_at(r, vo, so);
      if (!kTail || nb == 16) {
        __builtin_amdgcn_raw_buffer_store_b128(o, c.os, vo, so, kStreamStore);
      } else {
#pragma unroll
        for (int d = 0; d < 4; d++) {
          if (4 * d + 4 <= nb) {
            __builtin_amdgcn_raw_buffer_store_b32(ow[d], c.os, vo + 4u * d, so, 0);
          } else {
            for (int b = 4 * d; b < nb; b++)
              __builtin_amdgcn_raw_buffer_store_b8((uint8_t)(ow[d] >> (8 * (b - 4 * d))), c.os,
                                                   vo + b, so, 0);
          }
        }
      }
    }
  };

  const uint32_t groups_full = rows_full * kGroupsPerRow;
  uint32_t g0 = 0;
  if constexpr (kCK > 0) {
    // the first body apart: it leaves row 0's carried steps out
    if (kUnroll <= groups_full) {
      [&]<int... J>(std::integer_sequence<int, J...>) {
        (group(J, std::integral_constant<int, J>{}, std::false_type{}, std::true_type{}), ...);
      }(std::make_integer_sequence<int, kUnroll>{});
      g0 = kUnroll;
    }
  }
  for (; g0 + kUnroll <= groups_full; g0 += kUnroll) {
    [&]<int... J>(std::integer_sequence<int, J...>) {
      (group(g0 + J, std::integral_constant<int, J>{}, std::false_type{}, std::false_type{}),
       ...);
    }(std::make_integer_sequence<int, kUnroll>{});
  }
  // the remaining full groups, then the rows some lanes decode only in part
  // (the last row of a chunk; with two chunks per wave, every row past the
  // shorter chunk's full rows)
  for (; g0 < groups; g0 += kUnroll) {
    [&]<int... J>(std::integer_sequence<int, J...>) {
      ((g0 + J < groups ? group(g0 + J, std::integral_constant<int, J>{}, std::true_type{},
                                std::false_type{})
                        : void()),
       ...);
    }(std::make_integer_sequence<int, kUnroll>{});
  }

  if constexpr (kGemv) {
    // tile (band, column) adds its partial dot products to y
    const uint32_t n = (chunk0 / T.ntc) * 64u + sub;
    const uint64_t N = uint64_t(T.n_chunks / T.ntc) * 64u;
    float* y = reinterpret_cast<float*>(T.dst);
#pragma unroll
    for (int m = 0; m < kM; m++) unsafeAtomicAdd(y + uint64_t(m) * N + n, acc[m]);
  }
  if constexpr (kShare) share_store<kMB>(*sh, lane, sacc, reinterpret_cast<float*>(T.dst));
  if constexpr (kInt8) {
    // D[4 (sub div 16) + i][sub mod 16] of every x block, added to int32 y:
    // integer adds commute, so y is the same whatever order the tiles finish in
    const uint64_t N = uint64_t(T.n_chunks / T.ntc) * kMR;
    int* y = reinterpret_cast<int*>(T.dst);
    const uint32_t n = (chunk0 / T.ntc) * kMR + (sub % 16u);
#pragma unroll
    for (int mb = 0; mb < kMB; mb++)
#pragma unroll
      for (int i = 0; i < 4; i++) {
        const uint32_t m = mb * 16u + 4u * (sub >> 4) + i;
        if (m < a.m) atomicAdd(y + uint64_t(m) * N + n, iacc[mb][i]);
      }
  }
  if constexpr (kMfma && !kShare && !kInt8) {
    // D[row][sub mod kMM] of every x block and W block: y row, W row = y column
    const uint64_t N = uint64_t(T.n_chunks / T.ntc) * kMR;
    float* y = reinterpret_cast<float*>(T.dst);
#pragma unroll
    for (int nb = 0; nb < kNB; nb++) {
      const uint32_t n = (chunk0 / T.ntc) * kMR + nb * kMM + (sub % kMM);
#pragma unroll
      for (int mb = 0; mb < kMB; mb++)
#pragma unroll
        for (int i = 0; i < kMM * kMM / 64; i++) {
          const uint32_t row = kMM == 16 ? 4u * (sub >> 4) + i
                                         : 8u * (i >> 2) + 4u * (sub >> 5) + (i & 3);
          const uint32_t m = mb * kMM + row;
          if (m < a.m) unsafeAtomicAdd(y + uint64_t(m) * N + n, macc[mb][nb][i]);
        }
    }
  }

  // --- end-of-chunk checks: every lane back at its start, every word consumed
  uint32_t bits = 0;
  const uint32_t A_h = kH == 2 && h ? c.A[kH - 1] : c.A[0];
  if constexpr (kCK > 0) {
    // the carried symbols: the lane's first min(kCK, n0) symbols from D
    const uint32_t n0 = n_lane > sub * W ? min<uint32_t>(W, n_lane - sub * W) : 0u;
    const uint32_t kl = min(kCK, n0);
    const uint32_t D = c.x - (1u << kCS);
    const bool bad = (c.x >> kCS) != 1u || (D >> (kCB * kl)) != 0u;
    if (__ballot(sub < A_h && bad)) bits |= WC_DERR_STATE;
    if (n0 > 0) {
      uint32_t lc[G];
#pragma unroll
      for (int t = 0; t < G; t++)
        lc[t] = uint32_t(t) < kl ? ((D >> (kCB * t)) & ((1u << kCB) - 1u)) << 24 : 0u;
      const uint32_t dw = first_dw | assemble<G>(lc, 0u);
      // the lane's first dword again, now whole (only its valid bytes)
      const uint32_t nb = min(4u, n0 * 4u / G + (G == 8 ? (n0 & 1u) : 0u));
      uint32_t vo, so;
      out_at(0, vo, so);
      if (nb == 4) {
        __builtin_amdgcn_raw_buffer_store_b32(dw, c.os, vo, so, 0);
      } else {
        for (uint32_t b = 0; b < nb; b++)
          __builtin_amdgcn_raw_buffer_store_b8((uint8_t)(dw >> (8 * b)), c.os, vo + b, so, 0);
      }
    }
  } else {
    if (__ballot(sub < A_h && c.x != wc::kStateLow)) bits |= WC_DERR_STATE;
  }
#pragma unroll
  for (int k = 0; k < kH; k++)
    if (c.cursor[k] != c.nw[k]) bits |= WC_DERR_CURSOR;
  if (lane == 0) report(a, bits);
}

inline void fill_tensor(DevTensor& D, const wc::TensorInfo& T, const void* dst, uint32_t wg0) {
  D = DevTensor{};
  D.dst = reinterpret_cast<uint64_t>(dst);
  D.freq_off = T.freq_off;
  D.raw_off = T.raw_off;
  D.n_sym = T.n_sym;
  D.out_bytes = T.out_bytes;
  D.raw_padded = wc::has_raw(T.dtype) ? wc::pad16(T.n_sym) : 0;
  D.first_chunk = (uint32_t)T.first_chunk;
  D.n_chunks = (uint32_t)T.n_chunks;
  D.wg0 = wg0;
  D.per = (uint32_t)T.sym_per_chunk();
  D.chunk_bytes = T.chunk_bytes;
  D.kind = wc::is_nibble(T.dtype) ? kNibble : (wc::is_byte(T.dtype) ? kByte : kSplit16);
  D.alphabet = T.alphabet;
  D.lanes = T.lanes;
  D.tiled = T.tile_r ? 1u : 0u;
  if (D.tiled) {
    D.tile_r = T.tile_r;
    D.log_tc = uint32_t(__builtin_ctz(T.tile_c));
    D.ntc = uint32_t(T.cols / T.tile_c);
    D.pitch = uint32_t(T.cols * 16 / T.group);
    D.tile_row_bytes = uint32_t(uint64_t(T.tile_c) * 16 / T.group);
    D.order = T.tile_order;
    D.log_tr = T.tile_order == WC_TILE_COLUMN_BLOCKS ? uint32_t(__builtin_ctz(T.tile_r)) : 0u;
  }
}

inline void fill_common(LaunchArgs& args, const wc::BlobPriv& P, const void* dev_blob, int32_t* dev_err) {
  args.blob = reinterpret_cast<uint64_t>(dev_blob);
  args.index_off = P.index_off;
  args.records_off = P.records_off;
  args.records_end = P.size;
  args.err = reinterpret_cast<uint64_t>(dev_err);
}

}  // namespace
