// wc_decode.hip -- device half of libwc: chunked rANS decode for CDNA4 (gfx950).
//
// Paper: Alg. 2 (lane-parallel rANS tile decode: per-lane state, slot = state
// mod 2^b, on-chip table lookup of (symbol, freq, cumfreq), state update
// f * floor(x / 2^b) + slot - cum, renormalisation reads that are coalesced
// because the lanes' words are interleaved in one stream), Sec. V-C-3, and
// Sec. IV-A / V-B (independently decodable units located by an offset index).
//
// Mapping onto the MI355X:
//  * one wave64 decodes one chunk, one rANS lane per wave lane (64 lanes);
//  * a workgroup holds kWaves chunks of the same tensor and shares one
//    4096-entry decode table in LDS, built from the tensor's 2^12-normalised
//    frequencies; an entry is {f | symbol << 24, slot - cum}, so the state
//    update is a single 24-bit multiply-add (v_mad_u32_u24 ignores the symbol
//    byte);
//  * each wave streams its chunk's 16-bit words through a private 2 KiB LDS
//    ring, refilled 512 B at a time with bounds-checked buffer loads (reads
//    past the chunk record return zero), one segment prefetched ahead;
//  * the raw sign|mantissa bytes of bf16/fp16 rows are loaded 8 rows ahead;
//  * renormalisation: ballot of lanes whose state fell below 2^16, mbcnt gives
//    each such lane its word index (cursor + rank), the cursor advances by the
//    ballot's popcount -- the lanes' words are consecutive in the stream;
//  * every W steps a lane has 4 decoded bytes (two bf16 re-interleaved with
//    their raw sign|mantissa bytes, four int8, or eight int4) and the wave
//    stores 256 contiguous bytes with one dword store per lane.
// No MFMA: the work is integer table decoding, not a contraction.
#include <hip/hip_runtime.h>

#include "wc_internal.h"

namespace {

constexpr int kWaves = 8;                  // chunks (waves) per workgroup
constexpr int kThreads = kWaves * 64;
constexpr int kSegWords = 256;             // refill unit: 512 B, 8 B per lane
constexpr int kRingSegs = 4;               // 2 KiB word ring per wave
constexpr int kRingWords = kRingSegs * kSegWords;
constexpr int kMaxLaunchTensors = 32;

enum Kind : uint32_t { kSplit16 = 0, kByte = 1, kNibble = 2 };

struct DevTensor {
  uint64_t dst;          // device pointer of the decoded tensor
  uint64_t freq_off;     // u16 frequency table (blob offset)
  uint64_t raw_off;      // raw bytes (blob offset), 16-bit formats only
  uint64_t n_sym;        // coded symbols in the tensor
  uint64_t raw_padded;   // bytes of the (16-B padded) raw region
  uint32_t first_chunk;  // global index of the tensor's first chunk
  uint32_t n_chunks;
  uint32_t wg0;          // first workgroup of the tensor in this launch
  uint32_t per;          // symbols per chunk
  uint32_t chunk_bytes;  // decoded bytes per full chunk
  uint32_t kind;
  uint32_t alphabet;
  uint32_t pad;
};

struct LaunchArgs {
  uint64_t blob;
  uint64_t index_off;
  uint64_t records_off;
  uint64_t records_end;
  uint64_t err;          // int32_t* or 0
  uint32_t n_tensors;
  uint32_t pad;
  DevTensor t[kMaxLaunchTensors];
};

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint64_t dpad16(uint64_t x) { return (x + 15) & ~uint64_t(15); }

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  // raw buffer: stride 0, num_records in bytes, default data format for gfx9-class parts
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           0x00020000);
}

__device__ __forceinline__ void report(const LaunchArgs& a, uint32_t bits) {
  if (a.err && bits) atomicOr(reinterpret_cast<int32_t*>(a.err), (int32_t)bits);
}

// Decode table of one tensor: slot -> {f | sym << 24, slot - cum_sym}.
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
  constexpr uint32_t kPer = wc::kTableSize / kThreads;
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

template <int W>
__device__ __forceinline__ uint32_t assemble(const uint32_t (&s)[W], uint32_t raw2) {
  if constexpr (W == 2) {
    // two 16-bit words: coded byte -> bits 14..7, raw bit 7 -> bit 15, raw bits 6..0 stay
    uint32_t E = s[0] | (s[1] << 16);
    uint32_t R = (raw2 & 0xFFu) | ((raw2 & 0xFF00u) << 8);
    return (E << 7) | (R & 0x007F007Fu) | ((R & 0x00800080u) << 8);
  } else if constexpr (W == 4) {
    return s[0] | (s[1] << 8) | (s[2] << 16) | (s[3] << 24);
  } else {
    uint32_t v = 0;
#pragma unroll
    for (int k = 0; k < 8; k++) v |= s[k] << (4 * k);
    return v;
  }
}

// Raw-byte rows prefetched ahead of their use (16-bit formats): the loads of
// rows r+1 .. r+kRawAhead are in flight while row r decodes.
constexpr int kRawAhead = 8;

template <int W>
__device__ void decode_chunk(const LaunchArgs& a, const DevTensor& T, uint32_t chunk,
                             uint32_t lane, const uint2* __restrict__ tab,
                             uint16_t* __restrict__ ring) {
  const uint8_t* blob = reinterpret_cast<const uint8_t*>(a.blob);
  const uint32_t* index = reinterpret_cast<const uint32_t*>(blob + a.index_off);
  const uint32_t g = T.first_chunk + chunk;
  // per-chunk values are wave-uniform; readfirstlane keeps them (and the
  // buffer descriptors built from them) in scalar registers
  const uint64_t o0 = 16ull * __builtin_amdgcn_readfirstlane(index[g]);
  const uint64_t o1 = 16ull * __builtin_amdgcn_readfirstlane(index[g + 1]);
  const uint64_t s0 = uint64_t(chunk) * T.per;
  const uint32_t n_c = (uint32_t)min<uint64_t>(T.per, T.n_sym - s0);
  const uint32_t A = min<uint32_t>(64u, (n_c + W - 1) / W);
  if (o0 < a.records_off || o1 > a.records_end || o1 < o0 + 16) {
    if (lane == 0) report(a, WC_DERR_INDEX);
    return;
  }
  const uint32_t* rec = reinterpret_cast<const uint32_t*>(blob + o0);
  const uint32_t nw = __builtin_amdgcn_readfirstlane(rec[0]);
  const uint32_t recA = __builtin_amdgcn_readfirstlane(rec[1]);
  const uint32_t recN = __builtin_amdgcn_readfirstlane(rec[2]);
  const uint32_t wbase = 16u + (uint32_t)dpad16(4ull * A);
  if (recA != A || recN != n_c || wbase + dpad16(2ull * nw) != o1 - o0) {
    if (lane == 0) report(a, WC_DERR_INDEX);
    return;
  }
  const __amdgpu_buffer_rsrc_t rs = make_rsrc(blob + o0, (uint32_t)(o1 - o0));
  uint32_t x = __builtin_amdgcn_raw_buffer_load_b32(rs, 16u + 4u * lane, 0, 0);
  if (lane >= A) x = wc::kStateLow;  // lanes without symbols keep the initial state

  // --- word ring: segments of kSegWords words, kRingSegs of them per wave ---
  const uint32_t nseg = (nw + kSegWords - 1) / kSegWords;
  uint32_t next_seg = 0;  // first segment not yet in the ring
  bool pend = false;      // registers hold segment next_seg (load issued)
  u32x2 pbuf = {0, 0};
  uint32_t cursor = 0;
  auto issue = [&](uint32_t seg) {
    pbuf = __builtin_amdgcn_raw_buffer_load_b64(
        rs, wbase + seg * (2u * kSegWords) + lane * 8u, 0, 0);
  };
  auto commit = [&](uint32_t seg) {
    *reinterpret_cast<u32x2*>(ring + (seg % kRingSegs) * kSegWords + lane * 4) = pbuf;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
  };
  // make words [cursor, cursor + ahead) resident, then start the next segment
  auto refill = [&](uint32_t ahead) {
    uint32_t need = min((cursor + ahead + kSegWords - 1) / kSegWords, nseg);
    while (next_seg < need) {
      if (!pend) issue(next_seg);
      commit(next_seg);
      next_seg++;
      pend = false;
    }
    if (!pend && next_seg < nseg) {
      issue(next_seg);
      pend = true;
    }
  };

  // --- raw bytes (16-bit formats): row r of lane l is the u16 at r*128 + 2l --
  const uint32_t raw_avail = W == 2 ? (uint32_t)min<uint64_t>(T.per, T.raw_padded - s0) : 0u;
  const __amdgpu_buffer_rsrc_t rr = make_rsrc(blob + T.raw_off + s0, raw_avail);
  auto raw_row = [&](uint32_t r) -> uint32_t {
    // reads at or past raw_avail return 0 (buffer bounds)
    return __builtin_amdgcn_raw_buffer_load_b16(rr, r * 128u + lane * 2u, 0, 0);
  };

  // one decode step for every lane with `active` set
  auto step = [&](uint32_t& sym, bool active) {
    if (active) {
      uint2 e = tab[x & (wc::kTableSize - 1)];
      sym = e.x >> 24;
      x = __umul24(e.x, x >> wc::kProbBits) + e.y;
    }
    bool need = active && x < wc::kStateLow;
    uint64_t m = __ballot(need);
    if (need) {
      uint32_t p = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                             __builtin_amdgcn_mbcnt_lo((uint32_t)m, cursor));
      x = (x << 16) | ring[p & (kRingWords - 1)];
    }
    cursor += (uint32_t)__popcll(m);
  };

  uint32_t* out = reinterpret_cast<uint32_t*>(T.dst + uint64_t(chunk) * T.chunk_bytes);
  const uint32_t rows_full = n_c / (64u * W);
  const uint32_t rem = n_c % (64u * W);

  // a full row: every lane decodes W symbols and stores one dword
  auto full_row = [&](uint32_t r, uint32_t raw2) {
    refill(64u * W);
    uint32_t s[W];
#pragma unroll
    for (int k = 0; k < W; k++) step(s[k], true);
    out[r * 64u + lane] = assemble<W>(s, raw2);
  };
  // the last, partial row: lane l holds min(W, rem - l*W) symbols
  auto tail_row = [&](uint32_t r, uint32_t raw2) {
    refill(64u * W);
    const int v = max(0, min<int>(W, (int)rem - (int)(lane * W)));
    uint32_t s[W];
#pragma unroll
    for (int k = 0; k < W; k++) {
      s[k] = 0;
      step(s[k], k < v);
    }
    const uint32_t word = assemble<W>(s, raw2);
    uint8_t* ob = reinterpret_cast<uint8_t*>(out + r * 64u + lane);
    const int nb = v * 4 / W;  // valid output bytes of this lane
    if (nb == 4) {
      *reinterpret_cast<uint32_t*>(ob) = word;
    } else {
      for (int b = 0; b < nb; b++) ob[b] = (uint8_t)(word >> (8 * b));
    }
  };

  if constexpr (W == 2) {
    uint32_t q[kRawAhead];
#pragma unroll
    for (int j = 0; j < kRawAhead; j++) q[j] = raw_row(j);
    uint32_t r0 = 0;
    for (; r0 + kRawAhead <= rows_full; r0 += kRawAhead) {
#pragma unroll
      for (int j = 0; j < kRawAhead; j++) {
        const uint32_t raw2 = q[j];
        q[j] = raw_row(r0 + j + kRawAhead);
        full_row(r0 + j, raw2);
      }
    }
    // fewer than kRawAhead full rows left, then the partial row; q[j] holds row r0 + j
#pragma unroll
    for (int j = 0; j < kRawAhead; j++) {
      if (r0 + j < rows_full) full_row(r0 + j, q[j]);
      else if (r0 + j == rows_full && rem) tail_row(rows_full, q[j]);
    }
  } else {
    for (uint32_t r = 0; r < rows_full; r++) full_row(r, 0u);
    if (rem) tail_row(rows_full, 0u);
  }

  // --- end-of-chunk checks: every lane back at 2^16, every word consumed ----
  uint32_t bits = 0;
  if (__ballot(lane < A && x != wc::kStateLow)) bits |= WC_DERR_STATE;
  if (cursor != nw) bits |= WC_DERR_CURSOR;
  if (lane == 0) report(a, bits);
}

__global__ __launch_bounds__(kThreads) void wc_decode_kernel(LaunchArgs a) {
  __shared__ uint2 tab[wc::kTableSize];
  __shared__ uint32_t cum[260];
  __shared__ __attribute__((aligned(16))) uint16_t ring[kWaves][kRingWords];

  const uint32_t wg = blockIdx.x;
  uint32_t ti = 0;
  for (uint32_t k = 1; k < a.n_tensors; k++)
    if (wg >= a.t[k].wg0) ti = k;
  const DevTensor& T = a.t[ti];
  const uint32_t tid = threadIdx.x;
  build_table(a, T, tab, cum, tid);
  __syncthreads();
  // the wave index is uniform across the wave; say so, so chunk metadata and
  // buffer descriptors live in scalar registers
  const uint32_t wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const uint32_t lane = __lane_id();
  const uint32_t chunk = (wg - T.wg0) * kWaves + wave;
  if (chunk >= T.n_chunks) return;
  switch (T.kind) {
    case kSplit16: decode_chunk<2>(a, T, chunk, lane, tab, ring[wave]); break;
    case kByte: decode_chunk<4>(a, T, chunk, lane, tab, ring[wave]); break;
    default: decode_chunk<8>(a, T, chunk, lane, tab, ring[wave]); break;
  }
}

}  // namespace

extern "C" wc_status wc_decode(const wc_blob* desc, const void* dev_blob, void* const* dev_dst,
                               uint32_t n, void* stream, int32_t* dev_err) {
  if (!desc || !desc->priv || n != desc->n_tensors || (!dev_dst && n)) return WC_EINVAL;
  if (!dev_blob) return WC_EINVAL;
  const wc::BlobPriv& P = static_cast<const wc::BlobHandle*>(desc->priv)->priv;
  for (uint32_t t = 0; t < n; t++) {
    const wc::TensorInfo& T = P.tensors[t];
    if (T.n_chunks == 0) continue;
    if (T.lanes != 64) return WC_EUNSUPPORTED;
    if (!dev_dst[t]) return WC_EINVAL;
  }
  LaunchArgs args{};
  args.blob = reinterpret_cast<uint64_t>(dev_blob);
  args.index_off = P.index_off;
  args.records_off = P.records_off;
  args.records_end = P.raw_off;
  args.err = reinterpret_cast<uint64_t>(dev_err);
  uint32_t t = 0;
  while (t < n) {
    uint32_t nt = 0, wgs = 0;
    for (; t < n && nt < kMaxLaunchTensors; t++) {
      const wc::TensorInfo& T = P.tensors[t];
      if (T.n_chunks == 0) continue;
      DevTensor& D = args.t[nt++];
      D.dst = reinterpret_cast<uint64_t>(dev_dst[t]);
      D.freq_off = T.freq_off;
      D.raw_off = T.raw_off;
      D.n_sym = T.n_sym;
      D.raw_padded = wc::has_raw(T.dtype) ? wc::pad16(T.n_sym) : 0;
      D.first_chunk = (uint32_t)T.first_chunk;
      D.n_chunks = (uint32_t)T.n_chunks;
      D.wg0 = wgs;
      D.per = (uint32_t)T.sym_per_chunk();
      D.chunk_bytes = T.chunk_bytes;
      D.kind = T.dtype == WC_U4 ? kNibble : (T.dtype == WC_U8 ? kByte : kSplit16);
      D.alphabet = T.alphabet;
      wgs += (uint32_t)((T.n_chunks + kWaves - 1) / kWaves);
    }
    if (nt == 0) break;
    args.n_tensors = nt;
    hipLaunchKernelGGL(wc_decode_kernel, dim3(wgs), dim3(kThreads), 0,
                       reinterpret_cast<hipStream_t>(stream), args);
    if (hipGetLastError() != hipSuccess) return WC_EHIP;
  }
  return WC_OK;
}
