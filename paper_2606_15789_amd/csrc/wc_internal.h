// wc_internal.h -- definitions shared by the host half (wc_host.cpp) and the
// device half (wc_decode.hip) of libwc.  Not part of the public ABI.
#pragma once

#include <stdint.h>

#include <vector>

#include "../../include/wc.h"

namespace wc {

constexpr uint32_t kMagic = 0x31424357u;  // "WCB1"
constexpr uint32_t kVersion = 5;        // blob format version
constexpr uint32_t kProbBits = 12;        // b = 12 (Sec. VI-F)
constexpr uint32_t kTableSize = 1u << kProbBits;
constexpr uint32_t kStateLow = 1u << 16;  // lower end of the state interval
constexpr uint32_t kHeaderBytes = 64;
constexpr uint32_t kDescBytes = 96;
constexpr uint32_t kMaxLanes = 64;
constexpr int kWideWaves = 16;  // waves to a workgroup of the 16-bit decode kernel

// The 16-wave decode kernel for bf16 / fp16 tensors in untiled 64-lane chunks
// (wc_decode_wide.hip): the waves of it resident on the current device at
// once (0 when unknown), and a launch of it with wc_decode's launch arguments
// (`bytes` their size; false on a launch error).
uint64_t wide_resident_waves();
bool wide_launch(const void* launch_args, uint64_t bytes, uint32_t workgroups, void* stream);
// The same for the fused decode-GEMM on 16-row tiles with up to 16 rows of x
// (wc_gemm_wide.hip); kind: 0 int8, 1 fp8 e4m3, 2 fp8 e5m2 weights, 3 MXFP4
// and 4 int4 codes coded as bytes, 5 bf16 weights (0 resident waves, or
// false, for any other kind).
uint64_t gemv_wide_resident_waves(int kind);
bool gemv_wide_launch(int kind, const void* launch_args, uint64_t bytes, uint32_t workgroups,
                      void* stream);
// kind 5 of the two above (wc_gemm_wide_bf16.hip)
uint64_t gemv_wide_bf16_resident_waves();
bool gemv_wide_bf16_launch(const void* launch_args, uint64_t bytes, uint32_t workgroups,
                           void* stream);

inline bool dtype_ok(uint32_t dt) { return dt >= WC_BF16 && dt <= WC_FP4_E2M1; }
inline bool has_raw(uint32_t dt) { return dt == WC_BF16 || dt == WC_FP16; }
// one symbol per byte (int8, fp8) / per nibble, low first (int4, fp4)
inline bool is_byte(uint32_t dt) { return dt == WC_U8 || dt == WC_FP8_E4M3 || dt == WC_FP8_E5M2; }
inline bool is_nibble(uint32_t dt) { return dt == WC_U4 || dt == WC_FP4_E2M1; }
inline uint32_t alphabet_of(uint32_t dt) { return is_nibble(dt) ? 16u : 256u; }
// W: symbols per lane-group; a lane-group is always 16 decoded bytes.
inline uint32_t group_of(uint32_t dt) { return is_nibble(dt) ? 32u : (is_byte(dt) ? 16u : 8u); }
inline uint64_t symbols_of(uint32_t dt, uint64_t bytes) {
  return is_nibble(dt) ? 2 * bytes : (is_byte(dt) ? bytes : bytes / 2);
}
inline uint64_t pad16(uint64_t x) { return (x + 15) & ~uint64_t(15); }

// Start states that carry data (blob version 4).  The encoder's start state
// comes back to the decoder for free at the end of a lane, so an untiled
// chunk spends it: lane l starts at 2^S + D, D packing the lane's first K
// symbols (b bits each, the first lowest), and those steps are not coded.  A
// decoded lane must end at 2^S + D with D within the symbols it carries.
// Tiled chunks, the fused GEMMs' input, start at 2^16 and carry nothing.
struct Carry {
  uint32_t K, b, S;
};
inline Carry carry_of(uint32_t dt, bool tiled) {
  if (tiled) return {0, 8, 16};
  if (has_raw(dt)) return {2, 8, 16};    // exponent bytes of bf16 / fp16
  if (is_nibble(dt)) return {7, 4, 28};  // int4 / fp4 nibbles
  return {3, 8, 24};                     // int8 / fp8 bytes
}
inline bool pow2(uint64_t x) { return x && !(x & (x - 1)); }

// A tensor is cut into tile_r x tile_c tiles (one chunk each) when its shape
// is divided exactly, tile_c is a power of two covering whole lane-groups,
// and a tile's decoded bytes are a valid chunk size; the column-block order
// also needs tile_r to be a power of two.
inline uint64_t tile_bytes(uint32_t dt, uint32_t tr, uint32_t tc) {
  return uint64_t(tr) * tc * 16 / group_of(dt);
}
inline bool tile_ok(uint32_t dt, uint64_t rows, uint64_t cols, uint32_t tr, uint32_t tc,
                    uint32_t order) {
  if (!tr || !tc || !rows || !cols || rows % tr || cols % tc || !pow2(tc) || tc < group_of(dt))
    return false;
  if (order > WC_TILE_COLUMN_BLOCKS || (order == WC_TILE_COLUMN_BLOCKS && !pow2(tr))) return false;
  const uint64_t cb = tile_bytes(dt, tr, tc);
  return cb >= 256 && cb <= (1u << 20) && cb % 256 == 0;
}

struct TensorInfo {
  uint32_t dtype = 0, chunk_bytes = 0, lanes = 0, group = 0, alphabet = 0;
  uint32_t tile_r = 0, tile_c = 0;  // 0, 0: chunks are byte runs
  uint32_t tile_order = 0;          // WC_TILE_ROWS or WC_TILE_COLUMN_BLOCKS
  uint64_t n_sym = 0, out_bytes = 0, first_chunk = 0, n_chunks = 0;
  uint64_t freq_off = 0, raw_off = 0, rows = 0, cols = 0;
  uint64_t sym_per_chunk() const { return symbols_of(dtype, chunk_bytes); }
};

struct BlobPriv {
  std::vector<uint8_t> bytes;
  std::vector<uint64_t> out_bytes;
  std::vector<TensorInfo> tensors;
  // raw regions at [raw_off, records_off), records at [records_off, size)
  uint64_t n_chunks = 0, index_off = 0, raw_off = 0, records_off = 0, size = 0;
};

// What a wc_blob's `priv` points at: the public struct and the parsed blob.
struct BlobHandle {
  wc_blob pub;
  BlobPriv priv;
};

// The data-independent part of a blob's layout, shared by the host encoder
// (wc_encode) and the device encoder (wc_encode_device): per-tensor chunking
// and tiling, the table each tensor uses and where it sits, the chunk index,
// the raw regions (right after the index) and where the records start.  Only
// the records' sizes, and with them the index and the blob's end, depend on
// the coded data.
struct Plan {
  std::vector<TensorInfo> tensors;  // freq_off absolute; raw_off relative to the raw regions' start
  std::vector<uint32_t> owner;      // tensor whose table a tensor uses (itself unless a layer codebook)
  uint64_t n_chunks = 0, index_off = 0, raw_start = 0, records_off = 0;
  uint64_t raw_region_bytes = 0;    // sum of pad16(n_sym) over the 16-bit tensors
  uint64_t worst_record_bytes = 0;  // all records if every symbol emitted a word
};

// Validate the encoder parameters and tensor sizes (WC_EINVAL on any bad
// field; the tensors' pointers are the caller's to check) and lay out the blob.
wc_status plan_blob(const wc_tensor* ts, uint32_t n, const wc_params* p, Plan& out);

// Symbols of chunk c of T, its lane-state count and its largest record.
inline uint64_t chunk_symbols(const TensorInfo& T, uint64_t c) {
  const uint64_t per = T.sym_per_chunk(), s0 = c * per;
  return s0 >= T.n_sym ? 0 : (T.n_sym - s0 < per ? T.n_sym - s0 : per);
}
inline uint32_t chunk_states(const TensorInfo& T, uint64_t n_c) {
  const uint64_t a = (n_c + T.group - 1) / T.group;
  return uint32_t(a < T.lanes ? a : T.lanes);
}
inline uint64_t worst_record(const TensorInfo& T, uint64_t n_c) {
  return 16 + pad16(4ull * chunk_states(T, n_c)) + pad16(2ull * n_c);
}

// Fill the rest of *out from out->hist (the field histograms of a tensor of
// dtype dt with n symbols) and, for 16-bit formats, the 65 536 whole-word
// counts `joint16` (NULL otherwise): entropies, bounds, joint entropy.
void finish_stats(uint32_t dt, uint64_t n, const uint64_t* joint16, wc_stats* out);
// Add whole-word counts of a 16-bit format into out->hist[0] (coded field,
// bits 14..7) and out->hist[1] (raw field, bit 15 and bits 6..0).
void split_word_counts(const uint64_t* joint16, wc_stats* out);

// Validate `size` bytes at `p` and describe them.  Host-side checks of every
// header field, table sum and index entry; WC_EINVAL on the first failure.
wc_status parse_blob(const uint8_t* p, uint64_t size, BlobPriv& out);

}  // namespace wc
