// wc_gemm.hip -- the fused decode-GEMMs (Alg. 1 / 3): wc_gemv, wc_gemm,
// wc_gemm_workspace_bytes, wc_gemm_i8.  The weights are decoded by the
// decoder of wc_decoder.h and multiplied on chip, never written to memory.

#include <mutex>
#include <utility>
#include <vector>

#include "wc_decoder.h"

namespace {

// Packed x: the A operands of v_mfma_f32_32x32x16_bf16 in the order the shared
// GEMM reads them.  Unit (b, p, l) (16 bytes, at ((b K/16 + p) 64 + l) 16) holds
// x row 32 b + l mod 32, columns 16 p + 8 (l div 32) .. + 8, zero past row M, so
// the operand of one block of 32 rows and one pair of wave rows is 1 KiB in a
// row: one fully used load per lane.
__global__ __launch_bounds__(256) void pack_x_kernel(const uint16_t* __restrict__ x, uint32_t m,
                                                    uint32_t K, u32x4* __restrict__ xp,
                                                    uint64_t units) {
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(x, m * K * 2u);
  const uint32_t pairs = K / 16u;
  for (uint64_t u = uint64_t(blockIdx.x) * blockDim.x + threadIdx.x; u < units;
       u += uint64_t(gridDim.x) * blockDim.x) {
    const uint32_t l = uint32_t(u & 63u);
    const uint64_t bp = u >> 6;
    const uint32_t p = uint32_t(bp % pairs), b = uint32_t(bp / pairs);
    const uint32_t row = 32u * b + (l & 31u), col = 16u * p + 8u * (l >> 5);
    xp[u] = __builtin_bit_cast(
        u32x4, __builtin_amdgcn_raw_buffer_load_b128(xr, (row * K + col) * 2u, 0, 0));
  }
}

// The fused decode-GEMM of up to kMaxLaunchTensors tensors in one launch: one
// wave per tile, y += x * W^T for each tensor's own x and y.  kM > 0: column-
// block tiles of 64 x tile_c bf16, kM rows of x, dot products on the VALU;
// kMB > 0: column-block tiles of kMR x tile_c, up to kMR kMB rows of x, MFMA
// (G = 2: bf16; G = 4: int8 W and x, 16-row tiles, int32 y; G = 4 with kFp8:
// fp8 e4m3 W converted to bf16, bf16 x, 16-row tiles, fp32 y).
template <int kM, int kMB, int kMR = 16, int G = 2, bool kFp8 = false>
__global__ __launch_bounds__(kThreads) void wc_gemv_kernel(LaunchArgs a) {
  __shared__ uint2 tab[wc::kTableSize];
  __shared__ uint32_t cum[260];
  __shared__ uint32_t ring[kWaves][wc_ring_words() / 2];
  const uint32_t wg = blockIdx.x;
  uint32_t ti = 0;
  for (uint32_t k = 1; k < a.n_tensors; k++)
    if (wg >= a.t[k].wg0) ti = k;
  const DevTensor& T = a.t[ti];
  const uint32_t tid = threadIdx.x;
  const uint32_t wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const uint32_t lane = __lane_id();
  const uint32_t chunk = (wg - T.wg0) * kWaves + wave;
  const IndexPre pre = load_index(a, T, chunk, 1u);
  build_table(a, T, tab, cum, tid);
  __syncthreads();
  if (chunk >= T.n_chunks) return;
  decode_chunks<G, 64, true, kM, kMB, kMR, false, kFp8 ? 1 : 0>(a, T, chunk, lane, tab, ring[wave],
                                                                pre);
}

// The same fused decode-GEMM for fp8 e5m2 weights on 16-row tiles: kMB blocks
// of 16 x rows, each lane-group converted to bf16 as it is decoded.
template <int kMB>
__global__ __launch_bounds__(kThreads) void wc_gemv_e5m2_kernel(LaunchArgs a) {
  __shared__ uint2 tab[wc::kTableSize];
  __shared__ uint32_t cum[260];
  __shared__ uint32_t ring[kWaves][wc_ring_words() / 2];
  const uint32_t wg = blockIdx.x;
  uint32_t ti = 0;
  for (uint32_t k = 1; k < a.n_tensors; k++)
    if (wg >= a.t[k].wg0) ti = k;
  const DevTensor& T = a.t[ti];
  const uint32_t tid = threadIdx.x;
  const uint32_t wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const uint32_t lane = __lane_id();
  const uint32_t chunk = (wg - T.wg0) * kWaves + wave;
  const IndexPre pre = load_index(a, T, chunk, 1u);
  build_table(a, T, tab, cum, tid);
  __syncthreads();
  if (chunk >= T.n_chunks) return;
  decode_chunks<4, 64, true, 0, kMB, 16, false, 2>(a, T, chunk, lane, tab, ring[wave], pre);
}

// The same fused decode-GEMM for MXFP4 weights (e2m1 nibbles, 16-row tiles):
// kMB blocks of 16 x rows, each 32-weight lane-group converted to bf16 with
// its e8m0 scale as it is decoded.
template <int kMB>
__global__ __launch_bounds__(kThreads) void wc_gemv_mx_kernel(LaunchArgs a) {
  __shared__ uint2 tab[wc::kTableSize];
  __shared__ uint32_t cum[260];
  __shared__ uint32_t ring[kWaves][wc_ring_words() / 2];
  const uint32_t wg = blockIdx.x;
  uint32_t ti = 0;
  for (uint32_t k = 1; k < a.n_tensors; k++)
    if (wg >= a.t[k].wg0) ti = k;
  const DevTensor& T = a.t[ti];
  const uint32_t tid = threadIdx.x;
  const uint32_t wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const uint32_t lane = __lane_id();
  const uint32_t chunk = (wg - T.wg0) * kWaves + wave;
  const IndexPre pre = load_index(a, T, chunk, 1u);
  build_table(a, T, tab, cum, tid);
  __syncthreads();
  if (chunk >= T.n_chunks) return;
  decode_chunks<8, 64, true, 0, kMB, 16, false, 3>(a, T, chunk, lane, tab, ring[wave], pre);
}

// The same for MXFP4 codes coded as bytes (WC_U8 tensors holding the packed
// e2m1 pairs): byte symbols, half the decode steps per weight.
template <int kMB>
__global__ __launch_bounds__(kThreads) void wc_gemv_mxb_kernel(LaunchArgs a) {
  __shared__ uint2 tab[wc::kTableSize];
  __shared__ uint32_t cum[260];
  __shared__ uint32_t ring[kWaves][wc_ring_words() / 2];
  const uint32_t wg = blockIdx.x;
  uint32_t ti = 0;
  for (uint32_t k = 1; k < a.n_tensors; k++)
    if (wg >= a.t[k].wg0) ti = k;
  const DevTensor& T = a.t[ti];
  const uint32_t tid = threadIdx.x;
  const uint32_t wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const uint32_t lane = __lane_id();
  const uint32_t chunk = (wg - T.wg0) * kWaves + wave;
  const IndexPre pre = load_index(a, T, chunk, 1u);
  build_table(a, T, tab, cum, tid);
  __syncthreads();
  if (chunk >= T.n_chunks) return;
  decode_chunks<4, 64, true, 0, kMB, 16, false, 3>(a, T, chunk, lane, tab, ring[wave], pre);
}

// The fused decode-GEMM for group-quantised int4 weights (codes as bytes,
// 16-row tiles): kMB blocks of 16 x rows.
template <int kMB>
__global__ __launch_bounds__(kThreads) void wc_gemv_w4_kernel(LaunchArgs a) {
  __shared__ uint2 tab[wc::kTableSize];
  __shared__ uint32_t cum[260];
  __shared__ uint32_t ring[kWaves][wc_ring_words() / 2];
  const uint32_t wg = blockIdx.x;
  uint32_t ti = 0;
  for (uint32_t k = 1; k < a.n_tensors; k++)
    if (wg >= a.t[k].wg0) ti = k;
  const DevTensor& T = a.t[ti];
  const uint32_t tid = threadIdx.x;
  const uint32_t wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const uint32_t lane = __lane_id();
  const uint32_t chunk = (wg - T.wg0) * kWaves + wave;
  const IndexPre pre = load_index(a, T, chunk, 1u);
  build_table(a, T, tab, cum, tid);
  __syncthreads();
  if (chunk >= T.n_chunks) return;
  decode_chunks<4, 64, true, 0, kMB, 16, false, 4>(a, T, chunk, lane, tab, ring[wave], pre);
}

// The same for int4 codes as nibble symbols (WC_U4 tensors).
template <int kMB>
__global__ __launch_bounds__(kThreads) void wc_gemv_w4n_kernel(LaunchArgs a) {
  __shared__ uint2 tab[wc::kTableSize];
  __shared__ uint32_t cum[260];
  __shared__ uint32_t ring[kWaves][wc_ring_words() / 2];
  const uint32_t wg = blockIdx.x;
  uint32_t ti = 0;
  for (uint32_t k = 1; k < a.n_tensors; k++)
    if (wg >= a.t[k].wg0) ti = k;
  const DevTensor& T = a.t[ti];
  const uint32_t tid = threadIdx.x;
  const uint32_t wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const uint32_t lane = __lane_id();
  const uint32_t chunk = (wg - T.wg0) * kWaves + wave;
  const IndexPre pre = load_index(a, T, chunk, 1u);
  build_table(a, T, tab, cum, tid);
  __syncthreads();
  if (chunk >= T.n_chunks) return;
  decode_chunks<8, 64, true, 0, kMB, 16, false, 4>(a, T, chunk, lane, tab, ring[wave], pre);
}

// The shared fused GEMM: workgroup = (pass over 256 kXB rows of x, band of 64
// W rows, segment of kWaves consecutive tiles of the band); wave w decodes tile
// w of the segment (when the band has one) and owns x rows 32 kXB w .. of the
// pass.  Every tile must be full: 64 rows, tile_c columns.  DevTensor::x is the
// packed x of the job (pack_x_kernel).
template <int kXB>
__global__ __launch_bounds__(kThreads) void wc_gemm_kernel(LaunchArgs a) {
  __shared__ uint2 tab[wc::kTableSize];
  __shared__ uint32_t cum[260];
  __shared__ uint32_t ring[kWaves][wc_ring_words() / 2];
  __shared__ u32x4 frag[kWaves * 2 * 64];
  const uint32_t wg = blockIdx.x;
  uint32_t ti = 0;
  for (uint32_t k = 1; k < a.n_tensors; k++)
    if (wg >= a.t[k].wg0) ti = k;
  const DevTensor& T = a.t[ti];
  const uint32_t tid = threadIdx.x;
  const uint32_t wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const uint32_t lane = __lane_id();
  const uint32_t bands = T.n_chunks / T.ntc;
  const uint32_t segs = (T.ntc + kWaves - 1) / kWaves;
  const uint32_t local = wg - T.wg0;
  const uint32_t pass = local / (bands * segs), rest = local % (bands * segs);
  const uint32_t band = rest / segs, seg = rest % segs;
  Share s;
  s.frag = frag;
  s.wave = wave;
  s.n_act = min<uint32_t>(kWaves, T.ntc - seg * kWaves);
  const uint32_t K = T.ntc << T.log_tc;
  s.first = (pass * kWaves + wave) * 32u * kXB;
  s.mrows = s.first < a.m ? a.m - s.first : 0u;
  // packed x: 1 KiB per (block of 32 rows, pair of columns 16 p ..)
  s.xoff = s.mrows ? ((s.first / 32u) * (K / 16u) * 64u + lane) * 16u +
                         seg * kWaves * ((1u << T.log_tc) / 16u) * 1024u
                   : 0u;
  s.xtile = (1u << T.log_tc) * 64u;
  s.xblk = K * 64u;
  s.n0 = band * 64u;
  s.pairs = (1u << T.log_tc) / 16u;
  s.N = uint64_t(bands) * 64u;
  // waves past the band's last tile decode nothing; they index a tile that exists
  const bool decodes = wave < s.n_act;
  const uint32_t chunk = band * T.ntc + seg * kWaves + (decodes ? wave : 0u);
  const IndexPre pre = load_index(a, T, chunk, 1u);
  build_table(a, T, tab, cum, tid);
  __syncthreads();
  if (decodes)
    decode_chunks<2, 64, true, 0, kXB, 64, true>(a, T, chunk, lane, tab, ring[wave], pre, &s);
  else
    share_idle_wave<kXB>(a, T, s, lane);
}

}  // namespace

// Rows of x up to which 64-row tiles take the VALU dot products; above, the
// matrix cores (row pairs swapped into 32 x 32 x 16 MFMA operands).
constexpr uint32_t kDotRows = 5;
// Rows of x up to which wc_gemm runs wc_gemv's kernels; above, the shared
// fused GEMM (one decode of every tile per pass of kPassRows x rows) over
// packed x.  kMaxGemmRows: the most rows of x wc_gemm takes.
constexpr uint32_t kShareRows = 64;
constexpr uint32_t kMaxGemmRows = 4096;
constexpr uint32_t kPassRows = kWaves * 32u;

namespace {

uint64_t pad256(uint64_t v) { return (v + 255) & ~uint64_t(255); }

// Arguments of a fused GEMM call, before anything is launched.  share: the
// jobs go to the shared fused GEMM (64-row tiles, every tile full).
wc_status check_jobs(const wc_blob* desc, const void* dev_blob, uint32_t n,
                     const uint32_t* tensors, const void* const* dev_x, uint32_t m,
                     float* const* dev_y, bool share) {
  if (!desc || !desc->priv || !dev_blob || !tensors || !dev_x || !dev_y || n == 0 ||
      n > kMaxLaunchTensors)
    return WC_EINVAL;
  const wc::BlobPriv& P = static_cast<const wc::BlobHandle*>(desc->priv)->priv;
  for (uint32_t i = 0; i < n; i++) {
    if (tensors[i] >= desc->n_tensors || !dev_x[i] || !dev_y[i] ||
        reinterpret_cast<uintptr_t>(dev_x[i]) % 16)
      return WC_EINVAL;
    const wc::TensorInfo& T = P.tensors[tensors[i]];
    if (T.lanes != 64 || T.tile_order != WC_TILE_COLUMN_BLOCKS ||
        !(T.tile_r == 64 || T.tile_r == 32 || T.tile_r == 16))
      return WC_EUNSUPPORTED;
    // bf16 weights on every tile height; fp8 e4m3 or e5m2 on 16-row tiles (not shared)
    const bool fp8 = T.dtype == WC_FP8_E4M3 || T.dtype == WC_FP8_E5M2;
    if (!(T.dtype == WC_BF16 || (fp8 && T.tile_r == 16 && !share)))
      return WC_EUNSUPPORTED;
    // 64-row tiles past the dot-product rows pair k-blocks r and r+1 of one
    // tile: at least two k-blocks (16 columns) per tile
    if (T.tile_r == 64 && m > kDotRows && T.tile_c < 16) return WC_EUNSUPPORTED;
    if (T.rows > 0xFFFFFFFFull || T.cols > 0xFFFFFFFFull) return WC_EUNSUPPORTED;
    // x offsets of a lane reach 64 rows (4 blocks of 16) of 2 * cols bytes
    if (64ull * T.cols * 2 > 0x7FFFFFFFull) return WC_EUNSUPPORTED;
    if (share) {
      // every wave of a workgroup takes the same number of pairs of wave rows:
      // 64-row tiles, all full; packed x addressed below kFarOffset
      if (T.tile_r != 64 || T.rows % 64 || T.cols % T.tile_c) return WC_EUNSUPPORTED;
      if (uint64_t((m + 31) / 32 * 32) * T.cols * 2 > kFarOffset) return WC_EUNSUPPORTED;
    }
  }
  return WC_OK;
}

// Resident waves of the 8-wave fused-GEMM kernel for 16-row tiles with one
// block of x rows (kind: 0 int8, 1 fp8 e4m3, 2 fp8 e5m2 weights, 3 MXFP4 and
// 4 int4 codes coded as bytes, 5 bf16 weights), and of its
// 16-wave counterpart in wc_gemm_wide.hip, worked out once per device ({0, 0}
// when unknown).  A launch whose tiles overflow the first but fit the second
// runs on the 16-wave kernel, in one round.
bool gemv_wide(int kind, uint64_t tiles) {
  struct Cap {
    uint64_t general, wide;
  };
  if (kind < 0 || kind > 5) return false;
  static std::mutex mu;
  static std::vector<std::pair<int, Cap>> known[6];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return false;
  Cap c{0, 0};
  {
    std::lock_guard<std::mutex> lock(mu);
    bool found = false;
    for (const auto& k : known[kind])
      if (k.first == dev) c = k.second, found = true;
    if (!found) {
      int cus = 0, per_cu = 0;
      const void* k8 =
          kind == 5   ? reinterpret_cast<const void*>(wc_gemv_kernel<0, 1, 16>)
          : kind == 4 ? reinterpret_cast<const void*>(wc_gemv_w4_kernel<1>)
          : kind == 3 ? reinterpret_cast<const void*>(wc_gemv_mxb_kernel<1>)
          : kind == 2 ? reinterpret_cast<const void*>(wc_gemv_e5m2_kernel<1>)
          : kind == 1 ? reinterpret_cast<const void*>(wc_gemv_kernel<0, 1, 16, 4, true>)
                      : reinterpret_cast<const void*>(wc_gemv_kernel<0, 1, 16, 4, false>);
      if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
          hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k8, kThreads, 0) == hipSuccess)
        c = Cap{uint64_t(cus) * uint64_t(per_cu) * uint64_t(kWaves),
                wc::gemv_wide_resident_waves(kind)};
      known[kind].push_back({dev, c});
    }
  }
  return c.general && c.wide > c.general && tiles > c.general && tiles <= c.wide;
}

// Rows of x up to which the byte-coded MXFP4 and int4 launches take the 16-wave
// kernel (in its window): on the 8B layers it gains 3-9 % up to 8 rows, nothing
// at 12 and loses at 16 rows, where each wave row's conversions and products
// weigh more than the extra waves.
constexpr uint32_t kWideQ4Rows = 8;

// One launch per tile height and weight type (bf16 on 64 rows: VALU dot
// products up to kDotRows rows of x, MFMA above, or the shared GEMM; bf16 on
// 32 or 16 rows: MFMA; fp8 e4m3, then e5m2, on 16 rows: converted to bf16,
// MFMA; 16-row launches with one block of x rows may take the 16-wave kernel,
// see gemv_wide).  xs: the x (or, for the shared GEMM, packed x) of each job.
wc_status launch_jobs(const wc::BlobPriv& P, const void* dev_blob, uint32_t n,
                      const uint32_t* tensors, const uint64_t* xs, uint32_t m,
                      float* const* dev_y, bool share, hipStream_t st, int32_t* dev_err) {
  for (uint32_t kind = 0; kind < 5; kind++) {
    // bf16 weights on 64-, 32- and 16-row tiles, then fp8 e4m3 and e5m2 weights
    // on 16-row tiles
    const uint32_t rows = kind == 0 ? 64u : (kind == 1 ? 32u : 16u);
    const uint32_t f8 = kind < 3 ? 0u : kind - 2u;  // 0 bf16, 1 e4m3, 2 e5m2
    const uint32_t dtype = f8 == 0 ? WC_BF16 : (f8 == 1 ? WC_FP8_E4M3 : WC_FP8_E5M2);
    LaunchArgs args{};
    fill_common(args, P, dev_blob, dev_err);
    // bf16 or fp8 on 16-row tiles with one block of x rows: the 16-wave
    // kernel when its tiles fit it
    const int wide_kind = f8 ? int(f8) : 5;
    bool wide = false;
    if (rows == 16 && !share && m <= 16) {
      uint64_t tiles = 0;
      for (uint32_t i = 0; i < n; i++) {
        const wc::TensorInfo& T = P.tensors[tensors[i]];
        if (T.tile_r == rows && T.dtype == dtype) tiles += T.n_chunks;
      }
      wide = tiles && gemv_wide(wide_kind, tiles);
    }
    const uint64_t per_wg = wide ? uint64_t(wc::kWideWaves) : uint64_t(kWaves);
    uint32_t wgs = 0, nt = 0;
    for (uint32_t i = 0; i < n; i++) {
      const wc::TensorInfo& T = P.tensors[tensors[i]];
      if (T.tile_r != rows || T.dtype != dtype) continue;
      fill_tensor(args.t[nt], T, dev_y[i], wgs);
      args.t[nt].x = xs[i];
      if (share) {
        // (pass, band, segment of kWaves tiles) per workgroup
        const uint64_t ntc = T.cols / T.tile_c, bands = T.rows / 64;
        const uint64_t segs = (ntc + kWaves - 1) / kWaves, passes = (m + kPassRows - 1) / kPassRows;
        wgs += uint32_t(bands * segs * passes);
      } else {
        wgs += uint32_t((T.n_chunks + per_wg - 1) / per_wg);
      }
      nt++;
    }
    if (!nt) continue;
    args.n_tensors = nt;
    args.m = m;
    if (wide) {
      if (!wc::gemv_wide_launch(wide_kind, &args, sizeof args, wgs, st)) return WC_EHIP;
      continue;
    }
    const dim3 grid(wgs), block(kThreads);
    if (f8 == 1) {
      switch ((m + 15) / 16) {
        case 1: hipLaunchKernelGGL((wc_gemv_kernel<0, 1, 16, 4, true>), grid, block, 0, st, args); break;
        case 2: hipLaunchKernelGGL((wc_gemv_kernel<0, 2, 16, 4, true>), grid, block, 0, st, args); break;
        case 3: hipLaunchKernelGGL((wc_gemv_kernel<0, 3, 16, 4, true>), grid, block, 0, st, args); break;
        default: hipLaunchKernelGGL((wc_gemv_kernel<0, 4, 16, 4, true>), grid, block, 0, st, args); break;
      }
    } else if (f8 == 2) {
      switch ((m + 15) / 16) {
        case 1: hipLaunchKernelGGL((wc_gemv_e5m2_kernel<1>), grid, block, 0, st, args); break;
        case 2: hipLaunchKernelGGL((wc_gemv_e5m2_kernel<2>), grid, block, 0, st, args); break;
        case 3: hipLaunchKernelGGL((wc_gemv_e5m2_kernel<3>), grid, block, 0, st, args); break;
        default: hipLaunchKernelGGL((wc_gemv_e5m2_kernel<4>), grid, block, 0, st, args); break;
      }
    } else if (share) {
      hipLaunchKernelGGL((wc_gemm_kernel<1>), grid, block, 0, st, args);
    } else if (rows == 64 && m > kDotRows) {
      if (m <= 32) hipLaunchKernelGGL((wc_gemv_kernel<0, 1, 64>), grid, block, 0, st, args);
      else hipLaunchKernelGGL((wc_gemv_kernel<0, 2, 64>), grid, block, 0, st, args);
    } else if (rows == 64) {
      switch (m) {
        case 1: hipLaunchKernelGGL((wc_gemv_kernel<1, 0>), grid, block, 0, st, args); break;
        case 2: hipLaunchKernelGGL((wc_gemv_kernel<2, 0>), grid, block, 0, st, args); break;
        case 3: hipLaunchKernelGGL((wc_gemv_kernel<3, 0>), grid, block, 0, st, args); break;
        case 4: hipLaunchKernelGGL((wc_gemv_kernel<4, 0>), grid, block, 0, st, args); break;
        default: hipLaunchKernelGGL((wc_gemv_kernel<5, 0>), grid, block, 0, st, args); break;
      }
      static_assert(kDotRows == 5, "one dot-product instance per row count up to kDotRows");
    } else if (rows == 32) {
      if (m <= 32) hipLaunchKernelGGL((wc_gemv_kernel<0, 1, 32>), grid, block, 0, st, args);
      else hipLaunchKernelGGL((wc_gemv_kernel<0, 2, 32>), grid, block, 0, st, args);
    } else {
      switch ((m + 15) / 16) {
        case 1: hipLaunchKernelGGL((wc_gemv_kernel<0, 1, 16>), grid, block, 0, st, args); break;
        case 2: hipLaunchKernelGGL((wc_gemv_kernel<0, 2, 16>), grid, block, 0, st, args); break;
        case 3: hipLaunchKernelGGL((wc_gemv_kernel<0, 3, 16>), grid, block, 0, st, args); break;
        default: hipLaunchKernelGGL((wc_gemv_kernel<0, 4, 16>), grid, block, 0, st, args); break;
      }
    }
    if (hipGetLastError() != hipSuccess) return WC_EHIP;
  }
  return WC_OK;
}

// Packed-x slots of the jobs of a shared GEMM: jobs with the same x (pointer
// and length) share one slot.  Returns the workspace bytes; slot[i] is job i's
// byte offset in the workspace.
uint64_t packed_slots(const wc::BlobPriv& P, uint32_t n, const uint32_t* tensors,
                      const void* const* dev_x, uint32_t m, uint64_t* slot) {
  uint64_t total = 0;
  const uint64_t mpad = (m + 31) / 32 * 32;
  for (uint32_t i = 0; i < n; i++) {
    const uint64_t K = P.tensors[tensors[i]].cols;
    slot[i] = ~uint64_t(0);
    for (uint32_t j = 0; j < i; j++)
      if (dev_x[j] == dev_x[i] && P.tensors[tensors[j]].cols == K) slot[i] = slot[j];
    if (slot[i] == ~uint64_t(0)) {
      slot[i] = total;
      total += pad256(mpad * K * 2);
    }
  }
  return total;
}

}  // namespace

extern "C" wc_status wc_gemv(const wc_blob* desc, const void* dev_blob, uint32_t n,
                             const uint32_t* tensors, const void* const* dev_x, uint32_t m,
                             float* const* dev_y, void* stream, int32_t* dev_err) {
  if (m < 1 || m > 64) return WC_EINVAL;
  const wc_status rc = check_jobs(desc, dev_blob, n, tensors, dev_x, m, dev_y, false);
  if (rc != WC_OK) return rc;
  const wc::BlobPriv& P = static_cast<const wc::BlobHandle*>(desc->priv)->priv;
  uint64_t xs[kMaxLaunchTensors];
  for (uint32_t i = 0; i < n; i++) xs[i] = reinterpret_cast<uint64_t>(dev_x[i]);
  return launch_jobs(P, dev_blob, n, tensors, xs, m, dev_y, false,
                     reinterpret_cast<hipStream_t>(stream), dev_err);
}

extern "C" wc_status wc_gemm_i8(const wc_blob* desc, const void* dev_blob, uint32_t n,
                                const uint32_t* tensors, const void* const* dev_x, uint32_t m,
                                int32_t* const* dev_y, void* stream, int32_t* dev_err) {
  if (!desc || !desc->priv || !dev_blob || !tensors || !dev_x || !dev_y || n == 0 ||
      n > kMaxLaunchTensors || m < 1 || m > 64)
    return WC_EINVAL;
  const wc::BlobPriv& P = static_cast<const wc::BlobHandle*>(desc->priv)->priv;
  LaunchArgs args{};
  fill_common(args, P, dev_blob, dev_err);
  uint64_t tiles = 0;
  for (uint32_t i = 0; i < n; i++) {
    if (tensors[i] >= desc->n_tensors || !dev_x[i] || !dev_y[i] ||
        reinterpret_cast<uintptr_t>(dev_x[i]) % 16)
      return WC_EINVAL;
    const wc::TensorInfo& T = P.tensors[tensors[i]];
    if (T.dtype != WC_U8 || T.lanes != 64 || T.tile_order != WC_TILE_COLUMN_BLOCKS ||
        T.tile_r != 16)
      return WC_EUNSUPPORTED;
    // |x w| <= 2^14, so K <= 2^16 keeps every int32 sum below 2^30
    if (T.cols > 65536 || T.rows > 0xFFFFFFFFull) return WC_EUNSUPPORTED;
    tiles += T.n_chunks;
  }
  // one block of x rows: the 16-wave kernel when the tiles fit it
  const bool wide = m <= 16 && gemv_wide(0, tiles);
  const uint64_t per_wg = wide ? uint64_t(wc::kWideWaves) : uint64_t(kWaves);
  uint32_t wgs = 0;
  for (uint32_t i = 0; i < n; i++) {
    const wc::TensorInfo& T = P.tensors[tensors[i]];
    fill_tensor(args.t[i], T, dev_y[i], wgs);
    args.t[i].x = reinterpret_cast<uint64_t>(dev_x[i]);
    wgs += uint32_t((T.n_chunks + per_wg - 1) / per_wg);
  }
  args.n_tensors = n;
  args.m = m;
  const hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  if (wide) return wc::gemv_wide_launch(0, &args, sizeof args, wgs, st) ? WC_OK : WC_EHIP;
  const dim3 grid(wgs), block(kThreads);
  switch ((m + 15) / 16) {
    case 1: hipLaunchKernelGGL((wc_gemv_kernel<0, 1, 16, 4>), grid, block, 0, st, args); break;
    case 2: hipLaunchKernelGGL((wc_gemv_kernel<0, 2, 16, 4>), grid, block, 0, st, args); break;
    case 3: hipLaunchKernelGGL((wc_gemv_kernel<0, 3, 16, 4>), grid, block, 0, st, args); break;
    default: hipLaunchKernelGGL((wc_gemv_kernel<0, 4, 16, 4>), grid, block, 0, st, args); break;
  }
  return hipGetLastError() == hipSuccess ? WC_OK : WC_EHIP;
}

extern "C" wc_status wc_gemv_mx(const wc_blob* desc, const void* dev_blob, uint32_t n,
                                const uint32_t* tensors, const uint8_t* const* dev_scales,
                                const void* const* dev_x, uint32_t m, float* const* dev_y,
                                void* stream, int32_t* dev_err) {
  if (!desc || !desc->priv || !dev_blob || !tensors || !dev_scales || !dev_x || !dev_y || n == 0 ||
      n > kMaxLaunchTensors || m < 1 || m > 64)
    return WC_EINVAL;
  const wc::BlobPriv& P = static_cast<const wc::BlobHandle*>(desc->priv)->priv;
  for (uint32_t i = 0; i < n; i++) {
    if (tensors[i] >= desc->n_tensors || !dev_x[i] || !dev_y[i] || !dev_scales[i] ||
        reinterpret_cast<uintptr_t>(dev_x[i]) % 16)
      return WC_EINVAL;
    const wc::TensorInfo& T = P.tensors[tensors[i]];
    // e2m1 codes as nibble symbols, or their packed bytes as byte symbols (two
    // columns of x per symbol); a wave row of a 16-row tile is 4 lane-groups
    // (MX blocks) of each row: tiles of a multiple of 128 codes keep it whole
    const uint64_t per = T.dtype == WC_U8 ? 2 : 1;  // codes per symbol
    if ((T.dtype != WC_FP4_E2M1 && T.dtype != WC_U8) || T.lanes != 64 ||
        T.tile_order != WC_TILE_COLUMN_BLOCKS || T.tile_r != 16 || (T.tile_c * per) % 128)
      return WC_EUNSUPPORTED;
    const uint64_t K = T.cols * per;
    if (T.rows > 0xFFFFFFFFull || K > 0xFFFFFFFFull) return WC_EUNSUPPORTED;
    // x offsets of a lane reach 64 rows of 2 K bytes; scale offsets N * K / 32
    if (64ull * K * 2 > 0x7FFFFFFFull || T.rows * (K / 32) > 0xFFFFFFFFull)
      return WC_EUNSUPPORTED;
  }
  const hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  // one launch for the nibble-coded jobs, one for the byte-coded ones (the
  // latter on the 16-wave kernel when it has up to kWideQ4Rows rows of x and
  // its tiles fit it)
  for (int bytes = 0; bytes < 2; bytes++) {
    LaunchArgs args{};
    fill_common(args, P, dev_blob, dev_err);
    uint64_t tiles = 0;
    for (uint32_t i = 0; i < n; i++) {
      const wc::TensorInfo& T = P.tensors[tensors[i]];
      if ((T.dtype == WC_U8) == (bytes == 1)) tiles += T.n_chunks;
    }
    const bool wide = bytes && m <= kWideQ4Rows && tiles && gemv_wide(3, tiles);
    const uint64_t per_wg = wide ? uint64_t(wc::kWideWaves) : uint64_t(kWaves);
    uint32_t wgs = 0, nt = 0;
    for (uint32_t i = 0; i < n; i++) {
      const wc::TensorInfo& T = P.tensors[tensors[i]];
      if ((T.dtype == WC_U8) != (bytes == 1)) continue;
      fill_tensor(args.t[nt], T, dev_y[i], wgs);
      args.t[nt].x = reinterpret_cast<uint64_t>(dev_x[i]);
      args.t[nt].scales = reinterpret_cast<uint64_t>(dev_scales[i]);
      wgs += uint32_t((T.n_chunks + per_wg - 1) / per_wg);
      nt++;
    }
    if (!nt) continue;
    args.n_tensors = nt;
    args.m = m;
    if (wide) {
      if (!wc::gemv_wide_launch(3, &args, sizeof args, wgs, st)) return WC_EHIP;
      continue;
    }
    const dim3 grid(wgs), block(kThreads);
    if (bytes) {
      switch ((m + 15) / 16) {
        case 1: hipLaunchKernelGGL((wc_gemv_mxb_kernel<1>), grid, block, 0, st, args); break;
        case 2: hipLaunchKernelGGL((wc_gemv_mxb_kernel<2>), grid, block, 0, st, args); break;
        case 3: hipLaunchKernelGGL((wc_gemv_mxb_kernel<3>), grid, block, 0, st, args); break;
        default: hipLaunchKernelGGL((wc_gemv_mxb_kernel<4>), grid, block, 0, st, args); break;
      }
    } else {
      switch ((m + 15) / 16) {
        case 1: hipLaunchKernelGGL((wc_gemv_mx_kernel<1>), grid, block, 0, st, args); break;
        case 2: hipLaunchKernelGGL((wc_gemv_mx_kernel<2>), grid, block, 0, st, args); break;
        case 3: hipLaunchKernelGGL((wc_gemv_mx_kernel<3>), grid, block, 0, st, args); break;
        default: hipLaunchKernelGGL((wc_gemv_mx_kernel<4>), grid, block, 0, st, args); break;
      }
    }
    if (hipGetLastError() != hipSuccess) return WC_EHIP;
  }
  return WC_OK;
}

extern "C" wc_status wc_gemv_w4(const wc_blob* desc, const void* dev_blob, uint32_t n,
                                const uint32_t* tensors, const uint16_t* const* dev_scales,
                                const uint8_t* const* dev_zeros, const void* const* dev_x,
                                uint32_t m, float* const* dev_y, void* stream, int32_t* dev_err) {
  if (!desc || !desc->priv || !dev_blob || !tensors || !dev_scales || !dev_x || !dev_y || n == 0 ||
      n > kMaxLaunchTensors || m < 1 || m > 64)
    return WC_EINVAL;
  const wc::BlobPriv& P = static_cast<const wc::BlobHandle*>(desc->priv)->priv;
  for (uint32_t i = 0; i < n; i++) {
    if (tensors[i] >= desc->n_tensors || !dev_x[i] || !dev_y[i] || !dev_scales[i] ||
        reinterpret_cast<uintptr_t>(dev_x[i]) % 16 || reinterpret_cast<uintptr_t>(dev_scales[i]) % 2)
      return WC_EINVAL;
    const wc::TensorInfo& T = P.tensors[tensors[i]];
    // the codes as nibble symbols (WC_U4), or the packed bytes as byte symbols
    // (WC_U8); a wave row of a 16-row tile is 4 lane-groups of 32 codes of each
    // row: one 128-column group per row
    const uint64_t per = T.dtype == WC_U8 ? 2 : 1;  // codes per symbol
    if ((T.dtype != WC_U8 && T.dtype != WC_U4) || T.lanes != 64 ||
        T.tile_order != WC_TILE_COLUMN_BLOCKS || T.tile_r != 16 || (T.tile_c * per) % 128)
      return WC_EUNSUPPORTED;
    const uint64_t K = T.cols * per;
    if (T.rows > 0xFFFFFFFFull || K > 0xFFFFFFFFull) return WC_EUNSUPPORTED;
    // x offsets of a lane reach 64 rows of 2 K bytes; scale offsets 2 N K / 128
    if (64ull * K * 2 > 0x7FFFFFFFull || T.rows * (K / 128) * 2 > 0xFFFFFFFFull)
      return WC_EUNSUPPORTED;
  }
  const hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  // one launch for the byte-coded jobs (on the 16-wave kernel when it has up
  // to kWideQ4Rows rows of x and its tiles fit it), one for the nibble-coded
  // ones
  for (int nibbles = 0; nibbles < 2; nibbles++) {
    LaunchArgs args{};
    fill_common(args, P, dev_blob, dev_err);
    uint64_t tiles = 0;
    for (uint32_t i = 0; i < n; i++) {
      const wc::TensorInfo& T = P.tensors[tensors[i]];
      if ((T.dtype == WC_U4) == (nibbles == 1)) tiles += T.n_chunks;
    }
    const bool wide = !nibbles && m <= kWideQ4Rows && tiles && gemv_wide(4, tiles);
    const uint64_t per_wg = wide ? uint64_t(wc::kWideWaves) : uint64_t(kWaves);
    uint32_t wgs = 0, nt = 0;
    for (uint32_t i = 0; i < n; i++) {
      const wc::TensorInfo& T = P.tensors[tensors[i]];
      if ((T.dtype == WC_U4) != (nibbles == 1)) continue;
      fill_tensor(args.t[nt], T, dev_y[i], wgs);
      args.t[nt].x = reinterpret_cast<uint64_t>(dev_x[i]);
      args.t[nt].scales = reinterpret_cast<uint64_t>(dev_scales[i]);
      args.t[nt].zeros = dev_zeros ? reinterpret_cast<uint64_t>(dev_zeros[i]) : 0ull;
      wgs += uint32_t((T.n_chunks + per_wg - 1) / per_wg);
      nt++;
    }
    if (!nt) continue;
    args.n_tensors = nt;
    args.m = m;
    if (wide) {
      if (!wc::gemv_wide_launch(4, &args, sizeof args, wgs, st)) return WC_EHIP;
      continue;
    }
    const dim3 grid(wgs), block(kThreads);
    if (nibbles) {
      switch ((m + 15) / 16) {
        case 1: hipLaunchKernelGGL((wc_gemv_w4n_kernel<1>), grid, block, 0, st, args); break;
        case 2: hipLaunchKernelGGL((wc_gemv_w4n_kernel<2>), grid, block, 0, st, args); break;
        case 3: hipLaunchKernelGGL((wc_gemv_w4n_kernel<3>), grid, block, 0, st, args); break;
        default: hipLaunchKernelGGL((wc_gemv_w4n_kernel<4>), grid, block, 0, st, args); break;
      }
    } else {
      switch ((m + 15) / 16) {
        case 1: hipLaunchKernelGGL((wc_gemv_w4_kernel<1>), grid, block, 0, st, args); break;
        case 2: hipLaunchKernelGGL((wc_gemv_w4_kernel<2>), grid, block, 0, st, args); break;
        case 3: hipLaunchKernelGGL((wc_gemv_w4_kernel<3>), grid, block, 0, st, args); break;
        default: hipLaunchKernelGGL((wc_gemv_w4_kernel<4>), grid, block, 0, st, args); break;
      }
    }
    if (hipGetLastError() != hipSuccess) return WC_EHIP;
  }
  return WC_OK;
}

extern "C" wc_status wc_gemm_workspace_bytes(const wc_blob* desc, uint32_t n,
                                             const uint32_t* tensors, const void* const* dev_x,
                                             uint32_t m, uint64_t* bytes) {
  if (!bytes) return WC_EINVAL;
  *bytes = 0;
  if (!desc || !desc->priv || !tensors || !dev_x || n == 0 || n > kMaxLaunchTensors ||
      m < 1 || m > kMaxGemmRows)
    return WC_EINVAL;
  for (uint32_t i = 0; i < n; i++)
    if (tensors[i] >= desc->n_tensors) return WC_EINVAL;
  if (m <= kShareRows) return WC_OK;
  const wc::BlobPriv& P = static_cast<const wc::BlobHandle*>(desc->priv)->priv;
  uint64_t slot[kMaxLaunchTensors];
  *bytes = packed_slots(P, n, tensors, dev_x, m, slot);
  return WC_OK;
}

extern "C" wc_status wc_gemm(const wc_blob* desc, const void* dev_blob, uint32_t n,
                             const uint32_t* tensors, const void* const* dev_x, uint32_t m,
                             float* const* dev_y, void* dev_workspace, uint64_t workspace_bytes,
                             void* stream, int32_t* dev_err) {
  if (m < 1 || m > kMaxGemmRows) return WC_EINVAL;
  if (m <= kShareRows) return wc_gemv(desc, dev_blob, n, tensors, dev_x, m, dev_y, stream, dev_err);
  const wc_status rc = check_jobs(desc, dev_blob, n, tensors, dev_x, m, dev_y, true);
  if (rc != WC_OK) return rc;
  const wc::BlobPriv& P = static_cast<const wc::BlobHandle*>(desc->priv)->priv;
  uint64_t slot[kMaxLaunchTensors];
  const uint64_t need = packed_slots(P, n, tensors, dev_x, m, slot);
  if (!dev_workspace || reinterpret_cast<uintptr_t>(dev_workspace) % 256 ||
      workspace_bytes < need)
    return WC_EINVAL;
  const hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  uint64_t xs[kMaxLaunchTensors];
  const uint64_t mpad = (m + 31) / 32 * 32;
  for (uint32_t i = 0; i < n; i++) {
    const uint64_t K = P.tensors[tensors[i]].cols;
    xs[i] = reinterpret_cast<uint64_t>(dev_workspace) + slot[i];
    bool first = true;
    for (uint32_t j = 0; j < i; j++) first = first && slot[j] != slot[i];
    if (!first) continue;
    const uint64_t units = mpad * K / 8;  // 16-byte units
    const uint32_t blocks = uint32_t(std::min<uint64_t>((units + 255) / 256, 8192));
    hipLaunchKernelGGL(pack_x_kernel, dim3(blocks), dim3(256), 0, st,
                       static_cast<const uint16_t*>(dev_x[i]), m, uint32_t(K),
                       reinterpret_cast<u32x4*>(xs[i]), units);
    if (hipGetLastError() != hipSuccess) return WC_EHIP;
  }
  return launch_jobs(P, dev_blob, n, tensors, xs, m, dev_y, true, st, dev_err);
}
