// wc_gemm_wide.hip -- 16-wave-workgroup instances of the fused decode-GEMM
// (Alg. 1 / 3; the decoder is in wc_decoder.h) for int8 weights (wc_gemm_i8),
// fp8 e4m3 and e5m2 weights (wc_gemv) and MXFP4 and int4 codes coded as bytes
// (wc_gemv_mx, wc_gemv_w4) on 16-row tiles with up to 16 rows of x (bf16
// weights: wc_gemm_wide_bf16.hip).  One
// decode table serves 16 waves, so a compute unit holds 32 of these waves
// against 24 of the 8-wave kernels in wc_gemm.hip; the launches of those
// entry points whose tiles overflow the 8-wave kernel's resident waves but
// fit these run here, in one round.  A translation unit of its own, so that
// the 8-wave kernels' code does not change with it.

#include <string.h>

#include "wc_decoder.h"

namespace {

template <bool kFp8>
__global__ __launch_bounds__(wc::kWideWaves * 64) void wc_gemv_wide_kernel(LaunchArgs a) {
  __shared__ uint2 tab[wc::kTableSize];
  __shared__ uint32_t cum[260];
  __shared__ uint32_t ring[wc::kWideWaves][wc_ring_words() / 2];
  const uint32_t wg = blockIdx.x;
  uint32_t ti = 0;
  for (uint32_t k = 1; k < a.n_tensors; k++)
    if (wg >= a.t[k].wg0) ti = k;
  const DevTensor& T = a.t[ti];
  const uint32_t tid = threadIdx.x;
  const uint32_t wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const uint32_t lane = __lane_id();
  const uint32_t chunk = (wg - T.wg0) * wc::kWideWaves + wave;
  const IndexPre pre = load_index(a, T, chunk, 1u);
  build_table<wc::kWideWaves * 64>(a, T, tab, cum, tid);
  __syncthreads();
  if (chunk >= T.n_chunks) return;
  decode_chunks<4, 64, true, 0, 1, 16, false, kFp8 ? 1 : 0>(a, T, chunk, lane, tab, ring[wave],
                                                             pre);
}

// e5m2 weights: the exponent bits are coded and the rest travel raw, as for
// bf16 (the decoder's fp8 mode 2).
__global__ __launch_bounds__(wc::kWideWaves * 64) void wc_gemv_wide_e5m2_kernel(LaunchArgs a) {
  __shared__ uint2 tab[wc::kTableSize];
  __shared__ uint32_t cum[260];
  __shared__ uint32_t ring[wc::kWideWaves][wc_ring_words() / 2];
  const uint32_t wg = blockIdx.x;
  uint32_t ti = 0;
  for (uint32_t k = 1; k < a.n_tensors; k++)
    if (wg >= a.t[k].wg0) ti = k;
  const DevTensor& T = a.t[ti];
  const uint32_t tid = threadIdx.x;
  const uint32_t wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const uint32_t lane = __lane_id();
  const uint32_t chunk = (wg - T.wg0) * wc::kWideWaves + wave;
  const IndexPre pre = load_index(a, T, chunk, 1u);
  build_table<wc::kWideWaves * 64>(a, T, tab, cum, tid);
  __syncthreads();
  if (chunk >= T.n_chunks) return;
  decode_chunks<4, 64, true, 0, 1, 16, false, 2>(a, T, chunk, lane, tab, ring[wave], pre);
}

// 4-bit codes coded as bytes (the packed pairs): MXFP4 (kF8 = 3, e8m0 scale
// per 32 codes) or group-quantised int4 (kF8 = 4, scale and zero point per
// 128).  Their 8-wave kernels need 68-73 registers; held to 64 here, for 8
// waves per SIMD, the compiler keeps one or two values of the chunk's set-up
// in scratch across the decode loop (8-12 bytes per lane, stored before the
// loop and read after it).
template <int kF8>
__global__ __launch_bounds__(wc::kWideWaves * 64) __attribute__((amdgpu_waves_per_eu(8)))
void wc_gemv_wide_q4_kernel(LaunchArgs a) {
  __shared__ uint2 tab[wc::kTableSize];
  __shared__ uint32_t cum[260];
  __shared__ uint32_t ring[wc::kWideWaves][wc_ring_words() / 2];
  const uint32_t wg = blockIdx.x;
  uint32_t ti = 0;
  for (uint32_t k = 1; k < a.n_tensors; k++)
    if (wg >= a.t[k].wg0) ti = k;
  const DevTensor& T = a.t[ti];
  const uint32_t tid = threadIdx.x;
  const uint32_t wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const uint32_t lane = __lane_id();
  const uint32_t chunk = (wg - T.wg0) * wc::kWideWaves + wave;
  const IndexPre pre = load_index(a, T, chunk, 1u);
  build_table<wc::kWideWaves * 64>(a, T, tab, cum, tid);
  __syncthreads();
  if (chunk >= T.n_chunks) return;
  decode_chunks<4, 64, true, 0, 1, 16, false, kF8>(a, T, chunk, lane, tab, ring[wave], pre);
}

// kind: 0 int8, 1 fp8 e4m3, 2 fp8 e5m2, 3 MXFP4 as bytes, 4 int4 as bytes
// (5, bf16, is in wc_gemm_wide_bf16.hip)
const void* wide_kernel(int kind) {
  if (kind == 4) return reinterpret_cast<const void*>(wc_gemv_wide_q4_kernel<4>);
  if (kind == 3) return reinterpret_cast<const void*>(wc_gemv_wide_q4_kernel<3>);
  if (kind == 2) return reinterpret_cast<const void*>(wc_gemv_wide_e5m2_kernel);
  return kind == 1 ? reinterpret_cast<const void*>(wc_gemv_wide_kernel<true>)
                   : reinterpret_cast<const void*>(wc_gemv_wide_kernel<false>);
}

}  // namespace

namespace wc {

uint64_t gemv_wide_resident_waves(int kind) {
  if (kind == 5) return gemv_wide_bf16_resident_waves();
  int dev = 0, cus = 0, per_cu = 0;
  if (kind < 0 || kind > 4 || hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, wide_kernel(kind), kWideWaves * 64,
                                                   0) != hipSuccess)
    return 0;
  return uint64_t(cus) * uint64_t(per_cu) * uint64_t(kWideWaves);
}

bool gemv_wide_launch(int kind, const void* launch_args, uint64_t bytes, uint32_t workgroups,
                      void* stream) {
  if (kind == 5) return gemv_wide_bf16_launch(launch_args, bytes, workgroups, stream);
  if (bytes != sizeof(LaunchArgs) || kind < 0 || kind > 4) return false;
  LaunchArgs args;
  memcpy(&args, launch_args, sizeof args);
  const hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const dim3 grid(workgroups), block(kWideWaves * 64);
  if (kind == 4)
    hipLaunchKernelGGL((wc_gemv_wide_q4_kernel<4>), grid, block, 0, st, args);
  else if (kind == 3)
    hipLaunchKernelGGL((wc_gemv_wide_q4_kernel<3>), grid, block, 0, st, args);
  else if (kind == 2)
    hipLaunchKernelGGL(wc_gemv_wide_e5m2_kernel, grid, block, 0, st, args);
  else if (kind == 1)
    hipLaunchKernelGGL((wc_gemv_wide_kernel<true>), grid, block, 0, st, args);
  else
    hipLaunchKernelGGL((wc_gemv_wide_kernel<false>), grid, block, 0, st, args);
  return hipGetLastError() == hipSuccess;
}

}  // namespace wc
