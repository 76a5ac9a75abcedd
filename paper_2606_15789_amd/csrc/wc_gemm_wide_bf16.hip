// wc_gemm_wide_bf16.hip -- the 16-wave-workgroup instance of the fused
// decode-GEMM (Alg. 1 / 3; the decoder is in wc_decoder.h) for bf16 weights on
// 16-row tiles with up to 16 rows of x (wc_gemv, wc_gemm).  As in
// wc_gemm_wide.hip, one decode table serves 16 waves, so a compute unit holds
// 32 of these waves against 24 of the 8-wave kernel; a launch whose tiles
// overflow the 8-wave kernel's resident waves but fit these runs here, in one
// round.  A translation unit of its own, so that the other kernels' code does
// not change with it.

#include <string.h>

#include "wc_decoder.h"

namespace {

// bf16 weights: the exponent byte coded, the sign and mantissa byte raw.
__global__ __launch_bounds__(wc::kWideWaves * 64) void wc_gemv_wide_bf16_kernel(LaunchArgs a) {
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
  decode_chunks<2, 64, true, 0, 1, 16, false, 0>(a, T, chunk, lane, tab, ring[wave], pre);
}

}  // namespace

namespace wc {

uint64_t gemv_wide_bf16_resident_waves() {
  int dev = 0, cus = 0, per_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(
          &per_cu, reinterpret_cast<const void*>(wc_gemv_wide_bf16_kernel), kWideWaves * 64,
          0) != hipSuccess)
    return 0;
  return uint64_t(cus) * uint64_t(per_cu) * uint64_t(kWideWaves);
}

bool gemv_wide_bf16_launch(const void* launch_args, uint64_t bytes, uint32_t workgroups,
                           void* stream) {
  if (bytes != sizeof(LaunchArgs)) return false;
  LaunchArgs args;
  memcpy(&args, launch_args, sizeof args);
  hipLaunchKernelGGL(wc_gemv_wide_bf16_kernel, dim3(workgroups), dim3(kWideWaves * 64), 0,
                     reinterpret_cast<hipStream_t>(stream), args);
  return hipGetLastError() == hipSuccess;
}

}  // namespace wc
