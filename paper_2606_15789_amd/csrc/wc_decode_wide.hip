// wc_decode_wide.hip -- wc_decode's second kernel: bf16 / fp16 tensors in
// untiled 64-lane chunks, with 16 waves to a workgroup (Alg. 2; the decoder is
// in wc_decoder.h).  It sits in a translation unit of its own so that the
// compilation of the general kernel in wc_decode.hip stays as it is.

#include <string.h>

#include "wc_decoder.h"

namespace {

// That path alone needs few registers, and one decode table serves twice the
// waves, so a compute unit holds 32 of these waves against 24 of the general
// kernel.  wc_decode takes it for a launch whose chunks overflow the resident
// waves of the general kernel but fit in these: the launch then runs in one
// round instead of a full one and a short second.
__global__ __launch_bounds__(wc::kWideWaves * 64) void wc_decode_wide_kernel(LaunchArgs a) {
  __shared__ uint2 tab[wc::kTableSize];
  __shared__ uint32_t cum[260];
  __shared__ uint32_t ring[wc::kWideWaves][wc_ring_words() / 2];

  const uint32_t wg = xcd_order(blockIdx.x, gridDim.x);
  uint32_t ti = 0;
  for (uint32_t k = 1; k < a.n_tensors; k++)
    if (wg >= a.t[k].wg0) ti = k;
  const DevTensor& T = a.t[ti];
  const uint32_t tid = threadIdx.x;
  const uint32_t wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const uint32_t lane = __lane_id();
  const uint32_t chunk0 = (wg - T.wg0) * wc::kWideWaves + wave;
  const IndexPre pre = load_index(a, T, chunk0, 1u);
  build_table<wc::kWideWaves * 64>(a, T, tab, cum, tid);
  __syncthreads();
  if (chunk0 >= T.n_chunks) return;
  decode_chunks<2, 64, false>(a, T, chunk0, lane, tab, ring[wave], pre);
}

}  // namespace

namespace wc {

uint64_t wide_resident_waves() {
  int dev = 0, cus = 0, per_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(
          &per_cu, reinterpret_cast<const void*>(wc_decode_wide_kernel), kWideWaves * 64, 0) !=
          hipSuccess)
    return 0;
  return uint64_t(cus) * uint64_t(per_cu) * uint64_t(kWideWaves);
}

bool wide_launch(const void* launch_args, uint64_t bytes, uint32_t workgroups, void* stream) {
  if (bytes != sizeof(LaunchArgs)) return false;
  LaunchArgs args;
  memcpy(&args, launch_args, sizeof args);
  hipLaunchKernelGGL(wc_decode_wide_kernel, dim3(workgroups), dim3(kWideWaves * 64), 0,
                     reinterpret_cast<hipStream_t>(stream), args);
  return hipGetLastError() == hipSuccess;
}

}  // namespace wc
