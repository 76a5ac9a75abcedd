// wc_stream.hip -- wc_stream: a plain HBM streaming kernel that does no
// decoding.  It moves a decode's byte mix (every compressed byte read once,
// every decoded byte written once, non-temporal) so that a decode launch can
// be set against the rate the memory system gives the same traffic on the
// same device.  It is a measuring aid, not a step of the codec.
//
// Write unit j (16 bytes) of dst receives read unit r(j) = (j * q) >> 32 of
// src, q = floor(n_src * 2^32 / n_dst): r climbs by 0 or 1 from one unit to
// the next, so the reads sweep src once, in order, spread evenly over the
// writes, as the decode interleaves word and raw-byte loads with its stores.
// The grid strides over dst; each thread keeps kUnroll units in flight.
#include <hip/hip_runtime.h>

#include "../../include/wc.h"

namespace {

constexpr int kStreamThreads = 256;
constexpr int kUnroll = 4;
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// j < 2^32 and q <= 2^32, so j * q fits in 64 bits
__device__ __forceinline__ uint64_t read_unit(uint64_t j, uint64_t q) { return (j * q) >> 32; }

__global__ __launch_bounds__(kStreamThreads) void wc_stream_kernel(
    const u32x4* __restrict__ src, uint64_t n_src, u32x4* __restrict__ dst, uint64_t n_dst,
    uint64_t q) {
  const uint64_t stride = uint64_t(gridDim.x) * kStreamThreads;
  uint64_t j = uint64_t(blockIdx.x) * kStreamThreads + threadIdx.x;
  if (n_dst == 0) {
    // read only: fold everything read into one value that is stored only if
    // it equals a fixed pattern, so the loads cannot be dropped
    u32x4 acc = {0u, 0u, 0u, 0u};
    for (; j + (kUnroll - 1) * stride < n_src; j += kUnroll * stride) {
      u32x4 v[kUnroll];
#pragma unroll
      for (int k = 0; k < kUnroll; k++) v[k] = src[j + k * stride];
#pragma unroll
      for (int k = 0; k < kUnroll; k++) acc ^= v[k];
    }
    for (; j < n_src; j += stride) acc ^= src[j];
    if (acc.x == 0x9E3779B9u && acc.y == 0x7F4A7C15u && acc.z == 0xF39CC060u &&
        acc.w == 0x5CEDC834u)
      dst[0] = acc;
    return;
  }
  for (; j + (kUnroll - 1) * stride < n_dst; j += kUnroll * stride) {
    u32x4 v[kUnroll];
#pragma unroll
    for (int k = 0; k < kUnroll; k++) v[k] = src[read_unit(j + k * stride, q)];
#pragma unroll
    for (int k = 0; k < kUnroll; k++) __builtin_nontemporal_store(v[k], &dst[j + k * stride]);
  }
  for (; j < n_dst; j += stride) __builtin_nontemporal_store(src[read_unit(j, q)], &dst[j]);
}

}  // namespace

extern "C" wc_status wc_stream(const void* dev_src, uint64_t src_bytes, void* dev_dst,
                               uint64_t dst_bytes, uint32_t blocks, void* stream,
                               uint64_t* read_bytes) {
  if (!dev_src || !dev_dst || src_bytes == 0 || src_bytes % 16 || dst_bytes % 16) return WC_EINVAL;
  if ((reinterpret_cast<uintptr_t>(dev_src) | reinterpret_cast<uintptr_t>(dev_dst)) & 15)
    return WC_EINVAL;
  const uint64_t n_src = src_bytes / 16, n_dst = dst_bytes / 16;
  if (n_dst && (n_src > n_dst || n_dst >= (1ull << 32))) return WC_EINVAL;
  // q = floor(n_src * 2^32 / n_dst) <= 2^32; r(j) = (j * q) >> 32 < n_src
  uint64_t q = 0, reads = n_src;
  if (n_dst) {
    q = (uint64_t)(((unsigned __int128)n_src << 32) / n_dst);
    reads = (uint64_t)((((unsigned __int128)(n_dst - 1)) * q) >> 32) + 1;
  }
  if (blocks == 0) {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      return WC_EHIP;
    blocks = (uint32_t)cus * 16u;
  }
  hipLaunchKernelGGL(wc_stream_kernel, dim3(blocks), dim3(kStreamThreads), 0,
                     reinterpret_cast<hipStream_t>(stream), static_cast<const u32x4*>(dev_src),
                     n_src, static_cast<u32x4*>(dev_dst), n_dst, q);
  if (hipGetLastError() != hipSuccess) return WC_EHIP;
  if (read_bytes) *read_bytes = 16 * reads;
  return WC_OK;
}
