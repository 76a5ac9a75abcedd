// wc_decode.hip -- wc_decode: one launch decodes every chunk of a blob's
// tensors into the caller's buffers (Alg. 2; the decoder is in wc_decoder.h).
// The general kernel is here; bf16/fp16 launches that just overflow its
// resident waves run on the 16-wave kernel of wc_decode_wide.hip.

#include <mutex>
#include <utility>
#include <vector>

#include "wc_decoder.h"

namespace {

__global__ __launch_bounds__(kThreads) void wc_decode_kernel(LaunchArgs a) {
  __shared__ uint2 tab[wc::kTableSize];
  __shared__ uint32_t cum[260];
  __shared__ uint32_t ring[kWaves][wc_ring_words() / 2];

  const uint32_t wg = xcd_order(blockIdx.x, gridDim.x);
  uint32_t ti = 0;
  for (uint32_t k = 1; k < a.n_tensors; k++)
    if (wg >= a.t[k].wg0) ti = k;
  const DevTensor& T = a.t[ti];
  const uint32_t tid = threadIdx.x;
  // the wave index is uniform across the wave; say so, so chunk metadata and
  // buffer descriptors live in scalar registers
  const uint32_t wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const uint32_t lane = __lane_id();
  const uint32_t per_wave = T.lanes == 32 ? 2u : 1u;
  const uint32_t chunk0 = ((wg - T.wg0) * kWaves + wave) * per_wave;
  const IndexPre pre = load_index(a, T, chunk0, per_wave);
  build_table(a, T, tab, cum, tid);
  __syncthreads();
  if (chunk0 >= T.n_chunks) return;
  // instantiate one decoder per (format, lanes, tiling)
  auto run = [&](auto gc, auto lc) {
    constexpr int G = decltype(gc)::value, L = decltype(lc)::value;
    if (T.tiled)
      decode_chunks<G, L, true>(a, T, chunk0, lane, tab, ring[wave], pre);
    else
      decode_chunks<G, L, false>(a, T, chunk0, lane, tab, ring[wave], pre);
  };
  auto by_kind = [&](auto lc) {
    switch (T.kind) {
      case kSplit16: run(std::integral_constant<int, 2>{}, lc); break;
      case kByte: run(std::integral_constant<int, 4>{}, lc); break;
      default: run(std::integral_constant<int, 8>{}, lc); break;
    }
  };
  if (T.lanes == 32)
    by_kind(std::integral_constant<int, 32>{});
  else
    by_kind(std::integral_constant<int, 64>{});
}

// Waves of the general kernel and of the 16-bit wide kernel resident on the
// current device at once, from the runtime's occupancy calculation, worked
// out once per device ({0, 0} when unknown: the general kernel is used).
struct Capacity {
  uint64_t general, wide;
};

Capacity capacity() {
  static std::mutex mu;
  static std::vector<std::pair<int, Capacity>> known;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return Capacity{0, 0};
  std::lock_guard<std::mutex> lock(mu);
  for (const auto& k : known)
    if (k.first == dev) return k.second;
  Capacity c{0, 0};
  int cus = 0, per_cu = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
      hipOccupancyMaxActiveBlocksPerMultiprocessor(
          &per_cu, reinterpret_cast<const void*>(wc_decode_kernel), kThreads, 0) == hipSuccess)
    c = Capacity{uint64_t(cus) * uint64_t(per_cu) * uint64_t(kWaves), wc::wide_resident_waves()};
  known.push_back({dev, c});
  return c;
}

// A tiled tensor whose widest output descriptor (two tiles of a 32-lane wave)
// would not fit the 32-bit range the buffer descriptors address.
bool tile_span_ok(const wc::TensorInfo& T) {
  if (!T.tile_r) return true;
  const uint64_t pitch = T.cols * 16 / T.group;
  return (2 * uint64_t(T.tile_r) + 1) * pitch < (1ull << 31);
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
    if (T.lanes != 64 && T.lanes != 32) return WC_EUNSUPPORTED;
    if (!tile_span_ok(T)) return WC_EUNSUPPORTED;
    if (!dev_dst[t]) return WC_EINVAL;
  }
  LaunchArgs args{};
  fill_common(args, P, dev_blob, dev_err);
  uint32_t t = 0;
  while (t < n) {
    // the tensors of one launch: the next kMaxLaunchTensors that have chunks
    uint32_t end = t, nt = 0;
    uint64_t chunks = 0;
    bool wide_fits = true;
    for (; end < n && nt < kMaxLaunchTensors; end++) {
      const wc::TensorInfo& T = P.tensors[end];
      if (T.n_chunks == 0) continue;
      nt++;
      chunks += T.n_chunks;
      wide_fits = wide_fits && wc::has_raw(T.dtype) &&
                  T.lanes == 64 && !T.tile_r;
    }
    if (nt == 0) break;
    bool wide = false;
    if (wide_fits) {
      const Capacity cap = capacity();
      wide = cap.general && cap.wide > cap.general && chunks > cap.general && chunks <= cap.wide;
    }
    const uint64_t waves = wide ? uint64_t(wc::kWideWaves) : uint64_t(kWaves);
    uint32_t wgs = 0;
    nt = 0;
    for (; t < end; t++) {
      const wc::TensorInfo& T = P.tensors[t];
      if (T.n_chunks == 0) continue;
      fill_tensor(args.t[nt++], T, dev_dst[t], wgs);
      const uint64_t per_group = waves * (T.lanes == 32 ? 2u : 1u);
      wgs += (uint32_t)((T.n_chunks + per_group - 1) / per_group);
    }
    args.n_tensors = nt;
    if (wide) {
      if (!wc::wide_launch(&args, sizeof args, wgs, stream)) return WC_EHIP;
    } else {
      hipLaunchKernelGGL(wc_decode_kernel, dim3(wgs), dim3(kThreads), 0,
                         reinterpret_cast<hipStream_t>(stream), args);
      if (hipGetLastError() != hipSuccess) return WC_EHIP;
    }
  }
  return WC_OK;
}
