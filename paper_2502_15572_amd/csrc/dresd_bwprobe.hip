// Achievable HBM read bandwidth with the scans' access pattern: each wave
// streams one contiguous range of 1 KiB blocks (one 16-byte nontemporal load
// per lane per block, U blocks in flight), so the figure it reports is the
// ceiling a key stream of this layout can reach on the device.
#include "dresd_device.h"

namespace dresd {

// Never written in practice: the loads need a use the compiler cannot drop
// (a device variable with external linkage, which the host could read).
__device__ uint32_t g_probe_sink;

namespace {

template <int U>
__global__ void __launch_bounds__(256) dresd_bw_read(const u4 *__restrict__ p, int64_t nblocks) {
  const int lane = threadIdx.x & 63;
  const int64_t gw = blockIdx.x * (int64_t)(blockDim.x >> 6) + (threadIdx.x >> 6);
  const int64_t G = (int64_t)gridDim.x * (blockDim.x >> 6);
  const int64_t b0 = nblocks * gw / G, b1 = nblocks * (gw + 1) / G;
  const u4 *q = p + lane;
  uint32_t acc = 0;
  int64_t j = b0;
  for (; j + U <= b1; j += U) {
    u4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = __builtin_nontemporal_load(q + (j + u) * 64);
#pragma unroll
    for (int u = 0; u < U; ++u) acc ^= v[u][0] ^ v[u][1] ^ v[u][2] ^ v[u][3];
  }
  for (; j < b1; ++j) {
    const u4 v = __builtin_nontemporal_load(q + j * 64);
    acc ^= v[0] ^ v[1] ^ v[2] ^ v[3];
  }
  if (acc == 0x9e3779b9u && lane == 0) g_probe_sink = acc;
}

}  // namespace

hipError_t launch_bw_read(const void *buf, int64_t nblocks, int workgroups, hipStream_t st) {
  hipLaunchKernelGGL(dresd_bw_read<16>, dim3((unsigned)workgroups), dim3(256), 0, st,
                     static_cast<const u4 *>(buf), nblocks);
  return hipGetLastError();
}

}  // namespace dresd
