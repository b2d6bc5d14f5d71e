// Partitioned search (the approximate search of DReSD Section 3.5 read as an
// inverted file): turn each query's probe list into the segments its scan
// walks.  One workgroup per query, one thread per probe: ids outside [0, P)
// and repeats of an earlier probe get an empty segment; a workgroup prefix
// sum of the partitions' tile counts gives the segment offsets.  Keys grouped
// by their value's first token (the next-token filter of Section 3.5 as a
// partition) probe instead the one partition of the query's next token,
// found among the sorted tokens by the workgroup.
#include "dresd_device.h"
#include "dresd_ops.h"

namespace dresd {

namespace {

constexpr int kSegThreads = 1024;

__global__ void __launch_bounds__(kSegThreads) dresd_segments(SegParams p) {
  __shared__ int32_t pid[kSegThreads];
  __shared__ int32_t wsum[kSegThreads / kWaveSize];
  __shared__ int32_t found;
  __shared__ int64_t own;
  const int b = blockIdx.x;
  const int i = threadIdx.x, lane = i & 63, wid = i >> 6;
  int32_t id = -1;
  if (p.tok) {
    // Thread i owns the sorted tokens [lo, hi); the tokens are distinct, so
    // at most one thread's range [tok[lo], tok[hi - 1]] can hold t.  That
    // thread names its range, and the workgroup reads the range together.
    const int32_t t = p.next_tok[b];
    const int64_t chunk = ((int64_t)p.P + kSegThreads - 1) / kSegThreads;
    const int64_t lo = (int64_t)i * chunk;
    const int64_t hi = lo + chunk < (int64_t)p.P ? lo + chunk : (int64_t)p.P;
    if (i == 0) {
      found = -1;
      own = -1;
    }
    __syncthreads();
    if (lo < hi && p.tok[lo] <= t && t <= p.tok[hi - 1]) own = lo;
    __syncthreads();
    const int64_t o = own;
    if (o >= 0) {
      const int64_t oe = o + chunk < (int64_t)p.P ? o + chunk : (int64_t)p.P;
      for (int64_t j = o + i; j < oe; j += kSegThreads)
        if (p.tok[j] == t) found = (int32_t)j;
    }
    __syncthreads();
    if (i == 0) id = found;  // S == 1
  } else if (i < p.S) {
    const size_t o = (size_t)b * p.S + i;
    const int64_t v = p.probes64 ? p.probes64[o] : (int64_t)p.probes32[o];
    id = (v >= 0 && v < p.P) ? (int32_t)v : -1;
  }
  pid[i] = id;
  __syncthreads();
  if (id >= 0)
    for (int j = 0; j < i; ++j)
      if (pid[j] == id) {
        id = -1;
        break;
      }
  int32_t start = 0, len = 0;
  if (id >= 0) {
    start = p.part_tile[id];
    len = p.part_tile[id + 1] - start;
  }
  // inclusive prefix sum of len over the workgroup
  int32_t x = len;
#pragma unroll
  for (int off = 1; off < kWaveSize; off <<= 1) {
    const int32_t y = __shfl_up(x, off, kWaveSize);
    if (lane >= off) x += y;
  }
  if (lane == kWaveSize - 1) wsum[wid] = x;
  __syncthreads();
  for (int w = 0; w < wid; ++w) x += wsum[w];
  if (i < p.S) {
    p.seg_off[(size_t)b * (p.S + 1) + i + 1] = x;
    p.seg_tile[(size_t)b * p.S + i] = start;
  }
  if (i == 0) p.seg_off[(size_t)b * (p.S + 1)] = 0;
}

// First token of each slot's value in the partitioned layout (0 for
// padding): ftok[s] = cont[slot_row[s]][0].
__global__ void __launch_bounds__(256) dresd_slot_first_tokens(const uint32_t *slot_row,
                                                               const int32_t *cont, int L,
                                                               int64_t nslot, int32_t *ftok) {
  for (int64_t s = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; s < nslot;
       s += (int64_t)gridDim.x * blockDim.x) {
    const uint32_t r = slot_row[s];
    ftok[s] = r == kPadRow ? 0 : cont[(int64_t)r * L];
  }
}

// First token of each row's value: out[i] = cont[i][0].
__global__ void __launch_bounds__(256) dresd_first_tokens(const int32_t *cont, int L, int64_t n,
                                                          int32_t *out) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    out[i] = cont[i * L];
}

}  // namespace

hipError_t launch_first_tokens(const int32_t *cont, int L, int64_t n, int32_t *out,
                               hipStream_t st) {
  const int64_t want = (n + 255) / 256;
  const unsigned blocks = (unsigned)(want < 65536 ? (want > 0 ? want : 1) : 65536);
  hipLaunchKernelGGL(dresd_first_tokens, dim3(blocks), dim3(256), 0, st, cont, L, n, out);
  return hipGetLastError();
}

hipError_t launch_slot_first_tokens(const uint32_t *slot_row, const int32_t *cont, int L,
                                    int64_t nslot, int32_t *ftok, hipStream_t st) {
  const int64_t want = (nslot + 255) / 256;
  const unsigned blocks = (unsigned)(want < 65536 ? (want > 0 ? want : 1) : 65536);
  hipLaunchKernelGGL(dresd_slot_first_tokens, dim3(blocks), dim3(256), 0, st, slot_row, cont, L,
                     nslot, ftok);
  return hipGetLastError();
}

hipError_t launch_segments(const SegParams &p, hipStream_t st) {
  if (p.B == 0) return hipSuccess;
  SegParams q = p;
  void *args[] = {&q};
  return hipLaunchKernel((const void *)dresd_segments, dim3((unsigned)p.B), dim3(kSegThreads), args,
                         0, st);
}

}  // namespace dresd
