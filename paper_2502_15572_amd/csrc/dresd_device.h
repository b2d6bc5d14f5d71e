// Device helpers shared by the gfx950 scan and merge kernels.
//
// Ranking keys are 64-bit: high half = order-preserving bits of the fp32
// score, low half = ~row.  Larger key = better; equal scores rank the lower
// row first.  Keys are unique, so every selection over them is deterministic.
#pragma once
#include "dresd_internal.h"

namespace dresd {

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef __bf16 b8 __attribute__((ext_vector_type(8)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t order_bits(float f) {
  uint32_t u = (f == 0.0f) ? 0u : __float_as_uint(f);  // -0 ranks as +0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float order_value(uint32_t h) {
  uint32_t u = (h & 0x80000000u) ? (h & 0x7fffffffu) : ~h;
  return __uint_as_float(u);
}

__device__ __forceinline__ uint64_t make_key(float s, uint32_t row) {
  return ((uint64_t)order_bits(s) << 32) | (uint64_t)(uint32_t)(~row);
}

// The value of lane 0, so the compiler keeps it in scalar registers.
__device__ __forceinline__ int64_t wave_uniform(int64_t x) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)x);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)x >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

__device__ __forceinline__ void wave_sync_lds() {
  // Orders this wave's LDS accesses across lanes (DS ops of one wave run in
  // order; this keeps the compiler from moving them across the point).
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

// Asynchronous copies global -> LDS (global_load_lds_*), issued from inline
// assembly so that the compiler's wait-count model, which cannot tell which
// LDS bytes such a copy writes, adds no waits for them before unrelated LDS
// reads.  Callers wait with wait_vmcnt before reading the destination.
__device__ __forceinline__ void copy1_to_lds(const void *src, uint32_t lds) {
  // one dword per lane from its own address; lane l lands at lds + 4 l
  asm volatile(
      "s_mov_b32 m0, %1\n\t"
      "global_load_lds_dword %0, off"
      :
      : "v"(src), "s"(lds)
      : "memory");
}

// s_waitcnt immediate that waits for vmcnt == 0 only (gfx9 encoding: vmcnt
// bits [3:0] and [15:14], expcnt [6:4] and lgkmcnt [11:8] at their maxima).
constexpr int kWaitVmcnt0 = 0x0F70;

// Wait until at most N of this wave's vector memory operations are pending
// (they complete in issue order).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" : : "n"(N) : "memory");
}

// Sort n (power of two, >= 2) keys in LDS, descending, by one wave.
__device__ inline void wave_bitonic_desc(uint64_t *s, int n, int lane) {
  for (int size = 2; size <= n; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int p = lane; p < (n >> 1); p += kWaveSize) {
        int lo = ((p & ~(stride - 1)) << 1) | (p & (stride - 1));
        int hi = lo + stride;
        uint64_t a = s[lo], b = s[hi];
        bool desc = (lo & size) == 0;
        if ((a < b) == desc) {
          s[lo] = b;
          s[hi] = a;
        }
      }
      wave_sync_lds();
    }
  }
}

// Sets of keys up to this size are ordered by wave_rank_top.
constexpr int kWaveRankMax = 256;

// The keys of rank 0 and keep - 1 of an ordering (0 when absent).
struct RankEnds {
  uint64_t first, last;
};

// Ranks of the n distinct keys src[0..n) (LDS), E per lane: key
// lane + 64 e is x[e], its rank (number of greater keys) r[e].  Every key
// read serves all E of the lane's keys.
template <int E>
__device__ inline void wave_ranks(const uint64_t *src, int n, int lane, uint64_t (&x)[4],
                                  int (&r)[4]) {
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int i = lane + e * kWaveSize;
    x[e] = i < n ? src[i] : ~0ull;  // ~0: counts nothing and is never stored
    r[e] = 0;
  }
  const int n2 = n & ~1;
#pragma unroll 2
  for (int j = 0; j < n2; j += 2) {
    const uint64_t a = src[j], b = src[j + 1];
#pragma unroll
    for (int e = 0; e < E; ++e) r[e] += (int)(a > x[e]) + (int)(b > x[e]);
  }
  if (n & 1) {
    const uint64_t a = src[n - 1];
#pragma unroll
    for (int e = 0; e < E; ++e) r[e] += (int)(a > x[e]);
  }
}

// Top `keep` of n <= kWaveRankMax distinct keys src[0..n) (LDS; every key
// names its own row) in descending order, by one wave: the key of rank
// r < keep goes to dst[r] (LDS or global memory, not src).  Every lane
// returns the keys of rank 0 and keep - 1.
__device__ inline RankEnds wave_rank_top(const uint64_t *src, int n, uint64_t *dst, int keep,
                                         int lane) {
  uint64_t x[4] = {0ull, 0ull, 0ull, 0ull};
  int r[4] = {0, 0, 0, 0};
  const int E = (n + kWaveSize - 1) / kWaveSize;
  if (E <= 1) wave_ranks<1>(src, n, lane, x, r);
  else if (E == 2) wave_ranks<2>(src, n, lane, x, r);
  else if (E == 3) wave_ranks<3>(src, n, lane, x, r);
  else wave_ranks<4>(src, n, lane, x, r);
  uint64_t f = 0ull, l = 0ull;
  bool hf = false, hl = false;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    if (e >= E || lane + e * kWaveSize >= n) continue;
    if (r[e] < keep) dst[r[e]] = x[e];
    if (r[e] == 0) {
      f = x[e];
      hf = true;
    }
    if (r[e] == keep - 1) {
      l = x[e];
      hl = true;
    }
  }
  const uint64_t mf = __ballot(hf), ml = __ballot(hl);
  RankEnds ends;
  ends.first = mf ? __shfl(f, __ffsll((long long)mf) - 1, kWaveSize) : 0ull;
  ends.last = ml ? __shfl(l, __ffsll((long long)ml) - 1, kWaveSize) : 0ull;
  return ends;
}

// Same, by a whole workgroup.
__device__ inline void block_bitonic_desc(uint64_t *s, int n) {
  for (int size = 2; size <= n; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int p = threadIdx.x; p < (n >> 1); p += blockDim.x) {
        int lo = ((p & ~(stride - 1)) << 1) | (p & (stride - 1));
        int hi = lo + stride;
        uint64_t a = s[lo], b = s[hi];
        bool desc = (lo & size) == 0;
        if ((a < b) == desc) {
          s[lo] = b;
          s[hi] = a;
        }
      }
      __syncthreads();
    }
  }
}

}  // namespace dresd
