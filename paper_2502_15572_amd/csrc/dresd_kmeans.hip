// gfx950 kernels of spherical k-means, the partitioning behind the
// partitioned search (the paper's approximate search, Section 3.5, read as an
// inverted file; cosine similarity of unit vectors, Eq. 3, is the inner
// product).
//
//   assign : every row goes to the centroid with the largest inner product,
//            ties to the lower centroid id.  An LDS-tiled fp32 contraction on
//            the fp32 matrix cores (v_mfma_f32_16x16x4_f32): a workgroup owns
//            64 rows (decoded from their storage type, staged once when they
//            have at most 128 dims) and walks all centroids in tiles of 64 x
//            128 dims, loading the next tile while it multiplies this one; the
//            argmax is fused into the epilogue of each centroid tile.
//   update : each centroid becomes the unit vector along the sum of its
//            rows (unchanged when it has none).  Rows are added into 64-bit
//            fixed point (2^-30 units) with integer atomics, so the sums, and
//            the centroids, do not depend on the order of the additions.
//   init   : the starting centroids, P distinct rows taken at even spacing
//            through the row order from a seeded offset, each scaled to unit
//            length.
#include "dresd_device.h"
#include "dresd_ops.h"

namespace dresd {

namespace {

constexpr int kKR = 64;    // rows per workgroup
constexpr int kKC = 64;    // centroids per tile
constexpr int kKK = 128;   // dims staged per step
constexpr double kFixScale = 1073741824.0;  // 2^30

template <int DT>
__device__ __forceinline__ float load_elem(const void *x, int64_t off) {
  if constexpr (DT == kF32) {
    return static_cast<const float *>(x)[off];
  } else if constexpr (DT == kF16) {
    return (float)static_cast<const _Float16 *>(x)[off];
  } else {
    const uint32_t b = static_cast<const uint16_t *>(x)[off];
    return __uint_as_float(b << 16);
  }
}

// (score, id) order of the argmax: larger score, then lower id.
__device__ __forceinline__ bool beats(float s, int id, float bs, int bid) {
  return s > bs || (s == bs && id < bid);
}

// Rows [r0, r0 + 64) x dims [k0, k0 + 128) of x, decoded to fp32, into xs
// (zero past n and d): thread t takes row t / 4, dims 32 (t % 4) .. + 32,
// with 16-byte loads when the rows allow them (`vec`).
template <int DT>
__device__ __forceinline__ void stage_rows(const KmeansParams &p, int64_t r0, int k0,
                                           float (*xs)[kKK + 1], bool vec) {
  const int tid = threadIdx.x;
  const int r = tid >> 2, kk = (tid & 3) * 32;
  const int64_t row = r0 + r;
  const int d = p.d;
  if (vec && row < p.n && k0 + kk + 32 <= d) {
    if constexpr (DT == kF32) {
      const float4 *src =
          reinterpret_cast<const float4 *>(static_cast<const float *>(p.x) + row * d + k0 + kk);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float4 v = src[e];
        xs[r][kk + 4 * e] = v.x;
        xs[r][kk + 4 * e + 1] = v.y;
        xs[r][kk + 4 * e + 2] = v.z;
        xs[r][kk + 4 * e + 3] = v.w;
      }
    } else {
      const uint4 *src =
          reinterpret_cast<const uint4 *>(static_cast<const uint16_t *>(p.x) + row * d + k0 + kk);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint4 v = src[e];
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const uint16_t lo = (uint16_t)(w[j] & 0xffffu), hi = (uint16_t)(w[j] >> 16);
          if constexpr (DT == kF16) {
            xs[r][kk + 8 * e + 2 * j] = (float)__builtin_bit_cast(_Float16, lo);
            xs[r][kk + 8 * e + 2 * j + 1] = (float)__builtin_bit_cast(_Float16, hi);
          } else {
            xs[r][kk + 8 * e + 2 * j] = __uint_as_float((uint32_t)lo << 16);
            xs[r][kk + 8 * e + 2 * j + 1] = __uint_as_float((uint32_t)hi << 16);
          }
        }
      }
    }
  } else {
#pragma unroll 8
    for (int e = 0; e < 32; ++e) {
      const int k = k0 + kk + e;
      xs[r][kk + e] = (row < p.n && k < d) ? load_elem<DT>(p.x, row * d + k) : 0.f;
    }
  }
}

template <int DT>
__global__ void __launch_bounds__(256) dresd_kmeans_assign(KmeansParams p) {
  __shared__ float xs[kKR][kKK + 1];  // rows (padded: no bank conflicts)
  __shared__ float cs[kKK][kKC];      // centroids, dim-major
  const int tid = threadIdx.x, lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, m = lane & 15;
  const int64_t r0 = (int64_t)blockIdx.x * kKR;
  const int d = p.d, P = p.P;
  const int es = DT == kF32 ? 4 : 2;
  const bool xvec = (((uintptr_t)p.x & 15u) == 0) && ((d * es) % 16 == 0);
  const bool cvec = (((uintptr_t)p.centroids & 15u) == 0) && (d % 4 == 0);
  // running best of rows wv*16 + 4g + i (identical in the 16 lanes of a group)
  float best[4];
  int bid[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    best[i] = -__builtin_inff();
    bid[i] = 0x7fffffff;
  }
  // Centroid tile (c0, k0) goes through registers: thread t loads centroid
  // c0 + t / 4, dims k0 + 32 (t % 4) .. + 32 (one tile ahead of its use).
  float4 creg[8];
  auto load_c = [&](int c0, int k0) {
    const int c = c0 + (tid >> 2), kk = k0 + (tid & 3) * 32;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int k = kk + 4 * e;
      const float *src = p.centroids + (int64_t)c * d + k;
      if (c < P && cvec && k + 4 <= d) {
        creg[e] = *reinterpret_cast<const float4 *>(src);
      } else {
        creg[e].x = (c < P && k < d) ? src[0] : 0.f;
        creg[e].y = (c < P && k + 1 < d) ? src[1] : 0.f;
        creg[e].z = (c < P && k + 2 < d) ? src[2] : 0.f;
        creg[e].w = (c < P && k + 3 < d) ? src[3] : 0.f;
      }
    }
  };
  auto store_c = [&]() {
    const int cl = tid >> 2, kk = (tid & 3) * 32;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      cs[kk + 4 * e][cl] = creg[e].x;
      cs[kk + 4 * e + 1][cl] = creg[e].y;
      cs[kk + 4 * e + 2][cl] = creg[e].z;
      cs[kk + 4 * e + 3][cl] = creg[e].w;
    }
  };
  // Rows of at most 128 dims are staged once for all centroid tiles.
  const bool x_once = d <= kKK;
  if (x_once) stage_rows<DT>(p, r0, 0, xs, xvec);
  load_c(0, 0);
  for (int c0 = 0; c0 < P; c0 += kKC) {
    f4 acc[kKC / 16];
#pragma unroll
    for (int t = 0; t < kKC / 16; ++t) acc[t] = f4{0.f, 0.f, 0.f, 0.f};
    for (int k0 = 0; k0 < d; k0 += kKK) {
      if (!x_once) stage_rows<DT>(p, r0, k0, xs, xvec);
      store_c();
      __syncthreads();
      // the next centroid tile's loads overlap this tile's matrix work
      int nk0 = k0 + kKK, nc0 = c0;
      if (nk0 >= d) {
        nk0 = 0;
        nc0 = c0 + kKC;
      }
      if (nc0 < P) load_c(nc0, nk0);
      // lane (g, m) feeds A[row m][k g] and B[k g][centroid m]
#pragma unroll 8
      for (int ks = 0; ks < kKK; ks += 4) {
        const float a = xs[wv * 16 + m][ks + g];
#pragma unroll
        for (int t = 0; t < kKC / 16; ++t)
          acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, cs[ks + g][t * 16 + m], acc[t], 0, 0, 0);
      }
      __syncthreads();
    }
    // D layout: lane (g, m), register i -> row 4g + i, centroid t*16 + m.
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float s = -__builtin_inff();
      int id = 0x7fffffff;
#pragma unroll
      for (int t = 0; t < kKC / 16; ++t) {
        const int c = c0 + t * 16 + m;
        if (c < P && beats(acc[t][i], c, s, id)) {
          s = acc[t][i];
          id = c;
        }
      }
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) {
        const float os = __shfl_xor(s, off, kWaveSize);
        const int oid = __shfl_xor(id, off, kWaveSize);
        if (beats(os, oid, s, id)) {
          s = os;
          id = oid;
        }
      }
      if (beats(s, id, best[i], bid[i])) {
        best[i] = s;
        bid[i] = id;
      }
    }
  }
  if (m == 0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t row = r0 + wv * 16 + 4 * g + i;
      if (row < p.n) {
        p.assign[row] = bid[i];
        if (p.score) p.score[row] = best[i];
      }
    }
  }
}

// Zero the fixed-point sums and the counts.
__global__ void __launch_bounds__(256) dresd_kmeans_clear(KmeansParams p) {
  const int64_t nsum = (int64_t)p.P * p.d;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < nsum + p.P;
       i += (int64_t)gridDim.x * blockDim.x) {
    if (i < nsum) p.sums[i] = 0;
    else p.cnt[i - nsum] = 0;
  }
}

// Add every row into its partition's fixed-point sum: thread per (row, dim).
template <int DT>
__global__ void __launch_bounds__(256) dresd_kmeans_accumulate(KmeansParams p) {
  const int64_t total = p.n * p.d;
  for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t row = e / p.d;
    const int j = (int)(e - row * p.d);
    const int a = p.assign_in[row];
    const double v = (double)load_elem<DT>(p.x, e) * kFixScale;
    atomicAdd(reinterpret_cast<unsigned long long *>(p.sums + (int64_t)a * p.d + j),
              (unsigned long long)(long long)__double2ll_rn(v));
    if (j == 0) atomicAdd(p.cnt + a, 1);
  }
}

// One wave per partition: centroid = sum / ||sum|| when the partition has
// rows and a non-zero sum; otherwise unchanged.
__global__ void __launch_bounds__(256) dresd_kmeans_finish(KmeansParams p) {
  const int lane = threadIdx.x & 63;
  const int part = blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  if (part >= p.P) return;
  const long long *s = p.sums + (int64_t)part * p.d;
  double ss = 0.0;
  for (int j = lane; j < p.d; j += kWaveSize) {
    const double v = (double)s[j];
    ss += v * v;
  }
  for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off, kWaveSize);
  const int c = p.cnt[part];
  if (lane == 0 && p.counts) p.counts[part] = c;
  if (c == 0 || !(ss > 0.0)) return;
  const double inv = 1.0 / sqrt(ss);
  float *out = p.centroids_out + (int64_t)part * p.d;
  for (int j = lane; j < p.d; j += kWaveSize) out[j] = (float)((double)s[j] * inv);
}

// One wave per centroid: centroid j = row pick(j) / ||row pick(j)||, with
// pick(j) = (offset + floor(j n / P)) mod n; a zero row gives a zero centroid.
template <int DT>
__global__ void __launch_bounds__(256) dresd_kmeans_init(KmeansParams p) {
  const int lane = threadIdx.x & 63;
  const int part = blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  if (part >= p.P) return;
  const uint64_t n = (uint64_t)p.n;
  const uint64_t row = ((uint64_t)p.offset + (uint64_t)part * n / (uint64_t)p.P) % n;
  const int64_t base = (int64_t)row * p.d;
  double ss = 0.0;
  for (int j = lane; j < p.d; j += kWaveSize) {
    const double v = (double)load_elem<DT>(p.x, base + j);
    ss += v * v;
  }
  for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off, kWaveSize);
  const double inv = ss > 0.0 ? 1.0 / sqrt(ss) : 0.0;
  float *out = p.centroids_out + (int64_t)part * p.d;
  for (int j = lane; j < p.d; j += kWaveSize)
    out[j] = (float)((double)load_elem<DT>(p.x, base + j) * inv);
}

template <typename F>
hipError_t launch1(F *k, dim3 grid, dim3 block, KmeansParams &p, hipStream_t st) {
  void *args[] = {&p};
  return hipLaunchKernel((const void *)k, grid, block, args, 0, st);
}

}  // namespace

hipError_t launch_kmeans_assign(const KmeansParams &pin, hipStream_t st) {
  if (pin.n == 0) return hipSuccess;
  KmeansParams p = pin;
  const dim3 grid((unsigned)((p.n + kKR - 1) / kKR));
  if (p.dtype == kF32) return launch1(dresd_kmeans_assign<kF32>, grid, dim3(256), p, st);
  if (p.dtype == kF16) return launch1(dresd_kmeans_assign<kF16>, grid, dim3(256), p, st);
  return launch1(dresd_kmeans_assign<kBF16>, grid, dim3(256), p, st);
}

hipError_t launch_kmeans_update(const KmeansParams &pin, int cus, hipStream_t st) {
  KmeansParams p = pin;
  auto blocks = [](int64_t work, int64_t most) {
    const int64_t b = (work + 255) / 256;
    return dim3((unsigned)(b < most ? (b > 0 ? b : 1) : most));
  };
  hipError_t e = launch1(dresd_kmeans_clear, blocks((int64_t)p.P * p.d + p.P, cus * 8LL),
                         dim3(256), p, st);
  if (e != hipSuccess) return e;
  if (p.n > 0) {
    const dim3 grid = blocks(p.n * p.d, cus * 32LL);
    if (p.dtype == kF32) e = launch1(dresd_kmeans_accumulate<kF32>, grid, dim3(256), p, st);
    else if (p.dtype == kF16) e = launch1(dresd_kmeans_accumulate<kF16>, grid, dim3(256), p, st);
    else e = launch1(dresd_kmeans_accumulate<kBF16>, grid, dim3(256), p, st);
    if (e != hipSuccess) return e;
  }
  return launch1(dresd_kmeans_finish, dim3((unsigned)((p.P + 3) / 4)), dim3(256), p, st);
}

hipError_t launch_kmeans_init(const KmeansParams &pin, hipStream_t st) {
  KmeansParams p = pin;
  const dim3 grid((unsigned)((p.P + 3) / 4));
  if (p.dtype == kF32) return launch1(dresd_kmeans_init<kF32>, grid, dim3(256), p, st);
  if (p.dtype == kF16) return launch1(dresd_kmeans_init<kF16>, grid, dim3(256), p, st);
  return launch1(dresd_kmeans_init<kBF16>, grid, dim3(256), p, st);
}

}  // namespace dresd
