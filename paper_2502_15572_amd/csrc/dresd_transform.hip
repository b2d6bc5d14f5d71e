// gfx950 kernels of the query-side transform, Algorithm 1 steps 4-6:
// z-score normalisation with the datastore's per-dimension mean and variance
// (Section 3.2, Eq. 1), projection onto the first l principal components
// (Section 3.3, v W_l) and L2 normalisation (Section 3.4, Eq. 2).
//
// The projection is a dense contraction [M, D] x [D, l] in fp32 on the fp32
// matrix cores (v_mfma_f32_16x16x4_f32).  A workgroup computes a 64 x 64
// output tile over a slice of the D dims, staging 128 dims of z-scored inputs
// and weights in LDS per step (the inputs are z-scored while staged, with each
// dim's mean and 1 / sqrt(var + eps) computed once per step, so x is read once
// per column tile).  Few output tiles (decode-step batches) split D
// across workgroups so that the whole chip streams W; the partial sums go to a
// workspace; a second kernel adds them in a fixed order (deterministic) and
// scales every row to unit length.
#include "dresd_device.h"

namespace dresd {

namespace {

constexpr int kTR = 64;   // output rows per workgroup
constexpr int kTC = 64;   // output columns per workgroup
constexpr int kKS = 128;  // dims staged per step

__global__ void __launch_bounds__(256) dresd_project(TransformParams p) {
  __shared__ float zs[kTR][kKS + 1];  // z-scored inputs (padded rows: no bank conflicts)
  __shared__ float ws[kKS][kTC];      // projection weights
  __shared__ float mu[kKS], inv[kKS]; // the step's means and 1 / sqrt(var + eps_z)
  const int tid = threadIdx.x, lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int64_t r0 = (int64_t)blockIdx.x * kTR;
  const int c0 = blockIdx.y * kTC;
  const int split = blockIdx.z;
  const int D = p.D, l = p.l;
  const int kbeg = split * p.dslice;
  const int kend = kbeg + p.dslice < D ? kbeg + p.dslice : D;
  const int g = lane >> 4, m = lane & 15;
  // W rows start 16-byte aligned: stage them with 16-byte loads
  const bool wvec = ((l & 3) == 0) && (((uintptr_t)p.W & 15u) == 0);
  f4 acc[kTC / 16];
#pragma unroll
  for (int t = 0; t < kTC / 16; ++t) acc[t] = f4{0.f, 0.f, 0.f, 0.f};

  // x rows start 16-byte aligned: stage them with 16-byte loads
  const bool xvec = ((D & 3) == 0) && (((uintptr_t)p.x & 15u) == 0);
  for (int k0 = kbeg; k0 < kend; k0 += kKS) {
    // The step's per-dim normalisation (Eq. 1), once per dim.
    if (tid < kKS) {
      const int k = k0 + tid;
      mu[tid] = k < kend ? p.mean[k] : 0.f;
      inv[tid] = k < kend ? 1.0f / sqrtf(p.var[k] + p.eps_z) : 0.f;
    }
    __syncthreads();
    // Stage 64 rows x 128 dims of z (thread t: row t/4, dims 32(t%4)..+32)
    // and 128 dims x 64 columns of W (thread t: dim t/2, columns 32(t%2)..+32);
    // entries past M, D, l or the slice are zero.
    {
      const int r = tid >> 2, kk = (tid & 3) * 32;
      const int64_t row = r0 + r;
      if (xvec && row < p.M && ((k0 + kk) & 3) == 0 && k0 + kk + 32 <= kend) {
        const float4 *src = reinterpret_cast<const float4 *>(p.x + row * D + k0 + kk);
        float4 v[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = src[e];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          zs[r][kk + 4 * e] = (v[e].x - mu[kk + 4 * e]) * inv[kk + 4 * e];
          zs[r][kk + 4 * e + 1] = (v[e].y - mu[kk + 4 * e + 1]) * inv[kk + 4 * e + 1];
          zs[r][kk + 4 * e + 2] = (v[e].z - mu[kk + 4 * e + 2]) * inv[kk + 4 * e + 2];
          zs[r][kk + 4 * e + 3] = (v[e].w - mu[kk + 4 * e + 3]) * inv[kk + 4 * e + 3];
        }
      } else {
#pragma unroll 8
        for (int e = 0; e < 32; ++e) {
          const int k = k0 + kk + e;
          float z = 0.f;
          if (row < p.M && k < kend) z = (p.x[row * D + k] - mu[kk + e]) * inv[kk + e];  // Eq. 1
          zs[r][kk + e] = z;
        }
      }
      const int kw = tid >> 1, cc = (tid & 1) * 32;
      const int k = k0 + kw;
      if (wvec && k < kend && c0 + cc + 32 <= l) {
        const float4 *src = reinterpret_cast<const float4 *>(p.W + (int64_t)k * l + c0 + cc);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float4 v = src[e];
          ws[kw][cc + 4 * e] = v.x;
          ws[kw][cc + 4 * e + 1] = v.y;
          ws[kw][cc + 4 * e + 2] = v.z;
          ws[kw][cc + 4 * e + 3] = v.w;
        }
      } else {
#pragma unroll 8
        for (int e = 0; e < 32; ++e) {
          const int c = c0 + cc + e;
          ws[kw][cc + e] = (k < kend && c < l) ? p.W[(int64_t)k * l + c] : 0.f;
        }
      }
    }
    __syncthreads();
    // 32 k-steps of 4 dims; lane (g, m) feeds A[row m][k g] and B[k g][col m].
#pragma unroll 8
    for (int ks = 0; ks < kKS; ks += 4) {
      const float a = zs[wv * 16 + m][ks + g];
#pragma unroll
      for (int t = 0; t < kTC / 16; ++t)
        acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, ws[ks + g][t * 16 + m], acc[t], 0, 0, 0);
    }
    __syncthreads();
  }
  // D layout: lane (g, m), register i -> row 4 g + i, column m of the tile.
  float *out = p.splits > 1 ? p.part + (size_t)split * p.M * l : p.y;
#pragma unroll
  for (int t = 0; t < kTC / 16; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t row = r0 + wv * 16 + 4 * g + i;
      const int c = c0 + t * 16 + m;
      if (row < p.M && c < l) out[row * l + c] = acc[t][i];
    }
}

// One workgroup per row, one thread per column up to 1024 (the launch sizes
// the workgroup to the row): each thread adds its columns' split partial sums
// in split order (when D was split), then the row is scaled to unit length,
// y / max(||y||_2, eps) (Eq. 2).
constexpr int kFinishThreads = 1024;

__global__ void __launch_bounds__(kFinishThreads) dresd_finish_rows(TransformParams p) {
  __shared__ float part_ss[kFinishThreads / kWaveSize];
  const int64_t row = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int nth = blockDim.x, nw = nth / kWaveSize;
  const int64_t n = p.M * p.l;
  float *y = p.y + row * p.l;
  float ss = 0.f;
  for (int c = tid; c < p.l; c += nth) {
    float v;
    if (p.splits > 1) {
      v = 0.f;
#pragma unroll 8
      for (int s = 0; s < p.splits; ++s) v += p.part[(size_t)s * n + row * p.l + c];
      y[c] = v;
    } else {
      v = y[c];
    }
    ss += v * v;
  }
  for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off, kWaveSize);
  if (lane == 0) part_ss[wid] = ss;
  __syncthreads();
  float tot = 0.f;
  for (int w = 0; w < nw; ++w) tot += part_ss[w];
  const float inv = 1.0f / fmaxf(sqrtf(tot), p.eps_n);
  for (int c = tid; c < p.l; c += nth) y[c] = y[c] * inv;
}

}  // namespace

int transform_splits(int64_t M, int D, int l, int cus) {
  const int64_t tiles = ((M + kTR - 1) / kTR) * ((l + kTC - 1) / kTC);
  const int64_t want = (2 * (int64_t)cus + tiles - 1) / tiles;  // ~2 workgroups per CU
  const int64_t most = (D + kKS - 1) / kKS;
  int64_t s = want < most ? want : most;
  return (int)(s < 1 ? 1 : s);
}

hipError_t launch_transform(const TransformParams &p, hipStream_t st) {
  if (p.M == 0) return hipSuccess;
  TransformParams q = p;
  void *args[] = {&q};
  const dim3 grid1((unsigned)((p.M + kTR - 1) / kTR), (unsigned)((p.l + kTC - 1) / kTC),
                   (unsigned)p.splits);
  hipError_t e = hipLaunchKernel((const void *)dresd_project, grid1, dim3(256), args, 0, st);
  if (e != hipSuccess) return e;
  const int fin = std::min(kFinishThreads, std::max(kWaveSize, (p.l + kWaveSize - 1) / kWaveSize * kWaveSize));
  return hipLaunchKernel((const void *)dresd_finish_rows, dim3((unsigned)p.M), dim3((unsigned)fin),
                         args, 0, st);
}

}  // namespace dresd
