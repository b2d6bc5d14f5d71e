// gfx950 kernels of the query-side transform, Algorithm 1 steps 4-6:
// z-score normalisation with the datastore's per-dimension mean and variance
// (Section 3.2, Eq. 1), projection onto the first l principal components
// (Section 3.3, v W_l) and L2 normalisation (Section 3.4, Eq. 2).
//
// The projection is a dense contraction [M, D] x [D, l] in fp32 on the fp32
// matrix cores (v_mfma_f32_16x16x4_f32).  A workgroup computes a 64 x 64
// output tile (decode-step batches) or a 128 x 64 one (32 rows per wave, each
// weight operand serving two 16-row halves: datastore-sized batches) over a
// slice of the D dims, staging z-scored inputs and weights in LDS per step
// (the inputs are z-scored while staged, with each dim's mean and
// 1 / sqrt(var + eps) computed once per step, so x is read once per column
// tile).  Few output tiles (decode-step batches) split D
// across workgroups so that the whole chip streams W; the partial sums go to a
// workspace; a second kernel adds them in a fixed order (deterministic) and
// scales every row to unit length.
#include "dresd_device.h"
#include "dresd_ops.h"

namespace dresd {

namespace {

constexpr int kTC = 64;          // output columns per workgroup
constexpr int kSplitDims = 128;  // D is split into slices of whole multiples of this
// Batches up to this many rows take 64-row tiles staging 128 dims per step;
// larger ones 128-row tiles (32 rows per wave: each weight operand serves two
// 16-row halves, fewer LDS reads per matrix instruction) staging 64 dims.
constexpr int64_t kWideRowsFrom = 1024;

__host__ __device__ constexpr int project_rows(bool wide) { return wide ? 128 : 64; }

template <int HALVES, int KS>
__global__ void __launch_bounds__(256) dresd_project(TransformParams p) {
  constexpr int TR = 64 * HALVES;  // output rows per workgroup (16 * HALVES per wave)
  constexpr int TPR = 256 / TR;    // staging threads per row of z
  constexpr int DPT = KS / TPR;    // dims each of them stages
  constexpr int WTD = 256 / KS;    // staging threads per dim of W
  constexpr int CPT = kTC / WTD;   // columns each of them stages
  static_assert(DPT % 4 == 0 && CPT % 4 == 0, "staging shape");
  __shared__ float zs[TR][KS + 1];  // z-scored inputs (padded rows: no bank conflicts)
  __shared__ float ws[KS][kTC];     // projection weights
  __shared__ float mu[KS], inv[KS]; // the step's means and 1 / sqrt(var + eps_z)
  const int tid = threadIdx.x, lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int64_t r0 = (int64_t)blockIdx.x * TR;
  const int c0 = blockIdx.y * kTC;
  const int split = blockIdx.z;
  const int D = p.D, l = p.l;
  const int kbeg = split * p.dslice;
  const int kend = kbeg + p.dslice < D ? kbeg + p.dslice : D;
  const int g = lane >> 4, m = lane & 15;
  // W rows start 16-byte aligned: stage them with 16-byte loads
  const bool wvec = ((l & 3) == 0) && (((uintptr_t)p.W & 15u) == 0);
  f4 acc[HALVES][kTC / 16];  // the wave's 16-row halves x four 16-column tiles
#pragma unroll
  for (int h = 0; h < HALVES; ++h)
#pragma unroll
    for (int t = 0; t < kTC / 16; ++t) acc[h][t] = f4{0.f, 0.f, 0.f, 0.f};

  // x rows start 16-byte aligned: stage them with 16-byte loads
  const bool xvec = ((D & 3) == 0) && (((uintptr_t)p.x & 15u) == 0);
  for (int k0 = kbeg; k0 < kend; k0 += KS) {
    // The step's per-dim normalisation (Eq. 1), once per dim.
    if (tid < KS) {
      const int k = k0 + tid;
      mu[tid] = k < kend ? p.mean[k] : 0.f;
      inv[tid] = k < kend ? 1.0f / sqrtf(p.var[k] + p.eps_z) : 0.f;
    }
    __syncthreads();
    // Stage TR rows x KS dims of z (thread t: row t/TPR, DPT dims) and KS
    // dims x 64 columns of W (thread t: dim t/WTD, CPT columns); entries past
    // M, D, l or the slice are zero.
    {
      const int r = tid / TPR, kk = (tid % TPR) * DPT;
      const int64_t row = r0 + r;
      if (xvec && row < p.M && ((k0 + kk) & 3) == 0 && k0 + kk + DPT <= kend) {
        const float4 *src = reinterpret_cast<const float4 *>(p.x + row * D + k0 + kk);
        float4 v[DPT / 4];
#pragma unroll
        for (int e = 0; e < DPT / 4; ++e) v[e] = src[e];
#pragma unroll
        for (int e = 0; e < DPT / 4; ++e) {
          zs[r][kk + 4 * e] = (v[e].x - mu[kk + 4 * e]) * inv[kk + 4 * e];
          zs[r][kk + 4 * e + 1] = (v[e].y - mu[kk + 4 * e + 1]) * inv[kk + 4 * e + 1];
          zs[r][kk + 4 * e + 2] = (v[e].z - mu[kk + 4 * e + 2]) * inv[kk + 4 * e + 2];
          zs[r][kk + 4 * e + 3] = (v[e].w - mu[kk + 4 * e + 3]) * inv[kk + 4 * e + 3];
        }
      } else {
#pragma unroll 8
        for (int e = 0; e < DPT; ++e) {
          const int k = k0 + kk + e;
          float z = 0.f;
          if (row < p.M && k < kend) z = (p.x[row * D + k] - mu[kk + e]) * inv[kk + e];  // Eq. 1
          zs[r][kk + e] = z;
        }
      }
      const int kw = tid / WTD, cc = (tid % WTD) * CPT;
      const int k = k0 + kw;
      if (wvec && k < kend && c0 + cc + CPT <= l) {
        const float4 *src = reinterpret_cast<const float4 *>(p.W + (int64_t)k * l + c0 + cc);
#pragma unroll
        for (int e = 0; e < CPT / 4; ++e) {
          const float4 v = src[e];
          ws[kw][cc + 4 * e] = v.x;
          ws[kw][cc + 4 * e + 1] = v.y;
          ws[kw][cc + 4 * e + 2] = v.z;
          ws[kw][cc + 4 * e + 3] = v.w;
        }
      } else {
#pragma unroll 8
        for (int e = 0; e < CPT; ++e) {
          const int c = c0 + cc + e;
          ws[kw][cc + e] = (k < kend && c < l) ? p.W[(int64_t)k * l + c] : 0.f;
        }
      }
    }
    __syncthreads();
    // k-steps of 4 dims; lane (g, m) feeds A[row m][k g] and B[k g][col m].
#pragma unroll 4
    for (int ks = 0; ks < KS; ks += 4) {
      float a[HALVES];
#pragma unroll
      for (int h = 0; h < HALVES; ++h) a[h] = zs[wv * 16 * HALVES + 16 * h + m][ks + g];
#pragma unroll
      for (int t = 0; t < kTC / 16; ++t) {
        const float b = ws[ks + g][t * 16 + m];
#pragma unroll
        for (int h = 0; h < HALVES; ++h)
          acc[h][t] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[h], b, acc[h][t], 0, 0, 0);
      }
    }
    __syncthreads();
  }
  // D layout: lane (g, m), register i -> row 4 g + i, column m of the tile.
  float *out = p.splits > 1 ? p.part + (size_t)split * p.M * l : p.y;
#pragma unroll
  for (int h = 0; h < HALVES; ++h)
#pragma unroll
    for (int t = 0; t < kTC / 16; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int64_t row = r0 + wv * 16 * HALVES + 16 * h + 4 * g + i;
        const int c = c0 + t * 16 + m;
        if (row < p.M && c < l) out[row * l + c] = acc[h][t][i];
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
  const int tr = project_rows(M >= kWideRowsFrom);
  const int64_t tiles = ((M + tr - 1) / tr) * ((l + kTC - 1) / kTC);
  const int64_t want = (2 * (int64_t)cus + tiles - 1) / tiles;  // ~2 workgroups per CU
  const int64_t most = (D + kSplitDims - 1) / kSplitDims;
  int64_t s = want < most ? want : most;
  return (int)(s < 1 ? 1 : s);
}

hipError_t launch_transform(const TransformParams &p, hipStream_t st) {
  if (p.M == 0) return hipSuccess;
  TransformParams q = p;
  void *args[] = {&q};
  const bool wide = p.M >= kWideRowsFrom;
  const int tr = project_rows(wide);
  const dim3 grid1((unsigned)((p.M + tr - 1) / tr), (unsigned)((p.l + kTC - 1) / kTC),
                   (unsigned)p.splits);
  const void *proj = wide ? (const void *)dresd_project<2, 64> : (const void *)dresd_project<1, 128>;
  hipError_t e = hipLaunchKernel(proj, grid1, dim3(256), args, 0, st);
  if (e != hipSuccess) return e;
  const int fin = std::min(kFinishThreads, std::max(kWaveSize, (p.l + kWaveSize - 1) / kWaveSize * kWaveSize));
  return hipLaunchKernel((const void *)dresd_finish_rows, dim3((unsigned)p.M), dim3((unsigned)fin),
                         args, 0, st);
}

}  // namespace dresd
