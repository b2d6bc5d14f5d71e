// gfx950 draft assembly for batch verification (DReSD Section 3.6): the
// retrieved continuations become the rows of a [r, length] draft matrix
// padded with the EOS id.  A draft is the first `length` tokens of a
// continuation with every token after its first EOS replaced by EOS; drafts
// that start with EOS (nothing to propose) and repeats of an earlier draft
// are dropped, and the first r remaining drafts, in rank order, fill the rows.
//
// One workgroup (1024 threads) per query, one thread per retrieved rank:
// each thread hashes its normalised draft into LDS, compares with the hashes
// of all earlier ranks (exact comparison on a hash match), and a workgroup
// prefix sum over the kept flags gives every kept draft its row.
#include "dresd_device.h"
#include "dresd_ops.h"

namespace dresd {

namespace {

constexpr int kDraftThreads = 1024;

// Token j of rank i's draft: EOS once the continuation has reached EOS.
struct DraftView {
  const int32_t *t;  // [k, L] of this query
  int L, length, eos;
  __device__ int32_t at(int i, int j, bool &ended) const {
    const int32_t v = t[(size_t)i * L + j];
    if (ended) return eos;
    if (v == eos) ended = true;
    return v;
  }
};

__global__ void __launch_bounds__(kDraftThreads) dresd_pack(DraftParams p) {
  __shared__ uint64_t hash[DRESD_K_MAX_INTERNAL];
  __shared__ uint32_t nonempty[DRESD_K_MAX_INTERNAL];
  __shared__ uint32_t wsum[kDraftThreads / kWaveSize];
  const int b = blockIdx.x;
  const int i = threadIdx.x, lane = i & 63, wid = i >> 6;
  DraftView v{p.tokens + (size_t)b * p.k * p.L, p.L, p.length, p.eos};

  // 1. hash of the normalised draft (64-bit FNV-1a over the tokens)
  bool ne = false;
  if (i < p.k) {
    uint64_t h = 1469598103934665603ull;
    bool ended = false;
    for (int j = 0; j < p.length; ++j) {
      const int32_t x = v.at(i, j, ended);
      if (j == 0) ne = x != p.eos;
      h = (h ^ (uint32_t)x) * 1099511628211ull;
    }
    hash[i] = h;
    nonempty[i] = ne ? 1u : 0u;
  }
  __syncthreads();

  // 2. drop repeats of an earlier non-empty draft (exact check on equal hash)
  bool keep = false;
  if (i < p.k && ne) {
    keep = true;
    const uint64_t h = hash[i];
    for (int j = 0; j < i && keep; ++j) {
      if (!nonempty[j] || hash[j] != h) continue;
      bool same = true, ei = false, ej = false;
      for (int c = 0; c < p.length && same; ++c) same = v.at(i, c, ei) == v.at(j, c, ej);
      if (same) keep = false;
    }
  }

  // 3. row of each kept draft: workgroup prefix sum of the kept flags
  const uint64_t m = __ballot(keep);
  const uint32_t before = __popcll(m & ((1ull << lane) - 1ull));
  if (lane == 0) wsum[wid] = (uint32_t)__popcll(m);
  __syncthreads();
  uint32_t base = 0, total = 0;
  for (int w = 0; w < kDraftThreads / kWaveSize; ++w) {
    if (w < wid) base += wsum[w];
    total += wsum[w];
  }
  const uint32_t row = base + before;
  int32_t *out = p.drafts + (size_t)b * p.r * p.length;
  if (keep && row < (uint32_t)p.r) {
    bool ended = false;
    for (int j = 0; j < p.length; ++j) out[(size_t)row * p.length + j] = v.at(i, j, ended);
  }
  // 4. rows past the kept drafts are all EOS
  const int n = total < (uint32_t)p.r ? (int)total : p.r;
  for (int e = n * p.length + i; e < p.r * p.length; e += kDraftThreads) out[e] = p.eos;
  if (i == 0) p.count[b] = n;
}

}  // namespace

hipError_t launch_pack_drafts(const DraftParams &p, hipStream_t st) {
  if (p.B == 0) return hipSuccess;
  DraftParams q = p;
  void *args[] = {&q};
  return hipLaunchKernel((const void *)dresd_pack, dim3((unsigned)p.B), dim3(kDraftThreads), args,
                         0, st);
}

}  // namespace dresd
