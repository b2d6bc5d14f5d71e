// gfx950 merge + gather kernel: one workgroup per query turns the scan's
// per-wave candidate lists into the exact k best keys of that query
// (DReSD Section 3.5, Eq. 3 taken as top-k for batch verification,
// Section 3.6), then gathers the winners' continuations -- the value map of
// the key -> next-tokens datastore.  For a sampled pass it instead emits the
// k-th best key, a lower bound that prunes the next pass.
//
// Latency matters more than throughput here (one short kernel per pass), so
// every step is one round of independent loads followed by a few barriers:
// list summaries, then all listed keys at once (flattened over lists), and
// radix selections that start at the highest bit where the keys differ.
#include "dresd_device.h"
#include "dresd_ops.h"

namespace dresd {

// Candidate counts up to this are ordered whole (no selection first).
constexpr int kSmallMerge = 256;
// Winner counts up to this are ordered by rank, larger ones by a bitonic
// network over the workgroup.
constexpr int kRankSortMax = 512;
// Each thread owns this many lists (their offsets share the histogram).
constexpr int kListsPerThread = kMergeLists / kMergeThreads;

struct MergeShared {
  uint32_t hist[kMergeLists];  // radix histogram (256 bins); list offsets during the gather
  uint32_t part[kMergeThreads / kWaveSize];
  alignas(16) uint64_t cache[kMergeCap];
  alignas(16) uint64_t win[DRESD_K_MAX_INTERNAL];
  uint64_t sel_prefix, sel_mask, bound, v_and, v_or;
  uint32_t sel_krem, sel_done, win_cnt, ncand, total, any_known;
};

__device__ inline uint64_t wave_and(uint64_t v) {
  for (int off = 32; off > 0; off >>= 1) v &= __shfl_xor(v, off, kWaveSize);
  return v;
}
__device__ inline uint64_t wave_or(uint64_t v) {
  for (int off = 32; off > 0; off >>= 1) v |= __shfl_xor(v, off, kWaveSize);
  return v;
}
__device__ inline uint64_t wave_max(uint64_t v) {
  for (int off = 32; off > 0; off >>= 1) {
    const uint64_t o = __shfl_xor(v, off, kWaveSize);
    v = o > v ? o : v;
  }
  return v;
}

typedef uint64_t u64x2 __attribute__((ext_vector_type(2)));

// Descending order of n distinct keys src[0..n) (every key names its own
// row): key i goes to dst[number of keys greater than it] when that is below
// `keep`.  T adjacent lanes (a power of two, as many as the workgroup allows
// up to a wave) share a key's count, so every wave takes part; keys are read
// as LDS broadcasts and there is no barrier inside.  src and dst are 16-byte
// aligned LDS arrays; src is not written.
__device__ inline void rank_sort_desc(const uint64_t *src, uint32_t n, uint64_t *dst,
                                      uint32_t keep, int tid, int nth) {
  int T = 1;
  while (T < kWaveSize && n * (uint32_t)(2 * T) <= (uint32_t)nth) T <<= 1;
  const int sub = tid & (T - 1);
  const uint32_t per = (uint32_t)(nth / T), n2 = n & ~1u;
  for (uint32_t i0 = 0; i0 < n; i0 += per) {
    const uint32_t i = i0 + (uint32_t)(tid / T);
    const bool valid = i < n;
    const uint64_t x = valid ? src[i] : ~0ull;
    uint32_t r = 0;
#pragma unroll 4
    for (uint32_t j = 2u * (uint32_t)sub; j < n2; j += 2u * (uint32_t)T) {
      const u64x2 v = *reinterpret_cast<const u64x2 *>(src + j);
      r += (uint32_t)(v.x > x) + (uint32_t)(v.y > x);
    }
    if ((n & 1u) && sub == 0) r += (uint32_t)(src[n - 1] > x);
    for (int o = 1; o < T; o <<= 1) r += __shfl_xor(r, o, kWaveSize);
    if (valid && sub == 0 && r < keep) dst[r] = x;
  }
}

// Largest value v such that at least kk of the M values src(i) are >= v
// (1 <= kk <= M; the kk-th largest value, or a lower boundary of the digit
// bin holding exactly the kk largest values).  Radix selection 8 bits at a
// time from the highest bit in which the values differ: every thread adds
// its values to the 256-bin histogram, then one wave finds the bin holding
// the kk-th largest (and clears the histogram), two barriers per digit.
// Called by the whole workgroup.
template <class Src>
__device__ uint64_t radix_kth(MergeShared &sh, Src src, uint32_t M, uint32_t kk) {
  constexpr int kDigit = 8, kBins = 1 << kDigit, kBinsPerLane = kBins / kWaveSize;
  const int tid = threadIdx.x, nth = blockDim.x;
  const int lane = tid & (kWaveSize - 1), wid = tid / kWaveSize;
  if (tid == 0) {
    sh.v_and = ~0ull;
    sh.v_or = 0ull;
    sh.sel_done = 0u;
  }
  if (tid < kBins) sh.hist[tid] = 0;
  __syncthreads();
  uint64_t va = ~0ull, vo = 0ull;
  for (uint32_t i = tid; i < M; i += nth) {
    const uint64_t key = src(i);
    va &= key;
    vo |= key;
  }
  va = wave_and(va);
  vo = wave_or(vo);
  if (lane == 0) {
    atomicAnd((unsigned long long *)&sh.v_and, (unsigned long long)va);
    atomicOr((unsigned long long *)&sh.v_or, (unsigned long long)vo);
  }
  __syncthreads();
  const uint64_t diff = sh.v_and ^ sh.v_or;
  if (diff == 0) return sh.v_or;  // one distinct value
  int top = 63 - __clzll((long long)diff);
  uint64_t pm = (top == 63) ? 0ull : ~((2ull << top) - 1ull);  // bits fixed so far
  uint64_t pre = sh.v_and & pm;                                 // their values
  uint32_t krem = kk;  // rank of the answer among the values matching pre
  // Every thread follows the same (pre, pm, top, krem), published by wave 0.
  for (;;) {
    const int w = top + 1 < kDigit ? top + 1 : kDigit;
    const int s = top + 1 - w;
    const uint32_t wmask = (1u << w) - 1u;
    for (uint32_t i = tid; i < M; i += nth) {
      const uint64_t key = src(i);
      if ((key & pm) == pre) atomicAdd(&sh.hist[(uint32_t)(key >> s) & wmask], 1u);
    }
    __syncthreads();
    if (wid == 0) {
      // lane l owns bins [kBinsPerLane l, kBinsPerLane (l + 1)); count the
      // values in the bins of all higher lanes
      uint32_t h[kBinsPerLane], mine = 0;
#pragma unroll
      for (int j = 0; j < kBinsPerLane; ++j) {
        h[j] = sh.hist[lane * kBinsPerLane + j];
        mine += h[j];
      }
      uint32_t incl = mine;
      for (int off = 1; off < kWaveSize; off <<= 1) {
        const uint32_t v = __shfl_down(incl, off, kWaveSize);
        if (lane + off < kWaveSize) incl += v;
      }
      const uint32_t cnt_above = incl - mine;
      if (cnt_above < krem && krem <= cnt_above + mine) {
        uint32_t cum = cnt_above;
        for (int j = kBinsPerLane - 1; j >= 0; --j) {
          if (cum + h[j] >= krem) {
            const uint32_t dg = (uint32_t)(lane * kBinsPerLane + j);
            sh.sel_prefix = pre | ((uint64_t)dg << s);
            sh.sel_mask = pm | ((uint64_t)wmask << s);
            sh.sel_krem = krem - cum;
            sh.sel_done = (h[j] == krem - cum) ? 1u : 0u;  // the whole bin is in
            break;
          }
          cum += h[j];
        }
      }
#pragma unroll
      for (int j = 0; j < kBinsPerLane; ++j) sh.hist[lane * kBinsPerLane + j] = 0;
    }
    __syncthreads();
    pre = sh.sel_prefix;
    pm = sh.sel_mask;
    krem = sh.sel_krem;
    top = s - 1;
    if (sh.sel_done || top < 0) break;
    // wave 0 rewrites the state only after the next histogram's barrier,
    // which every thread reaches after reading it
  }
  return pre;
}

// Output of one query from its sorted winners win[0..kk): the k-th best key
// (sampled pass) or indices, scores and gathered continuations (final pass).
// Each thread issues all of its continuation loads before its first store,
// so the gather costs one memory latency rather than one per token.  A
// winner that names no row of the value table (only an upstream fault could
// produce one) is written as index -1, score -inf and zero tokens instead of
// being dereferenced.
__device__ inline void write_result(const MergeParams &p, int b, const uint64_t *win,
                                    uint32_t kk, int tid, int nth) {
  if (!p.final_mode) {
    // The k-th best key of any subset of the rows is a lower bound of the
    // k-th best of all of them; a pass that found fewer than k keys at or
    // above its (speculative) threshold keeps the bound it started from.
    // The speculative key for the next pass is the spec_rank-th best found,
    // never below the bound.
    if (tid == 0) {
      const uint64_t fb = p.tau_fb ? p.tau_fb[b] : 0ull;
      uint64_t v = (kk >= (uint32_t)p.k) ? win[p.k - 1] : 0ull;
      v = v > fb ? v : fb;
      p.tau_out[b] = v;
      if (p.spec_out) {
        const uint64_t s = (kk >= (uint32_t)p.spec_rank) ? win[p.spec_rank - 1] : 0ull;
        p.spec_out[b] = s > v ? s : v;
      }
    }
    return;
  }
  for (int r = tid; r < p.k; r += nth) {
    const size_t o = (size_t)b * p.k + r;
    const uint32_t row = r < (int)kk ? ~(uint32_t)win[r] : 0xFFFFFFFFu;
    if ((int64_t)row < p.N) {
      p.idx[o] = (int64_t)row;
      p.score[o] = order_value((uint32_t)(win[r] >> 32));
    } else {  // past the candidates (cannot happen when N >= k), or no row
      p.idx[o] = -1;
      p.score[o] = -__builtin_inff();
    }
  }
  if (p.tokens) {
    constexpr int R = 8;  // tokens per thread per round, loaded together
    const int L = p.L, n = p.k * L;
    int32_t *out = p.tokens + (size_t)b * p.k * L;
    for (int i0 = tid; i0 < n; i0 += R * nth) {
      int32_t v[R];
#pragma unroll
      for (int u = 0; u < R; ++u) {
        const int i = i0 + u * nth;
        const int r = i / L;
        v[u] = 0;
        if (i < n && r < (int)kk) {
          const uint32_t row = ~(uint32_t)win[r];
          if ((int64_t)row < p.N) v[u] = p.cont[(size_t)row * L + (i - r * L)];
        }
      }
#pragma unroll
      for (int u = 0; u < R; ++u)
        if (i0 + u * nth < n) out[i0 + u * nth] = v[u];
    }
  }
}

// 1. A lower bound on the query's k-th best key: the larger of (a) the best
//    k-th key published by any list holding k sorted keys and (b) the k-th
//    largest of the lists' known best keys -- k distinct listed keys reach
//    each, and the answer is among the listed keys.
// 2. Candidates: listed keys at or above the bound; lists whose best key is
//    below it are not opened.  All kept lists' keys are loaded at once.
// 3. The k best candidates: ordered by rank when few, else a radix select
//    finds the k-th and the keys at or above it are ordered.
__global__ void __launch_bounds__(kMergeThreads) dresd_merge(MergeParams p) {
  __shared__ MergeShared sh;
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int nth = blockDim.x;
  const int lane = tid & (kWaveSize - 1), wid = tid / kWaveSize;
  const int G = p.G;
  const uint32_t *lcnt = p.lcnt + (size_t)b * G;
  const uint64_t *lkth = p.lkth + (size_t)b * G;
  const uint64_t *lfirst = p.lfirst + (size_t)b * G;
  const uint64_t *lists = p.lists + (size_t)b * G * p.C;
  uint64_t *spill = p.spill + (size_t)b * p.spill_cap;
  if (tid == 0) {
    sh.bound = 0;
    sh.ncand = 0;
    sh.win_cnt = 0;
    sh.any_known = 0;
  }
  __syncthreads();
  // Thread t owns lists [L t, L t + L), L = kListsPerThread.
  uint32_t cnt[kListsPerThread];
  uint64_t first[kListsPerThread];
  uint64_t mb = 0;
  bool known = false;
#pragma unroll
  for (int j = 0; j < kListsPerThread; ++j) {
    const int w = tid * kListsPerThread + j;
    cnt[j] = 0;
    first[j] = 0;
    if (w < G) {
      cnt[j] = min(lcnt[w] & ~kSortedFlag, (uint32_t)p.C);
      first[j] = lfirst[w];
      const uint64_t v = lkth[w];
      mb = v > mb ? v : mb;
      const uint64_t f = first[j];
      sh.cache[w] = (f == ~0ull) ? 0ull : f;
      known |= (f != ~0ull && f != 0ull);
    }
  }
  mb = wave_max(mb);
  if (lane == 0 && mb) atomicMax((unsigned long long *)&sh.bound, (unsigned long long)mb);
  if (known) sh.any_known = 1u;
  __syncthreads();
  // (b), worth a selection only when some list's best key is known
  if (sh.any_known && G >= p.k) {
    const uint64_t t1 =
        radix_kth(sh, [&](uint32_t i) { return sh.cache[i]; }, (uint32_t)G, (uint32_t)p.k);
    if (tid == 0 && t1 > sh.bound) sh.bound = t1;
  }
  __syncthreads();
  const uint64_t bnd = sh.bound;

  // 2. offsets of the kept lists' keys (lists at or above the bound), then
  //    every key loaded by its own thread
  uint32_t mine = 0;
#pragma unroll
  for (int j = 0; j < kListsPerThread; ++j) {
    if (first[j] < bnd) cnt[j] = 0;
    mine += cnt[j];
  }
  uint32_t incl = mine;
  for (int off = 1; off < kWaveSize; off <<= 1) {
    const uint32_t v = __shfl_up(incl, off, kWaveSize);
    if (lane >= off) incl += v;
  }
  if (lane == kWaveSize - 1) sh.part[wid] = incl;
  __syncthreads();
  uint32_t base = incl - mine;
  for (int q = 0; q < wid; ++q) base += sh.part[q];
#pragma unroll
  for (int j = 0; j < kListsPerThread; ++j) {
    sh.hist[tid * kListsPerThread + j] = base;
    base += cnt[j];
  }
  if (tid == nth - 1) sh.total = base;
  __syncthreads();
  const uint32_t total = sh.total;
  const int nl = G;
  constexpr int R = 8;  // keys per thread per round, loaded together
  for (uint32_t i0 = tid; i0 < total; i0 += R * nth) {
    uint64_t key[R];
#pragma unroll
    for (int u = 0; u < R; ++u) {
      const uint32_t i = i0 + (uint32_t)(u * nth);
      key[u] = 0ull;
      if (i < total) {
        // the last list whose offset is <= i holds key i
        int lo = 0, hi = nl;  // answer in [lo, hi)
        while (hi - lo > 1) {
          const int mid = (lo + hi) >> 1;
          if (sh.hist[mid] <= i) lo = mid;
          else hi = mid;
        }
        key[u] = lists[(size_t)lo * p.C + (i - sh.hist[lo])];
      }
    }
#pragma unroll
    for (int u = 0; u < R; ++u) {
      if (i0 + (uint32_t)(u * nth) < total && key[u] >= bnd) {
        const uint32_t at = atomicAdd(&sh.ncand, 1u);
        if (at < (uint32_t)kMergeCap) sh.cache[at] = key[u];
        else if ((int64_t)(at - kMergeCap) < p.spill_cap) spill[at - kMergeCap] = key[u];
      }
    }
  }
  // Winner slots start empty (key 0 names no row), so that a slot no key
  // reaches is written as a missing result rather than as stale LDS.
  for (int i = tid; i < p.k; i += nth) sh.win[i] = 0ull;
  __threadfence_block();
  __syncthreads();
  const uint32_t M = sh.ncand;
  const uint32_t kk = M < (uint32_t)p.k ? M : (uint32_t)p.k;

  // 3. the k best
  if (M <= (uint32_t)kSmallMerge) {
    rank_sort_desc(sh.cache, M, sh.win, kk, tid, nth);
    __syncthreads();
    write_result(p, b, sh.win, kk, tid, nth);
    return;
  }
  auto cand = [&](uint32_t i) {
    return i < (uint32_t)kMergeCap ? sh.cache[i] : spill[i - kMergeCap];
  };
  const uint64_t cut = (kk == M) ? 0ull : radix_kth(sh, cand, M, kk);
  for (uint32_t i = tid; i < M; i += nth) {
    const uint64_t key = cand(i);
    if (key >= cut) {
      const uint32_t at = atomicAdd(&sh.win_cnt, 1u);
      if (at < (uint32_t)DRESD_K_MAX_INTERNAL) sh.win[at] = key;
    }
  }
  __syncthreads();
  if (kk <= (uint32_t)kRankSortMax) {  // the winners, ordered into the free cache
    for (uint32_t i = tid; i < kk; i += nth) sh.cache[i] = 0ull;
    __syncthreads();
    rank_sort_desc(sh.win, kk, sh.cache, kk, tid, nth);
    __syncthreads();
    write_result(p, b, sh.cache, kk, tid, nth);
    return;
  }
  int n = 1;
  while (n < (int)kk) n <<= 1;
  for (int i = (int)kk + tid; i < n; i += nth) sh.win[i] = 0ull;
  __syncthreads();
  block_bitonic_desc(sh.win, n);
  write_result(p, b, sh.win, kk, tid, nth);
}

void *merge_kernel_ptr() { return (void *)dresd_merge; }

}  // namespace dresd
