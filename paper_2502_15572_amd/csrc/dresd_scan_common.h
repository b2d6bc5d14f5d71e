// Candidate handling shared by the scan kernels (fused per-query top-k of
// exact top-k retrieval, DReSD Section 3.5 / Eq. 3 generalised to k drafts).
//
// Each wave keeps, for each of its queries, a bounded candidate list in HBM
// (capacity C >= k + 64) fronted by a small stage in LDS (capacity CL).
// Passing keys go to the stage with LDS operations only; the stage is moved
// to the HBM list only when it is full (rare), and the HBM list is cut to its
// k best when it would overflow, raising the query's threshold to the k-th
// key.  Keeping vector-memory traffic out of the common path keeps the
// stream loop's wait counts exact.
#pragma once
#include "dresd_device.h"

namespace dresd {

struct CandSink {
  uint64_t *st_key;   // LDS [nq]: keep keys > st_key (exact threshold)
  uint32_t *st_cnt;   // LDS [nq]: keys in the HBM list
  float *st_thr;      // LDS [nq]: float threshold of the fast filter
  uint64_t *stg;      // LDS [nq][cl]: staged keys
  uint32_t *stg_cnt;  // LDS [nq]
  uint64_t *scr;      // LDS [C]: sort scratch
  int cl, C, k, lane;
};

__device__ inline void sink_init(const CandSink &s, int nq, int B_local, const uint64_t *tau) {
  for (int i = s.lane; i < nq; i += kWaveSize) {
    uint64_t tk = 0;
    float tf = -__builtin_inff();
    if (i >= B_local) {
      tk = ~0ull;
      tf = __builtin_inff();
    } else if (tau && tau[i] != 0) {
      tk = tau[i] - 1;  // keep keys >= tau
      tf = order_value((uint32_t)(tk >> 32));
    }
    s.st_key[i] = tk;
    s.st_cnt[i] = 0;
    s.st_thr[i] = tf;
    s.stg_cnt[i] = 0;
  }
  wave_sync_lds();
}

// Move query i's stage into its HBM list (cutting the list to its k best
// when it would overflow).  Wave-uniform; issues vector memory operations.
// `early`: inside the stream, where a query without a threshold yet (-inf)
// is also cut once list + stage hold 2k keys: the threshold (the median of
// those or better) then rises after a few tiles instead of after C - cl
// insertions, and the sort covers only the keys present.
__device__ inline void sink_spill(const CandSink &s, int i, uint64_t *list, bool early = false) {
  const int ns = (int)s.stg_cnt[i];
  int cnt = (int)s.st_cnt[i];
  const uint64_t *stg = s.stg + (size_t)i * s.cl;
  // The HBM list holds at most C - cl keys, so list + stage fit the C-entry
  // scratch; C >= k + 2 cl leaves room for a full stage after a cut.
  const int m = cnt + ns;
  if (m > s.C - s.cl || (early && m >= 2 * s.k && s.st_thr[i] == -__builtin_inff())) {
    __threadfence_block();  // this wave's list stores are visible to its loads
    int n = 2;
    while (n < m) n <<= 1;
    for (int e = s.lane; e < n; e += kWaveSize) {
      uint64_t v = 0ull;
      if (e < cnt) v = list[e];
      else if (e < m) v = stg[e - cnt];
      s.scr[e] = v;
    }
    wave_sync_lds();
    wave_bitonic_desc(s.scr, n, s.lane);
    for (int e = s.lane; e < s.k; e += kWaveSize) list[e] = s.scr[e];
    const uint64_t kth = s.scr[s.k - 1];
    wave_sync_lds();
    cnt = s.k;
    if (kth > s.st_key[i]) {
      s.st_key[i] = kth;
      s.st_thr[i] = order_value((uint32_t)(kth >> 32));
    }
  } else {
    for (int e = s.lane; e < ns; e += kWaveSize) list[cnt + e] = stg[e];
    cnt += ns;
  }
  s.st_cnt[i] = (uint32_t)cnt;
  s.stg_cnt[i] = 0;
  wave_sync_lds();
}

// Offer this lane's key to query i (wave-uniform i).  `mine` marks the
// lanes holding a score of query i that passed the fast filter -- at most
// one tile's 16 rows, which an emptied stage always holds (cl >= 16).
// Returns true when the stage was spilled (vector memory was used).
__device__ inline bool sink_offer(const CandSink &s, int i, bool mine, uint64_t key,
                                  uint64_t *list) {
  bool spilled = false;
  bool take = mine && key > s.st_key[i];
  uint64_t tm = __ballot(take);
  int n = __popcll(tm);
  if (n == 0) return false;
  if ((int)s.stg_cnt[i] + n > s.cl) {
    sink_spill(s, i, list, true);
    spilled = true;
    take = mine && key > s.st_key[i];
    tm = __ballot(take);
    n = __popcll(tm);
  }
  const int at = (int)s.stg_cnt[i];
  if (take) s.stg[(size_t)i * s.cl + at + __popcll(tm & ((1ull << s.lane) - 1ull))] = key;
  s.stg_cnt[i] = (uint32_t)(at + n);
  wave_sync_lds();
  return spilled;
}

// End of the stream: spill what is staged, cut lists longer than k to their
// k best (sorting every list when `sort_all`), and publish per list its
// length (kSortedFlag when sorted), best key (~0 when unknown, 0 when empty)
// and k-th key (0 unless it holds k sorted keys).
__device__ inline void sink_publish(const CandSink &s, int i, uint64_t *list, bool sort_all,
                                    uint32_t *lcnt, uint64_t *lfirst, uint64_t *lkth) {
  if (s.stg_cnt[i] > 0) sink_spill(s, i, list);
  const int cnt = (int)s.st_cnt[i];
  uint64_t first = (cnt == 0) ? 0ull : ~0ull;
  uint64_t kth = 0ull;
  uint32_t flag = 0u;
  if (cnt > s.k || (sort_all && cnt > 0)) {
    __threadfence_block();
    const int keep = cnt < s.k ? cnt : s.k;
    if (cnt <= kWaveRankMax) {
      for (int e = s.lane; e < cnt; e += kWaveSize) s.scr[e] = list[e];
      wave_sync_lds();
      const RankEnds r = wave_rank_top(s.scr, cnt, list, keep, s.lane);
      first = r.first;
      kth = (keep == s.k) ? r.last : 0ull;
    } else {
      int n = 2;
      while (n < cnt) n <<= 1;
      for (int e = s.lane; e < n; e += kWaveSize) s.scr[e] = (e < cnt) ? list[e] : 0ull;
      wave_sync_lds();
      wave_bitonic_desc(s.scr, n, s.lane);
      for (int e = s.lane; e < keep; e += kWaveSize) list[e] = s.scr[e];
      first = s.scr[0];
      kth = (keep == s.k) ? s.scr[s.k - 1] : 0ull;
    }
    flag = kSortedFlag;
    s.st_cnt[i] = (uint32_t)keep;
    wave_sync_lds();
  }
  if (s.lane == 0) {
    *lcnt = s.st_cnt[i] | flag | ((cnt == 1) ? kSortedFlag : 0u);
    *lfirst = first;
    *lkth = kth;
  }
}

}  // namespace dresd
