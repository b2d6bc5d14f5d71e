// Host runtime behind the C ABI in include/dresd.h: argument checks, the
// one-time key layout, workspace management and the per-search launch plan
// (sampled threshold passes, main scan, merge + gather).
#include <algorithm>
#include <map>
#include <mutex>
#include <new>
#include <string>
#include <utility>
#include <vector>

#include "dresd.h"
#include <hip/hip_ext.h>
#include <math.h>

#include "dresd_internal.h"
#include "dresd_ops.h"

using namespace dresd;

// Fixed device scratch of the allocation-free search (dresd_search_noalloc):
// one copy per device, held until the process ends.  In host code `scratch`
// names a host-side stand-in, never the device array: host code uses only
// the per-device address that hipGetSymbolAddress returns (scratch_address).
static constexpr size_t kScratchBytes = (size_t)DRESD_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

struct dresd_index {
  int device = 0;
  int64_t N = 0;
  int32_t d = 0, L = 0, dtype = 0;
  int KB = 0;          // 1 KiB blocks per tile
  int64_t T = 0;       // tiles
  void *data = nullptr;
  int32_t *cont = nullptr;
  int32_t *ftok = nullptr;  // first token of each row's value [T * 16] (filtered search)
  int cus = 0;
  size_t lds_max = 0;
  // workspaces, one per stream the index is searched on (searches on
  // different streams may overlap); buffers they outgrew stay allocated
  // until destroy (a captured graph may still use them)
  std::map<hipStream_t, std::pair<unsigned char *, size_t>> ws;
  std::vector<void *> retired;
  // measurement
  bool prof = false;
  std::vector<hipEvent_t> ev_free;
  std::vector<hipEvent_t> ev_scan, ev_all;  // start/stop pairs
  std::vector<std::pair<const void *, size_t>> occ_key;
  std::vector<int> occ_val;
};

namespace {

thread_local std::string g_err;

dresd_status fail(dresd_status s, const std::string &msg) {
  g_err = msg;
  return s;
}

#define DRESD_HIP(call)                                                              \
  do {                                                                               \
    hipError_t e_ = (call);                                                          \
    if (e_ != hipSuccess) return fail(DRESD_EDEVICE, std::string(#call) + ": " + hipGetErrorString(e_)); \
  } while (0)

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Every device allocation of the library goes through here.  Test hook: with
// DRESD_FAIL_ALLOC_AT=n in the environment, the n-th allocation counted since
// the variable last changed fails as out of memory without allocating, so
// that each allocation-failure path can be driven on purpose.
hipError_t dev_alloc(void **ptr, size_t bytes) {
  static std::mutex mu;
  static std::string armed;
  static long seen = 0;
  {
    std::lock_guard<std::mutex> lock(mu);
    const char *s = getenv("DRESD_FAIL_ALLOC_AT");
    if (!s || !*s) {
      armed.clear();
    } else {
      if (armed != s) {
        armed = s;
        seen = 0;
      }
      const long n = strtol(s, nullptr, 10);
      if (n > 0 && ++seen == n) {
        *ptr = nullptr;
        return hipErrorOutOfMemory;
      }
    }
  }
  return hipMalloc(ptr, bytes);
}

// A buffer may only grow outside stream capture: growing allocates and
// synchronises, which a capture cannot record.
bool capturing(hipStream_t st) {
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(st, &cs) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  return cs != hipStreamCaptureStatusNone;
}

// Device address of `scratch` on each device, resolved once per device with
// that device current (at index creation, or at the first allocation-free
// search on the device).
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
unsigned char *g_scratch_addr[kMaxDevices] = {};

dresd_status scratch_address(int dev, unsigned char **out) {
  if (dev < 0 || dev >= kMaxDevices) return fail(DRESD_EUNSUPPORTED, "device ordinal too large");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_addr[dev]) {
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess || cur != dev)
      return fail(DRESD_EDEVICE, "the index's device must be current");
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      (void)hipGetLastError();
      return fail(DRESD_EDEVICE, std::string("hipGetSymbolAddress(scratch): ") +
                                     hipGetErrorString(e));
    }
    g_scratch_addr[dev] = static_cast<unsigned char *>(p);
  }
  *out = g_scratch_addr[dev];
  return DRESD_OK;
}

int next_pow2(int x) {
  int n = 1;
  while (n < x) n <<= 1;
  return n;
}

// Dimensions per 1 KiB block: 16 lanes' rows x 4 lane groups x (8 | 4) dims.
int block_dims(int dtype) { return dtype == kF32 ? 16 : 32; }

// Queries [b0, b0 + nb) of the batch, scanned by one launch as ng query
// groups (ng > 1 only for the single-tile scan).
struct Group {
  int b0, nb, ng;
};

constexpr size_t kMaxGroup = 256;  // queries per launch: 16 query tiles x 16 columns
constexpr int kMaxScanWgPerCu = 4;
// One workgroup (4 waves, one per SIMD) per CU where it measured faster:
// each wave (or workgroup) streams one contiguous range, and fewer, longer
// streams keep HBM rows open longer (single-tile scan with one query tile on
// 1M x 4096, 10M x 256 and 33.5M x 128 keys at B = 1: +1.5-3.5%; shared-key
// scan on 4M x 1024 keys at B = 64-256: +3%).  Scans whose per-block work is
// larger need the extra waves to hide latency.
constexpr int kMaxTileWgPerCu = 1;
// Query groups of the single-tile scan served by one launch: one per XCD
// for each key range, so the range is read from HBM about once and its
// re-reads come from that XCD's L2.
constexpr int kGroupsPerLaunch = 8;

struct Plan {
  int terms = 1, qpt = 16, qt = 1;  // columns per query, queries per tile, tiles
  bool mq = false;                  // shared-key scan (queries in registers)
  int nwq = 4;                      // shared-key scan: waves per workgroup
  bool tc = false;                  // tiled contraction (queries and keys through LDS)
  // tiled contraction: key tiles per wave and key groups of waves per pass
  // kind, query groups of waves (waves per workgroup: nk * nq)
  int tpw_main = 4, tpw_sample = 1;
  int nk_main = 4, nk_sample = 4, nq = 1;
  int bmax = 0;                 // queries per group
  int bl = 0;                   // queries per launch (several groups)
  int B = 0, nl = 0;            // batch, launches (launch i: group_of(pl, i))
  int C = 0;                    // per-wave list capacity
  int CL = 0;                   // per-query LDS stage
  int64_t strides[3] = {0, 0, 0};  // sampled passes, sparsest first
  int spec[3] = {0, 0, 0};         // rank of the speculative key each pass hands the next (0: none)
  int npass = 0;                   // sampled passes used
  ScanKernel kmain = nullptr, ksample = nullptr;
  size_t lds = 0, lds_s = 0;    // LDS bytes of the main and the sampled scans
  int wg_max = 0;               // resident workgroups of the scan kernels
  int G_max = 0;
  int64_t spill_cap = 0;        // merge candidates per query beyond its LDS cache
  bool sort_lists = false;
  bool filt = false;            // next-token-filtered search
  size_t off_tau = 0, off_lcnt = 0, off_lkth = 0, off_lfirst = 0, off_lists = 0, off_spill = 0;
  size_t off_qop = 0;               // shared-key scan: query operands of a group
  size_t bytes = 0;
};

// Threads per workgroup of a plan's main or sampled scan.
int threads_of(const Plan &pl, bool main_pass) {
  if (pl.mq) return pl.nwq * kWaveSize;
  if (!pl.tc) return kScanThreads;
  return (main_pass ? pl.nk_main : pl.nk_sample) * pl.nq * kWaveSize;
}

// Launch i of a plan: queries [B i / nl, B (i + 1) / nl), split into groups
// of at most bmax queries.
Group group_of(const Plan &pl, int i) {
  const int b0 = (int)((int64_t)pl.B * i / pl.nl), b1 = (int)((int64_t)pl.B * (i + 1) / pl.nl);
  return {b0, b1 - b0, (int)ceil_div(b1 - b0, pl.bmax)};
}

// Single-tile scan: query operand | zero chunk | candidate region per wave.
size_t scan_lds(int ncols, int KB, int nq, int cl, int C) {
  return (size_t)ncols * KB * 64 + 16 + scan_ntok_bytes(nq) + (size_t)4 * scan_wave_bytes(nq, cl, C) +
         (size_t)4 * kScanFtokBytes;
}

// Per-query LDS stage in front of each HBM list: larger when few queries
// share the wave.  One tile can pass all 16 of its rows for a query at once
// (after a spill has emptied the stage), so the stage holds at least a tile.
int stage_cap(int nq) { return nq >= 16 ? kTileRows : 2 * kTileRows; }

// Resident workgroups per CU of a scan kernel at an LDS size, cached per
// index (not cached with `keep` false: the allocation-free search adds
// nothing to the host-side cache).
int occupancy(dresd_index *ix, ScanKernel k, size_t lds, bool keep = true,
              int threads = kScanThreads) {
  for (size_t i = 0; i < ix->occ_key.size(); ++i)
    if (ix->occ_key[i].first == (const void *)k && ix->occ_key[i].second == lds) return ix->occ_val[i];
  int nb = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, (const void *)k, threads, lds) !=
      hipSuccess) {
    (void)hipGetLastError();
    nb = 1;
  }
  nb = std::max(nb, 1);
  if (keep) {
    ix->occ_key.emplace_back((const void *)k, lds);
    ix->occ_val.push_back(nb);
  }
  return nb;
}

dresd_status validate_search(const dresd_index *ix, int32_t B, int32_t k) {
  if (!ix) return fail(DRESD_EINVAL, "index is NULL");
  if (B < 0) return fail(DRESD_EINVAL, "B must be >= 0");
  if (k < 1 || k > DRESD_K_MAX) return fail(DRESD_EINVAL, "k must be in [1, DRESD_K_MAX]");
  if ((int64_t)k > ix->N) return fail(DRESD_EINVAL, "k exceeds the number of keys");
  return DRESD_OK;
}

// Rank j of the key a sampled pass hands the next, denser pass as its
// starting threshold.  The denser pass visits every tile of this one and
// r - 1 others in each stretch of r, so each of its k best keys lies in this
// pass's sample with probability 1/r; it finds fewer than k keys at or above
// this sample's j-th best only if at least j of them do, which happens with
// probability P[Binomial(k, 1/r) >= j].  The smallest j that keeps this at
// most 1e-3 is taken.  When it happens the pass falls back to the exact
// bound it would have started from, so results never depend on the choice.
int spec_rank(int k, int64_t r) {
  const double p = 1.0 / (double)r, q = 1.0 - p;
  double pmf = 1.0;  // P[X = 0] = q^k
  for (int i = 0; i < k; ++i) pmf *= q;
  double below = 0.0;  // P[X < j]
  for (int j = 1; j <= k; ++j) {
    below += pmf;                                    // adds P[X = j - 1]
    if (1.0 - below <= 1e-3) return j;
    pmf *= (double)(k - j + 1) / (double)j * p / q;  // P[X = j]
  }
  return k;
}

dresd_status make_plan(dresd_index *ix, int B, int k, Plan &pl, bool filt = false,
                       bool keep_cache = true, bool tc32 = true) {
  pl = Plan();
  pl.filt = filt;
  // The query enters the matrix cores as three 16-bit parts that sum to it
  // exactly (four columns per query) for batches that fit one 16-column tile
  // that way (B <= 4); larger batches take fewer columns: bf16 keys two
  // parts (high + rounded remainder, within 2^-17 relative of the query),
  // f16 keys the query rounded once to f16.
  if (ix->dtype == kBF16) pl.terms = (B <= 4) ? 4 : 2;
  else if (ix->dtype == kF16) pl.terms = (B <= 4) ? 4 : 1;
  else pl.terms = 1;
  pl.qpt = 16 / pl.terms;
  pl.C = next_pow2(std::max(k + 64, 128));
  const int qt_all = (int)ceil_div((int64_t)B * pl.terms, 16);  // query tiles of the batch
  const bool mq_type = (ix->dtype == kF16 && pl.terms == 1) || ix->dtype == kBF16;
  const bool mq_kb = ix->KB == 4 || ix->KB == 8 || ix->KB == 16 || ix->KB == 32;
  // Keys wider than the shared-key scan can hold the queries for (more than
  // 32 blocks per key tile) at batches of two or more query tiles, and
  // 32-block keys at batches past the four query tiles one shared-key launch
  // holds: the tiled contraction streams both operands through LDS.  One
  // query group of waves serves 4 query tiles (8 for bf16: 64 queries);
  // larger batches take 2 or 4 query groups (up to 256 f16 or 128 bf16
  // queries per launch), fewer where the lists leave too little LDS.
  const bool tc_kb = ix->KB > 32 || (tc32 && ix->KB == 32 && qt_all > 4);
  if (mq_type && tc_kb && qt_all >= 2 && pl.terms < 4) {
    const bool bf = ix->dtype == kBF16;
    const int qtw = (bf && qt_all > 4) ? 8 : 4;
    const int nqw = qtw * pl.qpt;         // queries per wave
    const int np = qtw * (4 / pl.terms);  // score slots per lane
    int nq = 1;
    while (nq < (bf ? 2 : 4) && nq * qtw < qt_all) nq <<= 1;
    struct TcShape {
      int tpw, nk, st;
    };
    // main-pass shapes, then sampled-pass shapes, in order of preference; one
    // query group: 8 waves over panels of 32 key tiles (one query read per 32
    // tiles) where that kernel exists and fits, else 4 waves over 16 tiles;
    // two or four query groups: 8 waves over 16-tile panels, with a 4-stage
    // ring (operand prefetch) where the lists leave room for it
    static const std::vector<TcShape> main1 = {{4, 8, 3}, {4, 4, 5}, {4, 4, 3}},
                                      samp1 = {{1, 4, 8}, {1, 4, 4}},
                                      main2 = {{4, 4, 4}, {4, 4, 3}}, samp2 = {{2, 4, 4}},
                                      main4 = {{8, 2, 4}, {8, 2, 3}}, samp4 = {{4, 2, 4}};
    for (; nq >= 1 && !pl.tc; nq >>= 1) {
      const auto &ms = nq == 4 ? main4 : nq == 2 ? main2 : main1;
      const auto &ss = nq == 4 ? samp4 : nq == 2 ? samp2 : samp1;
      const TcShape *m = nullptr, *smp = nullptr;
      for (const auto &c : ms)
        if (!m && scan_tc_kernel(ix->dtype, qtw, c.tpw, c.nk, nq, c.st, true, filt) &&
            scan_tc_lds_bytes(qtw, c.tpw, c.nk, nq, c.st, nqw, pl.C, np, filt) <= ix->lds_max)
          m = &c;
      for (const auto &c : ss)
        if (!smp && scan_tc_kernel(ix->dtype, qtw, c.tpw, c.nk, nq, c.st, false, filt) &&
            scan_tc_lds_bytes(qtw, c.tpw, c.nk, nq, c.st, nqw, pl.C, np, filt) <= ix->lds_max)
          smp = &c;
      if (!m || !smp) continue;
      pl.tc = true;
      pl.nq = nq;
      pl.tpw_main = m->tpw;
      pl.nk_main = m->nk;
      pl.tpw_sample = smp->tpw;
      pl.nk_sample = smp->nk;
      pl.qt = nq * qtw;
      pl.bmax = std::min(B, nq * nqw);
      pl.CL = 0;
      pl.kmain = scan_tc_kernel(ix->dtype, qtw, m->tpw, m->nk, nq, m->st, true, filt);
      pl.ksample = scan_tc_kernel(ix->dtype, qtw, smp->tpw, smp->nk, nq, smp->st, false, filt);
      pl.lds = scan_tc_lds_bytes(qtw, m->tpw, m->nk, nq, m->st, nqw, pl.C, np, filt);
      pl.lds_s = scan_tc_lds_bytes(qtw, smp->tpw, smp->nk, nq, smp->st, nqw, pl.C, np, filt);
    }
  }
  if (pl.tc) {
  } else if (mq_type && mq_kb && (qt_all >= 2 || pl.terms < 4)) {
    // Several query tiles, or one of one- or two-column queries (four or
    // two scores per lane per key tile): queries stationary in registers,
    // keys shared
    // through LDS.  Each of the 4 waves holds qtw tiles (operands for all
    // KB blocks: qtw * KB <= 32 chunks of 16 bytes); one to three tiles are
    // padded to four.  The single-tile scan re-reads every query operand
    // from LDS per block and runs such batches 2-3x slower.
    pl.mq = true;
    int qtw = 1;
    while (qtw < 4 && 4 * qtw < qt_all && 2 * qtw * ix->KB <= 32) qtw <<= 1;
    pl.qt = 4 * qtw;
    pl.nwq = 4;
    int stages = 0;
    // 8-block key tiles (256 dims) at 2-4 query tiles: one wave per
    // workgroup holds the whole batch (32 chunks of 16 bytes), so no wave
    // waits at a barrier for another's candidates (measured, 10M x 256:
    // main pass 0.776 -> 0.749 ms at B = 64, 0.759 -> 0.740 ms at B = 32;
    // at 128 dims and 64-128 queries it was 15-20% slower: four waves per
    // CU leave too little to overlap).
    if (ix->KB == 8 && qt_all >= 2 && qt_all * ix->KB <= 32 &&
        scan_mq_kernel(ix->dtype, 4, ix->KB, true, filt, &stages, 1)) {
      qtw = 4;
      pl.qt = qtw;
      pl.nwq = 1;
    }
    pl.bmax = std::min(B, pl.qt * pl.qpt);
    pl.kmain = scan_mq_kernel(ix->dtype, qtw, ix->KB, true, filt, &stages, pl.nwq);
    pl.ksample = scan_mq_kernel(ix->dtype, qtw, ix->KB, false, filt, &stages, pl.nwq);
    pl.CL = 0;
    pl.lds = scan_mq_lds_bytes(stages, qtw * pl.qpt, pl.C, pl.nwq) +
             (filt ? (size_t)pl.nwq * scan_mq_filter_bytes(stages, qtw * (4 / pl.terms)) : 0);
  } else {
    // Largest group (power-of-two number of query tiles, at most 16) whose
    // query operand and per-wave state fit in the workgroup's LDS.
    int qt = 16;
    for (;; qt >>= 1) {
      int nb = std::min(B, qt * pl.qpt);
      size_t lds = scan_lds(nb * pl.terms, ix->KB, qt * pl.qpt, stage_cap(qt * pl.qpt), pl.C);
      if (lds <= ix->lds_max || qt == 1) break;
    }
    int bmax = std::min(B, qt * pl.qpt);
    pl.CL = stage_cap(qt * pl.qpt);
    // the smallest group (one query) must fit; larger batches shrink to fit
    if (scan_lds(pl.terms, ix->KB, pl.qpt, pl.CL, pl.C) > ix->lds_max)
      return fail(DRESD_EUNSUPPORTED, "query tile does not fit in LDS for this d and k");
    // shrink bmax until it fits (qt == 1 case)
    while (bmax > 1 &&
           scan_lds(bmax * pl.terms, ix->KB, qt * pl.qpt, pl.CL, pl.C) > ix->lds_max)
      --bmax;
    // smallest qt that holds bmax
    int need = (int)ceil_div((int64_t)bmax * pl.terms, 16);
    pl.qt = 1;
    while (pl.qt < need) pl.qt <<= 1;
    pl.bmax = bmax;
    pl.kmain = scan_kernel(ix->dtype, pl.qt, pl.terms, true);
    pl.ksample = scan_kernel(ix->dtype, pl.qt, pl.terms, false);
    pl.CL = stage_cap(pl.qt * pl.qpt);
    pl.lds = scan_lds(bmax * pl.terms, ix->KB, pl.qt * pl.qpt, pl.CL, pl.C);
  }
  const int bmax = pl.bmax;
  const int ngr = (int)ceil_div(B, bmax);
  // The single-tile scan serves several groups per launch; launch sizes
  // differ by at most one query and each splits into groups of <= bmax.
  const int per = (pl.mq || pl.tc)
                      ? 1
                      : std::max(1, std::min({ngr, kGroupsPerLaunch, (int)(kMaxGroup / bmax)}));
  pl.B = B;
  pl.nl = (int)ceil_div(ngr, per);
  pl.bl = (int)ceil_div(B, pl.nl);  // launch sizes differ by at most one query
  if (per > 1 && pl.qt == 1) {
    pl.kmain = scan_kernel(ix->dtype, pl.qt, pl.terms, true, true);
    pl.ksample = scan_kernel(ix->dtype, pl.qt, pl.terms, false, true);
  }
  if (!pl.kmain || !pl.ksample) return fail(DRESD_EUNSUPPORTED, "no scan kernel for this shape");
  if (!pl.tc) pl.lds_s = pl.lds;
  if (pl.lds > ix->lds_max) return fail(DRESD_EUNSUPPORTED, "scan state does not fit in LDS");
  int occ = std::min(occupancy(ix, pl.kmain, pl.lds, keep_cache, threads_of(pl, true)),
                     occupancy(ix, pl.ksample, pl.lds_s, keep_cache, threads_of(pl, false)));
  // At most four workgroups per CU (few enough lists for the merge to keep
  // their best keys in LDS); one where fewer, longer HBM streams measured
  // faster: the single-tile scan with one query tile, and the shared-key
  // scan over 32-block (1 KiB-row) key tiles.
  const bool one_per_cu = pl.tc || (pl.mq ? ix->KB >= 32 : pl.qt == 1);
  pl.wg_max = ix->cus * std::min(occ, one_per_cu ? kMaxTileWgPerCu : kMaxScanWgPerCu);
  // lists per query from each workgroup (at most kMergeLists in all): one per
  // wave, one for the shared-key scan, and one per key group of waves for
  // the tiled contraction (of the pass kind with more)
  const int lists_per_wg = pl.mq ? 1 : pl.tc ? std::max(pl.nk_main, pl.nk_sample)
                                             : kScanThreads / kWaveSize;
  pl.wg_max = std::min(pl.wg_max, kMergeLists / lists_per_wg);
  pl.G_max = pl.wg_max * lists_per_wg;
  // Small batches (B <= 8): every wave keeps its own running top-k and sorts
  // it at the end; the merge then prunes with the best per-wave k-th key.
  // Batches past 8 queries, and smaller ones with k >= 16 and B * k >= 64
  // (query, rank) pairs (measured: +5% at 5-8 queries, k = 16; +28-60% at
  // 4-8 queries, k = 100; fewer (query, rank) pairs leave the main pass few
  // candidates anyway), first set per-query thresholds from sampled passes
  // over tiles
  // j*P, sparsest first (kept when they hold at least 4k rows and are at
  // most a quarter of the tiles).  A pass at stride P leaves about P*k
  // candidates per query for the next one, so batches with many
  // (query, rank) pairs add a denser level: its extra sampled scan costs less
  // than the candidates it removes from the full pass.  The single-tile
  // scan, whose waves cut their lists early on their own, does best with
  // one pass at stride 256 (measured: 1.5-4% faster than 4096, 64 at
  // 1-4 queries and at d = 4096 groups; the shared-key scan is faster with
  // the two levels).
  pl.sort_lists = B <= 8;
  if (!pl.sort_lists || (k >= 16 && (int64_t)B * k >= 64)) {
    const bool dense = (int64_t)B * k >= 8192;
    // The tiled contraction's passes take about as long at stride 64 as
    // at 256 (a K loop over every column per panel, whatever the panel
    // count): one pass, at the sparsest of 64, 16 and 4 that lists enough
    // tiles.
    const std::vector<int64_t> ladder =
        pl.tc    ? std::vector<int64_t>{64, 16, 4}
        : dense  ? std::vector<int64_t>{4096, 256, 16}
        : pl.mq  ? std::vector<int64_t>{4096, 64}
                 : std::vector<int64_t>{256};
    for (int64_t P : ladder) {
      int64_t nv = ceil_div(ix->T, P);
      // the tiled contraction's sampled pass lists one key per tile and query
      const int64_t rows = pl.tc ? nv : nv * kTileRows;
      if (rows >= 4 * (int64_t)k && ix->T >= 4 * P) {
        pl.strides[pl.npass++] = P;
        if (pl.tc) break;
      }
    }
    for (int i = 0; i + 1 < pl.npass; ++i)
      pl.spec[i] = spec_rank(k, pl.strides[i] / pl.strides[i + 1]);
  }
  // Lists end with at most k keys each, so a query never has more than
  // G_max * k merge candidates.
  pl.spill_cap = std::max<int64_t>(0, (int64_t)pl.G_max * k - kMergeCap);
  size_t nb = (size_t)pl.bl;
  auto up = [](size_t x) { return (x + 255) / 256 * 256; };
  pl.off_tau = 0;  // [2 levels][kMaxGroup] bounds, then [2 levels][kMaxGroup] speculative keys
  pl.off_lcnt = up(4 * kMaxGroup * 8);
  pl.off_lkth = pl.off_lcnt + up(nb * pl.G_max * 4);
  pl.off_lfirst = pl.off_lkth + up(nb * pl.G_max * 8);
  pl.off_lists = pl.off_lfirst + up(nb * pl.G_max * 8);
  pl.off_spill = pl.off_lists + up(nb * pl.G_max * pl.C * 8);
  pl.off_qop = pl.off_spill + up(nb * (size_t)std::max<int64_t>(1, pl.spill_cap) * 8);
  pl.bytes = pl.off_qop + ((pl.mq || pl.tc) ? up((size_t)pl.qt * ix->KB * kBlockBytes) : 0);
  return DRESD_OK;
}

// Workgroups per query group of one scan pass over nvisit tiles (the
// launch has gr.ng times as many).  Several groups: each gets a multiple of
// 8 (one key range per XCD slot) and together they fit the resident grid,
// so the readers of a range run at the same time.
int64_t pass_wgs(const Plan &pl, const Group &gr, int64_t nvisit, bool main_pass = true) {
  const int wpg = kScanThreads / kWaveSize;
  // tiled contraction: whole panels of nk * tpw tiles
  const int per_wg = pl.tc ? (main_pass ? pl.nk_main * pl.tpw_main : pl.nk_sample * pl.tpw_sample)
                   : pl.mq ? 1 : wpg;
  int64_t wgs = std::min<int64_t>(pl.wg_max, ceil_div(nvisit, per_wg));
  if (gr.ng > 1) wgs = std::min<int64_t>(wgs, std::max<int64_t>(8, pl.wg_max / gr.ng / 8 * 8));
  return wgs;
}

// The index's workspace for stream st, grown to at least `bytes`.
dresd_status ensure_workspace(dresd_index *ix, size_t bytes, hipStream_t st,
                              unsigned char **out) {
  auto &w = ix->ws[st];
  *out = w.first;
  if (w.second >= bytes) return DRESD_OK;
  if (capturing(st))
    return fail(DRESD_EUNSUPPORTED,
                "the search needs a larger workspace while its stream is being captured; run one "
                "uncaptured call of this shape first");
  void *p = nullptr;
  if (dev_alloc(&p, bytes) != hipSuccess) {
    (void)hipGetLastError();
    return fail(DRESD_ENOMEM, "workspace allocation of " + std::to_string(bytes) + " bytes failed");
  }
  // Every region is written before it is read in each search; clearing it
  // once keeps a fresh workspace deterministic to inspect.  The clear is
  // ordered on the search's own stream (not capturing: growth is refused
  // then), ahead of the kernels that use the workspace.
  if (hipMemsetAsync(p, 0, bytes, st) != hipSuccess) {
    (void)hipFree(p);
    return fail(DRESD_EDEVICE, "workspace clear failed");
  }
  // The outgrown buffer is kept until the index is destroyed: a graph
  // captured from an earlier search may still replay on it.
  if (w.first) ix->retired.push_back(w.first);
  w = {static_cast<unsigned char *>(p), bytes};
  *out = w.first;
  return DRESD_OK;
}

// Library buffers kept until the process ends (the transform's partial
// sums, the k-means sums), one per (device, stream): calls on different
// streams never share one, and calls on one stream are ordered by it.  One
// grows (allocating synchronously) when a call needs more; the buffer it
// outgrows is kept as well, because a graph captured from an earlier call
// may still replay on it.
struct DeviceBuffers {
  std::mutex mu;
  std::map<std::pair<int, hipStream_t>, std::pair<void *, size_t>> cur;
  std::vector<void *> retired;
};

dresd_status device_buffer(DeviceBuffers &db, int dev, size_t need, hipStream_t st,
                           const char *what, void **out) {
  std::lock_guard<std::mutex> lock(db.mu);
  auto &c = db.cur[{dev, st}];
  if (c.second < need) {
    if (capturing(st))
      return fail(DRESD_EUNSUPPORTED, std::string(what) +
                                          " must grow while the stream is being captured; run one "
                                          "uncaptured call of this shape first");
    void *b = nullptr;
    if (dev_alloc(&b, need) != hipSuccess) {
      (void)hipGetLastError();
      return fail(DRESD_ENOMEM, std::string(what) + " allocation failed");
    }
    if (c.first) db.retired.push_back(c.first);
    c = {b, need};
  }
  *out = c.first;
  return DRESD_OK;
}

hipEvent_t take_event(dresd_index *ix) {
  if (!ix->ev_free.empty()) {
    hipEvent_t e = ix->ev_free.back();
    ix->ev_free.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// Kernel launches of one search.  Profiling events are tied to kernels'
// own dispatches (their begin and end timestamps) instead of being recorded
// as packets of their own, which would leave the device idle between
// kernels: `first` marks the begin of the next launch (and is cleared),
// a launch's own start/stop pair its duration, `last` the end of the launch
// that the caller flags as the search's last.
struct Launcher {
  hipStream_t st;
  hipEvent_t first = nullptr;       // pending: begin of the next launch
  hipEvent_t first_used = nullptr;  // the event that marked it
  hipEvent_t last = nullptr;        // end of the flagged launch
  hipError_t operator()(const void *f, dim3 grid, dim3 block, void **args, size_t lds,
                        hipEvent_t start = nullptr, hipEvent_t stop = nullptr,
                        bool is_last = false) {
    if (first) {
      if (!start) start = first;  // else the launch's own start marks both
      first_used = start;
      first = nullptr;
    }
    if (is_last && last) stop = stop ? stop : last;
    if (!start && !stop) return hipLaunchKernel(f, grid, block, args, lds, st);
    return hipExtLaunchKernel(f, grid, block, args, lds, st, start, stop, 0);
  }
};

// Events of an index's profile, each once (a pair may share its start with
// a scan's pair).
std::vector<hipEvent_t> profile_events(const dresd_index *ix);

dresd_status index_build(const void *embeddings, const int32_t *continuations, int64_t N,
                         int32_t d, int32_t L, int32_t dtype, const uint32_t *slot_row,
                         int64_t T, dresd_stream stream, dresd_index **out);

// One search; next_tok (device [B]) selects the next-token-filtered form.
// `outer` (optional) carries the timing events of an enclosing search.
dresd_status search_impl(dresd_index *ix, const float *queries, const int32_t *next_tok, int32_t B,
                         int32_t k, int64_t *idx, float *score, int32_t *tokens,
                         dresd_stream stream, Launcher *outer = nullptr,
                         unsigned char *fixed_ws = nullptr, size_t fixed_bytes = 0);

}  // namespace

extern "C" {

const char *dresd_last_error(void) { return g_err.c_str(); }

dresd_status dresd_index_create(const void *embeddings, const int32_t *continuations, int64_t N,
                                int32_t d, int32_t L, int32_t dtype, dresd_stream stream,
                                dresd_index **out) {
  if (!embeddings || !continuations || !out) return fail(DRESD_EINVAL, "NULL pointer argument");
  if (N < 1 || N > DRESD_N_MAX) return fail(DRESD_EINVAL, "N out of range");
  if (d < 1 || d > 16384) return fail(DRESD_EINVAL, "d out of range");
  if (L < 1 || L > 4096) return fail(DRESD_EINVAL, "L out of range");
  if (dtype < DRESD_F32 || dtype > DRESD_BF16) return fail(DRESD_EINVAL, "unknown dtype");
  return index_build(embeddings, continuations, N, d, L, dtype, nullptr, 0, stream, out);
}

}  // extern "C"

namespace {
// Build an index (arguments already checked).  With a slot table (device
// [T * 16], the row of each slot or kPadRow) the keys are laid out in slot
// order over T tiles -- the partitioned layout -- and no first-token column
// is built; without one, slot = row.
dresd_status index_build(const void *embeddings, const int32_t *continuations, int64_t N,
                         int32_t d, int32_t L, int32_t dtype, const uint32_t *slot_row,
                         int64_t T, dresd_stream stream, dresd_index **out) {
  hipStream_t st = static_cast<hipStream_t>(stream);
  dresd_index *ix = new (std::nothrow) dresd_index();
  if (!ix) return fail(DRESD_ENOMEM, "host allocation failed");
  auto cleanup = [&](dresd_status s) {
    if (ix->data) (void)hipFree(ix->data);
    if (ix->cont) (void)hipFree(ix->cont);
    if (ix->ftok) (void)hipFree(ix->ftok);
    delete ix;
    return s;
  };
  if (hipGetDevice(&ix->device) != hipSuccess) return cleanup(fail(DRESD_EDEVICE, "hipGetDevice failed"));
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, ix->device) != hipSuccess)
    return cleanup(fail(DRESD_EDEVICE, "hipGetDeviceProperties failed"));
  ix->cus = prop.multiProcessorCount;
  ix->lds_max = prop.sharedMemPerBlock;
  {  // set-up of the allocation-free search on this device
    unsigned char *sc = nullptr;
    const dresd_status ss = scratch_address(ix->device, &sc);
    if (ss != DRESD_OK) return cleanup(ss);
  }
  ix->N = N;
  ix->d = d;
  ix->L = L;
  ix->dtype = dtype;
  const int bd = block_dims(dtype);
  ix->KB = (int)ceil_div(d, bd);
  ix->T = slot_row ? T : ceil_div(N, kTileRows);
  const size_t data_bytes = (size_t)ix->T * ix->KB * kBlockBytes;
  const size_t cont_bytes = (size_t)N * L * sizeof(int32_t);
  if (dev_alloc(&ix->data, data_bytes) != hipSuccess) {
    (void)hipGetLastError();
    ix->data = nullptr;
    return cleanup(fail(DRESD_ENOMEM, "key storage allocation failed"));
  }
  if (dev_alloc((void **)&ix->cont, cont_bytes) != hipSuccess) {
    (void)hipGetLastError();
    ix->cont = nullptr;
    return cleanup(fail(DRESD_ENOMEM, "continuation storage allocation failed"));
  }
  const size_t ftok_bytes = (size_t)ix->T * kTileRows * sizeof(int32_t);
  if (!slot_row && dev_alloc((void **)&ix->ftok, ftok_bytes) != hipSuccess) {
    (void)hipGetLastError();
    ix->ftok = nullptr;
    return cleanup(fail(DRESD_ENOMEM, "first-token column allocation failed"));
  }
  // Raise the dynamic-LDS limit of every scan kernel to the device's.
  for (int v = 0; v < 3; ++v)
    for (int qtw : {1, 2, 4, 8})
      for (int kbt : {4, 8, 16, 32})
        for (int nwq : {1, 4})
          for (int mp = 0; mp < 4; ++mp) {
            int stages = 0;
            ScanKernel kf = scan_mq_kernel(v, qtw, kbt, (mp & 1) != 0, mp >= 2, &stages, nwq);
            if (kf)
              (void)hipFuncSetAttribute((const void *)kf,
                                        hipFuncAttributeMaxDynamicSharedMemorySize,
                                        (int)ix->lds_max);
          }
  for (int v = 0; v < 3; ++v)
    for (int qt : {1, 2, 4, 8, 16})
      for (int cpq : {1, 2, 4})
        for (int mp = 0; mp < 2; ++mp) {
          for (bool shared : {false, true}) {
            ScanKernel kf = scan_kernel(v, qt, cpq, mp != 0, shared);
            if (kf)
              (void)hipFuncSetAttribute((const void *)kf,
                                        hipFuncAttributeMaxDynamicSharedMemorySize,
                                        (int)ix->lds_max);
          }
        }
  for (int v = 0; v < 3; ++v)
    for (int qtw : {4, 8})
      for (int tpw : {1, 2, 4, 8})
        for (int nk : {2, 4, 8})
          for (int nq : {1, 2, 4})
            for (int st : {3, 4, 5, 8})
              for (int mp = 0; mp < 4; ++mp)
                if (ScanKernel kf =
                        scan_tc_kernel(v, qtw, tpw, nk, nq, st, (mp & 1) != 0, mp >= 2))
                  (void)hipFuncSetAttribute((const void *)kf,
                                            hipFuncAttributeMaxDynamicSharedMemorySize,
                                            (int)ix->lds_max);
  for (int v = 0; v < 3; ++v)
    if (ScanKernel kf = scan_parts_kernel(v))
      (void)hipFuncSetAttribute((const void *)kf, hipFuncAttributeMaxDynamicSharedMemorySize,
                                (int)ix->lds_max);
  (void)hipGetLastError();
  LayoutParams lp;
  lp.src = embeddings;
  lp.dst = ix->data;
  lp.slot_row = slot_row;
  lp.N = N;
  lp.chunks = (int64_t)ix->T * ix->KB * 64;
  lp.d = d;
  lp.KB = ix->KB;
  const int64_t blocks = std::min<int64_t>(ceil_div(lp.chunks, 256), (int64_t)ix->cus * 64);
  void *args[] = {&lp};
  hipError_t e = hipLaunchKernel(layout_kernel_ptr(dtype), dim3((unsigned)blocks), dim3(256), args,
                                 0, st);
  if (e == hipSuccess)
    e = hipMemcpyAsync(ix->cont, continuations, cont_bytes, hipMemcpyDeviceToDevice, st);
  // First-token column: value[i][0] for every row, zero past N.
  if (e == hipSuccess && ix->ftok)
    e = hipMemsetAsync(ix->ftok, 0, ftok_bytes, st);
  if (e == hipSuccess && ix->ftok)
    e = hipMemcpy2DAsync(ix->ftok, sizeof(int32_t), continuations, (size_t)L * sizeof(int32_t),
                         sizeof(int32_t), (size_t)N, hipMemcpyDeviceToDevice, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e != hipSuccess)
    return cleanup(fail(DRESD_EDEVICE, std::string("index build failed: ") + hipGetErrorString(e)));
  *out = ix;
  return DRESD_OK;
}
}  // namespace

extern "C" {

dresd_status dresd_index_info(const dresd_index *ix, int64_t *N, int32_t *d, int32_t *L,
                              int32_t *dtype) {
  if (!ix) return fail(DRESD_EINVAL, "index is NULL");
  if (N) *N = ix->N;
  if (d) *d = ix->d;
  if (L) *L = ix->L;
  if (dtype) *dtype = ix->dtype;
  return DRESD_OK;
}

void dresd_index_destroy(dresd_index *ix) {
  if (!ix) return;
  int cur = 0;
  (void)hipGetDevice(&cur);
  (void)hipSetDevice(ix->device);
  (void)hipDeviceSynchronize();
  if (ix->data) (void)hipFree(ix->data);
  if (ix->cont) (void)hipFree(ix->cont);
  if (ix->ftok) (void)hipFree(ix->ftok);
  for (auto &w : ix->ws)
    if (w.second.first) (void)hipFree(w.second.first);
  for (void *r : ix->retired) (void)hipFree(r);
  for (auto e : ix->ev_free) (void)hipEventDestroy(e);
  for (auto e : profile_events(ix)) (void)hipEventDestroy(e);
  (void)hipSetDevice(cur);
  delete ix;
}

dresd_status dresd_search_plan(const dresd_index *cix, int32_t B, int32_t k, int32_t *sample_passes,
                               int32_t *scan_waves, int64_t *workspace_bytes, int32_t *scan_kind,
                               int32_t *launches) {
  dresd_status s = validate_search(cix, B, k);
  if (s != DRESD_OK) return s;
  dresd_index *ix = const_cast<dresd_index *>(cix);
  if (sample_passes) *sample_passes = 0;
  if (scan_waves) *scan_waves = 0;
  if (workspace_bytes) *workspace_bytes = 0;
  if (scan_kind) *scan_kind = 0;
  if (launches) *launches = 0;
  if (B == 0) return DRESD_OK;
  Plan pl;
  s = make_plan(ix, B, k, pl);
  if (s != DRESD_OK) return s;
  const Group g0 = group_of(pl, 0);
  if (sample_passes) *sample_passes = (int32_t)pl.npass;
  if (scan_waves)
    *scan_waves = (int32_t)(pass_wgs(pl, g0, ix->T) * g0.ng * (threads_of(pl, true) / kWaveSize));
  if (workspace_bytes) *workspace_bytes = (int64_t)pl.bytes;
  if (scan_kind) *scan_kind = pl.tc ? 3 : pl.mq ? 1 : (g0.ng > 1 ? 2 : 0);
  if (launches) *launches = (int32_t)pl.nl;
  return DRESD_OK;
}

dresd_status dresd_search(dresd_index *ix, const float *queries, int32_t B, int32_t k,
                          int64_t *idx, float *score, int32_t *tokens, dresd_stream stream) {
  dresd_status s = validate_search(ix, B, k);
  if (s != DRESD_OK) return s;
  if (B > 0 && (!queries || !idx || !score)) return fail(DRESD_EINVAL, "NULL pointer argument");
  if (B == 0) return DRESD_OK;
  return search_impl(ix, queries, nullptr, B, k, idx, score, tokens, stream);
}

dresd_status dresd_search_filtered(dresd_index *ix, const float *queries, const int32_t *next_tok,
                                   int32_t B, int32_t k, int64_t *idx, float *score,
                                   int32_t *tokens, dresd_stream stream) {
  dresd_status s = validate_search(ix, B, k);
  if (s != DRESD_OK) return s;
  if (B > 0 && (!queries || !next_tok || !idx || !score))
    return fail(DRESD_EINVAL, "NULL pointer argument");
  if (B == 0) return DRESD_OK;
  return search_impl(ix, queries, next_tok, B, k, idx, score, tokens, stream);
}

dresd_status dresd_search_noalloc(dresd_index *ix, const float *queries, int32_t B, int32_t k,
                                  int64_t *idx, float *score, int32_t *tokens,
                                  dresd_stream stream) {
  dresd_status s = validate_search(ix, B, k);
  if (s != DRESD_OK) return s;
  if (B > 0 && (!queries || !idx || !score)) return fail(DRESD_EINVAL, "NULL pointer argument");
  if (B == 0) return DRESD_OK;
  unsigned char *sc = nullptr;
  s = scratch_address(ix->device, &sc);
  if (s != DRESD_OK) return s;
  return search_impl(ix, queries, nullptr, B, k, idx, score, tokens, stream, nullptr, sc,
                     kScratchBytes);
}

}  // extern "C"

namespace {
std::vector<hipEvent_t> profile_events(const dresd_index *ix) {
  std::vector<hipEvent_t> v(ix->ev_scan);
  v.insert(v.end(), ix->ev_all.begin(), ix->ev_all.end());
  std::sort(v.begin(), v.end());
  v.erase(std::unique(v.begin(), v.end()), v.end());
  return v;
}

dresd_status search_impl(dresd_index *ix, const float *queries, const int32_t *next_tok, int32_t B,
                         int32_t k, int64_t *idx, float *score, int32_t *tokens,
                         dresd_stream stream, Launcher *outer, unsigned char *fixed_ws,
                         size_t fixed_bytes) {
  dresd_status s = DRESD_OK;
  hipStream_t st = static_cast<hipStream_t>(stream);
  Launcher own;
  own.st = st;
  Launcher &launch = outer ? *outer : own;
  // With a fixed workspace of fixed_bytes (the allocation-free search)
  // nothing is allocated on the device or the host, and no profiling events
  // are taken.
  const bool fixed = fixed_ws != nullptr;
  Plan pl;
  s = make_plan(ix, B, k, pl, next_tok != nullptr, !fixed);
  if (s != DRESD_OK) return s;
  // A fixed workspace too small for the tiled contraction's lists (one per
  // query per key group of waves of each workgroup): 1,024-dim keys take the
  // shared-key scan instead (one list per query per workgroup, a launch per
  // 64 queries).
  if (fixed && pl.bytes > fixed_bytes && pl.tc && ix->KB == 32) {
    s = make_plan(ix, B, k, pl, next_tok != nullptr, false, false);
    if (s != DRESD_OK) return s;
  }
  unsigned char *ws = fixed_ws;
  if (fixed) {
    if (pl.bytes > fixed_bytes)
      return fail(DRESD_EINVAL, "this search needs " + std::to_string(pl.bytes) +
                                    " bytes of workspace, more than the " +
                                    std::to_string(fixed_bytes) +
                                    " bytes of the fixed scratch (use dresd_search)");
  } else {
    s = ensure_workspace(ix, pl.bytes, st, &ws);
    if (s != DRESD_OK) return s;
  }
  const bool prof = ix->prof && !fixed;
  uint64_t *tau = reinterpret_cast<uint64_t *>(ws + pl.off_tau);
  uint32_t *lcnt = reinterpret_cast<uint32_t *>(ws + pl.off_lcnt);
  uint64_t *lkth = reinterpret_cast<uint64_t *>(ws + pl.off_lkth);
  uint64_t *lfirst = reinterpret_cast<uint64_t *>(ws + pl.off_lfirst);
  uint64_t *lists = reinterpret_cast<uint64_t *>(ws + pl.off_lists);
  uint64_t *spill = reinterpret_cast<uint64_t *>(ws + pl.off_spill);

  hipEvent_t e_all0 = nullptr, e_all1 = nullptr;
  if (prof && !outer) {
    e_all0 = take_event(ix);
    e_all1 = take_event(ix);
    if (!e_all0 || !e_all1) return fail(DRESD_EDEVICE, "hipEventCreate failed");
    own.first = e_all0;
    own.last = e_all1;
  }
  for (int li = 0; li < pl.nl; ++li) {
    const Group gr = group_of(pl, li);
    ScanParams sp;
    sp.data = ix->data;
    sp.queries = queries + (size_t)gr.b0 * ix->d;
    sp.N = ix->N;
    sp.lists = lists;
    sp.lcnt = lcnt;
    sp.lkth = lkth;
    sp.lfirst = lfirst;
    sp.sort_lists = pl.sort_lists ? 1 : 0;
    sp.B = gr.nb;
    sp.d = ix->d;
    sp.KB = ix->KB;
    sp.k = k;
    sp.C = pl.C;
    sp.CL = pl.CL;
    sp.ftok = next_tok ? ix->ftok : nullptr;
    sp.next_tok = next_tok ? next_tok + gr.b0 : nullptr;
    sp.ngroups = gr.ng;
    sp.qop = nullptr;
    sp.slot_row = nullptr;
    sp.seg_off = sp.seg_tile = nullptr;
    sp.S = sp.wgq = 0;
    sp.probes64 = nullptr;
    sp.part_tile = nullptr;
    sp.seg_lds = sp.P = 0;
    if (pl.mq || pl.tc) {
      QopParams qp;
      qp.queries = sp.queries;
      qp.out = ws + pl.off_qop;
      qp.B = gr.nb;
      qp.d = ix->d;
      qp.KB = ix->KB;
      qp.ntile = pl.qt;
      void *qargs[] = {&qp};
      const int64_t chunks = (int64_t)pl.qt * ix->KB * 64;
      DRESD_HIP(launch(qop_kernel(ix->dtype), dim3((unsigned)ceil_div(chunks, 256)), dim3(256),
                       qargs, 0));
      sp.qop = qp.out;
    }
    MergeParams mp;
    mp.lists = lists;
    mp.lcnt = lcnt;
    mp.lkth = lkth;
    mp.lfirst = lfirst;
    mp.spill = spill;
    mp.spill_cap = pl.spill_cap;
    mp.C = pl.C;
    mp.B = gr.nb;
    mp.k = k;
    mp.cont = ix->cont;
    mp.L = ix->L;
    mp.N = ix->N;
    // tau_in: the exact bound from the last pass (keys at or above the k-th
    // best of its sample); spec_in: the key a sampled pass starts from
    // instead, at or above tau_in.  The main pass starts from tau_in.
    const uint64_t *tau_in = nullptr, *spec_in = nullptr;
    int level = 0;
    auto run_pass = [&](int64_t stride, bool main_pass, int spec_rank_out) -> dresd_status {
      sp.stride = stride;
      sp.nvisit = ceil_div(ix->T, stride);
      sp.tau = (main_pass || !spec_in) ? tau_in : spec_in;
      const int64_t wgs = pass_wgs(pl, gr, sp.nvisit, main_pass);
      const int threads = threads_of(pl, main_pass);
      sp.G = (int)(pl.mq ? wgs
                         : pl.tc ? wgs * (main_pass ? pl.nk_main : pl.nk_sample)
                                 : wgs * (threads / kWaveSize));
      void *sargs[] = {&sp};
      hipEvent_t e0 = nullptr, e1 = nullptr;
      if (main_pass && prof) {
        e0 = take_event(ix);
        e1 = take_event(ix);
        if (!e0 || !e1) return fail(DRESD_EDEVICE, "hipEventCreate failed");
      }
      DRESD_HIP(launch((const void *)(main_pass ? pl.kmain : pl.ksample),
                       dim3((unsigned)(wgs * gr.ng)), dim3((unsigned)threads), sargs,
                       main_pass ? pl.lds : pl.lds_s, e0, e1));
      if (main_pass && prof) {
        ix->ev_scan.push_back(e0);
        ix->ev_scan.push_back(e1);
      }
      mp.G = sp.G;
      mp.final_mode = main_pass ? 1 : 0;
      mp.tau_out = tau + (size_t)(level & 1) * pl.bl;
      mp.tau_fb = tau_in;
      mp.spec_out = spec_rank_out > 0 ? tau + 2 * kMaxGroup + (size_t)(level & 1) * pl.bl : nullptr;
      mp.spec_rank = spec_rank_out;
      mp.idx = idx + (size_t)gr.b0 * k;
      mp.score = score + (size_t)gr.b0 * k;
      mp.tokens = tokens ? tokens + (size_t)gr.b0 * k * ix->L : nullptr;
      void *margs[] = {&mp};
      DRESD_HIP(launch(merge_kernel_ptr(), dim3((unsigned)gr.nb), dim3(kMergeThreads), margs, 0,
                       nullptr, nullptr, main_pass && li == pl.nl - 1));
      tau_in = mp.tau_out;
      spec_in = mp.spec_out;
      ++level;
      return DRESD_OK;
    };
    for (int pi = 0; pi < pl.npass; ++pi) {
      s = run_pass(pl.strides[pi], false, pl.spec[pi]);
      if (s != DRESD_OK) return s;
    }
    s = run_pass(1, true, 0);
    if (s != DRESD_OK) return s;
  }
  if (e_all0) {
    // the search's first kernel may have been the timed scan itself
    if (own.first_used != e_all0) ix->ev_free.push_back(e_all0);
    ix->ev_all.push_back(own.first_used);
    ix->ev_all.push_back(e_all1);
  }
  return DRESD_OK;
}

}  // namespace

extern "C" {

dresd_status dresd_bw_probe(const void *buf, int64_t bytes, int32_t reps, int32_t workgroups,
                            double *ms, dresd_stream stream) {
  if (!buf || !ms) return fail(DRESD_EINVAL, "NULL pointer argument");
  if (bytes < (1 << 20) || bytes % 1024 != 0)
    return fail(DRESD_EINVAL, "bytes must be a multiple of 1024 and at least 1 MiB");
  if (reps < 1 || reps > 1000) return fail(DRESD_EINVAL, "reps must be in [1, 1000]");
  if (workgroups < 0 || workgroups > (1 << 20)) return fail(DRESD_EINVAL, "workgroups out of range");
  hipStream_t st = static_cast<hipStream_t>(stream);
  int wg = workgroups;
  if (wg == 0) {
    int dev = 0, cus = 0;
    DRESD_HIP(hipGetDevice(&dev));
    DRESD_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
    wg = 4 * cus;
  }
  const int64_t nblocks = bytes / 1024;
  hipEvent_t a = nullptr, b = nullptr;
  DRESD_HIP(hipEventCreate(&a));
  if (hipEventCreate(&b) != hipSuccess) {
    (void)hipEventDestroy(a);
    return fail(DRESD_EDEVICE, "hipEventCreate failed");
  }
  hipError_t e = launch_bw_read(buf, nblocks, wg, st);  // untimed pass
  if (e == hipSuccess) e = hipEventRecord(a, st);
  for (int r = 0; e == hipSuccess && r < reps; ++r) e = launch_bw_read(buf, nblocks, wg, st);
  if (e == hipSuccess) e = hipEventRecord(b, st);
  if (e == hipSuccess) e = hipEventSynchronize(b);
  float t = 0.f;
  if (e == hipSuccess) e = hipEventElapsedTime(&t, a, b);
  (void)hipEventDestroy(a);
  (void)hipEventDestroy(b);
  if (e != hipSuccess) return fail(DRESD_EDEVICE, std::string("bandwidth probe: ") + hipGetErrorString(e));
  *ms = (double)t / reps;
  return DRESD_OK;
}

dresd_status dresd_transform(const float *x, int64_t M, int32_t D, const float *mean,
                             const float *var, float eps_z, const float *W, int32_t l, float eps_n,
                             float *y, dresd_stream stream) {
  if (M < 0 || M > (int64_t)0x7fffffff) return fail(DRESD_EINVAL, "M out of range");
  if (D < 1 || D > (1 << 20)) return fail(DRESD_EINVAL, "D out of range");
  if (l < 1 || l > 16384) return fail(DRESD_EINVAL, "l out of range");
  if (!(eps_z >= 0.f) || !(eps_n >= 0.f) || eps_z == HUGE_VALF || eps_n == HUGE_VALF)
    return fail(DRESD_EINVAL, "eps must be finite and >= 0");
  if (M == 0) return DRESD_OK;
  if (!x || !mean || !var || !W || !y) return fail(DRESD_EINVAL, "NULL pointer argument");
  int dev = 0;
  DRESD_HIP(hipGetDevice(&dev));
  int cus = 0;
  DRESD_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
  TransformParams p;
  p.splits = transform_splits(M, D, l, cus);
  p.dslice = (int)ceil_div(D, p.splits);
  p.part = nullptr;
  if (p.splits > 1) {
    // Partial sums of the D slices (a per-device buffer kept for the life of
    // the process).
    static DeviceBuffers bufs;
    const size_t need = (size_t)p.splits * (size_t)M * (size_t)l * sizeof(float);
    void *b = nullptr;
    dresd_status s = device_buffer(bufs, dev, need, static_cast<hipStream_t>(stream),
                                   "transform workspace", &b);
    if (s != DRESD_OK) return s;
    p.part = static_cast<float *>(b);
  }
  p.x = x;
  p.mean = mean;
  p.var = var;
  p.W = W;
  p.y = y;
  p.M = M;
  p.D = D;
  p.l = l;
  p.eps_z = eps_z;
  p.eps_n = eps_n;
  DRESD_HIP(launch_transform(p, static_cast<hipStream_t>(stream)));
  return DRESD_OK;
}

dresd_status dresd_pack_drafts(const int32_t *tokens, int32_t B, int32_t k, int32_t L, int32_t r,
                               int32_t length, int32_t eos, int32_t *drafts, int32_t *count,
                               dresd_stream stream) {
  if (B < 0) return fail(DRESD_EINVAL, "B must be >= 0");
  if (k < 1 || k > DRESD_K_MAX) return fail(DRESD_EINVAL, "k must be in [1, DRESD_K_MAX]");
  if (L < 1 || L > 4096) return fail(DRESD_EINVAL, "L out of range");
  if (length < 1 || length > L) return fail(DRESD_EINVAL, "length must be in [1, L]");
  if (r < 1 || r > k) return fail(DRESD_EINVAL, "r must be in [1, k]");
  if (B == 0) return DRESD_OK;
  if (!tokens || !drafts || !count) return fail(DRESD_EINVAL, "NULL pointer argument");
  DraftParams p;
  p.tokens = tokens;
  p.drafts = drafts;
  p.count = count;
  p.B = B;
  p.k = k;
  p.L = L;
  p.r = r;
  p.length = length;
  p.eos = eos;
  DRESD_HIP(launch_pack_drafts(p, static_cast<hipStream_t>(stream)));
  return DRESD_OK;
}

dresd_status dresd_profile_enable(dresd_index *ix, int32_t on) {
  if (!ix) return fail(DRESD_EINVAL, "index is NULL");
  ix->prof = on != 0;
  return DRESD_OK;
}

dresd_status dresd_profile_read(dresd_index *ix, double *scan_ms, double *search_ms,
                                int64_t *searches) {
  if (!ix) return fail(DRESD_EINVAL, "index is NULL");
  double a = 0, b = 0;
  auto sum = [&](std::vector<hipEvent_t> &v, double &acc) -> dresd_status {
    for (size_t i = 0; i + 1 < v.size(); i += 2) {
      DRESD_HIP(hipEventSynchronize(v[i + 1]));
      float ms = 0;
      DRESD_HIP(hipEventElapsedTime(&ms, v[i], v[i + 1]));
      acc += ms;
    }
    return DRESD_OK;
  };
  dresd_status s = sum(ix->ev_scan, a);
  if (s != DRESD_OK) return s;
  s = sum(ix->ev_all, b);
  if (s != DRESD_OK) return s;
  if (scan_ms) *scan_ms = a;
  if (search_ms) *search_ms = b;
  if (searches) *searches = (int64_t)(ix->ev_all.size() / 2);
  for (auto e : profile_events(ix)) ix->ev_free.push_back(e);
  ix->ev_scan.clear();
  ix->ev_all.clear();
  return DRESD_OK;
}


// ------------------------------------------------------ partitioned search ---

}  // extern "C"

struct dresd_ivf {
  dresd_index *ix = nullptr;     // keys in partition order, continuations by row
  dresd_index *cix = nullptr;    // the centroids (fp32 keys, exact probing)
  uint32_t *slot_row = nullptr;  // [T * 16] row of each slot, kPadRow for padding
  int32_t *ftok_slot = nullptr;  // [T * 16] first token of each slot's value (0: padding)
  int32_t *part_tile = nullptr;  // [P + 1] first tile of each partition
  int32_t *tok = nullptr;        // grouped by first token: [P] ascending, partition p's token
  int64_t probe_tiles = 0;       // grouped by first token: size-biased mean tiles of a partition
  int32_t P = 0;
  // probe results (ids + scores) of a search, one buffer per stream
  std::map<hipStream_t, std::pair<unsigned char *, int64_t>> probe;
  std::vector<void *> retired;   // outgrown probe buffers, freed at destroy
};

namespace {

void ivf_free(dresd_ivf *v) {
  if (!v) return;
  if (v->ix) dresd_index_destroy(v->ix);
  if (v->cix) dresd_index_destroy(v->cix);
  if (v->slot_row) (void)hipFree(v->slot_row);
  if (v->ftok_slot) (void)hipFree(v->ftok_slot);
  if (v->part_tile) (void)hipFree(v->part_tile);
  if (v->tok) (void)hipFree(v->tok);
  for (auto &pb : v->probe)
    if (pb.second.first) (void)hipFree(pb.second.first);
  for (void *r : v->retired) (void)hipFree(r);
  delete v;
}

// Scan of the probed partitions + merge.  probes64 (from the centroid
// search) or probes32 (caller's) is [B][S] on the device.
dresd_status parts_search(dresd_ivf *v, const float *queries, const int64_t *probes64,
                          const int32_t *probes32, const int32_t *tok_next, int32_t S,
                          const int32_t *next_tok, int32_t B, int32_t k, int64_t *idx,
                          float *score, int32_t *tokens, Launcher &launch) {
  dresd_index *ix = v->ix;
  hipStream_t st = launch.st;
  const int terms = ix->dtype == kF32 ? 1 : 4;  // the query as three exact 16-bit parts
  const int nq = 16 / terms;
  const int C = next_pow2(std::max(k + 64, 128));
  const int CL = stage_cap(nq);
  // Probes from the exact centroid search: each workgroup builds its
  // query's segments in LDS behind the scan's own state.
  const bool fused = probes64 != nullptr;
  const size_t lds_scan = scan_lds(terms, ix->KB, nq, CL, C);
  const size_t lds = lds_scan + (fused ? ((size_t)(2 * S + 1) * 4 + 15) / 16 * 16 : 0);
  if (lds > ix->lds_max) return fail(DRESD_EUNSUPPORTED, "scan state does not fit in LDS for this d and k");
  ScanKernel kern = scan_parts_kernel(ix->dtype);
  if (!kern) return fail(DRESD_EUNSUPPORTED, "no partitioned scan kernel for this key type");
  // Workgroups per query: enough for ~4 per CU over the batch, but no fewer
  // than 4 tiles per wave of an average probe set.  A probe set is small
  // (tens of MB), and one wave streams it slowly (its loads in flight bound
  // it), so short waves in large numbers finish first; the merge of their
  // lists costs less than longer waves do.
  // Partitions of one first token each differ widely in size, and a query
  // probes one in proportion to its rows: their size-biased mean.
  const int64_t avg_tiles =
      tok_next ? v->probe_tiles : std::max<int64_t>(1, (int64_t)S * ix->T / v->P);
  int64_t wgq = std::min<int64_t>(ceil_div(4LL * ix->cus, B), ceil_div(avg_tiles, 16));
  wgq = std::max<int64_t>(1, std::min<int64_t>(wgq, kMergeLists / 4));
  const int G = (int)wgq * (kScanThreads / kWaveSize);
  const int64_t spill_cap = std::max<int64_t>(0, (int64_t)G * k - kMergeCap);
  auto up = [](size_t x) { return (x + 255) / 256 * 256; };
  const size_t nb = (size_t)B;
  const size_t off_seg = 0;
  const size_t off_tile = off_seg + up(nb * (S + 1) * 4);
  const size_t off_lcnt = off_tile + up(nb * S * 4);
  const size_t off_lkth = off_lcnt + up(nb * G * 4);
  const size_t off_lfirst = off_lkth + up(nb * G * 8);
  const size_t off_lists = off_lfirst + up(nb * G * 8);
  const size_t off_spill = off_lists + up(nb * G * (size_t)C * 8);
  const size_t bytes = off_spill + up(nb * (size_t)std::max<int64_t>(1, spill_cap) * 8);
  unsigned char *ws = nullptr;
  dresd_status s = ensure_workspace(ix, bytes, st, &ws);
  if (s != DRESD_OK) return s;

  SegParams gp;
  gp.probes64 = nullptr;
  gp.probes32 = probes32;
  gp.tok = tok_next ? v->tok : nullptr;
  gp.next_tok = tok_next;
  gp.part_tile = v->part_tile;
  gp.seg_off = reinterpret_cast<int32_t *>(ws + off_seg);
  gp.seg_tile = reinterpret_cast<int32_t *>(ws + off_tile);
  gp.B = B;
  gp.S = S;
  gp.P = v->P;
  if (!fused) DRESD_HIP(launch_segments(gp, st));

  ScanParams sp;
  sp.data = ix->data;
  sp.queries = queries;
  sp.N = ix->N;
  sp.nvisit = 0;
  sp.stride = 1;
  sp.tau = nullptr;
  sp.lists = reinterpret_cast<uint64_t *>(ws + off_lists);
  sp.lcnt = reinterpret_cast<uint32_t *>(ws + off_lcnt);
  sp.lkth = reinterpret_cast<uint64_t *>(ws + off_lkth);
  sp.lfirst = reinterpret_cast<uint64_t *>(ws + off_lfirst);
  sp.B = B;
  sp.d = ix->d;
  sp.KB = ix->KB;
  sp.k = k;
  sp.C = C;
  sp.G = G;
  sp.CL = CL;
  sp.sort_lists = 1;
  sp.qop = nullptr;
  sp.ftok = next_tok ? v->ftok_slot : nullptr;
  sp.next_tok = next_tok;
  sp.slot_row = v->slot_row;
  sp.seg_off = gp.seg_off;
  sp.seg_tile = gp.seg_tile;
  sp.S = S;
  sp.wgq = (int)wgq;
  sp.probes64 = probes64;
  sp.part_tile = v->part_tile;
  sp.seg_lds = (int)lds_scan;
  sp.P = v->P;
  void *sargs[] = {&sp};
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (ix->prof) {
    e0 = take_event(ix);
    e1 = take_event(ix);
    if (!e0 || !e1) return fail(DRESD_EDEVICE, "hipEventCreate failed");
  }
  DRESD_HIP(launch((const void *)kern, dim3((unsigned)(B * wgq)), dim3(kScanThreads), sargs, lds,
                   e0, e1));
  if (ix->prof) {
    ix->ev_scan.push_back(e0);
    ix->ev_scan.push_back(e1);
  }
  MergeParams mp;
  mp.lists = sp.lists;
  mp.lcnt = sp.lcnt;
  mp.lkth = sp.lkth;
  mp.lfirst = sp.lfirst;
  mp.spill = reinterpret_cast<uint64_t *>(ws + off_spill);
  mp.spill_cap = spill_cap;
  mp.B = B;
  mp.k = k;
  mp.C = C;
  mp.G = G;
  mp.tau_out = nullptr;
  mp.tau_fb = nullptr;
  mp.spec_out = nullptr;
  mp.spec_rank = 0;
  mp.idx = idx;
  mp.score = score;
  mp.tokens = tokens;
  mp.cont = ix->cont;
  mp.L = ix->L;
  mp.N = ix->N;
  mp.final_mode = 1;
  void *margs[] = {&mp};
  DRESD_HIP(launch(merge_kernel_ptr(), dim3((unsigned)B), dim3(kMergeThreads), margs, 0, nullptr,
                   nullptr, true));
  return DRESD_OK;
}

dresd_status validate_ivf_search(const dresd_ivf *v, int32_t B, int32_t k) {
  if (!v) return fail(DRESD_EINVAL, "partitioned index is NULL");
  return validate_search(v->ix, B, k);
}

}  // namespace

extern "C" {

static dresd_status check_ivf_args(const void *embeddings, const int32_t *continuations,
                                   int64_t N, int32_t d, int32_t L, int32_t dtype) {
  if (!embeddings || !continuations) return fail(DRESD_EINVAL, "NULL pointer argument");
  if (N < 1 || N > DRESD_N_MAX) return fail(DRESD_EINVAL, "N out of range");
  if (d < 1 || d > 16384) return fail(DRESD_EINVAL, "d out of range");
  if (L < 1 || L > 4096) return fail(DRESD_EINVAL, "L out of range");
  if (dtype < DRESD_F32 || dtype > DRESD_BF16) return fail(DRESD_EINVAL, "unknown dtype");
  return DRESD_OK;
}

// The partitioned index of a host assignment a [N] (ids checked against
// [0, P)); without centroids it has no centroid index, and its searches
// take their probes from the caller.
static dresd_status ivf_build(const void *embeddings, const int32_t *continuations, int64_t N,
                              int32_t d, int32_t L, int32_t dtype, const float *centroids,
                              int32_t P, std::vector<int32_t> &a, hipStream_t st,
                              dresd_ivf **out) {
  const dresd_stream stream = st;
  // Slot table: partitions in id order, each padded to whole tiles, rows of
  // a partition in row order (a stable counting sort of the assignment).
  std::vector<int64_t> cnt((size_t)P, 0);
  for (int64_t i = 0; i < N; ++i) {
    if (a[i] < 0 || a[i] >= P) return fail(DRESD_EINVAL, "assignment outside [0, P)");
    ++cnt[a[i]];
  }
  std::vector<int32_t> pt((size_t)P + 1);
  int64_t T = 0;
  for (int32_t p = 0; p < P; ++p) {
    pt[p] = (int32_t)T;
    T += ceil_div(cnt[p], kTileRows);
  }
  pt[P] = (int32_t)T;
  double sq = 0.0;  // sum over partitions of their tile counts squared
  for (int32_t p = 0; p < P; ++p) sq += (double)(pt[p + 1] - pt[p]) * (double)(pt[p + 1] - pt[p]);
  std::vector<uint32_t> slot((size_t)T * kTileRows, kPadRow);
  std::vector<int64_t> next((size_t)P);
  for (int32_t p = 0; p < P; ++p) next[p] = (int64_t)pt[p] * kTileRows;
  for (int64_t i = 0; i < N; ++i) slot[next[a[i]]++] = (uint32_t)i;
  a.clear();
  a.shrink_to_fit();

  dresd_ivf *v = new (std::nothrow) dresd_ivf();
  if (!v) return fail(DRESD_ENOMEM, "host allocation failed");
  v->P = P;
  v->probe_tiles = std::max<int64_t>(1, (int64_t)(sq / (double)std::max<int64_t>(1, T)));
  auto bail = [&](dresd_status s) {
    ivf_free(v);
    return s;
  };
  if (dev_alloc((void **)&v->slot_row, slot.size() * 4) != hipSuccess ||
      dev_alloc((void **)&v->ftok_slot, slot.size() * 4) != hipSuccess ||
      dev_alloc((void **)&v->part_tile, pt.size() * 4) != hipSuccess) {
    (void)hipGetLastError();
    return bail(fail(DRESD_ENOMEM, "slot table allocation failed"));
  }
  if (hipMemcpy(v->slot_row, slot.data(), slot.size() * 4, hipMemcpyHostToDevice) != hipSuccess ||
      hipMemcpy(v->part_tile, pt.data(), pt.size() * 4, hipMemcpyHostToDevice) != hipSuccess)
    return bail(fail(DRESD_EDEVICE, "slot table upload failed"));
  // First token of each slot's value (the next-token filter).
  if (launch_slot_first_tokens(v->slot_row, continuations, L, (int64_t)slot.size(), v->ftok_slot,
                               st) != hipSuccess ||
      hipStreamSynchronize(st) != hipSuccess)
    return bail(fail(DRESD_EDEVICE, "first-token column build failed"));
  dresd_status s = index_build(embeddings, continuations, N, d, L, dtype, v->slot_row, T, stream,
                               &v->ix);
  if (s != DRESD_OK) return bail(s);
  if (!centroids) {
    *out = v;
    return DRESD_OK;
  }
  // Centroid index: fp32 keys, value = the partition id.
  std::vector<int32_t> ids((size_t)P);
  for (int32_t p = 0; p < P; ++p) ids[p] = p;
  int32_t *ids_dev = nullptr;
  if (dev_alloc((void **)&ids_dev, (size_t)P * 4) != hipSuccess) {
    (void)hipGetLastError();
    return bail(fail(DRESD_ENOMEM, "allocation failed"));
  }
  if (hipMemcpy(ids_dev, ids.data(), (size_t)P * 4, hipMemcpyHostToDevice) != hipSuccess) {
    (void)hipFree(ids_dev);
    return bail(fail(DRESD_EDEVICE, "partition id upload failed"));
  }
  s = index_build(centroids, ids_dev, P, d, 1, DRESD_F32, nullptr, 0, stream, &v->cix);
  (void)hipFree(ids_dev);
  if (s != DRESD_OK) return bail(s);
  *out = v;
  return DRESD_OK;
}

static dresd_status ivf_create_impl(const void *embeddings, const int32_t *continuations, int64_t N,
                              int32_t d, int32_t L, int32_t dtype, const float *centroids,
                              int32_t P, const int32_t *assign, dresd_stream stream,
                              dresd_ivf **out) {
  if (!centroids || !assign || !out) return fail(DRESD_EINVAL, "NULL pointer argument");
  dresd_status s = check_ivf_args(embeddings, continuations, N, d, L, dtype);
  if (s != DRESD_OK) return s;
  if (P < 1 || P > DRESD_PARTS_MAX) return fail(DRESD_EINVAL, "P out of range");
  hipStream_t st = static_cast<hipStream_t>(stream);
  std::vector<int32_t> a((size_t)N);
  DRESD_HIP(hipMemcpyAsync(a.data(), assign, (size_t)N * 4, hipMemcpyDeviceToHost, st));
  DRESD_HIP(hipStreamSynchronize(st));
  return ivf_build(embeddings, continuations, N, d, L, dtype, centroids, P, a, st, out);
}

// Keys grouped by the first token of their value: partition p holds the
// rows whose continuation starts with the p-th smallest distinct token.
static dresd_status ivf_by_token_impl(const void *embeddings, const int32_t *continuations,
                                      int64_t N, int32_t d, int32_t L, int32_t dtype,
                                      dresd_stream stream, dresd_ivf **out) {
  if (!out) return fail(DRESD_EINVAL, "NULL pointer argument");
  dresd_status s = check_ivf_args(embeddings, continuations, N, d, L, dtype);
  if (s != DRESD_OK) return s;
  hipStream_t st = static_cast<hipStream_t>(stream);
  std::vector<int32_t> a((size_t)N);  // first tokens, then their partitions
  {
    // gathered on the device, then one contiguous copy
    int32_t *col = nullptr;
    if (dev_alloc((void **)&col, (size_t)N * 4) != hipSuccess) {
      (void)hipGetLastError();
      return fail(DRESD_ENOMEM, "first-token column allocation failed");
    }
    hipError_t e = launch_first_tokens(continuations, L, N, col, st);
    if (e == hipSuccess) e = hipMemcpyAsync(a.data(), col, (size_t)N * 4, hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    (void)hipFree(col);
    if (e != hipSuccess) return fail(DRESD_EDEVICE, std::string("first-token column: ") + hipGetErrorString(e));
  }
  std::vector<int32_t> tok(a);
  std::sort(tok.begin(), tok.end());
  tok.erase(std::unique(tok.begin(), tok.end()), tok.end());
  if ((int64_t)tok.size() > DRESD_PARTS_MAX)
    return fail(DRESD_EINVAL, "more distinct first tokens than DRESD_PARTS_MAX");
  const int32_t P = (int32_t)tok.size();
  for (int32_t &x : a) x = (int32_t)(std::lower_bound(tok.begin(), tok.end(), x) - tok.begin());
  dresd_ivf *v = nullptr;
  s = ivf_build(embeddings, continuations, N, d, L, dtype, nullptr, P, a, st, &v);
  if (s != DRESD_OK) return s;
  if (dev_alloc((void **)&v->tok, (size_t)P * 4) != hipSuccess) {
    (void)hipGetLastError();
    ivf_free(v);
    return fail(DRESD_ENOMEM, "token table allocation failed");
  }
  if (hipMemcpy(v->tok, tok.data(), (size_t)P * 4, hipMemcpyHostToDevice) != hipSuccess) {
    ivf_free(v);
    return fail(DRESD_EDEVICE, "token table upload failed");
  }
  *out = v;
  return DRESD_OK;
}

dresd_status dresd_ivf_create(const void *embeddings, const int32_t *continuations, int64_t N,
                              int32_t d, int32_t L, int32_t dtype, const float *centroids,
                              int32_t P, const int32_t *assign, dresd_stream stream,
                              dresd_ivf **out) {
  // the slot table is built on the host: its vectors may fail to allocate
  try {
    return ivf_create_impl(embeddings, continuations, N, d, L, dtype, centroids, P, assign, stream,
                           out);
  } catch (const std::bad_alloc &) {
    return fail(DRESD_ENOMEM, "host allocation for the slot table failed");
  }
}

dresd_status dresd_ivf_create_by_token(const void *embeddings, const int32_t *continuations,
                                       int64_t N, int32_t d, int32_t L, int32_t dtype,
                                       dresd_stream stream, dresd_ivf **out) {
  try {
    return ivf_by_token_impl(embeddings, continuations, N, d, L, dtype, stream, out);
  } catch (const std::bad_alloc &) {
    return fail(DRESD_ENOMEM, "host allocation for the slot table failed");
  }
}

void dresd_ivf_destroy(dresd_ivf *v) {
  if (!v) return;
  int cur = 0;
  (void)hipGetDevice(&cur);
  if (v->ix) {
    (void)hipSetDevice(v->ix->device);
    (void)hipDeviceSynchronize();
  }
  ivf_free(v);
  (void)hipSetDevice(cur);
}

dresd_status dresd_ivf_info(const dresd_ivf *v, int64_t *N, int32_t *d, int32_t *L, int32_t *dtype,
                            int32_t *P, int64_t *tiles) {
  if (!v) return fail(DRESD_EINVAL, "partitioned index is NULL");
  dresd_status s = dresd_index_info(v->ix, N, d, L, dtype);
  if (s != DRESD_OK) return s;
  if (P) *P = v->P;
  if (tiles) *tiles = v->ix->T;
  return DRESD_OK;
}

}  // extern "C"

namespace {
dresd_status ivf_search_impl(dresd_ivf *v, const float *queries, const int32_t *next_tok,
                             int32_t B, int32_t k, int32_t nprobe, int64_t *idx, float *score,
                             int32_t *tokens, dresd_stream stream) {
  dresd_status s = validate_ivf_search(v, B, k);
  if (s != DRESD_OK) return s;
  if (!v->cix)
    return fail(DRESD_EINVAL,
                "the index is grouped by first token and has no centroids to probe "
                "(dresd_ivf_search_next_token searches it)");
  if (nprobe < 1 || nprobe > std::min<int32_t>(v->P, DRESD_K_MAX))
    return fail(DRESD_EINVAL, "nprobe must be in [1, min(P, DRESD_K_MAX)]");
  if (B > 0 && (!queries || !idx || !score)) return fail(DRESD_EINVAL, "NULL pointer argument");
  if (B == 0) return DRESD_OK;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int64_t need = (int64_t)B * nprobe * 12;
  auto &pb = v->probe[st];
  if (pb.second < need) {
    if (capturing(st))
      return fail(DRESD_EUNSUPPORTED,
                  "the probe buffer must grow while the stream is being captured; run one "
                  "uncaptured call of this shape first");
    void *p = nullptr;
    if (dev_alloc(&p, (size_t)need) != hipSuccess) {
      (void)hipGetLastError();
      return fail(DRESD_ENOMEM, "probe buffer allocation failed");
    }
    if (hipMemsetAsync(p, 0, (size_t)need, st) != hipSuccess) {  // ordered on the search's stream
      (void)hipFree(p);
      return fail(DRESD_EDEVICE, "probe buffer clear failed");
    }
    // kept until destroy: a captured graph may still use the outgrown buffer
    if (pb.first) v->retired.push_back(pb.first);
    pb = {static_cast<unsigned char *>(p), need};
  }
  int64_t *pid = reinterpret_cast<int64_t *>(pb.first);
  float *psc = reinterpret_cast<float *>(pb.first + (size_t)B * nprobe * 8);
  hipEvent_t a0 = nullptr, a1 = nullptr;
  dresd_index *ix = v->ix;
  Launcher launch;
  launch.st = st;
  if (ix->prof) {
    a0 = take_event(ix);
    a1 = take_event(ix);
    if (!a0 || !a1) return fail(DRESD_EDEVICE, "hipEventCreate failed");
    launch.first = a0;  // the begin of the probe's first kernel
  }
  // 1. probe: the nprobe best centroids of each query (exact search)
  s = search_impl(v->cix, queries, nullptr, B, nprobe, pid, psc, nullptr, stream, &launch);
  if (s != DRESD_OK) return s;
  // 2. exact top-k over the probed partitions (its merge ends the search)
  launch.last = a1;
  s = parts_search(v, queries, pid, nullptr, nullptr, nprobe, next_tok, B, k, idx, score, tokens,
                   launch);
  if (s != DRESD_OK) return s;
  if (a0) {
    if (launch.first_used != a0) ix->ev_free.push_back(a0);
    ix->ev_all.push_back(launch.first_used);
    ix->ev_all.push_back(a1);
  }
  return DRESD_OK;
}
}  // namespace

extern "C" {

dresd_status dresd_ivf_search(dresd_ivf *v, const float *queries, int32_t B, int32_t k,
                              int32_t nprobe, int64_t *idx, float *score, int32_t *tokens,
                              dresd_stream stream) {
  return ivf_search_impl(v, queries, nullptr, B, k, nprobe, idx, score, tokens, stream);
}

dresd_status dresd_ivf_search_filtered(dresd_ivf *v, const float *queries,
                                       const int32_t *next_tok, int32_t B, int32_t k,
                                       int32_t nprobe, int64_t *idx, float *score,
                                       int32_t *tokens, dresd_stream stream) {
  if (B > 0 && !next_tok) return fail(DRESD_EINVAL, "NULL pointer argument");
  return ivf_search_impl(v, queries, next_tok, B, k, nprobe, idx, score, tokens, stream);
}

dresd_status dresd_ivf_search_probes(dresd_ivf *v, const float *queries, const int32_t *probes,
                                     int32_t S, const int32_t *next_tok, int32_t B, int32_t k,
                                     int64_t *idx, float *score, int32_t *tokens,
                                     dresd_stream stream) {
  dresd_status s = validate_ivf_search(v, B, k);
  if (s != DRESD_OK) return s;
  if (S < 1 || S > DRESD_K_MAX) return fail(DRESD_EINVAL, "S must be in [1, DRESD_K_MAX]");
  if (B > 0 && (!queries || !probes || !idx || !score))
    return fail(DRESD_EINVAL, "NULL pointer argument");
  if (B == 0) return DRESD_OK;
  Launcher launch;
  launch.st = static_cast<hipStream_t>(stream);
  return parts_search(v, queries, nullptr, probes, nullptr, S, next_tok, B, k, idx, score, tokens,
                      launch);
}

dresd_status dresd_ivf_search_next_token(dresd_ivf *v, const float *queries,
                                         const int32_t *next_tok, int32_t B, int32_t k,
                                         int64_t *idx, float *score, int32_t *tokens,
                                         dresd_stream stream) {
  dresd_status s = validate_ivf_search(v, B, k);
  if (s != DRESD_OK) return s;
  if (!v->tok)
    return fail(DRESD_EINVAL, "the index was not grouped by first token (dresd_ivf_create_by_token)");
  if (B > 0 && (!queries || !next_tok || !idx || !score))
    return fail(DRESD_EINVAL, "NULL pointer argument");
  if (B == 0) return DRESD_OK;
  Launcher launch;
  launch.st = static_cast<hipStream_t>(stream);
  dresd_index *ix = v->ix;
  hipEvent_t a0 = nullptr, a1 = nullptr;
  if (ix->prof) {
    a0 = take_event(ix);
    a1 = take_event(ix);
    if (!a0 || !a1) return fail(DRESD_EDEVICE, "hipEventCreate failed");
    DRESD_HIP(hipEventRecord(a0, launch.st));  // ahead of the token lookup
    launch.last = a1;
  }
  s = parts_search(v, queries, nullptr, nullptr, next_tok, 1, nullptr, B, k, idx, score, tokens,
                   launch);
  if (s != DRESD_OK) return s;
  if (a0) {
    ix->ev_all.push_back(a0);
    ix->ev_all.push_back(a1);
  }
  return DRESD_OK;
}

dresd_status dresd_kmeans_assign(const void *x, int64_t n, int32_t d, int32_t dtype,
                                 const float *centroids, int32_t P, int32_t *assign, float *score,
                                 dresd_stream stream) {
  if (n < 0 || n > DRESD_N_MAX) return fail(DRESD_EINVAL, "n out of range");
  if (d < 1 || d > 16384) return fail(DRESD_EINVAL, "d out of range");
  if (dtype < DRESD_F32 || dtype > DRESD_BF16) return fail(DRESD_EINVAL, "unknown dtype");
  if (P < 1 || P > DRESD_PARTS_MAX) return fail(DRESD_EINVAL, "P out of range");
  if (n == 0) return DRESD_OK;
  if (!x || !centroids || !assign) return fail(DRESD_EINVAL, "NULL pointer argument");
  KmeansParams p = {};
  p.x = x;
  p.n = n;
  p.d = d;
  p.dtype = dtype;
  p.P = P;
  p.centroids = centroids;
  p.assign = assign;
  p.score = score;
  DRESD_HIP(launch_kmeans_assign(p, static_cast<hipStream_t>(stream)));
  return DRESD_OK;
}

dresd_status dresd_kmeans_update(const void *x, int64_t n, int32_t d, int32_t dtype,
                                 const int32_t *assign, int32_t P, float *centroids,
                                 int32_t *counts, dresd_stream stream) {
  if (n < 0 || n > (int64_t)1 << 31) return fail(DRESD_EINVAL, "n out of range");
  if (d < 1 || d > 16384) return fail(DRESD_EINVAL, "d out of range");
  if (dtype < DRESD_F32 || dtype > DRESD_BF16) return fail(DRESD_EINVAL, "unknown dtype");
  if (P < 1 || P > DRESD_PARTS_MAX) return fail(DRESD_EINVAL, "P out of range");
  if (!centroids || (n > 0 && (!x || !assign))) return fail(DRESD_EINVAL, "NULL pointer argument");
  int dev = 0;
  DRESD_HIP(hipGetDevice(&dev));
  int cus = 0;
  DRESD_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
  // Fixed-point sums and counts (a per-device buffer kept for the life of
  // the process).
  static DeviceBuffers bufs;
  const size_t need = (size_t)P * d * 8 + (size_t)P * 4;
  void *wsp = nullptr;
  dresd_status s = device_buffer(bufs, dev, need, static_cast<hipStream_t>(stream),
                                 "k-means workspace", &wsp);
  if (s != DRESD_OK) return s;
  KmeansParams p = {};
  p.x = x;
  p.n = n;
  p.d = d;
  p.dtype = dtype;
  p.P = P;
  p.assign_in = assign;
  p.centroids_out = centroids;
  p.counts = counts;
  p.sums = static_cast<long long *>(wsp);
  p.cnt = reinterpret_cast<int32_t *>(static_cast<unsigned char *>(wsp) + (size_t)P * d * 8);
  DRESD_HIP(launch_kmeans_update(p, cus, static_cast<hipStream_t>(stream)));
  return DRESD_OK;
}

// First output of SplitMix64 (Steele, Lea and Flood, "Fast splittable
// pseudorandom number generators", 2014) started from state `seed`.
static uint64_t splitmix64_first(uint64_t seed) {
  uint64_t z = seed + 0x9e3779b97f4a7c15ULL;
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
  return z ^ (z >> 31);
}

dresd_status dresd_kmeans_init(const void *x, int64_t n, int32_t d, int32_t dtype, int32_t P,
                               uint64_t seed, float *centroids, dresd_stream stream) {
  if (n < 1 || n > DRESD_N_MAX) return fail(DRESD_EINVAL, "n out of range");
  if (d < 1 || d > 16384) return fail(DRESD_EINVAL, "d out of range");
  if (dtype < DRESD_F32 || dtype > DRESD_BF16) return fail(DRESD_EINVAL, "unknown dtype");
  if (P < 1 || P > DRESD_PARTS_MAX || P > n) return fail(DRESD_EINVAL, "need 1 <= P <= n");
  if (!x || !centroids) return fail(DRESD_EINVAL, "NULL pointer argument");
  KmeansParams p = {};
  p.x = x;
  p.n = n;
  p.d = d;
  p.dtype = dtype;
  p.P = P;
  p.centroids_out = centroids;
  p.offset = (int64_t)(splitmix64_first(seed) % (uint64_t)n);
  DRESD_HIP(launch_kmeans_init(p, static_cast<hipStream_t>(stream)));
  return DRESD_OK;
}

dresd_status dresd_ivf_profile_enable(dresd_ivf *v, int32_t on) {
  if (!v) return fail(DRESD_EINVAL, "partitioned index is NULL");
  return dresd_profile_enable(v->ix, on);
}

dresd_status dresd_ivf_profile_read(dresd_ivf *v, double *scan_ms, double *search_ms,
                                    int64_t *searches) {
  if (!v) return fail(DRESD_EINVAL, "partitioned index is NULL");
  return dresd_profile_read(v->ix, scan_ms, search_ms, searches);
}

}  // extern "C"
