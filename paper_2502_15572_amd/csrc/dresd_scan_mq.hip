// gfx950 scans for batches spanning several 16-column query tiles (the same
// computation as the scan in dresd_kernels.hip: DReSD Section 3.5, Eq. 3
// with unit-norm keys as exact top-k, Section 3.6): the shared-key scan
// below, and the tiled contraction (scan_tc_body) for keys too wide for it
// and for batches larger than it holds at 1,024 dims.
//
// Shared-key scan: the queries stay in registers and the keys are shared
// through LDS:
//   * the workgroup's 4 waves split the query tiles; each wave holds its
//     tiles' A operands for every 32-dim block of the keys in VGPRs;
//   * the workgroup streams its key tiles through a ring of S LDS stages of
//     8 blocks (8 KiB).  Each wave copies 2 blocks of every stage straight
//     from HBM into LDS (global_load_lds_dwordx4, no VGPR round trip), S - 1
//     stages ahead; one barrier per stage publishes a stage to all waves,
//     which each read every block once (4 KiB of LDS reads per KiB of HBM);
//   * every stage issues exactly 2 copies per wave (copies past the end
//     re-read the last blocks), so the wait before each stage is a constant.
// The per-tile test against the per-query thresholds is a few VALU
// instructions; tiles with candidates append (key, query) pairs to a small
// per-wave LDS buffer, which is moved into per-(query, workgroup) lists in
// HBM only when it fills up.
#include "dresd_device.h"

namespace dresd {

namespace {

template <int DT>
struct MfmaMQ;
template <>
struct MfmaMQ<kF16> {
  __device__ __forceinline__ static f4 run(u4 a, u4 b, f4 acc) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(h8, a),
                                                  __builtin_bit_cast(h8, b), acc, 0, 0, 0);
  }
};
template <>
struct MfmaMQ<kBF16> {
  __device__ __forceinline__ static f4 run(u4 a, u4 b, f4 acc) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(b8, a),
                                                   __builtin_bit_cast(b8, b), acc, 0, 0, 0);
  }
};

// A-operand chunk of column `col` for dims [dim0, dim0+8): CPQ = 1 rounds the
// query once to the key type; CPQ = 2 (bf16) gives the high part and the
// rounded remainder (sum within 2^-17 relative of the query); CPQ = 4 gives
// three parts summing to it exactly (f16 lower parts scaled by 2^11, 2^22)
// and a zero column.  `vec`: rows of
// q start 16-byte aligned, so a whole chunk is two 16-byte loads.
template <int DT, int CPQ>
__device__ __forceinline__ u4 query_chunk_mq(const float *q, int d, int B, int col, int dim0,
                                             bool vec) {
  const int b = col / CPQ;
  const int h = col % CPQ;
  float x[8];
  if (vec && b < B && dim0 + 8 <= d) {
    const float4 *src = reinterpret_cast<const float4 *>(q + (int64_t)b * d + dim0);
    const float4 lo4 = src[0], hi4 = src[1];
    x[0] = lo4.x, x[1] = lo4.y, x[2] = lo4.z, x[3] = lo4.w;
    x[4] = hi4.x, x[5] = hi4.y, x[6] = hi4.z, x[7] = hi4.w;
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int dim = dim0 + e;
      x[e] = (b < B && dim < d) ? q[(int64_t)b * d + dim] : 0.0f;
    }
  }
  uint16_t v[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    if (DT == kF16) {
      _Float16 hi = (_Float16)x[e];
      _Float16 r = hi;
      if (CPQ == 4) {
        float r1 = x[e] - (float)hi;
        _Float16 mid = (_Float16)(r1 * 2048.0f);
        float r2 = r1 - (float)mid * (1.0f / 2048.0f);
        _Float16 lo = (_Float16)(r2 * 4194304.0f);
        r = (h == 0) ? hi : (h == 1) ? mid : (h == 2) ? lo : (_Float16)0.0f;
      }
      v[e] = __builtin_bit_cast(uint16_t, r);
    } else {
      __bf16 hi = (__bf16)x[e];
      float r1 = x[e] - (float)hi;
      __bf16 mid = (__bf16)r1;
      __bf16 lo = (__bf16)(r1 - (float)mid);
      __bf16 r = (h == 0) ? hi : (h == 1) ? mid : (CPQ == 4 && h == 2) ? lo : (__bf16)0.0f;
      v[e] = __builtin_bit_cast(uint16_t, r);
    }
  }
  u4 out;
#pragma unroll
  for (int e = 0; e < 4; ++e) out[e] = (uint32_t)v[2 * e] | ((uint32_t)v[2 * e + 1] << 16);
  return out;
}

// Copy two consecutive 1 KiB blocks at `src` into LDS at `lds` and lds + 1 KiB:
// lane l's 16 bytes go to lds + 16 l (the LDS address comes from M0 and the
// lane index, not from the global address).  Written as inline assembly so
// that the compiler's wait-count model, which does not know which LDS bytes
// an LDS-DMA copy writes, adds no waits for these copies before unrelated LDS
// reads; the caller waits with wait_vmcnt and a barrier before reading them.
__device__ __forceinline__ void copy2_to_lds(const void *src, uint32_t voff0, uint32_t voff1,
                                             uint32_t lds) {
  asm volatile(
      "s_mov_b32 m0, %3\n\t"
      "global_load_lds_dwordx4 %0, %2 nt\n\t"
      "s_add_u32 m0, m0, 0x400\n\t"
      "global_load_lds_dwordx4 %1, %2 nt"
      :
      : "v"(voff0), "v"(voff1), "s"(src), "s"(lds)
      : "memory");
}

}  // namespace

// Candidate state of one wave of the shared-key scans.  The wave owns NQW
// queries starting at q0.  For each it keeps, in LDS, an exact threshold
// (keys above it may enter), that threshold as a float for the per-tile
// test, the length of its list in HBM (one list per (query, list slot)) and
// the best key listed; and a buffer of (key, query) pairs that passed the
// test, moved into the lists only when it fills up.  QTW query tiles of CPQ
// operand columns per query; FILT: next-token-filtered search.
template <int DT, int QTW, int CPQ, bool FILT, int CBUF = kMqCandBuf>
struct WaveCands {
  static constexpr int QPT = 16 / CPQ;   // queries per tile
  static constexpr int NS = 4 / CPQ;     // scores per lane per query tile
  static constexpr int NQW = QTW * QPT;  // queries per wave
  static constexpr int NP = QTW * NS;    // scores per lane per key tile
  static constexpr int CB = CBUF;
  static_assert(NP <= 32, "score slots");

  const ScanParams &p;
  const int lane, g, m, q0, lslot;
  uint64_t *ck;       // buffered keys [CB]
  uint64_t *scr;      // sort scratch [C]
  uint64_t *st_key;   // keep keys > st_key [NQW]
  uint8_t *cq;        // query of ck[e] [CB]
  uint32_t *st_cnt;   // HBM list length [NQW]
  float *st_thr;      // float threshold [NQW]
  uint64_t *st_max;   // best listed key [NQW]
  int32_t *nt_slot;   // filtered search: next token per score slot [4 lane groups][NP]
  float thr[NP];      // this lane's thresholds, slot j = t * NS + s
  int ntr[NP <= 8 ? NP : 1];  // filtered search with few slots: nt_slot in VGPRs
  int cnt = 0;        // buffered candidates (wave-uniform)

  // `region`: the wave's scan_mq_wave_bytes(NQW, C, CB) bytes of LDS.
  __device__ __forceinline__ WaveCands(const ScanParams &p_, unsigned char *region, int32_t *nt,
                                       int q0_, int lslot_)
      : p(p_), lane(threadIdx.x & 63), g((threadIdx.x & 63) >> 4), m(threadIdx.x & 15), q0(q0_),
        lslot(lslot_), nt_slot(nt) {
    ck = reinterpret_cast<uint64_t *>(region);
    scr = ck + CB;
    st_key = scr + p.C;
    cq = reinterpret_cast<uint8_t *>(st_key + NQW);
    st_cnt = reinterpret_cast<uint32_t *>(cq + CB);
    st_thr = reinterpret_cast<float *>(st_cnt + NQW);
    st_max = reinterpret_cast<uint64_t *>(st_thr + NQW);
  }

  // Thresholds from the sampled passes (none: every key enters; queries
  // past the batch: none ever does).
  __device__ __forceinline__ void init() {
    const int B = p.B;
    for (int i = lane; i < NQW; i += kWaveSize) {
      uint64_t tk = 0;
      float tf = -__builtin_inff();
      if (q0 + i >= B) {
        tk = ~0ull;
        tf = __builtin_inff();
      } else if (p.tau && p.tau[q0 + i] != 0) {
        tk = p.tau[q0 + i] - 1;  // keep keys >= tau
        tf = order_value((uint32_t)(tk >> 32));
      }
      st_key[i] = tk;
      st_cnt[i] = 0;
      st_thr[i] = tf;
      st_max[i] = 0;
    }
    if (FILT)
      for (int i = lane; i < 4 * NP; i += kWaveSize) {
        const int gg = i / NP, j = i % NP;
        const int q = q0 + (j / NS) * QPT + gg * NS + (j % NS);
        nt_slot[i] = q < B ? p.next_tok[q] : 0;
      }
    wave_sync_lds();
    load_thr();
    if (FILT && NP <= 8) {
#pragma unroll
      for (int j = 0; j < (NP <= 8 ? NP : 1); ++j) ntr[j] = nt_slot[g * NP + j];
    }
  }

  // Score slot j = t * NS + s of a lane belongs to query t * QPT + g * NS + s.
  __device__ __forceinline__ void load_thr() {
#pragma unroll
    for (int j = 0; j < NP; ++j) thr[j] = st_thr[(j / NS) * QPT + g * NS + (j % NS)];
  }

  __device__ __forceinline__ uint64_t *list_of(int i) const {
    return p.lists + ((size_t)(q0 + i) * p.G + lslot) * p.C;
  }

  // Cut query i's full HBM list to its k best keys and raise its threshold.
  __device__ void cut(int i) {
    const int C = p.C, k = p.k;
    uint64_t *list = list_of(i);
    __threadfence_block();  // this wave's list stores are visible to its loads
    for (int e = lane; e < C; e += kWaveSize) scr[e] = list[e];
    wave_sync_lds();
    wave_bitonic_desc(scr, C, lane);
    for (int e = lane; e < k; e += kWaveSize) list[e] = scr[e];
    const uint64_t kth = scr[k - 1];
    wave_sync_lds();
    if (lane == 0) {
      st_cnt[i] = (uint32_t)k;
      if (kth > st_key[i]) {
        st_key[i] = kth;
        st_thr[i] = order_value((uint32_t)(kth >> 32));
      }
    }
    wave_sync_lds();
  }

  // Move the buffered candidates into the HBM lists (keys that still beat
  // their query's exact threshold), cutting lists that fill up.
  __device__ __forceinline__ void flush() {
    const int C = p.C;
    wave_sync_lds();
    for (int e0 = 0; e0 < cnt; e0 += kWaveSize) {
      const int e = e0 + lane;
      const bool valid = e < cnt;
      const int q = valid ? (int)cq[e] : 0;
      const uint64_t key = valid ? ck[e] : 0ull;
      bool has = valid && key > st_key[q];
      while (__ballot(has)) {
        const uint32_t pos = has ? atomicAdd(&st_cnt[q], 1u) : 0u;
        const bool over = has && pos >= (uint32_t)C;
        if (has && !over) {
          list_of(q)[pos] = key;
          atomicMax((unsigned long long *)&st_max[q], (unsigned long long)key);
        }
        uint64_t om = __ballot(over);
        if (om == 0) break;
        if (over) st_cnt[q] = (uint32_t)C;
        wave_sync_lds();
        while (om) {
          const int qq = __builtin_amdgcn_readlane(q, __ffsll((long long)om) - 1);
          cut(qq);
          om &= ~__ballot(over && q == qq);
        }
        has = over && key > st_key[q];
      }
    }
    cnt = 0;
    wave_sync_lds();
    load_thr();
  }

  // Lanes below this one holding a set bit of mask `mk`.
  __device__ __forceinline__ int rank_in(uint64_t mk) const {
    return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(mk >> 32),
                                          __builtin_amdgcn_mbcnt_lo((uint32_t)mk, 0u));
  }

  // Buffer the candidates of key tile `tile` (rows tile*16 .. +15); rare.
  // Bit t of hit_t: some score of query tile t reached its threshold.
  __device__ __forceinline__ void candidates(int64_t tile, const float (&sc)[NP], uint32_t hit_t) {
    const int64_t row64 = tile * kTileRows + m;
    const bool row_ok = row64 < p.N;
    const uint32_t row = (uint32_t)row64;
    // One pass over the slots of the query tiles with hits: a slot's hits
    // are appended while they fit; the first slot that does not fit stops
    // the pass, and the rest (rare: thresholds still low) goes one slot at
    // a time with a flush whenever the next one does not fit.
    const uint64_t okm = __ballot(row_ok);
    int jstop = NP;
#pragma unroll
    for (int j = 0; j < NP; ++j) {
      if (jstop < NP || !(hit_t & (1u << (j / NS)))) continue;
      const uint64_t mk = __ballot(sc[j] >= thr[j]) & okm;
      if (mk == 0) continue;
      if (cnt + __popcll(mk) > CB) {
        jstop = j;
        continue;
      }
      if ((mk >> lane) & 1ull) {
        const int at = cnt + rank_in(mk);
        ck[at] = make_key(sc[j], row);
        cq[at] = (uint8_t)((j / NS) * QPT + g * NS + (j % NS));
      }
      cnt += __popcll(mk);
    }
    if (jstop < NP) {
      // Slot j's score is rotated into cur[0] (no indexed register access).
      float cur[NP];
#pragma unroll
      for (int j = 0; j < NP; ++j) cur[j] = sc[j];
#pragma unroll 1
      for (int j = 0; j < NP; ++j) {
        if (j >= jstop && (hit_t & (1u << (j / NS)))) {
          const int qi = (j / NS) * QPT + g * NS + (j % NS);
          if (cnt + __popcll(__ballot(row_ok && cur[0] >= st_thr[qi])) > CB) flush();
          const bool h = row_ok && cur[0] >= st_thr[qi];
          const uint64_t mk = __ballot(h);
          if (h) {
            const int at = cnt + rank_in(mk);
            ck[at] = make_key(cur[0], row);
            cq[at] = (uint8_t)qi;
          }
          cnt += __popcll(mk);
        }
#pragma unroll
        for (int i = 0; i + 1 < NP; ++i) cur[i] = cur[i + 1];
      }
    }
  }

  // Scores of a finished key tile from its accumulators (the query parts
  // recombined), NaN where the filter drops the row (`f`: the row's first
  // token); NaN fails every threshold test and fmaxf ignores it.
  __device__ __forceinline__ void scores_of(const f4 (&a)[QTW], int f, float (&sc)[NP]) const {
#pragma unroll
    for (int t = 0; t < QTW; ++t)
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        float v = a[t][s * CPQ];
        if (CPQ == 4) {
          const float s1 = (DT == kF16) ? (1.0f / 2048.0f) : 1.0f;
          const float s2 = (DT == kF16) ? (1.0f / 4194304.0f) : 1.0f;
          v = (v + a[t][s * CPQ + 1] * s1) + a[t][s * CPQ + 2] * s2;
        } else if (CPQ == 2) {
          v = v + a[t][s * CPQ + 1];
        }
        sc[t * NS + s] = v;
      }
    if (FILT) {
#pragma unroll
      for (int j = 0; j < NP; ++j)
        if (f != (NP <= 8 ? ntr[j] : nt_slot[g * NP + j])) sc[j] = __builtin_nanf("");
    }
  }

  // Lanes whose row passes some threshold (v >= thr exactly when
  // v - thr >= 0: round-to-nearest keeps the sign).
  __device__ __forceinline__ uint64_t any_hit(const float (&sc)[NP]) const {
    float mx = sc[0] - thr[0];
#pragma unroll
    for (int j = 1; j < NP; ++j) mx = fmaxf(mx, sc[j] - thr[j]);
    return __ballot(mx >= 0.0f);
  }

  // The slow path of key tile `tile` with hits: which query tiles hit,
  // then buffer.
  __device__ __forceinline__ void take(int64_t tile, const float (&sc)[NP]) {
    uint32_t hit_t = 0;
#pragma unroll
    for (int t = 0; t < QTW; ++t) {
      float mt = sc[t * NS] - thr[t * NS];
#pragma unroll
      for (int s = 1; s < NS; ++s) mt = fmaxf(mt, sc[t * NS + s] - thr[t * NS + s]);
      if (__ballot(mt >= 0.0f)) hit_t |= 1u << t;
    }
    candidates(tile, sc, hit_t);
  }

  // A sampled pass's cheaper candidates: of key tile `tile`, only each
  // query's best key (the 16 rows of a lane group belong to one query per
  // slot).  The k-th best of these per-tile maxima is still the key of a
  // row, so it bounds the query's k-th best from below like the k-th best
  // of every sampled row, while a tile adds one candidate per query instead
  // of up to 16.  ROOM: room for the tile's maxima (at most one key per
  // score slot and lane group) is made once, before the slot loop, rather
  // than in it: for scans with several tiles per wave, whose epilogue would
  // otherwise hold a flush per slot and tile.
  template <bool ROOM>
  __device__ __forceinline__ void take_tile_max(int64_t tile, const float (&sc)[NP]) {
    static_assert(!ROOM || 4 * NP <= CB, "buffer holds one tile's maxima");
    if (ROOM && cnt + 4 * NP > CB) flush();
    const int64_t row64 = tile * kTileRows + m;
    const bool row_ok = row64 < p.N;
    const uint32_t row = (uint32_t)row64;
#pragma unroll
    for (int j = 0; j < NP; ++j) {
      // rows outside the datastore, and rows the filter drops (NaN), list nothing
      uint64_t key = (row_ok && sc[j] == sc[j]) ? make_key(sc[j], row) : 0ull;
#pragma unroll
      for (int off = 1; off < kTileRows; off <<= 1) {
        const uint64_t o = __shfl_xor(key, off, kWaveSize);
        key = o > key ? o : key;
      }
      const bool h = m == 0 && key != 0ull && order_value((uint32_t)(key >> 32)) >= thr[j];
      const uint64_t mk = __ballot(h);
      if (mk == 0) continue;
      if (!ROOM && cnt + __popcll(mk) > CB) flush();
      if (h) {
        const int at = cnt + rank_in(mk);
        ck[at] = key;
        cq[at] = (uint8_t)((j / NS) * QPT + g * NS + (j % NS));
      }
      cnt += __popcll(mk);
    }
  }

  // Publish this wave's lists (one per query per list slot) and per list
  // its length (kSortedFlag when sorted), best key (0 when empty) and k-th
  // key (0 unless it holds k sorted keys).  Lane i takes query i; lists
  // longer than k (every non-empty list when sort_lists) are sorted and cut
  // to k first.
  __device__ __forceinline__ void publish() {
    static_assert(NQW <= kWaveSize, "one lane per query");
    const int B = p.B, k = p.k, G = p.G;
    if (cnt > 0) flush();
    const int i = lane;
    const bool valid = i < NQW && q0 + i < B;
    const int n = valid ? (int)st_cnt[i] : 0;
    const bool sort_me = valid && (n > k || (p.sort_lists && n > 0));
    if (valid && !sort_me) {
      const size_t o = (size_t)(q0 + i) * G + lslot;
      p.lcnt[o] = (uint32_t)n | ((n == 1) ? kSortedFlag : 0u);
      p.lfirst[o] = (n == 0) ? 0ull : st_max[i];
      p.lkth[o] = 0ull;
    }
    uint64_t todo = __ballot(sort_me);
    // The lists are ordered one after another; a list of at most
    // kWaveRankMax keys is loaded (up to PF keys per lane) while the one
    // before it is being ordered, so the loads' latency is paid about once
    // rather than once per query.
    constexpr int PF = kWaveRankMax / kWaveSize;
    uint64_t nxt[PF];
    int qn = -1, nn = 0;
    auto prefetch = [&]() {
      if (!todo) {
        qn = -1;
        return;
      }
      qn = __ffsll((long long)todo) - 1;
      todo &= todo - 1;
      nn = __builtin_amdgcn_readlane(n, qn);
      const uint64_t *list = list_of(qn);
#pragma unroll
      for (int j = 0; j < PF; ++j) {
        const int e = lane + j * kWaveSize;
        nxt[j] = (nn <= kWaveRankMax && e < nn) ? list[e] : 0ull;
      }
    };
    __threadfence_block();  // this wave's list stores are visible to its loads
    prefetch();
    while (qn >= 0) {
      const int qi = qn, nq = nn;
      uint64_t cur[PF];
#pragma unroll
      for (int j = 0; j < PF; ++j) cur[j] = nxt[j];
      prefetch();
      uint64_t *list = list_of(qi);
      const int keep = nq < k ? nq : k;
      RankEnds ends;
      if (nq <= kWaveRankMax) {
#pragma unroll
        for (int j = 0; j < PF; ++j)
          if (lane + j * kWaveSize < nq) scr[lane + j * kWaveSize] = cur[j];
        wave_sync_lds();
        ends = wave_rank_top(scr, nq, list, keep, lane);
      } else {
        int np2 = 2;
        while (np2 < nq) np2 <<= 1;
        for (int e = lane; e < np2; e += kWaveSize) scr[e] = (e < nq) ? list[e] : 0ull;
        wave_sync_lds();
        wave_bitonic_desc(scr, np2, lane);
        for (int e = lane; e < keep; e += kWaveSize) list[e] = scr[e];
        ends.first = scr[0];
        ends.last = scr[keep - 1];
      }
      if (lane == 0) {
        const size_t o = (size_t)(q0 + qi) * G + lslot;
        p.lcnt[o] = (uint32_t)keep | kSortedFlag;
        p.lfirst[o] = ends.first;
        p.lkth[o] = (keep == k) ? ends.last : 0ull;
      }
      wave_sync_lds();
    }
  }
};

// QTW query tiles per wave, KBT 32-dim blocks per key tile (must equal the
// index's blocks per tile), CPQ operand columns per query, S LDS stages;
// FILT: next-token-filtered search (a separate instantiation, so the
// unfiltered stream loop carries none of its code).
template <int DT, int QTW, int KBT, int CPQ, int S, bool FILT, int NWQ>
__device__ __forceinline__ void scan_mq_body(const ScanParams &p) {
  using WC = WaveCands<DT, QTW, CPQ, FILT>;
  constexpr int NQW = WC::NQW;  // queries per wave
  constexpr int NP = WC::NP;    // scores per lane per key tile
  constexpr int SB = kMqStageBlocks;
  constexpr int TPS = KBT >= SB ? 1 : SB / KBT;  // key tiles per stage
  constexpr int SPT = KBT >= SB ? KBT / SB : 1;  // stages per key tile
  constexpr int BPT = KBT >= SB ? SB : KBT;      // blocks of a tile per stage
  constexpr int CPW = 4 / NWQ;  // pairs of blocks each wave copies per stage
  constexpr int WAIT = 2 * CPW * (S - 2);  // copies of later stages still in flight
  // Interleave each tile's threshold test with the next tile's matrix
  // instructions when a key tile carries few of them (measured: 33.5M keys x
  // 128 dims at 128 queries, 8 per tile, main pass 1.43 -> 1.37 ms; at
  // 10M x 256 and 256 queries, 32 per tile, it was slower).
  constexpr bool kDefer = BPT * QTW <= 16;
  static_assert(KBT >= 4 && S >= 3, "shape");
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];

  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int m = lane & 15;
  const int G = p.G;
  const int wg = blockIdx.x;

  // LDS: ring of S stages, then one candidate region per wave, then (filtered
  // search) per wave the next token of each score slot and a ring of
  // first-token copies, one per stage (its tiles' 16 rows each).
  const size_t wreg = scan_mq_wave_bytes(NQW, p.C);
  constexpr bool filt = FILT;
  int32_t *nt_slot = reinterpret_cast<int32_t *>(
      smem + (size_t)S * SB * kBlockBytes + (size_t)NWQ * wreg +
      (size_t)wv * scan_mq_filter_bytes(S, NP));  // [4 lane groups][NP]
  int32_t *fring = nt_slot + 4 * NP;              // [S][64]

  // Queries of this wave: tiles [wv*QTW, wv*QTW + QTW) of the batch.
  const int q0 = wv * NQW;
  const u4 *qop = static_cast<const u4 *>(p.qop) + lane;
  u4 qreg[QTW][KBT];
#pragma unroll
  for (int t = 0; t < QTW; ++t)
#pragma unroll
    for (int kb = 0; kb < KBT; ++kb) qreg[t][kb] = qop[((wv * QTW + t) * KBT + kb) * 64];
  // Wait for these loads here: left to the compiler, the wait lands at their
  // first use inside the stream loop, where (not knowing the LDS copies are
  // younger) it would drain the whole copy ring on every stage.
  __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
  WC wc(p, smem + (size_t)S * SB * kBlockBytes + (size_t)wv * wreg, nt_slot, q0, wg);
  wc.init();

  // This workgroup's key tiles: visited tiles [v0, v1), KBT blocks each.
  const int64_t v0 = wave_uniform(p.nvisit * wg / G);
  const int64_t v1 = wave_uniform(p.nvisit * (wg + 1) / G);
  const int ntile = (int)(v1 - v0);

  // The slow path of visited tile vt with hits.
  auto take = [&](int vt, const float (&sc)[NP]) { wc.take((v0 + vt) * p.stride, sc); };

  if (ntile > 0) {
    const int64_t NB = (int64_t)ntile * KBT;
    const int64_t tstep = p.stride * KBT * kBlockBytes;  // bytes between visited tiles
    const unsigned char *dbase = static_cast<const unsigned char *>(p.data) + v0 * tstep;
    const uint32_t voff0 = (uint32_t)lane * 16u, voff1 = voff0 + kBlockBytes;
    // LDS offsets: the low half of a generic LDS address.
    const uint32_t ring = (uint32_t)(uintptr_t)smem;
    const uint32_t fring_lds = (uint32_t)(uintptr_t)fring;
    // Source of pair c of this wave's blocks of stage `st` (blocks
    // j = st*SB + 2(wv CPW + c), +1 of the visited sequence; past the end,
    // the last two blocks again).
    const int64_t jl = NB - 2;
    const unsigned char *last_src =
        dbase + (jl / KBT) * tstep + (jl - (jl / KBT) * KBT) * kBlockBytes;
    const int64_t stage_step = (SPT == 1) ? (int64_t)TPS * tstep : 0;
    auto pair_blk = [&](int c) { return (wv * CPW + c) * 2; };
    auto src_of = [&](int64_t st, int c) -> const unsigned char * {
      const int bj = pair_blk(c);
      if (st * SB + bj > jl) return last_src;
      if constexpr (SPT == 1)
        return dbase + st * stage_step + (int64_t)(bj / KBT) * tstep +
               (int64_t)(bj % KBT) * kBlockBytes;
      return dbase + (st / SPT) * tstep + ((st % SPT) * SB + bj) * kBlockBytes;
    };
    // Copy this wave's blocks of stage `st` into ring slot `slot`.
    auto issue = [&](int64_t st, int slot) {
#pragma unroll
      for (int c = 0; c < CPW; ++c)
        copy2_to_lds(src_of(st, c), voff0, voff1,
                     ring + (uint32_t)(slot * SB + pair_blk(c)) * (uint32_t)kBlockBytes);
      if (filt) {
        // first tokens of the stage's tiles: lane l takes row l % 16 of the
        // stage's (l / 16)-th tile (clamped to the last tile)
        int64_t ft = (TPS > 1 ? st * TPS : st / SPT) + (lane >> 4);
        ft = ft < ntile ? ft : ntile - 1;
        copy1_to_lds(p.ftok + (v0 + ft) * p.stride * kTileRows + (lane & 15),
                     fring_lds + (uint32_t)slot * 256u);
      }
    };
#pragma unroll
    for (int st = 0; st < S - 1; ++st) issue(st, st);
    // The stream loop's copies: stage next_st, whose source address moves
    // by a fixed step per stage (and per key tile when a tile spans several
    // stages) instead of being recomputed; stages past last_ok repeat the
    // last two blocks.
    int last_ok[CPW];
    const unsigned char *next_src[CPW];
#pragma unroll
    for (int c = 0; c < CPW; ++c) {
      last_ok[c] = jl >= pair_blk(c) ? (int)((jl - pair_blk(c)) / SB) : -1;
      next_src[c] = src_of(S - 1, c);
    }
    int next_st = S - 1;  // next stage to copy
    int next_c = (S - 1) % SPT;  // its stage within its key tile
    int next_slot = S - 1;    // its ring slot
    int cur_slot = 0;         // ring slot of the stage being consumed
    auto issue_next = [&]() {
      if (filt) {
        issue(next_st, next_slot);
      } else {
#pragma unroll
        for (int c = 0; c < CPW; ++c) {
          if (next_st > last_ok[c])
            copy2_to_lds(last_src, voff0, voff1,
                         ring + (uint32_t)(next_slot * SB + pair_blk(c)) * (uint32_t)kBlockBytes);
          else
            copy2_to_lds(next_src[c], voff0, voff1,
                         ring + (uint32_t)(next_slot * SB + pair_blk(c)) * (uint32_t)kBlockBytes);
        }
      }
      ++next_st;
      int64_t step = stage_step;
      if constexpr (SPT > 1) {
        if (++next_c == SPT) {
          next_c = 0;
          step = tstep - (int64_t)(SPT - 1) * SB * kBlockBytes;
        } else {
          step = (int64_t)SB * kBlockBytes;
        }
      }
#pragma unroll
      for (int c = 0; c < CPW; ++c) next_src[c] += step;
      next_slot = next_slot == S - 1 ? 0 : next_slot + 1;
    };
    // Stage bookkeeping at the start of a key tile's c-th stage: this wave's
    // copies of it have landed; after the barrier so have every wave's, and
    // the slot consumed last is free for the copy S - 1 stages ahead.
    auto stage_start = [&](int vt) {
      if (TPS == 1 || (vt & (TPS - 1)) == 0) {
        if (filt) wait_vmcnt<WAIT + (S - 2)>();  // one more copy per stage
        else wait_vmcnt<WAIT>();
        __syncthreads();
        issue_next();
      }
    };
    // First token of this lane's row of tile vt (filtered search), read
    // from the tile's ring slot before a later stage may overwrite it; and
    // the ring slot advance at a stage end.
    auto stage_end = [&](int vt, int &ftok_row) {
      if (filt) ftok_row = fring[cur_slot * 64 + (TPS > 1 ? (int)(vt & (TPS - 1)) : 0) * 16 + m];
      if (TPS == 1 || (vt & (TPS - 1)) == TPS - 1) cur_slot = cur_slot == S - 1 ? 0 : cur_slot + 1;
    };
    auto stage_blocks = [&](int vt) {
      return reinterpret_cast<const u4 *>(smem + (size_t)cur_slot * SB * kBlockBytes +
                                          (size_t)((TPS > 1 ? (int)(vt & (TPS - 1)) : 0) * KBT) *
                                              kBlockBytes) +
             lane;
    };
    const int ntile_pad = (ntile + TPS - 1) / TPS * TPS;
    if constexpr (!kDefer) {
      // Many matrix instructions per key tile: the tile's threshold test
      // follows its own matrix instructions.
      f4 acc[QTW];
#pragma unroll 1
      for (int vt = 0; vt < ntile_pad; ++vt) {
        int fr = 0;
#pragma unroll
        for (int c = 0; c < SPT; ++c) {
          stage_start(vt);
          const u4 *blk = stage_blocks(vt);
          // Two blocks at a time, the next two read from LDS while the
          // matrix cores work on these.
          u4 kv0 = blk[0], kv1 = blk[64];
#pragma unroll
          for (int i = 0; i < BPT; i += 2) {
            u4 nx0 = kv0, nx1 = kv1;
            if (i + 2 < BPT) {
              nx0 = blk[(i + 2) * 64];
              nx1 = blk[(i + 3) * 64];
            }
            const int kb = c * SB + i;
#pragma unroll
            for (int t = 0; t < QTW; ++t)
              acc[t] = MfmaMQ<DT>::run(qreg[t][kb], kv0, kb == 0 ? f4{0.f, 0.f, 0.f, 0.f} : acc[t]);
#pragma unroll
            for (int t = 0; t < QTW; ++t) acc[t] = MfmaMQ<DT>::run(qreg[t][kb + 1], kv1, acc[t]);
            kv0 = nx0;
            kv1 = nx1;
          }
          // Keep that order through instruction scheduling: the first two
          // reads, then per pair of blocks the next two reads and the pair's
          // matrix instructions.
          __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
#pragma unroll
          for (int i = 0; i < BPT; i += 2) {
            if (i + 2 < BPT) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, 2 * QTW, 0);
          }
          stage_end(vt, fr);
        }
        if (vt < ntile) {
          float sc[NP];
          wc.scores_of(acc, fr, sc);
          if (wc.any_hit(sc)) take(vt, sc);
        }
      }
    } else {
      // Few matrix instructions per key tile (the threshold test is a large
      // share of a tile's work): each tile's test runs interleaved with the
      // next tile's matrix instructions, from a second set of accumulators.
      f4 accA[QTW], accB[QTW];
      int fA = 0, fB = 0;  // filtered search: this lane's first token of the tile in accA / accB
      // One key tile: its matrix instructions into `acc`, the test of the
      // previous tile (complete in `prev`) split over its pairs of blocks,
      // then that tile's slow path if it has hits.
      auto step = [&](int vt, f4 (&acc)[QTW], const f4 (&prev)[QTW], int &fcur, int fprev) {
        const int pv = vt - 1;
        float psc[NP];
        uint64_t hits = 0;
#pragma unroll
        for (int c = 0; c < SPT; ++c) {
          stage_start(vt);
          if (c == 0) wc.scores_of(prev, fprev, psc);
          const u4 *blk = stage_blocks(vt);
          constexpr int NPAIR = BPT / 2;
          constexpr int CH = (NP + NPAIR - 1) / NPAIR;  // test slots per pair of blocks
          float pmx[NPAIR];
          u4 kv0 = blk[0], kv1 = blk[64];
#pragma unroll
          for (int i = 0; i < BPT; i += 2) {
            u4 nx0 = kv0, nx1 = kv1;
            if (i + 2 < BPT) {
              nx0 = blk[(i + 2) * 64];
              nx1 = blk[(i + 3) * 64];
            }
            const int kb = c * SB + i;
#pragma unroll
            for (int t = 0; t < QTW; ++t)
              acc[t] = MfmaMQ<DT>::run(qreg[t][kb], kv0, kb == 0 ? f4{0.f, 0.f, 0.f, 0.f} : acc[t]);
            if (c == 0) {
              const int j0 = (i / 2) * CH;
              float mm = -__builtin_inff();
#pragma unroll
              for (int j = j0; j < j0 + CH; ++j)
                if (j < NP) mm = fmaxf(mm, psc[j] - wc.thr[j]);
              pmx[i / 2] = mm;
            }
#pragma unroll
            for (int t = 0; t < QTW; ++t) acc[t] = MfmaMQ<DT>::run(qreg[t][kb + 1], kv1, acc[t]);
            kv0 = nx0;
            kv1 = nx1;
            // per pair: the next two reads, half the matrix instructions,
            // the pair's share of the test, the other half
            if (i + 2 < BPT) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, QTW, 0);
            if (c == 0) __builtin_amdgcn_sched_group_barrier(0x002, 2 * CH, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, QTW, 0);
            __builtin_amdgcn_sched_barrier(0);
          }
          if (c == 0) {
            float mx = pmx[0];
#pragma unroll
            for (int q = 1; q < NPAIR; ++q) mx = fmaxf(mx, pmx[q]);
            hits = __ballot(mx >= 0.0f) & (0ull - (uint64_t)(pv >= 0 && pv < ntile));
          }
          stage_end(vt, fcur);
        }
        if (hits) take(pv, psc);
      };
      const int nsteps = (ntile_pad + 1) / 2 * 2;  // even: the last tile is in accB
#pragma unroll 1
      for (int vt = 0; vt < nsteps; vt += 2) {
        step(vt, accA, accB, fA, fB);
        step(vt + 1, accB, accA, fB, fA);
      }
      const int64_t lt = nsteps - 1;  // the last tile's test
      if (lt < ntile) {
        float sc[NP];
        wc.scores_of(accB, fB, sc);
        if (wc.any_hit(sc)) take(lt, sc);
      }
    }
    wait_vmcnt<0>();  // no LDS copy may land after the workgroup ends
  }

  wc.publish();
}

// NWQ waves per workgroup: 4 (two workgroups per CU), or 1 holding the
// whole batch (one wave per SIMD, up to 512 registers; four workgroups per
// CU, none waiting at a barrier for another wave's candidates).
template <int DT, int QTW, int KBT, int CPQ, int S, bool FILT, int NWQ>
__global__ void __launch_bounds__(NWQ * kWaveSize, NWQ == 4 ? 2 : 1)
    dresd_scanmq_main(ScanParams p) {
  scan_mq_body<DT, QTW, KBT, CPQ, S, FILT, NWQ>(p);
}

template <int DT, int QTW, int KBT, int CPQ, int S, bool FILT, int NWQ>
__global__ void __launch_bounds__(NWQ * kWaveSize, NWQ == 4 ? 2 : 1)
    dresd_scanmq_sample(ScanParams p) {
  scan_mq_body<DT, QTW, KBT, CPQ, S, FILT, NWQ>(p);
}

// Copy one 1 KiB block at `src` into LDS at `lds` (lane l's 16 bytes to
// lds + 16 l); `nt` marks data read once (keys), which should not stay in
// the caches.  Inline assembly for the reason given at copy2_to_lds.
template <bool NT>
__device__ __forceinline__ void copy_block_to_lds(const void *src, uint32_t voff, uint32_t lds) {
  if constexpr (NT) {
    asm volatile(
        "s_mov_b32 m0, %2\n\t"
        "global_load_lds_dwordx4 %0, %1 nt"
        :
        : "v"(voff), "s"(src), "s"(lds)
        : "memory");
  } else {
    asm volatile(
        "s_mov_b32 m0, %2\n\t"
        "global_load_lds_dwordx4 %0, %1"
        :
        : "v"(voff), "s"(src), "s"(lds)
        : "memory");
  }
}

// Tiled contraction for keys wider than the shared-key scan can hold the
// queries for (more than 32 blocks per key tile), and for 32-block keys at
// batches past one shared-key launch: both operands stream through LDS.  A
// workgroup of NW = NK x NQ waves (NK key groups, NQ query groups of QTW = 4
// or 8 query tiles each) walks its key tiles in panels of NK TPW tiles.  For
// each 32-dim column of the keys one ring stage holds the panel's key blocks
// and the batch's query blocks of that column (a plain GEMM K loop); a wave
// multiplies its key group's TPW tiles by its query group's tiles, column
// after column into one accumulator per (tile, query tile) -- the same order
// in every pass and launch shape, so a key scores the same in the sampled and
// the main passes -- and after the last column tests the finished tiles
// against the thresholds.  Each key block reaches the CU once for the whole
// batch; the query operand (NQ QTW KiB per column, shared by every
// workgroup) is re-read from L2 once per panel.  Wave w issues the copies of
// panel tiles w KPW ... w KPW + KPW - 1 and of query tiles w, w + NW, ... per
// stage (past the end, the last stage again), spread over its matrix
// instructions so that the copies' address work overlaps the matrix cores;
// its wait before each stage is a constant of its copy count.  Lists: one per
// (query, key group of a workgroup).  A sampled pass (TMAX) lists only each
// tile's best key per query.  FILT: the next-token filter; each wave copies
// its tiles' first tokens into LDS with one or two more LDS-DMA copies at the
// panel's first stage (a load the compiler tracked would make it drain the
// ring at every stage), covered by the later stages' constant waits.
template <int DT, int QTW, int CPQ, int TPW, int NK, int NQ, int S, bool TMAX, bool FILT>
__device__ __forceinline__ void scan_tc_body(const ScanParams &p) {
  using WC = WaveCands<DT, QTW, CPQ, FILT, kTcCandBuf>;
  constexpr int NP = WC::NP;
  constexpr int NW = NK * NQ;   // waves: NK key groups x NQ query groups
  constexpr int PT = NK * TPW;  // key tiles per panel
  constexpr int QT = NQ * QTW;  // query tiles of the launch
  constexpr int SB = PT + QT;   // 1 KiB blocks per stage
  // copies per wave per stage: KPW key blocks and one or more query blocks
  // (or none, when there are fewer query tiles than waves)
  constexpr int KPW = PT / NW;
  constexpr int CPW_HI = KPW + (QT + NW - 1) / NW;
  constexpr int CPW_LO = KPW + QT / NW;
  constexpr int FTW = TPW * kTileRows > kWaveSize ? TPW * kTileRows : kWaveSize;
  static_assert(S >= 3 && PT % NW == 0 && (QT % NW == 0 || NW % QT == 0), "shape");
  static_assert(TPW * kTileRows <= 2 * kWaveSize, "first tokens: at most two copies per panel");
  static_assert(KPW <= 4, "32-bit key copy offsets");
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];

  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // this wave's key group and query group
  const int kg = NQ == 1 ? wv : wv % NK, qg = NQ == 1 ? 0 : wv / NK;
  const int wg = blockIdx.x;
  const int nwg = p.G / NK;
  // this wave's copies per stage
  const int cpw = QT % NW == 0 ? CPW_HI : KPW + (QT - wv + NW - 1) / NW;
  const size_t wreg = scan_mq_wave_bytes(WC::NQW, p.C, kTcCandBuf);
  // LDS: ring | one candidate region per wave | (filtered search) per wave
  // the next token of each score slot [4 lane groups][NP] | per wave the
  // first tokens of its panel tiles' rows [FTW] (TPW * 16 used)
  int32_t *nt_slot = FILT ? reinterpret_cast<int32_t *>(smem + (size_t)S * SB * kBlockBytes +
                                                        (size_t)NW * wreg) +
                                wv * 4 * NP
                          : nullptr;
  int32_t *ftb = FILT ? reinterpret_cast<int32_t *>(smem + (size_t)S * SB * kBlockBytes +
                                                    (size_t)NW * wreg) +
                            NW * 4 * NP + wv * FTW
                      : nullptr;
  // queries [qg * NQW, (qg + 1) * NQW) of the launch; one list per query
  // per key group of each workgroup
  WC wc(p, smem + (size_t)S * SB * kBlockBytes + (size_t)wv * wreg, nt_slot, qg * WC::NQW,
        wg * NK + kg);
  wc.init();
  // a query group wholly past the batch only copies its share of the ring
  const bool active = NQ == 1 || qg * WC::NQW < p.B;

  // This workgroup's key tiles: visited tiles [v0, v1).
  const int64_t v0 = wave_uniform(p.nvisit * wg / nwg);
  const int64_t v1 = wave_uniform(p.nvisit * (wg + 1) / nwg);
  const int ntile = (int)(v1 - v0);
  if (ntile > 0) {
    const int KB = p.KB;
    const int npanel = (ntile + PT - 1) / PT;
    const int64_t tstep = p.stride * KB * kBlockBytes;  // bytes between visited tiles
    const unsigned char *dbase = static_cast<const unsigned char *>(p.data) + v0 * tstep;
    const unsigned char *qbase = static_cast<const unsigned char *>(p.qop);
    const uint32_t voff = (uint32_t)lane * 16u;
    const uint32_t ring = (uint32_t)(uintptr_t)smem;
    // The copy stream runs S - 1 stages ahead of the arithmetic: stage
    // (panel npn, column nc).  Copy j < KPW of a stage is panel tile
    // wv * KPW + j (clamped to the last tile), the others query tiles wv,
    // wv + NW, ...  The key tiles' base address and clamp change once per
    // panel; per stage only the column moves.  Offsets from the base fit 32
    // bits: at most KPW - 1 <= 3 tile steps of at most 64 tiles (the
    // sparsest sampled pass) of at most 512 blocks, plus a column.
    int npn = 0, nc = 0;
    const unsigned char *kbase = dbase;
    int kjmax = 0;  // key copies past this one read the last tile
    auto set_panel = [&]() {
      const int t0 = npn * PT + wv * KPW;
      const int t0c = t0 < ntile ? t0 : ntile - 1;
      kjmax = ntile - 1 - t0c;
      kbase = dbase + (int64_t)t0c * tstep;
    };
    set_panel();
    const uint32_t tstep32 = (uint32_t)tstep;
    auto copy = [&](int j, int slot) {
      const uint32_t sbase = ring + (uint32_t)(slot * SB) * (uint32_t)kBlockBytes;
      if (j < KPW) {
        const uint32_t jj = (uint32_t)(j < kjmax ? j : kjmax);
        const int64_t src = wave_uniform((int64_t)(uintptr_t)kbase +
                                         (int64_t)(jj * tstep32 + (uint32_t)nc * kBlockBytes));
        copy_block_to_lds<true>((const void *)(uintptr_t)src, voff,
                                sbase + (uint32_t)(wv * KPW + j) * (uint32_t)kBlockBytes);
      } else {
        const int qt = wv + NW * (j - KPW);
        const int64_t src = wave_uniform((int64_t)(uintptr_t)qbase +
                                         (int64_t)((uint32_t)(qt * KB + nc) * kBlockBytes));
        copy_block_to_lds<false>((const void *)(uintptr_t)src, voff,
                                 sbase + (uint32_t)(PT + qt) * (uint32_t)kBlockBytes);
      }
    };
    // Stages in order: (panel, column) with the column fastest; past the
    // last stage the copies repeat it.
    auto advance = [&]() {
      if (npn < npanel - 1 || nc < KB - 1) {
        if (++nc == KB) {
          nc = 0;
          ++npn;
          set_panel();
        }
      }
    };
#pragma unroll
    for (int st = 0; st < S - 1; ++st) {
#pragma unroll
      for (int j = 0; j < CPW_HI; ++j)
        if (j < cpw) copy(j, st);
      advance();
    }
    int next_slot = S - 1;  // ring slot of the next stage to copy
    int cur_slot = 0;       // ring slot of the stage being consumed
    f4 acc[TPW][QTW];
    // Operand prefetch (query-group kernels with four or more stages): a
    // stage's barrier also covers the next stage's copies, and each operand
    // register is refilled with the next stage's block once this stage's
    // last instruction reading it has issued, so that one stage's LDS reads
    // overlap the matrix instructions of the stage before.  Without it all
    // waves read their operands from LDS at once after the barrier, then
    // run their instructions.
    constexpr bool PF = NQ > 1 && S >= 4;
    constexpr int NO = TPW > QTW ? TPW : QTW;    // outer blocks
    constexpr int CPO = (CPW_HI + NO - 1) / NO;  // copies after each outer block's instructions
    u4 kv[TPW], qv[QTW];
    auto slot_ops = [&](int slot) {
      return reinterpret_cast<const u4 *>(smem + (size_t)slot * SB * kBlockBytes) + lane;
    };
    // The operand blocks of the smaller side are read first and the
    // instructions run over the larger side outermost, so that they can
    // start once one block of the larger side has arrived.
    auto read_inner = [&](const u4 *sl) {
      if constexpr (TPW > QTW) {
#pragma unroll
        for (int t = 0; t < QTW; ++t) qv[t] = sl[(PT + qg * QTW + t) * 64];
      } else {
#pragma unroll
        for (int i = 0; i < TPW; ++i) kv[i] = sl[(kg * TPW + i) * 64];
      }
    };
    auto read_outer = [&](const u4 *sl, int o) {
      if constexpr (TPW > QTW) kv[o] = sl[(kg * TPW + o) * 64];
      else qv[o] = sl[(PT + qg * QTW + o) * 64];
    };
    if constexpr (PF) {
      // stage 0 has landed and is visible; its operands into registers
      if (CPW_HI == CPW_LO || cpw == CPW_HI) wait_vmcnt<CPW_HI * (S - 2)>();
      else wait_vmcnt<CPW_LO * (S - 2)>();
      __syncthreads();
      if (active) {
        read_inner(slot_ops(0));
#pragma unroll
        for (int o = 0; o < NO; ++o) read_outer(slot_ops(0), o);
      }
    }
#pragma unroll 1
    for (int pn = 0; pn < npanel; ++pn) {
#pragma unroll
      for (int i = 0; i < TPW; ++i)
#pragma unroll
        for (int t = 0; t < QTW; ++t) acc[i][t] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll 1
      for (int c = 0; c < KB; ++c) {
        // this wave's copies of the stage (and with prefetch of the next
        // one) have landed, those of the later stages may still be in
        // flight; after the barrier so have every wave's, and the slot
        // consumed last is free again
        constexpr int WST = PF ? S - 3 : S - 2;
        if (CPW_HI == CPW_LO || cpw == CPW_HI) wait_vmcnt<CPW_HI * WST>();
        else wait_vmcnt<CPW_LO * WST>();
        __syncthreads();
        if (FILT && c == 0 && active) {
          // first tokens of this wave's tiles of the panel (lane l of copy
          // h: tile 4 h + l / 16, row l % 16; clamped to the last tile;
          // lanes past TPW tiles copy unused values), read after the
          // panel's last column.  Issued before this stage's copies, they
          // are complete once the next stage's wait leaves at most CPW
          // copies in flight.
#pragma unroll
          for (int h = 0; h < (TPW > 4 ? 2 : 1); ++h) {
            int64_t t = pn * PT + kg * TPW + 4 * h + (lane >> 4);
            t = t < ntile ? t : ntile - 1;
            copy1_to_lds(p.ftok + (v0 + t) * p.stride * kTileRows + (lane & 15),
                         (uint32_t)(uintptr_t)(ftb + h * kWaveSize));
          }
        }
        if (active) {
          // the next stage's operands (prefetch)
          const u4 *sn = slot_ops(cur_slot == S - 1 ? 0 : cur_slot + 1);
          if constexpr (!PF) {
            const u4 *sl = slot_ops(cur_slot);
            read_inner(sl);
#pragma unroll
            for (int o = 0; o < NO; ++o) read_outer(sl, o);
          }
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int o = 0; o < NO; ++o) {
            if constexpr (TPW > QTW) {
#pragma unroll
              for (int t = 0; t < QTW; ++t) acc[o][t] = MfmaMQ<DT>::run(qv[t], kv[o], acc[o][t]);
            } else {
#pragma unroll
              for (int i = 0; i < TPW; ++i) acc[i][o] = MfmaMQ<DT>::run(qv[o], kv[i], acc[i][o]);
            }
            if constexpr (PF) read_outer(sn, o);
            if (o * CPO < CPW_HI) {
              // the stage S - 1 ahead, CPO copies per outer block
              __builtin_amdgcn_sched_barrier(0);
#pragma unroll
              for (int j = o * CPO; j < (o + 1) * CPO && j < CPW_HI; ++j)
                if (j < cpw) copy(j, next_slot);
              __builtin_amdgcn_sched_barrier(0);
            }
          }
          if constexpr (PF) read_inner(sn);
        } else {
#pragma unroll
          for (int j = 0; j < CPW_HI; ++j)
            if (j < cpw) copy(j, next_slot);
        }
        advance();
        next_slot = next_slot == S - 1 ? 0 : next_slot + 1;
        cur_slot = cur_slot == S - 1 ? 0 : cur_slot + 1;
      }
      if (active) {
        int ft[TPW];  // filtered search: this lane's row's first token per tile
#pragma unroll
        for (int i = 0; i < TPW; ++i) ft[i] = FILT ? ftb[i * kTileRows + (lane & 15)] : 0;
#pragma unroll
        for (int i = 0; i < TPW; ++i) {
          const int vt = pn * PT + kg * TPW + i;
          if (vt < ntile) {
            float sc[NP];
            wc.scores_of(acc[i], ft[i], sc);
            if (TMAX) wc.template take_tile_max<(TPW >= 4)>((v0 + vt) * p.stride, sc);
            else if (wc.any_hit(sc)) wc.take((v0 + vt) * p.stride, sc);
          }
        }
      }
    }
    wait_vmcnt<0>();  // no LDS copy may land after the workgroup ends
  }
  wc.publish();
}

template <int DT, int QTW, int CPQ, int TPW, int NK, int NQ, int S, bool FILT>
__global__ void __launch_bounds__(NK * NQ * kWaveSize, 8 / (NK * NQ))
    dresd_scantc_main(ScanParams p) {
  scan_tc_body<DT, QTW, CPQ, TPW, NK, NQ, S, false, FILT>(p);
}

// Sampled pass: per-tile maxima as candidates.
template <int DT, int QTW, int CPQ, int TPW, int NK, int NQ, int S, bool FILT>
__global__ void __launch_bounds__(NK * NQ * kWaveSize, 8 / (NK * NQ))
    dresd_scantc_sample(ScanParams p) {
  scan_tc_body<DT, QTW, CPQ, TPW, NK, NQ, S, true, FILT>(p);
}

// One thread per 16-byte chunk (t, kb, lane) of the query operands.
template <int DT, int CPQ>
__global__ void __launch_bounds__(256) dresd_query_operand(QopParams p) {
  const int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (c >= (int64_t)p.ntile * p.KB * 64) return;
  const int lane = (int)(c & 63);
  const int kb = (int)((c >> 6) % p.KB);
  const int t = (int)((c >> 6) / p.KB);
  const bool vec = (((uintptr_t)p.queries & 15u) == 0) && ((p.d & 3) == 0);
  static_cast<u4 *>(p.out)[c] = query_chunk_mq<DT, CPQ>(p.queries, p.d, p.B, t * 16 + (lane & 15),
                                                        kb * 32 + (lane >> 4) * 8, vec);
}

// (QTW, KBT) pairs with QTW * KBT <= 32 (query operands <= 128 VGPRs), each
// with its ring depth S.
#define DRESD_MQ_CASE_W(DT, CPQ, QTW, KBT, S, NWQ)                                           \
  if (qtw == QTW && kbt == KBT && nwq == NWQ) {                                             \
    *stages = S;                                                                            \
    if (filtered)                                                                           \
      return main_pass ? (ScanKernel)dresd_scanmq_main<DT, QTW, KBT, CPQ, S, true, NWQ>     \
                       : (ScanKernel)dresd_scanmq_sample<DT, QTW, KBT, CPQ, S, true, NWQ>;  \
    return main_pass ? (ScanKernel)dresd_scanmq_main<DT, QTW, KBT, CPQ, S, false, NWQ>      \
                     : (ScanKernel)dresd_scanmq_sample<DT, QTW, KBT, CPQ, S, false, NWQ>;   \
  }
#define DRESD_MQ_CASE(DT, CPQ, QTW, KBT, S) DRESD_MQ_CASE_W(DT, CPQ, QTW, KBT, S, 4)
#define DRESD_MQ_ALL(DT, CPQ)                                                     \
  DRESD_MQ_CASE(DT, CPQ, 1, 4, 4) DRESD_MQ_CASE(DT, CPQ, 1, 8, 4)                 \
  DRESD_MQ_CASE(DT, CPQ, 1, 16, 4) DRESD_MQ_CASE(DT, CPQ, 1, 32, 6)               \
  DRESD_MQ_CASE(DT, CPQ, 2, 4, 4) DRESD_MQ_CASE(DT, CPQ, 2, 8, 4)                 \
  DRESD_MQ_CASE(DT, CPQ, 2, 16, 6) DRESD_MQ_CASE(DT, CPQ, 4, 4, 4)                \
  DRESD_MQ_CASE(DT, CPQ, 4, 8, 6) DRESD_MQ_CASE_W(DT, CPQ, 4, 8, 4, 1)

// Tiled contraction, one query group (NQ = 1): main passes with 4 key
// tiles per wave, 8 waves (3 stages: one query read per 32 key tiles) or 4
// waves (5 stages, or 3 where large lists leave less LDS); sampled passes
// with 1 key tile per wave and 4 waves (8 or 4 stages).  Larger batches: 2
// or 4 query groups of waves over 16-tile panels (8 waves), sampled passes
// over 8-tile panels (4 stages).
#define DRESD_TC_MAIN(DT, CPQ, QTW, TPW, NK, NQ, S)                                        \
  if (main_pass && qtw == QTW && tpw == TPW && nk == NK && nq == NQ && stages == S)      \
    return filtered ? (ScanKernel)dresd_scantc_main<DT, QTW, CPQ, TPW, NK, NQ, S, true>  \
                    : (ScanKernel)dresd_scantc_main<DT, QTW, CPQ, TPW, NK, NQ, S, false>;
#define DRESD_TC_SAMPLE(DT, CPQ, QTW, TPW, NK, NQ, S)                                       \
  if (!main_pass && qtw == QTW && tpw == TPW && nk == NK && nq == NQ && stages == S)      \
    return filtered ? (ScanKernel)dresd_scantc_sample<DT, QTW, CPQ, TPW, NK, NQ, S, true>  \
                    : (ScanKernel)dresd_scantc_sample<DT, QTW, CPQ, TPW, NK, NQ, S, false>;
#define DRESD_TC_ONE(DT, CPQ, QTW)                                                      \
  DRESD_TC_MAIN(DT, CPQ, QTW, 4, 8, 1, 3)                                               \
  DRESD_TC_MAIN(DT, CPQ, QTW, 4, 4, 1, 5) DRESD_TC_MAIN(DT, CPQ, QTW, 4, 4, 1, 3)       \
  DRESD_TC_SAMPLE(DT, CPQ, QTW, 1, 4, 1, 8) DRESD_TC_SAMPLE(DT, CPQ, QTW, 1, 4, 1, 4)

#if !defined(DRESD_MQ_TU) || DRESD_MQ_TU == 0
ScanKernel scan_tc_kernel_f16(int qtw, int tpw, int nk, int nq, int stages, bool main_pass,
                              bool filtered) {
  DRESD_TC_ONE(kF16, 1, 4)
  DRESD_TC_MAIN(kF16, 1, 4, 4, 4, 2, 4) DRESD_TC_MAIN(kF16, 1, 4, 4, 4, 2, 3)
  DRESD_TC_SAMPLE(kF16, 1, 4, 2, 4, 2, 4)
  DRESD_TC_MAIN(kF16, 1, 4, 8, 2, 4, 4) DRESD_TC_MAIN(kF16, 1, 4, 8, 2, 4, 3)
  DRESD_TC_SAMPLE(kF16, 1, 4, 4, 2, 4, 4)
  return nullptr;
}
#endif
#if !defined(DRESD_MQ_TU) || DRESD_MQ_TU == 1
ScanKernel scan_tc_kernel_bf16(int qtw, int tpw, int nk, int nq, int stages, bool main_pass,
                               bool filtered) {
  DRESD_TC_ONE(kBF16, 2, 4)
  DRESD_TC_ONE(kBF16, 2, 8)
  DRESD_TC_MAIN(kBF16, 2, 8, 4, 4, 2, 4) DRESD_TC_MAIN(kBF16, 2, 8, 4, 4, 2, 3)
  DRESD_TC_SAMPLE(kBF16, 2, 8, 2, 4, 2, 4)
  return nullptr;
}
#endif

#if !defined(DRESD_MQ_TU) || DRESD_MQ_TU == 0
ScanKernel scan_mq_kernel_f16(int qtw, int kbt, bool main_pass, bool filtered, int *stages,
                              int nwq) {
  DRESD_MQ_ALL(kF16, 1)
  return nullptr;
}
void *qop_kernel_f16() { return (void *)dresd_query_operand<kF16, 1>; }
#endif
#if !defined(DRESD_MQ_TU) || DRESD_MQ_TU == 1
ScanKernel scan_mq_kernel_bf16(int qtw, int kbt, bool main_pass, bool filtered, int *stages,
                               int nwq) {
  DRESD_MQ_ALL(kBF16, 2)
  return nullptr;
}
void *qop_kernel_bf16() { return (void *)dresd_query_operand<kBF16, 2>; }
#endif

}  // namespace dresd
