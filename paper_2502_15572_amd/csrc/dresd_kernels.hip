// gfx950 kernels for exact dense retrieval (DReSD Section 3.5, Eq. 3 with
// unit-norm keys and queries, Section 3.4, Eq. 2: the cosine is the inner
// product; the argmax is taken as the k best keys, Section 3.6).
//
//   layout : one-time copy of row-major keys into 16-row MFMA tiles.
//   scan   : streams the tiles once; MFMA scores (queries as the A operand,
//            key rows as the B operand); a per-query threshold filter; a
//            per-wave bounded candidate list, re-selected in LDS when full
//            and cut to its k best at the end.
// The merge that turns the per-wave lists into the answer is in
// dresd_merge.hip.
#include "dresd_scan_common.h"

namespace dresd {

// ---------------------------------------------------------------- layout ---

template <typename T>
__global__ void __launch_bounds__(256) dresd_layout(LayoutParams p) {
  constexpr int EPC = 16 / sizeof(T);  // elements per 16-byte chunk
  const T *src = static_cast<const T *>(p.src);
  u4 *dst = static_cast<u4 *>(p.dst);
  for (int64_t c = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; c < p.chunks;
       c += (int64_t)gridDim.x * blockDim.x) {
    int64_t per_tile = (int64_t)p.KB * 64;
    int64_t tile = c / per_tile;
    int r = (int)(c - tile * per_tile);
    int kb = r >> 6, ln = r & 63;
    int64_t row = tile * kTileRows + (ln & 15);
    if (p.slot_row) {  // partitioned layout: the slot's row, or padding
      const uint32_t r = p.slot_row[row];
      row = r == kPadRow ? p.N : (int64_t)r;
    }
    int dim0 = kb * 4 * EPC + (ln >> 4) * EPC;
    union {
      T e[EPC];
      u4 v;
    } u;
#pragma unroll
    for (int e = 0; e < EPC; ++e) {
      int dim = dim0 + e;
      u.e[e] = (row < p.N && dim < p.d) ? src[row * p.d + dim] : T(0);
    }
    dst[c] = u.v;
  }
}

// ------------------------------------------------------------------ scan ---

template <int DT>
struct Mfma;

template <>
struct Mfma<kF32> {
  __device__ __forceinline__ static f4 run(u4 a, u4 b, f4 acc) {
#pragma unroll
    for (int c = 0; c < 4; ++c)
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[c]), __uint_as_float(b[c]),
                                                 acc, 0, 0, 0);
    return acc;
  }
};

template <>
struct Mfma<kF16> {
  __device__ __forceinline__ static f4 run(u4 a, u4 b, f4 acc) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(h8, a),
                                                  __builtin_bit_cast(h8, b), acc, 0, 0, 0);
  }
};

template <>
struct Mfma<kBF16> {
  __device__ __forceinline__ static f4 run(u4 a, u4 b, f4 acc) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(b8, a),
                                                   __builtin_bit_cast(b8, b), acc, 0, 0, 0);
  }
};

// Query operand: CPQ consecutive columns of the A operand hold one query.
// CPQ = 1: the query itself (fp32 keys) or rounded once to f16;
// CPQ = 2: bf16 keys, two parts: high and the rounded remainder (their sum
//          is the query within 2^-17 relative);
// CPQ = 4: three parts whose sum is the fp32 query exactly, plus a zero
//          column.  bf16: high, middle, low.  f16: high, then the remainders
//          scaled by 2^11 and 2^22 so they stay in f16's normal range (the
//          epilogue scales their products back by the same powers of two).
template <int DT, int CPQ>
__device__ __forceinline__ u4 query_chunk(const float *q, int d, int B, int col, int dim0) {
  u4 out;
  const int b = col / CPQ;
  const int h = col % CPQ;
  if (DT == kF32) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      int dim = dim0 + e;
      float x = (b < B && dim < d) ? q[(int64_t)b * d + dim] : 0.0f;
      out[e] = __float_as_uint(x);
    }
    return out;
  }
  uint16_t v[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    int dim = dim0 + e;
    float x = (b < B && dim < d) ? q[(int64_t)b * d + dim] : 0.0f;
    if (DT == kF16) {
      _Float16 hi = (_Float16)x;
      _Float16 r = hi;
      if (CPQ == 4) {
        float r1 = x - (float)hi;                       // exact
        _Float16 mid = (_Float16)(r1 * 2048.0f);        // 2^11
        float r2 = r1 - (float)mid * (1.0f / 2048.0f);  // exact
        _Float16 lo = (_Float16)(r2 * 4194304.0f);      // 2^22
        r = (h == 0) ? hi : (h == 1) ? mid : (h == 2) ? lo : (_Float16)0.0f;
      }
      v[e] = __builtin_bit_cast(uint16_t, r);
    } else {
      __bf16 hi = (__bf16)x;
      float r1 = x - (float)hi;
      __bf16 mid = (__bf16)r1;
      __bf16 lo = (__bf16)(r1 - (float)mid);
      __bf16 r = (h == 0) ? hi : (h == 1) ? mid : (CPQ == 4 && h == 2) ? lo : (__bf16)0.0f;
      v[e] = __builtin_bit_cast(uint16_t, r);
    }
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) out[e] = (uint32_t)v[2 * e] | ((uint32_t)v[2 * e + 1] << 16);
  return out;
}

// Scan modes: the main pass over every tile, a sampled threshold pass over
// every stride-th tile, and the partitioned search (each workgroup serves one
// query and walks the tiles of the partitions that query probes).
constexpr int kModeMain = 0, kModeSample = 1, kModeParts = 2;

// `gw` is the wave's list within its query (or batch); seg_off / seg_tile
// are the query's probed segments in the partitioned search.
// SHARED: a launch of several query groups whose workgroups read each key
// range together (see scan_group_view).  Its key loads are cached, so that
// the XCD's L2 keeps a block for the range's other readers, and 16 deep:
// most of them wait on a line already in flight from HBM.  A lone reader
// streams past the cache (nontemporal loads, 8 deep).
template <int DT, int QT, int CPQ, int MODE, bool SHARED = false>
__device__ __forceinline__ void scan_body(const ScanParams &p, const int gw,
                                          const int32_t *seg_off, const int32_t *seg_tile) {
  constexpr bool MAIN = MODE == kModeMain;
  constexpr bool PARTS = MODE == kModeParts;
  constexpr int QPT = 16 / CPQ;  // queries per 16-column tile
  constexpr int NS = 4 / CPQ;    // scores per lane per tile
  constexpr int NQ = QT * QPT;   // queries held by one launch
  constexpr int U = SHARED ? 16 : 8;  // key blocks in flight per wave
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];

  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform
  const int G = p.G, C = p.C, KB = p.KB, B = p.B;
  const int ncols = B * CPQ;
  const int g = lane >> 4, m = lane & 15;

  // LDS carve-up: query operand | zero chunk | next tokens of the queries |
  // one candidate region per wave (staged keys, sort scratch, thresholds,
  // counters)
  const int qop_bytes = ncols * KB * 64;
  const int zero_off = qop_bytes;
  const int CL = p.CL;
  int32_t *nt_lds = reinterpret_cast<int32_t *>(smem + qop_bytes + 16);
  CandSink sink;
  sink.stg = reinterpret_cast<uint64_t *>(smem + qop_bytes + 16 + scan_ntok_bytes(NQ) +
                                          (size_t)wv * scan_wave_bytes(NQ, CL, C));
  sink.scr = sink.stg + (size_t)NQ * CL;
  sink.st_key = sink.scr + C;
  sink.st_cnt = reinterpret_cast<uint32_t *>(sink.st_key + NQ);
  sink.st_thr = reinterpret_cast<float *>(sink.st_cnt + NQ);
  sink.stg_cnt = reinterpret_cast<uint32_t *>(sink.st_thr + NQ);
  sink.cl = CL;
  sink.C = C;
  sink.k = p.k;
  sink.lane = lane;
  auto list_of = [&](int q) { return p.lists + ((size_t)q * G + gw) * C; };

  // 1. Query operand, in the lane order of the A operand.
  {
    constexpr int EPC = (DT == kF32) ? 4 : 8;
    const int entries = ncols * KB * 4;
    for (int e = threadIdx.x; e < entries; e += blockDim.x) {
      int c = e / (KB * 4);
      int r = e - c * (KB * 4);
      int kb = r >> 2, gg = r & 3;
      int t = c >> 4, mm = c & 15;
      int nct = min(16, ncols - 16 * t);
      int off = t * 16 * KB * 64 + ((kb * 4 + gg) * nct + mm) * 16;
      *reinterpret_cast<u4 *>(smem + off) =
          query_chunk<DT, CPQ>(p.queries, p.d, B, c, kb * 4 * EPC + gg * EPC);
    }
    if (threadIdx.x == 0) *reinterpret_cast<u4 *>(smem + zero_off) = u4{0, 0, 0, 0};
    if (p.next_tok)
      for (int q = threadIdx.x; q < NQ; q += blockDim.x) nt_lds[q] = q < B ? p.next_tok[q] : 0;
  }
  // 2. Per-wave state: thresholds start at the pass's tau (or none).
  sink_init(sink, NQ, B, p.tau);
  __syncthreads();

  // Per-lane A-operand addresses: column m of tile t, or the zero chunk.
  int qa0[QT], qstep[QT];
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    int nct = ncols - 16 * t;
    nct = nct > 16 ? 16 : nct;
    if (m < nct) {
      qa0[t] = t * 16 * KB * 64 + (g * nct + m) * 16;
      qstep[t] = 4 * nct * 16;
    } else {
      qa0[t] = zero_off;
      qstep[t] = 0;
    }
  }
  float thr[QT][NS];
#pragma unroll
  for (int t = 0; t < QT; ++t)
#pragma unroll
    for (int s = 0; s < NS; ++s) thr[t][s] = sink.st_thr[t * QPT + g * NS + s];

  // 3. Stream this wave's tiles.  Everything that steers the loop is
  // wave-uniform (scalar registers), so control flow never masks lanes.
  // Ring slot u is consumed by its MFMA and then reloaded with the block U
  // steps ahead, so no register is copied and U loads stay in flight.
  // Reloads past the wave's last block re-read that block (in bounds, and
  // served from cache) instead of branching.  The main pass visits every
  // tile, so its blocks are one contiguous run; a sampled pass jumps
  // `stride` tiles after each visited one.
  // Partitioned search: the probed partitions' tiles, in probe order, form
  // the query's virtual tile sequence [0, seg_off[S]); segment j (partition
  // probe j) is virtual tiles [seg_off[j], seg_off[j+1]) starting at physical
  // tile seg_tile[j].  The waves of the query split the sequence evenly.
  const int64_t vtot = PARTS ? (int64_t)seg_off[p.S] : p.nvisit;
  const int64_t v0 = wave_uniform(vtot * gw / G);
  const int64_t v1 = wave_uniform(vtot * (gw + 1) / G);
  const int64_t J = (v1 - v0) * KB;
  const u4 *base = static_cast<const u4 *>(p.data) + lane;
  // Two cursors walk the segments: one for block loads (ahead of use), one
  // for the tile being finished.  Each holds its segment, its position and
  // what is left of the segment.
  int lseg = 0, cseg = 0;
  int64_t lrem = 0, crem = 0;  // blocks (loads) / tiles (finish) left in the segment
  const u4 *lptr = base;
  int64_t lnext = 0;           // index of the block the load cursor points at
  auto seg_len = [&](int j) -> int64_t { return (int64_t)seg_off[j + 1] - seg_off[j]; };
  auto next_seg = [&](int j) -> int {
    do ++j;
    while (seg_len(j) == 0);
    return j;
  };
  if constexpr (PARTS) {
    if (J > 0) {
      int j = 0;
      while ((int64_t)seg_off[j + 1] <= v0) ++j;
      lseg = cseg = j;
      lptr = base + ((int64_t)seg_tile[j] + (v0 - seg_off[j])) * KB * 64;
      lrem = ((int64_t)seg_off[j + 1] - v0) * KB;
      crem = (int64_t)seg_off[j + 1] - v0;
    }
  }
  auto block = [&](int64_t i) -> const u4 * {
    if constexpr (PARTS) {
      // Calls come in order i = 0, 1, 2, ...; past the last block the
      // cursor stays on it (an in-bounds re-read, served from cache).
      const u4 *r = lptr;
      if (lnext + 1 < J) {
        ++lnext;
        lptr += 64;
        if (--lrem == 0) {
          lseg = next_seg(lseg);
          lptr = base + (int64_t)seg_tile[lseg] * KB * 64;
          lrem = seg_len(lseg) * KB;
        }
      }
      return r;
    }
    i = i < J ? i : J - 1;
    if (MAIN) return base + (v0 * KB + i) * 64;
    const int64_t vt = i / KB;
    return base + ((v0 + vt) * p.stride * KB + (i - vt * KB)) * 64;
  };
  auto fetch = [](const u4 *a) -> u4 {
    if constexpr (SHARED) return *a;
    else return __builtin_nontemporal_load(a);
  };
  u4 ring[U];
  if (J > 0) {
#pragma unroll
    for (int u = 0; u < U; ++u) ring[u] = fetch(block(u));
  }
  f4 acc[QT];
#pragma unroll
  for (int t = 0; t < QT; ++t) acc[t] = f4{0.f, 0.f, 0.f, 0.f};
  int64_t ctile = PARTS ? (J > 0 ? (int64_t)seg_tile[cseg] + (v0 - seg_off[cseg]) : 0)
                        : v0 * p.stride;
  int ckb = 0;

  // Filtered search (Section 3.5): the first tokens of a group of four
  // tiles (64 rows, lane l: row l % 16 of tile 4 i + l / 16) are copied into
  // one of two per-wave LDS slots by an LDS-DMA copy issued a whole group
  // ahead of use: the copy of group i + 2 at the end of tile 4 i + 3, read
  // from the end of tile 4 i + 8 on.  By then the loads of 5 tiles and one
  // more copy are younger, so waiting for at most U pending operations
  // covers it when 5 KB + 1 >= U.  The first group's copy has only the
  // second copy and the first tile's KB loads behind it (KB + 1 >= U).  Where
  // that does not hold, and in the last, partial group of blocks (which
  // issues no loads), the wait is for all of them.
  const bool filt = !PARTS && p.ftok != nullptr;
  const int64_t ntw = v1 - v0;  // tiles of this wave
  int64_t tdone = 0;            // tiles finished (wave-uniform)
  // two 64-entry slots per wave, after the waves' candidate regions
  int32_t *ftbuf = reinterpret_cast<int32_t *>(smem + qop_bytes + 16 + scan_ntok_bytes(NQ) +
                                               (size_t)4 * scan_wave_bytes(NQ, CL, C)) +
                   wv * 128;
  const uint32_t ftbuf_lds = (uint32_t)(uintptr_t)ftbuf;  // low half of an LDS address
  auto ftok_group = [&](int64_t grp) {
    int64_t vt = grp * 4 + (lane >> 4);
    vt = vt < ntw ? vt : ntw - 1;
    copy1_to_lds(p.ftok + (v0 + vt) * p.stride * kTileRows + (lane & 15),
                 ftbuf_lds + (uint32_t)(grp & 1) * 256u);
  };
  if (filt && ntw > 0) {
    ftok_group(0);
    ftok_group(1);
  }

  // A operands from LDS.  Up to 4 query tiles they are read one block ahead
  // (the next block's reads are in flight while this block's matrix
  // instructions run), so the LDS latency is not paid once per tile per
  // block; more tiles read them just in time (registers).
  constexpr bool PIPE = QT <= 4;
  auto read_a = [&](int kb, u4 (&a)[PIPE ? QT : 1]) {
#pragma unroll
    for (int t = 0; t < (PIPE ? QT : 1); ++t)
      a[t] = *reinterpret_cast<const u4 *>(smem + qa0[t] + kb * qstep[t]);
  };
  u4 a_cur[PIPE ? QT : 1];
  if (PIPE) read_a(0, a_cur);
  auto mfma_block = [&](const u4 &blk) {
    if constexpr (PIPE) {
      u4 a_nxt[QT];
      read_a(ckb + 1 == KB ? 0 : ckb + 1, a_nxt);
#pragma unroll
      for (int t = 0; t < QT; ++t) acc[t] = Mfma<DT>::run(a_cur[t], blk, acc[t]);
#pragma unroll
      for (int t = 0; t < QT; ++t) a_cur[t] = a_nxt[t];
    } else {
#pragma unroll
      for (int t = 0; t < QT; ++t) {
        u4 a = *reinterpret_cast<const u4 *>(smem + qa0[t] + ckb * qstep[t]);
        acc[t] = Mfma<DT>::run(a, blk, acc[t]);
      }
    }
  };
  // Tile epilogue: threshold filter, rare slow path, reset for the next tile.
  auto tile_end = [&](bool tail) {
    // Partitioned layout: a slot's row is known only from the slot table,
    // read when a score passes (padding slots hold kPadRow).
    const int64_t row64 = ctile * kTileRows + m;
    bool row_ok = PARTS || row64 < p.N;
    uint32_t row = (uint32_t)row64;
    float sc[QT][NS];
    bool any = false;
#pragma unroll
    for (int t = 0; t < QT; ++t)
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        float v = acc[t][s * CPQ];
        if (CPQ == 4) {
          const float s1 = (DT == kF16) ? (1.0f / 2048.0f) : 1.0f;
          const float s2 = (DT == kF16) ? (1.0f / 4194304.0f) : 1.0f;
          v = (v + acc[t][s * CPQ + 1] * s1) + acc[t][s * CPQ + 2] * s2;
        } else if (CPQ == 2) {
          v = v + acc[t][s * CPQ + 1];
        }
        sc[t][s] = v;
      }
    if (filt) {
      // Rows whose value does not start with the query's next token drop
      // out: their score becomes NaN, which fails every threshold test
      // (even a threshold of -inf).
      const int tg = (int)(tdone & 3);
      if (tg == 0) {
        if (tail || (tdone == 0 ? KB + 1 < U : 5 * KB + 1 < U)) wait_vmcnt<0>();
        else wait_vmcnt<U>();
      }
      const int f = ftbuf[(int)((tdone >> 2) & 1) * 64 + tg * 16 + m];
#pragma unroll
      for (int t = 0; t < QT; ++t)
#pragma unroll
        for (int s = 0; s < NS; ++s)
          if (f != nt_lds[t * QPT + g * NS + s]) sc[t][s] = __builtin_nanf("");
      if (tg == 3) ftok_group((tdone >> 2) + 2);  // the slot just finished
    }
    ++tdone;
#pragma unroll
    for (int t = 0; t < QT; ++t)
#pragma unroll
      for (int s = 0; s < NS; ++s) any |= row_ok && sc[t][s] >= thr[t][s];
    if (__ballot(any)) {
      if constexpr (PARTS) {
        // the slot's row; with the next-token filter (Section 3.5), only a
        // row whose value starts with the query's next token
        const int64_t slot = ctile * kTileRows + m;
        row = p.slot_row[slot];
        row_ok = row != kPadRow && (p.ftok == nullptr || p.ftok[slot] == nt_lds[0]);
      }
      bool spilled = false;
#pragma unroll
      for (int t = 0; t < QT; ++t)
#pragma unroll
        for (int s = 0; s < NS; ++s) {
          const bool ps = row_ok && sc[t][s] >= thr[t][s];
          uint64_t mk = __ballot(ps);
          while (mk) {
            const int gg = (__ffsll((long long)mk) - 1) >> 4;
            const int q = t * QPT + gg * NS + s;
            spilled |= sink_offer(sink, q, ps && (g == gg), make_key(sc[t][s], row), list_of(q));
            mk &= ~(0xFFFFull << (16 * gg));
          }
        }
#pragma unroll
      for (int t = 0; t < QT; ++t)
#pragma unroll
        for (int s = 0; s < NS; ++s) thr[t][s] = sink.st_thr[t * QPT + g * NS + s];
      // A spill used vector memory: drain it here, so that afterwards the only
      // loads in flight are the ring's and the fast path keeps exact waits.
      if (spilled) __threadfence_block();
    }
#pragma unroll
    for (int t = 0; t < QT; ++t) acc[t] = f4{0.f, 0.f, 0.f, 0.f};
    ckb = 0;
    if constexpr (PARTS) {
      ++ctile;
      if (--crem == 0 && tdone < ntw) {
        cseg = next_seg(cseg);
        ctile = seg_tile[cseg];
        crem = seg_len(cseg);
      }
    } else {
      ctile += p.stride;
    }
  };
  // Whole groups of U blocks: every step issues exactly one load, so the
  // wait before each MFMA is a fixed count on every path.
  int64_t j = 0;
  for (; j + U <= J; j += U) {
    const int64_t jj = wave_uniform(j);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      mfma_block(ring[u]);
      ring[u] = fetch(block(jj + u + U));
      if (++ckb == KB) tile_end(false);
    }
  }
  // The last partial group: its blocks are already in the ring.
#pragma unroll
  for (int u = 0; u < U; ++u) {
    if (j + u < J) {
      mfma_block(ring[u]);
      if (++ckb == KB) tile_end(true);
    }
  }

  if (filt) wait_vmcnt<0>();  // no LDS copy may land after the workgroup ends

  // 4. Publish the lists: lists holding more than k keys are cut to their k
  // best (every list is sorted with sort_lists); each publishes its length,
  // best key and k-th key, with which the merge bounds the answer.
  for (int q = 0; q < B; ++q) {
    const size_t o = (size_t)q * G + gw;
    sink_publish(sink, q, list_of(q), p.sort_lists != 0, p.lcnt + o, p.lfirst + o, p.lkth + o);
  }
}

// The workgroup's query group and key range, and its waves' list index.
// With several groups per launch, each group's R = gridDim.x / ngroups
// workgroups split the key tiles into R ranges, and the ngroups workgroups
// of one range sit next to each other in dispatch order on one XCD
// (workgroups are dispatched round-robin over the 8 XCDs): they stream the
// same keys at about the same time, so that XCD's L2 serves the re-reads.
__device__ __forceinline__ int scan_group_view(ScanParams &p) {
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int nwv = blockDim.x >> 6;
  const int ng = p.ngroups;
  if (ng <= 1) return (int)blockIdx.x * nwv + wv;
  const int R = (int)gridDim.x / ng;
  int gi, r;
  if ((R & 7) == 0) {
    const int x = (int)blockIdx.x & 7, j = (int)blockIdx.x >> 3;
    gi = j % ng;
    r = (j / ng) * 8 + x;
  } else {
    gi = (int)blockIdx.x % ng;
    r = (int)blockIdx.x / ng;
  }
  // (readfirstlane: the values are wave-uniform, and LDS addresses derived
  // from the group size must stay in scalar registers)
  const int b0 = __builtin_amdgcn_readfirstlane((int)((int64_t)p.B * gi / ng));
  const int b1 = __builtin_amdgcn_readfirstlane((int)((int64_t)p.B * (gi + 1) / ng));
  p.queries += (size_t)b0 * p.d;
  p.lists += (size_t)b0 * p.G * p.C;
  p.lcnt += (size_t)b0 * p.G;
  p.lkth += (size_t)b0 * p.G;
  p.lfirst += (size_t)b0 * p.G;
  if (p.tau) p.tau += b0;
  if (p.next_tok) p.next_tok += b0;
  p.B = b1 - b0;
  return __builtin_amdgcn_readfirstlane(r) * nwv + wv;
}

// Two kernel names so that profiles separate the main pass from the
// sampled passes that only set thresholds.
template <int DT, int QT, int CPQ>
__global__ void __launch_bounds__(kScanThreads) dresd_scan_main(ScanParams p) {
  const int gw = scan_group_view(p);
  scan_body<DT, QT, CPQ, kModeMain>(p, gw, nullptr, nullptr);
}

template <int DT, int QT, int CPQ>
__global__ void __launch_bounds__(kScanThreads) dresd_scan_sample(ScanParams p) {
  const int gw = scan_group_view(p);
  scan_body<DT, QT, CPQ, kModeSample>(p, gw, nullptr, nullptr);
}

// The same two passes for launches of several query groups of one query
// tile each (the groups' workgroups share the key ranges).
template <int DT, int CPQ>
__global__ void __launch_bounds__(kScanThreads) dresd_scan_main_shared(ScanParams p) {
  const int gw = scan_group_view(p);
  scan_body<DT, 1, CPQ, kModeMain, true>(p, gw, nullptr, nullptr);
}

template <int DT, int CPQ>
__global__ void __launch_bounds__(kScanThreads) dresd_scan_sample_shared(ScanParams p) {
  const int gw = scan_group_view(p);
  scan_body<DT, 1, CPQ, kModeSample, true>(p, gw, nullptr, nullptr);
}

// Segments of one query from its probe list (S <= 1024 ids, in probe
// order): off[j + 1] = tiles of probes 0..j, tile[j] = first tile of probe j.
// Ids outside [0, P) and repeats of an earlier probe get an empty segment, so
// that no partition is scanned twice (its keys would enter the lists twice).
// All threads of the workgroup take part.
__device__ void parts_segments(const int64_t *probes, const int32_t *part_tile, int S, int P,
                               int32_t *off, int32_t *tile) {
  constexpr int E = 4;  // entries per thread: S <= E * kScanThreads
  __shared__ int32_t wsum[kScanThreads / kWaveSize];
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  int32_t id[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int j = t * E + e;
    const int64_t v = j < S ? probes[j] : -1;
    id[e] = (v >= 0 && v < P) ? (int32_t)v : -1;
    if (j < S) tile[j] = id[e];  // the ids, until the segments replace them
  }
  __syncthreads();
  const int last = min(S, t * E + E - 1);  // earlier entries of this thread's last one
  for (int i = 0; i < last; ++i) {
    const int32_t o = tile[i];
#pragma unroll
    for (int e = 0; e < E; ++e)
      if (i < t * E + e && o == id[e]) id[e] = -1;
  }
  int32_t start[E], len[E], sum = 0;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const bool ok = id[e] >= 0;
    start[e] = ok ? part_tile[id[e]] : 0;
    len[e] = ok ? part_tile[id[e] + 1] - start[e] : 0;
    sum += len[e];
  }
  int32_t x = sum;  // inclusive scan over the wave
#pragma unroll
  for (int o = 1; o < kWaveSize; o <<= 1) {
    const int32_t y = __shfl_up(x, o, kWaveSize);
    if (lane >= o) x += y;
  }
  if (lane == kWaveSize - 1) wsum[w] = x;
  __syncthreads();
  int32_t run = x - sum;
  for (int v = 0; v < w; ++v) run += wsum[v];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int j = t * E + e;
    run += len[e];
    if (j < S) {
      off[j + 1] = run;
      tile[j] = start[e];
    }
  }
  if (t == 0) off[0] = 0;
  __syncthreads();
}

// Partitioned search (its own kernel name, so that profiles separate it from
// the exact search): workgroup blockIdx.x serves query blockIdx.x / wgq, and
// its waves own lists [G] of that query; otherwise it is a one-query scan.
template <int DT, int CPQ>
__global__ void __launch_bounds__(kScanThreads) dresd_scan_parts(ScanParams p) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int qb = blockIdx.x / p.wgq;
  const int gw = (blockIdx.x - qb * p.wgq) * (blockDim.x >> 6) +
                 __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  ScanParams q = p;
  q.queries += (size_t)qb * p.d;
  q.lists += (size_t)qb * p.G * p.C;
  q.lcnt += (size_t)qb * p.G;
  q.lkth += (size_t)qb * p.G;
  q.lfirst += (size_t)qb * p.G;
  q.B = 1;
  if (p.next_tok) q.next_tok += qb;
  if (p.probes64) {
    int32_t *off = reinterpret_cast<int32_t *>(smem + p.seg_lds);
    int32_t *tile = off + p.S + 1;
    parts_segments(p.probes64 + (size_t)qb * p.S, p.part_tile, p.S, p.P, off, tile);
    scan_body<DT, 1, CPQ, kModeParts>(q, gw, off, tile);
  } else {
    scan_body<DT, 1, CPQ, kModeParts>(q, gw, p.seg_off + (size_t)qb * (p.S + 1),
                                      p.seg_tile + (size_t)qb * p.S);
  }
}

// ---------------------------------------------------------------- tables ---
// This file is compiled once per scan variant (DRESD_TU = 1..4) and once for
// the layout and dispatch (DRESD_TU = 0) so that the variants build in
// parallel; without DRESD_TU it is one translation unit holding everything.

#define DRESD_SCAN_ROW(DT, CPQ)                                                             \
  {(ScanKernel)dresd_scan_main<DT, 1, CPQ>, (ScanKernel)dresd_scan_main<DT, 2, CPQ>,          \
   (ScanKernel)dresd_scan_main<DT, 4, CPQ>, (ScanKernel)dresd_scan_main<DT, 8, CPQ>,          \
   (ScanKernel)dresd_scan_main<DT, 16, CPQ>},                                                 \
  {                                                                                           \
    (ScanKernel)dresd_scan_sample<DT, 1, CPQ>, (ScanKernel)dresd_scan_sample<DT, 2, CPQ>,     \
        (ScanKernel)dresd_scan_sample<DT, 4, CPQ>, (ScanKernel)dresd_scan_sample<DT, 8, CPQ>, \
        (ScanKernel)dresd_scan_sample<DT, 16, CPQ>                                            \
  }

#define DRESD_VARIANT(V, DT, CPQ)                                                      \
  ScanKernel scan_kernel_variant##V(int qi, bool main_pass, bool shared) {             \
    static const ScanKernel table[2][5] = {DRESD_SCAN_ROW(DT, CPQ)};                   \
    if (shared)                                                                        \
      return qi != 0 ? nullptr                                                         \
             : main_pass ? (ScanKernel)dresd_scan_main_shared<DT, CPQ>                 \
                         : (ScanKernel)dresd_scan_sample_shared<DT, CPQ>;              \
    return table[main_pass ? 0 : 1][qi];                                               \
  }

// variants: 0 = f32 keys, 1 = f16 keys x1, 2 = f16 keys x4, 3 = bf16 keys x4,
// 4 = bf16 keys x2
#if !defined(DRESD_TU) || DRESD_TU == 1
DRESD_VARIANT(0, kF32, 1)
#endif
#if !defined(DRESD_TU) || DRESD_TU == 2
DRESD_VARIANT(1, kF16, 1)
#endif
#if !defined(DRESD_TU) || DRESD_TU == 3
DRESD_VARIANT(2, kF16, 4)
#endif
#if !defined(DRESD_TU) || DRESD_TU == 4
DRESD_VARIANT(3, kBF16, 4)
#endif
#if !defined(DRESD_TU) || DRESD_TU == 5
DRESD_VARIANT(4, kBF16, 2)
#endif

#if !defined(DRESD_TU) || DRESD_TU == 0
ScanKernel scan_kernel_variant0(int, bool, bool);
ScanKernel scan_kernel_variant1(int, bool, bool);
ScanKernel scan_kernel_variant2(int, bool, bool);
ScanKernel scan_kernel_variant3(int, bool, bool);
ScanKernel scan_kernel_variant4(int, bool, bool);

int qt_index(int qt) {
  switch (qt) {
  case 1: return 0;
  case 2: return 1;
  case 4: return 2;
  case 8: return 3;
  case 16: return 4;
  default: return -1;
  }
}

ScanKernel scan_kernel(int dtype, int qt, int cpq, bool main_pass, bool shared) {
  int qi = qt_index(qt);
  if (qi < 0) return nullptr;
  if (dtype == kF32 && cpq == 1) return scan_kernel_variant0(qi, main_pass, shared);
  if (dtype == kF16 && cpq == 1) return scan_kernel_variant1(qi, main_pass, shared);
  if (dtype == kF16 && cpq == 4) return scan_kernel_variant2(qi, main_pass, shared);
  if (dtype == kBF16 && cpq == 4) return scan_kernel_variant3(qi, main_pass, shared);
  if (dtype == kBF16 && cpq == 2) return scan_kernel_variant4(qi, main_pass, shared);
  return nullptr;
}

ScanKernel scan_parts_kernel(int dtype) {
  if (dtype == kF32) return (ScanKernel)dresd_scan_parts<kF32, 1>;
  if (dtype == kF16) return (ScanKernel)dresd_scan_parts<kF16, 4>;
  if (dtype == kBF16) return (ScanKernel)dresd_scan_parts<kBF16, 4>;
  return nullptr;
}

void *layout_kernel_ptr(int dtype) {
  if (dtype == kF32) return (void *)dresd_layout<float>;
  return (void *)dresd_layout<uint16_t>;
}
#endif

}  // namespace dresd
