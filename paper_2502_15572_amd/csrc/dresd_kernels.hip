// gfx950 kernels for exact dense retrieval (DReSD Section 3.5, Eq. 3 with
// unit-norm keys and queries, Section 3.4, Eq. 2: the cosine is the inner
// product; the argmax is taken as the k best keys, Section 3.6).
//
//   layout : one-time copy of row-major keys into 16-row MFMA tiles.
//   scan   : streams the tiles once; MFMA scores (queries as the A operand,
//            key rows as the B operand); a per-query threshold filter; a
//            per-wave bounded candidate list, re-selected in LDS when full;
//            the surviving candidates go to a per-query pool.
//   merge  : per query, radix-selects the k-th best key of its pool, sorts the
//            k winners and gathers their continuations (or, for a sampled
//            pass, emits the k-th best key as the next pass's threshold).
//
// Ranking keys are 64-bit: high half = order-preserving bits of the fp32
// score, low half = ~row.  Larger key = better; equal scores rank the lower
// row first.  Keys are unique, so every selection below is deterministic.
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

__device__ __forceinline__ void wave_sync_lds() {
  // Orders this wave's LDS accesses across lanes (DS ops of one wave run in
  // order; this keeps the compiler from moving them across the point).
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

// Sort n (power of two, >= 2) keys in LDS, descending, by one wave.
__device__ void wave_bitonic_desc(uint64_t *s, int n, int lane) {
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

// Same, by a whole workgroup.
__device__ void block_bitonic_desc(uint64_t *s, int n) {
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
        float r1 = x - (float)hi;                  // exact
        _Float16 mid = (_Float16)(r1 * 2048.0f);   // 2^11
        float r2 = r1 - (float)mid * (1.0f / 2048.0f);  // exact
        _Float16 lo = (_Float16)(r2 * 4194304.0f); // 2^22
        r = (h == 0) ? hi : (h == 1) ? mid : (h == 2) ? lo : (_Float16)0.0f;
      }
      v[e] = __builtin_bit_cast(uint16_t, r);
    } else {
      __bf16 hi = (__bf16)x;
      float r1 = x - (float)hi;
      __bf16 mid = (__bf16)r1;
      __bf16 lo = (__bf16)(r1 - (float)mid);
      __bf16 r = (h == 0) ? hi : (h == 1) ? mid : (h == 2) ? lo : (__bf16)0.0f;
      v[e] = __builtin_bit_cast(uint16_t, r);
    }
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) out[e] = (uint32_t)v[2 * e] | ((uint32_t)v[2 * e + 1] << 16);
  return out;
}

// Re-select a wave's list: keep its k best keys (sorted) and return the k-th.
__device__ uint64_t wave_flush(uint64_t *list, int cnt, int C, int k, uint64_t *scr, int lane) {
  __threadfence_block();  // this wave's list stores are visible to its loads
  for (int e = lane; e < C; e += kWaveSize) scr[e] = (e < cnt) ? list[e] : 0ull;
  wave_sync_lds();
  wave_bitonic_desc(scr, C, lane);
  for (int e = lane; e < k; e += kWaveSize) list[e] = scr[e];
  uint64_t kth = scr[k - 1];
  wave_sync_lds();
  return kth;
}

template <int DT, int QT, int CPQ>
__device__ __forceinline__ void scan_body(const ScanParams &p) {
  constexpr int QPT = 16 / CPQ;        // queries per 16-column tile
  constexpr int NS = 4 / CPQ;          // scores per lane per tile
  constexpr int NQ = QT * QPT;         // queries held by one launch
  constexpr int U = 8;                 // key blocks in flight per wave
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];

  const int lane = threadIdx.x & 63;
  const int wv = threadIdx.x >> 6;
  const int nwv = blockDim.x >> 6;
  const int gw = blockIdx.x * nwv + wv;
  const int G = p.G, C = p.C, KB = p.KB, B = p.B;
  const int ncols = B * CPQ;
  const int g = lane >> 4, m = lane & 15;

  // LDS carve-up: query operand | zero chunk | per-wave state | per-wave scratch
  const int qop_bytes = ncols * KB * 64;
  u4 *qop = reinterpret_cast<u4 *>(smem);
  const int zero_off = qop_bytes;
  unsigned char *st = smem + qop_bytes + 16;
  uint64_t *st_key = reinterpret_cast<uint64_t *>(st) + wv * NQ;
  uint32_t *st_cnt = reinterpret_cast<uint32_t *>(st + (size_t)nwv * NQ * 8) + wv * NQ;
  float *st_thr = reinterpret_cast<float *>(st + (size_t)nwv * NQ * 12) + wv * NQ;
  uint64_t *scr = reinterpret_cast<uint64_t *>(st + (size_t)nwv * NQ * 16) + (size_t)wv * C;

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
  }
  // 2. Per-wave state: thresholds start at the pass's tau (or none).
  for (int q = lane; q < NQ; q += kWaveSize) {
    uint64_t tk = 0;
    float tf = -__builtin_inff();
    if (q >= B) {
      tk = ~0ull;
      tf = __builtin_inff();
    } else if (p.tau && p.tau[q] != 0) {
      tk = p.tau[q] - 1;  // keep keys >= tau
      tf = order_value((uint32_t)(tk >> 32));
    }
    st_key[q] = tk;
    st_cnt[q] = 0;
    st_thr[q] = tf;
  }
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
    for (int s = 0; s < NS; ++s) thr[t][s] = st_thr[t * QPT + g * NS + s];

  // 3. Stream this wave's tiles.
  const int64_t v0 = p.nvisit * gw / G, v1 = p.nvisit * (gw + 1) / G;
  const int64_t J = (v1 - v0) * KB;
  const u4 *base = static_cast<const u4 *>(p.data) + lane;
  int64_t ltile = v0 * p.stride;
  int lkb = 0;
  u4 ring[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    if (u < J) {
      ring[u] = __builtin_nontemporal_load(base + (ltile * KB + lkb) * 64);
      if (++lkb == KB) {
        lkb = 0;
        ltile += p.stride;
      }
    }
  }
  f4 acc[QT];
#pragma unroll
  for (int t = 0; t < QT; ++t) acc[t] = f4{0.f, 0.f, 0.f, 0.f};
  int64_t ctile = v0 * p.stride;
  int ckb = 0;

  for (int64_t j = 0; j < J; j += U) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (j + u < J) {
        u4 cur = ring[u];
        if (j + u + U < J) {
          ring[u] = __builtin_nontemporal_load(base + (ltile * KB + lkb) * 64);
          if (++lkb == KB) {
            lkb = 0;
            ltile += p.stride;
          }
        }
#pragma unroll
        for (int t = 0; t < QT; ++t) {
          u4 a = *reinterpret_cast<const u4 *>(smem + qa0[t] + ckb * qstep[t]);
          acc[t] = Mfma<DT>::run(a, cur, acc[t]);
        }
        if (++ckb == KB) {
          // ---- tile epilogue: threshold filter, rare slow path ----
          const int64_t row64 = ctile * kTileRows + m;
          const bool row_ok = row64 < p.N;
          const uint32_t row = (uint32_t)row64;
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
              }
              sc[t][s] = v;
              any |= row_ok && sc[t][s] >= thr[t][s];
            }
          if (__ballot(any)) {
#pragma unroll
            for (int t = 0; t < QT; ++t)
#pragma unroll
              for (int s = 0; s < NS; ++s) {
                const bool ps = row_ok && sc[t][s] >= thr[t][s];
                uint64_t mk = __ballot(ps);
                while (mk) {
                  const int gg = (__ffsll((long long)mk) - 1) >> 4;
                  const int q = t * QPT + gg * NS + s;
                  const bool mine = ps && (g == gg);
                  const uint64_t key = make_key(sc[t][s], row);
                  uint64_t tk = st_key[q];
                  bool take = mine && key > tk;
                  uint64_t tm = __ballot(take);
                  int n = __popcll(tm);
                  int cnt = (int)st_cnt[q];
                  uint64_t *list = p.lists + ((size_t)q * G + gw) * C;
                  if (cnt + n > C) {
                    tk = wave_flush(list, cnt, C, p.k, scr, lane);
                    cnt = p.k;
                    st_key[q] = tk;
                    st_thr[q] = order_value((uint32_t)(tk >> 32));
                    take = mine && key > tk;
                    tm = __ballot(take);
                    n = __popcll(tm);
                  }
                  if (take) {
                    int pos = cnt + __popcll(tm & ((1ull << lane) - 1ull));
                    list[pos] = key;
                  }
                  st_cnt[q] = (uint32_t)(cnt + n);
                  wave_sync_lds();
                  mk &= ~(0xFFFFull << (16 * gg));
                }
              }
#pragma unroll
            for (int t = 0; t < QT; ++t)
#pragma unroll
              for (int s = 0; s < NS; ++s)
                thr[t][s] = st_thr[t * QPT + g * NS + s];
          }
#pragma unroll
          for (int t = 0; t < QT; ++t) acc[t] = f4{0.f, 0.f, 0.f, 0.f};
          ckb = 0;
          ctile += p.stride;
        }
      }
    }
  }

  // 4. Hand this wave's candidates to the per-query pools.
  __threadfence_block();
  for (int q = lane; q < B; q += kWaveSize) {
    const int cnt = (int)st_cnt[q];
    if (cnt > 0) {
      const uint64_t *list = p.lists + ((size_t)q * G + gw) * C;
      const uint32_t at = atomicAdd(p.pool_cnt + q, (uint32_t)cnt);
      uint64_t *dst = p.pool + (size_t)q * p.pool_cap + at;
      for (int e = 0; e < cnt; ++e) dst[e] = list[e];
    }
  }
}

// Two kernel names so that profiles separate the main pass from the
// sampled passes that only set thresholds.
template <int DT, int QT, int CPQ>
__global__ void __launch_bounds__(kScanThreads) dresd_scan_main(ScanParams p) {
  scan_body<DT, QT, CPQ>(p);
}

template <int DT, int QT, int CPQ>
__global__ void __launch_bounds__(kScanThreads) dresd_scan_sample(ScanParams p) {
  scan_body<DT, QT, CPQ>(p);
}

// ----------------------------------------------------------------- merge ---
#if !defined(DRESD_TU) || DRESD_TU == 0

// One workgroup per query: exact k best keys of the query's pool.
__global__ void __launch_bounds__(kMergeThreads) dresd_merge(MergeParams p) {
  __shared__ uint32_t hist[4096];
  __shared__ uint32_t part[kMergeThreads];
  __shared__ uint64_t cache[kMergeCap];
  __shared__ uint64_t win[DRESD_K_MAX_INTERNAL];
  __shared__ uint64_t sel_prefix, sel_mask;
  __shared__ uint32_t sel_krem, sel_done, win_cnt;

  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const uint32_t M = p.pool_cnt[b];
  const uint64_t *pool = p.pool + (size_t)b * p.pool_cap;
  const bool in_lds = M <= (uint32_t)kMergeCap;
  if (in_lds)
    for (uint32_t i = tid; i < M; i += blockDim.x) cache[i] = pool[i];
  const uint64_t *src = in_lds ? cache : pool;
  const uint32_t kk = M < (uint32_t)p.k ? M : (uint32_t)p.k;
  if (tid == 0) {
    sel_prefix = 0;
    sel_mask = 0;
    sel_krem = kk;
    sel_done = (kk == 0 || kk == M) ? 1u : 0u;  // all candidates are winners
    win_cnt = 0;
  }
  __syncthreads();

  // Radix select of the kk-th largest key, 12 bits at a time from the top.
  const int shifts[6] = {52, 40, 28, 16, 4, 0};
  for (int di = 0; di < 6 && !sel_done; ++di) {
    const int sh = shifts[di];
    const uint32_t wmask = (di == 5) ? 0xFu : 0xFFFu;
    for (int i = tid; i < 4096; i += blockDim.x) hist[i] = 0;
    __syncthreads();
    const uint64_t pre = sel_prefix, pm = sel_mask;
    for (uint32_t i = tid; i < M; i += blockDim.x) {
      uint64_t key = src[i];
      if ((key & pm) == pre) atomicAdd(&hist[(uint32_t)(key >> sh) & wmask], 1u);
    }
    __syncthreads();
    // suffix sums: thread t owns bins [16t, 16t+16)
    uint32_t mine = 0;
    for (int j = 0; j < 16; ++j) mine += hist[tid * 16 + j];
    part[tid] = mine;
    __syncthreads();
    for (int off = 1; off < kMergeThreads; off <<= 1) {
      uint32_t v = (tid + off < kMergeThreads) ? part[tid + off] : 0u;
      __syncthreads();
      part[tid] += v;
      __syncthreads();
    }
    // part[t] = sum of bins >= 16t
    const uint32_t krem = sel_krem;
    const uint32_t above = (tid + 1 < kMergeThreads) ? part[tid + 1] : 0u;
    __syncthreads();
    if (above < krem && krem <= above + mine) {
      uint32_t cum = above;
      for (int j = 15; j >= 0; --j) {
        const uint32_t h = hist[tid * 16 + j];
        if (cum + h >= krem) {
          const uint32_t dg = (uint32_t)(tid * 16 + j);
          sel_prefix = pre | ((uint64_t)dg << sh);
          sel_mask = pm | ((uint64_t)wmask << sh);
          sel_krem = krem - cum;
          if (h == krem - cum) sel_done = 1u;  // the whole bin is in
          break;
        }
        cum += h;
      }
    }
    __syncthreads();
  }
  // Winners: every key >= the selected prefix (exactly kk keys; keys are unique).
  const uint64_t cut = sel_prefix;
  if (kk == M) {
    for (uint32_t i = tid; i < M; i += blockDim.x) win[i] = src[i];
  } else {
    for (uint32_t i = tid; i < M; i += blockDim.x) {
      uint64_t key = src[i];
      if (key >= cut) {
        uint32_t at = atomicAdd(&win_cnt, 1u);
        if (at < (uint32_t)DRESD_K_MAX_INTERNAL) win[at] = key;
      }
    }
  }
  __syncthreads();
  int n = 1;
  while (n < (int)kk) n <<= 1;
  for (int i = (int)kk + tid; i < n; i += blockDim.x) win[i] = 0ull;
  __syncthreads();
  if (n >= 2) block_bitonic_desc(win, n);

  if (!p.final_mode) {
    if (tid == 0) p.tau_out[b] = (M >= (uint32_t)p.k) ? win[p.k - 1] : 0ull;
  } else {
    for (int r = tid; r < p.k; r += blockDim.x) {
      const size_t o = (size_t)b * p.k + r;
      if (r < (int)kk) {
        const uint64_t key = win[r];
        p.idx[o] = (int64_t)(uint32_t)(~(uint32_t)key);
        p.score[o] = order_value((uint32_t)(key >> 32));
      } else {  // cannot happen when N >= k; filled defensively
        p.idx[o] = -1;
        p.score[o] = -__builtin_inff();
      }
    }
    if (p.tokens) {
      const int L = p.L;
      for (int i = tid; i < p.k * L; i += blockDim.x) {
        const int r = i / L, l = i - r * L;
        int32_t v = 0;
        if (r < (int)kk) {
          const uint32_t row = ~(uint32_t)win[r];
          v = p.cont[(size_t)row * L + l];
        }
        p.tokens[((size_t)b * p.k + r) * L + l] = v;
      }
    }
  }
  __syncthreads();
  if (tid == 0) p.pool_cnt[b] = 0;  // ready for the next pass
}
#endif

// ---------------------------------------------------------------- tables ---
// This file is compiled once per scan variant (DRESD_TU = 1..4) and once for
// the merge, layout and dispatch (DRESD_TU = 0) so that the variants build in
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

#define DRESD_VARIANT(V, DT, CPQ)                                       \
  ScanKernel scan_kernel_variant##V(int qi, bool main_pass) {           \
    static const ScanKernel table[2][5] = {DRESD_SCAN_ROW(DT, CPQ)};    \
    return table[main_pass ? 0 : 1][qi];                                \
  }

// variants: 0 = f32 keys, 1 = f16 keys x1, 2 = f16 keys x4, 3 = bf16 keys x4
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

#if !defined(DRESD_TU) || DRESD_TU == 0
ScanKernel scan_kernel_variant0(int, bool);
ScanKernel scan_kernel_variant1(int, bool);
ScanKernel scan_kernel_variant2(int, bool);
ScanKernel scan_kernel_variant3(int, bool);

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

ScanKernel scan_kernel(int dtype, int qt, int cpq, bool main_pass) {
  int qi = qt_index(qt);
  if (qi < 0) return nullptr;
  if (dtype == kF32 && cpq == 1) return scan_kernel_variant0(qi, main_pass);
  if (dtype == kF16 && cpq == 1) return scan_kernel_variant1(qi, main_pass);
  if (dtype == kF16 && cpq == 4) return scan_kernel_variant2(qi, main_pass);
  if (dtype == kBF16 && cpq == 4) return scan_kernel_variant3(qi, main_pass);
  return nullptr;
}

void *merge_kernel_ptr() { return (void *)dresd_merge; }

void *layout_kernel_ptr(int dtype) {
  if (dtype == kF32) return (void *)dresd_layout<float>;
  return (void *)dresd_layout<uint16_t>;
}
#endif

}  // namespace dresd
