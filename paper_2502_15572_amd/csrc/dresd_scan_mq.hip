// gfx950 scan for batches spanning several 16-column query tiles (the same
// computation as the scan in dresd_kernels.hip: DReSD Section 3.5, Eq. 3
// with unit-norm keys as exact top-k, Section 3.6).
//
// The queries stay in registers and the keys are shared through LDS:
//   * the workgroup's 4 waves split the query tiles; each wave holds its
//     tiles' A operands for every 32-dim block of the keys in VGPRs;
//   * the workgroup streams its key tiles in stages of SB 1 KiB blocks; each
//     wave loads LPS blocks of a stage into registers D stages ahead, writes
//     them to a double-buffered LDS stage, and after one barrier every wave
//     reads every block of the stage once (4 KiB of LDS reads per KiB of HBM,
//     independent of the batch);
//   * every stage issues exactly LPS loads per wave (loads past the end
//     re-read the last block), so the wait before each stage is a constant.
// Candidates are filtered and listed exactly as in the single-tile scan,
// with one list per (query, workgroup).
#include "dresd_scan_common.h"

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
// query once to the key type; CPQ = 4 gives three parts summing to it exactly
// (f16 lower parts scaled by 2^11, 2^22) and a zero column.
template <int DT, int CPQ>
__device__ __forceinline__ u4 query_chunk_mq(const float *q, int d, int B, int col, int dim0) {
  const int b = col / CPQ;
  const int h = col % CPQ;
  uint16_t v[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int dim = dim0 + e;
    const float x = (b < B && dim < d) ? q[(int64_t)b * d + dim] : 0.0f;
    if (DT == kF16) {
      _Float16 hi = (_Float16)x;
      _Float16 r = hi;
      if (CPQ == 4) {
        float r1 = x - (float)hi;
        _Float16 mid = (_Float16)(r1 * 2048.0f);
        float r2 = r1 - (float)mid * (1.0f / 2048.0f);
        _Float16 lo = (_Float16)(r2 * 4194304.0f);
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
  u4 out;
#pragma unroll
  for (int e = 0; e < 4; ++e) out[e] = (uint32_t)v[2 * e] | ((uint32_t)v[2 * e + 1] << 16);
  return out;
}

}  // namespace

// QTW query tiles per wave, KBT 32-dim blocks per key tile (must equal the
// index's blocks per tile), CPQ operand columns per query.
template <int DT, int QTW, int KBT, int CPQ, bool MAIN>
__device__ __forceinline__ void scan_mq_body(const ScanParams &p) {
  constexpr int NW = kScanThreads / kWaveSize;  // waves per workgroup
  constexpr int QPT = 16 / CPQ;
  constexpr int NS = 4 / CPQ;
  constexpr int NQW = QTW * QPT;  // queries per wave
  constexpr int SB = 8;           // blocks per stage
  constexpr int LPS = SB / NW;    // loads per wave per stage
  constexpr int D = 4;            // stages loaded ahead (= stages per group)
  constexpr int GB = SB * D;      // blocks per group; a whole number of tiles
  static_assert(GB % KBT == 0, "a group must hold whole key tiles");
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];

  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g = lane >> 4, m = lane & 15;
  const int B = p.B, C = p.C;
  const int G = p.G;  // lists per query = workgroups
  const int wg = blockIdx.x;

  // LDS: two stages of keys, then one region per wave:
  //   staged keys [NQW][CL] | sort scratch [C] | thresholds [NQW] |
  //   scores of a tile with candidates [QTW*NS][64] | counts [NQW] x 3
  u4 *stage_buf = reinterpret_cast<u4 *>(smem);
  const int CL = p.CL;
  const size_t wreg = scan_mq_wave_bytes(NQW, QTW * NS, CL, C);
  unsigned char *w0 = smem + 2 * SB * kBlockBytes + (size_t)wv * wreg;
  CandSink sink;
  sink.stg = reinterpret_cast<uint64_t *>(w0);
  sink.scr = sink.stg + (size_t)NQW * CL;
  sink.st_key = sink.scr + C;
  float *scs = reinterpret_cast<float *>(sink.st_key + NQW);
  sink.st_cnt = reinterpret_cast<uint32_t *>(scs + (size_t)QTW * NS * kWaveSize);
  sink.st_thr = reinterpret_cast<float *>(sink.st_cnt + NQW);
  sink.stg_cnt = reinterpret_cast<uint32_t *>(sink.st_thr + NQW);
  sink.cl = CL;
  sink.C = C;
  sink.k = p.k;
  sink.lane = lane;

  // Queries of this wave: tiles [wv*QTW, wv*QTW + QTW) of the batch.
  const int q0 = wv * NQW;
  u4 qreg[QTW][KBT];
#pragma unroll
  for (int t = 0; t < QTW; ++t)
#pragma unroll
    for (int kb = 0; kb < KBT; ++kb)
      qreg[t][kb] = query_chunk_mq<DT, CPQ>(p.queries, p.d, B, (wv * QTW + t) * 16 + m,
                                            kb * 32 + g * 8);
  sink_init(sink, NQW, B - q0, p.tau ? p.tau + q0 : nullptr);
  auto list_of = [&](int i) { return p.lists + ((size_t)(q0 + i) * G + wg) * C; };

  // This workgroup's key blocks: tiles [v0, v1), KBT blocks each.
  const int64_t v0 = wave_uniform(p.nvisit * wg / G);
  const int64_t v1 = wave_uniform(p.nvisit * (wg + 1) / G);
  const int64_t NB = (v1 - v0) * KBT;
  const u4 *base = static_cast<const u4 *>(p.data) + lane;
  // Address of the workgroup's block j, clamped to its last block.
  auto block = [&](int64_t j) -> const u4 * {
    j = j < NB ? j : NB - 1;
    const int64_t vt = j / KBT;
    return base + ((v0 + vt) * p.stride * KBT + (j - vt * KBT)) * 64;
  };

  u4 ring[D][LPS];
  if (NB > 0) {
#pragma unroll
    for (int r = 0; r < D; ++r)
#pragma unroll
      for (int i = 0; i < LPS; ++i) ring[r][i] = __builtin_nontemporal_load(block(r * SB + wv * LPS + i));
  }

  f4 acc[QTW];
  auto tile_end = [&](int64_t tile) {
    const int64_t row64 = tile * kTileRows + m;
    const bool row_ok = row64 < p.N;
    const uint32_t row = (uint32_t)row64;
    float sc[QTW][NS];
    bool any = false;
#pragma unroll
    for (int t = 0; t < QTW; ++t)
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        float v = acc[t][s * CPQ];
        if (CPQ == 4) {
          const float s1 = (DT == kF16) ? (1.0f / 2048.0f) : 1.0f;
          const float s2 = (DT == kF16) ? (1.0f / 4194304.0f) : 1.0f;
          v = (v + acc[t][s * CPQ + 1] * s1) + acc[t][s * CPQ + 2] * s2;
        }
        sc[t][s] = v;
        any |= row_ok && v >= sink.st_thr[t * QPT + g * NS + s];
      }
    if (__ballot(any)) {
      // Rare: park the scores in LDS and walk them in a rolled loop (keeps
      // the unrolled stream loop small).
      bool spilled = false;
#pragma unroll
      for (int t = 0; t < QTW; ++t)
#pragma unroll
        for (int s = 0; s < NS; ++s) scs[(t * NS + s) * kWaveSize + lane] = sc[t][s];
      wave_sync_lds();
#pragma unroll 1
      for (int ts = 0; ts < QTW * NS; ++ts) {
        const int t = ts / NS, s = ts - t * NS;
        const float v = scs[ts * kWaveSize + lane];
        const bool ps = row_ok && v >= sink.st_thr[t * QPT + g * NS + s];
        uint64_t mk = __ballot(ps);
        while (mk) {
          const int gg = (__ffsll((long long)mk) - 1) >> 4;
          const int i = t * QPT + gg * NS + s;  // query q0 + i
          spilled |= sink_offer(sink, i, ps && (g == gg), make_key(v, row), list_of(i));
          mk &= ~(0xFFFFull << (16 * gg));
        }
      }
      // A spill used vector memory: drain it here so that afterwards only the
      // ring's loads are in flight and the stream keeps exact wait counts.
      if (spilled) __threadfence_block();
    }
  };

  // Groups of D stages, so that ring slots and the block -> (tile, block of
  // tile) map are static.  Every stage: stage data to LDS, reload its ring
  // slot D stages ahead, one barrier, then all waves consume the stage.
  for (int64_t j0 = 0; j0 < NB; j0 += GB) {
    const int64_t jb = wave_uniform(j0);
#pragma unroll
    for (int r = 0; r < D; ++r) {
      u4 *buf = stage_buf + (size_t)(r & 1) * SB * 64;
#pragma unroll
      for (int i = 0; i < LPS; ++i) buf[(wv * LPS + i) * 64 + lane] = ring[r][i];
#pragma unroll
      for (int i = 0; i < LPS; ++i)
        ring[r][i] = __builtin_nontemporal_load(block(jb + GB + r * SB + wv * LPS + i));
      __syncthreads();
#pragma unroll
      for (int i = 0; i < SB; ++i) {
        const int j = r * SB + i;  // block of the group (static)
        const int kb = j % KBT;
        if (jb + j < NB) {
          if (kb == 0) {
#pragma unroll
            for (int t = 0; t < QTW; ++t) acc[t] = f4{0.f, 0.f, 0.f, 0.f};
          }
          const u4 blk = buf[i * 64 + lane];
#pragma unroll
          for (int t = 0; t < QTW; ++t) acc[t] = MfmaMQ<DT>::run(qreg[t][kb], blk, acc[t]);
          if (kb == KBT - 1) tile_end((v0 + (jb + j) / KBT) * p.stride);
        }
      }
    }
  }

  // Publish this wave's lists (one per query per workgroup).
  for (int i = 0; i < NQW && q0 + i < B; ++i) {
    const size_t o = (size_t)(q0 + i) * G + wg;
    sink_publish(sink, i, list_of(i), p.sort_lists != 0, p.lcnt + o, p.lfirst + o, p.lkth + o);
  }
}

template <int DT, int QTW, int KBT, int CPQ>
__global__ void __launch_bounds__(kScanThreads, 2) dresd_scanmq_main(ScanParams p) {
  scan_mq_body<DT, QTW, KBT, CPQ, true>(p);
}

template <int DT, int QTW, int KBT, int CPQ>
__global__ void __launch_bounds__(kScanThreads, 2) dresd_scanmq_sample(ScanParams p) {
  scan_mq_body<DT, QTW, KBT, CPQ, false>(p);
}

// (QTW, KBT) pairs with QTW * KBT <= 32 (query operands <= 128 VGPRs).
#define DRESD_MQ_CASE(DT, CPQ, QTW, KBT)                                          \
  if (qtw == QTW && kbt == KBT)                                                   \
    return main_pass ? (ScanKernel)dresd_scanmq_main<DT, QTW, KBT, CPQ>           \
                     : (ScanKernel)dresd_scanmq_sample<DT, QTW, KBT, CPQ>;
#define DRESD_MQ_ALL(DT, CPQ)                                                     \
  DRESD_MQ_CASE(DT, CPQ, 1, 4) DRESD_MQ_CASE(DT, CPQ, 1, 8)                       \
  DRESD_MQ_CASE(DT, CPQ, 1, 16) DRESD_MQ_CASE(DT, CPQ, 1, 32)                     \
  DRESD_MQ_CASE(DT, CPQ, 2, 4) DRESD_MQ_CASE(DT, CPQ, 2, 8)                       \
  DRESD_MQ_CASE(DT, CPQ, 2, 16) DRESD_MQ_CASE(DT, CPQ, 4, 4)                      \
  DRESD_MQ_CASE(DT, CPQ, 4, 8)

#if !defined(DRESD_MQ_TU) || DRESD_MQ_TU == 0
ScanKernel scan_mq_kernel_f16(int qtw, int kbt, bool main_pass) {
  DRESD_MQ_ALL(kF16, 1)
  return nullptr;
}
#endif
#if !defined(DRESD_MQ_TU) || DRESD_MQ_TU == 1
ScanKernel scan_mq_kernel_bf16(int qtw, int kbt, bool main_pass) {
  DRESD_MQ_ALL(kBF16, 4)
  return nullptr;
}
#endif

}  // namespace dresd
