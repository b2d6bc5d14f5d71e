// Internal declarations shared by the host runtime and the gfx950 kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dresd {

// Keys are stored in tiles of 16 rows.  A tile is a run of 1 KiB blocks, one
// per group of dimensions (32 dims for 16-bit keys, 16 dims for fp32 keys).
// Inside a block, 16-byte chunk c (c = 0..63) holds row (c % 16) of the tile
// and dims [w*(c/16), w*(c/16) + w) of the block, w = 8 (16-bit) or 4 (fp32):
// exactly the per-lane operand of one 16x16 MFMA, so wave lane c loads chunk c
// and every wave load is one contiguous 1 KiB.
constexpr int kTileRows = 16;
constexpr int kBlockBytes = 1024;
constexpr int kWaveSize = 64;
constexpr int kScanThreads = 256;   // 4 waves per workgroup
constexpr int kMergeThreads = 1024;
constexpr int kMergeCap = 4096;     // candidates a merge keeps in LDS
constexpr int kMergeLists = 4096;   // most candidate lists per query a merge accepts
#define DRESD_K_MAX_INTERNAL 1024   // equals DRESD_K_MAX of the public header

enum DType { kF32 = 0, kF16 = 1, kBF16 = 2 };

struct ScanParams {
  const void *data;          // tiled keys
  const float *queries;      // [B, d] fp32
  int64_t N;                 // rows
  int64_t nvisit;            // tiles this pass visits: tile = j * stride
  int64_t stride;            // tile stride of the pass (1 = every tile)
  const uint64_t *tau;       // [B] keys below tau are pruned (0 = none); may be null
  uint64_t *lists;           // [B][G][C] per-wave candidate lists
  uint32_t *lcnt;            // [B][G] list lengths; bit 31 set = sorted descending
  uint64_t *lkth;            // [B][G] k-th best key of a sorted list of k keys, else 0
  uint64_t *lfirst;          // [B][G] best key of a sorted list; ~0 unknown; 0 empty
  int B, d, KB, k, C, G;     // batch, dims, blocks per tile, k, list capacity, lists
  int CL;                    // per-query LDS stage in front of each HBM list
  int sort_lists;            // sort every list at the end (small batches)
  const void *qop;           // shared-key scan: query operands [tiles][KB][64] x 16 B
  // Next-token-filtered search (both null otherwise): only rows whose value
  // starts with the query's next token compete.
  const int32_t *ftok;       // [tiles * 16] first token of each slot's value
  const int32_t *next_tok;   // [B] next token of each query
  // Partitioned search (dresd_scan_parts): slot table and each query's
  // probed segments; wgq workgroups per query, G lists per query.
  const uint32_t *slot_row;  // [tiles * 16] row of each slot, kPadRow for padding
  const int32_t *seg_off;    // [B][S + 1] cumulative tiles of the probed partitions
  const int32_t *seg_tile;   // [B][S] first tile of each probed partition
  int S, wgq;
  // ... or, when probes64 is set, each workgroup builds its query's segments
  // in LDS at byte offset seg_lds from the exact probe search's output
  // ([B][S] ids; outside [0, P) and repeats skipped) and the partitions'
  // first tiles.
  const int64_t *probes64;
  const int32_t *part_tile;  // [P + 1]
  int seg_lds, P;
  // Single-tile scan: query groups served by one launch.  Group i holds
  // queries [B i / ngroups, B (i + 1) / ngroups) of the launch's B; each
  // group has its own G lists per query and gridDim.x / ngroups workgroups.
  int ngroups = 1;
};

// Slot of the partitioned layout that holds no row.
constexpr uint32_t kPadRow = 0xFFFFFFFFu;

// Query operands of the shared-key scan, built once per search: chunk
// (t, kb, lane) is the MFMA A operand of lane `lane` for query tile t and
// 32-dim block kb (columns past the batch are zero).
struct QopParams {
  const float *queries;      // [B, d] fp32
  void *out;                 // [ntile][KB][64] x 16 B
  int B, d, KB, ntile;
};

// LDS bytes of one wave's candidate state in the single-tile scan: staged
// keys [nq][cl], sort scratch [C], exact thresholds [nq] and three counters
// per query, rounded up to 16 bytes.
__host__ __device__ inline size_t scan_wave_bytes(int nq, int cl, int C) {
  return ((size_t)nq * cl * 8 + (size_t)C * 8 + (size_t)nq * 8 + (size_t)nq * 12 + 15) / 16 * 16;
}

// Single-tile scan: next tokens of the launch's queries, shared by the waves,
// and per wave two slots of first tokens (four tiles' rows each).
__host__ __device__ inline size_t scan_ntok_bytes(int nq) { return ((size_t)nq * 4 + 15) / 16 * 16; }
constexpr int kScanFtokBytes = 2 * 64 * 4;

// Shared-key scan, filtered search: per wave, the next token of each score
// slot [4 lane groups][np] and a ring of first-token copies [stages][64].
__host__ __device__ inline size_t scan_mq_filter_bytes(int stages, int np) {
  return (size_t)16 * np + (size_t)stages * 256;
}

// Shared-key scan: a wave's candidate buffer holds kMqCandBuf (key, query)
// entries; its LDS region is key buffer [kMqCandBuf] u64 | sort scratch [C]
// u64 | exact thresholds [nqw] u64 | query of each buffered key [kMqCandBuf]
// u8 | list lengths [nqw] u32 | float thresholds [nqw] f32 | best listed
// key [nqw] u64.
constexpr int kMqCandBuf = 256;
constexpr int kMqStageBlocks = 8;  // 1 KiB key blocks per LDS stage
__host__ __device__ inline size_t scan_mq_wave_bytes(int nqw, int C, int cb = kMqCandBuf) {
  return ((size_t)cb * 9 + (size_t)C * 8 + (size_t)nqw * 24 + 15) / 16 * 16;
}
// The tiled contraction tests a tile once per K loop: a smaller buffer.
constexpr int kTcCandBuf = 128;
// LDS of the shared-key scan: ring | one candidate region per wave (nw
// waves per workgroup).
__host__ __device__ inline size_t scan_mq_lds_bytes(int stages, int nqw, int C, int nw = 4) {
  return (size_t)stages * kMqStageBlocks * kBlockBytes + (size_t)nw * scan_mq_wave_bytes(nqw, C);
}

// A list summary flag: the list is sorted, best key first.
constexpr uint32_t kSortedFlag = 0x80000000u;


struct LayoutParams {
  const void *src;           // [N, d] row-major
  void *dst;                 // tiles
  const uint32_t *slot_row;  // partitioned layout: row of each slot (null: slot = row)
  int64_t N;
  int64_t chunks;            // total 16-byte chunks of the tiled layout
  int d, KB;
};


// Kernel launch entry points (defined in dresd_kernels.hip).
typedef void (*ScanKernel)(ScanParams);
// cpq: columns per query; shared: the variant for launches of several query
// groups (one query tile only, else null)
ScanKernel scan_kernel(int dtype, int qt, int cpq, bool main_pass, bool shared = false);
// Shared-key scan (dresd_scan_mq.hip): qtw query tiles per wave, kbt blocks
// per key tile, filtered = next-token-filtered search, nwq waves per
// workgroup (4, or 1 for a wave holding the whole batch: qtw 4 with 8-block
// tiles); *stages receives the depth of its LDS ring of key stages.
ScanKernel scan_mq_kernel_f16(int qtw, int kbt, bool main_pass, bool filtered, int *stages,
                              int nwq);
ScanKernel scan_mq_kernel_bf16(int qtw, int kbt, bool main_pass, bool filtered, int *stages,
                               int nwq);
inline ScanKernel scan_mq_kernel(int dtype, int qtw, int kbt, bool main_pass, bool filtered,
                                 int *stages, int nwq = 4) {
  if (dtype == kF16) return scan_mq_kernel_f16(qtw, kbt, main_pass, filtered, stages, nwq);
  if (dtype == kBF16) return scan_mq_kernel_bf16(qtw, kbt, main_pass, filtered, stages, nwq);
  return nullptr;
}
// Tiled contraction (both operands through LDS): qtw query tiles per wave
// (4, or 8 for bf16), tpw key tiles per wave, nk key groups x nq query groups
// of waves per workgroup, ring stages.  One query group: main passes
// (tpw, nk, stages) = (4, 8, 3), (4, 4, 5) and (4, 4, 3), sampled passes
// (1, 4, 8) and (1, 4, 4).  Two query groups: main (4, 4, 3), sampled
// (2, 4, 4).  Four (f16): main (8, 2, 3), sampled (4, 2, 4).  Each also next-
// token filtered; null for other shapes.
ScanKernel scan_tc_kernel_f16(int qtw, int tpw, int nk, int nq, int stages, bool main_pass,
                              bool filtered);
ScanKernel scan_tc_kernel_bf16(int qtw, int tpw, int nk, int nq, int stages, bool main_pass,
                               bool filtered);
inline ScanKernel scan_tc_kernel(int dtype, int qtw, int tpw, int nk, int nq, int stages,
                                 bool main_pass, bool filtered) {
  if (dtype == kF16) return scan_tc_kernel_f16(qtw, tpw, nk, nq, stages, main_pass, filtered);
  if (dtype == kBF16) return scan_tc_kernel_bf16(qtw, tpw, nk, nq, stages, main_pass, filtered);
  return nullptr;
}
// LDS of the tiled contraction: ring | per wave a candidate region |
// (filtered search) per wave the next tokens of its score slots and the
// first tokens of its panel tiles' rows.  nqw queries and np score slots
// per lane per wave.
__host__ __device__ inline size_t scan_tc_lds_bytes(int qtw, int tpw, int nk, int nq, int stages,
                                                    int nqw, int C, int np, bool filtered) {
  const int nw = nk * nq;
  const int ftw = 16 * tpw > kWaveSize ? 16 * tpw : kWaveSize;
  return (size_t)stages * (nk * tpw + nq * qtw) * kBlockBytes +
         (size_t)nw * scan_mq_wave_bytes(nqw, C, kTcCandBuf) +
         (filtered ? (size_t)nw * (16 * np + 4 * ftw) : 0);
}
// Query-operand kernel of the shared-key scan and the tiled contraction for
// a key type (launch with 256 threads, one thread per 16-byte chunk).
void *qop_kernel_f16();
void *qop_kernel_bf16();
inline void *qop_kernel(int dtype) {
  return dtype == kF16 ? qop_kernel_f16() : dtype == kBF16 ? qop_kernel_bf16() : nullptr;
}
ScanKernel scan_parts_kernel(int dtype);  // partitioned search, one query per workgroup

void *merge_kernel_ptr();
// Bandwidth probe (dresd_bwprobe.hip): one read pass over nblocks 1 KiB
// blocks with `workgroups` workgroups of 4 waves.
hipError_t launch_bw_read(const void *buf, int64_t nblocks, int workgroups, hipStream_t st);
void *layout_kernel_ptr(int dtype);
int qt_index(int qt);  // 1,2,4,8,16 -> 0..4, else -1

}  // namespace dresd
