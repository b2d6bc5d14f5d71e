// Declarations of the kernels around the scans (dresd_merge.hip,
// dresd_transform.hip, dresd_drafts.hip, dresd_parts.hip, dresd_kmeans.hip),
// shared with the host runtime.  The scan kernels do not include this file.
#pragma once
#include "dresd_internal.h"

namespace dresd {

struct MergeParams {
  const uint64_t *lists;     // [B][G][C] from the scan
  const uint32_t *lcnt;      // [B][G]
  const uint64_t *lkth;      // [B][G]
  const uint64_t *lfirst;    // [B][G]
  uint64_t *spill;           // [B][spill_cap] candidates past the LDS cache
  int64_t spill_cap;
  int B, k, C, G;
  uint64_t *tau_out;         // sample mode: k-th best key per query, else tau_fb (0 if none)
  const uint64_t *tau_fb;    // sample mode: the bound the pass's sample falls back to (may be null)
  uint64_t *spec_out;        // sample mode: spec_rank-th best key per query (may be null)
  int spec_rank;             // 1 <= spec_rank <= k when spec_out is set
  int64_t *idx;              // final mode outputs
  float *score;
  int32_t *tokens;           // may be null
  const int32_t *cont;       // [N, L]
  int64_t N;                 // rows of cont: a winner outside [0, N) is written as (-1, -inf, 0)
  int L;
  int final_mode;
};

// Query-side transform (dresd_transform.hip): y = unit rows of
// ((x - mean) / sqrt(var + eps_z)) W.
struct TransformParams {
  const float *x;            // [M, D]
  const float *mean, *var;   // [D]
  const float *W;            // [D, l] row-major
  float *y;                  // [M, l]
  float *part;               // [splits][M][l] partial sums (splits > 1)
  int64_t M;
  int D, l;
  int splits, dslice;        // D split into `splits` slices of `dslice` dims
  float eps_z, eps_n;
};
// Splits of D for an M x l output on a device with `cus` compute units.
int transform_splits(int64_t M, int D, int l, int cus);
hipError_t launch_transform(const TransformParams &p, hipStream_t st);

// Draft assembly (dresd_drafts.hip): tokens [B, k, L] -> drafts [B, r, length],
// count [B].
struct DraftParams {
  const int32_t *tokens;
  int32_t *drafts, *count;
  int B, k, L, r, length, eos;
};
hipError_t launch_pack_drafts(const DraftParams &p, hipStream_t st);

// Probed segments of a partitioned search (dresd_parts.hip): one workgroup
// per query turns its probe list into seg_off / seg_tile.
struct SegParams {
  const int64_t *probes64;   // [B][S] partition ids (one of the three is set)
  const int32_t *probes32;
  const int32_t *tok;        // [P] ascending first tokens, partition p holding tok[p]; with
  const int32_t *next_tok;   //   next_tok [B] each query probes its token's partition (S = 1)
  const int32_t *part_tile;  // [P + 1] first tile of each partition
  int32_t *seg_off, *seg_tile;
  int B, S, P;
};
hipError_t launch_segments(const SegParams &p, hipStream_t st);
// out[i] = cont[i][0], the first token of row i's value.
hipError_t launch_first_tokens(const int32_t *cont, int L, int64_t n, int32_t *out,
                               hipStream_t st);
// ftok[s] = first token of slot s's value (0 for padding slots).
hipError_t launch_slot_first_tokens(const uint32_t *slot_row, const int32_t *cont, int L,
                                    int64_t nslot, int32_t *ftok, hipStream_t st);
// Spherical k-means (dresd_kmeans.hip).
struct KmeansParams {
  const void *x;             // [n, d] rows, storage type dtype
  int64_t n;
  int d, dtype, P;
  const float *centroids;    // [P, d] (assign)
  int32_t *assign;           // [n] out (assign)
  float *score;              // [n] out, may be null (assign)
  const int32_t *assign_in;  // [n] (update)
  float *centroids_out;      // [P, d] in/out (update)
  int32_t *counts;           // [P] out, may be null (update)
  long long *sums;           // [P, d] fixed-point workspace (update)
  int32_t *cnt;              // [P] workspace (update)
  int64_t offset;            // first picked row, in [0, n) (init)
};
hipError_t launch_kmeans_assign(const KmeansParams &p, hipStream_t st);
hipError_t launch_kmeans_update(const KmeansParams &p, int cus, hipStream_t st);
hipError_t launch_kmeans_init(const KmeansParams &p, hipStream_t st);

}  // namespace dresd
