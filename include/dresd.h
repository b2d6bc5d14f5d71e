/*
 * dresd.h -- C ABI of the MI355X (gfx950) dense-retrieval library.
 *
 * The library implements the drafting step of DReSD (Dense Retrieval for
 * Speculative Decoding): the datastore is a key -> value map whose keys are
 * L2-normalised token embeddings and whose values are the next L tokens that
 * followed each key (Section 3.5).  A query embedding, itself L2-normalised
 * (Section 3.4, Eq. 2), retrieves the value of the most similar key under
 * cosine similarity (Section 3.5, Eq. 3).  Keys and queries have unit norm, so
 * the cosine is the inner product and the library computes the raw inner
 * product without dividing by the norms.  Batch verification consumes several
 * drafts per decode step (Section 3.6), so the argmax of Eq. 3 is returned as
 * the k best keys.  The search is exact (every key is scored), not the
 * approximate search the paper used.
 *
 * Conventions shared by every call:
 *  - Pointers marked "device" are HIP device pointers on the current device.
 *    Pointers marked "host" are ordinary host memory.
 *  - dresd_stream is a hipStream_t (NULL = the null stream).  Work is enqueued
 *    on it and the call returns; results are valid once the stream has
 *    completed, except where a call says it synchronises.
 *  - Every argument is validated before any work is enqueued: on an error
 *    return nothing has been written to any output.
 *  - No C++ exception crosses this interface.  A failing call returns a status
 *    code and sets a thread-local message readable with dresd_last_error().
 *  - Inputs must be finite.  Keys and queries are expected to be
 *    L2-normalised; the library does not renormalise.
 */
#ifndef DRESD_H
#define DRESD_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Streams and graphs.  Every search, transform and draft call only enqueues
 * kernels on the given stream once a first call of the same shapes has sized
 * the workspaces it uses (that first call may allocate and synchronise).
 * After such a warm-up call these calls can be captured in a HIP graph:
 * they issue no allocation, no synchronisation and no memset while running.
 * A call that would have to grow a workspace while its stream is being
 * captured fails with DRESD_EUNSUPPORTED instead.  A workspace that a later,
 * larger call outgrows is never freed before its owner is (the index for
 * search workspaces, the process for the transform and k-means buffers, one
 * per device and stream), so a graph captured earlier stays valid after such
 * a call.
 *
 * Allocation-failure test hook: with DRESD_FAIL_ALLOC_AT=n in the
 * environment, the n-th device allocation the library makes (counted from
 * when the variable last took a new value) fails as out of memory.
 */
typedef struct dresd_index dresd_index; /* opaque, library-owned */
typedef struct dresd_ivf dresd_ivf;     /* opaque: partitioned index */
typedef void *dresd_stream;             /* a hipStream_t */

/* Storage type of the keys.  Queries are always fp32; scores are fp32. */
typedef enum { DRESD_F32 = 0, DRESD_F16 = 1, DRESD_BF16 = 2 } dresd_dtype;

typedef enum {
  DRESD_OK = 0,
  DRESD_EINVAL = 1,      /* an argument is out of its documented range     */
  DRESD_ENOMEM = 2,      /* a device allocation failed (nothing leaked)    */
  DRESD_EDEVICE = 3,     /* a HIP call failed; message in dresd_last_error */
  DRESD_EUNSUPPORTED = 4 /* valid request the library cannot serve        */
} dresd_status;

/* Largest k a search may ask for. */
#define DRESD_K_MAX 1024
/* Largest datastore: row indices are carried in 32 bits inside the kernels. */
#define DRESD_N_MAX 4294967040LL
/* Most partitions of a partitioned index. */
#define DRESD_PARTS_MAX (1 << 24)

/*
 * Build an index over N keys (Section 3.5: keys are token embeddings, values
 * the next L tokens; building the datastore is a one-time cost, Section 5.6).
 *
 *   embeddings    device, [N, d] row-major, element type `dtype`
 *                 (f32, IEEE binary16, or bfloat16), each row L2-normalised.
 *   continuations device, [N, L] row-major int32 token ids (opaque; copied
 *                 bit for bit, including any padding id).
 *   N, d, L       1 <= N <= DRESD_N_MAX, 1 <= d <= 16384, 1 <= L <= 4096.
 *   dtype         a dresd_dtype value.
 *   stream        stream used for the copies.
 *   out           host; receives the new index.
 *
 * Ownership: both arrays are copied into library-owned device memory (keys
 * re-laid out for the scan).  The call synchronises `stream` before it
 * returns, so the caller may free or reuse its arrays immediately.  The index
 * lives on the device that was current during this call.
 * Errors: EINVAL (null pointer, size out of range, unknown dtype), ENOMEM,
 * EDEVICE.  On error *out is left unchanged and nothing is allocated.
 */
dresd_status dresd_index_create(const void *embeddings,
                                const int32_t *continuations, int64_t N,
                                int32_t d, int32_t L, int32_t dtype,
                                dresd_stream stream, dresd_index **out);

/*
 * Exact top-k retrieval for a batch of B queries (Eq. 3 taken as the k best
 * keys; the drafts of Section 3.6 are their continuations).
 *
 *   ix        index from dresd_index_create.
 *   queries   device, [B, d] fp32 row-major, each row L2-normalised.
 *   B         B >= 0; B == 0 is a no-op returning DRESD_OK.
 *   k         1 <= k <= min(N, DRESD_K_MAX).
 *   idx       device, [B, k] int64: row indices of the k best keys.
 *   score     device, [B, k] fp32: their inner products with the query.
 *   tokens    device, [B, k, L] int32: continuations of those rows, gathered
 *             bit for bit; may be NULL to skip the gather.
 *   stream    stream the search runs on.
 *
 * Order: rank r holds the r-th largest score; equal scores are ordered by
 * ascending row index.  Scores are accumulated in fp32.  For 16-bit keys and
 * B <= 4 the query enters the matrix cores as three 16-bit parts that sum to
 * it exactly (scores within fp32 summation error of the exact inner
 * product); larger bf16 batches take two parts (their sum within 2^-17
 * relative of the query: score error below 8e-6) and larger f16 batches the
 * query rounded once to f16 (score error below 5e-4); both are inside the
 * 2e-3 parity bound for 16-bit keys.
 * Determinism: identical inputs give bitwise identical outputs.
 * Ownership: outputs are caller-owned and must stay alive until `stream`
 * completes.  The index owns a workspace per stream it is searched on, which
 * grows on first use with a new batch shape (that growth allocates and
 * synchronises; outgrown workspaces are kept until the index is destroyed):
 * searches on different streams may overlap on the device, searches on one
 * stream are ordered by it.  The calls themselves are not thread-safe: calls
 * on one index from several host threads must be serialised by the caller.
 * Errors: EINVAL (null index/queries/idx/score, k out of range, B < 0),
 * ENOMEM (workspace growth failed; no output written), EUNSUPPORTED (the
 * workspace would have to grow during stream capture), EDEVICE.
 */
dresd_status dresd_search(dresd_index *ix, const float *queries, int32_t B,
                          int32_t k, int64_t *idx, float *score,
                          int32_t *tokens, dresd_stream stream);

/*
 * Next-token-filtered retrieval (Section 3.5, with Section 3.1): the token
 * x_{t+1} that the LLM produced with the query embedding removes every draft
 * that does not start with it.  Read as filter-then-select: for query b only
 * rows whose continuation starts with next_tok[b] (continuations[i][0] ==
 * next_tok[b]) compete, and the k best of them are returned exactly as by
 * dresd_search.  When fewer than k rows match, the ranks past them hold
 * idx -1, score -inf and zero tokens.
 *
 *   next_tok  device, [B] int32: the next token of each query.
 *   Other arguments, order, determinism, ownership and errors as for
 *   dresd_search (EINVAL also for a null next_tok when B > 0).  The first
 *   token of every row is kept by the index (4 bytes per row, built by
 *   dresd_index_create), so a filtered scan reads 64 more bytes per 16 rows.
 */
dresd_status dresd_search_filtered(dresd_index *ix, const float *queries,
                                   const int32_t *next_tok, int32_t B, int32_t k,
                                   int64_t *idx, float *score, int32_t *tokens,
                                   dresd_stream stream);

/*
 * Allocation-free search, for callers that cannot allocate device memory:
 * code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc.  The same search as dresd_search (same kernels, bitwise the same
 * outputs; a batch of 1,024-dim keys whose tiled-contraction lists would
 * not fit the scratch runs the shared-key scan instead), with its workspace
 * in a fixed library scratch of
 * DRESD_SCRATCH_BYTES that every device the library runs on holds until the
 * process ends, instead of the index's growable workspace.  It allocates no
 * device or host memory and never synchronises; the caller still passes the
 * queries and the outputs.
 *
 *   Arguments, order, determinism and errors as for dresd_search, and
 *   EINVAL when the search needs more workspace than DRESD_SCRATCH_BYTES
 *   even so (dresd_search_plan's workspace_bytes, the need of dresd_search,
 *   is an upper bound; e.g. one query up to k = 1024, or 64 queries at
 *   k = 32, fit).  Profiling (dresd_profile_*)
 *   does not time these calls.
 * Every call on one device shares that device's scratch, which keeps the
 * last call's contents (each search writes every scratch byte it reads
 * before reading it, so nothing needs clearing): calls that overlap on one
 * device -- on different streams, or with different indexes -- race, and
 * must be serialised by the caller (e.g. issued on one stream).
 */
#define DRESD_SCRATCH_BYTES (64LL << 20)
dresd_status dresd_search_noalloc(dresd_index *ix, const float *queries, int32_t B,
                                  int32_t k, int64_t *idx, float *score,
                                  int32_t *tokens, dresd_stream stream);

/* Describe an index.  Any output pointer (host) may be NULL.
 * Errors: EINVAL when ix is NULL. */
dresd_status dresd_index_info(const dresd_index *ix, int64_t *N, int32_t *d,
                              int32_t *L, int32_t *dtype);

/* Free an index and its workspace (synchronises its device).  NULL is
 * ignored. */
void dresd_index_destroy(dresd_index *ix);

/* Message for the last failing call on this thread ("" if none).  The
 * pointer stays valid until the next call on this thread. */
const char *dresd_last_error(void);

/*
 * Measurement support.  When enabled, every search ties HIP events to its
 * kernels' own dispatches (hipExtLaunchKernel): the begin and end of the main
 * scan kernel (the full pass over the keys), and the begin of the search's
 * first kernel and the end of its last, so that profiling adds no packets
 * between kernels.  dresd_profile_read synchronises those events and
 * returns the summed device milliseconds and the number of searches since
 * the last read, then clears them.  Outputs are host pointers (NULL allowed).
 * Errors: EINVAL when ix is NULL; EDEVICE.
 */
dresd_status dresd_profile_enable(dresd_index *ix, int32_t on);
dresd_status dresd_profile_read(dresd_index *ix, double *scan_ms,
                                double *search_ms, int64_t *searches);

/*
 * Measurement support: the achievable HBM read bandwidth of the device with
 * the scans' access pattern (every wave streams one contiguous range in
 * 1 KiB wave loads, 16 nontemporal loads in flight), the ceiling against
 * which a scan's bandwidth is judged beside the spec sheet's figure.
 *
 *   buf         device, `bytes` readable bytes (contents do not matter;
 *               only read).
 *   bytes       a multiple of 1024, at least 1 MiB (use far more than the
 *               last-level caches, e.g. several GiB).
 *   reps        1 <= reps <= 1000 timed read passes, after one untimed pass.
 *   workgroups  workgroups of 4 waves (0: four per compute unit).
 *   ms          host; mean device milliseconds per pass (HIP events).
 * Synchronises `stream`.  Allocates nothing on the device.
 * Errors: EINVAL (null pointer, sizes out of range), EDEVICE.
 */
dresd_status dresd_bw_probe(const void *buf, int64_t bytes, int32_t reps, int32_t workgroups,
                            double *ms, dresd_stream stream);

/*
 * Query-side transform of Algorithm 1 steps 4-6, for decode-step queries (or,
 * once, for the datastore rows that become keys):
 *   z   = (x - mean) / sqrt(var + eps_z)        z-score normalisation, Eq. 1
 *   v   = z W                                   first l principal components,
 *                                               Section 3.3
 *   y   = v / max(||v||_2, eps_n)               L2 normalisation, Eq. 2
 *
 *   x       device, [M, D] fp32 row-major (e.g. last hidden states).
 *   M       0 <= M < 2^31; M == 0 is a no-op.
 *   D       1 <= D <= 2^20.
 *   mean    device, [D] fp32: E[V] of the datastore sample.
 *   var     device, [D] fp32: Var[V] of the datastore sample (>= 0).
 *   eps_z   finite, >= 0 (the paper's eps of Eq. 1; 1e-5 is a common choice).
 *   W       device, [D, l] fp32 row-major: the principal components W_l.
 *   l       1 <= l <= 16384.
 *   eps_n   finite, >= 0 (the eps of Eq. 2; 1e-12 is a common choice).
 *   y       device, [M, l] fp32 row-major output (ready for dresd_search).
 *   stream  stream the transform runs on (asynchronous).
 * Arithmetic: fp32, the projection on the fp32 matrix cores; batches with
 * few output tiles split D across workgroups and add the partial sums in a
 * fixed order, so results are deterministic.  Ownership: all buffers are
 * caller-owned and must stay alive until `stream` completes; the partial sums
 * use a library buffer per (device, stream) that is allocated (synchronously)
 * on the first call on that stream that needs a larger one and kept, like
 * every buffer it outgrows, until the process ends: calls on different
 * streams may overlap, calls on one stream are ordered by it.
 * Errors: EINVAL (null pointer with M > 0, sizes or eps out of range),
 * ENOMEM, EUNSUPPORTED (the buffer would have to grow during stream
 * capture), EDEVICE.
 */
dresd_status dresd_transform(const float *x, int64_t M, int32_t D, const float *mean,
                             const float *var, float eps_z, const float *W, int32_t l,
                             float eps_n, float *y, dresd_stream stream);

/*
 * Draft assembly for batch verification (Section 3.6): the retrieved
 * continuations become the rows of an EOS-padded draft matrix.  For each
 * query, in rank order: a draft is the first `length` tokens of a
 * continuation with every token after its first EOS replaced by EOS; drafts
 * that start with EOS (nothing to propose, e.g. the padding ranks of
 * dresd_search_filtered) and repeats of an earlier draft are dropped; the
 * first r remaining drafts fill the rows, and rows past them are all EOS.
 *
 *   tokens  device, [B, k, L] int32 (as written by dresd_search).
 *   B >= 0 (0 is a no-op); 1 <= k <= DRESD_K_MAX; 1 <= L <= 4096;
 *   1 <= r <= k drafts; 1 <= length <= L tokens per draft; eos: the EOS id.
 *   drafts  device, [B, r, length] int32 output.
 *   count   device, [B] int32 output: drafts kept per query (<= r).
 *   stream  stream it runs on (asynchronous).
 * Deterministic; allocates nothing; buffers are caller-owned.
 * Errors: EINVAL (null pointer with B > 0, sizes out of range), EDEVICE.
 */
dresd_status dresd_pack_drafts(const int32_t *tokens, int32_t B, int32_t k, int32_t L,
                               int32_t r, int32_t length, int32_t eos, int32_t *drafts,
                               int32_t *count, dresd_stream stream);

/*
 * Describe how the next search of this shape would run (host outputs, NULL
 * allowed): the number of passes over sampled keys before the main pass, the
 * number of waves of the main scan (of the first launch when the batch
 * takes several), the bytes of workspace it needs,
 * which scan kernel runs it: 0 = single-tile scan (batches within one
 * 16-column query tile group, queries staged in LDS), 1 = shared-key scan
 * (queries held in registers, keys staged through LDS), 2 = single-tile scan
 * serving several query groups per launch (batches whose query operands
 * exceed one workgroup's LDS; the groups share each key range through L2),
 * 3 = tiled contraction (keys of more than 1,024 dims at batches of two or
 * more query tiles, and 1,024-dim keys at batches past four query tiles: key
 * and query blocks both streamed through LDS, column by column, for panels
 * of 16 or 32 key tiles), and the number of launches of the main scan (each
 * one pass over the keys for a part of the batch).
 * Errors: EINVAL for the same argument errors as dresd_search.
 */
dresd_status dresd_search_plan(const dresd_index *ix, int32_t B, int32_t k,
                               int32_t *sample_passes, int32_t *scan_waves,
                               int64_t *workspace_bytes, int32_t *scan_kind,
                               int32_t *launches);

/*
 * Partitioned (approximate) search.  The paper retrieves with an approximate
 * nearest-neighbour library (Section 3.5); this is its partitioned reading,
 * an inverted file: every key belongs to one of P partitions, each with a
 * centroid, and a search scores only the keys of the nprobe partitions whose
 * centroids score highest for the query.  The result is the exact top-k over
 * those keys (same ranking, scores and tie rule as dresd_search), so it
 * differs from dresd_search only where a true top-k key lies in a partition
 * that was not probed.
 *
 * dresd_ivf_create: embeddings / continuations / N / d / L / dtype as in
 *   dresd_index_create; centroids device [P, d] fp32 (unit rows, e.g. from
 *   dresd_kmeans_*), 1 <= P <= DRESD_PARTS_MAX; assign device [N] int32, the
 *   partition of each key, in [0, P).  Keys are stored grouped by partition
 *   (each partition padded to a 16-row tile); continuations stay in row
 *   order.  Copies everything, synchronises `stream`; the caller may free its
 *   buffers afterwards.  One-time cost: the grouping is a counting sort on
 *   the host.  Errors: EINVAL (nulls, ranges, an assignment outside [0, P)),
 *   ENOMEM, EDEVICE.
 * dresd_ivf_search: like dresd_search, probing 1 <= nprobe <= min(P,
 *   DRESD_K_MAX) partitions per query (the nprobe best centroids by inner
 *   product, ties to the lower id).  Ranks past the keys of the probed
 *   partitions hold index -1, score -inf and zero tokens.  Workspaces and
 *   the probe buffer are per stream, as for dresd_search: searches on
 *   different streams may overlap on the device; calls from several host
 *   threads must be serialised by the caller.
 * dresd_ivf_search_filtered: dresd_ivf_search with the next-token filter of
 *   dresd_search_filtered (next_tok device [B] int32): among the keys of the
 *   probed partitions only those whose continuation starts with the query's
 *   next token compete; ranks past them are padded the same way.
 * dresd_ivf_search_probes: the search with caller-chosen partitions: probes
 *   device [B, S] int32, 1 <= S <= DRESD_K_MAX; entries outside [0, P) are
 *   ignored and repeats count once; next_tok: NULL, or device [B] int32 for
 *   the next-token filter.
 * dresd_ivf_create_by_token: the next-token filter of Section 3.5 (a draft
 *   that does not start with the next token is dropped) as a partitioning:
 *   partition p holds the keys whose continuation starts with the p-th
 *   smallest distinct first token (P = the number of distinct first tokens,
 *   at most DRESD_PARTS_MAX); no centroids.  Arguments as in
 *   dresd_index_create.  Copies everything and reads the first column of
 *   `continuations` back to the host (synchronises `stream`); the grouping is
 *   a host sort of the first tokens.  Errors as dresd_ivf_create.
 *   dresd_ivf_search and dresd_ivf_search_filtered reject such an index
 *   (EINVAL: no centroids); dresd_ivf_search_probes takes partition ids in
 *   ascending token order.
 * dresd_ivf_search_next_token: on an index from dresd_ivf_create_by_token,
 *   the result of dresd_search_filtered (same keys compete, same ranking and
 *   tie rule, exact top-k) computed by scanning only the query's next-token
 *   partition: next_tok device [B] int32, any value (a token no key starts
 *   with gives a fully padded row).  Its cost follows the probed partitions'
 *   sizes, so it pays when the batch's next tokens together select fewer
 *   keys than the datastore holds (small batches); the full filtered scan
 *   reads every key once for the whole batch.  Scores come from the
 *   three-part exact query split at every batch size (within the 1e-5 bound
 *   of the small-batch scans).  Errors: EINVAL (NULLs, B < 0, k out of range,
 *   an index not grouped by token), ENOMEM, EUNSUPPORTED, EDEVICE.
 * dresd_ivf_info: host outputs (NULL allowed); tiles = 16-row tiles of the
 *   partitioned layout (padding included).
 * dresd_ivf_profile_enable / _read: as dresd_profile_*, for the scan of the
 *   probed partitions and the whole search.
 */
dresd_status dresd_ivf_create(const void *embeddings, const int32_t *continuations, int64_t N,
                              int32_t d, int32_t L, int32_t dtype, const float *centroids,
                              int32_t P, const int32_t *assign, dresd_stream stream,
                              dresd_ivf **out);
void dresd_ivf_destroy(dresd_ivf *ivf);
dresd_status dresd_ivf_info(const dresd_ivf *ivf, int64_t *N, int32_t *d, int32_t *L,
                            int32_t *dtype, int32_t *P, int64_t *tiles);
dresd_status dresd_ivf_search(dresd_ivf *ivf, const float *queries, int32_t B, int32_t k,
                              int32_t nprobe, int64_t *idx, float *score, int32_t *tokens,
                              dresd_stream stream);
dresd_status dresd_ivf_search_filtered(dresd_ivf *ivf, const float *queries,
                                       const int32_t *next_tok, int32_t B, int32_t k,
                                       int32_t nprobe, int64_t *idx, float *score,
                                       int32_t *tokens, dresd_stream stream);
dresd_status dresd_ivf_search_probes(dresd_ivf *ivf, const float *queries, const int32_t *probes,
                                     int32_t S, const int32_t *next_tok, int32_t B, int32_t k,
                                     int64_t *idx, float *score, int32_t *tokens,
                                     dresd_stream stream);
dresd_status dresd_ivf_create_by_token(const void *embeddings, const int32_t *continuations,
                                       int64_t N, int32_t d, int32_t L, int32_t dtype,
                                       dresd_stream stream, dresd_ivf **out);
dresd_status dresd_ivf_search_next_token(dresd_ivf *ivf, const float *queries,
                                         const int32_t *next_tok, int32_t B, int32_t k,
                                         int64_t *idx, float *score, int32_t *tokens,
                                         dresd_stream stream);
/*
 * Spherical k-means, the partitioning of the partitioned search (the
 * centroids and assignment that dresd_ivf_create takes).  Cosine similarity
 * of unit vectors (Eq. 3) is the inner product.
 *
 * dresd_kmeans_assign: assign[i] = the centroid with the largest inner
 *   product with row i, ties to the lower id; score[i] (NULL allowed) = that
 *   inner product (fp32 accumulation of exact products).
 *   x device [n, d] row-major in dtype; 0 <= n <= DRESD_N_MAX (0: no-op);
 *   1 <= d <= 16384; centroids device [P, d] fp32, 1 <= P <= DRESD_PARTS_MAX;
 *   assign device [n] int32 out; score device [n] fp32 out.
 * dresd_kmeans_update: each centroid becomes the unit vector along the sum of
 *   the rows assigned to it; a centroid with no rows (or a zero sum) is left
 *   as it is.  Sums are exact to 2^-30 per element and independent of the
 *   order of the rows (deterministic).  x as above with n < 2^31; assign
 *   device [n] int32, each in [0, P) (not checked: the caller's contract);
 *   centroids device [P, d] fp32 in/out; counts device [P] int32 out (rows per
 *   centroid, NULL allowed).  Uses a workspace of P*d*8 + P*4 bytes per
 *   (device, stream), allocated (synchronously) on first use on that stream
 *   and kept, like every buffer it outgrows, until the process ends: calls
 *   on different streams may overlap, calls on one stream are ordered by it.
 * dresd_kmeans_init: the starting centroids of the iteration: P distinct
 *   rows spread evenly through the row order, centroid j = row pick(j)
 *   scaled to unit length (a zero row gives a zero centroid), with
 *   pick(j) = (o + floor(j n / P)) mod n and o = s mod n, where s is the
 *   first output of SplitMix64 (Steele, Lea and Flood, 2014) started from
 *   state `seed`.  x as above with 1 <= n; 1 <= P <= min(n,
 *   DRESD_PARTS_MAX); centroids device [P, d] fp32 out (the norm is taken in
 *   fp64 over the decoded elements, each element rounded to fp32 once).
 *   Allocates nothing.
 * All three are asynchronous on `stream`.  Errors: EINVAL (ranges, nulls),
 * ENOMEM, EDEVICE.
 */
dresd_status dresd_kmeans_assign(const void *x, int64_t n, int32_t d, int32_t dtype,
                                 const float *centroids, int32_t P, int32_t *assign,
                                 float *score, dresd_stream stream);
dresd_status dresd_kmeans_update(const void *x, int64_t n, int32_t d, int32_t dtype,
                                 const int32_t *assign, int32_t P, float *centroids,
                                 int32_t *counts, dresd_stream stream);
dresd_status dresd_kmeans_init(const void *x, int64_t n, int32_t d, int32_t dtype, int32_t P,
                               uint64_t seed, float *centroids, dresd_stream stream);

dresd_status dresd_ivf_profile_enable(dresd_ivf *ivf, int32_t on);
dresd_status dresd_ivf_profile_read(dresd_ivf *ivf, double *scan_ms, double *search_ms,
                                    int64_t *searches);

#ifdef __cplusplus
}
#endif
#endif /* DRESD_H */
