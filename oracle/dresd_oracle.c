/*
 * CPU oracle for DReSD's dense retrieval step -- TEST INFRASTRUCTURE ONLY.
 *
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg
 * may load this library.  The product path (the HIP library) never calls it,
 * shares no code, header, table or helper with it, and must fail loudly when
 * its own extension is missing instead of falling back to this file.
 *
 * What it computes (DReSD, Section 3.5, Eq. 3, read with Section 3.4, Eq. 2):
 * the datastore is a key -> value map whose keys are L2-normalised token
 * embeddings and whose values are the next L tokens.  Retrieval returns the
 * value of the key with the highest cosine similarity to the (L2-normalised)
 * query.  For unit-norm keys and queries the cosine is the plain inner
 * product, so the denominator max(|a||b|, eps) of Eq. 3 is 1 and is not
 * applied.  Batch verification (Section 3.6) consumes several drafts, so the
 * argmax of Eq. 3 is taken as the k best keys.
 *
 * Precision: the paper fixes none.  Each score is the exact inner product,
 * accumulated in fp64 in dimension order (every product of an fp32 query
 * element and an fp32/f16/bf16 key element is exact in fp64), then rounded
 * once to fp32.  Ranking is decided on that fp32 value, which is the
 * precision the device path decides in: score descending, equal scores by
 * lowest row index.  No blocking, fusion or reordering of the arithmetic
 * beyond that definition; queries are looped inside rows only so that the
 * datastore is read once per batch, which does not change any value.
 *
 * Filtered retrieval (Section 3.5, with Section 3.1): the next token x_{t+1}
 * that the LLM produced alongside the query embedding removes every draft
 * that does not start with it.  oracle_topk_filtered reads this as
 * filter-then-select: for query b only rows i whose value starts with
 * next_tok[b] (cont[i, 0] == next_tok[b]) compete, and the k best of them are
 * returned; ranks past the number of matching rows hold index -1, score
 * -inf and zero tokens.
 *
 * Partitioned retrieval (the approximate search the paper runs through its
 * ANN library, Section 3.5, read as an inverted file): every row belongs to
 * one partition (assign[i] in [0, P)), each query probes a set of
 * partitions, and oracle_topk_partitioned returns the exact k best rows among
 * the rows of the probed partitions, with the same padding as the filter.
 * Probe entries outside [0, P) are ignored and repeated entries count once.
 *
 * Parity pins live in the CPU tests (closed forms, exact brute force,
 * invariants, duplicates, self-retrieval MRR of Eq. 4, planted mutations).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { ORACLE_F32 = 0, ORACLE_F16 = 1, ORACLE_BF16 = 2 };

/* Planted-mistake hooks: a non-zero value makes the oracle wrong on purpose
 * so that the CPU tests can show each pin catches that class of mistake.
 * Zero (the default) is the oracle as specified. */
static int g_mutation = 0;
void oracle_set_mutation(int m) { g_mutation = m; }

/* IEEE binary16 bits -> value, from the format's definition:
 * sign, 5-bit biased exponent (bias 15), 10-bit fraction, subnormals at
 * exponent 0 scaled by 2^-24. */
static double f16_bits_value(uint16_t h) {
  int sign = h >> 15;
  int ex = (h >> 10) & 0x1f;
  int fr = h & 0x3ff;
  double v;
  if (ex == 0)
    v = ldexp((double)fr, -24);
  else if (ex == 31)
    v = fr ? NAN : INFINITY;
  else
    v = ldexp((double)(fr | 0x400), ex - 25);
  return sign ? -v : v;
}

/* bfloat16 bits are the upper half of an IEEE binary32. */
static double bf16_bits_value(uint16_t h) {
  uint32_t u = (uint32_t)h << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

double oracle_decode(const void *emb, int dtype, int64_t off) {
  switch (dtype) {
  case ORACLE_F32:
    return (double)((const float *)emb)[off];
  case ORACLE_F16:
    return f16_bits_value(((const uint16_t *)emb)[off]);
  default:
    return bf16_bits_value(((const uint16_t *)emb)[off]);
  }
}

/* Key row i decoded to fp64 (exact for every storage type). */
static void decode_row(const void *emb, int dtype, int32_t d, int64_t i, double *e) {
  for (int32_t j = 0; j < d; ++j) e[j] = oracle_decode(emb, dtype, i * (int64_t)d + j);
}

/* Eq. 3 with unit norms: the exact inner product of query q and a decoded
 * key row e, summed in dimension order in fp64, rounded once to fp32. */
static float score_row(const double *e, int32_t d, const float *q) {
  double s = 0.0;
  int32_t jn = (g_mutation == 1) ? d - 1 : d; /* mutation 1: drop a term */
  for (int32_t j = 0; j < jn; ++j) {
    /* mutation 3: key element taken at the mirrored dimension */
    int32_t je = (g_mutation == 3) ? d - 1 - j : j;
    double p = (double)q[j] * e[je];
    s = (g_mutation == 2 && j == 0) ? s - p : s + p; /* mutation 2: sign */
  }
  float f = (float)s;
  if (g_mutation == 6) { /* mutation 6: score truncated to 16 bits */
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    u &= 0xffff0000u;
    memcpy(&f, &u, sizeof f);
  }
  return f;
}

typedef struct {
  float s;
  int64_t i;
} item;

/* Ranking order: higher score first; equal scores by lower row index. */
static int better(item a, item b) {
  if (g_mutation == 4) /* mutation 4: ties broken by highest index */
    return a.s > b.s || (a.s == b.s && a.i > b.i);
  if (g_mutation == 5) /* mutation 5: ascending scores */
    return a.s < b.s || (a.s == b.s && a.i < b.i);
  return a.s > b.s || (a.s == b.s && a.i < b.i);
}

static int cmp_items(const void *pa, const void *pb) {
  item a = *(const item *)pa, b = *(const item *)pb;
  if (better(a, b)) return -1;
  if (better(b, a)) return 1;
  return 0;
}

/* Keep the m best items seen so far in 'best' (sorted, best first). */
static void offer(item *best, int64_t *count, int64_t m, item x) {
  int64_t c = *count;
  if (c == m && !better(x, best[m - 1])) return;
  int64_t pos = (c < m) ? c : m - 1;
  while (pos > 0 && better(x, best[pos - 1])) {
    best[pos] = best[pos - 1];
    --pos;
  }
  best[pos] = x;
  if (c < m) *count = c + 1;
}

/* Partitioned retrieval: probed[b * P + p] != 0 when query b probes
 * partition p; assign[i] is row i's partition.  NULL when not partitioned. */
static const int32_t *g_assign = NULL;
static const unsigned char *g_probed = NULL;
static int32_t g_parts = 0;

/* Row i takes part for query b: every row without a filter; with one, the
 * rows whose value starts with that query's next token; in a partitioned
 * search, the rows of the partitions the query probes. */
static int admitted(const int32_t *cont, int32_t L, const int32_t *next_tok, int64_t i,
                    int32_t b) {
  if (g_probed && !g_probed[(int64_t)b * g_parts + g_assign[i]]) return 0;
  if (!next_tok) return 1;
  /* mutation 8: the filter reads the value's second token */
  int32_t first = cont[i * L + ((g_mutation == 8 && L > 1) ? 1 : 0)];
  return first == next_tok[b];
}

/*
 * Exact top-k for B queries over N keys (the rows admitted by next_tok when
 * it is not NULL).
 *   emb   [N, d] row-major, dtype ORACLE_F32 / ORACLE_F16 / ORACLE_BF16
 *   Q     [B, d] fp32 row-major
 *   cont  [N, L] int32 (may be NULL when L == 0 and next_tok is NULL)
 * Outputs (caller-owned):
 *   idx [B, k] int64, score [B, k] fp32, tokens [B, k, L] int32 (NULL ok),
 *   next_score [B] fp32: the (k+1)-th best score, NaN when there is none
 *   (NULL ok).  Ranks past the admitted rows: idx -1, score -inf, tokens 0.
 * Returns 0, or -1 on invalid arguments / allocation failure.
 */
static int topk_impl(const void *emb, int dtype, int64_t N, int32_t d, const float *Q, int32_t B,
                     int32_t k, const int32_t *cont, int32_t L, const int32_t *next_tok,
                     int64_t *idx, float *score, int32_t *tokens, float *next_score,
                     int32_t nthreads) {
  if (!emb || !Q || !idx || !score || N < 1 || d < 1 || B < 0 || k < 1 ||
      k > N || dtype < 0 || dtype > 2)
    return -1;
  if (next_tok && (!cont || L < 1)) return -1;
  if (B == 0) return 0;
  int64_t m = (k < N) ? (int64_t)k + 1 : (int64_t)k;
  int nt = 1;
#ifdef _OPENMP
  nt = nthreads > 0 ? nthreads : omp_get_max_threads();
#endif
  int fail = 0;
  item *all = (item *)malloc(sizeof(item) * (size_t)nt * (size_t)B * (size_t)m);
  int64_t *cnt = (int64_t *)calloc((size_t)nt * (size_t)B, sizeof(int64_t));
  if (!all || !cnt) {
    free(all);
    free(cnt);
    return -1;
  }
#ifdef _OPENMP
#pragma omp parallel num_threads(nt)
#endif
  {
    int t = 0, T = 1;
#ifdef _OPENMP
    t = omp_get_thread_num();
    T = omp_get_num_threads();
#endif
    int64_t lo = N * t / T, hi = N * (t + 1) / T;
    double *e = (double *)malloc(sizeof(double) * (size_t)d);
    if (!e) fail = 1;
    for (int64_t i = lo; e && i < hi; ++i) {
      decode_row(emb, dtype, d, i, e);
      for (int32_t b = 0; b < B; ++b) {
        if (!admitted(cont, L, next_tok, i, b)) continue;
        item x;
        x.s = score_row(e, d, Q + (int64_t)b * d);
        x.i = i;
        offer(all + ((size_t)t * B + b) * m, cnt + (size_t)t * B + b, m, x);
      }
    }
    free(e);
  }
  if (fail) {
    free(all);
    free(cnt);
    return -1;
  }
  item *merged = (item *)malloc(sizeof(item) * (size_t)nt * (size_t)m);
  if (!merged) {
    free(all);
    free(cnt);
    return -1;
  }
  for (int32_t b = 0; b < B; ++b) {
    int64_t tot = 0;
    for (int t = 0; t < nt; ++t) {
      int64_t c = cnt[(size_t)t * B + b];
      memcpy(merged + tot, all + ((size_t)t * B + b) * m, sizeof(item) * (size_t)c);
      tot += c;
    }
    qsort(merged, (size_t)tot, sizeof(item), cmp_items);
    for (int32_t r = 0; r < k; ++r) {
      const int64_t o = (int64_t)b * k + r;
      if (r >= tot) { /* fewer admitted rows than k */
        idx[o] = -1;
        score[o] = -INFINITY;
        if (tokens && L > 0) memset(tokens + o * L, 0, sizeof(int32_t) * (size_t)L);
        continue;
      }
      idx[o] = merged[r].i;
      score[o] = merged[r].s;
      if (tokens && cont && L > 0) {
        int64_t src = merged[r].i;
        if (g_mutation == 7 && src + 1 < N) ++src; /* mutation 7: off-by-one */
        memcpy(tokens + o * L, cont + src * L, sizeof(int32_t) * (size_t)L);
      }
    }
    if (next_score) next_score[b] = (k < tot) ? merged[k].s : NAN;
  }
  free(merged);
  free(all);
  free(cnt);
  return 0;
}

int oracle_topk(const void *emb, int dtype, int64_t N, int32_t d,
                const float *Q, int32_t B, int32_t k, const int32_t *cont,
                int32_t L, int64_t *idx, float *score, int32_t *tokens,
                float *next_score, int32_t nthreads) {
  return topk_impl(emb, dtype, N, d, Q, B, k, cont, L, NULL, idx, score, tokens, next_score,
                   nthreads);
}

/* Filtered retrieval of Section 3.5: next_tok [B] int32, the token each
 * query's drafts must start with. */
int oracle_topk_filtered(const void *emb, int dtype, int64_t N, int32_t d, const float *Q,
                         int32_t B, int32_t k, const int32_t *cont, int32_t L,
                         const int32_t *next_tok, int64_t *idx, float *score, int32_t *tokens,
                         float *next_score, int32_t nthreads) {
  if (!next_tok) return -1;
  return topk_impl(emb, dtype, N, d, Q, B, k, cont, L, next_tok, idx, score, tokens, next_score,
                   nthreads);
}

/* Partitioned retrieval: assign [N] int32 in [0, P); probes [B, S] int32
 * (entries outside [0, P) ignored); next_tok [B] (NULL: no filter) adds the
 * next-token filter: a row takes part when its partition is probed and its
 * value starts with the query's next token.  Not reentrant (the probe sets
 * live in file-scope state for the duration of the call). */
int oracle_topk_partitioned(const void *emb, int dtype, int64_t N, int32_t d, const float *Q,
                            int32_t B, int32_t k, const int32_t *cont, int32_t L,
                            const int32_t *assign, int32_t P, const int32_t *probes, int32_t S,
                            const int32_t *next_tok, int64_t *idx, float *score, int32_t *tokens,
                            float *next_score, int32_t nthreads) {
  if (!assign || P < 1 || S < 0 || (S > 0 && !probes) || B < 0) return -1;
  if (next_tok && (!cont || L < 1)) return -1;
  for (int64_t i = 0; i < N; ++i)
    if (assign[i] < 0 || assign[i] >= P) return -1;
  unsigned char *probed = (unsigned char *)calloc((size_t)(B > 0 ? B : 1) * (size_t)P, 1);
  if (!probed) return -1;
  /* mutation 9: the last probe of every query is lost */
  const int32_t used = (g_mutation == 9 && S > 0) ? S - 1 : S;
  for (int32_t b = 0; b < B; ++b)
    for (int32_t j = 0; j < used; ++j) {
      const int32_t p = probes[(int64_t)b * S + j];
      if (p >= 0 && p < P) probed[(int64_t)b * P + p] = 1;
    }
  g_assign = assign;
  g_probed = probed;
  g_parts = P;
  const int rc = topk_impl(emb, dtype, N, d, Q, B, k, cont, L, next_tok, idx, score, tokens,
                           next_score, nthreads);
  g_assign = NULL;
  g_probed = NULL;
  g_parts = 0;
  free(probed);
  return rc;
}

/* Scores of the given rows for one query (the same arithmetic as above);
 * used to re-score whatever indices the device path returns. */
int oracle_score_rows(const void *emb, int dtype, int64_t N, int32_t d,
                      const float *q, const int64_t *rows, int64_t nrows,
                      float *out) {
  if (!emb || !q || !rows || !out || d < 1) return -1;
  double *e = (double *)malloc(sizeof(double) * (size_t)d);
  if (!e) return -1;
  for (int64_t r = 0; r < nrows; ++r) {
    if (rows[r] < 0 || rows[r] >= N) {
      free(e);
      return -1;
    }
    decode_row(emb, dtype, d, rows[r], e);
    out[r] = score_row(e, d, q);
  }
  free(e);
  return 0;
}
