/*
 * oracle.c -- plain, slow CPU oracle for exact top-k context-sparse decode
 * attention.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file: only the tests, the package smoke check and the benchmark's
 * CPU-baseline leg use it.  It shares no code, header, table or helper with
 * the HIP library; it is written from the paper's statement of the method.
 *
 * What it computes (arXiv 2605.24168):
 *   - Section 3 ("Algorithms"): at every decode step attention is restricted
 *     to the k context positions chosen by *exact* top-k selection on the
 *     attention scores ("oracle top-k"), as opposed to an approximate indexer.
 *   - Table 1 caption: an S-times sparsity means every query head attends to
 *     a 1/S fraction of the context, so k = N/S per query head.
 *   - Section 1 ("Sparsity can be leveraged for system gains") and Section 4:
 *     the sparsity is per query, per query head and per token (no blocks),
 *     also under grouped-query attention, where several query heads share one
 *     key/value head.
 *   - Section 1 (introduction): the attention that is sparsified is ordinary
 *     scaled dot-product attention, softmax(q K^T * scale) V.
 * Readings where the paper is silent (each is also listed in the design
 * notes of the repository):
 *   - scale = 1/sqrt(d) unless the caller passes another positive value;
 *   - k = clamp(round_half_up(L/S), 1, L) or clamp(ceil(L/S), 1, L);
 *   - ties in the score are broken toward the lower context position;
 *   - ranking uses the unscaled score q.k; the scale enters only the softmax;
 *   - query head h reads KV head floor(h / G), G = Hq / Hkv;
 *   - in "group-shared" mode one index set per KV head is chosen from the
 *     sum over the group's query heads of their raw scores, and every head
 *     then applies softmax to its own scores over that shared set;
 *   - only positions j < L_b of sequence b exist; positions beyond are
 *     never read.
 *
 * Arithmetic is IEEE double throughout.  bfloat16 inputs are decoded exactly
 * (a bfloat16 value is the upper half of a float32).  Rows are independent,
 * so OpenMP runs them in parallel; no arithmetic is reordered inside a row.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORACLE_OK 0
#define ORACLE_EINVAL (-1)
#define ORACLE_ENONFINITE (-2)
#define ORACLE_ENOMEM (-3)

/* Layout of a key or value cache, as the oracle sees it (host memory). */
typedef struct {
  const void *data;
  int32_t dtype;            /* 0: float32, 1: bfloat16 stored as uint16 bits   */
  int32_t paged;            /* 0: [B][Hkv][ncap][d]                           */
                            /* 1: [num_pages][page_size][Hkv][d] + block table */
  int64_t ncap;             /* contiguous: positions per sequence              */
  int64_t num_pages;        /* paged: pages in the pool                        */
  int32_t page_size;        /* paged: tokens per page                          */
  int32_t max_pages;        /* paged: columns of block_table                   */
  const int32_t *block_table; /* paged: [B][max_pages] physical page ids       */
} oracle_cache;

static double decode_elem(const void *base, int32_t dtype, int64_t off) {
  if (dtype == 1) {
    uint32_t u = (uint32_t)((const uint16_t *)base)[off] << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
  }
  return (double)((const float *)base)[off];
}

/* Element offset of (sequence b, KV head g, logical position j, channel 0). */
static int64_t cache_row_offset(const oracle_cache *c, int Hkv, int d, int b,
                                int g, int64_t j) {
  if (!c->paged) return (((int64_t)b * Hkv + g) * c->ncap + j) * d;
  int64_t page = c->block_table[(int64_t)b * c->max_pages + j / c->page_size];
  int64_t slot = j % c->page_size;
  return ((page * c->page_size + slot) * Hkv + g) * (int64_t)d;
}

static int64_t cache_capacity(const oracle_cache *c) {
  return c->paged ? (int64_t)c->max_pages * c->page_size : c->ncap;
}

/* Check that every position a sequence of length L may touch is addressable. */
static int check_cache(const oracle_cache *c, int b, int64_t L) {
  if (!c || !c->data) return ORACLE_EINVAL;
  if (L > cache_capacity(c)) return ORACLE_EINVAL;
  if (c->paged) {
    if (c->page_size <= 0 || !c->block_table) return ORACLE_EINVAL;
    int64_t pages = (L + c->page_size - 1) / c->page_size;
    for (int64_t p = 0; p < pages; ++p) {
      int32_t id = c->block_table[(int64_t)b * c->max_pages + p];
      if (id < 0 || id >= c->num_pages) return ORACLE_EINVAL;
    }
  }
  return ORACLE_OK;
}

/*
 * Budget k for a sequence of length L at sparsity S (Table 1 caption: each
 * query head attends to a 1/S fraction of the tokens).  rounding 0 = nearest
 * with halves rounded up, 1 = ceiling.  At least one position is kept when
 * the sequence is not empty, and never more than L.
 */
int64_t oracle_budget(int64_t L, double ratio, int32_t rounding) {
  if (L <= 0) return 0;
  double x = (double)L / ratio;
  double k = rounding == 1 ? ceil(x) : floor(x + 0.5);
  if (k < 1.0) k = 1.0;
  if (k > (double)L) k = (double)L;
  return (int64_t)k;
}

static int64_t row_budget(int64_t L, double ratio, int32_t rounding,
                          const int32_t *k_override, int b) {
  if (k_override) {
    int64_t k = k_override[b];
    if (k < 0) k = 0;
    if (k > L) k = L;
    return k;
  }
  return oracle_budget(L, ratio, rounding);
}

/* Plain dot product of two length-d double vectors, summed left to right. */
static double dot(const double *a, const double *b, int d) {
  double s = 0.0;
  for (int i = 0; i < d; ++i) s += a[i] * b[i];
  return s;
}

static void load_vec(const void *base, int32_t dtype, int64_t off, int d,
                     double *out) {
  for (int i = 0; i < d; ++i) out[i] = decode_elem(base, dtype, off + i);
}

/*
 * Total order used for selection: larger score first; equal scores go to
 * the lower position.
 */
typedef struct {
  double s;
  int64_t j;
} scored_pos;

static int by_score_desc_then_pos(const void *pa, const void *pb) {
  const scored_pos *a = (const scored_pos *)pa, *b = (const scored_pos *)pb;
  if (a->s > b->s) return -1;
  if (a->s < b->s) return 1;
  return (a->j > b->j) - (a->j < b->j);
}

static int by_int32_asc(const void *pa, const void *pb) {
  int32_t a = *(const int32_t *)pa, b = *(const int32_t *)pb;
  return (a > b) - (a < b);
}

/*
 * Exact top-k of one row of scores (Section 3, exact oracle top-k): sort all
 * L positions under the total order above and keep the first k.  Writes the
 * k kept positions in ascending order to idx[0..k) and -1 to idx[k..k_max).
 * *tau receives the k-th largest score (the smallest kept one), NaN if k = 0.
 */
int32_t oracle_select_row(const double *scores, int64_t L, int64_t k,
                          int64_t k_max, int32_t *idx, double *tau) {
  if (L < 0 || k < 0 || k > L || k > k_max) return ORACLE_EINVAL;
  for (int64_t j = 0; j < L; ++j)
    if (!isfinite(scores[j])) return ORACLE_ENONFINITE;
  scored_pos *all = (scored_pos *)malloc(sizeof(scored_pos) * (size_t)(L > 0 ? L : 1));
  if (!all) return ORACLE_ENOMEM;
  for (int64_t j = 0; j < L; ++j) {
    all[j].s = scores[j];
    all[j].j = j;
  }
  qsort(all, (size_t)L, sizeof(scored_pos), by_score_desc_then_pos);
  for (int64_t t = 0; t < k; ++t) idx[t] = (int32_t)all[t].j;
  if (tau) *tau = k > 0 ? all[k - 1].s : NAN;
  free(all);
  qsort(idx, (size_t)k, sizeof(int32_t), by_int32_asc);
  for (int64_t t = k; t < k_max; ++t) idx[t] = -1;
  return ORACLE_OK;
}

/*
 * Forced positions, the scaffolding of the paper's long-context runs (the
 * SWE-Bench appendix keeps 128 sink and 128 local positions besides the
 * exact top-k; the extreme top-K sweep keeps 64 sinks): the first n_sink
 * and the last n_local positions of a sequence are always attended, and
 * the exact top-k budget kh covers the positions in between.  Sinks take
 * precedence when the two overlap.
 */
static void forced_counts(int64_t L, int64_t n_sink, int64_t n_local, int64_t *ns, int64_t *nl) {
  *ns = n_sink < L ? n_sink : L;
  *nl = n_local < L - *ns ? n_local : L - *ns;
}

/*
 * The kept set of one row with forced positions: positions 0..ns-1, then
 * the exact top-kh of positions ns..L-nl-1 (scores descending, positions
 * ascending on ties; ascending in idx), then L-nl..L-1, then -1 padding to
 * k_max.  tau gets the kh-th largest middle score (NaN when kh = 0).
 */
int32_t oracle_select_forced(const double *scores, int64_t L, int64_t n_sink, int64_t n_local,
                             int64_t kh, int64_t k_max, int32_t *idx, double *tau) {
  if (L < 0 || n_sink < 0 || n_local < 0 || kh < 0) return ORACLE_EINVAL;
  int64_t ns, nl;
  forced_counts(L, n_sink, n_local, &ns, &nl);
  int64_t mid = L - ns - nl;
  if (kh > mid || ns + kh + nl > k_max) return ORACLE_EINVAL;
  for (int64_t t = 0; t < ns; ++t) idx[t] = (int32_t)t;
  int rc = oracle_select_row(scores + ns, mid, kh, kh, idx + ns, tau);
  if (rc) return rc;
  for (int64_t t = 0; t < kh; ++t) idx[ns + t] += (int32_t)ns;
  for (int64_t t = 0; t < nl; ++t) idx[ns + kh + t] = (int32_t)(L - nl + t);
  for (int64_t t = ns + kh + nl; t < k_max; ++t) idx[t] = -1;
  return ORACLE_OK;
}

/* Heavy budget of a row with forced positions: the ratio (or override) rule
 * on the whole sequence, capped by the positions left between the forced
 * ones; and the row's total. */
static int64_t heavy_budget(int64_t L, double ratio, int32_t rounding, const int32_t *k_override,
                            int b, int64_t n_sink, int64_t n_local, int64_t *total) {
  int64_t ns, nl;
  forced_counts(L, n_sink, n_local, &ns, &nl);
  int64_t kh = row_budget(L, ratio, rounding, k_override, b);
  if (kh > L - ns - nl) kh = L - ns - nl;
  if (total) *total = ns + nl + kh;
  return kh;
}

typedef struct {
  int B, Hq, Hkv, d;
  const void *q;
  int32_t q_dtype;
  const oracle_cache *K;
  const oracle_cache *V;
  const int32_t *seq_lens;
  int32_t group_shared;
  /* Low-channel indexer (Double Sparsity, Table 2 and Section 4): when lab
   * is set, selection scores come from a label cache holding nlab of the
   * d channels of every key; column c of KV head g's labels is channel
   * channels[g * nlab + c] (the query's channel it multiplies). */
  const oracle_cache *lab;
  int nlab;
  const int32_t *channels;
} problem;

static int check_problem(const problem *p, int need_v) {
  if (p->B < 0 || p->Hq <= 0 || p->Hkv <= 0 || p->d <= 0) return ORACLE_EINVAL;
  if (p->lab) {
    if (p->nlab <= 0 || p->nlab > p->d || !p->channels) return ORACLE_EINVAL;
    for (int64_t i = 0; i < (int64_t)p->Hkv * p->nlab; ++i)
      if (p->channels[i] < 0 || p->channels[i] >= p->d) return ORACLE_EINVAL;
    for (int b = 0; b < p->B; ++b)
      if (p->seq_lens[b] < 0 || check_cache(p->lab, b, p->seq_lens[b])) return ORACLE_EINVAL;
  }
  if (p->Hq % p->Hkv != 0) return ORACLE_EINVAL;
  if (!p->q || !p->K || !p->seq_lens) return ORACLE_EINVAL;
  if (need_v && !p->V) return ORACLE_EINVAL;
  for (int b = 0; b < p->B; ++b) {
    if (p->seq_lens[b] < 0) return ORACLE_EINVAL;
    if (check_cache(p->K, b, p->seq_lens[b])) return ORACLE_EINVAL;
    if (need_v && check_cache(p->V, b, p->seq_lens[b])) return ORACLE_EINVAL;
  }
  return ORACLE_OK;
}

/*
 * Selection scores of one row (Section 3 with the readings above).
 * Per-head mode: row = query head h, score_j = q_h . K[g(h)]_j.
 * Group-shared mode: row = KV head g, score_j = sum over the group's query
 * heads h of (q_h . K[g]_j), each dot product taken separately.
 */
static void row_scores(const problem *p, int b, int row, double *qbuf,
                       double *kbuf, double *out) {
  int G = p->Hq / p->Hkv;
  int64_t L = p->seq_lens[b];
  int g = p->group_shared ? row : row / G;
  int h0 = p->group_shared ? row * G : row;
  int nh = p->group_shared ? G : 1;
  for (int64_t j = 0; j < L; ++j) {
    double s = 0.0;
    if (p->lab) {
      /* Approximate score: the query's label channels times the key's labels. */
      const int32_t *ch = p->channels + (int64_t)g * p->nlab;
      load_vec(p->lab->data, p->lab->dtype, cache_row_offset(p->lab, p->Hkv, p->nlab, b, g, j),
               p->nlab, kbuf);
      for (int t = 0; t < nh; ++t) {
        load_vec(p->q, p->q_dtype, ((int64_t)b * p->Hq + h0 + t) * p->d, p->d, qbuf);
        for (int c = 0; c < p->nlab; ++c) s += qbuf[ch[c]] * kbuf[c];
      }
    } else {
      load_vec(p->K->data, p->K->dtype, cache_row_offset(p->K, p->Hkv, p->d, b, g, j),
               p->d, kbuf);
      for (int t = 0; t < nh; ++t) {
        load_vec(p->q, p->q_dtype, ((int64_t)b * p->Hq + h0 + t) * p->d, p->d, qbuf);
        s += dot(qbuf, kbuf, p->d);
      }
    }
    out[j] = s;
  }
}

static problem make_problem(int B, int Hq, int Hkv, int d, const void *q,
                            int32_t q_dtype, const oracle_cache *K,
                            const oracle_cache *V, const int32_t *seq_lens,
                            int32_t group_shared) {
  problem p;
  p.B = B; p.Hq = Hq; p.Hkv = Hkv; p.d = d;
  p.q = q; p.q_dtype = q_dtype; p.K = K; p.V = V;
  p.seq_lens = seq_lens; p.group_shared = group_shared;
  p.lab = NULL; p.nlab = 0; p.channels = NULL;
  return p;
}

static int set_threads(int nthreads) {
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
  return omp_get_max_threads();
#else
  (void)nthreads;
  return 1;
#endif
}

/* Scores of every row: out[b][row][j] for j < L_b; NaN for L_b <= j < ncap. */
static int32_t scores_impl(const problem *pp, int64_t ncap, double *out, int nthreads) {
  const problem p = *pp;
  int B = p.B, d = p.d;
  const int32_t *seq_lens = p.seq_lens;
  int rc = check_problem(&p, 0);
  if (rc) return rc;
  int R = p.group_shared ? p.Hkv : p.Hq;
  for (int b = 0; b < B; ++b)
    if (seq_lens[b] > ncap) return ORACLE_EINVAL;
  set_threads(nthreads);
  int failed = 0;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t r = 0; r < (int64_t)B * R; ++r) {
    int b = (int)(r / R), row = (int)(r % R);
    double *qbuf = (double *)malloc(sizeof(double) * d * 2);
    if (!qbuf) { failed = 1; continue; }
    double *dst = out + r * ncap;
    row_scores(&p, b, row, qbuf, qbuf + d, dst);
    for (int64_t j = seq_lens[b]; j < ncap; ++j) dst[j] = NAN;
    free(qbuf);
  }
  return failed ? ORACLE_ENOMEM : ORACLE_OK;
}

int32_t oracle_scores(int B, int Hq, int Hkv, int d, const void *q,
                      int32_t q_dtype, const oracle_cache *K,
                      const int32_t *seq_lens, int32_t group_shared,
                      int64_t ncap, double *out, int nthreads) {
  problem p = make_problem(B, Hq, Hkv, d, q, q_dtype, K, NULL, seq_lens, group_shared);
  return scores_impl(&p, ncap, out, nthreads);
}

/* Approximate selection scores of the low-channel indexer: for position j,
 * the sum over label columns c of q[channels[g][c]] * labels[j][c] (summed
 * over the group's query heads in group-shared mode).  NaN at j >= L_b. */
int32_t oracle_label_scores(int B, int Hq, int Hkv, int d, const void *q,
                            int32_t q_dtype, const oracle_cache *labels, int nlab,
                            const int32_t *channels, const int32_t *seq_lens,
                            int32_t group_shared, int64_t ncap, double *out, int nthreads) {
  problem p = make_problem(B, Hq, Hkv, d, q, q_dtype, labels, NULL, seq_lens, group_shared);
  p.lab = labels;
  p.nlab = nlab;
  p.channels = channels;
  return scores_impl(&p, ncap, out, nthreads);
}

/*
 * Exact top-k over caller-given float32 scores laid out [B][R][ncap]
 * (the scores are widened to double exactly, so the selection is the one
 * the total order defines on those very float32 values).
 */
int32_t oracle_select_f32(int B, int R, int64_t ncap, const float *scores,
                          const int32_t *seq_lens, double ratio,
                          int32_t rounding, const int32_t *k_override,
                          int64_t n_sink, int64_t n_local,
                          int64_t k_max, int32_t *idx, double *tau,
                          int nthreads) {
  if (B < 0 || R <= 0 || !scores || !seq_lens || !idx || !(ratio > 0.0))
    return ORACLE_EINVAL;
  if (n_sink < 0 || n_local < 0) return ORACLE_EINVAL;
  for (int b = 0; b < B; ++b) {
    int64_t total;
    if (seq_lens[b] < 0 || seq_lens[b] > ncap) return ORACLE_EINVAL;
    heavy_budget(seq_lens[b], ratio, rounding, k_override, b, n_sink, n_local, &total);
    if (total > k_max) return ORACLE_EINVAL;
  }
  set_threads(nthreads);
  int rc_all = ORACLE_OK;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t r = 0; r < (int64_t)B * R; ++r) {
    int b = (int)(r / R);
    int64_t L = seq_lens[b];
    double *row = (double *)malloc(sizeof(double) * (size_t)(L > 0 ? L : 1));
    if (!row) { rc_all = ORACLE_ENOMEM; continue; }
    for (int64_t j = 0; j < L; ++j) row[j] = (double)scores[r * ncap + j];
    int64_t kh = heavy_budget(L, ratio, rounding, k_override, b, n_sink, n_local, NULL);
    int rc = oracle_select_forced(row, L, n_sink, n_local, kh, k_max, idx + r * k_max,
                                  tau ? tau + r : NULL);
    if (rc) rc_all = rc;
    free(row);
  }
  return rc_all;
}

/*
 * Softmax attention of one query head over a given set of positions
 * (scaled dot-product attention restricted to the set).  z_j = scale*(q.k_j),
 * w_j = exp(z_j - max z) / sum exp(z - max z), o = sum_j w_j v_j.
 * With per-position weights omega (Section 4: the sparse backend attends
 * given the index set and associated weights; the formula is not given, and
 * the reading here is that omega_j >= 0 multiplies exp(z_j - max z) in both
 * the numerator and the normaliser): w_j = omega_j exp(z_j - max z) /
 * sum omega exp(z - max z).  absw[i] = sum_j w_j |v_j[i]| (the magnitude of
 * the summed terms, used by the tests to scale floating-point tolerances).
 * An empty set, or weights summing to zero, gives o = 0.
 */
static void attend_head(const problem *p, int b, int h, double scale,
                        const int32_t *set, const float *omega, int64_t k, double *qbuf,
                        double *kbuf, double *z, double *o, double *absw) {
  int G = p->Hq / p->Hkv;
  int g = h / G;
  int d = p->d;
  for (int i = 0; i < d; ++i) { o[i] = 0.0; if (absw) absw[i] = 0.0; }
  if (k == 0) return;
  load_vec(p->q, p->q_dtype, ((int64_t)b * p->Hq + h) * d, d, qbuf);
  double m = -INFINITY;
  for (int64_t t = 0; t < k; ++t) {
    load_vec(p->K->data, p->K->dtype, cache_row_offset(p->K, p->Hkv, d, b, g, set[t]), d, kbuf);
    z[t] = scale * dot(qbuf, kbuf, d);
    if (z[t] > m) m = z[t];
  }
  double Z = 0.0;
  for (int64_t t = 0; t < k; ++t) {
    z[t] = exp(z[t] - m);
    if (omega) z[t] *= (double)omega[t];
    Z += z[t];
  }
  if (!(Z > 0.0)) return;
  for (int64_t t = 0; t < k; ++t) {
    double w = z[t] / Z;
    load_vec(p->V->data, p->V->dtype, cache_row_offset(p->V, p->Hkv, d, b, g, set[t]), d, kbuf);
    for (int i = 0; i < d; ++i) {
      o[i] += w * kbuf[i];
      if (absw) absw[i] += w * fabs(kbuf[i]);
    }
  }
}

/*
 * Attention over caller-given index sets idx[b][row][0..k_max), each row
 * holding its positions followed by -1 padding (rows are query heads, or KV
 * heads in group-shared mode, where each query head of the group uses the
 * group's set).  weights: nullable float [B][R][k_max] aligned with idx (the
 * weighted form above; must be >= 0 and finite).  out and absw are
 * [B][Hq][d] doubles.
 */
static int32_t attend_sets(int B, int Hq, int Hkv, int d, const void *q, int32_t q_dtype,
                           const oracle_cache *K, const oracle_cache *V,
                           const int32_t *seq_lens, int32_t group_shared, double scale,
                           int64_t k_max, const int32_t *idx, const float *weights,
                           double *out, double *absw, int nthreads) {
  problem p = make_problem(B, Hq, Hkv, d, q, q_dtype, K, V, seq_lens, group_shared);
  int rc = check_problem(&p, 1);
  if (rc) return rc;
  if (!idx || !out || k_max < 0) return ORACLE_EINVAL;
  if (!(scale > 0.0)) scale = 1.0 / sqrt((double)d);
  int G = Hq / Hkv;
  int R = group_shared ? Hkv : Hq;
  for (int64_t r = 0; r < (int64_t)B * R; ++r) {
    int b = (int)(r / R);
    for (int64_t t = 0; t < k_max; ++t) {
      int32_t j = idx[r * k_max + t];
      if (j == -1) break;
      if (j < 0 || j >= seq_lens[b]) return ORACLE_EINVAL;
      if (weights) {
        float wv = weights[r * k_max + t];
        if (!(wv >= 0.0f) || isinf(wv)) return ORACLE_EINVAL;
      }
    }
  }
  set_threads(nthreads);
  int failed = 0;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t bh = 0; bh < (int64_t)B * Hq; ++bh) {
    int b = (int)(bh / Hq), h = (int)(bh % Hq);
    int row = group_shared ? h / G : h;
    const int32_t *set = idx + ((int64_t)b * R + row) * k_max;
    const float *omega = weights ? weights + ((int64_t)b * R + row) * k_max : NULL;
    int64_t k = 0;
    while (k < k_max && set[k] != -1) ++k;
    double *buf = (double *)malloc(sizeof(double) * (size_t)(2 * d + (k > 0 ? k : 1)));
    if (!buf) { failed = 1; continue; }
    attend_head(&p, b, h, scale, set, omega, k, buf, buf + d, buf + 2 * d, out + bh * d,
                absw ? absw + bh * d : NULL);
    free(buf);
  }
  return failed ? ORACLE_ENOMEM : ORACLE_OK;
}

int32_t oracle_attend(int B, int Hq, int Hkv, int d, const void *q,
                      int32_t q_dtype, const oracle_cache *K,
                      const oracle_cache *V, const int32_t *seq_lens,
                      int32_t group_shared, double scale, int64_t k_max,
                      const int32_t *idx, double *out, double *absw,
                      int nthreads) {
  return attend_sets(B, Hq, Hkv, d, q, q_dtype, K, V, seq_lens, group_shared, scale, k_max, idx,
                     NULL, out, absw, nthreads);
}

/* The weighted form (Section 4's sparse backend: index sets and weights). */
int32_t oracle_attend_weighted(int B, int Hq, int Hkv, int d, const void *q,
                               int32_t q_dtype, const oracle_cache *K,
                               const oracle_cache *V, const int32_t *seq_lens,
                               int32_t group_shared, double scale, int64_t k_max,
                               const int32_t *idx, const float *weights, double *out,
                               double *absw, int nthreads) {
  if (!weights) return ORACLE_EINVAL;
  return attend_sets(B, Hq, Hkv, d, q, q_dtype, K, V, seq_lens, group_shared, scale, k_max, idx,
                     weights, out, absw, nthreads);
}

/*
 * The whole method for one decode step: score every cached position, keep
 * the exact top-k per row, attend over the kept positions.
 * idx: [B][R][k_max] ascending positions then -1.  tau: [B][R] k-th largest
 * selection score (NaN when k = 0), nullable.  out, absw: [B][Hq][d].
 */
static int32_t sparse_attention_impl(const problem *pp, double ratio, int32_t rounding,
                                     double scale, const int32_t *k_override, int64_t n_sink,
                                     int64_t n_local, int64_t k_max, int32_t *idx, double *tau,
                                     double *out, double *absw, int nthreads) {
  const problem p = *pp;
  int B = p.B, Hq = p.Hq, Hkv = p.Hkv, d = p.d, group_shared = p.group_shared;
  const int32_t *seq_lens = p.seq_lens;
  int rc = check_problem(&p, 1);
  if (rc) return rc;
  if (!idx || !out || !(ratio > 0.0) || n_sink < 0 || n_local < 0) return ORACLE_EINVAL;
  int R = group_shared ? Hkv : Hq;
  for (int b = 0; b < B; ++b) {
    int64_t total;
    heavy_budget(seq_lens[b], ratio, rounding, k_override, b, n_sink, n_local, &total);
    if (total > k_max) return ORACLE_EINVAL;
  }
  set_threads(nthreads);
  int rc_all = ORACLE_OK;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t r = 0; r < (int64_t)B * R; ++r) {
    int b = (int)(r / R), row = (int)(r % R);
    int64_t L = seq_lens[b];
    double *buf = (double *)malloc(sizeof(double) * (size_t)(2 * d + (L > 0 ? L : 1)));
    if (!buf) { rc_all = ORACLE_ENOMEM; continue; }
    row_scores(&p, b, row, buf, buf + d, buf + 2 * d);
    int64_t kh = heavy_budget(L, ratio, rounding, k_override, b, n_sink, n_local, NULL);
    int rc1 = oracle_select_forced(buf + 2 * d, L, n_sink, n_local, kh, k_max, idx + r * k_max,
                                   tau ? tau + r : NULL);
    if (rc1) rc_all = rc1;
    free(buf);
  }
  if (rc_all) return rc_all;
  return oracle_attend(B, Hq, Hkv, d, p.q, p.q_dtype, p.K, p.V, seq_lens, group_shared,
                       scale, k_max, idx, out, absw, nthreads);
}

int32_t oracle_sparse_attention(int B, int Hq, int Hkv, int d, const void *q,
                                int32_t q_dtype, const oracle_cache *K,
                                const oracle_cache *V, const int32_t *seq_lens,
                                double ratio, int32_t rounding,
                                int32_t group_shared, double scale,
                                const int32_t *k_override, int64_t n_sink,
                                int64_t n_local, int64_t k_max,
                                int32_t *idx, double *tau, double *out,
                                double *absw, int nthreads) {
  problem p = make_problem(B, Hq, Hkv, d, q, q_dtype, K, V, seq_lens, group_shared);
  return sparse_attention_impl(&p, ratio, rounding, scale, k_override, n_sink, n_local, k_max,
                               idx, tau, out, absw, nthreads);
}

/*
 * The method with the low-channel indexer in place of exact scores (Table 2:
 * an 8-channel, 16-bit Double Sparsity indexer chooses the positions): the
 * top-k (with any forced positions) runs on the label scores above; the
 * attention over the kept positions uses the full keys and values.
 */
int32_t oracle_label_attention(int B, int Hq, int Hkv, int d, const void *q,
                               int32_t q_dtype, const oracle_cache *K,
                               const oracle_cache *V, const oracle_cache *labels, int nlab,
                               const int32_t *channels, const int32_t *seq_lens,
                               double ratio, int32_t rounding, int32_t group_shared,
                               double scale, const int32_t *k_override, int64_t n_sink,
                               int64_t n_local, int64_t k_max, int32_t *idx, double *tau,
                               double *out, double *absw, int nthreads) {
  problem p = make_problem(B, Hq, Hkv, d, q, q_dtype, K, V, seq_lens, group_shared);
  p.lab = labels;
  p.nlab = nlab;
  p.channels = channels;
  return sparse_attention_impl(&p, ratio, rounding, scale, k_override, n_sink, n_local, k_max,
                               idx, tau, out, absw, nthreads);
}

/* Number of threads OpenMP will use for the next parallel region. */
int32_t oracle_max_threads(int nthreads) { return set_threads(nthreads); }
