/*
 * sparse_decode.h -- C ABI of libsparse_decode.so: exact top-k context-sparse
 * decode attention on AMD Instinct MI355X (gfx950).
 *
 * The method (arXiv 2605.24168, "Inference Time Context Sparsity: Illusion or
 * Opportunity?"):
 *   Section 3, "Algorithms": at each decode step every query head attends only
 *   to the k context positions with the highest attention scores, found by
 *   exact ("oracle") top-k selection over all cached keys.
 *   Table 1 caption: an S-times sparsity means each query head attends to a
 *   1/S fraction of the tokens, i.e. k = N/S.
 *   Section 1 ("Sparsity can be leveraged for system gains") and Section 4:
 *   the sparsity is per query, per query head and per token, including under
 *   grouped-query attention (GQA), and runs on a paged KV cache (page size 16,
 *   NHD layout, in the paper's kernel benchmarks).
 *
 * Conventions shared by every entry point
 *   - Head dimension d = 128.  Query head h reads KV head h / G, G = Hq / Hkv.
 *   - All tensor data, seq_lens, block tables and k_override are DEVICE memory
 *     owned by the caller; descriptors (the structs below) are host memory read
 *     only during the call.  The library never retains or frees caller memory.
 *   - Tensors are dense and row-major (C-contiguous) in the shapes stated.
 *   - Work is enqueued on `stream` (a hipStream_t passed as void*, NULL = the
 *     default stream) and the call returns without synchronising.
 *   - All argument checks happen on the host before anything is enqueued: an
 *     invalid call returns a negative sd_status and has no side effect.
 *     Device-resident values (seq_lens, k_override, block tables, idx) are not
 *     read on the host; kernels clamp seq_lens[b] to [0, capacity].
 *   - Ranking uses the raw score q.k in float32 (exact bfloat16 products,
 *     float32 accumulation); ties go to the lower position.  The softmax scale
 *     enters only the softmax.  Outputs are rounded to the query's dtype
 *     (bfloat16: round to nearest even).
 *   - Inputs holding NaN or infinity give undefined (but memory-safe) results.
 *   - The library keeps one workspace per device; calls that share a device
 *     must be ordered on one stream (or use distinct processes).
 */
#ifndef SPARSE_DECODE_H
#define SPARSE_DECODE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SD_OK = 0,
  SD_ERR_INVALID_ARG = -1,  /* null pointer, bad shape, inconsistent sizes     */
  SD_ERR_UNSUPPORTED = -2,  /* valid request this build does not implement     */
  SD_ERR_WORKSPACE = -3,    /* caller workspace too small, or allocation failed */
  SD_ERR_HIP = -4           /* a HIP runtime call or kernel launch failed       */
} sd_status;

typedef enum { SD_F32 = 0, SD_BF16 = 1, SD_I32 = 2 } sd_dtype;

typedef enum {
  SD_KV_BHND = 0,      /* [B, Hkv, Ncap, d]: one contiguous slab per (sequence, KV head) */
  SD_KV_PAGED_NHD = 1  /* [P, page_size, Hkv, d] page pool + block table                 */
} sd_kv_layout;

/* A dense row-major device tensor. */
typedef struct {
  void *data;         /* device pointer                         */
  int32_t dtype;      /* sd_dtype                               */
  int32_t ndim;       /* number of used entries of shape        */
  int64_t shape[4];
} sd_tensor;

/* A key or value cache.  For SD_KV_PAGED_NHD, position j of sequence b lives
 * in page block_table[b * max_pages_per_seq + j / page_size], slot
 * j % page_size; the capacity of a sequence is max_pages_per_seq * page_size.
 * For SD_KV_BHND the capacity is Ncap = t.shape[2]. */
typedef struct {
  sd_tensor t;
  int32_t layout;                /* sd_kv_layout                                 */
  int32_t page_size;             /* paged: must be 16 and equal t.shape[1]       */
  const int32_t *block_table;    /* paged: device int32 [B, max_pages_per_seq]    */
  int32_t max_pages_per_seq;     /* paged: columns of block_table                 */
} sd_kv;

/* The sparsity rule (Table 1 caption: k = N / S per query head), with
 * optional forced positions: the scaffolding of the paper's long-context runs
 * keeps the first and last positions of each sequence besides the exact
 * top-k (Sink(128) + Local(128) + OracleTopK in the SWE-Bench appendix; 64
 * sinks in the extreme top-K sweep of Section 3).  With n_sink or n_local
 * set, a row keeps positions [0, ns), the exact top-k_b of [ns, L_b - nl)
 * (k_b capped by that range) and [L_b - nl, L_b), where ns = min(n_sink, L_b)
 * and nl = min(n_local, L_b - ns); its list holds ns + k_b + nl entries, all
 * ascending.  Positions that do not fit the list (k_override with a short
 * idx) are dropped, local ones first. */
typedef struct {
  double ratio;          /* S > 0.  k_b = clamp(R(L_b / S), 1, L_b) for L_b > 0, 0 for L_b = 0 */
  int32_t k_rounding;    /* R: 0 = nearest with halves up, 1 = ceiling                          */
  int32_t group_shared;  /* 0: one index set per query head (rows R = Hq);                       */
                         /* 1: one per KV head, chosen on the sum over the group's query heads   */
                         /*    of their raw scores; each head then softmaxes its own scores over */
                         /*    that set (rows R = Hkv)                                            */
  float softmax_scale;   /* > 0, or <= 0 for 1/sqrt(d)                                          */
  const int32_t *k_override; /* optional device int32 [B]: k_b = clamp(k_override[b], 0,
                                min(L_b, idx capacity)) instead of the ratio rule; NULL = unused */
  int32_t n_sink;        /* >= 0: first positions of every sequence always kept (0 = none)     */
  int32_t n_local;       /* >= 0: last positions of every sequence always kept (0 = none)      */
} sd_sparsity;

/* Label cache of the low-channel approximate indexer (Table 2 and Section 4:
 * a Double Sparsity indexer on 8 channels of 16 bits, untuned): for every
 * cached key, 8 of its d channels: [B, Hkv, Ncap, 8] beside a BHND cache;
 * [P, Hkv, 16, 8] beside a paged one (the key pool's P pages, read through
 * K's block table; head-major inside a page, so a KV head's 16 label rows
 * of a page are one contiguous 256-byte run).  Column c
 * of KV head g holds key channel channels[g * 8 + c]; the approximate score
 * of a key for query head h is sum_c q_h[channels[g * 8 + c]] * label[c]. */
typedef struct {
  sd_tensor t;                 /* bfloat16 label cache, device memory          */
  const int32_t *channels;     /* device int32 [Hkv, 8], values in [0, 128)    */
} sd_labels;

/* Stage timings of the last sparse_decode_attention call (profiling on). */
typedef struct {
  float pilot_ms;      /* threshold estimation from a strided sample of keys      */
  float score_ms;      /* full scoring stream + candidate filter                  */
  float select_ms;     /* exact top-k over the candidates                         */
  float repair_ms;     /* exact fallback for rows whose candidates were not enough */
  float attend_ms;     /* gather of the selected value rows + softmax + merge     */
  float total_ms;
  int32_t repaired_rows; /* rows that took the exact fallback                     */
  int32_t valid;         /* 1 if the fields above are filled                      */
} sd_profile;

/*
 * Scores of every cached position: scores[b, r, j] = q_h . K[b, g(h), j] for
 * row r = h (per-head mode) or, with sparsity->group_shared, the sum over the
 * group's query heads of those dot products (row r = g).  Positions
 * j >= L_b get -infinity.  (Section 3: exact scores feed the oracle top-k.)
 *   q       [B, Hq, 128], dtype of K
 *   K       key cache, bf16 or f32
 *   seq_lens device int32 [B]
 *   sparsity only group_shared is read
 *   scores  f32 [B, R, C], C = the cache capacity
 */
sd_status sparse_decode_score(const sd_tensor *q, const sd_kv *K, const int32_t *seq_lens,
                              const sd_sparsity *sparsity, sd_tensor *scores, void *stream);

/*
 * Exact top-k of each score row (Section 3, exact oracle top-k): for row
 * (b, r) the k_b positions j < L_b that come first under (score descending,
 * position ascending), written in ascending position order, then -1.  With
 * forced positions (sd_sparsity), the top-k runs over the positions between
 * them and the list holds sinks, top-k, local window.
 *   scores f32 [B, R, C] (e.g. from sparse_decode_score)
 *   idx    i32 [B, R, k_max], k_max >= the budget of a full sequence of C
 *   vals   f32 [B, R, k_max] or NULL: the score of each listed position,
 *          -infinity in the padding
 */
sd_status sparse_decode_topk(const sd_tensor *scores, const int32_t *seq_lens,
                             const sd_sparsity *sparsity, sd_tensor *idx, sd_tensor *vals,
                             void *stream);

/*
 * Softmax attention restricted to given positions: for query head h with
 * row r (r = h, or h / G with group_shared), over the entries j of
 * idx[b, r, :] with 0 <= j < L_b (others, e.g. the -1 padding, are skipped):
 * z_j = scale * q_h . K_j, out[b, h] = sum_j softmax(z)_j V_j.  A row with no
 * usable entry gives zeros.  (Table 1 / Section 4 describe the paper's sparse
 * backend as this computation given the index set.)
 *   out [B, Hq, 128], dtype of q
 */
sd_status sparse_decode_attend(const sd_tensor *q, const sd_kv *K, const sd_kv *V,
                               const int32_t *seq_lens, const sd_tensor *idx,
                               const sd_sparsity *sparsity, sd_tensor *out, void *stream);

/*
 * Weighted attention restricted to given positions (Section 4: the paper's
 * sparse backend attends a given sparse index list together with a weight
 * per index).  As sparse_decode_attend, with entry t of row (b, r) carrying
 * the weight omega = weights[b, r, t]: out[b, h] = sum_j w_j V_j with
 * w_j = omega_j exp(z_j - m) / sum over the row's usable entries of
 * omega exp(z - m), i.e. softmax attention with log(omega) added to each
 * logit.  Weights must be finite and >= 0 (others give undefined, memory-safe
 * results); an entry of weight 0 is skipped, and a row whose usable weights
 * are all 0 gives zeros.  All ones reproduce sparse_decode_attend.
 *   weights f32 [B, R, k_max], the shape of idx
 *   out     [B, Hq, 128], dtype of q
 */
sd_status sparse_decode_attend_weighted(const sd_tensor *q, const sd_kv *K, const sd_kv *V,
                                        const int32_t *seq_lens, const sd_tensor *idx,
                                        const sd_tensor *weights, const sd_sparsity *sparsity,
                                        sd_tensor *out, void *stream);

/*
 * Dense decode attention over every cached position: out[b, h] =
 * sum_{j < L_b} softmax(z)_j V_j with z_j = scale * q_h . K_j, the
 * full-attention baseline that Table 1 measures the sparse backend against
 * (it reads all of K and V).  A sequence with L_b = 0 gives zeros.
 *   q [B, Hq, 128] bfloat16; K, V bfloat16 caches of one layout
 *   (float32, or more than 8 query heads per KV head, returns
 *   SD_ERR_UNSUPPORTED)
 *   softmax_scale > 0, or <= 0 for 1/sqrt(128)
 *   out [B, Hq, 128] bfloat16
 * Uses the library workspace: sparse_decode_dense_workspace_size bytes.
 */
sd_status sparse_decode_dense_attention(const sd_tensor *q, const sd_kv *K, const sd_kv *V,
                                        const int32_t *seq_lens, float softmax_scale,
                                        sd_tensor *out, void *stream);
sd_status sparse_decode_dense_workspace_size(const sd_tensor *q, const sd_kv *K, size_t *bytes);

/*
 * The whole decode-step method fused: score every cached key, keep the exact
 * top-k per row, attend over the kept rows.  Results equal
 * sparse_decode_score -> sparse_decode_topk -> sparse_decode_attend, except
 * that the softmax reuses the selection's float32 scores instead of
 * recomputing them.  idx receives the kept positions as in sparse_decode_topk.
 *   q [B, Hq, 128]; K, V caches of q's dtype and the same layout;
 *   out [B, Hq, 128]; idx i32 [B, R, k_max]
 */
sd_status sparse_decode_attention(const sd_tensor *q, const sd_kv *K, const sd_kv *V,
                                  const int32_t *seq_lens, const sd_sparsity *sparsity,
                                  sd_tensor *out, sd_tensor *idx, void *stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops that must not allocate, harnesses that forbid
 * hipMalloc): sparse_decode_attention with the same arguments and results,
 * but its scratch is a static device array of SD_NOALLOC_SCRATCH_BYTES
 * inside the library (one per GPU, held until the process ends) instead of
 * the library workspace, and it calls no hipMalloc, hipFree or other
 * allocating routine.  A problem whose scratch (sparse_decode_workspace_size
 * for the same shapes, at most) exceeds it returns SD_ERR_WORKSPACE before
 * any launch.  Every call on one GPU shares that GPU's array: calls that
 * overlap on one GPU (different streams without ordering) race and must
 * not be issued.  Profiling does not apply to it.
 */
#define SD_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
sd_status sparse_decode_attention_noalloc(const sd_tensor *q, const sd_kv *K, const sd_kv *V,
                                          const int32_t *seq_lens, const sd_sparsity *sparsity,
                                          sd_tensor *out, sd_tensor *idx, void *stream);

/*
 * The method with the low-channel indexer choosing the positions (Table 2):
 * as sparse_decode_attention, but the exact top-k (with any forced
 * positions) runs on the approximate label scores, one 16-byte label row per
 * key instead of a 256-byte key row; the attention over the kept positions
 * then uses the full keys and values.  bfloat16 only.  Uses the same
 * workspace as sparse_decode_attention.
 */
sd_status sparse_decode_label_attention(const sd_tensor *q, const sd_kv *K, const sd_kv *V,
                                        const sd_labels *labels, const int32_t *seq_lens,
                                        const sd_sparsity *sparsity, sd_tensor *out,
                                        sd_tensor *idx, void *stream);

/* Approximate label scores of every cached position, laid out as
 * sparse_decode_score's (-infinity beyond each sequence).  K supplies the
 * layout, capacity and block table only. */
sd_status sparse_decode_label_score(const sd_tensor *q, const sd_kv *K, const sd_labels *labels,
                                    const int32_t *seq_lens, const sd_sparsity *sparsity,
                                    sd_tensor *scores, void *stream);

/* Stochastic index selection with importance weights (the vAttention runs
 * of Section 4; the paper does not define the method, and this is the
 * standard importance-weighted reading): per query head (row), the exact
 * top-k set S of sparse_decode_attention (with any forced positions), plus
 * s positions drawn uniformly with replacement from the rest
 * C = [0, L_b) \ S, each drawn entry weighted |C| / s; out is the weighted
 * softmax attention over S and the draws (as sparse_decode_attend_weighted).
 *   draws    int32 [B, R, s]: the random numbers, one per draw, read as
 *            uint32 bits u; draw i picks the floor(u |C| / 2^32)-th position
 *            of C in ascending order.
 *   idx      int32 [B, R, k_max + s], written: S ascending, then the s drawn
 *            positions, then -1; k_max >= the k of a full-capacity sequence
 *            (plus the forced positions), as for sparse_decode_attention.
 *   weights  float32 [B, R, k_max + s], written: 1 for S, |C| / s for a
 *            draw, 0 for padding.  A row with |C| = 0 draws nothing.
 * Per-head rows only (group_shared returns SD_ERR_UNSUPPORTED).  Uses the
 * same workspace as sparse_decode_attention for this idx. */
sd_status sparse_decode_sampled_attention(const sd_tensor *q, const sd_kv *K, const sd_kv *V,
                                          const int32_t *seq_lens, const sd_sparsity *sparsity,
                                          const sd_tensor *draws, sd_tensor *out, sd_tensor *idx,
                                          sd_tensor *weights, void *stream);

/* Bytes of device workspace sparse_decode_attention,
 * sparse_decode_label_attention and sparse_decode_attend need for these
 * shapes (idx gives k_max): the largest of their layouts. */
sd_status sparse_decode_workspace_size(const sd_tensor *q, const sd_kv *K,
                                       const sd_sparsity *sparsity, const sd_tensor *idx,
                                       size_t *bytes);

/* Use caller-owned device memory (256-byte aligned) as the workspace of the
 * current device.  NULL releases it; the library then allocates its own on
 * demand (hipMalloc) and keeps it until the process ends or a larger one is
 * needed.  Nothing is kept in the workspace between calls. */
sd_status sparse_decode_set_workspace(void *dev_ptr, size_t bytes);

/* Entries of the index list of a sequence of L positions under the ratio
 * rule of `sparsity`: k, plus the forced positions when n_sink or n_local
 * is set.  -1 for an invalid rule. */
int64_t sparse_decode_budget(int64_t L, const sd_sparsity *sparsity);

/* Profiling: while enabled, sparse_decode_attention records HIP events
 * between its stages on the call's stream (a ring of 64 calls per device;
 * enabling again starts a new series).  enable = 1 records every stage;
 * enable = 2 times only the scoring kernel, with events attached to its own
 * dispatch (the profile then holds score_ms alone; nothing is added to the
 * stream between kernels).  sparse_decode_last_profile waits for
 * the most recent call's events and fills `out`; sparse_decode_profile_mean
 * averages the stage times of the series' last min(n, 64) calls and stores
 * that count in *n_calls (repaired_rows is the last call's). */
sd_status sparse_decode_set_profiling(int32_t enable);
sd_status sparse_decode_last_profile(sd_profile *out);
sd_status sparse_decode_profile_mean(sd_profile *out, int32_t *n_calls);

/* Debug switch (used by tests to exercise paths): with flags & 1 every row of
 * sparse_decode_attention takes the exact fallback path; flags & 4 / & 8
 * turn the group-deduplicated attention off / on wherever it applies
 * (per-head rows with recomputed logits, bf16, 2 or more heads per group),
 * overriding the cost rule; flags & 16 / & 32 turn the candidate selection
 * over several workgroups per row off / on wherever it applies (calls with
 * fewer than 256 rows, no group-deduplicated attention), overriding its
 * cost rule (rows expecting 8K candidates or more).  0 restores normal. */
sd_status sparse_decode_set_debug(int32_t flags);

/* Measurement helper, not a step of the method: one streaming read of
 * `bytes` bytes of device memory at `buf` (16-byte aligned, bytes a nonzero
 * multiple of 16), enqueued on `stream`.  Every byte is read once: one
 * contiguous 256 KB span per workgroup, nontemporal 16-byte loads, eight in
 * flight per lane; nothing is written except, with
 * negligible probability, *sink (one caller-owned device uint32).  Timed by
 * the caller, it gives this device's plain streaming-read rate, the
 * reference for the bandwidth-bound kernels.  SD_ERR_INVALID_ARG for a null,
 * misaligned or empty buffer (checked before any HIP call). */
sd_status sparse_decode_read_probe(const void *buf, size_t bytes, uint32_t *sink, void *stream);

const char *sparse_decode_status_string(sd_status status);

#ifdef __cplusplus
}
#endif

#endif /* SPARSE_DECODE_H */
