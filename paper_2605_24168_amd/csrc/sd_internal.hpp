// sd_internal.hpp -- device-side building blocks of libsparse_decode.so
// (exact top-k context-sparse decode attention on gfx950).
//
// Everything here is written for CDNA4: 64-lane wavefronts, the
// v_mfma_f32_16x16x32_bf16 matrix instruction, LDS, and 16-byte vector loads.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace sd {

constexpr int kHeadDim = 128;
constexpr int kTile = 16;          // keys per scoring tile (= KV page size)
constexpr int kBlock = 256;        // threads per workgroup of every kernel
constexpr int kWaves = kBlock / 64;
constexpr int kMaxGroup = 16;      // query heads per KV head handled by one MFMA tile
constexpr int kWaveKeysMax = 2048; // keys one scoring wave streams (at most)
constexpr int kLabelWaveKeysMax = 8192;  // the same over label rows (16 bytes per key)
constexpr int kCandBuf = 1024;     // candidates one scoring wave holds, over all its rows
constexpr int kChunkCap = kWaves * kCandBuf;  // entries of one workgroup's packed block
constexpr int kDenseChunk = 8192;  // keys per workgroup of the full-score kernels
constexpr int kSampleMax = 2048;   // pilot samples per row
constexpr int kPartStride = kHeadDim + 2;  // (m, l, o[128]) per split partial
constexpr int kDselPartsMax = 64;  // pieces of a row in the multi-workgroup fallback selection
constexpr int kRepairParts = 16;   // work items per (sequence, KV head) of the fallback scoring
constexpr int kPselPartsMax = 32;  // pieces of a row in the multi-workgroup candidate selection
constexpr int kPselChunksMax = 64; // chunks per piece (at most)
constexpr int kPselSlots = 4;      // candidates per thread a piece holds (1024 threads)
constexpr int kPselItemsMax = 1024 * kPselSlots;  // candidates of a piece, at most
constexpr int kPselRunMax = 4096;  // keys of the k-th run of 32 buckets a piece collects
constexpr int kPselStride = 128;   // u32 per piece record (see Work::psel_rec)
constexpr int kSelectWideRows = 256; // fewer rows: 1024-thread selection workgroups
constexpr size_t kSelectShareLds = 70 * 1024;  // more dynamic LDS: one workgroup per CU
constexpr int kDenseWaveKeysMax = 8192; // keys per work item of the dense decode kernel
constexpr int kDenseMaxGroup = 8;     // query heads per KV head of the dense decode kernel
constexpr int kLabels = 8;            // label channels per key of the low-channel indexer
constexpr int kOutboxCap = 16384;     // candidates a persistent stream workgroup holds in LDS
constexpr int kOutboxBlocks = 64;     // blocks it holds at once

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// ---------------------------------------------------------------------------
// Problem description passed by value to every kernel.
// ---------------------------------------------------------------------------
struct KvView {
  const void *base;
  const int32_t *block_table;  // paged only: [B, max_pages]
  int64_t ncap;                // positions addressable per sequence
  int32_t paged;
  int32_t hkv;
  int32_t max_pages;
};

struct Params {
  const void *q;               // [B, Hq, 128]
  KvView K, V;
  const int32_t *seq_lens;     // [B]
  const int32_t *k_override;   // [B] or null
  double ratio;
  float scale;
  int32_t B, Hq, Hkv, G, R;
  int32_t bf16;
  int32_t group_shared;
  int32_t rounding;
  int32_t k_max;
  int64_t ncap;
  const float *weights;        // [B, R, k_max] per-entry weights of the index
                               // lists (weighted attention), or null
  int32_t n_sink, n_local;     // forced first / last positions of each sequence
  // Low-channel indexer: when labels is set, selection scores come from a
  // label cache of kLabels bf16 channels per key (layout: label_offset),
  // read through K's block table when paged; column c of KV head g is key
  // channel channels[g * kLabels + c].
  const uint16_t *labels;
  const int32_t *channels;     // [Hkv][kLabels]
  // Row stride of the index list the selection writes, when it is longer
  // than k_max (the sampled selection appends its draws); 0: k_max.
  int32_t idx_stride;
};

// Scratch carved from the library workspace (see the host orchestration).
struct Work {
  float *sample;     // [rows][kSampleMax] pilot sample scores
  float *theta;      // [rows] candidate threshold
  float *smax;       // [rows] largest pilot sample score
  int2 *dir;         // [rows][nchunk] (start, count) of the row's candidates in
                     // its chunk's block; count -1 = a staging area overflowed
  uint32_t *ckey;    // [B*Hkv][nchunk][blk_cap] order-preserving score keys
  uint16_t *cpos;    // [B*Hkv][nchunk][blk_cap] positions within the chunk
  int32_t *flags;    // [rows] 1 = the row needs the exact fallback
  float *dense;      // [rows][ncap] fallback scores
  float *sigma;      // [rows][k_max] softmax weights exp(scale*(s - max s)) of the
                     // kept entries, aligned with idx (per-head rows whose attention
                     // does not recompute its logits; otherwise unused)
  float *part;       // [B*Hq][nsplit][kPartStride] attend partials
  int32_t *stats;    // [4]: [0] rows repaired in the last call
  int32_t nchunk;      // chunks per sequence (of chunk_keys keys)
  int32_t wave_keys;   // keys per scoring wave: 256, 512, 1024 or 2048
  int32_t chunk_keys;  // keys per chunk: kWaves * wave_keys, or wave_keys when
                       // each wave of a workgroup scores its own KV head
  int32_t blk_cap;     // entries per packed block: kChunkCap, or kCandBuf
  int32_t nsplit;
  int32_t force_repair;  // every row takes the exact fallback
  // Group-deduplicated attention (per-head rows whose logits are recomputed,
  // GQA): ustart[row * ustride + c] is the first entry of the row's list at
  // or past position c * union_chunk (c = 0 .. ceil(L / union_chunk); the
  // selection writes it after the list); the attention then takes, chunk by
  // chunk, the positions any head of a group keeps and reads each kept key
  // and value row once for the whole group.  Null / 0: per-row lists.
  int32_t *ustart;
  int32_t ustride;
  int32_t union_chunk;
  // Exact fallback selection over several workgroups per row (calls whose
  // every row takes the fallback): dsel_parts pieces per row, 0 = each
  // row's selection runs in one workgroup of k_select.
  uint32_t *dsel_hist;  // [rows][2048] key-digit histograms (cleared by the repair)
  int32_t *dsel_state;  // [rows][4]: key prefix, its mask, rank still to place
  int2 *dsel_cnt;       // [rows][kDselPartsMax] (keys above, keys equal to) the threshold
  int32_t dsel_parts;
  // Candidate selection over several workgroups per row (rows too few to
  // fill the GPU one workgroup each): psel_parts pieces of consecutive
  // chunks per row, 0 = one workgroup per row.  Record of piece j of a row:
  // psel_rec[(row * psel_parts + j) * kPselStride + ...]: [0, 64) its
  // candidates per run of 32 value buckets, [64] its candidate count, [65]
  // its largest key.
  uint32_t *psel_rec;
  int32_t psel_parts;
  // Persistent scoring stream: one workgroup per compute unit takes units
  // (chunks) from a queue; k_pilot_select writes the work list and resets
  // the queue.  unit_pre[b] = units of the sequences before b (B + 1
  // entries); unit_heads = units per chunk of a sequence (Hkv, or Hkv / 4
  // when each wave of a workgroup scores its own KV head).
  int32_t persistent;
  int32_t stream_wgs;   // workgroups of the persistent launch (compute units)
  int32_t unit_heads;
  int32_t *queue;
  int32_t *unit_pre;
  // Sequences by descending length (ties: lower index first), written by
  // k_pilot_select; the selection and the attention take their rows in
  // that order, so that the longest rows start first.  Null: batch order.
  int32_t *seq_order;
};

// Row of workgroup i of a launch over rows (rows_per_b rows per sequence) in
// the order of w.seq_order (the identity when it is null).
__device__ __forceinline__ int ordered_row(const Work &w, int i, int rows_per_b) {
  return w.seq_order ? w.seq_order[i / rows_per_b] * rows_per_b + i % rows_per_b : i;
}

// Scratch of the dense decode kernels.
struct DenseWork {
  float *part;         // [B*Hq][nsplit][kPartStride] key-range partials
  int32_t wave_keys;   // keys per work item (a multiple of kTile)
  int32_t nsplit;      // key ranges per sequence: ceil(ncap / wave_keys)
};

// ---------------------------------------------------------------------------
// Small helpers.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }
__device__ __forceinline__ int wave_id() { return threadIdx.x >> 6; }

// Pilot threshold rank (see the pilot kernel): of m samples of n
// positions, for a top-k of k, the smallest r with r - z sqrt(r) >= e,
// e = k m / n, capped at ceil(2.5 e) (and at m).  z: the margin in
// standard deviations of the count above the r-th sample.
constexpr double kPilotZ = 4.3;
__host__ __device__ inline int64_t pilot_rank(int64_t k, int64_t m, int64_t n) {
  const int64_t rr = (5 * k * m + 2 * n - 1) / (2 * n);
  const double e = (double)k * m / n;
  const double sq = 0.5 * (kPilotZ + sqrt(kPilotZ * kPilotZ + 4.0 * e));
  const int64_t rz = (int64_t)ceil(sq * sq);
  const int64_t r = rz < rr ? rz : rr;
  return r < m ? r : m;
}

// k for a sequence of L positions (Table 1 caption: 1/S of the tokens).
__host__ __device__ inline int64_t budget_rule(int64_t L, double ratio, int rounding) {
  if (L <= 0) return 0;
  double x = (double)L / ratio;
  double k = rounding == 1 ? ceil(x) : floor(x + 0.5);
  if (k < 1.0) k = 1.0;
  if (k > (double)L) k = (double)L;
  return (int64_t)k;
}

__device__ __forceinline__ int seq_len(const Params &p, int b) {
  int64_t L = p.seq_lens[b];
  if (L < 0) L = 0;
  if (L > p.ncap) L = p.ncap;
  return (int)L;
}

// What a row keeps.  The first ns and last nl positions of the sequence
// are forced (the sink and local windows of the paper's long-context
// scaffolding, kept besides the exact top-k); the exact top-kh runs over the
// positions in between, [lo, hi).  kh is the ratio (or override) rule on the
// whole sequence, capped by the middle and by the index list's length.  The
// list holds the sinks, then the top-kh ascending, then the local window:
// total entries, all ascending.  With nothing forced, lo = 0, hi = L and kh
// is the plain budget.
struct RowPlan {
  int ns, nl, lo, hi, kh, total;
};

__host__ __device__ inline RowPlan row_plan(int L, int n_sink, int n_local, int64_t rule,
                                            int k_max) {
  RowPlan r;
  r.ns = n_sink < L ? n_sink : L;
  r.ns = r.ns < k_max ? r.ns : k_max;
  r.nl = n_local < L - r.ns ? n_local : L - r.ns;
  r.nl = r.nl < k_max - r.ns ? r.nl : k_max - r.ns;
  r.lo = r.ns;
  r.hi = L - r.nl;
  int64_t k = rule;
  if (k > r.hi - r.lo) k = r.hi - r.lo;
  if (k > k_max - r.ns - r.nl) k = k_max - r.ns - r.nl;
  r.kh = (int)(k > 0 ? k : 0);
  r.total = r.ns + r.kh + r.nl;
  return r;
}

__device__ __forceinline__ RowPlan row_plan(const Params &p, int b, int L) {
  int64_t k;
  if (p.k_override) {
    k = p.k_override[b];
    if (k < 0) k = 0;
    if (k > L) k = L;
  } else {
    k = budget_rule(L, p.ratio, p.rounding);
  }
  return row_plan(L, p.n_sink, p.n_local, k, p.k_max);
}

// Element offset of channel 0 of (sequence b, KV head g, position j).
__device__ __forceinline__ int64_t kv_offset(const KvView &kv, int b, int g, int64_t j) {
  if (!kv.paged) return (((int64_t)b * kv.hkv + g) * kv.ncap + j) * kHeadDim;
  int64_t page = kv.block_table[(int64_t)b * kv.max_pages + (j >> 4)];
  return ((page * kTile + (j & 15)) * kv.hkv + g) * kHeadDim;
}

// Element offset of label row (sequence b, KV head g, position j).  Beside
// a contiguous cache: [B][Hkv][Ncap][kLabels].  Beside a paged cache:
// [pages][Hkv][16][kLabels] through K's block table -- head-major inside a
// page, so a KV head's 16 label rows of a page are one 256-byte run.
__device__ __forceinline__ int64_t label_offset(const KvView &kv, int b, int g, int64_t j) {
  if (!kv.paged) return (((int64_t)b * kv.hkv + g) * kv.ncap + j) * kLabels;
  int64_t page = kv.block_table[(int64_t)b * kv.max_pages + (j >> 4)];
  return ((page * kv.hkv + g) * kTile + (j & 15)) * kLabels;
}

// Order-preserving 32-bit key of a float: larger float <=> larger key.
// -0 is folded onto +0 so that equal floats give equal keys.
__device__ __forceinline__ uint32_t f2key(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u << 1) == 0) u = 0;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float key2f(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) {
  return __uint_as_float(bits16 << 16);
}

// ---------------------------------------------------------------------------
// Scoring tile: 16 keys x up to 16 query heads of one KV group.
//
// MFMA 16x16x32 bf16 layout (gfx950): operand A row i / operand B column j
// come from lanes with (lane & 15) == i / j, and lane group s = lane >> 4
// supplies elements 8s..8s+7 of the 32-long contraction slice.  The result
// lane l holds C[4*(l>>4) + r][l & 15], r = 0..3.  A = the group's queries
// (rows = heads), B = the key tile (columns = keys); the four MFMAs of one
// tile walk d in slices of 32 channels, so lane group s reads channels
// 32*kk + 8s .. +7 of its key: per instruction the wave touches 16 keys x
// 64 contiguous bytes, and the tile's 4 KB exactly once.
// After the tile, lane l holds the scores of heads 4*(l>>4)+r for key l&15.
// ---------------------------------------------------------------------------
struct QFrag {
  u32x4 v[4];
};

// Query operand of nh (<= 16) consecutive query heads from `first`; rows
// beyond nh are zero.
__device__ __forceinline__ void load_q_heads(const Params &p, int b, int first, int nh,
                                             QFrag &qf) {
  const int l = lane_id();
  const int h = l & 15, s = l >> 4;
  if (h < nh) {
    const uint16_t *qp = (const uint16_t *)p.q + ((int64_t)b * p.Hq + first + h) * kHeadDim + 8 * s;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) qf.v[kk] = *(const u32x4 *)(qp + 32 * kk);
  } else {
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) qf.v[kk] = u32x4{0u, 0u, 0u, 0u};
  }
}

// The G query heads of KV head g.
__device__ __forceinline__ void load_q_bf16(const Params &p, int b, int g, QFrag &qf) {
  load_q_heads(p, b, g * p.G, p.G, qf);
}

struct KFrag {
  u32x4 v[4];
};

// Load this lane's slices of key row `off` (element offset of channel 0).
__device__ __forceinline__ void load_k_bf16(const KvView &K, int64_t off, KFrag &kf) {
  const uint16_t *kp = (const uint16_t *)K.base + off + 8 * (lane_id() >> 4);
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) kf.v[kk] = __builtin_nontemporal_load((const u32x4 *)(kp + 32 * kk));
}

// ---------------------------------------------------------------------------
// Coalesced tile loads.  Loading a tile straight into the MFMA layout makes
// every instruction touch 16 rows x 64 bytes; loading it with four fully
// coalesced 1 KB instructions (one 256-byte key row per 16-lane group) and
// re-reading it from LDS in the MFMA layout streams measurably faster.
// Instruction t (0..3), lane l = 16a + lo loads 16-byte chunk
// c = (lo - 4t - a) mod 16 of tile row 4t + a and stores it to LDS slot
// 64t + l, so the LDS writes are contiguous, and the MFMA read of chunk c of
// row 4t + a (slot 64t + 16a + ((4t + a + c) mod 16)) has each 16-lane group
// spread over all LDS banks.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int swz_chunk(int t) {
  const int l = lane_id();
  return ((l & 15) - 4 * t - (l >> 4)) & 15;
}

// row_ptr(r) is the address of tile row r (0..15) as a byte pointer.
template <class RowPtr>
__device__ __forceinline__ void load_tile_coalesced(RowPtr row_ptr, u32x4 v[4]) {
  const int a = lane_id() >> 4;
#pragma unroll
  for (int t = 0; t < 4; ++t)
    v[t] = __builtin_nontemporal_load((const u32x4 *)(row_ptr(4 * t + a) + 16 * swz_chunk(t)));
}

__device__ __forceinline__ void stage_tile(u32x4 *wl, const u32x4 v[4]) {
#pragma unroll
  for (int t = 0; t < 4; ++t) wl[64 * t + lane_id()] = v[t];
}

__device__ __forceinline__ void read_kfrag(const u32x4 *wl, KFrag &kf) {
  const int L = lane_id(), r = L & 15, s = L >> 4, t = r >> 2, a = r & 3;
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) kf.v[kk] = wl[64 * t + 16 * a + ((4 * t + a + 4 * kk + s) & 15)];
}

__device__ __forceinline__ f32x4 mfma_scores(const QFrag &qf, const KFrag &kf) {
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kk = 0; kk < 4; ++kk)
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, qf.v[kk]),
                                                  __builtin_bit_cast(bf16x8, kf.v[kk]), acc, 0,
                                                  0, 0);
  return acc;
}

// ---------------------------------------------------------------------------
// Label scores (the low-channel indexer).  A key's label row is kLabels
// bf16 channels, 16 bytes.  Every path computes a key's approximate score
// the same way, so the stream, the fallback and the stand-alone scores agree
// bit for bit.  Per-head rows: the query's label channels are bf16 values
// too, so the score is four packed bf16 dot products (v_dot2c_f32_bf16:
// two channel products added to a float32 accumulator, channel pairs in
// order) straight from the label row's 32-bit words.  Group-shared rows:
// the query side is first summed over the group's heads (in head order, in
// float32), then a fused multiply-add chain over the channels in order
// (products of bf16 values are exact in float32).
// ---------------------------------------------------------------------------
typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2;

__device__ __forceinline__ u32x4 load_labels(const uint16_t *base, int64_t off) {
  return __builtin_nontemporal_load((const u32x4 *)(base + off));
}

__device__ __forceinline__ void unpack_labels(u32x4 raw, float lab[kLabels]) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    lab[2 * e] = bf16_to_f32(raw[e] & 0xFFFFu);
    lab[2 * e + 1] = __uint_as_float(raw[e] & 0xFFFF0000u);
  }
}

__device__ __forceinline__ float label_dot(const float *ql, const float lab[kLabels]) {
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kLabels; ++c) s = fmaf(ql[c], lab[c], s);
  return s;
}

// Per-head rows: qp[e] holds the query's label channels 2e and 2e+1 as a
// bf16 pair (channel 2e in the low half, as in the label row).
// (Each word is copied to a scalar before the bit cast: a bit cast of a
// vector element subscript compiled here to a read of element 0 only.)
__device__ __forceinline__ float label_dot_packed(const uint32_t qp[4], u32x4 raw) {
  float s = 0.f;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const uint32_t qw = qp[e], lw = raw[e];
    s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, qw),
                                        __builtin_bit_cast(bf16x2, lw), s, false);
  }
  return s;
}

// The query side of row (b, KV head g, head index h within the group): q's
// label channels (channel indices clamped, so bad ones stay memory-safe),
// or in group-shared mode (h < 0) their sum over the group's heads.
__device__ __forceinline__ void q_label_row(const Params &p, int b, int g, int h,
                                            float ql[kLabels]) {
  const int32_t *ch = p.channels + (int64_t)g * kLabels;
  const int h0 = h < 0 ? 0 : h, h1 = h < 0 ? p.G : h + 1;
#pragma unroll
  for (int c = 0; c < kLabels; ++c) {
    int cc = ch[c];
    cc = cc < 0 ? 0 : (cc >= kHeadDim ? kHeadDim - 1 : cc);
    float v = 0.f;
    for (int t = h0; t < h1; ++t)
      v += bf16_to_f32(((const uint16_t *)p.q)[((int64_t)b * p.Hq + (int64_t)g * p.G + t) *
                                                  kHeadDim + cc]);
    ql[c] = v;
  }
}

// The same for a per-head row (h >= 0) as bf16 pairs (label_dot_packed).
__device__ __forceinline__ void q_label_row_packed(const Params &p, int b, int g, int h,
                                                   uint32_t qp[4]) {
  const int32_t *ch = p.channels + (int64_t)g * kLabels;
  const uint16_t *qh = (const uint16_t *)p.q + ((int64_t)b * p.Hq + (int64_t)g * p.G + h) * kHeadDim;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    int c0 = ch[2 * e], c1 = ch[2 * e + 1];
    c0 = c0 < 0 ? 0 : (c0 >= kHeadDim ? kHeadDim - 1 : c0);
    c1 = c1 < 0 ? 0 : (c1 >= kHeadDim ? kHeadDim - 1 : c1);
    qp[e] = (uint32_t)qh[c0] | ((uint32_t)qh[c1] << 16);
  }
}

// Label scores in the MFMA result layout (for the pilot and the full-score
// paths): lane (s, col) holds rows 4s+r of its key col.  Rows beyond G are
// zero; in group-shared mode row 0 of lane group 0 holds the group's score
// and every other row is zero, so group_sum returns it unchanged.
struct LabelRows {
  float ql[4][kLabels];  // group-shared rows
  uint32_t qp[4][4];     // per-head rows (label_dot_packed); zero beyond G
  int packed;
  __device__ __forceinline__ void init(const Params &p, int b, int g) {
    const int s = lane_id() >> 4;
    packed = !p.group_shared;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int h = 4 * s + r;
#pragma unroll
      for (int e = 0; e < 4; ++e) qp[r][e] = 0u;
#pragma unroll
      for (int c = 0; c < kLabels; ++c) ql[r][c] = 0.f;
      if (p.group_shared) {
        if (s == 0 && r == 0) q_label_row(p, b, g, -1, ql[r]);
      } else if (h < p.G) {
        q_label_row_packed(p, b, g, h, qp[r]);
      }
    }
  }
  __device__ __forceinline__ f32x4 score(u32x4 raw) const {
    f32x4 acc;
    if (packed) {
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[r] = label_dot_packed(qp[r], raw);
    } else {
      float lab[kLabels];
      unpack_labels(raw, lab);
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[r] = label_dot(ql[r], lab);
    }
    return acc;
  }
};

// float32 caches: the same result layout computed on the vector ALUs.
// q_lds holds the group's queries [16][128] (rows >= G are zero).  Each dot
// product runs over d in ascending order with fused multiply-adds.
__device__ __forceinline__ f32x4 valu_scores_f32(const float *q_lds, const float *krow, int G) {
  const int s = lane_id() >> 4;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int c = 0; c < kHeadDim / 4; ++c) {
    const float4 kv = ((const float4 *)krow)[c];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int h = 4 * s + r;
      if (h < G) {
        const float4 qv = ((const float4 *)(q_lds + h * kHeadDim))[c];
        float a = acc[r];
        a = fmaf(qv.x, kv.x, a);
        a = fmaf(qv.y, kv.y, a);
        a = fmaf(qv.z, kv.z, a);
        a = fmaf(qv.w, kv.w, a);
        acc[r] = a;
      }
    }
  }
  return acc;
}

__device__ __forceinline__ void load_q_f32_lds(const Params &p, int b, int g, float *q_lds) {
  for (int e = threadIdx.x; e < kMaxGroup * kHeadDim; e += blockDim.x) {
    const int h = e / kHeadDim;
    q_lds[e] = h < p.G ? ((const float *)p.q)[((int64_t)b * p.Hq + (int64_t)g * p.G + h) * kHeadDim +
                                               (e % kHeadDim)]
                       : 0.f;
  }
}

// Group-summed score of the tile's key for this lane: heads beyond G hold
// exact zeros, so summing all 16 rows equals summing the group.  The sum is
// formed the same way in every kernel, hence bit-identical everywhere.
__device__ __forceinline__ float group_sum(f32x4 acc) {
  float s = (acc[0] + acc[1]) + (acc[2] + acc[3]);
  s += __shfl_xor(s, 16);
  s += __shfl_xor(s, 32);
  return s;
}

// ---------------------------------------------------------------------------
// Block-wide primitives for blocks of NT threads (NT / 64 waves, default
// kBlock; the selection also runs 1024-thread blocks when rows are few).
constexpr int kMaxBlockWaves = 16;
// ---------------------------------------------------------------------------
__device__ __forceinline__ int wave_incl_scan(int v) {
  const int l = lane_id();
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int t = __shfl_up(v, o);
    if (l >= o) v += t;
  }
  return v;
}

// x itself, hidden from the optimiser: values derived from x in one phase
// are recomputed in the next instead of being kept alive across it.
__device__ __forceinline__ uint32_t fresh(uint32_t x) {
  asm volatile("" : "+v"(x));
  return x;
}

__device__ __forceinline__ int lanes_below(uint64_t m) {
  return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                        __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// Inclusive prefix sum over the wave's 64 lanes by DPP lane shifts within
// rows of 16 (1, 2, 4, 8) and the two row broadcasts (no LDS round trips).
__device__ __forceinline__ int wave_incl_scan_dpp(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xf, 0xf, false);  // row_shr:1
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xf, 0xf, false);  // row_shr:2
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xf, 0xf, false);  // row_shr:4
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xf, 0xf, false);  // row_shr:8
  v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xa, 0xf, false);  // row_bcast:15, rows 1, 3
  v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xc, 0xf, false);  // row_bcast:31, rows 2, 3
  return v;
}

// f(std::integral_constant<int, u>) for u = 0 .. N-1, unrolled in the
// source: register arrays indexed by u keep constant indices from the start
// and stay scalar registers (a loop unrolled later by the compiler can leave
// them promoted to one vector value that every branch then copies whole).
template <int I, int N, class F>
__device__ __forceinline__ void unroll_for_from(F &f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    unroll_for_from<I + 1, N>(f);
  }
}
template <int N, class F>
__device__ __forceinline__ void unroll_for(F &&f) {
  unroll_for_from<0, N>(f);
}

// Exclusive prefix sum over the block in thread order; *total gets the sum.
// tmp: LDS int[NT / 64].  Must be reached by every thread of the block.
template <int NT = kBlock>
__device__ __forceinline__ int block_excl_scan(int v, int *tmp, int *total) {
  constexpr int NW = NT / 64;
  const int inc = wave_incl_scan(v);
  if (lane_id() == 63) tmp[wave_id()] = inc;
  __syncthreads();
  int before = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    const int t = tmp[w];
    before += (w < wave_id()) ? t : 0;
    tot += t;
  }
  __syncthreads();
  *total = tot;
  return before + inc - v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

template <int NT = kBlock>
__device__ __forceinline__ float block_max(float v, float *tmp) {
  constexpr int NW = NT / 64;
  v = wave_max(v);
  if (lane_id() == 0) tmp[wave_id()] = v;
  __syncthreads();
  float m = tmp[0];
#pragma unroll
  for (int w = 1; w < NW; ++w) m = fmaxf(m, tmp[w]);
  __syncthreads();
  return m;
}

// Add 1 to hist[dig] for every active lane with act set.  Lanes sharing the
// first active lane's bin are counted with one atomic (the common case when
// the leading key bits cluster); the others add their own.
__device__ __forceinline__ void hist_add(uint32_t *hist, uint32_t dig, bool act) {
  const uint64_t am = __ballot(act);
  if (!am) return;
  const int leader = __ffsll((unsigned long long)am) - 1;
  const uint32_t v = __shfl(dig, leader);
  const uint64_t same = __ballot(act && dig == v);
  if (lane_id() == leader) atomicAdd(&hist[v], (uint32_t)__popcll(same));
  if (act && dig != v) atomicAdd(&hist[dig], 1u);
}

// ---------------------------------------------------------------------------
// Exact selection of the k-th largest key among n items by three histogram
// passes over 11, 11 and 10 key bits.  src.key(p) returns item p's key.
// On return T is the k-th largest key and need_eq the number of items equal
// to T that belong to the top k (the others with key == T are the later ones
// in item order).  hist: LDS uint32[2048]; sh: LDS scratch.  With passes < 3
// only the top bits of T are resolved (the rest are zero): T is then a lower
// bound of the k-th largest key.
// ---------------------------------------------------------------------------
constexpr int kSelU = 8;  // item loads in flight per thread in a selection pass

struct SelShared {
  int scan[kMaxBlockWaves];
  uint32_t digit;
  int above;
};

template <int NT = kBlock, class Src>
__device__ void radix_select(const Src &src, int n, int k, uint32_t *hist, SelShared *sh,
                             uint32_t &T, int &need_eq, int passes = 3) {
  uint32_t prefix = 0, mask = 0;
  int krem = k;
  const int tid = threadIdx.x;
#pragma unroll 1
  for (int pass = 0; pass < passes; ++pass) {
    const int shift = pass == 0 ? 21 : (pass == 1 ? 10 : 0);
    const int nb = pass == 2 ? 1024 : 2048;
    const uint32_t dmask = (uint32_t)nb - 1u;
    for (int i = tid; i < nb; i += NT) hist[i] = 0;
    __syncthreads();
    for (int base = 0; base < n; base += NT * kSelU) {
      uint32_t key[kSelU];
#pragma unroll
      for (int u = 0; u < kSelU; ++u) {  // the loads in flight together
        const int p = base + u * NT + tid;
        key[u] = p < n ? src.key(p) : 0u;
      }
#pragma unroll
      for (int u = 0; u < kSelU; ++u) {
        const bool act = base + u * NT + tid < n && (key[u] & mask) == prefix;
        hist_add(hist, (key[u] >> shift) & dmask, act);
      }
    }
    __syncthreads();
    // Thread t owns bins [nb - (t+1)*bpt, nb - t*bpt): counting from the top.
    const int bpt = nb / NT;
    const int hi = nb - tid * bpt;
    int mine = 0;
    for (int i = 1; i <= bpt; ++i) mine += (int)hist[hi - i];
    int tot;
    const int before = block_excl_scan<NT>(mine, sh->scan, &tot);
    if (before < krem && krem <= before + mine) {
      int cum = before;
      for (int i = 1; i <= bpt; ++i) {
        const int c = (int)hist[hi - i];
        if (cum + c >= krem) {
          sh->digit = (uint32_t)(hi - i);
          sh->above = cum;
          break;
        }
        cum += c;
      }
    }
    __syncthreads();
    prefix |= sh->digit << shift;
    mask |= dmask << shift;
    krem -= sh->above;
    __syncthreads();
  }
  T = prefix;
  need_eq = krem;
}

// ---------------------------------------------------------------------------
// Log-sum-exp merge of split partials.  pp points at nsp partials of one
// output row, kPartStride floats apart, each (m, l, o[128]): a maximum m of
// the split's logits, l = sum exp(z - m) and o = sum exp(z - m) v.  The merged
// row is sum_q e^(m_q - M) o_q / sum_q e^(m_q - M) l_q with M = max m_q (zeros
// when no split holds an entry).  Run by a block of kMergeThreads: the maxima
// and scale factors in parallel, then each channel's sum over the partials by
// the two halves of the block, several loads in flight per thread.  Returns
// channel threadIdx.x & 127's value (meaningful where threadIdx.x < 128).
// Every thread of the block must call it.
// ---------------------------------------------------------------------------
constexpr int kMergeThreads = 256;
constexpr int kMergeChunk = 1024;  // partials whose scale factors sit in LDS at once

struct MergeShared {
  float f[kMergeChunk];
  float red[kMergeThreads / 64];
  float half_o[kHeadDim];
};

__device__ __forceinline__ float merge_partials(const float *pp, int nsp, MergeShared &sh) {
  const int tid = threadIdx.x, c = tid & (kHeadDim - 1), half = tid >> 7;
  float m = -__builtin_inff();
  for (int q = tid; q < nsp; q += kMergeThreads) m = fmaxf(m, pp[(int64_t)q * kPartStride]);
  const float M = block_max<kMergeThreads>(m, sh.red);
  float ls = 0.f, o = 0.f;
  for (int q0 = 0; q0 < nsp; q0 += kMergeChunk) {
    const int n = (nsp - q0) < kMergeChunk ? (nsp - q0) : kMergeChunk;
    const float *base = pp + (int64_t)q0 * kPartStride;
    for (int q = tid; q < n; q += kMergeThreads) {
      const float mq = base[(int64_t)q * kPartStride];
      const float f = mq == -__builtin_inff() ? 0.f : expf(mq - M);
      sh.f[q] = f;
      ls += f * base[(int64_t)q * kPartStride + 1];
    }
    __syncthreads();
#pragma unroll 8
    for (int q = half; q < n; q += 2) o += sh.f[q] * base[(int64_t)q * kPartStride + 2 + c];
    __syncthreads();
  }
  // Sum of the l terms over the block; the two halves' channel sums.
  float t = ls;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) t += __shfl_xor(t, off);
  if (lane_id() == 0) sh.red[wave_id()] = t;
  if (half == 1) sh.half_o[c] = o;
  __syncthreads();
  float sum = 0.f;
#pragma unroll
  for (int w = 0; w < kMergeThreads / 64; ++w) sum += sh.red[w];
  o += sh.half_o[c];
  return sum > 0.f ? o / sum : 0.f;
}

// ---------------------------------------------------------------------------
// Order-preserving compaction of the selection: walk items in order and keep
// those with key > T plus the first need_eq with key == T.  emit(slot, i, key)
// is called for every kept item i with its output slot (0..k-1 in item
// order).  Only keys are read here; the caller fetches whatever else a kept
// item carries.  Each thread handles kIpt consecutive items per round.
// compact_selected_from continues a compaction begun elsewhere: eq_before
// items equal to T and sel_before kept items precede item 0 (slots start at
// sel_before).
// ---------------------------------------------------------------------------
constexpr int kIpt = 8;

template <int NT = kBlock, class Src, class Emit>
__device__ void compact_selected_from(const Src &src, int n, int k, uint32_t T, int need_eq,
                                      int *scan, int eq_before, int sel_before, Emit emit) {
  const int tid = threadIdx.x;
#pragma unroll 1
  for (int base = 0; base < n && sel_before < k; base += NT * kIpt) {
    const int p0 = base + tid * kIpt;
    uint32_t key[kIpt];
    int n_eq = 0;
#pragma unroll
    for (int u = 0; u < kIpt; ++u) {
      const int p = p0 + u;
      key[u] = p < n ? src.key(p) : 0u;
      n_eq += (p < n && key[u] == T) ? 1 : 0;
    }
    int eq_tot;
    int eq_rank = block_excl_scan<NT>(n_eq, scan, &eq_tot) + eq_before;
    unsigned sel_mask = 0;
    int n_sel = 0;
#pragma unroll
    for (int u = 0; u < kIpt; ++u) {
      const int p = p0 + u;
      bool sel = false;
      if (p < n) {
        if (key[u] > T) {
          sel = true;
        } else if (key[u] == T) {
          sel = eq_rank < need_eq;
          ++eq_rank;
        }
      }
      sel_mask |= sel ? (1u << u) : 0u;
      n_sel += sel ? 1 : 0;
    }
    int sel_tot;
    int slot = block_excl_scan<NT>(n_sel, scan, &sel_tot) + sel_before;
#pragma unroll
    for (int u = 0; u < kIpt; ++u)
      if (sel_mask & (1u << u)) emit(slot++, p0 + u, key[u]);
    eq_before += eq_tot;
    sel_before += sel_tot;
  }
}

// The same over a whole row: no items before it.
template <int NT = kBlock, class Src, class Emit>
__device__ void compact_selected(const Src &src, int n, int k, uint32_t T, int need_eq, int *scan,
                                 Emit emit) {
  compact_selected_from<NT>(src, n, k, T, need_eq, scan, 0, 0, emit);
}

}  // namespace sd
