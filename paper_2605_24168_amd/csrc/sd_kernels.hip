// sd_kernels.hip -- gfx950 kernels of exact top-k context-sparse decode
// attention (arXiv 2605.24168, Section 3: exact "oracle" top-k at decode
// time; Table 1: k = N/S per query head; per-query, per-head, token-level
// sparsity under GQA).
//
// Fused pipeline for one decode step, all on the caller's stream:
//   k_pilot_score   scores a strided sample of <= 2048 keys per row
//   k_pilot_select  picks a per-row threshold from the sample (aimed at about
//                   2.5 k candidates) and flags rows for the fallback
//   k_score_stream  streams every key once (MFMA scoring, one K tile shared
//                   by all query heads of the group), stages the keys at or
//                   above the threshold in LDS in position order (ballots,
//                   no atomics) and writes one packed block per workgroup
//   k_repair_score  flags the rows whose candidates cannot prove exactness
//                   and scores their groups in full (the exact fallback);
//                   with few rows, also the per-piece run counts of the
//                   candidate selection in pieces
//   k_select        exact top-k: over the candidates (with few rows of many
//                   candidates, one workgroup per piece of a row), or over
//                   the full scores for a flagged row
//   k_attend        gathers the kept value rows, split over workgroups
//   k_merge         combines the splits' (max, sum, output) partials by
//                   log-sum-exp (only when a row is split)
// The threshold is only a filter: the selection is exact whenever every
// kept position passed it, which holds iff at least k candidates passed
// (then the k-th largest candidate is >= the threshold, so nothing above
// the true k-th largest score was filtered out) and no staging area
// overflowed.  Otherwise the row takes the exact fallback.
#include <hip/hip_ext.h>

#include "sd_internal.hpp"
#include "sd_launch.hpp"

namespace sd {

// ---------------------------------------------------------------------------
// Scoring of one key per lane, in the MFMA result layout.
// ---------------------------------------------------------------------------
template <bool BF16, bool LABEL = false>
struct Scorer {
  QFrag qf;
  LabelRows lr;
  float *q_lds;
  // The loaded operand of one tile (bf16 keys or labels), so that several
  // tiles can be in flight: load() issues the loads, from_raw() scores.
  using Raw = std::conditional_t<LABEL, u32x4, KFrag>;
  __device__ __forceinline__ void load(const Params &p, int b, int g, int64_t j, Raw &r) const {
    if constexpr (LABEL) r = load_labels(p.labels, label_offset(p.K, b, g, j));
    else load_k_bf16(p.K, kv_offset(p.K, b, g, j), r);
  }
  __device__ __forceinline__ f32x4 from_raw(const Raw &r) const {
    if constexpr (LABEL) return lr.score(r);
    else return mfma_scores(qf, r);
  }
  __device__ __forceinline__ f32x4 score(const Params &p, int b, int g, int64_t j) const {
    if constexpr (LABEL) {
      return lr.score(load_labels(p.labels, label_offset(p.K, b, g, j)));
    } else if constexpr (BF16) {
      KFrag kf;
      load_k_bf16(p.K, kv_offset(p.K, b, g, j), kf);
      return mfma_scores(qf, kf);
    } else {
      return valu_scores_f32(q_lds, (const float *)p.K.base + kv_offset(p.K, b, g, j), p.G);
    }
  }
};

// Shared prologue: query fragments (bf16) or the group's queries in LDS (f32).
// Every thread of the block must call it.
template <bool BF16, bool LABEL>
__device__ __forceinline__ void scorer_init(const Params &p, int b, int g,
                                            Scorer<BF16, LABEL> &sc, float *q_lds) {
  sc.q_lds = q_lds;
  if constexpr (LABEL) {
    sc.lr.init(p, b, g);
  } else if constexpr (BF16) {
    load_q_bf16(p, b, g, sc.qf);
  } else {
    load_q_f32_lds(p, b, g, q_lds);
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Pilot: scores of a strided sample of each sequence (bfloat16 caches).
// grid = (kSampleMax / (kPilotTiles * kTile * kWaves), B*Hkv).  Sample i of a
// sequence of length L is position floor(i*L/m), m = min(L, kSampleMax), so
// m = L samples every position.  Each wave scores up to kPilotTiles sample
// tiles, all of their (scattered) key loads issued before the matrix ops.
// ---------------------------------------------------------------------------
constexpr int kPilotTiles = 4;

// LABEL: the samples are scored by the low-channel indexer (label tiles).
// QUAD (paged caches with a multiple of 4 KV heads): grid = (kSampleMax /
// (kPilotTiles * kTile), B*Hkv/4), and wave v of a workgroup takes KV head
// 4q + v over the same sample tiles as its neighbours: the four heads of a
// sampled position are adjacent in a page (256 B each), so their rows are
// requested together instead of by four workgroups at different times.
template <bool LABEL, bool QUAD>
__global__ __launch_bounds__(kBlock) void k_pilot_score(Params p, Work w) {
  const int hq = QUAD ? p.Hkv / kWaves : p.Hkv;
  const int by = blockIdx.y, b = by / hq;
  const int g = QUAD ? (by % hq) * kWaves + wave_id() : by % hq;
  const int L = seq_len(p, b);
  const RowPlan rp = row_plan(p, b, L);  // samples come from the top-k range only
  const int mid = rp.hi - rp.lo;
  const int m = mid < kSampleMax ? mid : kSampleMax;
  const int ntiles = (m + kTile - 1) / kTile;
  const int l = lane_id(), col = l & 15, s = l >> 4;
  const int t0 = QUAD ? (int)blockIdx.x : (int)blockIdx.x * kWaves + wave_id();
  const int stride = QUAD ? (int)gridDim.x : (int)gridDim.x * kWaves;
  if (t0 >= ntiles) return;  // wave-uniform; no barriers in this kernel
  QFrag qf;
  LabelRows lr;
  if constexpr (LABEL) lr.init(p, b, g);
  else load_q_bf16(p, b, g, qf);
  KFrag kf[kPilotTiles];
  u32x4 lf[kPilotTiles];
#pragma unroll
  for (int u = 0; u < kPilotTiles; ++u) {
    const int t = t0 + u * stride;
    const int si = t * kTile + col;
    const int64_t pos = rp.lo + ((t < ntiles && si < m) ? ((int64_t)si * mid) / m : 0);
    if constexpr (LABEL) lf[u] = load_labels(p.labels, label_offset(p.K, b, g, pos));
    else load_k_bf16(p.K, kv_offset(p.K, b, g, pos), kf[u]);
  }
#pragma unroll
  for (int u = 0; u < kPilotTiles; ++u) {
    const int t = t0 + u * stride;
    if (t >= ntiles) break;  // wave-uniform
    const int si = t * kTile + col;
    const bool valid = si < m;
    f32x4 acc;
    if constexpr (LABEL) acc = lr.score(lf[u]);
    else acc = mfma_scores(qf, kf[u]);
    if (!p.group_shared) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int h = 4 * s + r;
        if (valid && h < p.G)
          w.sample[((int64_t)b * p.R + (int64_t)g * p.G + h) * kSampleMax + si] = acc[r];
      }
    } else {
      const float gs = group_sum(acc);
      if (valid && s == 0) w.sample[((int64_t)b * p.R + g) * kSampleMax + si] = gs;
    }
  }
}

// ---------------------------------------------------------------------------
// k-th largest of n order-preserving keys staged in LDS, kmin..kmax their
// range (1 <= k <= n).  One histogram over kBuckets value buckets,
// bucket(v) = min(kBuckets-1, floor((v - vmin) * kBuckets / (vmax - vmin))),
// which is monotone in v (rounded subtraction and scaling by a positive
// constant preserve order), so a higher bucket holds only larger values;
// inside the bucket holding the k-th largest, an exact rank count over its
// items gives T (the k-th largest key) and need_eq (how many items equal to
// T belong to the top k).  Returns false, with T and need_eq unset, when the
// range is not finite or that bucket holds more items than the block has
// threads.
// Every thread of the block must call it.
// ---------------------------------------------------------------------------
constexpr int kBuckets = 2048;
constexpr int kPilotMinRank = 48;  // fewest sample ranks above the threshold

template <int NT = kBlock>
struct BucketShared {
  uint32_t items[NT];  // the k-th bucket's items, at most one per thread
  int n;
};

template <int NT = kBlock>
__device__ bool bucket_kth(const uint32_t *keys, int n, int k, uint32_t kmin, uint32_t kmax,
                           uint32_t *hist, SelShared *sh, BucketShared<NT> *bs, uint32_t &T,
                           int &need_eq) {
  if (kmin == kmax) {  // all equal: the first k
    T = kmin;
    need_eq = k;
    return true;
  }
  const int tid = threadIdx.x;
  const float vmin = key2f(kmin), vmax = key2f(kmax);
  const float inv = (float)kBuckets / (vmax - vmin);
  if (!(__builtin_isfinite(vmin) && __builtin_isfinite(inv) && inv > 0.f)) return false;
  auto bucket = [&](uint32_t key) {
    const int bk = (int)((key2f(key) - vmin) * inv);
    return bk < kBuckets - 1 ? bk : kBuckets - 1;
  };
  for (int i = tid; i < kBuckets; i += NT) hist[i] = 0;
  __syncthreads();
  // keys may sit in global memory: kSelU loads in flight per thread
  for (int base = 0; base < n; base += NT * kSelU) {
    uint32_t key[kSelU];
#pragma unroll
    for (int u = 0; u < kSelU; ++u) {
      const int i = base + u * NT + tid;
      key[u] = i < n ? keys[i] : kmin;
    }
#pragma unroll
    for (int u = 0; u < kSelU; ++u)
      if (base + u * NT + tid < n) atomicAdd(&hist[bucket(key[u])], 1u);  // buckets spread the items
  }
  __syncthreads();
  // Thread t owns buckets [nb - (t+1)*bpt, nb - t*bpt), counted from the top.
  constexpr int bpt = kBuckets / NT;
  const int hi = kBuckets - tid * bpt;
  int mine = 0;
  for (int j = 1; j <= bpt; ++j) mine += (int)hist[hi - j];
  int tot;
  const int before = block_excl_scan<NT>(mine, sh->scan, &tot);
  if (tid == 0) bs->n = 0;
  if (before < k && k <= before + mine) {
    int cum = before;
    for (int j = 1; j <= bpt; ++j) {
      const int c = (int)hist[hi - j];
      if (cum + c >= k) {
        sh->digit = (uint32_t)(hi - j);
        sh->above = cum;
        break;
      }
      cum += c;
    }
  }
  __syncthreads();
  const int bstar = (int)sh->digit;
  const int krem = k - sh->above;
  const int m = (int)hist[bstar];
  bool found = false;
  if (m <= NT) {  // uniform
    for (int base = 0; base < n; base += NT * kSelU) {
      uint32_t key[kSelU];
#pragma unroll
      for (int u = 0; u < kSelU; ++u) {
        const int i = base + u * NT + tid;
        key[u] = i < n ? keys[i] : kmin;
      }
#pragma unroll
      for (int u = 0; u < kSelU; ++u)
        if (base + u * NT + tid < n && bucket(key[u]) == bstar)
          bs->items[atomicAdd(&bs->n, 1)] = key[u];
    }
    __syncthreads();
    if (tid < m) {
      const uint32_t x = bs->items[tid];
      int gt = 0, ge = 0;
      for (int y = 0; y < m; ++y) {
        const uint32_t v = bs->items[y];
        gt += v > x ? 1 : 0;
        ge += v >= x ? 1 : 0;
      }
      if (gt < krem && krem <= ge) {  // x is the krem-th largest (equal items agree)
        sh->digit = x;
        sh->above = gt;
      }
    }
    __syncthreads();
    T = sh->digit;
    need_eq = krem - sh->above;
    found = true;
  }
  __syncthreads();  // sh and hist are reused by the caller
  return found;
}

// Block-wide (min, max) of per-thread key ranges; tmp: LDS uint32[NT/64][2].
// Ends with a barrier (so LDS written before the call is visible after it).
template <int NT = kBlock>
__device__ __forceinline__ void block_key_range(uint32_t &mn, uint32_t &mx, uint32_t (*tmp)[2]) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const uint32_t a = __shfl_xor(mn, o), c = __shfl_xor(mx, o);
    mn = a < mn ? a : mn;
    mx = c > mx ? c : mx;
  }
  if (lane_id() == 0) {
    tmp[wave_id()][0] = mn;
    tmp[wave_id()][1] = mx;
  }
  __syncthreads();
#pragma unroll
  for (int v = 0; v < NT / 64; ++v) {
    mn = tmp[v][0] < mn ? tmp[v][0] : mn;
    mx = tmp[v][1] > mx ? tmp[v][1] : mx;
  }
  __syncthreads();
}

struct LdsKeys {
  const uint32_t *keys;
  __device__ __forceinline__ uint32_t key(int i) const { return keys[i]; }
};

// Per-row threshold = the r-th largest sample score, r = ceil(2.5 k m / L)
// (so about 2.5 k of the L keys are expected to pass), or r = k when the
// sample is the whole sequence.  Also sets the row's fallback flag: rows
// with k = 0 need nothing; the row takes the exact fallback (threshold +inf,
// so it stages no candidates) when every row is forced to, or when its
// expected candidates per wave, r * min(L, wave_keys) / m, exceed half of
// its staging area (low sparsity).
constexpr int kOrderBatchMax = 2048;  // batches ordered by length (lengths staged in hist)

__global__ __launch_bounds__(kBlock) void k_pilot_select(Params p, Work w) {
  __shared__ uint32_t keys[kSampleMax];
  __shared__ uint32_t hist[2048];
  __shared__ SelShared sh;
  __shared__ BucketShared<> bs;
  __shared__ uint32_t range[kWaves][2];
  const int row = blockIdx.x, b = row / p.R;
  if (row == 0 && w.persistent) {
    // The persistent stream's work list: ceil(L_b / chunk_keys) chunks of
    // every sequence, unit_heads units each, and an empty queue.
    int carry = 0;
    for (int base = 0; base < p.B; base += kBlock) {
      const int bb = base + (int)threadIdx.x;
      const int units = bb < p.B ? (seq_len(p, bb) + w.chunk_keys - 1) / w.chunk_keys * w.unit_heads : 0;
      int tot;
      const int e = block_excl_scan(units, sh.scan, &tot);
      if (bb < p.B) w.unit_pre[bb] = carry + e;
      carry += tot;
    }
    if (threadIdx.x == 0) {
      w.unit_pre[p.B] = carry;
      w.queue[0] = 0;
    }
  }
  if (row == 0) {
    // Sequences by descending length (ties: lower index first): rank each
    // by counting the ones before it, over the lengths staged in LDS (batch
    // order for very large batches).
    const int nb = p.B <= kOrderBatchMax ? p.B : 0;
    int *lens = (int *)hist;  // (free until the row's own selection below)
    for (int bb = (int)threadIdx.x; bb < nb; bb += kBlock) lens[bb] = seq_len(p, bb);
    __syncthreads();
    for (int bb = (int)threadIdx.x; bb < p.B; bb += kBlock) {
      int rank = bb;
      if (nb) {
        const int Lb = lens[bb];
        rank = 0;
        for (int o = 0; o < nb; ++o) rank += (lens[o] > Lb || (lens[o] == Lb && o < bb)) ? 1 : 0;
      }
      w.seq_order[rank] = bb;
    }
    __syncthreads();  // (hist is the selection's again)
  }
  const int L = seq_len(p, b);
  const RowPlan rp = row_plan(p, b, L);
  const int k = rp.kh;
  const int mid = rp.hi - rp.lo;  // the positions the top-k runs over
  if (threadIdx.x == 0 && row == 0) w.stats[0] = 0;
  const int m = mid < kSampleMax ? mid : kSampleMax;
  const int cap = kCandBuf / (p.group_shared ? 1 : p.G);
  const int64_t span = mid < w.wave_keys ? mid : w.wave_keys;
  int r = k;
  if (m < mid) {
    // About 2.5 k candidates where the expected sample rank of the k-th key,
    // e = k m / n, is small; where it is large the count above the r-th
    // sample varies by about sqrt(r) ranks only, so r need only clear e by
    // kPilotZ of them (pilot_rank; at e of about 20 the two agree).
    r = (int)pilot_rank(k, m, mid);
    // A small rank leaves the candidate count a relative spread of about
    // 1/sqrt(r): with k of a few dozen, one row in five would come up short
    // of k.  Take at least kPilotMinRank (as far as the staging areas hold
    // the candidates it lets through), which then passes far more than k.
    const int64_t fit = (int64_t)cap * m / (2 * span);
    const int rmin = (int)(kPilotMinRank < fit ? kPilotMinRank : fit);
    if (r < rmin) r = rmin < m ? rmin : m;
    if (r < 1) r = 1;
  }
  // Rows whose expected candidates per wave would fill more than half of a
  // staging area take the exact fallback.  (r - 1): r is rounded up, and the
  // wave size was chosen on the unrounded expectation.
  const bool dense = w.force_repair || 2LL * (r - 1) * span > (int64_t)cap * m;
  if (k == 0 || dense) {
    if (threadIdx.x == 0) {
      w.flags[row] = k > 0 ? 1 : 0;
      w.theta[row] = __builtin_inff();
    }
    return;
  }
  if (threadIdx.x == 0) w.flags[row] = 0;
  uint32_t mn = 0xFFFFFFFFu, mx = 0u;
  for (int i = threadIdx.x; i < m; i += kBlock) {
    const uint32_t key = f2key(w.sample[(int64_t)row * kSampleMax + i]);
    keys[i] = key;
    mn = key < mn ? key : mn;
    mx = key > mx ? key : mx;
  }
  block_key_range(mn, mx, range);  // also publishes keys
  if (threadIdx.x == 0) w.smax[row] = key2f(mx);
  uint32_t T;
  int need_eq;
  // The r-th largest sample exactly; else (rare) two radix passes fix its
  // top 22 key bits and the threshold is the lowest key with those bits.
  if (!bucket_kth(keys, m, r, mn, mx, hist, &sh, &bs, T, need_eq))
    radix_select(LdsKeys{keys}, m, r, hist, &sh, T, need_eq, 2);
  if (threadIdx.x == 0) w.theta[row] = key2f(T);
}

// ---------------------------------------------------------------------------
// The scoring stream.  Its unit of work is one chunk of one (sequence, KV
// head): kWaves * wk keys (wk = w.wave_keys), wave v streaming keys
// [c*4wk + v*wk, +wk) in 16-key MFMA tiles, kDepth tiles in flight, and
// staging the keys at or above each row's threshold in LDS, in position
// order, one area of kCandBuf / rows entries per row of the group.  Each
// unit leaves one packed block: for every row its candidates (keys, then
// chunk-relative positions), in position order, rows one after another;
// dir[row][c] gets the row's (start, count) in the block, count -1 if one
// of its areas overflowed.  (QUAD: the unit is one chunk of wk keys of four
// KV heads, one per wave, and each wave's head gets its own block.)
//
// Persistent launch (w.persistent): one workgroup per compute unit takes
// units from a device-side queue until none is left.  The units are those
// of k_pilot_select's work list (unit_pre: units of the sequences before
// each one, so that chunks past a sequence's end are never handed out),
// hence a ragged batch stays balanced.  The blocks a workgroup produces are
// kept in an LDS outbox and written to HBM when it is full and when the
// workgroup runs out of work: HBM writes interleaved with the key stream
// cost far more than their bytes on this memory system (about 1.7 us per
// MB of candidates measured at the 128K batch-16 workload), while one burst
// at the end, after the reads, costs little.
// Otherwise (label rows: one workgroup per compute unit leaves that stream
// too few loads in flight and its latency chains unhidden, measured 50%
// slower) one workgroup per unit, several per compute unit, on a static grid
// that includes empty chunks, writes its block directly.
// The streaming loop issues no global stores, so its load waits stay exact.
// ---------------------------------------------------------------------------
constexpr int kDepth = 3;        // tiles in flight per wave
constexpr int kWavePages = kWaveKeysMax / kTile;
static_assert(kCandBuf / kMaxGroup >= kTile, "every row must hold a tile's keys");
static_assert(kChunkCap % 4 == 0 && kWaves * kMaxGroup == 64, "block layout");
static_assert(kOutboxCap >= kChunkCap && kOutboxCap % 4 == 0, "a unit's blocks fit an empty outbox");

struct WaveLds {
  u32x4 tile[256];
  uint2 cand[kCandBuf + 64];   // per-row areas of (score bits, position in wave), +64 discard slots
  int32_t page[kWavePages];
};

// The LDS outbox of a persistent stream workgroup: nb blocks of n entries
// in all (keys in obk, positions in obp, each block starting at a multiple
// of 4 entries), block j going to entry dst[j] of the candidate blocks.
// The key and position arrays follow the struct in dynamic LDS (16-byte
// aligned for the 16-byte accesses).
struct alignas(16) Outbox {
  uint32_t *obk;
  uint16_t *obp;
  int n, nb;
  int64_t dst[kOutboxBlocks];
  int off[kOutboxBlocks], cnt[kOutboxBlocks];
};

struct StreamLds {
  WaveLds wave[kWaves];
  int seg_n[kWaves * kMaxGroup];          // [row][wave] candidates found
  int seg_off[kWaves * (kMaxGroup + 1)];  // their offsets in the block(s)
  int wave_tot[kWaves];                   // QUAD: entries of each wave's block
  int unit;                               // the unit taken from the queue
};
// (Under a third of the 160 KB of a compute unit: three label-stream
// workgroups fit on one.)
static_assert(sizeof(StreamLds) <= 163840 / 3, "three label-stream workgroups per compute unit");

// Write the outbox's blocks to the candidate blocks (16- and 8-byte stores)
// and empty it.  Every thread of the block must call it.  Plain stores: the
// lines stay cached for the selection, and on the ragged paged batch the
// scoring kernel itself took 6 us less than with nontemporal stores.
__device__ __forceinline__ void outbox_flush(const Work &w, Outbox &ob) {
  __syncthreads();
  for (int j = 0; j < ob.nb; ++j) {
    const int off = ob.off[j], cnt = ob.cnt[j];
    const int64_t dst = ob.dst[j];
    for (int i0 = 4 * (int)threadIdx.x; i0 < cnt; i0 += 4 * kBlock) {
      *(u32x4 *)(w.ckey + dst + i0) = *(const u32x4 *)(ob.obk + off + i0);
      *(unsigned long long *)(w.cpos + dst + i0) = *(const unsigned long long *)(ob.obp + off + i0);
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    ob.n = 0;
    ob.nb = 0;
  }
  __syncthreads();
}

// Room in the outbox for `need` entries in `blocks` more blocks: returns
// where they start, after flushing it if they do not fit.  Every thread of
// the block must call it; it ends with a barrier, so that no thread reads
// the outbox state after thread 0 advances it.
__device__ __forceinline__ int outbox_reserve(const Work &w, Outbox &ob, int need, int blocks) {
  if (ob.n + need > kOutboxCap || ob.nb + blocks > kOutboxBlocks) outbox_flush(w, ob);
  const int base = ob.n;
  __syncthreads();
  return base;
}

// Pack entries [i0, i0 + 4) of a block (item i: entry i of the staged
// candidates, found by cand_of) into 16 + 8 bytes and store them at kdst /
// pdst + i0, in LDS (outbox) or in HBM (nontemporal).
template <class CandOf>
__device__ __forceinline__ void pack4(int i0, int ntot, CandOf cand_of, uint32_t *kdst,
                                      uint16_t *pdst, bool to_lds) {
  u32x4 kv;
  uint32_t pv[2] = {0u, 0u};
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int i = i0 + u;
    uint32_t key = 0u, pos = 0u;
    if (i < ntot) {
      const uint2 it = cand_of(i);
      key = f2key(__uint_as_float(it.x));
      pos = it.y;
    }
    kv[u] = key;
    pv[u >> 1] |= pos << (16 * (u & 1));
  }
  const unsigned long long pp = (unsigned long long)pv[0] | ((unsigned long long)pv[1] << 32);
  if (to_lds) {
    *(u32x4 *)(kdst + i0) = kv;
    *(unsigned long long *)(pdst + i0) = pp;
  } else {
    __builtin_nontemporal_store(kv, (u32x4 *)(kdst + i0));
    __builtin_nontemporal_store(pp, (unsigned long long *)(pdst + i0));
  }
}

// bfloat16 caches.  The loop body issues a fixed set of loads every step
// (tile indices past the end are clamped to the last tile, whose keys the
// filter then masks), so the compiler's memory waits are exact.
// QUAD (paged layout, Hkv a multiple of 4): a chunk is wk keys, and wave v
// of the workgroup of (quad q, chunk) scores KV head 4q + v over the whole
// chunk, so the workgroup reads four of the heads of every page block
// together; each wave then packs its own head's block.
// LABEL: the low-channel indexer scores label rows (16 bytes per key) on
// the vector ALUs instead of key rows; candidates, blocks and directory are
// the same.
constexpr int kLabelDepth = 8;  // 64-key label tiles in flight per wave (8 KB)
// In label waves the key-tile LDS area holds the wave's page ids.
constexpr int kLabelPageBase = 0;
static_assert(kLabelPageBase + kLabelWaveKeysMax / kTile <= 1024, "label page ids fit the tile area");

// One unit: sequence b, chunk `chunk`, KV head g0 (QUAD: heads g0 .. g0+3,
// one per wave).  ob: the outbox, or null to store the blocks in HBM.
// Every thread of the block must call it (it has barriers).
// NR: rows per wave held in registers by the label path (a power of two
// >= the group's rows; 0 for key rows).
template <bool PAGED, bool GRP, bool QUAD, bool LABEL, int NR>
__device__ __forceinline__ void stream_unit(const Params &p, const Work &w, int b, int g0,
                                            int chunk, StreamLds &sl, Outbox *ob) {
  static_assert(PAGED || !QUAD, "head quads are for the paged layout");
  const int wk = w.wave_keys;
  const int wv = wave_id();
  const int g = QUAD ? g0 + wv : g0;
  const int bg = b * p.Hkv + g;
  const int L = seq_len(p, b);
  const int64_t c0 = (int64_t)chunk * w.chunk_keys;
  if (c0 >= L) return;  // whole workgroup (every wave has the same chunk)
  const int64_t w0 = QUAD ? c0 : c0 + (int64_t)wv * wk;
  const int nvalid = w0 < L ? (int)((L - w0) < wk ? (L - w0) : wk) : 0;
  // Candidates lie in the top-k range [lo, hi) of the sequence (forced
  // positions are kept apart): wave-relative, [jlo, jhi).
  const RowPlan rp = row_plan(p, b, L);
  const int jlo = rp.lo > w0 ? (int)(rp.lo - w0) : 0;
  const int jhi = (int)((int64_t)rp.hi - w0 < nvalid ? (int64_t)rp.hi - w0 : nvalid);
  const int l = lane_id(), col = l & 15, s = l >> 4;
  const int64_t row0 = GRP ? (int64_t)b * p.R + g : (int64_t)b * p.R + (int64_t)g * p.G;
  const int nrows = GRP ? 1 : p.G;
  const int cap = kCandBuf / nrows;  // staging slots per row
  WaveLds &wl = sl.wave[wv];
  // Candidates found per row: lane group s counts rows 4s+r (wave-uniform
  // within the group); counting continues past cap to detect overflow.
  int cnt[4] = {0, 0, 0, 0};
  if (nvalid > 0) {  // wave-uniform
    QFrag qf;
    if constexpr (!LABEL) load_q_bf16(p, b, g, qf);
    // This lane filters rows 4s..4s+3 (heads of the group; heads beyond G
    // never pass) or, in group-shared mode, lanes 0..15 the group's one row.
    float th[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int h = 4 * s + r;
      if (GRP) th[r] = (s == 0 && r == 0) ? w.theta[row0] : __builtin_inff();
      else th[r] = h < p.G ? w.theta[row0 + h] : __builtin_inff();
    }
    const int ntiles = (nvalid + kTile - 1) / kTile;
    // Page ids of the wave's keys (label waves take longer ranges and keep
    // them in the unused key-tile area).
    int32_t *pg = LABEL ? (int32_t *)wl.tile + kLabelPageBase : wl.page;
    if (PAGED) {
      const int32_t *bt = p.K.block_table + (int64_t)b * p.K.max_pages + (w0 >> 4);
      for (int i = l; i < ntiles; i += 64) pg[i] = bt[i];
      __builtin_amdgcn_wave_barrier();  // every lane reads every page id
    }
    const char *kbase = (const char *)p.K.base;
    constexpr int64_t kRowBytes = kHeadDim * 2;
    const char *slab = kbase + (((int64_t)b * p.K.hkv + g) * p.K.ncap + w0) * kRowBytes;
    const int64_t page_bytes = (int64_t)kTile * p.K.hkv * kRowBytes;
    const int a = l >> 4;
    const int last = nvalid - 1;
    int lane_row[4], lane_chunk[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      lane_row[t] = 4 * t + a;
      lane_chunk[t] = 16 * swz_chunk(t);
    }
    // Issue the four coalesced loads of tile ti (clamped to the last tile).
    auto load = [&](int ti, u32x4 v[4]) {
      ti = ti < ntiles ? ti : ntiles - 1;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        int j = ti * kTile + lane_row[t];
        j = j < last ? j : last;
        const char *row;
        if (PAGED) row = kbase + wl.page[ti] * page_bytes + ((int64_t)(j & 15) * p.K.hkv + g) * kRowBytes;
        else row = slab + (int64_t)j * kRowBytes;
        v[t] = __builtin_nontemporal_load((const u32x4 *)(row + lane_chunk[t]));
      }
    };
    // Append the passing keys of one scored tile to their rows' areas;
    // keys past an area's end go to this lane's discard slot.
    auto filter = [&](f32x4 acc, int jl) {
      const bool live = jl >= jlo && jl < jhi;
      if (GRP) acc[0] = group_sum(acc);
#pragma unroll
      for (int r = 0; r < (GRP ? 1 : 4); ++r) {
        const bool pass = live && acc[r] >= th[r];
        const uint32_t gm = (uint32_t)(__ballot(pass) >> (16 * s)) & 0xFFFFu;
        const int slot = cnt[r] + __popc(gm & ((1u << col) - 1u));
        const int e = (pass && slot < cap) ? (4 * s + r) * cap + slot : kCandBuf + l;
        wl.cand[e] = make_uint2(__float_as_uint(acc[r]), (uint32_t)jl);
        cnt[r] += __popc(gm);
      }
    };

    if constexpr (LABEL) {
      // One key per lane: tiles of 64 keys, one 16-byte label row each
      // (a fully coalesced 1 KB load), scored on the vector ALUs for every
      // row of the group, kLabelDepth tiles in flight.  A row's keys that
      // pass are appended to its area in position order (ballot + prefix
      // count); a row that no key of the tile passes costs one compare.
      // The rows' query sides and thresholds in registers (rows past the
      // group's never pass).
      constexpr int NRr = NR > 0 ? NR : 1;
      // Group-shared: the summed query side in float32; per-head rows: the
      // query's label channels as bf16 pairs (label_dot_packed).
      float qlr[GRP ? NRr : 1][kLabels], thr[NRr];
      uint32_t qpr[GRP ? 1 : NRr][4];
      int cntr[NRr];
#pragma unroll
      for (int h = 0; h < NRr; ++h) {
        cntr[h] = 0;
        if constexpr (GRP) {
          if (h < nrows) q_label_row(p, b, g, -1, qlr[h]);
          else
#pragma unroll
            for (int c = 0; c < kLabels; ++c) qlr[h][c] = 0.f;
        } else {
          if (h < nrows) q_label_row_packed(p, b, g, h, qpr[h]);
          else
#pragma unroll
            for (int e = 0; e < 4; ++e) qpr[h][e] = 0u;
        }
        thr[h] = h < nrows ? w.theta[row0 + h] : __builtin_inff();
      }
      const int nt64 = (nvalid + 63) / 64;
      const int64_t lslab = (((int64_t)b * p.K.hkv + g) * p.K.ncap + w0) * kLabels;
      // (a page's label block is below 2^31 bytes: 32 x 32 -> 64-bit products)
      const uint32_t page_el = (uint32_t)(kTile * p.K.hkv * kLabels);
      const uint32_t head_el = (uint32_t)(g * kTile * kLabels);
      auto lload = [&](int ti) -> u32x4 {
        ti = ti < nt64 ? ti : nt64 - 1;
        int j = ti * 64 + l;
        j = j < last ? j : last;
        const int64_t off = PAGED ? (int64_t)((uint64_t)(uint32_t)pg[j >> 4] * page_el +
                                              (head_el + (uint32_t)(j & 15) * kLabels))
                                  : lslab + (int64_t)j * kLabels;
        return load_labels(p.labels, off);
      };
      const int nlsteps = (nt64 + kLabelDepth - 1) / kLabelDepth * kLabelDepth;
      u32x4 lb[kLabelDepth];
      // The first tiles are issued after the rows' operands and in tile
      // order, so that the loop's first use of a tile waits for that tile
      // only: a load issued after it would make the wait (placed once for
      // the loop's entry and every step) cover every tile in flight.
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int d = 0; d < kLabelDepth; ++d) {
        lb[d] = lload(d);
        __builtin_amdgcn_sched_barrier(0);
      }
      for (int tb = 0; tb < nlsteps; tb += kLabelDepth) {
#pragma unroll
        for (int u = 0; u < kLabelDepth; ++u) {
          const int ti = tb + u;
          // Every row's score of this lane's key first, then the load that
          // reuses the tile's registers: issued before the tile's last use,
          // it would need other registers and a copy back (with a wait for
          // the load) at the end of the step.
          float sc[NRr];
          {
            const u32x4 raw = lb[u];
            float lab[kLabels];
            if constexpr (GRP) unpack_labels(raw, lab);
#pragma unroll
            for (int h = 0; h < NRr; ++h) {
              if constexpr (GRP) sc[h] = label_dot(qlr[h], lab);
              else sc[h] = label_dot_packed(qpr[h], raw);
            }
          }
          __builtin_amdgcn_sched_barrier(0);
          lb[u] = lload(ti + kLabelDepth);
          const int jl = ti * 64 + l;
          const bool live = (jl >= jlo) & (jl < jhi);
          const uint64_t live_m = __builtin_amdgcn_ballot_w64(live);
#pragma unroll
          for (int h = 0; h < NRr; ++h) {
            // In-order entry from the ballot's count of lower lanes, counted
            // from the row's next free entry; lanes that do not pass (or run
            // past the row's area) write their discard slot, so no branch
            // or exec-mask change is needed.  (Ballots of the compares
            // themselves, and no short-circuit: no round trips through
            // vector registers, no masked regions.)
            const bool ge = sc[h] >= thr[h];
            const uint64_t m = __builtin_amdgcn_ballot_w64(ge) & live_m;
            const int at = (int)__builtin_amdgcn_mbcnt_hi(
                (uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, (uint32_t)(h * cap + cntr[h])));
            const bool ok = live & ge & (at < (h + 1) * cap);
            const int e = ok ? at : kCandBuf + l;
            wl.cand[e] = make_uint2(__float_as_uint(sc[h]), (uint32_t)jl);
            cntr[h] += __popcll(m);
          }
        }
      }
      // Counts in the layout the packing below reads: lane group s holds
      // rows 4s..4s+3.
#pragma unroll
      for (int r = 0; r < 4; ++r) {
#pragma unroll
        for (int sg = 0; sg < 4; ++sg)
          if (4 * sg + r < NRr && s == sg) cnt[r] = cntr[4 * sg + r];
      }
    } else {
      const int nsteps = (ntiles + kDepth - 1) / kDepth * kDepth;
      u32x4 buf[kDepth][4];
#pragma unroll
      for (int d = 0; d < kDepth; ++d) {
        load(d, buf[d]);
        __builtin_amdgcn_sched_barrier(0);
      }
      // The scores of a tile are filtered one step later, after the next
      // tile's loads and matrix ops are issued, so the appends (which wait on
      // the matrix results) never hold up the stream.
      f32x4 prev = {0.f, 0.f, 0.f, 0.f};
      int prev_jl = nvalid;  // nothing to filter before the first tile
      for (int tb = 0; tb < nsteps; tb += kDepth) {
#pragma unroll
        for (int u = 0; u < kDepth; ++u) {
          const int ti = tb + u;
          stage_tile(wl.tile, buf[u]);
          load(ti + kDepth, buf[u]);
          __builtin_amdgcn_wave_barrier();  // the tile is read back by other lanes
          KFrag kf;
          read_kfrag(wl.tile, kf);
          __builtin_amdgcn_wave_barrier();  // and overwritten by the next step
          const f32x4 acc = mfma_scores(qf, kf);
          filter(prev, prev_jl);
          prev = acc;
          prev_jl = ti * kTile + col;
        }
      }
      filter(prev, prev_jl);
    }
  }
  if constexpr (QUAD) {
    // This wave's block: its rows one after another, each in position order.
    int *off = sl.seg_off + wv * (kMaxGroup + 1);
    if (col == 0) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int h = 4 * s + r;
        if (h < nrows) sl.seg_n[wv * kMaxGroup + h] = cnt[r];
      }
    }
    __builtin_amdgcn_wave_barrier();  // counts were written by other lanes
    const int n = l < nrows ? sl.seg_n[wv * kMaxGroup + l] : 0;
    const int nc = n < cap ? n : cap;
    const int inc = wave_incl_scan(nc);
    if (l < nrows)
      w.dir[(row0 + l) * w.nchunk + chunk] = make_int2(inc - nc, n > cap ? -1 : nc);
    if (l <= kMaxGroup) off[l] = inc - nc;  // rows >= nrows: the total
    const int ntot = __shfl(inc, 63);
    if (l == 0) sl.wave_tot[wv] = ntot;
    const int64_t blk = ((int64_t)bg * w.nchunk + chunk) * w.blk_cap;
    uint32_t *kdst = w.ckey + blk;
    uint16_t *pdst = w.cpos + blk;
    int base = 0, before = 0, all = 0;
    if (ob) {
      __syncthreads();  // every wave's block size
#pragma unroll
      for (int v = 0; v < kWaves; ++v) {
        const int t = (sl.wave_tot[v] + 3) & ~3;
        before += v < wv ? t : 0;
        all += t;
      }
      base = outbox_reserve(w, *ob, all, kWaves);
      kdst = ob->obk + base + before;
      pdst = ob->obp + base + before;
    } else {
      __builtin_amdgcn_wave_barrier();  // offsets are read by every lane
    }
    for (int i0 = 4 * l; i0 < ntot; i0 += 4 * 64) {
      // Row of item i0: the last t with off[t] <= i0.
      int t = 0;
#pragma unroll
      for (int step = 8; step > 0; step >>= 1)
        if (off[t + step] <= i0) t += step;
      pack4(i0, ntot, [&](int i) {
        while (off[t + 1] <= i) ++t;  // stops at t = 15: off[16] = ntot > i
        return wl.cand[t * cap + (i - off[t])];
      }, kdst, pdst, ob != nullptr);
    }
    if (ob) {
      if (l == 0) {
        ob->dst[ob->nb + wv] = blk;
        ob->off[ob->nb + wv] = base + before;
        ob->cnt[ob->nb + wv] = ntot;
      }
      __syncthreads();  // every wave has read nb
      if (threadIdx.x == 0) {
        ob->nb += kWaves;
        ob->n = base + all;
      }
    }
    return;
  }
  if (col == 0) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int h = 4 * s + r;
      if (h < nrows) sl.seg_n[h * kWaves + wv] = cnt[r];
    }
  }
  __syncthreads();

  // Block layout: segment t = (row t/4, wave t%4), rows in order.
  const int tid = threadIdx.x;
  if (tid < 64) {
    const int h = tid / kWaves;
    const int n = h < nrows ? sl.seg_n[tid] : 0;
    const int nc = n < cap ? n : cap;
    const int inc = wave_incl_scan(nc);
    const int row_end = __shfl(inc, (tid | (kWaves - 1)));
    const uint64_t over = __ballot(n > cap);
    sl.seg_off[tid] = inc - nc;
    if (tid == 63) sl.seg_off[64] = inc;
    if (tid % kWaves == 0 && h < nrows) {
      const int start = inc - nc;
      const bool ovf = ((over >> tid) & ((1ull << kWaves) - 1ull)) != 0;
      w.dir[(row0 + h) * w.nchunk + chunk] = make_int2(start, ovf ? -1 : row_end - start);
    }
  }
  __syncthreads();
  const int ntot = sl.seg_off[64];
  const int64_t blk = ((int64_t)bg * w.nchunk + chunk) * w.blk_cap;
  uint32_t *kdst = w.ckey + blk;
  uint16_t *pdst = w.cpos + blk;
  int base = 0;
  if (ob) {
    base = outbox_reserve(w, *ob, (ntot + 3) & ~3, 1);
    kdst = ob->obk + base;
    pdst = ob->obp + base;
  }
  for (int i0 = 4 * tid; i0 < ntot; i0 += 4 * kBlock) {
    // Segment of item i0: the last t with seg_off[t] <= i0.
    int t = 0;
#pragma unroll
    for (int step = 32; step > 0; step >>= 1)
      if (sl.seg_off[t + step] <= i0) t += step;
    pack4(i0, ntot, [&](int i) {
      while (sl.seg_off[t + 1] <= i) ++t;  // stops at t = 63: seg_off[64] = ntot > i
      const int h = t / kWaves, v = t % kWaves;
      const uint2 it = sl.wave[v].cand[h * cap + (i - sl.seg_off[t])];
      return make_uint2(it.x, (uint32_t)(v * wk) + it.y);
    }, kdst, pdst, ob != nullptr);
  }
  if (ob && tid == 0) {
    ob->dst[ob->nb] = blk;
    ob->off[ob->nb] = base;
    ob->cnt[ob->nb] = ntot;
    ob->nb += 1;
    ob->n = base + ((ntot + 3) & ~3);
  }
}

template <bool PAGED, bool GRP, bool QUAD, bool LABEL, int NR>
__global__ __launch_bounds__(kBlock) void k_score_stream(Params p, Work w) {
  __shared__ StreamLds sl;
  if (!w.persistent) {
    // One unit per workgroup, empty chunks included.  Dispatch order
    // (consecutive workgroups run together): in the paged layout the KV
    // heads of a page block are adjacent in memory, so heads go fastest; in
    // the contiguous layout a head's slab is swept chunk by chunk.
    const int wid = (int)blockIdx.x;
    int chunk, g0, b;
    if (QUAD) {
      const int nq = p.Hkv / kWaves;
      chunk = (wid / nq) % w.nchunk;
      b = wid / (nq * w.nchunk);
      g0 = kWaves * (wid % nq);
    } else if (PAGED) {
      g0 = wid % p.Hkv;
      chunk = (wid / p.Hkv) % w.nchunk;
      b = wid / (p.Hkv * w.nchunk);
    } else {
      chunk = wid % w.nchunk;
      g0 = (wid / w.nchunk) % p.Hkv;
      b = wid / (w.nchunk * p.Hkv);
    }
    stream_unit<PAGED, GRP, QUAD, LABEL, NR>(p, w, b, g0, chunk, sl, nullptr);
    return;
  }
  // Persistent: units from the queue, in the work list's order (sequence by
  // sequence; within one, the same order as the static grid's).
  extern __shared__ u32x4 stream_dyn[];
  Outbox *ob = (Outbox *)stream_dyn;
  static_assert(sizeof(Outbox) % 16 == 0, "outbox arrays stay 16-byte aligned");
  if (threadIdx.x == 0) {
    ob->obk = (uint32_t *)(ob + 1);
    ob->obp = (uint16_t *)(ob->obk + kOutboxCap);
    ob->n = 0;
    ob->nb = 0;
  }
  const int total = w.unit_pre[p.B];
  int b = 0;
  for (;;) {
    if (threadIdx.x == 0) sl.unit = atomicAdd(w.queue, 1);
    __syncthreads();  // the unit, and (first pass) the outbox state
    const int u = sl.unit;
    if (u >= total) break;  // uniform
    while (u >= w.unit_pre[b + 1]) ++b;
    const int r = u - w.unit_pre[b];
    int chunk, g0;
    if (QUAD) {
      const int nq = p.Hkv / kWaves;
      chunk = r / nq;
      g0 = kWaves * (r % nq);
    } else if (PAGED) {
      chunk = r / p.Hkv;
      g0 = r % p.Hkv;
    } else {
      const int nch = (seq_len(p, b) + w.chunk_keys - 1) / w.chunk_keys;
      g0 = r / nch;
      chunk = r % nch;
    }
    stream_unit<PAGED, GRP, QUAD, LABEL, NR>(p, w, b, g0, chunk, sl, ob);
    __syncthreads();  // LDS areas and outbox state are reused by the next unit
  }
  outbox_flush(w, *ob);
}

// ---------------------------------------------------------------------------
// Full scores of one (sequence b, KV head g): part `part` of `parts` takes
// tiles part*4 + wave, stepping by parts*4.  dst[row][j] for j < L_b; with
// fill_tail, -inf for L_b <= j < ncap.  Every thread of the block must call
// it (the f32 scorer stages the queries in LDS behind a barrier).
// ---------------------------------------------------------------------------
// Tiles in flight per wave in the pipelined full scoring: one tile's loads
// are a single round trip (4 KB of keys, or 256 B of label rows).
constexpr int dense_depth(bool label) { return label ? 8 : 3; }

// PIPE: several tiles in flight per wave (a separate instance, launched when
// the waves have enough tiles for it: its registers would cost occupancy to
// the short waves too).
template <bool BF16, bool LABEL, bool PIPE = false>
__device__ __forceinline__ void dense_scores(const Params &p, float *dst, int64_t ld, int b, int g,
                                             int part, int parts, bool fill_tail, float *q_lds) {
  const int L = seq_len(p, b);
  const int64_t row0 = p.group_shared ? (int64_t)b * p.R + g : (int64_t)b * p.R + (int64_t)g * p.G;
  Scorer<BF16, LABEL> sc;
  scorer_init<BF16, LABEL>(p, b, g, sc, q_lds);
  const int64_t end = fill_tail ? p.ncap : (int64_t)L;
  const int64_t ntiles = (end + kTile - 1) / kTile;
  const int l = lane_id(), col = l & 15, s = l >> 4;
  const int64_t t0 = (int64_t)part * kWaves + wave_id(), step = (int64_t)parts * kWaves;
  auto put = [&](int64_t t, f32x4 acc) {
    const int64_t j = t * kTile + col;
    const bool in_seq = j < L;
    const float ninf = -__builtin_inff();
    if (!p.group_shared) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int h = 4 * s + r;
        if (h < p.G && j < end) dst[(row0 + h) * ld + j] = in_seq ? acc[r] : ninf;
      }
    } else {
      const float gs = group_sum(acc);
      if (s == 0 && j < end) dst[row0 * ld + j] = in_seq ? gs : ninf;
    }
  };
  if constexpr ((BF16 || LABEL) && PIPE) {
    // kD tiles in flight per wave (one at a time left the fallback waiting
    // on latency).  Positions past the sequence read its last key again
    // (their scores are replaced by -inf), and the step count is rounded up
    // to whole rounds with clamped loads, so every step issues the same
    // loads and the waits stay exact.  A wave with fewer than two rounds of
    // tiles keeps the plain loop: the rounding and the loads issued past its
    // last tile would cost it more than they hide.
    constexpr int kD = dense_depth(LABEL);
    const int64_t n = t0 < ntiles ? (ntiles - t0 + step - 1) / step : 0;
    if (L > 0 && n >= 2 * kD) {  // wave-uniform
      const int64_t nsteps = (n + kD - 1) / kD * kD;
      auto ld_tile = [&](int64_t i, typename Scorer<BF16, LABEL>::Raw &r) {
        const int64_t j = (t0 + i * step) * kTile + col;
        sc.load(p, b, g, j < L ? j : (int64_t)L - 1, r);
      };
      typename Scorer<BF16, LABEL>::Raw buf[kD];
#pragma unroll
      for (int d = 0; d < kD; ++d) {
        ld_tile(d, buf[d]);
        __builtin_amdgcn_sched_barrier(0);
      }
      for (int64_t i0 = 0; i0 < nsteps; i0 += kD) {
#pragma unroll
        for (int u = 0; u < kD; ++u) {
          const int64_t i = i0 + u;
          // (the tile is scored before the load that reuses its registers)
          const f32x4 acc = sc.from_raw(buf[u]);
          __builtin_amdgcn_sched_barrier(0);
          ld_tile(i + kD, buf[u]);
          const int64_t t = t0 + i * step;
          if (i < n && t * kTile < L) put(t, acc);
          else if (i < n) put(t, f32x4{0.f, 0.f, 0.f, 0.f});
        }
      }
      return;
    }
  }
  for (int64_t t = t0; t < ntiles; t += step) {
    const int64_t j = t * kTile + col;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    if (t * kTile < L) acc = sc.score(p, b, g, j < L ? j : (int64_t)L - 1);
    put(t, acc);
  }
}

// sparse_decode_score: grid = (parts, B*Hkv).
template <bool BF16, bool LABEL, bool PIPE>
__global__ __launch_bounds__(kBlock) void k_score_dense(Params p, float *dst, int64_t ld) {
  __shared__ float q_lds[BF16 ? 1 : kMaxGroup * kHeadDim];
  const int bg = blockIdx.y;
  dense_scores<BF16, LABEL, PIPE>(p, dst, ld, bg / p.Hkv, bg % p.Hkv, blockIdx.x, gridDim.x,
                                  true, q_lds);
}

// Exact fallback, scoring.  grid = (parts, B*Hkv), parts at least
// kRepairParts (repair_parts).  A row takes the
// fallback when every row is forced to, or when its candidates cannot prove
// exactness: fewer than k passed, or a staging area overflowed (a per-chunk
// count of -1).  Each workgroup derives its group's flags from the rows'
// per-chunk counts (part 0 records them in w.flags for the selection) and,
// when a row of the group is flagged, scores its part of the group into
// w.dense.
// LDS of piece_hist.
struct PieceHistLds {
  uint32_t runs[64];
  int pre[kPselChunksMax + 1], start[kPselChunksMax];
  uint32_t kmax;
};

// One piece of a row's candidate selection over several workgroups (defined
// with the selection below).
__device__ __forceinline__ void piece_hist(const Params &p, const Work &w, int row, int piece,
                                           PieceHistLds &sh);

template <bool BF16, bool LABEL, bool PIPE>
__global__ __launch_bounds__(kBlock) void k_repair_score(Params p, Work w) {
  __shared__ float q_lds[BF16 ? 1 : kMaxGroup * kHeadDim];
  __shared__ int cnt[kMaxGroup], bad[kMaxGroup];
  __shared__ int any;
  const int part = blockIdx.x, bg = blockIdx.y, b = bg / p.Hkv, g = bg % p.Hkv;
  const int nrows = p.group_shared ? 1 : p.G;
  const int L = seq_len(p, b);
  const int k = row_plan(p, b, L).kh;
  const int64_t row0 = p.group_shared ? (int64_t)b * p.R + g : (int64_t)b * p.R + (int64_t)g * p.G;
  const int tid = threadIdx.x;
  if (tid < kMaxGroup) {
    cnt[tid] = 0;
    bad[tid] = 0;
  }
  if (tid == 0) any = 0;
  // The multi-workgroup fallback selection's histograms start at zero; with
  // the pilot skipped (every row forced), the repaired-row count too.
  if (w.dsel_parts) {
    uint32_t *gh = w.dsel_hist + row0 * 2048;
    for (int e = part * kBlock + tid; e < nrows * 2048; e += gridDim.x * kBlock) gh[e] = 0u;
  }
  if (w.force_repair && part == 0 && bg == 0 && tid == 0) w.stats[0] = 0;
  __syncthreads();
  if (k > 0 && !w.force_repair) {
    const int ck = w.chunk_keys;
    const int nch = (L + ck - 1) / ck;
    for (int e = tid; e < nrows * nch; e += kBlock) {
      const int r = e / nch;
      const int2 d = w.dir[(row0 + r) * w.nchunk + (e % nch)];
      if (d.y < 0) bad[r] = 1;
      else if (d.y > 0) atomicAdd(&cnt[r], d.y);
    }
  }
  __syncthreads();
  if (tid < nrows) {
    const bool flag = k > 0 && (w.force_repair || bad[tid] || cnt[tid] < k);
    if (flag) any = 1;
    if (part == 0) w.flags[row0 + tid] = flag ? 1 : 0;
  }
  __syncthreads();
  // The pieces of the group's rows (candidate selection over several
  // workgroups per row), one task per workgroup of the group; none when a
  // row of the group is flagged, since the group's full scoring below then
  // writes the score rows the pieces would copy their keys to.
  if (w.psel_parts > 0 && k > 0 && !any) {
    __shared__ PieceHistLds ph;
    for (int t = part; t < nrows * w.psel_parts; t += (int)gridDim.x) {
      const int r = t / w.psel_parts;
      piece_hist(p, w, (int)row0 + r, t % w.psel_parts, ph);
    }
  }
  if (any)
    dense_scores<BF16, LABEL, PIPE>(p, w.dense, p.ncap, b, g, part, (int)gridDim.x, false, q_lds);
}

// ---------------------------------------------------------------------------
// Exact top-k of one row per workgroup.
//   MODE 0: the fused path.  A row flagged for the exact fallback (by
//           k_repair_score) is selected from its full scores in w.dense, any
//           other row from its candidates.
//   MODE 1: over a full score row (sparse_decode_topk).
// Output: idx[row][0..k) ascending positions, then -1; vals[row][...] the
// kept scores (or -inf), when vals is not null.
// ---------------------------------------------------------------------------
struct DenseSrc {
  const float *row;  // scores of positions base, base + 1, ...
  uint32_t base;
  __device__ __forceinline__ uint32_t key(int i) const { return f2key(row[i]); }
  __device__ __forceinline__ uint32_t pos(int i) const { return base + (uint32_t)i; }
};

// The candidates of one row, chunk by chunk: chunk c contributes
// pre[c+1] - pre[c] items stored from offset start[c] of its block.  Keys
// are read from the flat copy (flat[i] = item i's key, in LDS or global
// memory) once flatten_cands has made it; positions from the blocks.
struct ChunkCands {
  const uint32_t *flat;
  const int *pre;        // nch + 1 prefix sums (LDS)
  const int *start;      // nch block offsets (LDS)
  int nch;
  const uint32_t *gkey;  // the group's blocks, cap entries apart
  const uint16_t *gpos;
  int ck;                // keys per chunk
  int cap;               // entries per block
  // Chunk holding item i: the last c with pre[c] <= i (empty chunks share
  // their successor's prefix value, so this is the owner).
  __device__ __forceinline__ int chunk_of(int i) const {
    int lo = 0, hi = nch - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (pre[mid] <= i) lo = mid; else hi = mid - 1;
    }
    return lo;
  }
  __device__ __forceinline__ int64_t slot(int c, int i) const {
    return (int64_t)c * cap + start[c] + (i - pre[c]);
  }
  __device__ __forceinline__ uint32_t key(int i) const { return flat[i]; }
  __device__ __forceinline__ uint32_t pos(int i) const {
    const int c = chunk_of(i);
    return (uint32_t)c * (uint32_t)ck + gpos[slot(c, i)];
  }
};

// Softmax weight of a kept score s against the row's largest kept score:
// exp(scale (s - max s)) = 2^((s - max s) c2) with c2 = scale log2(e), by the
// hardware base-2 exponential.  Every selection path uses this one form, so
// the candidate path and the exact fallback give identical attention.
__device__ __forceinline__ float kept_weight(float s, float smax, float c2) {
  return __builtin_amdgcn_exp2f((s - smax) * c2);
}
__device__ __forceinline__ float weight_factor(float scale) { return scale * 1.44269504088896341f; }

template <int NT = kBlock, class Src>
__device__ __forceinline__ void select_and_write(const Src &src, int n, int k, uint32_t *hist,
                                                 SelShared *sh, int32_t *irow, float *vrow) {
  uint32_t T;
  int need_eq;
  radix_select<NT>(src, n, k, hist, sh, T, need_eq);
  compact_selected<NT>(src, n, k, T, need_eq, sh->scan, [&](int slot, int i, uint32_t key) {
    irow[slot] = (int32_t)src.pos(i);
    if (vrow) vrow[slot] = key2f(key);
  });
}

// Copy the candidates' keys into flat[0, n) in item order, one wave per
// chunk (coalesced reads of the chunk's block, coalesced writes), and widen
// (mn, mx) by the keys this thread copied.
template <int NT>
__device__ __forceinline__ void flatten_cands(const ChunkCands &src, uint32_t *flat,
                                              uint32_t &mn, uint32_t &mx) {
  constexpr int kU = 8;  // loads in flight per lane
  const int lane = lane_id();
  for (int c = wave_id(); c < src.nch; c += NT / 64) {
    const int cnt = src.pre[c + 1] - src.pre[c];
    const uint32_t *from = src.gkey + (int64_t)c * src.cap + src.start[c];
    uint32_t *to = flat + src.pre[c];
    for (int j0 = lane; j0 < cnt; j0 += 64 * kU) {
      uint32_t v[kU];
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        const int j = j0 + u * 64;
        v[u] = j < cnt ? from[j] : 0u;
      }
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        const int j = j0 + u * 64;
        if (j < cnt) {
          to[j] = v[u];
          mn = v[u] < mn ? v[u] : mn;
          mx = v[u] > mx ? v[u] : mx;
        }
      }
    }
  }
}

// Candidates whose keys sit in one flat array (src.flat: LDS, or the row's
// global scratch when they do not fit), kmin..kmax their key range: the
// k-th largest by bucket_kth (radix passes over the key bits when it
// declines).  The compaction then records each kept item's index in place
// of the consumed keys (slot <= item index, and a round reads all its keys
// before its scans) and, when vrow is given, writes the softmax weights
// exp(scale * (s - vmax)) (weights set) or the kept scores; finally every thread fetches
// the positions of its kept items with the loads in flight together.
template <int NT>
__device__ __forceinline__ void select_and_write_staged(const ChunkCands &src, int n, int k,
                                                        uint32_t kmin, uint32_t kmax,
                                                        uint32_t *hist, SelShared *sh,
                                                        BucketShared<NT> *bs, int32_t *irow,
                                                        float *vrow, bool weights, float scale) {
  const int tid = threadIdx.x;
  const float vmax = key2f(kmax);
  uint32_t T;
  int need_eq;
  if (!bucket_kth<NT>(src.flat, n, k, kmin, kmax, hist, sh, bs, T, need_eq))
    radix_select<NT>(src, n, k, hist, sh, T, need_eq);
  uint32_t *stage = const_cast<uint32_t *>(src.flat);
  compact_selected<NT>(src, n, k, T, need_eq, sh->scan, [&](int slot, int i, uint32_t key) {
    stage[slot] = (uint32_t)i;
    if (vrow) {
      const float v = key2f(key);
      vrow[slot] = weights ? kept_weight(v, vmax, weight_factor(scale)) : v;
    }
  });
  __syncthreads();
  constexpr int kP = 8;  // position loads in flight per thread
  for (int s0 = tid; s0 < k; s0 += NT * kP) {
    uint32_t item[kP], pos[kP];
#pragma unroll
    for (int u = 0; u < kP; ++u) {
      const int s = s0 + u * NT;
      item[u] = s < k ? stage[s] : 0u;
    }
#pragma unroll
    for (int u = 0; u < kP; ++u) {
      const int s = s0 + u * NT;
      pos[u] = s < k ? src.pos((int)item[u]) : 0u;
    }
#pragma unroll
    for (int u = 0; u < kP; ++u) {
      const int s = s0 + u * NT;
      if (s < k) irow[s] = (int32_t)pos[u];
    }
  }
}

// ---------------------------------------------------------------------------
// Candidate selection with the keys held in registers, for rows whose n
// candidates fit NT * UMAX register slots and whose positions fit the LDS
// array pos_l.  Wave w takes a contiguous share [i0, i1) of the item order,
// lane l the items i0 + 64 u + l (slot u): every key and position load of
// the row is issued before the first one returns, so the candidates cost one
// memory latency.  The k-th largest key then comes from a bucket histogram
// of the registers (exact three-pass radix over the key bits when a bucket
// holds more than NT keys), and the compaction numbers the kept items with
// wave ballots: in item order, the kept lanes of a slot writing consecutive
// list entries.  hist must be zero on entry; every thread must call it.
// ---------------------------------------------------------------------------
template <int NT>
constexpr int reg_select_slots() { return NT >= 1024 ? 40 : 32; }

// Thread t owns the nb / NT bins [nb - (t+1) nb/NT, nb - t nb/NT), counted
// from the top; the owner of the bin where the count from the top reaches
// krem stores it in sh->digit and the count above it in sh->above.  Ends
// with a barrier.
template <int NT>
__device__ __forceinline__ void find_rank_bin(const uint32_t *hist, int nb, int krem,
                                              SelShared *sh) {
  const int bpt = nb / NT;
  const int hi = nb - (int)threadIdx.x * bpt;
  int mine = 0;
  for (int j = 1; j <= bpt; ++j) mine += (int)hist[hi - j];
  // Exclusive scan of the bin sums over the block.
  const int inc = wave_incl_scan_dpp(mine);
  if (lane_id() == 63) sh->scan[wave_id()] = inc;
  __syncthreads();
  int before = inc - mine;
#pragma unroll
  for (int v = 0; v < NT / 64; ++v) before += v < wave_id() ? sh->scan[v] : 0;
  if (before < krem && krem <= before + mine) {
    int cum = before;
    for (int j = 1; j <= bpt; ++j) {
      const int c = (int)hist[hi - j];
      if (cum + c >= krem) {
        sh->digit = (uint32_t)(hi - j);
        sh->above = cum;
        break;
      }
      cum += c;
    }
  }
  __syncthreads();
}

// p (global memory) as a wave-uniform pointer: scalar registers, so that
// accesses through it take 32-bit lane offsets.
template <class T>
__device__ __forceinline__ __attribute__((address_space(1))) T *uniform_ptr(T *p) {
  const uint64_t a = (uint64_t)(uintptr_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
  return (__attribute__((address_space(1))) T *)(((uint64_t)hi << 32) | lo);
}

// LDS of the register selection besides hist, SelShared and BucketShared.
template <int NT>
struct RegSelShared {
  uint32_t gt[NT / 64], eq[NT / 64];  // per wave: kept keys above T, keys equal to T
  uint32_t wmax[NT / 64];             // per wave: its largest key
  uint32_t sink[64];                  // target of the atomics of lanes without an item
  uint8_t wave[NT];                   // the wave of each key collected in BucketShared
};

// Histogram buckets over keys: bucket b holds the keys lo + [b, b+1) << shift,
// those below lo joining bucket 0 and those past the last bucket the top one.
struct KeyBuckets {
  uint32_t lo;
  int shift;
  // Buckets from lo, with `span` keys to spread over them.
  __device__ __forceinline__ static KeyBuckets make(uint32_t lo, uint32_t span) {
    KeyBuckets kb;
    kb.lo = lo;
    kb.shift = span < (uint32_t)kBuckets ? 0 : (32 - __builtin_clz(span)) - 11;
    return kb;
  }
  __device__ __forceinline__ int of(uint32_t x) const {
    const uint32_t bk = (x > lo ? x - lo : 0u) >> shift;
    return bk < (uint32_t)kBuckets - 1u ? (int)bk : kBuckets - 1;
  }
};

// A wave's contiguous share [i0, i1) of the items [ia, ib): lane l holds the
// items i0 + 64 u + l, slots u < U.
struct RegShare {
  int i0, i1, U;
};
template <int NT>
__device__ __forceinline__ RegShare reg_share(int ia, int ib) {
  constexpr int NW = NT / 64;
  const int n = ib - ia, per = (n + NW - 1) / NW;
  RegShare s;
  s.i0 = ia + min(n, wave_id() * per);
  s.i1 = ia + min(n, wave_id() * per + per);
  s.U = (s.i1 - s.i0 + 63) >> 6;
  return s;
}

// The candidates of a share into registers (key[u]) and their positions
// (chunk base + offset) into pos_l[i - ia].  Every load is issued before the
// first returns; lanes past the share's end repeat its last item (so that no
// branch splits a slot).  Lane j first finds the chunk of the share's item
// i0 + 64 j; a slot within one chunk then takes its chunk and block offset
// from that lane (scalar registers), a slot across chunk boundaries counts
// the boundaries at or below each item.  As the loads land, on_key(key,
// valid) runs for every slot (the first histogram); returns the lane's
// largest key.  sink: 64 LDS words for the atomics of lanes without an item.
template <int UMAX, class OnKey>
__device__ __forceinline__ uint32_t reg_load(const ChunkCands &src, const RegShare &sh, int ia,
                                             uint32_t (&key)[UMAX], uint32_t *pos_l,
                                             uint32_t *sink, OnKey on_key) {
  const int lane = lane_id(), i0 = sh.i0, i1 = sh.i1, U = sh.U;
  int cs = 0, ds = 0;
  if (lane <= U && i1 > i0) {
    cs = src.chunk_of(min(i0 + 64 * lane, i1 - 1));
    ds = cs * src.cap + src.start[cs] - src.pre[cs];
  }
  // The blocks' base addresses are the row's (scalar registers: 32-bit
  // offsets per lane).
  const auto gkey = uniform_ptr(src.gkey);
  const auto gpos = uniform_ptr(src.gpos);
  uint32_t gp[UMAX];
  unroll_for<UMAX>([&](auto uc) {
    constexpr int u = decltype(uc)::value;
    key[u] = 0u;
    gp[u] = 0u;
    if (u < U) {  // wave-uniform
      const int ie = min(i0 + 64 * u + lane, i1 - 1);
      const int cu = __builtin_amdgcn_readlane(cs, u), cn = __builtin_amdgcn_readlane(cs, u + 1);
      int c = cu, d = __builtin_amdgcn_readlane(ds, u);
      if (cn != cu) {  // the slot crosses chunk boundaries: count those at or below ie
        for (int x = cu + 1; x <= cn; ++x) c += src.pre[x] <= ie ? 1 : 0;
        d = c * src.cap + src.start[c] - src.pre[c];
      }
      const uint32_t e = (uint32_t)(d + ie);
      key[u] = gkey[e];
      gp[u] = gpos[e];
      pos_l[ie - ia] = (uint32_t)c * (uint32_t)src.ck;
    }
  });
  uint32_t mx = 0u;
  unroll_for<UMAX>([&](auto uc) {
    constexpr int u = decltype(uc)::value;
    if (u < U) {
      const int i = i0 + 64 * u + lane;
      const bool valid = i < i1;
      const uint32_t x = fresh(key[u]);
      atomicAdd(valid ? &pos_l[i - ia] : &sink[lane], gp[u]);
      on_key(x, valid);
      mx = valid && x > mx ? x : mx;
    }
  });
  return mx;
}

// The kept keys of a share in item order: those above T, and those equal to
// T while fewer than need_eq of them came before (eq_b before the wave).
// Slot sel0 (the wave's first entry) onwards, each slot's kept lanes on
// consecutive list entries; with vrow, the kept scores or (weights) their
// softmax weights against vmax.  Entries at or past k are not written.
// ties: whether the wave holds a key equal to T (else a key is kept iff it
// is above T, and the tie count is skipped).
template <int UMAX>
__device__ __forceinline__ void reg_emit(const uint32_t (&key)[UMAX], const RegShare &sh, int ia,
                                         uint32_t T, int need_eq, int eq_b, int sel0, int k,
                                         bool ties, const uint32_t *pos_l, int32_t *irow,
                                         float *vrow, bool weights, float vmax, float c2) {
  const int lane = lane_id();
  const auto lst = uniform_ptr(irow);
  const auto val = uniform_ptr(vrow);
  auto emit = [&](auto vals, auto wts, auto tie) {
    int eq_run = eq_b, sel_run = sel0;
    unroll_for<UMAX>([&](auto uc) {
      constexpr int u = decltype(uc)::value;
      if (u < sh.U) {
        const int i = sh.i0 + 64 * u + lane;
        const bool valid = i < sh.i1;
        const uint32_t x = fresh(key[u]);
        bool kept = valid && x > T;
        if constexpr (decltype(tie)::value) {
          const uint64_t eqm = __ballot(valid && x == T);
          kept = kept || (valid && x == T && eq_run + lanes_below(eqm) < need_eq);
          eq_run += __popcll(eqm);
        }
        const uint64_t km = __ballot(kept);
        const int s = sel_run + lanes_below(km);
        if (kept && s < k) {
          lst[s] = (int32_t)pos_l[i - ia];
          if constexpr (decltype(vals)::value) {
            const float v = key2f(x);
            val[s] = decltype(wts)::value ? kept_weight(v, vmax, c2) : v;
          }
        }
        sel_run += __popcll(km);
      }
    });
  };
  auto emit_ties = [&](auto vals, auto wts) {
    if (ties) emit(vals, wts, std::true_type{});
    else emit(vals, wts, std::false_type{});
  };
  if (!vrow) emit_ties(std::false_type{}, std::false_type{});
  else if (weights) emit_ties(std::true_type{}, std::true_type{});
  else emit_ties(std::true_type{}, std::false_type{});
}

// Candidate selection of a row by one workgroup, the keys held in registers
// (n <= NT * UMAX, positions in pos_l).  kb_lo <= every candidate key (the
// row's threshold: the candidates passed score >= theta) and kb_hi the key
// of the row's largest pilot sample: the first histogram's buckets cut
// [kb_lo, kb_hi] into equal runs of keys, those above kb_hi joining the top
// one.  The mapping is known before the candidates arrive, so the histogram
// is taken as they do.  One more pass over the registers counts each wave's
// keys above the k-th bucket and collects the bucket's keys (typically a
// few dozen); an exact rank among them gives the threshold key T.  A k-th
// bucket of more than NT keys (rare) falls back to three radix passes over
// the key bits.  hist must be zero on entry; every thread must call it.
template <int NT, int UMAX>
__device__ __forceinline__ void select_regs(const ChunkCands &src, int n, int k, uint32_t kb_lo,
                                            uint32_t kb_hi, uint32_t *pos_l, uint32_t *hist,
                                            SelShared *sh, BucketShared<NT> *bs,
                                            RegSelShared<NT> *rs, int32_t *irow, float *vrow,
                                            bool weights, float scale) {
  constexpr int NW = NT / 64;
  const int lane = lane_id(), wv = wave_id();
  const RegShare shr = reg_share<NT>(0, n);  // U <= UMAX: the caller checked n <= NT * UMAX
  const int i0 = shr.i0, i1 = shr.i1, U = shr.U;
  const KeyBuckets kb = KeyBuckets::make(kb_lo, kb_hi > kb_lo ? kb_hi - kb_lo : 0u);
  if (threadIdx.x == 0) {
    bs->n = 0;
    sh->digit = 0u;  // (in range even if the candidates were fewer than k)
    sh->above = 0;
  }
  // 1-2. The candidates, their positions and the histogram.
  uint32_t key[UMAX];
  uint32_t mx = reg_load<UMAX>(src, shr, 0, key, pos_l, rs->sink, [&](uint32_t x, bool valid) {
    atomicAdd(valid ? &hist[kb.of(x)] : &rs->sink[lane_id()], 1u);
  });
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const uint32_t t = (uint32_t)__shfl_xor((int)mx, o);
    mx = t > mx ? t : mx;
  }
  if (lane == 0) rs->wmax[wv] = mx;
  __syncthreads();
  // 3. The k-th largest key T; need_eq of the keys equal to T are kept.
  find_rank_bin<NT>(hist, kBuckets, k, sh);
  const int bstar = (int)sh->digit;
  const int krem = k - (int)sh->above;
  const int m = (int)hist[bstar];
  uint32_t T;
  int need_eq;
  int gt_b = 0, eq_b = 0;  // kept keys of the waves before this one: above T, equal to T
  bool ties = false;
  if (m <= NT) {
    // Keys above the k-th bucket per wave; the bucket's keys (and waves).
    int gt_w = 0;
    unroll_for<UMAX>([&](auto uc) {
      constexpr int u = decltype(uc)::value;
      if (u < U) {
        const bool valid = i0 + 64 * u + lane < i1;
        const uint32_t x = fresh(key[u]);
        const int bk = kb.of(x);
        gt_w += __popcll(__ballot(valid && bk > bstar));
        if (valid && bk == bstar) {
          const int j = atomicAdd(&bs->n, 1);
          bs->items[j] = x;
          rs->wave[j] = (uint8_t)wv;
        }
      }
    });
    if (lane == 0) rs->gt[wv] = (uint32_t)gt_w;
    __syncthreads();
    if ((int)threadIdx.x < m) {
      const uint32_t x = bs->items[threadIdx.x];
      int gt = 0, ge = 0;
      for (int y = 0; y < m; ++y) {
        const uint32_t v = bs->items[y];
        gt += v > x ? 1 : 0;
        ge += v >= x ? 1 : 0;
      }
      if (gt < krem && krem <= ge) {  // x is the krem-th largest (equal keys agree)
        sh->digit = x;
        sh->above = gt;
      }
    }
    __syncthreads();
    T = sh->digit;
    need_eq = krem - (int)sh->above;
    // The bucket's keys of the waves before this one (above T, equal to
    // T), and whether this wave holds a key equal to T.
    for (int j0 = 0; j0 < m; j0 += 64) {
      const int j = j0 + lane;
      const bool in = j < m;
      const uint32_t x = in ? bs->items[j] : 0u;
      const int v = in ? (int)rs->wave[j] : NW;
      gt_b += __popcll(__ballot(in && v < wv && x > T));
      eq_b += __popcll(__ballot(in && v < wv && x == T));
      ties = ties || __ballot(in && v == wv && x == T) != 0;
    }
  } else {  // three radix passes over 11, 11 and 10 key bits
    uint32_t prefix = 0, mask = 0;
    int kr = k;
#pragma unroll 1
    for (int pass = 0; pass < 3; ++pass) {
      const int sft = pass == 0 ? 21 : (pass == 1 ? 10 : 0);
      const int nb = pass == 2 ? 1024 : 2048;
      const uint32_t dmask = (uint32_t)nb - 1u;
      __syncthreads();  // the previous readers of hist and sh are done
      for (int j = threadIdx.x; j < nb; j += NT) hist[j] = 0;
      __syncthreads();
      unroll_for<UMAX>([&](auto uc) {
        constexpr int u = decltype(uc)::value;
        if (u < U) {
          const uint32_t x = fresh(key[u]);
          hist_add(hist, (x >> sft) & dmask, i0 + 64 * u + lane < i1 && (x & mask) == prefix);
        }
      });
      __syncthreads();
      find_rank_bin<NT>(hist, nb, kr, sh);
      prefix |= sh->digit << sft;
      mask |= dmask << sft;
      kr -= (int)sh->above;
    }
    T = prefix;
    need_eq = kr;
    int gt_w = 0, eq_w = 0;
    unroll_for<UMAX>([&](auto uc) {
      constexpr int u = decltype(uc)::value;
      if (u < U) {
        const bool valid = i0 + 64 * u + lane < i1;
        const uint32_t x = fresh(key[u]);
        gt_w += __popcll(__ballot(valid && x > T));
        eq_w += __popcll(__ballot(valid && x == T));
      }
    });
    if (lane == 0) {
      rs->gt[wv] = (uint32_t)gt_w;
      rs->eq[wv] = (uint32_t)eq_w;
    }
    __syncthreads();
#pragma unroll
    for (int v = 0; v < NW; ++v)
      if (v < wv) eq_b += (int)rs->eq[v];
    ties = eq_w > 0;
  }
  // 4. Each wave's first list slot (the kept keys of the waves before it),
  // then its kept keys in item order.
  uint32_t kmax = 0u;
#pragma unroll
  for (int v = 0; v < NW; ++v) {
    if (v < wv) gt_b += (int)rs->gt[v];
    kmax = rs->wmax[v] > kmax ? rs->wmax[v] : kmax;
  }
  reg_emit<UMAX>(key, shr, 0, T, need_eq, eq_b, gt_b + min(eq_b, need_eq), k, ties, pos_l, irow,
                 vrow, weights, key2f(kmax), weight_factor(scale));
}

// Per-head rows of the fused path: turn the kept scores (vrow[0..k), written
// by this workgroup) into softmax weights exp(scale*(s - max s)) in place, so
// that the attention is a plain weighted gather whose splits all share one
// reference maximum.
template <int NT = kBlock>
__device__ __forceinline__ void kept_scores_to_weights(float *vrow, int k, float scale, float *ftmp) {
  __syncthreads();  // vrow was written by other threads of the block
  float m = -__builtin_inff();
  for (int i = threadIdx.x; i < k; i += NT) m = fmaxf(m, vrow[i]);
  m = block_max<NT>(m, ftmp);
  const float c2 = weight_factor(scale);
  for (int i = threadIdx.x; i < k; i += NT) vrow[i] = kept_weight(vrow[i], m, c2);
}

// ---------------------------------------------------------------------------
// Candidate selection of few rows over several workgroups each (rows too few
// to fill the GPU one workgroup each).  A row's chunks are cut into
// w.psel_parts pieces of consecutive chunks.  The value buckets are those of
// select_regs (equal runs of keys from the row's threshold to its largest
// pilot sample, known before the candidates), taken 32 at a time as "runs".
//
// piece_hist (in k_repair_score's launch, which settles the rows' flags):
// each piece counts its candidates per run, writes the counts,
// its candidate count and its largest key to its record, and copies its
// keys grouped by run, the highest run first, into the row's fallback score
// row from position c0 * chunk_keys (c0 its first chunk).  An unflagged row
// does not use that row, and a piece's candidates are distinct positions of
// its chunks, so the copy stays inside it.
//
// k_select then runs one workgroup per piece (piece_select): each sums the
// pieces' run counts to find the run holding the k-th largest key, loads
// that run's keys from every piece's copy (piece j's start there: its count
// above the run) while its own candidates load, counts them per bucket for
// the k-th bucket, ranks that bucket's keys for the threshold key T and the
// number of keys equal to T that are kept, and writes its own kept
// candidates in position order at the offset the pieces before it leave
// (keys equal to T kept in position order across pieces).  The list is the
// one a single workgroup writes.  Two dependent rounds of global loads,
// where a single workgroup takes passes over all of a row's candidates.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int piece_chunk(int nch, int parts, int j) {
  return (int)((int64_t)j * nch / parts);
}

// The chunks [c0, c0 + nc) of a row: prefix sums of their candidate counts
// (pre, nc + 1 entries) and their first block entries (start).  Run by the
// block's first wave (nc <= 64).
__device__ __forceinline__ void piece_directory(const Work &w, int row, int c0, int nc, int *pre,
                                                int *start) {
  const int lane = (int)threadIdx.x;
  const int2 d = lane < nc ? w.dir[(int64_t)row * w.nchunk + c0 + lane] : make_int2(0, 0);
  const int v = d.y > 0 ? d.y : 0;
  const int inc = wave_incl_scan_dpp(v);
  if (lane < nc) {
    pre[lane] = inc - v;
    start[lane] = d.x;
  }
  if (lane == 63) pre[nc] = inc;
}

// Piece `piece` of an unflagged row with a positive budget: its record and
// its run-grouped copy (see above).  Every thread of the block must call it
// (kBlock threads).
__device__ __forceinline__ void piece_hist(const Params &p, const Work &w, int row, int piece,
                                           PieceHistLds &sh) {
  static_assert(kPselStride >= 66 && kBuckets == 64 * 32, "piece record: 64 runs of 32 buckets");
  const int parts = w.psel_parts;
  const int b = row / p.R;
  const int L = seq_len(p, b);
  const int tid = threadIdx.x;
  const int ck = w.chunk_keys;
  const int nch = (L + ck - 1) / ck;
  const int c0 = piece_chunk(nch, parts, piece);
  const int nc = piece_chunk(nch, parts, piece + 1) - c0;  // <= kPselChunksMax (host)
  __syncthreads();  // (sh's previous readers are done)
  if (tid < 64) {
    sh.runs[tid] = 0u;
    if (tid == 0) sh.kmax = 0u;
    piece_directory(w, row, c0, nc, sh.pre, sh.start);
  }
  __syncthreads();
  const int n = sh.pre[nc];
  uint32_t *rec = w.psel_rec + ((int64_t)row * parts + piece) * kPselStride;
  if (n > kPselItemsMax) {  // the row goes back to one workgroup: its count is all it needs
    if (tid == 0) rec[64] = (uint32_t)n;
    return;
  }
  const int rr = row % p.R;
  const int g = p.group_shared ? rr : rr / p.G;
  const int64_t gblk = (((int64_t)b * p.Hkv + g) * w.nchunk + c0) * w.blk_cap;
  const ChunkCands src{nullptr, sh.pre, sh.start, nc, w.ckey + gblk, w.cpos + gblk, ck, w.blk_cap};
  const uint32_t lo = f2key(w.theta[row]), hi = f2key(w.smax[row]);
  const KeyBuckets kb = KeyBuckets::make(lo, hi > lo ? hi - lo : 0u);
  constexpr int kBatch = kBlock * kSelU;
  auto load_keys = [&](int base, uint32_t (&key)[kSelU]) {
#pragma unroll
    for (int u = 0; u < kSelU; ++u) {
      const int i = base + u * kBlock + tid;
      key[u] = i < n ? src.gkey[src.slot(src.chunk_of(i), i)] : 0u;
    }
  };
  // The first batch stays in registers for the copy.
  uint32_t key0[kSelU];
  load_keys(0, key0);
  uint32_t mx = 0u;
  auto count = [&](int base, const uint32_t (&key)[kSelU]) {
#pragma unroll
    for (int u = 0; u < kSelU; ++u)
      if (base + u * kBlock + tid < n) {
        atomicAdd(&sh.runs[kb.of(key[u]) >> 5], 1u);
        mx = key[u] > mx ? key[u] : mx;
      }
  };
  count(0, key0);
  for (int base = kBatch; base < n; base += kBatch) {
    uint32_t key[kSelU];
    load_keys(base, key);
    count(base, key);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const uint32_t t = (uint32_t)__shfl_xor((int)mx, o);
    mx = t > mx ? t : mx;
  }
  if (lane_id() == 0) atomicMax(&sh.kmax, mx);
  __syncthreads();
  // The record; then each run's first slot in the copy, from the top run.
  if (tid < 64) {
    const uint32_t c = sh.runs[63 - tid];
    rec[63 - tid] = c;
    if (tid == 0) {
      rec[64] = (uint32_t)n;
      rec[65] = sh.kmax;
    }
    const int inc = wave_incl_scan_dpp((int)c);
    sh.runs[63 - tid] = (uint32_t)inc - c;
  }
  __syncthreads();
  uint32_t *copy = (uint32_t *)(w.dense + (int64_t)row * p.ncap) + (int64_t)c0 * ck;
  auto scatter = [&](int base, const uint32_t (&key)[kSelU]) {
#pragma unroll
    for (int u = 0; u < kSelU; ++u)
      if (base + u * kBlock + tid < n) copy[atomicAdd(&sh.runs[kb.of(key[u]) >> 5], 1u)] = key[u];
  };
  scatter(0, key0);
  for (int base = kBatch; base < n; base += kBatch) {
    uint32_t key[kSelU];
    load_keys(base, key);
    scatter(base, key);
  }
}

// Dynamic LDS of piece_select (NT threads).
constexpr size_t psel_lds_bytes(int NT) {
  return (size_t)(16 + kPselPartsMax * 64 + 64 + 2 * kPselPartsMax + 1 + 32 + 2 * kPselChunksMax + 1 +
                  2 * kPselRunMax + NT * kPselSlots) * 4 +
         (size_t)kPselRunMax;
}

// Piece blockIdx.y of a row's candidate selection over w.psel_parts
// workgroups (see piece_hist).  Returns false, having written nothing, when
// the row is better selected by one workgroup: a piece holds more than
// kPselItemsMax candidates (its record then holds its count alone), the
// k-th run more than kPselRunMax keys, a row of its KV group is flagged,
// or the candidates are fewer than k.  Every piece decides this before any
// of them reads another's copy, so the row's first piece, selecting it
// alone, may then use the row's score row as scratch.  hist, sh: the
// selection's LDS (the radix passes of a crowded k-th bucket).  Every
// thread must call it.
template <int NT>
__device__ __forceinline__ bool piece_select(const Params &p, const Work &w, int row, int L, int k,
                                             int32_t *irow, float *vrow, bool weights,
                                             uint32_t *dyn, uint32_t *hist, SelShared *sh,
                                             RegSelShared<NT> *rs) {
  constexpr int NW = NT / 64;
  const int P = w.psel_parts, piece = (int)blockIdx.y;
  const int tid = threadIdx.x, lane = lane_id(), wv = wave_id();
  int *ctl = (int *)dyn;                            // 16 words, below
  uint32_t *suf = dyn + 16;                         // [P][64] counts from the top run down
  uint32_t *colsum = suf + kPselPartsMax * 64;      // [64] run counts of the row
  int *aq = (int *)(colsum + 64);                   // [P] candidates above the k-th run
  int *ro = aq + kPselPartsMax;                     // [P + 1] k-th run's keys before the piece
  uint32_t *fh = (uint32_t *)(ro + kPselPartsMax + 1);  // [32] the run's bucket counts
  int *pre = (int *)(fh + 32);                      // [kPselChunksMax + 1]
  int *start = pre + kPselChunksMax + 1;            // [kPselChunksMax]
  uint32_t *runk = (uint32_t *)(start + kPselChunksMax);  // [kPselRunMax] the run's keys
  uint32_t *bkeys = runk + kPselRunMax;             // [kPselRunMax] the k-th bucket's keys
  uint32_t *pos_l = bkeys + kPselRunMax;            // [NT * kPselSlots] own positions
  uint8_t *runq = (uint8_t *)(pos_l + NT * kPselSlots);  // [kPselRunMax] their pieces
  enum { kRun, kAboveRun, kKmax, kR, kOk, kBstar, kKrem, kM, kT, kAboveT, kGtBefore, kEqBefore, kNb };
  const uint32_t *rec0 = w.psel_rec + (int64_t)row * P * kPselStride;
  const int ck = w.chunk_keys;
  const int nch = (L + ck - 1) / ck;
  const int c0 = piece_chunk(nch, P, piece);
  const int nc = piece_chunk(nch, P, piece + 1) - c0;
  const uint32_t lo = f2key(w.theta[row]), hi = f2key(w.smax[row]);
  const KeyBuckets kb = KeyBuckets::make(lo, hi > lo ? hi - lo : 0u);
  auto give_up = [&]() {
    __syncthreads();  // (the caller reuses this LDS)
    return false;
  };
  // 1. The own chunks' directory; every piece's run counts (per piece, the
  // counts from the top run down to each run: one wave per piece, lane l on
  // run 63 - l), their sums over the pieces, each piece's candidate count
  // and largest key.
  static_assert(kPselPartsMax * 64 <= 2 * NT, "two pieces per wave at most");
  static_assert(NT * kPselSlots == kPselItemsMax, "a piece's candidates fit the registers");
  uint32_t c2[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int q = wv + h * NW;
    c2[h] = q < P ? rec0[(int64_t)q * kPselStride + 63 - lane] : 0u;
  }
  int nv = 0;
  uint32_t kv = 0u;
  if (tid < P) {
    nv = (int)rec0[(int64_t)tid * kPselStride + 64];
    kv = rec0[(int64_t)tid * kPselStride + 65];
  }
  // The rows of the KV group: with one of them flagged, the pieces of the
  // group wrote nothing (the repair's full scoring of the group takes their
  // copy space), and the row goes back to one workgroup.
  const int grows = p.group_shared ? 1 : p.G;
  const int64_t grow0 = (int64_t)(row / p.R) * p.R + (p.group_shared ? row % p.R : (row % p.R) / p.G * p.G);
  const int gflag = tid < grows ? w.flags[grow0 + tid] : 0;
  if (wv == 0) {
    piece_directory(w, row, c0, nc, pre, start);
    colsum[lane] = 0u;
  }
  __syncthreads();
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int q = wv + h * NW;
    if (q < P) {
      suf[q * 64 + 63 - lane] = (uint32_t)wave_incl_scan_dpp((int)c2[h]);
      atomicAdd(&colsum[63 - lane], c2[h]);
    }
  }
  __syncthreads();
  // 2. The run holding the k-th largest key (first wave, lane l on run
  // 63 - l); each piece's candidates above it and the run's keys before it.
  if (wv == 0) {
    int nmax = nv, ntot = nv;
    uint32_t km = kv;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const int a = __shfl_xor(nmax, o);
      nmax = a > nmax ? a : nmax;
      ntot += __shfl_xor(ntot, o);
      const uint32_t t = (uint32_t)__shfl_xor((int)km, o);
      km = t > km ? t : km;
    }
    const uint32_t v = colsum[63 - lane];
    const int inc = wave_incl_scan_dpp((int)v);
    const uint64_t hit = __ballot(inc >= k);
    const bool ok = nmax <= kPselItemsMax && ntot >= k && hit != 0 && __ballot(gflag != 0) == 0;
    const int l = hit ? __ffsll((unsigned long long)hit) - 1 : 0;
    const int run = 63 - l;
    const int above_run = __builtin_amdgcn_readlane(inc - (int)v, l);
    int above = 0, rq = 0;
    if (lane < P) {
      above = run < 63 ? (int)suf[lane * 64 + run + 1] : 0;
      rq = (int)suf[lane * 64 + run] - above;
      aq[lane] = above;
    }
    const int ri = wave_incl_scan_dpp(rq);
    if (lane < P) ro[lane] = ri - rq;
    if (lane < 32) fh[lane] = 0u;
    if (lane == 63) {
      ro[P] = ri;
      ctl[kR] = ri;
    }
    if (lane == 0) {
      ctl[kOk] = ok ? 1 : 0;
      ctl[kRun] = run;
      ctl[kAboveRun] = above_run;
      ctl[kKmax] = (int)km;
      ctl[kNb] = 0;
      ctl[kGtBefore] = 0;
      ctl[kEqBefore] = 0;
    }
  }
  __syncthreads();
  const int R = ctl[kR], run = ctl[kRun];
  if (!ctl[kOk] || R > kPselRunMax) return give_up();
  // 3. The run's keys from the pieces' copies, while the own candidates
  // load; the run's bucket counts.
  const float *drow = w.dense + (int64_t)row * p.ncap;
  constexpr int kRunU = kPselRunMax / NT;
  uint32_t rk[kRunU];
  int rqi[kRunU];
#pragma unroll
  for (int u = 0; u < kRunU; ++u) {
    const int i = u * NT + tid;
    rk[u] = 0u;
    rqi[u] = 0;
    if (i < R) {
      int q = 0, qh = P - 1;  // the last piece whose run keys start at or before i
      while (q < qh) {
        const int mid = (q + qh + 1) >> 1;
        if (ro[mid] <= i) q = mid; else qh = mid - 1;
      }
      rqi[u] = q;
      rk[u] = ((const uint32_t *)drow)[(int64_t)piece_chunk(nch, P, q) * ck + aq[q] + (i - ro[q])];
    }
  }
  const int n_own = pre[nc];
  const int rr = row % p.R;
  const int g = p.group_shared ? rr : rr / p.G;
  const int64_t gblk = (((int64_t)(row / p.R) * p.Hkv + g) * w.nchunk + c0) * w.blk_cap;
  const ChunkCands src{nullptr, pre, start, nc, w.ckey + gblk, w.cpos + gblk, ck, w.blk_cap};
  const RegShare shr = reg_share<NT>(0, n_own);
  uint32_t key[kPselSlots];
  reg_load<kPselSlots>(src, shr, 0, key, pos_l, rs->sink, [](uint32_t, bool) {});
#pragma unroll
  for (int u = 0; u < kRunU; ++u) {
    const int i = u * NT + tid;
    if (i < R) {
      runk[i] = rk[u];
      runq[i] = (uint8_t)rqi[u];
      atomicAdd(&fh[kb.of(rk[u]) - run * 32], 1u);
    }
  }
  __syncthreads();
  // 4. The k-th bucket (first wave, lane j summing bucket 31 - j of the run).
  if (wv == 0) {
    const uint32_t v = lane < 32 ? fh[31 - lane] : 0u;
    const int inc = wave_incl_scan_dpp((int)v) + ctl[kAboveRun];
    const uint64_t hit = __ballot(lane < 32 && inc >= k);
    const int l = __ffsll((unsigned long long)hit) - 1;
    if (lane == l) {
      ctl[kBstar] = run * 32 + 31 - l;
      ctl[kKrem] = k - (inc - (int)v);
      ctl[kM] = (int)v;
    }
  }
  __syncthreads();
  const int bstar = ctl[kBstar], krem = ctl[kKrem], m = ctl[kM];  // m <= R
  // 5. The k-th bucket's keys; the own positions become row positions.
  for (int i = tid; i < R; i += NT) {
    const uint32_t x = runk[i];
    if (kb.of(x) == bstar) bkeys[atomicAdd(&ctl[kNb], 1)] = x;
  }
  for (int i = tid; i < n_own; i += NT) pos_l[i] += (uint32_t)(c0 * ck);
  __syncthreads();
  // 6. The krem-th largest of them: T (equal keys agree), by an exact rank
  // count, or by three radix passes over the key bits when the bucket holds
  // more keys than the workgroup has threads.
  if (m <= NT) {
    if (tid < m) {
      const uint32_t x = bkeys[tid];
      int gt = 0, ge = 0;
      for (int y = 0; y < m; ++y) {
        const uint32_t v = bkeys[y];
        gt += v > x ? 1 : 0;
        ge += v >= x ? 1 : 0;
      }
      if (gt < krem && krem <= ge) {
        ctl[kT] = (int)x;
        ctl[kAboveT] = gt;
      }
    }
  } else {
    uint32_t t;
    int eq;
    radix_select<NT>(LdsKeys{bkeys}, m, krem, hist, sh, t, eq);
    if (tid == 0) {
      ctl[kT] = (int)t;
      ctl[kAboveT] = krem - eq;
    }
  }
  __syncthreads();
  const uint32_t T = (uint32_t)ctl[kT];
  const int need_eq = krem - ctl[kAboveT];
  // 7. Kept keys before this piece (above T, equal to T: the pieces'
  // candidates above the run, and the run's keys) and before each wave.
  {
    int gt_p = tid < piece ? aq[tid] : 0, eq_p = 0;
    for (int i = tid; i < R; i += NT) {
      const uint32_t x = runk[i];
      const bool before = (int)runq[i] < piece;
      gt_p += before && x > T ? 1 : 0;
      eq_p += before && x == T ? 1 : 0;
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      gt_p += __shfl_xor(gt_p, o);
      eq_p += __shfl_xor(eq_p, o);
    }
    if (lane == 0 && (gt_p | eq_p)) {
      atomicAdd(&ctl[kGtBefore], gt_p);
      atomicAdd(&ctl[kEqBefore], eq_p);
    }
  }
  int gt_w = 0, eq_w = 0;
  unroll_for<kPselSlots>([&](auto uc) {
    constexpr int u = decltype(uc)::value;
    if (u < shr.U) {
      const bool valid = shr.i0 + 64 * u + lane < shr.i1;
      const uint32_t x = fresh(key[u]);
      gt_w += __popcll(__ballot(valid && x > T));
      eq_w += __popcll(__ballot(valid && x == T));
    }
  });
  if (lane == 0) {
    rs->gt[wv] = (uint32_t)gt_w;
    rs->eq[wv] = (uint32_t)eq_w;
  }
  __syncthreads();
  int gt_b = ctl[kGtBefore], eq_b = ctl[kEqBefore];
#pragma unroll
  for (int v = 0; v < NW; ++v)
    if (v < wv) {
      gt_b += (int)rs->gt[v];
      eq_b += (int)rs->eq[v];
    }
  // 8. The own kept keys in position order.
  reg_emit<kPselSlots>(key, shr, 0, T, need_eq, eq_b, gt_b + min(eq_b, need_eq), k, eq_w > 0,
                       pos_l, irow, vrow, weights, key2f((uint32_t)ctl[kKmax]),
                       weight_factor(p.scale));
  return true;
}

// NT threads per workgroup: 256, or 1024 when the rows are too few to fill
// the GPU one workgroup each (every per-thread loop is then 4x shorter).
// PIECES: the launch has w.psel_parts workgroups per row (gridDim.y), and
// rows it can select in pieces are (a separate instance, so that the
// one-workgroup instances keep their register allocation).
template <int MODE, int NT, bool PIECES = false>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(4))) void k_select(Params p, Work w, const float *dense, int64_t ld,
                                               int32_t *idx, float *vals, int lds_cap) {
  extern __shared__ uint32_t dyn[];
  __shared__ uint32_t hist[2048];
  __shared__ SelShared sh;
  __shared__ float ftmp[NT / 64];
  __shared__ uint32_t range[NT / 64][2];
  __shared__ BucketShared<NT> bs;
  __shared__ RegSelShared<NT> rsh;
  bool weights_done = false;
  const int row = MODE == 0 ? ordered_row(w, (int)blockIdx.x, p.R) : (int)blockIdx.x;
  const int b = row / p.R;
  const int L = seq_len(p, b);
  // The row's list: its forced sinks, the exact top-k of [lo, hi), then its
  // forced local window.
  const RowPlan rp = row_plan(p, b, L);
  const bool forced = rp.ns + rp.nl > 0;
  const bool weights = MODE != 1 && !p.group_shared && !forced && vals != nullptr;
  const int k = rp.kh;
  const int64_t ist = p.idx_stride > 0 ? p.idx_stride : p.k_max;  // list row stride
  int32_t *lrow = idx + (int64_t)row * ist;
  float *lvals = vals ? vals + (int64_t)row * p.k_max : nullptr;
  int32_t *irow = lrow + rp.ns;
  float *vrow = lvals ? lvals + rp.ns : nullptr;
  const int tid = threadIdx.x;
  if (k > 0) {
    if (MODE == 0 && w.flags[row]) {  // the exact fallback: full scores
      if (blockIdx.y > 0) return;  // (one workgroup per row)
      if (tid == 0) atomicAdd(&w.stats[0], 1);
      if (!w.dsel_parts)  // (else the k_dsel kernels wrote the selection)
        select_and_write<NT>(DenseSrc{w.dense + (int64_t)row * p.ncap + rp.lo, (uint32_t)rp.lo},
                             rp.hi - rp.lo, k, hist, &sh, irow, vrow);
    } else if (MODE == 0 && [&] {
                 if constexpr (PIECES)
                   return piece_select<NT>(p, w, row, L, k, irow, vrow, weights, dyn, hist, &sh,
                                           &rsh);
                 return false;
               }()) {
      weights_done = true;  // (the pieces wrote weights when they were asked for)
    } else if (MODE == 0) {
      if (blockIdx.y > 0) return;  // the row is selected by its first piece alone
      // Candidates: at least k of them and no overflow (else flagged).
      const int ck = w.chunk_keys;
      const int nch = (L + ck - 1) / ck;
      const int rr = row % p.R;
      const int g = p.group_shared ? rr : rr / p.G;
      int *pre = (int *)dyn;          // nch + 1
      int *start = pre + (nch + 1);   // nch
      uint32_t *lkey = (uint32_t *)(start + nch);  // lds_cap keys
      const int2 *drow = w.dir + (int64_t)row * w.nchunk;
      for (int i = tid; i < kBuckets; i += NT) hist[i] = 0;  // (published by the scan's barriers)
      int carry = 0;
      for (int base = 0; base < nch; base += NT) {
        const int c = base + tid;
        const int2 d = c < nch ? drow[c] : make_int2(0, 0);
        int tot;
        const int e = block_excl_scan<NT>(d.y > 0 ? d.y : 0, sh.scan, &tot);
        if (c < nch) {
          pre[c] = carry + e;
          start[c] = d.x;
        }
        carry += tot;
      }
      if (tid == 0) pre[nch] = carry;
      __syncthreads();
      const int total = carry;
      const int64_t gblk = ((int64_t)b * p.Hkv + g) * w.nchunk * w.blk_cap;
      ChunkCands src{nullptr, pre, start, nch, w.ckey + gblk, w.cpos + gblk, ck, w.blk_cap};
      constexpr int kSlots = reg_select_slots<NT>();
      if (total <= lds_cap && total <= NT * kSlots && (int64_t)nch * w.blk_cap <= INT32_MAX) {
        select_regs<NT, kSlots>(src, total, k, f2key(w.theta[row]), f2key(w.smax[row]), lkey,
                                hist, &sh, &bs, &rsh, irow, vrow, weights, p.scale);
        weights_done = true;
      } else {
      // The flat copy goes to LDS when it fits, else to the row's fallback
      // score row, which an unflagged row does not use (the candidates are
      // distinct positions of [lo, hi), so total <= ncap).
      uint32_t *flat = total <= lds_cap ? lkey : (uint32_t *)(w.dense + (int64_t)row * p.ncap);
      uint32_t mn = 0xFFFFFFFFu, mx = 0u;
      flatten_cands<NT>(src, flat, mn, mx);
      block_key_range<NT>(mn, mx, range);  // its barrier publishes the copy
      src.flat = flat;
      select_and_write_staged<NT>(src, total, k, mn, mx, hist, &sh, &bs, irow, vrow, weights,
                                  p.scale);
      weights_done = true;
      }
    } else {
      select_and_write<NT>(DenseSrc{dense + (int64_t)row * ld + rp.lo, (uint32_t)rp.lo},
                           rp.hi - rp.lo, k, hist, &sh, irow, vrow);
    }
    if (weights && !weights_done) kept_scores_to_weights<NT>(vrow, k, p.scale, ftmp);
  }
  if (blockIdx.y > 0) return;  // (the rest of the list: the row's first piece)
  // Forced positions (their scores, for the stand-alone selection), then
  // the padding.
  for (int i = tid; i < rp.ns + rp.nl; i += NT) {
    const int slot = i < rp.ns ? i : rp.ns + k + (i - rp.ns);
    const int pos = i < rp.ns ? i : rp.hi + (i - rp.ns);
    lrow[slot] = pos;
    if (lvals) lvals[slot] = MODE == 1 ? dense[(int64_t)row * ld + pos] : 0.f;
  }
  for (int i = rp.total + tid; i < ist; i += NT) lrow[i] = -1;
  if (lvals)
    for (int i = rp.total + tid; i < p.k_max; i += NT) lvals[i] = -__builtin_inff();
  if (MODE == 0 && w.ustart) {
    // Union attention: where each chunk of union_chunk positions begins in
    // this row's (ascending) list; entry `total` closes the last chunk.
    __syncthreads();  // the list was written by every thread of the block
    const int uc = w.union_chunk;
    const int nck = (L + uc - 1) / uc;
    int32_t *us = w.ustart + (int64_t)row * w.ustride;
    for (int i = tid; i <= rp.total; i += NT) {
      const int cur = i < rp.total ? lrow[i] / uc : nck;
      const int prev = i > 0 ? lrow[i - 1] / uc : -1;
      for (int c = prev + 1; c <= cur; ++c) us[c] = i;
    }
  }
}

// ---------------------------------------------------------------------------
// Exact fallback selection over several workgroups per row, for calls whose
// every row takes the fallback while the rows are too few to fill the GPU
// one workgroup each.  A row's full scores (w.dense over its top-k range
// [lo, hi)) are cut into gridDim.x consecutive pieces.  Three rounds fix the
// k-th largest key 11, 11 and 10 bits at a time (the digits of
// radix_select): in each, every piece adds the histogram of its keys that
// match the bits fixed so far into the row's global histogram
// (k_dsel_hist), and one workgroup per row picks the digit holding the
// remaining rank and clears the histogram for the next round
// (k_dsel_digit).  Each piece then counts its keys above and equal to the
// threshold T (k_dsel_count) and writes its kept positions and scores, in
// position order, at the offset the pieces before it leave (k_dsel_write);
// keys equal to T are kept in position order up to the rank left over, so
// the list is the one a single workgroup would write.  k_select then adds
// the rest of each row's list (weights, forced positions, padding).
// grid = (pieces, B*R) for the piece kernels, B*R for k_dsel_digit.
// ---------------------------------------------------------------------------
struct DselPiece {
  const float *src;  // the row's scores from position lo
  int i0, i1;        // the piece: items [i0, i1) of the top-k range
  int k;             // the row's top-k budget (0: nothing to select)
};

__device__ __forceinline__ DselPiece dsel_piece(const Params &p, const Work &w, int row, int q,
                                                int parts) {
  const int b = row / p.R;
  const RowPlan rp = row_plan(p, b, seq_len(p, b));
  const int64_t n = rp.hi - rp.lo;
  DselPiece d;
  d.src = w.dense + (int64_t)row * p.ncap + rp.lo;
  d.i0 = (int)(n * q / parts);
  d.i1 = (int)(n * (q + 1) / parts);
  d.k = w.flags[row] ? rp.kh : 0;
  return d;
}

template <int PASS>
__global__ __launch_bounds__(kBlock) void k_dsel_hist(Params p, Work w) {
  __shared__ uint32_t hist[2048];
  const int row = blockIdx.y;
  const DselPiece d = dsel_piece(p, w, row, blockIdx.x, gridDim.x);
  if (d.k == 0) return;  // whole workgroup
  constexpr int shift = PASS == 0 ? 21 : (PASS == 1 ? 10 : 0);
  constexpr int nb = PASS == 2 ? 1024 : 2048;
  constexpr uint32_t dmask = (uint32_t)nb - 1u;
  const uint32_t prefix = PASS == 0 ? 0u : (uint32_t)w.dsel_state[row * 4 + 0];
  const uint32_t mask = PASS == 0 ? 0u : (uint32_t)w.dsel_state[row * 4 + 1];
  const int tid = threadIdx.x;
  for (int i = tid; i < nb; i += kBlock) hist[i] = 0;
  __syncthreads();
  for (int base = d.i0; base < d.i1; base += kBlock * kSelU) {
    uint32_t key[kSelU];
#pragma unroll
    for (int u = 0; u < kSelU; ++u) {  // the loads in flight together
      const int i = base + u * kBlock + tid;
      key[u] = i < d.i1 ? f2key(d.src[i]) : 0u;
    }
#pragma unroll
    for (int u = 0; u < kSelU; ++u) {
      const bool act = base + u * kBlock + tid < d.i1 && (key[u] & mask) == prefix;
      hist_add(hist, (key[u] >> shift) & dmask, act);
    }
  }
  __syncthreads();
  uint32_t *g = w.dsel_hist + (int64_t)row * 2048;
  for (int i = tid; i < nb; i += kBlock)
    if (hist[i]) atomicAdd(&g[i], hist[i]);
}

template <int PASS>
__global__ __launch_bounds__(kBlock) void k_dsel_digit(Params p, Work w) {
  __shared__ uint32_t hist[2048];
  __shared__ SelShared sh;
  const int row = blockIdx.x;
  const DselPiece d = dsel_piece(p, w, row, 0, 1);
  if (d.k == 0) return;
  constexpr int shift = PASS == 0 ? 21 : (PASS == 1 ? 10 : 0);
  constexpr int nb = PASS == 2 ? 1024 : 2048;
  constexpr uint32_t dmask = (uint32_t)nb - 1u;
  int32_t *st = w.dsel_state + row * 4;
  const uint32_t prefix = PASS == 0 ? 0u : (uint32_t)st[0];
  const uint32_t mask = PASS == 0 ? 0u : (uint32_t)st[1];
  const int krem = PASS == 0 ? d.k : st[2];
  const int tid = threadIdx.x;
  uint32_t *g = w.dsel_hist + (int64_t)row * 2048;
  for (int i = tid; i < 2048; i += kBlock) {
    hist[i] = i < nb ? g[i] : 0u;
    g[i] = 0u;
  }
  if (tid == 0) {
    sh.digit = 0;
    sh.above = 0;
  }
  __syncthreads();
  // Thread t owns bins [nb - (t+1)*bpt, nb - t*bpt): counting from the top.
  constexpr int bpt = nb / kBlock;
  const int hi = nb - tid * bpt;
  int mine = 0;
  for (int i = 1; i <= bpt; ++i) mine += (int)hist[hi - i];
  int tot;
  const int before = block_excl_scan<kBlock>(mine, sh.scan, &tot);
  if (before < krem && krem <= before + mine) {
    int cum = before;
    for (int i = 1; i <= bpt; ++i) {
      const int c = (int)hist[hi - i];
      if (cum + c >= krem) {
        sh.digit = (uint32_t)(hi - i);
        sh.above = cum;
        break;
      }
      cum += c;
    }
  }
  __syncthreads();
  if (tid == 0) {
    st[0] = (int32_t)(prefix | (sh.digit << shift));
    st[1] = (int32_t)(mask | (dmask << shift));
    st[2] = krem - sh.above;
  }
}

__global__ __launch_bounds__(kBlock) void k_dsel_count(Params p, Work w) {
  __shared__ int red[kWaves][2];
  const int row = blockIdx.y;
  const DselPiece d = dsel_piece(p, w, row, blockIdx.x, gridDim.x);
  if (d.k == 0) return;
  const uint32_t T = (uint32_t)w.dsel_state[row * 4 + 0];
  const int tid = threadIdx.x;
  int gt = 0, eq = 0;
  for (int base = d.i0; base < d.i1; base += kBlock * kSelU) {
    uint32_t key[kSelU];
#pragma unroll
    for (int u = 0; u < kSelU; ++u) {
      const int i = base + u * kBlock + tid;
      key[u] = i < d.i1 ? f2key(d.src[i]) : 0u;
    }
#pragma unroll
    for (int u = 0; u < kSelU; ++u) {
      const bool in = base + u * kBlock + tid < d.i1;
      gt += (in && key[u] > T) ? 1 : 0;
      eq += (in && key[u] == T) ? 1 : 0;
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    gt += __shfl_xor(gt, o);
    eq += __shfl_xor(eq, o);
  }
  if (lane_id() == 0) {
    red[wave_id()][0] = gt;
    red[wave_id()][1] = eq;
  }
  __syncthreads();
  if (tid == 0) {
    int a = 0, e = 0;
#pragma unroll
    for (int v = 0; v < kWaves; ++v) {
      a += red[v][0];
      e += red[v][1];
    }
    w.dsel_cnt[(int64_t)row * kDselPartsMax + blockIdx.x] = make_int2(a, e);
  }
}

struct PieceSrc {
  const float *row;  // the piece's first score
  __device__ __forceinline__ uint32_t key(int i) const { return f2key(row[i]); }
};

__global__ __launch_bounds__(kBlock) void k_dsel_write(Params p, Work w, int32_t *idx,
                                                       float *vals) {
  __shared__ int scan[kWaves];
  const int row = blockIdx.y, q = blockIdx.x;
  const DselPiece d = dsel_piece(p, w, row, q, gridDim.x);
  if (d.k == 0) return;
  const int b = row / p.R;
  const RowPlan rp = row_plan(p, b, seq_len(p, b));
  const uint32_t T = (uint32_t)w.dsel_state[row * 4 + 0];
  const int need_eq = w.dsel_state[row * 4 + 2];
  const int tid = threadIdx.x;
  // Keys above and equal to T in the pieces before this one.
  int2 c = make_int2(0, 0);
  if (tid < q) c = w.dsel_cnt[(int64_t)row * kDselPartsMax + tid];
  int gt_before, eq_before;
  block_excl_scan<kBlock>(c.x, scan, &gt_before);
  block_excl_scan<kBlock>(c.y, scan, &eq_before);
  const int sel_before = gt_before + (eq_before < need_eq ? eq_before : need_eq);
  const int64_t ist = p.idx_stride > 0 ? p.idx_stride : p.k_max;
  int32_t *irow = idx + (int64_t)row * ist + rp.ns;
  float *vrow = vals ? vals + (int64_t)row * p.k_max + rp.ns : nullptr;
  const uint32_t base = (uint32_t)(rp.lo + d.i0);
  compact_selected_from<kBlock>(PieceSrc{d.src + d.i0}, d.i1 - d.i0, d.k, T, need_eq, scan,
                                eq_before, sel_before, [&](int slot, int i, uint32_t key) {
                                  if (slot >= d.k) return;  // (never: exactly k are kept)
                                  irow[slot] = (int32_t)(base + (uint32_t)i);
                                  if (vrow) vrow[slot] = key2f(key);
                                });
}

// ---------------------------------------------------------------------------
// Sampled selection: after the exact selection has written each row's kept
// list S (ascending, total = |S| entries, row stride p.idx_stride), append
// the row's s draws from the rest C = [0, L) \ S and write every entry's
// weight: 1 for S, |C| / s for a draw (float32), 0 for the padding.  Draw i
// (a uint32 u) is the floor(u |C| / 2^32)-th position of C in ascending
// order: the rank rho plus the number of kept positions at or below the
// result, which is #{t : S[t] - t <= rho} (S[t] - t is non-decreasing), found
// by binary search.  grid = B*R rows.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kBlock) void k_sample_rest(Params p, int32_t *list,
                                                        const uint32_t *draws, int s,
                                                        float *weights) {
  const int row = blockIdx.x, b = row / p.R;
  const int L = seq_len(p, b);
  const RowPlan rp = row_plan(p, b, L);
  const int64_t ist = p.idx_stride;  // = k_max + s
  int32_t *lrow = list + (int64_t)row * ist;
  float *wrow = weights + (int64_t)row * ist;
  const uint32_t *drow = draws + (int64_t)row * s;
  const int total = rp.total;
  const int64_t c = (int64_t)L - total;  // positions outside the kept set
  const float wd = c > 0 && s > 0 ? (float)c / (float)s : 0.f;
  for (int t = threadIdx.x; t < ist; t += kBlock) {
    if (t < total) {
      wrow[t] = 1.f;
    } else if (t < total + s && c > 0) {
      const uint64_t rho = ((uint64_t)drow[t - total] * (uint64_t)c) >> 32;  // < c
      int lo = 0, hi = total;  // count of t' with S[t'] - t' <= rho, in [0, total]
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if ((int64_t)lrow[mid] - mid <= (int64_t)rho) lo = mid + 1;
        else hi = mid;
      }
      lrow[t] = (int32_t)((int64_t)rho + lo);
      wrow[t] = wd;
    } else {
      wrow[t] = 0.f;  // padding (the selection wrote -1)
    }
  }
}

// ---------------------------------------------------------------------------
// Gather-attend.  grid = (splits, rows).  Workgroup s of row (b, r) takes
// list entries [s*split, +split) of idx[b][r]; in per-head mode the row is
// query head r, in group-shared mode it serves the G heads of KV head r.
// FUSED: the list holds exactly k_b valid positions, and per-head rows take
// their softmax weights from sigma (formed by the selection); group-shared
// rows, and every row of the unfused call, recompute each head's logits
// from the kept key rows (MFMA tiles for bf16), skipping entries outside
// [0, L_b), and form the weights exp(z - max) once per position in LDS.  Each wave then walks 4 * U positions per step
// (U per 16-lane group, 16 lanes x 16 bytes covering one 256-byte
// bf16 value row), with the next step's loads issued before the current
// step is consumed.  A row split over several workgroups leaves (max, sum,
// unnormalised output) partials that k_merge combines.
// Dynamic LDS: voff[split] i64, koff[split] i64 (recompute only),
// e[nh][split] f32, pos[split] i32, q[nh][128] f32 (recompute only),
// red[kWaves][nhb][128] f32, lred[kWaves][nhb] f32, nhb = min(nh, kAttHeads).
// ---------------------------------------------------------------------------
constexpr int kAttHeads = 8;  // heads accumulated per pass over the value rows
constexpr int kUnionPerThread = 4;  // union attention: mask positions per thread
constexpr int kUnionChunkMax = kBlock * kUnionPerThread;  // positions per workgroup

template <bool BF16>
struct RowRaw {
  u32x4 v[BF16 ? 1 : 2];  // this lane's 8 channels of one value row
};

// Gathered rows are read once: nontemporal loads.  (Measured at the 128K
// batch-16 workload: right after a 1 GiB buffer had been written, the
// gather with plain loads took 0.117 ms instead of 0.061 ms, paying for the
// write's cached lines it evicted; with nontemporal loads it took 0.062.)
template <bool BF16>
__device__ __forceinline__ void load_raw(const void *base, int64_t off, int col, RowRaw<BF16> &r) {
  if constexpr (BF16) {
    r.v[0] = __builtin_nontemporal_load((const u32x4 *)((const uint16_t *)base + off + 8 * col));
  } else {
    const u32x4 *q = (const u32x4 *)((const float *)base + off + 8 * col);
    r.v[0] = __builtin_nontemporal_load(q);
    r.v[1] = __builtin_nontemporal_load(q + 1);
  }
}

template <bool BF16>
__device__ __forceinline__ void unpack_raw(const RowRaw<BF16> &r, float v[8]) {
  if constexpr (BF16) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      v[2 * e] = bf16_to_f32(r.v[0][e] & 0xFFFFu);
      v[2 * e + 1] = bf16_to_f32(r.v[0][e] >> 16);
    }
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      v[e] = __uint_as_float(r.v[0][e]);
      v[4 + e] = __uint_as_float(r.v[1][e]);
    }
  }
}

template <bool BF16>
__device__ __forceinline__ void load_row8(const void *base, int64_t off, int col, float v[8]) {
  RowRaw<BF16> r;
  load_raw<BF16>(base, off, col, r);
  unpack_raw<BF16>(r, v);
}

template <bool BF16>
__device__ __forceinline__ void store_out(void *out, int64_t off, float v) {
  if constexpr (BF16) ((uint16_t *)out)[off] = f32_to_bf16_rne(v);
  else ((float *)out)[off] = v;
}

__device__ __forceinline__ int attend_list_len(const Params &p, int b, int L, bool fused) {
  return fused ? row_plan(p, b, L).total : p.k_max;
}

// Logits are recomputed from the key rows unless the selection formed the
// softmax weights already (fused per-head rows on exact scores without
// forced positions).
__host__ __device__ inline bool attend_recompute(bool fused, const Params &p) {
  return !fused || p.group_shared || p.n_sink + p.n_local > 0 || p.labels != nullptr;
}

// Row index of position j of sequence b in a cache, 32 bits: j itself in
// the contiguous layout, the pool row page * 16 + j % 16 in the paged one
// (the block-table lookup done once); row_offset turns it into the element
// offset of KV head g's row.
__device__ __forceinline__ uint32_t kv_row(const KvView &kv, int b, int64_t j) {
  if (!kv.paged) return (uint32_t)j;
  const int64_t page = kv.block_table[(int64_t)b * kv.max_pages + (j >> 4)];
  return (uint32_t)(page * kTile + (j & 15));
}
__device__ __forceinline__ int64_t row_offset(const KvView &kv, int b, int g, uint32_t r) {
  if (!kv.paged) return (((int64_t)b * kv.hkv + g) * kv.ncap + r) * kHeadDim;
  return ((int64_t)r * kv.hkv + g) * kHeadDim;
}

// Byte offsets of the dynamic LDS areas of k_attend (host and device agree):
// per list entry its value row (and key row, when the logits are
// recomputed) as 32-bit row indices, its weights, and its position where
// entries can be skipped (recomputed logits) or are built (union).
struct AttLds {
  int voff, koff, e, pos, hm, q, red, lred, total;
  __host__ __device__ AttLds(int split, int nh, bool recompute, bool uni = false) {
    const int nhb = nh < kAttHeads ? nh : kAttHeads;
    int o = 0;
    voff = o; o += 4 * split;
    koff = o; o += recompute ? 4 * split : 0;
    e = o; o += 4 * nh * split;
    pos = o; o += (recompute || uni) ? 4 * split : 0;
    hm = o; o += uni ? 4 * split : 0;
    q = o; o += recompute ? 4 * nh * kHeadDim : 0;
    red = o; o += 4 * kWaves * nhb * kHeadDim;
    lred = o; o += 4 * kWaves * nhb;
    total = o;
  }
};

// UNI (union attention, with FUSED and GRP): the workgroup of (chunk s,
// group (b, g)) takes the positions [s*split, +split) that any head of the
// group keeps (from the heads' lists and chunk starts), in order, and serves every head,
// each over its own positions only.  HBU: heads accumulated per pass over
// the value rows in group mode (4 for groups of at most 4 heads: fewer
// registers, three waves per SIMD instead of two).
template <bool BF16, bool FUSED, bool GRP, bool UNI = false, int HBU = kAttHeads>
__global__ __launch_bounds__(kBlock) void k_attend(Params p, Work w, const int32_t *idx, void *out,
                                                   int split) {
  static_assert(!UNI || (BF16 && FUSED && GRP), "union attention: fused bf16 group rows");
  extern __shared__ int64_t att_dyn[];
  __shared__ float mh[kMaxGroup];
  __shared__ float hmax[kWaves][kMaxGroup];
  constexpr int U = (BF16 && !GRP) ? 8 : 4;  // positions per 16-lane group per step
  constexpr int HB = GRP ? HBU : 1;  // heads accumulated per pass

  const int rows_per_b = UNI ? p.Hkv : p.R;  // union rows are the groups
  const int s = blockIdx.x, row = FUSED ? ordered_row(w, (int)blockIdx.y, rows_per_b)
                                        : (int)blockIdx.y;
  const int b = row / rows_per_b, r = row % rows_per_b;
  constexpr bool grp = GRP;
  const int nh = grp ? p.G : 1;
  const int nhb = nh < kAttHeads ? nh : kAttHeads;
  const int h0 = grp ? r * p.G : r;
  const int g = grp ? r : r / p.G;
  const int L = seq_len(p, b);
  const int n_list = UNI ? L : attend_list_len(p, b, L, FUSED);
  const int nsp = (n_list + split - 1) / split;
  const int tid = threadIdx.x, l = lane_id(), col = l & 15, sub = l >> 4, wv = wave_id();
  const bool recompute = UNI || attend_recompute(FUSED, p);
  const AttLds lay(split, nh, recompute, UNI);
  char *dyn = (char *)att_dyn;
  uint32_t *voff_l = (uint32_t *)(dyn + lay.voff);  // value rows (kv_row)
  uint32_t *koff_l = (uint32_t *)(dyn + lay.koff);  // key rows (recompute)
  float *e_l = (float *)(dyn + lay.e);
  int32_t *pos_l = (int32_t *)(dyn + lay.pos);
  uint32_t *hm_l = (uint32_t *)(dyn + lay.hm);  // UNI: each entry's head bits
  float *q_l = (float *)(dyn + lay.q);        // [nh][128]
  float *red = (float *)(dyn + lay.red);      // [kWaves][nhb][128]
  float *lred = (float *)(dyn + lay.lred);    // [kWaves][nhb]

  if (n_list == 0 || L == 0) {  // nothing kept: zero output
    if (s == 0)
      for (int e = tid; e < nh * kHeadDim; e += kBlock)
        store_out<BF16>(out, ((int64_t)b * p.Hq + h0 + e / kHeadDim) * kHeadDim + e % kHeadDim, 0.f);
    return;
  }
  if (s >= nsp) return;
  const int e0 = s * split;
  int n = (n_list - e0) < split ? (n_list - e0) : split;

  if constexpr (UNI) {
    // The chunk's positions that some head keeps, in order, with their head
    // bits: each head's entries in the chunk (the span its chunk starts give)
    // set the head's bit of their positions in an LDS bitmap (the key
    // offset area, free until the offsets are resolved); then each thread
    // takes kUnionPerThread consecutive positions and one block scan places
    // the kept ones.
    __shared__ int scan_tmp[kWaves];
    __shared__ int hspan[kMaxGroup][2];
    uint32_t *hb = (uint32_t *)koff_l;  // n <= split <= kUnionChunkMax words
    for (int t = tid; t < n; t += kBlock) hb[t] = 0u;
    if (tid < nh) {
      const int32_t *us = w.ustart + ((int64_t)b * p.R + h0 + tid) * w.ustride;
      hspan[tid][0] = us[s];
      hspan[tid][1] = us[s + 1];
    }
    __syncthreads();
    // The heads' entries as one flat range (head by head), four per thread
    // per round with their loads in flight together.
    int tot_e = 0;
    for (int h = 0; h < nh; ++h) tot_e += hspan[h][1] - hspan[h][0];
    const int32_t *lists = idx + ((int64_t)b * p.R + h0) * p.k_max;
    for (int ebase = tid; ebase < tot_e; ebase += 4 * kBlock) {
      int pos[4], hh[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int e = ebase + u * kBlock;
        hh[u] = -1;
        pos[u] = 0;
        if (e < tot_e) {
          int h = 0, before = 0;
          while (h < nh - 1 && e >= before + hspan[h][1] - hspan[h][0]) {
            before += hspan[h][1] - hspan[h][0];
            ++h;
          }
          hh[u] = h;
          pos[u] = lists[(int64_t)h * p.k_max + hspan[h][0] + (e - before)];
        }
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int off = pos[u] - e0;
        if (hh[u] >= 0 && (unsigned)off < (unsigned)n) atomicOr(&hb[off], 1u << hh[u]);
      }
    }
    __syncthreads();
    uint32_t bits[kUnionPerThread];
    int cnt = 0;
    const int t0u = tid * kUnionPerThread;  // n <= split <= kUnionChunkMax
#pragma unroll
    for (int u = 0; u < kUnionPerThread; ++u) {
      const int t = t0u + u;
      bits[u] = t < n ? hb[t] : 0u;
      cnt += bits[u] != 0u ? 1 : 0;
    }
    int tot;
    int slot = block_excl_scan<kBlock>(cnt, scan_tmp, &tot);
#pragma unroll
    for (int u = 0; u < kUnionPerThread; ++u) {
      if (bits[u]) {
        pos_l[slot] = e0 + tid * kUnionPerThread + u;
        hm_l[slot] = bits[u];
        ++slot;
      }
    }
    n = tot;
    __syncthreads();
    for (int t = tid; t < n; t += kBlock) {
      const int64_t j = pos_l[t];
      voff_l[t] = kv_row(p.V, b, j);
      koff_l[t] = kv_row(p.K, b, j);
    }
  } else {
    // Resolve every entry to its row offsets once (page-table reads in
    // parallel); skipped entries point at position 0 and get weight 0.
    const int32_t *irow = idx + (int64_t)row * p.k_max + e0;
    for (int t = tid; t < n; t += kBlock) {
      int32_t j = irow[t];
      if (j < 0 || j >= L) j = -1;
      if (recompute) pos_l[t] = j;  // (fused lists hold only valid entries)
      const int64_t jc = j >= 0 ? j : 0;
      voff_l[t] = kv_row(p.V, b, jc);
      if (recompute) koff_l[t] = kv_row(p.K, b, jc);
    }
  }
  if (recompute && !BF16) {  // float32 queries for the vector-ALU logits
    for (int e = tid; e < nh * kHeadDim; e += kBlock) {
      const int64_t qo = ((int64_t)b * p.Hq + h0 + e / kHeadDim) * kHeadDim + e % kHeadDim;
      q_l[e] = ((const float *)p.q)[qo];
    }
  }
  __syncthreads();

  // Logits z[h][t] = scale * q_h . K_j (kept in e_l until the max is known).
  // Per-head fused rows arrive with their softmax weights already formed
  // (relative to the row's maximum, so all splits share one reference).
  if (!recompute) {
    const float *wrow = w.sigma + (int64_t)row * p.k_max + e0;
    for (int t = tid; t < n; t += kBlock) e_l[t] = wrow[t];
    if (tid == 0) mh[0] = 0.f;
  } else if constexpr (BF16) {
    // Logits by MFMA: a wave scores 16 kept positions per tile, each lane
    // loading its position's key slices straight into the operand layout;
    // the query operand's rows are the nh heads served.  Two tiles' loads
    // are in flight before their matrix ops.
    QFrag qf;
    load_q_heads(p, b, h0, nh, qf);
    const int ntile = (n + kTile - 1) / kTile;
    const int kcol = l & 15, quad = l >> 4;
    auto tile_off = [&](int ti) {
      const int t = ti * kTile + kcol;
      return row_offset(p.K, b, g, koff_l[t < n ? t : 0]);
    };
    for (int ti = wv; ti < ntile; ti += 2 * kWaves) {
      const int ti1 = ti + kWaves;
      KFrag kf[2];
      load_k_bf16(p.K, tile_off(ti), kf[0]);
      load_k_bf16(p.K, tile_off(ti1 < ntile ? ti1 : ti), kf[1]);
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int tt = u == 0 ? ti : ti1;
        if (tt >= ntile) break;  // wave-uniform
        const f32x4 acc = mfma_scores(qf, kf[u]);
        const int t = tt * kTile + kcol;
        if (t < n) {
          const bool skip = pos_l[t] < 0;
          const uint32_t hb = UNI ? hm_l[t] : 0xFFFFFFFFu;  // heads that keep it
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int h = 4 * quad + r;
            if (h < nh)
              e_l[h * split + t] = (skip || !((hb >> h) & 1u)) ? -__builtin_inff() : p.scale * acc[r];
          }
        }
      }
    }
  } else {
    for (int t = wv * 4 + sub; t < n; t += kWaves * 4) {
      const int32_t j = pos_l[t];
      if (j < 0) {  // uniform over the 16 lanes of this position
        if (col == 0)
          for (int h = 0; h < nh; ++h) e_l[h * split + t] = -__builtin_inff();
        continue;
      }
      float kv[8];
      load_row8<BF16>(p.K.base, row_offset(p.K, b, g, koff_l[t]), col, kv);
      for (int h = 0; h < nh; ++h) {
        float d = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) d = fmaf(q_l[h * kHeadDim + 8 * col + e], kv[e], d);
        d += __shfl_xor(d, 1);
        d += __shfl_xor(d, 2);
        d += __shfl_xor(d, 4);
        d += __shfl_xor(d, 8);
        if (col == 0) e_l[h * split + t] = p.scale * d;
      }
    }
  }
  __syncthreads();
  if (recompute) {
    // Per-head maxima: every wave reduces its share, one barrier, then
    // thread h combines the waves.  With per-entry weights omega the logit
    // becomes z + log(omega), so that exp(z' - m) = omega * exp(z - m) and
    // the maximum (shared by all splits through the merge) stays finite for
    // any positive weights; an entry of weight 0 is skipped.
    const float *wrow = p.weights ? p.weights + (int64_t)row * p.k_max + e0 : nullptr;
    for (int h = 0; h < nh; ++h) {
      float m = -__builtin_inff();
      for (int t = tid; t < n; t += kBlock) {
        float z = e_l[h * split + t];
        if (wrow) {
          const float om = wrow[t];
          z = om > 0.f ? z + logf(om) : -__builtin_inff();
          e_l[h * split + t] = z;
        }
        m = fmaxf(m, z);
      }
      m = wave_max(m);
      if (l == 0) hmax[wv][h] = m;
    }
    __syncthreads();
    if (tid < nh) {
      float m = hmax[0][tid];
#pragma unroll
      for (int v = 1; v < kWaves; ++v) m = fmaxf(m, hmax[v][tid]);
      mh[tid] = m;
    }
    __syncthreads();
    // Weights exp(z - m); skipped entries (z = -inf) give 0.
    for (int e = tid; e < nh * n; e += kBlock) {
      const int h = e / n, t = e % n;
      const float z = e_l[h * split + t];
      e_l[h * split + t] = z == -__builtin_inff() ? 0.f : expf(z - mh[h]);
    }
    __syncthreads();
  }

  const int stride = kWaves * 4 * U;  // positions per workgroup step
  for (int hb = 0; hb < nh; hb += HB) {
    const int nb = (nh - hb) < HB ? (nh - hb) : HB;
    float acc[HB][8];
    float lsum[HB];
#pragma unroll
    for (int h = 0; h < HB; ++h) {
      lsum[h] = 0.f;
#pragma unroll
      for (int c = 0; c < 8; ++c) acc[h][c] = 0.f;
    }
    // Branch-free gather: entries past the slice read entry 0's row (weight
    // 0), so every step issues the same loads, and the next step's loads are
    // in flight while this step's rows are accumulated.
    auto issue = [&](int tb, RowRaw<BF16> buf[U]) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int t = tb + 4 * u + sub;
        load_raw<BF16>(p.V.base, row_offset(p.V, b, g, voff_l[t < n ? t : 0]), col, buf[u]);
      }
    };
    auto consume = [&](int tb, const RowRaw<BF16> buf[U]) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int t = tb + 4 * u + sub;
        float vv[8];
        unpack_raw<BF16>(buf[u], vv);
#pragma unroll
        for (int h = 0; h < HB; ++h) {
          if (h < nb) {
            const float e = t < n ? e_l[(hb + h) * split + t] : 0.f;
            lsum[h] += e;
#pragma unroll
            for (int c = 0; c < 8; ++c) acc[h][c] = fmaf(e, vv[c], acc[h][c]);
          }
        }
      }
    };
    RowRaw<BF16> b0[U], b1[U];
    int t0 = wv * 4 * U;
    if (t0 < n) {  // wave-uniform
      issue(t0, b0);
      for (;; t0 += 2 * stride) {
        issue(t0 + stride, b1);
        consume(t0, b0);
        if (t0 + stride >= n) break;
        issue(t0 + 2 * stride, b0);
        consume(t0 + stride, b1);
        if (t0 + 2 * stride >= n) break;
      }
    }
    // Reduce over the four position groups of a wave, then over waves.
#pragma unroll
    for (int h = 0; h < HB; ++h) {
      if (h < nb) {
#pragma unroll
        for (int c = 0; c < 8; ++c) {
          float v = acc[h][c];
          v += __shfl_xor(v, 16);
          v += __shfl_xor(v, 32);
          acc[h][c] = v;
        }
        float ls = lsum[h];
        ls += __shfl_xor(ls, 16);
        ls += __shfl_xor(ls, 32);
        if (sub == 0) {
#pragma unroll
          for (int c = 0; c < 8; ++c) red[(wv * nhb + h) * kHeadDim + 8 * col + c] = acc[h][c];
          if (col == 0) lred[wv * nhb + h] = ls;
        }
      }
    }
    __syncthreads();
    for (int e = tid; e < nb * kHeadDim; e += kBlock) {
      const int h = e / kHeadDim, c = e % kHeadDim;
      float o = 0.f, ls = 0.f;
#pragma unroll
      for (int v = 0; v < kWaves; ++v) {
        o += red[(v * nhb + h) * kHeadDim + c];
        ls += lred[v * nhb + h];
      }
      const int hq = h0 + hb + h;
      if (nsp == 1) {
        store_out<BF16>(out, ((int64_t)b * p.Hq + hq) * kHeadDim + c, ls > 0.f ? o / ls : 0.f);
      } else {
        float *pp = w.part + (((int64_t)b * p.Hq + hq) * w.nsplit + s) * kPartStride;
        if (c == 0) {
          pp[0] = mh[hb + h];
          pp[1] = ls;
        }
        pp[2 + c] = o;
      }
    }
    __syncthreads();
  }
}

// Log-sum-exp merge of split partials: grid = B*Hq output rows, blocks of
// kMergeThreads.  Rows that fit one split were written by k_attend.
template <bool BF16, bool FUSED>
__global__ __launch_bounds__(kMergeThreads) void k_merge(Params p, Work w, void *out, int split) {
  __shared__ MergeShared sh;
  const int bh = blockIdx.x, b = bh / p.Hq;
  const int L = seq_len(p, b);
  const int n_list = w.union_chunk ? L : attend_list_len(p, b, L, FUSED);
  const int nsp = (n_list + split - 1) / split;
  if (nsp <= 1 || L == 0) return;  // written directly by k_attend
  const float v = merge_partials(w.part + (int64_t)bh * w.nsplit * kPartStride, nsp, sh);
  if (threadIdx.x < kHeadDim) store_out<BF16>(out, (int64_t)bh * kHeadDim + threadIdx.x, v);
}

// ---------------------------------------------------------------------------
// Launchers (host).
// ---------------------------------------------------------------------------
static inline unsigned cdiv(int64_t a, int64_t b) { return (unsigned)((a + b - 1) / b); }

hipError_t launch_pilot(const Params &p, const Work &w, hipStream_t st) {
  if (!w.force_repair) {
    if (p.K.paged && p.Hkv % kWaves == 0) {
      const dim3 g4(kSampleMax / (kPilotTiles * kTile), p.B * p.Hkv / kWaves);
      if (p.labels) k_pilot_score<true, true><<<g4, kBlock, 0, st>>>(p, w);
      else k_pilot_score<false, true><<<g4, kBlock, 0, st>>>(p, w);
    } else {
      const dim3 g1(kSampleMax / (kPilotTiles * kTile * kWaves), p.B * p.Hkv);
      if (p.labels) k_pilot_score<true, false><<<g1, kBlock, 0, st>>>(p, w);
      else k_pilot_score<false, false><<<g1, kBlock, 0, st>>>(p, w);
    }
  }
  k_pilot_select<<<p.B * p.R, kBlock, 0, st>>>(p, w);
  return hipGetLastError();
}

// Launch with start/stop events attached to the kernel's own dispatch (no
// extra packets on the stream), or a plain launch when they are null.
static hipError_t launch_with_events(void (*kern)(Params, Work), dim3 grid, size_t lds,
                                     const Params &p, const Work &w, hipStream_t st,
                                     hipEvent_t t0, hipEvent_t t1) {
  if (!t0) {
    kern<<<grid, kBlock, lds, st>>>(p, w);
    return hipGetLastError();
  }
  Params pa = p;
  Work wa = w;
  void *args[] = {&pa, &wa};
  return hipExtLaunchKernel((const void *)kern, grid, dim3(kBlock), args, lds, st, t0, t1, 0);
}

size_t stream_outbox_bytes() { return sizeof(Outbox) + (size_t)kOutboxCap * 6; }

bool stream_by_head_quads(const Work &w) { return w.chunk_keys == w.wave_keys; }

// The label stream instance holding `rows` rows per wave in registers.
template <bool PAGED, bool QUAD>
static void (*label_stream_kernel(bool group_shared, int rows))(Params, Work) {
  if (group_shared) return k_score_stream<PAGED, true, QUAD, true, 1>;
  if (rows <= 1) return k_score_stream<PAGED, false, QUAD, true, 1>;
  if (rows <= 2) return k_score_stream<PAGED, false, QUAD, true, 2>;
  if (rows <= 4) return k_score_stream<PAGED, false, QUAD, true, 4>;
  if (rows <= 8) return k_score_stream<PAGED, false, QUAD, true, 8>;
  return k_score_stream<PAGED, false, QUAD, true, 16>;
}

hipError_t launch_score_stream(const Params &p, const Work &w, hipStream_t st, hipEvent_t t0,
                               hipEvent_t t1) {
  if (w.force_repair) return hipSuccess;  // every row takes the fallback
  void (*kern)(Params, Work);
  int64_t wgs;
  const bool gs = p.group_shared != 0, lab = p.labels != nullptr;
  const int rows = gs ? 1 : p.G;
  if (stream_by_head_quads(w)) {
    if (lab) kern = label_stream_kernel<true, true>(gs, rows);
    else kern = gs ? k_score_stream<true, true, true, false, 0> : k_score_stream<true, false, true, false, 0>;
    wgs = (int64_t)w.nchunk * p.B * (p.Hkv / kWaves);
  } else if (p.K.paged) {
    if (lab) kern = label_stream_kernel<true, false>(gs, rows);
    else kern = gs ? k_score_stream<true, true, false, false, 0> : k_score_stream<true, false, false, false, 0>;
    wgs = (int64_t)w.nchunk * p.B * p.Hkv;
  } else {
    if (lab) kern = label_stream_kernel<false, false>(gs, rows);
    else kern = gs ? k_score_stream<false, true, false, false, 0> : k_score_stream<false, false, false, false, 0>;
    wgs = (int64_t)w.nchunk * p.B * p.Hkv;
  }
  if (!w.persistent) return launch_with_events(kern, dim3((unsigned)wgs), 0, p, w, st, t0, t1);
  // One workgroup per compute unit (w.stream_wgs), or one per unit of work.
  const int64_t grid = wgs < w.stream_wgs ? wgs : w.stream_wgs;
  return launch_with_events(kern, dim3((unsigned)grid), stream_outbox_bytes(), p, w, st, t0, t1);
}

size_t select_lds_bytes(int nchunk, int lds_cap) {
  return (size_t)(2 * nchunk + 1) * 4 + (size_t)lds_cap * 4;
}

bool select_wide(const Params &p, size_t lds_bytes) {
  return (size_t)(p.B * p.R) < (size_t)kSelectWideRows || lds_bytes > kSelectShareLds;
}

size_t select_lds_budget(bool wide) {
  // Dynamic LDS left by the selection kernel's static LDS (hist, scan and
  // bucket scratch: about 9.9 KB at 256 threads, 14.1 KB at 1024) under the
  // 160 KB of a workgroup.
  return wide ? 144 * 1024 : 150 * 1024;
}

hipError_t launch_select_candidates(const Params &p, const Work &w, int32_t *idx, int lds_cap,
                                    bool wide, hipStream_t st) {
  const size_t lds = select_lds_bytes(w.nchunk, lds_cap);
  const unsigned rows = (unsigned)(p.B * p.R);
  // The kept scores / weights only serve an attention that does not
  // recompute its logits.
  float *vals = attend_recompute(true, p) ? nullptr : w.sigma;
  if (w.psel_parts > 0) {  // (wide: the host asks for pieces only then)
    const size_t plds = psel_lds_bytes(1024);
    k_select<0, 1024, true><<<dim3(rows, (unsigned)w.psel_parts), 1024, lds > plds ? lds : plds, st>>>(
        p, w, nullptr, 0, idx, vals, lds_cap);
  } else if (wide)
    k_select<0, 1024><<<rows, 1024, lds, st>>>(p, w, nullptr, 0, idx, vals, lds_cap);
  else
    k_select<0, kBlock><<<rows, kBlock, lds, st>>>(p, w, nullptr, 0, idx, vals, lds_cap);
  return hipGetLastError();
}

// Workgroups per (sequence, KV head) of the fallback scoring.  Without
// forcing, flagged rows are rare and most calls only check the flags, so
// about 1024 workgroups in all, up to kRepairParts per group: a launch of
// 2048 or 4096 workgroups that only check the flags took 4.4 and 6.9 us at
// the 128K batch-16 and the ragged paged workloads.  When every row is
// forced onto the fallback and the groups are few, enough for about 2048 in
// all (with one sequence each wave would otherwise score a long run of
// tiles one after another, each waiting for its loads).
int repair_parts(const Params &p, const Work &w) {
  const int groups = p.B * p.Hkv;
  if (!w.force_repair) {
    int parts = (1024 + groups - 1) / groups;
    parts = parts < kRepairParts ? parts : kRepairParts;
    // With the candidate selection in pieces, a workgroup per piece of the
    // group's rows (their histograms run in this launch), up to 64.
    const int tasks = (p.group_shared ? 1 : p.G) * w.psel_parts;
    const int want = tasks < 64 ? tasks : 64;
    return parts > want ? parts : want;
  }
  int parts = (2048 + groups - 1) / groups;
  parts = parts < kRepairParts ? kRepairParts : parts;
  return parts > 256 ? 256 : parts;
}

hipError_t launch_dense_select(const Params &p, const Work &w, int32_t *idx, hipStream_t st) {
  if (!w.dsel_parts) return hipSuccess;
  const int rows = p.B * p.R;
  const dim3 grid(w.dsel_parts, rows);
  k_dsel_hist<0><<<grid, kBlock, 0, st>>>(p, w);
  k_dsel_digit<0><<<rows, kBlock, 0, st>>>(p, w);
  k_dsel_hist<1><<<grid, kBlock, 0, st>>>(p, w);
  k_dsel_digit<1><<<rows, kBlock, 0, st>>>(p, w);
  k_dsel_hist<2><<<grid, kBlock, 0, st>>>(p, w);
  k_dsel_digit<2><<<rows, kBlock, 0, st>>>(p, w);
  k_dsel_count<<<grid, kBlock, 0, st>>>(p, w);
  k_dsel_write<<<grid, kBlock, 0, st>>>(p, w, idx, attend_recompute(true, p) ? nullptr : w.sigma);
  return hipGetLastError();
}

// Whether the full scoring of `parts` workgroups per (sequence, KV head)
// takes the instance with several tiles in flight: bf16 keys or labels,
// every wave with at least two rounds of tiles, and groups of more than one
// row.  (With one row per group, MHA, the forced fallback of Table 2's label
// shape at 2x took 0.377 instead of 0.338 ms at batch 1 and 1.23 instead of
// 1.13 ms at batch 4; with groups of four rows it went from 0.257 to 0.246
// ms at batch 1, and the 128K batch-16 key fallback from 1.10 to 1.04 ms.)
static bool dense_pipelined(const Params &p, int parts) {
  const int64_t tiles = (p.ncap + kTile - 1) / kTile;
  const int64_t per_wave = (tiles + (int64_t)parts * kWaves - 1) / ((int64_t)parts * kWaves);
  return (p.labels || p.bf16) && (p.group_shared || p.G > 1) &&
         per_wave >= 2 * dense_depth(p.labels != nullptr);
}

hipError_t launch_repair(const Params &p, const Work &w, hipStream_t st) {
  const int parts = repair_parts(p, w);
  const dim3 grid(parts, p.B * p.Hkv);
  const bool pipe = dense_pipelined(p, parts);
  if (p.labels) {
    if (pipe) k_repair_score<true, true, true><<<grid, kBlock, 0, st>>>(p, w);
    else k_repair_score<true, true, false><<<grid, kBlock, 0, st>>>(p, w);
  } else if (p.bf16) {
    if (pipe) k_repair_score<true, false, true><<<grid, kBlock, 0, st>>>(p, w);
    else k_repair_score<true, false, false><<<grid, kBlock, 0, st>>>(p, w);
  } else {
    k_repair_score<false, false, false><<<grid, kBlock, 0, st>>>(p, w);
  }
  return hipGetLastError();
}

// Workgroups to aim for when rows are split.  Fused calls: two per CU; with
// 1024, few rows were cut into pieces short enough for their latency chains
// and the merge to dominate (1M-key group-shared batch of 8 rows: attention
// 36 -> 30 us at 512; Table 2's label shape at batch 1 and 4, 2-5% faster).
// Unfused calls (the weighted backend over caller lists, key and value rows
// per entry) keep four per CU: their low-sparsity lists are bandwidth-bound,
// and at 512 Table 1's batch 1 took 0.281 instead of 0.177 ms at 2x.
constexpr int kAttendWorkgroupsFused = 512;
constexpr int kAttendWorkgroups = 1024;
constexpr int kAttendLdsMax = 60 * 1024;  // dynamic LDS of one attend workgroup
constexpr int kAttendMinEntries = 64;     // fewest list entries worth a workgroup of their own
constexpr int kAttendRowsWhole = 256;     // this many rows fill the chip unsplit

// Positions per attend workgroup: a row is not split when there are enough
// rows to give every CU a workgroup and the whole list fits one workgroup's
// LDS (a split then costs the merge launch, more than the extra parallelism
// saves); otherwise rows are split into about kAttendWorkgroupsFused
// (fused) or kAttendWorkgroups (unfused) workgroups
// in all, at least 64 positions each, within the LDS budget.
int attend_split(const Params &p, int k_max_positions, bool fused) {
  const int64_t rows = (int64_t)p.B * p.R;
  const int64_t k_max = k_max_positions > 0 ? k_max_positions : 1;
  const int nh = p.group_shared ? p.G : 1;
  const bool rc = attend_recompute(fused, p);
  const int64_t target = fused ? kAttendWorkgroupsFused : kAttendWorkgroups;
  int64_t nsplit = (target + rows - 1) / rows;
  if (rows >= kAttendRowsWhole && k_max <= 4096 &&  // (bounded: the LDS sum stays in int)
      AttLds((int)((k_max + 63) / 64 * 64), nh, rc).total <= kAttendLdsMax)
    nsplit = 1;
  const int64_t most = (k_max + kAttendMinEntries - 1) / kAttendMinEntries;
  if (nsplit > most) nsplit = most;
  if (nsplit < 1) nsplit = 1;
  int64_t split = (k_max + nsplit - 1) / nsplit;
  split = (split + 63) / 64 * 64;
  while (split > 64 && AttLds((int)split, nh, rc).total > kAttendLdsMax) split -= 64;
  // As many splits as that takes, the entries spread evenly over them (no
  // smaller than the LDS-capped size, so still within the budget).
  nsplit = (k_max + split - 1) / split;
  split = ((k_max + nsplit - 1) / nsplit + 63) / 64 * 64;
  return (int)split;
}

int attend_nsplit(const Params &p) {
  // The larger of the fused and unfused split counts (the unfused layout
  // needs more LDS per entry, hence smaller splits).
  int most = 1;
  for (int fused = 0; fused < 2; ++fused) {
    const int split = attend_split(p, p.k_max, fused != 0);
    const int64_t k_max = p.k_max > 0 ? p.k_max : 1;
    const int ns = (int)((k_max + split - 1) / split);
    most = ns > most ? ns : most;
  }
  return most;
}

hipError_t launch_sample_rest(const Params &p, int32_t *list, const uint32_t *draws, int s,
                              float *weights, hipStream_t st) {
  if (p.idx_stride != p.k_max + s) return hipErrorInvalidValue;
  k_sample_rest<<<p.B * p.R, kBlock, 0, st>>>(p, list, draws, s, weights);
  return hipGetLastError();
}

int union_chunk(const Params &p) {
  int c = kUnionChunkMax;
  while (c > 64 && AttLds(c, p.G, true, true).total > kAttendLdsMax) c -= 64;
  return c;
}

hipError_t launch_attend(const Params &p, const Work &w, const int32_t *idx, void *out, bool fused,
                         hipStream_t st) {
  if (fused && w.union_chunk > 0) {  // group-deduplicated attention
    if (!p.bf16 || p.group_shared || w.union_chunk > kUnionChunkMax || !w.ustart)
      return hipErrorInvalidValue;
    const int split = w.union_chunk;
    const size_t lds = (size_t)AttLds(split, p.G, true, true).total;
    const int nsplit = (int)((p.ncap + split - 1) / split);
    const dim3 grid(nsplit, p.B * p.Hkv);
    if (p.G <= 4) k_attend<true, true, true, true, 4><<<grid, kBlock, lds, st>>>(p, w, idx, out, split);
    else k_attend<true, true, true, true><<<grid, kBlock, lds, st>>>(p, w, idx, out, split);
    if (nsplit > 1) k_merge<true, true><<<(unsigned)(p.B * p.Hq), kMergeThreads, 0, st>>>(p, w, out, split);
    return hipGetLastError();
  }
  const int split = attend_split(p, p.k_max, fused);
  const size_t lds = (size_t)AttLds(split, p.group_shared ? p.G : 1,
                                    attend_recompute(fused, p)).total;
  const int64_t kk = p.k_max > 0 ? p.k_max : 1;
  const int nsplit = (int)((kk + split - 1) / split);
  const dim3 grid(nsplit, p.B * p.R);
  const bool g = p.group_shared != 0;
  if (p.bf16) {
    if (fused) {
      if (g) k_attend<true, true, true><<<grid, kBlock, lds, st>>>(p, w, idx, out, split);
      else k_attend<true, true, false><<<grid, kBlock, lds, st>>>(p, w, idx, out, split);
    } else {
      if (g) k_attend<true, false, true><<<grid, kBlock, lds, st>>>(p, w, idx, out, split);
      else k_attend<true, false, false><<<grid, kBlock, lds, st>>>(p, w, idx, out, split);
    }
  } else {
    if (fused) {
      if (g) k_attend<false, true, true><<<grid, kBlock, lds, st>>>(p, w, idx, out, split);
      else k_attend<false, true, false><<<grid, kBlock, lds, st>>>(p, w, idx, out, split);
    } else {
      if (g) k_attend<false, false, true><<<grid, kBlock, lds, st>>>(p, w, idx, out, split);
      else k_attend<false, false, false><<<grid, kBlock, lds, st>>>(p, w, idx, out, split);
    }
  }
  if (nsplit > 1) {
    const unsigned rows = (unsigned)(p.B * p.Hq);
    if (p.bf16) {
      if (fused) k_merge<true, true><<<rows, kMergeThreads, 0, st>>>(p, w, out, split);
      else k_merge<true, false><<<rows, kMergeThreads, 0, st>>>(p, w, out, split);
    } else {
      if (fused) k_merge<false, true><<<rows, kMergeThreads, 0, st>>>(p, w, out, split);
      else k_merge<false, false><<<rows, kMergeThreads, 0, st>>>(p, w, out, split);
    }
  }
  return hipGetLastError();
}

hipError_t launch_score_dense(const Params &p, float *scores, hipStream_t st) {
  const int parts = (int)cdiv(p.ncap, kDenseChunk);
  const dim3 grid(parts, p.B * p.Hkv);
  const bool pipe = dense_pipelined(p, parts);
  if (p.labels) {
    if (pipe) k_score_dense<true, true, true><<<grid, kBlock, 0, st>>>(p, scores, p.ncap);
    else k_score_dense<true, true, false><<<grid, kBlock, 0, st>>>(p, scores, p.ncap);
  } else if (p.bf16) {
    if (pipe) k_score_dense<true, false, true><<<grid, kBlock, 0, st>>>(p, scores, p.ncap);
    else k_score_dense<true, false, false><<<grid, kBlock, 0, st>>>(p, scores, p.ncap);
  } else {
    k_score_dense<false, false, false><<<grid, kBlock, 0, st>>>(p, scores, p.ncap);
  }
  return hipGetLastError();
}

hipError_t launch_topk(const Params &p, const float *scores, int32_t *idx, float *vals,
                       hipStream_t st) {
  Work none{};
  k_select<1, kBlock><<<p.B * p.R, kBlock, 0, st>>>(p, none, scores, p.ncap, idx, vals, 0);
  return hipGetLastError();
}

}  // namespace sd
