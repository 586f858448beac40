// sd_api.hip -- the C ABI of libsparse_decode.so (declared in
// include/sparse_decode.h): argument checks, workspace carving and the
// ordering of the kernels on the caller's stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <mutex>

#include "sparse_decode.h"
#include "sd_internal.hpp"
#include "sd_launch.hpp"

namespace {

using sd::kHeadDim;

constexpr int kMaxDevices = 64;
constexpr size_t kAlign = 256;
constexpr int kRing = 64;          // profiled calls remembered per device
// Longest cache (positions per sequence): the selection keeps two entries
// per candidate chunk (at least 1024 keys) in LDS.
constexpr int64_t kMaxCapacity = int64_t(1) << 24;

struct DevState {
  void *ws = nullptr;
  size_t ws_bytes = 0;
  bool user_ws = false;
  bool events = false;
  hipEvent_t ev[kRing][6];
  int level[kRing] = {};  // profiling level each ring slot was recorded with
  int64_t n_calls = 0;  // profiled calls in the current series
  int n_cu = 0;         // compute units (0: not queried yet)
  // Device addresses of this GPU's copies of `scratch` and `stats_dev`
  // (hipGetSymbolAddress, taken once with the device current).
  bool symbols = false;
  void *scratch = nullptr;
  int32_t *stats = nullptr;
};

// Workspace of the allocation-free entry point: one copy per GPU the
// library runs on, held until the process ends.  In host code these names
// stand for the device arrays, not their addresses: host code uses only
// the addresses that device_state() takes with hipGetSymbolAddress.
constexpr size_t kScratchBytes = SD_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];
// Per-call counters the kernels keep (stats[0]: rows repaired by the last
// call of the fused path), outside every workspace so that the profile can
// read them whatever became of a workspace since.
static __device__ __align__(256) int32_t stats_dev[16];

std::mutex g_mu;
DevState g_dev[kMaxDevices];
std::atomic<int> g_profiling{0};
std::atomic<int> g_debug{0};

struct Shape {
  int B, Hq, Hkv, G, R;
  int64_t ncap;
  int bf16;
  int paged;
  int64_t k_max;
};

inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool is_dtype_float(int32_t d) { return d == SD_F32 || d == SD_BF16; }

sd_status check_q(const sd_tensor *q, Shape &s) {
  if (!q || !q->data || q->ndim != 3) return SD_ERR_INVALID_ARG;
  if (!is_dtype_float(q->dtype)) return SD_ERR_INVALID_ARG;
  if (q->shape[0] < 0 || q->shape[1] <= 0 || q->shape[2] <= 0) return SD_ERR_INVALID_ARG;
  if (q->shape[2] != kHeadDim) return SD_ERR_UNSUPPORTED;
  if (q->shape[0] > 65535 || q->shape[1] > 65535) return SD_ERR_UNSUPPORTED;
  s.B = (int)q->shape[0];
  s.Hq = (int)q->shape[1];
  s.bf16 = q->dtype == SD_BF16;
  return SD_OK;
}

// Checks a key/value cache against q's batch and dtype; fills Hkv and ncap.
sd_status check_kv(const sd_kv *kv, const Shape &s, int dtype, int &hkv, int64_t &ncap) {
  if (!kv || !kv->t.data || kv->t.ndim != 4) return SD_ERR_INVALID_ARG;
  if (kv->t.dtype != dtype) return SD_ERR_INVALID_ARG;
  for (int i = 0; i < 4; ++i)
    if (kv->t.shape[i] < 0) return SD_ERR_INVALID_ARG;
  if (kv->t.shape[3] != kHeadDim) return SD_ERR_UNSUPPORTED;
  if (kv->layout == SD_KV_BHND) {
    if (kv->t.shape[0] != s.B) return SD_ERR_INVALID_ARG;
    hkv = (int)kv->t.shape[1];
    ncap = kv->t.shape[2];
  } else if (kv->layout == SD_KV_PAGED_NHD) {
    if (kv->page_size != sd::kTile) return SD_ERR_UNSUPPORTED;
    if (kv->t.shape[1] != kv->page_size) return SD_ERR_INVALID_ARG;
    if (!kv->block_table || kv->max_pages_per_seq < 0) return SD_ERR_INVALID_ARG;
    hkv = (int)kv->t.shape[2];
    ncap = (int64_t)kv->max_pages_per_seq * kv->page_size;
  } else {
    return SD_ERR_INVALID_ARG;
  }
  if (hkv <= 0) return SD_ERR_INVALID_ARG;
  if (ncap > kMaxCapacity) return SD_ERR_UNSUPPORTED;
  return SD_OK;
}

sd_status check_problem(const sd_tensor *q, const sd_kv *K, const sd_kv *V, const sd_sparsity *sp,
                        Shape &s) {
  if (!sp) return SD_ERR_INVALID_ARG;
  sd_status st = check_q(q, s);
  if (st) return st;
  int hkv = 0;
  int64_t ncap = 0;
  st = check_kv(K, s, q->dtype, hkv, ncap);
  if (st) return st;
  if (V) {
    int hv = 0;
    int64_t nv = 0;
    st = check_kv(V, s, q->dtype, hv, nv);
    if (st) return st;
    if (V->layout != K->layout || hv != hkv || nv != ncap) return SD_ERR_INVALID_ARG;
  }
  if (s.Hq % hkv) return SD_ERR_INVALID_ARG;
  s.Hkv = hkv;
  s.paged = K->layout == SD_KV_PAGED_NHD;
  s.G = s.Hq / hkv;
  if (s.G > sd::kMaxGroup) return SD_ERR_UNSUPPORTED;
  s.ncap = ncap;
  s.R = sp->group_shared ? hkv : s.Hq;
  if (sp->k_rounding != 0 && sp->k_rounding != 1) return SD_ERR_INVALID_ARG;
  if (!sp->k_override && !(sp->ratio > 0.0 && std::isfinite(sp->ratio))) return SD_ERR_INVALID_ARG;
  if (!std::isfinite(sp->softmax_scale)) return SD_ERR_INVALID_ARG;
  if (sp->n_sink < 0 || sp->n_local < 0) return SD_ERR_INVALID_ARG;
  return SD_OK;
}

// Entries of a full-capacity row's list under the ratio rule: forced
// positions plus the top-k budget.
int64_t list_budget(int64_t L, const sd_sparsity *sp) {
  const int64_t rule = sd::budget_rule(L, sp->ratio, sp->k_rounding);
  const int Lc = (int)(L < INT32_MAX ? L : INT32_MAX);
  return sd::row_plan(Lc, sp->n_sink, sp->n_local, rule, INT32_MAX).total;
}

// idx [B, R, k_max] int32 large enough for a full-capacity sequence.
sd_status check_idx(const sd_tensor *idx, const Shape &s, const sd_sparsity *sp, int64_t &k_max) {
  if (!idx || idx->ndim != 3 || idx->dtype != SD_I32) return SD_ERR_INVALID_ARG;
  if (idx->shape[0] != s.B || idx->shape[1] != s.R || idx->shape[2] < 0) return SD_ERR_INVALID_ARG;
  k_max = idx->shape[2];
  if (k_max > 0 && !idx->data) return SD_ERR_INVALID_ARG;
  if (k_max > INT32_MAX / 2) return SD_ERR_UNSUPPORTED;
  if (!sp->k_override && k_max < list_budget(s.ncap, sp)) return SD_ERR_INVALID_ARG;
  return SD_OK;
}

sd_status check_out(const sd_tensor *out, const Shape &s, int dtype) {
  if (!out || !out->data || out->ndim != 3 || out->dtype != dtype) return SD_ERR_INVALID_ARG;
  if (out->shape[0] != s.B || out->shape[1] != s.Hq || out->shape[2] != kHeadDim)
    return SD_ERR_INVALID_ARG;
  return SD_OK;
}

// A label cache of sd::kLabels bf16 channels per key: [B][Hkv][Ncap][8]
// beside a contiguous cache, [pages][Hkv][16][8] beside a paged one.
sd_status check_labels(const sd_labels *lab, const sd_kv *K, const Shape &s) {
  if (!lab || !lab->t.data || !lab->channels || lab->t.ndim != 4) return SD_ERR_INVALID_ARG;
  if (lab->t.dtype != SD_BF16 || !s.bf16) return SD_ERR_UNSUPPORTED;
  if (lab->t.shape[3] != sd::kLabels) return SD_ERR_UNSUPPORTED;
  if (K->layout == SD_KV_BHND) {
    if (lab->t.shape[0] != s.B || lab->t.shape[1] != s.Hkv || lab->t.shape[2] != s.ncap)
      return SD_ERR_INVALID_ARG;
  } else {  // [pages][Hkv][16][8], the key pool's pages
    if (lab->t.shape[0] != K->t.shape[0] || lab->t.shape[1] != s.Hkv ||
        lab->t.shape[2] != K->page_size)
      return SD_ERR_INVALID_ARG;
  }
  return SD_OK;
}

sd::KvView kv_view(const sd_kv *kv, int hkv, int64_t ncap) {
  sd::KvView v;
  v.base = kv->t.data;
  v.block_table = kv->layout == SD_KV_PAGED_NHD ? kv->block_table : nullptr;
  v.ncap = ncap;
  v.paged = kv->layout == SD_KV_PAGED_NHD;
  v.hkv = hkv;
  v.max_pages = kv->layout == SD_KV_PAGED_NHD ? kv->max_pages_per_seq : 0;
  return v;
}

sd::Params make_params(const sd_tensor *q, const sd_kv *K, const sd_kv *V, const int32_t *seq_lens,
                       const sd_sparsity *sp, const Shape &s, int64_t k_max) {
  sd::Params p{};
  p.q = q->data;
  p.K = kv_view(K, s.Hkv, s.ncap);
  p.V = V ? kv_view(V, s.Hkv, s.ncap) : p.K;
  p.seq_lens = seq_lens;
  p.k_override = sp->k_override;
  p.ratio = sp->ratio > 0.0 ? sp->ratio : 1.0;
  p.scale = sp->softmax_scale > 0.f ? sp->softmax_scale : (float)(1.0 / std::sqrt((double)kHeadDim));
  p.B = s.B;
  p.Hq = s.Hq;
  p.Hkv = s.Hkv;
  p.G = s.G;
  p.R = s.R;
  p.bf16 = s.bf16;
  p.group_shared = sp->group_shared ? 1 : 0;
  p.rounding = sp->k_rounding;
  p.k_max = (int32_t)k_max;
  p.ncap = s.ncap;
  p.n_sink = sp->n_sink;
  p.n_local = sp->n_local;
  return p;
}

// Keys per scoring wave.  A row expects about 2.5 k / L of a wave's keys to
// pass its threshold; the wave must hold them in its staging area for the
// row, kCandBuf / rows entries, with 2x headroom.  With a sparsity ratio
// (k ~ L / ratio) the largest wave with 2 * 2.5 * wave / ratio <= area is
// taken (256 at least: rows that still do not fit are sent to the exact
// fallback by the pilot); with per-sequence k the 2048-key wave.  Label
// rows are 16 bytes, so label waves go up to 8192 keys (set-up amortised
// over as many bytes as a 512-key wave of key rows), as long as the grid
// still has 2048 waves.
int wave_keys_for(const Shape &s, const sd_sparsity *sp, int group_shared, bool labels) {
  if (sp->k_override) return sd::kWaveKeysMax;
  const int rows = group_shared ? 1 : s.G;
  const double area = (double)(sd::kCandBuf / rows);
  // Candidates per key the pilot aims at (about f k of n keys, f between 1
  // and 2.5: pilot_rank over a full-capacity sequence); a wave's expected
  // candidates must fill at most half of a row's staging area.
  double f = 2.5;
  const int64_t n = s.ncap, m = n < sd::kSampleMax ? n : sd::kSampleMax;
  const int64_t k = sd::budget_rule(n, sp->ratio, sp->k_rounding);
  if (n > 0 && k > 0 && m < n) f = (double)sd::pilot_rank(k, m, n) * n / ((double)k * m);
  int wk = labels ? sd::kLabelWaveKeysMax : sd::kWaveKeysMax;
  while (wk > 256 && 2.0 * f * wk / sp->ratio > area) wk /= 2;
  if (labels)
    while (wk > sd::kWaveKeysMax && (int64_t)s.B * s.Hkv * ((s.ncap + wk - 1) / wk) < 2048) wk /= 2;
  return wk;
}

// Workspace layout.  Sizes depend only on the shapes and the sparsity, so
// the same layout is recomputed on every call.
struct Layout {
  size_t sample, theta, dir, ckey, cpos, flags, dense, sigma, part, ustart, total;
  size_t queue, unit_pre, seq_order;
  size_t dsel_hist, dsel_state, dsel_cnt, psel_rec;
  int nchunk, wave_keys, chunk_keys, blk_cap, nsplit;
  int dsel_parts;        // pieces per row of the multi-workgroup fallback selection (0: none)
  int psel_parts;        // pieces per row of the multi-workgroup candidate selection (0: none)
  int ustride;           // chunk starts per row of the union attention (0: none)
  int union_chunk;       // positions per union-attention workgroup (0: per-row lists)
};

// The group-deduplicated attention applies to fused per-head rows whose
// logits are recomputed (label selection or forced positions), bf16 GQA.
bool union_eligible(const Shape &s, const sd_sparsity *sp, bool labels) {
  return !sp->group_shared && s.G >= 2 && s.bf16 && s.ncap > 0 &&
         (labels || sp->n_sink + sp->n_local > 0);
}

// Whether it is faster than per-head lists: each head's k_max kept rows
// (key + value, 512 B) against the expected union of G such sets of an
// Ncap-position range drawn independently (heads that agree only shrink the
// union), plus reading the heads' lists once more.  The group-row
// kernel gathers at about 0.87 of the per-head kernel's rate for up to 4
// heads (three waves per SIMD) and 0.7 for more (8 heads per pass: two
// waves), measured at 128K, so the union must move under 0.83 or 0.65 of
// the bytes.  Debug flags 4 / 8 force it off / on.
bool union_pays(const Shape &s, int64_t k_max) {
  const int dbg = g_debug.load();
  if (dbg & 4) return false;
  if (dbg & 8) return true;
  const double Lc = (double)s.ncap, G = s.G;
  const double kt = (double)(k_max < s.ncap ? k_max : s.ncap);
  const double per_head = G * kt * 512.0;
  const double uni = Lc * (1.0 - std::pow(1.0 - kt / Lc, G)) * 512.0 + 4.0 * G * kt;
  return uni < (s.G <= 4 ? 0.83 : 0.65) * per_head;
}

// Pieces per row for the fallback selection over several workgroups: about
// 2048 workgroups in all, pieces of at least 2048 positions, rows of at
// least 16K positions (shorter ones select fast enough in one workgroup);
// 0 when that leaves fewer than two pieces.
int dsel_parts_for(const Shape &s) {
  const int64_t rows = (int64_t)s.B * s.R;
  if (rows <= 0 || s.ncap < 16384) return 0;
  int64_t parts = (2048 + rows - 1) / rows;
  parts = std::min<int64_t>(parts, s.ncap / 2048);
  parts = std::min<int64_t>(parts, sd::kDselPartsMax);
  return parts >= 2 ? (int)parts : 0;
}

// Pieces per row for the candidate selection over several workgroups: rows
// too few for the 1024-thread selection to fill the GPU one each get about
// 256 workgroups in all, at most kPselPartsMax per row and at least one
// chunk and at most kPselChunksMax chunks per piece; 0 when that leaves
// fewer than two pieces.
int psel_parts_for(const Shape &s, int nchunk) {
  const int64_t rows = (int64_t)s.B * s.R;
  if (rows <= 0 || rows >= sd::kSelectWideRows || nchunk <= 0) return 0;
  int64_t parts = std::min<int64_t>(sd::kPselPartsMax, 256 / rows);
  parts = std::min<int64_t>(parts, nchunk);
  if (parts < 2 || (nchunk + parts - 1) / parts > sd::kPselChunksMax) return 0;
  return (int)parts;
}

constexpr int64_t kManyCandidates = 48 * 1024;
constexpr int64_t kPieceCandidates = 8 * 1024;  // fewest candidates per row worth the pieces
constexpr int64_t kPieceItems = 3 * 1024;       // most expected candidates per piece

// Whether the pilot would send a row of the full capacity to the exact
// fallback (its rule: the expected candidates of a scoring wave would fill
// more than half of a row's staging area), so that the call can take the
// fallback for every row without sampling or streaming first.  Per-sequence
// budgets are left to the pilot.
// cands: the candidates the pilot would pass in such a row (r n / m).
bool all_rows_fall_back(const Shape &s, const sd_sparsity *sp, int wave_keys, int64_t k_max,
                        int64_t *cands = nullptr) {
  if (cands) *cands = 0;
  if (sp->k_override || s.ncap <= 0 || s.ncap > INT32_MAX) return false;
  const sd::RowPlan rp = sd::row_plan((int)s.ncap, sp->n_sink, sp->n_local,
                                      sd::budget_rule(s.ncap, sp->ratio, sp->k_rounding),
                                      (int)std::min<int64_t>(k_max, INT32_MAX));
  const int64_t n = rp.hi - rp.lo, k = rp.kh;
  if (k <= 0 || n <= 0) return false;
  const int64_t m = n < sd::kSampleMax ? n : sd::kSampleMax;
  const int64_t r = m < n ? sd::pilot_rank(k, m, n) : k;
  if (cands) *cands = r * n / m;
  const int64_t cap = sd::kCandBuf / (sp->group_shared ? 1 : s.G);
  const int64_t span = n < wave_keys ? n : wave_keys;
  return 2 * (r - 1) * span > cap * m;
}

Layout layout_for(const Shape &s, int64_t k_max, bool fused, const sd_sparsity *sp,
                  bool labels = false, bool allow_union = true) {
  Layout L{};
  const int group_shared = sp->group_shared ? 1 : 0;
  const int64_t rows = (int64_t)s.B * s.R;
  L.wave_keys = wave_keys_for(s, sp, group_shared, labels);
  // Paged caches with a multiple of 4 KV heads are scored one head per wave
  // over shared chunks of wave_keys keys (the workgroup reads four heads of
  // each page block together), unless that makes too many chunks for the
  // selection's per-chunk tables.
  const int64_t qchunks = (s.ncap + L.wave_keys - 1) / L.wave_keys;
  const bool quad = s.paged && s.Hkv % sd::kWaves == 0 && qchunks <= 8192;
  L.chunk_keys = quad ? L.wave_keys : sd::kWaves * L.wave_keys;
  L.blk_cap = quad ? sd::kCandBuf : sd::kChunkCap;
  L.nchunk = (int)((s.ncap + L.chunk_keys - 1) / L.chunk_keys);
  sd::Params shape_only{};
  shape_only.B = s.B;
  shape_only.R = s.R;
  shape_only.G = s.G;
  shape_only.group_shared = group_shared;
  shape_only.k_max = (int32_t)k_max;
  shape_only.n_sink = sp->n_sink;
  shape_only.n_local = sp->n_local;
  L.nsplit = sd::attend_nsplit(shape_only);
  const bool uni_ok = fused && allow_union && union_eligible(s, sp, labels);
  if (uni_ok && union_pays(s, k_max)) {
    L.union_chunk = sd::union_chunk(shape_only);
    const int un = (int)((s.ncap + L.union_chunk - 1) / L.union_chunk);
    L.nsplit = un > L.nsplit ? un : L.nsplit;
  }
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += align_up(bytes);
    return o;
  };
  if (fused) {
    const size_t blocks = (size_t)s.B * s.Hkv * L.nchunk * L.blk_cap;
    L.sample = take((size_t)rows * sd::kSampleMax * 4);
    L.theta = take((size_t)rows * 8);  // thresholds, then largest samples
    L.dir = take((size_t)rows * L.nchunk * 8);
    L.ckey = take(blocks * 4);
    L.cpos = take(blocks * 2);
    L.flags = take((size_t)rows * 4);
    L.dense = take((size_t)rows * s.ncap * 4);
    L.sigma = take((size_t)rows * k_max * 4);
    L.queue = take(4);
    L.unit_pre = take((size_t)(s.B + 1) * 4);
    L.seq_order = take((size_t)s.B * 4);
    L.dsel_parts = dsel_parts_for(s);
    if (L.dsel_parts) {
      L.dsel_hist = take((size_t)rows * 2048 * 4);
      L.dsel_state = take((size_t)rows * 4 * 4);
      L.dsel_cnt = take((size_t)rows * sd::kDselPartsMax * 8);
    }
    L.psel_parts = psel_parts_for(s, L.nchunk);
    if (L.psel_parts) L.psel_rec = take((size_t)rows * L.psel_parts * sd::kPselStride * 4);
    if (uni_ok) {  // present whenever the call could use it (see union_pays)
      const int uc = sd::union_chunk(shape_only);
      L.ustride = (int)((s.ncap + uc - 1) / uc) + 1;
      L.ustart = take((size_t)rows * L.ustride * 4);
      L.nsplit = std::max<int>(L.nsplit, (int)((s.ncap + sd::union_chunk(shape_only) - 1) /
                                               sd::union_chunk(shape_only)));
    }
  }
  L.part = take((size_t)s.B * s.Hq * L.nsplit * sd::kPartStride * 4);
  L.total = off;
  return L;
}

sd_status hip_status(hipError_t e) { return e == hipSuccess ? SD_OK : SD_ERR_HIP; }

// The sparsity fields the dense path reads: none but the softmax scale.
sd_sparsity dense_sparsity(float softmax_scale) {
  sd_sparsity sp{};
  sp.ratio = 1.0;
  sp.softmax_scale = softmax_scale;
  return sp;
}

// Partials of the dense decode kernels (at least one aligned unit).
size_t dense_part_bytes(const sd::Params &p) {
  const int wk = sd::dense_wave_keys(p);
  const size_t n = (size_t)p.B * p.Hq * sd::dense_nsplit(p, wk) * sd::kPartStride * 4;
  return align_up(n > 0 ? n : 1);
}

// The current device's state, with its compute-unit count and the device
// addresses of the library's __device__ arrays (first call on a device).
sd_status device_state(DevState *&ds) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return SD_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return SD_ERR_UNSUPPORTED;
  ds = &g_dev[dev];
  if (ds->n_cu == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      return SD_ERR_HIP;
    ds->n_cu = n > 0 ? n : 1;
  }
  if (!ds->symbols) {
    void *sc = nullptr, *st = nullptr;
    if (hipGetSymbolAddress(&sc, HIP_SYMBOL(scratch)) != hipSuccess || !sc) return SD_ERR_HIP;
    if (hipGetSymbolAddress(&st, HIP_SYMBOL(stats_dev)) != hipSuccess || !st) return SD_ERR_HIP;
    ds->scratch = sc;
    ds->stats = (int32_t *)st;
    ds->symbols = true;
  }
  return SD_OK;
}

// The current device's workspace, at least `bytes` long.
sd_status get_workspace(size_t bytes, DevState *&ds, char *&base) {
  sd_status st = device_state(ds);
  if (st) return st;
  if (ds->ws_bytes < bytes) {
    if (ds->user_ws) return SD_ERR_WORKSPACE;
    if (ds->ws) {
      if (hipFree(ds->ws) != hipSuccess) return SD_ERR_HIP;
      ds->ws = nullptr;
      ds->ws_bytes = 0;
    }
    void *ptr = nullptr;
    if (hipMalloc(&ptr, bytes) != hipSuccess) return SD_ERR_WORKSPACE;
    ds->ws = ptr;
    ds->ws_bytes = bytes;
  }
  base = (char *)ds->ws;
  return SD_OK;
}

sd::Work carve(char *base, const Layout &L, bool fused, const Shape &s,
               int32_t *stats) {
  sd::Work w{};
  w.stats = stats;
  if (fused) {
    w.sample = (float *)(base + L.sample);
    w.theta = (float *)(base + L.theta);
    w.smax = w.theta + (int64_t)s.B * s.R;
    w.dir = (int2 *)(base + L.dir);
    w.ckey = (uint32_t *)(base + L.ckey);
    w.cpos = (uint16_t *)(base + L.cpos);
    w.flags = (int32_t *)(base + L.flags);
    w.dense = (float *)(base + L.dense);
    w.sigma = (float *)(base + L.sigma);
    w.queue = (int32_t *)(base + L.queue);
    w.unit_pre = (int32_t *)(base + L.unit_pre);
    w.seq_order = (int32_t *)(base + L.seq_order);
    w.unit_heads = L.chunk_keys == L.wave_keys ? s.Hkv / sd::kWaves : s.Hkv;
    if (L.dsel_parts) {
      w.dsel_hist = (uint32_t *)(base + L.dsel_hist);
      w.dsel_state = (int32_t *)(base + L.dsel_state);
      w.dsel_cnt = (int2 *)(base + L.dsel_cnt);
    }
    if (L.psel_parts) w.psel_rec = (uint32_t *)(base + L.psel_rec);
  }
  w.part = (float *)(base + L.part);
  w.ustart = L.union_chunk > 0 ? (int32_t *)(base + L.ustart) : nullptr;
  w.ustride = L.ustride;
  w.union_chunk = L.union_chunk;
  w.nchunk = L.nchunk;
  w.wave_keys = L.wave_keys;
  w.chunk_keys = L.chunk_keys;
  w.blk_cap = L.blk_cap;
  w.nsplit = L.nsplit;
  w.force_repair = (g_debug.load() & 1) ? 1 : 0;
  return w;
}

}  // namespace

extern "C" {

const char *sparse_decode_status_string(sd_status status) {
  switch (status) {
    case SD_OK: return "ok";
    case SD_ERR_INVALID_ARG: return "invalid argument";
    case SD_ERR_UNSUPPORTED: return "unsupported configuration";
    case SD_ERR_WORKSPACE: return "workspace too small or allocation failed";
    case SD_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

int64_t sparse_decode_budget(int64_t L, const sd_sparsity *sp) {
  if (!sp || !(sp->ratio > 0.0) || !std::isfinite(sp->ratio)) return -1;
  if (sp->n_sink < 0 || sp->n_local < 0) return -1;
  return list_budget(L, sp);
}

sd_status sparse_decode_set_profiling(int32_t enable) {
  std::lock_guard<std::mutex> lk(g_mu);
  g_profiling.store(enable == 2 ? 2 : (enable ? 1 : 0));
  if (enable)
    for (auto &d : g_dev) d.n_calls = 0;
  return SD_OK;
}

sd_status sparse_decode_set_debug(int32_t flags) {
  g_debug.store(flags);
  return SD_OK;
}

sd_status sparse_decode_workspace_size(const sd_tensor *q, const sd_kv *K, const sd_sparsity *sp,
                                       const sd_tensor *idx, size_t *bytes) {
  if (!bytes) return SD_ERR_INVALID_ARG;
  Shape s{};
  sd_status st = check_problem(q, K, nullptr, sp, s);
  if (st) return st;
  int64_t k_max = 0;
  st = check_idx(idx, s, sp, k_max);
  if (st) return st;
  // Enough for the exact-score and the label-indexer calls alike.
  *bytes = std::max(layout_for(s, k_max, true, sp, false).total,
                    layout_for(s, k_max, true, sp, true).total);
  return SD_OK;
}

sd_status sparse_decode_set_workspace(void *dev_ptr, size_t bytes) {
  if (dev_ptr && ((uintptr_t)dev_ptr % kAlign)) return SD_ERR_INVALID_ARG;
  std::lock_guard<std::mutex> lk(g_mu);
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return SD_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return SD_ERR_UNSUPPORTED;
  DevState &ds = g_dev[dev];
  if (ds.ws && !ds.user_ws) {
    if (hipFree(ds.ws) != hipSuccess) return SD_ERR_HIP;
  }
  ds.ws = dev_ptr;
  ds.ws_bytes = dev_ptr ? bytes : 0;
  ds.user_ws = dev_ptr != nullptr;
  return SD_OK;
}

sd_status sparse_decode_score(const sd_tensor *q, const sd_kv *K, const int32_t *seq_lens,
                              const sd_sparsity *sp, sd_tensor *scores, void *stream) {
  Shape s{};
  sd_status st = check_problem(q, K, nullptr, sp, s);
  if (st) return st;
  if (!seq_lens && s.B > 0) return SD_ERR_INVALID_ARG;
  if (!scores || scores->ndim != 3 || scores->dtype != SD_F32) return SD_ERR_INVALID_ARG;
  if (scores->shape[0] != s.B || scores->shape[1] != s.R || scores->shape[2] != s.ncap)
    return SD_ERR_INVALID_ARG;
  if (s.B == 0 || s.ncap == 0) return SD_OK;
  if (!scores->data) return SD_ERR_INVALID_ARG;
  const sd::Params p = make_params(q, K, nullptr, seq_lens, sp, s, 0);
  return hip_status(sd::launch_score_dense(p, (float *)scores->data, (hipStream_t)stream));
}

sd_status sparse_decode_topk(const sd_tensor *scores, const int32_t *seq_lens, const sd_sparsity *sp,
                             sd_tensor *idx, sd_tensor *vals, void *stream) {
  if (!sp || !scores || scores->ndim != 3 || scores->dtype != SD_F32) return SD_ERR_INVALID_ARG;
  for (int i = 0; i < 3; ++i)
    if (scores->shape[i] < 0) return SD_ERR_INVALID_ARG;
  if (scores->shape[0] > 65535 || scores->shape[1] > 65535) return SD_ERR_UNSUPPORTED;
  if (sp->k_rounding != 0 && sp->k_rounding != 1) return SD_ERR_INVALID_ARG;
  if (!sp->k_override && !(sp->ratio > 0.0 && std::isfinite(sp->ratio))) return SD_ERR_INVALID_ARG;
  if (sp->n_sink < 0 || sp->n_local < 0) return SD_ERR_INVALID_ARG;
  Shape s{};
  s.B = (int)scores->shape[0];
  s.R = (int)scores->shape[1];
  s.ncap = scores->shape[2];
  if (s.ncap > kMaxCapacity) return SD_ERR_UNSUPPORTED;
  int64_t k_max = 0;
  sd_status st = check_idx(idx, s, sp, k_max);
  if (st) return st;
  if (vals) {
    if (vals->ndim != 3 || vals->dtype != SD_F32 || vals->shape[0] != s.B ||
        vals->shape[1] != s.R || vals->shape[2] != k_max || (k_max > 0 && !vals->data))
      return SD_ERR_INVALID_ARG;
  }
  if (s.B == 0 || s.R == 0) return SD_OK;
  if (!seq_lens || (s.ncap > 0 && !scores->data)) return SD_ERR_INVALID_ARG;
  sd::Params p{};
  p.seq_lens = seq_lens;
  p.k_override = sp->k_override;
  p.ratio = sp->ratio > 0.0 ? sp->ratio : 1.0;
  p.rounding = sp->k_rounding;
  p.B = s.B;
  p.R = s.R;
  p.k_max = (int32_t)k_max;
  p.ncap = s.ncap;
  p.n_sink = sp->n_sink;
  p.n_local = sp->n_local;
  return hip_status(sd::launch_topk(p, (const float *)scores->data, (int32_t *)idx->data,
                                    vals ? (float *)vals->data : nullptr, (hipStream_t)stream));
}

sd_status sparse_decode_attend(const sd_tensor *q, const sd_kv *K, const sd_kv *V,
                               const int32_t *seq_lens, const sd_tensor *idx, const sd_sparsity *sp,
                               sd_tensor *out, void *stream) {
  Shape s{};
  sd_status st = check_problem(q, K, V, sp, s);
  if (st) return st;
  if (!V) return SD_ERR_INVALID_ARG;
  if (!idx || idx->ndim != 3 || idx->dtype != SD_I32 || idx->shape[0] != s.B ||
      idx->shape[1] != s.R || idx->shape[2] < 0)
    return SD_ERR_INVALID_ARG;
  const int64_t k_max = idx->shape[2];
  if (k_max > INT32_MAX / 2) return SD_ERR_UNSUPPORTED;
  st = check_out(out, s, q->dtype);
  if (st) return st;
  if (s.B == 0) return SD_OK;
  if (!seq_lens || (k_max > 0 && !idx->data)) return SD_ERR_INVALID_ARG;
  std::lock_guard<std::mutex> lk(g_mu);
  const Layout L = layout_for(s, k_max, false, sp);
  DevState *ds = nullptr;
  char *base = nullptr;
  st = get_workspace(L.total, ds, base);
  if (st) return st;
  const sd::Work w = carve(base, L, false, s, ds->stats);
  const sd::Params p = make_params(q, K, V, seq_lens, sp, s, k_max);
  return hip_status(sd::launch_attend(p, w, (const int32_t *)idx->data, out->data, false,
                                      (hipStream_t)stream));
}

sd_status sparse_decode_attend_weighted(const sd_tensor *q, const sd_kv *K, const sd_kv *V,
                                        const int32_t *seq_lens, const sd_tensor *idx,
                                        const sd_tensor *weights, const sd_sparsity *sp,
                                        sd_tensor *out, void *stream) {
  Shape s{};
  sd_status st = check_problem(q, K, V, sp, s);
  if (st) return st;
  if (!V) return SD_ERR_INVALID_ARG;
  if (!idx || idx->ndim != 3 || idx->dtype != SD_I32 || idx->shape[0] != s.B ||
      idx->shape[1] != s.R || idx->shape[2] < 0)
    return SD_ERR_INVALID_ARG;
  const int64_t k_max = idx->shape[2];
  if (k_max > INT32_MAX / 2) return SD_ERR_UNSUPPORTED;
  if (!weights || weights->ndim != 3 || weights->dtype != SD_F32)
    return SD_ERR_INVALID_ARG;
  for (int i = 0; i < 3; ++i)
    if (weights->shape[i] != idx->shape[i]) return SD_ERR_INVALID_ARG;
  st = check_out(out, s, q->dtype);
  if (st) return st;
  if (s.B == 0) return SD_OK;
  if (!seq_lens || (k_max > 0 && (!idx->data || !weights->data))) return SD_ERR_INVALID_ARG;
  std::lock_guard<std::mutex> lk(g_mu);
  const Layout L = layout_for(s, k_max, false, sp);
  DevState *ds = nullptr;
  char *base = nullptr;
  st = get_workspace(L.total, ds, base);
  if (st) return st;
  const sd::Work w = carve(base, L, false, s, ds->stats);
  sd::Params p = make_params(q, K, V, seq_lens, sp, s, k_max);
  p.weights = (const float *)weights->data;
  return hip_status(sd::launch_attend(p, w, (const int32_t *)idx->data, out->data, false,
                                      (hipStream_t)stream));
}

sd_status sparse_decode_dense_workspace_size(const sd_tensor *q, const sd_kv *K, size_t *bytes) {
  if (!bytes) return SD_ERR_INVALID_ARG;
  const sd_sparsity sp = dense_sparsity(0.f);
  Shape s{};
  sd_status st = check_problem(q, K, nullptr, &sp, s);
  if (st) return st;
  if (!s.bf16 || s.G > sd::kDenseMaxGroup) return SD_ERR_UNSUPPORTED;
  const sd::Params p = make_params(q, K, nullptr, nullptr, &sp, s, 0);
  *bytes = dense_part_bytes(p);
  return SD_OK;
}

sd_status sparse_decode_dense_attention(const sd_tensor *q, const sd_kv *K, const sd_kv *V,
                                        const int32_t *seq_lens, float softmax_scale,
                                        sd_tensor *out, void *stream) {
  const sd_sparsity sp = dense_sparsity(softmax_scale);
  Shape s{};
  sd_status st = check_problem(q, K, V, &sp, s);
  if (st) return st;
  if (!V) return SD_ERR_INVALID_ARG;
  if (!s.bf16 || s.G > sd::kDenseMaxGroup) return SD_ERR_UNSUPPORTED;
  st = check_out(out, s, q->dtype);
  if (st) return st;
  if (s.B == 0) return SD_OK;
  if (!seq_lens) return SD_ERR_INVALID_ARG;
  sd::Params p = make_params(q, K, V, seq_lens, &sp, s, 0);
  sd::DenseWork dw{};
  dw.wave_keys = sd::dense_wave_keys(p);
  dw.nsplit = sd::dense_nsplit(p, dw.wave_keys);
  std::lock_guard<std::mutex> lk(g_mu);
  DevState *ds = nullptr;
  char *base = nullptr;
  st = get_workspace(dense_part_bytes(p), ds, base);
  if (st) return st;
  dw.part = (float *)base;
  return hip_status(sd::launch_dense_attention(p, dw, out->data, (hipStream_t)stream));
}

}  // extern "C"

namespace {

// The fused call, with exact scores (labels null) or the low-channel
// indexer's label scores choosing the positions.
// The sampled selection's extra inputs and outputs (see
// sparse_decode_sampled_attention); null for the plain fused call.
struct Sampled {
  const uint32_t *draws;  // [B, R, n] device
  int n;
  float *weights;         // [B, R, k_max + n] device
};

sd_status attention_impl(const sd_tensor *q, const sd_kv *K, const sd_kv *V,
                         const sd_labels *labels, const int32_t *seq_lens,
                         const sd_sparsity *sp, sd_tensor *out, sd_tensor *idx, void *stream,
                         const Sampled *smp = nullptr, bool no_alloc = false) {
  Shape s{};
  sd_status st = check_problem(q, K, V, sp, s);
  if (st) return st;
  if (!V) return SD_ERR_INVALID_ARG;
  if (labels) {
    st = check_labels(labels, K, s);
    if (st) return st;
  }
  int64_t k_max = 0;  // the selection's list capacity
  int64_t k_list = 0;  // the index list's row length (k_max + draws)
  st = check_idx(idx, s, sp, k_list);
  if (st) return st;
  k_max = k_list - (smp ? smp->n : 0);
  if (k_max < 0 || (!sp->k_override && k_max < list_budget(s.ncap, sp)))
    return SD_ERR_INVALID_ARG;
  st = check_out(out, s, q->dtype);
  if (st) return st;
  if (s.B == 0) return SD_OK;
  if (!seq_lens) return SD_ERR_INVALID_ARG;
  const hipStream_t stream_h = (hipStream_t)stream;
  std::lock_guard<std::mutex> lk(g_mu);
  // (the sampled call's unfused weighted attention needs partials for the
  // whole list, and no union attention)
  const Layout L = layout_for(s, smp ? k_list : k_max, true, sp, labels != nullptr, !smp);
  // One scoring workgroup per (chunk, sequence, KV head) on a 1-D grid.
  if ((int64_t)L.nchunk * s.B * s.Hkv > INT32_MAX) return SD_ERR_UNSUPPORTED;
  DevState *ds = nullptr;
  char *base = nullptr;
  if (no_alloc) {  // the static scratch: nothing allocated, sizes beyond it refused
    st = device_state(ds);
    if (st) return st;
    if (L.total > kScratchBytes) return SD_ERR_WORKSPACE;
    base = (char *)ds->scratch;
  } else {
    st = get_workspace(L.total, ds, base);
    if (st) return st;
  }
  sd::Work w = carve(base, L, true, s, ds->stats);
  // float32 caches (small problems) take the full-score path for every row,
  // and so do calls whose rows the pilot would all send there.
  int64_t cands = 0;
  if (!s.bf16 || all_rows_fall_back(s, sp, L.wave_keys, k_max, &cands)) w.force_repair = 1;
  // So do few rows with very many candidates each (low sparsity): selecting
  // tens of thousands of candidates in one workgroup per row costs more than
  // selecting full rows over 16 or more workgroups each.
  if (L.dsel_parts >= 16 && cands >= kManyCandidates) w.force_repair = 1;
  // Those rows select over several workgroups each when they are few.
  if (w.force_repair && L.dsel_parts) w.dsel_parts = L.dsel_parts;
  sd::Params p = make_params(q, K, V, seq_lens, sp, s, k_max);
  if (labels) {
    p.labels = (const uint16_t *)labels->t.data;
    p.channels = labels->channels;
  }
  if (smp) p.idx_stride = (int32_t)k_list;
  // Exact key scores stream on one persistent workgroup per compute unit;
  // the label stream keeps one workgroup per chunk, several per compute
  // unit (with one per compute unit it was 50% slower).
  w.persistent = labels ? 0 : 1;
  w.stream_wgs = ds->n_cu;
  // (the length order is written by the pilot, which a call forced onto the
  // fallback skips: its rows keep the batch order)
  if (w.force_repair) w.seq_order = nullptr;
  int32_t *idx_ptr = (int32_t *)idx->data;

  const int prof_level = no_alloc ? 0 : g_profiling.load();  // (profiling creates events)
  const bool prof = prof_level != 0;
  if (prof && !ds->events) {
    for (auto &set : ds->ev)
      for (auto &e : set)
        if (hipEventCreate(&e) != hipSuccess) return SD_ERR_HIP;
    ds->events = true;
  }
  hipEvent_t *ev = ds->ev[ds->n_calls % kRing];
  auto mark = [&](int i) -> hipError_t {
    return prof_level == 1 ? hipEventRecord(ev[i], stream_h) : hipSuccess;
  };
  // Candidate keys the selection stages in LDS: what a full-capacity row
  // expects, f k (f the pilot's candidate factor: r n / (k m) for its rank
  // r of m samples; 2.5 at 100x, 1.2 at 5x), plus three relative
  // deviations of the count (about 1 / sqrt(r): the threshold is the r-th
  // largest sample) and 256; rows beyond it select from global memory.
  // Sized to the need, the selection fits four or more workgroups per
  // compute unit where 3.5 k + 1024 keys fitted three (ragged paged batch
  // of 8K-128K sequences at 50x: selection 60 -> 49 us).
  double fcand = 2.5, rank = 50.0;
  {
    const int64_t n = s.ncap, m = n < sd::kSampleMax ? n : sd::kSampleMax;
    const int64_t kk = sp->k_override ? k_max : sd::budget_rule(n, sp->ratio, sp->k_rounding);
    if (n > 0 && kk > 0 && m < n) {
      rank = (double)sd::pilot_rank(kk, m, n);
      fcand = rank * n / ((double)kk * m);
    }
    if (fcand < 1.0) fcand = 1.0;
    if (rank < 16.0) rank = 16.0;
  }
  const int64_t want = (int64_t)(fcand * (double)k_max * (1.0 + 3.0 / std::sqrt(rank))) + 256;
  const size_t pre_bytes = sd::select_lds_bytes(L.nchunk, 0);
  const int64_t room256 = (int64_t)sd::select_lds_budget(false) - (int64_t)pre_bytes;
  const bool wide = sd::select_wide(
      p, pre_bytes + 4 * (size_t)std::max<int64_t>(0, std::min<int64_t>(want, room256 / 4)));
  const size_t budget = sd::select_lds_budget(wide);
  if (pre_bytes >= budget) return SD_ERR_UNSUPPORTED;
  const int64_t lds_room = (int64_t)((budget - pre_bytes) / 4);
  const int lds_cap = (int)(want < lds_room ? want : lds_room);
  // Few rows with many candidates each select them over several workgroups
  // per row (unless the union attention needs each row's list read back by
  // the selection).  The pieces take about 12-16 us whatever the count; one
  // workgroup per row takes 13 us for 2.5K candidates and 26 us for 25K
  // (1M-key group-shared batch of 8 rows: 26 -> 12 us).  A piece holds at
  // most kPselItemsMax candidates (beyond, the row goes back to one
  // workgroup after the pieces' work: 128 label rows of 16K candidates in
  // two pieces each took 30 us more), so the expected count per piece must
  // stay well below it.  Debug flags 16 / 32 turn the pieces off / on
  // wherever they can apply.
  {
    const int dbg = g_debug.load();
    const bool can = L.psel_parts > 0 && wide && !w.force_repair && L.union_chunk == 0;
    const bool pays = cands >= kPieceCandidates && cands <= (int64_t)L.psel_parts * kPieceItems;
    if (can && !(dbg & 16) && (pays || (dbg & 32))) w.psel_parts = L.psel_parts;
  }
  hipError_t e = mark(0);
  // (the pilot's thresholds and flags serve only the scoring stream)
  if (e == hipSuccess && !w.force_repair) e = sd::launch_pilot(p, w, stream_h);
  if (e == hipSuccess) e = mark(1);
  // Level 2 times the scoring kernel alone, with events attached to its
  // dispatch (recorded back to back when the kernel does not run).
  const bool streams = s.ncap > 0 && !w.force_repair;
  if (e == hipSuccess && prof_level == 2 && !streams) e = hipEventRecord(ev[1], stream_h);
  if (e == hipSuccess && prof_level == 2 && !streams) e = hipEventRecord(ev[2], stream_h);
  if (e == hipSuccess && streams)
    e = prof_level == 2 ? sd::launch_score_stream(p, w, stream_h, ev[1], ev[2])
                        : sd::launch_score_stream(p, w, stream_h);
  if (e == hipSuccess) e = mark(2);
  if (e == hipSuccess && s.ncap > 0) e = sd::launch_repair(p, w, stream_h);
  if (e == hipSuccess) e = mark(3);
  if (e == hipSuccess) e = sd::launch_dense_select(p, w, idx_ptr, stream_h);
  if (e == hipSuccess) e = sd::launch_select_candidates(p, w, idx_ptr, lds_cap, wide, stream_h);
  if (e == hipSuccess && smp)
    e = sd::launch_sample_rest(p, idx_ptr, smp->draws, smp->n, smp->weights, stream_h);
  if (e == hipSuccess) e = mark(4);
  if (e == hipSuccess && !smp) e = sd::launch_attend(p, w, idx_ptr, out->data, true, stream_h);
  if (e == hipSuccess && smp) {
    // Weighted attention over the kept entries and the draws, logits
    // recomputed from the key rows.
    sd::Params pa = p;
    pa.k_max = (int32_t)k_list;
    pa.idx_stride = 0;
    pa.weights = smp->weights;
    e = sd::launch_attend(pa, w, idx_ptr, out->data, false, stream_h);
  }
  if (e == hipSuccess) e = mark(5);
  if (prof && e == hipSuccess) {
    ds->level[ds->n_calls % kRing] = prof_level;
    ds->n_calls++;
  }
  return hip_status(e);
}

}  // namespace

extern "C" {

sd_status sparse_decode_attention(const sd_tensor *q, const sd_kv *K, const sd_kv *V,
                                  const int32_t *seq_lens, const sd_sparsity *sp, sd_tensor *out,
                                  sd_tensor *idx, void *stream) {
  return attention_impl(q, K, V, nullptr, seq_lens, sp, out, idx, stream);
}

sd_status sparse_decode_attention_noalloc(const sd_tensor *q, const sd_kv *K, const sd_kv *V,
                                          const int32_t *seq_lens, const sd_sparsity *sp,
                                          sd_tensor *out, sd_tensor *idx, void *stream) {
  return attention_impl(q, K, V, nullptr, seq_lens, sp, out, idx, stream, nullptr, true);
}

sd_status sparse_decode_label_attention(const sd_tensor *q, const sd_kv *K, const sd_kv *V,
                                        const sd_labels *labels, const int32_t *seq_lens,
                                        const sd_sparsity *sp, sd_tensor *out, sd_tensor *idx,
                                        void *stream) {
  if (!labels) return SD_ERR_INVALID_ARG;
  return attention_impl(q, K, V, labels, seq_lens, sp, out, idx, stream);
}

sd_status sparse_decode_sampled_attention(const sd_tensor *q, const sd_kv *K, const sd_kv *V,
                                          const int32_t *seq_lens, const sd_sparsity *sparsity,
                                          const sd_tensor *draws, sd_tensor *out, sd_tensor *idx,
                                          sd_tensor *weights, void *stream) {
  if (!q || !draws || !idx || !weights) return SD_ERR_INVALID_ARG;
  if (draws->ndim != 3 || draws->dtype != SD_I32 || idx->ndim != 3 || weights->ndim != 3 ||
      weights->dtype != SD_F32)
    return SD_ERR_INVALID_ARG;
  const int64_t n = draws->shape[2];
  if (n < 0 || n > INT32_MAX / 4 || (n > 0 && !draws->data)) return SD_ERR_INVALID_ARG;
  for (int i = 0; i < 2; ++i)
    if (draws->shape[i] != idx->shape[i]) return SD_ERR_INVALID_ARG;
  for (int i = 0; i < 3; ++i)
    if (weights->shape[i] != idx->shape[i]) return SD_ERR_INVALID_ARG;
  if (idx->shape[2] > 0 && !weights->data) return SD_ERR_INVALID_ARG;
  if (sparsity && sparsity->group_shared) return SD_ERR_UNSUPPORTED;  // per-head rows only
  const Sampled smp{(const uint32_t *)draws->data, (int)n, (float *)weights->data};
  return attention_impl(q, K, V, nullptr, seq_lens, sparsity, out, idx, stream, &smp);
}

sd_status sparse_decode_label_score(const sd_tensor *q, const sd_kv *K, const sd_labels *labels,
                                    const int32_t *seq_lens, const sd_sparsity *sp,
                                    sd_tensor *scores, void *stream) {
  Shape s{};
  sd_status st = check_problem(q, K, nullptr, sp, s);
  if (st) return st;
  st = check_labels(labels, K, s);
  if (st) return st;
  if (!seq_lens && s.B > 0) return SD_ERR_INVALID_ARG;
  if (!scores || scores->ndim != 3 || scores->dtype != SD_F32) return SD_ERR_INVALID_ARG;
  if (scores->shape[0] != s.B || scores->shape[1] != s.R || scores->shape[2] != s.ncap)
    return SD_ERR_INVALID_ARG;
  if (s.B == 0 || s.ncap == 0) return SD_OK;
  if (!scores->data) return SD_ERR_INVALID_ARG;
  sd::Params p = make_params(q, K, nullptr, seq_lens, sp, s, 0);
  p.labels = (const uint16_t *)labels->t.data;
  p.channels = labels->channels;
  return hip_status(sd::launch_score_dense(p, (float *)scores->data, (hipStream_t)stream));
}

}  // extern "C"

namespace {

// Stage times of ring slot `slot` (its events must be complete).  A slot
// recorded at level 2 has only the scoring-stream time (t[1]); the other
// entries are 0.
sd_status read_slot(DevState &ds, int slot, float t[6]) {
  hipEvent_t *ev = ds.ev[slot];
  for (int i = 0; i < 6; ++i) t[i] = 0.f;
  if (ds.level[slot] == 2) {
    if (hipEventSynchronize(ev[2]) != hipSuccess) return SD_ERR_HIP;
    if (hipEventElapsedTime(&t[1], ev[1], ev[2]) != hipSuccess) return SD_ERR_HIP;
    return SD_OK;
  }
  if (hipEventSynchronize(ev[5]) != hipSuccess) return SD_ERR_HIP;
  for (int i = 0; i < 5; ++i)
    if (hipEventElapsedTime(&t[i], ev[i], ev[i + 1]) != hipSuccess) return SD_ERR_HIP;
  if (hipEventElapsedTime(&t[5], ev[0], ev[5]) != hipSuccess) return SD_ERR_HIP;
  return SD_OK;
}

sd_status summarize(sd_profile *out, int32_t *n_out, bool mean) {
  if (!out) return SD_ERR_INVALID_ARG;
  std::lock_guard<std::mutex> lk(g_mu);
  *out = sd_profile{};
  if (n_out) *n_out = 0;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return SD_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return SD_ERR_UNSUPPORTED;
  DevState &ds = g_dev[dev];
  if (ds.n_calls == 0) return SD_OK;
  const int64_t n = mean ? (ds.n_calls < kRing ? ds.n_calls : kRing) : 1;
  double acc[6] = {0, 0, 0, 0, 0, 0};
  for (int64_t c = ds.n_calls - n; c < ds.n_calls; ++c) {
    float t[6];
    const sd_status st = read_slot(ds, (int)(c % kRing), t);
    if (st) return st;
    for (int i = 0; i < 6; ++i) acc[i] += t[i];
  }
  out->pilot_ms = (float)(acc[0] / n);
  out->score_ms = (float)(acc[1] / n);
  out->repair_ms = (float)(acc[2] / n);  // stages run: pilot, score, repair, select, attend
  out->select_ms = (float)(acc[3] / n);
  out->attend_ms = (float)(acc[4] / n);
  out->total_ms = (float)(acc[5] / n);
  int32_t repaired = 0;
  if (ds.stats && hipMemcpy(&repaired, ds.stats, sizeof repaired, hipMemcpyDeviceToHost) != hipSuccess)
    return SD_ERR_HIP;
  out->repaired_rows = repaired;
  out->valid = 1;
  if (n_out) *n_out = (int32_t)n;
  return SD_OK;
}

}  // namespace

extern "C" {

sd_status sparse_decode_last_profile(sd_profile *out) { return summarize(out, nullptr, false); }

sd_status sparse_decode_profile_mean(sd_profile *out, int32_t *n_calls) {
  return summarize(out, n_calls, true);
}

}  // extern "C"
