// sd_dense.hip -- dense decode attention over every cached position on
// gfx950: the full-attention baseline that the paper's Table 1 sets the
// sparse backend against (its FlashInfer column reads all of K and V).
//
// One wave streams one (sequence, KV head, key range) work item: the key
// tile is loaded with coalesced 1 KB instructions, re-read from LDS in the
// MFMA operand layout and scored for all G query heads of the group by one
// 16x16x32 bf16 tile; the softmax runs online per 16-key tile (running
// maximum and sum per head, rescaling the accumulators only when a maximum
// moved); the value rows of the tile are accumulated on the vector ALUs
// (16 lanes per 256-byte row, 8 channels per lane) with the tile's weights
// broadcast through LDS.  Each work item leaves a (max, sum, unnormalised
// output) partial per query head, or the finished output when one item
// covers the whole sequence; k_dense_merge combines the partials by
// log-sum-exp.  Work items of a workgroup share their keys and read four
// adjacent KV heads of each page block when the cache is paged with a
// multiple of 4 KV heads, else they are four consecutive key ranges of one
// head.
#include <hip/hip_runtime.h>

#include "sd_internal.hpp"
#include "sd_launch.hpp"

namespace sd {

// Key/value tiles in flight per wave: two, or one where the accumulators
// of 8 or 16 heads leave no room for a second.
template <int NH>
constexpr int dense_depth() { return NH >= 8 ? 1 : 2; }
constexpr int kDenseWavePages = kDenseWaveKeysMax / kTile;

template <int NH>
struct DenseLds {
  u32x4 tile[256];                // one staged key tile (4 KB)
  float pw[kTile * NH];           // the tile's weights, [key][head]
  float alpha[NH < 4 ? 4 : NH];   // rescale factors of the heads
  int32_t page[kDenseWavePages];  // page ids of the item's tiles
};

// Output rows and the item of (sequence b, KV head g, range s) of one wave.
template <bool PAGED, bool QUAD>
__device__ __forceinline__ void dense_item(const Params &p, const DenseWork &dw, int &b, int &g,
                                           int &s) {
  const int wid = (int)blockIdx.x, wv = wave_id();
  const int nc4 = (dw.nsplit + kWaves - 1) / kWaves;
  if (QUAD) {  // heads fastest: the 8 KB of a page slot are read together
    const int nq = p.Hkv / kWaves;
    g = kWaves * (wid % nq) + wv;
    s = (wid / nq) % dw.nsplit;
    b = wid / (nq * dw.nsplit);
  } else if (PAGED) {
    g = wid % p.Hkv;
    s = kWaves * ((wid / p.Hkv) % nc4) + wv;
    b = wid / (p.Hkv * nc4);
  } else {  // a head's slab swept range by range
    s = kWaves * (wid % nc4) + wv;
    g = (wid / nc4) % p.Hkv;
    b = wid / (nc4 * p.Hkv);
  }
}

template <int NH, bool PAGED, bool QUAD>
__global__ __launch_bounds__(kBlock) void k_dense_attend(Params p, DenseWork dw, void *out) {
  static_assert(NH == 1 || NH == 2 || NH == 4 || NH == 8, "heads per pass");
  constexpr int kDenseDepth = dense_depth<NH>();
  __shared__ DenseLds<NH> lds[kWaves];
  int b, g, s;
  dense_item<PAGED, QUAD>(p, dw, b, g, s);
  const int L = seq_len(p, b);
  const int64_t k0 = (int64_t)s * dw.wave_keys;
  if (s >= dw.nsplit || k0 >= L) return;  // per wave: the kernel has no block barrier
  const int nvalid = (int)((L - k0) < dw.wave_keys ? (L - k0) : dw.wave_keys);
  const int nsp = (int)((L + dw.wave_keys - 1) / dw.wave_keys);
  const int l = lane_id(), col = l & 15, a = l >> 4;
  DenseLds<NH> &wl = lds[wave_id()];
  const int G = p.G;
  QFrag qf;
  load_q_heads(p, b, g * G, G, qf);

  const int ntiles = (nvalid + kTile - 1) / kTile;
  constexpr int64_t kRowBytes = kHeadDim * 2;
  const char *kbase = (const char *)p.K.base;
  const char *vbase = (const char *)p.V.base;
  int64_t slab = 0, page_bytes = 0;
  if (PAGED) {
    const int32_t *bt = p.K.block_table + (int64_t)b * p.K.max_pages + (k0 >> 4);
    for (int i = l; i < ntiles; i += 64) wl.page[i] = bt[i];
    __builtin_amdgcn_wave_barrier();  // every lane reads every page id
    page_bytes = (int64_t)kTile * p.K.hkv * kRowBytes;
  } else {
    slab = (((int64_t)b * p.K.hkv + g) * p.K.ncap + k0) * kRowBytes;
  }
  const int last = nvalid - 1;
  // Byte offset of row r (0..15) of tile ti, rows past the end clamped to
  // the last valid one (same page: a processed tile holds a valid key).
  auto row_off = [&](int ti, int r) -> int64_t {
    int j = ti * kTile + r;
    j = j < last ? j : last;
    if (PAGED) return (int64_t)wl.page[ti] * page_bytes + ((int64_t)(j & 15) * p.K.hkv + g) * kRowBytes;
    return slab + (int64_t)j * kRowBytes;
  };
  // Tile ti (clamped to the last tile): the key rows in the swizzled order
  // the LDS staging expects, the value rows plainly (lane group a reads row
  // 4t + a, lane col its 16-byte chunk col).
  auto load_k = [&](int ti, u32x4 kv[4]) {
    ti = ti < ntiles ? ti : ntiles - 1;
#pragma unroll
    for (int t = 0; t < 4; ++t)
      kv[t] = __builtin_nontemporal_load(
          (const u32x4 *)(kbase + row_off(ti, 4 * t + a) + 16 * swz_chunk(t)));
  };
  auto load_v = [&](int ti, u32x4 vv[4]) {
    ti = ti < ntiles ? ti : ntiles - 1;
#pragma unroll
    for (int t = 0; t < 4; ++t)
      vv[t] = __builtin_nontemporal_load((const u32x4 *)(vbase + row_off(ti, 4 * t + a) + 16 * col));
  };

  // Running state.  MFMA layout: lane group a holds heads 4a + r (r = 0..3)
  // for key column col; m and the per-lane sums ls are per head.  Value
  // layout: acc[h][c] is channel 8 col + c of head h, over rows 4t + a.
  float m[4], ls[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    m[r] = -__builtin_inff();
    ls[r] = 0.f;
  }
  float acc[NH][8];
#pragma unroll
  for (int h = 0; h < NH; ++h)
#pragma unroll
    for (int c = 0; c < 8; ++c) acc[h][c] = 0.f;

  // Every step issues the same loads (tiles past the end are clamped and
  // their keys masked), so the compiler's memory waits are exact.  A slot's
  // key loads are reissued as soon as the tile is staged, its value loads
  // once the tile's rows are accumulated.
  u32x4 kb[kDenseDepth][4], vb[kDenseDepth][4];
#pragma unroll
  for (int d = 0; d < kDenseDepth; ++d) {
    load_k(d, kb[d]);
    load_v(d, vb[d]);
    __builtin_amdgcn_sched_barrier(0);
  }
  const int nsteps = (ntiles + kDenseDepth - 1) / kDenseDepth * kDenseDepth;
  const float scale = p.scale;
  for (int tb = 0; tb < nsteps; tb += kDenseDepth) {
#pragma unroll
    for (int u = 0; u < kDenseDepth; ++u) {
      const int ti = tb + u;
      stage_tile(wl.tile, kb[u]);
      load_k(ti + kDenseDepth, kb[u]);
      __builtin_amdgcn_wave_barrier();  // the tile is read back by other lanes
      KFrag kf;
      read_kfrag(wl.tile, kf);
      __builtin_amdgcn_wave_barrier();  // and overwritten by the next step
      const f32x4 sc = mfma_scores(qf, kf);

      // Logits of this lane's key, the tile maximum per head (over the 16
      // lanes of the group), and the running maximum.
      const bool live = ti * kTile + col < nvalid;
      float z[4], mt[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        z[r] = live ? scale * sc[r] : -__builtin_inff();
        mt[r] = z[r];
      }
#pragma unroll
      for (int o = 1; o < 16; o <<= 1)
#pragma unroll
        for (int r = 0; r < 4; ++r) mt[r] = fmaxf(mt[r], __shfl_xor(mt[r], o));
      bool moved = false;
#pragma unroll
      for (int r = 0; r < 4; ++r) moved |= mt[r] > m[r];
      if (__ballot(moved)) {  // wave-uniform: rescale everything to the new maxima
        float al[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float mn = fmaxf(m[r], mt[r]);
          al[r] = m[r] == -__builtin_inff() ? 0.f : expf(m[r] - mn);  // first tile: 0
          ls[r] *= al[r];
          m[r] = mn;
        }
        if (col == 0 && 4 * a < NH) {
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (4 * a + r < NH) wl.alpha[4 * a + r] = al[r];
        }
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int h = 0; h < NH; ++h) {
          const float f = wl.alpha[h];
#pragma unroll
          for (int c = 0; c < 8; ++c) acc[h][c] *= f;
        }
        __builtin_amdgcn_wave_barrier();
      }
      // Weights exp(z - m) of the tile, published as [key][head].
      float pe[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        pe[r] = live ? expf(z[r] - m[r]) : 0.f;
        ls[r] += pe[r];
      }
      if (4 * a < NH) {
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (4 * a + r < NH) wl.pw[col * NH + 4 * a + r] = pe[r];
      }
      __builtin_amdgcn_wave_barrier();
      // Value rows 4t + a of the tile, channels 8 col .. 8 col + 7.
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int row = 4 * t + a;
        float pw[NH];
#pragma unroll
        for (int h = 0; h < NH; ++h) pw[h] = wl.pw[row * NH + h];
        float v[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          v[2 * e] = bf16_to_f32(vb[u][t][e] & 0xFFFFu);
          v[2 * e + 1] = bf16_to_f32(vb[u][t][e] >> 16);
        }
#pragma unroll
        for (int h = 0; h < NH; ++h)
#pragma unroll
          for (int c = 0; c < 8; ++c) acc[h][c] = fmaf(pw[h], v[c], acc[h][c]);
      }
      load_v(ti + kDenseDepth, vb[u]);
      __builtin_amdgcn_wave_barrier();  // the weights are overwritten next tile
    }
  }

  // Sums over the 16 key columns, and accumulators over the four row groups.
#pragma unroll
  for (int o = 1; o < 16; o <<= 1)
#pragma unroll
    for (int r = 0; r < 4; ++r) ls[r] += __shfl_xor(ls[r], o);
#pragma unroll
  for (int h = 0; h < NH; ++h)
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      float v = acc[h][c];
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      acc[h][c] = v;
    }
  // Head h's (max, sum) sit in lane group h / 4, register h % 4; pass them
  // to the value layout through LDS (alpha area: max, pw area: sum).
  if (col == 0 && 4 * a < NH) {
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (4 * a + r < NH) {
        wl.alpha[4 * a + r] = m[r];
        wl.pw[4 * a + r] = ls[r];
      }
  }
  __builtin_amdgcn_wave_barrier();
  if (a == 0) {
#pragma unroll
    for (int h = 0; h < NH; ++h) {
      if (h >= G) break;
      const int64_t orow = (int64_t)b * p.Hq + (int64_t)g * G + h;
      const float sum = wl.pw[h];
      if (nsp == 1) {
        const float inv = sum > 0.f ? 1.f / sum : 0.f;
        uint16_t *op = (uint16_t *)out + orow * kHeadDim + 8 * col;
#pragma unroll
        for (int c = 0; c < 8; ++c) op[c] = f32_to_bf16_rne(acc[h][c] * inv);
      } else {
        float *pp = dw.part + (orow * dw.nsplit + s) * kPartStride;
        if (col == 0) {
          pp[0] = wl.alpha[h];
          pp[1] = sum;
        }
#pragma unroll
        for (int c = 0; c < 8; ++c) pp[2 + 8 * col + c] = acc[h][c];
      }
    }
  }
}

// Log-sum-exp merge of the key-range partials of each query head: grid =
// B * Hq, blocks of kMergeThreads.  Sequences covered by one range were
// written by k_dense_attend; empty ones get zeros here.
__global__ __launch_bounds__(kMergeThreads) void k_dense_merge(Params p, DenseWork dw, void *out) {
  __shared__ MergeShared sh;
  const int bh = blockIdx.x, b = bh / p.Hq;
  const int L = seq_len(p, b);
  const int nsp = (int)((L + dw.wave_keys - 1) / dw.wave_keys);
  const int c = threadIdx.x;
  uint16_t *op = (uint16_t *)out + (int64_t)bh * kHeadDim + c;
  if (L == 0) {
    if (c < kHeadDim) *op = 0;
    return;
  }
  if (nsp == 1) return;
  const float v = merge_partials(dw.part + (int64_t)bh * dw.nsplit * kPartStride, nsp, sh);
  if (c < kHeadDim) *op = f32_to_bf16_rne(v);
}

// ---------------------------------------------------------------------------
// Host side.
// ---------------------------------------------------------------------------
// Keys per work item: the largest power of two in [256, kDenseWaveKeysMax]
// that still gives at least one wave per SIMD (4 SIMDs on each of 256
// compute units) over the whole grid of a full-capacity batch, so short or
// few sequences are split finer.  Longer items amortise each wave's set-up
// and leave fewer partials to merge; measured on the 128K paged workload,
// 1024 waves beat 2048 or 4096 at every batch size and 512 starve batch 1.
int dense_wave_keys(const Params &p) {
  const int64_t want_waves = 4LL * 256;
  int wk = kDenseWaveKeysMax;
  while (wk > 256) {
    const int64_t items = (int64_t)p.B * p.Hkv * ((p.ncap + wk - 1) / wk);
    if (items >= want_waves) break;
    wk /= 2;
  }
  return wk;
}

int dense_nsplit(const Params &p, int wave_keys) {
  return (int)((p.ncap + wave_keys - 1) / wave_keys);
}

template <int NH>
static hipError_t launch_dense_nh(const Params &p, const DenseWork &dw, void *out, hipStream_t st) {
  const int64_t nc4 = (dw.nsplit + kWaves - 1) / kWaves;
  const bool quad = p.K.paged && p.Hkv % kWaves == 0;
  int64_t grid;
  if (quad) grid = (int64_t)p.B * (p.Hkv / kWaves) * dw.nsplit;
  else grid = (int64_t)p.B * p.Hkv * nc4;
  if (grid > INT32_MAX) return hipErrorInvalidConfiguration;
  if (grid > 0) {
    if (quad) k_dense_attend<NH, true, true><<<(unsigned)grid, kBlock, 0, st>>>(p, dw, out);
    else if (p.K.paged) k_dense_attend<NH, true, false><<<(unsigned)grid, kBlock, 0, st>>>(p, dw, out);
    else k_dense_attend<NH, false, false><<<(unsigned)grid, kBlock, 0, st>>>(p, dw, out);
  }
  k_dense_merge<<<(unsigned)(p.B * p.Hq), kMergeThreads, 0, st>>>(p, dw, out);
  return hipGetLastError();
}

hipError_t launch_dense_attention(const Params &p, const DenseWork &dw, void *out,
                                  hipStream_t st) {
  if (p.B == 0) return hipSuccess;
  if (p.G <= 1) return launch_dense_nh<1>(p, dw, out, st);
  if (p.G <= 2) return launch_dense_nh<2>(p, dw, out, st);
  if (p.G <= 4) return launch_dense_nh<4>(p, dw, out, st);
  if (p.G <= kDenseMaxGroup) return launch_dense_nh<kDenseMaxGroup>(p, dw, out, st);
  return hipErrorInvalidValue;
}

}  // namespace sd
