// sd_launch.hpp -- host launchers of the kernels in sd_kernels.hip.
#pragma once

#include <hip/hip_runtime.h>

#include "sd_internal.hpp"

namespace sd {

hipError_t launch_pilot(const Params &p, const Work &w, hipStream_t st);
// True when the workspace was laid out for the scoring stream to run one KV
// head per wave over shared chunks of wave_keys keys (paged layout with a
// multiple of 4 KV heads); blocks are then kCandBuf entries.
bool stream_by_head_quads(const Work &w);
// t0/t1 (both or neither): events recorded at the scoring kernel's start and
// end, attached to its dispatch.
hipError_t launch_score_stream(const Params &p, const Work &w, hipStream_t st,
                               hipEvent_t t0 = nullptr, hipEvent_t t1 = nullptr);
size_t select_lds_bytes(int nchunk, int lds_cap);
// Whether the candidate selection runs 1024-thread workgroups: when the rows
// are too few to fill the GPU one workgroup each, or when a workgroup's LDS
// (lds_bytes, at the 256-thread budget) leaves room for no second one on a
// compute unit, so that more loads are in flight per compute unit.
bool select_wide(const Params &p, size_t lds_bytes);
// Dynamic LDS available to the candidate selection at that width.
size_t select_lds_budget(bool wide);
hipError_t launch_select_candidates(const Params &p, const Work &w, int32_t *idx, int lds_cap,
                                    bool wide, hipStream_t st);
hipError_t launch_repair(const Params &p, const Work &w, hipStream_t st);
// The fallback rows' selection over w.dsel_parts workgroups per row (after
// the repair, before launch_select_candidates); nothing when dsel_parts is 0.
hipError_t launch_dense_select(const Params &p, const Work &w, int32_t *idx, hipStream_t st);
hipError_t launch_attend(const Params &p, const Work &w, const int32_t *idx, void *out, bool fused,
                         hipStream_t st);
int attend_nsplit(const Params &p);
// The sampled selection's draws and weights after the exact selection wrote
// the kept lists (p: the selection's parameters, idx_stride = k_max + s).
hipError_t launch_sample_rest(const Params &p, int32_t *list, const uint32_t *draws, int s,
                              float *weights, hipStream_t st);
// Positions per workgroup of the group-deduplicated attention (fits the LDS).
int union_chunk(const Params &p);
hipError_t launch_score_dense(const Params &p, float *scores, hipStream_t st);
hipError_t launch_topk(const Params &p, const float *scores, int32_t *idx, float *vals,
                       hipStream_t st);
// Dense decode attention over every position (bfloat16 caches).
int dense_wave_keys(const Params &p);
int dense_nsplit(const Params &p, int wave_keys);
hipError_t launch_dense_attention(const Params &p, const DenseWork &dw, void *out, hipStream_t st);

}  // namespace sd
