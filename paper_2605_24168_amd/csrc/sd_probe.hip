// sd_probe.hip -- a plain streaming read of device memory: the same-device
// reference rate for the bandwidth-bound kernels of the library.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "sparse_decode.h"

namespace {

constexpr int kProbeThreads = 256;
constexpr int kProbeUnroll = 8;   // 16-byte loads in flight per lane
constexpr int kProbeSteps = 8;    // rounds of kProbeUnroll loads per workgroup
// 16-byte words per workgroup: one contiguous 256 KB span.
constexpr int64_t kProbeSpan = (int64_t)kProbeThreads * kProbeUnroll * kProbeSteps;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Workgroup w reads the words [w * kProbeSpan, +kProbeSpan) of p[0, n16)
// once, with nontemporal loads (the data is not reused); each load
// instruction of a wave covers 1 KB of consecutive bytes.  The XOR of the
// words decides a store that practically never happens, so the loads
// cannot be dropped and the kernel writes nothing.
__global__ __launch_bounds__(kProbeThreads) void k_read_probe(const u32x4 *p, int64_t n16,
                                                              uint32_t *sink) {
  const int64_t base = (int64_t)blockIdx.x * kProbeSpan + threadIdx.x;
  u32x4 acc = {0u, 0u, 0u, 0u};
  for (int s = 0; s < kProbeSteps; ++s) {
    const int64_t i0 = base + (int64_t)s * kProbeThreads * kProbeUnroll;
    u32x4 v[kProbeUnroll];
#pragma unroll
    for (int u = 0; u < kProbeUnroll; ++u) {
      const int64_t i = i0 + (int64_t)u * kProbeThreads;
      v[u] = i < n16 ? __builtin_nontemporal_load(p + i) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < kProbeUnroll; ++u) acc ^= v[u];
  }
  const uint32_t x = acc.x ^ acc.y ^ acc.z ^ acc.w;
  if (x == 0x9E3779B9u && threadIdx.x == 0) sink[0] = x;
}

}  // namespace

extern "C" sd_status sparse_decode_read_probe(const void *buf, size_t bytes, uint32_t *sink,
                                              void *stream) {
  if (!buf || !sink || bytes == 0 || bytes % 16 != 0 || (uintptr_t)buf % 16 != 0 ||
      (uintptr_t)sink % 4 != 0)
    return SD_ERR_INVALID_ARG;
  const int64_t n16 = (int64_t)(bytes / 16);
  const int64_t blocks = (n16 + kProbeSpan - 1) / kProbeSpan;
  if (blocks > 0x7FFFFFFF) return SD_ERR_UNSUPPORTED;
  k_read_probe<<<(unsigned)blocks, kProbeThreads, 0, (hipStream_t)stream>>>(
      (const u32x4 *)buf, n16, sink);
  return hipGetLastError() == hipSuccess ? SD_OK : SD_ERR_HIP;
}
