// Streaming-read probe: the read bandwidth a plain kernel reaches on this GPU, the ceiling that
// the attention kernels' achieved bandwidth is compared with.  Each workgroup reads one
// contiguous chunk with 16-byte loads, four in flight per thread.
#include "kernels_common.h"

namespace mkv {

namespace {

constexpr int kProbeThreads = 256;

__global__ __launch_bounds__(kProbeThreads) void k_probe_read(const uint4 *__restrict__ p, int64_t chunk_vec,
                                                               uint32_t *sink) {
  const uint4 *q = p + (int64_t)blockIdx.x * chunk_vec;
  uint32_t acc = 0;
  // chunk_vec is a multiple of 4 * kProbeThreads, so every load is in bounds
  for (int64_t i = threadIdx.x; i < chunk_vec; i += 4 * kProbeThreads) {
    const uint4 a = q[i], b = q[i + kProbeThreads], c = q[i + 2 * kProbeThreads], d = q[i + 3 * kProbeThreads];
    acc ^= a.x ^ a.y ^ a.z ^ a.w ^ b.x ^ b.y ^ b.z ^ b.w ^ c.x ^ c.y ^ c.z ^ c.w ^ d.x ^ d.y ^ d.z ^ d.w;
  }
  // keeps the loads alive; a per-lane address makes it a vector store
  if (acc == 0x9E3779B9u) sink[threadIdx.x] = acc;
}

}  // namespace

hipError_t launch_probe_read(const void *buf, size_t bytes, size_t chunk, uint32_t *sink, hipStream_t st) {
  const unsigned blocks = (unsigned)(bytes / chunk);
  hipLaunchKernelGGL(k_probe_read, dim3(blocks), dim3(kProbeThreads), 0, st, static_cast<const uint4 *>(buf),
                     (int64_t)(chunk / 16), sink);
  return hipGetLastError();
}

}  // namespace mkv
