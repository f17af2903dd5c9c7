// Streaming-read ceiling: a plain read-reduce kernel with the statistics
// pass's access pattern (16-byte streaming vector loads, each wavefront load
// 1 KiB contiguous) and no arithmetic beyond one XOR per word.  What it reaches over
// a buffer much larger than the last-level cache is the read bandwidth the
// statistics pass is measured against.
#include "common.hpp"
#include "row_io.hpp"

namespace dsde {
namespace {

constexpr int kProbeThreads = 256;
constexpr int kProbeLoads = 8;  // 16-byte loads per thread: 32 KiB per workgroup, as a statistics unit
static_assert(kProbeThreads == 256, "four wavefronts per workgroup");

// One workgroup per 32 KiB unit, every load issued before any is used; the
// unit's XOR goes to out[unit] (one 4-byte store per 32 KiB read).
__global__ __launch_bounds__(kProbeThreads) void stream_read_kernel(const uint4 *__restrict__ p, int64_t n,
                                                                    uint32_t *__restrict__ out) {
  __shared__ uint32_t red[kProbeThreads / 64];
  const int64_t base = int64_t(blockIdx.x) * kProbeThreads * kProbeLoads + threadIdx.x;
  uint4 v[kProbeLoads];
#pragma unroll
  for (int u = 0; u < kProbeLoads; ++u) {
    const int64_t i = base + int64_t(u) * kProbeThreads;
    v[u] = stream_load(p + (i < n ? i : n - 1));  // clamped: always in bounds
  }
  uint32_t acc = 0;
#pragma unroll
  for (int u = 0; u < kProbeLoads; ++u)
    if (base + int64_t(u) * kProbeThreads < n) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) acc ^= __shfl_xor(acc, o);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) out[blockIdx.x] = red[0] ^ red[1] ^ red[2] ^ red[3];
}

}  // namespace

int launch_stream_read(const void *buf, int64_t bytes, uint32_t *out, hipStream_t stream) {
  (void)hipGetLastError();
  const int64_t n = bytes / 16;
  const int64_t per_block = int64_t(kProbeThreads) * kProbeLoads;
  const int64_t blocks = (n + per_block - 1) / per_block;
  if (blocks >= (int64_t(1) << 31)) return DSDE_INVALID_ARG;
  stream_read_kernel<<<dim3(unsigned(blocks)), dim3(kProbeThreads), 0, stream>>>((const uint4 *)buf, n, out);
  return hipGetLastError() == hipSuccess ? DSDE_OK : DSDE_DEVICE_ERROR;
}

}  // namespace dsde
