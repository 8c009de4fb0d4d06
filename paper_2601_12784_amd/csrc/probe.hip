// Streaming-read probe: the bandwidth a plain kernel reaches reading a buffer
// once, the practical ceiling for HBM-bound kernels such as decode attention.
//
// Each block streams its own contiguous range; every 16-byte piece is loaded
// exactly once with a nontemporal load (the data is not reused), eight pieces
// in flight per lane, and XOR-reduced. The reduction is stored only if it
// equals an arbitrary constant, which keeps the loads live while writing
// (practically) nothing.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include "sf_internal.h"

namespace sf {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kProbeThreads = 512;
constexpr int kProbeUnroll = 8;

__global__ __launch_bounds__(kProbeThreads) void stream_read_kernel(const u32x4* __restrict__ p, uint64_t n,
                                                                     uint64_t per_block, u32x4* sink) {
  u32x4 acc = {0u, 0u, 0u, 0u};
  const uint64_t lo = uint64_t(blockIdx.x) * per_block;
  const uint64_t hi = lo + per_block < n ? lo + per_block : n;
  uint64_t i = lo + threadIdx.x;
  // all kProbeUnroll pieces of an iteration are in [lo, hi); the rest go one at a time
  for (; i + (kProbeUnroll - 1) * kProbeThreads < hi; i += kProbeUnroll * kProbeThreads) {
    u32x4 v[kProbeUnroll];
#pragma unroll
    for (int u = 0; u < kProbeUnroll; ++u) v[u] = __builtin_nontemporal_load(p + i + u * kProbeThreads);
#pragma unroll
    for (int u = 0; u < kProbeUnroll; ++u) acc ^= v[u];
  }
  for (; i < hi; i += kProbeThreads) acc ^= __builtin_nontemporal_load(p + i);
  if ((acc[0] ^ acc[1] ^ acc[2] ^ acc[3]) == 0x9E3779B9u) *sink = acc;
}

}  // namespace

hipError_t launch_stream_read(const void* buf, uint64_t bytes, void* sink, int blocks, hipStream_t stream,
                              hipEvent_t start, hipEvent_t stop) {
  const uint64_t n = bytes / 16;
  const uint64_t per_block = (n + blocks - 1) / blocks;
  const u32x4* p = static_cast<const u32x4*>(buf);
  u32x4* s = static_cast<u32x4*>(sink);
  if (start || stop)
    hipExtLaunchKernelGGL(stream_read_kernel, dim3(blocks), dim3(kProbeThreads), 0, stream, start, stop, 0, p, n,
                          per_block, s);
  else
    hipLaunchKernelGGL(stream_read_kernel, dim3(blocks), dim3(kProbeThreads), 0, stream, p, n, per_block, s);
  return hipGetLastError();
}

}  // namespace sf
