// HBM read probe: the rate a plain streaming read reaches on this device.
//
// The published HBM peak is not reachable by any kernel; the bandwidth-bound
// kernels of the library are better judged against what a read-only stream
// with nothing else to do achieves on the same chip.  A sweep on MI355X over
// grid size (1 to 32 workgroups per CU), loads in flight per lane (4 to 16)
// and access pattern (grid-stride, one chunk per workgroup, one row per wave)
// found the best at one 256-lane workgroup per CU, each lane streaming
// 16-byte non-temporal loads 8 at a time in a grid-stride loop; more bytes
// in flight per CU made it slower.
#include "common.hpp"

namespace moe {
namespace {

constexpr int kProbeThreads = 256;
constexpr int kProbeUnroll = 8;
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// sink is 0 on every launch; the store it guards only keeps the loads alive
__global__ __launch_bounds__(kProbeThreads) void hbm_read_probe_kernel(const u32x4 *__restrict__ p, size_t n,
                                                                      int sink, uint32_t *out) {
  const size_t tid = (size_t)blockIdx.x * kProbeThreads + threadIdx.x;
  const size_t stride = (size_t)gridDim.x * kProbeThreads;
  uint32_t acc = 0;
  size_t i = tid;
  for (; i + (kProbeUnroll - 1) * stride < n; i += kProbeUnroll * stride) {
    u32x4 v[kProbeUnroll];
#pragma unroll
    for (int u = 0; u < kProbeUnroll; ++u) v[u] = __builtin_nontemporal_load(p + i + u * stride);
#pragma unroll
    for (int u = 0; u < kProbeUnroll; ++u) acc += v[u][0] ^ v[u][1] ^ v[u][2] ^ v[u][3];
  }
  for (; i < n; i += stride) {
    const u32x4 v = __builtin_nontemporal_load(p + i);
    acc += v[0] ^ v[1] ^ v[2] ^ v[3];
  }
  if (sink) out[tid] = acc;
}

}  // namespace

hipError_t launch_hbm_read_probe(const void *buf, size_t bytes, int workgroups, hipStream_t s) {
  hipLaunchKernelGGL(hbm_read_probe_kernel, dim3(workgroups), dim3(kProbeThreads), 0, s,
                     static_cast<const u32x4 *>(buf), bytes / 16, 0, static_cast<uint32_t *>(nullptr));
  return hipGetLastError();
}

}  // namespace moe
