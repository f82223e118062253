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

// Host-to-device shader copy: the fetch kernel's access pattern (16-byte
// loads from mapped pinned host memory, four in flight a lane, grid-stride)
// over one buffer, so the host link's ceiling for a copy kernel is measured
// the same way as the runtime's DMA copy.
__global__ __launch_bounds__(kProbeThreads) void h2d_copy_probe_kernel(const uint4 *__restrict__ src,
                                                                       uint4 *__restrict__ dst, size_t nv) {
  const size_t stride = (size_t)gridDim.x * kProbeThreads;
  size_t j = (size_t)blockIdx.x * kProbeThreads + threadIdx.x;
  for (; j + 3 * stride < nv; j += 4 * stride) {
    const uint4 a = src[j], b = src[j + stride], c = src[j + 2 * stride], d = src[j + 3 * stride];
    dst[j] = a;
    dst[j + stride] = b;
    dst[j + 2 * stride] = c;
    dst[j + 3 * stride] = d;
  }
  for (; j < nv; j += stride) dst[j] = src[j];
}

// Matrix-core issue rate: every wave keeps `kChains` independent bf16 MFMA
// accumulations going on register operands, with no memory traffic, so the
// kernel is bound by the matrix cores alone.  SHAPE 0: v_mfma_f32_16x16x32_bf16
// (the prefill GEMMs' instruction, 16384 flop), 1: v_mfma_f32_32x32x16_bf16
// (32768 flop).  sink is 0 on every launch; its store keeps the results live.
typedef __bf16 probe_bf16x8 __attribute__((ext_vector_type(8)));
typedef float probe_f32x4 __attribute__((ext_vector_type(4)));
typedef float probe_f32x16 __attribute__((ext_vector_type(16)));
constexpr int kChains = 4;

template <int SHAPE>
__global__ __launch_bounds__(kProbeThreads) void mfma_bf16_probe_kernel(int iters, int sink, float *out) {
  probe_bf16x8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(float)((threadIdx.x + i) & 7);
    b[i] = (__bf16)(float)((threadIdx.x * 3 + i) & 7);
  }
  float total = 0.0f;
  if constexpr (SHAPE == 0) {
    probe_f32x4 c[kChains] = {};
    for (int it = 0; it < iters; ++it) {
#pragma unroll
      for (int k = 0; k < kChains; ++k) c[k] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c[k], 0, 0, 0);
    }
#pragma unroll
    for (int k = 0; k < kChains; ++k) total += c[k][0] + c[k][3];
  } else {
    probe_f32x16 c[kChains] = {};
    for (int it = 0; it < iters; ++it) {
#pragma unroll
      for (int k = 0; k < kChains; ++k) c[k] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c[k], 0, 0, 0);
    }
#pragma unroll
    for (int k = 0; k < kChains; ++k) total += c[k][0] + c[k][15];
  }
  if (sink) out[(size_t)blockIdx.x * kProbeThreads + threadIdx.x] = total;
}

}  // namespace

hipError_t launch_h2d_copy_probe(const void *src_dev, void *dst, size_t bytes, int workgroups, hipStream_t s) {
  hipLaunchKernelGGL(h2d_copy_probe_kernel, dim3(workgroups), dim3(kProbeThreads), 0, s,
                     static_cast<const uint4 *>(src_dev), static_cast<uint4 *>(dst), bytes / 16);
  return hipGetLastError();
}

double launch_mfma_bf16_probe(int shape, int workgroups, int iters, hipStream_t s) {
  if (shape == 0)
    hipLaunchKernelGGL(mfma_bf16_probe_kernel<0>, dim3(workgroups), dim3(kProbeThreads), 0, s, iters, 0,
                       static_cast<float *>(nullptr));
  else
    hipLaunchKernelGGL(mfma_bf16_probe_kernel<1>, dim3(workgroups), dim3(kProbeThreads), 0, s, iters, 0,
                       static_cast<float *>(nullptr));
  const double per_inst = shape == 0 ? 2.0 * 16 * 16 * 32 : 2.0 * 32 * 32 * 16;
  return per_inst * kChains * iters * (double)workgroups * (kProbeThreads / kWave);
}

hipError_t launch_hbm_read_probe(const void *buf, size_t bytes, int workgroups, hipStream_t s) {
  hipLaunchKernelGGL(hbm_read_probe_kernel, dim3(workgroups), dim3(kProbeThreads), 0, s,
                     static_cast<const u32x4 *>(buf), bytes / 16, 0, static_cast<uint32_t *>(nullptr));
  return hipGetLastError();
}

}  // namespace moe
