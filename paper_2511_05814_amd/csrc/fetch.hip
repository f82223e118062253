// Copy kernel for expert fetches (Sec. 2.2: experts stay in main memory and
// are sent to the GPU when needed).
//
// The router decides on the device which experts are missing and which slot
// each one goes to, and writes that list to device memory.  This kernel runs
// on the copy stream behind the router and reads the list itself, so no host
// round trip sits between the decision and the copy: it streams each missing
// expert with 16-byte loads straight from the pinned host store (mapped into
// the GPU's address space; one base address per layer) into its HBM slot.
// A few dozen workgroups keep enough reads in flight to saturate the host
// link while leaving the compute units to the FFN kernels.
#include "common.hpp"

#ifndef MOE_FETCH_BLOCKS
#define MOE_FETCH_BLOCKS 64
#endif

namespace moe {
namespace {

constexpr int kThreads = 256;
constexpr int kBlocks = MOE_FETCH_BLOCKS;

__global__ __launch_bounds__(kThreads) void fetch_kernel(const FetchList *list,
                                                         const uint8_t *const *layers, uint8_t *arena,
                                                         int L, int E, int S, int K, uint64_t expert_bytes,
                                                         uint64_t src_stride, uint8_t *staging, int32_t *err) {
  const int n = list->n;
  const int layer = list->layer;
  if (n < 0 || n > K || layer < 0 || layer >= L) {
    if (n != 0 && blockIdx.x == 0 && threadIdx.x == 0) *err = ERR_BAD_LIST;
    return;
  }
  const size_t nv = (staging ? src_stride : expert_bytes) / sizeof(uint4);
  const size_t stride = (size_t)gridDim.x * kThreads;
  const uint8_t *base = layers[layer];
  if (base == nullptr) {  // no mapped host store for this layer: refuse, never dereference
    if (blockIdx.x == 0 && threadIdx.x == 0) *err = ERR_BAD_LIST;
    return;
  }
  for (int i = 0; i < n; ++i) {
    const int e = list->expert[i];
    const int s = list->slot[i];
    if (e < 0 || e >= E || s < 0 || s >= S) {
      if (blockIdx.x == 0 && threadIdx.x == 0) *err = ERR_BAD_LIST;
      continue;
    }
    const uint4 *src = reinterpret_cast<const uint4 *>(base + (size_t)e * src_stride);
    uint4 *dst = reinterpret_cast<uint4 *>(staging ? staging + (size_t)i * src_stride
                                                   : arena + ((size_t)layer * S + s) * expert_bytes);
    size_t j = (size_t)blockIdx.x * kThreads + threadIdx.x;
    for (; j + 3 * stride < nv; j += 4 * stride) {
      const uint4 a = src[j], b = src[j + stride], c = src[j + 2 * stride], d = src[j + 3 * stride];
      dst[j] = a;
      dst[j + stride] = b;
      dst[j + 2 * stride] = c;
      dst[j + 3 * stride] = d;
    }
    for (; j < nv; j += stride) dst[j] = src[j];
  }
}

}  // namespace

hipError_t launch_fetch(const FetchList *list, const uint8_t *const *layers, uint8_t *arena, int L, int E,
                        int S, int K, uint64_t expert_bytes, uint64_t src_stride, uint8_t *staging,
                        int32_t *err, const Launch &l) {
  MOE_LAUNCH(fetch_kernel, dim3(kBlocks), dim3(kThreads), 0, l, list, layers, arena, L, E, S, K, expert_bytes,
             src_stride, staging, err);
  return hipGetLastError();
}

}  // namespace moe
