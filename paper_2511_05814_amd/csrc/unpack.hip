// Rebuild bf16 experts from the packed host format after their copy.
//
// A packed matrix of n weights is a run of 12560-byte blocks of 8192 weights
// (header: first exception and count; sign|mantissa bytes; 4-bit exponent
// offsets below the group maximum; one maximum exponent per group of 32),
// followed by the matrix's exceptions, ((index in block) << 8) | exponent, for
// the weights whose offset is 15 or more.  The copy puts entry i of a fetch
// list at staging + i * (3 * mat_cap); this kernel writes the identical bf16
// bits into the entry's HBM slot.  One workgroup per block, one thread per
// group of 32 weights: 48 bytes in, 64 bytes out, the rare exceptions looked
// up in the block's few entries.
#include "common.hpp"

namespace moe {
namespace {

constexpr int kThreads = 256;
constexpr int kBlockW = 8192;
constexpr int kBlockBytes = 16 + kBlockW + kBlockW / 2 + kBlockW / 32;  // 12560

__global__ __launch_bounds__(kThreads) void unpack_kernel(const FetchList *list, const uint8_t *staging,
                                                          uint8_t *arena, int L, int S, int K, uint64_t mat_cap,
                                                          uint64_t expert_bytes, uint64_t n, int32_t *err) {
  const int cnt = list->n;
  const int layer = list->layer;
  if (cnt <= 0 || cnt > K || layer < 0 || layer >= L) return;  // the copy kernel reports bad lists
  const uint64_t nb = (n + kBlockW - 1) / kBlockW;
  const uint64_t exc_cap = (mat_cap - nb * kBlockBytes) / 4;
  const uint64_t items = (uint64_t)cnt * 3 * nb;
  const int t = threadIdx.x;
  for (uint64_t it = blockIdx.x; it < items; it += gridDim.x) {
    const int i = (int)(it / (3 * nb));
    const uint64_t r = it - (uint64_t)i * 3 * nb;
    const int m = (int)(r / nb);
    const uint64_t b = r - (uint64_t)m * nb;
    const int s = list->slot[i];
    if (s < 0 || s >= S) continue;
    const uint8_t *mat = staging + ((uint64_t)i * 3 + m) * mat_cap;
    const uint8_t *blk = mat + b * kBlockBytes;
    const uint64_t w0 = b * kBlockW + (uint64_t)t * 32;  // first weight of this thread's group
    if (w0 >= n) continue;                               // n is a multiple of 64: groups are whole
    const uint32_t first = reinterpret_cast<const uint32_t *>(blk)[0];
    const uint32_t count = reinterpret_cast<const uint32_t *>(blk)[1];
    const uint4 sm0 = *reinterpret_cast<const uint4 *>(blk + 16 + 32 * t);
    const uint4 sm1 = *reinterpret_cast<const uint4 *>(blk + 16 + 32 * t + 16);
    const uint4 off = *reinterpret_cast<const uint4 *>(blk + 16 + kBlockW + 16 * t);
    const uint32_t base = blk[16 + kBlockW + kBlockW / 2 + t];
    const uint32_t smw[8] = {sm0.x, sm0.y, sm0.z, sm0.w, sm1.x, sm1.y, sm1.z, sm1.w};
    const uint32_t ofw[4] = {off.x, off.y, off.z, off.w};
    const uint32_t *exc = reinterpret_cast<const uint32_t *>(mat + nb * kBlockBytes);
    const uint32_t lo = first < exc_cap ? first : (uint32_t)exc_cap;
    const uint32_t hi = (uint64_t)lo + count < exc_cap ? lo + count : (uint32_t)exc_cap;
    uint32_t outw[16];
#pragma unroll
    for (int j = 0; j < 32; ++j) {
      const uint32_t sm = (smw[j / 4] >> (8 * (j % 4))) & 0xFFu;
      const uint32_t o = (ofw[j / 8] >> (4 * (j % 8))) & 0xFu;
      uint32_t e = base - o;
      if (o == 15) {  // exception: look the exponent up among the block's entries
        const uint32_t idx = (uint32_t)t * 32 + j;
        e = 0;
        bool found = false;
        for (uint32_t x = lo; x < hi; ++x) {
          const uint32_t v = exc[x];
          if ((v >> 8) == idx) {
            e = v & 0xFFu;
            found = true;
            break;
          }
        }
        if (!found) *err = ERR_BAD_PACK;
      }
      const uint32_t bits = ((sm & 0x80u) << 8) | ((e & 0xFFu) << 7) | (sm & 0x7Fu);
      if (j % 2 == 0)
        outw[j / 2] = bits;
      else
        outw[j / 2] |= bits << 16;
    }
    uint4 *dst = reinterpret_cast<uint4 *>(arena + ((uint64_t)layer * S + s) * expert_bytes +
                                           ((uint64_t)m * n + w0) * 2);
    dst[0] = make_uint4(outw[0], outw[1], outw[2], outw[3]);
    dst[1] = make_uint4(outw[4], outw[5], outw[6], outw[7]);
    dst[2] = make_uint4(outw[8], outw[9], outw[10], outw[11]);
    dst[3] = make_uint4(outw[12], outw[13], outw[14], outw[15]);
  }
}

}  // namespace

hipError_t launch_unpack(const FetchList *list, const uint8_t *staging, uint8_t *arena, int L, int S, int K,
                         uint64_t mat_cap, uint64_t expert_bytes, uint64_t n, int32_t *err, const Launch &l) {
  const uint64_t nb = (n + kBlockW - 1) / kBlockW;
  const uint64_t items = (uint64_t)K * 3 * nb;
  const unsigned grid = (unsigned)(items < 4096 ? items : 4096);
  MOE_LAUNCH(unpack_kernel, dim3(grid), dim3(kThreads), 0, l, list, staging, arena, L, S, K, mat_cap,
             expert_bytes, n, err);
  return hipGetLastError();
}

}  // namespace moe
