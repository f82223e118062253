// Entropy-coded bf16 experts: the host-side encoder and the GPU decoder that
// rebuilds the identical bf16 expert in its HBM slot after the copy.
//
// At batch-1 decode every miss moves a whole expert over the host link, so
// the bytes a weight costs in host memory set the decode rate.  Sign and
// mantissa of a bf16 weight carry close to 8 bits of information and are kept
// as one byte; the exponent of N(0, sigma) weights takes a handful of values
// with about 2.5 bits of entropy and is coded with a per-matrix canonical
// prefix code of at most 8 bits (optimal under that limit: package-merge;
// for N(0, sigma) weights it costs 0.07 bits a weight more than an
// unrestricted Huffman code and lets the decoder keep its table conflict-free).
//
// Matrix layout (n weights, n a multiple of 512; nspans = ceil(n / 32768)):
//   [0, 512)               256 uint16 decode entries (length << 8) | exponent,
//                          indexed by the next 8 stream bits
//   [512, +4 nspans, to 16) uint32 first stream word of each span
//   [.., +n)               (sign << 7) | mantissa per weight, weight order
//   [.., +4 cap_words)     the spans' streams
// Weight 32768 s + 512 j + 8 l + u (step j, lane l < 64, u < 8) is code
// 8 j + u of lane stream l of span s, so a wave decodes 512 consecutive
// weights per step: sign/mantissa loads and bf16 stores are contiguous
// across lanes.  A span's 64 lane streams are interleaved word by word (word
// k of lane l at span start + 64 k + l) over as many rows as its longest lane
// stream needs, so the lanes of a wave, which move through their streams at
// nearly the same pace, read nearly the same rows.
#include "common.hpp"

#include <algorithm>
#include <array>
#include <cstring>
#include <vector>

namespace moe {

constexpr int kEcMaxLen = 8;
constexpr uint64_t kEcTable = 2u << kEcMaxLen;  // bytes of the decode table
constexpr uint64_t kEcSpan = 32768;              // weights per span
constexpr int kEcLanes = 64;

__host__ __device__ inline uint64_t ec_spans(uint64_t n) { return (n + kEcSpan - 1) / kEcSpan; }

// bytes of the span-start table, padded to 16
__host__ __device__ inline uint64_t ec_starts_bytes(uint64_t n) { return (4 * ec_spans(n) + 15) / 16 * 16; }

uint64_t entropy_matrix_bytes(uint64_t n, uint64_t cap_words) {
  if (n == 0 || n % 512) return 0;
  return (kEcTable + ec_starts_bytes(n) + n + 4 * cap_words + 15) / 16 * 16;
}

// ---------------------------------------------------------------------------
// host encoder

namespace {

// Optimal prefix-code lengths of at most max_len bits (package-merge) for
// the symbols with a non-zero count; a lone symbol gets length 1.
void limited_lengths(const uint64_t *freq, int max_len, int *len) {
  std::vector<int> syms;
  for (int s = 0; s < 256; ++s) {
    len[s] = 0;
    if (freq[s]) syms.push_back(s);
  }
  const int n = (int)syms.size();
  if (n == 0) return;
  if (n == 1) {
    len[syms[0]] = 1;
    return;
  }
  std::stable_sort(syms.begin(), syms.end(), [&](int a, int b) { return freq[a] < freq[b]; });
  struct Item {
    uint64_t w;
    std::array<uint16_t, 256> use;  // times each leaf (by sorted index) is used
  };
  std::vector<Item> leaves(n);
  for (int i = 0; i < n; ++i) {
    leaves[i].w = freq[syms[i]];
    leaves[i].use.fill(0);
    leaves[i].use[i] = 1;
  }
  std::vector<Item> items = leaves, packages, merged;
  for (int level = 1; level < max_len; ++level) {
    packages.clear();
    for (size_t i = 0; i + 1 < items.size(); i += 2) {
      Item p;
      p.w = items[i].w + items[i + 1].w;
      for (int k = 0; k < n; ++k) p.use[k] = (uint16_t)(items[i].use[k] + items[i + 1].use[k]);
      packages.push_back(p);
    }
    merged.clear();
    // leaves come first among equal weights
    std::merge(leaves.begin(), leaves.end(), packages.begin(), packages.end(), std::back_inserter(merged),
               [](const Item &a, const Item &b) { return a.w < b.w; });
    items.swap(merged);
  }
  for (int i = 0; i < 2 * n - 2; ++i)
    for (int k = 0; k < n; ++k) len[syms[k]] += items[i].use[k];
}

inline void put16(uint8_t *p, uint16_t v) { std::memcpy(p, &v, 2); }
inline void put32(uint8_t *p, uint32_t v) { std::memcpy(p, &v, 4); }

}  // namespace

int entropy_pack(const uint16_t *w, uint64_t n, uint64_t cap_words, uint8_t *out, uint64_t *used,
                 const char **why) {
  if (n == 0 || n % 512) {
    *why = "n must be a positive multiple of 512";
    return -1;
  }
  uint64_t freq[256] = {0};
  for (uint64_t i = 0; i < n; ++i) ++freq[(w[i] >> 7) & 0xFF];
  int len[256];
  limited_lengths(freq, kEcMaxLen, len);
  // canonical codes, shorter first, equal lengths by symbol; stored with the
  // first bit lowest
  uint32_t code[256] = {0};
  {
    std::vector<int> order;
    for (int s = 0; s < 256; ++s)
      if (len[s]) order.push_back(s);
    std::sort(order.begin(), order.end(), [&](int a, int b) { return len[a] != len[b] ? len[a] < len[b] : a < b; });
    uint32_t c = 0;
    int prev = order.empty() ? 0 : len[order[0]];
    for (int s : order) {
      c <<= (len[s] - prev);
      prev = len[s];
      uint32_t r = 0;
      for (int b = 0; b < len[s]; ++b) r |= ((c >> b) & 1u) << (len[s] - 1 - b);
      code[s] = r;
      ++c;
    }
  }
  const uint64_t nspans = ec_spans(n);
  uint8_t *table = out;
  uint8_t *starts = out + kEcTable;
  uint8_t *sm = starts + ec_starts_bytes(n);
  uint8_t *streams = sm + n;
  for (int i = 0; i < (1 << kEcMaxLen); ++i) put16(table + 2 * i, 0);
  for (int s = 0; s < 256; ++s)
    if (len[s])
      for (uint32_t i = code[s]; i < (1u << kEcMaxLen); i += 1u << len[s])
        put16(table + 2 * i, (uint16_t)((len[s] << 8) | s));
  std::memset(starts, 0, ec_starts_bytes(n));

  uint64_t word = 0;  // first word of the current span
  std::vector<uint32_t> lane_words[kEcLanes];
  for (uint64_t sp = 0; sp < nspans; ++sp) {
    const uint64_t steps = std::min<uint64_t>(64, (n - sp * kEcSpan) / 512);
    uint64_t rows = 0;
    for (int l = 0; l < kEcLanes; ++l) {
      std::vector<uint32_t> &out_w = lane_words[l];
      out_w.clear();
      uint64_t acc = 0;
      int nb = 0;
      for (uint64_t j = 0; j < steps; ++j) {
        const uint16_t *src = w + sp * kEcSpan + j * 512 + (uint64_t)l * 8;
        for (int u = 0; u < 8; ++u) {
          const int e = (src[u] >> 7) & 0xFF;
          acc |= (uint64_t)code[e] << nb;
          nb += len[e];
          if (nb >= 32) {
            out_w.push_back((uint32_t)acc);
            acc >>= 32;
            nb -= 32;
          }
        }
      }
      if (nb > 0) out_w.push_back((uint32_t)acc);
      rows = std::max<uint64_t>(rows, out_w.size());
    }
    if (word + rows * kEcLanes > cap_words) {
      *why = "the exponent streams exceed the capacity";
      return -1;
    }
    put32(starts + 4 * sp, (uint32_t)word);
    for (uint64_t r = 0; r < rows; ++r)
      for (int l = 0; l < kEcLanes; ++l)
        put32(streams + 4 * (word + r * kEcLanes + l), r < lane_words[l].size() ? lane_words[l][r] : 0u);
    word += rows * kEcLanes;
  }
  for (uint64_t i = 0; i < n; ++i) sm[i] = (uint8_t)(((w[i] >> 8) & 0x80) | (w[i] & 0x7F));
  const uint64_t total = entropy_matrix_bytes(n, cap_words);
  std::memset(streams + 4 * word, 0, total - (uint64_t)(streams - out) - 4 * word);
  *used = word;
  return 0;
}

// ---------------------------------------------------------------------------
// GPU decoder

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kCopies = 16;  // decode-table copies: lane l reads copy l % 16
constexpr int kRing = 16;    // stream rows each lane keeps in LDS

// Workgroup b serves matrix m = (b / G) % 3 of fetch-list entry (b / G) / 3;
// its wave w decodes span kWaves (b % G) + w.
//
// A lane reads its stream with a funnel shift over two words (lo, hi) and a
// bit position below 32: the 32 bits from that position hold the next two
// codes (at most 16 bits), so at most one word leaves per pair of codes and
// at most two per step of 8 codes.  Stream words reach the lane through a
// ring of 16 rows in LDS (slot-major: the 64 lanes of a wave always hit
// distinct banks).  With W the lane's next row, a step reads rows W and W + 1
// from the ring and loads rows 2 (W / 2) + 8 and + 9 from memory (one word
// per lane, the lanes of a wave on nearly the same rows), and writes to the
// ring the two rows loaded two steps earlier.  W grows by at most two rows a
// step, so every row a step can need is in the ring, no slot is overwritten
// while still needed, and every load has two steps to arrive before anything
// waits for it; sign/mantissa bytes are loaded two steps ahead as well.  The
// decode table sits in LDS 16 times over, entry e of copy k at word 16 e + k,
// so in a half-wave of random lookups each bank serves at most two lanes.
__global__ __launch_bounds__(kThreads) void entropy_unpack_kernel(const FetchList *list, const uint8_t *staging,
                                                                  uint8_t *arena, int L, int S, int K,
                                                                  uint64_t mat_cap, uint64_t expert_bytes,
                                                                  uint64_t n, uint64_t cap_words, int G,
                                                                  int32_t *err) {
  __shared__ uint32_t lut[(1 << kEcMaxLen) * kCopies];
  __shared__ uint32_t ring[kWaves][kRing][kWave];
  const int cnt = list->n;
  const int layer = list->layer;
  if (cnt <= 0 || cnt > K || layer < 0 || layer >= L) return;  // the copy kernel reports bad lists
  const int grp = blockIdx.x / G, g = blockIdx.x % G;
  const int i = grp / 3, m = grp % 3;
  if (i >= cnt) return;
  const int slot = list->slot[i];
  if (slot < 0 || slot >= S) return;
  const uint8_t *mat = staging + ((uint64_t)i * 3 + m) * mat_cap;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  for (int k = tid; k < (1 << kEcMaxLen) * kCopies; k += kThreads)
    lut[k] = reinterpret_cast<const uint16_t *>(mat)[k / kCopies];
  __syncthreads();
  const uint64_t nspans = ec_spans(n);
  const uint64_t sp = (uint64_t)g * kWaves + wave;
  if (sp >= nspans) return;
  const uint32_t *starts = reinterpret_cast<const uint32_t *>(mat + kEcTable);
  const uint8_t *sm = mat + kEcTable + ec_starts_bytes(n);
  const uint32_t *streams = reinterpret_cast<const uint32_t *>(sm + n);
  // row r of this lane's stream, read from a clamped address
  const uint64_t first = (uint64_t)starts[sp] + lane;
  auto row = [&](uint64_t r) { return streams[min(first + r * kWave, cap_words - 1)]; };
  uint32_t(*rg)[kWave] = ring[wave];
  auto put = [&](uint64_t r, uint32_t v) { rg[r % kRing][lane] = v; };
  auto get = [&](uint64_t r) { return rg[r % kRing][lane]; };
  const uint32_t *tab = lut + (lane % kCopies);
  uint8_t *dst = arena + ((uint64_t)layer * S + slot) * expert_bytes + (uint64_t)m * n * 2;
  const int steps = (int)min((uint64_t)64, (n - sp * kEcSpan) / 512);
  {
    uint32_t v[10];
#pragma unroll
    for (int r = 0; r < 10; ++r) v[r] = row(r);
#pragma unroll
    for (int r = 0; r < 10; ++r) put(r, v[r]);
  }
  uint32_t lo = get(0), hi = get(1);
  uint64_t W = 2;  // next row to enter
  uint32_t pos = 0, lmin = 1;
  const uint8_t *smp = sm + sp * kEcSpan + (uint64_t)lane * 8;  // this lane's bytes of step 0
  // Three sets of buffers, used by the steps in turn: step j issues the
  // sign/mantissa load of step j + 2 and then its two stream rows, and
  // writes to the ring the rows step j - 2 loaded; no value still in flight
  // is ever copied (a copy would wait for the load).
  uint32_t fa[3], fb[3];
  uint64_t fr[3] = {0, 0, 0};
  uint2 smb[3];
  smb[0] = *reinterpret_cast<const uint2 *>(smp);
  smb[1] = *reinterpret_cast<const uint2 *>(smp + (steps > 1 ? 512 : 0));
  // wait for the first loads here, so that at the loop's head only the
  // previous steps' prefetches are outstanding
  asm volatile("" : : "v"(smb[0].x), "v"(smb[0].y), "v"(smb[1].x), "v"(smb[1].y));
  auto step = [&](int j, int par) {
    smb[(par + 2) % 3] = *reinterpret_cast<const uint2 *>(smp + 512 * (j + 2 < steps ? j + 2 : j));
    const uint64_t r_now = (W / 2) * 2 + 8;
    fa[par] = row(r_now);
    fb[par] = row(r_now + 1);
    fr[par] = r_now;
    const uint2 smw = smb[par];
    const uint32_t q0 = get(W), q1 = get(W + 1);
    uint32_t adv_n = 0;
    uint32_t outw[4];
#pragma unroll
    for (int pr = 0; pr < 4; ++pr) {
      const uint32_t peek = __builtin_amdgcn_alignbit(hi, lo, pos);
      const uint32_t e1 = tab[(peek & 0xFFu) * kCopies];
      const uint32_t l1 = e1 >> 8;
      const uint32_t e2 = tab[((peek >> l1) & 0xFFu) * kCopies];
      const uint32_t l2 = e2 >> 8;
      lmin = min(lmin, min(l1, l2));
      // sign and mantissa bytes of this pair to bits 0-6 and 15 of each
      // half, the two exponents to bits 7-14 of each half
      const uint32_t smword = pr < 2 ? smw.x : smw.y;
      const uint32_t y = __builtin_amdgcn_perm(0u, smword, (pr & 1) ? 0x0c030c02u : 0x0c010c00u);
      const uint32_t ex = __builtin_amdgcn_perm(e2, e1, 0x0c040c00u) << 7;  // e1 low byte, e2 low byte at 16
      outw[pr] = (y & 0x007F007Fu) | ((y & 0x00800080u) << 8) | ex;
      pos += l1 + l2;
      const bool adv = pos >= 32;
      pos -= adv ? 32 : 0;
      lo = adv ? hi : lo;
      hi = adv ? (adv_n == 0 ? q0 : q1) : hi;
      adv_n += adv ? 1 : 0;
    }
    const uint64_t base = sp * kEcSpan + (uint64_t)j * 512 + (uint64_t)lane * 8;
    *reinterpret_cast<uint4 *>(dst + 2 * base) = make_uint4(outw[0], outw[1], outw[2], outw[3]);
    if (j >= 2) {  // the rows loaded by step j - 2
      const int o = (par + 1) % 3;
      put(fr[o], fa[o]);
      put(fr[o] + 1, fb[o]);
    }
    W += adv_n;
  };
  // whole rounds of three steps in the loop (no branch inside, so the
  // compiler's wait bookkeeping at the loop head stays exact), then the rest
  int j = 0;
  for (; j + 3 <= steps; j += 3) {
    step(j, 0);
    step(j + 1, 1);
    step(j + 2, 2);
  }
  if (j < steps) step(j, 0);
  if (j + 1 < steps) step(j + 1, 1);
  if (lmin == 0) *err = ERR_BAD_PACK;
}

}  // namespace

hipError_t launch_entropy_unpack(const FetchList *list, const uint8_t *staging, uint8_t *arena, int L, int S, int K,
                                 uint64_t mat_cap, uint64_t expert_bytes, uint64_t n, uint64_t cap_words,
                                 int32_t *err, const Launch &l) {
  // one span per wave
  const int G = (int)((ec_spans(n) + kWaves - 1) / kWaves);
  MOE_LAUNCH(entropy_unpack_kernel, dim3((unsigned)(K * 3 * G)), dim3(kThreads), 0, l, list, staging, arena, L, S,
             K, mat_cap, expert_bytes, n, cap_words, G, err);
  return hipGetLastError();
}

}  // namespace moe
