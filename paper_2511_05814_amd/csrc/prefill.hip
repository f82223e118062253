// Batched prefill of T tokens through one layer.
//
// The paper's measurements cover generated tokens only (Sec. 5.1); this path
// runs a prompt's tokens through the same MoE layer at once, with the same
// per-token arithmetic, and lets the cache see the whole batch's routing:
//
//   1. gate    Z = H W_g^T in fp64 (exact products, fp64 sums), top-K per
//              token, renormalised softmax weights, x = h / rms(h) in bf16
//   2. plan    histogram of the T*K (token, rank) pairs by expert, exclusive
//              scan, scatter into expert-sorted order; the cache table takes
//              the batch at once: counts += per-expert routings, the clock
//              ticks once per pair, then the S highest-ranked experts stay
//              resident (LFU: count; aged LFU: the count aged to the batch's
//              last tick; LRU: last use; ties: resident first, lower id);
//              kept experts keep their slots, newcomers take the
//              freed slots in ascending order
//   3. experts grouped GEMMs (MFMA bf16, fp32 accumulate) on experts resident
//              at the start, while the copy stream streams every other routed
//              expert (into its new slot, or a staging ring) followed by the
//              grouped GEMMs on those; the host schedules them from the plan,
//              except with a slot for every expert, where the plan kernel
//              writes the GEMM jobs and tiles itself
//   4. unpermute  h_t += sum_r g_tr Y[pos(t, r)] in rank order (no atomics)
//
// The gate GEMM and the grouped GEMMs are dense contractions, so they run on
// the matrix cores: the gate on the fp64 ones (exact products, fp64 sums),
// the expert GEMMs (rows = pairs routed to one expert) on bf16 ones, each
// wave holding 64 x 64 output blocks: 256-row tiles of eight waves staged by
// LDS DMA for large launches, 128- or 64-row tiles of four waves otherwise,
// and a small-M kernel for groups of at most 32 rows.
#include "common.hpp"
#include "moe_offload.h"

#include <cmath>

namespace moe {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef double double4_t __attribute__((ext_vector_type(4)));

constexpr int kGateTok = 16;     // tokens per gate workgroup
constexpr int kKStep = 32;       // GEMM reduction step (one MFMA depth)

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ __forceinline__ float silu(float v) { return v / (1.0f + __expf(-v)); }

// ---------------------------------------------------------------------------
// 1. gate logits, top-K, combine weights, normalised bf16 rows
//
// Z = H W_g^T is a dense T x E x d contraction kept in fp64 (every bf16 x fp32
// product is exact there), so it runs on the fp64 matrix cores:
// v_mfma_f64_16x16x4_f64, A = 16 tokens x 4 columns, B = 4 columns x 16
// experts; lane l supplies A[l % 16][l / 16] and B[l / 16][l % 16] and gets
// back D[l / 16 + 4 v][l % 16], v = 0..3.
//
// A workgroup holds 16 tokens and all experts.  The columns are cut into
// 16-wide blocks dealt round-robin to the eight waves (two a SIMD, so one
// wave's loads and conversions overlap the other's products), so each wave
// reads a distinct eighth of H.  In a block, lane (i, kq) = (lane % 16, lane / 16)
// loads columns 4kq .. 4kq+3 of token row i and of expert row 16g + i for
// each expert group g, and MFMA step s uses column 4kq + s of both, so A and
// B always pair the same column.  The waves' partial sums meet in LDS and
// are added in wave order.
// At 4096 tokens, d 2048, 64 experts: four waves with eight blocks ahead
// 54.6 us, eight waves with two ahead 40.3 (four ahead: 43.3), sixteen with
// one 40.6.
constexpr int kGateWaves = 8;
constexpr int kGateThreads = kGateWaves * kWave;
constexpr int kGateAhead = 2;  // blocks in flight per wave

struct GateBlock {
  float4 h;              // 4 columns of this lane's token row
  uint2 w[kMaxE / 16];   // 4 bf16 columns of this lane's row in each expert group
  float4 wf[kMaxE / 16]; // fp32 gate weights instead (dtype 0)
};

// FAST (d a multiple of 16 * kGateWaves * kGateAhead): every block the loop
// multiplies lies inside d, so loads are unconditional; the look-ahead past
// the end reads the row's last columns and is never used, and rows past T or
// experts past E (clamped to the last valid one) only feed logits nobody reads.
// A guarded load would be waited for on the spot.
template <int DT, bool FAST>
__device__ __forceinline__ void gate_load(GateBlock &b, const float *hrow, const uint8_t *wbase, int ng, int k,
                                          int d, int E, int i) {
  if (FAST) {
    const int kk = min(k, d - 4);
    b.h = *reinterpret_cast<const float4 *>(hrow + kk);
#pragma unroll
    for (int g = 0; g < kMaxE / 16; ++g) {
      if (g >= ng) break;
      const int e = min(16 * g + i, E - 1);
      if (DT == 1)
        b.w[g] = *reinterpret_cast<const uint2 *>(reinterpret_cast<const uint16_t *>(wbase) + (size_t)e * d + kk);
      else
        b.wf[g] = *reinterpret_cast<const float4 *>(reinterpret_cast<const float *>(wbase) + (size_t)e * d + kk);
    }
    return;
  }
  b.h = make_float4(0.f, 0.f, 0.f, 0.f);
  if (hrow && k < d) b.h = *reinterpret_cast<const float4 *>(hrow + k);
#pragma unroll
  for (int g = 0; g < kMaxE / 16; ++g) {
    const int e = 16 * g + i;
    if (DT == 1) {
      b.w[g] = make_uint2(0, 0);
      if (g < ng && e < E && k < d)
        b.w[g] = *reinterpret_cast<const uint2 *>(reinterpret_cast<const uint16_t *>(wbase) + (size_t)e * d + k);
    } else {
      b.wf[g] = make_float4(0.f, 0.f, 0.f, 0.f);
      if (g < ng && e < E && k < d)
        b.wf[g] = *reinterpret_cast<const float4 *>(reinterpret_cast<const float *>(wbase) + (size_t)e * d + k);
    }
  }
}

template <int DT>
__device__ __forceinline__ void gate_mfma(const GateBlock &b, int ng, double4_t *acc, double &sq) {
  const double h4[4] = {b.h.x, b.h.y, b.h.z, b.h.w};
#pragma unroll
  for (int s = 0; s < 4; ++s) sq = fma(h4[s], h4[s], sq);
#pragma unroll
  for (int g = 0; g < kMaxE / 16; ++g) {
    if (g >= ng) break;
    double w4[4];
    if (DT == 1) {
      w4[0] = __uint_as_float(b.w[g].x << 16);
      w4[1] = __uint_as_float(b.w[g].x & 0xFFFF0000u);
      w4[2] = __uint_as_float(b.w[g].y << 16);
      w4[3] = __uint_as_float(b.w[g].y & 0xFFFF0000u);
    } else {
      w4[0] = b.wf[g].x;
      w4[1] = b.wf[g].y;
      w4[2] = b.wf[g].z;
      w4[3] = b.wf[g].w;
    }
#pragma unroll
    for (int s = 0; s < 4; ++s) acc[g] = __builtin_amdgcn_mfma_f64_16x16x4f64(h4[s], w4[s], acc[g], 0, 0, 0);
  }
}

template <int DT, bool FAST>
__device__ __forceinline__ void gate_partial(const PrefillArgs &a, int t0, int wave, int lane,
                                             double (*zp)[kGateTok][kMaxE], double (*rp)[kGateTok]) {
  const int d = a.d, E = a.E;
  const int i = lane % 16, kq = lane / 16;
  const int ng = (E + 15) / 16;
  const float *hrow = FAST ? a.H + (size_t)min(t0 + i, a.T - 1) * d
                           : (t0 + i < a.T ? a.H + (size_t)(t0 + i) * d : nullptr);
  const uint8_t *wbase = static_cast<const uint8_t *>(a.gate);
  double4_t acc[kMaxE / 16];
#pragma unroll
  for (int g = 0; g < kMaxE / 16; ++g) acc[g] = double4_t{0.0, 0.0, 0.0, 0.0};
  double sq = 0.0;
  const int stride = 16 * kGateWaves;
  GateBlock buf[kGateAhead];
#pragma unroll
  for (int j = 0; j < kGateAhead; ++j) gate_load<DT, FAST>(buf[j], hrow, wbase, ng, (wave + j * kGateWaves) * 16 + 4 * kq, d, E, i);
  for (int k0 = wave * 16; k0 < d; k0 += stride * kGateAhead) {
#pragma unroll
    for (int j = 0; j < kGateAhead; ++j) {
      const GateBlock cur = buf[j];
      gate_load<DT, FAST>(buf[j], hrow, wbase, ng, k0 + (j + kGateAhead) * stride + 4 * kq, d, E, i);
      gate_mfma<DT>(cur, ng, acc, sq);
    }
  }
#pragma unroll
  for (int g = 0; g < kMaxE / 16; ++g)
#pragma unroll
    for (int v = 0; v < 4; ++v)
      if (16 * g + i < E) zp[wave][kq + 4 * v][16 * g + i] = acc[g][v];
  sq += __shfl_xor(sq, 16, kWave);
  sq += __shfl_xor(sq, 32, kWave);
  if (kq == 0) rp[wave][i] = sq;
}

__global__ __launch_bounds__(kGateThreads) void prefill_gate_kernel(PrefillArgs a) {
  __shared__ double zp[kGateWaves][kGateTok][kMaxE];
  __shared__ double rp[kGateWaves][kGateTok];
  __shared__ int s_top[kGateWaves][kMaxK];
  __shared__ float s_inv[kGateTok];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int t0 = blockIdx.x * kGateTok;
  const int E = a.E, d = a.d;
  const bool fast = d % (16 * kGateWaves * kGateAhead) == 0;
  if (a.dtype == 1) {
    if (fast)
      gate_partial<1, true>(a, t0, wave, lane, zp, rp);
    else
      gate_partial<1, false>(a, t0, wave, lane, zp, rp);
  } else {
    if (fast)
      gate_partial<0, true>(a, t0, wave, lane, zp, rp);
    else
      gate_partial<0, false>(a, t0, wave, lane, zp, rp);
  }
  __syncthreads();
  // zs = zp[0] + zp[1] + ... in wave order, kept in zp[0]
  for (int x = tid; x < kGateTok * kMaxE; x += kGateThreads) {
    const int r = x / kMaxE, e = x % kMaxE;
    if (e < E) {
      double z = zp[0][r][e];
#pragma unroll
      for (int w = 1; w < kGateWaves; ++w) z += zp[w][r][e];
      zp[0][r][e] = z;
    }
  }
  if (tid < kGateTok) {
    double r = rp[0][tid];
#pragma unroll
    for (int w = 1; w < kGateWaves; ++w) r += rp[w][tid];
    rp[0][tid] = r;
    const float inv = (float)(1.0 / sqrt(r / (double)d + 1e-5));
    s_inv[tid] = inv;
    if (t0 + tid < a.T) a.inv_r[t0 + tid] = inv;
  }
  __syncthreads();
  double (*zs)[kMaxE] = zp[0];
  double *rs = rp[0];

  // top-K per token: wave w handles tokens TW w .. TW w + TW - 1
  constexpr int TW = kGateTok / kGateWaves;
  static_assert(kGateTok % kGateWaves == 0, "whole tokens per wave");
  for (int q = 0; q < TW; ++q) {
    const int r = wave * TW + q;
    const int t = t0 + r;
    if (t >= a.T) break;
    const int mine = wave_topk_lds(zs[r], E, a.K, lane, s_top[wave]);
    const double rr = sqrt(rs[r] / (double)d + 1e-5);
    const double zr = (lane < a.K) ? zs[r][mine] : 0.0;
    const double z0 = __shfl(zr, 0, kWave);
    const double ex = (lane < a.K) ? exp((zr - z0) / rr) : 0.0;
    double den = ex;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) den += __shfl_xor(den, o, kWave);
    if (lane < a.K) {
      a.ids[(size_t)t * a.K + lane] = mine;
      a.g[(size_t)t * a.K + lane] = (float)(ex / den);
    }
  }
  // normalised bf16 rows of all the workgroup's tokens, every thread taking
  // part, eight loads in flight (clamped, so none waits behind a branch); a
  // wave starts on them as soon as its tokens' top-K is written (1/r was set
  // with the sums)
  constexpr int kRowAhead = 8;
  const int nt = min(kGateTok, a.T - t0);
  const int q4 = d / 4;  // float4 per row
  const int total = nt * q4;
  for (int i0 = tid; i0 < total; i0 += kRowAhead * kGateThreads) {
    float4 v[kRowAhead];
#pragma unroll
    for (int u = 0; u < kRowAhead; ++u) {
      const int i = min(i0 + u * kGateThreads, total - 1);
      const int r = i / q4, c = (i - r * q4) * 4;
      v[u] = *reinterpret_cast<const float4 *>(a.H + (size_t)(t0 + r) * d + c);
    }
#pragma unroll
    for (int u = 0; u < kRowAhead; ++u) {
      const int i = i0 + u * kGateThreads;
      if (i < total) {
        const int r = i / q4, c = (i - r * q4) * 4;
        const float inv = s_inv[r];
        uint2 o;
        o.x = (uint32_t)f32_to_bf16_rne(v[u].x * inv) | ((uint32_t)f32_to_bf16_rne(v[u].y * inv) << 16);
        o.y = (uint32_t)f32_to_bf16_rne(v[u].z * inv) | ((uint32_t)f32_to_bf16_rne(v[u].w * inv) << 16);
        *reinterpret_cast<uint2 *>(a.xn + (size_t)(t0 + r) * d + c) = o;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// 2. sort by expert and update the layer's table for the whole batch
//
// A counting sort in one workgroup: count the pairs of each expert (LDS
// atomics that return nothing), take offsets, then give each pair the next
// position of its expert (atomics that return it).  Positions within an
// expert follow the atomics' order, which varies from run to run; nothing
// downstream depends on it, since every row of the grouped GEMMs is computed
// alone and the combine reads each (token, rank) pair through pos_of.  Each
// thread loads kPlanAhead ids before using the first.  (Placing each pair
// after the earlier pairs of its expert, with one wave's lanes of an expert
// found by ballots so no two lanes met on one counter, took 39 us against
// 22 us for these two passes at 4096 tokens of top-8 over 64 experts.)
constexpr int kPlanThreads = 1024;
constexpr int kPlanAhead = 8;

__global__ __launch_bounds__(kPlanThreads) void prefill_plan_kernel(PlanArgs a) {
  __shared__ int cnt[kMaxE], cur[kMaxE], lastp[kMaxE], offs[kMaxE];
  __shared__ int tfirst[2][kMaxE], trows[kMaxE], tlen[2];  // tile lists (when a.ntiles)
  __shared__ int bad;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int E = a.E, P = a.T * a.K;
  if (tid < kMaxE) {
    cnt[tid] = 0;
    cur[tid] = 0;
    lastp[tid] = 0;
  }
  if (tid == 0) bad = 0;
  if (a.jobs && tid < E) {  // empty until the table step below fills them in
    a.jobs[tid] = GemmJob{nullptr, 0, 0};
    if (!a.ntiles) a.tiles[tid] = GemmTile{tid, 0, 0, 0};
  }
  __syncthreads();
  for (int p0 = tid; p0 < P; p0 += kPlanAhead * kPlanThreads) {
    int ev[kPlanAhead];
#pragma unroll
    for (int u = 0; u < kPlanAhead; ++u) {
      const int p = p0 + u * kPlanThreads;
      ev[u] = p < P ? a.ids[p] : 0;
    }
#pragma unroll
    for (int u = 0; u < kPlanAhead; ++u) {
      const int p = p0 + u * kPlanThreads;
      if (p < P) {
        if (ev[u] < 0 || ev[u] >= E) {
          bad = 1;
        } else {
          atomicAdd(&cnt[ev[u]], 1);
          atomicMax(&lastp[ev[u]], p + 1);
        }
      }
    }
  }
  __syncthreads();
  if (bad) {
    if (tid == 0) {
      *a.err = ERR_BAD_LIST;
      *a.trace_out = *a.trace_in;
    }
    return;
  }
  if (wave == 0) {
    const int c = lane < E ? cnt[lane] : 0;
    int incl = c;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      const int v = __shfl_up(incl, o, kWave);
      if (lane >= o) incl += v;
    }
    if (lane < E) offs[lane] = incl - c;
    if (a.ntiles) {
      // expert e's tiles: rt row blocks in each column block; the lists'
      // first tile of each expert by the same scan
      const int rt = (c + a.tile_rows - 1) / a.tile_rows;
      int iu = rt * a.up_cb, id = rt * a.dn_cb;
#pragma unroll
      for (int o = 1; o < kWave; o <<= 1) {
        const int vu = __shfl_up(iu, o, kWave), vd = __shfl_up(id, o, kWave);
        if (lane >= o) {
          iu += vu;
          id += vd;
        }
      }
      if (lane < E) {
        trows[lane] = rt;
        tfirst[0][lane] = iu - rt * a.up_cb;
        tfirst[1][lane] = id - rt * a.dn_cb;
      }
      if (lane == kWave - 1) {
        const bool fits = iu <= a.up_cap && id <= a.dn_cap;  // the host's bound holds for any counts
        tlen[0] = fits ? iu : 0;
        tlen[1] = fits ? id : 0;
        a.ntiles[0] = tlen[0];
        a.ntiles[1] = tlen[1];
        if (!fits) *a.err = ERR_BAD_LIST;
      }
    }
  }
  __syncthreads();
  if (a.ntiles) {
    // tile i of a list belongs to the last expert whose first tile is <= i
    const int nup = tlen[0], n_all = tlen[0] + tlen[1];
    for (int i = tid; i < n_all; i += kPlanThreads) {
      const int list = i < nup ? 0 : 1;
      const int li = list == 0 ? i : i - nup;
      int lo = 0, hi = E - 1;
      while (lo < hi) {
        const int mid = (lo + hi + 1) / 2;
        if (tfirst[list][mid] <= li)
          lo = mid;
        else
          hi = mid - 1;
      }
      const int k = li - tfirst[list][lo], rt = trows[lo];
      const int cb = k / rt, mb = k - cb * rt;
      a.tiles[(list == 0 ? 0 : a.dn_first) + li] =
          GemmTile{lo, mb * a.tile_rows, cb * (list == 0 ? a.up_cols : a.dn_cols), 0};
    }
  }
  for (int p0 = tid; p0 < P; p0 += kPlanAhead * kPlanThreads) {
    int ev[kPlanAhead];
#pragma unroll
    for (int u = 0; u < kPlanAhead; ++u) {
      const int p = p0 + u * kPlanThreads;
      ev[u] = p < P ? a.ids[p] : 0;
    }
#pragma unroll
    for (int u = 0; u < kPlanAhead; ++u) {
      const int p = p0 + u * kPlanThreads;
      if (p < P) {
        const int pos = offs[ev[u]] + atomicAdd(&cur[ev[u]], 1);
        a.perm_tok[pos] = p / a.K;
        a.pos_of[p] = pos;
      }
    }
  }
  if (wave != 0) return;

  // table update: lane e = expert e
  LayerTable *T = a.table;
  const uint64_t tbase = *a.trace_in;
  const bool in_range = lane < E;
  const int slot0 = in_range ? T->expert_slot[lane] : -1;
  uint32_t count = in_range ? T->count[lane] : 0u;
  int64_t last = in_range ? T->last[lane] : 0;
  int pf = in_range ? T->pf[lane] : 0;
  const int64_t clock0 = T->clock;
  const int64_t token0 = T->lookups;
  const int n = in_range ? cnt[lane] : 0;
  const bool res_start = slot0 >= 0;
  count += (uint32_t)n;
  if (in_range && lastp[lane] > 0) last = clock0 + lastp[lane];
  const int64_t clock1 = clock0 + (int64_t)P;  // the batch's last tick

  // R*: the S highest-ranked experts, by the policy's value, then residency
  // at the batch's start, then the lower id.  Lane e counts the experts that
  // rank above it (a strict order, so the ranks are 0 .. E - 1 and S <= E of
  // them are kept).
  const uint64_t k1 = a.policy == 1   ? (uint64_t)count
                      : a.policy == 2 ? (uint64_t)aged_count(count, last, clock1, a.aging)
                                      : (uint64_t)(last + (1ll << 40));
  const int k2 = res_start ? 1 : 0;
  int above = 0;
  for (int j = 0; j < E; ++j) {
    const uint64_t o1 = ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(k1 >> 32), j) << 32) |
                        (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)k1, j);
    const int o2 = __builtin_amdgcn_readlane(k2, j);
    above += (o1 > k1 || (o1 == k1 && (o2 > k2 || (o2 == k2 && j < lane)))) ? 1 : 0;
  }
  const bool chosen = in_range && above < a.S;
  const bool newcomer = chosen && !res_start;
  const bool evicted = res_start && !chosen;
  // freed slots (ascending) are handed to newcomers (ascending id)
  unsigned long long freed = evicted ? (1ull << slot0) : 0ull;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) freed |= __shfl_xor(freed, o, kWave);
  const unsigned long long newmask = __ballot(newcomer);
  int slot1 = evicted ? -1 : slot0;
  int victim = -1;
  const int n_new = __popcll(newmask);
  unsigned long long fm = freed, nm = newmask;
  for (int i = 0; i < n_new; ++i) {
    const int s = __ffsll((long long)fm) - 1;
    const int e = __ffsll((long long)nm) - 1;
    fm &= fm - 1;
    nm &= nm - 1;
    const unsigned long long owner = __ballot(slot0 == s);
    if (lane == e) {
      slot1 = s;
      victim = owner ? __ffsll((long long)owner) - 1 : -1;
    }
  }
  const bool fetched = in_range && ((n > 0 && !res_start) || newcomer);
  int useful = 0, wasted = 0;
  if (pf) {
    if (n > 0)
      useful = 1;
    else
      wasted = 1;
  }
  const int hits = res_start ? n : 0;
  const int misses = res_start ? 0 : n;
  int sh = hits, sm = misses, su = useful, sw = wasted, sf = fetched ? 1 : 0;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    sh += __shfl_xor(sh, o, kWave);
    sm += __shfl_xor(sm, o, kWave);
    su += __shfl_xor(su, o, kWave);
    sw += __shfl_xor(sw, o, kWave);
    sf += __shfl_xor(sf, o, kWave);
  }
  if (in_range) {
    T->expert_slot[lane] = slot1;
    T->count[lane] = count;
    T->last[lane] = last;
    T->pf[lane] = 0;
    if (newcomer) T->slot_expert[slot1] = lane;
    PrefillPlan pl;
    pl.n = n;
    pl.off = offs[lane];
    pl.slot_start = slot0;
    pl.slot_after = slot1;
    pl.newcomer = newcomer ? 1 : 0;
    pl.pad[0] = pl.pad[1] = pl.pad[2] = 0;
    a.plan[lane] = pl;
    if (a.jobs) {
      // every expert with rows is resident after the batch on this path
      if (n > 0 && slot1 < 0) *a.err = ERR_BAD_LIST;
      if (slot1 >= 0) a.jobs[lane] = GemmJob{reinterpret_cast<const uint16_t *>(a.arena_layer + (size_t)slot1 * a.slot_bytes), offs[lane], n};
    }
    if (a.trace && a.trace_cap) {
      TraceRec r;
      r.kind = REC_PREFILL;
      r.token = (int32_t)token0;
      r.layer = a.layer;
      r.rank = n;
      r.expert = lane;
      r.flags = (res_start ? 1 : 0) | (chosen ? 2 : 0) | (fetched ? 4 : 0);
      r.slot = slot1;
      r.victim = newcomer ? victim : -1;
      a.trace[(tbase + lane) % a.trace_cap] = r;
    }
  }
  if (lane == 0) {
    T->clock = clock1;
    T->lookups = token0 + a.T;
    *a.trace_out = tbase + (a.trace && a.trace_cap ? (uint64_t)E : 0);
    LayerStats *st = a.stats;
    st->v[ST_HITS] += sh;
    st->v[ST_MISSES] += sm;
    st->v[ST_EVICT] += n_new;
    st->v[ST_PF_USEFUL] += su;
    st->v[ST_PF_WASTED] += sw;
    st->v[ST_LOOKUPS] += a.T;
    st->v[ST_BYTES] += (uint64_t)sf * a.expert_bytes;
  }
}

// ---------------------------------------------------------------------------
// 3. grouped GEMMs.  A rows come from the sorted pair order; B = expert
// weights stored out x in (K contiguous), so both operands are K-major.

// An LDS row holds one KS-deep slice of a row (KS = 32 or 64 bf16: 64 or
// 128 bytes, 16 or 32 of the 64 four-byte banks), so R = 128 / KS
// consecutive rows cover the banks once.  16-byte chunk c of row r sits at
// chunk c ^ ((r / R) % (KS / 8)): any 16 consecutive rows read at one chunk
// (the 16 lanes the LDS serves at once in a 16-byte read) touch all 64 banks
// once, and so do the 16 lanes of a staging write.  (With c ^ ((r / 2) % 4)
// on 64-byte rows, rows r and r + 8 collided, and bank conflicts took 37% of
// the LDS's active cycles in the grouped GEMMs.)
template <int KS>
__device__ __forceinline__ int lds_chunk(int row, int c) {
  return c ^ ((row / (128 / KS)) % (KS / 8));
}

// One MFMA 32x32x16 operand fragment for 16-deep part `h` of a K-major LDS
// tile: lane i holds row (i % 32), elements h * 16 + (i / 32) * 8 .. + 8.
template <int KS>
__device__ __forceinline__ bf16x8 lds_frag32(const uint16_t (*src)[KS], int row, int lane, int h) {
  const uint4 v = *reinterpret_cast<const uint4 *>(&src[row][lds_chunk<KS>(row, 2 * h + lane / 32) * 8]);
  bf16x8 r;
  __builtin_memcpy(&r, &v, sizeof v);
  return r;
}

// A workgroup takes a BM x BN output tile, against both W1 and W3 in the up
// projection (BN = 128) and against W2 in the down projection (BN = 256), so
// both keep the same accumulators and stage the same bytes per step.  BM is
// 256 (eight waves, one workgroup per CU) for launches with at least two such
// tiles per CU, else 128 or 64 (four waves, two or three workgroups per CU).
// The waves form a (waves / 2) x 2 grid; each owns a (BM / (waves / 2)) x
// (BN / 2) block of the tile, multiplied as 32 x 32 v_mfma_f32_32x32x16_bf16
// blocks, two per 32-deep slice.  (On MI355X a loop of nothing but 32x32x16
// bf16 MFMAs issues 2.17 PFLOP/s against 1.31 for the 16x16x32 form, and
// each 32-row fragment feeds twice the flops per LDS byte.)  A 256 x 128 up
// tile stages 32 KB per 32-deep slice for 4.2 MFLOP, half the global bytes
// per flop of a 128 x 128 one.  The next 32-deep K slice is loaded from
// global memory into registers kGemmStages slices ahead of the one
// multiplied out of LDS; LDS is double-buffered so one barrier per step
// suffices.  Every output accumulates its K slices in ascending order.
//
// The loads ahead must stay in flight across steps, so none of them is
// conditional: a row past the group's end or a column past N reads the last
// valid row instead (its outputs are not written), and a K tail (K not a
// multiple of 32; RAGGED) reads the row's last 8 elements and is zeroed when
// stored to LDS, where the wait for it happens anyway.  Loads under a branch
// leave the compiler unable to count what is outstanding, and it then waits
// for every load at each step.  The weight pointers come from the job table,
// which the compiler can only address with flat loads; those also count
// against the LDS counter, so the wait before each barrier would drain them.
// The weights are read with buffer loads instead, through a resource over the
// tile's own rows (uniform base, 32-bit byte offsets, and a record count that
// bounds every access to those rows).
constexpr int kGemmStages = 2;  // K slices loaded ahead of the one being multiplied
#ifndef MOE_GEMM_STAGES_TALL
#define MOE_GEMM_STAGES_TALL 2
#endif
#ifndef MOE_GEMM_KS_TALL
#define MOE_GEMM_KS_TALL 64
#endif
// 256-row tiles: slices loaded ahead, and slice depth (bf16 elements)
constexpr int kGemmStagesTall = MOE_GEMM_STAGES_TALL;
constexpr int kKsTall = MOE_GEMM_KS_TALL;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rows_rsrc(const uint16_t *base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t *>(base), 0, bytes, 0x00020000);
}

typedef uint32_t gemm_u32x4 __attribute__((ext_vector_type(4)));  // a 16-byte slice as a register value

__device__ __forceinline__ gemm_u32x4 buffer_load16(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_bit_cast(gemm_u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0, 0));
}

// Workgroup i runs on XCD i % 8; it takes tile (i % 8) * n / 8 + i / 8 (with
// the remainder spread over the first XCDs), so each XCD works through one
// contiguous stretch of the tile list and the tiles it runs at the same time
// share their A and B panels in that XCD's L2.
__device__ __forceinline__ int xcd_tile(int b, int n) {
  constexpr int kXcds = 8;
  const int x = b % kXcds, i = b / kXcds, per = n / kXcds, rem = n % kXcds;
  return x * per + min(x, rem) + i;
}

// Tiles in the launch's list: the grid, or the length the plan kernel wrote
// (never more than the grid, which the host sized for the longest list).
__device__ __forceinline__ int tile_count(const int32_t *dev_ntiles) {
  return dev_ntiles ? min(*dev_ntiles, (int)gridDim.x) : (int)gridDim.x;
}

// Output columns of a tile: 128 against W1 and W3 (the up projection keeps
// two accumulators per output), 256 against W2, so both hold the same number
// of accumulators and stage the same bytes per step.
template <bool UP>
constexpr int gemm_cols() {
  return UP ? 128 : 256;
}

template <bool UP, int P, int BM, int THREADS, int KS, bool RAGGED>
__global__ __launch_bounds__(THREADS, THREADS == 512 ? 1 : (BM == 64 ? 3 : 2)) void prefill_gemm_kernel(
    const GemmTile *tiles, const GemmJob *jobs, const uint16_t *a_src, const int32_t *perm_tok, void *out, int d,
    int d_ff, const int32_t *dev_ntiles) {
  constexpr int NB = UP ? 2 : 1;         // B matrices: W1 and W3, or W2
  constexpr int BN = gemm_cols<UP>();    // output columns of the tile
  constexpr int WM = THREADS / kWave / 2;  // waves along M (two along N)
  constexpr int WR = BM / WM;            // output rows per wave
  constexpr int WC = BN / 2;             // output columns per wave
  constexpr int CH = KS / 8;             // 16-byte chunks of a slice row
  constexpr int SR = THREADS / CH;       // rows one staging pass covers
  constexpr int HA = BM / SR;            // A rows each thread stages
  constexpr int HB = BN / SR;            // B rows each thread stages per matrix
  constexpr int MX = WR / 32;            // 32-row MFMA blocks per wave
  constexpr int NY = WC / 32;            // 32-column MFMA blocks per wave
  static_assert(WR % 32 == 0 && BM % SR == 0 && BN % SR == 0, "tile shape");
  __shared__ uint16_t As[2][BM][KS];
  __shared__ uint16_t Bs[2][NB][BN][KS];
  const int nt = tile_count(dev_ntiles);
  if ((int)blockIdx.x >= nt) return;  // a surplus workgroup of a device-sized list
  const GemmTile t = tiles[xcd_tile(blockIdx.x, nt)];
  const GemmJob j = jobs[t.job];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int wm = wave / 2, wn = wave % 2;
  const int K = UP ? d : d_ff;   // reduction length
  const int N = UP ? d_ff : d;   // output columns
  const int ldo = N;
  // staging: thread -> rows (tid / CH) + SR h, 16-byte chunk tid % CH
  const int r0 = tid / CH, q = tid % CH;
  if (j.nrows <= 0) return;  // no rows: nothing to clamp to (the plan makes no such tiles)
  const uint16_t *ap[HA];
#pragma unroll
  for (int h = 0; h < HA; ++h) {
    const int m = min(t.m0 + r0 + SR * h, j.nrows - 1);
    ap[h] = UP ? a_src + (size_t)perm_tok[j.row0 + m] * d : a_src + (size_t)(j.row0 + m) * d_ff;
  }
  // weight rows n0 .. n0 + nb - 1 of each B matrix (nb <= BN)
  const int nb = min(BN, N - t.n0);
  __amdgpu_buffer_rsrc_t brs[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b)
    brs[b] = rows_rsrc(j.w + (UP ? (size_t)b * d_ff * d : 2 * (size_t)d_ff * d) + (size_t)t.n0 * K,
                       (uint32_t)nb * K * 2);
  uint32_t boff[HB];
#pragma unroll
  for (int h = 0; h < HB; ++h) boff[h] = (uint32_t)min(r0 + SR * h, nb - 1) * K * 2;
  // K slices loaded ahead live in a ring of P register slots: slice t >= 1
  // sits in slot (t - 1) % P until it is stored to LDS.
  gemm_u32x4 ra[P][HA], rb[P][NB][HB];
  auto gload = [&](int slot, int k0) {
    const int k = RAGGED ? min(k0 + q * 8, K - 8) : k0 + q * 8;  // K is a multiple of 8
#pragma unroll
    for (int h = 0; h < HA; ++h) ra[slot][h] = *reinterpret_cast<const gemm_u32x4 *>(ap[h] + k);
#pragma unroll
    for (int h = 0; h < HB; ++h)
#pragma unroll
      for (int b = 0; b < NB; ++b) rb[slot][b][h] = buffer_load16(brs[b], boff[h] + 2 * k);
  };
  auto lstore = [&](int slot, int buf, int k0) {
    const bool tail = RAGGED && k0 + q * 8 >= K;
    const gemm_u32x4 zero = {0, 0, 0, 0};
#pragma unroll
    for (int h = 0; h < HA; ++h)
      *reinterpret_cast<gemm_u32x4 *>(&As[buf][r0 + SR * h][lds_chunk<KS>(r0 + SR * h, q) * 8]) =
          tail ? zero : ra[slot][h];
#pragma unroll
    for (int h = 0; h < HB; ++h)
#pragma unroll
      for (int b = 0; b < NB; ++b)
        *reinterpret_cast<gemm_u32x4 *>(&Bs[buf][b][r0 + SR * h][lds_chunk<KS>(r0 + SR * h, q) * 8]) =
            tail ? zero : rb[slot][b][h];
  };
  floatx16 c[NB][MX][NY];
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int x = 0; x < MX; ++x)
#pragma unroll
      for (int y = 0; y < NY; ++y)
#pragma unroll
        for (int i = 0; i < 16; ++i) c[b][x][y][i] = 0.0f;

  // The main loop is straight-line (every step stores a slice and loads one,
  // clamped to the last slice past the end, whose data is then never used), so
  // the compiler can keep the loads of the other ring slots in flight; the
  // last steps, which load nothing, are peeled off.
  auto mma = [&](int buf) {
#pragma unroll
    for (int h = 0; h < KS / 16; ++h) {  // the 16-deep parts of the slice, in K order
      bf16x8 af[MX];
#pragma unroll
      for (int x = 0; x < MX; ++x) af[x] = lds_frag32<KS>(As[buf], wm * WR + x * 32 + lane % 32, lane, h);
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        bf16x8 bf[NY];
#pragma unroll
        for (int y = 0; y < NY; ++y) bf[y] = lds_frag32<KS>(Bs[buf][b], wn * WC + y * 32 + lane % 32, lane, h);
#pragma unroll
        for (int x = 0; x < MX; ++x)
#pragma unroll
          for (int y = 0; y < NY; ++y)
            c[b][x][y] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[x], bf[y], c[b][x][y], 0, 0, 0);
      }
    }
  };
  const int nk = (K + KS - 1) / KS;
  // a wave whose rows all lie past the group's end stages and waits with the
  // others but skips its products
  const bool rows_here = t.m0 + wm * WR < j.nrows;
  gload(0, 0);
  lstore(0, 0, 0);
#pragma unroll
  for (int t = 1; t <= P; ++t) gload(t - 1, min(t, nk - 1) * KS);
  __syncthreads();
  int i = 0;
  for (; i + P < nk; i += P) {  // steps i .. i + P - 1, each followed by another
#pragma unroll
    for (int u = 0; u < P; ++u) {
      const int s = i + u;  // slice multiplied now, out of LDS buffer s & 1
      if (rows_here) mma(s & 1);
      lstore(u, (s & 1) ^ 1, (s + 1) * KS);            // slice s + 1 lives in slot s % P = u
      gload(u, min(s + 1 + P, nk - 1) * KS);           // slot u is free again
      __syncthreads();
    }
  }
#pragma unroll
  for (int u = 0; u < P; ++u) {  // the last nk - i <= P steps; their slices are all loaded
    const int s = i + u;
    if (s < nk) {
      if (rows_here) mma(s & 1);
      if (s + 1 < nk) lstore(u, (s & 1) ^ 1, (s + 1) * KS);
      __syncthreads();
    }
  }
  // lane i holds column i % 32 of each 32 x 32 block, rows 8 (v / 4) + 4 (i / 32) + v % 4
#pragma unroll
  for (int x = 0; x < MX; ++x)
#pragma unroll
    for (int y = 0; y < NY; ++y)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int m = t.m0 + wm * WR + x * 32 + 8 * (i / 4) + 4 * (lane / 32) + i % 4;
        if (m >= j.nrows) continue;
        const int n = t.n0 + wn * WC + y * 32 + lane % 32;
        if (n < N) {
          if (UP)
            static_cast<uint16_t *>(out)[(size_t)(j.row0 + m) * ldo + n] =
                f32_to_bf16_rne(silu(c[0][x][y][i]) * c[NB - 1][x][y][i]);
          else
            static_cast<float *>(out)[(size_t)(j.row0 + m) * ldo + n] = c[0][x][y][i];
        }
      }
}

// 256-row tiles with the operands staged by the memory system itself: every
// 16-byte load goes straight from global memory into LDS (buffer_load ...
// lds), so no register holds a slice on its way and no wave spends
// instructions storing one.  Two LDS buffers of one 64-deep slice each (64 KB:
// A 256 rows, B 256 rows) alternate: a step waits for its own slice's loads,
// meets the other waves at one barrier (after which the buffer multiplied in
// the previous step is free), issues the next slice's loads into that buffer
// and multiplies.  (Four buffers of 32-deep slices kept three slices in
// flight but met at twice as many barriers: 5-8% slower.)  One load
// instruction of a wave fills 1 KB of LDS, lane i at byte 16 i: 8 rows of 128
// bytes, so lane i fetches the chunk that the swizzle (lds_chunk) puts at its
// place, chunk (i % 8) ^ ((row / 2) % 8) of row i / 8.  The loads are issued
// as inline instructions the compiler does not track, so the waits are the
// kernel's own.  Rows past a group's end read its last row (not written); a K
// tail's chunks are fetched from an offset past the buffer's record count,
// which the hardware turns into zeros.
constexpr int kDmaStages = 2;
constexpr int kDmaKs = 64;
#ifndef MOE_GEMM_DMA_WAVES
#define MOE_GEMM_DMA_WAVES 8
#endif
// 8 waves (two a SIMD), 64 x 64 wave tiles.  Four waves with 128 x 64 tiles
// (a quarter fewer LDS reads per MFMA, the accumulators in AGPRs) measured
// slower on MI355X: 659 against 694 TFLOP/s in the 64-expert up projection.
constexpr int kDmaWaves = MOE_GEMM_DMA_WAVES;
// Offset for a chunk that must read zeros: at or past every record count used
// here (all below 2^31; the range check admits any dword that starts below the
// record count, so the offset must clear it, not merely approach it)
constexpr uint32_t kOobOffset = 0x80000000u;

typedef __attribute__((address_space(3))) void lds_void_t;

// One wave-wide 16-byte-a-lane load into LDS at lds_base + 16 * lane.  Written
// as an instruction of its own rather than the compiler's builtin: the
// compiler tracks loads in flight into LDS per array, loses track across the
// ring's loop and then waits for all of them before reading any buffer; here
// the kernel's own waits (wait_vm) are the only ones.  M0 carries the LDS
// address; the compiler sets M0 itself before any instruction of its own that
// reads it (none in this kernel: gfx9 LDS instructions do not use it).
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t r, void *lds_base, uint32_t voff) {
  const uint32_t m0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(lds_void_t *)lds_base);
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds" : : "s"(m0), "v"(voff), "s"(r) : "memory");
}

// s_waitcnt with vmcnt = N and the other counters left alone (gfx9 encoding)
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt field");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

template <bool UP, bool RAGGED, int WAVES, int BM, int KS>
__global__ __launch_bounds__(WAVES * kWave, BM == 256 ? 1 : 2) void prefill_gemm_dma_kernel(
    const GemmTile *tiles, const GemmJob *jobs, const uint16_t *a_src, uint32_t a_bytes, const int32_t *perm_tok,
    void *out, int d, int d_ff, const int32_t *dev_ntiles) {
  constexpr int S = kDmaStages;
  constexpr int NB = UP ? 2 : 1;
  constexpr int BN = gemm_cols<UP>();
  constexpr int WM = WAVES / 2, WR = BM / WM, WC = BN / 2, MX = WR / 32, NY = WC / 32;
  constexpr int CPR = KS / 8, RPI = kWave / CPR;  // 16-byte chunks a row; rows one load instruction fills
  constexpr int RPA = BM / WAVES, RPB = NB * BN / WAVES;  // A and B slice rows a wave fills
  constexpr int IPA = RPA / RPI, IPB = RPB / RPI;          // its load instructions per slice
  constexpr int LOADS = IPA + IPB;
  static_assert(WAVES == 4 || WAVES == 8, "four or eight waves");
  static_assert(NB * BN == 256, "B slice of 256 rows");
  static_assert(RPA % RPI == 0 && RPB % RPI == 0 && WR % 32 == 0, "slice rows per wave");

  // one array per ring buffer: the A slice (rows 0 .. BM - 1), then the B slice
  __shared__ uint16_t L0[BM + NB * BN][KS], L1[BM + NB * BN][KS];
  static_assert(S == 2, "the steps below are unrolled for two buffers");
  const int nt = tile_count(dev_ntiles);
  if ((int)blockIdx.x >= nt) return;  // a surplus workgroup of a device-sized list
  const GemmTile t = tiles[xcd_tile(blockIdx.x, nt)];
  const GemmJob j = jobs[t.job];
  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int wm = wave / 2, wn = wave % 2;
  const int K = UP ? d : d_ff;
  const int N = UP ? d_ff : d;
  if (j.nrows <= 0) return;  // the plan makes no such tiles

  // this lane's rows and chunks: load instruction i of the wave fills LDS
  // rows RPA wave + RPI i .. + RPI - 1 of the A slice, or RPB wave + RPI i ..
  // of the B slice
  const __amdgpu_buffer_rsrc_t ars = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t *>(a_src), 0, a_bytes,
                                                                        0x00020000);
  const int nb = min(BN, N - t.n0);
  __amdgpu_buffer_rsrc_t brs[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b)
    brs[b] = rows_rsrc(j.w + (UP ? (size_t)b * d_ff * d : 2 * (size_t)d_ff * d) + (size_t)t.n0 * K,
                       (uint32_t)nb * K * 2);
  uint32_t aoff[IPA], boff[IPB];
  int achunk[IPA], bchunk[IPB], bmat[IPB];
#pragma unroll
  for (int i = 0; i < IPA; ++i) {
    const int r = RPA * wave + lane / CPR + RPI * i;  // row of the A slice (0 .. BM - 1)
    const int c = lds_chunk<KS>(r, lane % CPR);       // the chunk the swizzle puts at this lane's place
    const int m = min(t.m0 + r, j.nrows - 1);
    const size_t arow = UP ? (size_t)perm_tok[j.row0 + m] * d : (size_t)(j.row0 + m) * d_ff;
    aoff[i] = (uint32_t)(arow * 2) + 16u * c;
    achunk[i] = c;
  }
#pragma unroll
  for (int i = 0; i < IPB; ++i) {
    const int r = RPB * wave + lane / CPR + RPI * i;  // row of the B slice (0..255)
    const int c = lds_chunk<KS>(r, lane % CPR);
    boff[i] = (uint32_t)min(r % BN, nb - 1) * K * 2 + 16u * c;
    bchunk[i] = c;
    bmat[i] = (RPB * wave + RPI * i) / BN;  // B matrix of the instruction (uniform)
  }

  auto issue = [&](int k0, uint16_t (*As)[KS], uint16_t (*Bs)[KS]) {
#pragma unroll
    for (int i = 0; i < IPA; ++i) {
      const bool oob_a = RAGGED && k0 + 8 * achunk[i] >= K;
      dma16(ars, &As[RPA * wave + RPI * i][0], oob_a ? kOobOffset : aoff[i] + 2u * k0);
    }
#pragma unroll
    for (int i = 0; i < IPB; ++i) {
      const bool oob_b = RAGGED && k0 + 8 * bchunk[i] >= K;
      const __amdgpu_buffer_rsrc_t r = bmat[i] == 0 ? brs[0] : brs[NB - 1];
      dma16(r, &Bs[RPB * wave + RPI * i][0], oob_b ? kOobOffset : boff[i] + 2u * k0);
    }
  };

  floatx16 c[NB][MX][NY];
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int x = 0; x < MX; ++x)
#pragma unroll
      for (int y = 0; y < NY; ++y)
#pragma unroll
        for (int i = 0; i < 16; ++i) c[b][x][y][i] = 0.0f;

  auto mma = [&](const uint16_t (*As)[KS], const uint16_t (*Bs)[KS]) {
#pragma unroll
    for (int h = 0; h < KS / 16; ++h) {
      bf16x8 af[MX];
#pragma unroll
      for (int x = 0; x < MX; ++x) af[x] = lds_frag32<KS>(As, wm * WR + x * 32 + lane % 32, lane, h);
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        bf16x8 bf[NY];
#pragma unroll
        for (int y = 0; y < NY; ++y) bf[y] = lds_frag32<KS>(Bs + b * BN, wn * WC + y * 32 + lane % 32, lane, h);
#pragma unroll
        for (int x = 0; x < MX; ++x)
#pragma unroll
          for (int y = 0; y < NY; ++y)
            c[b][x][y] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[x], bf[y], c[b][x][y], 0, 0, 0);
      }
    }
  };

  const int nk = (K + KS - 1) / KS;
  // A wave whose rows all lie past the group's end (the last tile of an
  // expert) still stages its share of every slice and meets the others at the
  // barriers, but skips its products: its SIMD's matrix core then serves the
  // other wave on it alone.
  const bool rows_here = t.m0 + wm * WR < j.nrows;
  // slices 0 .. S - 2 in flight before the first step
  issue(0, L0, L0 + BM);
  // step s: buffer s % S; the slice S - 1 ahead goes to buffer (s - 1) % S
#define MOE_DMA_STEP(U, AC, BC, AN, BN_)                                        \
  {                                                                             \
    const int s = s0 + U;                                                       \
    if (s < nk) {                                                               \
      __builtin_amdgcn_sched_barrier(0);                                        \
      if (s + S - 2 < nk)                                                       \
        wait_vm<LOADS *(S - 2)>();                                              \
      else                                                                      \
        wait_vm<0>();                                                           \
      __builtin_amdgcn_s_barrier();                                             \
      __builtin_amdgcn_sched_barrier(0);                                        \
      if (s + S - 1 < nk) issue((s + S - 1) * KS, AN, BN_);                     \
      if (rows_here) mma(AC, BC);                                               \
    }                                                                           \
  }
  for (int s0 = 0; s0 < nk; s0 += S) {
    MOE_DMA_STEP(0, L0, L0 + BM, L1, L1 + BM)
    MOE_DMA_STEP(1, L1, L1 + BM, L0, L0 + BM)
  }
#undef MOE_DMA_STEP
  // lane i holds column i % 32 of each 32 x 32 block, rows 8 (v / 4) + 4 (i / 32) + v % 4
#pragma unroll
  for (int x = 0; x < MX; ++x)
#pragma unroll
    for (int y = 0; y < NY; ++y)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int m = t.m0 + wm * WR + x * 32 + 8 * (i / 4) + 4 * (lane / 32) + i % 4;
        if (m >= j.nrows) continue;
        const int n = t.n0 + wn * WC + y * 32 + lane % 32;
        if (n < N) {
          if (UP)
            static_cast<uint16_t *>(out)[(size_t)(j.row0 + m) * N + n] =
                f32_to_bf16_rne(silu(c[0][x][y][i]) * c[NB - 1][x][y][i]);
          else
            static_cast<float *>(out)[(size_t)(j.row0 + m) * N + n] = c[0][x][y][i];
        }
      }
}

// Small-M grouped GEMM: groups whose experts have at most kSkinnyRows rows
// (batched decode).  The tiled kernel above stages 128-row slices through LDS
// and, with a handful of rows per expert, streams the weights at a few TB/s
// on too few resident waves.  Here a workgroup owns 16 output features of one
// expert for all of its rows (up to 32: two 16-row MFMA blocks).  Its four
// waves split K in four; each streams its quarter of the 16 weight rows (of W1
// and W3 in the up projection) from global memory straight into
// v_mfma_f32_16x16x32_bf16 fragments, several 32-deep steps ahead, with
// the rows' activations read alongside (from L2: every workgroup of the expert
// reads them).  A row or feature past the end reads a valid row instead (its
// outputs are not written); only a K tail that is not a multiple of 32 is
// zeroed.  The four partial products meet in LDS and are added in wave order.
constexpr int kSkinnyAheadUp = 8, kSkinnyAheadDown = 8;  // steps in flight per wave

__device__ __forceinline__ bf16x8 load_frag(const uint16_t *p) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const gemm_u32x4 *>(p));
}

__device__ __forceinline__ bf16x8 load_frag(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_bit_cast(bf16x8, buffer_load16(r, byte_off));
}

template <bool UP, int AHEAD, bool TWO>
__global__ __launch_bounds__(256) void prefill_skinny_kernel(const GemmTile *tiles, const GemmJob *jobs,
                                                             const uint16_t *a_src, const int32_t *perm_tok,
                                                             void *out, int d, int d_ff) {
  constexpr int NB = UP ? 2 : 1;  // B matrices: W1 and W3, or W2
  __shared__ floatx4 red[4][NB][2][kWave];
  const int K = UP ? d : d_ff;  // reduction length
  const int N = UP ? d_ff : d;  // output features
  const int nfb = (N + 15) / 16;
  const int ti = blockIdx.x / nfb, fb = blockIdx.x - ti * nfb;
  const GemmJob j = jobs[tiles[ti].job];
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  const int M = min(j.nrows, kSkinnyRows);
  if (M <= 0) return;       // the host makes tiles only for experts with rows
  const bool two = TWO && M > 16;  // second 16-row block (TWO: the launch may have groups of 17-32 rows)
  const int kg = (lane / 16) * 8;  // this lane's 8 elements of a 32-deep step
  // A rows (tokens of the expert) and B rows (features) of this lane, clamped
  const uint16_t *ap[2];
#pragma unroll
  for (int tb = 0; tb < 2; ++tb) {
    const int m = min(tb * 16 + lane % 16, M - 1);
    ap[tb] = (UP ? a_src + (size_t)perm_tok[j.row0 + m] * d : a_src + (size_t)(j.row0 + m) * d_ff) + kg;
  }
  // B rows: features fb * 16 .. + nf - 1 of each weight matrix, read with
  // buffer loads (the pointer comes from the job table; flat loads would make
  // every wait drain all the loads in flight)
  const int nf = min(16, N - fb * 16);
  __amdgpu_buffer_rsrc_t brs[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b)
    brs[b] = rows_rsrc(j.w + (UP ? (size_t)b * d_ff * d : 2 * (size_t)d_ff * d) + (size_t)fb * 16 * K,
                       (uint32_t)nf * K * 2);
  const uint32_t boff = ((uint32_t)min(lane % 16, nf - 1) * K + kg) * 2;

  floatx4 c[NB][2];
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int tb = 0; tb < 2; ++tb) c[b][tb] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};

  // this wave's full 32-deep steps
  const int full = K / 32;
  const int q = (full + 3) / 4;
  const int s0 = min(wave * q, full), s1 = min(s0 + q, full);
  const int n = s1 - s0;
  bf16x8 wa[AHEAD][NB], xa[AHEAD][2];
  // no load is conditional (in a launch with groups of more than 16 rows,
  // the second row block reads clamped rows where a group has fewer), so the
  // compiler can count the loads in flight
  auto load = [&](int slot, int step) {
    const int k = step * 32;
#pragma unroll
    for (int b = 0; b < NB; ++b) wa[slot][b] = load_frag(brs[b], boff + 2 * k);
    xa[slot][0] = load_frag(ap[0] + k);
    if (TWO) xa[slot][1] = load_frag(ap[1] + k);
  };
  auto mma = [&](int slot) {
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      c[b][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa[slot][0], wa[slot][b], c[b][0], 0, 0, 0);
      if (two) c[b][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa[slot][1], wa[slot][b], c[b][1], 0, 0, 0);
    }
  };
  // straight-line main loop: a step past the wave's last reloads that step
  // (in bounds, never used); the last steps, which load nothing, are peeled
  if (n > 0) {
#pragma unroll
    for (int u = 0; u < AHEAD; ++u) load(u, s0 + min(u, n - 1));
    int i = 0;
    for (; i + AHEAD < n; i += AHEAD) {
#pragma unroll
      for (int u = 0; u < AHEAD; ++u) {
        mma(u);
        load(u, s0 + min(i + u + AHEAD, n - 1));
        __builtin_amdgcn_sched_barrier(0);  // keep each refill next to its step, not batched at the end
      }
    }
#pragma unroll
    for (int u = 0; u < AHEAD; ++u)
      if (i + u < n) mma(u);
  }
  // K tail (K not a multiple of 32): the last wave adds it, zeroing past K
  if (K % 32 && wave == 3) {
    const bool in = full * 32 + kg < K;
    const int k = in ? full * 32 : 0;  // lanes past K read their row's start, then take zeros
    const bf16x8 z = {};
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const bf16x8 v = load_frag(brs[b], boff + 2 * k);
      wa[0][b] = in ? v : z;
    }
    const bf16x8 x0 = load_frag(ap[0] + k);
    xa[0][0] = in ? x0 : z;
    if (TWO) {
      const bf16x8 x1 = load_frag(ap[1] + k);
      xa[0][1] = in ? x1 : z;
    }
    mma(0);
  }
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int tb = 0; tb < 2; ++tb) red[wave][b][tb][lane] = c[b][tb];
  __syncthreads();
  if (wave == 0) {
    floatx4 r[NB][2];
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int tb = 0; tb < 2; ++tb) {
        r[b][tb] = red[0][b][tb][lane];
#pragma unroll
        for (int w = 1; w < 4; ++w) r[b][tb] += red[w][b][tb][lane];
      }
    const int n_out = fb * 16 + lane % 16;
    if (n_out < N) {
#pragma unroll
      for (int tb = 0; tb < 2; ++tb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int m = tb * 16 + (lane / 16) * 4 + i;
          if (m >= M) continue;
          if (UP)
            static_cast<uint16_t *>(out)[(size_t)(j.row0 + m) * N + n_out] =
                f32_to_bf16_rne(silu(r[0][tb][i]) * r[NB - 1][tb][i]);
          else
            static_cast<float *>(out)[(size_t)(j.row0 + m) * N + n_out] = r[0][tb][i];
        }
    }
  }
}

// ---------------------------------------------------------------------------
// 4. h_t += sum_r g_tr Y[pos(t, r)], ranks in order
constexpr int kUnpermRanks = 8;  // ranks whose rows are loaded before the first is added
constexpr int kUnpermSteps = 2;  // four-column steps per lane and pass

__global__ __launch_bounds__(256) void prefill_unpermute_kernel(float *H, const float *Y, const float *g,
                                                                const int32_t *pos_of, int T, int d, int K) {
  const int t = blockIdx.x;
  if (t >= T) return;
  // A workgroup per token.  Every rank's row is loaded before the first is
  // added, so a pass waits for its positions once and for the rows once (one
  // rank after another, each wait was two trips to memory).  Loads are
  // clamped to a valid rank and column, so none waits behind a branch; ranks
  // are added in order, and a rank past K adds nothing (selected, not
  // multiplied by zero).
  for (int c0 = threadIdx.x * 4; c0 < d; c0 += kUnpermSteps * 256 * 4) {
    float4 y[kUnpermSteps], h[kUnpermSteps];
#pragma unroll
    for (int u = 0; u < kUnpermSteps; ++u) {
      y[u] = make_float4(0.f, 0.f, 0.f, 0.f);
      h[u] = *reinterpret_cast<const float4 *>(H + (size_t)t * d + min(c0 + u * 1024, d - 4));
    }
    for (int r0 = 0; r0 < K; r0 += kUnpermRanks) {
      float4 v[kUnpermRanks][kUnpermSteps];
      float gr[kUnpermRanks];
#pragma unroll
      for (int i = 0; i < kUnpermRanks; ++i) {
        const int r = min(r0 + i, K - 1);
        gr[i] = g[(size_t)t * K + r];
        const float *yr = Y + (size_t)pos_of[(size_t)t * K + r] * d;
#pragma unroll
        for (int u = 0; u < kUnpermSteps; ++u)
          v[i][u] = *reinterpret_cast<const float4 *>(yr + min(c0 + u * 1024, d - 4));
      }
#pragma unroll
      for (int i = 0; i < kUnpermRanks; ++i) {
        const bool live = r0 + i < K;
#pragma unroll
        for (int u = 0; u < kUnpermSteps; ++u) {
          y[u].x = live ? fmaf(gr[i], v[i][u].x, y[u].x) : y[u].x;
          y[u].y = live ? fmaf(gr[i], v[i][u].y, y[u].y) : y[u].y;
          y[u].z = live ? fmaf(gr[i], v[i][u].z, y[u].z) : y[u].z;
          y[u].w = live ? fmaf(gr[i], v[i][u].w, y[u].w) : y[u].w;
        }
      }
    }
#pragma unroll
    for (int u = 0; u < kUnpermSteps; ++u) {
      const int c = c0 + u * 1024;
      if (c < d) {
        float4 o = h[u];
        o.x += y[u].x;
        o.y += y[u].y;
        o.z += y[u].z;
        o.w += y[u].w;
        *reinterpret_cast<float4 *>(H + (size_t)t * d + c) = o;
      }
    }
  }
}

}  // namespace

// ---------------------------------------------------------------------------
// launchers used by the host engine
hipError_t launch_prefill_gate(const PrefillArgs &a, const Launch &l) {
  MOE_LAUNCH(prefill_gate_kernel, dim3((a.T + kGateTok - 1) / kGateTok), dim3(kGateThreads), 0, l, a);
  return hipGetLastError();
}

hipError_t launch_prefill_plan(const PlanArgs &a, const Launch &l) {
  MOE_LAUNCH(prefill_plan_kernel, dim3(1), dim3(kPlanThreads), 0, l, a);
  return hipGetLastError();
}

#ifndef MOE_GEMM_DMA
#define MOE_GEMM_DMA 1
#endif
// the LDS-DMA kernel addresses its A operand with 32-bit offsets below kOobOffset
static bool dma_fits(size_t a_bytes) { return MOE_GEMM_DMA && a_bytes > 0 && a_bytes < kOobOffset; }

hipError_t launch_prefill_up(const GemmTile *tiles, int ntiles, const GemmJob *jobs, const uint16_t *xn,
                             const int32_t *perm_tok, uint16_t *act, int d, int d_ff, int rows, size_t a_bytes,
                             const Launch &l, const int32_t *dev_ntiles) {
  if (ntiles <= 0) return hipSuccess;
  if (rows == 256 && dma_fits(a_bytes)) {
    if (d % kDmaKs == 0)
      MOE_LAUNCH((prefill_gemm_dma_kernel<true, false, kDmaWaves, 256, kDmaKs>), dim3(ntiles), dim3(kDmaWaves * kWave), 0, l, tiles, jobs, xn,
                 (uint32_t)a_bytes, perm_tok, (void *)act, d, d_ff, dev_ntiles);
    else
      MOE_LAUNCH((prefill_gemm_dma_kernel<true, true, kDmaWaves, 256, kDmaKs>), dim3(ntiles), dim3(kDmaWaves * kWave), 0, l, tiles, jobs, xn,
                 (uint32_t)a_bytes, perm_tok, (void *)act, d, d_ff, dev_ntiles);
    return hipGetLastError();
  }
#define MOE_GEMM_UP(BM, TH, RG)                                                                                   \
  MOE_LAUNCH((prefill_gemm_kernel<true, kGemmStages, BM, TH, kKStep, RG>), dim3(ntiles), dim3(TH), 0, l, tiles, jobs, xn, \
             perm_tok, (void *)act, d, d_ff, dev_ntiles)
#define MOE_GEMM_UP_TALL(RG)                                                                                     \
  MOE_LAUNCH((prefill_gemm_kernel<true, kGemmStagesTall, 256, 512, kKsTall, RG>), dim3(ntiles), dim3(512), 0, l, tiles, jobs, \
             xn, perm_tok, (void *)act, d, d_ff, dev_ntiles)
  // a K not a multiple of the tall slice takes 32-deep slices three ahead
  // (the 64-deep kernel with its K-tail handling would spill registers)
#define MOE_GEMM_UP_TALL_RAGGED()                                                                                   \
  MOE_LAUNCH((prefill_gemm_kernel<true, 3, 256, 512, kKStep, true>), dim3(ntiles), dim3(512), 0, l, tiles, jobs, xn, \
             perm_tok, (void *)act, d, d_ff, dev_ntiles)
  const bool ragged = d % kKStep != 0;
  if (rows == 64) {
    if (ragged) MOE_GEMM_UP(64, 256, true); else MOE_GEMM_UP(64, 256, false);
  } else if (rows == 128) {
    if (ragged) MOE_GEMM_UP(128, 256, true); else MOE_GEMM_UP(128, 256, false);
  } else if (rows == 256) {
    if (d % kKsTall == 0) MOE_GEMM_UP_TALL(false); else MOE_GEMM_UP_TALL_RAGGED();
  } else {
    return hipErrorInvalidValue;
  }
#undef MOE_GEMM_UP
#undef MOE_GEMM_UP_TALL
#undef MOE_GEMM_UP_TALL_RAGGED
  return hipGetLastError();
}

hipError_t launch_prefill_skinny_up(const GemmTile *tiles, int ntiles, const GemmJob *jobs, const uint16_t *xn,
                                    const int32_t *perm_tok, uint16_t *act, int d, int d_ff, int max_rows,
                                    const Launch &l) {
  if (ntiles <= 0) return hipSuccess;
  if (max_rows < 1 || max_rows > kSkinnyRows) return hipErrorInvalidValue;
  if (max_rows > 16)
    MOE_LAUNCH((prefill_skinny_kernel<true, kSkinnyAheadUp, true>), dim3(ntiles * ((d_ff + 15) / 16)), dim3(256), 0, l,
               tiles, jobs, xn, perm_tok, (void *)act, d, d_ff);
  else
    MOE_LAUNCH((prefill_skinny_kernel<true, kSkinnyAheadUp, false>), dim3(ntiles * ((d_ff + 15) / 16)), dim3(256), 0, l,
               tiles, jobs, xn, perm_tok, (void *)act, d, d_ff);
  return hipGetLastError();
}

hipError_t launch_prefill_skinny_down(const GemmTile *tiles, int ntiles, const GemmJob *jobs, const uint16_t *act,
                                      float *Y, int d, int d_ff, int max_rows, const Launch &l) {
  if (ntiles <= 0) return hipSuccess;
  if (max_rows < 1 || max_rows > kSkinnyRows) return hipErrorInvalidValue;
  if (max_rows > 16)
    MOE_LAUNCH((prefill_skinny_kernel<false, kSkinnyAheadDown, true>), dim3(ntiles * ((d + 15) / 16)), dim3(256), 0, l,
               tiles, jobs, act, nullptr, (void *)Y, d, d_ff);
  else
    MOE_LAUNCH((prefill_skinny_kernel<false, kSkinnyAheadDown, false>), dim3(ntiles * ((d + 15) / 16)), dim3(256), 0, l,
               tiles, jobs, act, nullptr, (void *)Y, d, d_ff);
  return hipGetLastError();
}

hipError_t launch_prefill_down(const GemmTile *tiles, int ntiles, const GemmJob *jobs, const uint16_t *act,
                               float *Y, int d, int d_ff, int rows, size_t a_bytes, const Launch &l,
                               const int32_t *dev_ntiles) {
  if (ntiles <= 0) return hipSuccess;
  if (rows == 256 && dma_fits(a_bytes)) {
    if (d_ff % kDmaKs == 0)
      MOE_LAUNCH((prefill_gemm_dma_kernel<false, false, kDmaWaves, 256, kDmaKs>), dim3(ntiles), dim3(kDmaWaves * kWave), 0, l, tiles, jobs, act,
                 (uint32_t)a_bytes, (const int32_t *)nullptr, (void *)Y, d, d_ff, dev_ntiles);
    else
      MOE_LAUNCH((prefill_gemm_dma_kernel<false, true, kDmaWaves, 256, kDmaKs>), dim3(ntiles), dim3(kDmaWaves * kWave), 0, l, tiles, jobs, act,
                 (uint32_t)a_bytes, (const int32_t *)nullptr, (void *)Y, d, d_ff, dev_ntiles);
    return hipGetLastError();
  }
#define MOE_GEMM_DOWN(BM, TH, RG)                                                                                  \
  MOE_LAUNCH((prefill_gemm_kernel<false, kGemmStages, BM, TH, kKStep, RG>), dim3(ntiles), dim3(TH), 0, l, tiles, jobs, act, \
             (const int32_t *)nullptr, (void *)Y, d, d_ff, dev_ntiles)
#define MOE_GEMM_DOWN_TALL(RG)                                                                                     \
  MOE_LAUNCH((prefill_gemm_kernel<false, kGemmStagesTall, 256, 512, kKsTall, RG>), dim3(ntiles), dim3(512), 0, l, tiles, jobs, \
             act, (const int32_t *)nullptr, (void *)Y, d, d_ff, dev_ntiles)
#define MOE_GEMM_DOWN_TALL_RAGGED()                                                                                  \
  MOE_LAUNCH((prefill_gemm_kernel<false, 3, 256, 512, kKStep, true>), dim3(ntiles), dim3(512), 0, l, tiles, jobs, act, \
             (const int32_t *)nullptr, (void *)Y, d, d_ff, dev_ntiles)
  const bool ragged = d_ff % kKStep != 0;
  if (rows == 64) {
    if (ragged) MOE_GEMM_DOWN(64, 256, true); else MOE_GEMM_DOWN(64, 256, false);
  } else if (rows == 128) {
    if (ragged) MOE_GEMM_DOWN(128, 256, true); else MOE_GEMM_DOWN(128, 256, false);
  } else if (rows == 256) {
    if (d_ff % kKsTall == 0) MOE_GEMM_DOWN_TALL(false); else MOE_GEMM_DOWN_TALL_RAGGED();
  } else {
    return hipErrorInvalidValue;
  }
#undef MOE_GEMM_DOWN
#undef MOE_GEMM_DOWN_TALL
#undef MOE_GEMM_DOWN_TALL_RAGGED
  return hipGetLastError();
}

hipError_t launch_prefill_unpermute(float *H, const float *Y, const float *g, const int32_t *pos_of, int T,
                                    int d, int K, const Launch &l) {
  MOE_LAUNCH(prefill_unpermute_kernel, dim3(T), dim3(256), 0, l, H, Y, g, pos_of, T, d, K);
  return hipGetLastError();
}

int prefill_tile_cols(bool up) { return up ? gemm_cols<true>() : gemm_cols<false>(); }

}  // namespace moe
