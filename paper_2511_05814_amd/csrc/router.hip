// Router and cache-table kernel for batch-1 decode.
//
// One workgroup per role and call: routing and the table lookups of the layer
// being decoded, and, when speculating, the guess and insertion for the next
// layer.  All 16 waves of a workgroup first compute its role's gate logits
// z = W_g h (Sec. 4.3: the gate is a linear map [len_hidden, num_experts]):
// for the layer being decoded, or for the next layer (Sec. 3.2: the next
// layer's gate applied to the current hidden state).  Each product
// of a bf16/fp32 weight and an fp32 activation is exact in fp64, and the sums
// are accumulated in fp64 so that the top-K decision is the one an fp64
// evaluation makes.
//
// The whole workgroup then counts the top-K ranks (each thread compares one
// logit with an eighth of the others).  One wave owns each cache table: lane e
// holds expert e's slot, use count, last-use tick and prefetched flag.  When
// every selected expert is resident the K lookups change K distinct lanes and
// evict nothing, so they are applied at once; otherwise they are applied one
// by one in rank order, with wave-wide argmin reductions choosing the victim
// (LRU, Sec. 3.1: smallest last-use tick; LFU, Sec. 4.2: smallest count, then
// last-use tick; aged LFU, after Sec. 6.1: the count halved once per fixed
// number of ticks since the last use, then last-use tick; then lower slot).
// Wave 0 serves the demand lookup of this layer, wave 1 the speculative
// insertion into the next layer's table; the tables are disjoint, so the two
// run concurrently, in different workgroups when both are asked for.
#include "common.hpp"

#include <math.h>

namespace moe {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / kWave;

// Gate logits z[row] for up to two layers: rows 0..E-1 belong to a.layer (when
// routing here), rows E..2E-1 to a.spec_layer (when speculating); only the
// needed rows are visited.  Wave w owns needed rows r0 + w, r0 + w + stride,
// ... (at most MR of them) and accumulates all of them at once, one fp64
// chain per row: lane i covers columns EPL*i + EPL*64*c of a row (chunk c), in
// chunk order, with h from LDS.  The loads of the next chunk of all the
// wave's rows are issued before the current chunk's products, from addresses
// clamped into the gate array (past the wave's rows or chunks they reread a
// valid row or chunk, unused) so that no load sits behind a branch; the lanes
// of each row are then summed with DPP moves (no LDS round trips).
constexpr int kMaxD = 16384;

struct GateWork {
  int m = 0, cpr = 1;         // rows of this wave; 16-byte chunks per row
  int first = 0, stride = 1;  // this wave's rows: first, first + stride, ...
};

// Rows r0 .. r1-1 are dealt out one per wave, round robin.
template <int DT>
__device__ __forceinline__ GateWork gate_work(const RouterArgs &a, int r0, int r1, int wave) {
  constexpr int EPL = DT == 1 ? 8 : 4;  // elements per 16-byte load
  GateWork g;
  g.cpr = (a.d + kWave * EPL - 1) / (kWave * EPL);
  g.first = r0 + wave;
  g.stride = kWaves;
  g.m = g.first < r1 ? (r1 - g.first + g.stride - 1) / g.stride : 0;
  return g;
}

// Issue the weight loads of chunk c (clamped) of the wave's MR rows (m > 0).
template <int DT, int MR>
__device__ __forceinline__ void gate_load(const RouterArgs &a, int lane, const GateWork &g, int c, uint4 *v) {
  constexpr int EPL = DT == 1 ? 8 : 4;
  constexpr int ESZ = DT == 1 ? 2 : 4;
  const int E = a.E, d = a.d;
  const uint8_t *gate = static_cast<const uint8_t *>(a.gate);
  const int col = min(min(c, g.cpr - 1) * kWave * EPL + lane * EPL, d - EPL);
#pragma unroll
  for (int i = 0; i < MR; ++i) {
    const int row = g.first + g.stride * min(i, g.m - 1);
    const int gl = row < E ? a.layer : a.spec_layer;
    const int e = row < E ? row : row - E;
    v[i] = *reinterpret_cast<const uint4 *>(gate + (((size_t)gl * E + e) * d + col) * ESZ);
  }
}

// fp64 sum over a wave's lanes, left in lane 63: running sums within rows of
// 16 lanes (row_shr 1, 2, 4, 8), then row_bcast:15 and row_bcast:31; lanes
// whose DPP source lies outside the pattern add 0.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ double dpp_add_d(double v) {
  const int lo = __builtin_amdgcn_update_dpp(0, __double2loint(v), CTRL, ROW_MASK, 0xF, false);
  const int hi = __builtin_amdgcn_update_dpp(0, __double2hiint(v), CTRL, ROW_MASK, 0xF, false);
  return v + __hiloint2double(hi, lo);
}
__device__ __forceinline__ double wave_sum_d_to_lane63(double v) {
  v = dpp_add_d<0x111, 0xF>(v);
  v = dpp_add_d<0x112, 0xF>(v);
  v = dpp_add_d<0x114, 0xF>(v);
  v = dpp_add_d<0x118, 0xF>(v);
  v = dpp_add_d<0x142, 0xA>(v);
  v = dpp_add_d<0x143, 0xC>(v);
  return v;
}

// The products of chunk c (whose weights are in v) into acc.
template <int DT, int MR>
__device__ __forceinline__ void gate_chunk(const float *hs, int d, int lane, int c, const uint4 *v, double *acc) {
  constexpr int EPL = DT == 1 ? 8 : 4;
  const int col = c * kWave * EPL + lane * EPL;
  if (col < d) {
    const float4 h0 = *reinterpret_cast<const float4 *>(hs + col);
    if (DT == 1) {
      const float4 h1 = *reinterpret_cast<const float4 *>(hs + col + 4);
#pragma unroll
      for (int i = 0; i < MR; ++i) {
        float f[8];
        bf16x8_to_f32(v[i], f);
        acc[i] = fma((double)f[0], (double)h0.x, acc[i]);
        acc[i] = fma((double)f[1], (double)h0.y, acc[i]);
        acc[i] = fma((double)f[2], (double)h0.z, acc[i]);
        acc[i] = fma((double)f[3], (double)h0.w, acc[i]);
        acc[i] = fma((double)f[4], (double)h1.x, acc[i]);
        acc[i] = fma((double)f[5], (double)h1.y, acc[i]);
        acc[i] = fma((double)f[6], (double)h1.z, acc[i]);
        acc[i] = fma((double)f[7], (double)h1.w, acc[i]);
      }
    } else {
#pragma unroll
      for (int i = 0; i < MR; ++i) {
        acc[i] = fma((double)__uint_as_float(v[i].x), (double)h0.x, acc[i]);
        acc[i] = fma((double)__uint_as_float(v[i].y), (double)h0.y, acc[i]);
        acc[i] = fma((double)__uint_as_float(v[i].z), (double)h0.z, acc[i]);
        acc[i] = fma((double)__uint_as_float(v[i].w), (double)h0.w, acc[i]);
      }
    }
  }
}

// All of a wave's gate weights at once, when its rows have at most 16 / MR
// chunks (the 64-expert model: 4 rows of 4 chunks): the loads of chunks 1..
// are issued before any product, so one CU keeps the whole gate in flight.
// v holds chunk 0, loaded before h was staged.
template <int DT, int MR>
__device__ void gate_logits_all(const RouterArgs &a, const float *hs, int lane, const GateWork &g, uint4 *v,
                                double *zs) {
  constexpr int NC = 16 / MR;  // chunks held at once
  uint4 w[NC - 1][MR];
#pragma unroll
  for (int c = 1; c < NC; ++c) gate_load<DT, MR>(a, lane, g, c, w[c - 1]);  // past cpr: the last chunk, unused
  double acc[MR];
#pragma unroll
  for (int i = 0; i < MR; ++i) acc[i] = 0.0;
  gate_chunk<DT, MR>(hs, a.d, lane, 0, v, acc);
#pragma unroll
  for (int c = 1; c < NC; ++c)
    if (c < g.cpr) gate_chunk<DT, MR>(hs, a.d, lane, c, w[c - 1], acc);
#pragma unroll
  for (int i = 0; i < MR; ++i) {
    const double z = wave_sum_d_to_lane63(acc[i]);
    if (i < g.m && lane == kWave - 1) zs[g.first + g.stride * i] = z;
  }
}

// v holds chunk 0 of the wave's rows, loaded by gate_load(.., 0, v) before h
// was staged; logit `row` goes to zs[row].
template <int DT, int MR>
__device__ void gate_logits(const RouterArgs &a, const float *hs, int lane, const GateWork &g, uint4 *v,
                            double *zs) {
  if (g.cpr * MR <= 16) {  // the same for the whole wave
    gate_logits_all<DT, MR>(a, hs, lane, g, v, zs);
    return;
  }
  constexpr int EPL = DT == 1 ? 8 : 4;
  const int d = a.d, cpr = g.cpr;
  double acc[MR];
#pragma unroll
  for (int i = 0; i < MR; ++i) acc[i] = 0.0;
  for (int c = 0; c < cpr; ++c) {
    uint4 nv[MR];
    gate_load<DT, MR>(a, lane, g, c + 1, nv);  // the last chunk loads itself again, unused
    const int col = c * kWave * EPL + lane * EPL;
    if (col < d) {
      const float4 h0 = *reinterpret_cast<const float4 *>(hs + col);
      if (DT == 1) {
        const float4 h1 = *reinterpret_cast<const float4 *>(hs + col + 4);
#pragma unroll
        for (int i = 0; i < MR; ++i) {
          float f[8];
          bf16x8_to_f32(v[i], f);
          acc[i] = fma((double)f[0], (double)h0.x, acc[i]);
          acc[i] = fma((double)f[1], (double)h0.y, acc[i]);
          acc[i] = fma((double)f[2], (double)h0.z, acc[i]);
          acc[i] = fma((double)f[3], (double)h0.w, acc[i]);
          acc[i] = fma((double)f[4], (double)h1.x, acc[i]);
          acc[i] = fma((double)f[5], (double)h1.y, acc[i]);
          acc[i] = fma((double)f[6], (double)h1.z, acc[i]);
          acc[i] = fma((double)f[7], (double)h1.w, acc[i]);
        }
      } else {
#pragma unroll
        for (int i = 0; i < MR; ++i) {
          acc[i] = fma((double)__uint_as_float(v[i].x), (double)h0.x, acc[i]);
          acc[i] = fma((double)__uint_as_float(v[i].y), (double)h0.y, acc[i]);
          acc[i] = fma((double)__uint_as_float(v[i].z), (double)h0.z, acc[i]);
          acc[i] = fma((double)__uint_as_float(v[i].w), (double)h0.w, acc[i]);
        }
      }
    }
#pragma unroll
    for (int i = 0; i < MR; ++i) v[i] = nv[i];
  }
#pragma unroll
  for (int i = 0; i < MR; ++i) {
    const double z = wave_sum_d_to_lane63(acc[i]);
    if (i < g.m && lane == kWave - 1) zs[g.first + g.stride * i] = z;
  }
}

// One wave's view of a layer's table (lane e = expert e, for lanes < E) and
// of its statistics counter (lane i = counter i), read at kernel start so the
// reads overlap the gate GEMV.  Indices are clamped instead of guarded (a
// guarded load is waited for on the spot); lanes past E are masked where the
// values are used.
struct TableView {
  int32_t slot;
  uint32_t count;
  int64_t last;
  int32_t pf;
  int64_t clock, lookups;
  uint64_t stat;
};

__device__ __forceinline__ TableView load_table(const LayerTable *T, const LayerStats *st, int lane, int E) {
  const int e = min(lane, E - 1);
  TableView t;
  t.slot = T->expert_slot[e];
  t.count = T->count[e];
  t.last = T->last[e];
  t.pf = T->pf[e];
  t.clock = T->clock;
  t.lookups = T->lookups;
  t.stat = st->v[lane & 15];
  return t;
}

// Lane of the resident, unpinned expert with the smallest policy key
// (LFU: count, last, slot; aged LFU: count aged to `clock`, last, slot;
// LRU: last, slot), or -1 if there is none.
__device__ int wave_victim(bool cand, int policy, int aging, int64_t clock, uint32_t count, int64_t last,
                           int slot) {
  uint32_t k1 = !cand ? 0u
              : policy == 1 ? count
              : policy == 2 ? aged_count(count, last, clock, aging)
              : 0u;
  int64_t k2 = last;
  int k3 = slot;
  int bl = threadIdx.x & (kWave - 1);
  int bv = cand ? 1 : 0;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const uint32_t o1 = __shfl_xor(k1, o, kWave);
    const int64_t o2 = __shfl_xor(k2, o, kWave);
    const int o3 = __shfl_xor(k3, o, kWave);
    const int ol = __shfl_xor(bl, o, kWave);
    const int ov = __shfl_xor(bv, o, kWave);
    bool less;
    if (ov != bv) {
      less = ov > bv;
    } else {
      less = (o1 < k1) || (o1 == k1 && (o2 < k2 || (o2 == k2 && (o3 < k3 || (o3 == k3 && ol < bl)))));
    }
    if (less) {
      k1 = o1;
      k2 = o2;
      k3 = o3;
      bl = ol;
      bv = ov;
    }
  }
  return bv ? bl : -1;
}

// Value of x on lane src, for a src the whole wave agrees on (a scalar read,
// not an LDS round trip like a general shuffle).
__device__ __forceinline__ int lane_value(int x, int src) { return __builtin_amdgcn_readlane(x, src); }
__device__ __forceinline__ double lane_value_d(double x, int src) {
  return __hiloint2double(__builtin_amdgcn_readlane(__double2hiint(x), src),
                          __builtin_amdgcn_readlane(__double2loint(x), src));
}

// Ring position of record base + r, from base % cap computed once.
__device__ __forceinline__ uint64_t ring_pos(uint64_t base_pos, int r, uint64_t cap, int K) {
  uint64_t pos = base_pos + (uint64_t)r;
  if (pos >= cap) pos = cap >= (uint64_t)K ? pos - cap : pos % cap;
  return pos;
}

__device__ void put_rec(const RouterArgs &a, uint64_t pos, int kind, int64_t token, int layer,
                        int rank, int expert, int flags, int slot, int victim) {
  if (a.trace == nullptr || a.trace_cap == 0) return;
  TraceRec r;
  r.kind = kind;
  r.token = (int32_t)token;
  r.layer = layer;
  r.rank = rank;
  r.expert = expert;
  r.flags = flags;
  r.slot = slot;
  r.victim = victim;
  a.trace[pos] = r;
}

// Wave 0: the token's K lookups in layer a.layer, in rank order.
// `idreg` on lane r < K holds the expert of rank r.
__device__ void demand_lookup(const RouterArgs &a, int idreg, int lane, uint64_t rec_base, const TableView &tv) {
  LayerTable *T = a.tables + a.layer;
  LayerStats *st = a.stats + a.layer;
  FetchList *fl = a.dlists + a.layer;
  const int E = a.E, K = a.K;
  const bool in_range = lane < E;
  int my_slot = in_range ? tv.slot : -1;
  uint32_t my_count = in_range ? tv.count : 0u;
  int64_t my_last = in_range ? tv.last : 0;
  int my_pf = in_range ? tv.pf : 0;
  int64_t clock = tv.clock;
  const int64_t token = tv.lookups;

  int my_rank = -1;  // the rank that selected this lane's expert (ids are distinct)
  for (int r = 0; r < K; ++r) my_rank = lane_value(idreg, r) == lane ? r : my_rank;
  const bool pinned = my_rank >= 0;
  const uint64_t base_pos = a.trace_cap ? rec_base % a.trace_cap : 0;

  // Rank lane r's expert: its slot and prefetched flag before the lookups.
  const int j_l = lane < K ? idreg : 0;
  const int slot_l = __shfl(my_slot, j_l, kWave);
  const int pf_l = __shfl(my_pf, j_l, kWave);
  const bool all_hit = __ballot(lane < K && slot_l < 0) == 0;

  int n_miss = 0, hits = 0, useful = 0, wasted = 0;
  if (all_hit) {
    // Nothing is evicted, so the K lookups touch K distinct lanes and run at
    // once: rank r's use is tick clock + r + 1, as in the sequence below.
    if (pinned) {
      my_count += 1;
      my_last = clock + my_rank + 1;
      my_pf = 0;
    }
    clock += K;
    hits = K;
    useful = __popcll(__ballot(lane < K && pf_l != 0));
    if (lane < K) {
      const int flags = 1 | (pf_l ? 2 : 0);
      a.route->ids[lane] = idreg;
      a.route->slot[lane] = slot_l;
      a.route->hit[lane] = 1;
      put_rec(a, ring_pos(base_pos, lane, a.trace_cap, K), REC_ACCESS, token, a.layer, lane, idreg, flags, slot_l, -1);
    }
  }
  for (int r = 0; r < (all_hit ? 0 : K); ++r) {
    const int j = lane_value(idreg, r);
    clock += 1;
    const int slot_j = lane_value(my_slot, j);
    const int pf_j = lane_value(my_pf, j);
    if (lane == j) {
      my_count += 1;
      my_last = clock;
    }
    int flags, slot, victim;
    if (slot_j >= 0) {
      flags = 1 | (pf_j ? 2 : 0);
      if (pf_j) {
        useful += 1;
        if (lane == j) my_pf = 0;
      }
      slot = slot_j;
      victim = -1;
      hits += 1;
    } else {
      const bool cand = in_range && my_slot >= 0 && !pinned;
      const int v = wave_victim(cand, a.policy, a.aging, clock, my_count, my_last, my_slot);
      if (v < 0) {  // cannot happen with slots >= K; refuse rather than corrupt
        if (lane == 0) *a.err = ERR_BAD_LIST;
        break;
      }
      const int s = lane_value(my_slot, v);
      const int pf_v = lane_value(my_pf, v);
      if (pf_v) wasted += 1;
      if (lane == v) {
        my_slot = -1;
        my_pf = 0;
      }
      if (lane == j) my_slot = s;
      if (lane == 0) {
        T->slot_expert[s] = j;
        fl->expert[n_miss] = j;
        fl->slot[n_miss] = s;
      }
      n_miss += 1;
      flags = 0;
      slot = s;
      victim = v;
    }
    if (lane == 0) {
      a.route->ids[r] = j;
      a.route->slot[r] = slot;
      a.route->hit[r] = flags & 1;
      put_rec(a, ring_pos(base_pos, r, a.trace_cap, K), REC_ACCESS, token, a.layer, r, j, flags, slot, victim);
    }
  }
  // prefetched experts this token did not use are wasted
  const unsigned long long left = __ballot(in_range && my_pf != 0);
  wasted += __popcll(left);
  my_pf = 0;

  if (in_range) {
    T->expert_slot[lane] = my_slot;
    T->count[lane] = my_count;
    T->last[lane] = my_last;
    T->pf[lane] = my_pf;
  }
  if (lane == 0) {
    T->clock = clock;
    T->lookups = token + 1;
    fl->n = n_miss;
    fl->layer = a.layer;
    a.route->k = K;
  }
  // counters: one lane each, so the read-modify-writes overlap
  const uint64_t add = lane == ST_HITS ? (uint64_t)hits
                     : lane == ST_MISSES || lane == ST_EVICT ? (uint64_t)n_miss
                     : lane == ST_PF_USEFUL ? (uint64_t)useful
                     : lane == ST_PF_WASTED ? (uint64_t)wasted
                     : lane == ST_LOOKUPS ? 1ull
                     : lane == ST_BYTES ? (uint64_t)n_miss * a.expert_bytes : 0ull;
  if (add) st->v[lane] = tv.stat + add;
}

// Wave 1: insert up to pmax of the K guesses (lane r holds rank r's guess)
// into the table of a.spec_layer, all guesses pinned.
__device__ void prefetch_insert(const RouterArgs &a, int greg, int lane, uint64_t rec_base, const TableView &tv) {
  const int L2 = a.spec_layer;
  LayerTable *T = a.tables + L2;
  LayerStats *st = a.stats + L2;
  FetchList *fl = a.plists + L2;
  const int E = a.E, K = a.K;
  const bool in_range = lane < E;
  int my_slot = in_range ? tv.slot : -1;
  uint32_t my_count = in_range ? tv.count : 0u;
  int64_t my_last = in_range ? tv.last : 0;
  int my_pf = in_range ? tv.pf : 0;
  int64_t clock = tv.clock;
  const int64_t token = tv.lookups;

  bool pinned = false;
  for (int r = 0; r < K; ++r) pinned |= (lane_value(greg, r) == lane);
  const uint64_t base_pos = a.trace_cap ? rec_base % a.trace_cap : 0;

  // Every guess already resident: nothing to insert, only the records.
  const int slot_l = __shfl(my_slot, lane < K ? greg : 0, kWave);
  const bool all_res = __ballot(lane < K && slot_l < 0) == 0;
  if (all_res && lane < K)
    put_rec(a, ring_pos(base_pos, lane, a.trace_cap, K), REC_PREFETCH, token, L2, lane, greg, 1, slot_l, -1);

  int issued = 0, wasted = 0;
  for (int r = 0; r < (all_res ? 0 : K); ++r) {
    const int j = lane_value(greg, r);
    const int slot_j = lane_value(my_slot, j);
    int flags = 0, slot = -1, victim = -1;
    if (slot_j >= 0) {
      flags = 1;
      slot = slot_j;
    } else if (issued < a.pmax) {
      clock += 1;
      const bool cand = in_range && my_slot >= 0 && !pinned;
      const int v = wave_victim(cand, a.policy, a.aging, clock, my_count, my_last, my_slot);
      if (v < 0) {
        if (lane == 0) *a.err = ERR_BAD_LIST;
        break;
      }
      const int s = lane_value(my_slot, v);
      const int pf_v = lane_value(my_pf, v);
      if (pf_v) wasted += 1;
      if (lane == v) {
        my_slot = -1;
        my_pf = 0;
      }
      if (lane == j) {
        my_slot = s;
        my_last = clock;
        my_pf = 1;
      }
      if (lane == 0) {
        T->slot_expert[s] = j;
        fl->expert[issued] = j;
        fl->slot[issued] = s;
      }
      issued += 1;
      flags = 2;
      slot = s;
      victim = v;
    }
    if (lane == 0) put_rec(a, ring_pos(base_pos, r, a.trace_cap, K), REC_PREFETCH, token, L2, r, j, flags, slot, victim);
  }
  if (in_range) {
    T->expert_slot[lane] = my_slot;
    T->last[lane] = my_last;
    T->pf[lane] = my_pf;
  }
  if (lane == 0) {
    T->clock = clock;
    fl->n = issued;
    fl->layer = L2;
  }
  const uint64_t add = lane == ST_PF_GUESS ? (uint64_t)K
                     : lane == ST_PF_ISSUED ? (uint64_t)issued
                     : lane == ST_PF_WASTED ? (uint64_t)wasted
                     : lane == ST_BYTES ? (uint64_t)issued * a.expert_bytes : 0ull;
  if (add) st->v[lane] = tv.stat + add;
}

// Top-K of the logits in rank order: larger z first, lower id on ties, NaN
// ranked as -inf.  An expert's rank is the number of logits that come before
// it in that order; the whole workgroup counts, thread t taking expert t % 64
// of set t / 512 (0: this layer's logits zs[0, E), 1: the next layer's
// zs[E, 2E)) against the part (t / 64) % 8 of the other logits.
constexpr int kRankParts = 8;
static_assert(kThreads == 2 * kRankParts * kMaxE, "one thread per (set, part, expert)");

__device__ __forceinline__ void rank_parts(const double *zs, int E, bool set0, bool set1, int tid,
                                           int (*cnt)[kRankParts][kMaxE]) {
  const int set = tid / (kRankParts * kMaxE), part = (tid / kMaxE) % kRankParts, e = tid % kMaxE;
  if (e >= E || !(set == 0 ? set0 : set1)) return;
  const double *z = zs + set * E;
  const double mine = rank_key(z[e]);
  const int per = (E + kRankParts - 1) / kRankParts;
  const int o0 = part * per, o1 = min(E, o0 + per);
  int n = 0;
  for (int o = o0; o < o1; ++o) {
    const double zo = rank_key(z[o]);
    n += (zo > mine || (zo == mine && o < e)) ? 1 : 0;
  }
  cnt[set][part][e] = n;
}

// One wave: lane e < E adds its part counts into its rank, rank r < K writes
// its expert to out[r] (LDS of this wave).  Returns out[lane] on lanes < K,
// -1 elsewhere.
__device__ __forceinline__ int topk_from_parts(const int (*cnt)[kMaxE], int E, int K, int lane, int *out) {
  if (lane < E) {
    int rank = 0;
#pragma unroll
    for (int p = 0; p < kRankParts; ++p) rank += cnt[p][lane];
    if (rank < K) out[rank] = lane;
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  return lane < K ? out[lane] : -1;
}

// MR: most gate rows a wave holds at once.  A launch of two workgroups splits
// the roles: workgroup 0 routes and looks up this layer,
// workgroup 1 guesses and inserts for the next one (their tables, counters and
// trace records are disjoint), each with its own copy of h and a GEMV of E
// rows.  (Both roles in one workgroup, the speculative rows in a second GEMV
// pass, put that pass on every layer's critical path: 13.7 against 9.7 us a
// layer at 64 experts.)
template <int MR>
__global__ __launch_bounds__(kThreads) void router_kernel(RouterArgs a) {
  __shared__ __align__(16) float hs[kMaxD];
  __shared__ double zs[2 * kMaxE];
  __shared__ int s_top[2][kMaxK];
  __shared__ double red[kWaves];
  __shared__ int s_cnt[2][kRankParts][kMaxE];
  __shared__ uint64_t s_tbase;
  __shared__ int s_demand_ok;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int E = a.E, d = a.d;
  // role of this workgroup: 0 demand only, 1 speculation only, -1 both
  const int role = gridDim.x == 2 ? (int)blockIdx.x : -1;
  const bool demand = a.demand && role != 1;
  const bool route_here = demand && a.inj_ids == nullptr;
  const bool spec = a.spec_layer >= 0 && role != 0;

  // Every global read that does not depend on another is issued first: the
  // tables and counters of waves 0 and 1, the first batch of gate rows, then h.
  TableView tv{};
  if (wave == 0 && demand) tv = load_table(a.tables + a.layer, a.stats + a.layer, lane, E);
  if (wave == 1 && spec) tv = load_table(a.tables + a.spec_layer, a.stats + a.spec_layer, lane, E);
  const int r0 = route_here ? 0 : E, r1 = spec ? 2 * E : E;
  uint4 gv[MR];
  GateWork gw;
  if (route_here || spec) {
    gw = a.dtype == 1 ? gate_work<1>(a, r0, r1, wave) : gate_work<0>(a, r0, r1, wave);
    if (gw.m > 0) {
      if (a.dtype == 1)
        gate_load<1, MR>(a, lane, gw, 0, gv);
      else
        gate_load<0, MR>(a, lane, gw, 0, gv);
    }
  }
  if (tid == 0) {
    s_tbase = *a.trace_in;
    s_demand_ok = 0;
  }
  if (route_here || spec) {
    // h into LDS (h is NULL when no gate row is needed); sum of squares on the way
    double ss = 0.0;
    for (int i = tid * 4; i < d; i += kThreads * 4) {
      const float4 v = *reinterpret_cast<const float4 *>(a.h + i);
      *reinterpret_cast<float4 *>(hs + i) = v;
      ss = fma((double)v.x, (double)v.x, ss);
      ss = fma((double)v.y, (double)v.y, ss);
      ss = fma((double)v.z, (double)v.z, ss);
      ss = fma((double)v.w, (double)v.w, ss);
    }
    ss = wave_sum_d(ss);
    if (lane == 0) red[wave] = ss;
    __syncthreads();
    if (gw.m > 0) {  // the same for the whole wave
      if (a.dtype == 1)
        gate_logits<1, MR>(a, hs, lane, gw, gv, zs);
      else
        gate_logits<0, MR>(a, hs, lane, gw, gv, zs);
    }
  }
  __syncthreads();
  rank_parts(zs, E, route_here, spec, tid, s_cnt);
  __syncthreads();

  if (wave == 0 && demand) {
    int idreg;
    if (route_here) {
      idreg = topk_from_parts(s_cnt[0], E, a.K, lane, s_top[0]);
      // renormalised softmax over the selected logits z / rms (rank 0 is the max)
      const double zr = (lane < a.K) ? zs[idreg < 0 ? 0 : idreg] : 0.0;
      const double ss = lane_value_d(wave_sum_d_to_lane63(lane < kWaves ? red[lane] : 0.0), kWave - 1);
      const double r = sqrt(ss / (double)d + 1e-5);
      const double z0 = lane_value_d(zr, 0);
      const double ex = (lane < a.K) ? exp((zr - z0) / r) : 0.0;
      const double den = lane_value_d(wave_sum_d_to_lane63(ex), kWave - 1);
      if (lane < a.K) a.route->g[lane] = (float)(ex / den);
      if (lane == 0) a.route->inv_r = (float)(1.0 / r);
    } else {
      idreg = (lane < a.K) ? a.inj_ids[lane] : -1;
      bool ok = true;
      for (int r = 0; r < a.K; ++r) {
        const int j = lane_value(idreg, r);
        const unsigned long long same = __ballot(lane < a.K && idreg == j);
        ok = ok && j >= 0 && j < E && __popcll(same) == 1;
      }
      if (!ok) {
        if (lane == 0) {
          *a.err = ERR_BAD_IDS;
          a.dlists[a.layer].n = 0;
          a.dlists[a.layer].layer = a.layer;
          a.route->k = 0;
        }
        idreg = -1;
      } else {
        if (lane < a.K) a.route->g[lane] = 0.0f;
        if (lane == 0) a.route->inv_r = 0.0f;
      }
    }
    if (lane_value(idreg, 0) >= 0) {
      demand_lookup(a, idreg, lane, s_tbase, tv);
      if (lane == 0) s_demand_ok = 1;
    }
  }
  if (wave == 1 && spec) {
    const int greg = topk_from_parts(s_cnt[1], E, a.K, lane, s_top[1]);
    prefetch_insert(a, greg, lane, s_tbase + (a.demand ? (uint64_t)a.K : 0), tv);
  }
  __syncthreads();
  // the demand workgroup (or the only one) advances the count past both roles'
  // records; the speculative records sit at s_tbase + K either way
  if (tid == 0 && role != 1)
    *a.trace_out = s_tbase + (a.trace ? (s_demand_ok ? (uint64_t)a.K : 0) +
                                            (a.spec_layer >= 0 ? (uint64_t)a.K : 0)
                                      : 0);
}

}  // namespace

hipError_t launch_router(const RouterArgs &a, const Launch &l) {
  // With routing and speculation both asked for, the two roles run side by
  // side, one workgroup each; otherwise one workgroup does the call.  Each
  // role has at most 64 gate rows, 4 a wave.  (One workgroup for both roles,
  // the speculative rows in a second GEMV pass: 13.7 instead of 9.7 us a
  // layer at 64 experts; the GEMV spread over many workgroups with the last
  // one doing the table work cost about 7 us in device-scope fences.)
  const bool both = a.demand && a.inj_ids == nullptr && a.spec_layer >= 0;
  if (a.E > 4 * kWaves) return hipErrorInvalidValue;  // cannot happen: at most kMaxE experts
  const int per_wave = (a.E + kWaves - 1) / kWaves;
  const dim3 grid(both ? 2 : 1);
  if (per_wave <= 1)
    MOE_LAUNCH((router_kernel<1>), grid, dim3(kThreads), 0, l, a);
  else if (per_wave <= 2)
    MOE_LAUNCH((router_kernel<2>), grid, dim3(kThreads), 0, l, a);
  else
    MOE_LAUNCH((router_kernel<4>), grid, dim3(kThreads), 0, l, a);
  return hipGetLastError();
}

}  // namespace moe
