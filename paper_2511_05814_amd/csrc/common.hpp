// Internal layout shared by the kernels and the host engine of the MoE
// offloading library.  Everything here lives in the caller's device
// workspace; the host engine carves the workspace into these regions.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace moe {

constexpr int kMaxE = 64;   // experts per layer: one lane per expert in the table wave
constexpr int kMaxK = 16;   // experts per token
constexpr int kWave = 64;   // CDNA wavefront

// One layer's cache table.  slot_expert[s] = expert held by slot s;
// expert_slot[e] = slot of expert e or -1; count = LFU use count (persists
// across eviction); last = clock tick of the last use or insertion;
// pf = 1 while a prefetched expert has not yet been used.
struct LayerTable {
  int64_t clock;
  int64_t lookups;
  int32_t slot_expert[kMaxE];
  int32_t expert_slot[kMaxE];
  uint32_t count[kMaxE];
  int32_t pf[kMaxE];
  int64_t last[kMaxE];
};

enum StatIdx {
  ST_HITS = 0, ST_MISSES, ST_EVICT, ST_PF_GUESS, ST_PF_ISSUED, ST_PF_USEFUL,
  ST_PF_WASTED, ST_LOOKUPS, ST_BYTES, ST_COUNT
};
struct LayerStats {
  uint64_t v[16];
};

// Copies the router decided: expert e of `layer` from the host store into
// slot s of `layer` in the arena.
struct FetchList {
  int32_t n;
  int32_t layer;
  int32_t expert[kMaxK];
  int32_t slot[kMaxK];
  int32_t pad[2];
};

// Router output consumed by the decode FFN on the compute stream.
struct RouteOut {
  int32_t ids[kMaxK];
  int32_t slot[kMaxK];
  int32_t hit[kMaxK];
  float g[kMaxK];
  float inv_r;
  int32_t k;
  int32_t pad[2];
};

struct TraceRec {
  int32_t kind, token, layer, rank, expert, flags, slot, victim;
};

enum { REC_ACCESS = 0, REC_PREFETCH = 1, REC_PREFILL = 2 };
enum { ERR_NONE = 0, ERR_BAD_IDS = 1, ERR_BAD_LIST = 2, ERR_BAD_PACK = 3 };

struct RouterArgs {
  const void *gate;        // [L][E][d]
  const float *h;          // [d]
  const int32_t *inj_ids;  // injected routing (test hook) or nullptr
  LayerTable *tables;
  LayerStats *stats;
  FetchList *dlists;       // demand list of each layer
  FetchList *plists;       // prefetch list targeting each layer
  RouteOut *route;
  TraceRec *trace;
  int32_t *err;
  // Records written so far (ring position = count % cap).  A launch reads
  // trace_in and writes the new count to trace_out, a second word, so that
  // the workgroups of one launch never see a count another of them updated.
  const uint64_t *trace_in;
  uint64_t *trace_out;
  uint64_t trace_cap;
  uint64_t expert_bytes;
  int layer, L, E, S, K, d, dtype, policy;
  int aging;               // aged LFU: lookup-clock ticks per halving of a count
  int demand;              // 1: route + look up `layer`
  int spec_layer;          // >= 0: guess that layer's experts from h and prefetch
  int pmax;                // prefetch at most this many guesses
};

struct FfnArgs {
  const uint8_t *arena;
  const RouteOut *route;
  float *h;                // in/out [d]
  float *act;              // [K][d_ff]
  float *part;             // [chunks][d]
  uint64_t expert_bytes;
  int layer, S, K, d, d_ff;
};

// ---- batched prefill ------------------------------------------------------
struct PrefillPlan {
  int32_t n;           // pairs routed to the expert
  int32_t off;         // first sorted position
  int32_t slot_start;  // slot before the batch, -1 if not resident
  int32_t slot_after;  // slot after the batch, -1 if not resident
  int32_t newcomer;    // became resident in this batch
  int32_t pad[3];
};

struct GemmJob {
  const uint16_t *w;  // expert base (W1 | W3 | W2), bf16
  int32_t row0;       // first sorted row of the expert
  int32_t nrows;      // rows routed to it
};

struct GemmTile {
  int32_t job, m0, n0, pad;
};

struct PrefillArgs {
  const void *gate;  // layer's gate [E][d]
  const float *H;    // [T][d]
  int32_t *ids;      // [T][K]
  float *g;          // [T][K]
  float *inv_r;      // [T]
  uint16_t *xn;      // [T][d] bf16
  int T, d, E, K, dtype;
};

struct PlanArgs {
  const int32_t *ids;
  int32_t *perm_tok;  // [T*K] sorted position -> token
  int32_t *pos_of;    // [T*K] (token, rank) -> sorted position
  PrefillPlan *plan;  // [E]
  LayerTable *table;
  LayerStats *stats;
  TraceRec *trace;
  const uint64_t *trace_in;  // record count before / after, as in RouterArgs
  uint64_t *trace_out;
  uint64_t trace_cap;
  int32_t *err;
  uint64_t expert_bytes;
  int T, K, E, S, layer, policy;
  int aging;  // aged LFU: lookup-clock ticks per halving of a count
  // Batches planned on the device (a slot for every expert): the kernel also
  // writes one GEMM job per expert; nullptr otherwise.  Small batches
  // (ntiles == nullptr) take one small-M tile per expert.  Large ones take
  // tile lists of tile_rows rows by up_cols / dn_cols columns, ordered (expert,
  // column block, row block): the up list at tiles[0 ..], the down list at
  // tiles[dn_first ..], at most up_cap and dn_cap tiles, their lengths
  // written to ntiles[0] and ntiles[1].
  GemmJob *jobs;
  GemmTile *tiles;
  int32_t *ntiles;
  int tile_rows, up_cols, dn_cols, up_cb, dn_cb, dn_first, up_cap, dn_cap;
  const uint8_t *arena_layer;  // this layer's slots
  uint64_t slot_bytes;
};

// Where a kernel goes: its stream and, when kernel timing is on, two events
// the dispatch itself stamps at the kernel's start and end.
struct Launch {
  hipStream_t s = nullptr;
  hipEvent_t start = nullptr, stop = nullptr;
};
#define MOE_LAUNCH(kernel, grid, block, shmem, L, ...) \
  hipExtLaunchKernelGGL(kernel, grid, block, shmem, (L).s, (L).start, (L).stop, 0, __VA_ARGS__)

// launchers (one per translation unit that owns the kernel)
// Streaming read of bytes (a multiple of 16) at buf with the given number of
// workgroups; reads only.
hipError_t launch_hbm_read_probe(const void *buf, size_t bytes, int workgroups, hipStream_t s);
// Copy bytes (a multiple of 16) from src_dev (the device address of mapped
// pinned host memory) to dst with the fetch kernel's access pattern.
hipError_t launch_h2d_copy_probe(const void *src_dev, void *dst, size_t bytes, int workgroups, hipStream_t s);
// Register-only bf16 MFMA loop; returns the flops the launch performs.
double launch_mfma_bf16_probe(int shape, int workgroups, int iters, hipStream_t s);
hipError_t launch_router(const RouterArgs &a, const Launch &l);
// Copies of a fetch list: expert e of the list's layer from its host store
// (stride src_stride) into its HBM slot (stride expert_bytes), or, when
// staging is non-NULL, entry i into staging + i * src_stride.
hipError_t launch_fetch(const FetchList *list, const uint8_t *const *layers, uint8_t *arena, int L, int E,
                        int S, int K, uint64_t expert_bytes, uint64_t src_stride, uint8_t *staging,
                        int32_t *err, const Launch &l);
// Packed experts of a fetch list, entry i at staging + i * 3 * mat_cap, rebuilt
// as bf16 into their slots; n = weights per matrix.
hipError_t launch_unpack(const FetchList *list, const uint8_t *staging, uint8_t *arena, int L, int S, int K,
                         uint64_t mat_cap, uint64_t expert_bytes, uint64_t n, int32_t *err, const Launch &l);
// Entropy-coded experts (host format 2): the same, from the entropy layout
// with cap_words stream words per matrix.
hipError_t launch_entropy_unpack(const FetchList *list, const uint8_t *staging, uint8_t *arena, int L, int S, int K,
                                 uint64_t mat_cap, uint64_t expert_bytes, uint64_t n, uint64_t cap_words,
                                 int32_t *err, const Launch &l);
// Bytes of one entropy-coded matrix (0 unless n is a positive multiple of 512)
// and the host encoder (0, or -1 with *why set).
uint64_t entropy_matrix_bytes(uint64_t n, uint64_t cap_words);
int entropy_pack(const uint16_t *w, uint64_t n, uint64_t cap_words, uint8_t *out, uint64_t *used, const char **why);
hipError_t launch_ffn_up(const FfnArgs &a, int dtype, const Launch &l);
hipError_t launch_ffn_down(const FfnArgs &a, int dtype, const Launch &l);
hipError_t launch_ffn_reduce(const FfnArgs &a, int dtype, const Launch &l);
int ffn_down_chunks(int K, int d_ff, int dtype);
// True when launch_ffn_down also adds the partials into h (no reduce launch).
bool ffn_down_fused(int K, int d_ff, int dtype);
// group-quantised experts (dtype 2)
hipError_t launch_ffnq_up(const FfnArgs &a, const Launch &l);
hipError_t launch_ffnq_down(const FfnArgs &a, const Launch &l);
int ffnq_down_chunks(int K, int d_ff);
hipError_t launch_prefill_gate(const PrefillArgs &a, const Launch &l);
hipError_t launch_prefill_plan(const PlanArgs &a, const Launch &l);
// grouped GEMMs over tiles of `rows` (64, 128 or 256) sorted pairs by
// prefill_tile_cols(up) output columns; a_bytes: size of the A operand's
// buffer (xn for up, act for down).  With dev_ntiles, the list's length is
// read on the device (at most ntiles, the grid; the surplus workgroups exit).
hipError_t launch_prefill_up(const GemmTile *tiles, int ntiles, const GemmJob *jobs, const uint16_t *xn,
                             const int32_t *perm_tok, uint16_t *act, int d, int d_ff, int rows, size_t a_bytes,
                             const Launch &l, const int32_t *dev_ntiles = nullptr);
// Small-M grouped GEMMs: one tile {job, 0, 0} per expert, each with at most
// max_rows <= kSkinnyRows rows (the caller's bound: rows beyond 16 are read
// only when max_rows > 16); a workgroup per (tile, 16 output features).
constexpr int kSkinnyRows = 32;
hipError_t launch_prefill_skinny_up(const GemmTile *tiles, int ntiles, const GemmJob *jobs, const uint16_t *xn,
                                    const int32_t *perm_tok, uint16_t *act, int d, int d_ff, int max_rows,
                                    const Launch &l);
hipError_t launch_prefill_skinny_down(const GemmTile *tiles, int ntiles, const GemmJob *jobs, const uint16_t *act,
                                      float *Y, int d, int d_ff, int max_rows, const Launch &l);
hipError_t launch_prefill_down(const GemmTile *tiles, int ntiles, const GemmJob *jobs, const uint16_t *act,
                               float *Y, int d, int d_ff, int rows, size_t a_bytes, const Launch &l,
                               const int32_t *dev_ntiles = nullptr);
hipError_t launch_prefill_unpermute(float *H, const float *Y, const float *g, const int32_t *pos_of, int T,
                                    int d, int K, const Launch &l);
int prefill_tile_cols(bool up);  // GEMM output tile columns (act for up, Y for down)

// ---------------------------------------------------------------------------
// device helpers

// 8 bf16 (one 16-byte load) -> 8 fp32; bf16 is the top half of an fp32.
__device__ __forceinline__ void bf16x8_to_f32(const uint4 v, float *f) {
  f[0] = __uint_as_float(v.x << 16);
  f[1] = __uint_as_float(v.x & 0xFFFF0000u);
  f[2] = __uint_as_float(v.y << 16);
  f[3] = __uint_as_float(v.y & 0xFFFF0000u);
  f[4] = __uint_as_float(v.z << 16);
  f[5] = __uint_as_float(v.z & 0xFFFF0000u);
  f[6] = __uint_as_float(v.w << 16);
  f[7] = __uint_as_float(v.w & 0xFFFF0000u);
}

// Aged LFU key: the usage count halved (rounding down) once per `aging` ticks
// between the expert's last use and `clock`.
__device__ __forceinline__ uint32_t aged_count(uint32_t count, int64_t last, int64_t clock, int aging) {
  const int64_t halvings = (clock - last) / aging;
  return halvings >= 32 ? 0u : count >> (int)halvings;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

// Top-K of E <= 64 logits held in LDS, in rank order: larger z first, lower
// id on ties, NaN ranked as -inf.  Lane e < E counts the entries that come
// before its own in that order, which is its rank, and rank r < K writes its
// id to out[r].  Returns out[lane] on lanes < K and -1 elsewhere.  Called by
// one whole wave; `out` is LDS owned by that wave.
__device__ __forceinline__ double rank_key(double z) { return z != z ? -__builtin_inf() : z; }

__device__ inline int wave_topk_lds(const double *z, int E, int K, int lane, int *out) {
  if (lane < E) {
    const double mine = rank_key(z[lane]);
    int rank = 0;
#pragma unroll 8
    for (int o = 0; o < E; ++o) {
      const double zo = rank_key(z[o]);
      rank += (zo > mine || (zo == mine && o < lane)) ? 1 : 0;
    }
    if (rank < K) out[rank] = lane;
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  return lane < K ? out[lane] : -1;
}

}  // namespace moe
