// Host engine behind the C ABI: argument checks, workspace layout, stream and
// event choreography, fetch issue, readback of statistics, trace and tables.
//
// Per decoded token and layer the engine only enqueues work:
//   compute stream: router (routing + table update + fetch lists)
//                   [-> wait(P[l]) if layer l has speculative copies in flight]
//                   -> fetch demand misses -> FFN up -> FFN down -> reduce (h += y)
//   copy stream:    wait(router, demand fetch) -> fetch next-layer
//                   prefetches -> event P[l+1]
// (A coded host store's demand copies share the staging area with the
// speculative ones, so they run on the copy stream instead, ending in event
// D[l] that the FFN waits for.)  Every copy waits for the router that chose
// it, and that router runs after all compute that read the victim slot
// earlier (stream order), so a slot is never overwritten while an FFN still
// reads it.  Every FFN waits for the copies that filled its slots (Sec. 6.1
// asks for transfers overlapped with compute; here the next layer's
// speculative copies run while this layer's FFN computes).
#include "common.hpp"
#include "moe_offload.h"

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <new>
#include <string>
#include <vector>

using namespace moe;

namespace {

thread_local std::string g_err;

int fail(int code, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

struct Layout {
  size_t tables = 0, stats = 0, dlists = 0, plists = 0, route = 0, err = 0, act = 0, part = 0,
         hostptrs = 0, prefill = 0, staging = 0, total = 0;
};

bool misaligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) != 0; }

// Process-wide pool of the runtime objects handles own: events, the side
// stream and the small pinned host buffers.  A handle takes them at bind and
// gives them back at destroy; they are never destroyed while the process
// runs.  Draining a stream only waits for its last completion signal: the
// runtime, and a profiler attached to it, may still be running completion
// handlers for the same dispatches on worker threads, and those handlers
// read the events the dispatches stamped.  Releasing an event, stream or
// pinned buffer right after the drain could pull memory out from under such
// a handler; returning it to this pool cannot.
struct Pool {
  std::vector<hipEvent_t> sync_ev, timed_ev;
  std::vector<hipStream_t> streams;
  std::multimap<size_t, void *> pinned;  // by size
};
std::mutex g_pool_mu;
std::map<int, Pool> g_pool;  // by device

hipError_t pool_event(int dev, bool timed, hipEvent_t *e) {
  {
    std::lock_guard<std::mutex> g(g_pool_mu);
    auto &v = timed ? g_pool[dev].timed_ev : g_pool[dev].sync_ev;
    if (!v.empty()) {
      *e = v.back();
      v.pop_back();
      return hipSuccess;
    }
  }
  return timed ? hipEventCreate(e) : hipEventCreateWithFlags(e, hipEventDisableTiming);
}

hipError_t pool_stream(int dev, hipStream_t *s) {
  {
    std::lock_guard<std::mutex> g(g_pool_mu);
    auto &v = g_pool[dev].streams;
    if (!v.empty()) {
      *s = v.back();
      v.pop_back();
      return hipSuccess;
    }
  }
  return hipStreamCreateWithFlags(s, hipStreamNonBlocking);
}

// Pinned host memory of at least `bytes`; *got = the size actually held.
hipError_t pool_pinned(int dev, size_t bytes, void **p, size_t *got) {
  {
    std::lock_guard<std::mutex> g(g_pool_mu);
    auto &m = g_pool[dev].pinned;
    auto it = m.lower_bound(bytes);
    if (it != m.end() && it->first <= 2 * bytes + 4096) {
      *got = it->first;
      *p = it->second;
      m.erase(it);
      return hipSuccess;
    }
  }
  *got = bytes;
  return hipHostMalloc(p, bytes, hipHostMallocDefault);
}

void pool_give_back(int dev, const std::vector<hipEvent_t> &sync_ev, const std::vector<hipEvent_t> &timed_ev,
                    hipStream_t stream, const std::vector<std::pair<size_t, void *>> &pinned) {
  std::lock_guard<std::mutex> g(g_pool_mu);
  Pool &pl = g_pool[dev];
  for (hipEvent_t e : sync_ev)
    if (e) pl.sync_ev.push_back(e);
  for (hipEvent_t e : timed_ev)
    if (e) pl.timed_ev.push_back(e);
  if (stream) pl.streams.push_back(stream);
  for (const auto &b : pinned)
    if (b.second) pl.pinned.emplace(b.first, b.second);
}

// Scratch of moe_decode_layer_noalloc: the decode FFN's activations
// [K][d_ff] and partial row sums [chunks][d], and the router's logits of a
// separate GEMV launch, in device memory the library holds for the life of
// the process (one copy per device).  Host code never uses the array's name
// as an address: each device's address comes from hipGetSymbolAddress.
constexpr size_t kNoAllocScratchBytes = size_t(4) << 20;
}  // namespace
static __device__ __align__(256) uint8_t scratch[kNoAllocScratchBytes];
namespace {
std::mutex g_scratch_mu;
std::map<int, uint8_t *> g_scratch_ptr;  // by device

// The current device's copy of `scratch` (resolved once per device).
hipError_t scratch_on_device(int dev, uint8_t **out) {
  std::lock_guard<std::mutex> g(g_scratch_mu);
  auto it = g_scratch_ptr.find(dev);
  if (it != g_scratch_ptr.end()) {
    *out = it->second;
    return hipSuccess;
  }
  void *p = nullptr;
  hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  if (e != hipSuccess || p == nullptr) return e != hipSuccess ? e : hipErrorInvalidSymbol;
  g_scratch_ptr[dev] = static_cast<uint8_t *>(p);
  *out = static_cast<uint8_t *>(p);
  return hipSuccess;
}

}  // namespace

namespace moe {
// Prefill workspace for batches of up to T tokens (offsets from its base).
struct PrefillLayout {
  size_t ids = 0, g = 0, inv_r = 0, xn = 0, perm = 0, pos = 0, plan = 0, jobs = 0, tiles = 0, act = 0,
         y = 0, staging = 0, coded = 0, lists = 0, ntiles = 0, total = 0;
  int tile_cap = 0;  // GEMM tiles the schedule can hold
  int ring = 0;      // staging slots for experts streamed through the batch
};
// fetch lists one prefill layer can need with a coded host store
constexpr int kPrefillLists = 2 * kMaxE + 2;

// Bh > 0: a coded host store, whose experts are copied to `coded` (room for
// half a ring) and rebuilt from there through device-side fetch lists.
static PrefillLayout prefill_layout(int K, int d, int d_ff, int E, int S, int T, uint64_t B, uint64_t Bh) {
  PrefillLayout p;
  if (T <= 0) return p;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t at = off;
    off = align_up(off + bytes, 256);
    return at;
  };
  const size_t P = (size_t)T * K;
  const int rows = 64;
  p.tile_cap = (int)((P + rows - 1) / rows + E) * ((d_ff + rows - 1) / rows + (d + rows - 1) / rows);
  int half = (E - S + 1) / 2;
  half = half < 1 ? 1 : (half > 4 ? 4 : half);
  p.ring = 2 * half;
  p.ids = take(P * 4);
  p.g = take(P * 4);
  p.inv_r = take((size_t)T * 4);
  p.xn = take((size_t)T * d * 2);
  p.perm = take(P * 4);
  p.pos = take(P * 4);
  p.plan = take(sizeof(PrefillPlan) * kMaxE);
  p.jobs = take(sizeof(GemmJob) * kMaxE);
  p.tiles = take(sizeof(GemmTile) * (size_t)p.tile_cap);
  p.act = take(P * d_ff * 2);
  p.y = take(P * d * 4);
  p.staging = take((size_t)p.ring * B);
  p.coded = take(Bh ? (size_t)(p.ring / 2) * Bh : 0);
  p.lists = take(Bh ? sizeof(FetchList) * kPrefillLists : 0);
  p.ntiles = take(2 * sizeof(int32_t));  // lengths of device-written tile lists
  p.total = off;
  return p;
}
}  // namespace moe

struct moe_cache {
  int L = 0, E = 0, S = 0, policy = 0;
  bool bound = false;
  bool pooled = false;   // holds runtime objects taken from the process pool
  moe_model_desc desc{};
  int K = 0, d = 0, dff = 0, dtype = 0, pmax = 0, fetch_mode = 0, max_T = 0;
  int cus = 0;           // compute units of the device (prefill tile sizing), read on first use
  uint64_t B = 0;        // bytes of one expert in an HBM slot
  int host_format = 0;   // MOE_HOST_*
  uint64_t Bh = 0;       // stride of one expert in the host store (bytes a miss moves)
  uint64_t mat_cap = 0;  // packed store: bytes of one matrix
  uint64_t n_mat = 0;    // weights per matrix
  uint8_t *staging = nullptr;  // packed store: K copied experts before unpacking
  hipStream_t cs = nullptr, xs = nullptr;
  bool one_stream = true;
  Layout lay;
  uint8_t *ws = nullptr;
  LayerTable *tables = nullptr;
  LayerStats *stats = nullptr;
  FetchList *dl = nullptr, *pl = nullptr;
  RouteOut *route = nullptr;
  int32_t *err = nullptr;
  // device: records written to the trace ring, two words; each launch that
  // writes records reads trace_count[tpar] and writes trace_count[1 - tpar],
  // and the host flips tpar once it is enqueued
  uint64_t *trace_count = nullptr;
  int tpar = 0;
  float *act = nullptr, *part = nullptr;
  uint8_t *prefill_ws = nullptr;
  std::vector<const uint8_t *> host_layer;  // host address of layer l's experts
  const uint8_t *const *dev_layers = nullptr;  // device array: layer l's experts as the GPU sees them
  std::vector<const uint8_t *> dev_layer_host;  // what that array must hold
  std::vector<hipEvent_t> ev_demand, ev_pf;
  hipEvent_t ev_router = nullptr;
  hipStream_t ms = nullptr;  // library-owned: prefetch-list read-back (split fetch mode)
  std::vector<uint8_t> demand_pending, pf_pending;
  int sticky = MOE_OK;
  int dev = 0;                  // device the handle was bound on (owner of its pooled objects)
  uint8_t *scratch = nullptr;   // that device's static scratch (moe_decode_layer_noalloc)
  FetchList *mirror = nullptr;  // pinned host: demand list, prefetch list, error word (DMA / split modes)
  size_t mirror_bytes = 0, plan_bytes = 0, sched_bytes = 0;  // sizes of the pooled pinned buffers
  int last_route_kind = 0;      // 0 none, 1 decode, 2 prefill
  int last_prefill_T = 0;
  // batched prefill
  PrefillLayout play;
  PrefillPlan *h_plan = nullptr;   // pinned: plan of the last prefill layer
  uint8_t *h_sched = nullptr;      // pinned: GEMM jobs + tiles uploaded per layer
  std::vector<hipEvent_t> pf_ev;   // prefill ordering events
  // kernel timing (moe_cache_set_timing)
  int timing = MOE_TIMING_OFF;
  std::vector<hipEvent_t> ev_pool;
  struct Span {
    int kind;
    hipEvent_t a, b;
    double flop;
  };
  std::vector<Span> spans;
};

namespace moe {
enum SpanKind {
  SPAN_ROUTER = 0, SPAN_FETCH, SPAN_UP, SPAN_DOWN, SPAN_PREFILL, SPAN_GEMM_UP, SPAN_GEMM_DOWN, SPAN_REDUCE,
  SPAN_UNPACK, SPAN_WAIT, SPAN_PF_FETCH, SPAN_KINDS
};

// Whether spans of this kind are recorded at the handle's timing level.
bool timed(const moe_cache *c, int kind) {
  return c->timing == MOE_TIMING_ALL || (c->timing == MOE_TIMING_FFN_UP && kind == SPAN_UP);
}

// An event for a timed span: the handle's own spare, else one from the
// process pool.
hipError_t take_timed_event(moe_cache *c, hipEvent_t *e) {
  if (!c->ev_pool.empty()) {
    *e = c->ev_pool.back();
    c->ev_pool.pop_back();
    return hipSuccess;
  }
  return pool_event(c->dev, true, e);
}

// Start/stop a timed span on stream s (no-op unless its kind is timed).
hipError_t span_begin(moe_cache *c, hipStream_t s, hipEvent_t *out, int kind) {
  *out = nullptr;
  if (!timed(c, kind)) return hipSuccess;
  hipEvent_t e;
  hipError_t r = take_timed_event(c, &e);
  if (r != hipSuccess) return r;
  *out = e;
  return hipEventRecord(e, s);
}

hipError_t span_end(moe_cache *c, hipStream_t s, int kind, hipEvent_t begin, double flop = 0.0) {
  if (!begin) return hipSuccess;
  hipEvent_t e;
  hipError_t r = take_timed_event(c, &e);
  if (r != hipSuccess) return r;
  c->spans.push_back({kind, begin, e, flop});
  return hipEventRecord(e, s);
}

// A kernel launch on stream s; with timing on it carries two pooled events
// that the dispatch itself stamps at the kernel's start and end.
hipError_t kernel_span(moe_cache *c, hipStream_t s, Launch *l, int kind) {
  l->s = s;
  l->start = l->stop = nullptr;
  if (!timed(c, kind)) return hipSuccess;
  for (hipEvent_t *e : {&l->start, &l->stop}) {
    hipError_t r = take_timed_event(c, e);
    if (r != hipSuccess) return r;
  }
  return hipSuccess;
}

void kernel_span_done(moe_cache *c, int kind, const Launch &l, double flop = 0.0) {
  if (l.start) c->spans.push_back({kind, l.start, l.stop, flop});
}
}  // namespace moe

namespace moe {
int prefill_enqueue(moe_cache *c, int layer, float *H, int T);
int prefill_routing(moe_cache *c, int32_t *ids, float *g, size_t cap, size_t *n);
}  // namespace moe

#define HIP_TRY(c, expr)                                                                  \
  do {                                                                                    \
    hipError_t _e = (expr);                                                               \
    if (_e != hipSuccess) {                                                               \
      if (c) (c)->sticky = MOE_ERR_HIP;                                                   \
      return fail(MOE_ERR_HIP, "%s failed: %s", #expr, hipGetErrorString(_e));            \
    }                                                                                     \
  } while (0)

#define HIP_TRY0(expr)                                                                    \
  do {                                                                                    \
    hipError_t _e = (expr);                                                               \
    if (_e != hipSuccess) return fail(MOE_ERR_HIP, "%s failed: %s", #expr, hipGetErrorString(_e)); \
  } while (0)

// The kernel that rebuilds the bf16 experts of a fetch list (at most `max_n`
// entries) from a coded host store's bytes at `coded` (entry i at
// coded + i * Bh) into dst + (list layer * S + list slot) * B.
static hipError_t launch_rebuild(const moe_cache *c, const FetchList *list, const uint8_t *coded, uint8_t *dst,
                                 int L, int S, int max_n, const Launch &l) {
  if (c->host_format == MOE_HOST_ENTROPY)
    return launch_entropy_unpack(list, coded, dst, L, S, max_n, c->mat_cap, c->B, c->n_mat,
                                 (uint64_t)c->desc.packed_cap, c->err, l);
  return launch_unpack(list, coded, dst, L, S, max_n, c->mat_cap, c->B, c->n_mat, c->err, l);
}

// ... into the HBM slots of the list's layer, from the decode staging area
static hipError_t launch_rebuild(const moe_cache *c, const FetchList *list, const Launch &l) {
  return launch_rebuild(c, list, c->staging, static_cast<uint8_t *>(c->desc.arena), c->L, c->S, c->K, l);
}

static int check_ready(const moe_cache *c) {
  if (!c) return fail(MOE_ERR_ARG, "NULL handle");
  if (!c->bound) return fail(MOE_ERR_STATE, "handle is not bound (call moe_cache_bind)");
  if (c->sticky != MOE_OK)
    return fail(MOE_ERR_STATE, "an earlier device error is pending; call moe_cache_reset");
  return MOE_OK;
}

// Stored bytes of one expert (W1 | W3 | W2).
static uint64_t expert_bytes(const moe_model_desc *d) {
  const uint64_t n = (uint64_t)d->d_model * d->d_ff;
  if (d->dtype == MOE_DTYPE_Q2G16) return 3 * (n / 16 * 7);
  return 3 * n * (d->dtype == MOE_DTYPE_BF16 ? 2 : 4);
}

// Bytes of one matrix in a coded host store.  MOE_HOST_PACKED: blocks of 8192
// weights in 12560 bytes, then packed_cap exception words, rounded up to 16
// bytes; MOE_HOST_ENTROPY: see entropy_matrix_bytes.
static uint64_t coded_matrix_bytes(const moe_model_desc *d) {
  const uint64_t n = (uint64_t)d->d_model * d->d_ff;
  if (d->host_format == MOE_HOST_ENTROPY) return entropy_matrix_bytes(n, (uint64_t)d->packed_cap);
  const uint64_t nb = (n + 8191) / 8192;
  return (nb * 12560 + 4ull * (uint64_t)d->packed_cap + 15) / 16 * 16;
}

static bool coded_store(int host_format) {
  return host_format == MOE_HOST_PACKED || host_format == MOE_HOST_ENTROPY;
}

// Stride of one expert in the host store: the bytes one miss moves.
static uint64_t host_expert_bytes(const moe_model_desc *d) {
  return coded_store(d->host_format) ? 3 * coded_matrix_bytes(d) : expert_bytes(d);
}

// Element type of the gate: fp32 for fp32 models, bf16 otherwise (router dtype code).
static int gate_dtype(int dtype) { return dtype == MOE_DTYPE_F32 ? 0 : 1; }

static int validate_desc(const moe_cache *c, const moe_model_desc *d) {
  if (!c || !d) return fail(MOE_ERR_ARG, "NULL handle or description");
  if (d->d_model < 8 || d->d_model % 8 || d->d_model > 16384)
    return fail(MOE_ERR_ARG, "d_model must be a multiple of 8 in [8, 16384]");
  if (d->d_ff < 8 || d->d_ff % 8) return fail(MOE_ERR_ARG, "d_ff must be a positive multiple of 8");
  if (d->top_k < 1 || d->top_k > MOE_MAX_TOPK || d->top_k > c->E)
    return fail(MOE_ERR_ARG, "top_k must be in [1, min(experts, %d)]", MOE_MAX_TOPK);
  if (c->S < d->top_k) return fail(MOE_ERR_ARG, "slots (%d) < top_k (%d)", c->S, d->top_k);
  if (d->dtype != MOE_DTYPE_F32 && d->dtype != MOE_DTYPE_BF16 && d->dtype != MOE_DTYPE_Q2G16)
    return fail(MOE_ERR_ARG, "bad dtype");
  if (d->dtype == MOE_DTYPE_Q2G16 && (d->d_model % 64 || d->d_ff % 64 || d->d_model > 8192))
    return fail(MOE_ERR_ARG, "group-quantised experts need d_model and d_ff multiples of 64 and d_model <= 8192");
  if (d->prefetch_max < 0 || d->prefetch_max > d->top_k)
    return fail(MOE_ERR_ARG, "prefetch_max must be in [0, top_k]");
  if (d->fetch_mode != MOE_FETCH_KERNEL && d->fetch_mode != MOE_FETCH_DMA && d->fetch_mode != MOE_FETCH_SPLIT)
    return fail(MOE_ERR_ARG, "bad fetch_mode");
  if (d->max_prefill_tokens < 0) return fail(MOE_ERR_ARG, "max_prefill_tokens < 0");
  if (d->host_format != MOE_HOST_PLAIN && !coded_store(d->host_format))
    return fail(MOE_ERR_ARG, "bad host_format");
  if (coded_store(d->host_format)) {
    if (d->dtype != MOE_DTYPE_BF16) return fail(MOE_ERR_ARG, "a coded host store holds bf16 experts");
    const uint64_t n = (uint64_t)d->d_model * d->d_ff;
    if (d->host_format == MOE_HOST_PACKED && (d->packed_cap < 0 || (uint64_t)d->packed_cap > n))
      return fail(MOE_ERR_ARG, "packed_cap out of range");
    if (d->host_format == MOE_HOST_ENTROPY && (n % 512 || d->packed_cap < 1 || (uint64_t)d->packed_cap > n))
      return fail(MOE_ERR_ARG, "an entropy-coded store needs d_model * d_ff a multiple of 512 and "
                               "packed_cap in [1, d_model * d_ff]");
  }
  if (c->policy == MOE_POLICY_LFU_AGED && d->aging_ticks < 1)
    return fail(MOE_ERR_ARG, "aged LFU needs aging_ticks >= 1");
  if (d->max_prefill_tokens > 0 && d->dtype != MOE_DTYPE_BF16)
    return fail(MOE_ERR_ARG, "batched prefill runs on bf16 experts (matrix cores); dtype must be bf16");
  if ((int64_t)d->max_prefill_tokens * d->top_k > (1 << 28))
    return fail(MOE_ERR_ARG, "max_prefill_tokens * top_k too large");
  return MOE_OK;
}

static Layout make_layout(const moe_cache *c, const moe_model_desc *d) {
  Layout l;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t at = off;
    off = align_up(off + bytes, 256);
    return at;
  };
  l.tables = take(sizeof(LayerTable) * c->L);
  l.stats = take(sizeof(LayerStats) * c->L);
  l.dlists = take(sizeof(FetchList) * c->L);
  l.plists = take(sizeof(FetchList) * c->L);
  l.route = take(sizeof(RouteOut));
  l.hostptrs = take(sizeof(void *) * c->L);
  l.err = take(256);
  l.act = take(sizeof(float) * d->top_k * (size_t)d->d_ff);
  l.part = take(sizeof(float) * (size_t)ffn_down_chunks(d->top_k, d->d_ff, d->dtype) * d->d_model);
  const uint64_t B = expert_bytes(d);
  const uint64_t Bh_coded = coded_store(d->host_format) ? host_expert_bytes(d) : 0;
  l.prefill = take(prefill_layout(d->top_k, d->d_model, d->d_ff, c->E, c->S, d->max_prefill_tokens, B, Bh_coded).total);
  l.staging = take(coded_store(d->host_format) ? (size_t)d->top_k * host_expert_bytes(d) : 0);
  l.total = off;
  return l;
}

extern "C" {

const char *moe_last_error(void) { return g_err.c_str(); }

int moe_cache_create(int layers, int experts, int slots, int policy, moe_cache_t **out) {
  if (!out) return fail(MOE_ERR_ARG, "out is NULL");
  *out = nullptr;
  if (layers < 1) return fail(MOE_ERR_ARG, "layers must be >= 1");
  if (experts < 1 || experts > MOE_MAX_EXPERTS)
    return fail(MOE_ERR_ARG, "experts must be in [1, %d]", MOE_MAX_EXPERTS);
  if (slots < 1 || slots > experts) return fail(MOE_ERR_ARG, "slots must be in [1, experts]");
  if (policy != MOE_POLICY_LRU && policy != MOE_POLICY_LFU && policy != MOE_POLICY_LFU_AGED)
    return fail(MOE_ERR_ARG, "bad policy");
  moe_cache *c = new (std::nothrow) moe_cache();
  if (!c) return fail(MOE_ERR_NOMEM, "out of host memory");
  c->L = layers;
  c->E = experts;
  c->S = slots;
  c->policy = policy;
  *out = c;
  return MOE_OK;
}

size_t moe_cache_workspace_bytes(const moe_cache_t *c, const moe_model_desc *d) {
  if (validate_desc(c, d) != MOE_OK) return 0;
  return make_layout(c, d).total;
}

int moe_cache_bind(moe_cache_t *c, const moe_model_desc *d) {
  int rc = validate_desc(c, d);
  if (rc != MOE_OK) return rc;
  if (c->bound) return fail(MOE_ERR_STATE, "handle is already bound");
  if (!d->gate_w || (!d->host_experts && !d->host_layers) || !d->arena || !d->workspace)
    return fail(MOE_ERR_ARG, "gate_w, host_experts (or host_layers), arena and workspace must be non-NULL");
  if (misaligned(d->gate_w, 16) || misaligned(d->host_experts, 16) || misaligned(d->arena, 16))
    return fail(MOE_ERR_ARG, "gate_w, host_experts and arena must be 16-byte aligned");
  if (misaligned(d->workspace, 256)) return fail(MOE_ERR_ARG, "workspace must be 256-byte aligned");
  if (d->trace && (d->trace_cap == 0 || misaligned(d->trace, 16)))
    return fail(MOE_ERR_ARG, "trace needs trace_cap > 0 and 16-byte alignment");
  const Layout lay = make_layout(c, d);
  if (d->workspace_bytes < lay.total)
    return fail(MOE_ERR_ARG, "workspace too small: %zu < %zu bytes", d->workspace_bytes, lay.total);

  // per-layer host bases (one contiguous store, or the caller's per-layer table)
  const uint64_t Bh = host_expert_bytes(d);
  std::vector<const uint8_t *> hl(c->L), dl(c->L, nullptr);
  for (int l = 0; l < c->L; ++l) {
    hl[l] = d->host_layers ? static_cast<const uint8_t *>(d->host_layers[l])
                           : static_cast<const uint8_t *>(d->host_experts) + (size_t)l * c->E * Bh;
    if (!hl[l] || misaligned(hl[l], 16))
      return fail(MOE_ERR_ARG, "host store of layer %d is NULL or not 16-byte aligned", l);
  }
  if (d->fetch_mode != MOE_FETCH_DMA) {
    for (int l = 0; l < c->L; ++l) {
      void *p = nullptr;
      hipError_t e = hipHostGetDevicePointer(&p, const_cast<uint8_t *>(hl[l]), 0);
      if (e != hipSuccess || !p) {
        (void)hipGetLastError();
        return fail(MOE_ERR_ARG, "host store of layer %d is not pinned host memory mapped for the device (%s)",
                    l, hipGetErrorString(e));
      }
      dl[l] = static_cast<const uint8_t *>(p);
    }
  }
  c->desc = *d;
  c->host_layer = hl;
  c->K = d->top_k;
  c->d = d->d_model;
  c->dff = d->d_ff;
  c->dtype = d->dtype;
  c->pmax = d->prefetch_max;
  c->fetch_mode = d->fetch_mode;
  c->max_T = d->max_prefill_tokens;
  c->B = expert_bytes(d);
  c->host_format = d->host_format;
  c->Bh = host_expert_bytes(d);
  c->mat_cap = coded_store(d->host_format) ? coded_matrix_bytes(d) : 0;
  c->n_mat = (uint64_t)d->d_model * d->d_ff;
  c->cs = static_cast<hipStream_t>(d->compute_stream);
  c->xs = d->copy_stream ? static_cast<hipStream_t>(d->copy_stream) : c->cs;
  c->one_stream = (c->xs == c->cs);
  c->lay = lay;
  c->ws = static_cast<uint8_t *>(d->workspace);
  c->tables = reinterpret_cast<LayerTable *>(c->ws + lay.tables);
  c->stats = reinterpret_cast<LayerStats *>(c->ws + lay.stats);
  c->dl = reinterpret_cast<FetchList *>(c->ws + lay.dlists);
  c->pl = reinterpret_cast<FetchList *>(c->ws + lay.plists);
  c->route = reinterpret_cast<RouteOut *>(c->ws + lay.route);
  c->err = reinterpret_cast<int32_t *>(c->ws + lay.err);
  c->trace_count = reinterpret_cast<uint64_t *>(c->ws + lay.err + 8);
  c->act = reinterpret_cast<float *>(c->ws + lay.act);
  c->part = reinterpret_cast<float *>(c->ws + lay.part);
  c->prefill_ws = c->ws + lay.prefill;
  c->staging = coded_store(d->host_format) ? c->ws + lay.staging : nullptr;
  c->dev_layers = reinterpret_cast<const uint8_t *const *>(c->ws + lay.hostptrs);
  c->dev_layer_host = dl;
  HIP_TRY0(hipMemcpy(c->ws + lay.hostptrs, dl.data(), sizeof(void *) * c->L, hipMemcpyHostToDevice));

  // runtime objects come from the process pool (released there by destroy,
  // also when bind fails half way)
  HIP_TRY0(hipGetDevice(&c->dev));
  HIP_TRY0(scratch_on_device(c->dev, &c->scratch));
  c->ev_demand.assign(c->L, nullptr);
  c->ev_pf.assign(c->L, nullptr);
  c->demand_pending.assign(c->L, 0);
  c->pf_pending.assign(c->L, 0);
  c->pooled = true;  // from here on destroy returns what was taken
  for (int l = 0; l < c->L; ++l) {
    HIP_TRY0(pool_event(c->dev, false, &c->ev_demand[l]));
    HIP_TRY0(pool_event(c->dev, false, &c->ev_pf[l]));
  }
  HIP_TRY0(pool_event(c->dev, false, &c->ev_router));
  if (c->fetch_mode == MOE_FETCH_SPLIT && !c->one_stream) HIP_TRY0(pool_stream(c->dev, &c->ms));
  HIP_TRY0(pool_pinned(c->dev, 3 * sizeof(FetchList), reinterpret_cast<void **>(&c->mirror), &c->mirror_bytes));
  if (c->max_T > 0) {
    c->play = prefill_layout(c->K, c->d, c->dff, c->E, c->S, c->max_T, c->B, coded_store(c->host_format) ? c->Bh : 0);
    // the plan of every expert, then the device's error word
    HIP_TRY0(pool_pinned(c->dev, sizeof(PrefillPlan) * kMaxE + sizeof(int32_t), reinterpret_cast<void **>(&c->h_plan),
                         &c->plan_bytes));
    HIP_TRY0(pool_pinned(c->dev,
                         sizeof(GemmJob) * kMaxE + sizeof(GemmTile) * (size_t)c->play.tile_cap +
                             sizeof(FetchList) * kPrefillLists,
                         reinterpret_cast<void **>(&c->h_sched), &c->sched_bytes));
    c->pf_ev.assign(2 * kMaxE + 4, nullptr);
    for (auto &e : c->pf_ev) HIP_TRY0(pool_event(c->dev, false, &e));
  }
  c->bound = true;
  c->sticky = MOE_ERR_STATE;  // decode needs a reset first
  return MOE_OK;
}

int moe_cache_reset(moe_cache_t *c) {
  if (!c) return fail(MOE_ERR_ARG, "NULL handle");
  if (!c->bound) return fail(MOE_ERR_STATE, "handle is not bound");
  (void)hipStreamSynchronize(c->cs);
  if (!c->one_stream) (void)hipStreamSynchronize(c->xs);
  (void)hipGetLastError();

  std::vector<LayerTable> t(c->L);
  std::memset(t.data(), 0, sizeof(LayerTable) * t.size());
  for (int l = 0; l < c->L; ++l) {
    for (int s = 0; s < kMaxE; ++s) t[l].slot_expert[s] = s < c->S ? s : -1;
    for (int e = 0; e < kMaxE; ++e) {
      const bool res = e < c->S;
      t[l].expert_slot[e] = res ? e : -1;
      t[l].last[e] = res ? (int64_t)e - c->S : -(int64_t)c->S - 1;
    }
  }
  HIP_TRY(c, hipMemcpyAsync(c->tables, t.data(), sizeof(LayerTable) * c->L, hipMemcpyHostToDevice, c->cs));
  // clear exactly the regions that hold run state (never the host-pointer table)
  HIP_TRY(c, hipMemsetAsync(c->ws + c->lay.stats, 0, sizeof(LayerStats) * c->L, c->cs));
  HIP_TRY(c, hipMemsetAsync(c->ws + c->lay.dlists, 0, sizeof(FetchList) * c->L, c->cs));
  HIP_TRY(c, hipMemsetAsync(c->ws + c->lay.plists, 0, sizeof(FetchList) * c->L, c->cs));
  HIP_TRY(c, hipMemsetAsync(c->ws + c->lay.route, 0, sizeof(RouteOut), c->cs));
  HIP_TRY(c, hipMemsetAsync(c->ws + c->lay.err, 0, 256, c->cs));  // error word and both trace counts
  c->tpar = 0;
  {
    // the copy kernel dereferences this table: check it survived
    std::vector<const uint8_t *> got(c->L);
    HIP_TRY(c, hipMemcpyAsync(got.data(), c->ws + c->lay.hostptrs, sizeof(void *) * c->L,
                              hipMemcpyDeviceToHost, c->cs));
    HIP_TRY(c, hipStreamSynchronize(c->cs));
    if (got != c->dev_layer_host) {
      c->sticky = MOE_ERR_HIP;
      return fail(MOE_ERR_HIP, "device table of host-store addresses was overwritten");
    }
  }
  HIP_TRY(c, hipStreamSynchronize(c->cs));
  uint8_t *arena = static_cast<uint8_t *>(c->desc.arena);
  if (coded_store(c->host_format)) {
    // copy each coded expert to staging and rebuild it in its slot, through
    // the layer's demand list (cleared again afterwards)
    for (int l = 0; l < c->L; ++l)
      for (int s = 0; s < c->S; ++s) {
        FetchList f{};
        f.n = 1;
        f.layer = l;
        f.expert[0] = s;
        f.slot[0] = s;
        HIP_TRY(c, hipMemcpy(c->dl + l, &f, sizeof f, hipMemcpyHostToDevice));
        HIP_TRY(c, hipMemcpy(c->staging, c->host_layer[l] + (size_t)s * c->Bh, c->Bh, hipMemcpyHostToDevice));
        HIP_TRY(c, launch_rebuild(c, c->dl + l, Launch{c->xs}));
        HIP_TRY(c, hipStreamSynchronize(c->xs));
      }
    HIP_TRY(c, hipMemsetAsync(c->ws + c->lay.dlists, 0, sizeof(FetchList) * c->L, c->xs));
    int32_t e = 0;
    HIP_TRY(c, hipMemcpyAsync(&e, c->err, sizeof e, hipMemcpyDeviceToHost, c->xs));
    HIP_TRY(c, hipStreamSynchronize(c->xs));
    if (e != ERR_NONE) {
      c->sticky = MOE_ERR_ARG;
      return fail(MOE_ERR_ARG, c->host_format == MOE_HOST_PACKED
                                   ? "packed host store is corrupt (an exception entry is missing)"
                                   : "entropy-coded host store is corrupt (a stream holds no valid code)");
    }
  } else {
    for (int l = 0; l < c->L; ++l)
      for (int s = 0; s < c->S; ++s)
        HIP_TRY(c, hipMemcpyAsync(arena + ((size_t)l * c->S + s) * c->B, c->host_layer[l] + (size_t)s * c->B,
                                  c->B, hipMemcpyHostToDevice, c->xs));
  }
  HIP_TRY(c, hipStreamSynchronize(c->xs));
  std::fill(c->demand_pending.begin(), c->demand_pending.end(), 0);
  std::fill(c->pf_pending.begin(), c->pf_pending.end(), 0);
  c->last_route_kind = 0;
  c->last_prefill_T = 0;
  c->sticky = MOE_OK;
  return MOE_OK;
}

}  // extern "C"

// Issue the copies for one fetch list that the router just wrote.
// A packed store's experts land in staging and are rebuilt into their slots
// by an unpack kernel behind the copies on the same stream.
static int unpack_list(moe_cache *c, FetchList *list, hipStream_t q) {
  Launch l;
  HIP_TRY(c, kernel_span(c, q, &l, SPAN_UNPACK));
  HIP_TRY(c, launch_rebuild(c, list, l));
  kernel_span_done(c, SPAN_UNPACK, l);
  return MOE_OK;
}

static int issue_fetch(moe_cache *c, FetchList *list, int mirror_idx, hipStream_t q) {
  const bool by_kernel = c->fetch_mode == MOE_FETCH_KERNEL || (c->fetch_mode == MOE_FETCH_SPLIT && mirror_idx == 0);
  const bool packed = coded_store(c->host_format);
  const int kind = mirror_idx == 1 ? SPAN_PF_FETCH : SPAN_FETCH;  // speculative or demand copies
  if (by_kernel) {
    Launch l;
    HIP_TRY(c, kernel_span(c, q, &l, kind));
    HIP_TRY(c, launch_fetch(list, c->dev_layers, static_cast<uint8_t *>(c->desc.arena), c->L, c->E, c->S,
                            c->K, c->B, c->Bh, c->staging, c->err, l));
    kernel_span_done(c, kind, l);
    return packed ? unpack_list(c, list, q) : MOE_OK;
  }
  const FetchList &m = c->mirror[mirror_idx];
  if (m.n < 0 || m.n > c->K || m.layer < 0 || m.layer >= c->L) {
    c->sticky = MOE_ERR_HIP;
    return fail(MOE_ERR_HIP, "inconsistent fetch list from the device");
  }
  const uint8_t *host = c->host_layer[m.layer];
  uint8_t *arena = static_cast<uint8_t *>(c->desc.arena);
  if (m.n == 0) return MOE_OK;
  hipEvent_t t0;
  HIP_TRY(c, span_begin(c, q, &t0, kind));
  for (int i = 0; i < m.n; ++i) {
    const int e = m.expert[i], s = m.slot[i];
    if (e < 0 || e >= c->E || s < 0 || s >= c->S) {
      c->sticky = MOE_ERR_HIP;
      return fail(MOE_ERR_HIP, "inconsistent fetch entry from the device");
    }
    uint8_t *dst = packed ? c->staging + (size_t)i * c->Bh : arena + ((size_t)m.layer * c->S + s) * c->B;
    HIP_TRY(c, hipMemcpyAsync(dst, host + (size_t)e * c->Bh, c->Bh, hipMemcpyHostToDevice, q));
  }
  HIP_TRY(c, span_end(c, q, kind, t0));
  return packed ? unpack_list(c, list, q) : MOE_OK;
}

// Router (+ fetches, + FFN) for one call.  spec_layer < 0: no speculation.
// Scratch of one call: FFN activations and partial sums.
struct CallScratch {
  float *act, *part;
};

static CallScratch workspace_scratch(moe_cache *c) { return {c->act, c->part}; }

static int enqueue_layer(moe_cache *c, int layer, float *h, const int32_t *inj, int demand,
                         int spec_layer, int pmax, bool ffn, const CallScratch &scr) {
  if (!c->one_stream) {
    if (demand && c->demand_pending[layer]) HIP_TRY(c, hipStreamWaitEvent(c->cs, c->ev_demand[layer], 0));
    if (spec_layer >= 0 && c->pf_pending[spec_layer])
      HIP_TRY(c, hipStreamWaitEvent(c->cs, c->ev_pf[spec_layer], 0));
  }
  RouterArgs a{};
  a.gate = c->desc.gate_w;
  a.h = h;
  a.inj_ids = inj;
  a.tables = c->tables;
  a.stats = c->stats;
  a.dlists = c->dl;
  a.plists = c->pl;
  a.route = c->route;
  a.trace = static_cast<TraceRec *>(c->desc.trace);
  a.err = c->err;
  a.trace_in = c->trace_count + c->tpar;
  a.trace_out = c->trace_count + (1 - c->tpar);
  a.trace_cap = c->desc.trace ? c->desc.trace_cap : 0;
  a.expert_bytes = c->Bh;  // bytes one fetch moves (counters)
  a.layer = layer;
  a.L = c->L;
  a.E = c->E;
  a.S = c->S;
  a.K = c->K;
  a.d = c->d;
  a.dtype = gate_dtype(c->dtype);
  a.policy = c->policy;
  a.aging = c->policy == MOE_POLICY_LFU_AGED ? c->desc.aging_ticks : 0;
  a.demand = demand;
  a.spec_layer = spec_layer;
  a.pmax = pmax;
  Launch lr;
  HIP_TRY(c, kernel_span(c, c->cs, &lr, SPAN_ROUTER));
  HIP_TRY(c, launch_router(a, lr));
  c->tpar ^= 1;
  kernel_span_done(c, SPAN_ROUTER, lr);
  // from the router's end to the FFN's start: the compute stream's wait for
  // the copies that fill this layer's slots
  hipEvent_t t_wait = nullptr;
  if (ffn) HIP_TRY(c, span_begin(c, c->cs, &t_wait, SPAN_WAIT));

  hipStream_t q = c->xs;
  const bool split = c->fetch_mode == MOE_FETCH_SPLIT;
  // With a slot for every expert, all of them are resident from the warm
  // start on and no lookup or guess can ever need a copy: the fetch lists the
  // router writes are always empty, so no copy is issued and nothing waits
  // for one (no fetch launch, no cross-stream event, no host read-back).
  const bool no_copies = c->S == c->E;
  // A plain store's demand copies (kernel and split modes) go on the compute
  // stream: the FFN waits for them anyway, and stream order then replaces the
  // two cross-stream waits (router -> copy stream -> FFN) that cost tens of
  // microseconds a layer even when nothing misses.  Coded stores keep them on
  // the copy stream, where they share the staging area with speculative copies.
  const bool demand_on_cs =
      !c->one_stream && c->fetch_mode != MOE_FETCH_DMA && !coded_store(c->host_format);
  hipStream_t qd = demand_on_cs ? c->cs : q;
  if (no_copies) {
    // nothing to copy (see above)
  } else if (c->fetch_mode != MOE_FETCH_DMA) {
    if (!c->one_stream && ((demand && !demand_on_cs) || spec_layer >= 0)) {
      HIP_TRY(c, hipEventRecord(c->ev_router, c->cs));
      HIP_TRY(c, hipStreamWaitEvent(q, c->ev_router, 0));
    }
  } else {
    if (demand) HIP_TRY(c, hipMemcpyAsync(&c->mirror[0], c->dl + layer, sizeof(FetchList), hipMemcpyDeviceToHost, c->cs));
    if (spec_layer >= 0)
      HIP_TRY(c, hipMemcpyAsync(&c->mirror[1], c->pl + spec_layer, sizeof(FetchList), hipMemcpyDeviceToHost, c->cs));
    int32_t *err_mirror = reinterpret_cast<int32_t *>(&c->mirror[2]);
    HIP_TRY(c, hipMemcpyAsync(err_mirror, c->err, sizeof(int32_t), hipMemcpyDeviceToHost, c->cs));
    HIP_TRY(c, hipStreamSynchronize(c->cs));  // one wait for the lists and the error word
    if (*err_mirror != ERR_NONE) return MOE_OK;  // reported at the next synchronising call
  }
  if (demand && !no_copies) {
    // a slot the router just took may still be receiving a speculative copy
    if (demand_on_cs && c->pf_pending[layer]) {
      HIP_TRY(c, hipStreamWaitEvent(c->cs, c->ev_pf[layer], 0));
      c->pf_pending[layer] = 0;
    }
    int rc = issue_fetch(c, c->dl + layer, 0, qd);
    if (rc != MOE_OK) return rc;
    if (!c->one_stream) {
      HIP_TRY(c, hipEventRecord(c->ev_demand[layer], qd));
      if (demand_on_cs) {
        // speculative copies queue behind this layer's demand copies
        if (spec_layer >= 0) HIP_TRY(c, hipStreamWaitEvent(q, c->ev_demand[layer], 0));
      } else {
        c->demand_pending[layer] = 1;
      }
    }
  }
  if (spec_layer >= 0 && !split && !no_copies) {
    int rc = issue_fetch(c, c->pl + spec_layer, 1, q);
    if (rc != MOE_OK) return rc;
    if (!c->one_stream) {
      HIP_TRY(c, hipEventRecord(c->ev_pf[spec_layer], q));
      c->pf_pending[spec_layer] = 1;
    }
  }
  if (ffn) {
    if (!c->one_stream) {
      if (c->demand_pending[layer]) HIP_TRY(c, hipStreamWaitEvent(c->cs, c->ev_demand[layer], 0));
      if (c->pf_pending[layer]) HIP_TRY(c, hipStreamWaitEvent(c->cs, c->ev_pf[layer], 0));
      c->demand_pending[layer] = 0;
      c->pf_pending[layer] = 0;
    }
    FfnArgs f{};
    f.arena = static_cast<const uint8_t *>(c->desc.arena);
    f.route = c->route;
    f.h = h;
    f.act = scr.act;
    f.part = scr.part;
    f.expert_bytes = c->B;
    f.layer = layer;
    f.S = c->S;
    f.K = c->K;
    f.d = c->d;
    f.d_ff = c->dff;
    HIP_TRY(c, span_end(c, c->cs, SPAN_WAIT, t_wait));
    Launch lu, ld, lx;
    HIP_TRY(c, kernel_span(c, c->cs, &lu, SPAN_UP));
    HIP_TRY(c, launch_ffn_up(f, c->dtype, lu));
    kernel_span_done(c, SPAN_UP, lu);
    HIP_TRY(c, kernel_span(c, c->cs, &ld, SPAN_DOWN));
    HIP_TRY(c, launch_ffn_down(f, c->dtype, ld));
    kernel_span_done(c, SPAN_DOWN, ld);
    if (!ffn_down_fused(c->K, c->dff, c->dtype)) {
      HIP_TRY(c, kernel_span(c, c->cs, &lx, SPAN_REDUCE));
      HIP_TRY(c, launch_ffn_reduce(f, c->dtype, lx));
      kernel_span_done(c, SPAN_REDUCE, lx);
    }
    c->last_route_kind = 1;
  }
  if (spec_layer >= 0 && split && !no_copies) {
    // The prefetch list comes back on the library's own stream, so neither the
    // FFN just enqueued nor the demand copies wait for the host; the runtime copies
    // then queue on the copy stream behind this layer's demand copies.
    hipStream_t m = c->ms ? c->ms : c->cs;
    int32_t *err_mirror = reinterpret_cast<int32_t *>(&c->mirror[2]);
    if (c->ms) HIP_TRY(c, hipStreamWaitEvent(m, c->ev_router, 0));
    HIP_TRY(c, hipMemcpyAsync(&c->mirror[1], c->pl + spec_layer, sizeof(FetchList), hipMemcpyDeviceToHost, m));
    HIP_TRY(c, hipMemcpyAsync(err_mirror, c->err, sizeof(int32_t), hipMemcpyDeviceToHost, m));
    HIP_TRY(c, hipStreamSynchronize(m));
    if (*err_mirror != ERR_NONE) return MOE_OK;  // reported at the next synchronising call
    int rc = issue_fetch(c, c->pl + spec_layer, 1, q);
    if (rc != MOE_OK) return rc;
    if (!c->one_stream) {
      HIP_TRY(c, hipEventRecord(c->ev_pf[spec_layer], q));
      c->pf_pending[spec_layer] = 1;
    }
  }
  return MOE_OK;
}

namespace moe {

constexpr int kTallRows = 256;  // rows of a device-planned tile

// compute units of the handle's device (read once)
static int device_cus(moe_cache *c) {
  if (c->cus <= 0) {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
      cus = 256;
    (void)hipGetLastError();
    c->cus = cus;
  }
  return c->cus;
}

// Batched prefill of one layer.  Routing and the cache decision run on the
// device; the host then waits for the plan (a few hundred bytes), because it
// has to issue one copy per streamed expert and size the grouped GEMMs:
//   compute: GEMMs on experts resident at the start  -> event A
//   copy:    per batch of streamed experts: [wait the GEMMs that last used the
//            staging half] [wait A before the first copy into a freed slot]
//            copies -> event C_j
//   compute: wait C_j -> GEMMs of batch j -> event G_j
//   copy:    newcomers nobody routed (wait A) -> event F; compute waits F
//   compute: unpermute (h += sum_r g Y)
// With a slot for every expert nothing is streamed, and the plan kernel also
// plans the GEMMs (one small-M tile per expert for small batches, the tall
// tile lists for large ones), so the host waits for nothing.
int prefill_enqueue(moe_cache *c, int layer, float *H, int T) {
  const PrefillLayout &p = c->play;
  uint8_t *base = c->prefill_ws;
  int32_t *ids = reinterpret_cast<int32_t *>(base + p.ids);
  float *g = reinterpret_cast<float *>(base + p.g);
  float *inv_r = reinterpret_cast<float *>(base + p.inv_r);
  uint16_t *xn = reinterpret_cast<uint16_t *>(base + p.xn);
  int32_t *perm = reinterpret_cast<int32_t *>(base + p.perm);
  int32_t *pos = reinterpret_cast<int32_t *>(base + p.pos);
  PrefillPlan *plan = reinterpret_cast<PrefillPlan *>(base + p.plan);
  GemmJob *jobs = reinterpret_cast<GemmJob *>(base + p.jobs);
  GemmTile *tiles = reinterpret_cast<GemmTile *>(base + p.tiles);
  uint16_t *act = reinterpret_cast<uint16_t *>(base + p.act);
  float *Y = reinterpret_cast<float *>(base + p.y);
  uint8_t *staging = base + p.staging;
  const uint8_t *host = c->host_layer[layer];
  uint8_t *arena = static_cast<uint8_t *>(c->desc.arena);
  const int gate_elem = c->dtype == MOE_DTYPE_BF16 ? 2 : 4;

  hipEvent_t tp;
  HIP_TRY(c, span_begin(c, c->cs, &tp, SPAN_PREFILL));
  PrefillArgs ga{};
  ga.gate = static_cast<const uint8_t *>(c->desc.gate_w) + (size_t)layer * c->E * c->d * gate_elem;
  ga.H = H;
  ga.ids = ids;
  ga.g = g;
  ga.inv_r = inv_r;
  ga.xn = xn;
  ga.T = T;
  ga.d = c->d;
  ga.E = c->E;
  ga.K = c->K;
  ga.dtype = c->dtype;
  HIP_TRY(c, launch_prefill_gate(ga, Launch{c->cs}));
  PlanArgs pa{};
  pa.ids = ids;
  pa.perm_tok = perm;
  pa.pos_of = pos;
  pa.plan = plan;
  pa.table = c->tables + layer;
  pa.stats = c->stats + layer;
  pa.trace = static_cast<TraceRec *>(c->desc.trace);
  pa.trace_in = c->trace_count + c->tpar;
  pa.trace_out = c->trace_count + (1 - c->tpar);
  pa.trace_cap = c->desc.trace ? c->desc.trace_cap : 0;
  pa.err = c->err;
  pa.expert_bytes = c->Bh;  // bytes one fetch moves (counters)
  pa.T = T;
  pa.K = c->K;
  pa.E = c->E;
  pa.S = c->S;
  pa.layer = layer;
  pa.policy = c->policy;
  pa.aging = c->policy == MOE_POLICY_LFU_AGED ? c->desc.aging_ticks : 0;
  // With a slot for every expert nothing is ever streamed, and with at most
  // kSkinnyRows tokens every expert's rows fit the small-M GEMMs: the plan
  // kernel then writes the GEMM jobs itself and the host does not wait for it.
  const bool device_plan = c->S == c->E && T <= kSkinnyRows;
  // A larger batch with a slot for every expert, when 256-row tiles give every
  // CU two tiles whatever the routing (the rule the host applies below picks
  // them then): the plan kernel writes both tile lists and the GEMMs read
  // their lengths, so the host waits for nothing.  The grids cover the longest
  // lists any routing can give.
  const int up_cols = prefill_tile_cols(true), down_cols = prefill_tile_cols(false);
  const int up_cb = (c->dff + up_cols - 1) / up_cols, dn_cb = (c->d + down_cols - 1) / down_cols;
  const long pairs = (long)T * c->K;
  const int tall_cap_rows = (int)((pairs + kTallRows - 1) / kTallRows) + c->E;  // bounds the sum of ceil(n_e / rows)
  const int up_cap = tall_cap_rows * up_cb, dn_cap = tall_cap_rows * dn_cb;
  const bool device_tall = c->S == c->E && !device_plan && (pairs / kTallRows) * std::min(up_cb, dn_cb) >= 2L * device_cus(c) &&
                           up_cap + dn_cap <= p.tile_cap;
  int32_t *dev_ntiles = reinterpret_cast<int32_t *>(base + p.ntiles);
  pa.jobs = device_plan || device_tall ? jobs : nullptr;
  pa.tiles = device_plan || device_tall ? tiles : nullptr;
  pa.ntiles = device_tall ? dev_ntiles : nullptr;
  pa.tile_rows = kTallRows;
  pa.up_cols = up_cols;
  pa.dn_cols = down_cols;
  pa.up_cb = up_cb;
  pa.dn_cb = dn_cb;
  pa.dn_first = up_cap;
  pa.up_cap = up_cap;
  pa.dn_cap = dn_cap;
  pa.arena_layer = arena + (size_t)layer * c->S * c->B;
  pa.slot_bytes = c->B;
  HIP_TRY(c, launch_prefill_plan(pa, Launch{c->cs}));
  c->tpar ^= 1;
  if (device_tall) {
    const double rows = (double)pairs;
    Launch lu, ld;
    HIP_TRY(c, kernel_span(c, c->cs, &lu, SPAN_GEMM_UP));
    HIP_TRY(c, launch_prefill_up(tiles, up_cap, jobs, xn, perm, act, c->d, c->dff, kTallRows, (size_t)c->max_T * c->d * 2, lu,
                                 dev_ntiles));
    kernel_span_done(c, SPAN_GEMM_UP, lu, rows * 4.0 * c->d * c->dff);
    HIP_TRY(c, kernel_span(c, c->cs, &ld, SPAN_GEMM_DOWN));
    HIP_TRY(c, launch_prefill_down(tiles + up_cap, dn_cap, jobs, act, Y, c->d, c->dff, kTallRows,
                                   (size_t)c->max_T * c->K * c->dff * 2, ld, dev_ntiles + 1));
    kernel_span_done(c, SPAN_GEMM_DOWN, ld, rows * 2.0 * c->d * c->dff);
    HIP_TRY(c, launch_prefill_unpermute(H, Y, g, pos, T, c->d, c->K, Launch{c->cs}));
    HIP_TRY(c, span_end(c, c->cs, SPAN_PREFILL, tp));
    c->last_route_kind = 2;
    c->last_prefill_T = T;
    return MOE_OK;  // routing errors surface at the next synchronising call
  }
  if (device_plan) {
    const double rows = (double)T * c->K;
    Launch lu, ld;
    HIP_TRY(c, kernel_span(c, c->cs, &lu, SPAN_GEMM_UP));
    HIP_TRY(c, launch_prefill_skinny_up(tiles, c->E, jobs, xn, perm, act, c->d, c->dff, T, lu));
    kernel_span_done(c, SPAN_GEMM_UP, lu, rows * 4.0 * c->d * c->dff);
    HIP_TRY(c, kernel_span(c, c->cs, &ld, SPAN_GEMM_DOWN));
    HIP_TRY(c, launch_prefill_skinny_down(tiles, c->E, jobs, act, Y, c->d, c->dff, T, ld));
    kernel_span_done(c, SPAN_GEMM_DOWN, ld, rows * 2.0 * c->d * c->dff);
    HIP_TRY(c, launch_prefill_unpermute(H, Y, g, pos, T, c->d, c->K, Launch{c->cs}));
    HIP_TRY(c, span_end(c, c->cs, SPAN_PREFILL, tp));
    c->last_route_kind = 2;
    c->last_prefill_T = T;
    return MOE_OK;  // routing errors surface at the next synchronising call
  }
  // one wait for both the plan and the error word (a second, synchronous
  // read of the word cost another round trip of about 30 us per layer)
  int32_t *h_err = reinterpret_cast<int32_t *>(c->h_plan + kMaxE);
  HIP_TRY(c, hipMemcpyAsync(c->h_plan, plan, sizeof(PrefillPlan) * c->E, hipMemcpyDeviceToHost, c->cs));
  HIP_TRY(c, hipMemcpyAsync(h_err, c->err, sizeof(int32_t), hipMemcpyDeviceToHost, c->cs));
  HIP_TRY(c, hipStreamSynchronize(c->cs));
  {
    const int32_t e = *h_err;
    if (e != ERR_NONE) {
      c->sticky = MOE_ERR_HIP;
      return fail(MOE_ERR_HIP, "prefill routing produced an invalid expert id (code %d)", e);
    }
  }
  c->last_route_kind = 2;
  c->last_prefill_T = T;

  // jobs: weights of every routed expert, where the GEMMs will find them
  const int E = c->E;
  const PrefillPlan *pl = c->h_plan;
  GemmJob *hj = reinterpret_cast<GemmJob *>(c->h_sched);
  GemmTile *ht = reinterpret_cast<GemmTile *>(c->h_sched + sizeof(GemmJob) * kMaxE);
  std::vector<int> resident, streamed, unrouted_new;
  for (int e = 0; e < E; ++e) {
    if (pl[e].n < 0 || pl[e].off < 0 || pl[e].off + pl[e].n > T * c->K || pl[e].slot_start >= c->S ||
        pl[e].slot_after >= c->S) {
      c->sticky = MOE_ERR_HIP;
      return fail(MOE_ERR_HIP, "inconsistent prefill plan from the device");
    }
    hj[e].w = nullptr;
    hj[e].row0 = pl[e].off;
    hj[e].nrows = pl[e].n;
    if (pl[e].n > 0 && pl[e].slot_start >= 0) {
      resident.push_back(e);
      hj[e].w = reinterpret_cast<const uint16_t *>(arena + ((size_t)layer * c->S + pl[e].slot_start) * c->B);
    } else if (pl[e].n == 0 && pl[e].newcomer) {
      unrouted_new.push_back(e);
    }
  }
  for (int pass = 0; pass < 2; ++pass)  // staging-bound experts first, then newcomers
    for (int e = 0; e < E; ++e)
      if (pl[e].n > 0 && pl[e].slot_start < 0 && (pl[e].slot_after >= 0) == (pass == 1)) streamed.push_back(e);

  const int half = p.ring / 2;
  std::vector<std::vector<int>> batches;
  for (size_t i = 0; i < streamed.size(); i += half)
    batches.emplace_back(streamed.begin() + i, streamed.begin() + std::min(streamed.size(), i + half));
  // staging slots and tile lists
  std::vector<int> ring_of(E, -1);
  for (size_t bi = 0; bi < batches.size(); ++bi) {
    int used = 0;
    for (int e : batches[bi]) {
      if (pl[e].slot_after >= 0) {
        hj[e].w = reinterpret_cast<const uint16_t *>(arena + ((size_t)layer * c->S + pl[e].slot_after) * c->B);
      } else {
        ring_of[e] = (int)(bi % 2) * half + used++;
        hj[e].w = reinterpret_cast<const uint16_t *>(staging + (size_t)ring_of[e] * c->B);
      }
    }
  }
  // Output tiles of 256, 128 or 64 rows (sorted pairs) by 128 (up) or 256
  // (down) columns: the
  // tallest that still gives every CU two tiles (256-row tiles run one
  // 512-lane workgroup per CU, the others two or three of 256 lanes).  Within
  // an expert the tiles of one column block are consecutive, so a column
  // block's weights are read once for all of the expert's row blocks by
  // workgroups that run at the same time on one XCD (the kernel hands each
  // XCD a contiguous stretch of this list).
  const int cus = device_cus(c);
  int nt = 0;
  bool overflow = false;  // checked before each write: ht is a fixed-size pinned buffer
  auto add_tiles = [&](const std::vector<int> &group, int ncols, int cols, int &first, int &count, int &rows) {
    auto tiles_of = [&](int r) {
      long n = 0;
      for (int e : group) n += (long)((pl[e].n + r - 1) / r) * ((ncols + cols - 1) / cols);
      return n;
    };
    rows = tiles_of(256) >= 2L * cus ? 256 : (tiles_of(128) >= 2L * cus ? 128 : 64);
    first = nt;
    for (int e : group)
      for (int n0 = 0; n0 < ncols; n0 += cols)
        for (int m0 = 0; m0 < pl[e].n; m0 += rows) {
          if (nt >= p.tile_cap) {
            overflow = true;
            continue;
          }
          ht[nt++] = GemmTile{e, m0, n0, 0};
        }
    count = nt - first;
  };
  const size_t ngroups = batches.size() + 1;
  std::vector<int> up_first(ngroups), up_n(ngroups), dn_first(ngroups), dn_n(ngroups), up_rows(ngroups),
      dn_rows(ngroups), skinny(ngroups, 0);
  std::vector<double> group_rows(ngroups, 0.0);
  // a group whose experts all have few rows (batched decode) goes to the
  // small-M kernels: one tile per expert, shared by the up and down launches
  auto add_group = [&](const std::vector<int> &group, size_t gi) {
    int most = 0;
    for (int e : group) {
      most = std::max(most, pl[e].n);
      group_rows[gi] += pl[e].n;
    }
    if (most <= kSkinnyRows) {
      skinny[gi] = std::max(most, 1);  // the group's largest row count
      up_first[gi] = dn_first[gi] = nt;
      for (int e : group) {
        if (nt >= p.tile_cap) {
          overflow = true;
          continue;
        }
        ht[nt++] = GemmTile{e, 0, 0, 0};
      }
      up_n[gi] = dn_n[gi] = nt - up_first[gi];
    } else {
      add_tiles(group, c->dff, up_cols, up_first[gi], up_n[gi], up_rows[gi]);
      add_tiles(group, c->d, down_cols, dn_first[gi], dn_n[gi], dn_rows[gi]);
    }
  };
  add_group(resident, 0);
  for (size_t bi = 0; bi < batches.size(); ++bi) add_group(batches[bi], bi + 1);
  if (overflow) {  // cannot happen: the capacity counts 64 x 64 tiles
    c->sticky = MOE_ERR_HIP;
    return fail(MOE_ERR_HIP, "prefill tile schedule overflow (capacity %d)", p.tile_cap);
  }
  // A coded host store's experts are copied to the coded staging area and
  // rebuilt from there by a kernel that reads a device-side fetch list: per
  // batch one list for experts bound to their new slots and one for experts
  // bound to the ring, then the unrouted newcomers in lists of up to `half`.
  const bool coded = coded_store(c->host_format);
  struct Part {
    int list = -1;
    bool ring = false;
    std::vector<int> experts;
  };
  std::vector<std::vector<Part>> batch_parts(batches.size());
  std::vector<Part> unrouted_parts;
  FetchList *hl = reinterpret_cast<FetchList *>(c->h_sched + sizeof(GemmJob) * kMaxE +
                                                sizeof(GemmTile) * (size_t)p.tile_cap);
  FetchList *dlists = reinterpret_cast<FetchList *>(base + p.lists);
  int nl = 0;
  auto add_part = [&](std::vector<Part> &parts, const std::vector<int> &ex, bool ring) {
    if (ex.empty()) return;
    if (nl >= kPrefillLists || (int)ex.size() > kMaxK) {  // cannot happen: at most 48 lists of <= 4 experts
      nl = kPrefillLists + 1;
      return;
    }
    Part pt;
    pt.list = nl++;
    pt.ring = ring;
    pt.experts = ex;
    FetchList &f = hl[pt.list];
    std::memset(&f, 0, sizeof f);
    f.n = (int)ex.size();
    f.layer = ring ? 0 : layer;
    for (size_t i = 0; i < ex.size(); ++i) {
      f.expert[i] = ex[i];
      f.slot[i] = ring ? ring_of[ex[i]] : pl[ex[i]].slot_after;
    }
    parts.push_back(pt);
  };
  if (coded) {
    for (size_t bi = 0; bi < batches.size(); ++bi) {
      std::vector<int> to_slot, to_ring;
      for (int e : batches[bi]) (pl[e].slot_after >= 0 ? to_slot : to_ring).push_back(e);
      add_part(batch_parts[bi], to_slot, false);
      add_part(batch_parts[bi], to_ring, true);
    }
    for (size_t i = 0; i < unrouted_new.size(); i += half)
      add_part(unrouted_parts,
               std::vector<int>(unrouted_new.begin() + i, unrouted_new.begin() + std::min(unrouted_new.size(), i + half)),
               false);
  }
  if (nl > kPrefillLists) {
    c->sticky = MOE_ERR_HIP;
    return fail(MOE_ERR_HIP, "prefill fetch-list overflow");
  }
  // the jobs and the tiles after them, in one copy: the two lie back to back
  // in the pinned schedule and in the workspace
  static_assert(sizeof(GemmJob) * kMaxE % 256 == 0, "tiles follow the jobs in the workspace");
  HIP_TRY(c, hipMemcpyAsync(jobs, hj, sizeof(GemmJob) * kMaxE + sizeof(GemmTile) * nt, hipMemcpyHostToDevice, c->cs));
  if (nl > 0) HIP_TRY(c, hipMemcpyAsync(dlists, hl, sizeof(FetchList) * nl, hipMemcpyHostToDevice, c->cs));

  const double up_flop_per_row = 4.0 * c->d * c->dff, down_flop_per_row = 2.0 * c->d * c->dff;
  auto run_group = [&](size_t gi) -> int {
    if (up_n[gi] <= 0) return MOE_OK;
    Launch lu, ld;
    HIP_TRY(c, kernel_span(c, c->cs, &lu, SPAN_GEMM_UP));
    if (skinny[gi])
      HIP_TRY(c, launch_prefill_skinny_up(tiles + up_first[gi], up_n[gi], jobs, xn, perm, act, c->d, c->dff,
                                            skinny[gi], lu));
    else
      HIP_TRY(c, launch_prefill_up(tiles + up_first[gi], up_n[gi], jobs, xn, perm, act, c->d, c->dff, up_rows[gi],
                                   (size_t)c->max_T * c->d * 2, lu));
    kernel_span_done(c, SPAN_GEMM_UP, lu, group_rows[gi] * up_flop_per_row);
    HIP_TRY(c, kernel_span(c, c->cs, &ld, SPAN_GEMM_DOWN));
    if (skinny[gi])
      HIP_TRY(c, launch_prefill_skinny_down(tiles + dn_first[gi], dn_n[gi], jobs, act, Y, c->d, c->dff, skinny[gi], ld));
    else
      HIP_TRY(c, launch_prefill_down(tiles + dn_first[gi], dn_n[gi], jobs, act, Y, c->d, c->dff, dn_rows[gi],
                                     (size_t)c->max_T * c->K * c->dff * 2, ld));
    kernel_span_done(c, SPAN_GEMM_DOWN, ld, group_rows[gi] * down_flop_per_row);
    return MOE_OK;
  };
  hipEvent_t evA = c->pf_ev[0], evF = c->pf_ev[1];
  if (!resident.empty()) {
    int rc = run_group(0);
    if (rc != MOE_OK) return rc;
  }
  HIP_TRY(c, hipEventRecord(evA, c->cs));  // also orders the schedule uploads before any copy
  hipStream_t q = c->xs;
  bool waited_A = false;
  uint8_t *coded_stage = base + p.coded;
  // copies (and, for a coded store, the rebuild) of one part of a batch
  auto stream_part = [&](const Part &pt) -> int {
    for (size_t i = 0; i < pt.experts.size(); ++i) {
      const int e = pt.experts[i];
      HIP_TRY(c, hipMemcpyAsync(coded_stage + i * c->Bh, host + (size_t)e * c->Bh, c->Bh, hipMemcpyHostToDevice, q));
    }
    Launch lr;
    HIP_TRY(c, kernel_span(c, q, &lr, SPAN_UNPACK));
    HIP_TRY(c, pt.ring ? launch_rebuild(c, dlists + pt.list, coded_stage, staging, 1, p.ring, half, lr)
                       : launch_rebuild(c, dlists + pt.list, coded_stage, arena, c->L, c->S, half, lr));
    kernel_span_done(c, SPAN_UNPACK, lr);
    return MOE_OK;
  };
  for (size_t bi = 0; bi < batches.size(); ++bi) {
    hipEvent_t evC = c->pf_ev[2 + 2 * (bi % kMaxE)], evG = c->pf_ev[3 + 2 * (bi % kMaxE)];
    bool waited_ring = false;
    for (int e : batches[bi]) {
      if (pl[e].slot_after >= 0) {
        if (!waited_A) {
          HIP_TRY(c, hipStreamWaitEvent(q, evA, 0));
          waited_A = true;
        }
      } else if (!waited_ring && bi >= 2) {
        HIP_TRY(c, hipStreamWaitEvent(q, c->pf_ev[3 + 2 * ((bi - 2) % kMaxE)], 0));
        waited_ring = true;
      }
      if (coded) continue;  // streamed part by part below
      uint8_t *dst = pl[e].slot_after >= 0 ? arena + ((size_t)layer * c->S + pl[e].slot_after) * c->B
                                           : staging + (size_t)ring_of[e] * c->B;
      HIP_TRY(c, hipMemcpyAsync(dst, host + (size_t)e * c->B, c->B, hipMemcpyHostToDevice, q));
    }
    if (coded && !waited_A) {  // the lists were uploaded before event A
      HIP_TRY(c, hipStreamWaitEvent(q, evA, 0));
      waited_A = true;
    }
    for (const Part &pt : batch_parts[bi]) {
      int rc = stream_part(pt);
      if (rc != MOE_OK) return rc;
    }
    HIP_TRY(c, hipEventRecord(evC, q));
    HIP_TRY(c, hipStreamWaitEvent(c->cs, evC, 0));
    int rc = run_group(bi + 1);
    if (rc != MOE_OK) return rc;
    HIP_TRY(c, hipEventRecord(evG, c->cs));
  }
  if (!unrouted_new.empty()) {
    if (!waited_A) HIP_TRY(c, hipStreamWaitEvent(q, evA, 0));
    if (coded) {
      for (const Part &pt : unrouted_parts) {
        int rc = stream_part(pt);
        if (rc != MOE_OK) return rc;
      }
    } else {
      for (int e : unrouted_new)
        HIP_TRY(c, hipMemcpyAsync(arena + ((size_t)layer * c->S + pl[e].slot_after) * c->B,
                                  host + (size_t)e * c->B, c->B, hipMemcpyHostToDevice, q));
    }
  }
  if (!batches.empty() || !unrouted_new.empty()) {  // copies were issued on the copy stream
    HIP_TRY(c, hipEventRecord(evF, q));
    HIP_TRY(c, hipStreamWaitEvent(c->cs, evF, 0));
  }
  HIP_TRY(c, launch_prefill_unpermute(H, Y, g, pos, T, c->d, c->K, Launch{c->cs}));
  HIP_TRY(c, span_end(c, c->cs, SPAN_PREFILL, tp));
  // later decode calls on this layer need no extra wait: the compute stream
  // has already waited for every copy issued here
  return MOE_OK;
}

int prefill_routing(moe_cache *c, int32_t *ids, float *g, size_t cap, size_t *n) {
  const size_t P = (size_t)c->last_prefill_T * c->K;
  const size_t m = P < cap ? P : cap;
  if (ids && m) HIP_TRY(c, hipMemcpy(ids, c->prefill_ws + c->play.ids, m * 4, hipMemcpyDeviceToHost));
  if (g && m) HIP_TRY(c, hipMemcpy(g, c->prefill_ws + c->play.g, m * 4, hipMemcpyDeviceToHost));
  *n = P;
  return MOE_OK;
}

}  // namespace moe

namespace {
// Milliseconds between events recorded around `reps` calls of launch() on s,
// after one untimed call.  The events come from the process pool.
template <class F>
int time_launches(hipStream_t s, int reps, F launch, const char *what, float *ms) {
  int dev = 0;
  HIP_TRY0(hipGetDevice(&dev));
  hipEvent_t a = nullptr, b = nullptr;
  HIP_TRY0(pool_event(dev, true, &a));
  hipError_t e = pool_event(dev, true, &b);
  if (e == hipSuccess) e = launch();  // warm-up
  if (e == hipSuccess) e = hipEventRecord(a, s);
  for (int r = 0; r < reps && e == hipSuccess; ++r) e = launch();
  if (e == hipSuccess) e = hipEventRecord(b, s);
  if (e == hipSuccess) e = hipEventSynchronize(b);
  if (e == hipSuccess) e = hipEventElapsedTime(ms, a, b);
  pool_give_back(dev, {}, {a, b}, nullptr, {});
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(MOE_ERR_HIP, "%s failed: %s", what, hipGetErrorString(e));
  }
  return MOE_OK;
}

}  // namespace

extern "C" {

int moe_decode_layer(moe_cache_t *c, int layer, float *h, int flags) {
  int rc = check_ready(c);
  if (rc != MOE_OK) return rc;
  if (layer < 0 || layer >= c->L) return fail(MOE_ERR_ARG, "layer %d out of range [0, %d)", layer, c->L);
  if (!h || misaligned(h, 16)) return fail(MOE_ERR_ARG, "h must be a non-NULL 16-byte aligned device pointer");
  if (flags & ~MOE_PREFETCH_NEXT) return fail(MOE_ERR_ARG, "unknown flags 0x%x", flags);
  const int spec = (flags & MOE_PREFETCH_NEXT) && layer + 1 < c->L ? layer + 1 : -1;
  return enqueue_layer(c, layer, h, nullptr, 1, spec, c->pmax, true, workspace_scratch(c));
}

int moe_decode_layer_noalloc(moe_cache_t *c, int layer, float *h, int flags) {
  if (!c) return fail(MOE_ERR_ARG, "NULL handle");
  if (!c->bound || !c->scratch) return fail(MOE_ERR_STATE, "handle is not bound (call moe_cache_bind)");
  const size_t act_bytes = align_up(sizeof(float) * (size_t)c->K * c->dff, 256);
  const size_t part_bytes = align_up(sizeof(float) * (size_t)ffn_down_chunks(c->K, c->dff, c->dtype) * c->d, 256);
  if (act_bytes + part_bytes > kNoAllocScratchBytes)
    return fail(MOE_ERR_ARG,
                "this model needs %zu bytes of decode scratch (top_k * d_ff activations, partial sums of d_model "
                "rows); the static scratch of moe_decode_layer_noalloc holds %zu: use moe_decode_layer",
                act_bytes + part_bytes, kNoAllocScratchBytes);
  int rc = check_ready(c);
  if (rc != MOE_OK) return rc;
  if (c->timing != MOE_TIMING_OFF)
    return fail(MOE_ERR_STATE, "kernel timing creates events; turn it off (moe_cache_set_timing) for this call");
  if (layer < 0 || layer >= c->L) return fail(MOE_ERR_ARG, "layer %d out of range [0, %d)", layer, c->L);
  if (!h || misaligned(h, 16)) return fail(MOE_ERR_ARG, "h must be a non-NULL 16-byte aligned device pointer");
  if (flags & ~MOE_PREFETCH_NEXT) return fail(MOE_ERR_ARG, "unknown flags 0x%x", flags);
  const int spec = (flags & MOE_PREFETCH_NEXT) && layer + 1 < c->L ? layer + 1 : -1;
  const CallScratch scr{reinterpret_cast<float *>(c->scratch), reinterpret_cast<float *>(c->scratch + act_bytes)};
  return enqueue_layer(c, layer, h, nullptr, 1, spec, c->pmax, true, scr);
}

int moe_prefetch(moe_cache_t *c, int next_layer, const float *h, int max_experts) {
  int rc = check_ready(c);
  if (rc != MOE_OK) return rc;
  if (next_layer <= 0 || next_layer >= c->L)
    return fail(MOE_ERR_ARG, "next_layer %d out of range [1, %d)", next_layer, c->L);
  if (!h || misaligned(h, 16)) return fail(MOE_ERR_ARG, "h must be a non-NULL 16-byte aligned device pointer");
  if (max_experts < 0 || max_experts > c->K) return fail(MOE_ERR_ARG, "max_experts must be in [0, top_k]");
  return enqueue_layer(c, next_layer - 1, const_cast<float *>(h), nullptr, 0, next_layer, max_experts, false,
                       workspace_scratch(c));
}

int moe_cache_access(moe_cache_t *c, int layer, const int *ids) {
  int rc = check_ready(c);
  if (rc != MOE_OK) return rc;
  if (layer < 0 || layer >= c->L) return fail(MOE_ERR_ARG, "layer %d out of range [0, %d)", layer, c->L);
  if (!ids) return fail(MOE_ERR_ARG, "ids is NULL");
  return enqueue_layer(c, layer, nullptr, reinterpret_cast<const int32_t *>(ids), 1, -1, 0, false,
                       workspace_scratch(c));
}

int moe_prefill_layer(moe_cache_t *c, int layer, float *H, int tokens) {
  int rc = check_ready(c);
  if (rc != MOE_OK) return rc;
  if (layer < 0 || layer >= c->L) return fail(MOE_ERR_ARG, "layer %d out of range [0, %d)", layer, c->L);
  if (!H || misaligned(H, 16)) return fail(MOE_ERR_ARG, "H must be a non-NULL 16-byte aligned device pointer");
  if (tokens <= 0 || tokens > c->max_T)
    return fail(MOE_ERR_ARG, "tokens must be in [1, max_prefill_tokens=%d]", c->max_T);
  return prefill_enqueue(c, layer, H, tokens);
}

int moe_cache_sync(moe_cache_t *c) {
  if (!c) return fail(MOE_ERR_ARG, "NULL handle");
  if (!c->bound) return fail(MOE_ERR_STATE, "handle is not bound");
  hipError_t e1 = hipStreamSynchronize(c->cs);
  hipError_t e2 = c->one_stream ? hipSuccess : hipStreamSynchronize(c->xs);
  if (e1 != hipSuccess || e2 != hipSuccess) {
    c->sticky = MOE_ERR_HIP;
    return fail(MOE_ERR_HIP, "stream synchronize failed: %s",
                hipGetErrorString(e1 != hipSuccess ? e1 : e2));
  }
  if (c->sticky == MOE_ERR_STATE) return fail(MOE_ERR_STATE, "handle needs moe_cache_reset");
  if (c->sticky != MOE_OK) return fail(c->sticky, "an earlier device error is pending");
  int32_t e = 0;
  HIP_TRY(c, hipMemcpy(&e, c->err, sizeof e, hipMemcpyDeviceToHost));
  if (e == ERR_BAD_IDS) {
    const int32_t zero = 0;
    HIP_TRY(c, hipMemcpy(c->err, &zero, sizeof zero, hipMemcpyHostToDevice));
    return fail(MOE_ERR_ARG, "injected expert ids were invalid (out of range or repeated); nothing changed");
  }
  if (e != ERR_NONE) {
    c->sticky = MOE_ERR_HIP;
    if (e == ERR_BAD_PACK)
      return fail(MOE_ERR_HIP, "coded host store is corrupt (an expert could not be rebuilt)");
    return fail(MOE_ERR_HIP, "device reported an inconsistent fetch list (code %d)", e);
  }
  return MOE_OK;
}

int moe_cache_stats(moe_cache_t *c, moe_layer_stats *out, int n_layers) {
  int rc = moe_cache_sync(c);
  if (rc != MOE_OK) return rc;
  if (!out || n_layers < 0 || n_layers > c->L) return fail(MOE_ERR_ARG, "bad output or n_layers");
  std::vector<LayerStats> s(c->L);
  HIP_TRY(c, hipMemcpy(s.data(), c->stats, sizeof(LayerStats) * c->L, hipMemcpyDeviceToHost));
  for (int l = 0; l < n_layers; ++l) {
    moe_layer_stats &o = out[l];
    o.hits = s[l].v[ST_HITS];
    o.misses = s[l].v[ST_MISSES];
    o.evictions = s[l].v[ST_EVICT];
    o.pf_guesses = s[l].v[ST_PF_GUESS];
    o.pf_issued = s[l].v[ST_PF_ISSUED];
    o.pf_useful = s[l].v[ST_PF_USEFUL];
    o.pf_wasted = s[l].v[ST_PF_WASTED];
    o.lookups = s[l].v[ST_LOOKUPS];
    o.bytes_fetched = s[l].v[ST_BYTES];
  }
  return MOE_OK;
}

int moe_cache_read_trace(moe_cache_t *c, moe_trace_rec *out, size_t cap, size_t *n, uint64_t *dropped) {
  int rc = moe_cache_sync(c);
  if (rc != MOE_OK) return rc;
  if (!n || (!out && cap)) return fail(MOE_ERR_ARG, "bad output pointers");
  *n = 0;
  if (dropped) *dropped = 0;
  if (!c->desc.trace) return MOE_OK;
  uint64_t total = 0;
  HIP_TRY(c, hipMemcpy(&total, c->trace_count + c->tpar, sizeof total, hipMemcpyDeviceToHost));
  const uint64_t ring = c->desc.trace_cap;
  const uint64_t avail = total < ring ? total : ring;
  const uint64_t start = total - avail;
  const uint64_t want = avail < cap ? avail : cap;
  const moe_trace_rec *dev = static_cast<const moe_trace_rec *>(c->desc.trace);
  uint64_t done = 0;
  while (done < want) {
    const uint64_t at = (start + done) % ring;
    uint64_t chunk = ring - at;
    if (chunk > want - done) chunk = want - done;
    HIP_TRY(c, hipMemcpy(out + done, dev + at, chunk * sizeof(moe_trace_rec), hipMemcpyDeviceToHost));
    done += chunk;
  }
  *n = (size_t)want;
  if (dropped) *dropped = start;
  return MOE_OK;
}

int moe_cache_read_state(moe_cache_t *c, int layer, int32_t *slot_expert, int32_t *expert_slot,
                         uint32_t *count, int64_t *last, int64_t *clock) {
  int rc = moe_cache_sync(c);
  if (rc != MOE_OK) return rc;
  if (layer < 0 || layer >= c->L) return fail(MOE_ERR_ARG, "layer out of range");
  LayerTable t;
  HIP_TRY(c, hipMemcpy(&t, c->tables + layer, sizeof t, hipMemcpyDeviceToHost));
  if (slot_expert) std::memcpy(slot_expert, t.slot_expert, sizeof(int32_t) * c->S);
  if (expert_slot) std::memcpy(expert_slot, t.expert_slot, sizeof(int32_t) * c->E);
  if (count) std::memcpy(count, t.count, sizeof(uint32_t) * c->E);
  if (last) std::memcpy(last, t.last, sizeof(int64_t) * c->E);
  if (clock) *clock = t.clock;
  return MOE_OK;
}

int moe_cache_last_routing(moe_cache_t *c, int32_t *ids, float *g, size_t cap, size_t *n) {
  int rc = moe_cache_sync(c);
  if (rc != MOE_OK) return rc;
  if (!n) return fail(MOE_ERR_ARG, "n is NULL");
  *n = 0;
  if (c->last_route_kind == 1) {
    RouteOut r;
    HIP_TRY(c, hipMemcpy(&r, c->route, sizeof r, hipMemcpyDeviceToHost));
    const size_t m = (size_t)c->K < cap ? (size_t)c->K : cap;
    if (ids) std::memcpy(ids, r.ids, m * sizeof(int32_t));
    if (g) std::memcpy(g, r.g, m * sizeof(float));
    *n = (size_t)c->K;
    return MOE_OK;
  }
  if (c->last_route_kind == 2) return prefill_routing(c, ids, g, cap, n);
  return MOE_OK;
}

int moe_cache_set_timing(moe_cache_t *c, int enable) {
  if (!c) return fail(MOE_ERR_ARG, "NULL handle");
  if (enable < MOE_TIMING_OFF || enable > MOE_TIMING_FFN_UP)
    return fail(MOE_ERR_ARG, "timing level must be MOE_TIMING_OFF, MOE_TIMING_ALL or MOE_TIMING_FFN_UP");
  c->timing = enable;
  return MOE_OK;
}

int moe_cache_read_timing(moe_cache_t *c, moe_timing *out) {
  if (!c || !out) return fail(MOE_ERR_ARG, "NULL argument");
  std::memset(out, 0, sizeof *out);
  if (!c->bound) return MOE_OK;
  (void)hipStreamSynchronize(c->cs);
  if (!c->one_stream) (void)hipStreamSynchronize(c->xs);
  double *ms[SPAN_KINDS] = {&out->router_ms,  &out->fetch_ms,     &out->ffn_up_ms,
                            &out->ffn_down_ms, &out->prefill_ms,   &out->gemm_up_ms,
                            &out->gemm_down_ms, &out->ffn_reduce_ms, &out->unpack_ms,
                            &out->wait_ms,     &out->pf_fetch_ms};
  uint64_t *n[SPAN_KINDS] = {&out->router_n,  &out->fetch_n,     &out->ffn_up_n,
                             &out->ffn_down_n, &out->prefill_n,   &out->gemm_up_n,
                             &out->gemm_down_n, &out->ffn_reduce_n, &out->unpack_n,
                             &out->wait_n,     &out->pf_fetch_n};
  int rc = MOE_OK;
  for (const auto &sp : c->spans) {
    float t = 0.0f;
    hipError_t e = hipEventElapsedTime(&t, sp.a, sp.b);
    if (e != hipSuccess && rc == MOE_OK)
      rc = fail(MOE_ERR_HIP, "hipEventElapsedTime failed: %s", hipGetErrorString(e));
    *ms[sp.kind] += t;
    *n[sp.kind] += 1;
    if (sp.kind == SPAN_GEMM_UP) out->gemm_up_flop += sp.flop;
    if (sp.kind == SPAN_GEMM_DOWN) out->gemm_down_flop += sp.flop;
    c->ev_pool.push_back(sp.a);
    c->ev_pool.push_back(sp.b);
  }
  c->spans.clear();
  return rc;
}

void moe_cache_destroy(moe_cache_t *c) {
  if (!c) return;
  for (const auto &sp : c->spans) {
    c->ev_pool.push_back(sp.a);
    c->ev_pool.push_back(sp.b);
  }
  if (c->pooled) {
    // drain every stream the handle enqueued on (its own side stream too),
    // then hand its runtime objects back to the process pool rather than
    // releasing them (see Pool)
    (void)hipStreamSynchronize(c->cs);
    if (!c->one_stream) (void)hipStreamSynchronize(c->xs);
    if (c->ms) (void)hipStreamSynchronize(c->ms);
    std::vector<hipEvent_t> sync_ev(c->ev_demand);
    sync_ev.insert(sync_ev.end(), c->ev_pf.begin(), c->ev_pf.end());
    sync_ev.insert(sync_ev.end(), c->pf_ev.begin(), c->pf_ev.end());
    sync_ev.push_back(c->ev_router);
    pool_give_back(c->dev, sync_ev, c->ev_pool, c->ms,
                   {{c->mirror_bytes, c->mirror}, {c->plan_bytes, c->h_plan}, {c->sched_bytes, c->h_sched}});
    (void)hipGetLastError();
  }
  delete c;
}

int moe_host_alloc(size_t bytes, void **out) {
  if (!out || bytes == 0) return fail(MOE_ERR_ARG, "bad arguments");
  *out = nullptr;
  hipError_t e = hipHostMalloc(out, bytes, hipHostMallocDefault);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    *out = nullptr;
    return fail(MOE_ERR_NOMEM, "hipHostMalloc(%zu) failed: %s", bytes, hipGetErrorString(e));
  }
  return MOE_OK;
}

int moe_host_free(void *p) {
  if (!p) return MOE_OK;
  // copies from the store may still be queued on caller streams: let every
  // one of them finish before the pages go
  hipError_t e = hipDeviceSynchronize();
  if (e != hipSuccess) return fail(MOE_ERR_HIP, "hipDeviceSynchronize before hipHostFree failed: %s", hipGetErrorString(e));
  e = hipHostFree(p);
  if (e != hipSuccess) return fail(MOE_ERR_HIP, "hipHostFree failed: %s", hipGetErrorString(e));
  return MOE_OK;
}

size_t moe_entropy_matrix_bytes(size_t n, size_t cap_words) { return entropy_matrix_bytes(n, cap_words); }

int moe_entropy_pack(const uint16_t *w, size_t n, size_t cap_words, void *out, size_t *used) {
  if (!w || !out || !used) return fail(MOE_ERR_ARG, "NULL pointer");
  const char *why = "";
  uint64_t u = 0;
  if (entropy_pack(w, n, cap_words, static_cast<uint8_t *>(out), &u, &why) != 0) return fail(MOE_ERR_ARG, "%s", why);
  *used = u;
  return MOE_OK;
}

int moe_probe_h2d_copy(const void *host_src, void *dev_dst, size_t bytes, int workgroups, int reps, void *stream,
                       double *gbps) {
  if (!host_src || !dev_dst || !gbps) return fail(MOE_ERR_ARG, "NULL pointer");
  if (misaligned(host_src, 16) || misaligned(dev_dst, 16) || bytes < 16 || bytes % 16)
    return fail(MOE_ERR_ARG, "buffers must be 16-byte aligned and bytes a positive multiple of 16");
  if (workgroups < 1 || workgroups > 4096) return fail(MOE_ERR_ARG, "workgroups must be in [1, 4096]");
  if (reps < 1 || reps > 1000) return fail(MOE_ERR_ARG, "reps must be in [1, 1000]");
  void *src = nullptr;
  hipError_t he = hipHostGetDevicePointer(&src, const_cast<void *>(host_src), 0);
  if (he != hipSuccess || !src) {
    (void)hipGetLastError();
    return fail(MOE_ERR_ARG, "host_src is not pinned host memory mapped for the device (%s)", hipGetErrorString(he));
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  float ms = 0.0f;
  int rc = time_launches(s, reps, [&] { return launch_h2d_copy_probe(src, dev_dst, bytes, workgroups, s); },
                         "host-to-device copy probe", &ms);
  if (rc != MOE_OK) return rc;
  *gbps = ms > 0.0f ? (double)bytes * reps / (ms * 1e-3) / 1e9 : 0.0;
  return MOE_OK;
}

int moe_probe_mfma_bf16(int shape, int iters, void *stream, double *tflops) {
  if (!tflops) return fail(MOE_ERR_ARG, "NULL pointer");
  if (shape != 0 && shape != 1) return fail(MOE_ERR_ARG, "shape must be 0 (16x16x32) or 1 (32x32x16)");
  if (iters < 1 || iters > (1 << 20)) return fail(MOE_ERR_ARG, "iters must be in [1, 2^20]");
  hipStream_t s = static_cast<hipStream_t>(stream);
  int dev = 0, cus = 0;
  HIP_TRY0(hipGetDevice(&dev));
  HIP_TRY0(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
  const int wgs = 8 * cus;  // 32 waves per compute unit, 8 per SIMD
  double flop = 0.0;
  float ms = 0.0f;
  int rc = time_launches(s, 1, [&] {
    flop = launch_mfma_bf16_probe(shape, wgs, iters, s);
    return hipGetLastError();
  }, "MFMA probe", &ms);
  if (rc != MOE_OK) return rc;
  *tflops = ms > 0.0f ? flop / (ms * 1e-3) / 1e12 : 0.0;
  return MOE_OK;
}

int moe_probe_hbm_read(const void *buf, size_t bytes, int reps, void *stream, double *gbps) {
  if (!buf || !gbps) return fail(MOE_ERR_ARG, "NULL pointer");
  if (misaligned(buf, 16) || bytes < 16 || bytes % 16)
    return fail(MOE_ERR_ARG, "buf must be 16-byte aligned and bytes a positive multiple of 16");
  if (reps < 1 || reps > 1000) return fail(MOE_ERR_ARG, "reps must be in [1, 1000]");
  hipStream_t s = static_cast<hipStream_t>(stream);
  int dev = 0, cus = 0;
  HIP_TRY0(hipGetDevice(&dev));
  HIP_TRY0(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
  float ms = 0.0f;
  int rc = time_launches(s, reps, [&] { return launch_hbm_read_probe(buf, bytes, cus, s); }, "HBM read probe", &ms);
  if (rc != MOE_OK) return rc;
  *gbps = ms > 0.0f ? (double)bytes * reps / (ms * 1e-3) / 1e9 : 0.0;
  return MOE_OK;
}

}  // extern "C"
