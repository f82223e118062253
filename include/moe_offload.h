/*
 * moe_offload.h - C ABI of the MI355X (gfx950) library for Mixture-of-Experts
 * decode under expert offloading.
 *
 * The operation (Sec. 2.2, Sec. 3, Sec. 4.2-4.3 of "In-Depth Analysis on
 * Caching and Pre-fetching in Mixture of Experts Offloading"):
 *   - every layer has a gate W_g [E x d] and E SwiGLU experts; a token's
 *     hidden state h is routed to the top-K experts of z = W_g h and the
 *     layer adds sum_r g_r FFN_{i_r}(h / rms(h)) to h (Sec. 2.2, Sec. 4.3);
 *   - all experts live in pinned host memory; each layer keeps S of them in
 *     HBM slots and loads a missing one on demand (Sec. 2.2, Sec. 3.1);
 *   - the resident set is managed with LRU (Sec. 3.1) or LFU (Sec. 4.2);
 *   - optionally, layer l+1's gate applied to layer l's hidden state guesses
 *     layer l+1's experts, which are then fetched early (Sec. 3.2, Sec. 4.3).
 *
 * Conventions
 *   - All functions return MOE_OK (0) or a negative MOE_ERR_* code; no C++
 *     exception or abort crosses this boundary.  moe_last_error() gives a
 *     thread-local message for the last failure on the calling thread.
 *   - Pointers marked "device" are HBM addresses; "pinned host" is memory
 *     from hipHostMalloc (or moe_host_alloc); "host" is ordinary memory.
 *   - The caller owns every buffer it passes (gates, host store, arena,
 *     workspace, trace, hidden states) and both streams; they must outlive
 *     the handle.  The library owns the handle and the runtime objects it
 *     uses (HIP events, a side stream, small pinned buffers); those come
 *     from a process-wide pool and go back to it when the handle is
 *     destroyed, and are released only when the process ends.  It never
 *     frees caller memory.
 *   - Decode, prefetch, prefill and access calls only enqueue work on the
 *     streams; errors found while enqueuing are returned at once.  Faults of
 *     device work are sticky: they are reported by the next synchronising
 *     call (sync, stats, read_trace, read_state, last_routing, reset) and
 *     every later call then fails with MOE_ERR_STATE until moe_cache_reset
 *     succeeds.
 *   - One handle is used from one host thread at a time.
 */
#ifndef MOE_OFFLOAD_H
#define MOE_OFFLOAD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct moe_cache moe_cache_t; /* opaque, library-owned */

/* Eviction policies.  LRU (Sec. 3.1) evicts the expert unused for longest;
 * LFU (Sec. 4.2) the one with the smallest usage count, ties by recency.
 * MOE_POLICY_LFU_AGED weighs popularity together with how long an expert has
 * gone unused (the combination Sec. 6.1 proposes): its key is the usage count
 * halved, rounding down, once per moe_model_desc.aging_ticks ticks of the
 * layer's lookup clock since the expert's last use, evaluated at the moment of
 * the choice (the stored count is not changed); ties by recency, then slot. */
enum { MOE_POLICY_LRU = 0, MOE_POLICY_LFU = 1, MOE_POLICY_LFU_AGED = 2 };
enum {
  MOE_DTYPE_F32 = 0,  /* fp32 gates and experts                                   */
  MOE_DTYPE_BF16 = 1, /* bf16 gates and experts                                   */
  MOE_DTYPE_Q2G16 = 2 /* bf16 gates; experts group-quantised as in the paper's
                         measured model (Sec. 5.1: 2-bit codes, groups of 16,
                         compressed zero points).  Each matrix [rows x cols] is
                         three planes back to back: codes [rows][cols/4] bytes
                         (column c in bits 2*(c%4) of byte c/4), fp16 scales
                         [rows][cols/16], uint8 zero codes [rows][cols/16]
                         (zero point = code/64); weight = (q - zero) * scale.
                         Requires d_model and d_ff multiples of 64 and
                         d_model <= 8192; decode only (no batched prefill).  */
};
enum { MOE_OK = 0, MOE_ERR_ARG = -1, MOE_ERR_STATE = -2, MOE_ERR_HIP = -3, MOE_ERR_NOMEM = -4 };
/* flags of moe_decode_layer */
enum { MOE_PREFETCH_NEXT = 1 };
/* how missed experts are copied from the pinned host store into HBM slots */
enum {
  MOE_FETCH_KERNEL = 0, /* a copy kernel on the copy stream reads the host store
                           directly; no host round trip per layer            */
  MOE_FETCH_DMA = 1,    /* the host waits for the routing decision, then issues
                           one runtime copy (hipMemcpyAsync) per missed expert */
  MOE_FETCH_SPLIT = 2   /* demand misses by the copy kernel (no host round
                           trip on the critical path); speculative prefetches
                           by runtime copies (hipMemcpyAsync), which do not
                           slow the FFN kernels that run meanwhile the way the
                           copy kernel's host reads do.  The host reads each
                           prefetch list back on a stream the library owns,
                           after enqueueing the layer's FFN.                  */
};

/* Layout of the pinned host store (moe_model_desc.host_format). */
enum {
  MOE_HOST_PLAIN = 0,  /* experts stored as dtype, exactly as in the HBM slots   */
  MOE_HOST_PACKED = 1, /* bf16 experts packed losslessly to ~12.25 bits a weight:
                          each of W1, W3, W2 (n = d_model * d_ff weights) is cut
                          into blocks of 8192 weights of 12560 bytes each:
                            16-byte header: uint32 first exception of the
                              block, uint32 exceptions in the block, 8 zeros;
                            8192 bytes (sign << 7) | mantissa per weight;
                            4096 bytes of 4-bit exponent offsets (low nibble
                              for even weights) below the group maximum;
                            256 bytes: largest exponent of each group of 32;
                          then the matrix's exceptions, uint32
                          ((index in block) << 8) | exponent, for every weight
                          whose offset would be 15 or more (stored offset 15);
                          the matrix is padded to a capacity of
                          blocks * 12560 + 4 * packed_cap bytes rounded up
                          to 16, and an expert is W1 | W3 | W2 at that stride.
                          Copies move the packed bytes; a kernel on the copy
                          stream rebuilds the identical bf16 expert in its slot.
                          Needs dtype bf16.                                   */
  MOE_HOST_ENTROPY = 2 /* bf16 experts with entropy-coded exponents, ~10.9 bits
                          a weight for N(0, sigma) weights: each of W1, W3, W2
                          (n = d_model * d_ff weights, n a multiple of 512) is
                            512 bytes: 256 uint16 decode entries
                              (length << 8) | exponent, indexed by the next 8
                              bits of a stream (0 where no code starts);
                            one uint32 per span of 32768 weights (the last
                              may be short), padded to 16 bytes: the span's
                              first word in the stream area;
                            n bytes (sign << 7) | mantissa, in weight order;
                            packed_cap uint32 words of streams: the exponent
                              of weight 32768 s + 512 j + 8 l + u (l < 64,
                              u < 8) is code 8 j + u of lane stream l of span
                              s; canonical prefix codes of at most 8 bits,
                              first bit in the lowest free bit; word k of lane
                              stream l sits at the span's first word + 64 k +
                              l, over as many rows as the span's longest lane
                              stream needs (shorter ones padded with zeros);
                          the matrix occupies moe_entropy_matrix_bytes(n,
                          packed_cap) bytes and an expert is W1 | W3 | W2 at
                          that stride.  moe_entropy_pack writes this layout.
                          Copies move the coded bytes; a kernel on the copy
                          stream rebuilds the identical bf16 expert in its slot.
                          Needs dtype bf16.                                   */
};

/* Limits of this build. */
#define MOE_MAX_EXPERTS 64
#define MOE_MAX_TOPK 16

typedef struct {
  int d_model;            /* hidden size d; multiple of 8                            */
  int d_ff;               /* expert inner size; multiple of 8                        */
  int top_k;              /* K experts per token, 1 <= K <= min(E, 16)               */
  int dtype;              /* MOE_DTYPE_* of gates and experts                        */
  int prefetch_max;       /* at most this many guesses fetched per layer, 0..K      */
  int fetch_mode;         /* MOE_FETCH_*                                             */
  int max_prefill_tokens; /* largest T passed to moe_prefill_layer (0: no prefill)   */
  int host_format;        /* MOE_HOST_*                                              */
  const void *gate_w;        /* device [L][E][d], dtype, row-major                     */
  const void *host_experts;  /* pinned host [L][E][W1|W3|W2]; W1, W3 [d_ff x d],
                                W2 [d x d_ff], each row-major (out x in), dtype (or
                                packed, see MOE_HOST_PACKED); 16-byte aligned (may
                                be NULL if host_layers is set)                      */
  void *arena;               /* device [L][S][W1|W3|W2], 16-byte aligned              */
  void *workspace;           /* device, >= moe_cache_workspace_bytes(), 256-aligned   */
  size_t workspace_bytes;
  void *trace;               /* device ring of moe_trace_rec, or NULL for no trace   */
  size_t trace_cap;          /* records in the ring                                  */
  void *compute_stream;      /* hipStream_t for router and FFN work (NULL: default)  */
  void *copy_stream;         /* hipStream_t for expert copies (NULL: compute stream) */
  const void *const *host_layers; /* host array of L pinned pointers, layer l's experts
                                     [E][W1|W3|W2] at host_layers[l]; when non-NULL it
                                     replaces host_experts, so a store can span several
                                     allocations (entries may repeat); 16-byte aligned */
  int packed_cap;            /* per matrix: MOE_HOST_PACKED exception entries,
                                MOE_HOST_ENTROPY stream words                        */
  int aging_ticks;           /* MOE_POLICY_LFU_AGED: ticks per halving, >= 1;
                                ignored by the other policies                     */
} moe_model_desc;

/* One trace record.  kind 0 (access): a token's lookup of one of its K
 * experts; flags bit0 hit, bit1 the hit was a prefetched expert's first use;
 * slot = slot used, victim = expert evicted (-1 on a hit).
 * kind 1 (prefetch): one next-layer guess; layer = the guessed layer; flags
 * bit0 already resident, bit1 fetched now; slot = its slot (-1 if neither),
 * victim = expert evicted (-1 if none).
 * kind 2 (prefill): one record per expert after a batched prefill; token =
 * first token of the batch, rank = tokens routed to the expert, flags bit0
 * resident before, bit1 resident after, bit2 bytes fetched for it; slot =
 * slot after (-1 if not resident), victim = expert it replaced (-1 if none).
 * token is the layer's lookup index (0 for the first token after reset). */
typedef struct {
  int32_t kind, token, layer, rank, expert, flags, slot, victim;
} moe_trace_rec;

typedef struct {
  uint64_t hits, misses, evictions;                   /* demand lookups           */
  uint64_t pf_guesses, pf_issued, pf_useful, pf_wasted; /* speculative prefetch   */
  uint64_t lookups;                                   /* tokens seen by the layer */
  uint64_t bytes_fetched;                             /* demand + prefetch bytes  */
} moe_layer_stats;

/* Create a handle for `layers` layers of `experts` experts with `slots` HBM
 * slots per layer, evicting by `policy` (Sec. 3.1 LRU, Sec. 4.2 LFU, Sec. 6.1
 * aged LFU; see MOE_POLICY_*).
 * MOE_ERR_ARG: layers < 1, experts < 1 or > 64, slots < 1 or > experts, bad
 * policy, out == NULL.  No GPU work. */
int moe_cache_create(int layers, int experts, int slots, int policy, moe_cache_t **out);

/* Device workspace the handle needs for this model description (bytes);
 * 0 if the description is invalid. */
size_t moe_cache_workspace_bytes(const moe_cache_t *c, const moe_model_desc *d);

/* Record buffers, shapes and streams; create events.  MOE_ERR_ARG for an
 * invalid description (see the field comments; also slots < top_k, a NULL
 * buffer, a small workspace, misaligned pointers).  Does not reset state:
 * call moe_cache_reset before the first decode. */
int moe_cache_bind(moe_cache_t *c, const moe_model_desc *d);

/* Warm start (synchronous): slot s of every layer holds expert s, counts 0,
 * clocks 0, statistics and trace cleared; experts 0..S-1 are copied into the
 * slots.  Clears a sticky error.  The paper does not say how its caches start;
 * this reading follows Table 2, whose cache recall is exactly twice its
 * precision for a cache of 4 experts and top-2 routing (Sec. 5.3): that holds
 * only if the cache is full from the first counted token, so the caches start
 * full rather than empty. */
int moe_cache_reset(moe_cache_t *c);

/* One token through one layer (Sec. 2.2): route h [d] (device fp32, updated
 * in place: h += sum_r g_r FFN_{i_r}(h / rms(h))), look the K experts up in the
 * layer's cache, fetch the misses from the host store, run the SwiGLU experts.
 * With MOE_PREFETCH_NEXT and layer + 1 < L, also guess layer+1's experts from
 * this h and fetch up to prefetch_max of them (Sec. 3.2).  Enqueue only. */
int moe_decode_layer(moe_cache_t *c, int layer, float *h, int flags);

/* moe_decode_layer for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc).  Same arguments, work and results as moe_decode_layer (the
 * same kernels), but the call's scratch (the FFN's top_k x d_ff activations
 * and its partial row sums of d_model rows) lives in a
 * static 4 MiB device array that the library holds on each device until the
 * process ends, instead of the bound workspace; the call allocates nothing
 * (no hipMalloc, no event creation).  Every call on one device shares that
 * array and it keeps the last call's contents (each call writes all of it
 * that it reads): calls that overlap on one device, from any handle, race.
 * MOE_ERR_ARG if the model needs more scratch than the array holds (the
 * message gives the size), MOE_ERR_STATE if kernel timing is on (timed
 * spans create events); otherwise as moe_decode_layer.  Enqueue only. */
int moe_decode_layer_noalloc(moe_cache_t *c, int layer, float *h, int flags);

/* The speculative part alone (Sec. 3.2, Sec. 4.3: each layer also holds the
 * next layer's gate, and that gate applied to the current hidden state,
 * followed by softmax and top-K, guesses the next layer's experts): guess
 * next_layer's experts from h (device fp32 [d], read only) with next_layer's
 * gate and fetch up to max_experts of them (0..K), evicting by the layer's
 * policy with all K guesses protected; an inserted guess takes one tick of
 * the layer's clock and does not count as a use.  MOE_ERR_ARG if next_layer
 * is 0 or >= L, or max_experts is outside 0..K.  Enqueue only. */
int moe_prefetch(moe_cache_t *c, int next_layer, const float *h, int max_experts);

/* Batched prefill.  The paper measures generated tokens only and says nothing
 * about the prompt (Sec. 5.1); this call is this library's reading: the batch
 * is routed and computed row by row exactly as decode tokens (Sec. 2.2, Sec.
 * 4.3), and the cache takes the batch's routing at once by the same policy
 * (Sec. 3.1 LRU, Sec. 4.2 LFU).
 * A batch of `tokens` rows H [tokens][d] (device fp32, in place) through one
 * layer: every row is routed and computed as a decode token would be; the
 * layer's cache takes the batch's routing at once (counts += per-expert
 * routings, the clock ticks once per (token, rank), then the S experts with the
 * largest key stay resident: LFU the count, aged LFU the aged count at the
 * batch's last tick, LRU the last use; ties: resident first, lower id).  Kept
 * experts keep their slots; newcomers take the freed slots.  tokens must be
 * in 1..max_prefill_tokens.  The host waits for the device's plan of the batch
 * (a few hundred bytes) before it issues the copies of streamed experts and
 * sizes the GEMMs; when every expert has a slot (slots == experts) and tokens
 * <= 32 the plan stays on the device and the call only enqueues, and a bad
 * routing then surfaces at the next synchronising call. */
int moe_prefill_layer(moe_cache_t *c, int layer, float *H, int tokens);

/* Injected routing (test hook): the cache lookup alone (Sec. 3.1: a selected
 * expert already in the layer's cache is reused, a missing one is loaded and
 * the least recently used one evicted; Sec. 4.2: LFU keeps a usage count per
 * expert and evicts the least frequently used).  Runs layer `layer`'s lookup,
 * fetches and trace for the K expert ids at `ids` (device int32 [K], rank
 * order, distinct, each in [0, E)), with no router and no FFN.  Invalid ids
 * are detected on the device, nothing is changed, and the next synchronising
 * call returns MOE_ERR_ARG. */
int moe_cache_access(moe_cache_t *c, int layer, const int *ids);

/* Wait for both streams; report sticky errors. */
int moe_cache_sync(moe_cache_t *c);

/* Per-layer statistics into out[0..n_layers) (host); n_layers <= L. Syncs. */
int moe_cache_stats(moe_cache_t *c, moe_layer_stats *out, int n_layers);

/* Copy the trace (oldest first) into out (host, cap records); *n = records
 * copied.  If more were recorded than the ring holds, the oldest are lost and
 * *dropped (if non-NULL) says how many.  Syncs. */
int moe_cache_read_trace(moe_cache_t *c, moe_trace_rec *out, size_t cap, size_t *n,
                         uint64_t *dropped);

/* One layer's table (host outputs, any may be NULL): slot_expert [S],
 * expert_slot [E] (-1 if not resident), count [E], last [E], clock. Syncs. */
int moe_cache_read_state(moe_cache_t *c, int layer, int32_t *slot_expert,
                         int32_t *expert_slot, uint32_t *count, int64_t *last,
                         int64_t *clock);

/* Routing of the last decode (K entries) or prefill (tokens * K entries,
 * token-major) on the compute stream: ids (host int32) and combine weights
 * g (host fp32), each up to cap entries; *n = entries available. Syncs. */
int moe_cache_last_routing(moe_cache_t *c, int32_t *ids, float *g, size_t cap, size_t *n);

typedef struct {
  double router_ms, fetch_ms, ffn_up_ms, ffn_down_ms, prefill_ms, gemm_up_ms, gemm_down_ms,
      ffn_reduce_ms;
  uint64_t router_n, fetch_n, ffn_up_n, ffn_down_n, prefill_n, gemm_up_n, gemm_down_n, ffn_reduce_n;
  double gemm_up_flop, gemm_down_flop; /* algorithmic flops of the timed GEMM launches */
  double unpack_ms;                    /* coded host stores: rebuilding copied experts */
  uint64_t unpack_n;
  double wait_ms;     /* decode: compute stream from each router's end to the FFN's start,
                         i.e. waiting for the copies that fill the layer's slots        */
  uint64_t wait_n;
  double pf_fetch_ms; /* speculative (next-layer) copies; fetch_ms counts demand copies */
  uint64_t pf_fetch_n;
} moe_timing;

/* Kernel timing with HIP events, off by default.  At MOE_TIMING_ALL every
 * router, fetch, decode FFN and prefill grouped-GEMM launch is bracketed by a
 * pair of events on the stream it runs on (prefill_ms spans a whole layer's
 * prefill on the compute stream, waits for streamed experts included; wait_ms
 * spans the compute stream's work between a decode router and its FFN: the
 * demand copies, or the wait for them).  The events cost GPU time as well
 * (about a third of the kernel time of a layer whose experts are all
 * resident), so MOE_TIMING_FFN_UP times only the decode FFN up launches and
 * leaves every other count at zero.  enable: one of the MOE_TIMING_* levels
 * (0 and 1 keep their boolean meaning); MOE_ERR_ARG otherwise.
 * moe_cache_read_timing syncs, returns the summed durations (ms), launch
 * counts and GEMM flops since the previous read, and clears them. */
enum { MOE_TIMING_OFF = 0, MOE_TIMING_ALL = 1, MOE_TIMING_FFN_UP = 2 };
int moe_cache_set_timing(moe_cache_t *c, int enable);
int moe_cache_read_timing(moe_cache_t *c, moe_timing *out);

/* Drain every stream the handle enqueued on, return its events, side stream
 * and pinned buffers to the process pool, free the handle; NULL-safe. */
void moe_cache_destroy(moe_cache_t *c);

/* Pinned host memory for the expert store (hipHostMalloc); *out is usable
 * from both host and device.  moe_host_free waits for all work on the current
 * device (copies from the store may still be queued) before it frees;
 * moe_host_free(NULL) is a no-op. */
int moe_host_alloc(size_t bytes, void **out);
int moe_host_free(void *p);

/* Bytes one matrix of n weights occupies in a MOE_HOST_ENTROPY store whose
 * lane streams have room for cap_words words (the layout is described at
 * MOE_HOST_ENTROPY); 0 if n is 0 or not a multiple of 512. */
size_t moe_entropy_matrix_bytes(size_t n, size_t cap_words);

/* Encode one matrix of n bf16 weights (host memory, row-major bit patterns)
 * into the MOE_HOST_ENTROPY layout at out (host memory of
 * moe_entropy_matrix_bytes(n, cap_words) bytes, e.g. inside a pinned store),
 * with prefix codes built from this matrix's exponent counts (optimal among
 * codes of at most 8 bits).  *used receives the stream words the matrix
 * needs.  MOE_ERR_ARG: NULL pointers, n not a positive multiple of 512, or
 * the streams need more than cap_words words (out is then unspecified).
 * Host-only, no GPU work; different matrices may be encoded from different
 * threads at once. */
int moe_entropy_pack(const uint16_t *w, size_t n, size_t cap_words, void *out, size_t *used);

/* Calibration, not part of the decode path: the read bandwidth (GB/s) a
 * plain streaming kernel reaches on the current device, a practical ceiling
 * for the HBM-bound kernels above (the published peak is not reachable).
 * Reads `bytes` (a positive multiple of 16) of device memory at buf (16-byte
 * aligned, not written) `reps` times (1..1000) on `stream` (a hipStream_t,
 * NULL = the default stream) after one untimed pass, with one workgroup per
 * compute unit streaming 16-byte non-temporal loads; *gbps = bytes * reps
 * over the time between events recorded around the timed passes.
 * Synchronous.  MOE_ERR_ARG for bad arguments, MOE_ERR_HIP for runtime
 * failures.  Use a buffer well above the 256 MB last-level cache. */
int moe_probe_hbm_read(const void *buf, size_t bytes, int reps, void *stream, double *gbps);

/* Calibration, not part of the decode path: the host-to-device rate (GB/s)
 * of a shader copy with the fetch kernel's access pattern (16-byte loads from
 * mapped pinned host memory, four in flight a lane, `workgroups` workgroups
 * of 256 lanes, 1..4096), the other way besides the DMA engines that experts
 * reach HBM (Sec. 2.2: experts are loaded into GPU memory on demand).  Copies
 * `bytes` (a positive multiple of 16) from host_src (pinned host memory from
 * hipHostMalloc / moe_host_alloc, mapped for the device, 16-byte aligned) to
 * dev_dst (device, 16-byte aligned) `reps` times (1..1000) on `stream` after
 * one untimed copy; *gbps = bytes * reps over the time between events
 * recorded around the timed copies.  Synchronous.  MOE_ERR_ARG for bad
 * arguments or a host buffer the device cannot address, MOE_ERR_HIP for
 * runtime failures. */
int moe_probe_h2d_copy(const void *host_src, void *dev_dst, size_t bytes, int workgroups, int reps,
                       void *stream, double *gbps);

/* Calibration, not part of the decode path: the bf16 matrix-core rate
 * (TFLOP/s) of a kernel that does nothing but issue MFMA instructions on
 * register operands (four independent accumulations per wave, 32 waves per
 * compute unit), the practical ceiling of the batched prefill's grouped GEMMs
 * (Sec. 2.1: the experts of a batch are dense products).  shape 0:
 * v_mfma_f32_16x16x32_bf16 (the grouped GEMMs' instruction), 1:
 * v_mfma_f32_32x32x16_bf16; `iters` (1..2^20) instructions per accumulation.
 * One untimed launch, then one timed launch on `stream`.  Synchronous.
 * MOE_ERR_ARG for bad arguments, MOE_ERR_HIP for runtime failures. */
int moe_probe_mfma_bf16(int shape, int iters, void *stream, double *tflops);

/* Thread-local message of the last failure on this thread ("" if none). */
const char *moe_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* MOE_OFFLOAD_H */
