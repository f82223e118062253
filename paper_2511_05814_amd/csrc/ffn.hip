// Decode expert FFN (SwiGLU) over the experts resident in HBM slots.
//
// For a batch-1 token the K selected experts are matrix-vector products, so
// the work is bound by streaming the expert weights from HBM: 3 d d_ff
// elements per expert against 2 flops per element.  MFMA is no help here;
// the kernels are built for bandwidth instead:
//   * every lane issues 16-byte non-temporal loads (weights are read once per
//     token, so they are streamed past the caches);
//   * the activation a wave multiplies with stays in registers, and a wave
//     issues all of its weight loads for a row before the first FMA (in the
//     up kernel one row ahead), so each wave keeps several KB in flight;
//   * all K experts go into one launch.
//
//   up:   act_r = SiLU(W1_r x) * (W3_r x),  x = h / rms(h)      (per rank r)
//   down: h  += sum_r g_r W2_r act_r
//
// The down projection is split along its reduction axis (rank, column chunk)
// so that enough workgroups stream at once; each chunk writes a partial row
// sum and a small kernel adds the partials in a fixed order, so the result
// does not depend on scheduling.  Narrow experts (one chunk per rank) add the
// rank partials inside the down kernel, in the same order, instead.  Tile shapes were swept on MI355X at the
// Mixtral (d 4096, d_ff 14336) and 64-expert (d 2048, d_ff 1408) shapes.
#include "common.hpp"

namespace moe {
namespace {

constexpr int kThreads = 256;
constexpr int kWavesPerBlock = kThreads / kWave;
constexpr int kUpRows = 2;     // rows per wave (register path)
constexpr int kUpLdsRows = 1;  // row pairs per wave on the wide-model path
constexpr int kReduceThreads = 64;
constexpr int kFusedThreads = 512;  // fused down: eight waves, one rank each
#ifndef MOE_FFN_DOWN_FUSED_ROWS
#define MOE_FFN_DOWN_FUSED_ROWS 4
#endif
constexpr int kFusedRows = MOE_FFN_DOWN_FUSED_ROWS;  // rows of h per workgroup

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint4 load_stream(const void *p) {
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
  return make_uint4(v[0], v[1], v[2], v[3]);
}

// 16 bytes of weights -> fp32 values
template <int DT>
struct Elem;
template <>
struct Elem<0> {  // fp32
  using T = float;
  static constexpr int kVec = 4;
  __device__ static __forceinline__ void cvt(const uint4 v, float *f) {
    f[0] = __uint_as_float(v.x);
    f[1] = __uint_as_float(v.y);
    f[2] = __uint_as_float(v.z);
    f[3] = __uint_as_float(v.w);
  }
};
template <>
struct Elem<1> {  // bf16 stored as raw 16-bit patterns
  using T = uint16_t;
  static constexpr int kVec = 8;
  __device__ static __forceinline__ void cvt(const uint4 v, float *f) { bf16x8_to_f32(v, f); }
};

__device__ __forceinline__ float silu(float v) { return v / (1.0f + __expf(-v)); }

// Load V consecutive fp32 activations (scaled) or zeros past the end.
template <int V>
__device__ __forceinline__ void load_act(const float *p, bool ok, float scale, float *x) {
  if (ok) {
#pragma unroll
    for (int v = 0; v < V; v += 4) {
      const float4 t = *reinterpret_cast<const float4 *>(p + v);
      x[v] = t.x * scale;
      x[v + 1] = t.y * scale;
      x[v + 2] = t.z * scale;
      x[v + 3] = t.w * scale;
    }
  } else {
#pragma unroll
    for (int v = 0; v < V; ++v) x[v] = 0.0f;
  }
}

// Load this lane's STEPS x 16 bytes of row `row` (rows `stride` elements
// apart) of the matrix at mat.  Without RAGGED (every column below `cols`)
// the loads are unconditional; with it, columns from `cols` on read the
// matrix's first 16 bytes and the value is replaced by zeros.  Both forms are branch-free: guarded loads compile to
// exec-masked branches with a wait after each, and the zeroing selects make
// the compiler wait for the row before it issues the next one, so only
// ragged widths pay for them.
template <int DT, int STEPS, bool RAGGED>
__device__ __forceinline__ void load_row_strided(const typename Elem<DT>::T *mat, int row, int stride, int cols,
                                                 int lane, uint4 *u) {
  constexpr int V = Elem<DT>::kVec, COLS = kWave * V;
#pragma unroll
  for (int s = 0; s < STEPS; ++s) {
    const int c = s * COLS + lane * V;
    if (RAGGED) {
      const uint4 v = load_stream(c < cols ? mat + (size_t)row * stride + c : mat);
      u[s] = c < cols ? v : make_uint4(0, 0, 0, 0);
    } else {
      u[s] = load_stream(mat + (size_t)row * stride + c);
    }
  }
}

template <int DT, int STEPS, bool RAGGED>
__device__ __forceinline__ void load_row(const typename Elem<DT>::T *mat, int row, int d, int lane, uint4 *u) {
  load_row_strided<DT, STEPS, RAGGED>(mat, row, d, d, lane, u);
}

// V scaled activations per step, zeros past d (branch-free as load_row)
template <int V, int STEPS, bool RAGGED>
__device__ __forceinline__ void load_x(const float *h, int d, int lane, float scale, float (*x)[V]) {
  constexpr int COLS = kWave * V;
#pragma unroll
  for (int s = 0; s < STEPS; ++s) {
    const int c = s * COLS + lane * V;
    const bool ok = !RAGGED || c < d;
#pragma unroll
    for (int v = 0; v < V; v += 4) {
      const float4 t = *reinterpret_cast<const float4 *>(ok ? h + c + v : h);
      x[s][v] = ok ? t.x * scale : 0.0f;
      x[s][v + 1] = ok ? t.y * scale : 0.0f;
      x[s][v + 2] = ok ? t.z * scale : 0.0f;
      x[s][v + 3] = ok ? t.w * scale : 0.0f;
    }
  }
}

template <int DT, int STEPS>
__device__ __forceinline__ float row_dot(const uint4 *u, const float (*x)[Elem<DT>::kVec]) {
  constexpr int V = Elem<DT>::kVec;
  float acc = 0.0f;
#pragma unroll
  for (int s = 0; s < STEPS; ++s) {
    float f[V];
    Elem<DT>::cvt(u[s], f);
#pragma unroll
    for (int v = 0; v < V; ++v) acc = fmaf(f[v], x[s][v], acc);
  }
  return acc;
}

// up, activation in registers: d <= STEPS * 64 * V.  The waves of a
// workgroup work in pairs: the even wave of a pair streams RPW rows of W1,
// the odd wave the same rows of W3, each issuing the next row's loads before
// the current row's FMAs; the pair's two dot products per row meet in LDS.
// (One stream per wave, one row ahead, measured 3% faster on MI355X than a
// wave that streams a W1 and a W3 row together.)
template <int DT, int STEPS, int RPW, bool RAGGED>
__global__ __launch_bounds__(kThreads) void ffn_up_kernel(FfnArgs a) {
  using E = Elem<DT>;
  using T = typename E::T;
  constexpr int V = E::kVec;
  constexpr int kRows = kWavesPerBlock / 2 * RPW;  // rows per workgroup
  const int bpr = (a.d_ff + kRows - 1) / kRows;
  const int rank = blockIdx.x / bpr;
  const int rb = blockIdx.x - rank * bpr;
  if (rank >= a.route->k) return;
  const int slot = a.route->slot[rank];
  if (slot < 0 || slot >= a.S) return;
  const int d = a.d, d_ff = a.d_ff;
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  __shared__ float dots[kWavesPerBlock][RPW];

  float x[STEPS][V];
  load_x<V, STEPS, RAGGED>(a.h, d, lane, a.route->inv_r, x);
  // W3 follows W1 in the slot
  const T *w = reinterpret_cast<const T *>(a.arena + ((size_t)a.layer * a.S + slot) * a.expert_bytes) +
               (size_t)(wave & 1) * d_ff * d;
  const int base = rb * kRows;
  const int row0 = base + (wave >> 1) * RPW;
  // rows past d_ff (last workgroup of a rank) re-read the last row; their
  // results are not written
  // results are not written.  The scheduling barriers keep each row's loads
  // ahead of the previous row's FMAs (the scheduler would otherwise sink them).
  uint4 u[2][STEPS];
  load_row<DT, STEPS, RAGGED>(w, min(row0, d_ff - 1), d, lane, u[0]);
#pragma unroll
  for (int q = 0; q < RPW; ++q) {
    if (q + 1 < RPW) load_row<DT, STEPS, RAGGED>(w, min(row0 + q + 1, d_ff - 1), d, lane, u[(q + 1) & 1]);
    __builtin_amdgcn_sched_barrier(0);
    const float r = wave_sum(row_dot<DT, STEPS>(u[q & 1], x));
    if (lane == 0) dots[wave][q] = r;
  }
  __syncthreads();
  if (threadIdx.x < kRows && base + (int)threadIdx.x < d_ff) {
    const int pr = threadIdx.x / RPW, q = threadIdx.x - pr * RPW;
    a.act[(size_t)rank * d_ff + base + threadIdx.x] = silu(dots[2 * pr][q]) * dots[2 * pr + 1][q];
  }
}

// up for wide models (d beyond the register path): x staged in LDS
template <int DT, int RPW>
__global__ __launch_bounds__(kThreads) void ffn_up_lds_kernel(FfnArgs a) {
  using E = Elem<DT>;
  using T = typename E::T;
  constexpr int V = E::kVec;
  constexpr int kRowsPerBlock = kWavesPerBlock * RPW;
  extern __shared__ float xs[];
  const int bpr = (a.d_ff + kRowsPerBlock - 1) / kRowsPerBlock;
  const int rank = blockIdx.x / bpr;
  const int rb = blockIdx.x - rank * bpr;
  if (rank >= a.route->k) return;
  const int slot = a.route->slot[rank];
  if (slot < 0 || slot >= a.S) return;

  const int d = a.d, d_ff = a.d_ff;
  const float inv_r = a.route->inv_r;
  for (int i = threadIdx.x; i < d; i += kThreads) xs[i] = a.h[i] * inv_r;
  __syncthreads();

  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  const T *w1 = reinterpret_cast<const T *>(a.arena + ((size_t)a.layer * a.S + slot) * a.expert_bytes);
  const T *w3 = w1 + (size_t)d_ff * d;
  const int row0 = rb * kRowsPerBlock + wave * RPW;
  int nrows = d_ff - row0;
  nrows = nrows < 0 ? 0 : (nrows > RPW ? RPW : nrows);

  float acc1[RPW] = {}, acc3[RPW] = {};
  for (int c = lane * V; c < d; c += kWave * V) {
    float x[V];
    load_act<V>(xs + c, true, 1.0f, x);
#pragma unroll
    for (int q = 0; q < RPW; ++q) {
      if (q < nrows) {
        float f1[V], f3[V];
        E::cvt(load_stream(w1 + (size_t)(row0 + q) * d + c), f1);
        E::cvt(load_stream(w3 + (size_t)(row0 + q) * d + c), f3);
#pragma unroll
        for (int v = 0; v < V; ++v) {
          acc1[q] = fmaf(f1[v], x[v], acc1[q]);
          acc3[q] = fmaf(f3[v], x[v], acc3[q]);
        }
      }
    }
  }
#pragma unroll
  for (int q = 0; q < RPW; ++q) {
    const float s1 = wave_sum(acc1[q]);
    const float s3 = wave_sum(acc3[q]);
    if (lane == 0 && q < nrows) a.act[(size_t)rank * d_ff + row0 + q] = silu(s1) * s3;
  }
}

// down: one (row block, rank, column chunk) per workgroup; the chunk of
// g_r * act_r sits in registers; RPW rows of W2 per wave, all loads issued
// before the FMAs; writes one partial sum per row and chunk.  RAGGED: the
// last chunk of a rank runs past d_ff (those columns read zeros).
template <int DT, int STEPS, int RPW, bool RAGGED>
__global__ __launch_bounds__(kThreads) void ffn_down_kernel(FfnArgs a) {
  using E = Elem<DT>;
  using T = typename E::T;
  constexpr int V = E::kVec, COLS = kWave * V, CH = STEPS * COLS;
  const int d = a.d, d_ff = a.d_ff, K = a.route->k;
  const int cpr = (d_ff + CH - 1) / CH;
  const int nch = a.K * cpr;
  const int rb = blockIdx.x / nch;
  const int ch = blockIdx.x - rb * nch;
  const int rank = ch / cpr;
  const int c0 = (ch - rank * cpr) * CH;
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  const int row0 = rb * kWavesPerBlock * RPW + wave * RPW;

  const int slot = rank < K ? a.route->slot[rank] : -1;
  const bool valid = rank < K && slot >= 0 && slot < a.S;
  float acc[RPW] = {};
  if (valid) {
    float x[STEPS][V];
    load_x<V, STEPS, RAGGED>(a.act + (size_t)rank * d_ff + c0, d_ff - c0, lane, a.route->g[rank], x);
    // this chunk's columns of W2; rows past d re-read row d - 1 (not written)
    const T *w2 = reinterpret_cast<const T *>(a.arena + ((size_t)a.layer * a.S + slot) * a.expert_bytes) +
                  2 * (size_t)d_ff * d + c0;
    uint4 u[RPW][STEPS];
#pragma unroll
    for (int q = 0; q < RPW; ++q) load_row_strided<DT, STEPS, RAGGED>(w2, min(row0 + q, d - 1), d_ff, d_ff - c0, lane, u[q]);
#pragma unroll
    for (int q = 0; q < RPW; ++q) acc[q] = row_dot<DT, STEPS>(u[q], x);
  }
#pragma unroll
  for (int q = 0; q < RPW; ++q) {
    const float s = wave_sum(acc[q]);
    if (lane == 0 && row0 + q < d) a.part[(size_t)ch * d + row0 + q] = s;
  }
}

// down for narrow experts (each rank's row in one column chunk): the eight
// waves of a workgroup share its RPW rows of h, wave w taking ranks w, w + 8,
// ...; the rank partials meet in LDS and are added in rank order (the order
// the reduction below uses) and into h, so no partial-sum buffer and no
// second launch are needed.
template <int DT, int STEPS, int RPW, bool RAGGED>
__global__ __launch_bounds__(kFusedThreads) void ffn_down_fused_kernel(FfnArgs a) {
  using E = Elem<DT>;
  using T = typename E::T;
  constexpr int V = E::kVec, W = kFusedThreads / kWave;
  const int d = a.d, d_ff = a.d_ff, K = a.route->k;
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  const int row0 = blockIdx.x * RPW;
  __shared__ float dots[kMaxK][RPW];
  for (int rank = wave; rank < a.K; rank += W) {
    const int slot = rank < K ? a.route->slot[rank] : -1;
    const bool valid = rank < K && slot >= 0 && slot < a.S;
    float acc[RPW] = {};
    if (valid) {
      float x[STEPS][V];
      load_x<V, STEPS, RAGGED>(a.act + (size_t)rank * d_ff, d_ff, lane, a.route->g[rank], x);
      // rows past d re-read row d - 1 (not written)
      const T *w2 = reinterpret_cast<const T *>(a.arena + ((size_t)a.layer * a.S + slot) * a.expert_bytes) +
                    2 * (size_t)d_ff * d;
      uint4 u[RPW][STEPS];
#pragma unroll
      for (int q = 0; q < RPW; ++q) load_row_strided<DT, STEPS, RAGGED>(w2, min(row0 + q, d - 1), d_ff, d_ff, lane, u[q]);
#pragma unroll
      for (int q = 0; q < RPW; ++q) acc[q] = row_dot<DT, STEPS>(u[q], x);
    }
#pragma unroll
    for (int q = 0; q < RPW; ++q) {
      const float s = wave_sum(acc[q]);
      if (lane == 0) dots[rank][q] = s;
    }
  }
  __syncthreads();
  if ((int)threadIdx.x < RPW && row0 + (int)threadIdx.x < d) {
    float sum = 0.0f;
    for (int r = 0; r < a.K; ++r) sum += dots[r][threadIdx.x];
    a.h[row0 + threadIdx.x] += sum;
  }
}

// h += sum over chunks of the partial row sums, in chunk order; the loads of
// eight chunks are issued together.
__global__ __launch_bounds__(kReduceThreads) void ffn_reduce_kernel(const float *__restrict__ part, int nch,
                                                                    int d, float *__restrict__ h) {
  const int j = blockIdx.x * kReduceThreads + threadIdx.x;
  if (j >= d) return;
  float sum = 0.0f;
  int c = 0;
  for (; c + 8 <= nch; c += 8) {
    float t[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) t[i] = part[(size_t)(c + i) * d + j];
#pragma unroll
    for (int i = 0; i < 8; ++i) sum += t[i];
  }
  for (; c < nch; ++c) sum += part[(size_t)c * d + j];
  h[j] += sum;
}

// Down tile: (column steps per chunk, rows per wave) for a given d_ff.
struct DownShape {
  int steps, rows;
};
DownShape down_shape(int d_ff, int dtype) {
  const int cols = kWave * (dtype == 1 ? 8 : 4);
  // narrow experts: one chunk per rank, as few padding columns as possible
  if (d_ff <= 4 * cols) return {(d_ff + cols - 1) / cols, 2};
  return {2, 2};
}

template <int DT, int STEPS, int RPW>
void launch_up_steps(bool ragged, const FfnArgs &a, const Launch &l) {
  constexpr int kRows = kWavesPerBlock / 2 * RPW;
  const dim3 grid(a.K * ((a.d_ff + kRows - 1) / kRows));
  if (ragged)
    MOE_LAUNCH((ffn_up_kernel<DT, STEPS, RPW, true>), grid, dim3(kThreads), 0, l, a);
  else
    MOE_LAUNCH((ffn_up_kernel<DT, STEPS, RPW, false>), grid, dim3(kThreads), 0, l, a);
}

// (four rows a wave at d <= 2048 measured no faster than two)
template <int DT, int STEPS>
void launch_up_rows(bool ragged, const FfnArgs &a, const Launch &l) {
  // rows of fewer than STEPS whole steps (d = 1536 in bf16 on the 4-step
  // kernel) take the ragged form, which reads zeros past d
  ragged = ragged || a.d != STEPS * kWave * Elem<DT>::kVec;
  launch_up_steps<DT, STEPS, kUpRows>(ragged, a, l);
}

template <int DT>
hipError_t launch_up_t(const FfnArgs &a, const Launch &l) {
  constexpr int COLS = kWave * Elem<DT>::kVec;
  const int steps = (a.d + COLS - 1) / COLS;
  const bool ragged = a.d % COLS != 0;
  if (steps <= 1)
    launch_up_rows<DT, 1>(ragged, a, l);
  else if (steps <= 2)
    launch_up_rows<DT, 2>(ragged, a, l);
  else if (steps <= 4)
    launch_up_rows<DT, 4>(ragged, a, l);
  else if (steps <= 8)
    launch_up_rows<DT, 8>(ragged, a, l);
  else {
    const dim3 g2(a.K * ((a.d_ff + kWavesPerBlock * kUpLdsRows - 1) / (kWavesPerBlock * kUpLdsRows)));
    MOE_LAUNCH((ffn_up_lds_kernel<DT, kUpLdsRows>), g2, dim3(kThreads), (uint32_t)(a.d * sizeof(float)), l, a);
  }
  return hipGetLastError();
}

template <int DT, int STEPS, int RPW>
void launch_down_shape(dim3 grid, bool ragged, const FfnArgs &a, const Launch &l) {
  if (ragged)
    MOE_LAUNCH((ffn_down_kernel<DT, STEPS, RPW, true>), grid, dim3(kThreads), 0, l, a);
  else
    MOE_LAUNCH((ffn_down_kernel<DT, STEPS, RPW, false>), grid, dim3(kThreads), 0, l, a);
}

template <int DT, int STEPS>
void launch_down_fused(bool ragged, const FfnArgs &a, const Launch &l) {
  const dim3 grid((a.d + kFusedRows - 1) / kFusedRows);
  if (ragged)
    MOE_LAUNCH((ffn_down_fused_kernel<DT, STEPS, kFusedRows, true>), grid, dim3(kFusedThreads), 0, l, a);
  else
    MOE_LAUNCH((ffn_down_fused_kernel<DT, STEPS, kFusedRows, false>), grid, dim3(kFusedThreads), 0, l, a);
}

#ifndef MOE_FFN_DOWN_FUSE
#define MOE_FFN_DOWN_FUSE 1
#endif

bool down_fused(int K, int d_ff, int dtype) {
  if (!MOE_FFN_DOWN_FUSE || (dtype != 0 && dtype != 1)) return false;
  const int cols = kWave * (dtype == 1 ? 8 : 4);
  return K <= kMaxK && d_ff <= 4 * cols;
}

template <int DT>
hipError_t launch_down_t(const FfnArgs &a, const Launch &l) {
  const DownShape sh = down_shape(a.d_ff, DT);
  if (down_fused(a.K, a.d_ff, DT)) {
    const bool ragged = a.d_ff % (sh.steps * kWave * Elem<DT>::kVec) != 0;
    switch (sh.steps) {
      case 1: launch_down_fused<DT, 1>(ragged, a, l); break;
      case 2: launch_down_fused<DT, 2>(ragged, a, l); break;
      case 3: launch_down_fused<DT, 3>(ragged, a, l); break;
      default: launch_down_fused<DT, 4>(ragged, a, l); break;
    }
    return hipGetLastError();
  }
  const int rows = kWavesPerBlock * sh.rows;
  const int ch = sh.steps * kWave * Elem<DT>::kVec;
  const dim3 grid(((a.d + rows - 1) / rows) * ffn_down_chunks(a.K, a.d_ff, DT));
  switch (sh.steps) {
    case 1: launch_down_shape<DT, 1, 2>(grid, a.d_ff % ch != 0, a, l); break;
    case 2: launch_down_shape<DT, 2, 2>(grid, a.d_ff % ch != 0, a, l); break;
    case 3: launch_down_shape<DT, 3, 2>(grid, a.d_ff % ch != 0, a, l); break;
    default: launch_down_shape<DT, 4, 2>(grid, a.d_ff % ch != 0, a, l); break;
  }
  return hipGetLastError();
}

}  // namespace

bool ffn_down_fused(int K, int d_ff, int dtype) { return down_fused(K, d_ff, dtype); }

int ffn_down_chunks(int K, int d_ff, int dtype) {
  if (dtype == 2) return ffnq_down_chunks(K, d_ff);
  const int ch = down_shape(d_ff, dtype).steps * kWave * (dtype == 1 ? 8 : 4);
  return K * ((d_ff + ch - 1) / ch);
}

hipError_t launch_ffn_up(const FfnArgs &a, int dtype, const Launch &l) {
  if (dtype == 2) return launch_ffnq_up(a, l);
  return dtype == 1 ? launch_up_t<1>(a, l) : launch_up_t<0>(a, l);
}

hipError_t launch_ffn_down(const FfnArgs &a, int dtype, const Launch &l) {
  if (dtype == 2) return launch_ffnq_down(a, l);
  return dtype == 1 ? launch_down_t<1>(a, l) : launch_down_t<0>(a, l);
}

hipError_t launch_ffn_reduce(const FfnArgs &a, int dtype, const Launch &l) {
  MOE_LAUNCH(ffn_reduce_kernel, dim3((a.d + kReduceThreads - 1) / kReduceThreads), dim3(kReduceThreads), 0, l,
             (const float *)a.part, ffn_down_chunks(a.K, a.d_ff, dtype), a.d, a.h);
  return hipGetLastError();
}

}  // namespace moe
