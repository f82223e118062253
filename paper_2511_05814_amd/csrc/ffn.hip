// Decode expert FFN (SwiGLU) over the experts resident in HBM slots.
//
// For a batch-1 token the K selected experts are matrix-vector products, so
// the work is bound by streaming the expert weights from HBM: 3 d d_ff
// elements per expert against 2 flops per element.  MFMA is no help here;
// the kernels are built for bandwidth instead:
//   * every lane issues 16-byte non-temporal loads (weights are read once per
//     token, so they are streamed past the caches);
//   * the activation a wave multiplies with stays in registers, and a wave
//     issues all of its weight loads for a row before the first FMA, so each
//     wave keeps several KB in flight without LDS round trips or barriers;
//   * all K experts go into one launch.
//
//   up:   act_r = SiLU(W1_r x) * (W3_r x),  x = h / rms(h)      (per rank r)
//   down: h  += sum_r g_r W2_r act_r
//
// The down projection is split along its reduction axis (rank, column chunk)
// so that enough workgroups stream at once; each chunk writes a partial row
// sum and a small kernel adds the partials in a fixed order, so the result
// does not depend on scheduling.  Tile shapes were swept on MI355X at the
// Mixtral (d 4096, d_ff 14336) and 64-expert (d 2048, d_ff 1408) shapes.
#include "common.hpp"

namespace moe {
namespace {

constexpr int kThreads = 256;
constexpr int kWavesPerBlock = kThreads / kWave;
constexpr int kUpRows = 2;     // W1/W3 row pairs per wave (register path)
constexpr int kUpLdsRows = 1;  // row pairs per wave on the wide-model path

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

// up, activation in registers: d <= STEPS * 64 * V
template <int DT, int STEPS, int RPW>
__global__ __launch_bounds__(kThreads) void ffn_up_kernel(FfnArgs a) {
  using E = Elem<DT>;
  using T = typename E::T;
  constexpr int V = E::kVec, COLS = kWave * V;
  const int bpr = (a.d_ff + kWavesPerBlock * RPW - 1) / (kWavesPerBlock * RPW);
  const int rank = blockIdx.x / bpr;
  const int rb = blockIdx.x - rank * bpr;
  if (rank >= a.route->k) return;
  const int hit = a.route->hit[rank];
  if ((a.phase == 1 && !hit) || (a.phase == 2 && hit)) return;
  const int slot = a.route->slot[rank];
  if (slot < 0 || slot >= a.S) return;
  const int d = a.d, d_ff = a.d_ff;
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  const float inv_r = a.route->inv_r;

  float x[STEPS][V];
#pragma unroll
  for (int s = 0; s < STEPS; ++s) {
    const int c = s * COLS + lane * V;
    load_act<V>(a.h + c, c < d, inv_r, x[s]);
  }
  const T *w1 = reinterpret_cast<const T *>(a.arena + ((size_t)a.layer * a.S + slot) * a.expert_bytes);
  const T *w3 = w1 + (size_t)d_ff * d;
  const int row0 = rb * kWavesPerBlock * RPW + wave * RPW;
  for (int q = 0; q < RPW; ++q) {
    const int row = row0 + q;
    if (row >= d_ff) break;
    const T *r1 = w1 + (size_t)row * d + lane * V;
    const T *r3 = w3 + (size_t)row * d + lane * V;
    uint4 u1[STEPS], u3[STEPS];
#pragma unroll
    for (int s = 0; s < STEPS; ++s) {
      if (s * COLS + lane * V < d) {
        u1[s] = load_stream(r1 + s * COLS);
        u3[s] = load_stream(r3 + s * COLS);
      } else {
        u1[s] = u3[s] = make_uint4(0, 0, 0, 0);
      }
    }
    float a1 = 0.0f, a3 = 0.0f;
#pragma unroll
    for (int s = 0; s < STEPS; ++s) {
      float f1[V], f3[V];
      E::cvt(u1[s], f1);
      E::cvt(u3[s], f3);
#pragma unroll
      for (int v = 0; v < V; ++v) {
        a1 = fmaf(f1[v], x[s][v], a1);
        a3 = fmaf(f3[v], x[s][v], a3);
      }
    }
    a1 = wave_sum(a1);
    a3 = wave_sum(a3);
    if (lane == 0) a.act[(size_t)rank * d_ff + row] = silu(a1) * a3;
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
  const int hit = a.route->hit[rank];
  if ((a.phase == 1 && !hit) || (a.phase == 2 && hit)) return;
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
// before the FMAs; writes one partial sum per row and chunk.
template <int DT, int STEPS, int RPW>
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
    const float g = a.route->g[rank];
    const float *act = a.act + (size_t)rank * d_ff;
    float x[STEPS][V];
#pragma unroll
    for (int s = 0; s < STEPS; ++s) {
      const int c = c0 + s * COLS + lane * V;
      load_act<V>(act + c, c < d_ff, g, x[s]);
    }
    const T *w2 = reinterpret_cast<const T *>(a.arena + ((size_t)a.layer * a.S + slot) * a.expert_bytes) +
                  2 * (size_t)d_ff * d;
    uint4 u[RPW][STEPS];
#pragma unroll
    for (int q = 0; q < RPW; ++q)
#pragma unroll
      for (int s = 0; s < STEPS; ++s) {
        const int c = c0 + s * COLS + lane * V;
        u[q][s] = (row0 + q < d && c < d_ff) ? load_stream(w2 + (size_t)(row0 + q) * d_ff + c)
                                             : make_uint4(0, 0, 0, 0);
      }
#pragma unroll
    for (int q = 0; q < RPW; ++q)
#pragma unroll
      for (int s = 0; s < STEPS; ++s) {
        float f[V];
        E::cvt(u[q][s], f);
#pragma unroll
        for (int v = 0; v < V; ++v) acc[q] = fmaf(f[v], x[s][v], acc[q]);
      }
  }
#pragma unroll
  for (int q = 0; q < RPW; ++q) {
    const float s = wave_sum(acc[q]);
    if (lane == 0 && row0 + q < d) a.part[(size_t)ch * d + row0 + q] = s;
  }
}

// h += sum over chunks of the partial row sums, in chunk order.
__global__ __launch_bounds__(kThreads) void ffn_reduce_kernel(const float *__restrict__ part, int nch,
                                                              int d, float *__restrict__ h) {
  const int j = blockIdx.x * kThreads + threadIdx.x;
  if (j >= d) return;
  float sum = 0.0f;
  for (int c = 0; c < nch; ++c) sum += part[(size_t)c * d + j];
  h[j] += sum;
}

// Down tile: (column steps per chunk, rows per wave) for a given d_ff.
struct DownShape {
  int steps, rows;
};
DownShape down_shape(int d_ff, int dtype) {
  const int cols = kWave * (dtype == 1 ? 8 : 4);
  if (d_ff <= 4 * cols) return {4, 2};
  return {2, 4};
}

template <int DT>
hipError_t launch_up_t(const FfnArgs &a, const Launch &l) {
  constexpr int COLS = kWave * Elem<DT>::kVec;
  const int steps = (a.d + COLS - 1) / COLS;
  const dim3 grid(a.K * ((a.d_ff + kWavesPerBlock * kUpRows - 1) / (kWavesPerBlock * kUpRows)));
  if (steps <= 1)
    MOE_LAUNCH((ffn_up_kernel<DT, 1, kUpRows>), grid, dim3(kThreads), 0, l, a);
  else if (steps <= 2)
    MOE_LAUNCH((ffn_up_kernel<DT, 2, kUpRows>), grid, dim3(kThreads), 0, l, a);
  else if (steps <= 4)
    MOE_LAUNCH((ffn_up_kernel<DT, 4, kUpRows>), grid, dim3(kThreads), 0, l, a);
  else if (steps <= 8)
    MOE_LAUNCH((ffn_up_kernel<DT, 8, kUpRows>), grid, dim3(kThreads), 0, l, a);
  else {
    const dim3 g2(a.K * ((a.d_ff + kWavesPerBlock * kUpLdsRows - 1) / (kWavesPerBlock * kUpLdsRows)));
    MOE_LAUNCH((ffn_up_lds_kernel<DT, kUpLdsRows>), g2, dim3(kThreads), (uint32_t)(a.d * sizeof(float)), l, a);
  }
  return hipGetLastError();
}

template <int DT>
hipError_t launch_down_t(const FfnArgs &a, const Launch &l) {
  const DownShape sh = down_shape(a.d_ff, DT);
  const int rows = kWavesPerBlock * sh.rows;
  const dim3 grid(((a.d + rows - 1) / rows) * ffn_down_chunks(a.K, a.d_ff, DT));
  if (sh.steps == 4)
    MOE_LAUNCH((ffn_down_kernel<DT, 4, 2>), grid, dim3(kThreads), 0, l, a);
  else
    MOE_LAUNCH((ffn_down_kernel<DT, 2, 4>), grid, dim3(kThreads), 0, l, a);
  return hipGetLastError();
}

}  // namespace

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
  MOE_LAUNCH(ffn_reduce_kernel, dim3((a.d + kThreads - 1) / kThreads), dim3(kThreads), 0, l,
             (const float *)a.part, ffn_down_chunks(a.K, a.d_ff, dtype), a.d, a.h);
  return hipGetLastError();
}

}  // namespace moe
