// Decode expert FFN (SwiGLU) on group-quantised experts.
//
// The measured model of the paper kept its experts as 2-bit codes in groups
// of 16 weights with compressed zero points (Sec. 5.1).  Storage of one matrix
// [rows x cols] here (cols a multiple of 64), three planes back to back:
//   codes  [rows][cols / 4]  uint8, column c in bits 2 (c % 4) of byte c / 4
//   scales [rows][cols / 16] fp16, one per group of 16 consecutive columns
//   zeros  [rows][cols / 16] uint8, zero point = code / 64
// and the weight is (q - zero) * scale, an exact fp32 number.  An expert is
// W1 [d_ff x d] | W3 [d_ff x d] | W2 [d x d_ff], 7 bytes per 16 weights.
//
// Same structure as the bf16/fp32 kernels: an HBM-bound GEMV with the
// activation in registers, all of a wave's loads issued before its
// arithmetic, and a down projection split along its reduction axis whose
// partial sums the shared reduction kernel adds in a fixed order.  A lane owns
// 64 consecutive columns (four groups) per step: 16 bytes of codes, 8 bytes
// of scales and 4 bytes of zero codes.  Per group the dot product is taken as
// scale * (sum_i q_i x_i - zero * sum_i x_i) with the group sums of x formed
// once; four codes are masked out of a word at a time and converted byte by
// byte, so a weight costs about 2.4 vector instructions.
//
// Loads are issued from addresses clamped into the matrix (rows past the end
// read the last row, columns past the end the last unit) so that none sits
// behind a branch; those lanes multiply with x = 0 and those rows are not
// written.
#include "common.hpp"

namespace moe {
namespace {

constexpr int kThreads = 256;
constexpr int kWpb = kThreads / kWave;
constexpr int kLaneCols = 64;                 // four groups of 16
constexpr int kStepCols = kWave * kLaneCols;  // 4096 columns per wave step
constexpr int kQUpRows = 2;                   // rows of W1 and of W3 per wave and step
constexpr int kUpWaves = 256 * 4 * 3;         // waves of one up launch: 3 per SIMD
constexpr int kQDownRows = 8;                 // rows of W2 per wave

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

struct QUnit {
  u32x4 c;     // 64 codes
  u32x2 s;     // 4 fp16 scales
  uint32_t z;  // 4 zero codes
};

struct QMat {
  const uint8_t *codes, *scales, *zeros;
  int rows, cols;
};

__device__ __forceinline__ QMat qmat(const uint8_t *base, int rows, int cols) {
  const size_t n = (size_t)rows * cols;
  return QMat{base, base + n / 4, base + n / 4 + n / 8, rows, cols};
}

// The unit of row `row` that starts at column `col` (a multiple of 64), both
// clamped into the matrix.
__device__ __forceinline__ QUnit load_unit(const QMat &m, int row, int col) {
  row = min(row, m.rows - 1);
  col = min(col, m.cols - kLaneCols);
  const size_t e = (size_t)row * m.cols + col;
  QUnit u;
  u.c = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(m.codes + e / 4));
  u.s = __builtin_nontemporal_load(reinterpret_cast<const u32x2 *>(m.scales + e / 8));
  u.z = __builtin_nontemporal_load(reinterpret_cast<const uint32_t *>(m.zeros + e / 16));
  return u;
}

// 64 consecutive activations times `scale` (zeros past `n`) and their group sums.
__device__ __forceinline__ void load_x(const float *p, int c, int n, float scale, float *x, float *xs) {
#pragma unroll
  for (int v = 0; v < kLaneCols; v += 4) {
    float4 t = make_float4(0.f, 0.f, 0.f, 0.f);
    if (c + v < n) t = *reinterpret_cast<const float4 *>(p + c + v);
    x[v] = t.x * scale;
    x[v + 1] = t.y * scale;
    x[v + 2] = t.z * scale;
    x[v + 3] = t.w * scale;
  }
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    float s = 0.0f;
#pragma unroll
    for (int i = 0; i < 16; ++i) s += x[16 * g + i];
    xs[g] = s;
  }
}

// Byte j of a word as a float (v_cvt_f32_ubyte<j>).  Written out because the
// compiler otherwise extracts each 2-bit field on its own before converting.
template <int J>
__device__ __forceinline__ float byte_to_f32(uint32_t m) {
  float r;
  if constexpr (J == 0) asm("v_cvt_f32_ubyte0 %0, %1" : "=v"(r) : "v"(m));
  else if constexpr (J == 1) asm("v_cvt_f32_ubyte1 %0, %1" : "=v"(r) : "v"(m));
  else if constexpr (J == 2) asm("v_cvt_f32_ubyte2 %0, %1" : "=v"(r) : "v"(m));
  else asm("v_cvt_f32_ubyte3 %0, %1" : "=v"(r) : "v"(m));
  return r;
}

// sum over the unit's 64 columns of w_c x_c
__device__ __forceinline__ float unit_dot(const QUnit &u, const float *x, const float *xs) {
  float out = 0.0f;
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    const uint32_t w = u.c[g];
    float acc = 0.0f;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      // byte j of m holds the code of column 4 j + t
      const uint32_t m = (w >> (2 * t)) & 0x03030303u;
      acc = fmaf(byte_to_f32<0>(m), x[16 * g + t], acc);
      acc = fmaf(byte_to_f32<1>(m), x[16 * g + 4 + t], acc);
      acc = fmaf(byte_to_f32<2>(m), x[16 * g + 8 + t], acc);
      acc = fmaf(byte_to_f32<3>(m), x[16 * g + 12 + t], acc);
    }
    const uint32_t sb = (u.s[g >> 1] >> (16 * (g & 1))) & 0xFFFFu;
    const float s = (float)__builtin_bit_cast(_Float16, (uint16_t)sb);
    const float z = (float)((u.z >> (8 * g)) & 0xFFu) * (1.0f / 64.0f);
    out = fmaf(s, fmaf(-z, xs[g], acc), out);
  }
  return out;
}

__device__ __forceinline__ float silu(float v) { return v / (1.0f + __expf(-v)); }

// act_r = SiLU(W1_r x) * (W3_r x), x = h / rms(h); d <= STEPS * 4096.
// G workgroups per rank; each wave walks row groups of RPW rows with a stride
// of G * 4 groups, loading the next group's weights before it works on the
// current one, so memory latency hides behind the dequantising arithmetic.
template <int STEPS, int RPW>
__global__ __launch_bounds__(kThreads) void ffnq_up_kernel(FfnArgs a, int G) {
  const int rank = blockIdx.x / G;
  const int gb = blockIdx.x - rank * G;
  if (rank >= a.route->k) return;
  const int slot = a.route->slot[rank];
  if (slot < 0 || slot >= a.S) return;
  const int d = a.d, d_ff = a.d_ff;
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);  // wave-uniform
  const int nrg = (d_ff + RPW - 1) / RPW;
  const int stride = G * kWpb;
  int rg = gb * kWpb + wave;
  if (rg >= nrg) return;

  const uint8_t *base = a.arena + ((size_t)a.layer * a.S + slot) * a.expert_bytes;
  const size_t mbytes = (size_t)d_ff * d / 16 * 7;
  const QMat w1 = qmat(base, d_ff, d), w3 = qmat(base + mbytes, d_ff, d);
  QUnit c1[RPW][STEPS], c3[RPW][STEPS];
#pragma unroll
  for (int q = 0; q < RPW; ++q)
#pragma unroll
    for (int s = 0; s < STEPS; ++s) {
      c1[q][s] = load_unit(w1, rg * RPW + q, s * kStepCols + lane * kLaneCols);
      c3[q][s] = load_unit(w3, rg * RPW + q, s * kStepCols + lane * kLaneCols);
    }
  float x[STEPS][kLaneCols], xs[STEPS][4];
#pragma unroll
  for (int s = 0; s < STEPS; ++s) load_x(a.h, s * kStepCols + lane * kLaneCols, d, a.route->inv_r, x[s], xs[s]);

  for (; rg < nrg; rg += stride) {
    QUnit n1[RPW][STEPS], n3[RPW][STEPS];
    const bool more = rg + stride < nrg;  // same for the whole wave
    if (more) {
#pragma unroll
      for (int q = 0; q < RPW; ++q)
#pragma unroll
        for (int s = 0; s < STEPS; ++s) {
          n1[q][s] = load_unit(w1, (rg + stride) * RPW + q, s * kStepCols + lane * kLaneCols);
          n3[q][s] = load_unit(w3, (rg + stride) * RPW + q, s * kStepCols + lane * kLaneCols);
        }
    }
#pragma unroll
    for (int q = 0; q < RPW; ++q) {
      float a1 = 0.0f, a3 = 0.0f;
#pragma unroll
      for (int s = 0; s < STEPS; ++s) {
        a1 += unit_dot(c1[q][s], x[s], xs[s]);
        a3 += unit_dot(c3[q][s], x[s], xs[s]);
      }
      a1 = wave_sum(a1);
      a3 = wave_sum(a3);
      const int row = rg * RPW + q;
      if (lane == 0 && row < d_ff) a.act[(size_t)rank * d_ff + row] = silu(a1) * a3;
    }
    if (more) {
#pragma unroll
      for (int q = 0; q < RPW; ++q)
#pragma unroll
        for (int s = 0; s < STEPS; ++s) {
          c1[q][s] = n1[q][s];
          c3[q][s] = n3[q][s];
        }
    }
  }
}

// one (row block, rank, 4096-column chunk) per workgroup: partial sums of
// g_r W2_r act_r for RPW rows per wave
template <int RPW>
__global__ __launch_bounds__(kThreads) void ffnq_down_kernel(FfnArgs a) {
  const int d = a.d, d_ff = a.d_ff, K = a.route->k;
  const int cpr = (d_ff + kStepCols - 1) / kStepCols;
  const int nch = a.K * cpr;
  const int rb = blockIdx.x / nch;
  const int ch = blockIdx.x - rb * nch;
  const int rank = ch / cpr;
  const int c0 = (ch - rank * cpr) * kStepCols;
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  const int row0 = rb * kWpb * RPW + wave * RPW;

  const int slot = rank < K ? a.route->slot[rank] : -1;
  const bool valid = rank < K && slot >= 0 && slot < a.S;
  float acc[RPW] = {};
  if (valid) {
    const uint8_t *base = a.arena + ((size_t)a.layer * a.S + slot) * a.expert_bytes;
    const QMat w2 = qmat(base + 2 * ((size_t)d_ff * d / 16 * 7), d, d_ff);
    QUnit u[RPW];
#pragma unroll
    for (int q = 0; q < RPW; ++q) u[q] = load_unit(w2, row0 + q, c0 + lane * kLaneCols);
    float x[kLaneCols], xs[4];
    load_x(a.act + (size_t)rank * d_ff, c0 + lane * kLaneCols, d_ff, a.route->g[rank], x, xs);
#pragma unroll
    for (int q = 0; q < RPW; ++q) acc[q] = unit_dot(u[q], x, xs);
  }
#pragma unroll
  for (int q = 0; q < RPW; ++q) {
    const float s = wave_sum(acc[q]);
    if (lane == 0 && row0 + q < d) a.part[(size_t)ch * d + row0 + q] = s;
  }
}

}  // namespace

int ffnq_down_chunks(int K, int d_ff) { return K * ((d_ff + kStepCols - 1) / kStepCols); }

hipError_t launch_ffnq_up(const FfnArgs &a, const Launch &l) {
  // about kUpWaves waves in total, at most one row group each
  const int groups = (a.d_ff + kQUpRows - 1) / kQUpRows;
  const int G = max(1, min((groups + kWpb - 1) / kWpb, kUpWaves / (kWpb * max(1, a.K))));
  const dim3 grid(a.K * G);
  if (a.d <= kStepCols)
    MOE_LAUNCH((ffnq_up_kernel<1, kQUpRows>), grid, dim3(kThreads), 0, l, a, G);
  else
    MOE_LAUNCH((ffnq_up_kernel<2, kQUpRows>), grid, dim3(kThreads), 0, l, a, G);
  return hipGetLastError();
}

hipError_t launch_ffnq_down(const FfnArgs &a, const Launch &l) {
  const int rows = kWpb * kQDownRows;
  const dim3 grid(((a.d + rows - 1) / rows) * ffnq_down_chunks(a.K, a.d_ff));
  MOE_LAUNCH((ffnq_down_kernel<kQDownRows>), grid, dim3(kThreads), 0, l, a);
  return hipGetLastError();
}

}  // namespace moe
