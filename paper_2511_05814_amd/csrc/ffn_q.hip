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
// Same structure as the bf16/fp32 kernels: an HBM-bound GEMV, all of a
// wave's loads for the next rows issued before its arithmetic on the current
// ones, and a down projection split along its reduction axis (chunks of 4096
// columns) whose partial sums the shared reduction kernel adds in a fixed
// order.  A lane owns 64 consecutive columns (four groups) of a row: 16 bytes
// of codes, 8 bytes of scales and 4 bytes of zero codes.  Per group the dot
// product is scale * (sum_i q_i x_i - zero * sum_i x_i) with the group sums of
// x formed once.  For d <= 4096 (up) and for every 4096-column chunk (down)
// the sums of q_i x_i come from a table in LDS (see ffnq_up_lut_kernel); the
// up projection of wider models masks four codes out of a word at a time and
// converts them byte by byte (about 2.4 vector instructions a weight).
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

// Sum over the 64 lanes of a wave, left in lane 63, through DPP moves (no LDS
// round trips): running sums within each row of 16 lanes (row_shr 1, 2, 4,
// 8), then lane 15 of rows 0 and 2 into rows 1 and 3 (row_bcast:15) and lane
// 31 into rows 2 and 3 (row_bcast:31).  Lanes whose DPP source lies outside
// the pattern add the 0 passed as the old value.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float dpp_add(float v) {
  return v + __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, ROW_MASK,
                                                                   0xF, false));
}
__device__ __forceinline__ float wave_sum_to_lane63(float v) {
  v = dpp_add<0x111, 0xF>(v);  // row_shr:1
  v = dpp_add<0x112, 0xF>(v);  // row_shr:2
  v = dpp_add<0x114, 0xF>(v);  // row_shr:4
  v = dpp_add<0x118, 0xF>(v);  // row_shr:8
  v = dpp_add<0x142, 0xA>(v);  // row_bcast:15
  v = dpp_add<0x143, 0xC>(v);  // row_bcast:31
  return v;
}

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

// up through a lookup table, for d <= 4096 (one 64-column unit per lane).
// With x fixed for the whole launch, the contribution of a 4-bit nibble of
// codes (two adjacent columns c, c + 1 of a lane's 64) is one of 16 values
// q0 x_c + q1 x_c+1.  Each workgroup first writes those values for all 64
// lanes' 32 column pairs to LDS, laid out [pair][nibble][lane] (128 KB), so
// the 64 lanes of a lookup always hit 64 different banks.  A nibble then
// costs one v_perm_b32, which forms the LDS address (nibble << 8 | lane << 2,
// plus 64 KB for pairs 16..31) straight from the byte holding the nibble, one
// LDS read and one add: with the byte masks and the per-group scale and zero
// about 1.4 vector instructions a weight instead of 2.7.  The sums differ
// from the direct form only in rounding (one rounding per table entry).  One
// workgroup of 16 waves per CU; each wave walks rows of both ranks (W1 and W3
// of a row together), loading the codes of its next row (kQAhead) as it
// finishes one.
constexpr int kLutThreads = 1024;
constexpr int kLutWaves = kLutThreads / kWave;
constexpr int kLutPairs = kLaneCols / 2;  // column pairs per lane
#ifndef MOE_FFNQ_AHEAD
#define MOE_FFNQ_AHEAD 1
#endif
// Rows (items) whose codes a wave loads ahead of the one it works on.  One:
// the kernels are bound by vector-ALU and LDS issue, the 16 waves of a CU keep
// enough loads in flight between them, and every row held ahead costs
// registers and instructions (at the Mixtral shape, up/down: 21.9/13.2 us with
// one, 23.8/13.3 with two, 26.1/13.7 with three, 34.0/16.3 with six).
constexpr int kQAhead = MOE_FFNQ_AHEAD;

// Writes the table for x_c = scale * src[c] over columns c < n of every
// lane's 64 (zeros past n), then returns this lane's four group sums of x
// divided by 64.  Called by all kLutThreads threads; ends with the table
// readable.
__device__ __forceinline__ void lut_build(float *tab, const float *src, int n, float scale, int lane, int wave,
                                          float *xs64) {
#pragma unroll
  for (int i = 0; i < 2; ++i) {  // wave w writes pairs w and w + 16 of every lane
    const int p = wave + kLutWaves * i;
    const int c = lane * kLaneCols + 2 * p;
    float x0 = 0.0f, x1 = 0.0f;
    if (c < n) {
      const float2 v = *reinterpret_cast<const float2 *>(src + c);
      x0 = v.x * scale;
      x1 = v.y * scale;
    }
#pragma unroll
    for (int v = 0; v < 16; ++v) tab[(p * 16 + v) * kWave + lane] = fmaf((float)(v >> 2), x1, (float)(v & 3) * x0);
  }
  __syncthreads();
#pragma unroll
  for (int g = 0; g < 4; ++g) {  // nibble 5 = codes 1, 1: x_c + x_c+1
    float t = 0.0f;
#pragma unroll
    for (int n8 = 0; n8 < 8; ++n8) t += tab[((8 * g + n8) * 16 + 5) * kWave + lane];
    xs64[g] = t * (1.0f / 64.0f);
  }
}

// sum over this lane's 64 columns of w_c x_c for one unit, through the table
__device__ __forceinline__ float lut_dot(const float *tab, const QUnit &u, int lane, const float *xs64) {
  const uint32_t lb0 = (uint32_t)lane * 4u, lb1 = lb0 | 0x10000u;
  const char *tb = reinterpret_cast<const char *>(tab);
  float out = 0.0f;
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    const uint32_t w = u.c[g];
    const uint32_t lo = w & 0x0F0F0F0Fu, hi = (w >> 4) & 0x0F0F0F0Fu;
    const uint32_t lb = g < 2 ? lb0 : lb1;
    float acc = 0.0f;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      // byte j of lo: pair 8 g + 2 j; of hi: pair 8 g + 2 j + 1
      const uint32_t sel = 0x0C020000u | ((uint32_t)(4 + j) << 8);
      const uint32_t alo = __builtin_amdgcn_perm(lo, lb, sel);
      const uint32_t ahi = __builtin_amdgcn_perm(hi, lb, sel);
      const int p = (8 * g + 2 * j) & 15;
      acc += *reinterpret_cast<const float *>(tb + alo + p * 4096);
      acc += *reinterpret_cast<const float *>(tb + ahi + (p + 1) * 4096);
    }
    const uint32_t sb = (u.s[g >> 1] >> (16 * (g & 1))) & 0xFFFFu;
    const float sc = (float)__builtin_bit_cast(_Float16, (uint16_t)sb);
    const float z = (float)((u.z >> (8 * g)) & 0xFFu);
    out = fmaf(sc, fmaf(-z, xs64[g], acc), out);
  }
  return out;
}

__global__ __launch_bounds__(kLutThreads, 1) void ffnq_up_lut_kernel(FfnArgs a) {
  __shared__ float tab[kLutPairs * 16 * kWave];
  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int d = a.d, d_ff = a.d_ff, K = a.route->k;
  const uint8_t *const arena = a.arena;
  const size_t mbytes = (size_t)d_ff * d / 16 * 7;
  const int col = lane * kLaneCols;
  // work: row r of rank k (W1 and W3) is item k * d_ff + r; wave w takes
  // items w, w + stride, ... (with d_ff a multiple of 64 and 4096 waves, the
  // Mixtral shape gives every wave 7 of them)
  const int nitems = K * d_ff;
  const int stride = gridDim.x * kLutWaves;
  const int first = blockIdx.x * kLutWaves + wave;
  auto load_item = [&](int it, QUnit (&u)[2]) {
    it = min(it, nitems - 1);  // past the end: a valid row, never used
    const int rank = it / d_ff, row = it - rank * d_ff;
    int slot = a.route->slot[rank];
    slot = slot < 0 ? 0 : (slot >= a.S ? a.S - 1 : slot);  // the router never writes these; clamp, not branch
    const uint8_t *base = arena + ((size_t)a.layer * a.S + slot) * a.expert_bytes;
    u[0] = load_unit(qmat(base, d_ff, d), row, col);
    u[1] = load_unit(qmat(base + mbytes, d_ff, d), row, col);
  };
  // the first kQAhead items' codes are on their way while the table is built;
  // the ring of item slots is unrolled, so slot q stays in the same registers
  QUnit u[kQAhead][2];
#pragma unroll
  for (int q = 0; q < kQAhead; ++q) load_item(first + q * stride, u[q]);
  float xs64[4];
  lut_build(tab, a.h, d, a.route->inv_r, lane, wave, xs64);
  for (int it0 = first; it0 < nitems; it0 += kQAhead * stride) {
#pragma unroll
    for (int q = 0; q < kQAhead; ++q) {
      const int it = it0 + q * stride;  // item it = rank * d_ff + row
      if (it < nitems) {                // the same for the whole wave
        const float a1 = wave_sum_to_lane63(lut_dot(tab, u[q][0], lane, xs64));
        const float a3 = wave_sum_to_lane63(lut_dot(tab, u[q][1], lane, xs64));
        if (lane == kWave - 1) a.act[it] = silu(a1) * a3;
      }
      load_item(it + kQAhead * stride, u[q]);  // past the end: the last item again (from cache), unused
    }
  }
}

// down through the same kind of table, for d_ff chunks of 4096 columns: one
// workgroup per (block of `rpb` rows of W2, rank, chunk), the table built
// from g_r act_r over the chunk; each wave takes every 16th row of the block
// and writes the chunk's partial row sum.  Invalid ranks write zeros, as the
// reduction reads every chunk.
__global__ __launch_bounds__(kLutThreads, 1) void ffnq_down_lut_kernel(FfnArgs a, int rpb) {
  __shared__ float tab[kLutPairs * 16 * kWave];
  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int d = a.d, d_ff = a.d_ff, K = a.route->k;
  const int cpr = (d_ff + kStepCols - 1) / kStepCols;
  const int nch = a.K * cpr;
  const int rb = blockIdx.x / nch;
  const int ch = blockIdx.x - rb * nch;
  const int rank = ch / cpr;
  const int c0 = (ch - rank * cpr) * kStepCols;
  const int row_lo = rb * rpb, row_hi = min(d, row_lo + rpb);
  const int slot = rank < K ? a.route->slot[rank] : -1;
  if (rank >= K || slot < 0 || slot >= a.S) {
    for (int r = row_lo + tid; r < row_hi; r += kLutThreads) a.part[(size_t)ch * d + r] = 0.0f;
    return;
  }
  const uint8_t *base = a.arena + ((size_t)a.layer * a.S + slot) * a.expert_bytes;
  const QMat w2 = qmat(base + 2 * ((size_t)d_ff * d / 16 * 7), d, d_ff);
  const int col = c0 + lane * kLaneCols;  // load_unit clamps columns past d_ff (those x are zero)
  const int first = row_lo + wave;
  QUnit u[kQAhead];
#pragma unroll
  for (int q = 0; q < kQAhead; ++q) u[q] = load_unit(w2, min(first + q * kLutWaves, row_hi - 1), col);
  float xs64[4];
  lut_build(tab, a.act + (size_t)rank * d_ff + c0, d_ff - c0, a.route->g[rank], lane, wave, xs64);
  for (int r0 = first; r0 < row_hi; r0 += kQAhead * kLutWaves) {
#pragma unroll
    for (int q = 0; q < kQAhead; ++q) {
      const int r = r0 + q * kLutWaves;
      if (r < row_hi) {  // the same for the whole wave
        const float s = wave_sum_to_lane63(lut_dot(tab, u[q], lane, xs64));
        if (lane == kWave - 1) a.part[(size_t)ch * d + r] = s;
      }
      u[q] = load_unit(w2, min(r + kQAhead * kLutWaves, row_hi - 1), col);  // past the end: the last row again
    }
  }
}

}  // namespace

int ffnq_down_chunks(int K, int d_ff) { return K * ((d_ff + kStepCols - 1) / kStepCols); }

hipError_t launch_ffnq_up(const FfnArgs &a, const Launch &l) {
  if (a.d <= kStepCols) {
    // one workgroup per CU (its 128 KB table leaves room for no second one)
    MOE_LAUNCH(ffnq_up_lut_kernel, dim3(256), dim3(kLutThreads), 0, l, a);
    return hipGetLastError();
  }
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
  // about one workgroup per CU: blocks of rows per (rank, chunk)
  const int nch = ffnq_down_chunks(a.K, a.d_ff);
  const int nrb = max(1, 256 / nch);
  const int rpb = (a.d + nrb - 1) / nrb;
  MOE_LAUNCH(ffnq_down_lut_kernel, dim3(((a.d + rpb - 1) / rpb) * nch), dim3(kLutThreads), 0, l, a, rpb);
  return hipGetLastError();
}

}  // namespace moe
