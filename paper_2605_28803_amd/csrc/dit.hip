// DiT action-head denoising step built from the rotated W4A4 linears.
//
// Experimental Settings / Implementation Details: every linear of the DiT
// action head is W4A4 with RTN weights and the per-step activation scale
// table, and the head runs T Euler denoising steps.  The Appendix on per-step
// scaling describes the block: a time-conditioned norm feeding the attention
// q/k/v projections, attention output projection, a norm feeding the MLP.
// Block equations of the Pi-0.5 action expert used here:
//   h = fp16(rms(r) g1 (1 + sc1) + sh1); qkv = W4A4(h); o = attn(q, [Kp;k], [Vp;v]);
//   r += gt1 W4A4(o); h2 = fp16(rms(r) g2 (1 + sc2) + sh2); gu = W4A4(h2);
//   a = fp16(gelu_tanh(gate) up); r += gt2 W4A4(a)
// and the step r = x W_in^T + b_in -> blocks -> v = fp16(rms(r) g_f) W_out^T +
// b_out -> x += dt v.
//
// Nine launches per block, all on one stream, no allocation, no memset:
//   norm_rq_kernel       rms norm + modulation -> fp16 row -> rotate + quantize
//   gemm (w4a4_gemm.hip) q|k|v, fp16 out
//   attn_partial_kernel  softmax(q k^T / sqrt(hd)) v over one 64-key split (fp16 MFMA)
//   combine_rq_kernel    merge the splits (log-sum-exp) -> fp16 row -> rotate + quantize
//   gemm                 o projection, r += gt1 * y in the epilogue
//   norm_rq_kernel       second norm -> rotate + quantize
//   gemm                 gate|up, fp16 out
//   gelu_rq_kernel       gelu_tanh(gate) * up -> fp16 row -> rotate + quantize
//   gemm                 down projection, r += gt2 * y in the epilogue
// Each fused producer writes its fp16 row (the linear's input, kept for
// per-site checks) and quantizes the same values.  A whole denoising step (or
// several) is captured once into a HIP graph per (x, first step, count) on an
// internal stream and replayed on the caller's stream.
#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <type_traits>
#include <vector>

#include "common.h"
#include "rq_device.h"
#include "rq_mfma.h"

namespace oq {
namespace {

using rqd::f16r;
using rqd::h2f;
using rqd::f2h;

constexpr int kAttnKS = 64;     // keys per step of the cross-attention's running merge
constexpr int kAttnSplit = 64;  // keys per split of the split attention (partials, then a merge)
constexpr int kMaxTokens = 64;  // action tokens per sample handled by the attention kernels
constexpr int kMaxHeadDim = 128;
constexpr int kMaxSplits = 16;  // (prefix + tokens) <= 16 * 64 keys
constexpr float kEps = 1e-6f;

__device__ __forceinline__ void load8_f16(const uint16_t* p, float (&o)[8]) {
  const uint4 raw = *reinterpret_cast<const uint4*>(p);
  const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    o[2 * q] = h2f(w[q] & 0xFFFFu);
    o[2 * q + 1] = h2f(w[q] >> 16);
  }
}

__device__ __forceinline__ void store8_f16(uint16_t* p, const float (&v)[8]) {
  uint4 raw;
  raw.x = f2h(v[0]) | (static_cast<uint32_t>(f2h(v[1])) << 16);
  raw.y = f2h(v[2]) | (static_cast<uint32_t>(f2h(v[3])) << 16);
  raw.z = f2h(v[4]) | (static_cast<uint32_t>(f2h(v[5])) << 16);
  raw.w = f2h(v[6]) | (static_cast<uint32_t>(f2h(v[7])) << 16);
  *reinterpret_cast<uint4*>(p) = raw;
}

struct RQOut {
  uint8_t* xq;
  float* xs;
  int logT, logb;
  float s_t, s_over_sqrtb;
  bool tiled;  // codes in the 16-row tiled layout (the small-M product's operand)
  const float* sdelta;  // static per-channel steps of this site and step (null: per-token quantizer)
};

// One output of the action in-projection: sum over a ascending of
// x[a] W_in[n][a] (fma chain); 16-byte weight loads when the row allows them
// (the same sum either way).
__device__ __forceinline__ float inproj_dot(const float* xsh, const uint16_t* __restrict__ wr, int A, bool vec) {
  float acc = 0.0f;
  if (vec) {
    for (int a0 = 0; a0 < A; a0 += 8) {
      const uint4 q = *reinterpret_cast<const uint4*>(wr + a0);
      const uint32_t qw[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        acc = fmaf(xsh[a0 + 2 * j], h2f(qw[j] & 0xFFFFu), acc);
        acc = fmaf(xsh[a0 + 2 * j + 1], h2f(qw[j] >> 16), acc);
      }
    }
  } else {
    for (int a = 0; a < A; ++a) acc = fmaf(xsh[a], h2f(wr[a]), acc);
  }
  return acc;
}

// r = x W_in^T + b_in
__global__ __launch_bounds__(256) void inproj_kernel(const float* __restrict__ x, const uint16_t* __restrict__ w_in,
                                                     const uint16_t* __restrict__ b_in, float* __restrict__ r, int A,
                                                     int D) {
  extern __shared__ float xsh[];
  const int m = blockIdx.x;
  for (int a = threadIdx.x; a < A; a += blockDim.x) xsh[a] = x[static_cast<int64_t>(m) * A + a];
  __syncthreads();
  const bool vec = A % 8 == 0 && (reinterpret_cast<uintptr_t>(w_in) & 15) == 0;
  for (int n = threadIdx.x; n < D; n += blockDim.x)
    r[static_cast<int64_t>(m) * D + n] = inproj_dot(xsh, w_in + static_cast<int64_t>(n) * A, A, vec) + h2f(b_in[n]);
}

// In-projection with the weight row preloaded, for AP = A action channels in
// {8, 16, 24, 32} and 16-byte aligned rows: a W_in row is AP / 8 16-byte
// pieces, all issued before the first sum (the loop of inproj_dot waits for
// each piece before loading the next).  The sums are inproj_dot's: a
// ascending from 0, the bias added last.
constexpr int kInprojA = 32;

__host__ __device__ __forceinline__ int inproj_preload_a(int A, const void* w_in) {
  return A <= kInprojA && A % 8 == 0 && (reinterpret_cast<uintptr_t>(w_in) & 15) == 0 ? A : 0;
}

template <int AP>
__device__ __forceinline__ void inproj_load_row(const uint16_t* __restrict__ wr, uint4 (&q)[AP / 8]) {
#pragma unroll
  for (int i = 0; i < AP / 8; ++i) q[i] = *reinterpret_cast<const uint4*>(wr + 8 * i);
}

template <int AP>
__device__ __forceinline__ float inproj_dot_pre(const float* xa, const uint4 (&q)[AP / 8]) {
  float acc = 0.0f;
#pragma unroll
  for (int i = 0; i < AP / 8; ++i) {
    const uint32_t qw[4] = {q[i].x, q[i].y, q[i].z, q[i].w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      acc = fmaf(xa[8 * i + 2 * j], h2f(qw[j] & 0xFFFFu), acc);
      acc = fmaf(xa[8 * i + 2 * j + 1], h2f(qw[j] >> 16), acc);
    }
  }
  return acc;
}

// r = x W_in^T + b_in with preloaded rows: workgroup (i, j) computes channel
// n = 256 j + t of rows R i .. R i + R - 1 (R * AP <= 256), thread t loading
// its W_in row and bias once for the R rows before the action rows are
// staged in LDS (inproj_kernel reads the whole W_in once per row).
template <int R, int AP>
__global__ __launch_bounds__(256) void inproj_rows_kernel(const float* __restrict__ x,
                                                          const uint16_t* __restrict__ w_in,
                                                          const uint16_t* __restrict__ b_in, float* __restrict__ r,
                                                          int64_t M, int D) {
  static_assert(R * AP <= 256, "one action value per thread");
  __shared__ float xsh[R][AP];
  const int t = threadIdx.x;
  const int n = blockIdx.y * 256 + t;
  const int nn = n < D ? n : 0;
  const int64_t m0 = static_cast<int64_t>(blockIdx.x) * R;
  uint4 q[AP / 8];
  inproj_load_row<AP>(w_in + static_cast<int64_t>(nn) * AP, q);
  const float bb = h2f(b_in[nn]);
  if (t < R * AP) {
    const int i = t / AP, a = t % AP;
    const int64_t m = m0 + i < M ? m0 + i : 0;
    xsh[i][a] = x[m * AP + a];
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < R; ++i) {
    const float v = inproj_dot_pre<AP>(xsh[i], q) + bb;
    if (m0 + i < M && n < D) r[(m0 + i) * D + n] = v;
  }
}

// h = fp16(norm(r) g (1 + sc) + sh), then rotate + quantize h.  norm is the
// RMS norm (LN = false) or the layer norm (LN = true); SC = false means no
// scale vector (sc is not read, taken as zero); sh is always read.  Every
// load of the row is issued before the first reduction.
template <int C, bool LN, bool SC>
__global__ __launch_bounds__(256) void norm_rq_kernel(const float* __restrict__ r, const uint16_t* __restrict__ g,
                                                      const uint16_t* __restrict__ sc,
                                                      const uint16_t* __restrict__ sh, uint16_t* __restrict__ h,
                                                      int64_t M, int D, RQOut o) {
  extern __shared__ float lds[];
  __shared__ float red[4];
  __shared__ float red2[4];
  __shared__ float red3[4];
  const rqd::RowMap m = rqd::row_map(o.logT, M);
  float v[C][8];
  const float* rr = r + (m.valid ? m.row : 0) * D;
#pragma unroll
  for (int c = 0; c < C; ++c) {
    const int k = rqd::chan(m, c, 0);
    const float4 p0 = *reinterpret_cast<const float4*>(rr + k);
    const float4 p1 = *reinterpret_cast<const float4*>(rr + k + 4);
    v[c][0] = p0.x; v[c][1] = p0.y; v[c][2] = p0.z; v[c][3] = p0.w;
    v[c][4] = p1.x; v[c][5] = p1.y; v[c][6] = p1.z; v[c][7] = p1.w;
  }
  float gg[C][8], s1[C][8], s2[C][8];
#pragma unroll
  for (int c = 0; c < C; ++c) {
    const int k = rqd::chan(m, c, 0);
    load8_f16(g + k, gg[c]);
    load8_f16(sh + k, s2[c]);
    if (SC) {
      load8_f16(sc + k, s1[c]);
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j) s1[c][j] = 0.0f;
    }
  }
  float mu = 0.0f;
  if constexpr (LN) {
    float sum = 0.0f;
#pragma unroll
    for (int c = 0; c < C; ++c)
#pragma unroll
      for (int j = 0; j < 8; ++j) sum += v[c][j];
    mu = rqd::row_reduce<false>(sum, m, red3) / static_cast<float>(D);
  }
  float ss = 0.0f;
#pragma unroll
  for (int c = 0; c < C; ++c)
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float d = v[c][j] - mu;
      ss = fmaf(d, d, ss);
    }
  ss = rqd::row_reduce<false>(ss, m, red2);
  const float inv = 1.0f / sqrtf(ss / static_cast<float>(D) + kEps);
#pragma unroll
  for (int c = 0; c < C; ++c) {
    const int k = rqd::chan(m, c, 0);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float y = (v[c][j] - mu) * inv * gg[c][j];
      v[c][j] = f16r(fmaf(y, s1[c][j], y) + s2[c][j]);
    }
    if (m.valid && h) store8_f16(h + m.row * D + k, v[c]);
  }
  rqd::rq_core<C>(v, m, D, o.logb, o.s_t, o.s_over_sqrtb, lds, red, o.xq, o.xs, nullptr, o.tiled, o.sdelta);
}

// ---------------------------------------------------------------------------
// The RMS-norm producer for 1024-channel rows with few rows (the Pi-0.5 action
// tokens, Hadamard block = the row; per-token or static steps): 256 threads per row,
// 4 consecutive channels per thread (channel 4 t + j), so each thread's chain
// of arithmetic is half that of the 128-thread generic layout.  Channel bits
// 0-1 are in registers, bits 2-7 across the lanes of a wave, bits 8-9 across
// the four waves (one exchange through LDS).  Same arithmetic as
// norm_rq_kernel and rqd::rq_core; only the order of the fp32 sums differs.
// ---------------------------------------------------------------------------

__device__ __forceinline__ float wave_sum64(float v) {
  return rqd::wave_sum_xor(v);
}

template <int H>
__device__ __forceinline__ void lane_stage4(float (&x)[4], int lane) {
  const float sgn = (lane & H) ? -1.0f : 1.0f;
  float p[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) p[j] = rqd::lane_xor<H>(x[j]);
#pragma unroll
  for (int j = 0; j < 4; ++j) x[j] = fmaf(sgn, x[j], p[j]);  // upper: p - x, lower: p + x
}

template <int H>
__device__ __forceinline__ void lane_stage4_swap(float (&x)[4]) {
#pragma unroll
  for (int j = 0; j < 4; j += 2) {
    float a = x[j], b = x[j + 1];
    rqd::permlane_swap<H>(a, b);
    const float sm = a + b, df = a - b;
    a = sm;
    b = df;
    rqd::permlane_swap<H>(a, b);
    x[j] = a;
    x[j + 1] = b;
  }
}

// Rotation over the whole 256 NW-channel row (Hadamard block = K) and the int4
// codes (per-token, or with the static steps o.sdelta) of a row held as 4
// channels per thread (channel 4 t + j) by a workgroup of NW waves: channel
// bits 0-1 in registers, bits 2-7 across the lanes, the top log2(NW) bits
// across the waves through LDS (xch: 256 NW floats, 512 NW when NW = 16; red:
// NW floats, both unused by the caller meanwhile).  Every thread calls it.
template <int NW>
__device__ __forceinline__ void rq_row4(float (&x)[4], int64_t row, bool valid, const RQOut& o, float* xch,
                                        float* red) {
  constexpr int D = 256 * NW;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int k0 = 4 * t;
  // Channel bits 0-1.
  {
    const float a0 = x[0] + x[1], a1 = x[0] - x[1], a2 = x[2] + x[3], a3 = x[2] - x[3];
    x[0] = a0 + a2;
    x[2] = a0 - a2;
    x[1] = a1 + a3;
    x[3] = a1 - a3;
  }
  // Channel bits 2-7: lane bits 0-5.
  lane_stage4<1>(x, lane);
  lane_stage4<2>(x, lane);
  lane_stage4<4>(x, lane);
  lane_stage4<8>(x, lane);
  lane_stage4_swap<16>(x);
  lane_stage4_swap<32>(x);
  // Channel bits 8 and up: the NW waves.  With 16 waves, two radix-4 rounds
  // (wave bits 0-1, then 2-3; H_16 = H_4 x H_4) through two LDS buffers: each
  // thread reads 8 instead of 16 float4, half the LDS traffic of one round.
  if constexpr (NW == 16) {
    float* xch2 = xch + D;
    *reinterpret_cast<float4*>(&xch[k0]) = make_float4(x[0], x[1], x[2], x[3]);
    __syncthreads();
    float z[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const float sg = (__popc(w & u) & 1) ? -1.0f : 1.0f;
      const float4 q = *reinterpret_cast<const float4*>(&xch[(((w & ~3) + u) * 64 + lane) * 4]);
      z[0] = fmaf(sg, q.x, z[0]);
      z[1] = fmaf(sg, q.y, z[1]);
      z[2] = fmaf(sg, q.z, z[2]);
      z[3] = fmaf(sg, q.w, z[3]);
    }
    *reinterpret_cast<float4*>(&xch2[k0]) = make_float4(z[0], z[1], z[2], z[3]);
    __syncthreads();
    float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const float sg = (__popc((w >> 2) & u) & 1) ? -1.0f : 1.0f;
      const float4 q = *reinterpret_cast<const float4*>(&xch2[((4 * u + (w & 3)) * 64 + lane) * 4]);
      acc[0] = fmaf(sg, q.x, acc[0]);
      acc[1] = fmaf(sg, q.y, acc[1]);
      acc[2] = fmaf(sg, q.z, acc[2]);
      acc[3] = fmaf(sg, q.w, acc[3]);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) x[j] = acc[j];
  } else {
    *reinterpret_cast<float4*>(&xch[k0]) = make_float4(x[0], x[1], x[2], x[3]);
    __syncthreads();
    float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int u = 0; u < NW; ++u) {
      const float sg = (__popc(w & u) & 1) ? -1.0f : 1.0f;
      const float4 q = *reinterpret_cast<const float4*>(&xch[(u * 64 + lane) * 4]);
      acc[0] = fmaf(sg, q.x, acc[0]);
      acc[1] = fmaf(sg, q.y, acc[1]);
      acc[2] = fmaf(sg, q.z, acc[2]);
      acc[3] = fmaf(sg, q.w, acc[3]);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) x[j] = acc[j];
  }
  const int p = k0 / 2;  // even: both bytes in one 16-byte piece of the tiled layout
  uint8_t* dst = o.tiled ? o.xq + tiled_offset(row, p, D / 128) : o.xq + row * (D / 2) + p;
  uint32_t c[4];
  if (o.sdelta != nullptr) {
    // Static per-channel steps (as rq_core): token scale 1, no row maximum
    // (the branch is uniform over the grid).
    if (!valid) return;
    if (t == 0) o.xs[row] = 1.0f;
    const float4 d = *reinterpret_cast<const float4*>(o.sdelta + k0);
    c[0] = rqd::static_code(x[0], d.x, o.s_over_sqrtb) & 0xFu;
    c[1] = rqd::static_code(x[1], d.y, o.s_over_sqrtb) & 0xFu;
    c[2] = rqd::static_code(x[2], d.z, o.s_over_sqrtb) & 0xFu;
    c[3] = rqd::static_code(x[3], d.w, o.s_over_sqrtb) & 0xFu;
    *reinterpret_cast<uint16_t*>(dst) = static_cast<uint16_t>(c[0] | (c[1] << 4) | (c[2] << 8) | (c[3] << 12));
    return;
  }
  // Row maximum of the unnormalized transform, scales, codes (as rq_core).
  float amax = fmaxf(fmaxf(fabsf(x[0]), fabsf(x[1])), fmaxf(fabsf(x[2]), fabsf(x[3])));
  amax = rqd::wave_max(amax);
  if (lane == 0) red[w] = amax;
  __syncthreads();
  amax = red[0];
#pragma unroll
  for (int u = 1; u < NW; ++u) amax = fmaxf(amax, red[u]);
  const float a_z = amax * o.s_over_sqrtb;
  const float delta = a_z / 7.0f;
  const float gm = delta > 0.0f ? o.s_over_sqrtb / delta : 0.0f;
  if (!valid) return;
  if (t == 0) o.xs[row] = delta / o.s_t;
#pragma unroll
  for (int j = 0; j < 4; ++j) c[j] = __float_as_uint(fmaf(x[j], gm, rqd::kRoundMagic)) & 0xFu;
  // Byte i: channel 2i in the low nibble, 2i + 1 in the high nibble.
  *reinterpret_cast<uint16_t*>(dst) = static_cast<uint16_t>(c[0] | (c[1] << 4) | (c[2] << 8) | (c[3] << 12));
}

__device__ __forceinline__ void rq1024_row(float (&x)[4], int64_t row, bool valid, const RQOut& o, float* xch,
                                           float* red) {
  rq_row4<4>(x, row, valid, o, xch, red);
}

// h = fp16(norm(r) g (1 + sc) + sh) for 1536-channel rows (the GR00T hidden
// size: three 512-channel Hadamard blocks), then rotate + quantize h: one row
// per three-wave workgroup, wave w holding block w as 8 consecutive channels
// per lane in the matrix-core layout of rqm::rq_row (H_32 on the fp16 matrix
// cores, then the lane butterflies; only the row maximum is shared).  The norm
// statistics are summed in each wave, then over the three waves in LDS.
template <bool LN, bool SC>
__global__ __launch_bounds__(192) void norm_rq1536_kernel(const float* __restrict__ r, const uint16_t* __restrict__ g,
                                                          const uint16_t* __restrict__ sc,
                                                          const uint16_t* __restrict__ sh, uint16_t* __restrict__ h,
                                                          int64_t M, RQOut o) {
  constexpr int D = 1536;
  __shared__ float red[4];
  __shared__ float rs[2][3];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int64_t row = blockIdx.x;
  const bool valid = row < M;
  const int k = rqm::chan0<1>(wv, 0, lane);
  const float4* rr = reinterpret_cast<const float4*>(r + (valid ? row : 0) * D + k);
  const float4 p0 = rr[0], p1 = rr[1];
  const float v[8] = {p0.x, p0.y, p0.z, p0.w, p1.x, p1.y, p1.z, p1.w};
  float gg[8], s1[8], s2[8];
  load8_f16(g + k, gg);
  load8_f16(sh + k, s2);
  if (SC) {
    load8_f16(sc + k, s1);
  } else {
#pragma unroll
    for (int j = 0; j < 8; ++j) s1[j] = 0.0f;
  }
  float mu = 0.0f;
  if constexpr (LN) {
    float sum = 0.0f;
#pragma unroll
    for (int j = 0; j < 8; ++j) sum += v[j];
    sum = wave_sum64(sum);
    if (lane == 0) rs[0][wv] = sum;
    __syncthreads();
    mu = (rs[0][0] + rs[0][1] + rs[0][2]) / static_cast<float>(D);
  }
  float ss = 0.0f;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const float d = v[j] - mu;
    ss = fmaf(d, d, ss);
  }
  ss = wave_sum64(ss);
  if (lane == 0) rs[1][wv] = ss;
  __syncthreads();
  ss = rs[1][0] + rs[1][1] + rs[1][2];
  const float inv = 1.0f / sqrtf(ss / static_cast<float>(D) + kEps);
  float x[8];
  rqm::rv8h cur[1];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const float y = (v[j] - mu) * inv * gg[j];
    x[j] = valid ? f16r(fmaf(y, s1[j], y) + s2[j]) : 0.0f;
    cur[0][j] = static_cast<_Float16>(x[j]);
  }
  if (valid && h) store8_f16(h + row * D + k, x);
  rqm::rv8h a1, a2;
  rqm::hadamard_frags(lane, a1, a2);
  rqm::rq_row<1, 3, false>(cur, a1, a2, row, valid, lane, wv, o.logb, o.s_t, o.s_over_sqrtb, o.xq, o.xs, nullptr,
                           nullptr, red, o.tiled, o.sdelta);
}

// RMS norm, modulation, fp16 rounding and rotate-quantize of one 1024-channel
// row whose values v (channels 4 t .. 4 t + 3) thread t already holds; h
// (optional) receives the fp16 row.
template <bool SC>
__device__ __forceinline__ void norm1024_row(const float (&v)[4], const uint16_t* __restrict__ g,
                                             const uint16_t* __restrict__ sc, const uint16_t* __restrict__ sh,
                                             uint16_t* __restrict__ h, int64_t row, bool valid, const RQOut& o,
                                             float* xch, float (&red)[2][4]) {
  constexpr int D = 1024;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int k0 = 4 * t;
  const uint2 gq = *reinterpret_cast<const uint2*>(g + k0);
  const uint2 hq = *reinterpret_cast<const uint2*>(sh + k0);
  uint2 cq = make_uint2(0, 0);
  if (SC) cq = *reinterpret_cast<const uint2*>(sc + k0);
  const float gg[4] = {h2f(gq.x & 0xFFFFu), h2f(gq.x >> 16), h2f(gq.y & 0xFFFFu), h2f(gq.y >> 16)};
  const float s2[4] = {h2f(hq.x & 0xFFFFu), h2f(hq.x >> 16), h2f(hq.y & 0xFFFFu), h2f(hq.y >> 16)};
  const float s1[4] = {SC ? h2f(cq.x & 0xFFFFu) : 0.0f, SC ? h2f(cq.x >> 16) : 0.0f,
                       SC ? h2f(cq.y & 0xFFFFu) : 0.0f, SC ? h2f(cq.y >> 16) : 0.0f};
  float ss = 0.0f;
#pragma unroll
  for (int j = 0; j < 4; ++j) ss = fmaf(v[j], v[j], ss);
  ss = wave_sum64(ss);
  if (lane == 0) red[0][w] = ss;
  __syncthreads();
  ss = (red[0][0] + red[0][1]) + (red[0][2] + red[0][3]);
  const float inv = 1.0f / sqrtf(ss / static_cast<float>(D) + kEps);
  float x[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const float y = v[j] * inv * gg[j];
    x[j] = valid ? f16r(fmaf(y, s1[j], y) + s2[j]) : 0.0f;
  }
  if (valid && h)
    *reinterpret_cast<uint2*>(h + row * D + k0) =
        make_uint2(static_cast<uint32_t>(f2h(x[0])) | (static_cast<uint32_t>(f2h(x[1])) << 16),
                   static_cast<uint32_t>(f2h(x[2])) | (static_cast<uint32_t>(f2h(x[3])) << 16));
  rq1024_row(x, row, valid, o, xch, red[1]);
}

template <bool SC>
__global__ __launch_bounds__(256) void norm_rq1024_kernel(const float* __restrict__ r,
                                                          const uint16_t* __restrict__ g,
                                                          const uint16_t* __restrict__ sc,
                                                          const uint16_t* __restrict__ sh, uint16_t* __restrict__ h,
                                                          int64_t M, RQOut o) {
  constexpr int D = 1024;
  __shared__ __attribute__((aligned(16))) float xch[D];
  __shared__ float red[2][4];
  const int64_t row = blockIdx.x;
  const bool valid = row < M;
  const float4 rv = *reinterpret_cast<const float4*>(r + (valid ? row : 0) * D + 4 * threadIdx.x);
  const float v[4] = {rv.x, rv.y, rv.z, rv.w};
  norm1024_row<SC>(v, g, sc, sh, h, row, valid, o, xch, red);
}

// The action in-projection r = x W_in^T + b_in (the same sums as
// inproj_kernel) fused with the first block's norm producer (as
// norm_rq1024_kernel): one 1024-channel row per 256-thread workgroup, thread
// t computing channels 4 t .. 4 t + 3 (A <= 256 action channels).
template <bool SC>
__global__ __launch_bounds__(256) void inproj_norm_rq1024_kernel(const float* __restrict__ x,
                                                                 const uint16_t* __restrict__ w_in,
                                                                 const uint16_t* __restrict__ b_in,
                                                                 float* __restrict__ r, int A,
                                                                 const uint16_t* __restrict__ g,
                                                                 const uint16_t* __restrict__ sc,
                                                                 const uint16_t* __restrict__ sh,
                                                                 uint16_t* __restrict__ h, int64_t M, RQOut o) {
  constexpr int D = 1024;
  __shared__ __attribute__((aligned(16))) float xch[D];
  __shared__ float red[2][4];
  __shared__ float xsh[256];
  const int t = threadIdx.x;
  const int64_t row = blockIdx.x;
  const bool valid = row < M;
  if (t < A) xsh[t] = x[(valid ? row : 0) * A + t];
  __syncthreads();
  const bool vec = A % 8 == 0 && (reinterpret_cast<uintptr_t>(w_in) & 15) == 0;
  float v[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int n = 4 * t + j;
    v[j] = inproj_dot(xsh, w_in + static_cast<int64_t>(n) * A, A, vec) + h2f(b_in[n]);
  }
  if (valid) *reinterpret_cast<float4*>(r + row * D + 4 * t) = make_float4(v[0], v[1], v[2], v[3]);
  norm1024_row<SC>(v, g, sc, sh, h, row, valid, o, xch, red);
}

// gelu_rq_kernel for 4096-channel rows with few rows (the Pi-0.5 action
// tokens, Hadamard block = the row): one row per 1024-thread workgroup, 4
// consecutive channels per thread, the same activation arithmetic, then
// rq_row4 over 16 waves.
template <bool GATED>
__global__ __launch_bounds__(1024) void gelu_rq4096_kernel(const uint16_t* __restrict__ gu,
                                                           uint16_t* __restrict__ act, int64_t M, RQOut o) {
  constexpr int F = 4096;
  __shared__ __attribute__((aligned(16))) float xch[2 * F];  // the two rounds of the 16-wave exchange
  __shared__ float red[16];
  const int t = threadIdx.x;
  const int64_t row = blockIdx.x;
  const bool valid = row < M;
  const int k0 = 4 * t;
  const int64_t ld = GATED ? 2 * F : F;
  const uint16_t* gr = gu + (valid ? row : 0) * ld;
  const uint2 gq = *reinterpret_cast<const uint2*>(gr + k0);
  uint2 uq = make_uint2(0x3C003C00u, 0x3C003C00u);  // fp16 1.0 pairs
  if (GATED) uq = *reinterpret_cast<const uint2*>(gr + F + k0);
  const uint32_t gw[2] = {gq.x, gq.y}, uw[2] = {uq.x, uq.y};
  float x[4];
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    x[2 * q] = valid ? f16r(gelu_tanh(h2f(gw[q] & 0xFFFFu)) * h2f(uw[q] & 0xFFFFu)) : 0.0f;
    x[2 * q + 1] = valid ? f16r(gelu_tanh(h2f(gw[q] >> 16)) * h2f(uw[q] >> 16)) : 0.0f;
  }
  if (valid && act)
    *reinterpret_cast<uint2*>(act + row * F + k0) =
        make_uint2(static_cast<uint32_t>(f2h(x[0])) | (static_cast<uint32_t>(f2h(x[1])) << 16),
                   static_cast<uint32_t>(f2h(x[2])) | (static_cast<uint32_t>(f2h(x[3])) << 16));
  rq_row4<16>(x, row, valid, o, xch, red);
}

// GATED: a = fp16(gelu_tanh(gate) up) from gu = [gate | up] (fp16 [M][2F]);
// otherwise a = fp16(gelu_tanh(u)) from u (fp16 [M][F]).  Then rotate +
// quantize a.
template <int C, bool GATED>
__global__ __launch_bounds__(256) void gelu_rq_kernel(const uint16_t* __restrict__ gu, uint16_t* __restrict__ act,
                                                      int64_t M, int F, RQOut o) {
  extern __shared__ float lds[];
  __shared__ float red[4];
  const rqd::RowMap m = rqd::row_map(o.logT, M);
  float v[C][8];
  const int64_t ld = GATED ? 2 * static_cast<int64_t>(F) : F;
  const uint16_t* gr = gu + (m.valid ? m.row : 0) * ld;
  // Every chunk's loads first (one round trip), then the arithmetic.
  uint4 graw[C], uraw[C];
#pragma unroll
  for (int c = 0; c < C; ++c) {
    const int k = rqd::chan(m, c, 0);
    graw[c] = *reinterpret_cast<const uint4*>(gr + k);
    if (GATED) uraw[c] = *reinterpret_cast<const uint4*>(gr + F + k);
  }
#pragma unroll
  for (int c = 0; c < C; ++c) {
    const uint32_t gw[4] = {graw[c].x, graw[c].y, graw[c].z, graw[c].w};
    float up[8] = {1, 1, 1, 1, 1, 1, 1, 1};
    if (GATED) {
      const uint32_t uw[4] = {uraw[c].x, uraw[c].y, uraw[c].z, uraw[c].w};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        up[2 * q] = h2f(uw[q] & 0xFFFFu);
        up[2 * q + 1] = h2f(uw[q] >> 16);
      }
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      v[c][2 * q] = f16r(gelu_tanh(h2f(gw[q] & 0xFFFFu)) * up[2 * q]);
      v[c][2 * q + 1] = f16r(gelu_tanh(h2f(gw[q] >> 16)) * up[2 * q + 1]);
    }
    if (!m.valid) {
#pragma unroll
      for (int j = 0; j < 8; ++j) v[c][j] = 0.0f;
    }
  }
#pragma unroll
  for (int c = 0; c < C; ++c)
    if (m.valid && act) store8_f16(act + m.row * F + rqd::chan(m, c, 0), v[c]);
  rqd::rq_core<C>(v, m, F, o.logb, o.s_t, o.s_over_sqrtb, lds, red, o.xq, o.xs, nullptr, o.tiled, o.sdelta);
}

struct AttnArgs {
  const uint16_t* q; int64_t q_ld;                      // [B*S][..], head h at column h*hd
  const uint16_t* k_pre; const uint16_t* v_pre; int P;  // [B][P][pre_ld] (P may be 0)
  int64_t pre_ld;
  const uint16_t* k_own; const uint16_t* v_own; int64_t own_ld; int own_keys;  // [B*S][..]
  // Split partials: the split's normalized output o / l in fp16 (a convex
  // combination of value rows, so it cannot overflow) and (m, l) in fp32.
  uint16_t* part_o; float* part_ml;                     // [B*H][nsplit][S][hd], [B*H][nsplit][S][2]
  uint16_t* out; int64_t out_ld;
  int S, H, hd, D, nsplit;
  float scale;
  int direct;  // one split: write the normalized fp16 output to `out` instead of partials
};

typedef _Float16 v8h __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));

// One (sample b, head h, split of KS keys, KS a multiple of 32) on the fp16
// matrix cores (v_mfma_f32_16x16x32_f16), ceil(S / 16) waves.  Wave w owns
// query rows 16w .. 16w+15 (head_dim a multiple of 16; the q.k contraction is
// padded with zeros to a multiple of 32).  Both products are taken transposed,
// so that the probabilities never leave the registers:
//   S^T = K Q^T (KS x 16, fp32), scaled: lane l holds query l % 16 against
//     keys 16 nb + 4 (l / 16) + e (block nb, element e);
//   split maximum m and sum l of each query: 16 values in the lane, then the
//     four lanes l % 16 + 16 g;
//   P^T = exp(S^T - m) in fp16 is directly the B operand of
//   O^T = V^T P^T (hd x 16, fp32), V^T staged in LDS: the contraction index
//     k = 8 g + j of a 32-key step s stands for key 32 s + 4 g + j (j < 4) or
//     32 s + 16 + 4 g + j - 4 (j >= 4), the same keys in both operands (a
//     sum over keys does not depend on their order);
//   lane l then holds dims 16 nb + 4 (l / 16) .. + 3 of query l % 16: one
//     8-byte store of fp16(O / l) per dim block.
// The normalized O / l (fp16), m and l go to the workspace; combine_rq_kernel
// merges the splits with weights e^{m_s - m} l_s.
// MFMA operand layout used (the same k order for both operands): lane l holds
// row / column l % 16 and the 8 k values 8 * (l / 16) .. + 7 of a 32-wide k
// step; the 16 x 16 fp32 result has row 4 * (l / 16) + e, column l % 16 in
// element e.  WAVES = ceil(S / 16) waves; HD = head_dim when it is one of the
// compiled sizes (the loops then unroll completely), 0 otherwise (a.hd at run
// time).
//
// The split's K and V blocks are read from global memory once per workgroup
// (every wave needs all of K): K in 16-byte pieces along its rows (a wave
// reads whole rows) into LDS as [key][dim]; V as pairs of keys (2j, 2j + 1)
// by 8 dims, written to V^T [dim][key] as 4-byte key pairs.  Keys past the
// split and dims past head_dim are staged as zeros.
// Position of key j of a split in a V^T row.  Within each 32-key step the
// keys are stored in the order the O^T = V^T P^T operand of a lane takes them
// (keys 4 g .. 4 g + 3, then 16 + 4 g .. 16 + 4 g + 3, for g = 0 .. 3), so a
// lane's 8 keys are one 16-byte LDS read; keys j, j + 1 with j even stay
// adjacent.
__device__ __forceinline__ int vt_pos(int j) {
  const int jj = j & 31;
  return (j & ~31) + 8 * ((jj & 15) >> 2) + 4 * (jj >> 4) + (jj & 3);
}

template <int WAVES, int HD, int KS>
__global__ __launch_bounds__(64 * WAVES) void attn_partial_kernel(AttnArgs a) {
  static_assert(KS % 32 == 0, "keys per split");
  constexpr int NT = 64 * WAVES;
  constexpr int PAD = KS + 8;            // padded row (halves): 16-byte reads of 16 rows hit distinct banks
  constexpr int HDL = HD > 0 ? HD : kMaxHeadDim;
  constexpr int KPAD = HDL + 8;          // padded K row (halves), likewise
  constexpr int C8 = HDL / 8;            // 8-dim pieces per row
  // LDS sized for this instance (one wave and 48 dims need 16 KB, so many
  // workgroups share a CU).
  __shared__ __attribute__((aligned(16))) uint16_t sVt[HDL][PAD];  // V^T [dim][key]
  __shared__ __attribute__((aligned(16))) uint16_t sK[KS][KPAD];    // K [key][dim]

  const int bh = blockIdx.x, split = blockIdx.y;
  const int b = bh / a.H, h = bh % a.H;
  const int tid = threadIdx.x;
  const int lane = tid & 63, w = tid >> 6;
  const int n_keys = a.P + a.own_keys;
  const int k0 = split * KS;
  const int nk = min(KS, n_keys - k0);
  const int hd = HD > 0 ? HD : a.hd;

  __builtin_assume(tid < NT);
  // Row base of key j of this split: the first P keys are prefix rows, the
  // rest the sample's own rows.  Both candidate addresses are formed in full
  // and the per-lane choice selects between them (a select between two
  // argument fields would become a per-lane load from the selected argument
  // address, in front of every K / V load).
  const uint16_t* const k_pre = a.k_pre;
  const uint16_t* const v_pre = a.v_pre;
  const uint16_t* const k_own = a.k_own;
  const uint16_t* const v_own = a.v_own;
  const int64_t pre_ld = a.pre_ld, own_ld = a.own_ld;
  const int P = a.P, own_keys = a.own_keys;
  auto key_row = [&](int j, const uint16_t* pre_base, const uint16_t* own_base) -> const uint16_t* {
    const int key = k0 + j;
    const uint16_t* pre_p = pre_base + (static_cast<int64_t>(b) * P + key) * pre_ld + h * hd;
    const uint16_t* own_p = own_base + (static_cast<int64_t>(b) * own_keys + (key - P)) * own_ld + h * hd;
    return key < P ? pre_p : own_p;
  };

  // Every global load of the workgroup is issued before the first LDS write
  // or MFMA.  Loads are branch-free: an out-of-range key, query row or head
  // dimension reads a clamped valid address, and its value is replaced by
  // zero where it is staged or used (never by overwriting a register a load
  // is still filling, which would stall on that load).
  // K: piece p = tid + NT i is key p / C8, dims 8 (p % C8) .. + 7.
  constexpr int KIT = (KS * C8 + NT - 1) / NT;
  uint4 kraw[KIT];
#pragma unroll
  for (int i = 0; i < KIT; ++i) {
    const int p = tid + NT * i;
    const int j = p / C8, c8 = (p % C8) * 8;
    const bool ok = p < KS * C8 && j < nk && c8 < hd;
    kraw[i] = *reinterpret_cast<const uint4*>(key_row(ok ? j : 0, k_pre, k_own) + (ok ? c8 : 0));
  }
  // V: unit u = tid + NT i is keys 2 (u % (KS/2)) + {0, 1}, dims 8 (u / (KS/2)) .. + 7.
  constexpr int VIT = (KS / 2 * C8 + NT - 1) / NT;
  uint4 vraw[VIT][2];
#pragma unroll
  for (int i = 0; i < VIT; ++i) {
    const int u = tid + NT * i;
    const int j = 2 * (u % (KS / 2)), c8 = (u / (KS / 2)) * 8;
    const bool ok = u < KS / 2 * C8 && c8 < hd;
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const bool oke = ok && j + e < nk;
      vraw[i][e] = *reinterpret_cast<const uint4*>(key_row(oke ? j + e : 0, v_pre, v_own) + (ok ? c8 : 0));
    }
  }
  // Q (this wave's 16 rows).
  const int qrow = 16 * w + (lane & 15);
  const bool qok = qrow < a.S;
  const int kq = 8 * (lane >> 4);
  const int nkk = (hd + 31) / 32;  // 32-wide k steps over the head dimension (zero-padded)
  constexpr int KKMAX = HD > 0 ? (HD + 31) / 32 : kMaxHeadDim / 32;
  const uint16_t* qp = a.q + (static_cast<int64_t>(b) * a.S + (qok ? qrow : 0)) * a.q_ld + h * hd;
  v8h qraw[KKMAX];
  bool dok[KKMAX];
#pragma unroll
  for (int kk = 0; kk < KKMAX; ++kk) {
    // hd % 8 == 0: a chunk of 8 dims is wholly inside or outside the head.
    dok[kk] = kk < nkk && kk * 32 + kq < hd;
    qraw[kk] = *reinterpret_cast<const v8h*>(qp + (dok[kk] ? kk * 32 + kq : 0));
  }

  // Stage K [key][dim] and V^T [dim][key] in LDS.
#pragma unroll
  for (int i = 0; i < KIT; ++i) {
    const int p = tid + NT * i;
    const int j = p / C8, c8 = (p % C8) * 8;
    if (p < KS * C8) {
      const bool ok = j < nk && c8 < hd;
      const uint4 v = ok ? kraw[i] : make_uint4(0, 0, 0, 0);
      uint32_t* d = reinterpret_cast<uint32_t*>(&sK[j][c8]);
      d[0] = v.x;
      d[1] = v.y;
      d[2] = v.z;
      d[3] = v.w;
    }
  }
#pragma unroll
  for (int i = 0; i < VIT; ++i) {
    const int u = tid + NT * i;
    const int j = 2 * (u % (KS / 2)), c8 = (u / (KS / 2)) * 8;
    if (u < KS / 2 * C8) {
      const bool ok0 = c8 < hd && j < nk, ok1 = c8 < hd && j + 1 < nk;
      const uint32_t w0[4] = {ok0 ? vraw[i][0].x : 0u, ok0 ? vraw[i][0].y : 0u, ok0 ? vraw[i][0].z : 0u,
                              ok0 ? vraw[i][0].w : 0u};
      const uint32_t w1[4] = {ok1 ? vraw[i][1].x : 0u, ok1 ? vraw[i][1].y : 0u, ok1 ? vraw[i][1].z : 0u,
                              ok1 ? vraw[i][1].w : 0u};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        // dims c8 + 2q (low halves) and c8 + 2q + 1 (high halves) of keys j, j + 1
        *reinterpret_cast<uint32_t*>(&sVt[c8 + 2 * q][vt_pos(j)]) = (w0[q] & 0xFFFFu) | (w1[q] << 16);
        *reinterpret_cast<uint32_t*>(&sVt[c8 + 2 * q + 1][vt_pos(j)]) = (w0[q] >> 16) | (w1[q] & 0xFFFF0000u);
      }
    }
  }
  v8h qa[KKMAX];
#pragma unroll
  for (int kk = 0; kk < KKMAX; ++kk) qa[kk] = (dok[kk] && qok) ? qraw[kk] : v8h{};
  __syncthreads();

  // S^T = K Q^T: block nb of 16 keys against this wave's 16 queries.
  const int g = lane >> 4;
  v4f sc[KS / 16];
#pragma unroll
  for (int nb = 0; nb < KS / 16; ++nb) {
    sc[nb] = v4f{0, 0, 0, 0};
#pragma unroll
    for (int kk = 0; kk < KKMAX; ++kk)
      if (kk < nkk) {
        const v8h ka = *reinterpret_cast<const v8h*>(&sK[nb * 16 + (lane & 15)][dok[kk] ? kk * 32 + kq : 0]);
        sc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ka, qa[kk], sc[nb], 0, 0, 0);
      }
  }

  // Softmax statistics of query lane % 16: the lane's 16 keys, then the four
  // lanes of the same query (lane bits 4 and 5).
  float m_ = -INFINITY;
#pragma unroll
  for (int nb = 0; nb < KS / 16; ++nb)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int j = nb * 16 + 4 * g + e;
      const float v = j < nk ? sc[nb][e] * a.scale : -INFINITY;
      sc[nb][e] = v;
      m_ = fmaxf(m_, v);
    }
  m_ = fmaxf(m_, rqd::lane_xor_far<16>(m_));
  m_ = fmaxf(m_, rqd::lane_xor_far<32>(m_));
  float l_ = 0.0f;
  v8h pb[KS / 32];  // P^T fragments, one per 32-key step
#pragma unroll
  for (int st = 0; st < KS / 32; ++st)
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float p = __expf(sc[2 * st + (j >> 2)][j & 3] - m_);
      l_ += p;
      pb[st][j] = static_cast<_Float16>(p);
    }
  l_ += rqd::lane_xor_far<16>(l_);
  l_ += rqd::lane_xor_far<32>(l_);

  // O^T = V^T P^T, 16 dims x 16 queries per block.  With a single split
  // (a.direct) the row is complete: o / l, rounded to fp16, goes straight to
  // the head's columns of `out` (the same fp32 operations as the merge of one
  // split).
  const int q = 16 * w + (lane & 15);
  const bool qst = q < a.S;
  const int64_t po_off = ((static_cast<int64_t>(bh) * a.nsplit + split) * a.S + (qst ? q : 0)) * hd + 4 * g;
  const int64_t out_off = (static_cast<int64_t>(b) * a.S + (qst ? q : 0)) * a.out_ld + h * hd + 4 * g;
  const float inv = 1.0f / l_;
  constexpr int NBD = HDL / 16;
#pragma unroll
  for (int nb = 0; nb < NBD; ++nb) {
    if (nb * 16 < hd) {
      v4f o = v4f{0, 0, 0, 0};
#pragma unroll
      for (int st = 0; st < KS / 32; ++st) {
        const v8h va = *reinterpret_cast<const v8h*>(&sVt[nb * 16 + (lane & 15)][st * 32 + 8 * g]);
        o = __builtin_amdgcn_mfma_f32_16x16x32_f16(va, pb[st], o, 0, 0, 0);
      }
      if (qst) {
        if (a.direct)
          *reinterpret_cast<uint2*>(a.out + out_off + nb * 16) =
              make_uint2(static_cast<uint32_t>(f2h(o[0] * inv)) | (static_cast<uint32_t>(f2h(o[1] * inv)) << 16),
                         static_cast<uint32_t>(f2h(o[2] * inv)) | (static_cast<uint32_t>(f2h(o[3] * inv)) << 16));
        else
          *reinterpret_cast<uint2*>(a.part_o + po_off + nb * 16) =
              make_uint2(static_cast<uint32_t>(f2h(o[0] * inv)) | (static_cast<uint32_t>(f2h(o[1] * inv)) << 16),
                         static_cast<uint32_t>(f2h(o[2] * inv)) | (static_cast<uint32_t>(f2h(o[3] * inv)) << 16));
      }
    }
  }
  if (a.direct) return;
  if (g == 0 && qst) {
    float* ml = a.part_ml + ((static_cast<int64_t>(bh) * a.nsplit + split) * a.S + q) * 2;
    *reinterpret_cast<float2*>(ml) = make_float2(m_, l_);
  }
}

// Conditioning k|v rows [B*P][2D] (head h at columns h*hd of each half)
// rewritten head-major, [B][H][2][P][hd], so that the cross-attention of one
// (sample, head) reads its keys and values as two contiguous blocks.  One
// thread per 16-byte piece (hd % 8 == 0).
__global__ __launch_bounds__(256) void kv_head_major_kernel(const uint16_t* __restrict__ rows,
                                                            uint16_t* __restrict__ hm, int64_t B, int P, int H,
                                                            int hd) {
  const int64_t D = static_cast<int64_t>(H) * hd;
  const int64_t pieces = B * P * 2 * D / 8;
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= pieces) return;
  const int64_t row = i / (2 * D / 8), c = (i % (2 * D / 8)) * 8;  // row b * P + p, column c of 2D
  const int64_t b = row / P, p = row % P;
  const int64_t half = c / D, h = (c % D) / hd, d = (c % D) % hd;
  const uint4 v = *reinterpret_cast<const uint4*>(rows + row * 2 * D + c);
  *reinterpret_cast<uint4*>(hm + (((b * H + h) * 2 + half) * P + p) * hd + d) = v;
}

// Cross-attention of one (sample b, head h) over all P conditioning keys,
// read head-major (K then V blocks of P x hd).  The keys are taken 64 at a
// time with the transposed matrix-core steps of attn_partial_kernel (S^T =
// K Q^T, then O^T = V^T P^T with P^T in registers; K fragments are loaded
// straight from global memory in the A operand layout), and the splits are
// merged on the fly (running maximum m, sum l and output O per query, a
// lane's own: rescaled by e^{m_old - m_new}); the normalized output is
// written as fp16 to its head's columns of `out`.  WAVES = ceil(S / 16).
template <int WAVES, int HD>
__global__ __launch_bounds__(64 * WAVES) void attn_cross_kernel(const uint16_t* __restrict__ q, int64_t q_ld,
                                                                const uint16_t* __restrict__ kvh, int P, int S,
                                                                int H, float scale, uint16_t* __restrict__ out,
                                                                int64_t out_ld) {
  constexpr int KS = kAttnKS;
  constexpr int PAD = KS + 8;
  static_assert(HD % 16 == 0 && HD <= kMaxHeadDim, "head_dim");
  constexpr int KK = (HD + 31) / 32;               // 32-wide k steps of q.k (zero-padded)
  constexpr int VIT = (HD + 8 * WAVES - 1) / (8 * WAVES);
  __shared__ __attribute__((aligned(16))) uint16_t sVt[HD][PAD];
  const int bh = blockIdx.x;
  const int b = bh / H, h = bh % H;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  __builtin_assume(tid < 64 * WAVES);
  const uint16_t* kb_base = kvh + static_cast<int64_t>(bh) * 2 * P * HD;
  const uint16_t* vb_base = kb_base + static_cast<int64_t>(P) * HD;
  const int g = lane >> 4;
  const int qrow = 16 * w + (lane & 15);
  const bool qok = qrow < S;
  const int kq = 8 * g;
  const uint16_t* qp = q + (static_cast<int64_t>(b) * S + (qok ? qrow : 0)) * q_ld + h * HD;
  v8h qa[KK];
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) {
    const bool dok = kk * 32 + kq < HD;
    const v8h raw = *reinterpret_cast<const v8h*>(qp + (dok ? kk * 32 + kq : 0));
    qa[kk] = (dok && qok) ? raw : v8h{};
  }
  // Running statistics of query lane % 16 and O^T: o[nb][e] = dim 16 nb + 4 g + e.
  float m = -INFINITY, l = 0.0f;
  v4f o[HD / 16];
#pragma unroll
  for (int nb = 0; nb < HD / 16; ++nb) o[nb] = v4f{0, 0, 0, 0};

  const int nsplit = (P + KS - 1) / KS;
  for (int sp = 0; sp < nsplit; ++sp) {
    const int k0 = sp * KS;
    const int nk = min(KS, P - k0);
    // Loads first (clamped rows; values of keys past P are masked at use).
    const int vj = tid & 63;
    const bool vjok = vj < nk;
    uint4 vraw[VIT];
    {
      const uint16_t* vp = vb_base + static_cast<int64_t>(k0 + (vjok ? vj : 0)) * HD;
#pragma unroll
      for (int i = 0; i < VIT; ++i) {
        const int d8 = w * 8 + i * 8 * WAVES;
        vraw[i] = *reinterpret_cast<const uint4*>(vp + (d8 < HD ? d8 : 0));
      }
    }
    // K fragments (A operand): key 16 nb + lane % 16, dims 32 kk + 8 g .. + 7.
    v8h kraw[KK][KS / 16];
    bool kok[KS / 16];
#pragma unroll
    for (int nb = 0; nb < KS / 16; ++nb) {
      const int j = nb * 16 + (lane & 15);
      kok[nb] = j < nk;
      const uint16_t* kp = kb_base + static_cast<int64_t>(k0 + (kok[nb] ? j : 0)) * HD;
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) {
        const bool dok = kk * 32 + kq < HD;
        kraw[kk][nb] = *reinterpret_cast<const v8h*>(kp + (dok ? kk * 32 + kq : 0));
      }
    }
    __syncthreads();  // the previous split's V^T reads are done
#pragma unroll
    for (int i = 0; i < VIT; ++i) {
      const int d8 = w * 8 + i * 8 * WAVES;
      if (d8 < HD) {
        const uint32_t wv[4] = {vjok ? vraw[i].x : 0u, vjok ? vraw[i].y : 0u, vjok ? vraw[i].z : 0u,
                                vjok ? vraw[i].w : 0u};
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          sVt[d8 + 2 * t][vt_pos(vj)] = static_cast<uint16_t>(wv[t] & 0xFFFFu);
          sVt[d8 + 2 * t + 1][vt_pos(vj)] = static_cast<uint16_t>(wv[t] >> 16);
        }
      }
    }
    // S^T = K Q^T: sc[nb][e] = key 16 nb + 4 g + e against query lane % 16.
    v4f sc[KS / 16];
#pragma unroll
    for (int nb = 0; nb < KS / 16; ++nb) {
      sc[nb] = v4f{0, 0, 0, 0};
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) {
        const bool dok = kk * 32 + kq < HD;
        const v8h ka = (dok && kok[nb]) ? kraw[kk][nb] : v8h{};
        sc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ka, qa[kk], sc[nb], 0, 0, 0);
      }
    }
    // Running softmax of the lane's query: its 16 keys, then lane bits 4, 5.
    float mx = -INFINITY;
#pragma unroll
    for (int nb = 0; nb < KS / 16; ++nb)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int j = nb * 16 + 4 * g + e;
        const float v = j < nk ? sc[nb][e] * scale : -INFINITY;
        sc[nb][e] = v;
        mx = fmaxf(mx, v);
      }
    mx = fmaxf(mx, rqd::lane_xor_far<16>(mx));
    mx = fmaxf(mx, rqd::lane_xor_far<32>(mx));
    const float mn = fmaxf(m, mx);
    const float alpha = __expf(m - mn);  // 0 on the first split (m = -inf)
    float sum = 0.0f;
    v8h pb[KS / 32];
#pragma unroll
    for (int st = 0; st < KS / 32; ++st)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float pv = __expf(sc[2 * st + (j >> 2)][j & 3] - mn);
        sum += pv;
        pb[st][j] = static_cast<_Float16>(pv);
      }
    sum += rqd::lane_xor_far<16>(sum);
    sum += rqd::lane_xor_far<32>(sum);
    l = l * alpha + sum;
    m = mn;
    __syncthreads();  // V^T staged
#pragma unroll
    for (int nb = 0; nb < HD / 16; ++nb) {
      o[nb] *= alpha;
#pragma unroll
      for (int st = 0; st < KS / 32; ++st) {
        const v8h va = *reinterpret_cast<const v8h*>(&sVt[nb * 16 + (lane & 15)][st * 32 + 8 * g]);
        o[nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(va, pb[st], o[nb], 0, 0, 0);
      }
    }
  }
  if (!qok) return;
  const float inv = 1.0f / l;
  uint16_t* orow = out + (static_cast<int64_t>(b) * S + qrow) * out_ld + h * HD + 4 * g;
#pragma unroll
  for (int nb = 0; nb < HD / 16; ++nb)
    *reinterpret_cast<uint2*>(orow + nb * 16) =
        make_uint2(static_cast<uint32_t>(f2h(o[nb][0] * inv)) | (static_cast<uint32_t>(f2h(o[nb][1] * inv)) << 16),
                   static_cast<uint32_t>(f2h(o[nb][2] * inv)) | (static_cast<uint32_t>(f2h(o[nb][3] * inv)) << 16));
}

// Token row (b, s): out = sum_s e^{m_s - M} o_s / sum_s e^{m_s - M} l_s per
// head, rounded to fp16, then rotate + quantize the row.
template <int C>
__global__ __launch_bounds__(256) void combine_rq_kernel(AttnArgs a, int64_t M, RQOut o) {
  extern __shared__ float lds[];
  __shared__ float red[4];
  const rqd::RowMap m = rqd::row_map(o.logT, M);
  float v[C][8];
  const int64_t row = m.valid ? m.row : 0;
  const int b = static_cast<int>(row / a.S), q = static_cast<int>(row % a.S);
#pragma unroll
  for (int c = 0; c < C; ++c) {
    const int k = rqd::chan(m, c, 0);
    const int h = k / a.hd, d = k - h * a.hd;
    const int64_t bh = static_cast<int64_t>(b) * a.H + h;
    const float* ml = a.part_ml + bh * a.nsplit * a.S * 2 + 2 * q;
    const uint16_t* po = a.part_o + bh * a.nsplit * a.S * a.hd + static_cast<int64_t>(q) * a.hd + d;
    // All split statistics first (independent loads), then the weighted values
    // in groups of 8 splits (weight e^{m_s - m} l_s on the normalized o_s).
    float mv[kMaxSplits], lv[kMaxSplits];
#pragma unroll
    for (int s = 0; s < kMaxSplits; ++s) {
      mv[s] = -INFINITY;
      lv[s] = 0.0f;
      if (s < a.nsplit) {
        const float2 t = *reinterpret_cast<const float2*>(ml + s * a.S * 2);
        mv[s] = t.x;
        lv[s] = t.y;
      }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int s = 0; s < kMaxSplits; ++s) mx = fmaxf(mx, mv[s]);
    float den = 0.0f;
    float num[8] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
    for (int s0 = 0; s0 < kMaxSplits; s0 += 8) {
      uint4 pr[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        pr[u] = make_uint4(0, 0, 0, 0);
        if (s0 + u < a.nsplit) pr[u] = *reinterpret_cast<const uint4*>(po + static_cast<int64_t>(s0 + u) * a.S * a.hd);
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const float w = s0 + u < a.nsplit ? __expf(mv[s0 + u] - mx) * lv[s0 + u] : 0.0f;
        den += w;
        const uint32_t pw[4] = {pr[u].x, pr[u].y, pr[u].z, pr[u].w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          num[2 * j] = fmaf(w, h2f(pw[j] & 0xFFFFu), num[2 * j]);
          num[2 * j + 1] = fmaf(w, h2f(pw[j] >> 16), num[2 * j + 1]);
        }
      }
    }
    const float inv = 1.0f / den;
#pragma unroll
    for (int j = 0; j < 8; ++j) v[c][j] = m.valid ? f16r(num[j] * inv) : 0.0f;
    if (m.valid && a.out) store8_f16(a.out + m.row * a.out_ld + k, v[c]);
  }
  rqd::rq_core<C>(v, m, a.D, o.logb, o.s_t, o.s_over_sqrtb, lds, red, o.xq, o.xs, nullptr, o.tiled, o.sdelta);
}

// combine_rq_kernel for 1024-channel rows with few rows (the Pi-0.5 action
// tokens, Hadamard block = the row; per-token or static steps): 256 threads per row,
// 4 consecutive channels (one head's) per thread; every split's statistics
// and values are loaded before the first use (split indices past nsplit
// reread the last split and get weight 0), then rq1024_row.
__global__ __launch_bounds__(256) void combine_rq1024_kernel(AttnArgs a, int64_t M, RQOut o) {
  __shared__ __attribute__((aligned(16))) float xch[1024];
  __shared__ float red[4];
  const int t = threadIdx.x;
  const int64_t row = blockIdx.x;
  const bool valid = row < M;
  const int64_t rr = valid ? row : 0;
  const int b = static_cast<int>(rr / a.S), q = static_cast<int>(rr % a.S);
  const int k0 = 4 * t;
  const int h = k0 / a.hd, d = k0 - h * a.hd;
  const int64_t bh = static_cast<int64_t>(b) * a.H + h;
  const float* ml = a.part_ml + bh * a.nsplit * a.S * 2 + 2 * q;
  const uint16_t* po = a.part_o + bh * a.nsplit * a.S * a.hd + static_cast<int64_t>(q) * a.hd + d;
  const int slast = a.nsplit - 1;
  float2 st[kMaxSplits];
  uint2 pv[kMaxSplits];
#pragma unroll
  for (int s = 0; s < kMaxSplits; ++s) {
    const int sc = min(s, slast);
    st[s] = *reinterpret_cast<const float2*>(ml + static_cast<int64_t>(sc) * a.S * 2);
    pv[s] = *reinterpret_cast<const uint2*>(po + static_cast<int64_t>(sc) * a.S * a.hd);
  }
  float mx = -INFINITY;
#pragma unroll
  for (int s = 0; s < kMaxSplits; ++s) mx = fmaxf(mx, s < a.nsplit ? st[s].x : -INFINITY);
  float den = 0.0f;
  float num[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int s = 0; s < kMaxSplits; ++s) {
    const float wgt = s < a.nsplit ? __expf(st[s].x - mx) * st[s].y : 0.0f;  // e^{m_s - m} l_s
    den += wgt;
    num[0] = fmaf(wgt, h2f(pv[s].x & 0xFFFFu), num[0]);
    num[1] = fmaf(wgt, h2f(pv[s].x >> 16), num[1]);
    num[2] = fmaf(wgt, h2f(pv[s].y & 0xFFFFu), num[2]);
    num[3] = fmaf(wgt, h2f(pv[s].y >> 16), num[3]);
  }
  const float inv = 1.0f / den;
  float x[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) x[j] = valid ? f16r(num[j] * inv) : 0.0f;
  if (valid && a.out)
    *reinterpret_cast<uint2*>(a.out + row * a.out_ld + k0) =
        make_uint2(static_cast<uint32_t>(f2h(x[0])) | (static_cast<uint32_t>(f2h(x[1])) << 16),
                   static_cast<uint32_t>(f2h(x[2])) | (static_cast<uint32_t>(f2h(x[3])) << 16));
  rq1024_row(x, row, valid, o, xch, red);
}

__device__ __forceinline__ float wave_sum(float v) {
  return rqd::wave_sum_xor(v);
}

// x[m][:] += dt * (fp16(norm(r[m]) g_f) W_out^T + b_out), norm = RMS norm or
// (LN) layer norm.  R (1 or 4) rows per 256-thread workgroup: wave w < R
// normalizes row m0 + w into LDS (reductions inside the wave), then thread t
// computes the partial dot products of output a = t / 8 over the d-slice
// t % 8 for the R rows (16-byte W_out loads shared by the rows), reduced over
// the 8 slices with lane shuffles (outputs in groups of 32).  D % 64 == 0.
template <bool LN, int R>
__global__ __launch_bounds__(256) void final_kernel(const float* __restrict__ r, const uint16_t* __restrict__ g_f,
                                                    const uint16_t* __restrict__ w_out,
                                                    const uint16_t* __restrict__ b_out, float* __restrict__ x,
                                                    int64_t M, int D, int A, float dt) {
  extern __shared__ float sh[];  // [R][D] normalized rows
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t m0 = static_cast<int64_t>(blockIdx.x) * R;
  // Thread t takes output a = t / 8 over the dims 8 (t % 8) + 64 i.  With at
  // most 32 outputs and D <= 64 NW its W_out slice is loaded into registers
  // first, so that the loads overlap the norms.
  constexpr int NW = 24;
  const int sl = threadIdx.x & 7;
  const bool pre = A <= 32 && D <= 64 * NW;
  uint4 wreg[NW];
  if (pre) {
    const int a_idx = threadIdx.x >> 3;
    const uint16_t* wr = w_out + static_cast<int64_t>(a_idx < A ? a_idx : 0) * D;
#pragma unroll
    for (int i = 0; i < NW; ++i) {
      const int d = sl * 8 + 64 * i;
      wreg[i] = d < D ? *reinterpret_cast<const uint4*>(wr + d) : make_uint4(0, 0, 0, 0);
    }
  }
  if (w < R) {
    const int64_t m = m0 + w;
    const bool ok = m < M;
    const float* rr = r + (ok ? m : 0) * D;
    float* row = sh + w * D;
    // Rows of up to 2048 channels stay in registers (one batch of loads,
    // compile-time indices); wider rows are read again for each pass.
    constexpr int CR = 8;
    float s1 = 0.0f, ss = 0.0f, mu = 0.0f, inv = 0.0f;
    if (D <= 256 * CR) {
      float4 rv[CR];
#pragma unroll
      for (int c = 0; c < CR; ++c) {
        const int d = lane * 4 + 256 * c;
        rv[c] = d < D ? *reinterpret_cast<const float4*>(rr + d) : make_float4(0, 0, 0, 0);
        s1 += (rv[c].x + rv[c].y) + (rv[c].z + rv[c].w);
      }
      mu = LN ? wave_sum(s1) / static_cast<float>(D) : 0.0f;
#pragma unroll
      for (int c = 0; c < CR; ++c) {
        const int d = lane * 4 + 256 * c;
        if (d < D) {
          const float e0 = rv[c].x - mu, e1 = rv[c].y - mu, e2 = rv[c].z - mu, e3 = rv[c].w - mu;
          ss = fmaf(e0, e0, fmaf(e1, e1, fmaf(e2, e2, fmaf(e3, e3, ss))));
        }
      }
      inv = 1.0f / sqrtf(wave_sum(ss) / static_cast<float>(D) + kEps);
#pragma unroll
      for (int c = 0; c < CR; ++c) {
        const int d = lane * 4 + 256 * c;
        if (d < D) {
          const uint2 gq = *reinterpret_cast<const uint2*>(g_f + d);
          row[d] = f16r((rv[c].x - mu) * inv * h2f(gq.x & 0xFFFFu));
          row[d + 1] = f16r((rv[c].y - mu) * inv * h2f(gq.x >> 16));
          row[d + 2] = f16r((rv[c].z - mu) * inv * h2f(gq.y & 0xFFFFu));
          row[d + 3] = f16r((rv[c].w - mu) * inv * h2f(gq.y >> 16));
        }
      }
    } else {
      for (int d = lane * 4; d < D; d += 256) {
        const float4 v = *reinterpret_cast<const float4*>(rr + d);
        s1 += (v.x + v.y) + (v.z + v.w);
      }
      mu = LN ? wave_sum(s1) / static_cast<float>(D) : 0.0f;
      for (int d = lane * 4; d < D; d += 256) {
        const float4 v = *reinterpret_cast<const float4*>(rr + d);
        const float e0 = v.x - mu, e1 = v.y - mu, e2 = v.z - mu, e3 = v.w - mu;
        ss = fmaf(e0, e0, fmaf(e1, e1, fmaf(e2, e2, fmaf(e3, e3, ss))));
      }
      inv = 1.0f / sqrtf(wave_sum(ss) / static_cast<float>(D) + kEps);
      for (int d = lane * 4; d < D; d += 256) {
        const float4 v = *reinterpret_cast<const float4*>(rr + d);
        const uint2 gq = *reinterpret_cast<const uint2*>(g_f + d);
        row[d] = f16r((v.x - mu) * inv * h2f(gq.x & 0xFFFFu));
        row[d + 1] = f16r((v.y - mu) * inv * h2f(gq.x >> 16));
        row[d + 2] = f16r((v.z - mu) * inv * h2f(gq.y & 0xFFFFu));
        row[d + 3] = f16r((v.w - mu) * inv * h2f(gq.y >> 16));
      }
    }
  }
  __syncthreads();
  // The same sums in the same order on both paths (dims ascending per slice).
  auto accumulate = [&](float (&acc)[R], const float (&wv)[8], int d) {
#pragma unroll
    for (int rr = 0; rr < R; ++rr) {
      const float4 p0 = *reinterpret_cast<const float4*>(sh + rr * D + d);
      const float4 p1 = *reinterpret_cast<const float4*>(sh + rr * D + d + 4);
      acc[rr] = fmaf(p0.x, wv[0], fmaf(p0.y, wv[1], fmaf(p0.z, wv[2], fmaf(p0.w, wv[3], acc[rr]))));
      acc[rr] = fmaf(p1.x, wv[4], fmaf(p1.y, wv[5], fmaf(p1.z, wv[6], fmaf(p1.w, wv[7], acc[rr]))));
    }
  };
  auto finish = [&](float (&acc)[R], int a_idx, bool aok) {
#pragma unroll
    for (int rr = 0; rr < R; ++rr) {
      float v = acc[rr];
      v += rqd::lane_xor<1>(v);
      v += rqd::lane_xor<2>(v);
      v += rqd::lane_xor<4>(v);
      const int64_t m = m0 + rr;
      if (aok && sl == 0 && m < M) x[m * A + a_idx] += dt * (v + h2f(b_out[a_idx]));
    }
  };
  if (pre) {
    const int a_idx = threadIdx.x >> 3;
    float acc[R];
#pragma unroll
    for (int rr = 0; rr < R; ++rr) acc[rr] = 0.0f;
#pragma unroll
    for (int i = 0; i < NW; ++i) {
      const int d = sl * 8 + 64 * i;
      if (d < D) {
        const uint32_t q[4] = {wreg[i].x, wreg[i].y, wreg[i].z, wreg[i].w};
        float wv[8];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          wv[2 * j] = h2f(q[j] & 0xFFFFu);
          wv[2 * j + 1] = h2f(q[j] >> 16);
        }
        accumulate(acc, wv, d);
      }
    }
    finish(acc, a_idx, a_idx < A);
    return;
  }
  for (int a0 = 0; a0 < A; a0 += 32) {
    const int a_idx = a0 + (threadIdx.x >> 3);
    const bool aok = a_idx < A;
    const uint16_t* wr = w_out + static_cast<int64_t>(aok ? a_idx : 0) * D;
    float acc[R];
#pragma unroll
    for (int rr = 0; rr < R; ++rr) acc[rr] = 0.0f;
#pragma unroll 4
    for (int d = sl * 8; d < D; d += 64) {
      float wv[8];
      load8_f16(wr + d, wv);
      accumulate(acc, wv, d);
    }
    finish(acc, a_idx, aok);
  }
}

size_t align256(size_t n) { return (n + 255) & ~static_cast<size_t>(255); }

bool is_gr00t(const oq_dit_config& c) { return c.arch == OQ_DIT_GR00T; }
int n_cross(const oq_dit_config& c) { return is_gr00t(c) ? (c.n_blocks + 1) / 2 : 0; }

struct Layout {
  size_t r, h1, qkv, o, h2, gu, act, xq, xs, part_o, part_ml, ckv, ckvh, skp, skt, total;
  int64_t sk_words, sk_tickets;  // split-K scratch of the row-layout linears (0 with tiled codes)
};

Layout layout_for(const oq_dit_config& c) {
  const int64_t M = static_cast<int64_t>(c.batch) * c.tokens;
  const int64_t D = c.hidden, F = c.mlp;
  const int64_t Kmax = std::max(D, F);
  // Keys per sample: pi attends to [prefix ; own], gr00t to the conditioning
  // tokens (even blocks) or to its own tokens (odd blocks).
  const int keys = is_gr00t(c) ? std::max(c.prefix, c.tokens) : c.prefix + c.tokens;
  const int nsplit = (keys + kAttnSplit - 1) / kAttnSplit;
  const int64_t BH = static_cast<int64_t>(c.batch) * c.n_heads;
  const int64_t MC = is_gr00t(c) ? static_cast<int64_t>(c.batch) * c.prefix : 0;  // conditioning rows
  Layout L;
  size_t off = 0;
  L.r = off; off += align256(M * D * 4);
  L.h1 = off; off += align256(M * D * 2);
  L.qkv = off; off += align256(M * 3 * D * 2);
  L.o = off; off += align256(M * D * 2);
  L.h2 = off; off += align256(M * D * 2);
  L.gu = off; off += align256(M * 2 * F * 2);
  L.act = off; off += align256(M * F * 2);
  L.xq = off; off += align256(std::max(tiled_bytes(M, Kmax), MC * D / 2));
  L.xs = off; off += align256(std::max(M, MC) * 4);
  L.part_o = off; off += align256(BH * nsplit * c.tokens * c.head_dim * 2);
  L.part_ml = off; off += align256(BH * nsplit * c.tokens * 2 * 4);
  // The conditioning k|v: one block's linear output in row layout (staging),
  // and every cross-attention block's values head-major.
  L.ckv = off; off += align256(static_cast<size_t>(n_cross(c) > 0 ? 1 : 0) * MC * 2 * D * 2);
  L.ckvh = off; off += align256(static_cast<size_t>(n_cross(c)) * MC * 2 * D * 2);
  // Split-K scratch of the deep block linears with row-layout codes (M > 64):
  // two int32 partial 64 x 64 tiles for each of up to 512 tiles, and the
  // tiles' arrival tickets (zeroed by oq_dit_set_workspace).
  L.sk_tickets = M > 64 ? 512 : 0;
  L.sk_words = L.sk_tickets * 2 * 64 * 64;
  L.skp = off; off += align256(static_cast<size_t>(L.sk_words) * 4);
  L.skt = off; off += align256(static_cast<size_t>(L.sk_tickets) * 4);
  L.total = off;
  return L;
}

// Thread split of a fused row kernel: as many threads per row as possible (up
// to 256), few channels each, so that the small-M rows spread widely.
bool fused_plan(int64_t K, RQPlan* p) {
  const int64_t nvec = K / 8;
  static const int kChunks[] = {1, 2, 3, 4, 6, 8};
  for (int c : kChunks) {
    if (nvec % c) continue;
    const int64_t T = nvec / c;
    if (!is_pow2(T) || T > 256) continue;
    p->chunks = c;
    p->logT = ilog2(T);
    return true;
  }
  return false;
}

int validate_config(const oq_dit_config* c) {
  if (!c) return OQ_ERR_NULL;
  if (c->arch != OQ_DIT_PI && c->arch != OQ_DIT_GR00T) return OQ_ERR_ARG;
  if (c->n_blocks < 1 || c->steps < 1 || c->batch < 1 || c->tokens < 1 || c->prefix < 0) return OQ_ERR_SHAPE;
  if (c->hidden < 64 || c->hidden % 64 || c->mlp < 64 || c->mlp % 64) return OQ_ERR_SHAPE;
  if (c->hidden > 8192 || c->mlp > 16384) return OQ_ERR_SHAPE;
  if (c->n_heads < 1 || c->head_dim < 16 || c->head_dim > kMaxHeadDim || c->head_dim % 16 ||
      c->n_heads * c->head_dim != c->hidden)
    return OQ_ERR_SHAPE;
  if (c->tokens > kMaxTokens || c->action_dim < 1 || c->action_dim > 256) return OQ_ERR_SHAPE;
  const int keys = c->arch == OQ_DIT_GR00T ? std::max(c->prefix, c->tokens) : c->prefix + c->tokens;
  if (keys > kMaxSplits * kAttnSplit) return OQ_ERR_SHAPE;
  if (c->arch == OQ_DIT_GR00T && c->prefix < 1) return OQ_ERR_SHAPE;
  RQPlan p;
  if (!fused_plan(c->hidden, &p) || !fused_plan(c->mlp, &p)) return OQ_ERR_SHAPE;
  return OQ_OK;
}

int pow2_divisor(int n) { return n & (-n); }

}  // namespace
}  // namespace oq

struct oq_dit_graph {
  float* x;
  int t0, n;
  hipGraphExec_t exec;
  uint64_t last_use;
};

struct oq_dit {
  oq_dit_config cfg;
  oq_dit_weights w;
  std::vector<oq_dit_block> blocks;
  std::vector<float> s_table;
  oq::Layout lay;
  uint8_t* ws = nullptr;
  size_t ws_bytes = 0;
  bool cond_ready = false;    // gr00t: conditioning k|v computed into this workspace
  hipStream_t cap = nullptr;  // capture stream (graphs are replayed on the caller's stream)
  std::vector<oq_dit_graph> graphs;  // at most kMaxGraphs, least recently used dropped
  uint64_t graph_clock = 0;
  bool use_graphs = true;
  bool tiled = false;  // block linears' token codes in the 16-row tiled layout (M <= 64)
  // Static per-step, per-channel steps (null: the per-token quantizer with
  // the scalar step scale): device table [n_blocks][steps][3D + F] and the
  // per-(block, step) folded weights of the four block linears.
  const float* static_delta = nullptr;
  std::vector<oq_qweight> static_w;
};

namespace oq {
namespace {

template <typename T>
T* at(oq_dit* h, size_t off) { return reinterpret_cast<T*>(h->ws + off); }

int n_mod(const oq_dit_config& c) { return is_gr00t(c) ? 2 : 6; }

const uint16_t* mod_ptr(oq_dit* h, int l, int t, int k) {
  const int64_t D = h->cfg.hidden;
  const int nm = n_mod(h->cfg);
  return static_cast<const uint16_t*>(h->w.mod) + ((static_cast<int64_t>(l) * h->cfg.steps + t) * nm + k) * D;
}

RQOut rq_out(oq_dit* h, int64_t K, float s, RQPlan* p, const float* sdelta = nullptr) {
  fused_plan(K, p);
  RQOut o;
  o.sdelta = sdelta;
  if (sdelta) s = 1.0f;  // the static steps replace the token step and its scale
  o.xq = at<uint8_t>(h, h->lay.xq);
  o.xs = at<float>(h, h->lay.xs);
  o.logT = p->logT;
  const int b = pow2_divisor(static_cast<int>(K));
  o.logb = ilog2(b);
  o.s_t = s;
  o.s_over_sqrtb = static_cast<float>(static_cast<double>(s) / std::sqrt(static_cast<double>(b)));
  o.tiled = h->tiled;
  return o;
}

struct FusedLaunch {
  dim3 grid, block;
  size_t lds;
};

FusedLaunch fused_launch(int64_t M, int64_t K, const RQPlan& p) {
  const int T = 1 << p.logT;
  // Few rows (the action tokens): one row per workgroup, so the rows spread
  // over as many CUs as there are rows; else 256-thread workgroups.
  const int threads = T >= 256 || M <= 256 ? T : 256;
  const int rows_per_wg = threads / T;
  FusedLaunch f;
  f.grid = dim3(static_cast<unsigned>((M + rows_per_wg - 1) / rows_per_wg));
  f.block = dim3(threads);
  f.lds = p.logT > 6 ? static_cast<size_t>(rows_per_wg) * K * sizeof(float) : 0;
  return f;
}

// Calls f(std::integral_constant<int, C>) for the chunk count C of a fused
// row plan; false for an unsupported count.
template <typename F>
bool with_chunks(int chunks, F&& f) {
  switch (chunks) {
    case 1: f(std::integral_constant<int, 1>{}); return true;
    case 2: f(std::integral_constant<int, 2>{}); return true;
    case 3: f(std::integral_constant<int, 3>{}); return true;
    case 4: f(std::integral_constant<int, 4>{}); return true;
    case 6: f(std::integral_constant<int, 6>{}); return true;
    case 8: f(std::integral_constant<int, 8>{}); return true;
    default: return false;
  }
}

// h = fp16(norm(r) g (1 + sc) + sh) and its codes (sc may be null: no scale).
int norm_rq(oq_dit* h, const float* r, const void* g, const uint16_t* sc, const uint16_t* sh, uint16_t* out,
            float s, hipStream_t st, const float* sdelta) {
  const int64_t M = static_cast<int64_t>(h->cfg.batch) * h->cfg.tokens;
  const int64_t D = h->cfg.hidden;
  RQPlan p;
  const RQOut o = rq_out(h, D, s, &p, sdelta);
  const FusedLaunch fl = fused_launch(M, D, p);
  const uint16_t* gg = static_cast<const uint16_t*>(g);
  const bool ln = is_gr00t(h->cfg);
  if (!sh) return OQ_ERR_NULL;
  if (!ln && D == 1024 && o.logb == 10 && M <= 256) {
    if (sc)
      hipLaunchKernelGGL(norm_rq1024_kernel<true>, dim3(static_cast<unsigned>(M)), dim3(256), 0, st, r, gg, sc, sh,
                         out, M, o);
    else
      hipLaunchKernelGGL(norm_rq1024_kernel<false>, dim3(static_cast<unsigned>(M)), dim3(256), 0, st, r, gg, sc, sh,
                         out, M, o);
    return launch_status();
  }
  if (D == 1536 && o.logb == 9) {
    // Three 512-channel blocks: one row per three-wave workgroup.
    const dim3 grid(static_cast<unsigned>(M)), block(192);
    if (ln && sc) hipLaunchKernelGGL((norm_rq1536_kernel<true, true>), grid, block, 0, st, r, gg, sc, sh, out, M, o);
    else if (ln) hipLaunchKernelGGL((norm_rq1536_kernel<true, false>), grid, block, 0, st, r, gg, sc, sh, out, M, o);
    else if (sc) hipLaunchKernelGGL((norm_rq1536_kernel<false, true>), grid, block, 0, st, r, gg, sc, sh, out, M, o);
    else hipLaunchKernelGGL((norm_rq1536_kernel<false, false>), grid, block, 0, st, r, gg, sc, sh, out, M, o);
    return launch_status();
  }
  const bool ok = with_chunks(p.chunks, [&](auto C) {
    constexpr int CC = decltype(C)::value;
    if (ln && sc)
      hipLaunchKernelGGL((norm_rq_kernel<CC, true, true>), fl.grid, fl.block, fl.lds, st, r, gg, sc, sh, out, M,
                         static_cast<int>(D), o);
    else if (ln)
      hipLaunchKernelGGL((norm_rq_kernel<CC, true, false>), fl.grid, fl.block, fl.lds, st, r, gg, sc, sh, out, M,
                         static_cast<int>(D), o);
    else if (sc)
      hipLaunchKernelGGL((norm_rq_kernel<CC, false, true>), fl.grid, fl.block, fl.lds, st, r, gg, sc, sh, out, M,
                         static_cast<int>(D), o);
    else
      hipLaunchKernelGGL((norm_rq_kernel<CC, false, false>), fl.grid, fl.block, fl.lds, st, r, gg, sc, sh, out, M,
                         static_cast<int>(D), o);
  });
  return ok ? launch_status() : OQ_ERR_SHAPE;
}

// a = fp16(gelu(...)) of the MLP's first linear output and its codes.
int gelu_rq(oq_dit* h, const uint16_t* in, uint16_t* act, float s, hipStream_t st, const float* sdelta) {
  const int64_t M = static_cast<int64_t>(h->cfg.batch) * h->cfg.tokens;
  const int64_t F = h->cfg.mlp;
  RQPlan p;
  const RQOut o = rq_out(h, F, s, &p, sdelta);
  const bool gated = !is_gr00t(h->cfg);
  if (F == 4096 && o.logb == 12 && M <= 256) {
    if (gated)
      hipLaunchKernelGGL(gelu_rq4096_kernel<true>, dim3(static_cast<unsigned>(M)), dim3(1024), 0, st, in, act, M, o);
    else
      hipLaunchKernelGGL(gelu_rq4096_kernel<false>, dim3(static_cast<unsigned>(M)), dim3(1024), 0, st, in, act, M, o);
    return launch_status();
  }
  const FusedLaunch fl = fused_launch(M, F, p);
  const bool ok = with_chunks(p.chunks, [&](auto C) {
    if (gated)
      hipLaunchKernelGGL((gelu_rq_kernel<decltype(C)::value, true>), fl.grid, fl.block, fl.lds, st, in, act, M,
                         static_cast<int>(F), o);
    else
      hipLaunchKernelGGL((gelu_rq_kernel<decltype(C)::value, false>), fl.grid, fl.block, fl.lds, st, in, act, M,
                         static_cast<int>(F), o);
  });
  return ok ? launch_status() : OQ_ERR_SHAPE;
}

int gemm(oq_dit* h, const oq_qweight& wt, int64_t K, int64_t N, Epilogue epi, void* out, int64_t ldc,
         const uint16_t* gate, hipStream_t st) {
  const int64_t M = static_cast<int64_t>(h->cfg.batch) * h->cfg.tokens;
  GemmArgs a{at<uint8_t>(h, h->lay.xq), wt.wq, at<float>(h, h->lay.xs), wt.w_scale, nullptr, out, gate, M, N, K, ldc,
             h->tiled};
  if (h->lay.sk_tickets > 0) {
    a.part = at<int32_t>(h, h->lay.skp);
    a.tickets = at<int32_t>(h, h->lay.skt);
    a.part_words = h->lay.sk_words;
    a.n_tickets = h->lay.sk_tickets;
  }
  return gemm_launch(a, epi, st);
}

// Attention (partials over 64-key splits, then the merge fused with the o
// linear's rotate-quantize; with a single split the normalized rows and the
// stand-alone rotate-quantize).  Keys: `P` rows of k_pre / v_pre (row stride
// pre_ld) followed by `own` rows of the q|k|v buffer.
int attention_rq(oq_dit* h, const uint16_t* q, int64_t q_ld, const uint16_t* k_pre, const uint16_t* v_pre,
                 int P, int64_t pre_ld, const uint16_t* k_own, const uint16_t* v_own, int64_t own_ld, int own,
                 float s, hipStream_t st, const float* sdelta, bool keep) {
  const oq_dit_config& c = h->cfg;
  const int64_t M = static_cast<int64_t>(c.batch) * c.tokens;
  const int64_t D = c.hidden;
  AttnArgs a;
  a.q = q; a.q_ld = q_ld;
  a.k_pre = k_pre; a.v_pre = v_pre; a.P = P; a.pre_ld = pre_ld;
  a.k_own = k_own; a.v_own = v_own; a.own_ld = own_ld; a.own_keys = own;
  a.part_o = at<uint16_t>(h, h->lay.part_o);
  a.part_ml = at<float>(h, h->lay.part_ml);
  a.out = keep ? at<uint16_t>(h, h->lay.o) : nullptr; a.out_ld = D;
  a.S = c.tokens; a.H = c.n_heads; a.hd = c.head_dim; a.D = static_cast<int>(D);
  a.nsplit = (P + own + kAttnSplit - 1) / kAttnSplit;
  a.scale = static_cast<float>(1.0 / std::sqrt(static_cast<double>(c.head_dim)));
  // One split (the GR00T self-attention over its 16 action tokens): the
  // attention writes its normalized fp16 rows and the stand-alone
  // rotate-quantize takes them (no partials, no merge).
  a.direct = a.nsplit == 1 ? 1 : 0;
  if (a.direct) a.out = at<uint16_t>(h, h->lay.o);
  const unsigned waves = static_cast<unsigned>((c.tokens + 15) / 16);
  const dim3 grid(c.batch * c.n_heads, a.nsplit);
  // At most 32 keys in all (the GR00T self-attention over its 16 action
  // tokens): a 32-key instance, half the staging and products of 64.
  const bool short_keys = P + own <= 32;
  auto launch_ks = [&](auto W, auto KSc) {
    constexpr int WV = decltype(W)::value, KS = decltype(KSc)::value;
    switch (c.head_dim) {
      case 48: hipLaunchKernelGGL((attn_partial_kernel<WV, 48, KS>), grid, dim3(64 * WV), 0, st, a); break;
      case 64: hipLaunchKernelGGL((attn_partial_kernel<WV, 64, KS>), grid, dim3(64 * WV), 0, st, a); break;
      case 128: hipLaunchKernelGGL((attn_partial_kernel<WV, 128, KS>), grid, dim3(64 * WV), 0, st, a); break;
      default: hipLaunchKernelGGL((attn_partial_kernel<WV, 0, KS>), grid, dim3(64 * WV), 0, st, a); break;
    }
  };
  auto launch = [&](auto W) {
    if (short_keys) launch_ks(W, std::integral_constant<int, 32>{});
    else launch_ks(W, std::integral_constant<int, kAttnSplit>{});
  };
  switch (waves) {
    case 1: launch(std::integral_constant<int, 1>{}); break;
    case 2: launch(std::integral_constant<int, 2>{}); break;
    case 3: launch(std::integral_constant<int, 3>{}); break;
    default: launch(std::integral_constant<int, 4>{}); break;
  }
  int e = launch_status();
  if (e != OQ_OK) return e;
  if (a.direct)
    return rq_launch(a.out, M, D, D, pow2_divisor(static_cast<int>(D)), sdelta ? 1.0f : s, at<uint8_t>(h, h->lay.xq),
                     at<float>(h, h->lay.xs), nullptr, st, h->tiled, sdelta);
  RQPlan p;
  const RQOut ro = rq_out(h, D, s, &p, sdelta);
  if (D == 1024 && ro.logb == 10 && M <= 256 && c.head_dim % 4 == 0) {
    hipLaunchKernelGGL(combine_rq1024_kernel, dim3(static_cast<unsigned>(M)), dim3(256), 0, st, a, M, ro);
    return launch_status();
  }
  const FusedLaunch fl = fused_launch(M, D, p);
  const bool ok = with_chunks(p.chunks, [&](auto C) {
    hipLaunchKernelGGL((combine_rq_kernel<decltype(C)::value>), fl.grid, fl.block, fl.lds, st, a, M, ro);
  });
  return ok ? launch_status() : OQ_ERR_SHAPE;
}

// gr00t cross-attention of block l over the head-major conditioning k|v,
// then the o linear's rotate-quantize of the fp16 output rows.
int cross_attention_rq(oq_dit* h, const uint16_t* q, int64_t q_ld, int l, float s, hipStream_t st,
                       const float* sdelta) {
  const oq_dit_config& c = h->cfg;
  const int64_t M = static_cast<int64_t>(c.batch) * c.tokens;
  const int64_t D = c.hidden;
  const int64_t MC = static_cast<int64_t>(c.batch) * c.prefix;
  const uint16_t* kvh = at<uint16_t>(h, h->lay.ckvh) + static_cast<int64_t>(l / 2) * MC * 2 * D;
  uint16_t* out = at<uint16_t>(h, h->lay.o);
  const float scale = static_cast<float>(1.0 / std::sqrt(static_cast<double>(c.head_dim)));
  const unsigned waves = static_cast<unsigned>((c.tokens + 15) / 16);
  const dim3 grid(static_cast<unsigned>(c.batch * c.n_heads));
  auto launch = [&](auto W, auto HDc) {
    constexpr int WV = decltype(W)::value, HD = decltype(HDc)::value;
    hipLaunchKernelGGL((attn_cross_kernel<WV, HD>), grid, dim3(64 * WV), 0, st, q, q_ld, kvh, c.prefix,
                       c.tokens, c.n_heads, scale, out, D);
  };
  auto by_hd = [&](auto W) {
    switch (c.head_dim) {  // every multiple of 16 up to kMaxHeadDim (validate_config)
      case 16: launch(W, std::integral_constant<int, 16>{}); return true;
      case 32: launch(W, std::integral_constant<int, 32>{}); return true;
      case 48: launch(W, std::integral_constant<int, 48>{}); return true;
      case 64: launch(W, std::integral_constant<int, 64>{}); return true;
      case 80: launch(W, std::integral_constant<int, 80>{}); return true;
      case 96: launch(W, std::integral_constant<int, 96>{}); return true;
      case 112: launch(W, std::integral_constant<int, 112>{}); return true;
      case 128: launch(W, std::integral_constant<int, 128>{}); return true;
      default: return false;
    }
  };
  bool ok;
  switch (waves) {
    case 1: ok = by_hd(std::integral_constant<int, 1>{}); break;
    case 2: ok = by_hd(std::integral_constant<int, 2>{}); break;
    case 3: ok = by_hd(std::integral_constant<int, 3>{}); break;
    default: ok = by_hd(std::integral_constant<int, 4>{}); break;
  }
  if (!ok) return OQ_ERR_SHAPE;
  int e = launch_status();
  if (e != OQ_OK) return e;
  const int b = pow2_divisor(static_cast<int>(D));
  return rq_launch(out, M, D, D, b, sdelta ? 1.0f : s, at<uint8_t>(h, h->lay.xq), at<float>(h, h->lay.xs), nullptr,
                   st, h->tiled, sdelta);
}

// until: stop after the fused producer of quantization site `until` (0: the
// q|k|v input, 1: the o input, 2: the gate|up input, 3: the down input), or
// run the whole block (until = 4).
// Per-site static steps and the linears' weights of block l at step t: the
// per-step folded copies in the static mode, else the block's weights.
struct SiteSet {
  const float* d[4];
  const oq_qweight* w[4];
};

SiteSet site_set(oq_dit* h, int l, int t) {
  const oq_dit_config& c = h->cfg;
  const oq_dit_block& bw = h->blocks[l];
  SiteSet ss;
  const oq_qweight* own[4] = {&bw.qkv, &bw.o, &bw.gate_up, &bw.down};
  const size_t lt = static_cast<size_t>(l) * c.steps + t;
  const int64_t D = c.hidden;
  for (int i = 0; i < 4; ++i) {
    ss.d[i] = h->static_delta ? h->static_delta + lt * (3 * D + c.mlp) + i * D : nullptr;
    ss.w[i] = h->static_delta ? &h->static_w[lt * 4 + i] : own[i];
  }
  return ss;
}

// norm1_done: the first norm producer already ran (fused with the action
// in-projection of the step).
int run_block_pi(oq_dit* h, int l, int t, float* r, hipStream_t st, int until, bool keep, bool norm1_done = false) {
  const oq_dit_config& c = h->cfg;
  const oq_dit_block& bw = h->blocks[l];
  const int64_t D = c.hidden, F = c.mlp;
  const float* s = &h->s_table[(static_cast<size_t>(l) * c.steps + t) * 4];
  const SiteSet ss = site_set(h, l, t);
  // The fp16 site inputs are kept in the workspace for the parity calls
  // only; the producers write just the codes otherwise.
  uint16_t* h1 = keep ? at<uint16_t>(h, h->lay.h1) : nullptr;
  uint16_t* qkv = at<uint16_t>(h, h->lay.qkv);
  uint16_t* h2 = keep ? at<uint16_t>(h, h->lay.h2) : nullptr;
  uint16_t* gu = at<uint16_t>(h, h->lay.gu);
  uint16_t* act = keep ? at<uint16_t>(h, h->lay.act) : nullptr;
  int e;
  if (!norm1_done &&
      (e = norm_rq(h, r, bw.g1, mod_ptr(h, l, t, 0), mod_ptr(h, l, t, 1), h1, s[0], st, ss.d[0])) != OQ_OK)
    return e;
  if (until == 0) return OQ_OK;
  if ((e = gemm(h, *ss.w[0], D, 3 * D, EPI_F16, qkv, 3 * D, nullptr, st)) != OQ_OK) return e;
  if ((e = attention_rq(h, qkv, 3 * D, static_cast<const uint16_t*>(bw.prefix_k),
                        static_cast<const uint16_t*>(bw.prefix_v), c.prefix, D, qkv + D, qkv + 2 * D, 3 * D,
                        c.tokens, s[1], st, ss.d[1], keep)) != OQ_OK)
    return e;
  if (until == 1) return OQ_OK;
  if ((e = gemm(h, *ss.w[1], D, D, EPI_RESID_F32, r, D, mod_ptr(h, l, t, 2), st)) != OQ_OK) return e;
  if ((e = norm_rq(h, r, bw.g2, mod_ptr(h, l, t, 3), mod_ptr(h, l, t, 4), h2, s[2], st, ss.d[2])) != OQ_OK) return e;
  if (until == 2) return OQ_OK;
  if ((e = gemm(h, *ss.w[2], D, 2 * F, EPI_F16, gu, 2 * F, nullptr, st)) != OQ_OK) return e;
  if ((e = gelu_rq(h, gu, act, s[3], st, ss.d[3])) != OQ_OK) return e;
  if (until == 3) return OQ_OK;
  return gemm(h, *ss.w[3], F, D, EPI_RESID_F32, r, D, mod_ptr(h, l, t, 5), st);
}

int run_block_gr00t(oq_dit* h, int l, int t, float* r, hipStream_t st, int until, bool keep) {
  const oq_dit_config& c = h->cfg;
  const oq_dit_block& bw = h->blocks[l];
  const int64_t D = c.hidden, F = c.mlp;
  const float* s = &h->s_table[(static_cast<size_t>(l) * c.steps + t) * 4];
  const SiteSet ss = site_set(h, l, t);
  uint16_t* h1 = keep ? at<uint16_t>(h, h->lay.h1) : nullptr;
  uint16_t* qkv = at<uint16_t>(h, h->lay.qkv);
  uint16_t* h2 = keep ? at<uint16_t>(h, h->lay.h2) : nullptr;
  uint16_t* act = at<uint16_t>(h, h->lay.act);  // written by the ff0 epilogue, read by its quantizer
  int e;
  if ((e = norm_rq(h, r, bw.g1, mod_ptr(h, l, t, 0), mod_ptr(h, l, t, 1), h1, s[0], st, ss.d[0])) != OQ_OK) return e;
  if (until == 0) return OQ_OK;
  if (l % 2 == 0) {
    // Cross-attention to the conditioning k|v of this block ([B][P][2D]).
    if ((e = gemm(h, *ss.w[0], D, D, EPI_F16, qkv, D, nullptr, st)) != OQ_OK) return e;
    if ((e = cross_attention_rq(h, qkv, D, l, s[1], st, ss.d[1])) != OQ_OK) return e;
  } else {
    if ((e = gemm(h, *ss.w[0], D, 3 * D, EPI_F16, qkv, 3 * D, nullptr, st)) != OQ_OK) return e;
    if ((e = attention_rq(h, qkv, 3 * D, nullptr, nullptr, 0, 0, qkv + D, qkv + 2 * D, 3 * D, c.tokens, s[1], st,
                          ss.d[1], keep)) != OQ_OK)
      return e;
  }
  if (until == 1) return OQ_OK;
  if ((e = gemm(h, *ss.w[1], D, D, EPI_RESID_F32, r, D, nullptr, st)) != OQ_OK) return e;
  if ((e = norm_rq(h, r, bw.g2, nullptr, static_cast<const uint16_t*>(bw.b2), h2, s[2], st, ss.d[2])) != OQ_OK)
    return e;
  if (until == 2) return OQ_OK;
  // The non-gated GELU is elementwise: the ff0 linear applies it in its
  // epilogue (act = fp16(gelu(fp16(y)))), and the activation rows are then
  // rotated and quantized by the stand-alone kernel.
  if ((e = gemm(h, *ss.w[2], D, F, EPI_GELU_F16, act, F, nullptr, st)) != OQ_OK) return e;
  const int64_t M = static_cast<int64_t>(c.batch) * c.tokens;
  if ((e = rq_launch(act, M, F, F, pow2_divisor(static_cast<int>(F)), ss.d[3] ? 1.0f : s[3],
                     at<uint8_t>(h, h->lay.xq), at<float>(h, h->lay.xs), nullptr, st, h->tiled, ss.d[3])) != OQ_OK)
    return e;
  if (until == 3) return OQ_OK;
  return gemm(h, *ss.w[3], F, D, EPI_RESID_F32, r, D, nullptr, st);
}

int run_block(oq_dit* h, int l, int t, float* r, hipStream_t st, int until = 4, bool keep = true) {
  return is_gr00t(h->cfg) ? run_block_gr00t(h, l, t, r, st, until, keep) : run_block_pi(h, l, t, r, st, until, keep);
}

int final_stage(oq_dit* h, const float* r, float* x, hipStream_t st);

// r = x W_in^T + b_in for the M action rows: inproj_rows_kernel (8 rows per
// workgroup) when the weight rows can be preloaded, else inproj_kernel (one
// row per workgroup); the same sums either way.
int inproj_launch(const oq_dit* h, const float* x, float* r, hipStream_t st) {
  const oq_dit_config& c = h->cfg;
  const int64_t M = static_cast<int64_t>(c.batch) * c.tokens;
  const auto* w_in = static_cast<const uint16_t*>(h->w.w_in);
  const auto* b_in = static_cast<const uint16_t*>(h->w.b_in);
  constexpr int R = 8;  // R * A <= 256 for A <= kInprojA
  const dim3 grid(static_cast<unsigned>((M + R - 1) / R), static_cast<unsigned>((c.hidden + 255) / 256));
  const int ap = inproj_preload_a(c.action_dim, w_in);
  if (ap > 0) {
    switch (ap) {
      case 8: hipLaunchKernelGGL((inproj_rows_kernel<R, 8>), grid, dim3(256), 0, st, x, w_in, b_in, r, M, c.hidden); break;
      case 16: hipLaunchKernelGGL((inproj_rows_kernel<R, 16>), grid, dim3(256), 0, st, x, w_in, b_in, r, M, c.hidden); break;
      case 24: hipLaunchKernelGGL((inproj_rows_kernel<R, 24>), grid, dim3(256), 0, st, x, w_in, b_in, r, M, c.hidden); break;
      default: hipLaunchKernelGGL((inproj_rows_kernel<R, 32>), grid, dim3(256), 0, st, x, w_in, b_in, r, M, c.hidden); break;
    }
  } else {
    hipLaunchKernelGGL(inproj_kernel, dim3(static_cast<unsigned>(M)), dim3(256), c.action_dim * sizeof(float), st, x,
                       w_in, b_in, r, c.action_dim, c.hidden);
  }
  return launch_status();
}

// Pi-0.5 with 1024-channel rows on the 1024-wide producer path (at most 256
// rows, Hadamard block = the row): the step's in-projection and block 0's
// first norm producer as one kernel (the same arithmetic as inproj_kernel
// followed by norm_rq1024_kernel).  *fused = false when it does not apply.
int inproj_norm1(oq_dit* h, const float* x, float* r, int t, hipStream_t st, bool* fused) {
  const oq_dit_config& c = h->cfg;
  const int64_t M = static_cast<int64_t>(c.batch) * c.tokens;
  *fused = false;
  if (is_gr00t(c) || c.hidden != 1024 || M > 256) return OQ_OK;
  const float* s = &h->s_table[static_cast<size_t>(t) * 4];  // block 0
  const SiteSet ss = site_set(h, 0, t);
  RQPlan p;
  const RQOut o = rq_out(h, c.hidden, s[0], &p, ss.d[0]);
  if (o.logb != 10) return OQ_OK;
  hipLaunchKernelGGL(inproj_norm_rq1024_kernel<true>, dim3(static_cast<unsigned>(M)), dim3(256), 0, st, x,
                     static_cast<const uint16_t*>(h->w.w_in), static_cast<const uint16_t*>(h->w.b_in), r,
                     c.action_dim, static_cast<const uint16_t*>(h->blocks[0].g1), mod_ptr(h, 0, t, 0),
                     mod_ptr(h, 0, t, 1), nullptr, M, o);
  *fused = true;
  return launch_status();
}

int run_step(oq_dit* h, float* x, int t, hipStream_t st) {
  const oq_dit_config& c = h->cfg;
  const int64_t M = static_cast<int64_t>(c.batch) * c.tokens;
  float* r = at<float>(h, h->lay.r);
  bool fused = false;
  int e = inproj_norm1(h, x, r, t, st, &fused);
  if (e != OQ_OK) return e;
  if (!fused && (e = inproj_launch(h, x, r, st)) != OQ_OK) return e;
  for (int l = 0; l < c.n_blocks; ++l) {
    e = fused && l == 0 ? run_block_pi(h, 0, t, r, st, 4, false, true) : run_block(h, l, t, r, st, 4, false);
    if (e != OQ_OK) return e;
  }
  return final_stage(h, r, x, st);
}

// x += dt * (fp16(norm(r) g_f) W_out^T + b_out): the final norm, the
// out-projection and the Euler update of a step.
int final_stage(oq_dit* h, const float* r, float* x, hipStream_t st) {
  const oq_dit_config& c = h->cfg;
  const int64_t M = static_cast<int64_t>(c.batch) * c.tokens;
  const float dt = (is_gr00t(c) ? 1.0f : -1.0f) / static_cast<float>(c.steps);
  // Few rows (the Pi-0.5 action tokens): one row per workgroup, so the rows
  // spread over as many CUs; else two (the weight slices are read once per
  // workgroup; two rows gave 1024 GR00T rows 512 workgroups and a shorter
  // per-thread product chain than four, for twice the weight reads).
  auto launch = [&](auto LNc, auto Rc) {
    constexpr bool LN = decltype(LNc)::value;
    constexpr int R = decltype(Rc)::value;
    const size_t lds = static_cast<size_t>(R) * c.hidden * sizeof(float);
    hipLaunchKernelGGL((final_kernel<LN, R>), dim3(static_cast<unsigned>((M + R - 1) / R)), dim3(256), lds, st, r,
                       static_cast<const uint16_t*>(h->w.g_f), static_cast<const uint16_t*>(h->w.w_out),
                       static_cast<const uint16_t*>(h->w.b_out), x, M, c.hidden, c.action_dim, dt);
  };
  const bool few = M <= 256;
  if (is_gr00t(c)) {
    if (few) launch(std::true_type{}, std::integral_constant<int, 1>{});
    else launch(std::true_type{}, std::integral_constant<int, 2>{});
  } else {
    if (few) launch(std::false_type{}, std::integral_constant<int, 1>{});
    else launch(std::false_type{}, std::integral_constant<int, 4>{});
  }
  return launch_status();
}

// gr00t: k|v of the conditioning tokens of every cross-attention block.
int set_condition(oq_dit* h, const uint16_t* cond, hipStream_t st) {
  const oq_dit_config& c = h->cfg;
  const int64_t MC = static_cast<int64_t>(c.batch) * c.prefix;
  const int64_t D = c.hidden;
  uint8_t* xq = at<uint8_t>(h, h->lay.xq);
  float* xs = at<float>(h, h->lay.xs);
  int e = rq_launch(cond, MC, D, D, pow2_divisor(static_cast<int>(D)), 1.0f, xq, xs, nullptr, st);
  if (e != OQ_OK) return e;
  for (int l = 0; l < c.n_blocks; l += 2) {
    uint16_t* kv = at<uint16_t>(h, h->lay.ckv);  // staging, rewritten head-major below
    const oq_qweight& wt = h->blocks[l].cross_kv;
    GemmArgs a{xq, wt.wq, xs, wt.w_scale, nullptr, kv, nullptr, MC, 2 * D, D, 2 * D};
    if ((e = gemm_launch(a, EPI_F16, st)) != OQ_OK) return e;
    uint16_t* kvh = at<uint16_t>(h, h->lay.ckvh) + static_cast<int64_t>(l / 2) * MC * 2 * D;
    const int64_t pieces = MC * 2 * D / 8;
    hipLaunchKernelGGL(kv_head_major_kernel, dim3(static_cast<unsigned>((pieces + 255) / 256)), dim3(256), 0, st,
                       kv, kvh, static_cast<int64_t>(c.batch), c.prefix, c.n_heads, c.head_dim);
    if ((e = launch_status()) != OQ_OK) return e;
  }
  return OQ_OK;
}

// Replays still in flight finish before their executable graphs go.
void drop_graphs(oq_dit* h) {
  if (h->graphs.empty()) return;
  hipDeviceSynchronize();
  for (auto& g : h->graphs) hipGraphExecDestroy(g.exec);
  h->graphs.clear();
}

// Captured step graphs kept per handle (keyed by state pointer, first step
// and count); a denoising loop over one state buffer uses at most its T
// single steps plus one whole-loop graph.
constexpr size_t kMaxGraphs = 16;

// Steps t0 .. t0+n-1 on x: replay the cached graph for (x, t0, n), capturing it
// on the internal stream the first time (that first call instantiates the
// graph, a host-side allocation of the runtime; later calls allocate nothing).
int run_steps(oq_dit* h, float* x, int t0, int n, hipStream_t st) {
  if (!h->use_graphs) {
    for (int t = t0; t < t0 + n; ++t) {
      int e = run_step(h, x, t, st);
      if (e != OQ_OK) return e;
    }
    return OQ_OK;
  }
  ++h->graph_clock;
  for (auto& g : h->graphs)
    if (g.x == x && g.t0 == t0 && g.n == n) {
      g.last_use = h->graph_clock;
      return hipGraphLaunch(g.exec, st) == hipSuccess ? OQ_OK : OQ_ERR_HIP;
    }
  if (h->graphs.size() >= kMaxGraphs) {
    // Drop the least recently used capture once its replays have finished
    // (its last one may have been enqueued on another caller stream).
    hipDeviceSynchronize();
    auto lru = std::min_element(h->graphs.begin(), h->graphs.end(),
                                [](const oq_dit_graph& a, const oq_dit_graph& b) { return a.last_use < b.last_use; });
    hipGraphExecDestroy(lru->exec);
    h->graphs.erase(lru);
  }
  if (hipStreamBeginCapture(h->cap, hipStreamCaptureModeThreadLocal) != hipSuccess) return OQ_ERR_HIP;
  int e = OQ_OK;
  for (int t = t0; t < t0 + n && e == OQ_OK; ++t) e = run_step(h, x, t, h->cap);
  hipGraph_t graph = nullptr;
  const hipError_t ce = hipStreamEndCapture(h->cap, &graph);
  if (e != OQ_OK || ce != hipSuccess || !graph) {
    if (graph) hipGraphDestroy(graph);
    return e != OQ_OK ? e : OQ_ERR_HIP;
  }
  hipGraphExec_t exec = nullptr;
  const hipError_t ie = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
  hipGraphDestroy(graph);
  if (ie != hipSuccess) return OQ_ERR_HIP;
  h->graphs.push_back({x, t0, n, exec, h->graph_clock});
  return hipGraphLaunch(exec, st) == hipSuccess ? OQ_OK : OQ_ERR_HIP;
}

bool qw_ok(const oq_qweight& q) { return q.wq && q.w_scale; }
bool qw_aligned(const oq_qweight& q) { return aligned(q.wq, 16) && aligned(q.w_scale, 4); }

int validate_weights(const oq_dit_config* cfg, const oq_dit_weights* w) {
  if (!w->blocks || !w->mod || !w->s_table || !w->w_in || !w->b_in || !w->w_out || !w->b_out || !w->g_f)
    return OQ_ERR_NULL;
  const bool gr = cfg->arch == OQ_DIT_GR00T;
  for (int l = 0; l < cfg->n_blocks; ++l) {
    const oq_dit_block& b = w->blocks[l];
    if (!b.g1 || !b.g2 || !qw_ok(b.qkv) || !qw_ok(b.o) || !qw_ok(b.gate_up) || !qw_ok(b.down)) return OQ_ERR_NULL;
    if (!qw_aligned(b.qkv) || !qw_aligned(b.o) || !qw_aligned(b.gate_up) || !qw_aligned(b.down) ||
        !aligned(b.g1, 16) || !aligned(b.g2, 16))
      return OQ_ERR_ALIGN;
    if (gr) {
      if (!b.b2) return OQ_ERR_NULL;
      if (!aligned(b.b2, 16)) return OQ_ERR_ALIGN;
      if (l % 2 == 0) {
        if (!qw_ok(b.cross_kv)) return OQ_ERR_NULL;
        if (!qw_aligned(b.cross_kv)) return OQ_ERR_ALIGN;
      }
    } else if (cfg->prefix > 0) {
      if (!b.prefix_k || !b.prefix_v) return OQ_ERR_NULL;
      if (!aligned(b.prefix_k, 16) || !aligned(b.prefix_v, 16)) return OQ_ERR_ALIGN;
    }
  }
  if (!aligned(w->mod, 16)) return OQ_ERR_ALIGN;
  const size_t ns = static_cast<size_t>(cfg->n_blocks) * cfg->steps * 4;
  for (size_t i = 0; i < ns; ++i)
    if (!(w->s_table[i] > 0.0f) || !std::isfinite(w->s_table[i])) return OQ_ERR_ARG;
  return OQ_OK;
}

}  // namespace
}  // namespace oq

extern "C" int oq_dit_workspace_bytes(const oq_dit_config* cfg, size_t* bytes) {
  int e = oq::validate_config(cfg);
  if (e != OQ_OK) return e;
  if (!bytes) return OQ_ERR_NULL;
  *bytes = oq::layout_for(*cfg).total;
  return OQ_OK;
}

extern "C" int oq_dit_create(const oq_dit_config* cfg, const oq_dit_weights* w, oq_dit** out) {
  int e = oq::validate_config(cfg);
  if (e != OQ_OK) return e;
  if (!w || !out) return OQ_ERR_NULL;
  if ((e = oq::validate_weights(cfg, w)) != OQ_OK) return e;
  if ((e = oq::device_check()) != OQ_OK) return e;
  hipStream_t cap = nullptr;
  if (hipStreamCreateWithFlags(&cap, hipStreamNonBlocking) != hipSuccess) return OQ_ERR_HIP;
  oq_dit* h = new oq_dit();
  h->cfg = *cfg;
  h->w = *w;
  h->blocks.assign(w->blocks, w->blocks + cfg->n_blocks);
  h->s_table.assign(w->s_table, w->s_table + static_cast<size_t>(cfg->n_blocks) * cfg->steps * 4);
  h->w.blocks = h->blocks.data();
  h->w.s_table = h->s_table.data();
  h->lay = oq::layout_for(*cfg);
  h->cap = cap;
  const char* env = std::getenv("OQ_DIT_NO_GRAPH");
  h->use_graphs = !(env && env[0] == '1');
  // Up to 64 tokens the block products run on the small-M kernel, which reads
  // the token codes fastest in the tiled layout; the fused producers write it.
  const int64_t M = static_cast<int64_t>(cfg->batch) * cfg->tokens;
  h->tiled = M <= 64 && cfg->hidden % 128 == 0 && cfg->mlp % 128 == 0;
  *out = h;
  return OQ_OK;
}

extern "C" int oq_dit_set_workspace(oq_dit* h, void* workspace, size_t bytes) {
  if (!h || !workspace) return OQ_ERR_NULL;
  if (!oq::aligned(workspace, 256)) return OQ_ERR_ALIGN;
  if (bytes < h->lay.total) return OQ_ERR_WORKSPACE;
  if (h->ws != workspace) {
    oq::drop_graphs(h);
    h->cond_ready = false;
  }
  h->ws = static_cast<uint8_t*>(workspace);
  h->ws_bytes = bytes;
  // The split-K tickets start at zero (each launch leaves them so).
  if (h->lay.sk_tickets > 0 &&
      hipMemset(h->ws + h->lay.skt, 0, static_cast<size_t>(h->lay.sk_tickets) * 4) != hipSuccess)
    return OQ_ERR_HIP;
  return OQ_OK;
}

extern "C" int oq_dit_set_condition(oq_dit* h, const void* cond, void* stream) {
  if (!h || !cond) return OQ_ERR_NULL;
  if (!h->ws) return OQ_ERR_WORKSPACE;
  if (!oq::is_gr00t(h->cfg)) return OQ_ERR_ARG;
  if (!oq::aligned(cond, 16)) return OQ_ERR_ALIGN;
  const int e = oq::set_condition(h, static_cast<const uint16_t*>(cond), static_cast<hipStream_t>(stream));
  h->cond_ready = e == OQ_OK;
  return e;
}

namespace {
int step_ready(const oq_dit* h) {
  if (!h->ws) return OQ_ERR_WORKSPACE;
  if (oq::is_gr00t(h->cfg) && !h->cond_ready) return OQ_ERR_ARG;
  return OQ_OK;
}
}  // namespace

extern "C" int oq_dit_step(oq_dit* h, float* x, int32_t t, void* stream) {
  if (!h || !x) return OQ_ERR_NULL;
  int e = step_ready(h);
  if (e != OQ_OK) return e;
  if (t < 0 || t >= h->cfg.steps) return OQ_ERR_ARG;
  return oq::run_steps(h, x, t, 1, static_cast<hipStream_t>(stream));
}

extern "C" int oq_dit_denoise(oq_dit* h, float* x, int32_t n_steps, void* stream) {
  if (!h || !x) return OQ_ERR_NULL;
  int e = step_ready(h);
  if (e != OQ_OK) return e;
  if (n_steps < 0 || n_steps > h->cfg.steps) return OQ_ERR_ARG;
  if (n_steps == 0) return OQ_OK;
  return oq::run_steps(h, x, 0, n_steps, static_cast<hipStream_t>(stream));
}

extern "C" int oq_dit_run_block(oq_dit* h, int32_t l, int32_t t, float* resid, void* stream) {
  if (!h || !resid) return OQ_ERR_NULL;
  int e = step_ready(h);
  if (e != OQ_OK) return e;
  if (l < 0 || l >= h->cfg.n_blocks || t < 0 || t >= h->cfg.steps) return OQ_ERR_ARG;
  return oq::run_block(h, l, t, resid, static_cast<hipStream_t>(stream));
}

extern "C" int oq_dit_run_block_until(oq_dit* h, int32_t l, int32_t t, float* resid, int32_t site, void* stream) {
  if (!h || !resid) return OQ_ERR_NULL;
  int e = step_ready(h);
  if (e != OQ_OK) return e;
  if (l < 0 || l >= h->cfg.n_blocks || t < 0 || t >= h->cfg.steps || site < 0 || site > 3) return OQ_ERR_ARG;
  return oq::run_block(h, l, t, resid, static_cast<hipStream_t>(stream), site);
}

extern "C" int oq_dit_set_static_steps(oq_dit* h, const float* delta, const oq_qweight* step_weights) {
  if (!h) return OQ_ERR_NULL;
  oq::drop_graphs(h);  // captured steps hold the previous tables and weights
  if (!delta) {
    h->static_delta = nullptr;
    h->static_w.clear();
    return OQ_OK;
  }
  if (!step_weights) return OQ_ERR_NULL;
  if (!oq::aligned(delta, 16)) return OQ_ERR_ALIGN;
  const size_t n = static_cast<size_t>(h->cfg.n_blocks) * h->cfg.steps * 4;
  for (size_t i = 0; i < n; ++i) {
    if (!step_weights[i].wq || !step_weights[i].w_scale) return OQ_ERR_NULL;
    if (!oq::aligned(step_weights[i].wq, 16) || !oq::aligned(step_weights[i].w_scale, 4)) return OQ_ERR_ALIGN;
  }
  h->static_w.assign(step_weights, step_weights + n);
  h->static_delta = delta;
  return OQ_OK;
}

extern "C" int oq_dit_in_projection(oq_dit* h, const float* x, float* resid, void* stream) {
  if (!h || !x || !resid) return OQ_ERR_NULL;
  if (!oq::aligned(x, 4) || !oq::aligned(resid, 4)) return OQ_ERR_ALIGN;
  return oq::inproj_launch(h, x, resid, static_cast<hipStream_t>(stream));
}

extern "C" int oq_dit_final_stage(oq_dit* h, const float* resid, float* x, void* stream) {
  if (!h || !resid || !x) return OQ_ERR_NULL;
  if (!oq::aligned(x, 4) || !oq::aligned(resid, 16)) return OQ_ERR_ALIGN;
  return oq::final_stage(h, resid, x, static_cast<hipStream_t>(stream));
}

extern "C" int oq_dit_get_intermediates(const oq_dit* h, oq_dit_intermediates* out) {
  if (!h || !out) return OQ_ERR_NULL;
  if (!h->ws) return OQ_ERR_WORKSPACE;
  out->h1 = h->ws + h->lay.h1;
  out->qkv = h->ws + h->lay.qkv;
  out->attn = h->ws + h->lay.o;
  out->h2 = h->ws + h->lay.h2;
  out->gate_up = h->ws + h->lay.gu;
  out->act = h->ws + h->lay.act;
  out->resid = reinterpret_cast<const float*>(h->ws + h->lay.r);
  out->cond_kv = oq::is_gr00t(h->cfg) ? h->ws + h->lay.ckvh : nullptr;
  out->codes = h->ws + h->lay.xq;
  out->x_scale = reinterpret_cast<const float*>(h->ws + h->lay.xs);
  out->codes_tiled = h->tiled ? 1 : 0;
  return OQ_OK;
}

extern "C" void oq_dit_destroy(oq_dit* h) {
  if (!h) return;
  oq::drop_graphs(h);
  if (h->cap) hipStreamDestroy(h->cap);
  delete h;
}
