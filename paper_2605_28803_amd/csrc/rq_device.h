// Device-side building blocks of the fused Hadamard rotation + per-step scale +
// per-token int4 quantization (Section 4.1 eq:blockdiag / eq:transform; Section
// 4.2 eq:scale, eq:quant, eq:perstep_scale), shared by the stand-alone
// rotate-quantize kernel and by kernels that produce a row and quantize it in
// the same pass (the DiT norm, attention-combine and gated-GELU kernels).
//
// Row layout.  A row of K channels is owned by T = 2^logT threads; thread t
// holds C chunks of 8 consecutive channels, channel k = c * 8T + t * 8 + j.
// The Walsh-Hadamard butterflies over the index bits below log2(b) commute;
// each is done where its bit lives: bits 0..2 in registers, the next
// log2(min(T, 64)) bits across lanes (DPP, ds_swizzle, permlane swaps), wave
// bits through LDS, bits above the thread bits in registers again.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.h"

namespace oq {
namespace rqd {

constexpr float kRoundMagic = 12582912.0f;  // 1.5 * 2^23: x + magic rounds x half-to-even into the low mantissa bits

__device__ __forceinline__ float h2f(uint32_t h) {
  return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(h)));
}
__device__ __forceinline__ uint16_t f2h(float f) { return __builtin_bit_cast(uint16_t, static_cast<_Float16>(f)); }
// Round to fp16 and back: the value a tensor stored in fp16 holds.
__device__ __forceinline__ float f16r(float f) { return static_cast<float>(static_cast<_Float16>(f)); }

// Value of lane (lane ^ H) for H < 16: DPP quad permutations for 1 and 2,
// ds_swizzle (bit-mask mode, 32-lane groups) for 4 and 8.
template <int H>
__device__ __forceinline__ float lane_xor(float v) {
  const int x = __float_as_int(v);
  if constexpr (H == 1) return __int_as_float(__builtin_amdgcn_mov_dpp(x, 0xB1, 0xF, 0xF, false));  // [1,0,3,2]
  if constexpr (H == 2) return __int_as_float(__builtin_amdgcn_mov_dpp(x, 0x4E, 0xF, 0xF, false));  // [2,3,0,1]
  if constexpr (H == 4 || H == 8) return __int_as_float(__builtin_amdgcn_ds_swizzle(x, 0x1F | (H << 10)));
  if constexpr (H == 16) return __int_as_float(__builtin_amdgcn_ds_swizzle(x, 0x1F | (16 << 10)));
  static_assert(H == 1 || H == 2 || H == 4 || H == 8 || H == 16, "lane_xor: H < 32");
  return v;
}

// Butterfly over lane bit log2(H), H < 16, for every element.
template <int H, int C>
__device__ __forceinline__ void lane_stage(float (&v)[C][8], int lane) {
  const float sgn = (lane & H) ? -1.0f : 1.0f;
  float p[C][8];
#pragma unroll
  for (int c = 0; c < C; ++c)
#pragma unroll
    for (int j = 0; j < 8; ++j) p[c][j] = lane_xor<H>(v[c][j]);
#pragma unroll
  for (int c = 0; c < C; ++c)
#pragma unroll
    for (int j = 0; j < 8; ++j) v[c][j] = fmaf(sgn, v[c][j], p[c][j]);  // upper: p - v, lower: p + v
}

// Butterfly over lane bit 4 (H = 16) or 5 (H = 32) with the gfx950 permlane
// swaps.  For two registers a, b: permlane{16,32}_swap exchanges the upper
// half-group of a with the lower half-group of b, so afterwards the lower
// lanes hold (a[l], a[l+H]) and the upper lanes (b[l-H], b[l]); the butterfly
// is then lane-local, and a second swap returns every value to its lane.
template <int H>
__device__ __forceinline__ void permlane_swap(float& a, float& b) {
  int x = __float_as_int(a), y = __float_as_int(b);
  if constexpr (H == 16) {
    auto r = __builtin_amdgcn_permlane16_swap(x, y, false, false);
    x = r[0];
    y = r[1];
  } else {
    auto r = __builtin_amdgcn_permlane32_swap(x, y, false, false);
    x = r[0];
    y = r[1];
  }
  a = __int_as_float(x);
  b = __int_as_float(y);
}

// The same swap on two dwords: afterwards the lower half-group holds
// (a[l], a[l+H]) and the upper half-group (b[l-H], b[l]).
template <int H>
__device__ __forceinline__ void dword_swap(uint32_t& a, uint32_t& b) {
  float x = __uint_as_float(a), y = __uint_as_float(b);
  permlane_swap<H>(x, y);
  a = __float_as_uint(x);
  b = __float_as_uint(y);
}

// Value of lane (lane ^ H), H = 16 or 32, through the permlane swaps (VALU;
// no LDS-pipe round trip as with ds_bpermute / ds_swizzle).
template <int H>
__device__ __forceinline__ float lane_xor_far(float v) {
  static_assert(H == 16 || H == 32, "lane_xor_far: H = 16 or 32");
  float x = v, y = v;
  permlane_swap<H>(x, y);
  return (threadIdx.x & H) ? x : y;
}

// Value of lane (lane ^ H), H = 4 or 8, as two DPP row moves (H = 4: row
// half-mirror, lane ^ 7 within 8, then the quad reversal, ^ 3; H = 8: row
// mirror, ^ 15 within 16, then the half-mirror): shorter latency than a
// ds_swizzle in a dependent chain of one value, while stages over many values
// keep the swizzle (the LDS pipe works beside the VALU there).
template <int H>
__device__ __forceinline__ float lane_xor_dpp(float v) {
  static_assert(H == 4 || H == 8, "lane_xor_dpp: H = 4 or 8");
  const int x = __float_as_int(v);
  if constexpr (H == 4)
    return __int_as_float(__builtin_amdgcn_mov_dpp(__builtin_amdgcn_mov_dpp(x, 0x141, 0xF, 0xF, false), 0x1B, 0xF,
                                                   0xF, false));
  return __int_as_float(__builtin_amdgcn_mov_dpp(__builtin_amdgcn_mov_dpp(x, 0x140, 0xF, 0xF, false), 0x141, 0xF,
                                                 0xF, false));
}

// Sum over the 64 lanes of a wave, every lane receiving it: lane ^ 32, 16,
// 8, 4, 2, 1 in that order (the partners and order of a __shfl_xor loop from
// 32 down, so the same fp32 sum bit for bit), all on the VALU.
__device__ __forceinline__ float wave_sum_xor(float v) {
  v += lane_xor_far<32>(v);
  v += lane_xor_far<16>(v);
  v += lane_xor_dpp<8>(v);
  v += lane_xor_dpp<4>(v);
  v += lane_xor<2>(v);
  v += lane_xor<1>(v);
  return v;
}

// Maximum over the 64 lanes of a wave, every lane receiving it (order-free):
// quad permutations, the row half-mirror and mirror (8- and 16-lane groups),
// then the permlane swaps, all on the VALU.
__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, lane_xor<1>(v));
  v = fmaxf(v, lane_xor<2>(v));
  v = fmaxf(v, __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x141, 0xF, 0xF, false)));  // half-mirror
  v = fmaxf(v, __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x140, 0xF, 0xF, false)));  // mirror
  v = fmaxf(v, lane_xor_far<16>(v));
  v = fmaxf(v, lane_xor_far<32>(v));
  return v;
}

template <int H, int C>
__device__ __forceinline__ void lane_stage_swap(float (&v)[C][8]) {
#pragma unroll
  for (int c = 0; c < C; ++c)
#pragma unroll
    for (int j = 0; j < 8; j += 2) {
      float a = v[c][j], b = v[c][j + 1];
      permlane_swap<H>(a, b);
      const float s = a + b, d = a - b;
      a = s;
      b = d;
      permlane_swap<H>(a, b);
      v[c][j] = a;
      v[c][j + 1] = b;
    }
}

// Where the calling thread sits: T threads per row, rows_per_wg rows per
// workgroup (blockDim.x = max(T, 256)).
struct RowMap {
  int logT, T, t, lane, row_local, rows_per_wg;
  int64_t row;
  bool valid;
};

__device__ __forceinline__ RowMap row_map(int logT, int64_t M) {
  RowMap r;
  r.logT = logT;
  r.T = 1 << logT;
  const int tid = threadIdx.x;
  r.row_local = tid >> logT;
  r.t = tid & (r.T - 1);
  r.rows_per_wg = blockDim.x >> logT;
  r.row = static_cast<int64_t>(blockIdx.x) * r.rows_per_wg + r.row_local;
  r.valid = r.row < M;
  r.lane = tid & 63;
  return r;
}

// Channel index of element (c, j) of this thread.
__device__ __forceinline__ int chan(const RowMap& m, int c, int j) { return c * 8 * m.T + m.t * 8 + j; }

// Reduction across the T threads of a row (max or sum).  Every thread of the
// workgroup must call it (it synchronizes when a row spans several waves);
// `red` is a 4-entry shared array that must not be in use by the caller.
template <bool kMax>
__device__ __forceinline__ float row_reduce(float x, const RowMap& m, float* red) {
  const int lane_bits = m.logT < 6 ? m.logT : 6;
  auto op = [](float a, float b) { return kMax ? fmaxf(a, b) : a + b; };
  if (lane_bits > 0) x = op(x, lane_xor<1>(x));
  if (lane_bits > 1) x = op(x, lane_xor<2>(x));
  if (lane_bits > 2) x = op(x, lane_xor<4>(x));
  if (lane_bits > 3) x = op(x, lane_xor<8>(x));
  if (lane_bits > 4) x = op(x, lane_xor_far<16>(x));
  if (lane_bits > 5) x = op(x, lane_xor_far<32>(x));
  if (m.logT > 6) {
    const int w = threadIdx.x >> 6;
    __syncthreads();
    if (m.lane == 0) red[w] = x;
    __syncthreads();
    const int nwr = m.T >> 6;
    const int first = m.row_local * nwr;
    x = red[first];
    for (int u = 1; u < nwr; ++u) x = op(x, red[first + u]);
  }
  return x;
}

// Load C chunks of fp16 channels of row `row` (zeros when !valid).
template <int C>
__device__ __forceinline__ void load_row_f16(float (&v)[C][8], const uint16_t* __restrict__ X, int64_t ldx,
                                             const RowMap& m) {
  const uint16_t* xr = X + (m.valid ? m.row : 0) * ldx;
#pragma unroll
  for (int c = 0; c < C; ++c) {
    uint4 raw = make_uint4(0, 0, 0, 0);
    if (m.valid) raw = *reinterpret_cast<const uint4*>(xr + c * 8 * m.T + m.t * 8);
    const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      v[c][2 * q] = h2f(w[q] & 0xFFFFu);
      v[c][2 * q + 1] = h2f(w[q] >> 16);
    }
  }
}

// Pack eight codes, given as the bit patterns of (ratio + 1.5*2^23), into one
// dword: channel j in bits 4j..4j+3.  The low byte of each pattern is the code
// as a two's-complement byte (the constant's low byte is zero, |code| <= 7).
__device__ __forceinline__ uint32_t pack8(const uint32_t (&b)[8]) {
  // Low bytes of the even channels -> e = [b0 b2 b4 b6], odd -> o = [b1 b3 b5 b7].
  const uint32_t e = __builtin_amdgcn_perm(__builtin_amdgcn_perm(b[6], b[4], 0x04000c0cu),
                                           __builtin_amdgcn_perm(b[2], b[0], 0x0c0c0400u), 0x07060100u);
  const uint32_t o = __builtin_amdgcn_perm(__builtin_amdgcn_perm(b[7], b[5], 0x04000c0cu),
                                           __builtin_amdgcn_perm(b[3], b[1], 0x0c0c0400u), 0x07060100u);
  // Byte i = code(2i) in the low nibble, code(2i+1) in the high nibble.
  return (e & 0x0F0F0F0Fu) | ((o << 4) & 0xF0F0F0F0u);
}

// Static per-channel quantizer (eq:perstep_scale with the per-channel table
// in place of the token step, eq:quant): code = clamp(rne(y / Delta), -7, 7)
// for the unnormalized butterfly output u = y * sqrt(b) (inv_sqrtb =
// 1 / sqrt(b)), returned as the bit pattern of (code + 1.5 * 2^23) for pack8.
// A channel whose step is not a positive number (zero, negative, NaN) and
// one with an infinite step get code 0.  Clamping the ratio to [-7, 7]
// before rounding equals clamping the rounded code, the bounds being integers.
__device__ __forceinline__ uint32_t static_code(float u, float delta, float inv_sqrtb) {
  const float g = delta > 0.0f ? inv_sqrtb * __builtin_amdgcn_rcpf(delta) : 0.0f;
  const float r = __builtin_amdgcn_fmed3f(u * g, -7.0f, 7.0f);
  return __float_as_uint(r + kRoundMagic);
}

// Eight 8-bit codes, given as the bit patterns of (ratio + 1.5*2^23), as two
// dwords: channel j in byte j (two's complement, |code| <= 127).
__device__ __forceinline__ uint2 pack8_i8(const uint32_t (&b)[8]) {
  const uint32_t lo = __builtin_amdgcn_perm(__builtin_amdgcn_perm(b[3], b[2], 0x0c0c0400u),
                                            __builtin_amdgcn_perm(b[1], b[0], 0x0c0c0400u), 0x05040100u);
  const uint32_t hi = __builtin_amdgcn_perm(__builtin_amdgcn_perm(b[7], b[6], 0x0c0c0400u),
                                            __builtin_amdgcn_perm(b[5], b[4], 0x0c0c0400u), 0x05040100u);
  return make_uint2(lo, hi);
}

// The same with the multiplier g = inv_sqrtb * rcp(delta) (0 for a step
// that is not positive) already formed, as static_code forms it.
__device__ __forceinline__ float static_mult(float delta, float inv_sqrtb) {
  return delta > 0.0f ? inv_sqrtb * __builtin_amdgcn_rcpf(delta) : 0.0f;
}
__device__ __forceinline__ uint32_t static_code_g(float u, float g) {
  const float r = __builtin_amdgcn_fmed3f(u * g, -7.0f, 7.0f);
  return __float_as_uint(r + kRoundMagic);
}

// The rest of the fused pass once the row's fp32 values are in registers:
// butterflies, row maximum, scales, codes.  `lds` must hold rows_per_wg * K
// floats when logT > 6; `red` is a 4-float shared array.  Every thread of the
// workgroup must call it.  ratio != nullptr writes z / Delta instead of codes;
// tiled selects the 16-row tiled code layout for Xq (K % 128 == 0).
// sdelta != nullptr selects the static per-channel quantizer (step
// sdelta[k] of channel k, token scale 1, see static_code); rotate_only
// writes the normalized rotation s_t * y in fp32 to `ratio` and nothing else;
// i8 quantizes to 8 bits (q_max = 127) and writes one byte per code, Xq
// [M][K] row-major; cmul != nullptr multiplies channel k of the rotated row
// by cmul[k] before the row maximum (the per-step weight fold W' diag(Delta)).
template <int C>
__device__ __forceinline__ void rq_core(float (&v)[C][8], const RowMap& m, int K, int logb, float s_t,
                                        float s_over_sqrtb, float* lds, float* red, uint8_t* __restrict__ Xq,
                                        float* __restrict__ xs, float* __restrict__ ratio, bool tiled = false,
                                        const float* __restrict__ sdelta = nullptr, bool rotate_only = false,
                                        bool i8 = false, const float* __restrict__ cmul = nullptr) {
  // Bits 0..2: inside each 8-channel chunk.
#pragma unroll
  for (int q = 0; q < 3; ++q) {
    const int h = 1 << q;
    if (q < logb) {
#pragma unroll
      for (int c = 0; c < C; ++c)
#pragma unroll
        for (int j = 0; j < 8; ++j)
          if ((j & h) == 0) {
            const float a = v[c][j], b = v[c][j + h];
            v[c][j] = a + b;
            v[c][j + h] = a - b;
          }
    }
  }

  // Bits 3 .. 3 + log2(lanes per row) - 1: across lanes of one wave.
  const int lane_bits = m.logT < 6 ? m.logT : 6;
  const int lane_stages = min(lane_bits, max(logb - 3, 0));
  if (lane_stages > 0) lane_stage<1>(v, m.lane);
  if (lane_stages > 1) lane_stage<2>(v, m.lane);
  if (lane_stages > 2) lane_stage<4>(v, m.lane);
  if (lane_stages > 3) lane_stage<8>(v, m.lane);
  if (lane_stages > 4) lane_stage_swap<16>(v);
  if (lane_stages > 5) lane_stage_swap<32>(v);

  // Wave bits (rows wider than 64 threads): one exchange through LDS.
  if (m.logT > 6) {
    const int wave_stages = min(m.logT - 6, max(logb - 9, 0));
    if (wave_stages > 0) {
      float* rl = lds + m.row_local * K;
#pragma unroll
      for (int c = 0; c < C; ++c) {
        float4* dst = reinterpret_cast<float4*>(rl + chan(m, c, 0));
        dst[0] = make_float4(v[c][0], v[c][1], v[c][2], v[c][3]);
        dst[1] = make_float4(v[c][4], v[c][5], v[c][6], v[c][7]);
      }
      __syncthreads();
      const int w = m.t >> 6;
      const int nw = 1 << wave_stages;
      const int wlow = w & (nw - 1);
      const int wbase = w & ~(nw - 1);
#pragma unroll
      for (int c = 0; c < C; ++c) {
        float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        for (int u = 0; u < nw; ++u) {
          const float sg = (__popc(wlow & u) & 1) ? -1.0f : 1.0f;
          const int tt = ((wbase | u) << 6) | m.lane;
          const float4* src = reinterpret_cast<const float4*>(rl + c * 8 * m.T + tt * 8);
          const float4 p0 = src[0], p1 = src[1];
          acc[0] = fmaf(sg, p0.x, acc[0]);
          acc[1] = fmaf(sg, p0.y, acc[1]);
          acc[2] = fmaf(sg, p0.z, acc[2]);
          acc[3] = fmaf(sg, p0.w, acc[3]);
          acc[4] = fmaf(sg, p1.x, acc[4]);
          acc[5] = fmaf(sg, p1.y, acc[5]);
          acc[6] = fmaf(sg, p1.z, acc[6]);
          acc[7] = fmaf(sg, p1.w, acc[7]);
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) v[c][j] = acc[j];
      }
    }
  }

  // Bits above the thread bits: chunk index c, in registers.
  {
    const int cbit0 = 3 + m.logT;
#pragma unroll
    for (int q = 0; q < 3; ++q) {
      const int h = 1 << q;
      if (h < C && cbit0 + q < logb) {
#pragma unroll
        for (int c = 0; c < C; ++c)
          if ((c & h) == 0 && c + h < C)
#pragma unroll
            for (int j = 0; j < 8; ++j) {
              const float a = v[c][j], b = v[c + h][j];
              v[c][j] = a + b;
              v[c + h][j] = a - b;
            }
      }
    }
  }

  if (cmul != nullptr) {
#pragma unroll
    for (int c = 0; c < C; ++c) {
      const float4* mp = reinterpret_cast<const float4*>(cmul + chan(m, c, 0));
      const float4 a = mp[0], b = mp[1];
      v[c][0] *= a.x; v[c][1] *= a.y; v[c][2] *= a.z; v[c][3] *= a.w;
      v[c][4] *= b.x; v[c][5] *= b.y; v[c][6] *= b.z; v[c][7] *= b.w;
    }
  }

  // Rotation only, or the static quantizer: no row maximum (the branch is
  // uniform over the grid, so skipping row_reduce's barrier is safe).
  if (rotate_only) {
    if (!m.valid) return;
    float* yr = ratio + m.row * static_cast<int64_t>(K);
#pragma unroll
    for (int c = 0; c < C; ++c) {
      float4* dst = reinterpret_cast<float4*>(yr + chan(m, c, 0));
      const float g = s_over_sqrtb;
      dst[0] = make_float4(v[c][0] * g, v[c][1] * g, v[c][2] * g, v[c][3] * g);
      dst[1] = make_float4(v[c][4] * g, v[c][5] * g, v[c][6] * g, v[c][7] * g);
    }
    return;
  }
  if (sdelta != nullptr) {
    if (!m.valid) return;
    if (m.t == 0) xs[m.row] = 1.0f;
    uint8_t* qr = Xq + m.row * static_cast<int64_t>(K / 2);
#pragma unroll
    for (int c = 0; c < C; ++c) {
      const float4* dp = reinterpret_cast<const float4*>(sdelta + chan(m, c, 0));
      const float4 d0 = dp[0], d1 = dp[1];
      const float d[8] = {d0.x, d0.y, d0.z, d0.w, d1.x, d1.y, d1.z, d1.w};
      uint32_t b[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) b[j] = static_code(v[c][j], d[j], s_over_sqrtb);
      const int p = chan(m, c, 0) / 2;
      uint8_t* dst = tiled ? Xq + tiled_offset(m.row, p, K / 128) : qr + p;
      *reinterpret_cast<uint32_t*>(dst) = pack8(b);
    }
    return;
  }

  // Row absolute maximum of the unnormalized transform.
  float amax = 0.0f;
#pragma unroll
  for (int c = 0; c < C; ++c)
#pragma unroll
    for (int j = 0; j < 8; ++j) amax = fmaxf(amax, fabsf(v[c][j]));
  amax = row_reduce<true>(amax, m, red);

  // Scalars: a_z = max|s_t y|, Delta = a_z / q_max, x_scale = Delta / s_t,
  // and the multiplier g = (s_t / sqrt(b)) / Delta taking the unnormalized
  // butterfly output u to z / Delta.  |u g| <= q_max up to rounding, so
  // round-half-even of u g never leaves [-q_max, q_max] and needs no clamp.
  const float a_z = amax * s_over_sqrtb;
  const float delta = a_z / (i8 ? 127.0f : 7.0f);
  const float g = delta > 0.0f ? s_over_sqrtb / delta : 0.0f;
  if (m.valid && m.t == 0) xs[m.row] = delta / s_t;
  if (!m.valid) return;

  if (ratio != nullptr) {
    float* rr = ratio + m.row * static_cast<int64_t>(K);
#pragma unroll
    for (int c = 0; c < C; ++c) {
      float4* dst = reinterpret_cast<float4*>(rr + chan(m, c, 0));
      dst[0] = make_float4(v[c][0] * g, v[c][1] * g, v[c][2] * g, v[c][3] * g);
      dst[1] = make_float4(v[c][4] * g, v[c][5] * g, v[c][6] * g, v[c][7] * g);
    }
    return;
  }

  if (i8) {
    uint8_t* qr8 = Xq + m.row * static_cast<int64_t>(K);
#pragma unroll
    for (int c = 0; c < C; ++c) {
      uint32_t b[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) b[j] = __float_as_uint(fmaf(v[c][j], g, kRoundMagic));
      *reinterpret_cast<uint2*>(qr8 + chan(m, c, 0)) = pack8_i8(b);
    }
    return;
  }
  uint8_t* qr = Xq + m.row * static_cast<int64_t>(K / 2);
#pragma unroll
  for (int c = 0; c < C; ++c) {
    uint32_t b[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) b[j] = __float_as_uint(fmaf(v[c][j], g, kRoundMagic));
    const int p = chan(m, c, 0) / 2;  // a multiple of 4: the dword stays inside one 16-byte piece
    uint8_t* dst = tiled ? Xq + tiled_offset(m.row, p, K / 128) : qr + p;
    *reinterpret_cast<uint32_t*>(dst) = pack8(b);
  }
}

}  // namespace rqd
}  // namespace oq
