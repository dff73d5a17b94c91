// Fused online Hadamard rotation + per-step scale + per-token int4 quantization.
//
// Section 4.1 (eq:composite_rot, eq:blockdiag, eq:transform): the activation is
// multiplied by the block-diagonal normalized Hadamard matrix, blocks of b
// contiguous channels, Sylvester order.  Section 4.2 (eq:scale, eq:quant,
// eq:perstep_scale): per-token symmetric quantizer with q_max = 7, the step
// scale s_t multiplied in before it and divided out of the token scale.
//
// Work split.  One row (token) of K channels is owned by T = 2^logT threads;
// thread t holds C chunks of 8 consecutive channels, channel
//     k = c * 8T + t * 8 + j,   c < C, j < 8,
// loaded with one 16-byte load per chunk (consecutive lanes read consecutive
// 16-byte pieces: fully coalesced).  The Walsh-Hadamard transform is a product
// of independent butterflies, one per index bit below log2(b), and they
// commute, so each bit is handled where it lives:
//   bits 0..2          (j)      in registers,
//   bits 3..3+log2(min(T,64))-1  across lanes with ds_swizzle / DPP,
//   wave bits (T > 64)          through LDS, all wave bits in one exchange,
//   bits above the thread bits (c)  in registers.
// The row's absolute maximum is reduced across the same lanes / waves; the
// codes are rounded half-to-even with the 1.5*2^23 add inside one FMA and the
// low nibble of the float's bit pattern is the two's-complement code.
//
// Arithmetic is fp32 on the unnormalized butterflies; 1/sqrt(b) and s_t are
// applied to the per-row scalars only (scale the max, not every element), which
// is the same map in exact arithmetic.
#include <cmath>

#include "common.h"

namespace oq {
namespace {

constexpr float kRoundMagic = 12582912.0f;  // 1.5 * 2^23

__device__ __forceinline__ float lane_xor(float v, int m) {
  // m is a wave-uniform power of two below 64.
  int x = __float_as_int(v);
  switch (m) {
    case 1: return __int_as_float(__builtin_amdgcn_mov_dpp(x, 0xB1, 0xF, 0xF, false));  // quad_perm [1,0,3,2]
    case 2: return __int_as_float(__builtin_amdgcn_mov_dpp(x, 0x4E, 0xF, 0xF, false));  // quad_perm [2,3,0,1]
    case 4: return __int_as_float(__builtin_amdgcn_ds_swizzle(x, 0x1F | (4 << 10)));
    case 8: return __int_as_float(__builtin_amdgcn_ds_swizzle(x, 0x1F | (8 << 10)));
    case 16: return __int_as_float(__builtin_amdgcn_ds_swizzle(x, 0x1F | (16 << 10)));
    default: return __shfl_xor(v, 32, 64);
  }
}

__device__ __forceinline__ float half_bits_to_float(uint32_t h) {
  return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(h)));
}

template <int C>
__global__ __launch_bounds__(256) void rq_kernel(const uint16_t* __restrict__ X, int64_t M, int K,
                                                 int64_t ldx, int logT, int logb, float s_t,
                                                 float s_over_sqrtb, uint8_t* __restrict__ Xq,
                                                 float* __restrict__ xs, float* __restrict__ ratio) {
  extern __shared__ float lds[];  // [rows_per_wg][K] when a row spans several waves
  __shared__ float wave_max[4];

  const int T = 1 << logT;
  const int tid = threadIdx.x;
  const int row_local = tid >> logT;
  const int t = tid & (T - 1);
  const int rows_per_wg = blockDim.x >> logT;
  const int64_t row = static_cast<int64_t>(blockIdx.x) * rows_per_wg + row_local;
  const bool valid = row < M;
  const int lane = tid & 63;

  float v[C][8];
  {
    const uint16_t* xr = X + (valid ? row : 0) * ldx;
#pragma unroll
    for (int c = 0; c < C; ++c) {
      uint4 raw = make_uint4(0, 0, 0, 0);
      if (valid) raw = *reinterpret_cast<const uint4*>(xr + c * 8 * T + t * 8);
      const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        v[c][2 * q] = half_bits_to_float(w[q] & 0xFFFFu);
        v[c][2 * q + 1] = half_bits_to_float(w[q] >> 16);
      }
    }
  }

  // Bits 0..2: inside each 8-channel chunk.
#pragma unroll
  for (int m = 0; m < 3; ++m) {
    const int h = 1 << m;
    if (h < (1 << logb)) {
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

  // Bits 3 .. 3+log2(lanes per row)-1: across lanes of one wave.
  const int lane_bits = logT < 6 ? logT : 6;
  const int lane_stages = min(lane_bits, max(logb - 3, 0));
  for (int m = 0; m < lane_stages; ++m) {
    const int h = 1 << m;
    const float sgn = (lane & h) ? -1.0f : 1.0f;
#pragma unroll
    for (int c = 0; c < C; ++c)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float p = lane_xor(v[c][j], h);
        v[c][j] = fmaf(sgn, v[c][j], p);  // upper partner: p - v ; lower: p + v
      }
  }

  // Wave bits (rows wider than 64 threads): one exchange through LDS.
  if (logT > 6) {
    const int wave_stages = min(logT - 6, max(logb - 9, 0));
    if (wave_stages > 0) {
      float* rl = lds + row_local * K;
#pragma unroll
      for (int c = 0; c < C; ++c) {
        float4* dst = reinterpret_cast<float4*>(rl + c * 8 * T + t * 8);
        dst[0] = make_float4(v[c][0], v[c][1], v[c][2], v[c][3]);
        dst[1] = make_float4(v[c][4], v[c][5], v[c][6], v[c][7]);
      }
      __syncthreads();
      const int w = t >> 6;
      const int nw = 1 << wave_stages;
      const int wlow = w & (nw - 1);
      const int wbase = w & ~(nw - 1);
#pragma unroll
      for (int c = 0; c < C; ++c) {
        float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        for (int u = 0; u < nw; ++u) {
          const float sg = (__popc(wlow & u) & 1) ? -1.0f : 1.0f;
          const int tt = ((wbase | u) << 6) | lane;
          const float4* src = reinterpret_cast<const float4*>(rl + c * 8 * T + tt * 8);
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
    const int cbit0 = 3 + logT;
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

  // Row absolute maximum.
  float amax = 0.0f;
#pragma unroll
  for (int c = 0; c < C; ++c)
#pragma unroll
    for (int j = 0; j < 8; ++j) amax = fmaxf(amax, fabsf(v[c][j]));
  for (int m = 0; m < lane_bits; ++m) amax = fmaxf(amax, lane_xor(amax, 1 << m));
  if (logT > 6) {
    // One row per workgroup here (T >= 128 implies rows_per_wg <= 2; each row
    // has its own pair of slots).
    const int w = tid >> 6;
    if (lane == 0) wave_max[w] = amax;
    __syncthreads();
    const int nwr = T >> 6;
    const int first = row_local * nwr;
    amax = 0.0f;
    for (int u = 0; u < nwr; ++u) amax = fmaxf(amax, wave_max[first + u]);
  }

  // Scalars: a_z = max|s_t y|, Delta = a_z / 7, x_scale = Delta / s_t, and the
  // per-element multiplier g = (s_t / sqrt(b)) / Delta mapping the unnormalized
  // butterfly output u to the ratio z / Delta.
  const float a_z = amax * s_over_sqrtb;
  const float delta = a_z / 7.0f;
  const float g = delta > 0.0f ? s_over_sqrtb / delta : 0.0f;
  if (valid && t == 0) xs[row] = delta / s_t;
  if (!valid) return;

  if (ratio != nullptr) {
    float* rr = ratio + row * static_cast<int64_t>(K);
#pragma unroll
    for (int c = 0; c < C; ++c) {
      float4* dst = reinterpret_cast<float4*>(rr + c * 8 * T + t * 8);
      dst[0] = make_float4(v[c][0] * g, v[c][1] * g, v[c][2] * g, v[c][3] * g);
      dst[1] = make_float4(v[c][4] * g, v[c][5] * g, v[c][6] * g, v[c][7] * g);
    }
    return;
  }

  uint8_t* qr = Xq + row * static_cast<int64_t>(K / 2);
#pragma unroll
  for (int c = 0; c < C; ++c) {
    uint32_t word = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float r = fminf(fmaxf(v[c][j] * g, -7.0f), 7.0f);
      const uint32_t bits = __float_as_uint(r + kRoundMagic);
      word |= (bits & 0xFu) << (4 * j);
    }
    *reinterpret_cast<uint32_t*>(qr + (c * 8 * T + t * 8) / 2) = word;
  }
}

}  // namespace

bool rq_plan(int64_t K, RQPlan* p) {
  if (K < 8 || K % 8 != 0) return false;
  const int64_t nvec = K / 8;
  static const int kChunks[] = {8, 6, 4, 3, 2, 1};
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

int rq_validate(const void* X, int64_t M, int64_t K, int64_t ldx, int had_block, const void* out,
                const float* x_scale) {
  if (M < 0 || K < 8 || K % 8 != 0 || K > 16384 || ldx < K) return OQ_ERR_SHAPE;
  if (!is_pow2(had_block) || had_block > OQ_MAX_HAD_BLOCK || K % had_block != 0) return OQ_ERR_SHAPE;
  RQPlan p;
  if (!rq_plan(K, &p)) return OQ_ERR_SHAPE;
  if (ldx % 8 != 0) return OQ_ERR_ALIGN;
  if (M == 0) return OQ_OK;  // nothing is read or written; pointers may be NULL
  if (!X || !out || !x_scale) return OQ_ERR_NULL;
  if (!aligned(X, 16) || !aligned(out, 16) || !aligned(x_scale, 4)) return OQ_ERR_ALIGN;
  return OQ_OK;
}

int rq_launch(const void* X, int64_t M, int64_t K, int64_t ldx, int had_block, float s_t, uint8_t* Xq,
              float* x_scale, float* ratio, hipStream_t stream) {
  if (M == 0) return OQ_OK;
  RQPlan p;
  rq_plan(K, &p);
  const int T = 1 << p.logT;
  const int threads = T >= 256 ? T : 256;
  const int rows_per_wg = threads / T;
  const int64_t grid = (M + rows_per_wg - 1) / rows_per_wg;
  const size_t lds = p.logT > 6 ? static_cast<size_t>(rows_per_wg) * K * sizeof(float) : 0;
  const int logb = ilog2(had_block);
  const float s_over_sqrtb = static_cast<float>(static_cast<double>(s_t) / std::sqrt(static_cast<double>(had_block)));
  const uint16_t* x = static_cast<const uint16_t*>(X);
#define OQ_RQ_CASE(CH)                                                                                 \
  case CH:                                                                                             \
    hipLaunchKernelGGL(rq_kernel<CH>, dim3(static_cast<unsigned>(grid)), dim3(threads), lds, stream, x, \
                       M, static_cast<int>(K), ldx, p.logT, logb, s_t, s_over_sqrtb, Xq, x_scale, ratio); \
    break;
  switch (p.chunks) {
    OQ_RQ_CASE(1)
    OQ_RQ_CASE(2)
    OQ_RQ_CASE(3)
    OQ_RQ_CASE(4)
    OQ_RQ_CASE(6)
    OQ_RQ_CASE(8)
    default:
      return OQ_ERR_SHAPE;
  }
#undef OQ_RQ_CASE
  return launch_status();
}

}  // namespace oq

extern "C" int oq_rotate_quantize_act(const void* X, int64_t M, int64_t K, int64_t ldx, int32_t had_block,
                                      const float* s_table, int32_t t, uint8_t* Xq, float* x_scale,
                                      void* stream) {
  int st = oq::rq_validate(X, M, K, ldx, had_block, Xq, x_scale);
  if (st != OQ_OK) return st;
  if (t < 0) return OQ_ERR_ARG;
  if (M == 0) return OQ_OK;
  const float s = s_table ? s_table[t] : 1.0f;
  if (!(s > 0.0f) || !std::isfinite(s)) return OQ_ERR_ARG;
  if ((st = oq::device_check()) != OQ_OK) return st;
  return oq::rq_launch(X, M, K, ldx, had_block, s, Xq, x_scale, nullptr, static_cast<hipStream_t>(stream));
}

extern "C" int oq_rotate_debug_f32(const void* X, int64_t M, int64_t K, int64_t ldx, int32_t had_block,
                                   const float* s_table, int32_t t, float* ratio, float* x_scale,
                                   void* stream) {
  int st = oq::rq_validate(X, M, K, ldx, had_block, ratio, x_scale);
  if (st != OQ_OK) return st;
  if (t < 0) return OQ_ERR_ARG;
  if (M == 0) return OQ_OK;
  const float s = s_table ? s_table[t] : 1.0f;
  if (!(s > 0.0f) || !std::isfinite(s)) return OQ_ERR_ARG;
  if ((st = oq::device_check()) != OQ_OK) return st;
  return oq::rq_launch(X, M, K, ldx, had_block, s, nullptr, x_scale, ratio, static_cast<hipStream_t>(stream));
}

extern "C" int oq_quantize_weights(const void* W_u, int64_t N, int64_t K, int64_t ldw, int32_t had_block,
                                   uint8_t* Wq, float* w_scale, void* stream) {
  int st = oq::rq_validate(W_u, N, K, ldw, had_block, Wq, w_scale);
  if (st != OQ_OK || N == 0) return st;
  if ((st = oq::device_check()) != OQ_OK) return st;
  return oq::rq_launch(W_u, N, K, ldw, had_block, 1.0f, Wq, w_scale, nullptr, static_cast<hipStream_t>(stream));
}
