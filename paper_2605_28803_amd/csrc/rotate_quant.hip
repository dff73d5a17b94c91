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
#include "rq_device.h"

namespace oq {
namespace {

template <int C>
__global__ __launch_bounds__(256) void rq_kernel(const uint16_t* __restrict__ X, int64_t M, int K,
                                                 int64_t ldx, int logT, int logb, float s_t,
                                                 float s_over_sqrtb, uint8_t* __restrict__ Xq,
                                                 float* __restrict__ xs, float* __restrict__ ratio) {
  extern __shared__ float lds[];  // [rows_per_wg][K] when a row spans several waves
  __shared__ float red[4];
  const rqd::RowMap m = rqd::row_map(logT, M);
  float v[C][8];
  rqd::load_row_f16<C>(v, X, ldx, m);
  rqd::rq_core<C>(v, m, K, logb, s_t, s_over_sqrtb, lds, red, Xq, xs, ratio);
}

// ---------------------------------------------------------------------------
// Matrix-core variant for Hadamard blocks b >= 32 and K = 512 * NG * W.
//
// The first five butterfly stages (H_32 over each chunk of 32 channels) are a
// product with a constant +-1 matrix, done on v_mfma_f32_16x16x32_f16 straight
// from the fp16 input (exact products, fp32 sums): B operand = 16 chunks x 32
// channels of the row, A operand = H_32 with its rows permuted so that lane l
// receives channels 8q .. 8q+7 (q = l / 16) of chunk l % 16 -- eight
// consecutive channels, i.e. one packed dword of codes.  Chunk index bits 0-3
// are lane bits 0-3 (four cross-lane butterflies), the next bits are the
// register group index g.  A row wider than 4096 channels spans W waves; its
// top log2(W) channel bits are the wave index, and the butterflies over them
// run after a transpose through LDS that gives each wave all W wave-values of
// NG / W of the groups.  One wave (W = 1) or one workgroup (W > 1) per row
// pass, no prefetch: the register budget stays small enough for several
// workgroups per CU, and their loads overlap each other's arithmetic.
// ---------------------------------------------------------------------------

typedef _Float16 rv8h __attribute__((ext_vector_type(8)));
typedef float rv4f __attribute__((ext_vector_type(4)));

// Lane l's A fragments: A[m = l % 16][k = 8 (l / 16) + i] = H_32[rho(m)][k],
// rho(4q + r) = 8q + r (first product) and 8q + 4 + r (second product).
__device__ __forceinline__ void hadamard_frags(int lane, rv8h& a1, rv8h& a2) {
  const int m = lane & 15;
  const int row1 = 8 * (m >> 2) + (m & 3), row2 = row1 + 4;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int k = 8 * (lane >> 4) + i;
    a1[i] = (__popc(row1 & k) & 1) ? static_cast<_Float16>(-1.0f) : static_cast<_Float16>(1.0f);
    a2[i] = (__popc(row2 & k) & 1) ? static_cast<_Float16>(-1.0f) : static_cast<_Float16>(1.0f);
  }
}

template <int NG, int W, bool FULL>
__global__ __launch_bounds__(256) void rq_mfma_kernel(const uint16_t* __restrict__ X, int64_t M, int64_t ldx, int logb,
                                                      float s_t, float s_over_sqrtb, uint8_t* __restrict__ Xq,
                                                      float* __restrict__ xs, float* __restrict__ ratio) {
  // W > 1: [4 waves][NG groups][2 halves][64 lanes] float4 (consecutive lanes
  // hit consecutive 16-byte words: no bank conflicts on either side).
  extern __shared__ float4 xch[];
  __shared__ float red[4];
  constexpr int K = NG * W * 512;
  constexpr int RPB = 4 / W;  // rows per workgroup
  constexpr int LOGNG = NG >= 8 ? 3 : NG >= 4 ? 2 : NG >= 2 ? 1 : 0;
  constexpr int LOGW = W >= 4 ? 2 : W >= 2 ? 1 : 0;
  constexpr int GW = NG / W;  // groups per wave after the transpose
  static_assert(W == 1 || (NG % W == 0 && (NG & (NG - 1)) == 0), "NG must be a power of two >= W when W > 1");
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int rsub = wv / W, wr = wv % W;
  const int cl = lane & 15, q = lane >> 4;
  const int64_t row = static_cast<int64_t>(blockIdx.x) * RPB + rsub;
  const bool valid = row < M;
  // Butterfly over channel bit `bit` is needed when bit < log2(b); FULL means
  // b = K (every stage, no branches).
  auto need = [&](int bit) { return FULL || bit < logb; };

  // Element (g, e) of this lane is channel ((wr * NG + g) * 16 + cl) * 32 + 8q + e.
  rv8h cur[NG];
  {
    const uint16_t* xr = X + (valid ? row : 0) * ldx + (wr * NG * 16 + cl) * 32 + 8 * q;
#pragma unroll
    for (int g = 0; g < NG; ++g) cur[g] = valid ? *reinterpret_cast<const rv8h*>(xr + g * 512) : rv8h{};
  }
  rv8h a1, a2;
  hadamard_frags(lane, a1, a2);

  // H_32 on the matrix cores.
  float v[NG][8];
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    const rv4f d1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(a1, cur[g], rv4f{0, 0, 0, 0}, 0, 0, 0);
    const rv4f d2 = __builtin_amdgcn_mfma_f32_16x16x32_f16(a2, cur[g], rv4f{0, 0, 0, 0}, 0, 0, 0);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      v[g][r] = d1[r];
      v[g][4 + r] = d2[r];
    }
  }
  // Channel bits 5..8: chunk bits 0..3 = lane bits 0..3.
  if (need(5)) rqd::lane_stage<1>(v, lane);
  if (need(6)) rqd::lane_stage<2>(v, lane);
  if (need(7)) rqd::lane_stage<4>(v, lane);
  if (need(8)) rqd::lane_stage<8>(v, lane);
  // Channel bits 9 .. 9 + log2(NG) - 1: group index g in registers.
#pragma unroll
  for (int t = 0; t < LOGNG + 1; ++t) {
    const int h = 1 << t;
    if (h < NG && need(9 + t)) {
#pragma unroll
      for (int g = 0; g < NG; ++g)
        if ((g & h) == 0 && g + h < NG)
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float x0 = v[g][e], x1 = v[g + h][e];
            v[g][e] = x0 + x1;
            v[g + h][e] = x0 - x1;
          }
    }
  }
  // Register slot s holds channel group G(s) (units of 512 channels):
  // G = wr * NG + s without the wave transpose, and with it (s = gi * W + u)
  // G = u * NG + wr * GW + gi.
  const int wbit0 = 9 + LOGNG;
  const bool xpose = W > 1 && need(wbit0);
  if constexpr (W > 1) {
    if (xpose) {
      float4* mine = xch + static_cast<int64_t>(wv) * NG * 128 + lane;
#pragma unroll
      for (int g = 0; g < NG; ++g) {
        mine[g * 128] = make_float4(v[g][0], v[g][1], v[g][2], v[g][3]);
        mine[g * 128 + 64] = make_float4(v[g][4], v[g][5], v[g][6], v[g][7]);
      }
      __syncthreads();
#pragma unroll
      for (int gi = 0; gi < GW; ++gi)
#pragma unroll
        for (int u = 0; u < W; ++u) {
          const float4* src = xch + static_cast<int64_t>((rsub * W + u) * NG + wr * GW + gi) * 128 + lane;
          const float4 p0 = src[0], p1 = src[64];
          float* d = v[gi * W + u];
          d[0] = p0.x; d[1] = p0.y; d[2] = p0.z; d[3] = p0.w;
          d[4] = p1.x; d[5] = p1.y; d[6] = p1.z; d[7] = p1.w;
        }
      // Wave bits in registers: slot bits 0 .. log2(W) - 1 are u.
#pragma unroll
      for (int t = 0; t < LOGW; ++t) {
        const int h = 1 << t;
        if (need(wbit0 + t)) {
#pragma unroll
          for (int s = 0; s < NG; ++s)
            if ((s & h) == 0)
#pragma unroll
              for (int e = 0; e < 8; ++e) {
                const float x0 = v[s][e], x1 = v[s + h][e];
                v[s][e] = x0 + x1;
                v[s + h][e] = x0 - x1;
              }
        }
      }
    }
  }

  // Row maximum: registers, lanes, then the W waves of the row.
  float amax = 0.0f;
#pragma unroll
  for (int g = 0; g < NG; ++g)
#pragma unroll
    for (int e = 0; e < 8; ++e) amax = fmaxf(amax, fabsf(v[g][e]));
  amax = fmaxf(amax, rqd::lane_xor<1>(amax));
  amax = fmaxf(amax, rqd::lane_xor<2>(amax));
  amax = fmaxf(amax, rqd::lane_xor<4>(amax));
  amax = fmaxf(amax, rqd::lane_xor<8>(amax));
  amax = fmaxf(amax, rqd::lane_xor<16>(amax));
  amax = fmaxf(amax, __shfl_xor(amax, 32, 64));
  if constexpr (W > 1) {
    if (lane == 0) red[wv] = amax;
    __syncthreads();
    amax = red[rsub * W];
#pragma unroll
    for (int u = 1; u < W; ++u) amax = fmaxf(amax, red[rsub * W + u]);
  }

  const float a_z = amax * s_over_sqrtb;
  const float delta = a_z / 7.0f;
  const float gm = delta > 0.0f ? s_over_sqrtb / delta : 0.0f;
  if (!valid) return;
  if (wr == 0 && lane == 0) xs[row] = delta / s_t;
  auto group_of = [&](int s) { return xpose ? (s % W) * NG + wr * GW + s / W : wr * NG + s; };
  if (ratio != nullptr) {
#pragma unroll
    for (int s = 0; s < NG; ++s) {
      float* rr = ratio + row * K + (group_of(s) * 16 + cl) * 32 + 8 * q;
      reinterpret_cast<float4*>(rr)[0] = make_float4(v[s][0] * gm, v[s][1] * gm, v[s][2] * gm, v[s][3] * gm);
      reinterpret_cast<float4*>(rr)[1] = make_float4(v[s][4] * gm, v[s][5] * gm, v[s][6] * gm, v[s][7] * gm);
    }
    return;
  }
  uint8_t* qr = Xq + row * (K / 2);
#pragma unroll
  for (int s = 0; s < NG; ++s) {
    uint32_t b[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) b[e] = __float_as_uint(fmaf(v[s][e], gm, rqd::kRoundMagic));
    *reinterpret_cast<uint32_t*>(qr + (group_of(s) * 16 + cl) * 16 + 4 * q) = rqd::pack8(b);
  }
}

// (NG, W) of the matrix-core variant for K channels, or false.
bool rq_mfma_shape(int64_t K, int* ng, int* w) {
  switch (K) {
    case 512: *ng = 1; *w = 1; return true;
    case 1024: *ng = 2; *w = 1; return true;
    case 1536: *ng = 3; *w = 1; return true;
    case 2048: *ng = 4; *w = 1; return true;
    case 3072: *ng = 6; *w = 1; return true;
    case 4096: *ng = 8; *w = 1; return true;
    case 8192: *ng = 8; *w = 2; return true;
    case 16384: *ng = 8; *w = 4; return true;
    default: return false;
  }
}

int rq_mfma_launch(const void* X, int64_t M, int64_t K, int64_t ldx, int had_block, float s_t, uint8_t* Xq,
                   float* x_scale, float* ratio, hipStream_t stream) {
  int ng = 0, w = 0;
  rq_mfma_shape(K, &ng, &w);
  const int logb = ilog2(had_block);
  const float s_over_sqrtb = static_cast<float>(static_cast<double>(s_t) / std::sqrt(static_cast<double>(had_block)));
  const int rpb = 4 / w;
  const size_t lds = w > 1 ? static_cast<size_t>(4) * ng * 128 * sizeof(float4) : 0;
  // One row per wave (W = 1) or per workgroup (W > 1).
  const unsigned grid = static_cast<unsigned>((M + rpb - 1) / rpb);
  const uint16_t* x = static_cast<const uint16_t*>(X);
#define OQ_RQM(NG, W)                                                                                         \
  if (ng == NG && w == W) {                                                                                   \
    if (had_block == K)                                                                                       \
      hipLaunchKernelGGL((rq_mfma_kernel<NG, W, true>), dim3(grid), dim3(256), lds, stream, x, M, ldx, logb,  \
                         s_t, s_over_sqrtb, Xq, x_scale, ratio);                                              \
    else                                                                                                      \
      hipLaunchKernelGGL((rq_mfma_kernel<NG, W, false>), dim3(grid), dim3(256), lds, stream, x, M, ldx, logb, \
                         s_t, s_over_sqrtb, Xq, x_scale, ratio);                                              \
    return launch_status();                                                                                   \
  }
  OQ_RQM(1, 1)
  OQ_RQM(2, 1)
  OQ_RQM(3, 1)
  OQ_RQM(4, 1)
  OQ_RQM(6, 1)
  OQ_RQM(8, 1)
  OQ_RQM(8, 2)
  OQ_RQM(8, 4)
#undef OQ_RQM
  return OQ_ERR_SHAPE;
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
  int ng = 0, w = 0;
  if (had_block >= 32 && rq_mfma_shape(K, &ng, &w))
    return rq_mfma_launch(X, M, K, ldx, had_block, s_t, Xq, x_scale, ratio, stream);
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
