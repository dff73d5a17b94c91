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
#include "rq_mfma.h"

namespace oq {
namespace {

// Re-layout of packed codes [R][K/2] into the 16-row tiled layout: one thread
// per 16-byte piece; rows past R in the last block are written as zeros.
__global__ __launch_bounds__(256) void tile_codes_kernel(const uint8_t* __restrict__ Q, int64_t R, int64_t K,
                                                         uint8_t* __restrict__ T) {
  const int64_t pieces_per_row = K / 32;
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t rows16 = (R + 15) / 16 * 16;
  if (i >= rows16 * pieces_per_row) return;
  const int64_t r = i / pieces_per_row, p = (i % pieces_per_row) * 16;
  const uint4 v = r < R ? *reinterpret_cast<const uint4*>(Q + r * (K / 2) + p) : make_uint4(0, 0, 0, 0);
  *reinterpret_cast<uint4*>(T + tiled_offset(r, p, K / 128)) = v;
}

template <int C>
__global__ __launch_bounds__(256) void rq_kernel(const uint16_t* __restrict__ X, int64_t M, int K,
                                                 int64_t ldx, int logT, int logb, float s_t,
                                                 float s_over_sqrtb, uint8_t* __restrict__ Xq,
                                                 float* __restrict__ xs, float* __restrict__ ratio, bool tiled,
                                                 const float* __restrict__ sdelta, bool rotate_only, bool i8,
                                                 const float* __restrict__ cmul) {
  extern __shared__ float lds[];  // [rows_per_wg][K] when a row spans several waves
  __shared__ float red[4];
  const rqd::RowMap m = rqd::row_map(logT, M);
  float v[C][8];
  rqd::load_row_f16<C>(v, X, ldx, m);
  rqd::rq_core<C>(v, m, K, logb, s_t, s_over_sqrtb, lds, red, Xq, xs, ratio, tiled, sdelta, rotate_only, i8, cmul);
}

// One row per wave (W = 1), per workgroup (W = 2, 4: four waves), or per
// three-wave workgroup (W = 3).
template <int NG, int W, bool FULL>
__global__ __launch_bounds__(256) void rq_mfma_kernel(const uint16_t* __restrict__ X, int64_t M, int64_t ldx, int logb,
                                                      float s_t, float s_over_sqrtb, uint8_t* __restrict__ Xq,
                                                      float* __restrict__ xs, float* __restrict__ ratio, bool tiled,
                                                      const float* __restrict__ sdelta, bool rotate_only, bool i8,
                                                 const float* __restrict__ cmul) {
  // W > 1: [4 waves][NG groups][2 halves][32 lanes] float4, one half of the
  // lanes at a time (consecutive lanes hit consecutive 16-byte words).
  extern __shared__ float4 xch[];
  __shared__ float red[4];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int wr = wv % W;
  const int64_t row = static_cast<int64_t>(blockIdx.x) * rqm::Shape<NG, W>::RPB + wv / W;
  const bool valid = row < M;
  rqm::rv8h cur[NG];
  const uint16_t* xr = X + (valid ? row : 0) * ldx;
#pragma unroll
  for (int g = 0; g < NG; ++g)
    cur[g] = valid ? *reinterpret_cast<const rqm::rv8h*>(xr + rqm::chan0<NG>(wr, g, lane)) : rqm::rv8h{};
  // Static steps with one row per wave: the workgroup forms the K
  // multipliers once in LDS while the rows' loads are in flight.
  const float* sg = nullptr;
  if constexpr (W == 1) {
    if (sdelta != nullptr) {
      float* gt = reinterpret_cast<float*>(xch);
      constexpr int K = rqm::Shape<NG, W>::K;
      for (int k4 = threadIdx.x; k4 < K / 4; k4 += 256) {
        const float4 d = reinterpret_cast<const float4*>(sdelta)[k4];
        reinterpret_cast<float4*>(gt)[k4] =
            make_float4(rqd::static_mult(d.x, s_over_sqrtb), rqd::static_mult(d.y, s_over_sqrtb),
                        rqd::static_mult(d.z, s_over_sqrtb), rqd::static_mult(d.w, s_over_sqrtb));
      }
      __syncthreads();
      sg = gt;
    }
  }
  rqm::rv8h a1, a2;
  rqm::hadamard_frags(lane, a1, a2);
  rqm::rq_row<NG, W, FULL>(cur, a1, a2, row, valid, lane, wv, logb, s_t, s_over_sqrtb, Xq, xs, ratio, xch, red, tiled,
                           sdelta, rotate_only, i8, cmul, sg);
}

// (NG, W) of the matrix-core variant for K channels, or false.
bool rq_mfma_shape(int64_t K, int* ng, int* w) {
  switch (K) {
    case 512: *ng = 1; *w = 1; return true;
    case 1024: *ng = 2; *w = 1; return true;
    case 1536: *ng = 1; *w = 3; return true;  // three waves per row, one 512-channel block each
    case 2048: *ng = 4; *w = 1; return true;
    case 3072: *ng = 6; *w = 1; return true;
    case 4096: *ng = 8; *w = 1; return true;
    case 6144: *ng = 4; *w = 3; return true;  // the 6144-channel MLP input: three waves of one 2048-block each
    case 8192: *ng = 4; *w = 4; return true;  // 68 VGPRs (7 waves per SIMD) against 136 for (8, 2)
    case 16384: *ng = 8; *w = 4; return true;
    default: return false;
  }
}

int rq_mfma_launch(const void* X, int64_t M, int64_t K, int64_t ldx, int had_block, float s_t, uint8_t* Xq,
                   float* x_scale, float* ratio, hipStream_t stream, bool tiled, const float* sdelta,
                   bool rotate_only, bool i8, const float* cmul) {
  int ng = 0, w = 0;
  rq_mfma_shape(K, &ng, &w);
  // Few rows (the action tokens): two waves per 4096-channel row halve the
  // serial work of a wave (at most 512 rows: at most one wave per SIMD).
  if (K == 4096 && M <= 512) { ng = 4; w = 2; }
  const int logb = ilog2(had_block);
  const float s_over_sqrtb = static_cast<float>(static_cast<double>(s_t) / std::sqrt(static_cast<double>(had_block)));
  const int rpb = w == 3 ? 1 : 4 / w;
  const unsigned threads = w == 3 ? 192 : 256;
  const size_t lds = (w == 2 || w == 4) ? static_cast<size_t>(4) * ng * 64 * sizeof(float4)
                                        : (w == 1 && sdelta != nullptr ? static_cast<size_t>(K) * sizeof(float) : 0);
  // One row per wave (W = 1) or per workgroup (W > 1).
  const unsigned grid = static_cast<unsigned>((M + rpb - 1) / rpb);
  const uint16_t* x = static_cast<const uint16_t*>(X);
#define OQ_RQM(NG, W)                                                                                         \
  if (ng == NG && w == W) {                                                                                   \
    if (had_block == K)                                                                                       \
      hipLaunchKernelGGL((rq_mfma_kernel<NG, W, true>), dim3(grid), dim3(threads), lds, stream, x, M, ldx, logb, \
                         s_t, s_over_sqrtb, Xq, x_scale, ratio, tiled, sdelta, rotate_only, i8, cmul);        \
    else                                                                                                      \
      hipLaunchKernelGGL((rq_mfma_kernel<NG, W, false>), dim3(grid), dim3(threads), lds, stream, x, M, ldx, logb, \
                         s_t, s_over_sqrtb, Xq, x_scale, ratio, tiled, sdelta, rotate_only, i8, cmul);        \
    return launch_status();                                                                                   \
  }
  OQ_RQM(1, 1)
  OQ_RQM(2, 1)
  OQ_RQM(1, 3)
  OQ_RQM(4, 1)
  OQ_RQM(6, 1)
  OQ_RQM(8, 1)
  OQ_RQM(4, 2)
  OQ_RQM(4, 3)
  OQ_RQM(4, 4)
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
              float* x_scale, float* ratio, hipStream_t stream, bool tiled, const float* sdelta,
              bool rotate_only, bool i8, const float* cmul) {
  if (M == 0) return OQ_OK;
  int ng = 0, w = 0;
  // (With three waves per row a Hadamard block must not span waves: b <= 512 NG.)
  if (had_block >= 32 && rq_mfma_shape(K, &ng, &w) && (w != 3 || had_block <= 512 * ng))
    return rq_mfma_launch(X, M, K, ldx, had_block, s_t, Xq, x_scale, ratio, stream, tiled, sdelta, rotate_only,
                          i8, cmul);
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
                       M, static_cast<int>(K), ldx, p.logT, logb, s_t, s_over_sqrtb, Xq, x_scale, ratio, \
                       tiled, sdelta, rotate_only, i8, cmul);                                          \
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

extern "C" int oq_rotate_quantize_act_tiled(const void* X, int64_t M, int64_t K, int64_t ldx, int32_t had_block,
                                            const float* s_table, int32_t t, uint8_t* Xt, float* x_scale,
                                            void* stream) {
  int st = oq::rq_validate(X, M, K, ldx, had_block, Xt, x_scale);
  if (st != OQ_OK) return st;
  if (K % 128 != 0) return OQ_ERR_SHAPE;
  if (t < 0) return OQ_ERR_ARG;
  if (M == 0) return OQ_OK;
  const float s = s_table ? s_table[t] : 1.0f;
  if (!(s > 0.0f) || !std::isfinite(s)) return OQ_ERR_ARG;
  if ((st = oq::device_check()) != OQ_OK) return st;
  return oq::rq_launch(X, M, K, ldx, had_block, s, Xt, x_scale, nullptr, static_cast<hipStream_t>(stream), true);
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

extern "C" int oq_codes_to_tiled(const uint8_t* Q, int64_t rows, int64_t K, uint8_t* T, void* stream) {
  if (rows < 0 || K < 128 || K % 128 != 0 || K > 16384) return OQ_ERR_SHAPE;
  if (rows == 0) return OQ_OK;
  if (!Q || !T) return OQ_ERR_NULL;
  if (!oq::aligned(Q, 16) || !oq::aligned(T, 16)) return OQ_ERR_ALIGN;
  int st = oq::device_check();
  if (st != OQ_OK) return st;
  const int64_t pieces = (rows + 15) / 16 * 16 * (K / 32);
  hipLaunchKernelGGL(oq::tile_codes_kernel, dim3(static_cast<unsigned>((pieces + 255) / 256)), dim3(256), 0,
                     static_cast<hipStream_t>(stream), Q, rows, K, T);
  return oq::launch_status();
}

extern "C" int oq_rotate_act_f32(const void* X, int64_t M, int64_t K, int64_t ldx, int32_t had_block, float* Y,
                                 void* stream) {
  int st = oq::rq_validate(X, M, K, ldx, had_block, Y, reinterpret_cast<const float*>(Y));
  if (st != OQ_OK || M == 0) return st;
  if ((st = oq::device_check()) != OQ_OK) return st;
  return oq::rq_launch(X, M, K, ldx, had_block, 1.0f, nullptr, nullptr, Y, static_cast<hipStream_t>(stream), false,
                       nullptr, true);
}

namespace {
int rq_static(const void* X, int64_t M, int64_t K, int64_t ldx, int32_t had_block, const float* delta, uint8_t* Xq,
              float* x_scale, void* stream, bool tiled) {
  int st = oq::rq_validate(X, M, K, ldx, had_block, Xq, x_scale);
  if (st != OQ_OK) return st;
  if (tiled && K % 128 != 0) return OQ_ERR_SHAPE;
  if (M == 0) return OQ_OK;
  if (!delta) return OQ_ERR_NULL;
  if (!oq::aligned(delta, 16)) return OQ_ERR_ALIGN;
  if ((st = oq::device_check()) != OQ_OK) return st;
  return oq::rq_launch(X, M, K, ldx, had_block, 1.0f, Xq, x_scale, nullptr, static_cast<hipStream_t>(stream), tiled,
                       delta, false);
}
}  // namespace

extern "C" int oq_rotate_quantize_act_static(const void* X, int64_t M, int64_t K, int64_t ldx, int32_t had_block,
                                             const float* delta, uint8_t* Xq, float* x_scale, void* stream) {
  return rq_static(X, M, K, ldx, had_block, delta, Xq, x_scale, stream, false);
}

extern "C" int oq_rotate_quantize_act_static_tiled(const void* X, int64_t M, int64_t K, int64_t ldx,
                                                   int32_t had_block, const float* delta, uint8_t* Xt,
                                                   float* x_scale, void* stream) {
  return rq_static(X, M, K, ldx, had_block, delta, Xt, x_scale, stream, true);
}

extern "C" int oq_rotate_quantize_act_i8(const void* X, int64_t M, int64_t K, int64_t ldx, int32_t had_block,
                                         const float* s_table, int32_t t, int8_t* Xq8, float* x_scale,
                                         void* stream) {
  int st = oq::rq_validate(X, M, K, ldx, had_block, Xq8, x_scale);
  if (st != OQ_OK) return st;
  if (t < 0) return OQ_ERR_ARG;
  if (M == 0) return OQ_OK;
  const float s = s_table ? s_table[t] : 1.0f;
  if (!(s > 0.0f) || !std::isfinite(s)) return OQ_ERR_ARG;
  if ((st = oq::device_check()) != OQ_OK) return st;
  return oq::rq_launch(X, M, K, ldx, had_block, s, reinterpret_cast<uint8_t*>(Xq8), x_scale, nullptr,
                       static_cast<hipStream_t>(stream), false, nullptr, false, true);
}

extern "C" int oq_quantize_weights_step(const void* W_u, int64_t N, int64_t K, int64_t ldw, int32_t had_block,
                                        const float* delta, uint8_t* Wq, float* w_scale, void* stream) {
  int st = oq::rq_validate(W_u, N, K, ldw, had_block, Wq, w_scale);
  if (st != OQ_OK || N == 0) return st;
  if (!delta) return OQ_ERR_NULL;
  if (!oq::aligned(delta, 16)) return OQ_ERR_ALIGN;
  if ((st = oq::device_check()) != OQ_OK) return st;
  return oq::rq_launch(W_u, N, K, ldw, had_block, 1.0f, Wq, w_scale, nullptr, static_cast<hipStream_t>(stream), false,
                       nullptr, false, false, delta);
}
