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
#include <cstdlib>

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
// group index g in registers, and for rows wider than 4096 channels (W waves
// per row) the top bits are exchanged through LDS.  Waves are persistent: each
// loops over rows and loads the next row's fp16 fragments while it transforms
// the current one.
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

template <int NG, int W>
__global__ __launch_bounds__(256) void rq_mfma_kernel(const uint16_t* __restrict__ X, int64_t M, int64_t ldx, int logb,
                                                      float s_t, float s_over_sqrtb, uint8_t* __restrict__ Xq,
                                                      float* __restrict__ xs, float* __restrict__ ratio) {
  extern __shared__ float lds[];  // W > 1: [4 waves][NG][64 lanes][8] fp32
  __shared__ float red[4];
  constexpr int K = NG * W * 512;
  constexpr int RPB = 4 / W;  // rows per workgroup pass
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int rsub = wv / W, wr = wv % W;
  const int cl = lane & 15, q = lane >> 4;
  rv8h a1, a2;
  hadamard_frags(lane, a1, a2);

  // Element (g, e) of this lane is channel ((wr * NG + g) * 16 + cl) * 32 + 8q + e.
  auto load = [&](int64_t row, rv8h (&f)[NG]) {
    const uint16_t* xr = X + row * ldx + (wr * NG * 16 + cl) * 32 + 8 * q;
#pragma unroll
    for (int g = 0; g < NG; ++g) f[g] = *reinterpret_cast<const rv8h*>(xr + g * 512);
  };
  const int64_t step = static_cast<int64_t>(gridDim.x) * RPB;
  // The transform of one row from its fp16 fragments (everything after the loads).
  auto process = [&](const int64_t row, const bool valid, rv8h (&cur)[NG]) {
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
    if (logb > 5) rqd::lane_stage<1>(v, lane);
    if (logb > 6) rqd::lane_stage<2>(v, lane);
    if (logb > 7) rqd::lane_stage<4>(v, lane);
    if (logb > 8) rqd::lane_stage<8>(v, lane);
    // Channel bits 9..: group index g in registers.
#pragma unroll
    for (int t = 0; t < 5; ++t) {
      constexpr int dummy = 0;
      (void)dummy;
      const int h = 1 << t;
      if (h < NG && 9 + t < logb) {
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
    // Wave bits (rows wider than one wave): exchange through LDS.
    if constexpr (W > 1) {
      constexpr int LOGNG = NG >= 8 ? 3 : NG >= 4 ? 2 : NG >= 2 ? 1 : 0;
      const int wbit0 = 9 + LOGNG;
      const int ws = min(max(logb - wbit0, 0), W == 4 ? 2 : 1);
      __syncthreads();  // the previous row's LDS reads are done
      if (ws > 0) {
        float* mine = lds + (static_cast<int64_t>(wv) * NG * 64 + lane) * 8;
#pragma unroll
        for (int g = 0; g < NG; ++g) {
          float4* d = reinterpret_cast<float4*>(mine + g * 64 * 8);
          d[0] = make_float4(v[g][0], v[g][1], v[g][2], v[g][3]);
          d[1] = make_float4(v[g][4], v[g][5], v[g][6], v[g][7]);
        }
      }
      __syncthreads();
      if (ws > 0) {
        const int nw = 1 << ws;
        const int wlow = wr & (nw - 1), wbase = wr & ~(nw - 1);
#pragma unroll
        for (int g = 0; g < NG; ++g) {
          float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
          for (int u = 0; u < nw; ++u) {
            const float sg = (__popc(wlow & u) & 1) ? -1.0f : 1.0f;
            const float* src = lds + ((static_cast<int64_t>(rsub * W + (wbase | u)) * NG + g) * 64 + lane) * 8;
            const float4 p0 = reinterpret_cast<const float4*>(src)[0];
            const float4 p1 = reinterpret_cast<const float4*>(src)[1];
            acc[0] = fmaf(sg, p0.x, acc[0]); acc[1] = fmaf(sg, p0.y, acc[1]);
            acc[2] = fmaf(sg, p0.z, acc[2]); acc[3] = fmaf(sg, p0.w, acc[3]);
            acc[4] = fmaf(sg, p1.x, acc[4]); acc[5] = fmaf(sg, p1.y, acc[5]);
            acc[6] = fmaf(sg, p1.z, acc[6]); acc[7] = fmaf(sg, p1.w, acc[7]);
          }
#pragma unroll
          for (int e = 0; e < 8; ++e) v[g][e] = acc[e];
        }
      }
    }

    // Row maximum: lanes, then the W waves of the row.
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
    if (valid && wr == 0 && lane == 0) xs[row] = delta / s_t;
    if (!valid) return;
    if (ratio != nullptr) {
#pragma unroll
      for (int g = 0; g < NG; ++g) {
        float* rr = ratio + row * K + ((wr * NG + g) * 16 + cl) * 32 + 8 * q;
        reinterpret_cast<float4*>(rr)[0] = make_float4(v[g][0] * gm, v[g][1] * gm, v[g][2] * gm, v[g][3] * gm);
        reinterpret_cast<float4*>(rr)[1] = make_float4(v[g][4] * gm, v[g][5] * gm, v[g][6] * gm, v[g][7] * gm);
      }
      return;
    }
    uint8_t* qr = Xq + row * (K / 2);
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      uint32_t b[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) b[e] = __float_as_uint(fmaf(v[g][e], gm, rqd::kRoundMagic));
      *reinterpret_cast<uint32_t*>(qr + ((wr * NG + g) * 16 + cl) * 16 + 4 * q) = rqd::pack8(b);
    }
  };
  {
    // One row in flight ahead of the one being transformed.
    rv8h nxt[NG];
    const int64_t r0 = static_cast<int64_t>(blockIdx.x) * RPB + rsub;
    if (r0 < M) load(r0, nxt);
    for (int64_t base = static_cast<int64_t>(blockIdx.x) * RPB; base < M; base += step) {
      const int64_t row = base + rsub;
      const bool valid = row < M;
      rv8h cur[NG];
#pragma unroll
      for (int g = 0; g < NG; ++g) cur[g] = valid ? nxt[g] : rv8h{};
      if (row + step < M) load(row + step, nxt);
      process(row, valid, cur);
    }
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
  const size_t lds = w > 1 ? static_cast<size_t>(4) * ng * 64 * 8 * sizeof(float) : 0;
  // Persistent workgroups: enough to fill every CU several times over.
  const int64_t want = (M + rpb - 1) / rpb;
  const int64_t cap = w > 1 ? 512 : 1024;
  const unsigned grid = static_cast<unsigned>(want < cap ? want : cap);
  const uint16_t* x = static_cast<const uint16_t*>(X);
#define OQ_RQM(NG, W)                                                                                     \
  if (ng == NG && w == W) {                                                                               \
    hipLaunchKernelGGL((rq_mfma_kernel<NG, W>), dim3(grid), dim3(256), lds, stream, x, M, ldx, logb, s_t, \
                       s_over_sqrtb, Xq, x_scale, ratio);                                                 \
    return launch_status();                                                                               \
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
  if (had_block >= 32 && rq_mfma_shape(K, &ng, &w) && !std::getenv("OQ_RQ_VALU"))
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
