// Matrix-core rotate-quantize of one row held as fp16 fragments (Section 4.1
// eq:blockdiag / eq:transform, Section 4.2 eq:scale, eq:quant,
// eq:perstep_scale), shared by the stand-alone kernel and by the DiT kernels
// that produce an fp16 row and quantize it in the same pass.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rq_device.h"

namespace oq {
namespace rqm {

// ---------------------------------------------------------------------------
// Layout for Hadamard blocks b >= 32 and K = 512 * NG * W.
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

// Constants of the (NG, W) layout.
template <int NG, int W>
struct Shape {
  static constexpr int K = NG * W * 512;
  static constexpr int RPB = W == 3 ? 1 : 4 / W;  // rows per workgroup (256 threads; 192 when W = 3)
  static constexpr int LOGNG = NG >= 16 ? 4 : NG >= 8 ? 3 : NG >= 4 ? 2 : NG >= 2 ? 1 : 0;
  static constexpr int LOGW = W >= 4 ? 2 : W >= 2 ? 1 : 0;
  static constexpr int GW = NG / W;  // groups per wave after the transpose
  // W = 3: three waves per row, each holding whole Hadamard blocks (b <= 512 NG, checked by the launcher),
  // so no butterfly crosses a wave and only the row maximum is shared.
  static_assert(W == 1 || W == 3 || (NG % W == 0 && (NG & (NG - 1)) == 0),
                "NG must be a power of two >= W when W is 2 or 4");
  static_assert(NG <= 16, "at most 16 register groups");
};

// First of the 8 consecutive channels of group g held by `lane` of wave wr:
// ((wr * NG + g) * 16 + lane % 16) * 32 + 8 * (lane / 16).
template <int NG>
__device__ __forceinline__ int chan0(int wr, int g, int lane) {
  return ((wr * NG + g) * 16 + (lane & 15)) * 32 + 8 * (lane >> 4);
}

// Everything after the row is in fragments: H_32 on the matrix cores, the
// remaining butterflies, the row maximum, the scale and the codes (or, with
// ratio != nullptr, the fp32 ratios z / Delta).  cur[g] holds channels
// chan0(wr, g, lane) .. + 7.  Every wave of the workgroup calls it: it
// synchronizes when W > 1 (xch: [4][NG][2][32] float4 of LDS), and `red` is
// a 4-float shared array.  sdelta / rotate_only: the static per-channel
// quantizer and the fp32 rotation output, as in rqd::rq_core; i8: 8-bit codes
// (q_max = 127), one byte per code in [M][K]; cmul: per-channel multiplier
// before the row maximum, as in rqd::rq_core; sg (with sdelta): the static
// multipliers rqd::static_mult already formed per channel (in LDS).
template <int NG, int W, bool FULL>
__device__ __forceinline__ void rq_row(const rv8h (&cur)[NG], const rv8h& a1, const rv8h& a2, int64_t row, bool valid,
                                       int lane, int wv, int logb, float s_t, float s_over_sqrtb,
                                       uint8_t* __restrict__ Xq, float* __restrict__ xs, float* __restrict__ ratio,
                                       float4* xch, float* red, bool tiled,
                                       const float* __restrict__ sdelta = nullptr, bool rotate_only = false,
                                       bool i8 = false, const float* __restrict__ cmul = nullptr,
                                       const float* sg = nullptr) {
  using S = Shape<NG, W>;
  constexpr int K = S::K, LOGNG = S::LOGNG, LOGW = S::LOGW, GW = S::GW;
  const int rsub = wv / W, wr = wv % W;
  const int cl = lane & 15, q = lane >> 4;
  // Butterfly over channel bit `bit` is needed when bit < log2(b); FULL means
  // b = K (every stage, no branches).
  auto need = [&](int bit) { return FULL || bit < logb; };
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
  const bool xpose = W > 1 && W != 3 && need(wbit0);
  if constexpr (W == 2 || W == 4) {
    if (xpose) {
      // Two rounds, one per half of the lanes: the transpose only moves a
      // value between waves at the same lane, so each round needs half the
      // LDS (more workgroups per CU) and a lane overwrites only its own
      // registers after its own values are written.
      const int lh = lane & 31;
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        if ((lane >> 5) == half) {
          float4* mine = xch + static_cast<int64_t>(wv) * NG * 64 + lh;
#pragma unroll
          for (int g = 0; g < NG; ++g) {
            mine[g * 64] = make_float4(v[g][0], v[g][1], v[g][2], v[g][3]);
            mine[g * 64 + 32] = make_float4(v[g][4], v[g][5], v[g][6], v[g][7]);
          }
        }
        __syncthreads();
        if ((lane >> 5) == half) {
#pragma unroll
          for (int gi = 0; gi < GW; ++gi)
#pragma unroll
            for (int u = 0; u < W; ++u) {
              const float4* src = xch + static_cast<int64_t>((rsub * W + u) * NG + wr * GW + gi) * 64 + lh;
              const float4 p0 = src[0], p1 = src[32];
              float* d = v[gi * W + u];
              d[0] = p0.x; d[1] = p0.y; d[2] = p0.z; d[3] = p0.w;
              d[4] = p1.x; d[5] = p1.y; d[6] = p1.z; d[7] = p1.w;
            }
        }
        __syncthreads();
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

  auto group_of = [&](int s) { return xpose ? (s % W) * NG + wr * GW + s / W : wr * NG + s; };
  if (cmul != nullptr) {  // per-channel multiplier before the row maximum (the per-step weight fold)
#pragma unroll
    for (int s = 0; s < NG; ++s) {
      const float4* mp = reinterpret_cast<const float4*>(cmul + (group_of(s) * 16 + cl) * 32 + 8 * q);
      const float4 a = mp[0], b = mp[1];
      v[s][0] *= a.x; v[s][1] *= a.y; v[s][2] *= a.z; v[s][3] *= a.w;
      v[s][4] *= b.x; v[s][5] *= b.y; v[s][6] *= b.z; v[s][7] *= b.w;
    }
  }
  // Rotation only, or the static quantizer: no row maximum (uniform branch;
  // no barrier follows).
  if (rotate_only) {
    if (!valid) return;
#pragma unroll
    for (int s = 0; s < NG; ++s) {
      float* yr = ratio + row * K + (group_of(s) * 16 + cl) * 32 + 8 * q;
      const float g = s_over_sqrtb;
      reinterpret_cast<float4*>(yr)[0] = make_float4(v[s][0] * g, v[s][1] * g, v[s][2] * g, v[s][3] * g);
      reinterpret_cast<float4*>(yr)[1] = make_float4(v[s][4] * g, v[s][5] * g, v[s][6] * g, v[s][7] * g);
    }
    return;
  }
  if (sdelta != nullptr) {
    if (!valid) return;
    if (wr == 0 && lane == 0) xs[row] = 1.0f;
    uint8_t* qr = Xq + row * (K / 2);
#pragma unroll
    for (int s = 0; s < NG; ++s) {
      const int c0 = (group_of(s) * 16 + cl) * 32 + 8 * q;
      uint32_t b[8];
      if (sg != nullptr) {
        const float4 g0 = reinterpret_cast<const float4*>(sg + c0)[0];
        const float4 g1 = reinterpret_cast<const float4*>(sg + c0)[1];
        const float g[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
#pragma unroll
        for (int e = 0; e < 8; ++e) b[e] = rqd::static_code_g(v[s][e], g[e]);
      } else {
        const float4 d0 = reinterpret_cast<const float4*>(sdelta + c0)[0];
        const float4 d1 = reinterpret_cast<const float4*>(sdelta + c0)[1];
        const float d[8] = {d0.x, d0.y, d0.z, d0.w, d1.x, d1.y, d1.z, d1.w};
#pragma unroll
        for (int e = 0; e < 8; ++e) b[e] = rqd::static_code(v[s][e], d[e], s_over_sqrtb);
      }
      const int p = c0 / 2;
      uint8_t* dst = tiled ? Xq + tiled_offset(row, p, K / 128) : qr + p;
      *reinterpret_cast<uint32_t*>(dst) = rqd::pack8(b);
    }
    return;
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
  amax = fmaxf(amax, rqd::lane_xor_far<16>(amax));
  amax = fmaxf(amax, rqd::lane_xor_far<32>(amax));
  if constexpr (W > 1) {
    if (lane == 0) red[wv] = amax;
    __syncthreads();
    amax = red[rsub * W];
#pragma unroll
    for (int u = 1; u < W; ++u) amax = fmaxf(amax, red[rsub * W + u]);
  }

  const float a_z = amax * s_over_sqrtb;
  const float delta = a_z / (i8 ? 127.0f : 7.0f);
  const float gm = delta > 0.0f ? s_over_sqrtb / delta : 0.0f;
  if (!valid) return;
  if (wr == 0 && lane == 0) xs[row] = delta / s_t;
  if (ratio != nullptr) {
#pragma unroll
    for (int s = 0; s < NG; ++s) {
      float* rr = ratio + row * K + (group_of(s) * 16 + cl) * 32 + 8 * q;
      reinterpret_cast<float4*>(rr)[0] = make_float4(v[s][0] * gm, v[s][1] * gm, v[s][2] * gm, v[s][3] * gm);
      reinterpret_cast<float4*>(rr)[1] = make_float4(v[s][4] * gm, v[s][5] * gm, v[s][6] * gm, v[s][7] * gm);
    }
    return;
  }
  if (i8) {
#pragma unroll
    for (int s = 0; s < NG; ++s) {
      uint32_t b[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) b[e] = __float_as_uint(fmaf(v[s][e], gm, rqd::kRoundMagic));
      *reinterpret_cast<uint2*>(Xq + row * K + (group_of(s) * 16 + cl) * 32 + 8 * q) = rqd::pack8_i8(b);
    }
    return;
  }
  uint8_t* qr = Xq + row * (K / 2);
  if constexpr (NG % 4 == 0) {
    // Four slots at a time: lane (cl, q) packs one dword (8 codes) of each,
    // then a 4 x 4 transpose between the slot index and lane bits 4-5 (two
    // permlane32 swaps, then two permlane16 swaps) leaves lane q with all four
    // dwords of slot 4a + q -- the 32 codes of chunk cl, one 16-byte store.
#pragma unroll
    for (int a = 0; a < NG / 4; ++a) {
      uint32_t d[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        uint32_t b[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) b[e] = __float_as_uint(fmaf(v[4 * a + i][e], gm, rqd::kRoundMagic));
        d[i] = rqd::pack8(b);
      }
      rqd::dword_swap<32>(d[0], d[2]);
      rqd::dword_swap<32>(d[1], d[3]);
      rqd::dword_swap<16>(d[0], d[1]);
      rqd::dword_swap<16>(d[2], d[3]);
      const int p = (group_of(4 * a + q) * 16 + cl) * 16;
      uint8_t* dst = tiled ? Xq + tiled_offset(row, p, K / 128) : qr + p;
      *reinterpret_cast<uint4*>(dst) = make_uint4(d[0], d[1], d[2], d[3]);
    }
  } else {
#pragma unroll
    for (int s = 0; s < NG; ++s) {
      uint32_t b[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) b[e] = __float_as_uint(fmaf(v[s][e], gm, rqd::kRoundMagic));
      const int p = (group_of(s) * 16 + cl) * 16 + 4 * q;
      uint8_t* dst = tiled ? Xq + tiled_offset(row, p, K / 128) : qr + p;
      *reinterpret_cast<uint32_t*>(dst) = rqd::pack8(b);
    }
  }
}

}  // namespace rqm
}  // namespace oq
