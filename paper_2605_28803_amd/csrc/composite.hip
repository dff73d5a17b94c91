// Online composite rotation of Section 4.1 with per-token int4 quantization.
//
// eq:transform: X' = X P R_hat with P a channel permutation and R_hat =
// BlockDiag(R_1 .. R_K), R_b = U_b H_c (eq:blockdiag), block size c = 64 (the
// paper's setting).  Then the step scale and the per-token quantizer of
// Section 4.2 (eq:scale, eq:quant; eq:perstep_scale in its per-(layer, step)
// scalar form): z = s_t y, Delta = max|z| / 7, q = round_half_even(z / Delta),
// x_scale = Delta / s_t.
//
// One workgroup of four waves owns RW rows.  The rows are staged in LDS as
// fp16.  Pass 1: wave w takes the 64-channel blocks b = w, w + 4, ...; for
// each, the A fragment (rows x 32 permuted channels) is gathered from LDS
// through perm (the v_mfma_f32_16x16x32_f16 operand layout: lane l holds row
// l % 16 and the 8 consecutive k values 8 (l / 16) .. + 7), the B fragment is
// one 16-byte load of the column-major block matrix (lane l holds output
// column l % 16 and the same 8 k values), and the 16 x 16 fp32 products give
// y for four 16-channel column groups; only the row maxima are kept.  The
// maxima are combined across lanes and waves, then pass 2 recomputes y and
// writes int8 codes to LDS, which are packed two per byte and stored
// coalesced.  fp16 x fp16 products are exact in fp32; the 64-term sums are
// the only rounding of the transform.  Rows past RW in a fragment are zero.
#include <cmath>

#include "common.h"
#include "rq_device.h"

namespace oq {
namespace {

typedef _Float16 c8h __attribute__((ext_vector_type(8)));
typedef float c4f __attribute__((ext_vector_type(4)));

constexpr int kCB = 64;  // block size c

// Two nibbles per byte from 16 two's-complement int8 codes (even channel low).
__device__ __forceinline__ uint32_t pack4codes(uint32_t d) {
  const uint32_t e = d & 0x000F000Fu;          // codes 0, 2 -> bits 0-3, 16-19
  const uint32_t o = (d >> 4) & 0x00F000F0u;   // codes 1, 3 -> bits 4-7, 20-23
  const uint32_t t = e | o;
  return (t & 0xFFu) | ((t >> 8) & 0xFF00u);
}

template <int RW, int KMAX>
__global__ __launch_bounds__(256) void rq_composite_kernel(const uint16_t* __restrict__ X, int64_t M, int K,
                                                           int64_t ldx, const int32_t* __restrict__ perm,
                                                           const uint16_t* __restrict__ Rt, float s_t,
                                                           uint8_t* __restrict__ Xq, float* __restrict__ xs) {
  __shared__ __attribute__((aligned(16))) uint16_t sx[RW * KMAX];  // fp16 rows
  __shared__ __attribute__((aligned(16))) int8_t sc[RW * KMAX];    // int8 codes
  __shared__ float red[4][16];
  __shared__ float gscale[16];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t row0 = static_cast<int64_t>(blockIdx.x) * RW;
  const int nb = K / kCB;
  const int vpr = K / 8;  // 16-byte pieces per row

  // Stage the rows (rows past M are zeros): 8 loads in flight per thread.
  for (int p0 = tid; p0 < RW * vpr; p0 += 256 * 8) {
    uint4 v[8];
    bool ok[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int p = p0 + u * 256;
      const int r = p / vpr, c8 = p - r * vpr;
      ok[u] = p < RW * vpr && row0 + r < M;
      const int64_t gr = ok[u] ? row0 + r : 0;
      v[u] = *reinterpret_cast<const uint4*>(X + gr * ldx + (ok[u] ? c8 * 8 : 0));
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int p = p0 + u * 256;
      const int r = p / vpr, c8 = p - r * vpr;
      if (p < RW * vpr) *reinterpret_cast<uint4*>(&sx[r * KMAX + c8 * 8]) = ok[u] ? v[u] : make_uint4(0, 0, 0, 0);
    }
  }
  __syncthreads();

  const int r16 = lane & 15, q = lane >> 4;
  const bool rok = r16 < RW;
  const uint16_t* xrow = &sx[(rok ? r16 : 0) * KMAX];

  // y of block b, column group cb for this lane: rows 4q + e, column r16.
  auto gather = [&](int b, int kk) -> c8h {
    const int k0 = b * kCB + kk * 32 + 8 * q;
    const int4 pa = *reinterpret_cast<const int4*>(perm + k0);
    const int4 pb = *reinterpret_cast<const int4*>(perm + k0 + 4);
    const int idx[8] = {pa.x, pa.y, pa.z, pa.w, pb.x, pb.y, pb.z, pb.w};
    c8h a;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int src = min(max(idx[j], 0), K - 1);  // a non-permutation stays inside the staged row
      a[j] = __builtin_bit_cast(_Float16, rok ? xrow[src] : uint16_t(0));
    }
    return a;
  };
  auto bfrag = [&](int b, int cb, int kk) -> c8h {
    return *reinterpret_cast<const c8h*>(Rt + (static_cast<int64_t>(b) * kCB + cb * 16 + r16) * kCB + kk * 32 +
                                         8 * q);
  };

  // Pass 1: row maxima of |y|.
  float amax[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int b = wave; b < nb; b += 4) {
    const c8h a0 = gather(b, 0), a1 = gather(b, 1);
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) {
      c4f acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a0, bfrag(b, cb, 0), c4f{0, 0, 0, 0}, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a1, bfrag(b, cb, 1), acc, 0, 0, 0);
#pragma unroll
      for (int e = 0; e < 4; ++e) amax[e] = fmaxf(amax[e], fabsf(acc[e]));
    }
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    float m = amax[e];
    m = fmaxf(m, rqd::lane_xor<1>(m));
    m = fmaxf(m, rqd::lane_xor<2>(m));
    m = fmaxf(m, rqd::lane_xor<4>(m));
    m = fmaxf(m, rqd::lane_xor<8>(m));
    if (r16 == 0) red[wave][4 * q + e] = m;
  }
  __syncthreads();
  if (tid < 16) {
    const float m = fmaxf(fmaxf(red[0][tid], red[1][tid]), fmaxf(red[2][tid], red[3][tid]));
    // a_z = max|s_t y|, Delta = a_z / 7, code = round(y s_t / Delta).
    const float a_z = m * s_t;
    const float delta = a_z / 7.0f;
    gscale[tid] = delta > 0.0f ? s_t / delta : 0.0f;
    if (tid < RW && row0 + tid < M) xs[row0 + tid] = delta / s_t;
  }
  __syncthreads();

  // Pass 2: codes into LDS.
  float g[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) g[e] = gscale[4 * q + e];
  for (int b = wave; b < nb; b += 4) {
    const c8h a0 = gather(b, 0), a1 = gather(b, 1);
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) {
      c4f acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a0, bfrag(b, cb, 0), c4f{0, 0, 0, 0}, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a1, bfrag(b, cb, 1), acc, 0, 0, 0);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int row = 4 * q + e;
        if (row < RW) {
          const uint32_t bits = __float_as_uint(fmaf(acc[e], g[e], rqd::kRoundMagic));
          sc[row * KMAX + b * kCB + cb * 16 + r16] = static_cast<int8_t>(bits & 0xFFu);
        }
      }
    }
  }
  __syncthreads();

  // Pack 16 codes per thread into 8 bytes.
  const int ppr = K / 16;
  for (int p = tid; p < RW * ppr; p += 256) {
    const int r = p / ppr, c16 = p - r * ppr;
    if (row0 + r >= M) continue;
    const uint4 w = *reinterpret_cast<const uint4*>(&sc[r * KMAX + c16 * 16]);
    uint2 out;
    out.x = pack4codes(w.x) | (pack4codes(w.y) << 16);
    out.y = pack4codes(w.z) | (pack4codes(w.w) << 16);
    *reinterpret_cast<uint2*>(Xq + (row0 + r) * static_cast<int64_t>(K / 2) + c16 * 8) = out;
  }
}

template <int RW, int KMAX>
int launch_composite(const void* X, int64_t M, int64_t K, int64_t ldx, const int32_t* perm, const void* Rt,
                     float s, uint8_t* Xq, float* x_scale, hipStream_t stream) {
  const unsigned grid = static_cast<unsigned>((M + RW - 1) / RW);
  hipLaunchKernelGGL((rq_composite_kernel<RW, KMAX>), dim3(grid), dim3(256), 0, stream,
                     static_cast<const uint16_t*>(X), M, static_cast<int>(K), ldx, perm,
                     static_cast<const uint16_t*>(Rt), s, Xq, x_scale);
  return launch_status();
}

}  // namespace
}  // namespace oq

extern "C" int oq_rotate_quantize_act_composite(const void* X, int64_t M, int64_t K, int64_t ldx,
                                                const int32_t* perm, const void* Rt, const float* s_table,
                                                int32_t t, uint8_t* Xq, float* x_scale, void* stream) {
  if (M < 0 || K < 64 || K % 64 != 0 || K > 16384 || ldx < K) return OQ_ERR_SHAPE;
  if (ldx % 8 != 0) return OQ_ERR_ALIGN;
  if (t < 0) return OQ_ERR_ARG;
  if (M == 0) return OQ_OK;
  if (!X || !perm || !Rt || !Xq || !x_scale) return OQ_ERR_NULL;
  if (!oq::aligned(X, 16) || !oq::aligned(perm, 16) || !oq::aligned(Rt, 16) || !oq::aligned(Xq, 8) ||
      !oq::aligned(x_scale, 4))
    return OQ_ERR_ALIGN;
  const float s = s_table ? s_table[t] : 1.0f;
  if (!(s > 0.0f) || !std::isfinite(s)) return OQ_ERR_ARG;
  int st = oq::device_check();
  if (st != OQ_OK) return st;
  hipStream_t h = static_cast<hipStream_t>(stream);
  if (K <= 1024) return oq::launch_composite<16, 1024>(X, M, K, ldx, perm, Rt, s, Xq, x_scale, h);
  if (K <= 2048) return oq::launch_composite<16, 2048>(X, M, K, ldx, perm, Rt, s, Xq, x_scale, h);
  if (K <= 4096) return oq::launch_composite<8, 4096>(X, M, K, ldx, perm, Rt, s, Xq, x_scale, h);
  if (K <= 8192) return oq::launch_composite<4, 8192>(X, M, K, ldx, perm, Rt, s, Xq, x_scale, h);
  return oq::launch_composite<2, 16384>(X, M, K, ldx, perm, Rt, s, Xq, x_scale, h);
}
