// W4A4 product with int32 accumulation and the fused dequantization epilogue.
//
// eq:lowbit_linear: X'W' ~= Delta_X' Delta_W' Q_X' Q_W'.  acc[i][n] =
// sum_k q[i][k] wq[n][k] is formed exactly on the int8 matrix cores
// (v_mfma_i32_32x32x32_i8); the per-token and per-output-channel steps (and the
// bias) are applied to the accumulator in the epilogue, as the Implementation
// Details fold every scale into dequantization.
//
// CDNA4 has no int4 integer MFMA, so codes are widened to int8 once per tile,
// on the way into LDS.  A packed byte holds two codes (low nibble = even
// channel).  Masking instead of sign-extending keeps each code in the HIGH
// nibble of an int8 lane:  (w << 4) & 0xF0F0F0F0 gives 16*q_even per byte and
// w & 0xF0F0F0F0 gives 16*q_odd, both correctly signed.  Every product is then
// 256*q*wq; |256 * 49 * K| < 2^31 for K <= 16384, and the exact accumulator is
// recovered with an arithmetic shift by 8.  The two halves of each 8-code group
// are stored even-channels-first; A and B use the same order, so the dot
// products are unchanged.
//
// Tiling: 128 x 128 output tile per 256-thread workgroup, 2 x 2 waves of
// 64 x 64 (2 x 2 MFMA blocks of 32 x 32), K step 64 codes, two LDS buffers
// (global loads of step k+1 are in flight while step k runs on the matrix
// cores).  LDS rows are padded to 80 bytes so the 16-byte fragment reads of 16
// consecutive rows hit disjoint banks.
#include "common.h"

namespace oq {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int BM = 128, BN = 128, BK = 64;  // BK in codes (32 packed bytes per row)
constexpr int LDS_STRIDE = 80;              // bytes per LDS row: 64 int8 + 16 pad

__device__ __forceinline__ void unpack_store(uint8_t* dst, uint4 w) {
  const uint32_t m = 0xF0F0F0F0u;
  // Per packed dword: even-channel codes, then odd-channel codes.
  uint4 p0, p1;
  p0.x = (w.x << 4) & m; p0.y = w.x & m;
  p0.z = (w.y << 4) & m; p0.w = w.y & m;
  p1.x = (w.z << 4) & m; p1.y = w.z & m;
  p1.z = (w.w << 4) & m; p1.w = w.w & m;
  reinterpret_cast<uint4*>(dst)[0] = p0;
  reinterpret_cast<uint4*>(dst)[1] = p1;
}

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t b = __float_as_uint(f);
  b += 0x7FFFu + ((b >> 16) & 1u);
  return static_cast<uint16_t>(b >> 16);
}

template <int EPI>
__global__ __launch_bounds__(256) void gemm_w4a4_kernel(GemmArgs a) {
  __shared__ __attribute__((aligned(16))) uint8_t sA[2][BM * LDS_STRIDE];
  __shared__ __attribute__((aligned(16))) uint8_t sB[2][BN * LDS_STRIDE];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int64_t m0 = static_cast<int64_t>(blockIdx.y) * BM;
  const int64_t n0 = static_cast<int64_t>(blockIdx.x) * BN;
  const int64_t Kb = a.K / 2;
  const int nk = static_cast<int>(a.K / BK);

  // Global -> LDS assignment: thread loads 16 packed bytes (32 codes) of one row.
  const int lr = tid >> 1, lh = tid & 1;
  const bool a_ok = m0 + lr < a.M;
  const bool b_ok = n0 + lr < a.N;
  const uint8_t* gA = a.A + (a_ok ? (m0 + lr) : 0) * Kb + lh * 16;
  const uint8_t* gB = a.B + (b_ok ? (n0 + lr) : 0) * Kb + lh * 16;
  const int st_off = lr * LDS_STRIDE + lh * 32;

  uint4 ra = make_uint4(0, 0, 0, 0), rb = make_uint4(0, 0, 0, 0);
  if (a_ok) ra = *reinterpret_cast<const uint4*>(gA);
  if (b_ok) rb = *reinterpret_cast<const uint4*>(gB);
  unpack_store(&sA[0][st_off], ra);
  unpack_store(&sB[0][st_off], rb);
  __syncthreads();

  v16i acc[2][2];
#pragma unroll
  for (int r = 0; r < 2; ++r)
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[r][s][e] = 0;

  const int frag_row = lane & 31;
  const int frag_k = 16 * (lane >> 5);

  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    const bool more = kt + 1 < nk;
    if (more) {
      if (a_ok) ra = *reinterpret_cast<const uint4*>(gA + (kt + 1) * (BK / 2));
      if (b_ok) rb = *reinterpret_cast<const uint4*>(gB + (kt + 1) * (BK / 2));
    }
#pragma unroll
    for (int kk = 0; kk < BK; kk += 32) {
      v4i fa[2], fb[2];
#pragma unroll
      for (int r = 0; r < 2; ++r)
        fa[r] = *reinterpret_cast<const v4i*>(&sA[buf][(wm * 64 + r * 32 + frag_row) * LDS_STRIDE + kk + frag_k]);
#pragma unroll
      for (int s = 0; s < 2; ++s)
        fb[s] = *reinterpret_cast<const v4i*>(&sB[buf][(wn * 64 + s * 32 + frag_row) * LDS_STRIDE + kk + frag_k]);
#pragma unroll
      for (int r = 0; r < 2; ++r)
#pragma unroll
        for (int s = 0; s < 2; ++s)
          acc[r][s] = __builtin_amdgcn_mfma_i32_32x32x32_i8(fa[r], fb[s], acc[r][s], 0, 0, 0);
    }
    if (more) {
      unpack_store(&sA[buf ^ 1][st_off], ra);
      unpack_store(&sB[buf ^ 1][st_off], rb);
    }
    __syncthreads();
  }

  // Epilogue.  32x32 accumulator layout: element e of lane l is row
  // 8*(e/4) + 4*(l/32) + e%4, column l%32 of the block.
  const int col_in = lane & 31;
  const int row_grp = 4 * (lane >> 5);
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const int64_t gc = n0 + wn * 64 + s * 32 + col_in;
    if (gc >= a.N) continue;
    float wsc = 0.0f, bias = 0.0f, gate = 1.0f;
    if (EPI != EPI_I32) {
      wsc = a.ws[gc];
      if (a.bias) bias = static_cast<float>(__builtin_bit_cast(_Float16, a.bias[gc]));
      if (EPI == EPI_RESID_F32 && a.gate) gate = static_cast<float>(__builtin_bit_cast(_Float16, a.gate[gc]));
    }
#pragma unroll
    for (int r = 0; r < 2; ++r)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int64_t gr = m0 + wm * 64 + r * 32 + 8 * (e >> 2) + row_grp + (e & 3);
        if (gr >= a.M) continue;
        const int v = acc[r][s][e] >> 8;
        const int64_t off = gr * a.ldc + gc;
        if (EPI == EPI_I32) {
          static_cast<int32_t*>(a.C)[off] = v;
        } else {
          const float y = static_cast<float>(v) * a.xs[gr] * wsc + bias;
          if (EPI == EPI_F16) {
            static_cast<_Float16*>(a.C)[off] = static_cast<_Float16>(y);
          } else if (EPI == EPI_BF16) {
            static_cast<uint16_t*>(a.C)[off] = f32_to_bf16_rne(y);
          } else {
            float* rp = static_cast<float*>(a.C) + off;
            *rp = fmaf(gate, y, *rp);
          }
        }
      }
  }
}

}  // namespace

int gemm_validate(const uint8_t* Xq, int64_t M, const uint8_t* Wq, int64_t N, int64_t K, const void* C,
                  int64_t ldc, int64_t ldc_align) {
  if (M < 0 || N < 1 || K < BK || K % BK != 0 || K > 16384 || ldc < N) return OQ_ERR_SHAPE;
  if (ldc % ldc_align != 0) return OQ_ERR_ALIGN;
  if (M == 0) return OQ_OK;  // nothing is read or written; pointers may be NULL
  if (!Xq || !Wq || !C) return OQ_ERR_NULL;
  if (!aligned(Xq, 16) || !aligned(Wq, 16) || !aligned(C, 16) || ldc % ldc_align != 0) return OQ_ERR_ALIGN;
  return OQ_OK;
}

int gemm_launch(const GemmArgs& a, Epilogue epi, hipStream_t stream) {
  if (a.M == 0) return OQ_OK;
  const dim3 grid(static_cast<unsigned>((a.N + BN - 1) / BN), static_cast<unsigned>((a.M + BM - 1) / BM));
  switch (epi) {
    case EPI_I32: hipLaunchKernelGGL(gemm_w4a4_kernel<EPI_I32>, grid, dim3(256), 0, stream, a); break;
    case EPI_F16: hipLaunchKernelGGL(gemm_w4a4_kernel<EPI_F16>, grid, dim3(256), 0, stream, a); break;
    case EPI_BF16: hipLaunchKernelGGL(gemm_w4a4_kernel<EPI_BF16>, grid, dim3(256), 0, stream, a); break;
    case EPI_RESID_F32: hipLaunchKernelGGL(gemm_w4a4_kernel<EPI_RESID_F32>, grid, dim3(256), 0, stream, a); break;
    default: return OQ_ERR_ARG;
  }
  return launch_status();
}

}  // namespace oq

extern "C" int oq_w4a4_linear(const uint8_t* Xq, const float* x_scale, int64_t M, const uint8_t* Wq,
                              const float* w_scale, const void* bias, int64_t N, int64_t K, void* Y,
                              int64_t ldy, int32_t out_dtype, void* stream) {
  int st = oq::gemm_validate(Xq, M, Wq, N, K, Y, ldy, 8);
  if (st != OQ_OK || M == 0) return st;
  if (!x_scale || !w_scale) return OQ_ERR_NULL;
  if (out_dtype != OQ_OUT_F16 && out_dtype != OQ_OUT_BF16) return OQ_ERR_ARG;
  if (!oq::aligned(x_scale, 4) || !oq::aligned(w_scale, 4) || (bias && !oq::aligned(bias, 2))) return OQ_ERR_ALIGN;
  if ((st = oq::device_check()) != OQ_OK) return st;
  oq::GemmArgs a{Xq, Wq, x_scale, w_scale, static_cast<const uint16_t*>(bias), Y, nullptr, M, N, K, ldy};
  return oq::gemm_launch(a, out_dtype == OQ_OUT_F16 ? oq::EPI_F16 : oq::EPI_BF16, static_cast<hipStream_t>(stream));
}

extern "C" int oq_w4a4_gemm_i32(const uint8_t* Xq, int64_t M, const uint8_t* Wq, int64_t N, int64_t K,
                                int32_t* acc, int64_t ldc, void* stream) {
  int st = oq::gemm_validate(Xq, M, Wq, N, K, acc, ldc, 4);
  if (st != OQ_OK || M == 0) return st;
  if ((st = oq::device_check()) != OQ_OK) return st;
  oq::GemmArgs a{Xq, Wq, nullptr, nullptr, nullptr, acc, nullptr, M, N, K, ldc};
  return oq::gemm_launch(a, oq::EPI_I32, static_cast<hipStream_t>(stream));
}
