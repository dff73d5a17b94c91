// Internal helpers shared by the library's translation units (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "oq.h"

namespace oq {

// OQ_OK if the current device is gfx950 (result cached per device).
int device_check();

inline bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }
inline bool is_pow2(int64_t n) { return n >= 1 && (n & (n - 1)) == 0; }
inline int ilog2(int64_t n) {
  int l = 0;
  while ((int64_t(1) << (l + 1)) <= n) ++l;
  return l;
}

inline int launch_status() {
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? OQ_OK : OQ_ERR_HIP;
}

// ---- 16-row tiled code layout -----------------------------------------------
// Packed int4 codes of an R x K matrix (K % 128 == 0) stored for the small-M
// product: rows are grouped in blocks of 16 (R rounded up to a multiple of 16),
// each row in units of 64 packed bytes (128 codes).  Block (row block rb, unit
// u) is 1024 contiguous bytes laid out as [piece 0..3][row 0..15][16 bytes]:
// lane l of a wave loads bytes 16 l .. 16 l + 15 of a block and receives the
// 16-byte piece l / 16 of row l % 16, which is the operand layout of
// v_mfma_i32_16x16x64_i8.  Byte p of row r lives at
//   ((r / 16) * (K / 128) + p / 64) * 1024 + ((p / 16) % 4) * 256 + (r % 16) * 16 + p % 16.
__host__ __device__ inline int64_t tiled_offset(int64_t r, int64_t p, int64_t units) {
  return (((r >> 4) * units + (p >> 6)) << 10) + (((p >> 4) & 3) << 8) + ((r & 15) << 4) + (p & 15);
}
inline int64_t tiled_bytes(int64_t rows, int64_t K) { return ((rows + 15) / 16) * 16 * (K / 2); }

// ---- rotate-quantize ------------------------------------------------------
struct RQPlan {
  int chunks;   // 16-byte vectors (8 channels) per thread: 1, 2, 3, 4, 6 or 8
  int logT;     // log2(threads per row), 0..8
};
// Split K channels into threads x chunks; false if K is not supported.
bool rq_plan(int64_t K, RQPlan* p);

// Validated launch (no argument checks); ratio != nullptr selects the debug output.
// tiled: Xq is in the 16-row tiled layout (K % 128 == 0) instead of [M][K/2].
// sdelta: static per-channel steps [K] (token scale 1) instead of the
// per-token maximum; rotate_only: write s_t * y in fp32 to `ratio` only;
// i8: 8-bit codes (q_max = 127), one byte per code, Xq [M][K]; cmul:
// per-channel multiplier of the rotated row before its maximum.
int rq_launch(const void* X, int64_t M, int64_t K, int64_t ldx, int had_block, float s_t,
              uint8_t* Xq, float* x_scale, float* ratio, hipStream_t stream, bool tiled = false,
              const float* sdelta = nullptr, bool rotate_only = false, bool i8 = false,
              const float* cmul = nullptr);

// Shape/alignment validation shared by every rotate-quantize entry point.
int rq_validate(const void* X, int64_t M, int64_t K, int64_t ldx, int had_block,
                const void* out, const float* x_scale);

// ---- GELU (tanh form) ---------------------------------------------------------
// gelu_tanh(x) = 0.5 x (1 + tanh(u)), u = sqrt(2/pi) (x + 0.044715 x^3).
// Since 0.5 (1 + tanh(u)) = 1 / (1 + e^(-2u)), this is x / (1 + e^(-2u)):
// one hardware exp and one reciprocal (each within a few fp32 ulp; the result
// is rounded to fp16 by the caller).  e^(-2u) -> inf gives -0 for very
// negative x, e^(-2u) -> 0 gives x.
__device__ __forceinline__ float gelu_tanh(float x) {
  const float k0 = 0.7978845608028654f;  // sqrt(2/pi)
  const float k1 = 0.044715f;
  const float u = k0 * fmaf(k1 * x * x, x, x);
  return x * __builtin_amdgcn_rcpf(1.0f + __expf(-2.0f * u));
}

// ---- GEMM ------------------------------------------------------------------
// EPI_GELU_F16: y = fp16(gelu_tanh(fp16(acc x_scale w_scale + bias))), the
// activation of a non-gated MLP applied to the linear's fp16 output.
enum Epilogue { EPI_I32 = 0, EPI_F16 = 1, EPI_BF16 = 2, EPI_RESID_F32 = 3, EPI_GELU_F16 = 4 };

struct GemmArgs {
  const uint8_t* A;      // [M][K/2]
  const uint8_t* B;      // [N][K/2]
  const float* xs;       // [M]
  const float* ws;       // [N]
  const uint16_t* bias;  // [N] fp16 or null
  void* C;               // output
  const uint16_t* gate;  // EPI_RESID_F32: fp16 [N] per-channel multiplier (null = 1)
  int64_t M, N, K, ldc;
  bool a_tiled;          // A is in the 16-row tiled layout (K % 128 == 0)
  bool a_i8;             // A holds 8-bit codes, one byte each, [M][K] (W4A8)
  // Split-K scratch of the caller (null: no split): int32 partial tiles and
  // one arrival ticket per tile (zero between launches: the last arrival of
  // a tile resets its ticket).  Launches that share them must not overlap.
  int32_t* part = nullptr;
  int32_t* tickets = nullptr;
  int64_t part_words = 0, n_tickets = 0;
  int splitk = 1;        // set by the launcher
};

int gemm_validate(const uint8_t* Xq, int64_t M, const uint8_t* Wq, int64_t N, int64_t K,
                  const void* C, int64_t ldc, int64_t ldc_align);
int gemm_launch(const GemmArgs& a, Epilogue epi, hipStream_t stream);

}  // namespace oq
