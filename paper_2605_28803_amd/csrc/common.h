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

// ---- rotate-quantize ------------------------------------------------------
struct RQPlan {
  int chunks;   // 16-byte vectors (8 channels) per thread: 1, 2, 3, 4, 6 or 8
  int logT;     // log2(threads per row), 0..8
};
// Split K channels into threads x chunks; false if K is not supported.
bool rq_plan(int64_t K, RQPlan* p);

// Validated launch (no argument checks); ratio != nullptr selects the debug output.
int rq_launch(const void* X, int64_t M, int64_t K, int64_t ldx, int had_block, float s_t,
              uint8_t* Xq, float* x_scale, float* ratio, hipStream_t stream);

// Shape/alignment validation shared by every rotate-quantize entry point.
int rq_validate(const void* X, int64_t M, int64_t K, int64_t ldx, int had_block,
                const void* out, const float* x_scale);

// ---- GEMM ------------------------------------------------------------------
enum Epilogue { EPI_I32 = 0, EPI_F16 = 1, EPI_BF16 = 2, EPI_RESID_F32 = 3 };

struct GemmArgs {
  const uint8_t* A;      // [M][K/2]
  const uint8_t* B;      // [N][K/2]
  const float* xs;       // [M]
  const float* ws;       // [N]
  const uint16_t* bias;  // [N] fp16 or null
  void* C;               // output
  const uint16_t* gate;  // EPI_RESID_F32: fp16 [N] per-channel multiplier (null = 1)
  int64_t M, N, K, ldc;
};

int gemm_validate(const uint8_t* Xq, int64_t M, const uint8_t* Wq, int64_t N, int64_t K,
                  const void* C, int64_t ldc, int64_t ldc_align);
int gemm_launch(const GemmArgs& a, Epilogue epi, hipStream_t stream);

}  // namespace oq
