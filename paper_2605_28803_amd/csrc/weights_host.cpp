// Offline weight preparation on the host, float64: fold the Hadamard half of the
// rotation into each output row and quantize it per output channel with
// round-to-nearest (eq:transform, eq:scale, eq:quant; RTN as in the
// Implementation Details for the DiT side).  Rows are independent and split
// across std::thread workers.
//
// With a static per-channel activation step Delta_j (eq:perstep_scale, the
// per-channel table), the step multiplies input channel j of the rotated
// weight before the per-row quantization, W''[n][j] = W'[n][j] Delta_j, so
// that sum_j (Delta_j q_j) W'[n][j] = sum_j q_j W''[n][j] keeps an integer
// product with token scale 1.
#include <algorithm>
#include <cmath>
#include <thread>
#include <vector>

#include "common.h"

namespace {

void prepare_rows(const double* W, int64_t r0, int64_t r1, int64_t K, int b, const float* delta, uint8_t* Wq,
                  float* ws) {
  std::vector<double> y(static_cast<size_t>(K));
  const double norm = 1.0 / std::sqrt(static_cast<double>(b));
  for (int64_t n = r0; n < r1; ++n) {
    std::copy(W + n * K, W + (n + 1) * K, y.begin());
    for (int64_t base = 0; base < K; base += b)
      for (int h = 1; h < b; h <<= 1)
        for (int64_t i = base; i < base + b; i += 2 * h)
          for (int64_t j = i; j < i + h; ++j) {
            const double u = y[j], v = y[j + h];
            y[j] = u + v;
            y[j + h] = u - v;
          }
    double amax = 0.0;
    for (int64_t k = 0; k < K; ++k) {
      y[k] *= norm;
      if (delta) y[k] *= static_cast<double>(delta[k]);
      amax = std::max(amax, std::fabs(y[k]));
    }
    const double delta = amax / 7.0;
    ws[n] = static_cast<float>(delta);
    uint8_t* q = Wq + n * (K / 2);
    for (int64_t k = 0; k < K; k += 2) {
      int c[2];
      for (int e = 0; e < 2; ++e) {
        double r = delta > 0.0 ? y[k + e] / delta : 0.0;
        r = std::nearbyint(r);
        c[e] = static_cast<int>(std::min(7.0, std::max(-7.0, r)));
      }
      q[k / 2] = static_cast<uint8_t>((c[0] & 0xF) | ((c[1] & 0xF) << 4));
    }
  }
}

}  // namespace

namespace {

int quantize_rows(const double* W_u, int64_t N, int64_t K, int32_t had_block, const float* delta, uint8_t* Wq,
                  float* w_scale) {
  if (!W_u || !Wq || !w_scale) return OQ_ERR_NULL;
  if (N < 1 || K < 2 || K % 2 != 0 || !oq::is_pow2(had_block) || had_block > OQ_MAX_HAD_BLOCK ||
      K % had_block != 0)
    return OQ_ERR_SHAPE;
  const int64_t hw = std::max(1u, std::thread::hardware_concurrency());
  const int64_t nt = std::min<int64_t>(hw, std::max<int64_t>(1, N / 16));
  std::vector<std::thread> pool;
  for (int64_t i = 0; i < nt; ++i) {
    const int64_t r0 = N * i / nt, r1 = N * (i + 1) / nt;
    pool.emplace_back(prepare_rows, W_u, r0, r1, K, had_block, delta, Wq, w_scale);
  }
  for (auto& th : pool) th.join();
  return OQ_OK;
}

}  // namespace

extern "C" int oq_quantize_weights_host(const double* W_u, int64_t N, int64_t K, int32_t had_block, uint8_t* Wq,
                                        float* w_scale) {
  return quantize_rows(W_u, N, K, had_block, nullptr, Wq, w_scale);
}

extern "C" int oq_quantize_weights_step_host(const double* W_u, int64_t N, int64_t K, int32_t had_block,
                                             const float* delta, uint8_t* Wq, float* w_scale) {
  if (!delta) return OQ_ERR_NULL;
  for (int64_t k = 0; k < K; ++k)
    if (!(delta[k] >= 0.0f) || !std::isfinite(delta[k])) return OQ_ERR_ARG;
  return quantize_rows(W_u, N, K, had_block, delta, Wq, w_scale);
}
