// Offline preparation of the full composite rotation on the host, float64
// (Section 4.1, "Block-wise Implementation", eq:blockdiag, eq:transform):
//  - the zigzag channel permutation from per-channel weight energies,
//  - the block matrices R_b = U_b H_c / sqrt(c) in the device format of
//    oq_rotate_quantize_act_composite (fp16, each block column-major),
//  - the weight folded with the same transform and quantized per output
//    channel with round-to-nearest (eq:scale, eq:quant).
#include <algorithm>
#include <cmath>
#include <numeric>
#include <thread>
#include <vector>

#include "common.h"

namespace {

int hadamard_sign(int i, int j) { return (__builtin_popcount(static_cast<unsigned>(i & j)) & 1) ? -1 : 1; }

double f16_value(uint16_t h) { return static_cast<double>(__builtin_bit_cast(_Float16, h)); }

void fold_rows(const double* W, int64_t r0, int64_t r1, int64_t K, int c, const int32_t* perm, const uint16_t* Rt,
               uint8_t* Wq, float* ws) {
  std::vector<double> y(static_cast<size_t>(K));
  for (int64_t n = r0; n < r1; ++n) {
    const double* wr = W + n * K;
    double amax = 0.0;
    for (int64_t b = 0; b < K / c; ++b)
      for (int j = 0; j < c; ++j) {
        // y[b c + j] = sum_i W[n][perm[b c + i]] R_b[i][j], R_b[i][j] = Rt[b][j][i]
        const uint16_t* col = Rt + (b * c + j) * c;
        double acc = 0.0;
        for (int i = 0; i < c; ++i) acc += wr[perm[b * c + i]] * f16_value(col[i]);
        y[b * c + j] = acc;
        amax = std::max(amax, std::fabs(acc));
      }
    const double delta = amax / 7.0;
    ws[n] = static_cast<float>(delta);
    uint8_t* q = Wq + n * (K / 2);
    for (int64_t k = 0; k < K; k += 2) {
      int cd[2];
      for (int e = 0; e < 2; ++e) {
        const double r = delta > 0.0 ? std::nearbyint(y[k + e] / delta) : 0.0;
        cd[e] = static_cast<int>(std::min(7.0, std::max(-7.0, r)));
      }
      q[k / 2] = static_cast<uint8_t>((cd[0] & 0xF) | ((cd[1] & 0xF) << 4));
    }
  }
}

}  // namespace

extern "C" int oq_zigzag_permutation_host(const double* energy, int64_t K, int32_t block, int32_t* perm) {
  if (!energy || !perm) return OQ_ERR_NULL;
  if (K < 1 || block < 1 || K % block != 0) return OQ_ERR_SHAPE;
  const int64_t nblk = K / block;
  std::vector<int64_t> order(static_cast<size_t>(K));
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(), [&](int64_t a, int64_t b) { return energy[a] > energy[b]; });
  for (int64_t i = 0; i < K; ++i) {
    const int64_t r = i / nblk, p = i % nblk;
    const int64_t b = (r % 2 == 0) ? p : nblk - 1 - p;
    perm[b * block + r] = static_cast<int32_t>(order[static_cast<size_t>(i)]);
  }
  return OQ_OK;
}

extern "C" int oq_block_rotations_host(const double* U, int64_t K, int32_t block, uint16_t* Rt) {
  if (!U || !Rt) return OQ_ERR_NULL;
  if (!oq::is_pow2(block) || block > 4096 || K < block || K % block != 0) return OQ_ERR_SHAPE;
  const int c = block;
  const double norm = 1.0 / std::sqrt(static_cast<double>(c));
  for (int64_t b = 0; b < K / c; ++b) {
    const double* ub = U + b * c * c;  // row-major U_b[i][m]
    for (int i = 0; i < c; ++i)
      for (int j = 0; j < c; ++j) {
        double acc = 0.0;
        for (int m = 0; m < c; ++m) acc += ub[i * c + m] * hadamard_sign(m, j);
        const _Float16 h = static_cast<_Float16>(acc * norm);
        Rt[(b * c + j) * c + i] = __builtin_bit_cast(uint16_t, h);
      }
  }
  return OQ_OK;
}

extern "C" int oq_quantize_weights_composite_host(const double* W_u, int64_t N, int64_t K, int32_t block,
                                                  const int32_t* perm, const uint16_t* Rt, uint8_t* Wq,
                                                  float* w_scale) {
  if (!W_u || !perm || !Rt || !Wq || !w_scale) return OQ_ERR_NULL;
  if (N < 1 || !oq::is_pow2(block) || block > 4096 || K < block || K % block != 0 || K % 2 != 0)
    return OQ_ERR_SHAPE;
  for (int64_t k = 0; k < K; ++k)
    if (perm[k] < 0 || perm[k] >= K) return OQ_ERR_ARG;
  const int64_t hw = std::max(1u, std::thread::hardware_concurrency());
  const int64_t nt = std::min<int64_t>(hw, std::max<int64_t>(1, N / 16));
  std::vector<std::thread> pool;
  for (int64_t i = 0; i < nt; ++i) {
    const int64_t r0 = N * i / nt, r1 = N * (i + 1) / nt;
    pool.emplace_back(fold_rows, W_u, r0, r1, K, block, perm, Rt, Wq, w_scale);
  }
  for (auto& th : pool) th.join();
  return OQ_OK;
}
