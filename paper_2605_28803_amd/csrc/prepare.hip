// Offline preparation of a weight for the full composite rotation, on the
// GPU (Section 4.1: zigzag permutation P from weight channel energies, the
// per-block factor U_b of the SVD of each block's weight rows, R_b = U_b H_64 /
// 8, and the fold W' = W P R_hat with round-to-nearest per output channel).
//
// Orientation: the weight is stored [N][K] (output-major), so input channel j
// is column j and block b's weight rows (the paper's C_in x C_out orientation)
// are the 64 columns perm[64 b .. 64 b + 63] of W, a 64 x N matrix W_b.
//
//  * Channel energies e_j = sum_n W[n][j]^2 in fp64, one workgroup per 64
//    columns with a fixed reduction order (deterministic, so exactly equal
//    columns get exactly equal energies).
//  * Zigzag order: the descending rank of e_j (ties to the lower index) by
//    counting, one thread per channel, then the snake deal over the blocks.
//  * U_b: the left singular vectors of W_b are the eigenvectors of the Gram
//    matrix G_b = W_b W_b^T, with sigma_i^2 its eigenvalues.  G_b is formed in
//    fp64 (exact products of fp16 values) in LDS, and diagonalized by the
//    cyclic Jacobi method in fp64: each sweep visits all 2016 index pairs in
//    63 steps of 32 disjoint pairs (round-robin order), the rotations of a
//    step applied together as a column pass over G and V and a row pass over
//    G; sweeps stop when one applies no rotation (at most 40).  Eigenpairs are ordered by
//    descending eigenvalue (ties to the lower index) and each vector's sign
//    is fixed so that its entry of largest magnitude (the first on ties) is
//    positive.  One workgroup per block.
//  * R_b = U_b H_64 / 8 in fp64, rounded once to fp16 (round half to even)
//    and stored column-major per block, the operand the online composite
//    kernel reads.
//  * The fold and RTN are the online composite rotate-quantize applied to
//    the weight rows (s_t = 1): codes per output channel and its scale.
#include <cmath>

#include "common.h"

extern "C" int oq_rotate_quantize_act_composite(const void* X, int64_t M, int64_t K, int64_t ldx,
                                                const int32_t* perm, const void* Rt, const float* s_table,
                                                int32_t t, uint8_t* Xq, float* x_scale, void* stream);

namespace oq {
namespace {

constexpr int kB = 64;        // block size (the paper's)
constexpr int kLd = kB + 1;   // padded LDS row of the 64 x 64 matrices
constexpr int kMaxSweeps = 40;

__device__ __forceinline__ double h2d(uint16_t h) {
  return static_cast<double>(static_cast<float>(__builtin_bit_cast(_Float16, h)));
}

// fp64 -> fp16 bits, one rounding (half to even), from the fp64 bit pattern:
// the 53-bit significand is shifted to the fp16 precision of the value's
// binade (10 fraction bits for normal fp16, fewer for subnormal) with an
// exact remainder test.  |x| >= 65520 gives infinity (R_b entries are
// bounded by 1).
__device__ __forceinline__ uint16_t f64_to_f16_rne(double x) {
  const uint64_t bits = __double_as_longlong(x);
  const uint16_t sign = static_cast<uint16_t>((bits >> 48) & 0x8000u);
  const int e = static_cast<int>((bits >> 52) & 0x7FF);
  if (e == 0) return sign;                    // zero or fp64 subnormal: far below fp16 range
  if (e == 0x7FF) return sign | 0x7C00u;      // inf (NaN is not produced here)
  const int ue = e - 1023;                    // unbiased exponent
  if (ue >= 16) return sign | 0x7C00u;
  const uint64_t mant = (bits & ((uint64_t(1) << 52) - 1)) | (uint64_t(1) << 52);
  const int e16 = ue + 15;                    // biased fp16 exponent if normal
  const int shift = e16 >= 1 ? 42 : 42 + (1 - e16);
  if (shift >= 54) return sign;               // below half the smallest subnormal
  uint64_t q = mant >> shift;
  const uint64_t rem = mant & ((uint64_t(1) << shift) - 1);
  const uint64_t half = uint64_t(1) << (shift - 1);
  if (rem > half || (rem == half && (q & 1))) ++q;
  uint32_t r;
  if (e16 >= 1) r = (static_cast<uint32_t>(e16) << 10) + static_cast<uint32_t>(q) - 1024u;  // carry moves the exponent
  else r = static_cast<uint32_t>(q);                                                       // subnormal (q = 1024: smallest normal)
  if (r >= 0x7C00u) r = 0x7C00u;
  return sign | static_cast<uint16_t>(r);
}

// e[j] = sum_n W[n][j]^2: 64 columns per workgroup (one per lane), 16 waves
// over the rows (wave w takes rows w, w + 16, ...), waves summed in order.
__global__ __launch_bounds__(1024) void energy_kernel(const uint16_t* __restrict__ W, int64_t N, int64_t K,
                                                      int64_t ldw, double* __restrict__ e) {
  __shared__ double part[16][64];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int64_t col = static_cast<int64_t>(blockIdx.x) * 64 + lane;
  const bool ok = col < K;
  const uint16_t* wc = W + (ok ? col : 0);
  double acc = 0.0;
  int64_t n = wv;
  for (; n + 48 < N; n += 64) {
    const double a0 = h2d(wc[n * ldw]), a1 = h2d(wc[(n + 16) * ldw]);
    const double a2 = h2d(wc[(n + 32) * ldw]), a3 = h2d(wc[(n + 48) * ldw]);
    acc = fma(a0, a0, acc);
    acc = fma(a1, a1, acc);
    acc = fma(a2, a2, acc);
    acc = fma(a3, a3, acc);
  }
  for (; n < N; n += 16) {
    const double a = h2d(wc[n * ldw]);
    acc = fma(a, a, acc);
  }
  part[wv][lane] = acc;
  __syncthreads();
  if (wv == 0 && ok) {
    double s = 0.0;
    for (int w = 0; w < 16; ++w) s += part[w][lane];
    e[col] = s;
  }
}

// perm from energies: thread j counts the channels ranked before it
// (larger energy, or equal energy and lower index), then deals rank i to
// round i / nb and block (round even ? i % nb : nb - 1 - i % nb), slot round.
__global__ __launch_bounds__(256) void zigzag_kernel(const double* __restrict__ e, int K, int nb,
                                                     int32_t* __restrict__ perm) {
  __shared__ double chunk[2048];
  const int j = blockIdx.x * 256 + threadIdx.x;
  const double ej = j < K ? e[j] : 0.0;
  int rank = 0;
  for (int base = 0; base < K; base += 2048) {
    const int len = K - base < 2048 ? K - base : 2048;
    __syncthreads();
    for (int i = threadIdx.x; i < len; i += 256) chunk[i] = e[base + i];
    __syncthreads();
    for (int i = 0; i < len; ++i) {
      const double x = chunk[i];
      rank += (x > ej || (x == ej && base + i < j)) ? 1 : 0;
    }
  }
  if (j >= K) return;
  const int c = K / nb;
  const int r = rank / nb, p = rank % nb;
  const int b = (r & 1) ? nb - 1 - p : p;
  perm[b * c + r] = j;
}

// Pair m of step k of the round-robin order over 64 indices: (k, 63) for
// m = 0, ((k + m) mod 63, (k - m) mod 63) otherwise; every unordered pair
// occurs in exactly one of the 63 steps.
__device__ __forceinline__ void rr_pair(int k, int m, int* p, int* q) {
  int a, b;
  if (m == 0) {
    a = k;
    b = 63;
  } else {
    a = (k + m) % 63;
    b = (k - m + 63) % 63;
  }
  *p = a < b ? a : b;
  *q = a < b ? b : a;
}

// One workgroup (256 threads) per 64-channel block.
__global__ __launch_bounds__(256) void block_eig_kernel(const uint16_t* __restrict__ W, int64_t N, int64_t K,
                                                        int64_t ldw, const int32_t* __restrict__ perm,
                                                        double* __restrict__ U, double* __restrict__ lam) {
  __shared__ double X[64][64];    // a chunk of 64 rows of W_b^T (row n, column = block channel)
  __shared__ double A[kB][kLd];   // G_b, then its Jacobi iterates
  __shared__ double V[kB][kLd];   // accumulated rotations
  __shared__ int cols[kB];
  __shared__ int pp[32], pq[32];
  __shared__ double pc[32], ps[32];
  __shared__ int nrot;
  __shared__ double trace;
  __shared__ double dg[kB];
  __shared__ int rk[kB];
  const int tid = threadIdx.x;
  const int b = blockIdx.x;
  if (tid < kB) {
    const int32_t c = perm[b * kB + tid];  // clamped: an out-of-range entry cannot address outside the row
    cols[tid] = c < 0 ? 0 : (c >= K ? static_cast<int>(K - 1) : c);
  }
  __syncthreads();

  // Gram matrix: thread t accumulates G[i][j0 .. j0 + 15], i = t / 4.
  const int gi = tid >> 2, gj0 = (tid & 3) * 16;
  double acc[16];
#pragma unroll
  for (int u = 0; u < 16; ++u) acc[u] = 0.0;
  for (int64_t n0 = 0; n0 < N; n0 += 64) {
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int idx = tid + 256 * u;          // 4096 entries of the chunk
      const int rr = idx >> 6, cc = idx & 63;
      const int64_t n = n0 + rr;
      const int64_t nc = n < N ? n : N - 1;   // clamped row; its value is replaced by 0
      const double v = h2d(W[nc * ldw + cols[cc]]);
      X[rr][cc] = n < N ? v : 0.0;
    }
    __syncthreads();
    for (int rr = 0; rr < 64; ++rr) {
      const double xi = X[rr][gi];
#pragma unroll
      for (int u = 0; u < 16; ++u) acc[u] = fma(xi, X[rr][gj0 + u], acc[u]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int u = 0; u < 16; ++u) {
    A[gi][gj0 + u] = acc[u];
    V[gi][gj0 + u] = gi == gj0 + u ? 1.0 : 0.0;
  }
  __syncthreads();
  if (tid == 0) {
    double t = 0.0;
    for (int i = 0; i < kB; ++i) t += A[i][i];
    trace = t;
  }
  __syncthreads();
  const double abs_floor = 0x1p-52 * trace;

  // Cyclic Jacobi.  A pair is rotated unless |a_pq| is negligible against
  // the diagonal, |a_pq| <= 2^-53 sqrt(|a_pp a_qq|), or at the rounding level
  // of the whole matrix, |a_pq| <= 2^-52 trace(G) (entries of a numerically
  // null eigenspace would otherwise keep rotating among themselves).
  for (int sweep = 0; sweep < kMaxSweeps; ++sweep) {
    if (tid == 0) nrot = 0;
    __syncthreads();
    for (int k = 0; k < 63; ++k) {
      if (tid < 32) {
        int p, q;
        rr_pair(k, tid, &p, &q);
        const double app = A[p][p], aqq = A[q][q], apq = A[p][q];
        double c = 1.0, s = 0.0;
        if (apq != 0.0 && fabs(apq) > fmax(0x1p-53 * sqrt(fabs(app * aqq)), abs_floor)) {
          const double theta = (aqq - app) / (2.0 * apq);
          const double t = (theta >= 0.0 ? 1.0 : -1.0) / (fabs(theta) + sqrt(fma(theta, theta, 1.0)));
          c = 1.0 / sqrt(fma(t, t, 1.0));
          s = t * c;
          if (s != 0.0) atomicAdd(&nrot, 1);
          else c = 1.0;
        }
        pp[tid] = p;
        pq[tid] = q;
        pc[tid] = c;
        ps[tid] = s;
      }
      __syncthreads();
      // Columns p, q of A and V (rows r, 64 x 32 items over 256 threads).
      for (int it = tid; it < 64 * 32; it += 256) {
        const int m = it & 31, r = it >> 5;
        const int p = pp[m], q = pq[m];
        const double c = pc[m], s = ps[m];
        if (s != 0.0) {
          const double arp = A[r][p], arq = A[r][q];
          A[r][p] = c * arp - s * arq;
          A[r][q] = s * arp + c * arq;
          const double vrp = V[r][p], vrq = V[r][q];
          V[r][p] = c * vrp - s * vrq;
          V[r][q] = s * vrp + c * vrq;
        }
      }
      __syncthreads();
      // Rows p, q of A.
      for (int it = tid; it < 64 * 32; it += 256) {
        const int m = it & 31, r = it >> 5;
        const int p = pp[m], q = pq[m];
        const double c = pc[m], s = ps[m];
        if (s != 0.0) {
          const double apr = A[p][r], aqr = A[q][r];
          A[p][r] = c * apr - s * aqr;
          A[q][r] = s * apr + c * aqr;
        }
      }
      __syncthreads();
    }
    if (nrot == 0) break;  // read by every thread after the last barrier of the sweep
    __syncthreads();       // nobody resets nrot before everyone has read it
  }

  // Order and signs.
  if (tid < kB) dg[tid] = A[tid][tid];
  __syncthreads();
  if (tid < kB) {
    const double li = dg[tid];
    int r = 0;
    for (int j = 0; j < kB; ++j) r += (dg[j] > li || (dg[j] == li && j < tid)) ? 1 : 0;
    rk[tid] = r;
    lam[static_cast<int64_t>(b) * kB + r] = li;
    int arg = 0;
    double best = -1.0;
    for (int rr = 0; rr < kB; ++rr) {
      const double a = fabs(V[rr][tid]);
      if (a > best) {
        best = a;
        arg = rr;
      }
    }
    dg[tid] = V[arg][tid] < 0.0 ? -1.0 : 1.0;  // reuse: the sign of column tid
  }
  __syncthreads();
  for (int it = tid; it < kB * kB; it += 256) {
    const int r = it >> 6, i = it & 63;
    U[(static_cast<int64_t>(b) * kB + r) * kB + rk[i]] = dg[i] * V[r][i];
  }
}

// Rt[b][j][r] = fp16(R_b[r][j]), R_b[r][j] = sum_i U_b[r][i] H[i][j] / 8.
__global__ __launch_bounds__(256) void block_rot_kernel(const double* __restrict__ U, int nb,
                                                        uint16_t* __restrict__ Rt) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= static_cast<int64_t>(nb) * kB * kB) return;
  const int b = static_cast<int>(idx / (kB * kB));
  const int j = static_cast<int>((idx / kB) % kB), r = static_cast<int>(idx % kB);
  const double* ur = U + (static_cast<int64_t>(b) * kB + r) * kB;
  double s = 0.0;
  for (int i = 0; i < kB; ++i) s += (__popc(i & j) & 1) ? -ur[i] : ur[i];
  Rt[idx] = f64_to_f16_rne(s * 0.125);
}

int check_weight(const void* W, int64_t N, int64_t K, int64_t ldw) {
  if (N < 1 || K < kB || K % kB != 0 || K > 16384 || ldw < K) return OQ_ERR_SHAPE;
  if (!W) return OQ_ERR_NULL;
  if (!aligned(W, 2)) return OQ_ERR_ALIGN;
  return OQ_OK;
}

}  // namespace
}  // namespace oq

extern "C" int oq_channel_energy(const void* W, int64_t N, int64_t K, int64_t ldw, double* energy, void* stream) {
  if (N < 1 || K < 1 || ldw < K) return OQ_ERR_SHAPE;
  if (!W || !energy) return OQ_ERR_NULL;
  if (!oq::aligned(W, 2) || !oq::aligned(energy, 8)) return OQ_ERR_ALIGN;
  int st = oq::device_check();
  if (st != OQ_OK) return st;
  hipLaunchKernelGGL(oq::energy_kernel, dim3(static_cast<unsigned>((K + 63) / 64)), dim3(1024), 0,
                     static_cast<hipStream_t>(stream), static_cast<const uint16_t*>(W), N, K, ldw, energy);
  return oq::launch_status();
}

extern "C" int oq_zigzag_permutation(const double* energy, int64_t K, int32_t block, int32_t* perm, void* stream) {
  if (block < 1 || K < block || K % block != 0 || K > 65536) return OQ_ERR_SHAPE;
  if (!energy || !perm) return OQ_ERR_NULL;
  if (!oq::aligned(energy, 8) || !oq::aligned(perm, 4)) return OQ_ERR_ALIGN;
  int st = oq::device_check();
  if (st != OQ_OK) return st;
  hipLaunchKernelGGL(oq::zigzag_kernel, dim3(static_cast<unsigned>((K + 255) / 256)), dim3(256), 0,
                     static_cast<hipStream_t>(stream), energy, static_cast<int>(K), static_cast<int>(K / block),
                     perm);
  return oq::launch_status();
}

extern "C" int oq_block_svd(const void* W, int64_t N, int64_t K, int64_t ldw, const int32_t* perm, int32_t block,
                            double* U, double* sigma2, void* stream) {
  int st = oq::check_weight(W, N, K, ldw);
  if (st != OQ_OK) return st;
  if (block != oq::kB) return OQ_ERR_SHAPE;
  if (!perm || !U || !sigma2) return OQ_ERR_NULL;
  if (!oq::aligned(perm, 4) || !oq::aligned(U, 8) || !oq::aligned(sigma2, 8)) return OQ_ERR_ALIGN;
  if ((st = oq::device_check()) != OQ_OK) return st;
  hipLaunchKernelGGL(oq::block_eig_kernel, dim3(static_cast<unsigned>(K / oq::kB)), dim3(256), 0,
                     static_cast<hipStream_t>(stream), static_cast<const uint16_t*>(W), N, K, ldw, perm, U, sigma2);
  return oq::launch_status();
}

extern "C" int oq_block_rotations(const double* U, int64_t K, int32_t block, uint16_t* Rt, void* stream) {
  if (block != oq::kB || K < oq::kB || K % oq::kB != 0 || K > 16384) return OQ_ERR_SHAPE;
  if (!U || !Rt) return OQ_ERR_NULL;
  if (!oq::aligned(U, 8) || !oq::aligned(Rt, 2)) return OQ_ERR_ALIGN;
  int st = oq::device_check();
  if (st != OQ_OK) return st;
  const int64_t total = K * oq::kB;
  hipLaunchKernelGGL(oq::block_rot_kernel, dim3(static_cast<unsigned>((total + 255) / 256)), dim3(256), 0,
                     static_cast<hipStream_t>(stream), U, static_cast<int>(K / oq::kB), Rt);
  return oq::launch_status();
}

extern "C" size_t oq_prepare_weights_workspace_bytes(int64_t K) {
  if (K <= 0) return 0;
  // energies K doubles, U K * 64 doubles, sigma^2 K doubles
  return static_cast<size_t>(K) * (1 + oq::kB + 1) * sizeof(double);
}

extern "C" int oq_prepare_weights_composite(const void* W, int64_t N, int64_t K, int64_t ldw, int32_t* perm,
                                            uint16_t* Rt, uint8_t* Wq, float* w_scale, void* work,
                                            size_t work_bytes, void* stream) {
  int st = oq::check_weight(W, N, K, ldw);
  if (st != OQ_OK) return st;
  if (!perm || !Rt || !Wq || !w_scale || !work) return OQ_ERR_NULL;
  if (work_bytes < oq_prepare_weights_workspace_bytes(K)) return OQ_ERR_SHAPE;
  if (ldw % 8 != 0) return OQ_ERR_ALIGN;
  if (!oq::aligned(W, 16) || !oq::aligned(perm, 4) || !oq::aligned(Rt, 16) || !oq::aligned(Wq, 16) ||
      !oq::aligned(w_scale, 4) || !oq::aligned(work, 16))
    return OQ_ERR_ALIGN;
  if ((st = oq::device_check()) != OQ_OK) return st;
  double* energy = static_cast<double*>(work);
  double* U = energy + K;
  double* sigma2 = U + K * oq::kB;
  if ((st = oq_channel_energy(W, N, K, ldw, energy, stream)) != OQ_OK) return st;
  if ((st = oq_zigzag_permutation(energy, K, oq::kB, perm, stream)) != OQ_OK) return st;
  if ((st = oq_block_svd(W, N, K, ldw, perm, oq::kB, U, sigma2, stream)) != OQ_OK) return st;
  if ((st = oq_block_rotations(U, K, oq::kB, Rt, stream)) != OQ_OK) return st;
  return oq_rotate_quantize_act_composite(W, N, K, ldw, perm, Rt, nullptr, 0, Wq, w_scale, stream);
}
