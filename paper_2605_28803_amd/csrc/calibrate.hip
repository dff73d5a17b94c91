// Calibration of the static per-step, per-channel activation steps
// (Section 4.2, eq:perstep_scale): Delta_j = sigma_hat(|Y[:, j]|) / q_max with
// the robust peak sigma_hat taken as the nearest-rank p-th percentile of the
// magnitudes of column j (p = 99.9 in the paper's calibration settings).
//
// The percentile is an order statistic, computed exactly by radix selection
// over the bit patterns of |y|: for non-negative floats the unsigned order of
// the pattern is the numeric order (NaN patterns sort above +inf).  Four
// passes of 8 bits each, most significant first.  A pass histograms, per
// column, the next 8-bit digit of every value whose higher bits equal the
// prefix fixed so far, then one wave per column scans the 256 bins, finds the
// bin holding the remaining rank, appends its digit to the prefix and
// subtracts the counts below it.
//
// Work split of a histogram pass: a workgroup owns 64 columns (one per lane,
// so a wave reads 256 contiguous bytes of a row) and a chunk of rows; the 4
// waves walk the chunk's rows and count in an LDS histogram [256][64]
// (lanes of one wave never share an address), which is flushed to the global
// histogram [K][256] with one atomic per non-zero bin.  The row chunks give
// the launch enough workgroups to fill the chip for any column count.
#include <cmath>
#include <mutex>

#include "common.h"

namespace oq {
namespace {

constexpr int kSlab = 64;           // columns per workgroup
constexpr int kMaxRowSplits = 2048;  // row chunks per column slab

// hist = 0, prefix = 0, rank = k for every column.
__global__ __launch_bounds__(256) void quantile_init_kernel(uint32_t* __restrict__ hist, uint32_t* __restrict__ prefix,
                                                            uint32_t* __restrict__ rank, int64_t K, uint32_t k) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i < K * 64) reinterpret_cast<uint4*>(hist)[i] = make_uint4(0, 0, 0, 0);
  if (i < K) {
    prefix[i] = 0;
    rank[i] = k;
  }
}

__global__ __launch_bounds__(256) void quantile_hist_kernel(const float* __restrict__ Y, int64_t n, int64_t K,
                                                            int64_t ldy, int64_t chunk, int shift,
                                                            const uint32_t* __restrict__ prefix,
                                                            uint32_t* __restrict__ hist) {
  __shared__ uint32_t h[256 * kSlab];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int64_t col = static_cast<int64_t>(blockIdx.x) * kSlab + lane;
  const bool cok = col < K;
  for (int i = threadIdx.x; i < 256 * kSlab; i += 256) h[i] = 0;
  __syncthreads();
  const uint32_t pre = cok ? prefix[col] : 0u;
  const uint32_t hi_mask = shift >= 24 ? 0u : (0xFFFFFFFFu << (shift + 8));
  const int64_t r0 = static_cast<int64_t>(blockIdx.y) * chunk;
  const int64_t r1 = r0 + chunk < n ? r0 + chunk : n;
  const float* yc = Y + (cok ? col : 0);
  // Four rows per wave in flight: loads first, then the counts.
  int64_t r = r0 + wv;
  for (; r + 12 < r1; r += 16) {
    uint32_t b[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) b[u] = __float_as_uint(yc[(r + 4 * u) * ldy]) & 0x7FFFFFFFu;
    if (cok) {
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if ((b[u] & hi_mask) == pre) atomicAdd(&h[((b[u] >> shift) & 255u) * kSlab + lane], 1u);
    }
  }
  for (; r < r1; r += 4) {
    const uint32_t b = __float_as_uint(yc[r * ldy]) & 0x7FFFFFFFu;
    if (cok && (b & hi_mask) == pre) atomicAdd(&h[((b >> shift) & 255u) * kSlab + lane], 1u);
  }
  __syncthreads();
  for (int i = threadIdx.x; i < 256 * kSlab; i += 256) {
    const int d = i / kSlab, c = i % kSlab;
    const uint32_t v = h[i];
    const int64_t cc = static_cast<int64_t>(blockIdx.x) * kSlab + c;
    if (v != 0u && cc < K) atomicAdd(&hist[cc * 256 + d], v);
  }
}

// One wave per column: lane l holds bins 4l .. 4l + 3.  Finds the bin that
// holds the remaining rank, updates prefix and rank, clears the column's
// histogram for the next pass; the last pass writes prefix / q_max.
__global__ __launch_bounds__(256) void quantile_select_kernel(uint32_t* __restrict__ hist, int64_t K, int shift,
                                                              uint32_t* __restrict__ prefix,
                                                              uint32_t* __restrict__ rank, bool last, double qmax,
                                                              float* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  const int64_t col = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (col >= K) return;
  uint4* hc = reinterpret_cast<uint4*>(hist + col * 256) + lane;
  const uint4 c = *hc;
  const uint32_t s = c.x + c.y + c.z + c.w;
  // Inclusive prefix sum of s over the wave.
  uint32_t incl = s;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t t = __shfl_up(incl, o, 64);
    if (lane >= o) incl += t;
  }
  const uint32_t k = rank[col];
  const uint64_t hit = __ballot(incl >= k);
  // The candidates of this pass number at least k, so some lane reaches k;
  // a histogram that does not (it cannot happen) selects the top bin.
  const int L = hit ? __builtin_ctzll(hit) : 63;
  const uint32_t below_lane = __shfl(incl - s, L, 64);
  const uint4 cl = make_uint4(__shfl(c.x, L, 64), __shfl(c.y, L, 64), __shfl(c.z, L, 64), __shfl(c.w, L, 64));
  *hc = make_uint4(0, 0, 0, 0);
  if (lane != 0) return;
  uint32_t acc = below_lane;
  int d = 4 * L;
  const uint32_t cc[4] = {cl.x, cl.y, cl.z, cl.w};
  int i = 0;
  for (; i < 3; ++i) {
    if (acc + cc[i] >= k) break;
    acc += cc[i];
  }
  d += i;
  const uint32_t p = prefix[col] | (static_cast<uint32_t>(d) << shift);
  prefix[col] = p;
  rank[col] = k - acc;
  if (last) out[col] = static_cast<float>(static_cast<double>(__uint_as_float(p)) / qmax);
}

// Launches of one calibration: work = hist [K][256] | prefix [K] | rank [K].
int calibrate_launch(const float* Y, int64_t n, int64_t K, int64_t ldy, double p, float qmax, float* delta,
                     uint32_t* work, hipStream_t s) {
  // Nearest rank: the k-th smallest with k = ceil(p n / 100), in [1, n].  p is
  // taken to 1e-6 percent and the product formed in integers (pm n <= 1e8 *
  // INT32_MAX < 2^63): in floating point 99.9 / 100 * 1000 = 999.0000000000001
  // would round up to the maximum.
  const int64_t pm = std::llround(p * 1e6);
  int64_t k = (pm * n + 99999999) / 100000000;
  if (k < 1) k = 1;
  if (k > n) k = n;
  uint32_t* hist = work;
  uint32_t* prefix = hist + K * 256;
  uint32_t* rank = prefix + K;
  hipLaunchKernelGGL(quantile_init_kernel, dim3(static_cast<unsigned>((K * 64 + 255) / 256)), dim3(256), 0, s,
                     hist, prefix, rank, K, static_cast<uint32_t>(k));
  const int64_t slabs = (K + kSlab - 1) / kSlab;
  // Enough row chunks for ~8 workgroups per CU over the slabs, at least 64
  // rows per chunk.
  int64_t splits = (2048 + slabs - 1) / slabs;
  if (splits > kMaxRowSplits) splits = kMaxRowSplits;
  if (splits > (n + 63) / 64) splits = (n + 63) / 64;
  if (splits < 1) splits = 1;
  const int64_t chunk = (n + splits - 1) / splits;
  splits = (n + chunk - 1) / chunk;
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    hipLaunchKernelGGL(quantile_hist_kernel, dim3(static_cast<unsigned>(slabs), static_cast<unsigned>(splits)),
                       dim3(256), 0, s, Y, n, K, ldy, chunk, shift, prefix, hist);
    hipLaunchKernelGGL(quantile_select_kernel, dim3(static_cast<unsigned>((K + 3) / 4)), dim3(256), 0, s, hist,
                       K, shift, prefix, rank, pass == 3, static_cast<double>(qmax), delta);
  }
  return launch_status();
}

// Argument checks shared by both entry points (before any launch).
int calibrate_check(const float* Y, int64_t n, int64_t K, int64_t ldy, double p, float qmax, float* delta) {
  if (n < 0 || K < 0 || n > INT32_MAX || K > (int64_t(1) << 24) || ldy < K) return OQ_ERR_SHAPE;
  if (!(p > 0.0 && p <= 100.0) || !(qmax > 0.0f) || !std::isfinite(qmax)) return OQ_ERR_ARG;
  if (K == 0) return OQ_OK;
  if (n == 0) return OQ_ERR_SHAPE;  // no order statistic of an empty column
  if (!Y || !delta) return OQ_ERR_NULL;
  if (!aligned(Y, 4) || !aligned(delta, 4)) return OQ_ERR_ALIGN;
  return OQ_OK;
}

// ---- the allocation-free variant -----------------------------------------
// Its histogram, prefixes and ranks live in a file-scope device array, one
// copy per GPU for the life of the process, sized for kScratchMaxK columns.
constexpr int64_t kScratchMaxK = 16384;
constexpr size_t kScratchWords = static_cast<size_t>(kScratchMaxK) * (256 + 2);  // 16.9 MB
constexpr int kMaxDevices = 64;

// The array's address on each device, from hipGetSymbolAddress with that
// device current (the host-side name is not a device address).
std::mutex g_scratch_mu;
uint32_t* g_scratch_ptr[kMaxDevices] = {};

}  // namespace
}  // namespace oq

static __device__ __align__(256) uint32_t scratch[oq::kScratchWords];

namespace oq {
namespace {

int scratch_for_current_device(uint32_t** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return OQ_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return OQ_ERR_DEVICE;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return OQ_ERR_HIP;
    g_scratch_ptr[dev] = static_cast<uint32_t*>(ptr);
  }
  *out = g_scratch_ptr[dev];
  return OQ_OK;
}

}  // namespace
}  // namespace oq

extern "C" size_t oq_calibrate_workspace_bytes(int64_t K) {
  if (K <= 0) return 0;
  return static_cast<size_t>(K) * (256 + 2) * sizeof(uint32_t);
}

extern "C" int oq_calibrate_step_scales(const float* Y, int64_t n, int64_t K, int64_t ldy, double p, float qmax,
                                        float* delta, void* work, size_t work_bytes, void* stream) {
  int e = oq::calibrate_check(Y, n, K, ldy, p, qmax, delta);
  if (e != OQ_OK || K == 0) return e;
  if (!work) return OQ_ERR_NULL;
  if (work_bytes < oq_calibrate_workspace_bytes(K)) return OQ_ERR_SHAPE;
  if (!oq::aligned(work, 16)) return OQ_ERR_ALIGN;
  if ((e = oq::device_check()) != OQ_OK) return e;
  return oq::calibrate_launch(Y, n, K, ldy, p, qmax, delta, static_cast<uint32_t*>(work),
                              static_cast<hipStream_t>(stream));
}

extern "C" int oq_calibrate_step_scales_noalloc(const float* Y, int64_t n, int64_t K, int64_t ldy, double p,
                                                float qmax, float* delta, void* stream) {
  int e = oq::calibrate_check(Y, n, K, ldy, p, qmax, delta);
  if (e != OQ_OK || K == 0) return e;
  if (K > oq::kScratchMaxK) return OQ_ERR_WORKSPACE;
  if ((e = oq::device_check()) != OQ_OK) return e;
  uint32_t* work = nullptr;
  if ((e = oq::scratch_for_current_device(&work)) != OQ_OK) return e;
  return oq::calibrate_launch(Y, n, K, ldy, p, qmax, delta, work, static_cast<hipStream_t>(stream));
}
