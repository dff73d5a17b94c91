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

template <int RW, int KMAX, int G, bool GATHER>
__global__ __launch_bounds__(256) void rq_composite_kernel(const uint16_t* __restrict__ X, int64_t M, int K,
                                                           int64_t ldx, const int32_t* __restrict__ perm,
                                                           const uint16_t* __restrict__ Rt, float s_t,
                                                           uint8_t* __restrict__ Xq, float* __restrict__ xs) {
  // fp16 rows, padded by 16 bytes: the 16 rows of a gather read the same
  // permuted column, and the pad puts them in different LDS banks.
  constexpr int XS = KMAX + 8;
  __shared__ __attribute__((aligned(16))) uint16_t sx[GATHER ? RW * XS : 8];
  __shared__ __attribute__((aligned(16))) int32_t sp[GATHER ? KMAX : 4];  // the permutation
  __shared__ __attribute__((aligned(16))) uint8_t sc[RW * KMAX / 2];  // packed codes
  __shared__ float red[4][16];
  __shared__ float gscale[16];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t row0 = static_cast<int64_t>(blockIdx.x) * RW;
  const int nb = K / kCB;
  const int vpr = K / 8;  // 16-byte pieces per row

  // Stage the rows (rows past M are zeros) and the permutation (clamped into
  // range: a non-permutation keeps every access inside the staged rows).
  if constexpr (GATHER) {
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
        if (p < RW * vpr) *reinterpret_cast<uint4*>(&sx[r * XS + c8 * 8]) = ok[u] ? v[u] : make_uint4(0, 0, 0, 0);
      }
    }
    for (int k4 = tid; k4 < K / 4; k4 += 256) {
      int4 pv = *reinterpret_cast<const int4*>(perm + 4 * k4);
      pv.x = min(max(pv.x, 0), K - 1);
      pv.y = min(max(pv.y, 0), K - 1);
      pv.z = min(max(pv.z, 0), K - 1);
      pv.w = min(max(pv.w, 0), K - 1);
      *reinterpret_cast<int4*>(&sp[4 * k4]) = pv;
    }
  }
  __syncthreads();

  const int r16 = lane & 15, q = lane >> 4;
  const bool rok = r16 < RW;
  const uint16_t* xrow = &sx[GATHER && rok ? r16 * XS : 0];

  // A fragment: rows x 32 permuted channels of block b, k step kk (without a
  // permutation: one 16-byte load per lane from global memory, rows past RW
  // or M zero).
  const bool gok = rok && row0 + r16 < M;
  auto gather = [&](int b, int kk) -> c8h {
    if constexpr (!GATHER) {
      const c8h v = *reinterpret_cast<const c8h*>(X + (gok ? row0 + r16 : 0) * ldx + b * kCB + kk * 32 + 8 * q);
      return gok ? v : c8h{};
    }
    const int k0 = b * kCB + kk * 32 + 8 * q;
    const int4 pa = *reinterpret_cast<const int4*>(&sp[k0]);
    const int4 pb = *reinterpret_cast<const int4*>(&sp[k0 + 4]);
    const int idx[8] = {pa.x, pa.y, pa.z, pa.w, pb.x, pb.y, pb.z, pb.w};
    c8h a;
#pragma unroll
    for (int j = 0; j < 8; ++j) a[j] = __builtin_bit_cast(_Float16, rok ? xrow[idx[j]] : uint16_t(0));
    return a;
  };
  // B fragments of G consecutive blocks of this wave (blocks b0 + 4 g), all
  // loads issued together; blocks past the end read block 0 and are skipped.
  c8h bf[G][4][2];
  auto load_b = [&](int b0) {
#pragma unroll
    for (int gi = 0; gi < G; ++gi) {
      const int b = b0 + 4 * gi < nb ? b0 + 4 * gi : 0;
#pragma unroll
      for (int cb = 0; cb < 4; ++cb)
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
          bf[gi][cb][kk] = *reinterpret_cast<const c8h*>(
              Rt + (static_cast<int64_t>(b) * kCB + cb * 16 + r16) * kCB + kk * 32 + 8 * q);
    }
  };

  // Pass 1: row maxima of |y|.  The B fragments of the next group are in
  // flight while the current group is multiplied (the scheduling barrier
  // keeps the loads ahead of the products).
  float amax[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  load_b(wave);
  for (int b0 = wave; b0 < nb; b0 += 4 * G) {
    c8h cur[G][4][2];
#pragma unroll
    for (int gi = 0; gi < G; ++gi)
#pragma unroll
      for (int cb = 0; cb < 4; ++cb) {
        cur[gi][cb][0] = bf[gi][cb][0];
        cur[gi][cb][1] = bf[gi][cb][1];
      }
    if (b0 + 4 * G < nb) load_b(b0 + 4 * G);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int gi = 0; gi < G; ++gi) {
      const int b = b0 + 4 * gi;
      if (b < nb) {
        const c8h a0 = gather(b, 0), a1 = gather(b, 1);
#pragma unroll
        for (int cb = 0; cb < 4; ++cb) {
          c4f acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a0, cur[gi][cb][0], c4f{0, 0, 0, 0}, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a1, cur[gi][cb][1], acc, 0, 0, 0);
#pragma unroll
          for (int e = 0; e < 4; ++e) amax[e] = fmaxf(amax[e], fabsf(acc[e]));
        }
      }
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

  // Pass 2: codes.  Lanes r16 and r16 ^ 1 hold channels 2i and 2i + 1 of
  // the same row; the even lane packs both into one byte.
  float g[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) g[e] = gscale[4 * q + e];
  load_b(wave);
  for (int b0 = wave; b0 < nb; b0 += 4 * G) {
    c8h cur[G][4][2];
#pragma unroll
    for (int gi = 0; gi < G; ++gi)
#pragma unroll
      for (int cb = 0; cb < 4; ++cb) {
        cur[gi][cb][0] = bf[gi][cb][0];
        cur[gi][cb][1] = bf[gi][cb][1];
      }
    if (b0 + 4 * G < nb) load_b(b0 + 4 * G);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int gi = 0; gi < G; ++gi) {
      const int b = b0 + 4 * gi;
      if (b < nb) {
        const c8h a0 = gather(b, 0), a1 = gather(b, 1);
#pragma unroll
        for (int cb = 0; cb < 4; ++cb) {
          c4f acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a0, cur[gi][cb][0], c4f{0, 0, 0, 0}, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a1, cur[gi][cb][1], acc, 0, 0, 0);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const uint32_t code = __float_as_uint(fmaf(acc[e], g[e], rqd::kRoundMagic)) & 0xFu;
            const uint32_t other = __float_as_uint(rqd::lane_xor<1>(__uint_as_float(code)));
            const int row = 4 * q + e;
            if (row < RW && (r16 & 1) == 0)
              sc[row * (KMAX / 2) + (b * kCB + cb * 16 + r16) / 2] = static_cast<uint8_t>(code | (other << 4));
          }
        }
      }
    }
  }
  __syncthreads();

  // Store 16 packed bytes per thread.
  const int ppr = K / 32;
  for (int p = tid; p < RW * ppr; p += 256) {
    const int r = p / ppr, c32 = p - r * ppr;
    if (row0 + r >= M) continue;
    *reinterpret_cast<uint4*>(Xq + (row0 + r) * static_cast<int64_t>(K / 2) + c32 * 16) =
        *reinterpret_cast<const uint4*>(&sc[r * (KMAX / 2) + c32 * 16]);
  }
}

// Single pass for K <= 4096: eight waves, RG row groups of 16 rows (RW = 16 RG
// rows per workgroup), every y value kept in registers until the row maxima
// are known, so each block matrix is read once per workgroup and reused by
// the RG row groups.  Codes are packed across lanes (channel pairs, then 4
// and 8 channels) and stored as dwords by the lanes holding the first of 8
// channels.
template <int RG, int KMAX, bool GATHER>
__global__ __launch_bounds__(512) void rq_composite1_kernel(const uint16_t* __restrict__ X, int64_t M, int K,
                                                            int64_t ldx, const int32_t* __restrict__ perm,
                                                            const uint16_t* __restrict__ Rt, float s_t,
                                                            uint8_t* __restrict__ Xq, float* __restrict__ xs) {
  constexpr int WAVES = 8, RW = 16 * RG, XS = KMAX + 8;
  constexpr int NBW = KMAX / kCB / WAVES;  // blocks per wave at K = KMAX
  __shared__ __attribute__((aligned(16))) uint16_t sx[GATHER ? RW * XS : 8];
  __shared__ __attribute__((aligned(16))) int32_t sp[GATHER ? KMAX : 4];
  __shared__ float red[WAVES][RW];
  __shared__ float gscale[RW];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t row0 = static_cast<int64_t>(blockIdx.x) * RW;
  const int nb = K / kCB;
  const int vpr = K / 8;

  if constexpr (GATHER) {
    for (int p0 = tid; p0 < RW * vpr; p0 += 512 * 8) {
      uint4 v[8];
      bool ok[8];
  #pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int p = p0 + u * 512;
        const int r = p / vpr, c8 = p - r * vpr;
        ok[u] = p < RW * vpr && row0 + r < M;
        const int64_t gr = ok[u] ? row0 + r : 0;
        v[u] = *reinterpret_cast<const uint4*>(X + gr * ldx + (ok[u] ? c8 * 8 : 0));
      }
  #pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int p = p0 + u * 512;
        const int r = p / vpr, c8 = p - r * vpr;
        if (p < RW * vpr) *reinterpret_cast<uint4*>(&sx[r * XS + c8 * 8]) = ok[u] ? v[u] : make_uint4(0, 0, 0, 0);
      }
    }
    for (int k4 = tid; k4 < K / 4; k4 += 512) {
      int4 pv = *reinterpret_cast<const int4*>(perm + 4 * k4);
      pv.x = min(max(pv.x, 0), K - 1);
      pv.y = min(max(pv.y, 0), K - 1);
      pv.z = min(max(pv.z, 0), K - 1);
      pv.w = min(max(pv.w, 0), K - 1);
      *reinterpret_cast<int4*>(&sp[4 * k4]) = pv;
    }
  }
  __syncthreads();

  const int r16 = lane & 15, q = lane >> 4;
  // Without a permutation (X already in the permuted channel order): the A
  // fragment of rows rg*16 .. + 15 and k step kk of block b is one 16-byte
  // load per lane straight from global memory; rows past M read row 0 and
  // are zeroed where used.
  bool rv[RG];
#pragma unroll
  for (int rg = 0; rg < RG; ++rg) rv[rg] = row0 + rg * 16 + r16 < M;
  auto load_a = [&](int b, c8h (&f)[RG][2]) {
    const int bb = b < nb ? b : 0;
#pragma unroll
    for (int rg = 0; rg < RG; ++rg) {
      const int64_t gr = rv[rg] ? row0 + rg * 16 + r16 : 0;
#pragma unroll
      for (int kk = 0; kk < 2; ++kk)
        f[rg][kk] = *reinterpret_cast<const c8h*>(X + gr * ldx + bb * kCB + kk * 32 + 8 * q);
    }
  };
  auto gather = [&](int b, int kk, int rg) -> c8h {
    const int k0 = b * kCB + kk * 32 + 8 * q;
    const int4 pa = *reinterpret_cast<const int4*>(&sp[k0]);
    const int4 pb = *reinterpret_cast<const int4*>(&sp[k0 + 4]);
    const int idx[8] = {pa.x, pa.y, pa.z, pa.w, pb.x, pb.y, pb.z, pb.w};
    const uint16_t* xrow = &sx[(rg * 16 + r16) * XS];
    c8h a;
#pragma unroll
    for (int j = 0; j < 8; ++j) a[j] = __builtin_bit_cast(_Float16, xrow[idx[j]]);
    return a;
  };

  c4f y[NBW][4][RG];
  float amax[RG][4];
#pragma unroll
  for (int rg = 0; rg < RG; ++rg)
#pragma unroll
    for (int e = 0; e < 4; ++e) amax[rg][e] = 0.0f;
  // The block matrix fragments of block i + 1 are loaded while block i is
  // multiplied (blocks past the end read block 0 and are not used).
  auto load_b = [&](int b, c8h (&f)[4][2]) {
    const int bb = b < nb ? b : 0;
#pragma unroll
    for (int cb = 0; cb < 4; ++cb)
#pragma unroll
      for (int kk = 0; kk < 2; ++kk)
        f[cb][kk] = *reinterpret_cast<const c8h*>(Rt + (static_cast<int64_t>(bb) * kCB + cb * 16 + r16) * kCB +
                                                  kk * 32 + 8 * q);
  };
  c8h bnext[4][2];
  c8h anext[GATHER ? 1 : RG][2];
  load_b(wave, bnext);
  if constexpr (!GATHER) load_a(wave, anext);
#pragma unroll
  for (int i = 0; i < NBW; ++i) {
    const int b = wave + WAVES * i;
    c8h bf[4][2];
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) {
      bf[cb][0] = bnext[cb][0];
      bf[cb][1] = bnext[cb][1];
    }
    c8h af[GATHER ? 1 : RG][2];
    if constexpr (!GATHER) {
#pragma unroll
      for (int rg = 0; rg < RG; ++rg) {
        af[rg][0] = anext[rg][0];
        af[rg][1] = anext[rg][1];
      }
    }
    if (i + 1 < NBW) {
      load_b(b + WAVES, bnext);
      if constexpr (!GATHER) load_a(b + WAVES, anext);
    }
    __builtin_amdgcn_sched_barrier(0);
    if (b < nb) {
#pragma unroll
      for (int rg = 0; rg < RG; ++rg) {
        c8h a0, a1;
        if constexpr (GATHER) {
          a0 = gather(b, 0, rg);
          a1 = gather(b, 1, rg);
        } else {
          a0 = rv[rg] ? af[rg][0] : c8h{};
          a1 = rv[rg] ? af[rg][1] : c8h{};
        }
#pragma unroll
        for (int cb = 0; cb < 4; ++cb) {
          c4f acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a0, bf[cb][0], c4f{0, 0, 0, 0}, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a1, bf[cb][1], acc, 0, 0, 0);
          y[i][cb][rg] = acc;
#pragma unroll
          for (int e = 0; e < 4; ++e) amax[rg][e] = fmaxf(amax[rg][e], fabsf(acc[e]));
        }
      }
    }
  }
#pragma unroll
  for (int rg = 0; rg < RG; ++rg)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float m = amax[rg][e];
      m = fmaxf(m, rqd::lane_xor<1>(m));
      m = fmaxf(m, rqd::lane_xor<2>(m));
      m = fmaxf(m, rqd::lane_xor<4>(m));
      m = fmaxf(m, rqd::lane_xor<8>(m));
      if (r16 == 0) red[wave][rg * 16 + 4 * q + e] = m;
    }
  __syncthreads();
  if (tid < RW) {
    float m = red[0][tid];
#pragma unroll
    for (int w = 1; w < WAVES; ++w) m = fmaxf(m, red[w][tid]);
    const float a_z = m * s_t;
    const float delta = a_z / 7.0f;
    gscale[tid] = delta > 0.0f ? s_t / delta : 0.0f;
    if (row0 + tid < M) xs[row0 + tid] = delta / s_t;
  }
  __syncthreads();

#pragma unroll
  for (int i = 0; i < NBW; ++i) {
    const int b = wave + WAVES * i;
    if (b < nb) {
#pragma unroll
      for (int rg = 0; rg < RG; ++rg)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int row = rg * 16 + 4 * q + e;
          const float g = gscale[row];
#pragma unroll
          for (int cb = 0; cb < 4; ++cb) {
            // code of channel b*64 + cb*16 + r16; pack 8 consecutive channels
            uint32_t c = __float_as_uint(fmaf(y[i][cb][rg][e], g, rqd::kRoundMagic)) & 0xFu;
            c |= __float_as_uint(rqd::lane_xor<1>(__uint_as_float(c))) << 4;
            c |= __float_as_uint(rqd::lane_xor<2>(__uint_as_float(c))) << 8;
            c |= __float_as_uint(rqd::lane_xor<4>(__uint_as_float(c))) << 16;
            if ((r16 & 7) == 0 && row0 + row < M)
              *reinterpret_cast<uint32_t*>(Xq + (row0 + row) * static_cast<int64_t>(K / 2) +
                                           (b * kCB + cb * 16 + r16) / 2) = c;
          }
        }
    }
  }
}

template <int RG, int KMAX, bool GATHER = true>
int launch_composite1(const void* X, int64_t M, int64_t K, int64_t ldx, const int32_t* perm, const void* Rt,
                      float s, uint8_t* Xq, float* x_scale, hipStream_t stream) {
  const unsigned grid = static_cast<unsigned>((M + 16 * RG - 1) / (16 * RG));
  hipLaunchKernelGGL((rq_composite1_kernel<RG, KMAX, GATHER>), dim3(grid), dim3(512), 0, stream,
                     static_cast<const uint16_t*>(X), M, static_cast<int>(K), ldx, perm,
                     static_cast<const uint16_t*>(Rt), s, Xq, x_scale);
  return launch_status();
}

template <int RW, int KMAX, bool GATHER = true>
int launch_composite(const void* X, int64_t M, int64_t K, int64_t ldx, const int32_t* perm, const void* Rt,
                     float s, uint8_t* Xq, float* x_scale, hipStream_t stream) {
  const unsigned grid = static_cast<unsigned>((M + RW - 1) / RW);
  hipLaunchKernelGGL((rq_composite_kernel<RW, KMAX, 2, GATHER>), dim3(grid), dim3(256), 0, stream,
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
  if (!X || !Rt || !Xq || !x_scale) return OQ_ERR_NULL;
  if (!oq::aligned(X, 16) || (perm && !oq::aligned(perm, 16)) || !oq::aligned(Rt, 16) || !oq::aligned(Xq, 16) ||
      !oq::aligned(x_scale, 4))
    return OQ_ERR_ALIGN;
  const float s = s_table ? s_table[t] : 1.0f;
  if (!(s > 0.0f) || !std::isfinite(s)) return OQ_ERR_ARG;
  int st = oq::device_check();
  if (st != OQ_OK) return st;
  hipStream_t h = static_cast<hipStream_t>(stream);
  // Without a permutation the rows are read straight into the MFMA operands
  // (no LDS staging): row groups sized to the register budget.
  if (!perm) {
    // Few rows: one row group per workgroup, so the rows spread over more CUs.
    if (M <= 1024 && K <= 1024) return oq::launch_composite1<1, 1024, false>(X, M, K, ldx, perm, Rt, s, Xq, x_scale, h);
    if (M <= 1024 && K <= 2048) return oq::launch_composite1<1, 2048, false>(X, M, K, ldx, perm, Rt, s, Xq, x_scale, h);
    if (K <= 1024) return oq::launch_composite1<2, 1024, false>(X, M, K, ldx, perm, Rt, s, Xq, x_scale, h);
    if (K <= 2048) return oq::launch_composite1<2, 2048, false>(X, M, K, ldx, perm, Rt, s, Xq, x_scale, h);
    if (K <= 4096) return oq::launch_composite1<1, 4096, false>(X, M, K, ldx, perm, Rt, s, Xq, x_scale, h);
    if (K <= 8192) return oq::launch_composite<16, 8192, false>(X, M, K, ldx, perm, Rt, s, Xq, x_scale, h);
    return oq::launch_composite<16, 16384, false>(X, M, K, ldx, perm, Rt, s, Xq, x_scale, h);
  }
  // Single pass (y in registers) up to K = 4096, row groups sized to the
  // LDS budget; deeper rows take the two-pass kernel.
  // Few rows: one row group per workgroup, so the rows spread over more CUs.
  if (M <= 1024 && K <= 2048) return oq::launch_composite1<1, 2048>(X, M, K, ldx, perm, Rt, s, Xq, x_scale, h);
  if (K <= 1024) return oq::launch_composite1<4, 1024>(X, M, K, ldx, perm, Rt, s, Xq, x_scale, h);
  if (K <= 2048) return oq::launch_composite1<2, 2048>(X, M, K, ldx, perm, Rt, s, Xq, x_scale, h);
  if (K <= 4096) return oq::launch_composite1<1, 4096>(X, M, K, ldx, perm, Rt, s, Xq, x_scale, h);
  if (K <= 8192) return oq::launch_composite<4, 8192>(X, M, K, ldx, perm, Rt, s, Xq, x_scale, h);
  return oq::launch_composite<2, 16384>(X, M, K, ldx, perm, Rt, s, Xq, x_scale, h);
}
