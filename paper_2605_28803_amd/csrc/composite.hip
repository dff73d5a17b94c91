// Online composite rotation of Section 4.1 with per-token int4 quantization.
//
// eq:transform: X' = X P R_hat with P a channel permutation and R_hat =
// BlockDiag(R_1 .. R_K), R_b = U_b H_c (eq:blockdiag), block size c = 64 (the
// paper's setting).  Then the step scale and the per-token quantizer of
// Section 4.2 (eq:scale, eq:quant; eq:perstep_scale in its per-(layer, step)
// scalar form): z = s_t y, Delta = max|z| / 7, q = round_half_even(z / Delta),
// x_scale = Delta / s_t.
//
// Three kernels.  Up to K = 4096, rq_composite1_kernel keeps whole rows in
// LDS and every y value in registers (one pass).  Above, rq_composite_x_kernel
// splits each row into chunks of channels whose workgroups exchange their
// partial row maxima (one pass, each y computed once); K that no chunk width
// divides takes the two-pass rq_composite_kernel described next.
//
// Two-pass kernel: one workgroup of four waves owns RW rows.  The rows are
// staged in LDS as fp16.  Pass 1: wave w takes the 64-channel blocks b = w, w + 4, ...; for
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
#include <algorithm>
#include <cmath>
#include <mutex>

#include "common.h"
#include "rq_device.h"

namespace oq {
namespace {

typedef _Float16 c8h __attribute__((ext_vector_type(8)));
typedef float c4f __attribute__((ext_vector_type(4)));

constexpr int kCB = 64;  // block size c

// Address-space-qualified pointers for the direct global -> LDS load builtin.
typedef __attribute__((address_space(1))) void gmem_void;
typedef __attribute__((address_space(3))) void lds_void;

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

// ---------------------------------------------------------------------------
// Rows wider than a workgroup can stage (K > 4096, and K = 4096 with P
// folded): the permuted channels of a row are cut into nq = K / C chunks of C
// channels, and each (tile of R = 16 RG rows, chunk) pair is one workgroup, so
// that each block matrix R_b is read once per R rows instead of once per few
// rows.  The nq workgroups of a
// tile exchange their rows' partial maxima through per-launch slots in global
// memory (initialised to -1 by comp_prep_kernel; a published maximum is >= 0)
// and each quantizes its own chunk, so every y value is computed once and
// stays in registers.
//
// Staging: each thread owns K / 8 / 512 pieces of 8 input channels; with the
// online permutation it looks up the permuted position j = P^-1(k) of each of
// its channels once (pinv, written by comp_prep_kernel) and, for every row,
// loads the piece with one 16-byte read and writes the channels whose j falls
// in this chunk to LDS at j - qC.  The whole row is read by each of the nq
// workgroups (from L2: the tile's workgroups are placed on one XCD, adjacent
// in dispatch order).  Without a permutation the chunk's columns are copied
// directly.
//
// Exchange: the tile's workgroups are dispatched together (ids x + 8 (nq t' +
// q) for XCD x), so a workgroup only waits for partners dispatched at the same
// time.  The wait polls with agent-scope atomic loads and is bounded; if the
// bound is ever reached the tile's token scales are written as NaN (never a
// silent result) and the workgroup finishes, so the grid always drains.
// ---------------------------------------------------------------------------
constexpr int kPollLimit = 1 << 20;

__global__ __launch_bounds__(256) void comp_prep_kernel(const int32_t* __restrict__ perm, int K,
                                                        uint16_t* __restrict__ pinv, float* __restrict__ slots,
                                                        int64_t nslots) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  // A perm entry out of range is clamped, so every write stays inside pinv
  // (a non-permutation gives wrong codes, never an access out of bounds).
  if (perm && i < K) pinv[min(max(perm[i], 0), K - 1)] = static_cast<uint16_t>(i);
  if (i < nslots) slots[i] = -1.0f;
}

template <int RG, int C, bool GATHER, int WAVES, int PF>
__global__ __launch_bounds__(64 * WAVES) void rq_composite_x_kernel(
    const uint16_t* __restrict__ X, int64_t M, int K, int64_t ldx, const uint16_t* __restrict__ pinv,
    const uint16_t* __restrict__ Rt, float s_t, uint8_t* __restrict__ Xq, float* __restrict__ xs,
    float* __restrict__ slots, int nq, int ntiles) {
  constexpr int NT = 64 * WAVES;
  constexpr int R = 16 * RG, XS = C + 8;
  constexpr int NBC = C / kCB, NBW = NBC / WAVES;  // blocks per chunk, per wave
  static_assert(NBW >= 1 && NBC % WAVES == 0, "chunk blocks per wave");
  static_assert(PF >= 2, "block matrix ring depth");
  __shared__ __attribute__((aligned(16))) uint16_t sx[R * XS];
  __shared__ float red[WAVES][R];
  __shared__ float gscale[R];
  __shared__ int timed_out;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int xcd = blockIdx.x % 8, idx = blockIdx.x / 8;
  const int q = idx % nq;
  const int tile = (idx / nq) * 8 + xcd;
  if (tile >= ntiles) return;  // every workgroup of such a tile id returns
  const int64_t row0 = static_cast<int64_t>(tile) * R;
  const int cbase = q * C;
  if (tid == 0) timed_out = 0;

  // ---- y = x_chunk . BlockDiag(R_b) for this wave's NBW blocks, kept in
  // registers.  The block matrices run through a ring of PF register stages;
  // the first PF - 1 are requested before the rows are staged.
  const int r16 = lane & 15, qq = lane >> 4;
  const int wb0 = wave * NBW;  // first block of this wave within the chunk
  auto load_b = [&](int i, c8h (&f)[4][2]) {
    const int64_t gb = static_cast<int64_t>(q) * NBC + wb0 + (i < NBW ? i : 0);
#pragma unroll
    for (int cb = 0; cb < 4; ++cb)
#pragma unroll
      for (int kk = 0; kk < 2; ++kk)
        f[cb][kk] = *reinterpret_cast<const c8h*>(Rt + (gb * kCB + cb * 16 + r16) * kCB + kk * 32 + 8 * qq);
  };
  c8h bring[PF][4][2];
#pragma unroll
  for (int i = 0; i < PF - 1; ++i)
    if (i < NBW) load_b(i, bring[i]);
  // ---- Stage the chunk of R rows in LDS (rows past M as zeros).
  if constexpr (GATHER) {
    const int npc = K / 8;                       // pieces per row
    constexpr int PMAX = 16384 / 8 / NT;         // pieces per thread at K = 16384
    const int ppc = (npc + NT - 1) / NT;         // pieces per thread here
    uint32_t dst[PMAX][4];                       // local positions of the 8 channels, 2 per word, 0xFFFF = none
#pragma unroll
    for (int pi = 0; pi < PMAX; ++pi) {
      const int p = tid + NT * pi;
      uint4 pv = make_uint4(0xFFFFFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu);
      if (pi < ppc && p < npc) pv = *reinterpret_cast<const uint4*>(pinv + 8 * p);
      const uint32_t w[4] = {pv.x, pv.y, pv.z, pv.w};
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        uint32_t lo = (w[c] & 0xFFFFu) - cbase, hi = (w[c] >> 16) - cbase;
        lo = (pi < ppc && p < npc && lo < static_cast<uint32_t>(C)) ? lo : 0xFFFFu;
        hi = (pi < ppc && p < npc && hi < static_cast<uint32_t>(C)) ? hi : 0xFFFFu;
        dst[pi][c] = lo | (hi << 16);
      }
    }
    // Rows in batches of RB, double-buffered: the loads of batch b + 1 are
    // issued before batch b is written to LDS.
    constexpr int RB = 4;
    static_assert(R % RB == 0, "row batches");
    uint4 v[2][RB][PMAX];
    auto load_rows = [&](int r0, uint4 (&buf)[RB][PMAX]) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        const int64_t gr = row0 + r0 + rb;
        const bool rok = gr < M;
#pragma unroll
        for (int pi = 0; pi < PMAX; ++pi) {
          const int p = tid + NT * pi;
          const bool ok = rok && pi < ppc && p < npc;
          buf[rb][pi] = *reinterpret_cast<const uint4*>(X + (ok ? gr : 0) * ldx + (ok ? 8 * p : 0));
          if (!ok) buf[rb][pi] = make_uint4(0, 0, 0, 0);
        }
      }
    };
    load_rows(0, v[0]);
#pragma unroll
    for (int bt = 0; bt < R / RB; ++bt) {
      if (bt + 1 < R / RB) load_rows((bt + 1) * RB, v[(bt + 1) & 1]);
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        uint16_t* srow = sx + (bt * RB + rb) * XS;
#pragma unroll
        for (int pi = 0; pi < PMAX; ++pi) {
          const uint4 x4 = v[bt & 1][rb][pi];
          const uint32_t w[4] = {x4.x, x4.y, x4.z, x4.w};
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            const uint32_t lo = dst[pi][c] & 0xFFFFu, hi = dst[pi][c] >> 16;
            if (lo != 0xFFFFu) srow[lo] = static_cast<uint16_t>(w[c]);
            if (hi != 0xFFFFu) srow[hi] = static_cast<uint16_t>(w[c] >> 16);
          }
        }
      }
    }
    // A permutation gives every position of the chunk exactly one channel, so
    // every LDS element of the R rows is written (rows past M with zeros).
  } else {
    // The chunk's columns of each row go straight from global memory into
    // LDS (global_load_lds_dwordx4: lane l's 16 bytes land at the given LDS
    // address + 16 l), 1 KB (512 channels) per wave instruction, with no
    // registers in between, so every row of the tile is in flight at once.
    // Rows past M read row M - 1 (their results are not stored).
    constexpr int PARTS = C / 512;
    for (int j = wave; j < R * PARTS; j += WAVES) {
      const int r = j / PARTS, h = j % PARTS;
      const int64_t gr = row0 + r < M ? row0 + r : M - 1;
      const uint16_t* src = X + gr * ldx + cbase + 512 * h + 8 * lane;
      __builtin_amdgcn_global_load_lds((gmem_void*)src, (lds_void*)(sx + r * XS + 512 * h), 16, 0, 0);
    }
    __builtin_amdgcn_s_waitcnt(0);
  }
  __syncthreads();

  c4f y[NBW][4][RG];
  float amax[RG][4];
#pragma unroll
  for (int rg = 0; rg < RG; ++rg)
#pragma unroll
    for (int e = 0; e < 4; ++e) amax[rg][e] = 0.0f;
#pragma unroll
  for (int i = 0; i < NBW; ++i) {
    if (i + PF - 1 < NBW) load_b(i + PF - 1, bring[(i + PF - 1) % PF]);
    __builtin_amdgcn_sched_barrier(0);
    const c8h (&bf)[4][2] = bring[i % PF];
#pragma unroll
    for (int rg = 0; rg < RG; ++rg) {
      const uint16_t* ap = &sx[(rg * 16 + r16) * XS + (wb0 + i) * kCB + 8 * qq];
      const c8h a0 = *reinterpret_cast<const c8h*>(ap);
      const c8h a1 = *reinterpret_cast<const c8h*>(ap + 32);
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
  // Chunk maxima per row: across the 16 lanes of a row group, then the waves.
#pragma unroll
  for (int rg = 0; rg < RG; ++rg)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float m = amax[rg][e];
      m = fmaxf(m, rqd::lane_xor<1>(m));
      m = fmaxf(m, rqd::lane_xor<2>(m));
      m = fmaxf(m, rqd::lane_xor<4>(m));
      m = fmaxf(m, rqd::lane_xor<8>(m));
      if (r16 == 0) red[wave][rg * 16 + 4 * qq + e] = m;
    }
  __syncthreads();  // also: every wave's reads of sx are done (sx is reused for the codes)
  float* tslots = slots + static_cast<int64_t>(tile) * nq * R;  // [nq][R] of this tile
  if (tid < R) {
    float m = red[0][tid];
#pragma unroll
    for (int w = 1; w < WAVES; ++w) m = fmaxf(m, red[w][tid]);
    if (nq == 1) {
      red[0][tid] = m;
    } else {
      __hip_atomic_store(&tslots[q * R + tid], m, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  if (nq > 1) {
    // Thread t < nq R waits for partner t / R's maximum of row t % R (its own
    // chunk's included).
    for (int t = tid; t < nq * R; t += NT) {
      float v = __hip_atomic_load(&tslots[t], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      for (int it = 0; !(v >= 0.0f) && it < kPollLimit; ++it) {
        __builtin_amdgcn_s_sleep(2);
        v = __hip_atomic_load(&tslots[t], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      if (!(v >= 0.0f)) timed_out = 1;
    }
    __syncthreads();
    if (tid < R) {
      float m = 0.0f;
      for (int p = 0; p < nq; ++p)
        m = fmaxf(m, __hip_atomic_load(&tslots[p * R + tid], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
      red[0][tid] = m;
    }
  }
  __syncthreads();
  if (tid < R) {
    const float m = red[0][tid];
    const float a_z = m * s_t;
    const float delta = a_z / 7.0f;
    gscale[tid] = delta > 0.0f ? s_t / delta : 0.0f;
    if (q == 0 && row0 + tid < M) xs[row0 + tid] = timed_out ? __builtin_nanf("") : delta / s_t;
  }
  __syncthreads();

  // ---- Codes: 8 consecutive channels packed into a dword across lanes and
  // staged in LDS (the chunk's rows, C / 2 bytes each), then stored as 16-byte pieces.
  uint32_t* scodes = reinterpret_cast<uint32_t*>(sx);  // [R][C / 8] dwords
#pragma unroll
  for (int i = 0; i < NBW; ++i)
#pragma unroll
    for (int rg = 0; rg < RG; ++rg)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int row = rg * 16 + 4 * qq + e;
        const float g = gscale[row];
#pragma unroll
        for (int cb = 0; cb < 4; ++cb) {
          uint32_t c = __float_as_uint(fmaf(y[i][cb][rg][e], g, rqd::kRoundMagic)) & 0xFu;
          c |= __float_as_uint(rqd::lane_xor<1>(__uint_as_float(c))) << 4;
          c |= __float_as_uint(rqd::lane_xor<2>(__uint_as_float(c))) << 8;
          c |= __float_as_uint(rqd::lane_xor<4>(__uint_as_float(c))) << 16;
          if ((r16 & 7) == 0) scodes[row * (C / 8) + ((wb0 + i) * kCB + cb * 16 + r16) / 8] = c;
        }
      }
  __syncthreads();
  constexpr int CPR = C / 32;  // 16-byte code pieces per row of the chunk
  for (int p = tid; p < R * CPR; p += NT) {
    const int r = p / CPR, c16 = p % CPR;
    if (row0 + r >= M) continue;
    *reinterpret_cast<uint4*>(Xq + (row0 + r) * static_cast<int64_t>(K / 2) + cbase / 2 + 16 * c16) =
        *reinterpret_cast<const uint4*>(&scodes[r * (C / 8) + 4 * c16]);
  }
}

// Device workspace of the chunked kernel (the inverse permutation and the
// exchange slots), one per GPU, grown on demand and kept for the process.
struct CompWork {
  void* ptr = nullptr;
  size_t bytes = 0;
};
constexpr int kMaxDevices = 64;
CompWork g_comp_work[kMaxDevices];
std::mutex g_comp_mu;

int comp_workspace(size_t bytes, void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return OQ_ERR_HIP;
  std::lock_guard<std::mutex> lock(g_comp_mu);
  CompWork& w = g_comp_work[dev];
  if (w.bytes < bytes) {
    // hipFree waits for the device, so no launch still uses the old buffer.
    if (w.ptr && hipFree(w.ptr) != hipSuccess) return OQ_ERR_HIP;
    w.ptr = nullptr;
    w.bytes = 0;
    const size_t grow = bytes + bytes / 2;
    if (hipMalloc(&w.ptr, grow) != hipSuccess) {
      w.ptr = nullptr;
      return OQ_ERR_HIP;
    }
    w.bytes = grow;
  }
  *out = w.ptr;
  return OQ_OK;
}

template <int RG, int C, bool GATHER, int WAVES = 8, int PF = 2>
int launch_composite_x(const void* X, int64_t M, int64_t K, int64_t ldx, const int32_t* perm, const void* Rt,
                       float s, uint8_t* Xq, float* x_scale, hipStream_t stream) {
  constexpr int R = 16 * RG;
  const int64_t ntiles = (M + R - 1) / R;
  const int nq = static_cast<int>(K / C);
  if (ntiles > (int64_t{1} << 26)) return OQ_ERR_SHAPE;
  const size_t pinv_bytes = (static_cast<size_t>(K) * 2 + 255) / 256 * 256;
  const int64_t nslots = nq > 1 ? ntiles * nq * R : 0;
  void* ws = nullptr;
  int st = comp_workspace(pinv_bytes + static_cast<size_t>(nslots) * 4 + 256, &ws);
  if (st != OQ_OK) return st;
  uint16_t* pinv = static_cast<uint16_t*>(ws);
  float* slots = reinterpret_cast<float*>(static_cast<uint8_t*>(ws) + pinv_bytes);
  const int64_t nprep = std::max<int64_t>(GATHER ? K : 0, nslots);
  if (nprep > 0) {
    hipLaunchKernelGGL(comp_prep_kernel, dim3(static_cast<unsigned>((nprep + 255) / 256)), dim3(256), 0, stream,
                       GATHER ? perm : nullptr, static_cast<int>(K), pinv, slots, nslots);
    if ((st = launch_status()) != OQ_OK) return st;
  }
  const int64_t grid = (ntiles + 7) / 8 * 8 * nq;
  hipLaunchKernelGGL((rq_composite_x_kernel<RG, C, GATHER, WAVES, PF>), dim3(static_cast<unsigned>(grid)),
                     dim3(64 * WAVES), 0, stream, static_cast<const uint16_t*>(X), M, static_cast<int>(K), ldx,
                     pinv, static_cast<const uint16_t*>(Rt), s, Xq, x_scale, slots, nq,
                     static_cast<int>(ntiles));
  return launch_status();
}

// Chunk width: the widest of 4096 / 2048 / 1024 / 512 that divides K, at
// most `cap` (0: none; the two-pass kernel is used).  With the online
// permutation every chunk's workgroup reads whole rows, so 16-row tiles of the
// widest chunk (fewest re-reads) are best.  With P folded into the input a
// workgroup reads only its chunk's columns and the block matrices dominate
// the traffic from L2 (128 K / R bytes per row for R-row tiles), so 32-row
// tiles of at most 1024 channels (64 KB of LDS, two workgroups per CU) are
// best (measured at K = 4096 - 16384).
int comp_chunk(int64_t K, int cap) {
  for (int c : {4096, 2048, 1024, 512})
    if (c <= cap && K % c == 0) return c;
  return 0;
}

int launch_composite_chunked(bool gather, int C, const void* X, int64_t M, int64_t K, int64_t ldx,
                             const int32_t* perm, const void* Rt, float s, uint8_t* Xq, float* x_scale,
                             hipStream_t h) {
  if (gather) {
    switch (C) {
      case 4096: return launch_composite_x<1, 4096, true>(X, M, K, ldx, perm, Rt, s, Xq, x_scale, h);
      case 2048: return launch_composite_x<1, 2048, true>(X, M, K, ldx, perm, Rt, s, Xq, x_scale, h);
      case 1024: return launch_composite_x<1, 1024, true>(X, M, K, ldx, perm, Rt, s, Xq, x_scale, h);
      case 512: return launch_composite_x<1, 512, true>(X, M, K, ldx, perm, Rt, s, Xq, x_scale, h);
      default: return OQ_ERR_SHAPE;
    }
  }
  switch (C) {
    case 1024: return launch_composite_x<2, 1024, false>(X, M, K, ldx, perm, Rt, s, Xq, x_scale, h);
    case 512: return launch_composite_x<2, 512, false>(X, M, K, ldx, perm, Rt, s, Xq, x_scale, h);
    default: return OQ_ERR_SHAPE;
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
    // K = 4096 with many rows: 1024-channel chunks of 32-row tiles beat one
    // workgroup per 16 whole rows (78 vs 120 us at M = 16384).
    if (K == 4096 && M > 1024)
      return oq::launch_composite_chunked(false, 1024, X, M, K, ldx, perm, Rt, s, Xq, x_scale, h);
    if (K <= 4096) return oq::launch_composite1<1, 4096, false>(X, M, K, ldx, perm, Rt, s, Xq, x_scale, h);
    if (const int c = oq::comp_chunk(K, 1024))
      return oq::launch_composite_chunked(false, c, X, M, K, ldx, perm, Rt, s, Xq, x_scale, h);
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
  if (const int c = oq::comp_chunk(K, 4096))
    return oq::launch_composite_chunked(true, c, X, M, K, ldx, perm, Rt, s, Xq, x_scale, h);
  if (K <= 8192) return oq::launch_composite<4, 8192>(X, M, K, ldx, perm, Rt, s, Xq, x_scale, h);
  return oq::launch_composite<2, 16384>(X, M, K, ldx, perm, Rt, s, Xq, x_scale, h);
}
