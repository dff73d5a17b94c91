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
// Two kernels.  M > 64: LDS-staged tiles of 256 x 256, 128 x 128 or 64 x 64
// outputs on v_mfma_i32_32x32x32_i8, the largest tile that still gives every
// CU a workgroup (details at gemm_big_kernel).  M <= 64 (and token codes in
// the 16-row tiled layout): a weight-streaming kernel on
// v_mfma_i32_16x16x64_i8 with the operands loaded straight into registers
// (details at gemm_small_kernel).  8-bit token codes (W4A8) use both with
// the A operand loaded as bytes.
#include <utility>

#include "common.h"

namespace oq {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int BK = 64;  // K granularity in codes (one MFMA k step of 64 codes = 32 packed bytes)

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t b = __float_as_uint(f);
  b += 0x7FFFu + ((b >> 16) & 1u);
  return static_cast<uint16_t>(b >> 16);
}

// ---------------------------------------------------------------------------
// Products with M > 64 (prefill / batched shapes).  A workgroup of WM x WN
// waves owns a (32 TM WM) x (32 TN WN) output tile; each wave a (32 TM) x
// (32 TN) tile of v_mfma_i32_32x32x32_i8 blocks.  Two instances: 256 x 256
// (8 waves of 128 x 64, one workgroup per CU) for large problems and 128 x
// 128 (4 waves of 64 x 64, two workgroups per CU) when the large tiles would
// not fill the CUs.  Each LDS stage covers 128 codes of K: the packed codes
// are loaded from global memory (32 bytes per thread and row), widened once
// to int8 (16 * code) on the way into LDS, and read back as 16-byte fragments
// that feed the matrix cores directly; the fragments of the next 32-code
// sub-step are read while the current one is multiplied.  LDS rows are
// padded to 144 bytes (36 dwords: 16-byte reads and writes of 8 consecutive
// rows touch distinct bank groups); two LDS buffers.  Global loads run NS
// stages ahead through a ring of NS register stages (three, or twelve for
// the 64 x 64 tile at deep K) and each stage is stored to LDS after the
// MFMAs of the previous one; rows past M (N) and steps past the last read
// clamped addresses, so the loads are branch-free and the compiler counts
// them exactly.  fp16 / bf16 results are staged through the freed LDS and
// written as 16-byte row pieces.  Tiles are visited
// XCD-major: consecutive workgroup ids go to different XCDs, so ids are
// remapped so that each XCD works on a compact group of tiles (shared A rows /
// B columns stay in that XCD's L2).
// ---------------------------------------------------------------------------

constexpr int BIG_KSTAGE = 128;    // codes per LDS stage (64 packed bytes per row in global memory)
constexpr int BIG8_STRIDE = 144;   // int8 bytes per LDS row (128 + 16 pad)


__device__ __forceinline__ v4i widen16_u2(uint2 p) {
  const uint32_t m = 0xF0F0F0F0u;
  v4i r;
  r[0] = static_cast<int>((p.x << 4) & m);
  r[1] = static_cast<int>(p.x & m);
  r[2] = static_cast<int>((p.y << 4) & m);
  r[3] = static_cast<int>(p.y & m);
  return r;
}

// 16 bytes of 8-bit codes (natural channel order) in the order that
// widen16_u2 gives packed codes: within each group of 8 channels the even
// channels first, [0 2 4 6 1 3 5 7], so that a W4A8 A operand meets the
// widened weight fragment channel for channel.
__device__ __forceinline__ v4i order16_i8(uint4 p) {
  v4i r;
  r[0] = static_cast<int>(__builtin_amdgcn_perm(p.y, p.x, 0x06040200u));
  r[1] = static_cast<int>(__builtin_amdgcn_perm(p.y, p.x, 0x07050301u));
  r[2] = static_cast<int>(__builtin_amdgcn_perm(p.w, p.z, 0x06040200u));
  r[3] = static_cast<int>(__builtin_amdgcn_perm(p.w, p.z, 0x07050301u));
  return r;
}

// f(std::integral_constant<int, i>) for i = 0 .. N-1, fully unrolled.
template <typename F, int... I>
__device__ __forceinline__ void static_for_seq(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_seq(f, std::make_integer_sequence<int, N>{});
}

// Map a linear workgroup id to an output tile (tm, tn): the grid is cut into
// 8 contiguous chunks, one per XCD (hardware dispatches id i to XCD i % 8),
// and each chunk is walked in groups of GM tile rows.
__device__ __forceinline__ void big_tile(int id, int tiles_m, int tiles_n, int* tm, int* tn) {
  const int total = tiles_m * tiles_n;
  int lin = id;
  if (total % 8 == 0) {
    const int per = total / 8;
    lin = (id % 8) * per + id / 8;
  }
  constexpr int GM = 4;
  const int group = lin / (GM * tiles_n);
  const int first_m = group * GM;
  const int gsize = min(GM, tiles_m - first_m);
  const int in = lin - group * GM * tiles_n;
  *tm = first_m + in % gsize;
  *tn = in / gsize;
}

// A8: the token operand holds 8-bit codes (W4A8), one byte each, loaded 64
// bytes per thread and row per stage and reordered (not widened) into LDS;
// the products are then 16 * q * wq and the accumulator is shifted by 4.
template <int EPI, int WM, int WN, int TM, int TN, bool A8, int NS, int KG>
__global__ __launch_bounds__(64 * WM * WN * KG, (512 / (64 * WM * WN * KG) > 0 ? 512 / (64 * WM * WN * KG) : 1))
void gemm_big_kernel(GemmArgs a) {
  static_assert(NS >= 2, "at least two register stages");
  // KG groups of WM x WN waves; in each group every wave owns a (32 TM) x
  // (32 TN) tile of v_mfma_i32_32x32x32_i8 blocks.  Group g multiplies the
  // stages g, g + KG, g + 2 KG, ... of K through its own LDS buffers; the
  // groups' accumulators are summed through LDS before the epilogue (exact
  // integer sums, so any KG gives the same result bit for bit).
  constexpr int NTG = 64 * WM * WN;         // threads per group
  constexpr int NT = NTG * KG;              // threads
  constexpr int BM = 32 * TM * WM, BN = 32 * TN * WN;
  // Rows each thread loads per stage (two 32-byte pieces per row).  SPLIT:
  // fewer row pieces than threads (the 8-wave 128 x 128 tile), so the first
  // 2 BM threads load one piece of A each and the rest one piece of B.
  constexpr bool SPLIT = 2 * BM < NTG;
  constexpr int PA = SPLIT ? 0 : 2 * BM / NTG, PB = SPLIT ? 0 : 2 * BN / NTG;
  constexpr int PAa = PA > 0 ? PA : 1, PBa = PB > 0 ? PB : 1;  // array extents
  static_assert(SPLIT ? (2 * (BM + BN) == NTG && !A8)
                      : (PA >= 1 && PB >= 1 && 2 * BM % NTG == 0 && 2 * BN % NTG == 0),
                "load split");
  // Per group two LDS buffers per operand; after the K loop the same memory
  // holds the other groups' accumulators and the 2-byte output tile of the
  // staged epilogue.
  constexpr int GBYTES = 2 * (BM + BN) * BIG8_STRIDE;
  __shared__ __attribute__((aligned(16))) uint8_t smem[KG * GBYTES];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int grp = tid / NTG, tg = tid % NTG;
  const int wave = tg >> 6;  // wave within the group
  const int wm = wave / WN, wn = wave % WN;  // rows wm * 32 TM, columns wn * 32 TN
  uint8_t (*sA)[BM * BIG8_STRIDE] = reinterpret_cast<uint8_t (*)[BM * BIG8_STRIDE]>(smem + grp * GBYTES);
  uint8_t (*sB)[BN * BIG8_STRIDE] =
      reinterpret_cast<uint8_t (*)[BN * BIG8_STRIDE]>(smem + grp * GBYTES + 2 * BM * BIG8_STRIDE);
  const int tiles_m = static_cast<int>((a.M + BM - 1) / BM);
  const int tiles_n = static_cast<int>((a.N + BN - 1) / BN);
  // Split K (a.splitk > 1): workgroup id = ks * tiles + tile; split ks takes
  // stages [ks * sps, (ks + 1) * sps) of K.
  const int ntile = tiles_m * tiles_n;
  const int tile_id = static_cast<int>(blockIdx.x) % ntile, ks = static_cast<int>(blockIdx.x) / ntile;
  int tm, tn;
  big_tile(tile_id, tiles_m, tiles_n, &tm, &tn);
  const int64_t m0 = static_cast<int64_t>(tm) * BM;
  const int64_t n0 = static_cast<int64_t>(tn) * BN;
  const int64_t Kb = a.K / 2;
  constexpr int AW = A8 ? 2 : 1;  // A bytes per packed B byte
  const int64_t Ka = Kb * AW;
  const int nk_all = static_cast<int>((a.K + BIG_KSTAGE - 1) / BIG_KSTAGE);  // stages (the last may be half)
  const int sps = (nk_all + a.splitk - 1) / a.splitk;                         // stages per split
  const int s0 = ks * sps;                                                     // this split's first stage
  const int nk = min(nk_all - s0, sps);                                        // ... and its stage count
  const int h0 = 2 * s0;                                                       // its first 64-code half
  const int nk64 = min(static_cast<int>(a.K / 64), 2 * (s0 + sps)) - h0;       // ... and its half count

  // Global -> LDS: a stage is BM (A) and BN (B) rows x 64 packed bytes; a
  // thread loads 32 packed bytes (two 16-byte pieces) of rows tg/2 + r NTG/2.
  // Local stage j of group grp is stage KG j + grp of K.  A half stage past K,
  // and a stage past the end, read clamped addresses; their sub-steps past the
  // codes multiply zero A fragments (OQ_COMPUTE).
  const int lr = tg >> 1, lh = tg & 1;
  const int njl = (nk + KG - 1) / KG;  // local stages (the same count in every group)
  const uint8_t* gA[PAa];
  const uint8_t* gB[PBa];
#pragma unroll
  for (int r = 0; r < PA; ++r) gA[r] = a.A + min<int64_t>(m0 + lr + r * (NTG / 2), a.M - 1) * Ka + lh * 32 * AW;
#pragma unroll
  for (int r = 0; r < PB; ++r) gB[r] = a.B + min<int64_t>(n0 + lr + r * (NTG / 2), a.N - 1) * Kb + lh * 32;
  // SPLIT: this thread's operand, its row there and its source row.
  const bool s_isA = tg < 2 * BM;
  const int s_row = (s_isA ? tg : tg - 2 * BM) >> 1;
  const uint8_t* gS = s_isA ? a.A + min<int64_t>(m0 + s_row, a.M - 1) * Ka + lh * 32
                            : a.B + min<int64_t>(n0 + s_row, a.N - 1) * Kb + lh * 32;
  // NS register stages, indexed only by constants (they stay in VGPRs).
  uint4 ra[NS][2 * AW * PAa], rb[NS][2 * PBa], rs[NS][2];
#define OQ_GLOAD(KS, S)                                                                \
  {                                                                                    \
    const int h_ = h0 + min(2 * (KG * (KS) + grp) + lh, nk64 - 1);                      \
    const int64_t off_ = static_cast<int64_t>(h_) * 32 - lh * 32;                      \
    _Pragma("unroll") for (int r_ = 0; r_ < PA; ++r_)                                  \
    _Pragma("unroll") for (int c_ = 0; c_ < 2 * AW; ++c_)                              \
      ra[S][2 * AW * r_ + c_] = *reinterpret_cast<const uint4*>(gA[r_] + AW * off_ + 16 * c_); \
    _Pragma("unroll") for (int r_ = 0; r_ < PB; ++r_) {                          \
      rb[S][2 * r_] = *reinterpret_cast<const uint4*>(gB[r_] + off_);            \
      rb[S][2 * r_ + 1] = *reinterpret_cast<const uint4*>(gB[r_] + off_ + 16);   \
    }                                                                            \
    if constexpr (SPLIT) {                                                       \
      rs[S][0] = *reinterpret_cast<const uint4*>(gS + off_);                     \
      rs[S][1] = *reinterpret_cast<const uint4*>(gS + off_ + 16);                \
    }                                                                            \
  }
// Widen 16 packed bytes to 32 int8 (16 * code) and store them: the same
// within-8-byte order for A and B, so the k order of every 16-code fragment
// agrees between the operands.
#define OQ_ST32(P, V)                                                   \
  {                                                                     \
    v4i* q_ = reinterpret_cast<v4i*>(P);                                \
    q_[0] = widen16_u2(make_uint2((V).x, (V).y));                       \
    q_[1] = widen16_u2(make_uint2((V).z, (V).w));                       \
  }
#define OQ_LSTORE(BUF, S)                                                                          \
  {                                                                                                \
    _Pragma("unroll") for (int r_ = 0; r_ < PA; ++r_) {                                            \
      if constexpr (A8) {                                                                          \
        _Pragma("unroll") for (int c_ = 0; c_ < 4; ++c_)                                           \
          *reinterpret_cast<v4i*>(&sA[(BUF)][(lr + r_ * (NTG / 2)) * BIG8_STRIDE + lh * 64 + 16 * c_]) = \
              order16_i8(ra[S][4 * r_ + c_]);                                                      \
      } else {                                                                                     \
        OQ_ST32(&sA[(BUF)][(lr + r_ * (NTG / 2)) * BIG8_STRIDE + lh * 64], ra[S][2 * r_])          \
        OQ_ST32(&sA[(BUF)][(lr + r_ * (NTG / 2)) * BIG8_STRIDE + lh * 64 + 32], ra[S][2 * r_ + 1]) \
      }                                                                                            \
    }                                                                                              \
    _Pragma("unroll") for (int r_ = 0; r_ < PB; ++r_) {                                            \
      OQ_ST32(&sB[(BUF)][(lr + r_ * (NTG / 2)) * BIG8_STRIDE + lh * 64], rb[S][2 * r_])            \
      OQ_ST32(&sB[(BUF)][(lr + r_ * (NTG / 2)) * BIG8_STRIDE + lh * 64 + 32], rb[S][2 * r_ + 1])   \
    }                                                                                              \
    if constexpr (SPLIT) {                                                                         \
      uint8_t* d_ = s_isA ? &sA[(BUF)][s_row * BIG8_STRIDE + lh * 64]                              \
                          : &sB[(BUF)][s_row * BIG8_STRIDE + lh * 64];                             \
      OQ_ST32(d_, rs[S][0])                                                                        \
      OQ_ST32(d_ + 32, rs[S][1])                                                                   \
    }                                                                                              \
  }

  v16i acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0;

  const int frow = lane & 31;
  const int fofs = 16 * (lane >> 5);  // 16 int8 codes of a 32-code sub-step
  const uint8_t* pA = &sA[0][(wm * 32 * TM + frow) * BIG8_STRIDE + fofs];
  const uint8_t* pB = &sB[0][(wn * 32 * TN + frow) * BIG8_STRIDE + fofs];
  constexpr int ABUF = BM * BIG8_STRIDE, BBUF = BN * BIG8_STRIDE;
// The int8 fragments of sub-step sub + 1 are read from LDS while sub-step
// sub is multiplied (two register sets).  All four sub-steps of every stage
// are issued without a branch: a sub-step past the stage's codes (the second
// half of a final half stage, a stage past the end of K) multiplies a zero A
// fragment and adds exactly 0.  (A branch on the per-lane stage condition may
// be compiled as an EXEC mask alone, and an MFMA still accumulates with EXEC
// = 0.)  The fragment reads stay inside the stage's LDS rows.
#define OQ_COMPUTE(BUF, NSUB)                                                                               \
  {                                                                                                         \
    const int boa_ = (BUF) * ABUF, bob_ = (BUF) * BBUF;                                                      \
    const int nsub_ = (NSUB);                                                                               \
    v4i fa_[2][TM], fb_[2][TN];                                                                             \
    _Pragma("unroll") for (int i = 0; i < TM; ++i)                                                           \
      fa_[0][i] = *reinterpret_cast<const v4i*>(pA + boa_ + i * 32 * BIG8_STRIDE);                          \
    _Pragma("unroll") for (int j = 0; j < TN; ++j)                                                           \
      fb_[0][j] = *reinterpret_cast<const v4i*>(pB + bob_ + j * 32 * BIG8_STRIDE);                          \
    _Pragma("unroll") for (int sub = 0; sub < 4; ++sub) {                                                   \
      const int cur_ = sub & 1;                                                                             \
      if (sub + 1 < 4) {                                                                                    \
        _Pragma("unroll") for (int i = 0; i < TM; ++i)                                                       \
          fa_[cur_ ^ 1][i] = *reinterpret_cast<const v4i*>(pA + boa_ + i * 32 * BIG8_STRIDE + (sub + 1) * 32); \
        _Pragma("unroll") for (int j = 0; j < TN; ++j)                                                       \
          fb_[cur_ ^ 1][j] = *reinterpret_cast<const v4i*>(pB + bob_ + j * 32 * BIG8_STRIDE + (sub + 1) * 32); \
      }                                                                                                     \
      const bool on_ = sub < nsub_;                                                                         \
      __builtin_amdgcn_sched_barrier(0);                                                                    \
      _Pragma("unroll") for (int i = 0; i < TM; ++i) {                                                       \
        v4i a_;                                                                                             \
        _Pragma("unroll") for (int c_ = 0; c_ < 4; ++c_) a_[c_] = on_ ? fa_[cur_][i][c_] : 0;              \
        _Pragma("unroll") for (int j = 0; j < TN; ++j)                                                       \
          acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a_, fb_[cur_][j], acc[i][j], 0, 0, 0);          \
      }                                                                                                     \
      __builtin_amdgcn_sched_barrier(0);                                                                    \
    }                                                                                                       \
  }
  // Sub-steps of 32 codes that hold codes in local stage ks: 4, 2 for a final
  // half stage, 0 past the end of K (the rest multiply zero A fragments).
#define OQ_NSUB(KS) ((2 * (KG * (KS) + grp) + 2 <= nk64) ? 4 : (2 * (KG * (KS) + grp) < nk64 ? 2 : 0))

  // Global loads run NS - 1 stages ahead of the LDS stage being multiplied:
  // at the top of stage kt, ring slot (kt + i) % NS holds stage kt + i for
  // i = 1 .. NS - 1 and stage kt is in LDS buffer kt & 1.  Stage kt issues the
  // load of stage kt + NS into the slot it freed, runs its MFMAs, stores stage
  // kt + 1 into the other LDS buffer and synchronizes.  The loop is unrolled
  // by NS so that every ring index is a constant.
  static_for<NS>([&](auto S_) {
    constexpr int SV = decltype(S_)::value;
    OQ_GLOAD(SV, SV)
  });
  OQ_LSTORE(0, 0)
  __syncthreads();
  int kt = 0;
  for (; kt + NS <= njl; kt += NS) {
    static_for<NS>([&](auto S_) {
      constexpr int SV = decltype(S_)::value;
      constexpr int SN = (SV + 1) % NS;
      OQ_GLOAD(kt + SV + NS, SV)
      OQ_COMPUTE((kt + SV) & 1, OQ_NSUB(kt + SV))
      OQ_LSTORE((kt + SV + 1) & 1, SN)
      __syncthreads();
    });
  }
  // Fewer than NS stages left: stage kt is in LDS, slot i holds stage kt + i.
  static_for<NS>([&](auto S_) {
    constexpr int SV = decltype(S_)::value;
    constexpr int SN = (SV + 1) % NS;
    if (kt + SV < njl) {
      OQ_COMPUTE((kt + SV) & 1, OQ_NSUB(kt + SV))
      if (kt + SV + 1 < njl) OQ_LSTORE((kt + SV + 1) & 1, SN)
      __syncthreads();
    }
  });
#undef OQ_NSUB
  if constexpr (KG > 1) {
    // Groups 1 .. KG-1 leave their accumulators in their own (now unused)
    // LDS buffers, lane-major; group 0 adds them in group order.
    __syncthreads();
    constexpr int WORDS = WM * WN * TM * TN * 16 * 64;  // one group's accumulators
    static_assert(WORDS * 4 <= GBYTES, "accumulators exceed a group's buffers");
    if (grp > 0) {
      int32_t* red = reinterpret_cast<int32_t*>(smem + grp * GBYTES);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int e = 0; e < 16; ++e) red[((wave * TM + i) * TN + j) * 1024 + e * 64 + lane] = acc[i][j][e];
    }
    __syncthreads();
    if (grp == 0) {
#pragma unroll
      for (int gg = 1; gg < KG; ++gg) {
        const int32_t* red = reinterpret_cast<const int32_t*>(smem + gg * GBYTES);
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[i][j][e] += red[((wave * TM + i) * TN + j) * 1024 + e * 64 + lane];
      }
    }
  }
#undef OQ_GLOAD
#undef OQ_ST32
#undef OQ_LSTORE
#undef OQ_COMPUTE
  if (a.splitk > 1) {
    // Every split publishes its exact partial (group 0's accumulators,
    // lane-major) and takes a ticket; the last arrival adds the others' and
    // runs the epilogue, the rest leave.  No workgroup waits for another.
    // The partials move through device-scope atomic stores and loads (they
    // bypass the XCD-local caches) and the ticket is taken after every store
    // of the workgroup is acknowledged, so no cache-wide write-back or
    // invalidation is needed (those would evict the other workgroups' A / B
    // lines from the L2 mid-loop).
    constexpr int WORDS = WM * WN * TM * TN * 16 * 64;
    __shared__ int s_last;
    int32_t* mine = a.part + (static_cast<int64_t>(tile_id) * a.splitk + ks) * WORDS;
    if (grp == 0) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int e = 0; e < 16; ++e)
            __hip_atomic_store(&mine[((wave * TM + i) * TN + j) * 1024 + e * 64 + lane], acc[i][j][e],
                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __builtin_amdgcn_s_waitcnt(0);  // the stores are acknowledged
    __syncthreads();
    if (tid == 0)
      s_last = __hip_atomic_fetch_add(a.tickets + tile_id, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
               a.splitk - 1;
    __syncthreads();
    if (!s_last) return;
    if (grp == 0) {
      for (int k2 = 0; k2 < a.splitk; ++k2) {
        if (k2 == ks) continue;
        const int32_t* other = a.part + (static_cast<int64_t>(tile_id) * a.splitk + k2) * WORDS;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e)
              acc[i][j][e] += __hip_atomic_load(&other[((wave * TM + i) * TN + j) * 1024 + e * 64 + lane],
                                                __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
    if (tid == 0) __hip_atomic_store(a.tickets + tile_id, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }

  // Epilogue (32 x 32 layout: element e of lane l is row 8*(e/4) + 4*(l/32) + e%4, column l%32).
  // Each lane's rows come in runs of four consecutive rows: their token scales
  // are read as one float4 per run (rows past M read as 0).  fp16 / bf16
  // outputs are staged through LDS as a 256 x 256 tile and written as
  // 16-byte row pieces (whole cache lines); int32 and residual outputs are
  // written from the accumulator layout directly.
  const int col_in = lane & 31;
  const int row_grp = 4 * (lane >> 5);
  constexpr bool STAGED = EPI == EPI_F16 || EPI == EPI_BF16 || EPI == EPI_GELU_F16;
  constexpr int TP = BN + 8;  // halves per staged row
  static_assert(!STAGED || BM * TP * 2 <= 2 * (BM + BN) * BIG8_STRIDE, "staged tile exceeds LDS");
  uint16_t* tile = reinterpret_cast<uint16_t*>(smem);
  if (STAGED) __syncthreads();  // every fragment read of the last stage is done
  // Per-column operands, then per 32-row block: every load of the block
  // (token scales, and for the residual epilogue the old residual values) is
  // issued from clamped addresses before the block's first store, so that the
  // in-order memory counter never makes a load wait behind a store.
  float wsc[TN], bias[TN], gate[TN];
  int64_t gcs[TN];
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    gcs[j] = n0 + wn * 32 * TN + j * 32 + col_in;
    const int64_t gcc = gcs[j] < a.N ? gcs[j] : a.N - 1;
    wsc[j] = 0.0f;
    bias[j] = 0.0f;
    gate[j] = 1.0f;
    if (EPI != EPI_I32) {
      wsc[j] = a.ws[gcc];
      if (a.bias) bias[j] = static_cast<float>(__builtin_bit_cast(_Float16, a.bias[gcc]));
      if (EPI == EPI_RESID_F32 && a.gate) gate[j] = static_cast<float>(__builtin_bit_cast(_Float16, a.gate[gcc]));
    }
  }
  // (Only group 0 holds the summed accumulators.)
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    if (grp != 0) break;
    float xr[4][4];
    float rold[4][TN][4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int64_t r0 = m0 + wm * 32 * TM + i * 32 + 8 * q + row_grp;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int64_t gr = r0 + u < a.M ? r0 + u : a.M - 1;
        xr[q][u] = EPI != EPI_I32 ? a.xs[gr] : 0.0f;
        if (EPI == EPI_RESID_F32) {
#pragma unroll
          for (int j = 0; j < TN; ++j) {
            const int64_t gcc = gcs[j] < a.N ? gcs[j] : a.N - 1;
            rold[q][j][u] = static_cast<const float*>(a.C)[gr * a.ldc + gcc];
          }
        }
      }
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int lr0 = wm * 32 * TM + i * 32 + 8 * q + row_grp;  // row within the tile
      const int64_t r0 = m0 + lr0;
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int64_t gc = gcs[j];
        if (STAGED) {
          // Rows / columns past the edge are staged but not written back.
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const float y = static_cast<float>(acc[i][j][4 * q + u] >> (A8 ? 4 : 8)) * xr[q][u] * wsc[j] + bias[j];
            uint16_t hv;
            if constexpr (EPI == EPI_F16) {
              hv = __builtin_bit_cast(uint16_t, static_cast<_Float16>(y));
            } else if constexpr (EPI == EPI_GELU_F16) {
              hv = __builtin_bit_cast(
                  uint16_t, static_cast<_Float16>(gelu_tanh(static_cast<float>(static_cast<_Float16>(y)))));
            } else {
              hv = f32_to_bf16_rne(y);
            }
            tile[(lr0 + u) * TP + wn * 32 * TN + j * 32 + col_in] = hv;
          }
          continue;
        }
        if (gc >= a.N) continue;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int64_t gr = r0 + u;
          if (gr >= a.M) continue;
          const int v = acc[i][j][4 * q + u] >> (A8 ? 4 : 8);
          const int64_t off = gr * a.ldc + gc;
          if (EPI == EPI_I32) {
            static_cast<int32_t*>(a.C)[off] = v;
          } else {
            const float y = static_cast<float>(v) * xr[q][u] * wsc[j] + bias[j];
            static_cast<float*>(a.C)[off] = fmaf(gate[j], y, rold[q][j][u]);
          }
        }
      }
    }
  }
  if (STAGED) {
    static_assert((BM * BN / 8) % NT == 0, "output pieces per thread");
    __syncthreads();
    // BM rows x BN/8 pieces of 8 outputs; thread t writes pieces t + NT c.
    uint16_t* C = static_cast<uint16_t*>(a.C);
#pragma unroll
    for (int c = 0; c < (BM * BN / 8) / NT; ++c) {
      const int id = tid + NT * c;
      const int lr = id / (BN / 8), pc = (id % (BN / 8)) * 8;
      const int64_t gr = m0 + lr, gc = n0 + pc;
      if (gr >= a.M || gc >= a.N) continue;
      const uint4 v = *reinterpret_cast<const uint4*>(&tile[lr * TP + pc]);
      if (gc + 8 <= a.N) {
        *reinterpret_cast<uint4*>(C + gr * a.ldc + gc) = v;  // ldc % 8 == 0: 16-byte aligned
      } else {
        const uint16_t h[8] = {static_cast<uint16_t>(v.x), static_cast<uint16_t>(v.x >> 16),
                               static_cast<uint16_t>(v.y), static_cast<uint16_t>(v.y >> 16),
                               static_cast<uint16_t>(v.z), static_cast<uint16_t>(v.z >> 16),
                               static_cast<uint16_t>(v.w), static_cast<uint16_t>(v.w >> 16)};
        for (int e = 0; e < 8 && gc + e < a.N; ++e) C[gr * a.ldc + gc + e] = h[e];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Small-M product (the DiT's 50 action tokens, decode): weight-bandwidth and
// latency bound, so the weight is spread over many small workgroups.  A
// workgroup owns 16 MB rows x 16 NB columns of the output and all of K; its
// WAVES waves take contiguous ranges of 128-code units (64 packed bytes per
// row).  Every operand fragment is one 16-byte load per lane that feeds two
// v_mfma_i32_16x16x64_i8 steps (the two 8-byte halves, widened to int8 in
// registers); all of a wave's loads of UB units are issued before the first
// MFMA.  A comes either from the 16-row tiled layout -- one load is 1024
// contiguous bytes, 8 whole cache lines -- or from [M][K/2] rows (16 rows x
// 64 bytes per load).  The token codes are re-read by every workgroup, so the
// tiled form is what the DiT's fused producers write.  K % 128 == 64 (row
// layout only) ends with one 64-code step in 8-byte pieces on the last wave.
// The waves' partial accumulators are summed through LDS before the shared
// epilogue.
// ---------------------------------------------------------------------------

// Epilogue of one output from the exact accumulator; the per-row / per-column
// operands are passed in (loaded early by the caller).
template <int EPI>
__device__ __forceinline__ void store_out(const GemmArgs& a, int64_t off, int v, float xs, float ws, float bias,
                                          float gate, float resid) {
  if (EPI == EPI_I32) {
    static_cast<int32_t*>(a.C)[off] = v;
    return;
  }
  const float y = static_cast<float>(v) * xs * ws + bias;
  if (EPI == EPI_F16) {
    static_cast<_Float16*>(a.C)[off] = static_cast<_Float16>(y);
  } else if (EPI == EPI_GELU_F16) {
    static_cast<_Float16*>(a.C)[off] =
        static_cast<_Float16>(gelu_tanh(static_cast<float>(static_cast<_Float16>(y))));
  } else if (EPI == EPI_BF16) {
    static_cast<uint16_t*>(a.C)[off] = f32_to_bf16_rne(y);
  } else {
    static_cast<float*>(a.C)[off] = fmaf(gate, y, resid);
  }
}

// A8 (row layout only): 8-bit token codes, 32 bytes per lane and unit,
// reordered in registers; the accumulator is shifted by 4.
template <int EPI, int NB, int WAVES, int MB, int UB, bool TILED, bool A8 = false>
__global__ __launch_bounds__(64 * WAVES) void gemm_small_kernel(GemmArgs a) {
  static_assert(!(A8 && TILED), "8-bit token codes use the row layout");
  constexpr int BNs = 16 * NB, ROWS = 16 * MB, NOUT = ROWS * BNs, NT = 64 * WAVES;
  constexpr int OPT = (NOUT + NT - 1) / NT;  // outputs per thread
  static_assert(NT % BNs == 0, "a thread keeps one output column");
  __shared__ int red[WAVES][NOUT];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // scalar: the unit range bounds MFMA loops
  const int64_t n0 = static_cast<int64_t>(blockIdx.x) * BNs;
  const int64_t m0 = static_cast<int64_t>(blockIdx.y) * ROWS;
  const int64_t Kb = a.K / 2;
  const int nu = static_cast<int>(a.K / 128);
  const int ubeg = (nu * wave) / WAVES, uend = (nu * (wave + 1)) / WAVES;

  // Row-block bases: tiled -> block (m0 / 16 + rb) at unit 0 plus this lane's
  // 16 bytes; rows -> row m0 + 16 rb + lane % 16 at byte 0.  Out-of-range
  // blocks / rows read a clamped valid address; their fragments are replaced
  // by zeros where they are used.  Every load is unconditional, so the
  // compiler counts them exactly and each MFMA waits only for its own
  // operands.
  const uint8_t* abase[MB];
  bool aok[MB];
#pragma unroll
  for (int rb = 0; rb < MB; ++rb) {
    if (TILED) {
      const int64_t blk = m0 / 16 + rb;
      aok[rb] = blk * 16 < a.M;
      abase[rb] = a.A + (aok[rb] ? blk : 0) * nu * 1024 + lane * 16;
    } else {
      const int64_t r = m0 + rb * 16 + (lane & 15);
      aok[rb] = r < a.M;
      abase[rb] = a.A + (aok[rb] ? r : 0) * Kb * (A8 ? 2 : 1);
    }
  }
  const uint8_t* bbase[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) bbase[nb] = a.B + min<int64_t>(n0 + nb * 16 + (lane & 15), a.N - 1) * Kb;
  const int piece = 16 * (lane >> 4);  // this lane's 16 bytes of a 64-byte unit (row layout)

  // Fragments of UB units starting at u0 (a unit past uend reads unit uend - 1
  // or 0 again; its MFMAs are skipped).
  constexpr int AH = A8 ? 2 : 1;  // 16-byte A loads per unit and row block
  uint4 fa[UB][MB][AH], fb[UB][NB];
  auto load_units = [&](int u0) {
#pragma unroll
    for (int u = 0; u < UB; ++u) {
      const int uu = u0 + u < uend ? u0 + u : max(uend - 1, 0);
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) fb[u][nb] = *reinterpret_cast<const uint4*>(bbase[nb] + uu * 64 + piece);
#pragma unroll
      for (int rb = 0; rb < MB; ++rb)
#pragma unroll
        for (int c = 0; c < AH; ++c)
          fa[u][rb][c] = *reinterpret_cast<const uint4*>(
              TILED ? abase[rb] + static_cast<int64_t>(uu) * 1024
                    : abase[rb] + uu * 64 * AH + piece * AH + 16 * c);
    }
  };
  // The first units' loads go out before anything else.
  load_units(ubeg);

  // Epilogue operands of this thread's outputs (row (tid + u NT) / BNs,
  // column tid % BNs), loaded while the fragments are in flight, from clamped
  // addresses (the values of outputs that are not stored do not matter).
  const int ecol = tid % BNs;
  const int64_t egc = n0 + ecol;
  const bool ecol_ok = egc < a.N;
  const int64_t egc_c = ecol_ok ? egc : 0;
  float e_ws = 0.0f, e_bias = 0.0f, e_gate = 1.0f;
  float e_xs[OPT], e_res[OPT];
  if (EPI != EPI_I32) {
    e_ws = a.ws[egc_c];
    if (a.bias) e_bias = static_cast<float>(__builtin_bit_cast(_Float16, a.bias[egc_c]));
    if (EPI == EPI_RESID_F32 && a.gate) e_gate = static_cast<float>(__builtin_bit_cast(_Float16, a.gate[egc_c]));
  }
#pragma unroll
  for (int u = 0; u < OPT; ++u) {
    const int64_t gr = m0 + (tid + u * NT) / BNs;
    const int64_t gr_c = gr < a.M ? gr : 0;
    e_xs[u] = 0.0f;
    e_res[u] = 0.0f;
    if (EPI != EPI_I32) {
      e_xs[u] = a.xs[gr_c];
      if (EPI == EPI_RESID_F32) e_res[u] = static_cast<const float*>(a.C)[gr_c * a.ldc + egc_c];
    }
  }

  v4i acc[MB][NB];
#pragma unroll
  for (int rb = 0; rb < MB; ++rb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[rb][nb] = v4i{0, 0, 0, 0};
  auto mfma_units = [&](int u0) {
#pragma unroll
    for (int u = 0; u < UB; ++u) {
      if (u0 + u < uend) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          v4i wb[NB];
#pragma unroll
          for (int nb = 0; nb < NB; ++nb)
            wb[nb] = widen16_u2(h ? make_uint2(fb[u][nb].z, fb[u][nb].w) : make_uint2(fb[u][nb].x, fb[u][nb].y));
#pragma unroll
          for (int rb = 0; rb < MB; ++rb) {
            v4i xa;
            if constexpr (A8) {
              xa = order16_i8(aok[rb] ? fa[u][rb][h] : make_uint4(0, 0, 0, 0));
            } else {
              const uint2 pa = h ? make_uint2(fa[u][rb][0].z, fa[u][rb][0].w) : make_uint2(fa[u][rb][0].x, fa[u][rb][0].y);
              xa = widen16_u2(aok[rb] ? pa : make_uint2(0, 0));
            }
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
              acc[rb][nb] = __builtin_amdgcn_mfma_i32_16x16x64_i8(xa, wb[nb], acc[rb][nb], 0, 0, 0);
          }
        }
      }
    }
  };
  // First round straight-line (the MFMAs of a unit wait only for that unit's
  // loads); deeper K continues in rounds of UB units.
  mfma_units(ubeg);
  for (int u0 = ubeg + UB; u0 < uend; u0 += UB) {
    load_units(u0);
    mfma_units(u0);
  }
  if (!TILED && (a.K & 127) && wave == WAVES - 1) {
    // Final 64 codes: 32 packed bytes per row, 8 per lane.
    const int64_t off = static_cast<int64_t>(nu) * 64 + 8 * (lane >> 4);
    v4i wb[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) wb[nb] = widen16_u2(*reinterpret_cast<const uint2*>(bbase[nb] + off));
#pragma unroll
    for (int rb = 0; rb < MB; ++rb) {
      v4i xa;
      if constexpr (A8)
        xa = order16_i8(aok[rb] ? *reinterpret_cast<const uint4*>(abase[rb] + 2 * off) : make_uint4(0, 0, 0, 0));
      else
        xa = widen16_u2(aok[rb] ? *reinterpret_cast<const uint2*>(abase[rb] + off) : make_uint2(0, 0));
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
        acc[rb][nb] = __builtin_amdgcn_mfma_i32_16x16x64_i8(xa, wb[nb], acc[rb][nb], 0, 0, 0);
    }
  }

  // 16x16 accumulator layout: element e of lane l is row 4*(l/16) + e, column l%16.
#pragma unroll
  for (int rb = 0; rb < MB; ++rb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        red[wave][(rb * 16 + 4 * (lane >> 4) + e) * BNs + nb * 16 + (lane & 15)] = acc[rb][nb][e];
  __syncthreads();
#pragma unroll
  for (int u = 0; u < OPT; ++u) {
    const int i = tid + u * NT;
    const int64_t gr = m0 + i / BNs;
    if (i >= NOUT || gr >= a.M || !ecol_ok) continue;
    int sum = 0;
#pragma unroll
    for (int w = 0; w < WAVES; ++w) sum += red[w][i];
    store_out<EPI>(a, gr * a.ldc + egc, sum >> (A8 ? 4 : 8), e_xs[u], e_ws, e_bias, e_gate, e_res[u]);
  }
}

// Tile shape of the small-M product: 32 columns per workgroup when N is wide
// enough to keep more than 256 workgroups busy, else 16; waves sized so that
// each takes one or two 128-code units of K at K <= 1024 and up to 2 (16
// columns) or 4 (32 columns) at K <= 4096 in its first round; deeper K runs
// more rounds.
template <int EPI, bool TILED, int MB, bool A8 = false>
int launch_small_mb(const GemmArgs& a, hipStream_t stream) {
  const bool wide = a.N > 4096;
  const bool shallow = a.K <= 1024;
  const int bn = wide ? 32 : 16;
  // 8-bit token codes take twice the registers per unit: half the units per
  // round in the deep cases (1024 threads leave 128 registers per lane).
  constexpr int UBW = A8 ? 2 : 4;
  const dim3 grid(static_cast<unsigned>((a.N + bn - 1) / bn), static_cast<unsigned>((a.M + 16 * MB - 1) / (16 * MB)));
  if (wide && shallow) hipLaunchKernelGGL((gemm_small_kernel<EPI, 2, 8, MB, 1, TILED, A8>), grid, dim3(512), 0, stream, a);
  else if (wide) hipLaunchKernelGGL((gemm_small_kernel<EPI, 2, 8, MB, UBW, TILED, A8>), grid, dim3(512), 0, stream, a);
  else if (shallow) hipLaunchKernelGGL((gemm_small_kernel<EPI, 1, 4, MB, 2, TILED, A8>), grid, dim3(256), 0, stream, a);
  else hipLaunchKernelGGL((gemm_small_kernel<EPI, 1, 16, MB, A8 ? 1 : 2, TILED, A8>), grid, dim3(1024), 0, stream, a);
  return launch_status();
}

// Row blocks of 16 (one per workgroup) spread a small-M product over four
// times the workgroups of 64-row blocks; that pays while the grid stays
// within 16 waves per CU (the 50-row DiT linears: q|k|v, o and down, 1.5 to
// 5 thousand waves; not the 8192-column gate|up, whose 32-column workgroups of
// 8 waves would make 8 thousand).
bool small_row_blocks_of_16(const GemmArgs& a) {
  const bool wide = a.N > 4096, shallow = a.K <= 1024;
  const int64_t bn = wide ? 32 : 16, waves = wide ? 8 : (shallow ? 4 : 16);
  const int64_t total = (a.N + bn - 1) / bn * ((a.M + 15) / 16) * waves;
  return a.M <= 16 || total <= 4096;
}

template <int EPI, bool TILED>
int launch_small(const GemmArgs& a, hipStream_t stream) {
  return small_row_blocks_of_16(a) ? launch_small_mb<EPI, TILED, 1>(a, stream) : launch_small_mb<EPI, TILED, 4>(a, stream);
}

template <int EPI>
int launch_small_any(const GemmArgs& a, hipStream_t stream) {
  if (a.a_i8)
    return a.M <= 16 ? launch_small_mb<EPI, false, 1, true>(a, stream) : launch_small_mb<EPI, false, 4, true>(a, stream);
  return a.a_tiled ? launch_small<EPI, true>(a, stream) : launch_small<EPI, false>(a, stream);
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

template <int WM, int WN, int TM, int TN, bool A8, int NS, int KG>
int launch_big_a(const GemmArgs& a, Epilogue epi, int64_t tiles, hipStream_t stream) {
  const dim3 g(static_cast<unsigned>(tiles * a.splitk)), b(64 * WM * WN * KG);
  switch (epi) {
    case EPI_I32: hipLaunchKernelGGL((gemm_big_kernel<EPI_I32, WM, WN, TM, TN, A8, NS, KG>), g, b, 0, stream, a); break;
    case EPI_F16: hipLaunchKernelGGL((gemm_big_kernel<EPI_F16, WM, WN, TM, TN, A8, NS, KG>), g, b, 0, stream, a); break;
    case EPI_BF16:
      hipLaunchKernelGGL((gemm_big_kernel<EPI_BF16, WM, WN, TM, TN, A8, NS, KG>), g, b, 0, stream, a);
      break;
    case EPI_GELU_F16:
      if constexpr (A8) return OQ_ERR_ARG;  // a DiT path only
      else hipLaunchKernelGGL((gemm_big_kernel<EPI_GELU_F16, WM, WN, TM, TN, A8, NS, KG>), g, b, 0, stream, a);
      break;
    case EPI_RESID_F32:
      if constexpr (A8) return OQ_ERR_ARG;  // the residual epilogue is a W4A4 DiT path only
      else hipLaunchKernelGGL((gemm_big_kernel<EPI_RESID_F32, WM, WN, TM, TN, A8, NS, KG>), g, b, 0, stream, a);
      break;
    default: return OQ_ERR_ARG;
  }
  return launch_status();
}

template <int WM, int WN, int TM, int TN, int NS, int KG = 1>
int launch_big(const GemmArgs& a, Epilogue epi, int64_t tiles, hipStream_t stream) {
  if constexpr (WM * WN * TM * TN <= 16 && 2 * 32 * TM * WM >= 64 * WM * WN) {
    if (a.a_i8) return launch_big_a<WM, WN, TM, TN, true, NS, KG>(a, epi, tiles, stream);
  }
  return launch_big_a<WM, WN, TM, TN, false, NS, KG>(a, epi, tiles, stream);
}

int gemm_launch(const GemmArgs& a, Epilogue epi, hipStream_t stream) {
  if (a.M == 0) return OQ_OK;
  // Tiled token codes always take the small-M kernel (row groups of 64 along
  // grid.y when M > 64); row-layout codes take it up to M = 64.
  if (a.a_i8 && (epi == EPI_RESID_F32 || epi == EPI_GELU_F16)) return OQ_ERR_ARG;
  if (a.M <= 64 || a.a_tiled) {
    switch (epi) {
      case EPI_I32: return launch_small_any<EPI_I32>(a, stream);
      case EPI_F16: return launch_small_any<EPI_F16>(a, stream);
      case EPI_BF16: return launch_small_any<EPI_BF16>(a, stream);
      case EPI_RESID_F32: return launch_small_any<EPI_RESID_F32>(a, stream);
      case EPI_GELU_F16: return launch_small_any<EPI_GELU_F16>(a, stream);
      default: return OQ_ERR_ARG;
    }
  }
  // Large problems: 256 x 256 tiles (8 waves of 128 x 64) when they still
  // fill every CU, else 128 x 128 tiles (4 waves of 64 x 64, two workgroups
  // per CU), else 64 x 64 tiles (2 waves of 64 x 32, four workgroups per CU).
  // 8-bit token codes double the A register ring, which the 256 x 256 tile
  // cannot hold without spilling: they always take the 128 x 128 tile.
  const int64_t big_tiles = ((a.M + 255) / 256) * ((a.N + 255) / 256);
  // (At most 1024 rows, e.g. the 816-row prefill gate|up, 128 x 128 tiles
  // waste fewer rows: 80 against 83 us there.)
  if (big_tiles >= 256 && !a.a_i8 && a.M > 1024) return launch_big<2, 4, 4, 2, 3>(a, epi, big_tiles, stream);
  const int64_t mid_tiles = ((a.M + 127) / 128) * ((a.N + 127) / 128);
  // Two K groups (two wave groups of one workgroup on alternate stages of K,
  // summed through LDS) halve the serial stage chain of a tile; a K-grouped
  // workgroup needs twice the LDS, so they are used only while its tiles
  // still fit the CUs in one round: 128 x 128 tiles at one workgroup per CU,
  // 64 x 64 tiles at two.  (Measured 12-34% faster at M = 256 - 1024 with N =
  // 1536 - 8192; slower once a second round of workgroups is needed.)
  const bool kgroups = !a.a_i8;
  if (mid_tiles >= 256) {
    if (kgroups && mid_tiles <= 256) return launch_big<2, 4, 2, 1, 3, 2>(a, epi, mid_tiles, stream);
    if (!a.a_i8) return launch_big<2, 4, 2, 1, 3>(a, epi, mid_tiles, stream);
    return launch_big<2, 2, 2, 2, 3>(a, epi, mid_tiles, stream);
  }
  // Fewer 128 x 128 tiles than CUs (prefill-sized M with N ~ 2048): 64 x 64
  // tiles of two waves (64 x 32 each), several workgroups per CU.  Deep K
  // (K >= 6144) keeps more register stages in flight (twelve without K
  // groups: 7-11% faster at M = 816 - 1024, N = 1536 - 2048).
  const int64_t small_tiles = ((a.M + 63) / 64) * ((a.N + 63) / 64);
  // Deep K with the caller's split-K scratch: two K halves as separate
  // one-group workgroups (36 KB of LDS, four per CU), so that 257 - 512 tiles
  // make 514 - 1024 equal workgroups resident at once, where two-group
  // workgroups (two per CU) leave some CUs with one tile and others with two.
  constexpr int64_t kWords64 = 64 * 64;  // int32 partial of a 64 x 64 tile
  if (kgroups && small_tiles > 256 && small_tiles <= 512 && a.K >= 6144 && a.part && a.tickets &&
      a.part_words >= 2 * small_tiles * kWords64 && a.n_tickets >= small_tiles) {
    GemmArgs s2 = a;
    s2.splitk = 2;
    return launch_big<2, 2, 1, 1, 4>(s2, epi, small_tiles, stream);
  }
  if (kgroups && small_tiles <= 512) {
    if (a.K >= 6144) return launch_big<2, 2, 1, 1, 4, 2>(a, epi, small_tiles, stream);
    return launch_big<2, 2, 1, 1, 3, 2>(a, epi, small_tiles, stream);
  }
  if (a.a_i8) {
    if (a.K >= 6144) return launch_big<1, 2, 2, 1, 12>(a, epi, small_tiles, stream);
    return launch_big<1, 2, 2, 1, 3>(a, epi, small_tiles, stream);
  }
  if (a.K >= 6144) return launch_big<2, 2, 1, 1, 12>(a, epi, small_tiles, stream);
  return launch_big<2, 2, 1, 1, 3>(a, epi, small_tiles, stream);
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

extern "C" int oq_w4a4_linear_tiled(const uint8_t* Xt, const float* x_scale, int64_t M, const uint8_t* Wq,
                                    const float* w_scale, const void* bias, int64_t N, int64_t K, void* Y,
                                    int64_t ldy, int32_t out_dtype, void* stream) {
  int st = oq::gemm_validate(Xt, M, Wq, N, K, Y, ldy, 8);
  if (st != OQ_OK) return st;
  if (K % 128 != 0) return OQ_ERR_SHAPE;
  if (M == 0) return OQ_OK;
  if (!x_scale || !w_scale) return OQ_ERR_NULL;
  if (out_dtype != OQ_OUT_F16 && out_dtype != OQ_OUT_BF16) return OQ_ERR_ARG;
  if (!oq::aligned(x_scale, 4) || !oq::aligned(w_scale, 4) || (bias && !oq::aligned(bias, 2))) return OQ_ERR_ALIGN;
  if ((st = oq::device_check()) != OQ_OK) return st;
  oq::GemmArgs a{Xt, Wq, x_scale, w_scale, static_cast<const uint16_t*>(bias), Y, nullptr, M, N, K, ldy, true};
  return oq::gemm_launch(a, out_dtype == OQ_OUT_F16 ? oq::EPI_F16 : oq::EPI_BF16, static_cast<hipStream_t>(stream));
}

extern "C" int oq_w4a4_gemm_i32_tiled(const uint8_t* Xt, int64_t M, const uint8_t* Wq, int64_t N, int64_t K,
                                      int32_t* acc, int64_t ldc, void* stream) {
  int st = oq::gemm_validate(Xt, M, Wq, N, K, acc, ldc, 4);
  if (st != OQ_OK) return st;
  if (K % 128 != 0) return OQ_ERR_SHAPE;
  if (M == 0) return OQ_OK;
  if ((st = oq::device_check()) != OQ_OK) return st;
  oq::GemmArgs a{Xt, Wq, nullptr, nullptr, nullptr, acc, nullptr, M, N, K, ldc, true};
  return oq::gemm_launch(a, oq::EPI_I32, static_cast<hipStream_t>(stream));
}

extern "C" int oq_w4a8_linear(const int8_t* Xq8, const float* x_scale, int64_t M, const uint8_t* Wq,
                              const float* w_scale, const void* bias, int64_t N, int64_t K, void* Y,
                              int64_t ldy, int32_t out_dtype, void* stream) {
  const uint8_t* A = reinterpret_cast<const uint8_t*>(Xq8);
  int st = oq::gemm_validate(A, M, Wq, N, K, Y, ldy, 8);
  if (st != OQ_OK || M == 0) return st;
  if (!x_scale || !w_scale) return OQ_ERR_NULL;
  if (out_dtype != OQ_OUT_F16 && out_dtype != OQ_OUT_BF16) return OQ_ERR_ARG;
  if (!oq::aligned(x_scale, 4) || !oq::aligned(w_scale, 4) || (bias && !oq::aligned(bias, 2))) return OQ_ERR_ALIGN;
  if ((st = oq::device_check()) != OQ_OK) return st;
  oq::GemmArgs a{A, Wq, x_scale, w_scale, static_cast<const uint16_t*>(bias), Y, nullptr, M, N, K, ldy, false, true};
  return oq::gemm_launch(a, out_dtype == OQ_OUT_F16 ? oq::EPI_F16 : oq::EPI_BF16, static_cast<hipStream_t>(stream));
}

extern "C" int oq_w4a8_gemm_i32(const int8_t* Xq8, int64_t M, const uint8_t* Wq, int64_t N, int64_t K,
                                int32_t* acc, int64_t ldc, void* stream) {
  const uint8_t* A = reinterpret_cast<const uint8_t*>(Xq8);
  int st = oq::gemm_validate(A, M, Wq, N, K, acc, ldc, 4);
  if (st != OQ_OK || M == 0) return st;
  if ((st = oq::device_check()) != OQ_OK) return st;
  oq::GemmArgs a{A, Wq, nullptr, nullptr, nullptr, acc, nullptr, M, N, K, ldc, false, true};
  return oq::gemm_launch(a, oq::EPI_I32, static_cast<hipStream_t>(stream));
}
