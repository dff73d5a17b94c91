// DiT action-head denoising step built from the rotated W4A4 linears.
//
// Experimental Settings / Implementation Details: every linear of the DiT
// action head is W4A4 with RTN weights and the per-step activation scale
// table, and the head runs T Euler denoising steps.  The Appendix on per-step
// scaling describes the block: a time-conditioned norm feeding the attention
// q/k/v projections, attention output projection, a norm feeding the MLP.
// Block equations of the Pi-0.5 action expert used here:
//   h = fp16(rms(r) g1 (1 + sc1) + sh1); qkv = W4A4(h); o = attn(q, [Kp;k], [Vp;v]);
//   r += gt1 W4A4(o); h2 = fp16(rms(r) g2 (1 + sc2) + sh2); gu = W4A4(h2);
//   a = fp16(gelu_tanh(gate) up); r += gt2 W4A4(a)
// and the step r = x W_in^T + b_in -> blocks -> v = fp16(rms(r) g_f) W_out^T +
// b_out -> x += dt v.
//
// Kernels (all on the caller's stream, no allocation, no memset):
//   inproj_kernel      r = x W_in^T + b_in                      (fp32 residual)
//   adarms_kernel      h = fp16(rms(r) g (1 + sc) + sh)
//   rq / gemm          the rotated W4A4 linears (rotate_quant.hip, w4a4_gemm.hip);
//                      o and down projections add gate * y into r in the epilogue
//   attn_partial_kernel  softmax(q k^T / sqrt(hd)) v over one 32-key split
//   attn_combine_kernel  merge the splits (log-sum-exp), fp16 output
//   gelu_mul_kernel    a = fp16(gelu_tanh(gate) up)
//   final_kernel       rms norm, out projection, Euler update of x
#include <cmath>
#include <cstring>
#include <vector>

#include "common.h"

namespace oq {
namespace {

constexpr int kAttnKS = 32;     // keys per attention split
constexpr int kMaxTokens = 64;  // action tokens per sample handled by the attention kernels
constexpr int kMaxHeadDim = 128;
constexpr float kEps = 1e-6f;

__device__ __forceinline__ float h2f(uint16_t h) { return static_cast<float>(__builtin_bit_cast(_Float16, h)); }
__device__ __forceinline__ uint16_t f2h(float f) { return __builtin_bit_cast(uint16_t, static_cast<_Float16>(f)); }

__device__ float block_sum(float v, float* red) {
  // 256 threads.
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  float s = red[0] + red[1] + red[2] + red[3];
  __syncthreads();
  return s;
}

// r[m][n] = sum_a x[m][a] w_in[n][a] + b_in[n]
__global__ __launch_bounds__(256) void inproj_kernel(const float* __restrict__ x, const uint16_t* __restrict__ w_in,
                                                     const uint16_t* __restrict__ b_in, float* __restrict__ r, int A,
                                                     int D) {
  extern __shared__ float xs[];
  const int m = blockIdx.x;
  for (int a = threadIdx.x; a < A; a += blockDim.x) xs[a] = x[static_cast<int64_t>(m) * A + a];
  __syncthreads();
  for (int n = threadIdx.x; n < D; n += blockDim.x) {
    const uint16_t* wr = w_in + static_cast<int64_t>(n) * A;
    float acc = 0.0f;
    for (int a = 0; a < A; ++a) acc = fmaf(xs[a], h2f(wr[a]), acc);
    r[static_cast<int64_t>(m) * D + n] = acc + h2f(b_in[n]);
  }
}

// h = fp16(rms(r) * g * (1 + sc) + sh); sc / sh may be null (plain gain).
__global__ __launch_bounds__(256) void adarms_kernel(const float* __restrict__ r, const uint16_t* __restrict__ g,
                                                     const uint16_t* __restrict__ sc, const uint16_t* __restrict__ sh,
                                                     uint16_t* __restrict__ h, int D) {
  __shared__ float red[4];
  const int64_t m = blockIdx.x;
  const float* rr = r + m * D;
  float ss = 0.0f;
  for (int d = threadIdx.x; d < D; d += blockDim.x) ss = fmaf(rr[d], rr[d], ss);
  ss = block_sum(ss, red);
  const float inv = 1.0f / sqrtf(ss / static_cast<float>(D) + kEps);
  for (int d = threadIdx.x; d < D; d += blockDim.x) {
    float y = rr[d] * inv * h2f(g[d]);
    if (sc) y = fmaf(y, h2f(sc[d]), y);
    if (sh) y += h2f(sh[d]);
    h[m * D + d] = f2h(y);
  }
}

__device__ __forceinline__ float gelu_tanh(float x) {
  const float k0 = 0.7978845608028654f;  // sqrt(2/pi)
  const float k1 = 0.044715f;
  return 0.5f * x * (1.0f + tanhf(k0 * fmaf(k1 * x * x, x, x)));
}

// a[m][f] = fp16(gelu_tanh(gu[m][f]) * gu[m][F + f])
__global__ __launch_bounds__(256) void gelu_mul_kernel(const uint16_t* __restrict__ gu, uint16_t* __restrict__ out,
                                                       int64_t M, int F) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= M * F) return;
  const int64_t m = i / F, f = i % F;
  const float gate = h2f(gu[m * 2 * F + f]);
  const float up = h2f(gu[m * 2 * F + F + f]);
  out[i] = f2h(gelu_tanh(gate) * up);
}

struct AttnArgs {
  const uint16_t* q; int64_t q_ld;                      // [B*S][..], head h at column h*hd
  const uint16_t* k_pre; const uint16_t* v_pre; int P;  // [B][P][D] (P may be 0)
  const uint16_t* k_own; const uint16_t* v_own; int64_t own_ld; int own_keys;  // [B*S][..]
  float* part_o; float* part_ml;                        // workspace
  uint16_t* out; int64_t out_ld;
  int S, H, hd, D, nsplit;
  float scale;
};

// One (sample b, head h, 32-key split): partial max, sum and weighted values.
__global__ __launch_bounds__(256) void attn_partial_kernel(AttnArgs a) {
  __shared__ float sK[kAttnKS][kMaxHeadDim + 1];
  __shared__ float sV[kAttnKS][kMaxHeadDim];
  __shared__ uint16_t sQ[kMaxTokens][kMaxHeadDim];
  __shared__ float sP[kMaxTokens][kAttnKS + 1];

  const int bh = blockIdx.x, split = blockIdx.y;
  const int b = bh / a.H, h = bh % a.H;
  const int tid = threadIdx.x;
  const int n_keys = a.P + a.own_keys;
  const int k0 = split * kAttnKS;
  const int nk = min(kAttnKS, n_keys - k0);

  for (int i = tid; i < a.S * a.hd; i += blockDim.x) {
    const int q = i / a.hd, d = i % a.hd;
    sQ[q][d] = a.q[(static_cast<int64_t>(b) * a.S + q) * a.q_ld + h * a.hd + d];
  }
  for (int i = tid; i < kAttnKS * a.hd; i += blockDim.x) {
    const int j = i / a.hd, d = i % a.hd;
    float kv = 0.0f, vv = 0.0f;
    if (j < nk) {
      const int key = k0 + j;
      if (key < a.P) {
        const int64_t off = (static_cast<int64_t>(b) * a.P + key) * a.D + h * a.hd + d;
        kv = h2f(a.k_pre[off]);
        vv = h2f(a.v_pre[off]);
      } else {
        const int64_t off = (static_cast<int64_t>(b) * a.own_keys + (key - a.P)) * a.own_ld + h * a.hd + d;
        kv = h2f(a.k_own[off]);
        vv = h2f(a.v_own[off]);
      }
    }
    sK[j][d] = kv;
    sV[j][d] = vv;
  }
  __syncthreads();

  // Scores.
  {
    const int j = tid & (kAttnKS - 1);
    for (int q = tid / kAttnKS; q < a.S; q += blockDim.x / kAttnKS) {
      float s = -INFINITY;
      if (j < nk) {
        float acc = 0.0f;
        for (int d = 0; d < a.hd; ++d) acc = fmaf(h2f(sQ[q][d]), sK[j][d], acc);
        s = acc * a.scale;
      }
      sP[q][j] = s;
    }
  }
  __syncthreads();

  // Row max and sum of this split; probabilities relative to the split max.
  float* ml = a.part_ml + (static_cast<int64_t>(bh) * a.nsplit + split) * a.S * 2;
  for (int q = tid; q < a.S; q += blockDim.x) {
    float mx = -INFINITY;
    for (int j = 0; j < nk; ++j) mx = fmaxf(mx, sP[q][j]);
    float l = 0.0f;
    for (int j = 0; j < kAttnKS; ++j) {
      const float p = j < nk ? __expf(sP[q][j] - mx) : 0.0f;
      sP[q][j] = p;
      l += p;
    }
    ml[2 * q] = mx;
    ml[2 * q + 1] = l;
  }
  __syncthreads();

  float* po = a.part_o + (static_cast<int64_t>(bh) * a.nsplit + split) * a.S * a.hd;
  for (int i = tid; i < a.S * a.hd; i += blockDim.x) {
    const int q = i / a.hd, d = i % a.hd;
    float acc = 0.0f;
    for (int j = 0; j < kAttnKS; ++j) acc = fmaf(sP[q][j], sV[j][d], acc);
    po[i] = acc;
  }
}

// Merge the splits of one (b, h): out = sum_s e^{m_s - M} o_s / sum_s e^{m_s - M} l_s.
__global__ __launch_bounds__(256) void attn_combine_kernel(AttnArgs a) {
  const int bh = blockIdx.x;
  const int b = bh / a.H, h = bh % a.H;
  const float* ml = a.part_ml + static_cast<int64_t>(bh) * a.nsplit * a.S * 2;
  const float* po = a.part_o + static_cast<int64_t>(bh) * a.nsplit * a.S * a.hd;
  for (int i = threadIdx.x; i < a.S * a.hd; i += blockDim.x) {
    const int q = i / a.hd, d = i % a.hd;
    float M = -INFINITY;
    for (int s = 0; s < a.nsplit; ++s) M = fmaxf(M, ml[(s * a.S + q) * 2]);
    float num = 0.0f, den = 0.0f;
    for (int s = 0; s < a.nsplit; ++s) {
      const float w = __expf(ml[(s * a.S + q) * 2] - M);
      den = fmaf(w, ml[(s * a.S + q) * 2 + 1], den);
      num = fmaf(w, po[(static_cast<int64_t>(s) * a.S + q) * a.hd + d], num);
    }
    a.out[(static_cast<int64_t>(b) * a.S + q) * a.out_ld + h * a.hd + d] = f2h(num / den);
  }
}

// x[m][:] += dt * (fp16(rms(r[m]) g_f) W_out^T + b_out)
__global__ __launch_bounds__(256) void final_kernel(const float* __restrict__ r, const uint16_t* __restrict__ g_f,
                                                    const uint16_t* __restrict__ w_out,
                                                    const uint16_t* __restrict__ b_out, float* __restrict__ x, int D,
                                                    int A, float dt) {
  extern __shared__ float sh[];  // [D] normalized row, then [256] partial sums
  __shared__ float red[4];
  const int64_t m = blockIdx.x;
  const float* rr = r + m * D;
  float ss = 0.0f;
  for (int d = threadIdx.x; d < D; d += blockDim.x) ss = fmaf(rr[d], rr[d], ss);
  ss = block_sum(ss, red);
  const float inv = 1.0f / sqrtf(ss / static_cast<float>(D) + kEps);
  for (int d = threadIdx.x; d < D; d += blockDim.x) sh[d] = h2f(f2h(rr[d] * inv * h2f(g_f[d])));
  __syncthreads();
  float* part = sh + D;
  // Thread t: output a = t % A over the d-slice t / A (A divides 256 is not
  // required: threads beyond the last full slice idle).
  const int slices = blockDim.x / A;
  const int a_idx = threadIdx.x % A, sl = threadIdx.x / A;
  float acc = 0.0f;
  if (sl < slices) {
    const int per = (D + slices - 1) / slices;
    const int d0 = sl * per, d1 = min(D, d0 + per);
    const uint16_t* wr = w_out + static_cast<int64_t>(a_idx) * D;
    for (int d = d0; d < d1; ++d) acc = fmaf(sh[d], h2f(wr[d]), acc);
  }
  part[threadIdx.x] = acc;
  __syncthreads();
  if (threadIdx.x < A) {
    float v = h2f(b_out[threadIdx.x]);
    for (int s = 0; s < slices; ++s) v += part[s * A + threadIdx.x];
    x[m * A + threadIdx.x] += dt * v;
  }
}

size_t align256(size_t n) { return (n + 255) & ~static_cast<size_t>(255); }

struct Layout {
  size_t r, h1, qkv, o, h2, gu, act, xq, xs, part_o, part_ml, total;
};

Layout layout_for(const oq_dit_config& c) {
  const int64_t M = static_cast<int64_t>(c.batch) * c.tokens;
  const int64_t D = c.hidden, F = c.mlp;
  const int64_t Kmax = std::max(D, F);
  const int nsplit = (c.prefix + c.tokens + kAttnKS - 1) / kAttnKS;
  const int64_t BH = static_cast<int64_t>(c.batch) * c.n_heads;
  Layout L;
  size_t off = 0;
  L.r = off; off += align256(M * D * 4);
  L.h1 = off; off += align256(M * D * 2);
  L.qkv = off; off += align256(M * 3 * D * 2);
  L.o = off; off += align256(M * D * 2);
  L.h2 = off; off += align256(M * D * 2);
  L.gu = off; off += align256(M * 2 * F * 2);
  L.act = off; off += align256(M * F * 2);
  L.xq = off; off += align256(M * Kmax / 2);
  L.xs = off; off += align256(M * 4);
  L.part_o = off; off += align256(BH * nsplit * c.tokens * c.head_dim * 4);
  L.part_ml = off; off += align256(BH * nsplit * c.tokens * 2 * 4);
  L.total = off;
  return L;
}

int validate_config(const oq_dit_config* c) {
  if (!c) return OQ_ERR_NULL;
  if (c->arch != OQ_DIT_PI) return OQ_ERR_ARG;
  if (c->n_blocks < 1 || c->steps < 1 || c->batch < 1 || c->tokens < 1 || c->prefix < 0) return OQ_ERR_SHAPE;
  if (c->hidden < 64 || c->hidden % 64 || c->mlp < 64 || c->mlp % 64) return OQ_ERR_SHAPE;
  if (c->hidden > 16384 || c->mlp > 16384) return OQ_ERR_SHAPE;
  if (c->n_heads < 1 || c->head_dim < 8 || c->head_dim > kMaxHeadDim || c->head_dim % 8 ||
      c->n_heads * c->head_dim != c->hidden)
    return OQ_ERR_SHAPE;
  if (c->tokens > kMaxTokens || c->action_dim < 1 || c->action_dim > 256) return OQ_ERR_SHAPE;
  RQPlan p;
  if (!rq_plan(c->hidden, &p) || !rq_plan(c->mlp, &p)) return OQ_ERR_SHAPE;
  return OQ_OK;
}

int pow2_divisor(int n) { return n & (-n); }

}  // namespace
}  // namespace oq

struct oq_dit {
  oq_dit_config cfg;
  oq_dit_weights w;
  std::vector<oq_dit_block> blocks;
  std::vector<float> s_table;
  oq::Layout lay;
  uint8_t* ws = nullptr;
  size_t ws_bytes = 0;
};

namespace oq {
namespace {

template <typename T>
T* at(oq_dit* h, size_t off) { return reinterpret_cast<T*>(h->ws + off); }

const uint16_t* mod_ptr(oq_dit* h, int l, int t, int k) {
  const int64_t D = h->cfg.hidden;
  return static_cast<const uint16_t*>(h->w.mod) + ((static_cast<int64_t>(l) * h->cfg.steps + t) * 6 + k) * D;
}

int linear(oq_dit* h, const uint16_t* x, int64_t K, float s, const oq_qweight& wt, int64_t N, Epilogue epi,
           void* out, int64_t ldc, const uint16_t* gate, hipStream_t st) {
  const int64_t M = static_cast<int64_t>(h->cfg.batch) * h->cfg.tokens;
  uint8_t* xq = at<uint8_t>(h, h->lay.xq);
  float* xs = at<float>(h, h->lay.xs);
  int e = rq_launch(x, M, K, K, pow2_divisor(static_cast<int>(K)), s, xq, xs, nullptr, st);
  if (e != OQ_OK) return e;
  GemmArgs a{xq, wt.wq, xs, wt.w_scale, nullptr, out, gate, M, N, K, ldc};
  return gemm_launch(a, epi, st);
}

int run_block(oq_dit* h, int l, int t, float* r, hipStream_t st) {
  const oq_dit_config& c = h->cfg;
  const oq_dit_block& bw = h->blocks[l];
  const int64_t M = static_cast<int64_t>(c.batch) * c.tokens;
  const int64_t D = c.hidden, F = c.mlp;
  const float* s = &h->s_table[(static_cast<size_t>(l) * c.steps + t) * 4];
  uint16_t* h1 = at<uint16_t>(h, h->lay.h1);
  uint16_t* qkv = at<uint16_t>(h, h->lay.qkv);
  uint16_t* o = at<uint16_t>(h, h->lay.o);
  uint16_t* h2 = at<uint16_t>(h, h->lay.h2);
  uint16_t* gu = at<uint16_t>(h, h->lay.gu);
  uint16_t* act = at<uint16_t>(h, h->lay.act);
  int e;

  hipLaunchKernelGGL(adarms_kernel, dim3(static_cast<unsigned>(M)), dim3(256), 0, st, r,
                     static_cast<const uint16_t*>(bw.g1), mod_ptr(h, l, t, 0), mod_ptr(h, l, t, 1), h1,
                     static_cast<int>(D));
  if ((e = launch_status()) != OQ_OK) return e;
  if ((e = linear(h, h1, D, s[0], bw.qkv, 3 * D, EPI_F16, qkv, 3 * D, nullptr, st)) != OQ_OK) return e;

  AttnArgs a;
  a.q = qkv; a.q_ld = 3 * D;
  a.k_pre = static_cast<const uint16_t*>(bw.prefix_k);
  a.v_pre = static_cast<const uint16_t*>(bw.prefix_v);
  a.P = c.prefix;
  a.k_own = qkv + D; a.v_own = qkv + 2 * D; a.own_ld = 3 * D; a.own_keys = c.tokens;
  a.part_o = at<float>(h, h->lay.part_o);
  a.part_ml = at<float>(h, h->lay.part_ml);
  a.out = o; a.out_ld = D;
  a.S = c.tokens; a.H = c.n_heads; a.hd = c.head_dim; a.D = static_cast<int>(D);
  a.nsplit = (c.prefix + c.tokens + kAttnKS - 1) / kAttnKS;
  a.scale = static_cast<float>(1.0 / std::sqrt(static_cast<double>(c.head_dim)));
  hipLaunchKernelGGL(attn_partial_kernel, dim3(c.batch * c.n_heads, a.nsplit), dim3(256), 0, st, a);
  if ((e = launch_status()) != OQ_OK) return e;
  hipLaunchKernelGGL(attn_combine_kernel, dim3(c.batch * c.n_heads), dim3(256), 0, st, a);
  if ((e = launch_status()) != OQ_OK) return e;

  if ((e = linear(h, o, D, s[1], bw.o, D, EPI_RESID_F32, r, D, mod_ptr(h, l, t, 2), st)) != OQ_OK) return e;

  hipLaunchKernelGGL(adarms_kernel, dim3(static_cast<unsigned>(M)), dim3(256), 0, st, r,
                     static_cast<const uint16_t*>(bw.g2), mod_ptr(h, l, t, 3), mod_ptr(h, l, t, 4), h2,
                     static_cast<int>(D));
  if ((e = launch_status()) != OQ_OK) return e;
  if ((e = linear(h, h2, D, s[2], bw.gate_up, 2 * F, EPI_F16, gu, 2 * F, nullptr, st)) != OQ_OK) return e;

  const int64_t n = M * F;
  hipLaunchKernelGGL(gelu_mul_kernel, dim3(static_cast<unsigned>((n + 255) / 256)), dim3(256), 0, st, gu, act, M,
                     static_cast<int>(F));
  if ((e = launch_status()) != OQ_OK) return e;
  return linear(h, act, F, s[3], bw.down, D, EPI_RESID_F32, r, D, mod_ptr(h, l, t, 5), st);
}

int run_step(oq_dit* h, float* x, int t, hipStream_t st) {
  const oq_dit_config& c = h->cfg;
  const int64_t M = static_cast<int64_t>(c.batch) * c.tokens;
  float* r = at<float>(h, h->lay.r);
  hipLaunchKernelGGL(inproj_kernel, dim3(static_cast<unsigned>(M)), dim3(256), c.action_dim * sizeof(float), st, x,
                     static_cast<const uint16_t*>(h->w.w_in), static_cast<const uint16_t*>(h->w.b_in), r,
                     c.action_dim, c.hidden);
  int e = launch_status();
  if (e != OQ_OK) return e;
  for (int l = 0; l < c.n_blocks; ++l)
    if ((e = run_block(h, l, t, r, st)) != OQ_OK) return e;
  const float dt = -1.0f / static_cast<float>(c.steps);
  hipLaunchKernelGGL(final_kernel, dim3(static_cast<unsigned>(M)), dim3(256), (c.hidden + 256) * sizeof(float), st,
                     r, static_cast<const uint16_t*>(h->w.g_f), static_cast<const uint16_t*>(h->w.w_out),
                     static_cast<const uint16_t*>(h->w.b_out), x, c.hidden, c.action_dim, dt);
  return launch_status();
}

}  // namespace
}  // namespace oq

extern "C" int oq_dit_workspace_bytes(const oq_dit_config* cfg, size_t* bytes) {
  int e = oq::validate_config(cfg);
  if (e != OQ_OK) return e;
  if (!bytes) return OQ_ERR_NULL;
  *bytes = oq::layout_for(*cfg).total;
  return OQ_OK;
}

extern "C" int oq_dit_create(const oq_dit_config* cfg, const oq_dit_weights* w, oq_dit** out) {
  int e = oq::validate_config(cfg);
  if (e != OQ_OK) return e;
  if (!w || !out || !w->blocks || !w->mod || !w->s_table || !w->w_in || !w->b_in || !w->w_out || !w->b_out ||
      !w->g_f)
    return OQ_ERR_NULL;
  for (int l = 0; l < cfg->n_blocks; ++l) {
    const oq_dit_block& b = w->blocks[l];
    if (!b.g1 || !b.g2 || !b.qkv.wq || !b.qkv.w_scale || !b.o.wq || !b.o.w_scale || !b.gate_up.wq ||
        !b.gate_up.w_scale || !b.down.wq || !b.down.w_scale)
      return OQ_ERR_NULL;
    if (cfg->prefix > 0 && (!b.prefix_k || !b.prefix_v)) return OQ_ERR_NULL;
    if (!oq::aligned(b.qkv.wq, 16) || !oq::aligned(b.o.wq, 16) || !oq::aligned(b.gate_up.wq, 16) ||
        !oq::aligned(b.down.wq, 16))
      return OQ_ERR_ALIGN;
  }
  const size_t ns = static_cast<size_t>(cfg->n_blocks) * cfg->steps * 4;
  for (size_t i = 0; i < ns; ++i)
    if (!(w->s_table[i] > 0.0f) || !std::isfinite(w->s_table[i])) return OQ_ERR_ARG;
  if ((e = oq::device_check()) != OQ_OK) return e;
  oq_dit* h = new oq_dit();
  h->cfg = *cfg;
  h->w = *w;
  h->blocks.assign(w->blocks, w->blocks + cfg->n_blocks);
  h->s_table.assign(w->s_table, w->s_table + ns);
  h->w.blocks = h->blocks.data();
  h->w.s_table = h->s_table.data();
  h->lay = oq::layout_for(*cfg);
  *out = h;
  return OQ_OK;
}

extern "C" int oq_dit_set_workspace(oq_dit* h, void* workspace, size_t bytes) {
  if (!h || !workspace) return OQ_ERR_NULL;
  if (!oq::aligned(workspace, 256)) return OQ_ERR_ALIGN;
  if (bytes < h->lay.total) return OQ_ERR_WORKSPACE;
  h->ws = static_cast<uint8_t*>(workspace);
  h->ws_bytes = bytes;
  return OQ_OK;
}

extern "C" int oq_dit_step(oq_dit* h, float* x, int32_t t, void* stream) {
  if (!h || !x) return OQ_ERR_NULL;
  if (!h->ws) return OQ_ERR_WORKSPACE;
  if (t < 0 || t >= h->cfg.steps) return OQ_ERR_ARG;
  return oq::run_step(h, x, t, static_cast<hipStream_t>(stream));
}

extern "C" int oq_dit_denoise(oq_dit* h, float* x, int32_t n_steps, void* stream) {
  if (!h || !x) return OQ_ERR_NULL;
  if (!h->ws) return OQ_ERR_WORKSPACE;
  if (n_steps < 0 || n_steps > h->cfg.steps) return OQ_ERR_ARG;
  for (int t = 0; t < n_steps; ++t) {
    int e = oq::run_step(h, x, t, static_cast<hipStream_t>(stream));
    if (e != OQ_OK) return e;
  }
  return OQ_OK;
}

extern "C" int oq_dit_run_block(oq_dit* h, int32_t l, int32_t t, float* resid, void* stream) {
  if (!h || !resid) return OQ_ERR_NULL;
  if (!h->ws) return OQ_ERR_WORKSPACE;
  if (l < 0 || l >= h->cfg.n_blocks || t < 0 || t >= h->cfg.steps) return OQ_ERR_ARG;
  return oq::run_block(h, l, t, resid, static_cast<hipStream_t>(stream));
}

extern "C" int oq_dit_get_intermediates(const oq_dit* h, oq_dit_intermediates* out) {
  if (!h || !out) return OQ_ERR_NULL;
  if (!h->ws) return OQ_ERR_WORKSPACE;
  out->h1 = h->ws + h->lay.h1;
  out->qkv = h->ws + h->lay.qkv;
  out->attn = h->ws + h->lay.o;
  out->h2 = h->ws + h->lay.h2;
  out->gate_up = h->ws + h->lay.gu;
  out->act = h->ws + h->lay.act;
  out->resid = reinterpret_cast<const float*>(h->ws + h->lay.r);
  return OQ_OK;
}

extern "C" void oq_dit_destroy(oq_dit* h) { delete h; }
