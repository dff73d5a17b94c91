/*
 * oq.h -- C ABI of the MI355X (gfx950) W4A4 rotated-linear library.
 *
 * The library implements the inference hot path of the paper's W4A4 linear
 * layer: the online Hadamard half of the composite rotation R = R_SVD . H
 * (Section 4.1, eq:composite_rot, block-wise form eq:blockdiag, transform
 * eq:transform), the per-step DiT activation scale (Section 4.2,
 * eq:perstep_scale), symmetric per-token int4 activation quantization
 * (eq:scale, eq:quant), the packed-int4 x int4 product with int32
 * accumulation and the per-token x per-channel dequantization
 * (eq:lowbit_linear), plus a DiT denoising-step driver built from them
 * (Experimental Settings, Implementation Details).
 *
 * Conventions for every entry point
 * ---------------------------------
 *  - Device pointers point to memory of the current HIP device; host
 *    pointers are marked "host".  The caller allocates and owns every buffer;
 *    the stateless calls allocate nothing.
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *    Calls are asynchronous on that stream; outputs are valid after the
 *    stream is synchronized.
 *  - Every call validates its arguments before launching anything; a call
 *    that returns an error has launched nothing and written nothing.
 *  - Return value: OQ_OK (0) or a negative oq_status.  No exception crosses
 *    the ABI.  oq_status_string() names a code.
 *  - Stateless calls are thread-safe.  A DiT handle is used from one host
 *    thread / one stream at a time.
 *
 * Data layout
 * -----------
 *  X      fp16 activation, row-major [M][ldx], K used channels per row.  It is
 *         the linear's input already expressed in the SVD basis: the SVD
 *         factor of the composite rotation is folded into the producer and
 *         the weight offline; only the Hadamard half runs online.
 *  Xq     packed int4 codes, row-major [M][K/2] bytes; byte k/2 of a row
 *         holds channel k (even) in its low nibble and channel k+1 in its
 *         high nibble, two's complement.  Codes lie in [-7, 7]; 0x8 never
 *         occurs (q_max = 2^(4-1) - 1 = 7, eq:quant).
 *  x_scale fp32 [M]: per-token dequantization step, Delta_i / s_t.
 *  Wq     packed int4 weight codes, [N][K/2] bytes, same nibble order; row n
 *         is output channel n (the weight is stored output-major, so
 *         Y = X' . W'^T).
 *  w_scale fp32 [N]: per-output-channel step Delta_W'.
 */
#ifndef OQ_H
#define OQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  OQ_OK = 0,
  OQ_ERR_NULL = -1,      /* a required pointer is NULL                              */
  OQ_ERR_SHAPE = -2,     /* a size is out of range or inconsistent (see each call)  */
  OQ_ERR_ALIGN = -3,     /* a pointer or leading dimension is not aligned            */
  OQ_ERR_DEVICE = -4,    /* the current device is not gfx950                        */
  OQ_ERR_HIP = -5,       /* a HIP runtime call or kernel launch failed              */
  OQ_ERR_WORKSPACE = -6, /* DiT workspace missing or too small                      */
  OQ_ERR_ARG = -7        /* another invalid argument (enum value, step index, ...)  */
} oq_status;

/* Output element type of the dequantizing epilogue. */
typedef enum { OQ_OUT_F16 = 0, OQ_OUT_BF16 = 1 } oq_out_dtype;

/* Largest Hadamard block the rotation kernel accepts. */
#define OQ_MAX_HAD_BLOCK 16384

/* Human-readable name of a status code (static storage, never NULL). */
const char* oq_status_string(int status);

/* Library version string (static storage). */
const char* oq_version(void);

/*
 * oq_check_device -- OQ_OK if the current HIP device is gfx950, else
 * OQ_ERR_DEVICE (or OQ_ERR_HIP if the runtime cannot be queried).  Every
 * launching call performs the same check once per device.
 */
int oq_check_device(void);

/*
 * oq_rotate_quantize_act -- online Hadamard rotation, step scale and
 * per-token int4 quantization of one activation (Section 4.1 eq:transform
 * with the block-diagonal Hadamard of eq:blockdiag; Section 4.2 eq:scale,
 * eq:quant; the per-step scale of eq:perstep_scale in its per-(layer, step)
 * scalar form).
 *
 * For each row i:  y = X[i, 0:K] . blockdiag(H_b) / sqrt(b)   (Sylvester
 * order, H[r][c] = (-1)^popcount(r & c), blocks of b contiguous channels);
 * z = s_t * y;  Delta_i = max_k |z_k| / 7;  q_k = clamp(round_half_even(
 * z_k / Delta_i), -7, 7);  x_scale[i] = Delta_i / s_t.  A row of zeros gives
 * zero codes and x_scale 0.  s_t = s_table[t] when s_table is not NULL, else
 * 1; it is read on the host when the call is made.
 *
 * X        device fp16 [M][ldx]
 * M        rows (tokens), >= 0 (0 is a no-op)
 * K        channels, multiple of 8 and of had_block, <= 16384; K/8 must be a
 *          power of two times 1 or 3 (every hidden size used here is)
 * ldx      row stride of X in elements, >= K, multiple of 8
 * had_block Hadamard block b: power of two, 1 <= b <= OQ_MAX_HAD_BLOCK, b | K
 * s_table  host fp32 table or NULL; t indexes it (t >= 0)
 * Xq       device [M][K/2] bytes;  x_scale device fp32 [M]
 * Pointers X, Xq must be 16-byte aligned; x_scale 4-byte aligned.
 * Errors: OQ_ERR_NULL, OQ_ERR_SHAPE, OQ_ERR_ALIGN, OQ_ERR_ARG (t < 0),
 * OQ_ERR_DEVICE, OQ_ERR_HIP.
 */
int oq_rotate_quantize_act(const void* X, int64_t M, int64_t K, int64_t ldx,
                           int32_t had_block, const float* s_table, int32_t t,
                           uint8_t* Xq, float* x_scale, void* stream);

/*
 * oq_rotate_debug_f32 -- same computation as oq_rotate_quantize_act, but
 * writes the pre-rounding ratio r = z / Delta_i of every element as fp32
 * [M][K] (row-major, contiguous) together with x_scale, so that a code that
 * differs from a reference can be classified as a rounding-boundary case.
 * Arguments and errors as above; ratio must be 16-byte aligned.
 */
int oq_rotate_debug_f32(const void* X, int64_t M, int64_t K, int64_t ldx,
                        int32_t had_block, const float* s_table, int32_t t,
                        float* ratio, float* x_scale, void* stream);

/*
 * oq_w4a4_linear -- int4 x int4 product with int32 accumulation and the
 * fused dequantization epilogue (eq:lowbit_linear; all scales folded into
 * the dequantization as in the Implementation Details).
 *
 * acc[i][n] = sum_k q[i][k] * wq[n][k]           (exact, int32)
 * Y[i][n]   = round_to_out(float(acc) * x_scale[i] * w_scale[n] + bias[n])
 *
 * Xq, x_scale  device, as produced by oq_rotate_quantize_act, [M][K/2], [M]
 * Wq, w_scale  device, [N][K/2], [N] (oq_quantize_weights* produce them)
 * bias         device fp16 [N] or NULL
 * M >= 0, N >= 1, K >= 64 with K % 64 == 0, K <= 16384
 * Y            device [M][ldy] of out_dtype (oq_out_dtype), ldy >= N, ldy % 8 == 0
 * Xq, Wq, Y 16-byte aligned.  Errors: OQ_ERR_NULL, OQ_ERR_SHAPE,
 * OQ_ERR_ALIGN, OQ_ERR_ARG (out_dtype), OQ_ERR_DEVICE, OQ_ERR_HIP.
 */
int oq_w4a4_linear(const uint8_t* Xq, const float* x_scale, int64_t M,
                   const uint8_t* Wq, const float* w_scale, const void* bias,
                   int64_t N, int64_t K, void* Y, int64_t ldy, int32_t out_dtype,
                   void* stream);

/*
 * oq_w4a4_gemm_i32 -- the integer product alone: acc[i][n] (int32) written
 * to device [M][ldc], ldc >= N, ldc % 4 == 0.  Shapes and errors as
 * oq_w4a4_linear.  For parity checks of the accumulators.
 */
int oq_w4a4_gemm_i32(const uint8_t* Xq, int64_t M, const uint8_t* Wq, int64_t N,
                     int64_t K, int32_t* acc, int64_t ldc, void* stream);

/*
 * 16-row tiled token codes.  With few tokens (the DiT's action tokens, decode)
 * the product of eq:lowbit_linear is bound by how fast every workgroup can
 * re-read the token codes; this layout makes each 16-byte-per-lane load of a
 * 16-row operand fragment one contiguous kilobyte.  It holds the same codes
 * as Xq (K % 128 == 0):
 *   rows padded to R16 = 16 * ceil(R / 16); total R16 * K / 2 bytes;
 *   packed byte p (0 <= p < K/2) of row r is stored at byte
 *   ((r / 16) * (K / 128) + p / 64) * 1024 + ((p / 16) % 4) * 256
 *     + (r % 16) * 16 + p % 16.
 * Bytes of padding rows are never read into a result (they may hold anything).
 */

/*
 * oq_codes_to_tiled -- re-layout of packed codes Q [rows][K/2] (device) into
 * the tiled layout T (device, R16 * K / 2 bytes; padding rows written as 0).
 * rows >= 0, 128 <= K <= 16384, K % 128 == 0; Q, T 16-byte aligned.
 * Errors: OQ_ERR_NULL, OQ_ERR_SHAPE, OQ_ERR_ALIGN, OQ_ERR_DEVICE, OQ_ERR_HIP.
 */
int oq_codes_to_tiled(const uint8_t* Q, int64_t rows, int64_t K, uint8_t* T, void* stream);

/*
 * oq_rotate_quantize_act_tiled -- oq_rotate_quantize_act (the same rotation,
 * step scale and quantizer, identical codes and x_scale) writing the codes
 * in the tiled layout: Xt device, R16 * K / 2 bytes with R = M (padding rows
 * are left untouched).  Additionally K % 128 == 0.  Arguments and errors as
 * oq_rotate_quantize_act.
 */
int oq_rotate_quantize_act_tiled(const void* X, int64_t M, int64_t K, int64_t ldx,
                                 int32_t had_block, const float* s_table, int32_t t,
                                 uint8_t* Xt, float* x_scale, void* stream);

/*
 * oq_w4a4_linear_tiled / oq_w4a4_gemm_i32_tiled -- oq_w4a4_linear and
 * oq_w4a4_gemm_i32 (same results, bit for bit) with the token codes Xt in the
 * tiled layout (R = M); Wq stays [N][K/2].  Additionally K % 128 == 0.  Meant
 * for M <= 64; larger M is computed correctly in row groups of 64 but
 * without the large-tile kernel of the row-layout calls.  Arguments and
 * errors as the row-layout calls.
 */
int oq_w4a4_linear_tiled(const uint8_t* Xt, const float* x_scale, int64_t M,
                         const uint8_t* Wq, const float* w_scale, const void* bias,
                         int64_t N, int64_t K, void* Y, int64_t ldy, int32_t out_dtype,
                         void* stream);
int oq_w4a4_gemm_i32_tiled(const uint8_t* Xt, int64_t M, const uint8_t* Wq, int64_t N,
                           int64_t K, int32_t* acc, int64_t ldc, void* stream);

/*
 * Full composite rotation (Section 4.1, "Block-wise Implementation";
 * eq:blockdiag, eq:transform) with block size c = 64: X' = X P R_hat, where
 * P permutes the channels (zigzag over the blocks by descending weight
 * energy) and R_hat = BlockDiag(R_1 .. R_{K/64}), R_b = U_b H_64 / 8, U_b the
 * left singular vectors of the block's weight rows.  Unlike the entry points
 * above (whose input is already in the SVD basis, so only the Hadamard half
 * runs online), the whole transform runs online here.
 *
 * oq_rotate_quantize_act_composite -- for each row i:
 *   (X P)[i][k] = X[i][perm[k]];  y[i][64b + j] = sum_r (X P)[i][64b + r] R_b[r][j];
 *   z = s_t y;  Delta_i = max|z| / 7;  q = round_half_even(z / Delta_i)
 *   (|q| <= 7);  x_scale[i] = Delta_i / s_t.
 * X        device fp16 [M][ldx], ldx >= K, ldx % 8 == 0, 16-byte aligned
 * K        multiple of 64, 64 <= K <= 16384
 * perm     device int32 [K], a permutation of 0 .. K-1, 16-byte aligned
 *          (entries outside 0 .. K-1 are clamped into range; the result is
 *          then unspecified but every access stays in bounds); or NULL: X is
 *          already in the permuted channel order (P folded into the
 *          producer of X, as U is for the Hadamard path), so (X P) = X and
 *          the rows go straight from global memory into the matrix-core
 *          operands without a gather
 * Rt       device fp16 [K/64][64][64], block b column-major:
 *          Rt[b][j][r] = R_b[r][j] (oq_block_rotations_host writes it), 16-byte
 *          aligned.  The products are formed from these fp16 values exactly
 *          and summed in fp32.
 * s_table, t  as oq_rotate_quantize_act
 * Xq       device [M][K/2] codes (16-byte aligned), x_scale device fp32 [M]
 * Device memory: above K = 4096 (and at K = 4096 with perm NULL and M > 1024)
 * the rows are split into channel chunks whose workgroups exchange their
 * partial row maxima through a library-owned device buffer (the inverse
 * permutation and one float per row and chunk), allocated on the first call
 * on a GPU, grown when a call needs more and kept until the process ends.
 * Such calls therefore may allocate, and calls that overlap on one GPU (other
 * streams, other host threads) share that buffer and must not run
 * concurrently.  A token scale written as NaN reports that a chunk's
 * exchange did not complete (never expected; the codes of that row are then
 * unspecified).
 * Errors: OQ_ERR_NULL, OQ_ERR_SHAPE, OQ_ERR_ALIGN, OQ_ERR_ARG, OQ_ERR_DEVICE,
 * OQ_ERR_HIP.
 */
int oq_rotate_quantize_act_composite(const void* X, int64_t M, int64_t K, int64_t ldx,
                                     const int32_t* perm, const void* Rt, const float* s_table,
                                     int32_t t, uint8_t* Xq, float* x_scale, void* stream);

/*
 * oq_zigzag_permutation_host -- perm (host int32 [K]) from per-channel weight
 * energies ||W_{j,:}||^2 (host double [K]; for a weight stored [N][K] the sum
 * of squares of column j): channels sorted by descending energy (ties keep
 * the lower index first) and dealt to the K / block blocks in snake order --
 * sorted position i goes to round r = i / n_blocks and block i % n_blocks
 * (r even) or n_blocks - 1 - i % n_blocks (r odd), slot r; perm[b block + r]
 * is that channel.  Errors: OQ_ERR_NULL, OQ_ERR_SHAPE.
 */
int oq_zigzag_permutation_host(const double* energy, int64_t K, int32_t block, int32_t* perm);

/*
 * oq_block_rotations_host -- Rt (host fp16 [K/block][block][block], each block
 * column-major) = round_to_fp16(U_b H_block / sqrt(block)) from the row-major
 * host double factors U [K/block][block][block].  block a power of two
 * <= 4096 dividing K (the online kernel takes block 64).
 * Errors: OQ_ERR_NULL, OQ_ERR_SHAPE.
 */
int oq_block_rotations_host(const double* U, int64_t K, int32_t block, uint16_t* Rt);

/*
 * oq_quantize_weights_composite_host -- the weight side of eq:transform in the
 * output-major storage: W'[n] = (W[n] P) R_hat with the fp16 block matrices
 * Rt as given (the same values the activation side uses), in float64, then
 * per-output-channel RTN (eq:scale, eq:quant): Wq host [N][K/2], w_scale host
 * fp32 [N].  W_u host double [N][K] row-major, perm host int32 [K], Rt host
 * fp16 as above.  Runs on the calling thread's process (std::thread workers).
 * Errors: OQ_ERR_NULL, OQ_ERR_SHAPE, OQ_ERR_ARG (perm entry out of range).
 */
int oq_quantize_weights_composite_host(const double* W_u, int64_t N, int64_t K, int32_t block,
                                       const int32_t* perm, const uint16_t* Rt, uint8_t* Wq,
                                       float* w_scale);

/*
 * oq_quantize_weights -- offline weight preparation on the device: fold the
 * Hadamard half of the rotation into the weight and quantize it per output
 * channel with round-to-nearest (eq:transform W' = R^T W in the output-major
 * storage used here: row n of W' is row n of W_u times blockdiag(H_b)/sqrt(b);
 * eq:scale / eq:quant per output channel; the DiT-side RTN solver of the
 * Implementation Details).  W_u is the weight already expressed in the SVD
 * basis (the SVD factor folded offline), device fp16 [N][ldw].  Identical to
 * oq_rotate_quantize_act with s_t = 1 applied to the weight rows; writes Wq
 * [N][K/2] and w_scale [N].  Shapes, alignment and errors as
 * oq_rotate_quantize_act.
 */
int oq_quantize_weights(const void* W_u, int64_t N, int64_t K, int64_t ldw,
                        int32_t had_block, uint8_t* Wq, float* w_scale, void* stream);

/*
 * oq_quantize_weights_host -- the same weight preparation on the host in
 * float64 from a float64 weight (for weights that are not fp16-exact).
 * W_u host [N][K] row-major; Wq host [N][K/2]; w_scale host fp32 [N].
 * Runs synchronously on the calling thread.  Errors: OQ_ERR_NULL,
 * OQ_ERR_SHAPE.
 */
int oq_quantize_weights_host(const double* W_u, int64_t N, int64_t K, int32_t had_block,
                             uint8_t* Wq, float* w_scale);

/* ------------------------------------------------------------------------ */
/* Offline preparation of the composite-rotation weight on the GPU           */
/* (Section 4.1: zigzag P, per-block SVD factor U_b, R_b = U_b H_64 / 8,      */
/* fold and RTN)                                                              */
/* ------------------------------------------------------------------------ */
/*
 * The weight W is device fp16 [N][ldw] (row n = output channel n, K input
 * channels); block b is input channels perm[64 b .. 64 b + 63].  The steps
 * can be called one by one or through oq_prepare_weights_composite.
 *
 * oq_channel_energy -- energy[j] = sum_n W[n][j]^2 in fp64 (device [K]); a
 *   fixed summation order, so equal columns give equal energies.
 *   Errors: OQ_ERR_NULL, OQ_ERR_SHAPE, OQ_ERR_ALIGN, OQ_ERR_DEVICE, OQ_ERR_HIP.
 *
 * oq_zigzag_permutation -- perm (device int32 [K]) from device energies: the
 *   descending order of the energy (ties to the lower channel index) dealt
 *   to K / block blocks in snake order: sorted position i goes to round
 *   r = i / n_b and to block i mod n_b on even rounds, n_b - 1 - (i mod n_b)
 *   on odd rounds, slot r; perm[b * block + r] is the source channel.
 *   K % block == 0, K <= 65536.
 *
 * oq_block_svd -- for each block (block must be 64): U (device fp64
 *   [K/64][64][64], row-major, U_b[r][i]) holds the left singular vectors of
 *   W_b (64 x N, the block's input-channel rows) as columns, ordered by
 *   descending singular value (ties to the lower index), each column's
 *   largest-magnitude entry (the first on ties) positive; sigma2 (device fp64
 *   [K/64][64]) the squared singular values.  Computed as the eigenvectors of
 *   the fp64 Gram matrix W_b W_b^T by cyclic Jacobi in fp64; vectors of
 *   (numerically) repeated singular values, including a null space when
 *   N < 64, are an orthonormal basis of their eigenspace, not unique.
 *   perm entries out of [0, K) are clamped.
 *
 * oq_block_rotations -- Rt (device fp16 [K/64][64][64], column-major blocks:
 *   Rt[b][j][r] = R_b[r][j]) with R_b = U_b H_64 / 8 evaluated in fp64 and
 *   rounded once to fp16 (half to even): the operand of
 *   oq_rotate_quantize_act_composite.
 *
 * oq_prepare_weights_composite -- all of the above, then the fold and RTN:
 *   Wq, w_scale = oq_rotate_quantize_act_composite(W, perm, Rt) with s_t = 1
 *   (the weight rows rotated by P R_hat and quantized per output channel).
 *   perm device int32 [K]; Rt device [K/64][64][64] fp16, 16-byte aligned;
 *   Wq device [N][K/2]; w_scale device fp32 [N]; work device, 16-byte
 *   aligned, at least oq_prepare_weights_workspace_bytes(K) = 528 K bytes.
 *   ldw % 8 == 0 and W 16-byte aligned (the fold's row loads).
 *   Errors: OQ_ERR_NULL, OQ_ERR_SHAPE (K % 64, K > 16384, workspace),
 *   OQ_ERR_ALIGN, OQ_ERR_DEVICE, OQ_ERR_HIP.
 */
int oq_channel_energy(const void* W, int64_t N, int64_t K, int64_t ldw, double* energy,
                      void* stream);
int oq_zigzag_permutation(const double* energy, int64_t K, int32_t block, int32_t* perm,
                          void* stream);
int oq_block_svd(const void* W, int64_t N, int64_t K, int64_t ldw, const int32_t* perm,
                 int32_t block, double* U, double* sigma2, void* stream);
int oq_block_rotations(const double* U, int64_t K, int32_t block, uint16_t* Rt, void* stream);
size_t oq_prepare_weights_workspace_bytes(int64_t K);
int oq_prepare_weights_composite(const void* W, int64_t N, int64_t K, int64_t ldw,
                                 int32_t* perm, uint16_t* Rt, uint8_t* Wq, float* w_scale,
                                 void* work, size_t work_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* W4A8: 8-bit per-token activations against the int4 weights (the paper's   */
/* deployment mode, Appendix: W4A8 real-quantization latency)                */
/* ------------------------------------------------------------------------ */
/*
 * oq_rotate_quantize_act_i8 -- oq_rotate_quantize_act with the symmetric
 * quantizer at 8 bits (eq:scale, eq:quant with k = 8): Delta_i = max|z_i| /
 * 127, codes in [-127, 127] (-128 never occurs), one signed byte per code.
 * Xq8 device int8 [M][K] row-major, 16-byte aligned; x_scale as before.
 * Arguments, limits and errors as oq_rotate_quantize_act.
 */
int oq_rotate_quantize_act_i8(const void* X, int64_t M, int64_t K, int64_t ldx,
                              int32_t had_block, const float* s_table, int32_t t,
                              int8_t* Xq8, float* x_scale, void* stream);

/*
 * oq_w4a8_linear / oq_w4a8_gemm_i32 -- oq_w4a4_linear / oq_w4a4_gemm_i32 with
 * the token operand in 8-bit codes (Xq8 [M][K], as written by
 * oq_rotate_quantize_act_i8) and the weight unchanged (packed int4 [N][K/2]):
 * acc[i][n] = sum_k q8[i][k] * wq[n][k] exactly in int32 (|acc| <= 889 K),
 * then the same epilogue.  Shapes, alignment and errors as the W4A4 calls.
 */
int oq_w4a8_linear(const int8_t* Xq8, const float* x_scale, int64_t M,
                   const uint8_t* Wq, const float* w_scale, const void* bias,
                   int64_t N, int64_t K, void* Y, int64_t ldy, int32_t out_dtype,
                   void* stream);
int oq_w4a8_gemm_i32(const int8_t* Xq8, int64_t M, const uint8_t* Wq, int64_t N, int64_t K,
                     int32_t* acc, int64_t ldc, void* stream);

/* ------------------------------------------------------------------------ */
/* Static per-step, per-channel activation steps (Section 4.2,               */
/* eq:perstep_scale with the per-(layer, step, channel) table)               */
/* ------------------------------------------------------------------------ */
/*
 * The table holds Delta_{l,t,j} = sigma_hat(X'_{t,:,j}) / q_max for the
 * rotated activation X' of layer l at denoising step t, sigma_hat the
 * nearest-rank 99.9th percentile of the magnitudes over the calibration rows.
 * At inference the codes are q = clamp(round(y_j / Delta_j), -7, 7) (clipping
 * is live; round half to even) and the token scale is 1.  A per-channel step
 * cannot leave the sum over channels, so it is folded into the weight's input
 * channels per step: W''[n][j] = W'[n][j] Delta_j, quantized per output
 * channel (one weight copy per (layer, step)); the products are then the
 * ordinary oq_w4a4_linear / _tiled calls with x_scale = 1.
 */

/*
 * oq_rotate_act_f32 -- the rotated activation of eq:transform alone:
 * Y[i][k] = (x_i H_b / sqrt(b))[k] in fp32, Y device [M][K] contiguous,
 * 16-byte aligned (the calibration input of oq_calibrate_step_scales).
 * Arguments and shape limits as oq_rotate_quantize_act.  Errors: OQ_ERR_NULL,
 * OQ_ERR_SHAPE, OQ_ERR_ALIGN, OQ_ERR_DEVICE, OQ_ERR_HIP.
 */
int oq_rotate_act_f32(const void* X, int64_t M, int64_t K, int64_t ldx, int32_t had_block,
                      float* Y, void* stream);

/*
 * oq_calibrate_workspace_bytes -- device workspace needed by
 * oq_calibrate_step_scales for K channels (K * 1032 bytes).
 */
size_t oq_calibrate_workspace_bytes(int64_t K);

/*
 * oq_calibrate_step_scales -- delta[j] = v_j / qmax, v_j the nearest-rank
 * p-th percentile of |Y[:, j]| over the n rows: the k-th smallest magnitude
 * with k = ceil(p n / 100) clamped to [1, n], p taken to 1e-6 percent and
 * the product formed in integers (p = 99.9, n = 1000 gives k = 999, not the
 * maximum).  v_j is exact (an element of the column; selection over the bit
 * patterns, NaN ordered above +inf); the division is done in double and
 * rounded once to fp32.
 * Y device fp32 [n][ldy]; delta device fp32 [K]; work device, 16-byte
 * aligned, at least oq_calibrate_workspace_bytes(K) bytes, owned by the
 * caller and overwritten (calls that share it must not overlap).
 * p in (0, 100]; qmax > 0 (7 for int4 codes).
 * Errors: OQ_ERR_NULL, OQ_ERR_SHAPE (n == 0 with K > 0, ldy < K, workspace
 * too small), OQ_ERR_ARG (p, qmax), OQ_ERR_ALIGN, OQ_ERR_DEVICE, OQ_ERR_HIP.
 */
int oq_calibrate_step_scales(const float* Y, int64_t n, int64_t K, int64_t ldy, double p,
                             float qmax, float* delta, void* work, size_t work_bytes,
                             void* stream);

/*
 * oq_calibrate_step_scales_noalloc -- for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc): the same computation and results as
 * oq_calibrate_step_scales, bit for bit, with no workspace argument.  The
 * histogram, prefixes and ranks live in a device array inside the library
 * (16.9 MB per GPU, held until the process ends; its address is looked up
 * once per device on the first call with that device current).  The call
 * allocates nothing and clears what must start at zero with a kernel.
 * K <= 16384 columns; a larger K returns OQ_ERR_WORKSPACE and writes nothing.
 * The stream must belong to the current device.  Every call on one GPU
 * shares that GPU's array: calls that overlap on one GPU (other streams or
 * threads) race and must be serialized by the caller.
 * Errors: as oq_calibrate_step_scales, and OQ_ERR_WORKSPACE for K > 16384.
 */
int oq_calibrate_step_scales_noalloc(const float* Y, int64_t n, int64_t K, int64_t ldy, double p,
                                     float qmax, float* delta, void* stream);

/*
 * oq_rotate_quantize_act_static -- Hadamard rotation (as
 * oq_rotate_quantize_act) followed by the static quantizer with the step row
 * delta (device fp32 [K], 16-byte aligned: the table's row for this layer
 * and step): Xq[i][k] = clamp(round(y_ik / delta[k]), -7, 7), x_scale[i] = 1.
 * A channel whose step is zero, negative, NaN or infinite gets code 0.  The
 * ratio is formed in fp32 with the hardware reciprocal of delta (about one
 * ulp), so only ratios within a few ulps of a half integer can round
 * differently from exact arithmetic.
 * Errors: as oq_rotate_quantize_act; OQ_ERR_NULL (delta), OQ_ERR_ALIGN.
 */
int oq_rotate_quantize_act_static(const void* X, int64_t M, int64_t K, int64_t ldx,
                                  int32_t had_block, const float* delta, uint8_t* Xq,
                                  float* x_scale, void* stream);

/* The same with the codes in the 16-row tiled layout (K % 128 == 0). */
int oq_rotate_quantize_act_static_tiled(const void* X, int64_t M, int64_t K, int64_t ldx,
                                        int32_t had_block, const float* delta, uint8_t* Xt,
                                        float* x_scale, void* stream);

/*
 * oq_quantize_weights_step_host -- oq_quantize_weights_host with the step
 * folded in: row n of the quantized weight is RTN(W'[n][:] * delta[:]),
 * W' = W_u rotated by H_b / sqrt(b), in float64.  delta host fp32 [K], every
 * entry finite and >= 0.  Errors: OQ_ERR_NULL, OQ_ERR_SHAPE, OQ_ERR_ARG.
 */
int oq_quantize_weights_step_host(const double* W_u, int64_t N, int64_t K, int32_t had_block,
                                  const float* delta, uint8_t* Wq, float* w_scale);

/*
 * oq_quantize_weights_step -- the same fold on the device from an fp16
 * weight (as oq_quantize_weights, with channel j of each rotated row
 * multiplied by delta[j] before the row's maximum), in fp32.  delta device
 * fp32 [K], 16-byte aligned.  Errors: as oq_quantize_weights; OQ_ERR_NULL
 * (delta), OQ_ERR_ALIGN.
 */
int oq_quantize_weights_step(const void* W_u, int64_t N, int64_t K, int64_t ldw, int32_t had_block,
                             const float* delta, uint8_t* Wq, float* w_scale, void* stream);

/* ------------------------------------------------------------------------ */
/* DiT denoising-step driver                                                 */
/* ------------------------------------------------------------------------ */

/*
 * One denoising step of a DiT action head whose every block linear is a
 * rotated W4A4 linear (Experimental Settings: W4A4 on all linears, RTN
 * weights and the per-step activation scale table on the DiT side, Euler
 * denoising steps).  Block structure, arch OQ_DIT_PI (Pi-0.5 action expert):
 *
 *   r   = x_t . W_in^T + b_in                                (fp32 residual)
 *   per block l, step t (modulation m = mod[l][t], scales s = s_table[l][t]):
 *     h   = fp16(rms(r) * g1 * (1 + m.sc1) + m.sh1)
 *     qkv = fp16(W4A4(h; Wqkv, s[0]))                        q|k|v along N
 *     o   = fp16(softmax(q k^T / sqrt(hd)) v) per head, keys = [prefix ; k]
 *     r  += m.gt1 * W4A4(o; Wo, s[1])
 *     h2  = fp16(rms(r) * g2 * (1 + m.sc2) + m.sh2)
 *     gu  = fp16(W4A4(h2; Wgu, s[2]))                        gate|up along N
 *     a   = fp16(gelu_tanh(gate) * up)
 *     r  += m.gt2 * W4A4(a; Wd, s[3])
 *   v   = fp16(rms(r) * g_f) . W_out^T + b_out ;  x_{t+1} = x_t + dt * v
 *
 * Arch OQ_DIT_GR00T (GR00T-N1.5 DiT; the Appendix on per-step scaling names
 * AdaLayerNorm -> attention q/k/v -> ... -> LayerNorm -> ff.net[0] -> GELU ->
 * ff.net[2]):
 *
 *   per block l, step t (m = mod[l][t], s = s_table[l][t]):
 *     h   = fp16(ln(r) * g1 * (1 + m.sc1) + m.sh1)           AdaLayerNorm
 *     even l (cross-attention):  q = fp16(W4A4(h; Wq, s[0])),
 *            k|v = fp16(W4A4(cond; Wkv, 1)) per sample, from
 *            oq_dit_set_condition (step-invariant, computed once)
 *     odd l (self-attention):    q|k|v = fp16(W4A4(h; Wqkv, s[0]))
 *     o   = fp16(softmax(q k^T / sqrt(hd)) v) per head and sample
 *     r  += W4A4(o; Wo, s[1])
 *     h2  = fp16(ln(r) * g2 + b2)                            LayerNorm
 *     f   = fp16(gelu_tanh(W4A4(h2; Wff0, s[2])))
 *     r  += W4A4(f; Wff2, s[3])
 *   v   = fp16(ln(r) * g_f) . W_out^T + b_out ;  x_{t+1} = x_t + dt * v
 *
 * rms(r) = r / sqrt(mean(r^2) + 1e-6), ln(r) = (r - mean) / sqrt(var + 1e-6),
 * dt = -1/steps (pi, tau 1 -> 0) or +1/steps (gr00t, tau 0 -> 1), the Hadamard
 * block of a linear is the largest power of two dividing its input size.
 */
typedef enum { OQ_DIT_PI = 0, OQ_DIT_GR00T = 1 } oq_dit_arch;

typedef struct {
  int32_t arch;        /* oq_dit_arch                                        */
  int32_t n_blocks;    /* >= 1                                               */
  int32_t hidden;      /* D, multiple of 64, <= 8192; = n_heads * head_dim  */
  int32_t mlp;         /* F, multiple of 64                                  */
  int32_t n_heads;
  int32_t head_dim;    /* <= 128, multiple of 16                             */
  int32_t tokens;      /* S action tokens per sample, <= 64                  */
  int32_t prefix;      /* pi: P prefix tokens per sample (keys before the S
                          own); gr00t: P conditioning tokens per sample      */
  int32_t batch;       /* B samples                                          */
  int32_t steps;       /* T denoising steps                                  */
  int32_t action_dim;  /* A, multiple of 8                                   */
} oq_dit_config;

/* A prepared W4A4 weight: device Wq [N][K/2] and w_scale fp32 [N]. */
typedef struct {
  const uint8_t* wq;
  const float* w_scale;
} oq_qweight;

/* Per-block device pointers (borrowed; the caller keeps them alive until
 * oq_dit_destroy).  All vectors fp16. */
typedef struct {
  const void* g1;          /* [D] norm gain before attention                   */
  const void* g2;          /* [D] norm gain before the MLP                     */
  oq_qweight qkv;          /* pi and odd gr00t blocks: q|k|v, N = 3D, K = D;
                              even gr00t blocks: q only, N = D, K = D          */
  oq_qweight o;            /* N = D,  K = D                                    */
  oq_qweight gate_up;      /* pi: gate|up, N = 2F; gr00t: ff0, N = F; K = D    */
  oq_qweight down;         /* N = D,  K = F                                    */
  const void* prefix_k;    /* pi: [B][P][D] fp16, step-invariant; gr00t: NULL  */
  const void* prefix_v;    /* pi: [B][P][D] fp16; gr00t: NULL                  */
  const void* b2;          /* gr00t: [D] LayerNorm bias before the MLP; pi: NULL */
  oq_qweight cross_kv;     /* even gr00t blocks: k|v of the conditioning
                              tokens, N = 2D, K = D; otherwise NULL            */
} oq_dit_block;

typedef struct {
  const void* w_in;        /* fp16 [D][A]                                      */
  const void* b_in;        /* fp16 [D]                                         */
  const void* w_out;       /* fp16 [A][D]                                      */
  const void* b_out;       /* fp16 [A]                                         */
  const void* g_f;         /* fp16 [D] final norm gain                         */
  const oq_dit_block* blocks; /* host array [n_blocks], copied by oq_dit_create */
  const void* mod;         /* fp16 device [n_blocks][steps][NM][D] per-step
                              modulation; pi: NM = 6 (sc1, sh1, gt1, sc2, sh2,
                              gt2), gr00t: NM = 2 (sc1, sh1)                   */
  const float* s_table;    /* host fp32 [n_blocks][steps][4], copied           */
} oq_dit_weights;

typedef struct oq_dit oq_dit;

/* Workspace size in bytes for a config (device memory the caller provides). */
int oq_dit_workspace_bytes(const oq_dit_config* cfg, size_t* bytes);

/* Validate cfg and weights and create a handle (host memory only).
 * Errors: OQ_ERR_NULL, OQ_ERR_SHAPE, OQ_ERR_ARG, OQ_ERR_DEVICE. */
int oq_dit_create(const oq_dit_config* cfg, const oq_dit_weights* w, oq_dit** out);

/* Attach caller-owned device workspace (256-byte aligned, at least
 * oq_dit_workspace_bytes).  With more than 64 action rows (batch * tokens)
 * the workspace ends in the split-K scratch of the deep block linears: 16 MB
 * of int32 partial tiles and 512 arrival tickets, which this call zeroes
 * synchronously (hipMemset; every later linear leaves them zero).  Calls of
 * one handle must not overlap in time (they share the workspace).
 * Errors: OQ_ERR_NULL, OQ_ERR_WORKSPACE, OQ_ERR_ALIGN, OQ_ERR_HIP. */
int oq_dit_set_workspace(oq_dit* h, void* workspace, size_t bytes);

/* gr00t: compute every cross-attention block's conditioning k|v from cond
 * (device fp16 [B][P][D], read during the call only) into the workspace:
 * rotate-quantize with s = 1 and the W4A4 k|v linear, once per conditioning
 * input (it does not depend on the step).  Required before the first step
 * of a gr00t handle and again whenever the conditioning or the workspace
 * changes.  Errors: OQ_ERR_NULL, OQ_ERR_WORKSPACE, OQ_ERR_ARG (pi handle),
 * OQ_ERR_HIP. */
int oq_dit_set_condition(oq_dit* h, const void* cond, void* stream);

/* One Euler step t (0 <= t < steps) on x (device fp32 [B][S][A], in place).
 * Errors: OQ_ERR_NULL, OQ_ERR_WORKSPACE, OQ_ERR_ARG (bad t, or a gr00t handle
 * without a condition), OQ_ERR_HIP. */
int oq_dit_step(oq_dit* h, float* x, int32_t t, void* stream);

/* n_steps consecutive steps t = 0 .. n_steps-1 on x, in place. */
int oq_dit_denoise(oq_dit* h, float* x, int32_t n_steps, void* stream);

/* Run block l of step t alone on a residual (device fp32 [B*S][D], in place);
 * for per-block parity checks with a teacher-forced input. */
int oq_dit_run_block(oq_dit* h, int32_t l, int32_t t, float* resid, void* stream);

/* Parity check of the fused producers (each writes a linear's fp16 input and
 * quantizes it in the same kernel, eq:scale / eq:quant after the rotation of
 * eq:blockdiag): run block l of step t only up to and including the producer
 * of quantization site `site` (0: the q|k|v (q) input, 1: the o input, 2:
 * the gate|up (ff0) input, 3: the down (ff2) input).  That site's codes and
 * token scales are then in the workspace (oq_dit_intermediates.codes,
 * .x_scale).  Errors: as oq_dit_run_block; OQ_ERR_ARG for a bad site. */
int oq_dit_run_block_until(oq_dit* h, int32_t l, int32_t t, float* resid, int32_t site, void* stream);

/* Static per-step, per-channel steps inside the driver (eq:perstep_scale with
 * the per-(layer, step, channel) table; the scalar s_t of oq_dit_weights is
 * then unused for the four block sites).  delta: device fp32
 * [n_blocks][steps][3 D + F], 16-byte aligned: for block l and step t the step
 * rows of the q|k|v (q) input [D], the o input [D], the gate|up (ff0) input
 * [D] and the down (ff2) input [F], in that order.  step_weights: host array
 * [n_blocks][steps][4] of the same four linears folded with their step rows
 * (oq_quantize_weights_step: W''[n][j] = W'[n][j] Delta_j, RTN per output
 * channel), device pointers borrowed until the mode is cleared.  Each site's
 * producer then writes codes clamp(round(y_j / Delta_j), +-7) with token
 * scale 1 and each linear uses its step's folded weight.  delta = NULL
 * returns the handle to the per-token quantizer.  The array is copied; the
 * captured steps are dropped.  Not for the gr00t conditioning k|v linear
 * (step-invariant, computed once).  Errors: OQ_ERR_NULL, OQ_ERR_ALIGN. */
int oq_dit_set_static_steps(oq_dit* h, const float* delta, const oq_qweight* step_weights);

/* The step's in-projection alone: resid [M][D] fp32 = x W_in^T + b_in (the
 * residual at the input of block 0), for a caller that runs blocks one by
 * one (calibration rollouts).  Errors: OQ_ERR_NULL, OQ_ERR_ALIGN, OQ_ERR_HIP. */
int oq_dit_in_projection(oq_dit* h, const float* x, float* resid, void* stream);

/* The last stage of a step alone, on a caller residual (device fp32 [M][D],
 * 16-byte aligned, read only): v = fp16(norm(resid) g_f) W_out^T + b_out and
 * the Euler update x += dt v with dt = -1/T (pi) or +1/T (gr00t), x device
 * fp32 [B][S][A] in place (Experimental Settings: T Euler steps).  With
 * oq_dit_in_projection and oq_dit_run_block it rebuilds a step from its
 * parts, for checking oq_dit_step against them bit for bit.
 * Errors: OQ_ERR_NULL, OQ_ERR_ALIGN, OQ_ERR_HIP. */
int oq_dit_final_stage(oq_dit* h, const float* resid, float* x, void* stream);

/* Intermediate tensors of the most recent block the handle ran (fp16,
 * row-major, M = batch * tokens rows), for per-site parity checks: every
 * quantized linear's fp16 input and every fp16 output of the block can be
 * compared with the oracle fed the GPU's own upstream values.  Pointers into
 * the workspace, valid until the next call on the handle.  The fp16 linear
 * inputs h1, attn, h2 and act are written by oq_dit_run_block and
 * oq_dit_run_block_until only (oq_dit_step and oq_dit_denoise produce their
 * codes without storing them; gr00t's cross-attention output, which its
 * quantizer reads back, is the exception). */
typedef struct {
  const void* h1;        /* [M][D]  norm output, input of the q|k|v (q) linear  */
  const void* qkv;       /* [M][3D] q|k|v linear output (gr00t even: q, [M][D]) */
  const void* attn;      /* [M][D]  attention output, input of the o linear      */
  const void* h2;        /* [M][D]  norm output, input of the gate|up / ff0 linear */
  const void* gate_up;   /* pi: [M][2F] gate|up output; gr00t: not written (the
                            ff0 linear applies the GELU in its epilogue and
                            writes act directly)                              */
  const void* act;       /* [M][F]  input of the down / ff2 linear               */
  const float* resid;    /* [M][D]  fp32 residual of the last oq_dit_step after
                            its last block (oq_dit_run_block uses the caller's) */
  const void* cond_kv;   /* gr00t: k|v of the conditioning tokens of every
                            even block, head-major [n_blocks/2 rounded up][B]
                            [H][2 (k, v)][P][head_dim]; pi: NULL              */
  const void* codes;     /* packed codes of the last quantization site the
                            handle produced (its fp16 input is h1, attn, h2 or
                            act): [M][K/2], or the 16-row tiled layout when
                            codes_tiled is 1                                  */
  const float* x_scale;  /* [M] token scales of the same site                 */
  int32_t codes_tiled;   /* 1: codes in the 16-row tiled layout (M <= 64)      */
} oq_dit_intermediates;

/* Fill *out with the intermediate pointers.  Errors: OQ_ERR_NULL, OQ_ERR_WORKSPACE. */
int oq_dit_get_intermediates(const oq_dit* h, oq_dit_intermediates* out);

/* Free the handle (not the borrowed weights or the workspace). NULL is a no-op. */
void oq_dit_destroy(oq_dit* h);

#ifdef __cplusplus
}
#endif

#endif /* OQ_H */
