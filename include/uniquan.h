/*
 * uniquan.h -- C ABI of the MI355X (gfx950) UniQuan_F fake-quant library.
 *
 * UniQuan_F (arXiv 2506.03781) quantizes each group of g weights of a weight
 * matrix with the unified quantizer of Eq. (3):
 *     what = D_R( M*_B( T_F(w) ) )
 * T_F   flexible-mapping transform, Eq. (1):  wbar = w / (Delta * s * s_r) + z_U
 * M*_B  nearest binary-coding level z_B + sum_i c_i alpha_i, c in {-1,+1}^k
 *       (Sec. 2.3), with the local and periodic mapping of the appendix
 *       algorithm "Local and periodic mapping"
 * D_R   detransform:                          what = Delta * (wtilde - z_U)
 * and trains Delta, z_U, s, s_r, alpha, z_B by straight-through
 * backpropagation of the reconstruction loss ||X W^T - X What^T||_F^2
 * (Algorithm 1), with the gradient filter of the appendix "Implementation
 * details".  After training, Theorem 1 folds the parameters into plain
 * binary-coding ones and Eq. (4) extracts the deployable codes.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Memory.   Every pointer is DEVICE memory owned by the caller.  The library
 *           never allocates, frees or keeps a pointer after returning.
 * Streams.  `stream` is a hipStream_t passed as void* (NULL = default
 *           stream).  Calls only enqueue work and return; results are ready
 *           when the stream reaches them.  Calls on one stream are ordered;
 *           concurrent calls writing the same buffers race.
 * Layout.   Weight-shaped arrays are [R x C] row-major (R output channels,
 *           C input features).  A group is g contiguous weights of one row:
 *           group id gid = r * (C / g) + c / g, Gn = R * C / g groups.
 *           Per-group arrays are [Gn]; alpha is [Gn x k] with
 *           alpha[gid * k + i] = alpha_{i+1}.
 * Codes.    One byte per weight.  Bits 0..k-1 hold the binary code
 *           (bit i set <=> c_{i+1} = +1); bit 7 holds the gradient-filter
 *           mask m (1 = gradient kept).  Bits k..6 are zero on output and
 *           ignored on input.
 * Dtypes.   UQ_F32 = IEEE binary32, UQ_BF16 = bfloat16 (uint16 storage).
 * Sizes.    R, C, T >= 1.  g divides C and is either a power of two in
 *           [8, 512] or a multiple of 8 above 512 (e.g. the per-row groups
 *           g = C of the paper's 7B / 8B settings, 4096, 11008 or 14336
 *           weights; one workgroup per group then).  The unified
 *           initialisation takes g <= 16384, the fused gradient-GEMM
 *           backward g <= 128.
 *           1 <= k <= 7.  T (calibration tokens) is a multiple of 8.
 * Alignment Per-weight arrays, X, Xt, Yt and workspaces: 16 bytes.
 *           Per-group and per-row arrays: 4 bytes.
 * Errors.   Every call returns a uq_status.  Arguments are checked on the
 *           host before any HIP call: UQ_EINVAL for a bad size, pointer,
 *           alignment or enum, UQ_EUNSUPPORTED for a valid but unsupported
 *           shape; nothing is enqueued then.  UQ_EHIP reports a failed
 *           launch.  uniquan_last_error() gives a text for the last failure
 *           on the calling thread.  Device-data preconditions are NOT
 *           checked: Delta, s, s_r > 0 and finite; W, X, alpha, z_B, z_U
 *           finite.
 * Numerics. Codes and masks are decided in IEEE binary32 with correctly
 *           rounded division, no contraction and subnormals kept, in the
 *           operation order stated at each entry point, so they are
 *           reproducible bit for bit by any IEEE implementation.
 */
#ifndef UNIQUAN_H
#define UNIQUAN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { UQ_OK = 0, UQ_EINVAL = 1, UQ_EUNSUPPORTED = 2, UQ_EHIP = 3 } uq_status;
typedef enum { UQ_F32 = 0, UQ_BF16 = 1 } uq_dtype;
typedef enum { UQ_MAP_FULL = 0, UQ_MAP_LOCAL = 1, UQ_MAP_FROZEN = 2 } uq_map_mode;

#define UNIQUAN_ABI_VERSION 3

/* ABI version of the loaded library (UNIQUAN_ABI_VERSION). */
int uniquan_abi_version(void);

/* Text describing the last non-OK status returned on this thread
 * (thread-local, valid until the next call on the thread). */
const char* uniquan_last_error(void);

/*
 * uniquan_fq_fwd -- quantizer forward Q*_{I_F}, Eq. (3).
 *
 * Per group: the 2^k levels q(b) = z_B + (+-alpha_1) + ... + (+-alpha_k)
 * (sign + iff bit i of b is set), summed left to right in fp32, sorted
 * ascending (equal values ordered by code).  Per weight:
 *     den  = (Delta * s_r) * s ;  wbar = (w / den) + z_U          [Eq. (1)]
 *     FULL   : the nearest sorted level; on equal distance the lower one
 *     LOCAL  : the nearest of the previous code's sorted position d and its
 *              neighbours max(d-1,0), min(d+1,2^k-1), lower one on ties
 *              (appendix algorithm "Local and periodic mapping")
 *     FROZEN : keep the previous code
 *     distance = |fl(wbar - q)|;  wtilde = q(code)
 *     m    = NOT(|fl(wbar - wtilde)| > tau),  tau = min_i |alpha_i|
 *     what = Delta * (wtilde - z_U)                                [D_R]
 * The level value is recomputed from the current alpha, z_B on every call;
 * only the code is kept between calls.
 *
 * W       [R*C] w_dtype               in
 * s       [R*C] fp32 element-wise scales (> 0)                      in
 * s_r     [R] fp32 row-wise scales, or NULL for 1                   in
 * delta   [Gn] fp32 (> 0), or NULL for 1                            in
 * z_u     [Gn] fp32, or NULL for 0                                  in
 * alpha   [Gn*k] fp32, z_b [Gn] fp32                                in
 * mode    uq_map_mode
 * codes   [R*C] uint8: previous codes in (LOCAL, FROZEN), new code|mask out
 * W_hat   [R*C] w_hat_dtype (bf16 rounds to nearest even)           out
 */
uq_status uniquan_fq_fwd(int64_t R, int64_t C, int k, int g,
                         const void* W, int w_dtype,
                         const float* s, const float* s_r,
                         const float* delta, const float* z_u,
                         const float* alpha, const float* z_b,
                         int mode, uint8_t* codes,
                         void* W_hat, int w_hat_dtype,
                         void* stream);

/*
 * uniquan_fq_fwd_residual -- uniquan_fq_fwd with the reconstruction residual
 * in place of the quantized weight:
 *     R_out[j] = fl(what[j] - w[j])   (what as uniquan_fq_fwd computes it in
 *                                      fp32; then rounded to r_dtype, RNE)
 * For one linear layer the reconstruction error is X What^T - X W^T =
 * X (What - W)^T (Algorithm 1's loss with X_hat = X), so feeding R_out to
 * uniquan_layer_recon with Yt = NULL gives the loss without the fp32 target,
 * and the small residual keeps more bits in bf16 than What does.  The
 * gradient with respect to What is unchanged.  Arguments, codes and errors
 * as for uniquan_fq_fwd; R_out [R*C] r_dtype out.
 */
uq_status uniquan_fq_fwd_residual(int64_t R, int64_t C, int k, int g,
                                  const void* W, int w_dtype,
                                  const float* s, const float* s_r,
                                  const float* delta, const float* z_u,
                                  const float* alpha, const float* z_b,
                                  int mode, uint8_t* codes,
                                  void* R_out, int r_dtype,
                                  void* stream);

/*
 * uniquan_fq_bwd -- straight-through backward of uniquan_fq_fwd with the
 * gradient filter (appendix "Implementation details": the mapping is
 * treated as identity, d wtilde / d wbar := m, zero where |wbar - wtilde|
 * exceeds tau = min alpha).  With G = dL/dWhat and g~ = Delta * G:
 *     grad_alpha[gid, i] = sum_j g~_j c_{i+1}(code_j)
 *     grad_z_b[gid]      = sum_j g~_j
 *     grad_s_j           = -m_j g~_j (wbar_j - z_U) / s_j
 *     grad_delta[gid]    = sum_j G_j ((wtilde_j - z_U) - m_j (wbar_j - z_U))
 *     grad_z_u[gid]      = -Delta sum_j (1 - m_j) G_j
 *     grad_s_r[r]        = -sum_{j in row r} m_j g~_j (wbar_j - z_U) / s_r
 * Sums over a group and over a row run in a fixed order (bitwise
 * reproducible run to run).
 *
 * W, s, s_r, delta, z_u, alpha, z_b  as for uniquan_fq_fwd           in
 * codes       [R*C] code|mask bytes written by uniquan_fq_fwd        in
 * grad_W_hat  [R*C] grad_dtype, dL/dWhat                            in
 * grad_s      [R*C] fp32                                  out (required)
 * grad_alpha  [Gn*k] fp32, grad_z_b [Gn] fp32             out (required)
 * grad_delta, grad_z_u [Gn] fp32; grad_s_r [R] fp32   out, NULL = skipped
 * group_ws    [Gn] fp32 workspace, required iff grad_s_r != NULL
 */
uq_status uniquan_fq_bwd(int64_t R, int64_t C, int k, int g,
                         const void* W, int w_dtype,
                         const float* s, const float* s_r,
                         const float* delta, const float* z_u,
                         const float* alpha, const float* z_b,
                         const uint8_t* codes,
                         const void* grad_W_hat, int grad_dtype,
                         float* grad_s, float* grad_alpha, float* grad_z_b,
                         float* grad_delta, float* grad_z_u, float* grad_s_r,
                         float* group_ws,
                         void* stream);

/*
 * uniquan_fq_bwd_sgd -- uniquan_fq_bwd (required gradients only) fused with
 * the stochastic gradient descent update of Algorithm 1 for the trained
 * parameters, in place and in the same pass over the weights:
 *     s     <- s     - lr_f * grad_s          (Theta_F learning rate)
 *     alpha <- alpha - lr_b * grad_alpha      (Theta_B learning rate)
 *     z_b   <- z_b   - lr_b * grad_z_b
 * Gradients are those of the parameters before the update; they are also
 * written to grad_s, grad_alpha, grad_z_b unless those are NULL (a caller
 * that only steps the parameters saves the 4 B per weight of grad_s).  Each
 * update is the fp32
 * expression theta - lr * grad, as uniquan_sgd computes it, so the result
 * equals uniquan_fq_bwd followed by three uniquan_sgd calls bit for bit.
 * Arguments as for uniquan_fq_bwd; s, alpha, z_b are in/out.
 */
uq_status uniquan_fq_bwd_sgd(int64_t R, int64_t C, int k, int g,
                             const void* W, int w_dtype,
                             float* s, const float* s_r,
                             const float* delta, const float* z_u,
                             float* alpha, float* z_b,
                             const uint8_t* codes,
                             const void* grad_W_hat, int grad_dtype,
                             float* grad_s, float* grad_alpha, float* grad_z_b,
                             float lr_f, float lr_b,
                             void* stream);

/*
 * uniquan_fq_step -- the end of one optimisation step and the start of the
 * next in one pass over the weights (Algorithm 1's update line, then its
 * quantization line for the next step): uniquan_fq_bwd_sgd with the codes'
 * mask bits and dL/dWhat of step t (s, alpha, z_b updated in place), then
 * uniquan_fq_fwd (residual == 0) or uniquan_fq_fwd_residual (residual == 1)
 * with next_mode on the updated parameters, writing W_hat and the new code
 * bytes.  The results equal those two calls bit for bit.  Per weight it reads
 * dL/dWhat, W, s and the code byte once (9 B with bf16 W and dL/dWhat) and
 * writes s, W_hat and the code byte (7 B), against 23 B for the two passes.
 * Runs as one kernel for g <= 512 (LOCAL mapping: where the neighbour table
 * fits, i.e. (512 / g) 2^k <= 4096) and, with bf16 W and dL/dWhat, for
 * groups of 513 to 16384 weights (one workgroup per group, every mapping);
 * otherwise as the two calls.  Arguments
 * and errors as for those calls; the gradient outputs are not stored.
 */
uq_status uniquan_fq_step(int64_t R, int64_t C, int k, int g,
                          const void* W, int w_dtype,
                          float* s, const float* s_r,
                          const float* delta, const float* z_u,
                          float* alpha, float* z_b,
                          uint8_t* codes,
                          const void* grad_W_hat, int grad_dtype,
                          float lr_f, float lr_b,
                          int next_mode, void* W_hat, int w_hat_dtype, int residual,
                          void* stream);

/*
 * uniquan_layer_target -- the fixed reconstruction target of one linear
 * layer, Y = X W^T (Algorithm 1, output of the unquantized layer), stored
 * transposed: Yt[r, t] = sum_c W[r, c] X[t, c], fp32 accumulation on bf16
 * MFMA.  Computed once per layer.
 *
 * X  [T*C] bf16;  W [R*C] bf16;  Yt [R*T] fp32 out.
 */
uq_status uniquan_layer_target(int64_t T, int64_t R, int64_t C,
                               const uint16_t* X, const uint16_t* W,
                               float* Yt, void* stream);

/*
 * uniquan_transpose_bf16 -- out[c, r] = in[r, c] for a [rows x cols] bf16
 * matrix (used once per layer to form Xt for the weight-gradient GEMM).
 * rows and cols are multiples of 8.
 */
uq_status uniquan_transpose_bf16(int64_t rows, int64_t cols,
                                 const uint16_t* in, uint16_t* out, void* stream);

/* Number of fp32 loss partials uniquan_layer_recon needs for (T, R, C). */
size_t uniquan_recon_ws(int64_t T, int64_t R, int64_t C);

/*
 * uniquan_layer_recon -- single-layer reconstruction loss of Algorithm 1
 * (the quantized layer sees the same input, X_hat = X) and its weight
 * gradient:
 *     Et[r, t]   = sum_c What[r, c] X[t, c] - Yt[r, t]      (fp32, stored bf16)
 *     loss       = sum_{r,t} Et[r, t]^2    (squared Frobenius norm, a sum)
 *     grad_W_hat = 2 Et Xt^T,  i.e. grad[r, c] = 2 sum_t Et[r, t] X[t, c]
 * Both contractions run on bf16 MFMA with fp32 accumulation.  The loss is
 * reduced from per-workgroup fp32 partials in fp64 in a fixed order.
 *
 * X           [T*C] bf16                                          in
 * Xt          [C*T] bf16 (transpose of X), NULL => forward only   in
 * W_hat       [R*C] bf16 (uniquan_fq_fwd output)                  in
 * Yt          [R*T] fp32 (uniquan_layer_target output), or NULL:  in
 *             then W_hat holds the residual What - W
 *             (uniquan_fq_fwd_residual) and Et = W_hat X^T
 * loss        [1] fp32                                            out
 * Et_ws       [R*T] bf16 workspace; holds Et after the call      out
 * partials_ws [partials_len] fp32, partials_len >= uniquan_recon_ws()
 * grad_W_hat  [R*C] grad_dtype, NULL => forward only              out
 */
uq_status uniquan_layer_recon(int64_t T, int64_t R, int64_t C,
                              const uint16_t* X, const uint16_t* Xt,
                              const uint16_t* W_hat, const float* Yt,
                              float* loss, uint16_t* Et_ws,
                              float* partials_ws, size_t partials_len,
                              void* grad_W_hat, int grad_dtype,
                              void* stream);

/*
 * uniquan_layer_recon_noalloc -- uniquan_layer_recon for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation): no partials workspace argument; the
 * loss partials live in a fixed array of the library's device memory, one
 * per GPU, held until the process ends.  Nothing is allocated or freed by
 * the call.  Same arguments (minus partials_ws, partials_len), kernels,
 * results and errors as uniquan_layer_recon, plus UQ_EUNSUPPORTED when the
 * shape needs more than uniquan_recon_noalloc_max_partials() partials
 * (uniquan_recon_ws(T, R, C) > 65536, i.e. R * T beyond about 2^30).
 * Calls that overlap on one GPU (concurrent streams or threads) share the
 * array and race; calls ordered on one stream do not.
 */
uq_status uniquan_layer_recon_noalloc(int64_t T, int64_t R, int64_t C,
                                      const uint16_t* X, const uint16_t* Xt,
                                      const uint16_t* W_hat, const float* Yt,
                                      float* loss, uint16_t* Et,
                                      void* grad_W_hat, int grad_dtype,
                                      void* stream);
size_t uniquan_recon_noalloc_max_partials(void);

/*
 * uniquan_layer_grad -- the weight-gradient half of uniquan_layer_recon on
 * its own: grad_W_hat = 2 Et Xt^T, grad[r, c] = 2 sum_t Et[r, t] X[t, c]
 * (bf16 MFMA, fp32 accumulation).  For callers that run the forward with
 * grad_W_hat = NULL and the backward later on the same stream.
 *
 * Et [R*T] bf16 (left in Et_ws by uniquan_layer_recon); Xt [C*T] bf16;
 * grad_W_hat [R*C] grad_dtype out.
 */
uq_status uniquan_layer_grad(int64_t T, int64_t R, int64_t C,
                             const uint16_t* Et, const uint16_t* Xt,
                             void* grad_W_hat, int grad_dtype, void* stream);

/*
 * uniquan_layer_grad_ste_sgd -- the weight-gradient GEMM of
 * uniquan_layer_grad with the straight-through backward and the SGD update
 * of uniquan_fq_bwd_sgd run in its epilogue (Algorithm 1's backward and
 * update lines; appendix "Implementation details" for the filter).  The
 * gradient dL/dWhat = 2 Et Xt^T never leaves the chip: each 256 x 256 tile
 * applies, to the fp32 accumulators,
 *     grad_s = -m Delta G (wbar - z_U) / s,  s -= lr_f grad_s
 *     grad_alpha_i = Delta sum_g sigma_i G,  alpha -= lr_b grad_alpha
 *     grad_z_B = Delta sum_g G,              z_B -= lr_b grad_z_B
 * with the mask m from bit 7 of the code byte (as uniquan_fq_bwd), group
 * sums over g/8 lanes in a fixed butterfly order.  Differs from the
 * unfused path only in using the fp32 gradient instead of its bf16 copy.
 *
 * Et [R*T] bf16, Xt [C*T] bf16 (as uniquan_layer_grad); W, s (in/out),
 * s_r, delta, z_u, alpha (in/out), z_b (in/out), codes as for
 * uniquan_fq_bwd_sgd; grad_s [R*C], grad_alpha [Gn*k], grad_z_b [Gn]:
 * optional copies of the gradients (NULL = not stored).
 * Limits: 1 <= k <= 4, g <= 128, T % 32 == 0 (UQ_EUNSUPPORTED otherwise),
 * plus the shape rules of uniquan_fq_fwd and uniquan_layer_grad.
 */
uq_status uniquan_layer_grad_ste_sgd(int64_t T, int64_t R, int64_t C, int k, int g,
                                     const uint16_t* Et, const uint16_t* Xt,
                                     const void* W, int w_dtype,
                                     float* s, const float* s_r,
                                     const float* delta, const float* z_u,
                                     float* alpha, float* z_b,
                                     const uint8_t* codes,
                                     float lr_f, float lr_b,
                                     float* grad_s, float* grad_alpha, float* grad_z_b,
                                     void* stream);

/*
 * uniquan_fold_to_bcq -- Theorem 1 and Eq. (4): plain binary-coding
 * parameters that reproduce Delta * (C alpha + z_B - z_U) exactly in real
 * arithmetic:
 *     alpha_star = Delta * alpha,  z_star = Delta * (z_B - z_U)    (fp32)
 * and the deployable codes (bit 7 clear):
 *     code_src 0: FULL mapping of wbar = T_F(w) against the levels of
 *                 (alpha, z_B) -- keeps the trained flexible mapping;
 *     code_src 1: Eq. (4) as printed, FULL mapping of the raw w against
 *                 the levels of (alpha_star, z_star).
 * codes_out may be NULL (parameters only).
 */
uq_status uniquan_fold_to_bcq(int64_t R, int64_t C, int k, int g,
                              const void* W, int w_dtype,
                              const float* s, const float* s_r,
                              const float* delta, const float* z_u,
                              const float* alpha, const float* z_b,
                              float* alpha_star, float* z_star,
                              uint8_t* codes_out, int code_src,
                              void* stream);

/*
 * uniquan_bcq_dequant -- binary-coding reconstruction R_B(C; Theta)
 * = C alpha + z_B 1_g (Sec. 2.3), the deployed model's weights:
 *     W_out[j] = z_b[gid] + sum_i (+-alpha[gid, i])   (fp32, left to right)
 * codes [R*C] uint8 (bit 7 ignored); alpha [Gn*k]; z_b [Gn];
 * W_out [R*C] out_dtype.
 */
uq_status uniquan_bcq_dequant(int64_t R, int64_t C, int k, int g,
                              const uint8_t* codes, const float* alpha,
                              const float* z_b, void* W_out, int out_dtype,
                              void* stream);

/*
 * Block-level reconstruction of a Transformer block's MLP module
 * (Algorithm 1 with f = the SiLU-gated MLP G = X W_g^T, U = X W_u^T,
 * H = silu(G) * U, Y = H W_d^T; the loss is ||Y(X; W) - Y(X; What)||_F^2).
 * The block step is composed from uniquan_fq_fwd / uniquan_fq_bwd_sgd per
 * matrix, uniquan_layer_target / uniquan_layer_recon for the output and
 * the down matrix's gradient, uniquan_transpose_bf16, and the three calls
 * below.
 */

/*
 * uniquan_gemm_nt -- out[M x N] = scale * A[M x K] B[N x K]^T, bf16 operands
 * with K contiguous (16-byte aligned), fp32 accumulation, out bf16 (RNE) or
 * fp32 row-major.  N and K multiples of 8, N < 2^26.
 */
uq_status uniquan_gemm_nt(int64_t M, int64_t N, int64_t K, const uint16_t* A,
                          const uint16_t* B, void* out, int out_dtype,
                          float scale, void* stream);

/*
 * uniquan_gemm_nt_residual -- out[M x N] = R + A[M x K] B[N x K]^T (fp32
 * R and out row-major, 16-byte aligned; out may be R itself): the attention
 * module's output projection with the block's first residual added in the
 * product's store (Algorithm 1's forward through a pre-norm block), bit for
 * bit uniquan_gemm_nt (fp32 out, scale 1) followed by the fp32 sum R + P.
 * uniquan_gemm_nt's rules on the shape and operands.
 */
uq_status uniquan_gemm_nt_residual(int64_t M, int64_t N, int64_t K, const uint16_t* A,
                                   const uint16_t* B, const float* R, float* out,
                                   void* stream);

/*
 * uniquan_gemm -- out[M x N] = scale * sum_k A(m, k) B(n, k) with either
 * operand stored K-slow, the contractions of the block's backpropagation
 * (Algorithm 1): the weight gradient dL/dW = dY^T X reads dY [T x out] and
 * X [T x in] as stored (both K-slow, K = T), the input gradient dX = dY W
 * reads W [out x in] as stored (B K-slow, K = out).
 *   A(m, k) = A[m K + k] (a_kslow = 0) or A[k M + m] (a_kslow = 1);
 *   B(n, k) = B[n K + k] (b_kslow = 0) or B[k N + n] (b_kslow = 1).
 * bf16 operands (16-byte aligned), fp32 accumulation over k in the same
 * order as uniquan_gemm_nt (the result equals uniquan_gemm_nt on the
 * operands transposed to K-contiguous, bit for bit), out bf16 (RNE) or fp32
 * row-major.  With a K-slow operand: K a multiple of 32, N a multiple of 8,
 * M a multiple of 8 when A is K-slow; with neither, uniquan_gemm_nt's rules.
 */
uq_status uniquan_gemm(int64_t M, int64_t N, int64_t K, const uint16_t* A,
                       int a_kslow, const uint16_t* B, int b_kslow, void* out,
                       int out_dtype, float scale, void* stream);

/*
 * uniquan_gemm_swiglu -- the MLP module's gate and up products with the SiLU
 * product (Algorithm 1's forward through the SiLU-gated MLP) in one product:
 *     G = X W_g^T, U = X W_u^T   (X [T x K], W_g, W_u [I x K] bf16, fp32
 *                                 accumulation, G and U stored bf16 [T x I]),
 *     H = silu(G) U              (from the stored bf16 G and U, as
 *                                 uniquan_silu_mul_fwd computes it),
 * bit for bit uniquan_gemm_nt twice (bf16 out) and uniquan_silu_mul_fwd.
 * I and K multiples of 32; X, W 16-byte and G, U, H 8-byte aligned.
 */
uq_status uniquan_gemm_swiglu(int64_t T, int64_t I, int64_t K, const uint16_t* X,
                              const uint16_t* Wg, const uint16_t* Wu, uint16_t* G,
                              uint16_t* U, uint16_t* H, void* stream);

/*
 * uniquan_gemm_silu_bwd -- the MLP module's backward through the down
 * matrix and the SiLU product (Algorithm 1's backpropagation):
 *     dH = bf16(scale E W_d)   (E [T x K] bf16 K-contiguous, W_d stored as
 *                               [K x I] (the down matrix, K = C), fp32
 *                               accumulation; dH is not written),
 *     dG, dU = the SiLU product's backward at (dH, G, U) (bf16 [T x I], as
 *                               uniquan_silu_mul_bwd computes it),
 * bit for bit uniquan_gemm (b_kslow = 1, bf16 out) followed by
 * uniquan_silu_mul_bwd.  G and U are [T x I] row-major; the rows of dG and
 * of dU are ld_d elements apart (0 means I; ld_d = 2 I with dU = dG + I puts
 * the two side by side in one [T x 2I] array, the operand of the stacked
 * products dL/dW_g; dL/dW_u = [dG dU]^T X and dX = [dG dU] [W_g; W_u]).
 * I a multiple of 8, K of 32, ld_d >= I a multiple of 4; E, W_d 16-byte and
 * G, U, dG, dU 8-byte aligned.
 */
uq_status uniquan_gemm_silu_bwd(int64_t T, int64_t I, int64_t K, const uint16_t* E,
                                const uint16_t* Wd, float scale, const uint16_t* G,
                                const uint16_t* U, uint16_t* dG, uint16_t* dU,
                                int64_t ld_d, void* stream);

/*
 * uniquan_silu_mul_fwd -- H[i] = silu(G[i]) * U[i], i < n (bf16 in and out,
 * fp32 arithmetic, silu(x) = x / (1 + exp(-x))); n a multiple of 8,
 * pointers 16-byte aligned.
 */
uq_status uniquan_silu_mul_fwd(int64_t n, const uint16_t* G, const uint16_t* U,
                               uint16_t* H, void* stream);

/*
 * uniquan_silu_mul_bwd -- dG[i] = dH[i] U[i] silu'(G[i]),
 * dU[i] = dH[i] silu(G[i]) (bf16 in and out, fp32 arithmetic,
 * silu'(x) = sigma(x) (1 + x (1 - sigma(x)))); n a multiple of 8.
 */
uq_status uniquan_silu_mul_bwd(int64_t n, const uint16_t* dH, const uint16_t* G,
                               const uint16_t* U, uint16_t* dG, uint16_t* dU,
                               void* stream);

/*
 * Block-level reconstruction of a whole Transformer block (Algorithm 1; the
 * block is one multi-head attention module and one MLP module, appendix
 * "Units in LLMs"; the loss ||f(X; W) - f(X_hat; What)||_F^2 of the appendix
 * "Error Types").  Pre-norm block: Z1 = RMSNorm(X; g1); Q, K rotary-embedded
 * (pairs (i, i + d/2), angle p 1e4^(-2i/d) at position p of the sequence),
 * causal softmax attention per sequence and head; R = X + O W_o^T;
 * Z2 = RMSNorm(R; g2); Y = R + MLP(Z2).  RMSNorm(x; g) = x / sqrt(mean(x^2)
 * + 1e-5) g over the C hidden features.  Layouts: token-major [T, C];
 * head-major [H, T, d] (T = n_seq L tokens, one [L, d] block per sequence
 * and head); scores [H n_seq, L, L].  The step is composed from the calls
 * below, uniquan_gemm_nt(_batched), uniquan_silu_mul_*, uniquan_transpose_*
 * and the quantizer entry points; every pointer is a device pointer owned by
 * the caller, errors are reported before any launch.
 */

/*
 * uniquan_gemm_nt_batched -- for b < batch:
 * out_b[M x N] = scale * A_b[M x K] B_b[N x K]^T with A_b = A + b stride_a,
 * B_b = B + b stride_b (elements; 0 repeats an operand), out_b = out +
 * b stride_out (elements of out_dtype, >= M N).  Shape rules as
 * uniquan_gemm_nt; strides multiples of 8; batch <= 65535.
 * causal (the attention's square [L, L] operands, K % 32 == 0):
 *   0  the full product;
 *   1  M == N: tiles entirely above the diagonal (all columns > all rows)
 *      are skipped and their outputs left unwritten (the causal softmax
 *      reads only j <= i);
 *   2  M == K: A is zero above the diagonal; the K loop of a row tile ends
 *      at the tile's last row (the result equals the full product);
 *   3  M == K: A is zero below the diagonal; the K loop of a row tile starts
 *      at its first row (the result equals the full product).
 */
uq_status uniquan_gemm_nt_batched(int64_t M, int64_t N, int64_t K, int64_t batch,
                                  const uint16_t* A, int64_t stride_a,
                                  const uint16_t* B, int64_t stride_b, void* out,
                                  int64_t stride_out, int out_dtype, float scale,
                                  int causal, void* stream);

/*
 * uniquan_add_rmsnorm -- per row t < T of [T, C] (fp32): v = X + A (A may be
 * NULL), R = v (written when A is given; R may be NULL otherwise),
 * rinv[t] = 1 / sqrt(mean(v^2) + 1e-5), Z = bf16((v rinv) gamma).
 * C a multiple of 8; fp32 arrays 16-byte aligned, Z 8-byte aligned.
 */
uq_status uniquan_add_rmsnorm(int64_t T, int64_t C, const float* X,
                              const float* A, const float* gamma, float* R,
                              uint16_t* Z, float* rinv, void* stream);

/*
 * uniquan_rmsnorm_bwd -- backward of Z = (X rinv) gamma plus a residual
 * gradient: with g = gamma (dZa + dZb) (dZb may be NULL),
 * dR = escale E + rinv g - X rinv^3 sum(g X) / C per row; E (bf16) may be
 * NULL.  dR is written in bf16, and in fp32 to dRf when given.  fp32 arrays
 * 16-byte aligned, E and dR 8-byte aligned.
 */
uq_status uniquan_rmsnorm_bwd(int64_t T, int64_t C, const float* dZa,
                              const float* dZb, const float* X,
                              const float* gamma, const float* rinv,
                              const uint16_t* E, float escale, uint16_t* dR,
                              float* dRf, void* stream);

/*
 * uniquan_rope_split -- token-major in [T, H d] (UQ_F32 or UQ_BF16) to
 * head-major bf16 out [H, T, d]; with rotate != 0 each pair (i, i + d/2) of
 * token t is rotated by angle (t mod L) 1e4^(-2i/d).  d even, L divides T.
 * group (dividing H; 1 for the plain order) stores head h at slot
 * (h mod group) (H / group) + h / group: for grouped-query attention with
 * group query heads per key/value head, the query heads at one position of
 * their groups become contiguous in key/value head order.
 * uniquan_rope_merge -- the inverse layout change (head-major in with the
 * same slot order, token-major bf16 out), rotating by minus the angle when
 * rotate != 0; the input holds nsum stacked [H, T, d] partials that are
 * summed first (the gradient of a shared key/value head, nsum = group size);
 * the output rows are ld_out >= H d elements apart (0 means H d: the key and
 * value gradients of grouped-query attention side by side in one [T, 2 H d]
 * array, the operand of their stacked weight-gradient product).
 */
uq_status uniquan_rope_split(int64_t T, int H, int d, int L, int group,
                             const void* in, int in_dtype, int rotate,
                             uint16_t* out, void* stream);

/*
 * uniquan_rope_table -- cs [L, d/2] pairs (cos, sin) of the rotary angle
 * (p, i) -> p 1e4^(-2i/d) at every position p < L (fp32, 16-byte aligned),
 * the values uniquan_rope_split uses.  d even, at most 1024.
 *
 * uniquan_gemm_heads -- the block's query / key / value projection with the
 * head split (and rotation) of uniquan_rope_split folded into the product's
 * store (Algorithm 1's forward through the attention module):
 *     Y = A W^T  (A [T x K] bf16, W [H 128 x K] bf16, fp32 accumulation),
 *     out = uniquan_rope_split(Y) with d = 128 and group as there, the
 *           heads h < n_rot rotated (n_rot = 0: none, >= H: all; rotating
 *           only the leading heads, e.g. the keys of a stacked key/value
 *           product [W_k; W_v], needs group 1),
 * out bf16 head-major [H, T, 128], bit for bit the result of
 * uniquan_gemm_nt (fp32 out) followed by uniquan_rope_split of each head
 * range.  cs from uniquan_rope_table(L, 128) (read only when n_rot > 0).
 * K a multiple of 32, L divides T; out 8-byte and cs 32-byte aligned.
 */
uq_status uniquan_rope_table(int L, int d, float* cs, void* stream);
uq_status uniquan_gemm_heads(int64_t T, int H, int64_t K, const uint16_t* A,
                             const uint16_t* W, int L, int group, int n_rot,
                             const float* cs, uint16_t* out, void* stream);
uq_status uniquan_rope_merge(int64_t T, int H, int d, int L, int group,
                             int nsum, const void* in, int in_dtype, int rotate,
                             uint16_t* out, int64_t ld_out, void* stream);

/*
 * uniquan_softmax_causal -- for each row r < rows of S [rows, L] (fp32, row
 * i = r mod L of an [L, L] score block): P[r, j] = softmax over j <= i of
 * S[r, j], 0 for j > i (bf16).  rows a multiple of L.
 * uniquan_softmax_causal_bwd -- dS = P (dP - sum_j P dP) per row (bf16 out;
 * dP fp32, P bf16 as written by the forward).
 */
uq_status uniquan_softmax_causal(int64_t rows, int L, const float* S,
                                 uint16_t* P, void* stream);
uq_status uniquan_softmax_causal_bwd(int64_t rows, int L, const float* dP,
                                     const uint16_t* P, uint16_t* dS,
                                     void* stream);

/*
 * uniquan_attn_fwd / uniquan_attn_bwd -- the block's causal attention with
 * the [L, L] score tiles kept on chip (none is written to memory); the
 * attention of the Transformer block that Algorithm 1 reconstructs (appendix
 * "Units in LLMs").  Per sequence and query head b < batch, with key/value
 * head b mod kv_batch (the grouped slot order of uniquan_rope_split: query
 * batch g kv_batch + c pairs with key/value batch c), head dimension d = 128
 * and c = scale log2(e):
 *   S = Q K^T, row_lse_i = log2 sum_{j <= i} 2^(c S_ij) (the base-2
 *   log-sum-exp of the scaled scores), P = bf16(2^(c S - row_lse)) (the causal
 *   row softmax of S scale), O = bf16(P V).
 * Backward, recomputing the same P from row_lse:
 *   dP = dO V^T (fp32), delta_i = dO_i . O_i (fp32; equal to sum_j P_ij dP_ij
 *   in exact arithmetic), dS = bf16(P (dP - delta)), dQ = dS K scale, and per
 *   query head b the contributions dK_b = dS^T Q scale, dV_b = P^T dO (fp32
 *   out); the gradient of a key/value head shared by several query heads is
 *   the sum of their contributions (uniquan_rope_merge with nsum sums them).
 * The rounding points are those of the unfused path (P and dS in bf16, S and
 * dP in fp32).
 * Layouts (bf16 unless stated): Q [batch, L, d]; K, V [kv_batch, L, d] (the
 * products that contract over the rows of a tile read it through LDS
 * transpose reads, so no transposed copies are taken); row_lse, delta
 * [batch, L] fp32 (delta written by uniquan_attn_bwd).
 * With tok_seqs = 0: O, dO [batch, L, d]; dQ, dK, dV [batch, L, d] fp32 out.
 * With tok_seqs = n > 0 (n divides batch and kv_batch; H = batch / n query
 * heads, group dividing H): O and dO are token-major [n L, H d] bf16 rows,
 * query batch b = slot n + s holding head (slot mod (H/group)) group +
 * slot / (H/group) of sequence s (the slot order of uniquan_rope_split), so
 * O needs no merge and dO no split; dQ is written token-major bf16 after the
 * inverse rotation of uniquan_rope_merge (cs from uniquan_rope_table(L, 128),
 * 32-byte aligned), bit for bit what the fp32 dQ and a merge give; dK and dV
 * likewise (dK inverse-rotated, dV not) when kv_batch = batch, and fp32
 * per-query-head [batch, L, d] partials as with tok_seqs = 0 otherwise (the
 * merge sums them over each key/value head's group).  d = 128
 * and L a multiple of 32 (UQ_EUNSUPPORTED otherwise); batch a positive
 * multiple of kv_batch, at most 65535; every pointer 16-byte aligned.
 */
uq_status uniquan_attn_fwd(int64_t batch, int64_t kv_batch, int L, int d,
                           const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                           float scale, uint16_t* O, float* row_lse, int tok_seqs,
                           int group, void* stream);
uq_status uniquan_attn_bwd(int64_t batch, int64_t kv_batch, int L, int d,
                           const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                           const uint16_t* O, const uint16_t* dO, const float* row_lse,
                           float scale, float* delta, void* dQ, void* dK, void* dV,
                           int tok_seqs, int group, const float* cs, void* stream);

/*
 * uniquan_transpose_bf16_batched -- out_b = in_b^T for batch matrices
 * [R, C] stored back to back (bf16; in and out 8-byte aligned).
 */
uq_status uniquan_transpose_bf16_batched(int64_t batch, int64_t R, int64_t C,
                                         const uint16_t* in, uint16_t* out,
                                         void* stream);

/*
 * uniquan_block_loss -- E = (R + M) - Yref element-wise (fp32 in, bf16 out)
 * and loss[0] = sum of the unrounded E^2 (per-block fp32 partials summed in
 * fp64 in a fixed order).  partials holds uniquan_block_loss_ws() floats
 * (partials_len gives its size).
 */
size_t uniquan_block_loss_ws(void);

/*
 * uniquan_gemm_block_loss -- the block's output product with the loss in its
 * store (the loss of Algorithm 1 on the block's output, appendix "Error
 * Types"): with M = H W_d^T (H [T x K], W_d [C x K] bf16, fp32 accumulation)
 *     E = bf16((R + M) - Yref)   (R, Yref fp32 [T x C]; M is not written),
 *     loss[0] = sum of the unrounded e^2: per-workgroup fp32 partials (each
 *               workgroup's wavefronts in a fixed tree) summed in fp64 in a
 *               fixed order;
 * the values of uniquan_gemm_nt (fp32 M) followed by uniquan_block_loss, E bit
 * for bit, the loss to rounding (its partial sums are grouped by tile).
 * partials holds uniquan_gemm_block_loss_ws(T, C) floats.  C and K multiples
 * of 8; H, W_d, R, Yref 16-byte and E 8-byte aligned.
 */
size_t uniquan_gemm_block_loss_ws(int64_t T, int64_t C);
uq_status uniquan_gemm_block_loss(int64_t T, int64_t C, int64_t K, const uint16_t* H,
                                  const uint16_t* Wd, const float* R, const float* Yref,
                                  uint16_t* E, float* partials, size_t partials_len,
                                  float* loss, void* stream);
uq_status uniquan_block_loss(int64_t n, const float* R, const float* M,
                             const float* Yref, uint16_t* E, float* partials,
                             size_t partials_len, float* loss, void* stream);

/*
 * Deployment form of a folded layer and its inference product (the single
 * binary-coding step R_B(C; Theta*) that Theorem 1 leaves; storage as in the
 * appendix "Memory usage": g k + 16 (k + 1) bits per group).
 *
 * Layout (rows are the fastest index of every array):
 *   planes  uint32 [k][C/128][R][4]: word m of quad q of row r in plane i
 *           has bit j = bit i of the code of column 128 q + 32 m + j
 *           (1 <=> c_{i+1} = +1);
 *   alpha16 IEEE binary16 [k][C/g][R]: alpha*_{i+1} of group (r, j);
 *   z16     IEEE binary16 [C/g][R]:    z*_B of group (r, j).
 * Shape rules: 1 <= k <= 4, C % 128 == 0, C <= 2^22, g % 128 == 0,
 * C % g == 0 (UQ_EUNSUPPORTED otherwise; UQ_EINVAL if g does not divide C).
 */

/*
 * uniquan_bcq_pack -- the stored form from uniquan_fold_to_bcq's outputs:
 * codes [R*C] uint8 (bits 0..k-1 used, 16-byte aligned), alpha_star [Gn*k],
 * z_star [Gn] fp32 (rounded to binary16, to nearest even).  planes
 * (16-byte aligned) R*C*k/8 bytes, alpha16 Gn*k and z16 Gn halves out.
 */
uq_status uniquan_bcq_pack(int64_t R, int64_t C, int k, int g,
                           const uint8_t* codes, const float* alpha_star,
                           const float* z_star, uint32_t* planes,
                           uint16_t* alpha16, uint16_t* z16, void* stream);

/*
 * uniquan_bcq_matmul -- Y = X What^T for a batch of T <= 8 activation rows,
 * What[r][c] = z* + sum_i alpha*_i sigma_i(r, c) from the stored form:
 * X [T*C] bf16 (8-byte aligned), Y [T*R] fp32 out.  Per group the kernel
 * uses sum_c sigma_i x_c = 2 P_i - S (S: the group's activation sum, P_i:
 * the sum over columns whose bit i is set), P_i from 16-entry subset-sum
 * tables of 4 activations for T <= 3 and from bf16 MFMA products of the
 * activations with the 0/1 planes for T >= 4; fp32 accumulation,
 * deterministic order.
 * partials_ws [partials_len] fp32 workspace of at least
 * uniquan_bcq_matmul_ws(T, R, C) floats (0: may be NULL).
 */
size_t uniquan_bcq_matmul_ws(int T, int64_t R, int64_t C);
uq_status uniquan_bcq_matmul(int T, int64_t R, int64_t C, int k, int g,
                             const uint16_t* X, const uint32_t* planes,
                             const uint16_t* alpha16, const uint16_t* z16,
                             float* Y, float* partials_ws, size_t partials_len,
                             void* stream);

/*
 * uniquan_init_greedy -- greedy binary-coding start of the appendix
 * algorithm "General alternating update" (its first step): per group,
 * r = wbar - z_B with wbar = T_F(w) as in uniquan_fq_fwd; then for
 * i = 1..k: c_i = sign(r) (sign(0) = +1), alpha_i = mean_j |r_j|,
 * r <- r - alpha_i c_i.  fp32 arithmetic; group sums in a fixed order.
 *
 * W, s, s_r, delta, z_u as for uniquan_fq_fwd; z_b [Gn] in;
 * alpha [Gn*k] fp32 out.
 */
uq_status uniquan_init_greedy(int64_t R, int64_t C, int k, int g,
                              const void* W, int w_dtype,
                              const float* s, const float* s_r,
                              const float* delta, const float* z_u,
                              const float* z_b, float* alpha,
                              void* stream);

/*
 * uniquan_init_unified -- unified initialisation of Theta_{I_F} (Sec. 3
 * "Unified initialization"; appendix algorithms "Unified Initialization" and
 * "General alternating update"; appendix "Details of clipping strategies").
 *
 * Per group (w = its g weights, w_m / w_M their min / max, L1 = 2^k - 1):
 *   for j = 1..grid_G, gamma = j / grid_G (fp32 division):
 *     Delta' = (gamma (w_M - w_m)) / L1, or 1 if that is not > 0;
 *     z'_U   = -(w_m / Delta')              clip 0, fixed minimum
 *              L1 - (w_M / Delta')          clip 1, fixed maximum
 *              -((gamma w_m) / Delta')      clip 2, balanced
 *     wbar   = (w / Delta') + z'_U          (T_F with s = 1, s_r = 1)
 *     z_B = L1 / 2; greedy start on wbar - z_B (as uniquan_init_greedy);
 *     alt_T rounds of: alpha <- (C^T C)^{-1} C^T (wbar - z_B);
 *                      C <- nearest level's code of each wbar (FULL rule);
 *                      z_B <- mean(wbar - C alpha) when grid_G == 1;
 *     e' = ||w - what||^2, what = the fp32 output of uniquan_fq_fwd (FULL);
 *   keep the first candidate, then any with strictly smaller e'.
 * Fixed fp32 evaluation order: group sums are pairwise with adjacent pairing
 * over the group zero-padded to a power of two; means are those sums divided
 * by g; the inverse of C^T C is taken through its exact integer adjugate and
 * determinant, its product with C^T (wbar - z_B) formed in fp64 (each product
 * rounded, added in ascending order; exact for g <= 512) and divided by the
 * determinant, then rounded to fp32; a singular C^T C keeps the previous
 * alpha.  Results are bit-reproducible.  Groups above 512 weights (per-row
 * groups) run one workgroup per group.
 *
 * W [R*C] w_dtype (16-byte aligned).  Out (fp32, caller-owned): delta, z_u,
 * z_b [Gn], alpha [Gn*k].  Optional out (NULL = skipped): codes [R*C] uint8,
 * the kept candidate's FULL-mapping codes (bit 7 clear; 8-byte aligned);
 * err [Gn], its e'; s [R*C] and s_r [R] filled with 1.
 * Limits: 1 <= k <= 4 (UQ_EUNSUPPORTED above), g as for the quantizer and at
 * most 16384 (UQ_EUNSUPPORTED above), 1 <= grid_G <= 4096, 0 <= alt_T <= 10000, clip in {0, 1, 2} (UQ_EINVAL).
 * Preconditions (not checked): finite weights whose squares are finite.
 */
uq_status uniquan_init_unified(int64_t R, int64_t C, int k, int g,
                               const void* W, int w_dtype,
                               int grid_G, int alt_T, int clip,
                               float* delta, float* z_u, float* alpha, float* z_b,
                               uint8_t* codes, float* err, float* s, float* s_r,
                               void* stream);

/*
 * uniquan_sgd -- theta[i] -= lr * grad[i] for i < n (the stochastic
 * gradient descent update of Algorithm 1, applied per parameter tensor).
 * theta, grad fp32 [n].
 */
uq_status uniquan_sgd(int64_t n, float* theta, const float* grad, float lr, void* stream);

/*
 * Measurement probes (not part of the method): the streaming HBM rates and
 * the bf16 MFMA issue rate this GPU reaches, reported next to the nominal
 * peaks.  sink: 16 bytes of device memory (16-byte aligned) that a probe
 * writes only when its result equals a value the data cannot produce, so
 * that nothing is optimised away; its contents are meaningless.
 *
 * uniquan_probe_stream -- op 0 reads n_bytes of src, op 1 writes n_bytes of
 * dst, op 2 copies n_bytes from src to dst; 16-byte nontemporal accesses in a
 * grid-stride loop over `blocks` workgroups of 256 lanes (1 .. 2^20).
 * n_bytes a positive multiple of 16; src, dst 16-byte aligned device memory
 * (the unused one may be NULL).
 * uniquan_probe_mfma -- iters rounds of independent v_mfma_f32_32x32x16_bf16
 * chains on register operands over the whole GPU; the work done is
 * uniquan_probe_mfma_flops(iters) floating-point operations.
 */
double uniquan_probe_mfma_flops(int iters);
uq_status uniquan_probe_stream(int op, int64_t n_bytes, const void* src, void* dst,
                               void* sink, int blocks, void* stream);
uq_status uniquan_probe_mfma(int iters, float* sink, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* UNIQUAN_H */
