// C ABI of the library (declared in include/uniquan.h): argument validation
// on the host, before any HIP call, then the kernel launches.
#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <cstring>

#include "../../include/uniquan.h"
#include "uq_launch.h"

namespace {

thread_local char g_err[512] = "";

uq_status fail(uq_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return st;
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

#define REQ_PTR(p, al)                                                                   \
  do {                                                                                   \
    if ((p) == nullptr) return fail(UQ_EINVAL, "%s: %s must not be NULL", fn, #p);       \
    if (!aligned((p), (al))) return fail(UQ_EINVAL, "%s: %s must be %d-byte aligned", fn, #p, int(al)); \
  } while (0)
#define OPT_PTR(p, al)                                                                   \
  do {                                                                                   \
    if ((p) != nullptr && !aligned((p), (al)))                                           \
      return fail(UQ_EINVAL, "%s: %s must be %d-byte aligned", fn, #p, int(al));         \
  } while (0)

bool is_dtype(int d) { return d == UQ_F32 || d == UQ_BF16; }

// Shape rules shared by the per-weight entry points.
uq_status check_quant_shape(const char* fn, int64_t R, int64_t C, int k, int g) {
  if (R < 1 || C < 1) return fail(UQ_EINVAL, "%s: R=%lld and C=%lld must be >= 1", fn, (long long)R, (long long)C);
  if (k < 1 || k > 7) return fail(UQ_EINVAL, "%s: k=%d must be in [1, 7]", fn, k);
  if (g < 8 || g % 8 != 0) return fail(UQ_EINVAL, "%s: g=%d must be a positive multiple of 8", fn, g);
  if (g <= 512 && (g & (g - 1)) != 0)
    return fail(UQ_EUNSUPPORTED, "%s: g=%d: groups of up to 512 weights must be a power of two", fn, g);
  if (g > (1 << 24)) return fail(UQ_EUNSUPPORTED, "%s: g=%d > 2^24 is not supported", fn, g);
  if (C % g != 0) return fail(UQ_EINVAL, "%s: g=%d must divide C=%lld", fn, g, (long long)C);
  if (R > (int64_t(1) << 40) / C) return fail(UQ_EUNSUPPORTED, "%s: R*C too large", fn);
  if ((R * C) / g >= (int64_t(1) << 31)) return fail(UQ_EUNSUPPORTED, "%s: more than 2^31 groups", fn);
  return UQ_OK;
}

uq_status hip_status(const char* fn, hipError_t e) {
  if (e == hipSuccess) return UQ_OK;
  return fail(UQ_EHIP, "%s: launch failed: %s", fn, hipGetErrorString(e));
}

uq_status check_gemm_dims(const char* fn, int64_t T, int64_t R, int64_t C) {
  if (T < 1 || R < 1 || C < 1) return fail(UQ_EINVAL, "%s: T, R, C must be >= 1", fn);
  if (T % 8 != 0) return fail(UQ_EINVAL, "%s: T=%lld must be a multiple of 8", fn, (long long)T);
  if (C % 8 != 0) return fail(UQ_EINVAL, "%s: C=%lld must be a multiple of 8", fn, (long long)C);
  if (T >= (int64_t(1) << 26) || C >= (int64_t(1) << 26))
    return fail(UQ_EUNSUPPORTED, "%s: T and C must be < 2^26", fn);
  const int64_t lim = int64_t(1) << 31;
  if (T >= lim || R >= lim || C >= lim || T * C >= (int64_t(1) << 40) || R * C >= (int64_t(1) << 40) ||
      R * T >= (int64_t(1) << 40))
    return fail(UQ_EUNSUPPORTED, "%s: shape too large", fn);
  return UQ_OK;
}

}  // namespace

extern "C" {

int uniquan_abi_version(void) { return UNIQUAN_ABI_VERSION; }

const char* uniquan_last_error(void) { return g_err; }

static uq_status fq_fwd_common(const char* fn, int64_t R, int64_t C, int k, int g, const void* W, int w_dtype,
                               const float* s, const float* s_r, const float* delta, const float* z_u,
                               const float* alpha, const float* z_b, int mode, uint8_t* codes, void* W_hat,
                               int w_hat_dtype, int resid, void* stream) {
  if (uq_status st = check_quant_shape(fn, R, C, k, g)) return st;
  if (!is_dtype(w_dtype) || !is_dtype(w_hat_dtype)) return fail(UQ_EINVAL, "%s: bad dtype", fn);
  if (mode < UQ_MAP_FULL || mode > UQ_MAP_FROZEN) return fail(UQ_EINVAL, "%s: bad mapping mode %d", fn, mode);
  REQ_PTR(W, 16); REQ_PTR(s, 16); REQ_PTR(alpha, 4); REQ_PTR(z_b, 4); REQ_PTR(codes, 16); REQ_PTR(W_hat, 16);
  OPT_PTR(s_r, 4); OPT_PTR(delta, 4); OPT_PTR(z_u, 4);
  uq::FqFwdLaunch p{R, C, k, g, W, w_dtype, s, s_r, delta, z_u, alpha, z_b, mode, codes, W_hat, w_hat_dtype, resid};
  return hip_status(fn, uq::launch_fq_fwd(p, static_cast<hipStream_t>(stream)));
}

uq_status uniquan_fq_fwd(int64_t R, int64_t C, int k, int g, const void* W, int w_dtype, const float* s,
                         const float* s_r, const float* delta, const float* z_u, const float* alpha,
                         const float* z_b, int mode, uint8_t* codes, void* W_hat, int w_hat_dtype,
                         void* stream) {
  return fq_fwd_common("uniquan_fq_fwd", R, C, k, g, W, w_dtype, s, s_r, delta, z_u, alpha, z_b, mode, codes,
                       W_hat, w_hat_dtype, 0, stream);
}

uq_status uniquan_fq_fwd_residual(int64_t R, int64_t C, int k, int g, const void* W, int w_dtype, const float* s,
                                  const float* s_r, const float* delta, const float* z_u, const float* alpha,
                                  const float* z_b, int mode, uint8_t* codes, void* R_out, int r_dtype,
                                  void* stream) {
  return fq_fwd_common("uniquan_fq_fwd_residual", R, C, k, g, W, w_dtype, s, s_r, delta, z_u, alpha, z_b, mode,
                       codes, R_out, r_dtype, 1, stream);
}

uq_status uniquan_fq_bwd(int64_t R, int64_t C, int k, int g, const void* W, int w_dtype, const float* s,
                         const float* s_r, const float* delta, const float* z_u, const float* alpha,
                         const float* z_b, const uint8_t* codes, const void* grad_W_hat, int grad_dtype,
                         float* grad_s, float* grad_alpha, float* grad_z_b, float* grad_delta, float* grad_z_u,
                         float* grad_s_r, float* group_ws, void* stream) {
  const char* fn = "uniquan_fq_bwd";
  if (uq_status st = check_quant_shape(fn, R, C, k, g)) return st;
  if (!is_dtype(w_dtype) || !is_dtype(grad_dtype)) return fail(UQ_EINVAL, "%s: bad dtype", fn);
  REQ_PTR(W, 16); REQ_PTR(s, 16); REQ_PTR(alpha, 4); REQ_PTR(z_b, 4); REQ_PTR(codes, 16);
  REQ_PTR(grad_W_hat, 16); REQ_PTR(grad_s, 16); REQ_PTR(grad_alpha, 4); REQ_PTR(grad_z_b, 4);
  OPT_PTR(s_r, 4); OPT_PTR(delta, 4); OPT_PTR(z_u, 4);
  OPT_PTR(grad_delta, 4); OPT_PTR(grad_z_u, 4); OPT_PTR(grad_s_r, 4);
  if (grad_s_r != nullptr) REQ_PTR(group_ws, 4);
  uq::FqBwdLaunch p{R, C, k, g, W, w_dtype, s, s_r, delta, z_u, alpha, z_b, codes, grad_W_hat, grad_dtype,
                    grad_s, grad_alpha, grad_z_b, grad_delta, grad_z_u, grad_s_r, group_ws, 0, 0.0f, 0.0f};
  return hip_status(fn, uq::launch_fq_bwd(p, static_cast<hipStream_t>(stream)));
}

uq_status uniquan_fq_bwd_sgd(int64_t R, int64_t C, int k, int g, const void* W, int w_dtype, float* s,
                             const float* s_r, const float* delta, const float* z_u, float* alpha, float* z_b,
                             const uint8_t* codes, const void* grad_W_hat, int grad_dtype, float* grad_s,
                             float* grad_alpha, float* grad_z_b, float lr_f, float lr_b, void* stream) {
  const char* fn = "uniquan_fq_bwd_sgd";
  if (uq_status st = check_quant_shape(fn, R, C, k, g)) return st;
  if (!is_dtype(w_dtype) || !is_dtype(grad_dtype)) return fail(UQ_EINVAL, "%s: bad dtype", fn);
  REQ_PTR(W, 16); REQ_PTR(s, 16); REQ_PTR(alpha, 4); REQ_PTR(z_b, 4); REQ_PTR(codes, 16);
  REQ_PTR(grad_W_hat, 16); OPT_PTR(grad_s, 16); OPT_PTR(grad_alpha, 4); OPT_PTR(grad_z_b, 4);
  OPT_PTR(s_r, 4); OPT_PTR(delta, 4); OPT_PTR(z_u, 4);
  uq::FqBwdLaunch p{R, C, k, g, W, w_dtype, s, s_r, delta, z_u, alpha, z_b, codes, grad_W_hat, grad_dtype,
                    grad_s, grad_alpha, grad_z_b, nullptr, nullptr, nullptr, nullptr, 1, lr_f, lr_b};
  return hip_status(fn, uq::launch_fq_bwd(p, static_cast<hipStream_t>(stream)));
}

uq_status uniquan_fq_step(int64_t R, int64_t C, int k, int g, const void* W, int w_dtype, float* s,
                          const float* s_r, const float* delta, const float* z_u, float* alpha, float* z_b,
                          uint8_t* codes, const void* grad_W_hat, int grad_dtype, float lr_f, float lr_b,
                          int next_mode, void* W_hat, int w_hat_dtype, int residual, void* stream) {
  const char* fn = "uniquan_fq_step";
  if (uq_status st = check_quant_shape(fn, R, C, k, g)) return st;
  if (!is_dtype(w_dtype) || !is_dtype(grad_dtype) || !is_dtype(w_hat_dtype)) return fail(UQ_EINVAL, "%s: bad dtype", fn);
  if (next_mode < UQ_MAP_FULL || next_mode > UQ_MAP_FROZEN)
    return fail(UQ_EINVAL, "%s: bad mapping mode %d", fn, next_mode);
  if (residual != 0 && residual != 1) return fail(UQ_EINVAL, "%s: residual must be 0 or 1", fn);
  REQ_PTR(W, 16); REQ_PTR(s, 16); REQ_PTR(alpha, 4); REQ_PTR(z_b, 4); REQ_PTR(codes, 16);
  REQ_PTR(grad_W_hat, 16); REQ_PTR(W_hat, 16);
  OPT_PTR(s_r, 4); OPT_PTR(delta, 4); OPT_PTR(z_u, 4);
  uq::FqStepLaunch p{R, C, k, g, W, w_dtype, s, s_r, delta, z_u, alpha, z_b, codes, grad_W_hat, grad_dtype,
                     lr_f, lr_b, next_mode, W_hat, w_hat_dtype, residual};
  return hip_status(fn, uq::launch_fq_step(p, static_cast<hipStream_t>(stream)));
}

uq_status uniquan_layer_target(int64_t T, int64_t R, int64_t C, const uint16_t* X, const uint16_t* W, float* Yt,
                               void* stream) {
  const char* fn = "uniquan_layer_target";
  if (uq_status st = check_gemm_dims(fn, T, R, C)) return st;
  REQ_PTR(X, 16); REQ_PTR(W, 16); REQ_PTR(Yt, 16);
  uq::GemmLaunch q{W, X, R, T, C, uq::EPI_TARGET, nullptr, Yt, nullptr, 1.0f};
  return hip_status(fn, uq::launch_gemm(q, static_cast<hipStream_t>(stream)));
}

uq_status uniquan_transpose_bf16(int64_t rows, int64_t cols, const uint16_t* in, uint16_t* out, void* stream) {
  const char* fn = "uniquan_transpose_bf16";
  if (rows < 1 || cols < 1 || rows % 8 || cols % 8)
    return fail(UQ_EINVAL, "%s: rows, cols must be positive multiples of 8", fn);
  if (rows >= (int64_t(1) << 31) / 64 * 64 || cols >= (int64_t(1) << 31) / 64 * 64)
    return fail(UQ_EUNSUPPORTED, "%s: shape too large", fn);
  REQ_PTR(in, 16); REQ_PTR(out, 16);
  return hip_status(fn, uq::launch_transpose(rows, cols, in, out, static_cast<hipStream_t>(stream)));
}

size_t uniquan_recon_ws(int64_t T, int64_t R, int64_t C) {
  (void)C;
  if (T < 1 || R < 1) return 0;
  return uq::gemm_workgroups(R, T, uq::EPI_LOSS);
}

uq_status uniquan_layer_recon(int64_t T, int64_t R, int64_t C, const uint16_t* X, const uint16_t* Xt,
                              const uint16_t* W_hat, const float* Yt, float* loss, uint16_t* Et_ws,
                              float* partials_ws, size_t partials_len, void* grad_W_hat, int grad_dtype,
                              void* stream) {
  const char* fn = "uniquan_layer_recon";
  if (uq_status st = check_gemm_dims(fn, T, R, C)) return st;
  REQ_PTR(X, 16); REQ_PTR(W_hat, 16); OPT_PTR(Yt, 16); REQ_PTR(loss, 4); REQ_PTR(Et_ws, 16);
  REQ_PTR(partials_ws, 16);
  if (partials_len < uniquan_recon_ws(T, R, C))
    return fail(UQ_EINVAL, "%s: partials_len=%zu < %zu", fn, partials_len, uniquan_recon_ws(T, R, C));
  if (grad_W_hat != nullptr) {
    REQ_PTR(Xt, 16);
    REQ_PTR(grad_W_hat, 16);
    if (!is_dtype(grad_dtype)) return fail(UQ_EINVAL, "%s: bad dtype", fn);
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  uq::GemmLaunch f{W_hat, X, R, T, C, uq::EPI_LOSS, Yt, Et_ws, partials_ws, 1.0f};
  if (uq_status s = hip_status(fn, uq::launch_gemm(f, st))) return s;
  if (uq_status s = hip_status(fn, uq::launch_reduce_loss(partials_ws, int64_t(uniquan_recon_ws(T, R, C)), loss, st)))
    return s;
  if (grad_W_hat == nullptr) return UQ_OK;
  uq::GemmLaunch b{Et_ws, Xt, R, C, T, grad_dtype == UQ_BF16 ? uq::EPI_GRAD_BF16 : uq::EPI_GRAD_F32,
                   nullptr, grad_W_hat, nullptr, 2.0f};
  return hip_status(fn, uq::launch_gemm(b, st));
}

uq_status uniquan_layer_recon_noalloc(int64_t T, int64_t R, int64_t C, const uint16_t* X, const uint16_t* Xt,
                                      const uint16_t* W_hat, const float* Yt, float* loss, uint16_t* Et,
                                      void* grad_W_hat, int grad_dtype, void* stream) {
  const char* fn = "uniquan_layer_recon_noalloc";
  if (uq_status st = check_gemm_dims(fn, T, R, C)) return st;
  REQ_PTR(X, 16); REQ_PTR(W_hat, 16); OPT_PTR(Yt, 16); REQ_PTR(loss, 4); REQ_PTR(Et, 16);
  if (grad_W_hat != nullptr) {
    REQ_PTR(Xt, 16);
    REQ_PTR(grad_W_hat, 16);
    if (!is_dtype(grad_dtype)) return fail(UQ_EINVAL, "%s: bad dtype", fn);
  }
  const size_t need = uniquan_recon_ws(T, R, C);
  if (need > uq::kNoallocPartials)
    return fail(UQ_EUNSUPPORTED, "%s: T=%lld, R=%lld need %zu loss partials; the fixed scratch holds %zu", fn,
                (long long)T, (long long)R, need, uq::kNoallocPartials);
  float* partials = nullptr;
  if (uq_status s = hip_status(fn, uq::noalloc_scratch(&partials))) return s;
  hipStream_t st = static_cast<hipStream_t>(stream);
  uq::GemmLaunch f{W_hat, X, R, T, C, uq::EPI_LOSS, Yt, Et, partials, 1.0f};
  if (uq_status s = hip_status(fn, uq::launch_gemm(f, st))) return s;
  if (uq_status s = hip_status(fn, uq::launch_reduce_loss(partials, int64_t(need), loss, st))) return s;
  if (grad_W_hat == nullptr) return UQ_OK;
  uq::GemmLaunch b{Et, Xt, R, C, T, grad_dtype == UQ_BF16 ? uq::EPI_GRAD_BF16 : uq::EPI_GRAD_F32,
                   nullptr, grad_W_hat, nullptr, 2.0f};
  return hip_status(fn, uq::launch_gemm(b, st));
}

size_t uniquan_recon_noalloc_max_partials(void) { return uq::kNoallocPartials; }

uq_status uniquan_layer_grad(int64_t T, int64_t R, int64_t C, const uint16_t* Et, const uint16_t* Xt,
                             void* grad_W_hat, int grad_dtype, void* stream) {
  const char* fn = "uniquan_layer_grad";
  if (uq_status st = check_gemm_dims(fn, T, R, C)) return st;
  REQ_PTR(Et, 16); REQ_PTR(Xt, 16); REQ_PTR(grad_W_hat, 16);
  if (!is_dtype(grad_dtype)) return fail(UQ_EINVAL, "%s: bad dtype", fn);
  uq::GemmLaunch b{Et, Xt, R, C, T, grad_dtype == UQ_BF16 ? uq::EPI_GRAD_BF16 : uq::EPI_GRAD_F32,
                   nullptr, grad_W_hat, nullptr, 2.0f};
  return hip_status(fn, uq::launch_gemm(b, static_cast<hipStream_t>(stream)));
}

uq_status uniquan_layer_grad_ste_sgd(int64_t T, int64_t R, int64_t C, int k, int g, const uint16_t* Et,
                                     const uint16_t* Xt, const void* W, int w_dtype, float* s, const float* s_r,
                                     const float* delta, const float* z_u, float* alpha, float* z_b,
                                     const uint8_t* codes, float lr_f, float lr_b, float* grad_s,
                                     float* grad_alpha, float* grad_z_b, void* stream) {
  const char* fn = "uniquan_layer_grad_ste_sgd";
  if (uq_status st = check_gemm_dims(fn, T, R, C)) return st;
  if (uq_status st = check_quant_shape(fn, R, C, k, g)) return st;
  if (k > 4) return fail(UQ_EUNSUPPORTED, "%s: k = %d, supported 1..4", fn, k);
  if (g > 128) return fail(UQ_EUNSUPPORTED, "%s: g = %d, supported up to 128", fn, g);
  if (T % 32 != 0) return fail(UQ_EUNSUPPORTED, "%s: T = %lld, must be a multiple of 32", fn, (long long)T);
  if (!is_dtype(w_dtype)) return fail(UQ_EINVAL, "%s: bad dtype", fn);
  REQ_PTR(Et, 16); REQ_PTR(Xt, 16); REQ_PTR(W, 16); REQ_PTR(s, 16); REQ_PTR(alpha, 4); REQ_PTR(z_b, 4);
  REQ_PTR(codes, 16);
  OPT_PTR(s_r, 4); OPT_PTR(delta, 4); OPT_PTR(z_u, 4); OPT_PTR(grad_s, 16); OPT_PTR(grad_alpha, 4);
  OPT_PTR(grad_z_b, 4);
  uq::GemmLaunch b{Et, Xt, R, C, T, uq::EPI_STE, nullptr, nullptr, nullptr, 2.0f};
  b.ste = uq::SteParams{W, w_dtype == UQ_BF16 ? 1 : 0, s, s_r, delta, z_u, alpha, z_b, codes,
                        __builtin_ctz(unsigned(g)), int(C / g), lr_f, lr_b, grad_s, grad_alpha, grad_z_b};
  return hip_status(fn, uq::launch_gemm_ste(b, k, static_cast<hipStream_t>(stream)));
}

uq_status uniquan_fold_to_bcq(int64_t R, int64_t C, int k, int g, const void* W, int w_dtype, const float* s,
                              const float* s_r, const float* delta, const float* z_u, const float* alpha,
                              const float* z_b, float* alpha_star, float* z_star, uint8_t* codes_out,
                              int code_src, void* stream) {
  const char* fn = "uniquan_fold_to_bcq";
  if (uq_status st = check_quant_shape(fn, R, C, k, g)) return st;
  if (!is_dtype(w_dtype)) return fail(UQ_EINVAL, "%s: bad dtype", fn);
  if (code_src != 0 && code_src != 1) return fail(UQ_EINVAL, "%s: code_src must be 0 or 1", fn);
  REQ_PTR(alpha, 4); REQ_PTR(z_b, 4); REQ_PTR(alpha_star, 4); REQ_PTR(z_star, 4);
  OPT_PTR(s_r, 4); OPT_PTR(delta, 4); OPT_PTR(z_u, 4);
  if (codes_out != nullptr) {
    REQ_PTR(codes_out, 16);
    REQ_PTR(W, 16);
    if (code_src == 0) REQ_PTR(s, 16);
  }
  uq::FoldLaunch p{R, C, k, g, W, w_dtype, s, s_r, delta, z_u, alpha, z_b, alpha_star, z_star, codes_out, code_src};
  return hip_status(fn, uq::launch_fold(p, static_cast<hipStream_t>(stream)));
}

uq_status uniquan_bcq_dequant(int64_t R, int64_t C, int k, int g, const uint8_t* codes, const float* alpha,
                              const float* z_b, void* W_out, int out_dtype, void* stream) {
  const char* fn = "uniquan_bcq_dequant";
  if (uq_status st = check_quant_shape(fn, R, C, k, g)) return st;
  if (!is_dtype(out_dtype)) return fail(UQ_EINVAL, "%s: bad dtype", fn);
  REQ_PTR(codes, 16); REQ_PTR(alpha, 4); REQ_PTR(z_b, 4); REQ_PTR(W_out, 16);
  uq::DequantLaunch p{R, C, k, g, codes, alpha, z_b, W_out, out_dtype};
  return hip_status(fn, uq::launch_dequant(p, static_cast<hipStream_t>(stream)));
}

uq_status uniquan_init_greedy(int64_t R, int64_t C, int k, int g, const void* W, int w_dtype, const float* s,
                              const float* s_r, const float* delta, const float* z_u, const float* z_b,
                              float* alpha, void* stream) {
  const char* fn = "uniquan_init_greedy";
  if (uq_status st = check_quant_shape(fn, R, C, k, g)) return st;
  if (!is_dtype(w_dtype)) return fail(UQ_EINVAL, "%s: bad dtype", fn);
  REQ_PTR(W, 16); REQ_PTR(s, 16); REQ_PTR(z_b, 4); REQ_PTR(alpha, 4);
  OPT_PTR(s_r, 4); OPT_PTR(delta, 4); OPT_PTR(z_u, 4);
  uq::GreedyLaunch p{R, C, k, g, W, w_dtype, s, s_r, delta, z_u, z_b, alpha};
  return hip_status(fn, uq::launch_greedy(p, static_cast<hipStream_t>(stream)));
}

uq_status uniquan_init_unified(int64_t R, int64_t C, int k, int g, const void* W, int w_dtype, int grid_G,
                               int alt_T, int clip, float* delta, float* z_u, float* alpha, float* z_b,
                               uint8_t* codes, float* err, float* s, float* s_r, void* stream) {
  const char* fn = "uniquan_init_unified";
  if (uq_status st = check_quant_shape(fn, R, C, k, g)) return st;
  if (k > 4) return fail(UQ_EUNSUPPORTED, "%s: k = %d, supported 1..4", fn, k);
  if (g > 16384) return fail(UQ_EUNSUPPORTED, "%s: g = %d, supported up to 16384", fn, g);
  if (!is_dtype(w_dtype)) return fail(UQ_EINVAL, "%s: bad dtype", fn);
  if (grid_G < 1 || grid_G > 4096) return fail(UQ_EINVAL, "%s: grid_G = %d, must be in 1..4096", fn, grid_G);
  if (alt_T < 0 || alt_T > 10000) return fail(UQ_EINVAL, "%s: alt_T = %d, must be in 0..10000", fn, alt_T);
  if (clip < 0 || clip > 2) return fail(UQ_EINVAL, "%s: clip = %d, must be 0, 1 or 2", fn, clip);
  REQ_PTR(W, 16); REQ_PTR(delta, 4); REQ_PTR(z_u, 4); REQ_PTR(alpha, 4); REQ_PTR(z_b, 4);
  OPT_PTR(codes, 8); OPT_PTR(err, 4); OPT_PTR(s, 16); OPT_PTR(s_r, 4);
  uq::InitUnifiedLaunch p{R, C, k, g, W, w_dtype, grid_G, alt_T, clip,
                          delta, z_u, alpha, z_b, codes, err, s, s_r};
  return hip_status(fn, uq::launch_init_unified(p, static_cast<hipStream_t>(stream)));
}

// Shape rules of the deployment form: 16-byte plane words cover 128 columns
// and each word lies inside one group.
static uq_status check_bcq_shape(const char* fn, int64_t R, int64_t C, int k, int g) {
  if (R < 1 || C < 1) return fail(UQ_EINVAL, "%s: R=%lld and C=%lld must be >= 1", fn, (long long)R, (long long)C);
  if (k < 1 || k > 4) return fail(UQ_EUNSUPPORTED, "%s: k=%d, supported 1..4", fn, k);
  if (C % 128 != 0) return fail(UQ_EUNSUPPORTED, "%s: C=%lld must be a multiple of 128", fn, (long long)C);
  // column slabs form the grid's second dimension (at most 65535)
  if (C > (int64_t(1) << 22)) return fail(UQ_EUNSUPPORTED, "%s: C=%lld > 2^22 is not supported", fn, (long long)C);
  if (g < 128 || g % 128 != 0) return fail(UQ_EUNSUPPORTED, "%s: g=%d must be a multiple of 128", fn, g);
  if (C % g != 0) return fail(UQ_EINVAL, "%s: g=%d must divide C=%lld", fn, g, (long long)C);
  if (R >= (int64_t(1) << 31) || R > (int64_t(1) << 40) / C)
    return fail(UQ_EUNSUPPORTED, "%s: R*C too large", fn);
  return UQ_OK;
}

uq_status uniquan_bcq_pack(int64_t R, int64_t C, int k, int g, const uint8_t* codes, const float* alpha_star,
                           const float* z_star, uint32_t* planes, uint16_t* alpha16, uint16_t* z16,
                           void* stream) {
  const char* fn = "uniquan_bcq_pack";
  if (uq_status st = check_bcq_shape(fn, R, C, k, g)) return st;
  REQ_PTR(codes, 16); REQ_PTR(alpha_star, 4); REQ_PTR(z_star, 4);
  REQ_PTR(planes, 16); REQ_PTR(alpha16, 2); REQ_PTR(z16, 2);
  uq::BcqPackLaunch p{R, C, k, g, codes, alpha_star, z_star, planes, alpha16, z16};
  return hip_status(fn, uq::launch_bcq_pack(p, static_cast<hipStream_t>(stream)));
}

size_t uniquan_bcq_matmul_ws(int T, int64_t R, int64_t C) {
  if (T < 1 || R < 1 || C < 128) return 0;
  const int64_t slabs = uq::bcq_slabs(R, C / 128 * 128);
  return slabs > 1 ? size_t(slabs) * size_t(T) * size_t(R) : 0;
}

uq_status uniquan_bcq_matmul(int T, int64_t R, int64_t C, int k, int g, const uint16_t* X, const uint32_t* planes,
                             const uint16_t* alpha16, const uint16_t* z16, float* Y, float* partials_ws,
                             size_t partials_len, void* stream) {
  const char* fn = "uniquan_bcq_matmul";
  if (uq_status st = check_bcq_shape(fn, R, C, k, g)) return st;
  if (T < 1 || T > 8) return fail(UQ_EUNSUPPORTED, "%s: T=%d, supported 1..8", fn, T);
  REQ_PTR(X, 8); REQ_PTR(planes, 16); REQ_PTR(alpha16, 2); REQ_PTR(z16, 2); REQ_PTR(Y, 4);
  const size_t need = uniquan_bcq_matmul_ws(T, R, C);
  if (need > 0) {
    REQ_PTR(partials_ws, 4);
    if (partials_len < need)
      return fail(UQ_EINVAL, "%s: partials_len=%zu, need %zu floats (uniquan_bcq_matmul_ws)", fn, partials_len, need);
  }
  uq::BcqMatmulLaunch p{T, R, C, k, g, X, planes, alpha16, z16, Y, partials_ws};
  return hip_status(fn, uq::launch_bcq_matmul(p, static_cast<hipStream_t>(stream)));
}

uq_status uniquan_gemm_nt(int64_t M, int64_t N, int64_t K, const uint16_t* A, const uint16_t* B, void* out,
                          int out_dtype, float scale, void* stream) {
  const char* fn = "uniquan_gemm_nt";
  if (M < 1 || N < 1 || K < 1) return fail(UQ_EINVAL, "%s: M, N, K must be >= 1", fn);
  if (N % 8 != 0 || K % 8 != 0) return fail(UQ_EINVAL, "%s: N=%lld and K=%lld must be multiples of 8", fn,
                                            (long long)N, (long long)K);
  if (N >= (int64_t(1) << 26) || K >= (int64_t(1) << 31) || M >= (int64_t(1) << 31) ||
      M * K >= (int64_t(1) << 40) || N * K >= (int64_t(1) << 40) || M * N >= (int64_t(1) << 40))
    return fail(UQ_EUNSUPPORTED, "%s: shape too large", fn);
  if (!is_dtype(out_dtype)) return fail(UQ_EINVAL, "%s: bad dtype", fn);
  REQ_PTR(A, 16); REQ_PTR(B, 16); REQ_PTR(out, 16);
  uq::GemmLaunch g{A, B, M, N, K, out_dtype == UQ_BF16 ? uq::EPI_GRAD_BF16 : uq::EPI_GRAD_F32, nullptr, out, nullptr,
                   scale};
  return hip_status(fn, uq::launch_gemm(g, static_cast<hipStream_t>(stream)));
}

uq_status uniquan_gemm_nt_residual(int64_t M, int64_t N, int64_t K, const uint16_t* A, const uint16_t* B,
                                   const float* R, float* out, void* stream) {
  const char* fn = "uniquan_gemm_nt_residual";
  if (M < 1 || N < 1 || K < 1) return fail(UQ_EINVAL, "%s: M, N, K must be >= 1", fn);
  if (N % 8 != 0 || K % 8 != 0) return fail(UQ_EINVAL, "%s: N=%lld and K=%lld must be multiples of 8", fn,
                                            (long long)N, (long long)K);
  if (N >= (int64_t(1) << 26) || K >= (int64_t(1) << 31) || M >= (int64_t(1) << 31) ||
      M * K >= (int64_t(1) << 40) || N * K >= (int64_t(1) << 40) || M * N >= (int64_t(1) << 40))
    return fail(UQ_EUNSUPPORTED, "%s: shape too large", fn);
  REQ_PTR(A, 16); REQ_PTR(B, 16); REQ_PTR(R, 16); REQ_PTR(out, 16);
  uq::GemmLaunch g{A, B, M, N, K, uq::EPI_RESID, nullptr, out, nullptr, 1.0f};
  g.Rres = R;
  return hip_status(fn, uq::launch_gemm(g, static_cast<hipStream_t>(stream)));
}

uq_status uniquan_gemm(int64_t M, int64_t N, int64_t K, const uint16_t* A, int a_kslow, const uint16_t* B, int b_kslow,
                       void* out, int out_dtype, float scale, void* stream) {
  const char* fn = "uniquan_gemm";
  if (M < 1 || N < 1 || K < 1) return fail(UQ_EINVAL, "%s: M, N, K must be >= 1", fn);
  if ((a_kslow != 0 && a_kslow != 1) || (b_kslow != 0 && b_kslow != 1))
    return fail(UQ_EINVAL, "%s: a_kslow and b_kslow must be 0 or 1", fn);
  if (!a_kslow && !b_kslow) return uniquan_gemm_nt(M, N, K, A, B, out, out_dtype, scale, stream);
  if (N % 8 != 0 || K % 32 != 0 || (a_kslow && M % 8 != 0))
    return fail(UQ_EINVAL, "%s: N=%lld%s must be a multiple of 8 and K=%lld of 32", fn, (long long)N,
                a_kslow ? " and M" : "", (long long)K);
  if (N >= (int64_t(1) << 26) || K >= (int64_t(1) << 31) || M >= (int64_t(1) << 31) ||
      M * K >= (int64_t(1) << 40) || N * K >= (int64_t(1) << 40) || M * N >= (int64_t(1) << 40))
    return fail(UQ_EUNSUPPORTED, "%s: shape too large", fn);
  if (!is_dtype(out_dtype)) return fail(UQ_EINVAL, "%s: bad dtype", fn);
  REQ_PTR(A, 16); REQ_PTR(B, 16); REQ_PTR(out, 16);
  uq::GemmLaunch g{A, B, M, N, K, out_dtype == UQ_BF16 ? uq::EPI_GRAD_BF16 : uq::EPI_GRAD_F32, nullptr, out, nullptr,
                   scale};
  g.ta = a_kslow;
  g.tb = b_kslow;
  return hip_status(fn, uq::launch_gemm(g, static_cast<hipStream_t>(stream)));
}

uq_status uniquan_gemm_swiglu(int64_t T, int64_t I, int64_t K, const uint16_t* X, const uint16_t* Wg,
                              const uint16_t* Wu, uint16_t* G, uint16_t* U, uint16_t* H, void* stream) {
  const char* fn = "uniquan_gemm_swiglu";
  if (T < 1 || I < 1 || K < 1) return fail(UQ_EINVAL, "%s: T, I, K must be >= 1", fn);
  if (I % 32 != 0 || K % 32 != 0)
    return fail(UQ_EINVAL, "%s: I=%lld and K=%lld must be multiples of 32", fn, (long long)I, (long long)K);
  if (2 * I >= (int64_t(1) << 26) || K >= (int64_t(1) << 31) || T >= (int64_t(1) << 31) ||
      T * K >= (int64_t(1) << 40) || I * K >= (int64_t(1) << 40) || T * I >= (int64_t(1) << 40))
    return fail(UQ_EUNSUPPORTED, "%s: shape too large", fn);
  REQ_PTR(X, 16); REQ_PTR(Wg, 16); REQ_PTR(Wu, 16); REQ_PTR(G, 8); REQ_PTR(U, 8); REQ_PTR(H, 8);
  uq::GemmLaunch g{X, Wg, T, 2 * I, K, uq::EPI_SWIGLU, nullptr, G, nullptr, 1.0f};
  g.swiglu = uq::SwigluParams{Wu, U, H, I};
  return hip_status(fn, uq::launch_gemm(g, static_cast<hipStream_t>(stream)));
}

uq_status uniquan_gemm_silu_bwd(int64_t T, int64_t I, int64_t K, const uint16_t* E, const uint16_t* Wd, float scale,
                                const uint16_t* G, const uint16_t* U, uint16_t* dG, uint16_t* dU, int64_t ld_d,
                                void* stream) {
  const char* fn = "uniquan_gemm_silu_bwd";
  if (T < 1 || I < 1 || K < 1) return fail(UQ_EINVAL, "%s: T, I, K must be >= 1", fn);
  if (I % 8 != 0 || K % 32 != 0)
    return fail(UQ_EINVAL, "%s: I=%lld must be a multiple of 8 and K=%lld of 32", fn, (long long)I, (long long)K);
  if (ld_d == 0) ld_d = I;
  if (ld_d < I || ld_d % 4 != 0)
    return fail(UQ_EINVAL, "%s: ld_d=%lld must be >= I=%lld and a multiple of 4", fn, (long long)ld_d, (long long)I);
  if (I >= (int64_t(1) << 26) || K >= (int64_t(1) << 31) || T >= (int64_t(1) << 31) ||
      T * K >= (int64_t(1) << 40) || I * K >= (int64_t(1) << 40) || T * ld_d >= (int64_t(1) << 40))
    return fail(UQ_EUNSUPPORTED, "%s: shape too large", fn);
  REQ_PTR(E, 16); REQ_PTR(Wd, 16); REQ_PTR(G, 8); REQ_PTR(U, 8); REQ_PTR(dG, 8); REQ_PTR(dU, 8);
  uq::GemmLaunch g{E, Wd, T, I, K, uq::EPI_SWIGLU_BWD, nullptr, dG, nullptr, scale};
  g.tb = 1;
  g.swiglu.G_in = G;
  g.swiglu.U_in = U;
  g.swiglu.dU = dU;
  g.swiglu.ldo = ld_d;
  return hip_status(fn, uq::launch_gemm(g, static_cast<hipStream_t>(stream)));
}

uq_status uniquan_silu_mul_fwd(int64_t n, const uint16_t* G, const uint16_t* U, uint16_t* H, void* stream) {
  const char* fn = "uniquan_silu_mul_fwd";
  if (n < 8 || n % 8 != 0) return fail(UQ_EINVAL, "%s: n=%lld must be a positive multiple of 8", fn, (long long)n);
  REQ_PTR(G, 16); REQ_PTR(U, 16); REQ_PTR(H, 16);
  return hip_status(fn, uq::launch_silu_mul_fwd(n, G, U, H, static_cast<hipStream_t>(stream)));
}

uq_status uniquan_silu_mul_bwd(int64_t n, const uint16_t* dH, const uint16_t* G, const uint16_t* U, uint16_t* dG,
                               uint16_t* dU, void* stream) {
  const char* fn = "uniquan_silu_mul_bwd";
  if (n < 8 || n % 8 != 0) return fail(UQ_EINVAL, "%s: n=%lld must be a positive multiple of 8", fn, (long long)n);
  REQ_PTR(dH, 16); REQ_PTR(G, 16); REQ_PTR(U, 16); REQ_PTR(dG, 16); REQ_PTR(dU, 16);
  return hip_status(fn, uq::launch_silu_mul_bwd(n, dH, G, U, dG, dU, static_cast<hipStream_t>(stream)));
}

uq_status uniquan_gemm_nt_batched(int64_t M, int64_t N, int64_t K, int64_t batch, const uint16_t* A, int64_t stride_a,
                                  const uint16_t* B, int64_t stride_b, void* out, int64_t stride_out, int out_dtype,
                                  float scale, int causal, void* stream) {
  const char* fn = "uniquan_gemm_nt_batched";
  if (M < 1 || N < 1 || K < 1) return fail(UQ_EINVAL, "%s: M, N, K must be >= 1", fn);
  if (batch < 1 || batch > 65535) return fail(UQ_EINVAL, "%s: batch=%lld must be in 1..65535", fn, (long long)batch);
  if (N % 8 != 0 || K % 8 != 0) return fail(UQ_EINVAL, "%s: N=%lld and K=%lld must be multiples of 8", fn,
                                            (long long)N, (long long)K);
  if (N >= (int64_t(1) << 26) || K >= (int64_t(1) << 31) || M >= (int64_t(1) << 31) ||
      M * K >= (int64_t(1) << 40) || N * K >= (int64_t(1) << 40) || M * N >= (int64_t(1) << 40))
    return fail(UQ_EUNSUPPORTED, "%s: shape too large", fn);
  if (!is_dtype(out_dtype)) return fail(UQ_EINVAL, "%s: bad dtype", fn);
  if (stride_a < 0 || stride_b < 0 || stride_a % 8 != 0 || stride_b % 8 != 0)
    return fail(UQ_EINVAL, "%s: operand strides must be non-negative multiples of 8", fn);
  if (stride_out < M * N || stride_out % 8 != 0)
    return fail(UQ_EINVAL, "%s: stride_out=%lld must be a multiple of 8 and >= M*N", fn, (long long)stride_out);
  if ((batch - 1) * stride_out >= (int64_t(1) << 40)) return fail(UQ_EUNSUPPORTED, "%s: batch span too large", fn);
  if (causal < 0 || causal > 3) return fail(UQ_EINVAL, "%s: causal=%d must be 0..3", fn, causal);
  if (causal != 0 && K % 32 != 0) return fail(UQ_EINVAL, "%s: causal modes need K %% 32 == 0", fn);
  if (causal == 1 && M != N) return fail(UQ_EINVAL, "%s: causal mode 1 needs M == N", fn);
  if ((causal == 2 || causal == 3) && M != K) return fail(UQ_EINVAL, "%s: causal modes 2 and 3 need M == K", fn);
  REQ_PTR(A, 16); REQ_PTR(B, 16); REQ_PTR(out, 16);
  uq::GemmLaunch g{A, B, M, N, K, out_dtype == UQ_BF16 ? uq::EPI_GRAD_BF16 : uq::EPI_GRAD_F32, nullptr, out, nullptr,
                   scale};
  g.batch = batch;
  g.bsa = stride_a;
  g.bsb = stride_b;
  g.bso = stride_out * (out_dtype == UQ_BF16 ? 2 : 4);
  g.causal = causal;
  return hip_status(fn, uq::launch_gemm(g, static_cast<hipStream_t>(stream)));
}

uq_status uniquan_add_rmsnorm(int64_t T, int64_t C, const float* X, const float* A, const float* gamma, float* R,
                              uint16_t* Z, float* rinv, void* stream) {
  const char* fn = "uniquan_add_rmsnorm";
  if (T < 1 || C < 8 || C % 8 != 0) return fail(UQ_EINVAL, "%s: T >= 1 and C a positive multiple of 8 required", fn);
  if (A != nullptr && R == nullptr) return fail(UQ_EINVAL, "%s: R must be given with A", fn);
  REQ_PTR(X, 16); REQ_PTR(gamma, 16); REQ_PTR(Z, 8); REQ_PTR(rinv, 4);
  if (A && !aligned(A, 16)) return fail(UQ_EINVAL, "%s: A must be 16-byte aligned", fn);
  if (R && !aligned(R, 16)) return fail(UQ_EINVAL, "%s: R must be 16-byte aligned", fn);
  return hip_status(fn, uq::launch_add_rmsnorm(T, C, X, A, gamma, R, Z, rinv, static_cast<hipStream_t>(stream)));
}

uq_status uniquan_rmsnorm_bwd(int64_t T, int64_t C, const float* dZa, const float* dZb, const float* X,
                              const float* gamma, const float* rinv, const uint16_t* E, float escale, uint16_t* dR,
                              float* dRf, void* stream) {
  const char* fn = "uniquan_rmsnorm_bwd";
  if (T < 1 || C < 8 || C % 8 != 0) return fail(UQ_EINVAL, "%s: T >= 1 and C a positive multiple of 8 required", fn);
  REQ_PTR(dZa, 16); REQ_PTR(X, 16); REQ_PTR(gamma, 16); REQ_PTR(rinv, 4); REQ_PTR(dR, 8);
  if (dZb && !aligned(dZb, 16)) return fail(UQ_EINVAL, "%s: dZb must be 16-byte aligned", fn);
  if (E && !aligned(E, 8)) return fail(UQ_EINVAL, "%s: E must be 8-byte aligned", fn);
  if (dRf && !aligned(dRf, 16)) return fail(UQ_EINVAL, "%s: dRf must be 16-byte aligned", fn);
  return hip_status(fn, uq::launch_rmsnorm_bwd(T, C, dZa, dZb, X, gamma, rinv, E, escale, dR, dRf,
                                               static_cast<hipStream_t>(stream)));
}

static uq_status check_heads(const char* fn, int64_t T, int H, int d, int L, int in_dtype) {
  if (T < 1 || H < 1 || d < 2 || d % 2 != 0 || L < 1 || T % L != 0)
    return fail(UQ_EINVAL, "%s: need T >= 1, H >= 1, even d >= 2 and L dividing T", fn);
  if (T * H * d >= (int64_t(1) << 40) || L >= (1 << 24)) return fail(UQ_EUNSUPPORTED, "%s: shape too large", fn);
  if (!is_dtype(in_dtype)) return fail(UQ_EINVAL, "%s: bad dtype", fn);
  return UQ_OK;
}

uq_status uniquan_rope_split(int64_t T, int H, int d, int L, int group, const void* in, int in_dtype, int rotate,
                             uint16_t* out, void* stream) {
  const char* fn = "uniquan_rope_split";
  const uq_status c = check_heads(fn, T, H, d, L, in_dtype);
  if (c != UQ_OK) return c;
  if (group < 1 || H % group != 0) return fail(UQ_EINVAL, "%s: group=%d must divide H=%d", fn, group, H);
  REQ_PTR(in, in_dtype == UQ_F32 ? 4 : 2); REQ_PTR(out, 2);
  return hip_status(fn, uq::launch_rope_split(T, H, d, L, group, in, in_dtype == UQ_F32, rotate != 0, out,
                                              static_cast<hipStream_t>(stream)));
}

uq_status uniquan_rope_table(int L, int d, float* cs, void* stream) {
  const char* fn = "uniquan_rope_table";
  if (L < 1 || d < 2 || d % 2 != 0 || d > 1024) return fail(UQ_EINVAL, "%s: L=%d >= 1 and even d=%d <= 1024", fn, L, d);
  if (int64_t(L) * d >= (int64_t(1) << 31)) return fail(UQ_EUNSUPPORTED, "%s: L=%d too large", fn, L);
  REQ_PTR(cs, 16);
  return hip_status(fn, uq::launch_rope_table(L, d, cs, static_cast<hipStream_t>(stream)));
}

uq_status uniquan_gemm_heads(int64_t T, int H, int64_t K, const uint16_t* A, const uint16_t* W, int L, int group,
                             int n_rot, const float* cs, uint16_t* out, void* stream) {
  const char* fn = "uniquan_gemm_heads";
  if (T < 1 || H < 1 || K < 1 || L < 1) return fail(UQ_EINVAL, "%s: T, H, K, L must be >= 1", fn);
  if (K % 32 != 0) return fail(UQ_EINVAL, "%s: K=%lld must be a multiple of 32", fn, (long long)K);
  if (T % L != 0) return fail(UQ_EINVAL, "%s: L=%d must divide T=%lld", fn, L, (long long)T);
  if (group < 1 || H % group != 0) return fail(UQ_EINVAL, "%s: group=%d must divide H=%d", fn, group, H);
  const int64_t N = int64_t(H) * 128;
  if (N >= (int64_t(1) << 26) || K >= (int64_t(1) << 31) || T >= (int64_t(1) << 31) ||
      T * K >= (int64_t(1) << 40) || N * K >= (int64_t(1) << 40) || T * N >= (int64_t(1) << 40))
    return fail(UQ_EUNSUPPORTED, "%s: shape too large", fn);
  if (n_rot < 0) return fail(UQ_EINVAL, "%s: n_rot=%d must be >= 0", fn, n_rot);
  if (n_rot > H) n_rot = H;
  if (n_rot > 0 && group > 1 && n_rot < H)
    return fail(UQ_EINVAL, "%s: rotating only some heads needs group 1", fn);
  REQ_PTR(A, 16); REQ_PTR(W, 16); REQ_PTR(out, 8);
  if (n_rot) REQ_PTR(cs, 32);
  uq::GemmLaunch g{A, W, T, N, K, n_rot ? uq::EPI_HEADS_ROT : uq::EPI_HEADS, nullptr, out, nullptr, 1.0f};
  g.heads = uq::HeadsParams{cs, L, H, group, n_rot};
  return hip_status(fn, uq::launch_gemm(g, static_cast<hipStream_t>(stream)));
}

uq_status uniquan_rope_merge(int64_t T, int H, int d, int L, int group, int nsum, const void* in, int in_dtype,
                             int rotate, uint16_t* out, int64_t ld_out, void* stream) {
  const char* fn = "uniquan_rope_merge";
  const uq_status c = check_heads(fn, T, H, d, L, in_dtype);
  if (c != UQ_OK) return c;
  if (group < 1 || H % group != 0) return fail(UQ_EINVAL, "%s: group=%d must divide H=%d", fn, group, H);
  if (nsum < 1 || nsum > 256 || nsum * T * H * d >= (int64_t(1) << 40))
    return fail(UQ_EINVAL, "%s: nsum=%d must be in 1..256", fn, nsum);
  if (ld_out == 0) ld_out = int64_t(H) * d;
  if (ld_out < int64_t(H) * d || T * ld_out >= (int64_t(1) << 40))
    return fail(UQ_EINVAL, "%s: ld_out=%lld must be >= H d=%lld", fn, (long long)ld_out, (long long)(int64_t(H) * d));
  REQ_PTR(in, in_dtype == UQ_F32 ? 4 : 2); REQ_PTR(out, 2);
  return hip_status(fn, uq::launch_rope_merge(T, H, d, L, group, nsum, in, in_dtype == UQ_F32, rotate != 0, out,
                                              ld_out, static_cast<hipStream_t>(stream)));
}

uq_status uniquan_softmax_causal(int64_t rows, int L, const float* S, uint16_t* P, void* stream) {
  const char* fn = "uniquan_softmax_causal";
  if (L < 1 || rows < 1 || rows % L != 0) return fail(UQ_EINVAL, "%s: rows must be a positive multiple of L", fn);
  if (rows * L >= (int64_t(1) << 40)) return fail(UQ_EUNSUPPORTED, "%s: shape too large", fn);
  REQ_PTR(S, 4); REQ_PTR(P, 2);
  return hip_status(fn, uq::launch_softmax_causal(rows, L, S, P, static_cast<hipStream_t>(stream)));
}

uq_status uniquan_softmax_causal_bwd(int64_t rows, int L, const float* dP, const uint16_t* P, uint16_t* dS,
                                     void* stream) {
  const char* fn = "uniquan_softmax_causal_bwd";
  if (L < 1 || rows < 1 || rows % L != 0) return fail(UQ_EINVAL, "%s: rows must be a positive multiple of L", fn);
  if (rows * L >= (int64_t(1) << 40)) return fail(UQ_EUNSUPPORTED, "%s: shape too large", fn);
  REQ_PTR(dP, 4); REQ_PTR(P, 2); REQ_PTR(dS, 2);
  return hip_status(fn, uq::launch_softmax_bwd(rows, L, dP, P, dS, static_cast<hipStream_t>(stream)));
}

uq_status uniquan_transpose_bf16_batched(int64_t batch, int64_t R, int64_t C, const uint16_t* in, uint16_t* out,
                                         void* stream) {
  const char* fn = "uniquan_transpose_bf16_batched";
  if (batch < 1 || batch > 65535 || R < 1 || C < 1)
    return fail(UQ_EINVAL, "%s: need 1 <= batch <= 65535 and R, C >= 1", fn);
  if (batch * R * C >= (int64_t(1) << 40) || ((R + 63) / 64) * ((C + 63) / 64) >= (int64_t(1) << 31))
    return fail(UQ_EUNSUPPORTED, "%s: shape too large", fn);
  REQ_PTR(in, 8); REQ_PTR(out, 8);
  return hip_status(fn, uq::launch_transpose_batched(batch, R, C, in, out, static_cast<hipStream_t>(stream)));
}

size_t uniquan_block_loss_ws(void) { return uq::block_loss_ws(); }

size_t uniquan_gemm_block_loss_ws(int64_t T, int64_t C) {
  if (T < 1 || C < 1) return 0;
  return uq::gemm_workgroups(T, C, uq::EPI_LOSS_BLOCK);
}

uq_status uniquan_gemm_block_loss(int64_t T, int64_t C, int64_t K, const uint16_t* H, const uint16_t* Wd,
                                  const float* R, const float* Yref, uint16_t* E, float* partials, size_t partials_len,
                                  float* loss, void* stream) {
  const char* fn = "uniquan_gemm_block_loss";
  if (T < 1 || C < 1 || K < 1) return fail(UQ_EINVAL, "%s: T, C, K must be >= 1", fn);
  if (C % 8 != 0 || K % 8 != 0)
    return fail(UQ_EINVAL, "%s: C=%lld and K=%lld must be multiples of 8", fn, (long long)C, (long long)K);
  if (C >= (int64_t(1) << 26) || K >= (int64_t(1) << 31) || T >= (int64_t(1) << 31) ||
      T * K >= (int64_t(1) << 40) || C * K >= (int64_t(1) << 40) || T * C >= (int64_t(1) << 40))
    return fail(UQ_EUNSUPPORTED, "%s: shape too large", fn);
  const size_t need = uniquan_gemm_block_loss_ws(T, C);
  if (partials_len < need) return fail(UQ_EINVAL, "%s: partials_len=%zu < %zu", fn, partials_len, need);
  REQ_PTR(H, 16); REQ_PTR(Wd, 16); REQ_PTR(R, 16); REQ_PTR(Yref, 16); REQ_PTR(E, 8); REQ_PTR(partials, 4);
  REQ_PTR(loss, 4);
  const hipStream_t st = static_cast<hipStream_t>(stream);
  uq::GemmLaunch g{H, Wd, T, C, K, uq::EPI_LOSS_BLOCK, Yref, E, partials, 1.0f};
  g.Rres = R;
  if (uq_status s = hip_status(fn, uq::launch_gemm(g, st))) return s;
  return hip_status(fn, uq::launch_reduce_loss(partials, int64_t(need), loss, st));
}

uq_status uniquan_block_loss(int64_t n, const float* R, const float* M, const float* Yref, uint16_t* E,
                             float* partials, size_t partials_len, float* loss, void* stream) {
  const char* fn = "uniquan_block_loss";
  if (n < 1) return fail(UQ_EINVAL, "%s: n must be >= 1", fn);
  if (partials_len < uq::block_loss_ws())
    return fail(UQ_EINVAL, "%s: partials has %zu floats, needs %zu", fn, partials_len, uq::block_loss_ws());
  REQ_PTR(R, 4); REQ_PTR(M, 4); REQ_PTR(Yref, 4); REQ_PTR(E, 2); REQ_PTR(partials, 4); REQ_PTR(loss, 4);
  return hip_status(fn, uq::launch_block_loss(n, R, M, Yref, E, partials, loss, static_cast<hipStream_t>(stream)));
}

uq_status uniquan_sgd(int64_t n, float* theta, const float* grad, float lr, void* stream) {
  const char* fn = "uniquan_sgd";
  if (n < 1) return fail(UQ_EINVAL, "%s: n must be >= 1", fn);
  REQ_PTR(theta, 4); REQ_PTR(grad, 4);
  return hip_status(fn, uq::launch_sgd(n, theta, grad, lr, static_cast<hipStream_t>(stream)));
}

static uq_status check_attn(const char* fn, int64_t batch, int64_t kv_batch, int L, int d) {
  if (batch < 1 || kv_batch < 1 || batch % kv_batch != 0)
    return fail(UQ_EINVAL, "%s: batch=%lld must be a positive multiple of kv_batch=%lld", fn, (long long)batch,
                (long long)kv_batch);
  if (batch > 65535) return fail(UQ_EUNSUPPORTED, "%s: batch=%lld > 65535", fn, (long long)batch);
  if (d != 128) return fail(UQ_EUNSUPPORTED, "%s: d=%d, supported 128", fn, d);
  if (L < 32 || L % 32 != 0) return fail(UQ_EUNSUPPORTED, "%s: L=%d must be a positive multiple of 32", fn, L);
  if (int64_t(L) * L >= (int64_t(1) << 31)) return fail(UQ_EUNSUPPORTED, "%s: L=%d too large", fn, L);
  return UQ_OK;
}

static uq_status check_tok(const char* fn, int64_t batch, int64_t kv_batch, int tok_seqs, int group) {
  if (tok_seqs < 0 || (tok_seqs > 0 && (batch % tok_seqs != 0 || kv_batch % tok_seqs != 0)))
    return fail(UQ_EINVAL, "%s: tok_seqs=%d must be 0 or divide batch and kv_batch", fn, tok_seqs);
  if (tok_seqs > 0 && (group < 1 || (batch / tok_seqs) % group != 0))
    return fail(UQ_EINVAL, "%s: group=%d must divide the query heads", fn, group);
  if (tok_seqs > 0 && kv_batch == batch && group != 1)
    return fail(UQ_EINVAL, "%s: group=%d with one query head per key/value head (must be 1)", fn, group);
  return UQ_OK;
}

uq_status uniquan_attn_fwd(int64_t batch, int64_t kv_batch, int L, int d, const uint16_t* Q, const uint16_t* K,
                           const uint16_t* V, float scale, uint16_t* O, float* row_lse, int tok_seqs, int group,
                           void* stream) {
  const char* fn = "uniquan_attn_fwd";
  if (uq_status st = check_attn(fn, batch, kv_batch, L, d)) return st;
  if (uq_status st = check_tok(fn, batch, kv_batch, tok_seqs, group)) return st;
  REQ_PTR(Q, 16); REQ_PTR(K, 16); REQ_PTR(V, 16); REQ_PTR(O, 16); REQ_PTR(row_lse, 16);
  uq::AttnLaunch q{};
  q.batch = batch; q.kv_batch = kv_batch; q.L = L; q.scale = scale;
  q.Q = Q; q.K = K; q.V = V; q.O_out = O; q.lse = row_lse;
  q.tok_seqs = tok_seqs; q.group = group;
  return hip_status(fn, uq::launch_attn_fwd(q, static_cast<hipStream_t>(stream)));
}

uq_status uniquan_attn_bwd(int64_t batch, int64_t kv_batch, int L, int d, const uint16_t* Q, const uint16_t* K,
                           const uint16_t* V, const uint16_t* O, const uint16_t* dO, const float* row_lse, float scale,
                           float* delta, void* dQ, void* dK, void* dV, int tok_seqs, int group, const float* cs,
                           void* stream) {
  const char* fn = "uniquan_attn_bwd";
  if (uq_status st = check_attn(fn, batch, kv_batch, L, d)) return st;
  if (uq_status st = check_tok(fn, batch, kv_batch, tok_seqs, group)) return st;
  REQ_PTR(Q, 16); REQ_PTR(K, 16); REQ_PTR(V, 16); REQ_PTR(O, 16);
  REQ_PTR(dO, 16); REQ_PTR(row_lse, 16); REQ_PTR(delta, 16);
  REQ_PTR(dQ, 16); REQ_PTR(dK, 16); REQ_PTR(dV, 16);
  if (tok_seqs > 0) REQ_PTR(cs, 32);
  uq::AttnLaunch q{};
  q.batch = batch; q.kv_batch = kv_batch; q.L = L; q.scale = scale;
  q.Q = Q; q.K = K; q.V = V; q.O = O; q.dO = dO;
  q.tok_seqs = tok_seqs; q.group = group; q.cs = cs;
  const bool bf_kv = tok_seqs > 0 && kv_batch == batch;  // token-major bf16 dK, dV
  if (tok_seqs > 0) q.dQ_tok = static_cast<uint16_t*>(dQ);
  if (bf_kv) {
    q.dK_tok = static_cast<uint16_t*>(dK);
    q.dV_tok = static_cast<uint16_t*>(dV);
  }
  q.lse = const_cast<float*>(row_lse); q.delta = delta;
  if (tok_seqs == 0) q.dQ = static_cast<float*>(dQ);
  if (!bf_kv) {
    q.dK = static_cast<float*>(dK);
    q.dV = static_cast<float*>(dV);
  }
  return hip_status(fn, uq::launch_attn_bwd(q, static_cast<hipStream_t>(stream)));
}

double uniquan_probe_mfma_flops(int iters) {
  return 2.0 * 32 * 32 * 16 * double(uq::PROBE_MFMA_CHAINS) * double(iters) * (4.0 * uq::PROBE_MFMA_BLOCKS);
}

uq_status uniquan_probe_stream(int op, int64_t n_bytes, const void* src, void* dst, void* sink, int blocks,
                               void* stream) {
  const char* fn = "uniquan_probe_stream";
  if (op < 0 || op > 2) return fail(UQ_EINVAL, "%s: op=%d must be 0 (read), 1 (write) or 2 (copy)", fn, op);
  if (n_bytes < 16 || n_bytes % 16 != 0) return fail(UQ_EINVAL, "%s: n_bytes must be a positive multiple of 16", fn);
  if (blocks < 1 || blocks > (1 << 20)) return fail(UQ_EINVAL, "%s: blocks=%d must be in [1, 2^20]", fn, blocks);
  if (op != 1) REQ_PTR(src, 16);
  if (op != 0) REQ_PTR(dst, 16);
  REQ_PTR(sink, 16);
  return hip_status(fn, uq::launch_probe_stream(op, n_bytes / 16, src, dst, sink, blocks,
                                                static_cast<hipStream_t>(stream)));
}

uq_status uniquan_probe_mfma(int iters, float* sink, void* stream) {
  const char* fn = "uniquan_probe_mfma";
  if (iters < 1 || iters > (1 << 24)) return fail(UQ_EINVAL, "%s: iters=%d must be in [1, 2^24]", fn, iters);
  REQ_PTR(sink, 16);
  return hip_status(fn, uq::launch_probe_mfma(iters, reinterpret_cast<float*>(sink), static_cast<hipStream_t>(stream)));
}

}  // extern "C"
