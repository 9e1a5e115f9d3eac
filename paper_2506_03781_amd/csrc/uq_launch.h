// Internal launch interface between the C-ABI layer (abi.hip) and the
// kernel files.  Arguments are already validated when these are called.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace uq {

struct FqFwdLaunch {
  int64_t R, C;
  int k, g;
  const void* W; int w_dtype;
  const float* s; const float* s_r; const float* delta; const float* z_u;
  const float* alpha; const float* z_b;
  int mode;
  uint8_t* codes;
  void* W_hat; int w_hat_dtype;
  int resid;  // store What - W instead of What
};

struct FqBwdLaunch {
  int64_t R, C;
  int k, g;
  const void* W; int w_dtype;
  const float* s; const float* s_r; const float* delta; const float* z_u;
  const float* alpha; const float* z_b;
  const uint8_t* codes;
  const void* grad_W_hat; int grad_dtype;
  float* grad_s; float* grad_alpha; float* grad_z_b;
  float* grad_delta; float* grad_z_u; float* grad_s_r; float* group_ws;
  int update;            // uniquan_fq_bwd_sgd: apply SGD in place
  float lr_f, lr_b;
};

// Straight-through backward + SGD of one step fused with the next step's
// forward (uniquan_fq_step).
struct FqStepLaunch {
  int64_t R, C;
  int k, g;
  const void* W; int w_dtype;
  float* s; const float* s_r; const float* delta; const float* z_u;
  float* alpha; float* z_b;
  uint8_t* codes;
  const void* grad_W_hat; int grad_dtype;
  float lr_f, lr_b;
  int mode;
  void* W_hat; int w_hat_dtype;
  int resid;
};

struct FoldLaunch {
  int64_t R, C;
  int k, g;
  const void* W; int w_dtype;
  const float* s; const float* s_r; const float* delta; const float* z_u;
  const float* alpha; const float* z_b;
  float* alpha_star; float* z_star; uint8_t* codes; int code_src;
};

struct DequantLaunch {
  int64_t R, C;
  int k, g;
  const uint8_t* codes; const float* alpha; const float* z_b;
  void* W_out; int out_dtype;
};

struct GreedyLaunch {
  int64_t R, C;
  int k, g;
  const void* W; int w_dtype;
  const float* s; const float* s_r; const float* delta; const float* z_u;
  const float* z_b; float* alpha;
};

struct InitUnifiedLaunch {
  int64_t R, C;
  int k, g;
  const void* W; int w_dtype;
  int grid_G, alt_T, clip;
  float* delta; float* z_u; float* alpha; float* z_b;
  uint8_t* codes; float* err; float* s; float* s_r;
};

// GEMM epilogues of the reconstruction contractions.
// Straight-through backward with the SGD update, run in the weight-gradient
// GEMM's epilogue on the fp32 gradient tile (see uniquan_layer_grad_ste_sgd).
struct SteParams {
  const void* W; int w_bf16;
  float* s; const float* s_r; const float* delta; const float* z_u;
  float* alpha; float* z_b; const uint8_t* codes;
  int logg, gpr;
  float lr_f, lr_b;
  float* grad_s; float* grad_alpha; float* grad_z_b;  // optional copies of the gradients
};

enum GemmEpi : int {
  EPI_TARGET = 0,     // out fp32 = acc
  EPI_LOSS = 1,       // e = acc - Yt; out bf16 = e; partial sum of e^2 per workgroup
  EPI_GRAD_BF16 = 2,  // out bf16 = scale * acc
  EPI_STE = 16,       // EPI_STE + k: scale * acc is dL/dWhat; straight-through backward + SGD in place
  EPI_GRAD_F32 = 3,   // out fp32 = scale * acc
  EPI_LOSS_RES = 4,   // EPI_LOSS without a target (A holds What - W); chosen when Yt is NULL
  EPI_HEADS = 5,      // out bf16 head-major [H, M, 128] = scale * acc (column block h to head slot h)
  EPI_HEADS_ROT = 6,  // EPI_HEADS with the rotary rotation of each head's pairs (i, i + 64)
  EPI_SWIGLU = 7,     // gate and up products in one: G, U, H = silu(G) U (bf16), see SwigluParams
  EPI_SWIGLU_BWD = 8, // dH = bf16(scale acc) [M x N], then dG, dU of the SiLU product (SwigluParams)
  EPI_LOSS_BLOCK = 9, // e = (Rres + acc) - Yt (fp32, row-major [M x N]); out bf16 = e; partial sum of e^2
  EPI_RESID = 10,     // out fp32 = Rres + scale acc (Rres fp32 row-major [M x N]; may alias out)
};

// silu(g) u of the SiLU-gated MLP on bf16-rounded g and u (fp32 arithmetic:
// (g sigma(g)) u, sigma(x) = 1 / (1 + exp(-x))); one definition for the
// stand-alone kernel and the product's epilogue.
__device__ __forceinline__ float silu_mul(float g, float u) { return g * (1.0f / (1.0f + expf(-g))) * u; }

// Its backward on bf16-rounded dh, g, u: dg = (dh u) silu'(g), du = dh silu(g),
// silu'(x) = sigma(x) (1 + x (1 - sigma(x))).
__device__ __forceinline__ void silu_mul_grad(float dh, float g, float u, float& dg, float& du) {
  const float s = 1.0f / (1.0f + expf(-g));
  const float silu = g * s;
  const float dsilu = s * (1.0f + g * (1.0f - s));
  dg = dh * u * dsilu;
  du = dh * silu;
}

// EPI_SWIGLU: B is W_g and B2 W_u ([I x K] each); the product's columns
// interleave 32-row blocks of the two (block 2q of a 256-column tile: W_g
// rows 128 n + 32 q .., block 2q + 1: the same rows of W_u), so a 64-column
// wave tile holds G and U of the same 32 rows of W; out = G, U, H [M x I].
// EPI_SWIGLU_BWD: G, U in (gate, up) [M x N], out = dG, dU = dU, rows ldo
// elements apart (ldo = 2 N with dU = out + N: the two side by side in one
// [M x 2N] array, as the stacked products of the backward read them).
struct SwigluParams {
  const uint16_t* Wu;
  uint16_t* U;
  uint16_t* H;
  int64_t I;
  const uint16_t* G_in;
  const uint16_t* U_in;
  uint16_t* dU;
  int64_t ldo;
};

// Head-split epilogue (EPI_HEADS*): position of row m is m % L; cos and sin
// of pair i at position p in cs[p * 64 + i]; head h goes to slot
// (h % perm) * (H / perm) + h / perm (perm > 1) or h; with EPI_HEADS_ROT the
// heads h < nrot are rotated (the keys of a stacked key/value product).
struct HeadsParams {
  const float* cs;  // [L, 64] (cos, sin) pairs
  int L, H, perm;
  int nrot;
};

struct GemmLaunch {
  // C[M x N] = A[M x K] * B[N x K]^T, bf16 operands with K contiguous unless
  // ta / tb say otherwise.
  const uint16_t* A; const uint16_t* B;
  int64_t M, N, K;
  int epi;
  const float* Yt;     // EPI_LOSS
  void* out;
  float* partials;     // EPI_LOSS, one per workgroup
  float scale;
  SteParams ste;       // EPI_STE
  // strided batch (EPI_GRAD_*): batch > 1 products, operands and output of
  // batch b at A + b bsa, B + b bsb (elements), out + b bso (bytes)
  int64_t batch, bsa, bsb, bso;
  int causal;  // 0, or the causal mode of square attention products (see gemm.hip)
  // operands stored K-slow (EPI_GRAD_*, no batch, no causal mode): A as
  // [K x M] (ta = 1), B as [K x N] (tb = 1)
  int ta, tb;
  HeadsParams heads;   // EPI_HEADS*
  SwigluParams swiglu; // EPI_SWIGLU
  const float* Rres;   // EPI_LOSS_BLOCK
};

// Causal attention with the score tiles on chip (attn_fused.hip), d = 128.
struct AttnLaunch {
  int64_t batch, kv_batch;
  int L;
  float scale;
  const uint16_t* Q; const uint16_t* K; const uint16_t* V; const uint16_t* O; const uint16_t* dO;
  uint16_t* O_out; float* lse; float* delta; float* dQ; float* dK; float* dV;
  // token-major O / dO / gradients when tok_seqs > 0 (see uniquan_attn_fwd)
  int tok_seqs, group;
  const float* cs;
  uint16_t* dQ_tok; uint16_t* dK_tok; uint16_t* dV_tok;
};
hipError_t launch_attn_fwd(const AttnLaunch& p, hipStream_t st);
hipError_t launch_attn_bwd(const AttnLaunch& p, hipStream_t st);

// Deployment form (bit-planes + binary16 Theta*_B) and its product.
struct BcqPackLaunch {
  int64_t R, C;
  int k, g;
  const uint8_t* codes; const float* alpha_star; const float* z_star;
  uint32_t* planes; uint16_t* alpha16; uint16_t* z16;
};
struct BcqMatmulLaunch {
  int T;
  int64_t R, C;
  int k, g;
  const uint16_t* X; const uint32_t* planes; const uint16_t* alpha16; const uint16_t* z16;
  float* Y; float* partials;
};

hipError_t launch_fq_fwd(const FqFwdLaunch& p, hipStream_t st);
hipError_t launch_fq_bwd(const FqBwdLaunch& p, hipStream_t st);
hipError_t launch_fq_step(const FqStepLaunch& p, hipStream_t st);
hipError_t launch_fold(const FoldLaunch& p, hipStream_t st);
hipError_t launch_dequant(const DequantLaunch& p, hipStream_t st);
hipError_t launch_greedy(const GreedyLaunch& p, hipStream_t st);
hipError_t launch_init_unified(const InitUnifiedLaunch& p, hipStream_t st);
hipError_t launch_gemm(const GemmLaunch& p, hipStream_t st);
hipError_t launch_gemm_ste(const GemmLaunch& p, int k, hipStream_t st);
size_t gemm_workgroups(int64_t M, int64_t N, int epi);
hipError_t launch_reduce_loss(const float* partials, int64_t n, float* loss, hipStream_t st);
// Fixed device array (per GPU) of kNoallocPartials loss partials for
// uniquan_layer_recon_noalloc; *out receives its address on the current GPU.
constexpr size_t kNoallocPartials = size_t(1) << 16;
hipError_t noalloc_scratch(float** out);
hipError_t launch_transpose(int64_t rows, int64_t cols, const uint16_t* in, uint16_t* out, hipStream_t st);
hipError_t launch_sgd(int64_t n, float* theta, const float* grad, float lr, hipStream_t st);
hipError_t launch_bcq_pack(const BcqPackLaunch& p, hipStream_t st);
hipError_t launch_add_rmsnorm(int64_t T, int64_t C, const float* X, const float* A, const float* gamma, float* R,
                              uint16_t* Z, float* rinv, hipStream_t st);
hipError_t launch_rmsnorm_bwd(int64_t T, int64_t C, const float* dZa, const float* dZb, const float* X,
                              const float* gamma, const float* rinv, const uint16_t* E, float escale, uint16_t* dR,
                              float* dRf, hipStream_t st);
hipError_t launch_rope_table(int L, int d, float* cs, hipStream_t st);
hipError_t launch_rope_split(int64_t T, int H, int d, int L, int perm, const void* in, int in_f32, int rotate,
                             uint16_t* out, hipStream_t st);
hipError_t launch_rope_merge(int64_t T, int H, int d, int L, int perm, int nsum, const void* in, int in_f32,
                             int rotate, uint16_t* out, int64_t ldo, hipStream_t st);
hipError_t launch_softmax_causal(int64_t rows, int L, const float* S, uint16_t* P, hipStream_t st);
hipError_t launch_softmax_bwd(int64_t rows, int L, const float* dP, const uint16_t* P, uint16_t* dS, hipStream_t st);
hipError_t launch_transpose_batched(int64_t B, int64_t R, int64_t C, const uint16_t* in, uint16_t* out,
                                    hipStream_t st);
size_t block_loss_ws();
hipError_t launch_block_loss(int64_t n, const float* Rres, const float* M, const float* Yref, uint16_t* E,
                             float* partials, float* loss, hipStream_t st);
hipError_t launch_silu_mul_fwd(int64_t n, const uint16_t* G, const uint16_t* U, uint16_t* H, hipStream_t st);
hipError_t launch_silu_mul_bwd(int64_t n, const uint16_t* dH, const uint16_t* G, const uint16_t* U, uint16_t* dG,
                               uint16_t* dU, hipStream_t st);
hipError_t launch_bcq_matmul(const BcqMatmulLaunch& p, hipStream_t st);
int64_t bcq_slabs(int64_t R, int64_t C);

// Ceiling probes (probe.hip): the MFMA probe runs PROBE_MFMA_BLOCKS x 4
// wavefronts of PROBE_MFMA_CHAINS chains.
constexpr int PROBE_MFMA_BLOCKS = 1024;
constexpr int PROBE_MFMA_CHAINS = 8;
hipError_t launch_probe_stream(int op, int64_t n16, const void* src, void* dst, void* sink, int blocks,
                               hipStream_t st);
hipError_t launch_probe_mfma(int iters, float* sink, hipStream_t st);

}  // namespace uq
