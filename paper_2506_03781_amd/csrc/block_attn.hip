// Element-wise and layout kernels of block-level reconstruction for a whole
// Transformer block (Algorithm 1 with f = one multi-head attention module and
// one MLP module): RMSNorm with the residual add, the rotary embedding fused
// with the split into heads (and its inverse fused with the merge), the
// causal softmax and its backward, a batched transpose and the block's loss.
// The products run on the NT GEMM.  Layouts: token-major [T, C]; head-major
// [H, T, d] (one [L, d] block per sequence and head, L = T / n_seq); scores
// and probabilities [H * n_seq, L, L].
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "uq_launch.h"

namespace uq {

namespace {

__device__ __forceinline__ float bf(uint16_t h) { return __uint_as_float(uint32_t(h) << 16); }
__device__ __forceinline__ uint16_t to_bf(float x) {
  // round to nearest even (finite inputs)
  const uint32_t u = __float_as_uint(x);
  return uint16_t((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

__device__ __forceinline__ float wave_sum(float v) {
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
  for (int m = 32; m >= 1; m >>= 1) v = fmaxf(v, __shfl_xor(v, m, 64));
  return v;
}

// angle of pair i (< d/2) at position p: p * theta^(-2i/d), theta = 1e4
__device__ __forceinline__ float rope_angle(int p, int i, int d) {
  const float inv = powf(10000.0f, -float(2 * i) / float(d));
  return float(p) * inv;
}

}  // namespace

// One wavefront per row: R = X + A (A optional), r = 1 / sqrt(mean(R^2) + eps),
// Z = bf16((R r) gamma).  C is a multiple of 8.
__global__ __launch_bounds__(256) void add_rmsnorm_kernel(int64_t T, int64_t C, const float* __restrict__ X,
                                                          const float* __restrict__ A, const float* __restrict__ gamma,
                                                          float* __restrict__ R, uint16_t* __restrict__ Z,
                                                          float* __restrict__ rinv) {
  const int lane = threadIdx.x & 63;
  const int64_t row = int64_t(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (row >= T) return;
  const float* x = X + row * C;
  const float* a = A ? A + row * C : nullptr;
  float ss = 0.0f;
  for (int64_t c = int64_t(lane) * 8; c < C; c += 512) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float v = a ? x[c + i] + a[c + i] : x[c + i];
      ss += v * v;
    }
  }
  ss = wave_sum(ss);
  const float r = 1.0f / sqrtf(ss / float(C) + 1e-5f);
  if (lane == 0) rinv[row] = r;
  for (int64_t c = int64_t(lane) * 8; c < C; c += 512) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float v = a ? x[c + i] + a[c + i] : x[c + i];
      if (R) R[row * C + c + i] = v;
      Z[row * C + c + i] = to_bf((v * r) * gamma[c + i]);
    }
  }
}

// One wavefront per row: dR = escale * E + r g - x r^3 sum(g x) / C with
// g = gamma (dZa + dZb); writes dR in bf16 (and in fp32 when dRf is given).
__global__ __launch_bounds__(256) void rmsnorm_bwd_kernel(int64_t T, int64_t C, const float* __restrict__ dZa,
                                                          const float* __restrict__ dZb,
                                                          const float* __restrict__ Xin,
                                                          const float* __restrict__ gamma,
                                                          const float* __restrict__ rinv,
                                                          const uint16_t* __restrict__ E, float escale,
                                                          uint16_t* __restrict__ dR, float* __restrict__ dRf) {
  const int lane = threadIdx.x & 63;
  const int64_t row = int64_t(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (row >= T) return;
  const int64_t base = row * C;
  float dot = 0.0f;
  for (int64_t c = int64_t(lane) * 8; c < C; c += 512) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float dz = dZb ? dZa[base + c + i] + dZb[base + c + i] : dZa[base + c + i];
      dot += (gamma[c + i] * dz) * Xin[base + c + i];
    }
  }
  dot = wave_sum(dot);
  const float r = rinv[row];
  const float k3 = (r * r * r) * (dot / float(C));
  for (int64_t c = int64_t(lane) * 8; c < C; c += 512) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float dz = dZb ? dZa[base + c + i] + dZb[base + c + i] : dZa[base + c + i];
      float v = r * (gamma[c + i] * dz) - Xin[base + c + i] * k3;
      if (E) v += escale * bf(E[base + c + i]);
      dR[base + c + i] = to_bf(v);
      if (dRf) dRf[base + c + i] = v;
    }
  }
}

// Token-major [T, C] (fp32 or bf16) -> head-major bf16 [H, T, d], rotating
// pairs (i, i + d/2) by the position's angle when ROT.  One thread per pair.
template <bool IN_F32, bool ROT>
__global__ __launch_bounds__(256) void rope_split_kernel(int64_t T, int H, int d, int L, const void* __restrict__ in,
                                                         uint16_t* __restrict__ out) {
  const int hd = d >> 1;
  const int64_t n = T * H * hd;
  const int64_t idx = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= n) return;
  const int i = int(idx % hd);
  const int h = int((idx / hd) % H);
  const int64_t t = idx / (int64_t(hd) * H);
  const int64_t src = t * (int64_t(H) * d) + int64_t(h) * d + i;
  float x1, x2;
  if (IN_F32) {
    x1 = static_cast<const float*>(in)[src];
    x2 = static_cast<const float*>(in)[src + hd];
  } else {
    x1 = bf(static_cast<const uint16_t*>(in)[src]);
    x2 = bf(static_cast<const uint16_t*>(in)[src + hd]);
  }
  float y1 = x1, y2 = x2;
  if (ROT) {
    float s, c;
    sincosf(rope_angle(int(t % L), i, d), &s, &c);
    y1 = x1 * c - x2 * s;
    y2 = x2 * c + x1 * s;
  }
  const int64_t dst = (int64_t(h) * T + t) * d + i;
  out[dst] = to_bf(y1);
  out[dst + hd] = to_bf(y2);
}

// Head-major [H, T, d] (fp32 or bf16) -> token-major bf16 [T, C], rotating
// by minus the position's angle when ROT (the inverse rotation).
template <bool IN_F32, bool ROT>
__global__ __launch_bounds__(256) void rope_merge_kernel(int64_t T, int H, int d, int L, const void* __restrict__ in,
                                                         uint16_t* __restrict__ out) {
  const int hd = d >> 1;
  const int64_t n = T * H * hd;
  const int64_t idx = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= n) return;
  const int i = int(idx % hd);
  const int h = int((idx / hd) % H);
  const int64_t t = idx / (int64_t(hd) * H);
  const int64_t src = (int64_t(h) * T + t) * d + i;
  float x1, x2;
  if (IN_F32) {
    x1 = static_cast<const float*>(in)[src];
    x2 = static_cast<const float*>(in)[src + hd];
  } else {
    x1 = bf(static_cast<const uint16_t*>(in)[src]);
    x2 = bf(static_cast<const uint16_t*>(in)[src + hd]);
  }
  float y1 = x1, y2 = x2;
  if (ROT) {
    float s, c;
    sincosf(rope_angle(int(t % L), i, d), &s, &c);
    y1 = x1 * c + x2 * s;
    y2 = x2 * c - x1 * s;
  }
  const int64_t dst = t * (int64_t(H) * d) + int64_t(h) * d + i;
  out[dst] = to_bf(y1);
  out[dst + hd] = to_bf(y2);
}

// One wavefront per score row i of one [L, L] block: P[i, j] = softmax over
// j <= i of S[i, j], 0 for j > i (bf16).
__global__ __launch_bounds__(256) void softmax_causal_kernel(int64_t rows, int L, const float* __restrict__ S,
                                                             uint16_t* __restrict__ P) {
  const int lane = threadIdx.x & 63;
  const int64_t row = int64_t(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int i = int(row % L);
  const float* s = S + row * L;
  uint16_t* p = P + row * L;
  float m = -INFINITY;
  for (int j = lane; j <= i; j += 64) m = fmaxf(m, s[j]);
  m = wave_max(m);
  float sum = 0.0f;
  for (int j = lane; j <= i; j += 64) sum += expf(s[j] - m);
  sum = wave_sum(sum);
  const float inv = 1.0f / sum;
  for (int j = lane; j < L; j += 64) p[j] = j <= i ? to_bf(expf(s[j] - m) * inv) : uint16_t(0);
}

// dS[i, j] = P[i, j] (dP[i, j] - sum_j' P[i, j'] dP[i, j']) (bf16), one
// wavefront per row.
__global__ __launch_bounds__(256) void softmax_bwd_kernel(int64_t rows, int L, const float* __restrict__ dP,
                                                          const uint16_t* __restrict__ P, uint16_t* __restrict__ dS) {
  const int lane = threadIdx.x & 63;
  const int64_t row = int64_t(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int i = int(row % L);
  const float* dp = dP + row * L;
  const uint16_t* p = P + row * L;
  float dot = 0.0f;
  for (int j = lane; j <= i; j += 64) dot += bf(p[j]) * dp[j];
  dot = wave_sum(dot);
  for (int j = lane; j < L; j += 64) dS[row * L + j] = j <= i ? to_bf(bf(p[j]) * (dp[j] - dot)) : uint16_t(0);
}

// out[b] = in[b]^T for B matrices [R, C] (bf16), 64 x 64 tiles through LDS.
__global__ __launch_bounds__(256) void transpose_batched_kernel(int64_t R, int64_t C, const uint16_t* __restrict__ in,
                                                                uint16_t* __restrict__ out) {
  __shared__ uint16_t tile[64][66];
  const int64_t tiles_c = (C + 63) / 64;
  const int64_t r0 = (int64_t(blockIdx.x) / tiles_c) * 64, c0 = (int64_t(blockIdx.x) % tiles_c) * 64;
  const int64_t boff = int64_t(blockIdx.y) * R * C;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int y = ty; y < 64; y += 4) {
    const int64_t r = r0 + y, c = c0 + tx;
    tile[y][tx] = (r < R && c < C) ? in[boff + r * C + c] : uint16_t(0);
  }
  __syncthreads();
  for (int y = ty; y < 64; y += 4) {
    const int64_t c = c0 + y, r = r0 + tx;
    if (c < C && r < R) out[boff + c * R + r] = tile[tx][y];
  }
}

// E = (Rres + M) - Yref in bf16, and per-block partial sums of the unrounded
// E^2 (fp32 per thread, fixed-order block reduction).
__global__ __launch_bounds__(256) void block_loss_kernel(int64_t n, const float* __restrict__ Rres,
                                                         const float* __restrict__ M, const float* __restrict__ Yref,
                                                         uint16_t* __restrict__ E, float* __restrict__ partials) {
  __shared__ float red[4];
  float acc = 0.0f;
  for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < n; i += int64_t(gridDim.x) * 256) {
    const float e = (Rres[i] + M[i]) - Yref[i];
    E[i] = to_bf(e);
    acc += e * e;
  }
  acc = wave_sum(acc);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) partials[blockIdx.x] = (red[0] + red[1]) + (red[2] + red[3]);
}

// loss = sum of the partials, in fp64 in a fixed order.
__global__ __launch_bounds__(256) void block_loss_reduce_kernel(int np, const float* __restrict__ partials,
                                                                float* __restrict__ loss) {
  __shared__ double red[4];
  double acc = 0.0;
  for (int i = threadIdx.x; i < np; i += 256) acc += double(partials[i]);
  for (int m = 32; m >= 1; m >>= 1) acc += __shfl_xor(acc, m, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) loss[0] = float((red[0] + red[1]) + (red[2] + red[3]));
}

constexpr int kLossBlocks = 1024;

hipError_t launch_add_rmsnorm(int64_t T, int64_t C, const float* X, const float* A, const float* gamma, float* R,
                              uint16_t* Z, float* rinv, hipStream_t st) {
  hipLaunchKernelGGL(add_rmsnorm_kernel, dim3(unsigned((T + 3) / 4)), dim3(256), 0, st, T, C, X, A, gamma, R, Z, rinv);
  return hipGetLastError();
}

hipError_t launch_rmsnorm_bwd(int64_t T, int64_t C, const float* dZa, const float* dZb, const float* X,
                              const float* gamma, const float* rinv, const uint16_t* E, float escale, uint16_t* dR,
                              float* dRf, hipStream_t st) {
  hipLaunchKernelGGL(rmsnorm_bwd_kernel, dim3(unsigned((T + 3) / 4)), dim3(256), 0, st, T, C, dZa, dZb, X, gamma, rinv,
                     E, escale, dR, dRf);
  return hipGetLastError();
}

hipError_t launch_rope_split(int64_t T, int H, int d, int L, const void* in, int in_f32, int rotate, uint16_t* out,
                             hipStream_t st) {
  const dim3 grid(unsigned((T * H * (d / 2) + 255) / 256));
  if (in_f32 && rotate) hipLaunchKernelGGL((rope_split_kernel<true, true>), grid, dim3(256), 0, st, T, H, d, L, in, out);
  else if (in_f32) hipLaunchKernelGGL((rope_split_kernel<true, false>), grid, dim3(256), 0, st, T, H, d, L, in, out);
  else if (rotate) hipLaunchKernelGGL((rope_split_kernel<false, true>), grid, dim3(256), 0, st, T, H, d, L, in, out);
  else hipLaunchKernelGGL((rope_split_kernel<false, false>), grid, dim3(256), 0, st, T, H, d, L, in, out);
  return hipGetLastError();
}

hipError_t launch_rope_merge(int64_t T, int H, int d, int L, const void* in, int in_f32, int rotate, uint16_t* out,
                             hipStream_t st) {
  const dim3 grid(unsigned((T * H * (d / 2) + 255) / 256));
  if (in_f32 && rotate) hipLaunchKernelGGL((rope_merge_kernel<true, true>), grid, dim3(256), 0, st, T, H, d, L, in, out);
  else if (in_f32) hipLaunchKernelGGL((rope_merge_kernel<true, false>), grid, dim3(256), 0, st, T, H, d, L, in, out);
  else if (rotate) hipLaunchKernelGGL((rope_merge_kernel<false, true>), grid, dim3(256), 0, st, T, H, d, L, in, out);
  else hipLaunchKernelGGL((rope_merge_kernel<false, false>), grid, dim3(256), 0, st, T, H, d, L, in, out);
  return hipGetLastError();
}

hipError_t launch_softmax_causal(int64_t rows, int L, const float* S, uint16_t* P, hipStream_t st) {
  hipLaunchKernelGGL(softmax_causal_kernel, dim3(unsigned((rows + 3) / 4)), dim3(256), 0, st, rows, L, S, P);
  return hipGetLastError();
}

hipError_t launch_softmax_bwd(int64_t rows, int L, const float* dP, const uint16_t* P, uint16_t* dS, hipStream_t st) {
  hipLaunchKernelGGL(softmax_bwd_kernel, dim3(unsigned((rows + 3) / 4)), dim3(256), 0, st, rows, L, dP, P, dS);
  return hipGetLastError();
}

hipError_t launch_transpose_batched(int64_t B, int64_t R, int64_t C, const uint16_t* in, uint16_t* out,
                                    hipStream_t st) {
  const int64_t tiles = ((R + 63) / 64) * ((C + 63) / 64);
  hipLaunchKernelGGL(transpose_batched_kernel, dim3(unsigned(tiles), unsigned(B)), dim3(256), 0, st, R, C, in, out);
  return hipGetLastError();
}

size_t block_loss_ws() { return kLossBlocks; }

hipError_t launch_block_loss(int64_t n, const float* Rres, const float* M, const float* Yref, uint16_t* E,
                             float* partials, float* loss, hipStream_t st) {
  hipLaunchKernelGGL(block_loss_kernel, dim3(kLossBlocks), dim3(256), 0, st, n, Rres, M, Yref, E, partials);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(block_loss_reduce_kernel, dim3(1), dim3(256), 0, st, kLossBlocks, partials, loss);
  return hipGetLastError();
}

}  // namespace uq
