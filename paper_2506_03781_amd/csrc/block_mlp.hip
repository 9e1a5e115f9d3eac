// Element-wise parts of block-level reconstruction for a Transformer
// block's MLP module (Algorithm 1 with f = the SiLU-gated MLP):
//   forward   H = silu(G) * U
//   backward  dG = dH * U * silu'(G),  dU = dH * silu(G)
// with silu(x) = x sigma(x), silu'(x) = sigma(x) (1 + x (1 - sigma(x))).
// bf16 in and out, fp32 arithmetic, 8 elements per lane (16-byte accesses);
// HBM-bound (6 B per element forward, 10 B backward).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "uq_launch.h"

namespace uq {

namespace {

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float lo_bf16(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float hi_bf16(uint32_t v) { return __uint_as_float(v & 0xFFFF0000u); }
// two fp32 -> packed bf16 pair, round to nearest even
__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
  const f32x2_t f = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2_t));
}

__device__ __forceinline__ void unpack8(const uint4 v, float (&f)[8]) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = lo_bf16(w[i]);
    f[2 * i + 1] = hi_bf16(w[i]);
  }
}
__device__ __forceinline__ uint4 pack8(const float (&f)[8]) {
  return make_uint4(pack2(f[0], f[1]), pack2(f[2], f[3]), pack2(f[4], f[5]), pack2(f[6], f[7]));
}

}  // namespace

__global__ __launch_bounds__(256) void silu_mul_fwd_kernel(int64_t n8, const uint4* __restrict__ G,
                                                           const uint4* __restrict__ U, uint4* __restrict__ H) {
  const int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (i >= n8) return;
  float g[8], u[8], h[8];
  unpack8(G[i], g);
  unpack8(U[i], u);
#pragma unroll
  for (int j = 0; j < 8; ++j) h[j] = silu_mul(g[j], u[j]);
  H[i] = pack8(h);
}

__global__ __launch_bounds__(256) void silu_mul_bwd_kernel(int64_t n8, const uint4* __restrict__ dH,
                                                           const uint4* __restrict__ G, const uint4* __restrict__ U,
                                                           uint4* __restrict__ dG, uint4* __restrict__ dU) {
  const int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (i >= n8) return;
  float dh[8], g[8], u[8], dg[8], du[8];
  unpack8(dH[i], dh);
  unpack8(G[i], g);
  unpack8(U[i], u);
#pragma unroll
  for (int j = 0; j < 8; ++j) silu_mul_grad(dh[j], g[j], u[j], dg[j], du[j]);
  dG[i] = pack8(dg);
  dU[i] = pack8(du);
}

hipError_t launch_silu_mul_fwd(int64_t n, const uint16_t* G, const uint16_t* U, uint16_t* H, hipStream_t st) {
  const int64_t n8 = n / 8;
  hipLaunchKernelGGL(silu_mul_fwd_kernel, dim3(unsigned((n8 + 255) / 256)), dim3(256), 0, st, n8,
                     reinterpret_cast<const uint4*>(G), reinterpret_cast<const uint4*>(U), reinterpret_cast<uint4*>(H));
  return hipGetLastError();
}

hipError_t launch_silu_mul_bwd(int64_t n, const uint16_t* dH, const uint16_t* G, const uint16_t* U, uint16_t* dG,
                               uint16_t* dU, hipStream_t st) {
  const int64_t n8 = n / 8;
  hipLaunchKernelGGL(silu_mul_bwd_kernel, dim3(unsigned((n8 + 255) / 256)), dim3(256), 0, st, n8,
                     reinterpret_cast<const uint4*>(dH), reinterpret_cast<const uint4*>(G),
                     reinterpret_cast<const uint4*>(U), reinterpret_cast<uint4*>(dG), reinterpret_cast<uint4*>(dU));
  return hipGetLastError();
}

}  // namespace uq
