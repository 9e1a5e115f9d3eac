// Measured ceilings of the part the library runs on: streaming HBM read,
// write and copy rates and the bf16 MFMA issue rate.  They are reported next
// to the nominal peaks so that a kernel's throughput can also be read
// against what this GPU reaches in practice.  Not part of the method.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "uq_launch.h"

namespace uq {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8p __attribute__((ext_vector_type(8)));
typedef float f32x16p __attribute__((ext_vector_type(16)));

// Grid-stride streaming over n16 16-byte words with nontemporal accesses, one
// word per lane per iteration.  The read probe xors what it reads and writes
// the result only if it equals a value the data cannot produce, so the loads
// stay and the sink is one 16-byte word; every access stays inside [0, n16).
template <int OP>
__global__ __launch_bounds__(256) void probe_stream_kernel(const u32x4* __restrict__ src, u32x4* __restrict__ dst,
                                                           int64_t n16, u32x4* __restrict__ sink) {
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  u32x4 acc = {0u, 0u, 0u, 0u};
  const u32x4 pat = {0x3f800000u, 0x40000000u, 0x40400000u, 0x40800000u};
  for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n16; i += stride) {
    if constexpr (OP == 1) {
      __builtin_nontemporal_store(pat, dst + i);
    } else {
      const u32x4 v = __builtin_nontemporal_load(src + i);
      if constexpr (OP == 0) acc ^= v;
      else __builtin_nontemporal_store(v, dst + i);
    }
  }
  if constexpr (OP == 0) {
    if ((acc.x ^ acc.y ^ acc.z ^ acc.w) == 0x9e3779b9u) sink[0] = acc;
  }
}

// Independent accumulation chains of v_mfma_f32_32x32x16_bf16 on register
// operands, one wavefront per SIMD (four per workgroup), no memory traffic
// but a conditional store of the result.
__global__ __launch_bounds__(256) void probe_mfma_kernel(int iters, float* __restrict__ sink) {
  f32x16p acc[PROBE_MFMA_CHAINS];
#pragma unroll
  for (int c = 0; c < PROBE_MFMA_CHAINS; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[c][r] = 0.0f;
  bf16x8p a, b;
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    a[r] = __bf16(1e-3f * float(threadIdx.x + r));
    b[r] = __bf16(1e-3f * float(r + 1));
  }
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < PROBE_MFMA_CHAINS; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[c], 0, 0, 0);
  }
  float s = 0.0f;
#pragma unroll
  for (int c = 0; c < PROBE_MFMA_CHAINS; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += acc[c][r];
  if (s == -1.2345e-7f) sink[0] = s;
}

hipError_t launch_probe_stream(int op, int64_t n16, const void* src, void* dst, void* sink, int blocks,
                               hipStream_t st) {
  const dim3 grid(static_cast<unsigned>(blocks)), block(256);
  const u32x4* s = static_cast<const u32x4*>(src);
  u32x4* d = static_cast<u32x4*>(dst);
  u32x4* k = static_cast<u32x4*>(sink);
  switch (op) {
    case 0: hipLaunchKernelGGL(probe_stream_kernel<0>, grid, block, 0, st, s, d, n16, k); break;
    case 1: hipLaunchKernelGGL(probe_stream_kernel<1>, grid, block, 0, st, s, d, n16, k); break;
    default: hipLaunchKernelGGL(probe_stream_kernel<2>, grid, block, 0, st, s, d, n16, k); break;
  }
  return hipGetLastError();
}

hipError_t launch_probe_mfma(int iters, float* sink, hipStream_t st) {
  hipLaunchKernelGGL(probe_mfma_kernel, dim3(PROBE_MFMA_BLOCKS), dim3(256), 0, st, iters, sink);
  return hipGetLastError();
}

}  // namespace uq
