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

// Grid-stride streaming over n16 16-byte words with nontemporal accesses;
// four words in flight per lane.  Every lane writes its own sink word (the
// read probe's xor of what it read), so nothing is optimised away and every
// access stays inside [0, n16).
template <int OP>
__global__ __launch_bounds__(256) void probe_stream_kernel(const u32x4* __restrict__ src, u32x4* __restrict__ dst,
                                                           int64_t n16, uint32_t* __restrict__ sink) {
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  uint32_t acc = 0;
  const u32x4 pat = {0x3f800000u, 0x40000000u, uint32_t(i), 0x40400000u};
  for (; i + 3 * stride < n16; i += 4 * stride) {
    if constexpr (OP == 1) {
#pragma unroll
      for (int u = 0; u < 4; ++u) __builtin_nontemporal_store(pat, dst + i + u * stride);
    } else {
      u32x4 v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) v[u] = __builtin_nontemporal_load(src + i + u * stride);
      if constexpr (OP == 0) {
#pragma unroll
        for (int u = 0; u < 4; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
      } else {
#pragma unroll
        for (int u = 0; u < 4; ++u) __builtin_nontemporal_store(v[u], dst + i + u * stride);
      }
    }
  }
  for (; i < n16; i += stride) {
    if constexpr (OP == 1) {
      __builtin_nontemporal_store(pat, dst + i);
    } else {
      const u32x4 v = __builtin_nontemporal_load(src + i);
      if constexpr (OP == 0) acc ^= v.x ^ v.y ^ v.z ^ v.w;
      else __builtin_nontemporal_store(v, dst + i);
    }
  }
  sink[int64_t(blockIdx.x) * blockDim.x + threadIdx.x] = acc;
}

// Independent accumulation chains of v_mfma_f32_32x32x16_bf16 on register
// operands, one wavefront per SIMD (four per workgroup), no memory traffic
// but the final per-lane store.
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
  sink[int64_t(blockIdx.x) * blockDim.x + threadIdx.x] = s;
}

hipError_t launch_probe_stream(int op, int64_t n16, const void* src, void* dst, uint32_t* sink, hipStream_t st) {
  const dim3 grid(PROBE_BLOCKS), block(256);
  const u32x4* s = static_cast<const u32x4*>(src);
  u32x4* d = static_cast<u32x4*>(dst);
  switch (op) {
    case 0: hipLaunchKernelGGL(probe_stream_kernel<0>, grid, block, 0, st, s, d, n16, sink); break;
    case 1: hipLaunchKernelGGL(probe_stream_kernel<1>, grid, block, 0, st, s, d, n16, sink); break;
    default: hipLaunchKernelGGL(probe_stream_kernel<2>, grid, block, 0, st, s, d, n16, sink); break;
  }
  return hipGetLastError();
}

hipError_t launch_probe_mfma(int iters, float* sink, hipStream_t st) {
  hipLaunchKernelGGL(probe_mfma_kernel, dim3(PROBE_MFMA_BLOCKS), dim3(256), 0, st, iters, sink);
  return hipGetLastError();
}

}  // namespace uq
