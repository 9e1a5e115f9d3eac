// Deployment form of a folded layer (Theorem 1 output: codes C and
// Theta*_B = {alpha*, z*_B}) and the binary-coding product with a small
// batch of activations (the single inference step R_B(C; Theta*) of the
// table of quantization schemes).
//
// Stored form (g k + 16 (k + 1) bits per group, appendix "Memory usage"):
//   planes  uint32 [k][C/128][R][4]: word m of quad q of row r in plane i
//           holds bit i of the codes of columns 128 q + 32 m + j in bit j;
//   alpha16 fp16   [k][C/g][R], z16 fp16 [C/g][R] (round to nearest even).
// Rows are the fastest index of every array, so the 64 lanes of a wavefront
// that work on 64 consecutive rows read contiguous memory.
//
// Product Y[t][r] = sum_c X[t][c] What[r][c] with What = z* + sum_i alpha*_i
// sigma_i.  Per group, sum_c sigma_i x_c = 2 P_i - S with S the activation
// sum over the group and P_i the sum over the columns whose bit i is set, so
//   y = sum_groups [ sum_i (2 alpha*_i) P_i + (z* - sum_i alpha*_i) S ].
// P_i is gathered 4 columns at a time from per-workgroup lookup tables: for
// every 4-column nibble of the workgroup's column slab and every batch row,
// the 16 subset sums of those 4 activations.  One lookup replaces 4
// multiply-adds; the tables are built once per workgroup and shared by its
// 256 rows (one row per lane).  Slabs write fp32 partial rows that a second
// kernel sums in a fixed order (deterministic results).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "uq_launch.h"

namespace uq {

// ---------------------------------------------------------------------------
// Packing
// ---------------------------------------------------------------------------
// Bit i of each of the four bytes of v, as a 4-bit number (byte b -> bit b):
// after masking, the bits sit at 0, 8, 16, 24; multiplying by
// 2^21 + 2^14 + 2^7 + 1 places byte b's bit at 21 + b and every other partial
// product at a distinct position outside 21..24, so no carries reach them.
__device__ __forceinline__ uint32_t gather_bit(uint32_t v, int i) {
  const uint32_t t = (v >> i) & 0x01010101u;
  return ((t * 0x00204081u) >> 21) & 0xFu;
}

// One thread per (quad q, row r, word m): 32 code bytes -> one word per plane.
__global__ __launch_bounds__(256) void bcq_pack_planes_kernel(const uint8_t* __restrict__ codes,
                                                              uint32_t* __restrict__ planes, int64_t R, int64_t C,
                                                              int k) {
  const int64_t nq = C / 128;
  const int64_t idx = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= nq * R * 4) return;
  const int m = int(idx & 3);
  const int64_t rq = idx >> 2;  // q R + r
  const int64_t q = rq / R, r = rq - q * R;
  const uint4* src = reinterpret_cast<const uint4*>(codes + r * C + q * 128 + m * 32);
  const uint4 lo = src[0], hi = src[1];
  const uint32_t v[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
  for (int i = 0; i < k; ++i) {
    uint32_t word = 0;
#pragma unroll
    for (int e = 0; e < 8; ++e) word |= gather_bit(v[e], i) << (4 * e);
    planes[(int64_t(i) * nq * R + rq) * 4 + m] = word;
  }
}

// One thread per (group column j, row r): alpha*, z*_B -> binary16.
__global__ __launch_bounds__(256) void bcq_pack_params_kernel(const float* __restrict__ alpha_star,
                                                              const float* __restrict__ z_star,
                                                              uint16_t* __restrict__ alpha16,
                                                              uint16_t* __restrict__ z16, int64_t R, int64_t gpr,
                                                              int k) {
  const int64_t idx = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= gpr * R) return;
  const int64_t j = idx / R, r = idx - j * R;
  const int64_t gid = r * gpr + j;
  for (int i = 0; i < k; ++i)
    alpha16[(int64_t(i) * gpr + j) * R + r] = __builtin_bit_cast(uint16_t, _Float16(alpha_star[gid * k + i]));
  z16[j * R + r] = __builtin_bit_cast(uint16_t, _Float16(z_star[gid]));
}

hipError_t launch_bcq_pack(const BcqPackLaunch& p, hipStream_t st) {
  const int64_t nq = p.C / 128, gpr = p.C / p.g;
  const int64_t n1 = nq * p.R * 4, n2 = gpr * p.R;
  hipLaunchKernelGGL(bcq_pack_planes_kernel, dim3(unsigned((n1 + 255) / 256)), dim3(256), 0, st, p.codes, p.planes,
                     p.R, p.C, p.k);
  hipLaunchKernelGGL(bcq_pack_params_kernel, dim3(unsigned((n2 + 255) / 256)), dim3(256), 0, st, p.alpha_star,
                     p.z_star, p.alpha16, p.z16, p.R, gpr, p.k);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Product
// ---------------------------------------------------------------------------
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

struct BcqArgs {
  const uint16_t* X;
  const u32x4* planes;
  const uint16_t* alpha16;
  const uint16_t* z16;
  float* out;  // Y [T][R] (one slab) or partials [slabs][T][R]
  int64_t R, C, nq, gpr;
  int g, qps;
};

__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float(uint32_t(h) << 16); }
__device__ __forceinline__ float f16_to_f32(uint16_t h) { return float(__builtin_bit_cast(_Float16, h)); }

// Workgroup (bx, by): rows 256 bx .. 256 bx + 255 (one per lane), column
// quads qps by .. qps by + qps - 1.  LDS: T tables of qps * 32 nibbles x 16
// subset sums, then the T x qps quad sums.
template <int K, int T>
__global__ __launch_bounds__(256) void bcq_matmul_kernel(BcqArgs a) {
  extern __shared__ float lut[];
  const int tid = threadIdx.x;
  const int qps = a.qps;
  const int64_t q0 = int64_t(blockIdx.y) * qps;
  const int nqs = int(min<int64_t>(qps, a.nq - q0));
  const int per_t = qps * 512;  // floats per batch row's tables
  float* S = lut + T * per_t;

  // tables: entry v of nibble n is the sum, in ascending bit order, of the
  // activations of columns 4 n + b of the slab with bit b of v set
  const int per_t_used = nqs * 512;
  for (int e = tid; e < T * per_t_used; e += 256) {
    const int t = e / per_t_used, rem = e - t * per_t_used;
    const int n = rem >> 4, v = rem & 15;
    const uint2 xv = *reinterpret_cast<const uint2*>(a.X + int64_t(t) * a.C + q0 * 128 + 4 * n);
    const float x[4] = {bf16_to_f32(uint16_t(xv.x)), bf16_to_f32(uint16_t(xv.x >> 16)),
                        bf16_to_f32(uint16_t(xv.y)), bf16_to_f32(uint16_t(xv.y >> 16))};
    float s = 0.0f;
#pragma unroll
    for (int b = 0; b < 4; ++b)
      if ((v >> b) & 1) s += x[b];
    lut[t * per_t + rem] = s;
  }
  __syncthreads();
  // quad sums: the 32 nibble totals (entry 15) of the quad, ascending
  for (int e = tid; e < T * nqs; e += 256) {
    const int t = e / nqs, qq = e - t * nqs;
    float s = 0.0f;
    for (int n = 0; n < 32; ++n) s += lut[t * per_t + (qq * 32 + n) * 16 + 15];
    S[t * qps + qq] = s;
  }
  __syncthreads();

  const int64_t r = int64_t(blockIdx.x) * 256 + tid;
  if (r >= a.R) return;  // no barrier follows
  float acc[T];
#pragma unroll
  for (int t = 0; t < T; ++t) acc[t] = 0.0f;
  for (int qq = 0; qq < nqs; ++qq) {
    const int64_t q = q0 + qq;
    const int64_t j = (q * 128) / a.g;  // group column of this quad
    u32x4 pw[K];
    float al[K];
#pragma unroll
    for (int i = 0; i < K; ++i) {
      pw[i] = a.planes[(int64_t(i) * a.nq + q) * a.R + r];
      al[i] = f16_to_f32(a.alpha16[(int64_t(i) * a.gpr + j) * a.R + r]);
    }
    const float z = f16_to_f32(a.z16[j * a.R + r]);
    float asum = 0.0f;
#pragma unroll
    for (int i = 0; i < K; ++i) asum += al[i];
    const float* base = lut + qq * 512;
#pragma unroll
    for (int i = 0; i < K; ++i) {
      float P[T];
#pragma unroll
      for (int t = 0; t < T; ++t) P[t] = 0.0f;
      const uint32_t wv[4] = {pw[i].x, pw[i].y, pw[i].z, pw[i].w};
#pragma unroll
      for (int m = 0; m < 4; ++m)
#pragma unroll
        for (int nib = 0; nib < 8; ++nib) {
          const int v = int((wv[m] >> (4 * nib)) & 15u);
#pragma unroll
          for (int t = 0; t < T; ++t) P[t] += base[t * per_t + (m * 8 + nib) * 16 + v];
        }
      const float a2 = 2.0f * al[i];
#pragma unroll
      for (int t = 0; t < T; ++t) acc[t] += a2 * P[t];
    }
    const float zc = z - asum;
#pragma unroll
    for (int t = 0; t < T; ++t) acc[t] += zc * S[t * qps + qq];
  }
  float* out = a.out + int64_t(blockIdx.y) * T * a.R;
#pragma unroll
  for (int t = 0; t < T; ++t) out[int64_t(t) * a.R + r] = acc[t];
}

// Y[t][r] = sum over slabs of the partial rows, slabs in ascending order.
__global__ __launch_bounds__(256) void bcq_reduce_kernel(const float* __restrict__ part, float* __restrict__ Y,
                                                         int64_t n, int slabs) {
  const int64_t idx = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= n) return;
  float s = 0.0f;
  for (int b = 0; b < slabs; ++b) s += part[int64_t(b) * n + idx];
  Y[idx] = s;
}

// Quads per slab: the most (up to 4) that still give >= 512 workgroups.
int bcq_quads_per_slab(int64_t R, int64_t C) {
  const int64_t rb = (R + 255) / 256, nq = C / 128;
  for (int qps = 4; qps > 1; qps >>= 1)
    if (rb * ((nq + qps - 1) / qps) >= 512) return qps;
  return 1;
}

int64_t bcq_slabs(int64_t R, int64_t C) {
  const int qps = bcq_quads_per_slab(R, C);
  return (C / 128 + qps - 1) / qps;
}

template <int K, int T>
static void launch_mm(const BcqArgs& a, dim3 grid, size_t lds, hipStream_t st) {
  if (lds > 65536)
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(bcq_matmul_kernel<K, T>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
  hipLaunchKernelGGL((bcq_matmul_kernel<K, T>), grid, dim3(256), lds, st, a);
}

template <int K>
static void launch_mm_t(const BcqArgs& a, int T, dim3 grid, size_t lds, hipStream_t st) {
  switch (T) {
    case 1: launch_mm<K, 1>(a, grid, lds, st); break;
    case 2: launch_mm<K, 2>(a, grid, lds, st); break;
    case 3: launch_mm<K, 3>(a, grid, lds, st); break;
    case 4: launch_mm<K, 4>(a, grid, lds, st); break;
    case 5: launch_mm<K, 5>(a, grid, lds, st); break;
    case 6: launch_mm<K, 6>(a, grid, lds, st); break;
    case 7: launch_mm<K, 7>(a, grid, lds, st); break;
    default: launch_mm<K, 8>(a, grid, lds, st); break;
  }
}

hipError_t launch_bcq_matmul(const BcqMatmulLaunch& p, hipStream_t st) {
  BcqArgs a;
  a.X = p.X;
  a.planes = reinterpret_cast<const u32x4*>(p.planes);
  a.alpha16 = p.alpha16;
  a.z16 = p.z16;
  a.R = p.R;
  a.C = p.C;
  a.nq = p.C / 128;
  a.gpr = p.C / p.g;
  a.g = p.g;
  a.qps = bcq_quads_per_slab(p.R, p.C);
  const int64_t slabs = (a.nq + a.qps - 1) / a.qps;
  a.out = slabs == 1 ? p.Y : p.partials;
  const dim3 grid(unsigned((p.R + 255) / 256), unsigned(slabs));
  const size_t lds = (size_t(p.T) * a.qps * 512 + size_t(p.T) * a.qps) * sizeof(float);
  switch (p.k) {
    case 1: launch_mm_t<1>(a, p.T, grid, lds, st); break;
    case 2: launch_mm_t<2>(a, p.T, grid, lds, st); break;
    case 3: launch_mm_t<3>(a, p.T, grid, lds, st); break;
    default: launch_mm_t<4>(a, p.T, grid, lds, st); break;
  }
  if (slabs > 1) {
    const int64_t n = int64_t(p.T) * p.R;
    hipLaunchKernelGGL(bcq_reduce_kernel, dim3(unsigned((n + 255) / 256)), dim3(256), 0, st, p.partials, p.Y, n,
                       int(slabs));
  }
  return hipGetLastError();
}

}  // namespace uq
