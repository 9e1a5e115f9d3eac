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

// One v_bfe_u32 (the compiler otherwise splits a field extract of a masked
// word into a shift and an and).
template <int OFF>
__device__ __forceinline__ uint32_t byte_field(uint32_t w) {
  uint32_t r;
  asm volatile("v_bfe_u32 %0, %1, %2, 8" : "=v"(r) : "v"(w), "i"(OFF));
  return r;
}

__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float(uint32_t(h) << 16); }
__device__ __forceinline__ float f16_to_f32(uint16_t h) { return float(__builtin_bit_cast(_Float16, h)); }

// Workgroup (bx, by): rows 256 bx .. 256 bx + 255 (one per lane), column
// quads QPS by .. QPS by + QPS - 1.  LDS: T tables of QPS * 32 nibbles x 16
// subset sums, then the T x QPS quad sums (activation sums S of the quads).
template <int K, int T, int QPS>
__global__ __launch_bounds__(256) void bcq_matmul_kernel(BcqArgs a) {
  constexpr int PER_T = QPS * 512;  // floats per batch row's tables
  __shared__ __attribute__((aligned(16))) float lut[T * PER_T + T * QPS];
  const int tid = threadIdx.x;
  const int64_t q0 = int64_t(blockIdx.y) * QPS;
  const int nqs = int(min<int64_t>(QPS, a.nq - q0));
  float* S = lut + T * PER_T;
  const int64_t r = int64_t(blockIdx.x) * 256 + tid;
  const bool live = r < a.R;

  // The activations this thread turns into tables (nibble tables e = tid +
  // 256 u of the T x nqs x 32 in the slab) are loaded first, then this lane's
  // plane words and parameters for the whole slab: loads complete in issue
  // order, so the table build waits only for the activations while the
  // plane loads stay in flight.
  constexpr int NT = (T * QPS * 32 + 255) / 256;  // nibble tables per thread (upper bound)
  constexpr int LOG_FULL = QPS == 4 ? 7 : QPS == 2 ? 6 : 5;  // log2(QPS * 32)
  const bool full = nqs == QPS;
  const int n_tab = T * nqs * 32;
  const uint16_t* xs = a.X + q0 * 128;
  uint2 xv[NT];
  // loads are unconditional (indices clamped into range) so that no branch
  // splits the load sequence; clamped values are never used
#pragma unroll
  for (int u = 0; u < NT; ++u) {
    const int e = min(tid + 256 * u, n_tab - 1);
    const int t = full ? (e >> LOG_FULL) : e / (nqs * 32);
    const int n = e - t * (nqs * 32);
    xv[u] = *reinterpret_cast<const uint2*>(xs + int64_t(t) * a.C + 4 * n);
  }
  asm volatile("" ::: "memory");  // keep the activation loads ahead of the plane loads
  // plane i of quad q for row r at planes[(i nq + q) R + r]; parameters of
  // group column j at [(i gpr + j) R + r]; quad q lies in group q / qpg
  const int64_t R = a.R;
  const int64_t pstride = a.nq * R, astride = a.gpr * R;
  const int64_t rc = live ? r : R - 1;
  const u32x4* pp = a.planes + q0 * R + rc;
  const uint32_t qpg = uint32_t(a.g) >> 7;
  const uint32_t j0 = uint32_t(q0) / qpg, rem0 = uint32_t(q0) - j0 * qpg;
  u32x4 pw[QPS][K];
  float al[QPS][K], zz[QPS];
#pragma unroll
  for (int qq = 0; qq < QPS; ++qq) {
    const int qc = min(qq, nqs - 1);
    const int64_t j = int64_t(j0 + (rem0 + uint32_t(qc)) / qpg);
    const uint16_t* ap = a.alpha16 + j * R + rc;
#pragma unroll
    for (int i = 0; i < K; ++i) {
      pw[qq][i] = pp[qc * R + i * pstride];
      al[qq][i] = f16_to_f32(ap[i * astride]);
    }
    zz[qq] = f16_to_f32(a.z16[j * R + rc]);
  }

  // table of nibble n: entry v is the sum of the activations of columns
  // 4 n + b with bit b of v set, in ascending bit order (built by doubling:
  // entries 2^b .. 2^(b+1) - 1 are entries 0 .. 2^b - 1 plus x_b)
#pragma unroll
  for (int u = 0; u < NT; ++u) {
    // threads past the last table repeat it (identical values, same place)
    const int e = min(tid + 256 * u, n_tab - 1);
    {
      const int t = full ? (e >> LOG_FULL) : e / (nqs * 32);
      const int n = e - t * (nqs * 32);
      const float x0 = bf16_to_f32(uint16_t(xv[u].x)), x1 = bf16_to_f32(uint16_t(xv[u].x >> 16));
      const float x2 = bf16_to_f32(uint16_t(xv[u].y)), x3 = bf16_to_f32(uint16_t(xv[u].y >> 16));
      float L[16];
      L[0] = 0.0f;
      L[1] = x0;
      L[2] = x1;
      L[3] = x0 + x1;
#pragma unroll
      for (int v = 0; v < 4; ++v) L[4 + v] = L[v] + x2;
#pragma unroll
      for (int v = 0; v < 8; ++v) L[8 + v] = L[v] + x3;
      float4* dst = reinterpret_cast<float4*>(lut + t * PER_T + n * 16);
#pragma unroll
      for (int v = 0; v < 4; ++v) dst[v] = make_float4(L[4 * v], L[4 * v + 1], L[4 * v + 2], L[4 * v + 3]);
      // quad sum: the 32 nibble totals of a quad sit in 32 adjacent lanes
      // (tables are numbered quad-major and 256 u is a multiple of 32);
      // fixed xor-butterfly, written by the quad's first lane
      float tot = L[15];
#pragma unroll
      for (int msk = 16; msk >= 1; msk >>= 1) tot += __shfl_xor(tot, msk, 64);
      if ((tid & 31) == 0 && tid + 256 * u < n_tab) S[t * QPS + (n >> 5)] = tot;
    }
  }
  __syncthreads();
  if (!live) return;  // no barrier follows

  const char* lb = reinterpret_cast<const char*>(lut);
  float acc[T];
#pragma unroll
  for (int t = 0; t < T; ++t) acc[t] = 0.0f;
#pragma unroll
  for (int qq = 0; qq < QPS; ++qq) {
    if (qq >= nqs) break;
    float asum = 0.0f;
#pragma unroll
    for (int i = 0; i < K; ++i) asum += al[qq][i];
#pragma unroll
    for (int i = 0; i < K; ++i) {
      float P[T];
#pragma unroll
      for (int t = 0; t < T; ++t) P[t] = 0.0f;
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        // byte offsets of the table entries: the even nibbles of the word
        // shifted to bits 8 n + 2 .. 8 n + 5, the odd ones likewise, so one
        // field extract gives 4 v for each nibble
        const uint32_t ev = (pw[qq][i][m] << 2) & 0x3C3C3C3Cu;
        const uint32_t od = (pw[qq][i][m] >> 2) & 0x3C3C3C3Cu;
        const uint32_t boff[8] = {byte_field<0>(ev), byte_field<0>(od), byte_field<8>(ev), byte_field<8>(od),
                                  byte_field<16>(ev), byte_field<16>(od), byte_field<24>(ev),
                                  byte_field<24>(od)};
#pragma unroll
        for (int nib = 0; nib < 8; ++nib) {
          const int row0 = ((qq * 32 + m * 8 + nib) * 16) * 4;  // byte offset of the nibble's table
#pragma unroll
          for (int t = 0; t < T; ++t)
            P[t] += *reinterpret_cast<const float*>(lb + boff[nib] + (row0 + t * PER_T * 4));
        }
      }
      const float a2 = 2.0f * al[qq][i];
#pragma unroll
      for (int t = 0; t < T; ++t) acc[t] += a2 * P[t];
    }
    const float zc = zz[qq] - asum;
#pragma unroll
    for (int t = 0; t < T; ++t) acc[t] += zc * S[t * QPS + qq];
  }
  float* out = a.out + int64_t(blockIdx.y) * T * a.R;
#pragma unroll
  for (int t = 0; t < T; ++t) out[int64_t(t) * a.R + r] = acc[t];
}

// The same product for larger batches on MFMA (v_mfma_f32_32x32x16_bf16):
// P_i = X B_i^T with B_i the 0 / 1 matrix of plane i (exact in bf16) and S =
// X 1^T, per 128-column quad, then y += sum_i (2 alpha*_i) P_i + (z* -
// sum_i alpha*_i) S as in the table kernel.  C[m][n] is token m, row n: lane
// l supplies token l % 32 (zero past T) and the bits of row l % 32, both at
// columns 16 s + 8 (l / 32) .. + 8 of k-step s, and holds row l % 32 for
// tokens 4 (l / 32) + rr in accumulator slots rr < 4 (T <= 8).  Each of the
// 4 wavefronts takes 32 RT rows (RT 32-row tiles) of the workgroup's 128 RT;
// with RT = 2 the grid, slabs and partial rows are the table kernel's.  The bits of a
// fragment (8 columns of one row and plane) come from one LDS read of a
// 256-entry table, whatever T; the table kernel's lookups grow with T.
typedef __bf16 bf16x8b __attribute__((ext_vector_type(8)));
typedef float f32x16b __attribute__((ext_vector_type(16)));

// bits j of b (j < 8) as bf16 0.0 / 1.0 in element j: for each pair t of
// bits, t * 0x8001 puts bit 0 at position 0 and bit 1 at position 16 (the
// other partial products land at 1 and 15 and are masked off), and the
// product with 0x3F80 (bf16 1.0) makes the two halves.
__device__ __forceinline__ bf16x8b bits_bf16(uint32_t b) {
  u32x4 d;
#pragma unroll
  for (int j = 0; j < 4; ++j) d[j] = (((b >> (2 * j)) & 3u) * 0x8001u & 0x10001u) * 0x3F80u;
  return __builtin_bit_cast(bf16x8b, d);
}

template <int K, int QPS, int RT = 2>
__global__ __launch_bounds__(256) void bcq_mfma_kernel(BcqArgs a, int T) {
  // the 256 bytes as 8 bf16 each, built once: one LDS read per 8 bits
  __shared__ u32x4 tbl[256];
  // the slab's activations, T rows of QPS * 128 bf16 with a 32-byte pad
  // (the 16 fragments a k-step reads fall in distinct bank groups)
  constexpr int XLD = QPS * 128 + 16;
  __shared__ __attribute__((aligned(16))) uint16_t xs[8 * XLD];
  tbl[threadIdx.x] = __builtin_bit_cast(u32x4, bits_bf16(threadIdx.x));
  const int64_t q0 = int64_t(blockIdx.y) * QPS;
  const int nqs = int(min<int64_t>(QPS, a.nq - q0));
  {
    const int per_row = nqs * 32;  // 8-byte chunks per activation row
    for (int e = threadIdx.x; e < T * per_row; e += 256) {
      const int t = e / per_row, c = e - t * per_row;
      *reinterpret_cast<uint2*>(&xs[t * XLD + 4 * c]) =
          *reinterpret_cast<const uint2*>(a.X + int64_t(t) * a.C + q0 * 128 + 4 * c);
    }
  }
  __syncthreads();
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int tok = lane & 31, hk = lane >> 5;
  const int64_t R = a.R;
  const int64_t rbase = int64_t(blockIdx.x) * (128 * RT) + wave * (32 * RT);
  const int64_t astride = a.gpr * R;
  const uint32_t qpg = uint32_t(a.g) >> 7;
  bf16x8b ones;
#pragma unroll
  for (int e = 0; e < 8; ++e) ones[e] = __bf16(1.0f);
  float y[RT][4];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) y[rt][rr] = 0.0f;
  for (int qq = 0; qq < nqs; ++qq) {
    const int64_t q = q0 + qq;
    const int64_t j = int64_t(uint32_t(q) / qpg);
    // this lane's activations for the quad's 8 k-steps (zero past T)
    bf16x8b xa[8];
    const u32x4* xr = reinterpret_cast<const u32x4*>(&xs[min(tok, T - 1) * XLD + qq * 128 + 8 * hk]);
#pragma unroll
    for (int st = 0; st < 8; ++st) {
      const u32x4 v = xr[2 * st];
      const u32x4 z4 = {0u, 0u, 0u, 0u};
      xa[st] = __builtin_bit_cast(bf16x8b, tok < T ? v : z4);
    }
    f32x16b S = {};
#pragma unroll
    for (int st = 0; st < 8; ++st) S = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xa[st], ones, S, 0, 0, 0);
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      const int64_t r = rbase + 32 * rt + tok;
      const int64_t rc = r < R ? r : R - 1;
      u32x4 w[K];
      float al[K];
#pragma unroll
      for (int i = 0; i < K; ++i) {
        w[i] = a.planes[(i * a.nq + q) * R + rc];
        al[i] = f16_to_f32(a.alpha16[i * astride + j * R + rc]);
      }
      const float zc0 = f16_to_f32(a.z16[j * R + rc]);
      float asum = 0.0f;
#pragma unroll
      for (int i = 0; i < K; ++i) {
        asum += al[i];
        f32x16b P = {};
#pragma unroll
        for (int st = 0; st < 8; ++st) {
          const uint32_t byte = (w[i][st >> 1] >> (16 * (st & 1) + 8 * hk)) & 0xFFu;
          P = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xa[st], __builtin_bit_cast(bf16x8b, tbl[byte]), P, 0, 0, 0);
        }
        const float a2 = 2.0f * al[i];
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) y[rt][rr] += a2 * P[rr];
      }
      const float zc = zc0 - asum;
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) y[rt][rr] += zc * S[rr];
    }
  }
  float* out = a.out + int64_t(blockIdx.y) * T * R;
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const int64_t r = rbase + 32 * rt + tok;
    if (r >= R) continue;
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      const int t = 4 * hk + rr;
      if (t < T) out[int64_t(t) * R + r] = y[rt][rr];
    }
  }
}

// Y[t][r] = sum over slabs of the partial rows, slabs in ascending order.
__global__ __launch_bounds__(256) void bcq_reduce_kernel(const float* __restrict__ part, float* __restrict__ Y,
                                                         int64_t n, int slabs) {
  const int64_t idx = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= n) return;
  // up to 32 independent loads in flight (one memory round trip for most
  // shapes), added in slab order
  float s = 0.0f;
  for (int b0 = 0; b0 < slabs; b0 += 32) {
    float v[32];
#pragma unroll
    for (int j = 0; j < 32; ++j) v[j] = b0 + j < slabs ? part[int64_t(b0 + j) * n + idx] : 0.0f;
#pragma unroll
    for (int j = 0; j < 32; ++j)
      if (b0 + j < slabs) s += v[j];
  }
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

template <int K, int T, int QPS>
static void launch_mm(const BcqArgs& a, dim3 grid, hipStream_t st) {
  hipLaunchKernelGGL((bcq_matmul_kernel<K, T, QPS>), grid, dim3(256), 0, st, a);
}

template <int K, int T>
static void launch_mm_q(const BcqArgs& a, dim3 grid, hipStream_t st) {
  if (a.qps == 4) launch_mm<K, T, 4>(a, grid, st);
  else if (a.qps == 2) launch_mm<K, T, 2>(a, grid, st);
  else launch_mm<K, T, 1>(a, grid, st);
}

template <int K>
static void launch_mm_t(const BcqArgs& a, int T, dim3 grid, hipStream_t st) {
  switch (T) {
    case 1: launch_mm_q<K, 1>(a, grid, st); break;
    case 2: launch_mm_q<K, 2>(a, grid, st); break;
    case 3: launch_mm_q<K, 3>(a, grid, st); break;
    case 4: launch_mm_q<K, 4>(a, grid, st); break;
    case 5: launch_mm_q<K, 5>(a, grid, st); break;
    case 6: launch_mm_q<K, 6>(a, grid, st); break;
    case 7: launch_mm_q<K, 7>(a, grid, st); break;
    default: launch_mm_q<K, 8>(a, grid, st); break;
  }
}

template <int K>
static void launch_mfma_q(const BcqArgs& a, int T, dim3 grid, hipStream_t st) {
  if (a.qps == 4) hipLaunchKernelGGL((bcq_mfma_kernel<K, 4>), grid, dim3(256), 0, st, a, T);
  else if (a.qps == 2) hipLaunchKernelGGL((bcq_mfma_kernel<K, 2>), grid, dim3(256), 0, st, a, T);
  else hipLaunchKernelGGL((bcq_mfma_kernel<K, 1>), grid, dim3(256), 0, st, a, T);
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
  // tables for one to three batch rows, MFMA from four on (measured on the
  // 70B and 4096 x 4096 layers: equal at four rows with k = 2, the MFMA form
  // 1.9-2.2x faster at eight)
  if (p.T >= 4) {
    switch (p.k) {
      case 1: launch_mfma_q<1>(a, p.T, grid, st); break;
      case 2: launch_mfma_q<2>(a, p.T, grid, st); break;
      case 3: launch_mfma_q<3>(a, p.T, grid, st); break;
      default: launch_mfma_q<4>(a, p.T, grid, st); break;
    }
  } else {
    switch (p.k) {
      case 1: launch_mm_t<1>(a, p.T, grid, st); break;
      case 2: launch_mm_t<2>(a, p.T, grid, st); break;
      case 3: launch_mm_t<3>(a, p.T, grid, st); break;
      default: launch_mm_t<4>(a, p.T, grid, st); break;
    }
  }
  if (slabs > 1) {
    const int64_t n = int64_t(p.T) * p.R;
    hipLaunchKernelGGL(bcq_reduce_kernel, dim3(unsigned((n + 255) / 256)), dim3(256), 0, st, p.partials, p.Y, n,
                       int(slabs));
  }
  return hipGetLastError();
}

}  // namespace uq
