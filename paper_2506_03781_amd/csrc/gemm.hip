// Reconstruction contractions on bf16 MFMA (gfx950 v_mfma_f32_32x32x16_bf16)
// with fused epilogues:
//   target   Yt = W X^T                    (once per layer)
//   forward  Et = What X^T - Yt, sum Et^2   (loss partials per workgroup)
//   backward G  = 2 Et Xt^T                 (weight gradient)
// All three are C[M x N] = A[M x K] B[N x K]^T with both operands K-contiguous
// ("NT"), so one kernel template serves them.
//
// Tiling: a 256-thread workgroup (4 wavefronts, 2 x 2) computes a BM x BN
// tile (256x256, 256x128 or 128x128, the largest that still fills the 256
// compute units); each wavefront owns (BM/2) x (BN/2) as a grid of 32x32 MFMA
// blocks with fp32 accumulators.  K advances in slabs of 64: the next slab is
// fetched from global memory into registers (16-byte loads, 8 lanes per
// 128-byte row segment) while the MFMAs consume the current slab from one of
// two LDS buffers, so one barrier per slab suffices.  LDS rows are XOR-
// swizzled instead of padded.  Workgroups are renumbered so that each XCD
// gets a contiguous run of tiles walked in groups of 8 row-tiles, which keeps
// the operand panels it needs in its own L2.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "uq_launch.h"

namespace uq {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

struct GemmArgs {
  const uint16_t* A;
  const uint16_t* B;
  int64_t M, N, K;
  const float* Yt;
  void* out;
  float* partials;
  float scale;
  int tiles_m, tiles_n;
};

__device__ __forceinline__ uint32_t bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

// Map a linear workgroup id to (tile_m, tile_n).  Hardware dispatches
// workgroup i to XCD i % 8; renumber so that each XCD receives a contiguous
// run of logical tiles, then walk logical tiles in groups of GM row-tiles.
__device__ __forceinline__ void tile_of(int bid, int nb, int tiles_m, int tiles_n, int& tm, int& tn) {
  int logical = bid;
  if ((nb & 7) == 0) logical = (bid & 7) * (nb >> 3) + (bid >> 3);
  constexpr int GM = 8;
  const int per_group = GM * tiles_n;
  const int group = logical / per_group;
  const int first_m = group * GM;
  const int gsize = min(tiles_m - first_m, GM);
  const int in_group = logical - group * per_group;
  tm = first_m + in_group % gsize;
  tn = in_group / gsize;
}

// 16-byte LDS slot of chunk kc (8 bf16 along K) of tile row `row`: rows are
// 128 bytes (BK = 64) and the chunk index is XOR-swizzled with the row's low
// three bits, so the 16-byte fragment reads of 8 consecutive rows at one K
// offset land in 8 distinct bank groups (no padding needed).
__device__ __forceinline__ int slot(int row, int kc) { return row * 8 + (kc ^ (row & 7)); }

template <int BM, int BN, int EPI>
__global__ __launch_bounds__(256) void gemm_nt_kernel(GemmArgs p) {
  constexpr int BK = 64;
  constexpr int WM = BM / 2, WN = BN / 2;
  constexpr int FM = WM / 32, FN = WN / 32;
  constexpr int CA = BM * 8 / 256;  // 16-byte chunks per thread and K-slab
  constexpr int CB = BN * 8 / 256;
  static_assert(CA >= 1 && CB >= 1, "tile too small");

  __shared__ uint4 sA[2][BM * 8];
  __shared__ uint4 sB[2][BN * 8];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  int tm, tn;
  tile_of(blockIdx.x, gridDim.x, p.tiles_m, p.tiles_n, tm, tn);
  const int64_t m0 = int64_t(tm) * BM, n0 = int64_t(tn) * BN;
  const int64_t K = p.K;

  // Global -> register staging.  Chunk c of a slab: row c / 8, chunk c % 8,
  // so 8 consecutive lanes read one 128-byte row segment.
  const uint16_t* gA[CA];
  const uint16_t* gB[CB];
  bool okA[CA], okB[CB];
#pragma unroll
  for (int c = 0; c < CA; ++c) {
    const int idx = tid + c * 256;
    const int64_t r = m0 + (idx >> 3);
    okA[c] = r < p.M;
    gA[c] = p.A + (okA[c] ? r : 0) * K + (idx & 7) * 8;
  }
#pragma unroll
  for (int c = 0; c < CB; ++c) {
    const int idx = tid + c * 256;
    const int64_t r = n0 + (idx >> 3);
    okB[c] = r < p.N;
    gB[c] = p.B + (okB[c] ? r : 0) * K + (idx & 7) * 8;
  }
  uint4 ra[CA], rb[CB];
  const bool interior = (m0 + BM <= p.M) && (n0 + BN <= p.N);
  auto gload = [&](int64_t k0) {
    if (interior && k0 + BK <= K) {  // uniform: no per-chunk bounds checks
#pragma unroll
      for (int c = 0; c < CA; ++c) ra[c] = *reinterpret_cast<const uint4*>(gA[c] + k0);
#pragma unroll
      for (int c = 0; c < CB; ++c) rb[c] = *reinterpret_cast<const uint4*>(gB[c] + k0);
      return;
    }
#pragma unroll
    for (int c = 0; c < CA; ++c) {
      const bool ok = okA[c] && (k0 + ((tid + c * 256) & 7) * 8 < K);
      ra[c] = ok ? *reinterpret_cast<const uint4*>(gA[c] + k0) : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int c = 0; c < CB; ++c) {
      const bool ok = okB[c] && (k0 + ((tid + c * 256) & 7) * 8 < K);
      rb[c] = ok ? *reinterpret_cast<const uint4*>(gB[c] + k0) : make_uint4(0, 0, 0, 0);
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int c = 0; c < CA; ++c) {
      const int idx = tid + c * 256;
      sA[buf][slot(idx >> 3, idx & 7)] = ra[c];
    }
#pragma unroll
    for (int c = 0; c < CB; ++c) {
      const int idx = tid + c * 256;
      sB[buf][slot(idx >> 3, idx & 7)] = rb[c];
    }
  };

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int lr = lane & 31, lh = lane >> 5;
  const int nk = int((K + BK - 1) / BK);
  gload(0);
  lstore(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) gload(int64_t(kt + 1) * BK);
    const uint4* a_s = sA[buf];
    const uint4* b_s = sB[buf];
    // fragments of substep s+1 are read while the MFMAs of substep s run
    bf16x8 af[2][FM], bfr[2][FN];
    auto fload = [&](int s, int d) {
      const int kc = s * 2 + lh;
#pragma unroll
      for (int i = 0; i < FM; ++i)
        af[d][i] = __builtin_bit_cast(bf16x8, a_s[(wm * WM + i * 32 + lr) * 8 + (kc ^ (lr & 7))]);
#pragma unroll
      for (int j = 0; j < FN; ++j)
        bfr[d][j] = __builtin_bit_cast(bf16x8, b_s[(wn * WN + j * 32 + lr) * 8 + (kc ^ (lr & 7))]);
    };
    fload(0, 0);
#pragma unroll
    for (int s = 0; s < BK / 16; ++s) {
      if (s + 1 < BK / 16) fload(s + 1, (s + 1) & 1);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[s & 1][i], bfr[s & 1][j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) lstore(buf ^ 1);
    __syncthreads();
  }

  // Epilogue.  Accumulator register r of lane l holds row
  // 8*(r/4) + 4*(l/32) + r%4 and column l%32 of its 32x32 block.  For the
  // loss epilogue the 16 target values of a block are loaded in one batch
  // (16 independent loads in flight) before they are used.
  const bool full = (m0 + BM <= p.M) && (n0 + BN <= p.N);
  float lsum = 0.0f;
  const float* __restrict__ Yt = p.Yt;
#pragma unroll
  for (int i = 0; i < FM; ++i) {
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int64_t col = n0 + wn * WN + j * 32 + lr;
      const int64_t row0 = m0 + wm * WM + i * 32 + 4 * lh;
      const int64_t base = row0 * p.N + col;
      bool ok[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int dr = 8 * (r >> 2) + (r & 3);
        ok[r] = full || (row0 + dr < p.M && col < p.N);
      }
      float y[16];
      if constexpr (EPI == EPI_LOSS) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int dr = 8 * (r >> 2) + (r & 3);
          y[r] = ok[r] ? Yt[base + int64_t(dr) * p.N] : 0.0f;
        }
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        if (!ok[r]) continue;
        const int dr = 8 * (r >> 2) + (r & 3);
        const int64_t o = base + int64_t(dr) * p.N;
        const float v = acc[i][j][r];
        if constexpr (EPI == EPI_TARGET) {
          static_cast<float*>(p.out)[o] = v;
        } else if constexpr (EPI == EPI_LOSS) {
          const float e = v - y[r];
          lsum += e * e;
          static_cast<uint16_t*>(p.out)[o] = uint16_t(bf16_rne(e));
        } else if constexpr (EPI == EPI_GRAD_BF16) {
          static_cast<uint16_t*>(p.out)[o] = uint16_t(bf16_rne(p.scale * v));
        } else {
          static_cast<float*>(p.out)[o] = p.scale * v;
        }
      }
    }
  }
  if constexpr (EPI == EPI_LOSS) {
    __shared__ float sred[4];
    for (int msk = 32; msk >= 1; msk >>= 1) lsum += __shfl_xor(lsum, msk, 64);
    if (lane == 0) sred[wave] = lsum;
    __syncthreads();
    if (tid == 0) p.partials[blockIdx.x] = (sred[0] + sred[1]) + (sred[2] + sred[3]);
  }
}

template <int BM, int BN>
static int tiles(int64_t M, int64_t N) {
  return int(((M + BM - 1) / BM) * ((N + BN - 1) / BN));
}

// Tile shape: the largest of 256x256, 256x128, 128x128 that still gives at
// least one workgroup per compute unit (larger tiles move fewer operand
// bytes per flop through L2 and LDS).
enum TileShape { T256x256, T256x128, T128x128 };
static TileShape pick(int64_t M, int64_t N) {
  if (tiles<256, 256>(M, N) >= 256) return T256x256;
  if (tiles<256, 128>(M, N) >= 256) return T256x128;
  return T128x128;
}

size_t gemm_workgroups(int64_t M, int64_t N, int /*epi*/) {
  switch (pick(M, N)) {
    case T256x256: return size_t(tiles<256, 256>(M, N));
    case T256x128: return size_t(tiles<256, 128>(M, N));
    default: return size_t(tiles<128, 128>(M, N));
  }
}

template <int BM, int BN>
static hipError_t launch_bm(const GemmLaunch& q, hipStream_t st) {
  GemmArgs a;
  a.A = q.A; a.B = q.B; a.M = q.M; a.N = q.N; a.K = q.K;
  a.Yt = q.Yt; a.out = q.out; a.partials = q.partials; a.scale = q.scale;
  a.tiles_m = int((q.M + BM - 1) / BM);
  a.tiles_n = int((q.N + BN - 1) / BN);
  const dim3 grid(unsigned(a.tiles_m * a.tiles_n)), block(256);
  switch (q.epi) {
    case EPI_TARGET: hipLaunchKernelGGL((gemm_nt_kernel<BM, BN, EPI_TARGET>), grid, block, 0, st, a); break;
    case EPI_LOSS: hipLaunchKernelGGL((gemm_nt_kernel<BM, BN, EPI_LOSS>), grid, block, 0, st, a); break;
    case EPI_GRAD_BF16: hipLaunchKernelGGL((gemm_nt_kernel<BM, BN, EPI_GRAD_BF16>), grid, block, 0, st, a); break;
    default: hipLaunchKernelGGL((gemm_nt_kernel<BM, BN, EPI_GRAD_F32>), grid, block, 0, st, a); break;
  }
  return hipGetLastError();
}

hipError_t launch_gemm(const GemmLaunch& q, hipStream_t st) {
  switch (pick(q.M, q.N)) {
    case T256x256: return launch_bm<256, 256>(q, st);
    case T256x128: return launch_bm<256, 128>(q, st);
    default: return launch_bm<128, 128>(q, st);
  }
}

// Deterministic loss: fixed strided fp64 partial sums, then a fixed tree.
__global__ __launch_bounds__(256) void reduce_loss_kernel(const float* __restrict__ partials, int64_t n,
                                                          float* __restrict__ loss) {
  __shared__ double sm[256];
  double acc = 0.0;
  for (int64_t i = threadIdx.x; i < n; i += 256) acc += double(partials[i]);
  sm[threadIdx.x] = acc;
  __syncthreads();
  for (int w = 128; w >= 1; w >>= 1) {
    if (threadIdx.x < w) sm[threadIdx.x] += sm[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) loss[0] = float(sm[0]);
}

hipError_t launch_reduce_loss(const float* partials, int64_t n, float* loss, hipStream_t st) {
  hipLaunchKernelGGL(reduce_loss_kernel, dim3(1), dim3(256), 0, st, partials, n, loss);
  return hipGetLastError();
}

// out[c, r] = in[r, c]; 64 x 64 tiles through LDS (padded against conflicts).
__global__ __launch_bounds__(256) void transpose_kernel(const uint16_t* __restrict__ in, uint16_t* __restrict__ out,
                                                        int64_t rows, int64_t cols) {
  __shared__ uint16_t t[64][66];
  const int64_t r0 = int64_t(blockIdx.y) * 64, c0 = int64_t(blockIdx.x) * 64;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int i = ty; i < 64; i += 4) {
    const int64_t r = r0 + i, c = c0 + tx;
    t[i][tx] = (r < rows && c < cols) ? in[r * cols + c] : uint16_t(0);
  }
  __syncthreads();
  for (int i = ty; i < 64; i += 4) {
    const int64_t c = c0 + i, r = r0 + tx;
    if (c < cols && r < rows) out[c * rows + r] = t[tx][i];
  }
}

hipError_t launch_transpose(int64_t rows, int64_t cols, const uint16_t* in, uint16_t* out, hipStream_t st) {
  const dim3 grid(unsigned((cols + 63) / 64), unsigned((rows + 63) / 64));
  hipLaunchKernelGGL(transpose_kernel, grid, dim3(256), 0, st, in, out, rows, cols);
  return hipGetLastError();
}

__global__ __launch_bounds__(256) void sgd_kernel(int64_t n, float* __restrict__ theta,
                                                  const float* __restrict__ grad, float lr) {
  for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < n; i += int64_t(gridDim.x) * 256)
    theta[i] = theta[i] - lr * grad[i];
}

hipError_t launch_sgd(int64_t n, float* theta, const float* grad, float lr, hipStream_t st) {
  int64_t blocks = (n + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(sgd_kernel, dim3(unsigned(blocks)), dim3(256), 0, st, n, theta, grad, lr);
  return hipGetLastError();
}

}  // namespace uq
