// Straight-through backward of the quantizer with the gradient filter
// (appendix "Implementation details": the non-differentiable mapping passes
// the gradient of the mapped weight to the transformed weight, except where
// the stored mask bit says |wbar - wtilde| > tau).
//
// Each lane streams 8 consecutive weights (dL/dWhat, W, s, code byte) and
// writes 8 grad_s values; a 128-weight group is 16 lanes of one wavefront
// and its sums (k signed sums for alpha, one for z_B, optional ones for
// Delta, z_U and the row scale) are reduced with a fixed xor-butterfly, so
// results are bitwise reproducible.  Groups larger than 512 weights (per-row
// groups) take one workgroup each.  HBM-bound: 13 B per weight.
#include "uq_device.h"
#include "uq_launch.h"

namespace uq {

struct BwdArgs {
  int64_t N;
  int logg, gpr;
  const void* W;
  const float* s;
  const float* s_r;
  const float* delta;
  const float* z_u;
  const float* alpha;
  const float* z_b;
  const uint8_t* codes;
  const void* G;
  float* grad_s;
  float* grad_alpha;
  float* grad_z_b;
  float* grad_delta;
  float* grad_z_u;
  float* group_ws;
  // in-place SGD (update != 0): s -= lr_f grad_s; alpha, z_b -= lr_b grad
  int update;
  float lr_f, lr_b;
};

// Per-group values the straight-through backward of one weight needs.
template <int K>
struct BwdGroup {
  float dl, zu, ds, zb;
  float al[K];
};

template <int K>
__device__ __forceinline__ BwdGroup<K> bwd_group(const BwdArgs& a, int64_t gid, bool want_delta) {
  BwdGroup<K> q;
  q.dl = a.delta ? a.delta[gid] : 1.0f;
  const float sr = a.s_r ? a.s_r[uint32_t(gid) / uint32_t(a.gpr)] : 1.0f;
  q.zu = a.z_u ? a.z_u[gid] : 0.0f;
  q.ds = q.dl * sr;
  q.zb = 0.0f;
  if (want_delta) {
    q.zb = a.z_b[gid];
#pragma unroll
    for (int b = 0; b < K; ++b) q.al[b] = a.alpha[gid * K + b];
  }
  return q;
}

// Running group sums of one lane.
template <int K>
struct BwdSums {
  float S, Sa[K], GD, GZ, P;
  __device__ __forceinline__ void zero() {
    S = GD = GZ = P = 0.0f;
#pragma unroll
    for (int b = 0; b < K; ++b) Sa[b] = 0.0f;
  }
};

// The 8 weights at `off`: grad_s (stored, and the SGD update of s when
// requested) and this lane's contributions to the group sums.
template <int WDT, int GDT, int K>
__device__ __forceinline__ void bwd_chunk(const BwdArgs& a, int64_t off, const BwdGroup<K>& q, BwdSums<K>& t,
                                          bool want_delta, bool want_zu, bool want_sr) {
  float w[8], sv[8], G[8];
  load8<WDT>(a.W, off, w);
  load8f(a.s, off, sv);
  load8<GDT>(a.G, off, G);
  const uint2 cb = load8u8(a.codes, off);
  float gs[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const uint32_t byte = byte_of(cb, i);
    const bool m = (byte & 0x80u) != 0u;
    const float g = G[i];
    t.S += g;
#pragma unroll
    for (int b = 0; b < K; ++b) t.Sa[b] += ((byte >> b) & 1u) ? g : -g;
    // x = wbar - z_U = w / (Delta s_r s)
    const float x = w[i] * __builtin_amdgcn_rcpf(q.ds * sv[i]);
    gs[i] = m ? -(q.dl * g) * x * __builtin_amdgcn_rcpf(sv[i]) : 0.0f;
    if (want_delta) {
      float wt = q.zb;
#pragma unroll
      for (int b = 0; b < K; ++b) wt = ((byte >> b) & 1u) ? wt + q.al[b] : wt - q.al[b];
      t.GD += g * ((wt - q.zu) - (m ? x : 0.0f));
    }
    if (want_zu && !m) t.GZ += g;
    if (want_sr && m) t.P += g * x;
  }
  if (a.grad_s) store8f(a.grad_s, off, gs);
  if (a.update) {
    float sn[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) sn[i] = sv[i] - a.lr_f * gs[i];
    store8f(const_cast<float*>(a.s), off, sn);
  }
}

// The group's outputs from its reduced sums (one lane per group).
template <int K>
__device__ __forceinline__ void bwd_finish(const BwdArgs& a, int64_t gid, float dl, const BwdSums<K>& t,
                                           bool want_delta, bool want_zu, bool want_sr) {
  const float gzb = dl * t.S;
  if (a.grad_z_b) a.grad_z_b[gid] = gzb;
  if (a.grad_alpha) {
#pragma unroll
    for (int b = 0; b < K; ++b) a.grad_alpha[gid * K + b] = dl * t.Sa[b];
  }
  if (a.update) {
    // every lane of the group read alpha / z_b before the reduction
    float* alpha = const_cast<float*>(a.alpha);
    float* z_b = const_cast<float*>(a.z_b);
#pragma unroll
    for (int b = 0; b < K; ++b) alpha[gid * K + b] = alpha[gid * K + b] - a.lr_b * (dl * t.Sa[b]);
    z_b[gid] = z_b[gid] - a.lr_b * gzb;
  }
  if (want_delta) a.grad_delta[gid] = t.GD;
  if (want_zu) a.grad_z_u[gid] = -dl * t.GZ;
  if (want_sr) a.group_ws[gid] = -dl * t.P;
}

template <int WDT, int GDT, int K>
__global__ __launch_bounds__(kThreads) void fq_bwd_kernel(BwdArgs a) {
  const int64_t chunk = int64_t(blockIdx.x) * kThreads + threadIdx.x;
  const int64_t off = chunk * kVec;
  const bool active = off < a.N;
  const int lpg = 1 << (a.logg - 3);
  const int64_t gid = active ? (off >> a.logg) : 0;
  const bool want_delta = a.grad_delta != nullptr;
  const bool want_zu = a.grad_z_u != nullptr;
  const bool want_sr = a.group_ws != nullptr;

  BwdSums<K> t;
  t.zero();
  float dl = 1.0f;
  if (active) {
    const BwdGroup<K> q = bwd_group<K>(a, gid, want_delta);
    dl = q.dl;
    bwd_chunk<WDT, GDT, K>(a, off, q, t, want_delta, want_zu, want_sr);
  }
  // group reduction over lpg lanes (lpg is a power of two <= 64)
  for (int msk = lpg >> 1; msk >= 1; msk >>= 1) {
    t.S += __shfl_xor(t.S, msk, 64);
#pragma unroll
    for (int b = 0; b < K; ++b) t.Sa[b] += __shfl_xor(t.Sa[b], msk, 64);
    if (want_delta) t.GD += __shfl_xor(t.GD, msk, 64);
    if (want_zu) t.GZ += __shfl_xor(t.GZ, msk, 64);
    if (want_sr) t.P += __shfl_xor(t.P, msk, 64);
  }
  if (active && (threadIdx.x & (lpg - 1)) == 0) bwd_finish<K>(a, gid, dl, t, want_delta, want_zu, want_sr);
}

// Groups larger than 512 weights (per-row groups): one workgroup of 256
// lanes per group.  Each lane sums its chunks in order (chunk c = lane,
// lane + 256, ...), then the wavefront sums by a fixed xor butterfly and the
// four wavefront sums pairwise, so the results are bitwise reproducible.
constexpr int kBigBwdThreads = 256;

template <int WDT, int GDT, int K>
__global__ __launch_bounds__(kBigBwdThreads) void fq_bwd_big_kernel(BwdArgs a, int g) {
  __shared__ float red[4][K + 4];
  const int64_t gid = blockIdx.x;
  const bool want_delta = a.grad_delta != nullptr;
  const bool want_zu = a.grad_z_u != nullptr;
  const bool want_sr = a.group_ws != nullptr;
  const BwdGroup<K> q = bwd_group<K>(a, gid, want_delta);
  BwdSums<K> t;
  t.zero();
  const int nch = g >> 3;
  const int64_t base = gid * g;
  for (int c = threadIdx.x; c < nch; c += kBigBwdThreads)
    bwd_chunk<WDT, GDT, K>(a, base + int64_t(c) * kVec, q, t, want_delta, want_zu, want_sr);
  for (int msk = 32; msk >= 1; msk >>= 1) {
    t.S += __shfl_xor(t.S, msk, 64);
#pragma unroll
    for (int b = 0; b < K; ++b) t.Sa[b] += __shfl_xor(t.Sa[b], msk, 64);
    t.GD += __shfl_xor(t.GD, msk, 64);
    t.GZ += __shfl_xor(t.GZ, msk, 64);
    t.P += __shfl_xor(t.P, msk, 64);
  }
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    red[wave][0] = t.S;
#pragma unroll
    for (int b = 0; b < K; ++b) red[wave][1 + b] = t.Sa[b];
    red[wave][K + 1] = t.GD;
    red[wave][K + 2] = t.GZ;
    red[wave][K + 3] = t.P;
  }
  __syncthreads();  // also: every lane has read alpha / z_b before lane 0 updates them
  if (threadIdx.x == 0) {
    auto sum4 = [&](int j) { return (red[0][j] + red[1][j]) + (red[2][j] + red[3][j]); };
    t.S = sum4(0);
#pragma unroll
    for (int b = 0; b < K; ++b) t.Sa[b] = sum4(1 + b);
    t.GD = sum4(K + 1);
    t.GZ = sum4(K + 2);
    t.P = sum4(K + 3);
    bwd_finish<K>(a, gid, q.dl, t, want_delta, want_zu, want_sr);
  }
}

// grad_s_r[r] = (sum over the row's groups, in order) / s_r[r]
__global__ __launch_bounds__(256) void row_reduce_kernel(const float* __restrict__ ws, int64_t R, int gpr,
                                                         const float* __restrict__ s_r, float* __restrict__ out) {
  const int64_t r = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (r >= R) return;
  float acc = 0.0f;
  for (int j = 0; j < gpr; ++j) acc += ws[r * gpr + j];
  out[r] = acc / (s_r ? s_r[r] : 1.0f);
}

template <int WDT, int GDT>
static void launch_big(const BwdArgs& a, int k, int g, dim3 grid, hipStream_t st) {
  const dim3 block(kBigBwdThreads);
  switch (k) {
    case 1: hipLaunchKernelGGL((fq_bwd_big_kernel<WDT, GDT, 1>), grid, block, 0, st, a, g); break;
    case 2: hipLaunchKernelGGL((fq_bwd_big_kernel<WDT, GDT, 2>), grid, block, 0, st, a, g); break;
    case 3: hipLaunchKernelGGL((fq_bwd_big_kernel<WDT, GDT, 3>), grid, block, 0, st, a, g); break;
    case 4: hipLaunchKernelGGL((fq_bwd_big_kernel<WDT, GDT, 4>), grid, block, 0, st, a, g); break;
    case 5: hipLaunchKernelGGL((fq_bwd_big_kernel<WDT, GDT, 5>), grid, block, 0, st, a, g); break;
    case 6: hipLaunchKernelGGL((fq_bwd_big_kernel<WDT, GDT, 6>), grid, block, 0, st, a, g); break;
    default: hipLaunchKernelGGL((fq_bwd_big_kernel<WDT, GDT, 7>), grid, block, 0, st, a, g); break;
  }
}

template <int WDT, int GDT>
static void launch_k(const BwdArgs& a, int k, dim3 grid, hipStream_t st) {
  switch (k) {
    case 1: hipLaunchKernelGGL((fq_bwd_kernel<WDT, GDT, 1>), grid, dim3(kThreads), 0, st, a); break;
    case 2: hipLaunchKernelGGL((fq_bwd_kernel<WDT, GDT, 2>), grid, dim3(kThreads), 0, st, a); break;
    case 3: hipLaunchKernelGGL((fq_bwd_kernel<WDT, GDT, 3>), grid, dim3(kThreads), 0, st, a); break;
    case 4: hipLaunchKernelGGL((fq_bwd_kernel<WDT, GDT, 4>), grid, dim3(kThreads), 0, st, a); break;
    case 5: hipLaunchKernelGGL((fq_bwd_kernel<WDT, GDT, 5>), grid, dim3(kThreads), 0, st, a); break;
    case 6: hipLaunchKernelGGL((fq_bwd_kernel<WDT, GDT, 6>), grid, dim3(kThreads), 0, st, a); break;
    default: hipLaunchKernelGGL((fq_bwd_kernel<WDT, GDT, 7>), grid, dim3(kThreads), 0, st, a); break;
  }
}

hipError_t launch_fq_bwd(const FqBwdLaunch& p, hipStream_t st) {
  BwdArgs a;
  a.N = p.R * p.C;
  a.logg = p.g <= 512 ? __builtin_ctz(unsigned(p.g)) : 0;
  a.gpr = int(p.C / p.g);
  a.W = p.W; a.s = p.s; a.s_r = p.s_r; a.delta = p.delta; a.z_u = p.z_u;
  a.alpha = p.alpha; a.z_b = p.z_b; a.codes = p.codes; a.G = p.grad_W_hat;
  a.grad_s = p.grad_s; a.grad_alpha = p.grad_alpha; a.grad_z_b = p.grad_z_b;
  a.grad_delta = p.grad_delta; a.grad_z_u = p.grad_z_u;
  a.group_ws = p.grad_s_r ? p.group_ws : nullptr;
  a.update = p.update;
  a.lr_f = p.lr_f;
  a.lr_b = p.lr_b;
  if (p.g > 512) {
    const dim3 grid(unsigned(a.N / p.g));
    if (p.w_dtype == BF16 && p.grad_dtype == BF16) launch_big<BF16, BF16>(a, p.k, p.g, grid, st);
    else if (p.w_dtype == BF16) launch_big<BF16, F32>(a, p.k, p.g, grid, st);
    else if (p.grad_dtype == BF16) launch_big<F32, BF16>(a, p.k, p.g, grid, st);
    else launch_big<F32, F32>(a, p.k, p.g, grid, st);
  } else {
    const int64_t chunks = a.N / kVec;
    const dim3 grid(unsigned((chunks + kThreads - 1) / kThreads));
    if (p.w_dtype == BF16 && p.grad_dtype == BF16) launch_k<BF16, BF16>(a, p.k, grid, st);
    else if (p.w_dtype == BF16) launch_k<BF16, F32>(a, p.k, grid, st);
    else if (p.grad_dtype == BF16) launch_k<F32, BF16>(a, p.k, grid, st);
    else launch_k<F32, F32>(a, p.k, grid, st);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.grad_s_r == nullptr) return e;
  hipLaunchKernelGGL(row_reduce_kernel, dim3(unsigned((p.R + 255) / 256)), dim3(256), 0, st,
                     p.group_ws, p.R, a.gpr, p.s_r, p.grad_s_r);
  return hipGetLastError();
}

}  // namespace uq
