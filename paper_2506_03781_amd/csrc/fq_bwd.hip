// Straight-through backward of the quantizer with the gradient filter
// (appendix "Implementation details": the non-differentiable mapping passes
// the gradient of the mapped weight to the transformed weight, except where
// the stored mask bit says |wbar - wtilde| > tau).
//
// Each lane streams 8 consecutive weights (dL/dWhat, W, s, code byte) and
// writes 8 grad_s values; a 128-weight group is 16 lanes of one wavefront
// and its sums (k signed sums for alpha, one for z_B, optional ones for
// Delta, z_U and the row scale) are reduced with a fixed xor-butterfly, so
// results are bitwise reproducible.  HBM-bound: 13 B per weight.
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

  float S = 0.0f, Sa[K], GD = 0.0f, GZ = 0.0f, P = 0.0f;
#pragma unroll
  for (int b = 0; b < K; ++b) Sa[b] = 0.0f;
  float dl = 1.0f;
  if (active) {
    float w[8], sv[8], G[8];
    load8<WDT>(a.W, off, w);
    load8f(a.s, off, sv);
    load8<GDT>(a.G, off, G);
    const uint2 cb = load8u8(a.codes, off);
    dl = a.delta ? a.delta[gid] : 1.0f;
    const float sr = a.s_r ? a.s_r[uint32_t(gid) / uint32_t(a.gpr)] : 1.0f;
    const float zu = a.z_u ? a.z_u[gid] : 0.0f;
    const float ds = dl * sr;
    float al[K];
    float zb = 0.0f;
    if (want_delta) {
      zb = a.z_b[gid];
#pragma unroll
      for (int b = 0; b < K; ++b) al[b] = a.alpha[gid * K + b];
    }
    float gs[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const uint32_t byte = byte_of(cb, i);
      const bool m = (byte & 0x80u) != 0u;
      const float g = G[i];
      S += g;
#pragma unroll
      for (int b = 0; b < K; ++b) Sa[b] += ((byte >> b) & 1u) ? g : -g;
      // x = wbar - z_U = w / (Delta s_r s)
      const float x = w[i] * __builtin_amdgcn_rcpf(ds * sv[i]);
      gs[i] = m ? -(dl * g) * x * __builtin_amdgcn_rcpf(sv[i]) : 0.0f;
      if (want_delta) {
        float wt = zb;
#pragma unroll
        for (int b = 0; b < K; ++b) wt = ((byte >> b) & 1u) ? wt + al[b] : wt - al[b];
        GD += g * ((wt - zu) - (m ? x : 0.0f));
      }
      if (want_zu && !m) GZ += g;
      if (want_sr && m) P += g * x;
    }
    if (a.grad_s) store8f(a.grad_s, off, gs);
    if (a.update) {
      float sn[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) sn[i] = sv[i] - a.lr_f * gs[i];
      store8f(const_cast<float*>(a.s), off, sn);
    }
  }
  // group reduction over lpg lanes (lpg is a power of two <= 64)
  for (int msk = lpg >> 1; msk >= 1; msk >>= 1) {
    S += __shfl_xor(S, msk, 64);
#pragma unroll
    for (int b = 0; b < K; ++b) Sa[b] += __shfl_xor(Sa[b], msk, 64);
    if (want_delta) GD += __shfl_xor(GD, msk, 64);
    if (want_zu) GZ += __shfl_xor(GZ, msk, 64);
    if (want_sr) P += __shfl_xor(P, msk, 64);
  }
  if (active && (threadIdx.x & (lpg - 1)) == 0) {
    const float gzb = dl * S;
    if (a.grad_z_b) a.grad_z_b[gid] = gzb;
    if (a.grad_alpha) {
#pragma unroll
      for (int b = 0; b < K; ++b) a.grad_alpha[gid * K + b] = dl * Sa[b];
    }
    if (a.update) {
      // every lane of the group read alpha / z_b before the butterfly above
      float* alpha = const_cast<float*>(a.alpha);
      float* z_b = const_cast<float*>(a.z_b);
#pragma unroll
      for (int b = 0; b < K; ++b) alpha[gid * K + b] = alpha[gid * K + b] - a.lr_b * (dl * Sa[b]);
      z_b[gid] = z_b[gid] - a.lr_b * gzb;
    }
    if (want_delta) a.grad_delta[gid] = GD;
    if (want_zu) a.grad_z_u[gid] = -dl * GZ;
    if (want_sr) a.group_ws[gid] = -dl * P;
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
  a.logg = __builtin_ctz(unsigned(p.g));
  a.gpr = int(p.C / p.g);
  a.W = p.W; a.s = p.s; a.s_r = p.s_r; a.delta = p.delta; a.z_u = p.z_u;
  a.alpha = p.alpha; a.z_b = p.z_b; a.codes = p.codes; a.G = p.grad_W_hat;
  a.grad_s = p.grad_s; a.grad_alpha = p.grad_alpha; a.grad_z_b = p.grad_z_b;
  a.grad_delta = p.grad_delta; a.grad_z_u = p.grad_z_u;
  a.group_ws = p.grad_s_r ? p.group_ws : nullptr;
  a.update = p.update;
  a.lr_f = p.lr_f;
  a.lr_b = p.lr_b;
  const int64_t chunks = a.N / kVec;
  const dim3 grid(unsigned((chunks + kThreads - 1) / kThreads));
  if (p.w_dtype == BF16 && p.grad_dtype == BF16) launch_k<BF16, BF16>(a, p.k, grid, st);
  else if (p.w_dtype == BF16) launch_k<BF16, F32>(a, p.k, grid, st);
  else if (p.grad_dtype == BF16) launch_k<F32, BF16>(a, p.k, grid, st);
  else launch_k<F32, F32>(a, p.k, grid, st);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.grad_s_r == nullptr) return e;
  hipLaunchKernelGGL(row_reduce_kernel, dim3(unsigned((p.R + 255) / 256)), dim3(256), 0, st,
                     p.group_ws, p.R, a.gpr, p.s_r, p.grad_s_r);
  return hipGetLastError();
}

}  // namespace uq
