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
// Z = bf16((R r) gamma).  C is a multiple of 8; lane l takes the four
// consecutive columns 4 l + 256 j, so each load covers 1 KB of the row.
__global__ __launch_bounds__(256) void add_rmsnorm_kernel(int64_t T, int64_t C, const float* __restrict__ X,
                                                          const float* __restrict__ A, const float* __restrict__ gamma,
                                                          float* __restrict__ R, uint16_t* __restrict__ Z,
                                                          float* __restrict__ rinv) {
  const int lane = threadIdx.x & 63;
  const int64_t row = int64_t(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (row >= T) return;
  const float4* x = reinterpret_cast<const float4*>(X + row * C);
  const float4* a = A ? reinterpret_cast<const float4*>(A + row * C) : nullptr;
  const int64_t n4 = C / 4;
  float ss = 0.0f;
#pragma unroll 4
  for (int64_t c = lane; c < n4; c += 64) {
    float4 v = x[c];
    if (a) {
      const float4 w = a[c];
      v.x += w.x; v.y += w.y; v.z += w.z; v.w += w.w;
    }
    ss += v.x * v.x;
    ss += v.y * v.y;
    ss += v.z * v.z;
    ss += v.w * v.w;
  }
  ss = wave_sum(ss);
  const float r = 1.0f / sqrtf(ss / float(C) + 1e-5f);
  if (lane == 0) rinv[row] = r;
  const float4* g4 = reinterpret_cast<const float4*>(gamma);
  float4* R4 = R ? reinterpret_cast<float4*>(R + row * C) : nullptr;
  uint2* Z2 = reinterpret_cast<uint2*>(Z + row * C);
#pragma unroll 4
  for (int64_t c = lane; c < n4; c += 64) {
    float4 v = x[c];
    if (a) {
      const float4 w = a[c];
      v.x += w.x; v.y += w.y; v.z += w.z; v.w += w.w;
    }
    if (R4) R4[c] = v;
    const float4 g = g4[c];
    Z2[c] = make_uint2(uint32_t(to_bf((v.x * r) * g.x)) | (uint32_t(to_bf((v.y * r) * g.y)) << 16),
                       uint32_t(to_bf((v.z * r) * g.z)) | (uint32_t(to_bf((v.w * r) * g.w)) << 16));
  }
}

// One wavefront per row: dR = escale * E + r g - x r^3 sum(g x) / C with
// g = gamma (dZa + dZb); writes dR in bf16 (and in fp32 when dRf is given).
// Same lane layout as the forward (four consecutive columns per access).
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
  const int64_t n4 = C / 4;
  const float4* za = reinterpret_cast<const float4*>(dZa + base);
  const float4* zb = dZb ? reinterpret_cast<const float4*>(dZb + base) : nullptr;
  const float4* x4 = reinterpret_cast<const float4*>(Xin + base);
  const float4* g4 = reinterpret_cast<const float4*>(gamma);
  auto gdz = [&](int64_t c) {
    float4 z = za[c];
    if (zb) {
      const float4 w = zb[c];
      z.x += w.x; z.y += w.y; z.z += w.z; z.w += w.w;
    }
    const float4 g = g4[c];
    return make_float4(g.x * z.x, g.y * z.y, g.z * z.z, g.w * z.w);
  };
  float dot = 0.0f;
#pragma unroll 4
  for (int64_t c = lane; c < n4; c += 64) {
    const float4 g = gdz(c);
    const float4 v = x4[c];
    dot += g.x * v.x;
    dot += g.y * v.y;
    dot += g.z * v.z;
    dot += g.w * v.w;
  }
  dot = wave_sum(dot);
  const float r = rinv[row];
  const float k3 = (r * r * r) * (dot / float(C));
  const uint2* e2 = E ? reinterpret_cast<const uint2*>(E + base) : nullptr;
  uint2* d2 = reinterpret_cast<uint2*>(dR + base);
  float4* df = dRf ? reinterpret_cast<float4*>(dRf + base) : nullptr;
#pragma unroll 4
  for (int64_t c = lane; c < n4; c += 64) {
    const float4 g = gdz(c);
    const float4 v = x4[c];
    float o[4] = {r * g.x - v.x * k3, r * g.y - v.y * k3, r * g.z - v.z * k3, r * g.w - v.w * k3};
    if (e2) {
      const uint2 e = e2[c];
      o[0] += escale * bf(uint16_t(e.x & 0xFFFFu));
      o[1] += escale * bf(uint16_t(e.x >> 16));
      o[2] += escale * bf(uint16_t(e.y & 0xFFFFu));
      o[3] += escale * bf(uint16_t(e.y >> 16));
    }
    d2[c] = make_uint2(uint32_t(to_bf(o[0])) | (uint32_t(to_bf(o[1])) << 16),
                       uint32_t(to_bf(o[2])) | (uint32_t(to_bf(o[3])) << 16));
    if (df) df[c] = make_float4(o[0], o[1], o[2], o[3]);
  }
}

// Row-resident forms of the two kernels above for C = 256 NV (NV <= 16): the
// row's values stay in registers between the reduction and the output pass,
// so each input is read once.  Same lane layout (lane l takes float4 l + 64 k)
// and the same order of every sum and product as the two-pass kernels, so
// the results are the same bit for bit.
template <int NV>
__global__ __launch_bounds__(256) void add_rmsnorm_rows_kernel(int64_t T, int64_t C, const float* __restrict__ X,
                                                               const float* __restrict__ A,
                                                               const float* __restrict__ gamma,
                                                               float* __restrict__ R, uint16_t* __restrict__ Z,
                                                               float* __restrict__ rinv) {
  const int lane = threadIdx.x & 63;
  const int64_t row = int64_t(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (row >= T) return;
  const float4* x = reinterpret_cast<const float4*>(X + row * C);
  const float4* a = A ? reinterpret_cast<const float4*>(A + row * C) : nullptr;
  float4 v[NV];
#pragma unroll
  for (int k = 0; k < NV; ++k) v[k] = x[lane + 64 * k];
  if (a) {
#pragma unroll
    for (int k = 0; k < NV; ++k) {
      const float4 w = a[lane + 64 * k];
      v[k].x += w.x; v[k].y += w.y; v[k].z += w.z; v[k].w += w.w;
    }
  }
  float ss = 0.0f;
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    ss += v[k].x * v[k].x;
    ss += v[k].y * v[k].y;
    ss += v[k].z * v[k].z;
    ss += v[k].w * v[k].w;
  }
  ss = wave_sum(ss);
  const float r = 1.0f / sqrtf(ss / float(C) + 1e-5f);
  if (lane == 0) rinv[row] = r;
  const float4* g4 = reinterpret_cast<const float4*>(gamma);
  float4* R4 = R ? reinterpret_cast<float4*>(R + row * C) : nullptr;
  uint2* Z2 = reinterpret_cast<uint2*>(Z + row * C);
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const int64_t c = lane + 64 * k;
    if (R4) R4[c] = v[k];
    const float4 g = g4[c];
    Z2[c] = make_uint2(uint32_t(to_bf((v[k].x * r) * g.x)) | (uint32_t(to_bf((v[k].y * r) * g.y)) << 16),
                       uint32_t(to_bf((v[k].z * r) * g.z)) | (uint32_t(to_bf((v[k].w * r) * g.w)) << 16));
  }
}

template <int NV>
__global__ __launch_bounds__(256) void rmsnorm_bwd_rows_kernel(int64_t T, int64_t C, const float* __restrict__ dZa,
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
  const float4* za = reinterpret_cast<const float4*>(dZa + base);
  const float4* zb = dZb ? reinterpret_cast<const float4*>(dZb + base) : nullptr;
  const float4* x4 = reinterpret_cast<const float4*>(Xin + base);
  const float4* g4 = reinterpret_cast<const float4*>(gamma);
  float4 gz[NV], xv[NV];
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    gz[k] = za[lane + 64 * k];
    xv[k] = x4[lane + 64 * k];
  }
  if (zb) {
#pragma unroll
    for (int k = 0; k < NV; ++k) {
      const float4 w = zb[lane + 64 * k];
      gz[k].x += w.x; gz[k].y += w.y; gz[k].z += w.z; gz[k].w += w.w;
    }
  }
  float dot = 0.0f;
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const float4 g = g4[lane + 64 * k];
    gz[k] = make_float4(g.x * gz[k].x, g.y * gz[k].y, g.z * gz[k].z, g.w * gz[k].w);
    dot += gz[k].x * xv[k].x;
    dot += gz[k].y * xv[k].y;
    dot += gz[k].z * xv[k].z;
    dot += gz[k].w * xv[k].w;
  }
  dot = wave_sum(dot);
  const float r = rinv[row];
  const float k3 = (r * r * r) * (dot / float(C));
  const uint2* e2 = E ? reinterpret_cast<const uint2*>(E + base) : nullptr;
  uint2* d2 = reinterpret_cast<uint2*>(dR + base);
  float4* df = dRf ? reinterpret_cast<float4*>(dRf + base) : nullptr;
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const int64_t c = lane + 64 * k;
    const float4 g = gz[k], v = xv[k];
    float o[4] = {r * g.x - v.x * k3, r * g.y - v.y * k3, r * g.z - v.z * k3, r * g.w - v.w * k3};
    if (e2) {
      const uint2 e = e2[c];
      o[0] += escale * bf(uint16_t(e.x & 0xFFFFu));
      o[1] += escale * bf(uint16_t(e.x >> 16));
      o[2] += escale * bf(uint16_t(e.y & 0xFFFFu));
      o[3] += escale * bf(uint16_t(e.y >> 16));
    }
    d2[c] = make_uint2(uint32_t(to_bf(o[0])) | (uint32_t(to_bf(o[1])) << 16),
                       uint32_t(to_bf(o[2])) | (uint32_t(to_bf(o[3])) << 16));
    if (df) df[c] = make_float4(o[0], o[1], o[2], o[3]);
  }
}

// Head h of a grouped layout (perm heads sharing a key/value head) is stored
// at slot (h mod perm) (H / perm) + h / perm: the heads at one position of
// their groups are contiguous, in key/value head order.
__device__ __forceinline__ int head_slot(int h, int H, int perm) {
  return perm > 1 ? (h % perm) * (H / perm) + h / perm : h;
}

// Token-major [T, C] (fp32 or bf16) -> head-major bf16 [H, T, d] (head h at
// head_slot(h)), rotating pairs (i, i + d/2) by the position's angle when
// ROT.  One thread per pair.
template <bool IN_F32, bool ROT>
__global__ __launch_bounds__(256) void rope_split_kernel(int64_t T, int H, int d, int L, int perm,
                                                         const void* __restrict__ in, uint16_t* __restrict__ out) {
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
  const int64_t dst = (int64_t(head_slot(h, H, perm)) * T + t) * d + i;
  out[dst] = to_bf(y1);
  out[dst + hd] = to_bf(y2);
}

// The same two layout changes for d a multiple of 16 (up to 512) and 16-byte
// aligned buffers: a workgroup takes RT consecutive tokens, computes the cos
// and sin of their d/2 angles once into LDS (the same angle and sincosf as
// the one-pair kernels, so the results are bit-identical), and moves chunks
// of 8 pairs with 16-byte accesses.
constexpr int RT = 4;           // tokens per workgroup
constexpr int RT_MAX_HD = 256;  // d / 2 limit of the LDS angle table

__device__ __forceinline__ void load8(const void* in, bool f32, int64_t off, float (&x)[8]) {
  if (f32) {
    const float4 a = *reinterpret_cast<const float4*>(static_cast<const float*>(in) + off);
    const float4 b = *reinterpret_cast<const float4*>(static_cast<const float*>(in) + off + 4);
    x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w; x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
  } else {
    const uint4 v = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(in) + off);
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      x[2 * j] = __uint_as_float(w[j] << 16);
      x[2 * j + 1] = __uint_as_float(w[j] & 0xFFFF0000u);
    }
  }
}

__device__ __forceinline__ void store8(uint16_t* out, const float (&y)[8]) {
  uint32_t w[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) w[j] = uint32_t(to_bf(y[2 * j])) | (uint32_t(to_bf(y[2 * j + 1])) << 16);
  *reinterpret_cast<uint4*>(out) = make_uint4(w[0], w[1], w[2], w[3]);
}

// cos and sin of the RT tokens' angles: cs[tt * hd + i] for token t0 + tt.
template <bool ROT>
__device__ __forceinline__ void rope_table(float2* cs, int64_t t0, int64_t T, int L, int d) {
  if (!ROT) return;
  const int hd = d >> 1;
  for (int k = threadIdx.x; k < RT * hd; k += 256) {
    const int tt = k / hd, i = k % hd;
    float sn = 0.0f, cn = 1.0f;
    if (t0 + tt < T) sincosf(rope_angle(int((t0 + tt) % L), i, d), &sn, &cn);
    cs[k] = make_float2(cn, sn);
  }
  __syncthreads();
}

// cos and sin of every pair at every position of an L-token sequence:
// cs[(p * (d / 2) + i) * 2 + {0, 1}] = cos, sin of rope_angle(p, i, d), the
// values the rotary kernels compute in place.
__global__ __launch_bounds__(256) void rope_table_kernel(int L, int d, float* __restrict__ cs) {
  const int hd = d >> 1;
  const int64_t k = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (k >= int64_t(L) * hd) return;
  float sn, cn;
  sincosf(rope_angle(int(k / hd), int(k % hd), d), &sn, &cn);
  cs[2 * k] = cn;
  cs[2 * k + 1] = sn;
}

template <bool IN_F32, bool ROT>
__global__ __launch_bounds__(256) void rope_split_vec_kernel(int64_t T, int H, int d, int L, int perm,
                                                             const void* __restrict__ in, uint16_t* __restrict__ out) {
  __shared__ float2 cs[RT * RT_MAX_HD];
  const int hd = d >> 1, cph = hd / 8, cpt = H * cph;  // chunks per head, per token
  const int64_t t0 = int64_t(blockIdx.x) * RT;
  rope_table<ROT>(cs, t0, T, L, d);
  for (int k = threadIdx.x; k < RT * cpt; k += 256) {
    const int tt = k / cpt, r = k % cpt;
    const int64_t t = t0 + tt;
    if (t >= T) break;
    const int h = r / cph, i = (r % cph) * 8;
    const int64_t src = t * (int64_t(H) * d) + int64_t(h) * d + i;
    float x1[8], x2[8], y1[8], y2[8];
    load8(in, IN_F32, src, x1);
    load8(in, IN_F32, src + hd, x2);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      if (ROT) {
        const float2 a = cs[tt * hd + i + e];
        y1[e] = x1[e] * a.x - x2[e] * a.y;
        y2[e] = x2[e] * a.x + x1[e] * a.y;
      } else {
        y1[e] = x1[e];
        y2[e] = x2[e];
      }
    }
    const int64_t dst = (int64_t(head_slot(h, H, perm)) * T + t) * d + i;
    store8(out + dst, y1);
    store8(out + dst + hd, y2);
  }
}

template <bool IN_F32, bool ROT>
__global__ __launch_bounds__(256) void rope_merge_vec_kernel(int64_t T, int H, int d, int L, int perm, int nsum,
                                                             const void* __restrict__ in, uint16_t* __restrict__ out,
                                                             int64_t ldo) {
  __shared__ float2 cs[RT * RT_MAX_HD];
  const int hd = d >> 1, cph = hd / 8, cpt = H * cph;
  const int64_t t0 = int64_t(blockIdx.x) * RT;
  const int64_t pstride = int64_t(H) * T * d;
  rope_table<ROT>(cs, t0, T, L, d);
  for (int k = threadIdx.x; k < RT * cpt; k += 256) {
    const int tt = k / cpt, r = k % cpt;
    const int64_t t = t0 + tt;
    if (t >= T) break;
    const int h = r / cph, i = (r % cph) * 8;
    const int64_t src0 = (int64_t(head_slot(h, H, perm)) * T + t) * d + i;
    float x1[8] = {0, 0, 0, 0, 0, 0, 0, 0}, x2[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int q = 0; q < nsum; ++q) {
      float v1[8], v2[8];
      load8(in, IN_F32, src0 + q * pstride, v1);
      load8(in, IN_F32, src0 + q * pstride + hd, v2);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        x1[e] += v1[e];
        x2[e] += v2[e];
      }
    }
    float y1[8], y2[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      if (ROT) {
        const float2 a = cs[tt * hd + i + e];
        y1[e] = x1[e] * a.x + x2[e] * a.y;
        y2[e] = x2[e] * a.x - x1[e] * a.y;
      } else {
        y1[e] = x1[e];
        y2[e] = x2[e];
      }
    }
    const int64_t dst = t * ldo + int64_t(h) * d + i;
    store8(out + dst, y1);
    store8(out + dst + hd, y2);
  }
}

// Head-major [nsum, H, T, d] (fp32 or bf16; head h at head_slot(h)) ->
// token-major bf16 [T, C] with rows ldo elements apart: the nsum stacked
// partials are summed (the gradient of a key/value head shared by a group),
// then rotated by minus the position's angle when ROT (the inverse rotation).
template <bool IN_F32, bool ROT>
__global__ __launch_bounds__(256) void rope_merge_kernel(int64_t T, int H, int d, int L, int perm, int nsum,
                                                         const void* __restrict__ in, uint16_t* __restrict__ out,
                                                         int64_t ldo) {
  const int hd = d >> 1;
  const int64_t n = T * H * hd;
  const int64_t idx = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= n) return;
  const int i = int(idx % hd);
  const int h = int((idx / hd) % H);
  const int64_t t = idx / (int64_t(hd) * H);
  const int64_t src0 = (int64_t(head_slot(h, H, perm)) * T + t) * d + i;
  const int64_t pstride = int64_t(H) * T * d;
  float x1 = 0.0f, x2 = 0.0f;
  for (int q = 0; q < nsum; ++q) {
    const int64_t src = src0 + q * pstride;
    if (IN_F32) {
      x1 += static_cast<const float*>(in)[src];
      x2 += static_cast<const float*>(in)[src + hd];
    } else {
      x1 += bf(static_cast<const uint16_t*>(in)[src]);
      x2 += bf(static_cast<const uint16_t*>(in)[src + hd]);
    }
  }
  float y1 = x1, y2 = x2;
  if (ROT) {
    float s, c;
    sincosf(rope_angle(int(t % L), i, d), &s, &c);
    y1 = x1 * c + x2 * s;
    y2 = x2 * c - x1 * s;
  }
  const int64_t dst = t * ldo + int64_t(h) * d + i;
  out[dst] = to_bf(y1);
  out[dst + hd] = to_bf(y2);
}

// One wavefront per score row i of one [L, L] block: P[i, j] = softmax over
// j <= i of S[i, j], 0 for j > i (bf16).  Rows of up to 2048 are held in
// registers (NPL = 32 values per lane, one read of S); longer rows take three
// passes over S.
template <int NPL>
__global__ __launch_bounds__(256) void softmax_causal_kernel(int64_t rows, int L, const float* __restrict__ S,
                                                             uint16_t* __restrict__ P) {
  const int lane = threadIdx.x & 63;
  const int64_t row = int64_t(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int i = int(row % L);
  const float* s = S + row * L;
  uint16_t* p = P + row * L;
  if constexpr (NPL > 0) {
    float v[NPL];
    float m = -INFINITY;
#pragma unroll
    for (int k = 0; k < NPL; ++k) {
      const int j = lane + 64 * k;
      v[k] = j <= i ? s[j] : -INFINITY;
      m = fmaxf(m, v[k]);
    }
    m = wave_max(m);
    float sum = 0.0f;
#pragma unroll
    for (int k = 0; k < NPL; ++k) {
      v[k] = lane + 64 * k <= i ? expf(v[k] - m) : 0.0f;
      sum += v[k];
    }
    sum = wave_sum(sum);
    const float inv = 1.0f / sum;
#pragma unroll
    for (int k = 0; k < NPL; ++k) {
      const int j = lane + 64 * k;
      if (j < L) p[j] = j <= i ? to_bf(v[k] * inv) : uint16_t(0);
    }
  } else {
    float m = -INFINITY;
    for (int j = lane; j <= i; j += 64) m = fmaxf(m, s[j]);
    m = wave_max(m);
    float sum = 0.0f;
    for (int j = lane; j <= i; j += 64) sum += expf(s[j] - m);
    sum = wave_sum(sum);
    const float inv = 1.0f / sum;
    for (int j = lane; j < L; j += 64) p[j] = j <= i ? to_bf(expf(s[j] - m) * inv) : uint16_t(0);
  }
}

// dS[i, j] = P[i, j] (dP[i, j] - sum_j' P[i, j'] dP[i, j']) (bf16), one
// wavefront per row; rows of up to 2048 in registers as in the forward.
template <int NPL>
__global__ __launch_bounds__(256) void softmax_bwd_kernel(int64_t rows, int L, const float* __restrict__ dP,
                                                          const uint16_t* __restrict__ P, uint16_t* __restrict__ dS) {
  const int lane = threadIdx.x & 63;
  const int64_t row = int64_t(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int i = int(row % L);
  const float* dp = dP + row * L;
  const uint16_t* p = P + row * L;
  if constexpr (NPL > 0) {
    float pv[NPL], dv[NPL];
    float dot = 0.0f;
#pragma unroll
    for (int k = 0; k < NPL; ++k) {
      const int j = lane + 64 * k;
      pv[k] = j <= i ? bf(p[j]) : 0.0f;
      dv[k] = j <= i ? dp[j] : 0.0f;
      dot += pv[k] * dv[k];
    }
    dot = wave_sum(dot);
#pragma unroll
    for (int k = 0; k < NPL; ++k) {
      const int j = lane + 64 * k;
      if (j < L) dS[row * L + j] = j <= i ? to_bf(pv[k] * (dv[k] - dot)) : uint16_t(0);
    }
  } else {
    float dot = 0.0f;
    for (int j = lane; j <= i; j += 64) dot += bf(p[j]) * dp[j];
    dot = wave_sum(dot);
    for (int j = lane; j < L; j += 64) dS[row * L + j] = j <= i ? to_bf(bf(p[j]) * (dp[j] - dot)) : uint16_t(0);
  }
}

// out[b] = in[b]^T for B matrices [R, C] (bf16): 64 x 64 tiles through LDS,
// 8-byte accesses on both sides (four columns per lane and access).
__global__ __launch_bounds__(256) void transpose_batched_kernel(int64_t R, int64_t C, const uint16_t* __restrict__ in,
                                                                uint16_t* __restrict__ out) {
  __shared__ uint16_t tile[64][68];
  const int64_t tiles_c = (C + 63) / 64;
  const int64_t r0 = (int64_t(blockIdx.x) / tiles_c) * 64, c0 = (int64_t(blockIdx.x) % tiles_c) * 64;
  const int64_t boff = int64_t(blockIdx.y) * R * C;
  const int q = threadIdx.x & 15, y0 = threadIdx.x >> 4;  // column group, first row
  const bool vec = (C % 4 == 0) && (R % 4 == 0);
  for (int y = y0; y < 64; y += 16) {
    const int64_t r = r0 + y, c = c0 + 4 * q;
    if (vec && r < R && c + 3 < C) {
      const uint2 v = *reinterpret_cast<const uint2*>(in + boff + r * C + c);
      tile[y][4 * q] = uint16_t(v.x & 0xFFFFu);
      tile[y][4 * q + 1] = uint16_t(v.x >> 16);
      tile[y][4 * q + 2] = uint16_t(v.y & 0xFFFFu);
      tile[y][4 * q + 3] = uint16_t(v.y >> 16);
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) tile[y][4 * q + e] = (r < R && c + e < C) ? in[boff + r * C + c + e] : uint16_t(0);
    }
  }
  __syncthreads();
  for (int y = y0; y < 64; y += 16) {
    const int64_t c = c0 + y, r = r0 + 4 * q;  // output row c, columns r .. r+3
    if (c >= C) continue;
    if (vec && r + 3 < R) {
      const uint2 v = make_uint2(uint32_t(tile[4 * q][y]) | (uint32_t(tile[4 * q + 1][y]) << 16),
                                 uint32_t(tile[4 * q + 2][y]) | (uint32_t(tile[4 * q + 3][y]) << 16));
      *reinterpret_cast<uint2*>(out + boff + c * R + r) = v;
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (r + e < R) out[boff + c * R + r + e] = tile[4 * q + e][y];
    }
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
  const dim3 g(unsigned((T + 3) / 4));
  switch (C % 256 == 0 ? C / 256 : 0) {
    case 16: hipLaunchKernelGGL(add_rmsnorm_rows_kernel<16>, g, dim3(256), 0, st, T, C, X, A, gamma, R, Z, rinv); break;
    case 8: hipLaunchKernelGGL(add_rmsnorm_rows_kernel<8>, g, dim3(256), 0, st, T, C, X, A, gamma, R, Z, rinv); break;
    case 4: hipLaunchKernelGGL(add_rmsnorm_rows_kernel<4>, g, dim3(256), 0, st, T, C, X, A, gamma, R, Z, rinv); break;
    default: hipLaunchKernelGGL(add_rmsnorm_kernel, g, dim3(256), 0, st, T, C, X, A, gamma, R, Z, rinv); break;
  }
  return hipGetLastError();
}

hipError_t launch_rmsnorm_bwd(int64_t T, int64_t C, const float* dZa, const float* dZb, const float* X,
                              const float* gamma, const float* rinv, const uint16_t* E, float escale, uint16_t* dR,
                              float* dRf, hipStream_t st) {
  const dim3 g(unsigned((T + 3) / 4));
  switch (C % 256 == 0 ? C / 256 : 0) {
    case 16:
      hipLaunchKernelGGL(rmsnorm_bwd_rows_kernel<16>, g, dim3(256), 0, st, T, C, dZa, dZb, X, gamma, rinv, E, escale,
                         dR, dRf);
      break;
    case 8:
      hipLaunchKernelGGL(rmsnorm_bwd_rows_kernel<8>, g, dim3(256), 0, st, T, C, dZa, dZb, X, gamma, rinv, E, escale,
                         dR, dRf);
      break;
    case 4:
      hipLaunchKernelGGL(rmsnorm_bwd_rows_kernel<4>, g, dim3(256), 0, st, T, C, dZa, dZb, X, gamma, rinv, E, escale,
                         dR, dRf);
      break;
    default:
      hipLaunchKernelGGL(rmsnorm_bwd_kernel, g, dim3(256), 0, st, T, C, dZa, dZb, X, gamma, rinv, E, escale, dR, dRf);
      break;
  }
  return hipGetLastError();
}

static bool rope_vec_ok(int d, const void* in, const void* out) {
  return d % 16 == 0 && d / 2 <= RT_MAX_HD && (reinterpret_cast<uintptr_t>(in) & 15) == 0 &&
         (reinterpret_cast<uintptr_t>(out) & 15) == 0;
}

hipError_t launch_rope_table(int L, int d, float* cs, hipStream_t st) {
  const int64_t n = int64_t(L) * (d / 2);
  hipLaunchKernelGGL(rope_table_kernel, dim3(unsigned((n + 255) / 256)), dim3(256), 0, st, L, d, cs);
  return hipGetLastError();
}

hipError_t launch_rope_split(int64_t T, int H, int d, int L, int perm, const void* in, int in_f32, int rotate,
                             uint16_t* out, hipStream_t st) {
  if (rope_vec_ok(d, in, out)) {
    const dim3 grid(unsigned((T + RT - 1) / RT));
    if (in_f32 && rotate)
      hipLaunchKernelGGL((rope_split_vec_kernel<true, true>), grid, dim3(256), 0, st, T, H, d, L, perm, in, out);
    else if (in_f32)
      hipLaunchKernelGGL((rope_split_vec_kernel<true, false>), grid, dim3(256), 0, st, T, H, d, L, perm, in, out);
    else if (rotate)
      hipLaunchKernelGGL((rope_split_vec_kernel<false, true>), grid, dim3(256), 0, st, T, H, d, L, perm, in, out);
    else hipLaunchKernelGGL((rope_split_vec_kernel<false, false>), grid, dim3(256), 0, st, T, H, d, L, perm, in, out);
    return hipGetLastError();
  }
  const dim3 grid(unsigned((T * H * (d / 2) + 255) / 256));
  if (in_f32 && rotate)
    hipLaunchKernelGGL((rope_split_kernel<true, true>), grid, dim3(256), 0, st, T, H, d, L, perm, in, out);
  else if (in_f32)
    hipLaunchKernelGGL((rope_split_kernel<true, false>), grid, dim3(256), 0, st, T, H, d, L, perm, in, out);
  else if (rotate)
    hipLaunchKernelGGL((rope_split_kernel<false, true>), grid, dim3(256), 0, st, T, H, d, L, perm, in, out);
  else hipLaunchKernelGGL((rope_split_kernel<false, false>), grid, dim3(256), 0, st, T, H, d, L, perm, in, out);
  return hipGetLastError();
}

hipError_t launch_rope_merge(int64_t T, int H, int d, int L, int perm, int nsum, const void* in, int in_f32,
                             int rotate, uint16_t* out, int64_t ldo, hipStream_t st) {
  if (ldo == 0) ldo = int64_t(H) * d;
  if (rope_vec_ok(d, in, out) && ldo % 8 == 0) {
    const dim3 grid(unsigned((T + RT - 1) / RT));
    if (in_f32 && rotate)
      hipLaunchKernelGGL((rope_merge_vec_kernel<true, true>), grid, dim3(256), 0, st, T, H, d, L, perm, nsum, in, out,
                         ldo);
    else if (in_f32)
      hipLaunchKernelGGL((rope_merge_vec_kernel<true, false>), grid, dim3(256), 0, st, T, H, d, L, perm, nsum, in,
                         out, ldo);
    else if (rotate)
      hipLaunchKernelGGL((rope_merge_vec_kernel<false, true>), grid, dim3(256), 0, st, T, H, d, L, perm, nsum, in,
                         out, ldo);
    else
      hipLaunchKernelGGL((rope_merge_vec_kernel<false, false>), grid, dim3(256), 0, st, T, H, d, L, perm, nsum, in,
                         out, ldo);
    return hipGetLastError();
  }
  const dim3 grid(unsigned((T * H * (d / 2) + 255) / 256));
  if (in_f32 && rotate)
    hipLaunchKernelGGL((rope_merge_kernel<true, true>), grid, dim3(256), 0, st, T, H, d, L, perm, nsum, in, out, ldo);
  else if (in_f32)
    hipLaunchKernelGGL((rope_merge_kernel<true, false>), grid, dim3(256), 0, st, T, H, d, L, perm, nsum, in, out, ldo);
  else if (rotate)
    hipLaunchKernelGGL((rope_merge_kernel<false, true>), grid, dim3(256), 0, st, T, H, d, L, perm, nsum, in, out, ldo);
  else
    hipLaunchKernelGGL((rope_merge_kernel<false, false>), grid, dim3(256), 0, st, T, H, d, L, perm, nsum, in, out,
                       ldo);
  return hipGetLastError();
}

hipError_t launch_softmax_causal(int64_t rows, int L, const float* S, uint16_t* P, hipStream_t st) {
  const dim3 grid(unsigned((rows + 3) / 4));
  if (L <= 2048) hipLaunchKernelGGL(softmax_causal_kernel<32>, grid, dim3(256), 0, st, rows, L, S, P);
  else hipLaunchKernelGGL(softmax_causal_kernel<0>, grid, dim3(256), 0, st, rows, L, S, P);
  return hipGetLastError();
}

hipError_t launch_softmax_bwd(int64_t rows, int L, const float* dP, const uint16_t* P, uint16_t* dS, hipStream_t st) {
  const dim3 grid(unsigned((rows + 3) / 4));
  if (L <= 2048) hipLaunchKernelGGL(softmax_bwd_kernel<32>, grid, dim3(256), 0, st, rows, L, dP, P, dS);
  else hipLaunchKernelGGL(softmax_bwd_kernel<0>, grid, dim3(256), 0, st, rows, L, dP, P, dS);
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
