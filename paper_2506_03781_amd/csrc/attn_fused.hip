// Causal attention of the block-level reconstruction (Algorithm 1 with a
// Transformer block; appendix "Units in LLMs") with the score tiles kept on
// chip: no [L, L] score, probability or gradient array is written.
//
// Per sequence and query head b (key/value head b mod kv_batch), d = 128:
//   S = Q K^T * scale (fp32), P = bf16(softmax over keys j <= i of S),
//   O = bf16(P V) (fp32 accumulation);
//   backward with dP = dO V^T (fp32), delta_i = dO_i . O_i (fp32, from the
//   stored bf16 O and dO; equal to sum_j P_ij dP_ij in exact arithmetic),
//   dS = bf16(P (dP - delta)), dQ = dS K * scale, dK = dS^T Q * scale,
//   dV = P^T dO (fp32 out; the key/value gradients summed over the query heads
//   that share the head, in head order).
// These are the rounding points of the unfused path (P and dS stored in
// bf16, S and dP in fp32).  The forward runs two passes over the keys: the
// first finds each row's maximum m and sum l of exp(S - m), the second forms
// P = exp(S - m) / l exactly as the row softmax does and accumulates P V; m
// and l are kept so that the backward recomputes the same P bit for bit.
//
// MFMA layout (v_mfma_f32_32x32x16_bf16, C[m][n] += A[m][k] B[n][k]): lane l
// supplies row l % 32 of A and of B with k = 8 (l / 32) .. + 8, and holds
// C rows 8 (r / 4) + 4 (l / 32) + r % 4, r < 16, of column l % 32.  A score
// tile is computed transposed (keys as rows) where its columns must be
// queries, so a lane's 16 accumulator values are one query's scores for 16
// keys; those values then serve directly as the B operand of the next
// product, with the keys (its k dimension) in the permuted order
// kperm(i) = {0, 1, 2, 3, 8, 9, 10, 11}[i] (+4 in the upper half-wave), and
// the A operand of that product is read with the same permutation.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "uq_launch.h"

namespace uq {

namespace {

typedef __bf16 bf16x8a __attribute__((ext_vector_type(8)));
typedef float f32x16a __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4a __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2a __attribute__((ext_vector_type(2)));

constexpr int D = 128;      // head dimension
constexpr int NB = 32;      // keys (or queries) per tile

__device__ __forceinline__ f32x16a mfma(const bf16x8a& a, const bf16x8a& b, const f32x16a& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ uint32_t bf16_bits(float x) {  // round to nearest even
  const uint32_t u = __float_as_uint(x);
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ float bf16_round(float x) { return __uint_as_float(bf16_bits(x) << 16); }

// Row of the accumulator held in slot r by lane l.
__device__ __forceinline__ int acc_row(int r, int lane) { return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3); }

// Row-major tile [32 rows][128] bf16 in LDS: 16-byte chunk c of row r at
// r * 16 + (c ^ (r & 15)), so the 32 rows a fragment read touches at one
// chunk fall in distinct bank groups.
struct RowTile {
  u32x4a* p;
  __device__ __forceinline__ void load(const uint16_t* __restrict__ src, int64_t ld, int row0, int rows_valid) {
    // 512 chunks: two per lane of the workgroup
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int t = threadIdx.x + h * 256;
      const int r = t >> 4, c = t & 15;
      u32x4a v = {0u, 0u, 0u, 0u};
      if (r < rows_valid) v = *reinterpret_cast<const u32x4a*>(src + int64_t(row0 + r) * ld + c * 8);
      p[r * 16 + (c ^ (r & 15))] = v;
    }
  }
  // A or B fragment of k-step j for this lane: row (lane % 32), d = 16 j + 8 (lane / 32)
  __device__ __forceinline__ bf16x8a frag(int j, int lane) const {
    const int r = lane & 31, c = 2 * j + (lane >> 5);
    return __builtin_bit_cast(bf16x8a, p[r * 16 + (c ^ (r & 15))]);
  }
};

// Transposed tile [128 rows (d)][32 columns] bf16 in LDS from a [d][L]
// source: 8-byte unit u of row d at d * 8 + (u ^ ((d >> 2) & 7)).
struct ColTile {
  u32x2a* p;
  __device__ __forceinline__ void load(const uint16_t* __restrict__ src, int64_t ld, int col0) {
    // 128 rows x 4 pieces of 16 B: two per lane
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int t = threadIdx.x + h * 256;
      const int d = t >> 2, q = t & 3;
      const u32x4a v = *reinterpret_cast<const u32x4a*>(src + int64_t(d) * ld + col0 + q * 8);
      const int sw = (d >> 2) & 7;
      p[d * 8 + ((2 * q) ^ sw)] = u32x2a{v.x, v.y};
      p[d * 8 + ((2 * q + 1) ^ sw)] = u32x2a{v.z, v.w};
    }
  }
  // A fragment for the product over the tile's 32 columns, half h (16
  // columns), rows 32 db .. + 32: lane supplies row 32 db + lane % 32 and the
  // columns kperm: 16 h + 4 (lane / 32) + {0..3} and + 8 + {0..3}.
  __device__ __forceinline__ bf16x8a frag(int db, int h, int lane) const {
    const int d = 32 * db + (lane & 31);
    const int sw = (d >> 2) & 7;
    const int u1 = 4 * h + (lane >> 5), u2 = u1 + 2;
    const u32x2a a = p[d * 8 + (u1 ^ sw)], b = p[d * 8 + (u2 ^ sw)];
    return __builtin_bit_cast(bf16x8a, u32x4a{a.x, a.y, b.x, b.y});
  }
};

// The 8 accumulator values of half h (slots 8 h .. 8 h + 7) as a bf16 B
// operand (values already rounded or to be rounded here).
__device__ __forceinline__ bf16x8a pack_half(const float (&v)[16], int h) {
  u32x4a w;
#pragma unroll
  for (int i = 0; i < 4; ++i)
    w[i] = bf16_bits(v[8 * h + 2 * i]) | (bf16_bits(v[8 * h + 2 * i + 1]) << 16);
  return __builtin_bit_cast(bf16x8a, w);
}

__device__ __forceinline__ f32x16a zero16() {
  f32x16a z;
#pragma unroll
  for (int r = 0; r < 16; ++r) z[r] = 0.0f;
  return z;
}

}  // namespace

struct AttnArgs {
  int64_t batch, kv_batch;
  int L;
  float scale;
  const uint16_t* Q;    // [batch, L, D]
  const uint16_t* Qt;   // [batch, D, L]
  const uint16_t* K;    // [kv_batch, L, D]
  const uint16_t* Kt;   // [kv_batch, D, L]
  const uint16_t* V;    // [kv_batch, L, D]
  const uint16_t* Vt;   // [kv_batch, D, L]
  const uint16_t* O;    // [batch, L, D]
  const uint16_t* dO;   // [batch, L, D]
  const uint16_t* dOt;  // [batch, D, L]
  uint16_t* O_out;      // [batch, L, D]
  float* m;             // [batch, L] row maximum of S
  float* l;             // [batch, L] row sum of exp(S - m)
  float* delta;         // [batch, L]
  float* dQ;            // [batch, L, D]
  float* dK;            // [kv_batch, L, D]
  float* dV;            // [kv_batch, L, D]
};

// Forward: one workgroup per (128 queries, query batch); wave w owns queries
// q0 = 128 blockIdx.x + 32 w .. + 32 and loops over the key tiles up to its
// diagonal (the workgroup's tiles are loaded cooperatively).
__global__ __launch_bounds__(256) void attn_fwd_kernel(AttnArgs a) {
  __shared__ u32x4a sK[NB * 16];
  __shared__ u32x2a sVt[D * 8];
  RowTile tK{sK};
  ColTile tV{sVt};
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t b = blockIdx.y, bk = b % a.kv_batch;
  const int L = a.L;
  const int q0 = blockIdx.x * 128 + wave * NB;
  const bool active = q0 < L;
  const int qi = q0 + (lane & 31);  // this lane's query
  const int n_tiles = min(L, int(blockIdx.x) * 128 + 128) / NB;  // key tiles the workgroup needs
  const int my_tiles = active ? q0 / NB + 1 : 0;
  const uint16_t* Kb = a.K + bk * int64_t(L) * D;
  const uint16_t* Vtb = a.Vt + bk * int64_t(D) * L;
  // this lane's query row as B fragments
  bf16x8a qf[8];
  {
    const uint16_t* qrow = a.Q + (b * L + min(qi, L - 1)) * int64_t(D) + 8 * (lane >> 5);
#pragma unroll
    for (int j = 0; j < 8; ++j) qf[j] = __builtin_bit_cast(bf16x8a, *reinterpret_cast<const u32x4a*>(qrow + 16 * j));
  }
  // pass 1: row maximum and sum (per half-wave: 16 of each tile's 32 keys)
  float m = -INFINITY, l = 0.0f;
  for (int t = 0; t < n_tiles; ++t) {
    __syncthreads();
    tK.load(Kb, D, t * NB, NB);
    __syncthreads();
    if (t >= my_tiles) continue;
    f32x16a s = zero16();
#pragma unroll
    for (int j = 0; j < 8; ++j) s = mfma(tK.frag(j, lane), qf[j], s);
    float mt = m;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int key = t * NB + acc_row(r, lane);
      if (key <= qi) mt = fmaxf(mt, s[r] * a.scale);
    }
    float sum = 0.0f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int key = t * NB + acc_row(r, lane);
      if (key <= qi) sum += expf(s[r] * a.scale - mt);
    }
    l = (m == -INFINITY ? 0.0f : l * expf(m - mt)) + sum;
    m = mt;
  }
  // combine the two half-waves of each query (fixed order: lower half first)
  {
    const float m2 = __shfl_xor(m, 32, 64), l2 = __shfl_xor(l, 32, 64);
    const float mlo = (lane < 32) ? m : m2, llo = (lane < 32) ? l : l2;
    const float mhi = (lane < 32) ? m2 : m, lhi = (lane < 32) ? l2 : l;
    const float mm = fmaxf(mlo, mhi);
    const float a0 = mlo == -INFINITY ? 0.0f : llo * expf(mlo - mm);
    const float a1 = mhi == -INFINITY ? 0.0f : lhi * expf(mhi - mm);
    m = mm;
    l = a0 + a1;
  }
  const float inv = 1.0f / l;
  // pass 2: P = bf16(exp(S - m) / l), O += P V
  f32x16a o[4] = {zero16(), zero16(), zero16(), zero16()};
  for (int t = 0; t < n_tiles; ++t) {
    __syncthreads();
    tK.load(Kb, D, t * NB, NB);
    tV.load(Vtb, L, t * NB);
    __syncthreads();
    if (t >= my_tiles) continue;
    f32x16a s = zero16();
#pragma unroll
    for (int j = 0; j < 8; ++j) s = mfma(tK.frag(j, lane), qf[j], s);
    float p[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int key = t * NB + acc_row(r, lane);
      p[r] = key <= qi ? expf(s[r] * a.scale - m) * inv : 0.0f;
    }
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const bf16x8a pb = pack_half(p, h);
#pragma unroll
      for (int db = 0; db < 4; ++db) o[db] = mfma(tV.frag(db, h, lane), pb, o[db]);
    }
  }
  if (!active || qi >= L) return;
  uint16_t* orow = a.O_out + (b * L + qi) * int64_t(D);
#pragma unroll
  for (int db = 0; db < 4; ++db)
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
      const int d0 = 32 * db + 8 * g4 + 4 * (lane >> 5);
      const uint32_t w0 = bf16_bits(o[db][4 * g4]) | (bf16_bits(o[db][4 * g4 + 1]) << 16);
      const uint32_t w1 = bf16_bits(o[db][4 * g4 + 2]) | (bf16_bits(o[db][4 * g4 + 3]) << 16);
      *reinterpret_cast<u32x2a*>(orow + d0) = u32x2a{w0, w1};
    }
  if (lane < 32) {
    a.m[b * L + qi] = m;
    a.l[b * L + qi] = l;
  }
}

// Backward for the queries: delta = dO . O per row (written for the key
// kernel), then per key tile S -> P (the forward's m, l), dP = dO V^T,
// dS = bf16(P (dP - delta)), dQ += dS K; dQ * scale stored in fp32.
__global__ __launch_bounds__(256) void attn_bwd_dq_kernel(AttnArgs a) {
  __shared__ u32x4a sK[NB * 16];
  __shared__ u32x4a sV[NB * 16];
  __shared__ u32x2a sKt[D * 8];
  RowTile tK{sK}, tV{sV};
  ColTile tKt{sKt};
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t b = blockIdx.y, bk = b % a.kv_batch;
  const int L = a.L;
  const int q0 = blockIdx.x * 128 + wave * NB;
  const bool active = q0 < L;
  const int qi = q0 + (lane & 31);
  const int qc = min(qi, L - 1);
  const int n_tiles = min(L, int(blockIdx.x) * 128 + 128) / NB;
  const int my_tiles = active ? q0 / NB + 1 : 0;
  const uint16_t* Kb = a.K + bk * int64_t(L) * D;
  const uint16_t* Vb = a.V + bk * int64_t(L) * D;
  const uint16_t* Ktb = a.Kt + bk * int64_t(D) * L;
  bf16x8a qf[8], df[8];
  float dl = 0.0f;
  {
    const int64_t row = (b * L + qc) * int64_t(D) + 8 * (lane >> 5);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      qf[j] = __builtin_bit_cast(bf16x8a, *reinterpret_cast<const u32x4a*>(a.Q + row + 16 * j));
      df[j] = __builtin_bit_cast(bf16x8a, *reinterpret_cast<const u32x4a*>(a.dO + row + 16 * j));
      const bf16x8a ov = __builtin_bit_cast(bf16x8a, *reinterpret_cast<const u32x4a*>(a.O + row + 16 * j));
#pragma unroll
      for (int i = 0; i < 8; ++i) dl += float(df[j][i]) * float(ov[i]);
    }
  }
  // delta: this lane's 64 d values, then the other half-wave's (lower half first)
  {
    const float d2 = __shfl_xor(dl, 32, 64);
    dl = lane < 32 ? dl + d2 : d2 + dl;
  }
  const float mq = a.m[b * L + qc];
  const float inv = 1.0f / a.l[b * L + qc];
  if (active && lane < 32 && qi < L) a.delta[b * L + qi] = dl;
  f32x16a dq[4] = {zero16(), zero16(), zero16(), zero16()};
  for (int t = 0; t < n_tiles; ++t) {
    __syncthreads();
    tK.load(Kb, D, t * NB, NB);
    tV.load(Vb, D, t * NB, NB);
    tKt.load(Ktb, L, t * NB);
    __syncthreads();
    if (t >= my_tiles) continue;
    f32x16a s = zero16(), dp = zero16();
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      s = mfma(tK.frag(j, lane), qf[j], s);
      dp = mfma(tV.frag(j, lane), df[j], dp);
    }
    float ds[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int key = t * NB + acc_row(r, lane);
      const float p = key <= qi ? bf16_round(expf(s[r] * a.scale - mq) * inv) : 0.0f;
      ds[r] = p * (dp[r] - dl);
    }
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const bf16x8a sb = pack_half(ds, h);
#pragma unroll
      for (int db = 0; db < 4; ++db) dq[db] = mfma(tKt.frag(db, h, lane), sb, dq[db]);
    }
  }
  if (!active || qi >= L) return;
  float* out = a.dQ + (b * L + qi) * int64_t(D);
#pragma unroll
  for (int db = 0; db < 4; ++db)
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
      const int d0 = 32 * db + 8 * g4 + 4 * (lane >> 5);
      *reinterpret_cast<float4*>(out + d0) = make_float4(dq[db][4 * g4] * a.scale, dq[db][4 * g4 + 1] * a.scale,
                                                         dq[db][4 * g4 + 2] * a.scale, dq[db][4 * g4 + 3] * a.scale);
    }
}

// Backward for the keys and values: one workgroup per (128 keys, key/value
// batch); wave w owns keys k0 = 128 blockIdx.x + 32 w .. + 32 and loops over
// the query heads that share the key/value head (in head order) and over the
// query tiles from its diagonal on.  S = Q K^T and dP = dO V^T have queries
// as rows and this lane's key as column, so P and dS feed dV += P^T dO and
// dK += dS^T Q directly.
__global__ __launch_bounds__(256) void attn_bwd_dkv_kernel(AttnArgs a) {
  __shared__ u32x4a sQ[NB * 16];
  __shared__ u32x4a sdO[NB * 16];
  __shared__ u32x2a sQt[D * 8];
  __shared__ u32x2a sdOt[D * 8];
  __shared__ float sm[NB], sinv[NB], sdl[NB];
  RowTile tQ{sQ}, tdO{sdO};
  ColTile tQt{sQt}, tdOt{sdOt};
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t bk = blockIdx.y;
  const int L = a.L;
  const int k0 = blockIdx.x * 128 + wave * NB;
  const bool active = k0 < L;
  const int kj = k0 + (lane & 31);  // this lane's key
  const int kc = min(kj, L - 1);
  const int first_tile = int(blockIdx.x) * 128 / NB;  // query tiles the workgroup needs
  const int my_first = active ? k0 / NB : L / NB;
  const int groups = int(a.batch / a.kv_batch);
  bf16x8a kf[8], vf[8];
  {
    const int64_t row = (bk * L + kc) * int64_t(D) + 8 * (lane >> 5);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      kf[j] = __builtin_bit_cast(bf16x8a, *reinterpret_cast<const u32x4a*>(a.K + row + 16 * j));
      vf[j] = __builtin_bit_cast(bf16x8a, *reinterpret_cast<const u32x4a*>(a.V + row + 16 * j));
    }
  }
  f32x16a dk[4] = {zero16(), zero16(), zero16(), zero16()};
  f32x16a dv[4] = {zero16(), zero16(), zero16(), zero16()};
  for (int g = 0; g < groups; ++g) {
    const int64_t b = int64_t(g) * a.kv_batch + bk;  // query batch of head position g
    const uint16_t* Qb = a.Q + b * int64_t(L) * D;
    const uint16_t* dOb = a.dO + b * int64_t(L) * D;
    const uint16_t* Qtb = a.Qt + b * int64_t(D) * L;
    const uint16_t* dOtb = a.dOt + b * int64_t(D) * L;
    for (int t = first_tile; t < L / NB; ++t) {
      __syncthreads();
      tQ.load(Qb, D, t * NB, NB);
      tdO.load(dOb, D, t * NB, NB);
      tQt.load(Qtb, L, t * NB);
      tdOt.load(dOtb, L, t * NB);
      if (threadIdx.x < NB) {
        const int64_t i = b * L + t * NB + threadIdx.x;
        sm[threadIdx.x] = a.m[i];
        sinv[threadIdx.x] = 1.0f / a.l[i];
        sdl[threadIdx.x] = a.delta[i];
      }
      __syncthreads();
      if (t < my_first) continue;
      f32x16a s = zero16(), dp = zero16();
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        s = mfma(tQ.frag(j, lane), kf[j], s);
        dp = mfma(tdO.frag(j, lane), vf[j], dp);
      }
      float p[16], ds[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int qr = acc_row(r, lane);
        const int qi = t * NB + qr;
        const float pv = kj <= qi ? bf16_round(expf(s[r] * a.scale - sm[qr]) * sinv[qr]) : 0.0f;
        p[r] = pv;
        ds[r] = pv * (dp[r] - sdl[qr]);
      }
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const bf16x8a pb = pack_half(p, h), sb = pack_half(ds, h);
#pragma unroll
        for (int db = 0; db < 4; ++db) {
          dv[db] = mfma(tdOt.frag(db, h, lane), pb, dv[db]);
          dk[db] = mfma(tQt.frag(db, h, lane), sb, dk[db]);
        }
      }
    }
  }
  if (!active || kj >= L) return;
  float* ko = a.dK + (bk * L + kj) * int64_t(D);
  float* vo = a.dV + (bk * L + kj) * int64_t(D);
#pragma unroll
  for (int db = 0; db < 4; ++db)
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
      const int d0 = 32 * db + 8 * g4 + 4 * (lane >> 5);
      *reinterpret_cast<float4*>(ko + d0) = make_float4(dk[db][4 * g4] * a.scale, dk[db][4 * g4 + 1] * a.scale,
                                                        dk[db][4 * g4 + 2] * a.scale, dk[db][4 * g4 + 3] * a.scale);
      *reinterpret_cast<float4*>(vo + d0) =
          make_float4(dv[db][4 * g4], dv[db][4 * g4 + 1], dv[db][4 * g4 + 2], dv[db][4 * g4 + 3]);
    }
}

hipError_t launch_attn_fwd(const AttnLaunch& q, hipStream_t st) {
  AttnArgs a{};
  a.batch = q.batch; a.kv_batch = q.kv_batch; a.L = q.L; a.scale = q.scale;
  a.Q = q.Q; a.K = q.K; a.Vt = q.Vt; a.O_out = q.O_out; a.m = q.m; a.l = q.l;
  const dim3 grid(unsigned((q.L + 127) / 128), unsigned(q.batch));
  hipLaunchKernelGGL(attn_fwd_kernel, grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_attn_bwd(const AttnLaunch& q, hipStream_t st) {
  AttnArgs a{};
  a.batch = q.batch; a.kv_batch = q.kv_batch; a.L = q.L; a.scale = q.scale;
  a.Q = q.Q; a.Qt = q.Qt; a.K = q.K; a.Kt = q.Kt; a.V = q.V; a.O = q.O; a.dO = q.dO; a.dOt = q.dOt;
  a.m = q.m; a.l = q.l; a.delta = q.delta; a.dQ = q.dQ; a.dK = q.dK; a.dV = q.dV;
  const dim3 gq(unsigned((q.L + 127) / 128), unsigned(q.batch));
  hipLaunchKernelGGL(attn_bwd_dq_kernel, gq, dim3(256), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const dim3 gk(unsigned((q.L + 127) / 128), unsigned(q.kv_batch));
  hipLaunchKernelGGL(attn_bwd_dkv_kernel, gk, dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace uq
