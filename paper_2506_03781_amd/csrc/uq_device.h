// Device helpers shared by the quantizer kernels (forward, fold, dequant,
// init): storage conversions, vector loads of 8 consecutive weights, the
// per-group binary-coding level table kept in LDS and the nearest-level
// searches.  gfx950 only.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace uq {

constexpr int kThreads = 256;           // threads per quantizer workgroup
constexpr int kVec = 8;                 // consecutive weights per lane
constexpr int kTile = kThreads * kVec;  // weights per full tile
constexpr int kMaxEntries = 2048;       // level-table entries per tile (LDS)

enum DType : int { F32 = 0, BF16 = 1 };

__device__ __forceinline__ float bf16_to_f32(uint32_t h16) { return __uint_as_float(h16 << 16); }

// Two fp32 values -> packed bf16 pair (lo in bits 0..15), round to nearest
// even: one v_cvt_pk_bf16_f32 on gfx950.
typedef __bf16 uq_bf16x2 __attribute__((ext_vector_type(2)));
typedef float uq_f32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const uq_f32x2 f = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, uq_bf16x2));
}

// 8 consecutive weights starting at element `off` (16-byte aligned).
template <int DT>
__device__ __forceinline__ void load8(const void* base, int64_t off, float (&v)[8]) {
  if constexpr (DT == BF16) {
    const uint4 q = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(base) + off);
    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = __uint_as_float(w[i] << 16);
      v[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
  } else {
    const float4* p = reinterpret_cast<const float4*>(static_cast<const float*>(base) + off);
    const float4 a = p[0], b = p[1];
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
  }
}

__device__ __forceinline__ void load8f(const float* base, int64_t off, float (&v)[8]) {
  load8<F32>(base, off, v);
}

template <int DT>
__device__ __forceinline__ void store8(void* base, int64_t off, const float (&v)[8]) {
  if constexpr (DT == BF16) {
    uint4 q;
    q.x = pack_bf16x2(v[0], v[1]);
    q.y = pack_bf16x2(v[2], v[3]);
    q.z = pack_bf16x2(v[4], v[5]);
    q.w = pack_bf16x2(v[6], v[7]);
    *reinterpret_cast<uint4*>(static_cast<uint16_t*>(base) + off) = q;
  } else {
    float4* p = reinterpret_cast<float4*>(static_cast<float*>(base) + off);
    p[0] = make_float4(v[0], v[1], v[2], v[3]);
    p[1] = make_float4(v[4], v[5], v[6], v[7]);
  }
}

__device__ __forceinline__ void store8f(float* base, int64_t off, const float (&v)[8]) {
  store8<F32>(base, off, v);
}

__device__ __forceinline__ uint2 load8u8(const uint8_t* base, int64_t off) {
  return *reinterpret_cast<const uint2*>(base + off);
}

__device__ __forceinline__ void store8u8(uint8_t* base, int64_t off, uint2 v) {
  *reinterpret_cast<uint2*>(base + off) = v;
}

__device__ __forceinline__ uint32_t byte_of(uint2 v, int i) {
  return ((i < 4 ? v.x : v.y) >> (8 * (i & 3))) & 0xFFu;
}

// Level b of a group: z_B + (+-alpha_1) + ... + (+-alpha_k), fp32, left to
// right; the sign of alpha_{i+1} is + iff bit i of b is set.
__device__ __forceinline__ float level_value(const float* __restrict__ alpha_g, float zb, int k, int b) {
  float q = zb;
  for (int i = 0; i < k; ++i) {
    const float a = alpha_g[i];
    q = ((b >> i) & 1) ? q + a : q - a;
  }
  return q;
}

// Per-tile level tables in LDS.  A tile covers `ng` consecutive groups; the
// table of group gl occupies entries [gl*L, (gl+1)*L) of each array.
struct LevelTables {
  float* raw;         // q(b), unsorted
  float* qs;          // sorted ascending
  uint8_t* code_of;   // code at sorted position
  uint8_t* pos_of;    // sorted position of code
};

// Carve the tables for `entries` levels out of dynamic LDS starting at p;
// returns the first byte after them (16-byte aligned).
__device__ __forceinline__ char* carve_tables(LevelTables& t, char* p, int entries) {
  t.raw = reinterpret_cast<float*>(p);
  t.qs = t.raw + entries;
  t.code_of = reinterpret_cast<uint8_t*>(t.qs + entries);
  t.pos_of = t.code_of + entries;
  return p + ((size_t(entries) * 10 + 15) & ~size_t(15));
}

// Rank every raw level of the tile's groups (sort key (value, code)) and
// scatter into the sorted arrays.  Callers have filled t.raw and issued a
// barrier; ends with a barrier.
__device__ __forceinline__ void sort_tables(LevelTables& t, int ng, int logL) {
  const int L = 1 << logL;
  const int n = ng << logL;
  for (int e = threadIdx.x; e < n; e += blockDim.x) {
    const int gl = e >> logL;
    const int b = e & (L - 1);
    const float* row = t.raw + (gl << logL);
    const float q = row[b];
    int rank = 0;
    for (int b2 = 0; b2 < L; ++b2) {
      const float q2 = row[b2];
      rank += (q2 < q) | ((q2 == q) & (b2 < b));
    }
    t.qs[(gl << logL) + rank] = q;
    t.code_of[(gl << logL) + rank] = uint8_t(b);
    t.pos_of[(gl << logL) + b] = uint8_t(rank);
  }
  __syncthreads();
}

// Build the sorted tables of groups gid0 .. gid0+ng-1 from alpha and z_b.
// All threads of the block take part; ends with a block barrier.
__device__ __forceinline__ void build_tables(LevelTables& t, const float* __restrict__ alpha,
                                             const float* __restrict__ z_b, int64_t gid0, int ng,
                                             int k, int logL) {
  const int L = 1 << logL;
  const int n = ng << logL;
  for (int e = threadIdx.x; e < n; e += blockDim.x) {
    const int gl = e >> logL;
    const int b = e & (L - 1);
    const int64_t gid = gid0 + gl;
    t.raw[e] = level_value(alpha + gid * k, z_b[gid], k, b);
  }
  __syncthreads();
  sort_tables(t, ng, logL);
}

// Nearest sorted level of x among q[0..L-1] (ascending).  Returns the first
// position with the smallest |fl(x - q_j)|, i.e. the lower level on ties.
// Since rounding is monotone, |fl(x - q_j)| is non-increasing up to the last
// level <= x and non-decreasing after it, so the minimum sits at the bracket
// {a, b} found by binary search; a run of equal distances ending at a is
// walked back to its first element (duplicate levels, or levels closer than
// the distance's ulp).
__device__ __forceinline__ int nearest_full(const float* __restrict__ q, int logL, float x, float& dist) {
  int pos = 0;  // number of levels <= x among q[0 .. L-2]
  for (int step = (1 << logL) >> 1; step >= 1; step >>= 1)
    pos += (q[pos + step - 1] <= x) ? step : 0;
  const int a = pos > 0 ? pos - 1 : 0;
  const int b = pos;
  const float da = fabsf(x - q[a]);
  const float db = fabsf(x - q[b]);
  if (db < da) {
    dist = db;
    return b;
  }
  int j = a;
  if (a > 0 && fabsf(x - q[a - 1]) == da) {
    j = 0;
    while (j < a && fabsf(x - q[j]) != da) ++j;
  }
  dist = da;
  return j;
}

// Local mapping: first nearest of {max(d-1,0), d, min(d+1,L-1)}.
__device__ __forceinline__ int nearest_local(const float* __restrict__ q, int L, int d, float x, float& dist) {
  const int l = d > 0 ? d - 1 : 0;
  const int r = d < L - 1 ? d + 1 : L - 1;
  int best = l;
  float bd = fabsf(x - q[l]);
  const float dm = fabsf(x - q[d]);
  if (dm < bd) { best = d; bd = dm; }
  const float dr = fabsf(x - q[r]);
  if (dr < bd) { best = r; bd = dr; }
  dist = bd;
  return best;
}

// Makes a wavefront's earlier LDS writes visible to its later LDS reads from
// other lanes: LDS executes one wavefront's instructions in order, so waiting
// for its own outstanding LDS operations is enough (no workgroup barrier).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
  __builtin_amdgcn_wave_barrier();
}

// nearest_full with the table size fixed at compile time (unrolled search).
template <int LOGL>
__device__ __forceinline__ int nearest_full_k(const float* __restrict__ q, float x, float& dist) {
  constexpr int L = 1 << LOGL;
  int pos = 0;  // number of levels <= x among q[0 .. L-2]
#pragma unroll
  for (int step = L >> 1; step >= 1; step >>= 1) pos += (q[pos + step - 1] <= x) ? step : 0;
  const int a = pos > 0 ? pos - 1 : 0;
  const int b = pos;
  const float da = fabsf(x - q[a]);
  const float db = fabsf(x - q[b]);
  if (db < da) {
    dist = db;
    return b;
  }
  int j = a;
  if (a > 0 && fabsf(x - q[a - 1]) == da) {  // run of equal distances: take its first element
    j = 0;
    while (j < a && fabsf(x - q[j]) != da) ++j;
  }
  dist = da;
  return j;
}

}  // namespace uq
