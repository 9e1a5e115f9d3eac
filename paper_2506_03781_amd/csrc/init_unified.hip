// Unified initialisation of UniQuan_F's parameters (Sec. 3 "Unified
// initialization"; appendix algorithms "Unified Initialization" and "General
// alternating update"; appendix "Details of clipping strategies").
//
// Per group of g weights: a grid search over gamma = j/G of candidate
// (Delta', z'_U) from a clipping strategy; for each, wbar = T_F(w) with
// s = s_r = 1, the general alternating update (greedy start, then T rounds of
// least-squares alpha, nearest codes and, with a one-point grid, the mean
// shift z_B), and the error ||w - Q*(w)||^2; the first smallest error wins.
//
// Mapping: each lane holds 8 consecutive weights, a group is g/8 adjacent
// lanes, a wavefront 512 weights.  Everything stays in registers except each
// group's 2^k-level table (LDS, wave-private).  The arithmetic follows one
// fixed order so that every code and every scale is reproducible:
//   * group sums are pairwise with adjacent pairing: a lane's 8 values as
//     ((v0+v1)+(v2+v3))+((v4+v5)+(v6+v7)), then xor-butterflies over lane
//     distance 1, 2, 4, ... (each step adds the sibling subtree);
//   * C^T C holds integers; its inverse is exact: alpha_a =
//     fp32( fp64(sum_b adj_ab v_b) / det ) with the integer adjugate, where
//     every product adj_ab v_b is exact in fp64 (C^T C and its adjugate are
//     positive semidefinite, so |adj_ab| <= g^3 <= 2^27, and v is fp32);
//     det = 0 keeps the previous alpha; where a group has at least
//     k (k + 1) / 2 lanes, each of its lanes computes one distinct adjugate
//     entry and lane a forms alpha_a (shuffles gather the operands), instead
//     of every lane solving the whole system;
//   * nearest level: first minimum of |fl(wbar - q)| over the ascending table
//     (the forward's rule), a constant group takes Delta' = 1.
// ALU-bound: the weights are read once and stay in registers for all G * T
// rounds.
#include "uq_device.h"
#include "uq_launch.h"

namespace uq {

struct InitArgs {
  int64_t N;
  int logg, gpr, G, T, clip;
  const void* W;
  float* delta;
  float* z_u;
  float* alpha;
  float* z_b;
  uint8_t* codes;
  float* err;
  float* s;
  float* s_r;
};

// Value of the lane whose subtree is the sibling of this lane's at butterfly
// level M (lane distance M).  Levels 1 and 2 pair lanes by xor (quad_perm);
// from level 4 on every lane of a subtree holds the same partial sum, so the
// mirror patterns (lane i <-> 7-i within 8, 15-i within 16) reach the sibling
// subtree as xor would, without going through LDS.
template <int M>
__device__ __forceinline__ int sibling(int v) {
  if constexpr (M == 1) return __builtin_amdgcn_mov_dpp(v, 0xB1, 0xF, 0xF, false);   // quad_perm [1,0,3,2]
  else if constexpr (M == 2) return __builtin_amdgcn_mov_dpp(v, 0x4E, 0xF, 0xF, false);  // quad_perm [2,3,0,1]
  else if constexpr (M == 4) return __builtin_amdgcn_mov_dpp(v, 0x141, 0xF, 0xF, false); // row_half_mirror
  else if constexpr (M == 8) return __builtin_amdgcn_mov_dpp(v, 0x140, 0xF, 0xF, false); // row_mirror
  else if constexpr (M == 16) return __builtin_amdgcn_ds_swizzle(v, 0x401F);             // lane ^ 16
  else return __shfl_xor(v, 32, 64);
}

template <int M>
__device__ __forceinline__ float sibling(float v) {
  return __builtin_bit_cast(float, sibling<M>(__builtin_bit_cast(int, v)));
}

// Butterfly over the LPG lanes of a group (sum, min or max).
template <int LPG, typename T, typename Op>
__device__ __forceinline__ T group_reduce(T t, Op op) {
  if constexpr (LPG >= 2) t = op(t, sibling<1>(t));
  if constexpr (LPG >= 4) t = op(t, sibling<2>(t));
  if constexpr (LPG >= 8) t = op(t, sibling<4>(t));
  if constexpr (LPG >= 16) t = op(t, sibling<8>(t));
  if constexpr (LPG >= 32) t = op(t, sibling<16>(t));
  if constexpr (LPG >= 64) t = op(t, sibling<32>(t));
  return t;
}

struct AddF { __device__ float operator()(float a, float b) const { return a + b; } };
struct AddI { __device__ int operator()(int a, int b) const { return a + b; } };
struct MinF { __device__ float operator()(float a, float b) const { return fminf(a, b); } };
struct MaxF { __device__ float operator()(float a, float b) const { return fmaxf(a, b); } };

// Pairwise sum over a group: the lane's 8 values, then lane distances 1, 2, ...
// (IEEE addition is commutative, so both lanes of a pair hold the same sum).
template <int LPG>
__device__ __forceinline__ float group_sum(const float (&v)[8]) {
  const float t = ((v[0] + v[1]) + (v[2] + v[3])) + ((v[4] + v[5]) + (v[6] + v[7]));
  return group_reduce<LPG>(t, AddF());
}

__device__ __forceinline__ uint32_t pack4(int c0, int c1, int c2, int c3) {
  return uint32_t(c0) | (uint32_t(c1) << 8) | (uint32_t(c2) << 16) | (uint32_t(c3) << 24);
}

// Signed minors of C^T C.  M is symmetric with |M_ab| <= g <= 512, so every
// factor fits 24 bits (2x2 minors < 2^19) and every product 32 bits: the
// full-rate 24-bit multiply is exact here.
__device__ __forceinline__ int det2(int a, int b, int c, int d) { return __mul24(a, d) - __mul24(b, c); }

template <int K>
__device__ __forceinline__ int cofactor(const int (&M)[K][K], int r, int c) {
  // (-1)^(r+c) det(M without row r and column c); r, c are compile-time after
  // unrolling, so the index maps resolve statically.
  int S[3][3];
#pragma unroll
  for (int i = 0, ii = 0; i < K; ++i) {
    if (i == r) continue;
#pragma unroll
    for (int j = 0, jj = 0; j < K; ++j) {
      if (j == c) continue;
      S[ii][jj] = M[i][j];
      ++jj;
    }
    ++ii;
  }
  int d;
  if constexpr (K == 2) {
    d = S[0][0];
  } else if constexpr (K == 3) {
    d = det2(S[0][0], S[0][1], S[1][0], S[1][1]);
  } else {
    d = __mul24(S[0][0], det2(S[1][1], S[1][2], S[2][1], S[2][2])) -
        __mul24(S[0][1], det2(S[1][0], S[1][2], S[2][0], S[2][2])) +
        __mul24(S[0][2], det2(S[1][0], S[1][1], S[2][0], S[2][1]));
  }
  return ((r + c) & 1) ? -d : d;
}

// alpha = (C^T C)^{-1} v with the exact inverse adj / det; unchanged if det = 0.
template <int K>
__device__ __forceinline__ void solve_alpha(const int (&M)[K][K], const float (&v)[K], float (&al)[K]) {
  int adj[K][K];
  if constexpr (K == 1) {
    adj[0][0] = 1;
  } else {
#pragma unroll
    for (int a = 0; a < K; ++a)
#pragma unroll
      for (int b = a; b < K; ++b) {
        adj[a][b] = cofactor<K>(M, b, a);  // adj of a symmetric matrix is symmetric
        adj[b][a] = adj[a][b];
      }
  }
  // Laplace along row 0; exact (|terms| < 2^40).  Every product below is
  // exact in fp64, so fma(p, q, S) equals S + p*q rounded once, as in the
  // ascending-b sum it implements.
  double det = 0.0;
#pragma unroll
  for (int b = 0; b < K; ++b) det = __builtin_fma(double(M[0][b]), double(adj[b][0]), det);
  if (det == 0.0) return;
#pragma unroll
  for (int a = 0; a < K; ++a) {
    double S = double(adj[a][0]) * double(v[0]);
#pragma unroll
    for (int b = 1; b < K; ++b) S = __builtin_fma(double(adj[a][b]), double(v[b]), S);
    al[a] = float(S / det);
  }
}

// The same solve spread over the LPG lanes of a group (LPG >= K (K + 1) / 2):
// lane j < K (K + 1) / 2 computes the j-th of the adjugate's distinct entries
// adj_ab, a <= b in row-major order (the cofactor of M without row b and
// column a, its rows and columns chosen by per-lane selects), lane a < K
// gathers row a of the adjugate and forms alpha_a with the arithmetic of
// solve_alpha, and every lane gathers the K results.  The determinant is the
// same row-0 expansion, so the results are those of solve_alpha.
template <int K>
__device__ __forceinline__ int pair_index(int a, int b) {  // a <= b
  return a * K - (a * (a - 1)) / 2 + (b - a);
}

// The minor of M for adjugate entry jl (its rows and columns picked by
// per-lane selects) and the parity of its cofactor's sign.
template <int K>
__device__ __forceinline__ int lane_minor(const int (&M)[K][K], int jl, int (&S)[3][3]) {
  // (a, b) of pair jl, 2 bits each, 4 bits per pair
  uint64_t tab = 0;
#pragma unroll
  for (int a = 0; a < K; ++a)
#pragma unroll
    for (int b = a; b < K; ++b) tab |= uint64_t(a | (b << 2)) << (4 * pair_index<K>(a, b));
  const int jc = jl < K * (K + 1) / 2 ? jl : 0;
  const int e = int(tab >> (4 * jc)) & 15;
  const int c = e & 3, r = e >> 2;  // the minor without row r = b and column c = a
  int R[3][K];
#pragma unroll
  for (int i = 0; i < K - 1; ++i)
#pragma unroll
    for (int j = 0; j < K; ++j) R[i][j] = i >= r ? M[i + 1][j] : M[i][j];
#pragma unroll
  for (int i = 0; i < K - 1; ++i)
#pragma unroll
    for (int j = 0; j < K - 1; ++j) S[i][j] = j >= c ? R[i][j + 1] : R[i][j];
  return (r + c) & 1;
}

template <int K>
__device__ __forceinline__ int lane_cofactor(const int (&M)[K][K], int jl) {
  if constexpr (K == 1) {
    return 1;
  } else {
    int S[3][3];
    const int odd = lane_minor<K>(M, jl, S);
    int d;
    if constexpr (K == 2) {
      d = S[0][0];
    } else if constexpr (K == 3) {
      d = det2(S[0][0], S[0][1], S[1][0], S[1][1]);
    } else {
      d = __mul24(S[0][0], det2(S[1][1], S[1][2], S[2][1], S[2][2])) -
          __mul24(S[0][1], det2(S[1][0], S[1][2], S[2][0], S[2][2])) +
          __mul24(S[0][2], det2(S[1][0], S[1][1], S[2][0], S[2][1]));
    }
    return odd ? -d : d;
  }
}

template <int K, int LPG>
__device__ __forceinline__ void solve_alpha_dist(const int (&M)[K][K], const float (&v)[K], float (&al)[K], int jl,
                                                 int lane) {
  static_assert(LPG >= K * (K + 1) / 2, "one adjugate entry per lane");
  const int mine = lane_cofactor<K>(M, jl);
  const int base = lane - jl;
  // column 0 of the adjugate, the same in every lane of the group
  double det = 0.0;
#pragma unroll
  for (int b = 0; b < K; ++b)
    det = __builtin_fma(double(M[0][b]), double(__shfl(mine, base + pair_index<K>(0, b), 64)), det);
  if (det == 0.0) return;
  // row jl of the adjugate (lanes jl >= K take row K - 1 and discard it)
  const int ar = jl < K ? jl : K - 1;
  double S = 0.0;
#pragma unroll
  for (int b = 0; b < K; ++b) {
    const int idx = ar <= b ? pair_index<K>(ar, b) : pair_index<K>(b, ar);
    const double t = double(__shfl(mine, base + idx, 64));
    S = b == 0 ? t * double(v[0]) : __builtin_fma(t, double(v[b]), S);
  }
  const float out = float(S / det);
#pragma unroll
  for (int a = 0; a < K; ++a) al[a] = __shfl(out, base + a, 64);
}

// Ascending level table of the lane's group in LDS (raw, sorted, code_of).
// jl = lane index within the group.
template <int K>
__device__ __forceinline__ void build_table(float* raw, float* qs, uint8_t* cof, const float (&al)[K], float zb,
                                            int jl, int lpg) {
  constexpr int L = 1 << K;
  for (int b = jl; b < L; b += lpg) {
    float q = zb;
#pragma unroll
    for (int i = 0; i < K; ++i) q = ((b >> i) & 1) ? q + al[i] : q - al[i];
    raw[b] = q;
  }
  wave_lds_sync();
  for (int b = jl; b < L; b += lpg) {
    const float q = raw[b];
    int rank = 0;
#pragma unroll
    for (int b2 = 0; b2 < L; ++b2) {
      const float q2 = raw[b2];
      rank += (q2 < q) | ((q2 == q) & (b2 < b));
    }
    qs[rank] = q;
    cof[rank] = uint8_t(b);
  }
  wave_lds_sync();
}

__host__ __device__ inline size_t init_wave_lds_bytes(int logg, int k) {
  const size_t e = (size_t(512) >> logg) << k;  // levels per wave
  return (e * 9 + 15) & ~size_t(15);
}

template <int WDT, int K, int LOGG>
__global__ __launch_bounds__(kThreads) void init_unified_kernel(InitArgs a) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  constexpr int L = 1 << K;
  constexpr int lpg = 1 << (LOGG - 3);  // lanes per group
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int jl = lane & (lpg - 1);
  const int64_t wave_off = (int64_t(blockIdx.x) * (kThreads / 64) + wave) * 512;
  if (wave_off >= a.N) return;  // whole wavefront past the end (no block barriers below)
  const int64_t off = wave_off + lane * 8;
  const bool active = off < a.N;
  const int64_t gid = active ? (off >> LOGG) : 0;

  // This group's table in the wave's LDS region.
  char* wbase = smem + size_t(wave) * init_wave_lds_bytes(LOGG, K);
  const int gl = lane / lpg;  // group index within the wave
  const int gpw = 64 / lpg;
  float* raw = reinterpret_cast<float*>(wbase) + gl * L;
  float* qs = reinterpret_cast<float*>(wbase) + (gpw + gl) * L;
  uint8_t* cof = reinterpret_cast<uint8_t*>(wbase) + size_t(2 * gpw * L) * 4 + gl * L;

  float w[8];
  if (active) {
    load8<WDT>(a.W, off, w);
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i) w[i] = 0.0f;
  }
  float wm = w[0], wM = w[0];
#pragma unroll
  for (int i = 1; i < 8; ++i) {
    wm = fminf(wm, w[i]);
    wM = fmaxf(wM, w[i]);
  }
  wm = group_reduce<lpg>(wm, MinF());
  wM = group_reduce<lpg>(wM, MaxF());

  const float L1 = float(L - 1);
  const float zb0 = L1 * 0.5f;
  constexpr float inv_g = 1.0f / float(1 << LOGG);  // exact power of two
  constexpr int g = 1 << LOGG;

  float best_d = 1.0f, best_zu = 0.0f, best_zb = zb0, best_e = 0.0f, best_al[K];
  uint32_t best_c0 = 0, best_c1 = 0;
#pragma unroll
  for (int b = 0; b < K; ++b) best_al[b] = 0.0f;

  for (int j = 1; j <= a.G; ++j) {
    const float gamma = float(j) / float(a.G);
    float dl = (gamma * (wM - wm)) / L1;
    if (!(dl > 0.0f)) dl = 1.0f;
    float zu;
    if (a.clip == 0) zu = -(wm / dl);
    else if (a.clip == 1) zu = L1 - (wM / dl);
    else zu = -((gamma * wm) / dl);

    float wbar[8], x[8];
    float zb = zb0;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      wbar[i] = (w[i] / dl) + zu;
      x[i] = wbar[i] - zb;
    }

    // Greedy start: one bit at a time.
    float al[K];
    int code[8];
    {
      float r[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        r[i] = x[i];
        code[i] = 0;
      }
#pragma unroll
      for (int b = 0; b < K; ++b) {
        float ab[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) ab[i] = fabsf(r[i]);
        const float ai = group_sum<lpg>(ab) * inv_g;
        al[b] = ai;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const bool plus = r[i] >= 0.0f;
          code[i] |= int(plus) << b;
          r[i] = plus ? r[i] - ai : r[i] + ai;
        }
      }
    }

    // Codes packed 4 per word: the C^T C counts and the fixed-point test use them.
    uint32_t cw0 = pack4(code[0], code[1], code[2], code[3]);
    uint32_t cw1 = pack4(code[4], code[5], code[6], code[7]);
    for (int t = 0; t < a.T; ++t) {
      // alpha <- (C^T C)^{-1} C^T (wbar - z_B)
      float v[K];
#pragma unroll
      for (int b = 0; b < K; ++b) {
        float sx[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) sx[i] = ((code[i] >> b) & 1) ? x[i] : -x[i];
        v[b] = group_sum<lpg>(sx);
      }
      int M[K][K];
      {
        // bit b of the lane's 8 codes, one bit per byte
        uint32_t p0[K], p1[K];
#pragma unroll
        for (int b = 0; b < K; ++b) {
          p0[b] = (cw0 >> b) & 0x01010101u;
          p1[b] = (cw1 >> b) & 0x01010101u;
        }
#pragma unroll
        for (int p = 0; p < K; ++p) {
          M[p][p] = g;
#pragma unroll
          for (int q = p + 1; q < K; ++q) {
            const int dis = __builtin_popcount(p0[p] ^ p0[q]) + __builtin_popcount(p1[p] ^ p1[q]);
            M[p][q] = g - 2 * group_reduce<lpg>(dis, AddI());
            M[q][p] = M[p][q];
          }
        }
      }
      if constexpr (lpg >= K * (K + 1) / 2) solve_alpha_dist<K, lpg>(M, v, al, jl, lane);
      else solve_alpha<K>(M, v, al);

      // C <- nearest level's code
      build_table<K>(raw, qs, cof, al, zb, jl, lpg);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        float dist;
        code[i] = cof[nearest_full_k<K>(qs, wbar[i], dist)];
      }
      const uint32_t nw0 = pack4(code[0], code[1], code[2], code[3]);
      const uint32_t nw1 = pack4(code[4], code[5], code[6], code[7]);

      // z_B <- mean(wbar - C alpha), only with a one-point grid
      const float zb_prev = zb;
      if (a.G == 1) {
        float dd[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          float ca = 0.0f;
#pragma unroll
          for (int b = 0; b < K; ++b) ca = ((code[i] >> b) & 1) ? ca + al[b] : ca - al[b];
          dd[i] = wbar[i] - ca;
        }
        zb = group_sum<lpg>(dd) * inv_g;
#pragma unroll
        for (int i = 0; i < 8; ++i) x[i] = wbar[i] - zb;
      }

      // Unchanged codes and shift make this state a fixed point of the round
      // (the round is a deterministic function of C, z_B and, for a singular
      // C^T C, alpha), so the remaining rounds would reproduce it exactly.
      const bool same = (nw0 == cw0) & (nw1 == cw1) & (zb == zb_prev);
      cw0 = nw0;
      cw1 = nw1;
      if (__all(same || !active)) break;
    }

    // Candidate error ||w - Q*(w)||^2 with the forward's FULL mapping.
    build_table<K>(raw, qs, cof, al, zb, jl, lpg);
    float e2[8];
    uint32_t c0 = 0, c1 = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      float dist;
      const int pos = nearest_full_k<K>(qs, wbar[i], dist);
      const uint32_t cb = cof[pos];
      if (i < 4) c0 |= cb << (8 * i);
      else c1 |= cb << (8 * (i - 4));
      const float what = dl * (qs[pos] - zu);
      const float d = w[i] - what;
      e2[i] = d * d;
    }
    const float e = group_sum<lpg>(e2);
    if (j == 1 || e < best_e) {
      best_e = e;
      best_d = dl;
      best_zu = zu;
      best_zb = zb;
#pragma unroll
      for (int b = 0; b < K; ++b) best_al[b] = al[b];
      best_c0 = c0;
      best_c1 = c1;
    }
  }

  if (!active) return;
  if (a.codes) store8u8(a.codes, off, make_uint2(best_c0, best_c1));
  if (a.s) {
    const float one[8] = {1.0f, 1.0f, 1.0f, 1.0f, 1.0f, 1.0f, 1.0f, 1.0f};
    store8f(a.s, off, one);
  }
  if (jl == 0) {
    a.delta[gid] = best_d;
    a.z_u[gid] = best_zu;
    a.z_b[gid] = best_zb;
#pragma unroll
    for (int b = 0; b < K; ++b) a.alpha[gid * K + b] = best_al[b];
    if (a.err) a.err[gid] = best_e;
    if (a.s_r && (gid % a.gpr) == 0) a.s_r[gid / a.gpr] = 1.0f;
  }
}

// ---------------------------------------------------------------------------
// Groups of more than 512 weights (a whole row per group, up to 16384): one
// workgroup per group, NW wavefronts, lane l holding the E consecutive
// elements l E .. l E + E - 1 of the group zero-padded to P = 64 NW E (the
// next power of two; E >= 8), so the pairwise tree over the padded group is
// the lane's own pairwise sum of its E values, then the butterfly over the 64
// lanes of a wavefront, then the wavefronts' sums pairwise in order.  The
// weights, their transforms and the codes stay in registers; each wavefront
// keeps its own copy of the level table in LDS.  C^T C entries reach g, so
// its adjugate (|adj| <= g^3 < 2^42) and determinant are int64, exactly
// converted (the determinant rounded) to fp64, and the products adj_ab v_b
// round in fp64 and are added in ascending b, as written.
// ---------------------------------------------------------------------------
// Pairwise sum of E values produced in index order (adjacent pairing): a
// stack of partial sums, one per level.
template <int E>
struct LaneTree {
  static constexpr int LG = __builtin_ctz(E);
  float st[LG + 1];
  template <int I>
  __device__ __forceinline__ void push(float v) {
#pragma unroll
    for (int l = 0; l < LG; ++l) {
      if (((I >> l) & 1) == 0) {
        st[l] = v;
        return;
      }
      v = st[l] + v;
    }
    st[LG] = v;
  }
};

template <int E, int I = 0, typename F>
__device__ __forceinline__ void tree_push_all(LaneTree<E>& t, const F& f) {
  if constexpr (I < E) {
    t.template push<I>(f(I));
    tree_push_all<E, I + 1>(t, f);
  }
}

// Pairwise sum of the N (a power of two) values r[0 .. N-1] in order.
template <int N>
__device__ __forceinline__ float pairwise_lds(const float* r) {
  if constexpr (N == 1) return r[0];
  else return pairwise_lds<N / 2>(r) + pairwise_lds<N / 2>(r + N / 2);
}

// Workgroup-wide pairwise sums of NV lane values (each lane already holds its
// own subtree's sum), left in every lane; red holds NV values per wavefront.
template <int NW, int NV, int CAP>
__device__ __forceinline__ void block_tree(float (&t)[NV], float (&red)[CAP], int lane, int wave) {
  static_assert(NV * NW <= CAP, "reduction buffer too small");
#pragma unroll
  for (int v = 0; v < NV; ++v) t[v] = group_reduce<64>(t[v], AddF());
  if (lane == 0) {
#pragma unroll
    for (int v = 0; v < NV; ++v) red[v * NW + wave] = t[v];
  }
  __syncthreads();
#pragma unroll
  for (int v = 0; v < NV; ++v) t[v] = pairwise_lds<NW>(red + v * NW);
  __syncthreads();
}

template <int NW, int NV, int CAP>
__device__ __forceinline__ void block_isum(int (&t)[NV], int (&red)[CAP], int lane, int wave) {
  static_assert(NV * NW <= CAP, "reduction buffer too small");
#pragma unroll
  for (int v = 0; v < NV; ++v) t[v] = group_reduce<64>(t[v], AddI());
  if (lane == 0) {
#pragma unroll
    for (int v = 0; v < NV; ++v) red[v * NW + wave] = t[v];
  }
  __syncthreads();
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    int s = 0;
#pragma unroll
    for (int q = 0; q < NW; ++q) s += red[v * NW + q];
    t[v] = s;
  }
  __syncthreads();
}

// alpha = (C^T C)^{-1} v for C^T C entries up to 2^14, spread over the lanes
// of a wavefront as solve_alpha_dist: lane j < K (K + 1) / 2 computes one
// distinct adjugate entry in int64 (|adj| <= g^3 < 2^42), lane a < K forms
// alpha_a = (sum_b adj_ab v_b) / det with the exact int64 determinant (row-0
// expansion) converted to fp64 and the fp64 products added in ascending b,
// and every lane gathers the K results.  Unchanged if det = 0.
__device__ __forceinline__ int64_t shfl64(int64_t x, int src) {
  const int lo = __shfl(int(uint32_t(uint64_t(x))), src, 64);
  const int hi = __shfl(int(uint32_t(uint64_t(x) >> 32)), src, 64);
  return int64_t((uint64_t(uint32_t(hi)) << 32) | uint32_t(lo));
}

template <int K>
__device__ __forceinline__ void solve_alpha64_dist(const int (&M)[K][K], const float (&v)[K], float (&al)[K],
                                                   int lane) {
  int64_t mine = 1;
  if constexpr (K > 1) {
    int S0[3][3];
    const int odd = lane_minor<K>(M, lane, S0);
    int64_t S[3][3];
#pragma unroll
    for (int i = 0; i < K - 1; ++i)
#pragma unroll
      for (int j = 0; j < K - 1; ++j) S[i][j] = S0[i][j];
    int64_t d;
    if constexpr (K == 2) {
      d = S[0][0];
    } else if constexpr (K == 3) {
      d = S[0][0] * S[1][1] - S[0][1] * S[1][0];
    } else {
      d = S[0][0] * (S[1][1] * S[2][2] - S[1][2] * S[2][1]) - S[0][1] * (S[1][0] * S[2][2] - S[1][2] * S[2][0]) +
          S[0][2] * (S[1][0] * S[2][1] - S[1][1] * S[2][0]);
    }
    mine = odd ? -d : d;
  }
  int64_t det = 0;
#pragma unroll
  for (int b = 0; b < K; ++b) det += int64_t(M[0][b]) * shfl64(mine, pair_index<K>(0, b));
  if (det == 0) return;
  const double dd = double(det);
  const int ar = lane < K ? lane : K - 1;
  double S = 0.0;
#pragma unroll
  for (int b = 0; b < K; ++b) {
    const int idx = ar <= b ? pair_index<K>(ar, b) : pair_index<K>(b, ar);
    const double pr = double(shfl64(mine, idx)) * double(v[b]);
    S = b == 0 ? pr : S + pr;
  }
  const float out = float(S / dd);
#pragma unroll
  for (int a = 0; a < K; ++a) al[a] = __shfl(out, a, 64);
}

template <int WDT, int K, int NW, int E>
__global__ __launch_bounds__(NW * 64) void init_unified_big_kernel(InitArgs a, int g) {
  constexpr int L = 1 << K;
  constexpr int NP = E / 4;  // packed code words per lane
  __shared__ float tab_raw[NW][L], tab_qs[NW][L];
  __shared__ uint8_t tab_cof[NW][L];
  __shared__ float red[8 * NW];
  __shared__ int redi[8 * NW];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t gid = blockIdx.x;
  const int64_t goff = gid * int64_t(g);
  const int e0 = int(threadIdx.x) * E;  // first padded element of this lane
  float* raw = tab_raw[wave];
  float* qs = tab_qs[wave];
  uint8_t* cof = tab_cof[wave];

  float w[E];
#pragma unroll
  for (int c = 0; c < E; c += 8) {
    float v[8];
    if (e0 + c < g) {
      load8<WDT>(a.W, goff + e0 + c, v);
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = 0.0f;
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) w[c + i] = v[i];
  }
  // validity: g is a multiple of 8, so chunks of 8 are whole
  uint32_t valid8 = 0;  // bit c/8: chunk c .. c+7 real
#pragma unroll
  for (int c = 0; c < E; c += 8)
    if (e0 + c < g) valid8 |= 1u << (c / 8);
#define UQ_VALID(i) (((valid8 >> ((i) / 8)) & 1u) != 0u)
  // A wavefront whose elements are all padding adds exact zeros to every sum
  // and keeps code 0: it skips the per-element work and only joins the
  // workgroup reductions.
  const bool live = __builtin_amdgcn_readfirstlane(wave) * 64 * E < g;

  float mm[2] = {INFINITY, -INFINITY};
#pragma unroll
  for (int i = 0; i < E; ++i)
    if (UQ_VALID(i)) {
      mm[0] = fminf(mm[0], w[i]);
      mm[1] = fmaxf(mm[1], w[i]);
    }
  mm[0] = group_reduce<64>(mm[0], MinF());
  mm[1] = group_reduce<64>(mm[1], MaxF());
  if (lane == 0) {
    red[wave] = mm[0];
    red[NW + wave] = mm[1];
  }
  __syncthreads();
  float wm = red[0], wM = red[NW];
#pragma unroll
  for (int q = 1; q < NW; ++q) {
    wm = fminf(wm, red[q]);
    wM = fmaxf(wM, red[NW + q]);
  }
  __syncthreads();

  const float L1 = float(L - 1);
  const float zb0 = L1 * 0.5f;
  const float gf = float(g);
  float best_d = 1.0f, best_zu = 0.0f, best_zb = zb0, best_e = 0.0f, best_al[K];
  uint32_t best_cw[NP];
#pragma unroll
  for (int b = 0; b < K; ++b) best_al[b] = 0.0f;
#pragma unroll
  for (int q = 0; q < NP; ++q) best_cw[q] = 0u;

  for (int j = 1; j <= a.G; ++j) {
    const float gamma = float(j) / float(a.G);
    float dl = (gamma * (wM - wm)) / L1;
    if (!(dl > 0.0f)) dl = 1.0f;
    float zu;
    if (a.clip == 0) zu = -(wm / dl);
    else if (a.clip == 1) zu = L1 - (wM / dl);
    else zu = -((gamma * wm) / dl);
    float wbar[E];
#pragma unroll
    for (int i = 0; i < E; ++i) wbar[i] = (w[i] / dl) + zu;
    float zb = zb0;

    // greedy start, one bit at a time (r recomputed from x and the bits so far)
    float al[K];
    uint32_t cw[NP];
#pragma unroll
    for (int q = 0; q < NP; ++q) cw[q] = 0u;
#pragma unroll
    for (int b = 0; b < K; ++b) {
      float t[1] = {0.0f};
      if (live) {
        LaneTree<E> tr;
        tree_push_all<E>(tr, [&](int i) {
          float r = wbar[i] - zb;
          for (int bb = 0; bb < b; ++bb) r = ((cw[i / 4] >> (8 * (i & 3) + bb)) & 1u) ? r - al[bb] : r + al[bb];
          return UQ_VALID(i) ? fabsf(r) : 0.0f;
        });
        t[0] = tr.st[LaneTree<E>::LG];
      }
      block_tree<NW, 1>(t, red, lane, wave);
      const float ai = t[0] / gf;
      if (live) {
#pragma unroll
        for (int i = 0; i < E; ++i) {
          float r = wbar[i] - zb;
          for (int bb = 0; bb < b; ++bb) r = ((cw[i / 4] >> (8 * (i & 3) + bb)) & 1u) ? r - al[bb] : r + al[bb];
          if (UQ_VALID(i) && r >= 0.0f) cw[i / 4] |= 1u << (8 * (i & 3) + b);
        }
      }
      al[b] = ai;
    }

    for (int t = 0; t < a.T; ++t) {
      // alpha <- (C^T C)^{-1} C^T (wbar - z_B)
      float v[K];
#pragma unroll
      for (int b = 0; b < K; ++b) {
        v[b] = 0.0f;
        if (live) {
          LaneTree<E> tr;
          tree_push_all<E>(tr, [&](int i) {
            const float x = wbar[i] - zb;
            const bool bit = (cw[i / 4] >> (8 * (i & 3) + b)) & 1u;
            return UQ_VALID(i) ? (bit ? x : -x) : 0.0f;
          });
          v[b] = tr.st[LaneTree<E>::LG];
        }
      }
      block_tree<NW, K>(v, red, lane, wave);
      int M[K][K];
      {
        // disagreement counts of bit pairs p < q, in row-major order
        constexpr int NPQ = K > 1 ? K * (K - 1) / 2 : 1;
        int dis[NPQ];
        dis[0] = 0;
#pragma unroll
        for (int p = 0, n = 0; p < K; ++p)
#pragma unroll
          for (int q = p + 1; q < K; ++q, ++n) {
            int c = 0;
#pragma unroll
            for (int w4 = 0; w4 < NP; ++w4)
              c += __builtin_popcount(((cw[w4] >> p) ^ (cw[w4] >> q)) & 0x01010101u);
            dis[n] = c;
          }
        block_isum<NW, NPQ>(dis, redi, lane, wave);
#pragma unroll
        for (int p = 0, n = 0; p < K; ++p) {
          M[p][p] = g;
#pragma unroll
          for (int q = p + 1; q < K; ++q, ++n) {
            M[p][q] = g - 2 * dis[n];
            M[q][p] = M[p][q];
          }
        }
      }
      solve_alpha64_dist<K>(M, v, al, lane);

      // C <- nearest level's code (padding keeps code 0)
      uint32_t nw[NP];
#pragma unroll
      for (int q = 0; q < NP; ++q) nw[q] = 0u;
      if (live) {
        build_table<K>(raw, qs, cof, al, zb, lane, 64);
#pragma unroll
        for (int i = 0; i < E; ++i) {
          if (UQ_VALID(i)) {
            float dist;
            nw[i / 4] |= uint32_t(cof[nearest_full_k<K>(qs, wbar[i], dist)]) << (8 * (i & 3));
          }
        }
      }
      const float zb_prev = zb;
      if (a.G == 1) {
        float tz[1] = {0.0f};
        if (live) {
          LaneTree<E> tr;
          tree_push_all<E>(tr, [&](int i) {
            const uint32_t code = (nw[i / 4] >> (8 * (i & 3))) & 0xFFu;
            float ca = 0.0f;
            for (int b = 0; b < K; ++b) ca = ((code >> b) & 1u) ? ca + al[b] : ca - al[b];
            return UQ_VALID(i) ? wbar[i] - ca : 0.0f;
          });
          tz[0] = tr.st[LaneTree<E>::LG];
        }
        block_tree<NW, 1>(tz, red, lane, wave);
        zb = tz[0] / gf;
      }
      int same = 1;
#pragma unroll
      for (int q = 0; q < NP; ++q) same &= int(nw[q] == cw[q]);
      same &= int(zb == zb_prev);
#pragma unroll
      for (int q = 0; q < NP; ++q) cw[q] = nw[q];
      int st1[1] = {same};
      block_isum<NW, 1>(st1, redi, lane, wave);
      if (st1[0] == NW * 64) break;  // every lane at a fixed point (uniform)
    }

    // candidate error ||w - Q*(w)||^2 with the forward's FULL mapping
    uint32_t cc[NP];
#pragma unroll
    for (int q = 0; q < NP; ++q) cc[q] = 0u;
    float te[1] = {0.0f};
    if (live) {
      build_table<K>(raw, qs, cof, al, zb, lane, 64);
      LaneTree<E> tr;
      tree_push_all<E>(tr, [&](int i) {
        if (!UQ_VALID(i)) return 0.0f;
        float dist;
        const int pos = nearest_full_k<K>(qs, wbar[i], dist);
        cc[i / 4] |= uint32_t(cof[pos]) << (8 * (i & 3));
        const float what = dl * (qs[pos] - zu);
        const float d = w[i] - what;
        return d * d;
      });
      te[0] = tr.st[LaneTree<E>::LG];
    }
    block_tree<NW, 1>(te, red, lane, wave);
    const float e = te[0];
    if (j == 1 || e < best_e) {
      best_e = e;
      best_d = dl;
      best_zu = zu;
      best_zb = zb;
#pragma unroll
      for (int b = 0; b < K; ++b) best_al[b] = al[b];
#pragma unroll
      for (int q = 0; q < NP; ++q) best_cw[q] = cc[q];
    }
  }

#pragma unroll
  for (int c = 0; c < E; c += 8) {
    if (e0 + c >= g) continue;
    if (a.codes) store8u8(a.codes, goff + e0 + c, make_uint2(best_cw[c / 4], best_cw[c / 4 + 1]));
    if (a.s) {
      const float one[8] = {1.0f, 1.0f, 1.0f, 1.0f, 1.0f, 1.0f, 1.0f, 1.0f};
      store8f(a.s, goff + e0 + c, one);
    }
  }
#undef UQ_VALID
  if (threadIdx.x == 0) {
    a.delta[gid] = best_d;
    a.z_u[gid] = best_zu;
    a.z_b[gid] = best_zb;
#pragma unroll
    for (int b = 0; b < K; ++b) a.alpha[gid * K + b] = best_al[b];
    if (a.err) a.err[gid] = best_e;
    if (a.s_r && (gid % a.gpr) == 0) a.s_r[gid / a.gpr] = 1.0f;
  }
}

template <int WDT, int K>
static void launch_init_big(const InitArgs& a, int g, int64_t groups, hipStream_t st) {
  int p2 = 1024;
  while (p2 < g) p2 <<= 1;
  const dim3 grid(static_cast<unsigned>(groups));
  switch (p2) {
    case 1024: hipLaunchKernelGGL((init_unified_big_kernel<WDT, K, 2, 8>), grid, dim3(128), 0, st, a, g); break;
    case 2048: hipLaunchKernelGGL((init_unified_big_kernel<WDT, K, 4, 8>), grid, dim3(256), 0, st, a, g); break;
    case 4096: hipLaunchKernelGGL((init_unified_big_kernel<WDT, K, 4, 16>), grid, dim3(256), 0, st, a, g); break;
    case 8192: hipLaunchKernelGGL((init_unified_big_kernel<WDT, K, 8, 16>), grid, dim3(512), 0, st, a, g); break;
    default: hipLaunchKernelGGL((init_unified_big_kernel<WDT, K, 16, 16>), grid, dim3(1024), 0, st, a, g); break;
  }
}

template <int WDT>
static hipError_t launch_init_big_k(const InitArgs& a, int k, int g, int64_t groups, hipStream_t st) {
  switch (k) {
    case 1: launch_init_big<WDT, 1>(a, g, groups, st); break;
    case 2: launch_init_big<WDT, 2>(a, g, groups, st); break;
    case 3: launch_init_big<WDT, 3>(a, g, groups, st); break;
    default: launch_init_big<WDT, 4>(a, g, groups, st); break;
  }
  return hipGetLastError();
}

template <int WDT, int K>
static void launch_init_g(const InitArgs& a, dim3 grid, size_t lds, hipStream_t st) {
  switch (a.logg) {
    case 3: hipLaunchKernelGGL((init_unified_kernel<WDT, K, 3>), grid, dim3(kThreads), lds, st, a); break;
    case 4: hipLaunchKernelGGL((init_unified_kernel<WDT, K, 4>), grid, dim3(kThreads), lds, st, a); break;
    case 5: hipLaunchKernelGGL((init_unified_kernel<WDT, K, 5>), grid, dim3(kThreads), lds, st, a); break;
    case 6: hipLaunchKernelGGL((init_unified_kernel<WDT, K, 6>), grid, dim3(kThreads), lds, st, a); break;
    case 7: hipLaunchKernelGGL((init_unified_kernel<WDT, K, 7>), grid, dim3(kThreads), lds, st, a); break;
    case 8: hipLaunchKernelGGL((init_unified_kernel<WDT, K, 8>), grid, dim3(kThreads), lds, st, a); break;
    default: hipLaunchKernelGGL((init_unified_kernel<WDT, K, 9>), grid, dim3(kThreads), lds, st, a); break;
  }
}

template <int WDT>
static hipError_t launch_init_k(const InitArgs& a, int k, dim3 grid, size_t lds, hipStream_t st) {
  switch (k) {
    case 1: launch_init_g<WDT, 1>(a, grid, lds, st); break;
    case 2: launch_init_g<WDT, 2>(a, grid, lds, st); break;
    case 3: launch_init_g<WDT, 3>(a, grid, lds, st); break;
    default: launch_init_g<WDT, 4>(a, grid, lds, st); break;
  }
  return hipGetLastError();
}

hipError_t launch_init_unified(const InitUnifiedLaunch& p, hipStream_t st) {
  InitArgs a;
  a.N = p.R * p.C;
  a.logg = p.g > 512 ? 0 : __builtin_ctz(unsigned(p.g));
  a.gpr = int(p.C / p.g);
  a.G = p.grid_G;
  a.T = p.alt_T;
  a.clip = p.clip;
  a.W = p.W;
  a.delta = p.delta; a.z_u = p.z_u; a.alpha = p.alpha; a.z_b = p.z_b;
  a.codes = p.codes; a.err = p.err; a.s = p.s; a.s_r = p.s_r;
  if (p.g > 512) {
    const int64_t groups = a.N / p.g;
    if (p.w_dtype == BF16) return launch_init_big_k<BF16>(a, p.k, p.g, groups, st);
    return launch_init_big_k<F32>(a, p.k, p.g, groups, st);
  }
  const int64_t waves = (a.N + 511) / 512;
  const dim3 grid(unsigned((waves + 3) / 4));
  const size_t lds = 4 * init_wave_lds_bytes(a.logg, p.k);
  if (p.w_dtype == BF16) return launch_init_k<BF16>(a, p.k, grid, lds, st);
  return launch_init_k<F32>(a, p.k, grid, lds, st);
}

}  // namespace uq
