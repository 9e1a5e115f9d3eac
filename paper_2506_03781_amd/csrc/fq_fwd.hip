// Quantizer forward Q*_{I_F} (Eq. (3)), the unification-theorem fold
// (Theorem 1, Eq. (4)), binary-coding dequantization (Sec. 2.3) and the
// greedy binary-coding start (appendix "General alternating update").
//
// Work split of the forward for groups of up to 512 weights (a power of two,
// so a group never straddles wavefronts): each wavefront owns 512
// consecutive weights (8 per lane, 16-byte bf16 / 2 x 16-byte fp32 loads; a
// 128-weight group is 16 lanes) and builds the sorted level tables of its own
// groups in a private LDS region, with wave-local ordering only; every lane
// then maps its 8 weights by an LDS binary search (FULL), a neighbour-table
// lookup (LOCAL) or the stored code (FROZEN).  fq_step_kernel is the same
// forward preceded, in the same pass, by the straight-through backward and
// the SGD update of the group's parameters (the previous step's end).  The
// fold, dequantization and greedy kernels work on tiles of whole groups per
// workgroup with workgroup-wide tables.  Groups of more than 512 weights (a
// whole row per group) take the *_big kernels: one workgroup of 256 lanes per
// group, its tables built once in LDS and its sums reduced across the
// wavefronts in a fixed order.  HBM-bound: per weight the forward reads W
// (2 B) and s (4 B) and writes What (2 B) and the code byte (1 B).
#include "uq_device.h"
#include "uq_launch.h"

namespace uq {

struct TileGeom {
  int64_t N;        // R * C
  int logg;         // g = 1 << logg
  int logL;         // L = 2^k
  int k;
  int gpr;          // groups per row
  int tile_groups;  // groups per workgroup tile
};

__device__ __forceinline__ float tau_of(const float* __restrict__ alpha_g, int k) {
  float t = fabsf(alpha_g[0]);
  for (int i = 1; i < k; ++i) t = fminf(t, fabsf(alpha_g[i]));
  return t;
}

// The same two quantities with k fixed at compile time (unrolled, one base
// address for the k loads).
template <int K>
__device__ __forceinline__ float tau_k(const float* __restrict__ alpha_g) {
  float t = fabsf(alpha_g[0]);
#pragma unroll
  for (int i = 1; i < K; ++i) t = fminf(t, fabsf(alpha_g[i]));
  return t;
}

template <int K>
__device__ __forceinline__ float level_value_k(const float* __restrict__ alpha_g, float zb, int b) {
  float q = zb;
#pragma unroll
  for (int i = 0; i < K; ++i) q = ((b >> i) & 1) ? q + alpha_g[i] : q - alpha_g[i];
  return q;
}

// Raw storage of 8 weights as loaded (bf16 kept packed until use).
template <int DT> struct Raw8;
template <> struct Raw8<BF16> {
  uint4 q;
  __device__ __forceinline__ void load(const void* base, int64_t off) {
    q = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(base) + off);
  }
  __device__ __forceinline__ float get(int i) const {
    const uint32_t w = i < 2 ? q.x : i < 4 ? q.y : i < 6 ? q.z : q.w;
    return (i & 1) ? __uint_as_float(w & 0xFFFF0000u) : __uint_as_float(w << 16);
  }
};
template <> struct Raw8<F32> {
  float4 a, b;
  __device__ __forceinline__ void load(const void* base, int64_t off) {
    const float4* p = reinterpret_cast<const float4*>(static_cast<const float*>(base) + off);
    a = p[0];
    b = p[1];
  }
  __device__ __forceinline__ float get(int i) const {
    const float4& v = i < 4 ? a : b;
    const int j = i & 3;
    return j == 0 ? v.x : j == 1 ? v.y : j == 2 ? v.z : v.w;
  }
};

struct FwdArgs {
  TileGeom t;
  const void* W;
  const float* s;
  const float* s_r;
  const float* delta;
  const float* z_u;
  const float* alpha;
  const float* z_b;
  uint8_t* codes;
  void* W_hat;
  int resid;  // 1: store What - W (the reconstruction residual) instead of What
};

// Dynamic LDS of a quantizer tile: the level tables plus four per-group
// fp32 arrays.
static size_t tile_lds_bytes(const TileGeom& t) {
  const size_t e = size_t(t.tile_groups) << t.logL;
  return ((e * 10 + 15) & ~size_t(15)) + 16 * size_t(t.tile_groups);
}

// Per-wave LDS bytes: the level tables of (512 ch / g) groups of 2^k levels,
// optionally the local-mapping neighbour table (16 B per level), and 4
// floats per group.
__host__ __device__ inline size_t wave_lds_bytes(int logg, int k, bool nbt, int ch = 1) {
  const size_t groups = (size_t(512) * ch) >> logg;
  const size_t e = groups << k;
  return ((e * 10 + 15) & ~size_t(15)) + (nbt ? 16 * e : 0) + 16 * groups + (k <= 4 ? 8 * e : 0);
}

// Sort key of level b with value q: the value's bits mapped to an unsigned
// integer of the same order (-0 folded onto +0 first), then the code, so one
// 64-bit compare orders by (value, code).
__device__ __forceinline__ uint64_t level_key(float q, int b) {
  const uint32_t u = __float_as_uint(q + 0.0f);
  const uint32_t ord = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return (uint64_t(ord) << 8) | uint64_t(b);
}

// Neighbour tables for the local mapping are kept when they fit (16 B per
// level, at most 4096 levels per wave).
static bool use_neighbour_table(int logg, int k) { return ((size_t(512) >> logg) << k) <= 4096; }

// Forward kernel.  Each wavefront owns CH chunks of 512 consecutive weights
// (8 per lane per chunk; groups never straddle chunks since g divides 512)
// and keeps the level tables of their groups in a private LDS region, so
// table building needs only wave-local ordering and no workgroup barrier.
// The wave builds its tables first (one lane per level computes q(b), then
// ranks it among the group's levels by counting, sort key (value, code)) and
// only then issues the W, s (and code) loads of all its chunks, CH x 3.5 KB
// in flight: a wave's loads complete in issue order, so parameter loads
// issued behind the chunk loads kept the table build waiting for the whole
// chunk, while other wavefronts' chunk loads cover this one's table build.
// MODE: 0 FULL, 1 LOCAL by search, 2 FROZEN, 3 LOCAL through the neighbour
// table (the LOCAL variant used whenever the table fits).
template <int WDT, int ODT, int MODE, int LOGL, int CH>
__global__ __launch_bounds__(kThreads) void fq_fwd_kernel(FwdArgs a) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  constexpr int L = 1 << LOGL;
  constexpr int WPW = 512 * CH;                     // weights per wave
  constexpr bool has_nb = MODE == 3;
  constexpr bool keyed = LOGL <= 4;                 // rank by 64-bit keys
  const TileGeom& g = a.t;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int gw = WPW >> g.logg;                     // groups per wave (g divides 512)
  const int ew = gw << LOGL;                        // table entries per wave
  char* mine = smem + size_t(wave) * wave_lds_bytes(g.logg, LOGL, has_nb, CH);
  LevelTables tab;
  char* p = carve_tables(tab, mine, ew);
  float4* nb = reinterpret_cast<float4*>(p);        // [ew] (q_l, q_d, q_r, codes l|d<<8|r<<16)
  if (has_nb) p += 16 * size_t(ew);
  float* s_ds = reinterpret_cast<float*>(p);
  float* s_zu = s_ds + gw;
  float* s_dl = s_zu + gw;
  float* s_tau = s_dl + gw;
  uint64_t* keys = reinterpret_cast<uint64_t*>(s_tau + gw);  // [ew] when keyed; 16-byte aligned (16 gw bytes above)
  const int64_t wbase = (int64_t(blockIdx.x) * (blockDim.x >> 6) + wave) * WPW;  // first weight of this wave
  if (wbase >= g.N) return;                                       // whole wave past the end
  const int nvalid = int(min<int64_t>(WPW, g.N - wbase));        // a multiple of g (and of 8)
  const int gv = nvalid >> g.logg;                                // valid groups of this wave
  const int ev = gv << LOGL;                                      // valid table entries
  const int64_t gid0 = wbase >> g.logg;

  Raw8<WDT> w[CH];
  float4 s0[CH], s1[CH];
  uint2 prev[CH];
  // raw levels by code (and their sort keys), and the per-group parameters
  for (int e = lane; e < ev; e += 64) {
    const int gl = e >> LOGL;
    const float q = level_value_k<LOGL>(a.alpha + (gid0 + gl) * LOGL, a.z_b[gid0 + gl], e & (L - 1));
    tab.raw[e] = q;
    if constexpr (keyed && MODE != 2) keys[e] = level_key(q, e & (L - 1));
  }
  for (int gl = lane; gl < gv; gl += 64) {
    const int64_t gid = gid0 + gl;
    const float dl = a.delta ? a.delta[gid] : 1.0f;
    const float sr = a.s_r ? a.s_r[uint32_t(gid) / uint32_t(g.gpr)] : 1.0f;
    s_ds[gl] = dl * sr;
    s_dl[gl] = dl;
    s_zu[gl] = a.z_u ? a.z_u[gid] : 0.0f;
    s_tau[gl] = tau_k<LOGL>(a.alpha + gid * LOGL);
  }
  wave_lds_sync();
  if constexpr (MODE != 2) {
    // sorted order: rank of each level by counting, key (value, code)
    for (int e = lane; e < ev; e += 64) {
      const int gl = e >> LOGL;
      const int b = e & (L - 1);
      const float* row = tab.raw + (gl << LOGL);
      const float q = row[b];
      int rank = 0;
      if constexpr (keyed) {
        const uint64_t* krow = keys + (gl << LOGL);
        const uint64_t kb = krow[b];
#pragma unroll
        for (int b2 = 0; b2 < L; ++b2) rank += krow[b2] < kb;
      } else {
#pragma unroll
        for (int b2 = 0; b2 < L; ++b2) {
          const float q2 = row[b2];
          rank += (q2 < q) | ((q2 == q) & (b2 < b));
        }
      }
      tab.qs[(gl << LOGL) + rank] = q;
      tab.code_of[(gl << LOGL) + rank] = uint8_t(b);
      tab.pos_of[(gl << LOGL) + b] = uint8_t(rank);
    }
    wave_lds_sync();
  }
  if (has_nb) {
    // per code: the levels at sorted positions d-1, d, d+1 (clipped) and their codes
    for (int e = lane; e < ev; e += 64) {
      const int base = e & ~(L - 1);
      const int d = tab.pos_of[e];
      const int l = d > 0 ? d - 1 : 0;
      const int r = d < L - 1 ? d + 1 : L - 1;
      const uint32_t codes = uint32_t(tab.code_of[base + l]) | (uint32_t(tab.code_of[base + d]) << 8) |
                             (uint32_t(tab.code_of[base + r]) << 16);
      nb[e] = make_float4(tab.qs[base + l], tab.qs[base + d], tab.qs[base + r], __uint_as_float(codes));
    }
    wave_lds_sync();
  }

#pragma unroll
  for (int h = 0; h < CH; ++h) {
    const int lo = h * 512 + lane * kVec;  // this lane's first weight of chunk h, within the wave
    s0[h] = make_float4(0, 0, 0, 0);
    s1[h] = s0[h];
    prev[h] = make_uint2(0u, 0u);
    if (lo < nvalid) {
      const int64_t off = wbase + lo;
      w[h].load(a.W, off);
      const float4* sp = reinterpret_cast<const float4*>(a.s + off);
      s0[h] = sp[0];
      s1[h] = sp[1];
      if constexpr (MODE != 0) prev[h] = load8u8(a.codes, off);
    }
  }

#pragma unroll
  for (int h = 0; h < CH; ++h) {
    const int lo = h * 512 + lane * kVec;
    if (lo >= nvalid) break;  // later chunks start further out
    const int64_t off = wbase + lo;
    const int gl = lo >> g.logg;
    const float ds = s_ds[gl], zu = s_zu[gl], dl = s_dl[gl], tau = s_tau[gl];
    const float* q = tab.qs + (gl << LOGL);
    const float* qraw = tab.raw + (gl << LOGL);
    const float4* nbg = nb + (gl << LOGL);
    const uint8_t* code_of = tab.code_of + (gl << LOGL);
    const uint8_t* pos_of = tab.pos_of + (gl << LOGL);
    const float sv[8] = {s0[h].x, s0[h].y, s0[h].z, s0[h].w, s1[h].x, s1[h].y, s1[h].z, s1[h].w};
    float out[8];
    uint32_t cw[2] = {0u, 0u};
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float den = ds * sv[i];
      const float wb = w[h].get(i) / den + zu;
      float d, wt;
      uint32_t code;
      if constexpr (MODE == 0) {
        const int jj = nearest_full_k<LOGL>(q, wb, d);
        wt = q[jj];
        code = code_of[jj];
      } else if constexpr (MODE == 2) {
        code = byte_of(prev[h], i) & uint32_t(L - 1);
        wt = qraw[code];
        d = fabsf(wb - wt);
      } else {
        const uint32_t c0 = byte_of(prev[h], i) & uint32_t(L - 1);
        if constexpr (has_nb) {
          // first nearest of (d-1, d, d+1) in ascending order
          const float4 e4 = nbg[c0];
          const uint32_t cs = __float_as_uint(e4.w);
          float bd = fabsf(wb - e4.x);
          wt = e4.x;
          uint32_t sh = 0;
          const float dm = fabsf(wb - e4.y);
          if (dm < bd) { bd = dm; wt = e4.y; sh = 8; }
          const float dr = fabsf(wb - e4.z);
          if (dr < bd) { bd = dr; wt = e4.z; sh = 16; }
          d = bd;
          code = (cs >> sh) & 0xFFu;
        } else {
          const int jj = nearest_local(q, L, pos_of[c0], wb, d);
          wt = q[jj];
          code = code_of[jj];
        }
      }
      const uint32_t byte = code | (d > tau ? 0u : 0x80u);
      cw[i >> 2] |= byte << (8 * (i & 3));
      out[i] = dl * (wt - zu);
      if (a.resid) out[i] = out[i] - w[h].get(i);
    }
    store8<ODT>(a.W_hat, off, out);
    store8u8(a.codes, off, make_uint2(cw[0], cw[1]));
  }
}

// ---------------------------------------------------------------------------
// One pass per step over the weights: the straight-through backward of step
// t with its SGD update (the arithmetic of fq_bwd_kernel with update = 1,
// bit for bit), then the forward of step t + 1 with the updated s, alpha, z_B
// (the arithmetic of fq_fwd_kernel, bit for bit).  Each wavefront owns 512
// consecutive weights as in the forward: it loads dL/dWhat, W, s and the
// code bytes once, reduces the group sums with the backward's xor
// butterfly, writes the updated alpha and z_B of its groups to global memory
// and to its LDS region, builds the level tables from them, maps its weights
// and stores s, What (or the residual) and the new code bytes.  Per weight:
// 9 B read and 7 B written, against 10 + 13 for the two passes.
// ---------------------------------------------------------------------------
struct StepArgs {
  FwdArgs f;          // W, s (read), s_r, delta, z_u, alpha, z_b (read), codes, W_hat, resid
  float* s_out;       // = s (updated in place)
  float* alpha_out;   // = alpha
  float* z_b_out;     // = z_b
  const void* G;
  float lr_f, lr_b;
};

// Per-wave LDS of the fused pass: the forward's, plus alpha' and z_B' of each group.
__host__ __device__ inline size_t wave_step_lds_bytes(int logg, int k, bool nbt) {
  const size_t groups = size_t(512) >> logg;
  return wave_lds_bytes(logg, k, nbt, 1) + ((groups * (k + 1) * 4 + 15) & ~size_t(15));
}

template <int WDT, int GDT, int ODT, int MODE, int LOGL>
__global__ __launch_bounds__(kThreads) void fq_step_kernel(StepArgs sa) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const FwdArgs& a = sa.f;
  constexpr int L = 1 << LOGL;
  constexpr int K = LOGL;
  constexpr bool has_nb = MODE == 3;
  constexpr bool keyed = LOGL <= 4;
  const TileGeom& g = a.t;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int gw = 512 >> g.logg;
  const int ew = gw << LOGL;
  char* mine = smem + size_t(wave) * wave_step_lds_bytes(g.logg, LOGL, has_nb);
  LevelTables tab;
  char* p = carve_tables(tab, mine, ew);
  float4* nb = reinterpret_cast<float4*>(p);
  if (has_nb) p += 16 * size_t(ew);
  float* s_tau = reinterpret_cast<float*>(p) + 3 * gw;  // the forward's per-group slots; only tau is used
  uint64_t* keys = reinterpret_cast<uint64_t*>(s_tau + gw);
  float* s_par = reinterpret_cast<float*>(mine + wave_lds_bytes(g.logg, LOGL, has_nb, 1));  // [gw][K + 1]
  const int64_t wbase = (int64_t(blockIdx.x) * (blockDim.x >> 6) + wave) * 512;
  if (wbase >= g.N) return;
  const int nvalid = int(min<int64_t>(512, g.N - wbase));
  const int gv = nvalid >> g.logg;
  const int ev = gv << LOGL;
  const int64_t gid0 = wbase >> g.logg;
  const int lpg = 1 << (g.logg - 3);              // lanes per group
  const int lo = lane * kVec;
  const bool active = lo < nvalid;
  const int64_t off = wbase + lo;
  const int gl = active ? (lo >> g.logg) : 0;
  const int64_t gid = gid0 + gl;

  // loads: the chunk, then this lane's group parameters
  Raw8<WDT> w;
  float sv[8], G[8];
  uint2 cb = make_uint2(0u, 0u);
#pragma unroll
  for (int i = 0; i < 8; ++i) sv[i] = G[i] = 0.0f;
  float dl = 1.0f, sr = 1.0f, zu = 0.0f, zb = 0.0f, al[K];
#pragma unroll
  for (int b = 0; b < K; ++b) al[b] = 0.0f;
  if (active) {
    w.load(a.W, off);
    load8f(a.s, off, sv);
    load8<GDT>(sa.G, off, G);
    cb = load8u8(a.codes, off);
    dl = a.delta ? a.delta[gid] : 1.0f;
    sr = a.s_r ? a.s_r[uint32_t(gid) / uint32_t(g.gpr)] : 1.0f;
    zu = a.z_u ? a.z_u[gid] : 0.0f;
    zb = a.z_b[gid];
#pragma unroll
    for (int b = 0; b < K; ++b) al[b] = a.alpha[gid * K + b];
  }
  const float ds = dl * sr;

  // straight-through backward and the SGD update of s (fq_bwd_kernel's order)
  float S = 0.0f, Sa[K];
#pragma unroll
  for (int b = 0; b < K; ++b) Sa[b] = 0.0f;
  float sn[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const uint32_t byte = byte_of(cb, i);
    const bool m = (byte & 0x80u) != 0u;
    const float gg = G[i];
    S += gg;
#pragma unroll
    for (int b = 0; b < K; ++b) Sa[b] += ((byte >> b) & 1u) ? gg : -gg;
    const float x = w.get(i) * __builtin_amdgcn_rcpf(ds * sv[i]);
    const float gs = m ? -(dl * gg) * x * __builtin_amdgcn_rcpf(sv[i]) : 0.0f;
    sn[i] = sv[i] - sa.lr_f * gs;
  }
  for (int msk = lpg >> 1; msk >= 1; msk >>= 1) {
    S += __shfl_xor(S, msk, 64);
#pragma unroll
    for (int b = 0; b < K; ++b) Sa[b] += __shfl_xor(Sa[b], msk, 64);
  }
  // updated alpha', z_B' (every lane of a group holds the same sums); the
  // group's first lane publishes them
  if (active && (lane & (lpg - 1)) == 0) {
    float* par = s_par + gl * (K + 1);
#pragma unroll
    for (int b = 0; b < K; ++b) {
      const float an = al[b] - sa.lr_b * (dl * Sa[b]);
      sa.alpha_out[gid * K + b] = an;
      par[b] = an;
    }
    const float zn = zb - sa.lr_b * (dl * S);
    sa.z_b_out[gid] = zn;
    par[K] = zn;
  }
  wave_lds_sync();
  // level tables of the wave's groups from alpha', z_B' (fq_fwd_kernel's order)
  for (int e = lane; e < ev; e += 64) {
    const int gg = e >> LOGL;
    const float* par = s_par + gg * (K + 1);
    const float q = level_value_k<LOGL>(par, par[K], e & (L - 1));
    tab.raw[e] = q;
    if constexpr (keyed && MODE != 2) keys[e] = level_key(q, e & (L - 1));
  }
  for (int gg = lane; gg < gv; gg += 64) s_tau[gg] = tau_k<LOGL>(s_par + gg * (K + 1));
  wave_lds_sync();
  if constexpr (MODE != 2) {
    for (int e = lane; e < ev; e += 64) {
      const int gg = e >> LOGL;
      const int b = e & (L - 1);
      const float* row = tab.raw + (gg << LOGL);
      const float q = row[b];
      int rank = 0;
      if constexpr (keyed) {
        const uint64_t* krow = keys + (gg << LOGL);
        const uint64_t kb = krow[b];
#pragma unroll
        for (int b2 = 0; b2 < L; ++b2) rank += krow[b2] < kb;
      } else {
#pragma unroll
        for (int b2 = 0; b2 < L; ++b2) {
          const float q2 = row[b2];
          rank += (q2 < q) | ((q2 == q) & (b2 < b));
        }
      }
      tab.qs[(gg << LOGL) + rank] = q;
      tab.code_of[(gg << LOGL) + rank] = uint8_t(b);
      tab.pos_of[(gg << LOGL) + b] = uint8_t(rank);
    }
    wave_lds_sync();
  }
  if (has_nb) {
    for (int e = lane; e < ev; e += 64) {
      const int base = e & ~(L - 1);
      const int d = tab.pos_of[e];
      const int l = d > 0 ? d - 1 : 0;
      const int r = d < L - 1 ? d + 1 : L - 1;
      const uint32_t codes = uint32_t(tab.code_of[base + l]) | (uint32_t(tab.code_of[base + d]) << 8) |
                             (uint32_t(tab.code_of[base + r]) << 16);
      nb[e] = make_float4(tab.qs[base + l], tab.qs[base + d], tab.qs[base + r], __uint_as_float(codes));
    }
    wave_lds_sync();
  }
  if (!active) return;
  store8f(sa.s_out, off, sn);
  // the next step's forward on the updated parameters
  const float tau = s_tau[gl];
  const float* q = tab.qs + (gl << LOGL);
  const float* qraw = tab.raw + (gl << LOGL);
  const float4* nbg = nb + (gl << LOGL);
  const uint8_t* code_of = tab.code_of + (gl << LOGL);
  float out[8];
  uint32_t cw[2] = {0u, 0u};
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const float den = ds * sn[i];
    const float wb = w.get(i) / den + zu;
    float d, wt;
    uint32_t code;
    if constexpr (MODE == 0) {
      const int jj = nearest_full_k<LOGL>(q, wb, d);
      wt = q[jj];
      code = code_of[jj];
    } else if constexpr (MODE == 2) {
      code = byte_of(cb, i) & uint32_t(L - 1);
      wt = qraw[code];
      d = fabsf(wb - wt);
    } else {
      const float4 e4 = nbg[byte_of(cb, i) & uint32_t(L - 1)];
      const uint32_t cs = __float_as_uint(e4.w);
      float bd = fabsf(wb - e4.x);
      wt = e4.x;
      uint32_t sh = 0;
      const float dm = fabsf(wb - e4.y);
      if (dm < bd) { bd = dm; wt = e4.y; sh = 8; }
      const float dr = fabsf(wb - e4.z);
      if (dr < bd) { bd = dr; wt = e4.z; sh = 16; }
      d = bd;
      code = (cs >> sh) & 0xFFu;
    }
    const uint32_t byte = code | (d > tau ? 0u : 0x80u);
    cw[i >> 2] |= byte << (8 * (i & 3));
    out[i] = dl * (wt - zu);
    if (a.resid) out[i] = out[i] - w.get(i);
  }
  store8<ODT>(a.W_hat, off, out);
  store8u8(a.codes, off, make_uint2(cw[0], cw[1]));
}

// ---------------------------------------------------------------------------
// Fold (Theorem 1): alpha* = Delta alpha, z* = Delta (z_B - z_U); codes by
// FULL mapping of wbar (code_src 0) or of the raw w against the folded
// levels (code_src 1, Eq. (4) as printed).
// ---------------------------------------------------------------------------
struct FoldArgs {
  TileGeom t;
  const void* W;
  const float* s;
  const float* s_r;
  const float* delta;
  const float* z_u;
  const float* alpha;
  const float* z_b;
  float* alpha_star;
  float* z_star;
  uint8_t* codes;
  int code_src;
};

// LDS: tables, per-group (Delta s_r, z_U, z*) and the tile's alpha* (k per group)
static size_t fold_lds_bytes(const TileGeom& t) {
  return tile_lds_bytes(t) + 4 * size_t(t.tile_groups) * size_t(t.k);
}

template <int WDT>
__global__ __launch_bounds__(kThreads) void fold_kernel(FoldArgs a) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const TileGeom& g = a.t;
  LevelTables tab;
  float* s_ds = reinterpret_cast<float*>(carve_tables(tab, smem, g.tile_groups << g.logL));
  float* s_zu = s_ds + g.tile_groups;
  float* s_zst = s_zu + g.tile_groups;
  float* s_alpha = s_zst + 2 * g.tile_groups;  // tile_groups * k entries
  const int64_t Gn = g.N >> g.logg;
  const int64_t gid0 = int64_t(blockIdx.x) * g.tile_groups;
  const int ng = int(min<int64_t>(g.tile_groups, Gn - gid0));
  const int lane_w = threadIdx.x * kVec;
  const int64_t off = (gid0 << g.logg) + lane_w;

  for (int gl = threadIdx.x; gl < ng; gl += blockDim.x) {
    const int64_t gid = gid0 + gl;
    const float dl = a.delta ? a.delta[gid] : 1.0f;
    const float zu = a.z_u ? a.z_u[gid] : 0.0f;
    const float sr = a.s_r ? a.s_r[uint32_t(gid) / uint32_t(g.gpr)] : 1.0f;
    const float zst = dl * (a.z_b[gid] - zu);
    for (int i = 0; i < g.k; ++i) {
      const float as = dl * a.alpha[gid * g.k + i];
      a.alpha_star[gid * g.k + i] = as;
      s_alpha[gl * g.k + i] = as;
    }
    a.z_star[gid] = zst;
    s_zst[gl] = zst;
    s_ds[gl] = dl * sr;
    s_zu[gl] = zu;
  }
  if (a.codes == nullptr) return;  // uniform across the grid
  __syncthreads();
  if (a.code_src == 0) {
    build_tables(tab, a.alpha, a.z_b, gid0, ng, g.k, g.logL);
  } else {
    const int L = 1 << g.logL;
    for (int e = threadIdx.x; e < (ng << g.logL); e += blockDim.x) {
      const int gl = e >> g.logL;
      tab.raw[e] = level_value(s_alpha + gl * g.k, s_zst[gl], g.k, e & (L - 1));
    }
    __syncthreads();
    sort_tables(tab, ng, g.logL);
  }
  if (lane_w >= (ng << g.logg)) return;
  const int glw = lane_w >> g.logg;
  float w[8], sv[8];
  load8<WDT>(a.W, off, w);
  if (a.code_src == 0) load8f(a.s, off, sv);
  const float* q = tab.qs + (glw << g.logL);
  const uint8_t* code_of = tab.code_of + (glw << g.logL);
  uint32_t cw[2] = {0u, 0u};
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    float x = w[i];
    if (a.code_src == 0) {
      const float den = s_ds[glw] * sv[i];
      x = x / den + s_zu[glw];
    }
    float d;
    const int j = nearest_full(q, g.logL, x, d);
    cw[i >> 2] |= uint32_t(code_of[j]) << (8 * (i & 3));
  }
  store8u8(a.codes, off, make_uint2(cw[0], cw[1]));
}

// ---------------------------------------------------------------------------
// Binary-coding dequantization R_B(C; Theta) = C alpha + z_B 1_g.
// ---------------------------------------------------------------------------
struct DequantArgs {
  TileGeom t;
  const uint8_t* codes;
  const float* alpha;
  const float* z_b;
  void* W_out;
};

template <int ODT>
__global__ __launch_bounds__(kThreads) void dequant_kernel(DequantArgs a) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  float* raw = reinterpret_cast<float*>(smem);
  const TileGeom& g = a.t;
  const int64_t Gn = g.N >> g.logg;
  const int64_t gid0 = int64_t(blockIdx.x) * g.tile_groups;
  const int ng = int(min<int64_t>(g.tile_groups, Gn - gid0));
  const int L = 1 << g.logL;
  for (int e = threadIdx.x; e < (ng << g.logL); e += blockDim.x) {
    const int64_t gid = gid0 + (e >> g.logL);
    raw[e] = level_value(a.alpha + gid * g.k, a.z_b[gid], g.k, e & (L - 1));
  }
  __syncthreads();
  const int lane_w = threadIdx.x * kVec;
  if (lane_w >= (ng << g.logg)) return;
  const int64_t off = (gid0 << g.logg) + lane_w;
  const uint2 cb = load8u8(a.codes, off);
  const float* row = raw + ((lane_w >> g.logg) << g.logL);
  float out[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) out[i] = row[byte_of(cb, i) & uint32_t(L - 1)];
  store8<ODT>(a.W_out, off, out);
}

// ---------------------------------------------------------------------------
// Greedy start: per group r = wbar - z_B; for each bit, c = sign(r),
// alpha = mean |r|, r -= alpha c.  A group of g weights is g/8 lanes of one
// wavefront; group sums use a fixed xor-butterfly order.
// ---------------------------------------------------------------------------
struct GreedyArgs {
  TileGeom t;
  const void* W;
  const float* s;
  const float* s_r;
  const float* delta;
  const float* z_u;
  const float* z_b;
  float* alpha;
};

template <int WDT>
__global__ __launch_bounds__(kThreads) void greedy_kernel(GreedyArgs a) {
  const TileGeom& g = a.t;
  const int64_t chunk = int64_t(blockIdx.x) * kThreads + threadIdx.x;
  const int64_t off = chunk * kVec;
  const bool active = off < g.N;
  const int lpg = 1 << (g.logg - 3);  // lanes per group (<= 64)
  const int64_t gid = active ? (off >> g.logg) : 0;
  float r[8];
  if (active) {
    float w[8], sv[8];
    load8<WDT>(a.W, off, w);
    load8f(a.s, off, sv);
    const float dl = a.delta ? a.delta[gid] : 1.0f;
    const float sr = a.s_r ? a.s_r[uint32_t(gid) / uint32_t(g.gpr)] : 1.0f;
    const float zu = a.z_u ? a.z_u[gid] : 0.0f;
    const float zb = a.z_b[gid];
    const float ds = dl * sr;
#pragma unroll
    for (int i = 0; i < 8; ++i) r[i] = (w[i] / (ds * sv[i]) + zu) - zb;
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i) r[i] = 0.0f;
  }
  const float inv_g = 1.0f / float(1 << g.logg);  // exact power of two
  for (int b = 0; b < g.k; ++b) {
    float acc = 0.0f;
#pragma unroll
    for (int i = 0; i < 8; ++i) acc += fabsf(r[i]);
    for (int m = lpg >> 1; m >= 1; m >>= 1) acc += __shfl_xor(acc, m, 64);
    const float al = acc * inv_g;
#pragma unroll
    for (int i = 0; i < 8; ++i) r[i] = r[i] >= 0.0f ? r[i] - al : r[i] + al;
    if (active && (threadIdx.x & (lpg - 1)) == 0) a.alpha[gid * g.k + b] = al;
  }
}

// ---------------------------------------------------------------------------
// Groups larger than 512 weights: the paper's per-row groups for 7B / 8B
// models (g = C, e.g. 4096, 11008 or 14336 weights), or any multiple of 8
// that divides C.  One workgroup of 256 lanes per group reads the group's
// parameters once, builds its sorted level table (at most 128 levels) in
// LDS, and streams the group's weights 8 per lane, two chunks per lane in
// flight.  The per-weight arithmetic is that of fq_fwd_kernel and the fold,
// so codes and What are the same bit for bit.
// ---------------------------------------------------------------------------
constexpr int kBigThreads = 256;

struct BigArgs {
  int64_t Gn;
  int g, gpr, k;
  const void* W;
  const float* s;
  const float* s_r;
  const float* delta;
  const float* z_u;
  const float* alpha;
  const float* z_b;
  uint8_t* codes;
  void* W_hat;
  int resid;
  // fold
  float* alpha_star;
  float* z_star;
  int code_src;
};

// Sorted table of one group from its L raw levels (raw[b] already written by
// the caller and made visible by a barrier): qs[pos], code_of[pos],
// pos_of[b], sort key (value, code); with NB also the neighbour entries of
// the local mapping.  Ends with a barrier.
template <int LOGL, bool NB>
__device__ __forceinline__ void big_sort(const float* raw, float* qs, uint8_t* code_of, uint8_t* pos_of, float4* nb) {
  constexpr int L = 1 << LOGL;
  const int t = threadIdx.x;
  if (t < L) {
    const uint64_t kb = level_key(raw[t], t);
    int rank = 0;
    for (int b2 = 0; b2 < L; ++b2) rank += level_key(raw[b2], b2) < kb;
    qs[rank] = raw[t];
    code_of[rank] = uint8_t(t);
    pos_of[t] = uint8_t(rank);
  }
  __syncthreads();
  if constexpr (NB) {
    if (t < L) {
      const int d = pos_of[t];
      const int l = d > 0 ? d - 1 : 0;
      const int r = d < L - 1 ? d + 1 : L - 1;
      const uint32_t cs = uint32_t(code_of[l]) | (uint32_t(code_of[d]) << 8) | (uint32_t(code_of[r]) << 16);
      nb[t] = make_float4(qs[l], qs[d], qs[r], __uint_as_float(cs));
    }
    __syncthreads();
  }
}

// MODE: 0 FULL, 2 FROZEN, 3 LOCAL (neighbour entries).
template <int WDT, int ODT, int MODE, int LOGL>
__global__ __launch_bounds__(kBigThreads) void fq_fwd_big_kernel(BigArgs a) {
  constexpr int L = 1 << LOGL;
  __shared__ float raw[L], qs[L];
  __shared__ uint8_t code_of[L], pos_of[L];
  __shared__ float4 nb[MODE == 3 ? L : 1];
  const int64_t gid = blockIdx.x;
  const float* alpha_g = a.alpha + gid * LOGL;
  if (threadIdx.x < L) raw[threadIdx.x] = level_value_k<LOGL>(alpha_g, a.z_b[gid], threadIdx.x);
  __syncthreads();
  if constexpr (MODE != 2) big_sort<LOGL, MODE == 3>(raw, qs, code_of, pos_of, nb);
  const float dl = a.delta ? a.delta[gid] : 1.0f;
  const float sr = a.s_r ? a.s_r[gid / a.gpr] : 1.0f;
  const float zu = a.z_u ? a.z_u[gid] : 0.0f;
  const float ds = dl * sr;
  const float tau = tau_k<LOGL>(alpha_g);
  const int nch = a.g >> 3;
  const int64_t base = gid * a.g;
  for (int c0 = threadIdx.x; c0 < nch; c0 += 2 * kBigThreads) {
    Raw8<WDT> w[2];
    float4 s0[2], s1[2];
    uint2 prev[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int c = c0 + h * kBigThreads;
      s0[h] = s1[h] = make_float4(0, 0, 0, 0);
      prev[h] = make_uint2(0u, 0u);
      if (c < nch) {
        const int64_t off = base + int64_t(c) * kVec;
        w[h].load(a.W, off);
        const float4* sp = reinterpret_cast<const float4*>(a.s + off);
        s0[h] = sp[0];
        s1[h] = sp[1];
        if constexpr (MODE != 0) prev[h] = load8u8(a.codes, off);
      }
    }
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int c = c0 + h * kBigThreads;
      if (c >= nch) break;
      const int64_t off = base + int64_t(c) * kVec;
      const float sv[8] = {s0[h].x, s0[h].y, s0[h].z, s0[h].w, s1[h].x, s1[h].y, s1[h].z, s1[h].w};
      float out[8];
      uint32_t cw[2] = {0u, 0u};
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float den = ds * sv[i];
        const float wb = w[h].get(i) / den + zu;
        float d, wt;
        uint32_t code;
        if constexpr (MODE == 0) {
          const int jj = nearest_full_k<LOGL>(qs, wb, d);
          wt = qs[jj];
          code = code_of[jj];
        } else if constexpr (MODE == 2) {
          code = byte_of(prev[h], i) & uint32_t(L - 1);
          wt = raw[code];
          d = fabsf(wb - wt);
        } else {
          const float4 e4 = nb[byte_of(prev[h], i) & uint32_t(L - 1)];
          const uint32_t cs = __float_as_uint(e4.w);
          float bd = fabsf(wb - e4.x);
          wt = e4.x;
          uint32_t sh = 0;
          const float dm = fabsf(wb - e4.y);
          if (dm < bd) { bd = dm; wt = e4.y; sh = 8; }
          const float dr = fabsf(wb - e4.z);
          if (dr < bd) { bd = dr; wt = e4.z; sh = 16; }
          d = bd;
          code = (cs >> sh) & 0xFFu;
        }
        const uint32_t byte = code | (d > tau ? 0u : 0x80u);
        cw[i >> 2] |= byte << (8 * (i & 3));
        out[i] = dl * (wt - zu);
        if (a.resid) out[i] = out[i] - w[h].get(i);
      }
      store8<ODT>(a.W_hat, off, out);
      store8u8(a.codes, off, make_uint2(cw[0], cw[1]));
    }
  }
}

// The fused step for one large group (g up to 16384): the straight-through
// backward with the SGD update (fq_bwd_big_kernel's arithmetic and order:
// each lane's chunks c = lane, lane + 256, ..., the fixed xor butterfly, the
// four wavefront sums pairwise), then the forward of the next step with the
// updated s, alpha, z_B (fq_fwd_big_kernel's, bit for bit).  A lane keeps
// its chunks' W, updated s and code bytes in registers between the two
// halves, so each weight's W, s, dL/dWhat and code are read once.
constexpr int kStepBigChunks = 8;  // chunks per lane: g <= 256 * 8 * 8

template <int WDT, int GDT, int ODT, int MODE, int LOGL>
__global__ __launch_bounds__(kBigThreads) void fq_step_big_kernel(BigArgs a, const void* __restrict__ G, float lr_f,
                                                                  float lr_b) {
  constexpr int L = 1 << LOGL, K = LOGL, CPT = kStepBigChunks;
  __shared__ float raw[L], qs[L];
  __shared__ uint8_t code_of[L], pos_of[L];
  __shared__ float4 nb[MODE == 3 ? L : 1];
  __shared__ float red[4][K + 1];
  __shared__ float par[K + 1];  // alpha', z_B'
  const int64_t gid = blockIdx.x;
  const float dl = a.delta ? a.delta[gid] : 1.0f;
  const float sr = a.s_r ? a.s_r[gid / a.gpr] : 1.0f;
  const float zu = a.z_u ? a.z_u[gid] : 0.0f;
  const float ds = dl * sr;
  const int nch = a.g >> 3;
  const int64_t base = gid * a.g;
  float* s_io = const_cast<float*>(a.s);

  // backward with the update of s; this lane's group sums
  Raw8<WDT> w[CPT];
  float sv[CPT][8];
  uint2 cb[CPT];
  float S = 0.0f, Sa[K];
#pragma unroll
  for (int b = 0; b < K; ++b) Sa[b] = 0.0f;
#pragma unroll
  for (int u = 0; u < CPT; ++u) {
    const int c = int(threadIdx.x) + u * kBigThreads;
    cb[u] = make_uint2(0u, 0u);
    if (c < nch) {
      const int64_t off = base + int64_t(c) * kVec;
      w[u].load(a.W, off);
      load8f(a.s, off, sv[u]);
      float gv[8];
      load8<GDT>(G, off, gv);
      cb[u] = load8u8(a.codes, off);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const uint32_t byte = byte_of(cb[u], i);
        const bool m = (byte & 0x80u) != 0u;
        const float gg = gv[i];
        S += gg;
#pragma unroll
        for (int b = 0; b < K; ++b) Sa[b] += ((byte >> b) & 1u) ? gg : -gg;
        const float x = w[u].get(i) * __builtin_amdgcn_rcpf(ds * sv[u][i]);
        const float gs = m ? -(dl * gg) * x * __builtin_amdgcn_rcpf(sv[u][i]) : 0.0f;
        sv[u][i] = sv[u][i] - lr_f * gs;
      }
      store8f(s_io, off, sv[u]);
    }
  }
  for (int msk = 32; msk >= 1; msk >>= 1) {
    S += __shfl_xor(S, msk, 64);
#pragma unroll
    for (int b = 0; b < K; ++b) Sa[b] += __shfl_xor(Sa[b], msk, 64);
  }
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    red[wave][0] = S;
#pragma unroll
    for (int b = 0; b < K; ++b) red[wave][1 + b] = Sa[b];
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    auto sum4 = [&](int j) { return (red[0][j] + red[1][j]) + (red[2][j] + red[3][j]); };
    float* alpha = const_cast<float*>(a.alpha) + gid * K;
    float* z_b = const_cast<float*>(a.z_b);
#pragma unroll
    for (int b = 0; b < K; ++b) {
      const float an = alpha[b] - lr_b * (dl * sum4(1 + b));
      alpha[b] = an;
      par[b] = an;
    }
    const float zn = z_b[gid] - lr_b * (dl * sum4(0));
    z_b[gid] = zn;
    par[K] = zn;
  }
  __syncthreads();

  // forward of the next step on the updated parameters
  if (threadIdx.x < L) raw[threadIdx.x] = level_value_k<LOGL>(par, par[K], threadIdx.x);
  __syncthreads();
  if constexpr (MODE != 2) big_sort<LOGL, MODE == 3>(raw, qs, code_of, pos_of, nb);
  const float tau = tau_k<LOGL>(par);
#pragma unroll
  for (int u = 0; u < CPT; ++u) {
    const int c = int(threadIdx.x) + u * kBigThreads;
    if (c >= nch) break;
    const int64_t off = base + int64_t(c) * kVec;
    float out[8];
    uint32_t cw[2] = {0u, 0u};
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float den = ds * sv[u][i];
      const float wb = w[u].get(i) / den + zu;
      float d, wt;
      uint32_t code;
      if constexpr (MODE == 0) {
        const int jj = nearest_full_k<LOGL>(qs, wb, d);
        wt = qs[jj];
        code = code_of[jj];
      } else if constexpr (MODE == 2) {
        code = byte_of(cb[u], i) & uint32_t(L - 1);
        wt = raw[code];
        d = fabsf(wb - wt);
      } else {
        const float4 e4 = nb[byte_of(cb[u], i) & uint32_t(L - 1)];
        const uint32_t cs = __float_as_uint(e4.w);
        float bd = fabsf(wb - e4.x);
        wt = e4.x;
        uint32_t sh = 0;
        const float dm = fabsf(wb - e4.y);
        if (dm < bd) { bd = dm; wt = e4.y; sh = 8; }
        const float dr = fabsf(wb - e4.z);
        if (dr < bd) { bd = dr; wt = e4.z; sh = 16; }
        d = bd;
        code = (cs >> sh) & 0xFFu;
      }
      const uint32_t byte = code | (d > tau ? 0u : 0x80u);
      cw[i >> 2] |= byte << (8 * (i & 3));
      out[i] = dl * (wt - zu);
      if (a.resid) out[i] = out[i] - w[u].get(i);
    }
    store8<ODT>(a.W_hat, off, out);
    store8u8(a.codes, off, make_uint2(cw[0], cw[1]));
  }
}

// Fold of one large group: alpha* = Delta alpha, z* = Delta (z_B - z_U), and
// the codes of the FULL mapping of wbar (code_src 0) or of the raw w against
// the folded levels (code_src 1), as fold_kernel computes them.
template <int WDT, int LOGL>
__global__ __launch_bounds__(kBigThreads) void fold_big_kernel(BigArgs a) {
  constexpr int L = 1 << LOGL;
  __shared__ float raw[L], qs[L], s_alpha[LOGL];
  __shared__ uint8_t code_of[L], pos_of[L];
  const int64_t gid = blockIdx.x;
  const float dl = a.delta ? a.delta[gid] : 1.0f;
  const float zu = a.z_u ? a.z_u[gid] : 0.0f;
  const float sr = a.s_r ? a.s_r[gid / a.gpr] : 1.0f;
  const float zst = dl * (a.z_b[gid] - zu);
  if (threadIdx.x < LOGL) {
    const float as = dl * a.alpha[gid * LOGL + threadIdx.x];
    a.alpha_star[gid * LOGL + threadIdx.x] = as;
    s_alpha[threadIdx.x] = as;
  }
  if (threadIdx.x == 0) a.z_star[gid] = zst;
  if (a.codes == nullptr) return;  // uniform across the grid
  __syncthreads();
  if (threadIdx.x < L) {
    raw[threadIdx.x] = a.code_src == 0 ? level_value_k<LOGL>(a.alpha + gid * LOGL, a.z_b[gid], threadIdx.x)
                                       : level_value_k<LOGL>(s_alpha, zst, threadIdx.x);
  }
  __syncthreads();
  big_sort<LOGL, false>(raw, qs, code_of, pos_of, nullptr);
  const float ds = dl * sr;
  const int nch = a.g >> 3;
  const int64_t base = gid * a.g;
  for (int c = threadIdx.x; c < nch; c += kBigThreads) {
    const int64_t off = base + int64_t(c) * kVec;
    float w[8], sv[8];
    load8<WDT>(a.W, off, w);
    if (a.code_src == 0) load8f(a.s, off, sv);
    uint32_t cw[2] = {0u, 0u};
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      float x = w[i];
      if (a.code_src == 0) {
        const float den = ds * sv[i];
        x = x / den + zu;
      }
      float d;
      const int j = nearest_full_k<LOGL>(qs, x, d);
      cw[i >> 2] |= uint32_t(code_of[j]) << (8 * (i & 3));
    }
    store8u8(a.codes, off, make_uint2(cw[0], cw[1]));
  }
}

// Dequantization of one large group: W_out[j] = q(code_j).
template <int ODT>
__global__ __launch_bounds__(kBigThreads) void dequant_big_kernel(BigArgs a) {
  __shared__ float raw[128];
  const int64_t gid = blockIdx.x;
  const int L = 1 << a.k;
  if (int(threadIdx.x) < L) raw[threadIdx.x] = level_value(a.alpha + gid * a.k, a.z_b[gid], a.k, threadIdx.x);
  __syncthreads();
  const int nch = a.g >> 3;
  const int64_t base = gid * a.g;
  for (int c = threadIdx.x; c < nch; c += kBigThreads) {
    const int64_t off = base + int64_t(c) * kVec;
    const uint2 cb = load8u8(a.codes, off);
    float out[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) out[i] = raw[byte_of(cb, i) & uint32_t(L - 1)];
    store8<ODT>(a.W_hat, off, out);
  }
}

// Sum of v over the workgroup's 256 lanes in a fixed order: xor butterfly in
// each wavefront, then the four wavefront sums pairwise.  Every lane gets the
// result.
__device__ __forceinline__ float big_block_sum(float v, float* red) {
  for (int msk = 32; msk >= 1; msk >>= 1) v += __shfl_xor(v, msk, 64);
  __syncthreads();  // red is free (earlier readers are done)
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  return (red[0] + red[1]) + (red[2] + red[3]);
}

// Greedy start on one large group: per bit, alpha = (sum of |r|) / g with the
// workgroup sum above, r recomputed from w and s for every bit (set-up only,
// so the group need not stay in registers).
template <int WDT>
__global__ __launch_bounds__(kBigThreads) void greedy_big_kernel(BigArgs a) {
  __shared__ float red[4];
  __shared__ float s_al[8];
  const int64_t gid = blockIdx.x;
  const float dl = a.delta ? a.delta[gid] : 1.0f;
  const float sr = a.s_r ? a.s_r[gid / a.gpr] : 1.0f;
  const float zu = a.z_u ? a.z_u[gid] : 0.0f;
  const float zb = a.z_b[gid];
  const float ds = dl * sr;
  const int nch = a.g >> 3;
  const int64_t base = gid * a.g;
  for (int b = 0; b < a.k; ++b) {
    float acc = 0.0f;
    for (int c = threadIdx.x; c < nch; c += kBigThreads) {
      const int64_t off = base + int64_t(c) * kVec;
      float w[8], sv[8];
      load8<WDT>(a.W, off, w);
      load8f(a.s, off, sv);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        float r = (w[i] / (ds * sv[i]) + zu) - zb;
        for (int j = 0; j < b; ++j) r = r >= 0.0f ? r - s_al[j] : r + s_al[j];
        acc += fabsf(r);
      }
    }
    const float al = big_block_sum(acc, red) / float(a.g);
    if (threadIdx.x == 0) {
      s_al[b] = al;
      a.alpha_star[gid * a.k + b] = al;  // the greedy alpha (the launcher passes its output here)
    }
    __syncthreads();
  }
}

static BigArgs big_args(int64_t R, int64_t C, int k, int g) {
  BigArgs b{};
  b.Gn = R * C / g;
  b.g = g;
  b.gpr = int(C / g);
  b.k = k;
  return b;
}

template <int WD, int OD, int MD>
static hipError_t launch_fwd_big(const BigArgs& a, hipStream_t st) {
  const dim3 grid(unsigned(a.Gn)), block(kBigThreads);
  switch (a.k) {
    case 1: hipLaunchKernelGGL((fq_fwd_big_kernel<WD, OD, MD, 1>), grid, block, 0, st, a); break;
    case 2: hipLaunchKernelGGL((fq_fwd_big_kernel<WD, OD, MD, 2>), grid, block, 0, st, a); break;
    case 3: hipLaunchKernelGGL((fq_fwd_big_kernel<WD, OD, MD, 3>), grid, block, 0, st, a); break;
    case 4: hipLaunchKernelGGL((fq_fwd_big_kernel<WD, OD, MD, 4>), grid, block, 0, st, a); break;
    case 5: hipLaunchKernelGGL((fq_fwd_big_kernel<WD, OD, MD, 5>), grid, block, 0, st, a); break;
    case 6: hipLaunchKernelGGL((fq_fwd_big_kernel<WD, OD, MD, 6>), grid, block, 0, st, a); break;
    default: hipLaunchKernelGGL((fq_fwd_big_kernel<WD, OD, MD, 7>), grid, block, 0, st, a); break;
  }
  return hipGetLastError();
}

static hipError_t launch_fq_fwd_big(const FqFwdLaunch& p, hipStream_t st) {
  BigArgs a = big_args(p.R, p.C, p.k, p.g);
  a.W = p.W; a.s = p.s; a.s_r = p.s_r; a.delta = p.delta; a.z_u = p.z_u;
  a.alpha = p.alpha; a.z_b = p.z_b; a.codes = p.codes; a.W_hat = p.W_hat;
  a.resid = p.resid;
#define UQ_FWDB(WD, OD, MD, MK) \
  if (p.w_dtype == WD && p.w_hat_dtype == OD && p.mode == MD) return launch_fwd_big<WD, OD, MK>(a, st);
  UQ_FWDB(BF16, BF16, 0, 0) UQ_FWDB(BF16, BF16, 1, 3) UQ_FWDB(BF16, BF16, 2, 2)
  UQ_FWDB(BF16, F32, 0, 0) UQ_FWDB(BF16, F32, 1, 3) UQ_FWDB(BF16, F32, 2, 2)
  UQ_FWDB(F32, BF16, 0, 0) UQ_FWDB(F32, BF16, 1, 3) UQ_FWDB(F32, BF16, 2, 2)
  UQ_FWDB(F32, F32, 0, 0) UQ_FWDB(F32, F32, 1, 3) UQ_FWDB(F32, F32, 2, 2)
#undef UQ_FWDB
  return hipErrorInvalidValue;
}

template <int WD>
static hipError_t launch_fold_big(const BigArgs& a, hipStream_t st) {
  const dim3 grid(unsigned(a.Gn)), block(kBigThreads);
  switch (a.k) {
    case 1: hipLaunchKernelGGL((fold_big_kernel<WD, 1>), grid, block, 0, st, a); break;
    case 2: hipLaunchKernelGGL((fold_big_kernel<WD, 2>), grid, block, 0, st, a); break;
    case 3: hipLaunchKernelGGL((fold_big_kernel<WD, 3>), grid, block, 0, st, a); break;
    case 4: hipLaunchKernelGGL((fold_big_kernel<WD, 4>), grid, block, 0, st, a); break;
    case 5: hipLaunchKernelGGL((fold_big_kernel<WD, 5>), grid, block, 0, st, a); break;
    case 6: hipLaunchKernelGGL((fold_big_kernel<WD, 6>), grid, block, 0, st, a); break;
    default: hipLaunchKernelGGL((fold_big_kernel<WD, 7>), grid, block, 0, st, a); break;
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------
// Tile of `chunks` x 2048 weights, capped so the level tables stay within
// kMaxEntries entries.
static TileGeom make_geom(int64_t R, int64_t C, int k, int g, int chunks) {
  TileGeom t;
  t.N = R * C;
  t.logg = __builtin_ctz(unsigned(g));
  t.logL = k;
  t.k = k;
  t.gpr = int(C / g);
  int tg = (chunks * kTile) >> t.logg;
  const int by_lds = kMaxEntries >> k;
  if (tg > by_lds) tg = by_lds;
  if (tg < 1) tg = 1;
  t.tile_groups = tg;
  return t;
}

static unsigned grid_of(const TileGeom& t) {
  const int64_t Gn = t.N >> t.logg;
  return unsigned((Gn + t.tile_groups - 1) / t.tile_groups);
}

// Waves per workgroup: up to 4, as many as fit 64 KB of dynamic LDS; a
// single wave above that (tiny groups with many levels) opts in to the
// larger LDS of gfx950.
static int fwd_waves_per_block(size_t wave_bytes) {
  int wpb = int(65536 / wave_bytes);
  return wpb < 1 ? 1 : wpb > 4 ? 4 : wpb;
}

template <typename Kern>
static hipError_t launch_fwd_kern(Kern kern, const FwdArgs& a, size_t wave_bytes, int ch, hipStream_t st) {
  const int wpb = fwd_waves_per_block(wave_bytes);
  const size_t lds = size_t(wpb) * wave_bytes;
  if (lds > 65536) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
    if (e != hipSuccess) return e;
  }
  const int64_t per_wave = 512 * int64_t(ch);
  const int64_t waves = (a.t.N + per_wave - 1) / per_wave;
  hipLaunchKernelGGL(kern, dim3(unsigned((waves + wpb - 1) / wpb)), dim3(64 * wpb), lds, st, a);
  return hipGetLastError();
}

// One chunk per wavefront.  Two (twice the loads in flight per wave, half
// the wavefronts) measured faster on a layer whose working set stays in the
// last-level cache across repeated launches, and slower inside the training
// step, where every launch streams its chunk from HBM (fq_fwd 33.7 against
// 34.3 us at 4096 x 4096).
template <int WD, int OD, int MD, int LOGL>
static hipError_t launch_fwd_l(const FwdArgs& a, hipStream_t st) {
  constexpr bool nbt = MD == 3;
  return launch_fwd_kern(fq_fwd_kernel<WD, OD, MD, LOGL, 1>, a, wave_lds_bytes(a.t.logg, LOGL, nbt, 1), 1, st);
}

template <int WD, int OD, int MD>
static hipError_t launch_fwd_m(const FwdArgs& a, int k, hipStream_t st) {
  switch (k) {
    case 1: return launch_fwd_l<WD, OD, MD, 1>(a, st);
    case 2: return launch_fwd_l<WD, OD, MD, 2>(a, st);
    case 3: return launch_fwd_l<WD, OD, MD, 3>(a, st);
    case 4: return launch_fwd_l<WD, OD, MD, 4>(a, st);
    case 5: return launch_fwd_l<WD, OD, MD, 5>(a, st);
    case 6: return launch_fwd_l<WD, OD, MD, 6>(a, st);
    default: return launch_fwd_l<WD, OD, MD, 7>(a, st);
  }
}

template <int WD, int OD, int MD>
static hipError_t launch_fwd_k(const FwdArgs& a, int k, hipStream_t st) {
  if constexpr (MD == 1) {
    if (use_neighbour_table(a.t.logg, k)) return launch_fwd_m<WD, OD, 3>(a, k, st);
  }
  return launch_fwd_m<WD, OD, MD>(a, k, st);
}

hipError_t launch_fq_fwd(const FqFwdLaunch& p, hipStream_t st) {
  if (p.g > 512) return launch_fq_fwd_big(p, st);
  FwdArgs a;
  a.t = make_geom(p.R, p.C, p.k, p.g, 1);
  a.W = p.W; a.s = p.s; a.s_r = p.s_r; a.delta = p.delta; a.z_u = p.z_u;
  a.alpha = p.alpha; a.z_b = p.z_b; a.codes = p.codes; a.W_hat = p.W_hat;
  a.resid = p.resid;
#define UQ_FWD(WD, OD, MD) \
  if (p.w_dtype == WD && p.w_hat_dtype == OD && p.mode == MD) return launch_fwd_k<WD, OD, MD>(a, p.k, st);
  UQ_FWD(BF16, BF16, 0) UQ_FWD(BF16, BF16, 1) UQ_FWD(BF16, BF16, 2)
  UQ_FWD(BF16, F32, 0) UQ_FWD(BF16, F32, 1) UQ_FWD(BF16, F32, 2)
  UQ_FWD(F32, BF16, 0) UQ_FWD(F32, BF16, 1) UQ_FWD(F32, BF16, 2)
  UQ_FWD(F32, F32, 0) UQ_FWD(F32, F32, 1) UQ_FWD(F32, F32, 2)
#undef UQ_FWD
  return hipErrorInvalidValue;
}

template <int WD, int GD, int OD, int MD, int LOGL>
static hipError_t launch_step_l(const StepArgs& a, hipStream_t st) {
  auto kern = fq_step_kernel<WD, GD, OD, MD, LOGL>;
  const size_t wave_bytes = wave_step_lds_bytes(a.f.t.logg, LOGL, MD == 3);
  const int wpb = fwd_waves_per_block(wave_bytes);
  const size_t lds = size_t(wpb) * wave_bytes;
  if (lds > 65536) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
    if (e != hipSuccess) return e;
  }
  const int64_t waves = (a.f.t.N + 511) / 512;
  hipLaunchKernelGGL(kern, dim3(unsigned((waves + wpb - 1) / wpb)), dim3(64 * wpb), lds, st, a);
  return hipGetLastError();
}

template <int WD, int GD, int OD, int MD>
static hipError_t launch_step_m(const StepArgs& a, int k, hipStream_t st) {
  switch (k) {
    case 1: return launch_step_l<WD, GD, OD, MD, 1>(a, st);
    case 2: return launch_step_l<WD, GD, OD, MD, 2>(a, st);
    case 3: return launch_step_l<WD, GD, OD, MD, 3>(a, st);
    case 4: return launch_step_l<WD, GD, OD, MD, 4>(a, st);
    case 5: return launch_step_l<WD, GD, OD, MD, 5>(a, st);
    case 6: return launch_step_l<WD, GD, OD, MD, 6>(a, st);
    default: return launch_step_l<WD, GD, OD, MD, 7>(a, st);
  }
}

template <int WD, int GD, int OD>
static hipError_t launch_step_d(const StepArgs& a, int k, int mode, hipStream_t st) {
  if (mode == 0) return launch_step_m<WD, GD, OD, 0>(a, k, st);
  if (mode == 2) return launch_step_m<WD, GD, OD, 2>(a, k, st);
  if (use_neighbour_table(a.f.t.logg, k)) return launch_step_m<WD, GD, OD, 3>(a, k, st);
  return hipErrorNotSupported;  // LOCAL without a neighbour table: the caller runs the two passes
}

template <int ODT, int MD>
static hipError_t launch_step_big(const BigArgs& a, const void* G, float lr_f, float lr_b, hipStream_t st) {
  const dim3 grid(unsigned(a.Gn)), block(kBigThreads);
  switch (a.k) {
#define UQ_SB(KK) \
    case KK: hipLaunchKernelGGL((fq_step_big_kernel<BF16, BF16, ODT, MD, KK>), grid, block, 0, st, a, G, lr_f, lr_b); break;
    UQ_SB(1) UQ_SB(2) UQ_SB(3) UQ_SB(4) UQ_SB(5) UQ_SB(6) UQ_SB(7)
#undef UQ_SB
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// Fused pass for g <= 512 (whose neighbour tables fit when the next mapping is
// LOCAL) and, with bf16 W and dL/dWhat, for large groups up to 16384 weights
// (one workgroup per group); otherwise the backward with the update, then
// the forward.
hipError_t launch_fq_step(const FqStepLaunch& p, hipStream_t st) {
  if (p.g > 512 && p.g <= kBigThreads * kVec * kStepBigChunks && p.w_dtype == BF16 && p.grad_dtype == BF16) {
    BigArgs b = big_args(p.R, p.C, p.k, p.g);
    b.W = p.W; b.s = p.s; b.s_r = p.s_r; b.delta = p.delta; b.z_u = p.z_u;
    b.alpha = p.alpha; b.z_b = p.z_b; b.codes = p.codes; b.W_hat = p.W_hat; b.resid = p.resid;
    const int md = p.mode == 0 ? 0 : p.mode == 2 ? 2 : 3;
    if (p.w_hat_dtype == BF16) {
      if (md == 0) return launch_step_big<BF16, 0>(b, p.grad_W_hat, p.lr_f, p.lr_b, st);
      if (md == 2) return launch_step_big<BF16, 2>(b, p.grad_W_hat, p.lr_f, p.lr_b, st);
      return launch_step_big<BF16, 3>(b, p.grad_W_hat, p.lr_f, p.lr_b, st);
    }
    if (md == 0) return launch_step_big<F32, 0>(b, p.grad_W_hat, p.lr_f, p.lr_b, st);
    if (md == 2) return launch_step_big<F32, 2>(b, p.grad_W_hat, p.lr_f, p.lr_b, st);
    return launch_step_big<F32, 3>(b, p.grad_W_hat, p.lr_f, p.lr_b, st);
  }
  const bool fused = p.g <= 512 && !(p.mode == 1 && !use_neighbour_table(__builtin_ctz(unsigned(p.g)), p.k));
  if (fused) {
    StepArgs a;
    a.f.t = make_geom(p.R, p.C, p.k, p.g, 1);
    a.f.W = p.W; a.f.s = p.s; a.f.s_r = p.s_r; a.f.delta = p.delta; a.f.z_u = p.z_u;
    a.f.alpha = p.alpha; a.f.z_b = p.z_b; a.f.codes = p.codes; a.f.W_hat = p.W_hat; a.f.resid = p.resid;
    a.s_out = p.s; a.alpha_out = p.alpha; a.z_b_out = p.z_b;
    a.G = p.grad_W_hat; a.lr_f = p.lr_f; a.lr_b = p.lr_b;
#define UQ_STEP(WD, GD, OD) \
    if (p.w_dtype == WD && p.grad_dtype == GD && p.w_hat_dtype == OD) return launch_step_d<WD, GD, OD>(a, p.k, p.mode, st);
    UQ_STEP(BF16, BF16, BF16) UQ_STEP(BF16, BF16, F32) UQ_STEP(BF16, F32, BF16) UQ_STEP(BF16, F32, F32)
    UQ_STEP(F32, BF16, BF16) UQ_STEP(F32, BF16, F32) UQ_STEP(F32, F32, BF16) UQ_STEP(F32, F32, F32)
#undef UQ_STEP
    return hipErrorInvalidValue;
  }
  FqBwdLaunch b{p.R, p.C, p.k, p.g, p.W, p.w_dtype, p.s, p.s_r, p.delta, p.z_u, p.alpha, p.z_b, p.codes,
                p.grad_W_hat, p.grad_dtype, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                1, p.lr_f, p.lr_b};
  hipError_t e = launch_fq_bwd(b, st);
  if (e != hipSuccess) return e;
  FqFwdLaunch f{p.R, p.C, p.k, p.g, p.W, p.w_dtype, p.s, p.s_r, p.delta, p.z_u, p.alpha, p.z_b, p.mode, p.codes,
                p.W_hat, p.w_hat_dtype, p.resid};
  return launch_fq_fwd(f, st);
}

hipError_t launch_fold(const FoldLaunch& p, hipStream_t st) {
  if (p.g > 512) {
    BigArgs b = big_args(p.R, p.C, p.k, p.g);
    b.W = p.W; b.s = p.s; b.s_r = p.s_r; b.delta = p.delta; b.z_u = p.z_u;
    b.alpha = p.alpha; b.z_b = p.z_b; b.alpha_star = p.alpha_star; b.z_star = p.z_star;
    b.codes = p.codes; b.code_src = p.code_src;
    return p.w_dtype == BF16 ? launch_fold_big<BF16>(b, st) : launch_fold_big<F32>(b, st);
  }
  FoldArgs a;
  a.t = make_geom(p.R, p.C, p.k, p.g, 1);
  a.W = p.W; a.s = p.s; a.s_r = p.s_r; a.delta = p.delta; a.z_u = p.z_u;
  a.alpha = p.alpha; a.z_b = p.z_b; a.alpha_star = p.alpha_star; a.z_star = p.z_star;
  a.codes = p.codes; a.code_src = p.code_src;
  const dim3 grid(grid_of(a.t)), block(kThreads);
  const size_t lds = fold_lds_bytes(a.t);
  if (p.w_dtype == BF16) hipLaunchKernelGGL((fold_kernel<BF16>), grid, block, lds, st, a);
  else hipLaunchKernelGGL((fold_kernel<F32>), grid, block, lds, st, a);
  return hipGetLastError();
}

hipError_t launch_dequant(const DequantLaunch& p, hipStream_t st) {
  if (p.g > 512) {
    BigArgs b = big_args(p.R, p.C, p.k, p.g);
    b.codes = const_cast<uint8_t*>(p.codes); b.alpha = p.alpha; b.z_b = p.z_b; b.W_hat = p.W_out;
    const dim3 grid(unsigned(b.Gn)), block(kBigThreads);
    if (p.out_dtype == BF16) hipLaunchKernelGGL((dequant_big_kernel<BF16>), grid, block, 0, st, b);
    else hipLaunchKernelGGL((dequant_big_kernel<F32>), grid, block, 0, st, b);
    return hipGetLastError();
  }
  DequantArgs a;
  a.t = make_geom(p.R, p.C, p.k, p.g, 1);
  a.codes = p.codes; a.alpha = p.alpha; a.z_b = p.z_b; a.W_out = p.W_out;
  const dim3 grid(grid_of(a.t)), block(kThreads);
  const size_t lds = 4 * (size_t(a.t.tile_groups) << a.t.logL);
  if (p.out_dtype == BF16) hipLaunchKernelGGL((dequant_kernel<BF16>), grid, block, lds, st, a);
  else hipLaunchKernelGGL((dequant_kernel<F32>), grid, block, lds, st, a);
  return hipGetLastError();
}

hipError_t launch_greedy(const GreedyLaunch& p, hipStream_t st) {
  if (p.g > 512) {
    BigArgs b = big_args(p.R, p.C, p.k, p.g);
    b.W = p.W; b.s = p.s; b.s_r = p.s_r; b.delta = p.delta; b.z_u = p.z_u; b.z_b = p.z_b;
    b.alpha_star = p.alpha;  // output: alpha
    const dim3 grid(unsigned(b.Gn)), block(kBigThreads);
    if (p.w_dtype == BF16) hipLaunchKernelGGL((greedy_big_kernel<BF16>), grid, block, 0, st, b);
    else hipLaunchKernelGGL((greedy_big_kernel<F32>), grid, block, 0, st, b);
    return hipGetLastError();
  }
  GreedyArgs a;
  a.t = make_geom(p.R, p.C, p.k, p.g, 1);
  a.W = p.W; a.s = p.s; a.s_r = p.s_r; a.delta = p.delta; a.z_u = p.z_u;
  a.z_b = p.z_b; a.alpha = p.alpha;
  const int64_t chunks = a.t.N / kVec;
  const dim3 grid(unsigned((chunks + kThreads - 1) / kThreads)), block(kThreads);
  if (p.w_dtype == BF16) hipLaunchKernelGGL((greedy_kernel<BF16>), grid, block, 0, st, a);
  else hipLaunchKernelGGL((greedy_kernel<F32>), grid, block, 0, st, a);
  return hipGetLastError();
}

}  // namespace uq
