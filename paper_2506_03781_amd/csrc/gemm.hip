// Reconstruction contractions on bf16 MFMA (gfx950 v_mfma_f32_32x32x16_bf16)
// with fused epilogues:
//   target   Yt = W X^T                       (once per layer)
//   forward  Et = What X^T [- Yt], sum Et^2    (loss partials per workgroup;
//                                               no target in the residual form)
//   backward G  = 2 Et Xt^T                    (weight gradient, bf16 or fp32),
//            or the straight-through backward + SGD update applied to G in
//            the epilogue (G never stored)
// All are C[M x N] = A[M x K] B[N x K]^T with both operands K-contiguous
// ("NT"), so one kernel template serves them.  The block's backpropagation
// also takes operands stored K-slow (A as [K x M], B as [K x N]): the weight
// gradient dY^T X and the input gradient dY W read the activations and the
// weights as they are stored, with no transposed copies (ping-pong kernel
// only; the copies take whole k-rows and the MFMA fragments come from LDS
// transpose reads).
//
// Kernels (all bf16 MFMA v_mfma_f32_32x32x16_bf16, fp32 accumulation):
//   gemm_pp_kernel    the main one, for K % 32 == 0 on 256 x 256 and 256 x 128
//                     tiles: eight wavefronts in two groups that alternate
//                     ("ping-pong") between an MFMA phase and a memory phase
//                     (LDS fragment reads, global_load_lds copies into a ring
//                     of 32- or 64-deep stages, exact vmcnt waits, barriers);
//   gemm_pipe_kernel  four wavefronts, the same direct-to-LDS stage ring, for
//                     128 x 128 tiles (shapes too small to fill the GPU with
//                     256-row tiles);
//   gemm_nt_kernel    register-staged, 64-deep double-buffered slabs, for K
//                     not a multiple of 32.
// The tile is the largest of 256x256, 256x128, 128x128 that still gives a
// workgroup per compute unit.  Workgroups are renumbered so that each XCD
// gets a contiguous run of tiles walked in groups of row-tiles, which keeps
// the operand panels it needs in its own L2.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

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
  SteParams ste;
  // strided batch (gridDim.y > 1): element offsets of A and B and byte
  // offset of out per batch
  int64_t bsa, bsb, bso;
  // causal structure of square [L, L] products (attention): 1 skips tiles
  // entirely above the diagonal (their outputs are not written), 2 ends the
  // K loop at the row tile's end (A zero above the diagonal), 3 starts it at
  // the row tile's start (A zero below the diagonal)
  int causal;
  HeadsParams heads;
  SwigluParams swiglu;
  const float* Rres;  // EPI_LOSS_BLOCK, EPI_RESID: the residual added to the product
};

// Operands and output of batch blockIdx.y.
__device__ __forceinline__ void select_batch(GemmArgs& p) {
  if (gridDim.y > 1) {
    const int64_t b = blockIdx.y;
    p.A += b * p.bsa;
    p.B += b * p.bsb;
    p.out = static_cast<char*>(p.out) + b * p.bso;
  }
}

// Two fp32 values -> packed bf16 pair (lo in bits 0..15), round to nearest
// even: one v_cvt_pk_bf16_f32 on gfx950.
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const f32x2 f = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2));
}

// A 32-row strip of one head (128 columns, fp32 in LDS, row stride 128) to
// the head-major bf16 output: element (row_base + r, h * 128 + j) goes to
// out[(slot(h) * M + row_base + r) * 128 + j], with the pairs (j, j + 64)
// rotated by the row's position angle when ROT: y1 = x1 c - x2 s,
// y2 = x2 c + x1 s (products rounded, then the sum, as the stand-alone
// rotary split computes them).  Lane l takes 4 consecutive pairs of rows
// l / 16 + 4 k.
template <bool ROT>
__device__ __forceinline__ void heads_strip(const GemmArgs& p, const float* strip, int64_t row_base, int64_t col_base,
                                            int lane) {
  const HeadsParams& hp = p.heads;
  const int h = int(col_base >> 7);
  const int slot = hp.perm > 1 ? (h % hp.perm) * (hp.H / hp.perm) + h / hp.perm : h;
  const int i0 = 4 * (lane & 15);
  uint16_t* out = static_cast<uint16_t*>(p.out) + int64_t(slot) * p.M * 128 + i0;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const int r = (lane >> 4) + 4 * k;
    const int64_t m = row_base + r;
    if (m >= p.M) break;
    const float4 a = *reinterpret_cast<const float4*>(&strip[r * 128 + i0]);
    const float4 b = *reinterpret_cast<const float4*>(&strip[r * 128 + 64 + i0]);
    float x1[4] = {p.scale * a.x, p.scale * a.y, p.scale * a.z, p.scale * a.w};
    float x2[4] = {p.scale * b.x, p.scale * b.y, p.scale * b.z, p.scale * b.w};
    float y1[4], y2[4];
    if constexpr (ROT) {
      const float4* cs = reinterpret_cast<const float4*>(hp.cs + (int64_t(m % hp.L) * 64 + i0) * 2);
      const float4 c01 = cs[0], c23 = cs[1];  // (cos, sin) of pairs i0 .. i0 + 3
      const float cn[4] = {c01.x, c01.z, c23.x, c23.z}, sn[4] = {c01.y, c01.w, c23.y, c23.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        y1[e] = x1[e] * cn[e] - x2[e] * sn[e];
        y2[e] = x2[e] * cn[e] + x1[e] * sn[e];
      }
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        y1[e] = x1[e];
        y2[e] = x2[e];
      }
    }
    uint16_t* o = out + m * 128;
    *reinterpret_cast<uint2*>(o) = make_uint2(pack_bf16x2(y1[0], y1[1]), pack_bf16x2(y1[2], y1[3]));
    *reinterpret_cast<uint2*>(o + 64) = make_uint2(pack_bf16x2(y2[0], y2[1]), pack_bf16x2(y2[2], y2[3]));
  }
}

// Map a linear workgroup id to (tile_m, tile_n).  Hardware dispatches
// workgroup i to XCD i % 8; renumber so that each XCD receives a contiguous
// run of logical tiles, then walk logical tiles in groups of GM row-tiles.
// An XCD's run of tiles then covers GM row-tiles and (run / GM) column-tiles,
// whose operand panels it pulls into its L2.  GM = 4 for 256-row tiles: on
// 256 x 256 tiles it beat 1, 2, 3 (by 1-10%), 8 and 16 (by 5-11%) on the 70B
// and 7B products and matched 5 and 6; 8 for 128 x 128 tiles.
template <int GM>
__device__ __forceinline__ void tile_of(int bid, int nb, int tiles_m, int tiles_n, int& tm, int& tn) {
  int logical = bid;
  if ((nb & 7) == 0) logical = (bid & 7) * (nb >> 3) + (bid >> 3);
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

// Straight-through backward of one strip (32 rows x 128 columns of the
// wave's tile, staged in LDS as fp32 acc) with the SGD update, the same
// arithmetic as the standalone backward kernel: lane l takes 8 consecutive
// columns of row 4 it + l / 16, a group of g columns is g / 8 adjacent lanes,
// and the group sums use the same fixed xor-butterfly.
template <int KB, int NB>
__device__ __forceinline__ void ste_strip(const GemmArgs& p, const float* strip, int64_t row_base, int64_t col_base,
                                          int lane) {
  const SteParams& q = p.ste;
  const int lpg = 1 << (q.logg - 3);
#pragma unroll 1
  for (int it0 = 0; it0 < 8; it0 += NB) {
    uint4 wq[NB];
    float4 s0[NB], s1[NB];
    uint2 cb[NB];
    float dlv[NB], srv[NB];
    bool act[NB];
    int64_t off[NB];
    // loads of NB row-iterations first (the epilogue has few wavefronts per
    // CU, so bytes in flight per lane decide the memory phase's speed)
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const int lrow = (it0 + j) * 4 + (lane >> 4);
      const int64_t row = row_base + lrow, col = col_base + (lane & 15) * 8;
      act[j] = row < p.M && col < p.N;
      off[j] = row * p.N + col;
      wq[j] = make_uint4(0, 0, 0, 0);
      s0[j] = make_float4(1, 1, 1, 1);
      s1[j] = s0[j];
      cb[j] = make_uint2(0, 0);
      dlv[j] = 1.0f;
      srv[j] = 1.0f;
      if (act[j]) {
        // bf16 weights travel with this batch; fp32 weights are read at use
        if (q.w_bf16) wq[j] = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(q.W) + off[j]);
        const float4* sp = reinterpret_cast<const float4*>(q.s + off[j]);
        s0[j] = sp[0];
        s1[j] = sp[1];
        cb[j] = *reinterpret_cast<const uint2*>(q.codes + off[j]);
        const int64_t gid = off[j] >> q.logg;
        dlv[j] = q.delta ? q.delta[gid] : 1.0f;
        srv[j] = q.s_r ? q.s_r[row] : 1.0f;
      }
    }
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const int lrow = (it0 + j) * 4 + (lane >> 4);
      const int c8 = (lane & 15) * 8;
      const int64_t gid = act[j] ? (off[j] >> q.logg) : 0;
      float S = 0.0f, Sa[KB];
#pragma unroll
      for (int b = 0; b < KB; ++b) Sa[b] = 0.0f;
      const float dl = dlv[j];
      if (act[j]) {
        float G[8], w[8];
        const float4 g0 = *reinterpret_cast<const float4*>(strip + lrow * 128 + c8);
        const float4 g1 = *reinterpret_cast<const float4*>(strip + lrow * 128 + c8 + 4);
        G[0] = p.scale * g0.x; G[1] = p.scale * g0.y; G[2] = p.scale * g0.z; G[3] = p.scale * g0.w;
        G[4] = p.scale * g1.x; G[5] = p.scale * g1.y; G[6] = p.scale * g1.z; G[7] = p.scale * g1.w;
        if (q.w_bf16) {
          const uint32_t wv[4] = {wq[j].x, wq[j].y, wq[j].z, wq[j].w};
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            w[2 * i] = __uint_as_float(wv[i] << 16);
            w[2 * i + 1] = __uint_as_float(wv[i] & 0xFFFF0000u);
          }
        } else {
          const float4* wp = reinterpret_cast<const float4*>(static_cast<const float*>(q.W) + off[j]);
          const float4 a = wp[0], b = wp[1];
          w[0] = a.x; w[1] = a.y; w[2] = a.z; w[3] = a.w; w[4] = b.x; w[5] = b.y; w[6] = b.z; w[7] = b.w;
        }
        const float sv[8] = {s0[j].x, s0[j].y, s0[j].z, s0[j].w, s1[j].x, s1[j].y, s1[j].z, s1[j].w};
        const float ds = dl * srv[j];
        float gs[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const uint32_t byte = ((i < 4 ? cb[j].x : cb[j].y) >> (8 * (i & 3))) & 0xFFu;
          const bool m = (byte & 0x80u) != 0u;
          const float g = G[i];
          S += g;
#pragma unroll
          for (int b = 0; b < KB; ++b) Sa[b] += ((byte >> b) & 1u) ? g : -g;
          const float x = w[i] * __builtin_amdgcn_rcpf(ds * sv[i]);
          gs[i] = m ? -(dl * g) * x * __builtin_amdgcn_rcpf(sv[i]) : 0.0f;
        }
        if (q.grad_s) {
          float4* gp = reinterpret_cast<float4*>(q.grad_s + off[j]);
          gp[0] = make_float4(gs[0], gs[1], gs[2], gs[3]);
          gp[1] = make_float4(gs[4], gs[5], gs[6], gs[7]);
        }
        float4* sp = reinterpret_cast<float4*>(q.s + off[j]);
        sp[0] = make_float4(sv[0] - q.lr_f * gs[0], sv[1] - q.lr_f * gs[1], sv[2] - q.lr_f * gs[2],
                            sv[3] - q.lr_f * gs[3]);
        sp[1] = make_float4(sv[4] - q.lr_f * gs[4], sv[5] - q.lr_f * gs[5], sv[6] - q.lr_f * gs[6],
                            sv[7] - q.lr_f * gs[7]);
      }
      for (int msk = lpg >> 1; msk >= 1; msk >>= 1) {
        S += __shfl_xor(S, msk, 64);
#pragma unroll
        for (int b = 0; b < KB; ++b) Sa[b] += __shfl_xor(Sa[b], msk, 64);
      }
      if (act[j] && (lane & (lpg - 1)) == 0) {
        const float gzb = dl * S;
#pragma unroll
        for (int b = 0; b < KB; ++b) {
          const float ga = dl * Sa[b];
          if (q.grad_alpha) q.grad_alpha[gid * KB + b] = ga;
          q.alpha[gid * KB + b] = q.alpha[gid * KB + b] - q.lr_b * ga;
        }
        if (q.grad_z_b) q.grad_z_b[gid] = gzb;
        q.z_b[gid] = q.z_b[gid] - q.lr_b * gzb;
      }
    }
  }
}

// Store an accumulator tile with the requested epilogue, staged through LDS
// one 32-row strip at a time.  Accumulator register r of lane l of a 32x32
// MFMA block holds row 8*(r/4) + 4*(l/32) + r%4 and column l%32; each wave
// writes its strip (32 x WN fp32) to its own LDS region, then reads it back
// as rows of float4 so that the target is loaded and the output stored as
// contiguous 16-byte / 8-byte vectors.  `scratch` must hold 4 * 32 * WN
// floats and may alias the operand stages (all waves are past their last
// operand read when this is called).
template <int BM, int BN, int EPI, int WM = BM / 2, int WN = BN / 2, int NW = 4, int FM = WM / 32,
          int FN = WN / 32>
__device__ __forceinline__ void epilogue(const GemmArgs& p, f32x16 (&acc)[FM][FN], int64_t m0, int64_t n0,
                                         int wm, int wn, int lane, int wave, int tid, float* scratch) {
  constexpr int Q = WN / 4;            // float4 per strip row
  constexpr int ITER = 32 * Q / 64;    // float4 per lane per strip
  const int lr = lane & 31, lh = lane >> 5;
  float* strip = scratch + wave * 32 * WN;
  const bool full = (m0 + BM <= p.M) && (n0 + BN <= p.N);
  const float* __restrict__ Yt = p.Yt;
  float lsum = 0.0f;
#pragma unroll
  for (int i = 0; i < FM; ++i) {
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        strip[(8 * (r >> 2) + 4 * lh + (r & 3)) * WN + j * 32 + lr] = acc[i][j][r];
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): the strip is written (own wave only)
    __builtin_amdgcn_wave_barrier();
    const int64_t row_base = m0 + wm * WM + i * 32;
    const int64_t col_base = n0 + wn * WN;
    if constexpr (EPI == EPI_SWIGLU) {
      static_assert(WN == 64, "the SiLU product needs 64-column wave tiles (G and U halves)");
      // strip columns 0..31: G, 32..63: U of rows I0 .. I0 + 31 of W
      const int64_t I = p.swiglu.I, i0 = n0 / 2 + wn * 32;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int item = lane + 64 * k, rr = item >> 3, cq = (item & 7) * 4;
        const int64_t m = row_base + rr;
        if (m >= p.M || i0 + cq >= I) continue;
        const float4 g4 = *reinterpret_cast<const float4*>(&strip[rr * 64 + cq]);
        const float4 u4 = *reinterpret_cast<const float4*>(&strip[rr * 64 + 32 + cq]);
        const uint32_t g01 = pack_bf16x2(p.scale * g4.x, p.scale * g4.y), g23 = pack_bf16x2(p.scale * g4.z, p.scale * g4.w);
        const uint32_t u01 = pack_bf16x2(p.scale * u4.x, p.scale * u4.y), u23 = pack_bf16x2(p.scale * u4.z, p.scale * u4.w);
        const float gf[4] = {__uint_as_float(g01 << 16), __uint_as_float(g01 & 0xFFFF0000u),
                             __uint_as_float(g23 << 16), __uint_as_float(g23 & 0xFFFF0000u)};
        const float uf[4] = {__uint_as_float(u01 << 16), __uint_as_float(u01 & 0xFFFF0000u),
                             __uint_as_float(u23 << 16), __uint_as_float(u23 & 0xFFFF0000u)};
        const int64_t o = m * I + i0 + cq;
        *reinterpret_cast<uint2*>(static_cast<uint16_t*>(p.out) + o) = make_uint2(g01, g23);
        *reinterpret_cast<uint2*>(p.swiglu.U + o) = make_uint2(u01, u23);
        *reinterpret_cast<uint2*>(p.swiglu.H + o) =
            make_uint2(pack_bf16x2(silu_mul(gf[0], uf[0]), silu_mul(gf[1], uf[1])),
                       pack_bf16x2(silu_mul(gf[2], uf[2]), silu_mul(gf[3], uf[3])));
      }
      __builtin_amdgcn_s_waitcnt(0xC07F);  // strip reads done before the next strip overwrites it
      __builtin_amdgcn_wave_barrier();
      continue;
    }
    if constexpr (EPI == EPI_SWIGLU_BWD) {
      // dH = bf16(scale acc) of the strip, then the SiLU product's backward with
      // G and U of the same elements; the strip's G, U loads are issued first
      constexpr int IT = 32 * WN / 4 / 64;  // 4-column items per lane
      uint2 gq[IT], uq4[IT];
#pragma unroll
      for (int k = 0; k < IT; ++k) {
        const int item = lane + 64 * k, rr = item / (WN / 4), cq = (item % (WN / 4)) * 4;
        const int64_t m = row_base + rr, n = col_base + cq;
        const bool ok = m < p.M && n < p.N;
        const int64_t o = ok ? m * p.N + n : 0;
        gq[k] = *reinterpret_cast<const uint2*>(p.swiglu.G_in + o);
        uq4[k] = *reinterpret_cast<const uint2*>(p.swiglu.U_in + o);
      }
#pragma unroll
      for (int k = 0; k < IT; ++k) {
        const int item = lane + 64 * k, rr = item / (WN / 4), cq = (item % (WN / 4)) * 4;
        const int64_t m = row_base + rr, n = col_base + cq;
        if (m >= p.M || n >= p.N) continue;
        const float4 v = *reinterpret_cast<const float4*>(&strip[rr * WN + cq]);
        const uint32_t h01 = pack_bf16x2(p.scale * v.x, p.scale * v.y), h23 = pack_bf16x2(p.scale * v.z, p.scale * v.w);
        const uint32_t hw[2] = {h01, h23}, gw[2] = {gq[k].x, gq[k].y}, uw[2] = {uq4[k].x, uq4[k].y};
        float dg[4], du[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint32_t sh = (e & 1) ? 0u : 16u;
          const uint32_t mk = 0xFFFF0000u;
          const float dh = __uint_as_float((hw[e >> 1] << sh) & mk);
          const float g = __uint_as_float((gw[e >> 1] << sh) & mk);
          const float u = __uint_as_float((uw[e >> 1] << sh) & mk);
          silu_mul_grad(dh, g, u, dg[e], du[e]);
        }
        const int64_t o = m * p.swiglu.ldo + n;
        *reinterpret_cast<uint2*>(static_cast<uint16_t*>(p.out) + o) =
            make_uint2(pack_bf16x2(dg[0], dg[1]), pack_bf16x2(dg[2], dg[3]));
        *reinterpret_cast<uint2*>(p.swiglu.dU + o) = make_uint2(pack_bf16x2(du[0], du[1]), pack_bf16x2(du[2], du[3]));
      }
      __builtin_amdgcn_s_waitcnt(0xC07F);  // strip reads done before the next strip overwrites it
      __builtin_amdgcn_wave_barrier();
      continue;
    }
    if constexpr (EPI == EPI_HEADS || EPI == EPI_HEADS_ROT) {
      static_assert(WN == 128, "the head split needs 128-column wave tiles");
      if (col_base < p.N) {
        if (EPI == EPI_HEADS_ROT && int(col_base >> 7) < p.heads.nrot)
          heads_strip<true>(p, strip, row_base, col_base, lane);
        else
          heads_strip<false>(p, strip, row_base, col_base, lane);
      }
      __builtin_amdgcn_s_waitcnt(0xC07F);  // strip reads done before the next strip overwrites it
      __builtin_amdgcn_wave_barrier();
      continue;
    }
    if constexpr (EPI >= EPI_STE) {
      static_assert(WN == 128, "the fused backward needs 128-column wave tiles");
      // row-iterations whose loads are in flight together: 8 with four
      // wavefronts per workgroup, 2 with eight (they keep loads in flight)
      ste_strip<EPI - EPI_STE, (NW == 8 ? 2 : 8)>(p, strip, row_base, col_base, lane);
      __builtin_amdgcn_s_waitcnt(0xC07F);  // strip reads done before the next strip overwrites it
      __builtin_amdgcn_wave_barrier();
      continue;
    }
    // the strip's first element once in 64 bits; element offsets in 32 bits
    // (N < 2^26 is checked on the host)
    const int64_t base = row_base * p.N + col_base;
    const int ldn = int(p.N);
    float4 y[ITER], rq[ITER];
    if constexpr (EPI == EPI_LOSS || EPI == EPI_LOSS_BLOCK || EPI == EPI_RESID) {  // stored target and/or residual
#pragma unroll
      for (int it = 0; it < ITER; ++it) {
        const int idx = lane + it * 64, rr = idx / Q, cc = (idx % Q) * 4;
        const bool ok = full || (row_base + rr < p.M && col_base + cc < p.N);  // N % 4 == 0 here
        if constexpr (EPI != EPI_RESID)
          y[it] = ok ? *reinterpret_cast<const float4*>(Yt + base + rr * ldn + cc) : make_float4(0, 0, 0, 0);
        if constexpr (EPI == EPI_LOSS_BLOCK || EPI == EPI_RESID)
          rq[it] = ok ? *reinterpret_cast<const float4*>(p.Rres + base + rr * ldn + cc) : make_float4(0, 0, 0, 0);
      }
    }
    auto put = [&](int it) {
      const int idx = lane + it * 64, rr = idx / Q, cc = (idx % Q) * 4;
      const float4 v = *reinterpret_cast<const float4*>(&strip[rr * WN + cc]);
      const int64_t o = base + rr * ldn + cc;
      if constexpr (EPI == EPI_TARGET) {
        *reinterpret_cast<float4*>(static_cast<float*>(p.out) + o) = v;
      } else if constexpr (EPI == EPI_LOSS || EPI == EPI_LOSS_RES || EPI == EPI_LOSS_BLOCK) {
        float e0 = v.x, e1 = v.y, e2 = v.z, e3 = v.w;
        if constexpr (EPI == EPI_LOSS) {
          e0 = v.x - y[it].x;
          e1 = v.y - y[it].y;
          e2 = v.z - y[it].z;
          e3 = v.w - y[it].w;
        } else if constexpr (EPI == EPI_LOSS_BLOCK) {
          e0 = (rq[it].x + v.x) - y[it].x;
          e1 = (rq[it].y + v.y) - y[it].y;
          e2 = (rq[it].z + v.z) - y[it].z;
          e3 = (rq[it].w + v.w) - y[it].w;
        }
        lsum += e0 * e0;
        lsum += e1 * e1;
        lsum += e2 * e2;
        lsum += e3 * e3;
        *reinterpret_cast<uint2*>(static_cast<uint16_t*>(p.out) + o) =
            make_uint2(pack_bf16x2(e0, e1), pack_bf16x2(e2, e3));
      } else if constexpr (EPI == EPI_GRAD_BF16) {
        *reinterpret_cast<uint2*>(static_cast<uint16_t*>(p.out) + o) =
            make_uint2(pack_bf16x2(p.scale * v.x, p.scale * v.y), pack_bf16x2(p.scale * v.z, p.scale * v.w));
      } else if constexpr (EPI == EPI_GRAD_F32) {
        *reinterpret_cast<float4*>(static_cast<float*>(p.out) + o) =
            make_float4(p.scale * v.x, p.scale * v.y, p.scale * v.z, p.scale * v.w);
      } else if constexpr (EPI == EPI_RESID) {
        *reinterpret_cast<float4*>(static_cast<float*>(p.out) + o) =
            make_float4(rq[it].x + p.scale * v.x, rq[it].y + p.scale * v.y, rq[it].z + p.scale * v.z,
                        rq[it].w + p.scale * v.w);
      }
    };
    if (full) {  // uniform: interior tiles store without per-element checks
#pragma unroll
      for (int it = 0; it < ITER; ++it) put(it);
    } else {
#pragma unroll
      for (int it = 0; it < ITER; ++it) {
        const int idx = lane + it * 64;
        if (row_base + idx / Q < p.M && col_base + (idx % Q) * 4 < p.N) put(it);
      }
    }
    __builtin_amdgcn_s_waitcnt(0xC07F);  // strip reads done before the next strip overwrites it
    __builtin_amdgcn_wave_barrier();
  }
  if constexpr (EPI == EPI_LOSS || EPI == EPI_LOSS_RES || EPI == EPI_LOSS_BLOCK) {
    __shared__ float sred[NW];
    for (int msk = 32; msk >= 1; msk >>= 1) lsum += __shfl_xor(lsum, msk, 64);
    if (lane == 0) sred[wave] = lsum;
    __syncthreads();
    if (tid == 0) {
      float t;
      if constexpr (NW == 4) {
        t = (sred[0] + sred[1]) + (sred[2] + sred[3]);
      } else {
        t = ((sred[0] + sred[1]) + (sred[2] + sred[3])) + ((sred[4] + sred[5]) + (sred[6] + sred[7]));
      }
      p.partials[blockIdx.x] = t;
    }
  }
}

template <int BM, int BN, int EPI>
__global__ __launch_bounds__(256) void gemm_nt_kernel(GemmArgs p) {
  select_batch(p);
  constexpr int BK = 64;
  constexpr int WM = BM / 2, WN = BN / 2;
  constexpr int FM = WM / 32, FN = WN / 32;
  constexpr int CA = BM * 8 / 256;  // 16-byte chunks per thread and K-slab
  constexpr int CB = BN * 8 / 256;
  static_assert(CA >= 1 && CB >= 1, "tile too small");

  __shared__ uint4 smem[2 * (BM + BN) * 8];
  uint4 (*sA)[BM * 8] = reinterpret_cast<uint4 (*)[BM * 8]>(smem);
  uint4 (*sB)[BN * 8] = reinterpret_cast<uint4 (*)[BN * 8]>(smem + 2 * BM * 8);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  int tm, tn;
  tile_of<(BM == 128 && BN == 128) ? 8 : 4>(blockIdx.x, gridDim.x, p.tiles_m, p.tiles_n, tm, tn);
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

  epilogue<BM, BN, EPI>(p, acc, m0, n0, wm, wn, lane, wave, tid, reinterpret_cast<float*>(smem));
}

// ---------------------------------------------------------------------------
// Pipelined variant for K % 32 == 0: operands go straight from global memory
// into a ring of S LDS stages (gfx950 global_load_lds_dwordx4, no register
// staging), two stages ahead of the MFMAs; workgroup barriers carry no
// memory fence (each wave waits only for its own loads of the stage it is
// about to read, with an exact vmcnt), and the fragments of the next
// 16-deep substep are read while the MFMAs of the current one run.
// A stage holds BK = 32 of K: rows of 64 bytes, four 16-byte chunks per row,
// chunk position kc ^ ((row >> 1) & 3) so that 8 consecutive rows read at
// one K offset hit 8 distinct bank groups.  Rows past M or N are loaded from
// row M-1 / N-1 (valid addresses) and masked at the store.
// ---------------------------------------------------------------------------
typedef __attribute__((address_space(3))) void lds_void;
typedef const __attribute__((address_space(1))) void glb_void;

template <int VM>
__device__ __forceinline__ void wait_vmcnt() {
  // s_waitcnt fields: vmcnt[3:0] and [15:14], expcnt[6:4], lgkmcnt[11:8]
  __builtin_amdgcn_s_waitcnt((VM & 0xF) | ((VM >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

template <int BM, int BN, int EPI, int S>
__global__ __launch_bounds__(256) void gemm_pipe_kernel(GemmArgs p) {
  select_batch(p);
  constexpr int BK = 32;
  constexpr int WM = BM / 2, WN = BN / 2;
  constexpr int FM = WM / 32, FN = WN / 32;
  constexpr int ABLK = BM / 16, BBLK = BN / 16;      // 1 KB blocks (16 rows) per stage
  constexpr int PER_WAVE = (ABLK + BBLK) / 4;         // load instructions per wave and stage
  static_assert((ABLK + BBLK) % 4 == 0, "stage blocks must split over 4 waves");

  __shared__ uint4 smem[S * (BM + BN) * 4];
  uint4 (*sA)[BM * 4] = reinterpret_cast<uint4 (*)[BM * 4]>(smem);
  uint4 (*sB)[BN * 4] = reinterpret_cast<uint4 (*)[BN * 4]>(smem + S * BM * 4);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  int tm, tn;
  tile_of<(BM == 128 && BN == 128) ? 8 : 4>(blockIdx.x, gridDim.x, p.tiles_m, p.tiles_n, tm, tn);
  const int64_t m0 = int64_t(tm) * BM, n0 = int64_t(tn) * BN;
  const int64_t K = p.K;
  if (p.causal == 1 && n0 >= m0 + BM) return;  // whole tile above the diagonal (uniform per workgroup)
  const int64_t kb = p.causal == 3 ? m0 : 0;
  const int64_t ke = p.causal == 2 ? min(K, m0 + BM) : K;

  // This lane's source for each of the wave's load instructions.  Lane l
  // fills LDS slot l of a 1 KB block: row 16*blk + l/4, slot l%4, which holds
  // chunk (l%4) ^ ((row>>1)&3) of that row.
  const uint16_t* src[PER_WAVE];
  int dst_off[PER_WAVE];
  bool isA[PER_WAVE];
#pragma unroll
  for (int q = 0; q < PER_WAVE; ++q) {
    const int blk = wave * PER_WAVE + q;
    const bool a = blk < ABLK;
    const int b = a ? blk : blk - ABLK;
    const int row = b * 16 + (lane >> 2);
    const int kc = (lane & 3) ^ ((row >> 1) & 3);
    isA[q] = a;
    const int64_t gr = a ? min(m0 + row, p.M - 1) : min(n0 + row, p.N - 1);
    src[q] = (a ? p.A : p.B) + gr * K + kb + kc * 8;
    dst_off[q] = b * 64;
  }
  auto issue = [&](int stage, int64_t k0) {
#pragma unroll
    for (int q = 0; q < PER_WAVE; ++q) {
      uint4* dst = isA[q] ? &sA[stage][dst_off[q]] : &sB[stage][dst_off[q]];
      __builtin_amdgcn_global_load_lds((glb_void*)(src[q] + k0), (lds_void*)dst, 16, 0, 0);
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
  int offA[2][FM], offB[2][FN];
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const int kc = s * 2 + lh;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int row = wm * WM + i * 32 + lr;
      offA[s][i] = row * 4 + (kc ^ ((row >> 1) & 3));
    }
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int row = wn * WN + j * 32 + lr;
      offB[s][j] = row * 4 + (kc ^ ((row >> 1) & 3));
    }
  }
  bf16x8 a0[FM], b0[FN], a1[FM], b1[FN];
  auto rd = [&](int st, int s, bf16x8 (&af)[FM], bf16x8 (&bfr)[FN]) {
#pragma unroll
    for (int i = 0; i < FM; ++i) af[i] = __builtin_bit_cast(bf16x8, sA[st][offA[s][i]]);
#pragma unroll
    for (int j = 0; j < FN; ++j) bfr[j] = __builtin_bit_cast(bf16x8, sB[st][offB[s][j]]);
  };
  auto mma = [&](const bf16x8 (&af)[FM], const bf16x8 (&bfr)[FN]) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
  };
  // Each substep: one MFMA, half of the next substep's fragment reads, one
  // MFMA, the other half, then the remaining MFMAs.  An MFMA leads, so the
  // LDS wait in front of it covers only fragments read a whole substep
  // earlier (with LDS-DMA loads in flight the compiler can only wait for
  // every outstanding LDS read, so a read issued first would be waited for
  // too), and the last read is followed by FM*FN - 2 MFMAs before its data
  // is needed.
  auto interleave = [&]() {
    constexpr int R0 = (FM + FN) / 2;
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);             // MFMA
    __builtin_amdgcn_sched_group_barrier(0x100, R0, 0);            // LDS reads
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);             // MFMA
    __builtin_amdgcn_sched_group_barrier(0x100, FM + FN - R0, 0);  // LDS reads
    __builtin_amdgcn_sched_group_barrier(0x008, FM * FN - 2, 0);   // MFMAs
  };

  const int nk = int((ke - kb) / BK);
#pragma unroll
  for (int s = 0; s < S - 1; ++s)
    if (s < nk) issue(s, int64_t(s) * BK);
  if (nk >= S - 1) wait_vmcnt<(S - 2) * PER_WAVE>();
  else wait_vmcnt<0>();
  __builtin_amdgcn_s_barrier();
  rd(0, 0, a0, b0);
  int kt = 0;
  // Steady state: every iteration issues stage kt+S-1 and waits with the same
  // count, so the body has no branches and the compiler's LDS wait before the
  // first MFMA of each substep covers only the fragments it reads (with
  // branches its merged state forced a wait for every outstanding LDS read).
  for (; kt + S - 1 < nk; ++kt) {
    const int st = kt % S;
    __builtin_amdgcn_sched_barrier(0);
    rd(st, 1, a1, b1);
    mma(a0, b0);
    interleave();
    __builtin_amdgcn_sched_barrier(0);
    wait_vmcnt<(S - 3) * PER_WAVE>();  // stage kt+1 resident, kt+2..kt+S-2 may be in flight
    __builtin_amdgcn_s_barrier();
    issue((kt + S - 1) % S, int64_t(kt + S - 1) * BK);
    __builtin_amdgcn_sched_barrier(0);
    rd((kt + 1) % S, 0, a0, b0);
    mma(a1, b1);
    interleave();
  }
  // the last S-1 stages: nothing left to issue, the waits shrink to zero
  for (; kt < nk; ++kt) {
    const int st = kt % S;
    __builtin_amdgcn_sched_barrier(0);
    rd(st, 1, a1, b1);  // substep 1 of stage kt while substep 0 multiplies
    mma(a0, b0);
    interleave();
    __builtin_amdgcn_sched_barrier(0);
    if (kt + 1 < nk) {
      // stage kt+1 must be resident; loads of later stages may stay in flight
      const int later = min(nk - 1, kt + S - 2) - (kt + 1);
      if (later >= S - 3) wait_vmcnt<(S - 3) * PER_WAVE>();
      else if (later == 1) wait_vmcnt<PER_WAVE>();
      else wait_vmcnt<0>();
      __builtin_amdgcn_s_barrier();
      // the stage overwritten here was last read before this barrier
      if (kt + S - 1 < nk) issue((kt + S - 1) % S, int64_t(kt + S - 1) * BK);
    }
    __builtin_amdgcn_sched_barrier(0);
    rd((kt + 1) % S, 0, a0, b0);  // substep 0 of stage kt+1 (unused after the last stage)
    mma(a1, b1);
    interleave();
  }
  __syncthreads();  // every wave is past its last operand read: the stages become epilogue scratch
  epilogue<BM, BN, EPI>(p, acc, m0, n0, wm, wn, lane, wave, tid, reinterpret_cast<float*>(smem));
}

// ---------------------------------------------------------------------------
// Ping-pong main loop for single products on 256 x 256 or 256 x 128 tiles.
// Eight wavefronts in two groups of four, one wavefront of each group per
// SIMD.  The groups alternate between an MFMA phase on fragments held in
// registers and a memory phase (the next stage's fragments from LDS, this
// wavefront's share of the copy of stage k+S-1, the wait for its share of
// stage k+1), separated by workgroup barriers and offset by one phase: group
// 1 passes one barrier before the loop and group 0 one after it, so both
// pass the same number, and no stage is overwritten while either group may
// still read it.  While one group's MFMAs run, the other group's LDS reads
// and copies proceed on the same SIMDs.  Stages are BK = 32 deep (64-byte
// rows, 4-stage ring) or 64 deep (128-byte rows, 3-stage ring: twice the
// MFMAs per phase for the 64 x 64 wave tiles of 256 x 128).  Chunk kc of row
// r sits at kc ^ ((r >> 2) & 3) (BK 32) or kc ^ ((r >> 1) & 7) (BK 64), so
// the 16 rows a quarter-wavefront reads at one K offset fall in 16 distinct
// bank groups.  Copies past the last stage reload it into a slot no phase
// reads again, so every iteration issues and waits the same; rows past M or N
// are loaded from row M-1 / N-1 and masked at the store.
// ---------------------------------------------------------------------------
template <int BK>
__device__ __forceinline__ int pp_chunk(int row, int kc) {
  return BK == 64 ? (kc ^ ((row >> 1) & 7)) : (kc ^ ((row >> 2) & 3));
}

// Operands stored K-slow ([K x M], M contiguous): a 32-deep stage holds 32
// k-rows of the tile's BM columns, chunk c (8 columns) of k-row r in slot
// c ^ 4 (r & 3), so the four k-rows a 16-lane group reads sit 64 bytes apart
// in the bank space.  ds_read_b64_tr_b16 gives lane i of each 16-lane group,
// in slot j, element i % 4 of the 8 bytes addressed by lane 4 j + i / 4 of
// the group: with lane 4 q + r addressing k-row k0 + r, columns c0 + 4 q ..
// c0 + 4 q + 3, lane i receives column c0 + i at k-rows k0 .. k0 + 3, which
// is half of an MFMA operand fragment (8 consecutive k of one row); two
// reads, 4 k-rows apart, make the fragment.
typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;
__device__ __forceinline__ bf16x8 tr_fragment(const char* stage, int off_lo, int off_hi) {
  const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(stage + off_lo));
  const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(stage + off_hi));
  const v4i16 both[2] = {lo, hi};
  return __builtin_bit_cast(bf16x8, both);
}

// Byte offset, in a K-slow stage of W columns, of the 8 bytes this lane
// addresses for the fragment of rows (columns) col0 .. col0 + 31 at substep
// 0, first half.
template <int W>
__device__ __forceinline__ int tr_offset(int col0, int lane) {
  const int g16 = lane >> 4, s16 = lane & 15;
  const int kr = 8 * (g16 >> 1) + (s16 >> 2);
  const int c = col0 + 16 * (g16 & 1) + 4 * (s16 & 3);
  return kr * W * 2 + (((c >> 3) ^ (4 * (kr & 3))) << 4) + ((c & 7) >> 2) * 8;
}

template <int BM, int BN, int EPI, int WAVES_M = (BN == 256 ? 2 : 4), int BK = 32, bool TA = false,
          bool TB = false>
__global__ __launch_bounds__(512) void gemm_pp_kernel(GemmArgs p) {
  select_batch(p);
  static_assert(BK == 32 || !(TA || TB), "K-slow operands use 32-deep stages");
  constexpr int S = BK == 64 ? 3 : 4;
  constexpr int CPR = BK / 8;        // 16-byte chunks per stage row
  constexpr int RPB = 64 / CPR;      // stage rows per 1 KB copy
  constexpr int NS = BK / 16;        // MFMA substeps per stage
  constexpr int WAVES_N = 8 / WAVES_M;
  constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N, FM = WM / 32, FN = WN / 32;
  // K-slow operands: chunks per k-row and k-rows per 1 KB copy
  constexpr int CPKA = BM / 8, KPBA = 64 / CPKA, CPKB = BN / 8, KPBB = 64 / CPKB;
  constexpr int ABLK = TA ? BK / KPBA : BM / RPB, BBLK = TB ? BK / KPBB : BN / RPB;
  constexpr int PW = (ABLK + BBLK) / 8;  // 1 KB copies per wave and stage
  static_assert((ABLK + BBLK) % 8 == 0, "stage blocks must split over 8 waves");

  __shared__ uint4 smem[S * (BM + BN) * CPR];
  uint4 (*sA)[BM * CPR] = reinterpret_cast<uint4 (*)[BM * CPR]>(smem);
  uint4 (*sB)[BN * CPR] = reinterpret_cast<uint4 (*)[BN * CPR]>(smem + S * BM * CPR);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int grp = wave >> 2, qw = wave & 3;
  // 2 x 4 wave grid: rows by qw / 2, columns by (qw % 2, group); 4 x 2: rows by qw, columns by group
  const int wm = WAVES_M == 2 ? (qw >> 1) : qw;
  const int wn = WAVES_M == 2 ? ((qw & 1) * 2 + grp) : grp;
  int tm, tn;
  tile_of<(BM == 128 && BN == 128) ? 8 : 4>(blockIdx.x, gridDim.x, p.tiles_m, p.tiles_n, tm, tn);
  const int64_t m0 = int64_t(tm) * BM, n0 = int64_t(tn) * BN;
  const int64_t K = p.K;
  // causal structure (uniform per workgroup, before any barrier)
  if (p.causal == 1 && n0 >= m0 + BM) return;
  const int64_t kb = p.causal == 3 ? m0 : 0;
  const int64_t ke = p.causal == 2 ? min(K, m0 + BM) : K;

  // Lane l of a copy fills LDS slot l of a 1 KB block: row RPB blk + l / CPR,
  // slot l % CPR, which holds chunk pp_chunk(row, l % CPR) of that row.  A
  // K-slow operand's block is k-rows KPB blk .. (whole k-rows; slot l % CPK
  // of k-row r holds chunk (l % CPK) ^ 4 (r & 3)); columns past M or N are
  // loaded from the last chunk and masked at the store.
  const uint16_t* src[PW];
  int dst_off[PW];
  bool isA[PW];
  int64_t kstep[PW];  // elements per K stage
#pragma unroll
  for (int j = 0; j < PW; ++j) {
    const int blk = wave * PW + j;
    const bool a = blk < ABLK;
    const int b = a ? blk : blk - ABLK;
    isA[j] = a;
    dst_off[j] = b * 64;
    if ((a && TA) || (!a && TB)) {
      const int cpk = a ? CPKA : CPKB, kpb = a ? KPBA : KPBB;
      const int kr = b * kpb + lane / cpk;
      const int c = (lane % cpk) ^ (4 * (kr & 3));
      const int64_t ext = a ? p.M : p.N;
      const int64_t col = min((a ? m0 : n0) + 8 * c, ext - 8);
      src[j] = (a ? p.A : p.B) + int64_t(kr) * ext + col;
      kstep[j] = BK * ext;
    } else if (EPI == EPI_SWIGLU && !a) {
      // interleaved columns: 32-row blocks of W_g and W_u rows n0 / 2 + 32 (q / 2) ..
      const int row = b * RPB + lane / CPR;
      const int kc = pp_chunk<BK>(row, lane % CPR);
      const int64_t gr = min(n0 / 2 + 32 * (row >> 6) + (row & 31), p.swiglu.I - 1);
      src[j] = ((row >> 5) & 1 ? p.swiglu.Wu : p.B) + gr * K + kc * 8;
      kstep[j] = BK;
    } else {
      const int row = b * RPB + lane / CPR;
      const int kc = pp_chunk<BK>(row, lane % CPR);
      const int64_t gr = a ? min(m0 + row, p.M - 1) : min(n0 + row, p.N - 1);
      src[j] = (a ? p.A : p.B) + gr * K + kb + kc * 8;
      kstep[j] = BK;
    }
  }
  const int nk = int((ke - kb) / BK);
  auto issue = [&](int stage, int kstage) {
    const int64_t ks = int64_t(min(kstage, nk - 1));
#pragma unroll
    for (int j = 0; j < PW; ++j) {
      uint4* dst = isA[j] ? &sA[stage][dst_off[j]] : &sB[stage][dst_off[j]];
      const uint16_t* g = (TA || TB) ? src[j] + ks * kstep[j] : src[j] + ks * BK;
      __builtin_amdgcn_global_load_lds((glb_void*)g, (lds_void*)dst, 16, 0, 0);
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
  int offA[NS][FM], offB[NS][FN];
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    const int kc = s * 2 + lh;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int row = wm * WM + i * 32 + lr;
      offA[s][i] = row * CPR + pp_chunk<BK>(row, kc);
    }
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int row = wn * WN + j * 32 + lr;
      offB[s][j] = row * CPR + pp_chunk<BK>(row, kc);
    }
  }
  int toA[FM], toB[FN];  // K-slow fragments: byte offsets at substep 0, first half
#pragma unroll
  for (int i = 0; i < FM; ++i) toA[i] = TA ? tr_offset<BM>(wm * WM + i * 32, lane) : 0;
#pragma unroll
  for (int j = 0; j < FN; ++j) toB[j] = TB ? tr_offset<BN>(wn * WN + j * 32, lane) : 0;
  bf16x8 af[NS][FM], bfr[NS][FN];
  auto rd = [&](int st) {
    const char* stA = reinterpret_cast<const char*>(&sA[st][0]);
    const char* stB = reinterpret_cast<const char*>(&sB[st][0]);
#pragma unroll
    for (int s = 0; s < NS; ++s) {
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        if constexpr (TA) af[s][i] = tr_fragment(stA, toA[i] + 16 * s * BM * 2, toA[i] + (16 * s + 4) * BM * 2);
        else af[s][i] = __builtin_bit_cast(bf16x8, sA[st][offA[s][i]]);
      }
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        if constexpr (TB) bfr[s][j] = tr_fragment(stB, toB[j] + 16 * s * BN * 2, toB[j] + (16 * s + 4) * BN * 2);
        else bfr[s][j] = __builtin_bit_cast(bf16x8, sB[st][offB[s][j]]);
      }
    }
  };

#pragma unroll
  for (int s = 0; s < S - 1; ++s) issue(s, s);
  wait_vmcnt<(S - 2) * PW>();  // this wavefront's share of stage 0
  __builtin_amdgcn_s_barrier();
  if (grp == 1) __builtin_amdgcn_s_barrier();
  for (int k = 0; k < nk; ++k) {
    // memory phase: fragments of stage k, copy of stage k+S-1 into the slot
    // stage k-1 used (both groups finished reading it a phase ago)
    __builtin_amdgcn_sched_barrier(0);
    rd(k % S);
    issue((k + S - 1) % S, k + S - 1);
    wait_vmcnt<(S - 2) * PW>();            // this wavefront's share of stage k+1
    __builtin_amdgcn_s_waitcnt(0xC07F);    // lgkmcnt(0): fragments in registers
    __builtin_amdgcn_s_barrier();
    // MFMA phase
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int s = 0; s < NS; ++s)
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[s][i], bfr[s][j], acc[i][j], 0, 0, 0);
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_barrier();
  }
  if (grp == 0) __builtin_amdgcn_s_barrier();
  wait_vmcnt<0>();   // the reloads past the end have landed
  __syncthreads();   // every wave is past its last operand read: the stages become epilogue scratch
  epilogue<BM, BN, EPI, WM, WN, 8>(p, acc, m0, n0, wm, wn, lane, wave, tid, reinterpret_cast<float*>(smem));
}

template <int BM, int BN>
static int tiles(int64_t M, int64_t N) {
  return int(((M + BM - 1) / BM) * ((N + BN - 1) / BN));
}

// Tile shape: the largest of 256x256, 256x128, 128x128 that still gives at
// least one workgroup per compute unit (larger tiles move fewer operand
// bytes per flop through L2 and LDS).
enum TileShape { T256x256, T256x128, T128x128 };
static TileShape pick(int64_t M, int64_t N, int64_t batch = 1) {
  const int64_t nb = batch > 1 ? batch : 1;
  // a 256-wide side only where the matrix is wider than 128 (no half-empty tiles)
  if (M > 128 && N > 128 && tiles<256, 256>(M, N) * nb >= 256) return T256x256;
  if (M > 128 && tiles<256, 128>(M, N) * nb >= 256) return T256x128;
  return T128x128;
}

size_t gemm_workgroups(int64_t M, int64_t N, int /*epi*/) {
  switch (pick(M, N)) {
    case T256x256: return size_t(tiles<256, 256>(M, N));
    case T256x128: return size_t(tiles<256, 128>(M, N));
    default: return size_t(tiles<128, 128>(M, N));
  }
}

// Products with K a multiple of 32 on 256-row tiles (single, batched or
// causal): the ping-pong kernel; on 128-row tiles: the pipelined kernel; the
// register-staged kernel (any K that is a multiple of 8) otherwise.
template <int BM, int BN, int EPI>
static void launch_epi(const GemmArgs& a, dim3 grid, hipStream_t st) {
  if constexpr (BM == 256 && (BN == 256 || BN == 128)) {
    if (a.K % 32 == 0) {
      // 64-deep stages where 256 x 128 tiles allow them (three fit in LDS)
      if constexpr (BN == 128) {
        if (a.K % 64 == 0) {
          hipLaunchKernelGGL((gemm_pp_kernel<BM, BN, EPI, 4, 64>), grid, dim3(512), 0, st, a);
          return;
        }
      }
      hipLaunchKernelGGL((gemm_pp_kernel<BM, BN, EPI>), grid, dim3(512), 0, st, a);
      return;
    }
  }
  if (a.K % 32 == 0) hipLaunchKernelGGL((gemm_pipe_kernel<BM, BN, EPI, 4>), grid, dim3(256), 0, st, a);
  else hipLaunchKernelGGL((gemm_nt_kernel<BM, BN, EPI>), grid, dim3(256), 0, st, a);
}

template <int BM, int BN>
static hipError_t launch_bm(const GemmLaunch& q, hipStream_t st) {
  GemmArgs a;
  a.A = q.A; a.B = q.B; a.M = q.M; a.N = q.N; a.K = q.K;
  a.Yt = q.Yt; a.out = q.out; a.partials = q.partials; a.scale = q.scale;
  a.Rres = q.Rres;
  a.bsa = q.bsa; a.bsb = q.bsb; a.bso = q.bso;
  a.causal = q.causal;
  a.tiles_m = int((q.M + BM - 1) / BM);
  a.tiles_n = int((q.N + BN - 1) / BN);
  const dim3 grid(unsigned(a.tiles_m * a.tiles_n), unsigned(q.batch > 1 ? q.batch : 1));
  switch (q.epi) {
    case EPI_TARGET: launch_epi<BM, BN, EPI_TARGET>(a, grid, st); break;
    case EPI_LOSS:
      if (a.Yt != nullptr) launch_epi<BM, BN, EPI_LOSS>(a, grid, st);
      else launch_epi<BM, BN, EPI_LOSS_RES>(a, grid, st);
      break;
    case EPI_LOSS_BLOCK: launch_epi<BM, BN, EPI_LOSS_BLOCK>(a, grid, st); break;
    case EPI_RESID: launch_epi<BM, BN, EPI_RESID>(a, grid, st); break;
    case EPI_GRAD_BF16: launch_epi<BM, BN, EPI_GRAD_BF16>(a, grid, st); break;
    default: launch_epi<BM, BN, EPI_GRAD_F32>(a, grid, st); break;
  }
  return hipGetLastError();
}

// Weight-gradient GEMM with the fused straight-through backward: 256 x 256
// tiles, on the ping-pong kernel where there are at least 256 of them and on
// the pipelined kernel otherwise; both use 128-column wave tiles, which hold
// whole groups for g <= 128.  K % 32 == 0.
hipError_t launch_gemm_ste(const GemmLaunch& q, int k, hipStream_t st) {
  GemmArgs a;
  a.A = q.A; a.B = q.B; a.M = q.M; a.N = q.N; a.K = q.K;
  a.Yt = nullptr; a.out = nullptr; a.partials = nullptr; a.scale = q.scale;
  a.ste = q.ste;
  a.bsa = a.bsb = a.bso = 0;
  a.causal = 0;
  // ping-pong kernel (4 x 2 wave grid: 64 x 128 wave tiles) where the shape
  // gives at least one 256 x 256 tile per CU: the epilogue's memory phase then
  // runs on eight wavefronts per CU
  if (tiles<256, 256>(q.M, q.N) >= 256) {
    a.tiles_m = int((q.M + 255) / 256);
    a.tiles_n = int((q.N + 255) / 256);
    const dim3 grid(unsigned(a.tiles_m * a.tiles_n));
    switch (k) {
      case 1: hipLaunchKernelGGL((gemm_pp_kernel<256, 256, EPI_STE + 1, 4>), grid, dim3(512), 0, st, a); break;
      case 2: hipLaunchKernelGGL((gemm_pp_kernel<256, 256, EPI_STE + 2, 4>), grid, dim3(512), 0, st, a); break;
      case 3: hipLaunchKernelGGL((gemm_pp_kernel<256, 256, EPI_STE + 3, 4>), grid, dim3(512), 0, st, a); break;
      default: hipLaunchKernelGGL((gemm_pp_kernel<256, 256, EPI_STE + 4, 4>), grid, dim3(512), 0, st, a); break;
    }
    return hipGetLastError();
  }
  a.tiles_m = int((q.M + 255) / 256);
  a.tiles_n = int((q.N + 255) / 256);
  const dim3 grid(unsigned(a.tiles_m * a.tiles_n));
  switch (k) {
    case 1: hipLaunchKernelGGL((gemm_pipe_kernel<256, 256, EPI_STE + 1, 4>), grid, dim3(256), 0, st, a); break;
    case 2: hipLaunchKernelGGL((gemm_pipe_kernel<256, 256, EPI_STE + 2, 4>), grid, dim3(256), 0, st, a); break;
    case 3: hipLaunchKernelGGL((gemm_pipe_kernel<256, 256, EPI_STE + 3, 4>), grid, dim3(256), 0, st, a); break;
    default: hipLaunchKernelGGL((gemm_pipe_kernel<256, 256, EPI_STE + 4, 4>), grid, dim3(256), 0, st, a); break;
  }
  return hipGetLastError();
}

// Products with an operand stored K-slow: the ping-pong kernel with 32-deep
// stages on 256 x 256 tiles where there are at least 256 of them, on
// 256 x 128 tiles otherwise.  K % 32 == 0, M % 8 == 0 when A is K-slow.
template <int BM, int BN, int EPI>
static void launch_kslow(const GemmArgs& a, int ta, int tb, hipStream_t st) {
  const dim3 grid(unsigned(a.tiles_m * a.tiles_n));
  constexpr int WMM = BN == 256 ? 2 : 4;
  if (ta && tb) hipLaunchKernelGGL((gemm_pp_kernel<BM, BN, EPI, WMM, 32, true, true>), grid, dim3(512), 0, st, a);
  else if (tb) hipLaunchKernelGGL((gemm_pp_kernel<BM, BN, EPI, WMM, 32, false, true>), grid, dim3(512), 0, st, a);
  else hipLaunchKernelGGL((gemm_pp_kernel<BM, BN, EPI, WMM, 32, true, false>), grid, dim3(512), 0, st, a);
}

static hipError_t launch_gemm_kslow(const GemmLaunch& q, hipStream_t st) {
  GemmArgs a;
  a.A = q.A; a.B = q.B; a.M = q.M; a.N = q.N; a.K = q.K;
  a.Yt = nullptr; a.out = q.out; a.partials = nullptr; a.scale = q.scale;
  a.bsa = a.bsb = a.bso = 0;
  a.causal = 0;
  a.swiglu = q.swiglu;
  if (a.swiglu.ldo == 0) a.swiglu.ldo = q.N;
  const bool wide = q.M > 128 && q.N > 128 && tiles<256, 256>(q.M, q.N) >= 256;
  const int BN = wide ? 256 : 128;
  a.tiles_m = int((q.M + 255) / 256);
  a.tiles_n = int((q.N + BN - 1) / BN);
  const bool bf = q.epi == EPI_GRAD_BF16;
  if (q.epi == EPI_SWIGLU_BWD) {  // input-gradient product dH = E W_d: B K-slow, 256 x 256 tiles
    a.tiles_n = int((q.N + 255) / 256);
    hipLaunchKernelGGL((gemm_pp_kernel<256, 256, EPI_SWIGLU_BWD, 2, 32, false, true>),
                       dim3(unsigned(a.tiles_m * a.tiles_n)), dim3(512), 0, st, a);
    return hipGetLastError();
  }
  if (wide) {
    if (bf) launch_kslow<256, 256, EPI_GRAD_BF16>(a, q.ta, q.tb, st);
    else launch_kslow<256, 256, EPI_GRAD_F32>(a, q.ta, q.tb, st);
  } else {
    if (bf) launch_kslow<256, 128, EPI_GRAD_BF16>(a, q.ta, q.tb, st);
    else launch_kslow<256, 128, EPI_GRAD_F32>(a, q.ta, q.tb, st);
  }
  return hipGetLastError();
}

// Head-split products (EPI_HEADS*): 256 x 256 tiles on the ping-pong kernel
// with a 4 x 2 wave grid (64 x 128 wave tiles: a wave holds whole heads).
// K % 32 == 0, N % 128 == 0.
static hipError_t launch_gemm_heads(const GemmLaunch& q, hipStream_t st) {
  GemmArgs a;
  a.A = q.A; a.B = q.B; a.M = q.M; a.N = q.N; a.K = q.K;
  a.Yt = nullptr; a.out = q.out; a.partials = nullptr; a.scale = q.scale;
  a.bsa = a.bsb = a.bso = 0;
  a.causal = 0;
  a.heads = q.heads;
  a.tiles_m = int((q.M + 255) / 256);
  a.tiles_n = int((q.N + 255) / 256);
  const dim3 grid(unsigned(a.tiles_m * a.tiles_n));
  if (q.epi == EPI_HEADS_ROT)
    hipLaunchKernelGGL((gemm_pp_kernel<256, 256, EPI_HEADS_ROT, 4>), grid, dim3(512), 0, st, a);
  else
    hipLaunchKernelGGL((gemm_pp_kernel<256, 256, EPI_HEADS, 4>), grid, dim3(512), 0, st, a);
  return hipGetLastError();
}

// Gate and up products with the SiLU product (EPI_SWIGLU): 256 x 256 tiles
// of the interleaved columns (128 rows of W each) on the ping-pong kernel
// with the 2 x 4 wave grid.  K % 32 == 0, I % 32 == 0.
static hipError_t launch_gemm_swiglu(const GemmLaunch& q, hipStream_t st) {
  GemmArgs a;
  a.A = q.A; a.B = q.B; a.M = q.M; a.N = 2 * q.swiglu.I; a.K = q.K;
  a.Yt = nullptr; a.out = q.out; a.partials = nullptr; a.scale = q.scale;
  a.bsa = a.bsb = a.bso = 0;
  a.causal = 0;
  a.swiglu = q.swiglu;
  a.tiles_m = int((q.M + 255) / 256);
  a.tiles_n = int((a.N + 255) / 256);
  hipLaunchKernelGGL((gemm_pp_kernel<256, 256, EPI_SWIGLU>), dim3(unsigned(a.tiles_m * a.tiles_n)), dim3(512), 0, st,
                     a);
  return hipGetLastError();
}

hipError_t launch_gemm(const GemmLaunch& q, hipStream_t st) {
  if (q.epi == EPI_SWIGLU) return launch_gemm_swiglu(q, st);
  if (q.epi == EPI_HEADS || q.epi == EPI_HEADS_ROT) return launch_gemm_heads(q, st);
  if (q.ta || q.tb) return launch_gemm_kslow(q, st);
  switch (pick(q.M, q.N, q.batch)) {
    case T256x256: return launch_bm<256, 256>(q, st);
    case T256x128: return launch_bm<256, 128>(q, st);
    default: return launch_bm<128, 128>(q, st);
  }
}

// Deterministic loss: fixed strided fp64 partial sums, a fixed xor butterfly
// within each wavefront, then the four wavefront totals in order.
__global__ __launch_bounds__(256) void reduce_loss_kernel(const float* __restrict__ partials, int64_t n,
                                                          float* __restrict__ loss) {
  __shared__ double sm[4];
  double acc = 0.0;
  for (int64_t i = threadIdx.x; i < n; i += 256) acc += double(partials[i]);
  for (int msk = 32; msk >= 1; msk >>= 1) acc += __shfl_xor(acc, msk, 64);
  if ((threadIdx.x & 63) == 0) sm[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) loss[0] = float((sm[0] + sm[1]) + (sm[2] + sm[3]));
}

hipError_t launch_reduce_loss(const float* partials, int64_t n, float* loss, hipStream_t st) {
  hipLaunchKernelGGL(reduce_loss_kernel, dim3(1), dim3(256), 0, st, partials, n, loss);
  return hipGetLastError();
}

// Loss partials of uniquan_layer_recon_noalloc: a fixed array in device
// memory (one copy per GPU, for the life of the process) instead of a
// caller-provided workspace.  Host code never passes `scratch` itself to a
// kernel: its device address on the current GPU is looked up once per device
// with hipGetSymbolAddress and kept.  Every workgroup of the loss GEMM writes
// its own partial and the reduction reads exactly those, so nothing needs
// clearing between calls; calls that overlap on one GPU share the array and
// race.
static __device__ __align__(256) float scratch[kNoallocPartials];

hipError_t noalloc_scratch(float** out) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static float* ptrs[kMaxDevices] = {};
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (ptrs[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    ptrs[dev] = static_cast<float*>(p);
  }
  *out = ptrs[dev];
  return hipSuccess;
}

// out[c, r] = in[r, c] for rows and cols multiples of 8: 64 x 64 tiles
// through LDS with 16-byte global accesses (8 bf16 per lane).  A load chunk
// is 8 consecutive columns of one input row; a store chunk is 8 consecutive
// input rows of one column, and the 8 lanes of an output row write its 128
// bytes together.  Chunks past the edge of the matrix are skipped whole.
__global__ __launch_bounds__(256) void transpose_kernel(const uint16_t* __restrict__ in, uint16_t* __restrict__ out,
                                                        int64_t rows, int64_t cols) {
  __shared__ __align__(16) uint16_t t[64][72];  // 144-byte rows keep 16-byte chunks aligned
  const int64_t r0 = int64_t(blockIdx.y) * 64, c0 = int64_t(blockIdx.x) * 64;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int k = threadIdx.x + 256 * h;
    const int r = k >> 3, c8 = (k & 7) * 8;
    uint4 v = make_uint4(0u, 0u, 0u, 0u);
    if (r0 + r < rows && c0 + c8 < cols) v = *reinterpret_cast<const uint4*>(in + (r0 + r) * cols + c0 + c8);
    *reinterpret_cast<uint4*>(&t[r][c8]) = v;
  }
  __syncthreads();
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int k = threadIdx.x + 256 * h;
    const int c = k >> 3, r8 = (k & 7) * 8;  // output row c0 + c, columns r0 + r8 .. + 8
    if (c0 + c < cols && r0 + r8 < rows) {
      uint32_t w[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) w[j] = uint32_t(t[r8 + 2 * j][c]) | (uint32_t(t[r8 + 2 * j + 1][c]) << 16);
      *reinterpret_cast<uint4*>(out + (c0 + c) * rows + r0 + r8) = make_uint4(w[0], w[1], w[2], w[3]);
    }
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
