// Causal attention of the block-level reconstruction (Algorithm 1 with a
// Transformer block; appendix "Units in LLMs") with the score tiles kept on
// chip: no [L, L] score, probability or gradient array is written.
//
// Per sequence and query head b (key/value head b mod kv_batch), d = 128,
// with c = scale * log2(e):
//   S = Q K^T (fp32), lse_i = log2 sum_{j <= i} 2^(c S_ij) (base-2 log-sum-exp
//   of the scaled scores), P = bf16(2^(c S - lse)) (the causal row softmax),
//   O = bf16(P V) (fp32 accumulation);
//   backward with dP = dO V^T (fp32), delta_i = dO_i . O_i (fp32, from the
//   stored bf16 O and dO; equal to sum_j P_ij dP_ij in exact arithmetic),
//   dS = bf16(P (dP - delta)), dQ = dS K * scale, and per query head the
//   contributions dK_b = dS^T Q * scale, dV_b = P^T dO (fp32 out; the
//   gradient of a shared key/value head is the sum of its query heads').
// These are the rounding points of the unfused path (P and dS stored in
// bf16, S and dP in fp32).  The forward runs two passes over the keys: the
// first finds each row's maximum and exp-sum (online, per lane, then the two
// half-waves of a query combined) and so lse; the second forms P from lse and
// accumulates P V.  The backward recomputes the same P from the stored lse.
//
// MFMA layout (v_mfma_f32_32x32x16_bf16, C[m][n] += A[m][k] B[n][k]): lane l
// supplies row l % 32 of A and of B with k = 8 (l / 32) .. + 8, and holds
// C rows 8 (r / 4) + 4 (l / 32) + r % 4, r < 16, of column l % 32.  A score
// tile is computed with the 32 rows of its key (or query) tile as M, read
// from LDS in the order perm32 (bits 2 and 3 of the row index swapped): then
// accumulator slot r of lane l belongs to tile row 16 (r / 8) + 8 (l / 32) +
// r % 8, so the 8 values of each half (slots 8 h .. 8 h + 7) are 8
// consecutive rows and serve directly as the B operand of the next product
// (contraction over those rows), whose A operand (d rows, the tile's rows as
// k) comes from the same row tile through two LDS transpose reads.
//
// Tiles (32 rows of 128 bf16, as stored: Q, K, V, dO) go straight from
// global memory into a ring of S LDS stages (global_load_lds, 16 bytes per
// lane, S - 1 tiles ahead); each wave waits for its own copies with an exact
// vmcnt before the workgroup barrier that precedes the reads, and the barrier
// also orders the reuse of a stage.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "uq_launch.h"

namespace uq {

namespace {

typedef __bf16 bf16x8a __attribute__((ext_vector_type(8)));
typedef float f32x16a __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4a __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2a __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void_a;
typedef const __attribute__((address_space(1))) void glb_void_a;

constexpr int D = 128;                       // head dimension
constexpr int NB = 32;                       // rows (keys or queries) per tile
constexpr int TILE16 = NB * D * 2 / 16;      // 16-byte slots of a tile (512)
constexpr float LOG2E = 1.44269504088896341f;

__device__ __forceinline__ f32x16a mfma(const bf16x8a& a, const bf16x8a& b, const f32x16a& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float exp2a(float x) { return __builtin_amdgcn_exp2f(x); }

// bf16 value nearest to x (ties to even), as fp32.
__device__ __forceinline__ float bf16_round(float x) { return float(__bf16(x)); }

// Tile row held by accumulator slot r of this lane (rows read in perm32 order).
__device__ __forceinline__ int slot_row(int r, int lane) { return 16 * (r >> 3) + 8 * (lane >> 5) + (r & 7); }

// Swap bits 2 and 3 of a row index below 32 (an involution).
__device__ __forceinline__ int perm32(int r) { return (r & 19) | ((r & 4) << 1) | ((r >> 1) & 4); }

template <int N>
__device__ __forceinline__ void vm_wait() {
  // s_waitcnt fields: vmcnt[3:0] and [15:14], expcnt[6:4], lgkmcnt[11:8]
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Wait until at most `ahead` (0..2) later tiles of PW copies each are in flight.
template <int PW>
__device__ __forceinline__ void wait_tiles(int ahead) {
  if (ahead >= 2) vm_wait<2 * PW>();
  else if (ahead == 1) vm_wait<PW>();
  else vm_wait<0>();
}

__device__ __forceinline__ void lds_wait_barrier() {
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): this wave's LDS reads are done
  __builtin_amdgcn_s_barrier();
}

// Chunk swizzle of tile row rho: the two 2-bit fields of rho % 16 swapped.
// It is a bijection on rho % 16, so the 16 rows a quarter-wavefront reads at
// one chunk fall in 16 distinct slots, and four consecutive rows differ in
// bits 2-3, so the two adjacent chunks of four consecutive rows that a
// transpose read takes also fall in 8 distinct slots.
__device__ __forceinline__ int swz(int rho) { return ((rho & 3) << 2) | ((rho >> 2) & 3); }

// Row tile (32 rows of 128 bf16 = 512 slots of 16 bytes): slot s holds chunk
// (s % 16) ^ swz(rho) of tile row rho = s / 16, and tile row rho holds
// source row perm32(rho) of the tile.  Copy block blk fills slots 64 blk ..
// + 64; row_off is this lane's byte offset in the source tile for block blk.
__device__ __forceinline__ uint32_t row_off(int blk, int lane, int ld = D) {
  const int s = blk * 64 + lane;
  const int rho = s >> 4, c = (s & 15) ^ swz(rho);
  return uint32_t(perm32(rho)) * uint32_t(ld) * 2u + uint32_t(c * 16);
}

// A copy of 64 slots: lane l's 16 bytes at base + off land in slot l of dst.
__device__ __forceinline__ void copy16(const void* base, uint32_t off, u32x4a* dst) {
  __builtin_amdgcn_global_load_lds((glb_void_a*)(static_cast<const char*>(base) + off), (lds_void_a*)dst, 16, 0, 0);
}

// A or B fragment of k-step j (d = 16 j + 8 (lane / 32) .. + 8) of tile row lane % 32.
__device__ __forceinline__ bf16x8a row_frag(const u32x4a* tile, int j, int lane) {
  const int rho = lane & 31, c = 2 * j + (lane >> 5);
  return __builtin_bit_cast(bf16x8a, tile[rho * 16 + (c ^ swz(rho))]);
}

typedef short v4i16a __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16a lds_v4i16a;

// A fragment of the transposed row tile: rows d = 32 db .. + 32 over the 16
// tile rows (keys or queries, in source order) of half h; lane supplies
// d = 32 db + lane % 32 and source rows 16 h + 8 (lane / 32) .. + 8.
// ds_read_b64_tr_b16 gives lane i of each 16-lane group, in slot j, element
// i % 4 of the 8 bytes addressed by lane 4 j + i / 4 of the group; lane
// 4 j + q addresses source row r0 + j, columns d0 + 4 q .. + 3, so lane i
// receives column d0 + i of rows r0 .. r0 + 3: half the fragment.
__device__ __forceinline__ bf16x8a col_frag(const u32x4a* tile, int db, int h, int lane) {
  const int g = lane >> 4, i = lane & 15;
  const int d = 32 * db + 16 * (g & 1) + 4 * (i & 3);
  const char* base = reinterpret_cast<const char*>(tile);
  v4i16a part[2];
#pragma unroll
  for (int hh = 0; hh < 2; ++hh) {
    const int rho = perm32(16 * h + 8 * (g >> 1) + 4 * hh + (i >> 2));
    const int off = rho * D * 2 + (((d >> 3) ^ swz(rho)) << 4) + ((d & 7) >> 2) * 8;
    part[hh] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16a*)(base + off));
  }
  return __builtin_bit_cast(bf16x8a, part);
}

// Slots 8 h .. 8 h + 7 as a bf16 B operand.
__device__ __forceinline__ bf16x8a pack_half(const float (&v)[16], int h) {
  bf16x8a w;
#pragma unroll
  for (int i = 0; i < 8; ++i) w[i] = __bf16(v[8 * h + i]);
  return w;
}

__device__ __forceinline__ f32x16a zero16() {
  f32x16a z;
#pragma unroll
  for (int r = 0; r < 16; ++r) z[r] = 0.0f;
  return z;
}

// 16 fp32 accumulator values of 32 rows db (4 per row group) at this lane's
// column: store rows 32 db + 8 g4 + 4 (lane / 32) .. + 4 of column `row`.
__device__ __forceinline__ void store_f32_rows(float* out, const f32x16a (&acc)[4], float mul, int lane) {
#pragma unroll
  for (int db = 0; db < 4; ++db)
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
      const int d0 = 32 * db + 8 * g4 + 4 * (lane >> 5);
      *reinterpret_cast<float4*>(out + d0) = make_float4(acc[db][4 * g4] * mul, acc[db][4 * g4 + 1] * mul,
                                                         acc[db][4 * g4 + 2] * mul, acc[db][4 * g4 + 3] * mul);
    }
}

// 16 accumulator values per d block (rows d = 32 db + 8 g4 + 4 (lane / 32) ..
// + 4, scaled by mul) of this lane's row stored as one bf16 row of 128: the
// pairs (j, j + 64) (d blocks db and db + 2 of one lane) rotated by minus the
// angle of position pos when ROT, y1 = x1 c + x2 s, y2 = x2 c - x1 s, with
// x = 0 + mul acc (the arithmetic of the stand-alone inverse split, which
// sums its partials from zero).
template <bool ROT>
__device__ __forceinline__ void store_bf16_row(uint16_t* out, const f32x16a (&acc)[4], float mul, const float* cs,
                                               int pos, int lane) {
#pragma unroll
  for (int db = 0; db < 2; ++db)
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
      const int j0 = 32 * db + 8 * g4 + 4 * (lane >> 5);
      float y1[4], y2[4];
      float4 c01 = {}, c23 = {};
      if constexpr (ROT) {
        const float4* t = reinterpret_cast<const float4*>(cs + (int64_t(pos) * 64 + j0) * 2);
        c01 = t[0];
        c23 = t[1];
      }
      const float cn[4] = {c01.x, c01.z, c23.x, c23.z}, sn[4] = {c01.y, c01.w, c23.y, c23.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float x1 = 0.0f + acc[db][4 * g4 + e] * mul;
        const float x2 = 0.0f + acc[db + 2][4 * g4 + e] * mul;
        if constexpr (ROT) {
          y1[e] = x1 * cn[e] + x2 * sn[e];
          y2[e] = x2 * cn[e] - x1 * sn[e];
        } else {
          y1[e] = x1;
          y2[e] = x2;
        }
      }
      bf16x8a w;  // the first four halves of each store
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        w[e] = __bf16(y1[e]);
        w[4 + e] = __bf16(y2[e]);
      }
      const u32x4a u = __builtin_bit_cast(u32x4a, w);
      *reinterpret_cast<u32x2a*>(out + j0) = u32x2a{u.x, u.y};
      *reinterpret_cast<u32x2a*>(out + j0 + 64) = u32x2a{u.z, u.w};
    }
}

// Workgroup -> (row block, batch).  When the batch count is a multiple of 8
// the row blocks of one batch go to one XCD (workgroups are dealt to the 8
// XCDs round-robin), so its keys and values stay in that XCD's L2; within a
// batch the blocks with the most work come first.
__device__ __forceinline__ void block_of(int nblk, int64_t batch, int& blk, int64_t& b) {
  const int64_t w = blockIdx.x;
  if ((batch & 7) == 0) {
    const int64_t y = w >> 3;
    b = (w & 7) + 8 * (y / nblk);
    blk = nblk - 1 - int(y % nblk);
  } else {
    b = w / nblk;
    blk = nblk - 1 - int(w % nblk);
  }
}

}  // namespace

struct AttnArgs {
  int64_t batch, kv_batch;
  int L;
  float scale;
  const uint16_t* Q;    // [batch, L, D]
  const uint16_t* K;    // [kv_batch, L, D]
  const uint16_t* V;    // [kv_batch, L, D]
  const uint16_t* O;    // [batch, L, D]
  const uint16_t* dO;   // [batch, L, D]
  uint16_t* O_out;      // [batch, L, D]
  float* lse;           // [batch, L] base-2 log-sum-exp of the scaled scores
  float* delta;         // [batch, L]
  float* dQ;            // [batch, L, D]
  float* dK;            // [batch, L, D] per query head
  float* dV;            // [batch, L, D] per query head
  // token-major I/O (TOK kernels): O, dO and the bf16 gradients as rows of
  // [n_seq L, heads D]; query batch b = slot n_seq + s is head h(slot) of
  // sequence s, h(slot) = (slot % (heads / grp)) grp + slot / (heads / grp)
  // (the grouped slot order of the projections' head split)
  int n_seq, heads, grp;
  const float* cs;      // rotary (cos, sin) [L, 64]: the gradients' inverse rotation
  uint16_t* dQ_tok;     // bf16 [n_seq L, heads D]
  uint16_t* dK_tok;     // bf16, when kv_batch == batch (else dK, dV per query head)
  uint16_t* dV_tok;
};

// Element offset of row l of query batch b in the token-major layout.
__device__ __forceinline__ int64_t tok_off(const AttnArgs& a, int64_t b, int l) {
  const int slot = int(b / a.n_seq), s = int(b % a.n_seq);
  const int per = a.heads / a.grp;
  const int h = (slot % per) * a.grp + slot / per;
  return (int64_t(s) * a.L + l) * (int64_t(a.heads) * D) + int64_t(h) * D;
}

// Copies of one tile: PW blocks of 64 slots per wave (blocks wave PW .. + PW).
template <int PW>
__device__ __forceinline__ void copy_tile(const uint16_t* base, const uint32_t (&off)[PW], u32x4a* tile, int wave) {
#pragma unroll
  for (int q = 0; q < PW; ++q) copy16(base, off[q], tile + (wave * PW + q) * 64);
}

// Forward: one workgroup of NW waves per (NW * 32 queries, query batch); wave
// w owns 32 queries and multiplies the key tiles up to its diagonal (the
// workgroup copies the tiles up to its last diagonal).  Key and value
// fragments go from LDS straight into their MFMAs rather than into arrays
// held across the tile: 156 registers, so three waves share a SIMD and one
// wave's exponentials overlap another's products (two waves per SIMD at 243).
template <int NW, int S, bool TOK>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(3))) void attn_fwd_kernel(AttnArgs a) {
  constexpr int QB = NW * NB;
  constexpr int PW = 8 / NW;  // copy blocks per wave and tile
  constexpr int STAGE = 2 * TILE16;  // key tile, value tile
  __shared__ u32x4a smem[S * STAGE];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x >> 6));
  const int L = a.L;
  int qb;
  int64_t b;
  block_of((L + QB - 1) / QB, a.batch, qb, b);
  const int64_t bk = b % a.kv_batch;
  const int q0 = qb * QB + wave * NB;
  const bool active = q0 < L;
  const int qi = q0 + (lane & 31);  // this lane's query
  const int n_tiles = min(L, qb * QB + QB) / NB;
  const int my_tiles = active ? q0 / NB + 1 : 0;
  const uint16_t* Kb = a.K + bk * int64_t(L) * D;
  const uint16_t* Vb = a.V + bk * int64_t(L) * D;
  const float c = a.scale * LOG2E;
  uint32_t ro[PW];
#pragma unroll
  for (int q = 0; q < PW; ++q) ro[q] = row_off(wave * PW + q, lane);
  bf16x8a qf[8];
  {
    const uint16_t* qrow = a.Q + (b * L + min(qi, L - 1)) * int64_t(D) + 8 * (lane >> 5);
#pragma unroll
    for (int j = 0; j < 8; ++j) qf[j] = __builtin_bit_cast(bf16x8a, *reinterpret_cast<const u32x4a*>(qrow + 16 * j));
  }
  // pass 1: running maximum m (of c S) and sum l of 2^(c S - m) over this lane's keys
  float m = -INFINITY, l = 0.0f;
#pragma unroll
  for (int t = 0; t < S - 1; ++t)
    if (t < n_tiles) copy_tile<PW>(Kb + int64_t(t) * NB * D, ro, smem + (t % S) * STAGE, wave);
  for (int t = 0; t < n_tiles; ++t) {
    wait_tiles<PW>(min(S - 2, n_tiles - 1 - t));
    lds_wait_barrier();
    if (t + S - 1 < n_tiles) {
      const int u = t + S - 1;
      copy_tile<PW>(Kb + int64_t(u) * NB * D, ro, smem + (u % S) * STAGE, wave);
    }
    if (t >= my_tiles) continue;
    const u32x4a* tk = smem + (t % S) * STAGE;
    f32x16a s = zero16();
#pragma unroll
    for (int j = 0; j < 8; ++j) s = mfma(row_frag(tk, j, lane), qf[j], s);
    if (t == my_tiles - 1) {
#pragma unroll
      for (int r = 0; r < 16; ++r)
        if (t * NB + slot_row(r, lane) > qi) s[r] = -INFINITY;
    }
    float mx = s[0];
#pragma unroll
    for (int r = 1; r < 16; ++r) mx = fmaxf(mx, s[r]);
    const float mt = fmaxf(m, mx * c);
    const float ms = mt == -INFINITY ? 0.0f : mt;
    float sum = 0.0f;
#pragma unroll
    for (int r = 0; r < 16; ++r) sum += exp2a(fmaf(s[r], c, -ms));
    l = l * exp2a(m - ms) + sum;
    m = mt;
  }
  // the two half-waves of a query (lower half first) -> lse
  float lse;
  {
    const float m2 = __shfl_xor(m, 32, 64), l2 = __shfl_xor(l, 32, 64);
    const float mlo = (lane < 32) ? m : m2, llo = (lane < 32) ? l : l2;
    const float mhi = (lane < 32) ? m2 : m, lhi = (lane < 32) ? l2 : l;
    const float mm = fmaxf(mlo, mhi);
    const float ms = mm == -INFINITY ? 0.0f : mm;
    const float lt = llo * exp2a(mlo - ms) + lhi * exp2a(mhi - ms);
    lse = mm + __builtin_amdgcn_logf(lt);  // log2
  }
  lds_wait_barrier();  // every wave is past pass 1's reads before the stages are refilled
  // pass 2: P = bf16(2^(c S - lse)), O += P V
  f32x16a o[4] = {zero16(), zero16(), zero16(), zero16()};
#pragma unroll
  for (int t = 0; t < S - 1; ++t)
    if (t < n_tiles) {
      copy_tile<PW>(Kb + int64_t(t) * NB * D, ro, smem + (t % S) * STAGE, wave);
      copy_tile<PW>(Vb + int64_t(t) * NB * D, ro, smem + (t % S) * STAGE + TILE16, wave);
    }
  for (int t = 0; t < n_tiles; ++t) {
    wait_tiles<2 * PW>(min(S - 2, n_tiles - 1 - t));
    lds_wait_barrier();
    if (t + S - 1 < n_tiles) {
      const int u = t + S - 1;
      copy_tile<PW>(Kb + int64_t(u) * NB * D, ro, smem + (u % S) * STAGE, wave);
      copy_tile<PW>(Vb + int64_t(u) * NB * D, ro, smem + (u % S) * STAGE + TILE16, wave);
    }
    if (t >= my_tiles) continue;
    const u32x4a* tk = smem + (t % S) * STAGE;
    const u32x4a* tv = tk + TILE16;
    f32x16a s = zero16();
#pragma unroll
    for (int j = 0; j < 8; ++j) s = mfma(row_frag(tk, j, lane), qf[j], s);
    float p[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) p[r] = exp2a(fmaf(s[r], c, -lse));
    if (t == my_tiles - 1) {
#pragma unroll
      for (int r = 0; r < 16; ++r)
        if (t * NB + slot_row(r, lane) > qi) p[r] = 0.0f;
    }
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const bf16x8a pb = pack_half(p, h);
#pragma unroll
      for (int db = 0; db < 4; ++db) o[db] = mfma(col_frag(tv, db, h, lane), pb, o[db]);
    }
  }
  if (!active) return;
  uint16_t* orow = a.O_out + (TOK ? tok_off(a, b, qi) : (b * L + qi) * int64_t(D));
#pragma unroll
  for (int db = 0; db < 4; ++db)
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
      const int d0 = 32 * db + 8 * g4 + 4 * (lane >> 5);
      bf16x8a w;  // only the first four are stored
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        w[i] = __bf16(o[db][4 * g4 + (i & 3)]);
        // token-major: as the stand-alone merge stores it (0 + x: a -0 becomes +0)
        if (TOK) w[i] = __bf16(0.0f + float(w[i]));
      }
      const u32x4a u = __builtin_bit_cast(u32x4a, w);
      *reinterpret_cast<u32x2a*>(orow + d0) = u32x2a{u.x, u.y};
    }
  if (lane < 32) a.lse[b * L + qi] = lse;
}

// Backward for the queries: delta = dO . O per row, then per key tile
// S -> P (from lse), dP = dO V^T, dS = bf16(P (dP - delta)), dQ += dS K;
// dQ * scale stored in fp32, delta stored for the key kernel.
template <int NW, int S, bool TOK>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(2, 2))) void attn_bwd_dq_kernel(AttnArgs a) {
  constexpr int QB = NW * NB;
  constexpr int PW = 8 / NW;
  constexpr int STAGE = 2 * TILE16;  // key tile, value tile
  __shared__ u32x4a smem[S * STAGE];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x >> 6));
  const int L = a.L;
  int qb;
  int64_t b;
  block_of((L + QB - 1) / QB, a.batch, qb, b);
  const int64_t bk = b % a.kv_batch;
  const int q0 = qb * QB + wave * NB;
  const bool active = q0 < L;
  const int qi = q0 + (lane & 31);
  const int qc = min(qi, L - 1);
  const int n_tiles = min(L, qb * QB + QB) / NB;
  const int my_tiles = active ? q0 / NB + 1 : 0;
  const uint16_t* Kb = a.K + bk * int64_t(L) * D;
  const uint16_t* Vb = a.V + bk * int64_t(L) * D;
  const float c = a.scale * LOG2E;
  uint32_t ro[PW];
#pragma unroll
  for (int q = 0; q < PW; ++q) ro[q] = row_off(wave * PW + q, lane);
  bf16x8a qf[8], df[8];
  float dl = 0.0f;
  {
    const int64_t row = (b * L + qc) * int64_t(D) + 8 * (lane >> 5);
    const int64_t orow = (TOK ? tok_off(a, b, qc) : (b * L + qc) * int64_t(D)) + 8 * (lane >> 5);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      qf[j] = __builtin_bit_cast(bf16x8a, *reinterpret_cast<const u32x4a*>(a.Q + row + 16 * j));
      df[j] = __builtin_bit_cast(bf16x8a, *reinterpret_cast<const u32x4a*>(a.dO + orow + 16 * j));
      const bf16x8a ov = __builtin_bit_cast(bf16x8a, *reinterpret_cast<const u32x4a*>(a.O + orow + 16 * j));
#pragma unroll
      for (int i = 0; i < 8; ++i) dl += float(df[j][i]) * float(ov[i]);
    }
  }
  {  // delta: this lane's 64 d values plus the other half-wave's (lower half first)
    const float d2 = __shfl_xor(dl, 32, 64);
    dl = lane < 32 ? dl + d2 : d2 + dl;
  }
  const float lse = a.lse[b * L + qc];
  f32x16a dq[4] = {zero16(), zero16(), zero16(), zero16()};
#pragma unroll
  for (int t = 0; t < S - 1; ++t)
    if (t < n_tiles) {
      u32x4a* st = smem + (t % S) * STAGE;
      copy_tile<PW>(Kb + int64_t(t) * NB * D, ro, st, wave);
      copy_tile<PW>(Vb + int64_t(t) * NB * D, ro, st + TILE16, wave);
    }
  for (int t = 0; t < n_tiles; ++t) {
    wait_tiles<2 * PW>(min(S - 2, n_tiles - 1 - t));
    lds_wait_barrier();
    if (t + S - 1 < n_tiles) {
      const int u = t + S - 1;
      u32x4a* st = smem + (u % S) * STAGE;
      copy_tile<PW>(Kb + int64_t(u) * NB * D, ro, st, wave);
      copy_tile<PW>(Vb + int64_t(u) * NB * D, ro, st + TILE16, wave);
    }
    if (t >= my_tiles) continue;
    const u32x4a* tk = smem + (t % S) * STAGE;
    bf16x8a f[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) f[j] = row_frag(tk, j, lane);
    f32x16a s = zero16(), dp = zero16();
#pragma unroll
    for (int j = 0; j < 8; ++j) s = mfma(f[j], qf[j], s);
#pragma unroll
    for (int j = 0; j < 8; ++j) f[j] = row_frag(tk + TILE16, j, lane);
#pragma unroll
    for (int j = 0; j < 8; ++j) dp = mfma(f[j], df[j], dp);
#pragma unroll
    for (int i = 0; i < 8; ++i) f[i] = col_frag(tk, i & 3, i >> 2, lane);
    // dS in place of dP
#pragma unroll
    for (int r = 0; r < 16; ++r) dp[r] = bf16_round(exp2a(fmaf(s[r], c, -lse))) * (dp[r] - dl);
    if (t == my_tiles - 1) {
#pragma unroll
      for (int r = 0; r < 16; ++r)
        if (t * NB + slot_row(r, lane) > qi) dp[r] = 0.0f;
    }
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      bf16x8a sb;
#pragma unroll
      for (int i = 0; i < 8; ++i) sb[i] = __bf16(dp[8 * h + i]);
#pragma unroll
      for (int db = 0; db < 4; ++db) dq[db] = mfma(f[4 * h + db], sb, dq[db]);
    }
  }
  if (!active) return;
  if (lane < 32) a.delta[b * L + qi] = dl;
  if constexpr (TOK) store_bf16_row<true>(a.dQ_tok + tok_off(a, b, qi), dq, a.scale, a.cs, qi, lane);
  else store_f32_rows(a.dQ + (b * L + qi) * int64_t(D), dq, a.scale, lane);
}

// Backward for the keys and values of one query head: one workgroup of NW
// waves per (NW * 32 keys, query batch b); wave w owns 32 keys (K, V rows in
// registers) and multiplies the query tiles from its diagonal on.  S = Q K^T
// and dP = dO V^T have the query tile as M and this lane's key as column, so
// P and dS feed dV_b += P^T dO and dK_b += dS^T Q directly.  The row terms
// (lse, delta) of a query tile come through LDS: wave 0 copies them into a
// 1 KB slot of the stage (lanes 0-7 lse, 8-15 delta, the rest repeat them).
// To hold two workgroups of 256 registers per lane on a SIMD, the last NPARK
// of the wave's V fragments are kept in LDS and read back for each tile.
template <int NW, int S, bool TOK>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(2, 2))) void attn_bwd_dkv_kernel(AttnArgs a) {
  constexpr int KB = NW * NB;
  constexpr int PW = 8 / NW;
  constexpr int STAGE = 2 * TILE16 + 64;  // Q, dO tiles, row terms
  constexpr int NPARK = 3;
  __shared__ u32x4a smem[S * STAGE + NW * NPARK * 64];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x >> 6));
  const int L = a.L;
  int kb;
  int64_t b;
  block_of((L + KB - 1) / KB, a.batch, kb, b);
  const int64_t bk = b % a.kv_batch;
  const int k0 = kb * KB + wave * NB;
  const bool active = k0 < L;
  const int kj = k0 + (lane & 31);  // this lane's key
  const int kc = min(kj, L - 1);
  const int first = kb * KB / NB;   // first query tile of the workgroup
  const int n_tiles = L / NB;
  const int my_first = active ? k0 / NB : n_tiles;
  const float c = a.scale * LOG2E;
  const uint16_t* Qb = a.Q + b * int64_t(L) * D;
  // dO tile t starts at dOb + t NB ldo (token-major rows: a stride of heads D)
  const int ldo = TOK ? a.heads * D : D;
  const uint16_t* dOb = a.dO + (TOK ? tok_off(a, b, 0) : b * int64_t(L) * D);
  // row terms: lane (l % 16) copies 4 floats of lse (l % 16 < 8) or delta
  const float* rt_src = ((lane & 15) < 8 ? a.lse : a.delta) + b * L + 4 * (lane & 7);
  uint32_t ro[PW], rod[PW];
#pragma unroll
  for (int q = 0; q < PW; ++q) {
    ro[q] = row_off(wave * PW + q, lane);
    rod[q] = row_off(wave * PW + q, lane, ldo);
  }
  bf16x8a kf[8], vf[8 - NPARK];
  u32x4a* park = smem + S * STAGE + wave * NPARK * 64;
  {
    const int64_t row = (bk * L + kc) * int64_t(D) + 8 * (lane >> 5);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      kf[j] = __builtin_bit_cast(bf16x8a, *reinterpret_cast<const u32x4a*>(a.K + row + 16 * j));
      const u32x4a v = *reinterpret_cast<const u32x4a*>(a.V + row + 16 * j);
      if (j < 8 - NPARK) vf[j] = __builtin_bit_cast(bf16x8a, v);
      else park[(j - 8 + NPARK) * 64 + lane] = v;
    }
  }
  f32x16a dk[4] = {zero16(), zero16(), zero16(), zero16()};
  f32x16a dv[4] = {zero16(), zero16(), zero16(), zero16()};
  const int nt = n_tiles - first;  // tiles the workgroup walks
#pragma unroll
  for (int i = 0; i < S - 1; ++i)
    if (i < nt) {
      const int t = first + i;
      u32x4a* st = smem + (i % S) * STAGE;
      copy_tile<PW>(Qb + int64_t(t) * NB * D, ro, st, wave);
      copy_tile<PW>(dOb + int64_t(t) * NB * ldo, rod, st + TILE16, wave);
      if (wave == 0) copy16(rt_src + t * NB, 0, st + 2 * TILE16);
    }
  for (int i = 0; i < nt; ++i) {
    if (wave == 0) wait_tiles<2 * PW + 1>(min(S - 2, nt - 1 - i));
    else wait_tiles<2 * PW>(min(S - 2, nt - 1 - i));
    lds_wait_barrier();
    if (i + S - 1 < nt) {
      const int u = i + S - 1, t = first + u;
      u32x4a* st = smem + (u % S) * STAGE;
      copy_tile<PW>(Qb + int64_t(t) * NB * D, ro, st, wave);
      copy_tile<PW>(dOb + int64_t(t) * NB * ldo, rod, st + TILE16, wave);
      if (wave == 0) copy16(rt_src + t * NB, 0, st + 2 * TILE16);
    }
    const int t = first + i;
    if (t < my_first) continue;
    const u32x4a* st = smem + (i % S) * STAGE;
    const float* rt = reinterpret_cast<const float*>(st + 2 * TILE16);  // lse[32], delta[32]
    f32x16a s = zero16(), dp = zero16();
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      s = mfma(row_frag(st, j, lane), kf[j], s);
      const bf16x8a vj = j < 8 - NPARK ? vf[j] : __builtin_bit_cast(bf16x8a, park[(j - 8 + NPARK) * 64 + lane]);
      dp = mfma(row_frag(st + TILE16, j, lane), vj, dp);
    }
    // P and dS in place of S and dP
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int q8 = 16 * h + 8 * (lane >> 5);  // the 8 query rows of slots 8 h .. + 8
      const float4 l0 = *reinterpret_cast<const float4*>(rt + q8), l1 = *reinterpret_cast<const float4*>(rt + q8 + 4);
      const float4 e0 = *reinterpret_cast<const float4*>(rt + 32 + q8),
                   e1 = *reinterpret_cast<const float4*>(rt + 32 + q8 + 4);
      const float ls[8] = {l0.x, l0.y, l0.z, l0.w, l1.x, l1.y, l1.z, l1.w};
      const float de[8] = {e0.x, e0.y, e0.z, e0.w, e1.x, e1.y, e1.z, e1.w};
#pragma unroll
      for (int i8 = 0; i8 < 8; ++i8) {
        const int r = 8 * h + i8;
        const float pv = bf16_round(exp2a(fmaf(s[r], c, -ls[i8])));
        s[r] = pv;
        dp[r] = pv * (dp[r] - de[i8]);
      }
    }
    if (t == my_first) {
#pragma unroll
      for (int r = 0; r < 16; ++r)
        if (kj > t * NB + slot_row(r, lane)) {
          s[r] = 0.0f;
          dp[r] = 0.0f;
        }
    }
    // the transpose-read addresses are recomputed for each tile (an opaque
    // copy of the lane index keeps them from being held across the loop)
    int tl = lane;
    asm volatile("" : "+v"(tl));
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      bf16x8a pb, sb;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        pb[i] = __bf16(s[8 * h + i]);
        sb[i] = __bf16(dp[8 * h + i]);
      }
#pragma unroll
      for (int db = 0; db < 4; ++db) {
        dv[db] = mfma(col_frag(st + TILE16, db, h, tl), pb, dv[db]);
        dk[db] = mfma(col_frag(st, db, h, tl), sb, dk[db]);
      }
    }
  }
  if (!active) return;
  if (TOK && a.kv_batch == a.batch) {
    const int64_t o = tok_off(a, b, kj);
    store_bf16_row<true>(a.dK_tok + o, dk, a.scale, a.cs, kj, lane);
    store_bf16_row<false>(a.dV_tok + o, dv, 1.0f, a.cs, kj, lane);
    return;
  }
  store_f32_rows(a.dK + (b * L + kj) * int64_t(D), dk, a.scale, lane);
  store_f32_rows(a.dV + (b * L + kj) * int64_t(D), dv, 1.0f, lane);
}

namespace {
constexpr int FWD_NW = 4, FWD_S = 2;
constexpr int DQ_NW = 4, DQ_S = 2;
constexpr int DKV_NW = 4, DKV_S = 2;
}  // namespace

static void set_tok(AttnArgs& a, const AttnLaunch& q) {
  a.n_seq = q.tok_seqs > 0 ? q.tok_seqs : 1;
  a.heads = int(q.batch / a.n_seq);
  a.grp = q.group > 0 ? q.group : 1;
  a.cs = q.cs;
  a.dQ_tok = q.dQ_tok; a.dK_tok = q.dK_tok; a.dV_tok = q.dV_tok;
}

hipError_t launch_attn_fwd(const AttnLaunch& q, hipStream_t st) {
  AttnArgs a{};
  a.batch = q.batch; a.kv_batch = q.kv_batch; a.L = q.L; a.scale = q.scale;
  a.Q = q.Q; a.K = q.K; a.V = q.V; a.O_out = q.O_out; a.lse = q.lse;
  set_tok(a, q);
  const int64_t nblk = (q.L + FWD_NW * NB - 1) / (FWD_NW * NB);
  const dim3 grid(unsigned(nblk * q.batch));
  if (q.tok_seqs > 0) hipLaunchKernelGGL((attn_fwd_kernel<FWD_NW, FWD_S, true>), grid, dim3(FWD_NW * 64), 0, st, a);
  else hipLaunchKernelGGL((attn_fwd_kernel<FWD_NW, FWD_S, false>), grid, dim3(FWD_NW * 64), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_attn_bwd(const AttnLaunch& q, hipStream_t st) {
  AttnArgs a{};
  a.batch = q.batch; a.kv_batch = q.kv_batch; a.L = q.L; a.scale = q.scale;
  a.Q = q.Q; a.K = q.K; a.V = q.V; a.O = q.O; a.dO = q.dO;
  a.lse = q.lse; a.delta = q.delta; a.dQ = q.dQ; a.dK = q.dK; a.dV = q.dV;
  set_tok(a, q);
  const bool tok = q.tok_seqs > 0;
  const int64_t nq = (q.L + DQ_NW * NB - 1) / (DQ_NW * NB);
  const dim3 gq(unsigned(nq * q.batch));
  if (tok) hipLaunchKernelGGL((attn_bwd_dq_kernel<DQ_NW, DQ_S, true>), gq, dim3(DQ_NW * 64), 0, st, a);
  else hipLaunchKernelGGL((attn_bwd_dq_kernel<DQ_NW, DQ_S, false>), gq, dim3(DQ_NW * 64), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t nk = (q.L + DKV_NW * NB - 1) / (DKV_NW * NB);
  const dim3 gk(unsigned(nk * q.batch));
  if (tok) hipLaunchKernelGGL((attn_bwd_dkv_kernel<DKV_NW, DKV_S, true>), gk, dim3(DKV_NW * 64), 0, st, a);
  else hipLaunchKernelGGL((attn_bwd_dkv_kernel<DKV_NW, DKV_S, false>), gk, dim3(DKV_NW * 64), 0, st, a);
  return hipGetLastError();
}

}  // namespace uq
