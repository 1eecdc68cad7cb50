// Channel-wise members of the recurrence family on gfx950 (paper Sec. 4.1,
// Eq. (gdn) with its gates per channel; table "One recurrence, five models":
// full GDN, KDA, GLA and LA are gate settings of it):
//
//   S_t = (I - k_t (b_t * k_t)^T) Diag(e^{g_t}) S_{t-1} + k_t (w_t * v_t)^T,  o_t = S_t^T q_t
//
// with g_t, b_t in R^{d_k} and w_t in R^{d_v}; a NULL gate is neutral (g = 0,
// b = 0, w = 1).  Activations (q, k, v, dO and their gradients, o) are fp32 or
// bf16 (IO).  The prep and the channel-part gradients compute in fp32 (fp32
// matrix cores); the prep writes the operands of the later kernels in IO, so
// with bf16 activations the two scans (fp32 carry) and the value-part
// gradient products run on bf16 matrix cores, as the scalar-gate path.
//
// Chunked form (Sec. 4.2), per chunk of 64 tokens with G_r = sum_{s<=r} g_s (a
// d_k-vector per row), Gamma = e^G, Kb = b * K, Khat_r = e^{G_last - G_r} * k_r:
//   A_ri = sum_d Kb_rd K_id e^{G_rd - G_id}  (i < r),   T = (I + A)^{-1}
//   P_ri = sum_d Q_rd  K_id e^{G_rd - G_id}  (i <= r)
//   W = T (Gamma * Kb),   U = T (w * V),   U' = U - W h
//   O = (Gamma * Q) h + P U',   h <- Diag(e^{G_last}) h + Khat^T U'
// The carry and the output reuse the generic scans with a per-row decay.
//
// Decay-weighted contractions.  Every product above and in the backward
// that carries e^{G_r - G_i} inside its sum over channels is split by 16-row
// blocks.  Pairs (r, i) in different blocks go to the matrix cores with the
// exponent split at a reference row between them: for output rows in block R
// the row just before the block (the chunk's entry, G = 0, for R = 0), so both
// e^{G_r - G_ref} and e^{G_ref - G_i} are <= 1 for a decay (g <= 0) and nothing
// can overflow; the operand is zeroed (before the exponential) outside those
// blocks.  Contractions down the columns (the transposed gradients) use the
// last row of the block instead.  Pairs inside one block are summed exactly
// on the vector ALUs with e^{G_r - G_i} formed per term -- only for blocks whose log-decay moves by more than
// CW_SPREAD from the reference; the others take the block's reference on the
// matrix cores too (factors within e^{+-2 CW_SPREAD}: no overflow, no
// denormals, the same per-term rounding).
#pragma once

#include <type_traits>

#include "gdn_bwd.hpp"
#include "gdn_cw_exact.hpp"
#include "gdn_fwd.hpp"

namespace gdn {

// G (cumulative log-decay per channel) in place down each column of a 64 x D
// LDS tile with row stride LD: one wave per column, rows on lanes.  With
// wide, also sets bit R of *wide when some |G_r - G_ref| in 16-row block R
// (G_ref that of the row before the block, 0 for R = 0) exceeds CW_SPREAD or
// is not finite: such a block's in-block pairs are summed exactly.
constexpr float CW_SPREAD = 32.f;
template <int D, int LD>
__device__ __forceinline__ void cw_cumsum_columns(float* Gs, int* wide = nullptr) {
  const int nw = (int)blockDim.x / WAVE, l = lane_id(), src = l >= 16 ? (l & ~15) - 1 : 0;
  bool big = false;
  for (int d = wave_id(); d < D; d += nw) {
    const float x = wave_incl_scan(Gs[l * LD + d]);
    Gs[l * LD + d] = x;
    const float rf = shfl_idx(x, src);
    big |= !(fabsf(x - (l >= 16 ? rf : 0.f)) <= CW_SPREAD);
  }
  if (wide) {
    const unsigned long long m = __ballot(big);
    int f = 0;
#pragma unroll
    for (int R = 0; R < 4; ++R) f |= ((m >> (16 * R)) & 0xFFFFull) ? 1 << R : 0;
    if (l == 0 && f) atomicOr(wide, f);  // integer OR: order-free
  }
}

// A ROWS x D fp32 tile (rows rs floats apart in HBM), read by NT threads in
// one batch: every load is in flight before the first LDS store (a load /
// store loop would pay one memory round trip per iteration).
template <int ROWS, int D, int NT>
struct TileIn {
  static constexpr int PER_ROW = D / 4, N = ROWS * PER_ROW / NT;
  static_assert(ROWS * PER_ROW % NT == 0, "whole pieces per thread");
  float4 u[N];
  __device__ __forceinline__ void load(const float* __restrict__ src, long rs) {
#pragma unroll
    for (int t = 0; t < N; ++t) {
      const int idx = thread_x() + t * NT, r = idx / PER_ROW, c = (idx - r * PER_ROW) * 4;
      u[t] = *reinterpret_cast<const float4*>(src + r * rs + c);
    }
  }
  template <int LD>
  __device__ __forceinline__ void stage(float* dst) const {
#pragma unroll
    for (int t = 0; t < N; ++t) {
      const int idx = thread_x() + t * NT, r = idx / PER_ROW, c = (idx - r * PER_ROW) * 4;
      *reinterpret_cast<float4*>(dst + r * LD + c) = u[t];
    }
  }
  // rounded to bf16: one 8-byte store per piece
  template <int LD>
  __device__ __forceinline__ void stage16(bf16* dst) const {
#pragma unroll
    for (int t = 0; t < N; ++t) {
      const int idx = thread_x() + t * NT, r = idx / PER_ROW, c = (idx - r * PER_ROW) * 4;
      const bf16 x[4] = {from_f<bf16>(u[t].x), from_f<bf16>(u[t].y), from_f<bf16>(u[t].z), from_f<bf16>(u[t].w)};
      *reinterpret_cast<uint2*>(dst + r * LD + c) = pack4<bf16>(x);
    }
  }
};

// Rows [0, len) of a 64 x D tile of T (fp32 or bf16; rows rs elements apart
// in HBM), read in one batch like TileIn and staged to LDS as fp32 (rows past
// len are zero).  Pieces are 16 bytes; when they do not divide evenly over the
// NT threads the spare threads load a valid piece and stage nothing.
template <int D, int NT, typename T>
struct CwRows {
  static constexpr int V = 16 / (int)sizeof(T), PER_ROW = D / V, TOT = CH * PER_ROW;
  static constexpr int N = (TOT + NT - 1) / NT;
  uint4 u[N];
  __device__ __forceinline__ static void where(int t, int& idx, int& r, int& c) {
    idx = thread_x() + t * NT;
    const int i = idx < TOT ? idx : TOT - 1;
    r = i / PER_ROW;
    c = (i - r * PER_ROW) * V;
  }
  __device__ __forceinline__ void load(const T* __restrict__ src, long rs, int len) {
#pragma unroll
    for (int t = 0; t < N; ++t) {
      int idx, r, c;
      where(t, idx, r, c);
      u[t] = *reinterpret_cast<const uint4*>(src + clamp_row(r, len) * rs + c);
    }
  }
  // columns [lo, hi) of the tile (piece-aligned) to dst[r * LD + c - lo]
  template <int LD>
  __device__ __forceinline__ void stage(float* dst, int len, int lo = 0, int hi = D) const {
#pragma unroll
    for (int t = 0; t < N; ++t) {
      int idx, r, c;
      where(t, idx, r, c);
      if (idx >= TOT || c < lo || c >= hi) continue;
      const uint4 x = keep16(r < len, u[t]);
      float* d = dst + r * LD + (c - lo);
      if constexpr (sizeof(T) == 4) {
        *reinterpret_cast<uint4*>(d) = x;
      } else {
        float f[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) f[j] = to_f(elem16<bf16>(x, j));
        *reinterpret_cast<float4*>(d) = float4{f[0], f[1], f[2], f[3]};
        *reinterpret_cast<float4*>(d + 4) = float4{f[4], f[5], f[6], f[7]};
      }
    }
  }
  // whether every loaded element of rows [0, len) is finite
  __device__ __forceinline__ bool finite(int len) const {
    bool ok = true;
#pragma unroll
    for (int t = 0; t < N; ++t) {
      int idx, r, c;
      where(t, idx, r, c);
      if (idx < TOT && r < len) ok &= finite16B<T>(u[t]);
    }
    return ok;
  }
  // the same, kept in 16-bit (T = bf16 only): one 16-byte store per piece
  template <int LD>
  __device__ __forceinline__ void stage16(bf16* dst, int len) const {
    static_assert(sizeof(T) == 2, "bf16 pieces");
#pragma unroll
    for (int t = 0; t < N; ++t) {
      int idx, r, c;
      where(t, idx, r, c);
      if (idx >= TOT) continue;
      *reinterpret_cast<uint4*>(dst + r * LD + c) = keep16(r < len, u[t]);
    }
  }
  // transposed: element (r, c) to dst[c * LD + r] (rows past len zero)
  template <int LD>
  __device__ __forceinline__ void stageT(float* dst, int len) const {
#pragma unroll
    for (int t = 0; t < N; ++t) {
      int idx, r, c;
      where(t, idx, r, c);
      if (idx >= TOT) continue;
      const uint4 x = keep16(r < len, u[t]);
#pragma unroll
      for (int j = 0; j < V; ++j) dst[(c + j) * LD + r] = to_f(elem16<T>(x, j));
    }
  }
  // multiply a tile staged by stageT by this one's values (fp32 pieces)
  template <int LD>
  __device__ __forceinline__ void scaleT(float* dst, int len) const {
    static_assert(sizeof(T) == 4, "fp32 factors");
#pragma unroll
    for (int t = 0; t < N; ++t) {
      int idx, r, c;
      where(t, idx, r, c);
      if (idx >= TOT) continue;
      const uint4 x = keep16(r < len, u[t]);
#pragma unroll
      for (int j = 0; j < V; ++j) dst[(c + j) * LD + r] *= elem16<float>(x, j);
    }
  }
  // multiply the staged tile by this one's values (same layout, fp32 pieces)
  template <int LD>
  __device__ __forceinline__ void scale(float* dst, int len) const {
    static_assert(sizeof(T) == 4, "fp32 factors");
#pragma unroll
    for (int t = 0; t < N; ++t) {
      int idx, r, c;
      where(t, idx, r, c);
      if (idx >= TOT) continue;
      const float4 y = __builtin_bit_cast(float4, keep16(r < len, u[t]));
      float4* d = reinterpret_cast<float4*>(dst + r * LD + c);
      float4 x = *d;
      x.x *= y.x; x.y *= y.y; x.z *= y.z; x.w *= y.w;
      *d = x;
    }
  }
};

// Element (o, k) of a fp32 LDS array of rows of 64, its 16-byte groups
// XOR-swizzled by o & 15: a wave's float4 reads of 16 rows at one k hit 16
// different bank groups, with no padding.
struct KRowSw64 {
  const float* p;
  static constexpr bool kVec = true;
  __device__ __forceinline__ static int off(int o, int k) {
    return o * 64 + ((((k >> 2) ^ (o & 15)) << 2) | (k & 3));
  }
  __device__ __forceinline__ float get(int o, int k) const { return p[off(o, k)]; }
  __device__ __forceinline__ const float* ptr(int o, int k) const { return p + off(o, k); }
};

// Scan operands (P, diag-scaled Q, Khat, W, dO^T) in the activation dtype,
// laid out by op_off: row-major for fp32, MFMA fragment blocks for bf16.
// Piece idx (8 consecutive k of one row m) of a M x K operand: consecutive
// pieces are consecutive 16-byte runs of the bf16 layout (whole 1 KiB
// fragment blocks per wave) and consecutive runs of a row for fp32.
template <typename OP, int K>
__device__ __forceinline__ void op_piece(int idx, int& m, int& k0) {
  if constexpr (sizeof(OP) == 2) {
    const int f = idx >> 6, ll = idx & 63;
    m = (f / (K / 32)) * 16 + (ll & 15);
    k0 = (f % (K / 32)) * 32 + (ll >> 4) * 8;
  } else {
    m = idx / (K / 8);
    k0 = (idx - m * (K / 8)) * 8;
  }
}
template <typename OP, int K>
__device__ __forceinline__ void put_op8(OP* base, int m, int k0, const float* x) {
  OP* p = base + op_off<OP, K>(m, k0);
  if constexpr (sizeof(OP) == 2) {
    OP v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = from_f<OP>(x[j]);
    *reinterpret_cast<uint4*>(p) = pack16<OP>(v);
  } else {
    *reinterpret_cast<float4*>(p) = float4{x[0], x[1], x[2], x[3]};
    *reinterpret_cast<float4*>(p + 4) = float4{x[4], x[5], x[6], x[7]};
  }
}
// four consecutive k (k0 % 4 == 0) of row m
template <typename OP, int K>
__device__ __forceinline__ void put_op4(OP* base, int m, int k0, const float* x) {
  OP v[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) v[j] = from_f<OP>(x[j]);
  *reinterpret_cast<typename vec4_of<OP>::type*>(base + op_off<OP, K>(m, k0)) = pack4<OP>(v);
}

// Rows [m0, m0 + MR) x columns [k0, k0 + KC) of a bf16 operand laid out by
// op_off<bf16, K> (m0 % 16 == 0, k0 % 32 == 0, KC % 32 == 0), read by NT
// threads in one batch (whole 1 KiB fragment blocks) and staged to LDS as fp32
// [m - m0][k - k0].
template <int MR, int KC, int K, int NT>
struct OpIn16 {
  static constexpr int PIECES = MR * KC / 8, N = (PIECES + NT - 1) / NT;
  static_assert(MR % 16 == 0 && KC % 32 == 0, "whole fragment blocks");
  uint4 u[N];
  __device__ __forceinline__ static void where(int t, int& idx, int& m, int& k) {
    idx = thread_x() + t * NT;
    const int i = idx < PIECES ? idx : PIECES - 1, f = i >> 6, ll = i & 63;
    m = (f / (KC / 32)) * 16 + (ll & 15);
    k = (f % (KC / 32)) * 32 + (ll >> 4) * 8;
  }
  __device__ __forceinline__ void load(const bf16* __restrict__ base, int m0, int k0) {
#pragma unroll
    for (int t = 0; t < N; ++t) {
      int idx, m, k;
      where(t, idx, m, k);
      u[t] = *reinterpret_cast<const uint4*>(base + op_off<bf16, K>(m0 + m, k0 + k));
    }
  }
  template <int LD>
  __device__ __forceinline__ void stage(float* dst) const {
#pragma unroll
    for (int t = 0; t < N; ++t) {
      int idx, m, k;
      where(t, idx, m, k);
      if (idx >= PIECES) continue;
      float f[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) f[j] = to_f(elem16<bf16>(u[t], j));
      *reinterpret_cast<float4*>(dst + m * LD + k) = float4{f[0], f[1], f[2], f[3]};
      *reinterpret_cast<float4*>(dst + m * LD + k + 4) = float4{f[4], f[5], f[6], f[7]};
    }
  }
  // kept in bf16: one 16-byte store per piece
  template <int LD>
  __device__ __forceinline__ void stage16(bf16* dst) const {
#pragma unroll
    for (int t = 0; t < N; ++t) {
      int idx, m, k;
      where(t, idx, m, k);
      if (idx >= PIECES) continue;
      *reinterpret_cast<uint4*>(dst + m * LD + k) = u[t];
    }
  }
};

// One block per (chunk, head).  Forward mode writes the operands of the
// generic forward scan (P, diag-scaled Q, Khat^T, W, U); backward mode writes
// those of the reverse scan and the gradient kernels (P^T, (Gamma Q)^T,
// Khat, W^T, T, Gamma * Kb, dO^T).  Both write G_last per channel.  Every
// operand is written in the activation dtype IO: the scans' in the op_off
// layout, T and Gamma * Kb (read by the gradient kernel) row-major.
constexpr int CW_PREP_THREADS = 1024;  // 16 waves: one block per CU (LDS), so all its latency hiding is in-block
template <int DK, int DV, bool BWD, typename IO>
__global__ __launch_bounds__(CW_PREP_THREADS) void k_cw_prep(Geo geo, int H, const IO* __restrict__ q,
                                                 const IO* __restrict__ k, const IO* __restrict__ v,
                                                 const float* __restrict__ g, const float* __restrict__ b,
                                                 const float* __restrict__ w, const IO* __restrict__ dO,
                                                 float* __restrict__ gC, IO* __restrict__ Pg,
                                                 IO* __restrict__ Qgg, IO* __restrict__ Khg,
                                                 IO* __restrict__ Wg, IO* __restrict__ Ug,
                                                 IO* __restrict__ Tg, IO* __restrict__ KbGg,
                                                 IO* __restrict__ dOTg, int* __restrict__ flag) {
  constexpr int LK = DK + 4, LC = CH + 4, VS = 64;
  static_assert(CH * LC <= CH * LK && VS * LC <= CH * LK, "T and the (w * V)^T slices reuse Q's and K's tiles");
  __shared__ __align__(16) float Qs[CH * LK];  // Q, then T (stride LC)
  __shared__ __align__(16) float Ks[CH * LK];  // K, then slices of (w * V)^T [v][i] (stride LC)
  __shared__ __align__(16) float Gs[CH * LK];  // G, then (Gamma * Kb)^T (swizzled rows of 64)
  __shared__ __align__(16) float Bk[CH * LK];  // b * K
  __shared__ __align__(16) float As[CH * LC];  // A
  __shared__ __align__(16) float Pd[4 * 16 * 16];  // P inside the four diagonal 16 x 16 blocks (wide blocks)
  __shared__ int wide;                              // blocks summed exactly (bit R: block R)
  float* Tf = Qs;
  float* Vw = Ks;

  const int ci = blockIdx.x, h = blockIdx.y;
  const ChunkPos cp = chunk_pos(geo, ci);
  const long tile = (long)ci * H + h;
  const long rsk = (long)H * DK, bk = (cp.row0 * H + h) * DK;
  const long rsv = (long)H * DV, bv = (cp.row0 * H + h) * DV;
  // every input row of the block is requested up front: q, k, g, b, then the
  // forward's v and w slices (or the backward's dO)
  constexpr int NSL = BWD ? 1 : DV / VS;
  constexpr int NT = CW_PREP_THREADS, WN = NT / 256;  // wave columns of the 64-row products
  static_assert(NT / WAVE == 16, "sixteen 16 x 16 tiles of P and A, one per wave");
  CwRows<DK, NT, IO> qin, kin;
  CwRows<DK, NT, float> gin, bin;
  CwRows<VS, NT, IO> vin[NSL];
  CwRows<VS, NT, float> win[NSL];
  CwRows<DV, NT, IO> doin;
  qin.load(q + bk, rsk, cp.len);
  kin.load(k + bk, rsk, cp.len);
  if (g) gin.load(g + bk, rsk, cp.len);
  if (b) bin.load(b + bk, rsk, cp.len);
  if constexpr (!BWD) {
#pragma unroll
    for (int t = 0; t < NSL; ++t) {
      vin[t].load(v + bv + t * VS, rsv, cp.len);
      if (w) win[t].load(w + bv + t * VS, rsv, cp.len);
    }
  } else {
    doin.load(dO + bv, rsv, cp.len);
  }
  if (thread_x() == 0) wide = 0;
  // non-finite inputs send the stream to the exact token-serial pass
  bool ok = qin.finite(cp.len) && kin.finite(cp.len);
  if (g) ok &= gin.finite(cp.len);
  if (b) ok &= bin.finite(cp.len);
  if constexpr (BWD) ok &= doin.finite(cp.len);
  qin.template stage<LK>(Qs, cp.len);
  kin.template stage<LK>(Ks, cp.len);
  if (g) gin.template stage<LK>(Gs, cp.len);
  else
    for (int i = thread_x(); i < CH * LK; i += blockDim.x) Gs[i] = 0.f;
  if (b) bin.template stage<LK>(Bk, cp.len);
  __syncthreads();  // (stage writes fp32 tiles: the LDS layout below is the same for both I/O types)
  if (g) cw_cumsum_columns<DK, LK>(Gs, &wide);
  if (b)
    for (int i = thread_x(); i < CH * DK; i += blockDim.x) {
      const int r = i / DK, d = i - r * DK;
      Bk[r * LK + d] *= Ks[r * LK + d];
    }
  __syncthreads();

  // Pairs inside a wide 16-row block, exactly, spread over the whole block:
  // pair q of block RB is (rl, il) with il <= rl; one exponential per term
  // serves P and A.  A's sums land in As at their own positions, P's in Pd.
  const int wideb = wide;
  if (wideb) {
    for (int pi = thread_x(); pi < 4 * 136; pi += blockDim.x) {
      const int RB = pi / 136, q = pi - RB * 136;
      if (!((wideb >> RB) & 1)) continue;
      int rl = (int)((sqrtf(8.f * q + 1.f) - 1.f) * 0.5f);
      while ((rl + 1) * (rl + 2) / 2 <= q) ++rl;
      while (rl * (rl + 1) / 2 > q) --rl;
      const int il = q - rl * (rl + 1) / 2, r = 16 * RB + rl, i = 16 * RB + il;
      float sp = 0.f, sa = 0.f;
#pragma unroll 4
      for (int d = 0; d < DK; d += 4) {
        const float4 qr = *reinterpret_cast<const float4*>(Qs + r * LK + d);
        const float4 ki = *reinterpret_cast<const float4*>(Ks + i * LK + d);
        const float4 gr = *reinterpret_cast<const float4*>(Gs + r * LK + d);
        const float4 gi = *reinterpret_cast<const float4*>(Gs + i * LK + d);
        const float e0 = __expf(gr.x - gi.x), e1 = __expf(gr.y - gi.y), e2 = __expf(gr.z - gi.z), e3 = __expf(gr.w - gi.w);
        const float k0 = ki.x * e0, k1 = ki.y * e1, k2 = ki.z * e2, k3 = ki.w * e3;
        sp += qr.x * k0 + qr.y * k1 + qr.z * k2 + qr.w * k3;
        if (b) {
          const float4 br = *reinterpret_cast<const float4*>(Bk + r * LK + d);
          sa += br.x * k0 + br.y * k1 + br.z * k2 + br.w * k3;
        }
      }
      Pd[(RB * 16 + rl) * 16 + il] = sp;
      if (b && il < rl) As[r * LC + i] = sa;
    }
    __syncthreads();
  }

  // P and A by 16 x 16 tiles (R, c) of output rows 16R.. and columns 16c..:
  // waves 0..9 take the ten tiles c <= R (both products share the scaled K
  // fragment), waves 10..15 write the six zero tiles c > R.  Lane l holds
  // rows 16R + 4 (l >> 4) + j, column 16c + (l & 15).
  {
    const int wv = wave_id(), l = lane_id();
    IO* Pt = Pg + tile * CH * CH;
    int R, c;
    if (wv < 10) {
      R = wv < 1 ? 0 : wv < 3 ? 1 : wv < 6 ? 2 : 3;
      c = wv - R * (R + 1) / 2;
    } else {  // (0,1) (0,2) (0,3) (1,2) (1,3) (2,3)
      const int u = wv - 10;
      R = u < 3 ? 0 : u < 5 ? 1 : 2;
      c = u - (R == 0 ? 0 : R == 1 ? 3 : 5) + R + 1;
    }
    const bool lower = c <= R, exact = c == R && ((wideb >> R) & 1);
    f32x4 ap = {0.f, 0.f, 0.f, 0.f}, aa = {0.f, 0.f, 0.f, 0.f};
    if (lower && !exact) {
      const int r = 16 * R + (l & 15), i = 16 * c + (l & 15);
      const float* Gref = Gs + (R > 0 ? 16 * R - 1 : 0) * LK;
#pragma unroll 2
      for (int k16 = 0; k16 < DK; k16 += 16) {
        const int d = k16 + 4 * (l >> 4);
        const float4 rf = R > 0 ? *reinterpret_cast<const float4*>(Gref + d) : float4{0.f, 0.f, 0.f, 0.f};
        const float4 gr = *reinterpret_cast<const float4*>(Gs + r * LK + d);
        const float4 gi = *reinterpret_cast<const float4*>(Gs + i * LK + d);
        const float4 qr = *reinterpret_cast<const float4*>(Qs + r * LK + d);
        const float4 ki = *reinterpret_cast<const float4*>(Ks + i * LK + d);
        const float er[4] = {__expf(gr.x - rf.x), __expf(gr.y - rf.y), __expf(gr.z - rf.z), __expf(gr.w - rf.w)};
        const float kk[4] = {ki.x * __expf(rf.x - gi.x), ki.y * __expf(rf.y - gi.y), ki.z * __expf(rf.z - gi.z),
                             ki.w * __expf(rf.w - gi.w)};
        const float qq[4] = {qr.x * er[0], qr.y * er[1], qr.z * er[2], qr.w * er[3]};
#pragma unroll
        for (int t = 0; t < 4; ++t) ap = Mma<float>::mma(qq[t], kk[t], ap);
        if (b) {
          const float4 br = *reinterpret_cast<const float4*>(Bk + r * LK + d);
          const float bb[4] = {br.x * er[0], br.y * er[1], br.z * er[2], br.w * er[3]};
#pragma unroll
          for (int t = 0; t < 4; ++t) aa = Mma<float>::mma(bb[t], kk[t], aa);
        }
      }
    }
    const int i = 16 * c + (l & 15), r0 = 16 * R + 4 * (l >> 4);
    float pv[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = r0 + j;
      const float x = exact ? Pd[(R * 16 + (r & 15)) * 16 + (i & 15)] : ap[j];
      pv[j] = lower && i <= r ? x : 0.f;
      if (b) {
        const float y = exact ? As[r * LC + i] : aa[j];
        As[r * LC + i] = lower && i < r ? y : 0.f;
      }
    }
    if (BWD) {
      put_op4<IO, CH>(Pt, i, r0, pv);
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) Pt[op_off<IO, CH>(r0 + j, i)] = from_f<IO>(pv[j]);
    }
  }
  // Gamma * Q and Khat = e^{G_last - G} * K, each in the layout its scan reads
  {
    IO* Qt = Qgg + tile * CH * DK;
    IO* Kt = Khg + tile * CH * DK;
    // pieces of 8: rows r of the [r][d] output (forward Gamma * Q, backward
    // Khat), columns r of the [d][r] one (forward Khat^T, backward (Gamma Q)^T)
    for (int i = thread_x(); i < CH * DK / 8; i += blockDim.x) {
      int r, d0;
      op_piece<IO, DK>(i, r, d0);
      float x[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float G = Gs[r * LK + d0 + j];
        x[j] = BWD ? __expf(Gs[(CH - 1) * LK + d0 + j] - G) * Ks[r * LK + d0 + j] : __expf(G) * Qs[r * LK + d0 + j];
      }
      put_op8<IO, DK>(BWD ? Kt : Qt, r, d0, x);
      int d, r0;
      op_piece<IO, CH>(i, d, r0);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float G = Gs[(r0 + j) * LK + d];
        x[j] = BWD ? __expf(G) * Qs[(r0 + j) * LK + d] : __expf(Gs[(CH - 1) * LK + d] - G) * Ks[(r0 + j) * LK + d];
      }
      put_op8<IO, CH>(BWD ? Qt : Kt, d, r0, x);
    }
    for (int d = thread_x(); d < DK; d += blockDim.x) gC[tile * DK + d] = Gs[(CH - 1) * LK + d];
  }
  __syncthreads();  // Q is dead: T takes its tile
  if (b) {
    unit_lower_inverse<float, LC, LC, false>(As, Tf, (float*)nullptr, (float*)nullptr);
  } else {
    for (int i = thread_x(); i < CH * CH; i += blockDim.x) {
      const int r = i / CH, c = i - r * CH;
      Tf[r * LC + c] = r == c ? 1.f : 0.f;
    }
    __syncthreads();
  }
  // Gamma * Kb (A has been formed from b * K above), held in registers and
  // then written transposed, [d][i] swizzled, over G's tile (G is dead)
  constexpr int NG = CH * DK / NT;
  static_assert(CH * DK % NT == 0 && DK * 64 <= CH * LK, "whole pieces; Gamma * Kb^T fits G's tile");
  float gk[NG];
#pragma unroll
  for (int j = 0; j < NG; ++j) {
    const int i = thread_x() + j * NT, r = i / DK, d = i - r * DK;
    gk[j] = b ? Bk[r * LK + d] * __expf(Gs[r * LK + d]) : 0.f;
  }
  if (BWD) {
    IO* Tt = Tg + tile * CH * CH;
    for (int i = thread_x(); i < CH * CH; i += blockDim.x) Tt[i] = from_f<IO>(Tf[(i / CH) * LC + (i % CH)]);
    IO* Kb = KbGg + tile * CH * DK;
#pragma unroll
    for (int j = 0; j < NG; ++j) Kb[thread_x() + j * NT] = from_f<IO>(gk[j]);
  }
  __syncthreads();  // every read of G is done
  float* GkT = Gs;
  if (b)
#pragma unroll
    for (int j = 0; j < NG; ++j) {
      const int i = thread_x() + j * NT, r = i / DK, d = i - r * DK;
      GkT[KRowSw64::off(d, r)] = gk[j];
    }
  __syncthreads();
  // W = T (Gamma * Kb)
  {
    IO* Wt = Wg + tile * CH * DK;
    if (b) {
      Tiles<CH, DK, 4, WN> wt;
      wt.zero();
      wt.template mma<float, CH>(KRow<float, LC>{Tf}, KRowSw64{GkT});
      const int l = lane_id();
#pragma unroll
      for (int a = 0; a < wt.TM; ++a)
#pragma unroll
        for (int bb = 0; bb < wt.TN; ++bb) {
          const int r0 = wt.m0(a) + (l >> 4) * 4, d = wt.n0(bb) + (l & 15);
          const float x4[4] = {wt.acc[a][bb][0], wt.acc[a][bb][1], wt.acc[a][bb][2], wt.acc[a][bb][3]};
          if (BWD) {
            put_op4<IO, CH>(Wt, d, r0, x4);
          } else {
#pragma unroll
            for (int j = 0; j < 4; ++j) Wt[op_off<IO, DK>(r0 + j, d)] = from_f<IO>(x4[j]);
          }
        }
    } else {
      for (int i = thread_x(); i < CH * DK; i += blockDim.x) Wt[i] = from_f<IO>(0.f);
    }
  }
  // dO^T [v][r]: 64 columns of dO at a time staged row-major in K's tile (free
  // once W is formed), then written down its columns so each store instruction
  // covers whole rows of dO^T
  if constexpr (BWD) {
    constexpr int PW = 64;
    static_assert(PW <= LK && DV % PW == 0, "a pass fits K's tile");
    IO* Dt = dOTg + tile * DV * CH;
#pragma unroll
    for (int ps = 0; ps < DV / PW; ++ps) {
      __syncthreads();
      doin.template stage<LK>(Ks, cp.len, ps * PW, (ps + 1) * PW);
      __syncthreads();
      // the pass's rows v of dO^T are one contiguous range of pieces
      for (int i = thread_x(); i < PW * CH / 8; i += blockDim.x) {
        int vr, r0;
        op_piece<IO, CH>(ps * PW * CH / 8 + i, vr, r0);
        float x[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) x[j] = Ks[(r0 + j) * LK + vr - ps * PW];
        put_op8<IO, CH>(Dt, vr, r0, x);
      }
    }
  }
  // U = T (w * V) in the forward scan's accumulator-tile layout
  if constexpr (!BWD) {
    IO* Ut = Ug + tile * CH * DV;
#pragma unroll
    for (int t = 0; t < NSL; ++t) {
      const int c0 = t * VS;
      __syncthreads();  // K (first pass) or the previous slice is no longer read
      ok &= vin[t].finite(cp.len);
      if (w) ok &= win[t].finite(cp.len);
      vin[t].template stageT<LC>(Vw, cp.len);
      if (w) {
        __syncthreads();
        win[t].template scaleT<LC>(Vw, cp.len);
      }
      __syncthreads();
      Tiles<CH, VS, 4, WN> uu;
      uu.zero();
      uu.template mma<float, CH>(KRow<float, LC>{Tf}, KRow<float, LC>{Vw});
      const int l = lane_id();
#pragma unroll
      for (int bb = 0; bb < uu.TN; ++bb) {
        const int r0 = uu.m0(0) + (l >> 4) * 4, vcol = c0 + uu.n0(bb) + (l & 15);
        IO u4[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) u4[j] = from_f<IO>(uu.acc[0][bb][j]);
        *reinterpret_cast<typename vec4_of<IO>::type*>(Ut + cfrag_off<SCAN_BV>(r0, vcol)) = pack4<IO>(u4);
      }
    }
  }
  const int bad = __syncthreads_or(!ok);
  if (thread_x() == 0) flag[tile] = bad;
}

// Gradient kernel, value part (fp32 activations; k_cw_grad_v_bf below is the
// bf16 one): one block per (chunk, head), value slices of 32 columns.  With h the chunk's entry state, dh the state gradient after it and
// dU' from the reverse scan:
//   R = w * V - (Gamma * Kb) h,  U' = T R,  Y = T^T dU'  ->  dv = w * Y, dw = v * Y
// and, summed over the slices,
//   dP = dO U'^T (i <= r),  dA = -Y U'^T (i < r: the solve's VJP in its short
//   form, -T^T (dU' R^T) T^T = -Y U'^T),  X = -Y h^T,  dQg = dO h^T,
//   dKhat = U' dh^T,  <h, dh> per row d.
template <int DK, int DV>
__global__ __launch_bounds__(512) void k_cw_grad_v(Geo geo, int H, const float* __restrict__ v,
                                                   const float* __restrict__ w, const float* __restrict__ dO,
                                                   const float* __restrict__ states, const float* __restrict__ Tg,
                                                   const float* __restrict__ KbGg, const float* __restrict__ dhg,
                                                   const float* __restrict__ dUTg, float* __restrict__ dvo,
                                                   float* __restrict__ dwo, float* __restrict__ dPg,
                                                   float* __restrict__ dAg, float* __restrict__ Xg,
                                                   float* __restrict__ dQgg, float* __restrict__ dKhg,
                                                   float* __restrict__ hdhg, int* __restrict__ flag) {
  constexpr int LK = DK + 4, LC = CH + 4, VS = 32, LV = VS + 4;
  __shared__ __align__(16) float Ts[CH * LC];
  __shared__ __align__(16) float KbG[CH * LK];
  __shared__ __align__(16) float Vs[CH * LV], Ws[CH * LV], dOs[CH * LV], Ups[CH * LV], Ys[CH * LV];
  __shared__ __align__(16) float dUT[VS * LC], RT[VS * LC];  // dU'^T and R^T: [v][r]
  __shared__ __align__(16) float hs[DK * LV], dhs[DK * LV];

  const int ci = blockIdx.x, h = blockIdx.y;
  const ChunkPos cp = chunk_pos(geo, ci);
  const long tile = (long)ci * H + h;
  const long rsv = (long)H * DV, bv = (cp.row0 * H + h) * DV;
  // the tiles of one value slice, requested in one batch
  struct Slice {
    CwRows<VS, 512, float> v, dO, w;
    TileIn<DK, VS, 512> h, dh;
    TileIn<VS, CH, 512> dut;
  };
  const float* hp = states + tile * DK * DV;
  const float* dhp = dhg + tile * DK * DV;
  const float* dUp = dUTg + tile * DV * CH;
  auto load_slice = [&](Slice& sl, int c0) {
    sl.v.load(v + bv + c0, rsv, cp.len);
    if (w) sl.w.load(w + bv + c0, rsv, cp.len);
    sl.dO.load(dO + bv + c0, rsv, cp.len);
    sl.h.load(hp + c0, DV);
    sl.dh.load(dhp + c0, DV);
    sl.dut.load(dUp + (long)c0 * CH, CH);
  };
  Slice cur, nxt;
  {
    // T, Gamma * Kb and the first value slice in flight together
    TileIn<CH, CH, 512> tin;
    TileIn<CH, DK, 512> kin;
    tin.load(Tg + tile * CH * CH, CH);
    kin.load(KbGg + tile * CH * DK, DK);
    load_slice(cur, 0);
    tin.template stage<LC>(Ts);
    kin.template stage<LK>(KbG);
  }
  __syncthreads();
  // T^T fragments of this wave's rows, for Y = T^T dU' in every slice
  typedef Tiles<CH, VS, 4, 2> TV;
  typename TV::template AFr<float, CH> tT;
  tT.load(KCol<float, LC>{Ts});
  Tiles<CH, CH, 4, 2> dP, dA;
  Tiles<CH, DK, 4, 2> X, dQg, dKh;
  dP.zero(); dA.zero(); X.zero(); dQg.zero(); dKh.zero();
  float hdh = 0.f;  // thread d < DK: sum over v of h[d][v] dh[d][v]
  bool ok = true;   // v and w finite (the chunk state through <h, dh>)
#pragma unroll
  for (int c0 = 0; c0 < DV; c0 += VS) {
    ok &= cur.v.finite(cp.len);
    if (w) ok &= cur.w.finite(cp.len);
    cur.v.template stage<LV>(Vs, cp.len);
    if (w) cur.w.template stage<LV>(Ws, cp.len);
    cur.dO.template stage<LV>(dOs, cp.len);
    cur.h.template stage<LV>(hs);
    cur.dh.template stage<LV>(dhs);
    cur.dut.template stage<LC>(dUT);
    // the next slice's tiles load under this slice's products (the last slice
    // re-reads itself, so the count of loads in flight never changes)
    load_slice(nxt, c0 + VS < DV ? c0 + VS : c0);
    __syncthreads();
    if (thread_x() < DK) {
      const int d = thread_x();
#pragma unroll 8
      for (int c = 0; c < VS; ++c) hdh += hs[d * LV + c] * dhs[d * LV + c];
    }
    {
      TV rr;
      rr.zero();
      rr.template mma<float, DK>(KRow<float, LK>{KbG}, KCol<float, LV>{hs});
      rr.each([&](int r, int vv, float& x) {
        const float wv = w ? Ws[r * LV + vv] : 1.f;
        RT[vv * LC + r] = wv * Vs[r * LV + vv] - x;
      });
    }
    {
      TV y;
      y.zero();
      y.template mma<float, CH>(tT, KRow<float, LC>{dUT});
      y.each([&](int r, int vv, float& x) {
        Ys[r * LV + vv] = x;
        if (r < cp.len) {
          const long o = bv + (long)r * rsv + c0 + vv;
          dvo[o] = (w ? Ws[r * LV + vv] : 1.f) * x;
          if (w) dwo[o] = Vs[r * LV + vv] * x;
        }
      });
    }
    __syncthreads();
    {
      TV up;
      up.zero();
      up.template mma<float, CH>(KRow<float, LC>{Ts}, KRow<float, LC>{RT});
      up.each([&](int r, int vv, float& x) { Ups[r * LV + vv] = x; });
    }
    __syncthreads();
    dP.template mma<float, VS>(KRow<float, LV>{dOs}, KRow<float, LV>{Ups});
    dA.template mma<float, VS>(KRow<float, LV>{Ys}, KRow<float, LV>{Ups});
    X.template mma<float, VS>(KRow<float, LV>{Ys}, KRow<float, LV>{hs});
    dQg.template mma<float, VS>(KRow<float, LV>{dOs}, KRow<float, LV>{hs});
    dKh.template mma<float, VS>(KRow<float, LV>{Ups}, KRow<float, LV>{dhs});
    __syncthreads();
    cur = nxt;
  }
  float* dPt = dPg + tile * CH * CH;
  float* dAt = dAg + tile * CH * CH;
  dP.each([&](int r, int i, float& x) { dPt[r * CH + i] = i <= r ? x : 0.f; });
  dA.each([&](int r, int i, float& x) { dAt[r * CH + i] = i < r ? -x : 0.f; });
  float* Xt = Xg + tile * CH * DK;
  float* Qt = dQgg + tile * CH * DK;
  float* Kt = dKhg + tile * CH * DK;
  X.each([&](int r, int d, float& x) { Xt[r * DK + d] = -x; });
  dQg.each([&](int r, int d, float& x) { Qt[r * DK + d] = x; });
  dKh.each([&](int r, int d, float& x) { Kt[r * DK + d] = x; });
  if (thread_x() < DK) hdhg[tile * DK + thread_x()] = hdh;
  // a non-finite element of h (or dh) leaves its row's <h, dh> non-finite
  if (thread_x() < DK) ok &= finite_f(hdh);
  const int bad = __syncthreads_or(!ok);
  if (thread_x() == 0) flag[tile] = bad;
}

// Gradient kernel, value part, bf16 activations: the products of k_cw_grad_v
// on bf16 matrix cores (fp32 accumulation).  Every operand is staged to LDS in
// bf16 -- T and Gamma * Kb as the prep wrote them, dh and dU'^T as the reverse
// scan wrote them, v and dO as given, h (the fp32 chunk state) rounded -- and
// R, U' and Y are rounded where they feed a product; w stays fp32, and dv, dw
// are formed from the fp32 Y.  T^T and h (for R) are read down their columns
// with the transposing LDS load.
template <int DK, int DV>
__global__ __launch_bounds__(512) void k_cw_grad_v_bf(Geo geo, int H, const bf16* __restrict__ v,
                                                      const float* __restrict__ w, const bf16* __restrict__ dO,
                                                      const float* __restrict__ states, const bf16* __restrict__ Tg,
                                                      const bf16* __restrict__ KbGg, const bf16* __restrict__ dhg,
                                                      const bf16* __restrict__ dUTg, bf16* __restrict__ dvo,
                                                      float* __restrict__ dwo, float* __restrict__ dPg,
                                                      float* __restrict__ dAg, float* __restrict__ Xg,
                                                      float* __restrict__ dQgg, float* __restrict__ dKhg,
                                                      float* __restrict__ hdhg, int* __restrict__ flag) {
  constexpr int VS = 32, PD = pad_of<bf16>(), LK = DK + PD, LC = CH + PD, LV = VS + PD, LW = VS + 4;
  __shared__ __align__(16) bf16 Ts[CH * LC];                                 // T [i][r]
  __shared__ __align__(16) bf16 KbG[CH * LK];                                // Gamma * Kb [r][d]
  __shared__ __align__(16) bf16 Vs[CH * LV], dOs[CH * LV], Ups[CH * LV], Ys[CH * LV];  // [r][v]
  __shared__ __align__(16) float Ws[CH * LW];                                // w [r][v]
  __shared__ __align__(16) bf16 dUT[VS * LC], RT[VS * LC];                   // dU'^T, R^T [v][r]
  __shared__ __align__(16) bf16 hs[DK * LV], dhs[DK * LV];                   // h, dh [d][v]

  const int ci = blockIdx.x, h = blockIdx.y;
  const ChunkPos cp = chunk_pos(geo, ci);
  const long tile = (long)ci * H + h;
  const long rsv = (long)H * DV, bv = (cp.row0 * H + h) * DV;
  struct Slice {
    CwRows<VS, 512, bf16> v, dO;
    CwRows<VS, 512, float> w;
    TileIn<DK, VS, 512> h;
    OpIn16<DK, VS, DV, 512> dh;
    OpIn16<VS, CH, CH, 512> dut;
  };
  const float* hp = states + tile * DK * DV;
  const bf16* dhp = dhg + tile * DK * DV;
  const bf16* dUp = dUTg + tile * DV * CH;
  auto load_slice = [&](Slice& sl, int c0) {
    sl.v.load(v + bv + c0, rsv, cp.len);
    if (w) sl.w.load(w + bv + c0, rsv, cp.len);
    sl.dO.load(dO + bv + c0, rsv, cp.len);
    sl.h.load(hp + c0, DV);
    sl.dh.load(dhp, 0, c0);
    sl.dut.load(dUp, c0, 0);
  };
  Slice cur, nxt;
  {
    // T, Gamma * Kb and the first value slice in flight together
    CwRows<CH, 512, bf16> tin;
    CwRows<DK, 512, bf16> kin;
    tin.load(Tg + tile * CH * CH, CH, CH);
    kin.load(KbGg + tile * CH * DK, DK, CH);
    load_slice(cur, 0);
    tin.template stage16<LC>(Ts, CH);
    kin.template stage16<LK>(KbG, CH);
  }
  typedef Tiles<CH, VS, 4, 2> TV;
  Tiles<CH, CH, 4, 2> dP, dA;
  Tiles<CH, DK, 4, 2> X, dQg, dKh;
  dP.zero(); dA.zero(); X.zero(); dQg.zero(); dKh.zero();
  float hdh = 0.f;  // thread d < DK: sum over v of h[d][v] dh[d][v]
  bool ok = true;   // v and w finite (the chunk state through <h, dh>)
#pragma unroll
  for (int c0 = 0; c0 < DV; c0 += VS) {
    ok &= cur.v.finite(cp.len);
    if (w) ok &= cur.w.finite(cp.len);
    cur.v.template stage16<LV>(Vs, cp.len);
    if (w) cur.w.template stage<LW>(Ws, cp.len);
    cur.dO.template stage16<LV>(dOs, cp.len);
    cur.h.template stage16<LV>(hs);
    cur.dh.template stage16<LV>(dhs);
    cur.dut.template stage16<LC>(dUT);
    // the next slice's tiles load under this slice's products (the last slice
    // re-reads itself, so the count of loads in flight never changes)
    load_slice(nxt, c0 + VS < DV ? c0 + VS : c0);
    __syncthreads();
    if (thread_x() < DK) {
      const int d = thread_x();
#pragma unroll 8
      for (int c = 0; c < VS; ++c) hdh += to_f(hs[d * LV + c]) * to_f(dhs[d * LV + c]);
    }
    {
      TV rr;
      rr.zero();
      rr.template mma<bf16, DK>(KRow<bf16, LK>{KbG}, KColTr<LV>{hs, nullptr});
      rr.each([&](int r, int vv, float& x) {
        const float wv = w ? Ws[r * LW + vv] : 1.f;
        RT[vv * LC + r] = from_f<bf16>(wv * to_f(Vs[r * LV + vv]) - x);
      });
    }
    {
      TV y;
      y.zero();
      y.template mma<bf16, CH>(KColTr<LC>{Ts, nullptr}, KRow<bf16, LC>{dUT});
      y.each([&](int r, int vv, float& x) {
        Ys[r * LV + vv] = from_f<bf16>(x);
        if (r < cp.len) {
          const long o = bv + (long)r * rsv + c0 + vv;
          dvo[o] = from_f<bf16>((w ? Ws[r * LW + vv] : 1.f) * x);
          if (w) dwo[o] = to_f(Vs[r * LV + vv]) * x;
        }
      });
    }
    __syncthreads();
    {
      TV up;
      up.zero();
      up.template mma<bf16, CH>(KRow<bf16, LC>{Ts}, KRow<bf16, LC>{RT});
      up.each([&](int r, int vv, float& x) { Ups[r * LV + vv] = from_f<bf16>(x); });
    }
    __syncthreads();
    dP.template mma<bf16, VS>(KRow<bf16, LV>{dOs}, KRow<bf16, LV>{Ups});
    dA.template mma<bf16, VS>(KRow<bf16, LV>{Ys}, KRow<bf16, LV>{Ups});
    X.template mma<bf16, VS>(KRow<bf16, LV>{Ys}, KRow<bf16, LV>{hs});
    dQg.template mma<bf16, VS>(KRow<bf16, LV>{dOs}, KRow<bf16, LV>{hs});
    dKh.template mma<bf16, VS>(KRow<bf16, LV>{Ups}, KRow<bf16, LV>{dhs});
    __syncthreads();
    cur = nxt;
  }
  // the same fp32 outputs as k_cw_grad_v
  float* dPt = dPg + tile * CH * CH;
  float* dAt = dAg + tile * CH * CH;
  dP.each([&](int r, int i, float& x) { dPt[r * CH + i] = i <= r ? x : 0.f; });
  dA.each([&](int r, int i, float& x) { dAt[r * CH + i] = i < r ? -x : 0.f; });
  float* Xt = Xg + tile * CH * DK;
  float* Qt = dQgg + tile * CH * DK;
  float* Kt = dKhg + tile * CH * DK;
  X.each([&](int r, int d, float& x) { Xt[r * DK + d] = -x; });
  dQg.each([&](int r, int d, float& x) { Qt[r * DK + d] = x; });
  dKh.each([&](int r, int d, float& x) { Kt[r * DK + d] = x; });
  if (thread_x() < DK) hdhg[tile * DK + thread_x()] = hdh;
  // a non-finite element of h (or dh) leaves its row's <h, dh> non-finite
  if (thread_x() < DK) ok &= finite_f(hdh);
  const int bad = __syncthreads_or(!ok);
  if (thread_x() == 0) flag[tile] = bad;
}

// Gradient kernel, channel part: one block per (chunk, head, 32 channels).
// The four decay-weighted contractions (split by blocks as in the header):
//   dQ^P_rd  = sum_{i<=r} dP_ri K_id  e^{G_rd - G_id}     dK^P_id = sum_{r>=i} dP_ri Q_rd  e^{G_rd - G_id}
//   dKb^A_rd = sum_{i<r}  dA_ri K_id  e^{G_rd - G_id}     dK^A_id = sum_{r>i}  dA_ri Kb_rd e^{G_rd - G_id}
// then dKb = Gamma * X + dKb^A, db = K * dKb, dq = Gamma * dQg + dQ^P,
// dk = e^{G_last - G} * dKhat + dK^P + dK^A + b * dKb, and
//   dG = Gamma Q dQg + Q dQ^P - K dK^P + Kb dKb^A - K dK^A + Gamma Kb X - Khat dKhat
// (elementwise), with e^{G_last} <h, dh>_d + sum_r Khat_rd dKhat_rd added on the
// last row; dg is its reverse cumulative sum down each channel (one wave per
// channel, fixed order).
template <int DK, typename IO>
__global__ __launch_bounds__(512) void k_cw_grad_d(Geo geo, int H, const IO* __restrict__ q,
                                                   const IO* __restrict__ k, const float* __restrict__ g,
                                                   const float* __restrict__ b, const float* __restrict__ dPg,
                                                   const float* __restrict__ dAg, const float* __restrict__ Xg,
                                                   const float* __restrict__ dQgg, const float* __restrict__ dKhg,
                                                   const float* __restrict__ hdhg, IO* __restrict__ dq,
                                                   IO* __restrict__ dk, float* __restrict__ dg,
                                                   float* __restrict__ db) {
  constexpr int DS = 32, LS = DS + 4, LC = CH + 4;
  __shared__ __align__(16) float dPs[CH * LC], dAs[CH * LC];
  __shared__ __align__(16) float Qs[CH * LS], Ks[CH * LS], Bs[CH * LS], Gs[CH * LS];
  __shared__ int wide;  // 16-row blocks whose in-block pairs are summed exactly (bit R: block R)
  float* dGs = Qs;  // dG and Khat * dKhat take Q's and K's tiles once every wave is done with them
  float* Zs = Ks;
  // The channel slices of one (chunk, head) tile re-read its dP and dA: they
  // get block ids b, b + 8, b + 16, ... (blocks are dealt to the 8 XCDs round
  // robin), so they run together on one XCD and share its L2.
  constexpr int NSL = DK / DS;
  const int bid = blockIdx.x, grp = bid / (8 * NSL), within = bid - grp * 8 * NSL;
  const long tile = (long)grp * 8 + (within & 7);
  if (tile >= (long)geo.total_chunks * H) return;  // whole block: the grid is rounded up to groups of 8 tiles
  const int ci = (int)(tile / H), h = (int)(tile - (long)ci * H), d0 = (within >> 3) * DS;
  const ChunkPos cp = chunk_pos(geo, ci);
  const long rsk = (long)H * DK, bk = (cp.row0 * H + h) * DK + d0;
  {
    CwRows<DS, 512, IO> qin, kin;
    CwRows<DS, 512, float> gin, bin;
    TileIn<CH, CH, 512> pin, ain;
    qin.load(q + bk, rsk, cp.len);
    kin.load(k + bk, rsk, cp.len);
    if (g) gin.load(g + bk, rsk, cp.len);
    if (b) bin.load(b + bk, rsk, cp.len);
    pin.load(dPg + tile * CH * CH, CH);
    ain.load(dAg + tile * CH * CH, CH);
    if (thread_x() == 0) wide = 0;
    qin.template stage<LS>(Qs, cp.len);
    kin.template stage<LS>(Ks, cp.len);
    if (g) gin.template stage<LS>(Gs, cp.len);
    else
      for (int i = thread_x(); i < CH * LS; i += blockDim.x) Gs[i] = 0.f;
    if (b) bin.template stage<LS>(Bs, cp.len);
    else
      for (int i = thread_x(); i < CH * LS; i += blockDim.x) Bs[i] = 0.f;
    pin.template stage<LC>(dPs);
    ain.template stage<LC>(dAs);
  }
  __syncthreads();
  if (g) {
    cw_cumsum_columns<DS, LS>(Gs, &wide);
    __syncthreads();
  }

  typedef Tiles<CH, DS, 4, 2> TD;  // the 16 x 16 output tile of each wave
  static_assert(TD::TM == 1 && TD::TN == 1, "one tile per wave");
  const int R = wave_id() / 2;     // the wave's 16-row block
  const bool exact = (wide >> R) & 1;
  const int l = lane_id(), dl = TD::n0(0) + (l & 15);
  const float rf = R > 0 ? Gs[(16 * R - 1) * LS + dl] : 0.f;  // reference before block R
  const float lst = Gs[(16 * R + 15) * LS + dl];               // reference at its last row
  // this lane's X, dQg, dKhat and the <h, dh> of the channels whose dg this
  // wave scans at the end (issued ahead of the products)
  constexpr int NWG = 512 / WAVE;
  static_assert(DS % NWG == 0, "whole dg channels per wave");
  float xin[4], qgin[4], khin[4], hdv[DS / NWG];
#pragma unroll
  for (int it = 0; it < DS / NWG; ++it) hdv[it] = g ? hdhg[tile * DK + d0 + wave_id() + NWG * it] : 0.f;
  {
    const long base = tile * CH * DK + d0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = TD::m0(0) + (l >> 4) * 4 + j;
      xin[j] = Xg[base + r * DK + dl];
      qgin[j] = dQgg[base + r * DK + dl];
      khin[j] = dKhg[base + r * DK + dl];
    }
  }
  // Row sums (output rows r of block R, channel dl) over i in blocks before R
  // and, unless block R is summed exactly, in R (dP and dA are zero above
  // their diagonals): K_id e^{G_ref - G_id}, shared by dP and dA.  Column sums
  // (output rows i of block R) over r in blocks after R, and in R likewise:
  // e^{G_rd - G_last} shared by Q and Kb.  Lane l supplies contraction index
  // 16 cb + 4 (l >> 4) + t at sub-step t on both sides of each product.
  f32x4 aP = {0.f, 0.f, 0.f, 0.f}, aA = aP, bP = aP, bA = aP;
  {
    const int own = 16 * R + (l & 15);
    for (int cb = 0; cb < (exact ? R : R + 1); ++cb) {
      const int i0 = 16 * cb + 4 * (l >> 4);
      const float4 pr = *reinterpret_cast<const float4*>(dPs + own * LC + i0);
      const float4 ar = *reinterpret_cast<const float4*>(dAs + own * LC + i0);
      const float pv[4] = {pr.x, pr.y, pr.z, pr.w}, av[4] = {ar.x, ar.y, ar.z, ar.w};
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int i = i0 + t;
        const float kt = Ks[i * LS + dl] * __expf(rf - Gs[i * LS + dl]);
        aP = Mma<float>::mma(pv[t], kt, aP);
        if (b) aA = Mma<float>::mma(av[t], kt, aA);
      }
    }
    for (int cb = exact ? R + 1 : R; cb < 4; ++cb) {
      const int r0 = 16 * cb + 4 * (l >> 4);
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int r = r0 + t;
        const float e = __expf(Gs[r * LS + dl] - lst);
        bP = Mma<float>::mma(dPs[r * LC + own], Qs[r * LS + dl] * e, bP);
        if (b) bA = Mma<float>::mma(dAs[r * LC + own], Bs[r * LS + dl] * Ks[r * LS + dl] * e, bA);
      }
    }
  }
  // in a block summed exactly: row sums over i in [16R, r] and column sums
  // over r in [i, 16R + 15], one exponential e^{G_r - G_i} per term shared by
  // the dP and dA sums
  float dGv[4], Zv[4];
  {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = TD::m0(0) + (l >> 4) * 4 + j;
      const float G = Gs[r * LS + dl], GL = Gs[(CH - 1) * LS + dl];
      const float gam = __expf(G), dte = __expf(GL - G);
      const float qv = Qs[r * LS + dl], kv = Ks[r * LS + dl], bv = Bs[r * LS + dl], kb = bv * kv;
      const float xv = xin[j], dqg = qgin[j], dkh = khin[j];
      float dqP = 0.f, dkbA = 0.f, dkP = 0.f, dkA = 0.f;
      if (exact) {
        for (int i = 16 * R; i <= r; ++i) {
          const float ke = Ks[i * LS + dl] * __expf(G - Gs[i * LS + dl]);
          dqP += dPs[r * LC + i] * ke;
          dkbA += dAs[r * LC + i] * ke;  // dA is zero on the diagonal
        }
        for (int rr = r; rr <= 16 * R + 15; ++rr) {  // row r plays i
          const float e = __expf(Gs[rr * LS + dl] - G);
          dkP += dPs[rr * LC + r] * Qs[rr * LS + dl] * e;
          dkA += dAs[rr * LC + r] * Bs[rr * LS + dl] * Ks[rr * LS + dl] * e;  // zero at rr == r
        }
      }
      const float ea = __expf(G - rf), eb = __expf(lst - G);
      dqP += aP[j] * ea;
      dkP += bP[j] * eb;
      dkbA = b ? dkbA + aA[j] * ea : 0.f;
      dkA = b ? dkA + bA[j] * eb : 0.f;
      const float dkb = gam * xv + dkbA;
      const float khdkh = dte * kv * dkh;
      dGv[j] = gam * qv * dqg + qv * dqP - kv * dkP + kb * dkbA - kv * dkA + gam * kb * xv - khdkh;
      Zv[j] = khdkh;
      if (r < cp.len) {
        const long o = bk + (long)r * rsk + dl;
        dq[o] = from_f<IO>(gam * dqg + dqP);
        dk[o] = from_f<IO>(dte * dkh + dkP + dkA + bv * dkb);
        if (b) db[o] = kv * dkb;
      }
    }
  }
  if (g) {
    __syncthreads();  // every wave is done with Q and K
    {
      const int l = lane_id(), dl = TD::n0(0) + (l & 15);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = TD::m0(0) + (l >> 4) * 4 + j;
        dGs[r * LS + dl] = dGv[j];
        Zs[r * LS + dl] = Zv[j];
      }
    }
    __syncthreads();
    const int r = lane_id();
#pragma unroll
    for (int it = 0; it < DS / NWG; ++it) {
      const int dl = wave_id() + NWG * it;
      const float tot = wave_sum(Zs[r * LS + dl]);
      float x = dGs[r * LS + dl];
      if (r == CH - 1) x += __expf(Gs[(CH - 1) * LS + dl]) * hdv[it] + tot;
      dGs[r * LS + dl] = wave_reverse(wave_incl_scan(wave_reverse(x)));  // in place: this lane's own entry
    }
    __syncthreads();
    // dg leaves as whole 128-byte row segments (a wave's column would be 64
    // scattered 4-byte stores)
    static_assert(CH * DS / 4 <= 512, "one piece per thread");
    {
      const int i = thread_x(), rr = i / (DS / 4), c = (i - rr * (DS / 4)) * 4;
      if (i < CH * DS / 4 && rr < cp.len)
        *reinterpret_cast<float4*>(dg + bk + (long)rr * rsk + c) = *reinterpret_cast<const float4*>(dGs + rr * LS + c);
    }
  }
}

template <int DK, int DV, typename IO>
static hipError_t launch_cw_fwd_t(const CwFwdArgs& a) {
  constexpr int BV = SCAN_BV, NVT = DV / BV;
  const Geo& geo = a.geo;
  const int H = geo.H;
  const CwFwdWs& w = a.ws;
  stage_mark(a.events, 0, a.stream);
  if (geo.cu != nullptr) {
    const hipError_t e = launch_chunk_offsets(geo.cu, geo.N, const_cast<int*>(geo.chunk_off), a.stream);
    if (e != hipSuccess) return e;
  }
  if (geo.total_chunks > 0)
    hipLaunchKernelGGL((k_cw_prep<DK, DV, false, IO>), dim3(geo.total_chunks, H), dim3(CW_PREP_THREADS), 0, a.stream,
                       geo, H, (const IO*)a.q, (const IO*)a.k, (const IO*)a.v, a.g, a.b, a.w, (const IO*)nullptr,
                       w.gC, (IO*)w.P, (IO*)w.Qg, (IO*)w.KhT, (IO*)w.W, (IO*)w.U,
                       (IO*)nullptr, (IO*)nullptr, (IO*)nullptr, w.flag_prep);
  stage_mark(a.events, 1, a.stream);
  const int NS = geo.N * H;
  if (NS > 0)
    hipLaunchKernelGGL((k_scan_fwd<DK, DV, BV, IO, VAR_GATED, true, IO>), dim3(NS * NVT), dim3(256), 0,
                       a.stream, geo, H, (const IO*)w.Qg, (const IO*)nullptr, a.S0, w.gC, (const IO*)w.W,
                       (const IO*)w.KhT, (const IO*)w.P, (const IO*)w.U, a.states, a.ST, (IO*)a.o,
                       w.flag_scan);
  stage_mark(a.events, 2, a.stream);
  if (NS > 0)
    hipLaunchKernelGGL((k_cw_exact_fwd<DK, DV, IO>), dim3(NS), dim3(DV), 0, a.stream, geo, (const IO*)a.q,
                       (const IO*)a.k, (const IO*)a.v, a.g, a.b, a.w, a.S0, (IO*)a.o, a.ST, a.states,
                       w.flag_prep, w.flag_scan, NVT);
  stage_mark(a.events, 3, a.stream);
  stage_mark(a.events, 4, a.stream);
  return hipGetLastError();
}

template <int DK, int DV, typename IO>
static hipError_t launch_cw_bwd_t(const CwBwdArgs& a) {
  constexpr int BV = SCAN_BV, NVT = DV / BV;
  const Geo& geo = a.geo;
  const int H = geo.H;
  const CwBwdWs& w = a.ws;
  stage_mark(a.events, 0, a.stream);
  if (geo.cu != nullptr) {
    const hipError_t e = launch_chunk_offsets(geo.cu, geo.N, const_cast<int*>(geo.chunk_off), a.stream);
    if (e != hipSuccess) return e;
  }
  if (geo.total_chunks > 0)
    hipLaunchKernelGGL((k_cw_prep<DK, DV, true, IO>), dim3(geo.total_chunks, H), dim3(CW_PREP_THREADS), 0, a.stream,
                       geo, H, (const IO*)a.q, (const IO*)a.k, (const IO*)a.v, a.g, a.b, a.w, (const IO*)a.dO,
                       w.gC, (IO*)w.PT, (IO*)w.QgT, (IO*)w.Kh, (IO*)w.WT, (IO*)nullptr, (IO*)w.T,
                       (IO*)w.KbG, (IO*)w.dOT, w.flag_prep);
  stage_mark(a.events, 1, a.stream);
  const int NS = geo.N * H;
  if (NS > 0)
    hipLaunchKernelGGL((k_scan_bwd<DK, DV, BV, IO, VAR_GATED, true>), dim3(NS * NVT), dim3(256), 0, a.stream,
                       geo, H, (const IO*)w.Kh, a.dST, w.gC, (const IO*)w.WT, (const IO*)w.QgT,
                       (const IO*)w.dOT, (const IO*)w.PT, (IO*)w.dh, (IO*)w.dUT, a.dS0, w.flag_scan);
  stage_mark(a.events, 2, a.stream);
  if (geo.total_chunks > 0) {
    if constexpr (sizeof(IO) == 2)
      hipLaunchKernelGGL((k_cw_grad_v_bf<DK, DV>), dim3(geo.total_chunks, H), dim3(512), 0, a.stream, geo, H,
                         (const bf16*)a.v, a.w, (const bf16*)a.dO, a.states, (const bf16*)w.T, (const bf16*)w.KbG,
                         (const bf16*)w.dh, (const bf16*)w.dUT, (bf16*)a.dv_, a.dw, w.dP, w.dA, w.X, w.dQg,
                         w.dKh, w.hdh, w.flag_grad);
    else
      hipLaunchKernelGGL((k_cw_grad_v<DK, DV>), dim3(geo.total_chunks, H), dim3(512), 0, a.stream, geo, H,
                         (const float*)a.v, a.w, (const float*)a.dO, a.states, (const float*)w.T,
                         (const float*)w.KbG, (const float*)w.dh, (const float*)w.dUT, (float*)a.dv_, a.dw, w.dP,
                         w.dA, w.X, w.dQg, w.dKh, w.hdh, w.flag_grad);
    stage_mark(a.events, 3, a.stream);
    const long tiles = (long)geo.total_chunks * H;
    hipLaunchKernelGGL((k_cw_grad_d<DK, IO>), dim3((unsigned)((tiles + 7) / 8 * 8 * (DK / 32))), dim3(512), 0,
                       a.stream, geo, H, (const IO*)a.q, (const IO*)a.k, a.g, a.b, (const float*)w.dP, (const float*)w.dA, (const float*)w.X,
                       (const float*)w.dQg, (const float*)w.dKh, (const float*)w.hdh, (IO*)a.dq, (IO*)a.dk_, a.dg, a.db);
  } else {
    stage_mark(a.events, 3, a.stream);
  }
  if (NS > 0)
    hipLaunchKernelGGL((k_cw_exact_bwd<DK, DV, IO>), dim3(EXACT_SLOTS), dim3(DV), 0, a.stream, geo,
                       (const IO*)a.q, (const IO*)a.k, (const IO*)a.v, a.g, a.b, a.w, a.states, (const IO*)a.dO,
                       a.dST, (IO*)a.dq, (IO*)a.dk_, (IO*)a.dv_, a.dg, a.db, a.dw, a.dS0, w.flag_prep,
                       w.flag_grad, w.flag_scan, NVT, w.exact);
  stage_mark(a.events, 4, a.stream);
  return hipGetLastError();
}

}  // namespace gdn
