// Chunk-local pieces shared by the forward and backward kernels: tile loads
// and stores between HBM and LDS, the in-chunk gates, and the triangular
// inverse T = (I + A)^{-1} of the delta rule's erase coupling (paper Sec. 4.2,
// K#2: the forward computes T once per chunk and the backward reuses it).
#pragma once

#include "gdn_common.hpp"

namespace gdn {

template <typename T> constexpr int pad_of() { return 16 / (int)sizeof(T); }

// Element j of a 16-byte vector of T, and packing of T values into 16 bytes,
// by explicit bit casts (no pointer type punning of register values).
__device__ __forceinline__ uint32_t word_of(const uint4& u, int i) {
  return i == 0 ? u.x : (i == 1 ? u.y : (i == 2 ? u.z : u.w));
}
template <typename T> __device__ __forceinline__ T elem16(const uint4& u, int j);
template <> __device__ __forceinline__ bf16 elem16<bf16>(const uint4& u, int j) {
  return __builtin_bit_cast(bf16, (unsigned short)(word_of(u, j >> 1) >> ((j & 1) * 16)));
}
template <> __device__ __forceinline__ float elem16<float>(const uint4& u, int j) {
  return __builtin_bit_cast(float, word_of(u, j));
}
__device__ __forceinline__ uint32_t pack2(bf16 lo, bf16 hi) {
  return (uint32_t)__builtin_bit_cast(unsigned short, lo) | ((uint32_t)__builtin_bit_cast(unsigned short, hi) << 16);
}
// 16 bytes of T from 16 / sizeof(T) values
template <typename T> __device__ __forceinline__ uint4 pack16(const T* x);
template <> __device__ __forceinline__ uint4 pack16<bf16>(const bf16* x) {
  return uint4{pack2(x[0], x[1]), pack2(x[2], x[3]), pack2(x[4], x[5]), pack2(x[6], x[7])};
}
template <> __device__ __forceinline__ uint4 pack16<float>(const float* x) {
  return uint4{__builtin_bit_cast(uint32_t, x[0]), __builtin_bit_cast(uint32_t, x[1]),
               __builtin_bit_cast(uint32_t, x[2]), __builtin_bit_cast(uint32_t, x[3])};
}

__device__ __forceinline__ bool finite8_bf16(uint4 u) {
  // a bf16 value is non-finite when its 8 exponent bits are all ones
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
  bool ok = true;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    ok &= (w[i] & 0x7f80u) != 0x7f80u;
    ok &= (w[i] & 0x7f800000u) != 0x7f800000u;
  }
  return ok;
}
__device__ __forceinline__ bool finite4_f32(uint4 u) {
  return ((u.x & 0x7f800000u) != 0x7f800000u) & ((u.y & 0x7f800000u) != 0x7f800000u) &
         ((u.z & 0x7f800000u) != 0x7f800000u) & ((u.w & 0x7f800000u) != 0x7f800000u);
}
template <typename T> __device__ __forceinline__ bool finite16B(uint4 u);
template <> __device__ __forceinline__ bool finite16B<bf16>(uint4 u) { return finite8_bf16(u); }
template <> __device__ __forceinline__ bool finite16B<float>(uint4 u) { return finite4_f32(u); }

// 4 consecutive elements of the operand type as one load/store unit.
template <typename T> struct vec4_of;
template <> struct vec4_of<bf16> { typedef uint2 type; };
template <> struct vec4_of<float> { typedef uint4 type; };
template <typename T> __device__ __forceinline__ T elem4(const typename vec4_of<T>::type& u, int j);
template <> __device__ __forceinline__ bf16 elem4<bf16>(const uint2& u, int j) {
  return __builtin_bit_cast(bf16, (unsigned short)((j < 2 ? u.x : u.y) >> ((j & 1) * 16)));
}
template <> __device__ __forceinline__ float elem4<float>(const uint4& u, int j) {
  return elem16<float>(u, j);
}
template <typename T> __device__ __forceinline__ typename vec4_of<T>::type pack4(const T* x);
template <> __device__ __forceinline__ uint2 pack4<bf16>(const bf16* x) {
  return uint2{pack2(x[0], x[1]), pack2(x[2], x[3])};
}
template <> __device__ __forceinline__ uint4 pack4<float>(const float* x) { return pack16<float>(x); }

// Backward chunk prep: everything the reverse scan needs per chunk, laid out
// for direct MFMA fragment loads: P^T (P = (Q K^T) * D), W^T with
// W = T diag(beta e^G) K, (diag(e^G) Q)^T and dO^T, plus the cumulative decay.
// Copy rows [0, len) of a 64 x D tile whose rows sit `rs` elements apart in
// HBM into LDS dst[r * LD + d]; rows >= len are zero-filled.  Returns false
// if any loaded value is NaN or Inf.
template <int D, int LD, typename T>
__device__ __forceinline__ bool load_rows(const T* __restrict__ src, long rs, int len, T* dst) {
  constexpr int V = 16 / (int)sizeof(T);  // elements per 16-byte vector
  constexpr int PER_ROW = D / V;
  bool ok = true;
  for (int idx = thread_x(); idx < CH * PER_ROW; idx += blockDim.x) {
    const int r = idx / PER_ROW, c = (idx - r * PER_ROW) * V;
    const uint4 u = keep16(r < len, *reinterpret_cast<const uint4*>(src + clamp_row(r, len) * rs + c));
    ok &= finite16B<T>(u);
    *reinterpret_cast<uint4*>(dst + r * LD + c) = u;
  }
  return ok;
}

// Copy a contiguous R x D tile (row-major in HBM) into LDS with row stride LD.
template <int R, int D, int LD, typename T>
__device__ __forceinline__ void load_dense(const T* __restrict__ src, T* dst) {
  constexpr int V = 16 / (int)sizeof(T);
  constexpr int PER_ROW = D / V;
  for (int idx = thread_x(); idx < R * PER_ROW; idx += blockDim.x) {
    const int r = idx / PER_ROW, c = (idx - r * PER_ROW) * V;
    *reinterpret_cast<uint4*>(dst + r * LD + c) = *reinterpret_cast<const uint4*>(src + (long)r * D + c);
  }
}

// Write rows [0, len) of an LDS tile src[r * LD + d] (64 x D) to HBM rows `rs`
// elements apart.
// Rows [0, len) of a 64 x D chunk tile (rows rs elements apart in HBM), read
// by a block of NT threads in one batch: load() puts every 16-byte piece in
// flight at once (a load/wait/store loop would pay one memory round trip per
// iteration), stage() masks the rows past the end and writes the tile to LDS.
template <int D, int NT, typename T>
struct RowsIn {
  static constexpr int V = 16 / (int)sizeof(T), PER_ROW = D / V, N = CH * PER_ROW / NT;
  static_assert(CH * PER_ROW % NT == 0, "whole pieces per thread");
  uint4 u[N];
  __device__ __forceinline__ void load(const T* __restrict__ src, long rs, int len) {
#pragma unroll
    for (int t = 0; t < N; ++t) {
      const int idx = thread_x() + t * NT, r = idx / PER_ROW, c = (idx - r * PER_ROW) * V;
      u[t] = *reinterpret_cast<const uint4*>(src + clamp_row(r, len) * rs + c);
    }
  }
  template <int LD>
  __device__ __forceinline__ bool stage(T* dst, int len) const {
    bool ok = true;
#pragma unroll
    for (int t = 0; t < N; ++t) {
      const int idx = thread_x() + t * NT, r = idx / PER_ROW, c = (idx - r * PER_ROW) * V;
      const uint4 x = keep16(r < len, u[t]);
      ok &= finite16B<T>(x);
      *reinterpret_cast<uint4*>(dst + r * LD + c) = x;
    }
    return ok;
  }
};

template <int D, int LD, typename T>
__device__ __forceinline__ void store_rows(T* __restrict__ dst, long rs, int len, const T* src) {
  constexpr int V = 16 / (int)sizeof(T);
  constexpr int PER_ROW = D / V;
  for (int idx = thread_x(); idx < CH * PER_ROW; idx += blockDim.x) {
    const int r = idx / PER_ROW, c = (idx - r * PER_ROW) * V;
    if (r < len)
      *reinterpret_cast<uint4*>(dst + row_off(r, (int)rs) + c) = *reinterpret_cast<const uint4*>(src + r * LD + c);
  }
}

// In-chunk gates, computed by wave 0: G_r = sum_{s<=r} g_s (positions past the
// chunk's end add 0, so G there equals the last valid G), beta_r (0 past the
// end).  Returns false (on wave 0) if a loaded gate is non-finite.
template <int VAR>
__device__ __forceinline__ bool load_gates(const float* __restrict__ g, const float* __restrict__ beta,
                                           long row0, int H, int h, int len, float* Gs, float* Bs) {
  bool ok = true;
  if (wave_id() == 0) {
    const int r = lane_id();
    float gv = 0.f, bv = 0.f;
    const long o = (row0 + clamp_row(r, len)) * H + h;
    if (VAR != VAR_DELTA) {
      const float x = g[o];
      gv = r < len ? x : 0.f;
    }
    if (VAR != VAR_DECAY) {
      const float x = beta[o];
      bv = r < len ? x : 0.f;
    }
    ok = finite_f(gv) && finite_f(bv);
    Gs[r] = wave_incl_scan(gv);
    Bs[r] = bv;
  }
  return ok;
}

// T = (I + A)^{-1} for the strictly lower-triangular 64 x 64 matrix A held in
// fp32 in As (row stride LC), by blocked forward substitution over 16 x 16
// blocks.
//   Diagonal blocks: wave 0, one lane per (block, column); row r of a block's
//   inverse is e_r - sum_{i<r} A_ri T_i.
//   Blocks below the diagonal: wave j builds block column j top-down,
//   T_ij = -T_ii sum_{k=j}^{i-1} A_ik T_kj, on fp32 MFMA with the column's
//   finished blocks kept in accumulator registers.  The contraction index of
//   every 16x16x4 product is enumerated as k = 4 * (lane group) + step, which
//   makes an accumulator tile (lane holds rows 4g..4g+3 of column c) a ready B
//   operand, so no block leaves registers until it is stored.
// T lands in Tf (fp32, stride LC, zeros above the block diagonal); for bf16
// operands a rounded copy goes to Ts (stride LT) and, if TRANS, T^T to TT.
// Called by all threads of the block; ends with a barrier.
template <typename OP, int LC, int LT, bool TRANS>
__device__ __forceinline__ void unit_lower_inverse(const float* As, float* Tf, OP* Ts, OP* TT) {
  constexpr bool BF = sizeof(OP) == 2;
  const int w = wave_id(), l = lane_id(), g = l >> 4, c = l & 15;
  // the six blocks above the diagonal are zero (T^T: below it)
  for (int idx = thread_x(); idx < 6 * 256; idx += blockDim.x) {
    const int blk = idx >> 8, rr = (idx >> 4) & 15, cc = idx & 15;
    const int bi = blk < 3 ? 0 : (blk < 5 ? 1 : 2);
    const int bj = blk < 3 ? blk + 1 : (blk < 5 ? blk - 1 : 3);
    const int r = 16 * bi + rr, col = 16 * bj + cc;
    Tf[r * LC + col] = 0.f;
    if constexpr (BF) Ts[r * LT + col] = from_f<OP>(0.f);
    if constexpr (TRANS) TT[col * LT + r] = from_f<OP>(0.f);
  }
  if (w == 0) {
    // right-looking: once col_i is final, add its term to every later row, so
    // consecutive FMAs are independent (the sum over i still runs in order)
    const int base = 16 * g;
    float col[16], acc[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[r] = 0.f;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      col[i] = (i == c) ? 1.f : (i > c ? -acc[i] : 0.f);
#pragma unroll
      for (int r = i + 1; r < 16; ++r) acc[r] += As[(base + r) * LC + base + i] * col[i];
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      Tf[(base + r) * LC + base + c] = col[r];
      if constexpr (BF) Ts[(base + r) * LT + base + c] = from_f<OP>(col[r]);
    }
    if constexpr (TRANS) {
      OP t16[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) t16[r] = from_f<OP>(col[r]);
      if constexpr (BF) {
        *reinterpret_cast<uint4*>(TT + (base + c) * LT + base) = pack16<OP>(t16);
        *reinterpret_cast<uint4*>(TT + (base + c) * LT + base + 8) = pack16<OP>(t16 + 8);
      } else {
#pragma unroll
        for (int r = 0; r < 16; ++r) TT[(base + c) * LT + base + r] = t16[r];
      }
    }
  }
  __syncthreads();
  if (w < 3) {
    // block column j, right-looking over block rows: x_i accumulates
    // A_ik T_kj as soon as T_kj is known, so only one 4-MFMA chain per block
    // row lies on the critical path
    const int j = w;
    float4 ab[4][3], ti[4];
#pragma unroll
    for (int i = 1; i < 4; ++i) {
      ti[i] = *reinterpret_cast<const float4*>(Tf + (16 * i + c) * LC + 16 * i + 4 * g);
#pragma unroll
      for (int kb = 0; kb < i; ++kb)
        ab[i][kb] = *reinterpret_cast<const float4*>(As + (16 * i + c) * LC + 16 * kb + 4 * g);
    }
    f32x4 tk;  // T_kj of the latest finished block row k
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) tk[jj] = Tf[(16 * j + 4 * g + jj) * LC + 16 * j + c];
    f32x4 x[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) x[i] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int k = 0; k < 3; ++k) {
      if (k < j) continue;
      // x_i += A_ik T_kj for every later block row i
#pragma unroll
      for (int i = k + 1; i < 4; ++i) {
        x[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(ab[i][k].x, tk[0], x[i], 0, 0, 0);
        x[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(ab[i][k].y, tk[1], x[i], 0, 0, 0);
        x[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(ab[i][k].z, tk[2], x[i], 0, 0, 0);
        x[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(ab[i][k].w, tk[3], x[i], 0, 0, 0);
      }
      // T_{k+1,j} = -T_{k+1,k+1} x_{k+1}
      const int i = k + 1;
      f32x4 t = {0.f, 0.f, 0.f, 0.f};
      t = __builtin_amdgcn_mfma_f32_16x16x4f32(ti[i].x, x[i][0], t, 0, 0, 0);
      t = __builtin_amdgcn_mfma_f32_16x16x4f32(ti[i].y, x[i][1], t, 0, 0, 0);
      t = __builtin_amdgcn_mfma_f32_16x16x4f32(ti[i].z, x[i][2], t, 0, 0, 0);
      t = __builtin_amdgcn_mfma_f32_16x16x4f32(ti[i].w, x[i][3], t, 0, 0, 0);
      OP t4[4];
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        tk[jj] = -t[jj];
        t4[jj] = from_f<OP>(-t[jj]);
        Tf[(16 * i + 4 * g + jj) * LC + 16 * j + c] = -t[jj];
        if constexpr (BF) Ts[(16 * i + 4 * g + jj) * LT + 16 * j + c] = t4[jj];
      }
      if constexpr (TRANS) {
        if constexpr (BF) {
          *reinterpret_cast<uint2*>(TT + (16 * j + c) * LT + 16 * i + 4 * g) = uint2{pack2(t4[0], t4[1]), pack2(t4[2], t4[3])};
        } else {
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) TT[(16 * j + c) * LT + 16 * i + 4 * g + jj] = t4[jj];
        }
      }
    }
  }
  __syncthreads();
}

// A fragments (for the rows this wave owns in Tiles TT) of a pre-arranged
// operand with K contraction columns, laid out by op_off: one contiguous
// 16-byte read per lane for bf16, the row-major view for fp32.
template <class TT, typename OP, int K>
__device__ __forceinline__ void load_op_frags(typename TT::template AFr<OP, K>& f, const OP* base) {
  if constexpr (sizeof(OP) == 2) {
    const int l = lane_id();
#pragma unroll
    for (int s = 0; s < K / 32; ++s)
#pragma unroll
      for (int a = 0; a < TT::TM; ++a)
        f.f[s][a] = *reinterpret_cast<const bf16x8*>(base + ((long)((TT::m0(a) >> 4) * (K / 32) + s) * 64 + l) * 8);
  } else {
    f.load(KRow<OP, K>{base});
  }
}
// The same for B fragments (the columns this wave owns), n playing the row.
template <class TT, typename OP, int K>
__device__ __forceinline__ void load_op_frags_b(typename TT::template BFr<OP, K>& f, const OP* base) {
  if constexpr (sizeof(OP) == 2) {
    const int l = lane_id();
#pragma unroll
    for (int s = 0; s < K / 32; ++s)
#pragma unroll
      for (int b = 0; b < TT::TN; ++b)
        f.f[s][b] = *reinterpret_cast<const bf16x8*>(base + ((long)((TT::n0(b) >> 4) * (K / 32) + s) * 64 + l) * 8);
  } else {
    f.load(KRow<OP, K>{base});
  }
}

// XCD-aware placement of the (stream, value-tile) blocks of a state scan:
// blocks are dealt to the 8 XCDs round robin, so the value tiles of one
// stream get block ids that are equal modulo 8 and share that XCD's L2.
__device__ __forceinline__ void scan_block_coords(int bid, int NS, int NVT, int& s, int& vt) {
  if ((NS & 7) == 0) {
    const int x = bid & 7, slot = bid >> 3;
    s = (slot / NVT) * 8 + x;
    vt = slot - (slot / NVT) * NVT;
  } else {
    s = bid / NVT;
    vt = bid - s * NVT;
  }
}

}  // namespace gdn
