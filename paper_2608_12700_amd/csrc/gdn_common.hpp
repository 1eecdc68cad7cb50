// Device-side building blocks shared by the gated-delta-rule kernels (gfx950).
//
// Matrix products run on 16x16 MFMA tiles: v_mfma_f32_16x16x32_bf16 for bf16
// operands and v_mfma_f32_16x16x4_f32 for fp32 operands, always with fp32
// accumulation.  Lane l of a wave owns row/column (l & 15) of a tile and the
// k-group (l >> 4); the 16x16 fp32 result sits as C[4*(l>>4) + j][l & 15],
// j = 0..3, in four accumulator registers.  Operands are read from LDS through
// small "view" objects that map (outer index, k) to an element, so one product
// routine serves every transpose the chunk algebra needs; a view whose k index
// is contiguous turns into 16-byte LDS reads.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gdn_geo.hpp"

namespace gdn {

constexpr int CH = 64;  // chunk length (tokens)
constexpr int WAVE = 64;

typedef __bf16 bf16;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;

__device__ __forceinline__ float to_f(float x) { return x; }
__device__ __forceinline__ float to_f(bf16 x) { return static_cast<float>(x); }
template <typename T> __device__ __forceinline__ T from_f(float x);

template <int DT> struct op_of;
template <> struct op_of<DT_F32> { typedef float type; };
template <> struct op_of<DT_BF16> { typedef bf16 type; };
template <> __device__ __forceinline__ float from_f<float>(float x) { return x; }
template <> __device__ __forceinline__ bf16 from_f<bf16>(float x) { return static_cast<bf16>(x); }

// Thread index within the block.  A translation unit whose kernel walks
// several tiles in one launch defines GDN_TILE_LOOP: the index then reads
// gdn_tid_bias, an LDS word that is always 0 and that the kernel stores again
// on every pass of its tile loop.  Index arithmetic derived from it can be
// neither hoisted out of the loop (where it would sit in registers through
// every phase) nor carried across a barrier; it is recomputed next to its
// uses.  Such a kernel stores the word before its first barrier.
#ifdef GDN_TILE_LOOP
__shared__ int gdn_tid_bias;
__device__ __forceinline__ int thread_x() { return (int)threadIdx.x + gdn_tid_bias; }
#else
__device__ __forceinline__ int thread_x() { return (int)threadIdx.x; }
#endif
__device__ __forceinline__ int lane_id() { return (int)((unsigned)thread_x() & (WAVE - 1)); }
__device__ __forceinline__ int wave_id() { return (int)((unsigned)thread_x() / WAVE); }

// Value of x held by lane src (0..63) of the wave; addresses outside the
// wave wrap around.
__device__ __forceinline__ float shfl_idx(float x, int src) {
  return __builtin_bit_cast(float, __builtin_amdgcn_ds_bpermute(src << 2, __builtin_bit_cast(int, x)));
}
__device__ __forceinline__ float shfl_xor(float x, int m) { return shfl_idx(x, lane_id() ^ m); }

__device__ __forceinline__ bool finite_f(float x) {
  return (__float_as_uint(x) & 0x7f800000u) != 0x7f800000u;
}

// A zero the compiler cannot see through, held in a vector register.  Added to
// an otherwise uniform index it keeps a prefetch on the vector memory path: a
// uniform address becomes a scalar load, and copying its result into the
// prefetch registers makes the wave wait for it on the spot.
__device__ __forceinline__ int opaque_zero() {
  int z;
  asm volatile("v_mov_b32 %0, 0" : "=v"(z));
  return z;
}

// Layout of a pre-arranged MFMA operand of K columns (contraction index k) in
// HBM.  bf16: fragment-major -- the 8 elements lane l contributes to k-step s
// of 16-row tile mt are contiguous and the 64 lanes' pieces of one (mt, s)
// form one 1 KiB block, so a wave's fragment load reads whole cache lines.
// fp32: row-major.  Runs of 4 (or 8) consecutive k starting at a multiple of 4
// (or 8) stay contiguous in both.
template <typename OP, int K>
__device__ __forceinline__ long op_off(int m, int k) {
  if constexpr (sizeof(OP) == 2)
    return ((long)((m >> 4) * (K / 32) + (k >> 5)) * 64 + (m & 15) + 16 * ((k & 31) >> 3)) * 8 + (k & 7);
  else
    return (long)m * K + k;
}

// Token-major rows of a chunk operand (64 rows of DK 16-bit values, the
// contraction index contiguous) gathered into LDS for MFMA fragment reads by
// 1 KiB copies: block I holds 8 rows x one 128-byte line of each (DK / 64
// lines per row), so every copy instruction reads whole lines.  Within a row
// the eight 16-byte pieces of a line are permuted by (row >> 1) & 7: the 16
// rows of one fragment read then fall on distinct LDS banks.
template <int DK>
struct RowLines {
  static constexpr int LPR = DK / 64;         // 128-byte lines per row
  static constexpr int NBLK = CH * LPR / 8;   // 1 KiB blocks per chunk
  // lane l of block I copies row `row`, elements e .. e + 7
  __device__ __forceinline__ static void src(int I, int l, int& row, int& e) {
    const int rg = I / LPR, hl = I - rg * LPR;
    row = 8 * rg + (l >> 3);
    e = hl * 64 + (((l & 7) ^ ((row >> 1) & 7)) << 3);
  }
  // 16-byte slot, from the first block, of row r, elements k0 .. k0 + 7 (k0 % 8 == 0)
  __device__ __forceinline__ static int slot(int r, int k0) {
    const int p = k0 >> 3, hl = p >> 3;
    return ((r >> 3) * LPR + hl) * 64 + 8 * (r & 7) + ((p & 7) ^ ((r >> 1) & 7));
  }
  // lane l's slot of the A fragment (rows 16 mt .. 16 mt + 15, k-step st of 32)
  __device__ __forceinline__ static int frag_slot(int mt, int st, int l) {
    return slot(16 * mt + (l & 15), 32 * st + 8 * (l >> 4));
  }
};

// Layout of a 64 x D fp32 chunk operand read as accumulator tiles of
// Tiles<64, BV, 4, 1> (one 16-row tile per wave, BV-column value tiles): the
// four rows r..r+3 (r % 4 == 0) of column v that one lane holds are one float4,
// and the 64 lanes' float4 of one 16 x 16 tile are one 1 KiB block.
template <int BV>
__device__ __forceinline__ long cfrag_off(int r, int v) {
  return ((((long)(v / BV) * 4 + (r >> 4)) * (BV / 16) + ((v % BV) >> 4)) * 64 + (v & 15) + 16 * ((r & 15) >> 2)) * 4;
}

// Offset of row `row` (0 <= row < 64) of a token-major tile with row stride
// `stride` elements (stride < 2^24, which the C ABI checks): one full-rate
// 24-bit multiply.  The chunk's own base offset is formed separately in 64 bits.
__device__ __forceinline__ unsigned row_off(int row, int stride) {
  return __umul24((unsigned)row, (unsigned)stride);
}

// Masked tile rows: rows r >= len of a chunk are read from row len - 1
// (len >= 1 for every chunk) and zeroed with a select afterwards.  Keeping
// the load itself unconditional matters: a branch around a load forces the
// wave to wait for it at the join, which serialises every masked load.
__device__ __forceinline__ int clamp_row(int r, int len) { return r < len ? r : len - 1; }
__device__ __forceinline__ uint4 keep16(bool keep, uint4 u) {
  return uint4{keep ? u.x : 0u, keep ? u.y : 0u, keep ? u.z : 0u, keep ? u.w : 0u};
}
__device__ __forceinline__ uint2 keep8(bool keep, uint2 u) { return uint2{keep ? u.x : 0u, keep ? u.y : 0u}; }

// ---------------------------------------------------------------------------
// Operand views.  get(o, k): o is the row for an A operand (M x K) or the
// column for a B operand (K x N); k is the contraction index.
// ---------------------------------------------------------------------------

// Element (o, k) at p[o * LD + k]: k contiguous.
template <typename T, int LD>
struct KRow {
  const T* p;
  static constexpr bool kVec = true;
  __device__ __forceinline__ T get(int o, int k) const { return p[o * LD + k]; }
  __device__ __forceinline__ const T* ptr(int o, int k) const { return p + o * LD + k; }
};

// Element (o, k) at p[o * ld + k] with a runtime row stride; rows o >= rows
// read as zero (tail chunks read straight from the token-major inputs).
template <typename T>
struct KRowM {
  const T* p;
  long ld;
  int rows;
  static constexpr bool kVec = false;
  static constexpr bool kMasked = true;
  __device__ __forceinline__ T get(int o, int k) const {
    const T x = p[clamp_row(o, rows) * ld + k];
    return o < rows ? x : static_cast<T>(0.f);
  }
  __device__ __forceinline__ const T* ptr(int o, int k) const { return p + o * ld + k; }
};

// Element (o, k) at p[min(o, rows - 1) * ld + k]: rows past the end repeat the
// last valid row.  For operands whose rows past a chunk's end only reach
// results that are masked later, so the load needs no select (and no wait).
template <typename T>
struct KRowC {
  const T* p;
  long ld;
  int rows;
  static constexpr bool kVec = true;
  __device__ __forceinline__ T get(int o, int k) const { return p[clamp_row(o, rows) * ld + k]; }
  __device__ __forceinline__ const T* ptr(int o, int k) const { return p + clamp_row(o, rows) * ld + k; }
};

// Element (o, k) at p[k * LD + o]: o contiguous (a transposed use).
template <typename T, int LD>
struct KCol {
  const T* p;
  static constexpr bool kVec = false;
  __device__ __forceinline__ T get(int o, int k) const { return p[k * LD + o]; }
};

// Element (o, k) at p[k * LD + o] of a 16-bit LDS array (o contiguous), read
// with gfx950's transposing LDS load: a fragment takes two ds_read_b64_tr_b16
// instead of eight 2-byte gathers.  With SCALED, element (o, k) is multiplied
// by sc[k] (fp32, 16-byte aligned) before it is rounded back to bf16.
template <int LD, bool SCALED = false>
struct KColTr {
  const bf16* p;
  const float* sc;
  static constexpr bool kVec = false;
  static constexpr bool kTr = true;
};

// ds_read_b64_tr_b16: in each 16-lane group, lane s points at four
// consecutive 16-bit elements (row s >> 2 of a 4 x 16 block, columns
// 4 (s & 3) .. 4 (s & 3) + 3); lane i of the group receives column i of the
// block, rows 0..3, as four 16-bit values.
typedef __attribute__((ext_vector_type(4))) short i16x4;
__device__ __forceinline__ uint2 lds_read_tr16(const bf16* p) {
  typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
  const i16x4 r = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p));
  return __builtin_bit_cast(uint2, r);
}

// MFMA fragment (rows o..o+15, contraction k0..k0+31) of a matrix stored
// k-major in LDS, p[k * LD + o]: lane l receives o + (l & 15) and the eight
// k = k0 + 8 (l >> 4) + j, j = 0..7, the same placement a row-major read gives.
template <int LD>
__device__ __forceinline__ bf16x8 lds_frag_tr(const bf16* p, int o, int k0) {
  static_assert(LD % 4 == 0, "8-byte aligned rows");
  const int l = lane_id(), s = l & 15;
  const bf16* a = p + (k0 + 8 * (l >> 4) + (s >> 2)) * LD + o + 4 * (s & 3);
  const uint2 lo = lds_read_tr16(a), hi = lds_read_tr16(a + 4 * LD);
  return __builtin_bit_cast(bf16x8, uint4{lo.x, lo.y, hi.x, hi.y});
}

// Scale the eight k-values of a fragment by sc[k0 + 8 (l >> 4) + j].
__device__ __forceinline__ bf16x8 scale_frag(bf16x8 f, const float* sc, int k0) {
  const float* s8 = sc + k0 + 8 * (lane_id() >> 4);
  const float4 a = *reinterpret_cast<const float4*>(s8), b = *reinterpret_cast<const float4*>(s8 + 4);
  const float m[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
  for (int j = 0; j < 8; ++j) f[j] = static_cast<bf16>(static_cast<float>(f[j]) * m[j]);
  return f;
}

// Element computed by a functor f(o, k) -> T.
template <typename T, class F>
struct KFun {
  F f;
  static constexpr bool kVec = false;
  __device__ __forceinline__ T get(int o, int k) const { return f(o, k); }
};
template <typename T, class F>
__device__ __forceinline__ KFun<T, F> kfun(F f) { return KFun<T, F>{f}; }

template <class V, class = void> struct is_masked { static constexpr bool value = false; };
template <class V> struct is_masked<V, decltype((void)V::kMasked)> { static constexpr bool value = true; };
template <class V, class = void> struct is_tr { static constexpr bool value = false; };
template <class V> struct is_tr<V, decltype((void)V::kTr)> { static constexpr bool value = true; };
template <int LD, bool S>
__device__ __forceinline__ bf16x8 tr_load(const KColTr<LD, S>& v, int o, int k0) {
  const bf16x8 f = lds_frag_tr<LD>(v.p, o, k0);
  if constexpr (S) return scale_frag(f, v.sc, k0); else return f;
}

template <typename OP> struct Mma;

template <>
struct Mma<bf16> {
  static constexpr int KSTEP = 32;
  typedef bf16x8 frag;
  template <class V>
  __device__ __forceinline__ static frag load(const V& v, int o, int k0) {
    const int l = lane_id();
    const int oo = o + (l & 15), kk = k0 + (l >> 4) * 8;
    if constexpr (V::kVec) {
      return *reinterpret_cast<const bf16x8*>(v.ptr(oo, kk));
    } else if constexpr (is_tr<V>::value) {
      return tr_load(v, o, k0);
    } else if constexpr (is_masked<V>::value) {
      const uint4 u = *reinterpret_cast<const uint4*>(v.ptr(clamp_row(oo, v.rows), kk));
      return __builtin_bit_cast(frag, keep16(oo < v.rows, u));
    } else {
      frag r;
#pragma unroll
      for (int j = 0; j < 8; ++j) r[j] = v.get(oo, kk + j);
      return r;
    }
  }
  __device__ __forceinline__ static f32x4 mma(frag a, frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
};

// fp32: the contraction is enumerated in groups of 16 -- in group G, lane l
// supplies k = 16 G + 4 (l >> 4) + t at sub-step t (k-step k0 = 16 G + 4 t) --
// so a lane's four operands of a group are contiguous on both sides of every
// product: one 16-byte load (load4) serves four k-steps.  Every fp32 fragment
// goes through load or load4, so A and B always agree on the enumeration.
template <>
struct Mma<float> {
  static constexpr int KSTEP = 4;
  typedef float frag;
  template <class V>
  __device__ __forceinline__ static frag load(const V& v, int o, int k0) {
    const int l = lane_id();
    return v.get(o + (l & 15), (k0 & ~15) + 4 * (l >> 4) + ((k0 & 15) >> 2));
  }
  // the four sub-steps of group k16 / 16 (k16 % 16 == 0), for views with ptr()
  template <class V>
  __device__ __forceinline__ static f32x4 load4(const V& v, int o, int k16) {
    const int l = lane_id();
    return *reinterpret_cast<const f32x4*>(v.ptr(o + (l & 15), k16 + 4 * (l >> 4)));
  }
  __device__ __forceinline__ static f32x4 mma(frag a, frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
};

// A wave-level register-blocked product: the waves of a block form a WM x WN
// grid over the (M/16) x (N/16) output tiles; wave (wm, wn) owns TM x TN tiles
// and reuses each loaded fragment across its row or column of tiles.
template <int M, int N, int WM, int WN>
struct Tiles {
  static_assert(M % (16 * WM) == 0 && N % (16 * WN) == 0, "tile grid");
  static constexpr int TM = M / 16 / WM;
  static constexpr int TN = N / 16 / WN;
  f32x4 acc[TM][TN];

  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int a = 0; a < TM; ++a)
#pragma unroll
      for (int b = 0; b < TN; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  __device__ __forceinline__ static int m0(int a) { return ((wave_id() / WN) * TM + a) * 16; }
  __device__ __forceinline__ static int n0(int b) { return ((wave_id() % WN) * TN + b) * 16; }

  // acc += A (M x K) * B (K x N), K a multiple of the MFMA k-step.
  template <typename OP, int K, class VA, class VB>
  __device__ __forceinline__ void mma(const VA& A, const VB& B) {
    typedef Mma<OP> X;
    if constexpr (sizeof(OP) == 4 && VA::kVec && VB::kVec) {
      static_assert(K % 16 == 0, "whole groups of the fp32 enumeration");
      // one group (4 x TM x TN products) per iteration; with few output tiles a
      // second group in flight hides the loads, with more it would only double
      // the live fragments
      auto group = [&](int k16) __attribute__((always_inline)) {
        f32x4 fa[TM], fb[TN];
#pragma unroll
        for (int a = 0; a < TM; ++a) fa[a] = X::load4(A, m0(a), k16);
#pragma unroll
        for (int b = 0; b < TN; ++b) fb[b] = X::load4(B, n0(b), k16);
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
          for (int a = 0; a < TM; ++a)
#pragma unroll
            for (int b = 0; b < TN; ++b) acc[a][b] = X::mma(fa[a][t], fb[b][t], acc[a][b]);
      };
      if constexpr (TM * TN <= 2) {
#pragma unroll 2
        for (int k16 = 0; k16 < K; k16 += 16) group(k16);
      } else {
#pragma unroll 1
        for (int k16 = 0; k16 < K; k16 += 16) group(k16);
      }
      return;
    }
#pragma unroll 2
    for (int k0 = 0; k0 < K; k0 += X::KSTEP) {
      typename X::frag fa[TM], fb[TN];
#pragma unroll
      for (int a = 0; a < TM; ++a) fa[a] = X::load(A, m0(a), k0);
#pragma unroll
      for (int b = 0; b < TN; ++b) fb[b] = X::load(B, n0(b), k0);
#pragma unroll
      for (int a = 0; a < TM; ++a)
#pragma unroll
        for (int b = 0; b < TN; ++b) acc[a][b] = X::mma(fa[a], fb[b], acc[a][b]);
    }
  }

  // Fragments of A (this wave's rows) or B (this wave's columns) for the whole
  // contraction, loaded ahead of the product (e.g. a chunk early).
  template <typename OP, int K>
  struct AFr {
    typename Mma<OP>::frag f[K / Mma<OP>::KSTEP][TM];
    template <class V>
    __device__ __forceinline__ void load(const V& A) {
      if constexpr (sizeof(OP) == 4 && V::kVec) {
#pragma unroll
        for (int g = 0; g < K / 16; ++g)
#pragma unroll
          for (int a = 0; a < TM; ++a) {
            const f32x4 x = Mma<float>::load4(A, m0(a), 16 * g);
#pragma unroll
            for (int t = 0; t < 4; ++t) f[4 * g + t][a] = x[t];
          }
      } else {
#pragma unroll
        for (int s = 0; s < K / Mma<OP>::KSTEP; ++s)
#pragma unroll
          for (int a = 0; a < TM; ++a) f[s][a] = Mma<OP>::load(A, m0(a), s * Mma<OP>::KSTEP);
      }
    }
  };
  template <typename OP, int K>
  struct BFr {
    typename Mma<OP>::frag f[K / Mma<OP>::KSTEP][TN];
    template <class V>
    __device__ __forceinline__ void load(const V& B) {
      if constexpr (sizeof(OP) == 4 && V::kVec) {
#pragma unroll
        for (int g = 0; g < K / 16; ++g)
#pragma unroll
          for (int b = 0; b < TN; ++b) {
            const f32x4 x = Mma<float>::load4(B, n0(b), 16 * g);
#pragma unroll
            for (int t = 0; t < 4; ++t) f[4 * g + t][b] = x[t];
          }
      } else {
#pragma unroll
        for (int s = 0; s < K / Mma<OP>::KSTEP; ++s)
#pragma unroll
          for (int b = 0; b < TN; ++b) f[s][b] = Mma<OP>::load(B, n0(b), s * Mma<OP>::KSTEP);
      }
    }
  };

  // acc += A * B with A's fragments already in registers.
  template <typename OP, int K, class VB>
  __device__ __forceinline__ void mma(const AFr<OP, K>& fa, const VB& B) {
    typedef Mma<OP> X;
    if constexpr (sizeof(OP) == 4 && VB::kVec) {
#pragma unroll
      for (int g = 0; g < K / 16; ++g) {
        f32x4 fb[TN];
#pragma unroll
        for (int b = 0; b < TN; ++b) fb[b] = X::load4(B, n0(b), 16 * g);
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
          for (int a = 0; a < TM; ++a)
#pragma unroll
            for (int b = 0; b < TN; ++b) acc[a][b] = X::mma(fa.f[4 * g + t][a], fb[b][t], acc[a][b]);
      }
      return;
    }
#pragma unroll
    for (int s = 0; s < K / X::KSTEP; ++s) {
      typename X::frag fb[TN];
#pragma unroll
      for (int b = 0; b < TN; ++b) fb[b] = X::load(B, n0(b), s * X::KSTEP);
#pragma unroll
      for (int a = 0; a < TM; ++a)
#pragma unroll
        for (int b = 0; b < TN; ++b) acc[a][b] = X::mma(fa.f[s][a], fb[b], acc[a][b]);
    }
  }
  // acc += A * B with both operands' fragments already in registers.
  template <typename OP, int K>
  __device__ __forceinline__ void mma(const AFr<OP, K>& fa, const BFr<OP, K>& fb) {
    typedef Mma<OP> X;
#pragma unroll
    for (int s = 0; s < K / X::KSTEP; ++s)
#pragma unroll
      for (int a = 0; a < TM; ++a)
#pragma unroll
        for (int b = 0; b < TN; ++b) acc[a][b] = X::mma(fa.f[s][a], fb.f[s][b], acc[a][b]);
  }

  // acc += A * B from raw fragment arrays laid out like AFr / BFr of any
  // Tiles with the same TM / TN ownership.
  template <typename OP, int S>
  __device__ __forceinline__ void mma_raw(const typename Mma<OP>::frag (&fa)[S][TM],
                                          const typename Mma<OP>::frag (&fb)[S][TN]) {
#pragma unroll
    for (int s = 0; s < S; ++s)
#pragma unroll
      for (int a = 0; a < TM; ++a)
#pragma unroll
        for (int b = 0; b < TN; ++b) acc[a][b] = Mma<OP>::mma(fa[s][a], fb[s][b], acc[a][b]);
  }

  // Visit every owned element: f(row, col, value&).
  template <class F>
  __device__ __forceinline__ void each(F f) {
    const int l = lane_id();
#pragma unroll
    for (int a = 0; a < TM; ++a)
#pragma unroll
      for (int b = 0; b < TN; ++b)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          float x = acc[a][b][j];
          f(m0(a) + (l >> 4) * 4 + j, n0(b) + (l & 15), x);
          acc[a][b][j] = x;
        }
  }
};

// ---------------------------------------------------------------------------
// Chunk and sequence coordinates.
// ---------------------------------------------------------------------------
struct ChunkPos {
  int n;     // sequence
  int c;     // chunk index within the sequence
  long row0; // global token row (b*T + t) of the chunk's first token
  int len;   // tokens in this chunk (1..64)
};

__device__ __forceinline__ ChunkPos chunk_pos(const Geo& g, int ci) {
  ChunkPos p;
  if (g.cu == nullptr) {
    p.n = ci / g.NT;
    p.c = ci - p.n * g.NT;
    const int t0 = p.c * CH;
    p.row0 = (long)p.n * g.T + t0;
    p.len = min(CH, g.T - t0);
  } else {
    int lo = 0, hi = g.N;  // find n with chunk_off[n] <= ci < chunk_off[n+1]
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (g.chunk_off[mid] <= ci) lo = mid; else hi = mid;
    }
    // skip empty sequences that share the same offset
    while (lo + 1 < g.N && g.chunk_off[lo + 1] <= ci) ++lo;
    p.n = lo;
    p.c = ci - g.chunk_off[lo];
    const int t0 = g.cu[lo] + p.c * CH;
    p.row0 = t0;
    p.len = min(CH, g.cu[lo + 1] - t0);
  }
  return p;
}

struct SeqPos {
  long row0;  // first token row
  int len;    // tokens
  int c0;     // first chunk (global chunk index)
  int nch;    // chunks
};

__device__ __forceinline__ SeqPos seq_pos(const Geo& g, int n) {
  SeqPos s;
  if (g.cu == nullptr) {
    s.row0 = (long)n * g.T;
    s.len = g.T;
    s.c0 = n * g.NT;
    s.nch = g.NT;
  } else {
    s.row0 = g.cu[n];
    s.len = g.cu[n + 1] - g.cu[n];
    s.c0 = g.chunk_off[n];
    s.nch = g.chunk_off[n + 1] - g.chunk_off[n];
  }
  return s;
}

// Cross-lane sums on the VALU (no LDS traffic).  Every lane of a group ends
// with the same bits: each step adds a pair of partial sums that the two lanes
// of the pair hold in the same order.
template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}
// Sum over the 16 lanes of a row (lanes with equal l >> 4): quad xor 1, quad
// xor 2, half-row mirror, row mirror.
__device__ __forceinline__ float sum16(float x) {
  x += dpp<0xB1>(x);
  x += dpp<0x4E>(x);
  x += dpp<0x141>(x);
  x += dpp<0x140>(x);
  return x;
}
// Sum over the 4 rows (lanes l, l^16, l^32, l^48): swap the wave halves, then
// the odd and even rows (gfx950 v_permlane32_swap / v_permlane16_swap).
__device__ __forceinline__ float sum_groups(float x) {
  const unsigned u = __builtin_bit_cast(unsigned, x);
  const auto a = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  x = __builtin_bit_cast(float, (unsigned)a[0]) + __builtin_bit_cast(float, (unsigned)a[1]);
  const unsigned v = __builtin_bit_cast(unsigned, x);
  const auto b = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  return __builtin_bit_cast(float, (unsigned)b[0]) + __builtin_bit_cast(float, (unsigned)b[1]);
}
// Fixed-order wave reduction.
__device__ __forceinline__ float wave_sum(float x) { return sum_groups(sum16(x)); }

// DPP move with a row mask: rows outside the mask (and lanes without a
// source) receive 0.
template <int CTRL, int ROWS>
__device__ __forceinline__ float dpp_rows(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, ROWS, 0xF, false));
}

// Inclusive prefix sum of one value per lane over a wave, on the VALU: a
// Hillis-Steele scan inside each row of 16 (row shifts by 1, 2, 4, 8), then
// the last lane of row 0 / row 2 added to rows 1 / 3 and the last lane of row
// 1 to rows 2 and 3 (row broadcasts).  The order of additions is fixed, so
// the result is deterministic.
__device__ __forceinline__ float wave_incl_scan(float x) {
  x += dpp_rows<0x111, 0xF>(x);  // row_shr:1
  x += dpp_rows<0x112, 0xF>(x);  // row_shr:2
  x += dpp_rows<0x114, 0xF>(x);  // row_shr:4
  x += dpp_rows<0x118, 0xF>(x);  // row_shr:8
  x += dpp_rows<0x142, 0xA>(x);  // row_bcast:15 into rows 1 and 3
  x += dpp_rows<0x143, 0xC>(x);  // row_bcast:31 into rows 2 and 3
  return x;
}

// Lane l receives lane 63 - l: mirror inside each row of 16, then the row
// order reversed (swap the wave halves, then adjacent rows).
__device__ __forceinline__ float wave_reverse(float x) {
  const int l = lane_id();
  const unsigned u = __builtin_bit_cast(unsigned, dpp<0x140>(x));
  const auto a = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  const unsigned v = (l < 32) ? (unsigned)a[1] : (unsigned)a[0];
  const auto b = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  return __builtin_bit_cast(float, ((l >> 4) & 1) ? (unsigned)b[0] : (unsigned)b[1]);
}

}  // namespace gdn
