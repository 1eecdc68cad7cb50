// Forward of the chunked gated delta rule on gfx950 (paper Sec. 4.2: parallel
// work inside every chunk of 64 tokens, then a short sequential carry between
// chunks).  Two kernels per call:
//
//   prep   one block per (chunk, head): in-chunk cumulative decay G, the erase
//          coupling A = strict_lower(diag(beta) K K^T * exp(G_r - G_i)), the
//          inverse T = (I + A)^{-1}, the two applies W = T diag(beta e^G) K and
//          U = T diag(beta) V, Khat^T with Khat_r = e^{G_last - G_r} k_r, and
//          P = (Q K^T) * D with D_ri = e^{G_r - G_i} for i <= r (exponent formed
//          only there), all laid out for direct MFMA fragment loads.
//   scan   one block per (stream, value tile of BV columns): chunk by chunk,
//            U' = U - W h,   O = diag(e^G) Q h + P U',   h <- e^{G_last} h + Khat^T U',
//          writing every h (the saved chunk states), the output tile and S_T.
//          The carry splits over value columns with no communication.
#pragma once

#include <type_traits>

#include "gdn_chunk.hpp"
#include "gdn_exact.hpp"
#include "gdn_launch.hpp"

namespace gdn {

template <int DK, int DV, typename OP, int VAR>
__global__ __launch_bounds__(512) void k_prep_fwd(Geo geo, int H, const OP* __restrict__ q,
                                                  const OP* __restrict__ k, const OP* __restrict__ v,
                                                  const float* __restrict__ g, const float* __restrict__ beta,
                                                  float* __restrict__ gcum, OP* __restrict__ Wg,
                                                  OP* __restrict__ Ug, OP* __restrict__ KhTg,
                                                  OP* __restrict__ Pg, OP* __restrict__ Qgg, int* __restrict__ flag) {
  constexpr bool DT_ = VAR != VAR_DECAY;
  // bf16 operands read transposed tiles straight from row-major LDS with the
  // transposing load; fp32 operands go through explicit transposed copies
  constexpr bool TR = sizeof(OP) == 2;
  constexpr int LK = DK + pad_of<OP>();
  constexpr int LV = DV + pad_of<OP>();
  constexpr int LC = CH + 4;
  constexpr int LT = CH + pad_of<OP>();
  constexpr int VS = TR ? DV : 64;  // value columns per slice of U
  constexpr int VE = 16 / (int)sizeof(OP);
  typedef typename vec4_of<OP>::type V4;
  // LDS regions reused by lifetime (two blocks per CU):
  //   R1: Q, then T in fp32;  R2: K (bf16: alive through W; fp32: then T);
  //   R3: bf16: T in bf16; fp32: (diag(beta e^G) K)^T;
  //   R4: A in fp32, then diag(beta) V (bf16: row-major; fp32: transposed slices).
  constexpr int R1 = CH * LK * (int)sizeof(OP) > CH * LC * 4 ? CH * LK * (int)sizeof(OP) : CH * LC * 4;
  constexpr int R2 = CH * LK * (int)sizeof(OP);
  constexpr int R3 = !DT_ ? 16 : (TR ? CH * LT * (int)sizeof(OP) : DK * LT * (int)sizeof(OP));
  constexpr int VB = TR ? CH * LV * (int)sizeof(OP) : VS * LT * (int)sizeof(OP);
  constexpr int R4 = CH * LC * 4 > VB ? CH * LC * 4 : VB;
  static_assert(TR || CH * LT * (int)sizeof(OP) <= R2, "T fits where K was");
  __shared__ __align__(16) char r1[R1];
  __shared__ __align__(16) char r2[R2];
  __shared__ __align__(16) char r3[R3];
  __shared__ __align__(16) char r4[R4];
  __shared__ __align__(16) float Gs[CH], Bs[CH], Gam[CH], Dte[CH], BG[CH];
  OP* Qs = reinterpret_cast<OP*>(r1);
  float* Tf = reinterpret_cast<float*>(r1);
  OP* Ks = reinterpret_cast<OP*>(r2);
  OP* Ts = TR ? reinterpret_cast<OP*>(r3) : reinterpret_cast<OP*>(r2);
  OP* KbT = reinterpret_cast<OP*>(r3);
  float* As = reinterpret_cast<float*>(r4);
  OP* Vb = reinterpret_cast<OP*>(r4);

  const int ci = blockIdx.x, h = blockIdx.y;
  const ChunkPos cp = chunk_pos(geo, ci);
  const long tile = (long)ci * H + h;
  const int l = lane_id(), w = wave_id();
  // every input row of the block is requested up front: q, k, then the v
  // slices of the U product (slice t of VS columns is piece t of each thread)
  RowsIn<DK, 512, OP> qin, kin;
  qin.load(q + (cp.row0 * H + h) * DK, (long)H * DK, cp.len);
  kin.load(k + (cp.row0 * H + h) * DK, (long)H * DK, cp.len);
  const OP* vp = v + (cp.row0 * H + h) * DV;
  constexpr int NSL = DV / VS, NPS = CH * VS / VE / 512;  // slices; pieces per thread and slice
  uint4 vin[NSL][NPS];
#pragma unroll
  for (int t = 0; t < NSL; ++t)
#pragma unroll
    for (int p = 0; p < NPS; ++p) {
      const int idx = threadIdx.x + p * 512, i = idx / (VS / VE), c = t * VS + (idx % (VS / VE)) * VE;
      vin[t][p] = *reinterpret_cast<const uint4*>(vp + (long)clamp_row(i, cp.len) * H * DV + c);
    }
  bool ok = load_gates<VAR>(g, beta, cp.row0, H, h, cp.len, Gs, Bs);
  ok &= qin.template stage<LK>(Qs, cp.len);
  ok &= kin.template stage<LK>(Ks, cp.len);
  __syncthreads();
  if (threadIdx.x < CH) {
    const int r = threadIdx.x;
    gcum[tile * CH + r] = Gs[r];
    const float gam = __expf(Gs[r]);
    Gam[r] = gam;
    BG[r] = Bs[r] * gam;
    Dte[r] = __expf(Gs[CH - 1] - Gs[r]);
  }
  __syncthreads();
  // diag(e^G) Q, the A operand of the output term of the generic scan (the
  // split bf16 scan reads q itself): thread order follows the operand layout,
  // so each wave writes whole 1 KiB fragments
  if constexpr (!(TR && DT_)) {
    OP* Qg = Qgg + tile * CH * DK;
    for (int idx = threadIdx.x; idx < CH * DK / VE; idx += blockDim.x) {
      int r, d0;
      if constexpr (TR) {
        const int f = idx >> 6, ll = idx & 63;
        r = (f / (DK / 32)) * 16 + (ll & 15);
        d0 = (f % (DK / 32)) * 32 + (ll >> 4) * 8;
      } else {
        r = idx / (DK / VE);
        d0 = (idx - r * (DK / VE)) * VE;
      }
      const uint4 qv = *reinterpret_cast<const uint4*>(Qs + r * LK + d0);
      OP vals[VE];
#pragma unroll
      for (int j = 0; j < VE; ++j) vals[j] = from_f<OP>(Gam[r] * to_f(elem16<OP>(qv, j)));
      *reinterpret_cast<uint4*>(Qg + op_off<OP, DK>(r, d0)) = pack16<OP>(vals);
    }
  }
  // P[r][i] = (q_r . k_i) e^{G_r - G_i} (i <= r): computed as K Q^T so that a
  // lane's four accumulator rows are four consecutive i of one row r of P
  {
    Tiles<CH, CH, 4, 2> s;
    s.zero();
    s.template mma<OP, DK>(KRow<OP, LK>{Ks}, KRow<OP, LK>{Qs});
    OP* Pt = Pg + tile * CH * CH;
#pragma unroll
    for (int b = 0; b < s.TN; ++b) {
      const int r = s.n0(b) + (l & 15), i0 = s.m0(0) + (l >> 4) * 4;
      OP v4[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int i = i0 + j;
        v4[j] = from_f<OP>(i <= r ? s.acc[0][b][j] * __expf(Gs[r] - Gs[i]) : 0.f);
      }
      *reinterpret_cast<V4*>(Pt + op_off<OP, CH>(r, i0)) = pack4<OP>(v4);
    }
  }
  if constexpr (DT_) {
    Tiles<CH, CH, 4, 2> bm;
    bm.zero();
    bm.template mma<OP, DK>(KRow<OP, LK>{Ks}, KRow<OP, LK>{Ks});
    bm.each([&](int r, int i, float& x) {
      As[r * LC + i] = (i < r) ? Bs[r] * x * __expf(Gs[r] - Gs[i]) : 0.f;
    });
    if constexpr (!TR) {
      // (diag(beta e^G) K)^T for the W product
      for (int idx = threadIdx.x; idx < CH * DK / VE; idx += blockDim.x) {
        const int i = idx / (DK / VE), d0 = (idx - i * (DK / VE)) * VE;
        const uint4 kv = *reinterpret_cast<const uint4*>(Ks + i * LK + d0);
        const float sc = BG[i];
#pragma unroll
        for (int j = 0; j < VE; ++j) KbT[(d0 + j) * LT + i] = from_f<OP>(sc * to_f(elem16<OP>(kv, j)));
      }
    }
  }
  // Khat^T[d][r] = e^{G_last - G_r} k_r[d], the scan's A operand for the carry
  {
    OP* Kh = KhTg + tile * DK * CH;
    if constexpr (TR) {
      // one transposed fragment (16 d x 32 r) of K per wave and step, stored
      // as one contiguous 1 KiB block
#pragma unroll
      for (int t = 0; t < DK * CH / (512 * 8); ++t) {
        const int f = w + 8 * t, mt = f / (CH / 32), s = f % (CH / 32);
        const bf16x8 x = scale_frag(lds_frag_tr<LK>(Ks, 16 * mt, 32 * s), Dte, 32 * s);
        *reinterpret_cast<bf16x8*>(Kh + ((long)f * 64 + l) * 8) = x;
      }
    } else {
      for (int idx = threadIdx.x; idx < DK * CH / VE; idx += blockDim.x) {
        const int d = idx / (CH / VE), r0 = (idx - d * (CH / VE)) * VE;
        OP vals[VE];
#pragma unroll
        for (int j = 0; j < VE; ++j) vals[j] = from_f<OP>(Dte[r0 + j] * to_f(Ks[(r0 + j) * LK + d]));
        *reinterpret_cast<uint4*>(Kh + op_off<OP, CH>(d, r0)) = pack16<OP>(vals);
      }
    }
  }
  __syncthreads();  // Q (and for fp32 K) is dead from here on
  if constexpr (DT_) {
    unit_lower_inverse<OP, LC, LT, false>(As, Tf, Ts, (OP*)nullptr);
    const OP* Tp;
    if constexpr (TR) Tp = Ts; else Tp = reinterpret_cast<const OP*>(Tf);
    constexpr int LTT = TR ? LT : LC;
    if constexpr (TR) {
      // A is dead: stage diag(beta) V row-major for the U product
#pragma unroll
      for (int p = 0; p < NPS; ++p) {
        const int idx = threadIdx.x + p * 512, i = idx / (DV / VE), c = (idx % (DV / VE)) * VE;
        const uint4 vv = keep16(i < cp.len, vin[0][p]);
        ok &= finite16B<OP>(vv);
        OP vals[VE];
#pragma unroll
        for (int j = 0; j < VE; ++j) vals[j] = from_f<OP>(Bs[i] * to_f(elem16<OP>(vv, j)));
        *reinterpret_cast<uint4*>(Vb + i * LV + c) = pack16<OP>(vals);
      }
    }
    // W = T diag(beta e^G) K, computed as W^T = Kb^T T^T so a lane holds four
    // consecutive d of one row r of W
    {
      Tiles<DK, CH, 4, 2> wt;
      wt.zero();
      if constexpr (TR)
        wt.template mma<OP, CH>(KColTr<LK, true>{Ks, BG}, KRow<OP, LT>{Tp});
      else
        wt.template mma<OP, CH>(KRow<OP, LT>{KbT}, KRow<OP, LTT>{Tp});
      OP* Wt = Wg + tile * CH * DK;
#pragma unroll
      for (int a = 0; a < wt.TM; ++a)
#pragma unroll
        for (int b = 0; b < wt.TN; ++b) {
          const int r = wt.n0(b) + (l & 15), d0 = wt.m0(a) + (l >> 4) * 4;
          OP v4[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) v4[j] = from_f<OP>(wt.acc[a][b][j]);
          *reinterpret_cast<V4*>(Wt + op_off<OP, DK>(r, d0)) = pack4<OP>(v4);
        }
    }
    // U = T diag(beta) V, per slice of VS value columns, stored in the operand
    // dtype as the scan's accumulator tiles (four rows of one column per lane)
    OP* Ut = Ug + tile * CH * DV;
#pragma unroll
    for (int t = 0; t < NSL; ++t) {
      const int c0 = t * VS;
      if constexpr (!TR) {
#pragma unroll
        for (int p = 0; p < NPS; ++p) {
          const int idx = threadIdx.x + p * 512, i = idx / (VS / VE), v0 = (idx % (VS / VE)) * VE;
          const uint4 vv = keep16(i < cp.len, vin[t][p]);
          ok &= finite16B<OP>(vv);
#pragma unroll
          for (int j = 0; j < VE; ++j) Vb[(v0 + j) * LT + i] = from_f<OP>(Bs[i] * to_f(elem16<OP>(vv, j)));
        }
      }
      __syncthreads();
      Tiles<CH, VS, 4, 2> uu;
      uu.zero();
      if constexpr (TR)
        uu.template mma<OP, CH>(KRow<OP, LT>{Tp}, KColTr<LV>{Vb, nullptr});
      else
        uu.template mma<OP, CH>(KRow<OP, LTT>{Tp}, KRow<OP, LT>{Vb});
#pragma unroll
      for (int b = 0; b < uu.TN; ++b) {
        const int r0 = uu.m0(0) + (l >> 4) * 4, vcol = c0 + uu.n0(b) + (l & 15);
        OP u4[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) u4[j] = from_f<OP>(uu.acc[0][b][j]);
        *reinterpret_cast<V4*>(Ut + cfrag_off<SCAN_BV>(r0, vcol)) = pack4<OP>(u4);
      }
      if (t + 1 < NSL) __syncthreads();
    }
  } else {
    // scalar-decay member: T = I, W = 0, U = V; only check v for non-finite values
#pragma unroll
    for (int t = 0; t < NSL; ++t)
#pragma unroll
      for (int p = 0; p < NPS; ++p) ok &= finite16B<OP>(keep16((threadIdx.x + p * 512) / (VS / VE) < cp.len, vin[t][p]));
  }
  const int bad = __syncthreads_or(!ok);
  if (threadIdx.x == 0) flag[tile] = bad;
}

// The forward inter-chunk scan with the chunk output fused in.  Every operand
// except the carry arrives pre-laid-out (W, P row-major, Khat^T, U in fp32, q
// straight from the input), so the A fragments of chunk c+1 load from HBM/L2
// into registers while chunk c is computed; only h and U' pass through LDS
// (two barriers per chunk).
// CWD (channel-wise decay): the carry decays row by row, h[d, :] *= e^{G_last[d]},
// with gcum holding each chunk's d_k values of G_last instead of the 64 in-chunk
// values of a scalar G.  OUT: the element type of o (the operand type by default).
template <int DK, int DV, int BV, typename OP, int VAR, bool CWD = false, typename OUT = OP>
__global__ __launch_bounds__(256) void k_scan_fwd(Geo geo, int H, const OP* __restrict__ Qgg,
                                                  const OP* __restrict__ v, const float* __restrict__ S0,
                                                  const float* __restrict__ gcum, const OP* __restrict__ Wg,
                                                  const OP* __restrict__ KhTg, const OP* __restrict__ Pg,
                                                  const OP* __restrict__ Ug, float* __restrict__ states,
                                                  float* __restrict__ ST, OUT* __restrict__ o,
                                                  int* __restrict__ flag) {
  static_assert(BV == SCAN_BV, "U is laid out for the scan's value tiles");
  constexpr int NVT = DV / BV;
  constexpr int LK = DK + pad_of<OP>();
  constexpr int LU = CH + pad_of<OP>();
  constexpr int LF = BV + 4;            // row stride of the fp32 state staging
  constexpr bool PF = sizeof(OP) == 2;  // prefetch a chunk ahead (bf16 fragments are compact)
  typedef Tiles<DK, BV, 4, 1> HT;       // carried state slice h[:, v0:v0+BV]
  typedef Tiles<CH, BV, 4, 1> UT;       // U' and output slices
  __shared__ __align__(16) OP hT[BV * LK];
  __shared__ __align__(16) float hF[DK * LF];  // h in fp32, row-major, for whole-line state stores
  __shared__ __align__(16) OP UsT[BV * LU];

  int s, vt;
  scan_block_coords(blockIdx.x, geo.N * H, NVT, s, vt);
  const int n = s / H, h = s - (s / H) * H, v0 = vt * BV;
  const SeqPos sp = seq_pos(geo, n);
  const int l = lane_id();

  struct Pre {
    typename UT::template AFr<OP, DK> w;
    typename UT::template AFr<OP, DK> qf;
    typename UT::template AFr<OP, CH> pf;
    typename HT::template AFr<OP, CH> kh;
    typename vec4_of<OP>::type u[UT::TN];  // U (or V): four rows of one column per lane
    float gl;  // G_last, exponentiated at use so the prefetch never waits
    float gd[CWD ? HT::TM : 1][4];  // CWD: G_last of this lane's state rows
  };
  // A fragments of a pre-arranged operand (fragment-major for bf16, row-major for fp32)
  auto frags = [&](auto& f, const OP* base, auto tiles_tag, auto k_tag) {
    typedef decltype(tiles_tag) TT;
    constexpr int K = decltype(k_tag)::value;
    if constexpr (sizeof(OP) == 2) {
#pragma unroll
      for (int st = 0; st < K / 32; ++st)
#pragma unroll
        for (int a = 0; a < TT::TM; ++a)
          f.f[st][a] = *reinterpret_cast<const bf16x8*>(base + ((long)((TT::m0(a) >> 4) * (K / 32) + st) * 64 + l) * 8);
    } else {
      f.load(KRow<OP, K>{base});
    }
  };
  auto load_pre = [&](Pre& p, int c) {
    const long tile = (long)(sp.c0 + c) * H + h;
    const long row0 = sp.row0 + (long)c * CH;
    const int len = min(CH, sp.len - c * CH);
    if constexpr (VAR != VAR_DECAY) {
      frags(p.w, Wg + tile * CH * DK, UT{}, std::integral_constant<int, DK>{});
      const OP* Ut = Ug + tile * CH * DV;
#pragma unroll
      for (int b = 0; b < UT::TN; ++b)
        p.u[b] = *reinterpret_cast<const typename vec4_of<OP>::type*>(
            Ut + cfrag_off<BV>(UT::m0(0) + (l >> 4) * 4, v0 + UT::n0(b) + (l & 15)));
    } else {
      const OP* vp = v + (row0 * H + h) * DV + v0;
#pragma unroll
      for (int b = 0; b < UT::TN; ++b) {
        OP x4[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int r = UT::m0(0) + (l >> 4) * 4 + j;
          // U' = V here; its rows past the chunk's end meet only zero columns of
          // Khat^T and P, so the last valid row may stand in for them
          x4[j] = vp[(long)clamp_row(r, len) * H * DV + UT::n0(b) + (l & 15)];
        }
        p.u[b] = pack4<OP>(x4);
      }
    }
    frags(p.qf, Qgg + tile * CH * DK, UT{}, std::integral_constant<int, DK>{});
    frags(p.pf, Pg + tile * CH * CH, UT{}, std::integral_constant<int, CH>{});
    frags(p.kh, KhTg + tile * DK * CH, HT{}, std::integral_constant<int, CH>{});
    if constexpr (CWD) {
#pragma unroll
      for (int a = 0; a < HT::TM; ++a)
#pragma unroll
        for (int j = 0; j < 4; ++j) p.gd[a][j] = gcum[tile * DK + HT::m0(a) + (l >> 4) * 4 + j];
    } else {
      p.gl = gcum[tile * CH + CH - 1 + opaque_zero()];  // vector load: see opaque_zero
    }
  };

  HT hs;
  bool ok = true;
  const float* S0p = S0 ? S0 + ((long)n * H + h) * DK * DV : nullptr;
  hs.each([&](int d, int vv, float& x) {
    x = S0p ? S0p[d * DV + v0 + vv] : 0.f;
    ok &= finite_f(x);
  });

  // One chunk of the carry.  `prefetch` issues the loads of the next chunk
  // right after the barrier that opens this one; the two fragment buffers
  // alternate, so nothing is copied and no wait on the new loads is needed.
  auto step = [&](int c, const Pre& cur, auto&& prefetch) {
    const long tile = (long)(sp.c0 + c) * H + h;
    const long row0 = sp.row0 + (long)c * CH;
    const int len = min(CH, sp.len - c * CH);
    // h to LDS: operand copy (4 consecutive d per lane: one 8-byte write) and
    // fp32 row-major copy for the state store
#pragma unroll
    for (int a = 0; a < HT::TM; ++a)
#pragma unroll
      for (int b = 0; b < HT::TN; ++b) {
        const int d0 = HT::m0(a) + (l >> 4) * 4, vv = HT::n0(b) + (l & 15);
        OP h4[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          h4[j] = from_f<OP>(hs.acc[a][b][j]);
          hF[(d0 + j) * LF + vv] = hs.acc[a][b][j];
        }
        *reinterpret_cast<typename vec4_of<OP>::type*>(hT + vv * LK + d0) = pack4<OP>(h4);
      }
    __syncthreads();
    prefetch();
    {
      // the chunk state leaves as whole 128-byte rows (BV fp32 of one d)
      float* hp = states + tile * DK * DV + v0;
#pragma unroll
      for (int t = 0; t < DK * BV / 4 / 256; ++t) {
        const int idx = threadIdx.x + t * 256, d = idx / (BV / 4), c4 = (idx - d * (BV / 4)) * 4;
        *reinterpret_cast<float4*>(hp + (long)d * DV + c4) = *reinterpret_cast<const float4*>(hF + d * LF + c4);
      }
    }
    UT up, ot;
    ot.zero();
    ot.template mma<OP, DK>(cur.qf, KRow<OP, LK>{hT});  // diag(e^G) Q h
    if constexpr (VAR != VAR_DECAY) {
      up.zero();
      up.template mma<OP, DK>(cur.w, KRow<OP, LK>{hT});
#pragma unroll
      for (int b = 0; b < UT::TN; ++b)
#pragma unroll
        for (int j = 0; j < 4; ++j) up.acc[0][b][j] = to_f(elem4<OP>(cur.u[b], j)) - up.acc[0][b][j];
    } else {
#pragma unroll
      for (int b = 0; b < UT::TN; ++b)
#pragma unroll
        for (int j = 0; j < 4; ++j) up.acc[0][b][j] = to_f(elem4<OP>(cur.u[b], j));
    }
#pragma unroll
    for (int b = 0; b < UT::TN; ++b) {
      const int vv = UT::n0(b) + (l & 15), r0 = UT::m0(0) + (l >> 4) * 4;
      OP u4[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) u4[j] = from_f<OP>(up.acc[0][b][j]);
      *reinterpret_cast<typename vec4_of<OP>::type*>(UsT + vv * LU + r0) = pack4<OP>(u4);
    }
    __syncthreads();
    if constexpr (CWD) {
#pragma unroll
      for (int a = 0; a < HT::TM; ++a)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float gd = __expf(cur.gd[a][j]);
#pragma unroll
          for (int b = 0; b < HT::TN; ++b) hs.acc[a][b][j] *= gd;
        }
    } else {
      const float gl = __expf(cur.gl);
      hs.each([&](int, int, float& x) { x *= gl; });
    }
    hs.template mma<OP, CH>(cur.kh, KRow<OP, LU>{UsT});
    ot.template mma<OP, CH>(cur.pf, KRow<OP, LU>{UsT});  // + P U'
    OUT* op = o + (row0 * H + h) * DV + v0;
#pragma unroll
    for (int b = 0; b < UT::TN; ++b)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = UT::m0(0) + (l >> 4) * 4 + j;
        if (r < len) op[(long)r * H * DV + UT::n0(b) + (l & 15)] = from_f<OUT>(ot.acc[0][b][j]);
      }
  };
  const int nch = sp.nch;
  if constexpr (PF) {
    // The prefetch always issues (past the last chunk it re-reads that chunk):
    // a conditional prefetch would leave one path with fewer memory operations
    // in flight, and the wait counts, merged over both paths, would then wait
    // for the loads just issued.
    if (nch > 0) {
      Pre p0, p1;
      load_pre(p0, 0);
      for (int c = 0; c < nch; c += 2) {
        step(c, p0, [&] { load_pre(p1, min(c + 1, nch - 1)); });
        if (c + 1 < nch) step(c + 1, p1, [&] { load_pre(p0, min(c + 2, nch - 1)); });
      }
    }
  } else {
    Pre cur;
    for (int c = 0; c < nch; ++c) {
      load_pre(cur, c);
      step(c, cur, [] {});
    }
  }
  float* STp = ST + ((long)n * H + h) * DK * DV;
  hs.each([&](int d, int vv, float& x) { STp[d * DV + v0 + vv] = x; });
  const int bad = __syncthreads_or(!ok);
  if (threadIdx.x == 0) flag[(long)s * NVT + vt] = bad;
}

// The forward scan for bf16 operands of the delta-rule members, split into
// four chain waves and four copy waves.  Everything the chain reads per chunk
// except the carry (W, Q, P, Khat^T, this block's slice of U and the chunk's
// G) goes through LDS in 1 KiB blocks: the prep kernel's outputs are stored
// as MFMA fragment blocks in HBM, and q's token-major rows (the contraction
// index d_k is contiguous there) are gathered a line at a time (RowLines).
// The copy waves move the
// next chunk's 60 KiB straight into one of two LDS buffers with
// global_load_lds_dwordx4 and write the chunk state out of LDS, so the chain
// waves never queue behind the address unit.  Per chunk:
//   chain: h -> LDS | barrier | U' = U - W h, O = Q h | barrier |
//          O <- diag(e^G) O, h <- e^{G_last} h + Khat^T U', O += P U', store O
//   copy:             | next chunk's operands -> LDS, state -> HBM | | wait
template <int DK, int DV, int BV, int VAR>
__global__ __launch_bounds__(512) void k_scan_fwd_ws(Geo geo, int H, const bf16* __restrict__ q,
                                                     const float* __restrict__ S0, const float* __restrict__ gcum,
                                                     const bf16* __restrict__ Wg, const bf16* __restrict__ KhTg,
                                                     const bf16* __restrict__ Pg, const bf16* __restrict__ Ug,
                                                     float* __restrict__ states, float* __restrict__ ST,
                                                     bf16* __restrict__ o, int* __restrict__ flag) {
  static_assert(BV == SCAN_BV && VAR != VAR_DECAY, "U is laid out for the scan's value tiles");
  typedef RowLines<DK> QL;
  static_assert(QL::NBLK == (CH / 16) * (DK / 32), "q takes the blocks of a 64 x DK fragment operand");
  constexpr int NVT = DV / BV;
  constexpr int LK = DK + 8, LU = CH + 8, LF = BV + 4;
  typedef Tiles<DK, BV, 4, 1> HT;  // carried state slice h[:, v0:v0+BV] (chain waves)
  typedef Tiles<CH, BV, 4, 1> UT;  // U' and output slices (chain waves)
  // one operand buffer: fragment blocks of 1 KiB (64 lanes x 16 B) in HBM order
  constexpr int NW = (CH / 16) * (DK / 32), NP = (CH / 16) * (CH / 32), NK = (DK / 16) * (CH / 32);
  constexpr int NU = CH * BV * 2 / 1024;
  constexpr int OW = 0, OQ = OW + NW, OP_ = OQ + NW, OK = OP_ + NP, OU = OK + NK, NB = OU + NU;
  constexpr int BUF = NB * 1024 + CH * 4;  // + the chunk's G (64 fp32)
  __shared__ __align__(1024) char buf[2][BUF];
  __shared__ __align__(16) bf16 hT[BV * LK];
  __shared__ __align__(16) float hF[DK * LF];  // h in fp32, row-major, for whole-line state stores
  __shared__ __align__(16) bf16 UsT[BV * LU];
  __shared__ __align__(16) bf16 OsT[BV * LU];  // the chunk output, transposed (v, r), for the copy waves
  __shared__ __align__(16) char sink[256];  // target of the L2 warm-up loads (never read)

  int s, vt;
  scan_block_coords(blockIdx.x, geo.N * H, NVT, s, vt);
  const int n = s / H, h = s - (s / H) * H, v0 = vt * BV;
  const SeqPos sp = seq_pos(geo, n);
  const int w = wave_id(), l = lane_id();
  const bool chain = w < 4;  // waves 0-3: the carry; waves 4-7: copies
  const int nch = sp.nch;

  // copy waves: chunk c's operands into buffer b (block j of the list goes to
  // buf[b] + j KiB; the copy wave w - 4 takes every fourth block)
  typedef __attribute__((address_space(1))) void gvoid;
  typedef __attribute__((address_space(3))) void lvoid;
  // row r of q in chunk c (rows past the chunk's end repeat its last row:
  // they reach only output rows that are never stored)
  auto q_row = [&](int c, int r) __attribute__((always_inline)) -> const bf16* {
    const int len = min(CH, sp.len - c * CH);
    return q + ((sp.row0 + (long)c * CH + clamp_row(r, len)) * H + h) * DK;
  };
  // block j0 + (w - 4): the region bounds are multiples of 4, so the unrolled
  // j0 alone selects the region
  static_assert(OQ % 4 == 0 && OP_ % 4 == 0 && OK % 4 == 0 && OU % 4 == 0 && NB % 4 == 0, "region bounds");
  auto copy_block = [&](int c, int j0, int b) __attribute__((always_inline)) {
    const long tile = (long)(sp.c0 + c) * H + h;
    const int j = j0 + (w - 4);
    const bf16* src;
    if (j0 < OQ) src = Wg + tile * CH * DK + (j - OW) * 512 + l * 8;
    else if (j0 < OP_) {
      int r, e;
      QL::src(j - OQ, l, r, e);
      src = q_row(c, r) + e;
    }
    else if (j0 < OK) src = Pg + tile * CH * CH + (j - OP_) * 512 + l * 8;
    else if (j0 < OU) src = KhTg + tile * DK * CH + (j - OK) * 512 + l * 8;
    else src = Ug + tile * CH * DV + (long)vt * CH * BV + (j - OU) * 512 + l * 8;
    __builtin_amdgcn_global_load_lds((gvoid*)src, (lvoid*)(buf[b] + j * 1024), 16, 0, 0);
  };
  // The chain reads W, Q and U only before its second barrier and P, Khat^T
  // and G after it, so a buffer's W/Q/U region is free half a chunk before
  // the rest: "early" fills (W, Q, U) of chunk c + 2 go out right after the
  // chain's second barrier of chunk c, "late" fills (P, Khat^T, G) of chunk
  // c + 1 after its first barrier of chunk c.  Every copy wave issues the same
  // number of each (static: the waits below count them).
  static_assert(NU == 4, "one U block per copy wave");
  constexpr int NE = OP_ / 4 + 1;  // early fills per copy wave
  auto fill_early = [&](int c, int b) __attribute__((always_inline)) {
#pragma unroll
    for (int j0 = 0; j0 < OP_; j0 += 4) copy_block(c, j0, b);
    copy_block(c, OU, b);
  };
  auto fill_late = [&](int c, int b) __attribute__((always_inline)) {
#pragma unroll
    for (int j0 = OP_; j0 < OU; j0 += 4) copy_block(c, j0, b);
    if (w == 4) {
      const long tile = (long)(sp.c0 + c) * H + h;
      __builtin_amdgcn_global_load_lds((gvoid*)(gcum + tile * CH + l), (lvoid*)(buf[b] + NB * 1024), 4, 0, 0);
    }
  };
  // the copy waves' loads landed: their state stores, issued after them, may
  // stay in flight (vmcnt counts in issue order on gfx9)
  constexpr int NST = DK * BV / 4 / 256;  // state stores per copy-wave lane and chunk
  static_assert(NST < 16, "vmcnt field");
  // L2 warm-up two chunks ahead: the NVT blocks of a stream split the
  // chunk's W, Q, P and Khat^T blocks (one in NVT each) and each warms its
  // own U slice, touching every 128-byte line once: one 4-byte load per lane
  // (64 lines per instruction), so the warm-up costs the address unit little.
  constexpr int NSH = (OU + NVT - 1) / NVT;          // shared blocks warmed per block
  constexpr int NWL = (NSH + NU) * 8;                 // lines warmed per block
  constexpr int NWARM = (NWL + 255) / 256;            // loads per copy-wave lane
  auto warm = [&](int c) {
    const long tile = (long)(sp.c0 + c) * H + h;
#pragma unroll
    for (int t = 0; t < NWARM; ++t) {
      int L = ((w - 4) + 4 * t) * 64 + l;
      L = L < NWL ? L : NWL - 1;
      const int e = L >> 3;
      int j = e < NSH ? e * NVT + vt : OU + (e - NSH);
      j = j < NB ? j : NB - 1;
      const bf16* src;
      if (j < OQ) src = Wg + tile * CH * DK + (j - OW) * 512 + (L & 7) * 64;
      else if (j < OP_) {
        // line (L & 7) of q block j - OQ
        int r, e;
        QL::src(j - OQ, (L & 7) << 3, r, e);
        src = q_row(c, r) + (e & ~63);
      }
      else if (j < OK) src = Pg + tile * CH * CH + (j - OP_) * 512 + (L & 7) * 64;
      else if (j < OU) src = KhTg + tile * DK * CH + (j - OK) * 512 + (L & 7) * 64;
      else src = Ug + tile * CH * DV + (long)vt * CH * BV + (j - OU) * 512 + (L & 7) * 64;
      __builtin_amdgcn_global_load_lds((gvoid*)src, (lvoid*)sink, 4, 0, 0);
    }
  };
  static_assert(NWARM + NST + NE < 16, "vmcnt field");
  // vmcnt(NWARM + NST + NE): everything up to the late fills of the next chunk landed
  auto copies_done = [] { __builtin_amdgcn_s_waitcnt(0x0F70 | (NWARM + NST + NE)); };
  // A workgroup barrier that waits for this wave's LDS operations only.  Each
  // wave's global loads into LDS are waited for by that wave (copies_done);
  // a full __syncthreads would also wait for every store still in flight.
  auto lds_barrier = [] { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); };

  HT hs;
  bool ok = true;
  if (chain) {
    const float* S0p = S0 ? S0 + ((long)n * H + h) * DK * DV : nullptr;
    hs.each([&](int d, int vv, float& x) {
      x = S0p ? S0p[d * DV + v0 + vv] : 0.f;
      ok &= finite_f(x);
    });
    lds_barrier();
    // The chain and the copy waves run separate loops with the same barrier
    // sequence (two per chunk), so neither waits for the other's memory
    // operations at a barrier.
    for (int c = 0; c < nch; ++c) {
      const char* B = buf[c & 1];
      // h to LDS: operand copy (4 consecutive d per lane: one 8-byte write) and
      // fp32 row-major copy for the state store
#pragma unroll
      for (int a = 0; a < HT::TM; ++a)
#pragma unroll
        for (int bb = 0; bb < HT::TN; ++bb) {
          const int d0 = HT::m0(a) + (l >> 4) * 4, vv = HT::n0(bb) + (l & 15);
          bf16 h4[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            h4[j] = from_f<bf16>(hs.acc[a][bb][j]);
            hF[(d0 + j) * LF + vv] = hs.acc[a][bb][j];
          }
          *reinterpret_cast<uint2*>(hT + vv * LK + d0) = pack4<bf16>(h4);
        }
      lds_barrier();  // A: h in LDS, this chunk's operands in buffer c & 1
      // U' = U - W h and O = Q h; A fragments of wave w are 16-row tile w.
      // The row scales e^{G_r} of O are formed here, under the products.
      const float* Gc = reinterpret_cast<const float*>(B + NB * 1024);
      float gam[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) gam[j] = __expf(Gc[UT::m0(0) + (l >> 4) * 4 + j]);
      UT up, ot;
      const bf16x8* Wf = reinterpret_cast<const bf16x8*>(B + OW * 1024);
      const bf16x8* Qf = reinterpret_cast<const bf16x8*>(B + OQ * 1024);
      ot.zero();
      up.zero();
#pragma unroll
      for (int st = 0; st < DK / 32; ++st) {
        const bf16x8 fq = Qf[QL::frag_slot(w, st, l)];
        const bf16x8 fw = Wf[(w * (DK / 32) + st) * 64 + l];
#pragma unroll
        for (int bb = 0; bb < UT::TN; ++bb) {
          const bf16x8 fh = Mma<bf16>::load(KRow<bf16, LK>{hT}, UT::n0(bb), 32 * st);
          ot.acc[0][bb] = Mma<bf16>::mma(fq, fh, ot.acc[0][bb]);
          up.acc[0][bb] = Mma<bf16>::mma(fw, fh, up.acc[0][bb]);
        }
      }
      const uint2* Uf = reinterpret_cast<const uint2*>(B + OU * 1024);
#pragma unroll
      for (int bb = 0; bb < UT::TN; ++bb) {
        const uint2 u = Uf[(w * UT::TN + bb) * 64 + l];
        const int vv = UT::n0(bb) + (l & 15), r0 = UT::m0(0) + (l >> 4) * 4;
        bf16 u4[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          up.acc[0][bb][j] = to_f(elem4<bf16>(u, j)) - up.acc[0][bb][j];
          u4[j] = from_f<bf16>(up.acc[0][bb][j]);
        }
        *reinterpret_cast<uint2*>(UsT + vv * LU + r0) = pack4<bf16>(u4);
      }
      lds_barrier();  // B: U' in LDS
      const float gl = __expf(Gc[CH - 1]);
      hs.each([&](int, int, float& x) { x *= gl; });
      // O = diag(e^G) Q h: the row scale applied to the fp32 products
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int bb = 0; bb < UT::TN; ++bb) ot.acc[0][bb][j] *= gam[j];
      const bf16x8* Kf = reinterpret_cast<const bf16x8*>(B + OK * 1024);
      const bf16x8* Pf = reinterpret_cast<const bf16x8*>(B + OP_ * 1024);
#pragma unroll
      for (int st = 0; st < CH / 32; ++st) {
        bf16x8 fk[HT::TM];
#pragma unroll
        for (int a = 0; a < HT::TM; ++a) fk[a] = Kf[((HT::m0(a) >> 4) * (CH / 32) + st) * 64 + l];
        const bf16x8 fp = Pf[(w * (CH / 32) + st) * 64 + l];
#pragma unroll
        for (int bb = 0; bb < UT::TN; ++bb) {
          const bf16x8 fu = Mma<bf16>::load(KRow<bf16, LU>{UsT}, UT::n0(bb), 32 * st);
#pragma unroll
          for (int a = 0; a < HT::TM; ++a) hs.acc[a][bb] = Mma<bf16>::mma(fk[a], fu, hs.acc[a][bb]);
          ot.acc[0][bb] = Mma<bf16>::mma(fp, fu, ot.acc[0][bb]);
        }
      }
      // the output goes to LDS (4 consecutive rows per lane: one 8-byte write);
      // the copy waves store it after the next barrier
#pragma unroll
      for (int bb = 0; bb < UT::TN; ++bb) {
        const int vv = UT::n0(bb) + (l & 15), r0 = UT::m0(0) + (l >> 4) * 4;
        bf16 o4[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) o4[j] = from_f<bf16>(ot.acc[0][bb][j]);
        *reinterpret_cast<uint2*>(OsT + vv * LU + r0) = pack4<bf16>(o4);
      }
    }
    lds_barrier();  // the last chunk's output is in LDS
    float* STp = ST + ((long)n * H + h) * DK * DV;
    hs.each([&](int d, int vv, float& x) { STp[d * DV + v0 + vv] = x; });
  } else {
    // chunk c's output, read down the columns of O^T by the transposing load
    // (16 rows x 32 columns per wave: 64 bytes of each row per 16 lanes)
    static_assert(BV == 32, "one output fragment per copy wave");
    auto store_o = [&](int c) {
      const long row0 = sp.row0 + (long)c * CH;
      const int len = min(CH, sp.len - c * CH);
      const bf16x8 x = lds_frag_tr<LU>(OsT, 16 * (w - 4), 0);
      const int r = 16 * (w - 4) + (l & 15);
      if (r < len) *reinterpret_cast<bf16x8*>(o + ((row0 + r) * H + h) * DV + v0 + 8 * (l >> 4)) = x;
    };
    // chunks past the end are clamped to the last one (a redundant copy into
    // a buffer no chunk reads again), so the fill counts are always the same
    auto cl = [&](int c) { return c < nch ? c : nch - 1; };
    if (nch > 0) {
      fill_early(0, 0);
      fill_late(0, 0);
      fill_early(cl(1), 1);
      __builtin_amdgcn_s_waitcnt(0x0F70 | NE);  // chunk 0 landed
    }
    lds_barrier();
    for (int c = 0; c < nch; ++c) {
      const long tile = (long)(sp.c0 + c) * H + h;
      lds_barrier();  // A: h of this chunk in LDS; buffer (c + 1) & 1 is free
      // issue order (kept by the empty asm statements; copies_done counts on
      // it): the previous output (conditional, so before the counted
      // operations), late fills, warm-ups, state stores, early fills
      if (c > 0) store_o(c - 1);
      asm volatile("" ::: "memory");
      fill_late(cl(c + 1), (c + 1) & 1);
      asm volatile("" ::: "memory");
      warm(cl(c + 2));
      asm volatile("" ::: "memory");
      // the chunk state leaves as whole 128-byte rows (BV fp32 of one d)
      float* hp = states + tile * DK * DV + v0;
#pragma unroll
      for (int t = 0; t < NST; ++t) {
        const int idx = (thread_x() - 256) + t * 256, d = idx / (BV / 4), c4 = (idx - d * (BV / 4)) * 4;
        *reinterpret_cast<float4*>(hp + (long)d * DV + c4) = *reinterpret_cast<const float4*>(hF + d * LF + c4);
      }
      lds_barrier();  // B: hF read; the chain is done with this buffer's W, Q, U
      asm volatile("" ::: "memory");
      fill_early(cl(c + 2), c & 1);
      copies_done();  // the next chunk's operands are in LDS before barrier A
    }
    lds_barrier();
    if (nch > 0) store_o(nch - 1);
    __builtin_amdgcn_s_waitcnt(0x0F70);  // no copy into LDS outlives the block
  }
  const int bad = __syncthreads_or(!ok);
  if (threadIdx.x == 0) flag[(long)s * NVT + vt] = bad;
}

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------
template <int DK, int DV, typename OP, int VAR>
static hipError_t launch_fwd_t(const FwdArgs& a) {
  constexpr int BV = SCAN_BV;
  constexpr int NVT = DV / BV;
  const Geo& geo = a.geo;
  const int H = geo.H;
  const FwdWs& w = a.ws;
  stage_mark(a.events, 0, a.stream);
  if (geo.cu != nullptr) {
    const hipError_t e = launch_chunk_offsets(geo.cu, geo.N, const_cast<int*>(geo.chunk_off), a.stream);
    if (e != hipSuccess) return e;
  }
  if (geo.total_chunks > 0) {
    hipLaunchKernelGGL((k_prep_fwd<DK, DV, OP, VAR>), dim3(geo.total_chunks, H), dim3(512), 0, a.stream,
                       geo, H, (const OP*)a.q, (const OP*)a.k, (const OP*)a.v, a.g, a.beta, w.gcum,
                       (OP*)w.W, (OP*)w.U, (OP*)w.KhT, (OP*)w.P, (OP*)w.Qg, w.flag_prep);
  }
  stage_mark(a.events, 1, a.stream);
  const int NS = geo.N * H;
  if (NS > 0) {
    if constexpr (sizeof(OP) == 2 && VAR != VAR_DECAY) {
      hipLaunchKernelGGL((k_scan_fwd_ws<DK, DV, BV, VAR>), dim3(NS * NVT), dim3(512), 0, a.stream, geo, H,
                         (const bf16*)a.q, a.S0, w.gcum, (const bf16*)w.W, (const bf16*)w.KhT,
                         (const bf16*)w.P, (const bf16*)w.U, a.states, a.ST, (bf16*)a.o, w.flag_scan);
    } else {
      hipLaunchKernelGGL((k_scan_fwd<DK, DV, BV, OP, VAR>), dim3(NS * NVT), dim3(256), 0, a.stream, geo, H,
                         (const OP*)w.Qg, (const OP*)a.v, a.S0, w.gcum, (const OP*)w.W, (const OP*)w.KhT,
                         (const OP*)w.P, (const OP*)w.U, a.states, a.ST, (OP*)a.o, w.flag_scan);
    }
  }
  stage_mark(a.events, 2, a.stream);
  if (NS > 0) {
    hipLaunchKernelGGL((k_exact_fwd<DK, DV, OP, VAR>), dim3(NS), dim3(DV), 0, a.stream, geo, (const OP*)a.q,
                       (const OP*)a.k, (const OP*)a.v, a.g, a.beta, a.S0, (OP*)a.o, a.ST, a.states,
                       w.flag_prep, w.flag_prep, w.flag_scan, NVT);
  }
  stage_mark(a.events, 3, a.stream);  // the chunk output is fused into the scan: stage 3 is empty
  stage_mark(a.events, 4, a.stream);
  return hipGetLastError();
}

template <int DT, int VAR>
hipError_t launch_fwd_var(const FwdArgs& a) {
  typedef typename op_of<DT>::type OP;
  const int dk = a.dk, dv = a.dv;
  if (dk == 64 && dv == 64) return launch_fwd_t<64, 64, OP, VAR>(a);
  if (dk == 64 && dv == 128) return launch_fwd_t<64, 128, OP, VAR>(a);
  if (dk == 64 && dv == 256) return launch_fwd_t<64, 256, OP, VAR>(a);
  if (dk == 128 && dv == 64) return launch_fwd_t<128, 64, OP, VAR>(a);
  if (dk == 128 && dv == 128) return launch_fwd_t<128, 128, OP, VAR>(a);
  if (dk == 128 && dv == 256) return launch_fwd_t<128, 256, OP, VAR>(a);
  return hipErrorInvalidValue;
}

}  // namespace gdn
