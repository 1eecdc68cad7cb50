// Training backward of the chunked gated delta rule on gfx950.  Only the
// chunk states cross from the forward; everything else is recomputed.
//
//   prep   one block per (chunk, head): G, T = (I + A)^{-1}, W = T diag(beta e^G) K,
//          P = (Q K^T) * D, laid out for the scan.
//   scan   the reverse inter-chunk state scan (paper Sec. 4.2, K#1): one block
//          per (stream, value tile); an fp32 carry dh walks the chunks from the
//          last to the first,
//            dU' = P^T dO + Khat dh,   dh <- e^{G_last} dh + Q^T diag(e^G) dO - W^T dU',
//          storing the carry that enters every chunk; dS0 is the final carry.
//   grad   one block per (chunk, head): every chunk-local gradient, with the
//          triangular-inverse VJP (paper Sec. 4.2, K#2) that reuses T in four
//          triangular products, dA = -T^T dT T^T, and never re-inverts.
//
// The grad kernel avoids W and U: with R = diag(beta) V - diag(beta e^G) K h,
//   U' = T R,   Y = T^T dU',   X = -Y h^T  (= T^T dW),   dT = dU' R^T,
// which follow from W = T diag(beta e^G) K, U = T diag(beta) V, dW = -dU' h^T.
// Per chunk, with h the state entering the chunk and dh the carry leaving it:
//   dP  = dO U'^T,              dQ = diag(e^G) dO h^T + (dP * D) K
//   dK  = (dP * D)^T Q + diag(e^{G_last - G}) U' dh^T + diag(beta e^G) X
//         + (dB + dB^T) K,      dB = dA * beta_r * E   (strict lower)
//   dV  = diag(beta) Y,         dbeta_r = v_r.Y_r + e^{G_r} k_r.X_r + sum_i dA_ri (K K^T)_ri E_ri
//   dG_r = rowsum_r(Z) - colsum_r(Z) + e^{G_r} (q_r.(dO h^T)_r + beta_r k_r.X_r)
//          - khat_r.dkhat_r,   Z = dA * A + dP * P,
//   dG_last += e^{G_last} <h, dh> + sum_r khat_r.dkhat_r,   dg = reverse cumsum of dG.
#pragma once

#include "gdn_chunk.hpp"
#include "gdn_exact.hpp"
#include "gdn_launch.hpp"

namespace gdn {

template <int DK, int DV, typename OP, int VAR>
__global__ __launch_bounds__(512) void k_prep_bwd(Geo geo, int H, const OP* __restrict__ q,
                                                  const OP* __restrict__ k, const float* __restrict__ g,
                                                  const float* __restrict__ beta, const OP* __restrict__ dO,
                                                  float* __restrict__ gcum, OP* __restrict__ WTg,
                                                  OP* __restrict__ QgTg, OP* __restrict__ dOTg,
                                                  OP* __restrict__ PTg, OP* __restrict__ Tg,
                                                  OP* __restrict__ Khg, int* __restrict__ flag) {
  constexpr bool DT_ = VAR != VAR_DECAY;
  // bf16 operands read transposed tiles straight from row-major LDS with the
  // transposing load; fp32 operands go through explicit transposed copies
  constexpr bool TR = sizeof(OP) == 2;
  constexpr int LK = DK + pad_of<OP>();
  constexpr int LC = CH + 4;
  constexpr int LT = CH + pad_of<OP>();
  // dO^T is laid out only for the fp32 scan; the bf16 scan reads dO's rows itself
  constexpr bool DOT = !TR;
  constexpr int VS = 64;  // value columns per slice of dO
  constexpr int LVS = VS + pad_of<OP>();
  constexpr int VE = 16 / (int)sizeof(OP);
  typedef typename vec4_of<OP>::type V4;
  // LDS regions are reused by lifetime so that two blocks fit on a CU:
  //   R1: Q, then T in fp32;  R2: K (bf16: alive through W; fp32: then T);
  //   R3: bf16: T in bf16; fp32: (diag(beta e^G) K)^T;  R4: A in fp32 (fp32: then dO).
  constexpr int R1 = CH * LK * (int)sizeof(OP) > CH * LC * 4 ? CH * LK * (int)sizeof(OP) : CH * LC * 4;
  constexpr int R2 = CH * LK * (int)sizeof(OP);
  constexpr int R3 = !DT_ ? 16 : (TR ? CH * LT * (int)sizeof(OP) : DK * LT * (int)sizeof(OP));
  constexpr int R4 = (!DOT || CH * LC * 4 > CH * LVS * (int)sizeof(OP)) ? CH * LC * 4 : CH * LVS * (int)sizeof(OP);
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
  OP* dOs = reinterpret_cast<OP*>(r4);

  const int ci = blockIdx.x, h = blockIdx.y;
  const ChunkPos cp = chunk_pos(geo, ci);
  const long tile = (long)ci * H + h;
  const int l = lane_id(), wv = wave_id();
  // every input row of the block is requested up front: q, k, then (fp32)
  // the dO slices (slice t of VS columns is piece t of each thread)
  RowsIn<DK, 512, OP> qin, kin;
  qin.load(q + (cp.row0 * H + h) * DK, (long)H * DK, cp.len);
  kin.load(k + (cp.row0 * H + h) * DK, (long)H * DK, cp.len);
  const OP* dop = dO + (cp.row0 * H + h) * DV;
  constexpr int NSL = DOT ? DV / VS : 1, NPS = DOT ? CH * VS / VE / 512 : 1;  // slices; pieces per thread and slice
  uint4 din[NSL][NPS];
  if constexpr (DOT) {
#pragma unroll
    for (int t = 0; t < NSL; ++t)
#pragma unroll
      for (int p = 0; p < NPS; ++p) {
        const int idx = threadIdx.x + p * 512, i = idx / (VS / VE), c = t * VS + (idx % (VS / VE)) * VE;
        din[t][p] = *reinterpret_cast<const uint4*>(dop + (long)clamp_row(i, cp.len) * H * DV + c);
      }
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
  // P^T, written (i, r): the scan's A operand for P^T dO
  {
    Tiles<CH, CH, 4, 2> p;
    p.zero();
    p.template mma<OP, DK>(KRow<OP, LK>{Qs}, KRow<OP, LK>{Ks});
    OP* Pt = PTg + tile * CH * CH;
#pragma unroll
    for (int b = 0; b < p.TN; ++b) {
      const int i = p.n0(b) + (l & 15), r0 = p.m0(0) + (l >> 4) * 4;
      OP v4[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = r0 + j;
        v4[j] = from_f<OP>(i <= r ? p.acc[0][b][j] * __expf(Gs[r] - Gs[i]) : 0.f);
      }
      *reinterpret_cast<V4*>(Pt + op_off<OP, CH>(i, r0)) = pack4<OP>(v4);
    }
  }
  // (diag(e^G) Q)^T for the scan's injection term
  {
    OP* Qg = QgTg + tile * DK * CH;
    if constexpr (TR) {
      // one transposed fragment (16 d x 32 r) of Q per wave and step, stored
      // as one contiguous 1 KiB block
#pragma unroll
      for (int t = 0; t < DK * CH / (512 * 8); ++t) {
        const int f = wv + 8 * t, mt = f / (CH / 32), s = f % (CH / 32);
        const bf16x8 x = scale_frag(lds_frag_tr<LK>(Qs, 16 * mt, 32 * s), Gam, 32 * s);
        *reinterpret_cast<bf16x8*>(Qg + ((long)f * 64 + l) * 8) = x;
      }
    } else {
      for (int idx = threadIdx.x; idx < DK * CH / VE; idx += blockDim.x) {
        const int d = idx / (CH / VE), r0 = (idx - d * (CH / VE)) * VE;
        OP vals[VE];
#pragma unroll
        for (int j = 0; j < VE; ++j) vals[j] = from_f<OP>(Gam[r0 + j] * to_f(Qs[(r0 + j) * LK + d]));
        *reinterpret_cast<uint4*>(Qg + op_off<OP, CH>(d, r0)) = pack16<OP>(vals);
      }
    }
  }
  // Khat = diag(e^{G_last - G}) K, the A operand of dU' in the generic scan
  // (rows past the end stay zero; the split bf16 scan reads k itself)
  if constexpr (!TR) {
    OP* Kh = Khg + tile * CH * DK;
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
      const uint4 kv = *reinterpret_cast<const uint4*>(Ks + r * LK + d0);
      OP vals[VE];
#pragma unroll
      for (int j = 0; j < VE; ++j) vals[j] = from_f<OP>(Dte[r] * to_f(elem16<OP>(kv, j)));
      *reinterpret_cast<uint4*>(Kh + op_off<OP, DK>(r, d0)) = pack16<OP>(vals);
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
    __syncthreads();
    // Tf over Q (dead here); Ts over K for fp32, in its own region for bf16
    unit_lower_inverse<OP, LC, LT, false>(As, Tf, Ts, (OP*)nullptr);
    const OP* Tp;
    if constexpr (TR) Tp = Ts; else Tp = reinterpret_cast<const OP*>(Tf);
    constexpr int LTT = TR ? LT : LC;
    // T itself, row-major, for the gradient kernel
    for (int idx = threadIdx.x; idx < CH * CH / VE; idx += blockDim.x) {
      const int r = idx / (CH / VE), c = (idx - r * (CH / VE)) * VE;
      *reinterpret_cast<uint4*>(Tg + tile * CH * CH + r * CH + c) = *reinterpret_cast<const uint4*>(Tp + r * LTT + c);
    }
    // W = T diag(beta e^G) K, written transposed (d, r)
    Tiles<CH, DK, 4, 2> w;
    w.zero();
    if constexpr (TR)
      w.template mma<OP, CH>(KRow<OP, LT>{Tp}, KColTr<LK, true>{Ks, BG});
    else
      w.template mma<OP, CH>(KRow<OP, LTT>{Tp}, KRow<OP, LT>{KbT});
    OP* Wt = WTg + tile * DK * CH;
#pragma unroll
    for (int b = 0; b < w.TN; ++b) {
      const int d = w.n0(b) + (l & 15), r0 = w.m0(0) + (l >> 4) * 4;
      OP v4[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) v4[j] = from_f<OP>(w.acc[0][b][j]);
      *reinterpret_cast<V4*>(Wt + op_off<OP, CH>(d, r0)) = pack4<OP>(v4);
    }
  }
  if constexpr (DOT) {
    // dO^T, the fp32 scan's A operand for the injection term, in slices of VS
    // value columns (dO slices reuse the A region)
    OP* dOt = dOTg + tile * DV * CH;
    __syncthreads();
#pragma unroll
    for (int t = 0; t < NSL; ++t) {
      const int c0 = t * VS;
#pragma unroll
      for (int p = 0; p < NPS; ++p) {
        const int idx = threadIdx.x + p * 512, i = idx / (VS / VE), v0 = (idx % (VS / VE)) * VE;
        const uint4 x = keep16(i < cp.len, din[t][p]);
        ok &= finite16B<OP>(x);
        *reinterpret_cast<uint4*>(dOs + i * LVS + v0) = x;
      }
      __syncthreads();
      for (int idx = threadIdx.x; idx < VS * CH / VE; idx += blockDim.x) {
        const int vv = idx / (CH / VE), r0 = (idx - vv * (CH / VE)) * VE;
        OP vals[VE];
#pragma unroll
        for (int j = 0; j < VE; ++j) vals[j] = dOs[(r0 + j) * LVS + vv];
        *reinterpret_cast<uint4*>(dOt + op_off<OP, CH>(c0 + vv, r0)) = pack16<OP>(vals);
      }
      __syncthreads();
    }
  }
  const int bad = __syncthreads_or(!ok);
  if (threadIdx.x == 0) flag[tile] = bad;
}

// The reverse inter-chunk state scan (paper Sec. 4.2, K#1).  The fp32 carry dh
// (the gradient w.r.t. the state leaving the chunk) stays in registers; the
// prep kernel lays out every other operand for direct fragment loads (W^T,
// (diag(e^G) Q)^T, dO^T, P^T), and the fragments of chunk c-1 are fetched
// into registers while chunk c is processed:
//   dU' = P^T dO + diag(e^{G_last - G}) K dh
//   dh <- e^{G_last} dh + (diag(e^G) Q)^T dO - W^T dU'
// CWD (channel-wise decay): dh decays row by row, dh[d, :] *= e^{G_last[d]}, with
// gcum holding each chunk's d_k values of G_last.
template <int DK, int DV, int BV, typename OP, int VAR, bool CWD = false>
__global__ __launch_bounds__(256) void k_scan_bwd(Geo geo, int H, const OP* __restrict__ Khg,
                                                  const float* __restrict__ dST, const float* __restrict__ gcum,
                                                  const OP* __restrict__ WTg, const OP* __restrict__ QgTg,
                                                  const OP* __restrict__ dOTg, const OP* __restrict__ PTg,
                                                  OP* __restrict__ dhg, OP* __restrict__ dUTg,
                                                  float* __restrict__ dS0, int* __restrict__ flag) {
  constexpr int NVT = DV / BV;
  constexpr bool DT_ = VAR != VAR_DECAY;  // delta term present
  constexpr int LK = DK + pad_of<OP>();
  constexpr int LU = CH + pad_of<OP>();
  constexpr bool PF = sizeof(OP) == 2;
  typedef Tiles<DK, BV, 4, 1> HT;  // dh slice
  typedef Tiles<CH, BV, 4, 1> UT;  // dU' slice
  __shared__ __align__(16) OP dhT[BV * LK];
  __shared__ __align__(16) OP dUT[DT_ ? BV * LU : 1];

  int s, vt;
  scan_block_coords(blockIdx.x, geo.N * H, NVT, s, vt);
  const int n = s / H, h = s - (s / H) * H, v0 = vt * BV;
  const SeqPos sp = seq_pos(geo, n);
  const int l = lane_id();

  struct Pre {
    typename UT::template AFr<OP, DK> kf;
    typename HT::template AFr<OP, CH> wt;
    typename HT::template AFr<OP, CH> qg;
    typename HT::template BFr<OP, CH> dob;
    typename UT::template AFr<OP, CH> pt;
    float gl;  // G_last, exponentiated at use so the prefetch never waits
    float gd[CWD ? HT::TM : 1][4];  // CWD: G_last of this lane's rows of dh
  };
  auto load_pre = [&](Pre& p, int c) {
    const long tile = (long)(sp.c0 + c) * H + h;
    load_op_frags<HT, OP, CH>(p.qg, QgTg + tile * DK * CH);
    if constexpr (sizeof(OP) == 2)
      load_op_frags_b<HT, OP, CH>(p.dob, dOTg + tile * DV * CH + op_off<OP, CH>(v0, 0));
    else
      p.dob.load(KRow<OP, CH>{dOTg + tile * DV * CH + (long)v0 * CH});
    if constexpr (CWD) {
#pragma unroll
      for (int a = 0; a < HT::TM; ++a)
#pragma unroll
        for (int j = 0; j < 4; ++j) p.gd[a][j] = gcum[tile * DK + HT::m0(a) + (l >> 4) * 4 + j];
    } else {
      p.gl = gcum[tile * CH + CH - 1 + opaque_zero()];  // vector load: see opaque_zero
    }
    load_op_frags<UT, OP, DK>(p.kf, Khg + tile * CH * DK);
    if constexpr (DT_) load_op_frags<HT, OP, CH>(p.wt, WTg + tile * DK * CH);
    load_op_frags<UT, OP, CH>(p.pt, PTg + tile * CH * CH);
  };

  HT dh;
  bool ok = true;
  const float* dSTp = dST ? dST + ((long)n * H + h) * DK * DV : nullptr;
  dh.each([&](int d, int vv, float& x) {
    x = dSTp ? dSTp[d * DV + v0 + vv] : 0.f;
    ok &= finite_f(x);
  });

  // One chunk of the reverse carry.  `prefetch` issues the loads of the
  // previous chunk right after the barrier that opens this one; the two
  // fragment buffers alternate, so nothing is copied.
  auto step = [&](int c, const Pre& cur, auto&& prefetch) {
    const long tile = (long)(sp.c0 + c) * H + h;
    // dh to LDS (4 consecutive d per lane: one vector write)
#pragma unroll
    for (int a = 0; a < HT::TM; ++a)
#pragma unroll
      for (int b = 0; b < HT::TN; ++b) {
        const int d0 = HT::m0(a) + (l >> 4) * 4, vv = HT::n0(b) + (l & 15);
        OP h4[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) h4[j] = from_f<OP>(dh.acc[a][b][j]);
        *reinterpret_cast<typename vec4_of<OP>::type*>(dhT + vv * LK + d0) = pack4<OP>(h4);
      }
    __syncthreads();
    prefetch();
    {
      // dh entering this chunk, for the gradient kernel, in its fragment order
      constexpr int VE = 16 / (int)sizeof(OP);
      OP* dhp = dhg + tile * DK * DV;
      if constexpr (sizeof(OP) == 2) {
        // one (16 d x 32 v) fragment per wave and step, read down the columns
        // of dh^T by the transposing load and stored as one 1 KiB block
        static_assert(BV % 32 == 0 && (DK / 16) * (BV / 32) % 4 == 0, "whole fragments per wave");
#pragma unroll
        for (int t = 0; t < (DK / 16) * (BV / 32) / 4; ++t) {
          const int f = wave_id() + 4 * t, mt = f / (BV / 32), kb = f - mt * (BV / 32);
          const bf16x8 x = lds_frag_tr<LK>(dhT, 16 * mt, 32 * kb);
          *reinterpret_cast<bf16x8*>(dhp + op_off<OP, DV>(16 * mt, v0 + 32 * kb) + l * 8) = x;
        }
      } else {
#pragma unroll
        for (int t = 0; t < DK * BV / VE / 256; ++t) {
          const int idx = threadIdx.x + t * 256, d = idx / (BV / VE), vq = (idx - d * (BV / VE)) * VE;
          OP vals[VE];
#pragma unroll
          for (int j = 0; j < VE; ++j) vals[j] = dhT[(vq + j) * LK + d];
          *reinterpret_cast<uint4*>(dhp + op_off<OP, DV>(d, v0 + vq)) = pack16<OP>(vals);
        }
      }
    }
    HT inj;  // (diag(e^G) Q)^T dO, independent of the carry
    inj.zero();
    inj.template mma<OP, CH>(cur.qg, cur.dob);
    {
      // dU' = P^T dO + diag(e^{G_last - G}) K dh (written for the gradient kernel for every
      // family member; only the delta rule feeds it back into the carry)
      UT du;
      du.zero();
      du.template mma<OP, DK>(cur.kf, KRow<OP, LK>{dhT});  // Khat dh
      du.template mma_raw<OP, CH / Mma<OP>::KSTEP>(cur.pt.f, cur.dob.f);  // + P^T dO
      OP* dUg = dUTg + tile * DV * CH;
#pragma unroll
      for (int b = 0; b < UT::TN; ++b) {
        const int vv = UT::n0(b) + (l & 15), r0 = UT::m0(0) + (l >> 4) * 4;
        OP u4[4], n4[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float u = du.acc[0][b][j];
          n4[j] = from_f<OP>(-u);
          u4[j] = from_f<OP>(u);
        }
        if (DT_) *reinterpret_cast<typename vec4_of<OP>::type*>(dUT + vv * LU + r0) = pack4<OP>(n4);
        // dU' of this chunk for the gradient kernel, transposed (v, r), in its fragment order
        *reinterpret_cast<typename vec4_of<OP>::type*>(dUg + op_off<OP, CH>(v0 + vv, r0)) = pack4<OP>(u4);
      }
      __syncthreads();
    }
#pragma unroll
    for (int a = 0; a < HT::TM; ++a)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float gd = CWD ? expf(cur.gd[a][CWD ? j : 0]) : expf(cur.gl);
#pragma unroll
        for (int b = 0; b < HT::TN; ++b) dh.acc[a][b][j] = gd * dh.acc[a][b][j] + inj.acc[a][b][j];
      }
    if constexpr (DT_) dh.template mma<OP, CH>(cur.wt, KRow<OP, LU>{dUT});
  };
  const int nch = sp.nch;
  if constexpr (PF) {
    // The prefetch always issues (before the first chunk it re-reads chunk 0):
    // a conditional prefetch would leave one path with fewer memory operations
    // in flight, and the wait counts, merged over both paths, would then wait
    // for the loads just issued.
    if (nch > 0) {
      Pre p0, p1;
      load_pre(p0, nch - 1);
      for (int c = nch - 1; c >= 0; c -= 2) {
        step(c, p0, [&] { load_pre(p1, max(c - 1, 0)); });
        if (c - 1 >= 0) step(c - 1, p1, [&] { load_pre(p0, max(c - 2, 0)); });
      }
    }
  } else {
    Pre cur;
    for (int c = nch - 1; c >= 0; --c) {
      load_pre(cur, c);
      step(c, cur, [] {});
    }
  }
  float* dS0p = dS0 + ((long)n * H + h) * DK * DV;
  dh.each([&](int d, int vv, float& x) { dS0p[d * DV + v0 + vv] = x; });
  const int bad = __syncthreads_or(!ok);
  if (threadIdx.x == 0) flag[(long)s * NVT + vt] = bad;
}

// The reverse scan for bf16 operands, split into four chain waves and four
// copy waves (the layout of the forward scan's split): every per-chunk
// operand of the carry (K, (diag(e^G) Q)^T, W^T, this block's columns of dO,
// P^T and the chunk's G) goes through LDS in 1 KiB blocks, which the copy
// waves move into one of two LDS buffers with global_load_lds_dwordx4 a chunk
// ahead (warming L2 two chunks ahead): the prep kernel's outputs are stored
// as MFMA fragment blocks in HBM, k's token-major rows (the contraction
// index d_k is contiguous there) are gathered a line at a time (RowLines),
// and dO's rows are gathered as this block's 64 bytes of each (16 rows per
// block, row-major), whose B fragments the chain reads down the columns with
// the transposing load.
// The copy waves also write the dh
// entering each chunk out of LDS.  Per chunk:
//   chain: dh -> LDS | barrier | inj = Qg^T dO,
//          dU' = diag(e^{G_last - G}) (K dh) + P^T dO, store dU'^T | barrier |
//          dh <- e^{G_last} dh + inj - W^T dU'
//   copy:             | operands of the chunk before -> LDS, dh -> HBM | | wait
template <int DK, int DV, int BV, int VAR>
__global__ __launch_bounds__(512) void k_scan_bwd_ws(Geo geo, int H, const bf16* __restrict__ k,
                                                     const float* __restrict__ dST, const float* __restrict__ gcum,
                                                     const bf16* __restrict__ WTg, const bf16* __restrict__ QgTg,
                                                     const bf16* __restrict__ dO, const bf16* __restrict__ PTg,
                                                     bf16* __restrict__ dhg, bf16* __restrict__ dUTg,
                                                     float* __restrict__ dS0, int* __restrict__ flag) {
  static_assert(BV == SCAN_BV, "value tiles");
  // one row of this block's dO columns is BV bf16 = 4 pieces of 16 bytes: a
  // 1 KiB block holds 16 rows, row-major
  static_assert(BV * 2 == 64, "four 16-byte pieces per dO row");
  constexpr int NVT = DV / BV;
  constexpr bool DT_ = VAR != VAR_DECAY;  // delta term present
  typedef RowLines<DK> KL;
  static_assert(KL::NBLK == (CH / 16) * (DK / 32), "k takes the blocks of a 64 x DK fragment operand");
  constexpr int LK = DK + 8, LU = CH + 8;
  typedef Tiles<DK, BV, 4, 1> HT;  // dh slice (chain waves)
  typedef Tiles<CH, BV, 4, 1> UT;  // dU' slice (chain waves)
  constexpr int NKh = (CH / 16) * (DK / 32), NQ = (DK / 16) * (CH / 32), NWT = DT_ ? NQ : 0;
  constexpr int ND = CH * BV * 2 / 1024, NP = (CH / 16) * (CH / 32);
  constexpr int OKh = 0, OQ = OKh + NKh, OW = OQ + NQ, OD = OW + NWT, OP_ = OD + ND, NB = OP_ + NP;
  constexpr int BUF = NB * 1024 + CH * 4;  // + the chunk's G (64 fp32)
  __shared__ __align__(1024) char buf[2][BUF];
  __shared__ __align__(16) bf16 dhT[BV * LK];
  __shared__ __align__(16) bf16 dUT[DT_ ? BV * LU : 8];
  __shared__ __align__(16) char sink[256];  // target of the L2 warm-up loads (never read)

  int s, vt;
  scan_block_coords(blockIdx.x, geo.N * H, NVT, s, vt);
  const int n = s / H, h = s - (s / H) * H, v0 = vt * BV;
  const SeqPos sp = seq_pos(geo, n);
  const int w = wave_id(), l = lane_id();
  const bool chain = w < 4;
  const int nch = sp.nch;

  typedef __attribute__((address_space(1))) void gvoid;
  typedef __attribute__((address_space(3))) void lvoid;
  // row r of k in chunk c (rows past the chunk's end repeat its last row;
  // their products are masked)
  auto k_row = [&](int c, int r) -> const bf16* {
    const int len = min(CH, sp.len - c * CH);
    return k + ((sp.row0 + (long)c * CH + clamp_row(r, len)) * H + h) * DK;
  };
  // row r of this block's dO columns in chunk c (rows past the chunk's end
  // repeat its last row; they meet zero rows of P and of (diag(e^G) Q))
  auto do_row = [&](int c, int r) -> const bf16* {
    const int len = min(CH, sp.len - c * CH);
    return dO + ((sp.row0 + (long)c * CH + clamp_row(r, len)) * H + h) * DV + v0;
  };
  // start of prep-written block j (j >= OQ, outside the dO blocks)
  auto src_of = [&](long tile, int j) -> const bf16* {
    if (j < OW) return QgTg + tile * DK * CH + (j - OQ) * 512;
    if (j < OD) return WTg + tile * DK * CH + (j - OW) * 512;
    return PTg + tile * CH * CH + (j - OP_) * 512;
  };
  // copy waves: chunk c's operands into buffer b (wave w - 4 takes every fourth block)
  auto fill = [&](int c, int b) {
    const long tile = (long)(sp.c0 + c) * H + h;
#pragma unroll
    for (int j0 = 0; j0 < NB; j0 += 4) {
      const int j = j0 + (w - 4);
      if (j < NB) {
        const bf16* src;
        if (j < OQ) {
          int r, e;
          KL::src(j - OKh, l, r, e);
          src = k_row(c, r) + e;
        } else if (j >= OD && j < OP_) {
          src = do_row(c, 16 * (j - OD) + (l >> 2)) + 8 * (l & 3);
        } else {
          src = src_of(tile, j) + l * 8;
        }
        __builtin_amdgcn_global_load_lds((gvoid*)src, (lvoid*)(buf[b] + j * 1024), 16, 0, 0);
      }
    }
    if (w == 4) __builtin_amdgcn_global_load_lds((gvoid*)(gcum + tile * CH + l), (lvoid*)(buf[b] + NB * 1024), 4, 0, 0);
  };
  // L2 warm-up: the NVT blocks of a stream split the shared blocks (all but
  // the dO rows), touching every 128-byte line once, and each warms the 64
  // lines its own dO columns lie in: one 4-byte load per lane (64 lines per
  // instruction)
  constexpr int NSHB = NB - ND;
  constexpr int NSH = (NSHB + NVT - 1) / NVT;
  constexpr int NWL = NSH * 8 + CH;
  constexpr int NWARM = (NWL + 255) / 256;
  auto warm = [&](int c) {
    const long tile = (long)(sp.c0 + c) * H + h;
#pragma unroll
    for (int t = 0; t < NWARM; ++t) {
      int L = ((w - 4) + 4 * t) * 64 + l;
      L = L < NWL ? L : NWL - 1;
      // lanes past the shared lines take dO's rows: one load per lane either
      // way (the address is selected, the load is not branched around: every
      // iteration issues exactly one load, which the wait counts rely on)
      const bool own = L >= NSH * 8;
      const int Ls = own ? 0 : L;
      const int e = Ls >> 3;
      int j = e * NVT + vt;                 // index among the shared blocks
      j = j < NSHB ? j : NSHB - 1;
      j = j < OD ? j : j + ND;              // skip the dO rows
      const bf16* src;
      if (j < OQ) {
        // line (L & 7) of k block j - OKh
        int r, e;
        KL::src(j - OKh, (Ls & 7) << 3, r, e);
        src = k_row(c, r) + (e & ~63);
      } else {
        src = src_of(tile, j) + (Ls & 7) * 64;
      }
      src = own ? do_row(c, L - NSH * 8) : src;
      __builtin_amdgcn_global_load_lds((gvoid*)src, (lvoid*)sink, 4, 0, 0);
    }
  };
  constexpr int NST = (DK / 16) * (BV / 32) / 4;  // dh fragment stores per copy-wave lane and chunk
  static_assert((DK / 16) * (BV / 32) % 4 == 0 && NWARM + NST < 16, "whole fragments; vmcnt field");
  auto copies_done = [] { __builtin_amdgcn_s_waitcnt(0x0F70 | (NWARM + NST)); };  // vmcnt(NWARM + NST)
  auto lds_barrier = [] { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); };

  bool ok = true;
  if (chain) {
    HT dh;
    const float* dSTp = dST ? dST + ((long)n * H + h) * DK * DV : nullptr;
    dh.each([&](int d, int vv, float& x) {
      x = dSTp ? dSTp[d * DV + v0 + vv] : 0.f;
      ok &= finite_f(x);
    });
    lds_barrier();
    for (int i = 0; i < nch; ++i) {
      const int c = nch - 1 - i;
      const char* B = buf[i & 1];
      const long tile = (long)(sp.c0 + c) * H + h;
      // dh to LDS (4 consecutive d per lane: one 8-byte write)
#pragma unroll
      for (int a = 0; a < HT::TM; ++a)
#pragma unroll
        for (int bb = 0; bb < HT::TN; ++bb) {
          const int d0 = HT::m0(a) + (l >> 4) * 4, vv = HT::n0(bb) + (l & 15);
          bf16 h4[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) h4[j] = from_f<bf16>(dh.acc[a][bb][j]);
          *reinterpret_cast<uint2*>(dhT + vv * LK + d0) = pack4<bf16>(h4);
        }
      lds_barrier();  // A: dh in LDS, this chunk's operands in buffer i & 1
      const bf16x8* Kf = reinterpret_cast<const bf16x8*>(B + OKh * 1024);
      const bf16x8* Qf = reinterpret_cast<const bf16x8*>(B + OQ * 1024);
      // row scales e^{G_last - G_r} of K dh (0 past the chunk's end), formed
      // here under the products
      float er[4];
      {
        const float* Gc = reinterpret_cast<const float*>(B + NB * 1024);
        const int len = min(CH, sp.len - c * CH);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int r = UT::m0(0) + (l >> 4) * 4 + j;
          er[j] = r < len ? __expf(Gc[CH - 1] - Gc[r]) : 0.f;
        }
      }
      const bf16* Drows = reinterpret_cast<const bf16*>(B + OD * 1024);  // dO[r][v], row stride BV
      const bf16x8* Pf = reinterpret_cast<const bf16x8*>(B + OP_ * 1024);
      bf16x8 fd[CH / 32][HT::TN];  // dO columns: B fragments of both products
#pragma unroll
      for (int st = 0; st < CH / 32; ++st)
#pragma unroll
        for (int bb = 0; bb < HT::TN; ++bb) fd[st][bb] = lds_frag_tr<BV>(Drows, HT::n0(bb), 32 * st);
      HT inj;  // (diag(e^G) Q)^T dO, independent of the carry
      inj.zero();
#pragma unroll
      for (int st = 0; st < CH / 32; ++st)
#pragma unroll
        for (int a = 0; a < HT::TM; ++a) {
          const bf16x8 fq = Qf[((HT::m0(a) >> 4) * (CH / 32) + st) * 64 + l];
#pragma unroll
          for (int bb = 0; bb < HT::TN; ++bb) inj.acc[a][bb] = Mma<bf16>::mma(fq, fd[st][bb], inj.acc[a][bb]);
        }
      {
        // dU' = diag(e^{G_last - G}) (K dh) + P^T dO (written for the gradient
        // kernel for every family member; only the delta rule feeds it back
        // into the carry).  The row scale goes on the fp32 products; rows past
        // the chunk's end are zero.
        UT du;
        du.zero();
#pragma unroll
        for (int st = 0; st < DK / 32; ++st) {
          const bf16x8 fk = Kf[KL::frag_slot(w, st, l)];
#pragma unroll
          for (int bb = 0; bb < UT::TN; ++bb)
            du.acc[0][bb] = Mma<bf16>::mma(fk, Mma<bf16>::load(KRow<bf16, LK>{dhT}, UT::n0(bb), 32 * st), du.acc[0][bb]);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int bb = 0; bb < UT::TN; ++bb) du.acc[0][bb][j] *= er[j];
#pragma unroll
        for (int st = 0; st < CH / 32; ++st) {
          const bf16x8 fp = Pf[(w * (CH / 32) + st) * 64 + l];
#pragma unroll
          for (int bb = 0; bb < UT::TN; ++bb) du.acc[0][bb] = Mma<bf16>::mma(fp, fd[st][bb], du.acc[0][bb]);
        }
        bf16* dUg = dUTg + tile * DV * CH;
#pragma unroll
        for (int bb = 0; bb < UT::TN; ++bb) {
          const int vv = UT::n0(bb) + (l & 15), r0 = UT::m0(0) + (l >> 4) * 4;
          bf16 u4[4], n4[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const float u = du.acc[0][bb][j];
            n4[j] = from_f<bf16>(-u);
            u4[j] = from_f<bf16>(u);
          }
          if constexpr (DT_) *reinterpret_cast<uint2*>(dUT + vv * LU + r0) = pack4<bf16>(n4);
          // dU' of this chunk for the gradient kernel, transposed (v, r), in its fragment order
          *reinterpret_cast<uint2*>(dUg + op_off<bf16, CH>(v0 + vv, r0)) = pack4<bf16>(u4);
        }
      }
      lds_barrier();  // B: -dU' in LDS; dh read by the copy waves
      const float gl = __expf(reinterpret_cast<const float*>(B + NB * 1024)[CH - 1]);
#pragma unroll
      for (int a = 0; a < HT::TM; ++a)
#pragma unroll
        for (int bb = 0; bb < HT::TN; ++bb)
#pragma unroll
          for (int j = 0; j < 4; ++j) dh.acc[a][bb][j] = gl * dh.acc[a][bb][j] + inj.acc[a][bb][j];
      if constexpr (DT_) {
        const bf16x8* Wf = reinterpret_cast<const bf16x8*>(B + OW * 1024);
#pragma unroll
        for (int st = 0; st < CH / 32; ++st)
#pragma unroll
          for (int a = 0; a < HT::TM; ++a) {
            const bf16x8 fw = Wf[((HT::m0(a) >> 4) * (CH / 32) + st) * 64 + l];
#pragma unroll
            for (int bb = 0; bb < HT::TN; ++bb)
              dh.acc[a][bb] = Mma<bf16>::mma(fw, Mma<bf16>::load(KRow<bf16, LU>{dUT}, HT::n0(bb), 32 * st), dh.acc[a][bb]);
          }
      }
    }
    float* dS0p = dS0 + ((long)n * H + h) * DK * DV;
    dh.each([&](int d, int vv, float& x) { dS0p[d * DV + v0 + vv] = x; });
  } else {
    if (nch > 0) {
      fill(nch - 1, 0);
      __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
    }
    lds_barrier();
    for (int i = 0; i < nch; ++i) {
      const int c = nch - 1 - i;
      const long tile = (long)(sp.c0 + c) * H + h;
      lds_barrier();  // A: dh entering this chunk in LDS; buffer (i + 1) & 1 is free
      // issue order fills, warm-ups, stores (kept by the empty asm statements):
      // copies_done counts on it
      if (c > 0) fill(c - 1, (i + 1) & 1);
      asm volatile("" ::: "memory");
      warm(c > 1 ? c - 2 : 0);
      asm volatile("" ::: "memory");
      // dh entering this chunk, for the gradient kernel: (16 d x 32 v) fragments
      // read down the columns of dh^T by the transposing load, 1 KiB per store
      bf16* dhp = dhg + tile * DK * DV;
#pragma unroll
      for (int t = 0; t < NST; ++t) {
        const int f = (w - 4) + 4 * t, mt = f / (BV / 32), kb = f - mt * (BV / 32);
        const bf16x8 x = lds_frag_tr<LK>(dhT, 16 * mt, 32 * kb);
        *reinterpret_cast<bf16x8*>(dhp + op_off<bf16, DV>(16 * mt, v0 + 32 * kb) + l * 8) = x;
      }
      lds_barrier();  // B: dh read
      copies_done();  // the chunk before's operands are in LDS before barrier A
    }
  }
  const int bad = __syncthreads_or(!ok);
  if (threadIdx.x == 0) flag[(long)s * NVT + vt] = bad;
}

// Bytes of the phase-dependent region of the grad kernel (LDS for bf16
// operands, a per-block slice of the workspace for fp32 operands).
template <int DK, typename OP>
struct GradRegion {
  static constexpr int P8 = 16 / (int)sizeof(OP);
  static constexpr int LK = DK + P8, LT = CH + P8, LC = CH + 4;
  static constexpr int VS = 32, LV = VS + P8;
  static constexpr bool BF = sizeof(OP) == 2;
  // phase 0: Qs, As, Tf (bf16 only), Xs
  static constexpr int ph0 = CH * LK * (int)sizeof(OP) + CH * LC * 4 + (BF ? CH * LC * 4 : 0) + 4 * 16 * 20 * 4;
  // phase 1: Vs, dOs, Rs, Ups, dUs, Ys, dVst [64][LV]; hs, dhs [DK][LV]; hsT [VS][LK]; RT, dUT [VS][LT]
  static constexpr int ph1 = (7 * CH * LV + 2 * DK * LV + VS * LK + 2 * VS * LT) * (int)sizeof(OP);
  // phase 2: QT, KT [DK][LT]; SdT, M1, dPs, dPmT [64][LT]
  static constexpr int ph2 = (2 * DK * LT + 4 * CH * LT) * (int)sizeof(OP);
  static constexpr int bytes = ((ph0 > ph1 ? (ph0 > ph2 ? ph0 : ph2) : (ph1 > ph2 ? ph1 : ph2)) + 255) / 256 * 256;
  static_assert(bytes == grad_region_bytes(DK, (int)sizeof(OP)), "host and device disagree");
};

template <int DK, int DV, typename OP, int VAR>
__global__ __launch_bounds__(512) void k_grad_bwd(Geo geo, int H, const OP* __restrict__ q,
                                                  const OP* __restrict__ k, const OP* __restrict__ v,
                                                  const float* __restrict__ g, const float* __restrict__ beta,
                                                  const float* __restrict__ states, const OP* __restrict__ dO,
                                                  const OP* __restrict__ dhg, const OP* __restrict__ dUTg,
                                                  OP* __restrict__ dq,
                                                  OP* __restrict__ dk, OP* __restrict__ dvo,
                                                  float* __restrict__ dg, float* __restrict__ dbeta,
                                                  int* __restrict__ flag, char* __restrict__ gscratch) {
  typedef GradRegion<DK, OP> R;
  constexpr bool BF = R::BF;
  constexpr bool DT_ = VAR != VAR_DECAY;
  constexpr int LK = R::LK, LT = R::LT, LC = R::LC, VS = R::VS, LV = R::LV;

  // ---- persistent LDS
  __shared__ __align__(16) OP Ks[CH * LK];
  __shared__ __align__(16) OP Ts[DT_ ? CH * LT : 1];   // T (fp32 operands: T itself)
  __shared__ __align__(16) OP TT[DT_ ? CH * LT : 1];   // T^T
  __shared__ __align__(16) OP PT[BF ? 1 : CH * LT];    // P^T (fp32 operands)
  __shared__ __align__(16) float Pf[BF ? CH * LC : 1]; // P in fp32 (bf16 operands)
  __shared__ __align__(16) OP AE[DT_ ? CH * LT : 1];   // (K K^T)_ri E_ri, strict lower
  __shared__ float Gs[CH], Gam[CH], Bs[CH], Dte[CH];
  // per-row partial sums, one row of partials per wave column (wn) or row block (wm)
  __shared__ float rowZ[2][CH], colZ[4][CH], rowA[2][CH], rqp[2][CH], rxp[2][CH], rkp[2][CH], dbYp[2][CH];
  __shared__ float hdh_w[8];
  __shared__ __align__(16) char ulds[BF ? R::bytes : 16];
  char* ub = BF ? ulds : gscratch + ((long)blockIdx.y * gridDim.x + blockIdx.x) * R::bytes;

  const int ci = blockIdx.x, h = blockIdx.y;
  const ChunkPos cp = chunk_pos(geo, ci);
  const long tile = (long)ci * H + h;
  const int w = wave_id(), l = lane_id();

  // ================= phase 0: gates, P, A, T
  OP* Qs = reinterpret_cast<OP*>(ub);
  float* As = reinterpret_cast<float*>(ub + CH * LK * sizeof(OP));
  float* Tf = BF ? As + CH * LC : reinterpret_cast<float*>(Ts);
  bool ok = load_gates<VAR>(g, beta, cp.row0, H, h, cp.len, Gs, Bs);
  load_rows<DK, LK>(q + (cp.row0 * H + h) * DK, (long)H * DK, cp.len, Qs);
  load_rows<DK, LK>(k + (cp.row0 * H + h) * DK, (long)H * DK, cp.len, Ks);
  __syncthreads();
  if (threadIdx.x < CH) {
    const int r = threadIdx.x;
    Gam[r] = expf(Gs[r]);
    Dte[r] = expf(Gs[CH - 1] - Gs[r]);
  }
  {
    Tiles<CH, CH, 4, 2> p;
    p.zero();
    p.template mma<OP, DK>(KRow<OP, LK>{Qs}, KRow<OP, LK>{Ks});
    p.each([&](int r, int i, float& x) {
      const float pr = i <= r ? x * __expf(Gs[r] - Gs[i]) : 0.f;
      if (BF) Pf[r * LC + i] = pr;
      else PT[i * LT + r] = from_f<OP>(pr);
    });
  }
  if constexpr (DT_) {
    Tiles<CH, CH, 4, 2> bm;
    bm.zero();
    bm.template mma<OP, DK>(KRow<OP, LK>{Ks}, KRow<OP, LK>{Ks});
    bm.each([&](int r, int i, float& x) {
      const float ae = (i < r) ? x * __expf(Gs[r] - Gs[i]) : 0.f;
      AE[r * LT + i] = from_f<OP>(ae);
      As[r * LC + i] = Bs[r] * ae;
    });
    __syncthreads();
    unit_lower_inverse<OP, LC, LT, false>(As, Tf, Ts, (OP*)nullptr);
    for (int idx = threadIdx.x; idx < CH * CH; idx += blockDim.x) {
      const int r = idx >> 6, c = idx & 63;
      TT[c * LT + r] = Ts[r * LT + c];
    }
  }
  __syncthreads();

  // ================= phase 1: value slices
  OP* Vs = reinterpret_cast<OP*>(ub);
  OP* dOs = Vs + CH * LV;
  OP* Rs = dOs + CH * LV;
  OP* Ups = Rs + CH * LV;
  OP* dUs = Ups + CH * LV;
  OP* Ys = dUs + CH * LV;
  OP* dVst = Ys + CH * LV;
  OP* hs = dVst + CH * LV;
  OP* dhs = hs + DK * LV;
  OP* hsT = dhs + DK * LV;
  OP* RT = hsT + VS * LK;
  OP* dUT = RT + VS * LT;

  Tiles<CH, CH, 4, 2> dT, dP;
  Tiles<CH, DK, 4, 2> X, dQa, dKh;
  dT.zero(); dP.zero(); X.zero(); dQa.zero(); dKh.zero();
  float dbY[4] = {0.f, 0.f, 0.f, 0.f};
  float hdh = 0.f;
  const float* hp = states + tile * DK * DV;
  const OP* dhp = dhg + tile * DK * DV;
  const OP* vp = v + (cp.row0 * H + h) * DV;
  const OP* dop = dO + (cp.row0 * H + h) * DV;
  OP* dvp = dvo + (cp.row0 * H + h) * DV;

  const OP* dUp = dUTg + tile * DV * CH;
  for (int c0 = 0; c0 < DV; c0 += VS) {
    ok &= load_rows<VS, LV>(vp + c0, (long)H * DV, cp.len, Vs);
    load_rows<VS, LV>(dop + c0, (long)H * DV, cp.len, dOs);
    // h slice (fp32) -> hs (d, v) and hsT (v, d); dh slice -> dhs (d, v)
    for (int idx = threadIdx.x; idx < DK * VS / 4; idx += blockDim.x) {
      const int d = idx / (VS / 4), c = (idx - d * (VS / 4)) * 4;
      const float4 hx = *reinterpret_cast<const float4*>(hp + (long)d * DV + c0 + c);
      const typename vec4_of<OP>::type dv4 = *reinterpret_cast<const typename vec4_of<OP>::type*>(dhp + (long)d * DV + c0 + c);
      const float hv[4] = {hx.x, hx.y, hx.z, hx.w};
      OP h4[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        ok &= finite_f(hv[j]);
        hdh += hv[j] * to_f(elem4<OP>(dv4, j));
        h4[j] = from_f<OP>(hv[j]);
        hsT[(c + j) * LK + d] = h4[j];
      }
      *reinterpret_cast<typename vec4_of<OP>::type*>(hs + d * LV + c) = pack4<OP>(h4);
      *reinterpret_cast<typename vec4_of<OP>::type*>(dhs + d * LV + c) = dv4;
    }
    // dU' slice from the reverse scan: dUT (v, r) and dUs (r, v)
    {
      constexpr int VE = 16 / (int)sizeof(OP);
      for (int idx = threadIdx.x; idx < VS * CH / VE; idx += blockDim.x) {
        const int vv = idx / (CH / VE), r = (idx - vv * (CH / VE)) * VE;
        const uint4 u = *reinterpret_cast<const uint4*>(dUp + (long)(c0 + vv) * CH + r);
        *reinterpret_cast<uint4*>(dUT + vv * LT + r) = u;
#pragma unroll
        for (int j = 0; j < VE; ++j) dUs[(r + j) * LV + vv] = elem16<OP>(u, j);
      }
    }
    __syncthreads();
    const OP* Up = Vs;  // U' of the scalar-decay member is V
    if constexpr (DT_) {
      // R = diag(beta) V - diag(beta e^G) K h
      Tiles<CH, VS, 4, 2> rr;
      rr.zero();
      rr.template mma<OP, DK>(KRow<OP, LK>{Ks}, KRow<OP, LK>{hsT});
      rr.each([&](int r, int vv, float& x) {
        const float rv = Bs[r] * (to_f(Vs[r * LV + vv]) - Gam[r] * x);
        const OP ro = from_f<OP>(rv);
        Rs[r * LV + vv] = ro;
        RT[vv * LT + r] = ro;
      });
      // Y = T^T dU'; dV = diag(beta) Y; dbeta_r += v_r . Y_r; keep -Y for X
      Tiles<CH, VS, 4, 2> y;
      y.zero();
      y.template mma<OP, CH>(KRow<OP, LT>{TT}, KRow<OP, LT>{dUT});
      y.each([&](int r, int vv, float& x) {
        dVst[r * LV + vv] = from_f<OP>(Bs[r] * x);
        Ys[r * LV + vv] = from_f<OP>(-x);
      });
#pragma unroll
      for (int b = 0; b < y.TN; ++b)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int r = y.m0(0) + (l >> 4) * 4 + j, vv = y.n0(b) + (l & 15);
          dbY[j] += to_f(Vs[r * LV + vv]) * y.acc[0][b][j];
        }
      __syncthreads();
      // U' = T R
      Tiles<CH, VS, 4, 2> up;
      up.zero();
      up.template mma<OP, CH>(KRow<OP, LT>{Ts}, KRow<OP, LT>{RT});
      up.each([&](int r, int vv, float& x) { Ups[r * LV + vv] = from_f<OP>(x); });
      Up = Ups;
      __syncthreads();
      dT.template mma<OP, VS>(KRow<OP, LV>{dUs}, KRow<OP, LV>{Rs});
      X.template mma<OP, VS>(KRow<OP, LV>{Ys}, KRow<OP, LV>{hs});
    }
    dP.template mma<OP, VS>(KRow<OP, LV>{dOs}, KRow<OP, LV>{Up});
    dQa.template mma<OP, VS>(KRow<OP, LV>{dOs}, KRow<OP, LV>{hs});
    dKh.template mma<OP, VS>(KRow<OP, LV>{Up}, KRow<OP, LV>{dhs});
    store_rows<VS, LV>(dvp + c0, (long)H * DV, cp.len, DT_ ? dVst : dUs);  // scalar decay: dV = dU'
    __syncthreads();
  }

  // block-wide <h, dh> in a fixed order
  hdh = wave_sum(hdh);
  if (l == 0) hdh_w[w] = hdh;
  // dbeta partial from Y: reduce over the 16 lanes of a k-group, one partial per wave column
  if constexpr (DT_) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      dbY[j] = sum16(dbY[j]);
      if ((l & 15) == 0) dbYp[w % 2][(w / 2) * 16 + (l >> 4) * 4 + j] = dbY[j];
    }
  }

  // ================= phase 2: triangular VJP and the chunk-level gradients
  OP* QT = reinterpret_cast<OP*>(ub);
  OP* KT = QT + DK * LT;
  OP* SdT = KT + DK * LT;  // dT^T, later dB + dB^T
  OP* M1 = SdT + CH * LT;
  OP* dPs = M1 + CH * LT;
  OP* dPmT = dPs + CH * LT;
  {
    constexpr int VE = 16 / (int)sizeof(OP);
    const OP* qp = q + (cp.row0 * H + h) * DK;
    for (int idx = threadIdx.x; idx < CH * DK / VE; idx += blockDim.x) {
      const int r = idx / (DK / VE), c = (idx - r * (DK / VE)) * VE;
        const uint4 qv = keep16(r < cp.len, *reinterpret_cast<const uint4*>(qp + (long)clamp_row(r, cp.len) * H * DK + c));
      const uint4 kv = *reinterpret_cast<const uint4*>(Ks + r * LK + c);
#pragma unroll
      for (int j = 0; j < VE; ++j) {
        QT[(c + j) * LT + r] = elem16<OP>(qv, j);
        KT[(c + j) * LT + r] = elem16<OP>(kv, j);
      }
    }
  }
  Tiles<CH, CH, 4, 2> zs;  // Z = dA * A + dP * P, element by element
  dP.each([&](int r, int i, float& x) {
    const float dd = i <= r ? __expf(Gs[r] - Gs[i]) : 0.f;
    const float dpm = x * dd;
    dPs[r * LT + i] = from_f<OP>(dpm);
    dPmT[i * LT + r] = from_f<OP>(dpm);
  });
#pragma unroll
  for (int a = 0; a < zs.TM; ++a)
#pragma unroll
    for (int b = 0; b < zs.TN; ++b)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = zs.m0(a) + (l >> 4) * 4 + j, i = zs.n0(b) + (l & 15);
        const float pr = BF ? Pf[r * LC + i] : to_f(PT[i * LT + r]);
        zs.acc[a][b][j] = dP.acc[a][b][j] * pr;
      }
  if constexpr (DT_) dT.each([&](int r, int c, float& x) { SdT[c * LT + r] = from_f<OP>(x); });
  __syncthreads();

  float rowA_l[1][4] = {{0.f, 0.f, 0.f, 0.f}};
  if constexpr (DT_) {
    // M1 = T^T dT
    Tiles<CH, CH, 4, 2> m1;
    m1.zero();
    m1.template mma<OP, CH>(KRow<OP, LT>{TT}, KRow<OP, LT>{SdT});
    m1.each([&](int r, int c, float& x) { M1[r * LT + c] = from_f<OP>(x); });
    __syncthreads();
    // dA = -(T^T dT) T^T, strict lower part
    Tiles<CH, CH, 4, 2> da;
    da.zero();
    da.template mma<OP, CH>(KRow<OP, LT>{M1}, KRow<OP, LT>{Ts});
#pragma unroll
    for (int a = 0; a < da.TM; ++a)
#pragma unroll
      for (int b = 0; b < da.TN; ++b)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int r = da.m0(a) + (l >> 4) * 4 + j, i = da.n0(b) + (l & 15);
          const float dA = (i < r) ? -da.acc[a][b][j] : 0.f;
          const float ae = to_f(AE[r * LT + i]);
          const float e = (i < r) ? __expf(Gs[r] - Gs[i]) : 0.f;
          zs.acc[a][b][j] += dA * Bs[r] * ae;
          rowA_l[a][j] += dA * ae;
          const float db = dA * Bs[r] * e;
          if (i < r) {
            SdT[r * LT + i] = from_f<OP>(db);
            SdT[i * LT + r] = from_f<OP>(db);
          } else if (i == r) {
            SdT[r * LT + r] = from_f<OP>(0.f);
          }
        }
  }
  // row and column sums of Z, and the row sums of dA * (K K^T) * E, in fixed order
  {
    const int wm = w / 2, wn = w % 2;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      float rs = zs.acc[0][0][j] + zs.acc[0][1][j];
      rs = sum16(rs);
      const float ra = sum16(rowA_l[0][j]);
      const int r = zs.m0(0) + (l >> 4) * 4 + j;
      if ((l & 15) == 0) {
        rowZ[wn][r] = rs;
        rowA[wn][r] = ra;
      }
    }
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      float cs = 0.f;
#pragma unroll
      for (int j = 0; j < 4; ++j) cs += zs.acc[0][b][j];
      cs = sum_groups(cs);
      if ((l >> 4) == 0) colZ[wm][zs.n0(b) + (l & 15)] = cs;
    }
  }
  __syncthreads();

  // dQ = diag(e^G) dO h^T + (dP * D) K;   row sums q_r . (dO h^T)_r, k_r . X_r, k_r . dkhat_r
  {
    float rq[4], rx[4], rk[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) rq[j] = rx[j] = rk[j] = 0.f;
#pragma unroll
    for (int b = 0; b < dQa.TN; ++b)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = dQa.m0(0) + (l >> 4) * 4 + j, d = dQa.n0(b) + (l & 15);
        const float qv = to_f(QT[d * LT + r]);
        const float kv = to_f(Ks[r * LK + d]);
        rq[j] += qv * dQa.acc[0][b][j];
        rx[j] += kv * X.acc[0][b][j];
        rk[j] += kv * dKh.acc[0][b][j];
        dQa.acc[0][b][j] *= Gam[r];
        dKh.acc[0][b][j] = Dte[r] * dKh.acc[0][b][j] + Bs[r] * Gam[r] * X.acc[0][b][j];
      }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      rq[j] = sum16(rq[j]);
      rx[j] = sum16(rx[j]);
      rk[j] = sum16(rk[j]);
      if ((l & 15) == 0) {
        const int r = dQa.m0(0) + (l >> 4) * 4 + j;
        rqp[w % 2][r] = rq[j];
        rxp[w % 2][r] = rx[j];
        rkp[w % 2][r] = rk[j];
      }
    }
  }
  dQa.template mma<OP, CH>(KRow<OP, LT>{dPs}, KRow<OP, LT>{KT});
  dKh.template mma<OP, CH>(KRow<OP, LT>{dPmT}, KRow<OP, LT>{QT});
  if constexpr (DT_) dKh.template mma<OP, CH>(KRow<OP, LT>{SdT}, KRow<OP, LT>{KT});
  __syncthreads();
  // stage dq, dk (reusing QT / KT after every product has read them)
  OP* dqst = QT;
  OP* dkst = KT;
  dQa.each([&](int r, int d, float& x) { dqst[r * LK + d] = from_f<OP>(x); });
  dKh.each([&](int r, int d, float& x) { dkst[r * LK + d] = from_f<OP>(x); });
  if (w == 0) {
    // per-row scalars (row r = lane), combined from the wave partials in a fixed order
    const int r = l;
    const float rq = rqp[0][r] + rqp[1][r], rx = rxp[0][r] + rxp[1][r];
    const float kk_r = Dte[r] * (rkp[0][r] + rkp[1][r]);  // khat_r . dkhat_r
    float x = (rowZ[0][r] + rowZ[1][r]) - (((colZ[0][r] + colZ[1][r]) + colZ[2][r]) + colZ[3][r]);
    x += Gam[r] * (rq + Bs[r] * rx);
    x -= kk_r;
    const float db = (rowA[0][r] + rowA[1][r]) + Gam[r] * rx + (dbYp[0][r] + dbYp[1][r]);
    // dG_last += e^{G_last} <h, dh> + sum_r khat_r . dkhat_r ; dg = reverse cumsum of dG
    const float kk = wave_sum(kk_r);
    float hd = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) hd += hdh_w[i];
    if (l == CH - 1) x += Gam[CH - 1] * hd + kk;
    const float dgv = wave_reverse(wave_incl_scan(wave_reverse(x)));
    if (l < cp.len) {
      const long o = (cp.row0 + l) * H + h;
      if (VAR != VAR_DELTA) dg[o] = dgv;
      if (DT_) dbeta[o] = db;
    }
  }
  __syncthreads();
  store_rows<DK, LK>(dq + (cp.row0 * H + h) * DK, (long)H * DK, cp.len, dqst);
  store_rows<DK, LK>(dk + (cp.row0 * H + h) * DK, (long)H * DK, cp.len, dkst);
  const int bad = __syncthreads_or(!ok);
  if (threadIdx.x == 0) flag[tile] = bad;
}

// ---------------------------------------------------------------------------
// Chunk gradients for bf16 operands.  One block of 8 waves per (chunk, head);
// the value dimension is covered in slices of up to 128 columns (one slice for
// d_v <= 128).  Compared with the generic kernel above:
//   * the solve's VJP is taken in its short form: with U' = T R and
//     Y = T^T dU', the gradient of A = diag(beta)(K K^T * E) is -Y U'^T
//     (strict lower part), so no dT and no 64^3 products are needed;
//   * every operand that is already laid out for a fragment load in HBM (the
//     chunk state h in both orientations, dh, dU'^T, v) goes straight from
//     global memory into registers, issued at kernel entry or one step ahead,
//     instead of through LDS transposes;
//   * the 64 x d_k results (dQ, dK and X = -Y h^T) are accumulated transposed,
//     d along the tile rows, so their row sums over d are mostly in-lane and
//     the K^T, Q^T operands are read straight from the row-major tiles;
//   * the decay mask D (E is its strict lower part) is formed once and kept
//     in registers next to P and A for the phase that needs it again.
// ---------------------------------------------------------------------------
template <int DK, int DV>
struct GradBF {
  static constexpr int VS = DV > 128 ? 128 : DV;
  // waves per block: 16 with one value slice (four per SIMD, to hide the
  // phases' dependency chains), 8 with two (whose operands need more registers)
  static constexpr int NW = DV <= 128 ? 16 : 8, NT = 64 * NW;
  static constexpr int LK = DK + 8, LT = CH + 8, LC = CH + 4, LV = VS + 8;
  static constexpr int WMd = DK / 16, WNr = NW / WMd;  // waves along d and along r of the d x 64 results
  static constexpr int WNv = VS / 16, WMv = NW / WNv;
  static constexpr int WMc = 4, WNc = NW / 4;          // waves along the rows and columns of 64 x 64 results
  typedef Tiles<DK, CH, WMd, WNr> TD;  // X^T, dQ^T, dK^T: d x 64
  typedef Tiles<VS, CH, WNv, WMv> TY;  // Y^T, U'^T, (K h)^T: VS x 64
  typedef Tiles<CH, CH, WMc, WNc> TC;  // P, A, dP, dA
  static constexpr int PH1 = 4 * CH * LV * 2;
  static constexpr int PH2 = 2 * CH * LT * 2 > 2 * CH * LK * 2 ? 2 * CH * LT * 2 : 2 * CH * LK * 2;
  static constexpr int UB = PH1 > PH2 ? PH1 : PH2;
};

__device__ __forceinline__ bf16x8 cvt8(const float (&x)[8]) {
  bf16x8 r;
#pragma unroll
  for (int j = 0; j < 8; ++j) r[j] = from_f<bf16>(x[j]);
  return r;
}

#ifdef GDN_TILE_LOOP
template <int DK, int DV, int VAR>
__global__ __launch_bounds__(DV <= 128 ? 1024 : 512) void k_grad_bf(Geo geo, int H, int ntiles, const bf16* __restrict__ q,
                                                 const bf16* __restrict__ k, const bf16* __restrict__ v,
                                                 const float* __restrict__ g, const float* __restrict__ beta,
                                                 const float* __restrict__ states, const bf16* __restrict__ dO,
                                                 const bf16* __restrict__ dhg, const bf16* __restrict__ dUTg,
                                                 const bf16* __restrict__ Tg, bf16* __restrict__ dq, bf16* __restrict__ dk,
                                                 bf16* __restrict__ dvo, float* __restrict__ dg,
                                                 float* __restrict__ dbeta, int* __restrict__ flag) {
  typedef GradBF<DK, DV> C;
  typedef typename C::TD TD;
  typedef typename C::TY TY;
  typedef typename C::TC TC;
  typedef Mma<bf16> M;
  constexpr bool DT_ = VAR != VAR_DECAY;
  constexpr int VS = C::VS, LK = C::LK, LT = C::LT, LC = C::LC, LV = C::LV;
  constexpr int NW = C::NW, NT = C::NT;
  static_assert(NT == (DV <= 128 ? 1024 : 512), "launch bounds");
  // 16-byte pieces of a dO slice, of q (or k) and of T; each thread takes
  // every NT-th (threads past the end repeat the last piece: same value, same place)
  constexpr int PDO = CH * VS / 8, PQK = CH * DK / 8, PT = CH * CH / 8;
  constexpr int NDO = (PDO + NT - 1) / NT, NQK = (PQK + NT - 1) / NT;
  static_assert(PT <= NT, "one piece of T per thread");
  // With one value slice the chunk state h is read from HBM once, a tile
  // ahead, in the row-fragment layout of X^T and dQ^T; phase 0 stores it in
  // LDS as bf16, and (K h)^T takes its h^T fragments from there with
  // transposing reads.  With two slices both layouts are loaded per slice.
  constexpr bool HL = DV <= VS;
  constexpr int LH = VS + 8;
  // with one slice, the waves that share a block of d rows split its 32-column
  // steps s = wr, wr + WNr, ... (wr = the wave's column index) for the load of h
  constexpr int SH = HL ? (VS / 32 + C::WNr - 1) / C::WNr : VS / 32;

  __shared__ __align__(16) bf16 Qs[CH * LK];
  __shared__ __align__(16) bf16 Ks[CH * LK];
  __shared__ __align__(16) bf16 Ts[CH * LT];  // T (the identity for the scalar-decay member)
  __shared__ __align__(16) float Gs[CH];
  __shared__ __align__(16) float Gam[CH];
  __shared__ __align__(16) float Bs[CH];
  __shared__ __align__(16) float Dte[CH];
  __shared__ float rowZ[C::WNc][CH], colZ[C::WMc][CH], rowA[C::WNc][CH];
  __shared__ float rqp[C::WMd][CH], rxp[C::WMd][CH], rkp[C::WMd][CH], dbYp[C::WNv][CH];
  __shared__ float hdh_w[NW];
  __shared__ __align__(16) char ub[C::UB];
  __shared__ __align__(16) bf16 Hs[HL ? DK * LH : 8];
  // with two slices, P and (K K^T) * E wait in LDS from phase 0 to phase 2 (one
  // column per thread, 2 * TN * 4 entries each), keeping phase 1 within 256 VGPRs
  constexpr int NSTASH = HL ? 1 : 2 * TC::TN * 4;
  __shared__ float stash[NSTASH][HL ? 1 : NT];

  // the loop-safe thread index reads this word: it is stored before any use
  if (threadIdx.x == 0) gdn_tid_bias = 0;
  __syncthreads();
  const int rsv = H * DV;  // row strides (elements) of v, dO, dv and of q, k, dq, dk
  const int rsk = H * DK;

  // one (chunk, head) tile
  struct Tile {
    ChunkPos cp;
    int h;
    long t;
  };
  auto tile_at = [&](int t) {
    Tile x;
    const int ci = t / H;
    x.h = t - ci * H;
    x.t = t;
    x.cp = chunk_pos(geo, ci);
    return x;
  };

  // ---- operands loaded ahead of their use: a tile's q, k, T and raw gates
  // (during the previous tile's last phase), and the value-slice operands
  // (at the start of the tile, or a slice ahead)
  struct Pre0 {
    uint4 qk[2][NQK];  // q and k rows, masked at use
    uint4 tq;          // 8 entries of T: row (thread index) / 8
    float gv, bv;      // gate and beta of row l (wave 0 uses them), masked at use
  };
  struct PreA {
    uint4 dov[NDO];                      // dO slice, staged to LDS
    bf16x8 du[CH / 32][TY::TM];          // dU'^T rows: A fragments of Y^T
    bf16x8 hk[DK / 32][TY::TM];          // h^T: A fragments of (K h)^T (two slices only)
    uint2 vb[TY::TM][TY::TN];            // v[r][v0..v0+3] in the Y^T accumulator layout
  };
  struct PreB {
    float hx[SH][TD::TM][8];             // h (with one slice: this wave's steps only)
    bf16x8 dh[VS / 32][TD::TM];          // dh: A fragments of dK^T
  };
  auto load_0 = [&](Pre0& p, const Tile& x) {
    const int l = lane_id(), len = x.cp.len;
    const bf16* qp = q + (x.cp.row0 * H + x.h) * DK;
    const bf16* kp = k + (x.cp.row0 * H + x.h) * DK;
#pragma unroll
    for (int t = 0; t < NQK; ++t) {
      const int idx = min(thread_x() + t * NT, PQK - 1), r = idx / (DK / 8), c = (idx - r * (DK / 8)) * 8;
      const unsigned ro = row_off(clamp_row(r, len), rsk) + c;
      p.qk[0][t] = *reinterpret_cast<const uint4*>(qp + ro);
      p.qk[1][t] = *reinterpret_cast<const uint4*>(kp + ro);
    }
    p.tq = uint4{0u, 0u, 0u, 0u};
    if constexpr (DT_) p.tq = *reinterpret_cast<const uint4*>(Tg + x.t * CH * CH + min(thread_x(), PT - 1) * 8);
    const long o = (x.cp.row0 * H + x.h) + row_off(clamp_row(l, len), H);
    p.gv = 0.f;
    p.bv = 0.f;
    if constexpr (VAR != VAR_DELTA) p.gv = g[o];
    if constexpr (VAR != VAR_DECAY) p.bv = beta[o];
  };
  // dO, dU'^T and v of a value slice
  auto load_a1 = [&](PreA& p, const Tile& x, int c0) {
    const int l = lane_id(), lg = l >> 4, lc = l & 15, len = x.cp.len;
    const bf16* dop = dO + (x.cp.row0 * H + x.h) * DV;
    const bf16* dUp = dUTg + x.t * DV * CH;
    const bf16* vp = v + (x.cp.row0 * H + x.h) * DV;
#pragma unroll
    for (int t = 0; t < NDO; ++t) {
      const int idx = min(thread_x() + t * NT, PDO - 1), r = idx / (VS / 8), c = (idx - r * (VS / 8)) * 8;
      p.dov[t] = *reinterpret_cast<const uint4*>(dop + row_off(clamp_row(r, len), rsv) + c0 + c);  // masked at use
    }
#pragma unroll
    for (int s = 0; s < CH / 32; ++s)
#pragma unroll
      for (int a = 0; a < TY::TM; ++a)
        p.du[s][a] = *reinterpret_cast<const bf16x8*>(dUp + op_off<bf16, CH>(c0 + TY::m0(a), 32 * s) + l * 8);
    if constexpr (DT_) {
#pragma unroll
      for (int a = 0; a < TY::TM; ++a)
#pragma unroll
        for (int b = 0; b < TY::TN; ++b) {
          const int r = TY::n0(b) + lc;
          // masked at use
          p.vb[a][b] = *reinterpret_cast<const uint2*>(vp + row_off(clamp_row(r, len), rsv) + c0 + TY::m0(a) + 4 * lg);
        }
    }
  };
  // h^T of a value slice, in bf16 (loaded right before its product: the fp32
  // values are held only until they are converted)
  auto load_a2 = [&](PreA& p, const Tile& x, int c0) {
    const int l = lane_id(), lg = l >> 4, lc = l & 15;
    const float* hp = states + x.t * DK * DV;
    if constexpr (DT_) {
#pragma unroll
      for (int s = 0; s < DK / 32; ++s)
#pragma unroll
        for (int a = 0; a < TY::TM; ++a) {
          float f[8];
#pragma unroll
          for (int j = 0; j < 8; ++j) f[j] = hp[(32 * s + 8 * lg + j) * DV + c0 + TY::m0(a) + lc];
          p.hk[s][a] = cvt8(f);
        }
    }
  };
  auto load_h = [&](PreB& p, const Tile& x, int c0) {
    const int l = lane_id(), lg = l >> 4, lc = l & 15;
    const float* hp = states + x.t * DK * DV;
#pragma unroll
    for (int s = 0; s < VS / 32; ++s)
#pragma unroll
      for (int a = 0; a < TD::TM; ++a) {
        const float* src = hp + (TD::m0(a) + lc) * DV + c0 + 32 * s + 8 * lg;
        const float4 x0 = *reinterpret_cast<const float4*>(src);
        const float4 x1 = *reinterpret_cast<const float4*>(src + 4);
        p.hx[s][a][0] = x0.x; p.hx[s][a][1] = x0.y; p.hx[s][a][2] = x0.z; p.hx[s][a][3] = x0.w;
        p.hx[s][a][4] = x1.x; p.hx[s][a][5] = x1.y; p.hx[s][a][6] = x1.z; p.hx[s][a][7] = x1.w;
      }
  };
  // with one slice: step s = wr + WNr i of this wave's rows (clamped: a wave
  // without an i-th step repeats its last one and skips it at use)
  auto load_hs = [&](PreB& p, const Tile& x) {
    const int l = lane_id(), lg = l >> 4, lc = l & 15, wr = wave_id() % C::WNr;
    const float* hp = states + x.t * DK * DV;
#pragma unroll
    for (int i = 0; i < SH; ++i) {
      const int st = min(wr + C::WNr * i, VS / 32 - 1);
#pragma unroll
      for (int a = 0; a < TD::TM; ++a) {
        const float* src = hp + (TD::m0(a) + lc) * DV + 32 * st + 8 * lg;
        const float4 x0 = *reinterpret_cast<const float4*>(src);
        const float4 x1 = *reinterpret_cast<const float4*>(src + 4);
        p.hx[i][a][0] = x0.x; p.hx[i][a][1] = x0.y; p.hx[i][a][2] = x0.z; p.hx[i][a][3] = x0.w;
        p.hx[i][a][4] = x1.x; p.hx[i][a][5] = x1.y; p.hx[i][a][6] = x1.z; p.hx[i][a][7] = x1.w;
      }
    }
  };
  auto load_dh = [&](PreB& p, const Tile& x, int c0) {
    const int l = lane_id();
    const bf16* dhp = dhg + x.t * DK * DV;
#pragma unroll
    for (int s = 0; s < VS / 32; ++s)
#pragma unroll
      for (int a = 0; a < TD::TM; ++a)
        p.dh[s][a] = *reinterpret_cast<const bf16x8*>(dhp + op_off<bf16, DV>(TD::m0(a), c0 + 32 * s) + l * 8);
  };
  auto load_b = [&](PreB& p, const Tile& x, int c0) {
    if constexpr (HL) load_hs(p, x); else load_h(p, x, c0);
    load_dh(p, x, c0);
  };

  // Persistent: the block walks the tiles t = blockIdx.x, blockIdx.x + gridDim.x,
  // ... (the grid never exceeds the tile count), so the next tile's operands
  // load while this one's last phase runs.
  Tile cur = tile_at(blockIdx.x);
  Pre0 p0;
  PreA pa;
  PreB pb;
  load_0(p0, cur);
  load_a1(pa, cur, 0);
  if constexpr (HL) load_b(pb, cur, 0);
  for (int tt = blockIdx.x; tt < ntiles; tt += gridDim.x) {
  const int w = wave_id(), l = lane_id(), lg = l >> 4, lc = l & 15;
  const ChunkPos cp = cur.cp;
  const int h = cur.h, len = cp.len;
  const long tile = cur.t;
  const bf16* vp = v + (cp.row0 * H + h) * DV;
  bf16* dvp = dvo + (cp.row0 * H + h) * DV;
  bool ok = true;
  float hdh = 0.f;  // <h, dh> over this wave's part of the state

  // ================= phase 0: gates, P, A; T comes from the prep kernel
#pragma unroll
  for (int t = 0; t < NQK; ++t) {
    const int idx = min(thread_x() + t * NT, PQK - 1), r = idx / (DK / 8), c = (idx - r * (DK / 8)) * 8;
    *reinterpret_cast<uint4*>(Qs + r * LK + c) = keep16(r < len, p0.qk[0][t]);
    *reinterpret_cast<uint4*>(Ks + r * LK + c) = keep16(r < len, p0.qk[1][t]);
  }
  {
    const int pc = min(thread_x(), PT - 1), r = pc >> 3, c = (pc & 7) * 8;
    uint4 tq = p0.tq;
    if constexpr (!DT_) {
      bf16 e[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) e[j] = from_f<bf16>(c + j == r ? 1.f : 0.f);
      tq = pack16<bf16>(e);
    }
    *reinterpret_cast<uint4*>(Ts + r * LT + c) = tq;
  }
  if constexpr (HL) {
    // h -> LDS in bf16; <h, dh> takes the fp32 values (and checks them: a
    // non-finite element of h makes the sum non-finite).  Each wave does its
    // own 32-column steps of its rows.
    // (register arrays indexed by compile-time steps under a wave-uniform test)
    const int wr = w % C::WNr;
#pragma unroll
    for (int i = 0; i < SH; ++i)
#pragma unroll
      for (int st = 0; st < VS / 32; ++st) {
        if (st != wr + C::WNr * i) continue;
#pragma unroll
        for (int a = 0; a < TD::TM; ++a) {
          *reinterpret_cast<bf16x8*>(Hs + (TD::m0(a) + lc) * LH + 32 * st + 8 * lg) = cvt8(pb.hx[i][a]);
#pragma unroll
          for (int j = 0; j < 8; ++j) hdh += pb.hx[i][a][j] * to_f(pb.dh[st][a][j]);
        }
      }
  }
  if (w == 0) {
    // in-chunk gates: G = inclusive cumsum of g (0 past the end), beta (0 past
    // the end), e^{G_r} and e^{G_last - G_r}
    const float gv = l < len ? p0.gv : 0.f, bv = l < len ? p0.bv : 0.f;
    ok &= finite_f(gv) && finite_f(bv);
    const float gc = wave_incl_scan(gv);
    Gs[l] = gc;
    Bs[l] = bv;
    Gam[l] = __expf(gc);
    Dte[l] = __expf(shfl_idx(gc, CH - 1) - gc);
  }
  __syncthreads();
  // the next tile (this one again on the last pass: a clamped, unconditional
  // prefetch keeps the registers loop-carried).  With one slice, q, k, T and
  // the gates are in LDS now, and their next copies load from here on.
  const Tile nxt = tile_at(tt + (int)gridDim.x < ntiles ? tt + (int)gridDim.x : tt);
  if constexpr (HL) load_0(p0, nxt);
  TC pm, ae;  // P = (Q K^T) * D and (K K^T) * E, kept for phase 2
  float dd[TC::TN][4];  // D_ri = e^{G_r - G_i} for i <= r, else 0
  pm.zero();
  pm.template mma<bf16, DK>(KRow<bf16, LK>{Qs}, KRow<bf16, LK>{Ks});
#pragma unroll
  for (int b = 0; b < TC::TN; ++b)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = TC::m0(0) + 4 * lg + j, i = TC::n0(b) + lc;
      dd[b][j] = i <= r ? __expf(Gs[r] - Gs[i]) : 0.f;
      pm.acc[0][b][j] *= dd[b][j];
    }
  if constexpr (DT_) {
    ae.zero();
    ae.template mma<bf16, DK>(KRow<bf16, LK>{Ks}, KRow<bf16, LK>{Ks});
#pragma unroll
    for (int b = 0; b < TC::TN; ++b)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = TC::m0(0) + 4 * lg + j, i = TC::n0(b) + lc;
        ae.acc[0][b][j] = i < r ? ae.acc[0][b][j] * dd[b][j] : 0.f;
      }
  }
  if constexpr (!HL) {
#pragma unroll
    for (int b = 0; b < TC::TN; ++b)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        stash[b * 4 + j][thread_x()] = pm.acc[0][b][j];
        stash[TC::TN * 4 + b * 4 + j][thread_x()] = DT_ ? ae.acc[0][b][j] : 0.f;
      }
  }

  // ================= phase 1: value slices
  bf16* Rs = reinterpret_cast<bf16*>(ub);  // R, row-major
  bf16* Ys = Rs + CH * LV;
  bf16* Ups = Ys + CH * LV;
  bf16* dOs = Ups + CH * LV;
  TC dA, dP;
  TD Xt, dQt, dKt;  // X^T = -h Y^T, dQ^T (from dO h^T), dK^T (from U' dh^T)
  dA.zero(); dP.zero(); Xt.zero(); dQt.zero(); dKt.zero();
  float dbY[TY::TN];
#pragma unroll
  for (int b = 0; b < TY::TN; ++b) dbY[b] = 0.f;

  for (int c0 = 0; c0 < DV; c0 += VS) {
    if (c0 > 0) {
      __syncthreads();  // the previous slice's LDS operands are consumed
      load_a1(pa, cur, c0);
    }
    if constexpr (!HL) load_a2(pa, cur, c0);
    if constexpr (DT_) {
      // R = diag(beta) (V - diag(e^G) K h), computed transposed, (K h)^T = h^T K^T,
      // so that a lane needs v[r][v0..v0+3] as one 8-byte piece (the same
      // piece the dbeta term uses) and writes four values of a row of R
      TY kht;
      kht.zero();
#pragma unroll
      for (int s = 0; s < DK / 32; ++s) {
        bf16x8 fa[TY::TM];
#pragma unroll
        for (int a = 0; a < TY::TM; ++a) {
          if constexpr (HL) fa[a] = lds_frag_tr<LH>(Hs, TY::m0(a), 32 * s);
          else fa[a] = pa.hk[s][a];
        }
#pragma unroll
        for (int b = 0; b < TY::TN; ++b) {
          const bf16x8 fb = M::load(KRow<bf16, LK>{Ks}, TY::n0(b), 32 * s);
#pragma unroll
          for (int a = 0; a < TY::TM; ++a) kht.acc[a][b] = M::mma(fa[a], fb, kht.acc[a][b]);
        }
      }
      if constexpr (!HL) load_b(pb, cur, c0);
#pragma unroll
      for (int b = 0; b < TY::TN; ++b) {
        const int r = TY::n0(b) + lc;
        const float br = Bs[r], gr = Gam[r];
#pragma unroll
        for (int a = 0; a < TY::TM; ++a) {
          const int v0 = TY::m0(a) + 4 * lg;
          bf16 r4[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            // (v is checked through the dbeta partial sum v . Y below)
            const float vx = r < len ? to_f(elem4<bf16>(pa.vb[a][b], j)) : 0.f;
            r4[j] = from_f<bf16>(br * (vx - gr * kht.acc[a][b][j]));
          }
          *reinterpret_cast<uint2*>(Rs + r * LV + v0) = pack4<bf16>(r4);
        }
      }
    } else {
      if constexpr (!HL) load_b(pb, cur, c0);
    }
    // Y^T = dU'^T T, so Y = T^T dU'.  dV = diag(beta) Y; keep -Y for dA and X
    {
      TY yt;
      yt.zero();
#pragma unroll
      for (int s = 0; s < CH / 32; ++s) {
        bf16x8 fb[TY::TN];
#pragma unroll
        for (int b = 0; b < TY::TN; ++b) fb[b] = M::load(KColTr<LT>{Ts, nullptr}, TY::n0(b), 32 * s);
#pragma unroll
        for (int a = 0; a < TY::TM; ++a)
#pragma unroll
          for (int b = 0; b < TY::TN; ++b) yt.acc[a][b] = M::mma(pa.du[s][a], fb[b], yt.acc[a][b]);
      }
#pragma unroll
      for (int b = 0; b < TY::TN; ++b) {
        const int r = TY::n0(b) + lc;
        const float br = DT_ ? Bs[r] : 1.f;
#pragma unroll
        for (int a = 0; a < TY::TM; ++a) {
          const int v0 = TY::m0(a) + 4 * lg;
          bf16 d4[4], y4[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const float y = yt.acc[a][b][j];
            d4[j] = from_f<bf16>(br * y);
            y4[j] = from_f<bf16>(-y);
            if (DT_) dbY[b] += (r < len ? to_f(elem4<bf16>(pa.vb[a][b], j)) : 0.f) * y;
          }
          if (r < len) *reinterpret_cast<uint2*>(dvp + row_off(r, rsv) + c0 + v0) = pack4<bf16>(d4);
          if (DT_) *reinterpret_cast<uint2*>(Ys + r * LV + v0) = pack4<bf16>(y4);
        }
      }
    }
#pragma unroll
    for (int t = 0; t < NDO; ++t) {
      const int idx = min(thread_x() + t * NT, PDO - 1), r = idx / (VS / 8), c = (idx - r * (VS / 8)) * 8;
      *reinterpret_cast<uint4*>(dOs + r * LV + c) = keep16(r < len, pa.dov[t]);
    }
    if constexpr (!DT_) {
      // the scalar-decay member has U' = V
      for (int idx = thread_x(); idx < CH * VS / 8; idx += blockDim.x) {
        const int r = idx / (VS / 8), c = (idx - r * (VS / 8)) * 8;
        const uint4 u = keep16(r < len, *reinterpret_cast<const uint4*>(vp + row_off(clamp_row(r, len), rsv) + c0 + c));
        ok &= finite16B<bf16>(u);
        *reinterpret_cast<uint4*>(Ups + r * LV + c) = u;
      }
    }
    __syncthreads();
    if constexpr (DT_) {
      // U'^T = R^T T^T
      TY ut;
      ut.zero();
      ut.template mma<bf16, CH>(KColTr<LV>{Rs, nullptr}, KRow<bf16, LT>{Ts});
#pragma unroll
      for (int a = 0; a < TY::TM; ++a)
#pragma unroll
        for (int b = 0; b < TY::TN; ++b) {
          bf16 u4[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) u4[j] = from_f<bf16>(ut.acc[a][b][j]);
          *reinterpret_cast<uint2*>(Ups + (TY::n0(b) + lc) * LV + TY::m0(a) + 4 * lg) = pack4<bf16>(u4);
        }
      __syncthreads();
      dA.template mma<bf16, VS>(KRow<bf16, LV>{Ys}, KRow<bf16, LV>{Ups});  // -Y U'^T
    }
    dP.template mma<bf16, VS>(KRow<bf16, LV>{dOs}, KRow<bf16, LV>{Ups});
#pragma unroll
    for (int s = 0; s < VS / 32; ++s) {
      bf16x8 fh[TD::TM];
#pragma unroll
      for (int a = 0; a < TD::TM; ++a) {
        if constexpr (HL) {
          fh[a] = M::load(KRow<bf16, LH>{Hs}, TD::m0(a), 32 * s);
        } else {
          fh[a] = cvt8(pb.hx[s][a]);
#pragma unroll
          for (int j = 0; j < 8; ++j) ok &= finite_f(pb.hx[s][a][j]);
          if (TD::n0(0) == 0) {  // one wave column adds <h, dh> for its rows
#pragma unroll
            for (int j = 0; j < 8; ++j) hdh += pb.hx[s][a][j] * to_f(pb.dh[s][a][j]);
          }
        }
      }
#pragma unroll
      for (int b = 0; b < TD::TN; ++b) {
        const bf16x8 fo = M::load(KRow<bf16, LV>{dOs}, TD::n0(b), 32 * s);
        const bf16x8 fu = M::load(KRow<bf16, LV>{Ups}, TD::n0(b), 32 * s);
#pragma unroll
        for (int a = 0; a < TD::TM; ++a) {
          dQt.acc[a][b] = M::mma(fh[a], fo, dQt.acc[a][b]);
          dKt.acc[a][b] = M::mma(pb.dh[s][a], fu, dKt.acc[a][b]);
        }
        if constexpr (DT_) {
          const bf16x8 fy = M::load(KRow<bf16, LV>{Ys}, TD::n0(b), 32 * s);
#pragma unroll
          for (int a = 0; a < TD::TM; ++a) Xt.acc[a][b] = M::mma(fh[a], fy, Xt.acc[a][b]);
        }
      }
    }
  }

  hdh = wave_sum(hdh);
  if (l == 0) hdh_w[w] = hdh;
  // A non-finite element of h (or of dh) leaves <h, dh> non-finite; so does
  // one of v in v . Y (Inf times 0 is NaN).  An overflow of the sums alone
  // flags the stream as well, which only sends it to the exact path.
  if constexpr (HL) ok &= finite_f(hdh);
  if constexpr (DT_) {
    // dbeta partial v_r . Y_r: over the 4 lane groups, then one partial per wave row of Y^T
#pragma unroll
    for (int b = 0; b < TY::TN; ++b) {
      const float s = sum_groups(dbY[b]);
      ok &= finite_f(s);
      if (lg == 0) dbYp[w / C::WMv][TY::n0(b) + lc] = s;
    }
  }
  __syncthreads();  // phase-1 LDS operands are consumed
  // the next tile's value-slice operands.  With two slices (fewer waves, more
  // accumulators per wave) they, and the next q, k, T and gates, wait until
  // phase 2's accumulators are in LDS, so no register is held through phase 2.
  if constexpr (HL) load_a1(pa, nxt, 0);

  // ================= phase 2: the chunk-level gradients
  bf16* dPmT = reinterpret_cast<bf16*>(ub);  // (dP * D)^T
  bf16* dBT = dPmT + CH * LT;                 // dB^T, dB = dA * beta_r * E (strict lower)
  if constexpr (!HL) {
    // this thread's own entries (no other thread writes them)
#pragma unroll
    for (int b = 0; b < TC::TN; ++b)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        pm.acc[0][b][j] = stash[b * 4 + j][thread_x()];
        ae.acc[0][b][j] = stash[TC::TN * 4 + b * 4 + j][thread_x()];
        // the decay mask is formed again rather than held through phase 1
        const int r = TC::m0(0) + 4 * lg + j, i = TC::n0(b) + lc;
        dd[b][j] = i <= r ? __expf(Gs[r] - Gs[i]) : 0.f;
      }
  }
  TC zs;  // Z = dA * A + dP * P
  float rowA_l[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int b = 0; b < TC::TN; ++b) {
    const int i = TC::n0(b) + lc, r0 = TC::m0(0) + 4 * lg;
    bf16 pt4[4], bt4[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = r0 + j;
      const float dpm = dP.acc[0][b][j] * dd[b][j];
      pt4[j] = from_f<bf16>(dpm);
      float z = dP.acc[0][b][j] * pm.acc[0][b][j];
      if constexpr (DT_) {
        const float da = i < r ? dA.acc[0][b][j] : 0.f;
        z += da * Bs[r] * ae.acc[0][b][j];
        rowA_l[j] += da * ae.acc[0][b][j];
        bt4[j] = from_f<bf16>(da * Bs[r] * dd[b][j]);
      }
      zs.acc[0][b][j] = z;
    }
    // both written transposed, four consecutive r per lane; every entry of
    // the 64 x 64 tiles is written by exactly one lane
    *reinterpret_cast<uint2*>(dPmT + i * LT + r0) = pack4<bf16>(pt4);
    if constexpr (DT_) *reinterpret_cast<uint2*>(dBT + i * LT + r0) = pack4<bf16>(bt4);
  }
  {
    const int wm = w / C::WNc, wn = w % C::WNc;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      float zr = zs.acc[0][0][j];
#pragma unroll
      for (int b = 1; b < TC::TN; ++b) zr += zs.acc[0][b][j];
      const float rs = sum16(zr);
      const float ra = sum16(rowA_l[j]);
      const int r = TC::m0(0) + 4 * lg + j;
      if (lc == 0) {
        rowZ[wn][r] = rs;
        rowA[wn][r] = ra;
      }
    }
#pragma unroll
    for (int b = 0; b < TC::TN; ++b) {
      float cs = 0.f;
#pragma unroll
      for (int j = 0; j < 4; ++j) cs += zs.acc[0][b][j];
      cs = sum_groups(cs);
      if (lg == 0) colZ[wm][TC::n0(b) + lc] = cs;
    }
  }
  // row sums q_r . (dO h^T)_r, k_r . X_r, k_r . (U' dh^T)_r (over d: in-lane over
  // four d, then over the lane groups, then one partial per wave row), then the
  // per-row scalings
  {
    const int wd = w / C::WNr;
#pragma unroll
    for (int b = 0; b < TD::TN; ++b) {
      const int r = TD::n0(b) + lc;
      float rq = 0.f, rx = 0.f, rk = 0.f;
#pragma unroll
      for (int a = 0; a < TD::TM; ++a) {
        const int d0 = TD::m0(a) + 4 * lg;
        const uint2 q4 = *reinterpret_cast<const uint2*>(Qs + r * LK + d0);
        const uint2 k4 = *reinterpret_cast<const uint2*>(Ks + r * LK + d0);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float qv = to_f(elem4<bf16>(q4, j)), kv = to_f(elem4<bf16>(k4, j));
          rq += qv * dQt.acc[a][b][j];
          rx += kv * Xt.acc[a][b][j];
          rk += kv * dKt.acc[a][b][j];
        }
      }
      rq = sum_groups(rq);
      rx = sum_groups(rx);
      rk = sum_groups(rk);
      if (lg == 0) {
        rqp[wd][r] = rq;
        rxp[wd][r] = rx;
        rkp[wd][r] = rk;
      }
      const float gr = Gam[r], er = Dte[r], bgr = DT_ ? Bs[r] * gr : 0.f;
#pragma unroll
      for (int a = 0; a < TD::TM; ++a)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          dQt.acc[a][b][j] *= gr;
          dKt.acc[a][b][j] = er * dKt.acc[a][b][j] + bgr * Xt.acc[a][b][j];
        }
    }
  }
  __syncthreads();
  {
    // dQ^T += K^T (dP * D)^T,  dK^T += Q^T (dP * D) + K^T (dB + dB^T); the K^T and
    // Q^T fragments are read down the columns of the row-major tiles, and the
    // transposed tiles are read both ways (rows, or columns by the transposing load)
    typename TD::template AFr<bf16, CH> kt;
    kt.load(KColTr<LK>{Ks, nullptr});
    dQt.template mma<bf16, CH>(kt, KColTr<LT>{dPmT, nullptr});
    if constexpr (DT_) {
      dKt.template mma<bf16, CH>(kt, KRow<bf16, LT>{dBT});
      dKt.template mma<bf16, CH>(kt, KColTr<LT>{dBT, nullptr});
    }
    dKt.template mma<bf16, CH>(KColTr<LK>{Qs, nullptr}, KRow<bf16, LT>{dPmT});
  }
  __syncthreads();
  bf16* dqst = reinterpret_cast<bf16*>(ub);
  bf16* dkst = dqst + CH * LK;
#pragma unroll
  for (int a = 0; a < TD::TM; ++a)
#pragma unroll
    for (int b = 0; b < TD::TN; ++b) {
      const int r = TD::n0(b) + lc, d0 = TD::m0(a) + 4 * lg;
      bf16 q4[4], k4[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        q4[j] = from_f<bf16>(dQt.acc[a][b][j]);
        k4[j] = from_f<bf16>(dKt.acc[a][b][j]);
      }
      *reinterpret_cast<uint2*>(dqst + r * LK + d0) = pack4<bf16>(q4);
      *reinterpret_cast<uint2*>(dkst + r * LK + d0) = pack4<bf16>(k4);
    }
  // the accumulators are free: the next tile's h and dh (with two slices: q, k,
  // T, gates and the first slice's dO, dU'^T and v)
  if constexpr (HL) {
    load_b(pb, nxt, 0);
  } else {
    load_0(p0, nxt);
    load_a1(pa, nxt, 0);
  }
  __syncthreads();
  if (w == 0) {
    // dg (reverse cumsum of dG) and dbeta, while the other waves store dq, dk
    const int r = l;
    float rq = 0.f, rx = 0.f, rk = 0.f;
#pragma unroll
    for (int i = 0; i < C::WMd; ++i) {
      rq += rqp[i][r];
      rx += rxp[i][r];
      rk += rkp[i][r];
    }
    // dO is first read in full by this kernel: a NaN or Inf in row r of dO
    // makes every entry of row r of dO h^T non-finite (Inf times 0 is NaN), and
    // with it q_r . (dO h^T)_r, so that sum flags it
    ok &= finite_f(rq);
    float dbv = 0.f;
#pragma unroll
    for (int i = 0; i < C::WNv; ++i) dbv += dbYp[i][r];
    const float kk_r = Dte[r] * rk;  // khat_r . dkhat_r
    float zr = rowZ[0][r], zc = colZ[0][r], ra = rowA[0][r];
#pragma unroll
    for (int i = 1; i < C::WNc; ++i) {
      zr += rowZ[i][r];
      ra += rowA[i][r];
    }
#pragma unroll
    for (int i = 1; i < C::WMc; ++i) zc += colZ[i][r];
    float x = zr - zc;
    x += Gam[r] * (rq + Bs[r] * rx);
    x -= kk_r;
    const float db = ra + Gam[r] * rx + dbv;
    const float kk = wave_sum(kk_r);
    float hd = 0.f;
#pragma unroll
    for (int i = 0; i < NW; ++i) hd += hdh_w[i];
    if (l == CH - 1) x += Gam[CH - 1] * hd + kk;
    const float dgv = wave_reverse(wave_incl_scan(wave_reverse(x)));
    if (l < len) {
      const long o = (cp.row0 * H + h) + row_off(l, H);
      if (VAR != VAR_DELTA) dg[o] = dgv;
      if (DT_) dbeta[o] = db;
    }
  }
  store_rows<DK, LK>(dq + (cp.row0 * H + h) * DK, rsk, len, dqst);
  store_rows<DK, LK>(dk + (cp.row0 * H + h) * DK, rsk, len, dkst);
  if (threadIdx.x == 0) gdn_tid_bias = 0;  // a new pass: index arithmetic is recomputed
  const int bad = __syncthreads_or(!ok);
  if (threadIdx.x == 0) flag[tile] = bad;
  cur = nxt;
  }
}

// Persistent launch: one block per compute unit (never more than the tiles).
template <int DK, int DV, int VAR>
hipError_t launch_grad_bf(const BwdArgs& a) {
  const Geo& geo = a.geo;
  const int H = geo.H;
  const BwdWs& w = a.ws;
  const int ntiles = geo.total_chunks * H;
  const int grid = ntiles < a.num_cus ? ntiles : a.num_cus;
  hipLaunchKernelGGL((k_grad_bf<DK, DV, VAR>), dim3(grid), dim3(GradBF<DK, DV>::NT), 0, a.stream, geo, H, ntiles,
                     (const bf16*)a.q, (const bf16*)a.k, (const bf16*)a.v, a.g, a.beta, a.states,
                     (const bf16*)a.dO, (const bf16*)w.dh, (const bf16*)w.dUT, (const bf16*)w.T, (bf16*)a.dq,
                     (bf16*)a.dk_, (bf16*)a.dv_, a.dg, a.dbeta, w.flag_grad);
  return hipGetLastError();
}
#endif  // GDN_TILE_LOOP

// ---------------------------------------------------------------------------
// Launches the bf16 chunk-gradient kernel; instantiated in the translation
// units compiled with GDN_TILE_LOOP.
template <int DK, int DV, int VAR>
hipError_t launch_grad_bf(const BwdArgs& a);

template <int DK, int DV, typename OP, int VAR>
static hipError_t launch_bwd_t(const BwdArgs& a) {
  constexpr int BV = SCAN_BV;
  constexpr int NVT = DV / BV;
  const Geo& geo = a.geo;
  const int H = geo.H;
  const BwdWs& w = a.ws;
  stage_mark(a.events, 0, a.stream);
  if (geo.cu != nullptr) {
    const hipError_t e = launch_chunk_offsets(geo.cu, geo.N, const_cast<int*>(geo.chunk_off), a.stream);
    if (e != hipSuccess) return e;
  }
  if (geo.total_chunks > 0) {
    hipLaunchKernelGGL((k_prep_bwd<DK, DV, OP, VAR>), dim3(geo.total_chunks, H), dim3(512), 0, a.stream,
                       geo, H, (const OP*)a.q, (const OP*)a.k, a.g, a.beta, (const OP*)a.dO, w.gcum,
                       (OP*)w.W, (OP*)w.QgT, (OP*)w.dOT, (OP*)w.PT, (OP*)w.T, (OP*)w.Kh, w.flag_prep);
  }
  stage_mark(a.events, 1, a.stream);
  const int NS = geo.N * H;
  if (NS > 0) {
    if constexpr (sizeof(OP) == 2) {
      hipLaunchKernelGGL((k_scan_bwd_ws<DK, DV, BV, VAR>), dim3(NS * NVT), dim3(512), 0, a.stream, geo, H,
                         (const bf16*)a.k, a.dST, w.gcum, (const bf16*)w.W, (const bf16*)w.QgT,
                         (const bf16*)a.dO, (const bf16*)w.PT, (bf16*)w.dh, (bf16*)w.dUT, a.dS0, w.flag_scan);
    } else {
      hipLaunchKernelGGL((k_scan_bwd<DK, DV, BV, OP, VAR>), dim3(NS * NVT), dim3(256), 0, a.stream, geo, H,
                         (const OP*)w.Kh, a.dST, w.gcum, (const OP*)w.W, (const OP*)w.QgT, (const OP*)w.dOT,
                         (const OP*)w.PT, (OP*)w.dh, (OP*)w.dUT, a.dS0, w.flag_scan);
    }
  }
  stage_mark(a.events, 2, a.stream);
  if (geo.total_chunks > 0 && sizeof(OP) == 2) {
    const hipError_t e = launch_grad_bf<DK, DV, VAR>(a);
    if (e != hipSuccess) return e;
  } else if (geo.total_chunks > 0) {
    hipLaunchKernelGGL((k_grad_bwd<DK, DV, OP, VAR>), dim3(geo.total_chunks, H), dim3(512), 0, a.stream,
                       geo, H, (const OP*)a.q, (const OP*)a.k, (const OP*)a.v, a.g, a.beta, a.states,
                       (const OP*)a.dO, (const OP*)w.dh, (const OP*)w.dUT, (OP*)a.dq, (OP*)a.dk_, (OP*)a.dv_,
                       a.dg, a.dbeta, w.flag_grad, (char*)w.grad_scratch);
  }
  stage_mark(a.events, 3, a.stream);
  if (NS > 0) {
    hipLaunchKernelGGL((k_exact_bwd<DK, DV, OP, VAR>), dim3(EXACT_SLOTS), dim3(DV), 0, a.stream, geo,
                       (const OP*)a.q, (const OP*)a.k, (const OP*)a.v, a.g, a.beta, a.states,
                       (const OP*)a.dO, a.dST, (OP*)a.dq, (OP*)a.dk_, (OP*)a.dv_, a.dg, a.dbeta, a.dS0,
                       w.flag_prep, w.flag_grad, w.flag_scan, NVT, w.exact);
  }
  stage_mark(a.events, 4, a.stream);
  return hipGetLastError();
}

template <int DT, int VAR>
hipError_t launch_bwd_var(const BwdArgs& a) {
  typedef typename op_of<DT>::type OP;
  const int dk = a.dk, dv = a.dv;
  if (dk == 64 && dv == 64) return launch_bwd_t<64, 64, OP, VAR>(a);
  if (dk == 64 && dv == 128) return launch_bwd_t<64, 128, OP, VAR>(a);
  if (dk == 64 && dv == 256) return launch_bwd_t<64, 256, OP, VAR>(a);
  if (dk == 128 && dv == 64) return launch_bwd_t<128, 64, OP, VAR>(a);
  if (dk == 128 && dv == 128) return launch_bwd_t<128, 128, OP, VAR>(a);
  if (dk == 128 && dv == 256) return launch_bwd_t<128, 256, OP, VAR>(a);
  return hipErrorInvalidValue;
}

}  // namespace gdn
