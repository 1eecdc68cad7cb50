// Forward of the chunked gated delta rule on gfx950 (paper Sec. 4.2: parallel
// work inside every chunk of 64 tokens, then a short sequential carry between
// chunks).  Three kernels per call:
//
//   prep   one block per (chunk, head): in-chunk cumulative decay G, the erase
//          coupling A = strict_lower(diag(beta) K K^T * exp(G_r - G_i)), the
//          inverse T = (I + A)^{-1}, and the two applies
//          W = T diag(beta e^G) K, U = T diag(beta) V.
//   scan   one block per (stream, value tile of BV columns): the inter-chunk
//          carry, chunk by chunk,  U' = U - W h,  h <- e^{G_last} h + Khat^T U'
//          with Khat_r = e^{G_last - G_r} k_r; writes every h (the saved chunk
//          states), U' and S_T.  The carry splits over value columns with no
//          communication.
//   out    one block per (chunk, head): O = diag(e^G) Q h + ((Q K^T) * D) U'
//          with D_ri = e^{G_r - G_i} for i <= r (exponent formed only there).
#pragma once

#include "gdn_chunk.hpp"
#include "gdn_exact.hpp"
#include "gdn_launch.hpp"

namespace gdn {

template <int DK, int DV, typename OP, int VAR>
__global__ __launch_bounds__(256) void k_prep_fwd(Geo geo, int H, const OP* __restrict__ k,
                                                  const OP* __restrict__ v, const float* __restrict__ g,
                                                  const float* __restrict__ beta, float* __restrict__ gcum,
                                                  OP* __restrict__ Wg, float* __restrict__ Ug,
                                                  OP* __restrict__ KhTg, int* __restrict__ flag) {
  constexpr int LK = DK + pad_of<OP>();
  constexpr int LC = CH + 4;
  constexpr int LT = CH + pad_of<OP>();
  constexpr int VS = 64;  // value columns per slice of U
  constexpr int LVS = VS + pad_of<OP>();
  __shared__ __align__(16) OP Ks[CH * LK];
  __shared__ __align__(16) float As[CH * LC];
  __shared__ __align__(16) float Tf[CH * LC];
  __shared__ __align__(16) OP Ts[sizeof(OP) == 2 ? CH * LT : 1];
  __shared__ __align__(16) OP Vs[CH * LVS];
  __shared__ __align__(16) float Xs[4 * 16 * 20];
  __shared__ float Gs[CH], Bs[CH], GBs[CH];

  const int ci = blockIdx.x, h = blockIdx.y;
  const ChunkPos cp = chunk_pos(geo, ci);
  const long tile = (long)ci * H + h;
  bool ok = load_gates<VAR>(g, beta, cp.row0, H, h, cp.len, Gs, Bs);
  if (VAR != VAR_DECAY) ok &= load_rows<DK, LK>(k + (cp.row0 * H + h) * DK, (long)H * DK, cp.len, Ks);
  __syncthreads();
  if (threadIdx.x < CH) {
    gcum[tile * CH + threadIdx.x] = Gs[threadIdx.x];
    GBs[threadIdx.x] = Bs[threadIdx.x] * expf(Gs[threadIdx.x]);
  }
  if constexpr (VAR != VAR_DECAY) {
    // A = strict_lower(diag(beta) K K^T * exp(G_r - G_i))
    Tiles<CH, CH, 2, 2> bm;
    bm.zero();
    bm.template mma<OP, DK>(KRow<OP, LK>{Ks}, KRow<OP, LK>{Ks});
    bm.each([&](int r, int i, float& x) {
      As[r * LC + i] = (i < r) ? Bs[r] * x * expf(Gs[r] - Gs[i]) : 0.f;
    });
    __syncthreads();
    unit_lower_inverse<OP, LC, LT>(As, Tf, Ts, Xs);
    const OP* Tp;
    if constexpr (sizeof(OP) == 2) Tp = Ts; else Tp = Tf;
    constexpr int LTT = sizeof(OP) == 2 ? LT : LC;
    // W = T diag(beta e^G) K
    {
      Tiles<CH, DK, 2, 2> w;
      w.zero();
      w.template mma<OP, CH>(KRow<OP, LTT>{Tp}, kfun<OP>([&](int d, int i) {
                               return from_f<OP>(GBs[i] * to_f(Ks[i * LK + d]));
                             }));
      OP* Wt = Wg + tile * CH * DK;
      w.each([&](int r, int d, float& x) { Wt[r * DK + d] = from_f<OP>(x); });
    }
    // U = T diag(beta) V, in slices of VS value columns
    const OP* vp = v + (cp.row0 * H + h) * DV;
    float* Ut = Ug + tile * CH * DV;
    for (int c0 = 0; c0 < DV; c0 += VS) {
      ok &= load_rows<VS, LVS>(vp + c0, (long)H * DV, cp.len, Vs);
      __syncthreads();
      Tiles<CH, VS, 2, 2> u;
      u.zero();
      u.template mma<OP, CH>(KRow<OP, LTT>{Tp}, kfun<OP>([&](int vv, int i) {
                               return from_f<OP>(Bs[i] * to_f(Vs[i * LVS + vv]));
                             }));
      u.each([&](int r, int vv, float& x) { Ut[r * DV + c0 + vv] = x; });
      __syncthreads();
    }
  } else {
    // scalar-decay member: T = I, W = 0, U = V; only check v for non-finite values
    const OP* vp = v + (cp.row0 * H + h) * DV;
    for (int c0 = 0; c0 < DV; c0 += VS) {
      ok &= load_rows<VS, LVS>(vp + c0, (long)H * DV, cp.len, Vs);
      __syncthreads();
    }
    ok &= load_rows<DK, LK>(k + (cp.row0 * H + h) * DK, (long)H * DK, cp.len, Ks);
  }
  // Khat^T[d][r] = exp(G_last - G_r) k_r[d], the scan's A operand for the carry
  __syncthreads();
  if (threadIdx.x < CH) GBs[threadIdx.x] = expf(Gs[CH - 1] - Gs[threadIdx.x]);
  __syncthreads();
  OP* Kh = KhTg + tile * DK * CH;
  constexpr int VE = 16 / (int)sizeof(OP);
  for (int idx = threadIdx.x; idx < DK * CH / VE; idx += blockDim.x) {
    const int d = idx / (CH / VE), r0 = (idx - d * (CH / VE)) * VE;
    OP vals[VE];
#pragma unroll
    for (int j = 0; j < VE; ++j) vals[j] = from_f<OP>(GBs[r0 + j] * to_f(Ks[(r0 + j) * LK + d]));
    *reinterpret_cast<uint4*>(Kh + d * CH + r0) = pack16<OP>(vals);
  }
  const int bad = __syncthreads_or(!ok);
  if (threadIdx.x == 0) flag[tile] = bad;
}

// The forward inter-chunk scan.  Every operand except the carry arrives
// pre-laid-out by the prep kernel (W row-major, Khat^T row-major, U in fp32), so
// the A fragments of chunk c+1 are loaded from HBM/L2 straight into registers
// while chunk c is computed; only h and U' pass through LDS (two barriers per
// chunk).
template <int DK, int DV, int BV, typename OP, int VAR>
__global__ __launch_bounds__(256) void k_scan_fwd(Geo geo, int H, const OP* __restrict__ v,
                                                  const float* __restrict__ S0, const float* __restrict__ gcum,
                                                  const OP* __restrict__ Wg, const OP* __restrict__ KhTg,
                                                  const float* __restrict__ Ug, float* __restrict__ states,
                                                  float* __restrict__ ST, OP* __restrict__ UpTg,
                                                  int* __restrict__ flag) {
  constexpr int NVT = DV / BV;
  constexpr int LK = DK + pad_of<OP>();
  constexpr int LU = CH + pad_of<OP>();
  constexpr bool PF = sizeof(OP) == 2;  // prefetch a chunk ahead (bf16 fragments are compact)
  typedef Tiles<DK, BV, 4, 1> HT;       // carried state slice h[:, v0:v0+BV]
  typedef Tiles<CH, BV, 4, 1> UT;       // U' slice
  __shared__ __align__(16) OP hT[BV * LK];
  __shared__ __align__(16) OP UsT[BV * LU];

  int s, vt;
  scan_block_coords(blockIdx.x, geo.N * H, NVT, s, vt);
  const int n = s / H, h = s - (s / H) * H, v0 = vt * BV;
  const SeqPos sp = seq_pos(geo, n);
  const int l = lane_id();

  struct Pre {
    typename UT::template AFr<OP, DK> w;
    typename HT::template AFr<OP, CH> kh;
    float u[UT::TN][4];
    float gl;
  };
  auto load_pre = [&](Pre& p, int c) {
    const long tile = (long)(sp.c0 + c) * H + h;
    if constexpr (VAR != VAR_DECAY) {
      p.w.load(KRow<OP, DK>{Wg + tile * CH * DK});
      const float* Ut = Ug + tile * CH * DV + v0;
#pragma unroll
      for (int b = 0; b < UT::TN; ++b)
#pragma unroll
        for (int j = 0; j < 4; ++j) p.u[b][j] = Ut[(UT::m0(0) + (l >> 4) * 4 + j) * DV + UT::n0(b) + (l & 15)];
    } else {
      const long row0 = sp.row0 + (long)c * CH;
      const int len = min(CH, sp.len - c * CH);
      const OP* vp = v + (row0 * H + h) * DV + v0;
#pragma unroll
      for (int b = 0; b < UT::TN; ++b)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int r = UT::m0(0) + (l >> 4) * 4 + j;
          p.u[b][j] = r < len ? to_f(vp[(long)r * H * DV + UT::n0(b) + (l & 15)]) : 0.f;
        }
    }
    p.kh.load(KRow<OP, CH>{KhTg + tile * DK * CH});
    p.gl = expf(gcum[tile * CH + CH - 1]);
  };

  HT hs;
  bool ok = true;
  const float* S0p = S0 ? S0 + ((long)n * H + h) * DK * DV : nullptr;
  hs.each([&](int d, int vv, float& x) {
    x = S0p ? S0p[d * DV + v0 + vv] : 0.f;
    ok &= finite_f(x);
  });

  Pre cur, nxt;
  if (sp.nch > 0) load_pre(cur, 0);
  for (int c = 0; c < sp.nch; ++c) {
    const long tile = (long)(sp.c0 + c) * H + h;
    float* hp = states + tile * DK * DV;
    hs.each([&](int d, int vv, float& x) {
      hp[d * DV + v0 + vv] = x;
      hT[vv * LK + d] = from_f<OP>(x);
    });
    __syncthreads();
    if (!PF) {
      if (c > 0) load_pre(cur, c);
    } else if (c + 1 < sp.nch) {
      load_pre(nxt, c + 1);
    }
    UT up;
    if constexpr (VAR != VAR_DECAY) {
      up.zero();
      up.template mma<OP, DK>(cur.w, KRow<OP, LK>{hT});
#pragma unroll
      for (int b = 0; b < UT::TN; ++b)
#pragma unroll
        for (int j = 0; j < 4; ++j) up.acc[0][b][j] = cur.u[b][j] - up.acc[0][b][j];
    } else {
#pragma unroll
      for (int b = 0; b < UT::TN; ++b)
#pragma unroll
        for (int j = 0; j < 4; ++j) up.acc[0][b][j] = cur.u[b][j];
    }
    OP* Upt = UpTg + tile * DV * CH;
#pragma unroll
    for (int b = 0; b < UT::TN; ++b) {
      const int vv = UT::n0(b) + (l & 15), r0 = UT::m0(0) + (l >> 4) * 4;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const OP xo = from_f<OP>(up.acc[0][b][j]);
        if (VAR != VAR_DECAY) Upt[(v0 + vv) * CH + r0 + j] = xo;
        UsT[vv * LU + r0 + j] = xo;
      }
    }
    __syncthreads();
    const float gl = cur.gl;
    hs.each([&](int, int, float& x) { x *= gl; });
    hs.template mma<OP, CH>(cur.kh, KRow<OP, LU>{UsT});
    if (PF) cur = nxt;
  }
  float* STp = ST + ((long)n * H + h) * DK * DV;
  hs.each([&](int d, int vv, float& x) { STp[d * DV + v0 + vv] = x; });
  const int bad = __syncthreads_or(!ok);
  if (threadIdx.x == 0) flag[(long)s * NVT + vt] = bad;
}

template <int DK, int DV, typename OP, int VAR>
__global__ __launch_bounds__(256) void k_out_fwd(Geo geo, int H, const OP* __restrict__ q,
                                                 const OP* __restrict__ k, const OP* __restrict__ v,
                                                 const float* __restrict__ gcum,
                                                 const float* __restrict__ states,
                                                 const OP* __restrict__ UpTg, OP* __restrict__ o,
                                                 int* __restrict__ flag) {
  constexpr int DVS = (sizeof(OP) == 2) ? (DV < 128 ? DV : 128) : 64;  // value columns per slice
  constexpr int LK = DK + pad_of<OP>();
  constexpr int LT = CH + pad_of<OP>();
  constexpr int LH = DVS + pad_of<OP>();
  __shared__ __align__(16) OP Qs[CH * LK];
  __shared__ __align__(16) OP Ks[CH * LK];
  __shared__ __align__(16) OP Hs[DK * LH];   // h[:, slice], row-major (d, v)
  __shared__ __align__(16) OP Ps[CH * LT];
  __shared__ __align__(16) OP UT[DVS * LT];  // U'^T slice (v, i); scalar decay: V slice (i, v)
  static_assert(CH * LH <= DVS * LT, "V slice must fit the U' buffer");
  __shared__ __align__(16) OP Os[CH * LH];
  __shared__ float Gs[CH];

  const int ci = blockIdx.x, h = blockIdx.y;
  const ChunkPos cp = chunk_pos(geo, ci);
  const long tile = (long)ci * H + h;
  bool ok = load_rows<DK, LK>(q + (cp.row0 * H + h) * DK, (long)H * DK, cp.len, Qs);
  load_rows<DK, LK>(k + (cp.row0 * H + h) * DK, (long)H * DK, cp.len, Ks);
  if (threadIdx.x < CH) Gs[threadIdx.x] = gcum[tile * CH + threadIdx.x];
  __syncthreads();
  {
    Tiles<CH, CH, 2, 2> p;
    p.zero();
    p.template mma<OP, DK>(KRow<OP, LK>{Qs}, KRow<OP, LK>{Ks});
    p.each([&](int r, int i, float& x) {
      Ps[r * LT + i] = from_f<OP>(i <= r ? x * expf(Gs[r] - Gs[i]) : 0.f);
    });
  }
  const float* hp = states + tile * DK * DV;
  for (int c0 = 0; c0 < DV; c0 += DVS) {
    for (int idx = threadIdx.x; idx < DK * DVS / 4; idx += blockDim.x) {
      const int d = idx / (DVS / 4), c = (idx - d * (DVS / 4)) * 4;
      const float4 x = *reinterpret_cast<const float4*>(hp + (long)d * DV + c0 + c);
      Hs[d * LH + c + 0] = from_f<OP>(x.x);
      Hs[d * LH + c + 1] = from_f<OP>(x.y);
      Hs[d * LH + c + 2] = from_f<OP>(x.z);
      Hs[d * LH + c + 3] = from_f<OP>(x.w);
    }
    if constexpr (VAR != VAR_DECAY) {
      load_dense<DVS, CH, LT>(UpTg + tile * DV * CH + (long)c0 * CH, UT);
    } else {
      // V slice, row-major (i, v) with row stride LH; fits in UT (64*LH <= DVS*LT)
      load_rows<DVS, LH>(v + (cp.row0 * H + h) * DV + c0, (long)H * DV, cp.len, UT);
    }
    __syncthreads();
    Tiles<CH, DVS, 2, 2> ot;
    ot.zero();
    ot.template mma<OP, DK>(KRow<OP, LK>{Qs}, KCol<OP, LH>{Hs});
    ot.each([&](int r, int, float& x) { x *= expf(Gs[r]); });
    if constexpr (VAR != VAR_DECAY)
      ot.template mma<OP, CH>(KRow<OP, LT>{Ps}, KRow<OP, LT>{UT});
    else
      ot.template mma<OP, CH>(KRow<OP, LT>{Ps}, KCol<OP, LH>{UT});
    ot.each([&](int r, int vv, float& x) { Os[r * LH + vv] = from_f<OP>(x); });
    __syncthreads();
    store_rows<DVS, LH>(o + (cp.row0 * H + h) * DV + c0, (long)H * DV, cp.len, Os);
    __syncthreads();
  }
  const int bad = __syncthreads_or(!ok);
  if (threadIdx.x == 0) flag[tile] = bad;
}

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------
template <int DK, int DV, typename OP, int VAR>
static hipError_t launch_fwd_t(const FwdArgs& a) {
  constexpr int BV = 32;
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
    hipLaunchKernelGGL((k_prep_fwd<DK, DV, OP, VAR>), dim3(geo.total_chunks, H), dim3(256), 0, a.stream,
                       geo, H, (const OP*)a.k, (const OP*)a.v, a.g, a.beta, w.gcum, (OP*)w.W, w.U,
                       (OP*)w.KhT, w.flag_prep);
  }
  stage_mark(a.events, 1, a.stream);
  const int NS = geo.N * H;
  if (NS > 0) {
    hipLaunchKernelGGL((k_scan_fwd<DK, DV, BV, OP, VAR>), dim3(NS * NVT), dim3(256), 0, a.stream, geo, H,
                       (const OP*)a.v, a.S0, w.gcum, (const OP*)w.W, (const OP*)w.KhT, w.U, a.states,
                       a.ST, (OP*)w.UpT, w.flag_scan);
  }
  stage_mark(a.events, 2, a.stream);
  if (geo.total_chunks > 0) {
    hipLaunchKernelGGL((k_out_fwd<DK, DV, OP, VAR>), dim3(geo.total_chunks, H), dim3(256), 0, a.stream,
                       geo, H, (const OP*)a.q, (const OP*)a.k, (const OP*)a.v, w.gcum, a.states,
                       (const OP*)w.UpT, (OP*)a.o, w.flag_out);
  }
  stage_mark(a.events, 3, a.stream);
  if (NS > 0) {
    hipLaunchKernelGGL((k_exact_fwd<DK, DV, OP, VAR>), dim3(NS), dim3(DV), 0, a.stream, geo, (const OP*)a.q,
                       (const OP*)a.k, (const OP*)a.v, a.g, a.beta, a.S0, (OP*)a.o, a.ST, a.states,
                       w.flag_prep, w.flag_out, w.flag_scan, NVT);
  }
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
