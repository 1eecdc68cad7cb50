// Exact-semantics path of the channel-wise members for streams whose inputs
// hold a NaN or an Inf (paper Sec. 4.1, Eq. (gdn) with its gates per channel).
//
// The chunked channel-wise kernels multiply masked zeros by whole rows and
// split decays at reference rows, so inside a poisoned chunk they cannot
// reproduce which outputs of the token-serial recurrence become NaN or Inf.
// The prep kernels (q, k, g, b and the forward's v, w or the backward's dO),
// the reverse scan (dS_T), the forward scan (S0) and the value-part gradient
// kernel (v, w, the chunk states) record per (chunk, head) or (stream, value
// tile) whether they saw a non-finite input; the kernels below recompute each
// flagged (sequence, head) stream token by token in fp32 in the operation
// order of the recurrence as written:
//
//   St = e^{g_t} * S (row d scaled by e^{g_t[d]});  p = St^T (b_t * k_t);
//   u = w_t * v_t - p;  S = St + k_t u^T;  o_t = S^T q_t
//
// and its reverse-time adjoint
//
//   dS += q_t dO_t^T;  dq_t = S_t dO_t;  du = dS^T k_t;  dk_t = dS u;
//   dv_t = w_t * du;  dw_t = v_t * du;  dp = -du;
//   dSt = dS + (b_t * k_t) dp^T;  dkb = St dp;  dk_t += b_t * dkb;  db_t = k_t * dkb;
//   dg_t = rowsum(dSt * St);  dS = e^{g_t} * dSt,
//
// overwriting every output of the stream.  A gate that is absent takes its
// neutral value (g = 0, b = 0, w = 1) and its terms are skipped, as in the
// recurrence.  Thread v owns value column v of S and dS (d_k values each);
// sums over value columns (dq, dk, dkb, dg) go through LDS in a fixed order.
#pragma once

#include "gdn_exact.hpp"

namespace gdn {

// Forward: one block of DV threads per stream (clean streams only read flags).
template <int DK, int DV, typename IO>
__global__ __launch_bounds__(256) void k_cw_exact_fwd(Geo geo, const IO* __restrict__ q, const IO* __restrict__ k,
                                                      const IO* __restrict__ v, const float* __restrict__ g,
                                                      const float* __restrict__ b, const float* __restrict__ w,
                                                      const float* __restrict__ S0, IO* __restrict__ o,
                                                      float* __restrict__ ST, float* __restrict__ states,
                                                      const int* __restrict__ fa, const int* __restrict__ fs,
                                                      int nvt) {
  const int s = blockIdx.x;
  if (!stream_flagged(geo, s, fa, fa, fs, nvt)) return;
  const int H = geo.H;
  const int n = s / H, h = s - (s / H) * H;
  const SeqPos sp = seq_pos(geo, n);
  const int col = threadIdx.x;
  __shared__ float ks[DK], qs[DK], es[DK], kbs[DK];
  float S[DK];
  const float* s0 = S0 ? S0 + (long)s * DK * DV : nullptr;
#pragma unroll
  for (int d = 0; d < DK; ++d) S[d] = s0 ? s0[d * DV + col] : 0.f;
  for (int t = 0; t < sp.len; ++t) {
    const long row = sp.row0 + t;
    if (t % CH == 0) {
      float* st = states + ((long)(sp.c0 + t / CH) * H + h) * DK * DV;
#pragma unroll
      for (int d = 0; d < DK; ++d) st[d * DV + col] = S[d];
    }
    __syncthreads();
    for (int d = threadIdx.x; d < DK; d += blockDim.x) {
      const long i = (row * H + h) * DK + d;
      ks[d] = ld(k, i);
      qs[d] = ld(q, i);
      es[d] = g ? expf(g[i]) : 1.f;
      kbs[d] = b ? b[i] * ks[d] : 0.f;
    }
    __syncthreads();
    const long iv = (row * H + h) * DV + col;
    const float wv = w ? w[iv] * ld(v, iv) : ld(v, iv);
    if (g) {
#pragma unroll
      for (int d = 0; d < DK; ++d) S[d] = es[d] * S[d];
    }
    float u = wv;
    if (b) {
      float p = 0.f;
#pragma unroll
      for (int d = 0; d < DK; ++d) p += S[d] * kbs[d];
      u = wv - p;
    }
    float ov = 0.f;
#pragma unroll
    for (int d = 0; d < DK; ++d) {
      S[d] = S[d] + ks[d] * u;
      ov += S[d] * qs[d];
    }
    o[iv] = from_f<IO>(ov);
  }
  float* stp = ST + (long)s * DK * DV;
#pragma unroll
  for (int d = 0; d < DK; ++d) stp[d * DV + col] = S[d];
}

// Backward: EXACT_SLOTS blocks of DV threads; block b visits the streams
// s = b, b + EXACT_SLOTS, ... in order and recomputes the flagged ones.  Slot b
// of the scratch holds one chunk's states S_{t0-1}, S_{t0}, ..., S_{t1-1} as
// [index][column][row], followed by room to park dS while the chunk is replayed.
template <int DK, int DV, typename IO>
__global__ __launch_bounds__(256) void k_cw_exact_bwd(Geo geo, const IO* __restrict__ q, const IO* __restrict__ k,
                                                      const IO* __restrict__ v, const float* __restrict__ g,
                                                      const float* __restrict__ b, const float* __restrict__ w,
                                                      const float* __restrict__ states, const IO* __restrict__ dO,
                                                      const float* __restrict__ dST, IO* __restrict__ dq,
                                                      IO* __restrict__ dk, IO* __restrict__ dv,
                                                      float* __restrict__ dg, float* __restrict__ db,
                                                      float* __restrict__ dw, float* __restrict__ dS0,
                                                      const int* __restrict__ fa, const int* __restrict__ fb,
                                                      const int* __restrict__ fs, int nvt, float* __restrict__ scratch) {
  constexpr int LR = DK + 1;
  __shared__ float red[DV * LR];  // per-column terms, reduced over columns in a fixed order
  __shared__ float ks[DK], qs[DK], es[DK], bs[DK], kbs[DK], dkA[DK];
  const int H = geo.H;
  const int NS = geo.N * H;
  const int col = threadIdx.x;
  float* slot = scratch + (long)blockIdx.x * (CH + 2) * DK * DV;
  float* park = slot + (long)(CH + 1) * DK * DV + (long)col * DK;
  // sum over the value columns of red[.][d], for every d (threads d, d + DV, ...)
  auto column_sum = [&](int d) {
    float a = 0.f;
    for (int j = 0; j < DV; ++j) a += red[j * LR + d];
    return a;
  };
  unsigned mask = 0;
  for (int s = blockIdx.x, i = 0; s < NS; s += EXACT_SLOTS, i = (i + 1) & 7) {
    if (i == 0) mask = streams_flagged8(geo, s, EXACT_SLOTS, NS, fa, fb, fs, nvt);
    if (!(mask >> i & 1u)) continue;
    const int n = s / H, h = s - (s / H) * H;
    const SeqPos sp = seq_pos(geo, n);
    float dS[DK];
    const float* dsT = dST ? dST + (long)s * DK * DV : nullptr;
#pragma unroll
    for (int d = 0; d < DK; ++d) dS[d] = dsT ? dsT[d * DV + col] : 0.f;
    for (int c = sp.nch - 1; c >= 0; --c) {
      const int t0 = c * CH, t1 = min(sp.len, t0 + CH);
      // replay the chunk's forward from its saved state into the slot
#pragma unroll
      for (int d = 0; d < DK; ++d) park[d] = dS[d];
      {
        float S[DK];
        const float* st = states + ((long)(sp.c0 + c) * H + h) * DK * DV;
#pragma unroll
        for (int d = 0; d < DK; ++d) S[d] = st[d * DV + col];
        float* w0 = slot + (long)col * DK;
#pragma unroll
        for (int d = 0; d < DK; ++d) w0[d] = S[d];
        for (int t = t0; t < t1; ++t) {
          const long row = sp.row0 + t;
          __syncthreads();
          for (int d = threadIdx.x; d < DK; d += blockDim.x) {
            const long ik = (row * H + h) * DK + d;
            ks[d] = ld(k, ik);
            es[d] = g ? expf(g[ik]) : 1.f;
            kbs[d] = b ? b[ik] * ks[d] : 0.f;
          }
          __syncthreads();
          const long iv = (row * H + h) * DV + col;
          const float wv = w ? w[iv] * ld(v, iv) : ld(v, iv);
          if (g) {
#pragma unroll
            for (int d = 0; d < DK; ++d) S[d] = es[d] * S[d];
          }
          float u = wv;
          if (b) {
            float p = 0.f;
#pragma unroll
            for (int d = 0; d < DK; ++d) p += S[d] * kbs[d];
            u = wv - p;
          }
          float* wr = slot + ((long)(t - t0 + 1) * DV + col) * DK;
#pragma unroll
          for (int d = 0; d < DK; ++d) {
            S[d] = S[d] + ks[d] * u;
            wr[d] = S[d];
          }
        }
      }
#pragma unroll
      for (int d = 0; d < DK; ++d) dS[d] = park[d];
      // reverse through the chunk
      for (int t = t1 - 1; t >= t0; --t) {
        const long row = sp.row0 + t;
        __syncthreads();
        for (int d = threadIdx.x; d < DK; d += blockDim.x) {
          const long ik = (row * H + h) * DK + d;
          ks[d] = ld(k, ik);
          qs[d] = ld(q, ik);
          es[d] = g ? expf(g[ik]) : 1.f;
          bs[d] = b ? b[ik] : 0.f;
          kbs[d] = b ? bs[d] * ks[d] : 0.f;
        }
        __syncthreads();
        const long iv = (row * H + h) * DV + col;
        const float vt = ld(v, iv), wt = w ? w[iv] : 1.f;
        const float dot = ld(dO, iv);
        const float* Sp = slot + ((long)(t - t0) * DV + col) * DK;      // S_{t-1}
        const float* Sn = slot + ((long)(t - t0 + 1) * DV + col) * DK;  // S_t
        // dS += q dO^T; the terms of dq_t = S_t dO_t
#pragma unroll
        for (int d = 0; d < DK; ++d) {
          dS[d] = dS[d] + qs[d] * dot;
          red[col * LR + d] = Sn[d] * dot;
        }
        __syncthreads();
        for (int d = threadIdx.x; d < DK; d += blockDim.x) dq[(row * H + h) * DK + d] = from_f<IO>(column_sum(d));
        __syncthreads();
        // St, p and u again; du = dS^T k; the terms of dS u
        float u = w ? wt * vt : vt;
        if (b) {
          float p = 0.f;
#pragma unroll
          for (int d = 0; d < DK; ++d) p += (g ? es[d] * Sp[d] : Sp[d]) * kbs[d];
          u = u - p;
        }
        float du = 0.f;
#pragma unroll
        for (int d = 0; d < DK; ++d) {
          du += dS[d] * ks[d];
          red[col * LR + d] = dS[d] * u;
        }
        dv[iv] = from_f<IO>(w ? wt * du : du);
        if (w) dw[iv] = vt * du;
        __syncthreads();
        for (int d = threadIdx.x; d < DK; d += blockDim.x) dkA[d] = column_sum(d);
        __syncthreads();
        if (b) {
          // dSt = dS + (b k) dp^T with dp = -du; the terms of dkb = St dp
          const float dp = -du;
#pragma unroll
          for (int d = 0; d < DK; ++d) {
            red[col * LR + d] = (g ? es[d] * Sp[d] : Sp[d]) * dp;
            dS[d] = dS[d] + kbs[d] * dp;
          }
          __syncthreads();
          for (int d = threadIdx.x; d < DK; d += blockDim.x) {
            const float dkb = column_sum(d);
            const long ik = (row * H + h) * DK + d;
            dk[ik] = from_f<IO>(dkA[d] + bs[d] * dkb);
            db[ik] = ks[d] * dkb;
          }
          __syncthreads();
        } else {
          for (int d = threadIdx.x; d < DK; d += blockDim.x) dk[(row * H + h) * DK + d] = from_f<IO>(dkA[d]);
        }
        if (g) {
          // dg_t = rowsum(dSt * St); dS = e^{g_t} * dSt
#pragma unroll
          for (int d = 0; d < DK; ++d) {
            red[col * LR + d] = dS[d] * (es[d] * Sp[d]);
            dS[d] = es[d] * dS[d];
          }
          __syncthreads();
          for (int d = threadIdx.x; d < DK; d += blockDim.x) dg[(row * H + h) * DK + d] = column_sum(d);
        }
      }
    }
    float* d0 = dS0 + (long)s * DK * DV;
#pragma unroll
    for (int d = 0; d < DK; ++d) d0[d * DV + col] = dS[d];
    __syncthreads();
  }
}

}  // namespace gdn
