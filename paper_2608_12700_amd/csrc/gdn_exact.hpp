// Exact-semantics path for streams whose inputs hold a NaN or an Inf.
//
// The chunked kernels multiply masked zeros by whole rows and sum decays in
// blocks, so inside a poisoned chunk they cannot reproduce which outputs of
// the token-serial recurrence become NaN or Inf.  Every kernel that reads an
// input also records whether it saw a non-finite value, per (chunk, head) or
// per (stream, value tile); the kernels below then recompute each flagged
// (sequence, head) stream token by token in fp32, in the operation order of
// the recurrence as written (paper Sec. 4.1, Eq. (gdn) with scalar gates):
//
//   St = exp(g_t) S;  p = St^T k_t;  u = beta_t (v_t - p);  S = St + k_t u^T;  o_t = S^T q_t
//
// and its reverse-time adjoint
//
//   dS += q_t dO_t^T;  dq_t = S_t dO_t;  du = dS^T k_t;  dk_t = dS u + St dp;
//   dbeta_t = du.(v_t - p);  dv_t = beta_t du;  dp = -beta_t du;  dSt = dS + k_t dp^T;
//   dg_t = <dSt, St>;  dS = exp(g_t) dSt,
//
// overwriting every output of the stream.  The class (finite, NaN, +Inf,
// -Inf) of a sum depends only on the classes of its terms, so the reductions
// may run in any fixed order.  Clean streams only read their flags.
//
// The forward is column-separable: thread v owns column v of S (d_k values in
// registers) and needs no communication.  The backward owns dS the same way;
// the states S_t of one chunk are replayed into a per-block slot of the
// workspace, and the sums over value columns (dq, dk, dbeta, dg) go through LDS
// in a fixed order.
#pragma once

#include "gdn_chunk.hpp"

namespace gdn {

constexpr int EXACT_SLOTS = 16;  // blocks of the exact backward (one scratch slot each)

// Whether stream s = n*H + h saw a non-finite input: OR of its chunks' flags in
// fa and fb ([chunks*H]) and of its value tiles' flags in fs ([N*H*nvt]).
// Called by all threads of the block.
__device__ __forceinline__ bool stream_flagged(const Geo& geo, int s, const int* fa, const int* fb,
                                               const int* fs, int nvt) {
  const int H = geo.H;
  const int n = s / H, h = s - (s / H) * H;
  const SeqPos sp = seq_pos(geo, n);
  int any = 0;
  for (int c = threadIdx.x; c < sp.nch; c += blockDim.x) {
    const long t = (long)(sp.c0 + c) * H + h;
    any |= fa[t] | fb[t];
  }
  for (int j = threadIdx.x; j < nvt; j += blockDim.x) any |= fs[(long)s * nvt + j];
  return __syncthreads_or(any) != 0;
}

// Flags of the streams s0, s0 + step, ... (up to 8 of them, fewer past NS),
// checked in one pass: the block's threads split into eight groups, one per
// stream, and the group ORs its stream's chunk and value-tile flags into
// bit i of the result.
__device__ __forceinline__ unsigned streams_flagged8(const Geo& geo, int s0, int step, int NS, const int* fa,
                                                     const int* fb, const int* fs, int nvt) {
  __shared__ int fl[8];
  const int per = blockDim.x / 8, i = threadIdx.x / per, li = threadIdx.x - i * per;
  if (threadIdx.x < 8) fl[threadIdx.x] = 0;
  __syncthreads();
  const int s = s0 + i * step;
  int any = 0;
  if (s < NS) {
    const int H = geo.H;
    const int n = s / H, h = s - (s / H) * H;
    const SeqPos sp = seq_pos(geo, n);
    for (int c = li; c < sp.nch; c += per) {
      const long t = (long)(sp.c0 + c) * H + h;
      any |= fa[t] | fb[t];
    }
    for (int j = li; j < nvt; j += per) any |= fs[(long)s * nvt + j];
  }
  if (any) atomicOr(&fl[i], 1);  // integer OR: order-free
  __syncthreads();
  unsigned m = 0;
  for (int j = 0; j < 8; ++j) m |= fl[j] ? 1u << j : 0u;
  __syncthreads();
  return m;
}

template <typename IO>
__device__ __forceinline__ float ld(const IO* p, long i) { return to_f(p[i]); }

// Forward: one block of DV threads per stream.
template <int DK, int DV, typename IO, int VAR>
__global__ __launch_bounds__(256) void k_exact_fwd(Geo geo, const IO* __restrict__ q, const IO* __restrict__ k,
                                                   const IO* __restrict__ v, const float* __restrict__ g,
                                                   const float* __restrict__ beta, const float* __restrict__ S0,
                                                   IO* __restrict__ o, float* __restrict__ ST,
                                                   float* __restrict__ states, const int* __restrict__ fa,
                                                   const int* __restrict__ fb, const int* __restrict__ fs,
                                                   int nvt) {
  const int s = blockIdx.x;
  if (!stream_flagged(geo, s, fa, fb, fs, nvt)) return;
  const int H = geo.H;
  const int n = s / H, h = s - (s / H) * H;
  const SeqPos sp = seq_pos(geo, n);
  const int col = threadIdx.x;  // value column owned by this thread
  __shared__ float ks[DK], qs[DK], gb[2];
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
      ks[d] = ld(k, (row * H + h) * DK + d);
      qs[d] = ld(q, (row * H + h) * DK + d);
    }
    if (threadIdx.x == 0) {
      gb[0] = VAR != VAR_DELTA ? g[row * H + h] : 0.f;
      gb[1] = VAR != VAR_DECAY ? beta[row * H + h] : 0.f;
    }
    __syncthreads();
    const float vt = ld(v, (row * H + h) * DV + col);
    if (VAR != VAR_DELTA) {
      const float gam = expf(gb[0]);
#pragma unroll
      for (int d = 0; d < DK; ++d) S[d] = gam * S[d];
    }
    float u;
    if (VAR != VAR_DECAY) {
      float p = 0.f;
#pragma unroll
      for (int d = 0; d < DK; ++d) p += S[d] * ks[d];
      u = gb[1] * (vt - p);
    } else {
      u = vt;
    }
    float ov = 0.f;
#pragma unroll
    for (int d = 0; d < DK; ++d) {
      S[d] = S[d] + ks[d] * u;
      ov += S[d] * qs[d];
    }
    o[(row * H + h) * DV + col] = from_f<IO>(ov);
  }
  float* stp = ST + (long)s * DK * DV;
#pragma unroll
  for (int d = 0; d < DK; ++d) stp[d * DV + col] = S[d];
}

// Backward: EXACT_SLOTS blocks of DV threads; block b visits the streams
// s = b, b + EXACT_SLOTS, ... in order and recomputes the flagged ones, with
// slot b of the scratch holding one chunk's states S_{t0-1}, S_{t0}, ...,
// S_{t1-1} as [index][column][row], followed by room to park dS.
template <int DK, int DV, typename IO, int VAR>
__global__ __launch_bounds__(256) void k_exact_bwd(Geo geo, const IO* __restrict__ q, const IO* __restrict__ k,
                                                   const IO* __restrict__ v, const float* __restrict__ g,
                                                   const float* __restrict__ beta,
                                                   const float* __restrict__ states, const IO* __restrict__ dO,
                                                   const float* __restrict__ dST, IO* __restrict__ dq,
                                                   IO* __restrict__ dk, IO* __restrict__ dv,
                                                   float* __restrict__ dg, float* __restrict__ dbeta,
                                                   float* __restrict__ dS0, const int* __restrict__ fa,
                                                   const int* __restrict__ fb, const int* __restrict__ fs,
                                                   int nvt, float* __restrict__ scratch) {
  constexpr int LR = DK + 1;
  __shared__ float red[DV * LR];  // per-column terms, reduced over columns in a fixed order
  __shared__ float ks[DK], qs[DK], gb[2], sc[2][DV];
  const int H = geo.H;
  const int NS = geo.N * H;
  const int col = threadIdx.x;
  float* slot = scratch + (long)blockIdx.x * (CH + 2) * DK * DV;
  float* park = slot + (long)(CH + 1) * DK * DV + (long)col * DK;  // dS while a chunk is replayed
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
          for (int d = threadIdx.x; d < DK; d += blockDim.x) ks[d] = ld(k, (row * H + h) * DK + d);
          if (threadIdx.x == 0) {
            gb[0] = VAR != VAR_DELTA ? g[row * H + h] : 0.f;
            gb[1] = VAR != VAR_DECAY ? beta[row * H + h] : 0.f;
          }
          __syncthreads();
          const float vt = ld(v, (row * H + h) * DV + col);
          if (VAR != VAR_DELTA) {
            const float gam = expf(gb[0]);
#pragma unroll
            for (int d = 0; d < DK; ++d) S[d] = gam * S[d];
          }
          float u;
          if (VAR != VAR_DECAY) {
            float p = 0.f;
#pragma unroll
            for (int d = 0; d < DK; ++d) p += S[d] * ks[d];
            u = gb[1] * (vt - p);
          } else {
            u = vt;
          }
          float* w = slot + ((long)(t - t0 + 1) * DV + col) * DK;
#pragma unroll
          for (int d = 0; d < DK; ++d) {
            S[d] = S[d] + ks[d] * u;
            w[d] = S[d];
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
          ks[d] = ld(k, (row * H + h) * DK + d);
          qs[d] = ld(q, (row * H + h) * DK + d);
        }
        if (threadIdx.x == 0) {
          gb[0] = VAR != VAR_DELTA ? g[row * H + h] : 0.f;
          gb[1] = VAR != VAR_DECAY ? beta[row * H + h] : 0.f;
        }
        __syncthreads();
        const float vt = ld(v, (row * H + h) * DV + col);
        const float dot = ld(dO, (row * H + h) * DV + col);
        const float gam = VAR != VAR_DELTA ? expf(gb[0]) : 1.f;
        const float* Sp = slot + ((long)(t - t0) * DV + col) * DK;      // S_{t-1}
        const float* Sn = slot + ((long)(t - t0 + 1) * DV + col) * DK;  // S_t
        // dS += q dO^T ; dq terms S_t[d] dO_v ; p and du
        float p = 0.f, du = 0.f;
#pragma unroll
        for (int d = 0; d < DK; ++d) {
          dS[d] = dS[d] + qs[d] * dot;
          red[col * LR + d] = Sn[d] * dot;
          const float st = VAR != VAR_DELTA ? gam * Sp[d] : Sp[d];
          p += st * ks[d];
          du += dS[d] * ks[d];
        }
        __syncthreads();
        for (int d = threadIdx.x; d < DK; d += blockDim.x) {
          float a = 0.f;
          for (int j = 0; j < DV; ++j) a += red[j * LR + d];
          dq[(row * H + h) * DK + d] = from_f<IO>(a);
        }
        __syncthreads();
        float u, dp = 0.f;
        if (VAR != VAR_DECAY) {
          u = gb[1] * (vt - p);
          sc[0][col] = du * (vt - p);
          dv[(row * H + h) * DV + col] = from_f<IO>(gb[1] * du);
          dp = -gb[1] * du;
        } else {
          u = vt;
          dv[(row * H + h) * DV + col] = from_f<IO>(du);
        }
        float dgt = 0.f;
#pragma unroll
        for (int d = 0; d < DK; ++d) {
          const float st = VAR != VAR_DELTA ? gam * Sp[d] : Sp[d];
          float term = dS[d] * u;
          if (VAR != VAR_DECAY) {
            term = term + st * dp;
            dS[d] = dS[d] + ks[d] * dp;  // dSt
          }
          red[col * LR + d] = term;
          dgt += dS[d] * st;
          if (VAR != VAR_DELTA) dS[d] = gam * dS[d];
        }
        sc[1][col] = dgt;
        __syncthreads();
        for (int d = threadIdx.x; d < DK; d += blockDim.x) {
          float a = 0.f;
          for (int j = 0; j < DV; ++j) a += red[j * LR + d];
          dk[(row * H + h) * DK + d] = from_f<IO>(a);
        }
        if (threadIdx.x == 0) {
          if (VAR != VAR_DECAY) {
            float a = 0.f;
            for (int j = 0; j < DV; ++j) a += sc[0][j];
            dbeta[row * H + h] = a;
          }
          if (VAR != VAR_DELTA) {
            float a = 0.f;
            for (int j = 0; j < DV; ++j) a += sc[1][j];
            dg[row * H + h] = a;
          }
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
