// Host-side launch interface between the C ABI (gdn_api.cpp) and the kernel
// translation units.  Plain structs of device pointers and sizes.
#pragma once

#include <hip/hip_runtime_api.h>

#include "gdn_geo.hpp"

namespace gdn {

// Forward workspace regions (device pointers into the caller's workspace).
struct FwdWs {
  int* chunk_off;  // [N+1] packed layout only
  int* flag_prep;  // [chunks*H]   non-finite q, k, v, g, beta in the chunk
  int* flag_scan;  // [N*H*NVT]    non-finite S0 slice
  float* gcum;     // [chunks*H*64] in-chunk cumulative log-decay
  void* W;         // [chunks*H*64*dk] operand dtype
  float* U;        // [chunks*H*64*dv] in the operand dtype (sized for fp32)
  void* KhT;       // [chunks*H*dk*64] operand dtype, (e^{G_last-G} K)^T
  void* P;         // [chunks*H*64*64] operand dtype, (Q K^T) * D
  void* Qg;        // [chunks*H*64*dk] operand dtype, diag(e^G) Q
  float* exact;    // exact-path scratch
};

struct FwdArgs {
  Geo geo;
  int dk, dv, variant;
  const void *q, *k, *v;
  const float *g, *beta, *S0;
  void* o;
  float* ST;
  float* states;
  FwdWs ws;
  hipStream_t stream;
  hipEvent_t const* events;  // nullptr, or NUM_STAGES + 1 events
};

struct BwdWs {
  int* chunk_off;
  int* flag_prep;  // [chunks*H]   non-finite q, k, g, beta (fp32: and dO) in the chunk
  int* flag_grad;  // [chunks*H]   non-finite chunk state, v or (bf16) dO in the chunk
  int* flag_scan;  // [N*H*NVT]    non-finite dS_T slice
  float* gcum;     // [chunks*H*64]
  void* W;         // [chunks*H*dk*64] operand dtype, W^T
  void* QgT;       // [chunks*H*dk*64] operand dtype, (diag(e^G) Q)^T
  void* dOT;       // [chunks*H*dv*64] operand dtype, dO^T (fp32 operands only)
  void* PT;        // [chunks*H*64*64] operand dtype, P^T
  void* T;         // [chunks*H*64*64] operand dtype, T = (I + A)^{-1}
  void* Kh;        // [chunks*H*64*dk] operand dtype, diag(e^{G_last - G}) K
  void* dh;        // [chunks*H*dk*dv] operand dtype: state gradient after each chunk
  void* dUT;       // [chunks*H*dv*64] operand dtype: dU' of each chunk, transposed
  void* grad_scratch;  // [chunks*H*grad_region_bytes] fp32 operands only
  float* exact;
};

struct BwdArgs {
  Geo geo;
  int dk, dv, variant;
  const void *q, *k, *v;
  const float *g, *beta, *states;
  const void* dO;
  const float* dST;
  void *dq, *dk_, *dv_;
  float *dg, *dbeta, *dS0;
  BwdWs ws;
  hipStream_t stream;
  hipEvent_t const* events;
  int num_cus;  // compute units of the device (grid of the persistent gradient kernel)
};

constexpr int NUM_STAGES = 4;

// Records events[i] on the stream when per-stage timing was requested.
inline void stage_mark(hipEvent_t const* events, int i, hipStream_t stream) {
  if (events) (void)hipEventRecord(events[i], stream);
}

// value-tile width of the state scans
constexpr int SCAN_BV = 32;

// Bytes of the phase-dependent working region of the backward grad kernel
// (held in LDS for bf16 operands and in the workspace, one slice per block,
// for fp32 operands).  Must match GradRegion in gdn_bwd.hpp.
constexpr int grad_region_bytes(int dk, int es) {
  const int CHn = 64, P8 = 16 / es, LK = dk + P8, LT = CHn + P8, LC = CHn + 4, VS = 32, LV = VS + P8;
  const bool bf = es == 2;
  const int ph0 = CHn * LK * es + CHn * LC * 4 + (bf ? CHn * LC * 4 : 0) + 4 * 16 * 20 * 4;
  const int ph1 = (7 * CHn * LV + 2 * dk * LV + VS * LK + 2 * VS * LT) * es;
  const int ph2 = (2 * dk * LT + 4 * CHn * LT) * es;
  const int m = ph0 > ph1 ? (ph0 > ph2 ? ph0 : ph2) : (ph1 > ph2 ? ph1 : ph2);
  return (m + 255) / 256 * 256;
}

// Channel-wise members (per-channel g, b, w; fp32 or bf16 activations; the
// scans' operands in the activation dtype, everything else fp32).  A NULL gate is neutral: g = 0, b = 0 (no erase), w = 1.
struct CwFwdWs {
  int* chunk_off;
  int* flag_prep;  // [chunks*H]   non-finite q, k, v, g, b, w in the chunk
  int* flag_scan;  // [N*H*NVT]    non-finite S0 slice
  float* gC;       // [chunks*H*dk]    G of each chunk's last row, per channel
  // the scan's operands, in the activation dtype, op_off layout (U: accumulator tiles)
  void* W;         // [chunks*H*64*dk] T (Gamma * b * K)
  void* U;         // [chunks*H*64*dv] T (w * V)
  void* KhT;       // [chunks*H*dk*64] (e^{G_last - G} * K)^T
  void* P;         // [chunks*H*64*64] decay-weighted Q K^T, i <= r
  void* Qg;        // [chunks*H*64*dk] e^G * Q
};

struct CwFwdArgs {
  Geo geo;
  int dk, dv, io;  // io: DT_F32 or DT_BF16 (q, k, v, o)
  const void *q, *k, *v;
  const float *g, *b, *w, *S0;
  void* o;
  float *ST, *states;
  CwFwdWs ws;
  hipStream_t stream;
  hipEvent_t const* events;
};

struct CwBwdWs {
  int* chunk_off;
  int* flag_prep;  // [chunks*H]   non-finite q, k, g, b, dO in the chunk
  int* flag_grad;  // [chunks*H]   non-finite v, w or chunk state in the chunk
  int* flag_scan;  // [N*H*NVT]    non-finite dS_T slice
  float* gC;   // [chunks*H*dk]
  // the reverse scan's operands and outputs, in the activation dtype, op_off layout
  void* WT;    // [chunks*H*dk*64]
  void* QgT;   // [chunks*H*dk*64]
  void* dOT;   // [chunks*H*dv*64]
  void* PT;    // [chunks*H*64*64]
  void* Kh;    // [chunks*H*64*dk]
  void* dh;    // [chunks*H*dk*dv]
  void* dUT;   // [chunks*H*dv*64]
  // activation dtype, row-major, for the value-part gradient kernel
  void* T;     // [chunks*H*64*64]
  void* KbG;   // [chunks*H*64*dk] Gamma * b * K
  // fp32, between the two gradient kernels
  float* dP;   // [chunks*H*64*64]
  float* dA;   // [chunks*H*64*64]
  float* X;    // [chunks*H*64*dk]
  float* dQg;  // [chunks*H*64*dk]
  float* dKh;  // [chunks*H*64*dk]
  float* hdh;  // [chunks*H*dk]
  float* exact;  // the exact backward's per-slot chunk replay
};

struct CwBwdArgs {
  Geo geo;
  int dk, dv, io;  // io: DT_F32 or DT_BF16 (q, k, v, dO, dq, dk, dv)
  const void *q, *k, *v, *dO;
  const float *g, *b, *w, *states, *dST;
  void *dq, *dk_, *dv_;
  float *dg, *db, *dw, *dS0;
  CwBwdWs ws;
  hipStream_t stream;
  hipEvent_t const* events;
};

hipError_t launch_cw_fwd(const CwFwdArgs& a);
hipError_t launch_cw_bwd(const CwBwdArgs& a);

template <int DT, int VAR> hipError_t launch_fwd_var(const FwdArgs& a);
template <int DT, int VAR> hipError_t launch_bwd_var(const BwdArgs& a);

// chunk_off[n] = sum_{m<n} ceil((cu[m+1]-cu[m]) / 64), n = 0..N
hipError_t launch_chunk_offsets(const int* cu, int N, int* chunk_off, hipStream_t stream);

}  // namespace gdn
