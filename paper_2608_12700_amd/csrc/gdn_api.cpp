// C ABI of the gated-delta-rule library (declared in include/gdn.h).
//
// Everything here is host code.  Argument validation touches no HIP API, so
// a malformed call returns its error code even on a machine without a GPU,
// and nothing is enqueued on an error.  Kernels are launched through the
// per-(dtype, variant) entry points of gdn_launch.hpp.
#include <stdint.h>
#include <string.h>

#include <new>

#include "gdn.h"
#include "gdn_launch.hpp"

namespace {

using namespace gdn;

constexpr int kChunk = 64;
constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) & ~(kAlign - 1); }

bool dims_supported(int dk, int dv) {
  return (dk == 64 || dk == 128) && (dv == 64 || dv == 128 || dv == 256);
}

struct Shape {
  int64_t B, T, H, dk, dv, N, chunks, NT;
  bool packed;
  int es;  // bytes per activation element
  int variant;
};

// Validates the problem description (sizes, variant, dtype, packed offsets).
gdn_status check_problem(const gdn_problem* p, Shape* s) {
  if (!p) return GDN_ERR_NULL;
  if (p->B < 0 || p->T < 0 || p->H < 0 || p->dk <= 0 || p->dv <= 0) return GDN_ERR_SHAPE;
  if (p->chunk != kChunk || !dims_supported(p->dk, p->dv)) return GDN_ERR_UNSUPPORTED;
  // row strides H * d (elements) must fit the kernels' 24-bit in-chunk offsets
  if ((int64_t)p->H * (p->dk > p->dv ? p->dk : p->dv) >= (int64_t)1 << 24) return GDN_ERR_UNSUPPORTED;
  if (p->io_dtype != GDN_F32 && p->io_dtype != GDN_BF16) return GDN_ERR_DTYPE;
  if (p->variant != GDN_GATED_DELTA && p->variant != GDN_DELTA && p->variant != GDN_DECAY_ONLY)
    return GDN_ERR_VARIANT;
  const bool packed = p->cu_seqlens_host != nullptr || p->cu_seqlens_dev != nullptr;
  s->B = p->B; s->T = p->T; s->H = p->H; s->dk = p->dk; s->dv = p->dv;
  s->packed = packed;
  s->es = p->io_dtype == GDN_BF16 ? 2 : 4;
  s->variant = p->variant;
  if (packed) {
    if (!p->cu_seqlens_host || !p->cu_seqlens_dev) return GDN_ERR_NULL;
    if (p->B != 1 || p->num_seqs < 0) return GDN_ERR_VARLEN;
    const int32_t* cu = p->cu_seqlens_host;
    if (cu[0] != 0) return GDN_ERR_VARLEN;
    int64_t chunks = 0;
    for (int n = 0; n < p->num_seqs; ++n) {
      if (cu[n + 1] < cu[n]) return GDN_ERR_VARLEN;
      chunks += (cu[n + 1] - cu[n] + kChunk - 1) / kChunk;
    }
    if (cu[p->num_seqs] != p->T) return GDN_ERR_VARLEN;
    s->N = p->num_seqs;
    s->chunks = chunks;
    s->NT = 0;
  } else {
    if (p->num_seqs != p->B) return GDN_ERR_SHAPE;
    s->N = p->B;
    s->NT = (p->T + kChunk - 1) / kChunk;
    s->chunks = s->N * s->NT;
  }
  // grid limits: chunks on grid x, N*H*value-tiles on grid x of the scans
  if (s->chunks > (int64_t)INT32_MAX || s->N * s->H * (s->dv / SCAN_BV) > (int64_t)INT32_MAX)
    return GDN_ERR_SHAPE;
  if (s->B * s->T * s->H > ((int64_t)1 << 40)) return GDN_ERR_SHAPE;
  return GDN_OK;
}

struct Region {
  const void* p;
  size_t n;
};

bool overlap(Region a, Region b) {
  if (!a.p || !b.p || a.n == 0 || b.n == 0) return false;
  const uintptr_t a0 = (uintptr_t)a.p, b0 = (uintptr_t)b.p;
  return a0 < b0 + b.n && b0 < a0 + a.n;
}

// Outputs may overlap neither each other nor any input.
gdn_status check_alias(const Region* in, int nin, const Region* out, int nout) {
  for (int i = 0; i < nout; ++i) {
    for (int j = 0; j < nin; ++j)
      if (overlap(out[i], in[j])) return GDN_ERR_ALIAS;
    for (int j = i + 1; j < nout; ++j)
      if (overlap(out[i], out[j])) return GDN_ERR_ALIAS;
  }
  return GDN_OK;
}

// Workspace layout: a bump allocator over the caller's buffer.
struct Bump {
  char* base;
  size_t off = 0;
  template <typename T>
  T* take(size_t count) {
    T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += align_up(count * sizeof(T));
    return p;
  }
};

size_t exact_scratch_floats(const Shape& s);

void layout_fwd(const Shape& s, char* base, FwdWs* w, size_t* total) {
  Bump b{base};
  const size_t tiles = (size_t)s.chunks * s.H;
  w->chunk_off = b.take<int>(s.packed ? s.N + 1 : 0);
  w->flag_prep = b.take<int>(tiles);
  w->flag_scan = b.take<int>((size_t)s.N * s.H * (s.dv / SCAN_BV));
  w->gcum = b.take<float>(tiles * kChunk);
  w->W = b.take<char>(tiles * kChunk * s.dk * s.es);
  w->U = b.take<float>(tiles * kChunk * s.dv);
  w->KhT = b.take<char>(tiles * kChunk * s.dk * s.es);
  w->P = b.take<char>(tiles * kChunk * kChunk * s.es);
  // diag(e^G) Q: only the generic scan reads it (the split bf16 scan of the
  // delta-rule members reads q)
  const bool split = s.es == 2 && s.variant != GDN_DECAY_ONLY;
  w->Qg = b.take<char>(split ? 0 : tiles * kChunk * s.dk * s.es);
  w->exact = nullptr;  // the exact forward needs no scratch
  *total = b.off;
}

void layout_bwd(const Shape& s, char* base, BwdWs* w, size_t* total) {
  Bump b{base};
  const size_t tiles = (size_t)s.chunks * s.H;
  w->chunk_off = b.take<int>(s.packed ? s.N + 1 : 0);
  w->flag_prep = b.take<int>(tiles);
  w->flag_grad = b.take<int>(tiles);
  w->flag_scan = b.take<int>((size_t)s.N * s.H * (s.dv / SCAN_BV));
  w->gcum = b.take<float>(tiles * kChunk);
  w->W = b.take<char>(tiles * kChunk * s.dk * s.es);
  w->QgT = b.take<char>(tiles * kChunk * s.dk * s.es);
  w->dOT = b.take<char>(s.es == 2 ? 0 : tiles * kChunk * s.dv * s.es);  // the bf16 scan reads dO
  w->PT = b.take<char>(tiles * kChunk * kChunk * s.es);
  w->T = b.take<char>(tiles * kChunk * kChunk * s.es);
  w->Kh = b.take<char>(s.es == 2 ? 0 : tiles * kChunk * s.dk * s.es);  // the bf16 scan reads k
  w->dh = b.take<char>(tiles * (size_t)s.dk * s.dv * s.es);
  w->dUT = b.take<char>(tiles * kChunk * s.dv * s.es);
  w->grad_scratch = b.take<char>(s.es == 4 ? tiles * (size_t)grad_region_bytes((int)s.dk, 4) : 0);
  w->exact = b.take<float>(exact_scratch_floats(s));
  *total = b.off;
}

// The exact (token-serial) backward keeps the states of one chunk per slot
// (EXACT_SLOTS in gdn_exact.hpp).
constexpr int kExactSlots = 16;
size_t exact_scratch_floats(const Shape& s) {
  return (size_t)kExactSlots * (kChunk + 2) * s.dk * s.dv;
}

void layout_cw_fwd(const Shape& s, char* base, CwFwdWs* w, size_t* total) {
  Bump b{base};
  const size_t tiles = (size_t)s.chunks * s.H;
  w->chunk_off = b.take<int>(s.packed ? s.N + 1 : 0);
  w->flag_prep = b.take<int>(tiles);
  w->flag_scan = b.take<int>((size_t)s.N * s.H * (s.dv / SCAN_BV));
  w->gC = b.take<float>(tiles * s.dk);
  // the scan's operands in the activation dtype
  w->W = b.take<char>(tiles * kChunk * s.dk * s.es);
  w->U = b.take<char>(tiles * kChunk * s.dv * s.es);
  w->KhT = b.take<char>(tiles * kChunk * s.dk * s.es);
  w->P = b.take<char>(tiles * kChunk * kChunk * s.es);
  w->Qg = b.take<char>(tiles * kChunk * s.dk * s.es);
  *total = b.off;
}

void layout_cw_bwd(const Shape& s, char* base, CwBwdWs* w, size_t* total) {
  Bump b{base};
  const size_t tiles = (size_t)s.chunks * s.H;
  const size_t ck = tiles * kChunk * s.dk, cv = tiles * kChunk * s.dv, cc = tiles * kChunk * kChunk;
  w->chunk_off = b.take<int>(s.packed ? s.N + 1 : 0);
  w->flag_prep = b.take<int>(tiles);
  w->flag_grad = b.take<int>(tiles);
  w->flag_scan = b.take<int>((size_t)s.N * s.H * (s.dv / SCAN_BV));
  w->gC = b.take<float>(tiles * s.dk);
  // the reverse scan's operands and outputs in the activation dtype
  w->WT = b.take<char>(ck * s.es);
  w->QgT = b.take<char>(ck * s.es);
  w->dOT = b.take<char>(cv * s.es);
  w->PT = b.take<char>(cc * s.es);
  w->Kh = b.take<char>(ck * s.es);
  w->dh = b.take<char>(tiles * (size_t)s.dk * s.dv * s.es);
  w->dUT = b.take<char>(cv * s.es);
  // the value-part gradient kernel's T and Gamma * Kb, also in the activation dtype
  w->T = b.take<char>(cc * s.es);
  w->KbG = b.take<char>(ck * s.es);
  // fp32 between the two gradient kernels
  w->dP = b.take<float>(cc);
  w->dA = b.take<float>(cc);
  w->X = b.take<float>(ck);
  w->dQg = b.take<float>(ck);
  w->dKh = b.take<float>(ck);
  w->hdh = b.take<float>(tiles * s.dk);
  w->exact = b.take<float>(exact_scratch_floats(s));
  *total = b.off;
}

// The channel-wise entry points: the problem's variant is not read (the gate
// pointers select the member).
gdn_status check_cw_problem(const gdn_problem* p, Shape* s) { return check_problem(p, s); }

Geo make_geo(const Shape& s, const gdn_problem* p, const int* chunk_off) {
  Geo g;
  g.B = (int)s.B; g.T = (int)s.T; g.H = (int)s.H; g.N = (int)s.N;
  g.NT = (int)s.NT;
  g.total_chunks = (int)s.chunks;
  g.cu = s.packed ? p->cu_seqlens_dev : nullptr;
  g.chunk_off = s.packed ? chunk_off : nullptr;
  return g;
}

bool need(const void* ptr, size_t bytes) { return bytes == 0 || ptr != nullptr; }

}  // namespace

extern "C" {

int64_t gdn_num_chunks(const gdn_problem* p) {
  Shape s;
  const gdn_status st = check_problem(p, &s);
  return st == GDN_OK ? s.chunks : (int64_t)st;
}

size_t gdn_fwd_workspace_size(const gdn_problem* p) {
  Shape s;
  if (check_problem(p, &s) != GDN_OK) return 0;
  FwdWs w;
  size_t total = 0;
  layout_fwd(s, nullptr, &w, &total);
  return total;
}

size_t gdn_bwd_workspace_size(const gdn_problem* p) {
  Shape s;
  if (check_problem(p, &s) != GDN_OK) return 0;
  BwdWs w;
  size_t total = 0;
  layout_bwd(s, nullptr, &w, &total);
  return total;
}

gdn_status gdn_fwd(const gdn_problem* p, const void* q, const void* k, const void* v, const float* g,
                   const float* beta, const float* S0, void* o, float* S_T, float* chunk_states,
                   void* workspace, size_t workspace_bytes, void* stream) {
  return gdn_fwd_ex(p, q, k, v, g, beta, S0, o, S_T, chunk_states, workspace, workspace_bytes, stream,
                    nullptr);
}

gdn_status gdn_fwd_ex(const gdn_problem* p, const void* q, const void* k, const void* v,
                      const float* g, const float* beta, const float* S0, void* o, float* S_T,
                      float* chunk_states, void* workspace, size_t workspace_bytes, void* stream,
                      void* const* events) {
  try {
    Shape s;
    gdn_status st = check_problem(p, &s);
    if (st != GDN_OK) return st;
    const size_t tok = (size_t)s.B * s.T * s.H;
    const size_t qk_b = tok * s.dk * s.es, v_b = tok * s.dv * s.es, gate_b = tok * sizeof(float);
    const size_t state_b = (size_t)s.N * s.H * s.dk * s.dv * sizeof(float);
    const size_t states_b = (size_t)s.chunks * s.H * s.dk * s.dv * sizeof(float);
    const bool has_g = p->variant != GDN_DELTA, has_b = p->variant != GDN_DECAY_ONLY;
    if ((has_g && tok && !g) || (!has_g && g) || (has_b && tok && !beta) || (!has_b && beta))
      return GDN_ERR_VARIANT;
    if (!need(q, qk_b) || !need(k, qk_b) || !need(v, v_b) || !need(o, v_b) || !need(S_T, state_b) ||
        !need(chunk_states, states_b))
      return GDN_ERR_NULL;
    size_t ws_need = 0;
    FwdWs w;
    layout_fwd(s, nullptr, &w, &ws_need);
    if (!workspace || workspace_bytes < ws_need || ((uintptr_t)workspace & (kAlign - 1)))
      return GDN_ERR_WORKSPACE;
    const Region in[] = {{q, qk_b}, {k, qk_b}, {v, v_b}, {g, has_g ? gate_b : 0},
                         {beta, has_b ? gate_b : 0}, {S0, S0 ? state_b : 0},
                         {s.packed ? p->cu_seqlens_dev : nullptr, s.packed ? (size_t)(s.N + 1) * 4 : 0}};
    const Region out[] = {{o, v_b}, {S_T, state_b}, {chunk_states, states_b}, {workspace, ws_need}};
    st = check_alias(in, 7, out, 4);
    if (st != GDN_OK) return st;

    layout_fwd(s, static_cast<char*>(workspace), &w, &ws_need);
    FwdArgs a;
    a.geo = make_geo(s, p, w.chunk_off);
    a.dk = (int)s.dk; a.dv = (int)s.dv; a.variant = p->variant;
    a.q = q; a.k = k; a.v = v; a.g = g; a.beta = beta; a.S0 = S0;
    a.o = o; a.ST = S_T; a.states = chunk_states; a.ws = w;
    a.stream = static_cast<hipStream_t>(stream);
    a.events = reinterpret_cast<hipEvent_t const*>(events);
    if (s.N * s.H == 0) {
      for (int i = 0; i <= NUM_STAGES; ++i) stage_mark(a.events, i, a.stream);
      return GDN_OK;
    }
    hipError_t e;
    const bool bf = p->io_dtype == GDN_BF16;
    switch (p->variant) {
      case GDN_GATED_DELTA: e = bf ? launch_fwd_var<DT_BF16, VAR_GATED>(a) : launch_fwd_var<DT_F32, VAR_GATED>(a); break;
      case GDN_DELTA: e = bf ? launch_fwd_var<DT_BF16, VAR_DELTA>(a) : launch_fwd_var<DT_F32, VAR_DELTA>(a); break;
      default: e = bf ? launch_fwd_var<DT_BF16, VAR_DECAY>(a) : launch_fwd_var<DT_F32, VAR_DECAY>(a); break;
    }
    return e == hipSuccess ? GDN_OK : GDN_ERR_HIP;
  } catch (...) {
    return GDN_ERR_HIP;
  }
}

gdn_status gdn_bwd(const gdn_problem* p, const void* q, const void* k, const void* v, const float* g,
                   const float* beta, const float* chunk_states, const void* dO, const float* dS_T,
                   void* dq, void* dk, void* dv, float* dg, float* dbeta, float* dS0, void* workspace,
                   size_t workspace_bytes, void* stream) {
  return gdn_bwd_ex(p, q, k, v, g, beta, chunk_states, dO, dS_T, dq, dk, dv, dg, dbeta, dS0, workspace,
                    workspace_bytes, stream, nullptr);
}

gdn_status gdn_bwd_ex(const gdn_problem* p, const void* q, const void* k, const void* v,
                      const float* g, const float* beta, const float* chunk_states, const void* dO,
                      const float* dS_T, void* dq, void* dk, void* dv, float* dg, float* dbeta,
                      float* dS0, void* workspace, size_t workspace_bytes, void* stream,
                      void* const* events) {
  try {
    Shape s;
    gdn_status st = check_problem(p, &s);
    if (st != GDN_OK) return st;
    const size_t tok = (size_t)s.B * s.T * s.H;
    const size_t qk_b = tok * s.dk * s.es, v_b = tok * s.dv * s.es, gate_b = tok * sizeof(float);
    const size_t state_b = (size_t)s.N * s.H * s.dk * s.dv * sizeof(float);
    const size_t states_b = (size_t)s.chunks * s.H * s.dk * s.dv * sizeof(float);
    const bool has_g = p->variant != GDN_DELTA, has_b = p->variant != GDN_DECAY_ONLY;
    if ((has_g && tok && !g) || (!has_g && g) || (has_b && tok && !beta) || (!has_b && beta))
      return GDN_ERR_VARIANT;
    if ((has_g && tok && !dg) || (!has_g && dg) || (has_b && tok && !dbeta) || (!has_b && dbeta))
      return GDN_ERR_VARIANT;
    if (!need(q, qk_b) || !need(k, qk_b) || !need(v, v_b) || !need(dO, v_b) ||
        !need(chunk_states, states_b) || !need(dq, qk_b) || !need(dk, qk_b) || !need(dv, v_b) ||
        !need(dS0, state_b))
      return GDN_ERR_NULL;
    size_t ws_need = 0;
    BwdWs w;
    layout_bwd(s, nullptr, &w, &ws_need);
    if (!workspace || workspace_bytes < ws_need || ((uintptr_t)workspace & (kAlign - 1)))
      return GDN_ERR_WORKSPACE;
    const Region in[] = {{q, qk_b}, {k, qk_b}, {v, v_b}, {g, has_g ? gate_b : 0},
                         {beta, has_b ? gate_b : 0}, {chunk_states, states_b}, {dO, v_b},
                         {dS_T, dS_T ? state_b : 0},
                         {s.packed ? p->cu_seqlens_dev : nullptr, s.packed ? (size_t)(s.N + 1) * 4 : 0}};
    const Region out[] = {{dq, qk_b}, {dk, qk_b}, {dv, v_b}, {dg, has_g ? gate_b : 0},
                          {dbeta, has_b ? gate_b : 0}, {dS0, state_b}, {workspace, ws_need}};
    st = check_alias(in, 9, out, 7);
    if (st != GDN_OK) return st;

    layout_bwd(s, static_cast<char*>(workspace), &w, &ws_need);
    BwdArgs a;
    a.geo = make_geo(s, p, w.chunk_off);
    a.dk = (int)s.dk; a.dv = (int)s.dv; a.variant = p->variant;
    a.q = q; a.k = k; a.v = v; a.g = g; a.beta = beta; a.states = chunk_states;
    a.dO = dO; a.dST = dS_T;
    a.dq = dq; a.dk_ = dk; a.dv_ = dv; a.dg = dg; a.dbeta = dbeta; a.dS0 = dS0; a.ws = w;
    a.stream = static_cast<hipStream_t>(stream);
    a.events = reinterpret_cast<hipEvent_t const*>(events);
    if (s.N * s.H == 0) {
      for (int i = 0; i <= NUM_STAGES; ++i) stage_mark(a.events, i, a.stream);
      return GDN_OK;
    }
    int dev = 0;
    a.num_cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&a.num_cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        a.num_cus < 1)
      return GDN_ERR_HIP;
    hipError_t e;
    const bool bf = p->io_dtype == GDN_BF16;
    switch (p->variant) {
      case GDN_GATED_DELTA: e = bf ? launch_bwd_var<DT_BF16, VAR_GATED>(a) : launch_bwd_var<DT_F32, VAR_GATED>(a); break;
      case GDN_DELTA: e = bf ? launch_bwd_var<DT_BF16, VAR_DELTA>(a) : launch_bwd_var<DT_F32, VAR_DELTA>(a); break;
      default: e = bf ? launch_bwd_var<DT_BF16, VAR_DECAY>(a) : launch_bwd_var<DT_F32, VAR_DECAY>(a); break;
    }
    return e == hipSuccess ? GDN_OK : GDN_ERR_HIP;
  } catch (...) {
    return GDN_ERR_HIP;
  }
}

size_t gdn_cw_fwd_workspace_size(const gdn_problem* p) {
  Shape s;
  if (check_cw_problem(p, &s) != GDN_OK) return 0;
  CwFwdWs w;
  size_t total = 0;
  layout_cw_fwd(s, nullptr, &w, &total);
  return total;
}

size_t gdn_cw_bwd_workspace_size(const gdn_problem* p) {
  Shape s;
  if (check_cw_problem(p, &s) != GDN_OK) return 0;
  CwBwdWs w;
  size_t total = 0;
  layout_cw_bwd(s, nullptr, &w, &total);
  return total;
}

gdn_status gdn_cw_fwd(const gdn_problem* p, const void* q, const void* k, const void* v, const float* g,
                      const float* b, const float* w, const float* S0, void* o, float* S_T,
                      float* chunk_states, void* workspace, size_t workspace_bytes, void* stream) {
  return gdn_cw_fwd_ex(p, q, k, v, g, b, w, S0, o, S_T, chunk_states, workspace, workspace_bytes, stream,
                       nullptr);
}

gdn_status gdn_cw_fwd_ex(const gdn_problem* p, const void* q, const void* k, const void* v,
                         const float* g, const float* b, const float* w, const float* S0, void* o,
                         float* S_T, float* chunk_states, void* workspace, size_t workspace_bytes,
                         void* stream, void* const* events) {
  try {
    Shape s;
    gdn_status st = check_cw_problem(p, &s);
    if (st != GDN_OK) return st;
    const size_t tok = (size_t)s.B * s.T * s.H;
    const size_t qk_b = tok * s.dk * s.es, v_b = tok * s.dv * s.es;  // activations
    const size_t gk_b = tok * s.dk * 4, gv_b = tok * s.dv * 4;        // gates (fp32)
    const size_t state_b = (size_t)s.N * s.H * s.dk * s.dv * sizeof(float);
    const size_t states_b = (size_t)s.chunks * s.H * s.dk * s.dv * sizeof(float);
    if (!need(q, qk_b) || !need(k, qk_b) || !need(v, v_b) || !need(o, v_b) || !need(S_T, state_b) ||
        !need(chunk_states, states_b))
      return GDN_ERR_NULL;
    size_t ws_need = 0;
    CwFwdWs ws;
    layout_cw_fwd(s, nullptr, &ws, &ws_need);
    if (!workspace || workspace_bytes < ws_need || ((uintptr_t)workspace & (kAlign - 1)))
      return GDN_ERR_WORKSPACE;
    const Region in[] = {{q, qk_b}, {k, qk_b}, {v, v_b}, {g, g ? gk_b : 0}, {b, b ? gk_b : 0},
                         {w, w ? gv_b : 0}, {S0, S0 ? state_b : 0},
                         {s.packed ? p->cu_seqlens_dev : nullptr, s.packed ? (size_t)(s.N + 1) * 4 : 0}};
    const Region out[] = {{o, v_b}, {S_T, state_b}, {chunk_states, states_b}, {workspace, ws_need}};
    st = check_alias(in, 8, out, 4);
    if (st != GDN_OK) return st;

    layout_cw_fwd(s, static_cast<char*>(workspace), &ws, &ws_need);
    CwFwdArgs a;
    a.geo = make_geo(s, p, ws.chunk_off);
    a.dk = (int)s.dk; a.dv = (int)s.dv; a.io = p->io_dtype == GDN_BF16 ? DT_BF16 : DT_F32;
    a.q = q; a.k = k; a.v = v; a.g = g; a.b = b; a.w = w; a.S0 = S0;
    a.o = o; a.ST = S_T; a.states = chunk_states; a.ws = ws;
    a.stream = static_cast<hipStream_t>(stream);
    a.events = reinterpret_cast<hipEvent_t const*>(events);
    if (s.N * s.H == 0) {
      for (int i = 0; i <= NUM_STAGES; ++i) stage_mark(a.events, i, a.stream);
      return GDN_OK;
    }
    return launch_cw_fwd(a) == hipSuccess ? GDN_OK : GDN_ERR_HIP;
  } catch (...) {
    return GDN_ERR_HIP;
  }
}

gdn_status gdn_cw_bwd(const gdn_problem* p, const void* q, const void* k, const void* v, const float* g,
                      const float* b, const float* w, const float* chunk_states, const void* dO,
                      const float* dS_T, void* dq, void* dk, void* dv, float* dg, float* db, float* dw,
                      float* dS0, void* workspace, size_t workspace_bytes, void* stream) {
  return gdn_cw_bwd_ex(p, q, k, v, g, b, w, chunk_states, dO, dS_T, dq, dk, dv, dg, db, dw, dS0, workspace,
                       workspace_bytes, stream, nullptr);
}

gdn_status gdn_cw_bwd_ex(const gdn_problem* p, const void* q, const void* k, const void* v,
                         const float* g, const float* b, const float* w, const float* chunk_states,
                         const void* dO, const float* dS_T, void* dq, void* dk, void* dv, float* dg,
                         float* db, float* dw, float* dS0, void* workspace, size_t workspace_bytes,
                         void* stream, void* const* events) {
  try {
    Shape s;
    gdn_status st = check_cw_problem(p, &s);
    if (st != GDN_OK) return st;
    const size_t tok = (size_t)s.B * s.T * s.H;
    const size_t qk_b = tok * s.dk * s.es, v_b = tok * s.dv * s.es;  // activations
    const size_t gk_b = tok * s.dk * 4, gv_b = tok * s.dv * 4;        // gates (fp32)
    const size_t state_b = (size_t)s.N * s.H * s.dk * s.dv * sizeof(float);
    const size_t states_b = (size_t)s.chunks * s.H * s.dk * s.dv * sizeof(float);
    // a gradient is written exactly for the gates that are given
    if ((g == nullptr) != (dg == nullptr) || (b == nullptr) != (db == nullptr) || (w == nullptr) != (dw == nullptr))
      return GDN_ERR_VARIANT;
    if (!need(q, qk_b) || !need(k, qk_b) || !need(v, v_b) || !need(dO, v_b) ||
        !need(chunk_states, states_b) || !need(dq, qk_b) || !need(dk, qk_b) || !need(dv, v_b) ||
        !need(dS0, state_b))
      return GDN_ERR_NULL;
    size_t ws_need = 0;
    CwBwdWs ws;
    layout_cw_bwd(s, nullptr, &ws, &ws_need);
    if (!workspace || workspace_bytes < ws_need || ((uintptr_t)workspace & (kAlign - 1)))
      return GDN_ERR_WORKSPACE;
    const Region in[] = {{q, qk_b}, {k, qk_b}, {v, v_b}, {g, g ? gk_b : 0}, {b, b ? gk_b : 0},
                         {w, w ? gv_b : 0}, {chunk_states, states_b}, {dO, v_b}, {dS_T, dS_T ? state_b : 0},
                         {s.packed ? p->cu_seqlens_dev : nullptr, s.packed ? (size_t)(s.N + 1) * 4 : 0}};
    const Region out[] = {{dq, qk_b}, {dk, qk_b}, {dv, v_b}, {dg, dg ? gk_b : 0}, {db, db ? gk_b : 0},
                          {dw, dw ? gv_b : 0}, {dS0, state_b}, {workspace, ws_need}};
    st = check_alias(in, 10, out, 8);
    if (st != GDN_OK) return st;

    layout_cw_bwd(s, static_cast<char*>(workspace), &ws, &ws_need);
    CwBwdArgs a;
    a.geo = make_geo(s, p, ws.chunk_off);
    a.dk = (int)s.dk; a.dv = (int)s.dv; a.io = p->io_dtype == GDN_BF16 ? DT_BF16 : DT_F32;
    a.q = q; a.k = k; a.v = v; a.g = g; a.b = b; a.w = w; a.states = chunk_states; a.dO = dO; a.dST = dS_T;
    a.dq = dq; a.dk_ = dk; a.dv_ = dv; a.dg = dg; a.db = db; a.dw = dw; a.dS0 = dS0; a.ws = ws;
    a.stream = static_cast<hipStream_t>(stream);
    a.events = reinterpret_cast<hipEvent_t const*>(events);
    if (s.N * s.H == 0) {
      for (int i = 0; i <= NUM_STAGES; ++i) stage_mark(a.events, i, a.stream);
      return GDN_OK;
    }
    return launch_cw_bwd(a) == hipSuccess ? GDN_OK : GDN_ERR_HIP;
  } catch (...) {
    return GDN_ERR_HIP;
  }
}

const char* gdn_status_str(gdn_status s) {
  switch (s) {
    case GDN_OK: return "ok";
    case GDN_ERR_NULL: return "a required pointer is NULL";
    case GDN_ERR_SHAPE: return "negative or inconsistent sizes";
    case GDN_ERR_UNSUPPORTED: return "unsupported chunk, d_k or d_v";
    case GDN_ERR_DTYPE: return "unknown io_dtype";
    case GDN_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
    case GDN_ERR_ALIAS: return "an output overlaps an input or another output";
    case GDN_ERR_VARLEN: return "malformed cu_seqlens";
    case GDN_ERR_HIP: return "kernel launch failed";
    case GDN_ERR_VARIANT: return "unknown variant or gate pointers inconsistent with it";
    case GDN_ERR_TOO_LARGE: return "workspace larger than the no-allocation scratch array";
  }
  return "unknown status";
}

const char* gdn_version(void) { return "gdn-mi355x 0.1 (gfx950)"; }

}  // extern "C"
