/*
 * gdn.h — C ABI of the gated-delta-rule chunked forward and training backward
 * for AMD Instinct MI355X (gfx950).
 *
 * The operation (paper Sec. 4.1, Eq. (gdn), scalar gates b = w = beta and a
 * scalar log-decay g — the KDA row of the family table with a scalar gate):
 * for every sequence n and head h, a state S (d_k x d_v, fp32) evolves as
 *
 *     S_t = (I - beta_t k_t k_t^T) exp(g_t) S_{t-1} + beta_t k_t v_t^T,
 *     o_t = S_t^T q_t,
 *
 * starting from S0 and ending at S_T.  gdn_fwd computes o, S_T and the state
 * before every chunk of 64 tokens (the sequential inter-chunk carry of the
 * paper's chunked form, Sec. 4.2).  gdn_bwd computes the gradients of the
 * loss  sum(dO * o) + <dS_T, S_T>  with respect to q, k, v, g, beta and S0;
 * it walks the chunks in reverse with an fp32 state-gradient carry (the
 * reverse inter-chunk state scan, K#1 in Sec. 4.2) and differentiates the
 * chunk-local triangular solve T = (I + A)^{-1} by reusing T (the WY /
 * triangular-inverse VJP, K#2 in Sec. 4.2) without re-inverting.
 *
 * Family members (paper, table "One recurrence, five models"):
 *   GDN_GATED_DELTA  the recurrence above;
 *   GDN_DELTA        DeltaNet: g == 0 (g and dg are NULL);
 *   GDN_DECAY_ONLY   scalar-decay SSD / Mamba-2: S_t = exp(g_t) S_{t-1} + k_t v_t^T
 *                    (beta and dbeta are NULL).
 *
 * Layouts (row-major, token-major; every pointer is DEVICE memory unless
 * stated otherwise):
 *   q, k          [B, T, H, d_k]    io_dtype
 *   v, o, dO      [B, T, H, d_v]    io_dtype
 *   dq, dk        [B, T, H, d_k]    io_dtype
 *   dv            [B, T, H, d_v]    io_dtype
 *   g, beta       [B, T, H]         float32 (per-token scalars)
 *   dg, dbeta     [B, T, H]         float32
 *   S0, S_T, dS_T, dS0   [N, H, d_k, d_v]  float32, element S[k][v]
 *   chunk_states  [sum_n ceil(L_n / 64), H, d_k, d_v]  float32
 * Packed variable-length input: B = 1, T = sum_n L_n, sequence n occupies
 * tokens [cu_seqlens[n], cu_seqlens[n+1]), N = num_seqs.  Otherwise N = B and
 * every sequence has length T.  Sequence n's chunk states start at entry
 * sum_{m<n} ceil(L_m / 64); entry c holds the state before the sequence's
 * token 64 c (so its first entry equals S0).  The last chunk of a sequence may
 * be partial.  Only chunk_states carries data from gdn_fwd to gdn_bwd.
 *
 * io_dtype GDN_BF16 means bfloat16 activations with fp32 gates and states; the
 * chunk-local products then run on bf16 matrix cores with fp32 accumulation.
 * GDN_F32 keeps every operand in fp32 (fp32 matrix cores).
 *
 * Supported: chunk == 64, d_k in {64, 128}, d_v in {64, 128, 256}, T >= 0,
 * sequence lengths >= 0, H * d_v < 2^24 (the kernels form in-chunk row
 * offsets with 24-bit multiplies).  Anything else returns GDN_ERR_UNSUPPORTED.
 *
 * Non-finite inputs: a (sequence, head) stream whose inputs hold a NaN or Inf
 * is recomputed token by token in fp32 in the operation order written above,
 * so NaN/Inf land on exactly the outputs that order determines.
 *
 * Ownership and threading: the caller allocates every buffer, including the
 * workspace (size from gdn_*_workspace_size).  The library never allocates,
 * frees or synchronises; all work is enqueued on `stream` (a hipStream_t; NULL
 * is the default stream) and the call returns without waiting.  There is no
 * global mutable state: calls are reentrant and thread-safe; two calls that
 * share a workspace must not overlap on the device.  Workspace contents are
 * undefined between calls.
 *
 * Errors: every argument is validated on the host before anything is
 * enqueued; on error nothing is launched and no output is touched.  Outputs
 * whose byte ranges overlap an input or another output -> GDN_ERR_ALIAS.  A
 * failed launch returns GDN_ERR_HIP.  Device faults surface at the caller's
 * next synchronisation.  No C++ exception crosses this interface.
 *
 * Determinism: outputs are bitwise identical across runs for identical
 * inputs (no floating-point atomics; every output element has one writer and a
 * fixed reduction order).
 */
#ifndef GDN_H_
#define GDN_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  GDN_OK = 0,
  GDN_ERR_NULL = -1,        /* a required pointer is NULL */
  GDN_ERR_SHAPE = -2,       /* negative or inconsistent sizes */
  GDN_ERR_UNSUPPORTED = -3, /* chunk, d_k, d_v or H * d_v outside the supported set */
  GDN_ERR_DTYPE = -4,       /* unknown io_dtype */
  GDN_ERR_WORKSPACE = -5,   /* workspace NULL or smaller than required */
  GDN_ERR_ALIAS = -6,       /* an output overlaps an input or another output */
  GDN_ERR_VARLEN = -7,      /* cu_seqlens not 0-based, non-decreasing, ending at T */
  GDN_ERR_HIP = -8,         /* a kernel launch failed */
  GDN_ERR_VARIANT = -9,     /* unknown variant, or a gate pointer that the
                               variant forbids / requires */
  GDN_ERR_TOO_LARGE = -10   /* gdn_fwd_noalloc: the problem's workspace exceeds
                               GDN_NOALLOC_SCRATCH_BYTES */
} gdn_status;

typedef enum { GDN_F32 = 0, GDN_BF16 = 1 } gdn_dtype;

typedef enum {
  GDN_GATED_DELTA = 0,
  GDN_DELTA = 1,      /* g == 0: g and dg must be NULL */
  GDN_DECAY_ONLY = 2  /* no delta term: beta and dbeta must be NULL */
} gdn_variant;

typedef struct {
  int32_t B, T, H, dk, dv, chunk; /* chunk must be 64 */
  int32_t num_seqs;               /* N: B, or the number of packed sequences */
  /* Packed sequences: both NULL, or both non-NULL with identical contents
   * [num_seqs + 1].  The host copy is read during the call (validation and
   * chunk counts); the device copy is read by the kernels. */
  const int32_t* cu_seqlens_host;
  const int32_t* cu_seqlens_dev;
  gdn_dtype io_dtype;
  gdn_variant variant;
} gdn_problem;

/* Number of chunk states, sum_n ceil(L_n / 64); negative gdn_status on a
 * malformed problem. */
int64_t gdn_num_chunks(const gdn_problem* p);

/* Bytes of device workspace gdn_fwd / gdn_bwd need (0 on a malformed problem).
 * The workspace must be 256-byte aligned. */
size_t gdn_fwd_workspace_size(const gdn_problem* p);
size_t gdn_bwd_workspace_size(const gdn_problem* p);

/* Forward.  S0 may be NULL (zero initial state).  Writes o, S_T and
 * chunk_states. */
gdn_status gdn_fwd(const gdn_problem* p, const void* q, const void* k, const void* v,
                   const float* g, const float* beta, const float* S0, void* o, float* S_T,
                   float* chunk_states, void* workspace, size_t workspace_bytes, void* stream);

/* Backward.  chunk_states must hold gdn_fwd's output for the same inputs.
 * dS_T may be NULL (zero).  Writes dq, dk, dv, dg, dbeta and dS0. */
gdn_status gdn_bwd(const gdn_problem* p, const void* q, const void* k, const void* v,
                   const float* g, const float* beta, const float* chunk_states, const void* dO,
                   const float* dS_T, void* dq, void* dk, void* dv, float* dg, float* dbeta,
                   float* dS0, void* workspace, size_t workspace_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): gdn_fwd with
 * its workspace in a fixed array of GDN_NOALLOC_SCRATCH_BYTES that the library
 * itself holds in device memory, one per GPU, from its first use on that GPU
 * until the process ends.  Arguments, outputs, kernels and results are those
 * of gdn_fwd (bitwise); the caller still provides inputs and outputs.  The
 * call allocates and frees nothing.  A problem whose workspace
 * (gdn_fwd_workspace_size) exceeds the array returns GDN_ERR_TOO_LARGE before
 * anything is launched; a failed lookup of the array's device address returns
 * GDN_ERR_HIP.  All calls on one GPU share its array: calls that overlap in
 * time on one GPU (different streams or threads without ordering) race and
 * must be serialised by the caller.  The array keeps the last call's contents,
 * which no call depends on. */
#define GDN_NOALLOC_SCRATCH_BYTES (64u << 20)
gdn_status gdn_fwd_noalloc(const gdn_problem* p, const void* q, const void* k, const void* v,
                           const float* g, const float* beta, const float* S0, void* o, float* S_T,
                           float* chunk_states, void* stream);

/* Stages that gdn_fwd_ex / gdn_bwd_ex can bracket with events.  Forward:
 * 0 chunk prep (UT transform and the masked in-chunk scores), 1 forward state
 * scan with the chunk output, 2 exact token-serial pass for non-finite streams,
 * 3 empty.  Backward: 0 chunk prep, 1 reverse state scan, 2 chunk gradients,
 * 3 exact pass. */
#define GDN_NUM_STAGES 4

/* gdn_fwd / gdn_bwd with optional per-stage timing.  `events` is NULL or an
 * array of GDN_NUM_STAGES + 1 hipEvent_t handles created by the caller;
 * events[i] is recorded on `stream` right before stage i is enqueued and
 * events[GDN_NUM_STAGES] after the last one (a stage with nothing to do
 * records two adjacent events).  The kernels are exactly those of
 * gdn_fwd / gdn_bwd; argument checks and errors are the same. */
gdn_status gdn_fwd_ex(const gdn_problem* p, const void* q, const void* k, const void* v,
                      const float* g, const float* beta, const float* S0, void* o, float* S_T,
                      float* chunk_states, void* workspace, size_t workspace_bytes, void* stream,
                      void* const* events);
gdn_status gdn_bwd_ex(const gdn_problem* p, const void* q, const void* k, const void* v,
                      const float* g, const float* beta, const float* chunk_states, const void* dO,
                      const float* dS_T, void* dq, void* dk, void* dv, float* dg, float* dbeta,
                      float* dS0, void* workspace, size_t workspace_bytes, void* stream,
                      void* const* events);

/* ---------------------------------------------------------------------------
 * Channel-wise members (paper Sec. 4.1, Eq. (gdn) with its three gates per
 * channel; table "One recurrence, five models"):
 *
 *   S_t = (I - k_t (b_t * k_t)^T) Diag(exp(g_t)) S_{t-1} + k_t (w_t * v_t)^T,
 *   o_t = S_t^T q_t,
 *
 * g_t (log-decay) and b_t (erase) have d_k entries per token and head, w_t
 * (write) has d_v.  Each gate pointer may be NULL, which means its neutral
 * value: g = 0, b = 0 (no erase), w = 1.  The named members are gate settings:
 * full GDN (all three), KDA (b = w = beta_t broadcast over the channels),
 * GLA (g only), LA (none).
 *
 * Layouts as above, with g, b [B,T,H,d_k] and w [B,T,H,d_v] (and dg, db, dw)
 * fp32 row-major (packed sequences: B = 1 and cu_seqlens as above).  q, k, v,
 * o, dO, dq, dk, dv are in io_dtype (fp32 or bf16).  With GDN_F32 every
 * operand inside the chunked algorithm is fp32 (fp32 matrix cores).  With
 * GDN_BF16 the two scans and the value-part gradient products take bf16
 * operands, as gdn_fwd / gdn_bwd do (fp32 state and accumulation), while the
 * prep (cumulative decays, the decay-weighted products, the triangular
 * inverse) and the channel-part gradients compute in fp32.  `variant` is not
 * read.
 * chunk_states has the layout and meaning of gdn_fwd's.  The chunked kernels
 * form each decay exp(G_r - G_i) split at a reference row: for r and i in
 * different 16-token blocks a row between them, so for a decay (every g <= 0)
 * no factor exceeds 1; inside a block the row before it, used only where the
 * block's log-decay moves by at most 32 from that row in every channel
 * (factors within e^{+-64}), else exp(G_r - G_i) is formed per term.  A g > 0
 * (growth) is computed the same way and overflows where the true values do.
 * Non-finite inputs: a (sequence, head) stream whose inputs (q, k, v, g, b, w,
 * S0, and in the backward dO, dS_T and its chunk states) hold a NaN or Inf is
 * recomputed token by token in fp32 in the operation order written above, as
 * gdn_fwd / gdn_bwd do, so NaN/Inf land on exactly the outputs that order
 * determines; the workspace holds that pass's per-block scratch.
 * Ownership, workspace, aliasing and stream rules are those of gdn_fwd /
 * gdn_bwd; the workspace sizes come from the two functions below.
 * ------------------------------------------------------------------------- */
size_t gdn_cw_fwd_workspace_size(const gdn_problem* p);
size_t gdn_cw_bwd_workspace_size(const gdn_problem* p);

/* Forward: o [B,T,H,d_v], S_T and chunk_states as gdn_fwd. */
gdn_status gdn_cw_fwd(const gdn_problem* p, const void* q, const void* k, const void* v,
                      const float* g, const float* b, const float* w, const float* S0, void* o,
                      float* S_T, float* chunk_states, void* workspace, size_t workspace_bytes,
                      void* stream);

/* Backward of the loss sum(dO * o) + <dS_T, S_T> (dS_T may be NULL = zero).
 * dg, db, dw have the shapes of g, b, w and must be non-NULL exactly when the
 * gate is (else GDN_ERR_VARIANT); dq, dk, dv, dS0 as gdn_bwd. */
gdn_status gdn_cw_bwd(const gdn_problem* p, const void* q, const void* k, const void* v,
                      const float* g, const float* b, const float* w, const float* chunk_states,
                      const void* dO, const float* dS_T, void* dq, void* dk, void* dv, float* dg,
                      float* db, float* dw, float* dS0, void* workspace, size_t workspace_bytes,
                      void* stream);

/* With per-stage events as gdn_fwd_ex / gdn_bwd_ex.  Forward stages: 0 chunk
 * prep, 1 state scan with the chunk output, 2 exact token-serial pass for
 * non-finite streams, 3 empty.  Backward: 0 chunk prep, 1 reverse state scan,
 * 2 value-slice gradients (dv, dw and the chunk products), 3 channel gradients
 * (dq, dk, dg, db) followed by the exact pass for non-finite streams. */
gdn_status gdn_cw_fwd_ex(const gdn_problem* p, const void* q, const void* k, const void* v,
                         const float* g, const float* b, const float* w, const float* S0, void* o,
                         float* S_T, float* chunk_states, void* workspace, size_t workspace_bytes,
                         void* stream, void* const* events);
gdn_status gdn_cw_bwd_ex(const gdn_problem* p, const void* q, const void* k, const void* v,
                         const float* g, const float* b, const float* w, const float* chunk_states,
                         const void* dO, const float* dS_T, void* dq, void* dk, void* dv, float* dg,
                         float* db, float* dw, float* dS0, void* workspace, size_t workspace_bytes,
                         void* stream, void* const* events);

/* Static description of a status code. */
const char* gdn_status_str(gdn_status s);

/* Library version string. */
const char* gdn_version(void);

#ifdef __cplusplus
}
#endif

#endif /* GDN_H_ */
