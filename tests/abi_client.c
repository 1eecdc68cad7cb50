/*
 * A plain C99 caller of libgdn.so: the interface as a C program sees it, with
 * no Python or torch in between.  Built and driven by tests/test_abi_c_client.py.
 *
 *   abi_client host
 *       Host-side checks that need no GPU: chunk counts, workspace sizes and
 *       the status codes of malformed calls.  Prints "host checks passed".
 *   abi_client run IN OUT
 *       Reads a problem and its inputs from IN, allocates device memory with
 *       hipMalloc, runs gdn_fwd then gdn_bwd on the default stream, and writes
 *       every output to OUT.
 *
 * IN (little-endian): int32 magic 0x31444E47, B, T, H, dk, dv, io_dtype,
 * variant, num_seqs, packed, has_S0, has_dS_T; if packed, int32
 * cu_seqlens[num_seqs + 1]; then the arrays q, k, v, g (unless GDN_DELTA),
 * beta (unless GDN_DECAY_ONLY), S0 (if has_S0), dO, dS_T (if has_dS_T), each
 * row-major in its interface layout and element type (io_dtype elements are
 * raw bf16 or fp32).  OUT: o, S_T, chunk_states, dq, dk, dv, dg (unless
 * GDN_DELTA), dbeta (unless GDN_DECAY_ONLY), dS0, the same way.
 */
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "gdn.h"

#define MAGIC 0x31444E47

static int failures = 0;

static void expect_int(const char* what, long long got, long long want) {
  if (got != want) {
    fprintf(stderr, "FAIL %s: got %lld, want %lld\n", what, got, want);
    ++failures;
  }
}

static gdn_problem problem(int B, int T, int H, int dk, int dv) {
  gdn_problem p;
  memset(&p, 0, sizeof p);
  p.B = B;
  p.T = T;
  p.H = H;
  p.dk = dk;
  p.dv = dv;
  p.chunk = 64;
  p.num_seqs = B;
  p.io_dtype = GDN_BF16;
  p.variant = GDN_GATED_DELTA;
  return p;
}

static int host_checks(void) {
  printf("library %s\n", gdn_version());
  gdn_problem p = problem(2, 130, 3, 64, 64);
  expect_int("chunks, fixed length", gdn_num_chunks(&p), 2 * 3);
  const size_t wf = gdn_fwd_workspace_size(&p), wb = gdn_bwd_workspace_size(&p);
  if (wf == 0 || wb == 0 || wf % 256 != 0 || wb % 256 != 0) {
    fprintf(stderr, "FAIL workspace sizes %zu %zu\n", wf, wb);
    ++failures;
  }

  static const int32_t cu[] = {0, 5, 70, 70, 200};
  gdn_problem pk = problem(1, 200, 3, 128, 256);
  pk.num_seqs = 4;
  pk.cu_seqlens_host = cu;
  pk.cu_seqlens_dev = cu; /* only the host copy is read before a launch */
  expect_int("chunks, packed", gdn_num_chunks(&pk), 1 + 2 + 0 + 3);

  gdn_problem bad = p;
  bad.chunk = 32;
  expect_int("chunk 32", gdn_num_chunks(&bad), GDN_ERR_UNSUPPORTED);
  expect_int("workspace of a malformed problem", (long long)gdn_fwd_workspace_size(&bad), 0);
  bad = p;
  bad.dk = 96;
  expect_int("d_k 96", gdn_num_chunks(&bad), GDN_ERR_UNSUPPORTED);
  bad = p;
  bad.io_dtype = (gdn_dtype)7;
  expect_int("io_dtype 7", gdn_num_chunks(&bad), GDN_ERR_DTYPE);
  bad = p;
  bad.T = -1;
  expect_int("T -1", gdn_num_chunks(&bad), GDN_ERR_SHAPE);
  static const int32_t cu_bad[] = {0, 5, 70, 70, 199};
  bad = pk;
  bad.cu_seqlens_host = cu_bad;
  bad.cu_seqlens_dev = cu_bad;
  expect_int("cu_seqlens not ending at T", gdn_num_chunks(&bad), GDN_ERR_VARLEN);

  /* calls rejected before anything is enqueued: the addresses below are never
   * dereferenced (distinct, 1 GiB apart, the workspace 256-byte aligned) */
#define FAKE(i) ((void*)(uintptr_t)(((uint64_t)1 << 40) + ((uint64_t)(i) << 30)))
#define FAKEF(i) ((float*)FAKE(i))
  expect_int("NULL problem",
             gdn_fwd(NULL, FAKE(0), FAKE(1), FAKE(2), FAKEF(3), FAKEF(4), NULL, FAKE(5), FAKEF(6), FAKEF(7),
                     FAKE(8), wf, NULL),
             GDN_ERR_NULL);
  expect_int("NULL q",
             gdn_fwd(&p, NULL, FAKE(1), FAKE(2), FAKEF(3), FAKEF(4), NULL, FAKE(5), FAKEF(6), FAKEF(7), FAKE(8),
                     wf, NULL),
             GDN_ERR_NULL);
  expect_int("workspace one byte short",
             gdn_bwd(&p, FAKE(0), FAKE(1), FAKE(2), FAKEF(3), FAKEF(4), FAKEF(5), FAKE(6), NULL, FAKE(7), FAKE(8),
                     FAKE(9), FAKEF(10), FAKEF(11), FAKEF(12), FAKE(13), wb - 1, NULL),
             GDN_ERR_WORKSPACE);
  expect_int("output overlapping an input",
             gdn_fwd(&p, FAKE(0), FAKE(1), FAKE(2), FAKEF(3), FAKEF(4), NULL, FAKE(1), FAKEF(6), FAKEF(7),
                     FAKE(8), wf, NULL),
             GDN_ERR_ALIAS);
  bad = p;
  bad.variant = GDN_DELTA; /* DeltaNet takes no g */
  expect_int("g given to the DeltaNet member",
             gdn_fwd(&bad, FAKE(0), FAKE(1), FAKE(2), FAKEF(3), FAKEF(4), NULL, FAKE(5), FAKEF(6), FAKEF(7),
                     FAKE(8), wf, NULL),
             GDN_ERR_VARIANT);
  if (strlen(gdn_status_str(GDN_ERR_ALIAS)) == 0) {
    fprintf(stderr, "FAIL empty status string\n");
    ++failures;
  }
  if (failures) return 1;
  printf("host checks passed\n");
  return 0;
}

/* ---- run: file I/O and device buffers ---- */

static FILE* in_file;
static FILE* out_file;

static void* read_block(size_t bytes) {
  void* h = malloc(bytes ? bytes : 1);
  if (!h || fread(h, 1, bytes, in_file) != bytes) {
    fprintf(stderr, "short input (%zu bytes wanted)\n", bytes);
    exit(2);
  }
  void* dptr = NULL;
  if (hipMalloc(&dptr, bytes ? bytes : 1) != hipSuccess || hipMemcpy(dptr, h, bytes, hipMemcpyHostToDevice) != hipSuccess) {
    fprintf(stderr, "hipMalloc / hipMemcpy failed\n");
    exit(3);
  }
  free(h);
  return dptr;
}

static void* device_buffer(size_t bytes) {
  void* dptr = NULL;
  if (hipMalloc(&dptr, bytes ? bytes : 1) != hipSuccess) {
    fprintf(stderr, "hipMalloc failed\n");
    exit(3);
  }
  return dptr;
}

static void write_block(const void* dptr, size_t bytes) {
  void* h = malloc(bytes ? bytes : 1);
  if (!h || hipMemcpy(h, dptr, bytes, hipMemcpyDeviceToHost) != hipSuccess || fwrite(h, 1, bytes, out_file) != bytes) {
    fprintf(stderr, "copy-out failed\n");
    exit(3);
  }
  free(h);
}

static int run(const char* in_path, const char* out_path) {
  in_file = fopen(in_path, "rb");
  if (!in_file) return 2;
  int32_t hd[12];
  if (fread(hd, sizeof(int32_t), 12, in_file) != 12 || hd[0] != MAGIC) {
    fprintf(stderr, "bad input header\n");
    return 2;
  }
  gdn_problem p = problem(hd[1], hd[2], hd[3], hd[4], hd[5]);
  p.io_dtype = (gdn_dtype)hd[6];
  p.variant = (gdn_variant)hd[7];
  p.num_seqs = hd[8];
  const int packed = hd[9], has_S0 = hd[10], has_dST = hd[11];
  int32_t* cu_host = NULL;
  if (packed) {
    const size_t cb = (size_t)(p.num_seqs + 1) * sizeof(int32_t);
    cu_host = (int32_t*)malloc(cb);
    if (fread(cu_host, 1, cb, in_file) != cb) return 2;
    void* cu_dev = device_buffer(cb);
    if (hipMemcpy(cu_dev, cu_host, cb, hipMemcpyHostToDevice) != hipSuccess) return 3;
    p.cu_seqlens_host = cu_host;
    p.cu_seqlens_dev = (const int32_t*)cu_dev;
  }
  const int64_t nch = gdn_num_chunks(&p);
  if (nch < 0) {
    fprintf(stderr, "malformed problem: %s\n", gdn_status_str((gdn_status)nch));
    return 4;
  }
  const size_t es = p.io_dtype == GDN_BF16 ? 2 : 4;
  const size_t tok = (size_t)p.B * p.T * p.H;
  const size_t qk = tok * p.dk * es, vb = tok * p.dv * es, gb = tok * sizeof(float);
  const size_t sb = (size_t)p.num_seqs * p.H * p.dk * p.dv * sizeof(float);
  const size_t stb = (size_t)nch * p.H * p.dk * p.dv * sizeof(float);
  const int has_g = p.variant != GDN_DELTA, has_beta = p.variant != GDN_DECAY_ONLY;

  void* q = read_block(qk);
  void* k = read_block(qk);
  void* v = read_block(vb);
  float* g = has_g ? (float*)read_block(gb) : NULL;
  float* beta = has_beta ? (float*)read_block(gb) : NULL;
  float* S0 = has_S0 ? (float*)read_block(sb) : NULL;
  void* dO = read_block(vb);
  float* dST = has_dST ? (float*)read_block(sb) : NULL;
  fclose(in_file);

  void* o = device_buffer(vb);
  float* S_T = (float*)device_buffer(sb);
  float* states = (float*)device_buffer(stb);
  void* dq = device_buffer(qk);
  void* dk = device_buffer(qk);
  void* dv = device_buffer(vb);
  float* dg = has_g ? (float*)device_buffer(gb) : NULL;
  float* db = has_beta ? (float*)device_buffer(gb) : NULL;
  float* dS0 = (float*)device_buffer(sb);
  const size_t wfb = gdn_fwd_workspace_size(&p), wbb = gdn_bwd_workspace_size(&p);
  void* wf = device_buffer(wfb);
  void* wb = device_buffer(wbb);

  gdn_status st = gdn_fwd(&p, q, k, v, g, beta, S0, o, S_T, states, wf, wfb, NULL);
  if (st != GDN_OK) {
    fprintf(stderr, "gdn_fwd: %s\n", gdn_status_str(st));
    return 5;
  }
  st = gdn_bwd(&p, q, k, v, g, beta, states, dO, dST, dq, dk, dv, dg, db, dS0, wb, wbb, NULL);
  if (st != GDN_OK) {
    fprintf(stderr, "gdn_bwd: %s\n", gdn_status_str(st));
    return 5;
  }
  if (hipDeviceSynchronize() != hipSuccess) {
    fprintf(stderr, "device error\n");
    return 6;
  }

  out_file = fopen(out_path, "wb");
  if (!out_file) return 2;
  write_block(o, vb);
  write_block(S_T, sb);
  write_block(states, stb);
  write_block(dq, qk);
  write_block(dk, qk);
  write_block(dv, vb);
  if (has_g) write_block(dg, gb);
  if (has_beta) write_block(db, gb);
  write_block(dS0, sb);
  fclose(out_file);
  printf("ran %lld chunks\n", (long long)nch);
  return 0;
}

int main(int argc, char** argv) {
  if (argc >= 2 && strcmp(argv[1], "host") == 0) return host_checks();
  if (argc >= 4 && strcmp(argv[1], "run") == 0) return run(argv[2], argv[3]);
  fprintf(stderr, "usage: abi_client host | abi_client run IN OUT\n");
  return 2;
}
