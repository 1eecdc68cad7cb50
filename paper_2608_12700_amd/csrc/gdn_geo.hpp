// Plain data shared by host and device code (no device intrinsics here).
#pragma once

namespace gdn {

enum { VAR_GATED = 0, VAR_DELTA = 1, VAR_DECAY = 2 };  // family member
enum { DT_F32 = 0, DT_BF16 = 1 };                      // operand / I/O dtype

struct Geo {
  int B, T, H, N;        // N sequences
  int NT;                // chunks per sequence (fixed-length layout only)
  int total_chunks;
  const int* cu;         // device cu_seqlens [N+1] or nullptr
  const int* chunk_off;  // device [N+1] chunk offsets (packed layout) or nullptr
};

}  // namespace gdn
