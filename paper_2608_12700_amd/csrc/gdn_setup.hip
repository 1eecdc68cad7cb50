// Chunk map of packed variable-length input: sequence n's chunks start at
// chunk_off[n] = sum_{m<n} ceil(L_m / 64).  One wave, fixed summation order.
#include "gdn_common.hpp"
#include "gdn_launch.hpp"

namespace gdn {

__global__ __launch_bounds__(64) void k_chunk_offsets(const int* __restrict__ cu, int N,
                                                      int* __restrict__ chunk_off) {
  // each lane sums a contiguous run of sequences, then an exclusive scan over lanes
  const int l = threadIdx.x;
  const int per = (N + WAVE - 1) / WAVE;
  const int b = min(N, l * per), e = min(N, b + per);
  int local = 0;
  for (int n = b; n < e; ++n) local += (cu[n + 1] - cu[n] + CH - 1) / CH;
  int incl = local;
  for (int off = 1; off < WAVE; off <<= 1) {
    const int y = __shfl_up(incl, off, WAVE);
    if (l >= off) incl += y;
  }
  int run = incl - local;
  for (int n = b; n < e; ++n) {
    chunk_off[n] = run;
    run += (cu[n + 1] - cu[n] + CH - 1) / CH;
  }
  if (l == WAVE - 1) chunk_off[N] = incl;
}

hipError_t launch_chunk_offsets(const int* cu, int N, int* chunk_off, hipStream_t stream) {
  hipLaunchKernelGGL(k_chunk_offsets, dim3(1), dim3(WAVE), 0, stream, cu, N, chunk_off);
  return hipGetLastError();
}

}  // namespace gdn
