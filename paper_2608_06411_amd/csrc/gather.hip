// Gather of the kept tokens in their original order, with their positional
// indices (section "Inference-Time Token Pruning": the selected tokens are
// restored to their original order and keep their positions).
//
// A byte-exact copy: each workgroup moves kRows rows with 16-byte loads and
// stores, consecutive threads on consecutive chunks of a row.
#include "internal.h"

namespace mapk {

namespace {

constexpr int kRows = 8;

__global__ __launch_bounds__(256) void gather_kernel(const GatherArgs a) {
  __shared__ int rows[kRows];
  const int b = blockIdx.y, k0 = blockIdx.x * kRows;
  const int chunks = a.row_bytes >> 4;
  const int nrows = min(kRows, a.K - k0);
  if (threadIdx.x < nrows) {
    const int k = k0 + threadIdx.x;
    const int i = a.idx[(long long)b * a.K + k];
    const bool ok = i >= 0 && i < a.N;  // -1 marks an aborted selection
    rows[threadIdx.x] = ok ? i : -1;
    a.pos_out[(long long)b * a.K + k] = ok ? a.pos_v[(long long)b * a.N + i] : -1;
  }
  __syncthreads();
  const uint4* src = static_cast<const uint4*>(a.V) + (long long)b * a.N * chunks;
  uint4* dst = static_cast<uint4*>(a.V_out) + ((long long)b * a.K + k0) * chunks;
  const int total = nrows * chunks;
  constexpr int U = 8;  // independent 16-byte loads in flight per thread
  for (int e0 = threadIdx.x; e0 < total; e0 += U * 256) {
    uint4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int e = e0 + u * 256;
      v[u] = make_uint4(0u, 0u, 0u, 0u);
      if (e < total) {
        const int r = e / chunks, c = e - r * chunks;
        if (rows[r] >= 0) v[u] = src[(long long)rows[r] * chunks + c];
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int e = e0 + u * 256;
      if (e < total) dst[e] = v[u];
    }
  }
}

}  // namespace

hipError_t launch_gather(const GatherArgs& a, hipStream_t s) {
  return launch_kernel("gather", gather_kernel, dim3((a.K + kRows - 1) / kRows, a.B), dim3(256), 0, s, a);
}

}  // namespace mapk
