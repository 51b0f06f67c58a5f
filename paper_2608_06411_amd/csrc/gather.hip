// Gather of the kept tokens in their original order, with their positional
// indices (section "Inference-Time Token Pruning": the selected tokens are
// restored to their original order and keep their positions).
//
// One workgroup per kept row k: it finds the index of rank k in the
// selection order (indices are distinct, so the rank of an index is the
// number of smaller ones), writes it, and copies the row byte-exactly with
// 16-byte loads and stores, every load of a thread issued before its first
// store.  After an aborted selection every index is -1, every position -1
// and every row zero.
#include "internal.h"

namespace mapk {

namespace {

__global__ __launch_bounds__(256) void gather_kernel(const GatherArgs a) {
  __shared__ int found;
  const int b = blockIdx.y, k = blockIdx.x, K = a.K;
  const int chunks = a.row_bytes >> 4;
  if (threadIdx.x == 0) found = -1;
  __syncthreads();
  const bool aborted = __hip_atomic_load(a.err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0;
  const int32_t* ord = a.order + (long long)b * K;
  for (int j = threadIdx.x; j < K && !aborted; j += 256) {
    const int v = ord[j];
    int rank = 0;
    for (int q = 0; q < K; ++q) rank += ord[q] < v;
    if (rank == k) found = v;
  }
  __syncthreads();
  const int i = found;
  const bool ok = !aborted && i >= 0 && i < a.N;
  if (threadIdx.x == 0) {
    a.idx_out[(long long)b * K + k] = ok ? i : -1;
    a.pos_out[(long long)b * K + k] = ok ? a.pos_v[(long long)b * a.N + i] : -1;
  }
  const uint4* src = static_cast<const uint4*>(a.V) + ((long long)b * a.N + (ok ? i : 0)) * chunks;
  uint4* dst = static_cast<uint4*>(a.V_out) + ((long long)b * a.K + k) * chunks;
  constexpr int U = 4;  // 16-byte pieces per thread per batch (rows up to 16 KiB in one batch)
  for (int c0 = threadIdx.x; c0 < chunks; c0 += U * 256) {
    uint4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = src[min(c0 + u * 256, chunks - 1)];  // valid addresses, no branches
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int c = c0 + u * 256;
      if (c < chunks) dst[c] = ok ? v[u] : make_uint4(0u, 0u, 0u, 0u);
    }
  }
}

}  // namespace

hipError_t launch_gather(const GatherArgs& a, hipStream_t s) {
  return launch_kernel("gather", gather_kernel, dim3(a.K, a.B), dim3(256), 0, s, a);
}

}  // namespace mapk
