// Gather of the kept tokens in their original order, with their positional
// indices (section "Inference-Time Token Pruning": the selected tokens are
// restored to their original order and keep their positions).
//
// One workgroup per kept row k: it stages the selection order in LDS, finds
// the index of rank k (indices are distinct, so the rank of an index is the
// number of smaller ones), writes it, and copies the row byte-exactly with
// 16-byte loads and stores, every load of a thread issued before its first
// store.  After an aborted selection every index is -1, every position -1
// and every row zero.
#include "internal.h"

namespace mapk {

namespace {

__global__ __launch_bounds__(256) void gather_kernel(const GatherArgs a) {
  extern __shared__ int ord[];  // [K rounded up to 8] the selection order (padding: past any index)
  __shared__ int found;
  const int b = blockIdx.y, k = blockIdx.x, K = a.K, K8 = (K + 7) & ~7;
  const int chunks = a.row_bytes >> 4;
  if (threadIdx.x == 0) found = -1;
  const bool aborted = __hip_atomic_load(a.err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0;
  for (int j = threadIdx.x; j < K8; j += 256) ord[j] = j < K ? a.order[(long long)b * K + j] : 0x7fffffff;
  __syncthreads();
  for (int j = threadIdx.x; j < K && !aborted; j += 256) {
    const int v = ord[j];
    int r4[4] = {0, 0, 0, 0};
    for (int q = 0; q < K8; q += 8) {  // eight LDS broadcasts per step, four counters
      const int4 x = *reinterpret_cast<const int4*>(ord + q);
      const int4 y = *reinterpret_cast<const int4*>(ord + q + 4);
      r4[0] += (x.x < v) + (y.x < v);
      r4[1] += (x.y < v) + (y.y < v);
      r4[2] += (x.z < v) + (y.z < v);
      r4[3] += (x.w < v) + (y.w < v);
    }
    if ((r4[0] + r4[1]) + (r4[2] + r4[3]) == k) found = v;
  }
  __syncthreads();
  const int i = found;
  const bool ok = !aborted && i >= 0 && i < a.N;
  const long long orow = (long long)b * K + a.out_off[b];  // the image's first output row
  if (threadIdx.x == 0) {
    a.idx_out[(long long)b * K + k] = ok ? i : -1;
    a.pos_out[orow + k] = ok ? a.pos_v[(long long)b * a.N + i] : -1;
  }
  if (a.qT) {  // layer-0 assembly: question rows k, k + K, ... of the image after its kept rows
    const int m0 = a.q_off[b], M = a.q_off[b + 1] - m0;
    const uint4* qs = static_cast<const uint4*>(a.qT) + (long long)m0 * chunks;
    uint4* qd = static_cast<uint4*>(a.V_out) + (orow + K) * chunks;
    for (int m = k; m < M; m += K) {
      for (int c = threadIdx.x; c < chunks; c += 256) qd[(long long)m * chunks + c] = qs[(long long)m * chunks + c];
      if (threadIdx.x == 0) a.pos_out[orow + K + m] = a.qpos[m0 + m];
    }
  }
  const uint4* src = static_cast<const uint4*>(a.V) + ((long long)b * a.N + (ok ? i : 0)) * chunks;
  uint4* dst = static_cast<uint4*>(a.V_out) + (orow + k) * chunks;
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

// Workgroup (x, image b) copies row x of the image's K + M_b rows (one
// workgroup per row: the copy is short, so the grid spreads it over the
// chip), 16 bytes per thread per step, and its position.
__global__ __launch_bounds__(256) void assemble_kernel(const AssembleArgs a) {
  const int b = blockIdx.y, K = a.K, M = a.t_off[b + 1] - a.t_off[b];
  const int l = blockIdx.x;
  if (l >= K + M) return;
  const int chunks = a.row_bytes >> 4, out0 = b * K + a.t_off[b];
  const uint4* src = l < K ? static_cast<const uint4*>(a.V_out) + ((long long)b * K + l) * chunks
                           : static_cast<const uint4*>(a.T) + ((long long)a.t_off[b] + l - K) * chunks;
  uint4* dst = static_cast<uint4*>(a.X) + (long long)(out0 + l) * chunks;
  for (int c = threadIdx.x; c < chunks; c += 256) dst[c] = src[c];
  if (threadIdx.x == 0) a.pos_x[out0 + l] = l < K ? a.pos_out[(long long)b * K + l] : a.pos_t[a.t_off[b] + l - K];
}

}  // namespace

hipError_t launch_assemble(const AssembleArgs& a, hipStream_t s) {
  if (a.B == 0 || a.max_rows == 0) return hipSuccess;
  return launch_kernel("assemble", assemble_kernel, dim3(a.max_rows, a.B), dim3(256), 0, s, a);
}

hipError_t launch_gather(const GatherArgs& a, hipStream_t s) {
  return launch_kernel("gather", gather_kernel, dim3(a.K, a.B), dim3(256),
                       sizeof(int) * static_cast<size_t>((a.K + 7) & ~7), s, a);
}

}  // namespace mapk
