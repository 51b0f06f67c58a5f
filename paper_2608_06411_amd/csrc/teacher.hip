// Teacher selection for predictor training (section "Question Contrastive
// Teacher Selection", Eq. (1)-(2), and QCTS-n of the teacher ablation).
//
// Four launches per call:
//  * attn_colsum: the HBM-bound part.  Sample b's attention for layer l is a
//    slab of H*M rows (heads, then question tokens) of N visual tokens.  A
//    workgroup sums a slice of those rows for 64*VEC columns (16-byte
//    non-temporal loads, eight rows in flight per thread, four waves on
//    interleaved rows) and writes one float32 partial row.
//    Input and reference question share the launch (grid z).
//  * layer_sum: per column the partial rows summed in slice order, and per
//    256-column chunk their float64 total.
//  * layer_js: per chunk, p^l and p^l_ref (the column sums over the layer's
//    total: Eq. (1)'s 1/(H M) cancels in the l1 normalisation) and the
//    chunk's share of D_JS(p^l, p^l_ref), float64, natural log.
//  * teacher: per sample the divergence of each layer (chunk shares summed
//    in order), the layers ranked by it (ties to the lower layer), and the
//    mean of p^l over the n_top highest (Eq. (2) for n = 1).
// Every sum runs in a fixed order: the results are bitwise deterministic.
#include "internal.h"

namespace mapk {

namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// 16-byte load that bypasses the caches' retention (data read once)
__device__ __forceinline__ uint4 load_once(const uint4* p) {
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}

template <bool BF16>
__device__ __forceinline__ void accumulate(float* acc, const uint4 v) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
  if constexpr (BF16) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      acc[2 * k] += __uint_as_float(w[k] << 16);
      acc[2 * k + 1] += __uint_as_float(w[k] & 0xffff0000u);
    }
  } else {
#pragma unroll
    for (int k = 0; k < 4; ++k) acc[k] += __uint_as_float(w[k]);
  }
}

template <bool BF16>
__global__ __launch_bounds__(256) void attn_colsum_kernel(const TeacherArgs a) {
  constexpr int VEC = BF16 ? 8 : 4;
  const int z = blockIdx.z, t = z >= a.B, b = z - (t ? a.B : 0), l = blockIdx.y;
  const int cb = blockIdx.x / a.S, s = blockIdx.x - cb * a.S;
  const int N = a.N, M = t ? a.M_ref : a.m_off[b + 1] - a.m_off[b];
  const int rows = a.H * M, per = (rows + a.S - 1) / a.S;
  const int r_lo = min(rows, s * per), r_hi = min(rows, r_lo + per);
  const long long slab = t ? ((long long)b * a.L + l) * rows
                           : (long long)a.L * a.H * a.m_off[b] + (long long)l * rows;  // in rows
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int col = (cb * 64 + lane) * VEC, stride = N / VEC;
  float acc[VEC];
#pragma unroll
  for (int e = 0; e < VEC; ++e) acc[e] = 0.0f;
  if (col < N) {
    const uint4* src = static_cast<const uint4*>(t ? a.A_ref : a.A) + slab * stride + col / VEC;
    // the attention is read once: non-temporal loads, eight rows in flight
    int r = r_lo + w;
    for (; r + 28 < r_hi; r += 32) {
      uint4 v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = load_once(src + (long long)(r + 4 * u) * stride);
#pragma unroll
      for (int u = 0; u < 8; ++u) accumulate<BF16>(acc, v[u]);
    }
    for (; r < r_hi; r += 4) accumulate<BF16>(acc, load_once(src + (long long)r * stride));
  }
  __shared__ float red[3][VEC * 64];
  if (w > 0) {
#pragma unroll
    for (int e = 0; e < VEC; ++e) red[w - 1][e * 64 + lane] = acc[e];
  }
  __syncthreads();
  if (w == 0 && col < N) {
    float out[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) out[e] = ((acc[e] + red[0][e * 64 + lane]) + red[1][e * 64 + lane]) + red[2][e * 64 + lane];
    float4* dst = reinterpret_cast<float4*>(a.part + (((long long)z * a.L + l) * a.S + s) * N + col);
#pragma unroll
    for (int q = 0; q < VEC / 4; ++q) dst[q] = make_float4(out[4 * q], out[4 * q + 1], out[4 * q + 2], out[4 * q + 3]);
  }
}

// Sum of one double per thread over the workgroup, in a fixed tree order.
__device__ double block_sum(double v, double* red) {
  const int tid = threadIdx.x;
  red[tid] = v;
  __syncthreads();
  for (int off = 128; off > 0; off >>= 1) {
    if (tid < off) red[tid] += red[tid + off];
    __syncthreads();
  }
  const double r = red[0];
  __syncthreads();
  return r;
}

// Per column n of layer l: the slice partials summed in slice order, written
// back over slice 0; per 256-column chunk the float64 sum of those sums.
__global__ __launch_bounds__(256) void layer_sum_kernel(const TeacherArgs a) {
  __shared__ double red[256];
  const int z = blockIdx.z, l = blockIdx.y, n = blockIdx.x * 256 + threadIdx.x, N = a.N, S = a.S;
  float* col = a.part + (((long long)z * a.L + l) * S) * N;
  float v = 0.0f;
  if (n < N) {
    for (int s = 0; s < S; ++s) v += col[(long long)s * N + n];
  }
  const double t = block_sum(v, red);
  if (n < N) col[n] = v;  // every slice of this column has been read by this thread
  if (threadIdx.x == 0) a.tot[((long long)z * a.L + l) * a.NB + blockIdx.x] = t;
}

// Per 256-column chunk of layer l: p and p_ref from the column sums and the
// layer totals (chunk totals summed in chunk order), and the chunk's share of
// D_JS in float64 with the natural log.
__global__ __launch_bounds__(256) void layer_js_kernel(const TeacherArgs a) {
  __shared__ double red[256];
  const int b = blockIdx.z, l = blockIdx.y, n = blockIdx.x * 256 + threadIdx.x, N = a.N, NB = a.NB;
  const double* tq_part = a.tot + ((long long)b * a.L + l) * NB;
  const double* tr_part = a.tot + ((long long)(a.B + b) * a.L + l) * NB;
  double tq = 0.0, tr = 0.0;
  for (int k = 0; k < NB; ++k) {
    tq += tq_part[k];
    tr += tr_part[k];
  }
  double term = 0.0;
  if (n < N) {
    const float aq = a.part[(((long long)b * a.L + l) * a.S) * N + n];
    const float ar = a.part[(((long long)(a.B + b) * a.L + l) * a.S) * N + n];
    const double pd = tq > 0.0 ? aq / tq : 1.0 / N, qd = tr > 0.0 ? ar / tr : 1.0 / N;
    a.p[((long long)b * a.L + l) * N + n] = static_cast<float>(pd);
    a.p_ref[((long long)b * a.L + l) * N + n] = static_cast<float>(qd);
    const double m = 0.5 * (pd + qd);
    term = 0.5 * ((pd > 0.0 ? pd * log(pd / m) : 0.0) + (qd > 0.0 ? qd * log(qd / m) : 0.0));
  }
  const double js = block_sum(term, red);
  if (threadIdx.x == 0) a.js_part[((long long)b * a.L + l) * NB + blockIdx.x] = js;
}

// Workgroup (chunk c, sample b): the divergence of every layer (chunk
// shares summed in chunk order) and their ranking, repeated by each chunk's
// workgroup (L <= 256 values); chunk 0 writes js and the ranked layers; each
// writes the teacher's 256 columns of its chunk.
__global__ __launch_bounds__(256) void teacher_kernel(const TeacherArgs a) {
  __shared__ int top[kTeacherMaxLayers];
  __shared__ double jsl[kTeacherMaxLayers];
  const int b = blockIdx.y, L = a.L, tid = threadIdx.x, first = blockIdx.x == 0;
  top[tid] = 0;
  if (tid < L) {
    const double* part = a.js_part + ((long long)b * L + tid) * a.NB;
    double js = 0.0;
    for (int k = 0; k < a.NB; ++k) js += part[k];
    if (first) a.js[(long long)b * L + tid] = js;
    // A divergence is >= 0: a negative sum is rounding of terms below log's
    // precision (p close to p_ref) and ranks as 0, tying with exact zeros
    // (lower layer first); a NaN ranks below every number.
    jsl[tid] = js != js ? -1.0 : (js > 0.0 ? js : 0.0);
  }
  __syncthreads();
  if (tid < L) {
    const double mine = jsl[tid];
    int rank = 0;
    for (int k = 0; k < L; ++k) rank += (jsl[k] > mine) || (jsl[k] == mine && k < tid);
    if (rank < a.n_top) {
      top[rank] = tid;
      if (first) a.layers[(long long)b * a.n_top + rank] = tid;
    }
  }
  __syncthreads();
  const int n = blockIdx.x * 256 + tid;
  if (n < a.N) {
    double s = 0.0;
    for (int k = 0; k < a.n_top; ++k) s += a.p[((long long)b * L + top[k]) * a.N + n];
    a.teacher[(long long)b * a.N + n] = static_cast<float>(s / a.n_top);
  }
}

}  // namespace

hipError_t launch_teacher(map_dtype dt, const TeacherArgs& a, hipStream_t s) {
  const int vec = dt == MAP_BF16 ? 8 : 4;
  const dim3 g((a.N + 64 * vec - 1) / (64 * vec) * a.S, a.L, 2 * a.B);
  hipError_t e = dt == MAP_BF16 ? launch_kernel("attn_colsum", attn_colsum_kernel<true>, g, dim3(256), 0, s, a)
                                : launch_kernel("attn_colsum", attn_colsum_kernel<false>, g, dim3(256), 0, s, a);
  if (e != hipSuccess) return e;
  e = launch_kernel("layer_sum", layer_sum_kernel, dim3(a.NB, a.L, 2 * a.B), dim3(256), 0, s, a);
  if (e != hipSuccess) return e;
  e = launch_kernel("layer_js", layer_js_kernel, dim3(a.NB, a.L, a.B), dim3(256), 0, s, a);
  if (e != hipSuccess) return e;
  return launch_kernel("teacher", teacher_kernel, dim3(a.NB, a.B), dim3(256), 0, s, a);
}

}  // namespace mapk
