// Teacher selection for predictor training (section "Question Contrastive
// Teacher Selection", Eq. (1)-(2), and QCTS-n of the teacher ablation).
//
// Three launches per call:
//  * attn_colsum: the HBM-bound part.  Sample b's attention for layer l is a
//    slab of H*M rows (heads, then question tokens) of N visual tokens.  A
//    workgroup sums a slice of those rows for 64*VEC columns (16-byte loads,
//    four waves on interleaved rows) and writes one float32 partial row.
//    Input and reference question share the launch (grid z).
//  * layer_js: per (layer, sample) the partial rows summed in slice order,
//    their totals (Eq. (1)'s 1/(H M) cancels in the l1 normalisation), p^l
//    and p^l_ref, and D_JS(p^l, p^l_ref) in float64 with the natural log.
//  * teacher: per sample the layers ranked by divergence (ties to the lower
//    layer), and the mean of p^l over the n_top highest (Eq. (2) for n = 1).
// Every sum runs in a fixed order: the results are bitwise deterministic.
#include "internal.h"

namespace mapk {

namespace {

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
    int r = r_lo + w;
    for (; r + 12 < r_hi; r += 16) {
      const uint4 v0 = src[(long long)r * stride], v1 = src[(long long)(r + 4) * stride];
      const uint4 v2 = src[(long long)(r + 8) * stride], v3 = src[(long long)(r + 12) * stride];
      accumulate<BF16>(acc, v0);
      accumulate<BF16>(acc, v1);
      accumulate<BF16>(acc, v2);
      accumulate<BF16>(acc, v3);
    }
    for (; r < r_hi; r += 4) accumulate<BF16>(acc, src[(long long)r * stride]);
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

__global__ __launch_bounds__(256) void layer_js_kernel(const TeacherArgs a) {
  __shared__ double red[256];
  const int l = blockIdx.x, b = blockIdx.y, N = a.N, S = a.S;
  const float* q = a.part + (((long long)b * a.L + l) * S) * N;
  const float* r = a.part + (((long long)(a.B + b) * a.L + l) * S) * N;
  double tq = 0.0, tr = 0.0;
  for (int n = threadIdx.x; n < N; n += 256) {
    float aq = 0.0f, ar = 0.0f;
    for (int s = 0; s < S; ++s) {
      aq += q[(long long)s * N + n];
      ar += r[(long long)s * N + n];
    }
    tq += aq;
    tr += ar;
  }
  tq = block_sum(tq, red);
  tr = block_sum(tr, red);
  float* p_out = a.p + ((long long)b * a.L + l) * N;
  float* pr_out = a.p_ref + ((long long)b * a.L + l) * N;
  double js = 0.0;
  for (int n = threadIdx.x; n < N; n += 256) {
    float aq = 0.0f, ar = 0.0f;
    for (int s = 0; s < S; ++s) {
      aq += q[(long long)s * N + n];
      ar += r[(long long)s * N + n];
    }
    const double pd = tq > 0.0 ? aq / tq : 1.0 / N, qd = tr > 0.0 ? ar / tr : 1.0 / N;
    p_out[n] = static_cast<float>(pd);
    pr_out[n] = static_cast<float>(qd);
    const double m = 0.5 * (pd + qd);
    js += 0.5 * ((pd > 0.0 ? pd * log(pd / m) : 0.0) + (qd > 0.0 ? qd * log(qd / m) : 0.0));
  }
  js = block_sum(js, red);
  if (threadIdx.x == 0) a.js[(long long)b * a.L + l] = js;
}

__global__ __launch_bounds__(256) void teacher_kernel(const TeacherArgs a) {
  __shared__ int top[kTeacherMaxLayers];
  const int b = blockIdx.x, L = a.L, tid = threadIdx.x;
  top[tid] = 0;
  __syncthreads();
  const double* js = a.js + (long long)b * L;
  if (tid < L) {
    // a divergence is >= 0; a NaN ranks below every number
    const double mine = js[tid] >= 0.0 ? js[tid] : -1.0;
    int rank = 0;
    for (int k = 0; k < L; ++k) {
      const double o = js[k] >= 0.0 ? js[k] : -1.0;
      rank += (o > mine) || (o == mine && k < tid);
    }
    if (rank < a.n_top) {
      top[rank] = tid;
      a.layers[(long long)b * a.n_top + rank] = tid;
    }
  }
  __syncthreads();
  const double inv = 1.0 / a.n_top;
  for (int n = tid; n < a.N; n += 256) {
    double s = 0.0;
    for (int k = 0; k < a.n_top; ++k) s += a.p[((long long)b * L + top[k]) * a.N + n];
    a.teacher[(long long)b * a.N + n] = static_cast<float>(s * inv);
  }
}

}  // namespace

hipError_t launch_teacher(map_dtype dt, const TeacherArgs& a, hipStream_t s) {
  const int vec = dt == MAP_BF16 ? 8 : 4;
  const dim3 g((a.N + 64 * vec - 1) / (64 * vec) * a.S, a.L, 2 * a.B);
  hipError_t e = dt == MAP_BF16 ? launch_kernel("attn_colsum", attn_colsum_kernel<true>, g, dim3(256), 0, s, a)
                                : launch_kernel("attn_colsum", attn_colsum_kernel<false>, g, dim3(256), 0, s, a);
  if (e != hipSuccess) return e;
  e = launch_kernel("layer_js", layer_js_kernel, dim3(a.L, a.B), dim3(256), 0, s, a);
  if (e != hipSuccess) return e;
  return launch_kernel("teacher", teacher_kernel, dim3(a.B), dim3(256), 0, s, a);
}

}  // namespace mapk
