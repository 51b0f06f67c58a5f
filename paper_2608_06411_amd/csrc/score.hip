// Predicted attention, Eq. (3): logits, softmax over the visual tokens and
// the mean over the question tokens.
//
// logits_kernel: one workgroup per (block of 64 visual tokens, chunk of 16
// question tokens, image).  The block's keys and the chunk's queries sit in
// LDS; each thread forms q.k / sqrt(d_p) in float32 for one query and four
// keys, and the 16 lanes that share a query also emit the running (max, sum
// of exp) of its 64 logits, so that no pass over a whole logits row is needed
// later.
//
// softmax_mean_kernel: one workgroup per (block of 64 visual tokens, image).
// Each workgroup folds the per-block partials of its image into the row
// statistics (max_m, sum_m), four threads per row with all loads in flight,
// then for its 64 tokens averages exp(l_mn - max_m) / sum_m over m.  The sums
// run in a fixed order, so the result is bitwise reproducible.
#include "internal.h"

namespace mapk {

namespace {

constexpr int KB = 64;    // visual tokens per workgroup
constexpr int QB = 16;    // question tokens per workgroup
constexpr int DPAD = 132; // padded LDS row (d_p <= 128): 4 times an odd number, 16-byte aligned

__global__ __launch_bounds__(256) void logits_kernel(const ScoreArgs a) {
  __shared__ float ks[KB][DPAD];
  __shared__ float qs[QB][DPAD];
  const int blk = blockIdx.x, q0 = blockIdx.y * QB, b = blockIdx.z, tid = threadIdx.x;
  const int n0 = blk * KB, dp = a.d_p;
  const int mb = a.t_off[b], M = a.t_off[b + 1] - mb;
  if (q0 >= M) return;
  const float scale = 1.0f / sqrtf(static_cast<float>(dp));
  const int q4 = dp >> 2;
  {  // keys and queries: float4 loads at clamped addresses, all issued before the LDS stores
    constexpr int U = (KB + QB) * 32 / 256;  // pieces per thread for d_p = 128
    float4 v[U];
    const int kt = KB * q4, total = (KB + QB) * q4;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int e = min(tid + u * 256, total - 1);
      const bool key = e < kt;
      const int r = key ? e / q4 : (e - kt) / q4, d4 = key ? e - r * q4 : (e - kt) - r * q4;
      const float* src = key ? a.k + ((long long)b * a.N + min(n0 + r, a.N - 1)) * dp
                             : a.q + (long long)(mb + min(q0 + r, M - 1)) * dp;
      v[u] = *reinterpret_cast<const float4*>(src + 4 * d4);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int e = tid + u * 256;
      if (e >= total) continue;
      const bool key = e < kt;
      const int r = key ? e / q4 : (e - kt) / q4, d4 = key ? e - r * q4 : (e - kt) - r * q4;
      float* dst = key ? &ks[r][4 * d4] : &qs[r][4 * d4];
      dst[0] = v[u].x; dst[1] = v[u].y; dst[2] = v[u].z; dst[3] = v[u].w;
    }
    for (int e = tid + U * 256; e < total; e += 256) {  // (not reached for d_p <= 128)
      const bool key = e < kt;
      const int r = key ? e / q4 : (e - kt) / q4, d4 = key ? e - r * q4 : (e - kt) - r * q4;
      const float* src = key ? a.k + ((long long)b * a.N + min(n0 + r, a.N - 1)) * dp
                             : a.q + (long long)(mb + min(q0 + r, M - 1)) * dp;
      const float4 x = *reinterpret_cast<const float4*>(src + 4 * d4);
      float* dst = key ? &ks[r][4 * d4] : &qs[r][4 * d4];
      dst[0] = x.x; dst[1] = x.y; dst[2] = x.z; dst[3] = x.w;
    }
  }
  __syncthreads();
  const int tm = tid >> 4, tn = tid & 15;  // query q0 + tm, keys 4 tn .. 4 tn + 3
  float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll 4
  for (int d = 0; d < dp; d += 4) {  // d_p is a multiple of 4
    const float4 qv = *reinterpret_cast<const float4*>(&qs[tm][d]);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float4 kv = *reinterpret_cast<const float4*>(&ks[4 * tn + j][d]);
      acc[j] = fmaf(qv.x, kv.x, acc[j]);
      acc[j] = fmaf(qv.y, kv.y, acc[j]);
      acc[j] = fmaf(qv.z, kv.z, acc[j]);
      acc[j] = fmaf(qv.w, kv.w, acc[j]);
    }
  }
  const int m = q0 + tm;
  float mx = -INFINITY;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    acc[j] *= scale;
    if (n0 + 4 * tn + j < a.N) mx = fmaxf(mx, acc[j]);
  }
  if (m < M) {
    float* row = a.logits + (long long)(mb + m) * a.N + n0 + 4 * tn;
    if ((a.N & 3) == 0 && n0 + 4 * tn + 3 < a.N) {
      *reinterpret_cast<float4*>(row) = make_float4(acc[0], acc[1], acc[2], acc[3]);
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (n0 + 4 * tn + j < a.N) row[j] = acc[j];
    }
  }
  // the 16 lanes sharing tm are 16 consecutive lanes
#pragma unroll
  for (int off = 8; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off, 16));
  float sm = 0.0f;
#pragma unroll
  for (int j = 0; j < 4; ++j)
    if (n0 + 4 * tn + j < a.N) sm += expf(acc[j] - mx);
#pragma unroll
  for (int off = 8; off > 0; off >>= 1) sm += __shfl_xor(sm, off, 16);
  if (tn == 0 && m < M) a.partial[(long long)(mb + m) * a.nblk + blk] = make_float2(mx, sm);
}

__global__ __launch_bounds__(256) void softmax_mean_kernel(const ScoreArgs a) {
  extern __shared__ float2 stats[];  // [M] (max, 1/sum)
  __shared__ float part[4][KB];
  const int blk = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
  const int mb = a.t_off[b], M = a.t_off[b + 1] - mb;
  if (a.clear_bar && blk == 0 && b == 0) {  // the selection that follows starts from zero
    for (int i = tid; i < a.B; i += 256) a.clear_bar[i] = 0u;
    if (tid == 0) *a.clear_err = 0;
  }
  // row statistics from the per-block partials: four threads per row, each
  // folding every fourth block (all loads in flight), then the four
  // (max, sum) pairs combined in a fixed order
  constexpr int PU = 16;
  const int qtr = tid & 3;
  for (int m0 = 0; m0 < M; m0 += 64) {
    const int m = m0 + (tid >> 2);
    const float2* pr = a.partial + (long long)(mb + min(m, M - 1)) * a.nblk;
    float mx = -INFINITY, sm = 0.0f;
    for (int j0 = qtr; j0 < a.nblk; j0 += 4 * PU) {
      float2 v[PU];
#pragma unroll
      for (int u = 0; u < PU; ++u) v[u] = pr[min(j0 + 4 * u, a.nblk - 1)];
      float bm = mx;
#pragma unroll
      for (int u = 0; u < PU; ++u)
        if (j0 + 4 * u < a.nblk) bm = fmaxf(bm, v[u].x);
      sm = (mx == -INFINITY) ? 0.0f : sm * expf(mx - bm);
#pragma unroll
      for (int u = 0; u < PU; ++u)
        if (j0 + 4 * u < a.nblk) sm += v[u].y * expf(v[u].x - bm);
      mx = bm;
    }
#pragma unroll
    for (int off = 1; off < 4; off <<= 1) {
      const float om = __shfl_xor(mx, off, 4), os = __shfl_xor(sm, off, 4);
      const float nm = fmaxf(mx, om);
      // the pair order is fixed by the lane pattern, so all four lanes agree
      const float a0 = (qtr & off) ? os : sm, m0v = (qtr & off) ? om : mx;
      const float a1 = (qtr & off) ? sm : os, m1v = (qtr & off) ? mx : om;
      sm = (m0v == -INFINITY ? 0.0f : a0 * expf(m0v - nm)) + (m1v == -INFINITY ? 0.0f : a1 * expf(m1v - nm));
      mx = nm;
    }
    if (qtr == 0 && m < M) stats[m] = make_float2(mx, 1.0f / sm);
  }
  __syncthreads();
  const int c = tid & (KB - 1), g = tid >> 6;  // token, slice of question tokens
  const int n = blk * KB + c;
  float acc = 0.0f;
  if (n < a.N)
    for (int m0 = g; m0 < M; m0 += 4 * 8) {
      float l[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int m = m0 + 4 * u;
        l[u] = m < M ? a.logits[(long long)(mb + m) * a.N + n] : 0.0f;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int m = m0 + 4 * u;
        if (m < M) {
          const float2 st = stats[m];
          acc += expf(l[u] - st.x) * st.y;
        }
      }
    }
  part[g][c] = acc;
  __syncthreads();
  if (g == 0 && n < a.N)
    a.p_out[(long long)b * a.N + n] = ((part[0][c] + part[1][c]) + (part[2][c] + part[3][c])) /
                                      static_cast<float>(M);
}

}  // namespace

hipError_t launch_score(const ScoreArgs& a, hipStream_t s) {
  int maxM = 0;
  for (int b = 0; b < a.B; ++b) maxM = a.t_off[b + 1] - a.t_off[b] > maxM ? a.t_off[b + 1] - a.t_off[b] : maxM;
  const hipError_t e =
      launch_kernel("logits", logits_kernel, dim3(a.nblk, (maxM + QB - 1) / QB, a.B), dim3(256), 0, s, a);
  if (e != hipSuccess) return e;
  return launch_kernel("softmax_mean", softmax_mean_kernel, dim3(a.nblk, a.B), dim3(256), sizeof(float2) * maxM, s,
                       a);
}

}  // namespace mapk
