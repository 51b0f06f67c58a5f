// Predicted attention, Eq. (3): logits, softmax over the visual tokens and
// the mean over the question tokens.
//
// logits_kernel: one workgroup per (block of 64 visual tokens, chunk of 16
// question tokens, image).  Each wave forms a 16 x 16 tile of q.k / sqrt(d_p)
// on float32 matrix cores from operands read straight from global memory, and
// the workgroup also emits each query's (max, sum of exp) over its 64 logits,
// so that no pass over a whole logits row is needed later.
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

typedef __attribute__((ext_vector_type(4))) float f32x4_t;

__global__ __launch_bounds__(256) void logits_kernel(const ScoreArgs a) {
  __shared__ float wmax[4][QB];
  __shared__ float wsum[4][QB];
  const int blk = blockIdx.x, q0 = blockIdx.y * QB, b = blockIdx.z, tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int n0 = blk * KB, dp = a.d_p;
  const int mb = a.t_off[b], M = a.t_off[b + 1] - mb;
  if (q0 >= M) return;
  // Wave w forms the 16 x 16 tile (queries q0 .. q0 + 15) x (keys n0 + 16 w ..)
  // on float32 16 x 16 x 4 matrix cores.  Lane l supplies query row l & 15
  // and key row l & 15 at d = 16 t + 4 (l >> 4) + e to the e-th product of
  // step t, read as one float4 straight from global memory (rows past the
  // data read the last row; entries past d_p are zero).
  const int r = lane & 15, g = lane >> 4;
  const float* qr = a.q + (long long)(mb + min(q0 + r, M - 1)) * dp;
  const float* kr = a.k + ((long long)b * a.N + min(n0 + 16 * wave + r, a.N - 1)) * dp;
  constexpr int TS = 8;  // steps of 16 for d_p <= 128
  f32x4_t qv[TS], kv[TS];
#pragma unroll
  for (int t = 0; t < TS; ++t) {  // every load issued before the first product
    const int d = min(16 * t + 4 * g, dp - 4);
    qv[t] = *reinterpret_cast<const f32x4_t*>(qr + d);
    kv[t] = *reinterpret_cast<const f32x4_t*>(kr + d);
  }
  __builtin_amdgcn_sched_barrier(0);  // keep the loads ahead of the products
  f32x4_t acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int t = 0; t < TS; ++t) {
    const float in = 16 * t + 4 * g < dp ? 1.0f : 0.0f;  // zero past d_p (the load was clamped)
    qv[t] *= in;
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(qv[t].x, kv[t].x, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(qv[t].y, kv[t].y, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(qv[t].z, kv[t].z, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(qv[t].w, kv[t].w, acc, 0, 0, 0);
  }
  // acc[i]: query q0 + 4 g + i, key n0 + 16 w + r
  const float scale = 1.0f / sqrtf(static_cast<float>(dp));
  const int n = n0 + 16 * wave + r;
  const bool nok = n < a.N;
  float mx[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    acc[i] *= scale;
    const int m = q0 + 4 * g + i;
    if (m < M && nok) a.logits[(long long)(mb + m) * a.N + n] = acc[i];
    mx[i] = nok ? acc[i] : -INFINITY;
  }
  // per query: the maximum over the block's 64 keys (the 16 lanes of a group
  // hold one query's 16 keys of this wave), then the sum of exp in a fixed order
#pragma unroll
  for (int off = 8; off > 0; off >>= 1)
#pragma unroll
    for (int i = 0; i < 4; ++i) mx[i] = fmaxf(mx[i], __shfl_xor(mx[i], off, 16));
  if (r == 0)
#pragma unroll
    for (int i = 0; i < 4; ++i) wmax[wave][4 * g + i] = mx[i];
  __syncthreads();
  float sm[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int qi = 4 * g + i;
    const float bm = fmaxf(fmaxf(wmax[0][qi], wmax[1][qi]), fmaxf(wmax[2][qi], wmax[3][qi]));
    mx[i] = bm;
    sm[i] = nok ? expf(acc[i] - bm) : 0.0f;
  }
#pragma unroll
  for (int off = 8; off > 0; off >>= 1)
#pragma unroll
    for (int i = 0; i < 4; ++i) sm[i] += __shfl_xor(sm[i], off, 16);
  if (r == 0)
#pragma unroll
    for (int i = 0; i < 4; ++i) wsum[wave][4 * g + i] = sm[i];
  __syncthreads();
  if (tid < QB && q0 + tid < M)
    a.partial[(long long)(mb + q0 + tid) * a.nblk + blk] =
        make_float2(fmaxf(fmaxf(wmax[0][tid], wmax[1][tid]), fmaxf(wmax[2][tid], wmax[3][tid])),
                    (wsum[0][tid] + wsum[1][tid]) + (wsum[2][tid] + wsum[3][tid]));
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
  // the first LU logits of this thread's token (question tokens g, g + 4,
  // ...) are loaded now, at clamped addresses, so that they arrive while the
  // row statistics are formed
  const int c = tid & (KB - 1), g = tid >> 6;  // token, slice of question tokens
  const int n = blk * KB + c;
  constexpr int LU = 16;
  float l0[LU];
#pragma unroll
  for (int u = 0; u < LU; ++u)
    l0[u] = a.logits[(long long)(mb + min(g + 4 * u, M - 1)) * a.N + min(n, a.N - 1)];
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
  float acc = 0.0f;
  if (n < a.N) {
#pragma unroll
    for (int u = 0; u < LU; ++u) {
      const int m = g + 4 * u;
      if (m < M) {
        const float2 st = stats[m];
        acc += expf(l0[u] - st.x) * st.y;
      }
    }
    for (int m0 = g + 4 * LU; m0 < M; m0 += 4 * 8) {
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
