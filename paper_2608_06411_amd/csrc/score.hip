// Predicted attention, Eq. (3): logits, softmax over the visual tokens and
// the mean over the question tokens.
//
// logits_kernel: one workgroup per (block of 64 visual tokens, image).  The
// block's keys and, chunk by chunk, the image's queries sit in LDS; each
// thread forms a 4x4 patch of q.k / sqrt(d_p) in float32 and the workgroup
// also emits, per question token, the running (max, sum of exp) of its 64
// logits, so that no pass over a whole logits row is needed later.
//
// softmax_mean_kernel: same grid.  Each workgroup folds the per-block
// partials of its image into the row statistics (max_m, sum_m), then for its
// 64 tokens averages exp(l_mn - max_m) / sum_m over m.  The sums run in a
// fixed order, so the result is bitwise reproducible.
#include "internal.h"

namespace mapk {

namespace {

constexpr int KB = 64;    // visual tokens per workgroup
constexpr int QB = 64;    // question tokens per LDS chunk
constexpr int DPAD = 129; // padded LDS row (d_p <= 128)

__global__ __launch_bounds__(256) void logits_kernel(const ScoreArgs a) {
  __shared__ float ks[KB][DPAD];
  __shared__ float qs[QB][DPAD];
  const int blk = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
  const int n0 = blk * KB, dp = a.d_p;
  const int mb = a.t_off[b], M = a.t_off[b + 1] - mb;
  const float scale = 1.0f / sqrtf(static_cast<float>(dp));
  // stage the keys: float4 loads, all issued before the LDS stores
  {
    const int q4 = dp >> 2, total = KB * q4;
    for (int e0 = tid; e0 < total; e0 += 8 * 256) {
      float4 v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int e = e0 + u * 256, r = e / q4, d4 = e - r * q4;
        v[u] = (e < total && n0 + r < a.N)
                   ? *reinterpret_cast<const float4*>(a.k + ((long long)b * a.N + n0 + r) * dp + 4 * d4)
                   : make_float4(0.f, 0.f, 0.f, 0.f);
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int e = e0 + u * 256, r = e / q4, d4 = e - r * q4;
        if (e < total) {
          ks[r][4 * d4] = v[u].x; ks[r][4 * d4 + 1] = v[u].y;
          ks[r][4 * d4 + 2] = v[u].z; ks[r][4 * d4 + 3] = v[u].w;
        }
      }
    }
  }
  const int tm = tid >> 4, tn = tid & 15;  // rows 4 tm .. 4 tm + 3, keys 4 tn .. 4 tn + 3
  for (int q0 = 0; q0 < M; q0 += QB) {
    __syncthreads();
    {
      const int q4 = dp >> 2, total = QB * q4;
      for (int e0 = tid; e0 < total; e0 += 8 * 256) {
        float4 v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int e = e0 + u * 256, r = e / q4, d4 = e - r * q4;
          v[u] = (e < total && q0 + r < M)
                     ? *reinterpret_cast<const float4*>(a.q + (long long)(mb + q0 + r) * dp + 4 * d4)
                     : make_float4(0.f, 0.f, 0.f, 0.f);
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int e = e0 + u * 256, r = e / q4, d4 = e - r * q4;
          if (e < total) {
            qs[r][4 * d4] = v[u].x; qs[r][4 * d4 + 1] = v[u].y;
            qs[r][4 * d4 + 2] = v[u].z; qs[r][4 * d4 + 3] = v[u].w;
          }
        }
      }
    }
    __syncthreads();
    float acc[4][4] = {};
    for (int d = 0; d < dp; ++d) {
      float qv[4], kv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) qv[i] = qs[4 * tm + i][d];
#pragma unroll
      for (int j = 0; j < 4; ++j) kv[j] = ks[4 * tn + j][d];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(qv[i], kv[j], acc[i][j]);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = q0 + 4 * tm + i;
      float mx = -INFINITY;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int n = n0 + 4 * tn + j;
        acc[i][j] *= scale;
        if (n < a.N) {
          mx = fmaxf(mx, acc[i][j]);
          if (m < M) a.logits[(long long)(mb + m) * a.N + n] = acc[i][j];
        }
      }
      // the 16 threads sharing tm are 16 consecutive lanes
#pragma unroll
      for (int off = 8; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off, 16));
      float sm = 0.0f;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (n0 + 4 * tn + j < a.N) sm += expf(acc[i][j] - mx);
#pragma unroll
      for (int off = 8; off > 0; off >>= 1) sm += __shfl_xor(sm, off, 16);
      if (tn == 0 && m < M) a.partial[(long long)(mb + m) * a.nblk + blk] = make_float2(mx, sm);
    }
  }
}

__global__ __launch_bounds__(256) void softmax_mean_kernel(const ScoreArgs a) {
  extern __shared__ float2 stats[];  // [M] (max, 1/sum)
  __shared__ float part[4][KB];
  const int blk = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
  const int mb = a.t_off[b], M = a.t_off[b + 1] - mb;
  // row statistics from the per-block partials (independent loads batched)
  for (int m = tid; m < M; m += 256) {
    const float2* pr = a.partial + (long long)(mb + m) * a.nblk;
    float mx = -INFINITY, sm = 0.0f;
    for (int j0 = 0; j0 < a.nblk; j0 += 16) {
      float2 v[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) v[u] = j0 + u < a.nblk ? pr[j0 + u] : make_float2(-INFINITY, 0.0f);
      float bm = mx;
#pragma unroll
      for (int u = 0; u < 16; ++u) bm = fmaxf(bm, v[u].x);
      sm = (mx == -INFINITY) ? 0.0f : sm * expf(mx - bm);
#pragma unroll
      for (int u = 0; u < 16; ++u)
        if (j0 + u < a.nblk) sm += v[u].y * expf(v[u].x - bm);
      mx = bm;
    }
    stats[m] = make_float2(mx, 1.0f / sm);
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
  const dim3 grid(a.nblk, a.B);
  const hipError_t e = launch_kernel("logits", logits_kernel, grid, dim3(256), 0, s, a);
  if (e != hipSuccess) return e;
  return launch_kernel("softmax_mean", softmax_mean_kernel, grid, dim3(256), sizeof(float2) * maxM, s, a);
}

}  // namespace mapk
