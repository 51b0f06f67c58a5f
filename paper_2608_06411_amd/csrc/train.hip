// One predictor training step (section "Cross-Modal Attention
// Distillation"): the KL divergence from the teacher distribution p* to the
// predicted p_hat of Eq. (3), and its gradient with respect to every
// predictor parameter.  The forward pass is the scoring path's (its layer-1
// launch also keeps GELU'(a)); the kernels here carry the gradient from
// p_hat back to the projections' inputs, plus the transposes, row sums and
// rank-one terms around the matrix-core products that form the weight
// gradients:
//
//   kl_grad      dL/dlogits:  G_mn = P_mn (g_n - sum_n' P_mn' g_n') / (M_b sqrt(d))
//                with g_n = -p*_n / (B p_hat_n) (the batch mean of the images'
//                divergences), and each image's divergence
//   attn_grad_k  dL/dz_n (visual): R(pos_n)^T sum_m G_mn q_m   (RoPE's transpose)
//   attn_grad_q  dL/dz_m (text):   R(pos_m)^T sum_n G_mn k_n   (partials over token
//                chunks, summed in a fixed order by dq_finish)
//   transpose    the products below reduce over tokens: their operands are
//                stored with the tokens contiguous (padded with zeros to a
//                multiple of 8 tokens)
//   rowsum       bias gradients: sums over tokens of dL/da and dL/dz
//   finish       dL/db2 = W^T sum_n dz_n and the term (sum_n dz_n) b2^T of dL/dW
#include "internal.h"

namespace mapk {

namespace {

constexpr int NT = 256;

__device__ __forceinline__ float block_sum_f(float v, float* red) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  if ((tid & 63) == 0) red[tid >> 6] = v;
  __syncthreads();
  const float r = (red[0] + red[1]) + (red[2] + red[3]);
  __syncthreads();
  return r;
}

__device__ __forceinline__ double block_sum_d(double v, double* red) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  if ((tid & 63) == 0) red[tid >> 6] = v;
  __syncthreads();
  const double r = (red[0] + red[1]) + (red[2] + red[3]);
  __syncthreads();
  return r;
}

// dL/dp_hat_n up to the factor 1/B: -p*_n / p_hat_n, and 0 where p*_n = 0
// (its term of the divergence is 0 log 0 = 0).
__device__ __forceinline__ float kl_dp(float ps, float ph) { return ps > 0.0f ? -ps / ph : 0.0f; }

__device__ __forceinline__ int image_of_row(const TrainArgs& a, int row) {
  int b = 0;
  while (b + 1 < a.B && a.t_off[b + 1] <= row) ++b;
  return b;
}

// Workgroups [0, sum_M): one question row m each -- its softmax statistics
// from the scoring pass's per-block partials, the row sum s_m = sum_n P_mn g_n
// and then the row of G.  Workgroups [sum_M, sum_M + B): image b's divergence
// sum_n p*_n log(p*_n / p_hat_n) (0 log 0 = 0), accumulated in float64.
__global__ __launch_bounds__(NT) void kl_grad_kernel(const TrainArgs a) {
  __shared__ float redf[4];
  __shared__ double redd[4];
  const int tid = threadIdx.x, N = a.N, sumM = a.t_off[a.B];
  const int w = blockIdx.x;
  if (w >= sumM) {
    const int b = w - sumM;
    const float* ps = a.p_star + (long long)b * N;
    const float* ph = a.p_hat + (long long)b * N;
    double acc = 0.0;
    for (int n = tid; n < N; n += NT) {
      const float s = ps[n];
      if (s > 0.0f) acc += static_cast<double>(s) * (log(static_cast<double>(s)) - log(static_cast<double>(ph[n])));
    }
    const double t = block_sum_d(acc, redd);
    if (tid == 0) a.loss[b] = static_cast<float>(t);
    return;
  }
  const int m = w, b = image_of_row(a, m), M = a.t_off[b + 1] - a.t_off[b];
  // row statistics: max over the blocks' maxima, then the rescaled sums
  const float2* pr = a.partial + (long long)m * a.nblk;
  float mx = -INFINITY;
  for (int j = tid; j < a.nblk; j += NT) mx = fmaxf(mx, pr[j].x);
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off, 64));
  if ((tid & 63) == 0) redf[tid >> 6] = mx;
  __syncthreads();
  mx = fmaxf(fmaxf(redf[0], redf[1]), fmaxf(redf[2], redf[3]));
  __syncthreads();
  float sm = 0.0f;
  for (int j = tid; j < a.nblk; j += NT) sm += pr[j].y * __expf(pr[j].x - mx);
  const float inv_sum = 1.0f / block_sum_f(sm, redf);
  const float* lrow = a.logits + (long long)m * N;
  const float* ps = a.p_star + (long long)b * N;
  const float* ph = a.p_hat + (long long)b * N;
  float s = 0.0f;
  for (int n = tid; n < N; n += NT) {
    const float P = __expf(lrow[n] - mx) * inv_sum;
    s += P * kl_dp(ps[n], ph[n]);
  }
  s = block_sum_f(s, redf) * a.inv_B;
  const float c = a.scale / static_cast<float>(M);
  float* grow = a.G + (long long)m * N;
  for (int n = tid; n < N; n += NT) {
    const float P = __expf(lrow[n] - mx) * inv_sum;
    grow[n] = c * P * (kl_dp(ps[n], ph[n]) * a.inv_B - s);
  }
}

template <typename T>
__device__ __forceinline__ void store_T(void* base, long long i, float v) {
  static_cast<T*>(base)[i] = from_f32<T>(v);
}

// Workgroup (64 visual tokens, image b): dk_n = sum_m G_mn q_m over the
// image's question rows, 32 rows at a time through LDS; then RoPE's
// transpose, pair by pair, and the result in both layouts: rows
// [B N][d_p] and columns [d_p][ldv].
template <typename T>
__global__ __launch_bounds__(NT) void attn_grad_k_kernel(const TrainArgs a) {
  __shared__ float Qs[32][128];
  __shared__ float Gs[32][64];
  __shared__ float tile[64][129];
  const int tid = threadIdx.x, b = blockIdx.y, n0 = blockIdx.x * 64, N = a.N, dp = a.d_p;
  const int mb = a.t_off[b], M = a.t_off[b + 1] - mb;
  const int nl = tid >> 2, d0 = (tid & 3) * 32;
  float acc[32];
#pragma unroll
  for (int k = 0; k < 32; ++k) acc[k] = 0.0f;
  for (int m0 = 0; m0 < M; m0 += 32) {
    for (int i = tid; i < 32 * 128; i += NT) {
      const int r = i >> 7, d = i & 127;
      Qs[r][d] = (m0 + r < M && d < dp) ? a.q[(long long)(mb + m0 + r) * dp + d] : 0.0f;
    }
    for (int i = tid; i < 32 * 64; i += NT) {
      const int r = i >> 6, n = i & 63;
      Gs[r][n] = (m0 + r < M && n0 + n < N) ? a.G[(long long)(mb + m0 + r) * N + n0 + n] : 0.0f;
    }
    __syncthreads();
#pragma unroll 4
    for (int r = 0; r < 32; ++r) {
      const float g = Gs[r][nl];
#pragma unroll
      for (int k = 0; k < 32; k += 4) {
        const float4 q = *reinterpret_cast<const float4*>(&Qs[r][d0 + k]);
        acc[k] = fmaf(g, q.x, acc[k]);
        acc[k + 1] = fmaf(g, q.y, acc[k + 1]);
        acc[k + 2] = fmaf(g, q.z, acc[k + 2]);
        acc[k + 3] = fmaf(g, q.w, acc[k + 3]);
      }
    }
    __syncthreads();
  }
#pragma unroll
  for (int k = 0; k < 32; ++k) tile[nl][d0 + k] = acc[k];
  __syncthreads();
  // RoPE's transpose: (x, y) -> (c x + s y, -s x + c y) for pair (i, i + half)
  const int half = dp >> 1;
  for (int e = tid; e < 64 * half; e += NT) {
    const int nn = e / half, i = e - nn * half, n = n0 + nn;
    if (n >= N) continue;
    const float2 cs = a.cs_v[((long long)b * N + n) * half + i];
    const float x = tile[nn][i], y = tile[nn][i + half];
    tile[nn][i] = cs.x * x + cs.y * y;
    tile[nn][i + half] = cs.x * y - cs.y * x;
  }
  __syncthreads();
  const long long row0 = (long long)b * N + n0;
  for (int e = tid; e < 64 * dp; e += NT) {
    const int nn = e / dp, d = e - nn * dp;
    if (n0 + nn < N) store_T<T>(a.dk_rows, (row0 + nn) * dp + d, tile[nn][d]);
  }
  for (int e = tid; e < 64 * dp; e += NT) {
    const int d = e >> 6, nn = e & 63;
    if (n0 + nn < N) store_T<T>(a.dk_cols, (long long)d * a.ldv + row0 + nn, tile[nn][d]);
  }
  if (blockIdx.x == 0 && b == 0) {  // the padding columns of the transposed layout
    const int pad = a.ldv - a.B * N;
    for (int e = tid; e < pad * dp; e += NT)
      store_T<T>(a.dk_cols, (long long)(e / pad) * a.ldv + a.B * N + e % pad, 0.0f);
  }
}

// Workgroup (256-token chunk c, 16 question rows, image b): the chunk's part
// of dq_m = sum_n G_mn k_n, 64 tokens at a time through LDS, written to
// dq_part[c][m][:].
__global__ __launch_bounds__(NT) void attn_grad_q_kernel(const TrainArgs a) {
  __shared__ float Ks[64][128];
  __shared__ float Gs[16][64];
  const int tid = threadIdx.x, c = blockIdx.x, b = blockIdx.z, N = a.N, dp = a.d_p;
  const int mb = a.t_off[b], M = a.t_off[b + 1] - mb, m0 = blockIdx.y * 16;
  if (m0 >= M) return;
  const int ml = tid >> 4, d0 = (tid & 15) * 8;
  float acc[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) acc[k] = 0.0f;
  const int nbeg = c * 256, nend = min(N, nbeg + 256);
  for (int s0 = nbeg; s0 < nend; s0 += 64) {
    for (int i = tid; i < 64 * 128; i += NT) {
      const int r = i >> 7, d = i & 127;
      Ks[r][d] = (s0 + r < nend && d < dp) ? a.k[((long long)b * N + s0 + r) * dp + d] : 0.0f;
    }
    for (int i = tid; i < 16 * 64; i += NT) {
      const int r = i >> 6, n = i & 63;
      Gs[r][n] = (m0 + r < M && s0 + n < nend) ? a.G[(long long)(mb + m0 + r) * N + s0 + n] : 0.0f;
    }
    __syncthreads();
#pragma unroll 4
    for (int n = 0; n < 64; ++n) {
      const float g = Gs[ml][n];
      const float4 k0 = *reinterpret_cast<const float4*>(&Ks[n][d0]);
      const float4 k1 = *reinterpret_cast<const float4*>(&Ks[n][d0 + 4]);
      acc[0] = fmaf(g, k0.x, acc[0]);
      acc[1] = fmaf(g, k0.y, acc[1]);
      acc[2] = fmaf(g, k0.z, acc[2]);
      acc[3] = fmaf(g, k0.w, acc[3]);
      acc[4] = fmaf(g, k1.x, acc[4]);
      acc[5] = fmaf(g, k1.y, acc[5]);
      acc[6] = fmaf(g, k1.z, acc[6]);
      acc[7] = fmaf(g, k1.w, acc[7]);
    }
    __syncthreads();
  }
  if (m0 + ml < M && d0 < dp) {
    float* out = a.dq_part + ((long long)c * a.t_off[a.B] + mb + m0 + ml) * dp + d0;
#pragma unroll
    for (int k = 0; k < 8; ++k)
      if (d0 + k < dp) out[k] = acc[k];
  }
}

// Workgroup m (one question row): the chunks' partials summed in chunk
// order, RoPE's transpose, both layouts (rows [sum_M][d_p], columns
// [d_p][ldt]); workgroup 0 also zeroes the padding columns.
template <typename T>
__global__ __launch_bounds__(128) void dq_finish_kernel(const TrainArgs a) {
  __shared__ float v[128];
  const int m = blockIdx.x, tid = threadIdx.x, dp = a.d_p, sumM = a.t_off[a.B];
  if (tid < dp) {
    float s = 0.0f;
    for (int c = 0; c < a.nch; ++c) s += a.dq_part[((long long)c * sumM + m) * dp + tid];
    v[tid] = s;
  }
  __syncthreads();
  const int half = dp >> 1;
  if (tid < half) {
    const float2 cs = a.cs_t[(long long)m * half + tid];
    const float x = v[tid], y = v[tid + half];
    const float zx = cs.x * x + cs.y * y, zy = cs.x * y - cs.y * x;
    store_T<T>(a.dq_rows, (long long)m * dp + tid, zx);
    store_T<T>(a.dq_rows, (long long)m * dp + tid + half, zy);
    store_T<T>(a.dq_cols, (long long)tid * a.ldt + m, zx);
    store_T<T>(a.dq_cols, (long long)(tid + half) * a.ldt + m, zy);
  }
  if (m == 0) {
    const int pad = a.ldt - sumM;
    for (int e = tid; e < pad * dp; e += 128) store_T<T>(a.dq_cols, (long long)(e / pad) * a.ldt + sumM + e % pad, 0.0f);
  }
}

// dst[c][r] = src[r][c] for r < rows, and 0 for rows <= r < ldd: 64 x 64
// tiles through LDS, reads along the source rows and writes along the
// destination rows.
template <typename E>
__global__ __launch_bounds__(NT) void transpose_kernel(const TransposeBatch t) {
  __shared__ E tile[64][65];
  int j = 0, blk = blockIdx.x;
  while (j + 1 < t.count && blk >= t.job[j + 1].tile_begin) ++j;
  const TransposeJob& J = t.job[j];
  blk -= J.tile_begin;
  const int tr = (J.ldd + 63) / 64;  // tiles along the destination rows (source rows r)
  const int r0 = (blk % tr) * 64, c0 = (blk / tr) * 64;
  const E* src = static_cast<const E*>(J.src);
  E* dst = static_cast<E*>(J.dst);
  for (int i = threadIdx.x; i < 64 * 64; i += NT) {
    const int r = i >> 6, c = i & 63;
    tile[r][c] = (r0 + r < J.rows && c0 + c < J.cols) ? src[(long long)(r0 + r) * J.lds + c0 + c] : E(0);
  }
  __syncthreads();
  for (int i = threadIdx.x; i < 64 * 64; i += NT) {
    const int c = i >> 6, r = i & 63;
    if (c0 + c < J.cols && r0 + r < J.ldd) dst[(long long)(c0 + c) * J.ldd + r0 + r] = tile[r][c];
  }
}

// out[r] = sum_c src[r][c] in float32: one wave per row, lanes strided,
// then a butterfly (a fixed order).
template <typename T>
__global__ __launch_bounds__(NT) void rowsum_kernel(const RowsumBatch t) {
  int j = 0;
  const int wave_id = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  while (j + 1 < t.count && wave_id >= t.job[j + 1].row_begin) ++j;
  const RowsumJob& J = t.job[j];
  const int r = wave_id - J.row_begin;
  if (r >= J.rows) return;
  const T* src = static_cast<const T*>(J.src) + (long long)r * J.ld;
  float s = 0.0f;
  for (int c = lane; c < J.cols; c += 64) s += to_f32<T>(src[c]);
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
  if (lane == 0) J.out[r] = s;
}

// Per branch (blockIdx.y: visual, text) and column j of D_h:
//   db2[j] = sum_p W[p][j] csum[p]   and   dW[p][j] += csum[p] b2[j]
template <typename T>
__global__ __launch_bounds__(NT) void finish_kernel(const FinishArgs f) {
  const int j = blockIdx.x * NT + threadIdx.x, s = blockIdx.y;
  if (j >= f.D_h) return;
  const T* W = static_cast<const T*>(f.W[s]);
  const float b2 = to_f32<T>(static_cast<const T*>(f.b2[s])[j]);
  float acc = 0.0f;
  for (int p = 0; p < f.d_p; ++p) {
    const float cs = f.csum[s][p];
    acc = fmaf(to_f32<T>(W[(long long)p * f.D_h + j]), cs, acc);
    f.dW[s][(long long)p * f.D_h + j] += cs * b2;
  }
  f.db2[s][j] = acc;
}

}  // namespace

hipError_t launch_train_grads(map_dtype dt, const TrainArgs& a, hipStream_t s) {
  const int sumM = a.t_off[a.B];
  int maxM = 0;
  for (int b = 0; b < a.B; ++b) maxM = a.t_off[b + 1] - a.t_off[b] > maxM ? a.t_off[b + 1] - a.t_off[b] : maxM;
  hipError_t e = launch_kernel("kl_grad", kl_grad_kernel, dim3(sumM + a.B), dim3(NT), 0, s, a);
  if (e != hipSuccess) return e;
  e = dt == MAP_BF16 ? launch_kernel("attn_grad_k", attn_grad_k_kernel<bf16_t>, dim3((a.N + 63) / 64, a.B),
                                     dim3(NT), 0, s, a)
                     : launch_kernel("attn_grad_k", attn_grad_k_kernel<float>, dim3((a.N + 63) / 64, a.B),
                                     dim3(NT), 0, s, a);
  if (e != hipSuccess) return e;
  e = launch_kernel("attn_grad_q", attn_grad_q_kernel, dim3(a.nch, (maxM + 15) / 16, a.B), dim3(NT), 0, s, a);
  if (e != hipSuccess) return e;
  return dt == MAP_BF16 ? launch_kernel("dq_finish", dq_finish_kernel<bf16_t>, dim3(sumM), dim3(128), 0, s, a)
                        : launch_kernel("dq_finish", dq_finish_kernel<float>, dim3(sumM), dim3(128), 0, s, a);
}

void transpose_finalize(TransposeBatch& t) {
  int begin = 0;
  for (int j = 0; j < t.count; ++j) {
    t.job[j].tile_begin = begin;
    begin += ((t.job[j].ldd + 63) / 64) * ((t.job[j].cols + 63) / 64);
  }
  t.total_tiles = begin;
}

hipError_t launch_transpose(map_dtype dt, const TransposeBatch& t, const char* name, hipStream_t s) {
  if (t.total_tiles == 0) return hipSuccess;
  return dt == MAP_BF16 ? launch_kernel(name, transpose_kernel<uint16_t>, dim3(t.total_tiles), dim3(NT), 0, s, t)
                        : launch_kernel(name, transpose_kernel<float>, dim3(t.total_tiles), dim3(NT), 0, s, t);
}

hipError_t launch_rowsum(map_dtype dt, RowsumBatch& t, hipStream_t s) {
  int begin = 0;
  for (int j = 0; j < t.count; ++j) {
    t.job[j].row_begin = begin;
    begin += t.job[j].rows;
  }
  const dim3 grid((begin + 3) / 4);
  return dt == MAP_BF16 ? launch_kernel("rowsum", rowsum_kernel<bf16_t>, grid, dim3(NT), 0, s, t)
                        : launch_kernel("rowsum", rowsum_kernel<float>, grid, dim3(NT), 0, s, t);
}

hipError_t launch_finish(map_dtype dt, const FinishArgs& f, hipStream_t s) {
  const dim3 grid((f.D_h + NT - 1) / NT, 2);
  return dt == MAP_BF16 ? launch_kernel("finish", finish_kernel<bf16_t>, grid, dim3(NT), 0, s, f)
                        : launch_kernel("finish", finish_kernel<float>, grid, dim3(NT), 0, s, f);
}

}  // namespace mapk
