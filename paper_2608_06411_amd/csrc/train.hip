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
  const float c = a.scale / static_cast<float>(M);
  float* grow = a.G + (long long)m * N;
  // the row in chunks of 16 values per thread held in registers between the
  // row sum and the write (rows up to 4096 tokens in one chunk)
  constexpr int RV = 16;
  for (int n0 = 0; n0 < N; n0 += RV * NT) {
    float P[RV], g[RV];
#pragma unroll
    for (int u = 0; u < RV; ++u) {
      const int n = min(n0 + u * NT + tid, N - 1);
      P[u] = lrow[n];
      g[u] = kl_dp(ps[n], ph[n]);
    }
    float s = 0.0f;
#pragma unroll
    for (int u = 0; u < RV; ++u) {
      const bool ok = n0 + u * NT + tid < N;
      P[u] = ok ? __expf(P[u] - mx) * inv_sum : 0.0f;
      s += P[u] * g[u];
    }
    if (n0 == 0 && n0 + RV * NT >= N) {  // the whole row is in registers: one pass
      s = block_sum_f(s, redf) * a.inv_B;
#pragma unroll
      for (int u = 0; u < RV; ++u) {
        const int n = n0 + u * NT + tid;
        if (n < N) grow[n] = c * P[u] * (g[u] * a.inv_B - s);
      }
      return;
    }
    break;  // longer rows: the two-pass form below
  }
  float s = 0.0f;
  for (int n = tid; n < N; n += NT) s += __expf(lrow[n] - mx) * inv_sum * kl_dp(ps[n], ph[n]);
  s = block_sum_f(s, redf) * a.inv_B;
  for (int n = tid; n < N; n += NT) {
    const float P = __expf(lrow[n] - mx) * inv_sum;
    grow[n] = c * P * (kl_dp(ps[n], ph[n]) * a.inv_B - s);
  }
}

template <typename T>
__device__ __forceinline__ void store_T(void* base, long long i, float v) {
  static_cast<T*>(base)[i] = from_f32<T>(v);
}

// Workgroup (16 visual tokens, image b): dk_n = sum_m G_mn q_m over the
// image's question rows, 64 rows at a time through LDS (queries as float4,
// d_p % 8 == 0); then RoPE's transpose, pair by pair, and the result in
// both layouts: rows [B N][d_p] and columns [d_p][ldv].
template <typename T>
__global__ __launch_bounds__(NT) void attn_grad_k_kernel(const TrainArgs a) {
  constexpr int TK = 16;
  __shared__ float4 Qs[64][32];
  __shared__ float Gs[64][TK + 1];
  __shared__ float tile[TK][129];
  const int tid = threadIdx.x, b = blockIdx.y, n0 = blockIdx.x * TK, N = a.N, dp = a.d_p, dp4 = dp >> 2;
  const int mb = a.t_off[b], M = a.t_off[b + 1] - mb;
  const int nl = tid >> 4, d4 = (tid & 15) * 2;  // two float4 of dims per thread
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int m0 = 0; m0 < M; m0 += 64) {
    float4 qv[8];
    float gv[4];
#pragma unroll
    for (int u = 0; u < 8; ++u) {  // every load of the chunk issued before the first LDS store
      const int i = tid + u * NT, r = i >> 5, q = i & 31;
      qv[u] = (m0 + r < M && q < dp4) ? reinterpret_cast<const float4*>(a.q + (long long)(mb + m0 + r) * dp)[q]
                                      : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = tid + u * NT, r = i / TK, n = i - r * TK;
      gv[u] = (m0 + r < M && n0 + n < N) ? a.G[(long long)(mb + m0 + r) * N + n0 + n] : 0.0f;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) Qs[(tid + u * NT) >> 5][(tid + u * NT) & 31] = qv[u];
#pragma unroll
    for (int u = 0; u < 4; ++u) Gs[(tid + u * NT) / TK][(tid + u * NT) % TK] = gv[u];
    __syncthreads();
#pragma unroll 8
    for (int r = 0; r < 64; ++r) {
      const float g = Gs[r][nl];
      const float4 q0 = Qs[r][d4], q1 = Qs[r][d4 + 1];
      acc[0] = fmaf(g, q0.x, acc[0]);
      acc[1] = fmaf(g, q0.y, acc[1]);
      acc[2] = fmaf(g, q0.z, acc[2]);
      acc[3] = fmaf(g, q0.w, acc[3]);
      acc[4] = fmaf(g, q1.x, acc[4]);
      acc[5] = fmaf(g, q1.y, acc[5]);
      acc[6] = fmaf(g, q1.z, acc[6]);
      acc[7] = fmaf(g, q1.w, acc[7]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int k = 0; k < 8; ++k) tile[nl][4 * d4 + k] = acc[k];
  __syncthreads();
  // RoPE's transpose: (x, y) -> (c x + s y, -s x + c y) for pair (i, i + half)
  const int half = dp >> 1;
  for (int e = tid; e < TK * half; e += NT) {
    const int nn = e / half, i = e - nn * half, n = n0 + nn;
    if (n >= N) continue;
    const float2 cs = a.cs_v[((long long)b * N + n) * half + i];
    const float x = tile[nn][i], y = tile[nn][i + half];
    tile[nn][i] = cs.x * x + cs.y * y;
    tile[nn][i + half] = cs.x * y - cs.y * x;
  }
  __syncthreads();
  const long long row0 = (long long)b * N + n0;
  for (int e = tid; e < TK * a.kdp; e += NT) {  // rows padded with zeros to kdp columns
    const int nn = e / a.kdp, d = e - nn * a.kdp;
    if (n0 + nn < N) store_T<T>(a.dk_rows, (row0 + nn) * a.kdp + d, d < dp ? tile[nn][d] : 0.0f);
  }
  for (int e = tid; e < TK * dp; e += NT) {
    const int d = e / TK, nn = e - d * TK;
    if (n0 + nn < N) store_T<T>(a.dk_cols, (long long)d * a.ldv + row0 + nn, tile[nn][d]);
  }
  {  // the padding columns of the transposed layout, spread over every workgroup
    const int pad = a.ldv - a.B * N, wg = blockIdx.y * gridDim.x + blockIdx.x, nwg = gridDim.x * gridDim.y;
    for (int e = wg * NT + tid; e < pad * dp; e += nwg * NT)
      store_T<T>(a.dk_cols, (long long)(e / pad) * a.ldv + a.B * N + e % pad, 0.0f);
  }
}

// Workgroup (64-token chunk c, 16 question rows, image b): the chunk's part
// of dq_m = sum_n G_mn k_n through LDS (keys as float4, d_p % 8 == 0),
// written to dq_part[c][m][:].
__global__ __launch_bounds__(NT) void attn_grad_q_kernel(const TrainArgs a) {
  __shared__ float4 Ks[64][32];
  __shared__ float Gs[16][65];
  const int tid = threadIdx.x, c = blockIdx.x, b = blockIdx.z, N = a.N, dp = a.d_p, dp4 = dp >> 2;
  const int mb = a.t_off[b], M = a.t_off[b + 1] - mb, m0 = blockIdx.y * 16;
  if (m0 >= M) return;
  const int ml = tid >> 4, d4 = (tid & 15) * 2;  // two float4 of dims per thread
  const int s0 = c * 64, ns = min(64, N - s0);
  for (int i = tid; i < 64 * 32; i += NT) {
    const int r = i >> 5, q = i & 31;
    Ks[r][q] = (r < ns && q < dp4) ? reinterpret_cast<const float4*>(a.k + ((long long)b * N + s0 + r) * dp)[q]
                                   : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  for (int i = tid; i < 16 * 64; i += NT) {
    const int r = i >> 6, n = i & 63;
    Gs[r][n] = (m0 + r < M && n < ns) ? a.G[(long long)(mb + m0 + r) * N + s0 + n] : 0.0f;
  }
  __syncthreads();
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll 8
  for (int n = 0; n < 64; ++n) {
    const float g = Gs[ml][n];
    const float4 k0 = Ks[n][d4], k1 = Ks[n][d4 + 1];
    acc[0] = fmaf(g, k0.x, acc[0]);
    acc[1] = fmaf(g, k0.y, acc[1]);
    acc[2] = fmaf(g, k0.z, acc[2]);
    acc[3] = fmaf(g, k0.w, acc[3]);
    acc[4] = fmaf(g, k1.x, acc[4]);
    acc[5] = fmaf(g, k1.y, acc[5]);
    acc[6] = fmaf(g, k1.z, acc[6]);
    acc[7] = fmaf(g, k1.w, acc[7]);
  }
  if (m0 + ml < M && 4 * d4 < dp) {
    float4* out = reinterpret_cast<float4*>(a.dq_part + ((long long)c * a.t_off[a.B] + mb + m0 + ml) * dp) + d4;
    out[0] = make_float4(acc[0], acc[1], acc[2], acc[3]);
    out[1] = make_float4(acc[4], acc[5], acc[6], acc[7]);
  }
}

// Workgroup m (one question row): the chunks' partials summed in chunk
// order, RoPE's transpose, both layouts (rows [sum_M][d_p], columns
// [d_p][ldt]); workgroup 0 also zeroes the padding columns.
template <typename T>
__global__ __launch_bounds__(1024) void dq_finish_kernel(const TrainArgs a) {
  __shared__ float v[128];
  __shared__ float grp[8][128];
  const int m = blockIdx.x, dp = a.d_p, sumM = a.t_off[a.B];
  const int tid = threadIdx.x & 127, g = threadIdx.x >> 7;  // dimension, chunk group
  if (tid < dp) {  // group g sums chunks g, g + 8, ... (loads issued 8 at a time)
    const float* src = a.dq_part + (long long)m * dp + tid;
    const long long cs = (long long)sumM * dp;
    float s = 0.0f;
    for (int c0 = g; c0 < a.nch; c0 += 64) {
      float x[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) x[u] = c0 + 8 * u < a.nch ? src[(c0 + 8 * u) * cs] : 0.0f;
#pragma unroll
      for (int u = 0; u < 8; ++u) s += x[u];
    }
    grp[g][tid] = s;
  }
  __syncthreads();
  if (g == 0 && tid < dp)  // the eight groups in a fixed order
    v[tid] = ((grp[0][tid] + grp[1][tid]) + (grp[2][tid] + grp[3][tid])) +
             ((grp[4][tid] + grp[5][tid]) + (grp[6][tid] + grp[7][tid]));
  __syncthreads();
  {  // the padding columns of the transposed layout, spread over every workgroup
    const int pad = a.ldt - sumM;
    for (int e = m * 1024 + threadIdx.x; e < pad * dp; e += sumM * 1024)
      store_T<T>(a.dq_cols, (long long)(e / pad) * a.ldt + sumM + e % pad, 0.0f);
  }
  if (g != 0) return;
  const int half = dp >> 1;
  if (tid < half) {
    const float2 cs = a.cs_t[(long long)m * half + tid];
    const float x = v[tid], y = v[tid + half];
    const float zx = cs.x * x + cs.y * y, zy = cs.x * y - cs.y * x;
    store_T<T>(a.dq_rows, (long long)m * a.kdp + tid, zx);
    store_T<T>(a.dq_rows, (long long)m * a.kdp + tid + half, zy);
    store_T<T>(a.dq_cols, (long long)tid * a.ldt + m, zx);
    store_T<T>(a.dq_cols, (long long)(tid + half) * a.ldt + m, zy);
  }
  for (int d = dp + tid; d < a.kdp; d += 128) store_T<T>(a.dq_rows, (long long)m * a.kdp + d, 0.0f);
}

// X = dz^T h from its token-chunk partials (float32 [nc][d_p][D_h]), summed
// in chunk order: X [d_p][D_h] and its transpose [D_h][kdp] (zero past d_p),
// both in the call's element type; blockIdx.y is the branch.
template <typename T>
__global__ __launch_bounds__(NT) void x_reduce_kernel(const XReduceArgs r) {
  const int s = blockIdx.y, per = r.d_p * r.D_h;
  const int e = blockIdx.x * NT + threadIdx.x;
  if (e < per) {
    const float* src = r.part[s] + e;
    float v = 0.0f;
    for (int c0 = 0; c0 < r.nc[s]; c0 += 8) {
      float x[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) x[u] = c0 + u < r.nc[s] ? src[(long long)(c0 + u) * per] : 0.0f;
#pragma unroll
      for (int u = 0; u < 8; ++u) v += x[u];
    }
    const int p = e / r.D_h, j = e - p * r.D_h;
    store_T<T>(r.X[s], e, v);
    store_T<T>(r.XT[s], (long long)j * r.kdp + p, v);
  }
  // the transposed rows' padding
  const int pad = r.kdp - r.d_p;
  for (int q = e; q < r.D_h * pad; q += gridDim.x * NT) store_T<T>(r.XT[s], (long long)(q / pad) * r.kdp + r.d_p + q % pad, 0.0f);
}

// dst[c][r] = src[r][c] for r < rows, and 0 for rows <= r < ldd: 64 x 64
// tiles through LDS, 16-byte pieces along the source rows on the way in and
// along the destination rows on the way out (cols, lds and ldd multiples of
// the piece's element count VE, checked by the host).
template <typename E>
__global__ __launch_bounds__(NT) void transpose_kernel(const TransposeBatch t) {
  constexpr int VE = 16 / sizeof(E);
  union Piece {
    uint4 u;
    E e[VE];
  };
  __shared__ E tile[64][65];
  int j = 0, blk = blockIdx.x;
  while (j + 1 < t.count && blk >= t.job[j + 1].tile_begin) ++j;
  const TransposeJob& J = t.job[j];
  blk -= J.tile_begin;
  const int tr = (J.ldd + 63) / 64;  // tiles along the destination rows (source rows r)
  const int r0 = (blk % tr) * 64, c0 = (blk / tr) * 64;
  const E* src = static_cast<const E*>(J.src);
  E* dst = static_cast<E*>(J.dst);
  constexpr int PR = 64 / VE;  // pieces per tile row
  for (int i = threadIdx.x; i < 64 * PR; i += NT) {
    const int r = i / PR, q = i - r * PR;
    Piece v;
    v.u = make_uint4(0u, 0u, 0u, 0u);
    if (r0 + r < J.rows && c0 + VE * q < J.cols)
      v.u = *reinterpret_cast<const uint4*>(src + (long long)(r0 + r) * J.lds + c0 + VE * q);
#pragma unroll
    for (int e = 0; e < VE; ++e) tile[r][VE * q + e] = v.e[e];
  }
  __syncthreads();
  for (int i = threadIdx.x; i < 64 * PR; i += NT) {
    const int c = i / PR, q = i - c * PR;
    if (c0 + c >= J.cols || r0 + VE * q >= J.ldd) continue;
    Piece v;
#pragma unroll
    for (int e = 0; e < VE; ++e) v.e[e] = tile[VE * q + e][c];
    *reinterpret_cast<uint4*>(dst + (long long)(c0 + c) * J.ldd + r0 + VE * q) = v.u;
  }
}

// out[r] = sum_c src[r][c] in float32: one wave per row, 16-byte pieces
// strided over the lanes, then a butterfly (a fixed order); cols and ld are
// multiples of the piece's element count.
template <typename T>
__global__ __launch_bounds__(NT) void rowsum_kernel(const RowsumBatch t) {
  constexpr int VE = 16 / sizeof(T);
  union Piece {
    uint4 u;
    T e[VE];
  };
  int j = 0;
  const int wave_id = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  while (j + 1 < t.count && wave_id >= t.job[j + 1].row_begin) ++j;
  const RowsumJob& J = t.job[j];
  const int r = wave_id - J.row_begin;
  if (r >= J.rows) return;
  const T* src = static_cast<const T*>(J.src) + (long long)r * J.ld;
  float s = 0.0f;
  for (int c = lane * VE; c < J.cols; c += 64 * VE) {
    Piece v;
    v.u = *reinterpret_cast<const uint4*>(src + c);
#pragma unroll
    for (int e = 0; e < VE; ++e) s += to_f32<T>(v.e[e]);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
  if (lane == 0) J.out[r] = s;
}

// Both branches (s = 0 visual, 1 text).  Workgroups [0, nA): one element of
// dW each, dW[s][p][j] += csum[s][p] b2[s][j]; the rest: one j each,
// db2[s][j] = sum_p W[s][p][j] csum[s][p].
template <typename T>
__global__ __launch_bounds__(NT) void finish_kernel(const FinishArgs f) {
  const int Dh = f.D_h, dp = f.d_p, per = dp * Dh;
  const int nA = (2 * per + NT - 1) / NT;
  if (static_cast<int>(blockIdx.x) < nA) {
    const int e = blockIdx.x * NT + threadIdx.x;
    if (e >= 2 * per) return;
    const int s = e / per, rem = e - s * per, p = rem / Dh, jj = rem - p * Dh;
    f.dW[s][rem] += f.csum[s][p] * to_f32<T>(static_cast<const T*>(f.b2[s])[jj]);
    return;
  }
  const int e = (blockIdx.x - nA) * NT + threadIdx.x;
  if (e >= 2 * Dh) return;
  const int s = e / Dh, jj = e - s * Dh;
  const T* W = static_cast<const T*>(f.W[s]);
  float acc = 0.0f;
#pragma unroll 8
  for (int p = 0; p < dp; ++p) acc = fmaf(to_f32<T>(W[(long long)p * Dh + jj]), f.csum[s][p], acc);
  f.db2[s][jj] = acc;
}

}  // namespace

hipError_t launch_train_grads(map_dtype dt, const TrainArgs& a, hipStream_t s) {
  const int sumM = a.t_off[a.B];
  int maxM = 0;
  for (int b = 0; b < a.B; ++b) maxM = a.t_off[b + 1] - a.t_off[b] > maxM ? a.t_off[b + 1] - a.t_off[b] : maxM;
  hipError_t e = launch_kernel("kl_grad", kl_grad_kernel, dim3(sumM + a.B), dim3(NT), 0, s, a);
  if (e != hipSuccess) return e;
  e = dt == MAP_BF16 ? launch_kernel("attn_grad_k", attn_grad_k_kernel<bf16_t>, dim3((a.N + 15) / 16, a.B),
                                     dim3(NT), 0, s, a)
                     : launch_kernel("attn_grad_k", attn_grad_k_kernel<float>, dim3((a.N + 15) / 16, a.B),
                                     dim3(NT), 0, s, a);
  if (e != hipSuccess) return e;
  e = launch_kernel("attn_grad_q", attn_grad_q_kernel, dim3(a.nch, (maxM + 15) / 16, a.B), dim3(NT), 0, s, a);
  if (e != hipSuccess) return e;
  return dt == MAP_BF16 ? launch_kernel("dq_finish", dq_finish_kernel<bf16_t>, dim3(sumM), dim3(1024), 0, s, a)
                        : launch_kernel("dq_finish", dq_finish_kernel<float>, dim3(sumM), dim3(1024), 0, s, a);
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
  const int ve = dt == MAP_BF16 ? 8 : 4;  // elements per 16-byte piece
  for (int j = 0; j < t.count; ++j)
    if (t.job[j].cols % ve || t.job[j].lds % ve || t.job[j].ldd % ve) return hipErrorInvalidValue;
  return dt == MAP_BF16 ? launch_kernel(name, transpose_kernel<uint16_t>, dim3(t.total_tiles), dim3(NT), 0, s, t)
                        : launch_kernel(name, transpose_kernel<float>, dim3(t.total_tiles), dim3(NT), 0, s, t);
}

hipError_t launch_rowsum(map_dtype dt, RowsumBatch& t, hipStream_t s) {
  int begin = 0;
  for (int j = 0; j < t.count; ++j) {
    t.job[j].row_begin = begin;
    begin += t.job[j].rows;
  }
  const int ve = dt == MAP_BF16 ? 8 : 4;  // elements per 16-byte piece
  for (int j = 0; j < t.count; ++j)
    if (t.job[j].cols % ve || t.job[j].ld % ve) return hipErrorInvalidValue;
  const dim3 grid((begin + 3) / 4);
  return dt == MAP_BF16 ? launch_kernel("rowsum", rowsum_kernel<bf16_t>, grid, dim3(NT), 0, s, t)
                        : launch_kernel("rowsum", rowsum_kernel<float>, grid, dim3(NT), 0, s, t);
}

hipError_t launch_x_reduce(map_dtype dt, const XReduceArgs& r, hipStream_t s) {
  const dim3 grid((r.d_p * r.D_h + NT - 1) / NT, 2);
  return dt == MAP_BF16 ? launch_kernel("x_reduce", x_reduce_kernel<bf16_t>, grid, dim3(NT), 0, s, r)
                        : launch_kernel("x_reduce", x_reduce_kernel<float>, grid, dim3(NT), 0, s, r);
}

hipError_t launch_finish(map_dtype dt, const FinishArgs& f, hipStream_t s) {
  const dim3 grid((2 * f.d_p * f.D_h + NT - 1) / NT + (2 * f.D_h + NT - 1) / NT);
  return dt == MAP_BF16 ? launch_kernel("finish", finish_kernel<bf16_t>, grid, dim3(NT), 0, s, f)
                        : launch_kernel("finish", finish_kernel<float>, grid, dim3(NT), 0, s, f);
}

}  // namespace mapk
