// Predicted attention, Eq. (3): logits, softmax over the visual tokens and
// the mean over the question tokens.
//
// score_kernel (one launch): one workgroup per (block of 64 visual tokens,
// chunk of 16 question tokens, image).  Each wave forms a 16 x 16 tile of
// q.k / sqrt(d_p) on float32 matrix cores from operands read straight from
// global memory and keeps it in registers; the workgroup publishes each
// query's (max, sum of exp) over its 64 logits as one 64-bit word.  Each
// workgroup then waits for the words of its 16 queries from every token
// block of the image, folds them into the row statistics (max_m, sum_m),
// and publishes its 64 tokens' share sum_m exp(l_mn - max_m) / sum_m over
// those queries, again as 64-bit words; the workgroup of the image's first
// chunk waits for the other chunks' shares of its tokens, adds them in
// chunk order and divides by M.  A published word is never zero (a sum of
// exp includes exp(0) = 1; a share word carries a marker in its high half),
// and prep zeroes both arrays before the launch, so a nonzero word is a
// complete one: the exchange needs no counters and no cache flushes, only
// agent-scope atomic 64-bit stores and loads.  Every sum runs in a fixed
// order, so the result is bitwise reproducible.  The host launches it only
// for groups of images whose workgroups can all be resident at once.
//
// logits_kernel + softmax_mean_kernel: the same in two launches, for
// questions too long for the one-launch form: the first writes the logits
// and the per-block pairs, the second folds the pairs and averages over m.
#include "internal.h"

namespace mapk {

namespace {

constexpr int KB = 64;    // visual tokens per workgroup
constexpr int QB = 16;    // question tokens per workgroup

typedef __attribute__((ext_vector_type(4))) float f32x4_t;

__device__ __forceinline__ uint64_t load_word(const uint64_t* p) {
  return __hip_atomic_load(const_cast<uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void store_word(uint64_t* p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float2 word_pair(uint64_t w) {
  return make_float2(__uint_as_float(static_cast<uint32_t>(w)), __uint_as_float(static_cast<uint32_t>(w >> 32)));
}


// The 16 x 64 tile (queries q0 .., keys 64 blk ..) of image b: out[i] is the
// scaled logit of query q0 + 4 (lane >> 4) + i and key 64 blk + 16 wave +
// (lane & 15).  The logits are stored when `store`; each query's (max, sum
// of exp) over the 64 keys goes to a.partial.
__device__ __forceinline__ void logits_tile(const ScoreArgs& a, int b, int blk, int q0, bool store, float (&out)[4],
                                            float (*wmax)[QB], float (*wsum)[QB], bool words) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n0 = blk * KB, dp = a.d_p;
  const int mb = a.t_off[b], M = a.t_off[b + 1] - mb;
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
    out[i] = acc[i] * scale;
    const int m = q0 + 4 * g + i;
    if (store && m < M && nok) a.logits[(long long)(mb + m) * a.N + n] = out[i];
    mx[i] = nok ? out[i] : -INFINITY;
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
    sm[i] = nok ? expf(out[i] - bm) : 0.0f;
  }
#pragma unroll
  for (int off = 8; off > 0; off >>= 1)
#pragma unroll
    for (int i = 0; i < 4; ++i) sm[i] += __shfl_xor(sm[i], off, 16);
  if (r == 0)
#pragma unroll
    for (int i = 0; i < 4; ++i) wsum[wave][4 * g + i] = sm[i];
  __syncthreads();
  if (tid < QB && q0 + tid < M) {
    const float bm = fmaxf(fmaxf(wmax[0][tid], wmax[1][tid]), fmaxf(wmax[2][tid], wmax[3][tid]));
    const float bs = (wsum[0][tid] + wsum[1][tid]) + (wsum[2][tid] + wsum[3][tid]);
    float2* dst = a.partial + (long long)(mb + q0 + tid) * a.nblk + blk;
    if (words)
      store_word(reinterpret_cast<uint64_t*>(dst),
                 (static_cast<uint64_t>(__float_as_uint(bs)) << 32) | __float_as_uint(bm));
    else
      *dst = make_float2(bm, bs);
  }
}

// (max, sum of exp) pairs combined: lo is the pair of the lower lane (or the
// running pair), so every lane of a butterfly gets the same bits.
__device__ __forceinline__ float2 merge_pair(float2 lo, float2 hi) {
  const float nm = fmaxf(lo.x, hi.x);
  return make_float2(nm, (lo.x == -INFINITY ? 0.0f : lo.y * expf(lo.x - nm)) +
                             (hi.x == -INFINITY ? 0.0f : hi.y * expf(hi.x - nm)));
}

__device__ __forceinline__ void clear_selection_counters(const ScoreArgs& a) {
  for (int i = threadIdx.x; i < a.B; i += 256) a.clear_bar[i] = 0u;
  if (threadIdx.x == 0) *a.clear_err = 0;
}

constexpr unsigned kScoreSpinLimit = 1u << 20;  // polls of one word set (each sleeps about 64 clocks)

__global__ __launch_bounds__(256) void score_kernel(const ScoreArgs a, int b0) {
  __shared__ float wmax[4][QB];
  __shared__ float wsum[4][QB];
  __shared__ float2 stats[QB];
  const int blk = blockIdx.x, qc = blockIdx.y, b = b0 + blockIdx.z, tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int mb = a.t_off[b], M = a.t_off[b + 1] - mb, q0 = qc * QB;
  if (a.clear_bar && blk == 0 && qc == 0 && blockIdx.z == 0) clear_selection_counters(a);
  if (q0 >= M) return;
  float l[4];
  // the tile; its (max, sum) pairs go out as words (x in the low half)
  logits_tile(a, b, blk, q0, a.store_logits != 0, l, wmax, wsum, true);

  // row statistics of the 16 queries: 16 threads per query, thread j waiting
  // for the words of blocks j, j + 16, ... (all polled at once), then folding
  // them in block order and a butterfly over the 16 in a fixed pairing
  bool ok = true;
  {
    constexpr int PW = 16;  // blocks per thread (nblk <= 256)
    const int qi = tid >> 4, j = tid & 15, m = min(q0 + qi, M - 1);
    const uint64_t* pr = reinterpret_cast<const uint64_t*>(a.partial) + (long long)(mb + m) * a.nblk;
    uint64_t w[PW];
#pragma unroll
    for (int u = 0; u < PW; ++u) w[u] = j + 16 * u < a.nblk ? load_word(pr + j + 16 * u) : 1ull;
    for (unsigned spins = 0;; ++spins) {
      bool all = true;
#pragma unroll
      for (int u = 0; u < PW; ++u) all = all && w[u] != 0ull;
      if (all) break;
      if (spins > kScoreSpinLimit) {  // not every workgroup was resident
        ok = false;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
#pragma unroll
      for (int u = 0; u < PW; ++u)
        if (w[u] == 0ull) w[u] = load_word(pr + j + 16 * u);
    }
    float2 run = make_float2(-INFINITY, 0.0f);
#pragma unroll
    for (int u = 0; u < PW; ++u)
      if (j + 16 * u < a.nblk) run = merge_pair(run, word_pair(w[u]));
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) {
      const float2 o = make_float2(__shfl_xor(run.x, off, 16), __shfl_xor(run.y, off, 16));
      run = (j & off) ? merge_pair(o, run) : merge_pair(run, o);
    }
    if (j == 0) stats[qi] = make_float2(run.x, 1.0f / run.y);
  }
  ok = __syncthreads_and(ok);
  if (!ok && tid == 0 && a.clear_err) atomicExch(a.clear_err, 1);

  // this chunk's share of the mean for the 64 tokens: lane (g, r) of wave w
  // sums its four queries, then the four groups g are added
  const int r = lane & 15, g = lane >> 4, n = blk * KB + 16 * wave + r;
  float v = 0.0f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int qi = 4 * g + i;
    if (q0 + qi < M) v += expf(l[i] - stats[qi].x) * stats[qi].y;
  }
  v += __shfl_xor(v, 16);
  v += __shfl_xor(v, 32);
  if (!ok) v = NAN;
  uint64_t* pp = a.pp + (long long)a.q_off[b] * a.N;
  if (qc > 0) {
    if (g == 0 && n < a.N) store_word(pp + (long long)qc * a.N + n, (1ull << 32) | __float_as_uint(v));
    return;
  }
  // the first chunk's workgroup adds the other chunks' shares in chunk order
  const int nq = (M + QB - 1) / QB;
  if (g == 0 && n < a.N) {
    float s = v;
    constexpr int CW = 8;  // chunks polled at once
    for (int c0 = 1; c0 < nq; c0 += CW) {
      uint64_t x[CW];
#pragma unroll
      for (int u = 0; u < CW; ++u) x[u] = c0 + u < nq ? load_word(pp + (long long)(c0 + u) * a.N + n) : 1ull;
      for (unsigned spins = 0;; ++spins) {
        bool all = true;
#pragma unroll
        for (int u = 0; u < CW; ++u) all = all && x[u] != 0ull;
        if (all) break;
        if (spins > kScoreSpinLimit) {
#pragma unroll
          for (int u = 0; u < CW; ++u)
            if (x[u] == 0ull) x[u] = (1ull << 32) | __float_as_uint(NAN);
          if (a.clear_err) atomicExch(a.clear_err, 1);
          break;
        }
        __builtin_amdgcn_s_sleep(1);
#pragma unroll
        for (int u = 0; u < CW; ++u)
          if (x[u] == 0ull) x[u] = load_word(pp + (long long)(c0 + u) * a.N + n);
      }
#pragma unroll
      for (int u = 0; u < CW; ++u)
        if (c0 + u < nq) s += __uint_as_float(static_cast<uint32_t>(x[u]));
    }
    a.p_out[(long long)b * a.N + n] = s / static_cast<float>(M);
  }
}

__global__ __launch_bounds__(256) void logits_kernel(const ScoreArgs a) {
  __shared__ float wmax[4][QB];
  __shared__ float wsum[4][QB];
  const int blk = blockIdx.x, q0 = blockIdx.y * QB, b = blockIdx.z;
  const int M = a.t_off[b + 1] - a.t_off[b];
  if (q0 >= M) return;
  float l[4];
  logits_tile(a, b, blk, q0, true, l, wmax, wsum, false);
}

__global__ __launch_bounds__(256) void softmax_mean_kernel(const ScoreArgs a) {
  extern __shared__ float2 stats[];  // [M] (max, 1/sum)
  __shared__ float part[4][KB];
  const int blk = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
  const int mb = a.t_off[b], M = a.t_off[b + 1] - mb;
  if (a.clear_bar && blk == 0 && b == 0) clear_selection_counters(a);  // the selection starts from zero
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

// Workgroups of score_kernel that can be resident at once on the current
// device (cached per device; 0 when unknown).
static int score_capacity() {
  static int cached[16] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 16) return 0;
  if (cached[dev] == 0) {
    int cus = 0, per = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, score_kernel, 256, 0) != hipSuccess || cus <= 0 || per <= 0)
      return 0;
    cached[dev] = cus * per;
  }
  return cached[dev];
}

// The one-launch form: for several images (at one image it is no faster
// than the two launches: measured side by side, 0.5 us slower per step at
// the LLaVA-NeXT shape, it also needs its exchange arrays zeroed), with at
// most 256 token blocks and every image's workgroups resident at once.
bool score_one_launch(int B, int N, const int32_t* t_off) {
  const int nblk = (N + KB - 1) / KB, cap = B >= 2 && nblk <= 256 ? score_capacity() : 0;
  for (int b = 0; b < B && cap > 0; ++b)
    if ((long long)nblk * ((t_off[b + 1] - t_off[b] + QB - 1) / QB) > cap) return false;
  return cap > 0;
}

hipError_t launch_score(const ScoreArgs& a0, hipStream_t s) {
  ScoreArgs a = a0;
  int maxM = 0;
  a.q_off[0] = 0;
  for (int b = 0; b < a.B; ++b) {
    const int M = a.t_off[b + 1] - a.t_off[b];
    maxM = M > maxM ? M : maxM;
    a.q_off[b + 1] = a.q_off[b] + (M + QB - 1) / QB;
  }
  // one launch per group of images whose workgroups all fit on the device
  const int cap = score_capacity();
  if (a.pp && score_one_launch(a.B, a.N, a.t_off)) {
    for (int b0 = 0; b0 < a.B;) {
      int b1 = b0, mq = 0;
      long long wgs = 0;
      while (b1 < a.B && wgs + (long long)a.nblk * (a.q_off[b1 + 1] - a.q_off[b1]) <= cap) {
        const int nq = a.q_off[b1 + 1] - a.q_off[b1];
        wgs += (long long)a.nblk * nq;
        mq = nq > mq ? nq : mq;
        ++b1;
      }
      const hipError_t e = launch_kernel("score", score_kernel, dim3(a.nblk, mq, b1 - b0), dim3(256), 0, s, a, b0);
      if (e != hipSuccess) return e;
      a.clear_bar = nullptr;  // cleared by the first launch
      a.clear_err = nullptr;
      b0 = b1;
    }
    return hipSuccess;
  }
  const hipError_t e =
      launch_kernel("logits", logits_kernel, dim3(a.nblk, (maxM + QB - 1) / QB, a.B), dim3(256), 0, s, a);
  if (e != hipSuccess) return e;
  return launch_kernel("softmax_mean", softmax_mean_kernel, dim3(a.nblk, a.B), dim3(256), sizeof(float2) * maxM, s,
                       a);
}

}  // namespace mapk
