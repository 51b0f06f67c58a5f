// Matrix-core GEMM for the predictor projections and the cosine Gram matrix.
//
// C = epilogue(A * B^T) with A [M][K] and B [N][K] both K-contiguous, which is
// the layout of every contraction on the path: token rows times weight rows
// (torch.nn.Linear layout) and token rows times token rows (the Gram matrix).
//
// Tiling for gfx950: a 256-thread workgroup computes a 128x128 tile; its four
// wave64s each own a 64x64 quarter made of 2x2 MFMA 32x32 blocks
// (v_mfma_f32_32x32x16_bf16 for bf16, v_mfma_f32_32x32x2_f32 for float32),
// accumulating in float32.  K advances in 128-byte slices (64 bf16 or 32
// floats per row) that are staged through LDS with a two-slot ring: the next
// slice is fetched into registers while the matrix cores consume the current
// one.  LDS rows are 8 chunks of 16 bytes, XOR-swizzled by (row >> 1) & 7 so that
// the 32 rows one MFMA operand read touches land in different banks.
//
// Several independent problems (for example the first layer of f_V, the
// first layer of f_T and the Gram matrix, which all stream the same visual
// tokens) run in one launch so that the 256 compute units are filled even at
// batch 1.  Workgroups are dispatched round-robin over the 8 XCDs; the block
// index is remapped so that consecutive tiles of a problem run on the same
// XCD and share its L2.
#include "internal.h"

namespace mapk {

namespace {

constexpr int BM = 128;
constexpr int BN = 128;
constexpr int NT = 256;
constexpr int kXcds = 8;

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(16))) float f32x16_t;

template <typename T> struct Slice;
template <> struct Slice<bf16_t> { static constexpr int VEC = 8; static constexpr int BK = 64; };
template <> struct Slice<float> { static constexpr int VEC = 4; static constexpr int BK = 32; };

// LDS rows of a K slice are 8 chunks of 16 bytes; chunk c of row r sits at
// position c ^ swz(r).  Sixteen consecutive rows (the lanes one 16-byte LDS
// access serves together) then put a given chunk in 16 distinct 16-byte slots
// of the 256-byte bank window, so the operand reads are free of bank conflicts.
__device__ __forceinline__ int swz(int r) { return (r >> 1) & 7; }

// Block index -> tile index such that the tiles run by one XCD are contiguous.
__device__ __forceinline__ int xcd_remap(int b, int total) {
  const int per = total / kXcds, rem = total % kXcds;
  const int x = b % kXcds, local = b / kXcds;
  return x * per + min(x, rem) + local;
}

// erf by Abramowitz and Stegun, Handbook of Mathematical Functions, formula
// 7.1.26: for x >= 0, erf(x) = 1 - (a1 t + a2 t^2 + a3 t^3 + a4 t^4 + a5 t^5) e^(-x^2)
// with t = 1 / (1 + p x), absolute error at most 1.5e-7 (6e-7 in float32),
// far below the bfloat16 rounding of the layer's output; erf is odd.  One
// reciprocal, one exponential and five fused multiply-adds, no branches.
__device__ __forceinline__ float erf_as(float x) {
  const float ax = fabsf(x);
  const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f, ax, 1.0f));
  const float poly =
      t * fmaf(t, fmaf(t, fmaf(t, fmaf(t, 1.061405429f, -1.453152027f), 1.421413741f), -0.284496736f), 0.254829592f);
  return copysignf(fmaf(-poly, __expf(-ax * ax), 1.0f), x);
}

__device__ __forceinline__ float gelu_erf(float x) {
  return 0.5f * x * (1.0f + erf_as(x * 0.70710678118654752f));
}

// d/dx [x Phi(x)] = Phi(x) + x phi(x), with Phi from the same erf.
__device__ __forceinline__ float gelu_erf_grad(float x) {
  return fmaf(x * 0.39894228040143268f, __expf(-0.5f * x * x), 0.5f * (1.0f + erf_as(x * 0.70710678118654752f)));
}

template <typename T>
__device__ __forceinline__ void mma_slice(const uint4 (*As)[8], const uint4 (*Bs)[8], int wm, int wn,
                                          int lane, f32x16_t (&acc)[2][2]);

template <>
__device__ __forceinline__ void mma_slice<bf16_t>(const uint4 (*As)[8], const uint4 (*Bs)[8], int wm,
                                                  int wn, int lane, f32x16_t (&acc)[2][2]) {
  // The operands of step s + 1 are read into the other register set before
  // the products of step s issue, so the LDS latency runs under them (the
  // scheduling barriers keep the two sets apart).
  const int lr = lane & 31, lh = lane >> 5;
  bf16x8_t a[2][2], b[2][2];
  auto read = [&](int s, int buf) {
    const int v = 2 * s + lh;  // 16-byte chunk: k = 16 s + 8 lh + (0..7)
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int r = wm * 64 + i * 32 + lr;
      a[buf][i] = __builtin_bit_cast(bf16x8_t, As[r][v ^ swz(r)]);
    }
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int r = wn * 64 + j * 32 + lr;
      b[buf][j] = __builtin_bit_cast(bf16x8_t, Bs[r][v ^ swz(r)]);
    }
  };
  read(0, 0);
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    if (s < 3) read(s + 1, (s + 1) & 1);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[s & 1][i], b[s & 1][j], acc[i][j], 0, 0, 0);
    __builtin_amdgcn_sched_barrier(0);
  }
}

template <>
__device__ __forceinline__ void mma_slice<float>(const uint4 (*As)[8], const uint4 (*Bs)[8], int wm,
                                                 int wn, int lane, f32x16_t (&acc)[2][2]) {
  const int lr = lane & 31, lh = lane >> 5;
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    const int v = 4 * lh + g;  // lane half lh covers k = 16 lh + 4 g + (0..3)
    float4 a[2], b[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int r = wm * 64 + i * 32 + lr;
      a[i] = __builtin_bit_cast(float4, As[r][v ^ swz(r)]);
    }
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int r = wn * 64 + j * 32 + lr;
      b[j] = __builtin_bit_cast(float4, Bs[r][v ^ swz(r)]);
    }
#pragma unroll
    for (int e = 0; e < 4; ++e)
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i][e], b[j][e], acc[i][j], 0, 0, 0);
  }
}

// Row and column of accumulator register r of lane `lane` in a 32x32 block.
__device__ __forceinline__ int acc_row(int r, int lane) { return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3); }
__device__ __forceinline__ int acc_col(int lane) { return lane & 31; }

// Workgroup -> (problem, batch item, tile row, tile column).
// The tiles of the problems before args.first_tiles run first, each class
// XCD-contiguous: the launch puts the layer-1 and fold tiles there, so the
// second wave of workgroups holds only Gram tiles, whose epilogue is shorter.
// A problem split over K (ksplit > 1) runs its tiles once per K range kc,
// the ranges outermost, so that concurrent tiles read the same K columns.
__device__ __forceinline__ void decode_tile(const GemmBatch& args, int& pi, int& bt, int& tm, int& tn, int& kc,
                                            int& local) {
  const int b = blockIdx.x, f = args.first_tiles;
  const int tile = b < f ? xcd_remap(b, f) : f + xcd_remap(b - f, args.total_tiles - f);
  pi = 0;
#pragma unroll
  for (int q = 1; q < kMaxGemmProblems; ++q)
    if (q < args.count && tile >= args.p[q].tile_begin) pi = q;
  const GemmProblem& P = args.p[pi];
  local = tile - P.tile_begin;
  bt = local / P.tiles_per_batch;
  int tt = local - bt * P.tiles_per_batch;
  kc = tt / P.tiles_tri;
  tt -= kc * P.tiles_tri;
  if (P.triangular) {  // upper triangle, row by row: row tm holds tiles_n - tm tiles
    tm = 0;
    while (tt >= P.tiles_n - tm) { tt -= P.tiles_n - tm; ++tm; }
    tn = tm + tt;
  } else {
    tm = tt / P.tiles_n;
    tn = tt - tm * P.tiles_n;
  }
}

// Epilogues on the 128 x 128 accumulator tile.  The RoPE epilogue stages
// the tile through LDS: rows 0..63 in tile_lo, rows 64..127 in tile_hi
// (64 x 128 floats each).
template <typename T>
__device__ __forceinline__ void epilogue(const GemmProblem& P, int bt, int tm, int tn, f32x16_t (&acc)[2][2],
                                         float* tile_lo, float* tile_hi, int tid, int lane, int wm, int wn) {
  const int M = P.M, N = P.N;
  const int m0 = tm * BM, n0 = tn * BN;
  if (epi_direct(P.epi)) {
    const int e = P.epi;
    const T* __restrict__ bias = static_cast<const T*>(P.bias);
    const long long base = bt * P.strideC;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int col = n0 + wn * 64 + j * 32 + acc_col(lane);
      if (col >= N) continue;
      const float bv = (e == EPI_GELU2 && bias) ? to_f32<T>(bias[col]) : 0.0f;
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        // the factor or residual of all 16 entries first (clamped rows), so
        // that no load waits behind this lane's stores
        float f[16];
        if (e == EPI_MUL || e == EPI_RESID) {
          const T* __restrict__ aux = static_cast<const T*>(P.aux) + base;
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int row = min(m0 + wm * 64 + i * 32 + acc_row(r, lane), M - 1);
            f[r] = to_f32<T>(aux[(long long)row * P.ldc + col]);
          }
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = m0 + wm * 64 + i * 32 + acc_row(r, lane);
          if (row >= M) continue;
          const long long at = base + (long long)row * P.ldc + col;
          const float v = acc[i][j][r] + bv;
          if (e == EPI_F32) {
            static_cast<float*>(P.C)[at] = v;
          } else if (e == EPI_GELU2) {
            static_cast<T*>(P.C)[at] = from_f32<T>(gelu_erf(v));
            static_cast<T*>(P.aux)[at] = from_f32<T>(gelu_erf_grad(v));
          } else if (e == EPI_MUL) {
            static_cast<T*>(P.C)[at] = from_f32<T>(v * f[r]);
          } else {
            static_cast<T*>(P.C)[at] = from_f32<T>(v + f[r]);
          }
        }
      }
    }
  } else if (P.epi == EPI_BIAS_GELU || P.epi == EPI_BIAS) {
    T* __restrict__ C = static_cast<T*>(P.C) + bt * P.strideC;
    const T* __restrict__ bias = static_cast<const T*>(P.bias);
    const bool gelu = P.epi == EPI_BIAS_GELU;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int col = n0 + wn * 64 + j * 32 + acc_col(lane);
      if (col >= N) continue;
      const float bv = bias ? to_f32<T>(bias[col]) : 0.0f;
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = m0 + wm * 64 + i * 32 + acc_row(r, lane);
          if (row >= M) continue;
          float v = acc[i][j][r] + bv;
          if (gelu) v = gelu_erf(v);
          C[(long long)row * P.ldc + col] = from_f32<T>(v);
        }
    }
  } else if (P.epi == EPI_COSINE) {
    // Upper-triangle tiles only.  Each value is written to (row, col) and to
    // (col, row), so S is bitwise symmetric; inside a diagonal tile only the
    // entries with row <= col are taken from the accumulators.
    float* __restrict__ S = static_cast<float*>(P.C) + bt * P.strideC;
    const float* __restrict__ rs = P.rs + (long long)bt * M;
    const bool diag = tm == tn;
    const bool vec4 = (P.ldc & 3) == 0;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int col = n0 + wn * 64 + j * 32 + acc_col(lane);
      if (col >= N) continue;
      const float sc = rs[col];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int row0 = m0 + wm * 64 + i * 32 + 8 * q + 4 * (lane >> 5);
          float v[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int row = row0 + e;
            v[e] = row < M ? acc[i][j][4 * q + e] * (rs[row] * sc) : 0.0f;
            if (row < M && (!diag || row <= col)) S[(long long)row * P.ldc + col] = v[e];
          }
          float* dst = S + (long long)col * P.ldc + row0;  // S[col][row0 .. row0 + 3]
          if (!diag && vec4 && row0 + 3 < M) {
            *reinterpret_cast<float4*>(dst) = make_float4(v[0], v[1], v[2], v[3]);
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (row0 + e < M && (!diag || row0 + e < col)) dst[e] = v[e];
          }
        }
    }
  } else {  // EPI_ROPE: stage the tile (plus the bias) in LDS so each thread sees both halves of a pair
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int cl = wn * 64 + j * 32 + acc_col(lane);
      const float bv = (P.rope_bias && n0 + cl < N) ? P.rope_bias[n0 + cl] : 0.0f;
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int rl = wm * 64 + i * 32 + acc_row(r, lane);
          (rl < 64 ? tile_lo : tile_hi)[(rl & 63) * BN + cl] = acc[i][j][r] + bv;
        }
    }
    __syncthreads();
    float* __restrict__ out = static_cast<float*>(P.C) + bt * P.strideC;
    const int half = N >> 1;
    if ((half & 3) == 0 && (P.ldc & 3) == 0) {
      // four pairs per item; each thread issues all its cos/sin loads first
      const int q4 = half >> 2, items = BM * q4;
      for (int e0 = tid; e0 < items; e0 += 8 * NT) {
        float4 cs[8][2];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int e = e0 + u * NT, rl = e / q4, c = 4 * (e - rl * q4);
          const bool ok = e < items && m0 + rl < M;
          const float4* src = reinterpret_cast<const float4*>(P.rope_cs + (long long)(ok ? m0 + rl : 0) * half + c);
          cs[u][0] = ok ? src[0] : make_float4(0.f, 0.f, 0.f, 0.f);
          cs[u][1] = ok ? src[1] : make_float4(0.f, 0.f, 0.f, 0.f);
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int e = e0 + u * NT, rl = e / q4, c = 4 * (e - rl * q4);
          const int row = m0 + rl;
          if (e >= items || row >= M) continue;
          const float* tr = (rl < 64 ? tile_lo : tile_hi) + (rl & 63) * BN;
          const float4 a = *reinterpret_cast<const float4*>(tr + c);
          const float4 b = *reinterpret_cast<const float4*>(tr + c + half);
          const float4 c0 = cs[u][0], c1 = cs[u][1];  // (cos, sin) of pairs c, c+1 | c+2, c+3
          float* o = out + (long long)row * P.ldc + c;
          *reinterpret_cast<float4*>(o) = make_float4(a.x * c0.x - b.x * c0.y, a.y * c0.z - b.y * c0.w,
                                                      a.z * c1.x - b.z * c1.y, a.w * c1.z - b.w * c1.w);
          *reinterpret_cast<float4*>(o + half) = make_float4(b.x * c0.x + a.x * c0.y, b.y * c0.z + a.y * c0.w,
                                                             b.z * c1.x + a.z * c1.y, b.w * c1.z + a.w * c1.w);
        }
      }
      return;
    }
    for (int e = tid; e < BM * half; e += NT) {
      const int rl = e / half, c = e - rl * half;
      const int row = m0 + rl;
      if (row >= M) continue;
      const float* tr = (rl < 64 ? tile_lo : tile_hi) + (rl & 63) * BN;
      const float a = tr[c], b = tr[c + half];
      const float2 cs = P.rope_cs[(long long)row * half + c];
      out[(long long)row * P.ldc + c] = a * cs.x - b * cs.y;
      out[(long long)row * P.ldc + c + half] = b * cs.x + a * cs.y;
    }
  }
}

template <typename T>
__global__ __launch_bounds__(NT) void gemm_kernel(const GemmBatch args) {
  // One contiguous 64 KiB block: A slices in [0, 2), B slices in [2, 4); the
  // RoPE epilogue reuses all of it as a 128 x 128 float tile.
  __shared__ uint4 smem[4][BM][8];
  uint4 (*As)[BM][8] = smem;
  uint4 (*Bs)[BM][8] = smem + 2;
  constexpr int VEC = Slice<T>::VEC;
  constexpr int BK = Slice<T>::BK;

  int pi, bt, tm, tn, kc, local;
  decode_tile(args, pi, bt, tm, tn, kc, local);
  const GemmProblem& P = args.p[pi];
  if (P.run_if && P.run_if[bt] == 0) return;  // (index maps and K ranges: direct-load kernel only)
  const int M = P.M, N = P.N, K = P.K;
  const T* __restrict__ A = static_cast<const T*>(P.A) + bt * P.strideA;
  const T* __restrict__ B = static_cast<const T*>(P.B) + bt * P.strideB;
  const int m0 = tm * BM, n0 = tn * BN;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int lv = tid & 7;          // 16-byte chunk this thread moves
  const int lrow = tid >> 3;       // first row this thread moves (then +32, +64, +96)

  uint4 ra[4], rb[4];
  auto fetch = [&](int k0) {
    const int gk = k0 + lv * VEC;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = lrow + 32 * j;
      const int gm = m0 + r, gn = n0 + r;
      ra[j] = (gm < M && gk < K) ? *reinterpret_cast<const uint4*>(A + (long long)gm * P.lda + gk)
                                 : make_uint4(0, 0, 0, 0);
      rb[j] = (gn < N && gk < K) ? *reinterpret_cast<const uint4*>(B + (long long)gn * P.ldb + gk)
                                 : make_uint4(0, 0, 0, 0);
    }
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = lrow + 32 * j;
      As[buf][r][lv ^ swz(r)] = ra[j];
      Bs[buf][r][lv ^ swz(r)] = rb[j];
    }
  };

  f32x16_t acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int nk = (K + BK - 1) / BK;
  fetch(0);
  stash(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const bool more = kt + 1 < nk;
    if (more) fetch((kt + 1) * BK);
    mma_slice<T>(As[kt & 1], Bs[kt & 1], wm, wn, lane, acc);
    if (more) stash((kt + 1) & 1);
    __syncthreads();
  }

  __syncthreads();  // the RoPE epilogue reuses the LDS tiles
  epilogue<T>(P, bt, tm, tn, acc, reinterpret_cast<float*>(&smem[0][0][0]),
              reinterpret_cast<float*>(&smem[2][0][0]), tid, lane, wm, wn);
}

// Staged epilogues of the direct-load kernel.  After the main loop the four
// 32 KiB stage arrays are free; the finished tile goes through them so that
// every global store moves 16 bytes per lane along a row.
//   q0, q1: the tile in row-major order (rows 0..63 in q0, 64..127 in q1),
//           128 floats per row;
//   t0, t1: the tile transposed (tile columns 0..63 in t0, 64..127 in t1),
//           one tile column per 128-float row whose 16-byte chunks are
//           XOR-swizzled by the column (chunk r/4 at position r/4 ^ (c & 31)),
//           so both the staging writes and the row reads avoid bank conflicts.
struct StagedTile {
  float* q0;
  float* q1;
  float* t0;
  float* t1;
  __device__ float* row(int r) const { return (r < 64 ? q0 : q1) + (r & 63) * BN; }
  // chunk holding tile entries (4 ch .. 4 ch + 3, c), i.e. rows 4 ch .. of column c
  __device__ float* col_chunk(int c, int ch) const { return (c < 64 ? t0 : t1) + (c & 63) * BM + 4 * (ch ^ (c & 31)); }
};

// The staged epilogues take the accumulators of either layout of a 128 x
// 128 tile: J = 2, four waves (wm, wn) of 64 x 64 (2 x 2 blocks, columns
// 64 wn + 32 j), 256 threads; J = 1, eight waves (wm, wn) of 64 x 32 (rows
// 64 wm + 32 i, columns 32 wn), 512 threads.
template <int J> struct EpiThreads { static constexpr int value = J == 2 ? 256 : 512; };

// Bias (+ GELU) in float32, bf16 output.
template <int J>
__device__ __forceinline__ void epi_bias_staged(const GemmProblem& P, int bt, int m0, int n0,
                                                f32x16_t (&acc)[2][J], const StagedTile& L, int tid,
                                                int lane, int wm, int wn) {
  constexpr int NTH = EpiThreads<J>::value;
  const int M = P.M, N = P.N;
  const bf16_t* __restrict__ bias = static_cast<const bf16_t*>(P.bias);
  const bool gelu = P.epi == EPI_BIAS_GELU;
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int cl = wn * (32 * J) + j * 32 + acc_col(lane);
    const float bv = (bias && n0 + cl < N) ? bf16_to_f32(bias[n0 + cl]) : 0.0f;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float v = acc[i][j][r] + bv;
        if (gelu) v = gelu_erf(v);
        L.row(wm * 64 + i * 32 + acc_row(r, lane))[cl] = v;
      }
  }
  __syncthreads();
  bf16_t* __restrict__ C = static_cast<bf16_t*>(P.C) + bt * P.strideC;
  const bool vec = (P.ldc & 7) == 0 && (reinterpret_cast<uintptr_t>(C) & 15) == 0;
#pragma unroll 2
  for (int e = tid; e < BM * (BN / 8); e += NTH) {  // 8 columns per item
    const int r = e >> 4, c8 = (e & 15) * 8;
    const int row = m0 + r, col = n0 + c8;
    if (row >= M || col >= N) continue;
    const float4 x = *reinterpret_cast<const float4*>(L.row(r) + c8);
    const float4 y = *reinterpret_cast<const float4*>(L.row(r) + c8 + 4);
    const float f[8] = {x.x, x.y, x.z, x.w, y.x, y.y, y.z, y.w};
    bf16_t* dst = C + (long long)row * P.ldc + col;
    if (vec && col + 8 <= N) {
      uint4 o;
      o.x = f32_to_bf16(f[0]) | (static_cast<uint32_t>(f32_to_bf16(f[1])) << 16);
      o.y = f32_to_bf16(f[2]) | (static_cast<uint32_t>(f32_to_bf16(f[3])) << 16);
      o.z = f32_to_bf16(f[4]) | (static_cast<uint32_t>(f32_to_bf16(f[5])) << 16);
      o.w = f32_to_bf16(f[6]) | (static_cast<uint32_t>(f32_to_bf16(f[7])) << 16);
      *reinterpret_cast<uint4*>(dst) = o;
    } else {
#pragma unroll
      for (int k = 0; k < 8; ++k)
        if (col + k < N) dst[k] = f32_to_bf16(f[k]);
    }
  }
}

// The training step's and the decoder layer's epilogues, staged like the
// bias epilogue so that every global access moves 16 bytes along a row:
// EPI_F32 (float32 out), EPI_GELU2 (GELU and GELU' of acc + bias), EPI_MUL
// and EPI_RESID (acc times, or plus, the bf16 aux entry), bf16 out.
__device__ __forceinline__ uint4 pack_bf16x8(const float (&f)[8]) {
  uint4 o;
  o.x = f32_to_bf16(f[0]) | (static_cast<uint32_t>(f32_to_bf16(f[1])) << 16);
  o.y = f32_to_bf16(f[2]) | (static_cast<uint32_t>(f32_to_bf16(f[3])) << 16);
  o.z = f32_to_bf16(f[4]) | (static_cast<uint32_t>(f32_to_bf16(f[5])) << 16);
  o.w = f32_to_bf16(f[6]) | (static_cast<uint32_t>(f32_to_bf16(f[7])) << 16);
  return o;
}

template <int J>
__device__ __forceinline__ void epi_direct_staged(const GemmProblem& P, int bt, int m0, int n0,
                                                  f32x16_t (&acc)[2][J], const StagedTile& L, int tid,
                                                  int lane, int wm, int wn) {
  constexpr int NTH = EpiThreads<J>::value;
  const int M = P.M, N = P.N, e = P.epi;
  const bf16_t* __restrict__ bias = static_cast<const bf16_t*>(P.bias);
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int cl = wn * (32 * J) + j * 32 + acc_col(lane);
    const float bv = (e == EPI_GELU2 && bias && n0 + cl < N) ? bf16_to_f32(bias[n0 + cl]) : 0.0f;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) L.row(wm * 64 + i * 32 + acc_row(r, lane))[cl] = acc[i][j][r] + bv;
  }
  __syncthreads();
  const long long base = bt * P.strideC;
  const bool vec = (P.ldc & 7) == 0 && (reinterpret_cast<uintptr_t>(P.C) & 15) == 0 &&
                   (!P.aux || (reinterpret_cast<uintptr_t>(P.aux) & 15) == 0) && (base & 7) == 0;
#pragma unroll 2
  for (int it = tid; it < BM * (BN / 8); it += NTH) {  // 8 columns per item
    const int r = it >> 4, c8 = (it & 15) * 8;
    const int row = m0 + r, col = n0 + c8;
    if (row >= M || col >= N) continue;
    const float4 x = *reinterpret_cast<const float4*>(L.row(r) + c8);
    const float4 y = *reinterpret_cast<const float4*>(L.row(r) + c8 + 4);
    float f[8] = {x.x, x.y, x.z, x.w, y.x, y.y, y.z, y.w};
    const long long at = base + (long long)row * P.ldc + col;
    const int n = min(8, N - col);
    if (e == EPI_F32) {
      float* dst = static_cast<float*>(P.C) + at;
      if (vec && n == 8) {
        reinterpret_cast<float4*>(dst)[0] = x;
        reinterpret_cast<float4*>(dst)[1] = y;
      } else {
        for (int k = 0; k < n; ++k) dst[k] = f[k];
      }
      continue;
    }
    bf16_t* dst = static_cast<bf16_t*>(P.C) + at;
    if (e == EPI_GELU2) {
      float g[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        g[k] = gelu_erf_grad(f[k]);
        f[k] = gelu_erf(f[k]);
      }
      bf16_t* dst2 = static_cast<bf16_t*>(P.aux) + at;
      if (vec && n == 8) {
        *reinterpret_cast<uint4*>(dst) = pack_bf16x8(f);
        *reinterpret_cast<uint4*>(dst2) = pack_bf16x8(g);
      } else {
        for (int k = 0; k < n; ++k) {
          dst[k] = f32_to_bf16(f[k]);
          dst2[k] = f32_to_bf16(g[k]);
        }
      }
      continue;
    }
    const bf16_t* src = static_cast<const bf16_t*>(P.aux) + at;  // EPI_MUL, EPI_RESID
    float a8[8];
    if (vec && n == 8) {
      const uint4 u = *reinterpret_cast<const uint4*>(src);
      const uint32_t w4[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        a8[2 * k] = __uint_as_float(w4[k] << 16);
        a8[2 * k + 1] = __uint_as_float(w4[k] & 0xffff0000u);
      }
    } else {
      for (int k = 0; k < 8; ++k) a8[k] = k < n ? bf16_to_f32(src[k]) : 0.0f;
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) f[k] = e == EPI_MUL ? f[k] * a8[k] : f[k] + a8[k];
    if (vec && n == 8) {
      *reinterpret_cast<uint4*>(dst) = pack_bf16x8(f);
    } else {
      for (int k = 0; k < n; ++k) dst[k] = f32_to_bf16(f[k]);
    }
  }
}

// Cosine: S[row][col] = acc * rs[row] * rs[col] (float32), written to both
// (row, col) and (col, row) from the same float, so S is bitwise symmetric.
// A diagonal tile takes the entries below its diagonal from the transposed
// copy (the mirror of the entries above it).
template <int J>
__device__ __forceinline__ void epi_cosine_staged(const GemmProblem& P, int bt, int tm, int tn,
                                                  f32x16_t (&acc)[2][J], const StagedTile& L,
                                                  const float* rs_rows, const float* rs_cols, int tid,
                                                  int lane, int wm, int wn, bool active = true) {
  constexpr int NTH = EpiThreads<J>::value;
  const int M = P.M, N = P.N, m0 = tm * BM, n0 = tn * BN;
  const bool diag = tm == tn;
#pragma unroll
  for (int j = 0; active && j < J; ++j) {
    const int cl = wn * (32 * J) + j * 32 + acc_col(lane);
    const float sc = rs_cols[cl];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int rl0 = wm * 64 + i * 32 + 8 * q + 4 * (lane >> 5);
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          v[e] = acc[i][j][4 * q + e] * (rs_rows[rl0 + e] * sc);
          L.row(rl0 + e)[cl] = v[e];
        }
        *reinterpret_cast<float4*>(L.col_chunk(cl, rl0 >> 2)) = make_float4(v[0], v[1], v[2], v[3]);
      }
  }
  __syncthreads();
  if (!active) return;  // (a workgroup's other half: only the barrier above)
  float* __restrict__ S = static_cast<float*>(P.C) + bt * P.strideC;
  const bool vec = (P.ldc & 3) == 0;
  // S[m0 + r][n0 + 4 ch ..]: row r of the tile (the mirror below a diagonal tile's diagonal)
  for (int e = tid; e < BM * (BN / 4); e += NTH) {
    const int r = e >> 5, ch = e & 31;
    const int row = m0 + r, col = n0 + 4 * ch;
    if (row >= M || col >= N) continue;
    float4 x = *reinterpret_cast<const float4*>(L.row(r) + 4 * ch);
    if (diag) {  // entry (r, c) with c < r is tile entry (c, r): rows 4 ch .. of column r
      const float4 t = *reinterpret_cast<const float4*>(L.col_chunk(r, ch));
      if (4 * ch + 0 < r) x.x = t.x;
      if (4 * ch + 1 < r) x.y = t.y;
      if (4 * ch + 2 < r) x.z = t.z;
      if (4 * ch + 3 < r) x.w = t.w;
    }
    float* dst = S + (long long)row * P.ldc + col;
    if (vec && col + 4 <= N) {
      *reinterpret_cast<float4*>(dst) = x;
    } else {
      const float f[4] = {x.x, x.y, x.z, x.w};
      for (int k = 0; k < 4 && col + k < N; ++k) dst[k] = f[k];
    }
  }
  if (diag) return;
  // S[n0 + c][m0 + 4 ch ..]: column c of the tile
  for (int e = tid; e < BN * (BM / 4); e += NTH) {
    const int c = e >> 5, ch = e & 31;
    const int row = n0 + c, col = m0 + 4 * ch;
    if (row >= N || col >= M) continue;
    const float4 x = *reinterpret_cast<const float4*>(L.col_chunk(c, ch));
    float* dst = S + (long long)row * P.ldc + col;
    if (vec && col + 4 <= M) {
      *reinterpret_cast<float4*>(dst) = x;
    } else {
      const float f[4] = {x.x, x.y, x.z, x.w};
      for (int k = 0; k < 4 && col + k < M; ++k) dst[k] = f[k];
    }
  }
}

// bf16 variant with a five-stage LDS ring filled by direct global->LDS loads
// (global_load_lds_dwordx4): four K slices are in flight while the matrix
// cores consume the fifth, with no register staging, and the five 32 KiB
// stages fill gfx950's 160 KiB of LDS.  Eight waves, two per SIMD (one
// wave's products run while the other waits on LDS or at the barrier):
// wave (wm, wn) = (w / 4, w % 4) forms 64 x 32 of the tile.  Each wave moves
// 16 rows of A and 16 rows of B per slice, one instruction per 8 rows: lane l lands at row
// 8j + l/8, chunk position l%8 of its instruction's 1 KiB, and fetches the
// chunk the XOR swizzle puts there.  The stages are separate LDS arrays
// addressed with compile-time stage numbers, so the only waits on those
// loads are the explicit counted ones before each barrier.
// Requirements (checked by the host): K % 256 == 0, lda and ldb multiples of
// 8, A and B 16-byte aligned, a staged epilogue (bias, cosine, direct) or
// EPI_PARTIAL.

// LDS byte address of a __shared__ object (the value M0 takes for a direct load).
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) const void*)p));
}

// One global_load_lds_dwordx4: lane l's 16 bytes at gsrc land at byte 16 l
// of the wave's 1 KiB at LDS address m (wave-uniform, passed in M0).  Issued
// from inline assembly so that the compiler adds no waits of its own for
// these loads: it tracks at most four destination arrays of direct loads
// and otherwise drains all of them before every LDS read.  Every read of a
// stage is preceded by the explicit counted wait and the barrier.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"  // M0 is written here and nowhere else in the kernel
__device__ __forceinline__ void dma16(const void* gsrc, uint32_t m) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" : : "v"(gsrc), "s"(m) : "memory", "m0");
}
#pragma clang diagnostic pop

__device__ __forceinline__ void wait_vm_lgkm0(int outstanding) {
  // s_waitcnt encoding: vmcnt in bits [3:0] and [15:14], expcnt [6:4]
  // (7 = no wait), lgkmcnt [11:8]; here vmcnt = outstanding (0, 4, 8, 12,
  // 16 or 24; anything else waits for more) and lgkmcnt = 0
  if (outstanding >= 24) __builtin_amdgcn_s_waitcnt(0x4078);
  else if (outstanding >= 16) __builtin_amdgcn_s_waitcnt(0x4070);
  else if (outstanding >= 12) __builtin_amdgcn_s_waitcnt(0x007c);
  else if (outstanding >= 8) __builtin_amdgcn_s_waitcnt(0x0078);
  else if (outstanding >= 4) __builtin_amdgcn_s_waitcnt(0x0074);
  else __builtin_amdgcn_s_waitcnt(0x0070);
}

// One K slice of the eight-wave 128 x 128 tile: wave (wm, wn) forms rows
// 64 wm + (0..63) by columns 32 wn + (0..31), two 32x32 blocks sharing the B
// operand; the operands of step s + 1 are read before the products of
// step s issue.
__device__ __forceinline__ void mma_slice8(const uint4 (*As)[8], const uint4 (*Bs)[8], int wm, int wn, int lane,
                                           f32x16_t (&acc)[2][1]) {
  const int lr = lane & 31, lh = lane >> 5;
  bf16x8_t a[2][2], b[2];
  auto read = [&](int s, int buf) {
    const int v = 2 * s + lh;  // 16-byte chunk: k = 16 s + 8 lh + (0..7)
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int r = wm * 64 + i * 32 + lr;
      a[buf][i] = __builtin_bit_cast(bf16x8_t, As[r][v ^ swz(r)]);
    }
    const int r = wn * 32 + lr;
    b[buf] = __builtin_bit_cast(bf16x8_t, Bs[r][v ^ swz(r)]);
  };
  read(0, 0);
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    if (s < 3) read(s + 1, (s + 1) & 1);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < 2; ++i)
      acc[i][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[s & 1][i], b[s & 1], acc[i][0], 0, 0, 0);
    __builtin_amdgcn_sched_barrier(0);
  }
}

// Row norms for the workgroups past the tiles: rows of one block spread over
// its waves, two rows per wave at a time.  Each row is summed as prep sums
// it: lane l squares 16-byte chunks l, l + 64, ... in that order, in groups
// of eight, then the wave adds its lanes by a butterfly.
__device__ __forceinline__ void norm_rows(const GemmBatch& args, int blk) {
  const int rows = args.norm_rows, D = args.norm_D, nb = args.norm_blocks;
  const int per = (rows + nb - 1) / nb, r0 = blk * per, r1 = min(rows, r0 + per);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  constexpr int VEC = 8, U = 8;
  const int nchunk = D / VEC;
  for (int r = r0 + 2 * wave; r < r1; r += 2 * nw) {
    const bf16_t* row0 = static_cast<const bf16_t*>(args.norm_V) + (long long)r * D;
    const bf16_t* row1 = static_cast<const bf16_t*>(args.norm_V) + (long long)min(r + 1, r1 - 1) * D;
    float acc[2] = {0.0f, 0.0f};
    for (int c0 = lane; c0 < nchunk; c0 += 64 * U) {
      uint4 uv[2][U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        uv[0][u] = *reinterpret_cast<const uint4*>(row0 + min(c0 + 64 * u, nchunk - 1) * VEC);
        uv[1][u] = *reinterpret_cast<const uint4*>(row1 + min(c0 + 64 * u, nchunk - 1) * VEC);
      }
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int u = 0; u < U; ++u)
          if (c0 + 64 * u < nchunk) {
            // the chunk's eight values in order (low half of each word first)
            const uint32_t wv[4] = {uv[h][u].x, uv[h][u].y, uv[h][u].z, uv[h][u].w};
#pragma unroll
            for (int k = 0; k < VEC; ++k) {
              const uint32_t bits = (k & 1) ? (wv[k >> 1] & 0xffff0000u) : (wv[k >> 1] << 16);
              const float x = __uint_as_float(bits);
              acc[h] = fmaf(x, x, acc[h]);
            }
          }
    }
#pragma unroll
    for (int h = 0; h < 2; ++h) {
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) acc[h] += __shfl_xor(acc[h], off);
      if (lane == 0 && r + h < r1) {
        const float n = sqrtf(acc[h]);
        args.norms[r + h] = n;
        args.ninv[r + h] = n > 0.0f ? 1.0f / n : 0.0f;
      }
    }
  }
}

constexpr int kDmaThreads = 512;

__global__ __launch_bounds__(kDmaThreads) void gemm_dma_kernel(const GemmBatch args) {
  __shared__ uint4 st0[2][BM][8], st1[2][BM][8], st2[2][BM][8], st3[2][BM][8], st4[2][BM][8];  // 5 x 32 KiB
  if (static_cast<int>(blockIdx.x) >= args.total_tiles) {
    norm_rows(args, blockIdx.x - args.total_tiles);
    return;
  }
  int pi, bt, tm, tn, kc, local;
  decode_tile(args, pi, bt, tm, tn, kc, local);
  const GemmProblem& P = args.p[pi];
  if (P.run_if && P.run_if[bt] == 0) return;
  const int M = P.M, N = P.N;
  // this workgroup's K range: kc kl .. min(K, (kc + 1) kl), kl = kchunk (the
  // last range shorter) or K / ksplit
  const int kl = P.ksplit > 1 ? (P.kchunk > 0 ? P.kchunk : P.K / P.ksplit) : P.K;
  const bf16_t* __restrict__ A = static_cast<const bf16_t*>(P.A) + bt * P.strideA + (long long)kc * kl;
  const bf16_t* __restrict__ B = static_cast<const bf16_t*>(P.B) + bt * P.strideB + (long long)kc * kl;
  const int m0 = tm * BM, n0 = tn * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 2, wn = wave & 3;
  const int nk = min(kl, P.K - kc * kl) / 64;
  float rs_mine = 0.0f;  // cosine epilogue: reciprocal norm of tile row tid, or of column tid - BM
  if (P.epi == EPI_COSINE && tid < BM + BN) {
    const float* rs = P.rs + (long long)bt * M;
    const int k = tid < BM ? m0 + tid : n0 + tid - BM;
    if (k < (tid < BM ? M : N)) rs_mine = rs[k];
  }

  // Per-lane global row pointers of this wave's 2 A rows and 2 B rows
  // (rows past the matrix read its last row; they are never stored), through
  // the index maps when there are any.
  const int32_t* mapA = P.mapA ? P.mapA + bt * P.mapStride : nullptr;
  const int32_t* mapB = P.mapB ? P.mapB + bt * P.mapStride : nullptr;
  const bf16_t* ga[2];
  const bf16_t* gb[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int r = 16 * wave + 8 * j + (lane >> 3);
    const int v = (lane & 7) ^ swz(r);  // the chunk the swizzle puts at position lane & 7 of row r
    const int ra = min(m0 + r, M - 1), rb = min(n0 + r, N - 1);
    ga[j] = A + (long long)(mapA ? mapA[ra] : ra) * P.lda + 8 * v;
    gb[j] = B + (long long)(mapB ? mapB[rb] : rb) * P.ldb + 8 * v;
  }
  // this wave's first destination row inside a stage: 16 wave rows of 128 bytes
  const uint32_t wrow = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(wave)) * 16u * 128u;
  auto issue = [&](uint4 (*dst)[BM][8], int kt) {
    const int k0 = kt * 64;
    const uint32_t m = lds_addr(&dst[0][0][0]) + wrow;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      dma16(ga[j] + k0, m + 1024u * j);
      dma16(gb[j] + k0, m + BM * 128u + 1024u * j);
    }
  };

  f32x16_t acc[2][1];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[i][0][r] = 0.0f;

  // Step kt waits for slice kt (this wave's loads, then every wave's at the
  // barrier), refills the stage every wave finished reading in the previous
  // step with slice kt + 4, and runs the matrix cores on slice kt.  Slice kt
  // sits in stage kt % 5, a compile-time constant in the unrolled body; the
  // early exits are uniform scalar branches.
  auto mma = [&](uint4 (*cur)[BM][8]) { mma_slice8(cur[0], cur[1], wm, wn, lane, acc); };
  auto step = [&](uint4 (*cur)[BM][8], uint4 (*nxt)[BM][8], int kt) {
    wait_vm_lgkm0(4 * min(3, nk - 1 - kt));
    __builtin_amdgcn_s_barrier();
    if (kt + 4 < nk) issue(nxt, kt + 4);
    mma(cur);
  };
  issue(st0, 0);
  issue(st1, 1);
  issue(st2, 2);
  issue(st3, 3);
  step(st0, st4, 0);
  for (int kt = 1; kt < nk; kt += 5) {
    step(st1, st0, kt);
    if (kt + 1 >= nk) break;
    step(st2, st1, kt + 1);
    if (kt + 2 >= nk) break;
    step(st3, st2, kt + 2);
    if (kt + 3 >= nk) break;
    step(st4, st3, kt + 3);
    if (kt + 4 >= nk) break;
    step(st0, st4, kt + 4);
  }
  if (P.epi == EPI_PARTIAL) {
    // the raw sums of this K range in the four-wave layout the reductions
    // read: entries (i, j, 4 g .. 4 g + 3) of that layout's thread t (wave
    // 2 wm + wn / 2, j = wn % 2) as float4 q = (2 i + j) 4 + g at q * 256 + t
    // (every store of a wave contiguous)
    float4* dst = static_cast<float4*>(P.C) + (long long)local * (16 * 256);
    const int t4 = (2 * wm + (wn >> 1)) * 64 + lane, j4 = wn & 1;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        dst[((2 * i + j4) * 4 + g) * 256 + t4] =
            make_float4(acc[i][0][4 * g], acc[i][0][4 * g + 1], acc[i][0][4 * g + 2], acc[i][0][4 * g + 3]);
    return;
  }
  __syncthreads();  // the epilogues reuse the stage arrays
  float* rs_tile = reinterpret_cast<float*>(&st4[0][0][0]);
  if (P.epi == EPI_COSINE) {
    if (tid < BM + BN) rs_tile[tid] = rs_mine;
    __syncthreads();
  }
  const StagedTile L{reinterpret_cast<float*>(&st0[0][0][0]), reinterpret_cast<float*>(&st1[0][0][0]),
                     reinterpret_cast<float*>(&st2[0][0][0]), reinterpret_cast<float*>(&st3[0][0][0])};
  if (P.epi == EPI_COSINE)
    epi_cosine_staged<1>(P, bt, tm, tn, acc, L, rs_tile, rs_tile + BM, tid, lane, wm, wn);
  else if (P.epi == EPI_BIAS_GELU || P.epi == EPI_BIAS)
    epi_bias_staged<1>(P, bt, m0, n0, acc, L, tid, lane, wm, wn);
  else
    epi_direct_staged<1>(P, bt, m0, n0, acc, L, tid, lane, wm, wn);
}

// ------------------------------------------------------------ 256 x 256 tiles
// Launches of several waves of workgroups (the first layer over a batch of
// images, the decoder layer's long products) run 256 x 256 tiles: per
// product a compute unit then moves half the bytes from L2 into LDS and
// reads half as many operand bytes from LDS as with 128 x 128 tiles, which
// is what bounds the smaller tile.  512 threads, eight wave64s, two per
// SIMD; wave w (group h = w / 4, (qm, qn) = ((w / 2) % 2, w % 2)) owns rows
// 128 h + 64 qm + (0..63) and columns 128 s + 64 qn + (0..63) for s = 0, 1,
// i.e. 2 x 4 MFMA 32x32 blocks whose two A operands serve four products.
// Group h then holds sub-tiles (h, 0) and (h, 1) in the 128 x 128 kernel's
// accumulator layout and finishes them with its epilogues, staging through
// its own 64 KiB; the cosine epilogue (a Gram matrix's upper triangle of
// tiles, mirrored) needs 128 KiB per sub-tile, so the two groups take turns
// there, sub-tile by sub-tile, and a diagonal tile's sub-tile below the
// diagonal is the mirror of the one above it.  Two 64 KiB stages: one K
// slice loads while the matrix cores consume the other.  Tiles are ordered
// in groups of kBigRows tile rows, column by column inside a group (a
// triangular problem: its upper triangle row by row), each XCD taking a
// contiguous range.
constexpr int kBig = 256;
constexpr int kBigThreads = 512;
constexpr int kBigRows = 4;

__global__ __launch_bounds__(kBigThreads) void gemm_big_kernel(const GemmBatch args) {
  __shared__ uint4 bst0[2 * kBig][8], bst1[2 * kBig][8];  // per stage: A rows, then B rows
  __shared__ float rs_big[2 * kBig];                       // cosine: 1/norm of the tile's rows, then columns
  const int tile = xcd_remap(blockIdx.x, args.total_tiles);
  int pi = 0;
#pragma unroll
  for (int q = 1; q < kMaxGemmProblems; ++q)
    if (q < args.count && tile >= args.p[q].tile_begin) pi = q;
  const GemmProblem& P = args.p[pi];
  const int local = tile - P.tile_begin;
  const int bt = local / P.tiles_per_batch;
  int tt = local - bt * P.tiles_per_batch, tm, tn;
  if (P.triangular) {  // upper triangle, row by row: row tm holds tiles_n - tm tiles
    tm = 0;
    while (tt >= P.tiles_n - tm) { tt -= P.tiles_n - tm; ++tm; }
    tn = tm + tt;
  } else {
    const int grp = tt / (kBigRows * P.tiles_n), first = grp * kBigRows;
    const int rows = min(kBigRows, P.tiles_m - first), in = tt - grp * kBigRows * P.tiles_n;
    tm = first + in % rows;
    tn = in / rows;
  }
  if (P.run_if && P.run_if[bt] == 0) return;
  const int M = P.M, N = P.N, m0 = tm * kBig, n0 = tn * kBig;
  const bf16_t* __restrict__ A = static_cast<const bf16_t*>(P.A) + bt * P.strideA;
  const bf16_t* __restrict__ B = static_cast<const bf16_t*>(P.B) + bt * P.strideB;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int h = wave >> 2, qm = (wave >> 1) & 1, qn = wave & 1;
  const int nk = P.K / 64;
  float rs_mine = 0.0f;  // cosine epilogue: 1/norm of tile row tid, or of column tid - 256
  if (P.epi == EPI_COSINE) {
    const int k = tid < kBig ? m0 + tid : n0 + tid - kBig;
    if (k < (tid < kBig ? M : N)) rs_mine = P.rs[(long long)bt * M + k];
  }
  // wave w loads rows 32 w .. 32 w + 31 of the A tile and of the B tile,
  // one instruction per 8 rows (rows past the matrix read its last row)
  const int32_t* mapA = P.mapA ? P.mapA + bt * P.mapStride : nullptr;
  const int32_t* mapB = P.mapB ? P.mapB + bt * P.mapStride : nullptr;
  const bf16_t* ga[4];
  const bf16_t* gb[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int r = 32 * wave + 8 * j + (lane >> 3);
    const int v = (lane & 7) ^ swz(r);
    const int ra = min(m0 + r, M - 1), rb = min(n0 + r, N - 1);
    ga[j] = A + (long long)(mapA ? mapA[ra] : ra) * P.lda + 8 * v;
    gb[j] = B + (long long)(mapB ? mapB[rb] : rb) * P.ldb + 8 * v;
  }
  const uint32_t wrow = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(wave)) * 32u * 128u;
  auto issue = [&](uint4 (*dst)[8], int kt) {
    const int k0 = kt * 64;
    const uint32_t m = lds_addr(&dst[0][0]) + wrow;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      dma16(ga[j] + k0, m + 1024u * j);
      dma16(gb[j] + k0, m + kBig * 128u + 1024u * j);
    }
  };
  f32x16_t acc[2][2][2];  // [s][i][j]: rows 128 h + 64 qm + 32 i, columns 128 s + 64 qn + 32 j
#pragma unroll
  for (int s = 0; s < 2; ++s)
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[s][i][j][r] = 0.0f;
  const int lr = lane & 31, lh = lane >> 5;
  // Row norms (args.norm_tiles): in the first tile column each wave also
  // sums the squares of one of the two A operands it reads, the one of rows
  // 128 h + 64 qm + 32 qn + (0..31) (lane l: row l & 31, the k-half l >> 5 of
  // every 16), in float32, slice after slice; the two halves are added at
  // the end.  (The two waves of a (h, qm) pair read the same A operands and
  // sit on different SIMDs, so each SIMD gets an equal share.)
  const bool sumsq = args.norm_tiles == pi + 1 && tn == 0;
  float nacc = 0.0f;
  // The operands of one step of 16 (two buffers: those of the next step are
  // read while the products of this one run), and the step's products.
  bf16x8_t a[2][2], b[2][4];
  auto read = [&](const uint4 (*st)[8], int s, int buf) {
    const uint4 (*As)[8] = st;
    const uint4 (*Bs)[8] = st + kBig;
    const int v = 2 * s + lh;  // 16-byte chunk: k = 16 s + 8 lh + (0..7)
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int r = 128 * h + 64 * qm + 32 * i + lr;
      a[buf][i] = __builtin_bit_cast(bf16x8_t, As[r][v ^ swz(r)]);
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int r = 128 * (c >> 1) + 64 * qn + 32 * (c & 1) + lr;
      b[buf][c] = __builtin_bit_cast(bf16x8_t, Bs[r][v ^ swz(r)]);
    }
  };
  auto products = [&](int buf) {
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int c = 0; c < 4; ++c)
        acc[c >> 1][i][c & 1] =
            __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[buf][i], b[buf][c], acc[c >> 1][i][c & 1], 0, 0, 0);
    if (sumsq) {  // (vector ALU work under the products)
      const uint4 u = __builtin_bit_cast(uint4, qn ? a[buf][1] : a[buf][0]);
      const uint32_t wv[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const float x = __uint_as_float((k & 1) ? (wv[k >> 1] & 0xffff0000u) : (wv[k >> 1] << 16));
        nacc = fmaf(x, x, nacc);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
  };
  // Slice kt sits in stage kt % 2.  The wait for slice kt + 1 and the
  // barrier come before the products of kt's last step, so that the next
  // slice's first operands are read while those run; the barrier also means
  // every wave is done reading slice kt, whose stage receives slice kt + 2
  // at the start of the next step.
  issue(bst0, 0);
  wait_vm_lgkm0(0);
  __builtin_amdgcn_s_barrier();
  read(bst0, 0, 0);
  for (int kt = 0; kt < nk; ++kt) {
    uint4 (*cur)[8] = (kt & 1) ? bst1 : bst0;
    uint4 (*nxt)[8] = (kt & 1) ? bst0 : bst1;
    if (kt + 1 < nk) issue(nxt, kt + 1);
    read(cur, 1, 1);
    products(0);
    read(cur, 2, 0);
    products(1);
    read(cur, 3, 1);
    products(0);
    if (kt + 1 < nk) {
      wait_vm_lgkm0(0);
      __builtin_amdgcn_s_barrier();
      read(nxt, 0, 0);
    }
    products(1);
  }
  if (sumsq) {
    const float t = nacc + __shfl_xor(nacc, 32);
    const int row = m0 + 128 * h + 64 * qm + 32 * qn + lr;
    if (lh == 0 && row < M) {
      const float n = sqrtf(t);
      args.norms[row] = n;
      args.ninv[row] = n > 0.0f ? 1.0f / n : 0.0f;
    }
  }
  __syncthreads();  // the epilogues reuse the stages: group h stages through bst<h>
  if (P.epi == EPI_COSINE) {
    rs_big[tid] = rs_mine;
    const StagedTile LC{reinterpret_cast<float*>(&bst0[0][0]), reinterpret_cast<float*>(&bst0[0][0]) + 64 * BN,
                        reinterpret_cast<float*>(&bst1[0][0]), reinterpret_cast<float*>(&bst1[0][0]) + 64 * BM};
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const int TM = 2 * tm + hh, TN = 2 * tn + s;  // the sub-tile in 128 x 128 tiles
        if (TM > TN || TM * BM >= M || TN * BN >= N) continue;  // (uniform over the workgroup)
        __syncthreads();  // the staging is free (and rs_big written)
        epi_cosine_staged<2>(P, bt, TM, TN, acc[s], LC, rs_big + 128 * hh, rs_big + kBig + 128 * s,
                             tid & (NT - 1), lane, qm, qn, h == hh);
      }
    return;
  }
  float* stg = reinterpret_cast<float*>(h ? &bst1[0][0] : &bst0[0][0]);
  const StagedTile L{stg, stg + 64 * BN, nullptr, nullptr};
  const int t2 = tid & (NT - 1);
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    if (s) __syncthreads();  // the staging is read out before it is written again
    if (P.epi == EPI_BIAS_GELU || P.epi == EPI_BIAS)
      epi_bias_staged<2>(P, bt, m0 + 128 * h, n0 + 128 * s, acc[s], L, t2, lane, qm, qn);
    else
      epi_direct_staged<2>(P, bt, m0 + 128 * h, n0 + 128 * s, acc[s], L, t2, lane, qm, qn);
  }
}

// Projection to d_p <= 128 columns with the RoPE epilogue (the keys and
// queries of Eq. (3)): C = RoPE(A B^T + bias), A [M][K] and B [N][K] bf16
// (float32 inputs: the same with 32 x 32 x 2 float32 products).
// With N this small and rows for fewer than one wave of tiles, a 128 x 128
// tile leaves most compute units idle, each streaming the whole K with a
// few slices in flight.  Here a workgroup takes
// 32 rows and one of two groups of RoPE pairs: with half = N / 2 and
// PG = ceil(half / 2), group g holds pairs c = g PG .. (g + 1) PG - 1, i.e.
// columns c and c + half, so every rotation is local and each workgroup
// reads half of B.  Its eight waves split K: wave w takes the 64-wide chunks
// w, w + 8, ...  Lane l reads 64 contiguous bytes of row l & 31 per chunk, A
// and B alike, straight from global memory into registers, and the chunk's
// four products consume them in an order shared by both operands (any
// common order of k gives the same sum).  The eight partial tiles are summed
// in LDS in a fixed order.
// Requirements (checked by the host): N <= 128 and even, K, lda and ldb
// multiples of 8, A and B 16-byte aligned, one batch item.
constexpr int kPR = 32;   // rows per workgroup
constexpr int kPW = 8;    // waves per workgroup
constexpr int kPG = 2;    // groups of RoPE pairs per row block
constexpr int kPS = 68;   // LDS row stride of the partial tiles (floats)

typedef __attribute__((ext_vector_type(4))) float float4v;

template <typename T>
__global__ __launch_bounds__(kPW * 64) void proj_rope_kernel(const GemmBatch args) {
  __shared__ float part[kPW][kPR][kPS];
  const int t0 = args.p[0].tiles_m, pi = blockIdx.x < t0 ? 0 : 1;
  const GemmProblem& P = args.p[pi];
  const int local = blockIdx.x - (pi ? t0 : 0), g = local % kPG;
  const int m0 = (local / kPG) * kPR;
  const int M = P.M, K = P.K, half = P.N >> 1;
  const int PG = (half + kPG - 1) / kPG, c0 = g * PG, npg = min(PG, half - c0);
  if (npg <= 0) return;  // a group without pairs (half = 1)
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const T* __restrict__ A = static_cast<const T*>(P.A);
  const T* __restrict__ B = static_cast<const T*>(P.B);

  const int r = lane & 31, h = lane >> 5;
  const T* arow = A + (long long)min(m0 + r, M - 1) * P.lda;
  const int pr = c0 + min(r, npg - 1);  // the pair of tile column r (32 + r: its partner)
  const T* brow[2] = {B + (long long)pr * P.ldb, B + (long long)(pr + half) * P.ldb};
  f32x16_t acc[2];
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[j][e] = 0.0f;
  const int nchunk = (K + 63) >> 6;
  if constexpr (sizeof(T) == 4) {
    // float32: per 64-wide chunk lane l holds 32 contiguous k of its row
    // (half h = l >> 5 of the chunk), for A and B alike; the 32 x 32 x 2
    // products pair k = s of the first half with k = 32 + s of the second
    // (any common order of k gives the same sum)
    for (int kc = wave; kc < nchunk; kc += kPW) {
      const int kb = 64 * kc + 32 * h;
      float4v av[8], bv[2][8];
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const int k = kb + 4 * q;
        const int off = k < K ? k : 0;  // past K: a valid address, zeroed below
        av[q] = *reinterpret_cast<const float4v*>(arow + off);
#pragma unroll
        for (int j = 0; j < 2; ++j) bv[j][q] = *reinterpret_cast<const float4v*>(brow[j] + off);
      }
      __builtin_amdgcn_sched_barrier(0);  // keep the loads ahead of the products
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const float4v z = {0.0f, 0.0f, 0.0f, 0.0f};
        const float4v a = kb + 4 * q < K ? av[q] : z;
#pragma unroll
        for (int e = 0; e < 4; ++e)
#pragma unroll
          for (int j = 0; j < 2; ++j)
            acc[j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[e], bv[j][q][e], acc[j], 0, 0, 0);
      }
    }
  } else
  for (int kc = wave; kc < nchunk; kc += 2 * kPW) {  // two chunks per pass, every load issued first
    uint4 av[2][4], bv[2][2][4];
#pragma unroll
    for (int c2 = 0; c2 < 2; ++c2)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int k = 64 * (kc + kPW * c2) + 32 * h + 8 * q;
        const int off = k < K ? k : 0;  // past K: a valid address, zeroed below
        av[c2][q] = *reinterpret_cast<const uint4*>(arow + off);
#pragma unroll
        for (int j = 0; j < 2; ++j) bv[c2][j][q] = *reinterpret_cast<const uint4*>(brow[j] + off);
      }
    __builtin_amdgcn_sched_barrier(0);  // keep the loads ahead of the products
#pragma unroll
    for (int c2 = 0; c2 < 2; ++c2)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int k = 64 * (kc + kPW * c2) + 32 * h + 8 * q;
        const uint4 z = {0u, 0u, 0u, 0u};
        const bf16x8_t a = __builtin_bit_cast(bf16x8_t, k < K ? av[c2][q] : z);
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, __builtin_bit_cast(bf16x8_t, bv[c2][j][q]), acc[j],
                                                           0, 0, 0);
      }
  }
  // the epilogue's (cos, sin) pairs and biases (item e = row e / npg, pair
  // c0 + e % npg; at most two per thread), in flight while the partials meet
  constexpr int EI = kPR * 32 / (kPW * 64);
  float2 cs[EI];
  float bl[EI], bh[EI];
#pragma unroll
  for (int u = 0; u < EI; ++u) {
    const int e = min(tid + kPW * 64 * u, kPR * npg - 1), rl = e / npg, c = c0 + e - rl * npg;
    cs[u] = P.rope_cs[(long long)min(m0 + rl, M - 1) * half + c];
    bl[u] = P.rope_bias ? P.rope_bias[c] : 0.0f;
    bh[u] = P.rope_bias ? P.rope_bias[c + half] : 0.0f;
  }
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int e = 0; e < 16; ++e) part[wave][acc_row(e, lane)][32 * j + acc_col(lane)] = acc[j][e];
  __syncthreads();
  float* __restrict__ out = static_cast<float*>(P.C);
#pragma unroll
  for (int u = 0; u < EI; ++u) {
    const int e = tid + kPW * 64 * u, rl = e / npg, cl = e - rl * npg;
    if (e >= kPR * npg || m0 + rl >= M) continue;
    float s0[kPW], s1[kPW];
#pragma unroll
    for (int w = 0; w < kPW; ++w) {
      s0[w] = part[w][rl][cl];
      s1[w] = part[w][rl][32 + cl];
    }
    const float a = (((s0[0] + s0[1]) + (s0[2] + s0[3])) + ((s0[4] + s0[5]) + (s0[6] + s0[7]))) + bl[u];
    const float b = (((s1[0] + s1[1]) + (s1[2] + s1[3])) + ((s1[4] + s1[5]) + (s1[6] + s1[7]))) + bh[u];
    float* o = out + (long long)(m0 + rl) * P.ldc + c0 + cl;
    o[0] = a * cs[u].x - b * cs[u].y;
    o[half] = b * cs[u].x + a * cs[u].y;
  }
}

// The K ranges of a split problem summed in order kc = 0, 1, ...: workgroup
// (tile t, piece q, batch item) takes float4 q of every thread of the
// tile's partials, i.e. accumulator block (i, j) = (q / 8, q / 4 % 2), rows
// 4 (q % 4) .. + 3 of the thread's 32 x 32 block layout, and writes those
// entries of S and their mirror as the cosine epilogue does.
__global__ __launch_bounds__(NT) void gram_reduce_kernel(const GemmProblem P, float* out, int ldc,
                                                         const float* rs_all) {
  const int bt = blockIdx.y, t = blockIdx.x >> 4, q = blockIdx.x & 15;
  if (P.run_if && P.run_if[bt] == 0) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int ks = P.ksplit > 1 ? P.ksplit : 1;
  int tm = 0, tt = t;
  while (tt >= P.tiles_n - tm) {
    tt -= P.tiles_n - tm;
    ++tm;
  }
  const int tn = tm + tt;
  const float4* src = static_cast<const float4*>(P.C) + (long long)bt * P.tiles_per_batch * (16 * NT);
  float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
  float4 x[16];
#pragma unroll
  for (int kc = 0; kc < 16; ++kc)
    if (kc < ks) x[kc] = src[((long long)kc * P.tiles_tri + t) * (16 * NT) + q * NT + tid];
#pragma unroll
  for (int kc = 0; kc < 16; ++kc)
    if (kc < ks) {
      v.x += x[kc].x;
      v.y += x[kc].y;
      v.z += x[kc].z;
      v.w += x[kc].w;
    }
  for (int kc = 16; kc < ks; ++kc) {
    const float4 y = src[((long long)kc * P.tiles_tri + t) * (16 * NT) + q * NT + tid];
    v.x += y.x;
    v.y += y.y;
    v.z += y.z;
    v.w += y.w;
  }
  const int i = q >> 3, j = (q >> 2) & 1, g = q & 3;
  const int M = P.M, m0 = tm * BM, n0 = tn * BN;
  const bool diag = tm == tn;
  const int col = n0 + wn * 64 + j * 32 + acc_col(lane);
  const int row0 = m0 + wm * 64 + i * 32 + 8 * g + 4 * (lane >> 5);
  if (col >= M) return;
  const float* rs = rs_all + (long long)bt * M;
  float* S = out + (long long)bt * M * ldc;
  const float sc = rs[col];
  const float a[4] = {v.x, v.y, v.z, v.w};
  float w[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int row = row0 + e;
    w[e] = row < M ? a[e] * (rs[row] * sc) : 0.0f;
    if (row < M && (!diag || row <= col)) S[(long long)row * ldc + col] = w[e];
  }
  float* dst = S + (long long)col * ldc + row0;  // S[col][row0 .. row0 + 3]
  if (!diag && (ldc & 3) == 0 && row0 + 3 < M) {
    *reinterpret_cast<float4*>(dst) = make_float4(w[0], w[1], w[2], w[3]);
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (row0 + e < M && (!diag || row0 + e < col)) dst[e] = w[e];
  }
}

}  // namespace

// (tile t, piece q) of a plain (not triangular) problem split over K: the
// K ranges' float4 q of every thread summed in range order, plus the bf16
// residual at the same entries, stored as bf16 (the decoder layer's output
// projections).
__global__ __launch_bounds__(NT) void splitk_resid_kernel(const GemmProblem P, const bf16_t* __restrict__ res,
                                                          bf16_t* __restrict__ out, int ldc) {
  const int t = blockIdx.x >> 4, q = blockIdx.x & 15;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int ks = P.ksplit > 1 ? P.ksplit : 1;
  const int tm = t / P.tiles_n, tn = t - tm * P.tiles_n;
  const float4* src = static_cast<const float4*>(P.C);
  float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int kc0 = 0; kc0 < ks; kc0 += 8) {
    float4 x[8];
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (kc0 + u < ks) x[u] = src[((long long)(kc0 + u) * P.tiles_tri + t) * (16 * NT) + q * NT + tid];
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (kc0 + u < ks) {
        v.x += x[u].x;
        v.y += x[u].y;
        v.z += x[u].z;
        v.w += x[u].w;
      }
  }
  const int i = q >> 3, j = (q >> 2) & 1, g = q & 3;
  const int col = tn * BN + wn * 64 + j * 32 + acc_col(lane);
  const int row0 = tm * BM + wm * 64 + i * 32 + 8 * g + 4 * (lane >> 5);
  if (col >= P.N) return;
  const float f[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int row = row0 + e;
    if (row < P.M) {
      const long long at = (long long)row * ldc + col;
      out[at] = f32_to_bf16(f[e] + bf16_to_f32(res[at]));
    }
  }
}

hipError_t launch_splitk_resid(const GemmProblem& P, const void* res, void* out, int ldc, hipStream_t s) {
  if (P.tiles_tri == 0) return hipSuccess;
  return launch_kernel("splitk_resid", splitk_resid_kernel, dim3(P.tiles_tri * 16), dim3(NT), 0, s, P,
                       static_cast<const bf16_t*>(res), static_cast<bf16_t*>(out), ldc);
}

hipError_t launch_gram_reduce(const GemmProblem& partial, float* out, int ldc, const float* rs, hipStream_t s,
                              const char* name) {
  if (partial.tiles_tri == 0 || partial.batch == 0) return hipSuccess;
  return launch_kernel(name, gram_reduce_kernel, dim3(partial.tiles_tri * 16, partial.batch), dim3(NT), 0,
                       s, partial, out, ldc, rs);
}

void gemm_finalize(GemmBatch& g) {
  int begin = 0;
  for (int i = 0; i < g.count; ++i) {
    GemmProblem& p = g.p[i];
    p.tiles_m = (p.M + BM - 1) / BM;
    p.tiles_n = (p.N + BN - 1) / BN;
    p.tiles_tri = p.triangular ? p.tiles_m * (p.tiles_m + 1) / 2 : p.tiles_m * p.tiles_n;
    p.tiles_per_batch = p.tiles_tri * (p.ksplit > 1 ? p.ksplit : 1);
    p.tile_begin = begin;
    begin += p.tiles_per_batch * p.batch;
  }
  g.total_tiles = begin;
  // a trailing cosine problem (the Gram matrix) runs after the others
  g.first_tiles = g.count > 1 && g.p[g.count - 1].epi == EPI_COSINE ? g.p[g.count - 1].tile_begin : 0;
}

// K ranges of a split problem: equal ranges (K / ksplit) or kchunk-long ones
// with a shorter last range, each a positive multiple of 256.
static bool k_ranges_ok(const GemmProblem& p) {
  if (p.ksplit <= 1) return true;
  if (p.kchunk > 0) return p.kchunk % 256 == 0 && (long long)(p.ksplit - 1) * p.kchunk < p.K;
  return p.K % p.ksplit == 0 && (p.K / p.ksplit) % 256 == 0;
}

// The epilogues of the direct-load kernel (the RoPE epilogue runs in the
// register-staged kernel or the projection kernel).
static bool dma_epilogue(int e) {
  return e == EPI_BIAS_GELU || e == EPI_BIAS || e == EPI_COSINE || e == EPI_PARTIAL || epi_direct(e);
}

bool gemm_direct_loads(map_dtype dt, const GemmBatch& g) {
  if (dt != MAP_BF16) return false;
  bool dma = true;  // every problem meets the direct-load requirements
  for (int i = 0; i < g.count; ++i) {
    const GemmProblem& p = g.p[i];
    dma = dma && dma_epilogue(p.epi) && p.K % 256 == 0 && p.lda % 8 == 0 && p.ldb % 8 == 0 &&
          (reinterpret_cast<uintptr_t>(p.A) & 15) == 0 && (reinterpret_cast<uintptr_t>(p.B) & 15) == 0 &&
          p.strideA % 8 == 0 && p.strideB % 8 == 0 &&
          k_ranges_ok(p);
  }
  return dma;
}

// Compute units of the current device (cached per device).
static int gemm_cus() {
  static int cached[16] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 16) return 256;
  if (cached[dev] == 0) {
    int c = 0;
    cached[dev] = hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && c > 0 ? c : 256;
  }
  return cached[dev];
}

// 256 x 256 tiles for a direct-load launch whose problems all have a
// row-wise epilogue (bias, GELU, float32, GELU', product, residual) or are a
// Gram matrix's upper triangle (cosine), and no K split, when they take
// fewer waves of workgroups: a wave of 256 x 256
// tiles costs about 2.3 waves of 128 x 128 tiles (measured on the first
// layer's and the decoder layer's shapes).
static bool big_tiles_pay(const GemmBatch& g) {
  if (g.norm_blocks) return false;
  if (g.norm_tiles > 0 && (g.norm_tiles > g.count || g.p[g.norm_tiles - 1].batch != 1)) return false;
  long long t128 = 0, t256 = 0;
  for (int i = 0; i < g.count; ++i) {
    const GemmProblem& p = g.p[i];
    const bool gram = p.epi == EPI_COSINE && p.triangular && p.M == p.N;
    if (!(p.epi == EPI_BIAS || p.epi == EPI_BIAS_GELU || epi_direct(p.epi) || gram) || p.ksplit > 1 ||
        (p.triangular && !gram))
      return false;
    const long long a = (p.M + 127) / 128, b = (p.N + 127) / 128;
    const long long c = (p.M + kBig - 1) / kBig, d = (p.N + kBig - 1) / kBig;
    t128 += (gram ? a * (a + 1) / 2 : a * b) * p.batch;
    t256 += (gram ? c * (c + 1) / 2 : c * d) * p.batch;
  }
  const long long cus = gemm_cus();
  return 23 * ((t256 + cus - 1) / cus) < 10 * ((t128 + cus - 1) / cus);
}

static void finalize_big(GemmBatch& g) {
  int begin = 0;
  for (int i = 0; i < g.count; ++i) {
    GemmProblem& p = g.p[i];
    p.tiles_m = (p.M + kBig - 1) / kBig;
    p.tiles_n = (p.N + kBig - 1) / kBig;
    p.tiles_tri = p.triangular ? p.tiles_m * (p.tiles_m + 1) / 2 : p.tiles_m * p.tiles_n;
    p.tiles_per_batch = p.tiles_tri;
    p.tile_begin = begin;
    begin += p.tiles_per_batch * p.batch;
  }
  g.total_tiles = begin;
  g.first_tiles = 0;
}

bool gemm_big_tiles(map_dtype dt, const GemmBatch& g) { return gemm_direct_loads(dt, g) && big_tiles_pay(g); }

hipError_t launch_gemm(map_dtype dt, const GemmBatch& g, const char* name, hipStream_t s) {
  if (g.total_tiles == 0) return hipSuccess;
  // the in-tile row norms exist in the 256 x 256 kernel only
  if (g.norm_tiles > 0 && !gemm_big_tiles(dt, g)) return hipErrorInvalidValue;
  if (dt == MAP_BF16) {
    bool dma = true;  // every problem meets the direct-load requirements
    for (int i = 0; i < g.count; ++i) {
      const GemmProblem& p = g.p[i];
      dma = dma && dma_epilogue(p.epi) && p.K % 256 == 0 && p.lda % 8 == 0 && p.ldb % 8 == 0 &&
            (reinterpret_cast<uintptr_t>(p.A) & 15) == 0 && (reinterpret_cast<uintptr_t>(p.B) & 15) == 0 &&
            p.strideA % 8 == 0 && p.strideB % 8 == 0 &&
            k_ranges_ok(p);
    }
    if (dma && big_tiles_pay(g)) {
      GemmBatch q = g;
      finalize_big(q);
      return launch_kernel(name, gemm_big_kernel, dim3(q.total_tiles), dim3(kBigThreads), 0, s, q);
    }
    if (dma)
      return launch_kernel(name, gemm_dma_kernel, dim3(g.total_tiles + g.norm_blocks), dim3(kDmaThreads), 0, s, g);
    if (g.norm_blocks) return hipErrorInvalidValue;
    for (int i = 0; i < g.count; ++i)  // index maps and K ranges exist in the direct-load kernel only
      if (g.p[i].epi == EPI_PARTIAL || g.p[i].mapA || g.p[i].mapB) return hipErrorInvalidValue;
    return launch_kernel(name, gemm_kernel<bf16_t>, dim3(g.total_tiles), dim3(NT), 0, s, g);
  }
  return launch_kernel(name, gemm_kernel<float>, dim3(g.total_tiles), dim3(NT), 0, s, g);
}

hipError_t launch_proj_rope(map_dtype dt, const GemmBatch& g, const char* name, hipStream_t s) {
  bool fits = (dt == MAP_BF16 || dt == MAP_F32) && g.count >= 1 && g.count <= 2;
  const int vec = dt == MAP_F32 ? 4 : 8;  // elements per 16-byte load
  for (int i = 0; fits && i < g.count; ++i) {
    const GemmProblem& p = g.p[i];
    fits = p.epi == EPI_ROPE && p.batch == 1 && p.N <= 128 && p.N % 2 == 0 && p.K % vec == 0 &&
           p.lda % vec == 0 && p.ldb % vec == 0 && (reinterpret_cast<uintptr_t>(p.A) & 15) == 0 &&
           (reinterpret_cast<uintptr_t>(p.B) & 15) == 0;
  }
  // With enough rows for a wave of 128 x 128 tiles, the tiled kernel reads
  // B once per tile instead of once per 32 rows.
  long long rows = 0;
  for (int i = 0; i < g.count; ++i) rows += g.p[i].M;
  if (!fits || rows >= 128LL * gemm_cus()) return launch_gemm(dt, g, name, s);
  GemmBatch q = g;
  int total = 0;
  for (int i = 0; i < q.count; ++i) {
    q.p[i].tiles_m = q.p[i].M > 0 ? kPG * ((q.p[i].M + kPR - 1) / kPR) : 0;
    total += q.p[i].tiles_m;
  }
  if (q.count == 1) q.p[1].tiles_m = 0;
  q.total_tiles = total;
  if (total == 0) return hipSuccess;
  if (dt == MAP_F32) return launch_kernel(name, proj_rope_kernel<float>, dim3(total), dim3(kPW * 64), 0, s, q);
  return launch_kernel(name, proj_rope_kernel<bf16_t>, dim3(total), dim3(kPW * 64), 0, s, q);
}

}  // namespace mapk
