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
// one.  LDS rows are 8 chunks of 16 bytes, XOR-swizzled by (row & 7) so that
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

// Block index -> tile index such that the tiles run by one XCD are contiguous.
__device__ __forceinline__ int xcd_remap(int b, int total) {
  const int per = total / kXcds, rem = total % kXcds;
  const int x = b % kXcds, local = b / kXcds;
  return x * per + min(x, rem) + local;
}

__device__ __forceinline__ float gelu_erf(float x) {
  return 0.5f * x * (1.0f + erff(x * 0.70710678118654752f));
}

template <typename T>
__device__ __forceinline__ void mma_slice(const uint4 (*As)[8], const uint4 (*Bs)[8], int wm, int wn,
                                          int lane, f32x16_t (&acc)[2][2]);

template <>
__device__ __forceinline__ void mma_slice<bf16_t>(const uint4 (*As)[8], const uint4 (*Bs)[8], int wm,
                                                  int wn, int lane, f32x16_t (&acc)[2][2]) {
  const int lr = lane & 31, lh = lane >> 5;
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    const int v = 2 * s + lh;  // 16-byte chunk: k = 16 s + 8 lh + (0..7)
    bf16x8_t a[2], b[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int r = wm * 64 + i * 32 + lr;
      uint4 t = As[r][v ^ (r & 7)];
      a[i] = __builtin_bit_cast(bf16x8_t, t);
    }
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int r = wn * 64 + j * 32 + lr;
      uint4 t = Bs[r][v ^ (r & 7)];
      b[j] = __builtin_bit_cast(bf16x8_t, t);
    }
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
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
      a[i] = __builtin_bit_cast(float4, As[r][v ^ (r & 7)]);
    }
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int r = wn * 64 + j * 32 + lr;
      b[j] = __builtin_bit_cast(float4, Bs[r][v ^ (r & 7)]);
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

template <typename T>
__global__ __launch_bounds__(NT) void gemm_kernel(const GemmBatch args) {
  // One contiguous 64 KiB block: A slices in [0, 2), B slices in [2, 4); the
  // RoPE epilogue reuses all of it as a 128 x 128 float tile.
  __shared__ uint4 smem[4][BM][8];
  uint4 (*As)[BM][8] = smem;
  uint4 (*Bs)[BM][8] = smem + 2;
  constexpr int VEC = Slice<T>::VEC;
  constexpr int BK = Slice<T>::BK;

  const int tile = xcd_remap(blockIdx.x, args.total_tiles);
  int pi = 0;
#pragma unroll
  for (int q = 1; q < kMaxGemmProblems; ++q)
    if (q < args.count && tile >= args.p[q].tile_begin) pi = q;
  const GemmProblem& P = args.p[pi];

  const int local = tile - P.tile_begin;
  const int bt = local / P.tiles_per_batch;
  int tt = local - bt * P.tiles_per_batch;
  int tm, tn;
  if (P.triangular) {  // upper triangle, row by row: row tm holds tiles_n - tm tiles
    tm = 0;
    while (tt >= P.tiles_n - tm) { tt -= P.tiles_n - tm; ++tm; }
    tn = tm + tt;
  } else {
    tm = tt / P.tiles_n;
    tn = tt - tm * P.tiles_n;
  }
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
      As[buf][r][lv ^ (r & 7)] = ra[j];
      Bs[buf][r][lv ^ (r & 7)] = rb[j];
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

  // ------------------------------------------------------------ epilogues
  if (P.epi == EPI_BIAS_GELU || P.epi == EPI_BIAS) {
    T* __restrict__ C = static_cast<T*>(P.C) + bt * P.strideC;
    const T* __restrict__ bias = static_cast<const T*>(P.bias);
    const bool gelu = P.epi == EPI_BIAS_GELU;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int col = n0 + wn * 64 + j * 32 + acc_col(lane);
      if (col >= N) continue;
      const float bv = to_f32<T>(bias[col]);
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
  } else {  // EPI_ROPE: stage the tile in LDS so each thread sees both halves of a pair
    float* tileF = reinterpret_cast<float*>(&smem[0][0][0]);  // 128 x 128 floats = 64 KiB
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int rl = wm * 64 + i * 32 + acc_row(r, lane);
          const int cl = wn * 64 + j * 32 + acc_col(lane);
          tileF[rl * BN + cl] = acc[i][j][r];
        }
    __syncthreads();
    float* __restrict__ out = static_cast<float*>(P.C) + bt * P.strideC;
    const int half = N >> 1;
    for (int e = tid; e < BM * half; e += NT) {
      const int rl = e / half, c = e - rl * half;
      const int row = m0 + rl;
      if (row >= M) continue;
      const float a = tileF[rl * BN + c], b = tileF[rl * BN + c + half];
      const float2 cs = P.rope_cs[(long long)row * half + c];
      out[(long long)row * P.ldc + c] = a * cs.x - b * cs.y;
      out[(long long)row * P.ldc + c + half] = b * cs.x + a * cs.y;
    }
  }
}

}  // namespace

void gemm_finalize(GemmBatch& g) {
  int begin = 0;
  for (int i = 0; i < g.count; ++i) {
    GemmProblem& p = g.p[i];
    p.tiles_m = (p.M + BM - 1) / BM;
    p.tiles_n = (p.N + BN - 1) / BN;
    p.tiles_per_batch = p.triangular ? p.tiles_m * (p.tiles_m + 1) / 2 : p.tiles_m * p.tiles_n;
    p.tile_begin = begin;
    begin += p.tiles_per_batch * p.batch;
  }
  g.total_tiles = begin;
}

hipError_t launch_gemm(map_dtype dt, const GemmBatch& g, const char* name, hipStream_t s) {
  if (g.total_tiles == 0) return hipSuccess;
  if (dt == MAP_BF16) return launch_kernel(name, gemm_kernel<bf16_t>, dim3(g.total_tiles), dim3(NT), 0, s, g);
  return launch_kernel(name, gemm_kernel<float>, dim3(g.total_tiles), dim3(NT), 0, s, g);
}

}  // namespace mapk
