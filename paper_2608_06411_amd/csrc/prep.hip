// Row norms of the visual tokens and the RoPE cos/sin table.
//
// Norms: one wave64 per row; each lane streams 16-byte chunks of the row
// (64 lanes cover 1 KiB per step, fully coalesced), squares in float32 and
// the wave reduces with cross-lane shuffles.  The reciprocal norm (0 for a
// zero row) scales the Gram matrix into cosine similarity in the GEMM
// epilogue, so no normalised copy of V is ever written.
//
// RoPE table: one thread per (token, pair): angle = pos * theta^(-2i/d_p)
// formed and reduced in float64 (positions reach several thousand, where a
// float32 angle would be off by ~1e-4 rad), then rounded to float32.
#include "internal.h"

namespace mapk {

namespace {

constexpr int kRowsPerBlock = 4;

template <typename T>
__global__ __launch_bounds__(256) void prep_kernel(const PrepArgs a, int norm_blocks) {
  if (static_cast<int>(blockIdx.x) < norm_blocks) {
    const int row = blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (row >= a.rowsV) return;
    constexpr int VEC = 16 / sizeof(T);
    const T* r = static_cast<const T*>(a.V) + (long long)row * a.D;
    float acc = 0.0f;
    for (int c = lane; c < a.D / VEC; c += 64) {
      const uint4 u = *reinterpret_cast<const uint4*>(r + c * VEC);
      const T* e = reinterpret_cast<const T*>(&u);
#pragma unroll
      for (int k = 0; k < VEC; ++k) {
        const float x = to_f32<T>(e[k]);
        acc = fmaf(x, x, acc);
      }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
    if (lane == 0) {
      const float n = sqrtf(acc);
      a.norms[row] = n;
      a.ninv[row] = n > 0.0f ? 1.0f / n : 0.0f;
    }
    return;
  }
  const long long e = (long long)(blockIdx.x - norm_blocks) * blockDim.x + threadIdx.x;
  const long long total = (long long)(a.rowsV + a.rowsT) * a.half;
  if (e >= total) return;
  const int row = static_cast<int>(e / a.half), i = static_cast<int>(e % a.half);
  const bool vis = row < a.rowsV;
  const int pos = vis ? a.pos_v[row] : a.pos_t[row - a.rowsV];
  double s, c;
  sincos(static_cast<double>(pos) * a.inv_freq[i], &s, &c);
  float2* dst = vis ? a.cs_v + (long long)row * a.half : a.cs_t + (long long)(row - a.rowsV) * a.half;
  dst[i] = make_float2(static_cast<float>(c), static_cast<float>(s));
}

}  // namespace

hipError_t launch_prep(map_dtype dt, const PrepArgs& a, bool norms, bool table, hipStream_t s) {
  const int nb = norms ? (a.rowsV + kRowsPerBlock - 1) / kRowsPerBlock : 0;
  const long long entries = table ? (long long)(a.rowsV + a.rowsT) * a.half : 0;
  const int tb = static_cast<int>((entries + 255) / 256);
  if (nb + tb == 0) return hipSuccess;
  if (dt == MAP_BF16) return launch_kernel("prep", prep_kernel<bf16_t>, dim3(nb + tb), dim3(256), 0, s, a, nb);
  return launch_kernel("prep", prep_kernel<float>, dim3(nb + tb), dim3(256), 0, s, a, nb);
}

}  // namespace mapk
