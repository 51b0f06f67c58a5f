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
//
// Folded weights: the second layer of f_V (f_T) and W_K (W_Q) compose to
// one linear map, W_K (W2 h + b2) = (W_K W2) h + W_K b2.  These blocks
// transpose W2 (64 x 64 tiles through LDS) for the GEMM that forms W_K W2,
// and form the folded bias W_K b2 (one wave per output, float32).
#include "internal.h"

namespace mapk {

namespace {

constexpr int kRowsPerBlock = 4;

template <typename T>
__global__ __launch_bounds__(256) void prep_kernel(const PrepArgs a, int norm_blocks, int table_blocks,
                                                   int tr_blocks) {
#pragma unroll
  for (int c = 0; c < 2; ++c)
    if (a.clear[c])
      for (long long i = blockIdx.x * 256ll + threadIdx.x; i < a.nclear[c]; i += 256ll * gridDim.x) a.clear[c][i] = 0ull;
  int bid = static_cast<int>(blockIdx.x) - norm_blocks - table_blocks;
  if (bid >= 0) {
    if (bid < tr_blocks) {  // transpose tile (ti, tj) of matrix s, 16-byte pieces both ways
      constexpr int VEC = 16 / sizeof(T), TW = 64;  // elements per piece, tile width
      __shared__ T tile[TW][TW + VEC];
      const int per = (a.tn + TW - 1) / TW, s = bid / (per * per), t = bid % (per * per);
      const int ti = t / per, tj = t % per;
      const T* src = static_cast<const T*>(a.tsrc[s]);
      T* dst = static_cast<T*>(a.tdst[s]);
      const bool whole = a.tn % VEC == 0;
      constexpr int PP = TW * (TW / VEC) / 256;  // pieces per thread (2 for bf16, 4 for float)
      if (whole) {  // every piece's load issued before the first LDS store
        uint4 pv[PP];
#pragma unroll
        for (int u = 0; u < PP; ++u) {
          const int e = threadIdx.x + 256 * u, r = e / (TW / VEC), c = VEC * (e % (TW / VEC));
          const int gr = min(TW * ti + r, a.tn - 1), gc = min(TW * tj + c, a.tn - VEC);
          pv[u] = *reinterpret_cast<const uint4*>(src + (long long)gr * a.tn + gc);
        }
#pragma unroll
        for (int u = 0; u < PP; ++u) {
          const int e = threadIdx.x + 256 * u, r = e / (TW / VEC), c = VEC * (e % (TW / VEC));
          if (TW * ti + r < a.tn && TW * tj + c + VEC <= a.tn) *reinterpret_cast<uint4*>(&tile[r][c]) = pv[u];
        }
      } else {
        for (int e = threadIdx.x; e < TW * (TW / VEC); e += 256) {  // row r, piece c of the source tile
          const int r = e / (TW / VEC), c = VEC * (e % (TW / VEC)), gr = TW * ti + r, gc = TW * tj + c;
          if (gr >= a.tn) continue;
          for (int k = 0; k < VEC && gc + k < a.tn; ++k) tile[r][c + k] = src[(long long)gr * a.tn + gc + k];
        }
      }
      __syncthreads();
      for (int e = threadIdx.x; e < TW * (TW / VEC); e += 256) {  // row r, piece c of the destination tile
        const int r = e / (TW / VEC), c = VEC * (e % (TW / VEC)), gr = TW * tj + r, gc = TW * ti + c;
        if (gr >= a.tn) continue;
        if (whole && gc + VEC <= a.tn) {
          uint32_t w[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) {  // 16 bytes packed from the column
            if constexpr (sizeof(T) == 4) {
              w[q] = __builtin_bit_cast(uint32_t, tile[c + q][r]);
            } else {
              w[q] = static_cast<uint32_t>(__builtin_bit_cast(uint16_t, tile[c + 2 * q][r])) |
                     (static_cast<uint32_t>(__builtin_bit_cast(uint16_t, tile[c + 2 * q + 1][r])) << 16);
            }
          }
          *reinterpret_cast<uint4*>(dst + (long long)gr * a.tn + gc) = make_uint4(w[0], w[1], w[2], w[3]);
        } else {
          for (int k = 0; k < VEC && gc + k < a.tn; ++k) dst[(long long)gr * a.tn + gc + k] = tile[c + k][r];
        }
      }
      return;
    }
    bid -= tr_blocks;  // folded bias: output o = 4 (block) + wave of matrix s
    const int per = (a.frows + 3) / 4, s = bid / per, o = 4 * (bid % per) + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (o >= a.frows) return;
    const T* wr = static_cast<const T*>(a.fw[s]) + (long long)o * a.fcols;
    const T* bv = static_cast<const T*>(a.fb[s]);
    float acc = 0.0f;
    constexpr int U = 8;  // loads in flight per lane
    for (int k0 = lane; k0 < a.fcols; k0 += 64 * U) {
      T x[U], y[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int k = min(k0 + 64 * u, a.fcols - 1);
        x[u] = wr[k];
        y[u] = bv[k];
      }
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (k0 + 64 * u < a.fcols) acc = fmaf(to_f32<T>(x[u]), to_f32<T>(y[u]), acc);
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
    if (lane == 0) a.fout[s][o] = acc;
    return;
  }
  if (static_cast<int>(blockIdx.x) < norm_blocks) {
    const int row = blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (row >= a.rowsV) return;
    constexpr int VEC = 16 / sizeof(T);
    const T* r = static_cast<const T*>(a.V) + (long long)row * a.D;
    float acc = 0.0f;
    constexpr int U = 8;  // 16-byte loads in flight per lane
    const int nchunk = a.D / VEC;
    for (int c0 = lane; c0 < nchunk; c0 += 64 * U) {
      uint4 uv[U];
#pragma unroll
      for (int u = 0; u < U; ++u) uv[u] = *reinterpret_cast<const uint4*>(r + min(c0 + 64 * u, nchunk - 1) * VEC);
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (c0 + 64 * u < nchunk) {
          const T* e = reinterpret_cast<const T*>(&uv[u]);
#pragma unroll
          for (int k = 0; k < VEC; ++k) {
            const float x = to_f32<T>(e[k]);
            acc = fmaf(x, x, acc);
          }
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

hipError_t launch_prep(map_dtype dt, const PrepArgs& a, bool norms, bool table, bool fold, hipStream_t s) {
  const int nb = norms ? (a.rowsV + kRowsPerBlock - 1) / kRowsPerBlock : 0;
  const long long entries = table ? (long long)(a.rowsV + a.rowsT) * a.half : 0;
  const int tb = static_cast<int>((entries + 255) / 256);
  const int per = (a.tn + 63) / 64;
  const int xb = fold ? 2 * per * per : 0;
  const int fb = fold ? 2 * ((a.frows + 3) / 4) : 0;
  const int total = nb + tb + xb + fb;
  if (total == 0) return hipSuccess;
  if (dt == MAP_BF16)
    return launch_kernel("prep", prep_kernel<bf16_t>, dim3(total), dim3(256), 0, s, a, nb, tb, xb);
  return launch_kernel("prep", prep_kernel<float>, dim3(total), dim3(256), 0, s, a, nb, tb, xb);
}

}  // namespace mapk
