// The language model's first layer over the pruned input (section
// "Inference-Time Token Pruning": after pruning, the model processes only
// the K kept visual tokens and the question tokens, which is where the
// prefill speedup comes from).  The layer is LLaMA's, in bf16 with float32
// arithmetic:
//
//   h = RMSNorm(x) g_attn;  qkv = h W_qkv^T;  RoPE on q and k per head;
//   o = causal softmax(q k^T / sqrt(d_h)) v;  x1 = x + o W_o^T;
//   y = x1 + (SiLU(h2 W_g^T) * (h2 W_u^T)) W_d^T,  h2 = RMSNorm(x1) g_ffn.
//
// The four products run on the matrix-core GEMM (gemm.hip); this file holds
// the kernels between them:
//   rmsnorm     one workgroup per row, 16-byte pieces, float32 sum of squares
//   rope_qkv    rotates q and k in place, angles pos * theta^(-2i/d_h) in float64
//   attention   one workgroup per (64 query rows, head, sequence): the key
//               blocks up to the diagonal through LDS on the bf16 matrix
//               cores with an online softmax; the causal mask follows the
//               rows' order in their sequence
//   silu_mul    SiLU(gate) * up, 8 entries per thread
#include "internal.h"

namespace mapk {

namespace {

constexpr int NT = 256;
constexpr int DH = 128;  // head width (the 7B models' 4096 / 32)

union Bf8 {
  uint4 u;
  bf16_t e[8];
};

__device__ __forceinline__ float block_sum256(float v, float* red) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  const float r = (red[0] + red[1]) + (red[2] + red[3]);
  __syncthreads();
  return r;
}

// out[r] = x[r] / sqrt(mean(x[r]^2) + eps) * g, rows of d bf16 (d % 8 == 0,
// d <= 8192: each thread holds up to four 16-byte pieces of its row).
__global__ __launch_bounds__(NT) void rmsnorm_kernel(const bf16_t* __restrict__ x, const bf16_t* __restrict__ g,
                                                     bf16_t* __restrict__ out, int d, float eps) {
  __shared__ float red[4];
  const int r = blockIdx.x, pieces = d >> 3;
  const uint4* src = reinterpret_cast<const uint4*>(x + (long long)r * d);
  Bf8 v[4];
  float ss = 0.0f;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int c = threadIdx.x + u * NT;
    v[u].u = c < pieces ? src[c] : make_uint4(0u, 0u, 0u, 0u);
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const float f = bf16_to_f32(v[u].e[k]);
      ss = fmaf(f, f, ss);
    }
  }
  const float inv = 1.0f / sqrtf(block_sum256(ss, red) / static_cast<float>(d) + eps);
  const uint4* gp = reinterpret_cast<const uint4*>(g);
  uint4* dst = reinterpret_cast<uint4*>(out + (long long)r * d);
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int c = threadIdx.x + u * NT;
    if (c >= pieces) continue;
    Bf8 w, o;
    w.u = gp[c];
#pragma unroll
    for (int k = 0; k < 8; ++k) o.e[k] = f32_to_bf16(bf16_to_f32(v[u].e[k]) * inv * bf16_to_f32(w.e[k]));
    dst[c] = o.u;
  }
}

// Row r: pair i (i, i + 64) of every head of q and of k turned by the angle
// pos[r] theta^(-2i/128): (a, b) -> (a cos - b sin, b cos + a sin).
__global__ __launch_bounds__(NT) void rope_qkv_kernel(const DecoderArgs a) {
  const int r = blockIdx.x, i = threadIdx.x & 63, hg = threadIdx.x >> 6;
  double sn, cs;
  sincos(static_cast<double>(a.pos[r]) * a.inv_freq[i], &sn, &cs);
  const float c = static_cast<float>(cs), s = static_cast<float>(sn);
  bf16_t* row = static_cast<bf16_t*>(a.qkv) + (long long)r * 3 * a.d;
  for (int h = hg; h < 2 * a.n_heads; h += 4) {  // q heads, then k heads
    bf16_t* p = row + h * DH;
    const float x = bf16_to_f32(p[i]), y = bf16_to_f32(p[i + DH / 2]);
    p[i] = f32_to_bf16(x * c - y * s);
    p[i + DH / 2] = f32_to_bf16(y * c + x * s);
  }
}

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(16))) float f32x16_t;

// Row and column of accumulator register r of lane `lane` in a 32 x 32
// matrix-core block.
__device__ __forceinline__ int acc_row(int r, int lane) { return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3); }

// LDS strides of the attention tiles (bf16 entries; float32 for the scores).
constexpr int LQ = DH + 8;   // q and k rows: [64][LQ]
constexpr int LV = 64 + 8;   // v transposed (dims x keys) and p (queries x keys)
constexpr int LS = 64 + 4;   // scores [64][LS] float32
constexpr int kAttnLds = 2 * (2 * 64 * LQ + DH * LV + 64 * LV) + 4 * (64 * LS + 3 * 64);  // q, k, v^T, p; s, stats

// Workgroup (query block qb of 64 rows, head h, sequence b), flash-style on
// the bf16 matrix cores (32 x 32 x 16, float32 accumulation).  For each key
// block up to the diagonal: wave w forms the 32 x 32 score tile (rows
// 32 (w / 2), keys 32 (w % 2)) and stores it, scaled and masked, to LDS;
// four threads per row then take the row's maximum and sum over the block
// (two quad exchanges) and write p (bf16) and the running statistics; wave
// w rescales its output tiles (rows 32 (w / 2), dims 64 (w % 2) + 0 and
// + 32) and adds p v.
__global__ __launch_bounds__(NT) void attention_kernel(const DecoderArgs a) {
  extern __shared__ uint4 lds4[];
  bf16_t* Qs = reinterpret_cast<bf16_t*>(lds4);
  bf16_t* Ks = Qs + 64 * LQ;
  bf16_t* VT = Ks + 64 * LQ;
  bf16_t* Ps = VT + DH * LV;
  float* Ss = reinterpret_cast<float*>(Ps + 64 * LV);  // [64][LS]
  float* mrow = Ss + 64 * LS;                           // [64] running maximum
  float* lrow = mrow + 64;                              // [64] running sum
  float* alph = lrow + 64;                              // [64] this block's rescaling
  const int qb = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int s0 = a.seq_off[b], S = a.seq_off[b + 1] - s0, q0 = qb * 64;
  if (q0 >= S) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, wi = wave >> 1, wj = wave & 1;
  const int lr = lane & 31, lh = lane >> 5;
  const long long ld = 3LL * a.d;
  const bf16_t* qkv = static_cast<const bf16_t*>(a.qkv);
#pragma unroll
  for (int u = 0; u < 4; ++u) {  // the query block, row-major
    const int e = tid + u * NT, r = e >> 4, c = (e & 15) * 8;
    *reinterpret_cast<uint4*>(Qs + r * LQ + c) =
        q0 + r < S ? *reinterpret_cast<const uint4*>(qkv + (s0 + q0 + r) * ld + h * DH + c) : make_uint4(0u, 0u, 0u, 0u);
  }
  if (tid < 64) {
    mrow[tid] = -INFINITY;
    lrow[tid] = 0.0f;
  }
  const float scale = 1.0f / sqrtf(static_cast<float>(DH));
  f32x16_t o[2];
#pragma unroll
  for (int jj = 0; jj < 2; ++jj)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[jj][r] = 0.0f;
  const int srow = tid >> 2, sq = tid & 3;  // the row phase: row, quarter of its 64 keys
  for (int kb = 0; kb <= qb; ++kb) {
    const int k0 = kb * 64;
    __syncthreads();  // the previous block's k, v and p are no longer read
    // keys row-major (16 rows x 16 pieces per pass); values transposed, a
    // lane per pair of key rows so that each LDS store is one 32-bit word
    uint4 kv[4], va[2], vb[2];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int e = tid + u * NT, r = e >> 4, c = (e & 15) * 8;
      kv[u] = k0 + r < S ? *reinterpret_cast<const uint4*>(qkv + (s0 + k0 + r) * ld + a.d + h * DH + c)
                         : make_uint4(0u, 0u, 0u, 0u);
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int e = tid + u * NT, j = e & 31, c = (e >> 5) * 8, r = 2 * j;
      va[u] = k0 + r < S ? *reinterpret_cast<const uint4*>(qkv + (s0 + k0 + r) * ld + 2 * a.d + h * DH + c)
                         : make_uint4(0u, 0u, 0u, 0u);
      vb[u] = k0 + r + 1 < S ? *reinterpret_cast<const uint4*>(qkv + (s0 + k0 + r + 1) * ld + 2 * a.d + h * DH + c)
                             : make_uint4(0u, 0u, 0u, 0u);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int e = tid + u * NT, r = e >> 4, c = (e & 15) * 8;
      *reinterpret_cast<uint4*>(Ks + r * LQ + c) = kv[u];
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int e = tid + u * NT, j = e & 31, c = (e >> 5) * 8;
      Bf8 x, y;
      x.u = va[u];
      y.u = vb[u];
#pragma unroll
      for (int k = 0; k < 8; ++k)
        *reinterpret_cast<uint32_t*>(VT + (c + k) * LV + 2 * j) =
            static_cast<uint32_t>(x.e[k]) | (static_cast<uint32_t>(y.e[k]) << 16);
    }
    __syncthreads();
    // the score tile: rows 32 wi + lr (queries), columns 32 wj + lr (keys)
    f32x16_t sc;
#pragma unroll
    for (int r = 0; r < 16; ++r) sc[r] = 0.0f;
#pragma unroll
    for (int st = 0; st < DH / 16; ++st) {
      const bf16x8_t qa = *reinterpret_cast<const bf16x8_t*>(Qs + (32 * wi + lr) * LQ + 16 * st + 8 * lh);
      const bf16x8_t kk = *reinterpret_cast<const bf16x8_t*>(Ks + (32 * wj + lr) * LQ + 16 * st + 8 * lh);
      sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qa, kk, sc, 0, 0, 0);
    }
    {
      const int col = 32 * wj + lr, kj = k0 + col;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = 32 * wi + acc_row(r, lane);
        Ss[row * LS + col] = (kj <= q0 + row && kj < S) ? sc[r] * scale : -INFINITY;
      }
    }
    __syncthreads();
    {  // row srow, keys 16 sq .. 16 sq + 15
      float v[16];
#pragma unroll
      for (int k = 0; k < 16; k += 4) {
        const float4 x = *reinterpret_cast<const float4*>(Ss + srow * LS + 16 * sq + k);
        v[k] = x.x;
        v[k + 1] = x.y;
        v[k + 2] = x.z;
        v[k + 3] = x.w;
      }
      float mx = v[0];
#pragma unroll
      for (int k = 1; k < 16; ++k) mx = fmaxf(mx, v[k]);
      mx = fmaxf(mx, __shfl_xor(mx, 1, 4));
      mx = fmaxf(mx, __shfl_xor(mx, 2, 4));
      const float mo = mrow[srow], mn = fmaxf(mo, mx);
      float sum = 0.0f;
      Bf8 p0, p1;
#pragma unroll
      for (int k = 0; k < 16; ++k) {
        const float pv = mn == -INFINITY ? 0.0f : __expf(v[k] - mn);
        sum += pv;
        if (k < 8) p0.e[k] = f32_to_bf16(pv);
        else p1.e[k - 8] = f32_to_bf16(pv);
      }
      *reinterpret_cast<uint4*>(Ps + srow * LV + 16 * sq) = p0.u;
      *reinterpret_cast<uint4*>(Ps + srow * LV + 16 * sq + 8) = p1.u;
      sum += __shfl_xor(sum, 1, 4);
      sum += __shfl_xor(sum, 2, 4);
      __syncthreads();  // every quarter has read mrow before it changes
      if (sq == 0) {
        const float al = mn == -INFINITY ? 1.0f : (mo == -INFINITY ? 0.0f : __expf(mo - mn));
        lrow[srow] = lrow[srow] * al + sum;
        mrow[srow] = mn;
        alph[srow] = al;
      }
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const float al = alph[32 * wi + acc_row(r, lane)];
      o[0][r] *= al;
      o[1][r] *= al;
    }
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      const bf16x8_t pa = *reinterpret_cast<const bf16x8_t*>(Ps + (32 * wi + lr) * LV + 16 * st + 8 * lh);
#pragma unroll
      for (int jj = 0; jj < 2; ++jj) {
        const bf16x8_t vb2 = *reinterpret_cast<const bf16x8_t*>(VT + (64 * wj + 32 * jj + lr) * LV + 16 * st + 8 * lh);
        o[jj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(pa, vb2, o[jj], 0, 0, 0);
      }
    }
  }
  __syncthreads();
  bf16_t* out = static_cast<bf16_t*>(a.o);
#pragma unroll
  for (int jj = 0; jj < 2; ++jj)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = 32 * wi + acc_row(r, lane);
      if (q0 + row < S)
        out[(long long)(s0 + q0 + row) * a.d + h * DH + 64 * wj + 32 * jj + lr] = f32_to_bf16(o[jj][r] / lrow[row]);
    }
}

// act[r][i] = SiLU(gu[r][i]) * gu[r][ff + i], 8 entries per thread.
__global__ __launch_bounds__(NT) void silu_mul_kernel(const DecoderArgs a) {
  const long long e = (long long)blockIdx.x * NT + threadIdx.x, per = a.ff >> 3;
  if (e >= (long long)a.R * per) return;
  const long long r = e / per, p = e - r * per;
  const bf16_t* gu = static_cast<const bf16_t*>(a.gu) + r * 2 * a.ff;
  Bf8 g, u, o;
  g.u = reinterpret_cast<const uint4*>(gu)[p];
  u.u = reinterpret_cast<const uint4*>(gu + a.ff)[p];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const float x = bf16_to_f32(g.e[k]);
    o.e[k] = f32_to_bf16(x / (1.0f + __expf(-x)) * bf16_to_f32(u.e[k]));
  }
  reinterpret_cast<uint4*>(static_cast<bf16_t*>(a.act) + r * a.ff)[p] = o.u;
}

}  // namespace

hipError_t launch_rmsnorm(const DecoderArgs& a, const void* x, const void* g, void* out, hipStream_t s) {
  return launch_kernel("rmsnorm", rmsnorm_kernel, dim3(a.R), dim3(NT), 0, s, static_cast<const bf16_t*>(x),
                       static_cast<const bf16_t*>(g), static_cast<bf16_t*>(out), a.d, a.eps);
}

hipError_t launch_rope_qkv(const DecoderArgs& a, hipStream_t s) {
  return launch_kernel("rope_qkv", rope_qkv_kernel, dim3(a.R), dim3(NT), 0, s, a);
}

hipError_t launch_attention(const DecoderArgs& a, hipStream_t s) {
  constexpr int bytes = kAttnLds;
  const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(attention_kernel),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  if (e != hipSuccess) return e;
  return launch_kernel("attention", attention_kernel, dim3((a.max_len + 63) / 64, a.n_heads, a.B), dim3(NT), bytes,
                       s, a);
}

hipError_t launch_silu_mul(const DecoderArgs& a, hipStream_t s) {
  const long long n = (long long)a.R * (a.ff >> 3);
  return launch_kernel("silu_mul", silu_mul_kernel, dim3(static_cast<unsigned>((n + NT - 1) / NT)), dim3(NT), 0, s, a);
}

}  // namespace mapk
