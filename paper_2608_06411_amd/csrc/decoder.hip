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
//               blocks up to the diagonal through LDS with an online softmax;
//               the causal mask follows the rows' order in their sequence
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

// Workgroup (query block qb of 64 rows, head h, sequence b).  Thread
// (ti, tj) = (tid / 16, tid % 16) owns score rows 4 ti .. 4 ti + 3, columns
// 4 tj .. + 3, and output rows 4 ti .. + 3, dims 8 tj .. + 7; the 16 threads
// of a row group are 16 consecutive lanes.  LDS (dynamic): q and k
// transposed [128][68], v [64][132], p transposed [64][68], float32.
__global__ __launch_bounds__(NT) void attention_kernel(const DecoderArgs a) {
  extern __shared__ float lds[];
  float(*QT)[68] = reinterpret_cast<float(*)[68]>(lds);
  float(*KT)[68] = reinterpret_cast<float(*)[68]>(lds + 128 * 68);
  float(*Vs)[132] = reinterpret_cast<float(*)[132]>(lds + 2 * 128 * 68);
  float(*PT)[68] = reinterpret_cast<float(*)[68]>(lds + 2 * 128 * 68 + 64 * 132);
  const int qb = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int s0 = a.seq_off[b], S = a.seq_off[b + 1] - s0, q0 = qb * 64;
  if (q0 >= S) return;
  const int tid = threadIdx.x, ti = tid >> 4, tj = tid & 15;
  const long long ld = 3LL * a.d;
  const bf16_t* qkv = static_cast<const bf16_t*>(a.qkv);
  // the query block, transposed into LDS
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int e = tid + u * NT, r = e >> 4, c = (e & 15) * 8;
    Bf8 v;
    v.u = q0 + r < S ? *reinterpret_cast<const uint4*>(qkv + (s0 + q0 + r) * ld + h * DH + c)
                     : make_uint4(0u, 0u, 0u, 0u);
#pragma unroll
    for (int k = 0; k < 8; ++k) QT[c + k][r] = bf16_to_f32(v.e[k]);
  }
  const float scale = 1.0f / sqrtf(static_cast<float>(DH));
  float m[4], l[4], O[4][8];
#pragma unroll
  for (int x = 0; x < 4; ++x) {
    m[x] = -INFINITY;
    l[x] = 0.0f;
#pragma unroll
    for (int c = 0; c < 8; ++c) O[x][c] = 0.0f;
  }
  for (int kb = 0; kb <= qb; ++kb) {
    const int k0 = kb * 64;
    __syncthreads();  // the previous block's k, v and p are no longer read
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int e = tid + u * NT, r = e >> 4, c = (e & 15) * 8;
      const bool ok = k0 + r < S;
      Bf8 kv, vv;
      kv.u = ok ? *reinterpret_cast<const uint4*>(qkv + (s0 + k0 + r) * ld + a.d + h * DH + c)
                : make_uint4(0u, 0u, 0u, 0u);
      vv.u = ok ? *reinterpret_cast<const uint4*>(qkv + (s0 + k0 + r) * ld + 2 * a.d + h * DH + c)
                : make_uint4(0u, 0u, 0u, 0u);
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        KT[c + k][r] = bf16_to_f32(kv.e[k]);
        Vs[r][c + k] = bf16_to_f32(vv.e[k]);
      }
    }
    __syncthreads();
    float sc[4][4];
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
      for (int y = 0; y < 4; ++y) sc[x][y] = 0.0f;
#pragma unroll 4
    for (int dd = 0; dd < DH; ++dd) {
      const float4 qv = *reinterpret_cast<const float4*>(&QT[dd][4 * ti]);
      const float4 kv = *reinterpret_cast<const float4*>(&KT[dd][4 * tj]);
      const float qa[4] = {qv.x, qv.y, qv.z, qv.w}, ka[4] = {kv.x, kv.y, kv.z, kv.w};
#pragma unroll
      for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 4; ++y) sc[x][y] = fmaf(qa[x], ka[y], sc[x][y]);
    }
    // causal mask, online softmax over this block's keys
#pragma unroll
    for (int x = 0; x < 4; ++x) {
      const int qi = q0 + 4 * ti + x;
      float mx = -INFINITY;
#pragma unroll
      for (int y = 0; y < 4; ++y) {
        const int kj = k0 + 4 * tj + y;
        sc[x][y] = (kj <= qi && kj < S) ? sc[x][y] * scale : -INFINITY;
        mx = fmaxf(mx, sc[x][y]);
      }
#pragma unroll
      for (int off = 8; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off, 16));
      const float mn = fmaxf(m[x], mx);
      const float alpha = (mn == -INFINITY || m[x] == -INFINITY) ? (mn == -INFINITY ? 1.0f : 0.0f) : __expf(m[x] - mn);
      float rs = 0.0f;
#pragma unroll
      for (int y = 0; y < 4; ++y) {
        const float p = mn == -INFINITY ? 0.0f : __expf(sc[x][y] - mn);
        PT[4 * tj + y][4 * ti + x] = p;
        rs += p;
      }
#pragma unroll
      for (int off = 8; off > 0; off >>= 1) rs += __shfl_xor(rs, off, 16);
      l[x] = l[x] * alpha + rs;
      m[x] = mn;
#pragma unroll
      for (int c = 0; c < 8; ++c) O[x][c] *= alpha;
    }
    __syncthreads();
#pragma unroll 4
    for (int j = 0; j < 64; ++j) {
      const float4 pv = *reinterpret_cast<const float4*>(&PT[j][4 * ti]);
      const float4 v0 = *reinterpret_cast<const float4*>(&Vs[j][8 * tj]);
      const float4 v1 = *reinterpret_cast<const float4*>(&Vs[j][8 * tj + 4]);
      const float pa[4] = {pv.x, pv.y, pv.z, pv.w}, va[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
#pragma unroll
      for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int c = 0; c < 8; ++c) O[x][c] = fmaf(pa[x], va[c], O[x][c]);
    }
  }
  bf16_t* out = static_cast<bf16_t*>(a.o);
#pragma unroll
  for (int x = 0; x < 4; ++x) {
    const int row = q0 + 4 * ti + x;
    if (row >= S) continue;
    const float inv = 1.0f / l[x];
    Bf8 o;
#pragma unroll
    for (int c = 0; c < 8; ++c) o.e[c] = f32_to_bf16(O[x][c] * inv);
    *reinterpret_cast<uint4*>(out + (long long)(s0 + row) * a.d + h * DH + 8 * tj) = o.u;
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
  constexpr int bytes = sizeof(float) * (2 * 128 * 68 + 64 * 132 + 64 * 68);
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
