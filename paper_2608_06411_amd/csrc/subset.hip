// Candidate subset of map_prune: the tokens whose Eq. (4) scores can matter.
//
// A token's Eq. (4) score p n r never exceeds its bound p n: the unit
// residual r starts at 1 and only shrinks as the basis grows.  In the keys
// the selection compares (positive scores by (p n)^2 r^2, then zero scores
// by p, ties to the lower index) a token's key therefore never exceeds its
// bound key: 0x80000000 | bits((p n)^2) when that is a positive score (the
// float32 product r^2 (p n)^2 with r^2 <= 1 rounds to at most (p n)^2),
// else bits(p).
//
// For each image this kernel takes J = R0 (the K0 largest p, which the
// selection places first) plus the tokens with the largest bound keys, at
// most Nc tokens in ascending token order, padded to Nc with tokens of
// weight zero, and records hout, the largest bound key of a token left out.  A selection run on J then makes exactly
// the picks of the selection over all tokens if every greedy pick's key
// (its high word) exceeds hout: no token outside J could have beaten it.
// The selection checks that itself and flags the image otherwise, and the
// image is then selected again over all its tokens.
//
// One workgroup per image; each thread keeps its tokens' keys in registers
// as 46-bit integers (key high word << 14 | 16383 - index, which orders
// like the key for N <= 16384).  One 1024-bin histogram of each kind of key
// places the thresholds at bin edges: J holds whole bins.
#include "internal.h"

namespace mapk {

namespace {

constexpr int NT = 256;
constexpr int kBins = 1024;

__device__ __forceinline__ uint32_t sub_ordered_bits(float f) {
  return (f > 0.0f && f <= 3.402823466e38f) ? __float_as_uint(f) : 0u;
}

// The bound key's high word of a token with importance pv and norm nv.
__device__ __forceinline__ uint32_t bound_hi(float pv, float nv, float tau2) {
  const float pc = (pv > 0.0f && pv <= 3.402823466e38f) ? pv : 0.0f;
  const float qn = pc * nv;
  const float s2 = qn * qn;
  const bool positive = nv > 0.0f && 1.0f > tau2 && qn > 0.0f && s2 > 0.0f;
  return positive ? (0x80000000u | sub_ordered_bits(s2)) : sub_ordered_bits(pv);
}

struct BlockScratch {
  uint32_t red[2][NT / 64];
  int part[NT / 64];
  int sel[2];
  uint64_t key;
};

// wave64 maximum / minimum on the DPP network (row shifts, then row
// broadcasts; lanes a step does not reach keep the identity)
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ uint32_t dpp_max(uint32_t v) {
  const uint32_t o = __builtin_amdgcn_update_dpp(0u, v, CTRL, ROW_MASK, 0xf, false);
  return o > v ? o : v;
}
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ uint32_t dpp_min(uint32_t v) {
  const uint32_t o = __builtin_amdgcn_update_dpp(0xffffffffu, v, CTRL, ROW_MASK, 0xf, false);
  return o < v ? o : v;
}
__device__ __forceinline__ uint32_t wave_max32(uint32_t v) {
  v = dpp_max<0x111, 0xf>(v);
  v = dpp_max<0x112, 0xf>(v);
  v = dpp_max<0x114, 0xf>(v);
  v = dpp_max<0x118, 0xf>(v);
  v = dpp_max<0x142, 0xa>(v);
  v = dpp_max<0x143, 0xc>(v);
  return __builtin_amdgcn_readlane(v, 63);
}
__device__ __forceinline__ uint32_t wave_min32(uint32_t v) {
  v = dpp_min<0x111, 0xf>(v);
  v = dpp_min<0x112, 0xf>(v);
  v = dpp_min<0x114, 0xf>(v);
  v = dpp_min<0x118, 0xf>(v);
  v = dpp_min<0x142, 0xa>(v);
  v = dpp_min<0x143, 0xc>(v);
  return __builtin_amdgcn_readlane(v, 63);
}

// Workgroup maximum of mx and minimum of mn (one barrier pair).
__device__ void block_max_min32(uint32_t& mx, uint32_t& mn, BlockScratch& s) {
  mx = wave_max32(mx);
  mn = wave_min32(mn);
  if ((threadIdx.x & 63) == 0) {
    s.red[0][threadIdx.x >> 6] = mx;
    s.red[1][threadIdx.x >> 6] = mn;
  }
  __syncthreads();
  mx = s.red[0][0];
  mn = s.red[1][0];
  for (int w = 1; w < NT / 64; ++w) {
    mx = s.red[0][w] > mx ? s.red[0][w] : mx;
    mn = s.red[1][w] < mn ? s.red[1][w] : mn;
  }
  __syncthreads();
}

// Exclusive prefix sum over the workgroup's threads (thread order), and the total.
__device__ int block_exclusive_sum(int v, int& total, BlockScratch& s) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int x = v;
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) s.part[wave] = x;
  __syncthreads();
  int before = 0;
  total = 0;
  for (int w = 0; w < NT / 64; ++w) {
    before += w < wave ? s.part[w] : 0;
    total += s.part[w];
  }
  __syncthreads();
  return before + x - v;
}

// Keys per thread: token i = tid + NT u is kept in register slot u.
constexpr int kKpt = kSubsetMaxN / NT;

// One histogram of the keys (register slots u < nu) that lie in [lo, hi]
// over 1024 bins of equal width 2^sh; returns the lower edge of the highest
// bin at which the count from the top reaches `need` -- every key at or above
// it is taken, at least `need` of them -- when `atleast`, else the lowest
// edge above which at most `need` keys lie (fewer may).
__device__ uint64_t hist_edge(const uint64_t (&kr)[kKpt], int nu, int need, bool atleast, uint64_t lo,
                              uint64_t hi, int* hist, BlockScratch& s) {
  const int tid = threadIdx.x, lane = tid & 63;
  const uint64_t span = hi - lo;
  const int bits = span ? 64 - __builtin_clzll(span) : 0;
  const int sh = bits > 10 ? bits - 10 : 0;  // (span >> sh) < 1024
  for (int j = tid; j < kBins; j += NT) hist[j] = 0;
  __syncthreads();
#pragma unroll
  for (int u = 0; u < kKpt; ++u) {
    const uint64_t x = kr[u];
    if (u < nu && x >= lo && x <= hi) atomicAdd(&hist[static_cast<int>((x - lo) >> sh)], 1);
  }
  __syncthreads();
  if (tid < 64) {  // lane l: bins 16 l .. 16 l + 15
    int c[16], mine = 0;
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      c[q] = hist[16 * lane + q];
      mine += c[q];
    }
    int suf = mine;  // keys in bins 16 lane and above
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_down(suf, o);
      if (lane + o < 64) suf += y;
    }
    if (lane == 0) s.sel[1] = atleast ? 0 : -1;  // (not atleast and no bin overflows: every key fits)
    int cum = suf - mine;  // keys above bin 16 lane + 15
#pragma unroll
    for (int q = 15; q >= 0; --q) {
      const int bin = 16 * lane + q;
      if (atleast ? (cum < need && need <= cum + c[q]) : (cum <= need && cum + c[q] > need)) s.sel[1] = bin;
      cum += c[q];
    }
  }
  __syncthreads();
  // atleast: the bin where the count reaches need; else the bin that would
  // overflow it (the edge is the one above it)
  const int bin = s.sel[1];
  __syncthreads();
  return atleast ? lo + (static_cast<uint64_t>(bin) << sh) : lo + (static_cast<uint64_t>(bin + 1) << sh);
}

// LDS: p, the norms and their reciprocals [N] float each, then one
// membership byte per token.
__global__ __launch_bounds__(NT) void subset_kernel(const SubsetArgs a) {
  extern __shared__ __attribute__((aligned(16))) float pv[];
  __shared__ int hist[kBins];
  __shared__ BlockScratch s;
  const int b = blockIdx.x, N = a.N, Nc = a.Nc, K0 = a.K0, tid = threadIdx.x;
  float* nv = pv + N;
  float* iv = nv + N;
  unsigned char* member = reinterpret_cast<unsigned char*>(iv + N);
  const float* p = a.p + (long long)b * N;
  const float* nrm = a.norms + (long long)b * N;
  const float* ninv = a.ninv + (long long)b * N;
  const int nu = (N - tid + NT - 1) / NT;  // this thread's tokens: tid + NT u, u < nu
  // every load issued first, at clamped addresses
  float pr[kKpt], nr[kKpt], ir[kKpt];
#pragma unroll
  for (int u = 0; u < kKpt; ++u) {
    const int i = min(tid + NT * u, N - 1);
    pr[u] = p[i];
    nr[u] = nrm[i];
    ir[u] = ninv[i];
  }
  // R0 (the K0 largest p, ties to the lower index) is inside the tokens
  // whose p keys reach the histogram bin holding the K0-th largest
  uint64_t kr[kKpt];
  uint32_t mn = 0xffffffffu, mx = 0u;  // high words of the keys
#pragma unroll
  for (int u = 0; u < kKpt; ++u) {
    const int i = tid + NT * u;
    const uint32_t h = sub_ordered_bits(pr[u]);
    kr[u] = (static_cast<uint64_t>(h) << 14) | static_cast<uint64_t>(16383 - i);
    if (u < nu) {
      pv[i] = pr[u];
      nv[i] = nr[u];
      iv[i] = ir[u];
      mn = h < mn ? h : mn;
      mx = h > mx ? h : mx;
    }
  }
  block_max_min32(mx, mn, s);
  const uint64_t t0 = K0 > 0 ? hist_edge(kr, nu, K0, true, static_cast<uint64_t>(mn) << 14,
                                         (static_cast<uint64_t>(mx) << 14) | 16383u, hist, s)
                             : ~0ull;
  // the others by their bound keys (the R0 candidates' keys become 0)
  int nr0 = 0;
  mn = 0xffffffffu;
  mx = 0u;
#pragma unroll
  for (int u = 0; u < kKpt; ++u) {
    const int i = tid + NT * u;
    const bool r0 = kr[u] >= t0;
    const uint32_t h = bound_hi(pr[u], nr[u], a.tau2);
    kr[u] = r0 ? 0ull : ((static_cast<uint64_t>(h) << 14) | static_cast<uint64_t>(16383 - i));
    if (u < nu) {
      nr0 += r0 ? 1 : 0;
      if (!r0) {
        mn = h < mn ? h : mn;
        mx = h > mx ? h : mx;
      }
    }
  }
  int total_r0 = 0;
  (void)block_exclusive_sum(nr0, total_r0, s);
  block_max_min32(mx, mn, s);
  // the largest bound keys that still fit beside them (mn > mx: no token left)
  const int room = Nc - total_r0;
  const uint64_t t1 = (room > 0 && mn <= mx) ? hist_edge(kr, nu, room, false, static_cast<uint64_t>(mn) << 14,
                                                          (static_cast<uint64_t>(mx) << 14) | 16383u, hist, s)
                                             : ~0ull;
  // J = keys 0 (R0 candidates) and keys >= t1; hout = the largest bound key left out
  uint32_t hout = 0u, unused = 0u;
#pragma unroll
  for (int u = 0; u < kKpt; ++u) {
    if (u < nu) {
      const uint64_t x = kr[u];
      const bool in = x == 0ull || x >= t1;
      member[tid + NT * u] = in ? 1 : 0;
      const uint32_t h = static_cast<uint32_t>(x >> 14);
      if (!in) hout = h > hout ? h : hout;
    }
  }
  block_max_min32(hout, unused, s);  // (its barrier also publishes the membership bytes)
  // compaction in token order: thread t takes tokens t chunk .. (t + 1) chunk - 1
  const int chunk = (N + NT - 1) / NT, i0 = tid * chunk, i1 = min(N, i0 + chunk);
  int mine = 0;
  for (int i = i0; i < i1; ++i) mine += member[i];
  int total = 0;
  int o = block_exclusive_sum(mine, total, s);
  int32_t* jmap = a.jmap + (long long)b * Nc;
  float* pJ = a.pJ + (long long)b * Nc;
  float* nJ = a.nJ + (long long)b * Nc;
  float* ninvJ = a.ninvJ + (long long)b * Nc;
  for (int i = i0; i < i1 && o < Nc; ++i)
    if (member[i]) {
      jmap[o] = i;
      pJ[o] = pv[i];
      nJ[o] = nv[i];
      ninvJ[o] = iv[i];
      ++o;
    }
  // the positions past J: tokens of weight zero (p = 0, no norm), last in
  // index order, so they are never in R0 and never picked while a real
  // token is left; a pick of one fails the certificate
  for (int k = total + tid; k < Nc; k += NT) {
    jmap[k] = 0;
    pJ[k] = 0.0f;
    nJ[k] = 0.0f;
    ninvJ[k] = 0.0f;
  }
  if (tid == 0) {
    a.hout[b] = hout;
    // R0's candidates alone more than fill the subset (a wide histogram bin
    // of nearly equal p): J is cut short, and the image is selected in full
    a.uncert[b] = total > Nc ? 1 : 0;
    a.clear_bar[b] = 0u;
  }
}

}  // namespace

size_t subset_lds_bytes(int N) { return static_cast<size_t>(N) * (3 * sizeof(float) + 1); }

hipError_t launch_subset(const SubsetArgs& a, hipStream_t s) {
  const size_t bytes = subset_lds_bytes(a.N);
  if (bytes > 48 * 1024) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(subset_kernel),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(bytes));
    if (e != hipSuccess) return e;
  }
  return launch_kernel("subset", subset_kernel, dim3(a.B), dim3(NT), bytes, s, a);
}

}  // namespace mapk
