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
// For each image this kernel takes J = R0's candidates (a superset of the K0
// largest p, which the selection places first) plus the tokens with the
// largest bound keys, at most Nc tokens in ascending token order, padded to
// Nc with tokens of weight zero, and records hout, the largest bound key's
// high word of a token left out.  A selection run on J then makes exactly
// the picks of the selection over all tokens if every greedy pick's key
// (its high word) exceeds hout: no token outside J could have beaten it.
// The selection checks that itself and flags the image otherwise, and the
// image is then selected again over all its tokens.
//
// One workgroup of 1024 threads per image; each thread keeps its tokens' key
// high words in registers.  One 1024-bin histogram of each kind of key places the
// thresholds at bin edges: J holds whole bins (ties included).
#include "internal.h"

namespace mapk {

namespace {

constexpr int NT = 1024;  // 16 waves: a few tokens per thread (2.4 us faster per call than 256 threads at N = 2880)
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

// Inclusive prefix sum over the lanes of a wave64 (row shifts within each
// row of 16 lanes, then the row broadcasts).
template <int CTRL, int ROW_MASK, int BANK_MASK, bool BOUND>
__device__ __forceinline__ int dpp_add(int v) {
  return v + __builtin_amdgcn_update_dpp(0, v, CTRL, ROW_MASK, BANK_MASK, BOUND);
}
__device__ __forceinline__ int wave_inclusive_sum(int v) {
  v = dpp_add<0x111, 0xf, 0xf, true>(v);   // row_shr:1
  v = dpp_add<0x112, 0xf, 0xf, true>(v);   // row_shr:2
  v = dpp_add<0x114, 0xf, 0xf, true>(v);   // row_shr:4
  v = dpp_add<0x118, 0xf, 0xf, true>(v);   // row_shr:8: each row scanned
  v = dpp_add<0x142, 0xa, 0xf, false>(v);  // row_bcast:15 into rows 1 and 3
  v = dpp_add<0x143, 0xc, 0xf, false>(v);  // row_bcast:31 into rows 2 and 3
  return v;
}

// Exclusive prefix sum over the workgroup's threads (thread order), and the total.
__device__ int block_exclusive_sum(int v, int& total, BlockScratch& s) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int x = wave_inclusive_sum(v);
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

// Most register slots of one thread: token i = tid + NT u sits in slot u.
constexpr int kKpt = kSubsetMaxN / NT;

// One histogram of the keys over 1024 bins of equal width: the keys of the
// valid register slots (u < nu) whose high words lie in [mn, mx], binned by
// high word ((h - mn) >> sh, sh chosen so that the bins cover the range).
// Returns the lowest high word of the bin at which the count from the top
// reaches `need` (every key of that bin and above is taken, at least `need`
// of them) when `atleast`; else the lowest high word above which at most
// `need` keys lie (fewer may): the bin that would overflow is left out.
template <int KPT>
__device__ uint64_t hist_edge(const uint32_t (&hr)[KPT], uint32_t valid, int need, bool atleast, uint32_t mn,
                              uint32_t mx, int* hist, BlockScratch& s) {
  const int tid = threadIdx.x, lane = tid & 63;
  const uint32_t span = mx - mn;
  const int bits = span ? 32 - __builtin_clz(span) : 0;
  const int sh = bits > 10 ? bits - 10 : 0;  // (span >> sh) < 1024
  for (int j = tid; j < kBins; j += NT) hist[j] = 0;
  __syncthreads();
#pragma unroll
  for (int u = 0; u < KPT; ++u)
    if ((valid >> u) & 1u) atomicAdd(&hist[(hr[u] - mn) >> sh], 1);
  __syncthreads();
  if (tid < 64) {  // lane l: bins 16 (63 - l) .. + 15, so the lane prefix sums count from the top
    const int base = 16 * (63 - lane);
    int c[16], mine = 0;
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      c[q] = hist[base + q];
      mine += c[q];
    }
    if (lane == 0) s.sel[1] = atleast ? 0 : -1;  // (not atleast and no bin overflows: every key fits)
    int cum = wave_inclusive_sum(mine) - mine;  // keys above bin base + 15
#pragma unroll
    for (int q = 15; q >= 0; --q) {
      if (atleast ? (cum < need && need <= cum + c[q]) : (cum <= need && cum + c[q] > need)) s.sel[1] = base + q;
      cum += c[q];
    }
  }
  __syncthreads();
  const int bin = s.sel[1];
  __syncthreads();
  return static_cast<uint64_t>(mn) + (static_cast<uint64_t>(atleast ? bin : bin + 1) << sh);
}

// LDS: p, the norms and their reciprocals [N] float each, then one
// membership byte per token.  KPT >= ceil(N / NT) register slots per thread.
template <int KPT>
__global__ __launch_bounds__(NT) void subset_kernel(const SubsetArgs a) {
  extern __shared__ __attribute__((aligned(16))) float pv[];
  __shared__ int hist[kBins];
  __shared__ BlockScratch s;
  const int b = blockIdx.x, N = a.N, Nc = a.Nc, K0 = a.K0, tid = threadIdx.x;
  if (a.run_if && a.run_if[b] == 0) {  // (certified by the first subset)
    if (tid == 0) a.uncert[b] = 0;
    return;
  }
  float* nv = pv + N;
  float* iv = nv + N;
  unsigned char* member = reinterpret_cast<unsigned char*>(iv + N);
  const float* p = a.p + (long long)b * N;
  const float* nrm = a.norms + (long long)b * N;
  const float* ninv = a.ninv + (long long)b * N;
  // this thread's tokens: tid + NT u for the slots u set in `valid`; every
  // load issued first, at clamped addresses
  uint32_t valid = 0u;
  float pr[KPT], nr[KPT], ir[KPT];
#pragma unroll
  for (int u = 0; u < KPT; ++u) {
    const int i = tid + NT * u;
    valid |= i < N ? 1u << u : 0u;
    pr[u] = p[min(i, N - 1)];
    nr[u] = nrm[min(i, N - 1)];
    ir[u] = ninv[min(i, N - 1)];
  }
  // R0 (the K0 largest p, ties to the lower index) lies inside the tokens
  // whose p reaches the histogram bin holding the K0-th largest (ranked by
  // the keys' high words, bits(p): ties in p all fall in one bin)
  uint32_t hr[KPT];
  uint32_t mn = 0xffffffffu, mx = 0u;
#pragma unroll
  for (int u = 0; u < KPT; ++u) {
    const int i = tid + NT * u;
    hr[u] = sub_ordered_bits(pr[u]);
    if ((valid >> u) & 1u) {
      pv[i] = pr[u];
      nv[i] = nr[u];
      iv[i] = ir[u];
      mn = hr[u] < mn ? hr[u] : mn;
      mx = hr[u] > mx ? hr[u] : mx;
    }
  }
  block_max_min32(mx, mn, s);
  // R0's candidates: the p high words at or above the bin edge (all of them
  // when K0 = 0 is not the case; none when K0 = 0)
  const uint64_t e0 = K0 > 0 ? hist_edge<KPT>(hr, valid, K0, true, mn, mx, hist, s) : 0u;
  uint32_t r0m = 0u;  // slots holding R0 candidates
  int nr0 = 0;
#pragma unroll
  for (int u = 0; u < KPT; ++u)
    if (K0 > 0 && ((valid >> u) & 1u) && hr[u] >= e0) {
      r0m |= 1u << u;
      ++nr0;
    }
  // the others by their bound keys' high words
  mn = 0xffffffffu;
  mx = 0u;
#pragma unroll
  for (int u = 0; u < KPT; ++u) {
    hr[u] = bound_hi(pr[u], nr[u], a.tau2);
    if (((valid & ~r0m) >> u) & 1u) {
      mn = hr[u] < mn ? hr[u] : mn;
      mx = hr[u] > mx ? hr[u] : mx;
    }
  }
  int total_r0 = 0;
  (void)block_exclusive_sum(nr0, total_r0, s);
  block_max_min32(mx, mn, s);
  // the largest bounds that still fit beside them (mn > mx: no token left)
  const int room = Nc - total_r0;
  const uint64_t e1 = (room > 0 && mn <= mx) ? hist_edge<KPT>(hr, valid & ~r0m, room, false, mn, mx, hist, s)
                                             : 0x100000000ull;
  // J = R0's candidates and the bounds at or above e1 (above every high word: none)
  const bool none = e1 > mx;
  uint32_t hout = 0u, unused = 0u;
#pragma unroll
  for (int u = 0; u < KPT; ++u) {
    if ((valid >> u) & 1u) {
      const bool in = ((r0m >> u) & 1u) || (!none && hr[u] >= e1);
      member[tid + NT * u] = in ? 1 : 0;
      if (!in) hout = hr[u] > hout ? hr[u] : hout;
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
    a.clear_r0flag[b] = 0;
  }
}

}  // namespace

size_t subset_lds_bytes(int N) { return static_cast<size_t>(N) * (3 * sizeof(float) + 1); }

template <int KPT>
hipError_t launch_subset_kpt(const SubsetArgs& a, hipStream_t s) {
  const size_t bytes = subset_lds_bytes(a.N);
  if (bytes > 48 * 1024) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(subset_kernel<KPT>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(bytes));
    if (e != hipSuccess) return e;
  }
  return launch_kernel(a.tier2 ? "subset_t2" : "subset", subset_kernel<KPT>, dim3(a.B), dim3(NT), bytes, s, a);
}

hipError_t launch_subset(const SubsetArgs& a, hipStream_t s) {
  const int kpt = (a.N + NT - 1) / NT;
  if (a.N < 1 || kpt > kKpt) return hipErrorInvalidValue;
  if (kpt <= 4) return launch_subset_kpt<4>(a, s);
  if (kpt <= 8) return launch_subset_kpt<8>(a, s);
  if (kpt <= 12) return launch_subset_kpt<12>(a, s);
  if (kpt <= 16) return launch_subset_kpt<16>(a, s);
  if (kpt <= 24) return launch_subset_kpt<24>(a, s);
  return launch_subset_kpt<32>(a, s);
}

}  // namespace mapk
