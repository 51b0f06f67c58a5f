// Diversity-aware selection (section "Inference-Time Token Pruning", Eq. (4)).
//
// The residual of Eq. (4) is evaluated from the cosine similarity S and the
// row norms n: with v^_i = v_i / n_i, b_t the orthonormal basis in pick order
// and c_{t,i} = <b_t, v^_i>,
//     c_{t,i} = (S[i_t][i] - sum_{l<t} c_{l,i_t} c_{l,i}) / r_{i_t},
//     r_i^2   = 1 - sum_t c_{t,i}^2,
//     ||v_i - B B^T v_i|| = n_i r_i,
// so the score p_i ||v_i - B B^T v_i|| is p_i n_i r_i.  A pick whose r_i is
// at most tau adds no basis vector (its row of C is zero).
//
// One persistent launch runs the whole selection of every image.  An image
// is served by G workgroups; workgroup w owns `ch` consecutive tokens (their
// r^2 and their columns of C, kept token-major in global memory).  Work
// proceeds in rounds separated by one barrier across the image's workgroups:
//
//   pool     Every workgroup builds the same candidate pool and replays the
//            round's picks on it, redundantly and deterministically, so no
//            second barrier is needed to agree on them.  The first rounds
//            place R0 (forced picks in descending p).  Afterwards the pool is
//            the top of the keys the workgroups published in the previous
//            round, and the greedy rule runs on it while the best pool key
//            exceeds beta, an upper bound of every key outside the pool.
//            Scores never increase as the basis grows, so a pool key above
//            beta is the true argmax over all candidates: the picks are
//            exactly those of the step-by-step rule.  The pool keeps its
//            residual Gram matrix Rm = S - C^T C in LDS; one wave makes the
//            round's picks, each a wave-wide argmax and one dot product per
//            member against this round's coefficients, with no barrier.
//   update   Every workgroup applies the round's new basis rows to its own
//            tokens (a dense product over the rows of earlier rounds, then a
//            right-looking triangular solve over this round's rows), updates
//            their keys and publishes its top kPub keys plus its (kPub+1)-th
//            key as a bound.
//
// Keys order candidates as the rule does: positive scores first (by score),
// then zero scores by p, ties to the lower index; selected tokens key 0.
#include <atomic>

#include "internal.h"

namespace mapk {

namespace {

constexpr int NT = 256;
constexpr unsigned kSpinLimit = 1u << 22;
constexpr int kMaxPool = 64;  // one pool member per lane of the picking wave

typedef __attribute__((ext_vector_type(16))) float f32x16_t;

__device__ __forceinline__ uint32_t ordered_bits(float f) {
  // non-negative finite floats order like their bits; everything else -> 0
  return (f > 0.0f && f <= 3.402823466e38f) ? __float_as_uint(f) : 0u;
}

// A positive Eq. (4) score p n r is keyed by its square (qn)^2 r^2, which
// orders the same way and needs no square root per candidate.
__device__ __forceinline__ uint64_t make_key(float r2, float qn, float p, int i, float tau2) {
  uint32_t hi = ordered_bits(p);
  if (r2 > tau2 && qn > 0.0f) {
    const float s2 = qn * qn * r2;
    if (s2 > 0.0f) hi = 0x80000000u | ordered_bits(s2);
  }
  return (static_cast<uint64_t>(hi) << 32) | (0xffffffffu - static_cast<uint32_t>(i));
}

__device__ __forceinline__ int key_index(uint64_t k) {
  return static_cast<int>(0xffffffffu - static_cast<uint32_t>(k));
}

__device__ __forceinline__ float key_score(uint64_t k) {  // the Eq. (4) score of a key
  const uint32_t hi = static_cast<uint32_t>(k >> 32);
  return (hi & 0x80000000u) ? __builtin_amdgcn_sqrtf(__uint_as_float(hi & 0x7fffffffu)) : 0.0f;  // hardware square root (1 ulp)
}

// Ranking by counting compares keys as doubles: hi * 2^14 + (16383 - index)
// is exact (hi < 2^32, index < 2^14) and orders like the key, and a key y
// exceeds x exactly when x - y (exact) is negative, so a count is a sum of
// sign bits, with no compare masks.
__device__ __forceinline__ double key_rank_value(uint64_t k) {
  return static_cast<double>(static_cast<uint32_t>(k >> 32)) * 16384.0 + static_cast<double>(16383 - key_index(k));
}
__device__ __forceinline__ int above(double x, double y) {  // 1 when y > x
  return static_cast<int>(__builtin_bit_cast(uint64_t, x - y) >> 63);
}
__device__ __forceinline__ int rank_value_index(double v) {  // the index a rank value encodes
  const double hi = __builtin_floor(v * (1.0 / 16384.0));
  return 16383 - static_cast<int>(v - hi * 16384.0);
}
__device__ __forceinline__ uint64_t rank_value_key(double v) {
  const double hi = __builtin_floor(v * (1.0 / 16384.0));
  const int i = 16383 - static_cast<int>(v - hi * 16384.0);
  return (static_cast<uint64_t>(static_cast<uint32_t>(hi)) << 32) | (0xffffffffu - static_cast<uint32_t>(i));
}

// ---- wave64 reductions on the DPP network (row shifts, then row broadcasts)
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ uint32_t dpp_umax(uint32_t v) {
  const uint32_t o = __builtin_amdgcn_update_dpp(0u, v, CTRL, ROW_MASK, 0xf, false);
  return o > v ? o : v;
}

__device__ __forceinline__ uint32_t wave_umax32(uint32_t v) {
  v = dpp_umax<0x111, 0xf>(v);  // row_shr:1
  v = dpp_umax<0x112, 0xf>(v);  // row_shr:2
  v = dpp_umax<0x114, 0xf>(v);  // row_shr:4
  v = dpp_umax<0x118, 0xf>(v);  // row_shr:8   -> lane 15 of each row holds the row maximum
  v = dpp_umax<0x142, 0xa>(v);  // row_bcast:15
  v = dpp_umax<0x143, 0xc>(v);  // row_bcast:31 -> lane 63 holds the wave maximum
  return __builtin_amdgcn_readlane(v, 63);
}

template <int V>
struct IntC {  // a compile-time integer argument
  static constexpr int value = V;
};

// Lane n of each row of 16 lanes, broadcast to its row (DPP row_newbcast).
template <int N_>
__device__ __forceinline__ float row_bcast_c(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x150 + N_, 0xf, 0xf, false));
}
__device__ __forceinline__ float row_bcast(float v, int n) {  // n a constant after unrolling
  switch (n) {
    case 0: return row_bcast_c<0>(v);   case 1: return row_bcast_c<1>(v);
    case 2: return row_bcast_c<2>(v);   case 3: return row_bcast_c<3>(v);
    case 4: return row_bcast_c<4>(v);   case 5: return row_bcast_c<5>(v);
    case 6: return row_bcast_c<6>(v);   case 7: return row_bcast_c<7>(v);
    case 8: return row_bcast_c<8>(v);   case 9: return row_bcast_c<9>(v);
    case 10: return row_bcast_c<10>(v); case 11: return row_bcast_c<11>(v);
    case 12: return row_bcast_c<12>(v); case 13: return row_bcast_c<13>(v);
    case 14: return row_bcast_c<14>(v); default: return row_bcast_c<15>(v);
  }
}

// Largest 64-bit key of the wave (0 if every lane holds 0).
__device__ __forceinline__ uint64_t wave_max_key(uint64_t k) {
  const uint32_t hi = static_cast<uint32_t>(k >> 32);
  const uint32_t mhi = wave_umax32(hi);
  const uint32_t mlo = wave_umax32(hi == mhi ? static_cast<uint32_t>(k) : 0u);
  return (static_cast<uint64_t>(mhi) << 32) | mlo;
}

// ------------------------------------------------------------------ clear
// Zeroes the image barrier counters and the error flag before a selection
// launch (map_prune clears them in its scoring kernel instead).
__global__ __launch_bounds__(64) void select_clear_kernel(const SelectArgs a) {
  for (int i = threadIdx.x; i < a.B; i += 64) a.bar[i] = 0u;
  if (threadIdx.x == 0) *a.err = 0;
}

// ------------------------------------------------------------------ selection
// LDS row stride (floats) of the coefficient columns: 4 times an odd number,
// so float4 reads of 16 consecutive rows hit 16 different bank groups.
__host__ __device__ inline int col_stride(int K) { return ((K + 31) & ~31) + 4; }

struct Lds {
  // byte offsets into the dynamic LDS block
  int midx, mp, mn, mqn, mr2, mkey, pslot, pr, pgain, pcol, U, RW, merge, bnd, misc;
  int ownC, D, flags, r2acc;  // pipelined update only
  int bytes;
  int cs, us, rs, ws, ocs;
};

// RW holds the pool's residual Gram matrix during the picks and the own
// tokens' new rows (W) during the update; the two never live together.
// mr2 holds the members' r^2 at the round start; the mkey space is not
// read (the picking wave keeps the keys in registers).
__host__ __device__ inline Lds lds_layout(int K, int G, int ch, int pcap, bool pipe) {
  Lds L;
  int o = 0;
  auto take = [&](int bytes) { const int r = o; o += (bytes + 15) & ~15; return r; };
  L.cs = col_stride(K);
  // U rows hold kMaxPool entries whatever the pool capacity, so the pick
  // loop's fixed-length dot never leaves its row; 4 times an odd number
  L.us = kMaxPool + 4 + (((kMaxPool + 4) / 4) % 2 == 0 ? 4 : 0);
  L.rs = pcap + 1;
  L.ws = ch + 4;
  L.midx = take(4 * pcap);
  L.mp = take(4 * pcap);
  L.mn = take(4 * pcap);
  L.mqn = take(4 * pcap);
  L.mr2 = take(2 * 4 * pcap);
  L.mkey = take(2 * 8 * pcap);
  L.pslot = take(4 * pcap);
  L.pr = take(4 * pcap);
  L.pgain = take(4 * pcap);
  // pipelined: the pool members' coefficient rows, and once the round's
  // products are done this round's coefficients of the own tokens [ch][us];
  // the non-pipelined variant reads the members' rows from global memory
  L.pcol = take(4 * (pipe ? max(pcap * L.cs, ch * L.us) : 0));
  L.U = take(4 * pcap * L.us);
  const int rbytes = 4 * pcap * L.rs, wbytes = 4 * pcap * L.ws;
  L.RW = take(rbytes > wbytes ? rbytes : wbytes);
  L.merge = take(max(8 * (G * kPub + 2), 4 * ch));  // also the picked-token flags
  L.bnd = take(8 * ((kPub + 1) * (NT / 64)));
  L.misc = take(64);
  // pipelined update: the own tokens' coefficient rows of earlier rounds
  // (token-major, stride 4 times an odd number), the earlier rounds' part of
  // every pool member's row at the own tokens (D) and the stage counters
  L.ocs = ((K + 3) & ~3) + 4 + ((((K + 3) & ~3) / 4 + 1) % 2 == 0 ? 4 : 0);
  L.ownC = pipe ? take(4 * ch * L.ocs) : 0;
  L.D = pipe ? take(4 * pcap * L.ws) : 0;
  L.flags = pipe ? take(32) : 0;
  L.r2acc = pipe ? take(4 * 64) : 0;
  L.bytes = o;
  return L;
}

__device__ void image_barrier(unsigned int* ctr, unsigned int target, int32_t* err, int* abort_flag) {
  __syncthreads();
  if (threadIdx.x == 0) {
    __threadfence();
    atomicAdd(ctr, 1u);
    unsigned spins = 0;
    while (__hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
      __builtin_amdgcn_s_sleep(1);
      if (++spins > kSpinLimit) {
        atomicExch(err, 1);
        *abort_flag = 1;
        break;
      }
    }
    __threadfence();
  }
  __syncthreads();
}

// ------------------------------------------------------------------ R0 in one pass
// R0 is known from p alone, so its K0 picks need no argmax: their coefficients
// are the rows of one triangular factorisation,
//     c_{k,i} = (S[r_k][i] - sum_{l<k} c_{l,r_k} c_{l,i}) / r_k,
// over the pivots r_0 .. r_{K0-1} (descending p).  Every workgroup finds R0
// itself, loads X = [S among R0 ; S between R0 and its own tokens] (rows are
// tokens, columns pivots, the R0 diagonal set to 1, or 0 for a zero row) and
// factors it left-looking in column blocks of 16 (its own kernel: the
// selection kernel's registers and LDS are laid out for the rounds):
//   update  X[r][J] -= X[r][0:J0] X[J][0:J0]^T     (matrix cores, every row r at or past J)
//   pivot   the 16 x 16 diagonal block in one wave's registers; a pivot whose
//           unit residual is at most tau gets r = 0 and a zero column
//   panel   X[r][J] solved against the diagonal block, one thread per row
// The own rows end as the own tokens' coefficients, the R0 rows as the
// factor.  Workgroup w of an image owns tokens [64 w, 64 w + 64).
constexpr int kR0Max = 128;   // largest K0 placed this way (larger: by pool rounds)
constexpr int kR0Cand = 1024; // keys the top-K0 ranking holds

typedef __attribute__((ext_vector_type(4))) float f32x4_t;

__host__ __device__ inline bool r0_by_factor(int K0) { return K0 > 0 && K0 <= kR0Max; }

constexpr int kAs = 20;  // row stride of a solve operator: 4 times an odd number

struct R0Lds {
  int X, r0, ainv, cand, kmax, misc, flags, bytes;
  int K0p, xs, xrows;
};

__host__ __device__ inline R0Lds r0_layout(int K0) {
  R0Lds L;
  int o = 0;
  auto take = [&](int bytes) { const int r = o; o += (bytes + 15) & ~15; return r; };
  L.K0p = (K0 + 15) & ~15;
  L.xs = L.K0p + 4;  // 4 times an odd number: float4 reads of 16 rows hit 16 bank groups
  L.xrows = 64 * ((L.K0p + 64 + 63) / 64);  // R0 rows, then 64 own rows, in whole blocks of 64
  L.X = take(4 * L.xrows * L.xs);
  L.r0 = take(4 * L.K0p);
  L.ainv = take(4 * L.K0p * kAs);  // [K0p / 16][16][kAs]
  L.cand = take(8 * (kR0Cand + 8));
  L.kmax = take(8 * NT);
  L.misc = take(16);
  L.flags = take(16);
  L.bytes = o;
  return L;
}

// Places R0 for image blockIdx.y: the own tokens' coefficient rows on the
// K0 pivots (global C) and their r^2 (global r2), and (workgroup 0) the
// selection order and gains of the first K0 picks and the image's flag
// r0flag = 1.  When more than kR0Cand keys tie with or exceed the threads'
// K0-th largest maximum it writes nothing but r0flag = 0: the selection
// kernel then places R0 by pool rounds.
__global__ __launch_bounds__(NT) void r0_kernel(const SelectArgs a) {
  extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
  const int N = a.N, K0 = a.K0, K = a.K, Kp = (K + 3) & ~3;
  const int b = blockIdx.y, w = blockIdx.x;
  if (a.run_if && a.run_if[b] == 0) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const float* p = a.p + (long long)b * N;
  const float* nrm = a.norms + (long long)b * N;
  const float* S = a.S + (long long)b * N * N;
  float* Ct = a.C + (long long)b * N * Kp;
  float* r2g = a.r2 + (long long)b * N;
  const int c0 = 64 * w, cnt = min(64, N - c0);
  const R0Lds R = r0_layout(K0);
  float* X = reinterpret_cast<float*>(lds + R.X);
  int* r0 = reinterpret_cast<int*>(lds + R.r0);
  float* Ainv = reinterpret_cast<float*>(lds + R.ainv);
  int* flg = reinterpret_cast<int*>(lds + R.flags);
  double* cand = reinterpret_cast<double*>(lds + R.cand);  // rank values
  double* kmax = reinterpret_cast<double*>(lds + R.kmax);
  int* ncand = reinterpret_cast<int*>(lds + R.misc);
  uint64_t* T0p = reinterpret_cast<uint64_t*>(lds + R.misc + 8);
  const int K0p = R.K0p, xs = R.xs, nb = K0p / 16;

  // ---- R0 = the K0 largest keys.  Thread u sees tokens u, u + NT, ...; the
  // K0-th largest of the threads' maxima, T0, is at most the K0-th largest
  // key, so the keys >= T0 hold R0; each of them is ranked by counting.
  // The first PC tokens of each thread stay in registers for the second pass.
  constexpr int PC = 16, PB = 8;
  auto key_of = [](float pv, int i) -> uint64_t {
    return (static_cast<uint64_t>(ordered_bits(pv)) << 32) | (0xffffffffu - static_cast<uint32_t>(i));
  };
  float pc[PC];
#pragma unroll
  for (int u = 0; u < PC; ++u) pc[u] = p[min(tid + u * NT, N - 1)];
  uint64_t mx = 0;
#pragma unroll
  for (int u = 0; u < PC; ++u) {
    const int i = tid + u * NT;
    const uint64_t k = key_of(pc[u], i);
    mx = (i < N && k > mx) ? k : mx;
  }
  for (int i0 = tid + PC * NT; i0 < N; i0 += PB * NT) {
    float pv[PB];
#pragma unroll
    for (int u = 0; u < PB; ++u) pv[u] = p[min(i0 + u * NT, N - 1)];
#pragma unroll
    for (int u = 0; u < PB; ++u) {
      const int i = i0 + u * NT;
      const uint64_t k = key_of(pv[u], i);
      mx = (i < N && k > mx) ? k : mx;
    }
  }
  // threads t and t + NT/2 pool their maxima: the NT/2 pair maxima are keys of
  // disjoint token sets, so the K0-th largest of them (K0 <= NT/2) is still
  // at most the K0-th largest key
  uint64_t* kpair = reinterpret_cast<uint64_t*>(kmax);
  if (tid >= NT / 2) kpair[tid] = mx;
  if (tid == 0) *ncand = 0;
  __syncthreads();
  if (tid < NT / 2) {
    const uint64_t other = kpair[tid + NT / 2];
    mx = other > mx ? other : mx;
  }
  const double mxv = mx ? key_rank_value(mx) : -1.0;  // pairs without tokens rank last
  __syncthreads();
  if (tid < NT / 2) kmax[tid] = mxv;
  __syncthreads();
  if (tid < NT / 2) {
    const double2* y2 = reinterpret_cast<const double2*>(kmax);
    int r4[4] = {0, 0, 0, 0};  // independent counters: no serial chain
    for (int u0 = 0; u0 < NT / 4; u0 += 16) {
      double2 y[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) y[u] = y2[u0 + u];
#pragma unroll
      for (int u = 0; u < 16; ++u) r4[u & 3] += above(mxv, y[u].x) + above(mxv, y[u].y);
    }
    // at least K0 pairs hold tokens (N >= K0, K0 <= NT/2): pair p holds token
    // p; their maxima are distinct, and the empty pairs' zeros rank below them
    if ((r4[0] + r4[1]) + (r4[2] + r4[3]) == K0 - 1) *T0p = mx;
  }
  __syncthreads();
  const uint64_t T0 = *T0p;
  // candidates: the register-cached tokens first (a mask, then one LDS atomic
  // per thread for all of them), the rest one atomic each
  uint32_t cm = 0u;
#pragma unroll
  for (int u = 0; u < PC; ++u) {
    const int i = tid + u * NT;
    cm |= (i < N && key_of(pc[u], i) >= T0) ? 1u << u : 0u;
  }
  {
    // the wave's exclusive prefix sum of the counts (at most PC = 16, five
    // bit planes), then one atomic per wave
    const int c = __builtin_popcount(cm);
    int pre = 0, tot = 0;
#pragma unroll
    for (int bit = 0; bit < 5; ++bit) {
      const uint64_t m = __ballot((c >> bit) & 1);
      pre += static_cast<int>(__builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(m >> 32),
                                                         __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(m), 0u)))
             << bit;
      tot += __builtin_popcountll(m) << bit;
    }
    if (tot > 0) {
      int base = 0;
      if (lane == 0) base = atomicAdd(ncand, tot);
      int o = __builtin_amdgcn_readlane(base, 0) + pre;
#pragma unroll
      for (int u = 0; u < PC; ++u)
        if ((cm >> u) & 1u) {
          if (o < kR0Cand) cand[o] = key_rank_value(key_of(pc[u], tid + u * NT));
          ++o;
        }
    }
  }
  for (int i0 = tid + PC * NT; i0 < N; i0 += PB * NT) {
    float pv[PB];
#pragma unroll
    for (int u = 0; u < PB; ++u) pv[u] = p[min(i0 + u * NT, N - 1)];
#pragma unroll
    for (int u = 0; u < PB; ++u) {
      const int i = i0 + u * NT;
      const uint64_t k = key_of(pv[u], i);
      if (i < N && k >= T0) {
        const int o = atomicAdd(ncand, 1);
        if (o < kR0Cand) cand[o] = key_rank_value(k);
      }
    }
  }
  __syncthreads();
  const int nc = *ncand;
  if (nc > kR0Cand) {  // the same on every workgroup of the image
    if (w == 0 && tid == 0) a.r0flag[b] = 0;
    return;
  }
  if (tid < 8) cand[nc + tid] = -1.0;  // whole groups of 8 for the ranking loop
  __syncthreads();
  for (int c = tid; c < nc; c += NT) {
    const double x = cand[c];
    int r4[4] = {0, 0, 0, 0};
    const double2* y2 = reinterpret_cast<const double2*>(cand);
    for (int j = 0; j < nc; j += 8) {
      const double2 y0 = y2[j / 2], y1 = y2[j / 2 + 1], y2v = y2[j / 2 + 2], y3 = y2[j / 2 + 3];
      r4[0] += above(x, y0.x) + above(x, y0.y);
      r4[1] += above(x, y1.x) + above(x, y1.y);
      r4[2] += above(x, y2v.x) + above(x, y2v.y);
      r4[3] += above(x, y3.x) + above(x, y3.y);
    }
    const int rk = (r4[0] + r4[1]) + (r4[2] + r4[3]);
    if (rk < K0) r0[rk] = rank_value_index(x);
  }
  __syncthreads();
  const int rlast = r0[K0 - 1];  // own tokens with keys >= klast are in R0
  const uint64_t klast = key_of(p[rlast], rlast);
  const int rmine = r0[min(tid, K0 - 1)];
  const float pmine = p[rmine];  // gain of pick tid (workgroup 0 writes it below)

  // ---- the factorisation
  {
    const int ocnt = cnt;
    // X[row][c] = S[r0[c]][token(row)]: lane = row within a block of 64 rows,
    // wave w takes columns w, w + 4, ...  R0 rows load only their strictly
    // lower part (the factorisation never reads above the diagonal), own rows
    // the K0 columns; every load (lanes with nothing to load read one shared
    // address) is issued before the first store, and the stores are
    // branch-free selects over whole row blocks
    {
      constexpr int QB = kR0Max / 4;  // columns per wave at most
      const int nq = K0p / 4, nh = R.xrows / 64;
      int rc[QB];
#pragma unroll
      for (int q = 0; q < QB; ++q) rc[q] = r0[min(wave + 4 * q, K0 - 1)];
      int tok[3], lim[3];
      float dg[3];
#pragma unroll
      for (int h = 0; h < 3; ++h) {
        const int row = 64 * h + lane;
        const bool isr0 = row < K0p;
        const bool valid = isr0 ? row < K0 : row - K0p < ocnt;
        tok[h] = valid ? (isr0 ? r0[min(row, K0 - 1)] : c0 + min(row - K0p, ocnt - 1)) : c0;
        lim[h] = !valid ? 0 : isr0 ? row : K0;
        dg[h] = (isr0 && valid) ? nrm[tok[h]] : 0.0f;  // the diagonal: 1 for a nonzero row (below)
      }
      float v[3][QB];
#pragma unroll
      for (int qc = 0; qc < QB / 4; ++qc)
        if (4 * qc < nq) {
#pragma unroll
          for (int h = 0; h < 3; ++h)
            if (h < nh) {
#pragma unroll
              for (int qq = 0; qq < 4; ++qq) {
                const int q = 4 * qc + qq, c = wave + 4 * q;
                v[h][q] = S[(long long)rc[q] * N + (c < lim[h] ? tok[h] : c0)];
              }
            }
        }
#pragma unroll
      for (int qc = 0; qc < QB / 4; ++qc)
        if (4 * qc < nq) {
#pragma unroll
          for (int h = 0; h < 3; ++h)
            if (h < nh) {
              const int row = 64 * h + lane;
#pragma unroll
              for (int qq = 0; qq < 4; ++qq) {
                const int q = 4 * qc + qq, c = wave + 4 * q;
                X[row * xs + c] = c < lim[h] ? v[h][q] : (c == row && dg[h] > 0.0f ? 1.0f : 0.0f);
              }
            }
        }
    }
    if (w == 0) {  // the first K0 picks of the selection order
      if (tid == 0) a.r0flag[b] = 1;
      if (tid < K0) {
        a.order[(long long)b * K + tid] = rmine;
        a.gain[(long long)b * K + tid] = (pmine > 0.0f && pmine <= 3.402823466e38f) ? pmine : 0.0f;
        if (a.order_map) a.order_map[(long long)b * K + tid] = a.jmap[(long long)b * N + rmine];
      }
    }
    if (tid == 0) {
      flg[0] = 0;  // pivots done
      flg[1] = 0;  // row blocks past the diagonal solved by wave 0
      flg[2] = 1;  // next diagonal block prepared (nothing to prepare for block 1)
    }
    __syncthreads();
    // Row block R is rows 16 R .. 16 R + 15 of X for R < nb (R0) and own rows
    // 16 (R - nb) .. for R >= nb.  Column block j is columns 16 j ...
    //   pivot j   factor the diagonal block (j, j), already brought up to date,
    //             into its solve operator A_j (A_j b solves L_jj y = b, with
    //             the entries of skipped pivots zero)
    //   P(R, j)   X[R][j] = X[R][j] A_j^T (the coefficients on pivots of block j)
    //   U(R, c)   X[R][c] -= X[R][0:16 c] X[c][0:16 c]^T
    // Wave 0 runs the chain pivot j, P(j+1, j), the last term of U(j+1, j+1),
    // pivot j+1, ...; waves 1 to 3 run every other row block (block R on wave
    // 1 + R % 3): in phase j, P(R, j) and U(R, j+1), and for R = j + 2 also
    // U(R, R) over the blocks up to j, which wave 0 needs next.  Three LDS
    // counters order the two sides: pivots done, wave 0's P(j+1, j) stored,
    // next diagonal block prepared.
    const int nown = (ocnt + 15) >> 4;
    auto wait_ge = [&](const int* f, int v) {
      while (__hip_atomic_load(f, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP) < v) {
      }
    };
    auto signal = [&](int* f, int v) {  // after this wave's LDS writes
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
      if (lane == 0) __hip_atomic_store(f, v, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
    };
    // 16 x 16 tile X[rA + i][cC + n] -= sum over k in [16 s0, 16 s1) of
    // X[rA + i][k] X[rB + n][k] on matrix cores; lane group g supplies
    // k = 16 s + 4 g + e to the e-th product of step s; result row 4 g + e,
    // column lane & 15
    constexpr int KS = kR0Max / 16;
    auto tile_update = [&](int rA, int rB, int cC, int s0, int s1) {
      const float* arow = X + (rA + (lane & 15)) * xs + 4 * (lane >> 4);
      const float* brow = X + (rB + (lane & 15)) * xs + 4 * (lane >> 4);
      float* drow = X + (rA + 4 * (lane >> 4)) * xs + cC + (lane & 15);
      float cur[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) cur[e] = drow[e * xs];
      f32x4_t av[KS], bv[KS];
#pragma unroll
      for (int s = 0; s < KS; ++s)
        if (s >= s0 && s < s1) {
          av[s] = *reinterpret_cast<const f32x4_t*>(arow + 16 * s);
          bv[s] = *reinterpret_cast<const f32x4_t*>(brow + 16 * s);
        }
      f32x4_t acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int s = 0; s < KS; ++s)
        if (s >= s0 && s < s1) {
          acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av[s].x, bv[s].x, acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av[s].y, bv[s].y, acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av[s].z, bv[s].z, acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av[s].w, bv[s].w, acc, 0, 0, 0);
        }
#pragma unroll
      for (int e = 0; e < 4; ++e) drow[e * xs] = cur[e] - acc[e];
    };
    // P(R, j) for the 16 rows at rbase: X[..][16 j ..] = X[..][16 j ..] A_j^T
    auto panel = [&](int rbase, int j) {
      const int J0 = 16 * j;
      const f32x4_t av = *reinterpret_cast<const f32x4_t*>(X + (rbase + (lane & 15)) * xs + J0 + 4 * (lane >> 4));
      const f32x4_t bv = *reinterpret_cast<const f32x4_t*>(Ainv + (J0 + (lane & 15)) * kAs + 4 * (lane >> 4));
      f32x4_t acc = {0.0f, 0.0f, 0.0f, 0.0f};
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av.x, bv.x, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av.y, bv.y, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av.z, bv.z, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av.w, bv.w, acc, 0, 0, 0);
      float* drow = X + (rbase + 4 * (lane >> 4)) * xs + J0 + (lane & 15);
#pragma unroll
      for (int e = 0; e < 4; ++e) drow[e * xs] = acc[e];
    };
    if (wave == 0) {
      const int j = lane & 15, q = lane >> 4;
      float x[16];  // row j of the current diagonal block
      auto load_diag = [&](int jb) {
        const float* xr = X + (16 * jb + j) * xs + 16 * jb;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const f32x4_t v = *reinterpret_cast<const f32x4_t*>(xr + 4 * u);
          x[4 * u] = v.x; x[4 * u + 1] = v.y; x[4 * u + 2] = v.z; x[4 * u + 3] = v.w;
        }
      };
      load_diag(0);
      for (int jb = 0; jb < nb; ++jb) {
        // pivot: straight-line code (selects, no branches); every lane of a
        // row of 16 gets the pivot and the column entries it needs by DPP
        // broadcast within the row
        float myri = 0.0f;  // 1 / r of pivot j (0: no basis vector)
        float lz[16];       // L[j][k] below the diagonal, zero elsewhere
#pragma unroll
        for (int k = 0; k < 16; ++k) {
          const float d = row_bcast(x[k], k);
          const float rinv = d > a.tau2 ? __builtin_amdgcn_rsqf(d) : 0.0f;  // hardware reciprocal square root (1 ulp)
          const float lj = j > k ? x[k] * rinv : 0.0f;
          lz[k] = lj;
          myri = j == k ? rinv : myri;
#pragma unroll
          for (int j2 = k + 1; j2 < 16; ++j2) x[j2] = fmaf(-lj, row_bcast(lj, j2), x[j2]);
        }
        // A_j row by row: A[j] = ri_j (e_j - sum_{k<j} L[j][k] A[k]); copy q
        // of the row of 16 lanes forms columns q, q + 4, q + 8 and q + 12
        float bq[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) bq[i] = q + 4 * i == j ? 1.0f : 0.0f;
#pragma unroll
        for (int k = 0; k < 15; ++k) {
          const float sk = lz[k] * row_bcast(myri, k);
#pragma unroll
          for (int i = 0; i < 4; ++i) bq[i] = fmaf(-sk, row_bcast(bq[i], k), bq[i]);
        }
        float* ar = Ainv + (16 * jb + j) * kAs + q;
#pragma unroll
        for (int i = 0; i < 4; ++i) ar[4 * i] = myri * bq[i];
        signal(flg + 0, jb + 1);
        if (jb + 1 < nb) {
          const int r1 = 16 * (jb + 1);
          wait_ge(flg + 2, jb + 1);  // U(jb+1, jb) and the earlier terms of U(jb+1, jb+1) are in
          panel(r1, jb);
          signal(flg + 1, jb + 1);
          tile_update(r1, r1, r1, jb, jb + 1);  // the last term of U(jb+1, jb+1)
          load_diag(jb + 1);
        }
      }
    } else {
      for (int jb = 0; jb < nb; ++jb) {
        for (int R = min(jb + 2, nb); R < nb + nown; ++R) {  // R0 blocks past jb + 1, then the own blocks
          if (1 + R % 3 != wave) continue;
          const int rbase = R < nb ? 16 * R : K0p + 16 * (R - nb);
          wait_ge(flg + 0, jb + 1);
          panel(rbase, jb);
          if (jb + 1 < nb) {
            const int c1 = 16 * (jb + 1);
            wait_ge(flg + 1, jb + 1);  // row block jb+1 solved up to column block jb
            tile_update(rbase, c1, c1, 0, jb + 1);  // U(R, jb+1)
            if (R == jb + 2 && R < nb) {  // the next diagonal block but one
              tile_update(rbase, rbase, rbase, 0, jb + 1);  // U(R, R) up to column block jb
              signal(flg + 2, jb + 2);
            }
          }
        }
      }
    }
    __syncthreads();
    // own rows out: piece e = (own row e >> 5, float4 e & 31)
    const int K0q = (K0 + 3) >> 2;  // at most 32; columns K0 .. 4 K0q - 1 are zero
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int e = tid + NT * u, i = e >> 5, q = e & 31;
      if (i < ocnt && q < K0q)
        *reinterpret_cast<f32x4_t*>(Ct + (long long)(c0 + i) * Kp + 4 * q) =
            *reinterpret_cast<const f32x4_t*>(X + (K0p + i) * xs + 4 * q);
    }
    uint64_t mykey = 0ull;  // own candidate's Eq. (4) key (0: none)
    if (tid < ocnt) {  // R0 members get a NaN r^2: the selection kernel reads them as selected
      const float* xr = X + (K0p + tid) * xs;
      f32x4_t s4 = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int q = 0; q < kR0Max / 4; ++q)
        if (q < K0q) {
          const f32x4_t v = *reinterpret_cast<const f32x4_t*>(xr + 4 * q);
          s4 += v * v;
        }
      const int i = c0 + tid;
      const uint64_t ki = (static_cast<uint64_t>(ordered_bits(p[i])) << 32) | (0xffffffffu - static_cast<uint32_t>(i));
      const bool in_r0 = ki >= klast;
      const float r2v = (nrm[i] > 0.0f ? 1.0f : 0.0f) - ((s4.x + s4.y) + (s4.z + s4.w));
      r2g[i] = in_r0 ? __builtin_nanf("") : r2v;
      if (!in_r0) {
        const float pi = p[i];
        const float pv = (pi > 0.0f && pi <= 3.402823466e38f) ? pi : 0.0f;
        mykey = make_key(r2v, pv * nrm[i], pv, i, a.tau2);
      }
    }
    // The keys the selection's first round merges, when its workgroups own
    // the same 64 tokens: the own candidates' top kPub keys and the next one
    // as a bound (the kernel boundary orders them before their readers).
    if (a.ch == 64 && K0 < K && wave == 0) {
      uint64_t* pub = a.pub + ((long long)b * 2 + 1) * a.G * (kPub + 1) + w * (kPub + 1);
      for (int q = 0; q <= kPub; ++q) {
        const uint64_t best = wave_max_key(mykey);
        if (lane == 0) pub[q] = best;
        if (mykey == best) mykey = 0ull;
      }
    }
  }
}

// One 32 x 32 float32 tile, acc[e] = sum over l < tk of A[row][l] B[col][l]
// for row 8 (e >> 2) + 4 h + (e & 3) and column lane & 31 (h = lane >> 5),
// with arow and brow pointing at this lane's row and column plus 4 h; tk is
// a multiple of 8 and the entries up to tk are valid (zero past the data).
// Odd and even steps of eight accumulate separately and each step's
// operands are read before the previous step's products issue.
__device__ __forceinline__ void tile_product(const float* arow, const float* brow, int tk, f32x16_t& out) {
  f32x16_t acc[2];
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[x][e] = 0.0f;
  auto step = [&](int x, const f32x4_t& av, const f32x4_t& bv) {
    acc[x] = __builtin_amdgcn_mfma_f32_32x32x2f32(av.x, bv.x, acc[x], 0, 0, 0);
    acc[x] = __builtin_amdgcn_mfma_f32_32x32x2f32(av.y, bv.y, acc[x], 0, 0, 0);
    acc[x] = __builtin_amdgcn_mfma_f32_32x32x2f32(av.z, bv.z, acc[x], 0, 0, 0);
    acc[x] = __builtin_amdgcn_mfma_f32_32x32x2f32(av.w, bv.w, acc[x], 0, 0, 0);
  };
  f32x4_t a = *reinterpret_cast<const f32x4_t*>(arow);
  f32x4_t b = *reinterpret_cast<const f32x4_t*>(brow);
  int l0 = 0;
  for (; l0 + 16 <= tk; l0 += 16) {
    const f32x4_t a2 = *reinterpret_cast<const f32x4_t*>(arow + l0 + 8);
    const f32x4_t b2 = *reinterpret_cast<const f32x4_t*>(brow + l0 + 8);
    step(0, a, b);
    const int ln = min(l0 + 16, tk - 8);  // the next step's rows (a valid read at the end)
    a = *reinterpret_cast<const f32x4_t*>(arow + ln);
    b = *reinterpret_cast<const f32x4_t*>(brow + ln);
    step(1, a2, b2);
  }
  if (l0 < tk) step(0, a, b);  // an odd last step
  out = acc[0] + acc[1];
}

// The same tile with both operands in global memory: acc[e] += sum over
// l < t of A[row][l] B[col][l], arow and brow pointing at this lane's rows
// (rows of at least kp floats, kp a multiple of 4 and at least t).  The
// lane's pieces (columns 8 s + 4 h .. of step s) are loaded a group of PF
// steps ahead, in two register buffers used in turn; a read past the row
// stays at a valid address, and in the last step the columns at or past t
// are zero in both operands (entries past t may hold anything).
template <int PF>
__device__ __forceinline__ void gtile_product(const float* arow, const float* brow, int t, int kp, int h,
                                              f32x16_t& acc) {
  const int ns = (t + 7) >> 3;  // steps of eight columns, the last possibly partial
  auto load = [&](f32x4_t (&av)[PF], f32x4_t (&bv)[PF], int s0) {
#pragma unroll
    for (int q = 0; q < PF; ++q) {
      const int c = min(8 * (s0 + q) + 4 * h, kp - 4);
      av[q] = *reinterpret_cast<const f32x4_t*>(arow + c);
      bv[q] = *reinterpret_cast<const f32x4_t*>(brow + c);
    }
  };
  auto run = [&](const f32x4_t (&av)[PF], const f32x4_t (&bv)[PF], int s0) {
#pragma unroll
    for (int q = 0; q < PF; ++q) {
      const int st = s0 + q;
      if (st < ns) {  // (uniform)
        f32x4_t a4 = av[q], b4 = bv[q];
        if (st == ns - 1 && (t & 7)) {
          const int c = 8 * st + 4 * h;
          const f32x4_t z = {0.0f, 0.0f, 0.0f, 0.0f};
          a4.x = c < t ? a4.x : z.x; b4.x = c < t ? b4.x : z.x;
          a4.y = c + 1 < t ? a4.y : z.y; b4.y = c + 1 < t ? b4.y : z.y;
          a4.z = c + 2 < t ? a4.z : z.z; b4.z = c + 2 < t ? b4.z : z.z;
          a4.w = c + 3 < t ? a4.w : z.w; b4.w = c + 3 < t ? b4.w : z.w;
        }
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a4.x, b4.x, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a4.y, b4.y, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a4.z, b4.z, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a4.w, b4.w, acc, 0, 0, 0);
      }
    }
  };
  if (ns == 0) return;
  f32x4_t ax[PF], bx[PF], ay[PF], by[PF];
  load(ax, bx, 0);
  for (int s0 = 0; s0 < ns; s0 += 2 * PF) {
    load(ay, by, s0 + PF);
    __builtin_amdgcn_sched_barrier(0);
    run(ax, bx, s0);
    __builtin_amdgcn_sched_barrier(0);
    if (s0 + PF >= ns) break;
    load(ax, bx, s0 + 2 * PF);
    __builtin_amdgcn_sched_barrier(0);
    run(ay, by, s0 + PF);
    __builtin_amdgcn_sched_barrier(0);
  }
}

// Global C is token-major: Ct[i][l] = c_{l,i}, rows of Kp floats (Kp = K
// rounded up to 4), so one token's coefficients are contiguous.
template <bool PIPE>
__global__ __launch_bounds__(NT) void select_kernel(const SelectArgs a, int b_begin) {
  extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
  const int G = a.G, ch = a.ch, pcap = a.pcap, K = a.K, K0 = a.K0, N = a.N;
  const int Kp = (K + 3) & ~3;
  const int b = b_begin + blockIdx.x / G, w = blockIdx.x % G;
  const bool skip = a.run_if && a.run_if[b] == 0;  // (uniform over the image's workgroups)
  if (skip && !a.gV) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const Lds L = lds_layout(K, G, ch, pcap, PIPE);
  int* midx = reinterpret_cast<int*>(lds + L.midx);
  float* mp = reinterpret_cast<float*>(lds + L.mp);
  float* mn = reinterpret_cast<float*>(lds + L.mn);
  float* mqn = reinterpret_cast<float*>(lds + L.mqn);
  float* mr2 = reinterpret_cast<float*>(lds + L.mr2);     // [2][pcap]
  int* pslot = reinterpret_cast<int*>(lds + L.pslot);
  float* prr = reinterpret_cast<float*>(lds + L.pr);     // 1 / r of each pick (0: no basis vector)
  uint32_t* pgain = reinterpret_cast<uint32_t*>(lds + L.pgain);  // p (forced) or the key's high word, as bits
  float* pcol = reinterpret_cast<float*>(lds + L.pcol);
  float* U = reinterpret_cast<float*>(lds + L.U);
  float* Rm = reinterpret_cast<float*>(lds + L.RW);
  float* W = reinterpret_cast<float*>(lds + L.RW);
  uint64_t* merge = reinterpret_cast<uint64_t*>(lds + L.merge);
  uint64_t* bndk = reinterpret_cast<uint64_t*>(lds + L.bnd);
  int* misc = reinterpret_cast<int*>(lds + L.misc);
  const int cs = L.cs, us = L.us, rs = L.rs, wsd = L.ws, ocs = L.ocs;
  float* ownC = reinterpret_cast<float*>(lds + L.ownC);  // PIPE: [ch][ocs] own rows, earlier rounds
  float* Dm = reinterpret_cast<float*>(lds + L.D);       // PIPE: [pcap][wsd] pool rows at the own tokens
  float* crow = pcol;                                    // PIPE, picks: [ch][us] this round's own rows
  int* npub = reinterpret_cast<int*>(lds + L.flags);     // PIPE: picks published this round
  int* pdone = npub + 3;                                 // round tag once the picks are over
  int* dready = npub + 4;                                // waves done with their D tiles
  float* r2acc = reinterpret_cast<float*>(lds + L.r2acc);  // PIPE: finisher's sums of squares

  const float* p = a.p + (long long)b * N;
  const float* nrm = a.norms + (long long)b * N;
  const float* S = a.S + (long long)b * N * N;
  float* Ct = a.C + (long long)b * N * Kp;
  float* r2g = a.r2 + (long long)b * N;

  // ---- own tokens [c0, c0 + cnt); thread tid < ch keeps token c0 + tid
  const int c0 = w * ch;
  const int cnt = max(0, min(ch, N - c0));
  const int my_i = c0 + tid;
  // state: 0 candidate, 2 selected
  int my_state = 2;
  float my_r2 = 0.0f, my_qn = 0.0f, my_p = 0.0f;
  if (tid < cnt) {
    const float pi = p[my_i];
    const float ni = nrm[my_i];
    my_p = (pi > 0.0f && pi <= 3.402823466e38f) ? pi : 0.0f;
    my_qn = my_p * ni;
    my_r2 = ni > 0.0f ? 1.0f : 0.0f;
    my_state = 0;
  }
  // Publishes the top kPub + 1 keys of the own candidates into slot `slot`:
  // each wave extracts the top kPub + 1 of its tokens, then wave 0 the top
  // kPub + 1 of those.  While R0 is being placed the keys order by p alone
  // (descending p, then lower index), so the pools of those rounds are the
  // top of p; afterwards they order by the Eq. (4) score.
  auto publish = [&](int slot, bool by_p) {
    uint64_t k = 0ull;
    if (tid < cnt && my_state == 0)
      k = by_p ? ((static_cast<uint64_t>(ordered_bits(my_p)) << 32) | (0xffffffffu - static_cast<uint32_t>(my_i)))
               : make_key(my_r2, my_qn, my_p, my_i, a.tau2);
    if (ch <= 64) {  // the own tokens are wave 0's lanes: its top keys are the workgroup's
      if (wave == 0) {
        uint64_t* pub = a.pub + ((long long)b * 2 + slot) * G * (kPub + 1) + w * (kPub + 1);
        for (int q = 0; q <= kPub; ++q) {
          const uint64_t best = wave_max_key(k);
          if (lane == 0) __hip_atomic_store(pub + q, best, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          if (k == best) k = 0ull;
        }
      }
      return;
    }
    for (int q = 0; q <= kPub; ++q) {
      const uint64_t best = wave_max_key(k);
      if (lane == 0) bndk[wave * (kPub + 1) + q] = best;
      if (k == best) k = 0ull;
    }
    __syncthreads();
    if (wave == 0) {
      uint64_t k2 = lane < (NT / 64) * (kPub + 1) ? bndk[lane] : 0ull;
      uint64_t* pub = a.pub + ((long long)b * 2 + slot) * G * (kPub + 1) + w * (kPub + 1);
      for (int q = 0; q <= kPub; ++q) {
        const uint64_t best = wave_max_key(k2);
        if (lane == 0) __hip_atomic_store(pub + q, best, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (k2 == best) k2 = 0ull;
      }
    }
  };
  // Gather (map_prune): the kept rows and positions in ascending token
  // order (section "Inference-Time Token Pruning": the kept tokens return
  // to their original order and keep their positions).  Every workgroup
  // knows the whole order: the picks of the final round (from t_last) in
  // LDS, the earlier ones in the order array (written before a barrier).
  // Workgroup w writes ranks w, w + G, ...; after an abort, or with the
  // error flag set, its indices and positions are -1 and its rows zero.
  auto gather_share = [&](bool aborted, int t_last) {
    if (!a.gV) return;
    __syncthreads();  // LDS free
    const bool bad = aborted || __hip_atomic_load(a.err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0;
    int* ord = reinterpret_cast<int*>(lds + L.RW);  // [K rounded up to 8] (padding: past any index)
    int* share = reinterpret_cast<int*>(lds + L.merge);  // index of rank w + G s
    const int K8 = (K + 7) & ~7, nshare = w < K ? (K - w + G - 1) / G : 0;
    if (!bad) {
      for (int j = tid; j < K8; j += NT)
        ord[j] = j >= K ? 0x7fffffff : (j < t_last ? a.order[(long long)b * K + j] : midx[pslot[j - t_last]]);
      __syncthreads();
      for (int j = tid; j < K; j += NT) {  // rank = number of smaller indices (they are distinct)
        const int v = ord[j];
        int r4[4] = {0, 0, 0, 0};
        for (int q = 0; q < K8; q += 8) {
          const int4 x = *reinterpret_cast<const int4*>(ord + q);
          const int4 y = *reinterpret_cast<const int4*>(ord + q + 4);
          r4[0] += (x.x < v) + (y.x < v);
          r4[1] += (x.y < v) + (y.y < v);
          r4[2] += (x.z < v) + (y.z < v);
          r4[3] += (x.w < v) + (y.w < v);
        }
        const int rk = (r4[0] + r4[1]) + (r4[2] + r4[3]);
        // (a subset's positions order like its tokens: the ranks hold)
        if (rk % G == w) share[rk / G] = a.jmap ? a.jmap[(long long)b * N + v] : v;
      }
      __syncthreads();
    }
    const long long orow = (long long)b * K + a.out_off[b];  // the image's first output row
    for (int sI = tid; sI < nshare; sI += NT) {
      const int k = w + G * sI, v = bad ? -1 : share[sI];
      a.idx_out[(long long)b * K + k] = v;
      a.gpos_out[orow + k] = bad ? -1 : a.gpos[(long long)b * a.Ng + v];
    }
    // rows, 16 bytes per piece; every load of a thread before its first store
    const int chunks = a.row_bytes >> 4, total = nshare * chunks;
    const uint4* src = static_cast<const uint4*>(a.gV) + (long long)b * a.Ng * chunks;
    uint4* dst = static_cast<uint4*>(a.gV_out) + orow * chunks;
    if (a.qT) {  // layer-0 assembly: question rows w, w + G, ... of the image after its kept rows
      const int m0 = a.q_off[b], M = a.q_off[b + 1] - m0, nq = w < M ? (M - w + G - 1) / G : 0;
      const uint4* qs = static_cast<const uint4*>(a.qT) + (long long)m0 * chunks;
      uint4* qd = dst + (long long)K * chunks;
      constexpr int QU = 4;  // loads in flight per thread
      for (int e0 = tid; e0 < nq * chunks; e0 += QU * NT) {
        uint4 v[QU];
#pragma unroll
        for (int u = 0; u < QU; ++u) {
          const int e = min(e0 + u * NT, nq * chunks - 1), j = e / chunks, m = w + G * j;
          v[u] = qs[(long long)m * chunks + (e - j * chunks)];
        }
#pragma unroll
        for (int u = 0; u < QU; ++u) {
          const int e = e0 + u * NT, j = e / chunks, m = w + G * j;
          if (e < nq * chunks) qd[(long long)m * chunks + (e - j * chunks)] = v[u];
        }
      }
      for (int j = tid; j < nq; j += NT) a.gpos_out[orow + K + w + G * j] = a.qpos[m0 + w + G * j];
    }
    constexpr int GU = 4;
    for (int e0 = tid; e0 < total; e0 += GU * NT) {
      uint4 v[GU];
#pragma unroll
      for (int u = 0; u < GU; ++u) {
        const int e = min(e0 + u * NT, total - 1), sI = e / chunks;
        v[u] = src[(long long)(bad ? 0 : share[sI]) * chunks + (e - sI * chunks)];
      }
#pragma unroll
      for (int u = 0; u < GU; ++u) {
        const int e = e0 + u * NT;
        if (e < total) {
          const int sI = e / chunks;
          dst[(long long)(w + G * sI) * chunks + (e - sI * chunks)] = bad ? make_uint4(0u, 0u, 0u, 0u) : v[u];
        }
      }
    }
  };

  // A skipped image (its selection was made on a candidate subset) only
  // gathers: its whole order is in the order array, as image tokens.
  if (skip) {
    gather_share(false, K);
    return;
  }

  // R0 placed by r0_kernel (when it fits and did not give up): take over the
  // own tokens' state and coefficient rows; otherwise the first rounds place it
  bool r0_done = false;
  if (r0_by_factor(K0)) {
    // the flag, the own r^2 and the own rows are loaded together (the rows
    // are used only when the flag is set)
    const int K0q = (K0 + 3) >> 2;
    float4 rows[8];
    if (PIPE) {  // piece e = (own token e >> 5, float4 e & 31): at most 64 x 32
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int e = tid + NT * u, i = min(e >> 5, cnt - 1), q = min(e & 31, K0q - 1);
        rows[u] = *reinterpret_cast<const float4*>(Ct + (long long)(c0 + i) * Kp + 4 * q);
      }
    }
    const float r2v = r2g[c0 + min(tid, cnt - 1)];
    r0_done = a.r0flag[b] != 0;
    if (r0_done) {
      if (K0 >= K) {  // the selection is R0 alone
        gather_share(false, K);
        return;
      }
      if (tid < cnt) {
        if (r2v != r2v) my_state = 2;  // NaN: a member of R0
        else my_r2 = r2v;
      }
      if (PIPE) {
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int e = tid + NT * u, i = e >> 5, q = e & 31;
          if (i < cnt && q < K0q) *reinterpret_cast<float4*>(ownC + i * ocs + 4 * q) = rows[u];
        }
      }
    }
  }
  if (tid == 0) misc[0] = 0;  // abort flag
  if (PIPE && tid < 4) npub[tid] = 0;
  __syncthreads();
  // the keys the first round merges: published by r0_kernel when it placed
  // R0 for workgroups of 64 tokens, else here (followed by a barrier)
  const unsigned bar0 = r0_done && ch == 64 ? 0u : 1u;
  if (bar0) {
    publish(1, K0 > 0 && !r0_done);
    image_barrier(a.bar + b, static_cast<unsigned>(G), a.err, misc);
    if (misc[0]) {
      gather_share(true, 0);
      return;
    }
  }

  int t = r0_done ? K0 : 0, fq = r0_done ? K0 : 0, round = 0;
  while (t < K) {
    // ============================================================ pool
    const bool forced = fq < K0;  // this round places members of R0
    uint64_t beta = 0;
    int pn = 0;
    {
      // Each workgroup published its top kPub keys (descending) and its
      // (kPub+1)-th key.  beta0 = the largest of those bounds; the keys above
      // it are compacted (in any order) and each is ranked by counting the
      // compacted keys above it.  Ranks are unique, so every workgroup builds
      // the same pool in the same order.
      const uint64_t* pub = a.pub + ((long long)b * 2 + ((round - 1) & 1)) * G * (kPub + 1);
      const int nk = G * kPub;  // at most 128 x 8 = 4 NT
      constexpr int XK = 4;
      uint64_t x[XK];
#pragma unroll
      for (int h = 0; h < XK; ++h) {
        const int e = tid + h * NT;
        x[h] = e < nk ? __hip_atomic_load(pub + (e >> 3) * (kPub + 1) + (e & 7), __ATOMIC_RELAXED,
                                          __HIP_MEMORY_SCOPE_AGENT)
                      : 0ull;  // kPub == 8
      }
      uint64_t bmax = 0;
      for (int ww = tid; ww < G; ww += NT) {
        const uint64_t k = __hip_atomic_load(pub + ww * (kPub + 1) + kPub, __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT);
        bmax = k > bmax ? k : bmax;
      }
      bmax = wave_max_key(bmax);
      if (lane == 0) bndk[wave] = bmax;
      if (tid == 0) misc[2] = 0;  // candidates above beta0
      __syncthreads();
      uint64_t beta0 = bndk[0];
      for (int q = 1; q < NT / 64; ++q) beta0 = bndk[q] > beta0 ? bndk[q] : beta0;
      double* cand = reinterpret_cast<double*>(merge);  // rank values of the keys above beta0
#pragma unroll
      for (int h = 0; h < XK; ++h)
        if (x[h] > beta0) cand[atomicAdd(&misc[2], 1)] = key_rank_value(x[h]);
      __syncthreads();
      const int nc = misc[2];
      if ((nc & 1) && tid == 0) cand[nc] = -1.0;  // pad to whole pairs (the buffer holds nk + 2)
      __syncthreads();
      uint64_t nextk = 0;  // the largest key left out of the pool by the cap
      for (int c = tid; c < nc; c += NT) {  // candidate c: its rank = number of candidates above it
        const double xc = cand[c];
        int r4[4] = {0, 0, 0, 0};
        int j = 0;
        for (; j + 8 <= nc; j += 8) {
          const double2 y0 = *reinterpret_cast<const double2*>(cand + j);
          const double2 y1 = *reinterpret_cast<const double2*>(cand + j + 2);
          const double2 y2 = *reinterpret_cast<const double2*>(cand + j + 4);
          const double2 y3 = *reinterpret_cast<const double2*>(cand + j + 6);
          r4[0] += above(xc, y0.x) + above(xc, y0.y);
          r4[1] += above(xc, y1.x) + above(xc, y1.y);
          r4[2] += above(xc, y2.x) + above(xc, y2.y);
          r4[3] += above(xc, y3.x) + above(xc, y3.y);
        }
        for (; j < nc; j += 2) {
          const double2 y = *reinterpret_cast<const double2*>(cand + j);
          r4[0] += above(xc, y.x) + above(xc, y.y);
        }
        const int rk = (r4[0] + r4[1]) + (r4[2] + r4[3]);
        if (rk < pcap) {
          const int i = rank_value_index(xc);
          midx[rk] = (i >= 0 && i < N) ? i : 0;
        } else if (rk == pcap) {
          nextk = rank_value_key(xc);
        }
      }
      nextk = wave_max_key(nextk);
      if (lane == 0) bndk[NT / 64 + wave] = nextk;
      __syncthreads();
      pn = min(nc, pcap);
      beta = beta0;
      for (int q = 0; q < NT / 64; ++q) beta = bndk[NT / 64 + q] > beta ? bndk[NT / 64 + q] : beta;
    }
    __syncthreads();
    // members: state, their block of S and (pipelined variant) their
    // columns (rows < t, written by their owners before the barrier; the
    // other variant reads them from global memory where it needs them).
    // Every global load of a thread is issued, at clamped (valid) addresses,
    // before its first LDS store, so the phase costs about one memory round
    // trip.
    if (pn > 0) {
      constexpr int CB = 12;  // column pieces per thread per batch
      // pipelined: member (tid >> 2) is loaded by four threads, float4 pieces
      // q = (tid & 3) + 4 u; pieces up to column tk = t rounded up to 8 are
      // written, with the columns at or past t set to zero (the round-start
      // product then needs no masks)
      const int tq = (t + 3) >> 2, tk4 = ((t + 7) & ~7) >> 2;
      // scalars of member tid
      const int ms = min(tid, pn - 1), is = midx[ms];
      const float pi = p[is], ni = nrm[is];
      const float r2m = t == 0 ? 0.0f : __hip_atomic_load(r2g + is, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const int mq = tid >> 2;
      const float* csrc = Ct + (long long)midx[min(mq, pn - 1)] * Kp;
      f32x4_t cv[CB];
      if (PIPE)
#pragma unroll
        for (int u = 0; u < CB; ++u)
          cv[u] = *reinterpret_cast<const f32x4_t*>(csrc + 4 * min((tid & 3) + 4 * u, max(tq - 1, 0)));
      // S among the members: rows m1 = 16 wave + q, column m2 = lane
      constexpr int QMAX = kMaxPool / 4;
      float sv[QMAX];
      const long long colS = midx[min(lane, pn - 1)];
      // S is symmetric: entries below the diagonal come from the mirror, and
      // lanes with nothing to load read the row's diagonal (one shared line)
#pragma unroll
      for (int q = 0; q < QMAX; ++q) {
        const int m1 = min(QMAX * wave + q, pn - 1);
        const long long row = midx[m1];
        sv[q] = S[row * N + (lane >= m1 ? colS : row)];
      }
      // stores
      if (tid < pn) {
        const float pc = (pi > 0.0f && pi <= 3.402823466e38f) ? pi : 0.0f;
        mp[tid] = pc;
        mn[tid] = ni;
        mqn[tid] = pc * ni;
        mr2[tid] = t == 0 ? (ni > 0.0f ? 1.0f : 0.0f) : r2m;
      }
      if (PIPE && mq < pn) {
        auto put = [&](int q, f32x4_t v) {  // piece q, zero at and past column t
          const int l = 4 * q;
          v.x = l < t ? v.x : 0.0f;
          v.y = l + 1 < t ? v.y : 0.0f;
          v.z = l + 2 < t ? v.z : 0.0f;
          v.w = l + 3 < t ? v.w : 0.0f;
          *reinterpret_cast<f32x4_t*>(pcol + mq * cs + l) = v;
        };
#pragma unroll
        for (int u = 0; u < CB; ++u) {
          const int q = (tid & 3) + 4 * u;
          if (q < tk4) put(q, cv[u]);
        }
        for (int q = (tid & 3) + 4 * CB; q < tk4; q += 4)  // long columns: the rest
          put(q, *reinterpret_cast<const f32x4_t*>(csrc + 4 * min(q, tq - 1)));
      }
      if (PIPE && t > 0)  // the own rows' columns t .. tk - 1 are zero too
        for (int e = tid; e < cnt * 8; e += NT) {
          const int i = e >> 3, l = t + (e & 7);
          if (l < 4 * tk4) ownC[i * ocs + l] = 0.0f;
        }
#pragma unroll
      for (int q = 0; q < QMAX; ++q) {
        const int m1 = QMAX * wave + q;
        if (m1 < pn && lane < pn && lane >= m1) {
          Rm[m1 * rs + lane] = sv[q];
          Rm[lane * rs + m1] = sv[q];
        }
      }
    }
    __syncthreads();
    // this round's coefficients start at zero, so the pick loop needs no masks
    for (int e = tid; e < pn * (us / 4); e += NT)
      reinterpret_cast<float4*>(U)[e] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (PIPE && tid == 0) {  // picks published, waves done with their tiles
      npub[0] = 0;
      npub[4] = 0;
    }
    if (t > 0 && pn > 0) {
      // The pool's residual Gram matrix, one float32 matrix-core product over
      // the t rows so far (columns t .. tk - 1 are zero):
      //   Rm[m][j] -= sum_l c_{l,m} c_{l,j}
      // Wave w computes the 32 x 32 tile (w >> 1, w & 1); in the pipelined
      // variant the own tokens' part (D) is computed by waves 1 to 3 while
      // wave 0 picks.
      const int tr = wave >> 1, tc = wave & 1, r = lane & 31, h = lane >> 5;
      float cur[16];  // current entries of this lane's results, read ahead
#pragma unroll
      for (int e = 0; e < 16; ++e)
        cur[e] = Rm[min(32 * tr + 8 * (e >> 2) + 4 * h + (e & 3), pn - 1) * rs + min(32 * tc + r, pn - 1)];
      f32x16_t acc;
      if (PIPE) {
        tile_product(pcol + min(32 * tr + r, pn - 1) * cs + 4 * h, pcol + min(32 * tc + r, pn - 1) * cs + 4 * h,
                     (t + 7) & ~7, acc);
      } else {  // the members' rows in global C (written before the last image barrier)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[e] = 0.0f;
        gtile_product<4>(Ct + (long long)midx[min(32 * tr + r, pn - 1)] * Kp,
                         Ct + (long long)midx[min(32 * tc + r, pn - 1)] * Kp, t, Kp, h, acc);
      }
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int m = 32 * tr + 8 * (e >> 2) + 4 * h + (e & 3), j = 32 * tc + r;
        if (m < pn && j < pn) Rm[m * rs + j] = cur[e] - acc[e];
      }
    }
    __syncthreads();

    // ============================================================ picks
    // Wave 0 alone, without barriers; lane m holds pool member m (r^2, key
    // inputs, active flag in registers).  For the k-th pick s,
    //   c_m = (Rm[s][m] - sum_{k'<k} U[s][k'] U[m][k']) / r_s,
    // U[m][k'] being member m's coefficient on the k'-th basis vector of
    // this round.  Each step issues all its LDS reads (Rm[s][m], row s of U
    // and the lane's own row of U, whose entries past the live ones are
    // zero) before using them, so a pick costs about one LDS round trip; the
    // products are only formed for the groups of 16 picks made so far.
    const int t0 = t;
    if (wave == 0) {
      int np = 0;
      const bool in = lane < pn;
      float r2v = in ? mr2[lane] : 0.0f;
      const float qnv = in ? mqn[lane] : 0.0f, pv = in ? mp[lane] : 0.0f, nv = in ? mn[lane] : 0.0f;
      const int iv = in ? midx[lane] : 0;
      bool actv = in;
      const float* u0 = U + min(lane, pcap - 1) * us;  // member `lane`'s row (zero past np)
      // the parts of the member's key that do not change during the round
      // (make_key's inputs: (qn qn) r2 is formed in make_key's order)
      const float qsq = qnv * qnv;
      const bool qpos = qnv > 0.0f;
      const uint32_t hip = ordered_bits(pv);
      const uint32_t klo = 0xffffffffu - static_cast<uint32_t>(iv);
      // One pick; NG = the number of groups of 16 picks made so far, so only
      // those groups of the two U rows are read and multiplied.  Returns
      // false when the round's picks are over.
      auto pick = [&](auto ngc) -> bool {
        constexpr int NG = decltype(ngc)::value;
        if (t >= K) return false;
        // the lane's own row does not depend on the pick: its reads are
        // issued first and complete under the argmax
        float4 xs[4 * NG + 1], y0[4 * NG + 1];
#pragma unroll
        for (int q = 0; q < 4 * NG; ++q) y0[q] = *reinterpret_cast<const float4*>(u0 + 4 * q);
        int s;
        uint64_t best = 0;
        if (forced) {  // the pool is the top of p in descending order
          s = np < min(pn, K0 - fq) ? np : -1;
        } else {
          // make_key's high word without branches
          const float s2 = qsq * r2v;
          const uint32_t hs = 0x80000000u | (s2 <= 3.402823466e38f ? __float_as_uint(s2) : 0u);
          const bool pos = (r2v > a.tau2) & qpos & (s2 > 0.0f);
          uint32_t khi = pos ? hs : hip;
          khi = actv ? khi : 0u;
          // the largest high word nearly always belongs to one member; only
          // a tie needs the low words (keys are distinct, so one member wins)
          const uint32_t mhi = wave_umax32(khi);
          const uint64_t tied = __ballot(khi == mhi);
          int sl;
          if (__builtin_popcountll(tied) == 1) {
            sl = static_cast<int>(__builtin_ctzll(tied));
            best = (static_cast<uint64_t>(mhi) << 32) |
                   static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(klo), sl));
          } else {
            const uint64_t kl = actv ? ((static_cast<uint64_t>(khi) << 32) | klo) : 0ull;
            best = wave_max_key(kl);
            sl = static_cast<int>(__builtin_ctzll(__ballot(kl == best)));
          }
          s = best > beta ? sl : -1;
        }
        // the previous picks are published here, one pick late, when their
        // writes have long completed and the release costs no wait
        if (PIPE && np > 0) __hip_atomic_store(npub, np, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
        if (s < 0) return false;
        // a pick among the own tokens (wave 0's lanes when 64 tokens per workgroup)
        if (PIPE && __builtin_amdgcn_readlane(iv, s) == c0 + lane) my_state = 2;
        const float rm = Rm[s * rs + min(lane, pn - 1)];
        const float* usr = U + s * us;
#pragma unroll
        for (int q = 0; q < 4 * NG; ++q) xs[q] = *reinterpret_cast<const float4*>(usr + 4 * q);
        const float r2s = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, r2v), s));
        const float ns = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, nv), s));
        // no basis vector when the unit residual is at most tau (or the row is zero)
        const bool skip = !(r2s > a.tau2 && ns > 0.0f);
        const float rinv = skip ? 0.0f : __builtin_amdgcn_rsqf(r2s);  // hardware reciprocal square root (1 ulp)
        const float r = r2s * rinv;
        if (lane == 0) {
          pslot[np] = s;
          prr[np] = rinv;
          pgain[np] = forced ? static_cast<uint32_t>(__builtin_amdgcn_readlane(__builtin_bit_cast(int, pv), s))
                             : static_cast<uint32_t>(best >> 32);
        }
        // dot over the picks so far (entries past np are zero)
        float d4[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int q = 0; q < 4 * NG; ++q) {
          d4[0] = fmaf(xs[q].x, y0[q].x, d4[0]);
          d4[1] = fmaf(xs[q].y, y0[q].y, d4[1]);
          d4[2] = fmaf(xs[q].z, y0[q].z, d4[2]);
          d4[3] = fmaf(xs[q].w, y0[q].w, d4[3]);
        }
        const float d = (d4[0] + d4[1]) + (d4[2] + d4[3]);
        if (in) {
          float c;
          if (lane == s) {
            c = r;
            actv = false;
          } else {
            c = (rm - d) * rinv;
            if (!skip) r2v = r2v - c * c;
          }
          U[lane * us + np] = c;
        }
        ++t;
        ++np;
        return true;
      };
      bool going = pick(IntC<0>{});
      while (going && np <= 16) going = pick(IntC<1>{});
      while (going && np <= 32) going = pick(IntC<2>{});
      while (going && np <= 48) going = pick(IntC<3>{});
      while (going) going = pick(IntC<4>{});
      if (PIPE) __hip_atomic_store(npub, np, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
      if (lane == 0) misc[3] = np;
      if (PIPE) __hip_atomic_store(pdone, round + 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
    } else if (PIPE) {
      // The own tokens are brought up to date while wave 0 picks (lane i
      // serves own token i).  First every pool member's row at the own
      // tokens, with the earlier rounds' part removed:
      //   W[m][i] = S[m][i] - sum_{l<t0} c_{l,m} c_{l,i},
      // four 32 x 32 tiles (wave 1 tile 0, wave 3 tile 1, wave 2 tiles 2 and
      // 3), each tile's entries of S loaded before its products.  The member
      // columns share their space with this round's own rows, so the
      // finisher starts once every tile is done.  Then wave 1 finishes, in
      // pick order, c_{k,i} = (W[pick_k][i] - sum_{k'<k} U[pick_k][k'] c_{k',i}) / r_k.
      if (pn > 0) {
        const int r = lane & 31, h = lane >> 5;
        for (int q = wave == 1 ? 0 : wave == 3 ? 1 : 2; q < (wave == 2 ? 4 : (wave == 1 ? 1 : 2)); ++q) {
          const int ti = q >> 1, tj = q & 1;
          const int col = c0 + min(32 * tj + r, cnt - 1);
          float sv[16];
#pragma unroll
          for (int e = 0; e < 16; ++e)
            sv[e] = S[(long long)midx[min(32 * ti + 8 * (e >> 2) + 4 * h + (e & 3), pn - 1)] * N + col];
          f32x16_t acc;
#pragma unroll
          for (int e = 0; e < 16; ++e) acc[e] = 0.0f;
          if (t0 > 0)
            tile_product(pcol + min(32 * ti + r, pn - 1) * cs + 4 * h, ownC + min(32 * tj + r, cnt - 1) * ocs + 4 * h,
                         (t0 + 7) & ~7, acc);
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const int m = 32 * ti + 8 * (e >> 2) + 4 * h + (e & 3);
            if (m < pn) Dm[m * wsd + 32 * tj + r] = sv[e] - acc[e];
          }
        }
      }
      if (lane == 0) __hip_atomic_fetch_add(dready, 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);  // once per wave
      if (wave == 1) {
        while (__hip_atomic_load(dready, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP) < 3) __builtin_amdgcn_s_sleep(1);
        float* cr = crow + lane * us;  // this round's own row: zero past the finished entries
        for (int e = 0; e < us / 4; ++e) reinterpret_cast<float4*>(cr)[e] = make_float4(0.f, 0.f, 0.f, 0.f);
        // The finisher stops once the picks are over and it has handled every
        // one of them, or when this round completes the selection (its update
        // is then never used).
        const int rtag = round + 1;
        int k = 0;
        int ready = 0;  // picks known to be published
        float csq = 0.0f;  // sum of the own token's squared new coefficients
        while (true) {
          bool over = false;
          if (k >= ready || (k & 7) == 0) {  // poll (and look for the end now and then)
            while (true) {
              if (__hip_atomic_load(pdone, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP) == rtag) {
                ready = __hip_atomic_load(npub, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP);
                over = ready <= k || t0 + ready >= K;
              } else {
                ready = __hip_atomic_load(npub, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP);
              }
              if (over || ready > k) break;
              __builtin_amdgcn_s_sleep(1);
            }
            if (over) break;
          }
          const int sk = pslot[k];
          const float* ur = U + sk * us;
          const float rk = prr[k];
          const float w0 = Dm[sk * wsd + lane];
          // all reads first (one LDS round trip), products only for the
          // groups of 16 rows finished so far
          float4 u4[kMaxPool / 4], c4[kMaxPool / 4];
#pragma unroll
          for (int j = 0; j < kMaxPool / 4; ++j) {
            u4[j] = *reinterpret_cast<const float4*>(ur + 4 * j);
            c4[j] = *reinterpret_cast<const float4*>(cr + 4 * j);
          }
          float e4[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
          for (int g = 0; g < kMaxPool / 16; ++g) {
            if (16 * g >= k) break;
#pragma unroll
            for (int j = 4 * g; j < 4 * g + 4; ++j) {
              e4[0] = fmaf(u4[j].x, c4[j].x, e4[0]); e4[1] = fmaf(u4[j].y, c4[j].y, e4[1]);
              e4[2] = fmaf(u4[j].z, c4[j].z, e4[2]); e4[3] = fmaf(u4[j].w, c4[j].w, e4[3]);
            }
          }
          const float v = w0 - ((e4[0] + e4[1]) + (e4[2] + e4[3]));
          const float c = v * rk;  // rk = 1 / r_k, zero when the pick adds no basis vector
          cr[k] = c;
          // the finished row goes straight to the own rows in LDS and to C
          ownC[lane * ocs + t0 + k] = c;
          if (lane < cnt) Ct[(long long)(c0 + lane) * Kp + t0 + k] = c;
          csq = fmaf(c, c, csq);
          ++k;
        }
        r2acc[lane] = csq;
      }
    }
    __syncthreads();
    const int np = misc[3];
    t = t0 + np;
    if (w == 0)  // the selection order and gains of this round
      for (int k = tid; k < np; k += NT) {
        a.order[(long long)b * K + t0 + k] = midx[pslot[k]];
        a.gain[(long long)b * K + t0 + k] =
            forced ? __uint_as_float(pgain[k]) : key_score(static_cast<uint64_t>(pgain[k]) << 32);
        if (a.order_map) a.order_map[(long long)b * K + t0 + k] = a.jmap[(long long)b * N + midx[pslot[k]]];
        // on a subset a greedy pick stands only if no token left out could beat it
        if (a.hout && !forced && pgain[k] <= a.hout[b]) a.uncert[b] = 1;
      }
    if (forced) fq += np;
    if (t >= K) {
      gather_share(false, t0);
      break;
    }

    // ============================================================ update
    // The round's new rows t0 .. t-1 on the own tokens:
    //   W_k     = S[pick_k][i] - sum_{l<t0} c_{l,pick_k} c_{l,i}            (dense)
    //   c_{k,i} = (W_k - sum_{k'<k} U[pick_k][k'] c_{k',i}) / r_k           (triangular)
    if (!PIPE) {  // own tokens picked this round (the merge buffer is free here)
      int* picked = reinterpret_cast<int*>(merge);
      for (int i = tid; i < ch; i += NT) picked[i] = 0;
      __syncthreads();
      for (int k = tid; k < np; k += NT) {
        const int i = midx[pslot[k]] - c0;
        if (i >= 0 && i < cnt) picked[i] = 1;
      }
      __syncthreads();
      if (tid < cnt && picked[tid]) my_state = 2;
    }
    if (!PIPE) {
    // W rows: S rows of the picks at the own tokens; row j = wave + 4 u,
    // token c = lane + 64 h.  Every load of a thread (at most 4 x 16, at
    // clamped valid addresses) is issued before its first store: one memory
    // round trip
    if (np > 0) {
      constexpr int HP = 4;  // 256 own tokens at most
      int row[kMaxPool / 4];
#pragma unroll
      for (int u = 0; u < kMaxPool / 4; ++u) row[u] = midx[pslot[min(wave + 4 * u, np - 1)]];
      float v[HP][kMaxPool / 4];
#pragma unroll
      for (int h = 0; h < HP; ++h)
        if (64 * h < cnt)  // (uniform)
#pragma unroll
          for (int u = 0; u < kMaxPool / 4; ++u)
            if (wave + 4 * u < np)  // (uniform)
              v[h][u] = S[(long long)row[u] * N + c0 + min(lane + 64 * h, cnt - 1)];
#pragma unroll
      for (int h = 0; h < HP; ++h)
        if (64 * h < cnt)
#pragma unroll
          for (int u = 0; u < kMaxPool / 4; ++u) {
            const int j = wave + 4 * u, c = lane + 64 * h;
            if (j < np && c < cnt) W[j * wsd + c] = v[h][u];
          }
    }
    __syncthreads();
    if (t0 > 0 && np > 0) {
      // dense part on matrix cores: 32 x 32 tiles (picks by own tokens), wave
      // w taking tiles w, w + 4, ...; the picks' and the own tokens' rows
      // both come from global C
      const int r = lane & 31, h = lane >> 5;
      const int nti = (np + 31) >> 5, ntj = (cnt + 31) >> 5;
      for (int tile = wave; tile < nti * ntj; tile += NT / 64) {
        const int ti = tile / ntj, tj = tile - ti * ntj;
        f32x16_t acc;
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[e] = 0.0f;
        gtile_product<4>(Ct + (long long)midx[pslot[min(32 * ti + r, np - 1)]] * Kp,
                         Ct + (long long)(c0 + min(32 * tj + r, cnt - 1)) * Kp, t0, Kp, h, acc);
        // entry e of this lane: pick 32 ti + 8 (e >> 2) + 4 h + (e & 3), own token 32 tj + r
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int m = 32 * ti + 8 * (e >> 2) + 4 * h + (e & 3), c = 32 * tj + r;
          if (m < np && c < cnt) W[m * wsd + c] -= acc[e];
        }
      }
      __syncthreads();
    }
    // triangular part in blocks of 8 rows: one thread per own token solves
    // the block in registers, then every thread updates the later rows
    constexpr int TB = 8;
    for (int j0 = 0; j0 < np; j0 += TB) {
      const int nb = min(TB, np - j0);
      float lblk[TB][TB];  // lblk[q][q2] = coefficient of pick j0+q on row t0+j0+q2
      float rblk[TB];
#pragma unroll
      for (int q = 0; q < TB; ++q) {
        const float* lr = U + pslot[min(j0 + q, np - 1)] * us + j0;
        const float4 a0 = *reinterpret_cast<const float4*>(lr);
        const float4 a1 = *reinterpret_cast<const float4*>(lr + 4);
        lblk[q][0] = a0.x; lblk[q][1] = a0.y; lblk[q][2] = a0.z; lblk[q][3] = a0.w;
        lblk[q][4] = a1.x; lblk[q][5] = a1.y; lblk[q][6] = a1.z; lblk[q][7] = a1.w;
        rblk[q] = prr[min(j0 + q, np - 1)];
      }
      for (int c = tid; c < cnt; c += NT) {
        float x[TB];
#pragma unroll
        for (int q = 0; q < TB; ++q) x[q] = q < nb ? W[(j0 + q) * wsd + c] : 0.0f;
#pragma unroll
        for (int q = 0; q < TB; ++q) {
          float v = x[q];
#pragma unroll
          for (int q2 = 0; q2 < q; ++q2) v = fmaf(-lblk[q][q2], x[q2], v);
          x[q] = q < nb ? v * rblk[q] : 0.0f;  // rblk = 1 / r, zero when the pick adds no basis vector
        }
#pragma unroll
        for (int q = 0; q < TB; ++q)
          if (q < nb) W[(j0 + q) * wsd + c] = x[q];
      }
      __syncthreads();
      if (j0 + nb < np) {
        if (ch == 64) {  // one token per lane
          const int c = lane;
          float x[TB];
#pragma unroll
          for (int q = 0; q < TB; ++q) x[q] = q < nb ? W[(j0 + q) * wsd + c] : 0.0f;
          for (int j2 = j0 + nb + wave; j2 < np; j2 += 4 * (NT / 64)) {
            float4 l0[4], l1[4];
            float v[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              const int jr = min(j2 + (NT / 64) * u, np - 1);
              const float* lr = U + pslot[jr] * us + j0;
              l0[u] = *reinterpret_cast<const float4*>(lr);
              l1[u] = *reinterpret_cast<const float4*>(lr + 4);
              v[u] = W[jr * wsd + c];
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              const float lq[TB] = {l0[u].x, l0[u].y, l0[u].z, l0[u].w, l1[u].x, l1[u].y, l1[u].z, l1[u].w};
#pragma unroll
              for (int q = 0; q < TB; ++q)
                if (q < nb) v[u] = fmaf(-lq[q], x[q], v[u]);
            }
#pragma unroll
            for (int u = 0; u < 4; ++u)
              if (j2 + (NT / 64) * u < np && c < cnt) W[(j2 + (NT / 64) * u) * wsd + c] = v[u];
          }
        } else {
          // lane l serves own tokens l, l + 64, ... (CP at most); the block's
          // solved rows at those tokens stay in registers, and each group of
          // four later rows is read from U once for all of them
          constexpr int CP = 4;  // 256 own tokens at most
          float x[CP][TB];
#pragma unroll
          for (int pc = 0; pc < CP; ++pc)
#pragma unroll
            for (int q = 0; q < TB; ++q)
              x[pc][q] = (64 * pc < cnt && q < nb) ? W[(j0 + q) * wsd + min(lane + 64 * pc, ch - 1)] : 0.0f;
          for (int j2 = j0 + nb + wave; j2 < np; j2 += 4 * (NT / 64)) {
            float4 l0[4], l1[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              const int jr = min(j2 + (NT / 64) * u, np - 1);
              const float* lr = U + pslot[jr] * us + j0;
              l0[u] = *reinterpret_cast<const float4*>(lr);
              l1[u] = *reinterpret_cast<const float4*>(lr + 4);
            }
#pragma unroll
            for (int pc = 0; pc < CP; ++pc) {
              if (64 * pc >= cnt) break;  // (uniform)
              const int c = lane + 64 * pc;  // past cnt (the last pass): computed from valid entries, not stored
              float v[4];
#pragma unroll
              for (int u = 0; u < 4; ++u) v[u] = W[min(j2 + (NT / 64) * u, np - 1) * wsd + c];
#pragma unroll
              for (int u = 0; u < 4; ++u) {
                const float lq[TB] = {l0[u].x, l0[u].y, l0[u].z, l0[u].w, l1[u].x, l1[u].y, l1[u].z, l1[u].w};
#pragma unroll
                for (int q = 0; q < TB; ++q)
                  if (q < nb) v[u] = fmaf(-lq[q], x[pc][q], v[u]);
              }
#pragma unroll
              for (int u = 0; u < 4; ++u)
                if (j2 + (NT / 64) * u < np && c < cnt) W[(j2 + (NT / 64) * u) * wsd + c] = v[u];
            }
          }
        }
        __syncthreads();
      }
    }
    }  // !PIPE
    // new rows to global memory (token-major) and the own r2 (pipelined:
    // the finisher wrote the rows and summed the squares already)
    const bool live = tid < cnt && my_state != 2;
    if (PIPE) {
      if (live) my_r2 = my_r2 - r2acc[tid];
    } else {
      const int total = np * cnt;
      for (int e = tid; e < total; e += NT) {
        const int c = e / np, jj = e - c * np;
        Ct[(long long)(c0 + c) * Kp + t0 + jj] = W[jj * wsd + c];
      }
      if (live)
        for (int jj = 0; jj < np; ++jj) {
          const float c = W[jj * wsd + tid];
          my_r2 = my_r2 - c * c;
        }
    }
    if (live) __hip_atomic_store(r2g + my_i, my_r2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    publish(round & 1, fq < K0);
    ++round;
    image_barrier(a.bar + b, static_cast<unsigned>((round + bar0) * G), a.err, misc);
    if (misc[0]) {
      gather_share(true, 0);
      break;
    }
  }
}

// ------------------------------------------------------------------ restore
// One block per image: the K kept indices in ascending order (rank by count;
// indices are distinct).  After an aborted selection (error flag set) every
// index is -1.
__global__ __launch_bounds__(NT) void restore_kernel(const SelectArgs a) {
  extern __shared__ int ord[];
  const int b = blockIdx.x, K = a.K;
  if (__hip_atomic_load(a.err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0) {
    for (int i = threadIdx.x; i < K; i += NT) a.idx_out[(long long)b * K + i] = -1;
    return;
  }
  for (int i = threadIdx.x; i < K; i += NT) ord[i] = a.order[(long long)b * K + i];
  __syncthreads();
  for (int i = threadIdx.x; i < K; i += NT) {
    const int v = ord[i];
    int rank = 0;
    for (int j = 0; j < K; ++j) rank += ord[j] < v;
    a.idx_out[(long long)b * K + rank] = v;
  }
}

std::atomic<int> g_images_per_launch{0};

struct DeviceInfo {
  int cus = 0;
};

DeviceInfo& device_info() {
  static DeviceInfo info[64];
  int dev = 0;
  (void)hipGetDevice(&dev);
  DeviceInfo& d = info[dev & 63];
  if (d.cus == 0) {
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) == hipSuccess) d.cus = prop.multiProcessorCount;
  }
  return d;
}

}  // namespace

void set_select_images_per_launch(int n) { g_images_per_launch.store(n > 0 ? n : 0); }

hipError_t launch_select_clear(const SelectArgs& a, hipStream_t s) {
  return launch_kernel("select_clear", select_clear_kernel, dim3(1), dim3(64), 0, s, a);
}

// Picks the tokens per workgroup (hence workgroups per image) and the pool
// capacity within the LDS budget, then runs the images in as few launches as
// keep every launch's workgroups resident at once (the occupancy check
// below).  The image barriers rely on that residency; if other work on the
// device ever held them off for longer than their bounded wait, the launch
// ends early with the error flag set and restore_kernel reports -1 indices.
hipError_t launch_select(SelectArgs& a, hipStream_t s) {
  const int K = a.K, N = a.N;
  constexpr int kMaxLds = 160 * 1024;
  constexpr int kMinPipePool = 48;  // below this the pipelined variant loses more to extra rounds
  const int cus = device_info().cus > 0 ? device_info().cus : 1;
  int chosen_ch = 0, chosen_pcap = 0, chosen_G = 0, chosen_bytes = 0, per_cu = 0;
  bool chosen_pipe = false;
  for (int ch : {64, 128, 256}) {
    const int G = (N + ch - 1) / ch;
    if (G > 128) continue;
    bool pipe = ch == 64;
    int pcap = kMaxPool;
    while (pcap > 8 && lds_layout(K, G, ch, pcap, pipe).bytes > kMaxLds) pcap -= 8;
    if (pipe && pcap < kMinPipePool) {
      pipe = false;
      pcap = kMaxPool;
      while (pcap > 8 && lds_layout(K, G, ch, pcap, false).bytes > kMaxLds) pcap -= 8;
    }
    const int bytes = lds_layout(K, G, ch, pcap, pipe).bytes;
    if (bytes > kMaxLds) continue;
    const void* fn = pipe ? reinterpret_cast<const void*>(select_kernel<true>)
                          : reinterpret_cast<const void*>(select_kernel<false>);
    if (bytes > 65536) {
      hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
      if (e != hipSuccess) return e;
    }
    int pc = 0;
    hipError_t e = pipe ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&pc, select_kernel<true>, NT, bytes)
                        : hipOccupancyMaxActiveBlocksPerMultiprocessor(&pc, select_kernel<false>, NT, bytes);
    if (e != hipSuccess) return e;
    if (pc <= 0) continue;
    chosen_ch = ch;
    chosen_pcap = pcap;
    chosen_G = G;
    chosen_bytes = bytes;
    chosen_pipe = pipe;
    per_cu = pc;
    if ((long long)a.B * G <= (long long)pc * cus) break;  // every image at once
  }
  if (per_cu <= 0) return hipErrorInvalidConfiguration;
  a.ch = chosen_ch;
  a.G = chosen_G;
  a.pcap = chosen_pcap;
  if (a.gV) {  // the order must fit where the pool's Gram matrix was
    const Lds L = lds_layout(K, chosen_G, chosen_ch, chosen_pcap, chosen_pipe);
    const int rw = 4 * chosen_pcap * (L.rs > L.ws ? L.rs : L.ws);
    if (4 * ((K + 7) & ~7) > rw || (a.row_bytes & 15) != 0) a.gV = nullptr;
  }
  int per_launch = static_cast<int>(((long long)per_cu * cus) / chosen_G);
  if (per_launch < 1) return hipErrorInvalidConfiguration;
  const int cap = g_images_per_launch.load();
  if (cap > 0 && cap < per_launch) per_launch = cap;
  if (r0_by_factor(a.K0) && !a.no_r0_kernel) {
    const int rb = r0_layout(a.K0).bytes;
    if (rb > 65536) {
      const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(r0_kernel),
                                               hipFuncAttributeMaxDynamicSharedMemorySize, rb);
      if (e != hipSuccess) return e;
    }
    const hipError_t e = launch_kernel(a.fallback ? "select_r0_full" : a.tier2 ? "select_r0_t2" : "select_r0", r0_kernel,
                                       dim3((a.N + 63) / 64, a.B), dim3(NT),
                                       static_cast<size_t>(rb), s, a);
    if (e != hipSuccess) return e;
  }
  for (int b0 = 0; b0 < a.B; b0 += per_launch) {
    const int nb = a.B - b0 < per_launch ? a.B - b0 : per_launch;
    const hipError_t e =
        chosen_pipe ? launch_kernel(a.fallback ? "select_full" : a.tier2 ? "select_t2" : "select", select_kernel<true>,
                                    dim3(nb * chosen_G),
                                    dim3(NT), static_cast<size_t>(chosen_bytes), s, a, b0)
                    : launch_kernel(a.fallback ? "select_full" : a.tier2 ? "select_t2" : "select", select_kernel<false>,
                                    dim3(nb * chosen_G),
                                    dim3(NT), static_cast<size_t>(chosen_bytes), s, a, b0);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_restore(const SelectArgs& a, hipStream_t s) {
  return launch_kernel("restore", restore_kernel, dim3(a.B), dim3(NT), sizeof(int) * a.K, s, a);
}

}  // namespace mapk
