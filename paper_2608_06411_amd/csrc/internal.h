// Internal declarations shared by the host dispatch and the HIP kernels of
// libmap.  Nothing here is part of the public ABI (include/map.h).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <tuple>
#include <utility>

#include "map.h"

namespace mapk {

// ---------------------------------------------------------------- bf16
// Storage type of a bfloat16 value: its 16 raw bits.
typedef uint16_t bf16_t;

__device__ __forceinline__ float bf16_to_f32(bf16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// float -> bf16, round to nearest even (NaN stays NaN).
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<bf16_t>((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<bf16_t>(u >> 16);
}

template <typename T> __device__ __forceinline__ float to_f32(T v);
template <> __device__ __forceinline__ float to_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ float to_f32<bf16_t>(bf16_t v) { return bf16_to_f32(v); }

template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16_t from_f32<bf16_t>(float v) { return f32_to_bf16(v); }

// ---------------------------------------------------------------- launch
// Every kernel goes through launch_kernel.  While map_timing is enabled the
// registry hands out a pair of events, which the runtime stamps with the
// dispatch's own start and end (hipExtLaunchKernel); otherwise both are null
// and the launch is a plain one.
struct LaunchEvents {
  hipEvent_t start = nullptr, stop = nullptr;
};
LaunchEvents timing_events(const char* name);

template <typename Tuple, size_t... I>
inline void kernel_argv(void** argv, Tuple& t, std::index_sequence<I...>) {
  ((argv[I] = static_cast<void*>(&std::get<I>(t))), ...);
}

template <typename... P, typename... A>
hipError_t launch_kernel(const char* name, void (*kernel)(P...), dim3 grid, dim3 block, size_t lds_bytes,
                         hipStream_t s, A... args) {
  static_assert(sizeof...(P) == sizeof...(A), "kernel argument count");
  std::tuple<P...> vals{args...};
  void* argv[sizeof...(P)];
  kernel_argv(argv, vals, std::index_sequence_for<P...>{});
  const LaunchEvents ev = timing_events(name);
  return hipExtLaunchKernel(reinterpret_cast<const void*>(kernel), grid, block, argv, lds_bytes, s, ev.start,
                            ev.stop, 0);
}

// ---------------------------------------------------------------- GEMM
// C = epilogue(A * B^T): A [M][K] and B [N][K] row-major (K contiguous),
// float32 accumulation on the matrix cores.  Several independent problems
// share one launch; each may be batched.
enum EpiMode : int {
  EPI_BIAS_GELU = 0,  // C[m][n] = GELU(acc + bias[n]), stored as T
  EPI_BIAS = 1,       // C[m][n] = acc + bias[n] (no bias when null), stored as T
  EPI_COSINE = 2,     // S[m][n] = acc * rs[m] * rs[n] (float32), mirrored; A == B
  EPI_ROPE = 3,       // out[m][:] = RoPE(acc[m][:] + rope_bias) (float32) with the row's cos/sin
  EPI_PARTIAL = 4,    // the raw float32 accumulators of a K range, for gram_reduce (bf16 direct-load kernel)
  // the training step's and the decoder layer's products:
  EPI_F32 = 5,        // C[m][n] = acc, stored as float32
  EPI_GELU2 = 6,      // v = acc + bias[n]: C[m][n] = GELU(v) and aux[m][n] = GELU'(v), both stored as T
  EPI_MUL = 7,        // C[m][n] = acc * aux[m][n] (aux of type T, leading dimension ldc), stored as T
  EPI_RESID = 8,      // C[m][n] = acc + aux[m][n] (a residual connection), stored as T
};
// Epilogues written lane by lane in registers (no staging): every kernel runs them.
__host__ __device__ inline bool epi_direct(int e) { return e >= EPI_F32 && e <= EPI_RESID; }

struct GemmProblem {
  const void* A;
  const void* B;
  void* C;
  long long strideA, strideB, strideC;  // per batch item, in elements
  int M, N, K, lda, ldb, ldc;
  int batch;
  int epi;
  const void* bias;        // EPI_BIAS*: [N], element type T
  const float* rs;         // EPI_COSINE: [batch][M] reciprocal norms
  const float2* rope_cs;   // EPI_ROPE: [M][N/2] (cos, sin) per row and pair
  const float* rope_bias;  // EPI_ROPE: [N] float32 added before the rotation (may be null)
  int triangular;          // EPI_COSINE, EPI_PARTIAL: only tiles with tile_n >= tile_m
  // rows of A and B through index maps ([batch][mapStride]; null: row m is row m)
  const int32_t* mapA;
  const int32_t* mapB;
  long long mapStride;
  int ksplit;              // EPI_PARTIAL: K ranges per tile (K / ksplit each, a multiple of 256)
  int kchunk;              // EPI_PARTIAL, if > 0: ranges of kchunk (a multiple of 256), the last shorter
  const int32_t* run_if;   // [batch] batch items whose flag is 0 are skipped (null: none)
  void* aux;               // EPI_GELU2: second output; EPI_MUL, EPI_RESID: the factor or the residual
                           // (each [M][ldc] of type T)
  // filled by the host helper
  int tiles_m, tiles_n, tiles_tri, tiles_per_batch, tile_begin;
};

constexpr int kMaxGemmProblems = 6;
struct GemmBatch {
  GemmProblem p[kMaxGemmProblems];
  int count;
  int total_tiles;
  int first_tiles;  // tiles dispatched before the rest (0: one class)
  // bf16 direct-load launches only: norm_blocks more workgroups, dispatched
  // after every tile (on compute units the tiles leave idle), write the row
  // norms of norm_V [norm_rows][norm_D] and their reciprocals, summed in
  // prep's order (bitwise the same values)
  int norm_blocks;
  const void* norm_V;
  int norm_rows, norm_D;
  float* norms;
  float* ninv;
  // 256 x 256 tiles only (gemm_big_tiles): when norm_tiles = q + 1 > 0, the
  // tiles of problem q (batch 1) in its first tile column also write the row
  // norms of its A rows and their reciprocals (norm_blocks must be 0)
  int norm_tiles;
};

void gemm_finalize(GemmBatch& g);  // computes the tile counts
bool gemm_direct_loads(map_dtype dt, const GemmBatch& g);  // launch_gemm would use the direct-load kernel
bool gemm_big_tiles(map_dtype dt, const GemmBatch& g);     // ... with 256 x 256 tiles
hipError_t launch_gemm(map_dtype dt, const GemmBatch& g, const char* name, hipStream_t s);
// The projection with the RoPE epilogue (every problem EPI_ROPE, at most two):
// a K-split kernel for bf16 and N <= 128, else launch_gemm.
hipError_t launch_proj_rope(map_dtype dt, const GemmBatch& g, const char* name, hipStream_t s);
// The split-K sums of an EPI_PARTIAL problem (finalized, ksplit > 1) in a
// fixed order, then the cosine epilogue into out (symmetric, ldc, rs as in
// EPI_COSINE).
hipError_t launch_gram_reduce(const GemmProblem& partial, float* out, int ldc, const float* rs, hipStream_t s,
                              const char* name = "gram_reduce");

// ---------------------------------------------------------------- subset
// The candidate subset J of map_prune (R0 plus the largest score bounds),
// compacted in token order, and the largest bound key left out.
struct SubsetArgs {
  const float* p;       // [B][N]
  const float* norms;   // [B][N]
  const float* ninv;    // [B][N]
  int32_t* jmap;        // [B][Nc] token of each subset position, ascending
  float* pJ;            // [B][Nc]
  float* nJ;            // [B][Nc]
  float* ninvJ;         // [B][Nc]
  uint32_t* hout;       // [B] high word of the largest bound key outside J
  int32_t* uncert;      // [B] cleared here; set by the selection when a pick is not certified
  unsigned int* clear_bar;  // [B] barrier counters of the full selection behind the subset, cleared here
  int32_t* clear_r0flag;    // [B] its R0 flags, cleared here (it places R0 in its own rounds)
  // optional (a second, larger subset): image b is taken only when
  // run_if[b] != 0; the others get uncert = 0 and nothing else
  const int32_t* run_if;
  int tier2;                // timing names of the second subset's launches
  int B, N, Nc, K0;
  float tau2;
};
constexpr int kSubsetMaxN = 8192;
hipError_t launch_subset(const SubsetArgs& a, hipStream_t s);

// ---------------------------------------------------------------- prep
// Row norms of the visual tokens (and their reciprocals) plus the RoPE
// cos/sin table of every visual and question token.
struct PrepArgs {
  const void* V;          // [rowsV][D]
  int rowsV, D;
  float* norms;           // [rowsV]
  float* ninv;            // [rowsV]
  const int32_t* pos_v;   // [rowsV] (may be null when the table is not needed)
  const int32_t* pos_t;   // [rowsT]
  int rowsT;
  int half;               // d_p / 2
  float2* cs_v;           // [rowsV][half]
  float2* cs_t;           // [rowsT][half]
  double inv_freq[64];    // theta^(-2i/d_p), computed on the host in float64
  // the folded second layer and projection (one pair per modality):
  //   tdst[s] = tsrc[s]^T           (square, tn x tn, element type of the call)
  //   fout[s][o] = sum_k fw[s][o][k] fb[s][k]   (o < frows, k < fcols, float32)
  const void* tsrc[2];
  void* tdst[2];
  int tn;
  const void* fw[2];
  const void* fb[2];
  float* fout[2];
  int frows, fcols;
  uint64_t* clear[2];     // optional: arrays zeroed by the launch (the scoring's exchange words)
  long long nclear[2];
};
hipError_t launch_prep(map_dtype dt, const PrepArgs& a, bool norms, bool table, bool fold, hipStream_t s);

// ---------------------------------------------------------------- finite check
// The device flag of this device (nullptr on failure), and one scan that sets
// it when `count` elements of elem_bytes (2: bf16, 4: float32) at p hold an
// infinity or a NaN.
int* finite_flag();
hipError_t launch_finite_check(const void* p, long long count, int elem_bytes, int* flag, hipStream_t s);

// ---------------------------------------------------------------- score
struct ScoreArgs {
  const float* q;         // [sum_M][d_p] (after RoPE)
  const float* k;         // [B][N][d_p]  (after RoPE)
  float* logits;          // [sum_M][N]: written by the two-launch form, and by the
                          // one-launch form when store_logits (the training step)
  float2* partial;        // [sum_M][nblk] (running max, sum of exp) per key block
  unsigned int* clear_bar; // optional: selection barrier counters [B] to zero
  int32_t* clear_err;      // optional: selection error flag to zero (set when the
                           // one-launch form's barrier gives up)
  float* p_out;           // [B][N]
  // the one-launch form (null pp, or score_one_launch false: the two-launch
  // form) exchanges the pairs
  // in `partial` and each question chunk's share of p in `pp` as 64-bit
  // words; both arrays are zeroed before the launch (prep does it)
  uint64_t* pp;           // [q_off[B]][N], rows q_off[b] + chunk
  int store_logits;
  int B, N, d_p, nblk;
  int t_off[MAP_MAX_BATCH + 1];
  int q_off[MAP_MAX_BATCH + 1];  // chunks of 16 queries before image b (set by launch_score)
};
// Rows of ScoreArgs::pp a call with these question lengths needs at most.
inline long long score_pp_rows(int B, int sumM) { return (sumM + 15) / 16 + B; }
hipError_t launch_score(const ScoreArgs& a, hipStream_t s);
// Whether launch_score takes the one-launch form for these question lengths
// (t_off host, [B + 1]); its exchange arrays must then be zeroed first.
bool score_one_launch(int B, int N, const int32_t* t_off);

// ---------------------------------------------------------------- select
struct SelectArgs {
  const float* p;        // [B][N]
  const float* S;        // [B][N][N]
  const float* norms;    // [B][N]
  float* C;              // [B][N][Kp] basis coefficients, Ct[i][t] = c_{t,i}
  float* r2;             // [B][N]    squared unit residuals
  uint64_t* pub;         // [B][2][G][kPub+1] published keys
  unsigned int* bar;     // [B] barrier counters
  int32_t* err;          // [1] set when a barrier wait gives up
  int32_t* order;        // [B][K]
  float* gain;           // [B][K]
  int32_t* idx_out;      // [B][K] ascending
  int32_t* r0flag;       // [B] 1 where R0 was placed by one factorisation
  // map_prune: the gather of the kept rows at the end of the selection
  // (gV null: none; launch_select clears it when the order does not fit in LDS)
  const void* gV;         // [B][N] rows of row_bytes (the visual tokens)
  const int32_t* gpos;    // [B][N] positions
  void* gV_out;           // rows of row_bytes: image b's kept row k at row b K + out_off[b] + k
  int32_t* gpos_out;      // positions, indexed like gV_out's rows
  int row_bytes;
  // layer-0 assembly (qT non-null): image b's question rows follow its kept
  // rows, from row b K + out_off[b] + K on (out_off = q_off: the language
  // model's input, packed)
  const void* qT;         // [sum M] question rows of row_bytes
  const int32_t* qpos;    // [sum M]
  int out_off[MAP_MAX_BATCH];
  int q_off[MAP_MAX_BATCH + 1];
  // map_prune on a candidate subset: N is the subset's size, token k of the
  // subset is token jmap[b][k] of the image (Ng tokens in gV and gpos)
  const int32_t* jmap;    // [B][N] ascending (null: no subset)
  int32_t* order_map;     // [B][K] the selection order as image tokens (may be null)
  const uint32_t* hout;   // [B] greedy picks must key above it (null: no check)
  int32_t* uncert;        // [B] set to 1 when a greedy pick does not
  const int32_t* run_if;  // [B] images whose flag is 0 are skipped (null: none)
  int Ng;
  int fallback;           // the launches are the full selection behind a subset (timing names)
  int tier2;              // the launches select on the second, larger subset (timing names)
  int no_r0_kernel;       // R0 is placed by the selection's own rounds (r0flag must read 0)
  int B, N, K, K0, G, ch, pcap;
  float tau2;
};
constexpr int kPub = 8;  // keys each workgroup publishes per round
// At most this many images per selection launch (0: as many as can be
// resident at once); map_set_select_images_per_launch sets it.
void set_select_images_per_launch(int n);
hipError_t launch_select_clear(const SelectArgs& a, hipStream_t s);
hipError_t launch_select(SelectArgs& a, hipStream_t s);
hipError_t launch_restore(const SelectArgs& a, hipStream_t s);

// ---------------------------------------------------------------- gather
struct GatherArgs {
  const void* V;           // [B][N][D]
  const int32_t* pos_v;    // [B][N]
  const int32_t* order;    // [B][K] selection order (distinct indices)
  const int32_t* err;      // selection error flag (set: every index is -1)
  int32_t* idx_out;        // [B][K] kept indices, ascending (written here)
  void* V_out;             // image b's kept row k at row b K + out_off[b] + k
  int32_t* pos_out;        // indexed like V_out's rows
  int B, N, K, row_bytes;
  // layer-0 assembly (qT non-null), as in SelectArgs
  const void* qT;
  const int32_t* qpos;
  int out_off[MAP_MAX_BATCH];
  int q_off[MAP_MAX_BATCH + 1];
};
hipError_t launch_gather(const GatherArgs& a, hipStream_t s);

// The language model's layer-0 input: per image its K kept rows, then its
// question rows, packed (image b from row b K + t_off[b]).
struct AssembleArgs {
  const void* V_out;      // [B][K] rows of row_bytes
  const int32_t* pos_out; // [B][K]
  const void* T;          // [sum M] rows of row_bytes
  const int32_t* pos_t;   // [sum M]
  void* X;                // [B K + sum M] rows of row_bytes
  int32_t* pos_x;         // [B K + sum M]
  int B, K, row_bytes, max_rows;
  int t_off[MAP_MAX_BATCH + 1];
};
hipError_t launch_assemble(const AssembleArgs& a, hipStream_t s);

// ---------------------------------------------------------------- training step
// The gradient of the batch-mean KL divergence from the teacher to p_hat,
// from the logits back to the projections' inputs (before RoPE).
struct TrainArgs {
  const float* logits;     // [sum_M][N] (scaled by 1/sqrt(d_p))
  const float2* partial;   // [sum_M][nblk] per-block (max, sum of exp) of the logits
  const float* p_hat;      // [B][N]
  const float* p_star;     // [B][N] teacher distributions
  float* loss;             // [B] each image's divergence
  float* G;                // [sum_M][N] dL/dlogits / sqrt(d_p)
  const float* q;          // [sum_M][d_p] queries after RoPE
  const float* k;          // [B N][d_p] keys after RoPE
  const float2* cs_v;      // [B N][d_p / 2] RoPE (cos, sin)
  const float2* cs_t;      // [sum_M][d_p / 2]
  float* dq_part;          // [nch][sum_M][d_p] token-chunk partials of dL/dq
  void* dk_rows;           // [B N][kdp] dL/dz of the keys, element type of the call (zero past d_p)
  void* dk_cols;           // [d_p][ldv] the same, tokens contiguous (zero padded)
  void* dq_rows;           // [sum_M][kdp]
  void* dq_cols;           // [d_p][ldt]
  int B, N, d_p, nblk, nch, ldv, ldt, kdp;
  float inv_B, scale;      // 1 / B, 1 / sqrt(d_p)
  int t_off[MAP_MAX_BATCH + 1];
};
hipError_t launch_train_grads(map_dtype dt, const TrainArgs& a, hipStream_t s);

// X = dz^T h per branch from token-chunk partials (see train.hip).
struct XReduceArgs {
  const float* part[2];  // [nc][d_p][D_h]
  void* X[2];            // [d_p][D_h]
  void* XT[2];           // [D_h][kdp]
  int nc[2];
  int d_p, D_h, kdp;
};
hipError_t launch_x_reduce(map_dtype dt, const XReduceArgs& r, hipStream_t s);

// dst[c][r] = src[r][c] (r < rows, c < cols), zero for rows <= r < ldd.
struct TransposeJob {
  const void* src;
  void* dst;
  int rows, cols, lds, ldd;
  int tile_begin;  // filled by transpose_finalize
};
constexpr int kMaxTransposeJobs = 8;
struct TransposeBatch {
  TransposeJob job[kMaxTransposeJobs];
  int count, total_tiles;
};
void transpose_finalize(TransposeBatch& t);
hipError_t launch_transpose(map_dtype dt, const TransposeBatch& t, const char* name, hipStream_t s);

// out[r] = sum_{c < cols} src[r][c] (element type of the call), float32.
struct RowsumJob {
  const void* src;
  float* out;
  int rows, cols, ld;
  int row_begin;  // filled by launch_rowsum
};
struct RowsumBatch {
  RowsumJob job[4];
  int count;
};
hipError_t launch_rowsum(map_dtype dt, RowsumBatch& t, hipStream_t s);

// Per branch s (0 visual, 1 text): db2[s] = W[s]^T csum[s] and the rank-one
// term dW[s] += csum[s] b2[s]^T of the projection's gradient.
struct FinishArgs {
  const void* W[2];    // [d_p][D_h] W_K, W_Q
  const void* b2[2];   // [D_h]
  const float* csum[2];  // [d_p] sum over tokens of dL/dz
  float* db2[2];       // [D_h]
  float* dW[2];        // [d_p][D_h]
  int D_h, d_p;
};
hipError_t launch_finish(map_dtype dt, const FinishArgs& f, hipStream_t s);

// ---------------------------------------------------------------- decoder layer
// The language model's layer over the pruned input (LLaMA decoder layer,
// bf16): the kernels around the matrix-core products.
struct DecoderArgs {
  const void* X;          // [R][d] layer input (the residual of the attention block)
  const int32_t* pos;     // [R] positional index of each row
  const void* attn_norm;  // [d]
  const void* ffn_norm;   // [d]
  void* h;                // [R][d] RMSNorm output (attention block, then MLP block)
  void* qkv;              // [R][3 d] q, k (rotated in place), v
  void* o;                // [R][d] attention output
  void* x1;               // [R][d] after the attention block
  void* gu;               // [R][2 ff] gate, then up
  void* act;              // [R][ff] SiLU(gate) * up
  int R, d, n_heads, head_dim, ff, B, max_len;
  float eps;
  double inv_freq[64];    // theta^(-2i/head_dim), float64
  int seq_off[MAP_MAX_BATCH + 1];
};
hipError_t launch_rmsnorm(const DecoderArgs& a, const void* x, const void* g, void* out, hipStream_t s);
hipError_t launch_rope_qkv(const DecoderArgs& a, hipStream_t s);
hipError_t launch_attention(const DecoderArgs& a, hipStream_t s);
hipError_t launch_silu_mul(const DecoderArgs& a, hipStream_t s);
// out = (sum of the K-range partials of P, EPI_PARTIAL, not triangular, batch
// 1) + res, both [M][ldc] bf16
hipError_t launch_splitk_resid(const GemmProblem& P, const void* res, void* out, int ldc, hipStream_t s);

// ---------------------------------------------------------------- teacher selection
constexpr int kTeacherMaxLayers = 256;
constexpr int kTeacherMaxSlices = 16;
struct TeacherArgs {
  const void* A;      // per sample [L][H][M_b][N], samples back to back
  const void* A_ref;  // [B][L][H][M_ref][N]
  float* part;        // [2][B][L][S][N] partial column sums; slice 0 then holds the column sums
  double* tot;        // [2][B][L][NB] float64 totals of 256-column chunks
  double* js_part;    // [B][L][NB] each chunk's share of the divergence
  float* p;           // [B][L][N]
  float* p_ref;       // [B][L][N]
  double* js;         // [B][L]
  int32_t* layers;    // [B][n_top]
  float* teacher;     // [B][N]
  int B, L, H, N, M_ref, S, NB, n_top;  // NB = ceil(N / 256)
  int m_off[MAP_MAX_BATCH + 1];
};
hipError_t launch_teacher(map_dtype dt, const TeacherArgs& a, hipStream_t s);

}  // namespace mapk
