// Host side of the C ABI in include/map.h: argument checks, workspace
// layout, and the order in which the HIP kernels are enqueued.
//
//   map_score:      prep (RoPE table) -> GEMM layer 1 (f_V, f_T) -> GEMM layer 2
//                   -> GEMM projections + RoPE -> logits -> softmax-mean
//   map_similarity: prep (norms) -> GEMM (cosine Gram, upper tiles mirrored)
//   map_select:     top-K0 -> cooperative selection -> restore order
//   map_prune:      prep (norms + table) -> GEMM layer 1 together with the
//                   Gram matrix (one launch, both stream V) -> layer 2 ->
//                   projections -> logits -> softmax-mean -> top-K0 ->
//                   selection -> restore order -> gather
//                   or, on a candidate subset (bf16, N <= 8192):
//                   prep -> GEMM layer 1 -> projections -> logits ->
//                   softmax-mean -> subset -> cosine entries among the
//                   subset (K-split GEMM + ordered sum) -> selection with
//                   gather on the subset -> for the images whose picks are
//                   not certified: Gram matrix -> selection with gather
#include <math.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <initializer_list>
#include <mutex>
#include <vector>

#include "internal.h"

namespace {

using namespace mapk;

constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) & ~(kAlign - 1); }

size_t elem_size(map_dtype dt) { return dt == MAP_BF16 ? 2 : 4; }

// Sequential carve-up of the caller's workspace.
struct Carver {
  char* base;
  size_t off = 0;
  explicit Carver(void* p) : base(static_cast<char*>(p)) {}
  template <typename T> T* take(size_t count) {
    T* r = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += align_up(count * sizeof(T));
    return r;
  }
  void* take_bytes(size_t bytes) {
    void* r = base ? base + off : nullptr;
    off += align_up(bytes);
    return r;
  }
};

bool valid_dtype(map_dtype dt) { return dt == MAP_F32 || dt == MAP_BF16; }

bool valid_weights(const map_weights* w) {
  if (!w) return false;
  const void* ptrs[] = {w->w1_v, w->b1_v, w->w2_v, w->b2_v, w->w_k,
                        w->w1_t, w->b1_t, w->w2_t, w->b2_t, w->w_q};
  for (const void* p : ptrs)
    if (!p) return false;
  return w->D > 0 && w->D % 8 == 0 && w->D_h > 0 && w->D_h % 8 == 0 && w->d_p >= 4 &&
         w->d_p <= 128 && w->d_p % 4 == 0 && isfinite(w->rope_theta) && w->rope_theta > 0.0f;
}

bool valid_bn(int B, int N) { return B >= 1 && B <= MAP_MAX_BATCH && N >= 1 && N <= MAP_MAX_N; }

constexpr int kMaxQuestion = 8192;

bool valid_offsets(const int32_t* t_off, int B) {
  if (!t_off || t_off[0] != 0) return false;
  for (int b = 0; b < B; ++b) {
    const int m = t_off[b + 1] - t_off[b];
    if (m < 1 || m > kMaxQuestion) return false;
  }
  return true;
}

bool valid_select(const map_select_params& sp, int N) {
  return sp.K >= 1 && sp.K <= N && sp.K <= MAP_MAX_K && sp.K0 >= 0 && sp.K0 <= sp.K &&
         isfinite(sp.tau) && sp.tau >= 0.0f;
}

map_status check_ws(void* ws, size_t have, size_t need) {
  if (need == 0) return MAP_OK;
  if (!ws || (reinterpret_cast<uintptr_t>(ws) & (kAlign - 1)) || have < need) return MAP_ERR_WORKSPACE;
  return MAP_OK;
}

// ------------------------------------------------------------ layouts
struct ScoreWs {
  float2 *cs_v, *cs_t;
  void *h1_v, *h1_t;
  void *w2t_v, *w2t_t;  // W2^T of f_V, f_T
  void *wc_v, *wc_t;    // folded W_K W2, W_Q W2 [d_p][D_h]
  float *bc_v, *bc_t;   // folded W_K b2, W_Q b2 [d_p]
  float *k, *q, *logits;
  float2* partial;
  uint64_t* pp;  // the one-launch scoring's shares of p
  long long pp_words;
};

ScoreWs carve_score(Carver& c, map_dtype dt, int B, int N, int sumM, const map_weights& w) {
  ScoreWs s;
  const int half = w.d_p / 2, nblk = (N + 63) / 64;
  const size_t rowsV = (size_t)B * N;
  s.cs_v = c.take<float2>(rowsV * half);
  s.cs_t = c.take<float2>((size_t)sumM * half);
  s.h1_v = c.take_bytes(rowsV * w.D_h * elem_size(dt));
  s.h1_t = c.take_bytes((size_t)sumM * w.D_h * elem_size(dt));
  s.w2t_v = c.take_bytes((size_t)w.D_h * w.D_h * elem_size(dt));
  s.w2t_t = c.take_bytes((size_t)w.D_h * w.D_h * elem_size(dt));
  s.wc_v = c.take_bytes((size_t)w.d_p * w.D_h * elem_size(dt));
  s.wc_t = c.take_bytes((size_t)w.d_p * w.D_h * elem_size(dt));
  s.bc_v = c.take<float>(w.d_p);
  s.bc_t = c.take<float>(w.d_p);
  s.k = c.take<float>(rowsV * w.d_p);
  s.q = c.take<float>((size_t)sumM * w.d_p);
  s.logits = c.take<float>((size_t)sumM * N);
  s.partial = c.take<float2>((size_t)sumM * nblk);
  s.pp_words = score_pp_rows(B, sumM) * N;
  s.pp = c.take<uint64_t>((size_t)s.pp_words);
  return s;
}

// The first 256 bytes of map_select's and map_prune's workspaces hold the
// selection status word (map_selection_status copies it out).
constexpr size_t kStatusBytes = 256;

struct SelectWs {
  float* C;
  float* r2;
  uint64_t* pub;
  unsigned int* bar;
  int32_t* err;
  int32_t* order;
  float* gain;
  int32_t* r0flag;
};

// map_prune's candidate subset: its size per image (0: the full path).
std::atomic<int> g_subset_tokens{0};  // < 0 off, 0 automatic, > 0 that many tokens

int subset_size(map_dtype dt, int N, int D, const map_select_params& sp) {
  const int o = g_subset_tokens.load();
  if (o < 0 || dt != MAP_BF16 || D % 256 != 0 || N > kSubsetMaxN) return 0;
  int nc = o;
  if (o == 0) {
    // Past K = N / 12 the greedy picks' scores fall into the bulk of the
    // bounds and the certificate needs nearly every token (K = N / 9: 80-95 %
    // of them on the retention sweep's images), so the subset cannot pay.
    if (12 * sp.K > N) return 0;
    nc = (sp.K0 + std::max(2 * (sp.K - sp.K0), N / 4) + 63) & ~63;
    if (4 * nc > 3 * N) return 0;  // too close to N to pay
  }
  nc = std::max(nc, sp.K);
  return nc < N ? nc : 0;
}

// The second, larger subset behind the first for a batch (0: none): twice
// the first, if that stays below 3N/4.  Images the first cannot certify
// (correlated frames need more of their tokens: 1567-1820 of 4608 on the
// eight-frame batch against a first subset of 1280) are selected on it
// before the full path; at one image its launches would only add dispatch
// time to the headline call.
int subset_tier2_size(int B, int N, int nc) {
  if (B < 2 || nc <= 0) return 0;
  const int nc2 = (2 * nc + 63) & ~63;
  return 4 * nc2 <= 3 * N ? nc2 : 0;
}

int subset_ksplit(int D) { return D % 512 == 0 ? D / 512 : D / 256; }

int subset_tiles(int nc) {
  const int t = (nc + 127) / 128;
  return t * (t + 1) / 2;
}

struct SubsetWs {
  int32_t* jmap;
  float* pJ;
  float* nJ;
  float* ninvJ;
  uint32_t* hout;
  int32_t* uncert;
  float* SJ;
  float* partial;
  int32_t* order_img;
};

int device_cus();

// The subset's Gram entries come straight from the tiles' cosine epilogue
// when the batch's tiles fill a wave of workgroups; otherwise from K-range
// partial sums (which need the partial buffer).
bool subset_gram_direct(int B, int nc) { return (long long)B * subset_tiles(nc) >= device_cus(); }

SubsetWs carve_subset(Carver& c, int B, int K, int nc, int D) {
  SubsetWs s;
  s.jmap = c.take<int32_t>((size_t)B * nc);
  s.pJ = c.take<float>((size_t)B * nc);
  s.nJ = c.take<float>((size_t)B * nc);
  s.ninvJ = c.take<float>((size_t)B * nc);
  s.hout = c.take<uint32_t>(B);
  s.uncert = c.take<int32_t>(B);
  s.SJ = c.take<float>((size_t)B * nc * nc);
  s.partial = subset_gram_direct(B, nc) ? nullptr
                                        : c.take<float>((size_t)B * subset_tiles(nc) * subset_ksplit(D) * 128 * 128);
  s.order_img = c.take<int32_t>((size_t)B * K);
  return s;
}

SelectWs carve_select(Carver& c, int B, int N, int K) {
  SelectWs s;
  s.C = c.take<float>((size_t)B * N * ((K + 3) & ~3));  // token-major, rows of K rounded up to 4
  s.r2 = c.take<float>((size_t)B * N);
  s.pub = c.take<uint64_t>((size_t)B * 2 * 128 * (kPub + 1));
  s.bar = c.take<unsigned int>(3 * (size_t)B);  // then the full selection behind a subset, then its second subset
  s.err = nullptr;  // the status word at the workspace's start (see carve_status)
  s.order = c.take<int32_t>((size_t)B * K);
  s.gain = c.take<float>((size_t)B * K);
  s.r0flag = c.take<int32_t>(3 * (size_t)B);  // as the barriers
  return s;
}

int32_t* carve_status(Carver& c) { return static_cast<int32_t*>(c.take_bytes(kStatusBytes)); }

void fill_inv_freq(PrepArgs& pa, const map_weights& w) {
  const int half = w.d_p / 2;
  for (int i = 0; i < 64; ++i)
    pa.inv_freq[i] = i < half ? pow(static_cast<double>(w.rope_theta), -2.0 * i / w.d_p) : 0.0;
  pa.half = half;
}

GemmProblem linear(const void* A, int M, const void* W, const void* bias, void* C, int N, int K, int epi) {
  GemmProblem p;
  memset(&p, 0, sizeof(p));
  p.A = A;
  p.B = W;
  p.C = C;
  p.M = M;
  p.N = N;
  p.K = K;
  p.lda = K;
  p.ldb = K;
  p.ldc = N;
  p.batch = 1;
  p.epi = epi;
  p.bias = bias;
  return p;
}

GemmProblem gram(const void* V, int B, int N, int D, float* S, const float* ninv) {
  GemmProblem p;
  memset(&p, 0, sizeof(p));
  p.A = V;
  p.B = V;
  p.C = S;
  p.M = N;
  p.N = N;
  p.K = D;
  p.lda = D;
  p.ldb = D;
  p.ldc = N;
  p.batch = B;
  p.strideA = (long long)N * D;
  p.strideB = (long long)N * D;
  p.strideC = (long long)N * N;
  p.epi = EPI_COSINE;
  p.rs = ninv;
  p.triangular = 1;
  return p;
}

hipError_t enqueue_score(const map_weights& w, map_dtype dt, int B, int N, const void* V,
                         const int32_t* pos_v, const void* T, const int32_t* pos_t,
                         const int32_t* t_off, float* p_out, const ScoreWs& s,
                         const GemmProblem* extra_l1, float* norms, float* ninv, hipStream_t st,
                         unsigned int* clear_bar = nullptr, int32_t* clear_err = nullptr,
                         bool norms_in_layer1 = false, void* gprime_v = nullptr, void* gprime_t = nullptr) {
  const int sumM = t_off[B], rowsV = B * N;
  PrepArgs pa;
  memset(&pa, 0, sizeof(pa));
  pa.V = V;
  pa.rowsV = rowsV;
  pa.D = w.D;
  pa.norms = norms;
  pa.ninv = ninv;
  pa.pos_v = pos_v;
  pa.pos_t = pos_t;
  pa.rowsT = sumM;
  pa.cs_v = s.cs_v;
  pa.cs_t = s.cs_t;
  fill_inv_freq(pa, w);
  // the second layer and the projection as one product: W_K (W2 h + b2) =
  // (W_K W2) h + W_K b2 (and W_Q with f_T's second layer); prep transposes W2
  // and forms the folded biases, the layer-1 launch forms W_K W2
  pa.tsrc[0] = w.w2_v;
  pa.tsrc[1] = w.w2_t;
  pa.tdst[0] = s.w2t_v;
  pa.tdst[1] = s.w2t_t;
  pa.tn = w.D_h;
  pa.fw[0] = w.w_k;
  pa.fw[1] = w.w_q;
  pa.fb[0] = w.b2_v;
  pa.fb[1] = w.b2_t;
  pa.fout[0] = s.bc_v;
  pa.fout[1] = s.bc_t;
  pa.frows = w.d_p;
  pa.fcols = w.D_h;
  const bool one_launch = score_one_launch(B, N, t_off);  // the scoring's exchange arrays, zeroed here
  if (one_launch) {
    pa.clear[0] = reinterpret_cast<uint64_t*>(s.partial);
    pa.nclear[0] = (long long)sumM * ((N + 63) / 64);
    pa.clear[1] = s.pp;
    pa.nclear[1] = s.pp_words;
  }
  GemmBatch g1;
  memset(&g1, 0, sizeof(g1));
  g1.p[0] = linear(V, rowsV, w.w1_v, w.b1_v, s.h1_v, w.D_h, w.D, EPI_BIAS_GELU);
  g1.p[1] = linear(T, sumM, w.w1_t, w.b1_t, s.h1_t, w.D_h, w.D, EPI_BIAS_GELU);
  if (gprime_v && gprime_t) {  // the training step also keeps GELU'(a) of layer 1
    g1.p[0].epi = g1.p[1].epi = EPI_GELU2;
    g1.p[0].aux = gprime_v;
    g1.p[1].aux = gprime_t;
  }
  g1.count = 2;
  g1.p[g1.count++] = linear(w.w_k, w.d_p, s.w2t_v, nullptr, s.wc_v, w.D_h, w.D_h, EPI_BIAS);  // W_K W2
  g1.p[g1.count++] = linear(w.w_q, w.d_p, s.w2t_t, nullptr, s.wc_t, w.D_h, w.D_h, EPI_BIAS);  // W_Q W2
  // the Gram matrix last: its tiles are dispatched after every tile above
  if (extra_l1) g1.p[g1.count++] = *extra_l1;
  gemm_finalize(g1);
  // The row norms: by prep, or (norms_in_layer1) inside the layer-1 launch:
  // with 256 x 256 tiles, by the first column of f_V's tiles from the
  // operands they read; otherwise by workgroups on the compute units its
  // last wave of tiles leaves idle, when there are at least 16 of them and
  // at most 128 rows each.
  if (norms_in_layer1 && gemm_big_tiles(dt, g1)) {
    g1.norm_tiles = 1;  // problem 0: layer 1 of f_V, A = V
    g1.norms = norms;
    g1.ninv = ninv;
  } else if (norms_in_layer1 && gemm_direct_loads(dt, g1) && (reinterpret_cast<uintptr_t>(V) & 15) == 0) {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && cus > 0) {
      const int idle = (cus - g1.total_tiles % cus) % cus;
      if (idle >= 16 && (long long)idle * 128 >= rowsV) {
        g1.norm_blocks = idle;
        g1.norm_V = V;
        g1.norm_rows = rowsV;
        g1.norm_D = w.D;
        g1.norms = norms;
        g1.ninv = ninv;
      }
    }
  }
  hipError_t e = launch_prep(dt, pa, norms != nullptr && g1.norm_blocks == 0 && g1.norm_tiles == 0, true, true, st);
  if (e != hipSuccess) return e;
  if ((e = launch_gemm(dt, g1, extra_l1 ? "gemm_layer1_gram" : "gemm_layer1", st)) != hipSuccess) return e;

  GemmBatch g3;
  memset(&g3, 0, sizeof(g3));
  g3.p[0] = linear(s.h1_v, rowsV, s.wc_v, nullptr, s.k, w.d_p, w.D_h, EPI_ROPE);
  g3.p[0].rope_cs = s.cs_v;
  g3.p[0].rope_bias = s.bc_v;
  g3.p[1] = linear(s.h1_t, sumM, s.wc_t, nullptr, s.q, w.d_p, w.D_h, EPI_ROPE);
  g3.p[1].rope_cs = s.cs_t;
  g3.p[1].rope_bias = s.bc_t;
  g3.count = 2;
  gemm_finalize(g3);
  if ((e = launch_proj_rope(dt, g3, "gemm_proj_rope", st)) != hipSuccess) return e;

  ScoreArgs sa;
  memset(&sa, 0, sizeof(sa));
  sa.q = s.q;
  sa.k = s.k;
  sa.logits = s.logits;
  sa.store_logits = gprime_v != nullptr;  // the training step's backward reads them
  sa.partial = s.partial;
  sa.pp = one_launch ? s.pp : nullptr;
  sa.clear_bar = clear_bar;
  sa.clear_err = clear_err;
  sa.p_out = p_out;
  sa.B = B;
  sa.N = N;
  sa.d_p = w.d_p;
  sa.nblk = (N + 63) / 64;
  for (int b = 0; b <= B; ++b) sa.t_off[b] = t_off[b];
  return launch_score(sa, st);
}

// Inside map_prune (fused = true) the scoring kernel has already cleared the
// selection's counters and the gather ranks the selection order itself.
// With `ga` (map_prune), the selection kernel also gathers the kept rows when
// its order fits in LDS; *gathered says whether it did.
// With `sub` the selection runs on a candidate subset (or is the full
// selection behind one, for the images the subset's run flagged).
struct SubsetSel {
  const int32_t* jmap;
  int32_t* order_map;
  const uint32_t* hout;
  int32_t* uncert;
  const int32_t* run_if;
  int Ng;
  int fallback;
  int no_r0_kernel;
  int tier2;
};

hipError_t enqueue_select(int B, int N, const float* p, const float* S, const float* norms,
                          const map_select_params& sp, int32_t* idx_out, int32_t* order_out,
                          float* gain_out, const SelectWs& w, hipStream_t st, bool fused = false,
                          const GatherArgs* ga = nullptr, bool* gathered = nullptr,
                          const SubsetSel* sub = nullptr) {
  SelectArgs a;
  memset(&a, 0, sizeof(a));
  a.Ng = N;
  if (sub) {
    a.jmap = sub->jmap;
    a.order_map = sub->order_map;
    a.hout = sub->hout;
    a.uncert = sub->uncert;
    a.run_if = sub->run_if;
    a.Ng = sub->Ng;
    a.fallback = sub->fallback;
    a.tier2 = sub->tier2;
    a.no_r0_kernel = sub->no_r0_kernel;
  }
  a.p = p;
  a.S = S;
  a.norms = norms;
  a.C = w.C;
  a.r2 = w.r2;
  a.pub = w.pub;
  a.bar = w.bar;
  a.err = w.err;
  a.order = order_out ? order_out : w.order;
  a.gain = gain_out ? gain_out : w.gain;
  a.idx_out = idx_out;
  a.r0flag = w.r0flag;
  a.B = B;
  a.N = N;
  a.K = sp.K;
  a.K0 = sp.K0;
  a.tau2 = sp.tau * sp.tau;
  if (ga) {
    a.gV = ga->V;
    a.gpos = ga->pos_v;
    a.gV_out = ga->V_out;
    a.gpos_out = ga->pos_out;
    a.row_bytes = ga->row_bytes;
    a.qT = ga->qT;
    a.qpos = ga->qpos;
    memcpy(a.out_off, ga->out_off, sizeof(a.out_off));
    memcpy(a.q_off, ga->q_off, sizeof(a.q_off));
  }
  hipError_t e = fused ? hipSuccess : launch_select_clear(a, st);
  if (e != hipSuccess) return e;
  if ((e = launch_select(a, st)) != hipSuccess) return e;
  if (gathered) *gathered = a.gV != nullptr;
  return fused ? hipSuccess : launch_restore(a, st);
}

map_status hip_status(hipError_t e) { return e == hipSuccess ? MAP_OK : MAP_ERR_HIP; }

size_t score_ws_bytes(map_dtype dt, int B, int N, int sumM, const map_weights& w) {
  Carver c(nullptr);
  carve_score(c, dt, B, N, sumM, w);
  return c.off;
}

size_t select_ws_bytes(int B, int N, int K) {
  Carver c(nullptr);
  carve_status(c);
  carve_select(c, B, N, K);
  return c.off;
}

// ------------------------------------------------------------ training step
struct TrainWs {
  int32_t* status;
  ScoreWs s;
  void *gp_v, *gp_t;              // GELU'(a) of layer 1: [B N][D_h], [sum_M][D_h]
  float* G;                       // [sum_M][N]
  float* dq_part;                 // [nch][sum_M][d_p]
  void *dk_rows, *dk_cols, *dq_rows, *dq_cols;
  void *VT, *TT, *HvT, *HtT;      // [D][ldv], [D][ldt], [D_h][ldv], [D_h][ldt]
  void *WKT, *WQT, *WcvT, *WctT;  // [D_h][kdp]
  void *Xv, *Xt, *XvT, *XtT;      // [d_p][D_h], [D_h][kdp]
  float *Xpv, *Xpt;               // [ldv / 256][d_p][D_h], [ldt / 256][d_p][D_h] token-chunk partials of X
  void *dAv, *dAt, *dAvT, *dAtT;  // [B N][D_h], [sum_M][D_h], [D_h][ldv], [D_h][ldt]
  float *csum_v, *csum_t;         // [d_p]
  float* p;                       // [B][N]
  int ldv, ldt, nch, kdp;  // kdp: d_p padded with zeros to 256, the products over d_p on the direct-load GEMM
};

// Token counts of the token-contiguous operands, padded with zeros to a
// multiple of 256: the reductions over tokens then run on the direct-load GEMM.
int pad256(int n) { return (n + 255) & ~255; }

TrainWs carve_train(Carver& c, map_dtype dt, int B, int N, int sumM, const map_weights& w) {
  TrainWs t;
  const size_t es = elem_size(dt), BN = (size_t)B * N, Dh = w.D_h, dp = w.d_p;
  t.ldv = pad256(B * N);
  t.ldt = pad256(sumM);
  t.nch = (N + 63) / 64;
  t.kdp = pad256(w.d_p);
  const size_t kdp = t.kdp;
  t.status = carve_status(c);
  t.s = carve_score(c, dt, B, N, sumM, w);
  t.gp_v = c.take_bytes(BN * Dh * es);
  t.gp_t = c.take_bytes((size_t)sumM * Dh * es);
  t.G = c.take<float>((size_t)sumM * N);
  t.dq_part = c.take<float>((size_t)t.nch * sumM * dp);
  t.dk_rows = c.take_bytes(BN * kdp * es);
  t.dk_cols = c.take_bytes(dp * t.ldv * es);
  t.dq_rows = c.take_bytes((size_t)sumM * kdp * es);
  t.dq_cols = c.take_bytes(dp * t.ldt * es);
  t.VT = c.take_bytes((size_t)w.D * t.ldv * es);
  t.TT = c.take_bytes((size_t)w.D * t.ldt * es);
  t.HvT = c.take_bytes(Dh * t.ldv * es);
  t.HtT = c.take_bytes(Dh * t.ldt * es);
  t.WKT = c.take_bytes(Dh * kdp * es);
  t.WQT = c.take_bytes(Dh * kdp * es);
  t.WcvT = c.take_bytes(Dh * kdp * es);
  t.WctT = c.take_bytes(Dh * kdp * es);
  t.Xv = c.take_bytes(dp * Dh * es);
  t.Xt = c.take_bytes(dp * Dh * es);
  t.XvT = c.take_bytes(Dh * kdp * es);
  t.XtT = c.take_bytes(Dh * kdp * es);
  t.Xpv = c.take<float>((size_t)(t.ldv / 256) * dp * Dh);
  t.Xpt = c.take<float>((size_t)(t.ldt / 256) * dp * Dh);
  t.dAv = c.take_bytes(BN * Dh * es);
  t.dAt = c.take_bytes((size_t)sumM * Dh * es);
  t.dAvT = c.take_bytes(Dh * t.ldv * es);
  t.dAtT = c.take_bytes(Dh * t.ldt * es);
  t.csum_v = c.take<float>(dp);
  t.csum_t = c.take<float>(dp);
  t.p = c.take<float>(BN);
  return t;
}

size_t train_ws_bytes(map_dtype dt, int B, int N, int sumM, const map_weights& w) {
  Carver c(nullptr);
  carve_train(c, dt, B, N, sumM, w);
  return c.off;
}

bool valid_grads(const map_grads* g) {
  if (!g) return false;
  const float* ptrs[] = {g->w1_v, g->b1_v, g->w2_v, g->b2_v, g->w_k, g->w1_t, g->b1_t, g->w2_t, g->b2_t, g->w_q};
  for (const float* p : ptrs)
    if (!p) return false;
  return true;
}

TransposeJob tjob(const void* src, void* dst, int rows, int cols, int ldd) {
  TransposeJob j;
  memset(&j, 0, sizeof(j));
  j.src = src;
  j.dst = dst;
  j.rows = rows;
  j.cols = cols;
  j.lds = cols;
  j.ldd = ldd;
  return j;
}

hipError_t enqueue_train(const map_weights& w, map_dtype dt, int B, int N, const void* V, const int32_t* pos_v,
                         const void* T, const int32_t* pos_t, const int32_t* t_off, const float* p_teacher,
                         float* loss_out, float* p, const map_grads& g, const TrainWs& t, hipStream_t st) {
  const int sumM = t_off[B], BN = B * N, Dh = w.D_h, dp = w.d_p;
  hipError_t e = enqueue_score(w, dt, B, N, V, pos_v, T, pos_t, t_off, p, t.s, nullptr, nullptr, nullptr, st,
                               nullptr, nullptr, false, t.gp_v, t.gp_t);
  if (e != hipSuccess) return e;
  // dL/dlogits, then dL/dz of the keys and queries (before RoPE), in both layouts
  TrainArgs a;
  memset(&a, 0, sizeof(a));
  a.logits = t.s.logits;
  a.partial = t.s.partial;
  a.p_hat = p;
  a.p_star = p_teacher;
  a.loss = loss_out;
  a.G = t.G;
  a.q = t.s.q;
  a.k = t.s.k;
  a.cs_v = t.s.cs_v;
  a.cs_t = t.s.cs_t;
  a.dq_part = t.dq_part;
  a.dk_rows = t.dk_rows;
  a.dk_cols = t.dk_cols;
  a.dq_rows = t.dq_rows;
  a.dq_cols = t.dq_cols;
  a.B = B;
  a.N = N;
  a.d_p = dp;
  a.nblk = (N + 63) / 64;
  a.nch = t.nch;
  a.ldv = t.ldv;
  a.ldt = t.ldt;
  a.kdp = t.kdp;
  a.inv_B = 1.0f / static_cast<float>(B);
  a.scale = 1.0f / sqrtf(static_cast<float>(dp));
  for (int b = 0; b <= B; ++b) a.t_off[b] = t_off[b];
  if ((e = launch_train_grads(dt, a, st)) != hipSuccess) return e;
  // the operands of the reductions over tokens, tokens contiguous
  TransposeBatch ta;
  memset(&ta, 0, sizeof(ta));
  ta.job[ta.count++] = tjob(V, t.VT, BN, w.D, t.ldv);
  ta.job[ta.count++] = tjob(T, t.TT, sumM, w.D, t.ldt);
  ta.job[ta.count++] = tjob(t.s.h1_v, t.HvT, BN, Dh, t.ldv);
  ta.job[ta.count++] = tjob(t.s.h1_t, t.HtT, sumM, Dh, t.ldt);
  ta.job[ta.count++] = tjob(w.w_k, t.WKT, dp, Dh, t.kdp);
  ta.job[ta.count++] = tjob(w.w_q, t.WQT, dp, Dh, t.kdp);
  ta.job[ta.count++] = tjob(t.s.wc_v, t.WcvT, dp, Dh, t.kdp);
  ta.job[ta.count++] = tjob(t.s.wc_t, t.WctT, dp, Dh, t.kdp);
  transpose_finalize(ta);
  if ((e = launch_transpose(dt, ta, "transpose_in", st)) != hipSuccess) return e;
  // X = dz^T h per branch: a reduction over tokens, in chunks of 256 tokens
  // (batch items of one launch, float32 partials), then their ordered sum
  GemmBatch g1;
  memset(&g1, 0, sizeof(g1));
  const void* xa[2] = {t.dk_cols, t.dq_cols};
  const void* xb[2] = {t.HvT, t.HtT};
  float* xp[2] = {t.Xpv, t.Xpt};
  const int xld[2] = {t.ldv, t.ldt};
  for (int br = 0; br < 2; ++br) {
    GemmProblem& q = g1.p[g1.count++];
    q = linear(xa[br], dp, xb[br], nullptr, xp[br], Dh, 256, EPI_F32);
    q.lda = q.ldb = xld[br];
    q.batch = xld[br] / 256;
    q.strideA = q.strideB = 256;
    q.strideC = (long long)dp * Dh;
  }
  // and in the same launch dL/da = (dz (W W2)) * GELU'(a), over d_p padded to kdp
  g1.p[g1.count] = linear(t.dk_rows, BN, t.WcvT, nullptr, t.dAv, Dh, t.kdp, EPI_MUL);
  g1.p[g1.count++].aux = t.gp_v;
  g1.p[g1.count] = linear(t.dq_rows, sumM, t.WctT, nullptr, t.dAt, Dh, t.kdp, EPI_MUL);
  g1.p[g1.count++].aux = t.gp_t;
  gemm_finalize(g1);
  if ((e = launch_gemm(dt, g1, "gemm_train_x_da", st)) != hipSuccess) return e;
  XReduceArgs xr;
  memset(&xr, 0, sizeof(xr));
  xr.part[0] = t.Xpv;
  xr.part[1] = t.Xpt;
  xr.X[0] = t.Xv;
  xr.X[1] = t.Xt;
  xr.XT[0] = t.XvT;
  xr.XT[1] = t.XtT;
  xr.nc[0] = t.ldv / 256;
  xr.nc[1] = t.ldt / 256;
  xr.d_p = dp;
  xr.D_h = Dh;
  xr.kdp = t.kdp;
  if ((e = launch_x_reduce(dt, xr, st)) != hipSuccess) return e;
  TransposeBatch tb;
  memset(&tb, 0, sizeof(tb));
  tb.job[tb.count++] = tjob(t.dAv, t.dAvT, BN, Dh, t.ldv);
  tb.job[tb.count++] = tjob(t.dAt, t.dAtT, sumM, Dh, t.ldt);
  transpose_finalize(tb);
  if ((e = launch_transpose(dt, tb, "transpose_da", st)) != hipSuccess) return e;
  // the weight gradients (float32):
  //   dW1 = dA^T X_in,  dW_K = X W2^T (+ the rank-one term below),  dW2 = W_K^T X
  GemmBatch g2;
  memset(&g2, 0, sizeof(g2));
  g2.p[0] = linear(t.dAvT, Dh, t.VT, nullptr, g.w1_v, w.D, t.ldv, EPI_F32);
  g2.p[1] = linear(t.dAtT, Dh, t.TT, nullptr, g.w1_t, w.D, t.ldt, EPI_F32);
  g2.p[2] = linear(t.Xv, dp, w.w2_v, nullptr, g.w_k, Dh, Dh, EPI_F32);
  g2.p[3] = linear(t.Xt, dp, w.w2_t, nullptr, g.w_q, Dh, Dh, EPI_F32);
  g2.p[4] = linear(t.WKT, Dh, t.XvT, nullptr, g.w2_v, Dh, t.kdp, EPI_F32);
  g2.p[5] = linear(t.WQT, Dh, t.XtT, nullptr, g.w2_t, Dh, t.kdp, EPI_F32);
  g2.count = 6;
  // dW1_v's 256 long tiles (K = the visual tokens) in a launch of their own,
  // one wave over every compute unit; the five short problems after it
  // (sharing one launch with them took 79 us against 38 + 20)
  GemmBatch g3 = g2;
  g2.count = 1;
  gemm_finalize(g2);
  for (int i = 0; i < 5; ++i) g3.p[i] = g3.p[i + 1];
  g3.count = 5;
  gemm_finalize(g3);
  if ((e = launch_gemm(dt, g2, "gemm_train_dw", st)) != hipSuccess) return e;
  if ((e = launch_gemm(dt, g3, "gemm_train_dw_small", st)) != hipSuccess) return e;
  // bias gradients and the sums of dz over tokens
  RowsumBatch rs;
  memset(&rs, 0, sizeof(rs));
  rs.job[0] = RowsumJob{t.dAvT, g.b1_v, Dh, t.ldv, t.ldv, 0};
  rs.job[1] = RowsumJob{t.dAtT, g.b1_t, Dh, t.ldt, t.ldt, 0};
  rs.job[2] = RowsumJob{t.dk_cols, t.csum_v, dp, t.ldv, t.ldv, 0};
  rs.job[3] = RowsumJob{t.dq_cols, t.csum_t, dp, t.ldt, t.ldt, 0};
  rs.count = 4;
  if ((e = launch_rowsum(dt, rs, st)) != hipSuccess) return e;
  FinishArgs f;
  memset(&f, 0, sizeof(f));
  f.W[0] = w.w_k;
  f.W[1] = w.w_q;
  f.b2[0] = w.b2_v;
  f.b2[1] = w.b2_t;
  f.csum[0] = t.csum_v;
  f.csum[1] = t.csum_t;
  f.db2[0] = g.b2_v;
  f.db2[1] = g.b2_t;
  f.dW[0] = g.w_k;
  f.dW[1] = g.w_q;
  f.D_h = Dh;
  f.d_p = dp;
  return launch_finish(dt, f, st);
}

// ------------------------------------------------------------ decoder layer
bool valid_decoder(const map_decoder_weights* w) {
  return w && w->attn_norm && w->w_qkv && w->w_o && w->ffn_norm && w->w_gate_up && w->w_down && w->head_dim == 128 &&
         w->n_heads >= 1 && w->d == w->n_heads * w->head_dim && w->d % 256 == 0 && w->d <= 8192 && w->ff > 0 &&
         w->ff % 256 == 0 && isfinite(w->rope_theta) && w->rope_theta > 0.0f && isfinite(w->eps) && w->eps >= 0.0f;
}

constexpr int kMaxDecoderRows = 1 << 16;

// K ranges for a product of M rows and N columns over K: enough workgroups
// to cover the device once (split only when the tiles alone leave most of it
// idle), each range a multiple of 256.
void split_k(GemmProblem& p, int cus) {
  const int tiles = ((p.M + 127) / 128) * ((p.N + 127) / 128);
  int ks = tiles >= cus / 2 ? 1 : std::min(p.K / 256, std::max(1, cus / tiles));
  if (ks <= 1) return;
  const int chunk = ((p.K / 256 + ks - 1) / ks) * 256;
  ks = (p.K + chunk - 1) / chunk;
  if (ks <= 1) return;
  p.ksplit = ks;
  p.kchunk = chunk;
  p.epi = EPI_PARTIAL;
}

struct DecoderWs {
  void *h, *qkv, *o, *x1, *gu, *act;
  float* partial;
};

size_t partial_floats(int R, int N, int K, int cus) {
  GemmProblem p;
  memset(&p, 0, sizeof(p));
  p.M = R;
  p.N = N;
  p.K = K;
  split_k(p, cus);
  return p.ksplit > 1 ? (size_t)((R + 127) / 128) * ((N + 127) / 128) * p.ksplit * 128 * 128 : 0;
}

int device_cus() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) !=
                                              hipSuccess || cus <= 0)
    return 256;
  return cus;
}

DecoderWs carve_decoder(Carver& c, int R, const map_decoder_weights& w, int cus) {
  DecoderWs t;
  const size_t r = R, d = w.d, ff = w.ff;
  t.h = c.take_bytes(r * d * 2);
  t.qkv = c.take_bytes(r * 3 * d * 2);
  t.o = c.take_bytes(r * d * 2);
  t.x1 = c.take_bytes(r * d * 2);
  t.gu = c.take_bytes(r * 2 * ff * 2);
  t.act = c.take_bytes(r * ff * 2);
  t.partial = c.take<float>(std::max(partial_floats(R, w.d, w.d, cus), partial_floats(R, w.d, w.ff, cus)));
  return t;
}

// y = acc + residual: split over K into float32 partials and their ordered
// sum (when the tiles alone would leave the device mostly idle), else the
// residual epilogue.
hipError_t resid_product(const void* A, int M, const void* W, int N, int K, const void* res, void* out, float* part,
                         int cus, const char* name, hipStream_t st) {
  GemmBatch g;
  memset(&g, 0, sizeof(g));
  g.p[0] = linear(A, M, W, nullptr, out, N, K, EPI_RESID);
  g.p[0].aux = const_cast<void*>(res);
  split_k(g.p[0], cus);
  if (g.p[0].epi == EPI_PARTIAL) g.p[0].C = part;
  g.count = 1;
  gemm_finalize(g);
  hipError_t e = launch_gemm(MAP_BF16, g, name, st);
  if (e != hipSuccess || g.p[0].epi != EPI_PARTIAL) return e;
  return launch_splitk_resid(g.p[0], res, out, N, st);
}

hipError_t enqueue_decoder(const map_decoder_weights& w, int B, const void* X, const int32_t* pos,
                           const int32_t* seq_off, void* Y, const DecoderWs& t, int cus, hipStream_t st) {
  DecoderArgs a;
  memset(&a, 0, sizeof(a));
  const int R = seq_off[B];
  a.X = X;
  a.pos = pos;
  a.attn_norm = w.attn_norm;
  a.ffn_norm = w.ffn_norm;
  a.h = t.h;
  a.qkv = t.qkv;
  a.o = t.o;
  a.x1 = t.x1;
  a.gu = t.gu;
  a.act = t.act;
  a.R = R;
  a.d = w.d;
  a.n_heads = w.n_heads;
  a.head_dim = w.head_dim;
  a.ff = w.ff;
  a.B = B;
  a.eps = w.eps;
  for (int i = 0; i < 64; ++i) a.inv_freq[i] = pow(static_cast<double>(w.rope_theta), -2.0 * i / w.head_dim);
  for (int b = 0; b <= B; ++b) a.seq_off[b] = seq_off[b];
  for (int b = 0; b < B; ++b) a.max_len = std::max(a.max_len, seq_off[b + 1] - seq_off[b]);
  hipError_t e = launch_rmsnorm(a, X, w.attn_norm, t.h, st);
  if (e != hipSuccess) return e;
  GemmBatch g;
  memset(&g, 0, sizeof(g));
  g.p[0] = linear(t.h, R, w.w_qkv, nullptr, t.qkv, 3 * w.d, w.d, EPI_BIAS);
  g.count = 1;
  gemm_finalize(g);
  if ((e = launch_gemm(MAP_BF16, g, "gemm_qkv", st)) != hipSuccess) return e;
  if ((e = launch_rope_qkv(a, st)) != hipSuccess) return e;
  if ((e = launch_attention(a, st)) != hipSuccess) return e;
  if ((e = resid_product(t.o, R, w.w_o, w.d, w.d, X, t.x1, t.partial, cus, "gemm_o", st)) != hipSuccess) return e;
  if ((e = launch_rmsnorm(a, t.x1, w.ffn_norm, t.h, st)) != hipSuccess) return e;
  GemmBatch g2;
  memset(&g2, 0, sizeof(g2));
  g2.p[0] = linear(t.h, R, w.w_gate_up, nullptr, t.gu, 2 * w.ff, w.d, EPI_BIAS);
  g2.count = 1;
  gemm_finalize(g2);
  if ((e = launch_gemm(MAP_BF16, g2, "gemm_gate_up", st)) != hipSuccess) return e;
  if ((e = launch_silu_mul(a, st)) != hipSuccess) return e;
  return resid_product(t.act, R, w.w_down, w.d, w.ff, t.x1, Y, t.partial, cus, "gemm_down", st);
}

// ------------------------------------------------------------ timing
struct TimingRecord {
  const char* name;
  hipEvent_t start, stop;
};

struct TimingState {
  std::mutex mu;
  bool enabled = false;
  std::vector<TimingRecord> pending;
  std::vector<hipEvent_t> spare;
  std::vector<const char*> names;
  std::vector<double> total_ms;
  std::vector<int> launches;
};

TimingState& timing() {
  static TimingState t;
  return t;
}

hipEvent_t take_event(TimingState& t) {
  if (!t.spare.empty()) {
    hipEvent_t e = t.spare.back();
    t.spare.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

}  // namespace

namespace mapk {

LaunchEvents timing_events(const char* name) {
  TimingState& t = timing();
  std::lock_guard<std::mutex> g(t.mu);
  LaunchEvents ev;
  if (!t.enabled) return ev;
  TimingRecord r{name, take_event(t), take_event(t)};
  if (!r.start || !r.stop) return ev;
  t.pending.push_back(r);
  ev.start = r.start;
  ev.stop = r.stop;
  return ev;
}

}  // namespace mapk

// The language model's layer-0 input as map_prune's destination (section
// "Inference-Time Token Pruning"): each image's kept rows, then its
// question rows, packed (image b from row b K + t_off[b]).
struct Layer0 {
  const void* T;
  const int32_t* pos_t;
  const int32_t* t_off;  // host
};

GatherArgs gather_args(const void* V, const int32_t* pos_v, const int32_t* order, const int32_t* err,
                       int32_t* idx_out, void* V_out, int32_t* pos_out, int B, int N, int K, int row_bytes,
                       const Layer0* l0) {
  GatherArgs ga;
  memset(&ga, 0, sizeof(ga));
  ga.V = V;
  ga.pos_v = pos_v;
  ga.order = order;
  ga.err = err;
  ga.idx_out = idx_out;
  ga.V_out = V_out;
  ga.pos_out = pos_out;
  ga.B = B;
  ga.N = N;
  ga.K = K;
  ga.row_bytes = row_bytes;
  if (l0) {
    ga.qT = l0->T;
    ga.qpos = l0->pos_t;
    for (int b = 0; b < B; ++b) ga.out_off[b] = l0->t_off[b];
    for (int b = 0; b <= B; ++b) ga.q_off[b] = l0->t_off[b];
  }
  return ga;
}

// map_prune on a candidate subset (see subset.hip), with the full
// selection behind it for the images whose picks it cannot certify.
// One subset tier: J, its cosine matrix and the selection on it with the
// certificate check.  run_if (null: every image) limits it to the images an
// earlier tier flagged.  Its subset kernel zeroes clear_bar and
// clear_r0flag for the images it takes: the full selection's counters and
// R0 flags for the first tier (the scoring kernel zeroes the first tier's
// own), the second tier's own for the second.
hipError_t subset_tier(const map_weights& w, map_dtype dt, int B, int N, const void* V,
                       const map_select_params& sp, int32_t* idx_out, float* p, float* norms, float* ninv,
                       float* gain_out, const SelectWs& sw, const SubsetWs& u, int nc, int32_t* order_img,
                       const int32_t* run_if, unsigned int* clear_bar, int32_t* clear_r0flag, bool tier2,
                       hipStream_t st) {
  SubsetArgs sa;
  memset(&sa, 0, sizeof(sa));
  sa.p = p;
  sa.norms = norms;
  sa.ninv = ninv;
  sa.jmap = u.jmap;
  sa.pJ = u.pJ;
  sa.nJ = u.nJ;
  sa.ninvJ = u.ninvJ;
  sa.hout = u.hout;
  sa.uncert = u.uncert;
  sa.B = B;
  sa.N = N;
  sa.Nc = nc;
  sa.K0 = sp.K0;
  sa.tau2 = sp.tau * sp.tau;
  sa.clear_bar = clear_bar;
  sa.clear_r0flag = clear_r0flag;
  sa.run_if = run_if;
  sa.tier2 = tier2;
  hipError_t e = launch_subset(sa, st);
  if (e != hipSuccess) return e;

  // cosine entries among the subset: with tiles for a wave of workgroups,
  // straight from the tiles' cosine epilogue; otherwise raw sums per K
  // range, then their ordered sum with the cosine scaling
  const bool direct = subset_gram_direct(B, nc);
  GemmBatch g;
  memset(&g, 0, sizeof(g));
  g.p[0] = gram(V, B, nc, w.D, direct ? u.SJ : u.partial, direct ? u.ninvJ : nullptr);
  g.p[0].strideA = (long long)N * w.D;
  g.p[0].strideB = (long long)N * w.D;
  g.p[0].mapA = u.jmap;
  g.p[0].mapB = u.jmap;
  g.p[0].mapStride = nc;
  g.p[0].run_if = run_if;
  if (!direct) {
    g.p[0].epi = EPI_PARTIAL;
    g.p[0].ksplit = subset_ksplit(w.D);
  }
  g.count = 1;
  gemm_finalize(g);
  if ((e = launch_gemm(dt, g, tier2 ? "gemm_subset_t2" : "gemm_subset", st)) != hipSuccess) return e;
  if (!direct &&
      (e = launch_gram_reduce(g.p[0], u.SJ, nc, u.ninvJ, st, tier2 ? "gram_reduce_t2" : "gram_reduce")) != hipSuccess)
    return e;

  SubsetSel sub;
  memset(&sub, 0, sizeof(sub));
  sub.jmap = u.jmap;
  sub.order_map = order_img;
  sub.hout = u.hout;
  sub.uncert = u.uncert;
  sub.run_if = run_if;
  sub.Ng = N;
  sub.tier2 = tier2;
  return enqueue_select(B, nc, u.pJ, u.SJ, u.nJ, sp, idx_out, sw.order, gain_out, sw, st, true, nullptr, nullptr, &sub);
}

// map_prune on a candidate subset (see subset.hip), for a batch with a
// second, larger subset behind it, and the full selection behind those for
// the images whose picks they cannot certify.  The selection's barrier
// counters and R0 flags come in three sets of B: the first subset's, the full
// selection's, the second subset's.
map_status prune_on_subset(const map_weights& w, map_dtype dt, int B, int N, const void* V, const int32_t* pos_v,
                           const void* T, const int32_t* pos_t, const int32_t* t_off_host,
                           const map_select_params& sp, int32_t* idx_out, void* V_out, int32_t* pos_out, float* p,
                           int32_t* order_out, float* gain_out, const ScoreWs& s, const SelectWs& sw, float* S,
                           float* norms, float* ninv, const SubsetWs& u, int nc, const SubsetWs& u2, int nc2,
                           hipStream_t st, const Layer0* l0) {
  hipError_t e =
      enqueue_score(w, dt, B, N, V, pos_v, T, pos_t, t_off_host, p, s, nullptr, norms, ninv, st, sw.bar, sw.err, true);
  if (e != hipSuccess) return MAP_ERR_HIP;
  int32_t* order_img = order_out ? order_out : u.order_img;
  SelectWs sw_full = sw, sw_t2 = sw;
  sw_full.bar = sw.bar + B;
  sw_full.r0flag = sw.r0flag + B;
  sw_t2.bar = sw.bar + 2 * B;
  sw_t2.r0flag = sw.r0flag + 2 * B;
  e = subset_tier(w, dt, B, N, V, sp, idx_out, p, norms, ninv, gain_out, sw, u, nc, order_img, nullptr, sw_full.bar,
                  sw_full.r0flag, false, st);
  if (e != hipSuccess) return MAP_ERR_HIP;
  const int32_t* flagged = u.uncert;
  if (nc2 > 0) {
    e = subset_tier(w, dt, B, N, V, sp, idx_out, p, norms, ninv, gain_out, sw_t2, u2, nc2, order_img, u.uncert,
                    sw_t2.bar, sw_t2.r0flag, true, st);
    if (e != hipSuccess) return MAP_ERR_HIP;
    flagged = u2.uncert;
  }

  // the images whose picks were not certified: the full Gram matrix and
  // selection; the workgroups of a certified image only gather its kept
  // rows, from the order the subset's selection wrote as image tokens
  const GatherArgs ga = gather_args(V, pos_v, order_img, sw.err, idx_out, V_out, pos_out, B, N, sp.K,
                                    static_cast<int>(w.D * elem_size(dt)), l0);
  GemmBatch gf;
  memset(&gf, 0, sizeof(gf));
  gf.p[0] = gram(V, B, N, w.D, S, ninv);
  gf.p[0].run_if = flagged;
  gf.count = 1;
  gemm_finalize(gf);
  if ((e = launch_gemm(dt, gf, "gemm_gram_full", st)) != hipSuccess) return MAP_ERR_HIP;
  SubsetSel full;
  memset(&full, 0, sizeof(full));
  full.run_if = flagged;
  full.Ng = N;
  full.fallback = 1;
  // R0 of a flagged image in the selection's own rounds (slower than
  // r0_kernel, but a certified image then pays no launch for it); r0_kernel
  // (gated like the rest) only for a batch without a second subset
  full.no_r0_kernel = B == 1 || nc2 > 0;
  bool gathered = false;
  e = enqueue_select(B, N, p, S, norms, sp, idx_out, order_img, gain_out, sw_full, st, true, &ga, &gathered, &full);
  if (e != hipSuccess) return MAP_ERR_HIP;
  return gathered ? MAP_OK : hip_status(launch_gather(ga, st));
}

// ------------------------------------------------------------ finite check
std::atomic<int> g_finite_check{0};

struct FiniteBuf {
  const void* p;
  long long count;
  int elem_bytes;
};

// With the check on: scan the buffers on `st`, wait, and report
// MAP_ERR_NONFINITE if any holds an infinity or a NaN; MAP_OK otherwise
// (and at once with the check off).
map_status check_finite(hipStream_t st, std::initializer_list<FiniteBuf> bufs) {
  if (!g_finite_check.load()) return MAP_OK;
  int* flag = finite_flag();
  if (!flag || hipMemsetAsync(flag, 0, sizeof(int), st) != hipSuccess) return MAP_ERR_HIP;
  for (const FiniteBuf& f : bufs)
    if (launch_finite_check(f.p, f.count, f.elem_bytes, flag, st) != hipSuccess) return MAP_ERR_HIP;
  int found = 0;
  if (hipMemcpyAsync(&found, flag, sizeof(int), hipMemcpyDeviceToHost, st) != hipSuccess ||
      hipStreamSynchronize(st) != hipSuccess)
    return MAP_ERR_HIP;
  return found ? MAP_ERR_NONFINITE : MAP_OK;
}

// The predictor's inputs: V, T and the ten weight tensors.
map_status check_predictor_inputs(hipStream_t st, const map_weights& w, map_dtype dt, int B, int N, const void* V,
                                  const void* T, int sumM) {
  const int e = static_cast<int>(elem_size(dt));
  const long long D = w.D, H = w.D_h, dp = w.d_p;
  return check_finite(st, {{V, (long long)B * N * D, e}, {T, (long long)sumM * D, e}, {w.w1_v, H * D, e},
                           {w.b1_v, H, e}, {w.w2_v, H * H, e}, {w.b2_v, H, e}, {w.w_k, dp * H, e},
                           {w.w1_t, H * D, e}, {w.b1_t, H, e}, {w.w2_t, H * H, e}, {w.b2_t, H, e},
                           {w.w_q, dp * H, e}});
}

extern "C" {

const char* map_status_string(int status) {
  switch (status) {
    case MAP_OK: return "ok";
    case MAP_ERR_INVALID_ARG: return "invalid argument";
    case MAP_ERR_UNSUPPORTED: return "unsupported";
    case MAP_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
    case MAP_ERR_HIP: return "HIP runtime error";
    case MAP_ERR_TOO_LARGE: return "the call needs more scratch than map_prune_noalloc's static buffer holds";
    case MAP_ERR_NONFINITE: return "an input holds an infinity or a NaN (finite check)";
    default: return "unknown status";
  }
}

int map_version(void) { return 100; }

size_t map_score_workspace(map_dtype dt, int B, int N, int sum_M, const map_weights* w) {
  if (!valid_dtype(dt) || !valid_bn(B, N) || !valid_weights(w) || sum_M < B) return 0;
  return score_ws_bytes(dt, B, N, sum_M, *w);
}

size_t map_similarity_workspace(map_dtype dt, int B, int N, int D) {
  if (!valid_dtype(dt) || !valid_bn(B, N) || D <= 0 || D % 8) return 0;
  return align_up((size_t)B * N * sizeof(float));
}

size_t map_select_workspace(int B, int N, int K) {
  if (!valid_bn(B, N) || K < 1 || K > N || K > MAP_MAX_K) return 0;
  return select_ws_bytes(B, N, K);
}

size_t map_prune_workspace(map_dtype dt, int B, int N, int sum_M, const map_weights* w, int K) {
  if (!valid_dtype(dt) || !valid_bn(B, N) || !valid_weights(w) || sum_M < B || K < 1 || K > N ||
      K > MAP_MAX_K)
    return 0;
  map_select_params sp;
  sp.K = K;
  sp.K0 = K / 2;  // the subset's size does not depend on K0 beyond this bound
  sp.tau = 0.0f;
  size_t sub = 0;
  for (int k0 : {0, K}) {  // the largest subset any K0 can ask for
    sp.K0 = k0;
    const int nc = subset_size(dt, N, w->D, sp);
    if (nc > 0) {
      Carver c(nullptr);
      carve_subset(c, B, K, nc, w->D);
      const int nc2 = subset_tier2_size(B, N, nc);
      if (nc2 > 0) carve_subset(c, B, K, nc2, w->D);
      sub = std::max(sub, c.off);
    }
  }
  return score_ws_bytes(dt, B, N, sum_M, *w) + select_ws_bytes(B, N, K) +
         align_up((size_t)B * N * N * sizeof(float)) + 3 * align_up((size_t)B * N * sizeof(float)) + sub;
}

size_t map_workspace_bytes(int B, int N, int D, int sum_M, int K, const map_weights* w, map_dtype dt) {
  if (w && w->D != D) return 0;
  const size_t sim = map_similarity_workspace(dt, B, N, D), sel = map_select_workspace(B, N, K);
  if (!sim || !sel) return 0;
  size_t need = std::max(sim, sel);
  if (w) {
    const size_t sc = map_score_workspace(dt, B, N, sum_M, w), pr = map_prune_workspace(dt, B, N, sum_M, w, K);
    if (!sc || !pr) return 0;
    need = std::max(need, std::max(sc, pr));
  }
  return need;
}

map_status map_score(const map_weights* w, map_dtype dt, int B, int N, const void* V,
                     const int32_t* pos_v, const void* T, const int32_t* pos_t,
                     const int32_t* t_off_host, float* p_out, void* ws, size_t ws_bytes,
                     void* stream) {
  if (!valid_dtype(dt) || !valid_bn(B, N) || !valid_weights(w) || !V || !pos_v || !T || !pos_t ||
      !p_out || !valid_offsets(t_off_host, B))
    return MAP_ERR_INVALID_ARG;
  const int sumM = t_off_host[B];
  const map_status ws_ok = check_ws(ws, ws_bytes, score_ws_bytes(dt, B, N, sumM, *w));
  if (ws_ok != MAP_OK) return ws_ok;
  const map_status fin = check_predictor_inputs(static_cast<hipStream_t>(stream), *w, dt, B, N, V, T, sumM);
  if (fin != MAP_OK) return fin;
  Carver c(ws);
  const ScoreWs s = carve_score(c, dt, B, N, sumM, *w);
  return hip_status(enqueue_score(*w, dt, B, N, V, pos_v, T, pos_t, t_off_host, p_out, s, nullptr,
                                  nullptr, nullptr, static_cast<hipStream_t>(stream)));
}

map_status map_similarity(map_dtype dt, int B, int N, int D, const void* V, float* S_out,
                          float* norms_out, void* ws, size_t ws_bytes, void* stream) {
  if (!valid_dtype(dt) || !valid_bn(B, N) || D <= 0 || D % 8 || !V || !norms_out) return MAP_ERR_INVALID_ARG;
  const map_status ws_ok = check_ws(ws, ws_bytes, map_similarity_workspace(dt, B, N, D));
  if (ws_ok != MAP_OK) return ws_ok;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const map_status fin = check_finite(st, {{V, (long long)B * N * D, static_cast<int>(elem_size(dt))}});
  if (fin != MAP_OK) return fin;
  Carver c(ws);
  float* ninv = c.take<float>((size_t)B * N);
  PrepArgs pa;
  memset(&pa, 0, sizeof(pa));
  pa.V = V;
  pa.rowsV = B * N;
  pa.D = D;
  pa.norms = norms_out;
  pa.ninv = ninv;
  hipError_t e = launch_prep(dt, pa, true, false, false, st);
  if (e != hipSuccess) return MAP_ERR_HIP;
  if (!S_out) return MAP_OK;  // norms only
  GemmBatch g;
  memset(&g, 0, sizeof(g));
  g.p[0] = gram(V, B, N, D, S_out, ninv);
  g.count = 1;
  gemm_finalize(g);
  return hip_status(launch_gemm(dt, g, "gemm_gram", st));
}

map_status map_select(int B, int N, const float* p, const float* S, const float* norms,
                      map_select_params sp, int32_t* idx_out, int32_t* order_out, float* gain_out,
                      void* ws, size_t ws_bytes, void* stream) {
  if (!valid_bn(B, N) || !p || !S || !norms || !idx_out || !valid_select(sp, N))
    return MAP_ERR_INVALID_ARG;
  const map_status ws_ok = check_ws(ws, ws_bytes, select_ws_bytes(B, N, sp.K));
  if (ws_ok != MAP_OK) return ws_ok;
  const map_status fin = check_finite(static_cast<hipStream_t>(stream),
                                      {{p, (long long)B * N, 4}, {S, (long long)B * N * N, 4}, {norms, (long long)B * N, 4}});
  if (fin != MAP_OK) return fin;
  Carver c(ws);
  int32_t* status = carve_status(c);
  SelectWs w = carve_select(c, B, N, sp.K);
  w.err = status;
  return hip_status(enqueue_select(B, N, p, S, norms, sp, idx_out, order_out, gain_out, w,
                                   static_cast<hipStream_t>(stream)));
}

}  // extern "C"

static map_status prune_impl(const map_weights* w, map_dtype dt, int B, int N, const void* V, const int32_t* pos_v,
                             const void* T, const int32_t* pos_t, const int32_t* t_off_host, map_select_params sp,
                             int32_t* idx_out, void* V_out, int32_t* pos_out, float* p_out, int32_t* order_out,
                             float* gain_out, void* ws, size_t ws_bytes, void* stream, bool layer0) {
  if (!valid_dtype(dt) || !valid_bn(B, N) || !valid_weights(w) || !V || !pos_v || !T || !pos_t ||
      !idx_out || !V_out || !pos_out || !valid_offsets(t_off_host, B) || !valid_select(sp, N))
    return MAP_ERR_INVALID_ARG;
  const int sumM = t_off_host[B];
  const map_status ws_ok = check_ws(ws, ws_bytes, map_prune_workspace(dt, B, N, sumM, w, sp.K));
  if (ws_ok != MAP_OK) return ws_ok;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const map_status fin = check_predictor_inputs(st, *w, dt, B, N, V, T, sumM);
  if (fin != MAP_OK) return fin;
  Carver c(ws);
  int32_t* status = carve_status(c);
  const ScoreWs s = carve_score(c, dt, B, N, sumM, *w);
  SelectWs sw = carve_select(c, B, N, sp.K);
  sw.err = status;
  float* S = c.take<float>((size_t)B * N * N);
  float* norms = c.take<float>((size_t)B * N);
  float* ninv = c.take<float>((size_t)B * N);
  float* p = p_out ? p_out : c.take<float>((size_t)B * N);
  const int nc = subset_size(dt, N, w->D, sp);
  Layer0 l0{T, pos_t, t_off_host};
  const Layer0* l0p = layer0 ? &l0 : nullptr;
  if (nc > 0) {
    const SubsetWs u = carve_subset(c, B, sp.K, nc, w->D);
    const int nc2 = subset_tier2_size(B, N, nc);
    const SubsetWs u2 = nc2 > 0 ? carve_subset(c, B, sp.K, nc2, w->D) : SubsetWs{};
    return prune_on_subset(*w, dt, B, N, V, pos_v, T, pos_t, t_off_host, sp, idx_out, V_out, pos_out, p, order_out,
                           gain_out, s, sw, S, norms, ninv, u, nc, u2, nc2, st, l0p);
  }
  const GemmProblem g = gram(V, B, N, w->D, S, ninv);
  hipError_t e =
      enqueue_score(*w, dt, B, N, V, pos_v, T, pos_t, t_off_host, p, s, &g, norms, ninv, st, sw.bar, sw.err);
  if (e != hipSuccess) return MAP_ERR_HIP;
  const GatherArgs ga = gather_args(V, pos_v, order_out ? order_out : sw.order, sw.err, idx_out, V_out, pos_out, B,
                                    N, sp.K, static_cast<int>(w->D * elem_size(dt)), l0p);
  bool gathered = false;
  e = enqueue_select(B, N, p, S, norms, sp, idx_out, order_out, gain_out, sw, st, true, &ga, &gathered);
  if (e != hipSuccess) return MAP_ERR_HIP;
  return gathered ? MAP_OK : hip_status(launch_gather(ga, st));  // else its own kernel
}

extern "C" {

map_status map_prune(const map_weights* w, map_dtype dt, int B, int N, const void* V, const int32_t* pos_v,
                     const void* T, const int32_t* pos_t, const int32_t* t_off_host, map_select_params sp,
                     int32_t* idx_out, void* V_out, int32_t* pos_out, float* p_out, int32_t* order_out,
                     float* gain_out, void* ws, size_t ws_bytes, void* stream) {
  return prune_impl(w, dt, B, N, V, pos_v, T, pos_t, t_off_host, sp, idx_out, V_out, pos_out, p_out, order_out,
                    gain_out, ws, ws_bytes, stream, false);
}

map_status map_prune_assemble(const map_weights* w, map_dtype dt, int B, int N, const void* V,
                              const int32_t* pos_v, const void* T, const int32_t* pos_t,
                              const int32_t* t_off_host, map_select_params sp, int32_t* idx_out, void* X_out,
                              int32_t* pos_x_out, float* p_out, int32_t* order_out, float* gain_out, void* ws,
                              size_t ws_bytes, void* stream) {
  if (dt == MAP_BF16 || dt == MAP_F32) {  // the question rows are copied 16 bytes at a time
    if (w && ((w->D * elem_size(dt)) & 15)) return MAP_ERR_INVALID_ARG;
    if (((reinterpret_cast<uintptr_t>(T) | reinterpret_cast<uintptr_t>(X_out)) & 15) != 0) return MAP_ERR_INVALID_ARG;
  }
  return prune_impl(w, dt, B, N, V, pos_v, T, pos_t, t_off_host, sp, idx_out, X_out, pos_x_out, p_out, order_out,
                    gain_out, ws, ws_bytes, stream, true);
}

}  // extern "C"

// map_prune_noalloc's workspace: a static device array, one per device the
// library runs on, held until the process ends.  Host code never uses the
// array's name as an address (on the host it is only a stand-in for the
// symbol): its device address is looked up once per device, with that
// device current, and only that address is passed on.
static __device__ __align__(256) unsigned char scratch[MAP_PRUNE_NOALLOC_MAX_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_addr[kMaxDevices] = {};

// The current device's address of `scratch` (null if it cannot be had).
void* scratch_address() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> g(g_scratch_mu);
  if (!g_scratch_addr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
    g_scratch_addr[dev] = p;
  }
  return g_scratch_addr[dev];
}

}  // namespace

extern "C" {

map_status map_prune_noalloc(const map_weights* w, map_dtype dt, int B, int N, const void* V,
                             const int32_t* pos_v, const void* T, const int32_t* pos_t,
                             const int32_t* t_off_host, map_select_params sp, int32_t* idx_out, void* V_out,
                             int32_t* pos_out, float* p_out, int32_t* order_out, float* gain_out, void* stream) {
  if (!valid_bn(B, N) || !valid_offsets(t_off_host, B)) return MAP_ERR_INVALID_ARG;
  const size_t need = map_prune_workspace(dt, B, N, t_off_host[B], w, sp.K);
  if (need > MAP_PRUNE_NOALLOC_MAX_BYTES) return MAP_ERR_TOO_LARGE;
  void* ws = nullptr;
  if (need > 0 && !(ws = scratch_address())) return MAP_ERR_HIP;
  // (need == 0: invalid sizes, which map_prune reports before touching ws)
  return map_prune(w, dt, B, N, V, pos_v, T, pos_t, t_off_host, sp, idx_out, V_out, pos_out, p_out, order_out,
                   gain_out, ws, need > 0 ? MAP_PRUNE_NOALLOC_MAX_BYTES : 0, stream);
}

map_status map_assemble(map_dtype dt, int B, int K, int D, const void* V_out, const int32_t* pos_out,
                        const void* T, const int32_t* pos_t, const int32_t* t_off_host, void* X_out,
                        int32_t* pos_x_out, void* stream) {
  if (!valid_dtype(dt) || B < 1 || B > MAP_MAX_BATCH || K < 1 || K > MAP_MAX_K || D <= 0 || D % 8 || !V_out ||
      !pos_out || !T || !pos_t || !X_out || !pos_x_out || !valid_offsets(t_off_host, B) ||
      ((reinterpret_cast<uintptr_t>(V_out) | reinterpret_cast<uintptr_t>(T) | reinterpret_cast<uintptr_t>(X_out)) &
       15) != 0)
    return MAP_ERR_INVALID_ARG;
  AssembleArgs a;
  memset(&a, 0, sizeof(a));
  a.V_out = V_out;
  a.pos_out = pos_out;
  a.T = T;
  a.pos_t = pos_t;
  a.X = X_out;
  a.pos_x = pos_x_out;
  a.B = B;
  a.K = K;
  a.row_bytes = static_cast<int>(D * elem_size(dt));
  for (int b = 0; b <= B; ++b) a.t_off[b] = t_off_host[b];
  for (int b = 0; b < B; ++b) a.max_rows = std::max(a.max_rows, K + t_off_host[b + 1] - t_off_host[b]);
  return hip_status(launch_assemble(a, static_cast<hipStream_t>(stream)));
}

static int teacher_slices(int B, int L, int N) {
  // about 4096 workgroups (16 per compute unit) for the column sums
  const long long wgs = 2LL * B * L * ((N + 511) / 512);
  return static_cast<int>(std::min<long long>(kTeacherMaxSlices, std::max<long long>(1, (4096 + wgs - 1) / wgs)));
}

size_t map_teacher_workspace(int B, int L, int N) {
  if (B < 1 || B > MAP_MAX_BATCH || L < 1 || L > kTeacherMaxLayers || N < 1 || N > MAP_MAX_N) return 0;
  const size_t nb = (N + 255) / 256, part = 2ull * B * L * teacher_slices(B, L, N) * N * sizeof(float);
  return (part + 255) / 256 * 256 + 3ull * B * L * nb * sizeof(double);
}

map_status map_teacher(map_dtype dt, int B, int L, int H, int N, const void* A, const int32_t* m_off_host,
                       const void* A_ref, int M_ref, int n_top, float* p_out, float* p_ref_out, double* js_out,
                       int32_t* layers_out, float* teacher_out, void* ws, size_t ws_bytes, void* stream) {
  if (!valid_dtype(dt) || B < 1 || B > MAP_MAX_BATCH || L < 1 || L > kTeacherMaxLayers || H < 1 || H > 1024 ||
      N < 1 || N > MAP_MAX_N || (N * elem_size(dt)) % 16 != 0 || M_ref < 1 || M_ref > kMaxQuestion || n_top < 1 ||
      n_top > L || !A || !A_ref || !p_out || !p_ref_out || !js_out || !layers_out || !teacher_out ||
      !valid_offsets(m_off_host, B) ||
      ((reinterpret_cast<uintptr_t>(A) | reinterpret_cast<uintptr_t>(A_ref)) & 15) != 0)
    return MAP_ERR_INVALID_ARG;
  if (!ws || (reinterpret_cast<uintptr_t>(ws) & 15) || ws_bytes < map_teacher_workspace(B, L, N))
    return MAP_ERR_WORKSPACE;
  {
    const int e = static_cast<int>(elem_size(dt));
    const map_status fin = check_finite(static_cast<hipStream_t>(stream),
                                        {{A, (long long)L * H * m_off_host[B] * N, e},
                                         {A_ref, (long long)B * L * H * M_ref * N, e}});
    if (fin != MAP_OK) return fin;
  }
  TeacherArgs a;
  memset(&a, 0, sizeof(a));
  a.A = A;
  a.A_ref = A_ref;
  a.S = teacher_slices(B, L, N);
  a.NB = (N + 255) / 256;
  a.part = static_cast<float*>(ws);
  a.tot = reinterpret_cast<double*>(static_cast<char*>(ws) +
                                    (2ull * B * L * a.S * N * sizeof(float) + 255) / 256 * 256);
  a.js_part = a.tot + 2ull * B * L * a.NB;
  a.p = p_out;
  a.p_ref = p_ref_out;
  a.js = js_out;
  a.layers = layers_out;
  a.teacher = teacher_out;
  a.B = B;
  a.L = L;
  a.H = H;
  a.N = N;
  a.M_ref = M_ref;
  a.n_top = n_top;
  for (int b = 0; b <= B; ++b) a.m_off[b] = m_off_host[b];
  return hip_status(launch_teacher(dt, a, static_cast<hipStream_t>(stream)));
}

size_t map_train_workspace(map_dtype dt, int B, int N, int sum_M, const map_weights* w) {
  if (!valid_dtype(dt) || !valid_bn(B, N) || !valid_weights(w) || w->d_p % 8 || sum_M < B) return 0;
  return train_ws_bytes(dt, B, N, sum_M, *w);
}

map_status map_train_step(const map_weights* w, map_dtype dt, int B, int N, const void* V, const int32_t* pos_v,
                          const void* T, const int32_t* pos_t, const int32_t* t_off_host, const float* p_teacher,
                          float* loss_out, float* p_out, const map_grads* grads, void* ws, size_t ws_bytes,
                          void* stream) {
  if (!valid_dtype(dt) || !valid_bn(B, N) || !valid_weights(w) || w->d_p % 8 || !V || !pos_v || !T || !pos_t ||
      !p_teacher || !loss_out || !valid_grads(grads) || !valid_offsets(t_off_host, B))
    return MAP_ERR_INVALID_ARG;
  const int sumM = t_off_host[B];
  const map_status ws_ok = check_ws(ws, ws_bytes, train_ws_bytes(dt, B, N, sumM, *w));
  if (ws_ok != MAP_OK) return ws_ok;
  map_status fin = check_predictor_inputs(static_cast<hipStream_t>(stream), *w, dt, B, N, V, T, sumM);
  if (fin == MAP_OK) fin = check_finite(static_cast<hipStream_t>(stream), {{p_teacher, (long long)B * N, 4}});
  if (fin != MAP_OK) return fin;
  Carver c(ws);
  const TrainWs t = carve_train(c, dt, B, N, sumM, *w);
  return hip_status(enqueue_train(*w, dt, B, N, V, pos_v, T, pos_t, t_off_host, p_teacher, loss_out,
                                  p_out ? p_out : t.p, *grads, t, static_cast<hipStream_t>(stream)));
}

size_t map_decoder_workspace(int R, const map_decoder_weights* w) {
  if (R < 1 || R > kMaxDecoderRows || !valid_decoder(w)) return 0;
  Carver c(nullptr);
  carve_decoder(c, R, *w, device_cus());
  return c.off;
}

map_status map_decoder_layer(const map_decoder_weights* w, map_dtype dt, int B, const void* X, const int32_t* pos,
                             const int32_t* seq_off_host, void* Y, void* ws, size_t ws_bytes, void* stream) {
  if (!valid_dtype(dt) || !valid_decoder(w) || B < 1 || B > MAP_MAX_BATCH || !X || !pos || !Y ||
      !valid_offsets(seq_off_host, B) || seq_off_host[B] > kMaxDecoderRows ||
      ((reinterpret_cast<uintptr_t>(X) | reinterpret_cast<uintptr_t>(Y)) & 15) != 0)
    return MAP_ERR_INVALID_ARG;
  if (dt != MAP_BF16) return MAP_ERR_UNSUPPORTED;
  const int R = seq_off_host[B], cus = device_cus();
  const map_status ws_ok = check_ws(ws, ws_bytes, map_decoder_workspace(R, w));
  if (ws_ok != MAP_OK) return ws_ok;
  {
    const long long d = w->d, ff = w->ff;
    const map_status fin = check_finite(static_cast<hipStream_t>(stream),
                                        {{X, (long long)R * d, 2}, {w->attn_norm, d, 2}, {w->w_qkv, 3 * d * d, 2},
                                         {w->w_o, d * d, 2}, {w->ffn_norm, d, 2}, {w->w_gate_up, 2 * ff * d, 2},
                                         {w->w_down, d * ff, 2}});
    if (fin != MAP_OK) return fin;
  }
  Carver c(ws);
  const DecoderWs t = carve_decoder(c, R, *w, cus);
  return hip_status(enqueue_decoder(*w, B, X, pos, seq_off_host, Y, t, cus, static_cast<hipStream_t>(stream)));
}

map_status map_set_finite_check(int enable) {
  g_finite_check.store(enable != 0 ? 1 : 0);
  return MAP_OK;
}

map_status map_set_subset_tokens(int n) {
  g_subset_tokens.store(n);
  return MAP_OK;
}

map_status map_set_select_images_per_launch(int n) {
  set_select_images_per_launch(n);
  return MAP_OK;
}

map_status map_selection_status(const void* ws, int32_t* status_out, void* stream) {
  if (!ws || !status_out || (reinterpret_cast<uintptr_t>(ws) & (kAlign - 1))) return MAP_ERR_INVALID_ARG;
  return hip_status(hipMemcpyAsync(status_out, ws, sizeof(int32_t), hipMemcpyDeviceToDevice,
                                   static_cast<hipStream_t>(stream)));
}

map_status map_timing_enable(int enable) {
  TimingState& t = timing();
  std::lock_guard<std::mutex> g(t.mu);
  t.enabled = enable != 0;
  return MAP_OK;
}

int map_timing_read(const char** names, double* total_ms, int* launches, int cap) {
  TimingState& t = timing();
  std::lock_guard<std::mutex> g(t.mu);
  for (const TimingRecord& r : t.pending) {
    float ms = 0.0f;
    if (hipEventSynchronize(r.stop) == hipSuccess && hipEventElapsedTime(&ms, r.start, r.stop) == hipSuccess) {
      size_t k = 0;
      while (k < t.names.size() && strcmp(t.names[k], r.name) != 0) ++k;
      if (k == t.names.size()) {
        t.names.push_back(r.name);
        t.total_ms.push_back(0.0);
        t.launches.push_back(0);
      }
      t.total_ms[k] += ms;
      t.launches[k] += 1;
    }
    t.spare.push_back(r.start);
    t.spare.push_back(r.stop);
  }
  t.pending.clear();
  const int n = static_cast<int>(t.names.size());
  for (int i = 0; i < n && i < cap; ++i) {
    if (names) names[i] = t.names[i];
    if (total_ms) total_ms[i] = t.total_ms[i];
    if (launches) launches[i] = t.launches[i];
  }
  return n;
}

void map_timing_reset(void) {
  TimingState& t = timing();
  std::lock_guard<std::mutex> g(t.mu);
  // every event is destroyed here, so that after a reset the library holds
  // no HIP object (nothing is left for the runtime's teardown at exit)
  for (const TimingRecord& r : t.pending) {
    (void)hipEventSynchronize(r.stop);
    (void)hipEventDestroy(r.start);
    (void)hipEventDestroy(r.stop);
  }
  for (hipEvent_t e : t.spare) (void)hipEventDestroy(e);
  t.pending.clear();
  t.spare.clear();
  t.names.clear();
  t.total_ms.clear();
  t.launches.clear();
}

}  // extern "C"
