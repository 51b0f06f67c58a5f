/*
 * map.h -- C ABI of the MAP visual-token pruning stage on MI355X (gfx950).
 *
 * The stage runs in front of the first language-model layer of a multimodal
 * LLM and keeps K of the N visual tokens of each image ("Learning to Predict
 * Middle-Layer Attention in MLLMs for Visual Token Pruning", section
 * "Inference-Time Token Pruning"):
 *
 *   map_score       visual + question tokens -> predicted attention p_hat
 *                   (Eq. (3), section "Cross-Modal Attention Distillation")
 *   map_similarity  visual tokens -> row norms and cosine similarity, the
 *                   pairwise quantities the diversity term of Eq. (4) needs
 *   map_select      p_hat + similarity + K -> retained token indices
 *                   (top-K0 initial set, orthonormal basis, greedy Eq. (4),
 *                   original order restored)
 *   map_prune       all of the above fused, plus the gather of the kept rows
 *                   and of their positional indices
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Pointers.  Every tensor argument is a DEVICE pointer into memory the caller
 *   owns (allocated with hipMalloc or by a framework); the library never
 *   allocates, frees or retains it.  Host pointers are named *_host.
 * Layout.  Row-major and contiguous.  Batched tensors put the image index
 *   first.  Weight matrices use the W[out][in] layout.
 * Types.  map_dtype selects the storage type of V, T, the weights and V_out:
 *   MAP_F32 (float) or MAP_BF16 (bfloat16 bits).  Scores, norms, similarity
 *   and gains are always float32; indices and positions int32.
 * Streams.  `stream` is a hipStream_t (NULL = the default stream).  All work
 *   is enqueued on it; a call returns without waiting, and outputs are valid
 *   once the stream has been synchronised.  Calls on one stream are ordered.
 * Workspace.  Scratch memory comes from the caller: `ws` must be a device
 *   buffer of at least map_*_workspace() bytes, 256-byte aligned, not used by
 *   anything else until the stream has passed the call.  Calls that run at
 *   the same time need separate workspaces.
 * Errors.  Arguments are checked on the host before anything is enqueued;
 *   on failure the call returns a non-zero map_status and enqueues nothing.
 *   MAP_ERR_HIP means the HIP runtime rejected a launch (the stream may then
 *   hold part of the work).  No exception crosses this interface.
 * Determinism.  Identical inputs give bitwise identical outputs.
 * Residency.  The selection runs as one persistent launch per group of
 *   images whose workgroups must all be resident at once (they meet at
 *   device-wide barriers).  The library sizes each launch to fit the device;
 *   if other work kept them off the device past a bounded wait (seconds),
 *   the selection stops and every idx_out entry of the call is -1 (map_prune
 *   then writes pos_out = -1 and zero rows), and the workspace's status word
 *   reads 1 (map_selection_status).  The kernels never hang.
 * Limits.  1 <= B <= MAP_MAX_BATCH, 1 <= N <= MAP_MAX_N,
 *   1 <= K <= min(N, MAP_MAX_K), 0 <= K0 <= K, D % 8 == 0, D_h % 8 == 0,
 *   d_p a multiple of 4 and <= 128, 1 <= question length <= 8192.
 */
#ifndef MAP_H
#define MAP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MAP_MAX_BATCH 64
#define MAP_MAX_N 16384
#define MAP_MAX_K 1024

typedef enum {
  MAP_OK = 0,
  MAP_ERR_INVALID_ARG = 1,  /* a size, pointer or parameter is out of range */
  MAP_ERR_UNSUPPORTED = 2,  /* valid request the library does not implement */
  MAP_ERR_WORKSPACE = 3,    /* ws is NULL, misaligned or smaller than needed */
  MAP_ERR_HIP = 4,          /* the HIP runtime reported an error            */
  MAP_ERR_TOO_LARGE = 5,    /* the call needs more scratch than the static
                               buffer of map_prune_noalloc holds            */
  MAP_ERR_NONFINITE = 6     /* the finite check (map_set_finite_check) found
                               an infinity or a NaN in a float input        */
} map_status;

typedef enum { MAP_F32 = 0, MAP_BF16 = 1 } map_dtype;

/* Predictor parameters (section "Cross-Modal Attention Distillation").
 * f_V, f_T: Linear(D -> D_h) + bias, GELU (erf form), Linear(D_h -> D_h) +
 * bias.  W_K, W_Q: Linear(D_h -> d_p), no bias.  RoPE with rotate-half
 * pairing (i, i + d_p/2) and frequencies rope_theta^(-2i/d_p) is applied to
 * the projected keys and queries.  All pointers are device pointers of the
 * call's dtype:  w1_* [D_h][D], b1_* [D_h], w2_* [D_h][D_h], b2_* [D_h],
 * w_k and w_q [d_p][D_h]. */
typedef struct {
  const void *w1_v, *b1_v, *w2_v, *b2_v, *w_k;
  const void *w1_t, *b1_t, *w2_t, *b2_t, *w_q;
  int32_t D, D_h, d_p;
  float rope_theta;
} map_weights;

/* Selection parameters (section "Inference-Time Token Pruning").
 * K: tokens kept per image.  K0: size of the top-K0 initial retained set
 * (K0 == K gives plain top-K by p_hat; K0 == 0 starts the greedy rule from
 * an empty basis).  tau: rank-deficiency threshold; a token whose residual
 * against the current basis is at most tau times its own norm adds no basis
 * vector and scores 0 in Eq. (4).  Ties: the top-K0 set prefers the higher
 * p_hat, then the lower index; a greedy step takes the highest score, and
 * between equal scores the lower index.  When every remaining candidate
 * scores 0 the candidate with the highest p_hat (then the lower index) is
 * taken. */
typedef struct {
  int32_t K;
  int32_t K0;
  float tau;
} map_select_params;

/* Human-readable text of a status code (static storage). */
const char* map_status_string(int status);

/* Library interface version (major * 10000 + minor * 100 + patch). */
int map_version(void);

/* Workspace bytes of each call for the given sizes (0 if the sizes are
 * invalid).  sum_M is the total number of question tokens in the batch. */
size_t map_score_workspace(map_dtype dt, int B, int N, int sum_M, const map_weights* w);
size_t map_similarity_workspace(map_dtype dt, int B, int N, int D);
size_t map_select_workspace(int B, int N, int K);
size_t map_prune_workspace(map_dtype dt, int B, int N, int sum_M, const map_weights* w, int K);
/* One workspace size that serves map_score, map_similarity, map_select and
 * map_prune alike for these sizes: the largest of the four (map_score and
 * map_prune left out when w is NULL).  D must equal w->D when w is given;
 * 0 if the sizes are invalid. */
size_t map_workspace_bytes(int B, int N, int D, int sum_M, int K, const map_weights* w, map_dtype dt);

/* map_score -- predicted attention, Eq. (3):
 *   p_hat[b][n] = (1/M_b) sum_m softmax_n( <q_m, k_n> / sqrt(d_p) ),
 *   k_n = RoPE(W_K f_V(v_n), pos_v[b][n]),  q_m = RoPE(W_Q f_T(t_m), pos_t[m]).
 * V      [B][N][D]   visual tokens (projector output), dtype dt
 * pos_v  [B][N]      positional index of each visual token
 * T      [sum_M][D]  question tokens of all images, back to back, dtype dt
 * pos_t  [sum_M]     positional index of each question token
 * t_off_host [B+1]   HOST array; image b owns T rows [t_off[b], t_off[b+1]);
 *                    t_off[0] == 0, strictly increasing, t_off[B] == sum_M
 * p_out  [B][N]      float32 output; each row sums to 1.
 * Hidden activations are stored in dt (bf16 in bf16 calls), accumulation is
 * float32, keys and queries are float32.  The second MLP layer and the
 * projection are applied as one product: W_K f_V(v) = (W_K W2) h + W_K b2 with
 * h the first layer's output (likewise W_Q and f_T); the folded weights are
 * formed inside every call, in dt, from the weights passed. */
map_status map_score(const map_weights* w, map_dtype dt, int B, int N,
                     const void* V, const int32_t* pos_v,
                     const void* T, const int32_t* pos_t, const int32_t* t_off_host,
                     float* p_out, void* ws, size_t ws_bytes, void* stream);

/* map_similarity -- row norms and cosine similarity of the visual tokens:
 *   norms[b][i] = ||v_i||,  S[b][i][j] = <v_i, v_j> / (norms_i norms_j)
 * (a zero row has norm 0 and a zero row and column in S).  The residual of
 * Eq. (4) is evaluated from S and the norms.
 * V [B][N][D] dtype dt;  S_out [B][N][N] float32, or NULL for the norms
 * alone;  norms_out [B][N] float32 (required). */
map_status map_similarity(map_dtype dt, int B, int N, int D, const void* V,
                          float* S_out, float* norms_out,
                          void* ws, size_t ws_bytes, void* stream);

/* map_select -- diversity-aware selection, Eq. (4), for each image:
 * R0 = the K0 tokens with the highest p; the basis is built from R0 in
 * descending p order; then, until K tokens are kept, the candidate with the
 * largest p_i * ||v_i - B B^T v_i|| is added and its normalised residual
 * appended to the basis.  The residual is evaluated as
 * norms_i * sqrt(1 - sum_t c_ti^2) from the cosine similarity S.
 * p      [B][N]     float32 importance, finite and >= 0
 * S      [B][N][N]  float32 cosine similarity (as map_similarity writes it)
 * norms  [B][N]     float32 row norms
 * idx_out   [B][K]  int32 kept token indices, ascending (original order)
 * order_out [B][K]  int32 selection order (R0 first) or NULL
 * gain_out  [B][K]  float32: p of the R0 picks, then the Eq. (4) score of
 *                   each greedy pick (non-increasing); or NULL */
map_status map_select(int B, int N, const float* p, const float* S, const float* norms,
                      map_select_params sp, int32_t* idx_out, int32_t* order_out,
                      float* gain_out, void* ws, size_t ws_bytes, void* stream);

/* map_prune -- map_score, map_similarity and map_select fused, then the
 * gather of the kept tokens in their original order:
 *   V_out[b][k][:] = V[b][idx[b][k]][:] (byte-exact copy, dtype dt)
 *   pos_out[b][k]  = pos_v[b][idx[b][k]]
 * Arguments as in the calls above; p_out, order_out and gain_out may be NULL. */
map_status map_prune(const map_weights* w, map_dtype dt, int B, int N,
                     const void* V, const int32_t* pos_v,
                     const void* T, const int32_t* pos_t, const int32_t* t_off_host,
                     map_select_params sp, int32_t* idx_out, void* V_out, int32_t* pos_out,
                     float* p_out, int32_t* order_out, float* gain_out,
                     void* ws, size_t ws_bytes, void* stream);

/* map_prune_assemble -- map_prune writing the language model's layer-0
 * input directly (section "Inference-Time Token Pruning": the pruned visual
 * tokens, in their original order with their positional indices, are
 * combined with the question tokens before the first layer), so that no
 * separate copy of the kept rows is needed.  Same computation and arguments
 * as map_prune, except that the kept rows and positions go to
 *   X_out     [B*K + sum_M][D] (dtype dt): image b's K kept rows from row
 *             b*K + t_off[b], then its M_b question rows (copied from T)
 *   pos_x_out [B*K + sum_M]    their positional indices (pos_v of the kept
 *             tokens, then pos_t)
 * -- the layout map_assemble produces.  idx_out [B][K] as for map_prune.
 * X_out and T 16-byte aligned, D * sizeof(element) a multiple of 16.
 * Workspace: map_prune_workspace. */
map_status map_prune_assemble(const map_weights* w, map_dtype dt, int B, int N,
                              const void* V, const int32_t* pos_v,
                              const void* T, const int32_t* pos_t, const int32_t* t_off_host,
                              map_select_params sp, int32_t* idx_out, void* X_out, int32_t* pos_x_out,
                              float* p_out, int32_t* order_out, float* gain_out,
                              void* ws, size_t ws_bytes, void* stream);

/* map_prune_noalloc -- map_prune for callers that cannot allocate device
 * memory: code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc.  The same kernels, arguments and outputs as map_prune,
 * without ws / ws_bytes: the workspace is a static device buffer of
 * MAP_PRUNE_NOALLOC_MAX_BYTES that the library holds on every device it
 * runs on until the process ends.  The call allocates nothing and calls no
 * allocating routine.
 * Limit: map_prune_workspace(dt, B, N, sum_M, w, K) must not exceed
 * MAP_PRUNE_NOALLOC_MAX_BYTES (96 MiB: one image of 2880 tokens x 4096 up
 * to K = 640, or 4 images of 1024 tokens), else MAP_ERR_TOO_LARGE and
 * nothing is enqueued.  Other argument errors as for map_prune.
 * Sharing: every call on one device uses that device's one buffer, which
 * keeps the last call's contents (map_prune initialises what it reads);
 * calls that overlap in time on one device -- on several streams or from
 * several threads -- race on it, and the caller must order them (one
 * stream, or events between streams). */
#define MAP_PRUNE_NOALLOC_MAX_BYTES ((size_t)96 << 20)
map_status map_prune_noalloc(const map_weights* w, map_dtype dt, int B, int N,
                             const void* V, const int32_t* pos_v,
                             const void* T, const int32_t* pos_t, const int32_t* t_off_host,
                             map_select_params sp, int32_t* idx_out, void* V_out, int32_t* pos_out,
                             float* p_out, int32_t* order_out, float* gain_out, void* stream);

/* map_teacher -- teacher selection for training the predictor (section
 * "Question Contrastive Teacher Selection", Eq. (1)-(2); QCTS-n of the
 * teacher-selection ablation).  For each sample b and layer l:
 *   p[b][l][n]     = sum_{h,m} A[l][h][m][n] / sum_{h,m,n'} A[l][h][m][n']
 *                    (Eq. (1)'s head/question mean, l1-normalised; uniform
 *                    1/N for a layer whose attention sums to zero)
 *   p_ref[b][l][n] = the same for the reference question's attention
 *   js[b][l]       = D_JS(p, p_ref), natural logarithm, 0 log 0 = 0
 *   layers[b][k]   = the layer with the (k+1)-th largest js (ties to the
 *                    lower layer); layers[b][0] is Eq. (2)'s l*
 *   teacher[b][n]  = mean over k < n_top of p[b][layers[b][k]][n]
 * A      sample b's [L][H][M_b][N] text-to-vision attention (question token
 *        rows), samples back to back; M_b = m_off[b+1] - m_off[b]; dtype dt,
 *        values finite and >= 0; device, 16-byte aligned
 * A_ref  [B][L][H][M_ref][N] the reference question's attention, as A
 * m_off_host [B+1]  host, m_off[0] = 0, 1 <= M_b <= 8192
 * p_out, p_ref_out [B][L][N] float32; js_out [B][L] float64;
 * layers_out [B][n_top] int32; teacher_out [B][N] float32 (device, caller-owned)
 * ws     at least map_teacher_workspace(B, L, N) bytes of device memory
 * Limits: 1 <= B <= MAP_MAX_BATCH, 1 <= L <= 256, 1 <= H <= 1024,
 *   1 <= N <= MAP_MAX_N with N * sizeof(element) a multiple of 16,
 *   1 <= M_ref <= 8192, 1 <= n_top <= L.
 * MAP_ERR_INVALID_ARG for anything outside them (checked before any work is
 * enqueued); MAP_ERR_WORKSPACE for a short workspace.  Asynchronous on
 * `stream`, bitwise deterministic. */
size_t map_teacher_workspace(int B, int L, int N);
map_status map_teacher(map_dtype dt, int B, int L, int H, int N, const void* A, const int32_t* m_off_host,
                       const void* A_ref, int M_ref, int n_top, float* p_out, float* p_ref_out,
                       double* js_out, int32_t* layers_out, float* teacher_out, void* ws, size_t ws_bytes,
                       void* stream);

/* map_assemble -- the language model's layer-0 input after pruning (section
 * "Inference-Time Token Pruning": the kept tokens, in their original order
 * and with their positional indices, are combined with the question
 * tokens).  Image b's block starts at row b*K + t_off[b]: its K kept rows
 * (as map_prune wrote them), then its M_b question rows; the positions
 * likewise.  A pure copy: rows byte-exact, dt their element type.
 * V_out   [B][K][D], pos_out [B][K]   (device; map_prune's outputs)
 * T       [sum M][D], pos_t [sum M]   (device; map_prune's inputs)
 * t_off_host [B+1]                    (host, as for map_prune)
 * X_out   [B*K + sum M][D], pos_x_out [B*K + sum M]  (device, caller-owned)
 * V_out, T and X_out 16-byte aligned.  Asynchronous on `stream`.
 * MAP_ERR_INVALID_ARG: a null or misaligned pointer, an unknown dtype,
 * D % 8 != 0, B or K out of range, bad offsets. */
map_status map_assemble(map_dtype dt, int B, int K, int D, const void* V_out, const int32_t* pos_out,
                        const void* T, const int32_t* pos_t, const int32_t* t_off_host,
                        void* X_out, int32_t* pos_x_out, void* stream);

/* Gradients of the predictor parameters, float32 device buffers of the
 * shapes of the matching map_weights fields (w1_* [D_h][D], b1_* [D_h],
 * w2_* [D_h][D_h], b2_* [D_h], w_k and w_q [d_p][D_h]). */
typedef struct {
  float *w1_v, *b1_v, *w2_v, *b2_v, *w_k;
  float *w1_t, *b1_t, *w2_t, *b2_t, *w_q;
} map_grads;

/* map_train_step -- one training step of the predictor (section
 * "Cross-Modal Attention Distillation": the predictor is trained offline by
 * minimising the KL divergence from the teacher layer's distribution
 * p^{l*} of Eq. (1)-(2), e.g. map_teacher's teacher_out, to the predicted
 * p_hat of Eq. (3)):
 *   loss_out[b] = D_KL(p_teacher[b] || p_hat[b]) = sum_n p* log(p* / p_hat)
 *                 (natural log, 0 log 0 = 0), float32 per image;
 *   grads       = the gradient of (1/B) sum_b loss[b] with respect to every
 *                 predictor parameter (written, not accumulated).
 * The forward pass is map_score's (same arguments, same rounding points);
 * p_out [B][N] receives p_hat when not NULL.  p_teacher [B][N] float32
 * (device) must hold distributions over the N visual tokens.
 * Arithmetic: the call's dtype for stored activations and the operands of
 * the matrix-core products (hidden states, GELU'(a), the gradients of the
 * projections' inputs and of layer 1's pre-activation), float32
 * accumulation, float32 gradients.  Requires d_p % 8 == 0.
 * ws: map_train_workspace(dt, B, N, sum_M, w) bytes, 256-byte aligned.
 * MAP_ERR_INVALID_ARG / MAP_ERR_WORKSPACE / MAP_ERR_HIP as for map_score. */
size_t map_train_workspace(map_dtype dt, int B, int N, int sum_M, const map_weights* w);
map_status map_train_step(const map_weights* w, map_dtype dt, int B, int N,
                          const void* V, const int32_t* pos_v,
                          const void* T, const int32_t* pos_t, const int32_t* t_off_host,
                          const float* p_teacher, float* loss_out, float* p_out,
                          const map_grads* grads, void* ws, size_t ws_bytes, void* stream);

/* The language model's decoder layer that consumes the pruned input
 * (section "Inference-Time Token Pruning": after pruning the model processes
 * only the kept visual tokens and the question tokens; LLaVA's language
 * models use LLaMA's layer).  Device pointers, bf16, torch.nn.Linear layout:
 *   attn_norm, ffn_norm [d]      RMSNorm weights
 *   w_qkv     [3 d][d]           W_q, W_k, W_v stacked by rows
 *   w_o       [d][d]
 *   w_gate_up [2 ff][d]          the SwiGLU gate's rows, then the up rows
 *   w_down    [d][ff]
 * head_dim must be 128 and d = n_heads * head_dim, with d and ff multiples of
 * 256 and d <= 8192. */
typedef struct {
  const void *attn_norm, *w_qkv, *w_o, *ffn_norm, *w_gate_up, *w_down;
  int32_t d, n_heads, head_dim, ff;
  float rope_theta, eps;
} map_decoder_weights;

/* map_decoder_layer -- one decoder layer's prefill over B packed sequences:
 *   h = RMSNorm(X) attn_norm;  q, k, v = h W_qkv^T;  RoPE on q and k per
 *   head at each row's pos (pairs (i, i + 64), theta^(-2i/128));
 *   o = softmax(q k^T / sqrt(128) + causal mask) v per sequence and head;
 *   X1 = X + o W_o^T;  Y = X1 + (SiLU(g) * u) W_down^T with
 *   [g | u] = RMSNorm(X1) ffn_norm W_gate_up^T.
 * X, Y [R][d] bf16 (16-byte aligned), R = seq_off_host[B]; sequence b is rows
 * seq_off[b] .. seq_off[b+1]-1 (host array, strictly increasing from 0), and
 * a row attends to the rows before it in its sequence; pos [R] int32.  The
 * layout map_prune_assemble writes is such an input (seq_off[b] =
 * b K + t_off[b]).  Stored intermediates are bf16, arithmetic float32.
 * ws: map_decoder_workspace(R, w) bytes.  MAP_ERR_UNSUPPORTED for a dtype
 * other than MAP_BF16; MAP_ERR_INVALID_ARG for shapes outside the limits. */
size_t map_decoder_workspace(int R, const map_decoder_weights* w);
map_status map_decoder_layer(const map_decoder_weights* w, map_dtype dt, int B, const void* X,
                             const int32_t* pos, const int32_t* seq_off_host, void* Y,
                             void* ws, size_t ws_bytes, void* stream);

/* map_prune's candidate subset.  A greedy pick of Eq. (4) scores
 * p_i n_i r_i <= p_i n_i, so map_prune may run the selection on a subset J
 * of each image's tokens: R0 plus the tokens with the largest bounds
 * p_i n_i, about K0 + max(2 (K - K0), N / 4) of them (bf16, N <= 8192, K
 * at most N / 12).  It forms the cosine similarity only among J, and keeps
 * J's selection when every greedy pick scores above the largest bound left
 * out.  Otherwise, for a batch (B >= 2), that image is selected again on a
 * subset twice the size (when that stays below 3N / 4), and an image neither
 * subset certifies is selected over all its tokens.  Either way the result
 * is the selection over all tokens; only the time differs.
 *   n < 0: never use a subset; n = 0: automatic (the default); n > 0: a
 *   subset of max(n, K) tokens whenever that is fewer than N.
 * The setting is process-wide and read by map_prune_workspace and map_prune
 * alike: change it only between calls, and query the workspace after.
 * Returns MAP_OK. */
map_status map_set_subset_tokens(int n);

/* map_selection_status -- the selection status word of the last map_select
 * or map_prune call that used workspace `ws` (the word sits in the first
 * 256 bytes of those workspaces).  Enqueues a copy of it into the device
 * int32 *status_out on `stream`; read it once the stream has passed the
 * copy.  Values:
 *   0  the selection completed;
 *   1  a device-wide barrier wait of the selection expired: that call's
 *      idx_out entries are -1 (map_prune: pos_out -1 and zero rows).
 * MAP_ERR_INVALID_ARG for a null or misaligned pointer; MAP_ERR_HIP if the
 * copy cannot be enqueued. */
map_status map_selection_status(const void* ws, int32_t* status_out, void* stream);

/* map_set_finite_check -- a debugging aid, off by default.  While enabled
 * (enable != 0), map_score, map_similarity, map_select, map_prune,
 * map_prune_assemble, map_prune_noalloc, map_teacher, map_train_step and
 * map_decoder_layer first scan their floating-point inputs (activations,
 * weights, scores, similarities, attention, teacher distributions) on
 * `stream` for infinities and NaNs, wait for the scan (the call then blocks
 * until the stream has passed it, so it cannot be captured in a graph) and
 * return MAP_ERR_NONFINITE, having enqueued nothing else, if it finds one.
 * With the check off a non-finite input is not detected: the method's
 * arithmetic then follows IEEE rules (a non-finite or negative score keys
 * as 0 in the selection).  Process-wide; change it only between calls.
 * Returns MAP_OK. */
map_status map_set_finite_check(int enable);

/* At most n images per persistent selection launch (n <= 0: as many as
 * can be resident at once, the default).  Larger batches then run as
 * several launches, as they do by themselves when the device cannot hold
 * every image's workgroups; the result does not change.  Meant for testing
 * that multi-launch path at small sizes.  Process-wide; change it only
 * between calls.  Returns MAP_OK. */
map_status map_set_select_images_per_launch(int n);

/* Per-kernel timing for measurement.  While enabled, every kernel the
 * library launches is bracketed by a pair of HIP events recorded on the
 * launch stream.  map_timing_read() waits for those events, accumulates the
 * elapsed time per kernel name and fills up to `cap` entries (names point to
 * static strings); it returns the number of kernel names seen.
 * map_timing_reset() drops everything recorded so far and destroys the
 * library's events (after a reset the library holds no HIP object). */
map_status map_timing_enable(int enable);
int map_timing_read(const char** names, double* total_ms, int* launches, int cap);
void map_timing_reset(void);

#ifdef __cplusplus
}
#endif

#endif /* MAP_H */
