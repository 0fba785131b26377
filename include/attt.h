/*
 * attt.h -- C ABI of the aTTT in-episode update step on AMD Instinct MI355X (gfx950).
 *
 * "No Time Like the Present: Agentic Test-Time Training for LLM Agents" (arXiv 2607.03441).
 * One aTTT update (Algorithm 1) takes the new update text x_k, the episode's token history
 * H^tok_k (the concatenation of its previous updates), the n-gram size n and the weight
 * floor w_min, weights every token of x_k by its n-gram exposure (Eq. 8-9) and takes a
 * gradient step on the token-weighted next-token loss (Eq. 10) of an episode-specific
 * LoRA adapter. This library computes the data-parallel part of that step on one GPU:
 *
 *   attt_ngram_weights        exposure f and weights w of every update token (Eq. 8-9)
 *   attt_ngram_set_*          the same weights from persistent per-episode n-gram counts that
 *                             grow with every update (the history update of Algorithm 1)
 *   attt_weighted_ce_fwd_bwd  weighted CE through the frozen LM head, loss and dL/dh (Eq. 10)
 *   attt_lora_grad            LoRA dA / dB of the adapted projections (Sec. 3.1, Appendix C)
 *   attt_lora_sgd_step        the adapter step theta <- theta - lr grad (Eq. 2, Algorithm 1)
 *
 * Conventions shared by every call
 *   - Data pointers are device pointers unless a parameter says "host". The caller owns all
 *     memory; the library never allocates device memory, frees memory or synchronises the
 *     stream in these calls. Scratch space comes from the caller's `workspace`, whose size is
 *     given by the matching *_workspace_size query (any larger size is fine). The workspace
 *     must be 256-byte aligned; its contents need not be initialised and are garbage after.
 *   - Work is enqueued asynchronously on `stream` (a hipStream_t passed as void*; NULL is the
 *     null stream). Outputs are valid once the stream reaches that point.
 *   - Arguments are validated on the host before any HIP call, so ATTT_EINVAL and
 *     ATTT_ENOSPACE come back without touching the device. A failing launch returns
 *     ATTT_EHIP. attt_last_error() gives a message for the last failing call of this thread.
 *   - Matrices are dense row-major with the leading dimension equal to the row length, and
 *     must be 16-byte aligned. Floating-point dtypes: ATTT_F32 (float) or ATTT_BF16
 *     (bfloat16, accumulated in float32).
 *   - Calls are reentrant; concurrent calls must use distinct workspaces. Results are
 *     bitwise reproducible for identical inputs on the same device (ordered reductions,
 *     integer atomics only).
 */
#ifndef ATTT_H_
#define ATTT_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t attt_status;
#define ATTT_OK 0
#define ATTT_EINVAL 1       /* an argument is out of range, misaligned or inconsistent        */
#define ATTT_ENOSPACE 2     /* workspace smaller than the size query returned                 */
#define ATTT_EUNSUPPORTED 3 /* valid by the paper but beyond this build's limits (see below)  */
#define ATTT_EHIP 4         /* the HIP runtime reported an error while launching              */

#define ATTT_F32 0
#define ATTT_BF16 1

#define ATTT_NGRAM_MAX_N 16  /* largest n-gram size accepted                                   */
#define ATTT_LORA_MAX_RANK 64

const char* attt_status_string(attt_status status);
/* Message of the last failing call on the calling thread ("" if none). */
const char* attt_last_error(void);
/* Library version as major*10000 + minor*100 + patch. */
int32_t attt_version(void);

/* --------------------------------------------------------------------------------------
 * n-gram exposure and token weights (Sec. 3.3, Eq. 8-9; the weighting loop of Algorithm 1)
 *
 * For each of E episodes, history e is H^tok_k: the flat concatenation of the token ids
 * of that episode's previous updates. n-grams that straddle two previous updates count,
 * and occurrences overlap (every start position counts). For every position j of the
 * episode's update x_k:
 *     f(j) = max over the n-grams g of x_k that contain j of count(g, H^tok_k)
 *            (0 when no n-gram of x_k contains j, i.e. when L < n)
 *     w(j) = max(w_min, 1 / (1 + f(j)))   in float32, round to nearest even
 * Repeats of an n-gram inside x_k itself are not counted (only H^tok_k is).
 *
 * history          device int32 [history_offsets[E]]: all histories, back to back
 * history_offsets  HOST int64 [E+1]: history e is history[history_offsets[e] .. [e+1])
 * tokens           device int32 [token_offsets[E]]: all update texts x_k, back to back
 * token_offsets    HOST int64 [E+1]
 * num_episodes     E >= 1
 * n                1 <= n <= ATTT_NGRAM_MAX_N
 * w_min            weight floor, 2^-20 <= w_min <= 1 (the paper uses 0.05)
 * exposure         device uint32 [T] or NULL: f per update token (T = token_offsets[E])
 * weights          device float [T]: w per update token
 * Token ids are compared for equality only; any int32 value is allowed. Offsets must start
 * at 0 and be non-decreasing; each episode may hold up to 2^31 - 1 history tokens.
 * ------------------------------------------------------------------------------------ */
attt_status attt_ngram_workspace_size(const int64_t* history_offsets, const int64_t* token_offsets,
                                      int32_t num_episodes, int32_t n, size_t* bytes);
attt_status attt_ngram_weights(const int32_t* history, const int64_t* history_offsets,
                               const int32_t* tokens, const int64_t* token_offsets,
                               int32_t num_episodes, int32_t n, float w_min,
                               uint32_t* exposure, float* weights,
                               void* workspace, size_t workspace_bytes, void* stream);

/* attt_ngram_weights_noalloc: attt_ngram_weights without a workspace, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation). Same arguments, results and errors as attt_ngram_weights, except that the scratch
 * (16-bit partial counts, the size attt_ngram_workspace_size reports) lives in a static device
 * buffer of ATTT_NGRAM_NOALLOC_SCRATCH_BYTES that the library holds on every GPU it runs on
 * until the process ends. A call needing more returns ATTT_EUNSUPPORTED (before any HIP call).
 * Nothing is allocated: no hipMalloc, no hipFree. Every call on one GPU uses that GPU's buffer,
 * so calls that overlap in time on one GPU (other streams, other host threads) race and give
 * wrong results; calls ordered on one stream are fine. The buffer needs no initialisation: every
 * count a call reads was written earlier in the same call. */
#define ATTT_NGRAM_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)
attt_status attt_ngram_weights_noalloc(const int32_t* history, const int64_t* history_offsets,
                                       const int32_t* tokens, const int64_t* token_offsets,
                                       int32_t num_episodes, int32_t n, float w_min,
                                       uint32_t* exposure, float* weights, void* stream);

/* --------------------------------------------------------------------------------------
 * Backward of one adapted attention block: the gradients dY_q, dY_k, dY_v of the q, k and v
 * projection outputs, which are the upstream gradients of the LoRA gradient below (the
 * episode adapter on q/k/v/o of Sec. 3.1; rank and alpha in Appendix C). Causal attention with
 * grouped key/value heads, each episode an independent sequence:
 *     S = scale Q K^T (query t sees keys s <= t of its episode), P = softmax(S), O = P V,
 *     D = rowsum(dO * O),  dP = dO V^T,  dS = P * (dP - D),
 *     dQ = scale dS K,  dK = scale dS^T Q,  dV = P^T dO
 * with query head h reading key/value head h / (heads / kv_heads); dK and dV of a key/value
 * head are summed over its query heads. Q and K are the attention's inputs (after any position
 * encoding); dO is the gradient of the attention output (the o projection's input).
 * bf16 in and out, float32 accumulation; between the two products of each step P and dS are
 * carried as bf16 pairs hi + lo. Deterministic (fixed accumulation orders, no atomics).
 *
 * q, dout         device bf16 [N][heads][128] (token-major: row t is [heads x 128])
 * k, v            device bf16 [N][kv_heads][128]
 * row_offsets     host int64 [E+1] (episodes of rows; NULL: one episode of N rows)
 * heads, kv_heads kv_heads >= 1 divides heads; head_dim must be 128
 * scale           finite, > 0 (1/sqrt(128) for the standard block)
 * dq / dk, dv     device bf16, the layouts of q / k, v (written in full)
 * lse, dsum       device float32 [heads][N]: the forward's log-sum-exp and D (written)
 * All device pointers 16-byte aligned. Errors (before any HIP call): ATTT_EINVAL for bad
 * offsets, null or misaligned pointers, heads not a multiple of kv_heads, a bad scale;
 * ATTT_EUNSUPPORTED for head_dim != 128, heads >= 2^16 or N >= 2^31 / heads. */
attt_status attt_attention_bwd(const void* q, const void* k, const void* v, const void* dout,
                               const int64_t* row_offsets, int32_t num_episodes, int64_t N,
                               int32_t heads, int32_t kv_heads, int32_t head_dim, float scale,
                               void* dq, void* dk, void* dv, float* lse, float* dsum, void* stream);

/* --------------------------------------------------------------------------------------
 * Update-text repetition and the sequence-level filter (Sec. 3.2, Eq. 6-7; tau of Appendix C):
 *     rho(x_k) = max over x' in H_k of J(W(x_k), W(x')),   J(A, B) = |A & B| / |A | B|,
 *     nu(x_k) = 1 - rho(x_k),   skip the update when nu < tau   (tau = 0.5 in the paper)
 * W(x) is the set of whitespace-separated words of an update text. Texts arrive as word ids, one
 * int32 per word, equal words equal ids (splitting and mapping strings is the caller's work).
 * Episodes are independent; the texts of episode e are texts episode_texts[e] ..
 * episode_texts[e+1] - 1 in order, the last of them the candidate x_k and the others H_k. An
 * episode with one text has rho = 0. J of two empty word sets is 0. Counts are exact integers;
 * rho is the float64 nearest to the largest |A & B| / |A | B|, nu = RN(1 - rho) in float64,
 * skip = (nu < tau) in float64, so every output is bit-reproducible.
 *
 * words             device int32 [text_offsets[T]]: the word ids of all texts back to back;
 *                   ids in [0, 2^31) (a negative id is outside the contract: the counts of its
 *                   text are then not meaningful, nothing is read or written out of bounds)
 * text_offsets      host int64 [T+1], T = episode_texts[E]: text t is words[text_offsets[t] ..
 *                   text_offsets[t+1]); text_offsets[0] = 0, non-decreasing; a text may be empty
 * text_offsets_dev  the same T+1 values in device memory (the kernels read text ranges there)
 * episode_texts     host int64 [E+1], episode_texts[0] = 0, at least one text per episode
 * tau               the skip threshold, finite
 * rho, nu           device double [E];  skip  device int32 [E] (1 = skip the update)
 * best              device int32 [E]: index within the episode's texts of the first previous
 *                   text that attains rho, -1 for an episode with one text
 * pair_counts       device int32 [P][2] or NULL: (|A & B|, |A | B|) of every previous text
 *                   against its episode's candidate, episodes and texts in order;
 *                   P = sum over episodes of (texts - 1)
 * workspace         device, >= attt_repetition_workspace_size bytes, 256-byte aligned
 * Errors (before any HIP call): ATTT_EINVAL for bad offsets, null pointers, a non-finite tau or
 * E < 1; ATTT_EUNSUPPORTED for more than 2^31 - 1 words, more than 2^26 pairs x partitions, or a
 * text of more than 2^20 words. Should an LDS word set ever fill (not possible for hashes of
 * distinct ids spread as planned), that episode's rho and nu are NaN, skip 0 and best -1. */
attt_status attt_repetition_workspace_size(const int64_t* text_offsets, const int64_t* episode_texts,
                                           int32_t num_episodes, size_t* bytes);
attt_status attt_update_repetition(const int32_t* words, const int64_t* text_offsets,
                                   const int64_t* text_offsets_dev, const int64_t* episode_texts,
                                   int32_t num_episodes, double tau, double* rho, double* nu,
                                   int32_t* skip, int32_t* best, int32_t* pair_counts,
                                   void* workspace, size_t workspace_bytes, void* stream);

/* --------------------------------------------------------------------------------------
 * Persistent n-gram sets: the history update of Algorithm 1 (H^tok_{k+1} = H^tok_k followed by
 * x_k) kept as device-resident n-gram counts, so that the weights of the next update (Eq. 8-9)
 * cost O(|x_k|) lookups instead of a pass over the whole history.
 *
 * A set holds count(g, H) for every n-gram g of one episode's history H. Appending x adds the
 * n-grams whose last token lies in x, including the n-1 that start in the last n-1 tokens of
 * H (n-grams straddling two updates count, as in attt_ngram_weights; overlapping occurrences
 * all count). attt_ngram_set_weights then gives, for an update x and the set's history H,
 * exactly the f and w that attt_ngram_weights gives for x and the flat history H. Algorithm 1
 * per update: attt_ngram_set_weights(x_k), the gradient step, attt_ngram_set_append(x_k).
 *
 * A set is a caller-owned device buffer of attt_ngram_set_size(capacity, n) bytes, 256-byte
 * aligned, valid after attt_ngram_set_init (an empty history). capacity is the number of
 * distinct n-grams it can hold (at most the number of tokens ever appended is always enough);
 * the table is sized to stay at most half full. Every call on a set must pass the capacity
 * and n it was initialised with.
 *
 * sets           HOST array of num_sets device pointers, one set per episode (distinct buffers)
 * tokens         device int32 [token_offsets[num_sets]]: one text per set, back to back
 * token_offsets  HOST int64 [num_sets+1], starting at 0, non-decreasing
 * capacity       1 .. 2^30;  n: 1 <= n <= ATTT_NGRAM_MAX_N;  w_min as for attt_ngram_weights
 * set_bytes      size of every set buffer (init only; ATTT_ENOSPACE if below the size query)
 * exposure       device uint32 [T] or NULL;  weights: device float [T]
 * Errors the host cannot see without a synchronisation are reported in the outputs: a set that
 * received more distinct n-grams than its capacity, whose 64-bit n-gram keys collided (two
 * different n-grams, never observed), or that is used with another n or capacity than it was
 * initialised for, gives exposure 0xFFFFFFFF and weight NaN for every token queried against
 * it, until it is initialised again. Calls on one set must be ordered (one stream).
 * ------------------------------------------------------------------------------------ */
attt_status attt_ngram_set_size(int64_t capacity, int32_t n, size_t* bytes);
attt_status attt_ngram_set_init(void* const* sets, int32_t num_sets, int64_t capacity, int32_t n,
                                size_t set_bytes, void* stream);
attt_status attt_ngram_set_append(void* const* sets, const int32_t* tokens, const int64_t* token_offsets,
                                  int32_t num_sets, int64_t capacity, int32_t n, void* stream);
attt_status attt_ngram_set_weights(void* const* sets, const int32_t* tokens, const int64_t* token_offsets,
                                   int32_t num_sets, int64_t capacity, int32_t n, float w_min,
                                   uint32_t* exposure, float* weights, void* stream);

/* --------------------------------------------------------------------------------------
 * Token-weighted next-token cross-entropy through a frozen LM head (Sec. 3.3, Eq. 10;
 * the gradient of the weighted loss in Algorithm 1), forward and backward.
 *
 * Row t of `hidden` is the hidden state that predicts token labels[t]; weights[t] is that
 * token's weight w. Rows are grouped into E episodes by row_offsets; episode e has
 * L_e = row_offsets[e+1] - row_offsets[e] rows and
 *     z_t    = W h_t                                   (logits)
 *     lse_t  = log sum_v exp(z_tv)
 *     loss_e = (1 / L_e) sum_{t in e} w_t (lse_t - z_{t, labels[t]})
 *     dL/dh_t = (w_t / L_e) (softmax(z_t) - onehot(labels[t])) W
 * Natural log, full softmax over V, no bias, no label smoothing; the head gets no gradient.
 * The logits z are never written to memory, and the bf16 backward holds no buffer of (rows x
 * vocabulary) at all: one persistent kernel computes 256 x 256 tiles of the softmax numerators
 * e_tv = exp(z_tv - z_{t,labels[t]}) and, on other CUs of the same XCD, contracts them with W as
 * they arrive through a ring of a few MB in the workspace (dL/dh is a per-row scale of
 * sum_v e_tv W_v minus the label term). Below 16 slices of 256 in d, the consumers of a slice
 * split the vocabulary tiles, and the workspace also holds their float32 partial sums (at
 * most 30 MiB); they are added in a fixed order, so results stay bitwise repeatable. It needs the MI355X layout of 256 CUs in 8 XCDs and
 * cooperative launch (ATTT_EUNSUPPORTED otherwise). The float32 backward stages dL/dz for blocks
 * of at most 8192 rows x 131072 columns in the workspace.
 *
 * hidden       device [N, d] of dtype
 * lm_head      device [V, d] of dtype (the nn.Linear weight layout)
 * labels       device int32 [N], each in [0, V); a label outside that range is not an error
 *              the host can see: that row's loss term becomes NaN (and, with grad_hidden, its
 *              gradient row; on the bf16 path also its lse), and W is never read at that label
 * weights      device float [N]
 * row_offsets  HOST int64 [E+1], from 0 to N, non-decreasing; NULL means one episode of N rows
 * num_episodes E >= 1
 * N, d, V      N >= 0, 1 <= d < 2^20 with d % 8 == 0, 1 <= V < 2^31; the bf16 backward needs
 *              V <= 2^21 - 256 (ATTT_EUNSUPPORTED beyond)
 * dtype        ATTT_F32 or ATTT_BF16
 * loss         device float [E]
 * lse          device float [N] or NULL
 * grad_hidden  device [N, d] of dtype, or NULL for the forward only
 * The workspace query takes flags: ATTT_CE_WANT_GRAD when grad_hidden is passed, plus
 * ATTT_CE_HEAD_T when the call is given a prepared transposed head (attt_weighted_ce_fwd_bwd_ex).
 * ------------------------------------------------------------------------------------ */
#define ATTT_CE_WANT_GRAD 1
#define ATTT_CE_HEAD_T 2
attt_status attt_ce_workspace_size(int64_t N, int64_t d, int64_t V, int32_t dtype, int32_t flags,
                                   size_t* bytes);
attt_status attt_weighted_ce_fwd_bwd(const void* hidden, const void* lm_head, const int32_t* labels,
                                     const float* weights, const int64_t* row_offsets,
                                     int32_t num_episodes, int64_t N, int64_t d, int64_t V,
                                     int32_t dtype, float* loss, float* lse, void* grad_hidden,
                                     void* workspace, size_t workspace_bytes, void* stream);

/* Diagnostics: bounds (microseconds) of every wait inside the persistent bf16 backward, for its
 * label-referenced pass and for its exact pass (defaults 20000 each; both >= 0). A wait that runs
 * out aborts that pass: the label-referenced pass then falls back to the exact pass; an aborted
 * exact pass makes loss, lse and dL/dh NaN. Tests set tiny bounds to drive these paths. Applies
 * to later calls in the process; not synchronised against concurrent calls. */
attt_status attt_ce_set_wait_limit(int64_t label_us, int64_t exact_us);

/* The frozen head, transposed once (Sec. 3.1: only the episode's adapter is trained, so the
 * LM head of Eq. 10 is the same matrix in every update of every episode). The bf16 backward
 * contracts dL/dz with W over the vocabulary and reads W as W^T [d, Vp] (Vp = V rounded up to
 * 256, columns V .. Vp-1 zero) so that both GEMM operands are contiguous along the contraction.
 * attt_weighted_ce_fwd_bwd builds that copy in its workspace on every call;
 * attt_ce_head_transpose builds it once into a caller-owned buffer of attt_ce_head_t_size
 * bytes (16-byte aligned), and attt_weighted_ce_fwd_bwd_ex reads it from there (lm_head_t,
 * bf16 with grad_hidden only; NULL = build it in the workspace as the plain call does). The
 * buffer stays valid while lm_head is unchanged. */
attt_status attt_ce_head_t_size(int64_t d, int64_t V, size_t* bytes);
attt_status attt_ce_head_transpose(const void* lm_head, int64_t d, int64_t V, void* lm_head_t,
                                   size_t lm_head_t_bytes, void* stream);
attt_status attt_weighted_ce_fwd_bwd_ex(const void* hidden, const void* lm_head, const void* lm_head_t,
                                        const int32_t* labels, const float* weights,
                                        const int64_t* row_offsets, int32_t num_episodes, int64_t N,
                                        int64_t d, int64_t V, int32_t dtype, float* loss, float* lse,
                                        void* grad_hidden, void* workspace, size_t workspace_bytes,
                                        void* stream);

/* --------------------------------------------------------------------------------------
 * LoRA adapter gradients (episode-specific adapter, Sec. 3.1; rank and alpha, Appendix C).
 *
 * An adapted projection computes y = x W0^T + scale * (x A^T) B^T, scale = alpha / rank.
 * Given its input x and the upstream gradient dy = dL/dy, with U = x A^T:
 *     dB += scale * dy^T U          dA += (scale * dy B)^T x
 * Both outputs are float32 and accumulated into (+=), so several micro-batches can share
 * one gradient buffer; zero them first for a plain gradient.
 *
 * problems   HOST array of `count` descriptors, processed as one grouped launch:
 *   x      device [rows, d_in]  of dtype
 *   dy     device [rows, d_out] of dtype
 *   A      device [rank, d_in]  of dtype
 *   B      device [d_out, rank] of dtype
 *   dA     device float [rank, d_in]   (+=)
 *   dB     device float [d_out, rank]  (+=)
 *   rows >= 0, d_in and d_out >= 1 and multiples of 8, 1 <= rank <= ATTT_LORA_MAX_RANK;
 *   rows < 2^24 and d_in, d_out < 2^20 (ATTT_EUNSUPPORTED beyond)
 *   Outputs of different problems must not overlap. Problems with the same x pointer, d_in
 *   and rows (the q, k and v projections of one layer) are computed together, x being read
 *   once per pass for up to 64 of their combined (16-padded) ranks.
 * ------------------------------------------------------------------------------------ */
typedef struct attt_lora_problem {
  const void* x;
  const void* dy;
  const void* A;
  const void* B;
  float* dA;
  float* dB;
  int64_t rows;
  int64_t d_in;
  int64_t d_out;
  int32_t rank;
  float scale;
} attt_lora_problem;

attt_status attt_lora_workspace_size(const attt_lora_problem* problems, int32_t count, int32_t dtype,
                                     size_t* bytes);
attt_status attt_lora_grad(const attt_lora_problem* problems, int32_t count, int32_t dtype,
                           void* workspace, size_t workspace_bytes, void* stream);

/* --------------------------------------------------------------------------------------
 * attt_lora_sgd_step: the adapter update of Eq. 2 and Algorithm 1 (the parameter step that
 * follows the gradient of the weighted loss), theta <- theta - lr * grad, for adapter
 * parameters kept in float32. Per element, in float32: the product lr * grad is rounded to
 * nearest, then the difference is (two roundings, no fused multiply-add), so any IEEE float32
 * evaluation of  param - lr * grad  reproduces the result bit for bit.
 *
 * params  HOST array of `count` descriptors, processed as one grouped launch:
 *   param       device float [n], updated in place
 *   grad        device float [n]; read, then set to 0 when zero_grad != 0, ready for the next
 *               accumulation by attt_lora_grad (whose dA / dB are +=)
 *   param_bf16  device bf16 [n] or NULL: the updated param rounded to nearest even, the operand
 *               copy that the next bf16 attt_lora_grad call reads as A or B
 *   0 <= n < 2^31 (ATTT_EUNSUPPORTED beyond); descriptors with n == 0 are skipped
 * lr      finite (the paper's setting is 5e-4, two steps per update)
 * Arrays are caller-owned; param and grad 4-byte aligned, param_bf16 2-byte aligned; no array
 * may overlap another of any descriptor. Nothing is allocated; launches are asynchronous on
 * `stream`.
 * Errors: ATTT_EINVAL (count < 0, null params with count > 0, non-finite lr, n < 0, null param
 * or grad with n > 0, misalignment), ATTT_EUNSUPPORTED, ATTT_EHIP.
 * ------------------------------------------------------------------------------------ */
typedef struct attt_lora_param {
  float* param;
  float* grad;
  void* param_bf16;
  int64_t n;
} attt_lora_param;

attt_status attt_lora_sgd_step(const attt_lora_param* params, int32_t count, float lr, int32_t zero_grad,
                               void* stream);

/* --------------------------------------------------------------------------------------
 * Serving side: grouped multi-adapter forward. Concurrent episodes (16 in the paper's runs)
 * decode through one base model, each with its own episode adapter (Appendix A; adapter of
 * Sec. 3.1, rank and alpha in Appendix C). The adapted projection is
 *     y = x W0^T + scale * (x A^T) B^T.
 * The base product x W0^T is a plain GEMM the caller has already written into y; this call
 * adds the adapter term of every (episode, projection) in one grouped launch:
 *     y <- RN_bf16(y + scale * (x A^T) B^T)
 * with x A^T and the sum over the rank in float32, one rounding to bf16 (nearest even) at the
 * end. A result can differ from the correctly rounded value of the exact sum by one bf16 ulp
 * where that sum lies within float32 error of a rounding boundary. Deterministic.
 *
 * problems   HOST array of `count` descriptors (typically one per episode and projection):
 *   x      device bf16 [rows, d_in]   (the rows of one episode)
 *   y      device bf16 [rows, d_out]  read and written in place
 *   A      device bf16 [rank, d_in]
 *   B      device bf16 [d_out, rank]
 *   rows >= 0 (0: skipped), d_in and d_out positive multiples of 8, 1 <= rank <=
 *   ATTT_LORA_MAX_RANK; rows < 2^24 and d_in, d_out < 2^20 (ATTT_EUNSUPPORTED beyond);
 *   scale finite. x, y, A, B 16-byte aligned. The y of different problems must not overlap
 *   each other or any input. Problems with the same x pointer, d_in and rows (q, k and v of
 *   one layer) are computed together, x read once for up to 64 of their combined (16-padded)
 *   ranks.
 * Nothing is allocated and no workspace is needed (x A^T stays on chip). Asynchronous on
 * `stream`. Errors (before any HIP call): ATTT_EINVAL, ATTT_EUNSUPPORTED; ATTT_EHIP.
 * ------------------------------------------------------------------------------------ */
typedef struct attt_lora_fwd_problem {
  const void* x;
  void* y;
  const void* A;
  const void* B;
  int64_t rows;
  int64_t d_in;
  int64_t d_out;
  int32_t rank;
  float scale;
} attt_lora_fwd_problem;

attt_status attt_lora_forward(const attt_lora_fwd_problem* problems, int32_t count, void* stream);

/* --------------------------------------------------------------------------------------
 * Adapter hot swap into serving (Appendix A: the adapter trained by an update replaces the
 * episode's serving adapter): every float32 tensor of an adapter (the masters that
 * attt_lora_sgd_step updates) rounded to nearest even into the bf16 copy that
 * attt_lora_forward reads, in one launch per 96 tensors. Bit-exact.
 *
 * items  HOST array of `count` descriptors:
 *   src  device float [n]
 *   dst  device bf16 [n], written
 *   0 <= n < 2^31 (ATTT_EUNSUPPORTED beyond); n == 0 is skipped; src 4-byte and dst 2-byte
 *   aligned (16-byte alignment of both takes the vector path); no dst may overlap any array.
 * Ordered before later work on `stream`: a forward launched after the swap on the same stream
 * reads the new adapter. Errors: ATTT_EINVAL, ATTT_EUNSUPPORTED, ATTT_EHIP.
 * ------------------------------------------------------------------------------------ */
typedef struct attt_lora_swap_item {
  const float* src;
  void* dst;
  int64_t n;
} attt_lora_swap_item;

attt_status attt_lora_hot_swap(const attt_lora_swap_item* items, int32_t count, void* stream);

/* --------------------------------------------------------------------------------------
 * Kernel timing (diagnostics). When enabled, every launch of a named kernel is bracketed
 * by HIP events recorded on the launch stream. attt_timing_read waits for those events and
 * returns the summed duration and launch count of one kernel since the last reset; names
 * are those attt_timing_kernel_name enumerates. Not thread-safe against concurrent calls.
 * ------------------------------------------------------------------------------------ */
attt_status attt_timing_enable(int32_t on);
attt_status attt_timing_reset(void);
attt_status attt_timing_read(const char* kernel, double* total_ms, int64_t* launches);
/* Name of kernel number i (0-based), or NULL past the last one. */
const char* attt_timing_kernel_name(int32_t i);

#ifdef __cplusplus
}
#endif

#endif /* ATTT_H_ */
