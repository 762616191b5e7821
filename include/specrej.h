/*
 * specrej.h -- C interface of the MI355X (gfx950) Speculative Rejection
 * library (Sun et al., "Fast Best-of-N Decoding via Speculative Rejection",
 * NeurIPS 2024).
 *
 * Problem (section 3, "Inference-time Alignment"; Algorithm 1 of section
 * 4.2): given a prompt x, an auto-regressive generator p, a reward model s,
 * a number of candidates N, a rejection rate alpha and a decision token tau,
 * return the response with the highest reward among the completed
 * candidates, and its reward.  alpha = 0 is plain Best-of-N (section 5.1).
 *
 * Conventions shared by every entry point:
 *  - All functions return an sr_status; SR_OK is 0.  On any other status,
 *    sr_last_error() returns a message for the calling thread.  No C++
 *    exception crosses this interface.
 *  - Arguments are validated before any device work: an invalid call
 *    changes no memory and launches nothing.
 *  - The caller owns all memory.  Device pointers (weights, workspaces,
 *    buffers of the kernel-level entry points) must stay valid until the
 *    call's work on `stream` has finished; host pointers are borrowed for
 *    the duration of the call.  The library allocates no device memory.
 *  - `stream` is a hipStream_t (NULL = the default stream).  sr_generate
 *    and sr_reward_scores/sr_logits_teacher_forced block until their work
 *    is done; the other kernel-level entry points are asynchronous.
 *  - Calls are re-entrant given distinct workspaces and streams.
 *  - Matrices are row-major; weight matrices are stored [out][in].
 */
#ifndef SPECREJ_H
#define SPECREJ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SR_OK = 0,
  SR_ERR_INVALID_ARG = 1,          /* an argument is out of range or inconsistent */
  SR_ERR_WORKSPACE_TOO_SMALL = 2,  /* ws_bytes below what sr_workspace_size reports */
  SR_ERR_UNSUPPORTED = 3,          /* a valid shape this build has no kernel for */
  SR_ERR_DEVICE = 4,               /* a HIP call failed */
  SR_ERR_INTERNAL = 5              /* an internal consistency check failed */
} sr_status;

typedef enum { SR_F32 = 0, SR_BF16 = 1 } sr_dtype;

/* Shape of a pre-norm Llama-style decoder (section 5 uses Llama-3-8B and
 * Mistral-7B-shaped generators and reward models):
 * h = E[tok]; per layer h += Wo attn(rope(Wq a), rope(Wk a), Wv a) with
 * a = RMSNorm(h) * g_attn, then h += W2 (silu(W1 f) * (W3 f)) with
 * f = RMSNorm(h) * g_ffn; out = RMSNorm(h) * g_final.  Query head j reads
 * KV head floor(j * n_kv_heads / n_heads).  Rotate-half RoPE with
 * frequencies rope_theta^(-2i/head_dim).  Attention scale 1/sqrt(head_dim).
 * Supported: head_dim in {32, 64, 128}; d_model, n_heads*head_dim and
 * ffn_dim multiples of 64; n_heads a multiple of n_kv_heads. */
typedef struct {
  int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, ffn_dim, vocab;
  float rope_theta, rms_eps;
  int32_t dtype;      /* sr_dtype of every weight tensor and of the KV cache */
  int32_t is_reward;  /* 0: generator, head = LM head [vocab][d_model];
                         1: reward model, head = scalar head [d_model] and the
                            score is head . out[last token] (no bias) */
} sr_model_config;

/* Device pointers to packed weights, element type = cfg.dtype. */
typedef struct {
  const void *embed;       /* [vocab][d]                                   */
  const void *attn_norm;   /* [nl][d]                                      */
  const void *wqkv;        /* [nl][(hq + 2 hkv) hd][d]: q rows, k rows, v rows */
  const void *wo;          /* [nl][d][hq hd]                               */
  const void *ffn_norm;    /* [nl][d]                                      */
  const void *w13;         /* [nl][2][ff][d]: gate (W1) then up (W3)       */
  const void *w2;          /* [nl][d][ff]                                  */
  const void *final_norm;  /* [d]                                          */
  const void *head;        /* generator [vocab][d]; reward model [d]       */
} sr_weights;

typedef struct {
  sr_model_config cfg;
  sr_weights w;
} sr_model;

/* Run parameters (Algorithm 1 of section 4.2).
 *  n            initial batch (number of candidates), >= 1.
 *  alpha        rejection rate in [0, 1); each cut keeps
 *               K = b - floor(round(alpha * 1e6) * b / 1e6) = ceil((1-alpha) b)
 *               of b candidates, ranked by reward descending then candidate
 *               index ascending (NaN lowest).
 *  tau          first decision token (response tokens), >= 1.  The KV
 *               budget is B = n * tau response-token slots; a round with b
 *               unfinished candidates at length L runs to
 *               D = min(max_new_tokens, floor(B / b)), cutting again at once
 *               while D <= L.  Rounds where no candidate can be rejected,
 *               and rounds after max_rounds cuts, run to max_new_tokens.
 *  max_new_tokens  maximum response length Lmax, >= 1.
 *  temperature  softmax temperature T > 0, or 0 for greedy decoding.
 *  seed         key of the Philox4x32-10 draws: the uniform for candidate k
 *               at step t is word 0 of Philox(counter (t, k, 0, 0),
 *               key (seed mod 2^32, seed div 2^32)).
 *  eos_id       end-of-sequence token (part of the response), -1 = none.
 *  max_rounds   maximum number of cuts, 0 = unlimited.
 *  profile_every  0 = off; k > 0 = time kernels with HIP events on `stream`
 *               during every k-th decode step and every reward/cut phase,
 *               accumulating into sr_result.kernel_* (costs one host
 *               synchronisation per timed step).
 *  reward_kind  SR_REWARD_MODEL: s(x, y) is the reward model `rm`;
 *               SR_REWARD_LOGPROB: s(y) = (1/len(y)) ln p(y | x) under the
 *               generator's own softmax at temperature 1 (section 5.3),
 *               accumulated during sampling; `rm` is not evaluated and may
 *               be NULL.
 *  reward_recompute  with the reward model and a schedule that scores more
 *               than once: 0 = the reward model's keys/values of the
 *               survivors' responses stay in the workspace across rounds
 *               (compacted at each cut like the generator's) and a decision
 *               runs only the tokens generated since the previous one; the
 *               workspace then holds two more pools of the generator pools'
 *               slot counts.  1 = every decision runs the whole responses
 *               through the reward model again.  Both give the same scores up
 *               to floating-point rounding order. */
enum { SR_REWARD_MODEL = 0, SR_REWARD_LOGPROB = 1 };
typedef struct {
  int32_t n;
  double alpha;
  int32_t tau, max_new_tokens;
  float temperature;
  uint64_t seed;
  int32_t eos_id;
  int32_t max_rounds;
  int32_t profile_every;
  int32_t reward_kind;
  int32_t reward_recompute;
} sr_params;

/* Kernel classes of sr_result.kernel_*. */
enum {
  SR_K_GEN_GEMM_MFMA = 0,   /* generator projections with >= 312 rows (MFMA-bound)  */
  SR_K_GEN_GEMM_HBM = 1,    /* generator projections with < 312 rows (weight-bound) */
  SR_K_DECODE_ATTN = 2,     /* decode attention (+ split merge)                      */
  SR_K_RM_GEMM = 3,         /* reward-model and prompt-prefill projections           */
  SR_K_PREFILL_ATTN = 4,    /* prefill attention                                     */
  SR_K_SAMPLE = 5,          /* sampler + state update                                */
  SR_K_CUT = 6,             /* cut, compaction, arg max                              */
  SR_K_OTHER = 7,           /* embedding, RMSNorm, RoPE, reward head, gathers        */
  SR_K_NCLASS = 8
};

/* kernel_sec/launches/bytes/flops: per kernel class, the event-measured time,
 * the number of timed launches and their algorithmic HBM bytes and flops
 * (the bytes and flops the operation itself must move or compute: every
 * weight, activation and KV element once).  Zero unless profile_every > 0. */
typedef struct {
  int32_t best_index;        /* candidate index k* (eq. output)              */
  float best_score;          /* s(x, y_k*)                                   */
  int32_t n_tokens;          /* length of y_k* (written to out_tokens)        */
  int32_t rounds;            /* number of cuts performed                     */
  int64_t generated_tokens;  /* response tokens sampled over all candidates  */
  double sec_total, sec_prefill, sec_decode, sec_reward, sec_cut;
  double kernel_sec[SR_K_NCLASS];
  int64_t kernel_launches[SR_K_NCLASS];
  double kernel_bytes[SR_K_NCLASS];
  double kernel_flops[SR_K_NCLASS];
} sr_result;

/* Optional host buffers filled by sr_generate for tests and tracing; any
 * pointer may be NULL.  Entries beyond `rounds` are left untouched.
 *  round_L, round_b, round_keep  [max_rounds_cap] length, batch and keep
 *                                count of every cut.
 *  round_cand, round_scores      [max_rounds_cap][n] candidate index and
 *                                partial reward of each of the round_b rows
 *                                (rows in ascending candidate order).
 *  round_accept                  [max_rounds_cap][n] 1 if that row was kept.
 *  all_tokens, all_len           [n][max_new_tokens], [n] every candidate's
 *                                response as far as it was generated.
 *  final_scores                  [n] reward of completed candidates (members
 *                                of the set I), NaN for rejected ones.
 *  watch_cand, n_watch,          the logits rows the run sampled from, for
 *  watch_logits                  n_watch >= 0 chosen candidates (HOST int32
 *                                watch_cand[n_watch], each in [0, n)):
 *                                watch_logits (HOST float
 *                                [n_watch][max_new_tokens][vocab]) row
 *                                [w][t] receives the generator's logits from
 *                                which response token t of candidate
 *                                watch_cand[w] was drawn, for every t below
 *                                that candidate's length; rows of later steps
 *                                hold unspecified values.  Costs one host copy
 *                                per watched row and step.  n_watch = 0 (or
 *                                watch_logits NULL) watches nothing. */
typedef struct {
  int32_t *round_L, *round_b, *round_keep;
  int32_t *round_cand;
  float *round_scores;
  int32_t *round_accept;
  int32_t *all_tokens, *all_len;
  float *final_scores;
  int32_t max_rounds_cap;
  const int32_t *watch_cand;
  int32_t n_watch;
  float *watch_logits;
} sr_trace;

/* Bytes of device workspace sr_generate needs for these models, prompt
 * length and parameters.  gen must be a generator, rm a reward model of the
 * same dtype.  Writes *bytes; fails with SR_ERR_INVALID_ARG on bad input. */
sr_status sr_workspace_size(const sr_model *gen, const sr_model *rm, int32_t prompt_len,
                            const sr_params *p, size_t *bytes);

/* Memory-driven sizing (Algorithm 1, first step: the initial batch and the
 * decision token follow from the memory available, as in section 5 where
 * the system finds how many tokens fit before memory runs out).  Given the
 * bytes the caller can give the workspace (for instance the device's free
 * memory after the weights), writes to *out a copy of *p whose
 *   - tau is the largest in [1, max_new_tokens] with
 *     sr_workspace_size(out) <= capacity_bytes, when p->n >= 1 (b_init = n
 *     given, the KV budget n * tau taken from memory); or
 *   - n is the largest in [1, 4096] with sr_workspace_size(out) <=
 *     capacity_bytes, when p->n == 0 (tau given, b_init taken from memory).
 * Every other field is copied.  SR_ERR_WORKSPACE_TOO_SMALL if even tau = 1
 * (or n = 1) does not fit; other errors as sr_workspace_size.  Host only. */
sr_status sr_plan_for_memory(const sr_model *gen, const sr_model *rm, int32_t prompt_len,
                             const sr_params *p, size_t capacity_bytes, sr_params *out);

/* Speculative Rejection (section 4.2, Algorithm 1; Best-of-N when alpha=0).
 *  prompt       HOST int32 [prompt_len], token ids in [0, vocab).
 *  workspace    DEVICE buffer of ws_bytes >= sr_workspace_size(...), 256-byte
 *               aligned; its contents on entry are ignored.
 *  out_tokens   HOST int32 [max_new_tokens]: receives y_k* (EOS included).
 *  out          HOST result summary.  trace: optional (NULL).
 * Blocks until done.  The returned response is the best member of I by
 * (reward descending, candidate index ascending). */
sr_status sr_generate(const sr_model *gen, const sr_model *rm, const int32_t *prompt,
                      int32_t prompt_len, const sr_params *p, void *workspace, size_t ws_bytes,
                      void *stream, int32_t *out_tokens, sr_result *out, sr_trace *trace);

/* K = ceil((1 - alpha) b) as computed by the cut (see sr_params); -1 if
 * b < 0 or alpha outside [0, 1). */
int32_t sr_keep_count(int32_t b, double alpha);

/* Message describing the last failure on the calling thread ("" if none). */
const char *sr_last_error(void);

/* ---- kernel-level entry points (used by the parity tests) -------------
 * Device pointers, asynchronous on `stream` unless stated. */

/* Philox4x32-10 (Salmon et al., SC'11): out[i] = Philox(ctr[i], key(seed)).
 * ctr, out: DEVICE uint32 [n][4]. */
sr_status sr_philox_fill(uint64_t seed, const uint32_t *ctr, int32_t n, uint32_t *out,
                         void *stream);

/* Next-token draw of eq. (auto-regressive), section 3: for each row r,
 * tokens[r] = the token drawn from softmax(logits[r] / T) by the exact
 * integer inverse CDF keyed by (seed, cand[r], step) -- see sr_params.seed.
 * logits: DEVICE float [rows][vocab]; cand: DEVICE int32 [rows];
 * tokens: DEVICE int32 [rows].  temperature 0 = first arg max. */
sr_status sr_sample(const float *logits, int32_t rows, int32_t vocab, const int32_t *cand,
                    int32_t step, float temperature, uint64_t seed, int32_t *tokens,
                    void *stream);

/* The cut of eqs. (cutoff-threshold) and (accepted-set), section 4.2:
 * accept[i] = 1 for the `keep` best of b rows by (scores[i] descending,
 * cand[i] ascending, NaN lowest), else 0.  scores: DEVICE float [b];
 * cand, accept: DEVICE int32 [b].  1 <= keep <= b <= 4096. */
sr_status sr_select(const float *scores, const int32_t *cand, int32_t b, int32_t keep,
                    int32_t *accept, void *stream);

/* Stream compaction of the KV cache after a cut (section 4.2, "Promising
 * Utterances for Next Round"): rows with keep_flag[i] != 0 are packed, in
 * order, from `src` (row capacity cap_src tokens) into `dst` (row capacity
 * cap_dst): for every layer l, kv in {K, V}, kept row i -> new row j, head h,
 * t < len: dst[l][kv][j][h][t][:] = src[l][kv][i][h][t][:].
 * A pool holds 2 * n_layers blocks, block (l, kv) starting at element
 * (2 l + kv) * block_elems and laid out [rows][n_kv_heads][cap][head_dim];
 * elements are `elem_bytes` (2 or 4) bytes.  src, dst: DEVICE, not
 * overlapping.  keep_flag: DEVICE int32 [b].  src_row: DEVICE int32 [b],
 * receives the source row of every kept row in order.  new_count: DEVICE
 * int32 [1], receives the number of kept rows.  Requires 1 <= b <= 4096,
 * len <= cap_src, len <= cap_dst, b * n_kv_heads * cap_src * head_dim <=
 * src_block_elems and b * n_kv_heads * cap_dst * head_dim <= dst_block_elems.
 * Rows of dst beyond the kept ones and tokens beyond len are not written. */
sr_status sr_compact(const void *src, int64_t src_block_elems, void *dst,
                     int64_t dst_block_elems, const int32_t *keep_flag, int32_t b,
                     int32_t n_layers, int32_t n_kv_heads, int32_t head_dim, int32_t elem_bytes,
                     int32_t cap_src, int32_t cap_dst, int32_t len, int32_t *src_row,
                     int32_t *new_count, void *stream);

/* One projection of the decoder (the dense contraction of sections a3, a5,
 * a6 and a7 of the hot path): with X [M][K] and W [N][K] (dtype elements,
 * row-major, DEVICE),
 *   mode 0: out (float [M][N])  = X W^T
 *   mode 1: out (float [M][N]) += X W^T                      (residual add)
 *   mode 2: out (dtype [M][N])  = silu(X W1^T) * (X W3^T)     (SwiGLU; W holds
 *           [2][N][K]: W1 rows then W3 rows)
 *   mode 3: out (dtype [M][N])  = X W^T
 * fp32 accumulation.  partial: DEVICE float scratch of partial_elems >=
 * sr_projection_scratch(dtype, M, N, K, mode) elements (may be NULL when that
 * is 0).  K must be a multiple of 64.  Asynchronous. */
sr_status sr_projection(int32_t dtype, const void *x, const void *w, int32_t M, int32_t N,
                        int32_t K, int32_t mode, void *out, float *partial, size_t partial_elems,
                        void *stream);
size_t sr_projection_scratch(int32_t dtype, int32_t M, int32_t N, int32_t K, int32_t mode);

/* Decode attention of `rows` candidates (section a4 of the hot path; the
 * attention step of the decoder in section 4.2 with the prompt's keys stored
 * once): for row r and query head j, the single query q[r][j] (DEVICE float
 * [rows][n_heads][head_dim]) attends the keys/values of KV head
 * floor(j * n_kv_heads / n_heads): first the shared prefix kpre/vpre (DEVICE
 * dtype [n_kv_heads][P][head_dim]), then the row's own tail ktail/vtail
 * (DEVICE dtype [rows][n_kv_heads][cap][head_dim], tokens 0..lt-1 used);
 * out[r][j*head_dim + d] (DEVICE dtype [rows][n_heads*head_dim]) =
 * sum_k softmax_k(q . key_k / sqrt(head_dim)) value_k[d].  P + lt >= 1,
 * lt <= cap, head_dim in {32, 64, 128}, n_heads / n_kv_heads in {1,2,4,8}.
 * scratch: DEVICE float scratch of >= sr_decode_attention_scratch(...)
 * floats (split-K partials).  Asynchronous. */
sr_status sr_decode_attention(int32_t dtype, int32_t head_dim, int32_t n_heads, int32_t n_kv_heads,
                              int32_t rows, const float *q, const void *kpre, const void *vpre,
                              int32_t P, const void *ktail, const void *vtail, int32_t cap,
                              int32_t lt, void *out, float *scratch, size_t scratch_elems,
                              void *stream);
size_t sr_decode_attention_scratch(int32_t head_dim, int32_t n_heads, int32_t n_kv_heads,
                                   int32_t rows, int32_t P, int32_t lt);

/* The decode attention of sr_decode_attention without a caller scratch
 * buffer, for callers that cannot allocate device memory (code under graph
 * capture, serving loops that forbid allocation).  Same arguments, kernels
 * and results; the split partials go to a file-scope device array of
 * sr_decode_attention_noalloc_limit() bytes (32 MiB) that each device holds
 * once the library first runs this entry point on it, until the process
 * ends.  Calls whose partials exceed it (rows * n_heads * splits *
 * (head_dim + 2) floats, splits chosen by the kernel dispatch; up to 1024
 * rows of 32 query heads of 128 fit) fail with SR_ERR_WORKSPACE_TOO_SMALL
 * before any launch.  No device memory is allocated or freed.  Every call
 * on one device shares the array: calls that overlap on a device (other
 * streams, other threads) race and must be serialised by the caller.
 * Asynchronous. */
sr_status sr_decode_attention_noalloc(int32_t dtype, int32_t head_dim, int32_t n_heads, int32_t n_kv_heads,
                                      int32_t rows, const float *q, const void *kpre, const void *vpre, int32_t P,
                                      const void *ktail, const void *vtail, int32_t cap, int32_t lt, void *out,
                                      void *stream);
size_t sr_decode_attention_noalloc_limit(void);

/* Causal prefill attention of `rows` rows of lr new tokens each, which follow
 * t0 tokens of the same row whose keys/values are already cached (the
 * reward model's scoring pass over the tokens generated since the previous
 * decision, section 4.2; t0 = 0 scores whole responses).  New token t of row
 * r sits at row position t0 + t; its query q[r*lr + t][j] (DEVICE float
 * [rows*lr][n_heads][head_dim]) attends, for KV head
 * floor(j * n_kv_heads / n_heads), the shared prefix kpre/vpre (DEVICE dtype
 * [n_kv_heads][P][head_dim]) and the row's own keys/values 0..t0 + t in
 * kown/vown (DEVICE dtype [rows][n_kv_heads][cap][head_dim]; positions
 * t0..t0+lr-1 are the new tokens' own, written by the caller);
 * out[r*lr + t][j*head_dim + d] (DEVICE dtype [rows*lr][n_heads*head_dim]) =
 * sum_k softmax_k(q . key_k / sqrt(head_dim)) value_k[d].  t0 + lr <= cap,
 * head_dim in {32, 64, 128}, n_heads / n_kv_heads in {1,2,4,8}; bf16 with
 * head_dim 128 runs on the matrix cores.  No scratch.  Asynchronous. */
sr_status sr_prefill_attention(int32_t dtype, int32_t head_dim, int32_t n_heads, int32_t n_kv_heads,
                               int32_t rows, int32_t lr, const float *q, const void *kpre,
                               const void *vpre, int32_t P, const void *kown, const void *vown,
                               int32_t cap, int32_t t0, void *out, void *stream);

/* Teacher-forced generator logits through the decode path: all `rows`
 * continue `prompt` (HOST int32 [prompt_len]) with their own tokens
 * (DEVICE int32 [rows][len]); logits_out (DEVICE float [rows][len][vocab])
 * row (r, t) is the distribution of response token t given the prompt and
 * tokens[r][0..t).  Every token must lie in [0, vocab) (checked).  Uses the
 * workspace of an sr_generate call with p->n >= rows,
 * p->max_new_tokens >= len and rows * len <= p->n * tau-budget pool (the
 * first pool of that workspace).  Blocks until done. */
sr_status sr_logits_teacher_forced(const sr_model *gen, const sr_model *rm,
                                   const int32_t *prompt, int32_t prompt_len,
                                   const sr_params *p, const int32_t *tokens, int32_t rows,
                                   int32_t len, float *logits_out, void *workspace,
                                   size_t ws_bytes, void *stream);

/* Rewards s(x, y_r) of eq. (partial-reward-set), section 4.2, for `rows`
 * responses (DEVICE int32 [rows][max_len], row r has lens[r] >= 1 tokens;
 * lens: DEVICE int32 [rows]) after `prompt` (HOST int32 [prompt_len]).
 * scores: DEVICE float [rows].  1 <= lens[r] <= max_len and the first
 * lens[r] tokens of each row in [0, vocab) (checked).  Uses the workspace of
 * an sr_generate call with p->n >= rows and p->max_new_tokens >= max_len.
 * Blocks until done. */
sr_status sr_reward_scores(const sr_model *gen, const sr_model *rm, const int32_t *prompt,
                           int32_t prompt_len, const sr_params *p, const int32_t *tokens,
                           const int32_t *lens, int32_t rows, int32_t max_len, float *scores,
                           void *workspace, size_t ws_bytes, void *stream);

/* Evaluation diagnostics (host arrays, host only, double precision).
 * Pearson correlation and Kendall's coefficient of n >= 2 finite pairs, as
 * Appendix B defines them for the partial and final rewards of one
 * prompt's candidates: Kendall = 2 / (n (n - 1)) * sum over i < j of
 * sgn(x_i - x_j) sgn(y_i - y_j), tied pairs counting zero (O(n^2) pairs).
 * *pearson is NaN when either sample is constant.  SR_ERR_INVALID_ARG on
 * NULL pointers, n < 2 or non-finite values. */
sr_status sr_correlation(const float *x, const float *y, int32_t n, double *pearson, double *kendall);

/* Improvement score of section 5 (eq. subopt.experiment): the reward of the
 * Speculative Rejection answer sr_reward placed on the range of the n >= 1
 * Best-of-N rewards bon_rewards (HOST float [n]):
 * (1 - (max - sr_reward) / (max - min)) * 100; NaN when max == min.
 * SR_ERR_INVALID_ARG on NULL pointers, n < 1 or non-finite values. */
sr_status sr_improvement_score(const float *bon_rewards, int32_t n, float sr_reward, double *score);

#ifdef __cplusplus
}
#endif

#endif /* SPECREJ_H */
