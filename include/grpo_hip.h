/*
 * grpo_hip.h — C-ABI of the GRPO rollout / scoring / loss hot path on MI355X.
 *
 * The paper fine-tunes a Llama-family decoder with GRPO (Sec. VI-A, Alg. 1):
 * each iteration samples K completions per prompt from the policy, scores
 * them, normalises rewards within each group into advantages and applies the
 * clipped-ratio objective with a KL penalty towards a frozen reference copy
 * (Eq. 1).  Sec. I and Sec. VI-C name sample generation as the step that
 * dominates training time.  This library exposes that path as HIP kernels for
 * gfx950:
 *
 *   grpo_prefill          prompt forward + first sampled token of each group
 *                         member (Alg. 1, sampling step, generation step 0)
 *   grpo_rollout_step     n_steps batched decode steps (Alg. 1, sampling step)
 *   grpo_rollout_step_grouped  the same, reading each group's shared prompt
 *                         K/V once per group
 *   grpo_score_sequences  teacher-forced log pi(x_t | c, x_<t) (Eq. 1, KL term)
 *   grpo_score_sequences_grouped  the same, the group's shared prompt run once
 *   grpo_advantages       group-normalised rewards w(x) (Alg. 1, normalisation)
 *   grpo_token_loss       clipped-ratio + KL per-token loss, its gradient with
 *                         respect to logp, and statistics (Eq. 1, GRPO form)
 *
 * Conventions
 *  - Every tensor pointer is a DEVICE pointer owned by the caller.  The library
 *    allocates no device memory: scratch space comes from the caller's
 *    workspace (size from grpo_workspace_bytes).  A model handle keeps the
 *    weight pointers (host copies of the pointer values, not of the weights);
 *    the weights must outlive the handle.
 *  - Every compute call is asynchronous on `stream` (a hipStream_t passed as
 *    void*, NULL = the null stream).  Device faults surface at the caller's
 *    next synchronisation.
 *  - Every call returns 0 (GRPO_OK) or a negative grpo_status.  Arguments are
 *    validated on the host BEFORE anything is enqueued, so a rejected call
 *    leaves no partial work; grpo_last_error() returns a thread-local message.
 *  - Outputs never alias inputs.  Results are bit-deterministic for identical
 *    inputs and launch configuration: fixed-order reductions, no float atomics.
 *  - Weight matrices are row-major [out, in] (nn.Linear layout).  The model
 *    dtype (fp32 or bf16) is the dtype of every weight and of the KV cache.
 *
 * Precision contract (bf16 models): weights and KV in bf16; residual stream,
 * accumulation, softmax, logits and log-probs in fp32; bf16 round-to-nearest-
 * even at the inputs of the matrix products (normed activations, q/k after
 * RoPE and v, attention output, SwiGLU output, final normed state).  fp32
 * models round nowhere.
 */
#ifndef GRPO_HIP_H
#define GRPO_HIP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum grpo_status {
  GRPO_OK = 0,
  GRPO_INVALID_ARG = -1,          /* null pointer, bad size or range            */
  GRPO_UNSUPPORTED = -2,          /* shape/dtype outside what the kernels cover */
  GRPO_WORKSPACE_TOO_SMALL = -3,  /* ws_bytes below grpo_workspace_bytes(...)   */
  GRPO_HIP_ERROR = -4,            /* a HIP runtime call failed                  */
  GRPO_KV_CAPACITY = -5           /* positions would run past the KV capacity   */
};

enum grpo_dtype { GRPO_F32 = 0, GRPO_BF16 = 1 };

/* Workspace kinds for grpo_workspace_bytes. */
enum grpo_op {
  GRPO_OP_PREFILL = 0, GRPO_OP_ROLLOUT = 1, GRPO_OP_SCORE = 2, GRPO_OP_LOSS = 3,
  GRPO_OP_EXTEND = 4, GRPO_OP_BACKWARD = 5
};

/* Decoder shape.  Llama family: RMSNorm, RoPE (half-split pairs (i, i+hd/2),
 * angle pos * rope_theta^(-2i/hd)), grouped-query attention (query head h reads
 * kv head floor(h*n_kv_heads/n_heads)), SwiGLU MLP, untied LM head, no biases.
 * Supported: head_dim in {64, 128}; n_heads a multiple of n_kv_heads; d_model,
 * n_heads*head_dim and d_ffn multiples of 128 (of 32 for fp32 models); vocab
 * a multiple of 16 for bf16 models. */
typedef struct grpo_config {
  int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, d_ffn, vocab;
  float rms_eps, rope_theta;
  int32_t dtype; /* enum grpo_dtype */
} grpo_config;

/* Device pointers to the weights.  Per-layer entries are HOST arrays of
 * n_layers device pointers; the handle copies those arrays. */
typedef struct grpo_weights {
  const void* tok_emb;            /* [vocab, d]                       */
  const void* const* attn_norm;   /* L x [d]                          */
  const void* const* wq;          /* L x [n_heads*hd, d]              */
  const void* const* wk;          /* L x [n_kv_heads*hd, d]           */
  const void* const* wv;          /* L x [n_kv_heads*hd, d]           */
  const void* const* wo;          /* L x [d, n_heads*hd]              */
  const void* const* mlp_norm;    /* L x [d]                          */
  const void* const* w_gate;      /* L x [d_ffn, d]                   */
  const void* const* w_up;        /* L x [d_ffn, d]                   */
  const void* const* w_down;      /* L x [d, d_ffn]                   */
  const void* final_norm;         /* [d]                              */
  const void* lm_head;            /* [vocab, d]                       */
} grpo_weights;

/* Sampler.  z = logits / temperature.  temperature == 0 is greedy (lowest id
 * among the maxima; logp then uses temperature 1).  top_k > 0 restricts the
 * draw to the top_k logits ordered by (value desc, id asc).  Otherwise
 * Gumbel-max: token = lowest id among the maxima over the allowed set of
 * z_i - ln(-ln u_i), u_i = (2*(w >> 9) + 1) * 2^-24, w = word (i & 3) of
 * Philox4x32-10(key = (seed mod 2^32, seed >> 32), ctr = (i >> 2, step, seq, 0)).
 * The log-prob is always the full-vocabulary log_softmax(z)[token]. */
typedef struct grpo_sampling {
  float temperature;
  int32_t top_k;
  uint64_t seed;
} grpo_sampling;

/* Intermediate values of a forward pass, for parity tests that check each
 * rounding point of the precision contract against the plain definition fed
 * the same inputs.  Every member is NULL (not captured) or a DEVICE fp32
 * buffer, row-major; values stored in bf16 by the forward are written exactly
 * (as fp32).  "rows" is the entry point's row set:
 *   grpo_prefill:          R = P * Tp prompt rows (prompt-major); head rows = P
 *                          (the last position of each prompt)
 *   grpo_rollout_step[_grouped]: R = B batch rows, the call's last step
 *   grpo_score_sequences[_grouped]: R = N * T rows (sequence-major; rows a call
 *                          does not compute are left unwritten: the grouped call
 *                          computes no row T-1); head rows = N * (T - score_from),
 *                          the scored positions score_from-1 .. T-2
 * A call with a trace runs without graph replay.
 *   x        [n_layers + 1][R][d]   residual entering each layer, then leaving the last
 *   x_attn   [n_layers][R][d]       residual after the attention block (x + o Wo^T)
 *   h_attn   [n_layers][R][d]       normed input of the QKV projection
 *   q        [n_layers][R][H*hd]    queries after RoPE
 *   k, v     [n_layers][R][Hkv*hd]  keys after RoPE and values, as cached
 *   o        [n_layers][R][H*hd]    attention output
 *   h_mlp    [n_layers][R][d]       normed input of the gate/up projection
 *   act      [n_layers][R][d_ffn]   SwiGLU output
 *   h_final  [head rows][d]         normed input of the LM head
 *   logits   [head rows][vocab]     fp32 logits (decode: the sampler's input) */
typedef struct grpo_trace {
  float* x;
  float* x_attn;
  float* h_attn;
  float* q;
  float* k;
  float* v;
  float* o;
  float* h_mlp;
  float* act;
  float* h_final;
  float* logits;
} grpo_trace;

typedef struct grpo_model grpo_model;

/* Creates a handle over caller-owned weights.  Validates the shape (see
 * grpo_config).  Returns GRPO_INVALID_ARG / GRPO_UNSUPPORTED on bad input. */
int grpo_model_create(const grpo_config* cfg, const grpo_weights* w, grpo_model** out);
int grpo_model_destroy(grpo_model* m);

/* Decode copy of the projections (bf16 models).  A decode step multiplies a
 * few rows by every weight matrix (Alg. 1, sampling step), so it streams the
 * weights from HBM once per step; the decode GEMM reads them from a copy stored
 * in MFMA fragment order (16 rows x 32 columns as 1 KB in lane order; the
 * fragments of all 16-row blocks at one 32-column step consecutive, the steps in
 * column order; gate and up blocks alternate) so that every load is 1 KB of
 * contiguous memory.
 * grpo_decode_weights_bytes: bytes of that copy (0 for fp32 models or an
 * invalid config).
 * grpo_model_pack_decode: writes the copy of the handle's current weights into
 * buf (device, caller-owned, 256-byte aligned, >= grpo_decode_weights_bytes)
 * on `stream` and makes the handle's decode steps read it.  buf must outlive
 * the handle's use; call again after the weights change.  Required before
 * grpo_rollout_step on a bf16 model (GRPO_INVALID_ARG otherwise); a no-op for
 * fp32 models.  Returns GRPO_INVALID_ARG for a NULL handle or buffer, or a
 * buffer that is too small or misaligned. */
size_t grpo_decode_weights_bytes(const grpo_config* cfg);
int grpo_model_pack_decode(grpo_model* m, void* buf, size_t bytes, void* stream);

/* Bytes of a KV cache for n_seqs sequences of max_len positions.  Layout:
 * [n_layers][2 (K, V)][n_seqs][n_kv_heads][max_len][head_dim], model dtype.
 * Returns 0 for invalid arguments. */
size_t grpo_kv_cache_bytes(const grpo_config* cfg, int32_t n_seqs, int32_t max_len);

/* Workspace bytes of one call (0 for invalid arguments):
 *   GRPO_OP_PREFILL: n_rows = prompts P, seq_len = prompt length Tp
 *   GRPO_OP_ROLLOUT: n_rows = batch B,   seq_len = KV capacity max_len
 *   GRPO_OP_SCORE:   n_rows = sequences N, seq_len = T
 *   GRPO_OP_EXTEND:  n_rows = batch B,   seq_len = KV capacity max_len
 *   GRPO_OP_LOSS:    n_rows = sequences N, seq_len = Tr (model may be NULL)
 *   GRPO_OP_BACKWARD: n_rows = sequences N, seq_len = T (at most 16384) */
size_t grpo_workspace_bytes(const grpo_model* m, int32_t op, int32_t n_rows, int32_t seq_len);

/* Thread-local message of the last failed call on this thread ("" if none). */
const char* grpo_last_error(void);

/* Rollout generation step 0 (Alg. 1, sampling step): causal forward over every
 * prompt (once per prompt, not per sample), its K/V written into the G cache
 * slots p*G .. p*G+G-1, then G draws from the last position's logits with
 * Philox sequence id p*G+g and step 0.
 *   prompts   int32 [P, Tp] token ids in [0, vocab)
 *   kv        cache of n_seqs >= P*G sequences, max_len >= Tp
 *   tok_out   int32 [P*G] sampled tokens;  logp_out  fp32 [P*G]
 *   trace     NULL or the intermediates to capture (see grpo_trace)
 * Ids outside [0, vocab) are clamped by the kernels (memory safety only). */
int grpo_prefill(const grpo_model* m, void* kv, int32_t n_seqs, int32_t max_len,
                 const int32_t* prompts, int32_t P, int32_t Tp, int32_t G,
                 const grpo_sampling* s, int32_t* tok_out, float* logp_out,
                 const grpo_trace* trace, void* ws, size_t ws_bytes, void* stream);

/* n_steps decode steps for batch rows 0..B-1 (Alg. 1, sampling step).  Row b
 * is sequence seq_ids[b]: its K/V live in cache slot seq_ids[b] and its draws
 * use Philox sequence id seq_ids[b], so a row set that changes between calls
 * (sequences paused for a tool call, finished ones replaced) continues every
 * sequence exactly where it stopped.  Per step: token tok[b] enters at position
 * pos[b] (its K/V written there), attention over positions 0..pos[b], the next
 * token is drawn with Philox step step0+s and written to tok[b] and
 * tok_out[b, s], its log-prob to logp_out[b, s]; pos[b] += 1.
 *   seq_ids    HOST int32 [B], distinct, each in [0, n_seqs); NULL means
 *              seq_ids[b] = b.  Read before the call returns.
 *   pos, tok   int32 [B] device, in/out
 *   max_pos    host hint: the largest pos[b] on entry.  The call is rejected
 *              with GRPO_KV_CAPACITY unless max_pos + n_steps <= max_len; the
 *              kernels additionally never touch positions >= max_len.
 *   tok_out    int32 [B, n_steps];  logp_out  fp32 [B, n_steps]
 *   trace      NULL or the intermediates of the last step (see grpo_trace)
 * B <= 128 for bf16 models.  On bf16 models without a top-k cut the draw is
 * fused into the LM head (its logits are not stored; the same tokens as the
 * sampler on those logits).  With n_steps >= 2 and no trace the step is
 * captured once as a HIP graph and replayed n_steps times; the graph is kept in
 * the model handle and recaptured when an argument changes, so a handle must
 * not be used from two threads at once.  GRPO_INVALID_ARG for seq_ids out of
 * range or repeated. */
int grpo_rollout_step(const grpo_model* m, void* kv, int32_t n_seqs, int32_t max_len, int32_t B,
                      const int32_t* seq_ids, int32_t* pos, int32_t* tok, int32_t max_pos,
                      int32_t step0, int32_t n_steps, const grpo_sampling* s, int32_t* tok_out,
                      float* logp_out, const grpo_trace* trace, void* ws, size_t ws_bytes,
                      void* stream);

/* grpo_rollout_step for a batch of groups: rows g*G .. g*G+G-1 are the G
 * samples of one prompt (Alg. 1 samples G completions per prompt; grpo_prefill
 * lays them out so), and their cache positions 0 .. prefix_len-1 hold the same
 * K/V (the prompt, written once per prompt by grpo_prefill into every member's
 * slot).  Attention reads those positions once per group, from the slot of row
 * g*G (seq_ids[g*G]), instead of once per row; each row's later positions come
 * from its own slot.  Every row must be at pos[b] >= prefix_len on entry (true
 * after grpo_prefill with prefix_len = Tp), so that no step writes a shared
 * position; the kernels cut the shared length to min(prefix_len, pos[b] + 1)
 * over a group's rows, so they never read past a row's own context.  Under
 * these conditions the results are those of grpo_rollout_step except for the
 * order of floating-point additions in attention.  Arguments as
 * grpo_rollout_step, plus
 *   G           group size, >= 1, dividing B
 *   prefix_len  shared positions, 0 <= prefix_len <= max_len (0: no sharing)
 * fp32 models read every row's own cache (same results).  The workspace is the
 * one grpo_workspace_bytes(GRPO_OP_ROLLOUT) gives.  GRPO_INVALID_ARG for a G or
 * prefix_len outside these ranges. */
int grpo_rollout_step_grouped(const grpo_model* m, void* kv, int32_t n_seqs, int32_t max_len,
                              int32_t B, int32_t G, int32_t prefix_len, const int32_t* seq_ids,
                              int32_t* pos, int32_t* tok, int32_t max_pos, int32_t step0,
                              int32_t n_steps, const grpo_sampling* s, int32_t* tok_out,
                              float* logp_out, const grpo_trace* trace, void* ws,
                              size_t ws_bytes, void* stream);

/* Tool-output injection into live sequences (Sec. V-B: the model emits a tool
 * call, the tool's output is placed into its context and generation resumes;
 * Sec. VI-C: group members not waiting on a tool keep decoding).  For each row
 * b, sequence seq_ids[b] (cache slot and Philox sequence id, as in
 * grpo_rollout_step) receives the Te tokens tokens[b, :] at positions
 * pos0[b] .. pos0[b] + Te - 1: a causal forward of those rows over the
 * sequence's cached positions 0 .. pos0[b] - 1 and the span itself, their K/V
 * written into the cache; then the next token is drawn from the span's last
 * position with Philox step `step` (tok_out[b], logp_out[b] as in
 * grpo_rollout_step).  The injected tokens are context, not samples: they get no
 * log-probability (their loss mask is 0).  Rows may sit at different positions;
 * rows not in the call keep their cache untouched (a paused or finished
 * sequence simply is not listed).  Generation continues with grpo_rollout_step
 * from pos = pos0[b] + Te, tok = tok_out[b].
 *   seq_ids  HOST int32 [B] (NULL: b), distinct, in [0, n_seqs)
 *   pos0     HOST int32 [B], pos0[b] >= 0, pos0[b] + Te <= max_len
 *            (GRPO_KV_CAPACITY otherwise)
 *   tokens   DEVICE int32 [B, Te]; 1 <= Te <= GRPO_EXTEND_CHUNK (a longer
 *            output is injected by consecutive calls, pos0 advancing by Te)
 *   trace    NULL or the intermediates (rows R = B * Te; head rows = B)
 * Workspace: grpo_workspace_bytes(GRPO_OP_EXTEND, B, max_len). */
#define GRPO_EXTEND_CHUNK 512
int grpo_extend(const grpo_model* m, void* kv, int32_t n_seqs, int32_t max_len, int32_t B,
                const int32_t* seq_ids, const int32_t* pos0, const int32_t* tokens, int32_t Te,
                int32_t step, const grpo_sampling* s, int32_t* tok_out, float* logp_out,
                const grpo_trace* trace, void* ws, size_t ws_bytes, void* stream);

/* Teacher-forced scoring (Eq. 1's log pi and the KL term's reference): for
 * j in [score_from, T): logp_out[n, j - score_from] =
 * log_softmax(logits at position j-1 / temperature)[tokens[n, j]]
 * (temperature 0 is read as 1; a token outside [0, vocab) is read as the
 * nearest id).  tokens int32 [N, T]; 1 <= score_from < T.  The log-softmax is
 * fused into the LM-head product: the [rows, vocab] logits are not stored.
 * trace: NULL or the intermediates to capture (see grpo_trace; its logits are
 * then computed by a second product). */
int grpo_score_sequences(const grpo_model* m, const int32_t* tokens, int32_t N, int32_t T,
                         int32_t score_from, float temperature, float* logp_out,
                         const grpo_trace* trace, void* ws, size_t ws_bytes, void* stream);

/* grpo_score_sequences for groups that share a prefix: rows g*G .. g*G+G-1 of
 * tokens are the G samples of one prompt (Alg. 1) and hold the same tokens at
 * positions 0 .. prefix_len-1.  Under causal attention those positions' states
 * are the same for all G rows, so the forward runs them once per group (their
 * K/V shared by the group) and runs each row only from the multiple of 32 at or
 * below prefix_len-1 on.  The results are those of grpo_score_sequences except
 * for the order of floating-point additions; rows that do not share the prefix
 * are scored as if they did.  Arguments as grpo_score_sequences, plus
 *   G           group size, >= 1, dividing N
 *   prefix_len  shared positions, 0 <= prefix_len <= score_from
 * Same workspace as grpo_score_sequences.  fp32 models, G = 1 and short prefixes
 * (below 33 positions) take the per-row path.  GRPO_INVALID_ARG for a G or
 * prefix_len outside these ranges. */
int grpo_score_sequences_grouped(const grpo_model* m, const int32_t* tokens, int32_t N,
                                 int32_t T, int32_t score_from, float temperature, int32_t G,
                                 int32_t prefix_len, float* logp_out, const grpo_trace* trace,
                                 void* ws, size_t ws_bytes, void* stream);

/* Group advantages (Alg. 1, normalisation step): for each of the P groups of
 * G >= 2 rewards, A = (r - mean) / (sample std (divisor G-1) + eps); a group
 * whose rewards are all equal gets A = 0.  rewards, adv_out fp32 [P*G]. */
int grpo_advantages(const float* rewards, int32_t P, int32_t G, float eps, float* adv_out,
                    void* stream);

/* GRPO token loss (Eq. 1 in the clipped form of Sec. VI-A):
 *   rho = exp(logp - logp_old); s = min(rho*A, clip(rho, 1-clip_eps, 1+clip_eps)*A)
 *   kl  = exp(d) - d - 1, d = logp_ref - logp;  l = -s + beta*kl
 * agg 0: mean of each sequence's masked tokens, then mean over sequences;
 * agg 1: mean over all masked tokens.
 *   logp, logp_old, logp_ref fp32 [N, Tr]; mask uint8 [N, Tr] (1 = trained);
 *   adv fp32 [N]
 *   loss_out    fp32 [1]
 *   tok_loss    NULL or fp32 [N, Tr]: l where mask, else 0
 *   dloss_dlogp NULL or fp32 [N, Tr]: d loss / d logp (0 where not mask)
 *   stats       NULL or fp32 [4]: masked-token mean kl, fraction of tokens the
 *               clip zeroes, mean ratio, count of non-finite l
 * Arithmetic is fp64 inside; outputs fp32. */
int grpo_token_loss(const float* logp, const float* logp_old, const float* logp_ref,
                    const uint8_t* mask, const float* adv, int32_t N, int32_t Tr, float clip_eps,
                    float beta, int32_t agg, float* loss_out, float* tok_loss, float* dloss_dlogp,
                    float* stats, void* ws, size_t ws_bytes, void* stream);

/* Reward of one completion (Sec. VI-A, Eq. 2-4), on the host:
 *   r = r_perf + r_tools
 *   r_perf  = -2 if the final code is incorrect; -1 if correct but slower than
 *             the baseline (t > t_base); else min(10, t_base / t - 1)
 *   r_tools = 0.5 * tools_used / tools_avail (unique available tools used)
 * so r lies in [-2, 10.5].  All arguments are HOST arrays of n entries;
 * correct is 0/1, times in any common unit.  GRPO_INVALID_ARG for
 * non-positive or infinite times or tools_used outside [0, tools_avail]
 * (checked for every entry before any output is written). */
int grpo_reward(const uint8_t* correct, const double* t_base, const double* t,
                const int32_t* tools_used, const int32_t* tools_avail, int32_t n, float* r_out);

/* Distillation loss (Sec. VI-B: supervised fine-tuning of the small model on
 * the large model's reasoning traces, tool-call tokens and arguments kept in
 * the targets): the teacher-forced cross-entropy over the target tokens,
 *   agg 1: -sum(mask * logp) / max(1, sum(mask))   (token mean)
 *   agg 0: mean over sequences of each one's token mean (0 without targets)
 * logp fp32 [N, Tr] (as grpo_score_sequences returns it), mask uint8 [N, Tr];
 * loss_out fp32 [1]; dloss_dlogp NULL or fp32 [N, Tr].  fp64 inside.  The
 * workspace is grpo_workspace_bytes(GRPO_OP_LOSS, N, Tr). */
int grpo_sft_loss(const float* logp, const uint8_t* mask, int32_t N, int32_t Tr, int32_t agg,
                  float* loss_out, float* dloss_dlogp, void* ws, size_t ws_bytes, void* stream);

/* fp32 gradient accumulators, one per weight of grpo_weights with the same
 * shape (row-major).  The backward ADDS into them; the caller zeroes them at
 * the start of an accumulation. */
typedef struct grpo_grads {
  float* tok_emb;
  float* const* attn_norm; float* const* wq; float* const* wk; float* const* wv;
  float* const* wo; float* const* mlp_norm; float* const* w_gate; float* const* w_up;
  float* const* w_down;
  float* final_norm;
  float* lm_head;
} grpo_grads;

/* Gradient step of Alg. 1, first half: the weight gradient of the GRPO
 * objective (Eq. 1, clipped form of Sec. VI-A).  The objective reaches the
 * weights only through the scored log-probs, so given g = dL/dlogp (the
 * dloss_dlogp output of grpo_token_loss, fp32 [N, T - score_from] device) this
 * accumulates into `grads` the gradient of sum_{n,j} g[n, j] logp[n, j], with
 * logp as grpo_score_sequences defines it (tokens int32 [N, T] device, the
 * same score_from and temperature):
 *   dz_t = g_t / T (onehot(x_{t+1}) - softmax(z_t / T)) on each scored row,
 * then back through the LM head, the final RMSNorm, every layer in reverse and
 * the embedding gather.  Each sequence's forward is recomputed (its layer
 * inputs kept), the rounding points of the bf16 forward pass gradients
 * straight through.  Gradients accumulate in fp32; data-gradient operands are
 * the model dtype (bf16 products on the matrix cores).  Every sum has a fixed
 * order, the embedding rows' included (positions grouped by token, then added
 * in position order): results are bit-deterministic.
 * Where a layer's wq, wk and wv gradients are adjacent in memory (wk right
 * after wq, wv right after wk), and likewise its w_gate and w_up gradients,
 * each group's weight gradient is one product (the same sums, so the same
 * bits); otherwise one product per tensor.
 * Workspace: grpo_workspace_bytes(GRPO_OP_BACKWARD, N, T) (it holds transposed
 * copies of every weight matrix).  GRPO_INVALID_ARG for a NULL gradient buffer
 * or score_from outside [1, T); GRPO_UNSUPPORTED for T above 16384. */
int grpo_policy_backward(const grpo_model* m, const int32_t* tokens, int32_t N, int32_t T,
                         int32_t score_from, float temperature, const float* dlogp,
                         const grpo_grads* grads, void* ws, size_t ws_bytes, void* stream);

/* AdamW hyper-parameters (decoupled weight decay). */
typedef struct grpo_adamw {
  float lr, beta1, beta2, eps, weight_decay;
} grpo_adamw;

/* Gradient step of Alg. 1, second half (the paper names no optimizer; AdamW
 * with bias correction): over n elements of one parameter tensor,
 *   m = b1 m + (1 - b1) g,  v = b2 v + (1 - b2) g^2,
 *   p = p - lr wd p - lr (m / (1 - b1^step)) / (sqrt(v / (1 - b2^step)) + eps)
 * step counts from 1.  dtype GRPO_F32: param is the fp32 tensor itself and
 * master may be NULL; GRPO_BF16: master (fp32) is updated and param receives
 * its bf16 rounding.  m, v, grad fp32 device arrays of n entries. */
int grpo_adamw_step(int32_t dtype, void* param, float* master, float* m, float* v,
                    const float* grad, size_t n, const grpo_adamw* hp, int32_t step,
                    void* stream);

/* Exact full-vocabulary KL of the policy to the frozen reference (Alg. 1, KL
 * step; the GRPO loss uses its per-token estimator): for each of R rows,
 * kl_out[r] = sum_v p(v) (log p(v) - log p_ref(v)), p = softmax(logits[r] / T),
 * p_ref = softmax(logits_ref[r] / T) (temperature 0 read as 1).  logits,
 * logits_ref fp32 [R, ld] device rows of V entries; kl_out fp32 [R].  fp64
 * inside. */
int grpo_exact_kl(const float* logits, const float* logits_ref, int32_t R, int32_t V, int32_t ld,
                  float temperature, float* kl_out, void* stream);

/* grpo_token_loss for callers that cannot allocate device memory (code under
 * HIP graph capture, serving loops, harnesses that forbid hipMalloc): the same
 * kernels and results, with the per-sequence scratch in a static device array
 * of the library (one per GPU, GRPO_LOSS_STATIC_ROWS sequences x 72 bytes =
 * 1.2 MB, held until the process ends) instead of a workspace argument.  The
 * call allocates nothing.  All calls on one GPU share that array: calls that
 * overlap on one GPU (different streams or threads without ordering) race and
 * must be serialised by the caller.  Arguments and outputs as grpo_token_loss;
 * GRPO_INVALID_ARG for N above GRPO_LOSS_STATIC_ROWS. */
#define GRPO_LOSS_STATIC_ROWS 16384
int grpo_token_loss_noalloc(const float* logp, const float* logp_old, const float* logp_ref,
                            const uint8_t* mask, const float* adv, int32_t N, int32_t Tr,
                            float clip_eps, float beta, int32_t agg, float* loss_out,
                            float* tok_loss, float* dloss_dlogp, float* stats, void* stream);

/* Reduction structure of a decode step, for error analysis of its results
 * (the order in which partial sums meet decides the rounding).  For a model, a
 * batch of B rows, a KV capacity max_len and a grouping (G, prefix_len as
 * grpo_rollout_step_grouped; G = 0 for grpo_rollout_step) it writes
 *   out[0..3] split-K factors of the QKV, O, down and LM-head projections
 *   out[4]    planned positions per decode-attention span; out[5] spans (a
 *             row's positions past its shared length are cut evenly into
 *             out[5] spans of whole 128-position units, at least one unit;
 *             the last span runs to the row's end)
 *   out[6]    positions per prompt chunk of a grouped step; out[7] chunks
 *             (both 0 without grouping or for fp32 models)
 *   out[8]    waves per workgroup of the per-row decode attention (4 or 2:
 *             a span's 32-position tiles are dealt round-robin to them)
 * out holds 9 entries.  fp32 models: out[0..8] = 0 (one fma chain per output).
 * GRPO_INVALID_ARG for a NULL pointer or sizes outside the call's ranges. */
int grpo_decode_structure(const grpo_model* m, int32_t B, int32_t max_len, int32_t G,
                          int32_t prefix_len, int32_t* out);

/* Kernel timing for benchmarks.  Between grpo_profile_begin and
 * grpo_profile_end every kernel launch of the library is bracketed by HIP
 * events on its stream (decode steps run without graph replay meanwhile).
 * GRPO_UNSUPPORTED while rocprofv3 collects hardware counters in the process
 * (ROCPROF_COUNTER_COLLECTION set), which also turns decode graph replay off.
 * grpo_profile_end synchronises those events and writes NUL-terminated JSON
 * {"kernel": [launches, total_ms], ...} into json (len bytes); it returns
 * GRPO_INVALID_ARG if the text does not fit.  Process-wide; not for use while
 * other threads launch library work. */
int grpo_profile_begin(void);
int grpo_profile_end(char* json, size_t len);

#ifdef __cplusplus
}
#endif
#endif /* GRPO_HIP_H */
