/*
 * tandem.h — C ABI of the MI355X tandem co-generation library (libtandem.so).
 *
 * What it computes (Tandem RL with Verifiable Rewards):
 *   Section 3.3 and Algorithm 1 (rollout half): a trained senior and a frozen
 *   junior causal LM with one shared vocabulary co-generate each response.
 *   At every step BOTH models forward the shared history x . y_<t, the
 *   current owner a_t samples y_t from its own next-token distribution, the
 *   token is appended to both models' KV caches, and ownership is redrawn
 *   with a Bernoulli(p) coin after boundary tokens or once the span counter
 *   reaches the cap K.  Each step records y_t, the authorship bit
 *   m_t = 1[a_t = senior] and log pi_sen(y_t | x . y_<t), the quantity the
 *   senior-only GRPO loss of Section 3.4 (the L_TRL equation) consumes.
 *   The reproducibility appendix describes the same step inside a serving
 *   engine: shared per-step position metadata, one KV cache per model,
 *   a per-request seeded generator and a small per-request sampler state.
 *
 * Memory ownership: the CALLER owns every device buffer (weights, KV arena,
 * scratch, output arenas, boundary bitmap, prompts, forced tokens, debug
 * buffers).  The library borrows the pointers until tandem_destroy and owns
 * only host-side state.  Sizes of the KV arena and the scratch buffer come
 * from tandem_workspace_size.
 *
 * Streams: every call enqueues its work on the stream given to tandem_init
 * (a hipStream_t passed as void*) and returns without synchronising, except
 * where a call below says otherwise: a host result is requested (n_active,
 * tandem_get_state, tandem_timing_read), a batch with an EOS token compacts
 * its rows (once every 32 steps), tandem_timing_enable and tandem_destroy.
 *
 * Errors: every call returns a tandem_status; tandem_last_error(handle) (or
 * tandem_last_error(NULL) for calls that failed before a handle existed)
 * gives a message.  Arguments are validated before any HIP call.  A failing
 * HIP call returns TANDEM_E_HIP and poisons the handle: later calls return
 * TANDEM_E_STATE.  One handle must not be used from two threads at once.
 */
#ifndef TANDEM_H
#define TANDEM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  TANDEM_OK = 0,
  TANDEM_E_ARG = -1,          /* NULL pointer, bad enum, p outside [0,1], T <= 0, ... */
  TANDEM_E_SHAPE = -2,        /* inconsistent model shapes (vocab mismatch, n_q % n_kv, ...) */
  TANDEM_E_CAPACITY = -3,     /* request exceeds the capacity given at init / buffer too small */
  TANDEM_E_STATE = -4,        /* call out of order (step before prefill) or poisoned handle */
  TANDEM_E_HIP = -5,          /* a HIP runtime call failed */
  TANDEM_E_UNSUPPORTED = -6   /* a shape the library has no kernel for (head_dim, ...) */
} tandem_status;

/* first owner a_1 (Algorithm 1 draws it with the same Bernoulli(p) coin) */
enum { TANDEM_JUNIOR = 0, TANDEM_SENIOR = 1, TANDEM_DRAW = 2 };

/* What happens at a decision point (boundary token or span cap reached):
 *   REDRAW    next owner = senior with probability p (the paper's rule);
 *   SWITCH    owner flips with probability p ("per-token switch probability");
 *   ALTERNATE owner always flips (the deterministic reasoning-step schedule). */
enum { TANDEM_REDRAW = 0, TANDEM_SWITCH = 1, TANDEM_ALTERNATE = 2 };

/* element type of the weights and of the KV cache.  The residual stream is
 * fp32; inputs of the bf16 projections are carried as bf16 hi + lo pairs. */
enum { TANDEM_BF16 = 0, TANDEM_F32 = 1 };

/* Shape of one pre-norm decoder: RMSNorm, grouped-query attention with
 * NeoX-style rotary embedding (optional per-head q/k RMSNorm), SwiGLU FFN,
 * final RMSNorm and an untied LM head. */
typedef struct {
  int32_t n_layers, d_model, n_q_heads, n_kv_heads, head_dim, ffn_dim, vocab;
  float rope_theta;           /* rotary base theta */
  float rms_eps;              /* RMSNorm epsilon */
  int32_t qk_norm;            /* 1: per-head RMSNorm of q and k before RoPE */
  int32_t weight_dtype;       /* TANDEM_BF16 or TANDEM_F32 */
} tandem_model_cfg;

/* Device pointers to one model's weights.  Matrices are row-major
 * [out][in] in weight_dtype; norm gains are float32.
 *   embed      [vocab][d_model]
 *   layers     HOST array of n_layers * 8 device pointers, per layer in order:
 *              attn_norm [d], w_qkv [(n_q + 2 n_kv) * hd][d] (rows: q heads,
 *              then k heads, then v heads), q_norm [hd], k_norm [hd] (both
 *              NULL unless qk_norm), w_o [d][n_q * hd], ffn_norm [d],
 *              w_gate_up [2 ffn][d] (gate rows, then up rows), w_down [d][ffn]
 *   final_norm [d_model]
 *   lm_head    [vocab][d_model]
 * Every weight pointer must be 16-byte aligned; d_model and ffn_dim must be
 * multiples of 8.  The layers array is copied at tandem_init; the weights are
 * borrowed. */
typedef struct {
  tandem_model_cfg cfg;
  const void* embed;
  const void* const* layers;
  const void* final_norm;
  const void* lm_head;
} tandem_model;

/* Handoff rule (Algorithm 1's boundary-or-cap block). */
typedef struct {
  int32_t mode;                    /* TANDEM_REDRAW / TANDEM_SWITCH / TANDEM_ALTERNATE */
  double p;                        /* coin probability, 0 <= p <= 1 */
  int32_t cap_k;                   /* span cap K; < 0 disables the cap */
  const uint32_t* boundary_bits;   /* device bitmap, bit (v & 31) of word v >> 5 marks a
                                      boundary token; NULL = every token is a boundary */
  int32_t first_owner;             /* TANDEM_JUNIOR / TANDEM_SENIOR / TANDEM_DRAW */
} tandem_switch_cfg;

/* Sampling: scores s_m = (z_m + b_m * e_eos) / T; the owner's scores are
 * sampled by Gumbel-max with Philox4x32-10 noise keyed by (seed, sequence id,
 * step, vocab index); the handoff coin uses a separate Philox stream. */
typedef struct {
  float temperature;               /* T > 0 */
  int32_t eos_id;                  /* < 0: no end-of-sequence token */
  float eos_bias_senior;           /* logit bias added to eos_id (senior) */
  float eos_bias_junior;           /* logit bias added to eos_id (junior) */
  int32_t max_new_tokens;          /* L: tokens generated per sequence at most */
  uint64_t seed;                   /* request seed: Philox key (low word, high word) */
} tandem_sample_cfg;

typedef struct {
  int32_t max_seqs;                /* >= n_prompts * G */
  int32_t max_ctx;                 /* >= longest prompt - 1 + max_new_tokens */
  int32_t max_prefill_tokens;      /* rows of one prefill pass (prompts are chunked to fit) */
} tandem_capacity;

/* Caller-owned device output arenas, sequence-major [max_seqs][max_new_tokens].
 * Entry [s][t-1] is written at step t of sequence s (s = j * G + i). */
typedef struct {
  int32_t* tokens;                 /* y_t */
  uint8_t* owner;                  /* m_t = 1 if the senior emitted y_t */
  float* senior_logprob;           /* log softmax(s_sen)[y_t], every position */
  int32_t* length;                 /* [max_seqs] tokens recorded so far */
} tandem_outputs;

/* Optional device buffers filled by tandem_step_forced (any may be NULL). */
typedef struct {
  int32_t* sampled;                /* [max_seqs] the library's own sample of this step */
  float* margin;                   /* [max_seqs] best - second Gumbel score of the owner */
  float* logits_senior;            /* [max_seqs][vocab] raw senior logits z_sen */
  float* logits_junior;            /* [max_seqs][vocab] raw junior logits z_jun */
} tandem_debug;

typedef struct tandem_handle tandem_handle;

/* Bytes of KV arena and scratch that tandem_init needs for these shapes and
 * this capacity (junior NULL: the senior alone).  Both buffers must be
 * 256-byte aligned device memory. */
tandem_status tandem_workspace_size(const tandem_model_cfg* senior, const tandem_model_cfg* junior,
                                    const tandem_capacity* cap, size_t* kv_bytes,
                                    size_t* scratch_bytes);

/* Algorithm 1's inputs: the senior and the junior policies (one shared
 * vocabulary), the handoff probability p, the boundary set and the span cap K
 * (the reproducibility appendix's word-level handoff details), plus the
 * sampling settings and the per-request seed of the appendix's seeded
 * generator.  Validates the pair (shared vocabulary, supported head_dim, ...),
 * binds the weights, arenas and stream, and enqueues the per-model tables
 * (rotary table, MFMA-ordered weight copies in scratch) on the stream; it
 * does not wait for them (later calls on the same stream are ordered after
 * them).  stream is a hipStream_t (NULL = the null stream).  On success
 * *out_handle is set; on failure nothing is left allocated.
 * junior NULL: a single-model rollout of the senior through the same
 * kernels, the baseline the paper compares the tandem rollout with (plain
 * GRPO sampling, one model): the senior emits every token (m_t = 1), sw is
 * ignored (may be NULL), the junior's debug logits are not written, and
 * tandem_score_step returns TANDEM_E_STATE. */
tandem_status tandem_init(const tandem_model* senior, const tandem_model* junior,
                          const tandem_switch_cfg* sw, const tandem_sample_cfg* smp,
                          const tandem_capacity* cap, void* kv_arena, size_t kv_bytes,
                          void* scratch, size_t scratch_bytes, const tandem_outputs* out,
                          void* stream, tandem_handle** out_handle);

/* Section 3.3: both models condition on the prompt x before the first token
 * (the dual-decoder backend of the reproducibility appendix keeps one cache
 * per model on shared positions).  Prefills both models on every prompt but
 * its last token, shares the prompt's K/V among its G sequences, and sets each
 * sequence's state: pending token = last prompt token, position = P_j - 1,
 * step t = 1, span counter 0, first owner per first_owner (DRAW: Algorithm 1's
 * Bernoulli(p) first draw).
 *   prompt_tokens  device int32, prompts concatenated (read on the stream)
 *   prompt_offsets HOST int32 [n_prompts + 1], CSR offsets into prompt_tokens
 * Every prompt needs >= 1 token.  Sequence ids are s = j * G + i.  A new
 * prefill starts a new batch (all previous sequence state is replaced).
 * Asynchronous: the per-prompt table is uploaded from pinned staging and the
 * prefill rows are built on the device.  The call waits only if the previous
 * prefill's table upload is still queued on the stream.  Token ids are
 * checked on the device: an id outside [0, vocab) is read as 0 and makes the
 * next synchronising call (tandem_step with n_active, a compaction step,
 * tandem_get_state) return TANDEM_E_ARG; the batch is then void and steps
 * return TANDEM_E_STATE until the next prefill. */
tandem_status tandem_prefill(tandem_handle* h, const int32_t* prompt_tokens,
                             const int32_t* prompt_offsets, int32_t n_prompts, int32_t G);

/* One pass of Algorithm 1's rollout loop for every unfinished sequence:
 * forward the pending token through both models (appending to both caches,
 * Section 3.3), sample y_t from the owner a_t, write (y_t, m_t, senior
 * log-prob log pi_sen(y_t | .) for Section 3.4's L_TRL) to the output arenas,
 * stop at EOS or at t = max_new_tokens, apply the handoff block.  If
 * n_active is not NULL the call synchronises and stores the number of
 * unfinished sequences.  With an EOS token, every 32nd step first compacts
 * the batch (unfinished sequences to the front): that step synchronises once
 * to read the unfinished count.
 * The step's kernels are captured once per batch into a HIP graph (on the
 * first tandem_step after tandem_prefill, or after a timing-mode change)
 * and every step replays it on the handle's stream: the per-step state lives
 * in device memory, so the same graph serves every step.  Capture allocates
 * host-side graph objects owned by the handle.
 * Where both LM heads run on the streaming decode GEMM (bf16 weights whose
 * packed copy fits, vocab % 4 == 0) and at most 128 rows are launched, the
 * sampling runs inside the LM-head GEMMs: the step's Gumbel noise is
 * generated beside the forwards, each head folds its scores into per-row
 * partials (the senior's log-sum-exp, the owner's top two), and no logits
 * are stored. */
tandem_status tandem_step(tandem_handle* h, int32_t* n_active);

/* As tandem_step (the same pass of Algorithm 1's loop, launched kernel by
 * kernel), but the appended token of sequence s is forced[s] (device int32
 * [max_seqs]; entries < 0 keep the library's own sample): teacher forcing.
 * The owner rule and the outputs follow the appended token; dbg (may be
 * NULL) receives the library's own sample, its margin and the raw logits of
 * this step. */
tandem_status tandem_step_forced(tandem_handle* h, const int32_t* forced, const tandem_debug* dbg,
                                 int32_t* n_active);

/* Dual-distribution scores of the step just taken (teacher-forced or free):
 * the junior legibility and distribution overlap measures of the paper's
 * evaluation (junior per-token cross-entropy; overlap alpha = sum_v
 * min(p_sen(v), p_jun(v))) and the per-position divergence of the senior from
 * the junior that its KL-regularisation ablation penalises.  Both models'
 * next-token distributions are taken at temperature 1 with no EOS bias.  For
 * every sequence s that was not done before the step, scores[3 s .. 3 s + 2]
 * (device float [max_seqs][3], caller-owned) receive (-log p_jun(y), alpha,
 * KL(p_sen || p_jun)), y being the token the step appended to s; entries of
 * other sequences are left untouched.  Asynchronous on the handle's stream.
 * A step that sampled inside the LM heads stored no logits: both LM heads
 * then run again here, on the step's LM-head input rows.
 * TANDEM_E_STATE when no step has been taken since the last prefill;
 * TANDEM_E_ARG when scores is NULL. */
tandem_status tandem_score_step(tandem_handle* h, float* scores);

/* Senior-only GRPO loss pieces of a batch of tandem rollouts (Section 3.4, the
 * L_TRL equation; Algorithm 1's update half; the hyperparameter table's
 * group-relative, std-normalised advantage and clip ratio).  Handle-free:
 * it reads the rollout arenas tandem_step wrote (or any arrays of that
 * layout) and runs on the given stream (hipStream_t as void*, NULL = the null
 * stream), asynchronously.  S = n_groups * group_size rollouts, s = j * G + i.
 *   advantage  A_s = (r_s - mean_j) / (std_j + 1e-6), std_j the sample
 *              standard deviation (divisor G - 1; 0 when G = 1) of group j's
 *              rewards; every position of rollout s shares A_s.
 *   mask       position t of rollout s is counted iff t < length[s] and
 *              owner[s][t] != 0 (the senior emitted it); N = masked count.
 *   loss       L = -(1/N) sum_masked min(rho A_s, clip(rho, 1 - eps, 1 + eps) A_s),
 *              rho = exp(logp_new - logp_old); L = 0 when N = 0.
 *   gradient   dL/dlogp_new[s][t] = -rho A_s / N where the unclipped term is
 *              the minimum, 0 elsewhere (every unmasked position included).
 * All pointers are caller-owned device memory:
 *   rewards    float [S]; owner uint8 [S][T]; length int32 [S] (clamped to
 *              [0, T]); logp_old float [S][T] (the rollout's senior log-probs,
 *              pi_old); logp_new float [S][T] or NULL (= logp_old: rho = 1)
 *   advantages float [S] out; grad float [S][T] out or NULL; loss float [1]
 *              out; n_masked int32 [1] out
 *   workspace  >= tandem_grpo_workspace_size bytes, 256-byte aligned; its
 *              contents need no initialisation and are overwritten; calls
 *              that may overlap (other streams) must not share one.
 * T is the arenas' row stride (max_new_tokens).  TANDEM_E_ARG for a NULL
 * required pointer, eps outside [0, 1) or a short workspace; TANDEM_E_SHAPE
 * for sizes < 1 or S * T >= 2^24 (masked counts are summed exactly in fp32).
 * Errors are reported through tandem_last_error(NULL). */
typedef struct {
  int32_t n_groups;                /* prompts j */
  int32_t group_size;              /* G >= 1 */
  int32_t max_new_tokens;          /* T, row stride of the [S][T] arrays */
  float clip_eps;                  /* PPO clip ratio eps (0.2 in the paper) */
} tandem_grpo_cfg;

tandem_status tandem_grpo_workspace_size(const tandem_grpo_cfg* cfg, size_t* bytes);
tandem_status tandem_grpo_loss(const tandem_grpo_cfg* cfg, const float* rewards, const uint8_t* owner,
                               const int32_t* length, const float* logp_old, const float* logp_new,
                               float* advantages, float* grad, float* loss, int32_t* n_masked,
                               void* workspace, size_t workspace_bytes, void* stream);

/* tandem_grpo_loss without the workspace argument, for callers that cannot
 * allocate device memory: code under HIP graph capture, serving loops and
 * harnesses that forbid hipMalloc.  The workspace is a device array of the
 * library's own, 1 MiB per GPU, held from the first call on that GPU until
 * the process ends; the call allocates nothing (no hipMalloc, hipFree or
 * allocating library routine).  Batches whose tandem_grpo_workspace_size
 * exceeds 1 MiB (S * ceil(T / 1024) partial sums plus S counts, each
 * 256-byte aligned, plus 256 bytes) return TANDEM_E_CAPACITY.  Every call on
 * one GPU shares that GPU's array (the kernels overwrite or clear everything
 * they read), so calls that may overlap on one GPU (other streams, other
 * threads) race and must not be issued.  Arguments, results and the other
 * errors are those of tandem_grpo_loss. */
tandem_status tandem_grpo_loss_noalloc(const tandem_grpo_cfg* cfg, const float* rewards, const uint8_t* owner,
                                       const int32_t* length, const float* logp_old, const float* logp_new,
                                       float* advantages, float* grad, float* loss, int32_t* n_masked,
                                       void* stream);

/* The per-request sampler state of the reproducibility appendix (current
 * owner, span counter, step, position, finished), copied to HOST int32
 * arrays of n_seqs entries (any pointer may be NULL): owner (1 = senior),
 * span counter c, next step t, next position, done flag.  Synchronises the
 * stream; reports a token-range error of the batch's prompts (see
 * tandem_prefill). */
tandem_status tandem_get_state(tandem_handle* h, int32_t* owner, int32_t* c, int32_t* t,
                               int32_t* pos, int32_t* done);

/* Instrumentation (the benchmark's roofline and the per-kernel breakdown).
 * class_mask bit k enables class k: the library then records a hipEvent pair
 * around every launch of that class on the stream it runs on (the junior's
 * forward runs on a second stream joined back into the caller's, so its
 * launches may overlap the senior's); tandem_timing_read
 * synchronises and returns the summed device milliseconds and the number of
 * launches of one class since the last tandem_timing_enable.  Every call to
 * tandem_timing_enable waits for the stream's queued work and resets the sums
 * (mask 0 switches timing off).  Each
 * event pair adds a few microseconds of stream time.  While any class is
 * timed, tandem_step launches its kernels from the host instead of replaying
 * the step graph (event records inside a graph carry no launch times). */
enum { TANDEM_K_ATTENTION = 0,    /* decode / prompt attention            */
       TANDEM_K_GEMM = 1,         /* projection and LM-head GEMMs         */
       TANDEM_K_SAMPLE = 2,       /* sampling, log-prob, handoff rule     */
       TANDEM_K_OTHER = 3,        /* norms, QKV post-processing, copies   */
       TANDEM_K_CLASSES = 4 };
/* Flags for class_mask (they also apply with no class bit set):
 *   TANDEM_TIMING_SERIAL  the senior's and the junior's forwards run one after
 *                         the other instead of overlapping on two streams, so
 *                         each timed launch has the GPU to itself;
 *   TANDEM_TIMING_EAGER   tandem_step launches every kernel from the host
 *                         instead of replaying its captured HIP graph.
 * Results are unchanged; only the schedule differs.
 *   TANDEM_TIMING_SEPARATE_SAMPLE  the step stores both models' logits and
 *                         samples in a pass over them, instead of sampling
 *                         inside the LM-head GEMMs (the default where both LM
 *                         heads run as fp16 streaming GEMMs over at most 128
 *                         rows); the two agree up to float rounding (the
 *                         log-sum-exp is accumulated in another order, the
 *                         appended token's senior score is a separate dot
 *                         product), so a Gumbel tie inside that rounding may
 *                         sample differently. */
enum { TANDEM_TIMING_SERIAL = 1 << 8, TANDEM_TIMING_EAGER = 1 << 9, TANDEM_TIMING_SEPARATE_SAMPLE = 1 << 10 };
tandem_status tandem_timing_enable(tandem_handle* h, int32_t class_mask);
tandem_status tandem_timing_read(tandem_handle* h, int32_t kernel_class, double* total_ms, int64_t* launches);

/* Message of the last failure on this handle (or of this thread's last
 * handle-less failure when h is NULL).  Never NULL. */
const char* tandem_last_error(const tandem_handle* h);

/* Human-readable name of a status code. */
const char* tandem_status_string(tandem_status s);

/* Release host-side state; device buffers stay with the caller.  NULL is a no-op. */
void tandem_destroy(tandem_handle* h);

#ifdef __cplusplus
}
#endif

#endif /* TANDEM_H */
