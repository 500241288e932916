/*
 * rollout.h -- C ABI of librollout.so, the MI355X (gfx950) group-rollout library.
 *
 * What it computes.  Synchronous GRPO/DAPO training samples, for every prompt,
 * a group of G completions, scores them and forms group-relative advantages
 * (paper Sec. 3.1, problem statement; Sec. 4, requirements (i)-(iii)).  The
 * batched generation of such groups is gated by the longest completion of each
 * group (Sec. 3.1, Eq. ratio) and is the part of the training step this
 * library runs on the GPU:
 *
 *   rollout_group    -- prefill every prompt once, fork its G siblings over a
 *                       shared prompt prefix in a paged KV cache, then decode
 *                       all siblings together, sampling each token by
 *                       Gumbel-max from a Philox4x64-10 stream and retiring
 *                       every sequence at its EOS.
 *   group_advantage  -- A_i = (r_i - mean_g r) / (std_g r + eps) per group.
 *   group_filter     -- which groups carry a learning signal (rewards not all
 *                       equal), for DAPO-style dynamic sampling.
 *   recompute_logprobs, grpo_surrogate -- the loss forward that follows:
 *                       teacher-forced log-probabilities of the rollout under
 *                       the policy and the clipped surrogate built on them.
 *
 * Conventions for every entry point.
 *   - Status: 0 on success, a negative RG_E* code on error; rg_last_error()
 *     then returns a message (thread-local, valid until the next call made
 *     by the same thread).  No exception crosses the ABI.  Outputs are
 *     undefined after an error.
 *   - "device" pointers are HIP device memory of the current device; "host"
 *     pointers are ordinary CPU memory read before the call returns.
 *   - `stream` is a hipStream_t passed as void*.  NULL is the null stream.
 *   - Integer ids and sizes are int32 unless stated; tensors are dense,
 *     row-major, with the shapes given in brackets.
 */
#ifndef PAPER_2606_02218_ROLLOUT_H
#define PAPER_2606_02218_ROLLOUT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ---- */
#define RG_OK            0
#define RG_EINVAL       (-1)  /* an argument is out of range or inconsistent            */
#define RG_ENOMEM       (-2)  /* a size exceeds the policy's limits or its KV page pool  */
#define RG_EHIP         (-3)  /* a HIP runtime call failed                             */
#define RG_EUNSUPPORTED (-4)  /* a model shape the kernels do not handle              */

/* ---- element types ---- */
#define RG_DTYPE_F32  0
#define RG_DTYPE_BF16 1

/* Decoder shape.  Pre-norm blocks x += Attn(RMSNorm(x)), x += MLP(RMSNorm(x)),
 * final RMSNorm, untied lm_head, no biases.  RMSNorm(x) = x/sqrt(mean(x^2)+eps)*g.
 * RoPE rotates dims (i, i+head_dim/2) by pos*rope_theta^(-2i/head_dim); prompt
 * tokens are at positions 0..Lp-1, generated token t at Lp+t.  Query head h
 * reads key/value head floor(h*n_kv_heads/n_q_heads).  MLP =
 * W_down(silu(W_gate x) * (W_up x)).
 * Supported: head_dim 32, 64 or 128 (bf16 models: 64 or 128), n_q_heads a
 * multiple of n_kv_heads with at most 8 query heads per kv head, d_model,
 * n_q_heads*head_dim and ffn_dim multiples of 64, vocab a multiple of 16
 * (otherwise RG_EUNSUPPORTED). */
typedef struct rg_config {
  int32_t n_layers, d_model, n_q_heads, n_kv_heads, head_dim, ffn_dim, vocab;
  int32_t eos_id;       /* token that ends a completion, in [0, vocab)                   */
  float rope_theta;
  float rms_eps;
  int32_t dtype;        /* RG_DTYPE_F32: fp32 matrices and KV cache.  RG_DTYPE_BF16: bf16
                           matrices and KV cache (keys rounded to nearest-even bf16 after
                           RoPE, values after projection); every other value is fp32.
                           bf16 MFMA takes each fp32 activation as a hi + lo pair of bf16
                           values (about 17 significant bits), so products keep the
                           activation's fp32 precision.                                  */
} rg_config;

/* Weights, all DEVICE pointers, read during rg_policy_create only (the policy
 * keeps its own repacked copy; the caller may free these afterwards).
 * Matrices are [out, in] row-major (y = x W^T) in the config dtype; norm gains
 * are always fp32.  The per-layer members are HOST arrays of n_layers device
 * pointers. */
typedef struct rg_weights {
  const void* embed;               /* [vocab, d_model]                  */
  const void* final_norm;          /* [d_model] fp32                    */
  const void* lm_head;             /* [vocab, d_model]                  */
  const void* const* attn_norm;    /* [d_model] fp32                    */
  const void* const* wq;           /* [n_q_heads*head_dim, d_model]     */
  const void* const* wk;           /* [n_kv_heads*head_dim, d_model]    */
  const void* const* wv;           /* [n_kv_heads*head_dim, d_model]    */
  const void* const* wo;           /* [d_model, n_q_heads*head_dim]     */
  const void* const* ffn_norm;     /* [d_model] fp32                    */
  const void* const* w_gate;       /* [ffn_dim, d_model]                */
  const void* const* w_up;         /* [ffn_dim, d_model]                */
  const void* const* w_down;       /* [d_model, ffn_dim]                */
} rg_weights;

/* Capacity of a policy, fixed at creation: the device workspace (activations,
 * logits, attention partials) and the KV page pool are allocated once. */
typedef struct rg_limits {
  int32_t max_seqs;           /* largest N = sum(G) of one rollout                        */
  int32_t max_prompts;        /* largest P                                                */
  int32_t max_prompt_tokens;  /* largest sum of prompt lengths                            */
  int32_t max_context;        /* largest prompt length + max_new                          */
  int64_t kv_pool_pages;      /* KV pages in the pool; 0 = enough for the worst case of
                                 the other limits (every sequence reaching max_context)   */
} rg_limits;

typedef struct rg_policy rg_policy;  /* opaque: packed weights, KV pool, workspace */

/* Flags for rg_sampling.flags */
#define RG_FLAG_NO_PREFIX_SHARING 1  /* give every sibling private copies of its prompt's
                                        KV pages (results are bit-identical; a test aid) */
#define RG_FLAG_PROFILE           2  /* time kernel launches with HIP events (the classes in
                                        rg_sampling.profile_kinds, all when it is 0); read
                                        the totals with rg_kernel_times()                */
#define RG_FLAG_GROUP_PREFIX      4  /* bf16 models: decode steps attend to each prompt's
                                        full prefix pages once per group (one workgroup per
                                        prompt, kv head and prefix chunk scores every active
                                        sibling) instead of row by row.  Results agree up to
                                        the summation order of the softmax chunks.  Off by
                                        default: on MI355X the row-by-row pass reads the
                                        shared pages from L2 and is faster at G = 16.     */

#define RG_FLAG_NO_ROW_TILES      8  /* recompute_logprobs: attend row by row instead of by
                                        tiles of 32 positions (16 for wide GQA groups) of a
                                        sequence sharing each staged K/V block (a test and
                                        measurement aid)                                   */

/* Sampling options.  A NULL rg_sampling* means temperature 1, natural EOS, no
 * flags.  Token t of sequence s is argmax_v fp32(z_v/T) + g_v where g_v is the
 * fp32 Gumbel variate -log(-log(u)) of the stream documented at
 * rg_gumbel_bits() for (seed, t, s, v); ties go to the lowest id.  With
 * forced_len, EOS scores -inf while t < forced_len[s]-1 and token
 * forced_len[s]-1 is EOS (the synthetic stand-in for a policy's own stopping
 * time).  The reported log-probability is that of the emitted token under the
 * unmasked softmax(z/T). */
typedef struct rg_sampling {
  float temperature;            /* > 0                                                      */
  int32_t flags;                /* RG_FLAG_*                                                */
  const int32_t* forced_len;    /* HOST [N] in [1, max_new], or NULL for natural EOS       */
  const int32_t* force_tokens;  /* DEVICE [N*max_new] or NULL.  Teacher forcing: the token
                                   fed to step t+1 is force_tokens[s*max_new+t] (retirement
                                   follows it), `tokens` still receives the library's own
                                   sampling decision and `logprobs` the forced token's.    */
  float* dump_logits;           /* DEVICE [dump_steps*N*vocab] or NULL: raw logits z of
                                   sequence s at step t < dump_steps go to
                                   dump_logits[(t*N+s)*vocab ...]; untouched otherwise     */
  int32_t dump_steps;
  uint32_t profile_kinds;       /* with RG_FLAG_PROFILE: bit k times kernel class k
                                   (RG_K_*); 0 times every class                           */
} rg_sampling;

const char* rg_last_error(void);

/* Create a policy for one decoder.  Validates the shape, copies and repacks
 * the weights, allocates the workspace and KV pool for `limits` on the current
 * device.  *out receives the handle.  Errors: RG_EINVAL (NULL arguments,
 * non-positive sizes), RG_EUNSUPPORTED (shape), RG_ENOMEM / RG_EHIP
 * (allocation).  Read once here from the environment: RG_NO_GRAPHS=1 makes
 * rollout_group launch its decode steps directly instead of replaying
 * captured HIP graphs (the same kernels and arguments); RG_PROGRESS=N prints
 * a line to stderr every N decode steps of rollout_group. */
int rg_policy_create(const rg_config* cfg, const rg_weights* w, const rg_limits* limits,
                     rg_policy** out);
void rg_policy_destroy(rg_policy* pol);   /* NULL is a no-op */

/* Bytes of device memory the policy holds (weights + workspace + KV pool). */
int64_t rg_policy_device_bytes(const rg_policy* pol);

/* Generate G[p] completions for each prompt p (paper Sec. 3.1).
 *   prompts     DEVICE int32 [sum(prompt_len)], prompts packed back to back; ids in
 *               [0, vocab)
 *   prompt_len  HOST   int32 [P], each >= 1
 *   G           HOST   int32 [P], each >= 1; N = sum(G)
 *   max_new     >= 1; prompt_len[p] + max_new <= limits.max_context
 *   seed        Philox key word 0 of the sampling stream
 * Sequence s = off_p + j (off = exclusive prefix sum of G) is sibling j of
 * prompt p.  Outputs (caller-allocated DEVICE buffers):
 *   tokens    int32 [N*max_new]: tokens[s*max_new+t]; -1 after the completion
 *   lengths   int32 [N]: generated tokens including the final EOS (or max_new)
 *   logprobs  fp32  [N*max_new]: log-probability of each emitted token; 0 after
 * Work is enqueued on `stream`; the call returns once every sequence has
 * retired (it reads the active count back from the device), so the outputs
 * are complete when the stream's work is.  Not thread-safe per policy.
 * Errors: RG_EINVAL (arguments), RG_ENOMEM (N, P, prompt tokens or context
 * beyond the limits, or the KV page pool ran out during decoding), RG_EHIP. */
int rollout_group(rg_policy* pol, const int32_t* prompts, const int32_t* prompt_len, int32_t P,
                  const int32_t* G, int32_t max_new, uint64_t seed, const rg_sampling* opts,
                  int32_t* tokens, int32_t* lengths, float* logprobs, void* stream);

/* Group-relative advantage (paper Sec. 3.1: group-relative baseline from the
 * group's mean and standardized rewards).  For each group p of G[p] rewards:
 * mean and std (std with `ddof`, 0 or 1) in fp64, A = (r - mean)/(std + eps)
 * rounded to fp32; a group whose rewards are all equal, or with G[p] <= ddof,
 * gets A = 0.
 *   rewards  DEVICE fp32 [N], groups back to back (N = sum(G))
 *   G        DEVICE int32 [P], each >= 1 (read by the kernel)
 *   adv      DEVICE fp32 [N] (may not alias rewards)
 * Only enqueues work on `stream`; allocates nothing.  Errors: RG_EINVAL for
 * P < 1, N < 1, eps < 0 or ddof not in {0, 1}; a G[] entry < 1 or a sum that
 * differs from N makes the kernel write NaN to every adv[i].  */
int group_advantage(const float* rewards, const int32_t* G, int32_t P, int32_t N, float eps,
                    int32_t ddof, float* adv, void* stream);

/* Zero-variance group filter (DAPO-style dynamic sampling, which the paper
 * cites in Sec. 2 and uses in Sec. 5.1 without describing it): a group whose
 * rewards are all equal (exact fp32 equality) has A = 0 for every member
 * (see group_advantage) and gives no learning signal, so a trainer drops it
 * and samples further prompts in its place.
 *   rewards   DEVICE fp32 [N], groups back to back (N = sum(G))
 *   G         DEVICE int32 [P], each >= 1
 *   keep      DEVICE int32 [P]: 1 if group p's rewards vary, else 0
 *   kept_ids  DEVICE int32 [P]: ids of the kept groups, ascending, in the
 *             first n_kept entries
 *   n_kept    DEVICE int32 [1]: the number of kept groups; -1 if a G[]
 *             entry is < 1 or sum(G) != N (then nothing else is written)
 * Only enqueues work on `stream`; allocates nothing.  RG_EINVAL for NULL
 * pointers, P < 1 or N < 1. */
int group_filter(const float* rewards, const int32_t* G, int32_t P, int32_t N, int32_t* keep,
                 int32_t* kept_ids, int32_t* n_kept, void* stream);

/* Teacher-forced log-probabilities of finished completions under the policy
 * (the first half of the GRPO / DAPO loss forward, Sec. 2 and Sec. 5: the
 * trainer scores the rollout under the current weights before its update).
 * For every sequence s of prompt p and t < lengths[s]:
 *   logprobs[s*max_new + t] = z_{y_t}/T - logsumexp(z/T),
 * z the logits after the prompt and y_0 .. y_{t-1} = tokens[s*max_new ..].
 * The prompts are prefilled once, the siblings fork over their shared prompt
 * pages, and all completion positions then run as prefill-style rows (many
 * positions per sequence per launch) through the same decoder kernels as the
 * rollout, with the lm head in row slices and a fused logsumexp/gather.
 *   prompts, prompt_len, P, G, max_new   as for rollout_group
 *   tokens     DEVICE int32 [N*max_new], ids in [0, vocab) for t < lengths[s]
 *   lengths    DEVICE int32 [N], each in [1, max_new]
 *   temperature  > 0 (use the rollout's to reproduce its logprobs)
 *   flags      RG_FLAG_PROFILE, RG_FLAG_NO_PREFIX_SHARING as in
 *              rg_sampling.flags, RG_FLAG_NO_ROW_TILES; profiled kernel
 *              times land in phase 0
 *              (prompt prefill) and phase 1 (completion rows)
 *   logprobs   DEVICE fp32 [N*max_new] out; 0 for t >= lengths[s]
 * The KV pool must hold every completion position at once (the default pool
 * does).  Returns after the stream has finished the work.  Errors: RG_EINVAL
 * (arguments, a length outside [1, max_new], a token id outside [0, vocab)),
 * RG_ENOMEM (limits or KV pool), RG_EHIP. */
int recompute_logprobs(rg_policy* pol, const int32_t* prompts, const int32_t* prompt_len, int32_t P,
                       const int32_t* G, const int32_t* tokens, const int32_t* lengths, int32_t max_new,
                       float temperature, int32_t flags, float* logprobs, void* stream);

/* Aggregation modes of grpo_surrogate */
#define RG_LOSS_TOKEN_MEAN 0   /* DAPO: mean over every counted token                        */
#define RG_LOSS_SEQ_MEAN   1   /* GRPO: mean over sequences of each sequence's token mean    */

/* Clipped surrogate of the GRPO / DAPO objective (the PPO clip that both
 * papers the method trains with use; the paper itself gives no formula).  Per
 * token t < lengths[s]: rho = exp(new_lp - old_lp) and the term
 * min(rho*A_s, clip(rho, 1 - eps_lo, 1 + eps_hi)*A_s), all in fp64; eps_lo =
 * eps_hi is the PPO/GRPO clip, eps_hi > eps_lo DAPO's decoupled one.  No KL
 * term.  Sequences of groups with keep[p] == 0 are left out.
 *   new_lp, old_lp  DEVICE fp32 [N*max_new]
 *   adv             DEVICE fp32 [N] (group_advantage's output)
 *   lengths         DEVICE int32 [N], each in [1, max_new]
 *   G               DEVICE int32 [P], each >= 1, sum N
 *   keep            DEVICE int32 [P] (group_filter's keep) or NULL for all
 *   out             DEVICE fp64 [4]: loss = -(aggregate of the terms), the
 *                   fraction of counted tokens where the clip is active (the
 *                   clipped term strictly below the unclipped one), the
 *                   counted tokens and the counted sequences.  All zero when
 *                   nothing is counted; NaN in all four if G is invalid or a
 *                   length lies outside [1, max_new].
 * Two kernels: one wave per sequence sums its terms (fp64) into a 16-byte
 * record of device scratch, then one workgroup adds the records group by
 * group in sequence order; the summation order is fixed, so results are
 * reproducible.  The scratch (16*N bytes) is taken with hipMallocAsync on
 * `stream` and released with hipFreeAsync after the kernels, so concurrent
 * calls on different streams do not share it.  Only enqueues work on
 * `stream`.  Errors: RG_EINVAL for NULL pointers, P, N or max_new < 1, eps_lo
 * outside [0, 1), eps_hi < 0 or an unknown mode; RG_EHIP when the scratch
 * cannot be allocated. */
int grpo_surrogate(const float* new_lp, const float* old_lp, const float* adv, const int32_t* lengths,
                   const int32_t* G, int32_t P, int32_t N, int32_t max_new, const int32_t* keep,
                   double eps_lo, double eps_hi, int32_t mode, double* out, void* stream);

/* grpo_surrogate for callers that cannot allocate device memory: code under
 * HIP graph capture, serving loops that must not call hipMalloc, harnesses
 * that forbid allocation.  Same arguments, checks, kernels and result (bit
 * for bit) as grpo_surrogate, but the per-sequence records go to a static
 * device array of the library, so the call allocates nothing.
 *   Limit: N <= 65536 (the array holds 65536 records of 16 bytes: 1 MiB on
 *   every device the library runs on, held until the process ends); a larger
 *   N gives RG_EINVAL before any device work.
 * Every call on one device uses that device's array: calls that overlap on
 * one device (other streams or threads) race and must be serialized by the
 * caller.  Nothing in it needs clearing: a call writes every record it reads.
 * Only enqueues work on `stream`. */
int grpo_surrogate_noalloc(const float* new_lp, const float* old_lp, const float* adv, const int32_t* lengths,
                           const int32_t* G, int32_t P, int32_t N, int32_t max_new, const int32_t* keep,
                           double eps_lo, double eps_hi, int32_t mode, double* out, void* stream);

/* ---- test and measurement hooks ---- */


/* Raw Philox4x64-10 blocks: out[4i..4i+3] = Philox(ctr[4i..4i+3], key (key0, key1)).
 * ctr and out are DEVICE uint64 [4n].  Enqueue only. */
int rg_philox_blocks(uint64_t key0, uint64_t key1, const uint64_t* ctr, int64_t n, uint64_t* out,
                     void* stream);

/* The 32-bit values the sampler draws for sequence s at step t: out[v] for
 * v < vocab, from block Philox((v>>3, t, s, 0), (seed, 1)), 32-bit half (v&1)
 * (low first) of 64-bit word ((v&7)>>1).  out is DEVICE uint32 [vocab]. */
int rg_gumbel_bits(uint64_t seed, int32_t t, int32_t s, int32_t vocab, uint32_t* out, void* stream);

/* Measured streaming ceiling for the HBM rooflines (not a step of the path):
 * one launch of `blocks` workgroups of 256 threads that stream `bytes` (a
 * positive multiple of 16) of DEVICE memory at src in 16-byte pieces.
 * mode 1: copy to DEVICE dst [bytes]; mode 0: read only, one uint32 per
 * thread stored to DEVICE dst [blocks * 256 * 4 bytes].  src and dst must not
 * overlap and must be 16-byte aligned.  Enqueue only; RG_EINVAL on a bad
 * argument. */
int rg_hbm_probe(const void* src, void* dst, int64_t bytes, int32_t mode, int32_t blocks, void* stream);

/* Per-step record of the last rollout_group call: active[t] = sequences still
 * decoding at step t (t = 0 is the first sampled token), groups[t] = prompts
 * with at least one of them, ctx[t] = sum over those sequences of their prompt
 * length.  Each array is HOST [cap]; *n_steps receives the number of steps
 * (the longest completion), at most cap entries are written.  Any array may be
 * NULL. */
int rg_step_history(const rg_policy* pol, int32_t cap, int32_t* n_steps, int32_t* active,
                    int32_t* groups, int64_t* ctx);

/* Device-timeline split of the last successful rollout_group call, from HIP
 * events the call records on its stream: *prefill_ms from the start of the
 * prefill to the end of the sibling fork (set-up, every prompt token through
 * the decoder, the prompts' last-position lm head, page copies), *decode_ms
 * from there to the last decode step (step 0's sampling included).  Either
 * pointer may be NULL.  RG_EINVAL when no rollout_group call has completed. */
int rg_phase_times(const rg_policy* pol, double* prefill_ms, double* decode_ms);

/* Context chunks per row of a decode step's attention: for `rows` active
 * sequences (rounded up to the step's row bucket: 16, 32, 64, 128, 256, 384,
 * then multiples of 256), `n_kv` kv heads and the rollout's longest context
 * `ctx_max` (longest prompt + max_new).  Every row's context is cut into that
 * many chunks of at least 128 tokens (fewer when the context is shorter).  For
 * bf16 models with 2 to 8 chunks and at least 256 (row, kv head) pairs, one
 * workgroup per pair combines its chunks' partial softmax results in LDS;
 * otherwise (more than one chunk) each chunk's partial is written out and a
 * merge kernel combines them.  A test and measurement aid; RG_EINVAL (< 0)
 * for a non-positive argument. */
int32_t rg_decode_attention_chunks(int32_t rows, int32_t n_kv, int32_t ctx_max);

/* Kernel classes timed under RG_FLAG_PROFILE. */
#define RG_K_EMBED      0
#define RG_K_RMSNORM    1
#define RG_K_GEMM_QKV   2
#define RG_K_QKV_ROPE   3
#define RG_K_ATTN       4   /* both attention passes: shared prefix and per row */
#define RG_K_ATTN_MERGE 5
#define RG_K_GEMM_O     6
#define RG_K_GEMM_GU    7
#define RG_K_SWIGLU     8
#define RG_K_GEMM_DOWN  9
#define RG_K_RESIDUAL  10
#define RG_K_GEMM_LM   11
#define RG_K_SAMPLE    12
#define RG_K_COMPACT   13
#define RG_K_SETUP     14
#define RG_K_LOGPROB   15   /* token log-probability gather of recompute_logprobs */
#define RG_K_COUNT     16
/* Totals for kernel class `kind` over the prefill (phase 0), every decode
 * step (phase 1) or the decode steps of one row bucket (phase 2 + b for the
 * buckets of at most 16, 32, 64, 128, 256, 384, 512 rows and b = 7 for
 * larger ones) of the last profiled rollout: summed launch durations in
 * milliseconds (HIP events) and the number of launches.  recompute_logprobs
 * records its prompt prefill as phase 0 and its completion rows as phase 1. */
int rg_kernel_times(const rg_policy* pol, int32_t phase, int32_t kind, double* total_ms,
                    int64_t* launches);

#ifdef __cplusplus
}
#endif
#endif /* PAPER_2606_02218_ROLLOUT_H */
