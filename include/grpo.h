/*
 * grpo.h -- C ABI of libgrpo, the MI355X (gfx950) library for the multi-step
 * GRPO token loss of AsyncWebRL (arXiv 2606.05597) and its gradient.
 *
 * The objective (Eq. 1, Sec. 3.2), per task group of G trajectories:
 *   J = 1/(G k) sum_i sum_{j<=|tau_i|} sum_{t in step j}
 *         min( rho_t A_i , omega_t clip(r_t, 1-eps_low, 1+eps_high) A_i )
 *   rho = pi/pi_behave, r = pi/pi_prox, omega = pi_prox/pi_behave,
 *   A_i = (r_i - mean r)/std r over the group (Sec. 3.2),
 *   1/k replaced by 1/|tau_i| for the paper's baseline normaliser (Sec. 3.2),
 *   and, when dual_clip_c > 0 and A_i < 0, the per-token term floored at
 *   c*A_i (Eq. 2, Appendix B.2).  pi is the softmax of the policy's
 *   vocabulary logits at the token's position; importance sampling is per
 *   token (Table 5).
 * The library returns loss = -J averaged over groups,
 *   loss = -sum_t w_{i(t)} s_t,  w_i = 1/(n_groups*G*|tau_i|)  or  1/(n_groups*G*k),
 * and dlogits = grad_scale * dloss/dz, i.e. row t is
 *   g_t * (softmax(z_t) - onehot(a_t)),  g_t = grad_scale * w_i * ds_t/dl_t.
 * pi_behave and pi_prox are constants (no gradient).
 *
 * Conventions for every entry point:
 *  - Pointers named "device" are device memory owned by the caller; the
 *    library never allocates, frees or synchronises.  All work is enqueued on
 *    the caller's stream `s` (0 = the null stream) in stream order.
 *  - Scalars and the structs below are read on the host during the call;
 *    the structs may live on the caller's stack.
 *  - The return value is a grpo_status.  Argument errors are detected on the
 *    host before anything is enqueued; nothing is launched when the status is
 *    negative.  GRPO_ERR_HIP means a HIP launch failed (work enqueued before
 *    it may have run).
 *  - Errors in device data (action ids, offsets, non-finite values) cannot be
 *    seen by the host without a sync: they are reported through
 *    grpo_aux.error_flags and handled as documented there.
 *  - The ragged batch (Eq. 1's triple sum) is CSR: trajectory i owns steps
 *    [traj_step_off[i], traj_step_off[i+1]), step j owns action tokens
 *    [step_tok_off[j], step_tok_off[j+1]) of the packed token axis.  Groups are
 *    G consecutive trajectories.  Only loss-mask (action) tokens are packed.
 */
#ifndef GRPO_H_
#define GRPO_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  GRPO_OK = 0,
  GRPO_ERR_ARG = -1,       /* a required pointer is NULL or a scalar is out of range */
  GRPO_ERR_SHAPE = -2,     /* sizes inconsistent (ld < V, n_traj % group_size, ...)  */
  GRPO_ERR_DTYPE = -3,     /* unsupported dtype                                      */
  GRPO_ERR_WORKSPACE = -4, /* workspace NULL or smaller than the size query         */
  GRPO_ERR_ALIGN = -5,     /* a device pointer is not aligned as documented          */
  GRPO_ERR_HIP = -6        /* a HIP launch returned an error                         */
} grpo_status;

/* Element types of logits and dlogits.  Entry points take the code as an int32_t `dtype` argument, so that any
 * other value reaches their check and is refused with GRPO_ERR_DTYPE. */
typedef enum { GRPO_F32 = 0, GRPO_BF16 = 1 } grpo_dtype;

typedef enum {
  GRPO_NORM_TRAJ_STEPS = 0, /* 1/|tau_i|: the multi-step GRPO baseline (Sec. 3.2) */
  GRPO_NORM_CONST_K = 1     /* 1/k: the paper's constant normaliser (Sec. 3.2)    */
} grpo_norm;

/* Bits of grpo_aux.error_flags (device int32, overwritten by every call). */
#define GRPO_FLAG_ACTION 1    /* some a_t outside [0, V): that row adds 0 and gets a zero dlogits row  */
#define GRPO_FLAG_OFFSETS 2   /* malformed offsets: every dlogits row is zero and the loss is NaN     */
#define GRPO_FLAG_NONFINITE 4 /* a non-finite log-prob, input log-prob or advantage; values propagate */

/* The ragged batch.  Offsets are device int32 arrays.  Valid offsets:
 * step_tok_off[0] = 0, non-decreasing, step_tok_off[n_steps] = T (a step may
 * hold no action token); traj_step_off[0] = 0, strictly increasing (every
 * trajectory has >= 1 step, so |tau_i| >= 1), traj_step_off[n_traj] = n_steps. */
typedef struct {
  int32_t n_traj;               /* N >= 1, a multiple of group_size              */
  int32_t group_size;           /* G >= 1 (Table 5: 8)                           */
  int32_t n_steps;              /* >= n_traj                                     */
  const int32_t* step_tok_off;  /* device [n_steps + 1]                          */
  const int32_t* traj_step_off; /* device [n_traj + 1]                           */
} grpo_segments;

/* Loss hyper-parameters (Table 5 values in brackets). */
typedef struct {
  int32_t norm;          /* grpo_norm                                                      */
  float k;               /* constant normaliser, > 0 when norm = GRPO_NORM_CONST_K [10]    */
  float eps_low;         /* clip range [1 - eps_low, 1 + eps_high], 0 <= eps_low < 1 [0.2] */
  float eps_high;        /* >= 0 [0.2]                                                     */
  float dual_clip_c;     /* 0 disables the dual clip; otherwise > 1 (Eq. 2) [3.0]          */
  float grad_scale;      /* upstream d(objective)/d(loss), folded into dlogits [1]        */
  double n_groups_total; /* groups in the global batch for the normaliser; 0 = N/G        */
} grpo_loss_params;

/* Optional outputs; every field may be NULL (device pointers unless noted). */
typedef struct {
  float* token_logp;     /* [T] new log-prob l_t of each action token (fp32)               */
  int32_t* tok_traj;     /* [T] trajectory of each token                                   */
  int32_t* traj_tok_off; /* [n_traj + 1] first token of each trajectory, then T            */
  int64_t* gather_idx;   /* [T] flat element index t*ld + a_t of each action logit         */
  double* traj_loss;     /* [n_traj] -sum over the trajectory's tokens of w_i s_t          */
  int64_t* clip_counts;  /* [2] tokens whose gradient the eps clip / the dual clip cut     */
  double* ratio_stats;   /* [8] over the tokens that enter the loss: sum r, min r, max r,   */
                         /*   sum rho, min rho, max rho (r = pi/pi_prox, rho = pi/pi_behave, */
                         /*   Sec. 3.2), the number of tokens with r outside               */
                         /*   [1 - eps_low, 1 + eps_high], and the number of such tokens   */
  int32_t* error_flags;  /* [1] GRPO_FLAG_* bits seen by this call                         */
  hipEvent_t hot_begin;  /* host handles: when both are set, recorded on `s` right before  */
  hipEvent_t hot_end;    /*   and after the dominant kernel (for timing)                   */
} grpo_aux;

/*
 * Group-relative advantage (Sec. 3.2): for each group of `group_size`
 * consecutive trajectories, A_i = (r_i - mean)/(std + std_eps), with the std
 * taken with `ddof` degrees of freedom removed (1 = the unbiased estimate).
 * A group whose denominator is 0 gets A = 0.  Sums run in fp64 in index
 * order; the result is stored as fp32.
 *   rewards  device fp32 [n_traj]      adv_out  device fp32 [n_traj]
 * Errors: GRPO_ERR_ARG (NULL pointer, ddof not in {0, 1}, std_eps < 0),
 *         GRPO_ERR_SHAPE (n_traj < 1, group_size < 1, n_traj % group_size).
 */
int grpo_advantages(const float* rewards, int32_t n_traj, int32_t group_size, int32_t ddof, float std_eps,
                    float* adv_out, hipStream_t s);

/* Advantage modes of grpo_advantages_ex. */
typedef enum {
  GRPO_ADV_GROUP_NORM = 0,     /* (r_i - mean)/(std + std_eps) per group (Sec. 3.2)                    */
  GRPO_ADV_SUCCESS_FILTER = 1  /* RAFT++ / filtered behaviour cloning: A_i = 1 if r_i > 0 else 0, no   */
                               /* group normalisation (Sec. 3.2 "RAFT++ as a baseline", Table 5)       */
} grpo_adv_mode;

/*
 * grpo_advantages with a mode and DAPO's dynamic-sampling mask (Sec. 3.2: groups
 * whose rewards are all equal, all successes or all failures, carry no
 * group-relative signal and are skipped when a training batch is gathered).
 *   mode         grpo_adv_mode
 *   group_mixed  device int32 [n_traj / group_size] or NULL: 1 when the
 *                group's rewards are not all equal, else 0
 *   n_mixed      device int32 [1] or NULL: the number of mixed groups (what a
 *                caller that drops the other groups passes as n_groups_total)
 * Other arguments and errors as grpo_advantages, plus GRPO_ERR_ARG for an
 * unknown mode.  ddof and std_eps are checked but unused under the filter.
 */
int grpo_advantages_ex(const float* rewards, int32_t n_traj, int32_t group_size, int32_t mode, int32_t ddof,
                       float std_eps, float* adv_out, int32_t* group_mixed, int32_t* n_mixed, hipStream_t s);

/* Bytes of device workspace grpo_loss_fwd_bwd needs for T tokens and n_traj trajectories. */
size_t grpo_loss_workspace_bytes(int64_t T, int32_t n_traj);

/*
 * The logits path: loss and dlogits of Eq. 1 (+ Eq. 2) from the policy's
 * vocabulary logits at every action token.
 *   logits       device [T, ld] of `dt`, row t = token t; columns >= V unread
 *   dtype        GRPO_BF16 or GRPO_F32 (dlogits has the same dtype)
 *   T >= 0, 1 <= V <= ld
 *   actions      device int32 [T]  sampled token ids a_t
 *   behave_logp  device fp32 [T]   log pi_behave(a_t), recorded at rollout
 *   prox_logp    device fp32 [T]   log pi_prox(a_t); NULL = behave_logp (the
 *                                  coupled ratio, Sec. 4.3)
 *   adv          device fp32 [n_traj]  A_i (e.g. from grpo_advantages)
 *   seg, p       host structs (above)
 *   loss_out     device fp64 [1]   the loss (not multiplied by grad_scale)
 *   dlogits      device [T, ld] of `dt`; columns >= V are not written; NULL =
 *                forward only.  It may alias `logits` (each row is read in
 *                full before any of it is written).
 *   aux          host struct of optional outputs, or NULL
 *   ws, ws_bytes device workspace of at least grpo_loss_workspace_bytes(T, n_traj)
 * The loss and traj_loss are reduced in a fixed order (bitwise reproducible).
 * Errors: GRPO_ERR_ARG (NULL required pointer; k <= 0 under CONST_K;
 *   eps_low not in [0,1); eps_high < 0; dual_clip_c in (0, 1] or < 0;
 *   non-finite grad_scale; n_groups_total < 0), GRPO_ERR_SHAPE (T < 0, V < 1,
 *   ld < V, n_traj < 1, group_size < 1, n_traj % group_size, n_steps < n_traj,
 *   T >= 2^31), GRPO_ERR_DTYPE, GRPO_ERR_WORKSPACE, GRPO_ERR_ALIGN (logits or
 *   dlogits not aligned to the element size), GRPO_ERR_HIP.
 */
int grpo_loss_fwd_bwd(const void* logits, int32_t dtype, int64_t T, int64_t V, int64_t ld,
                      const int32_t* actions, const float* behave_logp, const float* prox_logp,
                      const float* adv, const grpo_segments* seg, const grpo_loss_params* p, double* loss_out,
                      void* dlogits, grpo_aux* aux, void* ws, size_t ws_bytes, hipStream_t s);

/* Size of the device scratch array behind grpo_loss_fwd_bwd_noalloc (24 MiB): the largest
 * grpo_loss_workspace_bytes(T, n_traj) it serves, e.g. T = 262,144 tokens with n_traj up to 16,384. */
#define GRPO_NOALLOC_SCRATCH_BYTES ((size_t)24 << 20)

/*
 * grpo_loss_fwd_bwd for callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): the same computation, kernels and results, with the
 * workspace taken from a device array of GRPO_NOALLOC_SCRATCH_BYTES that the library holds on each device
 * (reserved when the library's code is loaded on the device and kept until the process ends).  The call itself
 * allocates and frees nothing; on its first call on a device it looks the array's address up (with that
 * device current).  The caller still passes every input and output, as for grpo_loss_fwd_bwd.
 * Every call on a device shares that device's array and leaves the last call's contents in it: two calls that
 * overlap on one device (on different streams, or from different host threads without ordering) race and
 * their results are undefined.  Calls ordered on one stream are safe.
 * Arguments: as grpo_loss_fwd_bwd, without ws and ws_bytes.
 * Errors: as grpo_loss_fwd_bwd; GRPO_ERR_WORKSPACE when grpo_loss_workspace_bytes(T, n_traj) exceeds
 *   GRPO_NOALLOC_SCRATCH_BYTES (nothing is launched); GRPO_ERR_HIP when the stream's device cannot be found
 *   or the array's address cannot be looked up.
 */
int grpo_loss_fwd_bwd_noalloc(const void* logits, int32_t dtype, int64_t T, int64_t V, int64_t ld,
                              const int32_t* actions, const float* behave_logp, const float* prox_logp,
                              const float* adv, const grpo_segments* seg, const grpo_loss_params* p,
                              double* loss_out, void* dlogits, grpo_aux* aux, hipStream_t s);

/* Bytes of device workspace fused_lmhead_grpo needs. */
size_t fused_lmhead_workspace_bytes(int64_t T, int64_t H, int64_t V, int32_t vocab_chunk, int32_t n_traj);

/*
 * The fused LM-head path: the same loss computed from the final hidden states
 * h [T, H] and the LM-head weight W [H, V], with z = h W formed on the matrix
 * cores in vocabulary chunks of `vocab_chunk` columns and never stored whole.
 * Emits the loss, dhidden = dloss/dh = D W^T and dW = dloss/dW = h^T D, where
 * D = grad_scale * dloss/dz (bf16-rounded per chunk before the two products).
 *   hidden       device bf16 [T, H] row-major       w_lm device bf16 [H, V] row-major
 *   0 <= T <= 8,388,352 and 8 <= V <= 8,388,352 (2^23 - 256: the matrix-core products address
 *   256 of their T- or V-long operand rows with 32-bit offsets), V a multiple of 8, H >= 64 and
 *   a multiple of 64,
 *   vocab_chunk  a positive multiple of 256 (8192 is the tuned value)
 *   actions, behave_logp, prox_logp, adv, seg, p, loss_out, aux: as above
 *   (aux->gather_idx uses ld = V)
 *   dhidden      device bf16 [T, H]  (written)
 *   dw_lm        device fp32 [H, V]; written, or accumulated into when
 *                accumulate_dw != 0
 *   ws, ws_bytes device workspace of at least fused_lmhead_workspace_bytes(...)
 * hidden, w_lm, dhidden and dw_lm must be 16-byte aligned (GRPO_ERR_ALIGN).
 * Errors: as grpo_loss_fwd_bwd, plus GRPO_ERR_SHAPE for H, V or vocab_chunk
 *   outside the ranges above.
 */
int fused_lmhead_grpo(const void* hidden, const void* w_lm, int64_t T, int64_t H, int64_t V, int32_t vocab_chunk,
                      const int32_t* actions, const float* behave_logp, const float* prox_logp, const float* adv,
                      const grpo_segments* seg, const grpo_loss_params* p, double* loss_out, void* dhidden,
                      float* dw_lm, int32_t accumulate_dw, grpo_aux* aux, void* ws, size_t ws_bytes,
                      hipStream_t s);

/* Bytes of device workspace fused_lmhead_grpo_blocked needs: besides W^T, h^T and the per-row scales, the fp16
 * logit terms and tile partials of two blocks (one when a single block covers T) and one block's D and D^T,
 * about (2 + 2 + 2 + 2) * B * Vp bytes with B = min(token_block, T rounded up to 256) and Vp = V rounded up to
 * 256 (12.7 GB in all at T = 65,536, H = 3,584, V = 151,936, token_block = 8192).  0 for invalid sizes. */
size_t fused_lmhead_blocked_workspace_bytes(int64_t T, int64_t H, int64_t V, int32_t token_block, int32_t n_traj);

/*
 * The fused LM-head path of fused_lmhead_grpo, scheduled over blocks of tokens instead of vocabulary chunks, and
 * with the same results up to the order of fp32 sums.  The forward product of a block of `token_block` rows
 * (z = h W, on the matrix cores, 256-column tiles) is kept in the workspace until the block's rows have their
 * log-sum-exp, as each logit's term exp(z - m) in fp16 (m its row's maximum over the tile: terms <= 1, relative
 * error <= 2^-11 down to 2^-14); D of the block is then formed from the stored terms (one multiply per logit)
 * instead of a second product, so three products run instead of four.  The logits of the whole batch are never
 * stored: at most two blocks at a time.
 * Per block: dhidden rows = D W^T (the whole vocabulary as K, written once in bf16), dW (+)= h^T D.
 *   token_block  a positive multiple of 256, at most 8,388,352 (8192 is the tuned value)
 *   all other arguments as fused_lmhead_grpo
 *   ws, ws_bytes device workspace of at least fused_lmhead_blocked_workspace_bytes(...)
 *   s_aux        NULL (or s): everything runs on s.  Otherwise a second stream of the caller's, on the same
 *                device: each block's D pass (stored terms -> D, D^T) then runs on s_aux beside the next
 *                block's forward product on s.  The call orders the two streams with two HIP events it creates
 *                and releases itself; s_aux's work is joined back into s before the last launch on s, so the
 *                results are complete in s's order, as with one stream (and the call can be captured from s
 *                into a HIP graph).  The results are bit-identical either way.
 * Errors: as fused_lmhead_grpo (GRPO_ERR_SHAPE for token_block outside the range above); GRPO_ERR_ARG if s_aux
 *   is on another device than s; GRPO_ERR_HIP if an event cannot be created.
 */
int fused_lmhead_grpo_blocked(const void* hidden, const void* w_lm, int64_t T, int64_t H, int64_t V,
                              int32_t token_block, const int32_t* actions, const float* behave_logp,
                              const float* prox_logp, const float* adv, const grpo_segments* seg,
                              const grpo_loss_params* p, double* loss_out, void* dhidden, float* dw_lm,
                              int32_t accumulate_dw, grpo_aux* aux, void* ws, size_t ws_bytes, hipStream_t s,
                              hipStream_t s_aux);

/*
 * Forward only: the sampled action's log-prob and the policy entropy of each
 * token row, with no loss and no dlogits -- the proximal log-probs recomputed
 * before an update (Table 5: decoupled PPO, proximal logprobs recomputed) and
 * the per-token entropy the paper averages over the loss mask (Sec. 5).
 *   l_t = z_t[a_t] - log sum_v exp z_t[v],   H_t = -sum_v p_v log p_v,  p = softmax(z_t)
 *   logits       device [T, ld] of `dt`, row t = token t; columns >= V unread
 *   T >= 0, 1 <= V <= ld
 *   actions      device int32 [T]
 *   token_logp   device fp32 [T] or NULL   l_t (0 where a_t is outside [0, V))
 *   token_entropy device fp32 [T] or NULL  H_t
 *   error_flags  device int32 [1] or NULL: overwritten with GRPO_FLAG_ACTION when
 *                some a_t is outside [0, V), GRPO_FLAG_NONFINITE when a row's
 *                log-sum-exp is not finite
 * Each row is read once (2V or 4V bytes); sums run in fp32 per thread and fp64
 * across the row.
 * Errors: GRPO_ERR_ARG (logits or actions NULL), GRPO_ERR_SHAPE (T < 0, V < 1,
 *   ld < V, T >= 2^31), GRPO_ERR_DTYPE, GRPO_ERR_ALIGN (logits not aligned to
 *   the element size), GRPO_ERR_HIP.
 */
int grpo_token_logp(const void* logits, int32_t dtype, int64_t T, int64_t V, int64_t ld, const int32_t* actions,
                    float* token_logp, float* token_entropy, int32_t* error_flags, hipStream_t s);

/* Bytes of device workspace fused_lmhead_token_logp needs (W^T and the per-(row, 256-column tile) partials:
 * 2 V H + 12 T ceil(V / 256) bytes, rounded up); 0 for invalid sizes. */
size_t fused_lmhead_token_logp_workspace_bytes(int64_t T, int64_t H, int64_t V);

/*
 * Forward only from the final hidden states: grpo_token_logp's outputs (the action's log-prob and the policy
 * entropy per token, for the proximal log-probs recomputed before an update, Table 5, and the entropy of Sec. 5)
 * with z = h W formed on the matrix cores in 256-column tiles and never stored.
 *   hidden, w_lm, T, H, V: as fused_lmhead_grpo
 *   actions      device int32 [T]
 *   token_logp   device fp32 [T] or NULL   l_t (0 where a_t is outside [0, V))
 *   token_entropy device fp32 [T] or NULL  H_t; NULL skips its partial sums in the product's epilogue
 *   error_flags  device int32 [1] or NULL: overwritten with GRPO_FLAG_ACTION when some a_t is outside [0, V),
 *                GRPO_FLAG_NONFINITE when a row's log-sum-exp is not finite
 *   ws, ws_bytes device workspace of at least fused_lmhead_token_logp_workspace_bytes(T, H, V)
 * Per row: the tile partials (max, sum e^(z - m), sum e^(z - m)(z - m)) merged in fp64; the action logit
 * h_t . W[:, a_t] as an fp64 dot product of the bf16 inputs.
 * Errors: GRPO_ERR_ARG, GRPO_ERR_SHAPE (as fused_lmhead_grpo), GRPO_ERR_ALIGN (hidden, w_lm not 16-byte aligned,
 *   outputs not 4-byte aligned), GRPO_ERR_WORKSPACE, GRPO_ERR_HIP.
 */
int fused_lmhead_token_logp(const void* hidden, const void* w_lm, int64_t T, int64_t H, int64_t V,
                            const int32_t* actions, float* token_logp, float* token_entropy, int32_t* error_flags,
                            void* ws, size_t ws_bytes, hipStream_t s);

/*
 * The vocabulary split over devices (tensor-parallel LM head; the extension of
 * the loss of Eq. 1 to a sharded vocabulary): the calls one device makes for the
 * shard it holds, logits [T, V_shard] of global columns [v_begin, v_begin +
 * V_shard).  The exchange between the two calls (gathering every shard's
 * records on every device) is the caller's.
 *
 * One shard's per-token record, 24 bytes, all fp64 (no rounding between the
 * shard's reduction and the merge):
 *   m    max over the shard's columns of the row (-inf for a row of -inf)
 *   s    sum over the shard's columns of exp(z - m)
 *   z_a  the action's logit if a_t is one of the shard's columns, else -inf
 * Any split of a row merges back to its log-sum-exp M + log sum_g s_g exp(m_g - M),
 * M = max_g m_g, and to its action logit max_g z_a_g.
 */
typedef struct {
  double m;
  double s;
  double z_a;
} grpo_vocab_stats;

/*
 * Step 1 of the sharded loss: every row of the shard reduced to its record.
 *   logits       device [T, ld] of `dt`, the shard's columns; columns >= V_shard unread
 *   T >= 0, 1 <= V_shard <= ld, v_begin >= 0, v_begin + V_shard < 2^31
 *   actions      device int32 [T]  global token ids
 *   stats        device grpo_vocab_stats [T], 8-byte aligned (written)
 *   error_flags  device int32 [1] or NULL: overwritten with GRPO_FLAG_NONFINITE
 *                when a row's shard log-sum-exp is NaN or +inf (an action outside
 *                the shard is not an error here; step 2 checks a_t against V_total)
 * Each row is read once; the record's sums run in fp32 per thread and fp64 across the row.
 * Errors: GRPO_ERR_ARG (logits, actions or stats NULL), GRPO_ERR_SHAPE, GRPO_ERR_DTYPE,
 *   GRPO_ERR_ALIGN, GRPO_ERR_HIP.
 */
int grpo_vocab_shard_stats(const void* logits, int32_t dtype, int64_t T, int64_t V_shard, int64_t ld,
                           int64_t v_begin, const int32_t* actions, grpo_vocab_stats* stats, int32_t* error_flags,
                           hipStream_t s);

/*
 * Step 2 of the sharded loss: the loss and the shard's columns of dlogits.
 *   logits, dt, T, V_shard, ld, v_begin: the shard, as in step 1
 *   V_total      the whole vocabulary (actions outside [0, V_total) are flagged and
 *                their tokens leave the loss, as in grpo_loss_fwd_bwd)
 *   stats        device grpo_vocab_stats [n_shards][T]: every shard's records from
 *                step 1, in the same shard order on every device; 8-byte aligned
 *   n_shards     1 .. 65536
 *   actions, behave_logp, prox_logp, adv, seg, p, loss_out, aux, ws, ws_bytes: as
 *                grpo_loss_fwd_bwd (workspace from grpo_loss_workspace_bytes; the
 *                loss and every per-token output are the whole row's, the same on
 *                every shard; aux->gather_idx gets t*ld + a_t with the global a_t)
 *   dlogits      device [T, ld] of `dt`, the shard's columns of dloss/dz * grad_scale;
 *                NULL = forward only; may alias `logits`
 * Per row the records are merged in shard order (so every shard computes the same
 * bits), then the row's d_v = g_t (exp(z_v - lse) - [v = a_t]) over the shard's
 * columns.  Errors: as grpo_loss_fwd_bwd, plus GRPO_ERR_SHAPE for v_begin < 0,
 * v_begin + V_shard > V_total, V_total >= 2^31 or n_shards outside 1..65536, and
 * GRPO_ERR_ARG for stats NULL with T > 0.
 */
int grpo_loss_fwd_bwd_vocab_shard(const void* logits, int32_t dtype, int64_t T, int64_t V_shard, int64_t ld,
                                  int64_t v_begin, int64_t V_total, const grpo_vocab_stats* stats, int32_t n_shards,
                                  const int32_t* actions, const float* behave_logp, const float* prox_logp,
                                  const float* adv, const grpo_segments* seg, const grpo_loss_params* p,
                                  double* loss_out, void* dlogits, grpo_aux* aux, void* ws, size_t ws_bytes,
                                  hipStream_t s);

/* Bytes of device workspace fused_lmhead_vocab_shard_stats needs (the shard's W^T and pass-1 partials). */
size_t fused_lmhead_vocab_shard_stats_workspace_bytes(int64_t T, int64_t H, int64_t V_shard);

/*
 * Step 1 of the sharded fused LM head: the device holding W's columns
 * [v_begin, v_begin + V_shard) reduces every row of z = h W_shard to its
 * grpo_vocab_stats record (m and s from the matrix-core logits; z_a = h_t .
 * W[:, a_t] in fp64 when a_t is one of the shard's columns).
 *   hidden       device bf16 [T, H] row-major       w_shard device bf16 [H, V_shard] row-major
 *   T >= 0, H >= 64 and a multiple of 64, V_shard >= 8 and a multiple of 8,
 *   v_begin >= 0, v_begin + V_shard < 2^31
 *   actions      device int32 [T]  global token ids
 *   stats        device grpo_vocab_stats [T] (written)
 *   logits_out   NULL, or device fp32 [Tp, Vsp] (Tp = T and Vsp = V_shard rounded up to 256, row stride Vsp;
 *                fused_lmhead_vocab_shard_logits_bytes(T, V_shard) bytes, caller-owned): written with the
 *                shard's logits z = h W_shard as the matrix cores formed them (zeros past T and V_shard), for
 *                step 2 to use instead of forming them again
 *   ws, ws_bytes device workspace of at least fused_lmhead_vocab_shard_stats_workspace_bytes(T, H, V_shard)
 * hidden, w_shard and logits_out must be 16-byte aligned, stats 8-byte aligned.
 * Errors: GRPO_ERR_ARG, GRPO_ERR_SHAPE, GRPO_ERR_ALIGN, GRPO_ERR_WORKSPACE, GRPO_ERR_HIP.
 */
int fused_lmhead_vocab_shard_stats(const void* hidden, const void* w_shard, int64_t T, int64_t H, int64_t V_shard,
                                   int64_t v_begin, const int32_t* actions, grpo_vocab_stats* stats,
                                   float* logits_out, void* ws, size_t ws_bytes, hipStream_t s);

/* Bytes of the logits buffer of fused_lmhead_vocab_shard_stats and fused_lmhead_grpo_vocab_shard:
 * 4 * (T rounded up to 256) * (V_shard rounded up to 256); 0 for T < 0 or V_shard < 1. */
size_t fused_lmhead_vocab_shard_logits_bytes(int64_t T, int64_t V_shard);

/*
 * Step 2 of the sharded fused LM head: given every shard's records (gathered by the
 * caller, the same shard order on every device), the loss (the whole rows', the same
 * on every shard), this shard's dW columns and its partial dhidden.
 *   hidden, w_shard, T, H, V_shard, v_begin: as in step 1, and T, V_shard <= 8,388,352 as in
 *                fused_lmhead_grpo
 *   V_total      the whole vocabulary; vocab_chunk as in fused_lmhead_grpo
 *   stats        device grpo_vocab_stats [n_shards][T], 8-byte aligned; n_shards 1 .. 65536
 *   actions, behave_logp, prox_logp, adv, seg, p, loss_out, aux: as grpo_loss_fwd_bwd
 *   dhidden_partial device fp32 [T, H] (written): D_shard W_shard^T, the shard's share of
 *                dhidden; the caller sums the shards' partials (a reduce-scatter across
 *                devices) and rounds as it needs
 *   dw_shard     device fp32 [H, V_shard]: this shard's dW columns, written or
 *                accumulated into (accumulate_dw != 0)
 *   logits_in    NULL: the shard's logits are formed again on the matrix cores, chunk by chunk (four
 *                products in the two steps).  Otherwise the buffer step 1 filled through logits_out
 *                (unchanged since): D is formed from it and only the two backward products run (three
 *                in the two steps); vocab_chunk is then not used, the shard is one chunk of Vsp columns
 *   ws, ws_bytes device workspace of at least fused_lmhead_workspace_bytes(T, H, V_shard,
 *                vocab_chunk, n_traj), with vocab_chunk = Vsp when logits_in is given
 * D = grad_scale * dloss/dz is rounded to bf16 per chunk before the two products, as in
 * fused_lmhead_grpo; both ways give bit-identical loss, per-token outputs and D.  Errors: as
 * fused_lmhead_grpo, plus GRPO_ERR_SHAPE for v_begin < 0, v_begin + V_shard > V_total,
 * V_total >= 2^31 or n_shards outside 1..65536, GRPO_ERR_ARG for stats or dhidden_partial NULL
 * with T > 0, and GRPO_ERR_ALIGN for logits_in not 16-byte aligned.
 */
int fused_lmhead_grpo_vocab_shard(const void* hidden, const void* w_shard, int64_t T, int64_t H, int64_t V_shard,
                                  int64_t v_begin, int64_t V_total, int32_t vocab_chunk, const grpo_vocab_stats* stats,
                                  int32_t n_shards, const int32_t* actions, const float* behave_logp,
                                  const float* prox_logp, const float* adv, const grpo_segments* seg,
                                  const grpo_loss_params* p, double* loss_out, float* dhidden_partial, float* dw_shard,
                                  int32_t accumulate_dw, grpo_aux* aux, const float* logits_in, void* ws,
                                  size_t ws_bytes, hipStream_t s);

/* A static, human-readable name for a grpo_status value. */
const char* grpo_status_str(int status);

#ifdef __cplusplus
}
#endif

#endif /* GRPO_H_ */
