/*
 * Plain fp64 CPU oracle for the multi-step GRPO token loss and its gradient.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may include, link or
 * call this file; only the test suite, the smoke check and the CPU-baseline leg
 * of the benchmark use it.  It shares no code, header, table or helper with the
 * HIP library: every quantity is recomputed here from its definition, in double
 * precision, in the order the paper states it, with no blocking or fusion.
 *
 * What it follows (AsyncWebRL, arXiv 2606.05597):
 *   - Eq. 1 (Sec. 3.2): J = E[ 1/(G k) sum_i sum_j sum_t min( pi/pi_b * A_i ,
 *         pi_prox/pi_b * clip(pi/pi_prox, 1-eps, 1+eps) * A_i ) ].
 *   - Sec. 3.2, "Removing trajectory-length normalization": the baseline uses
 *     1/|tau_i| (step count of trajectory i) in place of 1/k.
 *   - Sec. 3.2, advantage: A_i = (r_i - mean(r)) / std(r) over the G rollouts
 *     of one task, shared by every token of trajectory i.
 *   - Appendix B.2, Eq. 2: for A < 0 the per-token term is floored at c*A.
 *   - Appendix C.5 (Table 5): token-level importance sampling, eps = 0.2,
 *     c = 3.0, G = 8, k = 10.
 * The per-token log-probability of the sampled action is the log-softmax of
 * the policy's vocabulary logits at that token (implied by Eq. 1; the paper
 * never spells the kernel out).  The loss handed to the optimiser is -J.
 * Forward only (oracle_logp_entropy): that log-probability and the policy
 * entropy -sum p log p per token, the quantity of the GRPO vs. RAFT++
 * comparison (Sec. 5).
 * Vocabulary split over devices (oracle_vocab_shard_stats): one shard's max,
 * sum of exponentials and action logit per token, by their plain definitions;
 * the paper trains on one node per update and does not split the vocabulary,
 * so this serves the sharded variant of the same loss.
 *
 * Readings where the paper is silent, as this file takes them: std uses
 * `ddof` (default 1) and a zero group std gives A = 0; groups combine by
 * their mean, so the per-token weight
 * is w_i = 1/(n_groups * G * |tau_i|) or 1/(n_groups * G * k); the eps clip is
 * inclusive (gradient flows at r = 1 +- eps); the dual clip is active only
 * when s < c*A strictly.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_ERR_ACTION 1    /* an action id outside [0, V)            */
#define ORACLE_ERR_OFFSETS 2   /* step/trajectory offsets are malformed  */
#define ORACLE_ERR_NONFINITE 4 /* a non-finite log-prob or input scalar  */

#define ORACLE_NORM_TRAJ_STEPS 0 /* 1/|tau_i|  (paper's baseline) */
#define ORACLE_NORM_CONST_K 1    /* 1/k        (paper's fix)      */

/* ---- element access: stored inputs converted exactly to double ---------- */

/* dtype 0: IEEE binary32; 1: bfloat16 (upper half of a binary32); 2: binary64 */
static double load_elem(const void* base, int dtype, int64_t idx) {
  if (dtype == 0) return (double)((const float*)base)[idx];
  if (dtype == 2) return ((const double*)base)[idx];
  uint16_t h = ((const uint16_t*)base)[idx];
  uint32_t bits = ((uint32_t)h) << 16; /* a bfloat16 is the top 16 bits of a float */
  float f;
  memcpy(&f, &bits, sizeof f);
  return (double)f;
}

/* ---- segments: trajectories -> steps -> tokens (Eq. 1's triple sum) ----- */

/* The ragged batch is given as CSR offsets: step j holds tokens
 * [step_tok_off[j], step_tok_off[j+1]) and trajectory i holds steps
 * [traj_step_off[i], traj_step_off[i+1]).  |tau_i| is the number of steps of
 * trajectory i (Eq. 1's middle sum).  Valid offsets: both start at 0, token
 * offsets never decrease and end at T, step offsets strictly increase (every
 * trajectory has at least one step) and end at n_steps.
 * Returns 0 or ORACLE_ERR_OFFSETS; on error the outputs are filled with -1. */
int oracle_segments(int64_t T, int32_t n_steps, const int32_t* step_tok_off, int32_t n_traj,
                    const int32_t* traj_step_off, int32_t* traj_tok_off, int32_t* tok_traj,
                    int32_t* traj_steps) {
  int ok = (n_steps >= 1 && n_traj >= 1);
  if (ok) ok = step_tok_off[0] == 0 && (int64_t)step_tok_off[n_steps] == T;
  for (int32_t j = 0; ok && j < n_steps; ++j)
    if (step_tok_off[j + 1] < step_tok_off[j]) ok = 0;
  if (ok) ok = traj_step_off[0] == 0 && traj_step_off[n_traj] == n_steps;
  for (int32_t i = 0; ok && i < n_traj; ++i)
    if (traj_step_off[i + 1] <= traj_step_off[i]) ok = 0;
  if (!ok) {
    if (traj_tok_off)
      for (int32_t i = 0; i <= n_traj; ++i) traj_tok_off[i] = -1;
    if (tok_traj)
      for (int64_t t = 0; t < T; ++t) tok_traj[t] = -1;
    if (traj_steps)
      for (int32_t i = 0; i < n_traj; ++i) traj_steps[i] = -1;
    return ORACLE_ERR_OFFSETS;
  }
  for (int32_t i = 0; i < n_traj; ++i) {
    int32_t first = step_tok_off[traj_step_off[i]];
    int32_t last = step_tok_off[traj_step_off[i + 1]];
    if (traj_tok_off) traj_tok_off[i] = first;
    if (traj_steps) traj_steps[i] = traj_step_off[i + 1] - traj_step_off[i];
    if (tok_traj)
      for (int32_t t = first; t < last; ++t) tok_traj[t] = i;
  }
  if (traj_tok_off) traj_tok_off[n_traj] = (int32_t)T;
  return 0;
}

/* ---- group-relative advantage (Sec. 3.2) -------------------------------- */

/* A_i = (r_i - mean_g r) / (std_g r + std_eps) over the G contiguous
 * trajectories of group g, std with `ddof` degrees of freedom removed.  A
 * group whose denominator is 0 (all rewards equal, std_eps = 0) gets A = 0. */
void oracle_advantages(const float* rewards, int32_t n_traj, int32_t G, int32_t ddof, double std_eps,
                       double* adv) {
  for (int32_t g0 = 0; g0 < n_traj; g0 += G) {
    double mean = 0.0;
    for (int32_t i = 0; i < G; ++i) mean += (double)rewards[g0 + i];
    mean /= (double)G;
    double ss = 0.0;
    for (int32_t i = 0; i < G; ++i) {
      double d = (double)rewards[g0 + i] - mean;
      ss += d * d;
    }
    double sd = (G - ddof > 0) ? sqrt(ss / (double)(G - ddof)) : 0.0;
    double den = sd + std_eps;
    for (int32_t i = 0; i < G; ++i)
      adv[g0 + i] = (den == 0.0) ? 0.0 : ((double)rewards[g0 + i] - mean) / den;
  }
}

/* RAFT++ / filtered behaviour cloning (Sec. 3.2, "RAFT++ as a baseline";
 * Table 5): group normalisation is off and the advantage is the success
 * filter, A_i = 1 when r_i > 0 and 0 otherwise, so only successful
 * trajectories carry gradient. */
void oracle_advantages_success_filter(const float* rewards, int32_t n_traj, double* adv) {
  for (int32_t i = 0; i < n_traj; ++i) adv[i] = (rewards[i] > 0.0f) ? 1.0 : 0.0;
}

/* DAPO dynamic sampling (Sec. 3.2): a group whose G rewards are all equal
 * (all successes or all failures) carries no group-relative signal and is
 * skipped.  mixed[g] = 1 when the rewards of group g are not all equal;
 * returns the number of such groups. */
int32_t oracle_mixed_groups(const float* rewards, int32_t n_traj, int32_t G, int32_t* mixed) {
  int32_t n = 0;
  for (int32_t g = 0; g * G < n_traj; ++g) {
    int m = 0;
    for (int32_t i = 1; i < G; ++i)
      if (rewards[g * G + i] != rewards[g * G]) m = 1;
    mixed[g] = m;
    n += m;
  }
  return n;
}

/* ---- per-token log-probability: log-softmax over V, then gather --------- */

/* lse = log sum_v exp(z_v), computed as m + log sum exp(z_v - m). */
static double row_logsumexp(const void* logits, int dtype, int64_t row_base, int64_t V) {
  double m = -INFINITY;
  for (int64_t v = 0; v < V; ++v) {
    double z = load_elem(logits, dtype, row_base + v);
    if (z > m || isnan(z)) m = z;
  }
  if (isnan(m) || isinf(m)) return m;
  double s = 0.0;
  for (int64_t v = 0; v < V; ++v) s += exp(load_elem(logits, dtype, row_base + v) - m);
  return m + log(s);
}

/* ---- per-token surrogate of Eq. 1 with the dual clip of Eq. 2 ----------- */

/* Returns s (the per-token term inside Eq. 1's sums) and ds/dl, its
 * derivative with respect to the token's new log-prob l.  b = behave log-prob,
 * p = proximal log-prob (p = b gives the coupled ratio).  *state gets bit 0
 * when the eps clip cut the gradient and bit 1 when the dual clip did. */
static double token_surrogate(double l, double b, double p, double A, double eps_lo, double eps_hi,
                              double c, double* dsdl, int* state) {
  double rho = exp(l - b);   /* pi_theta / pi_behave (unclipped ratio)  */
  double r = exp(l - p);     /* pi_theta / pi_prox   (clipped ratio)    */
  double omega = exp(p - b); /* pi_prox  / pi_behave (staleness weight) */
  double lo = 1.0 - eps_lo, hi = 1.0 + eps_hi;
  int outside = (r < lo) || (r > hi);
  double r_clip = r < lo ? lo : (r > hi ? hi : r);
  double u1 = rho * A;
  double u2 = omega * r_clip * A;
  double s, d;
  *state = 0;
  if (u1 <= u2) { /* min picks the unclipped term (ties too) */
    s = u1;
    d = u1; /* d(rho)/dl = rho */
  } else {
    s = u2;
    d = outside ? 0.0 : omega * r * A; /* inside the range clip(r) = r */
    if (outside) *state |= 1;
  }
  if (c > 0.0 && A < 0.0 && s < c * A) { /* Eq. 2: floor at c*A */
    s = c * A;
    d = 0.0;
    *state |= 2;
  }
  *dsdl = d;
  return s;
}

/* The quantities of Eq. 1 for one token once its new log-prob l is known:
 * the trajectory weight w_i = 1/(n_groups * G * (|tau_i| or k)), the term s_t,
 * the token's share of the loss -w_i s_t and its coefficient
 * g_t = grad_scale * w_i * ds_t/dl_t.  Returns ORACLE_ERR_NONFINITE when an
 * input is not finite (the values then propagate), else 0. */
static int token_terms(double l, float behave, float prox, double A, int32_t steps, int32_t group_size,
                       double n_groups, int norm, double k, double eps_lo, double eps_hi, double c,
                       double grad_scale, double* contrib, double* g, int* state) {
  double b = (double)behave;
  double p = (double)prox;
  double denom = (norm == ORACLE_NORM_CONST_K) ? k : (double)steps;
  double w = 1.0 / (n_groups * (double)group_size * denom);
  double dsdl;
  double s = token_surrogate(l, b, p, A, eps_lo, eps_hi, c, &dsdl, state);
  *contrib = -w * s;
  *g = grad_scale * w * dsdl;
  return (!isfinite(l) || !isfinite(b) || !isfinite(p) || !isfinite(A)) ? ORACLE_ERR_NONFINITE : 0;
}

/* ---- the loss and dlogits for a range of token rows --------------------- */

/* For rows t in [row_begin, row_end) of logits (row t starts at element
 * t*ld, dtype as in load_elem), with per-token actions, behave log-probs and
 * proximal log-probs (prox == NULL means prox = behave), per-trajectory
 * advantages adv[n_traj] (double), the token->trajectory map tok_traj[T] and
 * step counts traj_steps[n_traj] from oracle_segments:
 *   l_t       = z[t, a_t] - logsumexp(z[t, :])
 *   s_t       = token_surrogate(l_t, b_t, p_t, A_i)
 *   w_i       = 1 / (n_groups * G * |tau_i|)  or  1 / (n_groups * G * k)
 *   contrib_t = -w_i * s_t                       (loss = sum_t contrib_t)
 *   g_t       = grad_scale * w_i * ds_t/dl_t
 *   dlogits[t, v] = g_t * (exp(z[t,v] - lse_t) - [v == a_t])
 * since d l_t / d z_v = [v == a_t] - softmax_v and the loss is -J.
 * Every per-row output is indexed by (t - row_begin); any may be NULL.
 * dlogits rows have stride V.  A row whose action is out of range contributes
 * 0, has logp 0 and a zero dlogits row.  If seg_flags has ORACLE_ERR_OFFSETS
 * set, every row is treated like that and the loss outputs become NaN (the
 * caller sums contrib).  Returns the OR of the error flags seen. */
int oracle_loss_rows(const void* logits, int dtype, int64_t V, int64_t ld, const int32_t* actions,
                     const float* behave, const float* prox, const double* adv,
                     const int32_t* tok_traj, const int32_t* traj_steps, int32_t seg_flags,
                     int32_t group_size, double n_groups, int norm, double k, double eps_lo,
                     double eps_hi, double c, double grad_scale, int64_t row_begin, int64_t row_end,
                     double* token_logp, double* token_contrib, double* token_g, int32_t* token_state,
                     double* dlogits) {
  int flags = seg_flags & ORACLE_ERR_OFFSETS;
  int64_t n_rows = row_end - row_begin;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : flags)
  for (int64_t q = 0; q < n_rows; ++q) {
    int64_t t = row_begin + q;
    int64_t a = actions[t];
    double* drow = dlogits ? dlogits + q * V : NULL;
    if ((seg_flags & ORACLE_ERR_OFFSETS) || a < 0 || a >= V) {
      if (!(seg_flags & ORACLE_ERR_OFFSETS)) flags |= ORACLE_ERR_ACTION;
      if (token_logp) token_logp[q] = 0.0;
      if (token_contrib) token_contrib[q] = (seg_flags & ORACLE_ERR_OFFSETS) ? NAN : 0.0;
      if (token_g) token_g[q] = 0.0;
      if (token_state) token_state[q] = 0;
      if (drow)
        for (int64_t v = 0; v < V; ++v) drow[v] = 0.0;
      continue;
    }
    int32_t i = tok_traj[t];
    int64_t base = t * ld;
    double lse = row_logsumexp(logits, dtype, base, V);
    double l = load_elem(logits, dtype, base + a) - lse;
    double contrib, g;
    int st;
    flags |= token_terms(l, behave[t], prox ? prox[t] : behave[t], adv[i], traj_steps[i], group_size, n_groups,
                         norm, k, eps_lo, eps_hi, c, grad_scale, &contrib, &g, &st);
    if (token_logp) token_logp[q] = l;
    if (token_contrib) token_contrib[q] = contrib;
    if (token_g) token_g[q] = g;
    if (token_state) token_state[q] = st;
    if (drow) {
      for (int64_t v = 0; v < V; ++v) {
        double pv = exp(load_elem(logits, dtype, base + v) - lse);
        drow[v] = g * (pv - (v == a ? 1.0 : 0.0));
      }
    }
  }
  return flags;
}

/* Eq. 1 for token rows [row_begin, row_end) given their new log-probs
 * logp[t - row_begin] (as an earlier oracle_loss_rows call on the same rows
 * returned them), for another normaliser or other loss parameters without
 * forming the log-softmax again.  Rows are handled exactly as in
 * oracle_loss_rows: a token whose action is outside [0, V), or every token
 * when seg_flags has ORACLE_ERR_OFFSETS, contributes 0 (NaN for bad offsets)
 * with g = 0 and state 0.  Outputs are indexed by t - row_begin; returns the
 * OR of the error flags seen. */
int oracle_loss_from_logp(const double* logp, int64_t V, const int32_t* actions, const float* behave,
                          const float* prox, const double* adv, const int32_t* tok_traj,
                          const int32_t* traj_steps, int32_t seg_flags, int32_t group_size, double n_groups,
                          int norm, double k, double eps_lo, double eps_hi, double c, double grad_scale,
                          int64_t row_begin, int64_t row_end, double* token_contrib, double* token_g,
                          int32_t* token_state) {
  int flags = seg_flags & ORACLE_ERR_OFFSETS;
  for (int64_t t = row_begin; t < row_end; ++t) {
    int64_t q = t - row_begin;
    int64_t a = actions[t];
    if ((seg_flags & ORACLE_ERR_OFFSETS) || a < 0 || a >= V) {
      if (!(seg_flags & ORACLE_ERR_OFFSETS)) flags |= ORACLE_ERR_ACTION;
      token_contrib[q] = (seg_flags & ORACLE_ERR_OFFSETS) ? NAN : 0.0;
      token_g[q] = 0.0;
      token_state[q] = 0;
      continue;
    }
    int32_t i = tok_traj[t];
    int st;
    flags |= token_terms(logp[q], behave[t], prox ? prox[t] : behave[t], adv[i], traj_steps[i], group_size,
                         n_groups, norm, k, eps_lo, eps_hi, c, grad_scale, &token_contrib[q], &token_g[q], &st);
    token_state[q] = st;
  }
  return flags;
}

/* Sums per-token contributions into per-trajectory losses and the total, in
 * token order (fp64).  traj_loss[n_traj] may be NULL. */
double oracle_reduce(const double* token_contrib, const int32_t* tok_traj, int64_t T, int32_t n_traj,
                     double* traj_loss) {
  double total = 0.0;
  if (traj_loss)
    for (int32_t i = 0; i < n_traj; ++i) traj_loss[i] = 0.0;
  for (int64_t t = 0; t < T; ++t) {
    total += token_contrib[t];
    if (traj_loss && tok_traj[t] >= 0) traj_loss[tok_traj[t]] += token_contrib[t];
  }
  return total;
}

/* ---- importance-ratio statistics ----------------------------------------- */

/* Diagnostics of the ratios that enter Eq. 1, over the tokens that enter the
 * loss (valid[t] != 0: an action inside the vocabulary, well-formed offsets):
 * r = pi/pi_prox = exp(l - p) (the clipped ratio) and rho = pi/pi_behave =
 * exp(l - b) (the importance weight), where l is the token's new log-prob,
 * b its behaviour log-prob and p its proximal log-prob (p = b when prox is
 * NULL, the coupled ratio).  The paper reports how often the eps clip engages
 * and how the coupled ratio compares with the decoupled one (Sec. 4.3,
 * Sec. 5); these are those quantities' building blocks:
 *   out[0..2] = sum, min, max of r       out[3..5] = sum, min, max of rho
 *   out[6]    = tokens with r outside [1 - eps_lo, 1 + eps_hi] (inclusive range)
 *   out[7]    = tokens counted.
 * With no token counted the sums are 0, the minima +inf and the maxima -inf.
 * Sums run in token order in fp64. */
void oracle_ratio_stats(int64_t n, const double* logp, const float* behave, const float* prox,
                        const int32_t* valid, double eps_lo, double eps_hi, double* out) {
  double sr = 0.0, rmin = INFINITY, rmax = -INFINITY;
  double sp = 0.0, pmin = INFINITY, pmax = -INFINITY;
  double outside = 0.0, count = 0.0;
  for (int64_t t = 0; t < n; ++t) {
    if (!valid[t]) continue;
    double b = (double)behave[t];
    double p = prox ? (double)prox[t] : b;
    double r = exp(logp[t] - p);
    double rho = exp(logp[t] - b);
    sr += r;
    if (r < rmin) rmin = r;
    if (r > rmax) rmax = r;
    sp += rho;
    if (rho < pmin) pmin = rho;
    if (rho > pmax) pmax = rho;
    if (r < 1.0 - eps_lo || r > 1.0 + eps_hi) outside += 1.0;
    count += 1.0;
  }
  out[0] = sr;
  out[1] = rmin;
  out[2] = rmax;
  out[3] = sp;
  out[4] = pmin;
  out[5] = pmax;
  out[6] = outside;
  out[7] = count;
}

/* ---- forward only: the action's log-prob and the policy entropy ---------- */

/* Per token row t in [row_begin, row_end): l_t = z[a_t] - lse(z) (the
 * log-softmax at the sampled action; what a proximal-policy recompute
 * produces, Table 5 "proximal logprobs recomputed") and the policy entropy
 * H_t = -sum_v p_v log p_v with p = softmax(z), the per-token quantity the
 * paper averages over the loss mask (Sec. 5, GRPO vs. RAFT++).  Written from
 * the definitions: log p_v = z_v - lse, p_v = exp(log p_v); a term whose p_v
 * underflows to zero contributes its limit, zero.  An action outside [0, V)
 * gives l_t = 0 and ORACLE_ERR_ACTION; the entropy does not depend on it.
 * Outputs are indexed by t - row_begin. */
int oracle_logp_entropy(const void* logits, int dtype, int64_t V, int64_t ld, const int32_t* actions,
                        int64_t row_begin, int64_t row_end, double* token_logp, double* token_entropy) {
  int flags = 0;
#pragma omp parallel for reduction(| : flags) schedule(static)
  for (int64_t t = row_begin; t < row_end; ++t) {
    const int64_t q = t - row_begin;
    const int64_t base = t * ld;
    const double lse = row_logsumexp(logits, dtype, base, V);
    double H = 0.0;
    for (int64_t v = 0; v < V; ++v) {
      const double logp = load_elem(logits, dtype, base + v) - lse;
      const double p = exp(logp);
      if (p > 0.0) H -= p * logp;
    }
    const int32_t a = actions[t];
    double l = 0.0;
    if (a < 0 || (int64_t)a >= V) flags |= ORACLE_ERR_ACTION;
    else l = load_elem(logits, dtype, base + a) - lse;
    if (!isfinite(lse)) flags |= ORACLE_ERR_NONFINITE;
    if (token_logp) token_logp[q] = l;
    if (token_entropy) token_entropy[q] = H;
  }
  return flags;
}

/* ---- one shard of a vocabulary split over devices ----------------------- */

/* For a vocabulary split into column ranges held by different devices, each
 * range (a shard: global columns [v_begin, v_begin + V_shard)) reduces its own
 * part of every row to m = max_v z_v, s = sum_v exp(z_v - m) over its columns,
 * and z_a = the action's logit when the action falls in the range (-inf
 * otherwise).  These are plain definitions; any split of the row merges back to
 * the row's log-sum-exp through lse = M + log sum_g s_g exp(m_g - M) with
 * M = max_g m_g, and to z_a as the largest of the shards' values (only the
 * owner's is finite).  `logits` holds the shard's columns only (row stride ld).
 * Outputs are indexed by t - row_begin. */
void oracle_vocab_shard_stats(const void* logits, int dtype, int64_t V_shard, int64_t ld, int64_t v_begin,
                              const int32_t* actions, int64_t row_begin, int64_t row_end, double* m_out,
                              double* s_out, double* za_out) {
#pragma omp parallel for schedule(static)
  for (int64_t t = row_begin; t < row_end; ++t) {
    const int64_t q = t - row_begin;
    const int64_t base = t * ld;
    double m = -INFINITY;
    for (int64_t v = 0; v < V_shard; ++v) {
      const double z = load_elem(logits, dtype, base + v);
      if (z > m || isnan(z)) m = z;
    }
    double s = 0.0;
    if (m != -INFINITY) /* a shard of -inf logits holds no mass */
      for (int64_t v = 0; v < V_shard; ++v) s += exp(load_elem(logits, dtype, base + v) - m);
    const int64_t a = (int64_t)actions[t] - v_begin;
    m_out[q] = m;
    s_out[q] = s;
    za_out[q] = (a >= 0 && a < V_shard) ? load_elem(logits, dtype, base + a) : -INFINITY;
  }
}

/* Threads the row loop runs on (for reporting the oracle's timing). */
int oracle_threads(void) { return omp_get_max_threads(); }

/* Sets the OpenMP thread count of later calls (results do not depend on it). */
void oracle_set_threads(int n) { omp_set_num_threads(n > 0 ? n : 1); }
