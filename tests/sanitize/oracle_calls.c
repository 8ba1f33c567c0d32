/*
 * Runs every function of the fp64 oracle (oracle/grpo_oracle.c) on small batches, including its edge cases (a
 * batch with no tokens, steps with no tokens, actions outside the vocabulary, malformed offsets, a zero-variance
 * group, bf16 / fp32 / fp64 rows, rows of -inf, a one-column vocabulary), for a build with AddressSanitizer and
 * UndefinedBehaviorSanitizer: any out-of-bounds access or undefined operation aborts with a report.  It checks a
 * few results too, so a sanitizer build that computes nonsense fails.  Test infrastructure only.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int oracle_segments(int64_t T, int32_t n_steps, const int32_t* sto, int32_t n_traj, const int32_t* tso,
                    int32_t* traj_tok_off, int32_t* tok_traj, int32_t* traj_steps);
void oracle_advantages(const float* rewards, int32_t n_traj, int32_t G, int32_t ddof, double std_eps, double* adv);
void oracle_advantages_success_filter(const float* rewards, int32_t n_traj, double* adv);
int32_t oracle_mixed_groups(const float* rewards, int32_t n_traj, int32_t G, int32_t* mixed);
int oracle_loss_rows(const void* logits, int dtype, int64_t V, int64_t ld, const int32_t* actions, const float* behave,
                     const float* prox, const double* adv, const int32_t* tok_traj, const int32_t* traj_steps,
                     int32_t seg_flags, int32_t group_size, double n_groups, int norm, double k, double eps_lo,
                     double eps_hi, double c, double grad_scale, int64_t row_begin, int64_t row_end,
                     double* token_logp, double* token_contrib, double* token_g, int32_t* token_state,
                     double* dlogits);
int oracle_loss_from_logp(const double* logp, int64_t V, const int32_t* actions, const float* behave,
                          const float* prox, const double* adv, const int32_t* tok_traj, const int32_t* traj_steps,
                          int32_t seg_flags, int32_t group_size, double n_groups, int norm, double k, double eps_lo,
                          double eps_hi, double c, double grad_scale, int64_t row_begin, int64_t row_end,
                          double* token_contrib, double* token_g, int32_t* token_state);
double oracle_reduce(const double* token_contrib, const int32_t* tok_traj, int64_t T, int32_t n_traj,
                     double* traj_loss);
void oracle_ratio_stats(int64_t n, const double* logp, const float* behave, const float* prox, const int32_t* valid,
                        double eps_lo, double eps_hi, double* out);
int oracle_logp_entropy(const void* logits, int dtype, int64_t V, int64_t ld, const int32_t* actions,
                        int64_t row_begin, int64_t row_end, double* token_logp, double* token_entropy);
void oracle_vocab_shard_stats(const void* logits, int dtype, int64_t V_shard, int64_t ld, int64_t v_begin,
                              const int32_t* actions, int64_t row_begin, int64_t row_end, double* m_out,
                              double* s_out, double* za_out);
void oracle_set_threads(int n);

static int failures = 0;
#define CHECK(cond)                                                  \
  do {                                                               \
    if (!(cond)) {                                                   \
      fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #cond); \
      ++failures;                                                    \
    }                                                                \
  } while (0)

static uint32_t rng_state = 12345u;
static double urand(void) { /* xorshift32 in [0, 1) */
  rng_state ^= rng_state << 13;
  rng_state ^= rng_state >> 17;
  rng_state ^= rng_state << 5;
  return (double)rng_state / 4294967296.0;
}

/* one batch through every per-row function; T tokens, V columns, row stride ld, dtype 0/1/2 */
static void run_batch(int64_t T, int64_t V, int64_t ld, int dtype, int n_traj, int G, int bad_actions,
                      int bad_offsets) {
  const int n_steps = 2 * n_traj;
  int32_t* sto = calloc((size_t)n_steps + 1, sizeof *sto);
  int32_t* tso = calloc((size_t)n_traj + 1, sizeof *tso);
  for (int j = 0; j <= n_steps; ++j) sto[j] = (int32_t)((T * j) / n_steps); /* some steps may be empty */
  for (int i = 0; i <= n_traj; ++i) tso[i] = 2 * i;
  if (bad_offsets) sto[n_steps] += 1;
  int32_t* tto = malloc(((size_t)n_traj + 1) * sizeof *tto);
  int32_t* tt = malloc(((size_t)T + 1) * sizeof *tt);
  int32_t* ts = malloc((size_t)n_traj * sizeof *ts);
  const int sf = oracle_segments(T, n_steps, sto, n_traj, tso, tto, tt, ts);
  CHECK((sf != 0) == (bad_offsets != 0));

  const size_t esz = dtype == 0 ? 4 : (dtype == 1 ? 2 : 8);
  unsigned char* logits = malloc((size_t)(T > 0 ? T : 1) * (size_t)ld * esz);
  for (int64_t t = 0; t < T; ++t)
    for (int64_t v = 0; v < ld; ++v) {
      const double z = (v < V) ? 4.0 * urand() - 2.0 : 1e30; /* padding past V must never be read as a logit */
      const int64_t q = t * ld + v;
      if (dtype == 0) ((float*)logits)[q] = (float)z;
      else if (dtype == 2) ((double*)logits)[q] = z;
      else {
        float f = (float)z;
        uint32_t b;
        memcpy(&b, &f, sizeof b);
        ((uint16_t*)logits)[q] = (uint16_t)(b >> 16);
      }
    }
  int32_t* actions = malloc(((size_t)T + 1) * sizeof *actions);
  float* behave = malloc(((size_t)T + 1) * sizeof *behave);
  float* prox = malloc(((size_t)T + 1) * sizeof *prox);
  for (int64_t t = 0; t < T; ++t) {
    actions[t] = (int32_t)(urand() * (double)V);
    behave[t] = (float)(-log((double)V) + 0.3 * (urand() - 0.5));
    prox[t] = behave[t] + (float)(0.1 * (urand() - 0.5));
  }
  if (bad_actions && T > 2) {
    actions[0] = (int32_t)V;
    actions[T - 1] = -3;
  }
  float* rewards = malloc((size_t)n_traj * sizeof *rewards);
  for (int i = 0; i < n_traj; ++i) rewards[i] = (i % 3 == 0) ? 1.f : 0.f;
  if (n_traj >= 2 * G)
    for (int i = G; i < 2 * G; ++i) rewards[i] = 1.f; /* a zero-variance group */
  double* adv = malloc((size_t)n_traj * sizeof *adv);
  oracle_advantages(rewards, n_traj, G, 1, 0.0, adv);
  oracle_advantages(rewards, n_traj, G, 0, 1e-6, adv);
  int32_t* mixed = malloc((size_t)(n_traj / G) * sizeof *mixed);
  CHECK(oracle_mixed_groups(rewards, n_traj, G, mixed) <= n_traj / G);
  oracle_advantages_success_filter(rewards, n_traj, adv);
  oracle_advantages(rewards, n_traj, G, 1, 0.0, adv);

  const int64_t n = T;
  double* logp = malloc(((size_t)n + 1) * sizeof *logp);
  double* contrib = malloc(((size_t)n + 1) * sizeof *contrib);
  double* g = malloc(((size_t)n + 1) * sizeof *g);
  int32_t* st = malloc(((size_t)n + 1) * sizeof *st);
  double* dl = malloc(((size_t)n + 1) * (size_t)V * sizeof *dl);
  double* traj = malloc((size_t)n_traj * sizeof *traj);
  for (int norm = 0; norm < 2; ++norm)
    for (int dec = 0; dec < 2; ++dec) {
      const double c = dec ? 3.0 : 0.0;
      oracle_loss_rows(logits, dtype, V, ld, actions, behave, dec ? prox : NULL, adv, tt, ts, sf, G,
                       (double)(n_traj / G), norm, 10.0, 0.2, 0.28, c, 1.0, 0, T, logp, contrib, g, st, dl);
      const double total = oracle_reduce(contrib, tt, T, n_traj, traj);
      if (!bad_offsets) {
        CHECK(isfinite(total));
        for (int64_t t = 0; t < T; ++t) { /* each dlogits row sums to 0 */
          double rs = 0.0;
          for (int64_t v = 0; v < V; ++v) rs += dl[t * V + v];
          CHECK(fabs(rs) <= 1e-12 + 1e-9 * fabs(g[t]));
        }
      } else {
        CHECK(isnan(total) || T == 0);
      }
      double* c2 = malloc(((size_t)n + 1) * sizeof *c2);
      double* g2 = malloc(((size_t)n + 1) * sizeof *g2);
      int32_t* s2 = malloc(((size_t)n + 1) * sizeof *s2);
      oracle_loss_from_logp(logp, V, actions, behave, dec ? prox : NULL, adv, tt, ts, sf, G, (double)(n_traj / G),
                            norm, 10.0, 0.2, 0.28, c, 1.0, 0, T, c2, g2, s2);
      for (int64_t t = 0; t < T; ++t) CHECK(bad_offsets ? isnan(c2[t]) : (c2[t] == contrib[t] && g2[t] == g[t]));
      free(c2);
      free(g2);
      free(s2);
    }
  /* a sub-range of rows, forward only */
  if (T > 3)
    oracle_loss_rows(logits, dtype, V, ld, actions, behave, NULL, adv, tt, ts, sf, G, 0.5, 1, 10.0, 0.2, 0.2, 3.0,
                     2.0, 1, T - 1, logp, contrib, g, st, NULL);
  int32_t* valid = malloc(((size_t)n + 1) * sizeof *valid);
  for (int64_t t = 0; t < T; ++t) valid[t] = !bad_offsets && actions[t] >= 0 && actions[t] < V;
  double rstats[8];
  oracle_ratio_stats(T, logp, behave, prox, valid, 0.2, 0.2, rstats);
  oracle_ratio_stats(T, logp, behave, NULL, valid, 0.0, 0.0, rstats);
  double* ent = malloc(((size_t)n + 1) * sizeof *ent);
  oracle_logp_entropy(logits, dtype, V, ld, actions, 0, T, logp, ent);
  for (int64_t t = 0; t < T; ++t) CHECK(ent[t] >= -1e-12 && ent[t] <= log((double)V) + 1e-9);
  double *m = malloc(((size_t)n + 1) * sizeof *m), *s = malloc(((size_t)n + 1) * sizeof *s),
         *za = malloc(((size_t)n + 1) * sizeof *za);
  const int64_t half = V / 2 > 0 ? V / 2 : 1;
  oracle_vocab_shard_stats(logits, dtype, half, ld, 0, actions, 0, T, m, s, za);
  if (V > half)
    oracle_vocab_shard_stats((const unsigned char*)logits + (size_t)half * esz, dtype, V - half, ld, half, actions, 0,
                             T, m, s, za);
  free(m), free(s), free(za), free(ent), free(valid), free(traj), free(dl), free(st), free(g), free(contrib);
  free(logp), free(mixed), free(adv), free(rewards), free(prox), free(behave), free(actions), free(logits);
  free(ts), free(tt), free(tto), free(tso), free(sto);
}

int main(void) {
  oracle_set_threads(4);
  run_batch(40, 33, 33, 1, 8, 4, 0, 0);  /* bf16, odd V */
  run_batch(40, 64, 72, 0, 8, 4, 1, 0);  /* fp32, padded rows, actions outside the vocabulary */
  run_batch(25, 17, 17, 2, 4, 2, 0, 0);  /* fp64 */
  run_batch(12, 1, 1, 0, 4, 4, 0, 0);    /* one-column vocabulary */
  run_batch(30, 16, 16, 1, 6, 3, 0, 1);  /* malformed offsets */
  run_batch(0, 16, 16, 1, 4, 2, 0, 0);   /* no tokens at all */
  run_batch(5, 8, 8, 0, 8, 4, 0, 0);     /* more steps than tokens: empty steps */
  { /* a row of -inf in a shard */
    float row[4] = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};
    int32_t a = 2;
    double m, s, za;
    oracle_vocab_shard_stats(row, 0, 4, 4, 0, &a, 0, 1, &m, &s, &za);
    CHECK(m == -INFINITY && s == 0.0);
  }
  if (failures) {
    fprintf(stderr, "%d checks failed\n", failures);
    return 1;
  }
  printf("oracle calls ok\n");
  return 0;
}
