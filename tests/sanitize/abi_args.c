/*
 * Drives the host side of libgrpo's C ABI (include/grpo.h) under AddressSanitizer and UndefinedBehaviorSanitizer
 * (the library's host code built with -Xarch_host -fsanitize=...): every entry point with each kind of invalid
 * argument, which the library must reject on the host before anything is launched, and every workspace query at
 * ordinary, empty and extreme sizes (the queries must not overflow, and must return 0 for sizes their entry points
 * refuse).  No GPU is needed: nothing here gets past argument validation.  Test infrastructure only.
 */
#include <stdint.h>
#include <stdio.h>

#include "grpo.h"

static int failures = 0;
#define EXPECT(call, want)                                                                   \
  do {                                                                                       \
    const long long got_ = (long long)(call);                                                \
    if (got_ != (long long)(want)) {                                                         \
      fprintf(stderr, "line %d: %s returned %lld, expected %lld\n", __LINE__, #call, got_, \
              (long long)(want));                                                            \
      ++failures;                                                                            \
    }                                                                                        \
  } while (0)

#define D ((void*)0x100000) /* a dummy 256-byte-aligned device address: never dereferenced on the host */
#define DI ((int32_t*)D)
#define DF ((float*)D)
#define DD ((double*)D)

static grpo_segments seg_of(int32_t n_traj, int32_t G, int32_t n_steps) {
  grpo_segments s = {n_traj, G, n_steps, DI, DI};
  return s;
}
static grpo_loss_params params(void) {
  grpo_loss_params p = {GRPO_NORM_CONST_K, 10.f, 0.2f, 0.2f, 3.f, 1.f, 0.0};
  return p;
}

int main(void) {
  const int64_t BIG = INT64_MAX, HUGE_ = (int64_t)1 << 40;
  grpo_segments sg = seg_of(4, 4, 4);
  grpo_loss_params p = params();

  /* status strings */
  for (int c = -8; c <= 1; ++c)
    if (!grpo_status_str(c)) ++failures;

  /* advantages */
  EXPECT(grpo_advantages(NULL, 8, 4, 1, 0.f, DF, NULL), GRPO_ERR_ARG);
  EXPECT(grpo_advantages(DF, 8, 3, 1, 0.f, DF, NULL), GRPO_ERR_SHAPE);
  EXPECT(grpo_advantages(DF, 8, 4, 2, 0.f, DF, NULL), GRPO_ERR_ARG);
  EXPECT(grpo_advantages(DF, 8, 4, 1, -1.f, DF, NULL), GRPO_ERR_ARG);
  EXPECT(grpo_advantages(DF, 0, 4, 1, 0.f, DF, NULL), GRPO_ERR_SHAPE);
  EXPECT(grpo_advantages_ex(DF, 8, 4, 7, 1, 0.f, DF, NULL, NULL, NULL), GRPO_ERR_ARG);
  EXPECT(grpo_advantages_ex(DF, 8, 0, 0, 1, 0.f, DF, NULL, NULL, NULL), GRPO_ERR_SHAPE);

  /* the logits path and its allocation-free form */
  EXPECT(grpo_loss_fwd_bwd(D, GRPO_BF16, 8, 64, 64, NULL, DF, NULL, DF, &sg, &p, DD, D, NULL, D, 1 << 20, NULL),
         GRPO_ERR_ARG);
  EXPECT(grpo_loss_fwd_bwd(D, GRPO_BF16, 8, 64, 63, DI, DF, NULL, DF, &sg, &p, DD, D, NULL, D, 1 << 20, NULL),
         GRPO_ERR_SHAPE);
  EXPECT(grpo_loss_fwd_bwd(D, GRPO_BF16, BIG, 64, 64, DI, DF, NULL, DF, &sg, &p, DD, D, NULL, D, 1 << 20, NULL),
         GRPO_ERR_SHAPE);
  EXPECT(grpo_loss_fwd_bwd(D, GRPO_BF16, 8, BIG, BIG, DI, DF, NULL, DF, &sg, &p, DD, D, NULL, D, 1 << 20, NULL),
         GRPO_ERR_SHAPE);
  EXPECT(grpo_loss_fwd_bwd(D, (grpo_dtype)9, 8, 64, 64, DI, DF, NULL, DF, &sg, &p, DD, D, NULL, D, 1 << 20, NULL),
         GRPO_ERR_DTYPE);
  EXPECT(grpo_loss_fwd_bwd(D, GRPO_BF16, 8, 64, 64, DI, DF, NULL, DF, &sg, &p, DD, D, NULL, NULL, 0, NULL),
         GRPO_ERR_WORKSPACE);
  EXPECT(grpo_loss_fwd_bwd((char*)D + 1, GRPO_BF16, 8, 64, 64, DI, DF, NULL, DF, &sg, &p, DD, D, NULL, D, 1 << 20,
                           NULL),
         GRPO_ERR_ALIGN);
  EXPECT(grpo_loss_fwd_bwd(D, GRPO_BF16, 8, 64, 64, DI, DF, NULL, DF, NULL, &p, DD, D, NULL, D, 1 << 20, NULL),
         GRPO_ERR_ARG);
  {
    grpo_segments bad = seg_of(6, 4, 6);
    EXPECT(grpo_loss_fwd_bwd(D, GRPO_BF16, 8, 64, 64, DI, DF, NULL, DF, &bad, &p, DD, D, NULL, D, 1 << 20, NULL),
           GRPO_ERR_SHAPE);
    grpo_segments neg = seg_of(-4, 4, 4);
    EXPECT(grpo_loss_fwd_bwd(D, GRPO_BF16, 8, 64, 64, DI, DF, NULL, DF, &neg, &p, DD, D, NULL, D, 1 << 20, NULL),
           GRPO_ERR_SHAPE);
    grpo_loss_params q = params();
    q.k = 0.f;
    EXPECT(grpo_loss_fwd_bwd(D, GRPO_BF16, 8, 64, 64, DI, DF, NULL, DF, &sg, &q, DD, D, NULL, D, 1 << 20, NULL),
           GRPO_ERR_ARG);
    q = params();
    q.dual_clip_c = 0.5f;
    EXPECT(grpo_loss_fwd_bwd(D, GRPO_BF16, 8, 64, 64, DI, DF, NULL, DF, &sg, &q, DD, D, NULL, D, 1 << 20, NULL),
           GRPO_ERR_ARG);
    q = params();
    q.n_groups_total = -1.0;
    EXPECT(grpo_loss_fwd_bwd(D, GRPO_BF16, 8, 64, 64, DI, DF, NULL, DF, &sg, &q, DD, D, NULL, D, 1 << 20, NULL),
           GRPO_ERR_ARG);
    q = params();
    q.norm = 5;
    EXPECT(grpo_loss_fwd_bwd(D, GRPO_BF16, 8, 64, 64, DI, DF, NULL, DF, &sg, &q, DD, D, NULL, D, 1 << 20, NULL),
           GRPO_ERR_ARG);
  }
  EXPECT(grpo_loss_fwd_bwd_noalloc(D, GRPO_BF16, 8, 64, 63, DI, DF, NULL, DF, &sg, &p, DD, D, NULL, NULL),
         GRPO_ERR_SHAPE);
  EXPECT(grpo_loss_fwd_bwd_noalloc(D, GRPO_BF16, (int64_t)1 << 24, 8, 8, DI, DF, NULL, DF, &sg, &p, DD, D, NULL,
                                   NULL),
         GRPO_ERR_WORKSPACE);

  /* fused LM head: both schedules */
  EXPECT(fused_lmhead_grpo(D, D, 8, 64, 512, 300, DI, DF, NULL, DF, &sg, &p, DD, D, DF, 0, NULL, D, 1 << 30, NULL),
         GRPO_ERR_SHAPE);
  EXPECT(fused_lmhead_grpo(D, D, 8, 65, 512, 256, DI, DF, NULL, DF, &sg, &p, DD, D, DF, 0, NULL, D, 1 << 30, NULL),
         GRPO_ERR_SHAPE);
  EXPECT(fused_lmhead_grpo(D, D, 8, 64, BIG, 256, DI, DF, NULL, DF, &sg, &p, DD, D, DF, 0, NULL, D, 1 << 30, NULL),
         GRPO_ERR_SHAPE);
  EXPECT(fused_lmhead_grpo(D, D, BIG, 64, 512, 256, DI, DF, NULL, DF, &sg, &p, DD, D, DF, 0, NULL, D, 1 << 30, NULL),
         GRPO_ERR_SHAPE);
  EXPECT(fused_lmhead_grpo(D, NULL, 8, 64, 512, 256, DI, DF, NULL, DF, &sg, &p, DD, D, DF, 0, NULL, D, 1 << 30, NULL),
         GRPO_ERR_ARG);
  EXPECT(fused_lmhead_grpo(D, D, 8, 64, 512, 256, DI, DF, NULL, DF, &sg, &p, DD, D, DF, 0, NULL, D, 16, NULL),
         GRPO_ERR_WORKSPACE);
  EXPECT(fused_lmhead_grpo_blocked(D, D, 8, 64, 512, 300, DI, DF, NULL, DF, &sg, &p, DD, D, DF, 0, NULL, D, 1 << 30,
                                   NULL, NULL),
         GRPO_ERR_SHAPE);
  EXPECT(fused_lmhead_grpo_blocked(D, D, 8, 64, 512, 256, DI, DF, NULL, DF, &sg, &p, DD, D, DF, 0, NULL, D, 16, NULL,
                                   NULL),
         GRPO_ERR_WORKSPACE);
  EXPECT(fused_lmhead_grpo_blocked(D, D, 8, HUGE_, HUGE_, 256, DI, DF, NULL, DF, &sg, &p, DD, D, DF, 0, NULL, D,
                                   1 << 30, NULL, NULL),
         GRPO_ERR_SHAPE);

  /* forward only */
  EXPECT(grpo_token_logp(D, GRPO_BF16, 8, 64, 63, DI, DF, DF, NULL, NULL), GRPO_ERR_SHAPE);
  EXPECT(grpo_token_logp(NULL, GRPO_BF16, 8, 64, 64, DI, DF, DF, NULL, NULL), GRPO_ERR_ARG);
  EXPECT(grpo_token_logp(D, GRPO_BF16, BIG, BIG, BIG, DI, DF, DF, NULL, NULL), GRPO_ERR_SHAPE);
  EXPECT(fused_lmhead_token_logp(D, D, 8, 64, 512, DI, DF, DF, NULL, D, 16, NULL), GRPO_ERR_WORKSPACE);
  EXPECT(fused_lmhead_token_logp(D, D, 8, HUGE_, HUGE_, DI, DF, DF, NULL, D, 1 << 30, NULL), GRPO_ERR_SHAPE);

  /* vocabulary shards */
  grpo_vocab_stats* ST = (grpo_vocab_stats*)D;
  EXPECT(grpo_vocab_shard_stats(D, GRPO_BF16, 8, 64, 64, -1, DI, ST, NULL, NULL), GRPO_ERR_SHAPE);
  EXPECT(grpo_vocab_shard_stats(D, GRPO_BF16, 8, 64, 64, BIG, DI, ST, NULL, NULL), GRPO_ERR_SHAPE);
  EXPECT(grpo_loss_fwd_bwd_vocab_shard(D, GRPO_BF16, 8, 64, 64, 0, 128, ST, 0, DI, DF, NULL, DF, &sg, &p, DD, D, NULL,
                                       D, 1 << 20, NULL),
         GRPO_ERR_SHAPE);
  EXPECT(grpo_loss_fwd_bwd_vocab_shard(D, GRPO_BF16, 8, 64, 64, 100, 128, ST, 2, DI, DF, NULL, DF, &sg, &p, DD, D,
                                       NULL, D, 1 << 20, NULL),
         GRPO_ERR_SHAPE);
  EXPECT(grpo_loss_fwd_bwd_vocab_shard(D, GRPO_BF16, 8, 64, 64, BIG, BIG, ST, 2, DI, DF, NULL, DF, &sg, &p, DD, D,
                                       NULL, D, 1 << 20, NULL),
         GRPO_ERR_SHAPE);
  EXPECT(fused_lmhead_vocab_shard_stats(D, D, 8, 64, 512, BIG, DI, ST, NULL, D, 1 << 30, NULL), GRPO_ERR_SHAPE);
  EXPECT(fused_lmhead_vocab_shard_stats(D, D, 8, 64, 512, 0, DI, ST, NULL, D, 16, NULL), GRPO_ERR_WORKSPACE);
  EXPECT(fused_lmhead_grpo_vocab_shard(D, D, 8, 64, 512, 0, 1024, 256, ST, 0, DI, DF, NULL, DF, &sg, &p, DD, DF, DF,
                                       0, NULL, NULL, D, 1 << 30, NULL),
         GRPO_ERR_SHAPE);
  EXPECT(fused_lmhead_grpo_vocab_shard(D, D, 8, 64, 512, BIG, BIG, 256, ST, 2, DI, DF, NULL, DF, &sg, &p, DD, DF, DF,
                                       0, NULL, NULL, D, 1 << 30, NULL),
         GRPO_ERR_SHAPE);

  /* workspace queries: ordinary sizes are positive; empty batches still need their tables; sizes the entry points
     refuse, or that would overflow, give 0 */
  if (grpo_loss_workspace_bytes(120000, 128) == 0) ++failures;
  if (grpo_loss_workspace_bytes(0, 4) == 0) ++failures;
  EXPECT(grpo_loss_workspace_bytes(-1, 4), 0);
  EXPECT(grpo_loss_workspace_bytes(BIG, 4), 0);
  EXPECT(grpo_loss_workspace_bytes(8, 0), 0);
  if (fused_lmhead_workspace_bytes(65536, 3584, 151936, 8192, 64) == 0) ++failures;
  EXPECT(fused_lmhead_workspace_bytes(BIG, BIG, BIG, 8192, 64), 0);
  EXPECT(fused_lmhead_workspace_bytes(65536, HUGE_, HUGE_, 8192, 64), 0);
  if (fused_lmhead_blocked_workspace_bytes(65536, 3584, 151936, 8192, 64) == 0) ++failures;
  EXPECT(fused_lmhead_blocked_workspace_bytes(BIG, BIG, BIG, 8192, 64), 0);
  EXPECT(fused_lmhead_blocked_workspace_bytes(65536, HUGE_, HUGE_, 8192, 64), 0);
  if (fused_lmhead_token_logp_workspace_bytes(65536, 3584, 151936) == 0) ++failures;
  EXPECT(fused_lmhead_token_logp_workspace_bytes(BIG, BIG, BIG), 0);
  EXPECT(fused_lmhead_token_logp_workspace_bytes(65536, HUGE_, HUGE_), 0);
  if (fused_lmhead_vocab_shard_stats_workspace_bytes(65536, 3584, 18992) == 0) ++failures;
  EXPECT(fused_lmhead_vocab_shard_stats_workspace_bytes(BIG, BIG, BIG), 0);
  if (fused_lmhead_vocab_shard_logits_bytes(65536, 18992) == 0) ++failures;
  EXPECT(fused_lmhead_vocab_shard_logits_bytes(BIG, BIG), 0);

  if (failures) {
    fprintf(stderr, "%d checks failed\n", failures);
    return 1;
  }
  printf("abi argument checks ok\n");
  return 0;
}
