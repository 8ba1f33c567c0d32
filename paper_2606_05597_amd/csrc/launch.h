// Launchers shared by the logits path and the fused LM-head path.
#pragma once

#include <hip/hip_runtime.h>

#include "grpo.h"
#include "device.h"
#include "host.h"

namespace grpo {

// Validates the offsets on the device and writes the per-trajectory tables
// (first token of each trajectory, normaliser weight w_i) and, per token, its
// trajectory's advantage and weight; resets the workspace header (flags, counters).  Also writes
// aux->traj_tok_off, aux->tok_traj and aux->gather_idx (t*ld + a_t) if set.
hipError_t launch_segments(const grpo_segments* seg, int64_t T, int64_t ld, const int32_t* actions,
                           const float* adv, const grpo_loss_params* p, char* ws, const LossWs& L,
                           const grpo_aux* aux, hipStream_t s);

// The token-epilogue arguments of a loss call (device.h TokenArgs).
TokenArgs make_token_args(int64_t V, const int32_t* actions, const float* behave, const float* prox,
                          const float* adv, const grpo_loss_params* p, char* ws, const LossWs& L,
                          const grpo_aux* aux);

// One workgroup per row: each row of logits [T, ld] (columns [0, V), global ids from v_begin) reduced to its
// grpo_vocab_stats record; NONFINITE is OR-ed into *flags (nullable) for a NaN or +inf log-sum-exp.
hipError_t launch_vocab_records(const void* logits, grpo_dtype dt, int64_t T, int64_t V, int64_t ld,
                                int64_t v_begin, const int32_t* actions, grpo_vocab_stats* stats, int32_t* flags,
                                hipStream_t s);

// One workgroup per row: every shard's records merged, the token epilogue, then the row's columns [0, V)
// of dlogits (global ids from v_begin; dlogits nullable = forward only).
hipError_t launch_shard_rows(const void* logits, void* dlogits, grpo_dtype dt, int64_t T, int64_t V, int64_t ld,
                             int64_t v_begin, const grpo_vocab_stats* stats, int n_shards, const TokenArgs& tok,
                             hipStream_t s);

// Reduces the per-token loss contributions: per trajectory, then over
// trajectories, both in a fixed order; writes loss_out and the aux outputs.
hipError_t launch_reduce(int64_t T, int32_t n_traj, char* ws, const LossWs& L, double* loss_out,
                         const grpo_aux* aux, hipStream_t s);

}  // namespace grpo
