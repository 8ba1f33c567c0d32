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

// Reduces the per-token loss contributions: per trajectory, then over
// trajectories, both in a fixed order; writes loss_out and the aux outputs.
hipError_t launch_reduce(int64_t T, int32_t n_traj, char* ws, const LossWs& L, double* loss_out,
                         const grpo_aux* aux, hipStream_t s);

}  // namespace grpo
