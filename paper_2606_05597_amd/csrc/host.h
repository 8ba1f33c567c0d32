// Host-side helpers shared by the libgrpo entry points.
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>
#include <stddef.h>
#include <stdint.h>

#include "device.h"
#include "grpo.h"

namespace grpo {

constexpr size_t kAlign = 256;

inline size_t align_up(size_t x) { return (x + kAlign - 1) & ~(kAlign - 1); }

// Workspace of the loss: per-trajectory and per-token scratch.
struct LossWs {
  size_t hdr, traj_tok_off, w, traj_loss, traj_rstats, tok_adv, tok_w, contrib, state, tok_ratio, records, total;
};

inline LossWs loss_ws_layout(int64_t T, int32_t n_traj) {
  LossWs l;
  size_t o = 0;
  l.hdr = o;          o = align_up(o + sizeof(WsHeader));
  l.traj_tok_off = o; o = align_up(o + sizeof(int32_t) * ((size_t)n_traj + 1));
  l.w = o;            o = align_up(o + sizeof(double) * (size_t)n_traj);
  l.traj_loss = o;    o = align_up(o + sizeof(double) * (size_t)n_traj);
  l.traj_rstats = o;  o = align_up(o + 6 * sizeof(double) * (size_t)n_traj);
  l.tok_adv = o;      o = align_up(o + sizeof(float) * (size_t)(T > 0 ? T : 0));
  l.tok_w = o;        o = align_up(o + sizeof(double) * (size_t)(T > 0 ? T : 0));
  l.contrib = o;      o = align_up(o + sizeof(double) * (size_t)(T > 0 ? T : 0));
  l.state = o;        o = align_up(o + sizeof(int8_t) * (size_t)(T > 0 ? T : 0));
  l.tok_ratio = o;    o = align_up(o + 2 * sizeof(double) * (size_t)(T > 0 ? T : 0));
  l.records = o;      o = align_up(o + sizeof(grpo_vocab_stats) * (size_t)(T > 0 ? T : 0));  // two-pass rows
  l.total = o;
  return l;
}

// Checks shared by both loss entry points; returns GRPO_OK or the error.
inline int check_loss_common(int64_t T, const int32_t* actions, const float* behave, const float* adv,
                             const grpo_segments* seg, const grpo_loss_params* p, const double* loss_out) {
  if (!actions && T > 0) return GRPO_ERR_ARG;
  if (!behave && T > 0) return GRPO_ERR_ARG;
  if (!adv || !seg || !p || !loss_out) return GRPO_ERR_ARG;
  if (!seg->step_tok_off || !seg->traj_step_off) return GRPO_ERR_ARG;
  if (T < 0 || T >= ((int64_t)1 << 31)) return GRPO_ERR_SHAPE;
  if (seg->n_traj < 1 || seg->group_size < 1 || seg->n_traj % seg->group_size != 0) return GRPO_ERR_SHAPE;
  if (seg->n_steps < seg->n_traj) return GRPO_ERR_SHAPE;
  if (p->norm != GRPO_NORM_TRAJ_STEPS && p->norm != GRPO_NORM_CONST_K) return GRPO_ERR_ARG;
  if (p->norm == GRPO_NORM_CONST_K && !(p->k > 0.f && isfinite(p->k))) return GRPO_ERR_ARG;
  if (!(p->eps_low >= 0.f && p->eps_low < 1.f)) return GRPO_ERR_ARG;
  if (!(p->eps_high >= 0.f) || isnan(p->eps_high)) return GRPO_ERR_ARG;
  if (!(p->dual_clip_c == 0.f || (p->dual_clip_c > 1.f && isfinite(p->dual_clip_c)))) return GRPO_ERR_ARG;
  if (!isfinite(p->grad_scale)) return GRPO_ERR_ARG;
  if (!(p->n_groups_total >= 0.0) || !isfinite(p->n_groups_total)) return GRPO_ERR_ARG;
  return GRPO_OK;
}

inline double n_groups_of(const grpo_segments* seg, const grpo_loss_params* p) {
  return p->n_groups_total > 0.0 ? p->n_groups_total : (double)(seg->n_traj / seg->group_size);
}

inline bool aligned(const void* ptr, size_t a) { return ((uintptr_t)ptr % a) == 0; }

// Compute units of the device the stream belongs to (which need not be the current device), or 0 if the
// runtime cannot say.
inline int stream_cu_count(hipStream_t s) {
  hipDevice_t dev = 0;
  int n_cu = 0;
  if (hipStreamGetDevice(s, &dev) != hipSuccess ||
      hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n_cu < 1)
    return 0;
  return n_cu;
}

}  // namespace grpo
