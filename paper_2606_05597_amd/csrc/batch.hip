// Batch bookkeeping kernels: segment validation, group advantages, and the
// deterministic loss reduction.  All are small next to the row pass.
#include <hip/hip_runtime.h>
#include <math.h>

#include "device.h"
#include "launch.h"

namespace grpo {

// ---- segments ----------------------------------------------------------------
// One workgroup.  Checks the CSR offsets of Eq. 1's trajectory/step/token
// sums, writes traj_tok_off[i] = step_tok_off[traj_step_off[i]] and the
// per-trajectory weight w_i = 1/(n_groups * G * |tau_i| or k).
struct SegArgs {
  const int32_t* sto;  // [n_steps+1]
  const int32_t* tso;  // [n_traj+1]
  int32_t n_steps, n_traj, G, norm;
  int64_t T;
  double n_groups, k;
  WsHeader* hdr;
  int32_t* traj_tok_off;  // ws [n_traj+1]
  double* w;              // ws [n_traj]
  int32_t* aux_traj_tok_off;
};

__global__ __launch_bounds__(256) void k_segments(const SegArgs a) {
  const int tid = threadIdx.x;
  int bad = 0;
  for (int j = tid; j < a.n_steps; j += 256)
    if (a.sto[j + 1] < a.sto[j]) bad = 1;
  for (int i = tid; i < a.n_traj; i += 256)
    if (a.tso[i + 1] <= a.tso[i]) bad = 1;
  if (tid == 0) {
    if (a.sto[0] != 0 || (int64_t)a.sto[a.n_steps] != a.T) bad = 1;
    if (a.tso[0] != 0 || a.tso[a.n_traj] != a.n_steps) bad = 1;
  }
  bad = __syncthreads_or(bad);
  for (int i = tid; i <= a.n_traj; i += 256) {
    int off;
    if (i == a.n_traj) {
      off = (int)a.T;
    } else {
      int st = min(max(a.tso[i], 0), a.n_steps);  // clamped: offsets may be malformed
      off = a.sto[st];
      int steps = a.tso[i + 1] - a.tso[i];
      double den = (a.norm == GRPO_NORM_CONST_K) ? a.k : (double)steps;
      a.w[i] = 1.0 / (a.n_groups * (double)a.G * den);
    }
    a.traj_tok_off[i] = off;
    if (a.aux_traj_tok_off) a.aux_traj_tok_off[i] = bad ? -1 : off;
  }
  if (tid == 0) {
    a.hdr->flags = bad ? GRPO_FLAG_OFFSETS : 0;
    a.hdr->done = 0;
    for (int q = 0; q < 4; ++q) a.hdr->counts[q] = 0;
  }
}

// The trajectory of every token, found by binary search over the trajectory
// starts, and what the token epilogue needs from it (advantage, normaliser
// weight), so that the row passes read per-token values only.  Also the
// optional token outputs that need no logits.  One thread per token.
__global__ __launch_bounds__(256) void k_tok_traj(int64_t T, int32_t n_traj, const int32_t* traj_tok_off,
                                                  const WsHeader* hdr, const int32_t* actions, int64_t ld,
                                                  const float* adv, const double* w, float* tok_adv, double* tok_w,
                                                  int32_t* aux_tok_traj, int64_t* aux_gather) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= T) return;
  const int i = find_traj(traj_tok_off, n_traj, (int)t);
  tok_adv[t] = adv[i];
  tok_w[t] = w[i];
  if (aux_tok_traj) aux_tok_traj[t] = (hdr->flags & GRPO_FLAG_OFFSETS) ? -1 : i;
  if (aux_gather) aux_gather[t] = t * ld + actions[t];
}

hipError_t launch_segments(const grpo_segments* seg, int64_t T, int64_t ld, const int32_t* actions,
                           const float* adv, const grpo_loss_params* p, char* ws, const LossWs& L,
                           const grpo_aux* aux, hipStream_t s) {
  int32_t* aux_traj_tok_off = aux ? aux->traj_tok_off : nullptr;
  SegArgs a;
  a.sto = seg->step_tok_off;
  a.tso = seg->traj_step_off;
  a.n_steps = seg->n_steps;
  a.n_traj = seg->n_traj;
  a.G = seg->group_size;
  a.norm = p->norm;
  a.T = T;
  a.n_groups = n_groups_of(seg, p);
  a.k = (double)p->k;
  a.hdr = reinterpret_cast<WsHeader*>(ws + L.hdr);
  a.traj_tok_off = reinterpret_cast<int32_t*>(ws + L.traj_tok_off);
  a.w = reinterpret_cast<double*>(ws + L.w);
  a.aux_traj_tok_off = aux_traj_tok_off;
  hipLaunchKernelGGL(k_segments, dim3(1), dim3(256), 0, s, a);
  if (T > 0)
    hipLaunchKernelGGL(k_tok_traj, dim3((unsigned)((T + 255) / 256)), dim3(256), 0, s, T, seg->n_traj,
                       a.traj_tok_off, a.hdr, actions, ld, adv, a.w, reinterpret_cast<float*>(ws + L.tok_adv),
                       reinterpret_cast<double*>(ws + L.tok_w), aux ? aux->tok_traj : nullptr,
                       aux ? aux->gather_idx : nullptr);
  return hipGetLastError();
}

TokenArgs make_token_args(int64_t V, const int32_t* actions, const float* behave, const float* prox,
                          const float* adv, const grpo_loss_params* p, char* ws, const LossWs& L,
                          const grpo_aux* aux) {
  TokenArgs a;
  a.V = V;
  a.actions = actions;
  a.behave = behave;
  a.prox = prox;
  a.tok_adv = reinterpret_cast<const float*>(ws + L.tok_adv);
  a.tok_w = reinterpret_cast<const double*>(ws + L.tok_w);
  a.hdr = reinterpret_cast<WsHeader*>(ws + L.hdr);
  a.contrib = reinterpret_cast<double*>(ws + L.contrib);
  a.state = reinterpret_cast<int8_t*>(ws + L.state);
  a.tok_ratio = reinterpret_cast<double2*>(ws + L.tok_ratio);
  a.token_logp = aux ? aux->token_logp : nullptr;
  a.lo = 1.0 - (double)p->eps_low;
  a.hi = 1.0 + (double)p->eps_high;
  a.c = (double)p->dual_clip_c;
  a.grad_scale = (double)p->grad_scale;
  return a;
}

// ---- reduction -----------------------------------------------------------------
// One workgroup per trajectory sums its tokens' contributions in a fixed
// order; the last workgroup to finish sums the trajectories in index order.
struct ReduceArgs {
  int64_t T;
  int32_t n_traj;
  WsHeader* hdr;
  const int32_t* traj_tok_off;
  const double* contrib;
  const int8_t* state;
  const double2* tok_ratio;  // ws [T]: (r, rho), NaN outside the loss
  double* traj_loss;         // ws
  double* traj_rstats;       // ws [n_traj][6]: sum r, min r, max r, sum rho, min rho, max rho
  double* loss_out;
  double* aux_traj_loss;
  int64_t* aux_clip_counts;
  double* aux_ratio_stats;
  int32_t* aux_error_flags;
};

template <int NT>
__device__ __forceinline__ double block_sum(double v, double* sh) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  if (lane == 0) sh[wv] = v;
  __syncthreads();
  double r = 0.0;
  if (threadIdx.x == 0)
    for (int q = 0; q < NT / 64; ++q) r += sh[q];
  __syncthreads();
  return r;  // valid in thread 0
}

template <int NT, bool MAX>
__device__ __forceinline__ double block_ext(double v, double* sh) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const double u = __shfl_xor(v, o, 64);
    v = MAX ? fmax(v, u) : fmin(v, u);
  }
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  if (lane == 0) sh[wv] = v;
  __syncthreads();
  double r = v;
  if (threadIdx.x == 0)
    for (int q = 0; q < NT / 64; ++q) r = MAX ? fmax(r, sh[q]) : fmin(r, sh[q]);
  __syncthreads();
  return r;  // valid in thread 0
}

__global__ __launch_bounds__(256) void k_reduce(const ReduceArgs a) {
  __shared__ double sh[4];
  __shared__ int is_last;
  const int i = blockIdx.x, tid = threadIdx.x;
  const int64_t t0 = min(max((int64_t)a.traj_tok_off[i], (int64_t)0), a.T);
  const int64_t t1 = min(max((int64_t)a.traj_tok_off[i + 1], t0), a.T);
  double acc = 0.0, sr = 0.0, srho = 0.0;
  double rmin = INFINITY, rmax = -INFINITY, pmin = INFINITY, pmax = -INFINITY;
  int64_t c_eps = 0, c_dual = 0, c_out = 0, c_valid = 0;
  for (int64_t t = t0 + tid; t < t1; t += 256) {
    acc += a.contrib[t];
    const int st = a.state[t];
    c_eps += (st & kStateEpsCut) != 0;
    c_dual += (st & kStateDualCut) != 0;
    c_out += (st & kStateOutside) != 0;
    if (st & kStateValid) {
      ++c_valid;
      const double2 q = a.tok_ratio[t];
      sr += q.x;
      srho += q.y;
      rmin = fmin(rmin, q.x);
      rmax = fmax(rmax, q.x);
      pmin = fmin(pmin, q.y);
      pmax = fmax(pmax, q.y);
    }
  }
  const double tot = block_sum<256>(acc, sh);
  const double tsr = block_sum<256>(sr, sh), tsrho = block_sum<256>(srho, sh);
  const double trmin = block_ext<256, false>(rmin, sh), trmax = block_ext<256, true>(rmax, sh);
  const double tpmin = block_ext<256, false>(pmin, sh), tpmax = block_ext<256, true>(pmax, sh);
  c_eps = wave_sum_i64(c_eps);
  c_dual = wave_sum_i64(c_dual);
  c_out = wave_sum_i64(c_out);
  c_valid = wave_sum_i64(c_valid);
  if ((tid & 63) == 0 && (c_eps | c_dual | c_out | c_valid)) {
    atomicAdd((unsigned long long*)&a.hdr->counts[0], (unsigned long long)c_eps);
    atomicAdd((unsigned long long*)&a.hdr->counts[1], (unsigned long long)c_dual);
    atomicAdd((unsigned long long*)&a.hdr->counts[2], (unsigned long long)c_out);
    atomicAdd((unsigned long long*)&a.hdr->counts[3], (unsigned long long)c_valid);
  }
  __syncthreads();  // every wave's counter update is performed before the block reports done
  if (tid == 0) {
    a.traj_loss[i] = tot;
    double* rs = a.traj_rstats + 6 * (int64_t)i;
    rs[0] = tsr;
    rs[1] = trmin;
    rs[2] = trmax;
    rs[3] = tsrho;
    rs[4] = tpmin;
    rs[5] = tpmax;
    __threadfence();
    const unsigned prev = atomicAdd(&a.hdr->done, 1u);
    is_last = (prev == (unsigned)gridDim.x - 1);
  }
  __syncthreads();
  if (!is_last) return;
  __threadfence();
  double part = 0.0;
  for (int q = tid; q < a.n_traj; q += 256)
    part += __hip_atomic_load(&a.traj_loss[q], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const double loss = block_sum<256>(part, sh);
  const int flags = __hip_atomic_load(&a.hdr->flags, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const bool bad = flags & GRPO_FLAG_OFFSETS;
  if (a.aux_traj_loss)
    for (int q = tid; q < a.n_traj; q += 256)
      a.aux_traj_loss[q] =
          bad ? (double)NAN : __hip_atomic_load(&a.traj_loss[q], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (a.aux_ratio_stats) {
    // per-trajectory partials in index order (sums through the same fixed-shape tree as the loss)
    auto ld = [&](int q, int k) {
      return __hip_atomic_load(&a.traj_rstats[6 * (int64_t)q + k], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    };
    double p_sr = 0.0, p_srho = 0.0, p_rmin = INFINITY, p_rmax = -INFINITY, p_pmin = INFINITY, p_pmax = -INFINITY;
    for (int q = tid; q < a.n_traj; q += 256) {
      p_sr += ld(q, 0);
      p_rmin = fmin(p_rmin, ld(q, 1));
      p_rmax = fmax(p_rmax, ld(q, 2));
      p_srho += ld(q, 3);
      p_pmin = fmin(p_pmin, ld(q, 4));
      p_pmax = fmax(p_pmax, ld(q, 5));
    }
    const double v0 = block_sum<256>(p_sr, sh), v3 = block_sum<256>(p_srho, sh);
    const double v1 = block_ext<256, false>(p_rmin, sh), v2 = block_ext<256, true>(p_rmax, sh);
    const double v4 = block_ext<256, false>(p_pmin, sh), v5 = block_ext<256, true>(p_pmax, sh);
    if (tid == 0) {
      double* o = a.aux_ratio_stats;
      const double nan = (double)NAN;
      o[0] = bad ? nan : v0;
      o[1] = bad ? nan : v1;
      o[2] = bad ? nan : v2;
      o[3] = bad ? nan : v3;
      o[4] = bad ? nan : v4;
      o[5] = bad ? nan : v5;
      o[6] = (double)__hip_atomic_load(&a.hdr->counts[2], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      o[7] = (double)__hip_atomic_load(&a.hdr->counts[3], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  if (tid == 0) {
    *a.loss_out = bad ? (double)NAN : loss;
    if (a.aux_clip_counts) {
      a.aux_clip_counts[0] = __hip_atomic_load(&a.hdr->counts[0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      a.aux_clip_counts[1] = __hip_atomic_load(&a.hdr->counts[1], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    if (a.aux_error_flags) *a.aux_error_flags = flags;
  }
}

hipError_t launch_reduce(int64_t T, int32_t n_traj, char* ws, const LossWs& L, double* loss_out,
                         const grpo_aux* aux, hipStream_t s) {
  ReduceArgs a;
  a.T = T;
  a.n_traj = n_traj;
  a.hdr = reinterpret_cast<WsHeader*>(ws + L.hdr);
  a.traj_tok_off = reinterpret_cast<const int32_t*>(ws + L.traj_tok_off);
  a.contrib = reinterpret_cast<const double*>(ws + L.contrib);
  a.state = reinterpret_cast<const int8_t*>(ws + L.state);
  a.tok_ratio = reinterpret_cast<const double2*>(ws + L.tok_ratio);
  a.traj_loss = reinterpret_cast<double*>(ws + L.traj_loss);
  a.traj_rstats = reinterpret_cast<double*>(ws + L.traj_rstats);
  a.loss_out = loss_out;
  a.aux_traj_loss = aux ? aux->traj_loss : nullptr;
  a.aux_clip_counts = aux ? aux->clip_counts : nullptr;
  a.aux_ratio_stats = aux ? aux->ratio_stats : nullptr;
  a.aux_error_flags = aux ? aux->error_flags : nullptr;
  hipLaunchKernelGGL(k_reduce, dim3(n_traj), dim3(256), 0, s, a);
  return hipGetLastError();
}

// ---- group advantages (Sec. 3.2) -------------------------------------------------
// One workgroup per group; the moments are summed serially in fp64 so the
// result does not depend on the launch shape.
// mode GRPO_ADV_SUCCESS_FILTER: A_i = 1[r_i > 0] (RAFT++, Sec. 3.2 / Table 5).
// mixed (nullable): 1 when the group's rewards are not all equal (DAPO dynamic
// sampling, Sec. 3.2); n_mixed (nullable, cleared beforehand) counts them.
__global__ __launch_bounds__(64) void k_advantages(const float* __restrict__ r, int G, int mode, int ddof,
                                                   double std_eps, float* __restrict__ adv,
                                                   int32_t* __restrict__ mixed, int32_t* __restrict__ n_mixed) {
  __shared__ double sh_mean, sh_den;
  const int64_t base = (int64_t)blockIdx.x * G;
  if (threadIdx.x == 0 && (mixed || n_mixed)) {
    int m = 0;
    for (int q = 1; q < G; ++q) m |= (r[base + q] != r[base]);
    if (mixed) mixed[blockIdx.x] = m;
    if (n_mixed && m) atomicAdd(n_mixed, 1);
  }
  if (mode == GRPO_ADV_SUCCESS_FILTER) {
    for (int q = threadIdx.x; q < G; q += 64) adv[base + q] = (r[base + q] > 0.f) ? 1.f : 0.f;
    return;
  }
  if (threadIdx.x == 0) {
    double mean = 0.0;
    for (int q = 0; q < G; ++q) mean += (double)r[base + q];
    mean /= (double)G;
    double ss = 0.0;
    for (int q = 0; q < G; ++q) {
      const double d = (double)r[base + q] - mean;
      ss += d * d;
    }
    const double sd = (G - ddof > 0) ? sqrt(ss / (double)(G - ddof)) : 0.0;
    sh_mean = mean;
    sh_den = sd + std_eps;
  }
  __syncthreads();
  const double mean = sh_mean, den = sh_den;
  for (int q = threadIdx.x; q < G; q += 64)
    adv[base + q] = (den == 0.0) ? 0.f : (float)(((double)r[base + q] - mean) / den);
}

}  // namespace grpo

namespace grpo {
__global__ void k_clear_i32(int32_t* p) { *p = 0; }
}  // namespace grpo

extern "C" int grpo_advantages_ex(const float* rewards, int32_t n_traj, int32_t group_size, int32_t mode,
                                  int32_t ddof, float std_eps, float* adv_out, int32_t* group_mixed,
                                  int32_t* n_mixed, hipStream_t s) {
  if (!rewards || !adv_out) return GRPO_ERR_ARG;
  if (mode != GRPO_ADV_GROUP_NORM && mode != GRPO_ADV_SUCCESS_FILTER) return GRPO_ERR_ARG;
  if (ddof != 0 && ddof != 1) return GRPO_ERR_ARG;
  if (!(std_eps >= 0.f) || !isfinite(std_eps)) return GRPO_ERR_ARG;
  if (n_traj < 1 || group_size < 1 || n_traj % group_size != 0) return GRPO_ERR_SHAPE;
  if (n_mixed) hipLaunchKernelGGL(grpo::k_clear_i32, dim3(1), dim3(1), 0, s, n_mixed);
  hipLaunchKernelGGL(grpo::k_advantages, dim3(n_traj / group_size), dim3(64), 0, s, rewards, group_size, mode, ddof,
                     (double)std_eps, adv_out, group_mixed, n_mixed);
  return hipGetLastError() == hipSuccess ? GRPO_OK : GRPO_ERR_HIP;
}

extern "C" int grpo_advantages(const float* rewards, int32_t n_traj, int32_t group_size, int32_t ddof,
                               float std_eps, float* adv_out, hipStream_t s) {
  return grpo_advantages_ex(rewards, n_traj, group_size, GRPO_ADV_GROUP_NORM, ddof, std_eps, adv_out, nullptr,
                            nullptr, s);
}

extern "C" const char* grpo_status_str(int status) {
  switch (status) {
    case GRPO_OK: return "GRPO_OK";
    case GRPO_ERR_ARG: return "GRPO_ERR_ARG: a required pointer is NULL or a scalar is out of range";
    case GRPO_ERR_SHAPE: return "GRPO_ERR_SHAPE: inconsistent sizes";
    case GRPO_ERR_DTYPE: return "GRPO_ERR_DTYPE: unsupported dtype";
    case GRPO_ERR_WORKSPACE: return "GRPO_ERR_WORKSPACE: workspace missing or too small";
    case GRPO_ERR_ALIGN: return "GRPO_ERR_ALIGN: a device pointer is misaligned";
    case GRPO_ERR_HIP: return "GRPO_ERR_HIP: a HIP launch failed";
    default: return "unknown grpo status";
  }
}
