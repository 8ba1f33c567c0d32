// Forward only: the sampled action's log-prob and the policy entropy of each
// token row (the proximal log-probs recomputed before an update, Table 5, and
// the per-token entropy of Sec. 5), one workgroup per row.  The same kernels
// also reduce one shard of a vocabulary split over devices to its per-token
// record (max, sum exp, action logit; grpo_vocab_shard_stats).
//
// A row is read once.  Each thread walks its 16-byte vectors U at a time (all U
// loads in flight together) and keeps, relative to its running shift m,
//   s = sum e^(z - m)   and   t = sum e^(z - m) (z - m),
// rescaling both when a chunk raises m.  For any shift m >= max z the row's
// log-sum-exp is m + log s and its entropy -sum p log p = log s - t / s; both
// terms of the entropy are >= 0, so it has no cancellation even when small.
#include <hip/hip_runtime.h>
#include <float.h>
#include <math.h>

#include "device.h"
#include "host.h"
#include "launch.h"

namespace grpo {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

struct LogpArgs {
  const void* logits;
  int64_t ld, V;
  int64_t v_begin;  // global id of column 0 (a shard's first column; 0 otherwise)
  int T;
  const int32_t* actions;
  float* logp;      // nullable
  float* entropy;   // nullable
  int32_t* flags;   // nullable
  grpo_vocab_stats* stats;  // non-null: write each row's shard record instead of logp / entropy
};

// One element folded into (s, t) at the current shift m: s = sum e^(z - m), t = sum e^(z - m) w with
// w = (z - m) log2(e), the argument the exp2 takes anyway (t is in log2 units; row_out converts).  A -inf logit (a
// masked column) has e = 0 and adds no term (0 log 0 = 0): its w = -inf is clamped to -FLT_MAX in the product,
// which is then 0, not NaN.  A NaN logit still makes e, and so s and t, NaN.
// ENT = false: s only (t stays 0), for the calls that want no entropy.
template <bool ENT = true>
__device__ __forceinline__ void fold(float z, float nmb, float& s, float& t) {
  const float w = fmaf(z, kLog2e, nmb);
  const float e = __builtin_amdgcn_exp2f(w);
  s += e;
  if constexpr (ENT) t = fmaf(e, fmaxf(w, -FLT_MAX), t);
}

// Raises the shift to mn >= m: s and t are re-expressed relative to mn.
template <bool ENT = true>
__device__ __forceinline__ void rescale(float& m, float mn, float& s, float& t) {
  if (mn > m) {
    if (m != -INFINITY) {
      const float dl = (mn - m) * kLog2e, f = __builtin_amdgcn_exp2f(-dl);
      if constexpr (ENT) t = f * fmaf(-dl, s, t);
      s *= f;
    }
    m = mn;
  }
}

// Combines every thread's (m, s, t) into the row's (M, S, T) in fp64, valid in thread 0 (t and T in log2 units):
// within each wave (DPP within rows of 16 lanes, then the four rows), then across the NW <= 16 waves by the first
// 16 lanes of wave 0.  Every lane of the workgroup takes part.
template <int NW>
__device__ __forceinline__ void block_combine3(float m, float s, float t, float* sh_m, double* sh_s, double* sh_t,
                                               double& M_out, double& S_out, double& T_out) {
  static_assert(NW >= 1 && NW <= 16, "one wave partial per lane of a 16-lane row");
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const double L = (double)kLog2e;
  const float mw = wave_max_dpp(m);
  const double f = (m == -INFINITY) ? 0.0 : (double)__builtin_amdgcn_exp2f((m - mw) * kLog2e);
  const double sw = wave_sum_dpp(f * (double)s);
  const double tw = wave_sum_dpp(m == -INFINITY ? 0.0 : f * ((double)t + ((double)m - (double)mw) * L * (double)s));
  if (lane == 0) {
    sh_m[wv] = mw;
    sh_s[wv] = sw;
    sh_t[wv] = tw;
  }
  __syncthreads();
  if (wv == 0) {
    const float mq = lane < NW ? sh_m[lane] : -INFINITY;
    const float M = row16_max(mq);
    const double g = (mq == -INFINITY) ? 0.0 : exp((double)mq - (double)M);
    const int q = lane < NW ? lane : 0;
    const double S = row16_sum(g * sh_s[q]);
    const double T = row16_sum(mq == -INFINITY ? 0.0 : g * (sh_t[q] + ((double)mq - (double)M) * L * sh_s[q]));
    M_out = (double)M;
    S_out = S;
    T_out = T;
  }
}

// Element e of a 16-byte vector (8 bf16 or 4 fp32), widened to fp32.
template <typename Tin>
__device__ __forceinline__ float elem(const u32x4& x, int e) {
  if constexpr (sizeof(Tin) == 2) {
    const uint32_t w = x[e >> 1];
    return (e & 1) ? bf16_hi(w) : bf16_lo(w);
  } else {
    return __uint_as_float(x[e]);
  }
}

template <typename Tin>
__device__ __forceinline__ void row_out(const LogpArgs& a, int t, double M, double S, double Tsum, double za,
                                        bool act_ok) {
  if (a.stats) {
    grpo_vocab_stats r;
    r.m = M;  // the maximum of stored values: exact
    r.s = S;
    r.z_a = act_ok ? za : -INFINITY;
    a.stats[t] = r;
    if (a.flags && (isnan(M) || isnan(S) || M == INFINITY)) atomicOr(a.flags, GRPO_FLAG_NONFINITE);
    return;
  }
  const double lse = M + log(S);
  if (a.logp) a.logp[t] = act_ok ? (float)(za - lse) : 0.f;
  // Tsum is in log2 units: sum e^(z - M) (z - M) = Tsum / log2(e)
  if (a.entropy) a.entropy[t] = (float)(log(S) - Tsum / ((double)kLog2e * S));
  if (a.flags) {
    if (!act_ok) atomicOr(a.flags, GRPO_FLAG_ACTION);
    if (!isfinite(lse)) atomicOr(a.flags, GRPO_FLAG_NONFINITE);
  }
}

// Rows of 16-byte vectors (V a multiple of the vector width, 16-byte aligned rows).  ENT: the entropy moment
// is accumulated (not for a shard's records or a call without an entropy output).
template <typename Tin, int NT, int U, bool ENT>
__global__ __launch_bounds__(NT) void k_logp_vec(const LogpArgs a) {
  constexpr int EPV = 16 / sizeof(Tin), NW = NT / 64;
  __shared__ float sh_m[NW];
  __shared__ double sh_s[NW], sh_t[NW];
  __shared__ float sh_za;
  const int t = blockIdx.x, tid = threadIdx.x;
  const int nvec = (int)(a.V / EPV);
  const u32x4* row = reinterpret_cast<const u32x4*>(static_cast<const Tin*>(a.logits) + (int64_t)t * a.ld);
  const int64_t act64 = (int64_t)a.actions[t] - a.v_begin;
  const bool act_ok = act64 >= 0 && act64 < a.V;
  const int act = act_ok ? (int)act64 : 0;
  const int act_vec = act_ok ? act / EPV : -1;
  float m = -INFINITY, s = 0.f, tt = 0.f;
  for (int base = tid; base < nvec; base += NT * U) {
    u32x4 x[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int vi = base + u * NT;
      if (vi < nvec) x[u] = __builtin_nontemporal_load(row + vi);
    }
    float cm = -INFINITY;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int vi = base + u * NT;
      if (vi < nvec) {
        cm = vec_max<Tin>(x[u], cm);
        if (vi == act_vec) sh_za = elem<Tin>(x[u], act % EPV);
      }
    }
    rescale<ENT>(m, cm, s, tt);
    const float nmb = (m == -INFINITY) ? 0.f : -m * kLog2e;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int vi = base + u * NT;
      if (vi < nvec) {
#pragma unroll
        for (int e = 0; e < EPV; ++e) fold<ENT>(elem<Tin>(x[u], e), nmb, s, tt);
      }
    }
  }
  double M, S, Tsum;
  block_combine3<NW>(m, s, tt, sh_m, sh_s, sh_t, M, S, Tsum);  // its barrier publishes sh_za
  if (tid == 0) row_out<Tin>(a, t, M, S, Tsum, act_ok ? (double)sh_za : 0.0, act_ok);
}

template <typename Tin>
__device__ __forceinline__ float load_one(const Tin* p);
template <>
__device__ __forceinline__ float load_one<float>(const float* p) { return *p; }
template <>
__device__ __forceinline__ float load_one<uint16_t>(const uint16_t* p) { return bf16_to_f32(*p); }

// Any V, ld and element alignment: element loads, the row read twice (shift, then sums).
template <typename Tin>
__global__ __launch_bounds__(256) void k_logp_generic(const LogpArgs a) {
  constexpr int NT = 256, NW = NT / 64;
  __shared__ float sh_m[NW];
  __shared__ double sh_s[NW], sh_t[NW];
  const int t = blockIdx.x, tid = threadIdx.x;
  const Tin* row = static_cast<const Tin*>(a.logits) + (int64_t)t * a.ld;
  float m = -INFINITY;
  for (int64_t v = tid; v < a.V; v += NT) m = fmaxf(m, load_one<Tin>(row + v));
  const float nmb = (m == -INFINITY) ? 0.f : -m * kLog2e;
  float s = 0.f, tt = 0.f;
  if (m != -INFINITY)
    for (int64_t v = tid; v < a.V; v += NT) fold(load_one<Tin>(row + v), nmb, s, tt);
  double M, S, Tsum;
  block_combine3<NW>(m, s, tt, sh_m, sh_s, sh_t, M, S, Tsum);
  if (tid == 0) {
    const int64_t act = (int64_t)a.actions[t] - a.v_begin;
    const bool act_ok = act >= 0 && act < a.V;
    row_out<Tin>(a, t, M, S, Tsum, act_ok ? (double)load_one<Tin>(row + act) : 0.0, act_ok);
  }
}

__global__ void k_clear_flag(int32_t* f) { *f = 0; }

// One workgroup per row: the vector kernel when rows are whole 16-byte vectors, else the element kernel.
static void launch_logp(const LogpArgs& a, grpo_dtype dt, hipStream_t s) {
  const int esz = (dt == GRPO_BF16) ? 2 : 4, epv = 16 / esz;
  const bool vec = a.V % epv == 0 && a.ld % epv == 0 && aligned(a.logits, 16);
  const dim3 grid((unsigned)a.T);
  const bool ent = a.entropy && !a.stats;
  if (vec && dt == GRPO_BF16) {
    if (ent) hipLaunchKernelGGL((k_logp_vec<uint16_t, 256, 4, true>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((k_logp_vec<uint16_t, 256, 4, false>), grid, dim3(256), 0, s, a);
  } else if (vec) {
    if (ent) hipLaunchKernelGGL((k_logp_vec<float, 256, 4, true>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((k_logp_vec<float, 256, 4, false>), grid, dim3(256), 0, s, a);
  } else if (dt == GRPO_BF16) {
    hipLaunchKernelGGL(k_logp_generic<uint16_t>, grid, dim3(256), 0, s, a);
  } else {
    hipLaunchKernelGGL(k_logp_generic<float>, grid, dim3(256), 0, s, a);
  }
}

hipError_t launch_vocab_records(const void* logits, grpo_dtype dt, int64_t T, int64_t V, int64_t ld,
                                int64_t v_begin, const int32_t* actions, grpo_vocab_stats* stats, int32_t* flags,
                                hipStream_t s) {
  if (T > 0) {
    LogpArgs a{logits, ld, V, v_begin, (int)T, actions, nullptr, nullptr, flags, stats};
    launch_logp(a, dt, s);
  }
  return hipGetLastError();
}

}  // namespace grpo

using namespace grpo;

extern "C" int grpo_token_logp(const void* logits, int32_t dtype, int64_t T, int64_t V, int64_t ld,
                               const int32_t* actions, float* token_logp, float* token_entropy, int32_t* error_flags,
                               hipStream_t s) {
  if (T < 0 || T >= ((int64_t)1 << 31) || V < 1 || ld < V) return GRPO_ERR_SHAPE;
  if (T > 0 && (!logits || !actions)) return GRPO_ERR_ARG;
  if (dtype != GRPO_F32 && dtype != GRPO_BF16) return GRPO_ERR_DTYPE;
  const grpo_dtype dt = static_cast<grpo_dtype>(dtype);
  const int esz = (dt == GRPO_BF16) ? 2 : 4;
  if (!aligned(logits, esz)) return GRPO_ERR_ALIGN;
  if (error_flags) hipLaunchKernelGGL(k_clear_flag, dim3(1), dim3(1), 0, s, error_flags);
  if (T > 0) {
    LogpArgs a{logits, ld, V, 0, (int)T, actions, token_logp, token_entropy, error_flags, nullptr};
    launch_logp(a, dt, s);
  }
  return hipGetLastError() == hipSuccess ? GRPO_OK : GRPO_ERR_HIP;
}

extern "C" int grpo_vocab_shard_stats(const void* logits, int32_t dtype, int64_t T, int64_t V_shard, int64_t ld,
                                      int64_t v_begin, const int32_t* actions, grpo_vocab_stats* stats,
                                      int32_t* error_flags, hipStream_t s) {
  constexpr int64_t kLim = (int64_t)1 << 31;  // v_begin + V_shard < 2^31, tested without forming the sum first
  if (T < 0 || T >= kLim || V_shard < 1 || V_shard >= kLim || ld < V_shard || v_begin < 0 ||
      v_begin >= kLim - V_shard)
    return GRPO_ERR_SHAPE;
  if (T > 0 && (!logits || !actions || !stats)) return GRPO_ERR_ARG;
  if (dtype != GRPO_F32 && dtype != GRPO_BF16) return GRPO_ERR_DTYPE;
  const grpo_dtype dt = static_cast<grpo_dtype>(dtype);
  const int esz = (dt == GRPO_BF16) ? 2 : 4;
  if (!aligned(logits, esz) || !aligned(stats, 8)) return GRPO_ERR_ALIGN;
  if (error_flags) hipLaunchKernelGGL(k_clear_flag, dim3(1), dim3(1), 0, s, error_flags);
  if (T > 0) {
    LogpArgs a{logits, ld, V_shard, v_begin, (int)T, actions, nullptr, nullptr, error_flags, stats};
    launch_logp(a, dt, s);
  }
  return hipGetLastError() == hipSuccess ? GRPO_OK : GRPO_ERR_HIP;
}
