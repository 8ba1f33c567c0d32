// Device-side helpers shared by the libgrpo kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "grpo.h"

namespace grpo {

// Header block at the start of every loss workspace.
struct WsHeader {
  int32_t flags;      // GRPO_FLAG_* of this call (set by the segment pass, OR-ed by the row pass)
  uint32_t done;      // reduction workgroups finished (last-block pattern)
  int64_t counts[4];  // eps-clip cut, dual-clip cut, ratio outside the clip range, valid tokens
};

constexpr float kLog2e = 1.4426950408889634f;
constexpr double kLn2 = 0.69314718055994530942;

// ---- bf16 <-> fp32 ---------------------------------------------------------
// A bf16 value is the upper 16 bits of the fp32 with the same value, so the
// widening is a shift (low element of a dword) or a mask (high element).
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Round-to-nearest-even pack of two fp32 values into a bf16 pair (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  bf16x2 v = __builtin_convertvector((f32x2){lo, hi}, bf16x2);
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

// ---- wave64 reductions -----------------------------------------------------
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ int64_t wave_sum_i64(int64_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// ---- DPP reductions -----------------------------------------------------------
// Lane moves inside a row of 16 lanes go through the VALU (DPP) rather than the
// LDS crossbar that __shfl_xor uses, so a step costs a few cycles instead of an
// LDS round trip.  Every source lane of these patterns is valid.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, 0xF, 0xF, true);
}
template <int CTRL>
__device__ __forceinline__ float dpp_f32v(float x) { return __uint_as_float(dpp_u32<CTRL>(__float_as_uint(x))); }
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double x) {
  const uint64_t u = __builtin_bit_cast(uint64_t, x);
  const uint64_t lo = dpp_u32<CTRL>((uint32_t)u), hi = dpp_u32<CTRL>((uint32_t)(u >> 32));
  return __builtin_bit_cast(double, lo | (hi << 32));
}
// Max (sum) over each row of 16 lanes, in every lane of the row: swaps within
// quads (quad_perm [1, 0, 3, 2] = 0xB1, [2, 3, 0, 1] = 0x4E), then across the
// halves of each 8-lane group (row_half_mirror = 0x141), then across the two
// 8-lane groups (row_mirror = 0x140).
__device__ __forceinline__ float row16_max(float v) {
  v = fmaxf(v, dpp_f32v<0xB1>(v));
  v = fmaxf(v, dpp_f32v<0x4E>(v));
  v = fmaxf(v, dpp_f32v<0x141>(v));
  return fmaxf(v, dpp_f32v<0x140>(v));
}
__device__ __forceinline__ double row16_sum(double v) {
  v += dpp_f64<0xB1>(v);
  v += dpp_f64<0x4E>(v);
  v += dpp_f64<0x141>(v);
  return v + dpp_f64<0x140>(v);
}
__device__ __forceinline__ double readlane_f64(double v, int lane) {
  const uint64_t u = __builtin_bit_cast(uint64_t, v);
  const uint64_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, lane);
  const uint64_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), lane);
  return __builtin_bit_cast(double, lo | (hi << 32));
}
// Over the whole wave (all 64 lanes active), the same value in every lane.
__device__ __forceinline__ float wave_max_dpp(float v) {
  v = row16_max(v);
  const float a = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 0));
  const float b = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 16));
  const float c = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 32));
  const float d = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 48));
  return fmaxf(fmaxf(a, b), fmaxf(c, d));
}
__device__ __forceinline__ double wave_sum_dpp(double v) {
  v = row16_sum(v);
  return (readlane_f64(v, 0) + readlane_f64(v, 16)) + (readlane_f64(v, 32) + readlane_f64(v, 48));
}

// ---- per-token surrogate (Eq. 1 with the dual clip of Eq. 2) ----------------
// Bits of the per-token state.
constexpr int kStateEpsCut = 1;     // the eps clip held the term (its gradient is cut)
constexpr int kStateDualCut = 2;    // the dual clip held it
constexpr int kStateOutside = 4;    // r = pi/pi_prox lies outside [1 - eps_low, 1 + eps_high]
constexpr int kStateValid = 8;      // the token entered the loss (action in range, offsets valid)

struct TokenOut {
  double contrib;  // -w * s   (this token's share of the loss)
  double g;        // grad_scale * w * ds/dl
  double rho, r;   // pi/pi_behave and pi/pi_prox
  int state;       // kState* bits
};

// l: new log-prob, b: behave, p: prox, A: advantage, w: trajectory weight.
// The min of Eq. 1 picks the unclipped term rho*A unless the clipped term is
// smaller; inside the clip range both terms equal rho*A, so the derivative is
// rho*A except when the clip (or the dual-clip floor) holds the term fixed.
// The log-prob differences are formed in fp64 and the ratios, the min and the
// clips in fp32 (native exp2): one rounding of each ratio, far below the loss
// and dlogits tolerances; the token's share of the loss and its coefficient are
// scaled by the fp64 weight.
__device__ __forceinline__ float exp_f32(float x) { return __builtin_amdgcn_exp2f(x * kLog2e); }

__device__ __forceinline__ TokenOut token_surrogate(double l, double b, double p, double A_, double w,
                                                    double lo_, double hi_, double c_, double grad_scale) {
  // rho = pi / pi_behave, r = pi / pi_prox, omega = pi_prox / pi_behave; with
  // pi_prox = pi_behave (the coupled ratio) omega = 1 and r = rho exactly.
  const float A = (float)A_, lo = (float)lo_, hi = (float)hi_, c = (float)c_;
  const float rho = exp_f32((float)(l - b));
  const float r = (p == b) ? rho : exp_f32((float)(l - p));
  const float omega = (p == b) ? 1.f : exp_f32((float)(p - b));
  const bool inside = (r >= lo) && (r <= hi);
  const float r_cl = fminf(fmaxf(r, lo), hi);
  const float u1 = rho * A;
  const float u2 = omega * r_cl * A;
  float s = u1, ds = u1;
  int state = 0;
  if (u2 < u1) {
    s = u2;
    if (!inside) {
      ds = 0.f;
      state = kStateEpsCut;
    }
  }
  if (c > 0.f && A < 0.f && s < c * A) {
    s = c * A;
    ds = 0.f;
    state |= kStateDualCut;
  }
  TokenOut o;
  o.contrib = -w * (double)s;
  o.g = grad_scale * w * (double)ds;
  o.rho = rho;
  o.r = r;
  o.state = state | (inside ? 0 : kStateOutside) | kStateValid;
  return o;
}

// Log-sum-exp of a row from its shift M and fp64 sum S = sum e^(z - M) >= 1:
// S = f 2^e with f in [0.5, 1), and log2 f in fp32 (v_log_f32) is good to ~1e-7.
__device__ __forceinline__ double row_lse(double M, double S) {
  int e;
  const double f = frexp(S, &e);
  return M + ((double)e + (double)__builtin_amdgcn_logf((float)f)) * kLn2;
}

// Trajectory of token t: the largest i with traj_tok_off[i] <= t (trajectories
// with no token share a start and are skipped).  Indices stay in [0, n-1]
// whatever the contents, so malformed offsets cannot push reads out of range.
__device__ __forceinline__ int find_traj(const int32_t* __restrict__ traj_tok_off, int n, int t) {
  int lo = 0, hi = n - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (traj_tok_off[mid] <= t) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

// ---- the per-token epilogue shared by the logits and fused paths -------------
struct TokenArgs {
  int64_t V;
  const int32_t* actions;
  const float* behave;
  const float* prox;        // nullable: coupled ratio
  const float* tok_adv;     // ws [T]: advantage of each token's trajectory (segment pass)
  const double* tok_w;      // ws [T]: normaliser weight of each token's trajectory
  WsHeader* hdr;            // ws
  double* contrib;          // ws [T]
  int8_t* state;            // ws [T]
  double2* tok_ratio;       // ws [T]: (r, rho) of each token, NaN for tokens outside the loss
  float* token_logp;        // aux, nullable
  double lo, hi, c, grad_scale;
};

// The per-token inputs of the epilogue.  Every address depends only on t, so
// a workgroup can issue these loads long before it needs them.
struct TokenIn {
  int act, bad_off;
  float b, p, A;
  double w;
};

__device__ __forceinline__ TokenIn token_load(const TokenArgs& a, int t) {
  TokenIn in;
  in.act = a.actions[t];
  in.bad_off = a.hdr->flags & GRPO_FLAG_OFFSETS;  // final before any row pass starts
  in.b = a.behave[t];
  in.p = a.prox ? a.prox[t] : in.b;
  in.A = a.tok_adv[t];
  in.w = a.tok_w[t];
  return in;
}

// How the dlogits row is formed: d_v = sign * 2^(z_v*log2e + nc) for v != a_t
// (nc folds -lse*log2e + log2|g|), and d_a for the action column.  act < 0
// means the row is zero.
struct RowScale {
  float nc, sign, d_a;
  int act;
};

// The per-token epilogue, once the row's log-sum-exp is known, in two halves: token_eval forms the row's dlogits
// scale and the token's outputs without touching memory (so every wave of a row may run it), token_store writes
// those outputs (one thread per token).  z_a is the action's logit (ignored when the action is out of range).
struct TokenEval {
  TokenOut o;
  double l;  // the token's new log-prob
  bool bad_act, bad;
};

__device__ inline RowScale token_eval(const TokenArgs& a, const TokenIn& in, double lse, double z_a, TokenEval& e) {
  RowScale rs;
  e.bad_act = in.act < 0 || (int64_t)in.act >= a.V;
  e.bad = in.bad_off || e.bad_act;
  rs.act = in.act;
  if (e.bad) {
    rs.nc = -INFINITY;  // every d_v = 0
    rs.sign = 1.f;
    rs.d_a = 0.f;
    rs.act = -1;
    return rs;
  }
  e.l = z_a - lse;
  const double b = (double)in.b, p = (double)in.p, A = (double)in.A;
  e.o = token_surrogate(e.l, b, p, A, in.w, a.lo, a.hi, a.c, a.grad_scale);
  const TokenOut& o = e.o;
  // d_v = g exp(z_v - lse) = sign(g) 2^(z_v L - lse L + log2|g|), with L = log2(e) as rounded on the device
  rs.nc = (float)(-lse * (double)kLog2e) + __builtin_amdgcn_logf(fabsf((float)o.g));
  rs.sign = (o.g < 0.0) ? -1.f : 1.f;
  rs.d_a = (float)o.g * expm1f((float)e.l);  // g (p_a - 1), without cancellation
  if (isnan(o.g)) rs.nc = NAN;
  return rs;
}

// Writes the token's loss contribution, clip state, ratios and log-prob, and raises the flags.
__device__ inline void token_store(const TokenArgs& a, int t, const TokenIn& in, const TokenEval& e) {
  if (e.bad) {
    if (e.bad_act && !in.bad_off) atomicOr(&a.hdr->flags, GRPO_FLAG_ACTION);
    a.contrib[t] = in.bad_off ? (double)NAN : 0.0;
    a.state[t] = 0;
    a.tok_ratio[t] = make_double2((double)NAN, (double)NAN);
    if (a.token_logp) a.token_logp[t] = 0.f;
    return;
  }
  if (!isfinite(e.l) || !isfinite(in.b) || !isfinite(in.p) || !isfinite(in.A))
    atomicOr(&a.hdr->flags, GRPO_FLAG_NONFINITE);
  a.contrib[t] = e.o.contrib;
  a.state[t] = (int8_t)e.o.state;
  a.tok_ratio[t] = make_double2(e.o.r, e.o.rho);
  if (a.token_logp) a.token_logp[t] = (float)e.l;
}

// Both halves on one thread.
__device__ inline RowScale token_finish(const TokenArgs& a, int t, const TokenIn& in, double lse, double z_a) {
  TokenEval e;
  const RowScale rs = token_eval(a, in, lse, z_a, e);
  token_store(a, t, in, e);
  return rs;
}

// A row's log-sum-exp and action logit from the per-token records of every shard
// of a vocabulary split over devices (stats [n_shards][T]), merged in shard order
// so that every device gets the same bits: lse = M + log sum_g s_g e^(m_g - M),
// M = max_g m_g, and z_a = max_g z_a_g (only the owner's is finite).  A NaN
// maximum propagates.
__device__ inline void merge_vocab_stats(const grpo_vocab_stats* stats, int n_shards, int T, int t, double& lse,
                                         double& za) {
  double M = -INFINITY, z = -INFINITY;
  for (int g = 0; g < n_shards; ++g) {
    const grpo_vocab_stats r = stats[(int64_t)g * T + t];
    if (r.m > M || isnan(r.m)) M = r.m;
    z = fmax(z, r.z_a);
  }
  double S = 0.0;
  for (int g = 0; g < n_shards; ++g) {
    const grpo_vocab_stats r = stats[(int64_t)g * T + t];
    if (r.m != -INFINITY) S += r.s * exp(r.m - M);
  }
  lse = row_lse(M, S);
  za = z;
}

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// max(a, b, c) in one instruction.  Written as asm because the compiler otherwise canonicalises every loaded
// value before an fmaxf (two more instructions per dword of logits).  In IEEE mode a quiet NaN operand is
// ignored, as by fmaxf, and a signalling NaN makes the result NaN; either way a NaN logit also makes the row's
// sum of exponentials NaN, so the row is flagged as before.
__device__ __forceinline__ float max3f(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

// Maximum of m and the vector's elements (the exp shift of the row).
template <typename Tin>
__device__ __forceinline__ float vec_max(const u32x4& x, float m) {
  if constexpr (sizeof(Tin) == 2) {
    const float a = max3f(bf16_lo(x[0]), bf16_hi(x[0]), bf16_lo(x[1]));
    const float b = max3f(bf16_hi(x[1]), bf16_lo(x[2]), bf16_hi(x[2]));
    const float c = max3f(bf16_lo(x[3]), bf16_hi(x[3]), m);
    return max3f(a, b, c);
  } else {
    return max3f(max3f(m, __uint_as_float(x[0]), __uint_as_float(x[1])), __uint_as_float(x[2]),
                 __uint_as_float(x[3]));
  }
}

// dlogits of one vector: |d_v| = 2^(z_v*log2e + nc), the row's sign applied to
// the packed result, and the action column (when it falls in this vector)
// replaced by d_a.
template <typename Tin>
__device__ __forceinline__ u32x4 vec_dlogits(const u32x4& x, const RowScale& rs, uint32_t signmask, bool has_act,
                                             int act_lane) {
  u32x4 o;
  if constexpr (sizeof(Tin) == 2) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float lo = __builtin_amdgcn_exp2f(fmaf(bf16_lo(x[q]), kLog2e, rs.nc));
      const float hi = __builtin_amdgcn_exp2f(fmaf(bf16_hi(x[q]), kLog2e, rs.nc));
      o[q] = pack_bf16(lo, hi) ^ signmask;
    }
    if (has_act) {
      const uint32_t da = pack_bf16(rs.d_a, 0.f) & 0xffffu;
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if ((act_lane >> 1) == q) o[q] = (act_lane & 1) ? ((o[q] & 0xffffu) | (da << 16)) : ((o[q] & 0xffff0000u) | da);
    }
  } else {
#pragma unroll
    for (int q = 0; q < 4; ++q)
      o[q] = __float_as_uint(__builtin_amdgcn_exp2f(fmaf(__uint_as_float(x[q]), kLog2e, rs.nc))) ^ signmask;
    if (has_act) {
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (act_lane == q) o[q] = __float_as_uint(rs.d_a);
    }
  }
  return o;
}

template <typename Tin>
__device__ __forceinline__ uint32_t sign_mask(const RowScale& rs) {
  if (rs.sign >= 0.f) return 0u;
  return sizeof(Tin) == 2 ? 0x80008000u : 0x80000000u;
}

}  // namespace grpo
