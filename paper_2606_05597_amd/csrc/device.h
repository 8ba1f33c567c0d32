// Device-side helpers shared by the libgrpo kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "grpo.h"

namespace grpo {

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

// ---- per-token surrogate (Eq. 1 with the dual clip of Eq. 2) ----------------
struct TokenOut {
  double contrib;  // -w * s   (this token's share of the loss)
  double g;        // grad_scale * w * ds/dl
  int state;       // bit 0: eps clip held the term, bit 1: dual clip held it
};

// l: new log-prob, b: behave, p: prox, A: advantage, w: trajectory weight.
// The min of Eq. 1 picks the unclipped term rho*A unless the clipped term is
// smaller; inside the clip range both terms equal rho*A, so the derivative is
// rho*A except when the clip (or the dual-clip floor) holds the term fixed.
__device__ __forceinline__ TokenOut token_surrogate(double l, double b, double p, double A, double w,
                                                    double lo, double hi, double c, double grad_scale) {
  const double rho = exp(l - b);    // pi / pi_behave
  const double r = exp(l - p);      // pi / pi_prox
  const double omega = exp(p - b);  // pi_prox / pi_behave
  const bool inside = (r >= lo) && (r <= hi);
  const double r_cl = fmin(fmax(r, lo), hi);
  const double u1 = rho * A;
  const double u2 = omega * r_cl * A;
  double s = u1, ds = u1;
  int state = 0;
  if (u2 < u1) {
    s = u2;
    if (!inside) {
      ds = 0.0;
      state = 1;
    }
  }
  if (c > 0.0 && A < 0.0 && s < c * A) {
    s = c * A;
    ds = 0.0;
    state |= 2;
  }
  TokenOut o;
  o.contrib = -w * s;
  o.g = grad_scale * w * ds;
  o.state = state;
  return o;
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

}  // namespace grpo
