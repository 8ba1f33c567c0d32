// The logits path: streaming log-softmax + gather, the per-token surrogate of
// Eq. 1 (dual clip of Eq. 2), and dlogits, one workgroup per token row.
//
// Every row is read from HBM once with 16-byte loads (a wavefront covers 1 KiB
// contiguous per instruction), reduced to (max, sum exp) per thread, combined
// across the workgroup, and dlogits are formed from the same registers and
// written once: V*s bytes read and V*s written per token.
//
//  k_rows_pipe      long bf16 rows (V up to 188,416): persistent, one
//                   workgroup of 1024 threads per CU.  Row t+G streams in
//                   while row t's dlogits are written: part of each row lives
//                   in LDS (global_load_lds), the rest in registers.
//  k_rows_resident  shorter rows: one workgroup per row, several per CU.
//  two passes       vector rows too long for either (fp32 beyond 77,824
//                   columns, bf16 beyond 188,416): each row reduced to a
//                   record (logp.hip), then the record turned into the token
//                   epilogue and the row's dlogits (vocab.hip); the row is
//                   read twice.
//  k_rows_generic   any V, stride or alignment: element loads, three sweeps.
#include <hip/hip_runtime.h>
#include <math.h>

#include <algorithm>
#include <mutex>

#include "device.h"
#include "launch.h"

namespace grpo {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Row-pass arguments: the logits, the dlogits destination and the token epilogue.
struct RowArgs {
  const void* logits;
  void* dlogits;  // nullable: forward only
  int64_t ld;     // row stride in elements
  int T;
  int chunk;      // k_rows_pipe: consecutive rows a workgroup takes at a time (>= 1) in rows [0, r0)
  int r0;         // k_rows_pipe: a multiple of chunk * gridDim.x
  int chunk2;     // k_rows_pipe: rows [r0, T) go chunk2 at a time, one chunk per workgroup (>= 1)
  TokenArgs tok;
};

template <typename Tin>
__device__ __forceinline__ float load_elem(const Tin* p);
template <>
__device__ __forceinline__ float load_elem<float>(const float* p) { return *p; }
template <>
__device__ __forceinline__ float load_elem<uint16_t>(const uint16_t* p) { return bf16_to_f32(*p); }

// Element e of a 16-byte vector (8 bf16 or 4 fp32), widened to fp32.
template <typename Tin>
__device__ __forceinline__ float vec_elem(const u32x4& x, int e) {
  if constexpr (sizeof(Tin) == 2) {
    uint32_t w = x[0];
#pragma unroll
    for (int q = 1; q < 4; ++q)
      if ((e >> 1) == q) w = x[q];
    return (e & 1) ? bf16_hi(w) : bf16_lo(w);
  } else {
    uint32_t w = x[0];
#pragma unroll
    for (int q = 1; q < 4; ++q)
      if (e == q) w = x[q];
    return __uint_as_float(w);
  }
}

// sum of exp(z - m) over the vector, with nmb = -m*log2(e)
template <typename Tin>
__device__ __forceinline__ float vec_sumexp(const u32x4& x, float nmb) {
  float s = 0.f;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    if constexpr (sizeof(Tin) == 2) {
      s += __builtin_amdgcn_exp2f(fmaf(bf16_lo(x[q]), kLog2e, nmb)) +
           __builtin_amdgcn_exp2f(fmaf(bf16_hi(x[q]), kLog2e, nmb));
    } else {
      s += __builtin_amdgcn_exp2f(fmaf(__uint_as_float(x[q]), kLog2e, nmb));
    }
  }
  return s;
}

// The LDS part of a k_rows_pipe row keeps its terms: the sum pass overwrites each vector of 8 bf16 logits in the
// thread's own LDS slot with its terms e = exp(z - m) as fp16 pairs (round to nearest even), and the dlogits pass
// forms d = g exp(z - lse) = c e with one multiply, c = g exp(m - lse), instead of a second exponential.  The terms
// are <= 1: relative error at most 2^-11 for e >= 2^-14, absolute at most 2^-25 below, before the bf16 rounding of
// d.  The sum is formed from the fp32 terms in vec_sumexp's order.  (Not the register part: kept there, the
// compiler issued all of the part's exponentials ahead of their packs and spilled the fp32 terms; and with three
// register vectors' terms parked in the LDS left free, the kernel ran no faster.)
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_f16(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){lo, hi}, f16x2));
}
__device__ __forceinline__ f32x2 unpack_f16(uint32_t w) {
  return __builtin_convertvector(__builtin_bit_cast(f16x2, w), f32x2);
}
__device__ __forceinline__ float vec_sumexp_keep(u32x4& x, float nmb) {
  float s = 0.f;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const float lo = __builtin_amdgcn_exp2f(fmaf(bf16_lo(x[q]), kLog2e, nmb));
    const float hi = __builtin_amdgcn_exp2f(fmaf(bf16_hi(x[q]), kLog2e, nmb));
    s += lo + hi;
    x[q] = pack_f16(lo, hi);
  }
  return s;
}
// dlogits of a vector of kept terms, bf16 round to nearest even; c carries the row's sign; the action column (when
// it falls in this vector) replaced by d_a.
__device__ __forceinline__ u32x4 vec_dlogits_kept(const u32x4& e, float c, bool has_act, int act_lane, float d_a) {
  u32x4 o;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const f32x2 f = unpack_f16(e[q]);
    o[q] = pack_bf16(f[0] * c, f[1] * c);
  }
  if (has_act) {
    const uint32_t da = pack_bf16(d_a, 0.f) & 0xffffu;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if ((act_lane >> 1) == q) o[q] = (act_lane & 1) ? ((o[q] & 0xffffu) | (da << 16)) : ((o[q] & 0xffff0000u) | da);
  }
  return o;
}

// Combines every thread's (max m, sum s of exp(z - m)) into the row's (M, S),
// valid in thread 0: within each wave (DPP within rows of 16 lanes, then the
// four rows), then across the NW <= 16 waves by the first 16 lanes of wave 0,
// one wave partial per lane.  The rescale factors exp(m - M) <= 1 are fp32 and
// the sums fp64.  Every lane of the workgroup takes part.  Ends with every wave
// past a barrier.
template <int NW>
__device__ __forceinline__ void block_combine(float m, float s, float* sh_m, double* sh_s, double& M_out,
                                              double& S_out) {
  static_assert(NW >= 1 && NW <= 16, "one wave partial per lane of a 16-lane row");
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const float mw = wave_max_dpp(m);
  const double sw =
      wave_sum_dpp((m == -INFINITY) ? 0.0 : (double)s * (double)__builtin_amdgcn_exp2f((m - mw) * kLog2e));
  if (lane == 0) {
    sh_m[wv] = mw;
    sh_s[wv] = sw;
  }
  __syncthreads();
  if (wv == 0) {
    const float mq = lane < NW ? sh_m[lane] : -INFINITY;
    const float M = row16_max(mq);
    const double S =
        row16_sum(mq == -INFINITY ? 0.0 : sh_s[lane < NW ? lane : 0] * (double)__builtin_amdgcn_exp2f((mq - M) * kLog2e));
    M_out = (double)M;
    S_out = S;
  }
}

// As block_combine, but every wave reads the NW wave partials and forms the row's (M, S) itself, so that every
// lane of the workgroup holds them after the one barrier (each 16-lane row of a wave reduces the same partials).
template <int NW>
__device__ __forceinline__ void block_combine_all(float m, float s, float* sh_m, double* sh_s, double& M_out,
                                                  double& S_out) {
  static_assert(NW >= 1 && NW <= 16, "one wave partial per lane of a 16-lane row");
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, r = lane & 15;
  const float mw = wave_max_dpp(m);
  const double sw =
      wave_sum_dpp((m == -INFINITY) ? 0.0 : (double)s * (double)__builtin_amdgcn_exp2f((m - mw) * kLog2e));
  if (lane == 0) {
    sh_m[wv] = mw;
    sh_s[wv] = sw;
  }
  __syncthreads();
  const float mq = r < NW ? sh_m[r] : -INFINITY;
  const float M = row16_max(mq);
  M_out = (double)M;
  S_out = row16_sum(mq == -INFINITY ? 0.0 : sh_s[r < NW ? r : 0] * (double)__builtin_amdgcn_exp2f((mq - M) * kLog2e));
}

// ---- persistent pipelined kernel for long bf16 rows ----------------------------
// Buffer resources cover exactly one row (V*2 bytes): every access is a 32-bit
// lane offset (tid*16) plus a constant per-vector offset, and the hardware
// range check returns 0 for loads past the row and drops such stores.
constexpr uint32_t kRsrcWord3 = 0x00020000u;  // raw buffer, 32-bit data format
constexpr int kStream = 2;                    // non-temporal cache policy for streamed rows

__device__ __forceinline__ __amdgpu_buffer_rsrc_t row_rsrc(const void* base, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, bytes, kRsrcWord3);
}

// 16 bytes per lane from the buffer (rsrc, voff + soff) into LDS at lds_base + 16 * lane, non-temporal.
// Inline asm: the compiler's own handling of LDS DMA would hold every LDS read back until all LDS DMA in
// flight has landed; the kernel orders them with explicit waits instead.  M0 carries the LDS address;
// nothing else in this kernel uses it.  An LDS DMA must not follow the write of M0 directly: one wait state
// between them (the compiler inserts the same for its own LDS DMA; it cannot see inside this asm).
__device__ __forceinline__ void dma16_nt(uint32_t lds_base, uint32_t voff, uint32_t soff, u32x4 rsrc) {
  lds_base = __builtin_amdgcn_readfirstlane(lds_base);
  soff = __builtin_amdgcn_readfirstlane(soff);
#pragma unroll
  for (int k = 0; k < 4; ++k) rsrc[k] = __builtin_amdgcn_readfirstlane(rsrc[k]);
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, %3 offen nt lds" ::"s"(lds_base), "v"(voff), "s"(rsrc),
               "s"(soff)
               : "memory", "m0");
}
__device__ __forceinline__ u32x4 row_rsrc_words(const void* base, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  u32x4 r = {(uint32_t)a, (uint32_t)(a >> 32) & 0xffffu, bytes, kRsrcWord3};
  return r;
}
// waits until at most N vector-memory operations of this wave are outstanding (they complete in order)
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt(0x0F70 | (N & 15) | ((N >> 4) << 14));
}
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Hides the register vectors' values from the optimiser, so that the widened
// bf16 of one pass is recomputed in the next instead of kept live across it.
template <int N>
__device__ __forceinline__ void fresh(u32x4 (&v)[N]) {
#pragma unroll
  for (int q = 0; q < N; ++q) asm volatile("" : "+v"(v[q]));
}

// Each thread owns NV vectors of 8 bf16, with (NV-1)*1024 < V/8 <= NV*1024 so
// that only the last vector can be partial.  The first NP live in LDS (staged
// with buffer loads straight to LDS and read back in every pass), the other
// NR = NV - NP in registers.  Once the row's lse is known, dlogits are written
// first for the LDS part, which is then re-staged with the next row, and then
// for the register part, whose registers are then reloaded with the next
// row's vectors.
template <int NV, int NP>
__global__ __launch_bounds__(1024) void k_rows_pipe(const RowArgs a) {
  constexpr int NT = 1024, NW = NT / 64, NR = NV - NP, VB = NT * 16;  // VB: bytes per vector slot
  __shared__ __attribute__((aligned(16))) u32x4 stage[NP * NT];
  __shared__ float sh_m[NW];
  __shared__ double sh_s[NW];
  __shared__ float sh_za;
  __shared__ TokenIn sh_in;  // inputs of the row about to start (wave 1 loads them during the previous row)
  const int wv = threadIdx.x >> 6;
  const int nvec = (int)(a.tok.V / 8);
  const int row_bytes = nvec * 16;
  const uint16_t* logits = static_cast<const uint16_t*>(a.logits);
  uint16_t* dlogits = static_cast<uint16_t*>(a.dlogits);

  const uint32_t lds_stage =
      (uint32_t)reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) u32x4*)stage) + wv * 64 * 16;
  auto stage_row = [&](int r, int voff) {  // vectors 0..NP-1 of row r -> LDS, asynchronously
    const u32x4 src = row_rsrc_words(logits + (int64_t)r * a.ld, (uint32_t)row_bytes);
#pragma unroll
    for (int j = 0; j < NP; ++j) dma16_nt(lds_stage + j * NT * 16, voff, j * VB, src);
  };
  auto load_regs = [&](u32x4 (&dst)[NR], int r, int voff) {
    const __amdgpu_buffer_rsrc_t src = row_rsrc(logits + (int64_t)r * a.ld, row_bytes);
#pragma unroll
    for (int q = 0; q < NR; ++q) dst[q] = __builtin_amdgcn_raw_buffer_load_b128(src, voff, (NP + q) * VB, kStream);
  };

  // Rows [0, r0) go to workgroups in chunks of `chunk` consecutive rows, chunk c to workgroup c mod gridDim.x;
  // the rest, fewer than chunk * gridDim.x rows, in one chunk of chunk2 rows per workgroup, so that no workgroup
  // has more than chunk2 rows beyond the others.  A workgroup walks its chunks in order, so the row it stages
  // next is usually the one after the row it writes.  Past its last row, next_row returns T.
  const int C = a.chunk, R0 = a.r0, C2 = a.chunk2;
  auto next_row = [&](int r) {
    const int q = r + 1;
    if (r < R0) {
      if (q % C != 0) return q;
      const int nq = q + ((int)gridDim.x - 1) * C;
      return nq < R0 ? nq : min(R0 + (int)blockIdx.x * C2, a.T);
    }
    return ((q - R0) % C2 != 0 && q < a.T) ? q : a.T;
  };
  int t = R0 > 0 ? (int)blockIdx.x * C : R0 + (int)blockIdx.x * C2;
  if (t >= a.T) return;
  u32x4 reg[NR];
  if (threadIdx.x == 64) sh_in = token_load(a.tok, t);
  stage_row(t, threadIdx.x * 16);
  load_regs(reg, t, threadIdx.x * 16);
  wait_vmcnt<NR>();  // this wave's LDS part of row t has landed; the register loads may still be in flight

  for (int t_next = 0; t < a.T; t = t_next) {
    // The thread index is laundered per row so that nothing derived from it
    // is hoisted out of the row loop and kept live across it.
    int tid = threadIdx.x;
    asm volatile("" : "+v"(tid));
    const int voff = tid * 16;
    const bool last_full = tid < nvec - (NV - 1) * NT;
    const int tn = next_row(t);
    t_next = tn;
    lds_barrier();  // every wave's LDS part of row t has landed, and sh_in holds row t's inputs
    const TokenIn in = sh_in;
    const int act_vec = (in.act >= 0 && in.act < a.tok.V) ? in.act / 8 : -1;
    const int act_lane = in.act & 7;

    // (max, sum exp) over the LDS part first, while the register part is still landing
    float m1 = -INFINITY;
#pragma unroll 1
    for (int j = 0; j < NP; ++j) {
      const u32x4 x = stage[j * NT + tid];
      m1 = vec_max<uint16_t>(x, m1);
      if (j * NT + tid == act_vec) sh_za = vec_elem<uint16_t>(x, act_lane);
    }
    const float nmb1 = (m1 == -INFINITY) ? 0.f : -m1 * kLog2e;
    float s1 = 0.f;
#pragma unroll 1
    for (int j = 0; j < NP; ++j) {  // the terms replace the logits in the thread's own LDS slots
      u32x4 x = stage[j * NT + tid];
      s1 += vec_sumexp_keep(x, nmb1);
      stage[j * NT + tid] = x;
    }
    float m = m1;
#pragma unroll
    for (int q = 0; q < NR; ++q) {
      const int j = NP + q;
      if (j < NV - 1 || last_full) {
        m = vec_max<uint16_t>(reg[q], m);
        if (j * NT + tid == act_vec) sh_za = vec_elem<uint16_t>(reg[q], act_lane);
      }
    }
    const float nmb = (m == -INFINITY) ? 0.f : -m * kLog2e;
    float s = (m1 == -INFINITY) ? 0.f : s1 * __builtin_amdgcn_exp2f((m1 - m) * kLog2e);
    fresh(reg);
#pragma unroll
    for (int q = 0; q < NR; ++q)
      if (NP + q < NV - 1 || last_full) s += vec_sumexp<uint16_t>(reg[q], nmb);

    double M, S;
    block_combine_all<NW>(m, s, sh_m, sh_s, M, S);  // barrier: sh_za is visible, every lane holds (M, S)
    // every wave forms the row's scale itself (no second barrier, no one-lane section); thread 0 writes the
    // token's outputs
    TokenEval ev;
    const RowScale rs = token_eval(a.tok, in, row_lse(M, S), (double)sh_za, ev);
    if (tid == 0) token_store(a.tok, t, in, ev);
    // wave 1 fetches the next row's token inputs meanwhile (every wave read this row's from sh_in before the
    // barrier above; the next row reads them after its first barrier)
    if (tid == 64) sh_in = token_load(a.tok, tn < a.T ? tn : t);

    const uint32_t smask = sign_mask<uint16_t>(rs);
    const float c1 = rs.sign * __builtin_amdgcn_exp2f(rs.nc - nmb1);  // the LDS part's terms: d = c1 e
    const int act_v = rs.act >= 0 ? rs.act / 8 : -1;
    fresh(reg);
    // forward only: a zero-sized destination, so the range check drops every store
    const bool write = dlogits != nullptr;
    const __amdgpu_buffer_rsrc_t dst = row_rsrc(write ? dlogits + (int64_t)t * a.ld : logits, write ? row_bytes : 0);
#pragma unroll 1
    for (int j = 0; j < NP; ++j)
      __builtin_amdgcn_raw_buffer_store_b128(
          vec_dlogits_kept(stage[j * NT + tid], c1, j * NT + tid == act_v, rs.act & 7, rs.d_a), dst, voff, j * VB,
          kStream);
    lds_barrier();  // every wave is done reading stage[] (the stores read registers)
    if (tn < a.T) stage_row(tn, voff);
    // past the last row: a zero-sized source, every load returns 0
    const __amdgpu_buffer_rsrc_t nxt = row_rsrc(logits + (int64_t)(tn < a.T ? tn : t) * a.ld, tn < a.T ? row_bytes : 0);
    // All of the register part's stores, then all of its loads: a burst in each direction per wave runs 7-8%
    // faster than alternating store and load per vector.  Each store is followed by two wait states: the compiler
    // reuses a store's data registers in the very next instruction (it inserts no wait for a 16-byte buffer store
    // with a register offset), and when it did, the store wrote the overwritten values.
#pragma unroll
    for (int q = 0; q < NR; ++q) {
      const int j = NP + q;
      __builtin_amdgcn_raw_buffer_store_b128(
          vec_dlogits<uint16_t>(reg[q], rs, smask, j * NT + tid == act_v, rs.act & 7), dst, voff, j * VB, kStream);
      __builtin_amdgcn_sched_barrier(0);
      asm volatile("s_nop 1" ::: "memory");
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int q = 0; q < NR; ++q) reg[q] = __builtin_amdgcn_raw_buffer_load_b128(nxt, voff, (NP + q) * VB, kStream);
    // the 2 NR register stores and loads were issued after the LDS part of row tn, so this returns once
    // that part has landed
    wait_vmcnt<2 * NR>();
  }
}

// ---- register-resident row kernel -------------------------------------------
// NT threads per row, NV 16-byte vectors per thread: V <= NT*NV*EPV.  Rows are
// 16-byte aligned and V is a multiple of EPV (checked on the host).
template <typename Tin, int NT, int NV>
__global__ __launch_bounds__(NT) void k_rows_resident(const RowArgs a) {
  constexpr int EPV = 16 / sizeof(Tin);  // elements per vector: 8 bf16 or 4 fp32
  constexpr int NW = NT / 64;
  __shared__ float sh_m[NW];
  __shared__ double sh_s[NW];
  __shared__ float sh_za;

  const int t = blockIdx.x;
  const int tid = threadIdx.x;
  const int nvec = (int)(a.tok.V / EPV);
  const u32x4* src = reinterpret_cast<const u32x4*>(static_cast<const Tin*>(a.logits) + (int64_t)t * a.ld);
  const TokenIn in = token_load(a.tok, t);
  const int act_vec = (in.act >= 0 && in.act < a.tok.V) ? in.act / EPV : -1;
  const int act_lane = in.act % EPV;

  u32x4 buf[NV];
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int vi = j * NT + tid;
    if (vi < nvec) buf[j] = __builtin_nontemporal_load(src + vi);
  }
  float m = -INFINITY;
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int vi = j * NT + tid;
    if (vi < nvec) {
      m = vec_max<Tin>(buf[j], m);
      if (vi == act_vec) sh_za = vec_elem<Tin>(buf[j], act_lane);
    }
  }
  const float nmb = (m == -INFINITY) ? 0.f : -m * kLog2e;
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < NV; ++j)
    if (j * NT + tid < nvec) s += vec_sumexp<Tin>(buf[j], nmb);

  double M, S;
  block_combine_all<NW>(m, s, sh_m, sh_s, M, S);  // barrier: sh_za is visible, every lane holds (M, S)
  // every wave forms the row's scale itself; thread 0 writes the token's outputs
  TokenEval ev;
  const RowScale rs = token_eval(a.tok, in, row_lse(M, S), (double)sh_za, ev);
  if (tid == 0) token_store(a.tok, t, in, ev);
  if (!a.dlogits) return;

  const uint32_t smask = sign_mask<Tin>(rs);
  u32x4* dst = reinterpret_cast<u32x4*>(static_cast<Tin*>(a.dlogits) + (int64_t)t * a.ld);
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int vi = j * NT + tid;
    if (vi < nvec)
      __builtin_nontemporal_store(vec_dlogits<Tin>(buf[j], rs, smask, vi == rs.act / EPV && rs.act >= 0,
                                                   rs.act % EPV),
                                  dst + vi);
  }
}

// ---- generic row kernel ------------------------------------------------------
// Any V, ld and element alignment: element-wise loads, the row read three
// times (max, sum, dlogits).  Used when the vector kernels do not apply.
template <typename Tin>
__global__ __launch_bounds__(256) void k_rows_generic(const RowArgs a) {
  constexpr int NT = 256, NW = NT / 64;
  __shared__ float sh_m[NW];
  __shared__ double sh_s[NW];
  __shared__ RowScale sh_rs;
  const int t = blockIdx.x, tid = threadIdx.x;
  const Tin* row = static_cast<const Tin*>(a.logits) + (int64_t)t * a.ld;
  const TokenIn in = token_load(a.tok, t);
  float m = -INFINITY;
  for (int64_t v = tid; v < a.tok.V; v += NT) m = fmaxf(m, load_elem<Tin>(row + v));
  const float nmb = (m == -INFINITY) ? 0.f : -m * kLog2e;
  float s = 0.f;
  for (int64_t v = tid; v < a.tok.V; v += NT) s += __builtin_amdgcn_exp2f(fmaf(load_elem<Tin>(row + v), kLog2e, nmb));
  double M, S;
  block_combine<NW>(m, s, sh_m, sh_s, M, S);
  if (tid == 0) {
    const bool ok = in.act >= 0 && (int64_t)in.act < a.tok.V;
    sh_rs = token_finish(a.tok, t, in, row_lse(M, S), ok ? (double)load_elem<Tin>(row + in.act) : 0.0);
  }
  __syncthreads();
  if (!a.dlogits) return;
  const RowScale rs = sh_rs;
  Tin* drow = static_cast<Tin*>(a.dlogits) + (int64_t)t * a.ld;
  for (int64_t v = tid; v < a.tok.V; v += NT) {
    const float d =
        (v == rs.act) ? rs.d_a : rs.sign * __builtin_amdgcn_exp2f(fmaf(load_elem<Tin>(row + v), kLog2e, rs.nc));
    if constexpr (sizeof(Tin) == 2) {
      drow[v] = (uint16_t)(pack_bf16(d, 0.f) & 0xffffu);
    } else {
      drow[v] = d;
    }
  }
}

// ---- dispatch ------------------------------------------------------------------
typedef void (*RowKernel)(const RowArgs);

struct Variant {
  int nt, nv;
  RowKernel bf16, f32;
};

#define GRPO_VARIANT(NT, NV) \
  { NT, NV, k_rows_resident<uint16_t, NT, NV>, k_rows_resident<float, NT, NV> }

// Searched in order; the first that holds the row is used.  Rows of 3,073 to 4,096 vectors (a bf16 vocabulary of
// 32,000 among them) take 1024 threads x 4 vectors: 6% faster there than 256 x 16 (0.707 against 0.752 ms at
// 32,411 x 32,000), 5% faster than 512 x 8.
static const Variant kVariants[] = {
    GRPO_VARIANT(64, 1),    GRPO_VARIANT(64, 2),    GRPO_VARIANT(64, 4),    GRPO_VARIANT(64, 8),
    GRPO_VARIANT(256, 4),   GRPO_VARIANT(256, 8),   GRPO_VARIANT(256, 12),  GRPO_VARIANT(1024, 4),
    GRPO_VARIANT(256, 20),  GRPO_VARIANT(256, 24),  GRPO_VARIANT(1024, 8),  GRPO_VARIANT(1024, 12),
    GRPO_VARIANT(1024, 16), GRPO_VARIANT(1024, 19),
};  // 1024 threads x 19 vectors is the largest that does not spill

// The persistent kernels for long bf16 rows, one per NV = ceil(V/8/1024) so
// that only each thread's last vector can be partial; NP vectors in LDS.
static const RowKernel kPipe[] = {
    k_rows_pipe<7, 4>,   k_rows_pipe<8, 4>,   k_rows_pipe<9, 5>,   k_rows_pipe<10, 5>, k_rows_pipe<11, 6>,
    k_rows_pipe<12, 6>,  k_rows_pipe<13, 7>,  k_rows_pipe<14, 7>,  k_rows_pipe<15, 1>, k_rows_pipe<16, 2>,
    k_rows_pipe<17, 3>,  k_rows_pipe<18, 4>,  k_rows_pipe<19, 6>,  k_rows_pipe<20, 9>, k_rows_pipe<21, 9>,
    k_rows_pipe<22, 9>,  k_rows_pipe<23, 9>,
};  // from 15 vectors on, 14 in registers and the rest in LDS, except 19 (V = 151,936): 13 and 6, 0.3% faster
   // than 15 and 4 and 0.4% faster than 14 and 5, with 12 and 7 or 11 and 8 within 0.1% of it (before the LDS
   // part kept its terms, 15 and 4 was 0.4% faster than 14 and 5)
constexpr int kPipeMinNV = 7, kPipeMaxNV = 23;  // at most 15 register vectors and 9 LDS vectors per thread
constexpr int64_t kPipeMaxT = (int64_t)1 << 30;  // t + (gridDim.x - 1) * chunk + 1 stays far below 2^31

struct Launch {
  RowKernel k;
  int nt;
  unsigned grid;
  int chunk = 1, r0 = 0, chunk2 = 1;
};

static Launch pick_row_kernel(grpo_dtype dt, int64_t T, int64_t V, int64_t ld, const void* logits,
                              const void* dlogits, hipStream_t s) {
  const int epv = (dt == GRPO_BF16) ? 8 : 4;
  const bool vec_ok = (V % epv == 0) && (ld % epv == 0) && aligned(logits, 16) && aligned(dlogits, 16);
  if (vec_ok) {
    const int64_t nvec = V / epv;
    const int64_t nv = (nvec + 1023) / 1024;
    if (dt == GRPO_BF16 && nv >= kPipeMinNV && nv <= kPipeMaxNV && T <= kPipeMaxT) {
      int n_cu = stream_cu_count(s);  // of the stream's device
      if (n_cu < 1) n_cu = 256;
      // chunks of up to 8 rows (1.6-2.5% faster than single rows at 120,000 x 151,936), but at least four chunks
      // per CU, so that small batches still spread over the chip
      const int64_t chunk = std::max<int64_t>(1, std::min<int64_t>(8, T / (4 * (int64_t)n_cu)));
      const int64_t n_chunks = (T + chunk - 1) / chunk;
      const int64_t g = n_chunks < n_cu ? n_chunks : n_cu;  // one workgroup per CU (LDS bound)
      // whole rounds of chunks, then the remaining rows split evenly: at T = 120,000 the busiest workgroup has
      // 469 rows instead of 472
      const int64_t r0 = T / (chunk * g) * (chunk * g);
      const int64_t chunk2 = std::max<int64_t>(1, (T - r0 + g - 1) / g);
      return Launch{kPipe[nv - kPipeMinNV], 1024, (unsigned)g, (int)chunk, (int)r0, (int)chunk2};
    }
    for (const Variant& v : kVariants) {
      if ((int64_t)v.nt * v.nv >= nvec) return Launch{dt == GRPO_BF16 ? v.bf16 : v.f32, v.nt, (unsigned)T};
    }
    return Launch{nullptr, 0, 0};  // two passes
  }
  return Launch{dt == GRPO_BF16 ? k_rows_generic<uint16_t> : k_rows_generic<float>, 256, (unsigned)T};
}

}  // namespace grpo

using namespace grpo;

extern "C" size_t grpo_loss_workspace_bytes(int64_t T, int32_t n_traj) {
  if (T < 0 || T >= ((int64_t)1 << 31) || n_traj < 1) return 0;  // the loss entry points refuse T >= 2^31
  return loss_ws_layout(T, n_traj).total;
}

// Argument checks of the logits path other than the workspace's (GRPO_OK or the error).
static int check_logits_call(const void* logits, int32_t dt, int64_t T, int64_t V, int64_t ld,
                             const int32_t* actions, const float* behave_logp, const float* adv,
                             const grpo_segments* seg, const grpo_loss_params* p, const double* loss_out,
                             const void* dlogits) {
  int st = check_loss_common(T, actions, behave_logp, adv, seg, p, loss_out);
  if (st != GRPO_OK) return st;
  if (dt != GRPO_BF16 && dt != GRPO_F32) return GRPO_ERR_DTYPE;
  if (T > 0 && !logits) return GRPO_ERR_ARG;
  if (V < 1 || ld < V || V >= ((int64_t)1 << 31)) return GRPO_ERR_SHAPE;
  const size_t esz = (dt == GRPO_BF16) ? 2 : 4;
  if (!aligned(logits, esz) || !aligned(dlogits, esz)) return GRPO_ERR_ALIGN;
  return GRPO_OK;
}

extern "C" int grpo_loss_fwd_bwd(const void* logits, int32_t dtype, int64_t T, int64_t V, int64_t ld,
                                 const int32_t* actions, const float* behave_logp, const float* prox_logp,
                                 const float* adv, const grpo_segments* seg, const grpo_loss_params* p,
                                 double* loss_out, void* dlogits, grpo_aux* aux, void* ws, size_t ws_bytes,
                                 hipStream_t s) {
  const int st = check_logits_call(logits, dtype, T, V, ld, actions, behave_logp, adv, seg, p, loss_out, dlogits);
  if (st != GRPO_OK) return st;
  const grpo_dtype dt = static_cast<grpo_dtype>(dtype);
  const LossWs L = loss_ws_layout(T, seg->n_traj);
  if (!ws || ws_bytes < L.total) return GRPO_ERR_WORKSPACE;
  if (!aligned(ws, kAlign)) return GRPO_ERR_ALIGN;
  char* w = static_cast<char*>(ws);

  if (launch_segments(seg, T, ld, actions, adv, p, w, L, aux, s) != hipSuccess) return GRPO_ERR_HIP;
  if (T > 0) {
    RowArgs a;
    a.logits = logits;
    a.dlogits = dlogits;
    a.ld = ld;
    a.T = (int)T;
    a.tok = make_token_args(V, actions, behave_logp, prox_logp, adv, p, w, L, aux);
    const Launch k = pick_row_kernel(dt, T, V, ld, logits, dlogits, s);
    a.chunk = k.chunk;
    a.r0 = k.r0;
    a.chunk2 = k.chunk2;
    const bool timed = aux && aux->hot_begin && aux->hot_end;
    if (timed && hipEventRecord(aux->hot_begin, s) != hipSuccess) return GRPO_ERR_HIP;
    if (k.k) {
      hipLaunchKernelGGL(k.k, dim3(k.grid), dim3(k.nt), 0, s, a);
      if (hipGetLastError() != hipSuccess) return GRPO_ERR_HIP;
    } else {
      // the whole vocabulary as one shard: its records, then the merge (trivial), epilogue and dlogits
      grpo_vocab_stats* rec = reinterpret_cast<grpo_vocab_stats*>(w + L.records);
      int32_t* flags = &reinterpret_cast<WsHeader*>(w + L.hdr)->flags;
      if (launch_vocab_records(logits, dt, T, V, ld, 0, actions, rec, flags, s) != hipSuccess) return GRPO_ERR_HIP;
      if (launch_shard_rows(logits, dlogits, dt, T, V, ld, 0, rec, 1, a.tok, s) != hipSuccess) return GRPO_ERR_HIP;
    }
    if (timed && hipEventRecord(aux->hot_end, s) != hipSuccess) return GRPO_ERR_HIP;
  }
  if (launch_reduce(T, seg->n_traj, w, L, loss_out, aux, s) != hipSuccess) return GRPO_ERR_HIP;
  return GRPO_OK;
}

// ---- the logits path without a caller workspace ------------------------------------
// For callers that cannot allocate device memory, the workspace is a file-scope device array of fixed size.
// Each device the library runs on holds its own copy until the process ends; host code reaches it only through
// the address hipGetSymbolAddress returns on that device, looked up once per device and kept.
static __device__ __align__(256) char scratch[GRPO_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
char* g_scratch[kMaxDevices];  // device address of `scratch` per device (nullptr until its first call)
}  // namespace

// The scratch array's address on the stream's device: looked up with that device current on the device's first
// call, then read from the table.
static int scratch_of_stream(hipStream_t s, char** out) {
  hipDevice_t dev = 0;
  if (hipStreamGetDevice(s, &dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return GRPO_ERR_HIP;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    int cur = 0;
    if (hipGetDevice(&cur) != hipSuccess) return GRPO_ERR_HIP;
    if (cur != dev && hipSetDevice(dev) != hipSuccess) return GRPO_ERR_HIP;
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (cur != dev && hipSetDevice(cur) != hipSuccess) return GRPO_ERR_HIP;
    if (e != hipSuccess || !ptr) return GRPO_ERR_HIP;
    g_scratch[dev] = static_cast<char*>(ptr);
  }
  *out = g_scratch[dev];
  return GRPO_OK;
}

extern "C" int grpo_loss_fwd_bwd_noalloc(const void* logits, int32_t dt, int64_t T, int64_t V, int64_t ld,
                                         const int32_t* actions, const float* behave_logp, const float* prox_logp,
                                         const float* adv, const grpo_segments* seg, const grpo_loss_params* p,
                                         double* loss_out, void* dlogits, grpo_aux* aux, hipStream_t s) {
  const int st = check_logits_call(logits, dt, T, V, ld, actions, behave_logp, adv, seg, p, loss_out, dlogits);
  if (st != GRPO_OK) return st;
  if (loss_ws_layout(T, seg->n_traj).total > (size_t)GRPO_NOALLOC_SCRATCH_BYTES) return GRPO_ERR_WORKSPACE;
  char* ws = nullptr;
  const int sc = scratch_of_stream(s, &ws);
  if (sc != GRPO_OK) return sc;
  return grpo_loss_fwd_bwd(logits, dt, T, V, ld, actions, behave_logp, prox_logp, adv, seg, p, loss_out, dlogits,
                           aux, ws, (size_t)GRPO_NOALLOC_SCRATCH_BYTES, s);
}
