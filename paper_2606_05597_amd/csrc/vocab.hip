// The loss of Eq. 1 (dual clip of Eq. 2) with the vocabulary split over
// devices, the shard a device holds: logits [T, V_shard] for global columns
// [v_begin, v_begin + V_shard).
//
//   1. grpo_vocab_shard_stats (logp.hip): each shard reduces its columns of
//      every row to (max m, sum s of e^(z - m), the action logit z_a if the
//      action is one of its columns), 24 bytes per token.
//   2. the caller gathers every shard's records on every device (T x 24 bytes
//      per shard);
//   3. grpo_loss_fwd_bwd_vocab_shard (here): per row, the records are merged in
//      shard order into the row's log-sum-exp M + log sum_g s_g e^(m_g - M) and
//      action logit, the token epilogue runs as on one device, and the shard's
//      columns of dlogits are written.  Every shard computes the same per-token
//      values and the same loss, because they come from the same records in the
//      same order.
//
// A shard's row is read twice (once per step, with the exchange between them)
// and its dlogits written once: 6 V_shard bytes per bf16 token instead of the
// single-device 4 V.
#include <hip/hip_runtime.h>
#include <math.h>

#include "device.h"
#include "launch.h"

namespace grpo {

struct ShardArgs {
  const void* logits;
  void* dlogits;  // nullable: forward only
  int64_t ld;     // row stride in elements
  int64_t V;      // the shard's columns
  int64_t v_begin;
  int T, n_shards;
  const grpo_vocab_stats* stats;  // [n_shards][T]
  TokenArgs tok;                  // tok.V: the whole vocabulary
};

// Thread 0: merge, token epilogue, the action's column within this shard (-1 if
// another shard holds it).
__device__ inline void shard_row_head(const ShardArgs& a, int t, RowScale& rs, int& act_local) {
  double lse, za;
  merge_vocab_stats(a.stats, a.n_shards, a.T, t, lse, za);
  const TokenIn in = token_load(a.tok, t);
  rs = token_finish(a.tok, t, in, lse, za);
  const int64_t al = rs.act >= 0 ? (int64_t)rs.act - a.v_begin : -1;
  act_local = (al >= 0 && al < a.V) ? (int)al : -1;
}

// Rows of 16-byte vectors, one workgroup per row; U vectors per thread in flight.
// The row's first U vectors per thread are loaded before the records are merged (the loads do not depend on
// them), and every wave merges the records and forms the scale itself while they land: no barrier, no one-thread
// section ahead of the loads.  Thread 0 alone writes the token's outputs.
template <typename Tin, int NT, int U>
__global__ __launch_bounds__(NT) void k_shard_rows_vec(const ShardArgs a) {
  constexpr int EPV = 16 / sizeof(Tin);
  const int t = blockIdx.x, tid = threadIdx.x;
  if (!a.dlogits) {  // forward only: the token's outputs, no row traffic
    if (tid == 0) {
      RowScale rs;
      int al;
      shard_row_head(a, t, rs, al);
    }
    return;
  }
  const int nvec = (int)(a.V / EPV);
  const u32x4* src = reinterpret_cast<const u32x4*>(static_cast<const Tin*>(a.logits) + (int64_t)t * a.ld);
  u32x4* dst = reinterpret_cast<u32x4*>(static_cast<Tin*>(a.dlogits) + (int64_t)t * a.ld);
  u32x4 x[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int vi = tid + u * NT;
    if (vi < nvec) x[u] = __builtin_nontemporal_load(src + vi);
  }
  double lse, za;
  merge_vocab_stats(a.stats, a.n_shards, a.T, t, lse, za);
  const TokenIn in = token_load(a.tok, t);
  TokenEval ev;
  const RowScale rs = token_eval(a.tok, in, lse, za, ev);
  if (tid == 0) token_store(a.tok, t, in, ev);
  const int64_t al = rs.act >= 0 ? (int64_t)rs.act - a.v_begin : -1;
  const int act = (al >= 0 && al < a.V) ? (int)al : -1;  // the action's column in this shard, if it holds it
  const int act_vec = act >= 0 ? act / EPV : -1, act_lane = act >= 0 ? act % EPV : 0;
  const uint32_t smask = sign_mask<Tin>(rs);
  for (int base = tid; base < nvec; base += NT * U) {
    if (base != tid) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int vi = base + u * NT;
        if (vi < nvec) x[u] = __builtin_nontemporal_load(src + vi);
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int vi = base + u * NT;
      if (vi < nvec) __builtin_nontemporal_store(vec_dlogits<Tin>(x[u], rs, smask, vi == act_vec, act_lane), dst + vi);
    }
  }
}

template <typename Tin>
__device__ __forceinline__ float shard_load(const Tin* p);
template <>
__device__ __forceinline__ float shard_load<float>(const float* p) { return *p; }
template <>
__device__ __forceinline__ float shard_load<uint16_t>(const uint16_t* p) { return bf16_to_f32(*p); }
__device__ __forceinline__ void shard_store(float* p, float v) { *p = v; }
__device__ __forceinline__ void shard_store(uint16_t* p, float v) { *p = (uint16_t)(pack_bf16(v, 0.f) & 0xffffu); }

// Any V, stride or alignment: element loads and stores.
template <typename Tin>
__global__ __launch_bounds__(256) void k_shard_rows_generic(const ShardArgs a) {
  __shared__ RowScale sh_rs;
  __shared__ int sh_act;
  const int t = blockIdx.x, tid = threadIdx.x;
  if (tid == 0) {
    RowScale rs;
    int al;
    shard_row_head(a, t, rs, al);
    sh_rs = rs;
    sh_act = al;
  }
  __syncthreads();
  if (!a.dlogits) return;
  const RowScale rs = sh_rs;
  const int act = sh_act;
  const Tin* src = static_cast<const Tin*>(a.logits) + (int64_t)t * a.ld;
  Tin* dst = static_cast<Tin*>(a.dlogits) + (int64_t)t * a.ld;
  for (int64_t v = tid; v < a.V; v += 256) {
    const float d = (v == act) ? rs.d_a : rs.sign * __builtin_amdgcn_exp2f(fmaf(shard_load<Tin>(src + v), kLog2e, rs.nc));
    shard_store(dst + v, d);
  }
}

hipError_t launch_shard_rows(const void* logits, void* dlogits, grpo_dtype dt, int64_t T, int64_t V, int64_t ld,
                             int64_t v_begin, const grpo_vocab_stats* stats, int n_shards, const TokenArgs& tok,
                             hipStream_t s) {
  if (T <= 0) return hipSuccess;
  ShardArgs a;
  a.logits = logits;
  a.dlogits = dlogits;
  a.ld = ld;
  a.V = V;
  a.v_begin = v_begin;
  a.T = (int)T;
  a.n_shards = n_shards;
  a.stats = stats;
  a.tok = tok;
  const int epv = (dt == GRPO_BF16) ? 8 : 4;
  const bool vec = V % epv == 0 && ld % epv == 0 && aligned(logits, 16) && aligned(dlogits, 16);
  const dim3 grid((unsigned)T);
  if (vec && dt == GRPO_BF16) hipLaunchKernelGGL((k_shard_rows_vec<uint16_t, 512, 5>), grid, dim3(512), 0, s, a);
  else if (vec) hipLaunchKernelGGL((k_shard_rows_vec<float, 512, 5>), grid, dim3(512), 0, s, a);
  else if (dt == GRPO_BF16) hipLaunchKernelGGL(k_shard_rows_generic<uint16_t>, grid, dim3(256), 0, s, a);
  else hipLaunchKernelGGL(k_shard_rows_generic<float>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace grpo

using namespace grpo;

extern "C" int grpo_loss_fwd_bwd_vocab_shard(const void* logits, int32_t dtype, int64_t T, int64_t V_shard, int64_t ld,
                                             int64_t v_begin, int64_t V_total, const grpo_vocab_stats* stats,
                                             int32_t n_shards, const int32_t* actions, const float* behave_logp,
                                             const float* prox_logp, const float* adv, const grpo_segments* seg,
                                             const grpo_loss_params* p, double* loss_out, void* dlogits,
                                             grpo_aux* aux, void* ws, size_t ws_bytes, hipStream_t s) {
  int st = check_loss_common(T, actions, behave_logp, adv, seg, p, loss_out);
  if (st != GRPO_OK) return st;
  if (dtype != GRPO_BF16 && dtype != GRPO_F32) return GRPO_ERR_DTYPE;
  const grpo_dtype dt = static_cast<grpo_dtype>(dtype);
  // V_shard <= V_total < 2^31 is established before v_begin + V_shard is formed
  if (V_shard < 1 || ld < V_shard || v_begin < 0 || V_total < 1 || V_total >= ((int64_t)1 << 31) ||
      V_shard > V_total || v_begin > V_total - V_shard || n_shards < 1 || n_shards > 65536)
    return GRPO_ERR_SHAPE;
  if (T > 0 && (!logits || !stats)) return GRPO_ERR_ARG;
  const size_t esz = (dt == GRPO_BF16) ? 2 : 4;
  if (!aligned(logits, esz) || !aligned(dlogits, esz) || !aligned(stats, 8)) return GRPO_ERR_ALIGN;
  const LossWs L = loss_ws_layout(T, seg->n_traj);
  if (!ws || ws_bytes < L.total) return GRPO_ERR_WORKSPACE;
  if (!aligned(ws, kAlign)) return GRPO_ERR_ALIGN;
  char* w = static_cast<char*>(ws);

  if (launch_segments(seg, T, ld, actions, adv, p, w, L, aux, s) != hipSuccess) return GRPO_ERR_HIP;
  if (T > 0) {
    const TokenArgs tok = make_token_args(V_total, actions, behave_logp, prox_logp, adv, p, w, L, aux);
    const bool timed = aux && aux->hot_begin && aux->hot_end;
    if (timed && hipEventRecord(aux->hot_begin, s) != hipSuccess) return GRPO_ERR_HIP;
    if (launch_shard_rows(logits, dlogits, dt, T, V_shard, ld, v_begin, stats, n_shards, tok, s) != hipSuccess)
      return GRPO_ERR_HIP;
    if (timed && hipEventRecord(aux->hot_end, s) != hipSuccess) return GRPO_ERR_HIP;
  }
  if (launch_reduce(T, seg->n_traj, w, L, loss_out, aux, s) != hipSuccess) return GRPO_ERR_HIP;
  return GRPO_OK;
}
