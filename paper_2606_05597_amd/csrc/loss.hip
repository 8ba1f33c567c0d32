// The logits path: streaming log-softmax + gather, the per-token surrogate of
// Eq. 1 (dual clip of Eq. 2), and dlogits, one workgroup per token row.
//
// Hot kernel (k_rows_resident): the row is read from HBM exactly once into
// registers with 16-byte loads (the wavefront covers 1 KiB contiguous per
// instruction), reduced to (max, sum exp) per thread, combined across the
// workgroup, and dlogits are formed from the same registers and written once.
// Bytes per token: V*s read + V*s written + a few scalars.
#include <hip/hip_runtime.h>
#include <math.h>

#include "device.h"
#include "launch.h"

namespace grpo {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Row-pass arguments: the logits, the dlogits destination and the token epilogue.
struct RowArgs {
  const void* logits;
  void* dlogits;  // nullable: forward only
  TokenArgs tok;
};

template <typename Tin>
__device__ __forceinline__ float load_elem(const Tin* p);
template <>
__device__ __forceinline__ float load_elem<float>(const float* p) { return *p; }
template <>
__device__ __forceinline__ float load_elem<uint16_t>(const uint16_t* p) { return bf16_to_f32(*p); }

// The epilogue of one row once its max M and S = sum exp(z - M) are known.
template <typename Tin>
__device__ RowScale row_epilogue(const RowArgs& a, int t, const Tin* row, double M, double S) {
  const int act = a.tok.actions[t];
  const bool ok = act >= 0 && (int64_t)act < a.tok.V;
  const double z_a = ok ? (double)load_elem<Tin>(row + act) : 0.0;
  return token_finish(a.tok, t, act, M + log(S), z_a);
}

// ---- register-resident row kernel -------------------------------------------
// NT threads per row, NV 16-byte vectors per thread: V <= NT*NV*EPV.  Rows are
// 16-byte aligned and V is a multiple of EPV (checked on the host).
template <typename Tin, int NT, int NV>
__global__ __launch_bounds__(NT) void k_rows_resident(const RowArgs a) {
  constexpr int EPV = 16 / sizeof(Tin);  // elements per vector: 8 bf16 or 4 fp32
  constexpr int NW = NT / 64;
  constexpr bool kBF16 = sizeof(Tin) == 2;
  __shared__ float sh_m[NW];
  __shared__ double sh_s[NW];
  __shared__ RowScale sh_rs;

  const int t = blockIdx.x;
  const int tid = threadIdx.x;
  const int nvec = (int)(a.tok.V / EPV);
  const Tin* row = static_cast<const Tin*>(a.logits) + (int64_t)t * a.tok.ld;
  const u32x4* src = reinterpret_cast<const u32x4*>(row);

  u32x4 buf[NV];
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int vi = j * NT + tid;
    if (vi < nvec) buf[j] = __builtin_nontemporal_load(src + vi);
  }

  // pass A: this thread's max
  float m = -INFINITY;
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    if (j * NT + tid < nvec) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if constexpr (kBF16) m = fmaxf(m, fmaxf(bf16_hi(buf[j][q]), bf16_lo(buf[j][q])));
        else m = fmaxf(m, __uint_as_float(buf[j][q]));
      }
    }
  }
  // pass B: this thread's sum of exp(z - m)
  const float nmb = (m == -INFINITY) ? 0.f : -m * kLog2e;
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    if (j * NT + tid < nvec) {
      float part = 0.f;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if constexpr (kBF16) {
          part += __builtin_amdgcn_exp2f(fmaf(bf16_lo(buf[j][q]), kLog2e, nmb)) +
                  __builtin_amdgcn_exp2f(fmaf(bf16_hi(buf[j][q]), kLog2e, nmb));
        } else {
          part += __builtin_amdgcn_exp2f(fmaf(__uint_as_float(buf[j][q]), kLog2e, nmb));
        }
      }
      s += part;
    }
  }
  // combine (m, s) over the wave, then over the workgroup
  const float mw = wave_max(m);
  const double sw = wave_sum((m == -INFINITY) ? 0.0 : (double)s * exp2((double)((m - mw) * kLog2e)));
  const int lane = tid & 63, wv = tid >> 6;
  if (lane == 0) {
    sh_m[wv] = mw;
    sh_s[wv] = sw;
  }
  __syncthreads();
  if (tid == 0) {
    float M = -INFINITY;
#pragma unroll
    for (int q = 0; q < NW; ++q) M = fmaxf(M, sh_m[q]);
    double S = 0.0;
#pragma unroll
    for (int q = 0; q < NW; ++q)
      if (sh_m[q] != -INFINITY) S += sh_s[q] * exp((double)sh_m[q] - (double)M);
    sh_rs = row_epilogue<Tin>(a, t, row, (double)M, S);
  }
  __syncthreads();
  if (!a.dlogits) return;

  // pass C: dlogits from the registers, written once
  const RowScale rs = sh_rs;
  const int act_vec = rs.act >= 0 ? rs.act / EPV : -1;
  const int act_lane = rs.act >= 0 ? rs.act % EPV : 0;
  u32x4* dst = reinterpret_cast<u32x4*>(static_cast<Tin*>(a.dlogits) + (int64_t)t * a.tok.ld);
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int vi = j * NT + tid;
    if (vi < nvec) {
      u32x4 o;
      if constexpr (kBF16) {
        float d[8];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          d[2 * q] = rs.sign * __builtin_amdgcn_exp2f(fmaf(bf16_lo(buf[j][q]), kLog2e, rs.nc));
          d[2 * q + 1] = rs.sign * __builtin_amdgcn_exp2f(fmaf(bf16_hi(buf[j][q]), kLog2e, rs.nc));
        }
        if (vi == act_vec) {
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (e == act_lane) d[e] = rs.d_a;
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) o[q] = pack_bf16(d[2 * q], d[2 * q + 1]);
      } else {
        float d[4];
#pragma unroll
        for (int q = 0; q < 4; ++q)
          d[q] = rs.sign * __builtin_amdgcn_exp2f(fmaf(__uint_as_float(buf[j][q]), kLog2e, rs.nc));
        if (vi == act_vec) {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (e == act_lane) d[e] = rs.d_a;
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) o[q] = __float_as_uint(d[q]);
      }
      __builtin_nontemporal_store(o, dst + vi);
    }
  }
}

// ---- generic row kernel ------------------------------------------------------
// Any V, ld and element alignment: element-wise loads, the row read three
// times (max, sum, dlogits).  Used when the resident kernel does not apply.
template <typename Tin>
__global__ __launch_bounds__(256) void k_rows_generic(const RowArgs a) {
  constexpr int NT = 256, NW = NT / 64;
  __shared__ float sh_m[NW];
  __shared__ double sh_s[NW];
  __shared__ RowScale sh_rs;
  const int t = blockIdx.x, tid = threadIdx.x;
  const Tin* row = static_cast<const Tin*>(a.logits) + (int64_t)t * a.tok.ld;
  float m = -INFINITY;
  for (int64_t v = tid; v < a.tok.V; v += NT) m = fmaxf(m, load_elem<Tin>(row + v));
  const float mw = wave_max(m);
  const int lane = tid & 63, wv = tid >> 6;
  if (lane == 0) sh_m[wv] = mw;
  __syncthreads();
  float M = -INFINITY;
  for (int q = 0; q < NW; ++q) M = fmaxf(M, sh_m[q]);
  const float nmb = (M == -INFINITY) ? 0.f : -M * kLog2e;
  double s = 0.0;
  for (int64_t v = tid; v < a.tok.V; v += NT) s += (double)__builtin_amdgcn_exp2f(fmaf(load_elem<Tin>(row + v), kLog2e, nmb));
  s = wave_sum(s);
  if (lane == 0) sh_s[wv] = s;
  __syncthreads();
  if (tid == 0) {
    double S = 0.0;
    for (int q = 0; q < NW; ++q) S += sh_s[q];
    sh_rs = row_epilogue<Tin>(a, t, row, (double)M, S);
  }
  __syncthreads();
  if (!a.dlogits) return;
  const RowScale rs = sh_rs;
  Tin* drow = static_cast<Tin*>(a.dlogits) + (int64_t)t * a.tok.ld;
  for (int64_t v = tid; v < a.tok.V; v += NT) {
    float d = (v == rs.act) ? rs.d_a : rs.sign * __builtin_amdgcn_exp2f(fmaf(load_elem<Tin>(row + v), kLog2e, rs.nc));
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

// Ordered by NT, then NV; the first that holds the row is used.
static const Variant kVariants[] = {
    GRPO_VARIANT(64, 1),    GRPO_VARIANT(64, 2),    GRPO_VARIANT(64, 4),    GRPO_VARIANT(64, 8),
    GRPO_VARIANT(256, 4),   GRPO_VARIANT(256, 8),   GRPO_VARIANT(256, 12),  GRPO_VARIANT(256, 16),
    GRPO_VARIANT(256, 20),  GRPO_VARIANT(256, 24),  GRPO_VARIANT(1024, 8),  GRPO_VARIANT(1024, 12),
    GRPO_VARIANT(1024, 16), GRPO_VARIANT(1024, 19),
};  // 1024 threads x 19 vectors (127 VGPRs) is the largest that does not spill

static RowKernel pick_row_kernel(grpo_dtype dt, int64_t V, int64_t ld, const void* logits, const void* dlogits,
                                 int* nt_out) {
  const int epv = (dt == GRPO_BF16) ? 8 : 4;
  const bool vec_ok = (V % epv == 0) && (ld % epv == 0) && aligned(logits, 16) && aligned(dlogits, 16);
  if (vec_ok) {
    const int64_t nvec = V / epv;
    for (const Variant& v : kVariants) {
      if ((int64_t)v.nt * v.nv >= nvec) {
        *nt_out = v.nt;
        return dt == GRPO_BF16 ? v.bf16 : v.f32;
      }
    }
  }
  *nt_out = 256;
  return dt == GRPO_BF16 ? k_rows_generic<uint16_t> : k_rows_generic<float>;
}

}  // namespace grpo

using namespace grpo;

extern "C" size_t grpo_loss_workspace_bytes(int64_t T, int32_t n_traj) {
  if (T < 0 || n_traj < 1) return 0;
  return loss_ws_layout(T, n_traj).total;
}

extern "C" int grpo_loss_fwd_bwd(const void* logits, grpo_dtype dt, int64_t T, int64_t V, int64_t ld,
                                 const int32_t* actions, const float* behave_logp, const float* prox_logp,
                                 const float* adv, const grpo_segments* seg, const grpo_loss_params* p,
                                 double* loss_out, void* dlogits, grpo_aux* aux, void* ws, size_t ws_bytes,
                                 hipStream_t s) {
  int st = check_loss_common(T, actions, behave_logp, adv, seg, p, loss_out);
  if (st != GRPO_OK) return st;
  if (dt != GRPO_BF16 && dt != GRPO_F32) return GRPO_ERR_DTYPE;
  if (T > 0 && !logits) return GRPO_ERR_ARG;
  if (V < 1 || ld < V) return GRPO_ERR_SHAPE;
  const size_t esz = (dt == GRPO_BF16) ? 2 : 4;
  if (!aligned(logits, esz) || !aligned(dlogits, esz)) return GRPO_ERR_ALIGN;
  const LossWs L = loss_ws_layout(T, seg->n_traj);
  if (!ws || ws_bytes < L.total) return GRPO_ERR_WORKSPACE;
  if (!aligned(ws, kAlign)) return GRPO_ERR_ALIGN;
  char* w = static_cast<char*>(ws);

  if (launch_segments(seg, T, p, w, L, aux ? aux->traj_tok_off : nullptr, s) != hipSuccess) return GRPO_ERR_HIP;
  if (T > 0) {
    RowArgs a;
    a.logits = logits;
    a.dlogits = dlogits;
    a.tok = make_token_args(V, ld, actions, behave_logp, prox_logp, adv, seg, p, w, L, aux);
    int nt = 256;
    RowKernel k = pick_row_kernel(dt, V, ld, logits, dlogits, &nt);
    const bool timed = aux && aux->hot_begin && aux->hot_end;
    if (timed && hipEventRecord(aux->hot_begin, s) != hipSuccess) return GRPO_ERR_HIP;
    hipLaunchKernelGGL(k, dim3((unsigned)T), dim3(nt), 0, s, a);
    if (hipGetLastError() != hipSuccess) return GRPO_ERR_HIP;
    if (timed && hipEventRecord(aux->hot_end, s) != hipSuccess) return GRPO_ERR_HIP;
  }
  if (launch_reduce(T, seg->n_traj, w, L, loss_out, aux, s) != hipSuccess) return GRPO_ERR_HIP;
  return GRPO_OK;
}
