// The fused LM-head path: the GRPO loss of Eq. 1 (dual clip of Eq. 2) from the
// final hidden states h [T, H] and the LM-head weight W [H, V], with the logits
// z = h W formed on the matrix cores and never stored whole.
//
//   pass 1  z tiles = h W           -> per (row, 256-column tile) max and sum exp,
//                                      and the action logit
//   rows    combine the partials    -> lse, log-prob, token epilogue, dlogits scale
//   pass 2  for each vocabulary chunk c of `vocab_chunk` columns:
//             z_c = h W_c (recomputed), D_c = g (softmax - onehot) in bf16,
//             stored as D_c [Tp, C] and its transpose D_c^T [C, Tp]
//             dhidden += D_c W_c^T       (fp32 accumulator, bf16 at the end)
//             dW[:, c] = h^T D_c
// Every product is one GEMM core (gemm.h) with both operands K-contiguous
// (C[m, n] = sum_k A[m, k] B[n, k]); W and h are transposed once so that this
// holds for all four.  256 x 256 tiles, 8 waves, v_mfma_f32_32x32x16_bf16.
#include <hip/hip_runtime.h>
#include <math.h>

#include "device.h"
#include "gemm.h"
#include "launch.h"

namespace grpo {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

typedef GemmCfg<256, 256, 64, 2, 4> LmCfg;  // BM, BN, BK, waves in M, waves in N
constexpr int TILE = 256;                   // BM = BN

// Shared memory of every GEMM kernel: the mainloop's double-buffered slabs; the
// epilogues reuse it once the mainloop's final barrier has passed.
struct GemmSmem {
  uint16_t a[2 * LmCfg::BM * LmCfg::LDK];
  uint16_t b[2 * LmCfg::BN * LmCfg::LDK];
};

__device__ __forceinline__ int tiles_of(int n) { return (n + TILE - 1) / TILE; }

// ---- pass 1: per-tile (max, sum exp) of every row, and the action logit ---------
struct PartialArgs {
  GemmArgs g;               // A = h [T, H], B = W^T [V, H]
  const int32_t* actions;   // [T]
  float2* part;             // [T, n_tiles] (max, sum exp over the tile's columns)
  float* za;                // [T] action logit
  int n_tiles;
};

__global__ __launch_bounds__(LmCfg::NT) void k_lm_partial(const PartialArgs p) {
  __shared__ __attribute__((aligned(16))) GemmSmem sm;
  __shared__ int sh_act[TILE];
  int tm, tn;
  if (!gemm_tile_of(blockIdx.x, gridDim.x, tiles_of(p.g.M), tiles_of(p.g.N), tm, tn)) return;
  const int m0 = tm * TILE, n0 = tn * TILE;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / LmCfg::WGN, wn = wave % LmCfg::WGN;
  if (tid < TILE) sh_act[tid] = (m0 + tid < p.g.M) ? p.actions[m0 + tid] : -1;
  g_f32x16 acc[LmCfg::IB][LmCfg::JB];
  gemm_mainloop<LmCfg>(p.g, m0, n0, acc, sm.a, sm.b);  // ends with a barrier: sh_act visible, slabs free
  float* sh_m = reinterpret_cast<float*>(sm.a);       // [WGN][TILE]
  float* sh_s = sh_m + LmCfg::WGN * TILE;              // [WGN][TILE]
#pragma unroll
  for (int i = 0; i < LmCfg::IB; ++i) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = gemm_row<LmCfg>(wm, i, r, lane);
      const int act = sh_act[row];
      float v[LmCfg::JB];
      float m = -INFINITY;
#pragma unroll
      for (int j = 0; j < LmCfg::JB; ++j) {
        const int c = n0 + gemm_col<LmCfg>(wn, j, lane);
        v[j] = (c < p.g.N) ? acc[i][j][r] : -INFINITY;
        if (act == c) p.za[m0 + row] = v[j];
        m = fmaxf(m, v[j]);
      }
#pragma unroll
      for (int o = 16; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 64));  // within the 32-lane half
      const float nm = (m == -INFINITY) ? 0.f : -m * kLog2e;
      float s = 0.f;
#pragma unroll
      for (int j = 0; j < LmCfg::JB; ++j) s += __builtin_amdgcn_exp2f(fmaf(v[j], kLog2e, nm));
#pragma unroll
      for (int o = 16; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
      if ((lane & 31) == 0) {
        sh_m[wn * TILE + row] = m;
        sh_s[wn * TILE + row] = s;
      }
    }
  }
  __syncthreads();
  if (tid < TILE && m0 + tid < p.g.M) {
    float M = -INFINITY;
#pragma unroll
    for (int q = 0; q < LmCfg::WGN; ++q) M = fmaxf(M, sh_m[q * TILE + tid]);
    float S = 0.f;
    if (M != -INFINITY)
#pragma unroll
      for (int q = 0; q < LmCfg::WGN; ++q)
        S += sh_s[q * TILE + tid] * __builtin_amdgcn_exp2f((sh_m[q * TILE + tid] - M) * kLog2e);
    p.part[(int64_t)(m0 + tid) * p.n_tiles + tn] = make_float2(M, S);
  }
}

// ---- combine: lse, log-prob and the token epilogue, one workgroup per row --------
struct CombineArgs {
  TokenArgs tok;
  const float2* part;
  const float* za;
  RowScale* rs;  // [Tp]; rows >= T get the zero scale
  int T, n_tiles;
};

__global__ __launch_bounds__(256) void k_lm_combine(const CombineArgs a) {
  __shared__ float sh_m[4];
  __shared__ double sh_s[4];
  const int t = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  if (t >= a.T) {
    if (tid == 0) a.rs[t] = RowScale{-INFINITY, 1.f, 0.f, -1};
    return;
  }
  const float2* pr = a.part + (int64_t)t * a.n_tiles;
  float m = -INFINITY;
  for (int j = tid; j < a.n_tiles; j += 256) m = fmaxf(m, pr[j].x);
  m = wave_max(m);
  if (lane == 0) sh_m[wv] = m;
  __syncthreads();
  const float M = fmaxf(fmaxf(sh_m[0], sh_m[1]), fmaxf(sh_m[2], sh_m[3]));
  double s = 0.0;
  if (M != -INFINITY)
    for (int j = tid; j < a.n_tiles; j += 256) {
      const float2 q = pr[j];
      if (q.x != -INFINITY) s += (double)q.y * (double)__builtin_amdgcn_exp2f((q.x - M) * kLog2e);
    }
  s = wave_sum(s);
  if (lane == 0) sh_s[wv] = s;
  __syncthreads();
  if (tid == 0) {
    const double S = sh_s[0] + sh_s[1] + sh_s[2] + sh_s[3];
    const TokenIn in = token_load(a.tok, t);
    const bool ok = in.act >= 0 && (int64_t)in.act < a.tok.V;
    a.rs[t] = token_finish(a.tok, t, in, (double)M + log(S), ok ? (double)a.za[t] : 0.0);
  }
}

// ---- pass 2a: recompute z_c, form D_c = g (softmax - onehot), store D_c and D_c^T --
struct DlogitsArgs {
  GemmArgs g;            // A = h [T, H] (M = Tp), B = W^T rows of the chunk [Cw, H]
  const RowScale* rs;    // [Tp]
  uint16_t* D;           // [Tp, C]
  uint16_t* DT;          // [C, Tp]
  int c0, C, Tp;
};

__global__ __launch_bounds__(LmCfg::NT) void k_lm_dlogits(const DlogitsArgs p) {
  __shared__ __attribute__((aligned(16))) GemmSmem sm;
  __shared__ RowScale sh_rs[TILE];
  int tm, tn;
  if (!gemm_tile_of(blockIdx.x, gridDim.x, tiles_of(p.Tp), tiles_of(p.g.N), tm, tn)) return;
  const int m0 = tm * TILE, n0 = tn * TILE;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / LmCfg::WGN, wn = wave % LmCfg::WGN;
  if (tid < TILE) sh_rs[tid] = p.rs[m0 + tid];  // m0 + tid < Tp: Tp is a multiple of the tile
  g_f32x16 acc[LmCfg::IB][LmCfg::JB];
  gemm_mainloop<LmCfg>(p.g, m0, n0, acc, sm.a, sm.b);
#pragma unroll
  for (int i = 0; i < LmCfg::IB; ++i) {
#pragma unroll
    for (int j = 0; j < LmCfg::JB; ++j) {
      const int n = n0 + gemm_col<LmCfg>(wn, j, lane);
      if (n >= p.g.N) continue;
      const int vcol = p.c0 + n;
#pragma unroll
      for (int rq = 0; rq < 4; ++rq) {  // four consecutive rows per register quad
        float d[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = rq * 4 + e;
          const RowScale rs = sh_rs[gemm_row<LmCfg>(wm, i, r, lane)];
          d[e] = (vcol == rs.act) ? rs.d_a : rs.sign * __builtin_amdgcn_exp2f(fmaf(acc[i][j][r], kLog2e, rs.nc));
        }
        const int row0 = m0 + gemm_row<LmCfg>(wm, i, rq * 4, lane);
        u32x2 pk = {pack_bf16(d[0], d[1]), pack_bf16(d[2], d[3])};
        *reinterpret_cast<u32x2*>(p.DT + (int64_t)n * p.Tp + row0) = pk;
#pragma unroll
        for (int e = 0; e < 4; ++e) p.D[(int64_t)(row0 + e) * p.C + n] = (uint16_t)(pack_bf16(d[e], 0.f) & 0xffffu);
      }
    }
  }
}

// ---- pass 2b: dhidden += D_c W_c^T --------------------------------------------------
struct DhArgs {
  GemmArgs g;        // A = D_c [Tp, C] (M = T, K = Cw), B = W[:, chunk] as [H, Cw] with ldb = V
  float* acc;        // [Tp, H] fp32 accumulator (unused with a single chunk)
  uint16_t* dh;      // [T, H] bf16 output
  int first, last;
};

__global__ __launch_bounds__(LmCfg::NT) void k_lm_dh(const DhArgs p) {
  __shared__ __attribute__((aligned(16))) GemmSmem sm;
  int tm, tn;
  if (!gemm_tile_of(blockIdx.x, gridDim.x, tiles_of(p.g.M), tiles_of(p.g.N), tm, tn)) return;
  const int m0 = tm * TILE, n0 = tn * TILE;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / LmCfg::WGN, wn = wave % LmCfg::WGN;
  g_f32x16 acc[LmCfg::IB][LmCfg::JB];
  gemm_mainloop<LmCfg>(p.g, m0, n0, acc, sm.a, sm.b);
  const int H = p.g.N;
#pragma unroll
  for (int i = 0; i < LmCfg::IB; ++i)
#pragma unroll
    for (int j = 0; j < LmCfg::JB; ++j) {
      const int n = n0 + gemm_col<LmCfg>(wn, j, lane);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = m0 + gemm_row<LmCfg>(wm, i, r, lane);
        if (m >= p.g.M || n >= H) continue;
        const int64_t o = (int64_t)m * H + n;
        float v = acc[i][j][r];
        if (!p.first) v += p.acc[o];
        if (p.last) p.dh[o] = (uint16_t)(pack_bf16(v, 0.f) & 0xffffu);
        else p.acc[o] = v;
      }
    }
}

// ---- pass 2c: dW[:, chunk] = h^T D_c ----------------------------------------------
struct DwArgs {
  GemmArgs g;     // A = h^T [H, Tp], B = D_c^T [Cw, Tp], K = Tp
  float* dw;      // [H, V]
  int64_t V;
  int c0, accumulate;
};

__global__ __launch_bounds__(LmCfg::NT) void k_lm_dw(const DwArgs p) {
  __shared__ __attribute__((aligned(16))) GemmSmem sm;
  int tm, tn;
  if (!gemm_tile_of(blockIdx.x, gridDim.x, tiles_of(p.g.M), tiles_of(p.g.N), tm, tn)) return;
  const int m0 = tm * TILE, n0 = tn * TILE;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / LmCfg::WGN, wn = wave % LmCfg::WGN;
  g_f32x16 acc[LmCfg::IB][LmCfg::JB];
  gemm_mainloop<LmCfg>(p.g, m0, n0, acc, sm.a, sm.b);
#pragma unroll
  for (int i = 0; i < LmCfg::IB; ++i)
#pragma unroll
    for (int j = 0; j < LmCfg::JB; ++j) {
      const int n = n0 + gemm_col<LmCfg>(wn, j, lane);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = m0 + gemm_row<LmCfg>(wm, i, r, lane);
        if (m >= p.g.M || n >= p.g.N) continue;
        float* o = p.dw + (int64_t)m * p.V + p.c0 + n;
        *o = p.accumulate ? *o + acc[i][j][r] : acc[i][j][r];
      }
    }
}

// ---- bf16 transpose: dst[c][r] = src[r][c] for r < R, 0 for R <= r < Rp ------------
__global__ __launch_bounds__(256) void k_transpose_bf16(const uint16_t* __restrict__ src, int64_t lds_, int R,
                                                        int Cc, uint16_t* __restrict__ dst, int64_t ldd, int Rp) {
  __shared__ uint16_t tile[64][64 + 2];
  const int c0 = blockIdx.x * 64, r0 = blockIdx.y * 64;
  const int tid = threadIdx.x, ty = tid >> 3, tx = tid & 7;
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int rr = ty + 32 * q, r = r0 + rr, c = c0 + tx * 8;
    u32x4 v = {0u, 0u, 0u, 0u};
    if (r < R && c < Cc) v = *reinterpret_cast<const u32x4*>(src + (int64_t)r * lds_ + c);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      tile[rr][tx * 8 + 2 * e] = (uint16_t)(v[e] & 0xffffu);
      tile[rr][tx * 8 + 2 * e + 1] = (uint16_t)(v[e] >> 16);
    }
  }
  __syncthreads();
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int cc = ty + 32 * q, c = c0 + cc, r = r0 + tx * 8;
    if (c >= Cc || r >= Rp) continue;
    u32x4 v;
#pragma unroll
    for (int e = 0; e < 4; ++e)
      v[e] = (uint32_t)tile[tx * 8 + 2 * e][cc] | ((uint32_t)tile[tx * 8 + 2 * e + 1][cc] << 16);
    *reinterpret_cast<u32x4*>(dst + (int64_t)c * ldd + r) = v;
  }
}

__global__ void k_fill_f32(float* p, int64_t n, float v) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

// ---- workspace --------------------------------------------------------------------
struct LmWs {
  LossWs loss;
  size_t wt, ht, part, za, rs, d, dt, acc, total;
  int64_t Tp;
  int n_tiles, C;
};

static LmWs lm_ws_layout(int64_t T, int64_t H, int64_t V, int32_t C, int32_t n_traj) {
  LmWs l;
  l.loss = loss_ws_layout(T, n_traj);
  l.Tp = (T + TILE - 1) / TILE * TILE;
  l.n_tiles = (int)((V + TILE - 1) / TILE);
  l.C = C;
  const int64_t n_chunks = (V + C - 1) / C;
  size_t o = l.loss.total;
  l.wt = o;   o = align_up(o + sizeof(uint16_t) * (size_t)(V * H));
  l.ht = o;   o = align_up(o + sizeof(uint16_t) * (size_t)(H * l.Tp));
  l.part = o; o = align_up(o + sizeof(float2) * (size_t)(T * l.n_tiles));
  l.za = o;   o = align_up(o + sizeof(float) * (size_t)T);
  l.rs = o;   o = align_up(o + sizeof(RowScale) * (size_t)l.Tp);
  l.d = o;    o = align_up(o + sizeof(uint16_t) * (size_t)(l.Tp * C));
  l.dt = o;   o = align_up(o + sizeof(uint16_t) * (size_t)(l.Tp * C));
  l.acc = o;  o = align_up(o + (n_chunks > 1 ? sizeof(float) * (size_t)(l.Tp * H) : 0));
  l.total = o;
  return l;
}

// A multiple of 8 workgroups covering every tile of an M x N output (see gemm_tile_of).
static dim3 gemm_grid(int64_t M, int64_t N) {
  const int64_t tiles = ((M + TILE - 1) / TILE) * ((N + TILE - 1) / TILE);
  return dim3((unsigned)((tiles + 7) / 8 * 8));
}

}  // namespace grpo

using namespace grpo;

extern "C" size_t fused_lmhead_workspace_bytes(int64_t T, int64_t H, int64_t V, int32_t vocab_chunk, int32_t n_traj) {
  if (T < 0 || H < 1 || V < 1 || vocab_chunk < 1 || n_traj < 1) return 0;
  return lm_ws_layout(T, H, V, vocab_chunk, n_traj).total;
}

extern "C" int fused_lmhead_grpo(const void* hidden, const void* w_lm, int64_t T, int64_t H, int64_t V,
                                 int32_t vocab_chunk, const int32_t* actions, const float* behave_logp,
                                 const float* prox_logp, const float* adv, const grpo_segments* seg,
                                 const grpo_loss_params* p, double* loss_out, void* dhidden, float* dw_lm,
                                 int32_t accumulate_dw, grpo_aux* aux, void* ws, size_t ws_bytes, hipStream_t s) {
  int st = check_loss_common(T, actions, behave_logp, adv, seg, p, loss_out);
  if (st != GRPO_OK) return st;
  if (!w_lm || !dw_lm || (T > 0 && (!hidden || !dhidden))) return GRPO_ERR_ARG;
  if (H < 64 || H % 64 != 0 || H >= (1 << 30)) return GRPO_ERR_SHAPE;
  if (V < 8 || V % 8 != 0 || V >= ((int64_t)1 << 31)) return GRPO_ERR_SHAPE;
  if (vocab_chunk < 256 || vocab_chunk % 256 != 0) return GRPO_ERR_SHAPE;
  if (!aligned(hidden, 16) || !aligned(w_lm, 16) || !aligned(dhidden, 16) || !aligned(dw_lm, 16))
    return GRPO_ERR_ALIGN;
  const LmWs L = lm_ws_layout(T, H, V, vocab_chunk, seg->n_traj);
  if (!ws || ws_bytes < L.total) return GRPO_ERR_WORKSPACE;
  if (!aligned(ws, kAlign)) return GRPO_ERR_ALIGN;
  char* w = static_cast<char*>(ws);
  const uint16_t* h16 = static_cast<const uint16_t*>(hidden);
  const uint16_t* W16 = static_cast<const uint16_t*>(w_lm);
  uint16_t* WT = reinterpret_cast<uint16_t*>(w + L.wt);
  uint16_t* hT = reinterpret_cast<uint16_t*>(w + L.ht);
  float2* part = reinterpret_cast<float2*>(w + L.part);
  float* za = reinterpret_cast<float*>(w + L.za);
  RowScale* rs = reinterpret_cast<RowScale*>(w + L.rs);
  uint16_t* D = reinterpret_cast<uint16_t*>(w + L.d);
  uint16_t* DT = reinterpret_cast<uint16_t*>(w + L.dt);
  float* acc = reinterpret_cast<float*>(w + L.acc);
  const int C = vocab_chunk;
  const int Tp = (int)L.Tp;

  if (launch_segments(seg, T, V, actions, adv, p, w, L.loss, aux, s) != hipSuccess) return GRPO_ERR_HIP;
  if (T == 0) {
    if (!accumulate_dw) hipLaunchKernelGGL(k_fill_f32, dim3(1024), dim3(256), 0, s, dw_lm, H * V, 0.f);
    if (hipGetLastError() != hipSuccess) return GRPO_ERR_HIP;
    return launch_reduce(T, seg->n_traj, w, L.loss, loss_out, aux, s) == hipSuccess ? GRPO_OK : GRPO_ERR_HIP;
  }
  // W^T [V, H] and h^T [H, Tp] (zero columns T..Tp)
  hipLaunchKernelGGL(k_transpose_bf16, dim3((unsigned)((V + 63) / 64), (unsigned)((H + 63) / 64)), dim3(256), 0, s,
                     W16, V, (int)H, (int)V, WT, H, (int)H);
  hipLaunchKernelGGL(k_transpose_bf16, dim3((unsigned)((H + 63) / 64), (unsigned)((Tp + 63) / 64)), dim3(256), 0, s,
                     h16, H, (int)T, (int)H, hT, (int64_t)Tp, Tp);
  if (hipGetLastError() != hipSuccess) return GRPO_ERR_HIP;

  const bool timed = aux && aux->hot_begin && aux->hot_end;
  if (timed && hipEventRecord(aux->hot_begin, s) != hipSuccess) return GRPO_ERR_HIP;
  // pass 1
  PartialArgs pa;
  pa.g = GemmArgs{h16, WT, H, H, (int)T, (int)V, (int)H};
  pa.actions = actions;
  pa.part = part;
  pa.za = za;
  pa.n_tiles = L.n_tiles;
  hipLaunchKernelGGL(k_lm_partial, gemm_grid(T, V), dim3(LmCfg::NT), 0, s, pa);
  // combine
  CombineArgs ca;
  ca.tok = make_token_args(V, actions, behave_logp, prox_logp, adv, p, w, L.loss, aux);
  ca.part = part;
  ca.za = za;
  ca.rs = rs;
  ca.T = (int)T;
  ca.n_tiles = L.n_tiles;
  hipLaunchKernelGGL(k_lm_combine, dim3((unsigned)Tp), dim3(256), 0, s, ca);
  if (hipGetLastError() != hipSuccess) return GRPO_ERR_HIP;
  // pass 2, chunk by chunk
  const int n_chunks = (int)((V + C - 1) / C);
  for (int c = 0; c < n_chunks; ++c) {
    const int c0 = c * C;
    const int Cw = (int)((V - c0) < C ? (V - c0) : C);
    DlogitsArgs da;
    da.g = GemmArgs{h16, WT + (int64_t)c0 * H, H, H, (int)T, Cw, (int)H};
    da.rs = rs;
    da.D = D;
    da.DT = DT;
    da.c0 = c0;
    da.C = C;
    da.Tp = Tp;
    hipLaunchKernelGGL(k_lm_dlogits, gemm_grid(Tp, Cw), dim3(LmCfg::NT), 0, s, da);
    DhArgs ha;
    ha.g = GemmArgs{D, W16 + c0, C, V, (int)T, (int)H, Cw};
    ha.acc = acc;
    ha.dh = static_cast<uint16_t*>(dhidden);
    ha.first = (c == 0);
    ha.last = (c == n_chunks - 1);
    hipLaunchKernelGGL(k_lm_dh, gemm_grid(T, H), dim3(LmCfg::NT), 0, s, ha);
    DwArgs wa;
    wa.g = GemmArgs{hT, DT, Tp, Tp, (int)H, Cw, Tp};
    wa.dw = dw_lm;
    wa.V = V;
    wa.c0 = c0;
    wa.accumulate = accumulate_dw;
    hipLaunchKernelGGL(k_lm_dw, gemm_grid(H, Cw), dim3(LmCfg::NT), 0, s, wa);
    if (hipGetLastError() != hipSuccess) return GRPO_ERR_HIP;
  }
  if (timed && hipEventRecord(aux->hot_end, s) != hipSuccess) return GRPO_ERR_HIP;
  if (launch_reduce(T, seg->n_traj, w, L.loss, loss_out, aux, s) != hipSuccess) return GRPO_ERR_HIP;
  return GRPO_OK;
}
