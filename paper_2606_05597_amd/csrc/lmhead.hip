// The fused LM-head path: the GRPO loss of Eq. 1 (dual clip of Eq. 2) from the
// final hidden states h [T, H] and the LM-head weight W [H, V], with the logits
// z = h W formed on the matrix cores and never stored whole.
//
//   pass 1  z tiles = h W           -> per (row, 256-column tile) max and sum exp
//   rows    combine the partials    -> lse; the action logit h_t . W[:, a_t] in fp64;
//                                      log-prob, token epilogue, dlogits scale
//   pass 2  for each vocabulary chunk c of `vocab_chunk` columns:
//             z_c = h W_c (recomputed), D_c = g (softmax - onehot) in bf16,
//             stored as D_c (one half of a [Tp, 2C] pair buffer) and its transpose
//             D_c^T (one half of a [2C, Tp] pair buffer)
//           after every second chunk (and the last), in one launch:
//             dW[:, c-1..c] = h^T [D_c-1 D_c]
//             dhidden += [D_c-1 D_c] [W_c-1 W_c]^T   (fp32 accumulator, bf16 at the end)
// The token-blocked schedule (fused_lmhead_grpo_blocked) takes rows in blocks
// instead and keeps a block's logits, so the forward product is not recomputed:
//   per block of B rows:
//     z = h_block W  -> tile partials, and each logit's term exp(z - m) (m its row's
//                       maximum over the 256-column tile) as fp16 (HBM)
//     rows           combine, as above
//     D pass         stored terms -> D = g e^(m - lse) exp(z - m), D^T (bf16), a
//                    streaming pass with one multiply per logit
//     one launch     dhidden rows = D W^T (K = V, written once), then
//                    dW (+)= h_block^T D (K = B)
//   With a second stream, block b's D pass runs beside block b + 1's forward
//   product (one D-pass workgroup per CU next to the product's workgroup).
// Also here: a vocabulary shard's two calls (its per-token records from pass 1 on
// its columns; then, given every shard's records, pass 2 on its columns, with the
// logits formed again or kept from the first call), and the forward-only call
// (log-prob and entropy from tile partials that carry a third, entropy moment).
// Every product is one GEMM core (gemm.h) with both operands K-contiguous
// (C[m, n] = sum_k A[m, k] B[n, k]); W and h are transposed once so that this
// holds for all of them.  256 x 256 tiles, 8 waves, v_mfma_f32_32x32x16_bf16,
// slabs loaded straight into LDS.
#include <hip/hip_runtime.h>
#include <math.h>

#include <type_traits>

#include "device.h"
#include "gemm.h"
#include "launch.h"

namespace grpo {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// fp16 pairs: round-to-nearest-even pack of two fp32 values (v_cvt_pk_f16_f32), and the exact widening back.
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_f16(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){lo, hi}, f16x2));
}
__device__ __forceinline__ f32x2 unpack_f16(uint32_t w) {
  return __builtin_convertvector(__builtin_bit_cast(f16x2, w), f32x2);
}

typedef GemmCfg<256, 256, 2, 4> LmCfg;  // BM, BN, waves in M, waves in N
constexpr int TILE = 256;               // BM = BN

// Shared memory of every GEMM kernel: the mainloop's two slab buffers.  The
// epilogues reuse it once the mainloop's last barrier has passed (every wave has
// finished its LDS reads by then, and no DMA is left in flight).
struct GemmSmem {
  uint16_t s[2 * LmCfg::STAGE];
};

__device__ __forceinline__ int tiles_of(int n) { return (n + TILE - 1) / TILE; }

// ---- 16-lane DPP reductions ---------------------------------------------------------
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float x) {
  // every source lane of these patterns is valid, so bound_ctrl changes nothing; it
  // lets the move fold into the consuming max / add
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, true));
}
// Four steps give every lane of a 16-lane row the row's max (sum): swaps within
// quads, then across the halves of each 8-lane group (half mirror), then across the
// two 8-lane groups (mirror).
// DPP controls: quad_perm [1, 0, 3, 2] = 0xB1, quad_perm [2, 3, 0, 1] = 0x4E,
// row_half_mirror = 0x141, row_mirror = 0x140.
__device__ __forceinline__ float add_f32(float a, float b) { return a + b; }

// ---- pass 1: per-tile (max, sum exp) of every row ------------------------------------
struct PartialArgs {
  GemmArgs g;    // A = h [T, H], B = W^T [V, H]
  float2* part;  // [T, n_tiles] (max, sum exp over the tile's columns)
  int n_tiles;
  float* z;      // STORE_Z: the fp32 logits [tiles_of(M) * TILE, ldz], every tile stored whole
  int64_t ldz;   // a multiple of TILE, at least n_tiles * TILE
  float* part_t; // entropy partials [T, n_tiles]: sum over the tile of e^(z - m) (z - m), m the tile's max
  uint16_t* e16; // TERMS: every logit's term e = exp(z - m), m its row's max over the tile, fp16 [tiles_of(M) *
                 // TILE, ldz], every tile stored whole (0 past N)
};

// The forward product's epilogue: per (row, 256-column tile) the max m and sum exp(z - m) into part, and with ENT
// also sum exp(z - m) (z - m) into part_t (the entropy's second moment); with TERMS every logit's term exp(z - m)
// into p.e16 as fp16 (round to nearest even; the terms are <= 1, so the relative error is at most 2^-11 for terms
// >= 2^-14 and the absolute one at most 2^-25 below).  Columns past N are left out (their terms stored as 0).
template <bool ENT, bool TERMS = false>
__device__ __forceinline__ void lm_partial_epilogue(const PartialArgs& p, g_f32x16 (&acc)[LmCfg::IB][LmCfg::JB],
                                                    int m0, int n0, int tn, GemmSmem& sm);

// PACKED: B is W^T in the fragment-packed layout (gemm_mainloop_packed); the accumulators, and so every output,
// are bit-identical to the LDS-staged core's.  STORE_Z: the fp32 logits too; TERMS: the fp16 terms (p.e16).
template <bool STORE_Z, bool PACKED = false, bool TERMS = false>
__global__ __launch_bounds__(LmCfg::NT) void k_lm_partial(const PartialArgs p) {
  static_assert(!(STORE_Z && TERMS), "one kind of stored logits");
  __shared__ __attribute__((aligned(16))) GemmSmem sm;
  int tm, tn;
  if (!gemm_tile_of(blockIdx.x, gridDim.x, tiles_of(p.g.M), tiles_of(p.g.N), tm, tn)) return;
  const int m0 = tm * TILE, n0 = tn * TILE;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / LmCfg::WGN, wn = wave % LmCfg::WGN;
  g_f32x16 acc[LmCfg::IB][LmCfg::JB];
  if constexpr (PACKED) gemm_mainloop_packed<LmCfg>(p.g, m0, n0, acc, sm.s);
  else gemm_mainloop<LmCfg>(p.g, m0, n0, acc, sm.s);
  if constexpr (STORE_Z) {
    // Rows and columns past M and N hold zeros (their operand rows read as zero).  Accumulators 4g..4g+3 of a
    // lane are four consecutive rows of one column; a 4 x 4 transpose within each quad of lanes (two DPP
    // exchanges: lanes x ^ 1, then x ^ 2) leaves lane 4a + x with row x of the group and columns 4a..4a+3, so
    // each lane stores 16 bytes and one store instruction fills eight 128-byte row pieces.
    const int x = lane & 3;
    float* zt = p.z + (int64_t)m0 * p.ldz + n0 + wn * LmCfg::WTN + 4 * ((lane & 31) >> 2);
#pragma unroll
    for (int i = 0; i < LmCfg::IB; ++i)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        float* zr = zt + (int64_t)(wm * LmCfg::WTM + i * 32 + 8 * g + 4 * (lane >> 5) + x) * p.ldz;
#pragma unroll
        for (int j = 0; j < LmCfg::JB; ++j) {
          float v[4], t[4], o[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = acc[i][j][4 * g + e];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float q = dpp_f32<0xB1>(v[e ^ 1]);  // lane x ^ 1's accumulator e ^ 1
            t[e] = ((e ^ x) & 1) ? q : v[e];
          }
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float q = dpp_f32<0x4E>(t[e ^ 2]);  // lane x ^ 2's value e ^ 2
            o[e] = ((e ^ x) & 2) ? q : t[e];
          }
          __builtin_nontemporal_store(f32x4{o[0], o[1], o[2], o[3]}, reinterpret_cast<f32x4*>(zr + 32 * j));
        }
      }
  }
  lm_partial_epilogue<false, TERMS>(p, acc, m0, n0, tn, sm);
}

// The forward-only fused product: tile partials with the entropy moment, no logits stored.
__global__ __launch_bounds__(LmCfg::NT) void k_lm_partial_ent(const PartialArgs p) {
  __shared__ __attribute__((aligned(16))) GemmSmem sm;
  int tm, tn;
  if (!gemm_tile_of(blockIdx.x, gridDim.x, tiles_of(p.g.M), tiles_of(p.g.N), tm, tn)) return;
  g_f32x16 acc[LmCfg::IB][LmCfg::JB];
  gemm_mainloop<LmCfg>(p.g, tm * TILE, tn * TILE, acc, sm.s);
  lm_partial_epilogue<true, false>(p, acc, tm * TILE, tn * TILE, tn, sm);
}

template <bool ENT, bool TERMS>
__device__ __forceinline__ void lm_partial_epilogue(const PartialArgs& p, g_f32x16 (&acc)[LmCfg::IB][LmCfg::JB],
                                                    int m0, int n0, int tn, GemmSmem& sm) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / LmCfg::WGN, wn = wave % LmCfg::WGN;
  // A 16-lane row of a wave holds 16 x JB columns of one output row: reduce them with DPP, then the 2 x WGN such
  // groups of each row through LDS.  First the row's maximum over the tile, then one pass of exponentials against
  // it for the sums (and the stored terms).
  constexpr int NG = 2 * LmCfg::WGN;
  float* sh_m = reinterpret_cast<float*>(sm.s);  // [NG][TILE] group maxima
  float* sh_s = sh_m + NG * TILE;                 // [NG][TILE] group sums
  float* sh_t = sh_s + NG * TILE;                 // [NG][TILE] group entropy moments, ENT only
  float* sh_M = sh_t + NG * TILE;                 // [TILE] the rows' maxima over the tile
  const int grp = wn * 2 + ((lane >> 4) & 1);
  const int c = n0 + gemm_col<LmCfg>(wn, 0, lane);
  const bool full = n0 + TILE <= p.g.N;
  auto logit = [&](int i, int j, int r) { return (full || c + 32 * j < p.g.N) ? acc[i][j][r] : -INFINITY; };
#define GRPO_DPP_STEP(OP, X, CTRL) _Pragma("unroll") for (int u = 0; u < 4; ++u) X[u] = OP(X[u], dpp_f32<CTRL>(X[u]));
#pragma unroll
  for (int i = 0; i < LmCfg::IB; ++i) {
#pragma unroll
    for (int r0 = 0; r0 < 16; r0 += 4) {  // four rows at a time: independent DPP chains interleave
      float m[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        m[u] = -INFINITY;
#pragma unroll
        for (int j = 0; j < LmCfg::JB; ++j) m[u] = fmaxf(m[u], logit(i, j, r0 + u));
      }
      GRPO_DPP_STEP(fmaxf, m, 0xB1)
      GRPO_DPP_STEP(fmaxf, m, 0x4E)
      GRPO_DPP_STEP(fmaxf, m, 0x141)
      GRPO_DPP_STEP(fmaxf, m, 0x140)
      if ((lane & 15) == 0)
#pragma unroll
        for (int u = 0; u < 4; ++u) sh_m[grp * TILE + gemm_row<LmCfg>(wm, i, r0 + u, lane)] = m[u];
    }
  }
  __syncthreads();
  if (tid < TILE) {  // rows past M: the maximum of their zero logits
    float M = -INFINITY;
#pragma unroll
    for (int q = 0; q < NG; ++q) M = fmaxf(M, sh_m[q * TILE + tid]);
    sh_M[tid] = M;
  }
  __syncthreads();
  const int x = lane & 3;
#pragma unroll
  for (int i = 0; i < LmCfg::IB; ++i) {
#pragma unroll
    for (int r0 = 0; r0 < 16; r0 += 4) {
      // accumulators r0 .. r0 + 3 of a lane: rows rb .. rb + 3
      const int rb = wm * LmCfg::WTM + i * 32 + 2 * r0 + 4 * (lane >> 5);
      const f32x4 Mv = *reinterpret_cast<const f32x4*>(sh_M + rb);
      float e[4], tt[4], xs[LmCfg::JB][4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const float nm = (Mv[u] == -INFINITY) ? 0.f : -Mv[u] * kLog2e;
        e[u] = 0.f;
        tt[u] = 0.f;
#pragma unroll
        for (int j = 0; j < LmCfg::JB; ++j) {
          const float v = logit(i, j, r0 + u);
          xs[j][u] = __builtin_amdgcn_exp2f(fmaf(v, kLog2e, nm));
          e[u] += xs[j][u];
          if constexpr (ENT) tt[u] += (v == -INFINITY) ? 0.f : xs[j][u] * (v - Mv[u]);
        }
      }
      if constexpr (TERMS) {
        // A 4 x 4 transpose within each quad of lanes (two DPP exchanges: lanes x ^ 1, then x ^ 2) leaves lane
        // 4a + x with row rb + x and columns 4a .. 4a + 3 of each 32-column block j.  Lanes 4a + x and its
        // partner 4(a ^ 1) + x then trade one block's 8 bytes, so that a lane with a even holds columns
        // 4a .. 4a + 7 of block 0 and its partner the same columns of block 1: one 16-byte store per lane, and each
        // store instruction fills the wave's whole 128-byte piece of its 8 rows.
        uint16_t* er = p.e16 + (int64_t)(m0 + rb + x) * p.ldz + n0 + wn * LmCfg::WTN + 4 * ((lane & 31) >> 2);
        uint32_t pk[LmCfg::JB][2];
#pragma unroll
        for (int j = 0; j < LmCfg::JB; ++j) {
          float t[4], o[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const float q = dpp_f32<0xB1>(xs[j][u ^ 1]);  // lane x ^ 1's term u ^ 1
            t[u] = ((u ^ x) & 1) ? q : xs[j][u];
          }
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const float q = dpp_f32<0x4E>(t[u ^ 2]);  // lane x ^ 2's value u ^ 2
            o[u] = ((u ^ x) & 2) ? q : t[u];
          }
          pk[j][0] = pack_f16(o[0], o[1]);
          pk[j][1] = pack_f16(o[2], o[3]);
        }
        static_assert(LmCfg::JB == 2, "two 32-column blocks per wave");
        const bool even = ((lane >> 2) & 1) == 0;
        uint32_t r[2];
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          // lane L ^ 4: the quad reversed (quad_perm [3, 2, 1, 0] = 0x1B), then the 8-lane group mirrored (0x141)
          const float sent = __uint_as_float(even ? pk[1][q] : pk[0][q]);
          r[q] = __float_as_uint(dpp_f32<0x141>(dpp_f32<0x1B>(sent)));
        }
        const u32x4 w = even ? u32x4{pk[0][0], pk[0][1], r[0], r[1]} : u32x4{r[0], r[1], pk[1][0], pk[1][1]};
        __builtin_nontemporal_store(w, reinterpret_cast<u32x4*>(er + (even ? 0 : 32 - 4)));
      }
      GRPO_DPP_STEP(add_f32, e, 0xB1)
      GRPO_DPP_STEP(add_f32, e, 0x4E)
      GRPO_DPP_STEP(add_f32, e, 0x141)
      GRPO_DPP_STEP(add_f32, e, 0x140)
      if constexpr (ENT) {
        GRPO_DPP_STEP(add_f32, tt, 0xB1)
        GRPO_DPP_STEP(add_f32, tt, 0x4E)
        GRPO_DPP_STEP(add_f32, tt, 0x141)
        GRPO_DPP_STEP(add_f32, tt, 0x140)
      }
      if ((lane & 15) == 0)
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          sh_s[grp * TILE + rb + u] = e[u];
          if constexpr (ENT) sh_t[grp * TILE + rb + u] = tt[u];
        }
    }
  }
#undef GRPO_DPP_STEP
  __syncthreads();
  if (tid < TILE && m0 + tid < p.g.M) {
    float S = 0.f, Tm = 0.f;
#pragma unroll
    for (int q = 0; q < NG; ++q) {
      S += sh_s[q * TILE + tid];
      if constexpr (ENT) Tm += sh_t[q * TILE + tid];
    }
    p.part[(int64_t)(m0 + tid) * p.n_tiles + tn] = make_float2(sh_M[tid], S);
    if constexpr (ENT) p.part_t[(int64_t)(m0 + tid) * p.n_tiles + tn] = Tm;
  }
}

// ---- combine: lse, action logit, log-prob and the token epilogue, one workgroup per row
struct CombineArgs {
  TokenArgs tok;
  const float2* part;
  const uint16_t* h;   // [T, H]
  const uint16_t* WT;  // [V, H], or with PACKED W^T in the fragment-packed layout
  RowScale* rs;        // [Tp]; rows >= T get the zero scale
  int T, H, n_tiles;
  int t0;              // row of blockIdx.x 0; part holds rows from t0 on
};

// Row t of 256 threads: the row's shift M and S = sum over its tiles of the partials rescaled to M, and the
// action logit z_a = h_t . W[:, act] (row act of the transposed weight) in fp64, or 0 when act < 0.  The
// results are valid in thread 0.
struct RowStatsSmem {
  float m[4];
  double s[4], z[4];
};
// Elements 8 q .. 8 q + 7 of row `row` of a matrix with K = H columns: 16 contiguous bytes in either layout.
template <bool PACKED>
__device__ __forceinline__ const uint16_t* row_piece(const uint16_t* B, int64_t row, int q, int H) {
  if constexpr (PACKED)  // chunk (row / 32, q / 2), lane 32 (q % 2) + row % 32
    return B + ((row >> 5) * packed_kb_count(H) + (q >> 1)) * 512 + ((q & 1) * 32 + (row & 31)) * 8;
  else
    return B + row * H + 8 * q;
}

template <bool PACKED = false>
__device__ inline void lm_row_stats(const float2* pr, int n_tiles, const uint16_t* hr, const uint16_t* WT, int act,
                                    int H, RowStatsSmem& sh, float& M_out, double& S_out, double& z_out) {
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  float m = -INFINITY;
  for (int j = tid; j < n_tiles; j += 256) m = fmaxf(m, pr[j].x);
  m = wave_max(m);
  double z = 0.0;
  if (act >= 0) {
    for (int k = tid * 8; k < H; k += 256 * 8) {
      const u32x4 x = *reinterpret_cast<const u32x4*>(hr + k);
      const u32x4 y = *reinterpret_cast<const u32x4*>(row_piece<PACKED>(WT, act, k / 8, H));
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        z += (double)bf16_lo(x[q]) * (double)bf16_lo(y[q]);
        z += (double)bf16_hi(x[q]) * (double)bf16_hi(y[q]);
      }
    }
  }
  z = wave_sum(z);
  if (lane == 0) {
    sh.m[wv] = m;
    sh.z[wv] = z;
  }
  __syncthreads();
  const float M = fmaxf(fmaxf(sh.m[0], sh.m[1]), fmaxf(sh.m[2], sh.m[3]));
  double s = 0.0;
  if (M != -INFINITY)
    for (int j = tid; j < n_tiles; j += 256) {
      const float2 q = pr[j];
      if (q.x != -INFINITY) s += (double)q.y * (double)__builtin_amdgcn_exp2f((q.x - M) * kLog2e);
    }
  s = wave_sum(s);
  if (lane == 0) sh.s[wv] = s;
  __syncthreads();
  M_out = M;
  S_out = sh.s[0] + sh.s[1] + sh.s[2] + sh.s[3];
  z_out = sh.z[0] + sh.z[1] + sh.z[2] + sh.z[3];
}

template <bool PACKED = false>
__global__ __launch_bounds__(256) void k_lm_combine(const CombineArgs a) {
  __shared__ RowStatsSmem sh;
  const int t = a.t0 + (int)blockIdx.x, tid = threadIdx.x;
  if (t >= a.T) {
    if (tid == 0) a.rs[t] = RowScale{-INFINITY, 1.f, 0.f, -1};
    return;
  }
  const int act = a.tok.actions[t];
  const bool ok = act >= 0 && (int64_t)act < a.tok.V;
  float M;
  double S, za;
  lm_row_stats<PACKED>(a.part + (int64_t)(t - a.t0) * a.n_tiles, a.n_tiles, a.h + (int64_t)t * a.H, a.WT,
                       ok ? act : -1, a.H, sh, M, S, za);
  if (tid == 0) {
    const TokenIn in = token_load(a.tok, t);
    a.rs[t] = token_finish(a.tok, t, in, row_lse((double)M, S), za);
  }
}

// ---- a vocabulary shard's per-token record (the first call of the sharded fused path) --
struct RecordArgs {
  const float2* part;
  const uint16_t* h;       // [T, H]
  const uint16_t* WT;      // [V_shard, H]
  const int32_t* actions;  // global ids
  grpo_vocab_stats* stats; // [T]
  int64_t v_begin, V;      // the shard's first global column and width
  int T, H, n_tiles;
};

__global__ __launch_bounds__(256) void k_lm_record(const RecordArgs a) {
  __shared__ RowStatsSmem sh;
  const int t = blockIdx.x;
  const int64_t al = (int64_t)a.actions[t] - a.v_begin;
  const bool own = al >= 0 && al < a.V;
  float M;
  double S, za;
  lm_row_stats(a.part + (int64_t)t * a.n_tiles, a.n_tiles, a.h + (int64_t)t * a.H, a.WT, own ? (int)al : -1, a.H, sh,
               M, S, za);
  if (threadIdx.x == 0) {
    grpo_vocab_stats r;
    r.m = M;
    r.s = S;
    r.z_a = own ? za : -INFINITY;
    a.stats[t] = r;
  }
}

// ---- forward only: the action's log-prob and the entropy per row, one workgroup per row -------------------
struct LmLogpArgs {
  const float2* part;     // [T, n_tiles]
  const float* part_t;    // [T, n_tiles] or null (no entropy)
  const uint16_t* h;      // [T, H]
  const uint16_t* WT;     // [V, H]
  const int32_t* actions;
  float* logp;            // [T] or null
  float* entropy;         // [T] or null
  int32_t* flags;         // or null
  int64_t V;
  int T, H, n_tiles;
};

__global__ void k_lm_clear_flags(int32_t* f) { *f = 0; }

__global__ __launch_bounds__(256) void k_lm_logp(const LmLogpArgs a) {
  __shared__ RowStatsSmem sh;
  __shared__ double sh_t[4];
  const int t = blockIdx.x, tid = threadIdx.x;
  const int act = a.actions[t];
  const bool ok = act >= 0 && (int64_t)act < a.V;
  float M;
  double S, za;
  const float2* pr = a.part + (int64_t)t * a.n_tiles;
  lm_row_stats(pr, a.n_tiles, a.h + (int64_t)t * a.H, a.WT, ok ? act : -1, a.H, sh, M, S, za);
  double Tm = 0.0;
  if (a.entropy) {
    // the row's second moment about M: sum over tiles of e^(m_j - M) (T_j + S_j (m_j - M))
    const float* pt = a.part_t + (int64_t)t * a.n_tiles;
    double x = 0.0;
    if (M != -INFINITY)
      for (int j = tid; j < a.n_tiles; j += 256) {
        const float2 q = pr[j];
        if (q.x != -INFINITY) {
          const double d = (double)q.x - (double)M;
          x += exp(d) * ((double)pt[j] + (double)q.y * d);
        }
      }
    x = wave_sum(x);
    if ((tid & 63) == 0) sh_t[tid >> 6] = x;
    __syncthreads();
    Tm = sh_t[0] + sh_t[1] + sh_t[2] + sh_t[3];
  }
  if (tid == 0) {
    const double lse = (double)M + log(S);
    if (a.logp) a.logp[t] = ok ? (float)(za - lse) : 0.f;
    if (a.entropy) a.entropy[t] = (float)(log(S) - Tm / S);
    if (a.flags) {
      if (!ok) atomicOr(a.flags, GRPO_FLAG_ACTION);
      if (!isfinite(lse)) atomicOr(a.flags, GRPO_FLAG_NONFINITE);
    }
  }
}

// ---- the sharded fused path's row scales: every shard's records merged, token epilogue, one thread per row
struct ShardScaleArgs {
  TokenArgs tok;                  // tok.V: the whole vocabulary
  const grpo_vocab_stats* stats;  // [n_shards][T]
  RowScale* rs;                   // [Tp]; rows >= T get the zero scale; act is the column within the shard
  int64_t v_begin, V;             // the shard's first global column and width
  int T, Tp, n_shards;
};

__global__ __launch_bounds__(256) void k_lm_shard_scale(const ShardScaleArgs a) {
  const int t = blockIdx.x * 256 + threadIdx.x;
  if (t >= a.Tp) return;
  if (t >= a.T) {
    a.rs[t] = RowScale{-INFINITY, 1.f, 0.f, -1};
    return;
  }
  double lse, za;
  merge_vocab_stats(a.stats, a.n_shards, a.T, t, lse, za);
  const TokenIn in = token_load(a.tok, t);
  RowScale rs = token_finish(a.tok, t, in, lse, za);
  const int64_t al = rs.act >= 0 ? (int64_t)rs.act - a.v_begin : -1;
  rs.act = (al >= 0 && al < a.V) ? (int)al : -1;
  a.rs[t] = rs;
}

// ---- pass 2a: recompute z_c, form D_c = g (softmax - onehot), store D_c and D_c^T --
struct DlogitsArgs {
  GemmArgs g;            // A = h [T, H] (M = Tp), B = W^T rows of the chunk [Cw, H]
  const RowScale* rs;    // [Tp]
  uint16_t* D;           // the chunk's columns of the pair buffer, row stride C
  uint16_t* DT;          // [chunk width, Tp]
  int c0, C, Tp;         // C: D's row stride (twice the chunk when chunks are paired)
};

// Per-wave LDS staging of the dlogits epilogue: 64 rows x 64 columns of the wave's
// output, once row-major (stride 72 bf16: the two 32-lane halves of a 2-byte store
// land on different banks) for D, once column-major for D^T (64 rows per column,
// the eight 16-byte row chunks of column c permuted by (c ^ c >> 3) & 7, which
// keeps the 16-byte column reads free of bank conflicts).
constexpr int kLdr = 72;
constexpr int kStageD = 64 * kLdr, kStageT = 64 * 64;
__device__ __forceinline__ int dt_chunk(int c, int rc) { return rc ^ ((c ^ (c >> 3)) & 7); }

__global__ __launch_bounds__(LmCfg::NT) void k_lm_dlogits(const DlogitsArgs p) {
  constexpr int kMain = 2 * LmCfg::STAGE, kEpi = LmCfg::NW * (kStageD + kStageT);
  __shared__ __attribute__((aligned(16))) uint16_t smem[kMain > kEpi ? kMain : kEpi];
  __shared__ RowScale sh_rs[TILE];
  int tm, tn;
  if (!gemm_tile_of(blockIdx.x, gridDim.x, tiles_of(p.Tp), tiles_of(p.g.N), tm, tn)) return;
  const int m0 = tm * TILE, n0 = tn * TILE;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / LmCfg::WGN, wn = wave % LmCfg::WGN;
  if (tid < TILE) sh_rs[tid] = p.rs[m0 + tid];  // m0 + tid < Tp: Tp is a multiple of the tile
  g_f32x16 acc[LmCfg::IB][LmCfg::JB];
  gemm_mainloop<LmCfg>(p.g, m0, n0, acc, smem);  // its first barrier publishes sh_rs
  // Columns past the chunk's width (last tile of the last chunk) are written too: they
  // stay inside D's C columns and D^T's C rows, and no product reads them.
  // Both layouts go through LDS so that every global store is a 16-byte vector and
  // eight lanes fill one 128-byte line.
  uint16_t* stD = smem + wave * (kStageD + kStageT);
  uint16_t* stT = stD + kStageD;
#pragma unroll
  for (int half = 0; half < 2; ++half) {
#pragma unroll
    for (int ii = 0; ii < 2; ++ii) {
      const int i = half * 2 + ii;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        RowScale rs[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) rs[e] = sh_rs[gemm_row<LmCfg>(wm, i, 4 * q + e, lane)];
#pragma unroll
        for (int j = 0; j < LmCfg::JB; ++j) {
          const int vcol = p.c0 + n0 + gemm_col<LmCfg>(wn, j, lane);
          float d[4];
#pragma unroll
          for (int e = 0; e < 4; ++e)
            d[e] = (vcol == rs[e].act) ? rs[e].d_a
                                       : rs[e].sign * __builtin_amdgcn_exp2f(fmaf(acc[i][j][4 * q + e], kLog2e, rs[e].nc));
          const uint32_t lo = pack_bf16(d[0], d[1]), hi = pack_bf16(d[2], d[3]);
          // local row of the 4 values (in this half) and local column
          const int lr = ii * 32 + 8 * q + 4 * (lane >> 5), lc = j * 32 + (lane & 31);
          stD[(lr + 0) * kLdr + lc] = (uint16_t)(lo & 0xffffu);
          stD[(lr + 1) * kLdr + lc] = (uint16_t)(lo >> 16);
          stD[(lr + 2) * kLdr + lc] = (uint16_t)(hi & 0xffffu);
          stD[(lr + 3) * kLdr + lc] = (uint16_t)(hi >> 16);
          *reinterpret_cast<u32x2*>(stT + lc * 64 + dt_chunk(lc, lr >> 3) * 8 + (lr & 7)) = u32x2{lo, hi};
        }
      }
    }
    // LDS runs a wave's accesses in order: the staged values are read back by the same wave
#pragma unroll
    for (int it = 0; it < 8; ++it) {  // D: 8 rows per pass, 8 lanes per 64-column row
      const int lr = it * 8 + (lane >> 3), cv = (lane & 7) * 8;
      const u32x4 v = *reinterpret_cast<const u32x4*>(stD + lr * kLdr + cv);
      const int grow = m0 + wm * LmCfg::WTM + half * 64 + lr;
      *reinterpret_cast<u32x4*>(p.D + (int64_t)grow * p.C + n0 + wn * LmCfg::WTN + cv) = v;
    }
#pragma unroll
    for (int it = 0; it < 8; ++it) {  // D^T: 8 columns per pass, 8 lanes per 64-row column
      const int lc = it * 8 + (lane >> 3), rc = lane & 7;
      const u32x4 v = *reinterpret_cast<const u32x4*>(stT + lc * 64 + dt_chunk(lc, rc) * 8);
      const int64_t col = n0 + wn * LmCfg::WTN + lc;
      *reinterpret_cast<u32x4*>(p.DT + col * p.Tp + m0 + wm * LmCfg::WTM + half * 64 + rc * 8) = v;
    }
  }
}

// ---- pass 2b: dhidden += D_c W_c^T --------------------------------------------------
struct DhArgs {
  GemmArgs g;        // A = the pair buffer (M = T, K = the pair's width), B = W[:, pair] as [H, K], ldb = V
                     // (with PACKED: W packed as an H x V matrix)
  float* acc;        // [Tp, H] fp32 accumulator (unused with a single chunk)
  uint16_t* dh;      // [T, H] bf16 output
  int first, last;
};

// One tile of the dhidden product: block bid of nblocks (a multiple of 8, for the XCD order).
template <bool PACKED = false>
__device__ __forceinline__ void lm_dh_tile(const DhArgs& p, int bid, int nblocks, GemmSmem& sm) {
  int tm, tn;
  if (!gemm_tile_of(bid, nblocks, tiles_of(p.g.M), tiles_of(p.g.N), tm, tn)) return;
  const int m0 = tm * TILE, n0 = tn * TILE;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / LmCfg::WGN, wn = wave % LmCfg::WGN;
  g_f32x16 acc[LmCfg::IB][LmCfg::JB];
  if constexpr (PACKED) gemm_mainloop_packed<LmCfg>(p.g, m0, n0, acc, sm.s);
  else gemm_mainloop<LmCfg>(p.g, m0, n0, acc, sm.s);
  const int H = p.g.N;
  // the uniform choices (interior tile, first / last chunk) are template arguments, so
  // that the element loop has no branches
  // Per 32-row block i: after the first chunk, the block's accumulator values are all loaded first and waited
  // for once (element by element, every load would wait for the memory in turn).
  auto store = [&](auto full, auto first, auto last) {
#pragma unroll
    for (int i = 0; i < LmCfg::IB; ++i) {
      float old[16][LmCfg::JB];
      if (!first) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int m = m0 + gemm_row<LmCfg>(wm, i, r, lane);
          const int64_t o = (int64_t)m * H + n0 + gemm_col<LmCfg>(wn, 0, lane);
#pragma unroll
          for (int j = 0; j < LmCfg::JB; ++j)
            old[r][j] = (full || (m < p.g.M && n0 + gemm_col<LmCfg>(wn, j, lane) < H)) ? p.acc[o + 32 * j] : 0.f;
        }
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = m0 + gemm_row<LmCfg>(wm, i, r, lane);
        if (!full && m >= p.g.M) continue;
        const int64_t o = (int64_t)m * H + n0 + gemm_col<LmCfg>(wn, 0, lane);
#pragma unroll
        for (int j = 0; j < LmCfg::JB; ++j) {
          if (!full && n0 + gemm_col<LmCfg>(wn, j, lane) >= H) continue;
          float v = acc[i][j][r];
          if (!first) v += old[r][j];
          if (last) p.dh[o + 32 * j] = (uint16_t)(pack_bf16(v, 0.f) & 0xffffu);
          else p.acc[o + 32 * j] = v;
        }
      }
    }
  };
  typedef std::true_type Y;
  typedef std::false_type N;
  const bool full = m0 + TILE <= p.g.M && n0 + TILE <= H;
  const int mode = (full ? 4 : 0) | (p.first ? 2 : 0) | (p.last ? 1 : 0);
  switch (mode) {
    case 7: store(Y(), Y(), Y()); break;
    case 6: store(Y(), Y(), N()); break;
    case 5: store(Y(), N(), Y()); break;
    case 4: store(Y(), N(), N()); break;
    case 3: store(N(), Y(), Y()); break;
    case 2: store(N(), Y(), N()); break;
    case 1: store(N(), N(), Y()); break;
    default: store(N(), N(), N()); break;
  }
}

// ---- pass 2c: dW[:, chunks] = h^T D -------------------------------------------------
struct DwArgs {
  GemmArgs g;     // A = h^T [H, Tp], B = D^T of the pair [width, Tp], K = Tp (with PACKED: D^T packed)
  float* dw;      // [H, V]
  int64_t V;
  int c0, accumulate;
};

// One tile of the dW product: block bid of nblocks (a multiple of 8).  The XCD-aware order walks N with 8
// M-tiles at a time (the h^T panels shared along N) or, with N_MAJOR, walks M with 4 N-tiles at a time (the D^T
// panels shared along M).  With K = a token block, h^T is small ([H, 8192]: 59 MB, held by the last-level cache)
// and D^T is the whole vocabulary, so N_MAJOR reads D^T from HBM once instead of once per 8 of H's 14 tiles
// (3-4% faster on the bare product, 0.3% on the whole blocked call); with K = the whole batch h^T is the large operand and the first order is kept.
template <bool N_MAJOR, bool PACKED = false>
__device__ __forceinline__ void lm_dw_tile(const DwArgs& p, int bid, int nblocks, GemmSmem& sm) {
  int tm, tn;
  if (N_MAJOR) {
    if (!gemm_tile_of<4>(bid, nblocks, tiles_of(p.g.N), tiles_of(p.g.M), tn, tm)) return;
  } else {
    if (!gemm_tile_of(bid, nblocks, tiles_of(p.g.M), tiles_of(p.g.N), tm, tn)) return;
  }
  const int m0 = tm * TILE, n0 = tn * TILE;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / LmCfg::WGN, wn = wave % LmCfg::WGN;
  g_f32x16 acc[LmCfg::IB][LmCfg::JB];
  if constexpr (PACKED) gemm_mainloop_packed<LmCfg>(p.g, m0, n0, acc, sm.s);
  else gemm_mainloop<LmCfg>(p.g, m0, n0, acc, sm.s);
  // Per 32-row block i: with accumulate, all of its old values are loaded first and waited for once, then
  // added and stored (element by element, every load would wait for the memory in turn).
  auto store = [&](auto full, auto accumulate) {
#pragma unroll
    for (int i = 0; i < LmCfg::IB; ++i) {
      float old[16][LmCfg::JB];
      if (accumulate) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int m = m0 + gemm_row<LmCfg>(wm, i, r, lane);
          const float* o = p.dw + (int64_t)m * p.V + p.c0 + n0 + gemm_col<LmCfg>(wn, 0, lane);
#pragma unroll
          for (int j = 0; j < LmCfg::JB; ++j)
            old[r][j] = (full || (m < p.g.M && n0 + gemm_col<LmCfg>(wn, j, lane) < p.g.N)) ? o[32 * j] : 0.f;
        }
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = m0 + gemm_row<LmCfg>(wm, i, r, lane);
        if (!full && m >= p.g.M) continue;
        float* o = p.dw + (int64_t)m * p.V + p.c0 + n0 + gemm_col<LmCfg>(wn, 0, lane);
#pragma unroll
        for (int j = 0; j < LmCfg::JB; ++j) {
          if (!full && n0 + gemm_col<LmCfg>(wn, j, lane) >= p.g.N) continue;
          o[32 * j] = accumulate ? old[r][j] + acc[i][j][r] : acc[i][j][r];
        }
      }
    }
  };
  typedef std::true_type Y;
  typedef std::false_type N;
  const bool full = m0 + TILE <= p.g.M && n0 + TILE <= p.g.N;
  if (full) {
    if (p.accumulate) store(Y(), Y());
    else store(Y(), N());
  } else {
    if (p.accumulate) store(N(), Y());
    else store(N(), N());
  }
}

// Both backward products of a pair of chunks in one launch.  A dW tile runs over K = Tp, four to eight times
// longer than a dhidden tile (K = the pair's width), and a chunk's dW alone has 1.75 tiles per CU at the
// benchmark's shape; launched first, the long dW tiles are followed on every CU by short dhidden tiles, which
// fill the round the dW tiles leave ragged.
struct DhDwArgs {
  DhArgs dh;
  DwArgs dw;
  int dw_blocks;  // blocks [0, dw_blocks) take dW tiles, the rest dhidden tiles; a multiple of 8
};

__global__ __launch_bounds__(LmCfg::NT) void k_lm_dh_dw(const DhDwArgs p) {
  __shared__ __attribute__((aligned(16))) GemmSmem sm;
  const int b = blockIdx.x;
  if (b < p.dw_blocks) lm_dw_tile<false>(p.dw, b, p.dw_blocks, sm);
  else lm_dh_tile(p.dh, b - p.dw_blocks, (int)gridDim.x - p.dw_blocks, sm);
}

// The token-blocked schedule's backward launch: the dhidden tiles (K = the whole vocabulary) first, then the dW
// tiles (K = the block's rows).  A dhidden tile is then the longest unit by far; dispatched first, the long tiles
// spread over the CUs and the many short dW tiles fill the time the last of them leave.  Both B operands (W and
// D^T) come in the fragment-packed layout.
struct DhThenDwArgs {
  DhArgs dh;
  DwArgs dw;
  int dh_blocks;  // blocks [0, dh_blocks) take dhidden tiles, the rest dW tiles; a multiple of 8
};

__global__ __launch_bounds__(LmCfg::NT) void k_lm_dh_then_dw(const DhThenDwArgs p) {
  __shared__ __attribute__((aligned(16))) GemmSmem sm;
  const int b = blockIdx.x;
  if (b < p.dh_blocks) lm_dh_tile<true>(p.dh, b, p.dh_blocks, sm);
  else lm_dw_tile<true, true>(p.dw, b - p.dh_blocks, (int)gridDim.x - p.dh_blocks, sm);
}

// ---- D = g (softmax - onehot), bf16, as D and D^T: from fp32 logits (k_lm_block_d, a vocabulary shard's kept
// logits) or from a block's stored fp16 terms (k_lm_block_d16, the token-blocked schedule) ----
struct BlockDArgs {
  const float* z;      // [rows, ld] the block's logits (k_lm_block_d), or
  const uint16_t* e16; // [rows, ld] their fp16 terms e = exp(z - m) with m = part[row, tile].x (k_lm_block_d16)
  const float2* part;  // [rows, n_tiles] the block's tile partials (k_lm_block_d16)
  int n_tiles;
  const RowScale* rs;  // [rows] the block's row scales
  uint16_t* D;         // [rows, ld]
  uint16_t* DT;        // [ld, rows], or with packed_dt D^T in the fragment-packed layout (N = ld, K = rows)
  int64_t ld;          // a multiple of 64; columns V..ld get D = 0
  int V, rows;         // rows: a multiple of 64
  int packed_dt;
};
constexpr int kBlockDStrip = 512;  // columns per work item: eight 64 x 64 tiles
constexpr int64_t kBlockDMaxGrid = 1 << 20;  // workgroups per launch at most; they loop over the rest

// Workgroups for n work items: all of them up to the cap, or `grid` (> 0) when fewer.
static unsigned block_d_grid(int64_t rows, int64_t ld, int grid) {
  int64_t items = rows / 64 * ((ld + kBlockDStrip - 1) / kBlockDStrip);
  if (items > kBlockDMaxGrid) items = kBlockDMaxGrid;
  return (unsigned)(grid > 0 && grid < items ? grid : items);
}

// Work items of 64 rows and a strip of up to eight 64-column tiles, item i = strip * (rows / 64) + row tile; a
// workgroup of 256 threads takes items blockIdx.x, blockIdx.x + gridDim.x, ... (one each with a full grid; a
// grid of one workgroup per CU when the pass runs beside a matrix-core launch).  Per tile a thread takes two
// 2 x 4 pieces (rows 2p, 2p + 1 of four columns, p = tid / 16 and p + 16): two 16-byte logit loads each; the D
// rows go out as 8-byte stores (16 lanes fill a 128-byte line); for D^T every column's row pair is packed into
// one 32-bit LDS word (stride 33 words per column), read back as four words = eight rows, and stored 16 bytes
// at a time (8 lanes per 128-byte column piece, or with packed_dt one packed lane's 16 bytes, 8 lanes of
// consecutive columns side by side).  Two LDS buffers, one barrier per tile.
__global__ __launch_bounds__(256) void k_lm_block_d(const BlockDArgs a) {
  constexpr int kLdw = 33;
  __shared__ uint32_t tu[2][64 * kLdw];
  __shared__ RowScale srs[64];
  const int tid = threadIdx.x;
  const int64_t n_rt = a.rows / 64;
  const int64_t n_items = n_rt * ((a.ld + kBlockDStrip - 1) / kBlockDStrip);
  for (int64_t item = blockIdx.x; item < n_items; item += gridDim.x) {
    const int r0 = (int)(item % n_rt) * 64;
    const int64_t cs = (item / n_rt) * kBlockDStrip;
    __syncthreads();  // the previous item's last reads of tu and srs are done
    if (tid < 64) srs[tid] = a.rs[r0 + tid];
    __syncthreads();
    const int cq = tid & 15, rp = tid >> 4;
    const int ntiles = (int)min((int64_t)(kBlockDStrip / 64), (a.ld - cs) / 64);
    for (int it = 0; it < ntiles; ++it) {
      const int64_t c = cs + it * 64 + 4 * cq;
      uint32_t* t = tu[it & 1];
#pragma unroll
      for (int u = 0; u < 2; ++u) {  // rows 2 rp + 32 u and the next one
        const int row = 2 * rp + 32 * u;
        // the row scales are read from LDS where they are used (per element; the reads are merged): kept in
        // registers they take the pass past the 80 VGPRs that fit beside a forward-product workgroup (2 x 216 of
        // a SIMD's 512)
        float d0[4], d1[4];
        const float* zr = a.z + (int64_t)(r0 + row) * a.ld + c;
        const f32x4 x0 = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(zr));
        const f32x4 x1 = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(zr + a.ld));
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int64_t v = c + e;
          const RowScale& s0 = srs[row];
          const RowScale& s1 = srs[row + 1];
          d0[e] = v >= a.V ? 0.f : (v == s0.act) ? s0.d_a : s0.sign * __builtin_amdgcn_exp2f(fmaf(x0[e], kLog2e, s0.nc));
          d1[e] = v >= a.V ? 0.f : (v == s1.act) ? s1.d_a : s1.sign * __builtin_amdgcn_exp2f(fmaf(x1[e], kLog2e, s1.nc));
        }
        const uint32_t p00 = pack_bf16(d0[0], d0[1]), p01 = pack_bf16(d0[2], d0[3]);
        const uint32_t p10 = pack_bf16(d1[0], d1[1]), p11 = pack_bf16(d1[2], d1[3]);
        *reinterpret_cast<u32x2*>(a.D + (int64_t)(r0 + row) * a.ld + c) = u32x2{p00, p01};
        *reinterpret_cast<u32x2*>(a.D + (int64_t)(r0 + row + 1) * a.ld + c) = u32x2{p10, p11};
        // column e's word: row `row` in the low half, row + 1 in the high half
        uint32_t* tw = t + 4 * cq * kLdw + rp + 16 * u;
        tw[0 * kLdw] = (p00 & 0xffffu) | (p10 << 16);
        tw[1 * kLdw] = (p00 >> 16) | (p10 & 0xffff0000u);
        tw[2 * kLdw] = (p01 & 0xffffu) | (p11 << 16);
        tw[3 * kLdw] = (p01 >> 16) | (p11 & 0xffff0000u);
      }
      __syncthreads();
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        const int col = (tid >> 3) + 32 * q, rc = tid & 7;
        const uint32_t* src = t + col * kLdw + 4 * rc;
        const u32x4 v = {src[0], src[1], src[2], src[3]};
        const int64_t vc = cs + it * 64 + col;
        const int t8 = (r0 >> 3) + rc;  // rows 8 t8 .. 8 t8 + 7 of column vc: one packed lane's 16 bytes
        uint16_t* dst = a.packed_dt ? a.DT + ((vc >> 5) * (a.rows >> 4) + (t8 >> 1)) * 512 + ((t8 & 1) * 32 + (vc & 31)) * 8
                                    : a.DT + vc * a.rows + 8 * t8;
        *reinterpret_cast<u32x4*>(dst) = v;
      }
    }
  }
}


// k_lm_block_d for stored fp16 terms, with each thread on one row pair and 8 columns of a 64 x 64 tile: 16-byte
// term loads and D stores (6 vector-memory instructions per thread and tile instead of 10).
__global__ __launch_bounds__(256) void k_lm_block_d16(const BlockDArgs a) {
  constexpr int kLdw = 33;
  __shared__ uint32_t tu[2][64 * kLdw];
  __shared__ RowScale srs[64];
  const int tid = threadIdx.x;
  const int64_t n_rt = a.rows / 64;
  const int64_t n_items = n_rt * ((a.ld + kBlockDStrip - 1) / kBlockDStrip);
  for (int64_t item = blockIdx.x; item < n_items; item += gridDim.x) {
    const int r0 = (int)(item % n_rt) * 64;
    const int64_t cs = (item / n_rt) * kBlockDStrip;
    __syncthreads();  // the previous item's last reads of tu and srs are done
    if (tid < 64) srs[tid] = a.rs[r0 + tid];
    __syncthreads();
    const int cq = tid & 7, rp = tid >> 3;  // columns 8 cq .. 8 cq + 7 of rows 2 rp, 2 rp + 1
    const int row = 2 * rp;
    const int ntiles = (int)min((int64_t)(kBlockDStrip / 64), (a.ld - cs) / 64);
    for (int it = 0; it < ntiles; ++it) {
      const int64_t c = cs + it * 64 + 8 * cq;
      uint32_t* t = tu[it & 1];
      const uint16_t* er = a.e16 + (int64_t)(r0 + row) * a.ld + c;
      const u32x4 y0 = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(er));
      const u32x4 y1 = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(er + a.ld));
      const int64_t tile = (cs + it * 64) / TILE;
      const RowScale& s0 = srs[row];
      const RowScale& s1 = srs[row + 1];
      const float f0 = s0.nc == -INFINITY ? 0.f
                       : s0.sign * __builtin_amdgcn_exp2f(fmaf(a.part[(int64_t)(r0 + row) * a.n_tiles + tile].x,
                                                               kLog2e, s0.nc));
      const float f1 = s1.nc == -INFINITY ? 0.f
                       : s1.sign * __builtin_amdgcn_exp2f(fmaf(a.part[(int64_t)(r0 + row + 1) * a.n_tiles + tile].x,
                                                               kLog2e, s1.nc));
      uint32_t p0[4], p1[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const f32x2 e0 = unpack_f16(y0[q]), e1 = unpack_f16(y1[q]);
        const int64_t v = c + 2 * q;
        const float a00 = v >= a.V ? 0.f : (v == s0.act) ? s0.d_a : e0[0] * f0;
        const float a01 = v + 1 >= a.V ? 0.f : (v + 1 == s0.act) ? s0.d_a : e0[1] * f0;
        const float a10 = v >= a.V ? 0.f : (v == s1.act) ? s1.d_a : e1[0] * f1;
        const float a11 = v + 1 >= a.V ? 0.f : (v + 1 == s1.act) ? s1.d_a : e1[1] * f1;
        p0[q] = pack_bf16(a00, a01);
        p1[q] = pack_bf16(a10, a11);
      }
      *reinterpret_cast<u32x4*>(a.D + (int64_t)(r0 + row) * a.ld + c) = u32x4{p0[0], p0[1], p0[2], p0[3]};
      *reinterpret_cast<u32x4*>(a.D + (int64_t)(r0 + row + 1) * a.ld + c) = u32x4{p1[0], p1[1], p1[2], p1[3]};
      // column 8 cq + e's word: row `row` in the low half, row + 1 in the high half
      uint32_t* tw = t + 8 * cq * kLdw + rp;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        tw[(2 * q) * kLdw] = (p0[q] & 0xffffu) | (p1[q] << 16);
        tw[(2 * q + 1) * kLdw] = (p0[q] >> 16) | (p1[q] & 0xffff0000u);
      }
      __syncthreads();
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        const int col = (tid >> 3) + 32 * q, rc = tid & 7;
        const uint32_t* src = t + col * kLdw + 4 * rc;
        const u32x4 v = {src[0], src[1], src[2], src[3]};
        const int64_t vc = cs + it * 64 + col;
        const int t8 = (r0 >> 3) + rc;  // rows 8 t8 .. 8 t8 + 7 of column vc: one packed lane's 16 bytes
        uint16_t* dst = a.DT + ((vc >> 5) * (a.rows >> 4) + (t8 >> 1)) * 512 + ((t8 & 1) * 32 + (vc & 31)) * 8;
        *reinterpret_cast<u32x4*>(dst) = v;
      }
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

// ---- fragment-packed operands (gemm_mainloop_packed) -----------------------------------
// dst = src^T packed: src [R, Cc] (row stride lds_), its transpose an Cc x R matrix (N = Cc, K = R).  One 64 x 64
// tile of src per workgroup, staged in LDS as in k_transpose_bf16; it makes the chunks of n-blocks c0 / 32 and
// c0 / 32 + 1 (those that exist) and k-blocks r0 / 16 .. + 3, each lane's 16 bytes taken down a column of the
// tile.  Rows past R give zeros.
__global__ __launch_bounds__(256) void k_pack_t(const uint16_t* __restrict__ src, int64_t lds_, int R, int Cc,
                                                uint16_t* __restrict__ dst) {
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
  const int64_t kbc = packed_kb_count(R), n_nb = ((int64_t)Cc + 31) / 32;
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int piece = tid + 256 * q, chunk = piece >> 6, l = piece & 63;  // chunk = 4 n-block + k-block
    const int64_t nb = c0 / 32 + (chunk >> 2);
    if (nb >= n_nb) continue;
    const int cc = 32 * (chunk >> 2) + (l & 31), rr = 16 * (chunk & 3) + 8 * (l >> 5);
    u32x4 v;
#pragma unroll
    for (int e = 0; e < 4; ++e)
      v[e] = (uint32_t)tile[rr + 2 * e][cc] | ((uint32_t)tile[rr + 2 * e + 1][cc] << 16);
    *reinterpret_cast<u32x4*>(dst + (nb * kbc + r0 / 16 + (chunk & 3)) * 512 + l * 8) = v;
  }
}

// dst = src packed: src [R, Cc] (row stride lds_, Cc a multiple of 8) as an R x Cc matrix (N = R, K = Cc).  A
// workgroup makes the four chunks of n-block blockIdx.y and k-blocks 4 blockIdx.x .. + 3: each lane copies 16
// bytes of one row, and the workgroup reads 128 contiguous bytes of each of its 32 rows.  Columns past Cc and rows
// past R give zeros.
__global__ __launch_bounds__(256) void k_pack_rows(const uint16_t* __restrict__ src, int64_t lds_, int R, int Cc,
                                                   uint16_t* __restrict__ dst) {
  const int64_t kbc = packed_kb_count(Cc), nb = blockIdx.y;
  const int tid = threadIdx.x, kb = 4 * (int)blockIdx.x + (tid >> 6), l = tid & 63;
  const int64_t row = nb * 32 + (l & 31);
  const int col = kb * 16 + 8 * (l >> 5);
  u32x4 v = {0u, 0u, 0u, 0u};
  if (row < R && col < Cc) v = *reinterpret_cast<const u32x4*>(src + row * lds_ + col);
  *reinterpret_cast<u32x4*>(dst + (nb * kbc + kb) * 512 + l * 8) = v;
}

__global__ void k_fill_f32(float* p, int64_t n, float v) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

// ---- workspace --------------------------------------------------------------------
struct LmWs {
  LossWs loss;
  size_t wt, ht, part, rs, d, dt, acc, total;
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
  l.rs = o;   o = align_up(o + sizeof(RowScale) * (size_t)l.Tp);
  l.d = o;    o = align_up(o + sizeof(uint16_t) * (size_t)(l.Tp * C * (n_chunks > 1 ? 2 : 1)));  // a pair of chunks
  l.dt = o;   o = align_up(o + sizeof(uint16_t) * (size_t)(l.Tp * C * (n_chunks > 1 ? 2 : 1)));  // a pair too
  l.acc = o;  o = align_up(o + (n_chunks > 1 ? sizeof(float) * (size_t)(l.Tp * H) : 0));
  l.total = o;
  return l;
}

// A multiple of 8 workgroups covering every tile of an M x N output (see gemm_tile_of).
static dim3 gemm_grid(int64_t M, int64_t N) {
  const int64_t tiles = ((M + TILE - 1) / TILE) * ((N + TILE - 1) / TILE);
  return dim3((unsigned)((tiles + 7) / 8 * 8));
}

// W^T [V, H] from W [H, V] (when WT is set), and h^T [H, Tp] with zero columns T..Tp (when hT is set).
static void lm_transpose(const uint16_t* W16, const uint16_t* h16, int64_t T, int64_t H, int64_t V, int Tp,
                         uint16_t* WT, uint16_t* hT, hipStream_t s) {
  if (WT)
    hipLaunchKernelGGL(k_transpose_bf16, dim3((unsigned)((V + 63) / 64), (unsigned)((H + 63) / 64)), dim3(256), 0,
                       s, W16, V, (int)H, (int)V, WT, H, (int)H);
  if (hT)
    hipLaunchKernelGGL(k_transpose_bf16, dim3((unsigned)((H + 63) / 64), (unsigned)((Tp + 63) / 64)), dim3(256), 0,
                       s, h16, H, (int)T, (int)H, hT, (int64_t)Tp, Tp);
}

static void lm_pass1(const uint16_t* h16, const uint16_t* WT, int64_t T, int64_t H, int64_t V, float2* part,
                     int n_tiles, hipStream_t s) {
  PartialArgs pa{};
  pa.g = GemmArgs{h16, WT, H, H, (int)T, (int)V, (int)H};
  pa.part = part;
  pa.n_tiles = n_tiles;
  pa.z = nullptr;
  pa.ldz = 0;
  pa.part_t = nullptr;
  hipLaunchKernelGGL(k_lm_partial<false>, gemm_grid(T, V), dim3(LmCfg::NT), 0, s, pa);
}

// Pass 2 over the vocabulary chunks of W [H, V] (a whole LM head or one shard's columns), given every row's
// scale in rs.  dhidden: bf16 [T, H] through the fp32 accumulator acc [Tp, H]; or, when dh16 is null, the
// fp32 sum over this W's chunks written straight into acc (a shard's partial dhidden, [T, H]).
struct Pass2 {
  const uint16_t *h16, *W16, *WT, *hT;
  const RowScale* rs;
  uint16_t *D, *DT;
  float* acc;
  uint16_t* dh16;  // null: fp32 partial in acc
  float* dw;       // [H, V]
  int64_t T, H, V;
  int Tp, C, accumulate_dw;
};

static void lm_pass2(const Pass2& q, hipStream_t s) {
  // the backward products take the chunks in pairs (D holds two side by side, D^T one above the other), which
  // halves the passes over dhidden's fp32 accumulator and gives one dW launch per pair
  const int C = q.C;
  const int n_chunks = (int)((q.V + C - 1) / C);
  const int ldD = n_chunks > 1 ? 2 * C : C;
  for (int c = 0; c < n_chunks; ++c) {
    const int c0 = c * C;
    const int Cw = (int)((q.V - c0) < C ? (q.V - c0) : C);
    DlogitsArgs da;
    da.g = GemmArgs{q.h16, q.WT + (int64_t)c0 * q.H, q.H, q.H, (int)q.T, Cw, (int)q.H};
    da.rs = q.rs;
    da.D = q.D + (c & 1) * C;
    da.DT = q.DT + (int64_t)(c & 1) * C * q.Tp;
    da.c0 = c0;
    da.C = ldD;
    da.Tp = q.Tp;
    hipLaunchKernelGGL(k_lm_dlogits, gemm_grid(q.Tp, Cw), dim3(LmCfg::NT), 0, s, da);
    if ((c & 1) || c == n_chunks - 1) {
      const int p0 = c & ~1;                  // first chunk of the pair
      const int width = (c & 1) ? C + Cw : Cw;  // the pair's vocabulary columns
      DhDwArgs ba;
      ba.dh.g = GemmArgs{q.D, q.W16 + (int64_t)p0 * C, ldD, q.V, (int)q.T, (int)q.H, width};
      ba.dh.acc = q.acc;
      ba.dh.dh = q.dh16;
      ba.dh.first = (p0 == 0);
      ba.dh.last = q.dh16 != nullptr && c == n_chunks - 1;
      ba.dw.g = GemmArgs{q.hT, q.DT, q.Tp, q.Tp, (int)q.H, width, q.Tp};
      ba.dw.dw = q.dw;
      ba.dw.V = q.V;
      ba.dw.c0 = p0 * C;
      ba.dw.accumulate = q.accumulate_dw;
      ba.dw_blocks = (int)gemm_grid(q.H, width).x;
      hipLaunchKernelGGL(k_lm_dh_dw, dim3((unsigned)ba.dw_blocks + gemm_grid(q.T, q.H).x), dim3(LmCfg::NT), 0, s, ba);
    }
  }
}

// The token-blocked schedule's workspace: W^T and W in the fragment-packed layout (the B operands of the forward
// and dhidden products), h^T, the fp32 logits of two blocks (the next block's forward product runs while the D
// pass reads the previous block's when a second stream is given), the D and the packed D^T of one block.
struct LmBlockWs {
  LossWs loss;
  size_t wt, wp, ht, part, rs, z, d, dt, total;
  int64_t Tp, Tbp, ldz;
  int n_tiles;
};
static LmBlockWs lm_block_ws_layout(int64_t T, int64_t H, int64_t V, int32_t Tb, int32_t n_traj) {
  LmBlockWs l;
  l.loss = loss_ws_layout(T, n_traj);
  l.Tp = (T + TILE - 1) / TILE * TILE;
  l.Tbp = l.Tp < Tb ? l.Tp : Tb;
  l.n_tiles = (int)((V + TILE - 1) / TILE);
  l.ldz = (int64_t)l.n_tiles * TILE;
  size_t o = l.loss.total;
  l.wt = o;   o = align_up(o + (size_t)packed_bytes(V, H));
  l.wp = o;   o = align_up(o + (size_t)packed_bytes(H, V));
  l.ht = o;   o = align_up(o + sizeof(uint16_t) * (size_t)(H * l.Tp));
  const size_t nbuf = l.Tp > l.Tbp ? 2 : 1;  // the tile partials and terms of two blocks in flight
  l.part = o; o = align_up(o + sizeof(float2) * (size_t)(l.Tbp * l.n_tiles) * nbuf);
  l.rs = o;   o = align_up(o + sizeof(RowScale) * (size_t)l.Tp);
  l.z = o;    o = align_up(o + sizeof(uint16_t) * (size_t)(l.Tbp * l.ldz) * nbuf);
  l.d = o;    o = align_up(o + sizeof(uint16_t) * (size_t)(l.Tbp * l.ldz));
  l.dt = o;   o = align_up(o + (size_t)packed_bytes(l.ldz, l.Tbp));
  l.total = o;
  return l;
}

// The shard statistics call needs W^T of the shard and the pass-1 partials only.
struct LmStatsWs {
  size_t wt, part, total;
};
static LmStatsWs lm_stats_ws_layout(int64_t T, int64_t H, int64_t V) {
  LmStatsWs l;
  size_t o = 0;
  l.wt = o;   o = align_up(o + sizeof(uint16_t) * (size_t)(V * H));
  l.part = o; o = align_up(o + sizeof(float2) * (size_t)(T * ((V + TILE - 1) / TILE)));
  l.total = o;
  return l;
}

// The GEMMs address their operands through buffer descriptors with 32-bit byte offsets, 256 rows at a time: the
// T-long rows of h^T and D^T (dW) and the V-long rows of W (dhidden) must keep 256 rows below 2^32 bytes.
constexpr int64_t kMaxFusedLen = ((int64_t)1 << 23) - 256;

static int check_fused_shapes(int64_t T, int64_t H, int64_t V) {
  if (T < 0 || T >= ((int64_t)1 << 31)) return GRPO_ERR_SHAPE;
  if (H < 64 || H % 64 != 0 || H >= (1 << 30)) return GRPO_ERR_SHAPE;
  if (V < 8 || V % 8 != 0 || V >= ((int64_t)1 << 31)) return GRPO_ERR_SHAPE;
  return GRPO_OK;
}

}  // namespace grpo

using namespace grpo;

// Sizes a fused workspace query answers (the entry points accept no larger ones); their products cannot overflow.
static bool fused_query_sizes_ok(int64_t T, int64_t H, int64_t V) {
  return T >= 0 && T <= kMaxFusedLen && H >= 1 && H < (1 << 30) && V >= 1 && V <= kMaxFusedLen;
}

extern "C" size_t fused_lmhead_workspace_bytes(int64_t T, int64_t H, int64_t V, int32_t vocab_chunk, int32_t n_traj) {
  if (!fused_query_sizes_ok(T, H, V) || vocab_chunk < 1 || n_traj < 1) return 0;
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
  if (T > kMaxFusedLen || V > kMaxFusedLen) return GRPO_ERR_SHAPE;
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
  RowScale* rs = reinterpret_cast<RowScale*>(w + L.rs);
  uint16_t* D = reinterpret_cast<uint16_t*>(w + L.d);
  uint16_t* DT = reinterpret_cast<uint16_t*>(w + L.dt);
  float* acc = reinterpret_cast<float*>(w + L.acc);
  const int Tp = (int)L.Tp;

  if (launch_segments(seg, T, V, actions, adv, p, w, L.loss, aux, s) != hipSuccess) return GRPO_ERR_HIP;
  if (T == 0) {
    if (!accumulate_dw) hipLaunchKernelGGL(k_fill_f32, dim3(1024), dim3(256), 0, s, dw_lm, H * V, 0.f);
    if (hipGetLastError() != hipSuccess) return GRPO_ERR_HIP;
    return launch_reduce(T, seg->n_traj, w, L.loss, loss_out, aux, s) == hipSuccess ? GRPO_OK : GRPO_ERR_HIP;
  }
  lm_transpose(W16, h16, T, H, V, Tp, WT, hT, s);
  if (hipGetLastError() != hipSuccess) return GRPO_ERR_HIP;

  const bool timed = aux && aux->hot_begin && aux->hot_end;
  if (timed && hipEventRecord(aux->hot_begin, s) != hipSuccess) return GRPO_ERR_HIP;
  lm_pass1(h16, WT, T, H, V, part, L.n_tiles, s);
  // combine
  CombineArgs ca;
  ca.tok = make_token_args(V, actions, behave_logp, prox_logp, adv, p, w, L.loss, aux);
  ca.part = part;
  ca.h = h16;
  ca.WT = WT;
  ca.rs = rs;
  ca.T = (int)T;
  ca.H = (int)H;
  ca.n_tiles = L.n_tiles;
  ca.t0 = 0;
  hipLaunchKernelGGL(k_lm_combine<false>, dim3((unsigned)Tp), dim3(256), 0, s, ca);
  if (hipGetLastError() != hipSuccess) return GRPO_ERR_HIP;
  lm_pass2(Pass2{h16, W16, WT, hT, rs, D, DT, acc, static_cast<uint16_t*>(dhidden), dw_lm, T, H, V, Tp,
                 vocab_chunk, accumulate_dw},
           s);
  if (hipGetLastError() != hipSuccess) return GRPO_ERR_HIP;
  if (timed && hipEventRecord(aux->hot_end, s) != hipSuccess) return GRPO_ERR_HIP;
  if (launch_reduce(T, seg->n_traj, w, L.loss, loss_out, aux, s) != hipSuccess) return GRPO_ERR_HIP;
  return GRPO_OK;
}

extern "C" size_t fused_lmhead_blocked_workspace_bytes(int64_t T, int64_t H, int64_t V, int32_t token_block,
                                                      int32_t n_traj) {
  if (!fused_query_sizes_ok(T, H, V) || token_block < TILE || token_block % TILE != 0 || token_block > kMaxFusedLen ||
      n_traj < 1)
    return 0;
  return lm_block_ws_layout(T, H, V, token_block, n_traj).total;
}

extern "C" int fused_lmhead_grpo_blocked(const void* hidden, const void* w_lm, int64_t T, int64_t H, int64_t V,
                                         int32_t token_block, const int32_t* actions, const float* behave_logp,
                                         const float* prox_logp, const float* adv, const grpo_segments* seg,
                                         const grpo_loss_params* p, double* loss_out, void* dhidden, float* dw_lm,
                                         int32_t accumulate_dw, grpo_aux* aux, void* ws, size_t ws_bytes,
                                         hipStream_t s, hipStream_t s_aux) {
  int st = check_loss_common(T, actions, behave_logp, adv, seg, p, loss_out);
  if (st != GRPO_OK) return st;
  if (!w_lm || !dw_lm || (T > 0 && (!hidden || !dhidden))) return GRPO_ERR_ARG;
  st = check_fused_shapes(T, H, V);
  if (st != GRPO_OK) return st;
  if (T > kMaxFusedLen || V > kMaxFusedLen) return GRPO_ERR_SHAPE;
  if (token_block < TILE || token_block % TILE != 0 || token_block > kMaxFusedLen) return GRPO_ERR_SHAPE;
  if (!aligned(hidden, 16) || !aligned(w_lm, 16) || !aligned(dhidden, 16) || !aligned(dw_lm, 16))
    return GRPO_ERR_ALIGN;
  const LmBlockWs L = lm_block_ws_layout(T, H, V, token_block, seg->n_traj);
  if (!ws || ws_bytes < L.total) return GRPO_ERR_WORKSPACE;
  if (!aligned(ws, kAlign)) return GRPO_ERR_ALIGN;
  if (s_aux && s_aux != s) {  // the second stream must be on the first one's device
    hipDevice_t dev_s = 0, dev_aux = 0;
    if (hipStreamGetDevice(s, &dev_s) != hipSuccess || hipStreamGetDevice(s_aux, &dev_aux) != hipSuccess)
      return GRPO_ERR_HIP;
    if (dev_s != dev_aux) return GRPO_ERR_ARG;
  }
  char* w = static_cast<char*>(ws);
  const uint16_t* h16 = static_cast<const uint16_t*>(hidden);
  const uint16_t* W16 = static_cast<const uint16_t*>(w_lm);
  uint16_t* WT = reinterpret_cast<uint16_t*>(w + L.wt);  // packed
  uint16_t* WP = reinterpret_cast<uint16_t*>(w + L.wp);  // packed
  uint16_t* hT = reinterpret_cast<uint16_t*>(w + L.ht);
  float2* part = reinterpret_cast<float2*>(w + L.part);
  RowScale* rs = reinterpret_cast<RowScale*>(w + L.rs);
  uint16_t* e16 = reinterpret_cast<uint16_t*>(w + L.z);
  uint16_t* D = reinterpret_cast<uint16_t*>(w + L.d);
  uint16_t* DT = reinterpret_cast<uint16_t*>(w + L.dt);
  uint16_t* dh16 = static_cast<uint16_t*>(dhidden);
  const int Tp = (int)L.Tp;

  if (launch_segments(seg, T, V, actions, adv, p, w, L.loss, aux, s) != hipSuccess) return GRPO_ERR_HIP;
  if (T == 0) {
    if (!accumulate_dw) hipLaunchKernelGGL(k_fill_f32, dim3(1024), dim3(256), 0, s, dw_lm, H * V, 0.f);
    if (hipGetLastError() != hipSuccess) return GRPO_ERR_HIP;
    return launch_reduce(T, seg->n_traj, w, L.loss, loss_out, aux, s) == hipSuccess ? GRPO_OK : GRPO_ERR_HIP;
  }
  lm_transpose(W16, h16, T, H, V, Tp, nullptr, hT, s);
  hipLaunchKernelGGL(k_pack_t, dim3((unsigned)((V + 63) / 64), (unsigned)((H + 63) / 64)), dim3(256), 0, s, W16, V,
                     (int)H, (int)V, WT);
  hipLaunchKernelGGL(k_pack_rows, dim3((unsigned)(packed_kb_count(V) / 4), (unsigned)((H + 31) / 32)), dim3(256), 0,
                     s, W16, V, (int)H, (int)V, WP);
  if (hipGetLastError() != hipSuccess) return GRPO_ERR_HIP;
  const bool timed = aux && aux->hot_begin && aux->hot_end;
  if (timed && hipEventRecord(aux->hot_begin, s) != hipSuccess) return GRPO_ERR_HIP;
  const TokenArgs tok = make_token_args(V, actions, behave_logp, prox_logp, adv, p, w, L.loss, aux);
  const int n_blocks = (int)((T + L.Tbp - 1) / L.Tbp);
  auto rows_of = [&](int b) { return (int)(T - (int64_t)b * L.Tbp < L.Tbp ? T - (int64_t)b * L.Tbp : L.Tbp); };
  auto e_of = [&](int b) { return e16 + (size_t)(b & 1) * (size_t)(L.Tbp * L.ldz); };
  auto part_of = [&](int b) { return part + (size_t)(b & 1) * (size_t)(L.Tbp * L.n_tiles); };
  // block b's forward product (partials, logits into its buffer) and its rows' combine, on s
  auto forward = [&](int b) {
    const int64_t t0 = (int64_t)b * L.Tbp;
    const int rows = rows_of(b), rows_p = (rows + TILE - 1) / TILE * TILE;
    PartialArgs pa{};
    pa.g = GemmArgs{h16 + t0 * H, WT, H, 0, rows, (int)V, (int)H};
    pa.part = part_of(b);
    pa.n_tiles = L.n_tiles;
    pa.z = nullptr;
    pa.e16 = e_of(b);
    pa.ldz = L.ldz;
    pa.part_t = nullptr;
    hipLaunchKernelGGL((k_lm_partial<false, true, true>), gemm_grid(rows, V), dim3(LmCfg::NT), 0, s, pa);
    CombineArgs ca;
    ca.tok = tok;
    ca.part = part_of(b);
    ca.h = h16;
    ca.WT = WT;
    ca.rs = rs;
    ca.T = (int)T;
    ca.H = (int)H;
    ca.n_tiles = L.n_tiles;
    ca.t0 = (int)t0;
    hipLaunchKernelGGL(k_lm_combine<true>, dim3((unsigned)rows_p), dim3(256), 0, s, ca);
  };
  // block b's D and D^T from its stored logits; `grid` workgroups (0: one per work item)
  auto dpass = [&](int b, hipStream_t st, int grid) {
    const int rows_p = (rows_of(b) + TILE - 1) / TILE * TILE;
    const BlockDArgs da{nullptr, e_of(b), part_of(b), L.n_tiles, rs + (int64_t)b * L.Tbp, D, DT, L.ldz, (int)V,
                        rows_p, 1};
    hipLaunchKernelGGL(k_lm_block_d16, dim3(block_d_grid(rows_p, L.ldz, grid)), dim3(256), 0, st, da);
  };
  // block b's dhidden rows = D W^T (K = V) and dW (+)= h^T D (K = the block's rows, zero-padded), on s
  auto backward = [&](int b) {
    const int64_t t0 = (int64_t)b * L.Tbp;
    const int rows = rows_of(b), rows_p = (rows + TILE - 1) / TILE * TILE;
    DhThenDwArgs ba;
    ba.dh.g = GemmArgs{D, WP, L.ldz, 0, rows, (int)H, (int)V};
    ba.dh.acc = nullptr;
    ba.dh.dh = dh16 + t0 * H;
    ba.dh.first = 1;
    ba.dh.last = 1;
    ba.dw.g = GemmArgs{hT + t0, DT, Tp, 0, (int)H, (int)V, rows_p};
    ba.dw.dw = dw_lm;
    ba.dw.V = V;
    ba.dw.c0 = 0;
    ba.dw.accumulate = (b > 0 || accumulate_dw) ? 1 : 0;
    ba.dh_blocks = (int)gemm_grid(rows, H).x;
    hipLaunchKernelGGL(k_lm_dh_then_dw, dim3((unsigned)ba.dh_blocks + gemm_grid(H, V).x), dim3(LmCfg::NT), 0, s, ba);
  };
  const bool two = s_aux && s_aux != s && n_blocks > 1;
  if (!two) {
    for (int b = 0; b < n_blocks; ++b) {
      forward(b);
      dpass(b, s, 0);
      backward(b);
      if (hipGetLastError() != hipSuccess) return GRPO_ERR_HIP;
    }
  } else {
    // The D pass of block b runs on s_aux beside the forward product of block b + 1 on s, as one workgroup per
    // CU, so that each CU holds one of each: the forward product's workgroup leaves room in LDS and registers
    // for one D-pass workgroup.  ev_c: block b's rows are combined and the previous backward launch (the last
    // reader of D, D^T) is done; ev_d: block b's D pass is done.
    const int n_cu = stream_cu_count(s);  // of the streams' device, which need not be the current one
    if (n_cu < 1) return GRPO_ERR_HIP;
    hipEvent_t ev_c = nullptr, ev_d = nullptr;
    if (hipEventCreateWithFlags(&ev_c, hipEventDisableTiming) != hipSuccess) return GRPO_ERR_HIP;
    if (hipEventCreateWithFlags(&ev_d, hipEventDisableTiming) != hipSuccess) {
      (void)hipEventDestroy(ev_c);
      return GRPO_ERR_HIP;
    }
    bool ok = true;
    forward(0);
    ok = ok && hipEventRecord(ev_c, s) == hipSuccess && hipStreamWaitEvent(s_aux, ev_c, 0) == hipSuccess;
    dpass(0, s_aux, n_cu);
    ok = ok && hipEventRecord(ev_d, s_aux) == hipSuccess;
    for (int b = 1; ok && b < n_blocks; ++b) {
      forward(b);
      ok = ok && hipStreamWaitEvent(s, ev_d, 0) == hipSuccess;
      backward(b - 1);
      if (b == n_blocks - 1) break;
      ok = ok && hipEventRecord(ev_c, s) == hipSuccess && hipStreamWaitEvent(s_aux, ev_c, 0) == hipSuccess;
      dpass(b, s_aux, n_cu);
      ok = ok && hipEventRecord(ev_d, s_aux) == hipSuccess && hipGetLastError() == hipSuccess;
    }
    // the last block's D pass has no forward product to run beside: the whole grid, on s
    if (ok) {
      dpass(n_blocks - 1, s, 0);
      backward(n_blocks - 1);
    }
    ok = ok && hipGetLastError() == hipSuccess;
    // released by the runtime once the work that uses them has run
    (void)hipEventDestroy(ev_c);
    (void)hipEventDestroy(ev_d);
    if (!ok) return GRPO_ERR_HIP;
  }
  if (timed && hipEventRecord(aux->hot_end, s) != hipSuccess) return GRPO_ERR_HIP;
  if (launch_reduce(T, seg->n_traj, w, L.loss, loss_out, aux, s) != hipSuccess) return GRPO_ERR_HIP;
  return GRPO_OK;
}

// The forward-only call's workspace: W^T and the tile partials (with the entropy moment).
struct LmLogpWs {
  size_t wt, part, part_t, total;
};
static LmLogpWs lm_logp_ws_layout(int64_t T, int64_t H, int64_t V) {
  LmLogpWs l;
  const int64_t n_tiles = (V + TILE - 1) / TILE;
  size_t o = 0;
  l.wt = o;     o = align_up(o + sizeof(uint16_t) * (size_t)(V * H));
  l.part = o;   o = align_up(o + sizeof(float2) * (size_t)(T * n_tiles));
  l.part_t = o; o = align_up(o + sizeof(float) * (size_t)(T * n_tiles));
  l.total = o;
  return l;
}

extern "C" size_t fused_lmhead_token_logp_workspace_bytes(int64_t T, int64_t H, int64_t V) {
  if (!fused_query_sizes_ok(T, H, V)) return 0;
  return lm_logp_ws_layout(T, H, V).total;
}

extern "C" int fused_lmhead_token_logp(const void* hidden, const void* w_lm, int64_t T, int64_t H, int64_t V,
                                       const int32_t* actions, float* token_logp, float* token_entropy,
                                       int32_t* error_flags, void* ws, size_t ws_bytes, hipStream_t s) {
  int st = check_fused_shapes(T, H, V);
  if (st != GRPO_OK) return st;
  if (T > kMaxFusedLen || V > kMaxFusedLen) return GRPO_ERR_SHAPE;
  if (!w_lm || (T > 0 && (!hidden || !actions))) return GRPO_ERR_ARG;
  if (!aligned(hidden, 16) || !aligned(w_lm, 16) || !aligned(token_logp, 4) || !aligned(token_entropy, 4))
    return GRPO_ERR_ALIGN;
  const LmLogpWs L = lm_logp_ws_layout(T, H, V);
  if (!ws || ws_bytes < L.total) return GRPO_ERR_WORKSPACE;
  if (!aligned(ws, kAlign)) return GRPO_ERR_ALIGN;
  if (error_flags) hipLaunchKernelGGL(k_lm_clear_flags, dim3(1), dim3(1), 0, s, error_flags);
  if (T == 0) return hipGetLastError() == hipSuccess ? GRPO_OK : GRPO_ERR_HIP;
  char* w = static_cast<char*>(ws);
  const uint16_t* h16 = static_cast<const uint16_t*>(hidden);
  uint16_t* WT = reinterpret_cast<uint16_t*>(w + L.wt);
  float2* part = reinterpret_cast<float2*>(w + L.part);
  float* part_t = reinterpret_cast<float*>(w + L.part_t);
  const int n_tiles = (int)((V + TILE - 1) / TILE);
  lm_transpose(static_cast<const uint16_t*>(w_lm), h16, T, H, V, 0, WT, nullptr, s);
  if (token_entropy) {
    PartialArgs pa{};
    pa.g = GemmArgs{h16, WT, H, H, (int)T, (int)V, (int)H};
    pa.part = part;
    pa.n_tiles = n_tiles;
    pa.z = nullptr;
    pa.ldz = 0;
    pa.part_t = part_t;
    hipLaunchKernelGGL(k_lm_partial_ent, gemm_grid(T, V), dim3(LmCfg::NT), 0, s, pa);
  } else {
    lm_pass1(h16, WT, T, H, V, part, n_tiles, s);
  }
  const LmLogpArgs la{part, token_entropy ? part_t : nullptr, h16, WT, actions, token_logp, token_entropy,
                      error_flags, V, (int)T, (int)H, n_tiles};
  hipLaunchKernelGGL(k_lm_logp, dim3((unsigned)T), dim3(256), 0, s, la);
  return hipGetLastError() == hipSuccess ? GRPO_OK : GRPO_ERR_HIP;
}

extern "C" size_t fused_lmhead_vocab_shard_stats_workspace_bytes(int64_t T, int64_t H, int64_t V_shard) {
  if (!fused_query_sizes_ok(T, H, V_shard)) return 0;
  return lm_stats_ws_layout(T, H, V_shard).total;
}

extern "C" size_t fused_lmhead_vocab_shard_logits_bytes(int64_t T, int64_t V_shard) {
  if (!fused_query_sizes_ok(T, 1, V_shard)) return 0;
  return sizeof(float) * (size_t)((T + TILE - 1) / TILE * TILE) * (size_t)((V_shard + TILE - 1) / TILE * TILE);
}

extern "C" int fused_lmhead_vocab_shard_stats(const void* hidden, const void* w_shard, int64_t T, int64_t H,
                                              int64_t V_shard, int64_t v_begin, const int32_t* actions,
                                              grpo_vocab_stats* stats, float* logits_out, void* ws,
                                              size_t ws_bytes, hipStream_t s) {
  int st = check_fused_shapes(T, H, V_shard);
  if (st != GRPO_OK) return st;
  if (v_begin < 0 || v_begin >= ((int64_t)1 << 31) - V_shard) return GRPO_ERR_SHAPE;  // V_shard < 2^31 here
  if (!w_shard || (T > 0 && (!hidden || !actions || !stats))) return GRPO_ERR_ARG;
  if (!aligned(hidden, 16) || !aligned(w_shard, 16) || !aligned(stats, 8) || !aligned(logits_out, 16))
    return GRPO_ERR_ALIGN;
  const LmStatsWs L = lm_stats_ws_layout(T, H, V_shard);
  if (!ws || ws_bytes < L.total) return GRPO_ERR_WORKSPACE;
  if (!aligned(ws, kAlign)) return GRPO_ERR_ALIGN;
  if (T == 0) return GRPO_OK;
  char* w = static_cast<char*>(ws);
  const uint16_t* h16 = static_cast<const uint16_t*>(hidden);
  uint16_t* WT = reinterpret_cast<uint16_t*>(w + L.wt);
  float2* part = reinterpret_cast<float2*>(w + L.part);
  const int n_tiles = (int)((V_shard + TILE - 1) / TILE);
  lm_transpose(static_cast<const uint16_t*>(w_shard), h16, T, H, V_shard, 0, WT, nullptr, s);
  if (logits_out) {  // the shard's fp32 logits kept for the backward call
    PartialArgs pa{};
    pa.g = GemmArgs{h16, WT, H, H, (int)T, (int)V_shard, (int)H};
    pa.part = part;
    pa.n_tiles = n_tiles;
    pa.z = logits_out;
    pa.ldz = (int64_t)n_tiles * TILE;
    pa.part_t = nullptr;
    hipLaunchKernelGGL(k_lm_partial<true>, gemm_grid(T, V_shard), dim3(LmCfg::NT), 0, s, pa);
  } else {
    lm_pass1(h16, WT, T, H, V_shard, part, n_tiles, s);
  }
  RecordArgs ra{part, h16, WT, actions, stats, v_begin, V_shard, (int)T, (int)H, n_tiles};
  hipLaunchKernelGGL(k_lm_record, dim3((unsigned)T), dim3(256), 0, s, ra);
  return hipGetLastError() == hipSuccess ? GRPO_OK : GRPO_ERR_HIP;
}

extern "C" int fused_lmhead_grpo_vocab_shard(const void* hidden, const void* w_shard, int64_t T, int64_t H,
                                             int64_t V_shard, int64_t v_begin, int64_t V_total, int32_t vocab_chunk,
                                             const grpo_vocab_stats* stats, int32_t n_shards, const int32_t* actions,
                                             const float* behave_logp, const float* prox_logp, const float* adv,
                                             const grpo_segments* seg, const grpo_loss_params* p, double* loss_out,
                                             float* dhidden_partial, float* dw_shard, int32_t accumulate_dw,
                                             grpo_aux* aux, const float* logits_in, void* ws, size_t ws_bytes,
                                             hipStream_t s) {
  int st = check_loss_common(T, actions, behave_logp, adv, seg, p, loss_out);
  if (st != GRPO_OK) return st;
  if (!w_shard || !dw_shard || (T > 0 && (!hidden || !dhidden_partial || !stats))) return GRPO_ERR_ARG;
  st = check_fused_shapes(T, H, V_shard);
  if (st != GRPO_OK) return st;
  if (T > kMaxFusedLen || V_shard > kMaxFusedLen) return GRPO_ERR_SHAPE;
  // with the statistics call's logits, the shard is one chunk of V_shard rounded up to the tile
  const int64_t Vsp = (V_shard + TILE - 1) / TILE * TILE;
  if (logits_in) vocab_chunk = (int32_t)Vsp;
  if (vocab_chunk < 256 || vocab_chunk % 256 != 0) return GRPO_ERR_SHAPE;
  if (v_begin < 0 || V_total >= ((int64_t)1 << 31) || V_shard > V_total || v_begin > V_total - V_shard ||
      n_shards < 1 || n_shards > 65536)
    return GRPO_ERR_SHAPE;
  if (!aligned(hidden, 16) || !aligned(w_shard, 16) || !aligned(dhidden_partial, 16) || !aligned(dw_shard, 16) ||
      !aligned(stats, 8) || !aligned(logits_in, 16))
    return GRPO_ERR_ALIGN;
  const LmWs L = lm_ws_layout(T, H, V_shard, vocab_chunk, seg->n_traj);
  if (!ws || ws_bytes < L.total) return GRPO_ERR_WORKSPACE;
  if (!aligned(ws, kAlign)) return GRPO_ERR_ALIGN;
  char* w = static_cast<char*>(ws);
  const uint16_t* h16 = static_cast<const uint16_t*>(hidden);
  const uint16_t* W16 = static_cast<const uint16_t*>(w_shard);
  uint16_t* WT = reinterpret_cast<uint16_t*>(w + L.wt);
  uint16_t* hT = reinterpret_cast<uint16_t*>(w + L.ht);
  RowScale* rs = reinterpret_cast<RowScale*>(w + L.rs);
  uint16_t* D = reinterpret_cast<uint16_t*>(w + L.d);
  uint16_t* DT = reinterpret_cast<uint16_t*>(w + L.dt);
  const int Tp = (int)L.Tp;

  if (launch_segments(seg, T, V_total, actions, adv, p, w, L.loss, aux, s) != hipSuccess) return GRPO_ERR_HIP;
  if (T == 0) {
    if (!accumulate_dw) hipLaunchKernelGGL(k_fill_f32, dim3(1024), dim3(256), 0, s, dw_shard, H * V_shard, 0.f);
    if (hipGetLastError() != hipSuccess) return GRPO_ERR_HIP;
    return launch_reduce(T, seg->n_traj, w, L.loss, loss_out, aux, s) == hipSuccess ? GRPO_OK : GRPO_ERR_HIP;
  }
  lm_transpose(W16, h16, T, H, V_shard, Tp, logits_in ? nullptr : WT, hT, s);  // no W^T: nothing recomputed
  if (hipGetLastError() != hipSuccess) return GRPO_ERR_HIP;
  const bool timed = aux && aux->hot_begin && aux->hot_end;
  if (timed && hipEventRecord(aux->hot_begin, s) != hipSuccess) return GRPO_ERR_HIP;
  ShardScaleArgs sa;
  sa.tok = make_token_args(V_total, actions, behave_logp, prox_logp, adv, p, w, L.loss, aux);
  sa.stats = stats;
  sa.rs = rs;
  sa.v_begin = v_begin;
  sa.V = V_shard;
  sa.T = (int)T;
  sa.Tp = Tp;
  sa.n_shards = n_shards;
  hipLaunchKernelGGL(k_lm_shard_scale, dim3((unsigned)((Tp + 255) / 256)), dim3(256), 0, s, sa);
  if (hipGetLastError() != hipSuccess) return GRPO_ERR_HIP;
  if (logits_in) {
    // D, D^T of the whole shard from its stored logits, then dW (K = Tp) and the fp32 partial dhidden (K = V_shard)
    // in one launch, the long dW tiles first
    const BlockDArgs da{logits_in, nullptr, nullptr, 0, rs, D, DT, Vsp, (int)V_shard, Tp, 0};
    hipLaunchKernelGGL(k_lm_block_d, dim3(block_d_grid(Tp, Vsp, 0)), dim3(256), 0, s, da);
    DhDwArgs ba;
    ba.dh.g = GemmArgs{D, W16, Vsp, V_shard, (int)T, (int)H, (int)V_shard};
    ba.dh.acc = dhidden_partial;
    ba.dh.dh = nullptr;
    ba.dh.first = 1;
    ba.dh.last = 0;
    ba.dw.g = GemmArgs{hT, DT, Tp, Tp, (int)H, (int)V_shard, Tp};
    ba.dw.dw = dw_shard;
    ba.dw.V = V_shard;
    ba.dw.c0 = 0;
    ba.dw.accumulate = accumulate_dw;
    ba.dw_blocks = (int)gemm_grid(H, V_shard).x;
    hipLaunchKernelGGL(k_lm_dh_dw, dim3((unsigned)ba.dw_blocks + gemm_grid(T, H).x), dim3(LmCfg::NT), 0, s, ba);
  } else {
    lm_pass2(Pass2{h16, W16, WT, hT, rs, D, DT, dhidden_partial, nullptr, dw_shard, T, H, V_shard, Tp, vocab_chunk,
                   accumulate_dw},
             s);
  }
  if (hipGetLastError() != hipSuccess) return GRPO_ERR_HIP;
  if (timed && hipEventRecord(aux->hot_end, s) != hipSuccess) return GRPO_ERR_HIP;
  if (launch_reduce(T, seg->n_traj, w, L.loss, loss_out, aux, s) != hipSuccess) return GRPO_ERR_HIP;
  return GRPO_OK;
}
