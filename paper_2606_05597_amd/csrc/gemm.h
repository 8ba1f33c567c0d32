// bf16 GEMM core for gfx950: C[m, n] = sum_k A[m, k] B[n, k], both operands K-contiguous, fp32 accumulation
// on v_mfma_f32_32x32x16_bf16.  One workgroup computes a BM x BN tile with WGM x WGN waves; each wave a
// (BM/WGM) x (BN/WGN) sub-tile of 32x32 MFMA blocks.  The K loop stages BK-wide slabs of A and B through
// double-buffered LDS (rows padded by 16 bytes); the next slab's global loads are in flight while the current
// one feeds the matrix cores.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace grpo {

typedef uint32_t g_u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 g_bf16x8 __attribute__((ext_vector_type(8)));
typedef float g_f32x16 __attribute__((ext_vector_type(16)));

struct GemmArgs {
  const uint16_t* A;  // [M, K], row stride lda (elements)
  const uint16_t* B;  // [N, K], row stride ldb
  int64_t lda, ldb;
  int M, N, K;        // K a multiple of 8
};

template <int BM_, int BN_, int BK_, int WGM_, int WGN_>
struct GemmCfg {
  static constexpr int BM = BM_, BN = BN_, BK = BK_, WGM = WGM_, WGN = WGN_;
  static constexpr int NT = 64 * WGM * WGN;             // threads
  static constexpr int WTM = BM / WGM, WTN = BN / WGN;  // wave tile
  static constexpr int IB = WTM / 32, JB = WTN / 32;    // 32x32 MFMA blocks per wave
  static constexpr int LDK = BK + 8;                    // LDS row stride (bf16)
  static constexpr int VPR = BK / 8;                    // 16-byte vectors per slab row
  static constexpr int RPP = NT / VPR;                  // slab rows covered by one pass of the loader
  static constexpr int LA = BM / RPP, LB = BN / RPP;    // loader passes for A and B
  static constexpr int LDS_BYTES = 2 * (BM + BN) * LDK * 2;
  static_assert(BM % (32 * WGM) == 0 && BN % (32 * WGN) == 0, "wave tiles are whole MFMA blocks");
  static_assert(NT % VPR == 0 && BM % RPP == 0 && BN % RPP == 0, "loader covers the slab");
};

// Output coordinates (relative to the tile) of accumulator r of block (i, j) in lane `lane` of wave (wm, wn):
// 32x32x16 layout, column lane%32, rows 8(r/4) + 4(lane/32) + r%4.
template <class C>
__device__ __forceinline__ int gemm_row(int wm, int i, int r, int lane) {
  return wm * C::WTM + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
}
template <class C>
__device__ __forceinline__ int gemm_col(int wn, int j, int lane) {
  return wn * C::WTN + j * 32 + (lane & 31);
}

// XCD-aware grouped tile order.  Workgroups are dispatched to the 8 XCDs round-robin, so workgroup b runs on
// XCD b % 8; giving each XCD a contiguous range of logical tiles, ordered GM M-tiles at a time, lets the
// workgroups sharing an XCD's L2 reuse each other's A and B slabs.  Launch a multiple of 8 workgroups;
// returns false past the last tile.
template <int GM = 8>
__device__ __forceinline__ bool gemm_tile_of(int bid, int nblocks, int tiles_m, int tiles_n, int& tm, int& tn) {
  const int total = tiles_m * tiles_n;
  const int per = (nblocks + 7) / 8;
  const int L = (bid % 8) * per + bid / 8;
  if (L >= total) return false;
  const int group = GM * tiles_n;
  const int g = L / group, first = g * GM;
  const int gm = min(tiles_m - first, GM);
  tm = first + (L % group) % gm;
  tn = (L % group) / gm;
  return true;
}

template <class C>
__device__ __forceinline__ void gemm_mainloop(const GemmArgs& g, int m0, int n0, g_f32x16 (&acc)[C::IB][C::JB],
                                              uint16_t* sA, uint16_t* sB) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / C::WGN, wn = wave % C::WGN;
  const int lr = tid / C::VPR, lv = tid % C::VPR;  // loader: rows lr + RPP*q, vector lv
  g_u32x4 ra[C::LA], rb[C::LB];
  const g_u32x4 zero = {0u, 0u, 0u, 0u};
  auto gload = [&](int k0) {
    const int k = k0 + lv * 8;
#pragma unroll
    for (int q = 0; q < C::LA; ++q) {
      const int m = m0 + lr + C::RPP * q;
      ra[q] = (m < g.M && k < g.K) ? *reinterpret_cast<const g_u32x4*>(g.A + (int64_t)m * g.lda + k) : zero;
    }
#pragma unroll
    for (int q = 0; q < C::LB; ++q) {
      const int n = n0 + lr + C::RPP * q;
      rb[q] = (n < g.N && k < g.K) ? *reinterpret_cast<const g_u32x4*>(g.B + (int64_t)n * g.ldb + k) : zero;
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int q = 0; q < C::LA; ++q)
      *reinterpret_cast<g_u32x4*>(sA + (buf * C::BM + lr + C::RPP * q) * C::LDK + lv * 8) = ra[q];
#pragma unroll
    for (int q = 0; q < C::LB; ++q)
      *reinterpret_cast<g_u32x4*>(sB + (buf * C::BN + lr + C::RPP * q) * C::LDK + lv * 8) = rb[q];
  };
#pragma unroll
  for (int i = 0; i < C::IB; ++i)
#pragma unroll
    for (int j = 0; j < C::JB; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int nk = (g.K + C::BK - 1) / C::BK;
  gload(0);
  sstore(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) gload((kt + 1) * C::BK);
#pragma unroll
    for (int ks = 0; ks < C::BK / 16; ++ks) {
      g_bf16x8 a[C::IB], b[C::JB];
      const int kk = ks * 16 + (lane >> 5) * 8;
#pragma unroll
      for (int i = 0; i < C::IB; ++i)
        a[i] = *reinterpret_cast<const g_bf16x8*>(sA + (buf * C::BM + wm * C::WTM + i * 32 + (lane & 31)) * C::LDK + kk);
#pragma unroll
      for (int j = 0; j < C::JB; ++j)
        b[j] = *reinterpret_cast<const g_bf16x8*>(sB + (buf * C::BN + wn * C::WTN + j * 32 + (lane & 31)) * C::LDK + kk);
#pragma unroll
      for (int i = 0; i < C::IB; ++i)
#pragma unroll
        for (int j = 0; j < C::JB; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) sstore(buf ^ 1);
    __syncthreads();
  }
}

}  // namespace grpo
