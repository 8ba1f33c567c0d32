// bf16 GEMM core for gfx950: C[m, n] = sum_k A[m, k] B[n, k], both operands K-contiguous, fp32 accumulation on
// v_mfma_f32_32x32x16_bf16.  A workgroup of WGM x WGN waves computes a BM x BN tile, each wave a
// (BM/WGM) x (BN/WGN) block of 32 x 32 MFMA tiles.
//
// K is walked in slabs of BK = 64.  A slab goes from global memory straight into LDS (buffer_load_dwordx4 ...
// lds: no staging registers), written as inline asm so that the compiler does not hold every LDS read back until
// all LDS DMA in flight has landed; the explicit waits below order them instead.  Rows are 128 B, unpadded, and
// the eight 16-byte vectors of a row are permuted (lds_swizzle) so that fragment reads are free of bank
// conflicts.  Two LDS buffers: the DMA of slab k + 2 is issued right after the single barrier of
// step k, so it has a whole step to land, and the MFMA fragments are double-buffered in registers.
// Out-of-range rows and K columns read as zero through the buffer descriptor's range check.
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
  int M, N, K;        // K a multiple of 8; lda, ldb multiples of 8
};

template <int BM_, int BN_, int WGM_, int WGN_>
struct GemmCfg {
  static constexpr int BM = BM_, BN = BN_, BK = 64, WGM = WGM_, WGN = WGN_;
  static constexpr int NW = WGM * WGN, NT = 64 * NW;
  static constexpr int WTM = BM / WGM, WTN = BN / WGN;
  static constexpr int IB = WTM / 32, JB = WTN / 32;
  static constexpr int QA = BM / 8 / NW, QB = BN / 8 / NW;  // DMA instructions per wave per slab
  static constexpr int STAGE = (BM + BN) * BK;               // bf16 elements per LDS buffer
  static constexpr int LDS_BYTES = 2 * STAGE * 2;
  static_assert(BM % (8 * NW) == 0 && BN % (8 * NW) == 0, "whole DMA instructions per wave");
  static_assert(IB * JB >= IB + JB, "enough MFMAs to interleave the next fragment reads with");
};

// Output coordinates (relative to the tile) of accumulator r of block (i, j) in lane `lane` of wave (wm, wn):
// 32x32x16 layout, column lane % 32, row 8 (r / 4) + 4 (lane / 32) + r % 4.
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
// workgroups sharing an XCD's L2 reuse each other's A and B slabs.  Launch a multiple of 8 workgroups.
// Returns false past the last tile.
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

__device__ __forceinline__ g_u32x4 buffer_rsrc(const void* base, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  g_u32x4 r = {(uint32_t)a, (uint32_t)(a >> 32) & 0xffffu, bytes, 0x00020000u};
  return r;
}

// LDS slot permutation of a slab row (eight 16-byte slots per 128-byte row).  A fragment read takes
// one slot from each of 32 consecutive rows; the LDS serves 16 lanes (256 bytes) at a time, so every 16
// consecutive rows must spread over the 8 slots x 2 row parities, and every 8 over the 8 slots.
__device__ __forceinline__ int lds_swizzle(int row) { return (row & 7) ^ ((row >> 3) & 1); }

// 16 bytes per lane from rsrc + voff into LDS at lds_base + 16 * lane (lds_base wave-uniform).  M0 carries the
// LDS address; nothing else in these kernels uses it.  One wait state separates the write of M0 from the LDS DMA
// that reads it (the compiler inserts the same for its own LDS DMA; it cannot see inside this asm).
__device__ __forceinline__ void dma16(uint32_t lds_base, uint32_t voff, g_u32x4 rsrc) {
  // the operands are wave-uniform; readfirstlane keeps them in SGPRs whatever the register allocator prefers
  lds_base = __builtin_amdgcn_readfirstlane(lds_base);
#pragma unroll
  for (int k = 0; k < 4; ++k) rsrc[k] = __builtin_amdgcn_readfirstlane(rsrc[k]);
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds" ::"s"(lds_base), "v"(voff), "s"(rsrc)
               : "memory", "m0");
}

// The waits are builtins, not inline asm, so that the compiler's own wait insertion knows the counters have
// drained: behind an opaque wait it assumed the last fragment reads before the barrier were still in flight, and
// held the last MFMA group of every step back until the next slab's first reads had landed.
__device__ __forceinline__ void wait_vm0() { __builtin_amdgcn_s_waitcnt(0x0F70); }   // vmcnt(0)
__device__ __forceinline__ void wait_lgkm0() { __builtin_amdgcn_s_waitcnt(0xC07F); }  // lgkmcnt(0)
__device__ __forceinline__ void barrier() { asm volatile("s_barrier" ::: "memory"); }

template <class C>
__device__ __forceinline__ void gemm_mainloop(const GemmArgs& g, int m0, int n0, g_f32x16 (&acc)[C::IB][C::JB],
                                               uint16_t* lds) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / C::WGN, wn = wave % C::WGN;
  const int rows_a = min(C::BM, g.M - m0), rows_b = min(C::BN, g.N - n0);
  const g_u32x4 ra = buffer_rsrc(g.A + (int64_t)m0 * g.lda, (uint32_t)(((int64_t)(rows_a - 1) * g.lda + g.K) * 2));
  const g_u32x4 rb = buffer_rsrc(g.B + (int64_t)n0 * g.ldb, (uint32_t)(((int64_t)(rows_b - 1) * g.ldb + g.K) * 2));
  // DMA instruction q of this wave fills slab rows 8 (q NW + wave) .. + 7; lane -> row lane / 8, LDS slot
  // lane % 8, which holds global vector slot ^ swizzle(row)
  const int lrow = lane >> 3;
  const uint32_t lds0 = (uint32_t)reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) uint16_t*)lds);
  auto issue = [&](int buf, int k0) {
    const uint32_t la = lds0 + (uint32_t)(buf * C::STAGE + wave * 8 * C::BK) * 2u;
    const uint32_t lb = la + (uint32_t)(C::BM * C::BK) * 2u;
#pragma unroll
    for (int q = 0; q < C::QA; ++q) {
      const int row = (q * C::NW + wave) * 8 + lrow, kv = (lane & 7) ^ lds_swizzle(row);
      const bool kin = k0 + kv * 8 < g.K;  // vectors past K read as zero
      dma16(la + (uint32_t)(q * C::NW * 8 * C::BK) * 2u,
            kin ? (uint32_t)(row * g.lda + k0 + kv * 8) * 2u : 0x80000000u, ra);
    }
#pragma unroll
    for (int q = 0; q < C::QB; ++q) {
      const int row = (q * C::NW + wave) * 8 + lrow, kv = (lane & 7) ^ lds_swizzle(row);
      const bool kin = k0 + kv * 8 < g.K;
      dma16(lb + (uint32_t)(q * C::NW * 8 * C::BK) * 2u,
            kin ? (uint32_t)(row * g.ldb + k0 + kv * 8) * 2u : 0x80000000u, rb);
    }
  };
#pragma unroll
  for (int i = 0; i < C::IB; ++i)
#pragma unroll
    for (int j = 0; j < C::JB; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int fr = lane & 31, hi = lane >> 5;
  const int arow = (wm * C::WTM + fr) * C::BK, brow = C::BM * C::BK + (wn * C::WTN + fr) * C::BK;
  int sw[4];
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) sw[ks] = ((2 * ks + hi) ^ lds_swizzle(fr)) * 8;

  g_bf16x8 fa[2][C::IB], fb[2][C::JB];
  auto read = [&](int f, int buf, int ks) {
    const uint16_t* s = lds + buf * C::STAGE;
#pragma unroll
    for (int i = 0; i < C::IB; ++i) fa[f][i] = *reinterpret_cast<const g_bf16x8*>(s + arow + i * 32 * C::BK + sw[ks]);
#pragma unroll
    for (int j = 0; j < C::JB; ++j) fb[f][j] = *reinterpret_cast<const g_bf16x8*>(s + brow + j * 32 * C::BK + sw[ks]);
  };
  // the MFMAs of one fragment set, with the LDS reads of the next one interleaved (one read, one MFMA)
  auto mma = [&](int f) {
#pragma unroll
    for (int i = 0; i < C::IB; ++i)
#pragma unroll
      for (int j = 0; j < C::JB; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[f][i], fb[f][j], acc[i][j], 0, 0, 0);
#pragma unroll
    for (int x = 0; x < C::IB + C::JB; ++x) {
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
    }
    __builtin_amdgcn_sched_group_barrier(0x008, C::IB * C::JB - (C::IB + C::JB), 0);
  };

  const int nk = (g.K + C::BK - 1) / C::BK;
  issue(0, 0);
  if (nk > 1) issue(1, C::BK);
  wait_vm0();
  wait_lgkm0();  // also publishes what the caller stored to LDS before the mainloop
  barrier();
  read(0, 0, 0);
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    read(1, buf, 1);
    mma(0);
    read(0, buf, 2);
    mma(1);
    read(1, buf, 3);
    mma(0);
    wait_lgkm0();  // this wave's reads of slab kt are done
    wait_vm0();    // this wave's DMA of slab kt + 1 has landed
    barrier();     // ... and every wave's
    if (kt + 2 < nk) issue(buf, (kt + 2) * C::BK);
    if (kt + 1 < nk) read(0, buf ^ 1, 0);
    mma(1);
  }
}

}  // namespace grpo
