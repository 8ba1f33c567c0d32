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

// Byte offset of a load that must read zeros: past the range of every descriptor here (a tile's 256 rows of at
// most 2^23 - 256 elements end at or below 2^32 - 2^17 bytes), with room for the load's 16 bytes below 2^32.
constexpr uint32_t kOobOffset = 0xFFFF0000u;

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
            kin ? (uint32_t)(row * g.lda + k0 + kv * 8) * 2u : kOobOffset, ra);
    }
#pragma unroll
    for (int q = 0; q < C::QB; ++q) {
      const int row = (q * C::NW + wave) * 8 + lrow, kv = (lane & 7) ^ lds_swizzle(row);
      const bool kin = k0 + kv * 8 < g.K;
      dma16(lb + (uint32_t)(q * C::NW * 8 * C::BK) * 2u,
            kin ? (uint32_t)(row * g.ldb + k0 + kv * 8) * 2u : kOobOffset, rb);
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


// ---- the same core with B's fragments loaded from memory straight into registers ------------------------------
// B in the fragment-packed layout: for every 32 rows of B (n-block nb) and every 16 columns of K (k-block kb) one
// 1 KB chunk, the 32 x 16 operand of one MFMA as its 64 lanes read it: lane l's 16 bytes are
// B[32 nb + l % 32][16 kb + 8 (l / 32) .. + 7].  Chunk (nb, kb) sits at ((nb * kb_count) + kb) KB, kb_count =
// 16-column blocks of K rounded up to whole 64-deep slabs, and rows past N and columns past K hold zeros.  A wave
// then fetches each of its B fragments with one fully coalesced 16-byte-per-lane load, one slab ahead, so the LDS
// carries only A (a third of the LDS traffic of the LDS-staged core goes away: A's slab writes and fragment reads
// stay, B's go).
__host__ __device__ constexpr int64_t packed_kb_count(int64_t K) { return (K + 63) / 64 * 4; }
__host__ __device__ constexpr int64_t packed_bytes(int64_t N, int64_t K) {
  return (N + 31) / 32 * packed_kb_count(K) * 1024;
}

// vmcnt(N) with the other counters left alone
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt holds 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x70 | 0xF00);
}

// One B fragment: 16 bytes per lane from rsrc + voff into v.  Inline asm, so that the compiler leaves the wait to
// the explicit vmcnt below (it cannot count the LDS DMA, which is asm too, and would wait for the wrong load); the
// register is an in-out operand so that the load writes the register the MFMAs read, with no copy in between.
__device__ __forceinline__ void frag_load(g_bf16x8& v, uint32_t voff, g_u32x4 rsrc) {
#pragma unroll
  for (int k = 0; k < 4; ++k) rsrc[k] = __builtin_amdgcn_readfirstlane(rsrc[k]);
  asm volatile("buffer_load_dwordx4 %0, %1, %2, 0 offen" : "+v"(v) : "v"(voff), "s"(rsrc) : "memory");
}

// C[m, n] = sum_k A[m, k] B[n, k] with g.A as in gemm_mainloop and g.B the packed B of an N x K matrix (g.ldb
// unused).  Same tile, waves, accumulator layout and order of the K sum as gemm_mainloop, so the accumulators are
// bit-identical to its.  LDS: two A slabs, C::BM * C::BK * 2 elements.
template <class C>
__device__ __forceinline__ void gemm_mainloop_packed(const GemmArgs& g, int m0, int n0,
                                                     g_f32x16 (&acc)[C::IB][C::JB], uint16_t* lds) {
  constexpr int STA = C::BM * C::BK;  // elements per A slab buffer
  static_assert(C::WTN % 32 == 0 && C::BN % 32 == 0, "whole n-blocks per wave and tile");
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / C::WGN, wn = wave % C::WGN;
  const int rows_a = min(C::BM, g.M - m0);
  const g_u32x4 ra = buffer_rsrc(g.A + (int64_t)m0 * g.lda, (uint32_t)(((int64_t)(rows_a - 1) * g.lda + g.K) * 2));
  // the tile's n-blocks: its own descriptor, so that n-blocks past N and loads past the last slab of the last
  // n-block read as zero
  const int64_t kbc = packed_kb_count(g.K);
  const int nb_tile = (int)min((int64_t)C::BN / 32, ((int64_t)g.N + 31) / 32 - n0 / 32);
  const g_u32x4 rbp = buffer_rsrc(reinterpret_cast<const char*>(g.B) + (int64_t)(n0 / 32) * kbc * 1024,
                                  (uint32_t)(nb_tile * kbc * 1024));
  const int lrow = lane >> 3;
  const uint32_t lds0 = (uint32_t)reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) uint16_t*)lds);
  auto issue = [&](int buf, int k0) {
    const uint32_t la = lds0 + (uint32_t)(buf * STA + wave * 8 * C::BK) * 2u;
#pragma unroll
    for (int q = 0; q < C::QA; ++q) {
      const int row = (q * C::NW + wave) * 8 + lrow, kv = (lane & 7) ^ lds_swizzle(row);
      const bool kin = k0 + kv * 8 < g.K;
      dma16(la + (uint32_t)(q * C::NW * 8 * C::BK) * 2u,
            kin ? (uint32_t)(row * g.lda + k0 + kv * 8) * 2u : kOobOffset, ra);
    }
  };
  uint32_t boff[C::JB];
#pragma unroll
  for (int j = 0; j < C::JB; ++j) boff[j] = (uint32_t)((wn * C::WTN / 32 + j) * kbc * 1024) + lane * 16u;
  g_bf16x8 fb[4][C::JB];  // B fragments of one slab: k-substep, n-block
#pragma unroll
  for (int s = 0; s < 4; ++s)
#pragma unroll
    for (int j = 0; j < C::JB; ++j) fb[s][j] = g_bf16x8{};
  auto bload = [&](int s, int kt) {
#pragma unroll
    for (int j = 0; j < C::JB; ++j) frag_load(fb[s][j], boff[j] + (uint32_t)(4 * kt + s) * 1024u, rbp);
  };
#pragma unroll
  for (int i = 0; i < C::IB; ++i)
#pragma unroll
    for (int j = 0; j < C::JB; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int fr = lane & 31, hi = lane >> 5;
  const int arow = (wm * C::WTM + fr) * C::BK;
  int sw[4];
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) sw[ks] = ((2 * ks + hi) ^ lds_swizzle(fr)) * 8;
  g_bf16x8 fa[2][C::IB];
  auto read = [&](int f, int buf, int ks) {
    const uint16_t* s = lds + buf * STA;
#pragma unroll
    for (int i = 0; i < C::IB; ++i) fa[f][i] = *reinterpret_cast<const g_bf16x8*>(s + arow + i * 32 * C::BK + sw[ks]);
  };
  // the MFMAs of k-substep s with the A reads of the next substep interleaved (one read, one MFMA)
  auto mma = [&](int f, int s) {
#pragma unroll
    for (int i = 0; i < C::IB; ++i)
#pragma unroll
      for (int j = 0; j < C::JB; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[f][i], fb[s][j], acc[i][j], 0, 0, 0);
#pragma unroll
    for (int x = 0; x < C::IB; ++x) {
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
    }
    __builtin_amdgcn_sched_group_barrier(0x008, C::IB * C::JB - C::IB, 0);
  };
  // Per wave and slab kt the vector-memory queue gets, oldest first: B(kt+1, s) for s = 0, 1, 2, each after the
  // MFMAs of substep s (which were the last readers of those registers), the A DMA of slab kt+2 after the
  // barrier, B(kt+1, 3) after substep 3.  Counters drain in order, so substep s of slab kt, which needs B(kt, s),
  // leaves WB younger operations in flight, and the barrier, which needs this wave's DMA of slab kt+1, WD.  Loads
  // past the last slab are issued as well (they read zeros or values nobody uses) so that the counts are the same
  // on every slab; the sched_barriers keep the compiler from moving MFMAs above a wait it cannot see the reason for.
  constexpr int WB = 3 * C::JB + C::QA, WD = 4 * C::JB;
  const int nk = (g.K + C::BK - 1) / C::BK;
  issue(0, 0);
  issue(1, C::BK);
#pragma unroll
  for (int s = 0; s < 4; ++s) bload(s, 0);
  wait_vm0();
  wait_lgkm0();  // also publishes what the caller stored to LDS before the mainloop
  barrier();
  read(0, 0, 0);
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    wait_vm<WB>();
    __builtin_amdgcn_sched_barrier(0);
    read(1, buf, 1);
    mma(0, 0);
    __builtin_amdgcn_sched_barrier(0);
    bload(0, kt + 1);
    wait_vm<WB>();
    __builtin_amdgcn_sched_barrier(0);
    read(0, buf, 2);
    mma(1, 1);
    __builtin_amdgcn_sched_barrier(0);
    bload(1, kt + 1);
    wait_vm<WB>();
    __builtin_amdgcn_sched_barrier(0);
    read(1, buf, 3);
    mma(0, 2);
    __builtin_amdgcn_sched_barrier(0);
    bload(2, kt + 1);
    wait_lgkm0();  // this wave's reads of slab kt are done
    wait_vm<WD>();  // this wave's DMA of slab kt + 1 has landed
    barrier();      // ... and every wave's
    issue(buf, (kt + 2) * C::BK);
    wait_vm<WB>();
    __builtin_amdgcn_sched_barrier(0);
    read(0, buf ^ 1, 0);
    mma(1, 3);
    __builtin_amdgcn_sched_barrier(0);
    bload(3, kt + 1);
  }
  // The last slab's loads of the next one are still in flight.  The compiler cannot see them (asm), so the wait
  // names every fragment register: they stay allocated until the data has landed, and nothing of the caller's
  // can be given a register that a late load would then overwrite.  The barrier then keeps any wave from reusing
  // the LDS before every wave's last (zero) DMA has landed in it.
#pragma unroll
  for (int s = 0; s < 4; ++s)
#pragma unroll
    for (int j = 0; j < C::JB; ++j) asm volatile("s_waitcnt vmcnt(0)" : "+v"(fb[s][j])::"memory");
  barrier();
}

}  // namespace grpo
