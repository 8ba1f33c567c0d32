// Plain streaming copies, the memory-only ceiling the row pass is measured against: the row pass reads each
// logits row once and writes its dlogits row once, so a copy of the logits buffer into the dlogits buffer moves
// the same bytes in the same directions between the same two allocations (whose physical placement sets the
// rate HBM reaches for a mixed read/write stream).  Only the benchmark uses this library; it is not part of
// libgrpo's ABI.
//
// Each variant is a grid-stride loop of 16-byte non-temporal loads and stores, U vectors in flight per thread,
// all U loads issued before the U stores.
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// LDS_PAD > 0 reserves that many bytes of LDS per workgroup, so that (like the row kernel) only one workgroup fits a
// CU; the pad is never read or written.
template <int NT, int U, int LDS_PAD = 0>
__global__ __launch_bounds__(NT) void k_stream_copy(const u32x4* __restrict__ src, u32x4* __restrict__ dst,
                                                     int64_t n) {
  if constexpr (LDS_PAD > 0) {
    __shared__ uint32_t pad[LDS_PAD / 4];
    asm volatile("" ::"r"(pad));
  }
  const int64_t stride = (int64_t)gridDim.x * NT * U;
  for (int64_t base = (int64_t)blockIdx.x * NT * U + threadIdx.x; base < n; base += stride) {
    u32x4 x[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t i = base + (int64_t)u * NT;
      if (i < n) x[u] = __builtin_nontemporal_load(src + i);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t i = base + (int64_t)u * NT;
      if (i < n) __builtin_nontemporal_store(x[u], dst + i);
    }
  }
}

struct Variant {
  void (*k)(const u32x4*, u32x4*, int64_t);
  int nt, u;
  int wg_per_cu;  // workgroups per compute unit in the grid (0: one per NT*U vectors, as many as the copy needs)
  const char* name;
};

static const Variant kVariants[] = {
    {k_stream_copy<256, 4>, 256, 4, 0, "256 threads x 4 vectors, one workgroup per 16 KiB"},
    {k_stream_copy<1024, 16, 100000>, 1024, 16, 0,
     "1024 threads x 16 vectors, one workgroup per 256 KiB, one per CU at a time (LDS)"},
    {k_stream_copy<1024, 4>, 1024, 4, 1, "1024 threads x 4 vectors, one workgroup per CU"},
    {k_stream_copy<1024, 16>, 1024, 16, 1, "1024 threads x 16 vectors, one workgroup per CU"},
    {k_stream_copy<256, 16>, 256, 16, 8, "256 threads x 16 vectors, 8 workgroups per CU"},
    {k_stream_copy<256, 4>, 256, 4, 4, "256 threads x 4 vectors, 4 workgroups per CU"},
};

extern "C" int stream_copy_variants(void) { return (int)(sizeof(kVariants) / sizeof(kVariants[0])); }

extern "C" const char* stream_copy_name(int v) {
  return (v >= 0 && v < stream_copy_variants()) ? kVariants[v].name : "";
}

// Copies n_vec 16-byte vectors from src to dst (both 16-byte aligned device pointers) with variant v on stream s.
// Returns 0, -1 for a bad variant or arguments, or the HIP error of the launch.
extern "C" int stream_copy(int v, const void* src, void* dst, int64_t n_vec, hipStream_t s) {
  if (v < 0 || v >= stream_copy_variants() || n_vec < 0 || !src || !dst) return -1;
  if (((uintptr_t)src | (uintptr_t)dst) & 15) return -1;
  if (n_vec == 0) return 0;
  const Variant& k = kVariants[v];
  int64_t grid;
  if (k.wg_per_cu == 0) {
    const int64_t per_wg = (int64_t)k.nt * k.u;
    grid = (n_vec + per_wg - 1) / per_wg;
    if (grid > (int64_t)1 << 30) grid = (int64_t)1 << 30;
  } else {
    hipDevice_t dev = 0;
    int n_cu = 0;
    if (hipStreamGetDevice(s, &dev) != hipSuccess ||
        hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n_cu < 1)
      return -1;
    grid = (int64_t)n_cu * k.wg_per_cu;
  }
  hipLaunchKernelGGL(k.k, dim3((unsigned)grid), dim3(k.nt), 0, s, static_cast<const u32x4*>(src),
                     static_cast<u32x4*>(dst), n_vec);
  return (int)hipGetLastError();
}
