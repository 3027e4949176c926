// Streaming-copy probe: the practical HBM ceiling the benchmark reports next
// to the 8 TB/s peak.  A plain device-to-device copy of one contiguous
// buffer in several launch shapes; the benchmark takes the fastest.  It is
// measurement infrastructure, not part of the eviction step: it is built
// into its own library (libcopyprobe.so) and declared nowhere in epikv.h.
//
// Shapes (variant ids): workgroups of NT threads with V 16-byte vectors per
// thread, each copying one contiguous block of NT * V * 16 bytes (all loads
// issued before the stores), non-temporal or plain loads and stores,
// optionally with unused LDS reserved so that fewer workgroups share a CU;
// and a grid-stride form with a fixed grid of 8 workgroups per CU.
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;  // grid-stride form

template <bool NT>
__device__ __forceinline__ u32x4 ld(const u32x4* p) {
  if (NT) return __builtin_nontemporal_load(p);
  return *p;
}
template <bool NT>
__device__ __forceinline__ void st(u32x4* p, u32x4 v) {
  if (NT)
    __builtin_nontemporal_store(v, p);
  else
    *p = v;
}

// Workgroup w copies vectors [w*V*T, (w+1)*V*T): thread t takes vectors
// t, t+T, ... of the block, so every load instruction of a wavefront reads
// 1 KiB contiguous.
template <int T, int V, bool NT>
__global__ __launch_bounds__(T) void k_copy_block(const u32x4* __restrict__ src,
                                                 u32x4* __restrict__ dst, int64_t n_vec) {
  const int64_t base = (int64_t)blockIdx.x * (V * T) + threadIdx.x;
  u32x4 v[V];
#pragma unroll
  for (int k = 0; k < V; ++k) {
    const int64_t i = base + (int64_t)k * T;
    if (i < n_vec) v[k] = ld<NT>(src + i);
  }
#pragma unroll
  for (int k = 0; k < V; ++k) {
    const int64_t i = base + (int64_t)k * T;
    if (i < n_vec) st<NT>(dst + i, v[k]);
  }
}

// Fixed grid; each workgroup walks blocks of V*256 vectors with a stride of
// the grid.
template <int V>
__global__ __launch_bounds__(kThreads) void k_copy_stride(const u32x4* __restrict__ src,
                                                         u32x4* __restrict__ dst, int64_t n_vec) {
  const int64_t step = (int64_t)gridDim.x * (V * kThreads);
  for (int64_t base = (int64_t)blockIdx.x * (V * kThreads) + threadIdx.x; base < n_vec;
       base += step) {
    u32x4 v[V];
#pragma unroll
    for (int k = 0; k < V; ++k) {
      const int64_t i = base + (int64_t)k * kThreads;
      if (i < n_vec) v[k] = ld<true>(src + i);
    }
#pragma unroll
    for (int k = 0; k < V; ++k) {
      const int64_t i = base + (int64_t)k * kThreads;
      if (i < n_vec) st<true>(dst + i, v[k]);
    }
  }
}

// LDS_KIB > 0 reserves that much unused LDS per workgroup, capping how many
// share a CU (160 KiB of LDS per CU).
template <int T, int V, bool NT, int LDS_KIB = 0>
hipError_t block_launch(const void* s, void* d, int64_t n_vec, hipStream_t st) {
  const int64_t per = (int64_t)V * T;
  const int64_t blocks = (n_vec + per - 1) / per;
  if (blocks > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL((k_copy_block<T, V, NT>), dim3((unsigned)blocks), dim3(T), LDS_KIB * 1024,
                     st, (const u32x4*)s, (u32x4*)d, n_vec);
  return hipGetLastError();
}

template <int V>
hipError_t stride_launch(const void* s, void* d, int64_t n_vec, hipStream_t st) {
  hipLaunchKernelGGL((k_copy_stride<V>), dim3(256 * 8), dim3(kThreads), 0, st, (const u32x4*)s,
                     (u32x4*)d, n_vec);
  return hipGetLastError();
}

struct Variant {
  const char* name;
  hipError_t (*fn)(const void*, void*, int64_t, hipStream_t);
};

const Variant kVariants[] = {
    {"block 4 KiB, 256 threads x 1 vector, non-temporal", block_launch<256, 1, true>},
    {"block 8 KiB, 256 threads x 2 vectors, non-temporal", block_launch<256, 2, true>},
    {"block 16 KiB, 256 threads x 4 vectors, non-temporal", block_launch<256, 4, true>},
    {"block 32 KiB, 256 threads x 8 vectors, non-temporal", block_launch<256, 8, true>},
    {"block 1 KiB, 64 threads x 1 vector, non-temporal", block_launch<64, 1, true>},
    {"block 2 KiB, 128 threads x 1 vector, non-temporal", block_launch<128, 1, true>},
    {"block 4 KiB, 256 threads x 1 vector, non-temporal, 6 workgroups/CU",
     block_launch<256, 1, true, 24>},
    {"block 4 KiB, 256 threads x 1 vector, plain", block_launch<256, 1, false>},
    {"block 16 KiB, 256 threads x 4 vectors, plain", block_launch<256, 4, false>},
    {"grid-stride 8 workgroups/CU, 2 vectors/thread, non-temporal", stride_launch<2>},
    {"grid-stride 8 workgroups/CU, 4 vectors/thread, non-temporal", stride_launch<4>},
};
constexpr int kNumVariants = sizeof(kVariants) / sizeof(kVariants[0]);

}  // namespace

#define PROBE_EXPORT extern "C" __attribute__((visibility("default")))

// Number of copy shapes.
PROBE_EXPORT int copy_probe_variants() { return kNumVariants; }

// Description of a shape (NULL for an unknown id).
PROBE_EXPORT const char* copy_probe_name(int variant) {
  return (variant >= 0 && variant < kNumVariants) ? kVariants[variant].name : nullptr;
}

// Copy `bytes` (a multiple of 16; both pointers 16-byte aligned device
// memory, not overlapping) from src to dst on `stream` with shape
// `variant`.  Returns 0, or -1 for invalid arguments, -2 if the launch
// failed.
PROBE_EXPORT int copy_probe(const void* src, void* dst, size_t bytes, int variant,
                            hipStream_t stream) {
  if (!src || !dst || (bytes & 15u) || variant < 0 || variant >= kNumVariants) return -1;
  if (((uintptr_t)src & 15u) || ((uintptr_t)dst & 15u)) return -1;
  const uintptr_t a = (uintptr_t)src, b = (uintptr_t)dst;
  if (a < b + bytes && b < a + bytes) return -1;
  if (bytes == 0) return 0;
  return kVariants[variant].fn(src, dst, (int64_t)(bytes / 16), stream) == hipSuccess ? 0 : -2;
}
