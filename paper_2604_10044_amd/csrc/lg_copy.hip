// lg_copy.hip -- streaming copy used to measure the achievable HBM bandwidth of the device
// (reported beside the published peak). Each lane moves 16 B per access, four accesses in
// flight, grid-stride over the buffer; loads and stores are non-temporal (every byte is touched
// once), the access form the attention sweep and the compaction use.
#include "lg_internal.h"

namespace lg {

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ u32x4_t ld_nt(const u32x4_t* p) { return __builtin_nontemporal_load(p); }
__device__ __forceinline__ void st_nt(u32x4_t* p, u32x4_t v) { __builtin_nontemporal_store(v, p); }

__global__ __launch_bounds__(256) void copy_kernel(const u32x4_t* __restrict__ src,
                                                   u32x4_t* __restrict__ dst, size_t n) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (; i + 3 * stride < n; i += 4 * stride) {
    const u32x4_t a = ld_nt(src + i), b = ld_nt(src + i + stride), c = ld_nt(src + i + 2 * stride),
                  d = ld_nt(src + i + 3 * stride);
    st_nt(dst + i, a);
    st_nt(dst + i + stride, b);
    st_nt(dst + i + 2 * stride, c);
    st_nt(dst + i + 3 * stride, d);
  }
  for (; i < n; i += stride) st_nt(dst + i, ld_nt(src + i));
}

hipError_t launch_copy(const void* src, void* dst, size_t bytes, hipStream_t st) {
  const size_t n = bytes / 16;
  size_t blocks = (n + 255) / 256;
  if (blocks > 256 * 32) blocks = 256 * 32;
  hipLaunchKernelGGL(copy_kernel, dim3((unsigned)blocks), dim3(256), 0, st, (const u32x4_t*)src,
                     (u32x4_t*)dst, n);
  return hipGetLastError();
}

}  // namespace lg
