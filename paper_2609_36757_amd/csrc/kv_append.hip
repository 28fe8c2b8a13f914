// KV-cache append for streaming inference (FastVR, Sec. 3.1, last paragraph):
// the new chunk's K and V rows [B, n_new, H, d] are copied into the caches
// [B, capacity, H, d] at token offset cache_len.  For every batch the source and
// the destination are one contiguous run of n_new * H * d bf16, so the kernel
// is a 16-byte-vector copy bounded by HBM bandwidth.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "launch.h"

namespace fastvr {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kUnroll = 4;

// grid: x = blocks over the run, y = batch, z = 0 (K) / 1 (V).  Units of 16 bytes.
__global__ __launch_bounds__(kThreads) void kv_append_kernel(u32x4* __restrict__ k_cache, u32x4* __restrict__ v_cache,
                                                             const u32x4* __restrict__ k_new,
                                                             const u32x4* __restrict__ v_new, int64_t cache_bs,
                                                             int64_t new_bs, int64_t dst_off, int64_t n16) {
  const int64_t b = blockIdx.y;
  u32x4* dst = (blockIdx.z == 0 ? k_cache : v_cache) + b * cache_bs + dst_off;
  const u32x4* src = (blockIdx.z == 0 ? k_new : v_new) + b * new_bs;
  const int64_t step = (int64_t)gridDim.x * kThreads * kUnroll;
  for (int64_t base = (int64_t)blockIdx.x * kThreads * kUnroll + threadIdx.x; base < n16; base += step) {
    u32x4 r[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t i = base + (int64_t)u * kThreads;
      if (i < n16) r[u] = __builtin_nontemporal_load(src + i);
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t i = base + (int64_t)u * kThreads;
      if (i < n16) dst[i] = r[u];
    }
  }
}

}  // namespace

hipError_t launch_kv_append(void* k_cache, void* v_cache, const void* k_new, const void* v_new, int64_t B,
                            int64_t H, int64_t d, int64_t capacity, int64_t cache_len, int64_t n_new,
                            hipStream_t stream) {
  const int64_t row16 = H * d / 8;  // 16-byte units per token
  const int64_t n16 = n_new * row16;
  int64_t blocks = (n16 + (int64_t)kThreads * kUnroll - 1) / ((int64_t)kThreads * kUnroll);
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(kv_append_kernel, dim3((unsigned)blocks, (unsigned)B, 2), dim3(kThreads), 0, stream,
                     static_cast<u32x4*>(k_cache), static_cast<u32x4*>(v_cache), static_cast<const u32x4*>(k_new),
                     static_cast<const u32x4*>(v_new), capacity * row16, n16, cache_len * row16, n16);
  return hipGetLastError();
}

}  // namespace fastvr
