// One-step latent update (FastVR, Sec. 3.2, Eq. 9; the update used at inference,
// Sec. 4.1): z_hat = z_LQ - sigma_tau * v, element by element over the
// flattened latent.
//
// z_LQ and v are bf16; each element is one fused multiply-add in fp32
// (fma(-sigma, v, z): the exact value z - sigma * v rounded once), stored as
// fp32 or rounded again to bf16 (nearest even).  The kernel is bound by HBM
// bandwidth and runs a grid-stride loop: for fp32 output each lane takes 4
// elements (8-byte loads, one 16-byte store), so each store instruction of a
// wave writes one contiguous kilobyte; for bf16 output 8 elements (16-byte
// loads and store).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gfx950_ops.h"
#include "launch.h"

namespace fastvr {
namespace {

using namespace dev;

constexpr int kThreads = 256;
constexpr int kUnroll = 2;
// fp32 output: 4 elements per lane (8-byte loads, one 16-byte store, so every
// store instruction of a wave writes one contiguous kilobyte) instead of 8
#ifndef FASTVR_OS_LANE4
#define FASTVR_OS_LANE4 1
#endif
#ifndef FASTVR_OS_NT_STORE
#define FASTVR_OS_NT_STORE 1
#endif

template <typename T, typename P>
__device__ __forceinline__ void st(T v, P* p) {
#if FASTVR_OS_NT_STORE
  __builtin_nontemporal_store(v, p);
#else
  *p = v;
#endif
}

template <bool OUT_BF16>
__device__ __forceinline__ void update8(const u32x4 zz, const u32x4 vv, float neg_sigma, void* out, int64_t i) {
  const bf16x8 zb = __builtin_bit_cast(bf16x8, zz);
  const bf16x8 vb = __builtin_bit_cast(bf16x8, vv);
  float r[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) r[e] = __builtin_fmaf(neg_sigma, (float)vb[e], (float)zb[e]);
  if (OUT_BF16) {
    bf16x8 o;
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = (__bf16)r[e];
    st(__builtin_bit_cast(u32x4, o), static_cast<u32x4*>(out) + i);
  } else {
    f32x4* o = static_cast<f32x4*>(out) + 2 * i;
    st(f32x4{r[0], r[1], r[2], r[3]}, o);
    st(f32x4{r[4], r[5], r[6], r[7]}, o + 1);
  }
}

// n8 groups of 8 elements, then `tail` (< 8) single elements after them
template <bool OUT_BF16>
__global__ __launch_bounds__(kThreads) void one_step_kernel(const u32x4* __restrict__ z, const u32x4* __restrict__ v,
                                                            void* __restrict__ out, int64_t n8, int tail,
                                                            float neg_sigma) {
  const int64_t step = (int64_t)gridDim.x * kThreads * kUnroll;
  for (int64_t base = (int64_t)blockIdx.x * kThreads * kUnroll + threadIdx.x; base < n8; base += step) {
    u32x4 zr[kUnroll], vr[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t i = base + (int64_t)u * kThreads;
      if (i < n8) {
        zr[u] = __builtin_nontemporal_load(z + i);
        vr[u] = __builtin_nontemporal_load(v + i);
      }
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t i = base + (int64_t)u * kThreads;
      if (i < n8) update8<OUT_BF16>(zr[u], vr[u], neg_sigma, out, i);
    }
  }
  if (blockIdx.x == 0 && (int)threadIdx.x < tail) {
    const int64_t e = n8 * 8 + threadIdx.x;
    const __bf16 ze = reinterpret_cast<const __bf16*>(z)[e];
    const __bf16 ve = reinterpret_cast<const __bf16*>(v)[e];
    const float r = __builtin_fmaf(neg_sigma, (float)ve, (float)ze);
    if (OUT_BF16)
      static_cast<__bf16*>(out)[e] = (__bf16)r;
    else
      static_cast<float*>(out)[e] = r;
  }
}

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// fp32 output, 4 elements per lane: n4 groups of 4, then `tail` (< 4) elements
__global__ __launch_bounds__(kThreads) void one_step4_kernel(const u32x2* __restrict__ z, const u32x2* __restrict__ v,
                                                             f32x4* __restrict__ out, int64_t n4, int tail,
                                                             float neg_sigma) {
  constexpr int kU = 2 * kUnroll;
  const int64_t step = (int64_t)gridDim.x * kThreads * kU;
  for (int64_t base = (int64_t)blockIdx.x * kThreads * kU + threadIdx.x; base < n4; base += step) {
    u32x2 zr[kU], vr[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int64_t i = base + (int64_t)u * kThreads;
      if (i < n4) {
        zr[u] = __builtin_nontemporal_load(z + i);
        vr[u] = __builtin_nontemporal_load(v + i);
      }
    }
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int64_t i = base + (int64_t)u * kThreads;
      if (i < n4) {
        const uint32_t zw[2] = {zr[u].x, zr[u].y}, vw[2] = {vr[u].x, vr[u].y};
        float r[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float ze = __builtin_bit_cast(float, (zw[e >> 1] >> (16 * (e & 1))) << 16);
          const float ve = __builtin_bit_cast(float, (vw[e >> 1] >> (16 * (e & 1))) << 16);
          r[e] = __builtin_fmaf(neg_sigma, ve, ze);
        }
        st(f32x4{r[0], r[1], r[2], r[3]}, out + i);
      }
    }
  }
  if (blockIdx.x == 0 && (int)threadIdx.x < tail) {
    const int64_t e = n4 * 4 + threadIdx.x;
    const __bf16 ze = reinterpret_cast<const __bf16*>(z)[e];
    const __bf16 ve = reinterpret_cast<const __bf16*>(v)[e];
    reinterpret_cast<float*>(out)[e] = __builtin_fmaf(neg_sigma, (float)ve, (float)ze);
  }
}

}  // namespace

hipError_t launch_one_step(const void* z_lq, const void* v, void* z_hat, int64_t n, float sigma, bool out_bf16,
                           hipStream_t stream) {
  const int64_t n8 = n / 8;
  const int tail = (int)(n - n8 * 8);
  int64_t blocks = (n8 + (int64_t)kThreads * kUnroll - 1) / ((int64_t)kThreads * kUnroll);
  if (blocks > 8192) blocks = 8192;
  if (blocks < 1) blocks = 1;
  const u32x4* zp = static_cast<const u32x4*>(z_lq);
  const u32x4* vp = static_cast<const u32x4*>(v);
  if (FASTVR_OS_LANE4 && !out_bf16) {
    const int64_t n4 = n / 4;
    int64_t b4 = (n4 + (int64_t)kThreads * 2 * kUnroll - 1) / ((int64_t)kThreads * 2 * kUnroll);
    b4 = b4 > 8192 ? 8192 : (b4 < 1 ? 1 : b4);
    hipLaunchKernelGGL(one_step4_kernel, dim3((unsigned)b4), dim3(kThreads), 0, stream,
                       static_cast<const u32x2*>(z_lq), static_cast<const u32x2*>(v), static_cast<f32x4*>(z_hat), n4,
                       (int)(n - n4 * 4), -sigma);
    return hipGetLastError();
  }
  if (out_bf16)
    hipLaunchKernelGGL(one_step_kernel<true>, dim3((unsigned)blocks), dim3(kThreads), 0, stream, zp, vp, z_hat, n8,
                       tail, -sigma);
  else
    hipLaunchKernelGGL(one_step_kernel<false>, dim3((unsigned)blocks), dim3(kThreads), 0, stream, zp, vp, z_hat, n8,
                       tail, -sigma);
  return hipGetLastError();
}

}  // namespace fastvr
