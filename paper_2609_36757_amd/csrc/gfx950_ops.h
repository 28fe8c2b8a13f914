// Device helpers shared by the attention kernels for CDNA4 (gfx950): vector
// types, the bf16 MFMA, buffer descriptors, the LDS-DMA issue, workgroup
// barriers and counted vmcnt waits.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fastvr {
namespace dev {

constexpr float kLn2 = 0.693147180559945309f;
constexpr int kBufFlags = 0x00020000;  // raw buffer, 32-bit data format (gfx9 family)

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef short i16x8 __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

static __device__ __forceinline__ f32x16 mfma32(u32x4 a, u32x4 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

static __device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int64_t bytes) {
  const int n = bytes > 0x7fffffff ? 0x7fffffff : (int)bytes;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, n, kBufFlags);
}

// this lane's value and the value of the same lane in the other 32-lane half
static __device__ __forceinline__ float swap_halves(float x, float* other) {
  const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(uint32_t, x), __builtin_bit_cast(uint32_t, x),
                                                  false, false);
  *other = __builtin_bit_cast(float, (uint32_t)r[1]);
  return __builtin_bit_cast(float, (uint32_t)r[0]);
}

typedef int i32x4 __attribute__((ext_vector_type(4)));

// Buffer resource (V#) of `bytes` bytes at `base`: stride 0, raw addressing,
// 32-bit data format.  Reads at offsets >= bytes return zero.
static __device__ __forceinline__ i32x4 make_vsharp(const void* base, int64_t bytes) {
  const uint64_t a = (uint64_t)base;
  const int n = bytes > 0x7fffffff ? 0x7fffffff : (int)bytes;
  return i32x4{(int)(uint32_t)a, (int)((a >> 32) & 0xffff), n, kBufFlags};
}

// One 16-byte-per-lane DMA from a buffer straight into LDS at lds_addr + 16 * lane
// (buffer_load_dwordx4 ... lds).  Issued as inline assembly on purpose: the
// compiler then does not pair every later LDS read with a wait for all
// outstanding DMA; completion is ordered explicitly with counted vmcnt waits
// followed by a workgroup barrier.  M0 carries the LDS address and is not used
// by any other instruction of this kernel.
static __device__ __forceinline__ void dma16(uint32_t lds_addr, uint32_t voff, i32x4 rsrc, int soff) {
  // every scalar operand is wave-uniform; readfirstlane pins it to SGPRs
  rsrc.x = __builtin_amdgcn_readfirstlane(rsrc.x);
  rsrc.y = __builtin_amdgcn_readfirstlane(rsrc.y);
  rsrc.z = __builtin_amdgcn_readfirstlane(rsrc.z);
  rsrc.w = __builtin_amdgcn_readfirstlane(rsrc.w);
  soff = __builtin_amdgcn_readfirstlane(soff);
  lds_addr = __builtin_amdgcn_readfirstlane(lds_addr);
  // s_nop 4: the scalar operands may have just been written by v_readfirstlane
  // (a vector-ALU write of an SGPR needs 5 wait states before a buffer
  // instruction reads it); s_nop 0: one wait state between the M0 write and
  // the LDS-DMA that reads M0.  Hazards inside inline assembly are not
  // covered by the compiler.
  asm volatile("s_nop 4\n\ts_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
               :
               : "s"(lds_addr), "v"(voff), "s"(rsrc), "s"(soff)
               : "memory", "m0");
}

// The same with 4 bytes per lane (buffer_load_dword ... lds): lane data lands
// at lds_addr + 4 * lane; only a 4-byte aligned source is needed.
static __device__ __forceinline__ void dma4(uint32_t lds_addr, uint32_t voff, i32x4 rsrc, int soff) {
  rsrc.x = __builtin_amdgcn_readfirstlane(rsrc.x);
  rsrc.y = __builtin_amdgcn_readfirstlane(rsrc.y);
  rsrc.z = __builtin_amdgcn_readfirstlane(rsrc.z);
  rsrc.w = __builtin_amdgcn_readfirstlane(rsrc.w);
  soff = __builtin_amdgcn_readfirstlane(soff);
  lds_addr = __builtin_amdgcn_readfirstlane(lds_addr);
  asm volatile("s_nop 4\n\ts_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dword %1, %2, %3 offen lds"
               :
               : "s"(lds_addr), "v"(voff), "s"(rsrc), "s"(soff)
               : "memory", "m0");
}

static __device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// Workgroup barrier with LDS visibility; vector-memory (DMA) completion is
// handled separately with counted waits so that prefetches stay in flight.
static __device__ __forceinline__ void barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

// s_waitcnt vmcnt(N): every DMA issued by this wave except the newest N
// instructions has landed (inline assembly, so the compiler cannot relax it)
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt is a 6-bit counter");
  asm volatile("s_waitcnt vmcnt(%0)" ::"i"(N) : "memory");
}

// instruction-group ordering hints for the scheduler (sched_group_barrier masks)
#define SCHED_MFMA 0x008
#define SCHED_DS_READ 0x100
#define SCHED_VALU 0x002

}  // namespace dev
}  // namespace fastvr
