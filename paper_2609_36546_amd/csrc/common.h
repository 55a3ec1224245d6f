// Shared device helpers for the gfx950 kernels of libipdv.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ipdv {

typedef __bf16 bf16;
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float floatx4;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float floatx16;

constexpr int kWave = 64;

__device__ __forceinline__ int lane_id() { return __lane_id(); }

// 16-byte global load / store.
template <typename V>
__device__ __forceinline__ V ld16(const void* p) {
  return *reinterpret_cast<const V*>(p);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

__device__ __forceinline__ float wave_max_xor(float v, int mask) {
  return fmaxf(v, __shfl_xor(v, mask, kWave));
}

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16 x) { return static_cast<float>(x); }

template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float x) { return static_cast<bf16>(x); }

// One 16-byte direct-to-LDS load: lane i's bytes land at lds + 16 i (M0 holds
// the wave-uniform LDS address).  Written as inline assembly so the compiler
// does not add its own whole-queue waits before every LDS read: the ring's
// explicit vmcnt wait + barrier order the accesses.  Compiler-generated waits
// for its own loads stay correct, as vmcnt retires loads in issue order.
__device__ __forceinline__ void dma16(const void* src, char* lds) {
  const unsigned lds_addr = (unsigned)(uintptr_t)(__attribute__((address_space(3))) void*)lds;
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off"
               :
               : "s"(__builtin_amdgcn_readfirstlane(lds_addr)), "v"(src)
               : "memory", "m0");
}

}  // namespace ipdv
