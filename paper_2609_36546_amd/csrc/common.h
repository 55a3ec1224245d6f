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

// ---- wave reductions and scans with DPP moves (VALU, no LDS round trip) ----
// DPP controls (GFX9): quad_perm p0 | p1 << 2 | p2 << 4 | p3 << 6, row_shr:n
// 0x110 + n, row_mirror 0x140, row_half_mirror 0x141.  Rows are 16 lanes.
template <int CTRL>
__device__ __forceinline__ float dpp_move(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xf, 0xf, true));
}
// The value of lane i ^ 32 / i ^ 16 (v_permlane32_swap / v_permlane16_swap).
__device__ __forceinline__ float lane_xor32(float v) {
  const unsigned u = __float_as_uint(v);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return __uint_as_float(lane_id() < 32 ? r[1] : r[0]);
}
__device__ __forceinline__ int lane_xor32(int v) {
  const auto r = __builtin_amdgcn_permlane32_swap((unsigned)v, (unsigned)v, false, false);
  return (int)(lane_id() < 32 ? r[1] : r[0]);
}
__device__ __forceinline__ float lane_xor16(float v) {
  const unsigned u = __float_as_uint(v);
  const auto r = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  return __uint_as_float((lane_id() & 16) ? r[0] : r[1]);
}
// Combine over the wave, result in every lane: a butterfly inside each row
// (mirror, half mirror, then the quad swaps 2 and 1 pair disjoint lane sets
// at every step, so each lane's value enters once), then across the rows.
template <class OP>
__device__ __forceinline__ float wave_reduce(float v, OP op) {
  v = op(v, dpp_move<0x140>(v));
  v = op(v, dpp_move<0x141>(v));
  v = op(v, dpp_move<0x4E>(v));   // quad_perm [2, 3, 0, 1]
  v = op(v, dpp_move<0xB1>(v));   // quad_perm [1, 0, 3, 2]
  v = op(v, lane_xor16(v));
  return op(v, lane_xor32(v));
}
__device__ __forceinline__ float wave_sum(float v) {
  return wave_reduce(v, [](float a, float b) { return a + b; });
}
__device__ __forceinline__ float wave_max(float v) {
  return wave_reduce(v, [](float a, float b) { return fmaxf(a, b); });
}
// Inclusive prefix sum of ints over the wave's lanes (lane order).
template <int CTRL>
__device__ __forceinline__ int dpp_move_i(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xf, 0xf, true);
}
__device__ __forceinline__ int wave_incl_scan_i(int v) {
  v += dpp_move_i<0x111>(v);
  v += dpp_move_i<0x112>(v);
  v += dpp_move_i<0x114>(v);
  v += dpp_move_i<0x118>(v);
  const int r0 = __builtin_amdgcn_readlane(v, 15);
  const int r1 = __builtin_amdgcn_readlane(v, 31);
  const int r2 = __builtin_amdgcn_readlane(v, 47);
  const int row = lane_id() >> 4;
  return v + (row > 0 ? r0 : 0) + (row > 1 ? r1 : 0) + (row > 2 ? r2 : 0);
}
// Inclusive prefix sum over the wave's lanes (lane order).
__device__ __forceinline__ float wave_incl_scan(float v) {
  v += dpp_move<0x111>(v);   // row_shr:1 (lanes without a source add 0)
  v += dpp_move<0x112>(v);
  v += dpp_move<0x114>(v);
  v += dpp_move<0x118>(v);
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 15));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 31));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 47));
  const int row = lane_id() >> 4;
  return v + (row > 0 ? r0 : 0.f) + (row > 1 ? r1 : 0.f) + (row > 2 ? r2 : 0.f);
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
