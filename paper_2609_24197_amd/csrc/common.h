// Device-side building blocks shared by the gfx950 kernels of the drafting step:
// bf16 helpers, MFMA fragment types and wrappers, wave-level reductions.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace hspec {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));

constexpr int WAVE = 64;

// Device status word bits (first int32 of every workspace).
enum : int {
  ST_BAD_PAGE = 1,      // a page id outside [0, num_pages)
  ST_BAD_CTX_LEN = 2,   // ctx_len < 0 or beyond the table / max_ctx_len
};

__device__ __forceinline__ float bf2f(bf16 v) { return (float)v; }
__device__ __forceinline__ bf16 f2bf(float v) { return (bf16)v; }   // v_cvt_pk_bf16_f32, RNE

// Widening of storage element types to fp32 for VALU code.
__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(bf16 v) { return (float)v; }

// 16-byte fragment of 8 bf16 values.
__device__ __forceinline__ bf16x8 ld8(const bf16* p) {
  return *reinterpret_cast<const bf16x8*>(p);
}
__device__ __forceinline__ bf16x8 zero8() {
  u32x4 z = {0u, 0u, 0u, 0u};
  return __builtin_bit_cast(bf16x8, z);
}

// D += A(16x32) * B(32x16); lane l holds A[l%16][8(l/16)..+7], B[8(l/16)..+7][l%16],
// D[4(l/16)+i][l%16].
__device__ __forceinline__ f32x4 mma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
// The same 16x16x32 product on fp16 operands (11 significant bits).
__device__ __forceinline__ f32x4 mma16h(f16x8 a, f16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}
// D += A(32x16) * B(16x32); lane l holds A[l%32][8(l/32)..+7], B[8(l/32)..+7][l%32],
// D[8(i/4)+4(l/32)+i%4][l%32].
__device__ __forceinline__ f32x16 mma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Reductions over the four lanes l, l^16, l^32, l^48 (one column of a 16-wide MFMA tile),
// with the gfx950 lane-swap instructions: every lane ends with the same, identically ordered
// result.
__device__ __forceinline__ float wave_max16x4(float v) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
  auto q = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(q[0]), __uint_as_float(q[1]));
}
__device__ __forceinline__ float wave_sum16x4(float v) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  auto q = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(q[0]) + __uint_as_float(q[1]);
}
__device__ __forceinline__ float wave_sum(float v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// Wait until at most VM vector-memory operations (loads, LDS DMA) of this wave are pending.
template <int VM>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(VM >= 0 && VM < 64, "vmcnt range");
  // gfx9 s_waitcnt immediate: vmcnt[3:0] and [15:14], expcnt[6:4] = 7, lgkmcnt[11:8] = 15 (no wait)
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt((VM & 15) | (7 << 4) | (15 << 8) | ((VM >> 4) << 14));
  asm volatile("" ::: "memory");
}

template <int VM>
__device__ __forceinline__ void wait_vm_lgkm0() {
  // vmcnt <= VM and every LDS access of this wave complete
  static_assert(VM >= 0 && VM < 64, "vmcnt range");
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt((VM & 15) | (7 << 4) | (0 << 8) | ((VM >> 4) << 14));
  asm volatile("" ::: "memory");
}

// Workgroup barrier without the memory fence of __syncthreads (which would also wait for
// every outstanding global load); callers order LDS traffic with explicit waits.
__device__ __forceinline__ void wg_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

template <int V>
using Int = std::integral_constant<int, V>;

__device__ __forceinline__ void set_status(int* st, int bit) {
  if (st) atomicOr(st, bit);
}

}  // namespace hspec
