// Device helpers shared by the attention kernels (gfx950).
#pragma once

#include "../launch.h"

namespace uf {
namespace attn {

constexpr int kD = 128;
constexpr float kLazyLog2 = 8.0f;   // raise the running max only when it grows by more than 2^8

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(4))) int32_t const_i32;   // uniform -> scalar loads

__device__ inline bf16x8 as_bf16x8(uint4 u) { return __builtin_bit_cast(bf16x8, u); }

// Both lanes of a pair (l, l^32) get the same value.
__device__ inline float pair_max(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ inline float pair_sum(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ inline uint32_t pack_bf16x2(float lo, float hi) {
  bf16x2 v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

// One 16-byte-per-lane copy global -> LDS: lane l reads base + off and writes
// LDS byte lds + 16*l.  Issued as inline assembly so that the compiler's
// wait-count insertion does not treat every later LDS read as dependent on it;
// the kernels order the copies with explicit s_waitcnt vmcnt and barriers.
// The uniform base is a scalar pair and the LDS target goes through m0.
__device__ inline void dma16(const void* base, uint32_t off, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" : : "v"(off), "s"(base), "s"(lds) : "memory");
}

// s_waitcnt immediates (gfx9 encoding): vmcnt in [3:0] and [15:14], expcnt
// in [6:4], lgkmcnt in [11:8].
constexpr int waitcnt_vm(int n) { return (n & 15) | (7 << 4) | (15 << 8) | ((n >> 4) << 14); }
constexpr int kWaitLgkm0 = 15 | (7 << 4) | (0 << 8) | (3 << 14);

__device__ inline uint32_t lds_addr(const void* p) {
  return __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(lds_void*)p);
}

}  // namespace attn
}  // namespace uf
