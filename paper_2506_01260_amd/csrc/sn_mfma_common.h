// Device helpers shared by the matrix-core kernels (gfx950).
//
// MFMA 16x16x32 bf16 operand layout (wave64): lane l = 16 g + n (g = l / 16,
// n = l % 16) supplies 8 consecutive K values of row n of A and of column n of
// B, and receives D[4 g + i][n], i = 0..3.  The K values a lane supplies for A
// and for B are the same 8 indices, so any fixed assignment of (g, e) to
// contraction indices gives the same sum.
#pragma once

#include "sn_device.h"
#include "sn_internal.h"

namespace sn {

__device__ __forceinline__ u32x4 ld16(const bf16_t *p) {
  return *reinterpret_cast<const u32x4 *>(p);
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ f32x4 mfma(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a), as_bf16x8(b), c, 0, 0, 0);
}

// Negate 8 packed bf16 values (flip their sign bits).
__device__ __forceinline__ u32x4 neg8(u32x4 v) {
  const uint32_t s = 0x80008000u;
  return u32x4{v.x ^ s, v.y ^ s, v.z ^ s, v.w ^ s};
}

// Direct-to-LDS load: the 16 bytes at src (per lane) land at dst + 16 * lane,
// where dst is the wave-uniform LDS address of a 1 KiB block.
__device__ __forceinline__ void lds_dma_16(const bf16_t *src, u32x4 *dst) {
  __builtin_amdgcn_global_load_lds(static_cast<const void *>(src),
                                   (__attribute__((address_space(3))) void *)(dst), 16, 0, 0);
}

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding:
// vmcnt[3:0] in bits 3:0, vmcnt[5:4] in bits 15:14, expcnt 6:4, lgkmcnt 11:8).
template <int V>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(V >= 0 && V <= 63, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((V & 0xF) | ((V >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Workgroup barrier for LDS hand-over without a memory fence: the caller's LDS
// operations are complete (lgkmcnt(0)), outstanding global loads are not
// waited for, and the compiler may not move memory operations across it.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0); vmcnt, expcnt unconstrained
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

inline bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

}  // namespace sn
