// Device-side helpers shared by the codec's HIP kernels (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sn {

typedef uint16_t bf16_t;  // bf16 bit pattern in memory

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// ---- scalar element access as float -------------------------------------
__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(bf16_t v) {
  return __uint_as_float(static_cast<uint32_t>(v) << 16);
}

// Round-to-nearest-even conversion; gfx950 has a hardware pack instruction
// (v_cvt_pk_bf16_f32) that the vector convert lowers to.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  f32x2 v = {lo, hi};
  bf16x2 r = __builtin_convertvector(v, bf16x2);
  return __builtin_bit_cast(uint32_t, r);
}

template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16_t from_f32<bf16_t>(float v) {
  return static_cast<bf16_t>(pack_bf16x2(v, 0.0f) & 0xFFFFu);
}

// unpack the two bf16 halves of a dword to float
__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// ---- compensated accumulation ----------------------------------------------
// Dot2 of Ogita, Rump and Oishi ("Accurate sum and dot product", SIAM J. Sci.
// Comput. 26(6), 2005): Knuth's TwoSum and an FMA-based TwoProduct carry the
// rounding error of every step in a second float, so a sum or dot product is
// as accurate as if computed in twice the working precision and then rounded.
// The _rn intrinsics keep the compiler from contracting or reassociating the
// error-free transformations.
struct Dot2 {
  float s = 0.0f, c = 0.0f;
  __device__ __forceinline__ void add(float x) {
    const float t = __fadd_rn(s, x);
    const float z = __fsub_rn(t, s);
    const float err = __fadd_rn(__fsub_rn(s, __fsub_rn(t, z)), __fsub_rn(x, z));
    s = t;
    c = __fadd_rn(c, err);
  }
  __device__ __forceinline__ void add_prod(float a, float b) {
    const float p = __fmul_rn(a, b);
    const float e = fmaf(a, b, -p);
    add(p);
    c = __fadd_rn(c, e);
  }
  __device__ __forceinline__ void merge(float os, float oc) {
    add(os);
    c = __fadd_rn(c, oc);
  }
  __device__ __forceinline__ float value() const { return __fadd_rn(s, c); }
};

// Sum a Dot2 over the 64 lanes of a wave (every lane gets the result).
__device__ __forceinline__ float wave_sum_dot2(Dot2 a) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float os = __shfl_xor(a.s, off, 64);
    const float oc = __shfl_xor(a.c, off, 64);
    a.merge(os, oc);
  }
  return a.value();
}

// ---- wave64 reduction -----------------------------------------------------
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// ---- id handling: clamp out-of-range ids, flag them ----------------------
// bit 0: token id outside [0, vocab); bit 1: position id outside [0, n_pos)
__device__ __forceinline__ int64_t clamp_id(int64_t id, int64_t rows, int32_t *err_flag,
                                            int bit) {
  if (id < 0 || id >= rows) {
    if (err_flag) atomicOr(err_flag, bit);
    id = id < 0 ? 0 : rows - 1;
  }
  return id;
}

}  // namespace sn
