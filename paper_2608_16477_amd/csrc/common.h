// Shared device helpers for the gfx950 kernels: bf16 bit conversions, vector
// types, wave64 reductions, and the launch-error check used by the host side.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "pallas.h"

namespace pallas {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

// bf16 stored as its 16-bit pattern.
__device__ __forceinline__ float bf2f(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}
// Low / high bf16 of a packed pair.
__device__ __forceinline__ float bflo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bfhi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// float -> bf16 with the hardware conversion (v_cvt_pk_bf16_f32: round to
// nearest, ties to even; NaN stays NaN).
__device__ __forceinline__ uint32_t pack_bf2(float lo, float hi) {
  const f32x2 v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}
__device__ __forceinline__ uint16_t f2bf(float f) {
  return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
}

// SwiGLU of one output: silu(gate) * up, silu(g) = g / (1 + e^-g), the
// division taken as a multiply by the hardware reciprocal (v_rcp_f32,
// within 1 ulp): the IEEE division sequence costs a dozen instructions per
// output in the GEMM epilogues, and the result is rounded to bf16.
__device__ __forceinline__ float swiglu(float gate, float up) {
  return gate * __builtin_amdgcn_rcpf(1.0f + __expf(-gate)) * up;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}

}  // namespace pallas
