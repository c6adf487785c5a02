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

// Butterfly reductions over lane distances 32, 16, 8, 4, 2, 1 (in that
// order), done with register lane exchanges instead of LDS permutes.  Each
// step adds (or takes the max of) the values of lanes i and i ^ m, in one
// operand order or the other, which is exact either way, so the results
// are those of the __shfl_xor butterfly bit for bit:
//   32, 16: v_permlane32_swap / v_permlane16_swap of a value with itself
//           return the pair (v[i], v[i ^ m]) in some order;
//   8:      DPP row_ror:8 reads lane (i + 8) mod 16 = i ^ 8 of the row;
//   4:      DPP row_ror:4 reads lane i ^ 4 or i ^ 4 ^ 8, equal after the
//           8-step;
//   2, 1:   DPP quad permutes [2, 3, 0, 1] and [1, 0, 3, 2].
// Every lane of the group being reduced (the quad, the 16-lane row, the
// wave) must be active: a DPP read from an inactive lane does not return
// that lane's value.
template <int CTRL>
__device__ __forceinline__ float dpp_read(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}
constexpr int kDppXor1 = 0xB1;    // quad_perm [1, 0, 3, 2]
constexpr int kDppXor2 = 0x4E;    // quad_perm [2, 3, 0, 1]
constexpr int kDppRor4 = 0x124;   // row_ror:4
constexpr int kDppRor8 = 0x128;   // row_ror:8

// Sum of the 4 lanes of a quad (distances 1, 2).
__device__ __forceinline__ float quad_sum(float v) {
  v += dpp_read<kDppXor1>(v);
  v += dpp_read<kDppXor2>(v);
  return v;
}
// Sum of a 16-lane row (distances 8, 4, 2, 1).
__device__ __forceinline__ float row16_sum(float v) {
  v += dpp_read<kDppRor8>(v);
  v += dpp_read<kDppRor4>(v);
  v += dpp_read<kDppXor2>(v);
  v += dpp_read<kDppXor1>(v);
  return v;
}
__device__ __forceinline__ float row16_max(float v) {
  v = fmaxf(v, dpp_read<kDppRor8>(v));
  v = fmaxf(v, dpp_read<kDppRor4>(v));
  v = fmaxf(v, dpp_read<kDppXor2>(v));
  v = fmaxf(v, dpp_read<kDppXor1>(v));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  return row16_sum(v);
}
__device__ __forceinline__ float wave_max(float v) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
  r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
  return row16_max(v);
}

}  // namespace pallas
