// Element types of the kernels: raw storage bits and fp32 conversions.
#pragma once

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include <cstdint>

#include "sparoa.h"

namespace sparoa {

template <int DT>
struct Elem;

template <>
struct Elem<SPAROA_F32> {
  using raw = uint32_t;
  static constexpr int size = 4;
  static constexpr raw mag_mask = 0x7FFFFFFFu;   // all bits but the sign
  __device__ static float to_f32(raw v) { return __uint_as_float(v); }
  __device__ static raw from_f32(float v) { return __float_as_uint(v); }
};

template <>
struct Elem<SPAROA_F16> {
  using raw = uint16_t;
  static constexpr int size = 2;
  static constexpr raw mag_mask = 0x7FFFu;
  __device__ static float to_f32(raw v) { return __half2float(__ushort_as_half(v)); }
  __device__ static raw from_f32(float v) { return __half_as_ushort(__float2half_rn(v)); }
};

template <>
struct Elem<SPAROA_BF16> {
  using raw = uint16_t;
  static constexpr int size = 2;
  static constexpr raw mag_mask = 0x7FFFu;
  // bfloat16 is the upper half of a binary32.
  __device__ static float to_f32(raw v) { return __uint_as_float((uint32_t)v << 16); }
  // Round to nearest, ties to even (gfx950 converts in hardware: v_cvt_pk_bf16_f32).
  __device__ static raw from_f32(float f) { return __builtin_bit_cast(raw, (__bf16)f); }
};

// relu: v > 0 ? v : 0; relu6: v > 0 ? min(v, 6) : 0; none: v.  Written as
// selects: `act` is uniform, but early returns per element compile to scalar
// branches around every element of an unrolled epilogue.
__device__ __forceinline__ float apply_act(float v, int act) {
  const float t = v > 0.f ? v : 0.f;
  const float hi = act == SPAROA_ACT_RELU6 ? 6.f : __builtin_inff();
  const float u = t < hi ? t : hi;
  return act == SPAROA_ACT_NONE ? v : u;
}

}  // namespace sparoa
