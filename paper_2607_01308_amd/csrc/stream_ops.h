// Device helpers shared by the render kernels: 16-byte nontemporal global
// stores and the single-step fp64 -> bf16 rounding.
#pragma once

#include "internal.h"

namespace cm {

__device__ __forceinline__ void st_stream(uint8_t* p, u32x4 v) {
  __builtin_nontemporal_store(v, (CM_GLOBAL u32x4*)p);
}

// Round fp64 to the nearest bf16, ties to even, as one rounding step. Rounding
// to fp32 first can only go wrong when the fp32 value lands exactly on a bf16
// midpoint (every bf16 value and midpoint is an fp32 value, so otherwise y and
// its fp32 rounding lie on the same side of every midpoint); in that case the
// fp32 value is nudged one ulp towards y before the hardware bf16 conversion.
__device__ __forceinline__ uint32_t bf16_bits_rne(double y) {
  const float f = (float)y;
  uint32_t u = __float_as_uint(f);
  if (__builtin_expect((u & 0xFFFFu) == 0x8000u, 0)) {
    const double back = (double)f;
    if (y != back) u = (fabs(y) > fabs(back)) ? u + 1u : u - 1u;
  }
  return (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)__uint_as_float(u));
}

// Element e of a little-endian word array as fp64 (exact).
template <int ESIZE>
__device__ __forceinline__ double elem_f64(const uint32_t* w, int e) {
  if constexpr (ESIZE == 2) {
    const uint32_t x = w[e >> 1];
    return (double)__uint_as_float((e & 1) ? (x & 0xFFFF0000u) : (x << 16));
  } else {
    return (double)__uint_as_float(w[e]);
  }
}

// Storage bits of y rounded to the element type (low 16 bits for bf16).
template <int ESIZE>
__device__ __forceinline__ uint32_t round_bits(double y) {
  if constexpr (ESIZE == 2) return bf16_bits_rne(y);
  else return __float_as_uint((float)y);
}

}  // namespace cm
