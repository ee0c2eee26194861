// Device helpers: block-scale rules and the e4m3 cast (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace fmm {
namespace dev {

constexpr float kE4m3Max = 448.0f;
constexpr float kClamp = 1e-12f;  // fl32(1e-12): the block maximum is clamped from below

enum { RULE_FP32_AMAX = 0, RULE_POW2_CEIL = 1, RULE_POW2_OCP = 2 };

// Scale of one block from its absolute maximum.
//   FP32_AMAX : s = fl32(a / 448), returned in `s`; `inv_or_div` = s (divide by it)
//   POW2_*    : s = 2^e; `inv_or_div` = 2^-e (multiplying by it is exactly x / s)
// `stored` receives the stored form: the fp32 bits of s, or the E8M0 byte e + 127.
struct Scale {
  float div;       // FP32_AMAX: the divisor s
  float mul;       // POW2: 2^-e
  uint32_t stored;
};

__device__ __forceinline__ Scale block_scale(float amax, int rule) {
  Scale sc;
  const float a = fmaxf(amax, kClamp);
  if (rule == RULE_FP32_AMAX) {
    const float s = __fdiv_rn(a, kE4m3Max);
    sc.div = s;
    sc.mul = 1.0f;
    sc.stored = __float_as_uint(s);
    return sc;
  }
  // a >= 1e-12 is a normal binary32: a = m 2^E, m in [1, 2).
  const uint32_t bits = __float_as_uint(a);
  const int E = (int)((bits >> 23) & 0xffu) - 127;
  int e = E - 8;
  // POW2_CEIL: least e with a <= 448 2^e = 1.75 2^(e+8): e = E-8 iff m <= 1.75.
  if (rule == RULE_POW2_CEIL && (bits & 0x7fffffu) > 0x600000u) e += 1;
  sc.div = 1.0f;
  sc.mul = __uint_as_float((uint32_t)(127 - e) << 23);  // 2^-e, e in [-48, 121]
  sc.stored = (uint32_t)(e + 127);
  return sc;
}

// Scaled value v = fl32(x / s).
__device__ __forceinline__ float scaled(float x, const Scale &sc, int rule) {
  return rule == RULE_FP32_AMAX ? __fdiv_rn(x, sc.div) : x * sc.mul;
}

// e4m3 codes of four scaled values, packed little-endian into a word.
// v_cvt_pk_fp8_f32 rounds to nearest even and keeps the sign, but turns
// magnitudes above 448 into NaN, so saturate first: rounding then clamping to
// 448 equals clamping then rounding.
__device__ __forceinline__ uint32_t e4m3_pack4(float v0, float v1, float v2, float v3) {
  v0 = __builtin_amdgcn_fmed3f(v0, -kE4m3Max, kE4m3Max);
  v1 = __builtin_amdgcn_fmed3f(v1, -kE4m3Max, kE4m3Max);
  v2 = __builtin_amdgcn_fmed3f(v2, -kE4m3Max, kE4m3Max);
  v3 = __builtin_amdgcn_fmed3f(v3, -kE4m3Max, kE4m3Max);
  int w = __builtin_amdgcn_cvt_pk_fp8_f32(v0, v1, 0, false);
  w = __builtin_amdgcn_cvt_pk_fp8_f32(v2, v3, w, true);
  return (uint32_t)w;
}

// Codes of four values under a power-of-two scale s = 2^e, e in [-48, 120]:
// the e4m3 code of x / s with round to nearest even, saturated to 448.
// v_cvt_scalef32_pk_fp8_f32 divides by the power of two that its scale
// operand holds (exactly, subnormal binary32 inputs included) and rounds to
// nearest even, but, like the plain cast, does not saturate; clamping x to
// +-448 s first is exact because 448 s is.  Where 448 s overflows binary32
// (e = 120, reached only by the ceiling rule) |x| <= 448 s holds already and
// the clamp to +-inf is the identity.
__device__ __forceinline__ uint32_t e4m3_pack4_pow2(float v0, float v1, float v2, float v3, float s) {
  typedef short v2i16 __attribute__((ext_vector_type(2)));
  const float lim = 448.0f * s;
  v0 = __builtin_amdgcn_fmed3f(v0, -lim, lim);
  v1 = __builtin_amdgcn_fmed3f(v1, -lim, lim);
  v2 = __builtin_amdgcn_fmed3f(v2, -lim, lim);
  v3 = __builtin_amdgcn_fmed3f(v3, -lim, lim);
  v2i16 w = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32((v2i16){0, 0}, v0, v1, s, false);
  w = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(w, v2, v3, s, true);
  return __builtin_bit_cast(uint32_t, w);
}

}  // namespace dev
}  // namespace fmm
