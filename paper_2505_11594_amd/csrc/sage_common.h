// Device-side helpers shared by the gfx950 kernels of the microscaled-FP4
// attention forward (SageAttention3, arXiv 2505.11594).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef int v8i __attribute__((ext_vector_type(8)));
typedef int v4i __attribute__((ext_vector_type(4)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef short v8s __attribute__((ext_vector_type(8)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));

namespace sage {

// Compile-time loop: f(std::integral_constant<int, I>{}) for I in [0, N), so
// that loop indices can feed instruction immediates (MFMA op_sel fields).
template <int I> struct ic { static constexpr int value = I; };
template <int N, int I = 0, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(ic<I>{});
    static_for<N, I + 1>(f);
  }
}

// Status codes mirrored from the public header (kept in one place for kernels).
enum { kFmtMX = 0, kFmtNV16 = 1 };

// ---- 16-bit input widening (exact) ----------------------------------------
__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }
__device__ __forceinline__ float fp16_to_f32(uint16_t h) {
  _Float16 v;
  __builtin_memcpy(&v, &h, 2);
  return (float)v;
}
template <bool BF16>
__device__ __forceinline__ float widen(uint16_t x) { return BF16 ? bf16_to_f32(x) : fp16_to_f32(x); }

// Round fp32 to bf16 / fp16 (nearest even) for 16-bit outputs.
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
__device__ __forceinline__ uint16_t f32_to_fp16_rne(float f) {
  _Float16 h = (_Float16)f;  // IEEE conversion, round to nearest even
  uint16_t r;
  __builtin_memcpy(&r, &h, 2);
  return r;
}

// ---- E8M0 block exponent (MXFP4) --------------------------------------------
// Smallest e with 6 * 2^e >= amax (amax >= 0, finite), clamped to [-127, 127];
// amax == 0 gives -127.  With amax = 1.f * 2^(be-127): e = be - 129 if the
// mantissa is <= 1.5, else be - 128.  Subnormal amax always clamps to -127.
__device__ __forceinline__ int e8m0_exponent(float amax) {
  uint32_t u = __float_as_uint(amax);
  int be = (int)(u >> 23);
  if (be == 0) return -127;
  int e = be - 129 + ((u & 0x7FFFFFu) > 0x400000u ? 1 : 0);
  return e < -127 ? -127 : (e > 127 ? 127 : e);
}

// ---- E4M3 (FN) scale codec -------------------------------------------------
// Round to nearest even, saturating at 448 (0x7E); s >= 0.
__device__ __forceinline__ uint32_t e4m3_encode(float s) {
  if (!(s > 0.0f)) return 0u;
  if (s >= 448.0f) return 0x7Eu;
  if (s < 0.015625f) {                              // subnormal range: step 2^-9
    float q = __builtin_rintf(s * 512.0f);          // exact scaling, RNE
    return (uint32_t)q;                             // q == 8 is the smallest normal, code 0x08
  }
  uint32_t u = __float_as_uint(s);
  int E = (int)(u >> 23) - 127;                     // -6 .. 8
  uint32_t man = u & 0x7FFFFFu;
  uint32_t m3 = (man + 0x7FFFFu + ((man >> 20) & 1u)) >> 20;  // RNE to 3 bits (may carry to 8)
  uint32_t code = ((uint32_t)(E + 7) << 3) + m3;    // carry moves into the exponent field
  return code > 0x7Eu ? 0x7Eu : code;
}
__device__ __forceinline__ float e4m3_decode(uint32_t b) {
  uint32_t e = (b >> 3) & 15u, m = b & 7u;
  if (e == 0) return __builtin_ldexpf((float)m, -9);
  return __builtin_ldexpf((float)(8u + m), (int)e - 10);
}
// The same codec in one instruction each: gfx950's v_cvt_pk_fp8_f32 (OCP
// E4M3, nearest even) equals e4m3_encode on [0, 448] -- every rounding
// midpoint and the subnormal range included -- and v_cvt_f32_fp8 equals
// e4m3_decode on every code; values >= 448 are clamped first, as e4m3_encode
// saturates.  Byte `sel` of `word` is decoded.  The encoder converts the pair
// (s, +0) into the low half of a zero word, so bytes 1..3 of its result are 0.
__device__ __forceinline__ uint32_t e4m3_encode_hw(float s) {
  return (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(__builtin_fminf(s, 448.0f), 0.0f, 0, false);
}
template <int SEL>
__device__ __forceinline__ float e4m3_decode_hw(uint32_t word) { return __builtin_amdgcn_cvt_f32_fp8((int)word, SEL); }

// fl32(x / 6) for 2^-90 <= x <= 2^100 with a multiply and two FMAs instead of
// a division: q = x * fl32(1/6), the residual x - 6q is exact, and one FMA step
// rounds correctly -- checked on every significand of one binade, which covers
// every exponent in that range (the step commutes with powers of two).  Below
// 2^-90 the result stays under 2^-10, where the E4M3 code is 0 either way.
__device__ __forceinline__ float div6(float x) {
  const float y = 0x1.555556p-3f;                   // fl32(1/6)
  const float q = x * y;
  return __builtin_fmaf(__builtin_fmaf(-q, 6.0f, x), y, q);
}

// ---- FP4 (E2M1) conversion ----------------------------------------------
// v_cvt_scalef32_pk_fp4_f32 rounds to nearest even, saturates at +-6 and keeps
// the sign of zero; it divides by the power-of-two part of the scale operand.
// Inputs here are already scaled, so the scale is 1.0.  Returns the byte with
// a in the low nibble and b in the high nibble.
__device__ __forceinline__ uint32_t cvt_fp4x2(float a, float b) {
  return __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(__float_as_uint(a), a, b, 1.0f, 0) & 0xFFu;   // byte 0 only
}

__device__ __forceinline__ float fmax3(float a, float b, float c) { return __builtin_fmaxf(a, __builtin_fmaxf(b, c)); }

// Maximum / minimum of two scores or bounds (finite or +-inf, never NaN): the
// IEEE maximum and minimum, which unlike fmaxf / fminf need no NaN-quieting of
// their operands (v_maximum3_f32, v_minimum3_f32).
__device__ __forceinline__ float smax(float a, float b) { return __builtin_elementwise_maximum(a, b); }
__device__ __forceinline__ float smin(float a, float b) { return __builtin_elementwise_minimum(a, b); }

}  // namespace sage
