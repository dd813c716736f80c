// Device-side number-format helpers: exponent arithmetic on power-of-two
// scales (E8M0 simulated in fp32) and the round-to-nearest-even cast of an
// fp32 value times 2^-shift to OCP FP8 E4M3 / E5M2 or IEEE FP16, done with
// integer operations only.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace scalify {

enum Fmt : int { kE4M3 = 0, kE5M2 = 1, kF16 = 2, kF32 = 3 };

// Format parameters: mantissa bits P, minimum normal exponent, largest finite
// magnitude code, code of an overflowing non-saturated value, sign bit.
template <int F> struct FmtTraits;
template <> struct FmtTraits<kE4M3> {
  static constexpr int P = 3, EMIN = -6;
  static constexpr uint32_t MAXC = 0x7E, OVF = 0x7F, NANC = 0x7F, SIGN = 0x80;
};
template <> struct FmtTraits<kE5M2> {
  static constexpr int P = 2, EMIN = -14;
  static constexpr uint32_t MAXC = 0x7B, OVF = 0x7C, NANC = 0x7F, SIGN = 0x80;
};
template <> struct FmtTraits<kF16> {
  static constexpr int P = 10, EMIN = -14;
  static constexpr uint32_t MAXC = 0x7BFF, OVF = 0x7C00, NANC = 0x7E00, SIGN = 0x8000;
};

// Exponent of a positive finite power of two held in fp32 (normal or
// subnormal encoding). NULL means scale 1.
__device__ __forceinline__ int pow2_exponent(const float* s) {
  if (s == nullptr) return 0;
  uint32_t u = __float_as_uint(*s);
  int e = (int)((u >> 23) & 0xFF);
  if (e != 0) return e - 127;
  uint32_t m = u & 0x7FFFFF;
  return (m == 0) ? -127 : (31 - __clz((int)m)) - 149;
}

// fp32 encoding of 2^e for e in [-127, 127].
__device__ __forceinline__ float pow2_float(int e) {
  uint32_t u = (e >= -126) ? ((uint32_t)(e + 127) << 23) : (0x00400000u >> (-127 - e));
  return __uint_as_float(u);
}

__device__ __forceinline__ int clamp_e8m0(int e) { return e < -127 ? -127 : (e > 127 ? 127 : e); }

// floor(log2 x) of a positive finite fp32 given by its bits.
__device__ __forceinline__ int floor_log2_bits(uint32_t u) {
  int e = (int)((u >> 23) & 0xFF);
  if (e != 0) return e - 127;
  return (31 - __clz((int)(u & 0x7FFFFF))) - 149;
}

// Rescale exponent from an amax given by its (non-negative) fp32 bits.
__device__ __forceinline__ int rescale_exponent(uint32_t amax_bits, int target) {
  if (amax_bits == 0u || amax_bits >= 0x7F800000u) return 0;  // zero, Inf (NaN never stored)
  return floor_log2_bits(amax_bits) - target;
}

// Round the exact value (fp32 bits u) * 2^-shift to format F, ties to even.
// NaN -> NaN (sign kept); +-Inf and overflow -> +-max when sat, else the
// format's overflow code (E4M3 NaN, E5M2/F16 Inf). Target subnormals kept.
template <int F>
__device__ __forceinline__ uint32_t cast_bits(uint32_t u, int shift, bool sat) {
  using T = FmtTraits<F>;
  const uint32_t sign = (u >> 31) ? T::SIGN : 0u;
  const int ef = (int)((u >> 23) & 0xFF);
  uint32_t m = u & 0x7FFFFF;
  if (ef == 0xFF) {
    if (m) return T::NANC | sign;
    return (sat ? T::MAXC : T::OVF) | sign;
  }
  uint32_t sig;
  int ex;  // unbiased exponent of the leading bit of the value
  if (ef != 0) {
    sig = m | 0x800000u;
    ex = ef - 127;
  } else {
    if (m == 0) return sign;  // +-0
    int lz = __clz((int)m) - 8;  // shift bringing the top bit to bit 23
    sig = m << lz;
    ex = -126 - lz;
  }
  ex -= shift;
  // Bits of sig below the target quantum: 23 - P, plus the distance below
  // the smallest normal exponent for target subnormals.
  const int below = (ex < T::EMIN) ? (T::EMIN - ex) : 0;
  const int rs = 23 - T::P + below;
  uint32_t r;
  if (rs > 24) {
    r = 0;  // below half of the smallest subnormal
  } else {
    r = sig >> rs;
    const uint32_t rem = sig & ((1u << rs) - 1u);
    const uint32_t half = 1u << (rs - 1);
    if (rem > half || (rem == half && (r & 1u))) r += 1u;
  }
  // Magnitude code: biased-exponent field times 2^P plus r (carries of r
  // into the exponent field are the correct encoding).
  const int ebase = (ex < T::EMIN) ? 0 : (ex - T::EMIN);
  if (ebase > 64) return (sat ? T::MAXC : T::OVF) | sign;
  const uint32_t mag = ((uint32_t)ebase << T::P) + r;
  if (mag > T::MAXC) return (sat ? T::MAXC : T::OVF) | sign;
  return mag | sign;
}

// ---------------------------------------------------------------------------
// Fast path: the gfx950 conversion v_cvt_scalef32_pk_{fp8,bf8}_f32 computes
// round-to-nearest-even of x / scale into OCP E4M3 / E5M2 with the
// non-saturating overflow rule (E4M3 -> NaN code, E5M2 -> Inf code). With
// scale = 2^shift this is exactly cast_bits(u, shift, sat = false) for every
// non-NaN fp32 input (checked against cast_bits on a structured sweep of
// exponents, mantissa tie and sticky patterns, specials and random inputs,
// shifts -60..60). NaN inputs are not handled here: callers route chunks
// that contain a NaN to cast_bits.

typedef short v2s_t __attribute__((ext_vector_type(2)));

// Largest |shift| for which 2^shift is a normal fp32.
constexpr int kFastShiftMax = 126;

// Smallest shift for the fast paths when inputs may be fp32 subnormals: with
// shift >= kFastShiftMinSub a subnormal x (|x| < 2^-126) scales to less than
// 2^-26, under half the smallest FP16 (and FP8) subnormal, so its code is a
// zero of its sign whether or not the conversion flushes subnormal inputs
// (the sign is kept either way). Below it such inputs need the exact cast.
constexpr int kFastShiftMinSub = -100;

// Saturation fix-up on 4 packed codes: overflow codes -> +-max (same sign).
// E4M3 overflow is 0x7F|s (max 0x7E|s); E5M2 overflow is 0x7C|s (0x7B|s):
// subtract one in exactly the bytes whose low 7 bits equal the overflow code.
template <int F>
__device__ __forceinline__ uint32_t saturate4(uint32_t w) {
  const uint32_t low = w & 0x7F7F7F7Fu;
  uint32_t hit;
  if (F == kE4M3) {
    hit = (low + 0x01010101u) & 0x80808080u;  // 0x7F + 1 carries into bit 7
  } else {
    const uint32_t x = low ^ 0x7C7C7C7Cu;     // zero byte where low == 0x7C
    hit = (x - 0x01010101u) & ~x & 0x80808080u;
  }
  return w - (hit >> 7);
}

// 4 non-NaN fp32 values (bits) times 2^-shift -> 4 packed FP8 codes.
template <int F>
__device__ __forceinline__ uint32_t cast4_fp8_hw(uint32_t u0, uint32_t u1, uint32_t u2, uint32_t u3,
                                                 float scale, bool sat) {
  v2s_t r = {0, 0};
  if (F == kE4M3) {
    r = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(r, __uint_as_float(u0), __uint_as_float(u1), scale, false);
    r = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(r, __uint_as_float(u2), __uint_as_float(u3), scale, true);
  } else {
    r = __builtin_amdgcn_cvt_scalef32_pk_bf8_f32(r, __uint_as_float(u0), __uint_as_float(u1), scale, false);
    r = __builtin_amdgcn_cvt_scalef32_pk_bf8_f32(r, __uint_as_float(u2), __uint_as_float(u3), scale, true);
  }
  const uint32_t w = __builtin_bit_cast(uint32_t, r);
  return sat ? saturate4<F>(w) : w;
}

__device__ __forceinline__ bool is_nan_bits(uint32_t u) { return (u & 0x7FFFFFFFu) > 0x7F800000u; }

// Exact fp32 bits of an FP8 / FP16 code (all FP8 and FP16 values are fp32).
template <int F>
__device__ __forceinline__ uint32_t decode_bits(uint32_t c);

template <> __device__ __forceinline__ uint32_t decode_bits<kE4M3>(uint32_t c) {
  const uint32_t s = (c & 0x80u) << 24;
  const uint32_t e = (c >> 3) & 15u, m = c & 7u;
  if (e == 15u && m == 7u) return s | 0x7FC00000u;
  if (e == 0u) {
    if (m == 0u) return s;
    // m * 2^-9: normalise
    const int top = 31 - __clz((int)m);           // 0..2
    const uint32_t frac = (m << (23 - top)) & 0x7FFFFFu;
    return s | ((uint32_t)(top - 9 + 127) << 23) | frac;
  }
  return s | ((e - 7u + 127u) << 23) | (m << 20);
}

template <> __device__ __forceinline__ uint32_t decode_bits<kE5M2>(uint32_t c) {
  const uint32_t s = (c & 0x80u) << 24;
  const uint32_t e = (c >> 2) & 31u, m = c & 3u;
  if (e == 31u) return s | (m ? 0x7FC00000u : 0x7F800000u);
  if (e == 0u) {
    if (m == 0u) return s;
    const int top = 31 - __clz((int)m);           // 0..1
    const uint32_t frac = (m << (23 - top)) & 0x7FFFFFu;
    return s | ((uint32_t)(top - 16 + 127) << 23) | frac;
  }
  return s | ((e - 15u + 127u) << 23) | (m << 21);
}

template <> __device__ __forceinline__ uint32_t decode_bits<kF16>(uint32_t h) {
  const uint32_t s = (h & 0x8000u) << 16;
  const uint32_t e = (h >> 10) & 31u, m = h & 1023u;
  if (e == 31u) return s | (m ? (0x7FC00000u | (m << 13)) : 0x7F800000u);
  if (e == 0u) {
    if (m == 0u) return s;
    const int top = 31 - __clz((int)m);           // 0..9
    const uint32_t frac = (m << (23 - top)) & 0x7FFFFFu;
    return s | ((uint32_t)(top - 24 + 127) << 23) | frac;
  }
  return s | ((e - 15u + 127u) << 23) | (m << 13);
}

// Magnitude key whose unsigned order is the order of |value| over non-NaN
// codes; NaN codes map to 0 so that they never win a max.
template <int F>
__device__ __forceinline__ uint32_t magnitude_key(uint32_t c);
template <> __device__ __forceinline__ uint32_t magnitude_key<kE4M3>(uint32_t c) {
  const uint32_t a = c & 0x7Fu;
  return a == 0x7Fu ? 0u : a;
}
template <> __device__ __forceinline__ uint32_t magnitude_key<kE5M2>(uint32_t c) {
  const uint32_t a = c & 0x7Fu;
  return a > 0x7Cu ? 0u : a;
}
template <> __device__ __forceinline__ uint32_t magnitude_key<kF16>(uint32_t c) {
  const uint32_t a = c & 0x7FFFu;
  return a > 0x7C00u ? 0u : a;
}
template <> __device__ __forceinline__ uint32_t magnitude_key<kF32>(uint32_t c) {
  const uint32_t a = c & 0x7FFFFFFFu;
  return a > 0x7F800000u ? 0u : a;
}

// Compress an fp32 (bits) to 16 bits that keep sign, exponent, the top 6
// mantissa bits and a sticky bit (OR of the 17 lower mantissa bits) in the
// lowest position. Rounding the expanded value (h << 16) to any format with
// at most 5 mantissa bits, after any power-of-two shift, gives exactly the
// result of rounding the original value: the kept bits hold the result bits
// and the round bit, the sticky bit keeps "anything below". NaN stays NaN.
__device__ __forceinline__ uint32_t sticky16(uint32_t u) {
  return (u >> 16) | ((u & 0x1FFFFu) ? 1u : 0u);
}

}  // namespace scalify
