// Element access helpers of the HBM-bound kernels: 16-element loads of any
// storage format as raw codes or fp32 bits, the 16-value encoder (hardware
// conversions where exact, the integer cast otherwise) and the matching
// stores.
#pragma once
#include "codec.h"

namespace scalify {

typedef unsigned int u4 __attribute__((ext_vector_type(4)));

// Load 16 consecutive elements of format F as raw codes / fp32 bits.
template <int F>
__device__ __forceinline__ void load16(const void* base, int64_t e, uint32_t (&c)[16]) {
  if (F == kE4M3 || F == kE5M2) {
    const u4 v = *(const u4*)((const uint8_t*)base + e);
#pragma unroll
    for (int i = 0; i < 16; ++i) c[i] = (v[i >> 2] >> (8 * (i & 3))) & 0xFFu;
  } else if (F == kF16) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const u4 v = *(const u4*)((const uint16_t*)base + e + 8 * h);
#pragma unroll
      for (int i = 0; i < 8; ++i) c[8 * h + i] = (v[i >> 1] >> (16 * (i & 1))) & 0xFFFFu;
    }
  } else {
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      const u4 v = *(const u4*)((const uint32_t*)base + e + 4 * h);
#pragma unroll
      for (int i = 0; i < 4; ++i) c[4 * h + i] = v[i];
    }
  }
}

template <int F>
__device__ __forceinline__ uint32_t load1(const void* base, int64_t e) {
  if (F == kE4M3 || F == kE5M2) return ((const uint8_t*)base)[e];
  if (F == kF16) return ((const uint16_t*)base)[e];
  return ((const uint32_t*)base)[e];
}

template <int F>
__device__ __forceinline__ uint32_t to_bits(uint32_t c) {
  if constexpr (F == kF32) return c;
  else return decode_bits<F>(c);
}

template <int F>
__device__ __forceinline__ void store16(void* base, int64_t e, const uint32_t (&c)[16]) {
  if (F == kF16) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      u4 v;
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] = c[8 * h + 2 * i] | (c[8 * h + 2 * i + 1] << 16);
      *(u4*)((uint16_t*)base + e + 8 * h) = v;
    }
  } else {
    u4 v;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      v[i] = c[4 * i] | (c[4 * i + 1] << 8) | (c[4 * i + 2] << 16) | (c[4 * i + 3] << 24);
    *(u4*)((uint8_t*)base + e) = v;
  }
}

template <int F>
__device__ __forceinline__ void store1(void* base, int64_t e, uint32_t c) {
  if (F == kF16) ((uint16_t*)base)[e] = (uint16_t)c;
  else ((uint8_t*)base)[e] = (uint8_t)c;
}

// fp32 value of a code of format F (raw code, or fp32 bits for F32) by the
// hardware conversions: exact, since every FP8 and FP16 value is an fp32
// (OCP FP8 with a unit scale).
template <int F>
__device__ __forceinline__ float decode_hw(uint32_t c) {
  if constexpr (F == kF32) return __uint_as_float(c);
  else if constexpr (F == kF16) return (float)__builtin_bit_cast(_Float16, (uint16_t)c);
  else if constexpr (F == kE4M3) return __builtin_amdgcn_cvt_scalef32_f32_fp8(c, 1.0f, 0);
  else return __builtin_amdgcn_cvt_scalef32_f32_bf8(c, 1.0f, 0);
}

// Exact integer casts of 4 values, out of line: they run only for chunks
// that hold a NaN or for shifts outside the hardware conversions' window.
template <int OUTF>
[[maybe_unused]] static __device__ __attribute__((noinline)) uint32_t cast4_exact_fp8(uint32_t u0, uint32_t u1,
                                                                     uint32_t u2, uint32_t u3,
                                                                     int shift, bool sat) {
  return cast_bits<OUTF>(u0, shift, sat) | (cast_bits<OUTF>(u1, shift, sat) << 8) |
         (cast_bits<OUTF>(u2, shift, sat) << 16) | (cast_bits<OUTF>(u3, shift, sat) << 24);
}

[[maybe_unused]] static __device__ __attribute__((noinline)) uint32_t cast2_exact_f16(uint32_t u0, uint32_t u1,
                                                                     int shift, bool sat) {
  return cast_bits<kF16>(u0, shift, sat) | (cast_bits<kF16>(u1, shift, sat) << 16);
}

// Two values to FP16 with the hardware conversion: |x| * 2^-shift (inv) is
// exact in fp32 inside the fast window unless it overflows (then Inf, which
// saturation turns into max) or falls below 2^-126 (then below half the
// smallest FP16 subnormal: zero either way); v_cvt_f16_f32 rounds to
// nearest even. The sign is put back from the input bits.
__device__ __forceinline__ uint32_t cast2_f16_hw(uint32_t u0, uint32_t u1, float inv, bool sat) {
  const uint32_t u[2] = {u0, u1};
  uint32_t h[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const _Float16 f = (_Float16)(__uint_as_float(u[i] & 0x7FFFFFFFu) * inv);
    uint32_t b = (uint32_t)__builtin_bit_cast(uint16_t, f);
    if (sat && b == 0x7C00u) b = 0x7BFFu;
    h[i] = b | ((u[i] >> 16) & 0x8000u);
  }
  return h[0] | (h[1] << 16);
}

// 16 fp32 values (bits) times 2^-shift -> 16 codes packed in 4 words (FP8)
// or 8 words (FP16: two codes per word). The hardware conversions when
// `fast` (the shift is in the window where they are exact, fp32 subnormal
// inputs included) and no value is NaN, else the exact integer cast.
template <int OUTF>
__device__ __forceinline__ void encode16(const uint32_t (&u)[16], int shift, float scale, bool fast,
                                         bool sat, uint32_t (&w)[8]) {
  bool nan = false;
#pragma unroll
  for (int i = 0; i < 16; ++i) nan |= is_nan_bits(u[i]);
  const bool hw = fast && !nan;
  if (OUTF == kE4M3 || OUTF == kE5M2) {
    if (hw) {
#pragma unroll
      for (int q = 0; q < 4; ++q)
        w[q] = cast4_fp8_hw<OUTF>(u[4 * q], u[4 * q + 1], u[4 * q + 2], u[4 * q + 3], scale, sat);
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q)
        w[q] = cast4_exact_fp8<OUTF>(u[4 * q], u[4 * q + 1], u[4 * q + 2], u[4 * q + 3], shift, sat);
    }
#pragma unroll
    for (int q = 4; q < 8; ++q) w[q] = 0u;
  } else {
    if (hw) {
      const float inv = pow2_float(-shift);
#pragma unroll
      for (int q = 0; q < 8; ++q) w[q] = cast2_f16_hw(u[2 * q], u[2 * q + 1], inv, sat);
    } else {
#pragma unroll
      for (int q = 0; q < 8; ++q) w[q] = cast2_exact_f16(u[2 * q], u[2 * q + 1], shift, sat);
    }
  }
}

template <int OUTF>
__device__ __forceinline__ void store_words16(void* base, int64_t e, const uint32_t (&w)[8]) {
  if (OUTF == kF16) {
    *(u4*)((uint16_t*)base + e) = u4{w[0], w[1], w[2], w[3]};
    *(u4*)((uint16_t*)base + e + 8) = u4{w[4], w[5], w[6], w[7]};
  } else {
    *(u4*)((uint8_t*)base + e) = u4{w[0], w[1], w[2], w[3]};
  }
}

// Element i of the packed words.
template <int OUTF>
__device__ __forceinline__ uint32_t word_code(const uint32_t (&w)[8], int i) {
  if (OUTF == kF16) return (w[i >> 1] >> (16 * (i & 1))) & 0xFFFFu;
  return (w[i >> 2] >> (8 * (i & 3))) & 0xFFu;
}

}  // namespace scalify
