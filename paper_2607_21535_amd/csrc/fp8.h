// FP8 (OCP E4M3) draft KV entries on gfx950: conversion helpers shared by
// the attention kernels, the appends and the conversion exports.
//
// An fp8 cache stores one byte per K or V element; code c stands for
// value(c) * scale with one float32 scale per tensor (Windowed-MTP Section 7,
// KV-cache quantization, read as OCP E4M3 with per-tensor scales).  Every
// E4M3 value is exactly a bf16 value, so the kernels widen codes to bf16
// with the hardware conversion and feed the same bf16 MFMAs as the bf16
// cache; the scales are folded into the softmax scale (keys) and the output
// normalisation (values).  Appends quantise: y = x / scale in float32
// (correctly rounded), clamped to +-448, rounded to nearest even.
#pragma once

#include "common.h"

namespace wmtp {

constexpr float kFp8Max = 448.0f;

// Two E4M3 codes (bytes 0,1 of w, or bytes 2,3 when hi) -> two bf16 in one
// 32-bit word (first code in the low half).  Exact.
template <bool HI>
__device__ __forceinline__ uint32_t fp8x2_to_bf16x2(uint32_t w) {
  return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, HI));
}

// Eight codes (two words) -> eight bf16 (four words), in order.
__device__ __forceinline__ u32x4 fp8x8_to_bf16x8(uint32_t w0, uint32_t w1) {
  return u32x4{fp8x2_to_bf16x2<false>(w0), fp8x2_to_bf16x2<true>(w0), fp8x2_to_bf16x2<false>(w1),
               fp8x2_to_bf16x2<true>(w1)};
}

// One value to store with per-tensor `scale`: x / scale, saturated to the
// finite E4M3 range (the conversion then never overflows).
__device__ __forceinline__ float fp8_prescale(float x, float scale) {
  const float y = __fdiv_rn(x, scale);
  return fminf(fmaxf(y, -kFp8Max), kFp8Max);
}

// Four float values (already prescaled) -> four E4M3 codes in one word,
// first value in the low byte; round to nearest even.
__device__ __forceinline__ uint32_t f32x4_to_fp8x4(float a, float b, float c, float d) {
  int w = __builtin_amdgcn_cvt_pk_fp8_f32(a, b, 0, false);
  w = __builtin_amdgcn_cvt_pk_fp8_f32(c, d, w, true);
  return static_cast<uint32_t>(w);
}

// Eight bf16 (four words) -> eight codes (two words) with per-tensor scale.
__device__ __forceinline__ u32x2 bf16x8_to_fp8x8(u32x4 x, float scale) {
  return u32x2{f32x4_to_fp8x4(fp8_prescale(bf16_lo(x[0]), scale), fp8_prescale(bf16_hi(x[0]), scale),
                              fp8_prescale(bf16_lo(x[1]), scale), fp8_prescale(bf16_hi(x[1]), scale)),
               f32x4_to_fp8x4(fp8_prescale(bf16_lo(x[2]), scale), fp8_prescale(bf16_hi(x[2]), scale),
                              fp8_prescale(bf16_lo(x[3]), scale), fp8_prescale(bf16_hi(x[3]), scale))};
}

}  // namespace wmtp
