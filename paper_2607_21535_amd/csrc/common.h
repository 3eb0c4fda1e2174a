// Shared device helpers for the gfx950 draft-attention kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace wmtp {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;          // CDNA wavefront width
constexpr int kTileKeys = 16;      // keys per MFMA tile (the 16-row operand)
constexpr int kWaves = 4;          // waves per split workgroup
constexpr int kThreads = kWave * kWaves;
constexpr int kMaxGroup = 16;      // query heads one KV head can serve (MFMA N = 16)
constexpr int kChunkQuantum = kTileKeys * kWaves;  // work-item sizes are multiples of this

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ float neg_inf() { return -__builtin_inff(); }

// Low / high bfloat16 of a 32-bit word, widened to float (exact).
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Two floats -> two bfloat16 in one word (lo in bits 0..15), rounded to
// nearest even by the hardware conversion (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  typedef float f32x2 __attribute__((ext_vector_type(2)));
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

__device__ __forceinline__ int ceil_div_i(int a, int b) { return (a + b - 1) / b; }

__device__ __forceinline__ void raise_error(int32_t* err, int bits) {
  if (err != nullptr) atomicOr(err, bits);
}

}  // namespace wmtp
