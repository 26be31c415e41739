// Internal helpers shared by the libtfdense kernels (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tfd {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;      // CDNA wavefront width
constexpr int kNumXcd = 8;     // MI355X: 8 accelerator complex dies, one L2 each

// fp32 -> 16-bit float, round to nearest even (the conversion clang emits for
// gfx950 is the hardware v_cvt_pk_bf16_f32, which rounds to nearest even).
__device__ __forceinline__ bf16 to_bf16(float x) { return static_cast<bf16>(x); }
__device__ __forceinline__ float to_f32(bf16 x) { return static_cast<float>(x); }

__device__ __forceinline__ uint16_t bf16_bits(float x) {
  return __builtin_bit_cast(uint16_t, to_bf16(x));
}
__device__ __forceinline__ float bf16_bits_to_f32(uint32_t bits16) {
  return __builtin_bit_cast(float, bits16 << 16);
}

// The lossy 32 -> 16-bit converter of section 5.5: the low 16 mantissa bits
// are dropped (rounding toward zero). A NaN becomes the quiet NaN 0x7FC0 with
// its sign kept, so that no NaN turns into an infinity.
__device__ __forceinline__ uint16_t bf16_bits_trunc(float x) {
  const uint32_t u = __builtin_bit_cast(uint32_t, x);
  return x != x ? (uint16_t)(0x7FC0u | ((u >> 16) & 0x8000u)) : (uint16_t)(u >> 16);
}
// 16-bit pattern of x under the selected conversion (truncating or nearest even).
__device__ __forceinline__ uint16_t bf16_bits_mode(float x, bool trunc) {
  return trunc ? bf16_bits_trunc(x) : bf16_bits(x);
}

// Relu as a bit select: y > 0 ? y : +0. Written on the bit pattern so the
// compiler cannot turn it into a max, whose result for -0 is not +0.
__device__ __forceinline__ float relu_f32(float y) {
  return __builtin_bit_cast(float, y > 0.0f ? __builtin_bit_cast(uint32_t, y) : 0u);
}

template <typename T> struct elem_traits;
template <> struct elem_traits<float> {
  static constexpr int bytes = 4;
  static constexpr int vec = 4;  // elements per 16-byte chunk
};
template <> struct elem_traits<bf16> {
  static constexpr int bytes = 2;
  static constexpr int vec = 8;
};

__device__ __forceinline__ float load_f32(const float* p) { return *p; }
__device__ __forceinline__ float load_f32(const bf16* p) { return to_f32(*p); }
__device__ __forceinline__ void store_from_f32(float* p, float v) { *p = v; }
__device__ __forceinline__ void store_from_f32(bf16* p, float v) { *p = to_bf16(v); }
// Same, with the 16-bit conversion selectable (ignored for fp32 outputs).
__device__ __forceinline__ void store_from_f32(float* p, float v, bool) { *p = v; }
__device__ __forceinline__ void store_from_f32(bf16* p, float v, bool trunc) {
  if (trunc)
    *reinterpret_cast<uint16_t*>(p) = bf16_bits_trunc(v);
  else
    *p = to_bf16(v);
}

}  // namespace tfd
