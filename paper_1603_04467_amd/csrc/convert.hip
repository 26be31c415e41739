// The 32 <-> 16-bit conversion nodes of section 5.5 (lossy compression of
// tensors moved between devices): fp32 -> 16 bits by dropping the low 16
// mantissa bits (or, selectable, rounding to nearest even), and 16 -> 32 bits
// by filling the low half with zeros.
//
// Both kernels stream: each thread converts 8 elements per iteration with
// 16-byte loads and stores (fp32 -> 16: 32 bytes in, 16 out; 16 -> fp32: 16 in,
// 32 out), in a grid-stride loop. Unaligned buffers take the per-element path.

#include "common.h"
#include "kernels.h"

namespace tfd {

namespace {

constexpr int kThreads = 256;
constexpr int64_t kMaxBlocks = 1 << 20;

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

unsigned blocks_for(int64_t items) {
  const int64_t b = (items + kThreads - 1) / kThreads;
  return (unsigned)(b < 1 ? 1 : (b > kMaxBlocks ? kMaxBlocks : b));
}

template <bool VEC>
__global__ __launch_bounds__(kThreads) void to_bf16_kernel(const float* __restrict__ src, uint16_t* __restrict__ dst,
                                                           int64_t count, bool trunc) {
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  const int64_t first = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (VEC) {
    const int64_t chunks = count / 8;
    for (int64_t c = first; c < chunks; c += stride) {
      const f32x4 a = *reinterpret_cast<const f32x4*>(src + 8 * c);
      const f32x4 b = *reinterpret_cast<const f32x4*>(src + 8 * c + 4);
      u32x4 o;
      o[0] = (uint32_t)bf16_bits_mode(a[0], trunc) | ((uint32_t)bf16_bits_mode(a[1], trunc) << 16);
      o[1] = (uint32_t)bf16_bits_mode(a[2], trunc) | ((uint32_t)bf16_bits_mode(a[3], trunc) << 16);
      o[2] = (uint32_t)bf16_bits_mode(b[0], trunc) | ((uint32_t)bf16_bits_mode(b[1], trunc) << 16);
      o[3] = (uint32_t)bf16_bits_mode(b[2], trunc) | ((uint32_t)bf16_bits_mode(b[3], trunc) << 16);
      *reinterpret_cast<u32x4*>(dst + 8 * c) = o;
    }
    const int64_t i = 8 * chunks + first;  // tail: fewer than 8 elements
    if (first < 8 && i < count) dst[i] = bf16_bits_mode(src[i], trunc);
  } else {
    for (int64_t i = first; i < count; i += stride) dst[i] = bf16_bits_mode(src[i], trunc);
  }
}

template <bool VEC>
__global__ __launch_bounds__(kThreads) void to_f32_kernel(const uint16_t* __restrict__ src, float* __restrict__ dst,
                                                          int64_t count) {
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  const int64_t first = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (VEC) {
    const int64_t chunks = count / 8;
    for (int64_t c = first; c < chunks; c += stride) {
      const u32x4 v = *reinterpret_cast<const u32x4*>(src + 8 * c);
      u32x4 a, b;
      a[0] = v[0] << 16;
      a[1] = v[0] & 0xFFFF0000u;
      a[2] = v[1] << 16;
      a[3] = v[1] & 0xFFFF0000u;
      b[0] = v[2] << 16;
      b[1] = v[2] & 0xFFFF0000u;
      b[2] = v[3] << 16;
      b[3] = v[3] & 0xFFFF0000u;
      *reinterpret_cast<u32x4*>(dst + 8 * c) = a;
      *reinterpret_cast<u32x4*>(dst + 8 * c + 4) = b;
    }
    const int64_t i = 8 * chunks + first;
    if (first < 8 && i < count) dst[i] = bf16_bits_to_f32(src[i]);
  } else {
    for (int64_t i = first; i < count; i += stride) dst[i] = bf16_bits_to_f32(src[i]);
  }
}

}  // namespace

hipError_t launch_convert_to_bf16(const float* src, uint16_t* dst, int64_t count, bool trunc, hipStream_t s) {
  if (aligned16(src) && aligned16(dst))
    hipLaunchKernelGGL((to_bf16_kernel<true>), blocks_for(count / 8 > 0 ? count / 8 : 1), kThreads, 0, s, src, dst,
                       count, trunc);
  else
    hipLaunchKernelGGL((to_bf16_kernel<false>), blocks_for(count), kThreads, 0, s, src, dst, count, trunc);
  return hipGetLastError();
}

hipError_t launch_convert_to_f32(const uint16_t* src, float* dst, int64_t count, hipStream_t s) {
  if (aligned16(src) && aligned16(dst))
    hipLaunchKernelGGL((to_f32_kernel<true>), blocks_for(count / 8 > 0 ? count / 8 : 1), kThreads, 0, s, src, dst,
                       count);
  else
    hipLaunchKernelGGL((to_f32_kernel<false>), blocks_for(count), kThreads, 0, s, src, dst, count);
  return hipGetLastError();
}

}  // namespace tfd
