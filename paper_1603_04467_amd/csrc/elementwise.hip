// Element-wise ops of the dense-layer step: BiasAdd, Relu, ReluGrad (Table 1
// of the paper and their gradient functions, section 4.1), the squared-error
// cost head, and ApplyGradientDescent on an fp32 Variable (section 2,
// "Variables"). All are HBM-bound: each thread moves 16-byte chunks
// (4 fp32 / 8 bf16) so that a wavefront covers 1 KiB contiguous per access;
// misaligned or ragged tensors take a per-element path.

#include "common.h"
#include "kernels.h"

namespace tfd {

namespace {

constexpr int kThreads = 256;

inline bool aligned16(const void* p) { return p == nullptr || (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

inline unsigned grid_for(int64_t work_items) {
  int64_t g = (work_items + kThreads - 1) / kThreads;
  if (g < 1) g = 1;
  if (g > 0x7fffffff) g = 0x7fffffff;
  return (unsigned)g;
}

// Chunk of V elements of T converted to fp32 and back.
template <typename T> struct Vec;
template <> struct Vec<float> {
  static constexpr int V = 4;
  __device__ static void load(const float* p, float (&x)[4]) {
    const f32x4 v = *reinterpret_cast<const f32x4*>(p);
#pragma unroll
    for (int e = 0; e < 4; ++e) x[e] = v[e];
  }
  __device__ static void store(float* p, const float (&x)[4]) {
    *reinterpret_cast<f32x4*>(p) = f32x4{x[0], x[1], x[2], x[3]};
  }
};
template <> struct Vec<bf16> {
  static constexpr int V = 8;
  __device__ static void load(const bf16* p, float (&x)[8]) {
    const u32x4 v = *reinterpret_cast<const u32x4*>(p);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[2 * e] = bf16_bits_to_f32(v[e] & 0xFFFFu);
      x[2 * e + 1] = bf16_bits_to_f32(v[e] >> 16);
    }
  }
  __device__ static void store(bf16* p, const float (&x)[8]) {
    u32x4 v;
#pragma unroll
    for (int e = 0; e < 4; ++e)
      v[e] = (uint32_t)bf16_bits(x[2 * e]) | ((uint32_t)bf16_bits(x[2 * e + 1]) << 16);
    *reinterpret_cast<u32x4*>(p) = v;
  }
};

// ---------------------------------------------------------------- BiasAdd
template <typename T, bool VEC>
__global__ __launch_bounds__(kThreads) void bias_add_kernel(const T* v, const float* b, T* out,
                                                            int64_t rows, int64_t cols) {
  constexpr int V = Vec<T>::V;
  const int64_t chunk = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  const int64_t count = rows * cols;
  if (VEC) {
    const int64_t i0 = chunk * V;
    if (i0 >= count) return;
    const int64_t c0 = i0 % cols;  // cols % V == 0: a chunk stays in one row
    float x[V];
    Vec<T>::load(v + i0, x);
#pragma unroll
    for (int e = 0; e < V; ++e) x[e] = x[e] + b[c0 + e];
    Vec<T>::store(out + i0, x);
  } else {
    if (chunk >= count) return;
    store_from_f32(out + chunk, load_f32(v + chunk) + b[chunk % cols]);
  }
}

// ---------------------------------------------------------------- Relu
template <typename T, bool VEC>
__global__ __launch_bounds__(kThreads) void relu_kernel(const T* x, T* y, int64_t count) {
  constexpr int V = Vec<T>::V;
  const int64_t chunk = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (VEC) {
    const int64_t i0 = chunk * V;
    if (i0 + V <= count) {
      float a[V];
      Vec<T>::load(x + i0, a);
#pragma unroll
      for (int e = 0; e < V; ++e) a[e] = relu_f32(a[e]);
      Vec<T>::store(y + i0, a);
    } else {
      for (int64_t i = i0; i < count; ++i) store_from_f32(y + i, relu_f32(load_f32(x + i)));
    }
  } else {
    if (chunk < count) store_from_f32(y + chunk, relu_f32(load_f32(x + chunk)));
  }
}

// ---------------------------------------------------------------- ReluGrad
__device__ __forceinline__ float relu_grad_f32(float g, float f) {
  return __builtin_bit_cast(float, f > 0.0f ? __builtin_bit_cast(uint32_t, g) : 0u);
}

template <typename T, bool VEC>
__global__ __launch_bounds__(kThreads) void relu_grad_kernel(const T* g, const T* f, T* out,
                                                             int64_t count) {
  constexpr int V = Vec<T>::V;
  const int64_t chunk = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (VEC) {
    const int64_t i0 = chunk * V;
    if (i0 + V <= count) {
      float a[V], m[V];
      Vec<T>::load(g + i0, a);
      Vec<T>::load(f + i0, m);
#pragma unroll
      for (int e = 0; e < V; ++e) a[e] = relu_grad_f32(a[e], m[e]);
      Vec<T>::store(out + i0, a);
    } else {
      for (int64_t i = i0; i < count; ++i)
        store_from_f32(out + i, relu_grad_f32(load_f32(g + i), load_f32(f + i)));
    }
  } else {
    if (chunk < count) store_from_f32(out + chunk, relu_grad_f32(load_f32(g + chunk), load_f32(f + chunk)));
  }
}

// ---------------------------------------------------------------- squared-error cost head
// Pass 1: grad = out - target (fp32 difference, one rounding to T) and one
// float64 partial sum of squares per block (fixed grid for a given count,
// fixed order inside the block). Pass 2: one block sums the partials in
// index order and halves.
constexpr int kLossMaxBlocks = 1024;

inline int loss_blocks(int64_t count, int V) {
  int64_t chunks = (count + V - 1) / V;
  int64_t b = (chunks + kThreads - 1) / kThreads;
  if (b < 1) b = 1;
  if (b > kLossMaxBlocks) b = kLossMaxBlocks;
  return (int)b;
}

__device__ __forceinline__ double block_sum(double v, double* sh) {
  const int tid = threadIdx.x;
  sh[tid] = v;
  __syncthreads();
#pragma unroll
  for (int s = kThreads / 2; s > 0; s >>= 1) {
    if (tid < s) sh[tid] += sh[tid + s];
    __syncthreads();
  }
  return sh[0];
}

template <typename T, bool VEC>
__global__ __launch_bounds__(kThreads) void loss_grad_kernel(const T* out, const T* target, T* grad,
                                                             double* partial, int64_t count) {
  constexpr int V = Vec<T>::V;
  __shared__ double sh[kThreads];
  double acc = 0.0;
  const int64_t nchunks = (count + V - 1) / V;
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  for (int64_t c = (int64_t)blockIdx.x * kThreads + threadIdx.x; c < nchunks; c += stride) {
    const int64_t i0 = c * V;
    if (VEC && i0 + V <= count) {
      float o[V], t[V];
      Vec<T>::load(out + i0, o);
      if (target) {
        Vec<T>::load(target + i0, t);
      } else {
#pragma unroll
        for (int e = 0; e < V; ++e) t[e] = 0.0f;
      }
#pragma unroll
      for (int e = 0; e < V; ++e) {
        o[e] = o[e] - t[e];
        acc += (double)o[e] * (double)o[e];
      }
      Vec<T>::store(grad + i0, o);
    } else {
      for (int64_t i = i0; i < count && i < i0 + V; ++i) {
        const float d = load_f32(out + i) - (target ? load_f32(target + i) : 0.0f);
        acc += (double)d * (double)d;
        store_from_f32(grad + i, d);
      }
    }
  }
  const double s = block_sum(acc, sh);
  if (threadIdx.x == 0) partial[blockIdx.x] = s;
}

__global__ __launch_bounds__(kThreads) void loss_final_kernel(const double* partial, int n, double* loss) {
  __shared__ double sh[kThreads];
  double acc = 0.0;
  for (int i = threadIdx.x; i < n; i += kThreads) acc += partial[i];
  const double s = block_sum(acc, sh);
  if (threadIdx.x == 0) *loss = 0.5 * s;
}

// ---------------------------------------------------------------- ApplyGradientDescent
template <bool VEC, bool SHADOW>
__global__ __launch_bounds__(kThreads) void sgd_kernel(float* var, float alpha, const float* delta,
                                                       int64_t count, uint16_t* shadow, bool trunc) {
  const int64_t chunk = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  const float na = -alpha;
  if (VEC) {
    const int64_t i0 = chunk * 4;
    if (i0 + 4 <= count) {
      f32x4 v = *reinterpret_cast<const f32x4*>(var + i0);
      const f32x4 d = *reinterpret_cast<const f32x4*>(delta + i0);
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = __builtin_fmaf(na, d[e], v[e]);
      *reinterpret_cast<f32x4*>(var + i0) = v;
      if (SHADOW) {
        const uint32_t lo = (uint32_t)bf16_bits_mode(v[0], trunc) | ((uint32_t)bf16_bits_mode(v[1], trunc) << 16);
        const uint32_t hi = (uint32_t)bf16_bits_mode(v[2], trunc) | ((uint32_t)bf16_bits_mode(v[3], trunc) << 16);
        *reinterpret_cast<uint2*>(shadow + i0) = make_uint2(lo, hi);
      }
    } else {
      for (int64_t i = i0; i < count; ++i) {
        const float v = __builtin_fmaf(na, delta[i], var[i]);
        var[i] = v;
        if (SHADOW) shadow[i] = bf16_bits_mode(v, trunc);
      }
    }
  } else {
    if (chunk < count) {
      const float v = __builtin_fmaf(na, delta[chunk], var[chunk]);
      var[chunk] = v;
      if (SHADOW) shadow[chunk] = bf16_bits_mode(v, trunc);
    }
  }
}

// ApplyGradientDescent on a weight matrix, refreshing its 16-bit operand
// copies: 64 x 64 tiles, one block each. The updated tile's 16-bit bits are
// staged in LDS so that the transposed copy is also written in 16-byte row
// chunks. VEC: whole tiles with 16-byte aligned rows (else per-element).
constexpr int kSgdTile = 64;

template <bool VEC>
__global__ __launch_bounds__(kThreads) void sgd_matrix_kernel(float* __restrict__ var, float alpha,
                                                              const float* __restrict__ delta, int64_t rows,
                                                              int64_t cols, uint16_t* __restrict__ shadow,
                                                              uint16_t* __restrict__ shadow_t, bool trunc) {
  __shared__ uint16_t tile[kSgdTile][kSgdTile + 2];
  const int64_t r0 = (int64_t)blockIdx.y * kSgdTile, c0 = (int64_t)blockIdx.x * kSgdTile;
  const int tid = threadIdx.x;
  const float na = -alpha;
  const bool full = VEC && r0 + kSgdTile <= rows && c0 + kSgdTile <= cols;
  if (full) {
    const int cc = (tid & 15) * 4;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int rr = (tid >> 4) + 16 * i;
      const int64_t off = (r0 + rr) * cols + c0 + cc;
      f32x4 v = *reinterpret_cast<const f32x4*>(var + off);
      const f32x4 d = *reinterpret_cast<const f32x4*>(delta + off);
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = __builtin_fmaf(na, d[e], v[e]);
      *reinterpret_cast<f32x4*>(var + off) = v;
      uint16_t b[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        b[e] = bf16_bits_mode(v[e], trunc);
        tile[rr][cc + e] = b[e];
      }
      if (shadow)
        *reinterpret_cast<uint2*>(shadow + off) =
            make_uint2((uint32_t)b[0] | ((uint32_t)b[1] << 16), (uint32_t)b[2] | ((uint32_t)b[3] << 16));
    }
  } else {
    for (int i = tid; i < kSgdTile * kSgdTile; i += kThreads) {
      const int rr = i / kSgdTile, cc = i % kSgdTile;
      const int64_t r = r0 + rr, c = c0 + cc;
      if (r < rows && c < cols) {
        const int64_t off = r * cols + c;
        const float v = __builtin_fmaf(na, delta[off], var[off]);
        var[off] = v;
        const uint16_t b = bf16_bits_mode(v, trunc);
        tile[rr][cc] = b;
        if (shadow) shadow[off] = b;
      }
    }
  }
  if (!shadow_t) return;
  __syncthreads();
  // transposed copy: output row c (= input column), 64 input rows per tile
  if (full && (rows % 8) == 0) {
    const int oc = tid >> 2, seg = (tid & 3) * 16;
    uint32_t w[8];
#pragma unroll
    for (int e = 0; e < 8; ++e)
      w[e] = (uint32_t)tile[seg + 2 * e][oc] | ((uint32_t)tile[seg + 2 * e + 1][oc] << 16);
    uint16_t* dst = shadow_t + (c0 + oc) * rows + r0 + seg;
    *reinterpret_cast<u32x4*>(dst) = u32x4{w[0], w[1], w[2], w[3]};
    *reinterpret_cast<u32x4*>(dst + 8) = u32x4{w[4], w[5], w[6], w[7]};
  } else {
    for (int i = tid; i < kSgdTile * kSgdTile; i += kThreads) {
      const int oc = i / kSgdTile, rr = i % kSgdTile;
      const int64_t r = r0 + rr, c = c0 + oc;
      if (r < rows && c < cols) shadow_t[c * rows + r] = tile[rr][oc];
    }
  }
}

}  // namespace

hipError_t launch_sgd_matrix(float* var, float alpha, const float* delta, int64_t rows, int64_t cols,
                             uint16_t* shadow, uint16_t* shadow_t, bool trunc, hipStream_t s) {
  // without the transposed copy the matrix is one contiguous array: the
  // element-wise update (whole 1 KiB per wave instruction) does the same
  // arithmetic per element
  if (!shadow_t) return launch_sgd(var, alpha, delta, rows * cols, shadow, trunc, s);
  const bool vec = aligned16(var) && aligned16(delta) && cols % 4 == 0 &&
                   ((reinterpret_cast<uintptr_t>(shadow) & 7) == 0) && aligned16(shadow_t);
  dim3 grid((unsigned)((cols + kSgdTile - 1) / kSgdTile), (unsigned)((rows + kSgdTile - 1) / kSgdTile));
  if (vec)
    hipLaunchKernelGGL((sgd_matrix_kernel<true>), grid, kThreads, 0, s, var, alpha, delta, rows, cols, shadow, shadow_t,
                       trunc);
  else
    hipLaunchKernelGGL((sgd_matrix_kernel<false>), grid, kThreads, 0, s, var, alpha, delta, rows, cols, shadow,
                       shadow_t, trunc);
  return hipGetLastError();
}

hipError_t launch_bias_add(const void* value, const float* bias, void* out, int64_t rows, int64_t cols,
                           bool bf16_t, hipStream_t s) {
  const int V = bf16_t ? 8 : 4;
  const bool vec = cols % V == 0 && aligned16(value) && aligned16(out);
  const int64_t count = rows * cols;
  const unsigned g = grid_for(vec ? (count + V - 1) / V : count);
  if (bf16_t) {
    if (vec)
      hipLaunchKernelGGL((bias_add_kernel<bf16, true>), g, kThreads, 0, s, (const bf16*)value, bias, (bf16*)out, rows, cols);
    else
      hipLaunchKernelGGL((bias_add_kernel<bf16, false>), g, kThreads, 0, s, (const bf16*)value, bias, (bf16*)out, rows, cols);
  } else {
    if (vec)
      hipLaunchKernelGGL((bias_add_kernel<float, true>), g, kThreads, 0, s, (const float*)value, bias, (float*)out, rows, cols);
    else
      hipLaunchKernelGGL((bias_add_kernel<float, false>), g, kThreads, 0, s, (const float*)value, bias, (float*)out, rows, cols);
  }
  return hipGetLastError();
}

hipError_t launch_relu(const void* x, void* y, int64_t count, bool bf16_t, hipStream_t s) {
  const int V = bf16_t ? 8 : 4;
  const bool vec = aligned16(x) && aligned16(y);
  const unsigned g = grid_for(vec ? (count + V - 1) / V : count);
  if (bf16_t) {
    if (vec) hipLaunchKernelGGL((relu_kernel<bf16, true>), g, kThreads, 0, s, (const bf16*)x, (bf16*)y, count);
    else hipLaunchKernelGGL((relu_kernel<bf16, false>), g, kThreads, 0, s, (const bf16*)x, (bf16*)y, count);
  } else {
    if (vec) hipLaunchKernelGGL((relu_kernel<float, true>), g, kThreads, 0, s, (const float*)x, (float*)y, count);
    else hipLaunchKernelGGL((relu_kernel<float, false>), g, kThreads, 0, s, (const float*)x, (float*)y, count);
  }
  return hipGetLastError();
}

hipError_t launch_relu_grad(const void* gp, const void* f, void* out, int64_t count, bool bf16_t,
                            hipStream_t s) {
  const int V = bf16_t ? 8 : 4;
  const bool vec = aligned16(gp) && aligned16(f) && aligned16(out);
  const unsigned g = grid_for(vec ? (count + V - 1) / V : count);
  if (bf16_t) {
    if (vec) hipLaunchKernelGGL((relu_grad_kernel<bf16, true>), g, kThreads, 0, s, (const bf16*)gp, (const bf16*)f, (bf16*)out, count);
    else hipLaunchKernelGGL((relu_grad_kernel<bf16, false>), g, kThreads, 0, s, (const bf16*)gp, (const bf16*)f, (bf16*)out, count);
  } else {
    if (vec) hipLaunchKernelGGL((relu_grad_kernel<float, true>), g, kThreads, 0, s, (const float*)gp, (const float*)f, (float*)out, count);
    else hipLaunchKernelGGL((relu_grad_kernel<float, false>), g, kThreads, 0, s, (const float*)gp, (const float*)f, (float*)out, count);
  }
  return hipGetLastError();
}

size_t loss_ws_bytes(int64_t count, bool bf16_t) {
  return (size_t)loss_blocks(count, bf16_t ? 8 : 4) * sizeof(double);
}

hipError_t launch_l2_loss_grad(const void* out, const void* target, void* grad, double* loss,
                               int64_t count, bool bf16_t, void* ws, hipStream_t s) {
  const int V = bf16_t ? 8 : 4;
  const int blocks = loss_blocks(count, V);
  const bool vec = aligned16(out) && aligned16(target) && aligned16(grad);
  double* partial = static_cast<double*>(ws);
  if (bf16_t) {
    if (vec) hipLaunchKernelGGL((loss_grad_kernel<bf16, true>), blocks, kThreads, 0, s, (const bf16*)out, (const bf16*)target, (bf16*)grad, partial, count);
    else hipLaunchKernelGGL((loss_grad_kernel<bf16, false>), blocks, kThreads, 0, s, (const bf16*)out, (const bf16*)target, (bf16*)grad, partial, count);
  } else {
    if (vec) hipLaunchKernelGGL((loss_grad_kernel<float, true>), blocks, kThreads, 0, s, (const float*)out, (const float*)target, (float*)grad, partial, count);
    else hipLaunchKernelGGL((loss_grad_kernel<float, false>), blocks, kThreads, 0, s, (const float*)out, (const float*)target, (float*)grad, partial, count);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(loss_final_kernel, 1, kThreads, 0, s, (const double*)partial, blocks, loss);
  return hipGetLastError();
}

hipError_t launch_loss_final(const double* partial, int n, double* loss, hipStream_t s) {
  hipLaunchKernelGGL(loss_final_kernel, 1, kThreads, 0, s, partial, n, loss);
  return hipGetLastError();
}

hipError_t launch_sgd(float* var, float alpha, const float* delta, int64_t count, uint16_t* shadow, bool trunc,
                      hipStream_t s) {
  const bool vec = aligned16(var) && aligned16(delta) && ((reinterpret_cast<uintptr_t>(shadow) & 7) == 0);
  const unsigned g = grid_for(vec ? (count + 3) / 4 : count);
  if (vec) {
    if (shadow) hipLaunchKernelGGL((sgd_kernel<true, true>), g, kThreads, 0, s, var, alpha, delta, count, shadow, trunc);
    else hipLaunchKernelGGL((sgd_kernel<true, false>), g, kThreads, 0, s, var, alpha, delta, count, shadow, trunc);
  } else {
    if (shadow) hipLaunchKernelGGL((sgd_kernel<false, true>), g, kThreads, 0, s, var, alpha, delta, count, shadow, trunc);
    else hipLaunchKernelGGL((sgd_kernel<false, false>), g, kThreads, 0, s, var, alpha, delta, count, shadow, trunc);
  }
  return hipGetLastError();
}

}  // namespace tfd
