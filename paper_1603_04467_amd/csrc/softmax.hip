// Classifier cost head: SoftMax (the paper's section 2, Table 1) of the output
// layer's logits, the cross-entropy against integer class labels
// L = sum_n (log sum_j exp(z_nj) - z_n,y_n), and its gradient with respect to
// the logits, G = softmax(z) - onehot(y).
//
// One wavefront per row (4 rows per 256-thread block): the lanes stride over
// the row for the maximum, the sum of exp(z - max) and the gradient, with
// butterfly shuffles for the two row reductions. Each block writes one float64
// partial of its rows' loss terms (in row order); one final block sums the
// partials in index order, so the loss is bitwise reproducible.

#include "common.h"
#include "kernels.h"

namespace tfd {

namespace {

constexpr int kThreads = 256;
constexpr int kRowsPerBlock = kThreads / kWave;

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

template <typename T>
__global__ __launch_bounds__(kThreads) void softmax_xent_kernel(const T* __restrict__ z,
                                                                const int32_t* __restrict__ labels,
                                                                T* __restrict__ grad, double* __restrict__ partial,
                                                                int64_t rows, int64_t cols) {
  __shared__ double terms[kRowsPerBlock];
  const int lane = threadIdx.x & (kWave - 1), w = threadIdx.x / kWave;
  const int64_t row = (int64_t)blockIdx.x * kRowsPerBlock + w;
  double term = 0.0;
  if (row < rows) {
    const T* zr = z + row * cols;
    T* gr = grad + row * cols;
    float m = -INFINITY;
    for (int64_t c = lane; c < cols; c += kWave) m = fmaxf(m, load_f32(zr + c));
    m = wave_max(m);
    float s = 0.0f;
    for (int64_t c = lane; c < cols; c += kWave) s += expf(load_f32(zr + c) - m);
    s = wave_sum(s);
    const float inv = 1.0f / s;
    const int32_t y = labels[row];
    for (int64_t c = lane; c < cols; c += kWave) {
      float p = expf(load_f32(zr + c) - m) * inv;
      if (c == y) p -= 1.0f;
      store_from_f32(gr + c, p);
    }
    if (lane == 0) {
      term = (y >= 0 && y < cols) ? (double)logf(s) + (double)m - (double)load_f32(zr + y)
                                  : __builtin_nan("");
    }
  }
  if (lane == 0) terms[w] = term;
  __syncthreads();
  if (threadIdx.x == 0) {
    double acc = 0.0;
#pragma unroll
    for (int i = 0; i < kRowsPerBlock; ++i) acc += terms[i];
    partial[blockIdx.x] = acc;
  }
}

__global__ __launch_bounds__(kThreads) void sum_partials_kernel(const double* partial, int64_t n, double* out) {
  __shared__ double sh[kThreads];
  double acc = 0.0;
  for (int64_t i = threadIdx.x; i < n; i += kThreads) acc += partial[i];
  sh[threadIdx.x] = acc;
  __syncthreads();
#pragma unroll
  for (int s = kThreads / 2; s > 0; s >>= 1) {
    if ((int)threadIdx.x < s) sh[threadIdx.x] += sh[threadIdx.x + s];
    __syncthreads();
  }
  if (threadIdx.x == 0) *out = sh[0];
}

}  // namespace

size_t softmax_xent_ws_bytes(int64_t rows) {
  const int64_t blocks = rows > 0 ? (rows + kRowsPerBlock - 1) / kRowsPerBlock : 1;
  return (size_t)blocks * sizeof(double);
}

hipError_t launch_softmax_xent(const void* logits, const int32_t* labels, void* grad, double* loss, int64_t rows,
                               int64_t cols, bool bf16_t, void* ws, hipStream_t s) {
  double* partial = static_cast<double*>(ws);
  const int64_t blocks = rows > 0 ? (rows + kRowsPerBlock - 1) / kRowsPerBlock : 0;
  if (blocks > 0) {
    if (bf16_t)
      hipLaunchKernelGGL((softmax_xent_kernel<bf16>), dim3((unsigned)blocks), kThreads, 0, s, (const bf16*)logits,
                         labels, (bf16*)grad, partial, rows, cols);
    else
      hipLaunchKernelGGL((softmax_xent_kernel<float>), dim3((unsigned)blocks), kThreads, 0, s, (const float*)logits,
                         labels, (float*)grad, partial, rows, cols);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(sum_partials_kernel, 1, kThreads, 0, s, (const double*)partial, blocks, loss);
  return hipGetLastError();
}

}  // namespace tfd
