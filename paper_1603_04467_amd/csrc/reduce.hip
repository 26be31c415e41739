// BiasAddGrad (the bias gradient of the broadcast Add, section 4.1 of the
// paper), optionally fused with ReluGrad: one pass over the upstream
// gradient G (and the stored Relu output H) that writes the masked gradient
// dY and reduces it over the batch rows. The Relu test comes either from H
// (H > 0) or from a ReLU mask that holds the same test as one bit per
// element (written by the forward MatMul, or by relu_mask_kernel below).
//
// Pass 1 (grid: column groups x row chunks): each thread owns one 16-byte
// column chunk (4 fp32 / 8 bf16 columns) and walks the rows of its chunk with
// a stride of 4, so a wavefront reads 1 KiB of one row per access. The four
// row phases of a block are combined through LDS in a fixed order and the
// block writes one fp32 partial per column. Pass 2 sums the partials of each
// column in row-chunk order. The grid depends only on (rows, cols, type), so
// the bits of the result do not change from call to call.

#include <mutex>

#include "common.h"
#include "kernels.h"

namespace tfd {

namespace {

constexpr int kThreads = 256;
constexpr int kColChunks = 64;               // column chunks per block
constexpr int kRowPhases = kThreads / kColChunks;
// Target grid size of pass 1, by element width, and rows loaded per round
// (all loads of a round are issued before its ordered additions). Measured
// on MI355X: 16-bit tiles stream fastest with 1024 blocks, and with 2 rows
// per round when dY is written (16384 x 32768 with a mask: 0.475 -> 0.425
// ms); fp32 tiles with 2048 blocks and 4 rows.
constexpr int64_t target_blocks(int V) { return V == 8 ? 1024 : 2048; }
template <typename T, bool WRITE>
constexpr int row_unroll() { return sizeof(T) == 2 && WRITE ? 2 : 4; }

struct ReducePlan {
  int64_t col_groups, row_chunks, rows_per_chunk;
};

ReducePlan plan(int64_t rows, int64_t cols, int V) {
  ReducePlan p;
  p.col_groups = (cols + kColChunks * V - 1) / (kColChunks * V);
  if (p.col_groups < 1) p.col_groups = 1;
  int64_t want = (target_blocks(V) + p.col_groups - 1) / p.col_groups;
  int64_t max_chunks = (rows + 4 * kRowPhases - 1) / (4 * kRowPhases);  // >= 16 rows per chunk
  if (max_chunks < 1) max_chunks = 1;
  if (want > max_chunks) want = max_chunks;
  if (want < 1) want = 1;
  p.rows_per_chunk = (rows + want - 1) / want;
  p.row_chunks = p.rows_per_chunk > 0 ? (rows + p.rows_per_chunk - 1) / p.rows_per_chunk : 1;
  if (p.row_chunks < 1) p.row_chunks = 1;
  return p;
}

template <typename T> struct Chunk16;
template <> struct Chunk16<float> {
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
template <> struct Chunk16<bf16> {
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

__device__ __forceinline__ float masked(float g, float f) {
  return __builtin_bit_cast(float, f > 0.0f ? __builtin_bit_cast(uint32_t, g) : 0u);
}
__device__ __forceinline__ float kept(float g, uint32_t bit) {
  return __builtin_bit_cast(float, bit ? __builtin_bit_cast(uint32_t, g) : 0u);
}

// Where the Relu test comes from: none (BiasAddGrad alone), the stored
// features (f > 0), or a bit mask (bit (r, c) of mb, row r at word r * ldm).
constexpr int kNoMask = 0, kFeatures = 1, kBits = 2;

template <typename T, int MASK, bool WRITE, bool VEC>
__global__ __launch_bounds__(kThreads) void colsum_partial_kernel(const T* __restrict__ g,
                                                                  const T* __restrict__ f,
                                                                  const uint32_t* __restrict__ mb, int64_t ldm,
                                                                  T* __restrict__ out,
                                                                  float* __restrict__ partial, int64_t rows,
                                                                  int64_t cols, int64_t rows_per_chunk) {
  constexpr int V = Chunk16<T>::V;
  __shared__ float sh[kRowPhases][kColChunks * V];
  const int cv = threadIdx.x % kColChunks;
  const int phase = threadIdx.x / kColChunks;
  const int64_t c0 = ((int64_t)blockIdx.x * kColChunks + cv) * V;
  const int64_t chunk = blockIdx.y;
  const int64_t r_begin = chunk * rows_per_chunk;
  const int64_t r_end = min(rows, r_begin + rows_per_chunk);

  float acc[V];
#pragma unroll
  for (int e = 0; e < V; ++e) acc[e] = 0.0f;

  if (c0 < cols) {
    const bool full = VEC && (c0 + V <= cols);
    int64_t r = r_begin + phase;
    if (full) {
      // U rows per round: all loads issued before the ordered additions
      constexpr int U = row_unroll<T, WRITE>();
      for (; r + (U - 1) * kRowPhases < r_end; r += U * kRowPhases) {
        float x[U][V];
#pragma unroll
        for (int u = 0; u < U; ++u) Chunk16<T>::load(g + (r + u * kRowPhases) * cols + c0, x[u]);
        if (MASK == kFeatures) {
          float m[U][V];
#pragma unroll
          for (int u = 0; u < U; ++u) Chunk16<T>::load(f + (r + u * kRowPhases) * cols + c0, m[u]);
#pragma unroll
          for (int u = 0; u < U; ++u)
#pragma unroll
            for (int e = 0; e < V; ++e) x[u][e] = masked(x[u][e], m[u][e]);
        }
        if (MASK == kBits) {
          // the chunk's V bits lie in one word (c0 is a multiple of V)
          uint32_t w[U];
#pragma unroll
          for (int u = 0; u < U; ++u) w[u] = mb[(r + u * kRowPhases) * ldm + (c0 >> 5)] >> (c0 & 31);
#pragma unroll
          for (int u = 0; u < U; ++u)
#pragma unroll
            for (int e = 0; e < V; ++e) x[u][e] = kept(x[u][e], (w[u] >> e) & 1u);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
          if (WRITE) Chunk16<T>::store(out + (r + u * kRowPhases) * cols + c0, x[u]);
#pragma unroll
          for (int e = 0; e < V; ++e) acc[e] += x[u][e];
        }
      }
    }
    for (; r < r_end; r += kRowPhases) {
      const int64_t base = r * cols + c0;
      float x[V];
      if (full) {
        Chunk16<T>::load(g + base, x);
        if (MASK == kFeatures) {
          float m[V];
          Chunk16<T>::load(f + base, m);
#pragma unroll
          for (int e = 0; e < V; ++e) x[e] = masked(x[e], m[e]);
        }
        if (MASK == kBits) {
          const uint32_t w = mb[r * ldm + (c0 >> 5)] >> (c0 & 31);
#pragma unroll
          for (int e = 0; e < V; ++e) x[e] = kept(x[e], (w >> e) & 1u);
        }
        if (WRITE) Chunk16<T>::store(out + base, x);
#pragma unroll
        for (int e = 0; e < V; ++e) acc[e] += x[e];
      } else {
#pragma unroll
        for (int e = 0; e < V; ++e) {
          if (c0 + e < cols) {
            float v = load_f32(g + base + e);
            if (MASK == kFeatures) v = masked(v, load_f32(f + base + e));
            if (MASK == kBits) v = kept(v, (mb[r * ldm + ((c0 + e) >> 5)] >> ((c0 + e) & 31)) & 1u);
            if (WRITE) store_from_f32(out + base + e, v);
            acc[e] += v;
          }
        }
      }
    }
  }
#pragma unroll
  for (int e = 0; e < V; ++e) sh[phase][cv * V + e] = acc[e];
  __syncthreads();
  for (int i = threadIdx.x; i < kColChunks * V; i += kThreads) {
    const int64_t c = (int64_t)blockIdx.x * kColChunks * V + i;
    if (c < cols) {
      float s = sh[0][i];
#pragma unroll
      for (int ph = 1; ph < kRowPhases; ++ph) s += sh[ph][i];
      partial[chunk * cols + c] = s;
    }
  }
}

// ReLU mask: one thread per 32-column word of a row; bit j is set when
// element 32 w + j is > 0 (the test ReluGrad applies to the stored forward
// output). VEC: the row's 32 values are read as 16-byte chunks (cols a
// multiple of 32, aligned rows); otherwise per element, with the bits past
// the last column left 0.
template <typename T, bool VEC>
__global__ __launch_bounds__(kThreads) void relu_mask_kernel(const T* __restrict__ x, int64_t ldx,
                                                             uint32_t* __restrict__ mask, int64_t ldm,
                                                             int64_t rows, int64_t cols) {
  const int64_t words = (cols + 31) / 32;
  const int64_t total = rows * words;
  for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < total; i += (int64_t)gridDim.x * kThreads) {
    const int64_t r = i / words, w = i - r * words;
    const T* row = x + r * ldx + w * 32;
    uint32_t bits = 0;
    if (VEC) {
      constexpr int V = Chunk16<T>::V;
#pragma unroll
      for (int c = 0; c < 32 / V; ++c) {
        float v[V];
        Chunk16<T>::load(row + c * V, v);
#pragma unroll
        for (int e = 0; e < V; ++e) bits |= (v[e] > 0.0f ? 1u : 0u) << (c * V + e);
      }
    } else {
      const int n = (int)min<int64_t>(32, cols - w * 32);
      for (int e = 0; e < n; ++e) bits |= (load_f32(row + e) > 0.0f ? 1u : 0u) << e;
    }
    mask[r * ldm + w] = bits;
  }
}

// Sums the row-chunk partials of each column in chunk order. The loads are
// independent of the running sum, so they are issued kBatch at a time before
// the (ordered) additions.
__global__ __launch_bounds__(kThreads) void colsum_final_kernel(const float* partial, float* db,
                                                                int64_t row_chunks, int64_t cols) {
  constexpr int kBatch = 16;
  const int64_t c = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (c >= cols) return;
  float s = 0.0f;
  int64_t k = 0;
  for (; k + kBatch <= row_chunks; k += kBatch) {
    float v[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) v[u] = partial[(k + u) * cols + c];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) s += v[u];
  }
  for (; k < row_chunks; ++k) s += partial[k * cols + c];
  db[c] = s;
}

template <typename T>
hipError_t launch_t(const T* g, const T* f, const uint32_t* mb, int64_t ldm, T* out, float* db, int64_t rows,
                    int64_t cols, float* ws, hipStream_t s) {
  constexpr int V = Chunk16<T>::V;
  const ReducePlan p = plan(rows, cols, V);
  auto al = [](const void* q) { return (reinterpret_cast<uintptr_t>(q) & 15) == 0; };
  const bool vec = (cols % V == 0) && al(g) && (!f || al(f)) && (!out || al(out));
  dim3 grid((unsigned)p.col_groups, (unsigned)p.row_chunks);
#define TFD_LAUNCH(M, W, VE)                                                                             \
  hipLaunchKernelGGL((colsum_partial_kernel<T, M, W, VE>), grid, kThreads, 0, s, g, f, mb, ldm, out, ws, rows, \
                     cols, p.rows_per_chunk)
  const int mode = mb ? kBits : (f ? kFeatures : kNoMask);
  const bool write = out != nullptr;
  if (vec) {
    if (mode == kBits) {
      if (write) TFD_LAUNCH(kBits, true, true);
      else TFD_LAUNCH(kBits, false, true);
    } else if (mode == kFeatures) {
      if (write) TFD_LAUNCH(kFeatures, true, true);
      else TFD_LAUNCH(kFeatures, false, true);
    } else {
      if (write) TFD_LAUNCH(kNoMask, true, true);
      else TFD_LAUNCH(kNoMask, false, true);
    }
  } else {
    if (mode == kBits) {
      if (write) TFD_LAUNCH(kBits, true, false);
      else TFD_LAUNCH(kBits, false, false);
    } else if (mode == kFeatures) {
      if (write) TFD_LAUNCH(kFeatures, true, false);
      else TFD_LAUNCH(kFeatures, false, false);
    } else {
      if (write) TFD_LAUNCH(kNoMask, true, false);
      else TFD_LAUNCH(kNoMask, false, false);
    }
  }
#undef TFD_LAUNCH
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const unsigned g2 = (unsigned)((cols + kThreads - 1) / kThreads);
  hipLaunchKernelGGL(colsum_final_kernel, g2, kThreads, 0, s, (const float*)ws, db, p.row_chunks, cols);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_colsum_final(const float* partial, float* db, int64_t chunks, int64_t cols, hipStream_t s) {
  const unsigned g = (unsigned)((cols + kThreads - 1) / kThreads);
  hipLaunchKernelGGL(colsum_final_kernel, g, kThreads, 0, s, partial, db, chunks, cols);
  return hipGetLastError();
}

size_t reduction_ws_bytes(int64_t rows, int64_t cols, bool bf16_t) {
  const ReducePlan p = plan(rows, cols, bf16_t ? 8 : 4);
  return (size_t)(p.row_chunks * cols) * sizeof(float);
}

hipError_t launch_relu_grad_bias_add_grad(const void* g, const void* f, void* out, float* db,
                                          int64_t rows, int64_t cols, bool bf16_t, void* ws,
                                          hipStream_t s) {
  if (bf16_t)
    return launch_t<bf16>((const bf16*)g, (const bf16*)f, nullptr, 0, (bf16*)out, db, rows, cols, (float*)ws, s);
  return launch_t<float>((const float*)g, (const float*)f, nullptr, 0, (float*)out, db, rows, cols, (float*)ws, s);
}

hipError_t launch_relu_mask_grad_bias_add_grad(const void* g, const uint32_t* mask, int64_t ldm, void* out,
                                               float* db, int64_t rows, int64_t cols, bool bf16_t, void* ws,
                                               hipStream_t s) {
  if (bf16_t)
    return launch_t<bf16>((const bf16*)g, nullptr, mask, ldm, (bf16*)out, db, rows, cols, (float*)ws, s);
  return launch_t<float>((const float*)g, nullptr, mask, ldm, (float*)out, db, rows, cols, (float*)ws, s);
}

hipError_t launch_relu_mask(const void* x, int64_t ldx, uint32_t* mask, int64_t ldm, int64_t rows, int64_t cols,
                            bool bf16_t, hipStream_t s) {
  const int64_t total = rows * ((cols + 31) / 32);
  if (total == 0) return hipSuccess;
  int64_t blocks = (total + kThreads - 1) / kThreads;
  if (blocks > 65536) blocks = 65536;  // grid-stride beyond
  const int eb = bf16_t ? 2 : 4;
  const bool vec = cols % 32 == 0 && (reinterpret_cast<uintptr_t>(x) & 15) == 0 && (ldx * eb) % 16 == 0;
  if (bf16_t) {
    if (vec)
      hipLaunchKernelGGL((relu_mask_kernel<bf16, true>), (unsigned)blocks, kThreads, 0, s, (const bf16*)x, ldx, mask,
                         ldm, rows, cols);
    else
      hipLaunchKernelGGL((relu_mask_kernel<bf16, false>), (unsigned)blocks, kThreads, 0, s, (const bf16*)x, ldx, mask,
                         ldm, rows, cols);
  } else {
    if (vec)
      hipLaunchKernelGGL((relu_mask_kernel<float, true>), (unsigned)blocks, kThreads, 0, s, (const float*)x, ldx,
                         mask, ldm, rows, cols);
    else
      hipLaunchKernelGGL((relu_mask_kernel<float, false>), (unsigned)blocks, kThreads, 0, s, (const float*)x, ldx,
                         mask, ldm, rows, cols);
  }
  return hipGetLastError();
}

// Scratch of the entry point that allocates nothing
// (tfd_relu_grad_bias_add_grad_noalloc): the column partials of pass 1 live in
// this file-scope device array instead of a caller's workspace. Each GPU the
// library runs on holds its own copy until the process ends. In host code the
// array's name is not a device address: its address on a device comes from
// hipGetSymbolAddress, looked up once per device with that device current,
// and only that address is passed to kernels.
constexpr size_t kStaticScratchBytes = size_t(4) << 20;
static __device__ __align__(256) float scratch[kStaticScratchBytes / sizeof(float)];

size_t static_scratch_bytes() { return kStaticScratchBytes; }

hipError_t static_scratch(void** out) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  *out = nullptr;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    addr[dev] = p;
  }
  *out = addr[dev];
  return hipSuccess;
}

}  // namespace tfd
