// One training step of a small fp32 multilayer perceptron in one persistent
// kernel: the forward pass (MatMul, BiasAdd, Relu of section 2, Table 1), the
// cost head (squared error or softmax cross-entropy), the gradient subgraph of
// section 4.1 (ReluGrad, the two transposed MatMuls, BiasAddGrad) and the SGD
// update of the Variables. Meant for the MNIST-shaped steps (a few hundred
// rows, layers of a few thousand units at most), whose dozen-odd kernels each
// fill only part of the chip and spend most of the step in launch gaps.
//
// The step runs as a sequence of phases separated by grid-wide barriers; in
// each phase every workgroup takes work items (32 x 32 output tiles of a
// MatMul, column chunks of a BiasAddGrad, chunks of the cost head or of an
// update) round-robin. Phases, for L layers:
//   F_0 .. F_{L-1}  H_{l+1} = Relu(H_l W_l + b_l) (identity where the layer has
//                   no Relu); an output layer with few tiles over a long k is
//                   split into k chunks whose partial products the cost phase
//                   adds (with the bias and the Relu);
//   cost            G, the loss partials, and dY of the output layer
//                   (ReluGrad of G when that layer has a Relu);
//   B_{L-1} .. B_0  dW_l = H_l^T dY_l (64 x 64 tiles; 32 x 32 ones with the
//                   batch split over the waves for a narrow layer), db_l =
//                   column sums of dY_l, and
//                   dY_{l-1} = ReluGrad(dY_l W_l^T, H_l) (the input gradient
//                   dX_0 = dY_0 W_0^T for l = 0, when asked for); the update
//                   of layer l + 1, whose weights B_{l+1} was the last to read;
//                   in B_{L-1} the loss, summed from the cost phase's partials;
//   update          layer 0.
// A MatMul tile is the k loop of gemm_small_tile.h on 4 waves, each summing a
// quarter of k; the partial tiles are added in wave order, so the step is
// bitwise reproducible, as are the column sums (rows in order) and the loss
// (partials in order).
//
// The barrier: a workgroup's first thread makes its stores visible at device
// scope (fence), counts its arrival and waits until the last arrival resets
// the counters and advances a generation word; the wait spins a bounded
// number of times, so every wave exits even if the grid were not all resident
// (the launch is cooperative, which rules that out), and a timed-out wait sets
// the error word and ends the workgroup's step.

#include "common.h"
#include "gemm_small_tile.h"
#include "kernels.h"

namespace tfd {

namespace {

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;  // one 32 x 32 tile, k split 4 ways
constexpr uint32_t kSpinLimit = 1u << 22;
constexpr int kSgdChunk = 4096;   // elements per update item
constexpr int kCostChunk = 256;   // elements per squared-error item (one per thread)
constexpr int kXentRows = kWaves;  // rows per cross-entropy item (one per wave)
constexpr int kColsumCols = 32;   // columns per bias-gradient item

struct Layer {
  float* w;
  float* b;
  float* h;   // output activations [batch, fan_out]
  float* dy;  // dY [batch, fan_out] (Relu layers)
  float* dw;
  float* db;
  int fan_in, fan_out, relu;
};

struct StepArgs {
  Layer l[kMlpMaxLayers];
  int layers, batch, cost, update;
  int only_phase;  // >= 0: run this phase alone (one launch per phase, no barrier)
  float lr;
  const float* x;
  float* dx0;
  float* g;
  const float* target;
  const int32_t* labels;
  double* loss;
  uint32_t* ctl;  // barrier words (the persistent launch)
  double* part;   // cost phase's loss partials
  float* split_part;  // output layer's partial products [split][batch][classes]
  int split;
};

// ---------------------------------------------------------------- work counts
// (shared with the host, which sizes the grid and the workspace from them)

__host__ __device__ inline int tiles32(int m, int n) { return ((m + 31) / 32) * ((n + 31) / 32); }
__host__ __device__ inline int tiles64(int m, int n) { return ((m + 63) / 64) * ((n + 63) / 64); }

// The output layer's forward MatMul over k chunks when its output has few
// tiles (a narrow classifier layer over a long k): the chunks' partial
// products go to the workspace and the cost phase adds them, the bias and the
// Relu before the cost head. Returns the number of chunks (1: no split).
__host__ __device__ inline int top_split(int batch, int fan_in, int fan_out) {
  if (tiles32(batch, fan_out) >= 64) return 1;
  const int s = fan_in / 128;
  return s < 1 ? 1 : (s > 8 ? 8 : s);
}
// The weight gradient's tiles: 64 x 64 (one wave per 32 x 32 quadrant, each
// over the whole batch) when there are enough of them to fill the chip,
// else 32 x 32 with the batch split over the waves, so that a narrow layer's
// few tiles do not each run one long chain of loads (the 1024 x 10 gradient
// of a 10-class output layer: 16 tiles of 64 x 64, 32 of 32 x 32).
__host__ __device__ inline bool dw_small_tiles(int fan_in, int fan_out) { return tiles64(fan_in, fan_out) < 64; }
__host__ __device__ inline int dw_tiles(int fan_in, int fan_out) {
  return dw_small_tiles(fan_in, fan_out) ? tiles32(fan_in, fan_out) : tiles64(fan_in, fan_out);
}
// k values per chunk: a multiple of 8, so that every chunk starts on a
// 16-byte boundary of a k-contiguous row
__host__ __device__ inline int split_chunk(int fan_in, int split) { return (((fan_in + split - 1) / split + 7) / 8) * 8; }
__host__ __device__ inline int chunks(int64_t count, int chunk) { return (int)((count + chunk - 1) / chunk); }

__host__ __device__ inline int cost_items(int batch, int classes, int cost) {
  return cost == 0 ? chunks((int64_t)batch * classes, kCostChunk) : chunks(batch, kXentRows);
}

__host__ __device__ inline int update_items(int fan_in, int fan_out) {
  return chunks((int64_t)fan_in * fan_out, kSgdChunk) + chunks(fan_out, kSgdChunk);
}

// phases: F_0..F_{L-1}, cost, B_{L-1}..B_0, then (with the update) layer 0's update
__host__ __device__ inline int num_phases(int layers, int update) { return 2 * layers + 1 + (update ? 1 : 0); }

template <typename FI, typename FO>
__host__ __device__ inline int phase_items(FI fan_in, FO fan_out, int layers, int batch, int cost, int update,
                                           bool dx0, int ph) {
  const int L = layers;
  if (ph < L - 1) return tiles32(batch, fan_out(ph));
  if (ph == L - 1) return tiles32(batch, fan_out(ph)) * top_split(batch, fan_in(ph), fan_out(ph));
  if (ph == L) return cost_items(batch, fan_out(L - 1), cost);
  if (ph <= 2 * L) {
    const int l = 2 * L - ph;
    int n = dw_tiles(fan_in(l), fan_out(l)) + chunks(fan_out(l), kColsumCols);
    if (l > 0 || dx0) n += tiles32(batch, fan_in(l));
    if (update && l + 1 < L) n += update_items(fan_in(l + 1), fan_out(l + 1));
    if (l == L - 1) n += 1;
    return n;
  }
  return update_items(fan_in(0), fan_out(0));
}

// ---------------------------------------------------------------- device work

struct Mm {
  const float* a;
  const float* b;
  float* c;
  int64_t lda, ldb, ldc;
  int m, n, k;    // the k range is [kbeg, k)
  int ta, tb;
  int epi;  // 0 plain, 1 bias (+ Relu when relu), 2 ReluGrad against feat
  int relu;
  const float* bias;
  const float* feat;
  int kbeg;
};

__device__ __forceinline__ bool aligned16(const void* p, int64_t ld) {
  return ((reinterpret_cast<uintptr_t>(p) & 15) == 0) && (ld % 4 == 0);
}

template <bool TA, bool TB>
__device__ __forceinline__ void mm_k(const Mm& j, int row, int col, int kb, int ke, int h, f32x16& acc) {
  const bool vec = (TA || aligned16(j.a, j.lda)) && (!TB || aligned16(j.b, j.ldb));
  if (vec)
    small_tile::tile_k<TA, TB, true>(j.a, j.lda, j.b, j.ldb, row, col, kb, ke, h, acc);
  else
    small_tile::tile_k<TA, TB, false>(j.a, j.lda, j.b, j.ldb, row, col, kb, ke, h, acc);
}

// One 32 x 32 tile `t` of job `j` (row-major tiles), with its epilogue: each
// wave sums a 1 / kWaves share of k; the partial tiles are added in wave order.
__device__ void mm_tile(const Mm& j, int t, float* part) {
  const int lane = threadIdx.x & 63, w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int l32 = lane & 31, h = lane >> 5;
  const int tn = (j.n + 31) / 32;
  const int m0 = (t / tn) * 32, n0 = (t % tn) * 32;
  const int row = min(m0 + l32, j.m - 1), col = min(n0 + l32, j.n - 1);
  int kper = (((j.k - j.kbeg + kWaves - 1) / kWaves + 7) / 8) * 8;
  if (kper == 0) kper = 8;
  const int kb = j.kbeg + w * kper, ke = min(j.k, kb + kper);
  f32x16 acc;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = 0.0f;
  if (j.ta)
    mm_k<true, false>(j, row, col, kb, ke, h, acc);
  else if (j.tb)
    mm_k<false, true>(j, row, col, kb, ke, h, acc);
  else
    mm_k<false, false>(j, row, col, kb, ke, h, acc);
  small_tile::store_part(part + w * 1024, acc, h, l32);
  __syncthreads();
  for (int e = threadIdx.x; e < 1024; e += kThreads) {
    const int gr = m0 + (e >> 5), gc = n0 + (e & 31);
    if (gr < j.m && gc < j.n) {
      float v = part[e];
#pragma unroll
      for (int q = 1; q < kWaves; ++q) v += part[q * 1024 + e];
      if (j.epi == 1) {
        v += j.bias[gc];
        if (j.relu) v = relu_f32(v);
      } else if (j.epi == 2) {
        const float f = j.feat[(int64_t)gr * j.n + gc];
        v = __builtin_bit_cast(float, f > 0.0f ? __builtin_bit_cast(uint32_t, v) : 0u);
      }
      j.c[(int64_t)gr * j.ldc + gc] = v;
    }
  }
  __syncthreads();
}

// One 64 x 64 tile `t` of a plain job (row-major tiles): wave q sums k for the
// 32 x 32 quadrant q (q / 2, q % 2) (with 8 waves, waves q and q + 4 the two
// halves of k, the second half's partial added through LDS) and stores
// straight from its accumulators (each register is one row's 32
// consecutive columns across a half-wave). For the weight gradients (k =
// batch, both operands m/n-contiguous): a quarter as many tiles as 32 x 32
// ones, each wave with a longer loop over which its loads overlap.
__device__ void mm_tile64(const Mm& j, int t, float* part) {
  const int lane = threadIdx.x & 63, w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int l32 = lane & 31, h = lane >> 5;
  const int q = w & 3, kh = w >> 2;
  const int tn = (j.n + 63) / 64;
  const int m0 = (t / tn) * 64 + (q >> 1) * 32, n0 = (t % tn) * 64 + (q & 1) * 32;
  const bool live = m0 < j.m && n0 < j.n;
  const int row = min(m0 + l32, j.m - 1), col = min(n0 + l32, j.n - 1);
  // with 8 waves the two halves of k go to waves q and q + 4; with 4, one wave
  // per quadrant takes all of k
  const int kmid = kWaves == 8 ? min(j.k, ((j.k / 2 + 7) / 8) * 8) : j.k;
  const int kb = kh ? kmid : 0, ke = kh ? j.k : kmid;
  f32x16 acc;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = 0.0f;
  if (live) {
    if (j.ta)
      mm_k<true, false>(j, row, col, kb, ke, h, acc);
    else if (j.tb)
      mm_k<false, true>(j, row, col, kb, ke, h, acc);
    else
      mm_k<false, false>(j, row, col, kb, ke, h, acc);
  }
  if (kWaves == 8 && kh) small_tile::store_part(part + q * 1024, acc, h, l32);
  __syncthreads();
  if (!kh && live) {
    const int gc = n0 + l32;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int er = 8 * (r >> 2) + 4 * h + (r & 3);
      const int gr = m0 + er;
      if (gr < j.m && gc < j.n) j.c[(int64_t)gr * j.ldc + gc] = kWaves == 8 ? acc[r] + part[q * 1024 + er * 32 + l32] : acc[r];
    }
  }
  __syncthreads();
}

__device__ __forceinline__ float relu_grad(float g, float f) {
  return __builtin_bit_cast(float, f > 0.0f ? __builtin_bit_cast(uint32_t, g) : 0u);
}

// Column sums of x [rows, cols] for the kColsumCols columns of `item`: thread
// (c, g) sums rows g * span .. of column c (span = ceil(rows / groups)), in
// order; the partials of a column are then added in g order.
__device__ void colsum_item(const float* x, float* out, int rows, int cols, int item, float* part) {
  constexpr int kGroupsR = kThreads / kColsumCols;
  const int c = item * kColsumCols + (threadIdx.x % kColsumCols), g = threadIdx.x / kColsumCols;
  const int span = (rows + kGroupsR - 1) / kGroupsR;
  const int r0 = g * span, r1 = min(rows, r0 + span);
  float s = 0.0f;
  if (c < cols)
    for (int r = r0; r < r1; ++r) s += x[(int64_t)r * cols + c];
  part[threadIdx.x] = s;
  __syncthreads();
  if (threadIdx.x < kColsumCols && c < cols) {
    float t = part[threadIdx.x];
#pragma unroll
    for (int q = 1; q < kGroupsR; ++q) t += part[q * kColsumCols + threadIdx.x];
    out[c] = t;
  }
  __syncthreads();
}

// var[i] <- fma(-lr, delta[i], var[i]) for i in chunk `item` of kSgdChunk:
// 16-byte accesses where both arrays are 16-byte aligned.
__device__ void sgd_item(float* var, const float* delta, int64_t count, float lr, int item) {
  const int64_t i0 = (int64_t)item * kSgdChunk;
  const int64_t i1 = min(count, i0 + kSgdChunk);
  const float na = -lr;
  const bool vec = ((reinterpret_cast<uintptr_t>(var) | reinterpret_cast<uintptr_t>(delta)) & 15) == 0;
  int64_t i = i0;
  if (vec) {
    for (int64_t q = i0 + 4 * threadIdx.x; q + 4 <= i1; q += 4 * kThreads) {
      f32x4 v = *reinterpret_cast<const f32x4*>(var + q);
      const f32x4 d = *reinterpret_cast<const f32x4*>(delta + q);
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = __builtin_fmaf(na, d[e], v[e]);
      *reinterpret_cast<f32x4*>(var + q) = v;
    }
    i = i0 + ((i1 - i0) / 4) * 4;
  }
  for (int64_t k = i + threadIdx.x; k < i1; k += kThreads) var[k] = __builtin_fmaf(na, delta[k], var[k]);
}

// Sum of one double per thread in a fixed order (thread 0 gets the result):
// kSumRuns runs of consecutive threads, each summed in thread order, then the
// run sums in order. red holds kThreads + kSumRuns doubles.
constexpr int kSumRuns = 16;
__device__ double block_sum_ordered(double v, double* red) {
  constexpr int kRun = kThreads / kSumRuns;
  red[threadIdx.x] = v;
  __syncthreads();
  if (threadIdx.x < kSumRuns) {
    double s = 0.0;
#pragma unroll
    for (int i = 0; i < kRun; ++i) s += red[threadIdx.x * kRun + i];
    red[kThreads + threadIdx.x] = s;
  }
  __syncthreads();
  double acc = 0.0;
  if (threadIdx.x == 0)
#pragma unroll
    for (int i = 0; i < kSumRuns; ++i) acc += red[kThreads + i];
  __syncthreads();
  return acc;
}

// Element i of the output layer's activations: with a split forward MatMul,
// the chunks' partial products added in chunk order, then the bias and the
// Relu, stored; otherwise as the forward phase stored it.
__device__ __forceinline__ float top_value(const StepArgs& a, int64_t i) {
  const Layer& top = a.l[a.layers - 1];
  if (a.split <= 1) return top.h[i];
  const int64_t count = (int64_t)a.batch * top.fan_out;
  float v = a.split_part[i];
  for (int c = 1; c < a.split; ++c) v += a.split_part[c * count + i];
  v += top.b[i % top.fan_out];
  if (top.relu) v = relu_f32(v);
  top.h[i] = v;
  return v;
}

// Squared error over elements [item * kCostChunk, +kCostChunk) of the output:
// G = out - target (or out), dY = ReluGrad(G, out) for a Relu output layer,
// and the item's float64 sum of the exact squared differences.
__device__ void sq_item(const StepArgs& a, int item, double* red) {
  const Layer& top = a.l[a.layers - 1];
  const int64_t count = (int64_t)a.batch * top.fan_out;
  const int64_t i0 = (int64_t)item * kCostChunk;
  double s = 0.0;
  for (int64_t i = i0 + threadIdx.x; i < min(count, i0 + kCostChunk); i += kThreads) {
    const float o = top_value(a, i);
    const float t = a.target ? a.target[i] : 0.0f;
    const float d = o - t;
    a.g[i] = d;
    if (top.relu) top.dy[i] = relu_grad(d, o);
    const double e = (double)o - (double)t;
    s += e * e;
  }
  const double tot = block_sum_ordered(s, red);
  if (threadIdx.x == 0) a.part[item] = tot;
}

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

// Softmax cross-entropy of rows item * 4 + wave (one wave per row, lanes
// striding over the classes): G = softmax(z) - onehot(y), the row's term
// log sum exp(z) - z_y; the item's sum of terms in row order.
__device__ void xent_item(const StepArgs& a, int item, double* red) {
  const Layer& top = a.l[a.layers - 1];
  const int cols = top.fan_out;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int64_t row = (int64_t)item * kXentRows + wv;
  double term = 0.0;
  if (row < a.batch) {
    const float* zr = top.h + row * cols;
    float* gr = a.g + row * cols;
    float m = -INFINITY;
    for (int c = lane; c < cols; c += kWave) m = fmaxf(m, top_value(a, row * cols + c));
    m = wave_max(m);
    float s = 0.0f;
    for (int c = lane; c < cols; c += kWave) s += expf(zr[c] - m);
    s = wave_sum(s);
    const float inv = 1.0f / s;
    const int32_t y = a.labels[row];
    for (int c = lane; c < cols; c += kWave) {
      float p = expf(zr[c] - m) * inv;
      if (c == y) p -= 1.0f;
      gr[c] = p;
      if (top.relu) top.dy[row * cols + c] = relu_grad(p, zr[c]);
    }
    if (lane == 0)
      term = (y >= 0 && y < cols) ? (double)logf(s) + (double)m - (double)zr[y] : __builtin_nan("");
  }
  const double tot = block_sum_ordered(lane == 0 ? term : 0.0, red);
  if (threadIdx.x == 0) a.part[item] = tot;
}

// Grid barrier (see the file comment). Returns false once a wait timed out.
// Arrivals go through kGroups counters on separate lines (workgroup b counts
// in group b mod kGroups) and the last arrival of each group through one top
// counter, so that no single address takes every workgroup's atomic; waiters
// poll a generation word on a line of its own. The atomics are relaxed and
// device-scope (performed beyond the per-XCD L2s); the ordering comes from a
// release fence before an arrival or a counter reset (stores written back
// from this XCD's L2) and an acquire fence after the wait (stale lines
// dropped). An acquire load inside the spin would drop the whole L2 on every
// poll, under every other workgroup's loads.
constexpr int kGroups = 16;
constexpr int kCtlError = 0, kCtlGen = 64, kCtlTop = 128, kCtlGroup = 256, kCtlGroupStride = 32;  // uint32 words

__device__ __forceinline__ uint32_t ld_relaxed(uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t add_relaxed(uint32_t* p) {
  return __hip_atomic_fetch_add(p, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_relaxed(uint32_t* p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ bool grid_sync(uint32_t* ctl, uint32_t nblocks, int* abort_flag) {
  __syncthreads();
  if (threadIdx.x == 0) {
    int ok = 1;
    const uint32_t g = blockIdx.x % kGroups;
    const uint32_t ngroups = nblocks < (uint32_t)kGroups ? nblocks : (uint32_t)kGroups;
    const uint32_t gsize = (nblocks - 1 - g) / kGroups + 1;
    uint32_t* const gen_w = ctl + kCtlGen;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    const uint32_t gen = ld_relaxed(gen_w);
    bool wait = true;
    if (add_relaxed(ctl + kCtlGroup + g * kCtlGroupStride) == gsize - 1) {
      // last of its group: reset the group counter, then arrive at the top
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
      st_relaxed(ctl + kCtlGroup + g * kCtlGroupStride, 0u);
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
      if (add_relaxed(ctl + kCtlTop) == ngroups - 1) {
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        st_relaxed(ctl + kCtlTop, 0u);
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
        add_relaxed(gen_w);
        wait = false;
      }
    }
    if (wait) {
      uint32_t spins = 0;
      while (ld_relaxed(gen_w) == gen) {
        __builtin_amdgcn_s_sleep(1);
        if (++spins == kSpinLimit) {
          ok = 0;
          st_relaxed(ctl + kCtlError, 1u);
          break;
        }
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    *abort_flag = !ok;
  }
  __syncthreads();
  return *abort_flag == 0;
}

__device__ __forceinline__ const float* act_in(const StepArgs& a, int l) { return l == 0 ? a.x : a.l[l - 1].h; }
__device__ __forceinline__ const float* dy_of(const StepArgs& a, int l) {
  return (l == a.layers - 1 && !a.l[l].relu) ? a.g : a.l[l].dy;
}

__global__ __launch_bounds__(kThreads) void mlp_step_kernel(StepArgs a) {
  __shared__ float part[kWaves * 1024];
  __shared__ double red[kThreads + kSumRuns];
  __shared__ int abort_flag;
  const int L = a.layers;
  auto fan_in = [&](int l) { return a.l[l].fan_in; };
  auto fan_out = [&](int l) { return a.l[l].fan_out; };
  const int nph = a.only_phase >= 0 ? a.only_phase + 1 : num_phases(L, a.update);
  for (int ph = a.only_phase >= 0 ? a.only_phase : 0; ph < nph; ++ph) {
    if (a.only_phase < 0 && ph > 0 && !grid_sync(a.ctl, gridDim.x, &abort_flag)) return;
    const int items = phase_items(fan_in, fan_out, L, a.batch, a.cost, a.update, a.dx0 != nullptr, ph);
    for (int it = blockIdx.x; it < items; it += gridDim.x) {
      if (ph < L) {  // forward of layer ph
        const Layer& ly = a.l[ph];
        if (ph == L - 1 && a.split > 1) {  // k chunk it / tiles of the output layer: partial product
          const int tiles = tiles32(a.batch, ly.fan_out), c = it / tiles;
          const int kc = split_chunk(ly.fan_in, a.split);
          Mm j{act_in(a, ph), ly.w, a.split_part + (int64_t)c * a.batch * ly.fan_out, ly.fan_in, ly.fan_out,
               ly.fan_out, a.batch, ly.fan_out, min(ly.fan_in, (c + 1) * kc), 0, 0, 0, 0, nullptr, nullptr, c * kc};
          mm_tile(j, it - c * tiles, part);
          continue;
        }
        Mm j{act_in(a, ph), ly.w, ly.h, ly.fan_in, ly.fan_out, ly.fan_out, a.batch, ly.fan_out, ly.fan_in, 0, 0, 1,
             ly.relu, ly.b, nullptr, 0};
        mm_tile(j, it, part);
      } else if (ph == L) {
        if (a.cost == 0)
          sq_item(a, it, red);
        else
          xent_item(a, it, red);
      } else if (ph <= 2 * L) {
        const int l = 2 * L - ph;
        const Layer& ly = a.l[l];
        const float* dy = dy_of(a, l);
        int r = it;
        // longest items first: the input-gradient tiles sum over fan_out, the
        // weight-gradient tiles over the batch
        const bool want_dx = l > 0 || a.dx0 != nullptr;
        const int n_dx = want_dx ? tiles32(a.batch, ly.fan_in) : 0;
        if (r < n_dx) {  // dY_{l-1} = ReluGrad(dY_l W_l^T, H_l), or dX_0
          float* out = l > 0 ? a.l[l - 1].dy : a.dx0;
          Mm j{dy, ly.w, out, ly.fan_out, ly.fan_out, ly.fan_in, a.batch, ly.fan_in, ly.fan_out, 0, 1,
               l > 0 ? 2 : 0, 0, nullptr, l > 0 ? a.l[l - 1].h : nullptr, 0};
          mm_tile(j, r, part);
          continue;
        }
        r -= n_dx;
        const int n_dw = dw_tiles(ly.fan_in, ly.fan_out);
        if (r < n_dw) {  // dW_l = H_l^T dY_l
          Mm j{act_in(a, l), dy, ly.dw, ly.fan_in, ly.fan_out, ly.fan_out, ly.fan_in, ly.fan_out, a.batch, 1, 0, 0,
               0, nullptr, nullptr, 0};
          if (dw_small_tiles(ly.fan_in, ly.fan_out))
            mm_tile(j, r, part);
          else
            mm_tile64(j, r, part);
          continue;
        }
        r -= n_dw;
        const int n_db = chunks(ly.fan_out, kColsumCols);
        if (r < n_db) {
          colsum_item(dy, ly.db, a.batch, ly.fan_out, r, part);
          continue;
        }
        r -= n_db;
        if (a.update && l + 1 < L) {
          const Layer& up = a.l[l + 1];
          const int n_w = chunks((int64_t)up.fan_in * up.fan_out, kSgdChunk);
          if (r < n_w) {
            sgd_item(up.w, up.dw, (int64_t)up.fan_in * up.fan_out, a.lr, r);
            continue;
          }
          r -= n_w;
          const int n_b = chunks(up.fan_out, kSgdChunk);
          if (r < n_b) {
            sgd_item(up.b, up.db, up.fan_out, a.lr, r);
            continue;
          }
          r -= n_b;
        }
        // the loss, from the cost phase's partials in order
        if (threadIdx.x == 0) {
          const int np = cost_items(a.batch, a.l[L - 1].fan_out, a.cost);
          double acc = 0.0;
          for (int i = 0; i < np; ++i) acc += a.part[i];
          *a.loss = a.cost == 0 ? 0.5 * acc : acc;
        }
      } else {  // update of layer 0
        const Layer& ly = a.l[0];
        const int n_w = chunks((int64_t)ly.fan_in * ly.fan_out, kSgdChunk);
        if (it < n_w)
          sgd_item(ly.w, ly.dw, (int64_t)ly.fan_in * ly.fan_out, a.lr, it);
        else
          sgd_item(ly.b, ly.db, ly.fan_out, a.lr, it - n_w);
      }
    }
  }
}

int cu_count() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  if (cached[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
    cached[dev] = n;
  }
  return cached[dev];
}

}  // namespace

// [barrier words][loss partials][output layer's split partial products]
static size_t split_offset(int64_t batch, int64_t classes, int cost) {
  const size_t b = kMlpCtlBytes + sizeof(double) * (size_t)cost_items((int)batch, (int)classes, cost);
  return (b + 255) & ~size_t(255);
}

size_t mlp_step_ws_bytes(int64_t batch, int64_t top_fan_in, int64_t classes, int cost) {
  const int split = top_split((int)batch, (int)top_fan_in, (int)classes);
  return split_offset(batch, classes, cost) + (split > 1 ? sizeof(float) * (size_t)split * batch * classes : 0);
}

hipError_t launch_mlp_step(const MlpStep& d, void* ws, hipStream_t s) {
  StepArgs a{};
  int fan_in[kMlpMaxLayers] = {0}, fan_out[kMlpMaxLayers] = {0};
  for (int l = 0; l < d.layers; ++l) {
    a.l[l] = Layer{d.w[l], d.b[l], d.h[l], d.dy[l], d.dw[l], d.db[l], (int)d.fan_in[l], (int)d.fan_out[l], d.relu[l]};
    fan_in[l] = (int)d.fan_in[l];
    fan_out[l] = (int)d.fan_out[l];
  }
  a.layers = d.layers;
  a.batch = (int)d.batch;
  a.cost = d.cost;
  a.update = d.update;
  a.lr = d.lr;
  a.x = d.x;
  a.dx0 = d.dx0;
  a.g = d.g;
  a.target = d.target;
  a.labels = d.labels;
  a.loss = d.loss;
  a.ctl = static_cast<uint32_t*>(ws);
  a.part = reinterpret_cast<double*>(static_cast<char*>(ws) + kMlpCtlBytes);
  const int top = d.layers - 1;
  a.split = top_split(a.batch, fan_in[top], fan_out[top]);
  a.split_part = reinterpret_cast<float*>(static_cast<char*>(ws) + split_offset(d.batch, d.fan_out[top], d.cost));
  auto fi = [&](int l) { return fan_in[l]; };
  auto fo = [&](int l) { return fan_out[l]; };
  const int nph = num_phases(d.layers, d.update);
  if (!d.persistent) {
    // one launch per phase: stream order separates the phases, and each
    // launch has a workgroup per item
    for (int ph = 0; ph < nph; ++ph) {
      a.only_phase = ph;
      const int items = phase_items(fi, fo, d.layers, a.batch, d.cost, d.update, d.dx0 != nullptr, ph);
      hipLaunchKernelGGL(mlp_step_kernel, dim3((unsigned)max(items, 1)), dim3(kThreads), 0, s, a);
      const hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
    return hipSuccess;
  }
  a.only_phase = -1;
  int most = 1;
  for (int ph = 0; ph < nph; ++ph)
    most = max(most, phase_items(fi, fo, d.layers, a.batch, d.cost, d.update, d.dx0 != nullptr, ph));
  const int cus = cu_count();
  if (cus <= 0) return hipErrorInvalidDevice;
  // up to two workgroups per compute unit (a workgroup's tiles are
  // latency-bound chains of loads, which the other's overlap), as many as fit
  int per_cu = 0;
  const hipError_t oe = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, mlp_step_kernel, kThreads, 0);
  if (oe != hipSuccess) return oe;
  if (per_cu < 1) return hipErrorLaunchOutOfResources;
  const unsigned grid = (unsigned)min(most, min(per_cu, 2) * cus);
  void* args[] = {&a};
  return hipLaunchCooperativeKernel(reinterpret_cast<const void*>(mlp_step_kernel), dim3(grid), dim3(kThreads), args,
                                    0, s);
}

}  // namespace tfd
