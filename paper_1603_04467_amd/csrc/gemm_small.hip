// MatMul for small fp32 problems (the MNIST-shaped layers: a few hundred rows,
// outputs as narrow as 10 columns), where 64x64 or larger tiles leave most of
// the 256 compute units idle and a long k loop per tile sets the time.
//
// One workgroup per 32x32 output tile, W waves per workgroup, each wave
// summing a contiguous slice of k with v_mfma_f32_32x32x2_f32 straight from
// registers (no LDS staging: every operand element is used by one MFMA of one
// wave, and the small operands stay in L2). Per 8 values of k a lane loads 4
// consecutive k of its row of A and of its column of B: 16-byte loads for a
// k-contiguous operand, 4 coalesced loads for an m/n-contiguous one. The four
// instructions of a chunk take k + j (lanes 0-31) and k + 4 + j (lanes 32-63),
// j = 0..3, for A and B alike, so each k is summed exactly once.
//
// The W partial tiles meet in LDS and are added in wave order (a fixed order:
// results are bitwise reproducible), then the epilogue adds the bias, applies
// the ReLU and stores. Rows, columns and k beyond the problem are guarded
// (zeros are summed instead), so any shape and leading dimension works.

#include "common.h"
#include "kernels.h"

namespace tfd {

namespace {

struct SmallParams {
  const float* a;
  const float* b;
  float* c;
  const float* bias;
  int64_t lda, ldb, ldc;
  int m, n, k;
  int epi;
  int tiles_n;
  int kper;  // k values per wave, a multiple of 8
};

// Four consecutive k (kk .. kk+3, clipped at ke) of row r of a k-contiguous
// operand X (X[r * ld + k]).
template <bool VEC>
__device__ __forceinline__ f32x4 load_kc(const float* __restrict__ x, int64_t ld, int r, bool r_ok, int kk, int ke) {
  f32x4 v = {0.0f, 0.0f, 0.0f, 0.0f};
  if (!r_ok) return v;
  const float* p = x + (int64_t)r * ld + kk;
  if (VEC && kk + 4 <= ke) return *reinterpret_cast<const f32x4*>(p);
#pragma unroll
  for (int j = 0; j < 4; ++j)
    if (kk + j < ke) v[j] = p[j];
  return v;
}

// Four consecutive k of column c of an m/n-contiguous operand X (X[k * ld + c]).
__device__ __forceinline__ f32x4 load_mn(const float* __restrict__ x, int64_t ld, int c, bool c_ok, int kk, int ke) {
  f32x4 v = {0.0f, 0.0f, 0.0f, 0.0f};
  if (!c_ok) return v;
#pragma unroll
  for (int j = 0; j < 4; ++j)
    if (kk + j < ke) v[j] = x[(int64_t)(kk + j) * ld + c];
  return v;
}

template <bool TA, bool TB, bool VEC>
__device__ __forceinline__ void load_chunk(const SmallParams& p, int row, bool row_ok, int col, bool col_ok, int kk,
                                           int ke, f32x4& a, f32x4& b) {
  a = TA ? load_mn(p.a, p.lda, row, row_ok, kk, ke) : load_kc<VEC>(p.a, p.lda, row, row_ok, kk, ke);
  b = TB ? load_kc<VEC>(p.b, p.ldb, col, col_ok, kk, ke) : load_mn(p.b, p.ldb, col, col_ok, kk, ke);
}

__device__ __forceinline__ void mfma4(f32x16& acc, const f32x4& a, const f32x4& b) {
#pragma unroll
  for (int j = 0; j < 4; ++j) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a[j], b[j], acc, 0, 0, 0);
}

template <bool TA, bool TB, int W, bool VEC>
__global__ __launch_bounds__(64 * W) void gemm_small_f32(SmallParams p) {
  __shared__ float part[W * 1024];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int l32 = lane & 31, h = lane >> 5;
  const int m0 = (blockIdx.x / p.tiles_n) * 32, n0 = (blockIdx.x % p.tiles_n) * 32;
  const int row = m0 + l32, col = n0 + l32;
  const bool row_ok = row < p.m, col_ok = col < p.n;
  const int kb = w * p.kper;
  const int ke = min(p.k, kb + p.kper);

  f32x16 acc;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = 0.0f;

  int k0 = kb;
  // four chunks (32 k) per iteration: all loads first, then 16 MFMAs
  for (; k0 + 32 <= ke; k0 += 32) {
    f32x4 a[4], b[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) load_chunk<TA, TB, VEC>(p, row, row_ok, col, col_ok, k0 + 8 * c + 4 * h, ke, a[c], b[c]);
#pragma unroll
    for (int c = 0; c < 4; ++c) mfma4(acc, a[c], b[c]);
  }
  for (; k0 < ke; k0 += 8) {
    f32x4 a, b;
    load_chunk<TA, TB, VEC>(p, row, row_ok, col, col_ok, k0 + 4 * h, ke, a, b);
    mfma4(acc, a, b);
  }

#pragma unroll
  for (int r = 0; r < 16; ++r) part[w * 1024 + (8 * (r >> 2) + 4 * h + (r & 3)) * 32 + l32] = acc[r];
  __syncthreads();

  const int op = p.epi & kEpiOpMask;
  for (int e = threadIdx.x; e < 1024; e += 64 * W) {
    const int gr = m0 + (e >> 5), gc = n0 + (e & 31);
    if (gr < p.m && gc < p.n) {
      float v = 0.0f;
#pragma unroll
      for (int q = 0; q < W; ++q) v += part[q * 1024 + e];
      if (op != 0) v += p.bias[gc];
      if (op == 2) v = relu_f32(v);
      p.c[(int64_t)gr * p.ldc + gc] = v;
    }
  }
}

template <bool TA, bool TB, int W>
hipError_t launch_w(const SmallParams& p, bool vec, unsigned grid, hipStream_t s) {
  if (vec)
    hipLaunchKernelGGL((gemm_small_f32<TA, TB, W, true>), grid, 64 * W, 0, s, p);
  else
    hipLaunchKernelGGL((gemm_small_f32<TA, TB, W, false>), grid, 64 * W, 0, s, p);
  return hipGetLastError();
}

template <bool TA, bool TB>
hipError_t launch_layout(const SmallParams& p, int waves, bool vec, unsigned grid, hipStream_t s) {
  if (waves == 16) return launch_w<TA, TB, 16>(p, vec, grid, s);
  if (waves == 8) return launch_w<TA, TB, 8>(p, vec, grid, s);
  return launch_w<TA, TB, 4>(p, vec, grid, s);
}

}  // namespace

// Small problems: fewer than 128 output tiles of 128 x 128.
bool gemm_small_preferred(const GemmDesc& d) {
  const int64_t tiles128 = ((d.m + 127) / 128) * ((d.n + 127) / 128);
  return !d.in_bf16 && !d.out_bf16 && tiles128 < 128;
}

hipError_t launch_gemm_small_f32(const GemmDesc& d, hipStream_t s) {
  SmallParams p;
  p.a = static_cast<const float*>(d.a);
  p.b = static_cast<const float*>(d.b);
  p.c = static_cast<float*>(d.c);
  p.bias = d.bias;
  p.lda = d.lda;
  p.ldb = d.ldb;
  p.ldc = d.ldc;
  p.m = (int)d.m;
  p.n = (int)d.n;
  p.k = (int)d.k;
  p.epi = d.epi;
  const int64_t tiles_m = (d.m + 31) / 32, tiles_n = (d.n + 31) / 32;
  p.tiles_n = (int)tiles_n;
  const int64_t tiles = tiles_m * tiles_n;
  // about 2048 waves in flight (8 per compute unit), 4 to 16 per tile, but no
  // more waves than 32-wide slices of k
  int waves = 4;
  while (waves < 16 && tiles * waves < 2048 && (int64_t)waves * 32 < d.k) waves *= 2;
  const int64_t per = (d.k + waves - 1) / waves;
  p.kper = (int)(((per + 7) / 8) * 8);
  if (p.kper == 0) p.kper = 8;
  // 16-byte loads of the k-contiguous operands need 16-byte aligned rows
  auto al = [](const void* q) { return (reinterpret_cast<uintptr_t>(q) & 15) == 0; };
  const bool a_kc = !d.ta, b_kc = d.tb;
  const bool vec = (!a_kc || (al(d.a) && d.lda % 4 == 0)) && (!b_kc || (al(d.b) && d.ldb % 4 == 0));
  const unsigned grid = (unsigned)tiles;
  if (!d.ta && !d.tb) return launch_layout<false, false>(p, waves, vec, grid, s);
  if (!d.ta && d.tb) return launch_layout<false, true>(p, waves, vec, grid, s);
  return launch_layout<true, false>(p, waves, vec, grid, s);
}

}  // namespace tfd
