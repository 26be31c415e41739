// MatMul for small fp32 problems (the MNIST-shaped layers: a few hundred rows,
// outputs as narrow as 10 columns), where 64x64 or larger tiles leave most of
// the 256 compute units idle and a long k loop per tile sets the time.
//
// One workgroup per 32x32 output tile, W waves per workgroup, each wave
// summing a contiguous slice of k (the k loop of gemm_small_tile.h). The W
// partial tiles meet in LDS and are added in wave order (a fixed order:
// results are bitwise reproducible), then the epilogue adds the bias, applies
// the ReLU and stores.

#include <stdlib.h>

#include "common.h"
#include "gemm_small_tile.h"
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

// Few waves per SIMD are resident (one workgroup of W waves per tile): the
// occupancy hint lets the scheduler keep a whole group of loads in flight
// instead of moving each load next to its MFMA to save registers.
template <bool TA, bool TB, int W, bool VEC>
__global__ __launch_bounds__(64 * W) __attribute__((amdgpu_waves_per_eu(1, 4))) void gemm_small_f32(SmallParams p) {
  __shared__ float part[W * 1024];
  // the wave index is uniform across the wave: keep it (and the k slice
  // bounds derived from it) in scalar registers so the loop is scalar
  const int lane = threadIdx.x & 63, w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int l32 = lane & 31, h = lane >> 5;
  const int m0 = (blockIdx.x / p.tiles_n) * 32, n0 = (blockIdx.x % p.tiles_n) * 32;
  const int row = min(m0 + l32, p.m - 1), col = min(n0 + l32, p.n - 1);
  const int kb = w * p.kper;
  const int ke = min(p.k, kb + p.kper);

  f32x16 acc;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = 0.0f;

  small_tile::tile_k<TA, TB, VEC>(p.a, p.lda, p.b, p.ldb, row, col, kb, ke, h, acc);

  small_tile::store_part(part + w * 1024, acc, h, l32);
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

// Small problems: fewer than 128 output tiles of 128 x 128, except weight
// gradients (transpose_a) with 512 or more 32 x 32 tiles, where the LDS-staged
// 64 x 64 tiles of gemm.hip were measured faster.
bool gemm_small_preferred(const GemmDesc& d) {
  const int64_t tiles128 = ((d.m + 127) / 128) * ((d.n + 127) / 128);
  const int64_t tiles32 = ((d.m + 31) / 32) * ((d.n + 31) / 32);
  return !d.in_bf16 && !d.out_bf16 && tiles128 < 128 && !(d.ta && tiles32 >= 512);
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
  // 4 waves per tile: measured fastest for every MNIST-shaped problem, also
  // those with only a few tiles (8 or 16 waves per tile were slower)
  int waves = 4;
  if (const int v = tuning(kTuneSmallWaves)) waves = v;  // tuning knob: 4, 8 or 16
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
