// MatMul for small fp32 problems (the MNIST-shaped layers: a few hundred rows,
// outputs as narrow as 10 columns), where 64x64 or larger tiles leave most of
// the 256 compute units idle and a long k loop per tile sets the time.
//
// One workgroup per 32x32 output tile, W waves per workgroup, each wave
// summing a contiguous slice of k with v_mfma_f32_32x32x2_f32 straight from
// registers, with the next 32 k of operands loaded while the current 32 are
// multiplied (no LDS staging: every operand element is used by one MFMA of one
// wave, and the small operands stay in L2). Per 8 values of k a lane loads 4
// consecutive k of its row of A and of its column of B: 16-byte loads for a
// k-contiguous operand, 4 coalesced loads for an m/n-contiguous one. The four
// instructions of a chunk take k + j (lanes 0-31) and k + 4 + j (lanes 32-63),
// j = 0..3, for A and B alike, so each k is summed exactly once.
//
// The W partial tiles meet in LDS and are added in wave order (a fixed order:
// results are bitwise reproducible), then the epilogue adds the bias, applies
// the ReLU and stores. Lanes past the last row or column read clamped indices
// (their results are not stored) and k past the end reads zeros, so any
// shape and leading dimension works.

#include <stdlib.h>

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

// Four consecutive k (kk .. kk+3) of row r of a k-contiguous operand X
// (X[r * ld + k]). GUARD: k at or past ke reads element ke - 1 and is
// replaced by zero (branch-free selects; only the last group of a wave's
// slice needs it).
template <bool VEC, bool GUARD>
__device__ __forceinline__ f32x4 load_kc(const float* __restrict__ x, int64_t ld, int r, int kk, int ke) {
  const float* p = x + (int64_t)r * ld;
  f32x4 v;
  if (!GUARD && VEC) return *reinterpret_cast<const f32x4*>(p + kk);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    if (GUARD) {
      const float t = p[min(kk + j, ke - 1)];
      v[j] = kk + j < ke ? t : 0.0f;
    } else {
      v[j] = p[kk + j];
    }
  }
  return v;
}

// Four consecutive k of column c of an m/n-contiguous operand X (X[k * ld + c]).
template <bool GUARD>
__device__ __forceinline__ f32x4 load_mn(const float* __restrict__ x, int64_t ld, int c, int kk, int ke) {
  f32x4 v;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    if (GUARD) {
      const float t = x[(int64_t)min(kk + j, ke - 1) * ld + c];
      v[j] = kk + j < ke ? t : 0.0f;
    } else {
      v[j] = x[(int64_t)(kk + j) * ld + c];
    }
  }
  return v;
}

// Row and column indices are clamped into the problem by the caller: a lane
// past the last row or column computes a copy of an edge value that is never
// stored, so no load needs a row or column guard.
template <bool TA, bool TB, bool VEC, bool GUARD>
__device__ __forceinline__ void load_group(const SmallParams& p, int row, int col, int k0, int h, int ke,
                                           f32x4 (&a)[4], f32x4 (&b)[4]) {
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int kk = k0 + 8 * c + 4 * h;
    a[c] = TA ? load_mn<GUARD>(p.a, p.lda, row, kk, ke) : load_kc<VEC, GUARD>(p.a, p.lda, row, kk, ke);
    b[c] = TB ? load_kc<VEC, GUARD>(p.b, p.ldb, col, kk, ke) : load_mn<GUARD>(p.b, p.ldb, col, kk, ke);
  }
}

// Unguarded loads of whole groups through a per-lane pointer that advances
// by 32 k per group: k-contiguous operands step by 32 elements, m/n-contiguous
// ones by 32 rows (the per-element offsets are multiples of the uniform ld).
template <bool KC, bool VEC>
struct GroupReader {
  const float* ptr;
  int64_t ld;
  __device__ __forceinline__ GroupReader(const float* x, int64_t ld_, int rc, int k0, int h) : ld(ld_) {
    ptr = KC ? x + (int64_t)rc * ld_ + k0 + 4 * h : x + (int64_t)(k0 + 4 * h) * ld_ + rc;
  }
  __device__ __forceinline__ void read(f32x4 (&v)[4]) const {
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      if (KC && VEC) {
        v[c] = *reinterpret_cast<const f32x4*>(ptr + 8 * c);
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) v[c][j] = KC ? ptr[8 * c + j] : ptr[(int64_t)(8 * c + j) * ld];
      }
    }
  }
  // to the next group, or stay (the loads are then repeated, harmlessly):
  // unconditional loads keep the outstanding-load count the same on every
  // path, so the waits before the MFMAs cover only the older register set
  __device__ __forceinline__ void advance(bool go) { ptr += go ? (KC ? (int64_t)32 : 32 * ld) : 0; }
};

__device__ __forceinline__ void mfma4(f32x16& acc, const f32x4& a, const f32x4& b) {
#pragma unroll
  for (int j = 0; j < 4; ++j) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a[j], b[j], acc, 0, 0, 0);
}

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

  // whole groups of four chunks (32 k): the loads of group g+1 are issued
  // before the 16 MFMAs of group g; then one guarded partial group
  const int kfull = ke > kb ? kb + ((ke - kb) / 32) * 32 : kb;
  int k0 = kb;
  if (k0 < kfull) {
    // two register sets in turn: the loads into one are in flight while
    // the MFMAs read the other
    GroupReader<!TA, VEC> ra(p.a, p.lda, row, kb, h);
    GroupReader<TB, VEC> rb(p.b, p.ldb, col, kb, h);
    f32x4 a0[4], b0[4], a1[4], b1[4];
    ra.read(a0);
    rb.read(b0);
    for (;;) {
      const bool more1 = k0 + 32 < kfull;
      ra.advance(more1);
      rb.advance(more1);
      ra.read(a1);
      rb.read(b1);
      // keep the next group's loads ahead of this group's MFMAs
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int c = 0; c < 4; ++c) mfma4(acc, a0[c], b0[c]);
      k0 += 32;
      if (!more1) break;
      const bool more2 = k0 + 32 < kfull;
      ra.advance(more2);
      rb.advance(more2);
      ra.read(a0);
      rb.read(b0);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int c = 0; c < 4; ++c) mfma4(acc, a1[c], b1[c]);
      k0 += 32;
      if (!more2) break;
    }
  }
  if (k0 < ke) {
    f32x4 a[4], b[4];
    load_group<TA, TB, VEC, true>(p, row, col, k0, h, ke, a, b);
#pragma unroll
    for (int c = 0; c < 4; ++c) mfma4(acc, a[c], b[c]);
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
