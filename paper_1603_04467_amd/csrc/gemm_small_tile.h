// The k loop of a 32 x 32 fp32 output tile on v_mfma_f32_32x32x2_f32, shared
// by the small-problem MatMul (gemm_small.hip) and the one-kernel training
// step (step_fused.hip): each wave of a workgroup sums a contiguous slice of
// k straight from registers, with the next 32 k of operands loaded while the
// current 32 are multiplied (no LDS staging: every operand element is used
// by one MFMA of one wave, and small operands stay in L2). Per 8 values of k
// a lane loads 4 consecutive k of its row of A and of its column of B:
// 16-byte loads for a k-contiguous operand, 4 coalesced loads for an
// m/n-contiguous one. The four instructions of a chunk take k + j (lanes
// 0-31) and k + 4 + j (lanes 32-63), j = 0..3, for A and B alike, so each k is
// summed exactly once. Lanes past the last row or column read clamped indices
// (the caller clamps; their results are never stored) and k past the end
// reads zeros, so any shape and leading dimension works.
#pragma once

#include "common.h"

namespace tfd {
namespace small_tile {

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
__device__ __forceinline__ void load_group(const float* __restrict__ pa, int64_t lda, const float* __restrict__ pb,
                                           int64_t ldb, int row, int col, int k0, int h, int ke, f32x4 (&a)[4],
                                           f32x4 (&b)[4]) {
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int kk = k0 + 8 * c + 4 * h;
    a[c] = TA ? load_mn<GUARD>(pa, lda, row, kk, ke) : load_kc<VEC, GUARD>(pa, lda, row, kk, ke);
    b[c] = TB ? load_kc<VEC, GUARD>(pb, ldb, col, kk, ke) : load_mn<GUARD>(pb, ldb, col, kk, ke);
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

// acc += sum over k in [kb, ke) of op(A)[row][k] op(B)[k][col] in the MFMA's
// lane layout (lane l32 + 32 h: row or column l32; op(A) = A, or A^T when
// TA; op(B) = B, or B^T when TB). VEC: 16-byte loads of the k-contiguous
// operands (16-byte aligned rows).
template <bool TA, bool TB, bool VEC>
__device__ __forceinline__ void tile_k(const float* __restrict__ pa, int64_t lda, const float* __restrict__ pb,
                                       int64_t ldb, int row, int col, int kb, int ke, int h, f32x16& acc) {
  // whole groups of four chunks (32 k): the loads of group g+1 are issued
  // before the 16 MFMAs of group g; then one guarded partial group
  const int kfull = ke > kb ? kb + ((ke - kb) / 32) * 32 : kb;
  int k0 = kb;
  if (k0 < kfull) {
    // two register sets in turn: the loads into one are in flight while
    // the MFMAs read the other
    GroupReader<!TA, VEC> ra(pa, lda, row, kb, h);
    GroupReader<TB, VEC> rb(pb, ldb, col, kb, h);
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
    load_group<TA, TB, VEC, true>(pa, lda, pb, ldb, row, col, k0, h, ke, a, b);
#pragma unroll
    for (int c = 0; c < 4; ++c) mfma4(acc, a[c], b[c]);
  }
}

// Register r of a lane's accumulator holds tile element (8 (r / 4) + 4 h +
// r % 4, l32); stores the wave's partial tile at part[element].
__device__ __forceinline__ void store_part(float* part, const f32x16& acc, int h, int l32) {
#pragma unroll
  for (int r = 0; r < 16; ++r) part[(8 * (r >> 2) + 4 * h + (r & 3)) * 32 + l32] = acc[r];
}

}  // namespace small_tile
}  // namespace tfd
