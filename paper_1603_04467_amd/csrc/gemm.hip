// MatMul (the paper's section 2, Table 1) with the transpose attributes and a
// fused bias + ReLU epilogue (Figure 1's Relu(Wx + b)), on gfx950 matrix
// cores.
//
// C[m x n] = epi(op(A) op(B)), fp32 accumulation:
//   fp32 operands: v_mfma_f32_32x32x2_f32   (32x32 tile, 2 k per instruction)
//   bf16 operands: v_mfma_f32_32x32x16_bf16 (32x32 tile, 16 k per instruction)
//
// Block tile BM x BN, k-tile of 128 bytes per row (32 fp32 / 64 bf16), waves
// arranged WM x WN, each owning a (BM/WM) x (BN/WN) sub-tile of 32x32
// fragments. Both operand tiles live in LDS "k-contiguous": one 128-byte row
// per output row (A) or output column (B), split into eight 16-byte chunks
// whose positions are XOR-swizzled by the row index, so that the fragment
// reads (ds_read_b128, 32 rows per half-wave) and the tile writes hit
// distinct banks. An operand that is k-contiguous in memory (A of NN/NT, B
// of NT) is copied chunk for chunk; one that is m/n-contiguous (B of NN,
// both of TN) is loaded as V x V blocks (V = elements per 16 bytes) and
// transposed in registers on the way to LDS. LDS is double-buffered: the
// global loads of k-tile t+1 are in flight while the matrix cores consume
// k-tile t, with one barrier per k-tile. fp32 problems of whole 256 x 256
// tiles take gemm_f32_256 instead, whose copies go straight from global
// memory into LDS and whose m/n-contiguous operands stay m/n-major there.
//
// K-slot assignment: within a k-tile, lanes 0-31 supply k in [0, BK/2) and
// lanes 32-63 k in [BK/2, BK), eight (bf16) or one (fp32) per instruction,
// identically for A and B, so every k of the tile is summed exactly once.
//
// Output fragment layout of a 32x32 MFMA: lane l, accumulator register r
// holds C[8*(r/4) + 4*(l/32) + r%4][l%32].

#include <stdlib.h>

#include "common.h"
#include "kernels.h"

namespace tfd {

namespace {

struct GemmParams {
  const void* a;
  const void* b;
  void* c;
  const float* bias;
  int64_t lda, ldb, ldc;
  int m, n, k;
  int epi;
  int tiles_m, tiles_n;
};

__device__ __forceinline__ int swz(int row) { return (row ^ (row >> 3)) & 7; }
__device__ __forceinline__ int lds_off(int row, int chunk) {
  return row * 128 + ((chunk ^ swz(row)) << 4);
}

// Map a workgroup id to an output tile. Workgroups are dealt round-robin to
// the 8 XCDs; consecutive ids on one XCD get consecutive tile slots, and the
// tile slots are walked in bands of kGroupM tile-rows so that the tiles in
// flight on one XCD share A rows and B columns in that XCD's L2.
constexpr int kGroupM = 8;
__device__ __forceinline__ void tile_of_block(int bid, int tiles_m, int tiles_n, int& tm, int& tn) {
  const int total = tiles_m * tiles_n;
  int t = bid;
  if (total % kNumXcd == 0) t = (bid % kNumXcd) * (total / kNumXcd) + bid / kNumXcd;
  const int per_group = kGroupM * tiles_n;
  const int group = t / per_group;
  const int first_m = group * kGroupM;
  const int gsize = min(tiles_m - first_m, kGroupM);
  const int in_group = t - group * per_group;
  tm = first_m + in_group % gsize;
  tn = in_group / gsize;
}

// Load one 16-byte chunk of V elements starting at p (elements idx0..idx0+V-1
// of a row), with `valid` elements in range; the rest are zero.
template <typename T, bool ALIGNED>
__device__ __forceinline__ u32x4 load_chunk(const T* row_ptr, int idx0, int valid) {
  constexpr int V = elem_traits<T>::vec;
  if (ALIGNED) {
    if (valid >= V) return *reinterpret_cast<const u32x4*>(row_ptr + idx0);
    return u32x4{0u, 0u, 0u, 0u};
  } else {
    T tmp[V];
#pragma unroll
    for (int e = 0; e < V; ++e) tmp[e] = (e < valid) ? row_ptr[idx0 + e] : static_cast<T>(0.0f);
    u32x4 r;
    __builtin_memcpy(&r, tmp, 16);
    return r;
  }
}

// Transpose a V x V block held as V chunks (chunk r = row r, V elements) into
// V chunks where chunk c holds column c.
__device__ __forceinline__ void transpose_block(const u32x4 (&in)[4], u32x4 (&out)[4]) {
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int r = 0; r < 4; ++r) out[c][r] = in[r][c];
}
__device__ __forceinline__ void transpose_block(const u32x4 (&in)[8], u32x4 (&out)[8]) {
  // 8 x 8 block of 16-bit values; chunk r dword d = (elem 2d | elem 2d+1 << 16).
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    const int d = c >> 1;
    const bool hi = c & 1;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t lo_src = in[2 * j][d];
      const uint32_t hi_src = in[2 * j + 1][d];
      out[c][j] = hi ? ((lo_src >> 16) | (hi_src & 0xFFFF0000u))
                     : ((lo_src & 0xFFFFu) | (hi_src << 16));
    }
  }
}

// One operand's k-tile: global -> registers -> LDS.
//   KC = true : op(X)[mn][k] = X[mn * ld + k]   (k-contiguous)
//   KC = false: op(X)[mn][k] = X[k * ld + mn]   (mn-contiguous)
template <typename T, int R, int NT, bool KC, bool ALIGNED>
struct TileLoader {
  static constexpr int V = elem_traits<T>::vec;
  static constexpr int BK = 8 * V;
  static constexpr int kChunks = R * 8;         // 16-byte chunks in the tile
  static constexpr int kBlocks = 8 * (R / V);   // V x V blocks in the tile
  static constexpr int kChunksPerThread = KC ? (kChunks + NT - 1) / NT : 0;
  static constexpr int kBlocksPerThread = KC ? 0 : (kBlocks + NT - 1) / NT;
  static constexpr int kRegs = KC ? kChunksPerThread : kBlocksPerThread * V;
  static_assert(KC ? kChunks % NT == 0 : (kBlocks % NT == 0 || kBlocks < NT), "tile/thread mismatch");
  u32x4 regs[kRegs > 0 ? kRegs : 1];

  __device__ __forceinline__ void load(const T* X, int64_t ld, int mn0, int mn_ext, int k0, int k_ext,
                                       int tid) {
    if (KC) {
#pragma unroll
      for (int i = 0; i < kChunksPerThread; ++i) {
        const int c = tid + i * NT;
        const int row = c >> 3, ch = c & 7;
        const int mn = mn0 + row;
        const int kk = k0 + ch * V;
        const int valid = (mn < mn_ext) ? min(max(k_ext - kk, 0), V) : 0;
        const T* rp = X + (int64_t)min(mn, mn_ext - 1) * ld;
        regs[i] = (valid > 0) ? load_chunk<T, ALIGNED>(rp, kk, valid) : u32x4{0u, 0u, 0u, 0u};
      }
    } else {
#pragma unroll
      for (int i = 0; i < kBlocksPerThread; ++i) {
        const int s = tid + i * NT;
        if (s >= kBlocks) break;
        const int mb = s % (R / V), kb = s / (R / V);
        const int mn = mn0 + mb * V;
        const int vmn = min(max(mn_ext - mn, 0), V);
#pragma unroll
        for (int r = 0; r < V; ++r) {
          const int kk = k0 + kb * V + r;
          const int valid = (kk < k_ext) ? vmn : 0;
          const T* rp = X + (int64_t)min(kk, k_ext - 1) * ld;
          regs[i * V + r] = (valid > 0) ? load_chunk<T, ALIGNED>(rp, mn, valid) : u32x4{0u, 0u, 0u, 0u};
        }
      }
    }
  }

  __device__ __forceinline__ void store(char* lds, int tid) {
    if (KC) {
#pragma unroll
      for (int i = 0; i < kChunksPerThread; ++i) {
        const int c = tid + i * NT;
        *reinterpret_cast<u32x4*>(lds + lds_off(c >> 3, c & 7)) = regs[i];
      }
    } else {
#pragma unroll
      for (int i = 0; i < kBlocksPerThread; ++i) {
        const int s = tid + i * NT;
        if (s >= kBlocks) break;
        const int mb = s % (R / V), kb = s / (R / V);
        u32x4 in[V], out[V];
#pragma unroll
        for (int r = 0; r < V; ++r) in[r] = regs[i * V + r];
        transpose_block(in, out);
#pragma unroll
        for (int c = 0; c < V; ++c)
          *reinterpret_cast<u32x4*>(lds + lds_off(mb * V + c, kb)) = out[c];
      }
    }
  }
};

template <typename T>
__device__ __forceinline__ void mfma_chunk(f32x16& acc, const u32x4& a, const u32x4& b);

template <>
__device__ __forceinline__ void mfma_chunk<float>(f32x16& acc, const u32x4& a, const u32x4& b) {
  // Reinterpret the whole 16-byte chunk: a bit cast of a single vector
  // element (a[s]) is lowered by clang to element 0.
  const f32x4 af = __builtin_bit_cast(f32x4, a);
  const f32x4 bf = __builtin_bit_cast(f32x4, b);
#pragma unroll
  for (int s = 0; s < 4; ++s) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(af[s], bf[s], acc, 0, 0, 0);
}

template <>
__device__ __forceinline__ void mfma_chunk<bf16>(f32x16& acc, const u32x4& a, const u32x4& b) {
  acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                __builtin_bit_cast(bf16x8, b), acc, 0, 0, 0);
}

// Epilogue: bias, Relu, one rounding to OutT, for a wave's FM x FN
// fragments whose first output row / column are row0 / col0.
template <typename OutT, int FM, int FN>
__device__ __forceinline__ void store_tile(const GemmParams& p, const f32x16 (&acc)[FM][FN], int row0, int col0,
                                           int half, int l32) {
  OutT* C = static_cast<OutT*>(p.c);
  const bool trunc16 = (p.epi & kEpiTrunc16) != 0;
#pragma unroll
  for (int j = 0; j < FN; ++j) {
    const int col = col0 + j * 32 + l32;
    const bool col_ok = col < p.n;
    const float bv = ((p.epi & kEpiOpMask) != 0 && col_ok) ? p.bias[col] : 0.0f;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = row0 + i * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
        if (col_ok && row < p.m) {
          float v = acc[i][j][r] + bv;
          if ((p.epi & kEpiOpMask) == 2) v = relu_f32(v);
          store_from_f32(C + (int64_t)row * p.ldc + col, v, trunc16);
        }
      }
    }
  }
}

template <typename T, typename OutT, bool TA, bool TB, int BM, int BN, int WM, int WN, bool ALIGNED>
__global__ __launch_bounds__(WM * WN * kWave) void gemm_kernel(GemmParams p) {
  constexpr int NT = WM * WN * kWave;
  constexpr int V = elem_traits<T>::vec;
  constexpr int BK = 8 * V;
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int FM = WTM / 32, FN = WTN / 32;
  static_assert(FM >= 1 && FN >= 1, "wave tile must hold a 32x32 fragment");
  constexpr int kStageBytes = (BM + BN) * 128;

  __shared__ __attribute__((aligned(16))) char smem[2 * kStageBytes];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wave_m = wave / WN, wave_n = wave % WN;
  const int half = lane >> 5, l32 = lane & 31;

  int tm, tn;
  tile_of_block(blockIdx.x, p.tiles_m, p.tiles_n, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;

  const T* A = static_cast<const T*>(p.a);
  const T* B = static_cast<const T*>(p.b);

  TileLoader<T, BM, NT, !TA, ALIGNED> la;
  TileLoader<T, BN, NT, TB, ALIGNED> lb;

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int kt_count = (p.k + BK - 1) / BK;
  if (kt_count > 0) {
    la.load(A, p.lda, m0, p.m, 0, p.k, tid);
    lb.load(B, p.ldb, n0, p.n, 0, p.k, tid);
    la.store(smem, tid);
    lb.store(smem + BM * 128, tid);
    __syncthreads();
  }

  // The other stage is free from the barrier that opens k-tile t (every
  // wave has finished reading it), so k-tile t+1 is fetched after the
  // first k-step's fragment reads and written to LDS after the second
  // k-step's MFMAs: both hide behind the matrix-core work of the current
  // k-tile, and only the barrier and the first fragment reads remain
  // between k-tiles. (Writing after the first k-step waits on loads still
  // in flight; moving the barrier ahead of the last k-step's MFMAs to
  // prefetch the next k-tile's first fragments spills registers in the
  // loop. Both measured slower.)
  constexpr int kStoreAfter = 1;
  for (int kt = 0; kt < kt_count; ++kt) {
    const bool more = kt + 1 < kt_count;
    const char* sa = smem + (kt & 1) * kStageBytes;
    const char* sb = sa + BM * 128;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int chunk = half * 4 + q;
      u32x4 fa[FM], fb[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i)
        fa[i] = *reinterpret_cast<const u32x4*>(sa + lds_off(wave_m * WTM + i * 32 + l32, chunk));
#pragma unroll
      for (int j = 0; j < FN; ++j)
        fb[j] = *reinterpret_cast<const u32x4*>(sb + lds_off(wave_n * WTN + j * 32 + l32, chunk));
      if (q == 0 && more) {
        la.load(A, p.lda, m0, p.m, (kt + 1) * BK, p.k, tid);
        lb.load(B, p.ldb, n0, p.n, (kt + 1) * BK, p.k, tid);
      }
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) mfma_chunk<T>(acc[i][j], fa[i], fb[j]);
      if (q == kStoreAfter && more) {
        char* st = smem + ((kt + 1) & 1) * kStageBytes;
        la.store(st, tid);
        lb.store(st + BM * 128, tid);
      }
    }
    __syncthreads();
  }

  store_tile<OutT, FM, FN>(p, acc, m0 + wave_m * WTM, n0 + wave_n * WTN, half, l32);
}


// Whole 256 x 256 fp32 tiles (m, n multiples of 256, k a multiple of 32,
// 16-byte aligned rows): the same two LDS stages, k-slot assignment and
// MFMAs as above, with the copies going straight from global memory into LDS
// (global_load_lds_dwordx4: 64 lanes x 16 bytes land contiguously in 1 KiB
// of LDS), so that no registers stage them and no transpose pass or LDS
// write instruction is needed. 8 waves of 128 x 64.
//  - k-contiguous operand: the 128-byte-row layout above; in a 1 KiB block
//    (8 rows) lane i fills slot i % 8 of row i / 8, i.e. it fetches the chunk
//    that the row's swizzle puts in that slot.
//  - m/n-contiguous operand: k-rows of 256 values (1 KiB), value mn of k-row
//    kr at kr * 1024 + 16 * ((mn / 4) ^ mn_swz(kr)) + 4 * (mn % 4). A lane of
//    a fragment read takes four consecutive k of one column (four ds_read_b32
//    1 KiB apart, merged by the compiler into ds_read2st64_b32); mn_swz moves
//    the k-rows 16..31, read by lanes 32..63 at the same time as lanes 0..31
//    read rows 0..15, to the other 128 bytes of the banks.
typedef __attribute__((address_space(3))) void lds_void;
__device__ __forceinline__ int mn_swz(int krow) { return ((krow >> 4) & 1) << 3; }

template <bool KC>
__device__ __forceinline__ void copy_tile_f32(const float* X, int64_t ld, int mn0, int k0, char* lds, int wave,
                                              int lane) {
#pragma unroll
  for (int j = 0; j < 4; ++j) {  // 32 blocks of 1 KiB per operand, 4 per wave
    const int blk = wave * 4 + j;
    const float* g;
    if (KC) {
      const int r = blk * 8 + (lane >> 3);
      g = X + (int64_t)(mn0 + r) * ld + k0 + (((lane & 7) ^ swz(r)) << 2);
    } else {
      g = X + (int64_t)(k0 + blk) * ld + mn0 + ((lane ^ mn_swz(blk)) << 2);
    }
    __builtin_amdgcn_global_load_lds(g, (lds_void*)(lds + blk * 1024), 16, 0, 0);
  }
}

// Four consecutive k (k0 .. k0+3, one group of 16 k-rows) of column mn of an
// m/n-major operand tile.
__device__ __forceinline__ u32x4 read_mn_f32(const char* tile, int mn, int k0) {
  const char* q = tile + k0 * 1024 + (((mn >> 2) ^ mn_swz(k0)) << 4) + ((mn & 3) << 2);
  u32x4 r;
#pragma unroll
  for (int s = 0; s < 4; ++s) r[s] = *reinterpret_cast<const uint32_t*>(q + s * 1024);
  return r;
}

template <bool TA, bool TB>
__global__ __launch_bounds__(512) void gemm_f32_256(GemmParams p) {
  constexpr int WN = 4, WTM = 128, WTN = 64, FM = WTM / 32, FN = WTN / 32;
  constexpr bool A_KC = !TA, B_KC = TB;
  constexpr int kOperandBytes = 256 * 128, kStageBytes = 2 * kOperandBytes;
  __shared__ __attribute__((aligned(1024))) char smem[2 * kStageBytes];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wave_m = wave / WN, wave_n = wave % WN;
  const int half = lane >> 5, l32 = lane & 31;

  int tm, tn;
  tile_of_block(blockIdx.x, p.tiles_m, p.tiles_n, tm, tn);
  const int m0 = tm * 256, n0 = tn * 256;
  const float* A = static_cast<const float*>(p.a);
  const float* B = static_cast<const float*>(p.b);

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int kt_count = p.k / 32;
  copy_tile_f32<A_KC>(A, p.lda, m0, 0, smem, wave, lane);
  copy_tile_f32<B_KC>(B, p.ldb, n0, 0, smem + kOperandBytes, wave, lane);
  __builtin_amdgcn_s_waitcnt(0);  // vmcnt(0) lgkmcnt(0)
  __syncthreads();

  // Fragments of k-step q (k = 4 * chunk + s in MFMA sub-step s).
  auto read_frags = [&](const char* st, int q, u32x4 (&a_)[FM], u32x4 (&b_)[FN]) {
    const char* sb = st + kOperandBytes;
    const int chunk = half * 4 + q;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int r = wave_m * WTM + i * 32 + l32;
      a_[i] = A_KC ? *reinterpret_cast<const u32x4*>(st + lds_off(r, chunk)) : read_mn_f32(st, r, 4 * chunk);
    }
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int c = wave_n * WTN + j * 32 + l32;
      b_[j] = B_KC ? *reinterpret_cast<const u32x4*>(sb + lds_off(c, chunk)) : read_mn_f32(sb, c, 4 * chunk);
    }
  };
  // NN and NT pass the barrier that publishes k-tile t+1 before the last
  // k-step's MFMAs of k-tile t and read k-tile t+1's first fragments behind
  // them (measured 0.3 % and 1.6 % faster; TN, whose operands are both
  // read as dword pairs, 0.5 % slower).
  constexpr bool kEarlyBarrier = !TA;
  u32x4 fa[FM], fb[FN], na[FM], nb[FN];
  if constexpr (kEarlyBarrier) read_frags(smem, 0, na, nb);

  for (int kt = 0; kt < kt_count; ++kt) {
    const char* sa = smem + (kt & 1) * kStageBytes;
    char* nx = smem + ((kt + 1) & 1) * kStageBytes;
    const bool more = kt + 1 < kt_count;
    if (more) {
      copy_tile_f32<A_KC>(A, p.lda, m0, (kt + 1) * 32, nx, wave, lane);
      copy_tile_f32<B_KC>(B, p.ldb, n0, (kt + 1) * 32, nx + kOperandBytes, wave, lane);
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (kEarlyBarrier && q == 0) {
#pragma unroll
        for (int i = 0; i < FM; ++i) fa[i] = na[i];
#pragma unroll
        for (int j = 0; j < FN; ++j) fb[j] = nb[j];
      } else {
        read_frags(sa, q, fa, fb);
      }
      if (kEarlyBarrier && q == 3) {
        __builtin_amdgcn_s_waitcnt(0);  // this wave's copies of k-tile t+1 have landed
        __syncthreads();
        if (more) read_frags(nx, 0, na, nb);
      }
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) mfma_chunk<float>(acc[i][j], fa[i], fb[j]);
    }
    if constexpr (!kEarlyBarrier) {
      __builtin_amdgcn_s_waitcnt(0);  // this wave's copies of k-tile t+1 have landed
      __syncthreads();
    }
  }

  store_tile<float, FM, FN>(p, acc, m0 + wave_m * WTM, n0 + wave_n * WTN, half, l32);
}

template <bool TA, bool TB>
hipError_t launch_f32_256(const GemmDesc& d, hipStream_t s) {
  GemmParams p;
  p.a = d.a;
  p.b = d.b;
  p.c = d.c;
  p.bias = d.bias;
  p.lda = d.lda;
  p.ldb = d.ldb;
  p.ldc = d.ldc;
  p.m = (int)d.m;
  p.n = (int)d.n;
  p.k = (int)d.k;
  p.epi = d.epi;
  p.tiles_m = (int)(d.m / 256);
  p.tiles_n = (int)(d.n / 256);
  hipLaunchKernelGGL((gemm_f32_256<TA, TB>), dim3(p.tiles_m * p.tiles_n), dim3(512), 0, s, p);
  return hipGetLastError();
}

template <typename T, typename OutT, bool TA, bool TB, int BM, int BN, int WM, int WN, bool ALIGNED>
hipError_t launch_cfg(const GemmDesc& d, hipStream_t s) {
  GemmParams p;
  p.a = d.a;
  p.b = d.b;
  p.c = d.c;
  p.bias = d.bias;
  p.lda = d.lda;
  p.ldb = d.ldb;
  p.ldc = d.ldc;
  p.m = (int)d.m;
  p.n = (int)d.n;
  p.k = (int)d.k;
  p.epi = d.epi;
  p.tiles_m = (int)((d.m + BM - 1) / BM);
  p.tiles_n = (int)((d.n + BN - 1) / BN);
  dim3 grid(p.tiles_m * p.tiles_n), block(WM * WN * kWave);
  hipLaunchKernelGGL((gemm_kernel<T, OutT, TA, TB, BM, BN, WM, WN, ALIGNED>), grid, block, 0, s, p);
  return hipGetLastError();
}

// Tile configuration: 0 = pick by problem size (16-bit operands on whole
// 256 x 256 tiles go to the direct-to-LDS kernel of gemm_bf16.hip),
// 1 = 256x256 (4 waves of 128x128), 2 = 256x128 (4 waves of 128x64),
// 3 = 128x128 (4 waves of 64x64), 4 = 64x64 (4 waves of 32x32); fp32 only:
// 5 = 256x256 (8 waves of 128x64), 6 = 256x256 (16 waves of 64x64),
// 7 = 128x128 (8 waves of 64x32), 8 = the small-problem kernel of
// gemm_small.hip (the default for fp32 problems with fewer than 128 tiles of
// 128 x 128), 9 = the whole-tile direct-to-LDS kernel gemm_f32_256 (8 waves
// of 128x64; the default for fp32 problems of whole 256 x 256 tiles and at
// least 128 of them, else 5 takes its place). Non-zero values come from the
// "gemm_tile" tuning knob (tfd_set_tuning).
template <typename T, typename OutT, bool TA, bool TB>
hipError_t launch_layout(const GemmDesc& d, bool aligned, int tile, hipStream_t s) {
  if (!aligned) return launch_cfg<T, OutT, TA, TB, 64, 64, 2, 2, false>(d, s);
  if (tile == 0) {
    const int64_t tiles256 = ((d.m + 255) / 256) * ((d.n + 255) / 256);
    const int64_t tiles128 = ((d.m + 127) / 128) * ((d.n + 127) / 128);
    // fp32: 256x256 with 8 waves (2 per SIMD) measured fastest inside the step
    tile = tiles256 >= 128 ? (sizeof(T) == 4 ? 9 : 1) : (tiles128 >= 128 ? 3 : 4);
  }
  if constexpr (sizeof(T) == 4) {  // fp32-only shapes
    const bool whole = d.m % 256 == 0 && d.n % 256 == 0 && d.k % 32 == 0 && d.k > 0;
    if (tile == 9 && whole) return launch_f32_256<TA, TB>(d, s);
    switch (tile) {
      case 9:
      case 5: return launch_cfg<T, OutT, TA, TB, 256, 256, 2, 4, true>(d, s);
      case 6: return launch_cfg<T, OutT, TA, TB, 256, 256, 4, 4, true>(d, s);
      case 7: return launch_cfg<T, OutT, TA, TB, 128, 128, 2, 4, true>(d, s);
      default: break;
    }
  }
  switch (tile) {
    case 1: return launch_cfg<T, OutT, TA, TB, 256, 256, 2, 2, true>(d, s);
    case 2: return launch_cfg<T, OutT, TA, TB, 256, 128, 2, 2, true>(d, s);
    case 3: return launch_cfg<T, OutT, TA, TB, 128, 128, 2, 2, true>(d, s);
    default: return launch_cfg<T, OutT, TA, TB, 64, 64, 2, 2, true>(d, s);
  }
}

template <typename T, typename OutT>
hipError_t launch_types(const GemmDesc& d, bool aligned, int tile, hipStream_t s) {
  if (!d.ta && !d.tb) return launch_layout<T, OutT, false, false>(d, aligned, tile, s);
  if (!d.ta && d.tb) return launch_layout<T, OutT, false, true>(d, aligned, tile, s);
  return launch_layout<T, OutT, true, false>(d, aligned, tile, s);
}

}  // namespace

// Vector (16-byte) loads are legal when every row start of both operands is
// 16-byte aligned and each operand's contiguous extent is whole chunks.
bool gemm_vector_ok(const GemmDesc& d, int elem_bytes) {
  const int V = 16 / elem_bytes;
  auto al = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; };
  const int64_t a_contig = d.ta ? d.m : d.k;
  const int64_t b_contig = d.tb ? d.k : d.n;
  return al(d.a) && al(d.b) && d.lda % V == 0 && d.ldb % V == 0 && a_contig % V == 0 &&
         b_contig % V == 0;
}

hipError_t launch_gemm(const GemmDesc& d, hipStream_t s) {
  const int tile = gemm_tile_override();
  if (tile == 0 && gemm_bf16_256_ok(d)) return launch_gemm_bf16_256(d, s);
  if (!d.in_bf16 && (tile == 8 || (tile == 0 && gemm_small_preferred(d)))) return launch_gemm_small_f32(d, s);
  if (d.in_bf16) {
    const bool aligned = gemm_vector_ok(d, 2);
    return d.out_bf16 ? launch_types<bf16, bf16>(d, aligned, tile, s)
                      : launch_types<bf16, float>(d, aligned, tile, s);
  }
  return launch_types<float, float>(d, gemm_vector_ok(d, 4), tile, s);
}

}  // namespace tfd
