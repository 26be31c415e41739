// MatMul for 16-bit operands on whole 256 x 256 output tiles (the shapes of
// the wide dense layers), fp32 accumulation, with the epilogues of the
// training step fused into it.
//
// Per workgroup: one 256 x 256 output tile (or one k-range split of it),
// split over 4 waves of 128 x 128 (long k ranges; 16 x 16 fragments of
// v_mfma_f32_16x16x32_bf16 accumulators, brought into the 32 x 32 layout
// for the epilogue), 8 waves of 128 x 64 or 16 waves of 64 x 64 (32 x 32
// fragments of v_mfma_f32_32x32x16_bf16 accumulators).
// The k loop walks 64-wide k-tiles through two LDS stages of 64 KiB:
//  - global -> LDS copies go straight into LDS (global_load_lds_dwordx4, 1 KiB
//    per wave instruction), so no registers stage them; the copy of k-tile
//    t+1 is in flight while the matrix cores work on k-tile t;
//  - an operand that is k-contiguous in memory is kept as 256 rows of 64 k
//    (128 B rows, 16-byte chunks XOR-swizzled by row) and read with
//    ds_read_b128: eight consecutive k of one row per lane;
//  - an operand that is m/n-contiguous in memory is kept as 64 k-rows of 256
//    values (512 B rows, chunks XOR-swizzled by k) and read with the gfx950
//    transposing read ds_read_b64_tr_b16, which hands each lane of a 16-lane
//    group four consecutive k of one column (two reads make the eight k an
//    MFMA lane needs), so no transpose pass is needed anywhere (issued as
//    inline assembly, see ds_read_tr16_b64);
//  - fragments are double-buffered in registers: the reads for k-step q+1 are
//    interleaved with the MFMAs of k-step q.
// K-slot assignment (identical for both operands, so each k is summed once):
// with 8 or 16 waves lane l supplies k = 32*(l/32) + 8*q + e, e = 0..7, in
// k-step q (16 k) of a k-tile; with 4 waves k = 32*q + 8*c(l/16) + e in k-step
// q (32 k), c = 0, 2, 1, 3.
// Epilogues (see the EP list below): bias, ReLU and one rounding; a 16-bit
// tile is staged through LDS and leaves in 16-byte row chunks; ReLU masks
// from wave ballots; ReluGrad from features or a mask with the tile's column
// sums; the squared-error head. Outputs are written with non-temporal
// stores. A split k range writes fp32 partial tiles that
// splitk_reduce_kernel sums in order.
//
// Preconditions (checked by the dispatcher): m, n multiples of 256, k a
// multiple of 64, 16-byte aligned rows.

#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace tfd {

namespace {

typedef __attribute__((address_space(3))) void lds_void;

constexpr int kBM = 256, kBN = 256, kBK = 64;

constexpr int kOperandBytes = 256 * 128;          // one operand's k-tile (32 KiB)
constexpr int kStageBytes = 2 * kOperandBytes;   // A + B

struct Params {
  const bf16* a;
  const bf16* b;
  void* c;
  const float* bias;
  int64_t lda, ldb, ldc;
  int m, n, k;
  int epi;
  int tiles_m, tiles_n;
  const uint16_t* features;  // ReluGrad epilogue: the stored forward output
  int64_t ldf;
  float* col_partial;        // [tiles_m][n] column sums of the stored tiles
  const uint16_t* target;    // squared-error epilogue: target and gradient (ld = n)
  uint16_t* grad;
  double* loss_partial;      // [tiles] float64 sums of squared differences
  // ReLU masks, one bit per element: row r of a mask is ldm uint32 words,
  // bit j of word w holds element (r, 32 w + j).
  const uint32_t* mask_in;   // ReluGrad epilogue from a mask instead of features
  uint32_t* mask_out;        // forward epilogue: bits of the stored output's > 0
  int64_t ldm;
  // Split of the k range over `splits` workgroups per tile (1: none). Split
  // s covers k-tiles [s * kt_per, min((s + 1) * kt_per, k / 64)) and writes
  // its fp32 partial tile to c + s * m * ldc; the partials are summed by
  // splitk_reduce_kernel.
  int splits, kt_per;
  int group_m;  // tile-rows per band of the tile order (tile_of_block)
};

// Epilogues of the whole-tile kernel beyond bias/ReLU (16-bit outputs only).
constexpr int kEpPlain = 0, kEpReluGrad = 1, kEpLoss = 2, kEpReluGradBits = 3, kEpMaskOut = 4;

__device__ __forceinline__ int swz_kc(int row) { return (row ^ (row >> 3)) & 7; }
// m/n-contiguous operand: chunk c of k-row kr at slot c ^ swz_mn(kr). Bits 2-3
// come from kr's low two bits (the four k-rows of one transposing read), bit 1
// from kr's bit 4: the 4-wave loop's two 16-lane groups of a half-wave read
// k-rows 16 apart in the same columns, which this puts in different banks.
__device__ __forceinline__ int swz_mn(int krow) { return ((krow & 3) << 2) | (((krow >> 4) & 1) << 1); }

// Block -> tile: the blocks dispatched to one XCD (every eighth) take a
// contiguous range of tiles, walked in bands of group_m tile-rows, so that the
// tiles an XCD runs at a time share operand panels in its L2.
__device__ __forceinline__ void tile_of_block(int bid, int tiles_m, int tiles_n, int group_m, int& tm, int& tn) {
  const int total = tiles_m * tiles_n;
  int t = bid;
  if (total % kNumXcd == 0) t = (bid % kNumXcd) * (total / kNumXcd) + bid / kNumXcd;
  const int per_group = group_m * tiles_n;
  const int group = t / per_group;
  const int first_m = group * group_m;
  const int gsize = min(tiles_m - first_m, group_m);
  const int in_group = t - group * per_group;
  tm = first_m + in_group % gsize;
  tn = in_group / gsize;
}

// Copy one operand's k-tile into LDS. KC: op(X)[mn][k] = X[mn * ld + k];
// otherwise op(X)[mn][k] = X[k * ld + mn]. Each of the 4 waves issues 8
// instructions of 64 lanes x 16 bytes; lane i's bytes land at lds + 16 i.
template <bool KC, int kThreads>
__device__ __forceinline__ void copy_tile(const bf16* X, int64_t ld, int mn0, int k0, char* lds, int wave,
                                          int lane) {
  constexpr int kPerWave = 32 / (kThreads / 64);  // 1 KiB blocks per wave
#pragma unroll
  for (int j = 0; j < kPerWave; ++j) {
    const int blk = wave * kPerWave + j;  // 1 KiB block of the tile
    const bf16* g;
    if (KC) {
      const int r = blk * 8 + (lane >> 3);
      const int c = (lane & 7) ^ swz_kc(r);
      g = X + (int64_t)(mn0 + r) * ld + k0 + c * 8;
    } else {
      const int kr = blk * 2 + (lane >> 5);
      const int c = (lane & 31) ^ swz_mn(kr);
      g = X + (int64_t)(k0 + kr) * ld + mn0 + c * 8;
    }
    __builtin_amdgcn_global_load_lds(g, (lds_void*)(lds + blk * 1024), 16, 0, 0);
  }
}

// Byte offset of element (row, col) of the 256 x 256 16-bit output tile
// staged in LDS: 512-byte rows of 32 chunks of 16 bytes; chunk c of row r
// sits at slot c ^ (4 * ((r >> 2) & 7)).
__device__ __forceinline__ int epi_off(int row, int col) {
  return row * 512 + (((col >> 3) ^ (((row >> 2) & 7) << 2)) << 4) + (col & 7) * 2;
}

// The transposing read ds_read_b64_tr_b16 is issued as inline assembly.
// Through its builtin, the compiler's wait insertion treats it as an LDS
// access that may overlap the global -> LDS copies in flight and puts a
// vmcnt(0) before the first one of every k-tile: the copy of k-tile t+1 then
// completes before k-step 0 of k-tile t has run, and hardly overlaps the
// matrix work. As inline assembly it is not waited on; frag_wait() below
// waits for it (lgkmcnt) and ties the fragment registers, so no instruction
// that reads them can be scheduled before the wait.
__device__ __forceinline__ uint2 ds_read_tr16_b64(const char* p) {
  uint2 u;
  const uint32_t addr = (uint32_t)(uintptr_t)((lds_void*)p);
  asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(u) : "v"(addr));
  return u;
}
__device__ __forceinline__ void frag_wait(u32x4& f) { asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(f)); }

// Building blocks of the scheduled 4-wave k loop (one wave per SIMD). Its LDS
// reads are inline assembly, so that the compiler inserts no waits of its own
// for them; the loop waits explicitly (wait_lds). Its MFMAs are the builtin,
// fenced on both sides by scheduling barriers, so that they stay exactly
// where they are written among the reads and copies while the compiler still
// knows them for what they are: it inserts the wait states an MFMA needs
// around its operands and results, also where it copies accumulators between
// registers (an MFMA written as inline assembly gets none, and such a copy
// then reads a result the matrix core has not yet written).
// LDS reads into a fragment register tuple that is tied to its previous
// contents ("+v"), so the compiler keeps every fragment buffer in the same
// registers for the whole loop and never points a read at registers that an
// MFMA issued just before still has to read.
template <int IMM>
__device__ __forceinline__ void ds_read_b128_into(u32x4& v, uint32_t addr) {
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "+v"(v) : "v"(addr), "i"(IMM));
}
// The two transposing reads of an m/n-contiguous fragment, into the low and
// high halves (k 0-3 and 4-7 of the lane's eight).
// (Clang vectors, not HIP's uint2: an inline-assembly operand of a struct
// type keeps the buffer in memory, which the compiler then places in LDS.)
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
template <int IMM0, int IMM1>
__device__ __forceinline__ void ds_read_tr_pair_into(u32x2& lo, u32x2& hi, uint32_t addr) {
  asm volatile("ds_read_b64_tr_b16 %0, %2 offset:%3\n\tds_read_b64_tr_b16 %1, %2 offset:%4"
               : "+v"(lo), "+v"(hi)
               : "v"(addr), "i"(IMM0), "i"(IMM1));
}
// f(integral_constant<int, I>) for I = 0 .. N-1, unrolled at compile time.
template <int N, int I = 0, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<N, I + 1>(f);
  }
}
// 16 x 16 x 32 MFMA, pinned in place by scheduling barriers. The 4-wave loop
// uses this form: it does the same work per cycle as the 32 x 32 x 16 form
// within 6 %, and with half the accumulator traffic per product the chip
// holds a higher clock under it. It is inline assembly on an accumulator tied
// to one AGPR quadruple: through the builtin the compiler gives the result
// registers other than the input's and copies all 256 accumulators back at
// every loop turn. The compiler then knows nothing of its wait states, so
// its users keep them: the accumulators are written (zeroed) long before the
// first MFMA (mfma16_settle), its fragment operands come straight from LDS
// reads that were waited for, and nothing reads the results before
// mfma16_settle after the last MFMA.
__device__ __forceinline__ void mfma16_acc(f32x4& acc, const u32x4& a, const u32x4& b) {
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b));
  __builtin_amdgcn_sched_barrier(0);
}
// Wait states between accumulator writes outside the MFMAs and the MFMAs
// (before the first, after the last): more than the 19 an MFMA of 16 passes
// needs before another instruction may read its result. Each accumulator is
// tied to an empty statement after them, so that no read of it can be
// scheduled before them.
__device__ __forceinline__ void mfma16_settle(f32x4 (&acc)[8][8]) {
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
#pragma unroll
  for (int a = 0; a < 8; ++a)
#pragma unroll
    for (int b = 0; b < 8; ++b) asm volatile("" : "+a"(acc[a][b]));
}
// Fragment buffer of one operand for one k-step of the 4-wave loop (8
// fragments of 16 rows or columns x 32 k): a k-contiguous operand's fragment
// is one 16-byte LDS read, an m/n-contiguous one's two 8-byte transposing
// reads (low and high halves).
template <bool KC> struct FragBuf;
template <> struct FragBuf<true> {
  u32x4 f[8];
  template <int I>
  __device__ __forceinline__ u32x4 get() const { return f[I]; }
  // Wait for every outstanding LDS read; tie the registers to the wait so
  // that nothing reads them before their data arrived.
  __device__ __forceinline__ void tie() {
    asm volatile("" : "+v"(f[0]), "+v"(f[1]), "+v"(f[2]), "+v"(f[3]), "+v"(f[4]), "+v"(f[5]), "+v"(f[6]), "+v"(f[7]));
  }
};
template <> struct FragBuf<false> {
  u32x2 lo[8], hi[8];
  template <int I>
  __device__ __forceinline__ u32x4 get() const { return u32x4{lo[I].x, lo[I].y, hi[I].x, hi[I].y}; }
  __device__ __forceinline__ void tie() {
    asm volatile("" : "+v"(lo[0]), "+v"(lo[1]), "+v"(lo[2]), "+v"(lo[3]), "+v"(lo[4]), "+v"(lo[5]), "+v"(lo[6]),
                 "+v"(lo[7]));
    asm volatile("" : "+v"(hi[0]), "+v"(hi[1]), "+v"(hi[2]), "+v"(hi[3]), "+v"(hi[4]), "+v"(hi[5]), "+v"(hi[6]),
                 "+v"(hi[7]));
  }
};
// Accumulators of a 32 x 32 block in the 32 x 32 x 16 MFMA's layout (lane L,
// register R: column L % 32, row 8 (R / 4) + 4 (L / 32) + R % 4) from its four
// 16 x 16 blocks x[bi][bj] (rows 16 bi.., columns 16 bj..) in the 16 x 16 x
// 32 MFMA's layout (lane l, register t: column l % 16, row 4 (l / 16) + t).
// Per register t and row half bi, a 16-lane row swap then a 32-lane half swap
// move the four 16-lane rows of x[bi][0] and x[bi][1] into place.
__device__ __forceinline__ f32x16 acc16_to_32(const f32x4 (&x0)[2], const f32x4 (&x1)[2]) {
  f32x16 y;
#pragma unroll
  for (int bi = 0; bi < 2; ++bi)
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      // (scalar copies: a bit cast of a vector element reads element 0)
      const float v0 = x0[bi][t], v1 = x1[bi][t];
      const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(v0), __float_as_uint(v1), false, false);
      const uint32_t p0 = p[0], p1 = p[1];
      const auto q = __builtin_amdgcn_permlane32_swap(p0, p1, false, false);
      const uint32_t q0 = q[0], q1 = q[1];
      y[8 * bi + t] = __uint_as_float(q0);
      y[8 * bi + 4 + t] = __uint_as_float(q1);
    }
  return y;
}
template <typename FA, typename FB>
__device__ __forceinline__ void wait_lds(FA& a, FB& b, bool vm) {
  if (vm)
    asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
  else
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  a.tie();
  b.tie();
}

// Fragment of 32 rows (A) or 32 columns (B) starting at `base`, k-step q.
template <bool KC>
__device__ __forceinline__ u32x4 read_frag(const char* tile, int base, int q, int lane) {
  const int half = lane >> 5;
  if (KC) {
    const int r = base + (lane & 31);
    const int chunk = half * 4 + q;
    return *reinterpret_cast<const u32x4*>(tile + r * 128 + ((chunk ^ swz_kc(r)) << 4));
  } else {
    const int g = lane >> 4, lr = lane & 15;
    const int mn = base + 16 * (g & 1) + 4 * (lr & 3);
    const int kb = 32 * half + 8 * q + (lr >> 2);
    u32x4 out;
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const int kr = kb + 4 * s;
      const int off = kr * 512 + (((mn >> 3) ^ swz_mn(kr)) << 4) + (mn & 7) * 2;
      const uint2 u = ds_read_tr16_b64(tile + off);
      out[2 * s] = u.x;
      out[2 * s + 1] = u.y;
    }
    return out;
  }
}

// Outputs leave with the non-temporal hint (here and in the fp32 epilogue):
// this kernel never re-reads them, and without the hint the dirty lines of
// the output (1 GiB for a 16384 x 32768 layer) fill L2 and are written back
// while the next tiles' operand panels are being fetched through it.
__device__ __forceinline__ void store_stream(void* p, const u32x4& v) {
  __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(p));
}

// v_writelane_b32 through its LLVM intrinsic (the compiler offers no
// builtin for it): `old` with lane `lane` set to the wave-uniform `value`.
extern "C" __device__ int tfd_writelane(int value, int lane, int old) __asm("llvm.amdgcn.writelane");

// Two fp32 values as one word of 16-bit patterns (lo in the low half). The
// nearest-even pair is one v_cvt_pk_bf16_f32 (a vector conversion; two
// scalar ones would be two conversions and an OR).
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
template <bool kTrunc>
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  if constexpr (kTrunc)
    return (uint32_t)bf16_bits_trunc(lo) | ((uint32_t)bf16_bits_trunc(hi) << 16);
  else
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

// Scheduling hint: a k-step's kMfma MFMAs spread evenly over kReads groups,
// each followed by one LDS read.
template <int T, int kReads, int kMfma>
__device__ __forceinline__ void interleave_mfma_reads() {
  if constexpr (T < kReads) {
    __builtin_amdgcn_sched_group_barrier(0x008, kMfma / kReads + (T < kMfma % kReads ? 1 : 0), 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    interleave_mfma_reads<T + 1, kReads, kMfma>();
  }
}

// EP (16-bit output only):
//  kEpReluGrad: the stored value is the rounded product where the matching
//    feature is > 0 and +0 elsewhere; the tile's column sums of the stored
//    values go to col_partial (the first pass of BiasAddGrad);
//  kEpReluGradBits: the same with the feature test read from a ReLU mask;
//  kEpMaskOut: the output is stored and so is its ReLU mask (bit set where
//    the stored value is > 0);
//  kEpLoss: the output is stored, and also grad = output - target (fp32
//    difference, rounded to nearest even), the tile's float64 sum of squared
//    differences (loss_partial) and its column sums of grad (col_partial).
// Sums run in a fixed order: each thread's rows, then row groups in order.
template <bool A_KC, bool B_KC, typename OutT, int kWavesM, int kWavesN, int EP = kEpPlain>
__global__ __launch_bounds__(64 * kWavesM * kWavesN) void gemm_bf16_256(Params p) {
  constexpr int kThreads = 64 * kWavesM * kWavesN;
  constexpr int kFM = kBM / kWavesM / 32, kFN = kBN / kWavesN / 32;  // fragments per wave
  __shared__ __attribute__((aligned(1024))) char smem[2 * kStageBytes];
  // With 4 waves the accumulators fill all 256 AGPRs and the k loop's
  // fragments most of the VGPRs, so nothing is prefetched into registers
  // before the loop: the ReluGrad mask words of the tile (256 rows x 8 words)
  // are copied into LDS of their own with the first k-tile.
  constexpr bool kMaskLds = EP == kEpReluGradBits && kWavesM * kWavesN == 4;
  __shared__ uint32_t mask_lds[kMaskLds ? kBM * (kBN / 32) : 1];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / kWavesN, wn = wave % kWavesN;
  constexpr int kWTM = kBM / kWavesM, kWTN = kBN / kWavesN;  // wave tile
  const int half = lane >> 5, l32 = lane & 31;
  int tm, tn;
  int bid = blockIdx.x, split = 0;
  if (p.splits > 1) {
    const int tiles = p.tiles_m * p.tiles_n;
    split = bid / tiles;
    bid -= split * tiles;
  }
  tile_of_block(bid, p.tiles_m, p.tiles_n, p.group_m, tm, tn);
  const int m0 = tm * kBM, n0 = tn * kBN;
  if constexpr (kMaskLds) {
    // one dword per lane: instruction j of a wave covers rows 8 b .. 8 b + 7
    // (b = wave * 8 + j), lane i row 8 b + i / 8, word i % 8; the prologue's
    // wait for the first k-tile covers these copies too
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int b = wave * 8 + j;
      const uint32_t* g = p.mask_in + (int64_t)(m0 + 8 * b + (lane >> 3)) * p.ldm + (n0 >> 5) + (lane & 7);
      __builtin_amdgcn_global_load_lds(g, (lds_void*)(mask_lds + 64 * b), 4, 0, 0);
    }
  }
  // The epilogue op: fixed by the fused epilogues (mask out: bias + ReLU;
  // squared error: bias; ReluGrad: none), else read from p.epi. The bias
  // values of this lane's columns are fetched before the k loop so that
  // their latency hides behind the first copies (with 4 waves, whose 256
  // accumulators per lane leave no registers to spare, in the epilogue).
  constexpr int kFixedOp = EP == kEpMaskOut                             ? 2
                           : EP == kEpLoss                              ? 1
                           : (EP == kEpReluGrad || EP == kEpReluGradBits) ? 0
                                                                          : -1;
  const int op = kFixedOp >= 0 ? kFixedOp : (p.epi & kEpiOpMask);
  constexpr bool kEarlyBias = kWavesM * kWavesN >= 8;
  float bias_v[kFN];
  auto load_bias = [&]() {
#pragma unroll
    for (int j = 0; j < kFN; ++j) bias_v[j] = op != 0 ? p.bias[n0 + wn * kWTN + j * 32 + l32] : 0.0f;
  };
  if constexpr (kEarlyBias) load_bias();

  f32x16 acc[kFM][kFN];
#pragma unroll
  for (int i = 0; i < kFM; ++i)
#pragma unroll
    for (int j = 0; j < kFN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  // this workgroup's k-tiles: kt0 .. kt0 + kt_count - 1
  const int kt0 = split * p.kt_per;
  const int kt_count = min(p.k / kBK - kt0, p.kt_per);
  if constexpr (kWavesM * kWavesN == 4) {
    // One wave per SIMD (128 x 128 wave tiles: 128 KiB of fragment reads per
    // k-tile instead of 192 KiB with 8 waves and 256 KiB with 16), for every
    // layout, on 16 x 16 x 32 MFMAs: 8 x 8 accumulator blocks of 16 x 16 per
    // wave, two k-steps of 32 per k-tile, 64 MFMAs per k-step. A single wave
    // must keep its matrix core busy, so the schedule is explicit: in every
    // k-step, the LDS reads of the next k-step's 16 fragments one after every
    // second MFMA of the first 32 (their latency then hides behind the last
    // 32), and in k-step 1 the copies of the k-tile after next spread one pair
    // per eight MFMAs. The k-tile barrier sits between the two k-steps: by
    // then every wave holds k-step 1's fragments in registers and its copies
    // of the next k-tile have landed, so k-step 1's MFMAs run behind the
    // barrier while the next k-tile's first fragments are read and the copies
    // of the k-tile after it go into the stage just released. Everything that
    // varies per copy or read is a scalar or an immediate: copies take a
    // wave-uniform base address (SGPRs) plus a per-lane 32-bit offset fixed
    // for the whole loop, and the loop is unrolled over the two LDS stages,
    // whose offsets become immediates.
    // K-slots: lane l of 16-lane group g = l / 16 supplies k = 32 q + 8 c(g)
    // + e, e = 0..7, in k-step q of a k-tile (both operands), c(g) = 0, 2, 1, 3:
    // the two groups of a half-wave, whose LDS reads are served together, then
    // read 16-byte chunks two apart of the same rows (k-contiguous operand) or
    // k-rows 16 apart (m/n-contiguous), which puts them in different banks.
    // LDS: A of stage s at s * 32 KiB, B of stage s at 64 KiB + s * 32 KiB.
    f32x4 acc16[8][8];
#pragma unroll
    for (int a = 0; a < 8; ++a)
#pragma unroll
      for (int b = 0; b < 8; ++b) {
        acc16[a][b] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
        asm volatile("" : "+a"(acc16[a][b]));
      }
    mfma16_settle(acc16);
    const int wv = __builtin_amdgcn_readfirstlane(wave);  // wave-uniform: LDS bases go to M0 directly
    uint32_t offa[8], offb[8];  // per-lane byte offsets of copy instruction j, both operands
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int blk = wv * 8 + j;
      if constexpr (A_KC) {
        const int r = blk * 8 + (lane >> 3);
        offa[j] = (uint32_t)(((int64_t)r * p.lda + (((lane & 7) ^ swz_kc(r)) * 8)) * 2);
      } else {
        const int kr = blk * 2 + (lane >> 5);
        offa[j] = (uint32_t)(((int64_t)kr * p.lda + (((lane & 31) ^ swz_mn(kr)) * 8)) * 2);
      }
      if constexpr (B_KC) {
        const int r = blk * 8 + (lane >> 3);
        offb[j] = (uint32_t)(((int64_t)r * p.ldb + (((lane & 7) ^ swz_kc(r)) * 8)) * 2);
      } else {
        const int kr = blk * 2 + (lane >> 5);
        offb[j] = (uint32_t)(((int64_t)kr * p.ldb + (((lane & 31) ^ swz_mn(kr)) * 8)) * 2);
      }
    }
    // wave-uniform operand base of k-tile kt (absolute). The loop copies
    // ahead without conditions: past the last k-tile it copies the last one
    // again, into a stage that is not read any more.
    const int kt_last = kt0 + kt_count - 1;
    auto abase = [&](int kt_abs) -> const char* {
      kt_abs = min(kt_abs, kt_last);
      return reinterpret_cast<const char*>(A_KC ? p.a + (int64_t)m0 * p.lda + (int64_t)kt_abs * kBK
                                                : p.a + (int64_t)kt_abs * kBK * p.lda + m0);
    };
    auto bbase = [&](int kt_abs) -> const char* {
      kt_abs = min(kt_abs, kt_last);
      return reinterpret_cast<const char*>(B_KC ? p.b + (int64_t)n0 * p.ldb + (int64_t)kt_abs * kBK
                                                : p.b + (int64_t)kt_abs * kBK * p.ldb + n0);
    };
    auto a_lds = [&](int stage) { return smem + stage * kOperandBytes; };
    auto b_lds = [&](int stage) { return smem + 2 * kOperandBytes + stage * kOperandBytes; };
    auto copy_pair = [&](const char* ga, const char* gb, int stage, int j) {
      // the empty asm keeps the 32-bit offsets from being widened outside the
      // loop, so that the copies use the scalar-base form (SGPR pair + VGPR)
      uint32_t oa = offa[j], ob = offb[j];
      asm("" : "+v"(oa), "+v"(ob));
      __builtin_amdgcn_global_load_lds(ga + oa, (lds_void*)(a_lds(stage) + (wv * 8 + j) * 1024), 16, 0, 0);
      __builtin_amdgcn_global_load_lds(gb + ob, (lds_void*)(b_lds(stage) + (wv * 8 + j) * 1024), 16, 0, 0);
    };
    // Per-lane LDS read addresses of stage 0; the stage, the k-step and the
    // fragment index enter as immediate offsets where the layout allows.
    // k-contiguous operand (256 rows of 128 B, chunk c of row r at slot
    // c ^ swz_kc(r)): fragment f of k-step q reads rows R + 16 f + l % 16,
    // chunk 4 q + c(g); rows 64 apart share the swizzle, so an address per
    // (q, f mod 4) and +8 KiB for f >= 4. m/n-contiguous operand (64 k-rows of
    // 512 B): lane l of 16-lane group g supplies k-row 8 c(g) + (l % 16) / 4
    // and four columns 4 (l % 4).. of the fragment's 16; the k-step and the
    // half of the transposing pair move the k-row by 32 q + 4 h, an immediate
    // (the swizzle does not see those bits); an address per fragment.
    const int g16 = lane >> 4, l16 = lane & 15;
    const int cg = ((g16 & 1) << 1) | (g16 >> 1);  // c(g)
    auto kc_addr = [&](const char* base_lds, int wbase, int q, int f4) -> uint32_t {
      const int r = wbase + f4 * 16 + l16;
      return (uint32_t)(uintptr_t)((lds_void*)(base_lds + r * 128 + (((4 * q + cg) ^ swz_kc(r)) << 4)));
    };
    auto mn_addr = [&](const char* base_lds, int wbase, int f) -> uint32_t {
      const int mn = wbase + f * 16 + 4 * (l16 & 3);
      const int kr0 = 8 * cg + (l16 >> 2);
      return (uint32_t)(uintptr_t)((lds_void*)(base_lds + kr0 * 512 + (((mn >> 3) ^ swz_mn(kr0)) << 4) + (mn & 7) * 2));
    };
    uint32_t ra[8], rb[8];
#pragma unroll
    for (int x = 0; x < 8; ++x) {
      ra[x] = A_KC ? kc_addr(a_lds(0), wm * kWTM, x >> 2, x & 3) : mn_addr(a_lds(0), wm * kWTM, x);
      rb[x] = B_KC ? kc_addr(b_lds(0), wn * kWTN, x >> 2, x & 3) : mn_addr(b_lds(0), wn * kWTN, x);
    }
    // read fragment F (0..7) of an operand, k-step Q of stage S, into a buffer
    auto read_frag_into = [&](auto f_tag, auto q_tag, auto s_tag, auto& buf, const uint32_t (&ra_)[8]) {
      constexpr int F = decltype(f_tag)::value, Q = decltype(q_tag)::value, S = decltype(s_tag)::value;
      if constexpr (std::is_same<std::decay_t<decltype(buf)>, FragBuf<true>>::value)
        ds_read_b128_into<(F >> 2) * 8192 + S * kOperandBytes>(buf.f[F], ra_[Q * 4 + (F & 3)]);
      else
        ds_read_tr_pair_into<(32 * Q) * 512 + S * kOperandBytes, (32 * Q + 4) * 512 + S * kOperandBytes>(
            buf.lo[F], buf.hi[F], ra_[F]);
    };
    using T_ = std::true_type;
    using F_ = std::false_type;
    FragBuf<A_KC> fa0, fa1;
    FragBuf<B_KC> fb0, fb1;
    // k-step: 64 MFMAs on (fa, fb), A block a = i % 8 by B block b = i / 8
    // (0.3 % faster in the step than the A-major order). After MFMA 2 r
    // (r < 16) the read of the next k-step's fragment r (B 0..7, then A 0..7;
    // k-step RQ of stage RS; kRead): fragment B b was last read by MFMA 8 b + 7
    // of the previous k-step and A a by MFMA 56 + a, so at least 15 MFMAs lie
    // between an MFMA's last read of a fragment register and the LDS read that
    // overwrites it. After MFMAs 1, 9, .., 57 one copy pair each (kCopy).
    auto kstep = [&](auto read_tag, auto copy_tag, auto rq_tag, auto rs_tag, auto& fa, auto& fb, auto& na, auto& nb,
                     const char* ga, const char* gb, int cstage) {
      constexpr bool kRead = decltype(read_tag)::value, kCopy = decltype(copy_tag)::value;
      static_for<64>([&](auto i_tag) {
        constexpr int i = decltype(i_tag)::value;
        mfma16_acc(acc16[i & 7][i >> 3], fa.template get<(i & 7)>(), fb.template get<(i >> 3)>());
        if constexpr (kRead && (i & 1) == 0 && i < 32) {
          constexpr int r = i >> 1;
          if constexpr (r < 8)
            read_frag_into(std::integral_constant<int, r>{}, rq_tag, rs_tag, nb, rb);
          else
            read_frag_into(std::integral_constant<int, r - 8>{}, rq_tag, rs_tag, na, ra);
        }
        if constexpr (kCopy && (i & 7) == 1) copy_pair(ga, gb, cstage, i >> 3);
      });
    };
    using Q0 = std::integral_constant<int, 0>;
    using Q1 = std::integral_constant<int, 1>;
    // One k-tile in stage S. Every k-tile runs the same code, so the loop has
    // no tail: at a join after differently compiled tails the compiler moves
    // all 256 accumulators between register files and spills. Past the last
    // k-tile the reads and copies only touch a stage that no MFMA reads again.
    auto ktile = [&](auto stage_tag, int kt) {
      constexpr int S = decltype(stage_tag)::value;
      using SN = std::integral_constant<int, 1 - S>;
      kstep(T_{}, F_{}, Q1{}, stage_tag, fa0, fb0, fa1, fb1, nullptr, nullptr, 0);
      // the k-tile barrier: k-step 1's fragments are in registers, this
      // wave's copies of the next k-tile have landed
      wait_lds(fa1, fb1, true);
      __builtin_amdgcn_s_barrier();
      kstep(T_{}, T_{}, Q0{}, SN{}, fa1, fb1, fa0, fb0, abase(kt0 + kt + 2), bbase(kt0 + kt + 2), S);
      // The next k-tile's first fragments are waited for here, at the end of
      // the k-tile and not at the start of the next: no read is in flight
      // across a branch, where the compiler may move registers around.
      wait_lds(fa0, fb0, false);
    };
    using S0 = std::integral_constant<int, 0>;
    using S1 = std::integral_constant<int, 1>;
    // Two k-tiles per trip, stage 0 then stage 1. An odd count starts at
    // k-tile -1: stage 0 filled with zeros, whose products add exact zeros.
    int kt = (kt_count & 1) ? -1 : 0;
    // prologue: k-tile kt in stage 0, its first fragments, and k-tile kt + 1's
    // copies into stage 1
    if (kt == 0) {
#pragma unroll
      for (int j = 0; j < 8; ++j) copy_pair(abase(kt0), bbase(kt0), 0, j);
    } else {
      const u32x4 z = {0u, 0u, 0u, 0u};
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        *reinterpret_cast<u32x4*>(a_lds(0) + (j * kThreads + tid) * 16) = z;
        *reinterpret_cast<u32x4*>(b_lds(0) + (j * kThreads + tid) * 16) = z;
      }
    }
    __builtin_amdgcn_s_waitcnt(0);
    __builtin_amdgcn_s_barrier();
    static_for<8>([&](auto f_tag) {
      read_frag_into(f_tag, Q0{}, S0{}, fa0, ra);
      read_frag_into(f_tag, Q0{}, S0{}, fb0, rb);
    });
#pragma unroll
    for (int j = 0; j < 8; ++j) copy_pair(abase(kt0 + kt + 1), bbase(kt0 + kt + 1), 1, j);
    wait_lds(fa0, fb0, false);
    for (; kt < kt_count; kt += 2) {
      ktile(S0{}, kt);
      ktile(S1{}, kt + 1);
    }
    __builtin_amdgcn_s_waitcnt(0);
    mfma16_settle(acc16);
    // into the 32 x 32 accumulator layout the epilogue takes
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const f32x4 x0[2] = {acc16[2 * i][2 * j], acc16[2 * i + 1][2 * j]};
        const f32x4 x1[2] = {acc16[2 * i][2 * j + 1], acc16[2 * i + 1][2 * j + 1]};
        acc[i][j] = acc16_to_32(x0, x1);
      }
  } else {
  copy_tile<A_KC, kThreads>(p.a, p.lda, m0, kt0 * kBK, smem, wave, lane);
  copy_tile<B_KC, kThreads>(p.b, p.ldb, n0, kt0 * kBK, smem + kOperandBytes, wave, lane);
  __builtin_amdgcn_s_waitcnt(0);  // vmcnt(0) lgkmcnt(0)
  __syncthreads();

  u32x4 fa[2][kFM], fb[2][kFN];
#pragma unroll
  for (int i = 0; i < kFM; ++i) fa[0][i] = read_frag<A_KC>(smem, wm * kWTM + i * 32, 0, lane);
#pragma unroll
  for (int j = 0; j < kFN; ++j) fb[0][j] = read_frag<B_KC>(smem + kOperandBytes, wn * kWTN + j * 32, 0, lane);

  for (int kt = 0; kt < kt_count; ++kt) {
    const char* st = smem + (kt & 1) * kStageBytes;
    char* nx = smem + ((kt + 1) & 1) * kStageBytes;
    const bool more = kt + 1 < kt_count;
    if (more) {
      copy_tile<A_KC, kThreads>(p.a, p.lda, m0, (kt0 + kt + 1) * kBK, nx, wave, lane);
      copy_tile<B_KC, kThreads>(p.b, p.ldb, n0, (kt0 + kt + 1) * kBK, nx + kOperandBytes, wave, lane);
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int cb = q & 1, nb = cb ^ 1;
      if constexpr (!A_KC || !B_KC) {
        // this k-step's fragments include transposing (inline assembly) reads
#pragma unroll
        for (int i = 0; i < kFM; ++i) frag_wait(fa[cb][i]);
#pragma unroll
        for (int j = 0; j < kFN; ++j) frag_wait(fb[cb][j]);
      }
      if (q < 3) {
#pragma unroll
        for (int i = 0; i < kFM; ++i) fa[nb][i] = read_frag<A_KC>(st, wm * kWTM + i * 32, q + 1, lane);
#pragma unroll
        for (int j = 0; j < kFN; ++j) fb[nb][j] = read_frag<B_KC>(st + kOperandBytes, wn * kWTN + j * 32, q + 1, lane);
      }
#pragma unroll
      for (int i = 0; i < kFM; ++i)
#pragma unroll
        for (int j = 0; j < kFN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, fa[cb][i]),
                                                              __builtin_bit_cast(bf16x8, fb[cb][j]),
                                                              acc[i][j], 0, 0, 0);
      // Interleave the next k-step's fragment reads between this k-step's
      // MFMAs so their latency hides behind the matrix cores. LDS read
      // instructions per k-step: 4 per k-contiguous operand (ds_read_b128),
      // 8 per m/n-contiguous one (two transposing reads).
      if (q < 3) interleave_mfma_reads<0, kFM * (A_KC ? 1 : 2) + kFN * (B_KC ? 1 : 2), kFM * kFN>();
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (more) {
#pragma unroll
      for (int i = 0; i < kFM; ++i) fa[0][i] = read_frag<A_KC>(nx, wm * kWTM + i * 32, 0, lane);
#pragma unroll
      for (int j = 0; j < kFN; ++j) fb[0][j] = read_frag<B_KC>(nx + kOperandBytes, wn * kWTN + j * 32, 0, lane);
    }
  }
  }  // k loop of 8 or 16 waves

  if constexpr (!kEarlyBias) load_bias();
  const bool trunc16 = (p.epi & kEpiTrunc16) != 0;
  if constexpr (sizeof(OutT) == 2) {
    // 16-bit output: the rounded tile goes through LDS (row-major, 16-byte
    // chunks XOR-swizzled so that both the fragment-layout writes and the
    // row-chunk reads are free of bank conflicts), then leaves in coalesced
    // 16-byte row chunks. The k loop's last barrier has passed, but waves may
    // still be reading their last fragments: wait for all of them first.
    constexpr int kRowStep = kThreads / 32;
    constexpr int kRowIters = kBM / kRowStep;
    const int cc = tid & 31;  // 16-byte chunk of a row: columns 8cc .. 8cc+7
    // ReLU mask words of this thread's rows, fetched before the staging so
    // their latency overlaps it; the byte (cc & 3) of a word covers the chunk.
    uint32_t mw[EP == kEpReluGradBits && !kMaskLds ? kRowIters : 1];
    if constexpr (EP == kEpReluGradBits && !kMaskLds) {
#pragma unroll
      for (int it = 0; it < kRowIters; ++it)
        mw[it] = p.mask_in[(int64_t)(m0 + (tid >> 5) + it * kRowStep) * p.ldm + (n0 >> 5) + (cc >> 2)];
    }
    // Likewise the target chunks of the squared-error epilogue (16 bytes per
    // row of this thread: 64 registers with 8 waves, 128 with 4, where the
    // k loop's fragment registers are free by now; the 4-wave output layer
    // 0.516 -> 0.503 ms against loading them in the read-out).
    u32x4 tv[EP == kEpLoss ? kRowIters : 1];
    if constexpr (EP == kEpLoss) {
#pragma unroll
      for (int it = 0; it < kRowIters; ++it)
        tv[it] = *reinterpret_cast<const u32x4*>(p.target + (int64_t)(m0 + (tid >> 5) + it * kRowStep) * p.n + n0 +
                                                 8 * cc);
    }
    __syncthreads();
    char* tile = smem;  // 256 rows x 512 bytes
    // Staging. Accumulator registers r, r + 1 (r even) of a lane are rows R,
    // R + 1 of its column: one packed conversion rounds both, and the two
    // halves go to LDS as 16-bit writes. The epilogue op and the rounding
    // are uniform, so they select one of six copies of this loop instead of
    // being tested per element.
    //
    // With kEpMaskOut the ReLU mask comes from wave ballots of the rounded
    // values: the 64 lanes of a staging step hold 32 consecutive columns of
    // rows R (lanes 0-31) and R + 4 (lanes 32-63), so the ballot of "16-bit
    // value > 0" over one half of the packed words is the two rows' mask
    // words. They are gathered into registers (row rho of the wave tile,
    // column word j: register rho / kRowsPerReg, lane kFN (rho % kRowsPerReg)
    // + j) and stored after the staging.
    constexpr int kRowsPerReg = 64 / kFN;
    uint32_t mk[EP == kEpMaskOut ? kWTM / kRowsPerReg : 1];
#pragma unroll
    for (int e = 0; e < (int)(sizeof(mk) / sizeof(mk[0])); ++e) mk[e] = 0;
    auto stage = [&](auto op_tag, auto trunc_tag) {
      constexpr int kOp = decltype(op_tag)::value;
      constexpr bool kTrunc = decltype(trunc_tag)::value;
#pragma unroll
      for (int j = 0; j < kFN; ++j) {
        const int col = wn * kWTN + j * 32 + l32;
#pragma unroll
        for (int i = 0; i < kFM; ++i) {
#pragma unroll
          for (int r = 0; r < 16; r += 2) {
            const int q = i * 32 + 8 * (r >> 2) + (r & 3);  // wave-tile row R - 4 half
            const int row = wm * kWTM + q + 4 * half;
            float v0 = acc[i][j][r], v1 = acc[i][j][r + 1];
            if constexpr (kOp != 0) {
              v0 += bias_v[j];
              v1 += bias_v[j];
            }
            if constexpr (kOp == 2) {
              v0 = relu_f32(v0);
              v1 = relu_f32(v1);
            }
            const uint32_t w = pack_bf16x2<kTrunc>(v0, v1);
            *reinterpret_cast<uint16_t*>(tile + epi_off(row, col)) = (uint16_t)w;
            *reinterpret_cast<uint16_t*>(tile + epi_off(row + 1, col)) = (uint16_t)(w >> 16);
            if constexpr (EP == kEpMaskOut) {
              const uint64_t b0 = __builtin_amdgcn_ballot_w64((int16_t)(w & 0xFFFFu) > 0);  // rows R, R + 4
              const uint64_t b1 = __builtin_amdgcn_ballot_w64((int16_t)(w >> 16) > 0);      // rows R + 1, R + 5
              const uint32_t words[4] = {(uint32_t)b0, (uint32_t)b1, (uint32_t)(b0 >> 32), (uint32_t)(b1 >> 32)};
              constexpr int kDq[4] = {0, 1, 4, 5};
#pragma unroll
              for (int t = 0; t < 4; ++t) {
                const int rho = q + kDq[t];
                mk[rho / kRowsPerReg] =
                    (uint32_t)tfd_writelane((int)words[t], kFN * (rho % kRowsPerReg) + j, (int)mk[rho / kRowsPerReg]);
              }
            }
          }
        }
      }
    };
    auto stage_op = [&](auto op_tag) {
      if (trunc16)
        stage(op_tag, std::true_type{});
      else
        stage(op_tag, std::false_type{});
    };
    if constexpr (kFixedOp >= 0)
      stage_op(std::integral_constant<int, kFixedOp>{});
    else if (op == 2)
      stage_op(std::integral_constant<int, 2>{});
    else if (op == 1)
      stage_op(std::integral_constant<int, 1>{});
    else
      stage_op(std::integral_constant<int, 0>{});
    if constexpr (EP == kEpMaskOut) {
#pragma unroll
      for (int e = 0; e < kWTM / kRowsPerReg; ++e) {
        const int rho = e * kRowsPerReg + lane / kFN;
        p.mask_out[(int64_t)(m0 + wm * kWTM + rho) * p.ldm + ((n0 + wn * kWTN) >> 5) + lane % kFN] = mk[e];
      }
    }
    __syncthreads();
    float cs[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) cs[e] = 0.0f;
    double sq = 0.0;
#pragma unroll
    for (int it = 0; it < kRowIters; ++it) {
      const int row = (tid >> 5) + it * kRowStep;
      u32x4 v = *reinterpret_cast<const u32x4*>(tile + epi_off(row, 8 * cc));
      const int64_t at = (int64_t)(m0 + row) * p.n + n0 + 8 * cc;  // contiguous side buffers
      if constexpr (EP == kEpLoss) {
        const u32x4 t = tv[it];
        u32x4 g;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float d0 = bf16_bits_to_f32(v[e] & 0xFFFFu) - bf16_bits_to_f32(t[e] & 0xFFFFu);
          const float d1 = bf16_bits_to_f32(v[e] >> 16) - bf16_bits_to_f32(t[e] >> 16);
          sq += (double)d0 * (double)d0;
          sq += (double)d1 * (double)d1;
          const uint32_t g0 = bf16_bits(d0), g1 = bf16_bits(d1);
          g[e] = g0 | (g1 << 16);
          cs[2 * e] += bf16_bits_to_f32(g0);
          cs[2 * e + 1] += bf16_bits_to_f32(g1);
        }
        store_stream(p.grad + at, g);
      }
      if constexpr (EP == kEpReluGrad) {
        // ReluGrad: keep the value where the stored feature is > 0, +0
        // elsewhere; sum the kept values per column
        const u32x4 f = *reinterpret_cast<const u32x4*>(p.features + (int64_t)(m0 + row) * p.ldf + n0 + 8 * cc);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint32_t lo = bf16_bits_to_f32(f[e] & 0xFFFFu) > 0.0f ? (v[e] & 0xFFFFu) : 0u;
          const uint32_t hi = bf16_bits_to_f32(f[e] >> 16) > 0.0f ? (v[e] & 0xFFFF0000u) : 0u;
          v[e] = lo | hi;
          cs[2 * e] += bf16_bits_to_f32(lo);
          cs[2 * e + 1] += bf16_bits_to_f32(hi >> 16);
        }
      }
      if constexpr (EP == kEpReluGradBits) {
        uint32_t word;
        if constexpr (kMaskLds)
          word = mask_lds[row * (kBN / 32) + (cc >> 2)];
        else
          word = mw[it];
        const uint32_t bits = word >> (8 * (cc & 3));
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint32_t lo = (bits >> (2 * e)) & 1u ? (v[e] & 0xFFFFu) : 0u;
          const uint32_t hi = (bits >> (2 * e + 1)) & 1u ? (v[e] & 0xFFFF0000u) : 0u;
          v[e] = lo | hi;
          cs[2 * e] += bf16_bits_to_f32(lo);
          cs[2 * e + 1] += bf16_bits_to_f32(hi >> 16);
        }
      }
      store_stream(static_cast<uint16_t*>(p.c) + (int64_t)(m0 + row) * p.ldc + n0 + 8 * cc, v);
    }
    if constexpr (EP == kEpReluGrad || EP == kEpReluGradBits || EP == kEpLoss) {
      // column sums: each thread's rows, then the kRowStep threads of a
      // chunk in row-group order (a fixed order)
      __syncthreads();
      float* red = reinterpret_cast<float*>(smem);  // [kRowStep][256]
#pragma unroll
      for (int e = 0; e < 8; ++e) red[(tid >> 5) * kBN + 8 * cc + e] = cs[e];
      if constexpr (EP == kEpLoss) {
        double* dred = reinterpret_cast<double*>(smem + kRowStep * kBN * 4);  // [kThreads]
        dred[tid] = sq;
      }
      __syncthreads();
      for (int c = tid; c < kBN; c += kThreads) {
        float t = 0.0f;
#pragma unroll
        for (int g = 0; g < kRowStep; ++g) t += red[g * kBN + c];
        p.col_partial[(int64_t)tm * p.n + n0 + c] = t;
      }
      if constexpr (EP == kEpLoss) {
        // wave 0: lane i adds dred[i], dred[i + 64], ... in order, then a
        // butterfly over the 64 lanes (a fixed pattern)
        if (wave == 0) {
          const double* dred = reinterpret_cast<const double*>(smem + kRowStep * kBN * 4);
          double t = 0.0;
#pragma unroll
          for (int i = 0; i < kThreads / 64; ++i) t += dred[lane + 64 * i];
#pragma unroll
          for (int o = 32; o > 0; o >>= 1) t += __shfl_xor(t, o, 64);
          if (lane == 0) p.loss_partial[(int64_t)tm * p.tiles_n + tn] = t;
        }
      }
    }
    return;
  } else {
    OutT* C = static_cast<OutT*>(p.c) + (int64_t)split * p.m * p.ldc;
#pragma unroll
    for (int j = 0; j < kFN; ++j) {
      const int col = n0 + wn * kWTN + j * 32 + l32;
      const float bv = bias_v[j];
#pragma unroll
      for (int i = 0; i < kFM; ++i) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = m0 + wm * kWTM + i * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
          float v = acc[i][j][r] + bv;
          if (op == 2) v = relu_f32(v);
          __builtin_nontemporal_store(v, &C[(int64_t)row * p.ldc + col]);
        }
      }
    }
  }
}

template <bool A_KC, bool B_KC, int WM, int WN>
hipError_t launch(const GemmDesc& d, hipStream_t s) {
  Params p;
  p.a = static_cast<const bf16*>(d.a);
  p.b = static_cast<const bf16*>(d.b);
  p.c = d.c;
  p.bias = d.bias;
  p.lda = d.lda;
  p.ldb = d.ldb;
  p.ldc = d.ldc;
  p.m = (int)d.m;
  p.n = (int)d.n;
  p.k = (int)d.k;
  p.epi = d.epi;
  p.tiles_m = p.m / kBM;
  p.tiles_n = p.n / kBN;
  p.features = static_cast<const uint16_t*>(d.features);
  p.ldf = d.ldf;
  p.col_partial = d.col_partial;
  p.target = static_cast<const uint16_t*>(d.target);
  p.grad = static_cast<uint16_t*>(d.grad);
  p.loss_partial = d.loss_partial;
  p.mask_in = d.mask_in;
  p.mask_out = d.mask_out;
  p.ldm = d.ldm;
  p.splits = d.splits > 1 ? d.splits : 1;
  p.kt_per = p.splits > 1 ? (int)d.kt_per : p.k / kBK;
  // bands of 8 tile-rows; 4 for the unsplit 4-wave NT products (the input
  // gradients of the 4096-wide step: 0.416 vs 0.423 ms inside it, while the
  // NN forward and TN weight gradients are fastest with 8)
  p.group_m = (A_KC && B_KC && WM * WN == 4 && p.splits == 1) ? 4 : 8;
  dim3 grid(p.tiles_m * p.tiles_n * p.splits), block(64 * WM * WN);
  if (p.splits > 1)  // fp32 partial tiles, plain (the reduction applies the epilogue)
    hipLaunchKernelGGL((gemm_bf16_256<A_KC, B_KC, float, WM, WN>), grid, block, 0, s, p);
  else if (d.mask_in)
    hipLaunchKernelGGL((gemm_bf16_256<A_KC, B_KC, bf16, WM, WN, kEpReluGradBits>), grid, block, 0, s, p);
  else if (d.mask_out)
    hipLaunchKernelGGL((gemm_bf16_256<A_KC, B_KC, bf16, WM, WN, kEpMaskOut>), grid, block, 0, s, p);
  else if (d.features)
    hipLaunchKernelGGL((gemm_bf16_256<A_KC, B_KC, bf16, WM, WN, kEpReluGrad>), grid, block, 0, s, p);
  else if (d.target)
    hipLaunchKernelGGL((gemm_bf16_256<A_KC, B_KC, bf16, WM, WN, kEpLoss>), grid, block, 0, s, p);
  else if (d.out_bf16)
    hipLaunchKernelGGL((gemm_bf16_256<A_KC, B_KC, bf16, WM, WN>), grid, block, 0, s, p);
  else
    hipLaunchKernelGGL((gemm_bf16_256<A_KC, B_KC, float, WM, WN>), grid, block, 0, s, p);
  return hipGetLastError();
}

// Waves per workgroup: 4 (2x2 of 128x128), 8 (2x4 of 128x64) or 16 (4x4 of 64x64).
template <bool A_KC, bool B_KC>
hipError_t launch_waves(const GemmDesc& d, int waves, hipStream_t s) {
  // the 4-wave loop keeps per-lane copy offsets below 2^31 bytes
  if (waves == 4 && d.lda < (1 << 22) && d.ldb < (1 << 22)) return launch<A_KC, B_KC, 2, 2>(d, s);
  if (waves == 16) return launch<A_KC, B_KC, 4, 4>(d, s);
  return launch<A_KC, B_KC, 2, 4>(d, s);
}

// Waves per workgroup of a layout: the tuning knob when set (4, 8 or 16),
// else the default.
int waves_for(TuneKnob knob, int dflt) {
  const int v = tuning(knob);
  return v ? v : dflt;
}

}  // namespace

namespace {

// Sum of the fp32 partial tiles of a split k range, in split order, then
// the epilogue (bias, ReLU) and the single rounding to the output type. One
// thread per 4 consecutive columns of a row.
template <typename OutT>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ ws, int splits, int64_t m,
                                                            int64_t n, OutT* __restrict__ c, int64_t ldc,
                                                            const float* __restrict__ bias, int epi) {
  const int64_t groups = n / 4;
  const int64_t total = m * groups;
  const int op = epi & kEpiOpMask;
  const bool trunc16 = (epi & kEpiTrunc16) != 0;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += (int64_t)gridDim.x * 256) {
    const int64_t r = i / groups, c4 = (i - r * groups) * 4;
    f32x4 v = *reinterpret_cast<const f32x4*>(ws + r * n + c4);
    for (int sp = 1; sp < splits; ++sp) {
      const f32x4 w = *reinterpret_cast<const f32x4*>(ws + ((int64_t)sp * m + r) * n + c4);
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] += w[e];
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float x = v[e];
      if (op != 0) x += bias[c4 + e];
      if (op == 2) x = relu_f32(x);
      store_from_f32(c + r * ldc + c4 + e, x, trunc16);
    }
  }
}

}  // namespace

#ifdef TFD_GEMM_BF16_TN_UNIT
// The TN layout (both operands m/n-contiguous, transposing reads), built from
// this file in a translation unit of its own (gemm_bf16_tn.hip) so that it
// can take its own machine-scheduler setting.
hipError_t launch_gemm_bf16_256_tn(const GemmDesc& d, hipStream_t s) {
  const int64_t kt = d.splits > 1 ? d.kt_per : d.k / kBK;
  return launch_waves<false, false>(d, waves_for(kTuneBf16WavesTN, kt >= 32 ? 4 : 16), s);
}
#else
int gemm_bf16_256_splits(const GemmDesc& d, int cus) {
  // split the k range when the output has fewer whole tiles than compute
  // units, keeping at least 8 k-tiles per split
  const int64_t tiles = (d.m / kBM) * (d.n / kBN);
  const int64_t kt = d.k / kBK;
  if (tiles <= 0 || tiles >= cus || d.n % 4 != 0) return 1;
  int64_t s = (cus + tiles - 1) / tiles;
  if (s > kt / 8) s = kt / 8;
  return s >= 2 ? (int)s : 1;
}

hipError_t launch_splitk_reduce(const float* ws, int splits, const GemmDesc& d, hipStream_t s) {
  const int64_t total = d.m * (d.n / 4);
  int64_t blocks = (total + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  if (d.out_bf16)
    hipLaunchKernelGGL((splitk_reduce_kernel<bf16>), (unsigned)blocks, 256, 0, s, ws, splits, d.m, d.n,
                       static_cast<bf16*>(d.c), d.ldc, d.bias, d.epi);
  else
    hipLaunchKernelGGL((splitk_reduce_kernel<float>), (unsigned)blocks, 256, 0, s, ws, splits, d.m, d.n,
                       static_cast<float*>(d.c), d.ldc, d.bias, d.epi);
  return hipGetLastError();
}

bool gemm_bf16_256_ok(const GemmDesc& d) {
  // a 16-bit C leaves in 16-byte row chunks (and so do ReluGrad features in)
  auto al = [](const void* q) { return (reinterpret_cast<uintptr_t>(q) & 15) == 0; };
  const bool c_ok = !d.out_bf16 || (al(d.c) && d.ldc % 8 == 0);
  const bool f_ok = !d.features || (al(d.features) && d.ldf % 8 == 0);
  const bool l_ok = !d.target || (al(d.target) && al(d.grad) && d.n % 8 == 0);
  // mask epilogues write or read whole words of 16-bit tiles
  const bool m_ok = (!d.mask_in && !d.mask_out) || (d.out_bf16 && d.ldm >= d.n / 32);
  return d.in_bf16 && d.m % kBM == 0 && d.n % kBN == 0 && d.k % kBK == 0 && d.k > 0 &&
         gemm_vector_ok(d, 2) && !(d.ta && d.tb) && c_ok && f_ok && l_ok && m_ok;
}

hipError_t launch_gemm_bf16_256(const GemmDesc& d, hipStream_t s) {
  // A is k-contiguous unless transposed; B is k-contiguous when transposed.
  // Defaults measured inside the training step (4096-wide layers, batch
  // 16384; 512 -> 32768 layer): the scheduled 4-wave loop (one wave per SIMD,
  // 128 x 128 wave tiles, 16 x 16 x 32 MFMAs) for long k ranges: NT forward
  // with mask 0.433 vs 0.480 ms with 8 waves, the squared-error output layer
  // 0.510 vs 0.520, NT input gradient with ReluGrad 0.430 vs 0.476, TN
  // weight gradient 0.365 vs 0.445 with 16 waves. With 8 k-tiles or fewer
  // per workgroup the epilogue dominates and 2 waves per SIMD overlap it
  // better (512 -> 32768 forward 0.64 vs 0.76 ms). NN the same way: the
  // 4096-wide forward on W (B m/n-contiguous) 0.414-0.436 ms on 4 waves.
  const int64_t kt = d.splits > 1 ? d.kt_per : d.k / kBK;
  const bool long_k = kt >= 32;
  if (!d.ta && !d.tb) return launch_waves<true, false>(d, waves_for(kTuneBf16WavesNN, long_k ? 4 : 8), s);
  if (!d.ta && d.tb) return launch_waves<true, true>(d, waves_for(kTuneBf16WavesNT, long_k ? 4 : 8), s);
  return launch_gemm_bf16_256_tn(d, s);
}
#endif

}  // namespace tfd
