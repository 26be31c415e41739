// Internal launch interface between the C ABI (api.cpp) and the kernels.
// Callers have validated every argument; launchers only pick a kernel
// variant and enqueue it on the given stream.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace tfd {

struct GemmDesc {
  bool ta, tb;
  int64_t m, n, k;
  const void* a;
  int64_t lda;
  const void* b;
  int64_t ldb;
  void* c;
  int64_t ldc;
  bool in_bf16, out_bf16;
  const float* bias;
  int epi;  // (epi & kEpiOpMask): 0 none, 1 bias, 2 bias + relu; kEpiTrunc16: truncating 16-bit output
  // ReluGrad epilogue (16-bit whole-tile kernel only): when features != NULL
  // the stored output is features > 0 ? C : +0, and each workgroup writes the
  // column sums of its stored tile to col_partial[tile_row * n + col].
  const void* features = nullptr;
  int64_t ldf = 0;
  float* col_partial = nullptr;
  // Squared-error epilogue (16-bit whole-tile kernel only): when target !=
  // NULL, grad = C - target (contiguous, ld = n) is stored as well, each
  // workgroup writes its tile's float64 sum of squared differences to
  // loss_partial[tile] and the column sums of its grad tile to col_partial.
  const void* target = nullptr;
  void* grad = nullptr;
  double* loss_partial = nullptr;
  // ReLU masks (16-bit whole-tile kernel only), one bit per element, row r
  // at word r * ldm: mask_in replaces features in the ReluGrad epilogue;
  // mask_out receives the bits of the stored output's > 0 test.
  const uint32_t* mask_in = nullptr;
  uint32_t* mask_out = nullptr;
  int64_t ldm = 0;
  // Split of the k range (16-bit whole-tile kernel only): `splits`
  // workgroups per output tile, kt_per 64-wide k-tiles each; c then receives
  // `splits` fp32 partial matrices (ldc = n), summed by launch_splitk_reduce.
  int splits = 1;
  int64_t kt_per = 0;
};

constexpr int kEpiOpMask = 3;
constexpr int kEpiTrunc16 = 16;

bool gemm_vector_ok(const GemmDesc& d, int elem_bytes);
hipError_t launch_gemm(const GemmDesc& d, hipStream_t s);
// Tuning knobs set through tfd_set_tuning (0: the library's own choice). The
// default dispatch never reads the environment.
enum TuneKnob { kTuneGemmTile = 0, kTuneBf16WavesNN, kTuneBf16WavesNT, kTuneBf16WavesTN, kTuneSmallWaves, kTuneCount };
int tuning(TuneKnob knob);
inline int gemm_tile_override() { return tuning(kTuneGemmTile); }
// 16-bit operands, whole 256 x 256 tiles, k a multiple of 64 (gemm_bf16.hip).
bool gemm_bf16_256_ok(const GemmDesc& d);
hipError_t launch_gemm_bf16_256(const GemmDesc& d, hipStream_t s);
// Its TN layout, compiled in gemm_bf16_tn.hip.
hipError_t launch_gemm_bf16_256_tn(const GemmDesc& d, hipStream_t s);
// Number of k splits worth using for a whole-tile 16-bit problem on `cus`
// compute units (1: none).
int gemm_bf16_256_splits(const GemmDesc& d, int cus);
// c = epilogue(sum of the `splits` fp32 partials in ws, in order), rounded once (d: the
// original problem: c, ldc, out type, bias, epi).
hipError_t launch_splitk_reduce(const float* ws, int splits, const GemmDesc& d, hipStream_t s);
// fp32 problems too small to fill the GPU with 128 x 128 tiles (gemm_small.hip).
bool gemm_small_preferred(const GemmDesc& d);
hipError_t launch_gemm_small_f32(const GemmDesc& d, hipStream_t s);

hipError_t launch_bias_add(const void* value, const float* bias, void* out, int64_t rows, int64_t cols,
                           bool bf16, hipStream_t s);
hipError_t launch_relu(const void* x, void* y, int64_t count, bool bf16, hipStream_t s);
hipError_t launch_relu_grad(const void* g, const void* f, void* out, int64_t count, bool bf16,
                            hipStream_t s);

// Column reduction with optional Relu mask (features) and optional masked
// output (backprops). Partial sums go to `ws` (reduction_ws_bytes).
size_t reduction_ws_bytes(int64_t rows, int64_t cols, bool bf16);
hipError_t launch_relu_grad_bias_add_grad(const void* g, const void* f, void* out, float* db,
                                          int64_t rows, int64_t cols, bool bf16, void* ws,
                                          hipStream_t s);
// The device array that the no-allocation entry point uses instead of a
// workspace: its capacity, and its address on the current device (looked up
// once per device).
size_t static_scratch_bytes();
hipError_t static_scratch(void** out);
// Engine clock probe: counters[0] = shader clock cycles, counters[1] = 100 MHz
// real-time ticks over the same run of `iterations` dependent FMAs.
hipError_t launch_clock_probe(uint64_t* counters, int64_t iterations, hipStream_t s);
// One training step of a small fp32 MLP in one persistent kernel (the
// layers' buffers as in tfd_mlp_step_desc; validated by the caller).
constexpr int kMlpMaxLayers = 4;
constexpr size_t kMlpCtlBytes = 4096;  // barrier words at the start of the workspace
struct MlpStep {
  int layers, cost, update;
  int persistent;  // one cooperative launch with grid barriers, else one launch per phase
  int64_t batch;
  int64_t fan_in[kMlpMaxLayers], fan_out[kMlpMaxLayers];
  int relu[kMlpMaxLayers];
  float* w[kMlpMaxLayers];
  float* b[kMlpMaxLayers];
  float* h[kMlpMaxLayers];
  float* dy[kMlpMaxLayers];
  float* dw[kMlpMaxLayers];
  float* db[kMlpMaxLayers];
  const float* x;
  float* dx0;
  float* g;
  const float* target;
  const int32_t* labels;
  double* loss;
  float lr;
};
size_t mlp_step_ws_bytes(int64_t batch, int64_t top_fan_in, int64_t classes, int cost);
hipError_t launch_mlp_step(const MlpStep& d, void* ws, hipStream_t s);
// The same with the Relu test read from a bit mask (rows x ldm words).
hipError_t launch_relu_mask_grad_bias_add_grad(const void* g, const uint32_t* mask, int64_t ldm, void* out,
                                               float* db, int64_t rows, int64_t cols, bool bf16, void* ws,
                                               hipStream_t s);
// mask[r * ldm + w] bit j = x[r * ldx + 32 w + j] > 0 (bits past cols are 0).
hipError_t launch_relu_mask(const void* x, int64_t ldx, uint32_t* mask, int64_t ldm, int64_t rows, int64_t cols,
                            bool bf16, hipStream_t s);

size_t loss_ws_bytes(int64_t count, bool bf16);
hipError_t launch_l2_loss_grad(const void* out, const void* target, void* grad, double* loss,
                               int64_t count, bool bf16, void* ws, hipStream_t s);
// loss = 1/2 * (sum of n float64 partials, fixed order) (elementwise.hip).
hipError_t launch_loss_final(const double* partial, int n, double* loss, hipStream_t s);

// Sums `chunks` row-chunk partials of each column in chunk order (reduce.hip).
hipError_t launch_colsum_final(const float* partial, float* db, int64_t chunks, int64_t cols, hipStream_t s);

size_t softmax_xent_ws_bytes(int64_t rows);
hipError_t launch_softmax_xent(const void* logits, const int32_t* labels, void* grad, double* loss, int64_t rows,
                               int64_t cols, bool bf16, void* ws, hipStream_t s);

hipError_t launch_sgd(float* var, float alpha, const float* delta, int64_t count, uint16_t* shadow, bool trunc,
                      hipStream_t s);
hipError_t launch_sgd_matrix(float* var, float alpha, const float* delta, int64_t rows, int64_t cols,
                             uint16_t* shadow, uint16_t* shadow_t, bool trunc, hipStream_t s);

hipError_t launch_convert_to_bf16(const float* src, uint16_t* dst, int64_t count, bool trunc, hipStream_t s);
hipError_t launch_convert_to_f32(const uint16_t* src, float* dst, int64_t count, hipStream_t s);

}  // namespace tfd
