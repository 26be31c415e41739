/*
 * libtfdense — the dense-layer training step of the TensorFlow white paper
 * (Abadi et al., 2015) as hand-written HIP kernels for AMD CDNA4 (gfx950).
 *
 * The paper's canonical example (Figure 1) trains Relu(W x + b). Its graph
 * uses the ops MatMul, Add and ReLU (section 2, Table 1); automatic
 * differentiation (section 4.1) adds their gradient functions; the
 * parameters live in Variables that the step updates in place (section 2,
 * "Variables"). This library exports one call per op on that path.
 *
 * Conventions shared by every call
 * --------------------------------
 *  - Matrices are 2-D, row-major. A leading dimension ("ld") is the distance
 *    in elements between consecutive rows and must be >= the row length.
 *  - Element types: TFD_F32 (IEEE binary32) and TFD_BF16 (the 16-bit float
 *    of section 5.5: binary32 with 16 fewer mantissa bits). Products are
 *    accumulated in fp32. Values stored as TFD_BF16 are rounded to nearest
 *    even, unless a call's tfd_rounding argument or TFD_EPI_TRUNCATE_16
 *    selects the truncating converter of section 5.5. Biases, bias
 *    gradients and Variables are always fp32.
 *  - Pointers are device pointers unless stated otherwise. The caller owns
 *    every buffer; the library allocates no device memory, keeps no state
 *    between calls (besides the tuning knobs of tfd_set_tuning) and never
 *    synchronises. Scratch memory is passed in as a
 *    "workspace" sized by the matching *_workspace_size call.
 *  - Every call enqueues its kernels on `stream` (a hipStream_t passed as
 *    void*; NULL is the null stream) and returns. Stream order is the only
 *    ordering: it plays the role of the paper's control dependencies
 *    (section 2), e.g. a weight gradient that must read W before the update
 *    writes it is simply enqueued first.
 *  - Errors: a call returns TFD_OK, or an error status before enqueuing
 *    anything (TFD_EINVAL: a NULL pointer with a non-zero size, a negative
 *    size, a leading dimension smaller than the row, a workspace too small,
 *    an aliasing the call forbids; TFD_EUNSUPPORTED: an element-type
 *    combination the call does not implement; TFD_EHIP: the HIP runtime
 *    rejected a launch). tfd_last_error() then holds a message (per host
 *    thread). No C++ exception crosses this interface. A fault inside a
 *    kernel surfaces at the caller's next synchronisation.
 *  - Sizes of zero are valid and enqueue nothing (except where stated).
 */
#ifndef TFDENSE_H
#define TFDENSE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define TFD_ABI_VERSION 5

#if defined(__GNUC__)
#define TFD_API __attribute__((visibility("default")))
#else
#define TFD_API
#endif

typedef enum tfd_status {
  TFD_OK = 0,
  TFD_EINVAL = 1,
  TFD_EUNSUPPORTED = 2,
  TFD_EHIP = 3
} tfd_status;

typedef enum tfd_dtype { TFD_F32 = 0, TFD_BF16 = 1 } tfd_dtype;

/* How an fp32 value becomes a 16-bit one.
 * TFD_ROUND_NEAREST_EVEN: to the nearest 16-bit value, ties to even (the
 *   default of every call).
 * TFD_ROUND_TRUNCATE: the lossy converter of section 5.5: the low 16 bits of
 *   the fp32 pattern are dropped (rounding toward zero; infinities and zeros
 *   keep their sign). A NaN becomes the quiet NaN 0x7FC0 with its sign, so
 *   that no NaN turns into an infinity. */
typedef enum tfd_rounding { TFD_ROUND_NEAREST_EVEN = 0, TFD_ROUND_TRUNCATE = 1 } tfd_rounding;

/* What the MatMul producer applies to the fp32 accumulator before the
 * single rounding to the output type. */
typedef enum tfd_epilogue {
  TFD_EPI_NONE = 0,      /* C = op(A) op(B)                                 */
  TFD_EPI_BIAS = 1,      /* C = op(A) op(B) + 1 bias^T        (Add, Fig. 1) */
  TFD_EPI_BIAS_RELU = 2, /* C = Relu(op(A) op(B) + 1 bias^T)  (Relu(Wx+b))  */
  /* Flag, OR-ed with one of the above: a 16-bit C is written with the
   * truncating converter (TFD_ROUND_TRUNCATE) instead of nearest even. */
  TFD_EPI_TRUNCATE_16 = 16
} tfd_epilogue;

TFD_API int tfd_abi_version(void);
TFD_API const char* tfd_status_string(tfd_status status);
/* Message of the last failed call on this host thread ("" if none). */
TFD_API const char* tfd_last_error(void);

/*
 * Tuning and testing only (not part of the paper's ops): force a kernel
 * configuration that the library would otherwise choose itself, so that
 * every configuration can be measured and parity-tested. The setting is
 * process-wide and lasts until it is set again; 0 restores the library's
 * own choice. The default dispatch reads neither these knobs' defaults nor
 * the environment from anywhere else. Knobs:
 *   "gemm_tile"      1..9: the tile configuration of the general MatMul
 *                    kernels (which also disables the 16-bit whole-tile
 *                    kernel and the k split);
 *   "bf16_waves_nn", "bf16_waves_nt", "bf16_waves_tn"
 *                    4, 8 or 16: waves per workgroup of the 16-bit
 *                    whole-tile MatMul for that layout;
 *   "small_waves"    4, 8 or 16: waves per tile of the small fp32 MatMul.
 * Returns TFD_EINVAL for an unknown knob or a value out of range. Calls that
 * are in flight on other host threads may see either setting.
 */
TFD_API tfd_status tfd_set_tuning(const char* knob, int value);

/*
 * MatMul (section 2, Table 1) with the op's transpose attributes, fused with
 * the broadcast bias Add and the ReLU of Figure 1:
 *   C[m x n] = epilogue( op(A)[m x k] * op(B)[k x n] ),
 *   op(A) = A^T if transpose_a (A stored k x m, lda >= m) else A (m x k, lda >= k),
 *   op(B) = B^T if transpose_b (B stored n x k, ldb >= k) else B (k x n, ldb >= n).
 * The three layouts of one dense layer's step: forward Y = X W (NN), input
 * gradient dX = dY W^T (transpose_b = 1) and weight gradient dW = X^T dY
 * (transpose_a = 1).
 * Types: (a, b, c) in {(F32, F32, F32), (BF16, BF16, BF16), (BF16, BF16, F32)};
 * fp32 accumulation. bias is fp32[n] (may be NULL only with TFD_EPI_NONE).
 * ReLU keeps values > 0 and writes +0 otherwise. k = 0 gives
 * C = epilogue(0). C must not overlap A, B or bias. Returns TFD_EUNSUPPORTED
 * for other type combinations and for transpose_a && transpose_b.
 */
TFD_API tfd_status tfd_matmul(int transpose_a, int transpose_b, int64_t m, int64_t n, int64_t k,
                      const void* a, int64_t lda, tfd_dtype a_type,
                      const void* b, int64_t ldb, tfd_dtype b_type,
                      void* c, int64_t ldc, tfd_dtype c_type,
                      const float* bias, tfd_epilogue epilogue, void* stream);

/*
 * tfd_matmul with a caller-owned workspace. The contract (arguments, types,
 * epilogue, rounding, errors) is tfd_matmul's. The workspace lets the library
 * split the reduction over k across several workgroups per output tile when
 * the output has too few 256 x 256 tiles to occupy every compute unit (16-bit
 * operands, m and n multiples of 256, k a multiple of 64): each split writes
 * fp32 partial sums to the workspace and a second kernel adds them in split
 * order, applies the epilogue and rounds once. The result then differs from
 * tfd_matmul's only in how the k sum is grouped, and is the same on every
 * call. With a workspace smaller than tfd_matmul_workspace_size (or NULL),
 * or one that overlaps an operand, the call is exactly tfd_matmul.
 */
TFD_API size_t tfd_matmul_workspace_size(int transpose_a, int transpose_b, int64_t m, int64_t n, int64_t k,
                                         tfd_dtype a_type, tfd_dtype b_type, tfd_dtype c_type);
TFD_API tfd_status tfd_matmul_with_workspace(int transpose_a, int transpose_b, int64_t m, int64_t n, int64_t k,
                                             const void* a, int64_t lda, tfd_dtype a_type,
                                             const void* b, int64_t ldb, tfd_dtype b_type,
                                             void* c, int64_t ldc, tfd_dtype c_type,
                                             const float* bias, tfd_epilogue epilogue,
                                             void* workspace, size_t workspace_bytes, void* stream);

/*
 * BiasAdd, the broadcast Add of Figure 1 on its own:
 *   out[r, c] = value[r, c] + bias[c], rows x cols, contiguous (ld = cols).
 * value/out in `type` (fp32 arithmetic, one rounding); bias fp32[cols].
 * out may equal value.
 */
TFD_API tfd_status tfd_bias_add(const void* value, const float* bias, void* out,
                        int64_t rows, int64_t cols, tfd_dtype type, void* stream);

/*
 * ReLU (Table 1): activations[i] = features[i] > 0 ? features[i] : +0,
 * `count` contiguous elements of `type`. activations may equal features.
 */
TFD_API tfd_status tfd_relu(const void* features, void* activations, int64_t count,
                    tfd_dtype type, void* stream);

/*
 * ReluGrad, the gradient function of ReLU (section 4.1):
 *   backprops[i] = features[i] > 0 ? gradients[i] : +0,
 * with `features` the stored forward output of the Relu. backprops may
 * equal gradients.
 */
TFD_API tfd_status tfd_relu_grad(const void* gradients, const void* features, void* backprops,
                         int64_t count, tfd_dtype type, void* stream);

/* Workspace bytes that tfd_bias_add_grad and tfd_relu_grad_bias_add_grad
 * need for a rows x cols input. */
TFD_API size_t tfd_reduction_workspace_size(int64_t rows, int64_t cols, tfd_dtype type);

/*
 * BiasAddGrad, the gradient of the broadcast Add with respect to the bias
 * (the db of section 4.1's tf.gradients(C, [b, W, x])):
 *   bias_grad[c] = sum_r out_backprop[r, c]   (fp32 out, fp32 partial sums).
 * The summation order is fixed by (rows, cols), so repeated calls give
 * identical bits. rows = 0 writes zeros.
 */
TFD_API tfd_status tfd_bias_add_grad(const void* out_backprop, float* bias_grad,
                             int64_t rows, int64_t cols, tfd_dtype type,
                             void* workspace, size_t workspace_bytes, void* stream);

/*
 * ReluGrad fused with BiasAddGrad in one pass over the gradient:
 *   d = features[r, c] > 0 ? gradients[r, c] : +0,
 *   backprops[r, c] = d (skipped when backprops is NULL),
 *   bias_grad[c] = sum_r d.
 * features == NULL means an identity layer (d = gradients). backprops must
 * not overlap gradients or features. Deterministic like tfd_bias_add_grad.
 */
TFD_API tfd_status tfd_relu_grad_bias_add_grad(const void* gradients, const void* features,
                                       void* backprops, float* bias_grad,
                                       int64_t rows, int64_t cols, tfd_dtype type,
                                       void* workspace, size_t workspace_bytes,
                                       void* stream);

/*
 * tfd_relu_grad_bias_add_grad for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): the same arguments without the workspace, the same kernels
 * and the same result bit for bit. The column partials go to a fixed device
 * array inside the library instead (4 MiB per GPU, held until the process
 * ends), so the call allocates nothing. Every call on a GPU uses that GPU's
 * one array: calls that overlap in time on one GPU (other streams, other
 * host threads) race and must not be issued. Shapes whose partials exceed
 * the array return TFD_EINVAL (every shape up to at least 2^31 elements fits:
 * the partials need at most about 2 MiB); TFD_EHIP if the array's address
 * cannot be looked up on the current device.
 */
TFD_API tfd_status tfd_relu_grad_bias_add_grad_noalloc(const void* gradients, const void* features, void* backprops,
                                                       float* bias_grad, int64_t rows, int64_t cols, tfd_dtype type,
                                                       void* stream);

/* Workspace bytes that tfd_matmul_relu_grad_bias_add_grad needs for an m x n output. */
TFD_API size_t tfd_matmul_relu_grad_workspace_size(int64_t m, int64_t n, tfd_dtype type);

/*
 * The input-gradient MatMul of a dense layer fused with the ReluGrad and
 * BiasAddGrad of the layer below it (section 4.1: the gradient flows through
 * the upper layer's MatMul into the lower layer's Relu and Add):
 *   G[r, c]         = (op(A) op(B))[r, c], fp32 accumulation, rounded once to
 *                     `type` (with `rounding` for 16-bit outputs); not stored,
 *   backprops[r, c] = features[r, c] > 0 ? G[r, c] : +0,
 *   bias_grad[c]    = sum_r backprops[r, c]   (fp32, in a fixed order).
 * Operands as in tfd_matmul (transpose flags, leading dimensions; A and B of
 * `type`); features and backprops are m x n of `type`, contiguous (ld = n).
 * backprops equals what tfd_matmul followed by tfd_relu_grad_bias_add_grad
 * stores, bit for bit; bias_grad may differ from that path in the order of
 * its sum. backprops must not overlap A, B, features, bias_grad or the
 * workspace. TFD_EUNSUPPORTED as for tfd_matmul.
 */
TFD_API tfd_status tfd_matmul_relu_grad_bias_add_grad(int transpose_a, int transpose_b, int64_t m, int64_t n,
                                              int64_t k, const void* a, int64_t lda, const void* b,
                                              int64_t ldb, const void* features, void* backprops,
                                              float* bias_grad, tfd_dtype type, tfd_rounding rounding,
                                              void* workspace, size_t workspace_bytes, void* stream);

/*
 * ReLU masks
 * ----------
 * ReluGrad (section 4.1) needs only one fact about each forward output: is
 * the stored value > 0. A ReLU mask keeps that fact as one bit per element,
 * so the backward pass can read 1 bit instead of a 16- or 32-bit feature.
 * Layout of the mask of a rows x cols matrix: rows x ceil(cols / 32) uint32
 * words, contiguous (row r starts at word r * ceil(cols / 32)); bit j of
 * word w of row r is 1 iff element (r, 32 w + j) is > 0 (so -0, +0 and NaN
 * give 0); the bits past the last column of a row are 0. Masks are 4-byte
 * aligned device buffers owned by the caller. A mask-based call stores
 * exactly what its features-based counterpart stores, bit for bit.
 */

/* relu_mask = the mask of features (rows x cols of `type`, contiguous). */
TFD_API tfd_status tfd_relu_mask(const void* features, uint32_t* relu_mask, int64_t rows, int64_t cols,
                                 tfd_dtype type, void* stream);

/*
 * The forward MatMul + Add + ReLU of Figure 1 that also emits the ReLU mask
 * of its output (for the layer's ReluGrad in the backward pass):
 *   c = Relu(op(A) op(B) + 1 bias^T), as tfd_matmul with TFD_EPI_BIAS_RELU
 *       (and TFD_EPI_TRUNCATE_16 when rounding is TFD_ROUND_TRUNCATE), with
 *       A, B and c all of `type`,
 *   relu_mask = the mask of the stored c (m rows, ceil(n / 32) words each).
 * c is bit-identical to tfd_matmul's. bias is fp32[n] and required. The
 * mask must not overlap A, B, bias or c.
 */
TFD_API tfd_status tfd_matmul_relu_mask(int transpose_a, int transpose_b, int64_t m, int64_t n, int64_t k,
                                        const void* a, int64_t lda, const void* b, int64_t ldb,
                                        const float* bias, void* c, int64_t ldc, uint32_t* relu_mask,
                                        tfd_dtype type, tfd_rounding rounding, void* stream);

/*
 * tfd_relu_grad_bias_add_grad with the Relu test read from a ReLU mask of
 * the rows x cols forward output (instead of the features themselves):
 *   d = bit(r, c) ? gradients[r, c] : +0, backprops = d (skipped when
 *   backprops is NULL), bias_grad[c] = sum_r d.
 * backprops and bias_grad equal tfd_relu_grad_bias_add_grad's bit for bit
 * when relu_mask is the mask of its features. Workspace as
 * tfd_reduction_workspace_size. No output may overlap an input.
 */
TFD_API tfd_status tfd_relu_mask_grad_bias_add_grad(const void* gradients, const uint32_t* relu_mask,
                                                    void* backprops, float* bias_grad, int64_t rows,
                                                    int64_t cols, tfd_dtype type, void* workspace,
                                                    size_t workspace_bytes, void* stream);

/*
 * tfd_matmul_relu_grad_bias_add_grad with the Relu test read from a ReLU
 * mask of the m x n forward output instead of its features. backprops equals
 * the features-based call's bit for bit (and bias_grad too, on the same
 * shapes). Workspace as tfd_matmul_relu_grad_workspace_size.
 */
TFD_API tfd_status tfd_matmul_relu_mask_grad_bias_add_grad(int transpose_a, int transpose_b, int64_t m,
                                                           int64_t n, int64_t k, const void* a, int64_t lda,
                                                           const void* b, int64_t ldb,
                                                           const uint32_t* relu_mask, void* backprops,
                                                           float* bias_grad, tfd_dtype type,
                                                           tfd_rounding rounding, void* workspace,
                                                           size_t workspace_bytes, void* stream);

/* Workspace bytes that tfd_l2_loss_grad needs for `count` elements. */
TFD_API size_t tfd_loss_workspace_size(int64_t count, tfd_dtype type);

/*
 * Cost head: the squared error L = 1/2 sum_i (output[i] - target[i])^2 and
 * its gradient grad[i] = output[i] - target[i] (the exact difference rounded
 * once to `type`). target == NULL means 0 (L = 1/2 sum output^2,
 * grad = output). `loss` is a device double, written with a fixed summation
 * order (float64 partial sums of the fp32 squares). grad may equal output.
 */
TFD_API tfd_status tfd_l2_loss_grad(const void* output, const void* target, void* grad, double* loss,
                            int64_t count, tfd_dtype type,
                            void* workspace, size_t workspace_bytes, void* stream);

/* Workspace bytes that tfd_matmul_l2_loss_grad needs for an m x n output. */
TFD_API size_t tfd_matmul_l2_loss_grad_workspace_size(int64_t m, int64_t n, tfd_dtype type);

/*
 * The output layer's MatMul fused with the squared-error cost head and the
 * output layer's BiasAddGrad (Figure 1's MatMul and Add on the last layer,
 * then section 4.1's first gradient ops):
 *   output[r, c]    = (op(A) op(B))[r, c] + bias[c], fp32 accumulation, rounded
 *                     once to `type` (with `rounding` for 16-bit outputs),
 *   grad[r, c]      = output[r, c] - target[r, c], as tfd_l2_loss_grad computes it,
 *   loss            = 1/2 sum grad_exact^2 (float64, fixed order),
 *   bias_grad[c]    = sum_r grad[r, c] (fp32, fixed order).
 * Operands as in tfd_matmul; output, target and grad are m x n of `type`,
 * contiguous (ld = n); bias is fp32[n]; target == NULL means 0 (as in
 * tfd_l2_loss_grad). output and grad equal what
 * tfd_matmul, tfd_l2_loss_grad and tfd_bias_add_grad store, bit for bit;
 * loss and bias_grad may differ from that path in the order of their sums.
 * No output buffer may overlap an input or another output.
 */
TFD_API tfd_status tfd_matmul_l2_loss_grad(int transpose_a, int transpose_b, int64_t m, int64_t n, int64_t k,
                                   const void* a, int64_t lda, const void* b, int64_t ldb, const float* bias,
                                   void* output, const void* target, void* grad, double* loss,
                                   float* bias_grad, tfd_dtype type, tfd_rounding rounding,
                                   void* workspace, size_t workspace_bytes, void* stream);

/* Workspace bytes that tfd_softmax_cross_entropy_grad needs for `rows` rows. */
TFD_API size_t tfd_softmax_xent_workspace_size(int64_t rows);

/*
 * Classifier cost head: SoftMax (section 2, Table 1) of each row of
 * logits[rows x cols] (row-major, contiguous), its cross-entropy against one
 * integer class label per row, and the gradient with respect to the logits:
 *   p[r, :]    = softmax(logits[r, :]),
 *   loss       = sum_r ( log sum_c exp(logits[r, c]) - logits[r, labels[r]] ),
 *   grad[r, c] = p[r, c] - (c == labels[r])   (rounded once to `type`).
 * labels is a device int32[rows]. Work is fp32 with the row maximum
 * subtracted before exp; each row's loss term is formed in float64 from the
 * fp32 log-sum-exp and summed in a fixed order, so `loss` (a device double)
 * is reproducible bit for bit. A label outside [0, cols) is not detected on
 * the host: that row's gradient is p with nothing subtracted and its loss
 * term, hence `loss`, is NaN. rows = 0 writes loss = 0; cols must be >= 1
 * when rows > 0. grad must not overlap logits, labels, loss or workspace.
 */
TFD_API tfd_status tfd_softmax_cross_entropy_grad(const void* logits, const int32_t* labels, void* grad,
                                          double* loss, int64_t rows, int64_t cols, tfd_dtype type,
                                          void* workspace, size_t workspace_bytes, void* stream);

/*
 * ApplyGradientDescent on an fp32 Variable (section 2 "Variables"; the SGD
 * step of section 4.1), in place:
 *   var[i] = fma(-alpha, delta[i], var[i])   (one rounding),
 * and, when var_bf16 != NULL, var_bf16[i] = the updated var[i] converted to
 * the 16-bit format with `rounding` (the operand copy of 16-bit GEMMs).
 * delta must not overlap var.
 */
TFD_API tfd_status tfd_apply_gradient_descent(float* var, float alpha, const float* delta,
                                      int64_t count, uint16_t* var_bf16, tfd_rounding rounding,
                                      void* stream);

/*
 * ApplyGradientDescent on an fp32 weight matrix var[rows x cols] (row-major,
 * contiguous), in place, with the same update and rounding as
 * tfd_apply_gradient_descent, refreshing up to two 16-bit operand copies of
 * the updated weights in the same pass:
 *   var_bf16  (nullable): rows x cols, var_bf16[r * cols + c]   = bf16(var[r, c]),
 *   var_bf16_t (nullable): cols x rows, var_bf16_t[c * rows + r] = bf16(var[r, c]).
 * The transposed copy lets a forward MatMul read the weights k-contiguous
 * (transpose_b = 1) while the input-gradient MatMul reads the untransposed
 * copy (the step keeps it for layers with fan_in under 2048). None of the
 * four buffers may overlap another.
 */
TFD_API tfd_status tfd_apply_gradient_descent_matrix(float* var, float alpha, const float* delta,
                                             int64_t rows, int64_t cols, uint16_t* var_bf16,
                                             uint16_t* var_bf16_t, tfd_rounding rounding,
                                             void* stream);

/*
 * The conversion nodes of section 5.5 ("lossy compression" of the tensors a
 * Send/Recv pair moves between devices): fp32 -> 16 bits on the sending side,
 * 16 bits -> fp32 on the receiving side.
 *   tfd_convert_f32_to_bf16: dst[i] = 16-bit pattern of src[i] under
 *     `rounding` (TFD_ROUND_TRUNCATE is the paper's converter).
 *   tfd_convert_bf16_to_f32: dst[i] = the fp32 whose high half is src[i] and
 *     whose low 16 bits are zero (exact; NaN payloads are kept).
 * Contiguous arrays of `count` elements; src and dst must not overlap.
 */
TFD_API tfd_status tfd_convert_f32_to_bf16(const float* src, uint16_t* dst, int64_t count,
                                   tfd_rounding rounding, void* stream);
TFD_API tfd_status tfd_convert_bf16_to_f32(const uint16_t* src, float* dst, int64_t count, void* stream);

/*
 * Engine clock probe (measurement support for benchmarks; not an op of the
 * training step). One wave of 64 lanes runs `iterations` dependent fp32 FMAs
 * between two reads of the shader clock counter and of the constant 100 MHz
 * real-time counter, and writes counters[0] = shader clock cycles elapsed,
 * counters[1] = real-time ticks elapsed, counters[2] = the FMA chain's result
 * (it keeps the chain from being removed). The clock of the compute unit the
 * wave ran on, in MHz, is 100 * counters[0] / counters[1]; launched on a
 * second stream while other work runs, it measures the clock under that load.
 * counters: device, 3 uint64 (written, not read). iterations in [1, 2^31),
 * else TFD_EINVAL.
 */
TFD_API tfd_status tfd_clock_probe(uint64_t* counters, int64_t iterations, void* stream);

/*
 * One whole training step of a small fp32 multilayer perceptron in one
 * kernel, launched once per phase or once in all (persistent): the forward pass H_l = Relu(H_{l-1} W_l + b_l) (Figure 1;
 * MatMul, Add and ReLU of section 2, Table 1), the cost head, the gradient
 * subgraph that automatic differentiation adds (section 4.1: ReluGrad, the
 * transposed MatMuls, BiasAddGrad) and the SGD update of the Variables (the
 * in-place update of section 2, "Variables"). The same computation as the
 * per-op calls above, for steps too small to fill the GPU one kernel at a time
 * (a few hundred rows, layers of a few thousand units), where launch gaps
 * dominate: the ops are grouped into 2 L + 2 phases (forward layers, the cost
 * head, one phase per layer of the backward pass that also holds the update of
 * the layer above, the update of layer 0), each phase's MatMul tiles, column
 * sums and update chunks spread over the workgroups of one launch. With
 * `persistent` nonzero all phases run in one cooperative launch, separated by
 * grid-wide barriers; otherwise each phase is a launch of its own (stream order
 * separates them).
 *
 * Layer l (0-based, up to TFD_MLP_MAX_LAYERS), all fp32 row-major with
 * leading dimension = row length:
 *   weights [fan_in, fan_out] W_l (read, then updated in place when `update`),
 *   bias [fan_out] b_l (likewise), activations [batch, fan_out] H_{l+1}
 *   (written), backprop [batch, fan_out] dY_l (written; required for a Relu
 *   layer, ignored otherwise), weight_grad [fan_in, fan_out] dW_l and
 *   bias_grad [fan_out] db_l (written). fan_in of layer l must equal fan_out of
 *   layer l - 1; every layer but the last must have a Relu (relu != 0).
 * x [batch, fan_in of layer 0] is the input; input_grad [batch, same] receives
 * dX_0 = dY_0 W_0^T when not NULL. cost: TFD_COST_SQUARED_ERROR,
 * L = 1/2 sum (out - target)^2 (target NULL: target 0), G = out - target; or
 * TFD_COST_SOFTMAX_XENT with int32 labels [batch], L = sum_n (log sum_j
 * exp(z_nj) - z_n,y_n), G = softmax(z) - onehot(y) (a label outside
 * [0, classes) gives a NaN loss). cost_grad [batch, classes] receives G and
 * *loss (device float64) L. The output layer's dY is ReluGrad(G, out) when it
 * has a Relu, else G itself (its backprop is not written). Every Variable is
 * updated as var - learning_rate * grad, rounded once.
 *
 * workspace: tfd_mlp_step_workspace_size(desc) bytes, 8-byte aligned (the
 * cost head's loss partials, and for the persistent launch its barrier). Its
 * first 4096 bytes hold the grid barrier (an error word at offset 0, a
 * generation count at 256, arrival counters from 512 on) and must be zero
 * before the first call on it; a call that completes normally leaves the
 * error word and the arrival counters at zero (the generation count
 * advances), ready for the next. If a barrier wait times out (only possible
 * if the grid were not all resident), the error word is nonzero once the
 * stream has reached the call, the outputs are incomplete, and the first 4096
 * bytes must be zeroed again before the workspace is reused. Calls that share a workspace must not
 * overlap. Results are bitwise reproducible. Buffers must not overlap each
 * other except as stated. Errors: TFD_EINVAL for NULL required pointers,
 * sizes out of range (layers in [1, TFD_MLP_MAX_LAYERS], batch and fans in
 * [1, 2^20], batch x fan and fan_in x fan_out below 2^31), mismatched fans, a
 * small or misaligned workspace; TFD_EUNSUPPORTED for a hidden layer without
 * a Relu; TFD_EHIP if the cooperative launch is refused. batch == 0 enqueues
 * nothing.
 */
#define TFD_MLP_MAX_LAYERS 4
typedef enum tfd_cost { TFD_COST_SQUARED_ERROR = 0, TFD_COST_SOFTMAX_XENT = 1 } tfd_cost;
typedef struct tfd_mlp_layer {
  float* weights;
  float* bias;
  float* activations;
  float* backprop;
  float* weight_grad;
  float* bias_grad;
  int64_t fan_in, fan_out;
  int32_t relu;
} tfd_mlp_layer;
typedef struct tfd_mlp_step_desc {
  int32_t layers;
  int64_t batch;
  const float* x;
  float* input_grad;
  tfd_mlp_layer layer[TFD_MLP_MAX_LAYERS];
  int32_t cost;
  const float* target;
  const int32_t* labels;
  float* cost_grad;
  double* loss;
  float learning_rate;
  int32_t update;
  int32_t persistent;
} tfd_mlp_step_desc;
TFD_API size_t tfd_mlp_step_workspace_size(const tfd_mlp_step_desc* desc);
TFD_API tfd_status tfd_mlp_step(const tfd_mlp_step_desc* desc, void* workspace, size_t workspace_bytes,
                                void* stream);

#ifdef __cplusplus
}
#endif

#endif /* TFDENSE_H */
