// C ABI of libtfdense: argument validation and dispatch to the kernels.
// The contract of every entry point is documented in include/tfdense.h.

#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <atomic>

#include "../../include/tfdense.h"
#include "kernels.h"

namespace {

thread_local char g_err[512] = "";

tfd_status fail(tfd_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return st;
}

tfd_status hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return TFD_OK;
  return fail(TFD_EHIP, "%s: %s", what, hipGetErrorString(e));
}

inline hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

bool valid_dtype(tfd_dtype t) { return t == TFD_F32 || t == TFD_BF16; }
bool valid_rounding(tfd_rounding r) { return r == TFD_ROUND_NEAREST_EVEN || r == TFD_ROUND_TRUNCATE; }
int elem_bytes(tfd_dtype t) { return t == TFD_BF16 ? 2 : 4; }

// Byte ranges [p, p + bytes) overlap?
bool overlaps(const void* p, size_t pb, const void* q, size_t qb) {
  if (!p || !q || pb == 0 || qb == 0) return false;
  const uintptr_t a = reinterpret_cast<uintptr_t>(p), b = reinterpret_cast<uintptr_t>(q);
  return a < b + qb && b < a + pb;
}

// Extent in bytes of a rows x cols matrix with leading dimension ld.
size_t span(int64_t rows, int64_t cols, int64_t ld, int eb) {
  if (rows <= 0 || cols <= 0) return 0;
  return (size_t)((rows - 1) * ld + cols) * (size_t)eb;
}

}  // namespace

extern "C" {

int tfd_abi_version(void) { return TFD_ABI_VERSION; }

const char* tfd_status_string(tfd_status s) {
  switch (s) {
    case TFD_OK: return "ok";
    case TFD_EINVAL: return "invalid argument";
    case TFD_EUNSUPPORTED: return "unsupported";
    case TFD_EHIP: return "HIP runtime error";
  }
  return "unknown status";
}

const char* tfd_last_error(void) { return g_err; }

}  // extern "C"

namespace {

std::atomic<int> g_tune[tfd::kTuneCount];

struct KnobSpec {
  const char* name;
  tfd::TuneKnob knob;
  int lo, hi;      // accepted range besides 0
  bool waves;      // only 4, 8 or 16
};

constexpr KnobSpec kKnobs[] = {
    {"gemm_tile", tfd::kTuneGemmTile, 1, 9, false},
    {"bf16_waves_nn", tfd::kTuneBf16WavesNN, 4, 16, true},
    {"bf16_waves_nt", tfd::kTuneBf16WavesNT, 4, 16, true},
    {"bf16_waves_tn", tfd::kTuneBf16WavesTN, 4, 16, true},
    {"small_waves", tfd::kTuneSmallWaves, 4, 16, true},
};

}  // namespace

namespace tfd {
int tuning(TuneKnob knob) { return g_tune[knob].load(std::memory_order_relaxed); }
}  // namespace tfd

extern "C" {

tfd_status tfd_set_tuning(const char* knob, int value) {
  if (!knob) return fail(TFD_EINVAL, "tfd_set_tuning: null knob name");
  for (const KnobSpec& k : kKnobs) {
    if (strcmp(k.name, knob) != 0) continue;
    const bool ok = value == 0 || (k.waves ? (value == 4 || value == 8 || value == 16)
                                           : (value >= k.lo && value <= k.hi));
    if (!ok) return fail(TFD_EINVAL, "tfd_set_tuning: value %d out of range for %s", value, knob);
    g_tune[k.knob].store(value, std::memory_order_relaxed);
    return TFD_OK;
  }
  return fail(TFD_EINVAL, "tfd_set_tuning: unknown knob %s", knob);
}

}  // extern "C"

namespace {

// Compute units of the current device (cached per device).
int device_cus() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cached[dev] == 0) {
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0) cus = 256;
    cached[dev] = cus;
  }
  return cached[dev];
}

// The k split a 16-bit whole-tile problem would use, and its workspace bytes.
int split_plan(const tfd::GemmDesc& d, int64_t* kt_per, size_t* bytes) {
  *kt_per = 0;
  *bytes = 0;
  if (!tfd::gemm_bf16_256_ok(d) || tfd::gemm_tile_override() != 0) return 1;
  int s = tfd::gemm_bf16_256_splits(d, device_cus());
  if (s < 2) return 1;
  const int64_t kt = d.k / 64;
  const int64_t per = (kt + s - 1) / s;
  s = (int)((kt + per - 1) / per);  // every split non-empty
  if (s < 2) return 1;
  *kt_per = per;
  *bytes = (size_t)s * (size_t)d.m * (size_t)d.n * sizeof(float);
  return s;
}

tfd_status matmul_impl(const char* fn, int transpose_a, int transpose_b, int64_t m, int64_t n, int64_t k,
                       const void* a, int64_t lda, tfd_dtype a_type, const void* b, int64_t ldb, tfd_dtype b_type,
                       void* c, int64_t ldc, tfd_dtype c_type, const float* bias, tfd_epilogue epilogue,
                       void* workspace, size_t workspace_bytes, void* stream);

}  // namespace

extern "C" {

tfd_status tfd_matmul(int transpose_a, int transpose_b, int64_t m, int64_t n, int64_t k,
                      const void* a, int64_t lda, tfd_dtype a_type,
                      const void* b, int64_t ldb, tfd_dtype b_type,
                      void* c, int64_t ldc, tfd_dtype c_type,
                      const float* bias, tfd_epilogue epilogue, void* stream) {
  return matmul_impl("tfd_matmul", transpose_a, transpose_b, m, n, k, a, lda, a_type, b, ldb, b_type, c, ldc, c_type,
                     bias, epilogue, nullptr, 0, stream);
}

size_t tfd_matmul_workspace_size(int transpose_a, int transpose_b, int64_t m, int64_t n, int64_t k, tfd_dtype a_type,
                                 tfd_dtype b_type, tfd_dtype c_type) {
  if (m <= 0 || n <= 0 || k <= 0 || !valid_dtype(a_type) || !valid_dtype(b_type) || !valid_dtype(c_type)) return 0;
  if (transpose_a && transpose_b) return 0;
  tfd::GemmDesc d;
  d.ta = transpose_a != 0;
  d.tb = transpose_b != 0;
  d.m = m;
  d.n = n;
  d.k = k;
  // the plan depends on the shape and types; contiguous, aligned operands are assumed
  d.a = reinterpret_cast<const void*>(uintptr_t(256));
  d.b = d.a;
  d.c = reinterpret_cast<void*>(uintptr_t(256));
  d.lda = transpose_a ? m : k;
  d.ldb = transpose_b ? k : n;
  d.ldc = n;
  d.in_bf16 = a_type == TFD_BF16 && b_type == TFD_BF16;
  d.out_bf16 = c_type == TFD_BF16;
  d.bias = nullptr;
  d.epi = 0;
  int64_t per;
  size_t bytes;
  split_plan(d, &per, &bytes);
  return bytes;
}

tfd_status tfd_matmul_with_workspace(int transpose_a, int transpose_b, int64_t m, int64_t n, int64_t k,
                                     const void* a, int64_t lda, tfd_dtype a_type, const void* b, int64_t ldb,
                                     tfd_dtype b_type, void* c, int64_t ldc, tfd_dtype c_type, const float* bias,
                                     tfd_epilogue epilogue, void* workspace, size_t workspace_bytes, void* stream) {
  return matmul_impl("tfd_matmul_with_workspace", transpose_a, transpose_b, m, n, k, a, lda, a_type, b, ldb, b_type,
                     c, ldc, c_type, bias, epilogue, workspace, workspace_bytes, stream);
}

}  // extern "C"

namespace {

tfd_status matmul_impl(const char* fn, int transpose_a, int transpose_b, int64_t m, int64_t n, int64_t k,
                       const void* a, int64_t lda, tfd_dtype a_type, const void* b, int64_t ldb, tfd_dtype b_type,
                       void* c, int64_t ldc, tfd_dtype c_type, const float* bias, tfd_epilogue epilogue,
                       void* workspace, size_t workspace_bytes, void* stream) {
  g_err[0] = 0;
  if (m < 0 || n < 0 || k < 0) return fail(TFD_EINVAL, "%s: negative size m=%lld n=%lld k=%lld", fn, (long long)m, (long long)n, (long long)k);
  if (!valid_dtype(a_type) || !valid_dtype(b_type) || !valid_dtype(c_type))
    return fail(TFD_EINVAL, "%s: unknown element type", fn);
  const bool trunc16 = ((int)epilogue & TFD_EPI_TRUNCATE_16) != 0;
  const int op = (int)epilogue & ~(int)TFD_EPI_TRUNCATE_16;
  if (op != TFD_EPI_NONE && op != TFD_EPI_BIAS && op != TFD_EPI_BIAS_RELU)
    return fail(TFD_EINVAL, "%s: unknown epilogue %d", fn, (int)epilogue);
  if (trunc16 && c_type != TFD_BF16)
    return fail(TFD_EINVAL, "%s: TFD_EPI_TRUNCATE_16 needs a 16-bit output", fn);
  if (transpose_a && transpose_b)
    return fail(TFD_EUNSUPPORTED, "%s: transpose_a and transpose_b together are not implemented", fn);
  if (a_type != b_type || (a_type == TFD_F32 && c_type != TFD_F32))
    return fail(TFD_EUNSUPPORTED, "%s: element types (a=%d, b=%d, c=%d) not implemented", fn, a_type, b_type, c_type);
  // The kernels index with 32-bit tile coordinates.
  if (m > (1LL << 30) || n > (1LL << 30) || k > (1LL << 30))
    return fail(TFD_EUNSUPPORTED, "%s: dimension above 2^30", fn);
  const int64_t a_rows = transpose_a ? k : m, a_cols = transpose_a ? m : k;
  const int64_t b_rows = transpose_b ? n : k, b_cols = transpose_b ? k : n;
  if (lda < (a_cols > 0 ? a_cols : 1) || ldb < (b_cols > 0 ? b_cols : 1) || ldc < (n > 0 ? n : 1))
    return fail(TFD_EINVAL, "%s: leading dimension smaller than the row (lda=%lld ldb=%lld ldc=%lld)", fn, (long long)lda, (long long)ldb, (long long)ldc);
  if (m == 0 || n == 0) return TFD_OK;
  if (!c) return fail(TFD_EINVAL, "%s: c is NULL", fn);
  if (k > 0 && (!a || !b)) return fail(TFD_EINVAL, "%s: a or b is NULL", fn);
  if (op != TFD_EPI_NONE && !bias) return fail(TFD_EINVAL, "%s: the bias epilogue needs a bias", fn);
  const int ab = elem_bytes(a_type), cb = elem_bytes(c_type);
  const size_t c_span = span(m, n, ldc, cb);
  if (overlaps(c, c_span, a, span(a_rows, a_cols, lda, ab)) ||
      overlaps(c, c_span, b, span(b_rows, b_cols, ldb, ab)) ||
      (op != TFD_EPI_NONE && overlaps(c, c_span, bias, (size_t)n * 4)))
    return fail(TFD_EINVAL, "%s: c overlaps an input", fn);
  tfd::GemmDesc d;
  d.ta = transpose_a != 0;
  d.tb = transpose_b != 0;
  d.m = m;
  d.n = n;
  d.k = k;
  d.a = a;
  d.lda = lda;
  d.b = b;
  d.ldb = ldb;
  d.c = c;
  d.ldc = ldc;
  d.in_bf16 = a_type == TFD_BF16;
  d.out_bf16 = c_type == TFD_BF16;
  d.bias = bias;
  d.epi = op | (trunc16 ? tfd::kEpiTrunc16 : 0);
  hipStream_t st = as_stream(stream);
  if (workspace) {
    int64_t kt_per;
    size_t need;
    const int splits = split_plan(d, &kt_per, &need);
    if (splits > 1 && workspace_bytes >= need && (reinterpret_cast<uintptr_t>(workspace) & 15) == 0 &&
        !overlaps(workspace, need, a, span(a_rows, a_cols, lda, ab)) &&
        !overlaps(workspace, need, b, span(b_rows, b_cols, ldb, ab)) && !overlaps(workspace, need, c, c_span) &&
        !(op != TFD_EPI_NONE && overlaps(workspace, need, bias, (size_t)n * 4))) {
      // the k range split over `splits` workgroups per tile: fp32 partial
      // products in the workspace, then their ordered sum with the epilogue
      tfd::GemmDesc g = d;
      g.c = workspace;
      g.ldc = n;
      g.out_bf16 = false;
      g.bias = nullptr;
      g.epi = 0;
      g.splits = splits;
      g.kt_per = kt_per;
      hipError_t e = tfd::launch_gemm_bf16_256(g, st);
      if (e == hipSuccess) e = tfd::launch_splitk_reduce(static_cast<const float*>(workspace), splits, d, st);
      return hip_status(e, "tfd_matmul launch");
    }
  }
  return hip_status(tfd::launch_gemm(d, st), "tfd_matmul launch");
}

}  // namespace

extern "C" {


tfd_status tfd_bias_add(const void* value, const float* bias, void* out, int64_t rows, int64_t cols,
                        tfd_dtype type, void* stream) {
  g_err[0] = 0;
  if (rows < 0 || cols < 0) return fail(TFD_EINVAL, "tfd_bias_add: negative size");
  if (!valid_dtype(type)) return fail(TFD_EINVAL, "tfd_bias_add: unknown element type");
  if (rows == 0 || cols == 0) return TFD_OK;
  if (!value || !bias || !out) return fail(TFD_EINVAL, "tfd_bias_add: NULL pointer");
  const size_t bytes = (size_t)(rows * cols) * elem_bytes(type);
  if (value != out && overlaps(value, bytes, out, bytes))
    return fail(TFD_EINVAL, "tfd_bias_add: out partially overlaps value");
  if (overlaps(bias, (size_t)cols * 4, out, bytes)) return fail(TFD_EINVAL, "tfd_bias_add: out overlaps bias");
  return hip_status(tfd::launch_bias_add(value, bias, out, rows, cols, type == TFD_BF16, as_stream(stream)),
                    "tfd_bias_add launch");
}

tfd_status tfd_relu(const void* features, void* activations, int64_t count, tfd_dtype type, void* stream) {
  g_err[0] = 0;
  if (count < 0) return fail(TFD_EINVAL, "tfd_relu: negative count");
  if (!valid_dtype(type)) return fail(TFD_EINVAL, "tfd_relu: unknown element type");
  if (count == 0) return TFD_OK;
  if (!features || !activations) return fail(TFD_EINVAL, "tfd_relu: NULL pointer");
  const size_t bytes = (size_t)count * elem_bytes(type);
  if (features != activations && overlaps(features, bytes, activations, bytes))
    return fail(TFD_EINVAL, "tfd_relu: activations partially overlap features");
  return hip_status(tfd::launch_relu(features, activations, count, type == TFD_BF16, as_stream(stream)),
                    "tfd_relu launch");
}

tfd_status tfd_relu_grad(const void* gradients, const void* features, void* backprops, int64_t count,
                         tfd_dtype type, void* stream) {
  g_err[0] = 0;
  if (count < 0) return fail(TFD_EINVAL, "tfd_relu_grad: negative count");
  if (!valid_dtype(type)) return fail(TFD_EINVAL, "tfd_relu_grad: unknown element type");
  if (count == 0) return TFD_OK;
  if (!gradients || !features || !backprops) return fail(TFD_EINVAL, "tfd_relu_grad: NULL pointer");
  const size_t bytes = (size_t)count * elem_bytes(type);
  if ((backprops != gradients && overlaps(backprops, bytes, gradients, bytes)) ||
      overlaps(backprops, bytes, features, bytes))
    return fail(TFD_EINVAL, "tfd_relu_grad: backprops overlaps features or part of gradients");
  return hip_status(tfd::launch_relu_grad(gradients, features, backprops, count, type == TFD_BF16,
                                          as_stream(stream)),
                    "tfd_relu_grad launch");
}

size_t tfd_reduction_workspace_size(int64_t rows, int64_t cols, tfd_dtype type) {
  if (rows < 0 || cols <= 0 || !valid_dtype(type)) return 0;
  return tfd::reduction_ws_bytes(rows, cols, type == TFD_BF16);
}

tfd_status tfd_relu_grad_bias_add_grad(const void* gradients, const void* features, void* backprops,
                                       float* bias_grad, int64_t rows, int64_t cols, tfd_dtype type,
                                       void* workspace, size_t workspace_bytes, void* stream) {
  g_err[0] = 0;
  if (rows < 0 || cols < 0) return fail(TFD_EINVAL, "tfd_relu_grad_bias_add_grad: negative size");
  if (!valid_dtype(type)) return fail(TFD_EINVAL, "tfd_relu_grad_bias_add_grad: unknown element type");
  if (cols == 0) return TFD_OK;
  if (!bias_grad) return fail(TFD_EINVAL, "tfd_relu_grad_bias_add_grad: bias_grad is NULL");
  if (rows > 0 && !gradients) return fail(TFD_EINVAL, "tfd_relu_grad_bias_add_grad: gradients is NULL");
  const size_t need = tfd::reduction_ws_bytes(rows, cols, type == TFD_BF16);
  if (!workspace || workspace_bytes < need)
    return fail(TFD_EINVAL, "tfd_relu_grad_bias_add_grad: workspace of %zu bytes needed, %zu given", need, workspace_bytes);
  const size_t bytes = (size_t)(rows * cols) * elem_bytes(type);
  if (overlaps(backprops, bytes, gradients, bytes) || overlaps(backprops, bytes, features, bytes) ||
      overlaps(workspace, need, gradients, bytes) || overlaps(workspace, need, backprops, bytes) ||
      overlaps(bias_grad, (size_t)cols * 4, backprops, bytes) || overlaps(bias_grad, (size_t)cols * 4, workspace, need))
    return fail(TFD_EINVAL, "tfd_relu_grad_bias_add_grad: overlapping buffers");
  return hip_status(tfd::launch_relu_grad_bias_add_grad(gradients, features, backprops, bias_grad, rows, cols,
                                                        type == TFD_BF16, workspace, as_stream(stream)),
                    "tfd_relu_grad_bias_add_grad launch");
}

tfd_status tfd_relu_grad_bias_add_grad_noalloc(const void* gradients, const void* features, void* backprops,
                                               float* bias_grad, int64_t rows, int64_t cols, tfd_dtype type,
                                               void* stream) {
  g_err[0] = 0;
  const char* fn = "tfd_relu_grad_bias_add_grad_noalloc";
  if (rows < 0 || cols < 0) return fail(TFD_EINVAL, "%s: negative size", fn);
  if (!valid_dtype(type)) return fail(TFD_EINVAL, "%s: unknown element type", fn);
  if (cols == 0) return TFD_OK;
  if (!bias_grad) return fail(TFD_EINVAL, "%s: bias_grad is NULL", fn);
  if (rows > 0 && !gradients) return fail(TFD_EINVAL, "%s: gradients is NULL", fn);
  const size_t need = tfd::reduction_ws_bytes(rows, cols, type == TFD_BF16);
  if (need > tfd::static_scratch_bytes())
    return fail(TFD_EINVAL, "%s: %lld x %lld needs %zu bytes of scratch, above the fixed maximum of %zu", fn,
                (long long)rows, (long long)cols, need, tfd::static_scratch_bytes());
  const size_t bytes = (size_t)(rows * cols) * elem_bytes(type);
  if (overlaps(backprops, bytes, gradients, bytes) || overlaps(backprops, bytes, features, bytes) ||
      overlaps(bias_grad, (size_t)cols * 4, backprops, bytes))
    return fail(TFD_EINVAL, "%s: overlapping buffers", fn);
  void* ws = nullptr;
  tfd_status st = hip_status(tfd::static_scratch(&ws), "tfd_relu_grad_bias_add_grad_noalloc scratch lookup");
  if (st != TFD_OK) return st;
  return hip_status(tfd::launch_relu_grad_bias_add_grad(gradients, features, backprops, bias_grad, rows, cols,
                                                        type == TFD_BF16, ws, as_stream(stream)),
                    "tfd_relu_grad_bias_add_grad_noalloc launch");
}

tfd_status tfd_bias_add_grad(const void* out_backprop, float* bias_grad, int64_t rows, int64_t cols,
                             tfd_dtype type, void* workspace, size_t workspace_bytes, void* stream) {
  tfd_status st = tfd_relu_grad_bias_add_grad(out_backprop, nullptr, nullptr, bias_grad, rows, cols, type,
                                              workspace, workspace_bytes, stream);
  if (st != TFD_OK && strncmp(g_err, "tfd_relu_grad_bias_add_grad", 27) == 0) {
    char tmp[512];
    snprintf(tmp, sizeof(tmp), "tfd_bias_add_grad%s", g_err + 27);
    memcpy(g_err, tmp, sizeof(tmp));
  }
  return st;
}

size_t tfd_matmul_relu_grad_workspace_size(int64_t m, int64_t n, tfd_dtype type) {
  if (m < 0 || n < 0 || !valid_dtype(type)) return 0;
  const size_t fused = (size_t)((m + 255) / 256) * (size_t)n * sizeof(float);
  const size_t plain = tfd::reduction_ws_bytes(m, n, type == TFD_BF16);
  return fused > plain ? fused : plain;
}

tfd_status tfd_matmul_relu_grad_bias_add_grad(int transpose_a, int transpose_b, int64_t m, int64_t n, int64_t k,
                                              const void* a, int64_t lda, const void* b, int64_t ldb,
                                              const void* features, void* backprops, float* bias_grad,
                                              tfd_dtype type, tfd_rounding rounding, void* workspace,
                                              size_t workspace_bytes, void* stream) {
  g_err[0] = 0;
  if (m < 0 || n < 0 || k < 0) return fail(TFD_EINVAL, "tfd_matmul_relu_grad_bias_add_grad: negative size");
  if (!valid_dtype(type)) return fail(TFD_EINVAL, "tfd_matmul_relu_grad_bias_add_grad: unknown element type");
  if (!valid_rounding(rounding)) return fail(TFD_EINVAL, "tfd_matmul_relu_grad_bias_add_grad: unknown rounding");
  if (rounding == TFD_ROUND_TRUNCATE && type != TFD_BF16)
    return fail(TFD_EINVAL, "tfd_matmul_relu_grad_bias_add_grad: truncation needs a 16-bit output");
  if (transpose_a && transpose_b)
    return fail(TFD_EUNSUPPORTED, "tfd_matmul_relu_grad_bias_add_grad: transpose_a and transpose_b together");
  if (m > (1LL << 30) || n > (1LL << 30) || k > (1LL << 30))
    return fail(TFD_EUNSUPPORTED, "tfd_matmul_relu_grad_bias_add_grad: dimension above 2^30");
  const int64_t a_rows = transpose_a ? k : m, a_cols = transpose_a ? m : k;
  const int64_t b_rows = transpose_b ? n : k, b_cols = transpose_b ? k : n;
  if (lda < (a_cols > 0 ? a_cols : 1) || ldb < (b_cols > 0 ? b_cols : 1))
    return fail(TFD_EINVAL, "tfd_matmul_relu_grad_bias_add_grad: leading dimension smaller than the row");
  if (n == 0) return TFD_OK;
  if (!bias_grad) return fail(TFD_EINVAL, "tfd_matmul_relu_grad_bias_add_grad: bias_grad is NULL");
  const size_t need = tfd_matmul_relu_grad_workspace_size(m, n, type);
  if (!workspace || workspace_bytes < need)
    return fail(TFD_EINVAL, "tfd_matmul_relu_grad_bias_add_grad: workspace of %zu bytes needed, %zu given", need,
                workspace_bytes);
  if (m > 0 && (!features || !backprops || (k > 0 && (!a || !b))))
    return fail(TFD_EINVAL, "tfd_matmul_relu_grad_bias_add_grad: NULL pointer");
  const int eb = elem_bytes(type);
  const size_t c_span = (size_t)m * (size_t)n * eb;
  if (overlaps(backprops, c_span, a, span(a_rows, a_cols, lda, eb)) ||
      overlaps(backprops, c_span, b, span(b_rows, b_cols, ldb, eb)) || overlaps(backprops, c_span, features, c_span) ||
      overlaps(backprops, c_span, bias_grad, (size_t)n * 4) || overlaps(backprops, c_span, workspace, need) ||
      overlaps(bias_grad, (size_t)n * 4, workspace, need) || overlaps(bias_grad, (size_t)n * 4, features, c_span))
    return fail(TFD_EINVAL, "tfd_matmul_relu_grad_bias_add_grad: overlapping buffers");
  hipStream_t st = as_stream(stream);
  tfd::GemmDesc d;
  d.ta = transpose_a != 0;
  d.tb = transpose_b != 0;
  d.m = m;
  d.n = n;
  d.k = k;
  d.a = a;
  d.lda = lda;
  d.b = b;
  d.ldb = ldb;
  d.c = backprops;
  d.ldc = n;
  d.in_bf16 = type == TFD_BF16;
  d.out_bf16 = type == TFD_BF16;
  d.bias = nullptr;
  d.epi = rounding == TFD_ROUND_TRUNCATE ? tfd::kEpiTrunc16 : 0;
  d.features = features;
  d.ldf = n;
  d.col_partial = static_cast<float*>(workspace);
  if (m > 0 && tfd::gemm_bf16_256_ok(d) && tfd::gemm_tile_override() == 0) {
    hipError_t e = tfd::launch_gemm_bf16_256(d, st);
    if (e != hipSuccess) return hip_status(e, "tfd_matmul_relu_grad_bias_add_grad launch");
    return hip_status(tfd::launch_colsum_final(static_cast<const float*>(workspace), bias_grad, m / 256, n, st),
                      "tfd_matmul_relu_grad_bias_add_grad launch");
  }
  // other shapes: the MatMul writes G into backprops, then ReluGrad and
  // BiasAddGrad run in place over it
  d.features = nullptr;
  d.col_partial = nullptr;
  if (m > 0) {
    hipError_t e = tfd::launch_gemm(d, st);
    if (e != hipSuccess) return hip_status(e, "tfd_matmul_relu_grad_bias_add_grad launch");
  }
  return hip_status(tfd::launch_relu_grad_bias_add_grad(backprops, features, backprops, bias_grad, m, n,
                                                        type == TFD_BF16, workspace, st),
                    "tfd_matmul_relu_grad_bias_add_grad launch");
}

tfd_status tfd_relu_mask(const void* features, uint32_t* relu_mask, int64_t rows, int64_t cols, tfd_dtype type,
                         void* stream) {
  g_err[0] = 0;
  const char* fn = "tfd_relu_mask";
  if (rows < 0 || cols < 0) return fail(TFD_EINVAL, "%s: negative size", fn);
  if (!valid_dtype(type)) return fail(TFD_EINVAL, "%s: unknown element type", fn);
  if (rows == 0 || cols == 0) return TFD_OK;
  if (!features || !relu_mask) return fail(TFD_EINVAL, "%s: NULL pointer", fn);
  const size_t fb = (size_t)rows * (size_t)cols * elem_bytes(type), mb = (size_t)rows * ((cols + 31) / 32) * 4;
  if (overlaps(features, fb, relu_mask, mb)) return fail(TFD_EINVAL, "%s: relu_mask overlaps features", fn);
  if ((reinterpret_cast<uintptr_t>(relu_mask) & 3) != 0) return fail(TFD_EINVAL, "%s: relu_mask not 4-byte aligned", fn);
  return hip_status(tfd::launch_relu_mask(features, cols, relu_mask, (cols + 31) / 32, rows, cols, type == TFD_BF16,
                                          as_stream(stream)),
                    "tfd_relu_mask launch");
}

tfd_status tfd_matmul_relu_mask(int transpose_a, int transpose_b, int64_t m, int64_t n, int64_t k, const void* a,
                                int64_t lda, const void* b, int64_t ldb, const float* bias, void* c, int64_t ldc,
                                uint32_t* relu_mask, tfd_dtype type, tfd_rounding rounding, void* stream) {
  g_err[0] = 0;
  const char* fn = "tfd_matmul_relu_mask";
  if (m < 0 || n < 0 || k < 0) return fail(TFD_EINVAL, "%s: negative size", fn);
  if (!valid_dtype(type)) return fail(TFD_EINVAL, "%s: unknown element type", fn);
  if (!valid_rounding(rounding)) return fail(TFD_EINVAL, "%s: unknown rounding", fn);
  if (rounding == TFD_ROUND_TRUNCATE && type != TFD_BF16)
    return fail(TFD_EINVAL, "%s: truncation needs a 16-bit output", fn);
  if (transpose_a && transpose_b) return fail(TFD_EUNSUPPORTED, "%s: transpose_a and transpose_b together", fn);
  if (m > (1LL << 30) || n > (1LL << 30) || k > (1LL << 30)) return fail(TFD_EUNSUPPORTED, "%s: dimension above 2^30", fn);
  const int64_t a_rows = transpose_a ? k : m, a_cols = transpose_a ? m : k;
  const int64_t b_rows = transpose_b ? n : k, b_cols = transpose_b ? k : n;
  if (lda < (a_cols > 0 ? a_cols : 1) || ldb < (b_cols > 0 ? b_cols : 1) || ldc < (n > 0 ? n : 1))
    return fail(TFD_EINVAL, "%s: leading dimension smaller than the row", fn);
  if (m == 0 || n == 0) return TFD_OK;
  if (!c || !bias || !relu_mask) return fail(TFD_EINVAL, "%s: c, bias or relu_mask is NULL", fn);
  if (k > 0 && (!a || !b)) return fail(TFD_EINVAL, "%s: a or b is NULL", fn);
  if ((reinterpret_cast<uintptr_t>(relu_mask) & 3) != 0) return fail(TFD_EINVAL, "%s: relu_mask not 4-byte aligned", fn);
  const int eb = elem_bytes(type);
  const int64_t ldm = (n + 31) / 32;
  const size_t c_span = span(m, n, ldc, eb), mb = (size_t)m * (size_t)ldm * 4, nb = (size_t)n * 4;
  const size_t as = span(a_rows, a_cols, lda, eb), bs = span(b_rows, b_cols, ldb, eb);
  if (overlaps(c, c_span, a, as) || overlaps(c, c_span, b, bs) || overlaps(c, c_span, bias, nb) ||
      overlaps(relu_mask, mb, a, as) || overlaps(relu_mask, mb, b, bs) || overlaps(relu_mask, mb, bias, nb) ||
      overlaps(relu_mask, mb, c, c_span))
    return fail(TFD_EINVAL, "%s: overlapping buffers", fn);
  tfd::GemmDesc d;
  d.ta = transpose_a != 0;
  d.tb = transpose_b != 0;
  d.m = m;
  d.n = n;
  d.k = k;
  d.a = a;
  d.lda = lda;
  d.b = b;
  d.ldb = ldb;
  d.c = c;
  d.ldc = ldc;
  d.in_bf16 = type == TFD_BF16;
  d.out_bf16 = type == TFD_BF16;
  d.bias = bias;
  d.epi = TFD_EPI_BIAS_RELU | (rounding == TFD_ROUND_TRUNCATE ? tfd::kEpiTrunc16 : 0);
  d.mask_out = relu_mask;
  d.ldm = ldm;
  hipStream_t s = as_stream(stream);
  if (tfd::gemm_bf16_256_ok(d) && tfd::gemm_tile_override() == 0)
    return hip_status(tfd::launch_gemm_bf16_256(d, s), "tfd_matmul_relu_mask launch");
  // other shapes: the MatMul, then the mask of its stored output
  d.mask_out = nullptr;
  hipError_t e = tfd::launch_gemm(d, s);
  if (e == hipSuccess) e = tfd::launch_relu_mask(c, ldc, relu_mask, ldm, m, n, type == TFD_BF16, s);
  return hip_status(e, "tfd_matmul_relu_mask launch");
}

tfd_status tfd_relu_mask_grad_bias_add_grad(const void* gradients, const uint32_t* relu_mask, void* backprops,
                                            float* bias_grad, int64_t rows, int64_t cols, tfd_dtype type,
                                            void* workspace, size_t workspace_bytes, void* stream) {
  g_err[0] = 0;
  const char* fn = "tfd_relu_mask_grad_bias_add_grad";
  if (rows < 0 || cols < 0) return fail(TFD_EINVAL, "%s: negative size", fn);
  if (!valid_dtype(type)) return fail(TFD_EINVAL, "%s: unknown element type", fn);
  if (cols == 0) return TFD_OK;
  if (!bias_grad) return fail(TFD_EINVAL, "%s: bias_grad is NULL", fn);
  if (rows > 0 && (!gradients || !relu_mask)) return fail(TFD_EINVAL, "%s: gradients or relu_mask is NULL", fn);
  if (relu_mask && (reinterpret_cast<uintptr_t>(relu_mask) & 3) != 0)
    return fail(TFD_EINVAL, "%s: relu_mask not 4-byte aligned", fn);
  const size_t need = tfd::reduction_ws_bytes(rows, cols, type == TFD_BF16);
  if (!workspace || workspace_bytes < need)
    return fail(TFD_EINVAL, "%s: workspace of %zu bytes needed, %zu given", fn, need, workspace_bytes);
  const int64_t ldm = (cols + 31) / 32;
  const size_t bytes = (size_t)(rows * cols) * elem_bytes(type), mb = (size_t)rows * ldm * 4;
  if (overlaps(backprops, bytes, gradients, bytes) || overlaps(backprops, bytes, relu_mask, mb) ||
      overlaps(workspace, need, gradients, bytes) || overlaps(workspace, need, backprops, bytes) ||
      overlaps(workspace, need, relu_mask, mb) || overlaps(bias_grad, (size_t)cols * 4, backprops, bytes) ||
      overlaps(bias_grad, (size_t)cols * 4, workspace, need) || overlaps(bias_grad, (size_t)cols * 4, relu_mask, mb))
    return fail(TFD_EINVAL, "%s: overlapping buffers", fn);
  return hip_status(tfd::launch_relu_mask_grad_bias_add_grad(gradients, relu_mask, ldm, backprops, bias_grad, rows, cols,
                                                             type == TFD_BF16, workspace, as_stream(stream)),
                    "tfd_relu_mask_grad_bias_add_grad launch");
}

tfd_status tfd_matmul_relu_mask_grad_bias_add_grad(int transpose_a, int transpose_b, int64_t m, int64_t n, int64_t k,
                                                   const void* a, int64_t lda, const void* b, int64_t ldb,
                                                   const uint32_t* relu_mask, void* backprops, float* bias_grad,
                                                   tfd_dtype type, tfd_rounding rounding, void* workspace,
                                                   size_t workspace_bytes, void* stream) {
  g_err[0] = 0;
  const char* fn = "tfd_matmul_relu_mask_grad_bias_add_grad";
  if (m < 0 || n < 0 || k < 0) return fail(TFD_EINVAL, "%s: negative size", fn);
  if (!valid_dtype(type)) return fail(TFD_EINVAL, "%s: unknown element type", fn);
  if (!valid_rounding(rounding)) return fail(TFD_EINVAL, "%s: unknown rounding", fn);
  if (rounding == TFD_ROUND_TRUNCATE && type != TFD_BF16)
    return fail(TFD_EINVAL, "%s: truncation needs a 16-bit output", fn);
  if (transpose_a && transpose_b) return fail(TFD_EUNSUPPORTED, "%s: transpose_a and transpose_b together", fn);
  if (m > (1LL << 30) || n > (1LL << 30) || k > (1LL << 30)) return fail(TFD_EUNSUPPORTED, "%s: dimension above 2^30", fn);
  const int64_t a_rows = transpose_a ? k : m, a_cols = transpose_a ? m : k;
  const int64_t b_rows = transpose_b ? n : k, b_cols = transpose_b ? k : n;
  if (lda < (a_cols > 0 ? a_cols : 1) || ldb < (b_cols > 0 ? b_cols : 1))
    return fail(TFD_EINVAL, "%s: leading dimension smaller than the row", fn);
  if (n == 0) return TFD_OK;
  if (!bias_grad) return fail(TFD_EINVAL, "%s: bias_grad is NULL", fn);
  const size_t need = tfd_matmul_relu_grad_workspace_size(m, n, type);
  if (!workspace || workspace_bytes < need)
    return fail(TFD_EINVAL, "%s: workspace of %zu bytes needed, %zu given", fn, need, workspace_bytes);
  if (m > 0 && (!relu_mask || !backprops || (k > 0 && (!a || !b)))) return fail(TFD_EINVAL, "%s: NULL pointer", fn);
  if (relu_mask && (reinterpret_cast<uintptr_t>(relu_mask) & 3) != 0)
    return fail(TFD_EINVAL, "%s: relu_mask not 4-byte aligned", fn);
  const int eb = elem_bytes(type);
  const int64_t ldm = (n + 31) / 32;
  const size_t c_span = (size_t)m * (size_t)n * eb, mb = (size_t)m * ldm * 4, nb = (size_t)n * 4;
  if (overlaps(backprops, c_span, a, span(a_rows, a_cols, lda, eb)) ||
      overlaps(backprops, c_span, b, span(b_rows, b_cols, ldb, eb)) || overlaps(backprops, c_span, relu_mask, mb) ||
      overlaps(backprops, c_span, bias_grad, nb) || overlaps(backprops, c_span, workspace, need) ||
      overlaps(bias_grad, nb, workspace, need) || overlaps(bias_grad, nb, relu_mask, mb) ||
      overlaps(workspace, need, relu_mask, mb))
    return fail(TFD_EINVAL, "%s: overlapping buffers", fn);
  hipStream_t st = as_stream(stream);
  tfd::GemmDesc d;
  d.ta = transpose_a != 0;
  d.tb = transpose_b != 0;
  d.m = m;
  d.n = n;
  d.k = k;
  d.a = a;
  d.lda = lda;
  d.b = b;
  d.ldb = ldb;
  d.c = backprops;
  d.ldc = n;
  d.in_bf16 = type == TFD_BF16;
  d.out_bf16 = type == TFD_BF16;
  d.bias = nullptr;
  d.epi = rounding == TFD_ROUND_TRUNCATE ? tfd::kEpiTrunc16 : 0;
  d.mask_in = relu_mask;
  d.ldm = ldm;
  d.col_partial = static_cast<float*>(workspace);
  if (m > 0 && tfd::gemm_bf16_256_ok(d) && tfd::gemm_tile_override() == 0) {
    hipError_t e = tfd::launch_gemm_bf16_256(d, st);
    if (e != hipSuccess) return hip_status(e, "tfd_matmul_relu_mask_grad_bias_add_grad launch");
    return hip_status(tfd::launch_colsum_final(static_cast<const float*>(workspace), bias_grad, m / 256, n, st),
                      "tfd_matmul_relu_mask_grad_bias_add_grad launch");
  }
  // other shapes: the MatMul writes G into backprops, then ReluGrad (from the
  // mask) and BiasAddGrad run in place over it
  d.mask_in = nullptr;
  d.col_partial = nullptr;
  if (m > 0) {
    hipError_t e = tfd::launch_gemm(d, st);
    if (e != hipSuccess) return hip_status(e, "tfd_matmul_relu_mask_grad_bias_add_grad launch");
  }
  return hip_status(tfd::launch_relu_mask_grad_bias_add_grad(backprops, relu_mask, ldm, backprops, bias_grad, m, n,
                                                             type == TFD_BF16, workspace, st),
                    "tfd_matmul_relu_mask_grad_bias_add_grad launch");
}

size_t tfd_matmul_l2_loss_grad_workspace_size(int64_t m, int64_t n, tfd_dtype type) {
  if (m < 0 || n < 0 || !valid_dtype(type)) return 0;
  const bool h = type == TFD_BF16;
  const int64_t tiles = ((m + 255) / 256) * ((n + 255) / 256);
  const size_t fused = (size_t)((m + 255) / 256) * (size_t)n * sizeof(float) + (size_t)tiles * sizeof(double);
  size_t plain = tfd::loss_ws_bytes(m * n, h);
  const size_t red = tfd::reduction_ws_bytes(m, n, h);
  if (red > plain) plain = red;
  return fused > plain ? fused : plain;
}

tfd_status tfd_matmul_l2_loss_grad(int transpose_a, int transpose_b, int64_t m, int64_t n, int64_t k, const void* a,
                                   int64_t lda, const void* b, int64_t ldb, const float* bias, void* output,
                                   const void* target, void* grad, double* loss, float* bias_grad, tfd_dtype type,
                                   tfd_rounding rounding, void* workspace, size_t workspace_bytes, void* stream) {
  g_err[0] = 0;
  const char* fn = "tfd_matmul_l2_loss_grad";
  if (m < 0 || n < 0 || k < 0) return fail(TFD_EINVAL, "%s: negative size", fn);
  if (!valid_dtype(type)) return fail(TFD_EINVAL, "%s: unknown element type", fn);
  if (!valid_rounding(rounding)) return fail(TFD_EINVAL, "%s: unknown rounding", fn);
  if (rounding == TFD_ROUND_TRUNCATE && type != TFD_BF16)
    return fail(TFD_EINVAL, "%s: truncation needs a 16-bit output", fn);
  if (transpose_a && transpose_b) return fail(TFD_EUNSUPPORTED, "%s: transpose_a and transpose_b together", fn);
  if (m > (1LL << 30) || n > (1LL << 30) || k > (1LL << 30))
    return fail(TFD_EUNSUPPORTED, "%s: dimension above 2^30", fn);
  const int64_t a_rows = transpose_a ? k : m, a_cols = transpose_a ? m : k;
  const int64_t b_rows = transpose_b ? n : k, b_cols = transpose_b ? k : n;
  if (lda < (a_cols > 0 ? a_cols : 1) || ldb < (b_cols > 0 ? b_cols : 1))
    return fail(TFD_EINVAL, "%s: leading dimension smaller than the row", fn);
  if (!loss) return fail(TFD_EINVAL, "%s: loss is NULL", fn);
  if (n > 0 && (!bias || !bias_grad)) return fail(TFD_EINVAL, "%s: NULL bias or bias_grad", fn);
  const size_t need = tfd_matmul_l2_loss_grad_workspace_size(m, n, type);
  if (!workspace || workspace_bytes < need)
    return fail(TFD_EINVAL, "%s: workspace of %zu bytes needed, %zu given", fn, need, workspace_bytes);
  if (m > 0 && n > 0 && (!output || !grad || (k > 0 && (!a || !b))))
    return fail(TFD_EINVAL, "%s: NULL pointer", fn);
  const int eb = elem_bytes(type);
  const size_t cs = (size_t)m * (size_t)n * eb, as = span(a_rows, a_cols, lda, eb), bs = span(b_rows, b_cols, ldb, eb);
  const size_t nb = (size_t)n * 4;
  const void* outs[] = {output, grad, bias_grad, loss, workspace};
  const size_t out_sz[] = {cs, cs, nb, 8, need};
  const void* ins[] = {a, b, bias, target};
  const size_t in_sz[] = {as, bs, nb, cs};
  for (int i = 0; i < 5; ++i) {
    for (int j = 0; j < 4; ++j)
      if (overlaps(outs[i], out_sz[i], ins[j], in_sz[j])) return fail(TFD_EINVAL, "%s: overlapping buffers", fn);
    for (int j = i + 1; j < 5; ++j)
      if (overlaps(outs[i], out_sz[i], outs[j], out_sz[j])) return fail(TFD_EINVAL, "%s: overlapping buffers", fn);
  }
  hipStream_t st = as_stream(stream);
  if (n == 0)  // no columns: an empty sum
    return hip_status(tfd::launch_loss_final(static_cast<const double*>(workspace), 0, loss, st),
                      "tfd_matmul_l2_loss_grad launch");
  tfd::GemmDesc d;
  d.ta = transpose_a != 0;
  d.tb = transpose_b != 0;
  d.m = m;
  d.n = n;
  d.k = k;
  d.a = a;
  d.lda = lda;
  d.b = b;
  d.ldb = ldb;
  d.c = output;
  d.ldc = n;
  d.in_bf16 = type == TFD_BF16;
  d.out_bf16 = type == TFD_BF16;
  d.bias = bias;
  d.epi = TFD_EPI_BIAS | (rounding == TFD_ROUND_TRUNCATE ? tfd::kEpiTrunc16 : 0);
  d.target = target;
  d.grad = grad;
  const int64_t tiles_m = (m + 255) / 256, tiles = tiles_m * ((n + 255) / 256);
  d.col_partial = static_cast<float*>(workspace);
  d.loss_partial = reinterpret_cast<double*>(static_cast<char*>(workspace) + (size_t)tiles_m * n * sizeof(float));
  if (m > 0 && target && tfd::gemm_bf16_256_ok(d) && tfd::gemm_tile_override() == 0 &&
      (reinterpret_cast<uintptr_t>(d.loss_partial) & 7) == 0 && tiles < (1LL << 31)) {
    hipError_t e = tfd::launch_gemm_bf16_256(d, st);
    if (e == hipSuccess) e = tfd::launch_colsum_final(d.col_partial, bias_grad, tiles_m, n, st);
    if (e == hipSuccess) e = tfd::launch_loss_final(d.loss_partial, (int)tiles, loss, st);
    return hip_status(e, "tfd_matmul_l2_loss_grad launch");
  }
  // other shapes: the three calls in sequence (they share the workspace in
  // stream order)
  d.target = nullptr;
  d.grad = nullptr;
  d.col_partial = nullptr;
  d.loss_partial = nullptr;
  hipError_t e = hipSuccess;
  if (m > 0) e = tfd::launch_gemm(d, st);
  if (e == hipSuccess)
    e = tfd::launch_l2_loss_grad(output, target, grad, loss, m * n, type == TFD_BF16, workspace, st);
  if (e == hipSuccess)
    e = tfd::launch_relu_grad_bias_add_grad(grad, nullptr, nullptr, bias_grad, m, n, type == TFD_BF16, workspace, st);
  return hip_status(e, "tfd_matmul_l2_loss_grad launch");
}

size_t tfd_loss_workspace_size(int64_t count, tfd_dtype type) {
  if (count < 0 || !valid_dtype(type)) return 0;
  return tfd::loss_ws_bytes(count, type == TFD_BF16);
}

tfd_status tfd_l2_loss_grad(const void* output, const void* target, void* grad, double* loss, int64_t count,
                            tfd_dtype type, void* workspace, size_t workspace_bytes, void* stream) {
  g_err[0] = 0;
  if (count < 0) return fail(TFD_EINVAL, "tfd_l2_loss_grad: negative count");
  if (!valid_dtype(type)) return fail(TFD_EINVAL, "tfd_l2_loss_grad: unknown element type");
  if (!loss) return fail(TFD_EINVAL, "tfd_l2_loss_grad: loss is NULL");
  if (count > 0 && (!output || !grad)) return fail(TFD_EINVAL, "tfd_l2_loss_grad: NULL pointer");
  const size_t need = tfd::loss_ws_bytes(count, type == TFD_BF16);
  if (!workspace || workspace_bytes < need)
    return fail(TFD_EINVAL, "tfd_l2_loss_grad: workspace of %zu bytes needed, %zu given", need, workspace_bytes);
  const size_t bytes = (size_t)count * elem_bytes(type);
  if ((grad != output && overlaps(grad, bytes, output, bytes)) || overlaps(grad, bytes, target, bytes) ||
      overlaps(workspace, need, grad, bytes) || overlaps(loss, 8, grad, bytes) || overlaps(loss, 8, workspace, need))
    return fail(TFD_EINVAL, "tfd_l2_loss_grad: overlapping buffers");
  return hip_status(tfd::launch_l2_loss_grad(output, target, grad, loss, count, type == TFD_BF16, workspace,
                                             as_stream(stream)),
                    "tfd_l2_loss_grad launch");
}

size_t tfd_softmax_xent_workspace_size(int64_t rows) {
  if (rows < 0) return 0;
  return tfd::softmax_xent_ws_bytes(rows);
}

tfd_status tfd_softmax_cross_entropy_grad(const void* logits, const int32_t* labels, void* grad, double* loss,
                                          int64_t rows, int64_t cols, tfd_dtype type, void* workspace,
                                          size_t workspace_bytes, void* stream) {
  g_err[0] = 0;
  if (rows < 0 || cols < 0) return fail(TFD_EINVAL, "tfd_softmax_cross_entropy_grad: negative size");
  if (rows > 0 && cols == 0) return fail(TFD_EINVAL, "tfd_softmax_cross_entropy_grad: rows > 0 with cols = 0");
  if (!valid_dtype(type)) return fail(TFD_EINVAL, "tfd_softmax_cross_entropy_grad: unknown element type");
  if (!loss) return fail(TFD_EINVAL, "tfd_softmax_cross_entropy_grad: loss is NULL");
  if (rows > 0 && (!logits || !labels || !grad))
    return fail(TFD_EINVAL, "tfd_softmax_cross_entropy_grad: NULL pointer");
  if (rows > (int64_t)INT32_MAX * 4 || cols > (int64_t)INT32_MAX)
    return fail(TFD_EINVAL, "tfd_softmax_cross_entropy_grad: size out of range");
  const size_t need = tfd::softmax_xent_ws_bytes(rows);
  if (!workspace || workspace_bytes < need)
    return fail(TFD_EINVAL, "tfd_softmax_cross_entropy_grad: workspace of %zu bytes needed, %zu given", need,
                workspace_bytes);
  const size_t bytes = (size_t)rows * (size_t)cols * elem_bytes(type);
  const size_t lbytes = (size_t)rows * sizeof(int32_t);
  if (overlaps(grad, bytes, logits, bytes) || overlaps(grad, bytes, labels, lbytes) || overlaps(grad, bytes, loss, 8) ||
      overlaps(grad, bytes, workspace, need) || overlaps(loss, 8, workspace, need) ||
      overlaps(loss, 8, labels, lbytes) || overlaps(loss, 8, logits, bytes))
    return fail(TFD_EINVAL, "tfd_softmax_cross_entropy_grad: overlapping buffers");
  return hip_status(tfd::launch_softmax_xent(logits, labels, grad, loss, rows, cols, type == TFD_BF16, workspace,
                                             as_stream(stream)),
                    "tfd_softmax_cross_entropy_grad launch");
}

tfd_status tfd_apply_gradient_descent(float* var, float alpha, const float* delta, int64_t count,
                                      uint16_t* var_bf16, tfd_rounding rounding, void* stream) {
  g_err[0] = 0;
  if (count < 0) return fail(TFD_EINVAL, "tfd_apply_gradient_descent: negative count");
  if (!valid_rounding(rounding)) return fail(TFD_EINVAL, "tfd_apply_gradient_descent: unknown rounding");
  if (count == 0) return TFD_OK;
  if (!var || !delta) return fail(TFD_EINVAL, "tfd_apply_gradient_descent: NULL pointer");
  const size_t bytes = (size_t)count * 4;
  if (overlaps(var, bytes, delta, bytes) || overlaps(var_bf16, (size_t)count * 2, var, bytes) ||
      overlaps(var_bf16, (size_t)count * 2, delta, bytes))
    return fail(TFD_EINVAL, "tfd_apply_gradient_descent: overlapping buffers");
  return hip_status(tfd::launch_sgd(var, alpha, delta, count, var_bf16, rounding == TFD_ROUND_TRUNCATE,
                                    as_stream(stream)),
                    "tfd_apply_gradient_descent launch");
}

tfd_status tfd_apply_gradient_descent_matrix(float* var, float alpha, const float* delta, int64_t rows,
                                             int64_t cols, uint16_t* var_bf16, uint16_t* var_bf16_t,
                                             tfd_rounding rounding, void* stream) {
  g_err[0] = 0;
  if (rows < 0 || cols < 0) return fail(TFD_EINVAL, "tfd_apply_gradient_descent_matrix: negative size");
  if (!valid_rounding(rounding)) return fail(TFD_EINVAL, "tfd_apply_gradient_descent_matrix: unknown rounding");
  if (rows == 0 || cols == 0) return TFD_OK;
  if (!var || !delta) return fail(TFD_EINVAL, "tfd_apply_gradient_descent_matrix: NULL pointer");
  const size_t n = (size_t)rows * (size_t)cols;
  if (overlaps(var, n * 4, delta, n * 4) || overlaps(var_bf16, n * 2, var, n * 4) ||
      overlaps(var_bf16, n * 2, delta, n * 4) || overlaps(var_bf16_t, n * 2, var, n * 4) ||
      overlaps(var_bf16_t, n * 2, delta, n * 4) || overlaps(var_bf16, n * 2, var_bf16_t, n * 2))
    return fail(TFD_EINVAL, "tfd_apply_gradient_descent_matrix: overlapping buffers");
  return hip_status(tfd::launch_sgd_matrix(var, alpha, delta, rows, cols, var_bf16, var_bf16_t,
                                           rounding == TFD_ROUND_TRUNCATE, as_stream(stream)),
                    "tfd_apply_gradient_descent_matrix launch");
}

tfd_status tfd_convert_f32_to_bf16(const float* src, uint16_t* dst, int64_t count, tfd_rounding rounding,
                                   void* stream) {
  g_err[0] = 0;
  if (count < 0) return fail(TFD_EINVAL, "tfd_convert_f32_to_bf16: negative count");
  if (!valid_rounding(rounding)) return fail(TFD_EINVAL, "tfd_convert_f32_to_bf16: unknown rounding");
  if (count == 0) return TFD_OK;
  if (!src || !dst) return fail(TFD_EINVAL, "tfd_convert_f32_to_bf16: NULL pointer");
  if (overlaps(src, (size_t)count * 4, dst, (size_t)count * 2))
    return fail(TFD_EINVAL, "tfd_convert_f32_to_bf16: src and dst overlap");
  return hip_status(tfd::launch_convert_to_bf16(src, dst, count, rounding == TFD_ROUND_TRUNCATE, as_stream(stream)),
                    "tfd_convert_f32_to_bf16 launch");
}

tfd_status tfd_convert_bf16_to_f32(const uint16_t* src, float* dst, int64_t count, void* stream) {
  g_err[0] = 0;
  if (count < 0) return fail(TFD_EINVAL, "tfd_convert_bf16_to_f32: negative count");
  if (count == 0) return TFD_OK;
  if (!src || !dst) return fail(TFD_EINVAL, "tfd_convert_bf16_to_f32: NULL pointer");
  if (overlaps(src, (size_t)count * 2, dst, (size_t)count * 4))
    return fail(TFD_EINVAL, "tfd_convert_bf16_to_f32: src and dst overlap");
  return hip_status(tfd::launch_convert_to_f32(src, dst, count, as_stream(stream)), "tfd_convert_bf16_to_f32 launch");
}

tfd_status tfd_clock_probe(uint64_t* counters, int64_t iterations, void* stream) {
  g_err[0] = 0;
  if (!counters) return fail(TFD_EINVAL, "tfd_clock_probe: NULL counters");
  if (iterations < 1 || iterations >= (int64_t(1) << 31))
    return fail(TFD_EINVAL, "tfd_clock_probe: iterations %lld outside [1, 2^31)", (long long)iterations);
  return hip_status(tfd::launch_clock_probe(counters, iterations, as_stream(stream)), "tfd_clock_probe launch");
}

}  // extern "C"

namespace {

// Checks a step descriptor; fills `out` when valid.
tfd_status mlp_check(const tfd_mlp_step_desc* d, const char* fn, tfd::MlpStep* out) {
  if (!d) return fail(TFD_EINVAL, "%s: NULL descriptor", fn);
  const int L = d->layers;
  if (L < 1 || L > TFD_MLP_MAX_LAYERS) return fail(TFD_EINVAL, "%s: layers %d outside [1, %d]", fn, L, TFD_MLP_MAX_LAYERS);
  const int64_t lim = int64_t(1) << 20, big = int64_t(1) << 31;
  if (d->batch < 0 || d->batch > lim) return fail(TFD_EINVAL, "%s: batch %lld outside [0, 2^20]", fn, (long long)d->batch);
  if (d->cost != TFD_COST_SQUARED_ERROR && d->cost != TFD_COST_SOFTMAX_XENT)
    return fail(TFD_EINVAL, "%s: unknown cost %d", fn, d->cost);
  for (int l = 0; l < L; ++l) {
    const tfd_mlp_layer& y = d->layer[l];
    if (y.fan_in < 1 || y.fan_in > lim || y.fan_out < 1 || y.fan_out > lim)
      return fail(TFD_EINVAL, "%s: layer %d fans %lld x %lld outside [1, 2^20]", fn, l, (long long)y.fan_in,
                  (long long)y.fan_out);
    if (y.fan_in * y.fan_out >= big || d->batch * y.fan_in >= big || d->batch * y.fan_out >= big)
      return fail(TFD_EINVAL, "%s: layer %d too large", fn, l);
    if (l > 0 && y.fan_in != d->layer[l - 1].fan_out)
      return fail(TFD_EINVAL, "%s: layer %d fan_in %lld != fan_out %lld of layer %d", fn, l, (long long)y.fan_in,
                  (long long)d->layer[l - 1].fan_out, l - 1);
    if (!y.weights || !y.bias || !y.activations || !y.weight_grad || !y.bias_grad)
      return fail(TFD_EINVAL, "%s: layer %d: NULL buffer", fn, l);
    if (y.relu && !y.backprop) return fail(TFD_EINVAL, "%s: layer %d has a Relu but no backprop buffer", fn, l);
    if (l < L - 1 && !y.relu) return fail(TFD_EUNSUPPORTED, "%s: hidden layer %d without a Relu", fn, l);
  }
  if (!d->x || !d->cost_grad || !d->loss) return fail(TFD_EINVAL, "%s: NULL x, cost_grad or loss", fn);
  if (d->cost == TFD_COST_SOFTMAX_XENT && !d->labels) return fail(TFD_EINVAL, "%s: softmax cost without labels", fn);
  if (out) {
    *out = tfd::MlpStep{};
    out->layers = L;
    out->cost = d->cost;
    out->update = d->update != 0;
    out->persistent = d->persistent != 0;
    out->batch = d->batch;
    for (int l = 0; l < L; ++l) {
      const tfd_mlp_layer& y = d->layer[l];
      out->fan_in[l] = y.fan_in;
      out->fan_out[l] = y.fan_out;
      out->relu[l] = y.relu != 0;
      out->w[l] = y.weights;
      out->b[l] = y.bias;
      out->h[l] = y.activations;
      out->dy[l] = y.relu ? y.backprop : nullptr;
      out->dw[l] = y.weight_grad;
      out->db[l] = y.bias_grad;
    }
    out->x = d->x;
    out->dx0 = d->input_grad;
    out->g = d->cost_grad;
    out->target = d->cost == TFD_COST_SQUARED_ERROR ? d->target : nullptr;
    out->labels = d->cost == TFD_COST_SOFTMAX_XENT ? d->labels : nullptr;
    out->loss = d->loss;
    out->lr = d->learning_rate;
  }
  return TFD_OK;
}

}  // namespace

extern "C" {

size_t tfd_mlp_step_workspace_size(const tfd_mlp_step_desc* desc) {
  if (mlp_check(desc, "tfd_mlp_step_workspace_size", nullptr) != TFD_OK) return 0;
  const tfd_mlp_layer& top = desc->layer[desc->layers - 1];
  return tfd::mlp_step_ws_bytes(desc->batch, top.fan_in, top.fan_out, desc->cost);
}

tfd_status tfd_mlp_step(const tfd_mlp_step_desc* desc, void* workspace, size_t workspace_bytes, void* stream) {
  g_err[0] = 0;
  tfd::MlpStep st;
  const tfd_status c = mlp_check(desc, "tfd_mlp_step", &st);
  if (c != TFD_OK) return c;
  if (st.batch == 0) return TFD_OK;
  const size_t need = tfd::mlp_step_ws_bytes(st.batch, st.fan_in[st.layers - 1], st.fan_out[st.layers - 1], st.cost);
  if (!workspace || workspace_bytes < need)
    return fail(TFD_EINVAL, "tfd_mlp_step: workspace of %zu bytes, %zu needed", workspace_bytes, need);
  if (reinterpret_cast<uintptr_t>(workspace) & 7) return fail(TFD_EINVAL, "tfd_mlp_step: workspace not 8-byte aligned");
  return hip_status(tfd::launch_mlp_step(st, workspace, as_stream(stream)), "tfd_mlp_step launch");
}

}  // extern "C"
