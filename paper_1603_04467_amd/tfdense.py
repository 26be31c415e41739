"""Python binding of libtfdense (argument marshalling only).

Each function carries the name of the C entry point it calls and takes torch
tensors that already live on the GPU; it derives sizes, leading dimensions
and element types, passes ``data_ptr()`` and the current HIP stream, and
raises ``TfdError`` on a non-OK status. All arithmetic happens in the
library's HIP kernels. torch is used for device memory and streams only.

The library must be built (``python -m paper_1603_04467_amd.build``); there is
no fallback when it is missing.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libtfdense.so")

TFD_OK, TFD_EINVAL, TFD_EUNSUPPORTED, TFD_EHIP = 0, 1, 2, 3
TFD_F32, TFD_BF16 = 0, 1
TFD_ROUND_NEAREST_EVEN, TFD_ROUND_TRUNCATE = 0, 1
TFD_EPI_TRUNCATE_16 = 16
ROUNDINGS = {"nearest": TFD_ROUND_NEAREST_EVEN, "truncate": TFD_ROUND_TRUNCATE}
EPILOGUES = {"none": 0, "bias": 1, "bias_relu": 2}

EXPORTS = (
    "tfd_abi_version", "tfd_status_string", "tfd_last_error", "tfd_matmul", "tfd_bias_add",
    "tfd_relu", "tfd_relu_grad", "tfd_reduction_workspace_size", "tfd_bias_add_grad",
    "tfd_relu_grad_bias_add_grad", "tfd_matmul_relu_grad_workspace_size", "tfd_matmul_relu_grad_bias_add_grad",
    "tfd_matmul_l2_loss_grad_workspace_size", "tfd_matmul_l2_loss_grad", "tfd_loss_workspace_size", "tfd_l2_loss_grad",
    "tfd_softmax_xent_workspace_size", "tfd_softmax_cross_entropy_grad", "tfd_apply_gradient_descent",
    "tfd_apply_gradient_descent_matrix", "tfd_convert_f32_to_bf16", "tfd_convert_bf16_to_f32",
    "tfd_relu_mask", "tfd_matmul_relu_mask", "tfd_relu_mask_grad_bias_add_grad",
    "tfd_matmul_relu_mask_grad_bias_add_grad", "tfd_matmul_workspace_size", "tfd_matmul_with_workspace",
    "tfd_set_tuning", "tfd_relu_grad_bias_add_grad_noalloc", "tfd_clock_probe",
    "tfd_mlp_step_workspace_size", "tfd_mlp_step",
)

MLP_MAX_LAYERS = 4
COSTS = {"sq_err": 0, "softmax_xent": 1}


class MlpLayer(ctypes.Structure):
    """tfd_mlp_layer (include/tfdense.h)."""
    _fields_ = [("weights", ctypes.c_void_p), ("bias", ctypes.c_void_p), ("activations", ctypes.c_void_p),
                ("backprop", ctypes.c_void_p), ("weight_grad", ctypes.c_void_p), ("bias_grad", ctypes.c_void_p),
                ("fan_in", ctypes.c_int64), ("fan_out", ctypes.c_int64), ("relu", ctypes.c_int32)]


class MlpStepDesc(ctypes.Structure):
    """tfd_mlp_step_desc (include/tfdense.h)."""
    _fields_ = [("layers", ctypes.c_int32), ("batch", ctypes.c_int64), ("x", ctypes.c_void_p),
                ("input_grad", ctypes.c_void_p), ("layer", MlpLayer * MLP_MAX_LAYERS), ("cost", ctypes.c_int32),
                ("target", ctypes.c_void_p), ("labels", ctypes.c_void_p), ("cost_grad", ctypes.c_void_p),
                ("loss", ctypes.c_void_p), ("learning_rate", ctypes.c_float), ("update", ctypes.c_int32),
                ("persistent", ctypes.c_int32)]


class TfdError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"status {status}: {message}")
        self.status = status


_lib = None


def load(path: Optional[str] = None) -> ctypes.CDLL:
    """Load libtfdense (torch is imported first so that the library binds to
    the HIP runtime torch already uses). ``path`` loads another build of the
    same library instead (an explicit choice of the caller, e.g. a tuning
    variant); the first load fixes the library for the process."""
    global _lib
    if _lib is not None:
        if path is not None and os.path.abspath(path) != _lib._name:
            raise RuntimeError(f"libtfdense is already loaded from {_lib._name}")
        return _lib
    lib_path = os.path.abspath(path) if path is not None else LIB_PATH
    if not os.path.exists(lib_path):
        raise RuntimeError(f"{lib_path} is not built; run `python -m paper_1603_04467_amd.build`")
    lib = ctypes.CDLL(lib_path)
    i64, vp, i32, sz = ctypes.c_int64, ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
    sig = {
        "tfd_abi_version": ([], i32),
        "tfd_status_string": ([i32], ctypes.c_char_p),
        "tfd_last_error": ([], ctypes.c_char_p),
        "tfd_matmul": ([i32, i32, i64, i64, i64, vp, i64, i32, vp, i64, i32, vp, i64, i32, vp, i32, vp], i32),
        "tfd_bias_add": ([vp, vp, vp, i64, i64, i32, vp], i32),
        "tfd_relu": ([vp, vp, i64, i32, vp], i32),
        "tfd_relu_grad": ([vp, vp, vp, i64, i32, vp], i32),
        "tfd_reduction_workspace_size": ([i64, i64, i32], sz),
        "tfd_bias_add_grad": ([vp, vp, i64, i64, i32, vp, sz, vp], i32),
        "tfd_relu_grad_bias_add_grad": ([vp, vp, vp, vp, i64, i64, i32, vp, sz, vp], i32),
        "tfd_matmul_relu_grad_workspace_size": ([i64, i64, i32], sz),
        "tfd_matmul_relu_grad_bias_add_grad": ([i32, i32, i64, i64, i64, vp, i64, vp, i64, vp, vp, vp, i32, i32, vp,
                                                sz, vp], i32),
        "tfd_matmul_l2_loss_grad_workspace_size": ([i64, i64, i32], sz),
        "tfd_matmul_l2_loss_grad": ([i32, i32, i64, i64, i64, vp, i64, vp, i64, vp, vp, vp, vp, vp, vp, i32, i32, vp, sz,
                                     vp], i32),
        "tfd_loss_workspace_size": ([i64, i32], sz),
        "tfd_l2_loss_grad": ([vp, vp, vp, vp, i64, i32, vp, sz, vp], i32),
        "tfd_softmax_xent_workspace_size": ([i64], sz),
        "tfd_softmax_cross_entropy_grad": ([vp, vp, vp, vp, i64, i64, i32, vp, sz, vp], i32),
        "tfd_apply_gradient_descent": ([vp, ctypes.c_float, vp, i64, vp, i32, vp], i32),
        "tfd_apply_gradient_descent_matrix": ([vp, ctypes.c_float, vp, i64, i64, vp, vp, i32, vp], i32),
        "tfd_convert_f32_to_bf16": ([vp, vp, i64, i32, vp], i32),
        "tfd_convert_bf16_to_f32": ([vp, vp, i64, vp], i32),
        "tfd_relu_mask": ([vp, vp, i64, i64, i32, vp], i32),
        "tfd_matmul_workspace_size": ([i32, i32, i64, i64, i64, i32, i32, i32], sz),
        "tfd_matmul_with_workspace": ([i32, i32, i64, i64, i64, vp, i64, i32, vp, i64, i32, vp, i64, i32, vp, i32, vp, sz,
                                       vp], i32),
        "tfd_matmul_relu_mask": ([i32, i32, i64, i64, i64, vp, i64, vp, i64, vp, vp, i64, vp, i32, i32, vp], i32),
        "tfd_relu_mask_grad_bias_add_grad": ([vp, vp, vp, vp, i64, i64, i32, vp, sz, vp], i32),
        "tfd_matmul_relu_mask_grad_bias_add_grad": ([i32, i32, i64, i64, i64, vp, i64, vp, i64, vp, vp, vp, i32, i32,
                                                     vp, sz, vp], i32),
        "tfd_set_tuning": ([ctypes.c_char_p, i32], i32),
        "tfd_relu_grad_bias_add_grad_noalloc": ([vp, vp, vp, vp, i64, i64, i32, vp], i32),
        "tfd_clock_probe": ([vp, i64, vp], i32),
        "tfd_mlp_step_workspace_size": ([ctypes.POINTER(MlpStepDesc)], sz),
        "tfd_mlp_step": ([ctypes.POINTER(MlpStepDesc), vp, sz, vp], i32),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    _lib = lib
    return lib


def _check(status: int):
    if status != TFD_OK:
        raise TfdError(status, load().tfd_last_error().decode())


def _dtype(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return TFD_F32
    if t.dtype == torch.bfloat16:
        return TFD_BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else t.data_ptr()


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def _rowmajor(t: torch.Tensor, name: str) -> int:
    """Leading dimension of a 2-D row-major tensor (unit column stride)."""
    if t.dim() != 2:
        raise ValueError(f"{name} must be 2-D")
    if t.numel() == 0:          # an empty matrix: strides carry no meaning
        return max(t.size(1), 1)
    if t.stride(1) != 1 and t.size(1) > 1:
        raise ValueError(f"{name} must have unit column stride")
    return max(t.stride(0), t.size(1), 1)


def _flat(t: torch.Tensor, name: str):
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.numel()


def tfd_abi_version() -> int:
    return load().tfd_abi_version()


TUNING_KNOBS = ("gemm_tile", "bf16_waves_nn", "bf16_waves_nt", "bf16_waves_tn", "small_waves")


def tfd_set_tuning(knob: str, value: int):
    """Force a kernel configuration (tuning and tests only; 0 restores the
    library's choice; see include/tfdense.h)."""
    _check(load().tfd_set_tuning(knob.encode(), int(value)))


class tuning:
    """Context manager: ``with tuning(gemm_tile=9, bf16_waves_nt=4): ...``
    sets knobs and restores the library's choice (0) on exit."""

    def __init__(self, **knobs):
        self.knobs = knobs

    def __enter__(self):
        for k, v in self.knobs.items():
            tfd_set_tuning(k, v)
        return self

    def __exit__(self, *exc):
        for k in self.knobs:
            tfd_set_tuning(k, 0)
        return False


def tfd_matmul_workspace_size(m, n, k, a_dtype, c_dtype, transpose_a=False, transpose_b=False) -> int:
    """Workspace bytes that let tfd_matmul split the k range (0: no split)."""
    td = lambda d: TFD_BF16 if d == torch.bfloat16 else TFD_F32  # noqa: E731
    return load().tfd_matmul_workspace_size(int(transpose_a), int(transpose_b), m, n, k, td(a_dtype), td(a_dtype),
                                            td(c_dtype))


def tfd_matmul(a, b, c, transpose_a=False, transpose_b=False, bias=None, epilogue="none", rounding="nearest",
               workspace=None, stream=None):
    """c = epilogue(op(a) @ op(b)) (see include/tfdense.h); rounding="truncate"
    writes a 16-bit c with the truncating converter. With a `workspace`
    (uint8 device tensor) the call is tfd_matmul_with_workspace, which may
    split the k range of an under-filled problem."""
    lda, ldb, ldc = _rowmajor(a, "a"), _rowmajor(b, "b"), _rowmajor(c, "c")
    m = a.size(1) if transpose_a else a.size(0)
    k = a.size(0) if transpose_a else a.size(1)
    kb = b.size(1) if transpose_b else b.size(0)
    n = b.size(0) if transpose_b else b.size(1)
    if kb != k or tuple(c.shape) != (m, n):
        raise ValueError(f"shape mismatch: op(a) {m}x{k}, op(b) {kb}x{n}, c {tuple(c.shape)}")
    if bias is not None and (bias.dtype != torch.float32 or bias.numel() != n or not bias.is_contiguous()):
        raise ValueError("bias must be a contiguous fp32 vector of length n")
    epi = EPILOGUES[epilogue] | (TFD_EPI_TRUNCATE_16 if ROUNDINGS[rounding] else 0)
    if workspace is None:
        _check(load().tfd_matmul(int(transpose_a), int(transpose_b), m, n, k,
                                 _ptr(a), lda, _dtype(a), _ptr(b), ldb, _dtype(b), _ptr(c), ldc, _dtype(c),
                                 _ptr(bias), epi, _stream(stream)))
    else:
        _check(load().tfd_matmul_with_workspace(int(transpose_a), int(transpose_b), m, n, k,
                                                _ptr(a), lda, _dtype(a), _ptr(b), ldb, _dtype(b), _ptr(c), ldc,
                                                _dtype(c), _ptr(bias), epi, _ptr(workspace), workspace.numel(),
                                                _stream(stream)))
    return c


def tfd_bias_add(value, bias, out, stream=None):
    rows, cols = value.shape
    _flat(value, "value"), _flat(out, "out")
    _check(load().tfd_bias_add(_ptr(value), _ptr(bias), _ptr(out), rows, cols, _dtype(value), _stream(stream)))
    return out


def tfd_relu(features, activations, stream=None):
    n = _flat(features, "features")
    _check(load().tfd_relu(_ptr(features), _ptr(activations), n, _dtype(features), _stream(stream)))
    return activations


def tfd_relu_grad(gradients, features, backprops, stream=None):
    n = _flat(gradients, "gradients")
    _check(load().tfd_relu_grad(_ptr(gradients), _ptr(features), _ptr(backprops), n, _dtype(gradients),
                                _stream(stream)))
    return backprops


def tfd_reduction_workspace_size(rows, cols, dtype) -> int:
    return load().tfd_reduction_workspace_size(rows, cols, TFD_BF16 if dtype == torch.bfloat16 else TFD_F32)


def tfd_matmul_relu_grad_workspace_size(m, n, dtype) -> int:
    return load().tfd_matmul_relu_grad_workspace_size(m, n, TFD_BF16 if dtype == torch.bfloat16 else TFD_F32)


def tfd_matmul_relu_grad_bias_add_grad(a, b, features, backprops, bias_grad, transpose_a=False, transpose_b=False,
                                       rounding="nearest", workspace=None, stream=None):
    """backprops = ReluGrad(op(a) @ op(b), features), bias_grad = its column
    sums (the input-gradient MatMul fused with the lower layer's ReluGrad and
    BiasAddGrad; see include/tfdense.h)."""
    lda, ldb = _rowmajor(a, "a"), _rowmajor(b, "b")
    m = a.size(1) if transpose_a else a.size(0)
    k = a.size(0) if transpose_a else a.size(1)
    kb = b.size(1) if transpose_b else b.size(0)
    n = b.size(0) if transpose_b else b.size(1)
    if kb != k or tuple(backprops.shape) != (m, n) or tuple(features.shape) != (m, n):
        raise ValueError("shape mismatch")
    for t, name in ((features, "features"), (backprops, "backprops")):
        if not t.is_contiguous() or t.dtype != a.dtype:
            raise ValueError(f"{name} must be contiguous with the operands' dtype")
    if b.dtype != a.dtype:
        raise ValueError("a and b must have the same dtype")
    if bias_grad.dtype != torch.float32 or bias_grad.numel() != n or not bias_grad.is_contiguous():
        raise ValueError("bias_grad must be a contiguous fp32 vector of length n")
    ws = _workspace(tfd_matmul_relu_grad_workspace_size(m, n, a.dtype), a.device, workspace)
    _check(load().tfd_matmul_relu_grad_bias_add_grad(int(transpose_a), int(transpose_b), m, n, k, _ptr(a), lda,
                                                     _ptr(b), ldb, _ptr(features), _ptr(backprops), _ptr(bias_grad),
                                                     _dtype(a), ROUNDINGS[rounding], _ptr(ws), ws.numel(),
                                                     _stream(stream)))
    return backprops, bias_grad


def relu_mask_words(cols: int) -> int:
    """uint32 words per row of a ReLU mask of a matrix with ``cols`` columns."""
    return (cols + 31) // 32


def new_relu_mask(rows: int, cols: int, device) -> torch.Tensor:
    """An uninitialised ReLU mask buffer (int32 words holding the uint32 bits)."""
    return torch.empty(rows, relu_mask_words(cols), dtype=torch.int32, device=device)


def _mask(mask: torch.Tensor, rows: int, cols: int):
    if mask.dtype != torch.int32 or tuple(mask.shape) != (rows, relu_mask_words(cols)) or not mask.is_contiguous():
        raise ValueError(f"relu_mask must be a contiguous int32 [{rows}, {relu_mask_words(cols)}] tensor")


def tfd_relu_mask(features, relu_mask, stream=None):
    """relu_mask = one bit per element of features > 0 (see include/tfdense.h)."""
    rows, cols = features.shape
    _flat(features, "features")
    _mask(relu_mask, rows, cols)
    _check(load().tfd_relu_mask(_ptr(features), _ptr(relu_mask), rows, cols, _dtype(features), _stream(stream)))
    return relu_mask


def tfd_matmul_relu_mask(a, b, bias, c, relu_mask, transpose_a=False, transpose_b=False, rounding="nearest",
                         stream=None):
    """c = Relu(op(a) @ op(b) + bias) and relu_mask = the bits of c > 0 (the
    forward MatMul that also records its ReLU mask; see include/tfdense.h)."""
    lda, ldb, ldc = _rowmajor(a, "a"), _rowmajor(b, "b"), _rowmajor(c, "c")
    m = a.size(1) if transpose_a else a.size(0)
    k = a.size(0) if transpose_a else a.size(1)
    kb = b.size(1) if transpose_b else b.size(0)
    n = b.size(0) if transpose_b else b.size(1)
    if kb != k or tuple(c.shape) != (m, n):
        raise ValueError(f"shape mismatch: op(a) {m}x{k}, op(b) {kb}x{n}, c {tuple(c.shape)}")
    if b.dtype != a.dtype or c.dtype != a.dtype:
        raise ValueError("a, b and c must have the same dtype")
    if bias.dtype != torch.float32 or bias.numel() != n or not bias.is_contiguous():
        raise ValueError("bias must be a contiguous fp32 vector of length n")
    _mask(relu_mask, m, n)
    _check(load().tfd_matmul_relu_mask(int(transpose_a), int(transpose_b), m, n, k, _ptr(a), lda, _ptr(b), ldb,
                                       _ptr(bias), _ptr(c), ldc, _ptr(relu_mask), _dtype(a), ROUNDINGS[rounding],
                                       _stream(stream)))
    return c, relu_mask


def tfd_relu_mask_grad_bias_add_grad(gradients, relu_mask, backprops, bias_grad, workspace=None, stream=None):
    """tfd_relu_grad_bias_add_grad with the Relu test read from a ReLU mask."""
    rows, cols = gradients.shape
    _flat(gradients, "gradients")
    _mask(relu_mask, rows, cols)
    if backprops is not None:
        _flat(backprops, "backprops")
    need = tfd_reduction_workspace_size(rows, cols, gradients.dtype)
    ws = _workspace(need, gradients.device, workspace)
    _check(load().tfd_relu_mask_grad_bias_add_grad(_ptr(gradients), _ptr(relu_mask), _ptr(backprops),
                                                   _ptr(bias_grad), rows, cols, _dtype(gradients), _ptr(ws),
                                                   ws.numel(), _stream(stream)))
    return backprops, bias_grad


def tfd_matmul_relu_mask_grad_bias_add_grad(a, b, relu_mask, backprops, bias_grad, transpose_a=False,
                                            transpose_b=False, rounding="nearest", workspace=None, stream=None):
    """tfd_matmul_relu_grad_bias_add_grad with the Relu test read from a ReLU
    mask of the m x n forward output (see include/tfdense.h)."""
    lda, ldb = _rowmajor(a, "a"), _rowmajor(b, "b")
    m = a.size(1) if transpose_a else a.size(0)
    k = a.size(0) if transpose_a else a.size(1)
    kb = b.size(1) if transpose_b else b.size(0)
    n = b.size(0) if transpose_b else b.size(1)
    if kb != k or tuple(backprops.shape) != (m, n):
        raise ValueError("shape mismatch")
    if not backprops.is_contiguous() or backprops.dtype != a.dtype or b.dtype != a.dtype:
        raise ValueError("backprops must be contiguous; a, b and backprops must share a dtype")
    _mask(relu_mask, m, n)
    if bias_grad.dtype != torch.float32 or bias_grad.numel() != n or not bias_grad.is_contiguous():
        raise ValueError("bias_grad must be a contiguous fp32 vector of length n")
    ws = _workspace(tfd_matmul_relu_grad_workspace_size(m, n, a.dtype), a.device, workspace)
    _check(load().tfd_matmul_relu_mask_grad_bias_add_grad(int(transpose_a), int(transpose_b), m, n, k, _ptr(a), lda,
                                                          _ptr(b), ldb, _ptr(relu_mask), _ptr(backprops),
                                                          _ptr(bias_grad), _dtype(a), ROUNDINGS[rounding], _ptr(ws),
                                                          ws.numel(), _stream(stream)))
    return backprops, bias_grad


def tfd_matmul_l2_loss_grad_workspace_size(m, n, dtype) -> int:
    return load().tfd_matmul_l2_loss_grad_workspace_size(m, n, TFD_BF16 if dtype == torch.bfloat16 else TFD_F32)


def tfd_matmul_l2_loss_grad(a, b, bias, output, target, grad, loss, bias_grad, transpose_a=False, transpose_b=False,
                            rounding="nearest", workspace=None, stream=None):
    """output = op(a) @ op(b) + bias, grad = output - target, loss = 1/2 |grad|^2,
    bias_grad = column sums of grad (the output layer fused with the
    squared-error head and its BiasAddGrad; see include/tfdense.h)."""
    lda, ldb = _rowmajor(a, "a"), _rowmajor(b, "b")
    m = a.size(1) if transpose_a else a.size(0)
    k = a.size(0) if transpose_a else a.size(1)
    kb = b.size(1) if transpose_b else b.size(0)
    n = b.size(0) if transpose_b else b.size(1)
    if kb != k or tuple(output.shape) != (m, n) or tuple(grad.shape) != (m, n):
        raise ValueError("shape mismatch")
    for t, name in ((output, "output"), (grad, "grad")) + (() if target is None else ((target, "target"),)):
        if not t.is_contiguous() or t.dtype != a.dtype or tuple(t.shape) != (m, n):
            raise ValueError(f"{name} must be a contiguous {m}x{n} matrix with the operands' dtype")
    if b.dtype != a.dtype:
        raise ValueError("a and b must have the same dtype")
    for t, name in ((bias, "bias"), (bias_grad, "bias_grad")):
        if t.dtype != torch.float32 or t.numel() != n or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous fp32 vector of length n")
    if loss.dtype != torch.float64 or loss.numel() < 1:
        raise ValueError("loss must be a float64 tensor")
    ws = _workspace(tfd_matmul_l2_loss_grad_workspace_size(m, n, a.dtype), a.device, workspace)
    _check(load().tfd_matmul_l2_loss_grad(int(transpose_a), int(transpose_b), m, n, k, _ptr(a), lda, _ptr(b), ldb,
                                          _ptr(bias), _ptr(output), _ptr(target), _ptr(grad), _ptr(loss),
                                          _ptr(bias_grad), _dtype(a), ROUNDINGS[rounding], _ptr(ws), ws.numel(),
                                          _stream(stream)))
    return output, grad, loss, bias_grad


def tfd_loss_workspace_size(count, dtype) -> int:
    return load().tfd_loss_workspace_size(count, TFD_BF16 if dtype == torch.bfloat16 else TFD_F32)


def _workspace(nbytes, device, workspace):
    if workspace is not None:
        return workspace
    return torch.empty(max(nbytes, 1), dtype=torch.uint8, device=device)


def tfd_relu_grad_bias_add_grad(gradients, features, backprops, bias_grad, workspace=None, stream=None):
    rows, cols = gradients.shape
    _flat(gradients, "gradients")
    need = tfd_reduction_workspace_size(rows, cols, gradients.dtype)
    ws = _workspace(need, gradients.device, workspace)
    _check(load().tfd_relu_grad_bias_add_grad(_ptr(gradients), _ptr(features), _ptr(backprops), _ptr(bias_grad),
                                              rows, cols, _dtype(gradients), _ptr(ws), ws.numel(),
                                              _stream(stream)))
    return backprops, bias_grad


def tfd_relu_grad_bias_add_grad_noalloc(gradients, features, backprops, bias_grad, stream=None):
    """tfd_relu_grad_bias_add_grad without a workspace: the library's fixed
    device scratch holds the partials, so nothing is allocated (for callers
    that cannot allocate; calls that overlap on one GPU race)."""
    rows, cols = gradients.shape
    _flat(gradients, "gradients")
    for t, name in ((features, "features"), (backprops, "backprops")):
        if t is not None and (not t.is_contiguous() or t.dtype != gradients.dtype or t.shape != gradients.shape):
            raise ValueError(f"{name} must be contiguous and match gradients")
    if bias_grad.dtype != torch.float32 or bias_grad.numel() != cols or not bias_grad.is_contiguous():
        raise ValueError("bias_grad must be a contiguous fp32 vector of length cols")
    _check(load().tfd_relu_grad_bias_add_grad_noalloc(_ptr(gradients), _ptr(features), _ptr(backprops),
                                                      _ptr(bias_grad), rows, cols, _dtype(gradients),
                                                      _stream(stream)))
    return backprops, bias_grad


def tfd_bias_add_grad(out_backprop, bias_grad, workspace=None, stream=None):
    rows, cols = out_backprop.shape
    _flat(out_backprop, "out_backprop")
    need = tfd_reduction_workspace_size(rows, cols, out_backprop.dtype)
    ws = _workspace(need, out_backprop.device, workspace)
    _check(load().tfd_bias_add_grad(_ptr(out_backprop), _ptr(bias_grad), rows, cols, _dtype(out_backprop),
                                    _ptr(ws), ws.numel(), _stream(stream)))
    return bias_grad


def tfd_l2_loss_grad(output, target, grad, loss, workspace=None, stream=None):
    n = _flat(output, "output")
    need = tfd_loss_workspace_size(n, output.dtype)
    ws = _workspace(need, output.device, workspace)
    _check(load().tfd_l2_loss_grad(_ptr(output), _ptr(target), _ptr(grad), _ptr(loss), n, _dtype(output),
                                   _ptr(ws), ws.numel(), _stream(stream)))
    return grad, loss


def tfd_softmax_xent_workspace_size(rows) -> int:
    return load().tfd_softmax_xent_workspace_size(rows)


def tfd_softmax_cross_entropy_grad(logits, labels, grad, loss, workspace=None, stream=None):
    """grad = softmax(logits) - onehot(labels), loss = summed cross-entropy
    (a float64 device scalar); logits and grad are [rows, cols] contiguous,
    labels int32[rows]."""
    if logits.dim() != 2 or not logits.is_contiguous():
        raise ValueError("logits must be a contiguous matrix")
    rows, cols = logits.shape
    if grad.shape != logits.shape or grad.dtype != logits.dtype or not grad.is_contiguous():
        raise ValueError("grad must match logits")
    if labels.dtype != torch.int32 or labels.numel() != rows or not labels.is_contiguous():
        raise ValueError("labels must be contiguous int32 with one entry per row")
    if loss.dtype != torch.float64 or loss.numel() < 1:
        raise ValueError("loss must be a float64 tensor")
    ws = _workspace(tfd_softmax_xent_workspace_size(rows), logits.device, workspace)
    _check(load().tfd_softmax_cross_entropy_grad(_ptr(logits), _ptr(labels), _ptr(grad), _ptr(loss), rows, cols,
                                                 _dtype(logits), _ptr(ws), ws.numel(), _stream(stream)))
    return grad, loss


def tfd_apply_gradient_descent(var, alpha, delta, var_bf16=None, rounding="nearest", stream=None):
    n = _flat(var, "var")
    if var.dtype != torch.float32 or delta.dtype != torch.float32:
        raise TypeError("Variables and their deltas are fp32")
    if var_bf16 is not None and var_bf16.dtype != torch.bfloat16:
        raise TypeError("the 16-bit copy must be bfloat16")
    _check(load().tfd_apply_gradient_descent(_ptr(var), float(alpha), _ptr(delta), n, _ptr(var_bf16),
                                             ROUNDINGS[rounding], _stream(stream)))
    return var


def tfd_apply_gradient_descent_matrix(var, alpha, delta, var_bf16=None, var_bf16_t=None, rounding="nearest",
                                      stream=None):
    """var[rows, cols] -= alpha * delta (one rounding), refreshing the 16-bit
    copies var_bf16 [rows, cols] and var_bf16_t [cols, rows] when given."""
    if var.dim() != 2 or not var.is_contiguous() or var.dtype != torch.float32:
        raise ValueError("var must be a contiguous fp32 matrix")
    if delta.shape != var.shape or delta.dtype != torch.float32 or not delta.is_contiguous():
        raise ValueError("delta must match var")
    rows, cols = var.shape
    for t, shape in ((var_bf16, (rows, cols)), (var_bf16_t, (cols, rows))):
        if t is not None and (t.dtype != torch.bfloat16 or tuple(t.shape) != shape or not t.is_contiguous()):
            raise ValueError("16-bit copies must be contiguous bfloat16 of the matching shape")
    _check(load().tfd_apply_gradient_descent_matrix(_ptr(var), float(alpha), _ptr(delta), rows, cols,
                                                    _ptr(var_bf16), _ptr(var_bf16_t), ROUNDINGS[rounding],
                                                    _stream(stream)))
    return var


def tfd_convert_f32_to_bf16(src, dst, rounding="truncate", stream=None):
    """dst (bfloat16) = src (fp32) through the 32 -> 16-bit converter;
    rounding "truncate" (the default: the lossy converter) or "nearest"."""
    n = _flat(src, "src")
    if src.dtype != torch.float32 or dst.dtype != torch.bfloat16 or dst.numel() != n or not dst.is_contiguous():
        raise ValueError("src must be fp32 and dst contiguous bfloat16 of the same size")
    _check(load().tfd_convert_f32_to_bf16(_ptr(src), _ptr(dst), n, ROUNDINGS[rounding], _stream(stream)))
    return dst


def tfd_convert_bf16_to_f32(src, dst, stream=None):
    """dst (fp32) = src (bfloat16) with the low 16 bits zero."""
    n = _flat(src, "src")
    if src.dtype != torch.bfloat16 or dst.dtype != torch.float32 or dst.numel() != n or not dst.is_contiguous():
        raise ValueError("src must be bfloat16 and dst contiguous fp32 of the same size")
    _check(load().tfd_convert_bf16_to_f32(_ptr(src), _ptr(dst), n, _stream(stream)))
    return dst


def mlp_step_desc(x, layers, cost, cost_grad, loss, target=None, labels=None, input_grad=None,
                  learning_rate=0.01, update=True, persistent=False):
    """A tfd_mlp_step_desc over fp32 device tensors. ``layers``: one dict per
    layer with weights, bias, activations, backprop (or None), weight_grad,
    bias_grad and relu; ``cost``: "sq_err" or "softmax_xent". The tensors must
    stay alive while the descriptor is used."""
    if len(layers) > MLP_MAX_LAYERS:
        raise ValueError(f"at most {MLP_MAX_LAYERS} layers")
    d = MlpStepDesc()
    d.layers = len(layers)
    d.batch = x.shape[0]
    d.x = _ptr(x)
    d.input_grad = _ptr(input_grad) if input_grad is not None else None
    for i, ly in enumerate(layers):
        w = ly["weights"]
        d.layer[i] = MlpLayer(_ptr(w), _ptr(ly["bias"]), _ptr(ly["activations"]),
                              _ptr(ly["backprop"]) if ly.get("backprop") is not None else None,
                              _ptr(ly["weight_grad"]), _ptr(ly["bias_grad"]), w.shape[0], w.shape[1],
                              1 if ly["relu"] else 0)
    d.cost = COSTS[cost]
    d.target = _ptr(target) if target is not None else None
    d.labels = _ptr(labels) if labels is not None else None
    d.cost_grad = _ptr(cost_grad)
    d.loss = _ptr(loss)
    d.learning_rate = float(learning_rate)
    d.update = 1 if update else 0
    d.persistent = 1 if persistent else 0
    return d


def tfd_mlp_step_workspace_size(desc):
    return int(load().tfd_mlp_step_workspace_size(ctypes.byref(desc)))


def tfd_mlp_step(desc, workspace, stream=None):
    """One whole training step of a small fp32 MLP in one kernel (see the
    header); ``workspace``: a uint8 device tensor whose first 256 bytes are
    zero before its first use."""
    _check(load().tfd_mlp_step(ctypes.byref(desc), _ptr(workspace), workspace.numel() * workspace.element_size(),
                               _stream(stream)))


def tfd_clock_probe(counters, iterations, stream=None):
    """One wave's shader clock cycles and 100 MHz real-time ticks over
    `iterations` dependent FMAs into counters (int64 device tensor of 3)."""
    if counters.dtype != torch.int64 or counters.numel() != 3 or not counters.is_contiguous():
        raise ValueError("counters must be a contiguous int64 tensor of 3 elements")
    _check(load().tfd_clock_probe(_ptr(counters), int(iterations), _stream(stream)))
    return counters
