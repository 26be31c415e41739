"""The C-ABI library loads, exports every entry point that include/tfdense.h
declares, and rejects invalid arguments before launching anything (these
checks run without a GPU: no call here reaches a kernel launch)."""

import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "tfdense.h")


def _declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"TFD_API\s+[\w\s\*]+?\b(tfd_\w+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    from paper_1603_04467_amd import build, tfdense
    if not os.path.exists(tfdense.LIB_PATH):
        build.build()
    return tfdense.load()


def test_header_declares_the_op_set():
    names = _declared()
    for op in ("tfd_matmul", "tfd_bias_add", "tfd_relu", "tfd_relu_grad", "tfd_bias_add_grad",
               "tfd_relu_grad_bias_add_grad", "tfd_l2_loss_grad", "tfd_apply_gradient_descent"):
        assert op in names


def test_every_declared_symbol_is_exported(lib):
    from paper_1603_04467_amd import tfdense
    names = _declared()
    assert set(names) == set(tfdense.EXPORTS)
    for n in names:
        assert hasattr(lib, n), n


def test_version_and_status_strings(lib):
    assert lib.tfd_abi_version() == 5
    assert lib.tfd_status_string(0) == b"ok"
    assert lib.tfd_status_string(1) == b"invalid argument"
    assert lib.tfd_status_string(2) == b"unsupported"
    assert lib.tfd_status_string(3) == b"HIP runtime error"


def test_tuning_knobs(lib):
    """The tuning entry point validates knob names and values (no GPU work)."""
    for knob, bad in ((b"gemm_tile", 10), (b"gemm_tile", -1), (b"bf16_waves_nt", 6), (b"small_waves", 32),
                      (b"no_such_knob", 4)):
        assert lib.tfd_set_tuning(knob, bad) == 1
    assert lib.tfd_set_tuning(None, 0) == 1
    for knob, good in ((b"gemm_tile", 9), (b"bf16_waves_nn", 4), (b"bf16_waves_nt", 16), (b"bf16_waves_tn", 8),
                       (b"small_waves", 8)):
        assert lib.tfd_set_tuning(knob, good) == 0
        assert lib.tfd_set_tuning(knob, 0) == 0


FAKE = 0x10000  # never dereferenced: every call below fails validation first


def test_matmul_validation(lib):
    mm = lib.tfd_matmul
    # negative size
    assert mm(0, 0, -1, 2, 3, FAKE, 3, 0, FAKE, 2, 0, FAKE * 4, 2, 0, None, 0, None) == 1
    assert b"negative" in lib.tfd_last_error()
    # leading dimension too small (A is m x k = 4 x 8, lda 7)
    assert mm(0, 0, 4, 4, 8, FAKE, 7, 0, FAKE * 2, 4, 0, FAKE * 4, 4, 0, None, 0, None) == 1
    assert b"leading dimension" in lib.tfd_last_error()
    # NULL output
    assert mm(0, 0, 4, 4, 4, FAKE, 4, 0, FAKE * 2, 4, 0, None, 4, 0, None, 0, None) == 1
    # bias epilogue without a bias
    assert mm(0, 0, 4, 4, 4, FAKE, 4, 0, FAKE * 2, 4, 0, FAKE * 4, 4, 0, None, 2, None) == 1
    # unsupported type combinations and both transposes
    assert mm(0, 0, 4, 4, 4, FAKE, 4, 0, FAKE * 2, 4, 1, FAKE * 4, 4, 0, None, 0, None) == 2
    assert mm(0, 0, 4, 4, 4, FAKE, 4, 0, FAKE * 2, 4, 0, FAKE * 4, 4, 1, None, 0, None) == 2
    assert mm(1, 1, 4, 4, 4, FAKE, 4, 0, FAKE * 2, 4, 0, FAKE * 4, 4, 0, None, 0, None) == 2
    # unknown dtype / epilogue
    assert mm(0, 0, 4, 4, 4, FAKE, 4, 7, FAKE * 2, 4, 7, FAKE * 4, 4, 7, None, 0, None) == 1
    assert mm(0, 0, 4, 4, 4, FAKE, 4, 0, FAKE * 2, 4, 0, FAKE * 4, 4, 0, None, 9, None) == 1
    # output overlapping an input
    assert mm(0, 0, 4, 4, 4, FAKE, 4, 0, FAKE * 2, 4, 0, FAKE + 16, 4, 0, None, 0, None) == 1
    assert b"overlap" in lib.tfd_last_error()
    # empty output: a successful no-op, even with NULL pointers
    assert mm(0, 0, 0, 4, 4, None, 4, 0, None, 4, 0, None, 4, 0, None, 0, None) == 0
    assert mm(0, 0, 4, 0, 4, None, 4, 0, None, 1, 0, None, 1, 0, None, 0, None) == 0


def test_elementwise_and_reduction_validation(lib):
    assert lib.tfd_relu(None, None, -1, 0, None) == 1
    assert lib.tfd_relu(None, None, 0, 0, None) == 0
    assert lib.tfd_relu(None, FAKE, 5, 0, None) == 1
    assert lib.tfd_relu(FAKE, FAKE + 4, 5, 0, None) == 1          # partial overlap
    assert lib.tfd_relu_grad(FAKE, FAKE * 2, FAKE * 2, 5, 0, None) == 1  # backprops aliases features
    assert lib.tfd_bias_add(FAKE, FAKE * 2, FAKE * 3, -1, 3, 0, None) == 1
    need = lib.tfd_reduction_workspace_size(1000, 300, 0)
    assert need > 0
    assert lib.tfd_reduction_workspace_size(1000, 300, 0) == need  # depends only on the shape
    # workspace too small
    st = lib.tfd_relu_grad_bias_add_grad(FAKE, FAKE * 2, FAKE * 3, FAKE * 4, 1000, 300, 0, FAKE * 5,
                                         need - 1, None)
    assert st == 1 and b"workspace" in lib.tfd_last_error()
    st = lib.tfd_bias_add_grad(FAKE, FAKE * 4, 1000, 300, 0, None, 0, None)
    assert st == 1 and lib.tfd_last_error().startswith(b"tfd_bias_add_grad")
    lneed = lib.tfd_loss_workspace_size(1000, 0)
    assert lneed >= 8
    assert lib.tfd_l2_loss_grad(FAKE, None, FAKE * 2, None, 1000, 0, FAKE * 3, lneed, None) == 1
    assert lib.tfd_apply_gradient_descent(FAKE, ctypes.c_float(0.01), FAKE + 8, 100, None, 0, None) == 1
    assert lib.tfd_apply_gradient_descent(None, ctypes.c_float(0.01), None, 0, None, 0, None) == 0


def test_softmax_and_conversion_validation(lib):
    sneed = lib.tfd_softmax_xent_workspace_size(1000)
    assert sneed >= 8 and lib.tfd_softmax_xent_workspace_size(-1) == 0
    xent = lib.tfd_softmax_cross_entropy_grad
    assert xent(FAKE, FAKE * 2, FAKE * 3, FAKE * 4, -1, 10, 0, FAKE * 5, sneed, None) == 1
    assert xent(FAKE, FAKE * 2, FAKE * 3, FAKE * 4, 1000, 0, 0, FAKE * 5, sneed, None) == 1   # no classes
    assert xent(FAKE, FAKE * 2, FAKE * 3, None, 1000, 10, 0, FAKE * 5, sneed, None) == 1      # no loss
    assert xent(FAKE, FAKE * 2, FAKE * 3, FAKE * 4, 1000, 10, 0, FAKE * 5, sneed - 1, None) == 1
    assert b"workspace" in lib.tfd_last_error()
    assert xent(FAKE, FAKE * 2, FAKE + 64, FAKE * 4, 1000, 10, 0, FAKE * 5, sneed, None) == 1  # grad aliases
    assert b"overlap" in lib.tfd_last_error()
    # conversions: negative count, unknown rounding, overlap, empty no-op
    assert lib.tfd_convert_f32_to_bf16(FAKE, FAKE * 2, -1, 1, None) == 1
    assert lib.tfd_convert_f32_to_bf16(FAKE, FAKE * 2, 10, 7, None) == 1
    assert lib.tfd_convert_f32_to_bf16(FAKE, FAKE + 8, 10, 1, None) == 1
    assert lib.tfd_convert_f32_to_bf16(None, None, 0, 1, None) == 0
    assert lib.tfd_convert_bf16_to_f32(FAKE, FAKE + 8, 10, None) == 1
    assert lib.tfd_convert_bf16_to_f32(None, FAKE, 10, None) == 1
    # the truncating epilogue flag needs a 16-bit output; unknown SGD rounding
    mm = lib.tfd_matmul
    assert mm(0, 0, 4, 4, 4, FAKE, 4, 0, FAKE * 2, 4, 0, FAKE * 4, 4, 0, None, 16, None) == 1
    assert b"16-bit" in lib.tfd_last_error()
    assert mm(0, 0, 4, 4, 4, FAKE, 4, 0, FAKE * 2, 4, 0, FAKE * 4, 4, 0, None, 3 | 16, None) == 1
    assert lib.tfd_apply_gradient_descent(FAKE, ctypes.c_float(0.01), FAKE * 2, 100, None, 5, None) == 1
    assert lib.tfd_apply_gradient_descent_matrix(FAKE, ctypes.c_float(0.01), FAKE * 2, 10, 10, None, None, 5,
                                                 None) == 1

    # clock probe: counters required, iterations in [1, 2^31)
    assert lib.tfd_clock_probe(None, 100, None) == 1
    assert lib.tfd_clock_probe(FAKE, 0, None) == 1
    assert lib.tfd_clock_probe(FAKE, 1 << 31, None) == 1
    assert b"iterations" in lib.tfd_last_error()


def test_fused_relu_grad_matmul_validation(lib):
    f = lib.tfd_matmul_relu_grad_bias_add_grad
    need = lib.tfd_matmul_relu_grad_workspace_size(512, 256, 1)
    assert need >= 2 * 256 * 4
    args = dict(a=FAKE, b=FAKE * 2, feat=FAKE * 3, bp=FAKE * 4, db=FAKE * 5, ws=FAKE * 6)

    def call(ta=0, tb=1, m=512, n=256, k=128, lda=128, ldb=128, dtype=1, rounding=0, ws=args["ws"], ws_bytes=need,
             bp=args["bp"], feat=args["feat"], db=args["db"]):
        return f(ta, tb, m, n, k, args["a"], lda, args["b"], ldb, feat, bp, db, dtype, rounding, ws, ws_bytes, None)

    assert call(m=-1) == 1
    assert call(ta=1, tb=1) == 2
    assert call(lda=64) == 1 and b"leading dimension" in lib.tfd_last_error()
    assert call(ws_bytes=need - 1) == 1 and b"workspace" in lib.tfd_last_error()
    assert call(db=None) == 1
    assert call(feat=None) == 1
    assert call(dtype=0, rounding=1) == 1 and b"16-bit" in lib.tfd_last_error()
    assert call(rounding=9) == 1
    assert call(bp=args["feat"] + 64) == 1 and b"overlap" in lib.tfd_last_error()
    assert call(n=0, feat=None, bp=None, db=None, ws=None, ws_bytes=0) == 0      # nothing to do


def test_relu_mask_validation(lib):
    rm = lib.tfd_relu_mask
    assert rm(FAKE, FAKE * 2, -1, 32, 1, None) == 1
    assert rm(FAKE, FAKE * 2, 4, 32, 7, None) == 1                    # unknown type
    assert rm(None, None, 0, 32, 1, None) == 0                        # empty no-op
    assert rm(FAKE, None, 4, 32, 1, None) == 1
    assert rm(FAKE, FAKE + 8, 4, 32, 1, None) == 1 and b"overlap" in lib.tfd_last_error()
    assert rm(FAKE, FAKE * 2 + 2, 4, 32, 1, None) == 1 and b"aligned" in lib.tfd_last_error()

    mm = lib.tfd_matmul_relu_mask

    def fwd(ta=0, tb=1, m=512, n=256, k=128, lda=128, ldb=128, bias=FAKE * 3, c=FAKE * 4, ldc=256,
            mask=FAKE * 5, dtype=1, rounding=0):
        return mm(ta, tb, m, n, k, FAKE, lda, FAKE * 2, ldb, bias, c, ldc, mask, dtype, rounding, None)

    assert fwd(m=-1) == 1
    assert fwd(ta=1, tb=1) == 2
    assert fwd(ldc=255) == 1 and b"leading dimension" in lib.tfd_last_error()
    assert fwd(mask=None) == 1
    assert fwd(bias=None) == 1
    assert fwd(mask=FAKE * 5 + 2) == 1 and b"aligned" in lib.tfd_last_error()
    assert fwd(dtype=0, rounding=1) == 1 and b"16-bit" in lib.tfd_last_error()
    assert fwd(mask=FAKE * 4 + 64) == 1 and b"overlap" in lib.tfd_last_error()    # mask inside c
    assert fwd(m=0, c=None, mask=None, bias=None) == 0

    need = lib.tfd_reduction_workspace_size(1000, 300, 1)
    g = lib.tfd_relu_mask_grad_bias_add_grad
    assert g(FAKE, FAKE * 2, FAKE * 3, FAKE * 4, -1, 300, 1, FAKE * 5, need, None) == 1
    assert g(FAKE, None, FAKE * 3, FAKE * 4, 1000, 300, 1, FAKE * 5, need, None) == 1
    assert g(FAKE, FAKE * 2, FAKE * 3, FAKE * 4, 1000, 300, 1, FAKE * 5, need - 1, None) == 1
    assert b"workspace" in lib.tfd_last_error()
    assert g(FAKE, FAKE * 2, FAKE * 2 + 64, FAKE * 4, 1000, 300, 1, FAKE * 5, need, None) == 1   # backprops on mask
    assert b"overlap" in lib.tfd_last_error()

    f = lib.tfd_matmul_relu_mask_grad_bias_add_grad
    wneed = lib.tfd_matmul_relu_grad_workspace_size(512, 256, 1)

    def bwd(ta=0, tb=1, m=512, n=256, k=128, lda=128, ldb=128, mask=FAKE * 3, bp=FAKE * 4, db=FAKE * 5,
            dtype=1, rounding=0, ws=FAKE * 6, ws_bytes=wneed):
        return f(ta, tb, m, n, k, FAKE, lda, FAKE * 2, ldb, mask, bp, db, dtype, rounding, ws, ws_bytes, None)

    assert bwd(m=-1) == 1
    assert bwd(ta=1, tb=1) == 2
    assert bwd(lda=64) == 1
    assert bwd(ws_bytes=wneed - 1) == 1 and b"workspace" in lib.tfd_last_error()
    assert bwd(mask=None) == 1
    assert bwd(db=None) == 1
    assert bwd(mask=FAKE * 3 + 1) == 1 and b"aligned" in lib.tfd_last_error()
    assert bwd(bp=FAKE * 3 + 64) == 1 and b"overlap" in lib.tfd_last_error()
    assert bwd(n=0, mask=None, bp=None, db=None, ws=None, ws_bytes=0) == 0


def test_matmul_with_workspace_validation_and_plan(lib):
    ws = lib.tfd_matmul_workspace_size
    # 16-bit, 2 x 64 = 128 output tiles of 256 x 256 and 512 k-tiles: split in two
    assert ws(0, 1, 16384, 512, 32768, 1, 1, 1) == 2 * 16384 * 512 * 4
    assert ws(0, 1, 16384, 512, 32768, 1, 1, 0) == 2 * 16384 * 512 * 4
    assert ws(0, 1, 16384, 4096, 4096, 1, 1, 1) == 0       # 1024 tiles: no split
    assert ws(0, 1, 512, 512, 512, 1, 1, 1) == 0           # 8 k-tiles: too short to split
    assert ws(0, 1, 2048, 512, 32768, 0, 0, 0) == 0        # fp32: no split
    assert ws(0, 1, 300, 512, 32768, 1, 1, 1) == 0         # not whole tiles
    assert ws(1, 1, 2048, 512, 32768, 1, 1, 1) == 0
    assert ws(0, 1, -1, 512, 32768, 1, 1, 1) == 0
    mw = lib.tfd_matmul_with_workspace
    assert mw(0, 0, -1, 2, 3, FAKE, 3, 0, FAKE, 2, 0, FAKE * 4, 2, 0, None, 0, FAKE * 8, 64, None) == 1
    assert lib.tfd_last_error().startswith(b"tfd_matmul_with_workspace: negative")
    assert mw(0, 0, 4, 4, 8, FAKE, 7, 0, FAKE * 2, 4, 0, FAKE * 4, 4, 0, None, 0, FAKE * 8, 64, None) == 1
    assert b"leading dimension" in lib.tfd_last_error()
    assert mw(1, 1, 4, 4, 4, FAKE, 4, 0, FAKE * 2, 4, 0, FAKE * 4, 4, 0, None, 0, FAKE * 8, 64, None) == 2
    assert mw(0, 0, 4, 4, 4, FAKE, 4, 0, FAKE * 2, 4, 0, FAKE + 16, 4, 0, None, 0, FAKE * 8, 64, None) == 1
    assert mw(0, 0, 0, 4, 4, None, 4, 0, None, 4, 0, None, 4, 0, None, 0, None, 0, None) == 0


def _mlp_desc(dims, relus, batch=256, cost=0, fake=FAKE):
    import ctypes as C

    from paper_1603_04467_amd import tfdense as T
    d = T.MlpStepDesc()
    d.layers = len(dims) - 1
    d.batch = batch
    d.x = fake
    d.input_grad = None
    for i in range(len(dims) - 1):
        base = fake * (16 + 8 * i)
        d.layer[i] = T.MlpLayer(base, base + 0x1000, base + 0x2000, base + 0x3000 if relus[i] else None,
                                base + 0x4000, base + 0x5000, dims[i], dims[i + 1], 1 if relus[i] else 0)
    d.cost = cost
    d.target = None
    d.labels = fake * 3 if cost == 1 else None
    d.cost_grad = fake * 5
    d.loss = fake * 6
    d.learning_rate = C.c_float(0.01)
    d.update = 1
    return d


def test_fused_step_validation(lib):
    """tfd_mlp_step: the descriptor is read field by field (the workspace size
    follows the cost head's item count) and rejected before any launch."""
    import ctypes as C
    step = lib.tfd_mlp_step
    size = lib.tfd_mlp_step_workspace_size
    d = _mlp_desc((784, 1024, 1024, 10), (1, 1, 0))
    # 4096 control bytes, one float64 loss partial per 256 elements of G
    # (256 x 10), padded to 256 bytes, then the output layer's forward split
    # into 8 k chunks of fp32 partial products (8 tiles of 32 x 32 < 64)
    split = 4 * 8 * 256 * 10
    assert size(C.byref(d)) == 4352 + split
    dx = _mlp_desc((784, 1024, 1024, 10), (1, 1, 0), cost=1)
    assert size(C.byref(dx)) == 4096 + 8 * 64 + split           # one loss partial per 4 rows
    wide = _mlp_desc((784, 4096, 4096), (1, 1), batch=512)    # 256 output tiles: no split
    assert size(C.byref(wide)) == 4096 + 8 * 8192              # 512 x 4096 / 256 loss partials
    assert step(C.byref(d), FAKE * 9, 4352 + split - 1, None) == 1
    assert b"workspace" in lib.tfd_last_error()
    assert step(C.byref(d), FAKE * 9 + 4, 1 << 20, None) == 1   # misaligned
    assert b"aligned" in lib.tfd_last_error()
    bad = _mlp_desc((784, 1024, 1024, 10), (1, 0, 0))           # hidden layer without Relu
    assert step(C.byref(bad), FAKE * 9, 8192, None) == 2
    bad = _mlp_desc((784, 1024, 1024, 10), (1, 1, 0))
    bad.layer[1].fan_in = 1000                                  # fans do not chain
    assert step(C.byref(bad), FAKE * 9, 8192, None) == 1 and b"fan_in" in lib.tfd_last_error()
    bad = _mlp_desc((784, 100), (1,))
    bad.layer[0].backprop = None                                # Relu layer without dY buffer
    assert step(C.byref(bad), FAKE * 9, 8192, None) == 1
    bad = _mlp_desc((784, 100), (1,), cost=1)
    bad.labels = None
    assert step(C.byref(bad), FAKE * 9, 8192, None) == 1
    bad = _mlp_desc((784, 100), (1,))
    bad.layers = 5
    assert step(C.byref(bad), FAKE * 9, 8192, None) == 1 and size(C.byref(bad)) == 0
    bad = _mlp_desc((784, 100), (1,), batch=-1)
    assert step(C.byref(bad), FAKE * 9, 8192, None) == 1
    assert step(None, FAKE * 9, 8192, None) == 1
    empty = _mlp_desc((784, 100), (1,), batch=0)
    assert step(C.byref(empty), None, 0, None) == 0              # nothing to do
