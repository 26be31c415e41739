"""Per-op parity of the HIP kernels against the oracle, through the C ABI.

Inputs are seeded host arrays handed to both sides; the oracle never sees a
value produced on the GPU. Shapes span several tiles of every GEMM tile
configuration, ragged tails, unaligned rows (the per-element load path) and
strided leading dimensions.
"""

import numpy as np
import pytest
import torch

import oracle
from paper_1603_04467_amd import tfdense as T
from paper_1603_04467_amd.workloads import to_bf16_bits
from tests.parity import (TAU, amax, assert_bits, assert_close, assert_elementwise, check_relu_decisions,
                          mask_mismatch, product_bound, to_f64)

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _host(rng, shape, dt, scale=1.0, kind="normal"):
    """Seeded operand: float64 values exactly representable in `dt` and the
    matching device tensor."""
    if kind == "normal":
        a = (rng.standard_normal(shape) * scale).astype(np.float32)
    elif kind == "int":
        a = rng.integers(-2, 3, size=shape).astype(np.float32)
    else:
        raise ValueError(kind)
    if dt == "bf16":
        bits = to_bf16_bits(a)
        t = torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).to(DEV)
        return oracle.bf16_bits_to_f64(bits), t
    return a.astype(np.float64), torch.from_numpy(a).to(DEV)


def _empty(shape, dt, ld=None):
    tdt = torch.bfloat16 if dt == "bf16" else torch.float32
    if ld is None or ld == shape[1]:
        return torch.full(shape, float("nan"), dtype=tdt, device=DEV)
    big = torch.full((shape[0], ld), float("nan"), dtype=tdt, device=DEV)
    return big[:, : shape[1]]


def _strided(host, t, extra):
    """Copy `t` into a wider buffer so that its leading dimension grows by `extra`."""
    if extra == 0:
        return t
    big = torch.zeros(t.shape[0], t.shape[1] + extra, dtype=t.dtype, device=DEV)
    big[:, : t.shape[1]] = t
    return big[:, : t.shape[1]]


def _check_elementwise(got, a_h, b_h, ta, tb, bias_h, epi, store, what):
    """Per-element product bound on the operands the kernel read, and exact
    ReLU decisions outside its band."""
    A = a_h.T if ta else a_h
    B = b_h.T if tb else b_h
    K = A.shape[1]
    y = oracle.matmul(A, B, out="f64", bias=None if epi == "none" else bias_h)
    bound = product_bound(np.abs(A) @ np.abs(B), K, got, store,
                          abs_bias=None if epi == "none" else np.abs(bias_h))
    assert_elementwise(got, oracle.relu(y) if epi == "bias_relu" else y, bound, what)
    if epi == "bias_relu":
        check_relu_decisions(got, y, bound, what)


_LAST = {}   # host operands of the latest _run_gemm call


def _run_gemm(m, n, k, layout, din, dout, epi, seed=0, kind="normal", ld_extra=0, tile=None):
    rng = np.random.default_rng([seed, m, n, k])
    ta, tb = layout == "TN", layout == "NT"
    a_h, a = _host(rng, (k, m) if ta else (m, k), din, kind=kind)
    b_h, b = _host(rng, (n, k) if tb else (k, n), din, kind=kind)
    a, b = _strided(a_h, a, ld_extra), _strided(b_h, b, ld_extra)
    bias_h = bias = None
    if epi != "none":
        bias_h = (rng.standard_normal(n) * 0.5).astype(np.float32)
        bias = torch.from_numpy(bias_h).to(DEV)
        bias_h = bias_h.astype(np.float64)
    c = _empty((m, n), dout, ld=n + ld_extra if ld_extra else None)
    with T.tuning(gemm_tile=tile or 0):
        T.tfd_matmul(a, b, c, transpose_a=ta, transpose_b=tb, bias=bias, epilogue=epi)
        torch.cuda.synchronize()
    want = oracle.matmul(a_h, b_h, ta, tb, out=dout, bias=bias_h, relu=epi == "bias_relu")
    pre = oracle.matmul(a_h, b_h, ta, tb, out="f64", bias=bias_h)
    _LAST.update(a=a_h, b=b_h, bias=bias_h)
    D = k * amax(a_h) * amax(b_h) + (amax(bias_h) if bias_h is not None else 0.0)
    return to_f64(c), want, pre, D


SHAPES = [(1, 1, 1), (3, 5, 7), (32, 32, 32), (64, 64, 64), (65, 33, 17), (100, 100, 784),
          (127, 129, 200), (256, 10, 1024), (300, 264, 136), (513, 256, 96), (1000, 784, 100)]
TYPES = [("f32", "f32"), ("bf16", "bf16"), ("bf16", "f32")]


@pytest.mark.parametrize("din,dout", TYPES)
@pytest.mark.parametrize("layout", ["NN", "NT", "TN"])
@pytest.mark.parametrize("m,n,k", SHAPES)
def test_matmul_parity(m, n, k, layout, din, dout):
    epi = "bias_relu" if layout == "NN" else "none"
    got, want, pre, D = _run_gemm(m, n, k, layout, din, dout, epi)
    assert_close(got, want, D, TAU[din], f"{layout} {din}->{dout} {m}x{n}x{k}")
    a_h, b_h, bias_h = _LAST["a"], _LAST["b"], _LAST["bias"]
    _check_elementwise(got, a_h, b_h, layout == "TN", layout == "NT", bias_h, epi, dout,
                       f"{layout} {din}->{dout} {m}x{n}x{k} per element")
    if epi == "bias_relu":
        assert not np.any(np.signbit(got)), "Relu output with a sign bit"
        bad, _ = mask_mismatch(got, pre, TAU[din] * D)
        assert bad == 0, f"{bad} Relu mask decisions differ outside the rounding band"


@pytest.mark.parametrize("tile", [1, 2, 3, 4, 5, 6, 7, 8, 9])
@pytest.mark.parametrize("layout", ["NN", "NT", "TN"])
@pytest.mark.parametrize("din,dout", TYPES)
def test_matmul_every_tile_config(tile, layout, din, dout):
    m, n, k = 600, 520, 264   # ragged against 256 and 128 in m, several k-tiles
    got, want, pre, D = _run_gemm(m, n, k, layout, din, dout, "bias", seed=tile, tile=tile)
    assert_close(got, want, D, TAU[din], f"tile {tile} {layout} {din}->{dout}")


WHOLE_TILES = [(256, 256, 64), (512, 768, 192), (768, 512, 1024), (1024, 256, 4096)]


@pytest.mark.parametrize("epi", ["none", "bias", "bias_relu"])
@pytest.mark.parametrize("layout", ["NN", "NT", "TN"])
@pytest.mark.parametrize("m,n,k", [(256, 256, 32), *WHOLE_TILES])
def test_matmul_f32_whole_tiles(m, n, k, layout, epi):
    """fp32 operands on whole 256 x 256 tiles: the direct-to-LDS kernel
    (configuration 9, the default from 128 such tiles up), one k-tile and
    many, against the oracle."""
    got, want, pre, D = _run_gemm(m, n, k, layout, "f32", "f32", epi, seed=k + 1, tile=9)
    assert_close(got, want, D, TAU["f32"], f"{layout} f32 {m}x{n}x{k} {epi}")
    _check_elementwise(got, _LAST["a"], _LAST["b"], layout == "TN", layout == "NT", _LAST["bias"], epi, "f32",
                       f"{layout} f32 {m}x{n}x{k} {epi} per element")
    if epi == "bias_relu":
        assert not np.any(np.signbit(got)), "Relu output with a sign bit"
        bad, _ = mask_mismatch(got, pre, TAU["f32"] * D)
        assert bad == 0


@pytest.mark.parametrize("epi", ["none", "bias", "bias_relu"])
@pytest.mark.parametrize("dout", ["bf16", "f32"])
@pytest.mark.parametrize("layout", ["NN", "NT", "TN"])
@pytest.mark.parametrize("m,n,k", WHOLE_TILES)
def test_matmul_bf16_whole_tiles(m, n, k, layout, dout, epi):
    """16-bit operands on whole 256 x 256 tiles (the direct-to-LDS kernel)."""
    got, want, pre, D = _run_gemm(m, n, k, layout, "bf16", dout, epi, seed=k)
    assert_close(got, want, D, TAU["bf16"], f"{layout} bf16->{dout} {m}x{n}x{k} {epi}")
    _check_elementwise(got, _LAST["a"], _LAST["b"], layout == "TN", layout == "NT", _LAST["bias"], epi, dout,
                       f"{layout} bf16->{dout} {m}x{n}x{k} {epi} per element")
    if epi == "bias_relu":
        bad, _ = mask_mismatch(got, pre, TAU["bf16"] * D)
        assert bad == 0


@pytest.mark.parametrize("waves", [4, 8, 16])
@pytest.mark.parametrize("layout", ["NN", "NT", "TN"])
def test_matmul_bf16_every_wave_layout(layout, waves):
    """Every workgroup shape of the whole-tile kernel (the tuning knob)."""
    with T.tuning(bf16_waves_nn=waves, bf16_waves_nt=waves, bf16_waves_tn=waves):
        got, want, _, D = _run_gemm(512, 768, 320, layout, "bf16", "bf16", "bias", seed=waves)
        assert_close(got, want, D, TAU["bf16"], f"{layout} waves {waves}")
        _check_elementwise(got, _LAST["a"], _LAST["b"], layout == "TN", layout == "NT", _LAST["bias"], "bias",
                           "bf16", f"{layout} waves {waves} per element")
        got, want, _, _ = _run_gemm(512, 256, 128, layout, "bf16", "f32", "none", kind="int")
        assert_bits(got, want, f"integer {layout} waves {waves}")



@pytest.mark.parametrize("layout", ["NN", "NT", "TN"])
def test_matmul_bf16_whole_tiles_integers_exact(layout):
    got, want, _, _ = _run_gemm(512, 512, 64, layout, "bf16", "bf16", "none", kind="int")
    assert_bits(got, want, f"integer whole tiles {layout}")
    got, want, _, _ = _run_gemm(512, 256, 128, layout, "bf16", "f32", "none", kind="int")
    assert_bits(got, want, f"integer whole tiles {layout} f32 out")


@pytest.mark.parametrize("layout", ["NN", "NT", "TN"])
@pytest.mark.parametrize("din", ["f32", "bf16"])
def test_matmul_small_integers_exact(layout, din):
    # integer operands in [-2, 2]: every partial sum is an exact integer < 2**24,
    # |C| <= 4 * 64 = 256 is exact in both output types
    got, want, _, _ = _run_gemm(200, 136, 64, layout, din, din, "none", kind="int")
    assert_bits(got, want, f"integer {layout} {din}")


@pytest.mark.parametrize("layout", ["NN", "NT", "TN"])
@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("rows,n", [(264, 136), (512, 256)])
def test_matmul_identity_and_permutation_bit_exact(layout, dt, rows, n):
    rng = np.random.default_rng(9)
    x_h, x = _host(rng, (rows, n), dt)
    perm = rng.permutation(n)
    P = np.ascontiguousarray(np.eye(n)[:, perm])
    P_dev = torch.from_numpy(P.astype(np.float32)).to(DEV).to(x.dtype)
    out = _empty((rows, n), dt)
    if layout == "NN":
        T.tfd_matmul(x, P_dev, out)                                   # x @ P
        want = x_h[:, perm]
    elif layout == "NT":
        T.tfd_matmul(x, P_dev.t().contiguous(), out, transpose_b=True)  # x @ (P^T)^T
        want = x_h[:, perm]
    else:
        xt = x.t().contiguous()
        T.tfd_matmul(xt, P_dev, out, transpose_a=True)               # (x^T)^T @ P
        want = x_h[:, perm]
    torch.cuda.synchronize()
    assert_bits(to_f64(out), want, f"permutation {layout} {dt}")


@pytest.mark.parametrize("ld_extra", [4, 8, 24])
@pytest.mark.parametrize("layout", ["NN", "NT", "TN"])
def test_matmul_leading_dimensions(layout, ld_extra):
    got, want, _, D = _run_gemm(130, 72, 88, layout, "f32", "f32", "bias", ld_extra=ld_extra)
    assert_close(got, want, D, TAU["f32"], f"ld+{ld_extra} {layout}")
    got, want, _, D = _run_gemm(130, 72, 88, layout, "bf16", "bf16", "bias", ld_extra=ld_extra)
    assert_close(got, want, D, TAU["bf16"], f"ld+{ld_extra} {layout} bf16")


@pytest.mark.parametrize("ld_extra", [4, 36])
@pytest.mark.parametrize("layout", ["NN", "NT", "TN"])
def test_matmul_f32_whole_tiles_leading_dimensions(layout, ld_extra):
    """Strided operands and output in the fp32 whole-tile kernel."""
    got, want, _, D = _run_gemm(512, 256, 96, layout, "f32", "f32", "bias", ld_extra=ld_extra, tile=9)
    assert_close(got, want, D, TAU["f32"], f"ld+{ld_extra} {layout} whole tiles")


def test_matmul_k_zero_gives_relu_of_bias():
    bias = torch.tensor([0.5, -1.0, 0.0, 2.0], device=DEV)
    a = torch.empty(3, 0, device=DEV)
    b = torch.empty(0, 4, device=DEV)
    c = torch.full((3, 4), float("nan"), device=DEV)
    T.tfd_matmul(a, b, c, bias=bias, epilogue="bias_relu")
    torch.cuda.synchronize()
    assert_bits(to_f64(c), np.array([[0.5, 0.0, 0.0, 2.0]] * 3), "k=0")


def test_matmul_is_deterministic():
    a = torch.randn(1000, 777, device=DEV)
    b = torch.randn(777, 512, device=DEV)
    c1 = torch.empty(1000, 512, device=DEV)
    c2 = torch.empty(1000, 512, device=DEV)
    T.tfd_matmul(a, b, c1)
    T.tfd_matmul(a, b, c2)
    torch.cuda.synchronize()
    assert torch.equal(c1, c2)


# ---------------------------------------------------------------- element-wise

@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("count", [1, 7, 8, 1000, 4096 * 3 + 5])
def test_relu_and_relu_grad_bit_exact(dt, count):
    rng = np.random.default_rng(count)
    x_h, x = _host(rng, (count,), dt)
    x[: min(count, 3)] = torch.tensor([0.0, -0.0, -1.0], dtype=x.dtype, device=DEV)[: min(count, 3)]
    x_h = to_f64(x)
    g_h, g = _host(rng, (count,), dt)
    y = torch.empty_like(x)
    T.tfd_relu(x, y)
    bp = torch.empty_like(x)
    T.tfd_relu_grad(g, x, bp)
    torch.cuda.synchronize()
    assert_bits(to_f64(y), oracle.relu(x_h), "relu")
    assert_bits(to_f64(bp), oracle.relu_grad(g_h, x_h), "relu_grad")
    # in place
    T.tfd_relu(x, x)
    torch.cuda.synchronize()
    assert_bits(to_f64(x), oracle.relu(x_h), "relu in place")


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("rows,cols", [(1, 1), (5, 10), (64, 4096), (33, 1029)])
def test_bias_add(dt, rows, cols):
    rng = np.random.default_rng(rows * 7 + cols)
    v_h, v = _host(rng, (rows, cols), dt)
    b32 = rng.standard_normal(cols).astype(np.float32)
    out = torch.empty_like(v)
    T.tfd_bias_add(v, torch.from_numpy(b32).to(DEV), out)
    torch.cuda.synchronize()
    want = oracle.bias_add(v_h, b32.astype(np.float64), out=dt)
    if dt == "f32":
        assert_bits(to_f64(out), want, "bias_add f32")   # one correctly rounded fp32 add
    else:
        assert_close(to_f64(out), want, amax(v_h) + float(np.max(np.abs(b32))), TAU["bf16"], "bias_add bf16")


@pytest.mark.parametrize("count", [1, 3, 4, 1000, 16 * 1024 + 3])
@pytest.mark.parametrize("shadow", [False, True])
def test_apply_gradient_descent_bit_exact(count, shadow):
    rng = np.random.default_rng(count)
    var = rng.standard_normal(count).astype(np.float32)
    delta = (rng.standard_normal(count) * 10.0 ** rng.integers(-6, 4, count)).astype(np.float32)
    v = torch.from_numpy(var).to(DEV)
    d = torch.from_numpy(delta).to(DEV)
    sh = torch.empty(count, dtype=torch.bfloat16, device=DEV) if shadow else None
    T.tfd_apply_gradient_descent(v, 0.01, d, var_bf16=sh)
    torch.cuda.synchronize()
    want = oracle.apply_gradient_descent(var, np.float32(0.01), delta)
    assert_bits(to_f64(v), want, "sgd")
    if shadow:
        assert_bits(to_f64(sh), oracle.round_bf16(want), "sgd shadow")


@pytest.mark.parametrize("rows,cols", [(1, 1), (3, 5), (64, 64), (100, 37), (130, 72), (512, 768), (4096, 4096)])
def test_apply_gradient_descent_matrix_bit_exact(rows, cols):
    rng = np.random.default_rng([rows, cols])
    var = rng.standard_normal((rows, cols)).astype(np.float32)
    delta = (rng.standard_normal((rows, cols)) * 10.0 ** rng.integers(-6, 4, (rows, cols))).astype(np.float32)
    v = torch.from_numpy(var).to(DEV)
    d = torch.from_numpy(delta).to(DEV)
    sh = torch.empty(rows, cols, dtype=torch.bfloat16, device=DEV)
    sht = torch.empty(cols, rows, dtype=torch.bfloat16, device=DEV)
    T.tfd_apply_gradient_descent_matrix(v, 0.01, d, var_bf16=sh, var_bf16_t=sht)
    torch.cuda.synchronize()
    want = oracle.apply_gradient_descent(var, np.float32(0.01), delta)
    assert_bits(to_f64(v), want, "sgd matrix")
    assert_bits(to_f64(sh), oracle.round_bf16(want), "sgd matrix copy")
    assert_bits(to_f64(sht), oracle.round_bf16(want).T, "sgd matrix transposed copy")
    # copies are optional
    v2 = torch.from_numpy(var).to(DEV)
    T.tfd_apply_gradient_descent_matrix(v2, 0.01, d)
    torch.cuda.synchronize()
    assert torch.equal(v, v2)


def test_apply_gradient_descent_lr_zero_is_identity():
    var = torch.randn(12345, device=DEV)
    keep = var.clone()
    T.tfd_apply_gradient_descent(var, 0.0, torch.randn(12345, device=DEV))
    torch.cuda.synchronize()
    assert torch.equal(var, keep)


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("count", [1, 9, 100 * 100, 256 * 10, 1 << 20])
@pytest.mark.parametrize("with_target", [False, True])
def test_l2_loss_grad(dt, count, with_target):
    rng = np.random.default_rng(count + with_target)
    o_h, o = _host(rng, (count,), dt)
    t_h, t = _host(rng, (count,), dt) if with_target else (None, None)
    g = torch.empty_like(o)
    loss = torch.zeros(1, dtype=torch.float64, device=DEV)
    T.tfd_l2_loss_grad(o, t, g, loss)
    torch.cuda.synchronize()
    g_want, l_want = oracle.l2_loss_grad(o_h, t_h, grad_dtype=dt)
    assert_bits(to_f64(g), g_want, "loss gradient")
    assert abs(loss.item() - l_want) <= 1e-6 * l_want


# ---------------------------------------------------------------- reductions

@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("rows,cols", [(1, 1), (3, 5), (16, 4096), (1000, 300), (257, 1029), (8192, 4096),
                                       (0, 7)])
@pytest.mark.parametrize("mask", [True, False])
def test_relu_grad_bias_add_grad(dt, rows, cols, mask):
    rng = np.random.default_rng([rows, cols, mask])
    g_h, g = _host(rng, (rows, cols), dt)
    f_h, f = _host(rng, (rows, cols), dt)
    db = torch.full((cols,), float("nan"), device=DEV)
    if mask:
        bp = torch.empty_like(g)
        T.tfd_relu_grad_bias_add_grad(g, f, bp, db)
        dy = oracle.relu_grad(g_h, f_h)
    else:
        T.tfd_bias_add_grad(g, db)
        dy = g_h
    torch.cuda.synchronize()
    if mask:
        assert_bits(to_f64(bp), dy, "ReluGrad output")
    want = oracle.bias_add_grad(dy)
    D = max(rows, 1) * max(amax(dy), 1e-30)
    assert_close(to_f64(db), want, D, TAU["f32"], "BiasAddGrad")
    # the summation order is fixed: a second call gives the same bits
    db2 = torch.empty_like(db)
    if mask:
        T.tfd_relu_grad_bias_add_grad(g, f, None, db2)
    else:
        T.tfd_bias_add_grad(g, db2)
    torch.cuda.synchronize()
    assert torch.equal(db, db2)


# ------------------------------------- fused input gradient + ReluGrad + BiasAddGrad

@pytest.mark.parametrize("m,n,k,layout,dt,rounding", [
    (512, 768, 512, "NT", "bf16", "nearest"),     # whole 256 tiles: the fused epilogue
    (1024, 512, 768, "NN", "bf16", "nearest"),
    (512, 256, 1024, "TN", "bf16", "nearest"),
    (512, 768, 512, "NT", "bf16", "truncate"),
    (300, 200, 136, "NT", "bf16", "nearest"),     # ragged: MatMul, then ReluGrad in place
    (256, 1024, 1024, "NT", "f32", "nearest"),    # fp32 small-problem path
    (1024, 512, 256, "NT", "f32", "nearest"),
    (0, 64, 32, "NT", "f32", "nearest"),          # no rows: bias_grad = 0
])
def test_matmul_relu_grad_bias_add_grad(m, n, k, layout, dt, rounding):
    rng = np.random.default_rng([m, n, k, len(layout), dt == "bf16", rounding == "truncate"])
    ta, tb = layout == "TN", layout == "NT"
    a_h, a = _host(rng, (k, m) if ta else (m, k), dt)
    b_h, b = _host(rng, (n, k) if tb else (k, n), dt)
    f_h, f = _host(rng, (m, n), dt)
    bp = _empty((m, n), dt)
    db = torch.full((n,), float("nan"), device=DEV)
    T.tfd_matmul_relu_grad_bias_add_grad(a, b, f, bp, db, transpose_a=ta, transpose_b=tb, rounding=rounding)
    # the two calls it replaces
    g = _empty((m, n), dt)
    T.tfd_matmul(a, b, g, transpose_a=ta, transpose_b=tb, rounding=rounding)
    bp2 = _empty((m, n), dt)
    db2 = torch.full((n,), float("nan"), device=DEV)
    T.tfd_relu_grad_bias_add_grad(g, f, bp2, db2)
    torch.cuda.synchronize()
    assert torch.equal(bp, bp2), "backprops differ from MatMul + ReluGrad"
    # ReluGrad is an exact select: the fused dY is the oracle's ReluGrad of
    # the plain MatMul's output, bit for bit
    dy = to_f64(bp)
    assert_bits(dy, oracle.relu_grad(to_f64(g), f_h), "fused dY = ReluGrad(plain MatMul output)")
    D = max(m, 1) * max(amax(dy), 1e-30)
    assert_close(to_f64(db), oracle.bias_add_grad(dy), D, TAU["f32"], "fused BiasAddGrad")
    _check_colsum(to_f64(db), dy, "fused BiasAddGrad per column")
    # against the oracle's chain (mask decisions are exact here: features are given)
    store = "bf16t" if rounding == "truncate" else dt
    want = oracle.relu_grad(oracle.matmul(a_h, b_h, ta, tb, out=store), f_h)
    Dg = k * amax(a_h) * amax(b_h)
    assert_close(dy, want, Dg, TAU[dt], "fused dY")
    if m > 0:
        keep = f_h > 0
        A, B = (a_h.T if ta else a_h), (b_h.T if tb else b_h)
        exact = oracle.matmul(A, B, out="f64")
        bound = product_bound(np.abs(A) @ np.abs(B), k, dy, store)
        assert_elementwise(np.where(keep, dy, 0.0), np.where(keep, exact, 0.0), bound, "fused dY per element")
    # fixed summation order: a second call gives the same bits
    db3 = torch.empty_like(db)
    T.tfd_matmul_relu_grad_bias_add_grad(a, b, f, torch.empty_like(bp), db3, transpose_a=ta, transpose_b=tb,
                                         rounding=rounding)
    torch.cuda.synchronize()
    assert torch.equal(db, db3)


def _check_colsum(db, dy, what):
    """fp32 column sums of dy: within C_ACC * rows * u * sum |dy| + half an ulp."""
    from tests.parity import C_ACC, U32, ulp
    rows = dy.shape[0]
    bound = C_ACC * rows * U32 * np.abs(dy).sum(axis=0) + 0.5 * ulp(db, "f32")
    assert_elementwise(db, oracle.bias_add_grad(dy, out="f64"), bound, what)


# ------------------------------------- fused output layer + squared error + BiasAddGrad

@pytest.mark.parametrize("m,n,k,layout,dt,rounding,with_target", [
    (512, 768, 512, "NT", "bf16", "nearest", True),     # whole 256 tiles: the fused epilogue
    (1024, 512, 768, "NN", "bf16", "nearest", True),
    (512, 256, 1024, "TN", "bf16", "nearest", True),
    (512, 768, 512, "NT", "bf16", "truncate", True),
    (512, 768, 512, "NT", "bf16", "nearest", False),   # no target: MatMul, then the two calls
    (300, 200, 136, "NT", "bf16", "nearest", True),     # ragged
    (256, 1024, 1024, "NN", "f32", "nearest", True),
    (256, 10, 1024, "NN", "f32", "nearest", False),
    (0, 64, 32, "NT", "f32", "nearest", True),
])
def test_matmul_l2_loss_grad(m, n, k, layout, dt, rounding, with_target):
    rng = np.random.default_rng([m, n, k, len(layout), dt == "bf16", rounding == "truncate", with_target])
    ta, tb = layout == "TN", layout == "NT"
    a_h, a = _host(rng, (k, m) if ta else (m, k), dt)
    b_h, b = _host(rng, (n, k) if tb else (k, n), dt)
    t_h, t = _host(rng, (m, n), dt) if with_target else (None, None)
    bias_h = (rng.standard_normal(n) * 0.5).astype(np.float32)
    bias = torch.from_numpy(bias_h).to(DEV)
    out, g = _empty((m, n), dt), _empty((m, n), dt)
    loss = torch.full((1,), float("nan"), dtype=torch.float64, device=DEV)
    db = torch.full((n,), float("nan"), device=DEV)
    T.tfd_matmul_l2_loss_grad(a, b, bias, out, t, g, loss, db, transpose_a=ta, transpose_b=tb, rounding=rounding)
    # the three calls it replaces
    out2, g2 = _empty((m, n), dt), _empty((m, n), dt)
    loss2 = torch.full((1,), float("nan"), dtype=torch.float64, device=DEV)
    db2 = torch.full((n,), float("nan"), device=DEV)
    T.tfd_matmul(a, b, out2, transpose_a=ta, transpose_b=tb, bias=bias, epilogue="bias", rounding=rounding)
    T.tfd_l2_loss_grad(out2, t, g2, loss2)
    T.tfd_bias_add_grad(g2, db2)
    torch.cuda.synchronize()
    assert torch.equal(out, out2) and torch.equal(g, g2), "output or gradient differs from the three calls"
    l1, l2 = loss.item(), loss2.item()
    assert abs(l1 - l2) <= 1e-10 * max(abs(l2), 1e-300), (l1, l2)   # float64 sums in another order
    gh = to_f64(g2)
    assert_close(to_f64(db), oracle.bias_add_grad(gh), max(m, 1) * max(amax(gh), 1e-30), TAU["f32"], "fused db")
    # against the oracle: output within the GEMM tolerance, gradient exact from the stored output
    store = "bf16t" if rounding == "truncate" else dt
    want = oracle.matmul(a_h, b_h, ta, tb, out=store, bias=bias_h.astype(np.float64))
    assert_close(to_f64(out), want, k * amax(a_h) * amax(b_h) + amax(bias_h), TAU[dt], "fused output")
    g_want, l_want = oracle.l2_loss_grad(to_f64(out), t_h, grad_dtype=dt)
    assert_bits(gh, g_want, "fused gradient")
    assert abs(l1 - l_want) <= 1e-6 * max(l_want, 1e-300)
    # fixed summation order
    loss3 = torch.empty_like(loss)
    db3 = torch.empty_like(db)
    T.tfd_matmul_l2_loss_grad(a, b, bias, torch.empty_like(out), t, torch.empty_like(g), loss3, db3,
                              transpose_a=ta, transpose_b=tb, rounding=rounding)
    torch.cuda.synchronize()
    assert torch.equal(loss, loss3) and torch.equal(db, db3)
