"""ReLU masks (one bit per element of the test ReluGrad applies, H > 0):
parity of the mask kernels and of the mask-based calls through the C ABI.

The mask is a pure function of a stored tensor, so every mask is compared
bit for bit with the oracle's mask of the same values; each mask-based call
must store exactly what its features-based counterpart stores.
"""

import numpy as np
import pytest
import torch

import oracle
from paper_1603_04467_amd import tfdense as T
from paper_1603_04467_amd.workloads import to_bf16_bits
from tests.parity import C_ACC, U32, assert_elementwise, product_bound, ulp  # noqa: F401
from tests.parity import TAU, amax, assert_bits, assert_close, to_f64

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _host(rng, shape, dt, zeros=0.1):
    """Seeded values exactly representable in `dt` (a share of them +0 and
    -0, the cases the test must send to 0) and the matching device tensor."""
    a = rng.standard_normal(shape).astype(np.float32)
    z = rng.random(shape)
    a[z < zeros / 2] = 0.0
    a[(z >= zeros / 2) & (z < zeros)] = -0.0
    if dt == "bf16":
        bits = to_bf16_bits(a)
        t = torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).to(DEV)
        return oracle.bf16_bits_to_f64(bits), t
    return a.astype(np.float64), torch.from_numpy(a).to(DEV)


def _words(mask: torch.Tensor) -> np.ndarray:
    return mask.cpu().numpy().view(np.uint32)


def _mask_buf(rows, cols):
    # every word starts with a pattern the kernels must overwrite
    return torch.full((rows, T.relu_mask_words(cols)), -0x5A5A5A5B, dtype=torch.int32, device=DEV)


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("rows,cols", [(1, 1), (3, 5), (7, 32), (9, 33), (100, 300), (257, 1029), (64, 4096),
                                       (2, 96), (0, 7)])
def test_relu_mask_bit_exact(dt, rows, cols):
    rng = np.random.default_rng([rows, cols, dt == "bf16"])
    f_h, f = _host(rng, (rows, cols), dt)
    m = _mask_buf(rows, cols)
    T.tfd_relu_mask(f, m)
    torch.cuda.synchronize()
    assert np.array_equal(_words(m), oracle.relu_mask(f_h))


@pytest.fixture
def waves_knob():
    """Sets the 16-bit whole-tile kernel's waves per workgroup for every
    layout (tuning knob) and restores the library's choice afterwards."""
    def set_(waves):
        if waves is not None:
            for lay in ("nn", "nt", "tn"):
                T.tfd_set_tuning(f"bf16_waves_{lay}", waves)
    yield set_
    for lay in ("nn", "nt", "tn"):
        T.tfd_set_tuning(f"bf16_waves_{lay}", 0)


@pytest.mark.parametrize("m,n,k,layout,dt,rounding,waves", [
    (512, 768, 512, "NT", "bf16", "nearest", None),     # whole 256 tiles: the mask epilogue
    (1024, 512, 768, "NN", "bf16", "nearest", None),
    (512, 256, 1024, "TN", "bf16", "nearest", None),
    (512, 512, 256, "NT", "bf16", "nearest", 4),
    (512, 512, 256, "NN", "bf16", "nearest", 16),
    (512, 512, 256, "TN", "bf16", "nearest", 8),
    (512, 768, 512, "NT", "bf16", "truncate", None),
    (300, 200, 136, "NT", "bf16", "nearest", None),     # ragged: MatMul, then the mask kernel
    (256, 1024, 784, "NN", "f32", "nearest", None),
    (100, 100, 784, "NN", "f32", "nearest", None),
    (256, 10, 1024, "NN", "f32", "nearest", None),
    (0, 64, 32, "NT", "bf16", "nearest", None),
])
def test_matmul_relu_mask(m, n, k, layout, dt, rounding, waves, waves_knob):
    waves_knob(waves)
    rng = np.random.default_rng([m, n, k, len(layout), dt == "bf16", rounding == "truncate"])
    ta, tb = layout == "TN", layout == "NT"
    a_h, a = _host(rng, (k, m) if ta else (m, k), dt)
    b_h, b = _host(rng, (n, k) if tb else (k, n), dt)
    bias_h = (rng.standard_normal(n) * 0.5).astype(np.float32)
    bias = torch.from_numpy(bias_h).to(DEV)
    tdt = torch.bfloat16 if dt == "bf16" else torch.float32
    c = torch.full((m, n), float("nan"), dtype=tdt, device=DEV)
    mask = _mask_buf(m, n)
    T.tfd_matmul_relu_mask(a, b, bias, c, mask, transpose_a=ta, transpose_b=tb, rounding=rounding)
    c2 = torch.full((m, n), float("nan"), dtype=tdt, device=DEV)
    T.tfd_matmul(a, b, c2, transpose_a=ta, transpose_b=tb, bias=bias, epilogue="bias_relu", rounding=rounding)
    torch.cuda.synchronize()
    assert torch.equal(c.view(torch.int16) if dt == "bf16" else c.view(torch.int32),
                       c2.view(torch.int16) if dt == "bf16" else c2.view(torch.int32)), "output differs from tfd_matmul"
    got = to_f64(c)
    assert np.array_equal(_words(mask), oracle.relu_mask(got)), "mask differs from the stored output's > 0"
    store = "bf16t" if rounding == "truncate" else dt
    want = oracle.matmul(a_h, b_h, ta, tb, out=store, bias=bias_h.astype(np.float64), relu=True)
    D = max(k, 1) * amax(a_h) * amax(b_h) + amax(bias_h)
    assert_close(got, want, D, TAU[dt], "Relu(AB + b)")


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("rows,cols", [(1, 1), (3, 5), (16, 4096), (1000, 300), (257, 1029), (64, 40), (0, 7)])
def test_relu_mask_grad_bias_add_grad(dt, rows, cols):
    rng = np.random.default_rng([rows, cols, dt == "bf16", 7])
    g_h, g = _host(rng, (rows, cols), dt, zeros=0.0)
    f_h, f = _host(rng, (rows, cols), dt)
    mask = _mask_buf(rows, cols)
    T.tfd_relu_mask(f, mask)
    bp = torch.empty_like(g)
    db = torch.full((cols,), float("nan"), device=DEV)
    T.tfd_relu_mask_grad_bias_add_grad(g, mask, bp, db)
    # the features-based call it stands for
    bp2 = torch.empty_like(g)
    db2 = torch.full((cols,), float("nan"), device=DEV)
    T.tfd_relu_grad_bias_add_grad(g, f, bp2, db2)
    # without a stored output
    db3 = torch.full((cols,), float("nan"), device=DEV)
    T.tfd_relu_mask_grad_bias_add_grad(g, mask, None, db3)
    torch.cuda.synchronize()
    dy = oracle.relu_grad_from_mask(g_h, oracle.relu_mask(f_h))
    assert_bits(to_f64(bp), dy, "ReluGrad from the mask")
    assert torch.equal(bp, bp2) and torch.equal(db, db2) and torch.equal(db, db3)
    D = max(rows, 1) * max(amax(dy), 1e-30)
    assert_close(to_f64(db), oracle.bias_add_grad(dy), D, TAU["f32"], "BiasAddGrad")


@pytest.mark.parametrize("m,n,k,layout,dt,rounding,waves", [
    (512, 768, 512, "NT", "bf16", "nearest", None),     # whole 256 tiles: the mask epilogue
    (1024, 512, 768, "NN", "bf16", "nearest", None),
    (512, 256, 1024, "TN", "bf16", "nearest", None),
    (512, 512, 256, "NT", "bf16", "nearest", 4),
    (512, 512, 256, "NT", "bf16", "nearest", 16),
    (512, 512, 256, "TN", "bf16", "nearest", 8),
    (512, 768, 512, "NT", "bf16", "truncate", None),
    (300, 200, 136, "NT", "bf16", "nearest", None),     # ragged: MatMul, then ReluGrad in place
    (256, 1024, 1024, "NT", "f32", "nearest", None),
    (1024, 512, 256, "NT", "f32", "nearest", None),
    (0, 64, 32, "NT", "bf16", "nearest", None),         # no rows: bias_grad = 0
])
def test_matmul_relu_mask_grad_bias_add_grad(m, n, k, layout, dt, rounding, waves, waves_knob):
    waves_knob(waves)
    rng = np.random.default_rng([m, n, k, len(layout), dt == "bf16", rounding == "truncate", 11])
    ta, tb = layout == "TN", layout == "NT"
    a_h, a = _host(rng, (k, m) if ta else (m, k), dt, zeros=0.0)
    b_h, b = _host(rng, (n, k) if tb else (k, n), dt, zeros=0.0)
    f_h, f = _host(rng, (m, n), dt)
    mask = _mask_buf(m, n)
    T.tfd_relu_mask(f, mask)
    tdt = torch.bfloat16 if dt == "bf16" else torch.float32
    bp = torch.full((m, n), float("nan"), dtype=tdt, device=DEV)
    db = torch.full((n,), float("nan"), device=DEV)
    T.tfd_matmul_relu_mask_grad_bias_add_grad(a, b, mask, bp, db, transpose_a=ta, transpose_b=tb, rounding=rounding)
    bp2 = torch.full((m, n), float("nan"), dtype=tdt, device=DEV)
    db2 = torch.full((n,), float("nan"), device=DEV)
    T.tfd_matmul_relu_grad_bias_add_grad(a, b, f, bp2, db2, transpose_a=ta, transpose_b=tb, rounding=rounding)
    torch.cuda.synchronize()
    assert torch.equal(bp, bp2), "backprops differ from the features-based call"
    assert torch.equal(db, db2), "bias_grad differs from the features-based call"
    # the plain MatMul on the same operands: the fused dY is the oracle's
    # ReluGrad of its output from the mask, bit for bit (an exact select)
    g = torch.full((m, n), float("nan"), dtype=tdt, device=DEV)
    T.tfd_matmul(a, b, g, transpose_a=ta, transpose_b=tb, rounding=rounding)
    torch.cuda.synchronize()
    dy = to_f64(bp)
    assert_bits(dy, oracle.relu_grad_from_mask(to_f64(g), oracle.relu_mask(f_h)), "fused dY = ReluGrad(plain output)")
    store = "bf16t" if rounding == "truncate" else dt
    want = oracle.relu_grad_from_mask(oracle.matmul(a_h, b_h, ta, tb, out=store), oracle.relu_mask(f_h))
    Dg = max(k, 1) * amax(a_h) * amax(b_h)
    assert_close(dy, want, Dg, TAU[dt], "fused dY")
    D = max(m, 1) * max(amax(dy), 1e-30)
    assert_close(to_f64(db), oracle.bias_add_grad(dy), D, TAU["f32"], "fused BiasAddGrad")
    if m > 0:
        keep = f_h > 0
        A, B = (a_h.T if ta else a_h), (b_h.T if tb else b_h)
        bound = product_bound(np.abs(A) @ np.abs(B), k, dy, store)
        assert_elementwise(np.where(keep, dy, 0.0), np.where(keep, oracle.matmul(A, B, out="f64"), 0.0), bound,
                           "fused dY per element")
        cbound = C_ACC * m * U32 * np.abs(dy).sum(axis=0) + 0.5 * ulp(to_f64(db), "f32")
        assert_elementwise(to_f64(db), oracle.bias_add_grad(dy, out="f64"), cbound, "fused db per column")


@pytest.mark.parametrize("rounding", ["nearest", "truncate"])
def test_mask_out_at_the_rounding_boundary(rounding):
    """Outputs around the smallest 16-bit magnitudes (2^-134 .. 2^-131, fp32
    denormals): which of them round to +0 depends on the rounding mode, and
    the mask written beside the output must be exactly "stored value > 0".
    C[r, c] = a_r b_c from one nonzero k per row; the products are exact in
    fp32. Whether the matrix cores keep fp32 denormals is not asserted: each
    stored value must be the oracle's rounding of the exact product, or +0."""
    m = n = 256
    k = 64
    r = np.arange(m)
    a_h = np.zeros((m, k))
    a_h[:, 0] = 2.0 ** -70 * (1 + (r % 128) / 128)           # exact in 16 bits
    c = np.arange(n)
    s = (1 + (c % 64) / 64) * np.where(c % 3 == 0, -1.0, 1.0) * 2.0 ** ((c // 64) % 3 - 1)
    b_h = np.zeros((n, k))                                   # B stored n x k (NT)
    b_h[:, 0] = 2.0 ** -64 * s
    a = torch.from_numpy(to_bf16_bits(a_h.astype(np.float32)).view(np.int16).copy()).view(torch.bfloat16).to(DEV)
    b = torch.from_numpy(to_bf16_bits(b_h.astype(np.float32)).view(np.int16).copy()).view(torch.bfloat16).to(DEV)
    assert np.array_equal(oracle.bf16_bits_to_f64(to_bf16_bits(a_h.astype(np.float32))), a_h)
    assert np.array_equal(oracle.bf16_bits_to_f64(to_bf16_bits(b_h.astype(np.float32))), b_h)
    bias = torch.zeros(n, device=DEV)
    out = torch.full((m, n), float("nan"), dtype=torch.bfloat16, device=DEV)
    mask = _mask_buf(m, n)
    T.tfd_matmul_relu_mask(a, b, bias, out, mask, transpose_b=True, rounding=rounding)
    torch.cuda.synchronize()
    got = to_f64(out)
    assert np.array_equal(_words(mask), oracle.relu_mask(got)), "mask differs from the stored output's > 0"
    exact = np.maximum(np.outer(a_h[:, 0], b_h[:, 0]), 0.0)
    want = oracle.round_to(exact, "bf16t" if rounding == "truncate" else "bf16")
    assert np.all((got == want) | (got == 0.0)), "stored value is neither the rounded product nor +0"
    # the case is not vacuous: products on both sides of the rounding boundary
    assert np.any(want > 0) and np.any((exact > 0) & (want == 0))
