"""Pins of the oracle's per-op definitions against what the mathematics fixes.

Each test checks an oracle function against something other than itself:
a brute-force loop with exact (rational or integer) sums, identity and
permutation matrices, closed forms, or the bit-level definition of the
16-bit format's round-to-nearest-even conversion.
"""

import math
from fractions import Fraction

import numpy as np
import pytest

import oracle


def _exact_matmul(A, B, ta, tb):
    """Triple loop with exact rational sums (independent of numpy's product)."""
    A = np.asarray(A)
    B = np.asarray(B)
    m, k = (A.shape[1], A.shape[0]) if ta else A.shape
    n = B.shape[0] if tb else B.shape[1]

    def a_(i, p):
        return Fraction(float(A[p, i] if ta else A[i, p]))

    def b_(p, j):
        return Fraction(float(B[j, p] if tb else B[p, j]))

    return [[sum((a_(i, p) * b_(p, j) for p in range(k)), Fraction(0)) for j in range(n)]
            for i in range(m)]


def _nearest_f32(q: Fraction) -> float:
    """fp32 nearest to a rational (ties to even), found by exact comparison
    of the three fp32 candidates around float32(float(q))."""
    c = np.float32(float(q))
    cands = [np.nextafter(c, np.float32(-np.inf)), c, np.nextafter(c, np.float32(np.inf))]
    best = None
    for v in cands:
        d = abs(Fraction(float(v)) - q)
        key = (d, int(np.array(v, np.float32).view(np.uint32)) & 1)  # ties -> even mantissa
        if best is None or key < best[0]:
            best = (key, v)
    return float(best[1])


@pytest.mark.parametrize("ta,tb", [(False, False), (False, True), (True, False), (True, True)])
@pytest.mark.parametrize("m,n,k", [(3, 4, 5), (1, 1, 1), (2, 7, 3), (4, 3, 0)])
def test_matmul_brute_force(ta, tb, m, n, k):
    rng = np.random.default_rng(11)
    a = rng.standard_normal((k, m) if ta else (m, k)).astype(np.float32)
    b = rng.standard_normal((n, k) if tb else (k, n)).astype(np.float32)
    got = oracle.matmul(a, b, ta, tb, out="f64")
    exact = _exact_matmul(a, b, ta, tb)
    absprod = _exact_matmul(np.abs(a), np.abs(b), ta, tb)
    assert got.shape == (m, n)
    for i in range(m):
        for j in range(n):
            # float64 summation error bound: k * 2**-53 * sum |a||b|
            assert abs(Fraction(float(got[i, j])) - exact[i][j]) <= (k + 1) * Fraction(1, 2 ** 53) * absprod[i][j]
    # rounding once to fp32 gives the nearest fp32 of the exact sum
    got32 = oracle.matmul(a, b, ta, tb, out="f32")
    for i in range(m):
        for j in range(n):
            assert got32[i, j] == _nearest_f32(exact[i][j])


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_matmul_identity_and_permutation(dt):
    rng = np.random.default_rng(3)
    x = oracle.round_to(rng.standard_normal((6, 5)), dt)
    eye5 = np.eye(5)
    eye6 = np.eye(6)
    perm = rng.permutation(5)
    P = eye5[:, perm]  # x @ P == x[:, perm]
    assert np.array_equal(oracle.matmul(x, eye5, out=dt), x)
    assert np.array_equal(oracle.matmul(eye6, x, out=dt), x)
    assert np.array_equal(oracle.matmul(x, P, out=dt), x[:, perm])
    # NT: x @ P.T.T ; TN: x.T.T @ P
    assert np.array_equal(oracle.matmul(x, P.T, transpose_b=True, out=dt), x[:, perm])
    assert np.array_equal(oracle.matmul(x.T, P, transpose_a=True, out=dt), x[:, perm])
    # transposed identity products give the transpose
    assert np.array_equal(oracle.matmul(x, eye6, transpose_a=True, out=dt), x.T)
    assert np.array_equal(oracle.matmul(eye5, x, transpose_b=True, out=dt), x.T)


@pytest.mark.parametrize("ta,tb", [(False, False), (False, True), (True, False)])
def test_matmul_small_integers_exact(ta, tb):
    rng = np.random.default_rng(5)
    m, n, k = 9, 11, 13
    a = rng.integers(-4, 5, size=(k, m) if ta else (m, k)).astype(np.float64)
    b = rng.integers(-4, 5, size=(n, k) if tb else (k, n)).astype(np.float64)
    ia = a.T if ta else a
    ib = b.T if tb else b
    want = [[sum(int(ia[i, p]) * int(ib[p, j]) for p in range(k)) for j in range(n)] for i in range(m)]
    for dt in ("f32", "bf16"):
        assert np.array_equal(oracle.matmul(a, b, ta, tb, out=dt), np.array(want, dtype=np.float64))


def test_matmul_bias_relu_closed_form():
    a = np.array([[1.0, 2.0], [3.0, -4.0]])
    w = np.array([[0.5, -1.0, 0.0], [0.25, 1.0, 2.0]])
    b = np.array([0.5, -3.0, 1.0])
    # z = a @ w: [[1.0, 1.0, 4.0], [0.5, -7.0, -8.0]]; + b; relu
    y = oracle.matmul(a, w, out="f32", bias=b, relu=False)
    assert np.array_equal(y, [[1.5, -2.0, 5.0], [1.0, -10.0, -7.0]])
    h = oracle.matmul(a, w, out="f32", bias=b, relu=True)
    assert np.array_equal(h, [[1.5, 0.0, 5.0], [1.0, 0.0, 0.0]])
    assert not np.any(np.signbit(h))
    # k = 0: the product is empty, the output is Relu(bias)
    h0 = oracle.matmul(np.zeros((2, 0)), np.zeros((0, 3)), out="f32", bias=b, relu=True)
    assert np.array_equal(h0, [[0.5, 0.0, 1.0]] * 2)
    # zero bias leaves the product unchanged
    assert np.array_equal(oracle.matmul(a, w, out="f32", bias=np.zeros(3)), oracle.matmul(a, w, out="f32"))
    assert np.array_equal(oracle.bias_add(oracle.matmul(a, w, out="f64"), b, out="f32"), y)


def test_relu_values_idempotence_sign():
    x = np.array([-2.5, -0.0, 0.0, 1e-40, 3.0, -1e-40, np.float32(1e-45)])
    r = oracle.relu(x)
    assert np.array_equal(r, [0.0, 0.0, 0.0, 1e-40, 3.0, 0.0, float(np.float32(1e-45))])
    assert not np.any(np.signbit(r))
    rng = np.random.default_rng(0)
    y = rng.standard_normal(1000)
    r = oracle.relu(y)
    assert np.array_equal(oracle.relu(r), r)
    assert np.all(r >= 0) and not np.any(np.signbit(r))
    assert np.array_equal(r[y > 0], y[y > 0])


def test_relu_grad_mask_is_strict():
    f = np.array([1.0, 0.0, -0.0, -1.0, 2e-30])
    g = np.array([5.0, 6.0, 7.0, 8.0, -9.0])
    assert np.array_equal(oracle.relu_grad(g, f), [5.0, 0.0, 0.0, 0.0, -9.0])
    assert not np.any(np.signbit(oracle.relu_grad(-g, f)[1:4]))


def test_relu_mask_worked_example():
    # row 0: positives in columns 0, 5, 31 (word 0) and 32, 39 (word 1);
    # row 1: only non-positive values, NaN and a subnormal positive in column 33
    f = np.zeros((2, 40))
    f[0, [0, 5, 31, 32, 39]] = [1.0, 2.0, 1e-30, 3.0, 7.0]
    f[0, [1, 2, 33]] = [-1.0, -0.0, -5.0]
    f[1, :] = -1.0
    f[1, [3, 4, 5, 33]] = [0.0, -0.0, np.nan, 1e-40]
    want = np.array([[0x80000021, 0x00000081], [0x00000000, 0x00000002]], dtype=np.uint32)
    got = oracle.relu_mask(f)
    assert got.dtype == np.uint32 and got.shape == (2, 2)
    assert np.array_equal(got, want)


@pytest.mark.parametrize("cols", [1, 31, 32, 33, 100, 257])
def test_relu_mask_unpacks_to_the_test_and_pads_with_zeros(cols):
    rng = np.random.default_rng(cols)
    f = rng.standard_normal((7, cols))
    f[rng.random((7, cols)) < 0.1] = 0.0
    w = oracle.relu_mask(f)
    assert w.shape == (7, (cols + 31) // 32)
    # little-endian bytes of each word, then bits least significant first
    bits = np.unpackbits(w.astype("<u4").view(np.uint8), axis=1, bitorder="little")
    assert np.array_equal(bits[:, :cols].astype(bool), f > 0)
    assert not bits[:, cols:].any()
    assert np.array_equal(bits.sum(axis=1), (f > 0).sum(axis=1))


def test_relu_grad_from_mask_equals_relu_grad():
    rng = np.random.default_rng(3)
    for cols in (5, 32, 70):
        g = rng.standard_normal((9, cols))
        h = oracle.relu(rng.standard_normal((9, cols)))
        h[0, :3] = [0.0, -0.0, 1e-45]
        got = oracle.relu_grad_from_mask(g, oracle.relu_mask(h))
        want = oracle.relu_grad(g, h)
        assert np.array_equal(got, want)
        assert not np.any(np.signbit(got[want == 0]))


def test_bias_add_grad_exact_sums():
    rng = np.random.default_rng(1)
    g = rng.integers(-100, 101, size=(37, 9)).astype(np.float64)
    want = [sum(int(g[n, m]) for n in range(37)) for m in range(9)]
    assert np.array_equal(oracle.bias_add_grad(g), want)
    c = np.tile(np.array([0.25, -3.0, 7.5]), (1000, 1))
    assert np.array_equal(oracle.bias_add_grad(c), [250.0, -3000.0, 7500.0])
    # rounded once: an exact rational sum rounded to fp32
    x = rng.standard_normal((50, 4)).astype(np.float32).astype(np.float64)
    got = oracle.bias_add_grad(x)
    for m in range(4):
        q = sum((Fraction(float(v)) for v in x[:, m]), Fraction(0))
        assert got[m] == _nearest_f32(q)
    assert oracle.bias_add_grad(np.zeros((0, 3))).tolist() == [0.0, 0.0, 0.0]


def test_l2_loss_grad_difference_and_fd():
    rng = np.random.default_rng(2)
    h = rng.standard_normal((4, 3)).astype(np.float32).astype(np.float64)
    t = rng.standard_normal((4, 3)).astype(np.float32).astype(np.float64)
    g, loss = oracle.l2_loss_grad(h, t, grad_dtype="f32")
    for idx in np.ndindex(h.shape):
        q = Fraction(float(h[idx])) - Fraction(float(t[idx]))
        assert g[idx] == _nearest_f32(q)
    assert loss == pytest.approx(0.5 * math.fsum(float((a - b) ** 2) for a, b in zip(h.ravel(), t.ravel())), rel=1e-15)
    # central finite differences of the loss reproduce the gradient
    eps = 1e-4
    for idx in [(0, 0), (3, 2), (1, 1)]:
        hp, hm = h.copy(), h.copy()
        hp[idx] += eps
        hm[idx] -= eps
        fd = (oracle.l2_loss_grad(hp, t, "f64")[1] - oracle.l2_loss_grad(hm, t, "f64")[1]) / (2 * eps)
        assert fd == pytest.approx(h[idx] - t[idx], rel=1e-8, abs=1e-10)
    # no target: L = 1/2 sum h^2, G = h
    g0, l0 = oracle.l2_loss_grad(h, None, grad_dtype="f32")
    assert np.array_equal(g0, h)
    assert l0 == pytest.approx(0.5 * float(np.sum(h * h)), rel=1e-15)


def _sgd_exact(var, alpha, delta):
    return _nearest_f32(Fraction(float(var)) - Fraction(float(np.float32(alpha))) * Fraction(float(delta)))


def test_apply_gradient_descent_rounds_exact_value_once():
    rng = np.random.default_rng(4)
    alpha = np.float32(0.01)
    var = rng.standard_normal(4000).astype(np.float32)
    delta = (rng.standard_normal(4000) * 10.0 ** rng.integers(-6, 4, 4000)).astype(np.float32)
    got = oracle.apply_gradient_descent(var, alpha, delta)
    for i in range(4000):
        assert got[i] == _sgd_exact(var[i], alpha, delta[i]), i

    # hard cases: alpha*delta = 2**-24 * (1 + t) with 0 < |t| < 2**-29, i.e.
    # half an fp32 ulp of var in [1, 2) plus a remainder below float64's
    # resolution there, so that a float64 sum lands exactly on an fp32 midpoint
    hard_a, hard_d, hard_v = [], [], []
    while len(hard_a) < 400:
        x = np.float32(rng.uniform(1.0, 2.0))
        y = np.float32(1.0 / float(x))
        t = float(x) * float(y) - 1.0          # exact in float64
        if t == 0.0 or abs(t) >= 2.0 ** -29:
            continue
        j = int(rng.integers(1, 12))
        sgn = 1.0 if rng.random() < 0.5 else -1.0
        a = np.float32(float(x) * 2.0 ** -j)
        d = np.float32(sgn * float(y) * 2.0 ** (j - 24))
        v = np.float32(1.0 + 2.0 ** -22 * int(rng.integers(0, 1 << 22)))  # even mantissa
        hard_a.append(a), hard_d.append(d), hard_v.append(v)
    naive_diff = 0
    for a, d, v in zip(hard_a, hard_d, hard_v):
        want = _sgd_exact(v, a, d)
        got = float(oracle.apply_gradient_descent(np.array([v]), a, np.array([d]))[0])
        assert got == want
        naive = float(np.float32(float(v) - float(a) * float(d)))
        naive_diff += naive != want
    # the sample must contain cases where rounding twice (float64, then fp32) is wrong
    assert naive_diff > 0


def test_apply_gradient_descent_lr_zero_and_zero_delta():
    rng = np.random.default_rng(6)
    var = rng.standard_normal(1000).astype(np.float32)
    delta = rng.standard_normal(1000).astype(np.float32)
    assert np.array_equal(oracle.apply_gradient_descent(var, 0.0, delta), var.astype(np.float64))
    assert np.array_equal(oracle.apply_gradient_descent(var, 0.01, np.zeros(1000, np.float32)), var.astype(np.float64))
    # fp32(0.01) is 0x3C23D70A
    assert np.array(np.float32(0.01)).view(np.uint32) == 0x3C23D70A


def _bf16_bits_formula(u32):
    """Round-to-nearest-even fp32 -> 16-bit by integer arithmetic on the bits."""
    u = u32.astype(np.uint64)
    r = (u + np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)
    return r.astype(np.uint16)


def test_round_bf16_matches_bit_formula_over_fp32_patterns():
    hi = np.arange(1 << 16, dtype=np.uint32) << np.uint32(16)
    lows = [0, 1, 0x7FFE, 0x7FFF, 0x8000, 0x8001, 0xFFFE, 0xFFFF, 0x4000, 0xC000]
    rng = np.random.default_rng(7)
    lows += list(rng.integers(0, 1 << 16, 10))
    u = (hi[:, None] | np.array(lows, dtype=np.uint32)[None, :]).ravel()
    f = u.view(np.float32)
    keep = ~np.isnan(f)
    u, f = u[keep], f[keep]
    got = oracle.round_bf16(f.astype(np.float64))
    want = oracle.bf16_bits_to_f64(_bf16_bits_formula(u))
    both_inf = np.isinf(got) & np.isinf(want) & (np.sign(got) == np.sign(want))
    assert np.all((got == want) | both_inf)
    assert np.array_equal(np.signbit(got), np.signbit(want))


def test_round_bf16_rounds_float64_once():
    # a value just above a 16-bit midpoint, closer than fp32 can resolve:
    # rounding to fp32 first would land on the midpoint and round to even (down)
    mid = 1.0 + 2.0 ** -8           # halfway between 1.0 (0x3F80) and 1 + 2**-7 (0x3F81)
    x = mid + 2.0 ** -40
    assert oracle.round_bf16(np.array([x]))[0] == 1.0 + 2.0 ** -7
    assert float(np.float32(x)) == mid                                  # fp32 cannot see the excess
    assert oracle.round_bf16(np.array([mid]))[0] == 1.0                 # tie -> even (0x3F80)
    assert oracle.round_bf16(np.array([1.0 + 3 * 2.0 ** -8]))[0] == 1.0 + 2.0 ** -6  # tie -> even (0x3F82)
    assert oracle.round_bf16(np.array([-0.0]))[0] == 0.0 and np.signbit(oracle.round_bf16(np.array([-0.0]))[0])
    # subnormal quantum and overflow
    assert oracle.round_bf16(np.array([3 * 2.0 ** -134]))[0] == 2 * 2.0 ** -133
    assert np.isinf(oracle.round_bf16(np.array([(2 - 2 ** -8) * 2.0 ** 127]))[0])  # midpoint above the largest value -> even (inf)
    assert oracle.round_bf16(np.array([3.3894e38]))[0] == (2 - 2 ** -7) * 2.0 ** 127
    bits = oracle.f64_to_bf16_bits(np.array([1.0, -2.0, 1.0 + 2.0 ** -7]))
    assert bits.tolist() == [0x3F80, 0xC000, 0x3F81]
