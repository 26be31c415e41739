"""Pins of the softmax cross-entropy cost head (SoftMax and Log of Table 1)."""

import math

import numpy as np
import pytest

import oracle


def test_softmax_rows_are_distributions_and_shift_invariant():
    rng = np.random.default_rng(0)
    z = rng.standard_normal((50, 10)) * 3
    p = oracle.softmax(z)
    assert np.all(p > 0)
    assert np.allclose(p.sum(axis=1), 1.0, rtol=0, atol=1e-15)
    assert np.allclose(oracle.softmax(z + 123.25), p, rtol=1e-13, atol=0)
    # order is preserved
    assert np.array_equal(np.argsort(z, axis=1), np.argsort(p, axis=1))


def test_softmax_two_classes_is_the_logistic_function():
    z = np.array([[0.3, -1.2], [5.0, 5.0], [-20.0, 20.0]])
    p = oracle.softmax(z)
    for row, (a, b) in zip(p, z):
        assert row[0] == pytest.approx(1.0 / (1.0 + math.exp(b - a)), rel=1e-14)


def test_cross_entropy_gradient_is_p_minus_onehot():
    rng = np.random.default_rng(1)
    z = rng.standard_normal((40, 7))
    y = rng.integers(0, 7, 40)
    g, loss = oracle.softmax_cross_entropy_grad(z, y, grad_dtype="f64")
    p = oracle.softmax(z)
    onehot = np.zeros_like(p)
    onehot[np.arange(40), y] = 1.0
    assert np.allclose(g, p - onehot, rtol=0, atol=1e-15)
    assert np.allclose(g.sum(axis=1), 0.0, atol=1e-14)
    want = -sum(math.log(p[n, y[n]]) for n in range(40))
    assert loss == pytest.approx(want, rel=1e-13)


def test_cross_entropy_finite_differences():
    rng = np.random.default_rng(2)
    z = rng.standard_normal((5, 6))
    y = rng.integers(0, 6, 5)
    g, _ = oracle.softmax_cross_entropy_grad(z, y, grad_dtype="f64")
    eps = 1e-6
    for idx in np.ndindex(z.shape):
        zp, zm = z.copy(), z.copy()
        zp[idx] += eps
        zm[idx] -= eps
        fd = (oracle.softmax_cross_entropy_grad(zp, y, "f64")[1] - oracle.softmax_cross_entropy_grad(zm, y, "f64")[1]) / (2 * eps)
        assert g[idx] == pytest.approx(fd, rel=1e-6, abs=1e-9)


def test_cross_entropy_uniform_logits_and_large_values():
    n, c = 8, 10
    g, loss = oracle.softmax_cross_entropy_grad(np.zeros((n, c)), np.arange(n) % c, grad_dtype="f64")
    assert loss == pytest.approx(n * math.log(c), rel=1e-15)
    assert np.allclose(g[np.arange(n), np.arange(n) % c], 1.0 / c - 1.0)
    # no overflow for large logits: the result depends only on differences
    z = np.array([[1000.0, 1001.0, 999.0]])
    g1, l1 = oracle.softmax_cross_entropy_grad(z, np.array([1]), "f64")
    g0, l0 = oracle.softmax_cross_entropy_grad(z - 1000.0, np.array([1]), "f64")
    assert np.all(np.isfinite(g1)) and l1 == pytest.approx(l0, rel=1e-14)
    assert np.allclose(g1, g0, atol=1e-15)


def test_cross_entropy_batch_sum_is_additive():
    rng = np.random.default_rng(3)
    z = rng.standard_normal((30, 10))
    y = rng.integers(0, 10, 30)
    _, full = oracle.softmax_cross_entropy_grad(z, y, "f64")
    parts = sum(oracle.softmax_cross_entropy_grad(z[s:s + 10], y[s:s + 10], "f64")[1] for s in range(0, 30, 10))
    assert parts == pytest.approx(full, rel=1e-14)


def test_classifier_step_matches_finite_differences():
    """3-layer MLP with the classifier cost: backward chain vs finite
    differences of the loss (float64)."""
    rng = np.random.default_rng(4)
    dims = (5, 7, 6, 4)
    while True:
        x = rng.standard_normal((3, 5))
        ws = [rng.standard_normal((dims[l], dims[l + 1])) / np.sqrt(dims[l]) for l in range(3)]
        bs = [rng.standard_normal(dims[l + 1]) * 0.3 for l in range(3)]
        h, ok = x, True
        for w_, b_ in zip(ws, bs):
            y_ = h @ w_ + b_
            ok &= bool(np.min(np.abs(y_)) > 1e-3)
            h = np.maximum(y_, 0.0)
        if ok:
            break
    labels = rng.integers(0, 4, 3)
    relus = [True, True, False]
    out = oracle.dense_step(x, ws, bs, relus, act="f64", labels=labels, update=False)

    def loss(ws_):
        h_ = x
        for w_, b_, r in zip(ws_, bs, relus):
            h_ = oracle.matmul(h_, w_, out="f64", bias=b_, relu=r)
        return oracle.softmax_cross_entropy_grad(h_, labels, "f64")[1]

    eps = 1e-6
    for l in range(3):
        for idx in [(0, 0), (ws[l].shape[0] - 1, ws[l].shape[1] - 1), (1, 2)]:
            wp = [w_.copy() for w_ in ws]
            wm = [w_.copy() for w_ in ws]
            wp[l][idx] += eps
            wm[l][idx] -= eps
            fd = (loss(wp) - loss(wm)) / (2 * eps)
            assert out["dw"][l][idx] == pytest.approx(fd, rel=1e-6, abs=1e-9)
