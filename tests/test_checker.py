"""The per-element product bound of tests/parity.py rejects wrong results.

The GPU parity tests bound each output element of a MatMul by
C_ACC * (K + 1) * u * (|A| @ |B| + |bias|) + (half an ulp of the stored value),
computed from the operands the kernel read. These CPU tests feed the checker
the oracle's result (section 2, Table 1 MatMul, BiasAdd, Relu; section 4.1
gradients) on rows with the statistics of the 4096-wide 16-bit step (X ~ N(0, 1),
W ~ N(0, 1/64), K = 4096; dW with K = 1024 batch rows), perturbed on the host
as a faulty kernel would perturb it, and check that every fault is rejected
while a correct result reached by another fp32 summation order passes.
The normalised rule max|err| / (K max|A| max|B|) <= 1e-2 of 16-bit operands
accepts some of these faults at K = 4096; that is why the per-element bound
exists.
"""

import numpy as np
import pytest

import oracle
from tests.parity import TAU, assert_elementwise, check_relu_decisions, norm_err, product_bound, ulp


def _bf16(rng, shape, std):
    return oracle.round_to(rng.standard_normal(shape) * std, "bf16")


@pytest.fixture(scope="module")
def layer():
    """64 rows of a 4096 -> 4096 layer with 16-bit operands and a nonzero bias."""
    rng = np.random.default_rng(7)
    x = _bf16(rng, (64, 4096), 1.0)
    w = _bf16(rng, (4096, 4096), 1.0 / 64)
    b = oracle.round_to(rng.standard_normal(4096) * 0.5, "f32")
    z = oracle.matmul(x, w, out="f64")
    y = z + b[None, :]
    absprod = np.abs(x) @ np.abs(w)
    return {"x": x, "w": w, "b": b, "z": z, "y": y, "abs": absprod, "K": 4096}


def _fp32_other_order(a, b):
    """A correct fp32-accumulated product in another summation order (BLAS
    float32 blocks): products of 16-bit values are exact in fp32."""
    return (a.astype(np.float32) @ b.astype(np.float32)).astype(np.float64)


def _store(v):
    return oracle.round_to(v, "bf16")


def _check(L, got, relu=True):
    bound = product_bound(L["abs"], L["K"], got, "bf16", abs_bias=np.abs(L["b"]))
    want = oracle.relu(L["y"]) if relu else L["y"]
    assert_elementwise(got, want, bound, "forward")
    if relu:
        check_relu_decisions(got, L["y"], bound, "forward")


def test_correct_results_pass(layer):
    L = layer
    _check(L, _store(oracle.relu(L["y"])))
    z32 = _fp32_other_order(L["x"], L["w"])
    y32 = (z32.astype(np.float32) + L["b"].astype(np.float32)).astype(np.float64)
    _check(L, _store(oracle.relu(y32)))
    # truncating store: a whole ulp
    got = oracle.round_to(oracle.relu(y32), "bf16t")
    bound = product_bound(L["abs"], L["K"], got, "bf16t", abs_bias=np.abs(L["b"]))
    assert_elementwise(got, oracle.relu(L["y"]), bound, "truncating forward")


@pytest.mark.parametrize("fault", ["zero", "dropped_k_tile", "repeated_k_tile", "relu_before_bias", "no_bias",
                                   "swapped_rows", "last_k_tile_only"])
def test_faults_are_rejected(layer, fault):
    L = layer
    x, w, b = L["x"], L["w"], L["b"]
    kt = slice(1024, 1088)
    if fault == "zero":
        got = np.zeros_like(L["y"])
    elif fault == "dropped_k_tile":
        got = _store(oracle.relu(L["y"] - x[:, kt] @ w[kt]))
    elif fault == "repeated_k_tile":
        got = _store(oracle.relu(L["y"] + x[:, kt] @ w[kt]))
    elif fault == "relu_before_bias":
        got = _store(oracle.relu(L["z"]) + b[None, :])
    elif fault == "no_bias":
        got = _store(oracle.relu(L["z"]))
    elif fault == "swapped_rows":
        got = _store(oracle.relu(L["y"]))[[1, 0] + list(range(2, 64))]
    elif fault == "last_k_tile_only":
        got = _store(oracle.relu(x[:, -64:] @ w[-64:] + b[None, :]))
    with pytest.raises(AssertionError):
        _check(L, got)


def test_normalised_rule_alone_misses_faults(layer):
    """Why the per-element bound is needed: at K = 4096 the normalised rule
    with the 16-bit tolerance accepts a zero output and a dropped k-tile."""
    L = layer
    D = L["K"] * np.max(np.abs(L["x"])) * np.max(np.abs(L["w"])) + np.max(np.abs(L["b"]))
    want = _store(oracle.relu(L["y"]))
    assert norm_err(np.zeros_like(want), want, D) <= TAU["bf16"]
    dropped = _store(oracle.relu(L["y"] - L["x"][:, 1024:1088] @ L["w"][1024:1088]))
    assert norm_err(dropped, want, D) <= TAU["bf16"]


def test_relu_decisions_reject_a_shifted_mask(layer):
    L = layer
    h = _store(oracle.relu(L["y"]))
    bound = product_bound(L["abs"], L["K"], h, "bf16", abs_bias=np.abs(L["b"]))
    shifted = np.roll(h, 1, axis=1)
    with pytest.raises(AssertionError):
        check_relu_decisions(shifted, L["y"], bound, "shifted mask")
    # flips inside the band only, but more than the cap: rejected
    y = L["y"]
    inband = np.abs(y) <= bound
    flipped = np.where(inband, np.where(h > 0, 0.0, np.abs(y) + 1.0), h)
    assert np.count_nonzero(inband) > 1e-3 * y.size
    with pytest.raises(AssertionError):
        check_relu_decisions(flipped, y, bound, "many in-band flips")


def test_gradient_products(layer):
    """Input gradient dX = dY W^T (K = 4096) and weight gradient
    dW = X^T dY (K = batch = 1024, fp32 output): correct results in another
    summation order pass, a dropped k-tile or a zero output does not."""
    rng = np.random.default_rng(8)
    w = layer["w"]
    h = _bf16(rng, (64, 4096), 1.0)
    dy = oracle.relu_grad(_bf16(rng, (64, 4096), 0.5), h)
    dx = oracle.matmul(dy, w, transpose_b=True, out="f64")
    absdx = np.abs(dy) @ np.abs(w).T
    got = _store(_fp32_other_order(dy, w.T))
    assert_elementwise(got, dx, product_bound(absdx, 4096, got, "bf16"), "dX")
    bad = _store(dx - dy[:, 64:128] @ w.T[64:128])
    with pytest.raises(AssertionError):
        assert_elementwise(bad, dx, product_bound(absdx, 4096, bad, "bf16"), "dX")
    # weight gradient over 1024 batch rows
    x = _bf16(rng, (1024, 512), 1.0)
    g = _bf16(rng, (1024, 256), 0.5)
    dw = oracle.matmul(x, g, transpose_a=True, out="f64")
    absdw = np.abs(x).T @ np.abs(g)
    got = oracle.round_to(_fp32_other_order(x.T, g), "f32")
    assert_elementwise(got, dw, product_bound(absdw, 1024, got, "f32"), "dW")
    for bad in (np.zeros_like(dw), oracle.round_to(dw - x[512:576].T @ g[512:576], "f32")):
        with pytest.raises(AssertionError):
            assert_elementwise(bad, dw, product_bound(absdw, 1024, bad, "f32"), "dW")


def test_ulp():
    assert ulp(np.array([1.0]), "bf16")[0] == 2.0 ** -7
    assert ulp(np.array([1.0]), "f32")[0] == 2.0 ** -23
    assert ulp(np.array([255.0]), "bf16")[0] == 1.0
    assert ulp(np.array([0.0]), "bf16")[0] == 2.0 ** -133
    assert ulp(np.array([-3.0]), "bf16")[0] == 2.0 ** -6


class _FakeStep:
    """The tensors of one step as a DenseStep holds them, filled from the
    oracle's chain (CPU tensors), for exercising the teacher-forced checks."""

    def __init__(self, w, inp, fuse):
        import torch

        import oracle as O
        from paper_1603_04467_amd.step import fused_below

        self.w, self.fuse, self.masks = w, fuse, [None] * w.layers
        conv = O.bf16_bits_to_f64 if w.act == "bf16" else (lambda a: a.astype(np.float64))
        x = conv(inp["x"])
        W = [conv(a) for a in inp["weights"]]
        b = [a.astype(np.float64) for a in inp["biases"]]
        masters = None if inp["masters"] is None else [a.astype(np.float64) for a in inp["masters"]]
        t = None if inp["target"] is None else conv(inp["target"])
        ref = O.dense_step(x, W, b, list(w.relus), act=w.act, target=t, lr=w.lr, masters=masters)
        tdt = torch.bfloat16 if w.act == "bf16" else torch.float32
        T = lambda a, dt=tdt: torch.from_numpy(np.asarray(a, np.float64)).to(dt)  # noqa: E731
        self.h = [T(a) for a in ref["h"]]
        self.g = T(ref["g"])
        self.target = None if t is None else T(t)
        self.loss = torch.tensor([ref["loss"]], dtype=torch.float64)
        self._dy = [T(a) for a in ref["dy"]]
        self.dy = [self._dy[l] if w.relus[l] else None for l in range(w.layers)]
        self.dx = [T(a) for a in ref["dx"]]
        for l in range(w.layers):
            if fused_below(w, l, fuse):
                self.dx[l] = None
        self.dw = [T(a, torch.float32) for a in ref["dw"]]
        self.db = [T(a, torch.float32) for a in ref["db"]]
        self.weights = [T(a) for a in ref["new_weights"]]
        self.biases = [T(a, torch.float32) for a in ref["new_biases"]]
        self.masters = None if masters is None else [T(a, torch.float32) for a in ref["new_masters"]]
        self.weights_t = None if masters is None else [t_.t() for t_ in self.weights]
        self._saved = [T(a) for a in W] + [T(a, torch.float32) for a in b] + \
            ([] if masters is None else [T(a, torch.float32) for a in masters])

    def dy_of(self, l):
        return self._dy[l]


@pytest.mark.parametrize("name,fuse", [("wide4096x4-bf16", True), ("wide4096x4-bf16", False),
                                       ("wide4096x4-f32", True), ("mlp784-1024-1024-10", False)])
def test_teacher_forced_checks_accept_the_oracle_and_reject_faults(name, fuse):
    from paper_1603_04467_amd import workloads
    from tests.teacher import check_step, sample_cols, sample_rows

    w = workloads.workload(name)
    if w.batch > 256:
        w = w.scaled(batch=96, dims=(64, 128, 96, 64, 32))
    s = _FakeStep(w, workloads.generate(w, seed=4), fuse)
    check_step(s)
    check_step(s, rows=sample_rows(w.batch, tile=32, tiles=2, extra=8), cols=lambda M: sample_cols(M, 16, 2, 4))
    # planted faults, one at a time
    for fault in ("h1_zero_row", "dw_dropped_rows", "db_scaled", "master_twice", "dx_or_dy_scaled"):
        f = _FakeStep(w, workloads.generate(w, seed=4), fuse)
        if fault == "h1_zero_row":
            f.h[1][3] = 0
        elif fault == "dw_dropped_rows":
            f.dw[0] = f.dw[0] * 0.97
        elif fault == "db_scaled":
            f.db[-1] = f.db[-1] * 1.01
        elif fault == "master_twice":
            if f.masters is None:
                f.weights[0] = f.weights[0] - 0.01 * f.dw[0]
            else:
                f.masters[0] = f.masters[0] - 0.01 * f.dw[0]
        else:
            lo = 0 if fuse else 1
            t = f._dy[lo] if fuse and w.relus[0] else f.dx[1]
            t.mul_(1.05)
        with pytest.raises(AssertionError):
            check_step(f)
