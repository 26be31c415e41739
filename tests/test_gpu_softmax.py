"""Parity of the softmax cross-entropy cost head (tfd_softmax_cross_entropy_grad)
with the oracle's definition, element by element.

Error model of the kernel (fp32 arithmetic, row maximum m subtracted): each
exp(z - m) carries the rounding of z - m (at most |z - m| 2^-24 relative
after exp) and a few ulp of its own; the row sum adds at most
(cols / 64 + 6) ulp (a strided sum per lane, then a 64-lane butterfly); the
reciprocal and the product one ulp each. So |p_gpu - p| is bounded by
K 2^-24 p with K = cols / 64 + 2 max|z - m| + 16, and the subtraction of one
adds at most 2^-24. A 16-bit gradient adds its own rounding (2^-8 |G|
relative). Each row's loss term is log(s) + m - z_y with m and z_y exact in
float64, so it is off by at most the error of log(s): (K + 4 |log s| + 4)
2^-24 per row.
"""

import numpy as np
import pytest
import torch

import oracle
from paper_1603_04467_amd import tfdense as T
from paper_1603_04467_amd.workloads import to_bf16_bits
from tests.parity import to_f64

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _logits(rng, rows, cols, dt, scale):
    a = (rng.standard_normal((rows, cols)) * scale).astype(np.float32)
    if dt == "bf16":
        bits = to_bf16_bits(a)
        return oracle.bf16_bits_to_f64(bits), torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).to(DEV)
    return a.astype(np.float64), torch.from_numpy(a).to(DEV)


def _run(z, labels):
    g = torch.full_like(z, float("nan"))
    loss = torch.full((1,), float("nan"), dtype=torch.float64, device=DEV)
    T.tfd_softmax_cross_entropy_grad(z, labels, g, loss)
    torch.cuda.synchronize()
    return g, loss


def _bounds(z_h, dt):
    rows, cols = z_h.shape
    spread = float(np.max(z_h.max(axis=1) - z_h.min(axis=1))) if z_h.size else 0.0
    K = cols / 64 + 2 * spread + 16
    p = oracle.softmax(z_h)
    return K, p


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("rows,cols", [(1, 1), (3, 10), (256, 10), (100, 1000), (64, 4096), (7, 32768),
                                       (1029, 65)])
@pytest.mark.parametrize("scale", [1.0, 30.0])
def test_softmax_xent_matches_oracle(dt, rows, cols, scale):
    rng = np.random.default_rng([rows, cols, int(scale), dt == "bf16"])
    z_h, z = _logits(rng, rows, cols, dt, scale)
    y = rng.integers(0, cols, size=rows, dtype=np.int32)
    g, loss = _run(z, torch.from_numpy(y).to(DEV))
    g_want, l_want = oracle.softmax_cross_entropy_grad(z_h, y, grad_dtype="f64")
    K, p = _bounds(z_h, dt)
    allowed = K * 2.0 ** -24 * p + 2.0 ** -24
    if dt == "bf16":
        allowed = allowed + 2.0 ** -8 * np.abs(g_want)
    err = np.abs(to_f64(g) - g_want)
    assert np.all(np.isfinite(to_f64(g)))
    bad = err > allowed
    assert not np.any(bad), f"gradient: {int(bad.sum())} elements outside the bound, max|err| {err.max():.3e}"
    # rows of the gradient sum to zero up to the same rounding
    lse = np.log(np.sum(np.exp(z_h - z_h.max(axis=1, keepdims=True)), axis=1))
    allowed_loss = float(np.sum(K + 4 * np.abs(lse) + 4)) * 2.0 ** -24
    assert abs(loss.item() - l_want) <= allowed_loss, (loss.item(), l_want, allowed_loss)


def test_softmax_xent_one_class_and_uniform_rows_exact():
    # a single class: p = 1, G = 0, loss = 0 exactly
    z = torch.randn(5, 1, device=DEV)
    g, loss = _run(z, torch.zeros(5, dtype=torch.int32, device=DEV))
    assert torch.equal(g, torch.zeros_like(g)) and loss.item() == 0.0
    # equal logits over a power-of-two class count: p = 2^-e exactly
    z = torch.full((3, 256), 2.5, device=DEV)
    labels = torch.tensor([0, 100, 255], dtype=torch.int32, device=DEV)
    g, loss = _run(z, labels)
    want = torch.full_like(z, 1.0 / 256)
    want[torch.arange(3), labels.long()] -= 1.0
    assert torch.equal(g, want)
    assert abs(loss.item() - 3 * np.log(256.0)) <= 3 * 8 * 2.0 ** -23


def test_softmax_xent_empty_batch_writes_zero_loss():
    z = torch.empty(0, 10, device=DEV)
    g, loss = _run(z, torch.empty(0, dtype=torch.int32, device=DEV))
    assert loss.item() == 0.0


def test_softmax_xent_label_out_of_range_gives_nan_loss():
    rng = np.random.default_rng(7)
    z_h, z = _logits(rng, 4, 12, "f32", 1.0)
    y = np.array([3, 12, -1, 0], dtype=np.int32)
    g, loss = _run(z, torch.from_numpy(y).to(DEV))
    assert np.isnan(loss.item())
    p = oracle.softmax(z_h)
    gh = to_f64(g)
    K, _ = _bounds(z_h, "f32")
    # the two bad rows are p itself; the good rows are p - onehot
    for r in (1, 2):
        assert np.all(np.abs(gh[r] - p[r]) <= K * 2.0 ** -24 * p[r])
    g_want, _ = oracle.softmax_cross_entropy_grad(z_h[[0, 3]], y[[0, 3]], grad_dtype="f64")
    assert np.all(np.abs(gh[[0, 3]] - g_want) <= K * 2.0 ** -24 * p[[0, 3]] + 2.0 ** -24)


def test_softmax_xent_is_deterministic():
    rng = np.random.default_rng(11)
    _, z = _logits(rng, 4099, 1000, "f32", 3.0)
    y = torch.from_numpy(rng.integers(0, 1000, size=4099, dtype=np.int32)).to(DEV)
    g1, l1 = _run(z, y)
    g2, l2 = _run(z, y)
    assert torch.equal(g1, g2) and torch.equal(l1, l2)


def test_softmax_xent_rejects_bad_arguments():
    z = torch.zeros(4, 3, device=DEV)
    y = torch.zeros(4, dtype=torch.int32, device=DEV)
    loss = torch.zeros(1, dtype=torch.float64, device=DEV)
    with pytest.raises(T.TfdError):
        T.tfd_softmax_cross_entropy_grad(z, y, z, loss)          # grad aliases the logits
    with pytest.raises(T.TfdError):
        T.tfd_softmax_cross_entropy_grad(torch.zeros(4, 0, device=DEV), y, torch.zeros(4, 0, device=DEV), loss)
    with pytest.raises(T.TfdError):
        T.tfd_softmax_cross_entropy_grad(z, y, torch.empty_like(z), loss, workspace=torch.empty(0, dtype=torch.uint8,
                                                                                               device=DEV))
