"""Parity rules shared by the GPU tests.

The normalised error of an output is ``max|got - want| / D`` with ``D`` the
scale the output's reduction can reach: for a product of length K,
``K * max|A| * max|B|`` (+ ``max|bias|``). It must stay within
``TAU["f32"] = 1e-5`` for fp32 operands and ``TAU["bf16"] = 1e-2`` for 16-bit
operands with fp32 accumulation. Integer-valued, select-only and rounding-only
results (Relu, ReluGrad, the SGD update, the 16-bit cast, the Relu masks
outside the rounding band of zero) must match bit for bit.
"""

import numpy as np
import torch

TAU = {"f32": 1e-5, "bf16": 1e-2}


def to_f64(t: torch.Tensor) -> np.ndarray:
    """Exact float64 values of a device tensor (fp32 or bf16)."""
    return t.detach().to("cpu", torch.float32).numpy().astype(np.float64)


def amax(a) -> float:
    a = np.asarray(a)
    return float(np.max(np.abs(a))) if a.size else 0.0


def norm_err(got, want, D: float) -> float:
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    assert got.shape == want.shape, (got.shape, want.shape)
    assert np.all(np.isfinite(got)), "non-finite output"
    if got.size == 0:
        return 0.0
    e = float(np.max(np.abs(got - want)))
    if D == 0.0:
        return 0.0 if e == 0.0 else float("inf")
    return e / D


def assert_close(got, want, D: float, tau: float, what: str = ""):
    r = norm_err(got, want, D)
    assert r <= tau, f"{what}: max|err|/D = {r:.3e} > {tau:.1e} (D = {D:.3e})"
    return r


def assert_bits(got, want, what: str = ""):
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    assert got.shape == want.shape, (what, got.shape, want.shape)
    bad = ~((got == want) & (np.signbit(got) == np.signbit(want)))
    n = int(np.count_nonzero(bad))
    assert n == 0, f"{what}: {n} of {got.size} elements differ in bits (first at {np.argwhere(bad)[0].tolist()})"


def mask_mismatch(h_gpu, y_ref, band: float):
    """Relu masks: count elements whose sign decision differs from the
    reference pre-activation outside the rounding band |y| <= band, and how
    many fall inside the band."""
    g = np.asarray(h_gpu) > 0
    r = np.asarray(y_ref) > 0
    outside = np.abs(np.asarray(y_ref)) > band
    return int(np.count_nonzero((g != r) & outside)), int(np.count_nonzero(~outside))
