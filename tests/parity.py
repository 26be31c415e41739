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


# ---------------------------------------------------------------------------
# Per-element bounds for one product, on the operands the kernel actually read
# ("teacher forcing"). The normalised rule above scales with the largest
# operands of the whole matrix; at production K it allows more than the size
# of a typical output element. The bound below scales with each element's own
# sum of |terms| and is tight enough to reject a dropped k-tile, a zero tile
# or an epilogue applied in the wrong order.
# ---------------------------------------------------------------------------

U32 = 2.0 ** -24           # unit roundoff of fp32
C_ACC = 2.0                # slack for accumulation orders and rounding inside the matrix cores

# significand bits of each storage type
_PREC = {"f32": 24, "bf16": 8, "bf16t": 8}


def ulp(values, store: str) -> np.ndarray:
    """Spacing of the storage format at each value (for 0 and subnormals,
    the subnormal quantum)."""
    v = np.abs(np.asarray(values, np.float64))
    p = _PREC[store]
    emin = -126
    _, e = np.frexp(v)                  # v = m * 2**e, 0.5 <= m < 1
    e = np.where(v > 0, np.maximum(e - 1, emin), emin)  # floor(log2 v), clamped to the normal range
    return np.ldexp(1.0, e - (p - 1))


def round_slack(store: str) -> float:
    """Largest rounding error of one store, in ulps of the stored value:
    half an ulp rounding to nearest, a whole one truncating."""
    return 1.0 if store == "bf16t" else 0.5


def product_bound(abs_terms, K: int, got, store: str, abs_bias=None) -> np.ndarray:
    """Bound on |stored - exact| for each element of an fp32-accumulated
    product of length K (products of 16-bit values are exact in fp32; fp32
    products add one rounding each, hence K + 1):
    C_ACC * (K + 1) * u * (sum |a_p b_p| + |bias|) + round_slack * ulp(stored).
    The bound also holds through ReLU (a 1-Lipschitz map that commutes with
    the rounding)."""
    s = np.asarray(abs_terms, np.float64)
    if abs_bias is not None:
        s = s + np.asarray(abs_bias, np.float64)[None, :]
    return C_ACC * (K + 1) * U32 * s + round_slack(store) * ulp(got, store)


def elementwise_excess(got, exact, bound) -> np.ndarray:
    """|got - exact| - bound per element (> 0 where the bound is broken)."""
    got = np.asarray(got, np.float64)
    return np.abs(got - np.asarray(exact, np.float64)) - np.asarray(bound, np.float64)


def assert_elementwise(got, exact, bound, what: str = ""):
    got = np.asarray(got, np.float64)
    assert got.shape == np.shape(exact), (what, got.shape, np.shape(exact))
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    ex = elementwise_excess(got, exact, bound)
    bad = ex > 0
    n = int(np.count_nonzero(bad))
    if n:
        i = tuple(np.argwhere(bad)[0])
        raise AssertionError(f"{what}: {n} of {got.size} elements outside the per-element bound "
                             f"(first at {list(i)}: got {got[i]!r}, exact {np.asarray(exact)[i]!r}, "
                             f"bound {np.asarray(bound)[i]:.3e})")


def check_relu_decisions(h_got, y_exact, bound, what: str = "", max_flip_frac: float = 1e-3):
    """ReLU decisions of a stored output against the exact pre-activation:
    outside the band |y| <= bound (the same per-element bound) the stored
    value must be > 0 exactly where y > 0; inside it either decision is a
    correct rounding of the method. Flips (decisions that differ from the
    sign of y) must stay below ``max_flip_frac`` of the elements (at least 4
    are allowed on tiny outputs). Returns (flips, in-band count)."""
    h = np.asarray(h_got, np.float64) > 0
    y = np.asarray(y_exact, np.float64)
    pos = y > 0
    band = np.abs(y) <= np.asarray(bound, np.float64)
    diff = h != pos
    outside = int(np.count_nonzero(diff & ~band))
    assert outside == 0, f"{what}: {outside} ReLU decisions differ from the exact sign outside the band"
    flips = int(np.count_nonzero(diff))
    assert flips <= max(max_flip_frac * diff.size, 4), \
        f"{what}: {flips} flipped ReLU decisions of {diff.size} (cap {max_flip_frac:.0e})"
    return flips, int(np.count_nonzero(band))
