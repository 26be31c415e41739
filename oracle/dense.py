"""Plain float64 definitions of the ops that train the paper's dense layer.

The paper's canonical example (Figure 1, section 1) builds ``Relu(Wx + b)``
from the graph ops MatMul, Add and ReLU (section 2, Table 1), asks for
``[db, dW, dx] = tf.gradients(C, [b, W, x])`` (section 4.1) and keeps ``W``
and ``b`` in Variables that the training step mutates in place (section 2,
"Variables"). The functions below write those definitions out directly: each
output element is the exact mathematical value (a float64 sum of exactly
upcast operands) rounded once to the storage type. Batch-major layout is
used: activations are [batch, features], a layer's weight is
[fan_in, fan_out], so the layer computes ``H = Relu(X @ W + b)``.

Test infrastructure only; nothing in the product package imports this file.
"""

from __future__ import annotations

import numpy as np

STORAGE_TYPES = ("f64", "f32", "bf16", "bf16t")

# Largest finite value of the 16-bit format: fp32's exponent range with an
# 8-bit significand, (2 - 2**-7) * 2**127.
_BF16_MAX = (2.0 - 2.0 ** -7) * 2.0 ** 127
_BF16_MIN_NORMAL = 2.0 ** -126
_BF16_SUBNORMAL_QUANTUM = 2.0 ** -133


# --------------------------------------------------------------------------
# Storage rounding
# --------------------------------------------------------------------------

def round_bf16(x) -> np.ndarray:
    """Round float64 values once, to nearest (ties to even), to the 16-bit
    float of section 5.5: an IEEE fp32 with 16 fewer mantissa bits (sign,
    8-bit exponent, 7 stored fraction bits).

    The paper's converter truncates the dropped bits; tensors stored in this
    format here are rounded to nearest even instead (a reading, recorded in the
    design notes). Written from the format's arithmetic, not its bit layout:
    a normal value keeps 8 significant bits, the subnormal range has the fixed
    quantum 2**-133, and a value at or beyond the midpoint above the largest
    finite value becomes infinity. Returns float64 values that the format
    represents exactly.
    """
    x = np.asarray(x, dtype=np.float64)
    mant, expo = np.frexp(x)  # x = mant * 2**expo, 0.5 <= |mant| < 1
    with np.errstate(over="ignore", invalid="ignore"):
        normal = np.ldexp(np.round(mant * 256.0), expo - 8)  # np.round: ties to even
        subnormal = np.round(x / _BF16_SUBNORMAL_QUANTUM) * _BF16_SUBNORMAL_QUANTUM
        out = np.where(np.abs(x) >= _BF16_MIN_NORMAL, normal, subnormal)
        out = np.where(np.abs(out) > _BF16_MAX, np.copysign(np.inf, x), out)
    return np.where(np.isfinite(x), out, x)


def round_to(x, dtype: str) -> np.ndarray:
    """Round float64 values once to the storage type ``dtype``."""
    x = np.asarray(x, dtype=np.float64)
    if dtype == "f64":
        return x
    if dtype == "f32":
        # IEEE conversion float64 -> float32 rounds to nearest even.
        return x.astype(np.float32).astype(np.float64)
    if dtype == "bf16":
        return round_bf16(x)
    if dtype == "bf16t":
        # the 16-bit format reached through the lossy converter of section
        # 5.5: the producer's fp32 value (one rounding), then truncation
        from .convert import truncate_bf16
        return truncate_bf16(x)
    raise ValueError(f"unknown storage type {dtype!r}")


def bf16_bits_to_f64(bits) -> np.ndarray:
    """Exact value of 16-bit-format bit patterns (the top half of an fp32)."""
    u = np.asarray(bits).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def f64_to_bf16_bits(x) -> np.ndarray:
    """Bit patterns of float64 values that the 16-bit format represents exactly."""
    x = np.asarray(x, dtype=np.float64)
    f = x.astype(np.float32)
    if not np.array_equal(f.astype(np.float64), x, equal_nan=True):
        raise ValueError("value not representable as fp32")
    u = f.view(np.uint32)
    if np.any(u & np.uint32(0xFFFF)):
        raise ValueError("value not representable in the 16-bit format")
    return (u >> np.uint32(16)).astype(np.uint16)


# --------------------------------------------------------------------------
# Forward ops: MatMul, BiasAdd (the "+ b" Add), Relu
# --------------------------------------------------------------------------

def matmul(a, b, transpose_a=False, transpose_b=False, out="f32", bias=None, relu=False):
    """MatMul of section 2, Table 1, with the transpose attributes of the
    op: ``C = op(a) @ op(b)``, ``op(a) = a.T`` when ``transpose_a``.

    ``C[i, j] = sum_p op(a)[i, p] * op(b)[p, j]`` is formed in float64 (the
    library product stands for the sum). With ``bias`` the broadcast Add of
    Figure 1 (``Wx + b``) is applied before the single rounding, and with
    ``relu`` the ReLU (Table 1) as well, as in a fused producer. An empty
    reduction (k = 0) gives zeros.
    """
    A = np.asarray(a, dtype=np.float64)
    B = np.asarray(b, dtype=np.float64)
    if transpose_a:
        A = A.T
    if transpose_b:
        B = B.T
    if A.ndim != 2 or B.ndim != 2 or A.shape[1] != B.shape[0]:
        raise ValueError(f"shape mismatch {A.shape} x {B.shape}")
    z = A @ B
    if bias is not None:
        z = z + np.asarray(bias, dtype=np.float64)[None, :]
    if relu:
        z = np.where(z > 0.0, z, 0.0)
    return round_to(z, out)


def bias_add(value, bias, out="f32"):
    """BiasAdd: ``value[n, m] + bias[m]``, the broadcast Add of ``Wx + b``
    (Figure 1; Add in Table 1), rounded once."""
    v = np.asarray(value, dtype=np.float64)
    return round_to(v + np.asarray(bias, dtype=np.float64)[None, :], out)


def relu(features):
    """ReLU of Table 1: ``y > 0 ? y : +0``. Zero and negative zero map to
    +0; the derivative is taken as 0 at 0 (strict comparison)."""
    f = np.asarray(features, dtype=np.float64)
    return np.where(f > 0.0, f, 0.0)


# --------------------------------------------------------------------------
# Gradient functions added by automatic differentiation (section 4.1)
# --------------------------------------------------------------------------

def relu_grad(gradients, features):
    """Gradient function of ReLU: pass the upstream gradient where the
    forward output (``features``, the stored Relu output) is positive, +0
    elsewhere."""
    g = np.asarray(gradients, dtype=np.float64)
    f = np.asarray(features, dtype=np.float64)
    return np.where(f > 0.0, g, 0.0)


def relu_mask(features):
    """The test that ReluGrad applies to the stored forward output,
    ``features > 0``, kept as one bit per element (a storage form of the
    same predicate; the backward pass then reads bits instead of features).

    Row r of the result holds ``ceil(cols / 32)`` uint32 words; bit j of word
    w is 1 iff ``features[r, 32 w + j] > 0`` (so -0, +0 and NaN give 0), and
    the bits past the last column are 0.
    """
    f = np.asarray(features, dtype=np.float64)
    rows, cols = f.shape
    words = np.zeros((rows, (cols + 31) // 32), dtype=np.uint32)
    for c in range(cols):
        words[:, c // 32] |= (f[:, c] > 0.0).astype(np.uint32) << np.uint32(c % 32)
    return words


def relu_grad_from_mask(gradients, mask):
    """ReluGrad with its test read from a mask made by ``relu_mask``:
    ``gradients`` where the element's bit is 1, +0 elsewhere."""
    g = np.asarray(gradients, dtype=np.float64)
    rows, cols = g.shape
    m = np.asarray(mask, dtype=np.uint32)
    keep = np.zeros((rows, cols), dtype=bool)
    for c in range(cols):
        keep[:, c] = ((m[:, c // 32] >> np.uint32(c % 32)) & np.uint32(1)) == 1
    return np.where(keep, g, 0.0)


def bias_add_grad(out_backprop, out="f32"):
    """Gradient of the broadcast Add with respect to the bias: the sum of
    the upstream gradient over the broadcast (batch) dimension,
    ``db[m] = sum_n g[n, m]``, formed in float64 and rounded once."""
    g = np.asarray(out_backprop, dtype=np.float64)
    return round_to(g.sum(axis=0), out)


def l2_loss_grad(output, target=None, grad_dtype="f32"):
    """Cost head of the step and its gradient.

    Figure 1 leaves the cost as a function of the Relu output. The squared
    error ``L = 1/2 * sum (out - target)**2`` is used (with ``target = 0``,
    i.e. ``1/2 * sum out**2``, when no target is given); its gradient is
    ``G = out - target``. ``G`` is the exact difference rounded once to
    ``grad_dtype``; ``L`` is a float64 sum of exact terms.
    """
    o = np.asarray(output, dtype=np.float64)
    d = o if target is None else o - np.asarray(target, dtype=np.float64)
    loss = 0.5 * float(np.sum(d * d))
    return round_to(d, grad_dtype), loss


def softmax(logits):
    """SoftMax of section 2, Table 1, over the last axis:
    ``p[n, c] = exp(z[n, c]) / sum_j exp(z[n, j])``, evaluated with the row
    maximum subtracted (the same value, without overflow)."""
    z = np.asarray(logits, dtype=np.float64)
    e = np.exp(z - z.max(axis=1, keepdims=True))
    return e / e.sum(axis=1, keepdims=True)


def softmax_cross_entropy_grad(logits, labels, grad_dtype="f32"):
    """Classifier cost on the output layer: ``L = -sum_n log softmax(z_n)[y_n]``
    (a sum over the batch, like the squared error) and its gradient with
    respect to the logits, ``G = softmax(z) - onehot(y)``.

    Figure 1 leaves the cost open; this one is built from the SoftMax and Log
    ops of Table 1. ``L`` uses ``log sum_j exp(z_j) - z_y`` in float64; ``G`` is
    rounded once to ``grad_dtype``.
    """
    z = np.asarray(logits, dtype=np.float64)
    y = np.asarray(labels, dtype=np.int64)
    n = z.shape[0]
    m = z.max(axis=1)
    lse = m + np.log(np.exp(z - m[:, None]).sum(axis=1))
    loss = float(np.sum(lse - z[np.arange(n), y]))
    g = softmax(z)
    g[np.arange(n), y] -= 1.0
    return round_to(g, grad_dtype), loss


# --------------------------------------------------------------------------
# Stateful update (section 2 "Variables"; SGD of section 4.1)
# --------------------------------------------------------------------------

def _round_exact_fma_f32(alpha, delta, var):
    """fp32 value of the exact ``var - alpha * delta`` rounded once.

    ``alpha * delta`` of two fp32 values is exact in float64 (48-bit
    significand). The float64 sum ``s`` may be rounded; its exact error ``e``
    is recovered with Knuth's TwoSum. The nearest fp32 to ``s`` is then the
    nearest fp32 to ``s + e``, except when ``s`` sits exactly halfway between
    two fp32 values and ``e != 0``: then the exact value lies on ``e``'s side.
    """
    a = np.asarray(alpha, dtype=np.float32).astype(np.float64)
    d = np.asarray(delta, dtype=np.float32).astype(np.float64)
    v = np.asarray(var, dtype=np.float32).astype(np.float64)
    p = -a * d                      # exact
    s = p + v                       # rounded float64 sum
    bv = s - p                      # TwoSum
    e = (p - (s - bv)) + (v - bv)   # exact error: p + v == s + e
    r = s.astype(np.float32)        # nearest fp32 to s (ties to even)
    r64 = r.astype(np.float64)
    toward = np.where(s > r64, np.float32(np.inf), np.float32(-np.inf)).astype(np.float32)
    other = np.nextafter(r, toward)  # fp32 neighbour on s's side
    mid = (r64 + other.astype(np.float64)) * 0.5
    tie = (s != r64) & (s == mid) & (e != 0.0)
    beyond = tie & (np.sign(e) == np.sign(other.astype(np.float64) - r64))
    return np.where(beyond, other, r).astype(np.float64)


def apply_gradient_descent(var, alpha, delta, dtype="f32"):
    """ApplyGradientDescent on a Variable: ``var <- var - alpha * delta``.

    The update is the in-place mutation of a Variable's tensor (section 2,
    "Variables": AssignAdd is ``+=``) with the SGD step of section 4.1. For
    fp32 Variables the exact value is rounded once (the result of a fused
    multiply-add); ``dtype="f64"`` keeps it unrounded.
    """
    if dtype == "f64":
        return np.asarray(var, np.float64) - float(alpha) * np.asarray(delta, np.float64)
    if dtype != "f32":
        raise ValueError("Variables are fp32 or f64")
    return _round_exact_fma_f32(np.float32(alpha), delta, var)


# --------------------------------------------------------------------------
# One training step of a stack of dense layers
# --------------------------------------------------------------------------

def dense_step(x, weights, biases, relus, act="f32", target=None, upstream_grad=None,
               lr=0.01, masters=None, update=True, labels=None, rounding="nearest"):
    """Forward, gradient subgraph and SGD update of ``len(weights)`` dense
    layers, in the order a dependency-respecting schedule runs them.

    Forward (Figure 1): ``H_l = Relu(H_{l-1} @ W_l + b_l)`` (identity where
    ``relus[l]`` is False), stored in ``act``.
    Cost (section 4.1 computes ``dC/dX`` for a cost C): ``l2_loss_grad`` of
    the last output against ``target``, ``softmax_cross_entropy_grad`` against
    class ``labels``, or the given ``upstream_grad``.
    Backward, last layer first (section 4.1 backtracks from C): the ReLU
    gradient ``dY_l = relu_grad(G_l, H_l)`` (``dY_l = G_l`` on an identity
    layer), ``db_l = bias_add_grad(dY_l)``, ``dX_l = dY_l @ W_l.T`` (stored in
    ``act``, it is ``G_{l-1}``; computed for layer 1 too, the ``dx`` of
    ``tf.gradients``) and ``dW_l = H_{l-1}.T @ dY_l`` (fp32).
    Update: after every read of ``W_l`` by the backward pass (a control
    dependency, section 2), ``W_l`` and ``b_l`` take one SGD step of size
    ``lr``. ``weights`` are the GEMM operands; ``masters`` (default: the
    weights themselves) are the fp32 Variables that are updated. With 16-bit
    activations the operand is re-derived from the updated master by
    rounding.
    ``rounding="truncate"`` (16-bit activations only) stores the forward
    outputs H, the input gradients dX and the re-derived 16-bit weights
    through the truncating converter of section 5.5 instead of rounding to
    nearest even; the cost gradient keeps its exact rounding.
    """
    L = len(weights)
    if not (len(biases) == len(relus) == L):
        raise ValueError("one bias and one activation flag per layer")
    var_t = "f64" if act == "f64" else "f32"
    if rounding not in ("nearest", "truncate") or (rounding == "truncate" and act != "bf16"):
        raise ValueError("truncation applies to 16-bit activations only")
    store = "bf16t" if rounding == "truncate" else act
    h = [np.asarray(x, dtype=np.float64)]
    for l in range(L):
        h.append(matmul(h[l], weights[l], out=store, bias=biases[l], relu=relus[l]))

    if upstream_grad is not None:
        g, loss = np.asarray(upstream_grad, dtype=np.float64), None
    elif labels is not None:
        g, loss = softmax_cross_entropy_grad(h[L], labels, grad_dtype=act)
    else:
        g, loss = l2_loss_grad(h[L], target, grad_dtype=act)
    top_grad = g

    dy = [None] * L
    db = [None] * L
    dx = [None] * L
    dw = [None] * L
    new_w = list(weights)
    new_m = None if masters is None else list(masters)
    new_b = list(biases)
    for l in reversed(range(L)):
        dy[l] = relu_grad(g, h[l + 1]) if relus[l] else g
        db[l] = bias_add_grad(dy[l], out=var_t)
        dx[l] = matmul(dy[l], weights[l], transpose_b=True, out=store)
        dw[l] = matmul(h[l], dy[l], transpose_a=True, out=var_t)
        if update:
            master = weights[l] if masters is None else masters[l]
            m_new = apply_gradient_descent(master, lr, dw[l], dtype=var_t)
            if masters is not None:
                new_m[l] = m_new
            new_w[l] = round_to(m_new, store) if act == "bf16" else m_new
            new_b[l] = apply_gradient_descent(biases[l], lr, db[l], dtype=var_t)
        g = dx[l]

    return {
        "h": h, "loss": loss, "g": top_grad, "dy": dy, "db": db, "dx": dx, "dw": dw,
        "new_weights": new_w, "new_masters": new_m, "new_biases": new_b,
    }
