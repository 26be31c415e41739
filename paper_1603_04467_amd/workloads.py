"""Seeded synthetic inputs for the dense-layer training step.

This module only draws inputs; it holds none of the step's arithmetic, and it
is the one piece that both the HIP path and the oracle consume. Each tensor
has its own random stream, ``numpy.random.Generator(PCG64(SeedSequence([seed,
workload_id, tensor_id])))``, drawn in float32. Tensors stored in the 16-bit
format are converted once with torch's round-to-nearest-even cast (a library
routine), so both sides receive identical bits.

The workloads are MNIST-shaped (784 = 28x28 inputs, 10 classes, batch 100 as
in Figure 1 of the paper) and wide 4096-feature stacks; uniform [0, 1)
values stand in for pixel intensities. No dataset is read.
"""

from __future__ import annotations

import dataclasses
import math
from typing import Optional

import numpy as np

__all__ = ["Workload", "WORKLOADS", "workload", "generate", "to_bf16_bits"]


@dataclasses.dataclass(frozen=True)
class Workload:
    """Shape and initialisation recipe of one training-step workload.

    ``dims = (d0, d1, ..., dL)``: layer l maps ``d_{l-1} -> d_l``.
    ``act`` is the activation/GEMM-operand storage type ("f32" or "bf16").
    ``weight_init``: ("normal", std) or ("glorot",).
    ``bias_init``: ("zero",) or ("normal", std).
    ``cost``: "half_sq" (1/2 sum h^2), "sq_err" (1/2 sum (h - t)^2 against
    t ~ N(0,1)), "xent" (softmax cross-entropy against class labels drawn
    uniformly from [0, d_L)) or "upstream" (a given upstream gradient ~ N(0,1)).
    ``masters``: the updated fp32 Variables are separate from the 16-bit
    GEMM operands.
    ``rounding``: how 16-bit activations, input gradients and weight copies
    are produced from fp32: "nearest" (even) or "truncate" (the lossy
    converter of section 5.5).
    """
    name: str
    wid: int
    batch: int
    dims: tuple
    relus: tuple
    act: str
    input_dist: str            # "uniform01" or "normal"
    weight_init: tuple
    bias_init: tuple
    cost: str
    lr: float = 0.01
    update: bool = True
    masters: bool = False
    rounding: str = "nearest"

    @property
    def layers(self):
        return len(self.dims) - 1

    def gemm_shapes(self):
        """(m, n, k, layout) of every GEMM in one step, in launch order."""
        out = []
        N = self.batch
        for l in range(self.layers):
            out.append((N, self.dims[l + 1], self.dims[l], "NN"))
        for l in reversed(range(self.layers)):
            out.append((N, self.dims[l], self.dims[l + 1], "NT"))
            out.append((self.dims[l], self.dims[l + 1], N, "TN"))
        return out

    def flops(self):
        """GEMM FLOPs of one step: sum of 2*m*n*k."""
        return sum(2 * m * n * k for m, n, k, _ in self.gemm_shapes())

    def scaled(self, batch=None, dims=None, name=None):
        return dataclasses.replace(self, batch=batch or self.batch, dims=tuple(dims or self.dims),
                                   name=name or self.name + "-scaled")


WORKLOADS = {
    "dense784x100": Workload(
        name="dense784x100", wid=0, batch=100, dims=(784, 100), relus=(True,), act="f32",
        input_dist="uniform01", weight_init=("normal", 0.1), bias_init=("zero",), cost="half_sq"),
    "mlp784-1024-1024-10": Workload(
        name="mlp784-1024-1024-10", wid=1, batch=256, dims=(784, 1024, 1024, 10),
        relus=(True, True, False), act="f32", input_dist="uniform01", weight_init=("glorot",),
        bias_init=("zero",), cost="sq_err"),
    "mlp784-1024-1024-10-xent": Workload(
        name="mlp784-1024-1024-10-xent", wid=5, batch=256, dims=(784, 1024, 1024, 10),
        relus=(True, True, False), act="f32", input_dist="uniform01", weight_init=("glorot",),
        bias_init=("zero",), cost="xent"),
    "wide4096x4-f32": Workload(
        name="wide4096x4-f32", wid=2, batch=8192, dims=(4096,) * 5, relus=(True, True, True, False),
        act="f32", input_dist="normal", weight_init=("normal", 1.0 / 64.0), bias_init=("zero",),
        cost="sq_err"),
    "wide4096x4-bf16": Workload(
        name="wide4096x4-bf16", wid=3, batch=16384, dims=(4096,) * 5,
        relus=(True, True, True, False), act="bf16", input_dist="normal",
        weight_init=("normal", 1.0 / 64.0), bias_init=("zero",), cost="sq_err", masters=True),
    # same inputs as wide4096x4-bf16 (same workload id), truncating conversions
    "wide4096x4-bf16-trunc": Workload(
        name="wide4096x4-bf16-trunc", wid=3, batch=16384, dims=(4096,) * 5,
        relus=(True, True, True, False), act="bf16", input_dist="normal",
        weight_init=("normal", 1.0 / 64.0), bias_init=("zero",), cost="sq_err", masters=True,
        rounding="truncate"),
    "tall512x32768-bf16": Workload(
        name="tall512x32768-bf16", wid=4, batch=16384, dims=(512, 32768), relus=(True,),
        act="bf16", input_dist="normal", weight_init=("normal", 0.02), bias_init=("normal", 0.01),
        cost="upstream", update=False),
}


def workload(name: str) -> Workload:
    return WORKLOADS[name]


def _rng(seed, wid, tid):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, wid, tid])))


def to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Bits of the 16-bit float nearest to each float32 value (torch's cast)."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16).copy()


def _draw(rng, shape, dist):
    if dist[0] == "uniform01":
        return rng.random(shape, dtype=np.float32)
    if dist[0] == "normal":
        return rng.standard_normal(shape, dtype=np.float32) * np.float32(dist[1])
    if dist[0] == "uniform":
        a = np.float32(dist[1])
        return (rng.random(shape, dtype=np.float32) * np.float32(2.0) - np.float32(1.0)) * a
    raise ValueError(dist)


def generate(w: Workload, seed: int = 0) -> dict:
    """Draw every input of one step of ``w``.

    Returns numpy arrays: float32 for fp32 tensors, uint16 bit patterns for
    16-bit tensors. Keys: ``x``, ``weights`` (GEMM operands), ``masters``
    (fp32 Variables, or None), ``biases`` (fp32), ``target`` or ``upstream``
    (or None), ``labels`` (int32 class per row, or None), plus ``act``.
    """
    tid = 0
    out = {"act": w.act}
    in_dist = ("uniform01",) if w.input_dist == "uniform01" else ("normal", 1.0)
    x = _draw(_rng(seed, w.wid, tid), (w.batch, w.dims[0]), in_dist)
    tid += 1
    masters, weights, biases = [], [], []
    for l in range(w.layers):
        fi, fo = w.dims[l], w.dims[l + 1]
        if w.weight_init[0] == "glorot":
            dist = ("uniform", math.sqrt(6.0 / (fi + fo)))
        else:
            dist = ("normal", w.weight_init[1])
        wl = _draw(_rng(seed, w.wid, tid), (fi, fo), dist)
        tid += 1
        masters.append(wl)
    for l in range(w.layers):
        fo = w.dims[l + 1]
        if w.bias_init[0] == "zero":
            biases.append(np.zeros(fo, dtype=np.float32))
        else:
            biases.append(_draw(_rng(seed, w.wid, tid), (fo,), ("normal", w.bias_init[1])))
        tid += 1
    target: Optional[np.ndarray] = None
    upstream: Optional[np.ndarray] = None
    if w.cost == "sq_err":
        target = _draw(_rng(seed, w.wid, tid), (w.batch, w.dims[-1]), ("normal", 1.0))
    elif w.cost == "upstream":
        upstream = _draw(_rng(seed, w.wid, tid), (w.batch, w.dims[-1]), ("normal", 1.0))
    elif w.cost == "xent":
        out["labels"] = _rng(seed, w.wid, tid).integers(0, w.dims[-1], size=w.batch, dtype=np.int32)
    tid += 1
    out.setdefault("labels", None)

    if w.act == "bf16":
        out["x"] = to_bf16_bits(x)
        weights = [to_bf16_bits(m) for m in masters]
        out["masters"] = masters if w.masters else None
        out["target"] = None if target is None else to_bf16_bits(target)
        out["upstream"] = None if upstream is None else to_bf16_bits(upstream)
    else:
        out["x"] = x
        weights = masters
        out["masters"] = None
        out["target"] = target
        out["upstream"] = upstream
    out["weights"] = weights
    out["biases"] = biases
    return out
