"""MatMul with a workspace: the k range of an under-filled 16-bit problem is
split over several workgroups per output tile and the fp32 partials are added
in a fixed order. Parity against the oracle, against the unsplit call, and
determinism, through the C ABI."""

import numpy as np
import pytest
import torch

import oracle
from paper_1603_04467_amd import tfdense as T
from paper_1603_04467_amd.workloads import to_bf16_bits
from tests.parity import TAU, amax, assert_close, to_f64

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _host(rng, shape, scale=1.0):
    a = (rng.standard_normal(shape) * scale).astype(np.float32)
    bits = to_bf16_bits(a)
    t = torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).to(DEV)
    return oracle.bf16_bits_to_f64(bits), t


CASES = [
    # m, n, k, layout, out, epilogue, rounding
    (2048, 512, 4096, "NT", "bf16", "none", "nearest"),      # 16 tiles, 8 splits
    (512, 512, 8192, "NN", "bf16", "bias_relu", "nearest"),  # 4 tiles, 16 splits
    (512, 256, 16384, "TN", "f32", "none", "nearest"),       # 2 tiles, 32 splits (weight-gradient layout)
    (1024, 768, 4096, "NT", "f32", "bias", "nearest"),
    (2048, 512, 4096, "NT", "bf16", "bias_relu", "truncate"),
    (4096, 512, 2624, "NN", "bf16", "bias", "nearest"),      # 41 k-tiles: splits of 9, 9, 9, 9, 5
]


@pytest.mark.parametrize("m,n,k,layout,out,epi,rounding", CASES)
def test_split_k_matches_oracle_and_unsplit(m, n, k, layout, out, epi, rounding):
    rng = np.random.default_rng([m, n, k, len(layout), out == "f32", len(epi), rounding == "truncate"])
    ta, tb = layout == "TN", layout == "NT"
    a_h, a = _host(rng, (k, m) if ta else (m, k))
    b_h, b = _host(rng, (n, k) if tb else (k, n))
    bias_h = bias = None
    if epi != "none":
        bias_h = (rng.standard_normal(n) * 0.5).astype(np.float32)
        bias = torch.from_numpy(bias_h).to(DEV)
    odt = torch.bfloat16 if out == "bf16" else torch.float32
    need = T.tfd_matmul_workspace_size(m, n, k, torch.bfloat16, odt, transpose_a=ta, transpose_b=tb)
    assert need > 0, "this shape is meant to split"
    ws = torch.empty(need, dtype=torch.uint8, device=DEV)
    c = torch.full((m, n), float("nan"), dtype=odt, device=DEV)
    T.tfd_matmul(a, b, c, transpose_a=ta, transpose_b=tb, bias=bias, epilogue=epi, rounding=rounding, workspace=ws)
    c2 = torch.full((m, n), float("nan"), dtype=odt, device=DEV)
    T.tfd_matmul(a, b, c2, transpose_a=ta, transpose_b=tb, bias=bias, epilogue=epi, rounding=rounding, workspace=ws)
    c_plain = torch.full((m, n), float("nan"), dtype=odt, device=DEV)
    T.tfd_matmul(a, b, c_plain, transpose_a=ta, transpose_b=tb, bias=bias, epilogue=epi, rounding=rounding)
    # too small a workspace: exactly the plain call
    c_small = torch.full((m, n), float("nan"), dtype=odt, device=DEV)
    T.tfd_matmul(a, b, c_small, transpose_a=ta, transpose_b=tb, bias=bias, epilogue=epi, rounding=rounding,
                 workspace=ws[: need - 16])
    torch.cuda.synchronize()
    iv = torch.int16 if out == "bf16" else torch.int32
    assert torch.equal(c.view(iv), c2.view(iv)), "split result not reproducible"
    assert torch.equal(c_small.view(iv), c_plain.view(iv)), "workspace too small must give tfd_matmul's bits"
    store = out if rounding == "nearest" else "bf16t"
    bh = None if bias_h is None else bias_h.astype(np.float64)
    want = oracle.matmul(a_h, b_h, ta, tb, out=store, bias=bh, relu=epi == "bias_relu")
    D = k * amax(a_h) * amax(b_h) + (amax(bias_h) if bias_h is not None else 0.0)
    assert_close(to_f64(c), want, D, TAU["bf16"], "split-k MatMul")
    assert_close(to_f64(c), to_f64(c_plain), D, TAU["bf16"], "split-k vs unsplit")
    if epi == "bias_relu":
        assert not torch.any(torch.signbit(c.float()))


def test_split_k_integers_exact():
    # small integers: every partial and the sum are exact in fp32 and 16 bits
    rng = np.random.default_rng(7)
    m, n, k = 1024, 512, 8192
    a = rng.integers(-1, 2, size=(m, k)).astype(np.float32)
    b = rng.integers(-1, 2, size=(n, k)).astype(np.float32)
    at = torch.from_numpy(a).to(DEV).to(torch.bfloat16)
    bt = torch.from_numpy(b).to(DEV).to(torch.bfloat16)
    need = T.tfd_matmul_workspace_size(m, n, k, torch.bfloat16, torch.float32, transpose_b=True)
    assert need > 0
    ws = torch.empty(need, dtype=torch.uint8, device=DEV)
    c = torch.empty(m, n, device=DEV)
    T.tfd_matmul(at, bt, c, transpose_b=True, workspace=ws)
    torch.cuda.synchronize()
    assert np.array_equal(c.cpu().numpy().astype(np.float64), a.astype(np.float64) @ b.astype(np.float64).T)
