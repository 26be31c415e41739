"""Bit-exact parity of the 16-bit whole-tile MatMul at the production shapes.

The operands are sparse matrices of -1, 0 and +1 (bf16 holds them exactly),
the biases and targets small integers. Every product is then exact in fp32,
every partial sum an integer far below 2**24, and every output an integer of
magnitude <= 256, which the 16-bit format holds exactly (so the single
rounding to the storage type leaves the exact value unchanged and is not
applied on the oracle's side; the magnitude is asserted). Any correct kernel,
whatever its summation order, must therefore store exactly the oracle's
values: the output, the ReLU mask, the ReluGrad-masked output, the column
sums of BiasAddGrad (integers < 2**24, exact in fp32 in any order), the
squared-error gradient and its float64 loss. A dropped or repeated k-tile, a
wrong epilogue order or a misplaced mask bit changes some of these bits.

Shapes: the 4096-wide layers' forward and input-gradient MatMuls
(16384 x 4096 x 4096), their weight gradient (4096 x 4096 x 16384), the tall
layer's forward (16384 x 32768 x 512) and input gradient (16384 x 512 x 32768,
split k and not); every layout and every fused epilogue of the kernel; and
2048 x 2048 x 2112, an odd number (33) of 64-wide k-tiles on the kernel the
default picks for long k ranges, and 2048 x 2048 x 12864 with its k range
split over four workgroups of 51, 51, 51 and 48 k-tiles.
The oracle forms each product once in float64 (section 2, Table 1 MatMul),
and applies the epilogue ops (BiasAdd, Relu, ReluGrad, BiasAddGrad, the
squared error) as separate definitions. Every output element is compared,
except for the 16384 x 32768 output of the tall forward MatMul, whose launch
is checked on 8 whole tile-rows (2048 rows: the first, the last and six
spread between them, each spanning every tile column and every k-tile).
"""

import numpy as np
import pytest
import torch

import oracle
from paper_1603_04467_amd import tfdense as T
from tests.parity import assert_bits, to_f64

pytestmark = pytest.mark.gpu

DEV = "cuda"

# (m, n, k) -> density of the nonzero signs in op(A) and op(B): about 256
# nonzero products per output at K = 4096, so that every k-tile of 64 holds
# nonzero terms of many outputs while |C| stays well below 256.
SHAPES = {
    (16384, 4096, 4096): 0.25,
    (4096, 4096, 16384): 0.125,
    (16384, 32768, 512): 0.5,
    (16384, 512, 32768): 0.0625,
    (2048, 2048, 2112): 0.34375,   # 33 k-tiles: an odd count on the default long-k kernel
    (2048, 2048, 12864): 0.09375,  # 201 k-tiles over 4 splits of 51, 51, 51 and 48
}


def _signs(rng, shape, density):
    """int8 matrix of -1, 0, +1 with P(nonzero) = density (even split of signs)."""
    q = int(round(density * 64))
    r = rng.integers(0, 64, size=shape, dtype=np.int8)
    out = np.zeros(shape, dtype=np.int8)
    out[r < q // 2] = -1
    out[(r >= q // 2) & (r < q)] = 1
    return out


def _bf16_dev(a_int: np.ndarray) -> torch.Tensor:
    """Device bf16 tensor of small integers (|v| <= 256): their fp32 patterns
    have 16 zero low bits, so the top halves are the 16-bit patterns."""
    bits = (np.ascontiguousarray(a_int).astype(np.float32).view(np.uint32) >> np.uint32(16)).astype(np.uint16)
    return torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(DEV)


_CACHE = {}


def _checked_rows(m, n):
    """Rows whose outputs are compared: all of them, or for outputs above
    2**27 elements (the 16384 x 32768 one) 8 whole tile-rows of 256 (first,
    last and six between)."""
    if m * n <= 1 << 27:
        return np.arange(m)
    tiles = np.unique(np.linspace(0, m // 256 - 1, 8).round().astype(int))
    return np.concatenate([np.arange(256 * t, 256 * t + 256) for t in tiles])


def _problem(shape):
    """Seeded operands of one shape (logical op(A) [m, k] and op(B) [k, n]),
    the integer bias and the oracle's product on the checked rows. One shape
    is kept at a time; targets and features are drawn when a case needs them."""
    if shape in _CACHE:
        return _CACHE[shape]
    _CACHE.clear()
    torch.cuda.empty_cache()
    m, n, k = shape
    rng = np.random.default_rng([11, m, n, k])
    A = _signs(rng, (m, k), SHAPES[shape])
    B = _signs(rng, (k, n), SHAPES[shape])
    rows = _checked_rows(m, n)
    z = oracle.matmul(A[rows].astype(np.float64), B.astype(np.float64), out="f64")
    bias = rng.integers(-4, 5, size=n).astype(np.float32)
    assert np.max(np.abs(z)) + 8 <= 256, "operands too dense for exact 16-bit outputs"
    # not trivial: every k-tile holds nonzero terms of most outputs, so
    # dropping one changes them
    for kt in (0, k // 128, k // 64 - 1):
        part = A[:64, 64 * kt:64 * (kt + 1)].astype(np.float64) @ B[64 * kt:64 * (kt + 1)].astype(np.float64)
        assert np.mean(part != 0) > 0.15, "a k-tile without nonzero terms"
    assert np.mean(z[:64] != 0) > 0.8
    p = {"A": A, "B": B, "z": z, "rows": rows, "bias": bias, "dev": {}, "rng": rng}
    _CACHE[shape] = p
    return p


def _ints(p, key, lo, hi):
    """A seeded integer matrix in [lo, hi] of the output's shape (targets,
    ReluGrad features), drawn once per shape."""
    if key not in p:
        m, n = p["A"].shape[0], p["B"].shape[1]
        p[key] = p["rng"].integers(lo, hi + 1, size=(m, n)).astype(np.int8)
    return p[key]


def _operands(p, layout):
    """Device operands a, b for `layout` holding the same logical op(A), op(B)."""
    if layout not in p["dev"]:
        A, B = p["A"], p["B"]
        a = A.T if layout == "TN" else A
        b = B.T if layout == "NT" else B
        p["dev"][layout] = (_bf16_dev(np.ascontiguousarray(a)), _bf16_dev(np.ascontiguousarray(b)))
    return p["dev"][layout]


def _out(shape, dt=torch.bfloat16):
    return torch.full(shape, float("nan"), dtype=dt, device=DEV)


def _chunks(p, chunk=2048):
    """(device row indices, positions in the oracle's checked rows) per chunk."""
    rows = p["rows"]
    for i0 in range(0, len(rows), chunk):
        sel = slice(i0, min(i0 + chunk, len(rows)))
        yield torch.from_numpy(rows[sel]).to(DEV), sel


def _assert_bits_rows(p, got: torch.Tensor, want_fn, what: str):
    """Bitwise comparison of the checked rows in chunks; want_fn(sel) gives
    the oracle's values of the checked rows at positions sel."""
    for dev_rows, sel in _chunks(p):
        assert_bits(to_f64(got.index_select(0, dev_rows)), want_fn(sel), f"{what} (checked rows {sel.start}..)")


CASES = []
for _layout in ("NT", "NN", "TN"):
    for _epi in ("none", "bias", "bias_relu", "relu_mask", "relu_grad", "relu_mask_grad", "l2_loss", "f32"):
        CASES.append(((16384, 4096, 4096), _layout, _epi))
for _layout in ("TN", "NT", "NN"):
    CASES.append(((4096, 4096, 16384), _layout, "f32"))
CASES += [((4096, 4096, 16384), "TN", "relu_mask"), ((4096, 4096, 16384), "TN", "relu_grad")]
for _layout in ("NT", "NN"):
    for _epi in ("relu_mask", "bias_relu", "none"):
        CASES.append(((16384, 32768, 512), _layout, _epi))
CASES += [((16384, 512, 32768), "NT", "split"), ((16384, 512, 32768), "NT", "none"),
          ((16384, 512, 32768), "NN", "f32"), ((16384, 512, 32768), "TN", "none")]
# an odd number of k-tiles (33) where the default picks the scheduled 4-wave
# loop, which then starts from a stage of zeros
for _layout in ("NT", "TN"):
    for _epi in ("none", "relu_mask", "relu_mask_grad", "f32"):
        CASES.append(((2048, 2048, 2112), _layout, _epi))
# the k range split over 4 workgroups per tile, 51 k-tiles each but the last
# (48): odd and even counts on the 4-wave loop, partial sums added by the
# split-k reduction
CASES += [((2048, 2048, 12864), "NT", "split"), ((2048, 2048, 12864), "TN", "split")]


@pytest.mark.parametrize("shape,layout,epi", CASES, ids=[f"{s[0]}x{s[1]}x{s[2]}-{l}-{e}" for s, l, e in CASES])
def test_whole_tile_exact(shape, layout, epi):
    m, n, k = shape
    p = _problem(shape)
    a, b = _operands(p, layout)
    ta, tb = layout == "TN", layout == "NT"
    z, rows = p["z"], p["rows"]
    bias_h = p["bias"].astype(np.float64)
    bias = torch.from_numpy(p["bias"]).to(DEV)
    print(f"exact {m}x{n}x{k} {layout} {epi}", flush=True)

    def forward(sel, op):
        """The oracle's forward ops on checked rows: BiasAdd, then Relu (the
        exact integers need no rounding to the storage type)."""
        y = z[sel] if op == "none" else oracle.bias_add(z[sel], bias_h, out="f64")
        return oracle.relu(y) if op == "bias_relu" else y

    if epi in ("none", "bias", "bias_relu", "split"):
        c = _out((m, n))
        op = "none" if epi == "split" else epi
        ws = None
        if epi == "split":
            need = T.tfd_matmul_workspace_size(m, n, k, torch.bfloat16, torch.bfloat16, transpose_b=tb)
            assert need > 0, "the tall input gradient is expected to split its k range"
            ws = torch.empty(need, dtype=torch.uint8, device=DEV)
        T.tfd_matmul(a, b, c, transpose_a=ta, transpose_b=tb, bias=None if op == "none" else bias, epilogue=op,
                     workspace=ws)
        torch.cuda.synchronize()
        _assert_bits_rows(p, c, lambda sel: forward(sel, op), f"{layout} {epi}")
    elif epi == "f32":
        c = _out((m, n), torch.float32)
        T.tfd_matmul(a, b, c, transpose_a=ta, transpose_b=tb)
        torch.cuda.synchronize()
        _assert_bits_rows(p, c, lambda sel: z[sel], f"{layout} fp32 output")
    elif epi == "relu_mask":
        c = _out((m, n))
        mask = T.new_relu_mask(m, n, DEV)
        mask.fill_(-1)
        T.tfd_matmul_relu_mask(a, b, bias, c, mask, transpose_a=ta, transpose_b=tb)
        torch.cuda.synchronize()
        _assert_bits_rows(p, c, lambda sel: forward(sel, "bias_relu"), f"{layout} Relu output")
        for dev_rows, sel in _chunks(p):
            got = mask.index_select(0, dev_rows).cpu().numpy().view(np.uint32)
            assert np.array_equal(got, oracle.relu_mask(forward(sel, "bias_relu"))), \
                f"{layout}: ReLU mask bits differ (checked rows {sel.start}..)"
    elif epi in ("relu_grad", "relu_mask_grad"):
        feats = _ints(p, "feats", -2, 2)       # 40 % positive, exact zeros included
        bp = _out((m, n))
        db = torch.full((n,), float("nan"), device=DEV)
        if epi == "relu_grad":
            T.tfd_matmul_relu_grad_bias_add_grad(a, b, _bf16_dev(feats), bp, db, transpose_a=ta, transpose_b=tb)
            dy = lambda sel: oracle.relu_grad(z[sel], feats[rows[sel]].astype(np.float64))  # noqa: E731
        else:
            words = oracle.relu_mask(feats.astype(np.float64))
            T.tfd_matmul_relu_mask_grad_bias_add_grad(a, b, torch.from_numpy(words.view(np.int32)).to(DEV), bp, db,
                                                      transpose_a=ta, transpose_b=tb)
            dy = lambda sel: oracle.relu_grad_from_mask(z[sel], words[rows[sel]])  # noqa: E731
        torch.cuda.synchronize()
        _assert_bits_rows(p, bp, dy, f"{layout} {epi} dY")
        assert len(rows) == m
        db_want = np.sum([oracle.bias_add_grad(dy(sel), out="f64") for _, sel in _chunks(p)], axis=0)
        assert_bits(to_f64(db), db_want, f"{layout} {epi} db (integers < 2**24)")
    elif epi == "l2_loss":
        target = _ints(p, "target", -4, 4)
        out, g = _out((m, n)), _out((m, n))
        loss = torch.full((1,), float("nan"), dtype=torch.float64, device=DEV)
        db = torch.full((n,), float("nan"), device=DEV)
        T.tfd_matmul_l2_loss_grad(a, b, bias, out, _bf16_dev(target), g, loss, db, transpose_a=ta, transpose_b=tb)
        torch.cuda.synchronize()
        assert len(rows) == m
        _assert_bits_rows(p, out, lambda sel: forward(sel, "bias"), f"{layout} output layer")
        l_want, db_want = 0.0, np.zeros(n)
        for dev_rows, sel in _chunks(p):
            g_want, l_part = oracle.l2_loss_grad(forward(sel, "bias"), target[rows[sel]].astype(np.float64),
                                                 grad_dtype="f64")
            assert np.max(np.abs(g_want)) <= 256
            assert_bits(to_f64(g.index_select(0, dev_rows)), g_want,
                        f"{layout} squared-error gradient (checked rows {sel.start}..)")
            l_want += l_part
            db_want += oracle.bias_add_grad(g_want, out="f64")
        assert loss.item() == l_want, f"{layout}: loss {loss.item()!r} != {l_want!r} (exact integers)"
        assert_bits(to_f64(db), db_want, f"{layout} squared-error db (integers < 2**24)")
    else:
        raise ValueError(epi)
