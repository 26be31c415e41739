"""Teacher-forced checks of every op of a training step.

After one step on the GPU, each op is checked against the oracle on the
operands the GPU itself read (its own activations, gradients and the
Variables' values before the update), so that no error of an earlier op
leaks into the check of a later one:

  forward   H_l = Relu(H_{l-1} W_l + b_l)       per-element product bound;
            ReLU decisions exact outside the band |y| <= bound, flips capped;
            ReLU masks equal the bits of the stored H_l > 0
  cost      G = H_L - T, L = 1/2 |G|^2          bit-exact / float64 sum bound
  backward  dY_l = ReluGrad(G_l, H_l)           bit-exact select where G_l is stored;
            fused into the input-gradient MatMul above it: per-element bound
            where H_l > 0 and +0 elsewhere
            dX_l = dY_l W_l^T                   per-element product bound
            dW_l = H_{l-1}^T dY_l               per-element product bound (fp32)
            db_l = column sums of dY_l          per-element sum bound (fp32)
  update    W_l, b_l <- fma(-lr, dW_l / db_l, old value)
                                                bit-exact, the 16-bit copies
                                                bit-exact from the new master

The bound of a product of length K is C_ACC * (K + 1) * u * (|A| @ |B| + |b|)
plus the rounding of the store (tests/parity.py); it follows each element's
own magnitude, so a dropped k-tile, a zero tile or a misplaced epilogue
breaks it at any K. The ops follow section 2 (MatMul, Add, ReLU, Variables)
and section 4.1 (the gradient subgraph, SGD) of the paper.
"""

from __future__ import annotations

import numpy as np
import torch

import oracle
from paper_1603_04467_amd.step import fused_below
from tests.parity import C_ACC, U32, assert_bits, assert_elementwise, check_relu_decisions, product_bound, to_f64, ulp


def _store(w):
    return "bf16t" if w.rounding == "truncate" else w.act


def _rows_of(t: torch.Tensor, rows):
    if rows is None:
        return to_f64(t)
    return to_f64(t.index_select(0, torch.as_tensor(rows, device=t.device)))


def _cols_of(t: torch.Tensor, cols):
    if cols is None:
        return to_f64(t)
    return to_f64(t.index_select(1, torch.as_tensor(cols, device=t.device)))


def _old(s, kind, l):
    """The Variables' values before the step (the pristine copies)."""
    L = s.w.layers
    i = {"W": 0, "b": L, "master": 2 * L}[kind] + l
    return s._saved[i]


def check_step(s, rows=None, cols=None, max_flip_frac=1e-3):
    """Teacher-forced checks of one completed step `s` (a DenseStep after
    run()). `rows` selects the batch rows of the row-local products (forward,
    input gradients); `cols(M)` gives the columns of a weight gradient with M
    columns to check (None: all rows, all columns). Returns the number of ReLU decisions that differ from the
    exact sign (all inside the band)."""
    w = s.w
    L = w.layers
    st = _store(w)
    flips = 0
    Wold = [to_f64(_old(s, "W", l)) for l in range(L)]
    bold = [to_f64(_old(s, "b", l)) for l in range(L)]
    H = [None] * (L + 1)
    for l in range(L + 1):
        H[l] = _rows_of(s.h[l], rows)

    # forward
    for l in range(L):
        K = w.dims[l]
        y = oracle.matmul(H[l], Wold[l], out="f64", bias=bold[l])
        bound = product_bound(np.abs(H[l]) @ np.abs(Wold[l]), K, H[l + 1], st, abs_bias=np.abs(bold[l]))
        if w.relus[l]:
            assert_elementwise(H[l + 1], oracle.relu(y), bound, f"H_{l + 1}")
            assert not np.any(np.signbit(H[l + 1])), f"H_{l + 1}: Relu output with a sign bit"
            f, _ = check_relu_decisions(H[l + 1], y, bound, f"layer {l + 1}", max_flip_frac)
            flips += f
            if s.masks[l] is not None:
                got = s.masks[l].cpu().numpy().view(np.uint32)
                got = got if rows is None else got[rows]
                assert np.array_equal(got, oracle.relu_mask(H[l + 1])), f"mask_{l + 1}"
        else:
            assert_elementwise(H[l + 1], y, bound, f"H_{l + 1}")

    # cost gradient (the whole output: the fused output layer also sums G's columns)
    top = L - 1
    G_full = to_f64(s.g)
    if w.cost in ("sq_err", "half_sq"):
        Hl = to_f64(s.h[L])
        T = None if s.target is None else to_f64(s.target)
        g_want, l_want = oracle.l2_loss_grad(Hl, T, grad_dtype=w.act)
        assert_bits(G_full, g_want, "G")
        # float64 sum of n squares of fp32 differences (each difference
        # rounded at most once): relative error <= 4u + n 2^-53
        n = Hl.size
        assert abs(s.loss.item() - l_want) <= (4 * U32 + n * 2.0 ** -53) * l_want, ("loss", s.loss.item(), l_want)

    # backward, last layer first
    for l in reversed(range(L)):
        M = w.dims[l + 1]
        # dY_l on all rows (the bias gradient sums them)
        dY_full = to_f64(s.dy_of(l))
        if l == top:
            if w.relus[l]:
                assert_bits(dY_full, oracle.relu_grad(G_full, to_f64(s.h[L])), f"dY_{l + 1} = ReluGrad(G)")
            else:
                assert_bits(dY_full, G_full, f"dY_{l + 1} = G")
        elif not fused_below(w, l + 1, s.fuse):
            # the input gradient above was stored: dY is the exact select
            if w.relus[l]:
                assert_bits(dY_full, oracle.relu_grad(to_f64(s.dx[l + 1]), to_f64(s.h[l + 1])),
                            f"dY_{l + 1} = ReluGrad(dX_{l + 2})")
        dY = dY_full if rows is None else dY_full[rows]

        # input gradient of layer l + 1 (0-based l): dX_l = dY_l W_l^T, stored,
        # or fused with the ReluGrad of the layer below into dY_{l-1}
        K = M
        gx = oracle.matmul(dY, Wold[l], transpose_b=True, out="f64")
        absx = np.abs(dY) @ np.abs(Wold[l]).T
        if fused_below(w, l, s.fuse):
            got = _rows_of(s.dy[l - 1], rows)
            keep = H[l] > 0
            bound = product_bound(absx, K, got, st)
            assert_elementwise(np.where(keep, got, 0.0), np.where(keep, gx, 0.0), bound,
                               f"dY_{l} (fused input gradient of layer {l + 1})")
            assert_bits(np.where(keep, 0.0, got), np.zeros_like(got), f"dY_{l} where H_{l} <= 0")
        else:
            got = _rows_of(s.dx[l], rows)
            assert_elementwise(got, gx, product_bound(absx, K, got, st), f"dX_{l + 1}")

        # bias gradient over all rows: fp32 sums of the stored dY
        db = to_f64(s.db[l])
        colsum = oracle.bias_add_grad(dY_full, out="f64")
        abssum = np.abs(dY_full).sum(axis=0)
        bound = C_ACC * w.batch * U32 * abssum + 0.5 * ulp(db, "f32")
        assert_elementwise(db, colsum, bound, f"db_{l + 1}")

        # weight gradient on the selected columns: dW = H_{l-1}^T dY, K = batch
        Hin = to_f64(s.h[l])
        cl = None if cols is None else cols(M)
        dYc = dY_full if cl is None else dY_full[:, cl]
        dw_want = oracle.matmul(Hin, dYc, transpose_a=True, out="f64")
        got = _cols_of(s.dw[l], cl)
        bound = product_bound(np.abs(Hin).T @ np.abs(dYc), w.batch, got, "f32")
        assert_elementwise(got, dw_want, bound, f"dW_{l + 1}")

        # update: bit-exact from the GPU's own gradients and the old values
        if w.update:
            dW_full = s.dw[l].cpu().numpy()
            if s.masters is not None:
                new = oracle.apply_gradient_descent(_old(s, "master", l).cpu().numpy(), np.float32(w.lr), dW_full)
                assert_bits(to_f64(s.masters[l]), new, f"W_{l + 1} (master)")
                assert_bits(to_f64(s.weights[l]), oracle.round_to(new, st), f"W16_{l + 1}")
                if s.weights_t is not None:
                    assert torch.equal(s.weights_t[l], s.weights[l].t()), f"W^T_{l + 1}"
            else:
                new = oracle.apply_gradient_descent(_old(s, "W", l).cpu().numpy(), np.float32(w.lr), dW_full)
                assert_bits(to_f64(s.weights[l]), new, f"W_{l + 1}")
            newb = oracle.apply_gradient_descent(_old(s, "b", l).cpu().numpy(), np.float32(w.lr),
                                                 s.db[l].cpu().numpy())
            assert_bits(to_f64(s.biases[l]), newb, f"b_{l + 1}")
        else:
            assert torch.equal(s.weights[l], _old(s, "W", l)), f"W_{l + 1} changed without an update"
    return flips


def sample_rows(n, tile=256, tiles=4, extra=64, seed=0):
    """Whole tile-rows (first, last and spread between) plus random rows."""
    nt = max(n // tile, 1)
    picks = np.unique(np.linspace(0, nt - 1, min(tiles, nt)).round().astype(int))
    rows = [np.arange(t * tile, min(t * tile + tile, n)) for t in picks]
    rng = np.random.default_rng(seed)
    rows.append(rng.choice(n, size=min(extra, n), replace=False))
    return np.unique(np.concatenate(rows))


def sample_cols(n, tile=256, tiles=2, extra=64, seed=1):
    return sample_rows(n, tile, tiles, extra, seed)


__all__ = ["check_step", "sample_rows", "sample_cols"]
