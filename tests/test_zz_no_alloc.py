"""The entry point that allocates nothing: tfd_relu_grad_bias_add_grad_noalloc
(ReluGrad + BiasAddGrad, section 4.1) keeps its column partials in the
library's fixed device scratch instead of a caller's workspace. Through the
C ABI it must give exactly what tfd_relu_grad_bias_add_grad gives (same
kernels, same partial layout): dY and db bit for bit, on two calls in a row,
the second with a smaller input (the scratch keeps the first call's contents,
which the second must not see)."""

import numpy as np
import pytest
import torch

from paper_1603_04467_amd import tfdense as T

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _pair(rows, cols, dt, seed):
    g = torch.from_numpy(np.random.default_rng([seed, rows, cols]).standard_normal((rows, cols),
                                                                                   dtype=np.float32)).to(DEV).to(dt)
    f = torch.from_numpy(np.random.default_rng([seed + 1, rows, cols]).standard_normal((rows, cols),
                                                                                       dtype=np.float32)).to(DEV).to(dt)
    return g, f


def _reference(g, f, with_features=True):
    bp = torch.full_like(g, float("nan"))
    db = torch.full((g.shape[1],), float("nan"), device=DEV)
    T.tfd_relu_grad_bias_add_grad(g, f if with_features else None, bp if with_features else None, db)
    return bp, db


@pytest.mark.parametrize("dt", [torch.bfloat16, torch.float32])
def test_noalloc_equals_workspace_call_twice_shrinking(dt):
    for i, (rows, cols) in enumerate([(16384, 4096), (1000, 300)]):
        g, f = _pair(rows, cols, dt, 3 + i)
        bp = torch.full_like(g, float("nan"))
        db = torch.full((cols,), float("nan"), device=DEV)
        T.tfd_relu_grad_bias_add_grad_noalloc(g, f, bp, db)
        bp_ref, db_ref = _reference(g, f)
        torch.cuda.synchronize()
        assert torch.equal(bp.view(torch.uint8), bp_ref.view(torch.uint8)), (rows, cols, "dY")
        assert torch.equal(db.view(torch.uint8), db_ref.view(torch.uint8)), (rows, cols, "db")


def test_noalloc_bias_grad_only_and_tall_shape():
    for rows, cols in [(16384, 32768), (257, 1029)]:
        g, _ = _pair(rows, cols, torch.bfloat16, 9)
        db = torch.full((cols,), float("nan"), device=DEV)
        T.tfd_relu_grad_bias_add_grad_noalloc(g, None, None, db)
        _, db_ref = _reference(g, None, with_features=False)
        torch.cuda.synchronize()
        assert torch.equal(db.view(torch.uint8), db_ref.view(torch.uint8)), (rows, cols)


def test_noalloc_argument_errors():
    lib = T.load()
    assert lib.tfd_relu_grad_bias_add_grad_noalloc(None, None, None, None, -1, 4, 0, None) == T.TFD_EINVAL
    assert lib.tfd_relu_grad_bias_add_grad_noalloc(None, None, None, None, 4, 4, 0, None) == T.TFD_EINVAL
    assert lib.tfd_relu_grad_bias_add_grad_noalloc(None, None, None, None, 4, 0, 0, None) == T.TFD_OK
