"""End-to-end parity of one training step (the exact launch sequence that
bench.py times) against the oracle's chain from the same seeded inputs.

Forward tensors, the loss and the output layer's gradients are continuous in
the rounding errors and are compared with the normalised-error rule. Below a
Relu, a mask decision on a pre-activation inside the rounding band of zero
may legitimately differ between the GPU and the oracle (both are correct
steps of the method); such a flip changes the whole row of every input
gradient below it. The checks therefore
  - require every mask difference to lie inside the band (and count them),
  - compare row-local tensors (dY, dX) on the rows no flip touched,
  - bound the batch reductions (dW, db) by tau * D plus the largest change
    the touched rows can make,
  - check on the GPU's own tensors that dY is exactly G where H > 0 and +0
    elsewhere, and the per-layer adjoint identity
    <G_l, H_l> = <W_l, dW_l> + <b_l, db_l>.
At the full sizes the oracle runs the whole forward pass and the output
layer's backward pass, and the Relu layers' input gradients on sampled rows.
"""

import numpy as np
import pytest
import torch

import oracle
from paper_1603_04467_amd import workloads
from paper_1603_04467_amd.step import DenseStep, fused_below
from tests.parity import TAU, amax, assert_bits, assert_close, product_bound, to_f64
from tests.teacher import check_step, sample_cols, sample_rows

pytestmark = pytest.mark.gpu


def _store(w):
    """Oracle storage type of the step's 16-bit activations and weight copies."""
    return "bf16t" if w.rounding == "truncate" else w.act


def _host_inputs(w, inp):
    conv = oracle.bf16_bits_to_f64 if w.act == "bf16" else (lambda a: a.astype(np.float64))
    if w.rounding == "truncate":
        # the 16-bit operand copies are derived from the fp32 masters by the converter
        weights = [oracle.round_to(a.astype(np.float64), "bf16t") for a in inp["masters"]]
    else:
        weights = [conv(a) for a in inp["weights"]]
    return {
        "x": conv(inp["x"]),
        "weights": weights,
        "masters": None if inp["masters"] is None else [a.astype(np.float64) for a in inp["masters"]],
        "biases": [a.astype(np.float64) for a in inp["biases"]],
        "target": None if inp["target"] is None else conv(inp["target"]),
        "upstream": None if inp["upstream"] is None else conv(inp["upstream"]),
        "labels": inp.get("labels"),
    }


def _assert_within(got, want, allowed, what):
    got = np.asarray(got, np.float64)
    assert np.all(np.isfinite(got)), f"{what}: non-finite"
    if got.size == 0:
        return
    e = float(np.max(np.abs(got - want)))
    assert e <= allowed, f"{what}: max|err| = {e:.3e} > allowed {allowed:.3e}"


def _run_gpu(w, inp, fuse=True, masks=None):
    s = DenseStep(w, inp, fuse=fuse, masks=masks)
    s.run()
    torch.cuda.synchronize()
    return s


# Caps on ReLU decisions that differ between the GPU's chain and the oracle's
# (all inside the band): at most this share of a layer's elements, and of the
# batch rows across all layers. A float32 emulation of the chain on the host
# (another summation order) flips about 1.5e-5 of the elements of the deepest
# Relu layer and touches about 5 % of the rows of the 4096-wide step.
MAX_FLIP_FRAC = 1e-3
MAX_TOUCHED_ROWS = 0.25


def _band(h_in_gpu, h_in_ref, W, b, h_out_gpu, y_ref, store):
    """Per-element band of a Relu layer's decision in the end-to-end chain:
    the GPU's pre-activation differs from the oracle's by at most the
    product bound on the GPU's own inputs plus |(H_gpu - H_ref) W| (the
    exact effect of the inputs' earlier differences)."""
    K = W.shape[0]
    bound = product_bound(np.abs(h_in_gpu) @ np.abs(W), K, h_out_gpu, store, abs_bias=np.abs(b))
    y_gpu = oracle.matmul(h_in_gpu, W, out="f64", bias=b)
    return bound + np.abs(y_gpu - y_ref)


def _flip_rows(h_gpu, y_ref, band, what):
    """Rows where the GPU's Relu decision differs from the sign of the
    oracle's pre-activation; every such element must be inside the band, and
    their number below MAX_FLIP_FRAC of the layer."""
    diff = (h_gpu > 0) != (y_ref > 0)
    outside = diff & (np.abs(y_ref) > band)
    assert not np.any(outside), f"{what}: {int(outside.sum())} mask decisions differ outside the band"
    n = int(diff.sum())
    assert n <= MAX_FLIP_FRAC * diff.size, f"{what}: {n} flipped mask decisions of {diff.size}"
    return np.any(diff, axis=1)


def _check_mask_consistency(s, l):
    """dY = G where the stored H > 0, +0 elsewhere (bit for bit, GPU tensors)."""
    g = s.g if l == s.w.layers - 1 else s.dx[l + 1]
    h = s.h[l + 1]
    want = torch.where(h > 0, g, torch.zeros_like(g))
    assert torch.equal(s.dy[l], want), f"layer {l + 1}: dY is not G masked by H > 0"
    assert not torch.any(torch.signbit(h)), f"layer {l + 1}: Relu output with a sign bit"


def _check_adjoint(s, l, tau):
    """<G_l, H_l> = <W_l, dW_l> + <b_l, db_l> on the GPU's tensors (with
    <dY_l, H_l> for <G_l, H_l>: the mask only zeroes entries where H_l = 0)."""
    g = to_f64(s.dy_of(l))
    h = to_f64(s.h[l + 1])
    x = to_f64(s.h[l])
    dy = to_f64(s.dy_of(l))
    W = s._saved[l].float().cpu().numpy().astype(np.float64)
    b = s._saved[len(s.weights) + l].cpu().numpy().astype(np.float64)
    dw = to_f64(s.dw[l])
    db = to_f64(s.db[l])
    lhs = float(np.sum(g * h))
    rhs = float(np.sum(W * dw) + np.sum(b * db))
    K = x.shape[1]
    D = float(np.sum(np.abs(dy))) * (K * amax(x) * amax(W) + amax(b))
    assert abs(lhs - rhs) <= tau * D, f"layer {l + 1}: adjoint identity off by {abs(lhs - rhs):.3e} (D {D:.3e})"


def _compare_full(w, inp, s):
    """Whole-step comparison against the oracle's full chain."""
    hi = _host_inputs(w, inp)
    tau = TAU[w.act]
    L = w.layers
    ref = oracle.dense_step(hi["x"], hi["weights"], hi["biases"], list(w.relus), act=w.act,
                            target=hi["target"], upstream_grad=hi["upstream"], lr=w.lr,
                            masters=hi["masters"], update=w.update, labels=hi["labels"], rounding=w.rounding)
    h_gpu = [to_f64(t) for t in s.h]
    # forward
    D_fwd = []
    for l in range(L):
        D = w.dims[l] * amax(ref["h"][l]) * amax(hi["weights"][l]) + amax(hi["biases"][l])
        D_fwd.append(D)
        assert_close(h_gpu[l + 1], ref["h"][l + 1], D, tau, f"H_{l + 1}")
    # mask flips (rows touched, cumulated from the top)
    touched = np.zeros(w.batch, dtype=bool)
    touched_at = [None] * L
    flips = 0
    for l in reversed(range(L)):
        if w.relus[l]:
            y = oracle.matmul(ref["h"][l], hi["weights"][l], out="f64", bias=hi["biases"][l])
            band = _band(h_gpu[l], ref["h"][l], hi["weights"][l], hi["biases"][l], h_gpu[l + 1], y, _store(w))
            rows = _flip_rows(h_gpu[l + 1], y, band, f"layer {l + 1}")
            flips += int(rows.sum())
            touched |= rows
        touched_at[l] = touched.copy()
    assert touched.sum() <= MAX_TOUCHED_ROWS * w.batch, f"{int(touched.sum())} rows touched by mask flips"
    # cost
    g_gpu = to_f64(s.g)
    if ref["loss"] is not None and hi["labels"] is not None:
        # softmax is 1/2-Lipschitz per element in the max-norm of the logits,
        # each row's cross-entropy 2-Lipschitz; the fp32 exp/log/sum add
        # a few ulp of p and of log-sum-exp per row
        D_G = D_fwd[-1] + amax(ref["g"])
        assert_close(g_gpu, ref["g"], D_G, tau, "G")
        C = w.dims[-1]
        per_row = 2.0 * tau * D_fwd[-1] + (C / 64 + 80 + 2 * amax(ref["h"][L])) * 2.0 ** -23
        _assert_within(np.array([s.loss.item()]), np.array([ref["loss"]]), w.batch * per_row, "loss")
    elif ref["loss"] is not None:
        D_G = D_fwd[-1] + amax(ref["g"])
        assert_close(g_gpu, ref["g"], D_G, tau, "G")
        allowed = tau * D_fwd[-1] * float(np.sum(np.abs(ref["g"]))) + 1e-12 * ref["loss"]
        _assert_within(np.array([s.loss.item()]), np.array([ref["loss"]]), allowed, "loss")
    else:
        D_G = amax(ref["g"])
        assert_bits(g_gpu, ref["g"], "upstream gradient")
    # backward
    D_g = D_G
    for l in reversed(range(L)):
        keep = ~touched_at[l]
        nt = int((~keep).sum())
        dy_ref = ref["dy"][l]
        dy_gpu = to_f64(s.dy_of(l))
        if w.relus[l]:
            if not fused_below(w, l + 1, s.fuse):
                _check_mask_consistency(s, l)
            assert_close(dy_gpu[keep], dy_ref[keep], D_g, tau, f"dY_{l + 1}")
        W = hi["weights"][l]
        M = w.dims[l + 1]
        md = amax(dy_ref)
        D_dx = M * md * amax(W)
        if not fused_below(w, l, s.fuse):     # fused: dX_l is not stored, only the dY below it
            assert_close(to_f64(s.dx[l])[keep], ref["dx"][l][keep], D_dx, tau, f"dX_{l + 1}")
        mh = amax(ref["h"][l])
        _assert_within(to_f64(s.dw[l]), ref["dw"][l], tau * w.batch * mh * md + 2 * nt * mh * md, f"dW_{l + 1}")
        _assert_within(to_f64(s.db[l]), ref["db"][l], tau * w.batch * md + 2 * nt * md, f"db_{l + 1}")
        _check_adjoint(s, l, tau)
        if w.update:
            allowed_w = w.lr * (tau * w.batch * mh * md + 2 * nt * mh * md)
            if s.masters is not None:
                if s.weights_t is not None:
                    assert torch.equal(s.weights_t[l], s.weights[l].t()), f"W^T_{l + 1} is not the transposed copy"
                mw = amax(ref["new_masters"][l])
                _assert_within(to_f64(s.masters[l]), ref["new_masters"][l], allowed_w + 2.0 ** -23 * mw, f"W_{l + 1}")
                # one 16-bit step: half of one under nearest even, a whole one under truncation
                step16 = 2.0 ** -7 if w.rounding == "truncate" else 2.0 ** -8
                _assert_within(to_f64(s.weights[l]), ref["new_weights"][l], allowed_w + step16 * mw, f"W16_{l + 1}")
                # the copy is exactly the GPU's own updated master through the converter
                own = oracle.round_to(to_f64(s.masters[l]), _store(w))
                assert_bits(to_f64(s.weights[l]), own, f"W16_{l + 1} from the updated master")
            else:
                mw = amax(ref["new_weights"][l])
                _assert_within(to_f64(s.weights[l]), ref["new_weights"][l], allowed_w + 2.0 ** -23 * mw, f"W_{l + 1}")
            allowed_b = w.lr * (tau * w.batch * md + 2 * nt * md) + 2.0 ** -23 * amax(ref["new_biases"][l])
            _assert_within(to_f64(s.biases[l]), ref["new_biases"][l], allowed_b, f"b_{l + 1}")
        else:
            assert torch.equal(s.weights[l], s._saved[l])
        D_g = D_dx
    return flips


SCALED = [
    ("dense784x100", None, None),
    ("mlp784-1024-1024-10", None, None),
    ("mlp784-1024-1024-10-xent", None, None),
    ("mlp784-1024-1024-10-xent", 200, (784, 1024, 1024, 1000)),
    ("wide4096x4-f32", 600, (256, 384, 264, 128, 200)),
    ("wide4096x4-f32", 520, (136, 256, 512, 264, 128)),
    ("wide4096x4-bf16", 600, (256, 384, 264, 128, 200)),
    ("wide4096x4-bf16", 1032, (512, 768, 512, 256, 512)),
    ("wide4096x4-bf16", 1024, (512, 1024, 768, 512, 256)),      # whole 256 x 256 tiles everywhere
    ("wide4096x4-bf16-trunc", 600, (256, 384, 264, 128, 200)),
    ("wide4096x4-bf16-trunc", 768, (256, 512, 256, 256, 512)),
    ("wide4096x4-bf16-trunc", 1032, (512, 768, 512, 256, 512)),
    ("tall512x32768-bf16", 1000, (512, 2048)),
    ("tall512x32768-bf16", 1024, (512, 4096)),
    ("tall512x32768-bf16", 264, (96, 4104)),
    ("tall512x32768-bf16", 130, (100, 1030)),
]


@pytest.mark.parametrize("fuse", [True, False])
@pytest.mark.parametrize("name,batch,dims", SCALED)
def test_step_matches_oracle(name, batch, dims, fuse):
    w = workloads.workload(name)
    if batch is not None:
        w = w.scaled(batch=batch, dims=dims)
    inp = workloads.generate(w, seed=0)
    s = _run_gpu(w, inp, fuse=fuse)
    flips = _compare_full(w, inp, s)
    tf = check_step(s)
    print(f"{w.name}: {flips} rows with in-band Relu mask differences; {tf} teacher-forced flips")


@pytest.mark.parametrize("name,batch,dims", [("mlp784-1024-1024-10", None, None),
                                             ("wide4096x4-bf16", 1032, (512, 768, 512, 256, 512)),
                                             ("wide4096x4-bf16-trunc", 600, (256, 384, 264, 128, 200)),
                                             ("wide4096x4-f32", 520, (136, 256, 512, 264, 128))])
def test_fused_step_equals_unfused(name, batch, dims):
    """The fused input-gradient/ReluGrad/BiasAddGrad call stores the same dY
    bits as the two calls it replaces, so every tensor downstream of dY is
    bitwise equal; only db (and the bias update) may differ, by the order of
    the column sums."""
    w = workloads.workload(name)
    if batch is not None:
        w = w.scaled(batch=batch, dims=dims)
    inp = workloads.generate(w, seed=5)
    a = _run_gpu(w, inp, fuse=True)
    b = _run_gpu(w, inp, fuse=False)
    for l in range(w.layers):
        assert torch.equal(a.h[l + 1], b.h[l + 1])
        assert torch.equal(a.dy_of(l), b.dy_of(l)), f"dY_{l + 1}"
        assert torch.equal(a.dw[l], b.dw[l]), f"dW_{l + 1}"
        assert torch.equal(a.weights[l], b.weights[l]), f"W_{l + 1}"
        md = float(b.dy_of(l).abs().max())
        tol = TAU["f32"] * w.batch * md
        assert float((a.db[l] - b.db[l]).abs().max()) <= tol, f"db_{l + 1}"
        assert float((a.biases[l] - b.biases[l]).abs().max()) <= w.lr * tol + 2.0 ** -23 * float(
            b.biases[l].abs().max()), f"b_{l + 1}"
    assert torch.equal(a.dx[0], b.dx[0])


@pytest.mark.parametrize("fuse", [True, False])
@pytest.mark.parametrize("name,batch,dims", [("wide4096x4-bf16", 512, (512, 768, 512, 256, 512)),
                                             ("wide4096x4-bf16", 1032, (512, 768, 512, 256, 512)),
                                             ("wide4096x4-bf16-trunc", 768, (256, 512, 256, 256, 512)),
                                             ("tall512x32768-bf16", 512, (512, 1024)),
                                             ("wide4096x4-f32", 520, (136, 256, 512, 264, 128)),
                                             ("mlp784-1024-1024-10-xent", None, None)])
def test_masked_step_equals_features_step(name, batch, dims, fuse):
    """A step that keeps ReLU masks (one bit of H > 0 per element, written by
    the forward MatMul) stores exactly what the features-based step stores:
    every tensor, db included, bit for bit."""
    w = workloads.workload(name)
    if batch is not None:
        w = w.scaled(batch=batch, dims=dims)
    inp = workloads.generate(w, seed=6)
    a = _run_gpu(w, inp, fuse=fuse, masks=True)
    b = _run_gpu(w, inp, fuse=fuse, masks=False)
    assert any(m is not None for m in a.masks) and all(m is None for m in b.masks)
    for l in range(w.layers):
        if a.masks[l] is not None:
            want = oracle.relu_mask(to_f64(a.h[l + 1]))
            assert np.array_equal(a.masks[l].cpu().numpy().view(np.uint32), want), f"mask_{l + 1}"
    pairs = [(a.h[l + 1], b.h[l + 1]) for l in range(w.layers)] + [(a.dy_of(l), b.dy_of(l)) for l in range(w.layers)]
    pairs += list(zip(a.dw + a.db + a.variables(), b.dw + b.db + b.variables())) + [(a.loss, b.loss), (a.dx[0], b.dx[0])]
    for x, y in pairs:
        assert torch.equal(x.view(torch.uint8), y.view(torch.uint8))


@pytest.mark.parametrize("name", ["dense784x100", "mlp784-1024-1024-10-xent", "wide4096x4-bf16"])
def test_step_is_deterministic(name):
    w = workloads.workload(name)
    if name == "wide4096x4-bf16":
        w = w.scaled(batch=1032, dims=(512, 768, 512, 256, 512))
    inp = workloads.generate(w, seed=3)
    s = DenseStep(w, inp)
    dx = [s.dx[l] for l in range(w.layers) if not fused_below(w, l, s.fuse)]
    s.run()
    first = [t.clone() for t in dx + s.dw + s.db + s.variables()] + [s.loss.clone()]
    s.restore()
    s.run()
    torch.cuda.synchronize()
    second = [t for t in dx + s.dw + s.db + s.variables()] + [s.loss]
    for a, b in zip(first, second):
        assert torch.equal(a.view(torch.uint8), b.view(torch.uint8))


# ---------------------------------------------------------------- full sizes

def _sampled_rows(n, count=48, seed=0):
    rng = np.random.default_rng(seed)
    return np.unique(np.concatenate([[0, n - 1], rng.choice(n, size=min(count, n), replace=False)]))


def _check_full_size(name):
    """Full-size step: the oracle's whole forward pass, the output layer's
    backward pass in full, the Relu layers' input gradients on sampled rows,
    and the identities on the GPU's own tensors."""
    w = workloads.workload(name)
    inp = workloads.generate(w, seed=0)
    s = _run_gpu(w, inp)
    hi = _host_inputs(w, inp)
    tau = TAU[w.act]
    L = w.layers
    if L == 1:
        return _compare_full(w, inp, s)
    # forward in full (continuous: compared everywhere)
    h_ref = [hi["x"]]
    D_fwd = []
    y_ref = []
    for l in range(L):
        D = w.dims[l] * amax(h_ref[l]) * amax(hi["weights"][l]) + amax(hi["biases"][l])
        y = oracle.matmul(h_ref[l], hi["weights"][l], out="f64", bias=hi["biases"][l])
        h = oracle.round_to(oracle.relu(y) if w.relus[l] else y, _store(w))
        y_ref.append(y)
        h_ref.append(h)
        D_fwd.append(D)
        assert_close(to_f64(s.h[l + 1]), h, D, tau, f"H_{l + 1}")
    g_ref, loss_ref = oracle.l2_loss_grad(h_ref[L], hi["target"], grad_dtype=w.act)
    D_G = D_fwd[-1] + amax(g_ref)
    assert_close(to_f64(s.g), g_ref, D_G, tau, "G")
    allowed = tau * D_fwd[-1] * float(np.sum(np.abs(g_ref))) + 1e-12 * loss_ref
    _assert_within(np.array([s.loss.item()]), np.array([loss_ref]), allowed, "loss")
    # mask decisions of every Relu layer: in-band only
    touched = np.zeros(w.batch, dtype=bool)
    for l in range(L):
        if w.relus[l]:
            band = _band(to_f64(s.h[l]), h_ref[l], hi["weights"][l], hi["biases"][l], to_f64(s.h[l + 1]), y_ref[l],
                         _store(w))
            touched |= _flip_rows(to_f64(s.h[l + 1]), y_ref[l], band, f"layer {l + 1}")
    assert touched.sum() <= MAX_TOUCHED_ROWS * w.batch, f"{int(touched.sum())} rows touched by mask flips"
    # output (identity) layer: no mask above it, compared in full
    top = L - 1
    assert not w.relus[top]
    md = amax(g_ref)
    mh = amax(h_ref[top])
    dx_top = oracle.matmul(g_ref, hi["weights"][top], transpose_b=True, out=_store(w))
    if not fused_below(w, top, s.fuse):
        assert_close(to_f64(s.dx[top]), dx_top, w.dims[-1] * md * amax(hi["weights"][top]), tau, f"dX_{L}")
    assert_close(to_f64(s.dw[top]), oracle.matmul(h_ref[top], g_ref, transpose_a=True, out="f32"),
                 w.batch * mh * md, tau, f"dW_{L}")
    assert_close(to_f64(s.db[top]), oracle.bias_add_grad(g_ref), w.batch * md, tau, f"db_{L}")
    # Relu layers: row-local chain on sampled rows the flips did not touch
    rows = _sampled_rows(w.batch)
    rows = rows[~touched[rows]]
    g_rows = dx_top[rows]
    D_g = w.dims[-1] * md * amax(hi["weights"][top])
    for l in reversed(range(top)):
        dy_rows = oracle.relu_grad(g_rows, h_ref[l + 1][rows])
        assert_close(to_f64(s.dy[l])[rows], dy_rows, D_g, tau, f"dY_{l + 1} (sampled rows)")
        dx_rows = oracle.matmul(dy_rows, hi["weights"][l], transpose_b=True, out=_store(w))
        D_dx = w.dims[l + 1] * amax(dy_rows) * amax(hi["weights"][l])
        if not fused_below(w, l, s.fuse):
            assert_close(to_f64(s.dx[l])[rows], dx_rows, D_dx, tau, f"dX_{l + 1} (sampled rows)")
        g_rows, D_g = dx_rows, D_dx
    for l in range(L):
        if w.relus[l] and not fused_below(w, l + 1, s.fuse):
            _check_mask_consistency(s, l)
        _check_adjoint(s, l, tau)
    # every op on the GPU's own operands, on sampled rows and columns
    check_step(s, rows=sample_rows(w.batch), cols=sample_cols)
    return int(touched.sum())


@pytest.mark.parametrize("name", ["wide4096x4-f32", "wide4096x4-bf16", "wide4096x4-bf16-trunc",
                                  "tall512x32768-bf16"])
def test_full_size_step(name):
    flips = _check_full_size(name)
    print(f"{name}: {flips} rows with in-band Relu mask differences")


@pytest.mark.parametrize("batch,dims", [(256, (512, 1024)), (130, (100, 1030))])
def test_constant_weights_get_an_exact_transposed_copy(batch, dims):
    """A 16-bit weight that is never updated (the tall layer) is also kept
    transposed for the forward MatMul: the copy is W^T bit for bit."""
    w = workloads.workload("tall512x32768-bf16").scaled(batch=batch, dims=dims)
    s = DenseStep(w, workloads.generate(w, seed=9))
    torch.cuda.synchronize()
    assert s.forward_layout == "NT"
    for W, Wt in zip(s.weights, s.weights_t):
        assert torch.equal(Wt.view(torch.int16), W.t().contiguous().view(torch.int16))
