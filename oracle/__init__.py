"""CPU oracle for the dense-layer training step (test infrastructure only).

This package is the slow, obviously correct reference that the HIP path is
checked against. It is test infrastructure: only ``tests/``, the smoke check in
``__graft_entry__`` and the ``cpu_baseline`` leg of ``bench.py`` may import it.
The product path never calls it, and it imports nothing from the product
package (the two share no code; the seeded input generator hands both sides
the same arrays).

Every function works on float64 numpy arrays. The 32 <-> 16-bit converter
of section 5.5 lives in ``oracle.convert`` (a C loop compiled with gcc on
first use). Sums and dot products are
carried out in float64 from the stored values (bf16 and fp32 values upcast
exactly) and rounded once, round-to-nearest-even, to the storage type at the
points where a tensor is stored. Storage types are named ``"f64"`` (no
rounding; used by the finite-difference pins), ``"f32"``, ``"bf16"`` and
``"bf16t"`` (fp32 first, then the truncating converter).

Pins (see ``tests/test_oracle_*.py``): brute-force triple loops, identity and
permutation matrices, exact small-integer sums, finite differences of the
loss, exact rational rounding of the SGD update, the bit formula of the bf16
cast, the adjoint/homogeneity identities of a Relu layer and the
data-parallel gradient-sum identity. Parity unpinned: which way a Relu mask
falls for pre-activations inside the rounding band of zero (several answers
are correct there).
"""

from .dense import (  # noqa: F401
    STORAGE_TYPES,
    round_to,
    round_bf16,
    bf16_bits_to_f64,
    f64_to_bf16_bits,
    matmul,
    bias_add,
    relu,
    relu_grad,
    relu_mask,
    relu_grad_from_mask,
    bias_add_grad,
    l2_loss_grad,
    softmax,
    softmax_cross_entropy_grad,
    apply_gradient_descent,
    dense_step,
)
