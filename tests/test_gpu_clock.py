"""tfd_clock_probe: shader clock cycles over real-time ticks of one wave give
a clock within the chip's range, and the probe's FMA chain ran in full."""

import numpy as np
import pytest
import torch

from paper_1603_04467_amd import tfdense as T

pytestmark = pytest.mark.gpu


def test_clock_probe_counts_and_chain():
    n = 20000
    c = torch.zeros(3, dtype=torch.int64, device="cuda")
    T.tfd_clock_probe(c, n)
    torch.cuda.synchronize()
    cycles, ticks, bits = (int(v) for v in c.cpu())
    assert cycles > n and ticks > 0
    mhz = 100.0 * cycles / ticks
    assert 100.0 <= mhz <= 3000.0, mhz
    # lane 2's chain x <- fma(x, a, b) from x = 2, replayed on the host (the
    # float64 product of two floats is exact; its sum with b is rounded twice,
    # which can move a step by one ulp, and the map contracts such offsets)
    a, b = np.float32(0.999999), np.float32(1e-7)
    want = np.float32(2.0)
    for _ in range(n):
        want = np.float32(float(want) * float(a) + float(b))
    x = np.array([bits], dtype=np.uint32).view(np.float32)[0]
    assert abs(float(x) - float(want)) <= 4 * float(np.spacing(want)), (float(x), float(want))
