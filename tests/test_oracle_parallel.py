"""oracle.step_parallel (the oracle's step run on several host threads, one
contiguous range of elements each) gives the bits of oracle.step for every
cut of the element range, both orders and storage types, with the raw sum
and the broadcast; used for the full-size parity checks."""
import numpy as np
import pytest

import oracle
from workloads import gen


@pytest.mark.parametrize("dtype", [np.float32, np.float16])
@pytest.mark.parametrize("order", ["tree", "linear"])
@pytest.mark.parametrize("threads", [1, 2, 3, 7, 16])
def test_parallel_step_equals_step(dtype, order, threads):
    rng = np.random.default_rng(threads * 10 + (dtype == np.float16) + (order == "tree") * 2)
    rows, n = gen.random_table(rng, 11, 3000, 4, gap_max=5)
    rows = [(o, m, float(rng.choice([1.0, 2.0])), float(rng.choice([1.0, 0.0]))) for o, m, _, _ in rows]
    K = 13
    reps = (rng.standard_normal((K, n + 64), dtype=np.float32) * 0.01).astype(dtype)
    w = rng.standard_normal(n + 64, dtype=np.float32)
    v = rng.standard_normal(n + 64, dtype=np.float32) * np.float32(1e-3)
    out_a, out_b = np.full(n + 64, -1.0, np.float32), np.full(n + 64, -1.0, np.float32)
    dst_a = [np.full(n + 64, -2.0, np.float32) for _ in range(K)]
    dst_b = [np.full(n + 64, -2.0, np.float32) for _ in range(K)]
    wa, va, _, _ = oracle.step(rows, list(reps), w, v, 0.01, 0.9, 5e-4, 256, order=order, out=out_a, bcast=dst_a)
    wb, vb, _, _ = oracle.step_parallel(rows, reps, w, v, 0.01, 0.9, 5e-4, 256, order=order, out=out_b,
                                        bcast=dst_b, threads=threads)
    for a, b in [(wa, wb), (va, vb), (out_a, out_b)] + list(zip(dst_a, dst_b)):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
