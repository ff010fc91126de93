"""Seeded random configurations through the C ABI, each compared bit for bit
with the oracle: worker count, replica type, summation order, schedule,
launch shape, grid cap (and so the number of resident rounds), segment table
(count, lengths, gaps, per-segment multipliers), special values, and which
optional outputs the step writes are all drawn from one seed per case, so a
failure names a case that can be rerun on its own."""
import numpy as np
import pytest

from gpu_cases import alloc_len, run_reduce, run_steps
from workloads import gen

pytestmark = pytest.mark.gpu

# (block_threads, vecs_per_thread, kchunk) the fused and two-pass kernels are compiled for
FUSED_SHAPES = [(64, 1, 16), (64, 1, 8), (128, 2, 16), (256, 2, 8), (256, 4, 8), (256, 4, 4), (128, 4, 2)]


@pytest.fixture(scope="module")
def fc(device):
    import paper_1511_00175_amd as m
    return m


def draw(seed):
    """One configuration: (segments, K, dtype, order, opts, with_out, with_bcast, special)."""
    rng = np.random.default_rng(seed)
    K = int(rng.choice([1, 2, 3, 4, 5, 7, 8, 13, 16, 24, 31, 33, 64, 100, 128, 257, 300]))
    dtype = str(rng.choice(["f32", "f16"]))
    order = str(rng.choice(["tree", "linear"]))
    nseg = int(rng.integers(1, 13))
    max_len = int(rng.choice([40, 700, 5000, 30000]))
    rows, _ = gen.random_table(rng, nseg, max_len, 4, gap_max=20)
    # per-segment multipliers, as Caffe's bias convention (2, 0) and others
    rows = [(o, n, float(rng.choice([1.0, 2.0, 0.5])), float(rng.choice([1.0, 0.0, 3.0]))) for o, n, _, _ in rows]
    schedule = int(rng.integers(0, 5))
    opts = {"schedule": schedule}
    if schedule in (1, 2) and rng.random() < 0.7:
        b, u, c = FUSED_SHAPES[int(rng.integers(len(FUSED_SHAPES)))]
        opts.update(block_threads=b, vecs_per_thread=u, kchunk=c)
    if schedule in (3, 4) and K // 4 < 128 and rng.random() < 0.5:
        opts["vecs_per_thread"] = 2
    opts["max_blocks"] = int(rng.choice([0, 0, 1, 2, 5, 37]))
    with_out = bool(rng.random() < 0.5)
    with_bcast = bool(K <= 64 and rng.random() < 0.4)
    special = bool(rng.random() < 0.3)
    return rows, K, dtype, order, opts, with_out, with_bcast, special


@pytest.mark.parametrize("seed", range(160))
def test_random_configuration_matches_oracle(fc, seed):
    rows, K, dtype, order, opts, with_out, with_bcast, special = draw(seed)
    case = dict(K=K, dtype=dtype, order=order, opts=opts, nseg=len(rows), n=alloc_len(rows), out=with_out,
                bcast=with_bcast, special=special)
    print(f"case {seed}: {case}", flush=True)
    rng = np.random.default_rng(10_000 + seed)
    bad, _, _ = run_reduce(fc, rows, K, dtype, order, rng, opts=opts, special=special)
    assert bad == 0, case
    assert run_steps(fc, rows, K, dtype, order, rng, steps=2, opts=opts, with_out=with_out, with_bcast=with_bcast,
                     special=special) == 0, case
