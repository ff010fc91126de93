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


@pytest.mark.parametrize("seed", range(1000, 1064))
def test_random_composed_step_matches_oracle(fc, seed):
    """The step composed from the boundary's separate calls -- fc_tree_reduce,
    then fc_sgd_step from that raw sum, then fc_broadcast of w' -- on the
    same random configurations: w', v' and every copy equal the oracle's
    fused step."""
    import torch
    import oracle
    from gpu_cases import LR, MU, WD, host_replicas, same_bits, to_dev
    rows, K, dtype, order, opts, _, _, special = draw(seed)
    K = min(K, 64)  # K broadcast copies
    print(f"case {seed}: K={K} {dtype} {order} {opts} nseg={len(rows)}", flush=True)
    rng = np.random.default_rng(20_000 + seed)
    n = alloc_len(rows)
    npdt = np.float16 if dtype == "f16" else np.float32
    reps = host_replicas(rng, K, n, npdt, scale=0.01, special=special)
    w = rng.standard_normal(n, dtype=np.float32) * np.float32(0.05)
    v = rng.standard_normal(n, dtype=np.float32) * np.float32(0.001)
    dst_h = [np.full(n, -2.0, np.float32) for _ in range(K)]
    ew, ev, _, _ = oracle.step(rows, list(reps), w.copy(), v.copy(), LR, MU, WD, 256, order=order, bcast=dst_h)
    plan = fc.Plan(rows, K, dtype, order, **opts)
    w_d, v_d, g_d = to_dev(w), to_dev(v), torch.zeros(n, device="cuda")
    dst_d = torch.full((K, n), -2.0, device="cuda")
    plan.tree_reduce(to_dev(reps), g_d)
    plan.sgd_step(w_d, v_d, g_d, LR, MU, WD, 256)
    plan.broadcast(w_d, dst_d)
    torch.cuda.synchronize()
    plan.close()
    assert same_bits(w_d.cpu().numpy(), ew) == 0
    assert same_bits(v_d.cpu().numpy(), ev) == 0
    got = dst_d.cpu().numpy()
    assert sum(same_bits(got[k], dst_h[k]) for k in range(K)) == 0


@pytest.mark.parametrize("seed", range(2000, 2032))
def test_random_step_noalloc_matches_oracle(fc, seed):
    """fc_step_noalloc (the step in two passes with the raw sum in the
    library's fixed device array) on seeded random configurations, two
    chained steps of shrinking size: w', v' and the optional outputs equal
    the oracle's."""
    import torch
    import oracle
    from gpu_cases import LR, MU, WD, host_replicas, same_bits, to_dev
    rows, K, dtype, order, opts, with_out, with_bcast, special = draw(seed)
    print(f"case {seed}: K={K} {dtype} {order} {opts} nseg={len(rows)} out={with_out} bcast={with_bcast}",
          flush=True)
    rng = np.random.default_rng(30_000 + seed)
    npdt = np.float16 if dtype == "f16" else np.float32
    for table in (rows, rows[:max(1, len(rows) // 2)]):
        n = alloc_len(table)
        reps = host_replicas(rng, K, n, npdt, scale=0.01, special=special)
        w = rng.standard_normal(n, dtype=np.float32) * np.float32(0.05)
        v = np.zeros(n, np.float32)
        out_h = np.full(n, -1.0, np.float32) if with_out else None
        dst_h = [np.full(n, -2.0, np.float32) for _ in range(K)] if with_bcast else None
        ew, ev, _, _ = oracle.step(table, list(reps), w, v, LR, MU, WD, 256, order=order, out=out_h, bcast=dst_h)
        plan = fc.Plan(table, K, dtype, order, **opts)
        w_d, v_d = to_dev(w), to_dev(v)
        out_d = torch.full((n,), -1.0, device="cuda") if with_out else None
        dst_d = torch.full((K, n), -2.0, device="cuda") if with_bcast else None
        plan.step_noalloc(to_dev(reps), w_d, v_d, LR, MU, WD, 256, out=out_d, bcast=dst_d)
        torch.cuda.synchronize()
        plan.close()
        assert same_bits(w_d.cpu().numpy(), ew) == 0 and same_bits(v_d.cpu().numpy(), ev) == 0
        if with_out:
            assert same_bits(out_d.cpu().numpy(), out_h) == 0
        if with_bcast:
            got = dst_d.cpu().numpy()
            assert sum(same_bits(got[k], dst_h[k]) for k in range(K)) == 0
