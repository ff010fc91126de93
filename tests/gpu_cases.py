"""Helpers for the GPU parity tests: run one case through the C ABI and
through the oracle on the same seeded inputs and compare bit for bit."""
import numpy as np

import oracle

LR, MU, WD = 0.01, 0.9, 5e-4


def same_bits(a, b):
    """Element-wise bit equality, any NaN equal to any NaN; returns the
    number of mismatches."""
    a = np.asarray(a, dtype=np.float32)
    b = np.asarray(b, dtype=np.float32)
    nan = np.isnan(a) & np.isnan(b)
    return int(np.count_nonzero(~nan & (a.view(np.uint32) != b.view(np.uint32))))


def alloc_len(segs, vec=8, slack=64):
    ext = oracle.extent(segs) if len(segs) else 0
    return (ext + vec - 1) // vec * vec + slack


def host_replicas(rng, K, n, dtype, scale=1.0, special=False):
    x = (rng.standard_normal((K, n), dtype=np.float32) * np.float32(scale))
    if special:
        pick = rng.random((K, n))
        x[pick < 0.01] = 0.0
        x[(pick >= 0.01) & (pick < 0.02)] = -0.0
        if dtype == np.float16:
            tiny = np.float32(2.0 ** -20)  # an fp16 subnormal
        else:
            tiny = np.float32(2.0 ** -140)  # an fp32 subnormal
        x[(pick >= 0.02) & (pick < 0.04)] *= tiny
        x[(pick >= 0.04) & (pick < 0.041)] = np.inf
        x[(pick >= 0.041) & (pick < 0.042)] = -np.inf
        x[(pick >= 0.042) & (pick < 0.043)] = np.nan
    return x.astype(dtype)


def to_dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def run_reduce(plan_mod, segs, K, dtype, order, rng, opts=None, special=False, sentinel=-3.5):
    """fc_tree_reduce vs the oracle over every element of the buffer (gaps
    must keep the sentinel)."""
    npdt = np.float16 if dtype == "f16" else np.float32
    n = alloc_len(segs)
    reps = host_replicas(rng, K, n, npdt, special=special)
    out = np.full(n, sentinel, dtype=np.float32)
    expect = oracle.tree_reduce(segs, list(reps), order=order, out=out.copy())
    plan = plan_mod.Plan(segs, K, dtype, order, **(opts or {}))
    out_d = to_dev(out)
    plan.tree_reduce(to_dev(reps), out_d)
    got = out_d.cpu().numpy()
    plan.close()
    return same_bits(got, expect), got, expect


def run_steps(plan_mod, segs, K, dtype, order, rng, steps=3, opts=None, with_out=False, with_bcast=False,
              special=False, batch=256, after_step=None):
    """`steps` chained fc_step calls (new replicas each step) vs the oracle;
    returns the total number of mismatching elements over w, v, out, bcast.
    after_step(plan), when given, runs after every step."""
    import torch
    npdt = np.float16 if dtype == "f16" else np.float32
    n = alloc_len(segs)
    w = (rng.standard_normal(n, dtype=np.float32) * np.float32(0.05))
    v = np.zeros(n, dtype=np.float32)
    plan = plan_mod.Plan(segs, K, dtype, order, **(opts or {}))
    w_d, v_d = to_dev(w), to_dev(v)
    out_d = torch.full((n,), -1.0, device="cuda") if with_out else None
    dst_d = torch.full((K, n), -2.0, device="cuda") if with_bcast else None
    out_h = np.full(n, -1.0, np.float32) if with_out else None
    dst_h = [np.full(n, -2.0, np.float32) for _ in range(K)] if with_bcast else None
    bad = 0
    for _ in range(steps):
        reps = host_replicas(rng, K, n, npdt, scale=0.01, special=special)
        w, v, _, _ = oracle.step(segs, list(reps), w, v, LR, MU, WD, batch, order=order, out=out_h, bcast=dst_h)
        plan.step(to_dev(reps), w_d, v_d, LR, MU, WD, batch, out=out_d, bcast=dst_d)
        torch.cuda.synchronize()
        bad += same_bits(w_d.cpu().numpy(), w) + same_bits(v_d.cpu().numpy(), v)
        if with_out:
            bad += same_bits(out_d.cpu().numpy(), out_h)
        if with_bcast:
            got = dst_d.cpu().numpy()
            bad += sum(same_bits(got[k], dst_h[k]) for k in range(K))
        if after_step is not None:
            after_step(plan)
    plan.close()
    return bad
