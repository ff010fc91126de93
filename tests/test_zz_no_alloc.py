"""fc_step_noalloc (the step with its raw sum in the library's fixed device
array) against fc_step on the same plan and inputs, bit for bit, through the
C ABI: two calls in a row, the second on a smaller plan, so that the array
still holds the first call's sums when the second runs.  Also the size limit
(FC_ESIZE, refused before anything is enqueued), an `out` buffer (the array
unused), the broadcast, fp16 replicas, the linear order and a resident plan
whose tiles the reduce pass reads in batches of 8."""
import numpy as np
import pytest

import oracle
from gpu_cases import LR, MU, WD, alloc_len, host_replicas, same_bits, to_dev
from workloads import gen

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def fc(device):
    import paper_1511_00175_amd as m
    return m


def rows_of(t):
    base, step = t.data_ptr(), t.stride(0) * t.element_size()
    return [base + k * step for k in range(t.shape[0])]


def run_both(fc, segs, K, dtype, order, rng, opts=None, with_out=False, with_bcast=False, batch=256):
    """One fc_step_noalloc and one fc_step on clones of the same w, v (same
    plan, same replicas); returns the mismatches between the two over w, v
    (and out, bcast) and between fc_step_noalloc and the oracle."""
    import torch
    f = fc._fc
    npdt = np.float16 if dtype == "f16" else np.float32
    n = alloc_len(segs)
    reps_h = host_replicas(rng, K, n, npdt, scale=0.01)
    w_h = rng.standard_normal(n, dtype=np.float32) * np.float32(0.05)
    v_h = rng.standard_normal(n, dtype=np.float32) * np.float32(1e-3)
    reps = to_dev(reps_h)
    w1, v1 = to_dev(w_h), to_dev(v_h)
    w2, v2 = w1.clone(), v1.clone()
    out1 = torch.full((n,), -1.0, device="cuda") if with_out else None
    out2 = torch.full((n,), -1.0, device="cuda") if with_out else None
    d1 = torch.full((K, n), -2.0, device="cuda") if with_bcast else None
    d2 = torch.full((K, n), -2.0, device="cuda") if with_bcast else None
    plan = fc.Plan(segs, K, dtype, order, **(opts or {}))
    s = torch.cuda.current_stream().cuda_stream
    rc = f.fc_step_noalloc(plan.handle, rows_of(reps), w1.data_ptr(), v1.data_ptr(), LR, MU, WD, batch,
                           None if out1 is None else out1.data_ptr(), None if d1 is None else rows_of(d1), s)
    assert rc == f.FC_OK, f.fc_strerror(rc)
    rc = f.fc_step(plan.handle, rows_of(reps), w2.data_ptr(), v2.data_ptr(), LR, MU, WD, batch,
                   None if out2 is None else out2.data_ptr(), None if d2 is None else rows_of(d2), s)
    assert rc == f.FC_OK
    torch.cuda.synchronize()
    plan.close()
    pairs = [(w1, w2), (v1, v2)] + ([(out1, out2)] if with_out else []) + ([(d1, d2)] if with_bcast else [])
    vs_step = sum(same_bits(a.cpu().numpy().ravel(), b.cpu().numpy().ravel()) for a, b in pairs)
    out_h = np.full(n, -1.0, np.float32) if with_out else None
    dst_h = [np.full(n, -2.0, np.float32) for _ in range(K)] if with_bcast else None
    ew, ev, _, _ = oracle.step(segs, list(reps_h), w_h, v_h, LR, MU, WD, batch, order=order, out=out_h,
                               bcast=dst_h)
    vs_oracle = same_bits(w1.cpu().numpy(), ew) + same_bits(v1.cpu().numpy(), ev)
    if with_out:
        vs_oracle += same_bits(out1.cpu().numpy(), out_h)
    if with_bcast:
        got = d1.cpu().numpy()
        vs_oracle += sum(same_bits(got[k], dst_h[k]) for k in range(K))
    return vs_step, vs_oracle


def big_table(rng, n_total, dtype):
    rows, ext = gen.random_table(rng, 9, n_total // 9, 4, gap_max=3, min_len=n_total // 12)
    return rows


@pytest.mark.parametrize("dtype,order,K,opts", [
    ("f32", "tree", 70, None),              # a two-pass plan: fc_step uses the plan's own scratch
    ("f32", "tree", 9, None),               # a fused plan (no scratch of its own)
    ("f16", "linear", 33, None),
    ("f32", "tree", 16, dict(schedule=3)),  # resident tiles of 2 vectors, batches of 4
    ("f32", "tree", 130, dict(schedule=3)),
])
def test_noalloc_equals_step_twice(fc, dtype, order, K, opts):
    """Two calls in a row, the second on a plan a quarter the size: both
    equal fc_step and the oracle bit for bit."""
    rng = np.random.default_rng(K)
    first = big_table(rng, 1_200_000, dtype)
    second = big_table(rng, 300_000, dtype)
    for segs in (first, second):
        vs_step, vs_oracle = run_both(fc, segs, K, dtype, order, rng, opts=opts)
        assert vs_step == 0 and vs_oracle == 0, (len(segs), vs_step, vs_oracle)


@pytest.mark.parametrize("with_out,with_bcast", [(True, False), (False, True), (True, True)])
def test_noalloc_with_sum_and_broadcast(fc, with_out, with_bcast):
    rng = np.random.default_rng(3)
    for segs, K in ((big_table(rng, 400_000, "f32"), 12), (big_table(rng, 100_000, "f32"), 5)):
        vs_step, vs_oracle = run_both(fc, segs, K, "f32", "tree", rng, with_out=with_out, with_bcast=with_bcast)
        assert vs_step == 0 and vs_oracle == 0, (K, vs_step, vs_oracle)


def test_noalloc_size_limit(fc):
    """A plan whose extent exceeds the array is refused before anything is
    enqueued (FC_ESIZE) -- unless `out` takes the raw sum; the limit itself
    is allowed."""
    import torch
    f = fc._fc
    lim = f.FC_NOALLOC_MAX_ELEMS
    K = 2
    s = torch.cuda.current_stream().cuda_stream
    reps = torch.zeros((K, lim + 64), device="cuda")
    w = torch.ones(lim + 64, device="cuda")
    v = torch.zeros(lim + 64, device="cuda")
    out = torch.zeros(lim + 64, device="cuda")
    over = fc.Plan([(0, lim + 4, 1.0, 1.0)], K, "f32", "tree")
    w0 = w.clone()
    rc = f.fc_step_noalloc(over.handle, rows_of(reps), w.data_ptr(), v.data_ptr(), 1.0, 0.0, 0.0, 1, None, None, s)
    assert rc == f.FC_ESIZE and "fixed" in f.fc_strerror(rc)
    torch.cuda.synchronize()
    assert torch.equal(w, w0)
    rc = f.fc_step_noalloc(over.handle, rows_of(reps), w.data_ptr(), v.data_ptr(), 1.0, 0.0, 0.0, 1,
                           out.data_ptr(), None, s)
    assert rc == f.FC_OK
    torch.cuda.synchronize()
    over.close()
    at = fc.Plan([(0, lim, 1.0, 1.0)], K, "f32", "tree")
    reps[:, :lim] = 1.0
    rc = f.fc_step_noalloc(at.handle, rows_of(reps), w.data_ptr(), v.data_ptr(), 1.0, 0.0, 0.0, 1, None, None, s)
    assert rc == f.FC_OK
    torch.cuda.synchronize()
    at.close()
    # the call with `out` summed zeros (w stays 1); this one sums two ones on
    # [0, lim): w' = 1 - 1 * 2, and w keeps 1 beyond the plan
    assert bool((w[:lim] == -1.0).all()) and bool((w[lim:lim + 4] == 1.0).all())
    del reps, w, v, out
    torch.cuda.empty_cache()
