"""Parity at the full workload sizes on every element, in the launch
configuration bench.py times (the plan defaults, resident shares rebalanced
per XCD after the first step as bench.py does after its warm-up).

For each workload -- flat 2^20 x K=4, NiN x K=32, GoogLeNet x K=128, VGG-19
x K=16, AlexNet fp16 x K=128 in tree and in parameter-server order, and Table
1's variants (GoogLeNet with its auxiliary classifiers, GoogLeNet with
Caffe's bias multipliers, ungrouped AlexNet) -- the inputs are drawn on the
device and copied to the host, three steps run on the GPU (fc_plan_balance
after the first), and the oracle runs the same three steps on the host copies
on every host thread (oracle.step_parallel: one range of elements per thread,
the same scalar arithmetic for every element).  Every element of w' and v',
the padding between segments included (which neither side may write), must
match bit for bit.  GoogLeNet (K = 128 copies, one resident round) and
VGG-19 (K = 16 copies, 8 rounds) also run steps that keep the raw sum and
broadcast w' into the K worker copies: every element of those too.
"""
import numpy as np
import pytest

import oracle
from gpu_cases import same_bits
from workloads import gen, tables

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def fc(device):
    import paper_1511_00175_amd as m
    return m


@pytest.fixture(scope="module", autouse=True)
def release_device_memory():
    """The full-size inputs take tens of GB: the cached device memory goes back
    to the driver when this module ends, not when the test process exits."""
    yield
    import gc
    import torch
    gc.collect()
    if torch.cuda.is_available():
        torch.cuda.empty_cache()


def host(t):
    return t.cpu().numpy()


@pytest.mark.parametrize("name,order", [
    ("flat", "tree"), ("nin", "tree"), ("googlenet", "tree"), ("vgg19", "tree"), ("alexnet", "tree"),
    ("alexnet", "linear"), ("googlenet_aux", "tree"), ("googlenet_caffe_bias", "tree"),
    ("alexnet_ungrouped", "tree")])
def test_fullsize_every_element(fc, name, order):
    import torch
    wl = tables.get(name)
    dev = torch.device("cuda:0")
    reps, w, v = gen.device_inputs(wl, 1511, dev)
    reps_h, w_h, v_h = host(reps), host(w), host(v)
    plan = fc.Plan(wl.table(), wl.K, wl.dtype, order)
    for i in range(3):
        plan.step(reps, w, v, wl.lr, wl.mu, wl.wd, wl.batch)
        if i == 0:
            plan.balance()
    torch.cuda.synchronize()
    plan.close()
    got_w, got_v = host(w), host(v)
    del reps, w, v
    torch.cuda.empty_cache()
    ew, ev = w_h, v_h
    for _ in range(3):
        ew, ev, _, _ = oracle.step_parallel(wl.table(), reps_h, ew, ev, wl.lr, wl.mu, wl.wd, wl.batch, order=order)
    assert same_bits(got_w, ew) == 0 and same_bits(got_v, ev) == 0


@pytest.mark.parametrize("name", ["googlenet", "vgg19"])
def test_fullsize_sum_and_broadcast(fc, name):
    """Two steps that also keep the raw sum and broadcast w' to the K worker
    copies, shares rebalanced per XCD between them: w', v', the raw sum and
    every copy against the oracle on every element (outside the segments the
    copies and the sum keep their fill values)."""
    import torch
    wl = tables.get(name)
    dev = torch.device("cuda:0")
    reps, w, v = gen.device_inputs(wl, 5, dev)
    reps_h, w_h, v_h = host(reps), host(w), host(v)
    n = w.numel()
    dst = torch.full((wl.K, n), -2.0, device=dev)
    out = torch.full((n,), -1.0, device=dev)
    plan = fc.Plan(wl.table(), wl.K, wl.dtype, "tree")
    plan.step(reps, w, v, wl.lr, wl.mu, wl.wd, wl.batch, out=out, bcast=dst)
    plan.balance()
    plan.step(reps, w, v, wl.lr, wl.mu, wl.wd, wl.batch, out=out, bcast=dst)
    torch.cuda.synchronize()
    plan.close()
    out_h = np.full(n, -1.0, np.float32)
    dst_h = [np.full(n, -2.0, np.float32) for _ in range(wl.K)]
    ew, ev = w_h, v_h
    for _ in range(2):
        ew, ev, _, _ = oracle.step_parallel(wl.table(), reps_h, ew, ev, wl.lr, wl.mu, wl.wd, wl.batch,
                                            out=out_h, bcast=dst_h)
    assert same_bits(host(w), ew) == 0 and same_bits(host(v), ev) == 0
    assert same_bits(host(out), out_h) == 0
    for k in range(wl.K):
        assert same_bits(host(dst[k]), dst_h[k]) == 0, k
    del reps, w, v, dst, out
    torch.cuda.empty_cache()


def test_fullsize_fused_equals_composed(fc):
    """At full GoogLeNet size: one fused step == tree reduce, then SGD, on the
    whole buffer (a property independent of the oracle), with the resident
    shares rebalanced per XCD between the fused step and the other two."""
    import torch
    wl = tables.googlenet()
    dev = torch.device("cuda:0")
    reps, w, v = gen.device_inputs(wl, 7, dev)
    v.normal_(0, 1e-3, generator=torch.Generator(device=dev).manual_seed(8))
    w2, v2 = w.clone(), v.clone()
    g = torch.zeros_like(w)
    plan = fc.Plan(wl.table(), wl.K, wl.dtype, "tree")
    plan.step(reps, w, v, wl.lr, wl.mu, wl.wd, wl.batch)
    assert sum(1 for r in plan.balance() if r > 0) == 8
    plan.tree_reduce(reps, g)
    plan.sgd_step(w2, v2, g, wl.lr, wl.mu, wl.wd, wl.batch)
    torch.cuda.synchronize()
    assert torch.equal(w.view(torch.int32), w2.view(torch.int32))
    assert torch.equal(v.view(torch.int32), v2.view(torch.int32))
    plan.close()


@pytest.mark.parametrize("dtype,schedule", [("f16", 1), ("f16", 3), ("f32", 2), ("f32", 3), ("f32", 4)])
def test_offsets_beyond_4gib(fc, dtype, schedule):
    """A segment of 2^31 + 100 elements: element indices pass 2^31 and byte
    offsets pass 4 GiB (8 GiB of fp32) in every buffer, the tile map holds
    8.4 M tiles and the resident schedule takes 100-200 rounds (one launch
    each, or all of them in one launch), rebalanced per XCD between the two
    steps.  Windows at the start, around element 2^31
    and at the end are recomputed by the oracle from the gathered inputs
    (elements are independent within a segment)."""
    import torch
    dev = torch.device("cuda:0")
    big = (1 << 31) + 100
    rows = [(0, 1000, 1.0, 1.0), (1024, big, 2.0, 0.5)]
    n = 1024 + big + 28
    K = 2
    g = torch.Generator(device=dev)
    g.manual_seed(31)
    tdt = torch.float16 if dtype == "f16" else torch.float32
    reps = torch.empty((K, n), dtype=tdt, device=dev)
    for k in range(K):
        reps[k] = (torch.randn(n, generator=g, device=dev) * 1e-3).to(tdt)
    w = torch.randn(n, generator=g, device=dev) * 0.01
    v = torch.randn(n, generator=g, device=dev) * 1e-4
    # windows inside one segment each: element 2^31 sits at byte 4 GiB of an
    # fp16 replica and at byte 8 GiB of an fp32 replica, w and v
    wins = [(0, 1000), (1024, 1024 + 512), ((1 << 31) - 256, (1 << 31) + 256), (1024 + big - 512, 1024 + big)]
    before = [(reps[:, a:b].cpu().numpy(), w[a:b].cpu().numpy(), v[a:b].cpu().numpy()) for a, b in wins]
    plan = fc.Plan(rows, K, dtype, "tree", schedule=schedule)
    if schedule in (3, 4):
        assert plan.info().rounds > 50 and plan.info().schedule == schedule
    plan.step(reps, w, v, 0.01, 0.9, 5e-4, 256)
    plan.balance()
    plan.step(reps, w, v, 0.01, 0.9, 5e-4, 256)
    torch.cuda.synchronize()
    plan.close()
    for (a, b), (r_h, w_h, v_h) in zip(wins, before):
        seg = [r for r in rows if r[0] <= a < r[0] + r[1]][0]
        ew, ev = w_h, v_h
        for _ in range(2):
            ew, ev, _, _ = oracle.step([(0, b - a, seg[2], seg[3])], list(r_h), ew, ev, 0.01, 0.9, 5e-4, 256)
        assert same_bits(w[a:b].cpu().numpy(), ew) == 0, (a, b)
        assert same_bits(v[a:b].cpu().numpy(), ev) == 0, (a, b)
    del reps, w, v
    torch.cuda.empty_cache()
