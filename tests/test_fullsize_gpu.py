"""Parity at the full workload sizes, in the launch configuration bench.py
times (the plan defaults, resident shares rebalanced per XCD after the first
step as bench.py does after its warm-up), on sampled outputs the oracle
computes one by one.

For each of the five workloads (flat 2^20 x K=4, NiN x K=32, GoogLeNet
x K=128, VGG-19 x K=16, AlexNet fp16 x K=128), and Table 1's variants
(GoogLeNet with its auxiliary classifiers, ungrouped AlexNet), the inputs are drawn on the
device, three fused steps run on the GPU (fc_plan_balance after the first),
and at every segment's first, second, last and one random element plus 1500
random elements the oracle recomputes the same three steps from the gathered
inputs; w' and v' must match bit for bit.
Properties that hold at any size are checked on the whole buffer: the fused
step equals reduce, then SGD (GoogLeNet), and the broadcast copies and raw
sum fused into the step equal w' and the reduce's sum (GoogLeNet, VGG-19).
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


def sample_indices(wl, rng, n_random=1500):
    """Each segment's first, second, last and one random element, plus
    n_random elements drawn with probability proportional to segment length."""
    idx = []
    for s in wl.segments:
        idx += [s.offset, s.offset + min(1, s.length - 1), s.offset + s.length - 1,
                s.offset + int(rng.integers(0, s.length))]
    lens = np.array([s.length for s in wl.segments], dtype=np.float64)
    js = rng.choice(len(wl.segments), n_random, p=lens / lens.sum())
    idx += [wl.segments[j].offset + int(rng.integers(0, wl.segments[j].length)) for j in js]
    return np.unique(np.array(idx, dtype=np.int64))


def segment_of(wl, idx):
    offs = np.array([s.offset for s in wl.segments])
    return np.searchsorted(offs, idx, side="right") - 1


@pytest.mark.parametrize("name", ["flat", "nin", "googlenet", "vgg19", "alexnet", "googlenet_aux",
                                  "alexnet_ungrouped"])
def test_fullsize_sampled(fc, name):
    import torch
    wl = tables.get(name)
    dev = torch.device("cuda:0")
    rng = np.random.default_rng(len(name))
    reps, w, v = gen.device_inputs(wl, 1511, dev)
    idx = sample_indices(wl, rng)
    it = torch.from_numpy(idx).to(dev)
    g_s = reps[:, it].cpu().numpy()                 # (K, S) gathered replica values
    w_s, v_s = w[it].cpu().numpy(), v[it].cpu().numpy()
    plan = fc.Plan(wl.table(), wl.K, wl.dtype, "tree")
    for i in range(3):
        plan.step(reps, w, v, wl.lr, wl.mu, wl.wd, wl.batch)
        if i == 0:
            plan.balance()
    torch.cuda.synchronize()
    got_w, got_v = w[it].cpu().numpy(), v[it].cpu().numpy()
    plan.close()
    del reps, w, v
    torch.cuda.empty_cache()
    # oracle on the gathered samples: each sample is a one-element segment
    # carrying its own segment's multipliers
    js = segment_of(wl, idx)
    rows = [(i, 1, wl.segments[j].lr_mult, wl.segments[j].decay_mult) for i, j in enumerate(js)]
    ew, ev = w_s, v_s
    for _ in range(3):
        ew, ev, _, _ = oracle.step(rows, list(g_s), ew, ev, wl.lr, wl.mu, wl.wd, wl.batch)
    assert same_bits(got_w, ew) == 0 and same_bits(got_v, ev) == 0


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


@pytest.mark.parametrize("name", ["googlenet", "vgg19"])
def test_fullsize_broadcast(fc, name):
    """The raw sum and the broadcast of w' fused into the step at full size
    (GoogLeNet: K = 128 copies, one resident round; VGG-19: K = 16 copies,
    14 rounds), shares rebalanced per XCD after it: every worker copy equals
    w' bit for bit on every parameter and keeps its fill value on the
    padding, the raw sum equals fc_tree_reduce's, and w', v' equal those of
    a step without either (properties that hold at any size)."""
    import torch
    wl = tables.get(name)
    dev = torch.device("cuda:0")
    reps, w, v = gen.device_inputs(wl, 5, dev)
    w2, v2 = w.clone(), v.clone()
    n = w.numel()
    mask = torch.zeros(n, dtype=torch.bool, device=dev)
    for s in wl.segments:
        mask[s.offset:s.offset + s.length] = True
    dst = torch.full((wl.K, n), -2.0, device=dev)
    out = torch.full((n,), -1.0, device=dev)
    g = torch.full((n,), -1.0, device=dev)
    plan = fc.Plan(wl.table(), wl.K, wl.dtype, "tree")
    plan.step(reps, w, v, wl.lr, wl.mu, wl.wd, wl.batch, out=out, bcast=dst)
    plan.balance()
    plan.step(reps, w2, v2, wl.lr, wl.mu, wl.wd, wl.batch)
    plan.tree_reduce(reps, g)
    torch.cuda.synchronize()
    plan.close()
    assert torch.equal(w.view(torch.int32), w2.view(torch.int32))
    assert torch.equal(v.view(torch.int32), v2.view(torch.int32))
    assert torch.equal(out.view(torch.int32), g.view(torch.int32))
    wm = w[mask].view(torch.int32)
    for k in range(wl.K):
        assert torch.equal(dst[k][mask].view(torch.int32), wm), k
        assert bool((dst[k][~mask] == -2.0).all()), k
    del reps, w, v, w2, v2, dst, out, g
    torch.cuda.empty_cache()


@pytest.mark.parametrize("dtype,schedule", [("f16", 1), ("f16", 3), ("f32", 2), ("f32", 3)])
def test_offsets_beyond_4gib(fc, dtype, schedule):
    """A segment of 2^31 + 100 elements: element indices pass 2^31 and byte
    offsets pass 4 GiB (8 GiB of fp32) in every buffer, the tile map holds
    8.4 M tiles and the resident schedule takes about 200 rounds, rebalanced
    per XCD between the two steps.  Windows at the start, around element 2^31
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
    if schedule == 3:
        assert plan.info().rounds > 100
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
