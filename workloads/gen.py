"""Seeded synthetic inputs for the gradient-aggregation workloads.

Draws the K workers' gradient replicas, the weights and the velocity for a
segment table; holds none of the method's arithmetic (no sums, no update).
Both the oracle-side tests and the GPU path take their inputs from here.

Value recipe per segment (weight or bias block of one layer):
  gradients  N(0, sigma): sigma = 1e-3/sqrt(fan_in) ("fan_in"), or a fixed
             number; fp16 replicas are the fp32 draw rounded to nearest even
  weights    "gauss0.01"     : N(0, 0.01), bias 0
             "nin"           : N(0, 0.01) for 1x1 filters, N(0, 0.05) otherwise,
                               bias 0 (Sec. 7.1 item 2)
             "xavier_bias0.2": U(-sqrt(3/fan_in), +sqrt(3/fan_in)), bias 0.2
                               (Sec. 7.1 item 2)
  velocity   zero
Padding between segments is zero in every buffer.

Layout: replicas are one slab of shape (K, stride); replica k starts at
element k*stride.  stride = padded length + `stagger` elements, so that the K
replica bases do not all share one power-of-two alignment.
"""
import math

import numpy as np

from .tables import ALIGN


def grad_sigma(wl, seg):
    if wl.grad_std == "fan_in":
        return 1e-3 / math.sqrt(seg.fan_in)
    return float(wl.grad_std)


def weight_recipe(wl, seg):
    """('normal', std) | ('uniform', half_width) | ('const', value)."""
    if wl.weight_init == "gauss0.01":
        return ("const", 0.0) if seg.is_bias else ("normal", 0.01)
    if wl.weight_init == "nin":
        if seg.is_bias:
            return ("const", 0.0)
        one_by_one = seg.layer.kh == 1 and seg.layer.kw == 1
        return ("normal", 0.01 if one_by_one else 0.05)
    if wl.weight_init == "xavier_bias0.2":
        return ("const", 0.2) if seg.is_bias else ("uniform", math.sqrt(3.0 / seg.fan_in))
    raise ValueError(wl.weight_init)


def default_stride(wl, stagger=ALIGN):
    return wl.padded + stagger


# ---------------------------------------------------------------- host (numpy)
def host_inputs(wl, seed, K=None, stride=None, segments=None):
    """numpy replicas (K, stride), w, v for workload `wl` (optionally with a
    different K or a subset of its segments)."""
    K = wl.K if K is None else K
    segs = wl.segments if segments is None else segments
    stride = default_stride(wl) if stride is None else stride
    gdt = np.float16 if wl.dtype == "f16" else np.float32
    rng = np.random.default_rng(seed)
    reps = np.zeros((K, stride), dtype=gdt)
    w = np.zeros(wl.padded, dtype=np.float32)
    v = np.zeros(wl.padded, dtype=np.float32)
    for s in segs:
        sig = grad_sigma(wl, s)
        reps[:, s.offset:s.offset + s.length] = (
            rng.standard_normal((K, s.length), dtype=np.float32) * np.float32(sig)).astype(gdt)
    rng_w = np.random.default_rng(seed + 1)
    for s in segs:
        kind, a = weight_recipe(wl, s)
        sl = slice(s.offset, s.offset + s.length)
        if kind == "normal":
            w[sl] = rng_w.standard_normal(s.length, dtype=np.float32) * np.float32(a)
        elif kind == "uniform":
            w[sl] = rng_w.uniform(-a, a, s.length).astype(np.float32)
        else:
            w[sl] = np.float32(a)
    return reps, w, v


# ---------------------------------------------------------------- device (torch)
def device_inputs(wl, seed, device, K=None, stride=None):
    """torch replicas (K, stride), w, v allocated and drawn on `device`."""
    import torch

    K = wl.K if K is None else K
    stride = default_stride(wl) if stride is None else stride
    gdt = torch.float16 if wl.dtype == "f16" else torch.float32
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    reps = torch.zeros((K, stride), dtype=gdt, device=device)
    w = torch.zeros(wl.padded, dtype=torch.float32, device=device)
    v = torch.zeros(wl.padded, dtype=torch.float32, device=device)
    for s in wl.segments:
        sig = grad_sigma(wl, s)
        x = torch.randn((K, s.length), generator=g, device=device, dtype=torch.float32)
        reps[:, s.offset:s.offset + s.length] = (x * sig).to(gdt)
        del x
    _draw_weights(wl, seed + 1, g, w)
    return reps, w, v


def _draw_weights(wl, seed, g, w):
    import torch

    g.manual_seed(seed)
    for s in wl.segments:
        kind, a = weight_recipe(wl, s)
        sl = slice(s.offset, s.offset + s.length)
        if kind == "normal":
            w[sl] = torch.randn(s.length, generator=g, device=w.device) * a
        elif kind == "uniform":
            w[sl] = (torch.rand(s.length, generator=g, device=w.device) * 2 - 1) * a
        else:
            w[sl] = a


def device_weights(wl, seed, device):
    """torch w, v on `device` drawn as device_inputs(wl, seed, ...) draws
    them (same recipe and seed): extra weight/velocity sets for a benchmark
    that rotates them independently of the replicas."""
    import torch

    g = torch.Generator(device=device)
    w = torch.zeros(wl.padded, dtype=torch.float32, device=device)
    v = torch.zeros(wl.padded, dtype=torch.float32, device=device)
    _draw_weights(wl, seed + 1, g, w)
    return w, v


# ---------------------------------------------------------------- random tables for tests
def random_table(rng, nseg, max_len, vec, gap_max=3, min_len=1):
    """A ragged, sorted, non-overlapping segment table: lengths in
    [min_len, max_len], each offset a multiple of `vec`, random gaps."""
    rows, off = [], 0
    for _ in range(nseg):
        off += int(rng.integers(0, gap_max + 1)) * vec
        n = int(rng.integers(min_len, max_len + 1))
        rows.append((off, n, 1.0, 1.0))
        off = (off + n + vec - 1) // vec * vec
    return rows, off


def random_replicas(rng, K, n, dtype, scale=1.0, stride=None):
    """(K, stride) replicas of N(0, scale) values in `dtype` (np.float32 or
    np.float16); stride defaults to n."""
    stride = n if stride is None else stride
    x = (rng.standard_normal((K, stride), dtype=np.float32) * np.float32(scale)).astype(dtype)
    return x
