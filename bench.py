#!/usr/bin/env python3
"""Benchmark of the fused tree-reduce + momentum-SGD step on one MI355X.

One step = one fc_step call over all K synthetic gradient replicas of a
workload (reduce in binary-tree order, average, SGD with momentum and weight
decay, write back w and v), with every input resident in device memory.  The
plan's schedule runs the step as one resident kernel (reduce into LDS, then
update from it), one fused kernel, or a reduce pass and an update pass.
Consecutive steps alternate between two independent replica sets (--rotate),
and w, v rotate over enough sets of their own (--wv-sets) that no step finds
earlier steps' w and v in the Infinity Cache.

Prints ONE JSON line: effective HBM GB/s of the step (algorithmic bytes per
step / wall time per step over the timed steps), the roofline entry of the
dominant kernel (its algorithmic bytes per call / its call time from HIP
events the library records on the launch stream around each call, all of the
call's launches included, against the 8 TB/s HBM3E peak; beside it the
kernel time rocprofv3 recorded for the same sources, when committed), a
parity verdict (one more step of the timed plan, outside the timed regions,
compared bit for bit with the oracle on every element) and the oracle timed
on the host cores as a CPU baseline.  Exits with status 1 when parity fails.

    python bench.py [--workload googlenet] [--steps 200] [--warmup 20]
"""
import argparse
import hashlib
import json
import math
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, AMD published peak
INFINITY_CACHE_BYTES = 256 << 20  # MI355X last-level (memory-side) cache
# Two replica sets by default, each far larger than the caches.  w and v are
# rotated over enough sets of their own that their footprint is at least
# twice the Infinity Cache: measured on MI355X, with up to four (w, v) sets
# of a GoogLeNet- or NiN-sized plan (56-60 MB each) every step found the
# previous steps' w and v in that cache (GoogLeNet 533-535 us per step with
# 1, 2 or 4 sets, 541 with 8; NiN 162-165 vs 168).  In training the forward
# and backward passes between two steps would evict them.
DEFAULT_ROTATE = 2


def default_wv_sets(wl, rotate):
    return max(rotate, math.ceil(2 * INFINITY_CACHE_BYTES / (8 * wl.padded)))
METRIC = "effective HBM GB/s (and % of peak) for tree-reduce+SGD step; µs per step"
CSRC = os.path.join(ROOT, "paper_1511_00175_amd", "csrc")


KERNEL_SOURCES = ("fc_device.h", "fc_internal.h", "fc_shape.h", "fc_reduce_f32.hip", "fc_reduce_f16.hip",
                  "fc_update.hip")


def _code_tokens(text):
    """C++ source with comments removed and whitespace collapsed (the sources
    hashed here hold no string literal with comment markers)."""
    import re
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split())


def kernel_hash():
    """Hash of what decides the kernels that run: the device code and the
    launch-shape / schedule rules (host-only code is left out), comments and
    layout ignored."""
    h = hashlib.sha256()
    for fn in KERNEL_SOURCES:
        with open(os.path.join(CSRC, fn), encoding="utf-8") as f:
            h.update(fn.encode() + b"\0" + _code_tokens(f.read()).encode())
    return h.hexdigest()[:16]


def kernel_bytes(wl, kind, out=False, bcast=False):
    """Algorithmic HBM bytes of one launch of a kernel kind over N parameters:
    step   : K replicas + w, v read, w', v' written (+ raw sum, + broadcast)
    reduce : K replicas read, raw sum written
    sgd    : raw sum, w, v read, w', v' written (+ broadcast)"""
    n, K, sg = wl.n_params, wl.K, wl.s_g
    if kind == "step":
        return n * (K * sg + 16) + (4 * n if out else 0) + (4 * n * K if bcast else 0)
    if kind == "reduce":
        return n * (K * sg + 4)
    if kind == "sgd":
        return n * 20 + (4 * n * K if bcast else 0)
    if kind == "bcast":
        return n * (4 + 4 * K)
    raise ValueError(kind)


def read_traffic(workload, kernel):
    """HBM bytes per step moved by `kernel` (all its launches in one step)
    from the committed rocprofv3 counter summary for this workload, or None
    when absent or taken on another version of the library sources."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip()
    if kv.get("kernel_source_sha256_16") != kernel_hash() or kv.get("kernel") != kernel:
        return None
    try:
        return float(kv["hbm_bytes_per_step"])
    except (KeyError, ValueError):
        return None


def read_profile_us(workload, kernel):
    """Average kernel time per step (us) that rocprofv3 recorded for `kernel`
    in profiles/traffic_<workload>.txt, or None when absent or taken on
    another version of the kernel sources."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip()
    if kv.get("kernel_source_sha256_16") != kernel_hash() or kv.get("kernel") != kernel:
        return None
    try:
        return float(kv["rocprof_us_per_step"])
    except (KeyError, ValueError):
        return None


def mismatches(a, b):
    """Elements whose bits differ (any NaN equal to any NaN)."""
    import numpy as np
    a, b = np.asarray(a, dtype=np.float32).ravel(), np.asarray(b, dtype=np.float32).ravel()
    nan = np.isnan(a) & np.isnan(b)
    return int(np.count_nonzero(~nan & (a.view(np.uint32) != b.view(np.uint32))))


def parity_check(plan, wl, reps, wv, order, out, bcast):
    """One more step of the timed plan (shares as timed) on replica set 0 and
    on copies of (w, v) set 0 as the timed steps left it, outside the timed regions,
    against the oracle run on host copies of the same inputs (every host
    thread, one range of elements each): every element of w', v' (and of
    the raw sum and the K worker copies when the step writes them), padding
    included.  Returns the JSON object and the host copies of the inputs."""
    import numpy as np
    import torch

    import oracle

    w, v = wv[0].clone(), wv[1].clone()
    reps_h, w_h, v_h = reps.cpu().numpy(), w.cpu().numpy(), v.cpu().numpy()
    n = w.numel()
    out_d = torch.full((n,), -1.0, device=w.device) if out else None
    dst_d = torch.full((wl.K, n), -2.0, device=w.device) if bcast else None
    plan.step(reps, w, v, wl.lr, wl.mu, wl.wd, wl.batch, out=out_d, bcast=dst_d)
    torch.cuda.synchronize()
    out_h = np.full(n, -1.0, np.float32) if out else None
    dst_h = [np.full(n, -2.0, np.float32) for _ in range(wl.K)] if bcast else None
    threads = oracle.default_threads()
    t0 = time.perf_counter()
    ew, ev, _, _ = oracle.step_parallel(wl.table(), reps_h, w_h, v_h, wl.lr, wl.mu, wl.wd, wl.batch, order=order,
                                        out=out_h, bcast=dst_h, threads=threads)
    dt = time.perf_counter() - t0
    bad = mismatches(w.cpu().numpy(), ew) + mismatches(v.cpu().numpy(), ev)
    names = ["w", "v"]
    if out:
        bad += mismatches(out_d.cpu().numpy(), out_h)
        names.append("raw sum")
    if bcast:
        bad += sum(mismatches(dst_d[k].cpu().numpy(), dst_h[k]) for k in range(wl.K))
        names.append(f"{wl.K} worker copies")
    elements = n * (2 + (1 if out else 0) + (wl.K if bcast else 0))
    res = {"bit_exact": bad == 0, "elements": elements, "mismatches": bad, "outputs": names,
           "checked": f"every element of {', '.join(names)} ({n} per buffer, padding included) after one "
                      "more step of the timed plan, against the oracle on the same inputs",
           "oracle": f"oracle.step_parallel, {threads} host threads", "oracle_seconds": round(dt, 3)}
    return res, (reps_h, w_h, v_h)


def host_info():
    model = platform.processor() or ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return model, os.cpu_count()


def cpu_baseline(wl, reps_h, w_h, v_h, order, target_s=10.0):
    """Time the oracle on a contiguous window [0, m) of the workload's
    elements, all K replicas, from host copies of the inputs: on one host
    core (oracle.step; the window grown to about target_s seconds, or the
    whole step, repeated until about target_s seconds of work), then on every
    host thread (oracle.step_parallel: one range of elements per thread, the
    same arithmetic for every element; at least 3 runs, repeated until the
    threads have done about target_s seconds of work).  Each leg reports its
    fastest run.  Returns the JSON object."""
    import oracle

    table = wl.table()

    def window(m):
        # segments clipped to [0, m)
        return [(o, min(n, m - o), lm, dm) for o, n, lm, dm in table if o < m]

    def run(m):
        rows = window(m)
        t0 = time.perf_counter()
        oracle.step(rows, list(reps_h[:, :m]), w_h[:m], v_h[:m], wl.lr, wl.mu, wl.wd, wl.batch, order=order)
        return time.perf_counter() - t0, sum(n for _, n, _, _ in rows)

    def repeat(fn, threads, min_runs, times):
        # fastest of at least min_runs runs, and of as many as make about
        # target_s seconds of work over `threads` threads
        while len(times) < min_runs or (sum(times) * threads < target_s and len(times) < 1000):
            times.append(fn())
        return min(times), len(times), sum(times)

    total = max(o + n for o, n, _, _ in table)
    m = min(total, 1 << 16)
    dt, n = run(m)
    # grow the window to about target_s seconds of single-thread oracle work
    m2 = min(total, int(m * target_s / max(dt, 1e-6)))
    if m2 > m:
        dt, n = run(m2)
        m = m2
    dt, runs1, _ = repeat(lambda: run(m)[0], 1, 1, [dt])
    bytes_ = n * (wl.K * wl.s_g + 16)
    model, ncpu = host_info()
    nthreads = oracle.default_threads()
    rows = window(m)

    def run_mt():
        t0 = time.perf_counter()
        oracle.step_parallel(rows, reps_h[:, :m], w_h[:m], v_h[:m], wl.lr, wl.mu, wl.wd, wl.batch, order=order,
                             threads=nthreads)
        return time.perf_counter() - t0

    dt_mt, runs_mt, wall_mt = repeat(run_mt, nthreads, 3, [])
    return {"value": round(bytes_ / dt_mt / 1e9, 4), "unit": "GB/s", "cores": nthreads, "kind": "oracle",
            "sample": f"{n} of {wl.n_params} parameters (elements [0, {m}) of the layout), all K={wl.K} "
                      f"replicas, one fused step, cut into {nthreads} element ranges run on {nthreads} host "
                      f"threads (fastest of {runs_mt} runs, {wall_mt:.2f} s in all: {dt_mt:.3f} s) of {ncpu} "
                      f"({model})",
            "seconds": round(dt_mt, 3), "runs": runs_mt, "us_per_step_equiv": round(dt_mt / n * wl.n_params * 1e6, 1),
            "single_thread": {"value": round(bytes_ / dt / 1e9, 4), "seconds": round(dt, 3), "cores": 1,
                              "runs": runs1}}


FIG4_KS = (1, 2, 4, 8, 16, 32, 64, 128)


def sweep_k(n, ks=FIG4_KS, reps_per_k=20, seed=1511, samples=1 << 16):
    """One-GPU analog of Fig. 4 (parameter server vs reduction tree, NiN's 30 MB
    per worker at n = 7,595,176): for each K, time fc_tree_reduce in tree and
    in linear (parameter-server) order over one n-element fp32 vector per
    worker, and measure each order's rounding error against an fp64 sum on
    `samples` sampled elements.  On one GPU both orders read the same K*n*4
    bytes, so time grows linearly in K for both (Eq. 3 vs Eq. 4 is a network
    cost model); what the order changes is the error bound: |s - exact| <=
    gamma_d * sum|x| with d = ceil(log2 K) for the tree, d = K-1 for the
    linear order.  Returns one record per (K, order)."""
    import torch

    import paper_1511_00175_amd as fc

    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    kmax = max(ks)
    stride = (n + 63) // 64 * 64 + 64  # 256-byte aligned replica rows, staggered
    reps = (torch.randn((kmax, stride), generator=g, device=dev) * 1e-3)
    out = torch.empty(n, device=dev)
    rows = [(0, n, 1.0, 1.0)]
    sample = torch.randint(0, n, (min(samples, n),), generator=g, device=dev)
    u = 2.0 ** -24
    recs = []
    for K in ks:
        x = reps[:K]
        exact = x[:, sample].double().sum(0)
        absum = x[:, sample].double().abs().sum(0)
        for order in ("tree", "linear"):
            plan = fc.Plan(rows, K, "f32", order)
            plan.set_timing(True)
            for _ in range(3):
                plan.tree_reduce(x, out)
            plan.read_timing()
            for _ in range(reps_per_k):
                plan.tree_reduce(x, out)
            torch.cuda.synchronize()
            launches, total = plan.read_timing()["reduce"]
            plan.close()
            rel = ((out[sample].double() - exact).abs() / absum).cpu()
            d = 0 if K == 1 else (math.ceil(math.log2(K)) if order == "tree" else K - 1)
            us = total / launches
            recs.append({"sweep": "fig4_one_gpu", "K": K, "order": order, "n_params": n,
                         "mb_per_worker": round(4 * n / 1e6, 1), "us": round(us, 2),
                         "gb_s": round((K * 4 + 4) * n / us / 1e3, 1),
                         "err_rel_median": float(rel.median()), "err_rel_max": float(rel.max()),
                         "bound_gamma_d": d * u / (1 - d * u)})
    return recs


XGMI_LINK_GBS = 153.0  # one MI355X xGMI link, per direction (7 links per GPU)


def _mean_call_us(plan, kind, fn, n):
    """Mean duration of a call kind over n calls (the library's HIP events)."""
    import torch

    plan.set_timing(True)
    fn()
    torch.cuda.synchronize()
    plan.read_timing()
    for _ in range(n):
        fn()
    torch.cuda.synchronize()
    launches, total = plan.read_timing()[kind]
    plan.set_timing(False)
    return total / launches


def shard_tables(table, G):
    """The G owners' segment tables: the element range [0, extent) cut at
    multiples of 64 elements into G slices, each segment clipped to each
    slice (offsets stay those of the full buffers).  Every segment element
    lies in exactly one slice's table, with its segment's multipliers."""
    ext = max((o + n for o, n, _, _ in table), default=0)
    bounds = [min(ext, (r * ext // G) // 64 * 64) for r in range(G)] + [ext]
    return [[(max(o, a), min(o + n, b) - max(o, a), lr, dm) for o, n, lr, dm in table if min(o + n, b) > max(o, a)]
            for a, b in zip(bounds[:-1], bounds[1:])], bounds


def shard_share(wl, G, seed=1511, reps=20):
    """One GPU's share of the step when G GPUs split the K workers into G
    aligned runs of S = K/G (one subtree each) and the parameters into G
    slices, measured on this GPU at the real per-GPU shapes; the exchange
    between GPUs is not built, its time is modelled from the xGMI link rate.
      leaf : fc_tree_reduce over this GPU's S workers for all N parameters
             (its subtree's partial sums, written once);
      owner: fc_step on this GPU's slice with the G subtree partials as its
             workers (the top of the tree, the average, SGD).
    Parity: all G leaf reduces and all G owner steps run here, and every
    element of the sharded w', v' is compared bit for bit with the oracle's
    one-GPU step on the same inputs (reducing aligned runs of 2^m leaves and
    then the run sums in order is the tree over all K leaves, Sec. 6.2)."""
    import numpy as np
    import torch

    import oracle
    import paper_1511_00175_amd as fc
    from workloads import gen

    K = wl.K
    S = K // G
    if G < 1 or K % G or S & (S - 1):
        raise SystemExit(f"bench.py: --shard {G} must divide K={K} into runs of a power of two")
    dev = torch.device("cuda:0")
    reps_d, w0, v0 = gen.device_inputs(wl, seed, dev)
    table = wl.table()
    slices, bounds = shard_tables(table, G)

    # the leaves: G subtree partial sums, each a full-length fp32 vector
    leaf = fc.Plan(table, S, wl.dtype, "tree")
    parts = torch.zeros((G, wl.padded), device=dev)
    for k in range(G):
        leaf.tree_reduce(reps_d[k * S:(k + 1) * S], parts[k])
    torch.cuda.synchronize()
    leaf_us = _mean_call_us(leaf, "reduce", lambda: leaf.tree_reduce(reps_d[:S], parts[0]), reps)
    for k in range(G):  # the timed calls rewrote partial 0 with the same values
        leaf.tree_reduce(reps_d[k * S:(k + 1) * S], parts[k])
    leaf.close()
    # the owners: one plan per slice over the G partials; every slice stepped once
    w_s, v_s = w0.clone(), v0.clone()
    owners = [fc.Plan(slices[r], G, "f32", "tree") for r in range(G)]
    for r in range(G):
        owners[r].step(parts, w_s, v_s, wl.lr, wl.mu, wl.wd, wl.batch)
    torch.cuda.synchronize()
    w_t, v_t = w0.clone(), v0.clone()
    owner_us = _mean_call_us(owners[0], "step",
                             lambda: owners[0].step(parts, w_t, v_t, wl.lr, wl.mu, wl.wd, wl.batch), reps)
    slice_params = sum(n for _, n, _, _ in slices[0])
    for p in owners:
        p.close()
    # the whole step on one GPU, for comparison
    full = fc.Plan(table, K, wl.dtype, "tree")
    w_f, v_f = w0.clone(), v0.clone()
    one_us = _mean_call_us(full, "step", lambda: full.step(reps_d, w_f, v_f, wl.lr, wl.mu, wl.wd, wl.batch), reps)
    full.close()
    # parity of the sharded step against the oracle's one-GPU step
    threads = oracle.default_threads()
    ew, ev, _, _ = oracle.step_parallel(table, reps_d.cpu().numpy(), w0.cpu().numpy(), v0.cpu().numpy(), wl.lr, wl.mu,
                                        wl.wd, wl.batch, threads=threads)
    bad = mismatches(w_s.cpu().numpy(), ew) + mismatches(v_s.cpu().numpy(), ev)
    slice_bytes = 4 * (bounds[1] - bounds[0])
    rs_us = slice_bytes / (XGMI_LINK_GBS * 1e3)  # 7 foreign slices out and in, one per link, at once
    ag_us = slice_bytes / (XGMI_LINK_GBS * 1e3)  # w' slice to the 7 peers, one per link
    per_gpu = leaf_us + rs_us + owner_us + ag_us
    return {"shard": G, "workload": f"{wl.name}_k{K}_{wl.dtype}", "workers_per_gpu": S, "n_params": wl.n_params,
            "slice_params": slice_params,
            "leaf_reduce_us": round(leaf_us, 2),
            "leaf_gb_s": round((S * wl.s_g + 4) * wl.n_params / leaf_us / 1e3, 1),
            "owner_step_us": round(owner_us, 2),
            "exchange_model_us": {"reduce_scatter": round(rs_us, 2), "all_gather": round(ag_us, 2),
                                  "link_gb_s": XGMI_LINK_GBS, "bytes_per_link": slice_bytes},
            "per_gpu_step_us": round(per_gpu, 2), "one_gpu_step_us": round(one_us, 2),
            "step_speedup_model": round(one_us / per_gpu, 2),
            "parity": {"bit_exact": bad == 0, "elements": 2 * w_s.numel(), "mismatches": bad,
                       "checked": "every element of the sharded w', v' (all G slices' owner steps) against the "
                                  "oracle's one-GPU step on the same inputs"},
            "timing": "mean of the library's HIP events over the calls; the owner's G partial slices and w, v "
                      "slice fit the Infinity Cache"}


def input_hash(sets, wv):
    """sha256 (first 16 hex digits) over the first and last 4 KiB of every
    input buffer (each replica row of every replica set, then w and v of
    every (w, v) set), in order: names the synthetic inputs a run measured."""
    import torch

    h = hashlib.sha256()
    bufs = [reps[k] for reps, _, _ in sets for k in range(reps.shape[0])] + [t for pair in wv for t in pair]
    for t in bufs:
        b = t.view(-1).view(dtype=torch.uint8)
        h.update(b[:4096].cpu().numpy().tobytes())
        h.update(b[-4096:].cpu().numpy().tobytes())
    return h.hexdigest()[:16]


def graph_steps(plan, wl, inputs, out, bcast, n):
    """Capture n consecutive steps on one input set in one HIP graph (the
    plan's device tables already hold these pointers, so the captured calls
    are kernel launches only) and time its replays; returns µs per step."""
    import torch

    r, w, v = inputs
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        for _ in range(3):
            plan.step(r, w, v, wl.lr, wl.mu, wl.wd, wl.batch, out=out, bcast=bcast)
    s.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        for _ in range(n):
            plan.step(r, w, v, wl.lr, wl.mu, wl.wd, wl.batch, out=out, bcast=bcast)
    with torch.cuda.stream(s):
        for _ in range(3):
            g.replay()
        s.synchronize()
        reps = max(1, 2000 // n)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(s)
        for _ in range(reps):
            g.replay()
        e1.record(s)
    s.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / (reps * n)
    return {"us_per_step": round(us, 3), "steps_per_graph": n, "replays": reps,
            "value": round(wl.algorithmic_bytes() / us / 1e3, 2), "input_sets": 1}


def train_steps(plan, wl, inputs, n):
    """fc_train over n iterations of a poly learning-rate policy (power 0.5,
    the paper's GoogLeNet schedule, Sec. 7.3) on one input set, against a
    Python loop of n fc_step calls at the base rate on the same buffers; µs
    per iteration from HIP events on the current stream, best of 3."""
    import torch

    r, w, v = inputs
    policy = dict(kind="poly", base_lr=wl.lr, max_iter=n, power=0.5)

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        best = float("inf")
        for _ in range(3):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            best = min(best, e0.elapsed_time(e1) * 1e3 / n)
        return best

    def loop():
        for _ in range(n):
            plan.step(r, w, v, wl.lr, wl.mu, wl.wd, wl.batch)

    us_train = timed(lambda: plan.train(r, w, v, policy, 0, n, wl.mu, wl.wd, wl.batch))
    us_loop = timed(loop)
    return {"iters": n, "policy": policy, "us_per_iter": round(us_train, 2),
            "value": round(wl.algorithmic_bytes() / us_train / 1e3, 2),
            "step_loop_us_per_iter": round(us_loop, 2), "input_sets": 1}


def bandwidth_probes(dev):
    """Bandwidth ceilings measured on this GPU: the library's streaming read
    probe over 4 GiB, and torch's device copy of 1 GiB (1 GiB read + 1 GiB
    written); best of 10, GB/s."""
    import torch

    import paper_1511_00175_amd as fc

    def best(fn, nbytes, n=10):
        fn()
        torch.cuda.synchronize()
        t = float("inf")
        for _ in range(n):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            t = min(t, e0.elapsed_time(e1) * 1e-3)
        return nbytes / t / 1e9

    x = torch.ones(1 << 30, device=dev)
    part = torch.empty(fc.fc_read_probe_blocks(4 << 30), device=dev)
    read = best(lambda: fc.read_probe(x, part), 4 << 30)
    del x, part
    a = torch.ones(1 << 28, device=dev)
    b = torch.empty_like(a)
    copy = best(lambda: b.copy_(a), 2 << 30)
    del a, b
    return {"read_gbs": round(read, 1), "copy_gbs": round(copy, 1),
            "read": "fc_read_probe over 4 GiB", "copy": "torch copy of 1 GiB (bytes read + written)"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--warmup-seconds", type=float, default=3.0,
                    help="warm up for at least this long as well as for --warmup steps")
    ap.add_argument("--workload", default="googlenet",
                    choices=["flat", "nin", "googlenet", "vgg19", "alexnet", "googlenet_aux", "googlenet_caffe_bias",
                             "alexnet_ungrouped"])
    ap.add_argument("--order", default="tree", choices=["tree", "linear"])
    ap.add_argument("--out", action="store_true", help="also write the raw sum")
    ap.add_argument("--bcast", action="store_true", help="also broadcast w' to K worker copies")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-parity", action="store_true",
                    help="skip the parity check (one more step against the oracle on every element)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--seed", type=int, default=1511)
    ap.add_argument("--opts", default="", help="launch shape, e.g. block_threads=256,vecs_per_thread=1")
    ap.add_argument("--profile-loop", type=int, default=0,
                    help="after the measurement, launch this many extra steps (for rocprofv3 runs)")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="after the measurement, run a plain device copy of this many MiB three times "
                         "(reference kernel of known size for hardware byte counters)")
    ap.add_argument("--print-hash", action="store_true", help="print the library source hash and exit")
    ap.add_argument("--sweep-k", action="store_true",
                    help="instead of the benchmark line, print the tree vs parameter-server K sweep")
    ap.add_argument("--sweep-reps", type=int, default=20)
    ap.add_argument("--shard", type=int, default=0,
                    help="instead of the benchmark line, measure one GPU's share of the step on G GPUs "
                         "(leaf reduce + owner step, exchange modelled) and check the sharded result's bits")
    ap.add_argument("--no-kernel-timing", action="store_true",
                    help="do not record per-kernel events (roofline entry then uses the wall time per step)")
    ap.add_argument("--graph", type=int, default=0,
                    help="also capture this many steps (one input set) in one HIP graph and report the "
                         "graph-amortized time per step")
    ap.add_argument("--train-iters", type=int, default=0,
                    help="also time fc_train (poly learning-rate policy) over this many iterations on one input "
                         "set, beside a Python loop of fc_step calls on the same buffers")
    ap.add_argument("--no-probes", action="store_true",
                    help="skip the read and copy bandwidth probes reported beside the roofline")
    ap.add_argument("--no-balance", action="store_true",
                    help="keep equal resident shares (no fc_plan_balance after the warm-up)")
    ap.add_argument("--rotate", type=int, default=DEFAULT_ROTATE,
                    help="R independent replica sets, step i using set i mod R (1: one set)")
    ap.add_argument("--wv-sets", type=int, default=0,
                    help="W independent (w, v) sets, step i using set i mod W (default: at least R and enough "
                         "for twice the Infinity Cache, so that no step finds earlier steps' w and v cached)")
    args = ap.parse_args()

    if args.print_hash:
        print(kernel_hash())
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py: this benchmark measures one GPU only (the K workers are replicas on one device); "
              "--gpus must be 1", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_1511_00175_amd as fc
    from workloads import gen, tables

    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(2)
    if args.sweep_k:
        from workloads import tables as _t
        for rec in sweep_k(_t.nin().n_params, reps_per_k=args.sweep_reps, seed=args.seed):
            rec["kernel_source_sha256_16"] = kernel_hash()
            print(json.dumps(rec), flush=True)
        return
    dev = torch.device("cuda:0")
    wl = tables.get(args.workload)
    if args.shard:
        rec = shard_share(wl, args.shard, seed=args.seed)
        rec["kernel_source_sha256_16"] = kernel_hash()
        print(json.dumps(rec), flush=True)
        if not rec["parity"]["bit_exact"]:
            sys.exit(1)
        return
    opts = {}
    for kv in filter(None, args.opts.split(",")):
        k, v = kv.split("=")
        opts[k] = int(v)

    print(f"# workload {wl.name}: K={wl.K} {wl.dtype} N={wl.n_params} segs={len(wl.segments)}", file=sys.stderr,
          flush=True)
    if args.rotate < 1 or args.wv_sets < 0:
        ap.error("--rotate must be >= 1 and --wv-sets >= 0")
    sets = [gen.device_inputs(wl, args.seed + 7919 * i, dev) for i in range(args.rotate)]
    n_wv = args.wv_sets or default_wv_sets(wl, args.rotate)
    wv = [(ww, vv) for _, ww, vv in sets][:n_wv]
    wv += [gen.device_weights(wl, args.seed + 7919 * i, dev) for i in range(len(wv), n_wv)]
    reps, w, v = sets[0]
    out = torch.zeros_like(w) if args.out else None
    bcast = torch.zeros((wl.K, wl.padded), device=dev) if args.bcast else None
    # one plan per input set: each plan's device pointer table then stays
    # valid from step to step, as in a training loop that reuses its buffers
    plans = [fc.Plan(wl.table(), wl.K, wl.dtype, args.order, **opts) for _ in sets]
    plan = plans[0]
    info = plan.info()
    torch.cuda.synchronize()
    count = [0]

    def step():
        i = count[0] % len(sets)
        ww, vv = wv[count[0] % len(wv)]
        count[0] += 1
        plans[i].step(sets[i][0], ww, vv, wl.lr, wl.mu, wl.wd, wl.batch, out=out, bcast=bcast)

    # warm-up: at least W steps and at least --warmup-seconds of back-to-back
    # steps (a process started within seconds of another process freeing tens
    # of GB of device memory runs its first second or two about 4% slower)
    warm_steps, t_warm = 0, time.perf_counter()
    while warm_steps < args.warmup or time.perf_counter() - t_warm < args.warmup_seconds:
        step()
        warm_steps += 1
        if warm_steps % 20 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()
    # XCD-aware shares (resident schedule): each plan re-divides its tiles by
    # the per-XCD rates of its launches so far, twice, with warm-up steps
    # after each
    balance = None
    resident = info.schedule in (3, 4)
    if not args.no_balance and resident:
        for _ in range(2):
            rates = [p.balance() for p in plans]
            for _ in range(max(args.warmup, 2 * len(plans))):
                step()
            torch.cuda.synchronize()
        measured = [round(r, 4) for r in rates[0] if r > 0]
        # plans whose blocks take few tiles per round record nothing (fc.h)
        balance = {"xcd_rate": measured, "calls": 2} if measured else None
    # timed region 1: the steps alone (barrier = device synchronize on both sides)
    t0 = time.perf_counter()
    for i in range(args.steps):
        step()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    # timed region 2: the same steps with per-kernel HIP events, which the
    # library records on the launch stream (the current torch stream); the
    # events add small gaps between kernels, so `value` comes from region 1
    timing = {}
    if not args.no_kernel_timing:
        for p in plans:
            p.set_timing(True)
            p.read_timing()
        for i in range(args.steps):
            step()
        torch.cuda.synchronize()
        for p in plans:
            for k, (n, us) in p.read_timing().items():
                n0, us0 = timing.get(k, (0, 0.0))
                timing[k] = (n0 + n, us0 + us)
            p.set_timing(False)
    # timed region 3: one pair of torch events around every step (the library
    # launches on torch's current stream), for the median and spread
    per_step = []
    for _ in range(max(50, min(args.steps, 200))):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        step()
        e1.record()
        per_step.append((e0, e1))
    torch.cuda.synchronize()
    step_us = sorted(a.elapsed_time(b) * 1e3 for a, b in per_step)
    step_times = {"events": len(step_us), "median_us": round(step_us[len(step_us) // 2], 2),
                  "p10_us": round(step_us[len(step_us) // 10], 2), "p90_us": round(step_us[len(step_us) * 9 // 10], 2)}
    graph = None
    if args.graph > 0:
        graph = graph_steps(plan, wl, sets[0], out, bcast, args.graph)
    train = None
    if args.train_iters > 0:
        train = train_steps(plan, wl, sets[0], args.train_iters)
    for _ in range(args.profile_loop):
        step()
    torch.cuda.synchronize()
    probes = None if args.no_probes else bandwidth_probes(dev)
    if args.calib_copy_mib:
        n = args.calib_copy_mib * (1 << 20) // 4
        src = torch.ones(n, device=dev)
        dst = torch.empty(n, device=dev)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    bytes_step = wl.algorithmic_bytes(out=args.out, bcast=args.bcast)
    ms_per_step = wall / args.steps * 1e3
    value = bytes_step / (wall / args.steps) / 1e9
    # per kernel kind: calls, and the mean time between the HIP events the
    # library records around each call on its launch stream (all of a call's
    # launches: one per resident round)
    kernels = {k: {"calls": n, "call_us_avg": round(us / n, 2),
                   "algorithmic_bytes": kernel_bytes(wl, k, args.out, bcast=args.bcast and k != "reduce")}
               for k, (n, us) in timing.items() if n}
    if not kernels:  # no per-kernel events: the whole step stands in for its kernels
        kernels = {"step": {"calls": args.steps, "call_us_avg": round(ms_per_step * 1e3, 2),
                            "algorithmic_bytes": bytes_step}}
    dom = max(kernels, key=lambda k: kernels[k]["calls"] * kernels[k]["call_us_avg"])
    avg = kernels[dom]["call_us_avg"] * 1e-6
    achieved = kernels[dom]["algorithmic_bytes"] / avg / 1e9
    # the committed profiles cover each workload (and its linear order) in
    # the default launch configuration
    plain = not (args.out or args.bcast or opts or args.rotate != DEFAULT_ROTATE or args.no_balance or args.wv_sets)
    variant = wl.name + ("_linear" if args.order == "linear" else "")
    traffic = read_traffic(variant, dom) if plain else None
    prof_us = read_profile_us(variant, dom) if plain else None
    sched = {1: "fused", 2: "two-pass", 3: "resident", 4: "resident, one launch"}.get(info.schedule,
                                                                                      str(info.schedule))
    rk = "resident_kernel" if resident else "reduce_kernel"

    res = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "warmup_steps_run": warm_steps,
        "ms_per_step": round(ms_per_step, 4),
        "us_per_step": round(ms_per_step * 1e3, 2),
        "pct_of_peak": round(100 * value / HBM_PEAK_GBS, 2),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": f"{wl.name}_k{wl.K}_{wl.dtype}",
            "K": wl.K, "n_params": wl.n_params, "segments": len(wl.segments), "replica_dtype": wl.dtype,
            "order": args.order, "batch": wl.batch, "lr": wl.lr, "momentum": wl.mu, "weight_decay": wl.wd,
            "write_sum": args.out, "broadcast": args.bcast,
            "algorithmic_bytes_per_step": bytes_step,
            "launch": {"grid": info.grid, "tiles": info.ntiles, "block_threads": info.block_threads,
                       "vecs_per_thread": info.vecs_per_thread, "kchunk": info.kchunk,
                       "schedule": sched, "rounds": info.rounds, "lds_bytes": info.lds_bytes},
            "input_sets": args.rotate,
            "w_v_sets": n_wv,
            "balance": balance,
            "input_hash": input_hash(sets, wv),
            "step_times": step_times,
            "kernels": kernels,
            "parallelism": "single GPU",
        },
        "roofline": {
            "bound": "hbm",
            "achieved": round(achieved, 2),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": traffic,
            "kernel": {"step": f"fc::{rk} (fused step)", "reduce": f"fc::{rk} (reduce pass)",
                       "sgd": "fc::sgd_kernel", "bcast": "fc::bcast_kernel"}[dom],
            "call_us_avg": round(avg * 1e6, 2),
            "timing": "HIP events recorded by the library on the launch stream around each call of the "
                      "dominant kernel kind over timed region 2",
            "launches_per_call": info.rounds if info.schedule == 3 and dom in ("step", "reduce") else 1,
            "kernel_us_avg": prof_us,
            "kernel_us_source": "rocprofv3 kernel trace committed in profiles/ for these kernel sources"
                                if prof_us else None,
            "kernel_algorithmic_bytes": kernels[dom]["algorithmic_bytes"],
        },
        "cpu_baseline": None,
    }
    if probes:
        res["config"]["probes"] = probes
        res["roofline"]["frac_of_read_probe"] = round(achieved / probes["read_gbs"], 4)
        # a ceiling from the two probes: the replicas at the streaming-read rate,
        # then w, v read and written at the copy rate (the path's bytes, each at
        # the best rate this GPU showed for that kind of traffic)
        rep = wl.n_params * wl.K * wl.s_g
        rest = bytes_step - rep
        model_us = (rep / probes["read_gbs"] + rest / probes["copy_gbs"]) / 1e3
        res["roofline"]["probe_model"] = {"us_per_step": round(model_us, 2),
                                          "frac": round(model_us / (ms_per_step * 1e3), 4)}
    if graph:
        res["graph"] = graph
    if train:
        res["train"] = train
    res["parity"] = None
    host_copies = None
    if not args.no_parity:
        res["parity"], host_copies = parity_check(plans[0], wl, sets[0][0], wv[0], args.order, args.out, args.bcast)
    for p in plans:
        p.close()
    if not args.no_cpu_baseline:
        if host_copies is None:
            host_copies = (sets[0][0].cpu().numpy(), wv[0][0].cpu().numpy(), wv[0][1].cpu().numpy())
        res["cpu_baseline"] = cpu_baseline(wl, *host_copies, args.order, args.cpu_seconds)
    print(json.dumps(res), flush=True)
    if res["parity"] is not None and not res["parity"]["bit_exact"]:
        print(f"bench.py: {res['parity']['mismatches']} elements differ from the oracle", file=sys.stderr)
        sys.exit(1)


if __name__ == "__main__":
    main()
