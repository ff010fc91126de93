"""bench.py on the GPU: its JSON line carries the parity verdict of the step it
timed, and the Fig. 4 K sweep measures errors within each order's bound."""
import json
import math
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
pytestmark = pytest.mark.gpu


def test_bench_line_carries_parity(device):
    """A short run on the flat workload (one fused kernel per step): the line
    reports every element of w' and v' checked against the oracle, none
    differing, and the exit status is 0; the multi-step driver is timed beside
    the step loop."""
    r = subprocess.run([sys.executable, "-u", os.path.join(ROOT, "bench.py"), "--workload", "flat", "--steps", "5",
                        "--warmup", "2", "--no-probes", "--cpu-seconds", "0.2", "--train-iters", "10"],
                       capture_output=True, text=True, cwd=ROOT, timeout=240)
    assert r.returncode == 0, r.stderr[-2000:]
    line = json.loads(r.stdout.strip().splitlines()[-1])
    par = line["parity"]
    assert par["bit_exact"] and par["mismatches"] == 0
    assert par["elements"] == 2 * (1 << 20) and par["outputs"] == ["w", "v"]
    assert line["cpu_baseline"]["cores"] >= 1 and line["roofline"]["call_us_avg"] > 0
    tr = line["train"]
    assert tr["iters"] == 10 and tr["policy"]["kind"] == "poly"
    assert tr["us_per_iter"] > 0 and tr["step_loop_us_per_iter"] > 0


def test_sweep_k_errors_within_bounds(device):
    """The sweep behind the Fig. 4 analog at a small size: for every K and
    both orders the worst relative error against the fp64 sum stays within
    gamma_d (d = ceil(log2 K) for the tree, K - 1 for the linear order), K = 1
    is exact, and the tree's bound is never the larger one."""
    sys.path.insert(0, ROOT)
    import bench
    ks = (1, 2, 3, 4, 7, 8, 16, 33, 64, 128)
    recs = bench.sweep_k(50_000, ks=ks, reps_per_k=2, samples=20_000)
    assert len(recs) == 2 * len(ks)
    u = 2.0 ** -24
    for r in recs:
        K = r["K"]
        d = 0 if K == 1 else (math.ceil(math.log2(K)) if r["order"] == "tree" else K - 1)
        assert r["bound_gamma_d"] == pytest.approx(d * u / (1 - d * u))
        assert r["err_rel_max"] <= r["bound_gamma_d"] * (1 + 1e-6) + 1e-15, r
        if K == 1:
            assert r["err_rel_max"] == 0.0
        assert r["us"] > 0
    by = {(r["K"], r["order"]): r for r in recs}
    for K in ks:
        assert by[(K, "tree")]["bound_gamma_d"] <= by[(K, "linear")]["bound_gamma_d"]


def test_shard_share_is_bit_exact(device):
    """--shard 8 on NiN (32 workers: 8 subtrees of 4): the leaf reduces and the
    owners' steps over the 8 subtree partials reproduce the oracle's one-GPU
    step on every element, and each part of one GPU's share is timed."""
    r = subprocess.run([sys.executable, "-u", os.path.join(ROOT, "bench.py"), "--workload", "nin", "--shard", "8"],
                       capture_output=True, text=True, cwd=ROOT, timeout=240)
    assert r.returncode == 0, r.stderr[-2000:]
    rec = json.loads(r.stdout.strip().splitlines()[-1])
    assert rec["shard"] == 8 and rec["workers_per_gpu"] == 4
    assert rec["parity"]["bit_exact"] and rec["parity"]["mismatches"] == 0
    assert rec["leaf_reduce_us"] > 0 and rec["owner_step_us"] > 0 and rec["per_gpu_step_us"] > rec["leaf_reduce_us"]
