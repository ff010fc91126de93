"""bench.py's parts that need no GPU: the one-GPU contract, the kernel-source
hash that ties profiles/ to the sources, the algorithmic byte counts the
roofline entry divides by, and the slicing of --shard."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def run_bench(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True, text=True,
                          cwd=ROOT, timeout=120)


def test_more_than_one_gpu_is_refused_with_a_message():
    r = run_bench("--gpus", "2")
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_kernel_hash_is_stable_and_ignores_comments(tmp_path, monkeypatch):
    import bench
    h = bench.kernel_hash()
    assert len(h) == 16 and h == bench.kernel_hash()
    assert run_bench("--print-hash").stdout.strip() == h
    src = "int f(int x) { // a comment\n  return x; /* another */ }\n"
    assert bench._code_tokens(src) == bench._code_tokens("int f(int x) {\n return x;  }")
    assert bench._code_tokens(src) != bench._code_tokens("int f(int x) { return x + 1; }")


@pytest.mark.parametrize("name", ["flat", "nin", "googlenet", "vgg19", "alexnet"])
def test_kernel_bytes_match_the_workload(name):
    import bench
    from workloads import tables
    wl = tables.get(name)
    n, K, sg = wl.n_params, wl.K, wl.s_g
    assert bench.kernel_bytes(wl, "step") == wl.algorithmic_bytes() == n * (K * sg + 16)
    assert bench.kernel_bytes(wl, "step", out=True) == wl.algorithmic_bytes(out=True) == n * (K * sg + 20)
    assert bench.kernel_bytes(wl, "step", bcast=True) == wl.algorithmic_bytes(bcast=True) == n * (K * sg + 16 + 4 * K)
    # the two passes of the two-pass schedule add up to the step plus the raw sum written and read back
    assert bench.kernel_bytes(wl, "reduce") + bench.kernel_bytes(wl, "sgd") == n * (K * sg + 16) + 8 * n


def test_traffic_profiles_name_their_kernel_and_bytes():
    """Every committed traffic summary states its workload, kernel, the source
    hash it was taken on and HBM bytes within 3% of the algorithmic bytes
    (the network-sized steps are within 0.2%; the flat 2^20 x K=4 step, one
    fused block per 256 elements, reads 1.9% more: each of its 4096 blocks
    also reads its kernel arguments, tile entry and replica pointers)."""
    for name in ("flat", "nin", "googlenet", "vgg19", "alexnet"):
        kv = {}
        with open(os.path.join(ROOT, "profiles", f"traffic_{name}.txt")) as f:
            for line in f:
                if ":" in line and not line.startswith("#"):
                    k, v = line.split(":", 1)
                    kv[k.strip()] = v.strip()
        assert kv["workload"] == name and kv["kernel"] == "step"
        assert len(kv["kernel_source_sha256_16"]) == 16
        ratio = float(kv["hbm_bytes_per_step"]) / float(kv["algorithmic_bytes_per_step"])
        assert 0.99 < ratio < 1.03, (name, ratio)


def test_mismatches_compares_bits():
    import numpy as np

    import bench
    a = np.array([0.0, -0.0, 1.0, np.nan, 2.0], np.float32)
    b = np.array([0.0, 0.0, 1.0, np.nan, np.nextafter(np.float32(2.0), np.float32(3.0))], np.float32)
    assert bench.mismatches(a, a) == 0
    assert bench.mismatches(a, b) == 2  # -0 vs +0, and one ulp


def test_cpu_baseline_times_the_oracle_on_host_copies():
    """The baseline leg runs the oracle on one core and on every host thread
    over the same window of host copies and reports the thread count."""
    import bench
    from workloads import gen, tables
    wl = tables.flat()
    reps, w, v = gen.host_inputs(wl, 3)
    r = bench.cpu_baseline(wl, reps, w, v, "tree", target_s=0.05)
    assert r["kind"] == "oracle" and r["unit"] == "GB/s" and r["value"] > 0 and r["cores"] >= 1
    assert r["single_thread"]["cores"] == 1 and f"{r['cores']} host threads" in r["sample"]


def test_profile_time_needs_the_current_sources(tmp_path, monkeypatch):
    """roofline.kernel_us_avg comes from a committed profile only when it was
    taken on the current kernel sources."""
    import bench
    prof = tmp_path / "profiles"
    prof.mkdir()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    (prof / "traffic_x.txt").write_text(f"kernel: step\nkernel_source_sha256_16: {bench.kernel_hash()}\n"
                                        "rocprof_us_per_step: 12.5\n")
    assert bench.read_profile_us("x", "step") == 12.5
    assert bench.read_profile_us("x", "reduce") is None
    (prof / "traffic_x.txt").write_text("kernel: step\nkernel_source_sha256_16: 0000000000000000\n"
                                        "rocprof_us_per_step: 12.5\n")
    assert bench.read_profile_us("x", "step") is None


@pytest.mark.parametrize("G", [1, 2, 3, 8, 64])
def test_shard_tables_partition_the_segments(G):
    """The owners' tables of --shard cover every segment element exactly once,
    keep each element's multipliers, start every slice on a multiple of 64
    elements, and keep offsets on multiples of 4 (what a plan requires)."""
    import numpy as np

    import bench
    from workloads import gen, tables

    rng = np.random.default_rng(G)
    cases = [tables.get("googlenet").table(), tables.get("nin").table()]
    for _ in range(5):
        rows, _ = gen.random_table(rng, int(rng.integers(1, 20)), int(rng.integers(1, 5000)), 4, gap_max=40)
        cases.append([(o, n, float(rng.integers(1, 4)), float(rng.integers(0, 3))) for o, n, _, _ in rows])
    for table in cases:
        slices, bounds = bench.shard_tables(table, G)
        assert len(slices) == G and bounds[0] == 0 and all(b % 64 == 0 for b in bounds[:-1])
        ext = max(o + n for o, n, _, _ in table)
        want = np.full((2, ext), np.nan)
        for o, n, lr, dm in table:
            want[:, o:o + n] = [[lr], [dm]]
        got = np.full((2, ext), np.nan)
        count = np.zeros(ext, np.int64)
        for r, sl in enumerate(slices):
            for o, n, lr, dm in sl:
                assert o % 4 == 0 and n > 0 and bounds[r] <= o and o + n <= bounds[r + 1]
                got[:, o:o + n] = [[lr], [dm]]
                count[o:o + n] += 1
        assert np.array_equal(count, (~np.isnan(want[0])).astype(np.int64))
        assert np.array_equal(got, want, equal_nan=True)
