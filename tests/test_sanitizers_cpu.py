"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer, on the CPU.

1. The oracle, built with gcc and both sanitizers, through every pin and
   through the threaded driver (oracle.step_parallel, whose ranges hand the
   C code pointers into the middle of every buffer).
2. The host side of libfc.so -- plan construction, validation, aliasing,
   pointer tables, learning-rate policies -- compiled by hipcc with both
   sanitizers on the host pass only (the kernels are the normal build's
   objects), linked against the shared sanitizer runtime, and loaded in
   place of the library by the device-free ABI, binding and learning-rate
   tests.
Each runs in a subprocess with the sanitizer runtime preloaded; a report
aborts it (no recovery)."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_1511_00175_amd")
CSRC = os.path.join(PKG, "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:verify_asan_link_order=0",
           UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")


def _out(r):
    return (r.stdout + r.stderr)[-4000:]


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_oracle_under_sanitizers(tmp_path):
    sys.path.insert(0, ROOT)
    from oracle import build as obuild
    lib = obuild.build(lib=str(tmp_path / "liboracle_san.so"),
                       extra=["-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                              "-fno-sanitize-recover=all"])
    script = tmp_path / "run.py"
    script.write_text(f"""
import sys
sys.path[:0] = [{ROOT!r}, {os.path.join(ROOT, 'tests')!r}]
import numpy as np
import oracle
from oracle_pins import PINS
from workloads import gen
with oracle.use({lib!r}):
    for pin in PINS:
        pin()
    rng = np.random.default_rng(5)
    rows, n = gen.random_table(rng, 13, 2000, 4, gap_max=4)
    for dt in (np.float32, np.float16):
        reps = (rng.standard_normal((9, n + 8), dtype=np.float32) * 0.01).astype(dt)
        w = rng.standard_normal(n + 8, dtype=np.float32)
        dst = [np.zeros(n + 8, np.float32) for _ in range(9)]
        out = np.zeros(n + 8, np.float32)
        for th in (1, 3, 8):
            oracle.step_parallel(rows, reps, w, w * 0, 0.01, 0.9, 5e-4, 256, out=out, bcast=dst, threads=th)
print("sanitized oracle ok", len(PINS))
""")
    asan = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    r = subprocess.run([sys.executable, str(script)], capture_output=True, text=True, timeout=600,
                       env=dict(ENV, LD_PRELOAD=asan))
    assert r.returncode == 0, _out(r)
    assert "sanitized oracle ok" in r.stdout and "runtime error" not in r.stderr, _out(r)


def _clang_asan_runtime():
    r = subprocess.run([HIPCC, "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True, text=True)
    path = r.stdout.strip()
    return path if r.returncode == 0 and os.path.isabs(path) and os.path.exists(path) else None


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="needs hipcc")
def test_host_library_under_sanitizers(tmp_path):
    runtime = _clang_asan_runtime()
    if runtime is None:
        pytest.skip("no clang AddressSanitizer runtime")
    kernels = [os.path.join(PKG, "_build", s + ".o") for s in ("fc_reduce_f32.hip", "fc_reduce_f16.hip",
                                                               "fc_update.hip")]
    if not all(os.path.exists(o) for o in kernels):
        pytest.skip("kernel objects not built (run __graft_entry__.build())")
    api = tmp_path / "fc_api.o"
    lib = tmp_path / "libfc_san.so"
    # the sanitizers on the host pass only: each flag behind -Xarch_host
    san = ["-Xarch_host", "-fsanitize=address,undefined", "-Xarch_host", "-fno-sanitize-recover=all",
           "-Xarch_host", "-fno-omit-frame-pointer"]
    r = subprocess.run([HIPCC, "-O1", "-g", "-std=c++17", "-fPIC", "--offload-arch=gfx950", "-ffp-contract=off",
                        f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}", *san, "-c",
                        os.path.join(CSRC, "fc_api.cpp"), "-o", str(api)], capture_output=True, text=True)
    assert r.returncode == 0, _out(r)
    r = subprocess.run([HIPCC, "-shared", "-fPIC", "--offload-arch=gfx950", *kernels, str(api),
                        "-Xarch_host", "-fsanitize=address,undefined", "-Xarch_host", "-shared-libsan",
                        "-o", str(lib)], capture_output=True, text=True)
    assert r.returncode == 0, _out(r)
    env = dict(ENV, LD_PRELOAD=runtime, FC_LIBRARY=str(lib))
    # the sanitized library is the one loaded
    probe = ("import paper_1511_00175_amd as m; maps = open('/proc/self/maps').read(); "
             f"assert m._fc.LIB_PATH == {str(lib)!r} and {str(lib)!r} in maps and 'libclang_rt.asan' in maps; "
             "print('loaded')")
    r = subprocess.run([sys.executable, "-c", probe], capture_output=True, text=True, cwd=ROOT, env=env, timeout=300)
    assert r.returncode == 0 and "loaded" in r.stdout, _out(r)
    tests = [os.path.join(ROOT, "tests", t) for t in ("test_abi.py", "test_lr.py", "test_binding_cpu.py")]
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider", "-m", "not gpu", *tests],
                       capture_output=True, text=True, cwd=ROOT, env=env, timeout=600)
    assert r.returncode == 0, _out(r)
    assert " passed" in r.stdout and "runtime error" not in r.stderr, _out(r)
