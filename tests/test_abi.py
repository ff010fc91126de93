"""The C ABI library loads on the host and exports every symbol include/fc.h
declares; argument errors that need no device are reported as documented."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fc.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(fc_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def fcmod():
    import paper_1511_00175_amd as m
    return m


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ("fc_plan_create", "fc_plan_create_ex", "fc_plan_destroy", "fc_tree_reduce", "fc_sgd_step",
              "fc_broadcast", "fc_step", "fc_strerror", "fc_plan_query", "fc_plan_set_timing",
              "fc_plan_read_timing", "fc_plan_balance"):
        assert n in names


def test_library_exports_every_declared_symbol(fcmod):
    lib = fcmod._fc.lib
    for n in declared_functions():
        assert hasattr(lib, n), n
        assert ctypes.cast(getattr(lib, n), ctypes.c_void_p).value


def test_strerror(fcmod):
    f = fcmod._fc
    assert f.fc_strerror(0) == "success"
    for code in (f.FC_EINVAL, f.FC_EALIGN, f.FC_EALIAS, f.FC_EHIP, f.FC_ENOMEM):
        assert f.fc_strerror(code) not in ("", "success", "unknown error code")
    assert f.fc_strerror(12345) == "unknown error code"


@pytest.mark.parametrize("segs,K,gdt,opts,code", [
    ([(0, 16)], 0, 0, None, -1),                       # K < 1
    ([(0, 16)], 1025, 0, None, -1),                    # K > 1024
    ([(2, 16)], 4, 0, None, -2),                       # fp32 offset not a multiple of 4
    ([(2, 16)], 4, 1, None, -2),                       # fp16 offset not a multiple of 4
    ([(64, 16), (0, 16)], 4, 0, None, -1),             # unsorted
    ([(0, 16), (8, 16)], 4, 0, None, -1),              # overlapping
    ([(0, 16)], 4, 7, None, -1),                       # bad dtype
    ([(0, 16)], 4, 0, {"block_threads": 96}, -1),      # bad launch shape
    ([(0, 16)], 4, 0, {"vecs_per_thread": 3}, -1),
    ([(0, 16)], 4, 0, {"vecs_per_thread": 1, "kchunk": 4}, -1),   # pair not compiled
    ([(0, 16)], 4, 0, {"vecs_per_thread": 4, "kchunk": 16}, -1),
    ([(0, 16)], 4, 0, {"max_blocks": -1}, -1),
    ([(0, 16)], 4, 0, {"schedule": 5}, -1),
    ([(0, 16)], 4, 0, {"schedule": -1}, -1),
    ([(0, 16)], 4, 0, {"schedule": 4, "vecs_per_thread": 4}, -1),   # one launch: the resident shapes
    ([(0, 16)], 512, 0, {"schedule": 4, "vecs_per_thread": 2}, -1),
    ([(0, 16)], 4, 0, {"schedule": 3, "k_waves": 4}, -1),        # resident: one launch shape
    ([(0, 16)], 4, 0, {"schedule": 3, "vecs_per_thread": 4}, -1),
    ([(0, 16)], 4, 0, {"schedule": 3, "block_threads": 128}, -1),
    ([(0, 16)], 4, 0, {"schedule": 3, "kchunk": 8}, -1),
    ([(0, 16)], 4, 0, {"schedule": 3, "vecs_per_thread": 2, "kchunk": 8}, -1),
    ([(0, 16)], 512, 0, {"schedule": 3, "vecs_per_thread": 2}, -1),   # two vectors: K / 4 < 128
])
def test_plan_argument_errors(fcmod, segs, K, gdt, opts, code):
    rc, h = fcmod._fc.fc_plan_create(segs, K, gdt, 0, opts)
    assert rc == code and not h.value


@pytest.mark.parametrize("K,order,opts", [
    (8, 0, {"k_waves": 2}),                             # one wave per lane-vector only
    (8, 1, {"k_waves": 4}),
    (128, 0, {"k_waves": 16}),
    (8, 0, {"k_waves": -1}),
])
def test_k_waves_errors(fcmod, K, order, opts):
    rc, h = fcmod._fc.fc_plan_create([(0, 16)], K, 0, order, opts)
    assert rc == fcmod._fc.FC_EINVAL and not h.value


def test_null_arguments(fcmod):
    f = fcmod._fc
    assert f.lib.fc_plan_create(None, None, 0, 1, 0, 0) == f.FC_EINVAL
    assert f.fc_tree_reduce(None, [0], 0) == f.FC_EINVAL
    assert f.fc_sgd_step(None, 0, 0, 0, 0.1, 0.9, 0.0, 1) == f.FC_EINVAL
    assert f.fc_broadcast(None, 0, [0]) == f.FC_EINVAL
    assert f.fc_step(None, [0], 0, 0, 0.1, 0.9, 0.0, 1) == f.FC_EINVAL
    assert f.lib.fc_plan_query(None, None) == f.FC_EINVAL
    assert f.lib.fc_plan_set_timing(None, 1) == f.FC_EINVAL
    assert f.lib.fc_plan_read_timing(None, None) == f.FC_EINVAL
    rates = (ctypes.c_float * 4)(1, 1, 1, 1)
    assert f.lib.fc_plan_balance(None, None, rates, 4) == f.FC_EINVAL
    assert f.lib.fc_plan_balance(None, None, None, 0) == f.FC_EINVAL
    f.fc_plan_destroy(None)


def test_oracle_and_library_share_nothing():
    """The oracle is built from its own source only and the HIP sources do
    not refer to it (and the other way round)."""
    csrc = os.path.join(ROOT, "paper_1511_00175_amd", "csrc")
    for fn in os.listdir(csrc):
        text = open(os.path.join(csrc, fn)).read()
        assert "orc_" not in text and "oracle" not in text.lower(), fn
    otext = open(os.path.join(ROOT, "oracle", "fc_oracle.c")).read()
    assert "#include \"fc" not in otext and "fc_internal" not in otext
    for fn in ("__init__.py", "_fc.py", "build.py"):
        text = open(os.path.join(ROOT, "paper_1511_00175_amd", fn)).read()
        assert "import oracle" not in text and "from oracle" not in text


def test_kernels_use_no_scratch_memory():
    """The build records the compiler's per-kernel resource usage: every
    kernel keeps its pending-subtree stack and partial sums in registers and
    LDS (no scratch memory)."""
    path = os.path.join(ROOT, "paper_1511_00175_amd", "_build", "kernel_resources.txt")
    if not os.path.exists(path):
        pytest.skip("library not built by paper_1511_00175_amd/build.py")
    rows = {}
    with open(path) as f:
        for line in f:
            name, *kv = line.split()
            rows[name] = dict(x.split("=") for x in kv)
    assert len(rows) >= 100
    assert all(r["ScratchSize"] == "0" for r in rows.values())
    assert any("resident_kernel" in n for n in rows) and any("reduce_kernel" in n for n in rows)


def test_read_probe_argument_errors(fcmod):
    f = fcmod._fc
    assert f.fc_read_probe(None, 16, 64, None) == f.FC_EINVAL
    assert f.fc_read_probe(64, 16, None, None) == f.FC_EINVAL
    assert f.fc_read_probe(64, 0, 64, None) == f.FC_EINVAL
    assert f.fc_read_probe(64, 20, 64, None) == f.FC_EINVAL     # not a multiple of 16
    assert f.fc_read_probe(72, 16, 64, None) == f.FC_EALIGN     # source not 16-byte aligned
    assert f.fc_read_probe_blocks(1) == 1 and f.fc_read_probe_blocks(16384) == 1
    assert f.fc_read_probe_blocks(16384 + 16) == 2


def test_header_is_plain_c(tmp_path):
    """include/fc.h is a C header: strict C99 with every warning an error."""
    import subprocess
    src = tmp_path / "use_fc.c"
    src.write_text('#include "fc.h"\nint main(void) { return fc_strerror(FC_OK) == 0; }\n')
    r = subprocess.run(["gcc", "-std=c99", "-pedantic", "-Wall", "-Wextra", "-Werror", "-fsyntax-only",
                        f"-I{os.path.join(ROOT, 'include')}", str(src)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


def test_binding_matches_header(tmp_path, fcmod):
    """Every constant the header defines has the same value in the binding,
    and every structure the binding passes has the header's size and field
    offsets (a C program built with gcc reports the header's view)."""
    import subprocess
    f = fcmod._fc
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    consts = sorted(set(re.findall(r"\b(FC_[A-Z0-9_]+)\s*(?:=|\(|[0-9])", text)) - {"FC_H"})
    consts = [c for c in consts if re.search(rf"(#define\s+{c}\b|\b{c}\s*=)", text)]
    assert "FC_SCHED_RESIDENT_ONE_LAUNCH" in consts and "FC_NOALLOC_MAX_ELEMS" in consts
    structs = {name: [fname for fname, _ in getattr(f, name)._fields_]
               for name in ("fc_segment", "fc_launch_opts", "fc_plan_info", "fc_timing", "fc_lr_policy")}
    lines = ['#include <stddef.h>', '#include <stdio.h>', '#include "fc.h"', "int main(void) {"]
    lines += [f'    printf("{c} %lld\\n", (long long)({c}));' for c in consts]
    for s, fields in structs.items():
        lines.append(f'    printf("sizeof {s} %zu\\n", sizeof({s}));')
        lines += [f'    printf("offsetof {s}.{fl} %zu\\n", offsetof({s}, {fl}));' for fl in fields]
    lines += ["    return 0;", "}"]
    src = tmp_path / "abi_view.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "abi_view"
    r = subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", f"-I{os.path.join(ROOT, 'include')}", str(src),
                        "-o", str(exe)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    out = subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout.splitlines()
    seen = 0
    for line in out:
        key, val = line.rsplit(" ", 1)
        val = int(val)
        if key.startswith("sizeof "):
            assert ctypes.sizeof(getattr(f, key.split()[1])) == val, key
        elif key.startswith("offsetof "):
            s, fl = key.split()[1].split(".")
            assert getattr(getattr(f, s), fl).offset == val, key
        else:
            assert getattr(f, key) == val, key
        seen += 1
    assert seen == len(consts) + sum(1 + len(v) for v in structs.values())
