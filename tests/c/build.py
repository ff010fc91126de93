"""Compile the plain-C client of the library's ABI (tests/c/abi_step.c) with
gcc against include/fc.h, libfc.so, the oracle's liboracle.so and the HIP
runtime.  Test infrastructure: the GPU test tests/test_c_client_gpu.py runs
the binary."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
SRC = os.path.join(HERE, "abi_step.c")
BIN = os.path.join(HERE, "abi_step")


def build():
    cmd = ["gcc", "-std=c11", "-O2", "-Wall", "-Wextra", "-Werror", "-ffp-contract=off",
           "-D__HIP_PLATFORM_AMD__", f"-I{ROOT}/include", f"-I{ROCM}/include", SRC, "-o", BIN + ".tmp",
           f"-L{ROOT}/paper_1511_00175_amd", "-l:libfc.so", f"-L{ROOT}/oracle", "-l:liboracle.so",
           f"-L{ROCM}/lib", "-lamdhip64",
           "-Wl,-rpath,$ORIGIN/../../paper_1511_00175_amd", "-Wl,-rpath,$ORIGIN/../../oracle",
           f"-Wl,-rpath,{ROCM}/lib"]
    subprocess.run(cmd, check=True)
    os.replace(BIN + ".tmp", BIN)
    return BIN


if __name__ == "__main__":
    print(build())
