"""Build the standalone C ABI check (host code only): g++ against include/epl.h, linked with the
library and, as the reference, the CPU oracle. Run by __graft_entry__.build() after both exist."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
SRC = os.path.join(HERE, "epl_c_check.cpp")
BIN = os.path.join(HERE, "epl_c_check")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def build() -> str:
    cmd = ["g++", "-O2", "-std=c++17", "-Wall", "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"),
           "-I", os.path.join(ROCM, "include"), SRC,
           "-L", os.path.join(ROOT, "paper_2607_06202_amd"), "-lepl",
           "-L", os.path.join(ROOT, "oracle"), "-loracle",
           "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
           "-Wl,-rpath,$ORIGIN/../../paper_2607_06202_amd:$ORIGIN/../../oracle:" + os.path.join(ROCM, "lib"),
           "-o", BIN + ".tmp"]
    subprocess.check_call(cmd)
    os.replace(BIN + ".tmp", BIN)
    return BIN


if __name__ == "__main__":
    print(build())
