"""Build the native consumer of the C ABI (host code only: g++ against the
HIP runtime and libciera.so, no Python, no torch)."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
EXE = os.path.join(HERE, "abi_roundtrip")


def build() -> str:
    cmd = ["g++", "-O2", "-std=c++17", "-Wall", "-Werror",
           "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"),
           "-I", os.path.join(ROCM, "include"),
           os.path.join(HERE, "abi_roundtrip.cpp"),
           "-L", os.path.join(ROOT, "paper_2609_04609_amd"), "-lciera",
           "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
           "-Wl,-rpath,$ORIGIN/../../paper_2609_04609_amd",
           "-Wl,-rpath," + os.path.join(ROCM, "lib"),
           "-o", EXE]
    subprocess.run(cmd, check=True)
    return EXE


if __name__ == "__main__":
    print(build())
