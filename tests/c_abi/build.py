"""Build tests/c_abi/abi_example (a C-ABI consumer with no Python) with hipcc.

Test infrastructure: it links the in-tree libfewbit.so through a relative
run path, so the binary finds the library wherever the tree is copied.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
OUT = os.path.join(HERE, "abi_example")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def build(verbose: bool = False) -> str:
    cmd = [HIPCC, "-O2", "-std=c++17", "-I", os.path.join(ROOT, "include"),
           os.path.join(HERE, "abi_example.cpp"), "-L", os.path.join(ROOT, "paper_2202_00441_amd"),
           "-lfewbit", "-Wl,-rpath,$ORIGIN/../../paper_2202_00441_amd", "-o", OUT + ".tmp"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(OUT + ".tmp", OUT)
    return OUT


if __name__ == "__main__":
    print(build(verbose=True))
