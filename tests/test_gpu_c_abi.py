"""The C ABI from a program with no Python and no PyTorch.

tests/c_abi/abi_example (built by __graft_entry__.build()) allocates with
hipMalloc, fits its tables with fewbit_fit_table and runs fewbit_fwd and
fewbit_bwd on the null stream (bf16 GELU 3-bit, through the table kernel)
and on a stream it created (fp32 Sigmoid 4-bit, symmetric table), on ragged
element counts.  Its inputs, tables and outputs are checked here against
the CPU oracle: codes and grad_in bit for bit, y within the type's
tolerance.
"""
import os
import subprocess
import sys

import numpy as np
import pytest

import oracle as O
from parity import THREADS, check_exact, check_y

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
EXE = os.path.join(ROOT, "tests", "c_abi", "abi_example")

CASES = [("gelu_bf16_b3", O.GELU, "bf16"), ("sigmoid_f32_b4_sym", O.SIGMOID, "f32")]


def test_c_program_against_oracle(tmp_path):
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    assert os.path.exists(EXE), "tests/c_abi/abi_example is built by __graft_entry__.build()"
    print("[c-abi] running", EXE, flush=True)
    r = subprocess.run([EXE, str(tmp_path)], capture_output=True, text=True, timeout=300)
    print(r.stdout, r.stderr, flush=True)
    assert r.returncode == 0
    sys.path.insert(0, ROOT)
    from paper_2202_00441_amd._lib import CTable
    for name, act, dt in CASES:
        base = str(tmp_path / name)
        with open(base + ".table", "rb") as fh:
            t = CTable.from_buffer_copy(fh.read())
        K = 1 << t.bits
        s = np.float32([t.s[m] for m in range(K - 1)])
        v = np.float32([t.v[m] for m in range(K)])
        view = np.uint32 if dt == "f32" else np.uint16
        x = np.fromfile(base + ".x", dtype=view)
        g = np.fromfile(base + ".g", dtype=view)
        y = np.fromfile(base + ".y", dtype=view)
        gin = np.fromfile(base + ".gin", dtype=view)
        codes = np.fromfile(base + ".codes", dtype=np.uint32)
        print(f"[c-abi] {name} n={x.size} bits={t.bits} flags={t.flags}", flush=True)
        y_ref, c_ref = O.fwd(act, O.F32 if dt == "f32" else O.BF16, t.bits, s, x,
                             symmetric=bool(t.flags & 1), threads=THREADS)
        gin_ref = O.bwd(O.F32 if dt == "f32" else O.BF16, t.bits, v, g, c_ref, threads=THREADS)
        check_exact(codes, c_ref, f"{name} codes")
        check_y(y, y_ref, dt, f"{name} y")
        check_exact(gin, gin_ref, f"{name} grad_in")
