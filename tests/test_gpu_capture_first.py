"""A process's very first fp16 / bf16 forward can be made inside a graph
capture: the library keeps no per-device state to set up and never
synchronises, so the first call needs nothing outside the stream it is given.

The case runs in a child process of its own, so that nothing in the test
process has called the library before: it captures forward + backward of a
bf16 tensor through the table kernel (and another through the per-element
kernel, each chosen in the table) into a HIP graph before any eager call, replays the graph three times with
synchronisation in between, and checks every replay against the CPU oracle
(codes and grad_in bit-exact, y within 1 ulp).
"""
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

CHILD = r"""
import sys
import numpy as np
sys.path.insert(0, ROOT); sys.path.insert(0, ROOT + "/tests")
import torch
import paper_2202_00441_amd as P
import oracle as O
from parity import THREADS, check_exact, check_y, download, download_codes, golden_table, upload
spec, table = golden_table("gelu_bf16_lm_ffn_16x2048x8192/b3")
s = np.float32([float.fromhex(h) for h in spec["s"]])
v = np.float32([float.fromhex(h) for h in spec["v"]])
rng = np.random.default_rng(77)
for n, flags in (((1 << 22) + 12345, P.FLAG_TABLE_FWD), (70001, P.FLAG_ELEMENT_FWD)):
    tab = table.with_flags(flags)
    xb = O.round_array(O.BF16, rng.normal(0, 2, n))
    gb = O.round_array(O.BF16, rng.normal(0, 1, n))
    x, g = upload(xb, "bf16"), upload(gb, "bf16")
    y = torch.empty_like(x)
    gin = torch.empty_like(g)
    codes = torch.empty(P.packed_words(n, 3), dtype=torch.int32, device="cuda")
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    print(f"[capture-first] n={n} capturing", flush=True)
    with torch.cuda.stream(side):
        with torch.cuda.graph(graph, stream=side):
            P.fwd(tab, x, y=y, codes=codes)
            P.bwd(tab, g, codes, grad_in=gin)
    torch.cuda.current_stream().wait_stream(side)
    y_ref, c_ref = O.fwd(O.GELU, O.BF16, 3, s, xb, threads=THREADS)
    gin_ref = O.bwd(O.BF16, 3, v, gb, c_ref, threads=THREADS)
    for rep in range(3):
        y.fill_(0); codes.fill_(-1); gin.fill_(0)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        check_exact(download_codes(codes), c_ref, f"replay {rep} codes n={n}")
        check_y(download(y, "bf16"), y_ref, "bf16", f"replay {rep} y n={n}")
        check_exact(download(gin, "bf16"), gin_ref, f"replay {rep} grad_in n={n}")
    print(f"[capture-first] n={n} ok", flush=True)
print("CAPTURE_FIRST_OK", flush=True)
"""


def test_first_call_inside_graph_capture():
    code = f"ROOT = {ROOT!r}\n" + CHILD
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=240)
    print(r.stdout[-4000:], r.stderr[-4000:], flush=True)
    assert r.returncode == 0 and "CAPTURE_FIRST_OK" in r.stdout
