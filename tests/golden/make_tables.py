"""Write tests/golden/tables.json: the fitted tables every parity case uses.

Calls only the CPU oracle (oracle/), never the product library.  Each table
is the oracle's dynamic-programming fit (Sec. 3) of f' under the weight named
by the workload, on a uniform grid; boundaries and values are stored as
hexadecimal floats of their fp32 values so both sides read identical bits.

Run:  python tests/golden/make_tables.py
"""
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import oracle as O  # noqa: E402
from workloads import WORKLOADS  # noqa: E402

ACT = {"gelu": O.GELU, "silu": O.SILU, "sigmoid": O.SIGMOID, "tanh": O.TANH}


def weight(spec):
    if spec["kind"] == "uniform":
        return O.uniform(spec["A"], spec["B"])
    if spec["kind"] == "normal":
        return O.normal(spec["A"], spec["B"], 0.0, spec["sigma"])
    if spec["kind"] == "mixture":
        return O.mixture(spec["A"], spec["B"], spec["p"], spec["sigma"], spec["sigma2"])
    raise ValueError(spec)


# Activations with an even f' also get the symmetric fit of the Fig. 3
# caption (bins of |x|, fit on [0, B]), keyed "<workload>/b<bits>/sym".
SYMMETRIC = ("sigmoid", "tanh")


def main():
    out = {}
    for name, w in WORKLOADS.items():
        for b in w.bits:
            for sym in ((False, True) if w.act in SYMMETRIC else (False,)):
                t0 = time.time()
                F = O.fit(ACT[w.act], b, weight(w.fit), w.fit["n_grid"], symmetric=sym)
                key = f"{name}/b{b}" + ("/sym" if sym else "")
                out[key] = {
                    "act": w.act, "bits": b, "symmetric": sym, "weight": w.fit,
                    "s": [float(v).hex() for v in F.s],
                    "v": [float(v).hex() for v in F.v],
                    "loss": F.loss,
                }
                print(f"{key}: loss={F.loss:.6g} ({time.time() - t0:.1f}s)", flush=True)
    with open(os.path.join(HERE, "tables.json"), "w") as fh:
        json.dump(out, fh, indent=1, sort_keys=True)
        fh.write("\n")


if __name__ == "__main__":
    main()
