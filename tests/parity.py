"""Shared helpers of the GPU parity tests: device upload / download of raw
storage bits and the comparison rules.

Rules (element by element, GPU vs oracle on the same seeded bits):
  * packed codes and grad_in: bit-exact;
  * y, fp32: |gpu - ref| <= 2e-6 + 1e-5 |ref|;
  * y, fp16 / bf16: at most 1 unit in the last place, measured on the ordered
    integer image of the bit patterns with -0 == +0;
  * NaN where and only where the oracle has NaN.
"""
from __future__ import annotations

import json
import os

import numpy as np

import oracle as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
TABLES = json.load(open(os.path.join(ROOT, "tests", "golden", "tables.json")))
ODT = {"f32": O.F32, "f16": O.F16, "bf16": O.BF16}
OACT = {"gelu": O.GELU, "silu": O.SILU, "sigmoid": O.SIGMOID, "tanh": O.TANH,
        "relu": O.RELU, "selu": O.SELU, "softplus": O.SOFTPLUS}
THREADS = max(1, min(16, os.cpu_count() or 1))


def torch_dtype(dt: str):
    import torch
    return {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}[dt]


def upload(bits: np.ndarray, dt: str):
    import torch
    if dt == "f32":
        t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int32))
    else:
        t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.cuda().view(torch_dtype(dt))


def download(t, dt: str) -> np.ndarray:
    import torch
    if dt == "f32":
        return t.view(torch.int32).cpu().numpy().view(np.uint32)
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def download_codes(t) -> np.ndarray:
    return t.cpu().numpy().view(np.uint32)


def golden_table(key: str):
    import paper_2202_00441_amd as P
    spec = TABLES[key]
    s = [float.fromhex(h) for h in spec["s"]]
    v = [float.fromhex(h) for h in spec["v"]]
    return spec, P.Table.from_values(P.ACTS[spec["act"]], spec["bits"], s, v,
                                     flags=P.FLAG_SYMMETRIC if spec.get("symmetric") else 0,
                                     loss=spec["loss"])


def _ordered(bits: np.ndarray, dt: str) -> np.ndarray:
    if dt == "f32":
        u = bits.astype(np.int64)
        mag = u & 0x7FFFFFFF
        return np.where(u >> 31, -mag, mag)
    u = bits.astype(np.int32)
    mag = u & 0x7FFF
    return np.where(u >> 15, -mag, mag)


def _isnan(bits: np.ndarray, dt: str) -> np.ndarray:
    if dt == "f32":
        return ((bits & 0x7F800000) == 0x7F800000) & ((bits & 0x007FFFFF) != 0)
    if dt == "bf16":
        return ((bits & 0x7F80) == 0x7F80) & ((bits & 0x007F) != 0)
    return ((bits & 0x7C00) == 0x7C00) & ((bits & 0x03FF) != 0)


def check_y(got: np.ndarray, ref: np.ndarray, dt: str, what: str = "y") -> dict:
    assert got.shape == ref.shape
    nan_g, nan_r = _isnan(got, dt), _isnan(ref, dt)
    bad_nan = np.flatnonzero(nan_g != nan_r)
    assert bad_nan.size == 0, f"{what}: NaN mismatch at {bad_nan[:8]}"
    ok = ~nan_r
    if dt == "f32":
        g = got[ok].view(np.float32).astype(np.float64)
        r = ref[ok].view(np.float32).astype(np.float64)
        inf = np.isinf(r)
        assert np.array_equal(g[inf], r[inf]), f"{what}: infinity mismatch"
        err = np.abs(g[~inf] - r[~inf])
        tol = 2e-6 + 1e-5 * np.abs(r[~inf])
        bad = np.flatnonzero(err > tol)
        assert bad.size == 0, (f"{what}: {bad.size} elements outside 2e-6 abs + 1e-5 rel, "
                               f"first {bad[:5]} got {g[~inf][bad[:5]]} ref {r[~inf][bad[:5]]}")
        return {"max_abs": float(err.max()) if err.size else 0.0,
                "exact_frac": float((got[ok] == ref[ok]).mean()) if ok.any() else 1.0}
    d = np.abs(_ordered(got[ok], dt) - _ordered(ref[ok], dt))
    bad = np.flatnonzero(d > 1)
    assert bad.size == 0, (f"{what}: {bad.size} elements differ by more than 1 ulp; first "
                           f"{bad[:5]} got {got[ok][bad[:5]]} ref {ref[ok][bad[:5]]}")
    return {"max_ulp": int(d.max()) if d.size else 0,
            "exact_frac": float((d == 0).mean()) if d.size else 1.0}


def check_exact(got: np.ndarray, ref: np.ndarray, what: str):
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    bad = np.flatnonzero(got != ref)
    assert bad.size == 0, (f"{what}: {bad.size} mismatches, first at {bad[:8]}: got "
                           f"{[hex(int(v)) for v in got[bad[:4]]]} ref "
                           f"{[hex(int(v)) for v in ref[bad[:4]]]}")


def run_case(key: str, dt: str, x_bits: np.ndarray, g_bits: np.ndarray, label: str = "",
             flags: int = 0):
    """fwd + bwd on the GPU through the C ABI vs the oracle on the same bits
    (flags: a forward kernel choice added to the table)."""
    import torch
    import paper_2202_00441_amd as P
    spec, table = golden_table(key)
    table = table.with_flags(flags)
    bits = spec["bits"]
    n = x_bits.size
    print(f"[parity] {label or key} dt={dt} n={n} bits={bits}", flush=True)
    s = np.float32([float.fromhex(h) for h in spec["s"]])
    v = np.float32([float.fromhex(h) for h in spec["v"]])
    y_ref, c_ref = O.fwd(OACT[spec["act"]], ODT[dt], bits, s, x_bits,
                         symmetric=bool(spec.get("symmetric")), threads=THREADS)
    gin_ref = O.bwd(ODT[dt], bits, v, g_bits, c_ref, threads=THREADS)

    x = upload(x_bits, dt)
    y, codes = P.fwd(table, x)
    g = upload(g_bits, dt)
    gin = P.bwd(table, g, codes)
    torch.cuda.synchronize()
    nw = P.packed_words(n, bits)
    check_exact(download_codes(codes)[:nw], c_ref, f"{label} codes")
    stats = check_y(download(y, dt), y_ref, dt, f"{label} y")
    check_exact(download(gin, dt), gin_ref, f"{label} grad_in")
    return stats
