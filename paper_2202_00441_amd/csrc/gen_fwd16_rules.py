#!/usr/bin/env python3
"""Generate fwd16_rules.h: how the 16-bit forward fills its output table.

For an fp16 / bf16 input the output of f is a function of the 16-bit input
pattern alone, so the table forward keeps the outputs of all 65536 patterns
in LDS.  Most of that table follows a simple rule: above some size GELU(x)
rounds to x itself, far on the negative side to -0, near zero to x/2; sigmoid
saturates to constants; SELU's positive side is lambda x; and so on.  Each
workgroup fills those parts by rule and evaluates f (the kernel's own fp32
f, then one rounding) only where no rule holds.

The table is cut into 512 blocks of 128 patterns (the pattern's top 9 bits:
sign and exponent for bf16; sign, exponent and 3 mantissa bits for fp16).
For every activation and 16-bit type this script evaluates f(x) for every
pattern in double precision (scipy's special functions), rounds it once to
the storage type (round to nearest even, subnormals kept), and gives each
block the first rule that reproduces all 128 rounded outputs exactly:

  IDENTITY  y = x                       (the input pattern itself)
  CONST     y = one 16-bit pattern      (the payload)
  HALF      y = RNE(x / 2)              (only in blocks where x / 2 is one
                                         exponent step down: exponent field
                                         from 2 to the largest finite one)
  SCALE     y = RNE(fl32(c x))          (c = SELU's lambda as fp32; the
                                         fp32 product, then one rounding)
  EVAL      y = the kernel's f          (no rule holds)

Consecutive blocks with the same rule form a run; a table is at most 16 runs
(start block, rule, payload), and when a table has more the shortest constant
runs are evaluated instead until it fits.  The kernel receives the runs of
its (activation, type) as kernel arguments.

The rules hold for the correctly rounded outputs; the evaluated blocks come
from the kernel's fp32 f, within one unit in the last place of them.  This
script shares nothing with the oracle: it is the library's own evaluation.

    python paper_2202_00441_amd/csrc/gen_fwd16_rules.py      # rewrites fwd16_rules.h
"""
import os
import sys

import numpy as np
from scipy.special import expit, ndtr

HERE = os.path.dirname(os.path.abspath(__file__))
OUT = os.path.join(HERE, "fwd16_rules.h")

ACTS = ["gelu", "silu", "sigmoid", "tanh", "relu", "selu", "softplus"]   # the library's order
DTYPES = ["f16", "bf16"]                                                # FEWBIT_F16, FEWBIT_BF16
MAX_RUNS = 16
IDENTITY, CONST, HALF, SCALE, EVAL = 0, 1, 2, 3, 4
RULE_NAMES = {IDENTITY: "IDENTITY", CONST: "CONST", HALF: "HALF", SCALE: "SCALE", EVAL: "EVAL"}

# SELU (Klambauer et al., 2017)
SELU_LAMBDA = 1.0507009873554804934193349852946
SELU_ALPHA = 1.6732632423543772848170429916717


def f_exact(act: str, x: np.ndarray) -> np.ndarray:
    """f in double; NaN in gives NaN out."""
    with np.errstate(all="ignore"):
        if act == "gelu":
            y = x * ndtr(x)
            y = np.where(np.isinf(x), np.where(x > 0, x, -0.0), y)
        elif act == "silu":
            y = x * expit(x)
            y = np.where(np.isinf(x), np.where(x > 0, x, -0.0), y)
        elif act == "sigmoid":
            y = expit(x)
        elif act == "tanh":
            y = np.tanh(x)
        elif act == "relu":
            y = np.where(x > 0, x, 0.0)
        elif act == "selu":
            y = np.where(x > 0, SELU_LAMBDA * x, SELU_LAMBDA * SELU_ALPHA * np.expm1(x))
        elif act == "softplus":
            y = np.where(x > 0, x + np.log1p(np.exp(-x)), np.log1p(np.exp(x)))
        else:
            raise ValueError(act)
    return np.where(np.isnan(x), x, y)


def widen(dt: str, p: np.ndarray) -> np.ndarray:
    """16-bit patterns -> double (exact)."""
    p = p.astype(np.uint32)
    if dt == "bf16":
        return (p << 16).view(np.float32).astype(np.float64)
    return p.astype(np.uint16).view(np.float16).astype(np.float64)


def round_to(dt: str, v: np.ndarray) -> np.ndarray:
    """double -> 16-bit pattern, one round to nearest even (subnormals kept,
    overflow to infinity, NaN to the canonical quiet NaN)."""
    v = np.asarray(v, np.float64)
    if dt == "f16":
        with np.errstate(all="ignore"):
            return v.astype(np.float16).view(np.uint16).astype(np.uint32)
    sign = np.signbit(v).astype(np.uint32) << 15
    a = np.abs(v)
    out = np.zeros(v.shape, np.uint32)
    with np.errstate(all="ignore"):
        m, e = np.frexp(a)                       # a = m 2^e, m in [0.5, 1)
        # quantum: 2^(e-8) for normals (8 significant bits), 2^-133 below 2^-126
        qexp = np.maximum(e - 8, -133)
        q = np.ldexp(a, -qexp)                   # exact: a / quantum
        r = np.floor(q)
        d = q - r
        up = (d > 0.5) | ((d == 0.5) & (np.fmod(r, 2.0) == 1.0))
        r = r + up
        val = np.ldexp(r, qexp)                  # exactly representable in fp32 (or inf)
        bits = (val.astype(np.float32).view(np.uint32) >> 16).astype(np.uint32)
    out = sign | bits
    out = np.where(np.isinf(a) | (val >= 2.0 ** 128), sign | 0x7F80, out)
    out = np.where(np.isnan(v), 0x7FC0, out)
    return out.astype(np.uint32)


EXP_ALL_ONES = {"bf16": 0xFF, "f16": 0x1F}


def block_exponent(dt: str, b: int) -> int:
    """Exponent field of the patterns of block b (pattern >> 7)."""
    return b & 0xFF if dt == "bf16" else (b >> 3) & 0x1F


def fl32(v: np.ndarray) -> np.ndarray:
    with np.errstate(all="ignore"):
        return v.astype(np.float32).astype(np.float64)


def block_rules(act: str, dt: str):
    pats = np.arange(65536, dtype=np.uint32)
    x = widen(dt, pats)
    y = round_to(dt, f_exact(act, x))
    half = round_to(dt, x * 0.5)
    scale = None
    if act == "selu":
        lam32 = float(np.float32(SELU_LAMBDA))
        scale = round_to(dt, fl32(x * lam32))          # exact product of two floats, then fp32
    rules = []
    for b in range(512):
        sl = slice(128 * b, 128 * b + 128)
        yy = y[sl]
        if np.array_equal(yy, pats[sl]):
            rules.append((IDENTITY, 0))
        elif np.all(yy == yy[0]):
            rules.append((CONST, int(yy[0])))
        elif np.array_equal(yy, half[sl]) and 2 <= block_exponent(dt, b) < EXP_ALL_ONES[dt]:
            rules.append((HALF, 0))
        elif scale is not None and np.array_equal(yy, scale[sl]):
            rules.append((SCALE, 0))
        else:
            rules.append((EVAL, 0))
    return rules


def runs_of(rules):
    runs = []
    for b, r in enumerate(rules):
        if not runs or runs[-1][1:] != r:
            runs.append((b,) + r)
    return runs


def fit_runs(rules):
    """Runs of the block rules, at most MAX_RUNS: while there are more, the
    shortest constant run is evaluated instead."""
    rules = list(rules)
    while True:
        runs = runs_of(rules)
        if len(runs) <= MAX_RUNS:
            return runs
        lengths = []
        for i, (start, rule, _) in enumerate(runs):
            end = runs[i + 1][0] if i + 1 < len(runs) else 512
            if rule == CONST:
                lengths.append((end - start, start, end))
        _, start, end = min(lengths)
        for b in range(start, end):
            rules[b] = (EVAL, 0)


def generate() -> str:
    lines = [
        "// fwd16_rules.h -- GENERATED by gen_fwd16_rules.py; do not edit.",
        "//",
        "// How the 16-bit forward fills its output table over all 65536 input",
        "// patterns: runs of 128-pattern blocks (pattern >> 7) and the rule each",
        "// run follows (see gen_fwd16_rules.py).  Indexed [activation][type],",
        "// activation in fewbit_act order, type 0 = fp16, 1 = bf16.",
        "#pragma once",
        "#include <cstdint>",
        "",
        "namespace fwd16_rules {",
        "",
        f"constexpr int kMaxRuns = {MAX_RUNS};",
        "enum Rule : uint32_t { "
        + ", ".join(f"{RULE_NAMES[k]} = {k}" for k in sorted(RULE_NAMES)) + " };",
        "",
        "// a run: first block (bits 0-9), rule (bits 12-15), payload pattern (bits 16-31);",
        "// unused entries start at block 1023, past every block",
        "constexpr uint32_t run(uint32_t start, Rule rule, uint32_t payload) {",
        "  return start | (static_cast<uint32_t>(rule) << 12) | (payload << 16);",
        "}",
        "",
        "constexpr uint32_t kUnused = 1023u | (static_cast<uint32_t>(EVAL) << 12);",
        "",
        "struct Runs {",
        "  int count;",
        f"  uint32_t r[{MAX_RUNS}];",
        "};",
        "",
        f"constexpr Runs kRuns[{len(ACTS)}][{len(DTYPES)}] = {{",
    ]
    stats = []
    for act in ACTS:
        lines.append(f"    {{  // {act}")
        for dt in DTYPES:
            rules = block_rules(act, dt)
            runs = fit_runs(rules)
            ev = sum(1 for i, (s, r, _) in enumerate(runs) if r == EVAL
                     for _ in range(s, runs[i + 1][0] if i + 1 < len(runs) else 512))
            stats.append((act, dt, len(runs), ev))
            body = ", ".join(f"run({s}, {RULE_NAMES[r]}, 0x{p:04x})" for s, r, p in runs)
            lines.append(f"        {{{len(runs)}, {{{body}}}}},  // {dt}: {ev} blocks evaluated")
        lines.append("    },")
    lines += ["};", "", "}  // namespace fwd16_rules", ""]
    return "\n".join(lines), stats


def main():
    text, stats = generate()
    with open(OUT, "w") as fh:
        fh.write(text)
    for act, dt, nr, ev in stats:
        print(f"{act:9s} {dt:5s} runs {nr:2d}  evaluated blocks {ev:3d}")
    print("wrote", OUT)


if __name__ == "__main__":
    sys.exit(main())
