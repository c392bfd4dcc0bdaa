"""Host-side checks of the C ABI (no GPU needed, nothing is launched).

* the library loads and exports every function include/fewbit.h declares;
* packed-word counts and status strings;
* fewbit_fit_table (host code) against the oracle's fit: same loss, same
  boundaries or their mirror image (GELU' and SiLU' are point-symmetric, so
  with a symmetric weight the mirrored partition is equally optimal);
* every argument error of fwd / bwd is returned before any launch.
"""
import ctypes as C
import json
import os
import re

import numpy as np
import pytest

import oracle as O
import paper_2202_00441_amd as P
from paper_2202_00441_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fewbit.h")
TABLES = json.load(open(os.path.join(ROOT, "tests", "golden", "tables.json")))


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(fewbit_\w+)\s*\(", src)))


def test_exports_every_declared_symbol():
    names = declared_functions()
    assert set(names) == {"fewbit_fit_table", "fewbit_packed_words", "fewbit_fwd",
                          "fewbit_fwd16_table_min", "fewbit_bwd", "fewbit_strerror"}
    raw = C.CDLL(P.LIB_PATH)
    for name in names:
        assert hasattr(raw, name), name


def test_fwd16_table_min():
    # a whole number of 512-element tiles, or "never"; per type, activation
    # and bit width; -1 for bad arguments (fp32 has no table kernel)
    never = 2 ** 63 - 1
    for dt in ("f16", "bf16"):
        for act in P.ACTS:
            for bits in (1, 2, 3, 4):
                m = P.fwd16_table_min(act, bits, dt)
                assert m == never or (m > 0 and m % 512 == 0), (act, bits, dt)
    # some entries never switch to the table kernel
    assert any(P.fwd16_table_min(a, b, d) == never
               for d in ("f16", "bf16") for a in P.ACTS for b in (1, 2, 3, 4))
    assert P.fwd16_table_min("gelu", 3, "bf16") <= 1 << 28     # the large-LM workload
    L = _lib.lib
    assert L.fewbit_fwd16_table_min(7, 3, P.BF16) == -1
    assert L.fewbit_fwd16_table_min(0, 0, P.BF16) == -1
    assert L.fewbit_fwd16_table_min(0, 5, P.BF16) == -1
    assert L.fewbit_fwd16_table_min(0, 3, P.F32) == -1
    assert L.fewbit_fwd16_table_min(0, 3, 3) == -1
    with pytest.raises(P.FewbitError):
        P.fwd16_table_min(-1, 3)


def test_kernel_choice_flags():
    # either forward kernel may be chosen in the table, not both
    A = 16
    for flags, ok in ((P.FLAG_TABLE_FWD, True), (P.FLAG_ELEMENT_FWD, True),
                      (P.FLAG_TABLE_FWD | P.FLAG_ELEMENT_FWD, False)):
        t = _table().with_flags(flags)
        # a stream of another device would be rejected after the table check,
        # so only the table checks are reached with n = 0 (a no-op when valid)
        rc = _lib.lib.fewbit_fwd(C.byref(t.c), P.BF16, A, A, A, 0, None)
        assert (rc == _lib.OK) == ok, flags
    assert _table().with_flags(P.FLAG_TABLE_FWD).flags == P.FLAG_TABLE_FWD


def test_packed_words():
    for bits in (1, 2, 3, 4):
        for n in (0, 1, 31, 32, 33, 1000, 67108863, 268435456):
            assert P.packed_words(n, bits) == (n * bits + 31) // 32 == O.packed_words(n, bits)
    assert P.packed_words(-1, 3) == -1
    # no overflow up to the largest count the type holds
    for n in (2 ** 61, 2 ** 62 + 5, 2 ** 63 - 1):
        for bits in (1, 2, 3, 4):
            assert P.packed_words(n, bits) == (n * bits + 31) // 32
    assert P.packed_words(10, 0) == -1 and P.packed_words(10, 5) == -1


def test_strerror():
    for code in range(-8, 1):
        s = P.strerror(code)
        assert s and s != "unknown status"
    assert P.strerror(-99) == "unknown status"


ORACLE_ACT = {"gelu": O.GELU, "silu": O.SILU, "sigmoid": O.SIGMOID, "tanh": O.TANH,
              "relu": O.RELU, "selu": O.SELU, "softplus": O.SOFTPLUS}


def _oracle_weight(spec):
    if spec["kind"] == "uniform":
        return O.uniform(spec["A"], spec["B"])
    if spec["kind"] == "normal":
        return O.normal(spec["A"], spec["B"], 0.0, spec["sigma"])
    return O.mixture(spec["A"], spec["B"], spec["p"], spec["sigma"], spec["sigma2"])


@pytest.mark.parametrize("key", sorted(TABLES))
def test_library_fit_matches_oracle_fit(key):
    spec = TABLES[key]
    w = spec["weight"]
    sym = bool(spec["symmetric"])
    T = P.fit_table(spec["act"], spec["bits"], P.Weight.from_spec(w), w["n_grid"], symmetric=sym)
    F = O.fit(ORACLE_ACT[spec["act"]], spec["bits"], _oracle_weight(w), w["n_grid"],
              symmetric=sym)
    assert T.flags == (P.FLAG_SYMMETRIC if sym else 0)
    assert T.loss == pytest.approx(F.loss, rel=1e-9)
    s_lib = np.float32(T.s)
    same = np.array_equal(s_lib, F.s)
    mirror = np.array_equal(s_lib, -F.s[::-1])
    assert same or mirror
    if same:
        assert np.allclose(T.v, F.v, rtol=0, atol=1e-6)
    elif spec["act"] in ("gelu", "silu"):
        # f'(-x) = 1 - f'(x): mirrored values are 1 - reversed
        assert np.allclose(T.v, 1.0 - F.v[::-1], rtol=0, atol=1e-6)
    else:
        # even f': mirrored values are the reversed ones
        assert np.allclose(T.v, F.v[::-1], rtol=0, atol=1e-6)


@pytest.mark.parametrize("key", sorted(TABLES))
def test_stored_tables_are_the_oracles_fit(key):
    # tables.json is written by tests/golden/make_tables.py from the oracle
    # alone: refitting with the oracle gives the stored bits back
    spec = TABLES[key]
    w = spec["weight"]
    F = O.fit(ORACLE_ACT[spec["act"]], spec["bits"], _oracle_weight(w), w["n_grid"],
              symmetric=bool(spec["symmetric"]))
    assert [float(x).hex() for x in F.s] == spec["s"]
    assert [float(x).hex() for x in F.v] == spec["v"]
    assert F.loss == spec["loss"]


@pytest.mark.parametrize("act,bits,sym", [("sigmoid", 3, True), ("tanh", 2, True),
                                          ("silu", 4, False), ("gelu", 1, False)])
def test_library_fit_other_cases(act, bits, sym):
    w = P.Weight(P.W_UNIFORM, -10.0, 10.0)
    T = P.fit_table(act, bits, w, 2000, symmetric=sym)
    F = O.fit(ORACLE_ACT[act], bits, O.uniform(-10.0, 10.0), 2000, symmetric=sym)
    assert T.loss == pytest.approx(F.loss, rel=1e-9)
    assert T.flags == (P.FLAG_SYMMETRIC if sym else 0)
    assert np.array_equal(np.float32(T.s), F.s) or np.array_equal(np.float32(T.s), -F.s[::-1])


@pytest.mark.parametrize("act,bits", [(a, b) for a in ("relu", "selu", "softplus")
                                      for b in (1, 2, 3, 4)])
def test_library_fit_more_activations(act, bits):
    w = P.Weight(P.W_UNIFORM, -10.0, 10.0)
    T = P.fit_table(act, bits, w, 1000)
    F = O.fit(ORACLE_ACT[act], bits, O.uniform(-10.0, 10.0), 1000)
    assert T.loss == pytest.approx(F.loss, rel=1e-9, abs=1e-12)
    assert np.all(np.diff(np.float32(T.s)) > 0)


def _paper_table1():
    rows = []
    with open(os.path.join(os.path.dirname(__file__), "golden", "table1_fit_errors.txt")) as fh:
        for line in fh:
            if line.startswith("#") or not line.strip():
                continue
            name, sym, *vals = line.split()
            for b, v in enumerate(vals, start=1):
                if v != "-":
                    rows.append((name, sym == "1", b, float(v)))
    return rows


@pytest.mark.parametrize("name,symmetric,bits,paper", _paper_table1())
def test_library_fit_reproduces_table1(name, symmetric, bits, paper):
    """The library's own fit (independent of the oracle) against the fit
    errors the paper prints in Table 1 (4 decimals): w = 1 on [-10, 10]."""
    act = "silu" if name == "swish" else name
    T = P.fit_table(act, bits, P.Weight(P.W_UNIFORM, -10.0, 10.0), 4000, symmetric=symmetric)
    assert abs(T.loss - paper) <= 1.01e-4, (T.loss, paper)


REFINE_CASES = [
    ("gelu", 3, P.Weight(P.W_UNIFORM, -10.0, 10.0), O.uniform(-10.0, 10.0), False),
    ("gelu", 4, P.Weight(P.W_NORMAL, -10.0, 10.0), O.normal(-10.0, 10.0), False),
    ("silu", 2, P.Weight(P.W_MIXTURE, -40.0, 40.0, p=0.01, sigma2=10.0),
     O.mixture(-40.0, 40.0, 0.01, 1.0, 10.0), False),
    ("sigmoid", 3, P.Weight(P.W_UNIFORM, -10.0, 10.0), O.uniform(-10.0, 10.0), True),
    ("tanh", 4, P.Weight(P.W_UNIFORM, -8.0, 8.0), O.uniform(-8.0, 8.0), True),
    ("softplus", 3, P.Weight(P.W_UNIFORM, -10.0, 10.0), O.uniform(-10.0, 10.0), False),
]


@pytest.mark.parametrize("act,bits,w,ow,sym", REFINE_CASES)
def test_library_refinement_matches_oracle(act, bits, w, ow, sym):
    n = 1000
    T = P.fit_table(act, bits, w, n, symmetric=sym, refine=True)
    D = P.fit_table(act, bits, w, n, symmetric=sym)
    R = O.fit_refined(ORACLE_ACT[act], bits, ow, n, symmetric=sym)
    assert T.flags == (P.FLAG_SYMMETRIC if sym else 0)
    assert T.loss <= D.loss
    assert T.loss == pytest.approx(R.loss, rel=1e-8)
    s = np.float64(T.s)
    # both descend to the same local optimum (or its mirror image)
    assert (np.allclose(s, R.s_double, rtol=0, atol=2e-5)
            or np.allclose(s, -R.s_double[::-1], rtol=0, atol=2e-5))


def test_library_refinement_reaches_lloyd_max_off_grid():
    # f' = x is not a library activation; the uniform source's optimum is
    # checked through GELU's symmetric structure instead: the refined 1-bit
    # GELU split on a grid without 0 returns to 0
    w = P.Weight(P.W_UNIFORM, -10.0, 10.0)
    T = P.fit_table("gelu", 1, w, 999, refine=True)
    D = P.fit_table("gelu", 1, w, 999)
    assert abs(D.s[0]) > 1e-3 and abs(T.s[0]) < 1e-5
    assert T.loss < D.loss
    assert T.loss == pytest.approx(0.1410474, abs=2e-7)


def test_parity_helpers_cover_every_activation():
    # the GPU parity helpers name the oracle's activation for every library one
    from parity import OACT
    for name, code in P.ACTS.items():
        if name == "swish":
            continue
        assert OACT[name] == code == ORACLE_ACT[name]


def test_fit_argument_errors():
    w = P.Weight(P.W_NORMAL, -10.0, 10.0)
    cases = [
        (dict(act="gelu", bits=0, weight=w, n_grid=100), _lib.E_BITS),
        (dict(act="gelu", bits=5, weight=w, n_grid=100), _lib.E_BITS),
        (dict(act=7, bits=3, weight=w, n_grid=100), _lib.E_INVALID),
        (dict(act="gelu", bits=4, weight=w, n_grid=15), _lib.E_INVALID),
        (dict(act="gelu", bits=3, weight=P.Weight(P.W_NORMAL, 1.0, -1.0), n_grid=100), _lib.E_INVALID),
        (dict(act="gelu", bits=3, weight=P.Weight(P.W_NORMAL, -1.0, 1.0, sigma=0.0), n_grid=100), _lib.E_INVALID),
        (dict(act="gelu", bits=3, weight=P.Weight(9, -1.0, 1.0), n_grid=100), _lib.E_INVALID),
        (dict(act="gelu", bits=3, weight=P.Weight(P.W_MIXTURE, -1.0, 1.0, p=1.5), n_grid=100), _lib.E_INVALID),
        (dict(act="gelu", bits=3, weight=P.Weight(P.W_UNIFORM, -1.0, float("inf")), n_grid=100), _lib.E_INVALID),
    ]
    for kw, code in cases:
        with pytest.raises(P.FewbitError) as ei:
            P.fit_table(kw["act"], kw["bits"], kw["weight"], kw["n_grid"])
        assert ei.value.status == code, kw
    ct = _lib.CTable()
    assert _lib.lib.fewbit_fit_table(0, 3, None, 100, 0, C.byref(ct)) == _lib.E_NULL
    cw = w.c()
    assert _lib.lib.fewbit_fit_table(0, 3, C.byref(cw), 100, 4, C.byref(ct)) == _lib.E_INVALID
    assert _lib.lib.fewbit_fit_table(0, 3, C.byref(cw), 100, 8, C.byref(ct)) == _lib.E_INVALID
    # grid above 2^20 cells, a reserved field set, no output
    assert _lib.lib.fewbit_fit_table(0, 3, C.byref(cw), (1 << 20) + 1, 0, C.byref(ct)) == _lib.E_INVALID
    cw.reserved = 1
    assert _lib.lib.fewbit_fit_table(0, 3, C.byref(cw), 100, 0, C.byref(ct)) == _lib.E_INVALID
    cw.reserved = 0
    assert _lib.lib.fewbit_fit_table(0, 3, C.byref(cw), 100, 0, None) == _lib.E_NULL


def _table(bits=3):
    K = 1 << bits
    s = np.linspace(-1, 1, K - 1).astype(np.float32)
    v = np.linspace(0, 1, K).astype(np.float32)
    return P.Table.from_values(P.GELU, bits, s, v)


def test_fwd_bwd_errors_before_launch():
    t = _table()
    fwd, bwd = P.fwd_raw, P.bwd_raw
    A = 0x10000          # aligned, never dereferenced: every case fails first
    # n == 0 is a no-op even with NULL pointers
    assert fwd(t, P.BF16, 0, 0, 0, 0, 0) == _lib.OK
    assert bwd(t, P.BF16, 0, 0, 0, 0, 0) == _lib.OK
    assert fwd(t, P.BF16, A, A, A, -1, 0) == _lib.E_INVALID
    assert fwd(t, 3, A, A, A, 10, 0) == _lib.E_DTYPE
    assert bwd(t, -1, A, A, A, 10, 0) == _lib.E_DTYPE
    assert fwd(t, P.F32, 0, A, A, 10, 0) == _lib.E_NULL
    assert fwd(t, P.F32, A, 0, A, 10, 0) == _lib.E_NULL
    assert fwd(t, P.F32, A, A, 0, 10, 0) == _lib.E_NULL
    assert bwd(t, P.F32, A, 0, A, 10, 0) == _lib.E_NULL
    assert fwd(t, P.F32, A + 4, A, A, 10, 0) == _lib.E_ALIGN
    assert fwd(t, P.F32, A, A + 8, A, 10, 0) == _lib.E_ALIGN
    assert fwd(t, P.F32, A, A, A + 4, 10, 0) == _lib.E_ALIGN
    assert bwd(t, P.BF16, A, A + 2, A, 10, 0) == _lib.E_ALIGN
    assert bwd(t, P.BF16, A, A, A + 2, 10, 0) == _lib.E_ALIGN
    # table errors
    bad = _table()
    bad.c.bits = 5
    assert fwd(bad, P.F32, A, A, A, 10, 0) == _lib.E_BITS
    assert bwd(bad, P.F32, A, A, A, 10, 0) == _lib.E_BITS
    bad = _table()
    bad.c.s[2], bad.c.s[3] = bad.c.s[3], bad.c.s[2]          # unsorted
    assert fwd(bad, P.F32, A, A, A, 10, 0) == _lib.E_NUMERIC
    bad = _table()
    bad.c.s[1] = float("nan")
    assert fwd(bad, P.F32, A, A, A, 10, 0) == _lib.E_NUMERIC
    bad = _table()
    bad.c.v[7] = float("inf")
    assert bwd(bad, P.F32, A, A, A, 10, 0) == _lib.E_NUMERIC
    bad = _table()
    bad.c.act = 9
    assert fwd(bad, P.F32, A, A, A, 10, 0) == _lib.E_INVALID
    bad = _table()
    bad.c.flags = 2
    assert fwd(bad, P.F32, A, A, A, 10, 0) == _lib.E_INVALID
    bad = _table()
    bad.c.reserved = 1
    assert bwd(bad, P.F32, A, A, A, 10, 0) == _lib.E_INVALID
    assert _lib.lib.fewbit_fwd(None, 0, A, A, A, 10, None) == _lib.E_NULL


def test_table_from_values_rejects_wrong_lengths():
    with pytest.raises(ValueError):
        P.Table.from_values(P.GELU, 3, [0.0] * 6, [0.0] * 8)


def test_single_hip_runtime_in_process():
    # one HIP runtime per process: the library must bind to torch's
    import torch  # noqa: F401
    paths = set()
    with open("/proc/self/maps") as fh:
        for line in fh:
            if "libamdhip64" in line:
                paths.add(os.path.realpath(line.split()[-1]))
    assert len(paths) == 1, paths
