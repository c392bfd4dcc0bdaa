"""CPU oracle for the few-bit activation path (test infrastructure only).

This package wraps ``oracle/liboracle.so`` (plain C, IEEE double, built from
``oracle/oracle.c`` by ``oracle/build.py``).  Only the test suite, the smoke
check in ``__graft_entry__`` and the CPU-baseline leg of ``bench.py`` may
import it.  The product library and its Python binding never do.

Every function here is argument marshalling around the C code; the paper
passages each C function follows are listed at the top of ``oracle.c``.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "liboracle.so")

GELU, SILU, SIGMOID, TANH, RELU, SELU, SOFTPLUS, HALFSQ = range(8)
F32, F16, BF16 = 0, 1, 2
W_UNIFORM, W_NORMAL, W_MIXTURE = 0, 1, 2

ACT_NAMES = {"gelu": GELU, "silu": SILU, "swish": SILU, "sigmoid": SIGMOID,
             "tanh": TANH, "relu": RELU, "selu": SELU, "softplus": SOFTPLUS,
             "halfsq": HALFSQ}
DTYPE_NAMES = {"f32": F32, "fp32": F32, "float32": F32, "f16": F16, "fp16": F16,
               "float16": F16, "bf16": BF16, "bfloat16": BF16}


class _Weight(C.Structure):
    _fields_ = [("kind", C.c_int32), ("pad", C.c_int32), ("A", C.c_double),
                ("B", C.c_double), ("mu", C.c_double), ("sigma", C.c_double),
                ("p", C.c_double), ("sigma2", C.c_double)]


@dataclass(frozen=True)
class Weight:
    """w(x) of Eq. (3): uniform (w = 1) or a normal / normal-mixture density,
    zero outside [A, B]."""
    kind: int
    A: float
    B: float
    mu: float = 0.0
    sigma: float = 1.0
    p: float = 0.0
    sigma2: float = 1.0

    def _c(self) -> _Weight:
        return _Weight(self.kind, 0, self.A, self.B, self.mu, self.sigma, self.p,
                       self.sigma2)


def uniform(A: float, B: float) -> Weight:
    return Weight(W_UNIFORM, A, B)


def normal(A: float, B: float, mu: float = 0.0, sigma: float = 1.0) -> Weight:
    return Weight(W_NORMAL, A, B, mu, sigma)


def mixture(A: float, B: float, p: float, sigma: float, sigma2: float,
            mu: float = 0.0) -> Weight:
    return Weight(W_MIXTURE, A, B, mu, sigma, p, sigma2)


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_SO):
            from . import build as _b
            _b.build()
        L = C.CDLL(_SO)
        d, i64, i32 = C.c_double, C.c_int64, C.c_int
        vp = C.c_void_p
        L.oracle_f.restype = d
        L.oracle_f.argtypes = [i32, d]
        L.oracle_df.restype = d
        L.oracle_df.argtypes = [i32, d]
        L.oracle_prefix.restype = i32
        L.oracle_prefix.argtypes = [i32, C.POINTER(_Weight), i64, vp, vp, vp]
        L.oracle_interval_cost.restype = d
        L.oracle_interval_cost.argtypes = [vp, vp, vp, i64, i64, i32, d, d]
        L.oracle_loss_at.restype = i32
        L.oracle_loss_at.argtypes = [i32, i32, C.POINTER(_Weight), i64, i32, vp, vp, vp, vp]
        L.oracle_fit_refined.restype = i32
        L.oracle_fit_refined.argtypes = [i32, i32, C.POINTER(_Weight), i64, i32, i32, vp, vp,
                                         vp, vp, vp, vp, vp]
        L.oracle_fit.restype = i32
        L.oracle_fit.argtypes = [i32, i32, C.POINTER(_Weight), i64, i32, vp, vp,
                                 C.POINTER(d), vp, vp, vp]
        L.oracle_double_to_bf16.restype = C.c_uint16
        L.oracle_double_to_bf16.argtypes = [d]
        L.oracle_double_to_f16.restype = C.c_uint16
        L.oracle_double_to_f16.argtypes = [d]
        L.oracle_double_to_f32.restype = C.c_uint32
        L.oracle_double_to_f32.argtypes = [d]
        L.oracle_bf16_to_double.restype = d
        L.oracle_bf16_to_double.argtypes = [C.c_uint16]
        L.oracle_f16_to_double.restype = d
        L.oracle_f16_to_double.argtypes = [C.c_uint16]
        L.oracle_classify.restype = i32
        L.oracle_classify.argtypes = [d, vp, i32, i32]
        L.oracle_packed_words.restype = i64
        L.oracle_packed_words.argtypes = [i64, i32]
        L.oracle_pack.restype = None
        L.oracle_pack.argtypes = [vp, i64, i32, vp]
        L.oracle_unpack.restype = None
        L.oracle_unpack.argtypes = [vp, i64, i32, vp]
        L.oracle_fwd.restype = i32
        L.oracle_fwd.argtypes = [i32, i32, i32, i32, vp, vp, vp, vp, vp, i64]
        L.oracle_bwd.restype = i32
        L.oracle_bwd.argtypes = [i32, i32, vp, vp, vp, vp, i64]
        L.oracle_fwd_mt.restype = i32
        L.oracle_fwd_mt.argtypes = [i32, i32, i32, i32, vp, vp, vp, vp, i64, i32]
        L.oracle_bwd_mt.restype = i32
        L.oracle_bwd_mt.argtypes = [i32, i32, vp, vp, vp, vp, i64, i32]
        L.oracle_round_array.restype = None
        L.oracle_round_array.argtypes = [i32, vp, vp, i64]
        L.oracle_widen_array.restype = None
        L.oracle_widen_array.argtypes = [i32, vp, vp, i64]
        _lib = L
    return _lib


def _ptr(a: np.ndarray) -> int:
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data


# ---------------------------------------------------------------- scalars
def f(act: int, x: float) -> float:
    return lib().oracle_f(act, float(x))


def df(act: int, x: float) -> float:
    return lib().oracle_df(act, float(x))


def to_bf16(x: float) -> int:
    return lib().oracle_double_to_bf16(float(x))


def to_f16(x: float) -> int:
    return lib().oracle_double_to_f16(float(x))


def to_f32(x: float) -> int:
    return lib().oracle_double_to_f32(float(x))


def from_bf16(h: int) -> float:
    return lib().oracle_bf16_to_double(int(h))


def from_f16(h: int) -> float:
    return lib().oracle_f16_to_double(int(h))


def round_array(dtype: int, x) -> np.ndarray:
    """double -> storage bits of dtype (one round-to-nearest-even)."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    out = np.zeros(max(x.size, 1), _STORE[dtype])
    lib().oracle_round_array(dtype, _ptr(x), _ptr(out), x.size)
    return out[:x.size]


def widen_array(dtype: int, bits) -> np.ndarray:
    """storage bits of dtype -> double (exact)."""
    bits = np.ascontiguousarray(bits, dtype=_STORE[dtype])
    out = np.zeros(max(bits.size, 1), np.float64)
    lib().oracle_widen_array(dtype, _ptr(bits), _ptr(out), bits.size)
    return out[:bits.size]


# ---------------------------------------------------------------- fit
def prefix(act: int, w: Weight, n: int):
    """W, FW, F2 prefix integrals on the uniform n-cell grid over [A, B]."""
    W = np.zeros(n + 1)
    FW = np.zeros(n + 1)
    F2 = np.zeros(n + 1)
    cw = w._c()
    rc = lib().oracle_prefix(act, C.byref(cw), n, _ptr(W), _ptr(FW), _ptr(F2))
    assert rc == 0
    return W, FW, F2


def interval_cost(W, FW, F2, j: int, i: int, act: int, tj: float, ti: float) -> float:
    return lib().oracle_interval_cost(_ptr(W), _ptr(FW), _ptr(F2), j, i, act, tj, ti)


@dataclass
class Fit:
    act: int
    bits: int
    symmetric: bool
    s: np.ndarray        # float32[K-1] interior boundaries
    v: np.ndarray        # float32[K] values
    loss: float          # DP(n, K) (doubled for the symmetric fit)
    cuts: np.ndarray     # int64[K+1] grid indices of the cut points
    dp_last: np.ndarray  # DP(n, k), k = 1..K
    v_double: np.ndarray


def fit(act: int, bits: int, w: Weight, n: int, symmetric: bool = False) -> Fit:
    """Optimal piecewise-constant fit of f' by the dynamic programme."""
    K = 1 << bits
    s = np.zeros(K - 1, np.float32)
    v = np.zeros(K, np.float32)
    cuts = np.zeros(K + 1, np.int64)
    dpl = np.zeros(K)
    vd = np.zeros(K)
    loss = C.c_double(0.0)
    cw = w._c()
    rc = lib().oracle_fit(act, bits, C.byref(cw), n, int(symmetric), _ptr(s),
                          _ptr(v), C.byref(loss), _ptr(cuts), _ptr(dpl), _ptr(vd))
    if rc != 0:
        raise ValueError(f"oracle_fit failed rc={rc}")
    return Fit(act, bits, symmetric, s, v, loss.value, cuts, dpl, vd)


def loss_at(act: int, bits: int, w: Weight, n: int, s, symmetric: bool = False):
    """(L, y, dL/ds) of Eq. (3) at interior boundaries s (double), Sec. 3."""
    K = 1 << bits
    sd = np.ascontiguousarray(s, dtype=np.float64)
    assert sd.size == K - 1
    y = np.zeros(K)
    g = np.zeros(K - 1)
    loss = C.c_double(0.0)
    cw = w._c()
    rc = lib().oracle_loss_at(act, bits, C.byref(cw), n, int(symmetric), _ptr(sd), _ptr(y),
                              _ptr(g), C.byref(loss))
    if rc != 0:
        raise ValueError(f"oracle_loss_at failed rc={rc}")
    return loss.value, y, g


@dataclass
class RefinedFit:
    act: int
    bits: int
    symmetric: bool
    s: np.ndarray        # fp32 boundaries after refinement
    v: np.ndarray        # fp32 values
    s_double: np.ndarray
    v_double: np.ndarray
    loss: float          # L after refinement (doubled for the symmetric fit)
    loss_dp: float       # L of the DP starting point
    iters: int


def fit_refined(act: int, bits: int, w: Weight, n: int, symmetric: bool = False,
                max_iter: int = 5000) -> RefinedFit:
    """The DP fit, then gradient descent on the boundaries (Sec. 3)."""
    K = 1 << bits
    s = np.zeros(K - 1, np.float32)
    v = np.zeros(K, np.float32)
    sd = np.zeros(K - 1)
    vd = np.zeros(K)
    loss = C.c_double(0.0)
    loss_dp = C.c_double(0.0)
    iters = C.c_int(0)
    cw = w._c()
    rc = lib().oracle_fit_refined(act, bits, C.byref(cw), n, int(symmetric), max_iter, _ptr(s),
                                  _ptr(v), _ptr(sd), _ptr(vd), C.byref(loss), C.byref(loss_dp),
                                  C.byref(iters))
    if rc != 0:
        raise ValueError(f"oracle_fit_refined failed rc={rc}")
    return RefinedFit(act, bits, symmetric, s, v, sd, vd, loss.value, loss_dp.value, iters.value)


# ---------------------------------------------------------------- codes
def packed_words(n: int, bits: int) -> int:
    return lib().oracle_packed_words(n, bits)


def pack(idx: np.ndarray, bits: int) -> np.ndarray:
    idx = np.ascontiguousarray(idx, dtype=np.uint8)
    out = np.zeros(max(packed_words(idx.size, bits), 1), np.uint32)
    lib().oracle_pack(_ptr(idx), idx.size, bits, _ptr(out))
    return out[:packed_words(idx.size, bits)]


def unpack(words: np.ndarray, n: int, bits: int) -> np.ndarray:
    words = np.ascontiguousarray(words, dtype=np.uint32)
    assert words.size >= packed_words(n, bits)
    out = np.zeros(max(n, 1), np.uint8)
    lib().oracle_unpack(_ptr(words) if words.size else 0, n, bits, _ptr(out))
    return out[:n]


def classify(x: float, s: np.ndarray, bits: int, symmetric: bool = False) -> int:
    s = np.ascontiguousarray(s, dtype=np.float32)
    return lib().oracle_classify(float(x), _ptr(s), bits, int(symmetric))


_STORE = {F32: np.uint32, F16: np.uint16, BF16: np.uint16}


def fwd(act: int, dtype: int, bits: int, s: np.ndarray, x_bits: np.ndarray,
        symmetric: bool = False, threads: int = 1, want_idx: bool = False):
    """Forward of Listing 1 on raw storage bits.

    x_bits: uint32 (fp32) or uint16 (fp16 / bf16) bit patterns.
    Returns (y_bits, codes[, idx]) with the same storage type for y.
    """
    x_bits = np.ascontiguousarray(x_bits, dtype=_STORE[dtype])
    n = x_bits.size
    s = np.ascontiguousarray(s, dtype=np.float32)
    y = np.zeros(max(n, 1), _STORE[dtype])
    codes = np.zeros(max(packed_words(n, bits), 1), np.uint32)
    xp = _ptr(x_bits) if n else _ptr(y)
    if want_idx or threads <= 1:
        idx = np.zeros(max(n, 1), np.uint8)
        rc = lib().oracle_fwd(act, dtype, bits, int(symmetric), _ptr(s), xp, _ptr(y),
                              _ptr(codes), _ptr(idx), n)
    else:
        idx = None
        rc = lib().oracle_fwd_mt(act, dtype, bits, int(symmetric), _ptr(s), xp,
                                 _ptr(y), _ptr(codes), n, threads)
    assert rc == 0
    out = (y[:n], codes[:packed_words(n, bits)])
    if want_idx:
        return out + (idx[:n],)
    return out


def bwd(dtype: int, bits: int, v: np.ndarray, g_bits: np.ndarray, codes: np.ndarray,
        threads: int = 1) -> np.ndarray:
    """Backward of Listing 1 / Eq. (1) on raw storage bits."""
    g_bits = np.ascontiguousarray(g_bits, dtype=_STORE[dtype])
    n = g_bits.size
    v = np.ascontiguousarray(v, dtype=np.float32)
    codes = np.ascontiguousarray(codes, dtype=np.uint32)
    assert codes.size >= packed_words(n, bits)
    gin = np.zeros(max(n, 1), _STORE[dtype])
    if n == 0:
        return gin[:0]
    if threads <= 1:
        rc = lib().oracle_bwd(dtype, bits, _ptr(v), _ptr(g_bits), _ptr(codes),
                              _ptr(gin), n)
    else:
        rc = lib().oracle_bwd_mt(dtype, bits, _ptr(v), _ptr(g_bits), _ptr(codes),
                                 _ptr(gin), n, threads)
    assert rc == 0
    return gin[:n]
