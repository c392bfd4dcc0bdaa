"""ctypes binding of libfewbit.so (the C ABI declared in include/fewbit.h).

Argument marshalling only: every step of the forward and backward runs in
the library's HIP kernels; PyTorch supplies device memory and the stream.
There is no fallback: if the shared library is missing or fails to load,
importing this module raises.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass
from typing import Sequence

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libfewbit.so")

# status codes, activations, storage types, weights, flags (include/fewbit.h)
OK, E_INVALID, E_NULL, E_ALIGN, E_DTYPE, E_BITS, E_NOMEM, E_NUMERIC, E_HIP = \
    0, -1, -2, -3, -4, -5, -6, -7, -8
GELU, SILU, SIGMOID, TANH, RELU, SELU, SOFTPLUS = 0, 1, 2, 3, 4, 5, 6
F32, F16, BF16 = 0, 1, 2
W_UNIFORM, W_NORMAL, W_MIXTURE = 0, 1, 2
FLAG_SYMMETRIC = 1
FLAG_REFINE = 2
FLAG_TABLE_FWD = 4        # fp16 / bf16 forward: table kernel at every size
FLAG_ELEMENT_FWD = 8      # fp16 / bf16 forward: per-element kernel at every size

ACTS = {"gelu": GELU, "silu": SILU, "swish": SILU, "sigmoid": SIGMOID, "tanh": TANH,
        "relu": RELU, "selu": SELU, "softplus": SOFTPLUS}
DTYPES = {"f32": F32, "f16": F16, "bf16": BF16}


class FewbitError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: {strerror(status)} (status {status})")
        self.status = status


class CWeight(C.Structure):
    _fields_ = [("kind", C.c_int32), ("reserved", C.c_int32), ("A", C.c_double),
                ("B", C.c_double), ("mu", C.c_double), ("sigma", C.c_double),
                ("p", C.c_double), ("sigma2", C.c_double)]


class CTable(C.Structure):
    _fields_ = [("act", C.c_int32), ("bits", C.c_int32), ("flags", C.c_int32),
                ("reserved", C.c_int32), ("s", C.c_float * 15), ("v", C.c_float * 16),
                ("loss", C.c_double)]


def _load():
    # torch ships its own HIP runtime (file libamdhip64.so, soname
    # libamdhip64.so.7).  Loading torch first makes the dynamic loader reuse
    # that runtime for libfewbit.so's libamdhip64.so.7 dependency; loading
    # libfewbit.so first would map the system runtime and torch would then
    # map a second one, and launches through the first would see no device.
    import torch  # noqa: F401
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is missing: build it with `python -m paper_2202_00441_amd.build` "
            "(there is no CPU fallback)")
    L = C.CDLL(LIB_PATH)
    i32, i64, vp = C.c_int32, C.c_int64, C.c_void_p
    L.fewbit_fit_table.restype = C.c_int
    L.fewbit_fit_table.argtypes = [i32, i32, C.POINTER(CWeight), i64, i32, C.POINTER(CTable)]
    L.fewbit_packed_words.restype = i64
    L.fewbit_packed_words.argtypes = [i64, i32]
    L.fewbit_fwd.restype = C.c_int
    L.fewbit_fwd.argtypes = [C.POINTER(CTable), i32, vp, vp, vp, i64, vp]
    L.fewbit_bwd.restype = C.c_int
    L.fewbit_bwd.argtypes = [C.POINTER(CTable), i32, vp, vp, vp, i64, vp]
    L.fewbit_fwd16_table_min.restype = i64
    L.fewbit_fwd16_table_min.argtypes = [i32, i32, i32]
    L.fewbit_strerror.restype = C.c_char_p
    L.fewbit_strerror.argtypes = [i32]
    return L


lib = _load()


def strerror(status: int) -> str:
    return lib.fewbit_strerror(int(status)).decode()


@dataclass(frozen=True)
class Weight:
    """w(x) of Eq. (3); zero outside [A, B]."""
    kind: int
    A: float
    B: float
    mu: float = 0.0
    sigma: float = 1.0
    p: float = 0.0
    sigma2: float = 1.0

    def c(self) -> CWeight:
        return CWeight(self.kind, 0, self.A, self.B, self.mu, self.sigma, self.p, self.sigma2)

    @staticmethod
    def from_spec(spec: dict) -> "Weight":
        kind = {"uniform": W_UNIFORM, "normal": W_NORMAL, "mixture": W_MIXTURE}[spec["kind"]]
        return Weight(kind, spec["A"], spec["B"], spec.get("mu", 0.0), spec.get("sigma", 1.0),
                      spec.get("p", 0.0), spec.get("sigma2", 1.0))


class Table:
    """A fitted approximation (fewbit_table): K-1 boundaries, K values."""

    def __init__(self, ct: CTable):
        self.c = ct

    @property
    def act(self) -> int:
        return self.c.act

    @property
    def bits(self) -> int:
        return self.c.bits

    @property
    def flags(self) -> int:
        return self.c.flags

    @property
    def s(self) -> list:
        return [self.c.s[i] for i in range((1 << self.bits) - 1)]

    @property
    def v(self) -> list:
        return [self.c.v[i] for i in range(1 << self.bits)]

    @property
    def loss(self) -> float:
        return self.c.loss

    def with_flags(self, flags: int) -> "Table":
        """A copy of the table with `flags` added (e.g. a forward kernel
        choice, FLAG_TABLE_FWD or FLAG_ELEMENT_FWD)."""
        ct = CTable.from_buffer_copy(self.c)
        ct.flags |= flags
        return Table(ct)

    @staticmethod
    def from_values(act: int, bits: int, s: Sequence[float], v: Sequence[float],
                    flags: int = 0, loss: float = 0.0) -> "Table":
        K = 1 << bits
        if len(s) != K - 1 or len(v) != K:
            raise ValueError("need 2^bits - 1 boundaries and 2^bits values")
        ct = CTable()
        ct.act, ct.bits, ct.flags, ct.reserved = act, bits, flags, 0
        for i in range(15):
            ct.s[i] = float(s[i]) if i < K - 1 else float("inf")
        for i in range(16):
            ct.v[i] = float(v[i]) if i < K else 0.0
        ct.loss = loss
        return Table(ct)


def fit_table(act, bits: int, weight: Weight, n_grid: int, symmetric: bool = False,
              refine: bool = False) -> Table:
    """fewbit_fit_table: the dynamic-programming fit of Sec. 3 (host), with
    refine=True followed by gradient descent on the boundaries."""
    a = ACTS[act] if isinstance(act, str) else int(act)
    ct = CTable()
    cw = weight.c()
    flags = (FLAG_SYMMETRIC if symmetric else 0) | (FLAG_REFINE if refine else 0)
    rc = lib.fewbit_fit_table(a, int(bits), C.byref(cw), int(n_grid), flags, C.byref(ct))
    if rc != OK:
        raise FewbitError(rc, "fewbit_fit_table")
    return Table(ct)


def packed_words(n: int, bits: int) -> int:
    return int(lib.fewbit_packed_words(int(n), int(bits)))


def fwd16_table_min(act, bits: int, dtype="bf16") -> int:
    """Element count from which fp16 / bf16 forwards of this activation,
    bit width and type use the table kernel (2^63 - 1: never, the
    per-element kernel runs at every size)."""
    a = ACTS[act] if isinstance(act, str) else int(act)
    d = {"f16": F16, "fp16": F16, "bf16": BF16}[dtype] if isinstance(dtype, str) else int(dtype)
    r = int(lib.fewbit_fwd16_table_min(a, int(bits), d))
    if r < 0:
        raise FewbitError(E_INVALID, "fewbit_fwd16_table_min")
    return r


# ---------------------------------------------------------------- raw pointers
def fwd_raw(table: Table, dtype: int, x: int, y: int, codes: int, n: int, stream: int) -> int:
    return lib.fewbit_fwd(C.byref(table.c), dtype, x, y, codes, n, stream)


def bwd_raw(table: Table, dtype: int, g: int, codes: int, gin: int, n: int, stream: int) -> int:
    return lib.fewbit_bwd(C.byref(table.c), dtype, g, codes, gin, n, stream)


# ---------------------------------------------------------------- torch tensors
def _dtype_code(t) -> int:
    import torch
    m = {torch.float32: F32, torch.float16: F16, torch.bfloat16: BF16}
    if t.dtype not in m:
        raise TypeError(f"unsupported dtype {t.dtype}")
    return m[t.dtype]


def _stream(dev) -> int:
    import torch
    return torch.cuda.current_stream(dev).cuda_stream


def _check_like(name: str, t, ref, n: int) -> None:
    """t must be a contiguous device tensor on ref's device with ref's dtype
    and n elements (an output the caller passes in)."""
    if not t.is_cuda or t.device != ref.device:
        raise ValueError(f"{name} must be a device tensor on {ref.device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.dtype != ref.dtype:
        raise ValueError(f"{name} must have dtype {ref.dtype}, not {t.dtype}")
    if t.numel() != n:
        raise ValueError(f"{name} must have {n} elements, not {t.numel()}")


def _check_codes(codes, ref, n: int, bits: int) -> None:
    """codes must be a contiguous device tensor of 4-byte words on ref's
    device holding at least packed_words(n, bits) words."""
    if not codes.is_cuda or codes.device != ref.device:
        raise ValueError(f"codes must be a device tensor on {ref.device}")
    if not codes.is_contiguous():
        raise ValueError("codes must be contiguous")
    if codes.element_size() != 4 or codes.is_floating_point():
        raise ValueError(f"codes must hold 4-byte integer words, not {codes.dtype}")
    need = packed_words(n, bits)
    if codes.numel() < need:
        raise ValueError(f"codes holds {codes.numel()} words, {need} are needed")


def fwd(table: Table, x, y=None, codes=None):
    """y = f(x) and the packed interval indices (Listing 1, forward).

    x: contiguous CUDA tensor (fp32 / fp16 / bf16).  Returns (y, codes) with
    codes a uint32-sized int32 tensor of packed_words(x.numel(), bits) words.
    y and codes may be passed in; they are checked (device, layout, dtype,
    size) before the call, so a wrong buffer raises instead of reaching the
    kernels.
    """
    import torch
    if not x.is_cuda or not x.is_contiguous():
        raise ValueError("x must be a contiguous device tensor")
    dt = _dtype_code(x)
    n = x.numel()
    if y is None:
        y = torch.empty_like(x)
    else:
        _check_like("y", y, x, n)
    if codes is None:
        codes = torch.empty(max(packed_words(n, table.bits), 1), dtype=torch.int32,
                            device=x.device)
    else:
        _check_codes(codes, x, n, table.bits)
    with torch.cuda.device(x.device):
        rc = fwd_raw(table, dt, x.data_ptr(), y.data_ptr(), codes.data_ptr(), n,
                     _stream(x.device))
    if rc != OK:
        raise FewbitError(rc, "fewbit_fwd")
    return y, codes


def bwd(table: Table, grad_out, codes, grad_in=None):
    """grad_in = grad_out * v[idx] (Eq. (1) with the approximation of f').

    codes must hold at least packed_words(grad_out.numel(), bits) words on
    grad_out's device; codes and grad_in (if passed) are checked before the
    call."""
    import torch
    if not grad_out.is_cuda or not grad_out.is_contiguous():
        raise ValueError("grad_out must be a contiguous device tensor")
    dt = _dtype_code(grad_out)
    n = grad_out.numel()
    _check_codes(codes, grad_out, n, table.bits)
    if grad_in is None:
        grad_in = torch.empty_like(grad_out)
    else:
        _check_like("grad_in", grad_in, grad_out, n)
    with torch.cuda.device(grad_out.device):
        rc = bwd_raw(table, dt, grad_out.data_ptr(), codes.data_ptr(),
                     grad_in.data_ptr(), n, _stream(grad_out.device))
    if rc != OK:
        raise FewbitError(rc, "fewbit_bwd")
    return grad_in
