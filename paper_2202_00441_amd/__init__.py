"""Few-bit backward for pointwise activations on AMD MI355X (gfx950).

Drop-in activation whose backward keeps only b-bit interval indices of a
piecewise-constant approximation of f' (Novikov et al., ICML 2022; Sec. 2,
Listing 1).  The compute path is libfewbit.so (HIP kernels + C ABI in
include/fewbit.h); this package is its Python binding.
"""
from ._lib import (ACTS, BF16, DTYPES, F16, F32, FLAG_ELEMENT_FWD, FLAG_REFINE, FLAG_SYMMETRIC,
                   FLAG_TABLE_FWD, GELU, LIB_PATH, RELU, SELU,
                   SIGMOID, SILU, SOFTPLUS, TANH, W_MIXTURE, W_NORMAL, W_UNIFORM, FewbitError,
                   Table, Weight, bwd, bwd_raw, fit_table, fwd, fwd16_table_min, fwd_raw, packed_words,
                   strerror)
from .autograd import FewBitActivation, FewBitAct

__all__ = [
    "ACTS", "BF16", "DTYPES", "F16", "F32", "FLAG_ELEMENT_FWD", "FLAG_REFINE", "FLAG_SYMMETRIC",
    "FLAG_TABLE_FWD", "GELU", "LIB_PATH", "RELU", "SELU",
    "SIGMOID", "SILU", "SOFTPLUS", "TANH", "W_MIXTURE", "W_NORMAL", "W_UNIFORM", "FewbitError", "Table", "Weight",
    "bwd", "bwd_raw", "fit_table", "fwd", "fwd16_table_min", "fwd_raw", "packed_words", "strerror",
    "FewBitActivation", "FewBitAct",
]
