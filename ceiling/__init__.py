"""Streaming reference kernels of the benchmark (ceiling/ceiling.hip).

stream(kind, shape, x, y, codes, tiles, bits): moves `tiles` whole 512-element
tiles with the byte mix of a copy ("copy"), of the few-bit forward ("fwd":
read x, write y and the codes) or of the backward ("bwd": read grad_out and
the codes, write grad_in), on the current stream.  Launch shapes: 64 or 256
threads per workgroup in tile order, 65 (64 threads, tiles 2p and 2p+1 on
workgroups 8 apart, i.e. on one XCD), or PERSISTENT (512: one persistent
512-thread workgroup per compute unit, the 16-bit table forward's launch
shape; not a ceiling candidate).  Used only by bench.py, to measure in the
same run what the device streams for each byte mix.
"""
import ctypes as C
import os

_SO = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libceiling.so")
if not os.path.exists(_SO):
    raise ImportError(f"{_SO} is not built: run python ceiling/build.py")
_lib = C.CDLL(_SO)
_lib.ceiling_stream.restype = C.c_int
_lib.ceiling_stream.argtypes = [C.c_int, C.c_int, C.c_int, C.c_int, C.c_void_p, C.c_void_p,
                                C.c_void_p, C.c_int64, C.c_void_p]
KINDS = {"copy": 0, "fwd": 1, "bwd": 2}


def tile_bytes(kind: str, elem_bytes: int, bits: int) -> int:
    """Bytes one tile moves (reads + writes) for the byte mix of `kind`."""
    data = 512 * elem_bytes
    return 2 * data + (0 if kind == "copy" else 64 * bits)


SHAPES = (64, 256, 65)       # the ceiling candidates
PERSISTENT = 512


def stream(kind: str, shape: int, src, dst, codes, tiles: int, bits: int) -> None:
    import torch
    rc = _lib.ceiling_stream(KINDS[kind], shape, src.element_size(), bits, src.data_ptr(),
                             dst.data_ptr(), codes.data_ptr() if codes is not None else None,
                             tiles, torch.cuda.current_stream(src.device).cuda_stream)
    if rc != 0:
        raise RuntimeError(f"ceiling_stream({kind}, {shape}) failed: {rc}")
