"""The Python binding rejects wrong output and code buffers before any call.

fwd() and bwd() check every buffer the caller passes in (device, layout,
dtype, size, and for the code buffer the word size and the word count
packed_words(n, bits)), so a short, mistyped, strided or wrong-device buffer
raises ValueError instead of reaching the kernels.  The checks use only a
tensor's attributes, so the tests run on the CPU with stand-in objects that
describe device tensors; each case raises before anything is launched.
"""
import pytest
import torch

import paper_2202_00441_amd as P
from paper_2202_00441_amd import _lib

DEV0, DEV1 = torch.device("cuda:0"), torch.device("cuda:1")


class Fake:
    """Attributes of a device tensor, nothing more."""

    def __init__(self, n, dtype, device=DEV0, contiguous=True, cuda=True):
        self._n, self.dtype, self.device = n, dtype, device
        self._contig, self.is_cuda = contiguous, cuda

    def numel(self):
        return self._n

    def is_contiguous(self):
        return self._contig

    def element_size(self):
        return torch.empty(0, dtype=self.dtype).element_size()

    def is_floating_point(self):
        return self.dtype.is_floating_point

    def data_ptr(self):
        raise AssertionError("a rejected call must not reach the library")


def _table(bits):
    ct = _lib.CTable()
    ct.act, ct.bits = 0, bits
    return P.Table(ct)


TABLE = _table(3)

N = 1000
WORDS = P.packed_words(N, 3)


def _fwd(y=None, codes=None, x=None):
    x = x or Fake(N, torch.bfloat16)
    return _lib.fwd(TABLE, x, y if y is not None else Fake(N, torch.bfloat16),
                    codes if codes is not None else Fake(WORDS, torch.int32))


def _bwd(codes=None, gin=None):
    g = Fake(N, torch.bfloat16)
    return _lib.bwd(TABLE, g, codes if codes is not None else Fake(WORDS, torch.int32),
                    gin if gin is not None else Fake(N, torch.bfloat16))


@pytest.mark.parametrize("y", [
    Fake(N, torch.float16),                      # wrong dtype
    Fake(N - 1, torch.bfloat16),                 # short
    Fake(N + 1, torch.bfloat16),                 # long
    Fake(N, torch.bfloat16, contiguous=False),   # strided
    Fake(N, torch.bfloat16, device=DEV1),        # other device
    Fake(N, torch.bfloat16, cuda=False),         # host memory
])
def test_fwd_rejects_bad_y(y):
    with pytest.raises(ValueError):
        _fwd(y=y)


@pytest.mark.parametrize("codes", [
    Fake(WORDS - 1, torch.int32),                # one word short
    Fake(WORDS, torch.int16),                    # 2-byte words
    Fake(WORDS, torch.float32),                  # floats
    Fake(WORDS, torch.int32, contiguous=False),
    Fake(WORDS, torch.int32, device=DEV1),
    Fake(WORDS, torch.int32, cuda=False),
])
def test_fwd_and_bwd_reject_bad_codes(codes):
    with pytest.raises(ValueError):
        _fwd(codes=codes)
    with pytest.raises(ValueError):
        _bwd(codes=codes)


@pytest.mark.parametrize("gin", [
    Fake(N, torch.float32),
    Fake(N - 3, torch.bfloat16),
    Fake(N, torch.bfloat16, contiguous=False),
    Fake(N, torch.bfloat16, device=DEV1),
])
def test_bwd_rejects_bad_grad_in(gin):
    with pytest.raises(ValueError):
        _bwd(gin=gin)


def test_rejects_strided_or_host_input():
    with pytest.raises(ValueError):
        _fwd(x=Fake(N, torch.bfloat16, contiguous=False))
    with pytest.raises(ValueError):
        _fwd(x=Fake(N, torch.bfloat16, cuda=False))


def test_code_words_needed_follow_the_bit_width():
    # a buffer sized for 3 bits is too short for 4
    with pytest.raises(ValueError):
        _lib.fwd(_table(4), Fake(N, torch.bfloat16), Fake(N, torch.bfloat16),
                 Fake(WORDS, torch.int32))
    assert P.packed_words(N, 4) > WORDS
