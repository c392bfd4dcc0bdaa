"""Pins for the oracle's storage conversions, classification, packing and the
forward / backward passes of Listing 1.

* conversions: fp32 -> bf16 against torch's CPU conversion and fp32 -> fp16
  against numpy, over a broad sample of fp32 bit patterns (every bf16-relevant
  high half with the rounding-critical low halves), all 2^16 half patterns
  decoded, and direct double -> half rounding against exact rational
  arithmetic;
* classification against numpy.searchsorted(side="right") and at the
  boundaries themselves (half-open bins);
* packing against hand-worked bit vectors and round trips;
* forward / backward against independent numpy / scipy / torch computations.
"""
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch
from scipy import special

import oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ------------------------------------------------------------------ conversions
def _fp32_sample():
    hi = np.arange(1 << 16, dtype=np.uint32) << 16
    lows = np.array([0x0000, 0x0001, 0x7FFF, 0x8000, 0x8001, 0xFFFF, 0x1234, 0xC000],
                    dtype=np.uint32)
    pats = (hi[:, None] | lows[None, :]).ravel()
    rng = np.random.default_rng(1)
    return np.concatenate([pats, rng.integers(0, 1 << 32, 1 << 20, dtype=np.uint64)
                           .astype(np.uint32)])


def test_fp32_to_bf16_matches_torch():
    pats = _fp32_sample()
    f = pats.view(np.float32)
    ours = O.round_array(O.BF16, f.astype(np.float64))
    ref = torch.from_numpy(f.copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    nan = np.isnan(f)
    assert np.array_equal(ours[~nan], ref[~nan])
    # NaN stays NaN (quiet, sign kept)
    o = ours[nan]
    assert np.all((o & 0x7F80) == 0x7F80) and np.all((o & 0x7F) != 0)


def test_fp32_to_f16_matches_numpy():
    pats = _fp32_sample()
    f = pats.view(np.float32)
    ours = O.round_array(O.F16, f.astype(np.float64))
    with np.errstate(over="ignore", invalid="ignore"):
        ref = f.astype(np.float16).view(np.uint16)
    nan = np.isnan(f)
    assert np.array_equal(ours[~nan], ref[~nan])
    o = ours[nan]
    assert np.all((o & 0x7C00) == 0x7C00) and np.all((o & 0x3FF) != 0)


def test_fp32_roundtrip_identity():
    pats = _fp32_sample()
    f = pats.view(np.float32)
    ours = O.round_array(O.F32, f.astype(np.float64))
    nan = np.isnan(f)
    assert np.array_equal(ours[~nan], pats[~nan])


def test_half_decode_exhaustive():
    h = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    d16 = O.widen_array(O.F16, h)
    ref16 = h.view(np.float16).astype(np.float64)
    dbf = O.widen_array(O.BF16, h)
    refbf = torch.from_numpy(h.view(np.int16).copy()).view(torch.bfloat16).to(torch.float64).numpy()
    for d, r in ((d16, ref16), (dbf, refbf)):
        nan = np.isnan(r)
        assert np.array_equal(np.isnan(d), nan)
        assert np.array_equal(d[~nan], r[~nan])
        assert np.array_equal(np.signbit(d[~nan]), np.signbit(r[~nan]))


def _exact_round(x: float, p: int, emin: int, vmax: float) -> float:
    """Exact round-to-nearest-even of a double with rational arithmetic."""
    a = Fraction(abs(x))
    if a == 0:
        return 0.0
    e = math.floor(math.log2(abs(x)))
    if Fraction(2) ** e > a:
        e -= 1
    if Fraction(2) ** (e + 1) <= a:
        e += 1
    e = max(e, emin)
    q = Fraction(2) ** (e - p)
    m = a / q
    fl = math.floor(m)
    r = m - fl
    k = fl + (1 if (r > Fraction(1, 2) or (r == Fraction(1, 2) and fl % 2 == 1)) else 0)
    v = k * q
    if v > Fraction(vmax):
        return math.inf
    return float(v)


@pytest.mark.parametrize("dtype,p,emin,vmax", [(O.BF16, 7, -126, 255 * 2.0 ** 120),
                                               (O.F16, 10, -14, 65504.0)])
def test_double_to_half_single_rounding(dtype, p, emin, vmax):
    rng = np.random.default_rng(2)
    # doubles near ties: representable midpoints +- tiny offsets, and randoms
    base = rng.uniform(-1, 1, 4000) * np.exp2(rng.integers(-150 if dtype == O.BF16 else -26,
                                                            16, 4000))
    xs = list(base)
    for b in base[:500]:
        if b == 0:
            continue
        e = max(math.floor(math.log2(abs(b))), emin)
        q = 2.0 ** (e - p)
        mid = (math.floor(abs(b) / q) + 0.5) * q
        for d in (0.0, 1e-9, -1e-9):
            xs.append(math.copysign(mid * (1 + d), b))
    xs = np.array(xs)
    ours = O.round_array(dtype, xs)
    dec = O.widen_array(dtype, ours)
    for x, got in zip(xs, dec):
        ref = _exact_round(float(x), p, emin, vmax)
        assert abs(got) == ref, (x, got, ref)
        if got != 0:
            assert math.copysign(1, got) == math.copysign(1, x)


# ------------------------------------------------------------------ classify
def test_classify_matches_searchsorted():
    F = O.fit(O.GELU, 3, O.normal(-10.0, 10.0), 800)
    rng = np.random.default_rng(3)
    x = np.concatenate([rng.normal(0, 1.5, 5000), F.s.astype(np.float64),
                        np.nextafter(F.s, -np.inf).astype(np.float64),
                        np.nextafter(F.s, np.inf).astype(np.float64)])
    ref = np.searchsorted(F.s.astype(np.float64), x, side="right")
    got = np.array([O.classify(v, F.s, 3) for v in x])
    assert np.array_equal(got, ref)


def test_classify_boundary_semantics():
    s = np.float32([-1.5, -0.25, 0.0, 0.25, 0.5, 1.0, 2.0])
    for m, sm in enumerate(s):
        assert O.classify(float(sm), s, 3) == m + 1                    # upper bin
        below = float(np.nextafter(sm, np.float32(-np.inf)))
        assert O.classify(below, s, 3) == m                            # lower bin
    assert O.classify(-0.0, s, 3) == 3                                 # -0 == +0
    assert O.classify(-1e-45, s, 3) == 2                               # denormal, not flushed
    assert O.classify(math.nan, s, 3) == 0
    assert O.classify(math.inf, s, 3) == 7
    assert O.classify(-math.inf, s, 3) == 0
    # symmetric: bins of |x|
    ss = np.float32([0.5, 1.0, 2.0])
    assert O.classify(-0.75, ss, 2, symmetric=True) == 1
    assert O.classify(-3.0, ss, 2, symmetric=True) == 3


# ------------------------------------------------------------------ packing
def _read_pack_vectors():
    out = []
    with open(os.path.join(GOLDEN, "pack_vectors.txt")) as fh:
        for line in fh:
            line = line.split("#")[0].strip()
            if not line:
                continue
            b, codes, words = [p.strip() for p in line.split("|")]
            out.append((int(b), [int(c) for c in codes.split()],
                        [int(w, 16) for w in words.split()]))
    return out


@pytest.mark.parametrize("bits,codes,words", _read_pack_vectors())
def test_pack_hand_vectors(bits, codes, words):
    got = O.pack(np.array(codes, np.uint8), bits)
    assert got.tolist() == words
    assert O.unpack(got, len(codes), bits).tolist() == codes


@pytest.mark.parametrize("bits", [1, 2, 3, 4])
def test_pack_roundtrip_and_word_count(bits):
    rng = np.random.default_rng(bits)
    for n in list(range(0, 258)) + [4099, 100003]:
        idx = rng.integers(0, 1 << bits, n).astype(np.uint8)
        w = O.pack(idx, bits)
        assert w.size == (n * bits + 31) // 32
        assert np.array_equal(O.unpack(w, n, bits), idx)
        if n * bits % 32:
            assert int(w[-1]) >> (n * bits % 32) == 0       # padding bits zero


@pytest.mark.parametrize("bits", [1, 2, 3, 4])
def test_pack_chunk_invariance(bits):
    rng = np.random.default_rng(10 + bits)
    idx = rng.integers(0, 1 << bits, 32 * 37 + 5).astype(np.uint8)
    whole = O.pack(idx, bits)
    parts = np.concatenate([O.pack(idx[i:i + 32 * 5], bits) for i in range(0, idx.size, 32 * 5)])
    assert np.array_equal(whole, parts)


# ------------------------------------------------------------------ fwd / bwd
def _bf16_bits(a: np.ndarray) -> np.ndarray:
    return torch.from_numpy(a.astype(np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def _bf16_val(bits: np.ndarray) -> np.ndarray:
    return torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).to(torch.float64).numpy()


def test_forward_fp32_against_scipy():
    rng = np.random.default_rng(4)
    x = rng.normal(0, 3, 20000).astype(np.float32)
    F = O.fit(O.GELU, 3, O.normal(-10.0, 10.0), 800)
    y, codes, idx = O.fwd(O.GELU, O.F32, 3, F.s, x.view(np.uint32), want_idx=True)
    xd = x.astype(np.float64)
    ref = (xd * special.ndtr(xd)).astype(np.float32)
    yv = y.view(np.float32)
    ulp = np.abs(yv.view(np.int32).astype(np.int64) - ref.view(np.int32).astype(np.int64))
    assert ulp.max() <= 1 and (ulp == 0).mean() > 0.999
    assert np.array_equal(idx, np.searchsorted(F.s.astype(np.float64), xd, side="right"))
    assert np.array_equal(codes, O.pack(idx, 3))


@pytest.mark.parametrize("act,ref", [
    (O.SILU, lambda x: x * special.expit(x)),
    (O.SIGMOID, special.expit),
    (O.TANH, np.tanh),
])
def test_forward_other_acts_fp32(act, ref):
    rng = np.random.default_rng(5)
    x = rng.uniform(-8, 8, 20000).astype(np.float32)
    F = O.fit(act, 2, O.uniform(-8.0, 8.0), 400)
    y, _ = O.fwd(act, O.F32, 2, F.s, x.view(np.uint32))
    r = ref(x.astype(np.float64)).astype(np.float32)
    ulp = np.abs(y.view(np.int32).astype(np.int64) - r.view(np.int32).astype(np.int64))
    assert ulp.max() <= 1


def test_forward_bf16_single_rounding():
    rng = np.random.default_rng(6)
    xb = _bf16_bits(rng.normal(0, 1.5, 20000))
    F = O.fit(O.GELU, 3, O.normal(-15.0, 15.0, sigma=1.5), 600)
    y, codes, idx = O.fwd(O.GELU, O.BF16, 3, F.s, xb, want_idx=True)
    xd = _bf16_val(xb)
    exact = xd * special.ndtr(xd)
    # the bf16 result is one of the two neighbours of the exact value, the nearer
    yd = _bf16_val(y)
    lo = np.minimum(yd, exact)
    assert np.all(np.abs(yd - exact) <= np.abs(exact) * 2.0 ** -8 + 1e-45)
    assert np.array_equal(idx, np.searchsorted(F.s.astype(np.float64), xd, side="right"))


@pytest.mark.parametrize("dtype", [O.F32, O.F16, O.BF16])
def test_backward_against_numpy(dtype):
    rng = np.random.default_rng(7)
    n = 5001
    bits = 3
    v = np.float32(rng.normal(0.5, 0.4, 8))
    idx = rng.integers(0, 8, n).astype(np.uint8)
    codes = O.pack(idx, bits)
    g32 = np.float32(rng.normal(0, 1, n))
    if dtype == O.F32:
        g = g32.view(np.uint32)
        ref = (g32 * v[idx]).view(np.uint32)                    # fp32 product
    elif dtype == O.F16:
        gh = g32.astype(np.float16)
        g = gh.view(np.uint16)
        ref = (gh.astype(np.float32) * v[idx]).astype(np.float16).view(np.uint16)
    else:
        g = _bf16_bits(g32)
        prod = (_bf16_val(g).astype(np.float32) * v[idx]).astype(np.float32)
        ref = _bf16_bits(prod)
    gin = O.bwd(dtype, bits, v, g, codes)
    assert np.array_equal(gin, ref)


@pytest.mark.parametrize("dtype,bits", [(O.F32, 3), (O.BF16, 1), (O.F16, 4), (O.BF16, 2)])
def test_threaded_equals_scalar(dtype, bits):
    rng = np.random.default_rng(8)
    n = 100003
    F = O.fit(O.GELU, bits, O.normal(-10.0, 10.0), 400)
    xf = rng.normal(0, 2, n)
    x = O.round_array(dtype, xf)
    y1, c1 = O.fwd(O.GELU, dtype, bits, F.s, x, threads=1)
    y2, c2 = O.fwd(O.GELU, dtype, bits, F.s, x, threads=7)
    assert np.array_equal(y1, y2) and np.array_equal(c1, c2)
    g = O.round_array(dtype, rng.normal(0, 1, n))
    a = O.bwd(dtype, bits, F.v, g, c1, threads=1)
    b = O.bwd(dtype, bits, F.v, g, c1, threads=5)
    assert np.array_equal(a, b)


def test_empty_inputs():
    F = O.fit(O.GELU, 3, O.normal(-10.0, 10.0), 100)
    y, c = O.fwd(O.GELU, O.BF16, 3, F.s, np.zeros(0, np.uint16))
    assert y.size == 0 and c.size == 0
    assert O.bwd(O.BF16, 3, F.v, np.zeros(0, np.uint16), np.zeros(0, np.uint32)).size == 0
