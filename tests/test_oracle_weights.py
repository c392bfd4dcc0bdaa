"""Pins for the oracle's weight functions w(x) of Eq. (3) and for SELU's f.

The prefix integrals W(i) = int_A^{t_i} w, FW(i) = int f' w and F2(i) =
int f'^2 w are what the dynamic programme of Sec. 3 runs on.  Here they are
checked against closed forms of the normal and normal-mixture densities that
the oracle does not use (the oracle integrates the density cell by cell with
a Gauss-Legendre rule; the tests use the normal cdf and the moments of a
truncated normal):

  int_a^b N(0, s^2)        = Phi(b/s) - Phi(a/s)
  int_a^b x   N(0, s^2) dx = s (phi(a/s) - phi(b/s))
  int_a^b x^2 N(0, s^2) dx = s^2 [Phi(z) - z phi(z)]_{a/s}^{b/s}

With f = x^2 / 2 (f' = x) the prefix sums FW and F2 are the first and second
moments of w, and with ReLU (f' = 1 for x > 0) FW is the weight of the
positive half-line.  The mixture weights (1 - p) N(mu, sigma^2) + p
N(mu, sigma2^2) use p != 1/2, sigma != sigma2 and a support that cuts both
components, so swapping p and 1 - p, or reading sigma2 as a variance, moves
every value here by far more than the tolerance.

SELU is pinned by the property its constants are defined by (Klambauer et al.,
2017): for z ~ N(0, 1) the output has mean 0 and second moment 1.  Dropping
the -1 of e^x - 1 on the negative side, or swapping lambda and alpha, breaks
both.
"""
import math

import numpy as np
import pytest
from scipy import integrate
from scipy.special import ndtr

import oracle as O


def _phi(z):
    return np.exp(-0.5 * z * z) / math.sqrt(2.0 * math.pi)


def _mass(a, b, s, mu=0.0):
    return ndtr((b - mu) / s) - ndtr((a - mu) / s)


def _m1(a, b, s):
    return s * (_phi(a / s) - _phi(b / s))


def _m2(a, b, s):
    za, zb = a / s, b / s
    return s * s * ((ndtr(zb) - zb * _phi(zb)) - (ndtr(za) - za * _phi(za)))


def _grid(w, n):
    return w.A + (w.B - w.A) * np.arange(n + 1) / n


MIXTURES = [
    O.mixture(-2.0, 1.5, 0.2, 1.0, 3.0),
    O.mixture(-40.0, 40.0, 0.01, 1.0, 10.0),     # the large-LM workload's weight
    O.mixture(-5.0, 7.0, 0.7, 0.5, 2.5),
]


@pytest.mark.parametrize("w", MIXTURES)
def test_mixture_weight_mass(w):
    n = 600
    W, _, _ = O.prefix(O.HALFSQ, w, n)
    t = _grid(w, n)
    ref = (1 - w.p) * _mass(w.A, t, w.sigma) + w.p * _mass(w.A, t, w.sigma2)
    assert np.max(np.abs(W - ref)) < 1e-12


@pytest.mark.parametrize("w", MIXTURES)
def test_mixture_weight_moments(w):
    n = 600
    _, FW, F2 = O.prefix(O.HALFSQ, w, n)
    t = _grid(w, n)
    m1 = (1 - w.p) * _m1(w.A, t, w.sigma) + w.p * _m1(w.A, t, w.sigma2)
    m2 = (1 - w.p) * _m2(w.A, t, w.sigma) + w.p * _m2(w.A, t, w.sigma2)
    assert np.max(np.abs(FW - m1)) < 1e-11
    assert np.max(np.abs(F2 - m2)) < 1e-9


def test_mixture_weight_positive_half_line():
    w = O.mixture(-3.0, 4.0, 0.3, 0.8, 2.0)
    n = 700                         # t = 0 is grid point 300
    _, FW, _ = O.prefix(O.RELU, w, n)
    ref = (1 - w.p) * _mass(0.0, 4.0, w.sigma) + w.p * _mass(0.0, 4.0, w.sigma2)
    assert abs(FW[-1] - ref) < 1e-12
    assert np.all(FW[:301] == 0.0)


def test_mixture_weight_distinguishes_its_parameters():
    # the closed forms above tell the plausible misreadings apart
    w = MIXTURES[0]
    good = (1 - w.p) * _mass(w.A, w.B, w.sigma) + w.p * _mass(w.A, w.B, w.sigma2)
    swapped = w.p * _mass(w.A, w.B, w.sigma) + (1 - w.p) * _mass(w.A, w.B, w.sigma2)
    variance = (1 - w.p) * _mass(w.A, w.B, w.sigma) + w.p * _mass(w.A, w.B, w.sigma2 ** 2)
    W, _, _ = O.prefix(O.HALFSQ, w, 400)
    assert abs(W[-1] - good) < 1e-12
    assert abs(W[-1] - swapped) > 1e-2 and abs(W[-1] - variance) > 1e-2


@pytest.mark.parametrize("mu,sigma", [(0.0, 1.0), (0.5, 1.5), (-1.0, 0.25)])
def test_normal_weight_mass_and_mean(mu, sigma):
    w = O.normal(-6.0, 6.0, mu, sigma)
    n = 480
    W, FW, _ = O.prefix(O.HALFSQ, w, n)
    t = _grid(w, n)
    assert np.max(np.abs(W - _mass(w.A, t, sigma, mu))) < 1e-12
    # first moment of N(mu, s^2) over [A, t]: mu * mass + s (phi(a') - phi(t'))
    za, zt = (w.A - mu) / sigma, (t - mu) / sigma
    m1 = mu * _mass(w.A, t, sigma, mu) + sigma * (_phi(za) - _phi(zt))
    assert np.max(np.abs(FW - m1)) < 1e-11


def test_uniform_weight_is_unnormalised_length():
    w = O.uniform(-10.0, 10.0)
    W, FW, F2 = O.prefix(O.HALFSQ, w, 400)
    t = _grid(w, 400)
    assert np.max(np.abs(W - (t + 10.0))) < 1e-12
    assert np.max(np.abs(FW - (t * t - 100.0) / 2)) < 1e-10
    assert np.max(np.abs(F2 - (t ** 3 + 1000.0) / 3)) < 1e-9


# ---------------------------------------------------------------- SELU
def _selu_normal_moment(k):
    g = lambda z: O.f(O.SELU, z) ** k * _phi(z)
    a, _ = integrate.quad(g, -40.0, 0.0, epsabs=1e-14, epsrel=1e-13)
    b, _ = integrate.quad(g, 0.0, 40.0, epsabs=1e-14, epsrel=1e-13)
    return a + b


def test_selu_is_self_normalising():
    # the defining property of SELU's lambda and alpha: a standard normal
    # input keeps mean 0 and second moment 1
    assert abs(_selu_normal_moment(1)) < 1e-9
    assert abs(_selu_normal_moment(2) - 1.0) < 1e-9


def test_selu_shape():
    lam = O.df(O.SELU, 1.0)                     # slope of the positive side
    assert abs(O.f(O.SELU, 2.0) - 2.0 * lam) < 1e-15
    assert O.f(O.SELU, 0.0) == 0.0
    # continuous at 0, negative side saturates at -lambda alpha = -f'(0-)
    left = O.df(O.SELU, -0.0)                   # lambda alpha e^0
    assert abs(O.f(O.SELU, -1e-9)) < 2e-9
    assert abs(O.f(O.SELU, -60.0) + left) < 1e-12
    assert O.f(O.SELU, -math.inf) == -left
    # the negative side is lambda alpha (e^x - 1): its derivative is
    # lambda alpha e^x, so f(x) = f'(x) - f'(0-)
    for x in (-0.1, -1.0, -3.0):
        assert abs(O.f(O.SELU, x) - (O.df(O.SELU, x) - left)) < 1e-15
