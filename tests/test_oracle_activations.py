"""Pins for the oracle's activations f and closed-form derivatives f'.

The derivatives are pinned against central differences of f (so a dropped
term or a sign slip in either fails), against the symmetry identities of the
four in-scope activations, and against textbook values of the normal cdf.
"""
import math

import numpy as np
import pytest

import oracle as O

ACTS = [O.GELU, O.SILU, O.SIGMOID, O.TANH, O.SOFTPLUS, O.SELU, O.HALFSQ]


@pytest.mark.parametrize("act", ACTS)
def test_derivative_matches_central_difference(act):
    h = 1e-5
    for x in np.linspace(-8.0, 8.0, 161):
        if act == O.SELU and abs(x) < 2 * h:
            continue  # kink at 0
        fd = (O.f(act, x + h) - O.f(act, x - h)) / (2 * h)
        assert abs(fd - O.df(act, x)) < 2e-8 * max(1.0, abs(x)), (act, x)


@pytest.mark.parametrize("act", [O.GELU, O.SILU])
def test_derivative_point_symmetry(act):
    # x*F(x) with F(-x) = 1 - F(x) gives f'(x) + f'(-x) = 1
    for x in np.linspace(0.0, 12.0, 97):
        assert abs(O.df(act, x) + O.df(act, -x) - 1.0) < 1e-14


@pytest.mark.parametrize("act", [O.SIGMOID, O.TANH])
def test_derivative_is_even(act):
    for x in np.linspace(0.0, 12.0, 97):
        assert abs(O.df(act, x) - O.df(act, -x)) < 1e-15


def test_gelu_textbook_values():
    # Phi(1), Phi(2), Phi(-3) from standard normal tables
    assert abs(O.f(O.GELU, 1.0) - 0.8413447460685429) < 1e-15
    assert abs(O.f(O.GELU, -1.0) + 0.15865525393145705) < 1e-15
    assert abs(O.f(O.GELU, 2.0) - 2 * 0.9772498680518208) < 1e-15
    assert abs(O.f(O.GELU, -3.0) + 3 * 0.0013498980316300946) < 1e-16
    assert O.f(O.GELU, 0.0) == 0.0


def test_gelu_derivative_extrema():
    # (GELU')' = phi(x) (2 - x^2): extrema at +-sqrt(2); values 1 +- 0.128904
    r = math.sqrt(2.0)
    top = O.df(O.GELU, r)
    assert abs(top - 1.1289039) < 1e-6
    assert abs(O.df(O.GELU, -r) - (1.0 - top)) < 1e-14
    for d in (1e-3, 1e-2, 0.1):
        assert O.df(O.GELU, r + d) < top and O.df(O.GELU, r - d) < top


def test_other_textbook_values():
    assert abs(O.f(O.SILU, 1.0) - 0.7310585786300049) < 1e-15
    assert abs(O.f(O.SIGMOID, 0.0) - 0.5) == 0.0
    assert abs(O.f(O.TANH, 1.0) - 0.7615941559557649) < 1e-15
    assert abs(O.f(O.SOFTPLUS, 0.0) - math.log(2.0)) < 1e-16
    assert O.df(O.RELU, 1.0) == 1.0 and O.df(O.RELU, -1.0) == 0.0


@pytest.mark.parametrize("act", [O.GELU, O.SILU])
def test_limits_and_nan(act):
    assert O.f(act, math.inf) == math.inf
    v = O.f(act, -math.inf)
    assert v == 0.0 and math.copysign(1.0, v) == -1.0
    assert math.isnan(O.f(act, math.nan))
    # far tail underflows to -0
    v = O.f(act, -1e4)
    assert v == 0.0 and math.copysign(1.0, v) == -1.0


def test_sigmoid_tanh_limits():
    assert O.f(O.SIGMOID, math.inf) == 1.0
    assert O.f(O.SIGMOID, -math.inf) == 0.0
    assert O.f(O.TANH, math.inf) == 1.0
    assert O.f(O.TANH, -math.inf) == -1.0
    assert math.isnan(O.f(O.SIGMOID, math.nan))
    assert math.isnan(O.f(O.TANH, math.nan))


def test_sigmoid_left_tail_keeps_relative_accuracy():
    # sigma(-50) = e^-50 / (1 + e^-50)
    ref = math.exp(-50.0) / (1.0 + math.exp(-50.0))
    assert abs(O.f(O.SIGMOID, -50.0) / ref - 1.0) < 1e-14
