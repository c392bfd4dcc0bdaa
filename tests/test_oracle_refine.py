"""Pins for the oracle's gradient refinement of the fitted boundaries (Sec. 3).

* the analytic gradient of L(s, y(s)) against central finite differences of
  L itself (a dropped factor, a swapped y_{i-1} / y_i or a missing w(s_i)
  fails it);
* refinement never increases the DP loss (every row of Table 1);
* continuum optima that the grid cannot represent: the uniform Lloyd-Max
  quantizer (boundaries m/K, MSE 1/(12 K^2)) from a grid that does not hold
  m/K, the Gaussian quantizer of Max (1960) beyond the grid resolution, and
  the Sigmoid / Tanh 1-bit symmetric optima found by scalar minimisation of
  closed-form interval integrals;
* first-order optimality f'(s_i) = (y_{i-1} + y_i) / 2 after refinement.
"""
import numpy as np
import pytest

import oracle as O
from test_oracle_fit import ACT_BY_NAME, _read_max, _read_table1, _sym_one_bit


FD_CASES = [
    (O.GELU, 3, O.uniform(-10.0, 10.0), False),
    (O.GELU, 2, O.normal(-10.0, 10.0), False),
    (O.SILU, 4, O.mixture(-40.0, 40.0, 0.01, 1.0, 10.0), False),
    (O.SIGMOID, 2, O.uniform(-8.0, 8.0), True),
    (O.TANH, 3, O.normal(-10.0, 10.0, 0.0, 2.0), True),
    (O.SOFTPLUS, 2, O.uniform(-10.0, 10.0), False),
]


@pytest.mark.parametrize("act,bits,w,sym", FD_CASES)
def test_gradient_matches_finite_differences(act, bits, w, sym):
    n = 800
    K = 1 << bits
    F = O.fit(act, bits, w, n, symmetric=sym)
    A = max(w.A, 0.0) if sym else w.A
    h = (w.B - A) / n
    rng = np.random.default_rng(3)
    for trial in range(3):
        # off-grid boundaries near the DP optimum, away from it (less than
        # half a cell, so they stay sorted)
        s = np.array([A + c * h for c in F.cuts[1:K]], dtype=np.float64)
        s += rng.uniform(-0.4, 0.4, K - 1) * h
        assert np.all(np.diff(s) > 0)
        L, y, g = O.loss_at(act, bits, w, n, s, symmetric=sym)
        for i in range(K - 1):
            d = 1e-3 * h    # L is a difference of O(1) prefix sums: keep the step
                            # well above their rounding
            sp, sm = s.copy(), s.copy()
            sp[i] += d
            sm[i] -= d
            Lp = O.loss_at(act, bits, w, n, sp, symmetric=sym)[0]
            Lm = O.loss_at(act, bits, w, n, sm, symmetric=sym)[0]
            fd = (Lp - Lm) / (2 * d)
            assert fd == pytest.approx(g[i], rel=1e-4, abs=1e-10), (trial, i, fd, g[i])


@pytest.mark.parametrize("name,symmetric,vals", _read_table1())
def test_refinement_never_increases_the_dp_loss(name, symmetric, vals):
    for bits in (1, 2, 3, 4):
        if vals[bits - 1] is None:
            continue
        R = O.fit_refined(ACT_BY_NAME[name], bits, O.uniform(-10.0, 10.0), 1000,
                          symmetric=symmetric)
        assert R.loss <= R.loss_dp + 1e-15
        assert np.all(np.diff(R.s_double) > 0)
        # still the paper's number to the 4 printed decimals, or better
        assert R.loss <= vals[bits - 1] + 1.01e-4


@pytest.mark.parametrize("bits", [1, 2, 3, 4])
def test_lloyd_max_uniform_source_off_grid(bits):
    # f' = x, w = 1 on [0, 1]; 999 cells: m/K is not a grid point for K > 1
    K = 1 << bits
    R = O.fit_refined(O.HALFSQ, bits, O.uniform(0.0, 1.0), 999)
    # L is flat at the optimum (second order in s), so descent on L locates
    # the boundaries to about sqrt(machine epsilon) and L far better
    assert np.allclose(R.s_double, [m / K for m in range(1, K)], rtol=0, atol=1e-6)
    assert R.loss == pytest.approx(1.0 / (12 * K * K), rel=1e-9)
    assert np.allclose(R.v_double, [(m + 0.5) / K for m in range(K)], rtol=0, atol=1e-6)
    if K > 1:
        assert R.loss_dp > R.loss


@pytest.mark.parametrize("bits", [1, 2, 3, 4])
def test_lloyd_max_gaussian_source_refined(bits):
    # a coarse grid (step 0.02) and Max's 4-digit table: the refined quantizer
    # matches to the table's rounding, which the DP on this grid does not
    K = 1 << bits
    bnd, outs, mse = _read_max()[K]
    R = O.fit_refined(O.HALFSQ, bits, O.normal(-10.0, 10.0), 1000)
    assert np.allclose(R.s_double[K // 2:], bnd, rtol=0, atol=1e-3)
    assert np.allclose(R.v_double[K // 2:], outs, rtol=0, atol=1e-3)
    assert abs(R.loss - mse) <= 0.5e-4 + 5e-4 * mse
    if K > 1:
        assert abs(R.s_double[K // 2 - 1]) < 1e-7      # 0 by symmetry


def test_sigmoid_tanh_one_bit_symmetric_continuum_optimum():
    import math
    sig = lambda x: 1.0 / (1.0 + math.exp(-x))
    cases = [
        (O.SIGMOID, lambda x: sig(x) ** 2 / 2 - sig(x) ** 3 / 3, lambda x: sig(x) - 0.5),
        (O.TANH, lambda x: math.tanh(x) - math.tanh(x) ** 3 / 3, math.tanh),
    ]
    for act, G, S in cases:
        Lc, sstar = _sym_one_bit(G, S)
        R = O.fit_refined(act, 1, O.uniform(-10.0, 10.0), 400, symmetric=True)
        assert R.loss == pytest.approx(Lc, rel=1e-9)
        assert abs(R.s_double[0] - sstar) < 1e-6


@pytest.mark.parametrize("act,w,sym", [
    (O.GELU, O.uniform(-10.0, 10.0), False),
    (O.SILU, O.normal(-10.0, 10.0), False),
    (O.SIGMOID, O.uniform(-10.0, 10.0), True),
    (O.TANH, O.uniform(-10.0, 10.0), True),
    (O.SOFTPLUS, O.uniform(-10.0, 10.0), False),
])
def test_first_order_optimality_after_refinement(act, w, sym):
    R = O.fit_refined(act, 3, w, 1000, symmetric=sym)
    for i in range(7):
        mid = 0.5 * (R.v_double[i] + R.v_double[i + 1])
        assert abs(O.df(act, R.s_double[i]) - mid) < 1e-6
