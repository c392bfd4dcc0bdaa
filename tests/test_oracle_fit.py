"""Pins for the oracle's optimal piecewise-constant fit (Sec. 3).

* brute force over every partition of a coarse grid (the DP minimum and its
  cut points, bitwise: same left-to-right sums);
* the paper's Table 1 (fit errors of 7 activations x 4 bit widths);
* closed forms (GELU and Softplus 1-bit; Sigmoid / Tanh 1-bit symmetric; ReLU);
* textbook quantizers: Lloyd-Max of a uniform source (boundaries m/K,
  MSE 1/(12K^2)) and of a Gaussian source (Max 1960);
* invariants: sorted boundaries, non-increasing loss in the number of
  intervals, mean preservation, values within the range of f', first-order
  optimality (the gradient formula of Sec. 3 vanishes at the optimum),
  prefix-sum costs equal to direct quadrature per interval.
"""
import itertools
import math
import os

import numpy as np
import pytest
from scipy import integrate, optimize

import oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
ACT_BY_NAME = {"relu": O.RELU, "gelu": O.GELU, "swish": O.SILU, "sigmoid": O.SIGMOID,
               "tanh": O.TANH, "selu": O.SELU, "softplus": O.SOFTPLUS}


def _read_table1():
    rows = []
    with open(os.path.join(GOLDEN, "table1_fit_errors.txt")) as fh:
        for line in fh:
            line = line.split("#")[0].strip()
            if not line:
                continue
            parts = line.split()
            vals = [None if p == "-" else float(p) for p in parts[2:6]]
            rows.append((parts[0], bool(int(parts[1])), vals))
    return rows


# ------------------------------------------------------------------ Table 1
@pytest.mark.parametrize("name,symmetric,vals", _read_table1())
def test_table1_fit_errors(name, symmetric, vals):
    # one K=16 run yields DP(n, k) for every k; 1..4 bits are k = 2, 4, 8, 16
    F = O.fit(ACT_BY_NAME[name], 4, O.uniform(-10.0, 10.0), 4000, symmetric=symmetric)
    for b, printed in enumerate(vals, start=1):
        if printed is None:
            continue
        got = F.dp_last[(1 << b) - 1]
        # printed to 4 decimals (+-5e-5) plus the grid's discretisation error
        assert abs(got - printed) <= 1.01e-4, (name, b, got, printed)


def test_error_drops_per_extra_bit():
    # Sec. 3 observes a factor of roughly 2-4 per extra bit (informative bound)
    F = O.fit(O.GELU, 4, O.uniform(-10.0, 10.0), 2000)
    L = [F.dp_last[(1 << b) - 1] for b in range(1, 5)]
    for a, b in zip(L, L[1:]):
        assert 1.5 < a / b < 5.0


# ------------------------------------------------------------------ brute force
def _brute(act, w, n, K):
    W, FW, F2 = O.prefix(act, w, n)
    t = [w.A + i * (w.B - w.A) / n for i in range(n + 1)]
    cost = {}

    def T(j, i):
        key = (j, i)
        if key not in cost:
            cost[key] = O.interval_cost(W, FW, F2, j, i, act, t[j], t[i])
        return cost[key]

    best, arg = math.inf, None
    for cuts in itertools.combinations(range(1, n), K - 1):
        pts = (0,) + cuts + (n,)
        c = T(pts[0], pts[1])
        for a, b in zip(pts[1:], pts[2:]):
            c = c + T(a, b)
        if c < best:
            best, arg = c, pts
    return best, arg, T


@pytest.mark.parametrize("act,w,n,bits", [
    (O.GELU, O.normal(-4.0, 4.0), 200, 1),
    (O.SILU, O.uniform(-6.0, 5.0), 150, 1),
    (O.GELU, O.normal(-4.0, 4.0), 60, 2),
    (O.TANH, O.uniform(-3.0, 3.5), 48, 2),
    (O.SIGMOID, O.mixture(-6.0, 6.0, 0.1, 1.0, 3.0), 56, 2),
])
def test_dp_equals_brute_force(act, w, n, bits):
    K = 1 << bits
    F = O.fit(act, bits, w, n)
    best, arg, T = _brute(act, w, n, K)
    assert F.loss == best                       # bitwise: same sums, same order
    pts = list(F.cuts)
    c = T(pts[0], pts[1])
    for a, b in zip(pts[1:], pts[2:]):
        c = c + T(a, b)
    assert c == best                            # the DP's cut points attain it
    if tuple(pts) != arg:                       # a tie: both optimal
        assert c == best


# ------------------------------------------------------------------ closed forms
def test_gelu_one_bit_closed_form():
    # split at 0 by the point symmetry of GELU'; y0 = (GELU(0)-GELU(-10))/10,
    # y1 = (GELU(10)-GELU(0))/10; L = int GELU'^2 - 10 (y0^2 + y1^2)
    def dgelu(x):
        return 0.5 * (1 + math.erf(x / math.sqrt(2))) + x * math.exp(-x * x / 2) / math.sqrt(2 * math.pi)

    def gelu(x):
        return 0.5 * x * (1 + math.erf(x / math.sqrt(2)))

    I = integrate.quad(lambda x: dgelu(x) ** 2, -10, 0, epsabs=1e-14, epsrel=1e-14)[0] \
        + integrate.quad(lambda x: dgelu(x) ** 2, 0, 10, epsabs=1e-14, epsrel=1e-14)[0]
    y0 = (gelu(0) - gelu(-10)) / 10
    y1 = (gelu(10) - gelu(0)) / 10
    L = I - 10 * (y0 ** 2 + y1 ** 2)
    F = O.fit(O.GELU, 1, O.uniform(-10.0, 10.0), 4000)
    assert abs(F.loss - L) < 1e-10
    assert F.s[0] == 0.0
    assert abs(L - 0.1410474) < 1e-7


def test_softplus_one_bit_closed_form():
    # f' = sigma, int sigma^2 over [-10,10] = 10 - tanh 5; split at 0
    ln2 = math.log(2.0)
    sp10 = 10 + math.log1p(math.exp(-10))
    L = 10 - math.tanh(5) - ((ln2 - math.log1p(math.exp(-10))) ** 2 + (sp10 - ln2) ** 2) / 10
    F = O.fit(O.SOFTPLUS, 1, O.uniform(-10.0, 10.0), 4000)
    assert abs(F.loss - L) < 1e-10
    assert abs(L - 0.2902163) < 1e-7


def _sym_one_bit(G, S, B=10.0):
    """min_s of the symmetric 1-bit loss, closed-form interval integrals.

    G(u): antiderivative of f'^2 in the variable u = f; S(x): f(x) - f(0)."""
    def L(s):
        tot = G(B) - G(0.0)
        return 2 * (tot - S(s) ** 2 / s - (S(B) - S(s)) ** 2 / (B - s))
    r = optimize.minimize_scalar(L, bounds=(0.01, B - 0.01), method="bounded",
                                 options={"xatol": 1e-10})
    return r.fun, r.x


def test_sigmoid_one_bit_symmetric_closed_form():
    sig = lambda x: 1.0 / (1.0 + math.exp(-x))
    # int sigma'^2 dx = int u (1-u) du = u^2/2 - u^3/3 with u = sigma
    G = lambda x: sig(x) ** 2 / 2 - sig(x) ** 3 / 3
    Lc, sstar = _sym_one_bit(G, lambda x: sig(x) - 0.5)
    F = O.fit(O.SIGMOID, 1, O.uniform(-10.0, 10.0), 4000, symmetric=True)
    assert abs(Lc - 0.018074) < 1e-6 and abs(sstar - 2.04495) < 1e-4
    assert Lc - 1e-12 <= F.loss <= Lc + 2e-7        # grid optimum >= continuum
    assert abs(F.s[0] - sstar) < 2.5e-3             # grid spacing 10/4000


def test_tanh_one_bit_symmetric_closed_form():
    # int (1-tanh^2)^2 dx = int (1-u^2) du = u - u^3/3 with u = tanh
    G = lambda x: math.tanh(x) - math.tanh(x) ** 3 / 3
    Lc, sstar = _sym_one_bit(G, math.tanh)
    F = O.fit(O.TANH, 1, O.uniform(-10.0, 10.0), 4000, symmetric=True)
    assert abs(Lc - 0.158400) < 1e-6 and abs(sstar - 1.06036) < 1e-4
    assert Lc - 1e-12 <= F.loss <= Lc + 2e-7
    assert abs(F.s[0] - sstar) < 2.5e-3


def test_relu_one_bit_is_exact():
    F = O.fit(O.RELU, 1, O.uniform(-10.0, 10.0), 4000)
    assert F.loss < 1e-12
    assert F.s[0] == 0.0
    assert abs(F.v[0]) < 1e-12 and abs(F.v[1] - 1.0) < 1e-12


# ------------------------------------------------------------------ Lloyd-Max
@pytest.mark.parametrize("bits", [1, 2, 3, 4])
def test_lloyd_max_uniform_source(bits):
    # f'(x) = x, w = 1 on [0,1]: K equal cells, MSE 1/(12 K^2) (exact on the grid)
    K = 1 << bits
    F = O.fit(O.HALFSQ, bits, O.uniform(0.0, 1.0), 64 * K)
    assert np.array_equal(F.s, np.float32([m / K for m in range(1, K)]))
    assert abs(F.loss - 1.0 / (12 * K * K)) < 1e-14
    assert np.allclose(F.v_double, [(m + 0.5) / K for m in range(K)], atol=1e-14)


def _read_max():
    rows = {}
    with open(os.path.join(GOLDEN, "lloyd_max_gaussian.txt")) as fh:
        for line in fh:
            line = line.split("#")[0].strip()
            if not line:
                continue
            toks = line.split()
            K = int(toks[0])
            nb = K // 2 - 1
            bnd = [] if toks[1] == "-" else [float(t) for t in toks[1:1 + nb]]
            off = 1 + max(nb, 1) if toks[1] == "-" else 1 + nb
            outs = [float(t) for t in toks[off:off + K // 2]]
            mse = float(toks[off + K // 2])
            rows[K] = (bnd, outs, mse)
    return rows


@pytest.mark.parametrize("bits", [1, 2, 3, 4])
def test_lloyd_max_gaussian_source(bits):
    K = 1 << bits
    bnd, outs, mse = _read_max()[K]
    F = O.fit(O.HALFSQ, bits, O.normal(-10.0, 10.0), 4000)   # grid step 0.005
    half_s = F.s[K // 2:]                   # positive boundaries
    assert F.s[K // 2 - 1] == 0.0
    assert np.allclose(half_s, bnd, atol=4e-3)
    assert np.allclose(F.v[K // 2:], outs, atol=3e-3)          # grid-limited
    assert abs(F.loss - mse) < 1.5e-4


# ------------------------------------------------------------------ invariants
CASES = [
    (O.GELU, O.uniform(-10.0, 10.0), 2000),
    (O.GELU, O.normal(-10.0, 10.0), 2000),
    (O.SILU, O.normal(-10.0, 10.0), 2000),
    (O.GELU, O.mixture(-40.0, 40.0, 0.01, 1.0, 10.0), 3200),
    (O.SIGMOID, O.uniform(-8.0, 8.0), 1600),
    (O.TANH, O.uniform(-8.0, 8.0), 1600),
]


@pytest.mark.parametrize("act,w,n", CASES)
def test_fit_invariants(act, w, n):
    F = O.fit(act, 4, w, n)
    W, FW, F2 = O.prefix(act, w, n)
    # loss non-increasing in the number of intervals
    assert np.all(np.diff(F.dp_last) <= 1e-15)
    assert np.all(np.isfinite(F.dp_last)) and np.all(F.dp_last >= 0)
    for bits in (1, 2, 3, 4):
        G = O.fit(act, bits, w, n)
        K = 1 << bits
        assert np.all(np.diff(G.s) > 0)                         # strictly sorted
        assert np.all(np.isfinite(G.v))
        assert G.loss == pytest.approx(F.dp_last[K - 1], rel=0, abs=0)
        # mean preservation: sum v_m dW_m = int f' w
        dW = np.diff(W[G.cuts])
        assert abs(np.dot(G.v_double, dW) - FW[-1]) < 1e-12 * max(1.0, abs(FW[-1]))
        # each value lies within the range of f' over its interval
        t = lambda i: w.A + i * (w.B - w.A) / n
        for m in range(K):
            xs = np.linspace(t(G.cuts[m]), t(G.cuts[m + 1]), 257)
            d = np.array([O.df(act, x) for x in xs])
            assert d.min() - 1e-12 <= G.v_double[m] <= d.max() + 1e-12


@pytest.mark.parametrize("act", [O.GELU, O.SILU, O.TANH])
def test_first_order_optimality(act):
    # dL/ds_m = (2 f'(s_m) - y_m - y_{m-1}) (y_m - y_{m-1}) w(s_m) vanishes at
    # the optimum, so f'(s_m) = (y_{m-1} + y_m)/2 up to the grid resolution
    F = O.fit(act, 3, O.uniform(-10.0, 10.0), 4000)
    for m in range(7):
        mid = 0.5 * (F.v_double[m] + F.v_double[m + 1])
        assert abs(O.df(act, float(F.s[m])) - mid) < 4e-3


@pytest.mark.parametrize("act,w", [(O.GELU, O.normal(-6.0, 6.0)),
                                   (O.SILU, O.uniform(-5.0, 5.0))])
def test_prefix_costs_equal_direct_quadrature(act, w):
    n = 240
    W, FW, F2 = O.prefix(act, w, n)
    t = lambda i: w.A + i * (w.B - w.A) / n
    pdf = (lambda x: 1.0) if w.kind == O.W_UNIFORM else \
        (lambda x: math.exp(-x * x / 2) / math.sqrt(2 * math.pi))
    rng = np.random.default_rng(0)
    for _ in range(12):
        j, i = sorted(rng.choice(n + 1, 2, replace=False))
        a, b = t(j), t(i)
        ww = integrate.quad(pdf, a, b, epsabs=1e-15, epsrel=1e-13)[0]
        fw = integrate.quad(lambda x: O.df(act, x) * pdf(x), a, b, epsabs=1e-15, epsrel=1e-13)[0]
        y = fw / ww
        Td = integrate.quad(lambda x: (O.df(act, x) - y) ** 2 * pdf(x), a, b,
                            epsabs=1e-15, epsrel=1e-12, limit=200)[0]
        Tp = O.interval_cost(W, FW, F2, int(j), int(i), act, a, b)
        assert abs(Tp - Td) < 1e-12 + 1e-9 * Td


def test_far_tail_cells_are_clamped():
    # normal weight on a wide support: prefix sums saturate; costs stay >= 0
    F = O.fit(O.GELU, 4, O.normal(-40.0, 40.0), 8000)
    assert np.all(np.isfinite(F.v)) and np.all(np.diff(F.s) > 0) and F.loss >= 0


def test_fit_rejects_bad_arguments():
    with pytest.raises(ValueError):
        O.fit(O.GELU, 5, O.uniform(-1, 1), 100)
    with pytest.raises(ValueError):
        O.fit(O.GELU, 4, O.uniform(-1, 1), 8)
