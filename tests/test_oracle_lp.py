"""Pins of the oracle's LP meta-solver (the zero-sum meta-game's exact
equilibrium; the LP solver of the PSRO experiments, Sec. 4.2), against what
the minimax theorem fixes independently of the LP code:

- 2x2 games without a saddle point: the closed-form mixed equilibrium
  x_0 = (d - c) / (a - b - c + d), value (ad - bc) / (a - b - c + d);
- saddle points: the pure value; rock-paper-scissors: value 0, uniform;
- the equilibrium property on random games: min_j (x^T M)_j = v =
  max_i (M y)_i (neither side can gain), x and y distributions;
- fictitious play (the oracle's own C solver, another method) brackets the
  value: min_j (xbar^T M)_j <= v <= max_i (M ybar)_i for its averages;
- v(-M^T) = -v(M) (the sides swapped), v(M + c) = v(M) + c.
"""
import numpy as np
import pytest

import oracle


def test_two_by_two_closed_form():
    rng = np.random.default_rng(4)
    n = 0
    while n < 20:
        a, b, c, d = rng.normal(size=4)
        # no saddle point: the diagonals beat the off-diagonals on one side
        if not ((a > b and d > c and a > c and d > b) or (a < b and d < c and a < c and d < b)):
            continue
        den = a - b - c + d
        v, x, y = oracle.solve_lp(np.array([[a, b], [c, d]]))
        assert v == pytest.approx((a * d - b * c) / den, abs=1e-9)
        assert x[0] == pytest.approx((d - c) / den, abs=1e-8)
        assert y[0] == pytest.approx((d - b) / den, abs=1e-8)
        n += 1


def test_saddle_and_symmetric():
    M = np.array([[1.0, 2.0], [0.0, 3.0]])           # row 0 guarantees 1; column 0 caps 1
    v, x, y = oracle.solve_lp(M)
    assert v == pytest.approx(1.0) and x[0] == pytest.approx(1.0) and y[0] == pytest.approx(1.0)
    rps = np.array([[0, -1, 1], [1, 0, -1], [-1, 1, 0]], np.float64)
    v, x, y = oracle.solve_lp(rps)
    assert abs(v) < 1e-12 and np.allclose(x, 1 / 3) and np.allclose(y, 1 / 3)


@pytest.mark.parametrize("P", [1, 3, 7, 20, 64])
def test_equilibrium_property(P):
    rng = np.random.default_rng(P)
    M = rng.normal(size=(P, P))
    v, x, y = oracle.solve_lp(M)
    for s in (x, y):
        assert (s >= -1e-12).all() and abs(s.sum() - 1) < 1e-9
    assert (x @ M).min() == pytest.approx(v, abs=1e-8)
    assert (M @ y).max() == pytest.approx(v, abs=1e-8)
    # sides swapped, shifted payoffs
    assert oracle.solve_lp(-M.T)[0] == pytest.approx(-v, abs=1e-8)
    assert oracle.solve_lp(M + 2.5)[0] == pytest.approx(v + 2.5, abs=1e-8)


def test_fictitious_play_brackets_the_value():
    rng = np.random.default_rng(9)
    M = rng.normal(size=(12, 12))
    v, _, _ = oracle.solve_lp(M)
    cx, cy, gap = oracle.solve_fp(M, 20000)
    xb = cx / cx.sum()
    yb = cy / cy.sum()
    lo, hi = (xb @ M).min(), (M @ yb).max()
    assert lo - 1e-12 <= v <= hi + 1e-12
    assert hi - lo == pytest.approx(gap, rel=1e-6, abs=1e-9)
