"""Pins of the oracle's alpha-rank meta-solver (single-population alpha-rank
of Omidshafiei et al., 2019, the solver named for PSRO in Sec. 4.2 / Table 3),
against what the mathematics fixes independently of its linear solve:

- the fixation probability's closed forms: m = 2 gives the logistic function
  1 / (1 + e^-u); u -> 0 gives 1/m; the ratio rho(u) / rho(-u) = e^((m-1) u);
- two policies: the stationary distribution of a two-state chain is
  pi_0 = C[1][0] / (C[0][1] + C[1][0]);
- symmetric games: rock-paper-scissors and a constant table give the uniform
  distribution, and relabelling the policies permutes pi;
- a strictly dominant policy takes (almost) all the mass at large alpha;
- at any size: pi >= 0, sum 1, pi^T C = pi^T, and pi equals the limit of
  the chain's powers (brute force, a different method from the solve), on
  small random tables.
A misread sign of the fitness difference, a transposed table or a wrong
mutation rate fails one of these.
"""
import math

import numpy as np
import pytest

import oracle


def test_fixation_closed_forms():
    for u in (-7.0, -1.3, -1e-3, 1e-3, 0.4, 3.0, 20.0):
        assert oracle.alpharank_fixation(u, 2) == pytest.approx(1.0 / (1.0 + math.exp(-u)),
                                                               rel=1e-13)
        for m in (2, 5, 50):
            if abs(u) * (m - 1) > 600:
                continue
            r = oracle.alpharank_fixation(u, m) / oracle.alpharank_fixation(-u, m)
            assert r == pytest.approx(math.exp((m - 1) * u), rel=1e-10)
    for m in (2, 7, 50):
        assert oracle.alpharank_fixation(0.0, m) == 1.0 / m
        assert oracle.alpharank_fixation(1e-9, m) == pytest.approx(1.0 / m, rel=1e-6)
    # large advantages: fixation -> 1 - e^-u, never above 1
    assert oracle.alpharank_fixation(40.0, 50) == pytest.approx(1.0, abs=1e-15)
    # and a large disadvantage: e^-(m-1)u (1 - e^-u) / (1 - e^-mu), no overflow
    assert oracle.alpharank_fixation(-10.0, 50) == pytest.approx(
        math.exp(-490.0) * (1 - math.exp(-10.0)), rel=1e-12)
    assert oracle.alpharank_fixation(-40.0, 50) == 0.0       # underflows, no error


def test_two_policies_closed_form():
    rng = np.random.default_rng(11)
    for _ in range(20):
        M = rng.normal(size=(2, 2))
        alpha, m = float(rng.uniform(0.1, 5)), int(rng.integers(2, 60))
        u01 = alpha * (M[1, 0] - M[0, 1])          # resident 0, mutant 1
        r01 = oracle.alpharank_fixation(u01, m)
        r10 = oracle.alpharank_fixation(-u01, m)
        pi = oracle.alpharank(M, alpha, m)
        assert pi[0] == pytest.approx(r10 / (r01 + r10), rel=1e-12)
        # the linear solve is accurate to rounding of the largest component
        assert pi[1] == pytest.approx(r01 / (r01 + r10), rel=1e-10, abs=1e-15)
    # the policy that wins the meeting takes the larger share
    M = np.array([[0.0, 0.5], [-0.5, 0.0]])
    pi = oracle.alpharank(M, 1.0, 10)
    assert pi[0] > 0.99


def test_symmetric_games_uniform():
    rps = np.array([[0, -1, 1], [1, 0, -1], [-1, 1, 0]], np.float64)
    for alpha in (0.1, 1.0, 10.0):
        assert np.allclose(oracle.alpharank(rps, alpha, 50), 1 / 3, atol=1e-12)
    const = np.full((6, 6), 0.7)
    assert np.allclose(oracle.alpharank(const, 3.0, 20), 1 / 6, atol=1e-13)


def test_relabelling_permutes():
    rng = np.random.default_rng(5)
    M = rng.normal(size=(7, 7))
    perm = rng.permutation(7)
    pi = oracle.alpharank(M, 0.8, 30)
    pi_p = oracle.alpharank(M[np.ix_(perm, perm)], 0.8, 30)
    assert np.allclose(pi_p, pi[perm], atol=1e-13)


def test_dominant_policy_takes_the_mass():
    rng = np.random.default_rng(3)
    M = rng.uniform(-0.2, 0.2, size=(5, 5))
    M[2, :] = 1.0          # policy 2 beats everyone
    M[:, 2] = -1.0
    M[2, 2] = 0.0
    pi = oracle.alpharank(M, 20.0, 50)
    assert pi[2] > 1 - 1e-12
    assert oracle.alpharank(-M, 20.0, 50)[2] < 1e-12     # and loses it when it loses


def test_invariants_and_brute_force():
    rng = np.random.default_rng(7)
    for P in (1, 3, 5, 8):
        M = rng.normal(size=(P, P))
        alpha, m = 0.7, 12
        C = oracle.alpharank_chain(M, alpha, m)
        assert np.allclose(C.sum(axis=1), 1.0, atol=1e-14)
        assert (C >= 0).all()
        pi = oracle.alpharank(M, alpha, m)
        assert (pi >= 0).all() and abs(pi.sum() - 1) < 1e-13
        assert np.allclose(pi @ C, pi, atol=1e-14)
        # brute force: the rows of C^(2^k) converge to pi (aperiodic: C[r][r] > 0);
        # rows renormalized after each squaring against the drift of rounding
        Q = C.copy()
        for _ in range(40):
            Q = Q @ Q
            Q /= Q.sum(axis=1, keepdims=True)
        assert np.allclose(Q, np.tile(pi, (P, 1)), atol=1e-12)


def test_mutation_rate_and_orientation():
    """C[r][s] = rho(alpha (M[s][r] - M[r][s])) / (P - 1), hand-computed for
    one entry of a 3-policy table (a transposed table or a missing 1/(P-1)
    fails)."""
    M = np.array([[0.0, 2.0, 0.0], [1.0, 0.0, 0.0], [0.0, 0.0, 0.0]])
    C = oracle.alpharank_chain(M, 0.5, 4)
    u = 0.5 * (1.0 - 2.0)                       # resident 0, mutant 1
    rho = (1 - math.exp(-u)) / (1 - math.exp(-4 * u))
    assert C[0, 1] == pytest.approx(rho / 2, rel=1e-14)
    assert C[0, 2] == pytest.approx(0.25 / 2, rel=1e-14)   # neutral: 1/m
