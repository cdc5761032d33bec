"""The LP meta-solver on the GPU (malib_solve_lp, through the C ABI) against
the oracle's LPs (scipy's HiGHS): the value within 1e-9 (relative to the
payoff scale), and the GPU's own strategies checked for what makes them
optimal, since optimal strategies need not be unique: distributions, and
min_j (x^T M)_j >= v - 1e-9, max_i (M y)_i <= v + 1e-9.  Games of 1 to 256
policies (LDS tableau up to 96, workspace above), a degenerate game with many
ties, rock-paper-scissors, and the game of a real 4v4 table."""
import numpy as np
import pytest

from gpu_helpers import say

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _check(M, tag):
    import oracle
    import paper_2106_07551_amd as MA
    g = torch.from_numpy(np.ascontiguousarray(M, np.float64)).cuda()
    value, x, y, sigma, piv = MA.solve_lp(g)
    torch.cuda.synchronize()
    v = float(value.cpu()[0])
    x = x.cpu().numpy()
    y = y.cpu().numpy()
    v_ref = oracle.solve_lp(M)[0]
    scale = max(1.0, float(np.abs(M).max()))
    say(f"[lp] {tag}: P={M.shape[0]} value {v:.12g} (oracle {v_ref:.12g}), pivots "
        f"{int(piv.cpu()[0])}")
    assert int(piv.cpu()[0]) >= 0
    assert abs(v - v_ref) <= 1e-9 * scale
    for s in (x, y):
        assert (s >= -1e-12).all() and abs(s.sum() - 1) < 1e-9
    assert (x @ M).min() >= v - 1e-9 * scale
    assert (M @ y).max() <= v + 1e-9 * scale
    sg = sigma.cpu().numpy()
    assert np.array_equal(sg[0], x.astype(np.float32))
    assert np.array_equal(sg[1], y.astype(np.float32))


@pytest.mark.parametrize("P", [1, 2, 5, 32, 96, 97, 128, 256])
def test_lp_random_games(P):
    rng = np.random.default_rng(1000 + P)
    _check(rng.normal(size=(P, P)), "normal")


def test_lp_structured_games():
    rps = np.array([[0, -1, 1], [1, 0, -1], [-1, 1, 0]], np.float64)
    _check(rps, "rps")
    rng = np.random.default_rng(3)
    _check(rng.integers(-2, 3, size=(40, 40)).astype(np.float64), "integer ties")
    _check(np.full((10, 10), 0.25), "constant")
    M = rng.normal(size=(20, 20))
    M[7, :] = 5.0                                    # a dominant row
    _check(M, "dominant row")


def test_lp_on_a_4v4_table():
    import workloads as W
    import paper_2106_07551_amd as MA
    from paper_2106_07551_amd import workload_io as IO
    wl = W.make(5, n_envs=4096, horizon=8)
    pop = IO.make_population(wl)
    env = IO.make_env(wl)
    pairs = torch.empty((wl.n_envs, wl.n_agents), dtype=torch.int32, device="cuda")
    MA.meta_sample(wl.sigma, wl.P, wl.n_envs, wl.n_agents, wl.seed, out=pairs)
    pop.rollout(env, wl.n_envs, pairs, wl.seed, wl.horizon)
    game = pop.payoff_matrix().cpu().numpy()
    pop.close()
    _check(game, "4v4 table")


@pytest.mark.parametrize("bad", [float("nan"), float("inf"), -float("inf")])
@pytest.mark.parametrize("P", [3, 120])
def test_lp_non_finite_game_gives_nan(bad, P):
    """A NaN or infinite payoff leaves no game to solve: value, both
    strategies and the weight rows are NaN and pivots is -1, for the tableau
    in LDS (P <= 96) and in the workspace."""
    import paper_2106_07551_amd as MA
    M = np.random.default_rng(P).uniform(-1, 1, (P, P))
    M[P // 2, P - 1] = bad
    g = torch.from_numpy(M).cuda()
    value, x, y, sigma, piv = MA.solve_lp(g)
    torch.cuda.synchronize()
    assert np.isnan(float(value.cpu()[0]))
    assert np.isnan(x.cpu().numpy()).all() and np.isnan(y.cpu().numpy()).all()
    assert np.isnan(sigma.cpu().numpy()).all()
    assert int(piv.cpu()[0]) == -1
