"""alpha-rank on the GPU (malib_solve_alpharank, through the C ABI) against
the oracle's definition (oracle.alpharank: the stationary distribution of the
alpha-rank chain by a dense linear solve), on random games from 1 to 256
policies (LDS path up to 128, workspace path above), several ranking
intensities and population sizes, a symmetric game, alpha = 0, and the game
of a real 4v4 table.  Tolerance: |pi_gpu - pi_oracle| <= 1e-12 + 1e-9 pi (both
sides are fp64; the elimination orders differ, and the oracle's solve is
accurate to rounding of the largest component)."""
import numpy as np
import pytest

from gpu_helpers import say

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _gpu_ar(M, alpha, m):
    import paper_2106_07551_amd as MA
    g = torch.from_numpy(np.ascontiguousarray(M, np.float64)).cuda()
    pi, sigma = MA.solve_alpharank(g, alpha, m)
    torch.cuda.synchronize()
    return pi.cpu().numpy(), sigma.cpu().numpy()


def _close(a, b):
    return np.all(np.abs(a - b) <= 1e-12 + 1e-9 * np.abs(b))


CASES = [(1, 1.0, 50), (2, 0.5, 2), (3, 2.0, 50), (8, 0.3, 10), (64, 1.0, 50), (128, 2.0, 50),
         (129, 1.0, 50), (200, 0.7, 20), (256, 1.0, 50), (256, 3.0, 2)]


@pytest.mark.parametrize("P,alpha,m", CASES)
def test_alpharank_matches_oracle(P, alpha, m):
    import oracle
    rng = np.random.default_rng(P * 31 + m)
    M = rng.normal(size=(P, P))
    say(f"[alpharank] P={P} alpha={alpha} m={m}")
    pi, sigma = _gpu_ar(M, alpha, m)
    ref = oracle.alpharank(M, alpha, m)
    err = np.abs(pi - ref).max()
    say(f"[alpharank] P={P}: max |pi - oracle| {err:.3g}, max pi {ref.max():.3g}")
    assert _close(pi, ref), err
    assert abs(pi.sum() - 1) < 1e-12
    assert np.array_equal(sigma[0], sigma[1])
    assert np.array_equal(sigma[0], pi.astype(np.float32))


def test_alpharank_symmetric_and_neutral():
    rps = np.array([[0, -1, 1], [1, 0, -1], [-1, 1, 0]], np.float64)
    pi, _ = _gpu_ar(rps, 5.0, 50)
    assert np.allclose(pi, 1 / 3, atol=1e-14)
    rng = np.random.default_rng(2)
    pi, _ = _gpu_ar(rng.normal(size=(40, 40)), 0.0, 50)       # alpha = 0: all neutral
    assert np.allclose(pi, 1 / 40, atol=1e-14)


def test_alpharank_on_a_4v4_table():
    """The game of a real table (the 4v4 game, 128 policies, a short fill)."""
    import oracle
    import workloads as W
    import paper_2106_07551_amd as MA
    from paper_2106_07551_amd import workload_io as IO
    wl = W.make(5, n_envs=4096, horizon=8)
    pop = IO.make_population(wl)
    env = IO.make_env(wl)
    pairs = torch.empty((wl.n_envs, wl.n_agents), dtype=torch.int32, device="cuda")
    MA.meta_sample(wl.sigma, wl.P, wl.n_envs, wl.n_agents, wl.seed, out=pairs)
    pop.rollout(env, wl.n_envs, pairs, wl.seed, wl.horizon)
    game = pop.payoff_matrix()
    pi, sigma = MA.solve_alpharank(game, 1.0, 50)
    torch.cuda.synchronize()
    ref = oracle.alpharank(game.cpu().numpy(), 1.0, 50)
    pop.close()
    assert _close(pi.cpu().numpy(), ref)
