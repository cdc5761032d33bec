"""GPU parity of the meta-update closed on the device: payoff table -> game
matrix -> fictitious play -> play counts -> meta-sampling from device weights
-> next rollout (Sec. 3.1 meta-update with the fictitious-play solver of the
PSRO experiments, Sec. 4.2), each step against the oracle through the C ABI.

Bars: play counts and policy ids bit for bit; the game matrix and the gap bit
for bit (the same fp64 arithmetic on both sides, in the same order); the
matrix from a rollout bit for bit against the oracle's table where every
return is a multiple of 2^-32 (then both the fixed-point and the fp64 sums are
exact).
"""
import copy

import numpy as np
import pytest

import oracle
import workloads as W
from gpu_helpers import say

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2106_07551_amd as M
    M.lib()


def _solve_gpu(Mx, T):
    import paper_2106_07551_amd as M
    Md = torch.from_numpy(np.ascontiguousarray(Mx, dtype=np.float64)).cuda()
    sig, gap = M.solve_fp(Md, T)
    torch.cuda.synchronize()
    return sig.cpu().numpy(), float(gap.cpu().numpy()[0])


def _check_solve(Mx, T):
    say(f"[gpu] solve_fp P={Mx.shape[0]} T={T}")
    sig, gap = _solve_gpu(Mx, T)
    cx, cy, ogap = oracle.solve_fp(Mx, T)
    assert np.array_equal(sig[0], cx.astype(np.float32)), np.nonzero(sig[0] != cx)[0][:5]
    assert np.array_equal(sig[1], cy.astype(np.float32)), np.nonzero(sig[1] != cy)[0][:5]
    assert np.float64(gap).tobytes() == np.float64(ogap).tobytes(), (gap, ogap)
    assert sig[0].sum() == T and sig[1].sum() == T


# P across the LDS-resident (<= 128) and the global-memory (> 128) variants,
# 1 and 256 the ends of the allowed range
@pytest.mark.parametrize("P", [1, 2, 3, 17, 64, 127, 128, 129, 200, 256])
def test_solve_fp_continuous(P):
    rng = np.random.default_rng(1000 + P)
    _check_solve(rng.uniform(-1.0, 1.0, (P, P)), 700)


@pytest.mark.parametrize("P", [5, 128, 256])
def test_solve_fp_integer_ties(P):
    """Small-integer games: v and w tie all the time, so every iteration
    exercises the first-index rule of both best responses."""
    rng = np.random.default_rng(2000 + P)
    _check_solve(rng.integers(-2, 3, (P, P)).astype(np.float64), 500)
    _check_solve(np.zeros((P, P)), 37)


def test_solve_fp_antisymmetric_and_long_run():
    """A symmetric zero-sum game (antisymmetric M, value 0) over many
    iterations: parity, and the gap of the averages shrinks."""
    rng = np.random.default_rng(7)
    X = rng.normal(size=(32, 32))
    A = X - X.T
    _check_solve(A, 20000)
    g_short = _solve_gpu(A, 100)[1]
    g_long = _solve_gpu(A, 20000)[1]
    assert g_long < g_short and g_long > 0.0


def test_solve_fp_rejects_bad_arguments():
    import paper_2106_07551_amd as M
    Md = torch.zeros((4, 4), dtype=torch.float64, device="cuda")
    for T in (0, -3, (1 << 24) + 1):
        with pytest.raises(M.MalibError):
            M.solve_fp(Md, T)
    big = torch.zeros((257, 257), dtype=torch.float64, device="cuda")
    with pytest.raises(M.MalibError):
        M.solve_fp(big, 10)


def test_solve_fp_nan_gives_nan_gap():
    """A NaN that the iteration reads (here in every column, so v of one
    policy turns NaN at the first step) keeps every read inside the game and
    is reported through a NaN gap."""
    rng = np.random.default_rng(3)
    for P in (8, 200):
        Mx = rng.uniform(-1, 1, (P, P))
        Mx[P // 2, :] = np.nan
        sig, gap = _solve_gpu(Mx, 50)
        assert np.isnan(gap)
        assert sig[0].sum() == 50 and sig[1].sum() == 50


@pytest.mark.parametrize("P,n_sigma", [(1, 1), (9, 1), (9, 2), (256, 3)])
def test_meta_sample_device_weights(P, n_sigma):
    """Thresholds computed on the device from device weights: the same ids
    as the host-threshold path and as the oracle, zero weights never drawn."""
    import paper_2106_07551_amd as M
    n_agents = max(n_sigma, 2)
    rng = np.random.default_rng(P * 10 + n_sigma)
    s = rng.random((n_sigma, P)).astype(np.float32)
    if P > 4:
        s[0, :3] = 0
        s[-1, -1] = 0
    # play counts as weights (the solver's output form)
    s[0] = np.floor(s[0] * 1000)
    if s[0].sum() == 0:
        s[0, -1] = 1
    n = 2049
    for off in (0, 99991):
        g = M.meta_sample_device(torch.from_numpy(s).cuda(), P, n, n_agents, 4242,
                                 env_offset=off).cpu().numpy()
        h = M.meta_sample(s, P, n, n_agents, 4242, env_offset=off).cpu().numpy()
        ref = oracle.meta_sample(s, P, n, n_agents, 4242, off)
        assert np.array_equal(g, ref) and np.array_equal(h, ref)
        seat_rows = s if n_sigma > 1 else np.repeat(s, n_agents, 0)
        for a in range(n_agents):
            assert (seat_rows[a][g[:, a]] > 0).all()


def test_meta_sample_device_seat_rows():
    """Seats mapped onto weight rows (a 4v4 game: the row side's counts for
    seats 0-3, the column side's for 4-7) draw as the oracle does with each
    seat's row written out."""
    import paper_2106_07551_amd as M
    P, n = 128, 3000
    rng = np.random.default_rng(11)
    s = np.floor(rng.random((2, P)) * 50).astype(np.float32)
    s[1, :64] = 0
    seat_row = np.array([0, 0, 0, 0, 1, 1, 1, 1], np.int32)
    g = M.meta_sample_device(torch.from_numpy(s).cuda(), P, n, 8, 99, env_offset=7,
                             seat_row=seat_row).cpu().numpy()
    ref = oracle.meta_sample(s[seat_row], P, n, 8, 99, 7)
    assert np.array_equal(g, ref)
    assert (g[:, 4:] >= 64).all()
    # one row for all seats through the map equals the shared-row default
    g1 = M.meta_sample_device(torch.from_numpy(s[:1].copy()).cuda(), P, n, 8, 99,
                              seat_row=np.zeros(8, np.int32)).cpu().numpy()
    assert np.array_equal(g1, oracle.meta_sample(s[:1], P, n, 8, 99, 0))


def test_meta_sample_device_invalid_row_flags_rollout():
    """A device weight row with no mass, a negative or a NaN weight yields
    policy id -1 for its seat; the next rollout flags those envs and leaves
    them out of the table."""
    import paper_2106_07551_amd as M
    from paper_2106_07551_amd import workload_io as IO
    wl = W.make(1, per_pair=16)
    P = wl.P
    for bad in (np.zeros(P), np.array([1.0] * (P - 1) + [-1.0]),
                np.array([np.nan] + [1.0] * (P - 1))):
        s = np.stack([np.ones(P), bad]).astype(np.float32)
        ids = M.meta_sample_device(torch.from_numpy(s).cuda(), P, wl.n_envs, 2, 5)
        h = ids.cpu().numpy()
        assert (h[:, 1] == -1).all() and (h[:, 0] >= 0).all() and (h[:, 0] < P).all()
        pop = IO.make_population(wl)
        env = IO.make_env(wl)
        pop.rollout(env, wl.n_envs, ids, wl.seed, 1)
        t = pop.payoff(check=False)
        assert t["status"] == M.binding.E_DEVICE and t["device_flags"] & 1
        assert t["counts"].sum() == 0
        pop.close()


def _exact_fixed_point(x):
    x = np.asarray(x, np.float64)
    return np.array_equal(np.ldexp(x, 32), np.round(np.ldexp(x, 32)))


def test_payoff_matrix_after_rollouts():
    """The device game matrix equals the host read-back of the table (NaN -> 0)
    bit for bit, and the oracle's table built from the oracle's own rollout."""
    import paper_2106_07551_amd as M
    from paper_2106_07551_amd import workload_io as IO
    wl = W.make(1, per_pair=64)
    assert _exact_fixed_point(wl.A)
    pop = IO.make_population(wl)
    env = IO.make_env(wl)
    M0 = pop.payoff_matrix().cpu().numpy()
    assert not M0.any()
    pairs = wl.pairs.copy()
    pairs[: wl.n_envs // 2, 0] = 0      # leave some cells empty
    pops = torch.from_numpy(pairs).cuda()
    pop.rollout(env, wl.n_envs, pops, wl.seed, 1)
    Mg = pop.payoff_matrix().cpu().numpy()
    t = pop.payoff()
    host = np.where(t["counts"] > 0, t["mean"], 0.0)
    assert np.array_equal(Mg.view(np.uint64), host.view(np.uint64))
    o = oracle.rollout(wl, np.arange(wl.n_envs), pairs, horizon=1)
    assert o["fails"] == 0
    mean = oracle.payoff(o["returns"], pairs, wl.team, wl.P)[0]
    ref = oracle.payoff_matrix(mean)
    assert (t["counts"] == 0).any()
    assert np.array_equal(Mg.view(np.uint64), ref.view(np.uint64))
    pop.close()


@pytest.mark.parametrize("c,iters,T", [(1, 4, 2000), (2, 3, 500)])
def test_meta_update_loop_closed_on_device(c, iters, T):
    """Rollout -> table -> game -> fictitious play -> per-seat play counts as
    weights -> meta-sample -> next rollout, all on the device with no host
    round trip; the oracle runs the same loop from the same seeds on its own.
    Policy ids of every round, the game matrix and the counts match bit for
    bit (returns of these games are multiples of 2^-32, so the tables agree
    exactly)."""
    import paper_2106_07551_amd as M
    from paper_2106_07551_amd import workload_io as IO
    if c == 1:
        wl = W.make(1, per_pair=128)
    else:
        wl = W.make(2, P=4, per_pair=16, horizon=4)
    n, na, P = wl.n_envs, wl.n_agents, wl.P
    base = wl.seed
    pop = IO.make_population(wl)
    env = IO.make_env(wl)
    ids = torch.from_numpy(wl.pairs.copy()).cuda()
    o_ids = wl.pairs.copy()
    o_ret, o_pid = [], []
    for k in range(iters):
        say(f"[loop] workload={wl.name} round={k} P={P} n={n} T={T}")
        seed = base + 17 * k
        off = k * n
        pop.rollout(env, n, ids, seed, wl.horizon, env_offset=off)
        Mg = pop.payoff_matrix()
        sig, gap = M.solve_fp(Mg, T)
        ids = M.meta_sample_device(sig, P, n, na, seed + 1, env_offset=off)
        # the oracle's loop
        wo = copy.copy(wl)
        wo.seed = seed
        o = oracle.rollout(wo, np.arange(n), o_ids, horizon=wl.horizon, env_offset=off)
        assert o["fails"] == 0
        assert _exact_fixed_point(o["returns"])
        o_ret.append(o["returns"])
        o_pid.append(o_ids)
        mean = oracle.payoff(np.concatenate(o_ret), np.concatenate(o_pid), wl.team, P)[0]
        Mo = oracle.payoff_matrix(mean)
        cx, cy, ogap = oracle.solve_fp(Mo, T)
        o_ids = oracle.meta_sample(np.stack([cx, cy]).astype(np.float32), P, n, na,
                                   seed + 1, off)
        assert np.array_equal(Mg.cpu().numpy().view(np.uint64), Mo.view(np.uint64)), k
        s = sig.cpu().numpy()
        assert np.array_equal(s[0], cx) and np.array_equal(s[1], cy), k
        assert float(gap.cpu()[0]) == ogap
        assert np.array_equal(ids.cpu().numpy(), o_ids), k
    assert pop.payoff()["status"] == 0
    pop.close()


@pytest.mark.parametrize("P", [1, 2, 17, 128, 256])
def test_aggregate_matches_oracle(P):
    """Aggregate payoffs bit for bit (the same sequential fp64 sums on both
    sides), on count-weighted and sparse meta-strategies."""
    import paper_2106_07551_amd as M
    rng = np.random.default_rng(300 + P)
    Mx = rng.normal(size=(P, P))
    sig = np.floor(rng.random((2, P)) * 40).astype(np.float32)
    sig[0, 0] += 1
    sig[1, P // 2] += 1
    if P > 4:
        sig[:, 1::3] = 0
    Md = torch.from_numpy(Mx).cuda()
    sd = torch.from_numpy(sig).cuda()
    for br_row, br_col in ((0, P - 1), (P - 1, 0), (-1, P // 2), (P // 3, -1), (-1, -1)):
        g = M.aggregate(Md, sd, br_row, br_col).cpu().numpy()
        ref = np.array(oracle.aggregate(Mx, sig, br_row, br_col))
        same = (g.view(np.uint64) == ref.view(np.uint64)) | (np.isnan(g) & np.isnan(ref))
        assert same.all(), (br_row, br_col, g, ref)


def test_psro_convergence_on_device():
    """Rock-paper-scissors extended by one dominated policy: fictitious play
    on the device, then the aggregate payoffs of its averages; the new
    policy's gain is negative and the improvement shrinks with more steps."""
    import paper_2106_07551_amd as M
    R = np.array([[0, -1, 1, 2], [1, 0, -1, 2], [-1, 1, 0, 2], [-2, -2, -2, 0]], np.float64)
    Md = torch.from_numpy(R).cuda()
    worst = []
    for T in (10, 100, 1000, 10000):
        sig, gap = M.solve_fp(Md, T)
        out = M.aggregate(Md, sig, 3, 3).cpu().numpy()
        ref = oracle.aggregate(R, sig.cpu().numpy(), 3, 3)
        assert np.array_equal(out.view(np.uint64), np.array(ref).view(np.uint64))
        assert out[2] - out[0] < 0 and out[3] - out[1] < 0
        # no single best response gains more than the exploitability of the
        # averages (which adds both sides' best gains)
        imp = max(float(M.aggregate(Md, sig, br, br).cpu()[4]) for br in range(4))
        assert imp <= float(gap.cpu()[0]) + 1e-12
        worst.append(imp)
    assert worst[-1] < worst[0] and worst[-1] < 0.02
