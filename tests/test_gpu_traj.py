"""GPU parity of trajectory records: the env-step kernels write one record
per (step, env) into a device ring for learners (the Actors' samples for the
offline dataset server, Sec. 3.1-3.2; the episode buffer of the example API,
Appendix C.2).  Each record is checked against the oracle run in lockstep on
the same envs.

Bars: actions and flags bit for bit; rewards bit for bit (the same fp32
arithmetic as the returns); observations bit for bit (ITER history, PURSUIT
cells, FEATURE bf16_rne of the oracle's fp32 state); returns and the table
bit for bit equal to a rollout without records; the ring keeps exactly the
newest `capacity` records.
"""
import numpy as np
import pytest

import oracle
import workloads as W
from gpu_helpers import TOL, say

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2106_07551_amd as M
    M.lib()


def _obs_spec(wl):
    if wl.env_kind == W.ITER_MATRIX:
        return (), torch.int16
    if wl.env_kind == W.PURSUIT:
        return (2,), torch.uint8
    if wl.env_kind == W.FEATURE:
        return (wl.d,), torch.int16
    return None, None


def _expected(wl, pairs, env_offset, acts, H):
    """Oracle records [H][n] in lockstep with the GPU's actions."""
    n = len(pairs)
    o = oracle.rollout(wl, np.arange(n), pairs, forced=acts, tol=TOL[wl.pol_kind], horizon=H,
                       env_offset=env_offset, want_actions=True, want_states=True,
                       want_rewards=True)
    assert o["fails"] == 0, o["first_fail"]
    row = int(np.nonzero(wl.team > 0)[0][0])
    rew = o["rewards"][:, :, row]
    dead = o["actions"][:, :, 0] == 255
    flags = np.zeros((H, n), np.uint8)
    if wl.env_kind == W.PURSUIT:
        flags |= ((rew == 1.0) & ~dead).astype(np.uint8)
        flags |= (dead.astype(np.uint8) << 2)
    flags[H - 1] |= 2
    obs = None
    if wl.env_kind == W.ITER_MATRIX:
        obs = o["states"].view(np.uint16)
    elif wl.env_kind == W.PURSUIT:
        obs = o["states"][:, :, :2]
    elif wl.env_kind == W.FEATURE:
        obs = np.vectorize(oracle.bf16_bits, otypes=[np.uint16])(o["states"])
    return o, rew, flags, obs


def _run(wl, pairs, H, capacity, *, env_offset=0, cursor=0):
    import paper_2106_07551_amd as M
    from paper_2106_07551_amd import workload_io as IO
    n, na = len(pairs), wl.n_agents
    say(f"[gpu] traj {wl.name} n={n} H={H} cap={capacity} cursor={cursor}")
    pop = IO.make_population(wl)
    env = IO.make_env(wl)
    shp, dt = _obs_spec(wl)
    tr = M.Traj(capacity, na, obs_shape=shp, obs_dtype=dt)
    tr.desc.cursor = cursor
    pt = torch.from_numpy(np.ascontiguousarray(pairs, dtype=np.int32)).cuda()
    ret = torch.empty((na, n), dtype=torch.float32, device="cuda")
    pop.rollout_traj(env, n, pt, wl.seed, H, tr, env_offset=env_offset, returns=ret)
    tab = pop.payoff(reset=True)
    # the same batch without records
    ret2 = torch.empty_like(ret)
    pop.rollout(env, n, pt, wl.seed, H, env_offset=env_offset, returns=ret2)
    tab2 = pop.payoff(reset=True)
    torch.cuda.synchronize()
    assert np.array_equal(ret.cpu().numpy().view(np.uint32), ret2.cpu().numpy().view(np.uint32))
    assert np.array_equal(tab["counts"], tab2["counts"])
    assert np.array_equal(tab["mean"].view(np.uint64), tab2["mean"].view(np.uint64))
    assert tr.cursor == cursor + H * n
    out = {"actions": tr.actions.cpu().numpy(), "rewards": tr.rewards.cpu().numpy(),
           "flags": tr.flags.cpu().numpy(),
           "obs": None if tr.obs is None else tr.obs.cpu().numpy()}
    pop.close()
    return out


def _check(wl, pairs, H, capacity, *, env_offset=0, cursor=0):
    n, na = len(pairs), wl.n_agents
    g = _run(wl, pairs, H, capacity, env_offset=env_offset, cursor=cursor)
    # the newest `capacity` records survive: record k (0 .. H*n-1, k = t*n + e)
    # sits at (cursor + k) mod capacity
    total = H * n
    keep = np.arange(max(0, total - capacity), total)
    slot = (cursor + keep) % capacity
    t_of, e_of = keep // n, keep % n
    acts = np.full((H, n, na), 255, np.uint8)
    acts[t_of, e_of] = g["actions"][slot]
    if capacity < total:
        # lockstep needs every step's actions: take them from a full-size run
        full = _run(wl, pairs, H, total, env_offset=env_offset)
        acts = full["actions"].reshape(H, n, na)
        assert np.array_equal(acts[t_of, e_of], g["actions"][slot])
    o, rew, flags, obs = _expected(wl, pairs, env_offset, acts, H)
    assert np.array_equal(g["actions"][slot], o["actions"][t_of, e_of])
    assert np.array_equal(g["rewards"][slot].view(np.uint32), rew[t_of, e_of].view(np.uint32))
    assert np.array_equal(g["flags"][slot], flags[t_of, e_of])
    if obs is not None:
        got = g["obs"][slot]
        want = obs[t_of, e_of]
        assert np.array_equal(got.view(np.uint8).reshape(len(slot), -1),
                              np.ascontiguousarray(want).view(np.uint8).reshape(len(slot), -1))
    # rewards add up to the returns in step order (fp32)
    if capacity >= total:
        acc = np.zeros(n, np.float32)
        r = g["rewards"][(cursor + np.arange(total)) % capacity].reshape(H, n)
        for t in range(H):
            acc = acc + r[t]
        assert np.array_equal(acc.view(np.uint32),
                              o["returns"][:, int(np.nonzero(wl.team > 0)[0][0])].view(np.uint32))


def test_traj_matrix():
    wl = W.make(1, per_pair=64)
    _check(wl, wl.pairs, 1, 4096)


def test_traj_iter_fp32():
    wl = W.make(2, P=4, per_pair=20, horizon=12)
    _check(wl, wl.pairs, 12, 12 * 320 + 100, cursor=57)


def test_traj_pursuit_with_captures_and_wrap():
    wl = W.make(3, P=6, n_envs=1, horizon=60)
    pairs = W.blocked_pairs(6, 5)
    _check(wl, pairs, 60, 60 * 180)
    _check(wl, pairs, 60, 1000, cursor=123)   # the ring wraps


def test_traj_feature_team_4v4():
    wl = W.make(5, P=8, n_envs=40, horizon=4)
    pairs = W.random_pairs(8, 40, 8)
    _check(wl, pairs, 4, 160, env_offset=9)


def test_traj_feature_d512():
    wl = W.make(4, P=3, per_pair=3, horizon=3)
    _check(wl, wl.pairs, 3, 27)


def test_traj_rejects_bad_ring():
    import paper_2106_07551_amd as M
    from paper_2106_07551_amd import workload_io as IO
    wl = W.make(1, per_pair=4)
    pop = IO.make_population(wl)
    env = IO.make_env(wl)
    pt = torch.from_numpy(wl.pairs).cuda()
    tr = M.Traj(10, 2)
    tr.desc.capacity = 0
    with pytest.raises(M.MalibError):
        pop.rollout_traj(env, wl.n_envs, pt, wl.seed, 1, tr)
    tr.desc.capacity = 10
    tr.desc.rewards = None
    with pytest.raises(M.MalibError):
        pop.rollout_traj(env, wl.n_envs, pt, wl.seed, 1, tr)
    assert pop.payoff()["counts"].sum() == 0
    pop.close()
