"""GPU parity of incremental payoff-table expansion: a population of P0
policies fills its table, grows to P (malib_pop_extend), and one batch
simulates only the new rows and columns (malib_expansion_pairs) into the same
table (Sec. 3.1's auto-curriculum adds policies; the example API extends the
pool and simulates the new combinations, Appendix C.2).  The oracle rolls out
the same envs with the grown population and builds the table from both
batches.

Bars: the expansion batch's policy ids bit for bit; every rollout in lockstep
with the oracle (0 failures, returns bit for bit); the merged table's counts
exact and its means within 1e-9 of the oracle's fp64 reduction of the same
returns; the old block of the table bit for bit unchanged by the extension.
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


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def _policies(wl, lo, hi):
    """Keyword arguments of Population / extend for policies lo .. hi-1."""
    if wl.pol_kind == W.TABULAR:
        return {"tab_logits": _dev(wl.tab_logits[lo:hi])}
    return {"weights": [_dev(w[lo:hi]) for w in wl.weights],
            "biases": [_dev(b[lo:hi]) for b in wl.biases] if wl.biases else None}


def _roll(pop, env, wl, pairs, env_offset):
    """One traced batch on the GPU and the oracle in lockstep on it."""
    import paper_2106_07551_amd as M
    n, H = len(pairs), wl.horizon
    say(f"[gpu] {wl.name} rollout n={n} P={pop.P} offset={env_offset}")
    acts = torch.empty((H, n * wl.n_agents), dtype=torch.uint8, device="cuda")
    ret = torch.empty((wl.n_agents, n), dtype=torch.float32, device="cuda")
    pt = torch.from_numpy(np.ascontiguousarray(pairs, dtype=np.int32)).cuda()
    pop.rollout(env, n, pt, wl.seed, H, env_offset=env_offset, returns=ret,
                trace=M.Trace(actions=acts))
    torch.cuda.synchronize()
    g_ret = ret.cpu().numpy().T.copy()
    a = acts.cpu().numpy().reshape(H, n, wl.n_agents)
    o = oracle.rollout(wl, np.arange(n), pairs, forced=a, tol=TOL[wl.pol_kind],
                       env_offset=env_offset)
    assert o["fails"] == 0, o["first_fail"]
    assert np.array_equal(g_ret.view(np.uint32), o["returns"].view(np.uint32))
    return o["returns"]


def _bits(x):
    return np.ascontiguousarray(x).view(np.uint64)


def _check_expansion(wl, P0, steps, pairs0, per_pair):
    """Fill with P0 policies, then grow by `steps` (policy counts), simulating
    each growth's new cells; compare with the oracle after every stage."""
    import paper_2106_07551_amd as M
    from paper_2106_07551_amd import workload_io as IO
    team = np.asarray(wl.team)
    env = IO.make_env(wl)
    pop = M.Population(wl.pol_kind, P0, wl.n_actions, dims=wl.dims, **_policies(wl, 0, P0))
    rets, pids = [_roll(pop, env, wl, pairs0, 0)], [pairs0]
    off = len(pairs0)
    P = P0
    for k in steps:
        before = pop.payoff()
        pop.extend(k, **_policies(wl, P, P + k))
        after = pop.payoff()
        assert pop.P == P + k and after["counts"].shape == (P + k, P + k)
        assert np.array_equal(after["counts"][:P, :P], before["counts"])
        assert np.array_equal(_bits(after["mean"][:P, :P]), _bits(before["mean"]))
        assert (after["counts"][P:, :] == 0).all() and (after["counts"][:, P:] == 0).all()
        assert after["live_frames"] == before["live_frames"]
        new = M.expansion_pairs(P + k, P, per_pair, wl.n_agents, team).cpu().numpy()
        assert np.array_equal(new, oracle.expansion_pairs(P + k, P, per_pair, team))
        rets.append(_roll(pop, env, wl, new, off))
        pids.append(new)
        off += len(new)
        P += k
        tab = pop.payoff()
        mean, cnt, _, _ = oracle.payoff(np.concatenate(rets), np.concatenate(pids), team, P)
        assert np.array_equal(tab["counts"], cnt)
        m = cnt > 0
        assert np.abs(tab["mean"][m] - mean[m]).max() <= 1e-9
        assert np.array_equal(np.isnan(tab["mean"]), ~m)
        # the device game grows with the table
        g = pop.payoff_matrix().cpu().numpy()
        assert g.shape == (P, P)
        assert np.array_equal(_bits(g), _bits(np.where(m, tab["mean"], 0.0)))
    assert pop.payoff(reset=True)["status"] == 0
    pop.close()


@pytest.mark.parametrize("P,f,per_pair,team", [
    (5, 3, 7, [1, -1]), (4, 0, 3, [1, -1]), (256, 255, 2, [1, -1]),
    (128, 100, 1, [1, 1, 1, 1, -1, -1, -1, -1]), (9, 2, 5, [-1, 1, 1])])
def test_expansion_pairs_match_oracle(P, f, per_pair, team):
    import paper_2106_07551_amd as M
    team = np.array(team, np.int8)
    g = M.expansion_pairs(P, f, per_pair, len(team), team).cpu().numpy()
    assert np.array_equal(g, oracle.expansion_pairs(P, f, per_pair, team))


def test_expand_matrix_tabular():
    wl = W.make(1, P=6, per_pair=32)
    _check_expansion(wl, 3, [2, 1], W.blocked_pairs(3, 32), 32)


def test_expand_iter_fp32_with_biases():
    """fp32 MLP: packed weights and nonzero biases of old and new policies
    both land where the forward looks for them."""
    wl = W.make(2, P=7, per_pair=6, horizon=6)
    rng = np.random.default_rng(5)
    wl.biases = [rng.normal(0, 0.3, b.shape).astype(np.float32) for b in wl.biases]
    _check_expansion(wl, 4, [1, 2], W.blocked_pairs(4, 6), 6)


def test_expand_pursuit_bf16():
    wl = W.make(3, P=10, n_envs=1, horizon=40)
    _check_expansion(wl, 7, [3], W.blocked_pairs(7, 4), 4)


def test_expand_team_feature_bf16():
    """The 4v4 team game (d=256, bf16 256-512-512-18): row-side seats take the
    cell's row policy, column-side seats its column policy."""
    wl = W.make(5, P=4, n_envs=24, horizon=3)
    rng = np.random.default_rng(6)
    pairs0 = rng.integers(0, 3, size=(24, 8)).astype(np.int32)
    _check_expansion(wl, 3, [1], pairs0, 2)


def test_extend_rejects_mismatch_and_keeps_population():
    """Extensions that do not fit the population fail on the host and leave
    the population and its table as they were."""
    import paper_2106_07551_amd as M
    from paper_2106_07551_amd import workload_io as IO
    B = M.binding
    wl = W.make(2, P=5, per_pair=4, horizon=2)
    pop = M.Population(wl.pol_kind, 4, wl.n_actions, dims=wl.dims, **_policies(wl, 0, 4))
    env = IO.make_env(wl)
    pop.rollout(env, 16, torch.from_numpy(W.blocked_pairs(4, 4)).cuda(), wl.seed, 2)
    before = pop.payoff()
    # hidden width 32 against the population's 64
    w32 = [_dev(np.zeros((1, 32, 24))), _dev(np.zeros((1, 32, 32))), _dev(np.zeros((1, 3, 32)))]
    d, keep = B._pop_desc(wl.pol_kind, 1, wl.n_actions, [24, 32, 32, 3], w32, None, None)
    assert B.lib().malib_pop_extend(pop.handle, B.C.byref(d), None) == B.E_INVAL
    # another policy kind
    d, keep = B._pop_desc(M.POLICY_TABULAR, 1, wl.n_actions, None, (), None,
                          _dev(np.zeros((1, 3))))
    assert B.lib().malib_pop_extend(pop.handle, B.C.byref(d), None) == B.E_INVAL
    with pytest.raises(M.MalibError):
        pop.extend(1)                                 # no weights
    with pytest.raises(M.MalibError):
        pop.extend(253, **_policies(wl, 0, 1))        # 4 + 253 > 256
    assert pop.P == 4
    after = pop.payoff()
    assert np.array_equal(after["counts"], before["counts"])
    assert np.array_equal(_bits(after["mean"]), _bits(before["mean"]))
    pop.extend(1, **_policies(wl, 4, 5))
    assert pop.payoff()["counts"].shape == (5, 5)
    pop.close()


def test_policy_ids_echoed_and_extended():
    """The caller's policy ids (Sec. 3.1 pools keyed by policy id; Appendix
    C.2 distributions Dict[PolicyID, float]) come back in index order, default
    to the indices, grow with malib_pop_extend; a colliding id is rejected and
    leaves the population, its ids and its table unchanged."""
    import paper_2106_07551_amd as M
    from paper_2106_07551_amd import workload_io as IO
    wl = W.make(1, P=4, per_pair=16)
    ids = [1001, -7, 42, 2 ** 40]
    pop = M.Population(M.POLICY_TABULAR, 3, 3, policy_ids=ids[:3],
                       **_policies(wl, 0, 3))
    assert pop.policy_ids().tolist() == ids[:3]
    pairs = wl.pairs[(wl.pairs < 3).all(axis=1)]
    env = IO.make_env(wl)
    pop.rollout(env, len(pairs), torch.from_numpy(pairs).cuda(), wl.seed, 1)
    before = pop.payoff()
    with pytest.raises(M.MalibError) as e:
        pop.extend(1, policy_ids=[42], **_policies(wl, 3, 4))
    assert e.value.status == M.binding.E_INVAL
    assert pop.P == 3 and pop.policy_ids().tolist() == ids[:3]
    after = pop.payoff()
    assert np.array_equal(after["counts"], before["counts"])
    pop.extend(1, policy_ids=ids[3:], **_policies(wl, 3, 4))
    assert pop.policy_ids().tolist() == ids
    t = pop.payoff()
    assert np.array_equal(t["counts"][:3, :3], before["counts"])
    pop.close()
    dflt = M.Population(M.POLICY_TABULAR, 3, 3, **_policies(wl, 0, 3))
    assert dflt.policy_ids().tolist() == [0, 1, 2]
    dflt.extend(1, **_policies(wl, 3, 4))
    assert dflt.policy_ids().tolist() == [0, 1, 2, 3]
    with pytest.raises(M.MalibError):
        M.Population(M.POLICY_TABULAR, 3, 3, policy_ids=[9, 9, 1], **_policies(wl, 0, 3))
    dflt.close()
