"""Graph mode (malib_pop_set_graph) against direct launches.

Two handles built from the same population run the same batches through the C
ABI, one launching directly, one recording each batch into a HIP graph and
replaying it.  Three batches in a row on each: the first instantiates the
executable graph, the second (another seed and env offset, same sizes) updates
it in place, the third (fewer envs) has another launch structure.  Returns,
per-step records and the whole table must be equal bit for bit.  A caller's
own capture (torch.cuda.graph) of a direct-mode batch is replayed several
times, with eager batches between the replays, and every replay checked
against the eager result.
"""
import numpy as np
import pytest

import workloads as W
from gpu_helpers import say

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _pairs(wl):
    import oracle
    if wl.pairs is not None:
        return wl.pairs
    return oracle.meta_sample(wl.sigma, wl.P, wl.n_envs, wl.n_agents, wl.seed)


def _same_table(ta, tb):
    assert np.array_equal(ta["counts"], tb["counts"])
    for k in ("mean", "stderr"):
        assert np.array_equal(np.isnan(ta[k]), np.isnan(tb[k]))
        m = ~np.isnan(ta[k])
        assert np.array_equal(ta[k][m].view(np.uint64), tb[k][m].view(np.uint64)), k
    assert ta["live_frames"] == tb["live_frames"] and ta["envs"] == tb["envs"]
    assert ta["status"] == tb["status"] == 0


CASES = {
    "team_full": lambda: W.make(5),                                   # 16384 x 8, d = 256
    "feature_d512_persistent": lambda: W.make(4, P=4, per_pair=40, horizon=20),
    "feature_1v1_d256": lambda: W.team_variant(2, P=6, n_envs=600, horizon=12),
    "pursuit": lambda: W.make(3, n_envs=4000, horizon=60),
    "iter": lambda: W.make(2, P=8, per_pair=64),
    "matrix": lambda: W.make(1, per_pair=512),
    "iter_generic_f32": lambda: W.with_policies(W.make(2, P=4, per_pair=40, horizon=6),
                                                W.MLP_F32, [24, 80, 48, 3]),
}


@pytest.mark.parametrize("name", list(CASES))
def test_graph_mode_matches_direct(name):
    from paper_2106_07551_amd import workload_io as IO
    wl = CASES[name]()
    pairs = _pairs(wl)
    env = IO.make_env(wl)
    pa, pb = IO.make_population(wl), IO.make_population(wl)
    pb.set_graph(True)
    n1, n2 = wl.n_envs, max(1, wl.n_envs // 3 + 5)
    for n, seed, offset in ((n1, wl.seed, 0), (n1, wl.seed + 1, 777), (n2, wl.seed, 12345)):
        say(f"[graph] {name}: n_envs={n} seed={seed} offset={offset}")
        pt = torch.from_numpy(np.ascontiguousarray(pairs[:n], dtype=np.int32)).cuda()
        out = []
        for pop in (pa, pb):
            ret = torch.empty((wl.n_agents, n), dtype=torch.float32, device="cuda")
            pop.rollout(env, n, pt, seed, wl.horizon, env_offset=offset, returns=ret)
            out.append((ret.cpu().numpy(), pop.payoff(reset=True)))
        (ra, ta), (rb, tb) = out
        assert np.array_equal(ra.view(np.uint32), rb.view(np.uint32)), name
        _same_table(ta, tb)
        assert tb["envs"] == n
    pa.close()
    pb.close()


def test_graph_mode_trajectory_records():
    """malib_rollout_batch_traj in graph mode: the same records and table as
    direct launches, and the ring cursor advanced the same way over two
    batches (the second wraps the ring)."""
    import paper_2106_07551_amd as M
    from paper_2106_07551_amd import workload_io as IO
    wl = W.make(3, n_envs=500, horizon=40)
    env = IO.make_env(wl)
    pt = torch.from_numpy(np.ascontiguousarray(_pairs(wl), dtype=np.int32)).cuda()
    cap = wl.n_envs * wl.horizon + 3000
    res = []
    for graph in (False, True):
        pop = IO.make_population(wl)
        pop.set_graph(graph)
        tr = M.Traj(cap, wl.n_agents, obs_shape=(2,), obs_dtype=torch.uint8)
        tabs = []
        for b in range(2):
            say(f"[graph] traj graph={graph} batch={b}")
            pop.rollout_traj(env, wl.n_envs, pt, wl.seed + b, wl.horizon, tr,
                             env_offset=b * wl.n_envs)
            tabs.append(pop.payoff(reset=True))
        torch.cuda.synchronize()
        res.append((tabs, tr.cursor, {k: getattr(tr, k).cpu().numpy()
                                      for k in ("actions", "rewards", "flags", "obs")}))
        pop.close()
    (ta, ca, ra), (tb, cb, rb) = res
    assert ca == cb == 2 * wl.n_envs * wl.horizon
    for x, y in zip(ta, tb):
        _same_table(x, y)
    for k in ra:
        assert np.array_equal(ra[k].view(np.uint8), rb[k].view(np.uint8)), k


def test_caller_capture_replays():
    """A direct-mode batch captured by the caller (torch.cuda.graph) joins
    that graph: each replay adds one batch to the table, identical to an
    eager batch, with eager batches and synchronisations between replays."""
    from paper_2106_07551_amd import workload_io as IO
    wl = W.make(5, n_envs=2048)
    env = IO.make_env(wl)
    pt = torch.from_numpy(np.ascontiguousarray(_pairs(wl), dtype=np.int32)).cuda()
    eager = IO.make_population(wl)
    ref_ret = torch.empty((wl.n_agents, wl.n_envs), dtype=torch.float32, device="cuda")
    eager.rollout(env, wl.n_envs, pt, wl.seed, wl.horizon, returns=ref_ret)
    ref_tab = eager.payoff(reset=True)
    ref_ret = ref_ret.cpu().numpy()

    pop = IO.make_population(wl)
    ret = torch.empty((wl.n_agents, wl.n_envs), dtype=torch.float32, device="cuda")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        # one eager batch first: the handle's buffers exist before the capture
        pop.rollout(env, wl.n_envs, pt, wl.seed, wl.horizon, returns=ret, stream=s)
        pop.payoff(reset=True, stream=s)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        pop.rollout(env, wl.n_envs, pt, wl.seed, wl.horizon, returns=ret)
    torch.cuda.synchronize()
    assert pop.payoff(reset=True)["envs"] == wl.n_envs    # host-side count of the capture
    for rep in range(3):
        say(f"[graph] caller capture replay {rep}")
        ret.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(ret.cpu().numpy().view(np.uint32), ref_ret.view(np.uint32))
        tab = pop.payoff(reset=True)
        assert np.array_equal(tab["counts"], ref_tab["counts"])
        m = ~np.isnan(ref_tab["mean"])
        assert np.array_equal(tab["mean"][m].view(np.uint64), ref_tab["mean"][m].view(np.uint64))
        # eager work between replays
        eager.rollout(env, wl.n_envs, pt, wl.seed + rep, wl.horizon)
        eager.payoff(reset=True)
    eager.close()
    pop.close()


def test_caller_capture_of_a_larger_batch_is_refused():
    """Under the caller's capture, a batch that would grow the handle's device
    buffers (growing synchronizes the device and frees memory, which a capture
    does not allow) is refused with MALIB_E_INVAL before any device work: the
    capture stays valid and ends cleanly, and the same batch runs afterwards
    outside the capture."""
    from paper_2106_07551_amd import workload_io as IO
    from paper_2106_07551_amd import binding as B
    small, big = W.make(5, n_envs=256, horizon=4), W.make(5, n_envs=1024, horizon=4)
    env = IO.make_env(small)
    p_small = torch.from_numpy(np.ascontiguousarray(_pairs(small), dtype=np.int32)).cuda()
    p_big = torch.from_numpy(np.ascontiguousarray(_pairs(big), dtype=np.int32)).cuda()
    pop = IO.make_population(small)
    pop.rollout(env, small.n_envs, p_small, small.seed, small.horizon)   # buffers for 256 envs
    pop.payoff(reset=True)
    torch.cuda.synchronize()
    x = torch.zeros(16, device="cuda")
    g = torch.cuda.CUDAGraph()
    err = None
    with torch.cuda.graph(g):
        x.add_(1.0)                        # the capture holds one node of its own
        try:
            pop.rollout(env, big.n_envs, p_big, big.seed, big.horizon)
        except B.MalibError as e:
            err = e
    torch.cuda.synchronize()
    assert err is not None and err.status == B.E_INVAL, err
    assert "captured" in str(err)
    g.replay()
    torch.cuda.synchronize()
    assert float(x[0]) == 1.0              # the capture ended valid; nothing of the batch in it
    pop.rollout(env, big.n_envs, p_big, big.seed, big.horizon)
    tab = pop.payoff(reset=True)
    assert tab["envs"] == big.n_envs and tab["status"] == 0
    pop.close()


def test_two_handles_on_two_streams_concurrently():
    """Two handles of the same population, each filling half of a batch on a
    stream of its own at the same time: their returns and merged table equal
    one handle's fill of the whole batch (handles share no device state; the
    fixed-point sums make the merge exact)."""
    import paper_2106_07551_amd as M
    from paper_2106_07551_amd import workload_io as IO
    wl = W.team_variant(8, d=128, P=12, n_envs=2000, horizon=6, dims=[128, 256, 256, 18])
    n, na = wl.n_envs, wl.n_agents
    env = IO.make_env(wl)
    pairs = IO.make_pairs(wl)
    whole = IO.make_population(wl)
    ref = torch.empty((na, n), dtype=torch.float32, device="cuda")
    whole.rollout(env, n, pairs, wl.seed, wl.horizon, returns=ref)
    t_ref = whole.payoff(reset=True)
    halves = [IO.make_population(wl) for _ in range(2)]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    m = n // 2
    rets = [torch.empty((na, m), dtype=torch.float32, device="cuda") for _ in range(2)]
    torch.cuda.synchronize()
    say("[streams] two handles, two streams, halves of 2000 envs")
    for i in range(2):
        halves[i].rollout(env, m, pairs[i * m:(i + 1) * m].contiguous(), wl.seed, wl.horizon,
                          env_offset=i * m, returns=rets[i], stream=streams[i])
    torch.cuda.synchronize()
    assert torch.equal(torch.cat(rets, dim=1), ref)
    tabs = [h.payoff(reset=True) for h in halves]
    cnt = tabs[0]["counts"] + tabs[1]["counts"]
    assert np.array_equal(cnt, t_ref["counts"])
    s = sum(np.nan_to_num(t["mean"]) * t["counts"] for t in tabs)
    merged = np.where(cnt > 0, s / np.maximum(cnt, 1), 0.0)
    assert np.allclose(merged, np.nan_to_num(t_ref["mean"]), rtol=1e-12, atol=1e-12)
    for h in halves + [whole]:
        h.close()
