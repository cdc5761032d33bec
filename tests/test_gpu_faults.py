"""Forced allocation failures (MALIB_FAULT_ALLOC) on the GPU, through the C
ABI: creating a handle, extending it, and growing its batch buffers each
return MALIB_E_NOMEM and leave everything as it was (the partly built handle
is released; an extension keeps the old weights, ids and table; a batch that
could not grow its buffers leaves the table untouched), and the same calls
succeed once the hook is cleared."""
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


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def _pairs(wl, n):
    import oracle
    return torch.from_numpy(np.ascontiguousarray(
        oracle.meta_sample(wl.sigma, wl.P, n, wl.n_agents, wl.seed), dtype=np.int32)).cuda()


def test_create_under_forced_nomem(monkeypatch):
    from paper_2106_07551_amd import binding as B
    from paper_2106_07551_amd import workload_io as IO
    wl = W.team_variant(4, P=6, n_envs=64, horizon=3)
    monkeypatch.setenv("MALIB_FAULT_ALLOC", "1")
    with pytest.raises(B.MalibError) as ei:
        IO.make_population(wl)
    assert ei.value.status == B.E_NOMEM
    monkeypatch.delenv("MALIB_FAULT_ALLOC")
    pop = IO.make_population(wl)
    env = IO.make_env(wl)
    pop.rollout(env, wl.n_envs, _pairs(wl, wl.n_envs), wl.seed, wl.horizon)
    tab = pop.payoff(reset=True)
    assert tab["envs"] == wl.n_envs and tab["status"] == 0
    pop.close()


def test_extend_and_batch_growth_under_forced_nomem(monkeypatch):
    from paper_2106_07551_amd import binding as B
    from paper_2106_07551_amd import workload_io as IO
    wl = W.team_variant(4, P=5, n_envs=128, horizon=3)
    extra = W.team_variant(4, P=6, n_envs=8, horizon=3)     # a sixth policy of the same dims
    env = IO.make_env(wl)
    pop = IO.make_population(wl)
    p_small = _pairs(wl, wl.n_envs)
    pop.rollout(env, wl.n_envs, p_small, wl.seed, wl.horizon)
    before = pop.payoff(reset=False)
    # extension: fails, the handle keeps its policies, ids and table
    monkeypatch.setenv("MALIB_FAULT_ALLOC", "1")
    new = {"weights": [_dev(w[5:6]) for w in extra.weights],
           "biases": [_dev(b[5:6]) for b in extra.biases] if extra.biases else None}
    with pytest.raises(B.MalibError) as ei:
        pop.extend(1, **new)
    assert ei.value.status == B.E_NOMEM
    assert pop.P == 5 and list(pop.policy_ids()) == list(range(5))
    # a batch that needs larger buffers: fails before any device work
    p_big = _pairs(wl, 4 * wl.n_envs)
    with pytest.raises(B.MalibError) as ei:
        pop.rollout(env, 4 * wl.n_envs, p_big, wl.seed, wl.horizon)
    assert ei.value.status == B.E_NOMEM
    monkeypatch.delenv("MALIB_FAULT_ALLOC")
    after = pop.payoff(reset=False)
    say(f"[faults] table envs before {before['envs']} after {after['envs']}")
    assert after["envs"] == before["envs"]
    assert np.array_equal(after["counts"], before["counts"])
    m = ~np.isnan(before["mean"])
    assert np.array_equal(after["mean"][m].view(np.uint64), before["mean"][m].view(np.uint64))
    # cleared: the same extension and batch succeed
    pop.extend(1, **new)
    assert pop.P == 6 and list(pop.policy_ids()) == list(range(6))
    pop.rollout(env, 4 * wl.n_envs, p_big, wl.seed, wl.horizon)
    tab = pop.payoff(reset=True)
    assert tab["envs"] == 5 * wl.n_envs and tab["status"] == 0
    pop.close()


def test_handle_alive_at_interpreter_exit():
    """A population still alive when the interpreter exits (a module-level
    handle) neither raises from its finalizer nor calls into the torn-down
    runtime: the process exits 0 with nothing on stderr about it."""
    import os
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    code = (
        "import sys; sys.path.insert(0, %r)\n"
        "import numpy as np, torch, workloads as W\n"
        "from paper_2106_07551_amd import workload_io as IO\n"
        "wl = W.make(1, P=3, per_pair=4)\n"
        "pop = IO.make_population(wl); env = IO.make_env(wl)\n"
        "pop.rollout(env, wl.n_envs, IO.make_pairs(wl), wl.seed, 1)\n"
        "assert pop.payoff()['counts'].sum() == wl.n_envs\n"
        "print('done', flush=True)\n" % root)
    say("[exit] module-level handle in a child process")
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 0, r.stderr[-2000:]
    assert "done" in r.stdout
    assert "Exception ignored" not in r.stderr and "Traceback" not in r.stderr, r.stderr[-2000:]
