"""The generic MLP kernel (shapes outside the specialized kernels: unequal
hidden widths, widths up to 1024, fp32 policies on every environment)
against the oracle, replaying every env in lockstep (gpu_helpers.check_parity:
states and returns bit for bit given the same actions, logits within 1e-5
(fp32) / 1e-2 (bf16), counted near ties, the table within 1e-3 of the
oracle's); nonzero biases; a NaN hidden weight raises the NaN flag; growing a
generic population equals creating it at the larger size."""
import numpy as np
import pytest

import oracle
import workloads as W
from gpu_helpers import check_parity, run_gpu, say

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


CASES = {
    "iter_f32_96x40": lambda: W.with_policies(W.make(2, P=4, per_pair=9, horizon=6), W.MLP_F32,
                                              [24, 96, 40, 3], bias_var=0.05),
    "iter_bf16_48": lambda: W.with_policies(W.make(2, P=3, per_pair=11, horizon=5), W.MLP_BF16,
                                            [24, 48, 48, 3]),
    "pursuit_f32_64x32": lambda: W.with_policies(W.make(3, P=5, n_envs=150, horizon=30),
                                                 W.MLP_F32, [75, 64, 32, 5], bias_var=0.05),
    "pursuit_bf16_100x60": lambda: W.with_policies(W.make(3, P=4, n_envs=120, horizon=25),
                                                   W.MLP_BF16, [75, 100, 60, 5]),
    "feature_bf16_1024": lambda: W.with_policies(W.team_variant(2, d=64, P=3, n_envs=40,
                                                                horizon=4),
                                                 W.MLP_BF16, [64, 1024, 1024, 18],
                                                 bias_var=0.01),
    "team2v2_f32_200x72": lambda: W.with_policies(W.team_variant(4, d=128, P=5, n_envs=60,
                                                                 horizon=5),
                                                  W.MLP_F32, [128, 200, 72, 18]),
    "feature_bf16_d512_1000": lambda: W.with_policies(W.make(4, P=2, per_pair=5, horizon=3),
                                                      W.MLP_BF16, [512, 1000, 17, 18]),
}


@pytest.mark.parametrize("name", list(CASES))
def test_generic_parity(name):
    wl = CASES[name]()
    say(f"[generic] {name}: P={wl.P} envs={wl.n_envs} dims={wl.dims}")
    g = run_gpu(wl, snaps=[0, wl.horizon - 1])
    rep = check_parity(wl, g)
    say(f"[generic] {name}: {rep}")
    assert rep["fails"] == 0


@pytest.mark.parametrize("layer", [0, 1])
def test_generic_nan_hidden_weight_flagged(layer):
    import paper_2106_07551_amd as M
    wl = W.with_policies(W.make(3, P=2, n_envs=60, horizon=3), W.MLP_BF16, [75, 40, 30, 5])
    wl.weights = [w.copy() for w in wl.weights]
    wl.weights[layer][1, 2, 3] = np.float32("nan")
    g = run_gpu(wl, snaps=[0], check=False)
    t = g["table"]
    assert t["status"] == M.binding.E_DEVICE and t["device_flags"] & 2
    clean = np.nonzero(~(g["pairs"] == 1).any(axis=1))[0]
    if len(clean):
        check_parity(wl, g, clean)


def test_generic_extend_equals_create():
    """A generic population of 3 policies grown by 2 gives the same table as
    the population created with all 5, on the same batch."""
    import paper_2106_07551_amd as M
    from paper_2106_07551_amd import workload_io as IO
    wl = W.with_policies(W.make(2, P=5, per_pair=6, horizon=4), W.MLP_F32, [24, 70, 33, 3],
                         bias_var=0.05)
    env = IO.make_env(wl)
    pt = torch.from_numpy(wl.pairs).cuda()

    def dev(a):
        return torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda()

    full = IO.make_population(wl)
    grown = M.Population(wl.pol_kind, 3, wl.n_actions, dims=wl.dims,
                         weights=[dev(w[:3]) for w in wl.weights],
                         biases=[dev(b[:3]) for b in wl.biases])
    grown.extend(2, weights=[dev(w[3:]) for w in wl.weights],
                 biases=[dev(b[3:]) for b in wl.biases])
    tabs = []
    for pop in (full, grown):
        pop.rollout(env, wl.n_envs, pt, wl.seed, wl.horizon)
        tabs.append(pop.payoff())
        pop.close()
    a, b = tabs
    assert np.array_equal(a["counts"], b["counts"])
    m = ~np.isnan(a["mean"])
    assert np.array_equal(a["mean"][m].view(np.uint64), b["mean"][m].view(np.uint64))
