"""GPU parity at the full workload sizes (the configuration bench.py times).

The whole batch runs on the GPU with an action log and one logits/state
snapshot; the oracle replays a sample of envs in lockstep (the oracle cannot
afford every env at these sizes).  At any size: the table equals the fp64
reduction of the GPU's own per-env returns (counts exact), zero-sum sides are
exact negatives, the bucketing is the stable sort of the pair assignment.
"""
import numpy as np
import pytest

import workloads as W
from gpu_helpers import check_parity, run_gpu, say

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


# (workload number, sampled envs, snapshot step)
CASES = [(1, None, 0), (2, 96, 16), (3, 64, 40), (4, 3, 100), (5, 2, 100)]


@pytest.mark.parametrize("c,n_sel,snap", CASES, ids=[W.NAMES[c[0]] for c in CASES])
def test_fullsize_sampled_parity(c, n_sel, snap):
    wl = W.make(c)
    g = run_gpu(wl, snaps=[snap])
    if n_sel is None:
        sel = None
    else:
        rng = np.random.default_rng(c)
        sel = np.sort(np.concatenate([[0, wl.n_envs - 1],
                                      rng.choice(wl.n_envs, n_sel - 2, replace=False)]))
    rep = check_parity(wl, g, sel)
    say(f"[fullsize] {wl.name}: table cells {int((g['table']['counts'] > 0).sum())}, "
        f"live frames {g['table']['live_frames']}")
    if c in (1, 2, 4):
        per = wl.n_envs // (wl.P * wl.P)
        assert np.all(g["table"]["counts"] == per)
    if c == 5:
        assert g["table"]["counts"].sum() == 16 * wl.n_envs
