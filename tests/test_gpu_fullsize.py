"""GPU parity at the full workload sizes (the configuration bench.py times).

The whole batch runs on the GPU with an action log and logits/state snapshots
at the first, middle and last step; the oracle replays a selection of envs in
lockstep (it cannot afford every env at these sizes).  The selection covers
every policy of the population: for the 4v4 game a greedy cover of every
policy the meta-strategy drew (nearly all 128) plus envs spread over the rows
of the largest bucket (the policy with the most slots, thousands of rows over
many tiles); for the d=512 feature game
one env per (row policy, column policy) diagonal so that all 64 row and all 64
column policies play.  At any size: the table equals the fp64 reduction of the
GPU's own per-env returns (counts exact, standard errors within the fixed-point
bound), zero-sum sides are exact negatives, the bucketing is the stable sort of
the pair assignment.
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


def _cover_all_policies(pairs, P, rng):
    """Envs, chosen greedily, whose seats together play every policy that
    appears in ``pairs`` [n_envs][n_agents]."""
    left = set(np.unique(pairs).tolist())
    order = rng.permutation(len(pairs))
    chosen = []
    while left:
        best, gain = -1, 0
        for e in order:
            g = len(left.intersection(pairs[e].tolist()))
            if g > gain:
                best, gain = int(e), g
        chosen.append(best)
        left -= set(pairs[best].tolist())
    return chosen


def _largest_bucket_envs(pairs, k):
    """k envs spread over the sorted rows of the most played policy."""
    flat = pairs.reshape(-1)
    p = int(np.bincount(flat).argmax())
    slots = np.nonzero(flat == p)[0]             # the bucket's rows, in sorted order
    pick = slots[np.linspace(0, len(slots) - 1, k).astype(int)]
    return p, len(slots), (pick // pairs.shape[1]).tolist()


def _selection(c, wl, g):
    rng = np.random.default_rng(c)
    n = wl.n_envs
    if c == 1:
        return None
    if c == 5:
        pairs = g["pairs"]
        cover = _cover_all_policies(pairs, wl.P, rng)
        p, rows, big = _largest_bucket_envs(pairs, 8)
        played = len(np.unique(pairs))
        say(f"[fullsize] team: {len(cover)} envs cover all {played} played policies (of "
            f"{wl.P}); largest bucket policy {p} with {rows} rows, 8 envs over it")
        sel = np.unique(np.concatenate([[0, n - 1], cover, big]))
        assert len(np.unique(pairs[sel])) == played
        return sel
    if c == 4:
        per = n // (wl.P * wl.P)
        # env of pair (r, (r + 17) % P), a different repetition for each r
        cells = [(r * wl.P + (r + 17) % wl.P) * per + r % per for r in range(wl.P)]
        sel = np.unique(np.concatenate([[0, n - 1], cells]))
        assert len(np.unique(g["pairs"][sel, 0])) == wl.P
        assert len(np.unique(g["pairs"][sel, 1])) == wl.P
        return sel
    n_sel = {2: 96, 3: 64}[c]
    return np.sort(np.concatenate([[0, n - 1], rng.choice(np.arange(1, n - 1), n_sel - 2,
                                                           replace=False)]))


CASES = [1, 2, 3, 4, 5]


@pytest.mark.parametrize("c", CASES, ids=[W.NAMES[c] for c in CASES])
def test_fullsize_sampled_parity(c):
    wl = W.make(c)
    H = wl.horizon
    snaps = sorted({0, H // 2, H - 1})
    g = run_gpu(wl, snaps=snaps)
    sel = _selection(c, wl, g)
    rep = check_parity(wl, g, sel)
    say(f"[fullsize] {wl.name}: envs {wl.n_envs if sel is None else len(sel)}, snapshots "
        f"{snaps}, table cells {int((g['table']['counts'] > 0).sum())}, "
        f"live frames {g['table']['live_frames']}, {rep}")
    if c in (1, 2, 4):
        per = wl.n_envs // (wl.P * wl.P)
        assert np.all(g["table"]["counts"] == per)
    if c == 5:
        assert g["table"]["counts"].sum() == 16 * wl.n_envs


@pytest.mark.parametrize("n_envs", [5000, 2043])
def test_team_env_step_workgroup_sizes(n_envs):
    """The 4v4 game at batch sizes whose env step runs 16-env workgroups (5000
    envs: 2 per thread, the last workgroup half full) and 8-env workgroups
    (2043 envs: 1 per thread, the last one with 3): lockstep parity on envs
    that cover every played policy plus both ends of the batch, the table
    against the GPU's own returns."""
    wl = W.make(5, n_envs=n_envs, horizon=12)
    H = wl.horizon
    snaps = sorted({0, H // 2, H - 1})
    g = run_gpu(wl, snaps=snaps)
    sel = _selection(5, wl, g)
    rep = check_parity(wl, g, sel)
    say(f"[team {n_envs} envs] envs {len(sel)}, snapshots {snaps}, {rep}")
    assert g["table"]["counts"].sum() == 16 * wl.n_envs
