"""Shared GPU-vs-oracle parity machinery for the -m gpu tests.

The HIP path runs through the C ABI (paper_2106_07551_amd); the oracle runs the
selected envs in lockstep on the GPU's action log: a differing action is
accepted only where the oracle's own top-two Gumbel-perturbed values are
within the policy tolerance (counted), and everything after is compared from
the same actions.
"""
from __future__ import annotations

import sys

import numpy as np

import oracle
import workloads as W

TOL = {W.MLP_F32: 1e-5, W.MLP_BF16: 1e-2, W.TABULAR: 1e-5}


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def run_gpu(wl, *, horizon=None, snaps=(0,), pairs=None, env_offset=0, trace=True,
            check=True):
    """One rollout batch on the GPU with a full trace; returns host arrays.
    ``check=False`` returns the table even when the device flagged bad data
    (its status and flags are in the table dict)."""
    import torch
    import paper_2106_07551_amd as M
    from paper_2106_07551_amd import workload_io as IO
    H = wl.horizon if horizon is None else horizon
    n = wl.n_envs
    ns = n * wl.n_agents
    say(f"[gpu] workload={wl.name} n_envs={n} agents={wl.n_agents} P={wl.P} H={H} "
        f"offset={env_offset}")
    pop = IO.make_population(wl)
    env = IO.make_env(wl)
    if pairs is None:
        pairs_t = IO.make_pairs(wl, env_offset=env_offset)
    else:
        pairs_t = torch.from_numpy(np.ascontiguousarray(pairs, dtype=np.int32)).cuda()
    ret = torch.empty((wl.n_agents, n), dtype=torch.float32, device="cuda")
    tr = None
    bufs = {}
    if trace:
        snaps = [s for s in snaps if s < H]
        bufs["actions"] = torch.empty((H, ns), dtype=torch.uint8, device="cuda")
        bufs["logits"] = torch.empty((len(snaps), ns, wl.n_actions), dtype=torch.float32,
                                     device="cuda")
        shp, dt = oracle.state_shape(wl, n)
        if shp is not None:
            tdt = {np.uint16: torch.int16, np.uint8: torch.uint8, np.float32: torch.float32}[dt]
            bufs["states"] = torch.empty((len(snaps),) + shp, dtype=tdt, device="cuda")
        if wl.pol_kind != W.TABULAR:
            bufs["perm"] = torch.empty(ns, dtype=torch.int32, device="cuda")
            bufs["offsets"] = torch.empty(wl.P + 1, dtype=torch.int32, device="cuda")
        tr = M.Trace(snap_steps=snaps, **bufs)
    pop.rollout(env, n, pairs_t, wl.seed, H, env_offset=env_offset, returns=ret, trace=tr)
    tab = pop.payoff(check=check)
    torch.cuda.synchronize()
    out = {"returns": ret.cpu().numpy().T.copy(), "pairs": pairs_t.cpu().numpy(),
           "table": tab, "snaps": list(snaps), "H": H}
    for k, v in bufs.items():
        a = v.cpu().numpy()
        if k == "states" and a.dtype == np.int16:
            a = a.view(np.uint16)
        out[k] = a
    pop.close()
    return out


def check_parity(wl, g, sel=None, *, env_offset=0, check_table_vs_oracle=None):
    """Compare a GPU run ``g`` with the oracle on envs ``sel`` (default: all)."""
    H = g["H"]
    n, na = wl.n_envs, wl.n_agents
    sel = np.arange(n) if sel is None else np.asarray(sel)
    tol = TOL[wl.pol_kind]
    acts = g["actions"].reshape(H, n, na)[:, sel, :]
    say(f"[oracle] workload={wl.name} envs={len(sel)} H={H}")
    o = oracle.rollout_threads(wl, sel, g["pairs"][sel], forced=acts, tol=tol, horizon=H,
                               env_offset=env_offset, want_actions=True, want_logits=True,
                               want_states=True)
    rep = {"near_ties": o["near_ties"], "flips": o["flips"], "fails": o["fails"],
           "first_fail": o["first_fail"]}
    assert o["fails"] == 0, rep
    # finished envs: both sides mark 255 at the same steps
    assert np.array_equal(acts == 255, o["actions"] == 255)
    # returns bit for bit (same actions, same fp32 order)
    assert np.array_equal(g["returns"][sel].view(np.uint32), o["returns"].view(np.uint32)), \
        np.abs(g["returns"][sel] - o["returns"]).max()
    # zero-sum sides, bit for bit
    row = np.nonzero(wl.team > 0)[0]
    col = np.nonzero(wl.team < 0)[0]
    for a in row:
        assert np.array_equal(g["returns"][:, a], g["returns"][:, row[0]])
    for b in col:
        assert np.array_equal(g["returns"][:, b], -g["returns"][:, row[0]])
    # logits at the snapshot steps, live rows only
    worst = 0.0
    for i, t in enumerate(g["snaps"]):
        lg = g["logits"][i].reshape(n, na, -1)[sel]
        lo = o["logits"][t]
        live = o["actions"][t] != 255
        if not live.any():
            continue
        scale = np.maximum(1.0, np.abs(lo).max(axis=-1))
        err = (np.abs(lg - lo).max(axis=-1) / scale)[live]
        worst = max(worst, float(err.max()))
    rep["logit_rel_err"] = worst
    assert worst <= tol, rep
    # states before the snapshot steps, bit for bit
    if "states" in g:
        for i, t in enumerate(g["snaps"]):
            gs = g["states"][i][sel]
            os_ = o["states"][t]
            assert np.array_equal(gs.view(np.uint8), os_.view(np.uint8)), (wl.name, t)
    # bucketing: stable sort of slots by policy id
    if "perm" in g:
        pid = g["pairs"].reshape(-1)
        assert np.array_equal(g["perm"], np.argsort(pid, kind="stable"))
        cnt = np.bincount(pid, minlength=wl.P)
        assert np.array_equal(g["offsets"], np.concatenate([[0], np.cumsum(cnt)]))
    # payoff table
    tab = g["table"]
    full = len(sel) == n
    ref_ret = o["returns"] if full else g["returns"]
    mean, cnt, s1, s2 = oracle.payoff(ref_ret, g["pairs"], wl.team, wl.P)
    assert np.array_equal(tab["counts"], cnt)
    assert np.array_equal(np.isnan(tab["mean"]), cnt == 0)
    m = cnt > 0
    rep["payoff_max_abs"] = float(np.abs(tab["mean"][m] - mean[m]).max()) if m.any() else 0.0
    assert rep["payoff_max_abs"] <= (1e-3 if full else 1e-9), rep
    # standard error of the mean, sqrt(sample variance / n), NaN below two
    # simulations; the table keeps squares in 2^-20 fixed point, so its sum of
    # squares is within n * 2^-21 of the exact one and its variance within
    # 2^-21 * n / (n - 1) (+ fp64 cancellation); since |sqrt(a) - sqrt(b)| <=
    # sqrt(|a - b|), the SE is within sqrt(2^-20 / (n - 1) + 1e-13 * s2 / n^2)
    se_gpu = tab["stderr"]
    assert np.array_equal(np.isnan(se_gpu), cnt < 2)
    k = cnt >= 2
    if k.any():
        n = cnt[k].astype(np.float64)
        var = np.maximum(s2[k] - s1[k] * s1[k] / n, 0.0) / (n - 1.0)
        se_ora = np.sqrt(var / n)
        tol_se = np.sqrt(2.0 ** -20 / (n - 1.0) + 1e-13 * s2[k] / (n * n))
        err = np.abs(se_gpu[k] - se_ora)
        rep["stderr_max_abs"] = float(err.max())
        assert np.all(err <= tol_se), (rep, float((err / tol_se).max()))
    if full:
        assert tab["live_frames"] == o["live_frames"]
    say(f"[parity] {wl.name}: {rep}")
    return rep
