"""Upload a generated workload (workloads.Workload) to the device and create
its population / environment handles and policy-pair assignment."""
from __future__ import annotations

import numpy as np

from . import binding as B


def _t(a, dtype=None):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a))
    return t.to(device="cuda", dtype=dtype) if dtype is not None else t.to("cuda")


def make_population(wl, stream=None) -> B.Population:
    import torch
    if wl.pol_kind == B.POLICY_TABULAR:
        return B.Population(B.POLICY_TABULAR, wl.P, wl.n_actions,
                            tab_logits=_t(wl.tab_logits, torch.float32), stream=stream)
    ws = [_t(w, torch.float32) for w in wl.weights]
    bs = [_t(b, torch.float32) for b in wl.biases] if wl.biases else None
    pop = B.Population(wl.pol_kind, wl.P, wl.n_actions, dims=list(wl.dims), weights=ws,
                       biases=bs, stream=stream)
    del ws, bs
    return pop


def make_env(wl) -> B.Env:
    import torch
    f = lambda a: None if a is None else _t(a, torch.float32)
    return B.Env(wl.env_kind, wl.n_agents, wl.n_actions, team=list(wl.team), A=f(wl.A),
                 grid=wl.grid, d=wl.d, W=f(wl.W), emb=f(wl.emb), u=f(wl.u),
                 init_mode=wl.init_mode)


def make_pairs(wl, n_envs=None, env_offset=0, stream=None):
    """Blocked assignment from the workload, else a meta-sample from its sigma."""
    import torch
    n = wl.n_envs if n_envs is None else n_envs
    if wl.pairs is not None:
        return _t(wl.pairs[env_offset:env_offset + n], torch.int32)
    return B.meta_sample(wl.sigma, wl.P, n, wl.n_agents, wl.seed, env_offset=env_offset,
                         stream=stream)
