"""Seeded synthetic workloads for the payoff-table rollout path.

This module only draws inputs: game matrices, environment parameters, policy
weights, meta-strategies and blocked policy-pair assignments.  It holds none of
the method's arithmetic (no observation encoding, no policy forward, no
sampling, no environment rule, no payoff reduction), so both the HIP path and
the CPU oracle can consume the very same bytes.

The five workloads stand in for the paper's evaluation setting, where every
policy combination of a population is simulated many times (2000 simulations
per combination, populations up to 100, Sec. 4.2 "Population-based training for
Leduc Poker") to fill the evaluator's payoff table (Sec. 3.2).  Their shapes:

  matrix   one-step 3x3 zero-sum matrix game, 4 tabular policies, 16 pairs x 1024
  iter     iterated 3x3 matrix game, H=32, fp32 MLP 24-64-64-3, P=16, 256 pairs x 4096
  pursuit  8x8 torus pursuit-evasion, H=100, bf16 MLP 75-256-256-5, P=32, 16384 envs
  feature  R^512 feature dynamics, H=200, bf16 MLP 512-512-512-18, P=64, 4096 pairs x 16
  team     4v4 R^256 feature dynamics, H=200, bf16 MLP 256-512-512-18, P=128,
           16384 envs, per-seat policy drawn from a Dirichlet(1) meta-strategy

Every array is drawn from ``numpy.random.default_rng([2106, 7551, c])`` with c the
workload number (1..5), in a fixed order; ``variant`` adds a fourth seed word so
that tests can draw independent replicas.  Normal distributions are given by
their variance (N(0, 1/fan_in) has standard deviation fan_in**-0.5).
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

# environment families
MATRIX, ITER_MATRIX, PURSUIT, FEATURE = 0, 1, 2, 3
# policy kinds
TABULAR, MLP_F32, MLP_BF16 = 0, 1, 2
# reset modes
INIT_PER_ENV, INIT_SHARED = 0, 1

NAMES = {1: "matrix", 2: "iter", 3: "pursuit", 4: "feature", 5: "team"}
ROLLOUT_KEY_BASE = 0x2106075510000000


@dataclasses.dataclass
class Workload:
    number: int
    name: str
    env_kind: int
    n_agents: int
    n_actions: int
    team: np.ndarray               # int8 [n_agents]: +1 row side, -1 column side
    horizon: int
    n_envs: int
    pol_kind: int
    P: int
    dims: list                     # [in, h1, h2, A] for MLPs; [] for tabular
    weights: list                  # per layer float32 [P][out][in]
    biases: list                   # per layer float32 [P][out] (zeros)
    tab_logits: Optional[np.ndarray] = None   # float32 [P][A]
    A: Optional[np.ndarray] = None            # float32 [n_actions][n_actions]
    grid: int = 0
    d: int = 0
    W: Optional[np.ndarray] = None            # float32 [d][d]
    emb: Optional[np.ndarray] = None          # float32 [n_agents][n_actions][d]
    u: Optional[np.ndarray] = None            # float32 [d]
    sigma: Optional[np.ndarray] = None        # float32 [n_sigma][P]
    pairs: Optional[np.ndarray] = None        # int32 [n_envs][n_agents] (blocked)
    seed: int = 0
    init_mode: int = INIT_PER_ENV

    @property
    def n_slots(self) -> int:
        return self.n_envs * self.n_agents


def _rng(c: int, variant: int) -> np.random.Generator:
    words = [2106, 7551, c] + ([variant] if variant else [])
    return np.random.default_rng(words)


def _antisym(rng: np.random.Generator, n: int) -> np.ndarray:
    A = np.zeros((n, n), dtype=np.float64)
    for i in range(n):
        for j in range(i + 1, n):
            A[i, j] = rng.uniform(-1.0, 1.0)
            A[j, i] = -A[i, j]
    return A.astype(np.float32)


def _normal(rng, var, shape):
    return (rng.standard_normal(shape) * np.sqrt(var)).astype(np.float32)


def _to_bf16_values(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 with the torch library
    (the populations are stored in bf16; this only prepares input bytes)."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).to(torch.float32).numpy()


def _mlp(rng, P, dims, bf16: bool):
    Ws, bs = [], []
    per_pol = [[] for _ in range(len(dims) - 1)]
    for _p in range(P):
        for l in range(len(dims) - 1):
            fan_in, fan_out = dims[l], dims[l + 1]
            per_pol[l].append(_normal(rng, 1.0 / fan_in, (fan_out, fan_in)))
    for l in range(len(dims) - 1):
        w = np.stack(per_pol[l]).astype(np.float32)
        if bf16:
            w = _to_bf16_values(w)
        Ws.append(np.ascontiguousarray(w))
        bs.append(np.zeros((P, dims[l + 1]), dtype=np.float32))
    return Ws, bs


def blocked_pairs(P: int, per_pair: int, n_agents: int = 2) -> np.ndarray:
    """All P*P ordered pairs, each repeated per_pair times: env e plays pair
    e // per_pair = (row, col) = (pair // P, pair % P)."""
    pair = np.arange(P * P * per_pair, dtype=np.int64) // per_pair
    out = np.empty((P * P * per_pair, n_agents), dtype=np.int32)
    out[:, 0] = pair // P
    out[:, 1] = pair % P
    return out


def make(c: int, *, n_envs: Optional[int] = None, horizon: Optional[int] = None,
         P: Optional[int] = None, per_pair: Optional[int] = None,
         variant: int = 0) -> Workload:
    """Build workload ``c`` (1..5).  Overrides shrink it for tests: ``P`` and
    ``per_pair`` (blocked workloads) or ``n_envs`` (sampled ones), ``horizon``."""
    rng = _rng(c, variant)
    seed = ROLLOUT_KEY_BASE + c + (variant << 8)
    if c == 1:
        P = P or 4
        per_pair = per_pair or 1024
        A = _antisym(rng, 3)
        tab = _normal(rng, 1.0, (P, 3))
        wl = Workload(1, "matrix", MATRIX, 2, 3, np.array([1, -1], np.int8),
                      horizon or 1, P * P * per_pair, TABULAR, P, [], [], [],
                      tab_logits=tab, A=A)
        wl.pairs = blocked_pairs(P, per_pair)
    elif c == 2:
        P = P or 16
        per_pair = per_pair or 4096
        A = _antisym(rng, 3)
        dims = [24, 64, 64, 3]
        Ws, bs = _mlp(rng, P, dims, bf16=False)
        wl = Workload(2, "iter", ITER_MATRIX, 2, 3, np.array([1, -1], np.int8),
                      horizon or 32, P * P * per_pair, MLP_F32, P, dims, Ws, bs, A=A)
        wl.pairs = blocked_pairs(P, per_pair)
    elif c == 3:
        P = P or 32
        dims = [75, 256, 256, 5]
        Ws, bs = _mlp(rng, P, dims, bf16=True)
        wl = Workload(3, "pursuit", PURSUIT, 2, 5, np.array([1, -1], np.int8),
                      horizon or 100, n_envs or 16384, MLP_BF16, P, dims, Ws, bs, grid=8)
        wl.sigma = np.full((1, P), 1.0 / P, dtype=np.float32)
    elif c == 4:
        P = P or 64
        per_pair = per_pair or 16
        d = 512
        W = _normal(rng, 1.0 / d, (d, d))
        emb = _normal(rng, 0.1, (2, 18, d))
        u = _normal(rng, 1.0 / d, (d,))
        dims = [d, 512, 512, 18]
        Ws, bs = _mlp(rng, P, dims, bf16=True)
        wl = Workload(4, "feature", FEATURE, 2, 18, np.array([1, -1], np.int8),
                      horizon or 200, P * P * per_pair, MLP_BF16, P, dims, Ws, bs,
                      d=d, W=W, emb=emb, u=u)
        wl.pairs = blocked_pairs(P, per_pair)
    elif c == 5:
        P = P or 128
        d = 256
        W = _normal(rng, 1.0 / d, (d, d))
        emb = _normal(rng, 0.1, (8, 18, d))
        u = _normal(rng, 1.0 / d, (d,))
        sigma = rng.dirichlet(np.ones(P)).astype(np.float32)[None, :]
        dims = [d, 512, 512, 18]
        Ws, bs = _mlp(rng, P, dims, bf16=True)
        wl = Workload(5, "team", FEATURE, 8, 18,
                      np.array([1, 1, 1, 1, -1, -1, -1, -1], np.int8),
                      horizon or 200, n_envs or 16384, MLP_BF16, P, dims, Ws, bs,
                      d=d, W=W, emb=emb, u=u, sigma=sigma)
    else:
        raise ValueError(f"unknown workload {c}")
    wl.seed = seed
    return wl


def team_variant(n_agents: int, *, d: int = 256, P: int = 8, n_envs: int = 64,
                 horizon: int = 4, variant: int = 0, dims=None, team=None) -> Workload:
    """A smaller team game on the feature dynamics, used to pin the team
    reduction by brute force (2v2) and for quick parity cases.  Sides: `team`
    (+1 row side, -1 column side per seat), else the first ceil(n_agents/2)
    seats against the rest."""
    rng = _rng(50 + n_agents, variant)
    W = _normal(rng, 1.0 / d, (d, d))
    emb = _normal(rng, 0.1, (n_agents, 18, d))
    u = _normal(rng, 1.0 / d, (d,))
    sigma = rng.dirichlet(np.ones(P)).astype(np.float32)[None, :]
    dims = dims or [d, 64, 64, 18]
    Ws, bs = _mlp(rng, P, dims, bf16=True)
    if team is None:
        team = [1] * ((n_agents + 1) // 2) + [-1] * (n_agents // 2)
    team = np.array(team, np.int8)
    assert team.shape == (n_agents,)
    wl = Workload(50 + n_agents, f"team{n_agents}", FEATURE, n_agents, 18, team, horizon,
                  n_envs, MLP_BF16, P, dims, Ws, bs, d=d, W=W, emb=emb, u=u, sigma=sigma)
    wl.seed = ROLLOUT_KEY_BASE + 50 + n_agents + (variant << 8)
    return wl


def random_pairs(P: int, n_envs: int, n_agents: int, variant: int = 0) -> np.ndarray:
    """Uniform i.i.d. policy ids (an input-side assignment for tests)."""
    rng = np.random.default_rng([2106, 7551, 99, variant])
    return rng.integers(0, P, size=(n_envs, n_agents), dtype=np.int64).astype(np.int32)


def with_policies(wl: Workload, pol_kind: int, dims, *, variant: int = 0,
                  bias_var: float = 0.0) -> Workload:
    """The same game, pairings and seed with another population of wl.P MLP
    policies of the given kind and dims [in, h1, h2, A] (weights N(0,
    1/fan_in), bf16 values for bf16 policies; biases N(0, bias_var), zero
    when bias_var is 0)."""
    rng = _rng(90 + wl.number, variant)
    Ws, bs = _mlp(rng, wl.P, list(dims), bf16=pol_kind == MLP_BF16)
    if bias_var > 0.0:
        bs = [_normal(rng, bias_var, b.shape) for b in bs]
    out = dataclasses.replace(wl, pol_kind=pol_kind, dims=list(dims), weights=Ws, biases=bs)
    out.name = f"{wl.name}-{'f32' if pol_kind == MLP_F32 else 'bf16'}-" + \
        "x".join(str(x) for x in dims)
    return out
