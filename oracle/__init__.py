"""CPU oracle for the population payoff-table rollout path.

TEST INFRASTRUCTURE ONLY: tests/, __graft_entry__.smoke() and the cpu_baseline
leg of bench.py are the only callers.  The product library never imports,
links or runs anything here, and nothing here imports the product package.

The arithmetic lives in ``oracle.c`` (plain single-threaded C, built with
``-ffp-contract=off`` and no fast-math); this module builds it with gcc, wraps
it with ctypes and adds the payoff table, written out in numpy fp64 from its
definition: the evaluator's table holds, for each policy combination, the
mean evaluation result of the simulations run under it (MALib Sec. 3.2,
Actor-Evaluator-Learner; Appendix C.2 ``run_simulation_and_update_payoff``).
Here the result is the undiscounted return of the row-side seat and, for team
games, every (row-side seat, column-side seat) pair of an env is one entry.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_CFLAGS = ["-O2", "-march=x86-64-v3", "-ffp-contract=off", "-fno-fast-math",
           "-fPIC", "-shared", "-std=c11", "-Wall"]
# A prebuilt oracle library to load instead (the sanitizer test's instrumented
# build, see build_sanitized); never rebuilt here.
_LIB_OVERRIDE = os.environ.get("MALIB_ORACLE_LIB")

TOL_BF16 = 1e-2
TOL_F32 = 1e-5


def build(force: bool = True) -> str:
    """Compile oracle.c into liboracle.so (always, when ``force``)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", *_CFLAGS, _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def build_sanitized(path: str) -> str:
    """Compile oracle.c with AddressSanitizer and UndefinedBehaviorSanitizer
    (gcc; any UB report aborts) into ``path``, same floating-point flags.  Load
    it by starting a process with MALIB_ORACLE_LIB=path and gcc's libasan.so
    in LD_PRELOAD."""
    flags = [f for f in _CFLAGS if f != "-O2"] + [
        "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
        "-fno-sanitize-recover=undefined"]
    subprocess.check_call(["gcc", *flags, _SRC, "-o", path, "-lm"])
    return path


class Config(C.Structure):
    _fields_ = [
        ("env_kind", C.c_int32), ("n_agents", C.c_int32), ("n_actions", C.c_int32),
        ("grid", C.c_int32), ("team", C.c_void_p), ("A", C.c_void_p),
        ("d", C.c_int32), ("init_mode", C.c_int32),
        ("W", C.c_void_p), ("emb", C.c_void_p), ("u", C.c_void_p),
        ("pol_kind", C.c_int32), ("P", C.c_int32), ("n_layers", C.c_int32),
        ("horizon", C.c_int32), ("dims", C.c_void_p),
        ("Wl", C.POINTER(C.c_void_p)), ("bl", C.POINTER(C.c_void_p)),
        ("tab", C.c_void_p), ("seed", C.c_uint64), ("env_offset", C.c_int64),
    ]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if _LIB_OVERRIDE:
            L = C.CDLL(_LIB_OVERRIDE)
        else:
            if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
                build()
            L = C.CDLL(_LIB)
        L.ora_philox4x64_10.argtypes = [C.c_void_p, C.c_void_p, C.c_void_p]
        L.ora_lane.restype = C.c_uint32
        L.ora_lane.argtypes = [C.c_uint64, C.c_int64, C.c_int64, C.c_int32, C.c_int32,
                               C.c_int64, C.c_int32]
        L.ora_uniform.restype = C.c_float
        L.ora_uniform.argtypes = [C.c_uint32]
        L.ora_gumbel.restype = C.c_double
        L.ora_gumbel.argtypes = [C.c_float]
        L.ora_bf16_bits.restype = C.c_uint16
        L.ora_bf16_bits.argtypes = [C.c_float]
        L.ora_bf16_round.restype = C.c_float
        L.ora_bf16_round.argtypes = [C.c_float]
        L.ora_bf16_relu.restype = C.c_float
        L.ora_bf16_relu.argtypes = [C.c_float]
        L.ora_exp_ref.restype = C.c_float
        L.ora_exp_ref.argtypes = [C.c_float]
        L.ora_tanh_ref.restype = C.c_float
        L.ora_tanh_ref.argtypes = [C.c_float]
        L.ora_tanh_range.argtypes = [C.c_uint32, C.c_int64, C.c_void_p]
        L.ora_tanh_max_ulp.restype = C.c_double
        L.ora_tanh_max_ulp.argtypes = [C.c_uint32, C.c_int64, C.c_void_p]
        L.ora_meta_sample.restype = C.c_int
        L.ora_meta_sample.argtypes = [C.c_void_p, C.c_int32, C.c_int32, C.c_int64,
                                      C.c_int32, C.c_uint64, C.c_int64, C.c_void_p]
        L.ora_solve_fp.restype = C.c_int
        L.ora_solve_fp.argtypes = [C.c_void_p, C.c_int32, C.c_int32, C.c_void_p, C.c_void_p,
                                   C.c_void_p]
        L.ora_rollout.restype = C.c_int
        L.ora_rollout.argtypes = [C.POINTER(Config), C.c_int64, C.c_void_p, C.c_void_p,
                                  C.c_void_p, C.c_double, C.c_void_p, C.c_void_p,
                                  C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p]
        L.ora_state_elems.restype = C.c_int64
        L.ora_state_elems.argtypes = [C.c_int32, C.c_int32]
        L.ora_obs_iter.argtypes = [C.c_void_p, C.c_int32, C.c_void_p]
        L.ora_obs_pursuit.argtypes = [C.c_int32, C.c_int32, C.c_int32, C.c_int32, C.c_void_p]
        L.ora_pursuit_step.restype = C.c_int
        L.ora_pursuit_step.argtypes = [C.c_void_p, C.c_void_p, C.c_int32, C.c_int32, C.c_int32]
        L.ora_pursuit_reset.argtypes = [C.c_uint64, C.c_int64, C.c_int32, C.c_void_p, C.c_void_p]
        L.ora_feature_reset.argtypes = [C.c_uint64, C.c_int64, C.c_int32, C.c_void_p]
        L.ora_feature_step.restype = C.c_float
        L.ora_feature_step.argtypes = [C.POINTER(Config), C.c_void_p, C.c_void_p, C.c_void_p]
        L.ora_policy_logits.restype = C.c_int
        L.ora_policy_logits.argtypes = [C.POINTER(Config), C.c_int32, C.c_void_p, C.c_void_p]
        L.ora_bf16_range.argtypes = [C.c_uint32, C.c_int64, C.c_void_p]
        L.ora_uniform_range.argtypes = [C.c_uint32, C.c_int64, C.c_void_p]
        L.ora_exp_many.argtypes = [C.c_void_p, C.c_int64, C.c_void_p]
        L.ora_tanh_many.argtypes = [C.c_void_p, C.c_int64, C.c_void_p]
        _lib = L
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data


# ----------------------------------------------------------------- primitives

def philox(ctr, key):
    c = np.ascontiguousarray(ctr, dtype=np.uint64)
    k = np.ascontiguousarray(key, dtype=np.uint64)
    out = np.zeros(4, np.uint64)
    lib().ora_philox4x64_10(_ptr(c), _ptr(k), _ptr(out))
    return out


def lane(seed, g, t, purpose, slot, block, ln):
    return lib().ora_lane(seed, g, t, purpose, slot, block, ln)


def uniform(x):
    return lib().ora_uniform(int(x))


def gumbel(u):
    return lib().ora_gumbel(float(u))


def bf16_bits(x):
    return lib().ora_bf16_bits(float(x))


def bf16_round(x):
    return lib().ora_bf16_round(float(x))


def bf16_relu(x):
    """Hidden-unit ReLU of the bf16 policies (on the rounded value)."""
    return lib().ora_bf16_relu(float(x))


def exp_ref(x):
    return lib().ora_exp_ref(float(x))


def tanh_ref(x):
    return lib().ora_tanh_ref(float(x))


def tanh_range(first_bits: int, n: int) -> np.ndarray:
    out = np.empty(n, np.float32)
    lib().ora_tanh_range(first_bits, n, _ptr(out))
    return out


def bf16_range(first_bits: int, n: int) -> np.ndarray:
    out = np.empty(n, np.uint16)
    lib().ora_bf16_range(first_bits, n, _ptr(out))
    return out


def uniform_range(first: int, n: int) -> np.ndarray:
    out = np.empty(n, np.float32)
    lib().ora_uniform_range(first, n, _ptr(out))
    return out


def exp_many(x) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty_like(x)
    lib().ora_exp_many(_ptr(x), x.size, _ptr(out))
    return out


def tanh_many(x) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty_like(x)
    lib().ora_tanh_many(_ptr(x), x.size, _ptr(out))
    return out


def tanh_max_ulp(first_bits: int, n: int):
    w = np.zeros(1, np.uint32)
    e = lib().ora_tanh_max_ulp(first_bits, n, _ptr(w))
    return e, int(w[0])


def meta_sample(sigma, P, n_envs, n_agents, seed, env_offset=0):
    s = np.ascontiguousarray(sigma, dtype=np.float32).reshape(-1, P)
    out = np.zeros((n_envs, n_agents), np.int32)
    rc = lib().ora_meta_sample(_ptr(s), s.shape[0], P, n_envs, n_agents, seed,
                               env_offset, _ptr(out))
    if rc != 0:
        raise ValueError(f"ora_meta_sample rejected its input ({rc})")
    return out


def solve_fp(M, T):
    """Simultaneous fictitious play on the zero-sum game with row payoff M
    (P x P, fp64; the column side receives -M) for T iterations (oracle.c,
    ora_solve_fp).  Returns (cx, cy, gap): the play counts of the row and
    column side (int32) and the exploitability of the average strategies."""
    m = np.ascontiguousarray(M, dtype=np.float64)
    P = m.shape[0]
    assert m.shape == (P, P)
    cx = np.zeros(P, np.int32)
    cy = np.zeros(P, np.int32)
    gap = np.zeros(1, np.float64)
    rc = lib().ora_solve_fp(_ptr(m), P, int(T), _ptr(cx), _ptr(cy), _ptr(gap))
    if rc != 0:
        raise ValueError(f"ora_solve_fp rejected its input ({rc})")
    return cx, cy, float(gap[0])


def expansion_pairs(P, first_new, per_pair, team):
    """The combinations to simulate after a population grew from first_new to P
    policies: every cell (r, c) of the P x P grid with r >= first_new or
    c >= first_new, in row-major order, each played by per_pair consecutive
    envs; in each env the row-side seats (team +1) take r, the others c."""
    team = np.asarray(team)
    cells = [(r, c) for r in range(P) for c in range(P) if r >= first_new or c >= first_new]
    out = np.empty((len(cells) * per_pair, len(team)), np.int32)
    for q, (r, c) in enumerate(cells):
        for k in range(len(team)):
            out[q * per_pair:(q + 1) * per_pair, k] = r if team[k] > 0 else c
    return out


def aggregate(M, sigma, br_row, br_col):
    """Aggregate payoffs of a meta-strategy pair on the game M (the PSRO
    convergence judgement of the example API's main loop, Appendix C.2):
    x, y = the two weight rows of sigma (fp32) normalized in fp64; u = M y and
    v = x^T M, each entry a sequential fp64 sum (products rounded, then
    added); nash = x^T u (sequential).  Returns (nash payoff of the row side,
    of the column side (= -nash, zero-sum), the row side's payoff of policy
    br_row against y (u[br_row]), the column side's of br_col against x
    (-v[br_col]), improvement = the larger gain of a best response over the
    equilibrium payoff); a side with br = -1 is left out (NaN)."""
    M = np.asarray(M, np.float64)
    P = M.shape[0]
    s = np.asarray(sigma, np.float32).reshape(2, P)
    w0 = [float(a) for a in s[0]]
    w1 = [float(a) for a in s[1]]
    S0 = 0.0
    S1 = 0.0
    for a in w0:
        S0 += a
    for a in w1:
        S1 += a
    x = [a / S0 for a in w0]
    y = [a / S1 for a in w1]
    u = []
    for i in range(P):
        acc = 0.0
        for j in range(P):
            acc += float(M[i, j]) * y[j]
        u.append(acc)
    v = []
    for j in range(P):
        acc = 0.0
        for i in range(P):
            acc += x[i] * float(M[i, j])
        v.append(acc)
    nash = 0.0
    for i in range(P):
        nash += x[i] * u[i]
    nan = float("nan")
    w_row = u[br_row] if br_row >= 0 else nan
    w_col = -v[br_col] if br_col >= 0 else nan
    gains = []
    if br_row >= 0:
        gains.append(w_row - nash)
    if br_col >= 0:
        gains.append(w_col - (-nash))
    improvement = max(gains) if gains else nan
    return nash, -nash, w_row, w_col, improvement


def payoff_matrix(mean):
    """The solver's game from a payoff table: the means, 0 where a cell has no
    simulations."""
    return np.where(np.isnan(mean), 0.0, mean)


# ---------------------------------------------------------------- alpha-rank
#
# The alpha-rank meta-solver that the paper names beside fictitious play and
# the LP solver for PSRO (Sec. 4.2, Table 3), as defined by its authors
# (Omidshafiei et al., 2019, "alpha-Rank: Multi-Agent Evaluation by
# Evolution"), single-population form: the P policies form one population
# (every seat draws from the same pool, Sec. 3.1), and the table's game is
# made symmetric by letting two policies meet once on each side.

def alpharank_fixation(u, m):
    """Fixation probability of a mutant whose fitness exceeds the resident's
    by u / alpha (u = alpha * difference) in a population of m (Fermi/Moran
    selection): (1 - e^-u) / (1 - e^-(m u)); 1/m when u = 0.  fp64."""
    u = float(u)
    if u == 0.0:
        return 1.0 / m
    if u > 0.0:
        return float(np.expm1(-u) / np.expm1(-m * u))
    # u < 0: the same ratio with e^((m-1) u) taken out, so that it underflows
    # gracefully instead of dividing two overflowing terms
    v = -u
    return float(np.exp(-(m - 1) * v) * (np.expm1(-v) / np.expm1(-m * v)))


def alpharank_chain(M, alpha, m):
    """Transition matrix C [P][P] (fp64) of the alpha-rank Markov chain on the
    monomorphic states of the game with row payoff M (the column side gets
    -M): resident r, mutant s != r meet once on each side, so the mutant's
    payoff is (M[s][r] - M[r][s]) / 2 and the resident's its negative; the
    fitness difference is u = alpha (M[s][r] - M[r][s]).  C[r][s] =
    rho(u) / (P - 1) for s != r (a mutation picks one of the other policies
    uniformly), C[r][r] = 1 - (sum of the row's other entries)."""
    M = np.asarray(M, np.float64)
    P = M.shape[0]
    C = np.zeros((P, P), np.float64)
    if P == 1:
        C[0, 0] = 1.0
        return C
    for r in range(P):
        for s in range(P):
            if s != r:
                u = alpha * (float(M[s, r]) - float(M[r, s]))
                C[r, s] = alpharank_fixation(u, m) / (P - 1)
        C[r, r] = 1.0 - (C[r].sum() - C[r, r])
    return C


def alpharank(M, alpha, m):
    """alpha-rank distribution pi [P] (fp64): the stationary distribution of
    alpharank_chain, pi^T C = pi^T with sum(pi) = 1, solved as the linear
    system (C^T - I) pi = 0 with the last equation replaced by sum(pi) = 1
    (unique: for finite alpha every rho is positive, so the chain is
    irreducible)."""
    C = alpharank_chain(M, alpha, m)
    P = C.shape[0]
    A = C.T - np.eye(P)
    A[P - 1, :] = 1.0
    b = np.zeros(P, np.float64)
    b[P - 1] = 1.0
    return np.linalg.solve(A, b)


# ---------------------------------------------------------------- LP solver
#
# The LP meta-solver the paper lists beside fictitious play and alpha-rank for
# PSRO (Sec. 4.2): the exact equilibrium of the two-player zero-sum meta-game
# (the row side receives M[i][j], the column side -M[i][j]).  By the minimax
# theorem its value v = max over x of min over j of (x^T M)_j = min over y of
# max over i of (M y)_i; the row side's optimal x solves
#   maximize v  subject to  sum_i x_i M[i][j] >= v for every j,
#                           sum_i x_i = 1,  x >= 0,
# and the column side's y the mirror problem.  Each is handed to scipy's
# linprog (HiGHS) as written.

def solve_lp(M):
    """Value and optimal strategies of the zero-sum game M (P x P, fp64):
    returns (v, x, y), x and y fp64 [P].  The strategies need not be unique;
    the value is."""
    from scipy.optimize import linprog
    M = np.asarray(M, np.float64)
    P, Q = M.shape
    # row side: variables (x_0 .. x_{P-1}, v); minimize -v
    c = np.zeros(P + 1)
    c[-1] = -1.0
    A_ub = np.hstack([-M.T, np.ones((Q, 1))])          # v - (x^T M)_j <= 0
    b_ub = np.zeros(Q)
    A_eq = np.zeros((1, P + 1))
    A_eq[0, :P] = 1.0
    bounds = [(0, None)] * P + [(None, None)]
    rx = linprog(c, A_ub=A_ub, b_ub=b_ub, A_eq=A_eq, b_eq=[1.0], bounds=bounds,
                 method="highs")
    # column side: variables (y, w); minimize w subject to (M y)_i <= w
    c2 = np.zeros(Q + 1)
    c2[-1] = 1.0
    A2 = np.hstack([M, -np.ones((P, 1))])
    A2eq = np.zeros((1, Q + 1))
    A2eq[0, :Q] = 1.0
    ry = linprog(c2, A_ub=A2, b_ub=np.zeros(P), A_eq=A2eq, b_eq=[1.0],
                 bounds=[(0, None)] * Q + [(None, None)], method="highs")
    if rx.status != 0 or ry.status != 0:
        raise RuntimeError(f"linprog failed: {rx.message} / {ry.message}")
    return float(-rx.fun), rx.x[:P].copy(), ry.x[:Q].copy()


# ---------------------------------------------------------------- configuration

class _Cfg:
    """Keeps the numpy buffers a ctypes Config points at alive."""

    def __init__(self, wl, horizon=None, env_offset=0, init_mode=None):
        keep = []

        def arr(a, dt):
            if a is None:
                return None
            a = np.ascontiguousarray(a, dtype=dt)
            keep.append(a)
            return a

        cfg = Config()
        cfg.env_kind = wl.env_kind
        cfg.n_agents = wl.n_agents
        cfg.n_actions = wl.n_actions
        cfg.grid = wl.grid
        cfg.team = _ptr(arr(wl.team, np.int8))
        cfg.A = _ptr(arr(wl.A, np.float32))
        cfg.d = wl.d
        cfg.init_mode = wl.init_mode if init_mode is None else init_mode
        cfg.W = _ptr(arr(wl.W, np.float32))
        cfg.emb = _ptr(arr(wl.emb, np.float32))
        cfg.u = _ptr(arr(wl.u, np.float32))
        cfg.pol_kind = wl.pol_kind
        cfg.P = wl.P
        L = len(wl.dims) - 1 if wl.dims else 0
        cfg.n_layers = L
        cfg.horizon = wl.horizon if horizon is None else horizon
        cfg.dims = _ptr(arr(np.array(wl.dims or [0], np.int32), np.int32))
        wl_ptrs = (C.c_void_p * max(L, 1))()
        bl_ptrs = (C.c_void_p * max(L, 1))()
        for l in range(L):
            wl_ptrs[l] = _ptr(arr(wl.weights[l], np.float32))
            bl_ptrs[l] = _ptr(arr(wl.biases[l], np.float32)) if wl.biases else None
        keep += [wl_ptrs, bl_ptrs]
        cfg.Wl = C.cast(wl_ptrs, C.POINTER(C.c_void_p))
        cfg.bl = C.cast(bl_ptrs, C.POINTER(C.c_void_p))
        cfg.tab = _ptr(arr(wl.tab_logits, np.float32))
        cfg.seed = wl.seed
        cfg.env_offset = env_offset
        self.cfg = cfg
        self.keep = keep


def state_shape(wl, n):
    if wl.env_kind == 1:
        return (n,), np.uint16
    if wl.env_kind == 2:
        return (n, 3), np.uint8
    if wl.env_kind == 3:
        return (n, wl.d), np.float32
    return None, None


def rollout(wl, env_idx, pids, *, forced=None, tol=None, horizon=None, env_offset=0,
            want_actions=False, want_logits=False, want_states=False, want_rewards=False,
            init_mode=None):
    """Roll out the selected envs (local indices ``env_idx`` of a batch that
    starts at global env ``env_offset``) with per-env policy ids ``pids``
    [n_sel][n_agents].  ``forced`` is an action log [H][n_sel][n_agents] to
    follow in lockstep (see oracle.c).  Returns a dict."""
    H = wl.horizon if horizon is None else horizon
    if tol is None:
        tol = TOL_F32 if wl.pol_kind == 1 else TOL_BF16
    idx = np.ascontiguousarray(env_idx, dtype=np.int64)
    n = idx.shape[0]
    p = np.ascontiguousarray(pids, dtype=np.int32).reshape(n, wl.n_agents)
    f = None if forced is None else np.ascontiguousarray(forced, dtype=np.uint8).reshape(
        H, n, wl.n_agents)
    cfg = _Cfg(wl, horizon=H, env_offset=env_offset, init_mode=init_mode)
    ret = np.zeros((n, wl.n_agents), np.float32)
    acts = np.zeros((H, n, wl.n_agents), np.uint8) if want_actions else None
    logits = np.zeros((H, n, wl.n_agents, wl.n_actions), np.float32) if want_logits else None
    states = None
    if want_states:
        shp, dt = state_shape(wl, n)
        if shp is not None:
            states = np.zeros((H,) + shp, dt)
    stats = np.zeros(7, np.int64)
    rews = np.zeros((H, n, wl.n_agents), np.float32) if want_rewards else None
    rc = lib().ora_rollout(C.byref(cfg.cfg), n, _ptr(idx), _ptr(p), _ptr(f), float(tol),
                           _ptr(ret), _ptr(acts), _ptr(logits), _ptr(states), _ptr(stats),
                           _ptr(rews))
    if rc != 0:
        raise RuntimeError(f"ora_rollout failed ({rc})")
    return {
        "returns": ret, "actions": acts, "logits": logits, "states": states,
        "rewards": rews,
        "near_ties": int(stats[0]), "flips": int(stats[1]), "fails": int(stats[2]),
        "live_frames": int(stats[3]),
        "first_fail": tuple(int(x) for x in stats[4:7]),
    }


def rollout_threads(wl, env_idx, pids, *, threads=None, forced=None, **kw):
    """``rollout`` over shards of the selected envs in parallel threads (the C
    oracle holds no shared state and ctypes releases the GIL during the call);
    every env is still simulated by the same single-threaded code, so the
    merged result equals one ``rollout`` over all of them."""
    import concurrent.futures as cf
    idx = np.ascontiguousarray(env_idx, dtype=np.int64)
    n = idx.shape[0]
    if threads is None:
        threads = min(16, len(os.sched_getaffinity(0)))
    k = max(1, min(threads, n))
    bounds = np.linspace(0, n, k + 1).astype(int)
    p = np.asarray(pids).reshape(n, wl.n_agents)

    def one(i):
        lo, hi = bounds[i], bounds[i + 1]
        f = None if forced is None else np.asarray(forced)[:, lo:hi]
        return rollout(wl, idx[lo:hi], p[lo:hi], forced=f, **kw)

    with cf.ThreadPoolExecutor(max_workers=k) as ex:
        parts = list(ex.map(one, range(k)))
    out = {"returns": np.concatenate([q["returns"] for q in parts])}
    for key in ("actions", "logits", "states", "rewards"):
        out[key] = (None if parts[0][key] is None
                    else np.concatenate([q[key] for q in parts], axis=1))
    for key in ("near_ties", "flips", "fails", "live_frames"):
        out[key] = sum(q[key] for q in parts)
    out["first_fail"] = next(((q["first_fail"][0], q["first_fail"][1] + int(lo),
                               q["first_fail"][2]) for q, lo in zip(parts, bounds)
                              if q["fails"]), parts[0]["first_fail"])
    return out


def policy_logits(wl, p, obs):
    cfg = _Cfg(wl)
    o = np.ascontiguousarray(obs, dtype=np.float64)
    out = np.zeros(wl.n_actions, np.float32)
    if lib().ora_policy_logits(C.byref(cfg.cfg), p, _ptr(o), _ptr(out)) != 0:
        raise ValueError("bad policy id")
    return out


def feature_step(wl, s, acts):
    cfg = _Cfg(wl)
    s = np.ascontiguousarray(s, dtype=np.float32)
    a = np.ascontiguousarray(acts, dtype=np.int32)
    out = np.zeros_like(s)
    r = lib().ora_feature_step(C.byref(cfg.cfg), _ptr(s), _ptr(a), _ptr(out))
    return out, r


def feature_reset(seed, g, d):
    s = np.zeros(d, np.float32)
    lib().ora_feature_reset(seed, g, d, _ptr(s))
    return s


def pursuit_reset(seed, g, grid=8):
    pc = np.zeros(1, np.int32)
    ec = np.zeros(1, np.int32)
    lib().ora_pursuit_reset(seed, g, grid, _ptr(pc), _ptr(ec))
    return int(pc[0]), int(ec[0])


def pursuit_step(pc, ec, a0, a1, grid=8):
    p = np.array([pc], np.int32)
    e = np.array([ec], np.int32)
    cap = lib().ora_pursuit_step(_ptr(p), _ptr(e), a0, a1, grid)
    return int(p[0]), int(e[0]), bool(cap)


def obs_pursuit(pc, ec, seat, grid=8):
    out = np.zeros(75, np.float64)
    lib().ora_obs_pursuit(pc, ec, seat, grid, _ptr(out))
    return out


def obs_iter(hist, seat):
    h = np.ascontiguousarray(hist, dtype=np.int32)
    out = np.zeros(24, np.float64)
    lib().ora_obs_iter(_ptr(h), seat, _ptr(out))
    return out


# ----------------------------------------------------------------- payoff table

def payoff(returns, pids, team, P):
    """Payoff table from per-env returns [n_envs][n_agents] and policy ids
    [n_envs][n_agents]: every (row-side seat a, column-side seat b) of an env adds
    the return of seat a to cell (pid[a], pid[b]).  Returns (mean, counts, sum,
    sumsq) in fp64; mean is NaN where the count is zero."""
    returns = np.asarray(returns, dtype=np.float64)
    pids = np.asarray(pids, dtype=np.int64)
    team = np.asarray(team)
    rows = np.nonzero(team > 0)[0]
    cols = np.nonzero(team < 0)[0]
    s = np.zeros((P, P), np.float64)
    s2 = np.zeros((P, P), np.float64)
    n = np.zeros((P, P), np.int64)
    for a in rows:
        for b in cols:
            cell = pids[:, a] * P + pids[:, b]
            g = returns[:, a]
            s += np.bincount(cell, weights=g, minlength=P * P).reshape(P, P)
            s2 += np.bincount(cell, weights=g * g, minlength=P * P).reshape(P, P)
            n += np.bincount(cell, minlength=P * P).reshape(P, P)
    with np.errstate(invalid="ignore", divide="ignore"):
        mean = np.where(n > 0, s / np.maximum(n, 1), np.nan)
    return mean, n, s, s2
