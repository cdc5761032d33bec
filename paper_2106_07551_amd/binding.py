"""ctypes binding of libmalib.so (argument marshalling only).

Device buffers are torch CUDA (HIP) tensors; streams are torch streams.  Every
call goes straight to the C ABI of ``include/malib.h``; names follow it.
"""
from __future__ import annotations

import ctypes as C
import sys
import os
from typing import Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmalib.so")

MALIB_OK, E_INVAL, E_NOMEM, E_HIP, E_UNSUPPORTED, E_DEVICE = 0, -1, -2, -3, -4, -5
POLICY_TABULAR, POLICY_MLP_F32, POLICY_MLP_BF16 = 0, 1, 2
ENV_MATRIX, ENV_ITER_MATRIX, ENV_PURSUIT, ENV_FEATURE = 0, 1, 2, 3
INIT_PER_ENV, INIT_SHARED = 0, 1
K_POLICY, K_SAMPLE, K_ENV, K_SETUP, K_PAYOFF = 0, 1, 2, 3, 4

# every function declared in include/malib.h
EXPORTS = [
    "malib_pop_create", "malib_pop_destroy", "malib_rollout_batch", "malib_payoff_eval",
    "malib_meta_sample", "malib_last_error", "malib_profile_enable", "malib_profile_read",
    "malib_debug_tanh_ref", "malib_debug_bf16", "malib_debug_philox",
    "malib_payoff_matrix", "malib_solve_fp", "malib_meta_sample_device",
    "malib_pop_extend", "malib_expansion_pairs", "malib_aggregate", "malib_rollout_batch_traj",
    "malib_pop_policy_ids", "malib_rollout_batch_noalloc", "malib_pop_set_graph",
    "malib_solve_alpharank", "malib_solve_lp",
]


class MalibError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"malib status {status}: {msg}")
        self.status = status


class ArgumentError(MalibError, ValueError):
    """An argument the binding rejects before calling the library (wrong
    dtype, size, layout or device of a buffer): status MALIB_E_INVAL, as the
    library itself reports invalid arguments."""

    def __init__(self, msg: str):
        super().__init__(E_INVAL, msg)


class PopDesc(C.Structure):
    _fields_ = [("kind", C.c_int32), ("n_policies", C.c_int32), ("n_actions", C.c_int32),
                ("n_layers", C.c_int32), ("dims", C.POINTER(C.c_int32)),
                ("weights", C.POINTER(C.c_void_p)), ("biases", C.POINTER(C.c_void_p)),
                ("tab_logits", C.c_void_p), ("policy_ids", C.POINTER(C.c_int64))]


class EnvDesc(C.Structure):
    _fields_ = [("kind", C.c_int32), ("n_agents", C.c_int32), ("n_actions", C.c_int32),
                ("grid", C.c_int32), ("team", C.POINTER(C.c_int8)), ("A", C.c_void_p),
                ("d", C.c_int32), ("init_mode", C.c_int32), ("W", C.c_void_p),
                ("emb", C.c_void_p), ("u", C.c_void_p)]


class TraceDesc(C.Structure):
    _fields_ = [("actions", C.c_void_p), ("n_snap", C.c_int32),
                ("snap_steps", C.POINTER(C.c_int32)), ("logits", C.c_void_p),
                ("states", C.c_void_p), ("perm", C.c_void_p), ("offsets", C.c_void_p)]


class TrajDesc(C.Structure):
    _fields_ = [("actions", C.c_void_p), ("rewards", C.c_void_p), ("flags", C.c_void_p),
                ("obs", C.c_void_p), ("capacity", C.c_int64), ("cursor", C.c_int64)]


class EvalStats(C.Structure):
    _fields_ = [("live_frames", C.c_int64), ("envs", C.c_int64), ("device_flags", C.c_int32)]


_lib = None


def lib():
    """Load libmalib.so; raises if it has not been built (no fallback)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                              "(hipcc, gfx950); there is no CPU fallback")
        L = C.CDLL(LIB_PATH)
        vp, i32, i64, u64 = C.c_void_p, C.c_int32, C.c_int64, C.c_uint64
        L.malib_pop_create.argtypes = [C.POINTER(PopDesc), vp, C.POINTER(vp)]
        L.malib_pop_create.restype = i32
        L.malib_pop_destroy.argtypes = [vp]
        L.malib_pop_destroy.restype = None
        L.malib_rollout_batch.argtypes = [vp, C.POINTER(EnvDesc), i64, vp, u64, i64, i32, vp,
                                          C.POINTER(TraceDesc), vp]
        L.malib_rollout_batch.restype = i32
        L.malib_payoff_eval.argtypes = [vp, vp, i32, vp, vp, vp, C.POINTER(EvalStats)]
        L.malib_payoff_eval.restype = i32
        L.malib_meta_sample.argtypes = [vp, i32, i32, i64, i32, u64, i64, vp, vp]
        L.malib_meta_sample.restype = i32
        L.malib_last_error.argtypes = []
        L.malib_last_error.restype = C.c_char_p
        L.malib_profile_enable.argtypes = [vp, i32, i32]
        L.malib_profile_enable.restype = i32
        L.malib_profile_read.argtypes = [vp, i32, C.POINTER(C.c_double), C.POINTER(i64)]
        L.malib_profile_read.restype = i32
        L.malib_debug_tanh_ref.argtypes = [vp, vp, i64, vp]
        L.malib_debug_tanh_ref.restype = i32
        L.malib_debug_bf16.argtypes = [vp, vp, i64, vp]
        L.malib_debug_bf16.restype = i32
        L.malib_debug_philox.argtypes = [vp, u64, u64, vp, i64, vp]
        L.malib_debug_philox.restype = i32
        L.malib_payoff_matrix.argtypes = [vp, vp, vp]
        L.malib_payoff_matrix.restype = i32
        L.malib_solve_fp.argtypes = [vp, i32, i32, vp, vp, vp]
        L.malib_solve_fp.restype = i32
        L.malib_solve_alpharank.argtypes = [vp, i32, C.c_double, i32, vp, vp, vp, vp]
        L.malib_solve_alpharank.restype = i32
        L.malib_solve_lp.argtypes = [vp, i32, vp, vp, vp, vp, vp, vp, vp]
        L.malib_solve_lp.restype = i32
        L.malib_meta_sample_device.argtypes = [vp, i32, i32, i64, i32, vp, u64, i64, vp, vp]
        L.malib_meta_sample_device.restype = i32
        L.malib_rollout_batch_traj.argtypes = [vp, C.POINTER(EnvDesc), i64, vp, u64, i64, i32,
                                               vp, C.POINTER(TrajDesc), vp]
        L.malib_rollout_batch_traj.restype = i32
        L.malib_aggregate.argtypes = [vp, i32, vp, i32, i32, vp, vp]
        L.malib_aggregate.restype = i32
        L.malib_pop_extend.argtypes = [vp, vp, vp]
        L.malib_pop_extend.restype = i32
        L.malib_expansion_pairs.argtypes = [i32, i32, i32, i32, vp, vp, vp]
        L.malib_expansion_pairs.restype = i32
        L.malib_rollout_batch_noalloc.argtypes = [vp, C.POINTER(EnvDesc), i64, vp, u64, i64,
                                                  i32, vp, vp]
        L.malib_rollout_batch_noalloc.restype = i32
        L.malib_pop_set_graph.argtypes = [vp, i32]
        L.malib_pop_set_graph.restype = i32
        L.malib_pop_policy_ids.argtypes = [vp, vp, i32, C.POINTER(i32)]
        L.malib_pop_policy_ids.restype = i32
        _lib = L
    return _lib


def _check(st: int):
    if st != MALIB_OK:
        raise MalibError(st, lib().malib_last_error().decode())


def _stream(stream):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return C.c_void_p(s.cuda_stream)


def _dptr(t, dtype=None, numel: Optional[int] = None, *, at_least: bool = False,
          what: str = "tensor") -> Optional[int]:
    """Device address of a contiguous device tensor (None passes through).

    The library's kernels read and write the buffers it is given with the
    sizes and element types the header states, so a tensor of another dtype
    or with fewer elements would be accessed out of bounds on the device:
    both are errors here (ArgumentError, raised, not asserted), as are host
    tensors and non-contiguous views.  `numel` is the exact count, or the minimum with
    `at_least`."""
    if t is None:
        return None
    _check_buf(t, dtype, numel, at_least, what)
    if not t.is_cuda:
        raise ArgumentError(f"{what}: expected a device tensor, got one on {t.device}")
    return t.data_ptr()


def _check_buf(t, dtype, numel, at_least, what):
    """dtype, element count and layout of a buffer (not its device)."""
    if t is None:
        return
    if dtype is not None and t.dtype != dtype:
        raise ArgumentError(f"{what}: expected dtype {dtype}, got {t.dtype}")
    if numel is not None:
        n = t.numel()
        if (n < numel) if at_least else (n != numel):
            raise ArgumentError(f"{what}: expected {'at least ' if at_least else ''}{numel} "
                                f"elements, got {n}")
    if not t.is_contiguous():
        raise ArgumentError(f"{what}: expected a contiguous tensor")


def _dptrs(*specs):
    """_dptr over several buffers (t, dtype, numel, at_least, what): every
    dtype, size and layout is checked before any device, so that the first
    error reported is the most specific one."""
    for sp in specs:
        _check_buf(*sp)
    return [_dptr(*sp[:3], at_least=sp[3], what=sp[4]) for sp in specs]


def _dbytes(t, nbytes: int, what: str) -> Optional[int]:
    """Like _dptr for buffers whose element type the caller chooses: at least
    `nbytes` bytes."""
    if t is None:
        return None
    if t.numel() * t.element_size() < nbytes:
        raise ArgumentError(f"{what}: expected at least {nbytes} bytes, got "
                         f"{t.numel() * t.element_size()}")
    return _dptr(t, what=what)


def _f32():
    import torch
    return torch.float32


def _pop_desc(kind, n_policies, n_actions, dims, weights, biases, tab_logits,
              policy_ids=None):
    """A malib_pop_desc over device tensors, with the ctypes arrays it points
    into (keep them alive until the call returns)."""
    d = PopDesc()
    d.kind, d.n_policies, d.n_actions = kind, n_policies, n_actions
    keep = []
    if policy_ids is not None:
        if len(policy_ids) != n_policies:
            raise ArgumentError(f"policy_ids: expected {n_policies} ids, got {len(policy_ids)}")
        ids = (C.c_int64 * n_policies)(*[int(x) for x in policy_ids])
        keep.append(ids)
        d.policy_ids = C.cast(ids, C.POINTER(C.c_int64))
    if kind == POLICY_TABULAR:
        d.n_layers = 0
        if tab_logits is None:
            raise ArgumentError("a tabular population needs tab_logits")
        d.tab_logits = _dptr(tab_logits, _f32(), n_policies * n_actions, what="tab_logits")
    else:
        if dims is None or len(dims) != 4 or len(weights) != 3:
            raise ArgumentError("an MLP population needs dims [in, h1, h2, A] and three weights")
        if biases is not None and len(biases) != 3:
            raise ArgumentError("biases: expected three entries (each a tensor or None)")
        d.n_layers = 3
        f32 = _f32()
        specs = [(w, f32, n_policies * dims[l + 1] * dims[l], False, f"weights[{l}]")
                 for l, w in enumerate(weights)]
        if biases is not None:
            specs += [(b, f32, n_policies * dims[l + 1], False, f"biases[{l}]")
                      for l, b in enumerate(biases)]
        ptrs = _dptrs(*specs)
        dd = (C.c_int32 * 4)(*dims)
        ww = (C.c_void_p * 3)(*ptrs[:3])
        keep += [dd, ww]
        d.dims = C.cast(dd, C.POINTER(C.c_int32))
        d.weights = C.cast(ww, C.POINTER(C.c_void_p))
        if biases is not None:
            bb = (C.c_void_p * 3)(*ptrs[3:])
            keep.append(bb)
            d.biases = C.cast(bb, C.POINTER(C.c_void_p))
    return d, keep


class Population:
    """A policy population handle (malib_pop_create / malib_pop_destroy) with its
    payoff table."""

    def __init__(self, kind: int, n_policies: int, n_actions: int, *, dims=None,
                 weights: Sequence = (), biases: Optional[Sequence] = None,
                 tab_logits=None, policy_ids: Optional[Sequence[int]] = None, stream=None):
        d, keep = _pop_desc(kind, n_policies, n_actions, dims, weights, biases, tab_logits,
                            policy_ids)
        h = C.c_void_p()
        self._destroy = lib().malib_pop_destroy
        self._finalizing = sys.is_finalizing
        _check(lib().malib_pop_create(C.byref(d), _stream(stream), C.byref(h)))
        del keep
        self.handle = h
        self.kind = kind
        self.dims = list(dims) if dims is not None else None
        self.P = n_policies
        self.A = n_actions

    def extend(self, n_new: int, *, weights: Sequence = (), biases: Optional[Sequence] = None,
               tab_logits=None, policy_ids: Optional[Sequence[int]] = None, stream=None):
        """malib_pop_extend: append n_new policies (indices P .. P + n_new - 1,
        caller ids ``policy_ids``, default the indices); the table keeps its
        cells and gains empty rows and columns."""
        d, keep = _pop_desc(self.kind, n_new, self.A, self.dims, weights, biases, tab_logits,
                            policy_ids)
        _check(lib().malib_pop_extend(self.handle, C.byref(d), _stream(stream)))
        del keep
        self.P += n_new

    def set_graph(self, enable: bool = True):
        """malib_pop_set_graph: replay each batch's launch sequence as one HIP graph."""
        _check(lib().malib_pop_set_graph(self.handle, int(bool(enable))))

    def policy_ids(self) -> np.ndarray:
        """malib_pop_policy_ids: the caller id of each index 0 .. P-1."""
        n = C.c_int32()
        out = np.zeros(self.P, np.int64)
        _check(lib().malib_pop_policy_ids(self.handle, out.ctypes.data, self.P, C.byref(n)))
        if n.value != self.P:
            raise RuntimeError(f"malib_pop_policy_ids returned {n.value} ids for P = {self.P}")
        return out

    def close(self):
        """malib_pop_destroy (also on garbage collection).  At interpreter exit
        the call is skipped: module globals and the HIP runtime may already be
        torn down, and the process's device memory is released with it; the
        functions used here are the ones captured when the handle was made."""
        h = getattr(self, "handle", None)
        if not h:
            return
        self.handle = None
        if self._finalizing():
            return
        self._destroy(h)

    __del__ = close

    def _batch_ptrs(self, env: "Env", n_envs: int, pair_assign, returns):
        """pair_assign int32 [n_envs][n_agents] and returns fp32 [n_agents][n_envs]
        (at least that many elements; counts the library rejects pass through
        to it)."""
        import torch
        ns = max(int(n_envs), 0) * env.n_agents
        return (_dptr(pair_assign, torch.int32, ns, at_least=True, what="pair_assign"),
                _dptr(returns, torch.float32, ns, at_least=True, what="returns"))

    def rollout(self, env: "Env", n_envs: int, pair_assign, seed: int, horizon: int, *,
                env_offset: int = 0, returns=None, trace: "Trace" = None, stream=None):
        pa, rp = self._batch_ptrs(env, n_envs, pair_assign, returns)
        tr = trace.checked(env, n_envs, horizon, self.P, self.A) if trace is not None else None
        _check(lib().malib_rollout_batch(
            self.handle, C.byref(env.desc), n_envs, pa, seed, env_offset,
            horizon, rp, C.byref(tr) if tr is not None else None,
            _stream(stream)))

    def rollout_noalloc(self, env: "Env", n_envs: int, pair_assign, seed: int, horizon: int,
                        *, env_offset: int = 0, returns=None, stream=None):
        """malib_rollout_batch_noalloc: the same batch on the library's static
        scratch (no device allocation; calls on one GPU must not overlap)."""
        pa, rp = self._batch_ptrs(env, n_envs, pair_assign, returns)
        _check(lib().malib_rollout_batch_noalloc(
            self.handle, C.byref(env.desc), n_envs, pa, seed, env_offset,
            horizon, rp, _stream(stream)))

    def rollout_traj(self, env: "Env", n_envs: int, pair_assign, seed: int, horizon: int,
                     traj: Traj, *, env_offset: int = 0, returns=None, stream=None):
        """malib_rollout_batch_traj: a rollout that also writes its per-step
        records into `traj` (advancing its cursor)."""
        pa, rp = self._batch_ptrs(env, n_envs, pair_assign, returns)
        traj.check(env)
        _check(lib().malib_rollout_batch_traj(
            self.handle, C.byref(env.desc), n_envs, pa, seed, env_offset,
            horizon, rp, C.byref(traj.desc), _stream(stream)))

    def payoff_matrix(self, out=None, stream=None):
        """malib_payoff_matrix: the table's means as a device fp64 [P][P] game
        (0 for empty cells)."""
        import torch
        if out is None:
            out = torch.empty((self.P, self.P), dtype=torch.float64, device="cuda")
        _check(lib().malib_payoff_matrix(
            self.handle, _dptr(out, torch.float64, self.P * self.P, what="out"),
            _stream(stream)))
        return out

    def payoff(self, reset: bool = False, stream=None, check: bool = True):
        P = self.P
        mean = np.zeros((P, P), np.float64)
        counts = np.zeros((P, P), np.int64)
        se = np.zeros((P, P), np.float64)
        st = EvalStats()
        rc = lib().malib_payoff_eval(self.handle, _stream(stream), int(reset),
                                     mean.ctypes.data, counts.ctypes.data, se.ctypes.data,
                                     C.byref(st))
        if check:
            _check(rc)
        out = {"mean": mean, "counts": counts, "stderr": se, "live_frames": st.live_frames,
               "envs": st.envs, "device_flags": st.device_flags, "status": rc}
        return out

    def profile_enable(self, on: bool = True, *, kernels=None, every: int = 1):
        """Time launches of the kernel classes in ``kernels`` (default: all when
        ``on``), one in ``every``."""
        mask = 0
        if on:
            ks = range(5) if kernels is None else kernels
            for k in ks:
                mask |= 1 << k
        _check(lib().malib_profile_enable(self.handle, mask, every))

    def profile_read(self, kernel: int):
        ms = C.c_double()
        n = C.c_int64()
        _check(lib().malib_profile_read(self.handle, kernel, C.byref(ms), C.byref(n)))
        return ms.value, n.value


class Env:
    """An environment description (malib_env_desc); keeps its device tensors alive."""

    def __init__(self, kind: int, n_agents: int, n_actions: int, *, team=None, A=None,
                 grid: int = 0, d: int = 0, W=None, emb=None, u=None,
                 init_mode: int = INIT_PER_ENV):
        e = EnvDesc()
        e.kind, e.n_agents, e.n_actions, e.grid, e.d, e.init_mode = (
            kind, n_agents, n_actions, grid, d, init_mode)
        self._keep = [A, W, emb, u]
        if team is not None:
            if len(team) != n_agents:
                raise ArgumentError(f"team: expected {n_agents} entries, got {len(team)}")
            tt = (C.c_int8 * n_agents)(*[int(x) for x in team])
            self._keep.append(tt)
            e.team = C.cast(tt, C.POINTER(C.c_int8))
        f32 = _f32()
        e.A, e.W, e.emb, e.u = _dptrs((A, f32, n_actions * n_actions, False, "A"),
                                      (W, f32, d * d, False, "W"),
                                      (emb, f32, n_agents * n_actions * d, False, "emb"),
                                      (u, f32, d, False, "u"))
        self.desc = e
        self.kind = kind
        self.n_agents = n_agents
        self.n_actions = n_actions
        self.d = d


class Traj:
    """A device ring of per-step records (malib_traj): actions [cap][n_agents]
    uint8, rewards [cap] fp32, flags [cap] uint8 and, optionally, obs in the
    environment's compact form (see malib.h)."""

    def __init__(self, capacity: int, n_agents: int, *, obs_shape=None, obs_dtype=None,
                 device="cuda"):
        import torch
        self.capacity = capacity
        self.actions = torch.empty((capacity, n_agents), dtype=torch.uint8, device=device)
        self.rewards = torch.empty(capacity, dtype=torch.float32, device=device)
        self.flags = torch.empty(capacity, dtype=torch.uint8, device=device)
        self.obs = None
        if obs_shape is not None:
            self.obs = torch.empty((capacity,) + tuple(obs_shape), dtype=obs_dtype,
                                   device=device)
        # its own tensors: the device is checked before each rollout (check)
        self.desc = TrajDesc(self.actions.data_ptr(), self.rewards.data_ptr(),
                             self.flags.data_ptr(),
                             None if self.obs is None else self.obs.data_ptr(), capacity, 0)

    @property
    def cursor(self) -> int:
        return self.desc.cursor

    def check(self, env: "Env"):
        """The ring's buffers against the environment's record layout."""
        if not 0 <= self.desc.capacity <= self.capacity:
            raise ArgumentError(f"traj: capacity {self.desc.capacity} is outside the ring's "
                             f"{self.capacity} records")
        if self.actions.shape[1] != env.n_agents:
            raise ArgumentError(f"traj: actions hold {self.actions.shape[1]} seats, the "
                             f"environment has {env.n_agents}")
        per = {ENV_ITER_MATRIX: 2, ENV_PURSUIT: 2, ENV_FEATURE: 2 * env.d}.get(env.kind, 0)
        if self.obs is not None and per:
            _dbytes(self.obs, self.capacity * per, "traj.obs")
        if not self.actions.is_cuda:
            raise ArgumentError(f"traj: expected device tensors, got ones on "
                                f"{self.actions.device}")


class Trace:
    """Parity trace buffers (malib_trace); any of them may be omitted."""

    def __init__(self, *, actions=None, snap_steps=(), logits=None, states=None, perm=None,
                 offsets=None):
        t = TraceDesc()
        t.actions = _dptr(actions)
        steps = list(snap_steps)
        t.n_snap = len(steps)
        ss = (C.c_int32 * max(1, len(steps)))(*steps)
        t.snap_steps = C.cast(ss, C.POINTER(C.c_int32))
        t.logits, t.states = _dptr(logits), _dptr(states)
        t.perm, t.offsets = _dptr(perm), _dptr(offsets)
        self._keep = [ss, actions, logits, states, perm, offsets]
        self.desc = t
        self.n_snap = len(steps)
        self.actions, self.logits, self.states = actions, logits, states
        self.perm, self.offsets = perm, offsets

    def checked(self, env: "Env", n_envs: int, horizon: int, P: int, A: int):
        """The descriptor, after checking each buffer against the batch that
        will write it (sizes as in malib.h's malib_trace)."""
        import torch
        ns = max(int(n_envs), 0) * env.n_agents
        h = max(int(horizon), 0)
        per = {ENV_ITER_MATRIX: 2, ENV_PURSUIT: 3, ENV_FEATURE: 4 * env.d}.get(env.kind, 0)
        st = self.states
        if st is not None and st.numel() * st.element_size() < self.n_snap * per * max(n_envs, 0):
            raise ArgumentError(f"trace.states: expected at least "
                                f"{self.n_snap * per * max(n_envs, 0)} bytes, got "
                                f"{st.numel() * st.element_size()}")
        _dptrs((self.actions, torch.uint8, h * ns, True, "trace.actions"),
               (self.logits, torch.float32, self.n_snap * ns * A, True, "trace.logits"),
               (st, None, None, True, "trace.states"),
               (self.perm, torch.int32, ns, True, "trace.perm"),
               (self.offsets, torch.int32, P + 1, True, "trace.offsets"))
        return self.desc


def meta_sample(sigma, n_policies: int, n_envs: int, n_agents: int, seed: int, *,
                env_offset: int = 0, out=None, stream=None):
    """malib_meta_sample: policy id per (env, seat) drawn from sigma [n_sigma][P]."""
    import torch
    s = np.ascontiguousarray(sigma, dtype=np.float32).reshape(-1, n_policies)
    if out is None:
        out = torch.empty((n_envs, n_agents), dtype=torch.int32, device="cuda")
    op = _dptr(out, torch.int32, max(n_envs, 0) * max(n_agents, 0), at_least=True, what="out")
    _check(lib().malib_meta_sample(s.ctypes.data, s.shape[0], n_policies, n_envs, n_agents,
                                   seed, env_offset, op, _stream(stream)))
    return out


def expansion_pairs(n_policies: int, first_new: int, per_pair: int, n_agents: int = 2,
                    team=None, *, out=None, stream=None):
    """malib_expansion_pairs: policy ids [(P^2 - first_new^2) * per_pair][n_agents]
    of the batch that simulates the cells of the new rows and columns."""
    import torch
    n = (n_policies * n_policies - first_new * first_new) * per_pair
    if out is None:
        out = torch.empty((max(n, 0), n_agents), dtype=torch.int32, device="cuda")
    tm = None
    if team is not None:
        tm = np.ascontiguousarray(team, dtype=np.int8)
        if tm.shape != (n_agents,):
            raise ArgumentError(f"team: expected shape ({n_agents},), got {tm.shape}")
    op = _dptr(out, torch.int32, max(n, 0) * max(n_agents, 0), at_least=True, what="out")
    _check(lib().malib_expansion_pairs(n_policies, first_new, per_pair, n_agents,
                                       None if tm is None else tm.ctypes.data, op,
                                       _stream(stream)))
    return out


def _game(M) -> int:
    """P of a device fp64 [P][P] game, checked."""
    import torch
    if M.dim() != 2 or M.shape[0] != M.shape[1]:
        raise ArgumentError(f"M: expected a square [P][P] game, got shape {tuple(M.shape)}")
    _dptr(M, torch.float64, what="M")
    return int(M.shape[0])


def solve_fp(M, iterations: int, *, sigma=None, gap=None, stream=None):
    """malib_solve_fp on a device fp64 [P][P] game: returns (sigma [2][P] play
    counts as fp32, gap [1] fp64), both device tensors."""
    import torch
    P = _game(M)
    if sigma is None:
        sigma = torch.empty((2, P), dtype=torch.float32, device=M.device)
    if gap is None:
        gap = torch.empty(1, dtype=torch.float64, device=M.device)
    _check(lib().malib_solve_fp(_dptr(M), P, iterations,
                                _dptr(sigma, torch.float32, 2 * P, what="sigma"),
                                _dptr(gap, torch.float64, 1, what="gap"), _stream(stream)))
    return sigma, gap


def solve_lp(M, *, work=None, stream=None):
    """malib_solve_lp on a device fp64 [P][P] game: returns (value [1] fp64,
    x [P] fp64, y [P] fp64, sigma [2][P] fp32, pivots [1] int32), device
    tensors; a workspace is allocated here when P > 96 and none is given."""
    import torch
    P = _game(M)
    dev = M.device
    value = torch.empty(1, dtype=torch.float64, device=dev)
    x = torch.empty(P, dtype=torch.float64, device=dev)
    y = torch.empty(P, dtype=torch.float64, device=dev)
    sigma = torch.empty((2, P), dtype=torch.float32, device=dev)
    pivots = torch.empty(1, dtype=torch.int32, device=dev)
    if work is None and P > 96:
        work = torch.empty((P + 1) * (2 * P + 1), dtype=torch.float64, device=dev)
    wp = _dptr(work, torch.float64, (P + 1) * (2 * P + 1), at_least=True, what="work")
    _check(lib().malib_solve_lp(_dptr(M), P, wp, _dptr(value), _dptr(x), _dptr(y),
                                _dptr(sigma), _dptr(pivots), _stream(stream)))
    return value, x, y, sigma, pivots


def solve_alpharank(M, alpha: float, m: int, *, pi=None, sigma=None, work=None, stream=None):
    """malib_solve_alpharank on a device fp64 [P][P] game: returns (pi [P]
    fp64, sigma [2][P] fp32 weight rows), device tensors; a [P][P] fp64
    workspace is allocated here when P > 128 and none is given."""
    import torch
    P = _game(M)
    if pi is None:
        pi = torch.empty(P, dtype=torch.float64, device=M.device)
    if sigma is None:
        sigma = torch.empty((2, P), dtype=torch.float32, device=M.device)
    if work is None and P > 128:
        work = torch.empty((P, P), dtype=torch.float64, device=M.device)
    _check(lib().malib_solve_alpharank(
        _dptr(M), P, float(alpha), int(m),
        _dptr(work, torch.float64, P * P, at_least=True, what="work"),
        _dptr(pi, torch.float64, P, what="pi"), _dptr(sigma, torch.float32, 2 * P, what="sigma"),
        _stream(stream)))
    return pi, sigma


def aggregate(M, sigma, br_row: int = -1, br_col: int = -1, *, out=None, stream=None):
    """malib_aggregate: device fp64 [5] = (nash payoff of the row side, of
    the column side, best-response payoff of br_row, of br_col, improvement)."""
    import torch
    P = _game(M)
    if out is None:
        out = torch.empty(5, dtype=torch.float64, device=M.device)
    _check(lib().malib_aggregate(_dptr(M), P, _dptr(sigma, torch.float32, 2 * P, what="sigma"),
                                 br_row, br_col, _dptr(out, torch.float64, 5, what="out"),
                                 _stream(stream)))
    return out


def meta_sample_device(sigma, n_policies: int, n_envs: int, n_agents: int, seed: int, *,
                       env_offset: int = 0, seat_row=None, out=None, stream=None):
    """malib_meta_sample_device: policy ids drawn from device weight rows
    sigma [n_sigma][P] (fp32); seat k uses row seat_row[k] (default: row 0
    for all seats when there is one row, else row k)."""
    import torch
    if n_policies < 1 or sigma.numel() % n_policies or sigma.numel() == 0:
        raise ArgumentError(f"sigma: expected [n_sigma][{n_policies}] weights, got "
                         f"{sigma.numel()} elements")
    n_sigma = sigma.numel() // n_policies
    sr = None
    if seat_row is not None:
        sr = np.ascontiguousarray(seat_row, dtype=np.int32)
        if sr.shape != (n_agents,):
            raise ArgumentError(f"seat_row: expected shape ({n_agents},), got {sr.shape}")
    if out is None:
        out = torch.empty((n_envs, n_agents), dtype=torch.int32, device=sigma.device)
    sp, op = _dptrs((sigma, torch.float32, None, False, "sigma"),
                    (out, torch.int32, max(n_envs, 0) * max(n_agents, 0), True, "out"))
    _check(lib().malib_meta_sample_device(sp, n_sigma, n_policies, n_envs, n_agents,
                                          None if sr is None else sr.ctypes.data, seed,
                                          env_offset, op, _stream(stream)))
    return out


def debug_tanh_ref(x, y=None, stream=None):
    import torch
    if y is None:
        y = torch.empty_like(x)
    _check(lib().malib_debug_tanh_ref(_dptr(x, torch.float32, what="x"),
                                      _dptr(y, torch.float32, x.numel(), what="y"), x.numel(),
                                      _stream(stream)))
    return y


def debug_bf16(x, stream=None):
    """bf16 bit patterns (as int16) of an even-length fp32 device tensor."""
    import torch
    y = torch.empty(x.shape, dtype=torch.int16, device=x.device)
    _check(lib().malib_debug_bf16(_dptr(x, torch.float32, what="x"), _dptr(y), x.numel(),
                                  _stream(stream)))
    return y


def debug_philox(ctr, key0: int, key1: int, stream=None):
    import torch
    if ctr.dim() != 2 or ctr.shape[1] != 4:
        raise ArgumentError(f"ctr: expected [n][4] counters, got shape {tuple(ctr.shape)}")
    out = torch.empty_like(ctr)
    _check(lib().malib_debug_philox(_dptr(ctr, torch.int64, what="ctr"), key0, key1, _dptr(out),
                                    ctr.shape[0], _stream(stream)))
    return out
