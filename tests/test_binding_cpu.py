"""The Python binding's argument checks (host only, no GPU): every device
buffer handed to the library is checked for dtype, element count, layout and
device before the call, since a kernel given a smaller or differently typed
buffer than the header states would access it out of bounds.  The checks
raise ArgumentError (a MalibError with status MALIB_E_INVAL that is also a
ValueError); dtype and size are checked before the device, so host tensors
exercise them here."""
import numpy as np
import pytest
import torch

import paper_2106_07551_amd as M
from paper_2106_07551_amd import binding as B


def test_argument_error_is_an_inval_malib_error():
    e = M.ArgumentError("x")
    assert isinstance(e, M.MalibError) and isinstance(e, ValueError)
    assert e.status == B.E_INVAL


@pytest.mark.parametrize("t, dtype, n, at_least, msg", [
    (torch.zeros(4, dtype=torch.float64), torch.float32, 4, False, "dtype"),
    (torch.zeros(3), torch.float32, 4, False, "4 elements"),
    (torch.zeros(5), torch.float32, 4, False, "4 elements"),
    (torch.zeros(3), torch.float32, 4, True, "at least 4"),
    (torch.zeros(4, 2).t(), torch.float32, 8, False, "contiguous"),
    (torch.zeros(4), torch.float32, 4, False, "device tensor"),
    (torch.zeros(6), torch.float32, 4, True, "device tensor"),
])
def test_dptr_rejects(t, dtype, n, at_least, msg):
    with pytest.raises(M.ArgumentError, match=msg):
        B._dptr(t, dtype, n, at_least=at_least, what="buf")
    assert B._dptr(None, dtype, n) is None


def test_population_buffers_checked_before_the_library():
    dims = [24, 32, 32, 3]
    ok = [torch.zeros(2 * dims[l + 1] * dims[l]) for l in range(3)]
    short = list(ok)
    short[1] = torch.zeros(2 * 32 * 32 - 1)
    with pytest.raises(M.ArgumentError, match=r"weights\[1\]"):
        M.Population(M.POLICY_MLP_F32, 2, 3, dims=dims, weights=short)
    half = list(ok)
    half[0] = torch.zeros(2 * 32 * 24, dtype=torch.float16)
    with pytest.raises(M.ArgumentError, match=r"weights\[0\].*dtype"):
        M.Population(M.POLICY_MLP_F32, 2, 3, dims=dims, weights=half)
    with pytest.raises(M.ArgumentError, match=r"biases\[2\]"):
        M.Population(M.POLICY_MLP_F32, 2, 3, dims=dims, weights=ok,
                     biases=[None, None, torch.zeros(5)])
    with pytest.raises(M.ArgumentError, match="three weights"):
        M.Population(M.POLICY_MLP_F32, 2, 3, dims=dims, weights=ok[:2])
    with pytest.raises(M.ArgumentError, match="tab_logits"):
        M.Population(M.POLICY_TABULAR, 4, 3, tab_logits=torch.zeros(11))
    with pytest.raises(M.ArgumentError, match="policy_ids"):
        M.Population(M.POLICY_TABULAR, 4, 3, tab_logits=torch.zeros(12), policy_ids=[1, 2])
    # right sizes on the host: stopped at the device check, not in the library
    with pytest.raises(M.ArgumentError, match="device tensor"):
        M.Population(M.POLICY_MLP_F32, 2, 3, dims=dims, weights=ok)


def test_env_buffers_checked():
    d, na, A = 64, 4, 18
    good = dict(W=torch.zeros(d * d), emb=torch.zeros(na * A * d), u=torch.zeros(d))
    for k, bad in (("W", torch.zeros(d * d - 1)), ("emb", torch.zeros(2 * A * d)),
                   ("u", torch.zeros(d, dtype=torch.float64))):
        args = dict(good)
        args[k] = bad
        with pytest.raises(M.ArgumentError, match=k):
            M.Env(M.ENV_FEATURE, na, A, team=[1, 1, -1, -1], d=d, **args)
    with pytest.raises(M.ArgumentError, match="team"):
        M.Env(M.ENV_FEATURE, na, A, team=[1, -1], d=d, W=None, emb=None, u=None)
    with pytest.raises(M.ArgumentError, match="A"):
        M.Env(M.ENV_MATRIX, 2, 3, A=torch.zeros(8))


def test_trace_and_ring_checked_against_the_batch():
    env = M.Env(M.ENV_PURSUIT, 2, 5, grid=8)
    n, H = 10, 4
    ok = dict(actions=torch.zeros(H * n * 2, dtype=torch.uint8),
              logits=torch.zeros(2 * n * 2 * 5), states=torch.zeros(2 * n * 3, dtype=torch.uint8),
              perm=torch.zeros(n * 2, dtype=torch.int32), offsets=torch.zeros(4, dtype=torch.int32))
    for k, bad in (("actions", torch.zeros(H * n * 2 - 1, dtype=torch.uint8)),
                   ("logits", torch.zeros(2 * n * 2 * 5 - 1)),
                   ("states", torch.zeros(2 * n * 3 - 1, dtype=torch.uint8)),
                   ("perm", torch.zeros(n * 2, dtype=torch.int64)),
                   ("offsets", torch.zeros(3, dtype=torch.int32))):
        args = dict(ok)
        args[k] = bad
        tr = M.Trace(snap_steps=[0, 3], **{kk: None for kk in args})
        tr.actions, tr.logits, tr.states, tr.perm, tr.offsets = (
            args["actions"], args["logits"], args["states"], args["perm"], args["offsets"])
        with pytest.raises(M.ArgumentError, match=k):
            tr.checked(env, n, H, 3, 5)
    ring = M.Traj(8, 2, obs_shape=(1,), obs_dtype=torch.uint8, device="cpu")
    with pytest.raises(M.ArgumentError, match="traj.obs"):
        ring.check(env)                      # pursuit records hold 2 bytes each
    ring = M.Traj(8, 2, device="cpu")
    ring.desc.capacity = 9
    with pytest.raises(M.ArgumentError, match="capacity"):
        ring.check(env)
    with pytest.raises(M.ArgumentError, match="seats"):
        M.Traj(8, 3, device="cpu").check(env)


def test_solver_and_sampler_arguments_checked():
    with pytest.raises(M.ArgumentError, match="square"):
        M.solve_fp(torch.zeros((3, 4), dtype=torch.float64), 10)
    with pytest.raises(M.ArgumentError, match="dtype"):
        M.solve_fp(torch.zeros((3, 3)), 10)
    with pytest.raises(M.ArgumentError, match="sigma"):
        M.meta_sample_device(torch.zeros(7), 3, 10, 2, 1)
    with pytest.raises(M.ArgumentError, match="seat_row"):
        M.meta_sample_device(torch.zeros(6), 3, 10, 2, 1, seat_row=[0, 1, 1],
                             out=torch.zeros((10, 2), dtype=torch.int32))
    with pytest.raises(M.ArgumentError, match="ctr"):
        M.debug_philox(torch.zeros((5, 3), dtype=torch.int64), 1, 2)


def test_binding_has_no_bare_asserts():
    # argument checks must survive python -O
    import inspect
    src = inspect.getsource(B)
    assert "\n    assert " not in src and "\n        assert " not in src
