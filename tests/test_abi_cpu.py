"""Host-side checks of the C ABI that need no GPU: the library loads, exports
every function include/malib.h declares, and rejects invalid arguments
before touching the device."""
import ctypes as C
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _header_functions():
    src = open(os.path.join(ROOT, "include", "malib.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(malib_[a-z_0-9]+)\s*\(", src)))


def test_header_declares_the_boundary():
    fns = _header_functions()
    for need in ("malib_pop_create", "malib_rollout_batch", "malib_payoff_eval",
                 "malib_meta_sample"):
        assert need in fns


def test_library_exports_every_declared_symbol():
    import paper_2106_07551_amd as M
    L = M.lib()
    fns = _header_functions()
    assert sorted(M.EXPORTS) == fns
    for f in fns:
        assert hasattr(L, f), f


def test_validation_before_device_work():
    import paper_2106_07551_amd as M
    L = M.lib()
    B = M.binding
    h = C.c_void_p()
    d = B.PopDesc()
    d.kind, d.n_policies, d.n_actions = B.POLICY_TABULAR, 0, 3
    assert L.malib_pop_create(C.byref(d), None, C.byref(h)) == B.E_INVAL
    assert b"n_policies" in L.malib_last_error()
    d.n_policies, d.n_actions = 4, 40
    assert L.malib_pop_create(C.byref(d), None, C.byref(h)) == B.E_INVAL
    d.n_actions = 3
    assert L.malib_pop_create(C.byref(d), None, C.byref(h)) == B.E_INVAL   # no tab_logits
    d.kind, d.n_layers = B.POLICY_MLP_BF16, 2
    assert L.malib_pop_create(C.byref(d), None, C.byref(h)) == B.E_UNSUPPORTED
    # widths beyond 1024, for either MLP kind (the weight pointers are never read)
    fake = (C.c_void_p * 3)(16, 16, 16)
    for kind in (B.POLICY_MLP_F32, B.POLICY_MLP_BF16):
        for dims in ([24, 1025, 64, 3], [2048, 64, 64, 3], [24, 64, 4096, 3]):
            dd = (C.c_int32 * 4)(*dims)
            d.kind, d.n_layers, d.n_actions = kind, 3, 3
            d.dims = C.cast(dd, type(d.dims))
            d.weights = C.cast(fake, type(d.weights))
            assert L.malib_pop_create(C.byref(d), None, C.byref(h)) == B.E_UNSUPPORTED, dims
            assert b"1024" in L.malib_last_error()
    dd = (C.c_int32 * 4)(24, 64, 64, 5)        # dims[3] != n_actions
    d.dims = C.cast(dd, type(d.dims))
    assert L.malib_pop_create(C.byref(d), None, C.byref(h)) == B.E_INVAL
    assert L.malib_pop_create(None, None, C.byref(h)) == B.E_INVAL
    assert L.malib_rollout_batch(None, None, 1, None, 0, 0, 1, None, None, None) == B.E_INVAL
    assert L.malib_payoff_eval(None, None, 0, None, None, None, None) == B.E_INVAL
    sig = np.array([1.0, -0.5], np.float32)
    out = C.c_void_p(16)  # never dereferenced: validation fails first
    assert L.malib_meta_sample(sig.ctypes.data, 1, 2, 10, 2, 1, 0, out, None) == B.E_INVAL
    sig = np.array([0.0, 0.0], np.float32)
    assert L.malib_meta_sample(sig.ctypes.data, 1, 2, 10, 2, 1, 0, out, None) == B.E_INVAL
    sig = np.array([1.0, np.inf], np.float32)
    assert L.malib_meta_sample(sig.ctypes.data, 1, 2, 10, 2, 1, 0, out, None) == B.E_INVAL
    sig = np.array([1.0, 1.0], np.float32)
    assert L.malib_meta_sample(sig.ctypes.data, 3, 2, 10, 2, 1, 0, out, None) == B.E_INVAL
    # n_envs far past the 2^26-slot limit: rejected, no int64 overflow in the check
    assert L.malib_meta_sample(sig.ctypes.data, 1, 2, 1 << 62, 8, 1, 0, out, None) == B.E_INVAL
    assert L.malib_meta_sample_device(C.c_void_p(16), 1, 2, 1 << 62, 8, None, 1, 0, out,
                                      None) == B.E_INVAL
    assert L.malib_meta_sample(sig.ctypes.data, 1, 2, 10, 9, 1, 0, out, None) == B.E_INVAL
    # device-weight sampling and the solver: argument checks come before any
    # device access (the pointers below are never dereferenced)
    dev = C.c_void_p(16)
    bad_rows = np.array([0, 2], np.int32)
    assert L.malib_meta_sample_device(dev, 2, 4, 10, 2, bad_rows.ctypes.data, 1, 0, out,
                                      None) == B.E_INVAL
    assert b"seat_row[1]" in L.malib_last_error()
    rows = np.zeros(2, np.int32)
    assert L.malib_meta_sample_device(dev, 9, 4, 10, 2, rows.ctypes.data, 1, 0, out,
                                      None) == B.E_INVAL
    assert L.malib_meta_sample_device(dev, 3, 4, 10, 2, None, 1, 0, out, None) == B.E_INVAL
    assert L.malib_meta_sample_device(None, 1, 4, 10, 2, None, 1, 0, out, None) == B.E_INVAL
    assert L.malib_meta_sample_device(dev, 1, 0, 10, 2, None, 1, 0, out, None) == B.E_INVAL
    assert L.malib_solve_fp(dev, 4, 0, dev, None, None) == B.E_INVAL
    assert L.malib_solve_fp(dev, 4, (1 << 24) + 1, dev, None, None) == B.E_INVAL
    assert L.malib_solve_fp(dev, 257, 10, dev, None, None) == B.E_INVAL
    assert L.malib_solve_fp(None, 4, 10, dev, None, None) == B.E_INVAL
    assert L.malib_solve_alpharank(None, 4, 1.0, 10, None, dev, None, None) == B.E_INVAL
    assert L.malib_solve_alpharank(dev, 4, 1.0, 10, None, None, None, None) == B.E_INVAL
    assert L.malib_solve_alpharank(dev, 0, 1.0, 10, None, dev, None, None) == B.E_INVAL
    assert L.malib_solve_alpharank(dev, 257, 1.0, 10, None, dev, None, None) == B.E_INVAL
    assert L.malib_solve_alpharank(dev, 4, -1.0, 10, None, dev, None, None) == B.E_INVAL
    assert L.malib_solve_alpharank(dev, 4, float("nan"), 10, None, dev, None, None) == B.E_INVAL
    assert L.malib_solve_alpharank(dev, 4, float("inf"), 10, None, dev, None, None) == B.E_INVAL
    assert L.malib_solve_alpharank(dev, 4, 1.0, 0, None, dev, None, None) == B.E_INVAL
    assert L.malib_solve_alpharank(dev, 200, 1.0, 10, None, dev, None, None) == B.E_INVAL
    assert b"workspace" in L.malib_last_error()
    assert L.malib_solve_lp(None, 4, None, dev, dev, dev, None, None, None) == B.E_INVAL
    assert L.malib_solve_lp(dev, 4, None, None, dev, dev, None, None, None) == B.E_INVAL
    assert L.malib_solve_lp(dev, 0, None, dev, dev, dev, None, None, None) == B.E_INVAL
    assert L.malib_solve_lp(dev, 257, None, dev, dev, dev, None, None, None) == B.E_INVAL
    assert L.malib_solve_lp(dev, 97, None, dev, dev, dev, None, None, None) == B.E_INVAL
    assert b"workspace" in L.malib_last_error()
    assert L.malib_payoff_matrix(None, dev, None) == B.E_INVAL
    assert L.malib_aggregate(dev, 4, dev, 4, 0, dev, None) == B.E_INVAL
    assert L.malib_aggregate(dev, 4, dev, 0, -2, dev, None) == B.E_INVAL
    assert L.malib_aggregate(dev, 0, dev, 0, 0, dev, None) == B.E_INVAL
    assert L.malib_aggregate(None, 4, dev, 0, 0, dev, None) == B.E_INVAL
    assert L.malib_expansion_pairs(4, 4, 1, 2, None, out, None) == B.E_INVAL
    assert L.malib_expansion_pairs(4, 1, 0, 2, None, out, None) == B.E_INVAL
    assert L.malib_expansion_pairs(4, 1, 1, 3, None, out, None) == B.E_INVAL
    # 256^2 cells x 1100 envs x 2 seats exceeds the 2^26-slot batch limit
    assert L.malib_expansion_pairs(256, 0, 1100, 2, None, out, None) == B.E_INVAL
    assert b"2^26" in L.malib_last_error()
    bad_team = np.array([1, 1], np.int8)
    assert L.malib_expansion_pairs(4, 1, 1, 2, bad_team.ctypes.data, out, None) == B.E_INVAL
    assert L.malib_pop_extend(None, None, None) == B.E_INVAL
    # trajectory rings: the descriptor is checked before the rollout's own checks
    assert L.malib_rollout_batch_traj(None, None, 1, None, 0, 0, 1, None, None,
                                      None) == B.E_INVAL
    td = B.TrajDesc(16, 16, 16, None, 0, 0)             # capacity 0
    assert L.malib_rollout_batch_traj(None, None, 1, None, 0, 0, 1, None, C.byref(td),
                                      None) == B.E_INVAL
    assert b"capacity" in L.malib_last_error()
    td = B.TrajDesc(16, None, 16, None, 8, 0)           # no reward buffer
    assert L.malib_rollout_batch_traj(None, None, 1, None, 0, 0, 1, None, C.byref(td),
                                      None) == B.E_INVAL
    td = B.TrajDesc(16, 16, 16, None, 8, 0)             # a valid ring, no population
    assert L.malib_rollout_batch_traj(None, None, 1, None, 0, 0, 1, None, C.byref(td),
                                      None) == B.E_INVAL
    assert td.cursor == 0
    assert L.malib_profile_enable(None, 1, 1) == B.E_INVAL
    assert L.malib_debug_tanh_ref(None, None, 4, None) == B.E_INVAL


def test_binding_fails_loudly_without_library(tmp_path, monkeypatch):
    import paper_2106_07551_amd.binding as B
    monkeypatch.setattr(B, "_lib", None)
    monkeypatch.setattr(B, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(ImportError):
        B.lib()


def test_product_never_imports_oracle():
    pkg = os.path.join(ROOT, "paper_2106_07551_amd")
    for dp, _, fs in os.walk(pkg):
        for f in fs:
            if f.endswith((".py", ".hip", ".hpp", ".cpp", ".h")):
                src = open(os.path.join(dp, f)).read()
                assert "oracle" not in src.replace("Oracle", ""), f


def test_policy_ids_validated_before_device_work():
    """Policy ids are the caller's keys (Sec. 3.1 pools, Appendix C.2
    Dict[PolicyID, float]): duplicates are rejected on the host before any
    device work; the getter rejects a NULL handle and a short buffer."""
    import paper_2106_07551_amd as M
    L = M.lib()
    B = M.binding
    h = C.c_void_p()
    d = B.PopDesc()
    d.kind, d.n_policies, d.n_actions = B.POLICY_TABULAR, 3, 3
    d.tab_logits = 16      # never dereferenced: validation fails first
    ids = (C.c_int64 * 3)(5, 7, 5)
    d.policy_ids = C.cast(ids, C.POINTER(C.c_int64))
    assert L.malib_pop_create(C.byref(d), None, C.byref(h)) == B.E_INVAL
    assert b"appears twice" in L.malib_last_error()
    assert not h.value
    n = C.c_int32()
    assert L.malib_pop_policy_ids(None, None, 0, C.byref(n)) == B.E_INVAL


def test_fault_hook_forces_nomem(monkeypatch):
    """MALIB_FAULT_ALLOC makes the library's allocations fail as out of memory
    (here the meta-sampler's threshold buffer, reached after validation with no
    device work before it); cleared, the same call gets past the hook."""
    import paper_2106_07551_amd as M
    L = M.lib()
    B = M.binding
    sig = np.array([1.0, 2.0, 3.0], np.float32)
    out = C.c_void_p(16)   # never dereferenced: the allocation fails first
    monkeypatch.setenv("MALIB_FAULT_ALLOC", "1")
    assert L.malib_meta_sample(sig.ctypes.data, 1, 3, 10, 2, 1, 0, out, None) == B.E_NOMEM
    assert b"out of memory" in L.malib_last_error().lower() or b"dev_malloc_async" in \
        L.malib_last_error()
    monkeypatch.setenv("MALIB_FAULT_ALLOC", "0")
    # without the hook the call reaches the HIP runtime (no GPU here: a HIP error)
    st = L.malib_meta_sample(sig.ctypes.data, 1, 3, 10, 2, 1, 0, out, None)
    assert st != B.E_NOMEM and st != B.E_INVAL
