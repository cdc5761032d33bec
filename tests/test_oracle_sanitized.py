"""The oracle under AddressSanitizer and UndefinedBehaviorSanitizer (CPU).

oracle.c is rebuilt with gcc -fsanitize=address,undefined (any UB report
aborts) and exercised in a child process that preloads gcc's ASan runtime:
whole episodes of all five games (both MLP kinds with nonzero biases,
tabular policies, the team game), the meta-sampler, fictitious play, the
tanh/exp/bf16 ranges and the payoff reduction.  The child must exit cleanly
with no sanitizer report."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

CHILD = r"""
import numpy as np
import oracle
import workloads as W

def run(wl, n, horizon):
    pids = oracle.meta_sample(wl.sigma, wl.P, n, wl.n_agents, wl.seed) if wl.pairs is None \
        else wl.pairs[:n]
    o = oracle.rollout(wl, np.arange(n), pids, horizon=horizon, want_actions=True,
                       want_logits=True, want_states=True, want_rewards=True)
    assert o["fails"] == 0 and np.isfinite(o["returns"]).all()
    return o

for c, kw, n, h in [(1, dict(per_pair=4), 16, 1), (2, dict(P=4, per_pair=2), 32, 6),
                    (3, dict(n_envs=64), 24, 12), (4, dict(P=3, per_pair=2), 9, 3),
                    (5, dict(n_envs=32), 6, 3)]:
    wl = W.make(c, **kw)
    if wl.pol_kind != 0:
        wl = W.with_policies(wl, wl.pol_kind, wl.dims, variant=1, bias_var=0.1)
    run(wl, n, h)
run(W.team_variant(4, P=5, n_envs=12, horizon=4), 12, 4)

sig = np.random.default_rng(0).random((2, 7)).astype(np.float32)
ids = oracle.meta_sample(sig, 7, 100, 2, 3)
assert ids.min() >= 0 and ids.max() < 7
M = np.random.default_rng(1).uniform(-1, 1, (9, 9))
cx, cy, gap = oracle.solve_fp(M, 200)
assert np.isfinite(gap)
assert oracle.tanh_range(0x3F000000, 4096).shape == (4096,)
assert oracle.bf16_range(0x7F7F0000, 4096).shape == (4096,)
x = np.random.default_rng(2).uniform(-20, 20, 4096).astype(np.float32)
assert np.isfinite(oracle.exp_many(x)).all() and np.isfinite(oracle.tanh_many(x)).all()
print("sanitized oracle ok")
"""


def test_oracle_clean_under_asan_and_ubsan(tmp_path):
    import oracle
    asan = subprocess.check_output(["gcc", "-print-file-name=libasan.so"], text=True).strip()
    if not os.path.isabs(asan) or not os.path.exists(asan):
        pytest.skip("gcc's AddressSanitizer runtime is not installed")
    lib = oracle.build_sanitized(str(tmp_path / "liboracle_san.so"))
    env = dict(os.environ)
    env.update({
        "LD_PRELOAD": asan,
        "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=0:halt_on_error=1",
        "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1",
        "MALIB_ORACLE_LIB": lib,
        "PYTHONPATH": ROOT + os.pathsep + env.get("PYTHONPATH", ""),
    })
    p = subprocess.run([sys.executable, "-c", CHILD], cwd=ROOT, env=env, capture_output=True,
                       text=True, timeout=600)
    out = p.stdout + p.stderr
    assert p.returncode == 0, out[-4000:]
    assert "sanitized oracle ok" in p.stdout
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
