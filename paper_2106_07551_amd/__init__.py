"""MI355X (gfx950) payoff-table rollout library: Python binding.

The compute path is ``libmalib.so`` (hand-written HIP kernels behind the C ABI
in ``include/malib.h``); this package only marshals arguments to it with
ctypes and uses torch for device memory and streams.  There is no CPU
fallback: importing the binding without the built library raises.
"""
from .binding import (  # noqa: F401
    MalibError, ArgumentError, Population, Env, Trace, Traj, meta_sample,
    meta_sample_device, solve_fp, solve_alpharank, solve_lp,
    expansion_pairs, aggregate,
    debug_tanh_ref, debug_bf16, debug_philox,
    lib, LIB_PATH, POLICY_TABULAR, POLICY_MLP_F32, POLICY_MLP_BF16, ENV_MATRIX,
    ENV_ITER_MATRIX, ENV_PURSUIT, ENV_FEATURE, INIT_PER_ENV, INIT_SHARED, K_POLICY,
    K_SAMPLE, K_ENV, K_SETUP, K_PAYOFF, EXPORTS,
)
