#!/usr/bin/env python3
"""Benchmark: payoff-table fill throughput on one MI355X.

One step = one full pass of the rollout path over one batch: draw every seat's
policy from the meta-strategy, bucket slots by policy, reset, H x (grouped
policy forward -> Gumbel-max sampling -> environment step with return
accumulation), reduce returns into the payoff table and read it back on the
host.  Inputs (weights, environment parameters, meta-strategy) are resident in
HBM before timing starts.

Default workload: the 4v4 team game on R^256 feature dynamics, 16384 envs x 8
seats, population of 128 bf16 MLPs 256-512-512-18, horizon 200 (the largest
configuration).  Other workloads: --workload matrix|iter|pursuit|feature|team.

Prints one JSON line with the throughput (live agent-frames/s), the fill time
(ms per step), the roofline of the grouped policy forward (HIP events on the
kernel's stream, over the timed region) and the CPU oracle timed on a bounded
sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_F32_MFMA_TFLOPS = 157.3  # MI355X dense fp32 MFMA
PEAK_HBM_GBS = 8000.0
NAME_TO_C = {"matrix": 1, "iter": 2, "pursuit": 3, "feature": 4, "team": 5}


def policy_flops_per_frame(dims):
    """Algorithmic flops of one policy forward (2 per multiply-add)."""
    return 2 * sum(dims[i] * dims[i + 1] for i in range(len(dims) - 1))


def describe(wl):
    d = {"workload": wl.name, "n_envs": wl.n_envs, "agents": wl.n_agents,
         "policies": wl.P, "horizon": wl.horizon, "actions": wl.n_actions}
    if wl.dims:
        d["policy"] = ("bf16" if wl.pol_kind == 2 else "fp32") + " MLP " + \
            "-".join(str(x) for x in wl.dims)
    else:
        d["policy"] = "tabular"
    if wl.d:
        d["state_dim"] = wl.d
    d["pairing"] = "blocked all pairs" if wl.pairs is not None else "meta-strategy sample"
    return d


PEAK_F32_ALU_TFLOPS = 78.6   # fp32 FMA without packed fp32 (256 CU x 4 SIMD x 16 lanes x 2 x 2.4 GHz)


def algorithmic_work(wl):
    """Per-launch algorithmic HBM bytes (and flops where the kernel is ALU- or
    MFMA-bound) of the per-step kernels: unique data each launch must read or
    write, counted once."""
    import workloads as W
    n, na, A = wl.n_envs, wl.n_agents, wl.n_actions
    ns = n * na
    out = {}
    # feature games on the 64-row bf16 kernel sample inside the policy kernel,
    # which hands the env step one action byte per slot; elsewhere the env
    # step samples and reads the step's logits once
    ksample = wl.env_kind == W.FEATURE and wl.pol_kind == W.MLP_BF16 and \
        policy_kernel(wl) == "mlp_bf16_kernel"
    sample = ns if ksample else ns * 4 * A
    if wl.env_kind == W.FEATURE:
        d = wl.d
        # state in and out, returns read-modify-write, W and the embedding
        # table once
        b = n * (8 * d + 8 * na) + 4 * d * d + 4 * na * A * d + 4 * d
        if wl.pol_kind == W.MLP_BF16 and policy_kernel(wl) == "mlp_bf16_kernel":
            b += n * 2 * d       # the bf16 observation rows for the 64-row kernel
        out["env"] = {"bytes": b, "flops": 2 * d * d * n}
    elif wl.env_kind == W.PURSUIT:
        out["env"] = {"bytes": n * (2 * 2 + 1 + 8 * na)}     # cells, done, returns
    elif wl.env_kind == W.ITER_MATRIX:
        out["env"] = {"bytes": n * (2 * 2 + 8 * na)}         # history, returns
    else:
        out["env"] = {"bytes": n * 8 * na}                   # returns
    out["env"]["bytes"] += sample
    if wl.dims:
        wbytes = (2 if wl.pol_kind == W.MLP_BF16 else 4) * wl.P * sum(
            wl.dims[i] * wl.dims[i + 1] for i in range(len(wl.dims) - 1))
        # feature observations, each env's once: fp32 state rows for the
        # persistent kernel, the env step's bf16 rows for the 64-row kernel
        obs = 0
        if wl.env_kind == W.FEATURE:
            obs = n * wl.d * (4 if policy_kernel(wl) == "mlp_bf16_persist_kernel" else 2)
        out["policy"] = {"bytes": wbytes + obs + sample,
                         "flops": policy_flops_per_frame(wl.dims) * ns}
    else:
        out["policy"] = {"bytes": wl.P * A * 4 + ns * 4 * A}
    # payoff reduction, once per fill: every seat's int32 policy id and each
    # row-side seat's fp32 return read once, the table's three accumulators
    # (sum, sum of squares: int64; count: uint32) updated once per cell
    n_row = int((wl.team > 0).sum())
    out["payoff"] = {"bytes": ns * 4 + n * n_row * 4 + wl.P * wl.P * 20}
    return out


def policy_kernel(wl):
    """Which bf16 policy kernel the library runs for this workload: the
    persistent 128-row kernel for d=512 feature observations with >= 256 slots
    per policy, the 64-row kernel otherwise."""
    import workloads as W
    if wl.env_kind == W.FEATURE and wl.d == 512 and wl.n_envs * wl.n_agents >= 256 * wl.P:
        return "mlp_bf16_persist_kernel"
    return "mlp_bf16_kernel"


def profiled_traffic(workload):
    """HBM bytes per launch of the grouped policy forward from the committed
    rocprofv3 summary of this workload (FETCH_SIZE and WRITE_SIZE scaled by the
    plain-copy calibration), or None when there is none or the kernel sources
    changed since it was taken."""
    import glob
    import hashlib
    h = hashlib.sha256()
    for f in ("k_policy.hip", "device.hpp", "internal.hpp"):
        with open(os.path.join(ROOT, "paper_2106_07551_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    cur = h.hexdigest()
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*.md"))):
        kv = {}
        for line in open(path):
            if "=" in line and not line.startswith(("#", "|", "-")):
                k, _, v = line.strip().partition("=")
                kv[k] = v
        if kv.get("workload") == workload and kv.get("kernel_source_sha256") == cur \
                and "traffic_bytes_per_launch" in kv:
            return int(kv["traffic_bytes_per_launch"]), os.path.relpath(path, ROOT)
    return None, None


# ---- CPU baseline: the oracle in one process per host core.  The processes
# are forked at the top of main(), before anything touches the GPU, and wait
# until the GPU measurements are done; each simulates its own disjoint whole
# episodes (env k*N + i of a fixed scramble of the batch) for a fixed wall-time
# budget.
_CPU = {}


def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or platform.machine()


def _oracle_shard(args):
    """Worker: whole episodes of envs i, i + N, ... (scrambled) until budget_s
    of wall time has passed; returns (frames, episodes, elapsed, cpu seconds)."""
    import numpy as np
    import oracle
    i, nproc, budget_s = args
    wl, pids = _CPU["wl"], _CPU["pids"]
    frames = envs = 0
    c0 = time.process_time()
    t0 = time.perf_counter()
    k = i
    while k < wl.n_envs:
        e = k * 997 % wl.n_envs
        r = oracle.rollout(wl, np.array([e]), pids[e:e + 1])
        frames += r["live_frames"]
        envs += 1
        k += nproc
        if time.perf_counter() - t0 >= budget_s:
            break
    return frames, envs, time.perf_counter() - t0, time.process_time() - c0


def cpu_pool_start(wl):
    """Fork one oracle process per usable host core (at most 16, the host
    share of one GPU on the target machines) before the GPU is initialised."""
    import multiprocessing as mp
    import oracle
    oracle.lib()
    _CPU["wl"] = wl
    _CPU["pids"] = wl.pairs if wl.pairs is not None else oracle.meta_sample(
        wl.sigma, wl.P, wl.n_envs, wl.n_agents, wl.seed)
    nproc = max(1, min(16, len(os.sched_getaffinity(0))))
    _CPU["nproc"] = nproc
    _CPU["pool"] = mp.get_context("fork").Pool(nproc)
    return nproc


def cpu_baseline(wl, budget_s=10.0):
    """The oracle (single-threaded C, one process per core) on disjoint whole
    episodes of the same workload: per-core and all-core agent-frames/s, and
    the projected all-core time of the whole table fill."""
    nproc, pool = _CPU["nproc"], _CPU["pool"]
    t0 = time.perf_counter()
    res = pool.map(_oracle_shard, [(i, nproc, budget_s) for i in range(nproc)])
    wall = time.perf_counter() - t0
    pool.close()
    pool.join()
    frames = sum(r[0] for r in res)
    envs = sum(r[1] for r in res)
    per_core = [r[0] / r[2] for r in res if r[2] > 0]
    all_core = frames / wall
    total_frames = wl.n_envs * wl.n_agents * wl.horizon   # live frames at most
    return {"value": all_core, "unit": "agent-frames/s", "cores": nproc, "kind": "oracle",
            "sample": f"{envs} whole episodes (H={wl.horizon}) of {wl.name} in {nproc} "
                      f"processes (disjoint envs), {frames} agent-frames in {wall:.1f} s "
                      f"wall",
            "cpu_model": _cpu_model(),
            "single_core_frames_per_s": round(sum(per_core) / len(per_core), 1),
            "single_core_note": "mean rate of one process while all run",
            "all_core_frames_per_s": round(all_core, 1),
            "cpu_seconds": round(sum(r[3] for r in res), 1),
            "projected_fill_s_all_cores": round(total_frames / all_core, 1),
            "projected_fill_note": f"{total_frames} agent-frames of the full table at the "
                                   f"all-core rate"}


def trajectory_timing(M, pop, env, wl, pairs, fill_ms, reps=2):
    """Fills that also write every step's records (actions, reward, flags and
    the compact observation) into a device ring holding the whole fill
    (malib_rollout_batch_traj), timed like the fills, beside the fill time
    without records."""
    import torch
    import workloads as W
    n, na, H = wl.n_envs, wl.n_agents, wl.horizon
    obs = {W.ITER_MATRIX: ((), torch.int16, 2), W.PURSUIT: ((2,), torch.uint8, 2),
           W.FEATURE: ((wl.d,), torch.int16, 2 * wl.d)}.get(wl.env_kind, (None, None, 0))
    cap = H * n
    tr = M.Traj(cap, na, obs_shape=obs[0], obs_dtype=obs[1])
    def fill():
        if wl.pairs is None:
            M.meta_sample(wl.sigma, wl.P, n, na, wl.seed, out=pairs)
        pop.rollout_traj(env, n, pairs, wl.seed, H, tr)
        return pop.payoff(reset=True)
    fill()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        fill()
    torch.cuda.synchronize()
    ms = 1000.0 * (time.perf_counter() - t0) / reps
    rec_bytes = na + 4 + 1 + obs[2]
    out = {"records": cap, "bytes_per_record": rec_bytes,
           "ring_bytes": cap * rec_bytes, "fill_ms_with_records": round(ms, 3),
           "fill_ms_without": round(fill_ms, 3),
           "overhead_frac": round(ms / fill_ms - 1.0, 4)}
    del tr
    return out


def meta_update_timing(M, pop, env, wl, pairs, iters, reps=5):
    """The meta-update after a fill, on the device: the table as a game
    (malib_payoff_matrix), `iters` steps of fictitious play (malib_solve_fp),
    the next policy ids drawn from the play counts, row side's counts for
    the row-side seats and the column side's for the others
    (malib_meta_sample_device), and the convergence figures of the last
    policy against the averages (malib_aggregate).  Each stage timed with HIP events on the
    stream it runs on, averaged over `reps` calls, after one untimed fill that
    leaves the table full."""
    import torch
    n, na, P = wl.n_envs, wl.n_agents, wl.P
    if wl.pairs is None:
        M.meta_sample(wl.sigma, P, n, na, wl.seed, out=pairs)
    pop.rollout(env, n, pairs, wl.seed, wl.horizon)
    seat_row = (wl.team < 0).astype("int32")
    game = torch.empty((P, P), dtype=torch.float64, device="cuda")
    sigma = torch.empty((2, P), dtype=torch.float32, device="cuda")
    gap = torch.empty(1, dtype=torch.float64, device="cuda")
    ids = torch.empty((n, na), dtype=torch.int32, device="cuda")
    agg = torch.empty(5, dtype=torch.float64, device="cuda")
    pi_ar = torch.empty(P, dtype=torch.float64, device="cuda")
    sig_ar = torch.empty((2, P), dtype=torch.float32, device="cuda")
    work_ar = torch.empty((P, P), dtype=torch.float64, device="cuda")
    work_lp = torch.empty((P + 1) * (2 * P + 1), dtype=torch.float64, device="cuda")
    stages = {
        "payoff_matrix": lambda: pop.payoff_matrix(out=game),
        "solve_fp": lambda: M.solve_fp(game, iters, sigma=sigma, gap=gap),
        "meta_sample_device": lambda: M.meta_sample_device(sigma, P, n, na, wl.seed + 1,
                                                           seat_row=seat_row, out=ids),
        "aggregate": lambda: M.aggregate(game, sigma, P - 1, P - 1, out=agg),
        # the alternative meta-solver (alpha = 1, population 50), timed alone:
        # it is not part of the fictitious-play update's total
        "solve_alpharank": lambda: M.solve_alpharank(game, 1.0, 50, pi=pi_ar, sigma=sig_ar,
                                                     work=work_ar),
        # and the LP solver (exact equilibrium), also outside the total
        "solve_lp": lambda: M.solve_lp(game, work=work_lp),
    }
    out = {"fp_iterations": iters, "policies": P, "envs": n}
    for name, fn in stages.items():
        fn()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        out[name + "_us"] = round(1000.0 * e0.elapsed_time(e1) / reps, 2)
    out["solve_fp_ns_per_iteration"] = round(1000.0 * out["solve_fp_us"] / iters, 1)
    out["total_us"] = round(sum(out[k + "_us"] for k in stages
                                if k not in ("solve_alpharank", "solve_lp")), 2)
    out["gap"] = float(gap.cpu()[0])
    out["improvement_of_policy_P-1"] = float(agg.cpu()[4])
    pop.payoff(reset=True)
    return out


def expansion_timing(M, IO, W, pop, env, wl, fill_ms):
    """Growing the population by one policy and simulating only the new row
    and column (2P + 1 cells) into the same table: malib_pop_extend, then
    malib_expansion_pairs + rollout + table read-back.  Blocked workloads
    play as many envs per new cell as the fill gives each cell; the sampled
    ones (pursuit, team) per_pair = n_envs / P^2, at least 1.  The new
    policy's weights come from the workload generator with one more policy."""
    import numpy as np
    import torch
    n, na, P = wl.n_envs, wl.n_agents, wl.P
    per_pair = max(1, n // (P * P))
    big = W.make(wl.number, P=P + 1, **({"per_pair": per_pair} if wl.pairs is not None else {}))
    def dev(a):
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()
    if wl.pol_kind == W.TABULAR:
        new = {"tab_logits": dev(big.tab_logits[P:])}
    else:
        new = {"weights": [dev(w[P:]) for w in big.weights],
               "biases": [dev(b[P:]) for b in big.biases] if big.biases else None}
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    pop.extend(1, **new)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    pairs = M.expansion_pairs(P + 1, P, per_pair, na, wl.team)
    n_new = pairs.shape[0]
    pop.rollout(env, n_new, pairs, wl.seed, wl.horizon, env_offset=n)
    tab = pop.payoff(reset=True)
    t2 = time.perf_counter()
    # the same new cells again in graph mode: the first fill records and
    # instantiates the graph, the second updates it in place (another seed)
    graph_ms = []
    pop.set_graph(True)
    for k in range(2):
        torch.cuda.synchronize()
        ta = time.perf_counter()
        pop.rollout(env, n_new, pairs, wl.seed + 1 + k, wl.horizon, env_offset=n)
        pop.payoff(reset=True)
        graph_ms.append(round(1000.0 * (time.perf_counter() - ta), 3))
    pop.set_graph(False)
    cells = (P + 1) ** 2 - P * P
    return {"policies": f"{P} -> {P + 1}", "cells": cells, "per_pair": per_pair,
            "envs": n_new, "extend_ms": round(1000.0 * (t1 - t0), 3),
            "fill_ms": round(1000.0 * (t2 - t1), 3),
            "fill_ms_graph_first": graph_ms[0], "fill_ms_graph_updated": graph_ms[1],
            "agent_frames_per_s": round(tab["live_frames"] / (t2 - t1), 1),
            "full_refill_cells": (P + 1) ** 2,
            "full_fill_ms_at_P": round(fill_ms, 3)}


def graph_timing(pop, one_step, steps, direct_ms):
    """The same fills with the handle in graph mode: each fill's launches
    (set-up, H x (forward, env step), payoff) recorded into a HIP graph and
    replayed with one launch; the executable graph is instantiated on the
    first (untimed) fill and updated in place on the timed ones."""
    import torch
    pop.set_graph(True)
    t0 = time.perf_counter()
    one_step()
    first = time.perf_counter() - t0
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        one_step()
    torch.cuda.synchronize()
    el = time.perf_counter() - t0
    pop.set_graph(False)
    ms = 1000.0 * el / steps
    return {"fill_ms": round(ms, 3), "first_fill_ms": round(1000.0 * first, 3),
            "direct_fill_ms": round(direct_ms, 3), "speedup": round(direct_ms / ms, 3),
            "steps": steps}


SWEEP_BASE = {"matrix": ("per_pair", 1024), "iter": ("per_pair", 4096),
              "pursuit": ("n_envs", 16384), "team": ("n_envs", 16384)}


def bandwidth_sweep(factors, horizon):
    """Bandwidth sweep of the streaming kernels: the env step (K2; the
    4v4 game's K3, which is fp32-ALU-bound, for comparison) and the payoff
    reduction (K4), with the env count of each workload scaled by each factor
    and every launch timed with HIP events.  One JSON line per point, labelled
    "bandwidth_sweep"; not the bench metric."""
    import torch
    import workloads as W
    import paper_2106_07551_amd as M
    from paper_2106_07551_amd import workload_io as IO
    torch.cuda.set_device(0)
    for name, (key, base) in SWEEP_BASE.items():
        c = NAME_TO_C[name]
        for f in factors:
            h = 1 if name == "matrix" else horizon
            wl = W.make(c, horizon=h, **{key: base * f})
            if wl.n_envs * wl.n_agents > (1 << 26):       # the batch limit of the library
                print(json.dumps({"bandwidth_sweep": name, "scale": f, "skipped":
                                  "more than 2^26 slots in one batch"}), flush=True)
                continue
            n, na = wl.n_envs, wl.n_agents
            pop = IO.make_population(wl)
            env = IO.make_env(wl)
            if wl.pairs is not None:
                pairs = IO.make_pairs(wl)
            else:
                pairs = torch.empty((n, na), dtype=torch.int32, device="cuda")
                M.meta_sample(wl.sigma, wl.P, n, na, wl.seed, out=pairs)
            pop.rollout(env, n, pairs, wl.seed, h)           # warm-up (buffers, caches)
            pop.payoff(reset=True)
            pop.profile_enable(True)
            pop.rollout(env, n, pairs, wl.seed + 1, h)
            pop.payoff(reset=True)
            work = algorithmic_work(wl)
            for kname, k in (("env", M.K_ENV), ("payoff", M.K_PAYOFF)):
                ms, cnt = pop.profile_read(k)
                avg_us = 1000.0 * ms / max(cnt, 1)
                b = work[kname]["bytes"]
                gbs = b / (avg_us * 1e-6) / 1e9
                row = {"bandwidth_sweep": name, "kernel": kname, "scale": f, "n_envs": n,
                       "slots": n * na, "launches": cnt, "avg_us": round(avg_us, 3),
                       "alg_bytes": b, "GBps": round(gbs, 1),
                       "hbm_frac": round(gbs / PEAK_HBM_GBS, 4)}
                if kname == "env" and "flops" in work["env"]:
                    tf = work["env"]["flops"] / (avg_us * 1e-6) / 1e12
                    row["fp32_TFLOPs"] = round(tf, 2)
                    row["alu_frac"] = round(tf / PEAK_F32_ALU_TFLOPS, 4)
                print(json.dumps(row), flush=True)
            pop.close()
            del pairs
            torch.cuda.empty_cache()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="team", choices=sorted(NAME_TO_C))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--event-every", type=int, default=0, metavar="K",
                    help="time one grouped-forward launch in K with HIP events during the "
                         "timed fills (default: about 16 per fill, at least every 4th)")
    ap.add_argument("--fill-only", action="store_true",
                    help="skip the trajectory, meta-update and expansion timings after the "
                         "fills (profiling runs: their small or extra launches would mix "
                         "into the per-kernel statistics)")
    ap.add_argument("--fp-iters", type=int, default=1000, metavar="T",
                    help="fictitious-play iterations of the meta-update timed after the "
                         "fills (table -> game -> solver -> meta-sample)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run 5 plain device-to-device copies of MIB MiB (the "
                         "reference kernel for scaling HBM byte counters) and exit")
    ap.add_argument("--envs", type=int, default=0, metavar="N",
                    help="envs of the batch for the sampled workloads (pursuit, team) "
                         "instead of the configuration's; e.g. one GPU's share of a "
                         "table split over several GPUs")
    ap.add_argument("--sweep", default="", metavar="F1,F2,...",
                    help="only run the bandwidth sweep of the env step and the payoff "
                         "reduction at these env-count factors (e.g. 1,8,16,32,64) and exit")
    ap.add_argument("--sweep-horizon", type=int, default=8)
    args = ap.parse_args()
    if args.sweep:
        bandwidth_sweep([int(x) for x in args.sweep.split(",")], args.sweep_horizon)
        return
    if args.copy_calibration:
        import torch
        nbytes = args.copy_calibration << 20
        src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": nbytes, "copies": 5}))
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the rollout path "
              "shards by env across GPUs with one all-reduce of the table, which is not "
              "built here", file=sys.stderr)
        sys.exit(2)

    import workloads as W
    if args.envs:
        if args.workload not in ("pursuit", "team") or args.envs < 1:
            print("--envs applies to the sampled workloads (pursuit, team) and must be "
                  ">= 1", file=sys.stderr)
            sys.exit(2)
        wl = W.make(NAME_TO_C[args.workload], n_envs=args.envs)
    else:
        wl = W.make(NAME_TO_C[args.workload])
    if not args.no_cpu_baseline:
        cpu_pool_start(wl)        # before anything initialises the GPU

    import numpy as np
    import torch
    import paper_2106_07551_amd as M
    from paper_2106_07551_amd import workload_io as IO

    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    pop = IO.make_population(wl)
    env = IO.make_env(wl)
    n, na = wl.n_envs, wl.n_agents
    pairs = None
    if wl.pairs is not None:
        pairs = IO.make_pairs(wl)
    else:
        pairs = torch.empty((n, na), dtype=torch.int32, device="cuda")
    torch.cuda.synchronize()

    def one_step():
        if wl.pairs is None:
            M.meta_sample(wl.sigma, wl.P, n, na, wl.seed, out=pairs)
        pop.rollout(env, n, pairs, wl.seed, wl.horizon)
        return pop.payoff(reset=True)

    for _ in range(args.warmup):
        one_step()
    torch.cuda.synchronize()

    # timed region: HIP events around one grouped-forward launch in `every`
    # (about 16 per fill): the events' own cost shows up in the fill time, by
    # ~1% on the 4v4 game and ~2% on pursuit at one launch in four
    every = args.event_every or max(4, wl.horizon // 16)
    pop.profile_enable(True, kernels=[M.K_POLICY], every=every)
    frames = 0
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    step_s = []
    for _ in range(args.steps):
        ts = time.perf_counter()
        tab = one_step()          # ends with the table on the host (synchronizes)
        step_s.append(time.perf_counter() - ts)
        frames += tab["live_frames"]
    torch.cuda.synchronize()
    el = time.perf_counter() - t0
    kern = {}
    ms, cnt = pop.profile_read(M.K_POLICY)
    policy_avg_us = 1000.0 * ms / max(cnt, 1)
    policy_timed = cnt
    # per-kernel breakdown from one more (untimed) fill with every launch timed
    pop.profile_enable(True)
    one_step()
    work = algorithmic_work(wl)
    # per step for the policy forward and the env step, per fill for set-up
    # and payoff
    for name, k in (("policy", M.K_POLICY), ("env", M.K_ENV), ("setup", M.K_SETUP),
                    ("payoff", M.K_PAYOFF)):
        ms, cnt = pop.profile_read(k)
        per = wl.horizon if name in ("policy", "env") else 1
        kern[name] = {"total_ms": round(ms, 3), "launches": cnt,
                      "avg_us": round(1000.0 * ms / max(cnt, 1), 3),
                      "per_step_us" if per > 1 else "per_fill_us": round(1000.0 * ms / per, 3)}
        if name in work and cnt:
            t = ms * 1e-3 / per
            w = work[name]
            kern[name]["alg_bytes"] = w["bytes"]
            kern[name]["hbm_GBps"] = round(w["bytes"] / t / 1e9, 1)
            kern[name]["hbm_frac"] = round(w["bytes"] / t / 1e9 / PEAK_HBM_GBS, 4)
            if name == "env" and "flops" in w:
                kern[name]["fp32_TFLOPs"] = round(w["flops"] / t / 1e12, 2)
                kern[name]["alu_frac"] = round(w["flops"] / t / 1e12 / PEAK_F32_ALU_TFLOPS, 4)
    pop.profile_enable(False)
    traj = meta = expand = graph = None
    if not args.fill_only:
        graph = graph_timing(pop, one_step, args.steps, 1000.0 * el / args.steps)
        traj = trajectory_timing(M, pop, env, wl, pairs, 1000.0 * el / args.steps)
        meta = meta_update_timing(M, pop, env, wl, pairs, args.fp_iters)
        expand = expansion_timing(M, IO, W, pop, env, wl, 1000.0 * el / args.steps)

    ms_step = 1000.0 * el / args.steps
    value = frames / el
    roof = None
    if wl.pol_kind in (W.MLP_BF16, W.MLP_F32):
        # the grouped policy forward on MFMA: bf16 operands (fp32 accumulation)
        # or fp32 throughout (iterated game), each against its own dense peak
        bf16 = wl.pol_kind == W.MLP_BF16
        peak = PEAK_BF16_TFLOPS if bf16 else PEAK_F32_MFMA_TFLOPS
        kname = policy_kernel(wl) if bf16 else "mlp_f32_kernel"
        flops = policy_flops_per_frame(wl.dims) * n * na        # per launch
        avg_s = policy_avg_us * 1e-6
        ach = flops / avg_s / 1e12
        # the committed counters are per launch of the configuration's batch
        traffic, src = profiled_traffic(wl.name) if not args.envs else (None, None)
        roof = {"bound": "mfma", "achieved": round(ach, 2), "peak": peak,
                "unit": "TFLOP/s", "frac": round(ach / peak, 4),
                "traffic": traffic, "kernel": "grouped policy forward (" + kname + ")",
                "flops_per_launch": flops, "avg_launch_us": round(policy_avg_us, 3),
                "timed_launches": policy_timed}
        if traffic is not None:
            roof["traffic_unit"] = "bytes per launch (HBM, rocprofv3 FETCH_SIZE+WRITE_SIZE)"
            roof["traffic_source"] = src
            roof["traffic_GBps"] = round(traffic / avg_s / 1e9, 1)
    out = {
        "metric": "agent-frames/s on 1 MI355X (payoff-table fill)",
        "value": round(value, 1),
        "unit": "agent-frames/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 3),
        "fill_time_ms": round(ms_step, 3),
        "fill_time_ms_median": round(1000.0 * sorted(step_s)[len(step_s) // 2], 3),
        "fill_time_ms_min": round(1000.0 * min(step_s), 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if wl.pol_kind == W.MLP_BF16 else "fp32",
        "data": "synthetic (seeded generator; random-init policies)",
        "config": describe(wl),
        "roofline": roof,
        "kernels": kern,
        "trajectory": traj,
        "meta_update": meta,
        "expansion": expand,
        "graph_mode": graph,
        "frames_per_step": frames // max(args.steps, 1),
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl)
        out["cpu_baseline"]["value"] = round(out["cpu_baseline"]["value"], 1)
        out["cpu_baseline"]["gpu_speedup_all_cores"] = round(
            value / out["cpu_baseline"]["value"], 1)
    pop.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
