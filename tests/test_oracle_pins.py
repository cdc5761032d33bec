"""Pins of the CPU oracle against things other than itself.

Each test checks one oracle component against a library routine, a closed
form, an invariant the mathematics fixes, or brute-force enumeration, so that a
plausible slip in it (a dropped term, a wrong sign or index, a transposed
operand) fails here.  Citations are to MALib (arXiv 2106.07551) and to the
published definitions the design reads into it.
"""
import math
import os

import numpy as np
import pytest
import scipy.stats as st
import torch

import oracle
import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def softmax(l):
    l = np.asarray(l, np.float64)
    e = np.exp(l - l.max())
    return e / e.sum()


# ---------------------------------------------------------------- random stream

def test_philox_known_answers():
    """Philox4x64-10 against the Random123 known-answer vectors (Salmon et al.,
    SC'11)."""
    rows = [l.split() for l in open(os.path.join(GOLDEN, "philox4x64_10_kat.txt"))
            if l.strip() and not l.startswith("#")]
    assert len(rows) == 3
    for r in rows:
        v = [int(x, 16) for x in r]
        out = oracle.philox(v[0:4], v[4:6])
        assert [int(x) for x in out] == v[6:10]


def test_philox_matches_numpy():
    """numpy's Philox is Philox4x64-10; it increments the 256-bit counter before
    hashing, so the block of counter c is numpy's first draw from c - 1."""
    rng = np.random.default_rng(1)
    for _ in range(200):
        ctr = rng.integers(1, 2**63, size=4, dtype=np.uint64)
        key = rng.integers(0, 2**63, size=2, dtype=np.uint64)
        before = ctr.copy()
        before[0] -= np.uint64(1)
        g = np.random.Philox(key=key, counter=before)
        assert np.array_equal(g.random_raw(4), oracle.philox(ctr, key))


def test_lane_layout():
    """Lane 2w is the low half of word w, lane 2w+1 the high half; counter =
    (env, step, purpose<<32 | slot, block), key = (seed, 0)."""
    seed, g, t, purpose, slot, block = 0x1234, 77, 5, 2, 3, 1
    ctr = [g, t, (purpose << 32) | slot, block]
    out = oracle.philox(ctr, [seed, 0])
    for ln in range(8):
        w = int(out[ln // 2])
        want = (w >> 32) if ln & 1 else (w & 0xFFFFFFFF)
        assert oracle.lane(seed, g, t, purpose, slot, block, ln) == want


def test_uniform_open_interval_exact():
    """u = (2*(x>>9)+1) * 2^-24: every value is an odd multiple of 2^-24 strictly
    inside (0, 1), monotone in x, and each 23-bit prefix maps to its own value."""
    xs = np.arange(0, 1 << 32, 1 << 9, dtype=np.uint64)   # one x per prefix
    u = np.concatenate([oracle.uniform_range(int(x0), 1) for x0 in xs[:4]] +
                       [oracle.uniform_range(0, 1 << 16)[::1 << 9]])
    assert oracle.uniform(0) == 2.0**-24
    assert oracle.uniform(0xFFFFFFFF) == 1.0 - 2.0**-24
    full = np.array([oracle.uniform(int(x)) for x in xs[::4096]], np.float64)
    k = full * 2**24
    assert np.all(k == np.round(k)) and np.all(k % 2 == 1)
    assert np.all(np.diff(full) > 0)
    assert np.all((u > 0) & (u < 1))


def test_gumbel_distribution_ks():
    """-log(-log u) on the uniform stream is standard Gumbel: KS test against
    the CDF exp(-exp(-g))."""
    x = np.random.default_rng(3).integers(0, 2**32, size=100000, dtype=np.uint64)
    g = np.array([oracle.gumbel(oracle.uniform(int(v))) for v in x[:20000]])
    res = st.kstest(g, lambda v: np.exp(-np.exp(-v)))
    assert res.pvalue > 1e-3


def _tabular(n_actions, logits, n_envs, seed_variant=0):
    """A one-step game with one tabular policy per seat (for sampling pins)."""
    P = logits.shape[0]
    wl = W.Workload(90, "tab", W.MATRIX, 2, n_actions, np.array([1, -1], np.int8), 1,
                    n_envs, W.TABULAR, P, [], [], [], tab_logits=logits.astype(np.float32),
                    A=np.zeros((n_actions, n_actions), np.float32))
    wl.seed = W.ROLLOUT_KEY_BASE + 90 + seed_variant
    return wl


@pytest.mark.parametrize("n_actions", [3, 18])
def test_gumbel_max_is_softmax(n_actions):
    """Gumbel-max sampling draws action a with probability softmax(l)_a
    (textbook identity); checked by a chi-square test over 60000 draws.  The
    18-action case spans three Philox blocks."""
    rng = np.random.default_rng(n_actions)
    logits = rng.standard_normal((2, n_actions)).astype(np.float32)
    n = 60000
    wl = _tabular(n_actions, logits, n)
    pids = np.tile(np.array([[0, 1]], np.int32), (n, 1))
    r = oracle.rollout(wl, np.arange(n), pids, want_actions=True)
    for seat in range(2):
        counts = np.bincount(r["actions"][0, :, seat], minlength=n_actions)
        p = softmax(logits[seat])
        res = st.chisquare(counts, p * n)
        assert res.pvalue > 1e-4, (seat, res)


# ------------------------------------------------------------------------ bf16

def test_bf16_rne_matches_torch():
    """Round-to-nearest-even to bfloat16 against torch's conversion, for every
    low half-word under a set of high half-words that covers zeros, subnormals,
    normals of many exponents, the largest finite values, infinities and NaNs,
    with both signs."""
    highs = set()
    for e in list(range(0, 6)) + list(range(120, 136)) + list(range(250, 256)):
        for m in (0x00, 0x01, 0x3F, 0x40, 0x7E, 0x7F):
            highs.add((e << 7) | m)
    highs = sorted(highs)
    for sign in (0, 0x8000):
        for h in highs:
            first = ((sign | h) << 16)
            o = oracle.bf16_range(first, 1 << 16)
            bits = (np.arange(1 << 16, dtype=np.uint32) + np.uint32(first))
            x = torch.from_numpy(bits.view(np.float32).copy())
            ref = x.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
            nan = np.isnan(bits.view(np.float32))
            ok = (o == ref) | (nan & ((o & 0x7F80) == 0x7F80) & ((o & 0x7F) != 0))
            assert ok.all(), hex(first + int(np.argmin(ok)))


# --------------------------------------------------------------- exp/tanh defs

def _ulps(got, ref):
    ref = np.asarray(ref, np.float64)
    got = np.asarray(got, np.float64)
    ex = np.frexp(np.abs(ref))[1]
    ulp = np.maximum(np.ldexp(1.0, ex - 24), 2.0**-149)
    return np.abs(got - ref) / ulp


def test_exp_ref_accuracy():
    """exp_ref on [1.1, 18.02] (the range tanh_ref uses) within 2 ulp of fp64 exp."""
    x = np.linspace(1.1, 18.02, 400001).astype(np.float32)
    assert _ulps(oracle.exp_many(x), np.exp(x.astype(np.float64))).max() <= 2.0


def test_tanh_ref_accuracy_sweep():
    """tanh_ref within 2 ulp of fp64 tanh: every 97th fp32 bit pattern of each
    sign, plus dense sweeps across both branch points (0.55, 9.01) and near 0.
    (The full sweep over all 2^31 positive patterns gives 1.59 ulp.)"""
    worst = 0.0
    for sign in (0, 1 << 31):
        bits = (np.arange(0, 0x7F800000, 97, dtype=np.uint64) | sign).astype(np.uint32)
        x = bits.view(np.float32)
        worst = max(worst, _ulps(oracle.tanh_many(x), np.tanh(x.astype(np.float64))).max())
    for c in (0.55, 9.01, 1e-3):
        x = np.float32(c)
        b = int(np.array([x]).view(np.uint32)[0])
        bits = np.arange(b - 200000, b + 200000, dtype=np.uint32)
        xs = bits.view(np.float32)
        worst = max(worst, _ulps(oracle.tanh_many(xs), np.tanh(xs.astype(np.float64))).max())
    assert worst <= 2.0, worst


def test_tanh_ref_odd_and_special():
    rng = np.random.default_rng(5)
    x = (rng.standard_normal(200000) * 4).astype(np.float32)
    assert np.array_equal(oracle.tanh_many(-x), -oracle.tanh_many(x))
    assert oracle.tanh_ref(0.0) == 0.0
    assert math.copysign(1, oracle.tanh_ref(-0.0)) == -1
    assert oracle.tanh_ref(float("inf")) == 1.0
    assert oracle.tanh_ref(float("-inf")) == -1.0
    assert math.isnan(oracle.tanh_ref(float("nan")))
    assert oracle.tanh_ref(9.02) == 1.0
    # monotone (non-decreasing) on a dense grid
    g = np.linspace(-10, 10, 2000001).astype(np.float32)
    assert np.all(np.diff(oracle.tanh_many(g)) >= 0)


# ----------------------------------------------------------------- meta-sample

def test_meta_sample_chi_square():
    """Per-seat policy draws follow the meta-strategy sigma (the per-agent
    policy distribution of Appendix C.2's single-instance example)."""
    wl = W.make(5, P=128)
    n = 20000
    pids = oracle.meta_sample(wl.sigma, wl.P, n, 8, wl.seed)
    counts = np.bincount(pids.ravel(), minlength=128)
    exp = wl.sigma[0].astype(np.float64) / wl.sigma[0].sum() * pids.size
    big = exp >= 5
    obs = np.append(counts[big], counts[~big].sum())
    ex = np.append(exp[big], exp[~big].sum())
    assert st.chisquare(obs, ex).pvalue > 1e-4


def test_meta_sample_point_mass_and_zeros():
    P = 7
    s = np.zeros(P, np.float32)
    s[4] = 3.0
    assert np.all(oracle.meta_sample(s, P, 500, 3, 11) == 4)
    s = np.array([0, 1, 0, 1, 0, 0, 1], np.float32)
    pids = oracle.meta_sample(s, P, 3000, 2, 12)
    assert set(np.unique(pids)) == {1, 3, 6}
    # one distribution per seat
    s2 = np.zeros((2, P), np.float32)
    s2[0, 2] = 1
    s2[1, 5] = 1
    pids = oracle.meta_sample(s2, P, 100, 2, 13)
    assert np.all(pids[:, 0] == 2) and np.all(pids[:, 1] == 5)
    for bad in ([-1, 2], [0, 0], [np.nan, 1], [np.inf, 1]):
        with pytest.raises(ValueError):
            oracle.meta_sample(np.array(bad, np.float32), 2, 4, 1, 1)


def test_meta_sample_shard_invariant():
    wl = W.make(3)
    a = oracle.meta_sample(wl.sigma, wl.P, 1000, 2, wl.seed)
    b = np.concatenate([oracle.meta_sample(wl.sigma, wl.P, 400, 2, wl.seed, 0),
                        oracle.meta_sample(wl.sigma, wl.P, 600, 2, wl.seed, 400)])
    assert np.array_equal(a, b)


# -------------------------------------------------------------------- policies

def _torch_mlp_f32(Ws, bs, p, x):
    """fp64 torch reference of an fp32 MLP: linear layers with bias, ReLU on
    the hidden ones."""
    h = torch.from_numpy(np.asarray(x, np.float64))
    L = len(Ws)
    for l in range(L):
        b = None if bs is None else torch.from_numpy(bs[l][p].astype(np.float64))
        h = torch.nn.functional.linear(h, torch.from_numpy(Ws[l][p].astype(np.float64)), b)
        if l + 1 < L:
            h = torch.relu(h)
    return h.numpy()


def _random_biases(wl, seed, scale=0.3):
    """Distinct nonzero fp32 biases for every policy and layer (the generated
    populations have zero biases)."""
    rng = np.random.default_rng([2106, 7551, 90, seed])
    wl.biases = [rng.normal(0.0, scale, b.shape).astype(np.float32) for b in wl.biases]
    return wl


def test_mlp_f32_matches_torch():
    wl = W.make(2, P=4, per_pair=1)
    rng = np.random.default_rng(7)
    for p in range(4):
        x = rng.standard_normal(24)
        got = oracle.policy_logits(wl, p, x)
        ref = _torch_mlp_f32(wl.weights, None, p, x)
        assert np.allclose(got, ref, rtol=1e-6, atol=1e-6)


def test_mlp_f32_biases_match_torch():
    """fp32 MLP with distinct nonzero biases per policy and layer against torch
    fp64 linear(x, W, b): the bias enters each unit before its ReLU, from the
    row of the policy that runs (another policy's biases give other logits)."""
    wl = _random_biases(W.make(2, P=4, per_pair=1), 1)
    rng = np.random.default_rng(17)
    for p in range(4):
        for _ in range(4):
            x = rng.standard_normal(24)
            got = oracle.policy_logits(wl, p, x)
            ref = _torch_mlp_f32(wl.weights, wl.biases, p, x)
            assert np.allclose(got, ref, rtol=1e-6, atol=1e-6), p
            other = _torch_mlp_f32(wl.weights, [np.roll(b, 1, axis=0) for b in wl.biases], p, x)
            assert not np.allclose(got, other, rtol=1e-6, atol=1e-6)


def test_bf16_relu_is_relu_of_the_rounded_value():
    """ReLU of a hidden unit: bf16(max(x, 0)) (torch) for every non-NaN x,
    including -0 (-> +0), tiny negatives, values that round up to a power of
    two and infinities; a NaN of either sign stays NaN (torch.relu keeps NaN)."""
    xs = [0.0, -0.0, 1e-40, -1e-40, 1.0, -1.0, 3.0e38, -3.0e38, np.inf, -np.inf,
          1.00390625, 1.0039062500001, -2.9e-39, 65504.0, -7.5]
    rng = np.random.default_rng(3)
    xs += list(rng.standard_normal(2000).astype(np.float32) * 10.0 ** rng.integers(-30, 30, 2000))
    t = torch.tensor(np.array(xs, np.float32))
    ref = torch.relu(t).to(torch.bfloat16).float().numpy()
    ref = np.where(ref == 0, np.float32(0), ref)     # max(-0, 0) is taken as +0
    got = np.array([oracle.bf16_relu(x) for x in xs], np.float32)
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))
    for bits in (0x7FC01234, 0xFFC01234, 0x7F800001, 0xFF800001):
        nan = np.frombuffer(np.uint32(bits).tobytes(), np.float32)[0]
        assert np.isnan(torch.relu(torch.tensor([nan])).item())
        assert np.isnan(oracle.bf16_relu(nan))


def _torch_mlp_bf16(wl, p, x):
    """torch emulation of a bf16 policy: bf16 input, weights and hidden
    activations; exact products summed in fp64 and rounded to the fp32
    accumulator; the fp32 bias added in fp32 to that accumulator, before the
    hidden ReLU; logits fp32."""
    bf = lambda t: t.to(torch.bfloat16).to(torch.float64)
    h = bf(torch.from_numpy(np.asarray(x, np.float64)).float())
    for l in range(3):
        w = bf(torch.from_numpy(wl.weights[l][p]))
        acc = torch.nn.functional.linear(h, w).float()
        if wl.biases is not None:
            acc = acc + torch.from_numpy(wl.biases[l][p])
        h = bf(torch.relu(acc)) if l < 2 else acc.double()
    return h.numpy()


def test_mlp_bf16_matches_torch_emulation():
    """bf16 policy: bf16 input and hidden activations, exact products, fp32
    accumulator; emulated with torch's bf16 conversion and fp64 linear."""
    wl = W.make(3, P=3, n_envs=1)
    rng = np.random.default_rng(8)
    for p in range(3):
        x = rng.standard_normal(75)
        got = oracle.policy_logits(wl, p, x)
        assert np.allclose(got, _torch_mlp_bf16(wl, p, x), rtol=1e-5, atol=1e-5)


def test_mlp_bf16_biases_match_torch_emulation():
    """bf16 policy with distinct nonzero fp32 biases per policy and layer: the
    bias is added in fp32 after the layer sum is rounded to fp32 and before
    the ReLU and bf16 rounding of the hidden units (the torch emulation
    follows that order); another policy's biases give other logits."""
    wl = _random_biases(W.make(3, P=3, n_envs=1), 2)
    rng = np.random.default_rng(18)
    for p in range(3):
        for _ in range(4):
            x = rng.standard_normal(75)
            got = oracle.policy_logits(wl, p, x)
            assert np.allclose(got, _torch_mlp_bf16(wl, p, x), rtol=1e-5, atol=1e-5), p
            swapped = W.Workload(**{**wl.__dict__,
                                    "biases": [np.roll(b, 1, axis=0) for b in wl.biases]})
            assert not np.allclose(got, _torch_mlp_bf16(swapped, p, x), rtol=1e-5, atol=1e-5)


def _tiny_bf16(dims, Ws, bs):
    wl = W.make(3, P=1, n_envs=1)
    wl.dims = list(dims)
    wl.n_actions = dims[-1]
    wl.weights = [np.asarray(w, np.float32)[None] for w in Ws]
    wl.biases = [np.asarray(b, np.float32)[None] for b in bs]
    return wl


def test_mlp_bf16_bias_order_hand_values():
    """Hand-computed bf16 policies that fix where the bias enters.
    (a) Output unit with inputs h = [1, 2^-30] (exact in bf16), weights [1, 1]
    and bias 2^-24: the sum 1 + 2^-30 rounds to the fp32 accumulator 1, and
    1 + 2^-24 is a tie that rounds to even, so the logit is exactly 1.0; adding
    the bias before the fp32 rounding would give 1 + 2^-23.
    (b) Hidden unit with pre-activation -1 and bias 0.5: ReLU(-0.5) = 0, so the
    logit is 0; a bias added after the ReLU would give 0.5."""
    eye = np.eye(2)
    wl = _tiny_bf16([2, 2, 2, 1], [eye, eye, [[1.0, 1.0]]],
                    [[0, 0], [0, 0], [2.0 ** -24]])
    got = oracle.policy_logits(wl, 0, np.array([1.0, 2.0 ** -30]))
    assert got[0] == np.float32(1.0), got[0]
    wl = _tiny_bf16([2, 2, 2, 1], [[[-1.0, 0.0], [0.0, 0.0]], eye, [[1.0, 0.0]]],
                    [[0.5, 0.0], [0, 0], [0.0]])
    got = oracle.policy_logits(wl, 0, np.array([1.0, 0.0]))
    assert got[0] == np.float32(0.0), got[0]


def test_mlp_hidden_nan_reaches_the_logits():
    """A NaN weight (either sign) in a hidden layer of a policy makes all of its
    logits NaN in both policy kinds, so the rollout stops on it; the other
    policies are unaffected."""
    for c, n_in in ((2, 24), (3, 75)):
        for layer in (0, 1):
            for bits in (0x7FC00000, 0xFFC00000):
                wl = W.make(c, P=2, per_pair=1) if c == 2 else W.make(c, P=2, n_envs=1)
                wl.weights = [w.copy() for w in wl.weights]
                wl.weights[layer][1, 3, 5] = np.frombuffer(np.uint32(bits).tobytes(),
                                                           np.float32)[0]
                x = np.random.default_rng(c).standard_normal(n_in)
                assert np.isnan(oracle.policy_logits(wl, 1, x)).all(), (c, layer, hex(bits))
                assert np.isfinite(oracle.policy_logits(wl, 0, x)).all()


# ---------------------------------------------------------- matrix game (C1)

def test_matrix_game_closed_form():
    """One-step matrix game: the payoff of (pi_i, pi_j) is pi_i^T A pi_j with
    pi = softmax(logits); the Monte-Carlo table over 1024 episodes per pair is
    within 4 standard errors of it, and the closed form is antisymmetric."""
    wl = W.make(1)
    n = wl.n_envs
    r = oracle.rollout(wl, np.arange(n), wl.pairs)
    mean, cnt, s, s2 = oracle.payoff(r["returns"], wl.pairs, wl.team, wl.P)
    assert np.all(cnt == 1024)
    pis = [softmax(wl.tab_logits[p]) for p in range(wl.P)]
    A = wl.A.astype(np.float64)
    exact = np.array([[pis[i] @ A @ pis[j] for j in range(wl.P)] for i in range(wl.P)])
    var = s2 / cnt - mean**2
    se = np.sqrt(var / cnt)
    assert np.all(np.abs(mean - exact) <= 4 * se + 1e-12)
    assert np.allclose(exact, -exact.T)
    assert np.allclose(np.diag(exact), 0)
    # zero-sum per env, bitwise
    assert np.array_equal(r["returns"][:, 1], -r["returns"][:, 0])


# --------------------------------------------------------- iterated game (C2)

def test_iter_obs_encoding():
    """Lag 1..4, most recent first: [onehot(own), onehot(other)]; zeros before
    the start."""
    o = oracle.obs_iter([2 * 3 + 1, 0 * 3 + 2, -1, -1], 0)
    want = np.zeros(24)
    want[0 + 2] = 1; want[3 + 1] = 1      # lag 1: own 2, other 1
    want[6 + 0] = 1; want[9 + 2] = 1      # lag 2: own 0, other 2
    assert np.array_equal(o, want)
    o = oracle.obs_iter([2 * 3 + 1, 0 * 3 + 2, -1, -1], 1)
    want = np.zeros(24)
    want[0 + 1] = 1; want[3 + 2] = 1
    want[6 + 2] = 1; want[9 + 0] = 1
    assert np.array_equal(o, want)
    assert not oracle.obs_iter([-1] * 4, 0).any()


def test_iter_brute_force():
    """E[G_0] over every joint-action sequence of a horizon-3 episode (9^3
    paths, probabilities from softmax of the oracle's logits) agrees with the
    sampled mean of 4096 episodes within 4 standard errors."""
    H = 3
    wl = W.make(2, P=3, per_pair=1, horizon=H)
    i, j = 1, 2
    A = wl.A.astype(np.float64)

    def rec(hist, t):
        if t == H:
            return 0.0
        p0 = softmax(oracle.policy_logits(wl, i, oracle.obs_iter(hist, 0)))
        p1 = softmax(oracle.policy_logits(wl, j, oracle.obs_iter(hist, 1)))
        tot = 0.0
        for a0 in range(3):
            for a1 in range(3):
                nh = [a0 * 3 + a1] + hist[:3]
                tot += p0[a0] * p1[a1] * (A[a0, a1] + rec(nh, t + 1))
        return tot

    exact = rec([-1, -1, -1, -1], 0)
    n = 4096
    pids = np.tile(np.array([[i, j]], np.int32), (n, 1))
    r = oracle.rollout(wl, np.arange(n), pids)
    g = r["returns"][:, 0].astype(np.float64)
    assert abs(g.mean() - exact) <= 4 * g.std() / math.sqrt(n)
    assert np.array_equal(r["returns"][:, 1], -r["returns"][:, 0])


def test_iter_antisymmetric_table():
    """The iterated game is symmetric under a seat swap (egocentric
    observations, antisymmetric A), so M_ij = -M_ji within Monte-Carlo error."""
    wl = W.make(2, P=4, per_pair=512, horizon=8)
    r = oracle.rollout(wl, np.arange(wl.n_envs), wl.pairs)
    mean, cnt, s, s2 = oracle.payoff(r["returns"], wl.pairs, wl.team, wl.P)
    var = s2 / cnt - mean**2
    se2 = var / cnt
    dev = np.abs(mean + mean.T)
    assert np.all(dev <= 4 * np.sqrt(se2 + se2.T) + 1e-9)


# ---------------------------------------------------------------- pursuit (C3)

def test_pursuit_moves_and_capture():
    cell = lambda x, y: 8 * y + x
    # wrap-around moves
    assert oracle.pursuit_step(cell(0, 0), cell(4, 4), 1, 0)[0] == cell(0, 7)
    assert oracle.pursuit_step(cell(0, 0), cell(4, 4), 3, 0)[0] == cell(7, 0)
    assert oracle.pursuit_step(cell(7, 7), cell(4, 4), 2, 0)[0] == cell(7, 0)
    assert oracle.pursuit_step(cell(7, 7), cell(4, 4), 4, 0)[0] == cell(0, 7)
    # same cell after the move
    assert oracle.pursuit_step(cell(1, 0), cell(2, 0), 4, 0)[2]
    # the two swap cells
    p, e, cap = oracle.pursuit_step(cell(1, 0), cell(2, 0), 4, 3)
    assert cap and p == cell(2, 0) and e == cell(1, 0)
    # no contact
    assert not oracle.pursuit_step(cell(0, 0), cell(2, 2), 0, 0)[2]
    assert not oracle.pursuit_step(cell(0, 0), cell(2, 0), 4, 4)[2]


def test_pursuit_obs_index_map():
    """Egocentric 5x5 window, index ((dy+2)*5 + (dx+2))*3 + channel; channels:
    pursuer, evader, self (centre)."""
    cell = lambda x, y: 8 * y + x
    o = oracle.obs_pursuit(cell(0, 0), cell(1, 0), 0)
    assert o.sum() == 3 and o[36] == 1 and o[38] == 1 and o[40] == 1
    o = oracle.obs_pursuit(cell(0, 0), cell(1, 0), 1)
    assert o.sum() == 3 and o[37] == 1 and o[38] == 1 and o[33] == 1
    o = oracle.obs_pursuit(cell(0, 0), cell(7, 7), 0)      # wraps to dx=dy=-1
    assert o[((1 * 5) + 1) * 3 + 1] == 1
    o = oracle.obs_pursuit(cell(0, 0), cell(4, 4), 0)      # out of view
    assert o.sum() == 2


def test_pursuit_reset_distinct_uniform():
    wl = W.make(3)
    pcs, ecs = zip(*[oracle.pursuit_reset(wl.seed, g) for g in range(6400)])
    pcs, ecs = np.array(pcs), np.array(ecs)
    assert np.all(pcs != ecs) and pcs.max() < 64 and ecs.max() < 64
    assert st.chisquare(np.bincount(pcs, minlength=64)).pvalue > 1e-4
    assert st.chisquare(np.bincount(ecs, minlength=64)).pvalue > 1e-4


@pytest.mark.parametrize("grid", [5, 8, 11, 16])
def test_pursuit_reset_any_grid(grid):
    """The reset cells on a G x G torus against lanes 0 and 1 of the reset block
    drawn with numpy's Philox (independent of the oracle's generator): pursuer
    floor(lane0 G^2 / 2^32), which is lane0 >> 26 for G = 8; evader pursuer + 1
    + floor(lane1 (G^2 - 1) / 2^32) mod G^2."""
    seed, cells = W.make(3).seed, grid * grid
    for g in range(1, 400):
        # the block of counter (g, 0, 1 << 32, 0) is numpy's first draw from (g - 1, ...)
        gen = np.random.Philox(key=np.array([seed, 0], np.uint64),
                               counter=np.array([g - 1, 0, 1 << 32, 0], np.uint64))
        w0 = int(gen.random_raw(4)[0])
        lane0, lane1 = w0 & 0xFFFFFFFF, w0 >> 32
        pc, ec = oracle.pursuit_reset(seed, g, grid)
        assert pc == (lane0 * cells) >> 32
        if grid == 8:
            assert pc == lane0 >> 26
        assert ec == (pc + 1 + ((lane1 * (cells - 1)) >> 32)) % cells
        assert 0 <= pc < cells and 0 <= ec < cells and pc != ec


def test_pursuit_one_step_brute_force():
    """E[G_0] of a horizon-1 episode: average over the 64*63 distinct starts of
    sum_{a0,a1} pi_i(a0) pi_j(a1) [capture]; vs 16384 sampled episodes."""
    wl = W.make(3, P=2, n_envs=8192, horizon=1)
    i, j = 0, 1
    tot = 0.0
    for p in range(64):
        for e in range(64):
            if p == e:
                continue
            p0 = softmax(oracle.policy_logits(wl, i, oracle.obs_pursuit(p, e, 0)))
            p1 = softmax(oracle.policy_logits(wl, j, oracle.obs_pursuit(p, e, 1)))
            for a0 in range(5):
                for a1 in range(5):
                    if oracle.pursuit_step(p, e, a0, a1)[2]:
                        tot += p0[a0] * p1[a1]
    exact = tot / (64 * 63)
    n = wl.n_envs
    r = oracle.rollout(wl, np.arange(n), np.tile(np.array([[i, j]], np.int32), (n, 1)))
    g = r["returns"][:, 0].astype(np.float64)
    assert abs(g.mean() - exact) <= 4 * g.std() / math.sqrt(n)


def test_pursuit_termination_freezes():
    wl = W.make(3, P=2, n_envs=128, horizon=100)
    pids = np.tile(np.array([[0, 1]], np.int32), (128, 1))
    r = oracle.rollout(wl, np.arange(128), pids, want_actions=True, want_states=True)
    g = r["returns"]
    assert set(np.unique(g[:, 0])) <= {0.0, 1.0}
    assert np.array_equal(g[:, 1], -g[:, 0])
    done = r["states"][:, :, 2]
    # once done, stays done; no actions afterwards
    assert np.all(np.diff(done.astype(np.int8), axis=0) >= 0)
    assert np.all(r["actions"][done == 1] == 255)
    live_envs = (done == 0).sum()
    assert r["live_frames"] == 2 * live_envs
    captured = done[-1] == 1
    # a capture at the last step is not visible in the pre-step snapshot
    assert np.all(g[captured, 0] == 1.0)


# ---------------------------------------------------------------- feature (C4)

def test_feature_step_vs_numpy():
    """s' = tanh(W s + B[a0] + C[a1]) and r = u . s', against fp64 numpy."""
    wl = W.make(4, P=1, per_pair=1)
    s0 = oracle.feature_reset(wl.seed, 5, wl.d)
    assert np.all(np.abs(s0) < 1) and abs(s0.mean()) < 0.1
    k = (s0.astype(np.float64) * 2**23)
    assert np.all(k == np.round(k)) and np.all(k % 2 == 1)
    for a0, a1 in [(0, 0), (3, 17), (17, 5)]:
        s1, r = oracle.feature_step(wl, s0, [a0, a1])
        pre = wl.W.astype(np.float64) @ s0 + wl.emb[0, a0] + wl.emb[1, a1]
        ref = np.tanh(pre)
        assert np.abs(s1 - ref).max() <= 2e-6
        assert abs(r - wl.u.astype(np.float64) @ ref) <= 1e-5


def test_feature_one_step_brute_force():
    """Shared start s0: E[G_0] = sum_{a0,a1} pi_i(a0|s0) pi_j(a1|s0) u.tanh(W s0 +
    B[a0] + C[a1]) (324 terms, fp64) vs 1024 sampled episodes."""
    wl = W.make(4, P=2, per_pair=1, horizon=1)
    wl.init_mode = W.INIT_SHARED
    s0 = oracle.feature_reset(wl.seed, 0, wl.d)
    i, j = 0, 1
    pi = softmax(oracle.policy_logits(wl, i, s0))
    pj = softmax(oracle.policy_logits(wl, j, s0))
    base = wl.W.astype(np.float64) @ s0
    pre = base[None, None, :] + wl.emb[0][:, None, :] + wl.emb[1][None, :, :]
    rew = np.tanh(pre) @ wl.u.astype(np.float64)
    exact = float(pi @ rew @ pj)
    n = 1024
    r = oracle.rollout(wl, np.arange(n), np.tile(np.array([[i, j]], np.int32), (n, 1)))
    g = r["returns"][:, 0].astype(np.float64)
    assert abs(g.mean() - exact) <= 4 * g.std() / math.sqrt(n)
    assert np.array_equal(r["returns"][:, 1], -r["returns"][:, 0])


# ----------------------------------------------------------- team game (C5)

def test_team_2v2_brute_force_and_reduction():
    """2v2 feature game, shared start, horizon 1: E[G_A] over all 18^4 joint
    actions vs 2048 sampled episodes; the payoff reduction puts each env into
    the 4 (row seat, column seat) cells."""
    wl = W.team_variant(4, P=6, n_envs=2048, horizon=1)
    wl.init_mode = W.INIT_SHARED
    s0 = oracle.feature_reset(wl.seed, 0, wl.d)
    pids_one = np.array([0, 3, 5, 1], np.int32)
    probs = [softmax(oracle.policy_logits(wl, int(p), s0)) for p in pids_one]
    base = wl.W.astype(np.float64) @ s0
    E = wl.emb.astype(np.float64)
    u = wl.u.astype(np.float64)
    exact = 0.0
    for a0 in range(18):
        pre = (base + E[0, a0])[None, None, None, :] + E[1][:, None, None, :] + \
            E[2][None, :, None, :] + E[3][None, None, :, :]
        rew = np.tanh(pre) @ u
        w = probs[0][a0] * probs[1][:, None, None] * probs[2][None, :, None] * \
            probs[3][None, None, :]
        exact += float((w * rew).sum())
    n = wl.n_envs
    pids = np.tile(pids_one[None], (n, 1))
    r = oracle.rollout(wl, np.arange(n), pids)
    g = r["returns"][:, 0].astype(np.float64)
    assert abs(g.mean() - exact) <= 4 * g.std() / math.sqrt(n)
    R = r["returns"]
    assert np.array_equal(R[:, 1], R[:, 0]) and np.array_equal(R[:, 2], -R[:, 0])
    mean, cnt, _, _ = oracle.payoff(R, pids, wl.team, wl.P)
    assert cnt.sum() == 4 * n
    for a in (0, 1):
        for b in (2, 3):
            assert cnt[pids_one[a], pids_one[b]] == n
            assert np.isclose(mean[pids_one[a], pids_one[b]], g.mean())


def test_team_4v4_step_vs_numpy():
    """The 4v4 game's step (R13, R15): s' = tanh(W s + sum over the eight
    seats of emb[k][a_k]) and r = u . s', against fp64 numpy, for action
    vectors that differ in every seat (a dropped or repeated seat, a seat
    read from another seat's table or an action from another seat moves s'
    far beyond the tolerance)."""
    wl = W.make(5, P=2, n_envs=4, horizon=1)
    assert wl.n_agents == 8 and wl.emb.shape == (8, 18, wl.d)
    s0 = oracle.feature_reset(wl.seed, 3, wl.d)
    rng = np.random.default_rng(12)
    for acts in ([0] * 8, list(range(8)), list(range(17, 9, -1)),
                 rng.integers(0, 18, 8).tolist(), rng.integers(0, 18, 8).tolist()):
        s1, r = oracle.feature_step(wl, s0, acts)
        pre = wl.W.astype(np.float64) @ s0
        for k, a in enumerate(acts):
            pre = pre + wl.emb[k, a]
        ref = np.tanh(pre)
        assert np.abs(s1 - ref).max() <= 2e-6, acts
        assert abs(r - wl.u.astype(np.float64) @ ref) <= 1e-5
        # each seat's embedding matters: swapping two seats' different actions
        # changes the state
        if acts[0] != acts[7]:
            sw = list(acts)
            sw[0], sw[7] = sw[7], sw[0]
            s_sw, _ = oracle.feature_step(wl, s0, sw)
            assert np.abs(s_sw - s1).max() > 1e-3


def test_team_4v4_reduction_plain_loops():
    """The 4v4 reduction (R16): every (team +1 seat, team -1 seat) pair of an
    env adds that env's row-side return to cell (pid_a, pid_b), 16 incidences
    per env, against plain loops."""
    wl = W.make(5, P=7, n_envs=4, horizon=1)
    team = wl.team
    assert list(team) == [1, 1, 1, 1, -1, -1, -1, -1]
    rng = np.random.default_rng(13)
    n, P = 200, 7
    R = rng.standard_normal((n, 8)).astype(np.float32)
    R[:, 1:4] = R[:, :1]          # a side's seats share the side's return
    R[:, 4:] = -R[:, :1]
    pids = rng.integers(0, P, size=(n, 8))
    mean, cnt, s, _ = oracle.payoff(R, pids, team, P)
    S = np.zeros((P, P)); N = np.zeros((P, P), np.int64)
    for e in range(n):
        for a in range(4):
            for b in range(4, 8):
                S[pids[e, a], pids[e, b]] += float(R[e, a])
                N[pids[e, a], pids[e, b]] += 1
    assert cnt.sum() == 16 * n
    assert np.array_equal(cnt, N) and np.allclose(s, S)


# --------------------------------------------------------------------- payoff

def test_payoff_table_plain_loops():
    rng = np.random.default_rng(9)
    n, P = 300, 5
    team = np.array([1, 1, -1, -1, -1], np.int8)
    R = rng.standard_normal((n, 5)).astype(np.float32)
    pids = rng.integers(0, P, size=(n, 5))
    mean, cnt, s, s2 = oracle.payoff(R, pids, team, P)
    S = np.zeros((P, P)); N = np.zeros((P, P), np.int64)
    for e in range(n):
        for a in range(5):
            for b in range(5):
                if team[a] > 0 and team[b] < 0:
                    S[pids[e, a], pids[e, b]] += float(R[e, a])
                    N[pids[e, a], pids[e, b]] += 1
    assert np.array_equal(cnt, N)
    assert np.allclose(s, S)
    with np.errstate(invalid="ignore"):
        assert np.array_equal(np.isnan(mean), N == 0)


# -------------------------------------------------------------- determinism

@pytest.mark.parametrize("c", [2, 3, 5])
def test_oracle_shard_invariant(c):
    """Results depend only on (seed, global env index): two half batches with
    env_offset reproduce one full batch bit for bit."""
    if c == 2:
        wl = W.make(2, P=2, per_pair=4, horizon=6)
    elif c == 3:
        wl = W.make(3, P=4, n_envs=16, horizon=20)
    else:
        wl = W.make(5, P=4, n_envs=4, horizon=2)
        wl.dims = [256, 512, 512, 18]
    n = wl.n_envs if c != 2 else wl.n_envs
    pids = wl.pairs if wl.pairs is not None else oracle.meta_sample(
        wl.sigma, wl.P, n, wl.n_agents, wl.seed)
    full = oracle.rollout(wl, np.arange(n), pids)["returns"]
    h = n // 2
    a = oracle.rollout(wl, np.arange(h), pids[:h])["returns"]
    b = oracle.rollout(wl, np.arange(n - h), pids[h:], env_offset=h)["returns"]
    assert np.array_equal(full, np.concatenate([a, b]))


# ------------------------------------------------------------ meta-solver (FP)
def test_solve_fp_hand_trace():
    """Three iterations on M = [[1, 2], [3, 0]] worked by hand: (i, j) =
    (0, 0), (1, 0), (1, 1); v = [4, 6], w = [7, 2] afterwards."""
    cx, cy, gap = oracle.solve_fp(np.array([[1.0, 2.0], [3.0, 0.0]]), 3)
    assert cx.tolist() == [1, 2] and cy.tolist() == [2, 1]
    assert gap == (6.0 - 2.0) / 3.0


def test_solve_fp_zero_game_and_dominance():
    """All-zero game: every tie goes to index 0.  Strictly dominant row 1 and
    column 1 of [[3, 1], [4, 2]]: after the first iteration both sides play 1,
    and the gap is 3/T in closed form."""
    cx, cy, gap = oracle.solve_fp(np.zeros((5, 5)), 40)
    assert cx.tolist() == [40, 0, 0, 0, 0] and cy.tolist() == [40, 0, 0, 0, 0] and gap == 0.0
    T = 500
    cx, cy, gap = oracle.solve_fp(np.array([[3.0, 1.0], [4.0, 2.0]]), T)
    assert cx.tolist() == [1, T - 1] and cy.tolist() == [1, T - 1]
    assert abs(gap - 3.0 / T) < 1e-15


@pytest.mark.parametrize("M,x0,y0,value", [
    # 2x2 without a saddle point: x* = (d-c)/D, y* = (d-b)/D, value (ad-bc)/D,
    # D = a-b-c+d
    ([[1.0, 2.0], [3.0, 0.0]], 0.75, 0.5, 1.5),
    ([[2.0, -1.0], [-1.0, 1.0]], 0.4, 0.4, 0.2),
])
def test_solve_fp_converges_to_the_2x2_equilibrium(M, x0, y0, value):
    T = 20000
    M = np.array(M)
    cx, cy, gap = oracle.solve_fp(M, T)
    assert abs(cx[0] / T - x0) < 0.02 and abs(cy[0] / T - y0) < 0.02
    # the averages' best-response values bracket the game value
    lo, hi = (cx @ M).min() / T, (M @ cy).max() / T
    assert lo <= value + 1e-12 and value <= hi + 1e-12 and gap == pytest.approx(hi - lo, abs=1e-12)
    assert gap < 0.02


def test_solve_fp_rock_paper_scissors_and_gap_definition():
    """Rock-paper-scissors: the averages approach uniform play, and the gap is
    max(M cy) - min(cx M), recomputed from the counts."""
    M = np.array([[0.0, -1.0, 1.0], [1.0, 0.0, -1.0], [-1.0, 1.0, 0.0]])
    T = 30000
    cx, cy, gap = oracle.solve_fp(M, T)
    assert np.abs(cx / T - 1 / 3).max() < 0.03 and np.abs(cy / T - 1 / 3).max() < 0.03
    assert gap == pytest.approx(((M @ cy).max() - (cx @ M).min()) / T, abs=1e-12)
    assert 0.0 <= gap < 0.05
    rng = np.random.default_rng(5)
    R = rng.normal(size=(17, 17))
    cx, cy, gap = oracle.solve_fp(R, 777)
    assert cx.sum() == 777 and cy.sum() == 777
    assert gap == pytest.approx(((R @ cy).max() - (cx @ R).min()) / 777, abs=1e-12)


# ---------------------------------------------------- incremental expansion

@pytest.mark.parametrize("P,f,per_pair", [(1, 0, 3), (4, 0, 5), (5, 3, 2), (7, 6, 1),
                                           (9, 1, 2)])
def test_expansion_pairs_cover_exactly_the_new_cells(P, f, per_pair):
    """The expansion batch plays every cell of the grown grid that is outside
    the old f x f block exactly per_pair times and no old cell; with no old
    block it is the blocked all-pairs assignment (an independent generator)."""
    team = np.array([1, -1], np.int8)
    pairs = oracle.expansion_pairs(P, f, per_pair, team)
    assert pairs.shape == ((P * P - f * f) * per_pair, 2)
    grid = np.zeros((P, P), np.int64)
    np.add.at(grid, (pairs[:, 0], pairs[:, 1]), 1)
    want = np.full((P, P), per_pair)
    want[:f, :f] = 0
    assert np.array_equal(grid, want)
    # row-major order of the cells, per_pair consecutive envs each
    cells = pairs[::per_pair]
    key = cells[:, 0] * P + cells[:, 1]
    assert np.all(np.diff(key) > 0)
    assert np.array_equal(pairs, np.repeat(cells, per_pair, axis=0))
    if f == 0:
        assert np.array_equal(pairs, W.blocked_pairs(P, per_pair))


def test_expansion_merge_keeps_old_cells():
    """A table filled with the P0 blocked pairs, grown, then filled with the
    expansion batch: the old block keeps its sums and counts (the batch never
    touches it) and every new cell gets the team game's seat pairs per env."""
    rng = np.random.default_rng(4)
    P0, P, per_pair = 3, 5, 4
    team = np.array([1, 1, -1, -1, -1], np.int8)
    p0 = W.blocked_pairs(P0, per_pair)
    p0 = np.stack([p0[:, 0], p0[:, 0], p0[:, 1], p0[:, 1], p0[:, 1]], 1)
    r0 = rng.standard_normal((len(p0), 5)).astype(np.float32)
    p1 = oracle.expansion_pairs(P, P0, per_pair, team)
    r1 = rng.standard_normal((len(p1), 5)).astype(np.float32)
    m0, c0, s0, _ = oracle.payoff(r0, p0, team, P)
    m1, c1, s1, _ = oracle.payoff(np.concatenate([r0, r1]), np.concatenate([p0, p1]), team, P)
    assert np.array_equal(c1[:P0, :P0], c0[:P0, :P0])
    assert np.array_equal(s1[:P0, :P0], s0[:P0, :P0])
    new = np.ones((P, P), bool)
    new[:P0, :P0] = False
    assert (c1[new] == per_pair * 2 * 3).all()
    assert (c0[new] == 0).all()


# ----------------------------------------------- aggregate / convergence

def test_aggregate_matches_bilinear_forms():
    """nash = x^T M y and the best-response payoffs (M y)[i], -(x^T M)[j],
    against numpy's products (another summation order: 1e-13 relative)."""
    rng = np.random.default_rng(12)
    for P in (1, 3, 20, 200):
        M = rng.normal(size=(P, P))
        sig = (rng.random((2, P)) * 10).astype(np.float32)
        sig[0, 0] += 1
        sig[1, -1] += 1
        x = sig[0].astype(np.float64) / sig[0].astype(np.float64).sum()
        y = sig[1].astype(np.float64) / sig[1].astype(np.float64).sum()
        for br in (0, P - 1):
            nr, nc, wr, wc, imp = oracle.aggregate(M, sig, br, P - 1 - br)
            tol = 1e-13 * max(1.0, np.abs(M).max())
            assert abs(nr - x @ M @ y) <= tol and nc == -nr
            assert abs(wr - (M @ y)[br]) <= tol
            assert abs(wc + (x @ M)[P - 1 - br]) <= tol
            assert imp == max(wr - nr, wc - nc)


def test_aggregate_equilibria_and_a_hand_case():
    # rock-paper-scissors at the uniform equilibrium: every payoff is 0
    R = np.array([[0, -1, 1], [1, 0, -1], [-1, 1, 0]], np.float64)
    for br in range(3):
        out = oracle.aggregate(R, np.ones((2, 3), np.float32), br, br)
        assert out[0] == 0.0 and out[2] == 0.0 and out[3] == 0.0 and out[4] == 0.0
    # a 2x2 game with the mixed equilibrium x = (3/4, 1/4), y = (1/2, 1/2),
    # value 1/2: no pure deviation gains
    G = np.array([[1.0, 0.0], [-1.0, 2.0]])
    out = oracle.aggregate(G, np.array([[3, 1], [1, 1]], np.float32), 1, 0)
    assert abs(out[0] - 0.5) < 1e-15 and abs(out[4]) < 1e-15
    # pure profile (0, 0) of [[1, 0], [0, 2]]: nash 1; the row side's policy 1
    # earns 0 (gain -1), the column side's policy 1 pays 0 instead of 1 (gain 1)
    H = np.array([[1.0, 0.0], [0.0, 2.0]])
    nr, nc, wr, wc, imp = oracle.aggregate(H, np.array([[1, 0], [1, 0]], np.float32), 1, 1)
    assert (nr, nc, wr, wc, imp) == (1.0, -1.0, 0.0, 0.0, 1.0)
    # one side left out
    out = oracle.aggregate(H, np.array([[1, 0], [1, 0]], np.float32), -1, 1)
    assert np.isnan(out[2]) and out[4] == 1.0


# --------------------------------------------------------- per-step rewards

@pytest.mark.parametrize("c", [1, 2, 3])
def test_step_rewards_add_up_to_returns(c):
    """The per-step rewards the oracle reports for trajectory records: summed
    in step order (fp32) they are the returns bit for bit; the matrix games'
    are the payoff entries of the actions taken, zero-sum per step; pursuit's
    are +1 / -1 at the capture step only."""
    if c == 1:
        wl = W.make(1, per_pair=8)
    elif c == 2:
        wl = W.make(2, P=2, per_pair=4, horizon=7)
    else:
        wl = W.make(3, P=3, n_envs=1, horizon=40)
    pairs = wl.pairs if wl.pairs is not None else W.blocked_pairs(3, 6)
    n = len(pairs)
    o = oracle.rollout(wl, np.arange(n), pairs, want_actions=True, want_rewards=True)
    r = o["rewards"]
    acc = np.zeros((n, 2), np.float32)
    for t in range(r.shape[0]):
        acc = acc + r[t]
    assert np.array_equal(acc.view(np.uint32), o["returns"].view(np.uint32))
    assert np.array_equal(r[:, :, 1], -r[:, :, 0])
    a = o["actions"]
    if c in (1, 2):
        assert np.array_equal(r[:, :, 0], wl.A[a[:, :, 0], a[:, :, 1]])
    else:
        assert set(np.unique(r[:, :, 0])) <= {0.0, 1.0}
        caught = r[:, :, 0] == 1.0
        assert (caught.sum(axis=0) <= 1).all() and caught.any()
        t_c = np.argmax(caught, axis=0)
        for e in np.nonzero(caught.any(axis=0))[0]:
            assert (a[t_c[e] + 1:, e] == 255).all()


def test_payoff_matrix_is_the_means_with_empty_cells_zero():
    """The solver's game from a table: a filled cell keeps its mean, an empty
    one (NaN mean, count 0) becomes 0; built from the plain-loop table."""
    rng = np.random.default_rng(21)
    P = 4
    pids = np.array([[0, 1], [0, 1], [2, 3], [1, 0]])
    R = rng.standard_normal((4, 2)).astype(np.float32)
    mean, cnt, s, _ = oracle.payoff(R, pids, np.array([1, -1], np.int8), P)
    g = oracle.payoff_matrix(mean)
    assert g[0, 1] == (float(R[0, 0]) + float(R[1, 0])) / 2
    assert g[2, 3] == float(R[2, 0]) and g[1, 0] == float(R[3, 0])
    assert (g[cnt == 0] == 0.0).all() and not np.isnan(g).any()


def test_threaded_oracle_equals_single_thread():
    """The parity tests split the oracle's envs over threads: the merged
    result equals one single-threaded rollout of the same envs, element by
    element (returns, actions, logits, states, counters)."""
    wl = W.make(5, P=8, n_envs=24, horizon=6)
    pairs = oracle.meta_sample(wl.sigma, wl.P, wl.n_envs, wl.n_agents, wl.seed)
    idx = np.arange(3, 24)
    kw = dict(want_actions=True, want_logits=True, want_states=True, want_rewards=True)
    a = oracle.rollout(wl, idx, pairs[idx], **kw)
    b = oracle.rollout_threads(wl, idx, pairs[idx], threads=5, **kw)
    for k in ("returns", "actions", "logits", "states", "rewards"):
        assert np.array_equal(a[k], b[k]), k
    for k in ("near_ties", "flips", "fails", "live_frames"):
        assert a[k] == b[k], k
