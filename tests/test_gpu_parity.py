"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Reduced sizes that the oracle finishes in seconds but that still span several
policy tiles and a ragged tail; full-size sampled checks live in
test_gpu_fullsize.py.  Bars: integer/byte/index results and the environment
state bit for bit (given the same actions); logits within 1e-5 (fp32) /
1e-2 (bf16) relative to max(1, max|l|); actions equal except counted near
ties; payoff entries within 1e-3; counts exact.
"""
import numpy as np
import pytest

import oracle
import workloads as W
from gpu_helpers import check_parity, run_gpu, say

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2106_07551_amd as M
    M.lib()


# ------------------------------------------------------------ kernel pieces

def test_philox_device_matches_oracle():
    import paper_2106_07551_amd as M
    rng = np.random.default_rng(1)
    ctr = rng.integers(0, 2**64 - 1, size=(4096, 4), dtype=np.uint64)
    ctr[:3] = [[0, 0, 0, 0], [2**64 - 1] * 4, [5, 6, (2 << 32) | 3, 1]]
    key = (0x452821E638D01377, 0xBE5466CF34E90C6C)
    out = M.debug_philox(torch.from_numpy(ctr.view(np.int64)).cuda(), *key).cpu().numpy()
    out = out.view(np.uint64)
    for i in range(0, 4096, 37):
        assert np.array_equal(out[i], oracle.philox(ctr[i], key)), i


def test_tanh_ref_device_bitwise_sampled():
    """tanh_ref on the device equals the oracle's bit for bit on a strided
    sample of all 2^32 patterns plus every pattern of [0.25, 16) (both signs)."""
    import paper_2106_07551_amd as M
    chunks = [np.arange(0, 2**32, 251, dtype=np.uint64).astype(np.uint32)]
    lo = np.array([0.25], np.float32).view(np.uint32)[0]
    hi = np.array([16.0], np.float32).view(np.uint32)[0]
    dense = np.arange(lo, hi, dtype=np.uint32)
    chunks += [dense, dense | np.uint32(0x80000000)]
    for bits in chunks:
        x = bits.view(np.float32)
        y = M.debug_tanh_ref(torch.from_numpy(x.copy()).cuda()).cpu().numpy()
        ref = oracle.tanh_many(x)
        same = (y.view(np.uint32) == ref.view(np.uint32)) | (np.isnan(y) & np.isnan(ref))
        assert same.all(), hex(int(bits[np.argmin(same)]))


def test_tanh_ref_device_bitwise_exhaustive():
    """tanh_ref on the device equals the oracle's bit for bit over all 2^32 fp32
    bit patterns (NaNs compared as NaN), in chunks of 2^27."""
    import paper_2106_07551_amd as M
    chunk = 1 << 27
    x = torch.empty(chunk, dtype=torch.int32, device="cuda")
    base = torch.arange(chunk, dtype=torch.int32, device="cuda")
    for c in range(1 << 5):
        first = c * chunk
        x.copy_(base + (first - (1 << 32) if first >= (1 << 31) else first))
        y = M.debug_tanh_ref(x.view(torch.float32)).cpu().numpy()
        ref = oracle.tanh_range(first, chunk)
        same = (y.view(np.uint32) == ref.view(np.uint32)) | (np.isnan(y) & np.isnan(ref))
        assert same.all(), hex(first + int(np.argmin(same)))


def test_bf16_device_matches_oracle():
    """The device bf16 conversion (observations, weights, hidden activations)
    equals the oracle's round-to-nearest-even bit for bit: every low half-word
    under a set of high half-words (zeros, subnormals, normals, the largest
    finite values, infinities, NaNs; both signs) plus a strided sample of all
    patterns (NaNs compared as NaN)."""
    import paper_2106_07551_amd as M
    highs = sorted({(e << 7) | m for e in list(range(0, 6)) + list(range(118, 138)) +
                    list(range(250, 256)) for m in (0, 1, 0x3F, 0x40, 0x7E, 0x7F)})
    bits, ref = [], []
    for sign in (0, 0x8000):
        for h in highs:
            first = (sign | h) << 16
            bits.append(np.arange(1 << 16, dtype=np.uint32) + np.uint32(first))
            ref.append(oracle.bf16_range(first, 1 << 16))
    stride = np.arange(0, 2**32, 65521, dtype=np.uint64).astype(np.uint32)
    bits.append(stride)
    ref.append(np.array([oracle.bf16_bits(float(v)) for v in stride.view(np.float32)],
                        np.uint16))
    bits = np.concatenate(bits)
    ref = np.concatenate(ref)
    if bits.size % 2:
        bits, ref = bits[:-1], ref[:-1]
    x = bits.view(np.float32)
    y = M.debug_bf16(torch.from_numpy(x.copy()).cuda()).cpu().numpy().view(np.uint16)
    nan = np.isnan(x)
    ok = (y == ref) | (nan & ((y & 0x7F80) == 0x7F80) & ((y & 0x7F) != 0))
    assert ok.all(), hex(int(bits[np.argmin(ok)]))


@pytest.mark.parametrize("c", [3, 5])
def test_meta_sample_device_matches_oracle(c):
    import paper_2106_07551_amd as M
    wl = W.make(c)
    n = 3001
    for off in (0, 12345):
        g = M.meta_sample(wl.sigma, wl.P, n, wl.n_agents, wl.seed, env_offset=off)
        ref = oracle.meta_sample(wl.sigma, wl.P, n, wl.n_agents, wl.seed, off)
        assert np.array_equal(g.cpu().numpy(), ref)


def test_meta_sample_per_seat_rows_and_errors():
    import paper_2106_07551_amd as M
    P = 9
    s = np.random.default_rng(2).random((3, P)).astype(np.float32)
    s[1, :4] = 0
    g = M.meta_sample(s, P, 500, 3, 77).cpu().numpy()
    assert np.array_equal(g, oracle.meta_sample(s, P, 500, 3, 77))
    assert g[:, 1].min() >= 4
    for bad in (np.array([1, -1], np.float32), np.array([0, 0], np.float32),
                np.array([np.nan, 1], np.float32)):
        with pytest.raises(M.MalibError):
            M.meta_sample(bad, 2, 10, 1, 1)


# ------------------------------------------------------------ parity by workload

def test_parity_matrix_full():
    """One-step matrix game at its full size (16 pairs x 1024 envs)."""
    wl = W.make(1)
    g = run_gpu(wl, snaps=[0])
    check_parity(wl, g)


def test_parity_iter_ragged():
    """Iterated game, fp32 MLP: 4 policies x 50 envs per pair (400 rows per
    policy = 12 full 32-row tiles + a ragged one), horizon 32."""
    wl = W.make(2, P=4, per_pair=50)
    g = run_gpu(wl, snaps=[0, 1, 5, 31])
    check_parity(wl, g)


def test_parity_pursuit_ragged():
    """Pursuit, bf16 MLP 75-256-256-5, full population of 32, 300 envs with
    uniformly sampled pairs (ragged 64-row tiles), horizon 100 with captures."""
    wl = W.make(3, n_envs=300)
    g = run_gpu(wl, snaps=[0, 3, 50, 99])
    rep = check_parity(wl, g)
    assert (g["actions"] == 255).any(), "expected some captures"


def test_parity_feature_ragged():
    """Feature dynamics d=512, bf16 MLP 512-512-512-18: 4 policies x 5 envs per
    pair, horizon 8."""
    wl = W.make(4, P=4, per_pair=5, horizon=8)
    g = run_gpu(wl, snaps=[0, 4, 7])
    check_parity(wl, g)


def test_parity_team_reduced():
    """4v4 team game d=256, bf16 MLP 256-512-512-18, 16 policies from a
    Dirichlet meta-strategy, 100 envs, horizon 6."""
    wl = W.make(5, P=16, n_envs=100, horizon=6)
    g = run_gpu(wl, snaps=[0, 3, 5])
    check_parity(wl, g)


@pytest.mark.parametrize("hid", [64, 128, 256])
def test_parity_team_2v2_hidden_widths(hid):
    """2v2 feature game with narrower hidden layers (other MFMA wave splits)."""
    wl = W.team_variant(4, P=6, n_envs=150, horizon=3, dims=[256, hid, hid, 18])
    g = run_gpu(wl, snaps=[0, 2])
    check_parity(wl, g)


_HID512 = {
    # hidden width 512 (four wavefronts per 64-row tile, 128 output units
    # each) under every observation build of the 64-row kernel
    "pursuit_75": lambda: W.with_policies(W.make(3, P=2, n_envs=150, horizon=20), W.MLP_BF16,
                                          [75, 512, 512, 5]),
    "iter_24": lambda: W.with_policies(W.make(2, P=3, per_pair=11, horizon=5), W.MLP_BF16,
                                       [24, 512, 512, 3]),
    "feature_d64": lambda: W.with_policies(W.team_variant(2, d=64, P=3, n_envs=70, horizon=3),
                                           W.MLP_BF16, [64, 512, 512, 18]),
    "feature_d128": lambda: W.with_policies(W.team_variant(4, d=128, P=3, n_envs=60,
                                                          horizon=3),
                                            W.MLP_BF16, [128, 512, 512, 18]),
}


@pytest.mark.parametrize("name", sorted(_HID512))
def test_parity_hidden_width_512_every_observation(name):
    """Hidden width 512 on the pursuit, iterated-game and narrow feature
    observations (input widths 80, 32, 64, 128 after padding): ragged and
    multi-tile buckets, every env against the oracle."""
    wl = _HID512[name]()
    g = run_gpu(wl, snaps=[0, wl.horizon - 1])
    check_parity(wl, g)


def test_parity_feature_shared_init_d64():
    wl = W.team_variant(2, d=64, P=3, n_envs=70, horizon=5, dims=[64, 64, 64, 18])
    wl.init_mode = W.INIT_SHARED
    g = run_gpu(wl, snaps=[0, 4])
    check_parity(wl, g)
    assert np.all(g["states"][0] == g["states"][0][0])


# Larger buckets: several full tiles per policy plus ragged tails.  With d=512
# observations and >= 256 slots per policy the persistent 128-row kernel runs
# (output layer fed from the accumulators, next tile prefetched); below that,
# and for narrower observations, the 64-row kernel.

def test_parity_team_large_buckets():
    """4v4 team game, 4 policies, 150 envs x 8 seats = 1200 slots (uneven
    Dirichlet buckets)."""
    wl = W.make(5, P=4, n_envs=150, horizon=4)
    g = run_gpu(wl, snaps=[0, 3])
    check_parity(wl, g)


def test_parity_feature_d512_large_buckets():
    """d=512, 2 policies x 70 envs per pair = 560 slots (persistent kernel)."""
    wl = W.make(4, P=2, per_pair=70, horizon=4)
    g = run_gpu(wl, snaps=[0, 3])
    check_parity(wl, g)


@pytest.mark.parametrize("hid", [64, 128, 256, 512])
def test_parity_persistent_hidden_widths(hid):
    """d=512 2v2 game, 2 policies x 320 slots: every wave split of the
    persistent kernel."""
    wl = W.team_variant(4, d=512, P=2, n_envs=160, horizon=3, dims=[512, hid, hid, 18])
    g = run_gpu(wl, snaps=[0, 2])
    check_parity(wl, g)


@pytest.mark.parametrize("hid", [64, 128, 256])
def test_parity_team_2v2_large_buckets_hidden_widths(hid):
    wl = W.team_variant(4, P=2, n_envs=200, horizon=3, dims=[256, hid, hid, 18])
    g = run_gpu(wl, snaps=[0, 2])
    check_parity(wl, g)


@pytest.mark.parametrize("P", [8, 64])
def test_parity_team_many_tiles_sampled(P):
    """4v4 d=256 game with the 256-512-512-18 policies: 6000 envs x 8 seats =
    48000 slots, 750+ 64-row tiles (more than one round of workgroups, ragged
    policy ends); the oracle replays a sample of envs whose slots fall in most
    tiles."""
    wl = W.team_variant(8, P=P, n_envs=6000, horizon=3, dims=[256, 512, 512, 18])
    g = run_gpu(wl, snaps=[0, 2])
    rng = np.random.default_rng(P)
    sel = np.unique(np.concatenate([[0, 1, wl.n_envs - 1],
                                    rng.choice(wl.n_envs, 250, replace=False)]))
    check_parity(wl, g, sel)


def test_parity_team_large_buckets_biases():
    """4v4 d=256 game, 256-512-512-18 policies with nonzero biases, 4
    policies, 300 envs (2400 slots, several full tiles per policy), every env
    against the oracle."""
    wl = _with_biases(W.team_variant(8, d=256, P=4, n_envs=300, horizon=3,
                                     dims=[256, 512, 512, 18]), 6)
    g = run_gpu(wl, snaps=[0, 2])
    check_parity(wl, g)


@pytest.mark.parametrize("d", [256, 512])
def test_parity_many_tiles_sampled(d):
    """80000 slots (more tiles than workgroups: 64-row tiles for d=256, several
    128-row tiles per persistent workgroup for d=512); the oracle replays a
    sample of envs including both ends of the batch."""
    wl = W.team_variant(4, d=d, P=2, n_envs=20000, horizon=3, dims=[d, 64, 64, 18])
    g = run_gpu(wl, snaps=[0, 2])
    rng = np.random.default_rng(7)
    sel = np.sort(np.concatenate([[0, 1, wl.n_envs - 1],
                                  rng.choice(np.arange(2, wl.n_envs - 1), 197, replace=False)]))
    check_parity(wl, g, sel)


# ------------------------------------------------------------ invariants

def test_determinism_and_shard_merge():
    """Same seed twice gives identical tables; two half batches with
    env_offset give the same returns and table as one batch."""
    import paper_2106_07551_amd as M
    from paper_2106_07551_amd import workload_io as IO
    wl = W.make(3, n_envs=2000, horizon=30)
    pop = IO.make_population(wl)
    env = IO.make_env(wl)
    full = IO.make_pairs(wl)
    r1 = torch.empty((2, 2000), device="cuda")
    pop.rollout(env, 2000, full, wl.seed, 30, returns=r1)
    t1 = pop.payoff(reset=True)
    pop.rollout(env, 2000, full, wl.seed, 30)
    t2 = pop.payoff(reset=True)
    assert np.array_equal(t1["counts"], t2["counts"])
    assert np.array_equal(np.nan_to_num(t1["mean"]), np.nan_to_num(t2["mean"]))
    ra = torch.empty((2, 1200), device="cuda")
    rb = torch.empty((2, 800), device="cuda")
    pa = IO.make_pairs(wl, n_envs=1200, env_offset=0)
    pb = IO.make_pairs(wl, n_envs=800, env_offset=1200)
    assert torch.equal(torch.cat([pa, pb]), full)
    pop.rollout(env, 1200, pa, wl.seed, 30, returns=ra)
    pop.rollout(env, 800, pb, wl.seed, 30, env_offset=1200, returns=rb)
    t3 = pop.payoff(reset=True)
    assert torch.equal(torch.cat([ra, rb], dim=1), r1)
    assert np.array_equal(t3["counts"], t1["counts"])
    assert np.array_equal(np.nan_to_num(t3["mean"]), np.nan_to_num(t1["mean"]))
    assert t3["live_frames"] == t1["live_frames"]
    pop.close()


def test_single_env_and_horizon_one():
    wl = W.make(5, P=4, n_envs=1, horizon=1)
    g = run_gpu(wl, snaps=[0])
    check_parity(wl, g)


def test_profile_mask_and_stride():
    """Only the enabled kernel classes are timed, one launch in `every`."""
    import paper_2106_07551_amd as M
    from paper_2106_07551_amd import workload_io as IO
    wl = W.make(5, P=8, n_envs=64, horizon=10)
    pop = IO.make_population(wl)
    env = IO.make_env(wl)
    pairs = IO.make_pairs(wl)
    pop.profile_enable(True, kernels=[M.K_POLICY], every=4)
    pop.rollout(env, wl.n_envs, pairs, wl.seed, 10)
    ms, n = pop.profile_read(M.K_POLICY)
    assert n == 3 and ms > 0          # launches 0, 4, 8
    assert pop.profile_read(M.K_ENV) == (0.0, 0)
    pop.profile_enable(True)
    pop.rollout(env, wl.n_envs, pairs, wl.seed, 10)
    assert pop.profile_read(M.K_ENV)[1] == 10 and pop.profile_read(M.K_SETUP)[1] == 1
    pop.profile_enable(False)
    pop.payoff(reset=True)
    pop.close()


def test_bad_policy_id_is_flagged():
    import paper_2106_07551_amd as M
    from paper_2106_07551_amd import workload_io as IO
    wl = W.make(2, P=2, per_pair=64, horizon=2)
    pop = IO.make_population(wl)
    env = IO.make_env(wl)
    pairs = wl.pairs.copy()
    pairs[5, 1] = 7
    pop.rollout(env, wl.n_envs, torch.from_numpy(pairs).cuda(), wl.seed, 2)
    t = pop.payoff(check=False)
    assert t["status"] == M.binding.E_DEVICE and t["device_flags"] & 1
    assert t["counts"].sum() == wl.n_envs - 1
    # flags are cleared once reported
    pop.rollout(env, wl.n_envs, torch.from_numpy(wl.pairs).cuda(), wl.seed, 2)
    assert pop.payoff(reset=True)["status"] == 0
    pop.close()


def test_nan_logits_are_flagged():
    import paper_2106_07551_amd as M
    wl = W.make(1, per_pair=8)
    tab = wl.tab_logits.copy()
    tab[2, 1] = np.nan
    pop = M.Population(M.POLICY_TABULAR, 4, 3, tab_logits=torch.from_numpy(tab).cuda())
    from paper_2106_07551_amd import workload_io as IO
    env = IO.make_env(wl)
    pop.rollout(env, wl.n_envs, IO.make_pairs(wl), wl.seed, 1)
    t = pop.payoff(check=False)
    assert t["status"] == M.binding.E_DEVICE and t["device_flags"] & 2
    pop.close()


@pytest.mark.parametrize("c,n_envs", [(3, 96), (5, 40), (4, 0)])
def test_nan_logits_are_flagged_bf16(c, n_envs):
    """A NaN output weight of policy 1 makes that policy's logits NaN; the
    bf16 kernels (64-row, and the persistent one for the d=512 feature game)
    raise the device flag while sampling."""
    from paper_2106_07551_amd import workload_io as IO
    import paper_2106_07551_amd as M
    wl = W.make(c, P=2, per_pair=80, horizon=2) if c == 4 else W.make(c, P=2, n_envs=n_envs,
                                                                      horizon=2)
    wl.weights[2] = wl.weights[2].copy()
    wl.weights[2][1, 0, 0] = np.nan
    pop = IO.make_population(wl)
    env = IO.make_env(wl)
    pop.rollout(env, wl.n_envs, IO.make_pairs(wl), wl.seed, 2)
    t = pop.payoff(check=False)
    assert t["status"] == M.binding.E_DEVICE and t["device_flags"] & 2
    pop.close()


@pytest.mark.parametrize("bits", [0x7FC00000, 0xFFC00000], ids=["pos_nan", "neg_nan"])
@pytest.mark.parametrize("layer", [0, 1])
@pytest.mark.parametrize("c", [2, 3, 4, 5], ids=["iter_f32", "pursuit", "feature_persist",
                                                 "team"])
def test_nan_hidden_weights_are_flagged(c, layer, bits):
    """A NaN weight of either sign in the first or second layer of policy 1
    reaches every logit of that policy (the hidden ReLU keeps a NaN of either
    sign) and raises the NaN flag on the device, in the fp32 kernel, the 64-row
    bf16 kernel and the persistent one; the oracle stops with a NaN logit on an
    env that plays policy 1, and envs that play only policy 0 still match it."""
    import paper_2106_07551_amd as M
    if c == 2:
        wl = W.make(2, P=2, per_pair=64, horizon=3)
    elif c == 4:
        wl = W.make(4, P=2, per_pair=80, horizon=3)    # 640 slots: persistent kernel
    else:
        wl = W.make(c, P=2, n_envs=96 if c == 3 else 40, horizon=3)
    wl.weights = [w.copy() for w in wl.weights]
    wl.weights[layer][1, 3, 5] = np.frombuffer(np.uint32(bits).tobytes(), np.float32)[0]
    g = run_gpu(wl, snaps=[0, 2], check=False)
    t = g["table"]
    assert t["status"] == M.binding.E_DEVICE and t["device_flags"] & 2, t["device_flags"]
    uses1 = (g["pairs"] == 1).any(axis=1)
    e1 = int(np.nonzero(uses1)[0][0])
    with pytest.raises(RuntimeError, match=r"\(-2\)"):
        oracle.rollout(wl, [e1], g["pairs"][[e1]], horizon=3)
    clean = np.nonzero(~uses1)[0]
    say(f"[nan-hidden] c={c} layer={layer} bits={bits:#x}: {len(clean)} clean envs")
    if len(clean):
        check_parity(wl, g, clean)


def test_host_validation_errors():
    import paper_2106_07551_amd as M
    from paper_2106_07551_amd import workload_io as IO
    wl = W.make(4, P=2, per_pair=1, horizon=2)
    pop = IO.make_population(wl)
    env = IO.make_env(wl)
    pairs = IO.make_pairs(wl)
    with pytest.raises(M.MalibError) as e:
        pop.rollout(env, wl.n_envs, pairs, wl.seed, 0)
    assert e.value.status == M.binding.E_INVAL
    with pytest.raises(M.MalibError):
        pop.rollout(env, 0, pairs, wl.seed, 2)
    bad = M.Env(M.ENV_FEATURE, 2, 18, team=[1, -1], d=96, W=None, emb=None, u=None)
    with pytest.raises(M.MalibError):
        pop.rollout(bad, wl.n_envs, pairs, wl.seed, 2)
    # widths beyond 1024 are rejected by the library before any device work
    # (the weights below, sized as the header requires, are never read)
    dims = [512, 2048, 2048, 18]
    ws = [torch.zeros(2 * dims[l + 1] * dims[l], device="cuda") for l in range(3)]
    with pytest.raises(M.MalibError) as e:
        M.Population(M.POLICY_MLP_BF16, 2, 18, dims=dims, weights=ws)
    assert e.value.status == M.binding.E_UNSUPPORTED
    del ws
    # buffers of the wrong size or dtype never reach the library
    with pytest.raises(M.ArgumentError):
        pop.rollout(env, wl.n_envs, pairs[:-1], wl.seed, 2)
    with pytest.raises(M.ArgumentError):
        pop.rollout(env, wl.n_envs, pairs.to(torch.int64), wl.seed, 2)
    with pytest.raises(M.ArgumentError):
        pop.rollout(env, wl.n_envs, pairs, wl.seed, 2,
                    returns=torch.empty(wl.n_envs, device="cuda"))
    assert pop.payoff()["counts"].sum() == 0
    pop.close()


# ------------------------------------------------------------ nonzero biases
# The generated populations have zero biases; these cases give every layer a
# random fp32 bias, so that the bias-to-unit mapping of each policy kernel
# (accumulator layout, output reduction) is compared with the oracle.
def _with_biases(wl, seed, scale=0.3):
    rng = np.random.default_rng([2106, 7551, 77, seed])
    wl.biases = [rng.normal(0.0, scale, b.shape).astype(np.float32) for b in wl.biases]
    return wl


def _with_dims(wl, dims, seed):
    """Fresh fp32 weights of the given widths (iterated game)."""
    rng = np.random.default_rng([2106, 7551, 78, seed])
    wl.dims = dims
    wl.weights, wl.biases = W._mlp(rng, wl.P, dims, bf16=wl.pol_kind == W.MLP_BF16)
    return wl


@pytest.mark.parametrize("hid", [32, 64])
def test_parity_iter_biases_hidden_widths(hid):
    """fp32 MFMA kernel, both hidden widths, nonzero biases: 3 policies x 37
    envs per pair (111 rows per policy: three 32-row tiles + a ragged one)."""
    wl = _with_biases(_with_dims(W.make(2, P=3, per_pair=37), [24, hid, hid, 3], hid), hid)
    g = run_gpu(wl, snaps=[0, 7, 31])
    check_parity(wl, g)


def test_parity_team_biases():
    """64-row bf16 kernel on feature observations (4v4, d=256), nonzero biases."""
    wl = _with_biases(W.team_variant(8, d=256, P=4, n_envs=48, horizon=4,
                                     dims=[256, 512, 512, 18]), 5)
    g = run_gpu(wl, snaps=[0, 3])
    check_parity(wl, g)


def test_parity_pursuit_biases():
    """64-row bf16 kernel on the pursuit window (one partial-logit group),
    nonzero biases."""
    wl = _with_biases(W.make(3, n_envs=300, horizon=30), 3)
    g = run_gpu(wl, snaps=[0, 10, 29])
    check_parity(wl, g)


def test_parity_persistent_biases():
    """Persistent d=512 kernel, nonzero biases: 2 policies x 320 slots."""
    wl = _with_biases(W.team_variant(4, d=512, P=2, n_envs=160, horizon=3,
                                     dims=[512, 512, 512, 18]), 4)
    g = run_gpu(wl, snaps=[0, 2])
    check_parity(wl, g)


@pytest.mark.parametrize("grid", [5, 13])
def test_parity_pursuit_other_grids(grid):
    """Pursuit on a 5x5 and a 13x13 torus (reset cells, moves, captures and the
    window's wrap-around off the 8x8 case)."""
    wl = W.make(3, n_envs=256, horizon=40)
    wl.grid = grid
    g = run_gpu(wl, snaps=[0, 9, 39])
    check_parity(wl, g)


@pytest.mark.parametrize("n_actions", [11, 20, 32])
def test_parity_matrix_many_actions(n_actions):
    """One-step matrix game with 11, 20 and 32 actions (tabular policies): the
    sampling's two-, three- and four-block Philox cases inside the env step."""
    rng = np.random.default_rng([2106, 7551, 79, n_actions])
    wl = W.make(1, P=3, per_pair=300)
    a = rng.uniform(-1.0, 1.0, (n_actions, n_actions)).astype(np.float32)
    wl.A = np.triu(a, 1) - np.triu(a, 1).T
    wl.n_actions = n_actions
    wl.tab_logits = rng.normal(0.0, 1.0, (wl.P, n_actions)).astype(np.float32)
    g = run_gpu(wl, snaps=[0])
    check_parity(wl, g)


# ------------------------------------------------------------ action counts

@pytest.mark.parametrize("A, hid", [(32, 512), (9, 256), (1, 128)])
def test_parity_feature_action_counts(A, hid):
    """The feature game's sampling inside the 64-row kernel at 32 actions
    (four full Philox blocks per row, every partial-logit register group),
    9 (a block of one) and 1 (the only action always wins): 2v2 game, d = 128,
    every env against the oracle."""
    wl = W.team_variant(4, d=128, P=5, n_envs=90, horizon=3)
    rng = np.random.default_rng([2106, 7551, 32, A])
    wl.n_actions = A
    wl.emb = rng.normal(0.0, np.sqrt(0.1), (wl.n_agents, A, wl.d)).astype(np.float32)
    wl = W.with_policies(wl, W.MLP_BF16, [wl.d, hid, hid, A], variant=A)
    g = run_gpu(wl, snaps=[0, 2])
    check_parity(wl, g)
    if A == 1:
        assert (g["actions"] == 0).all()


@pytest.mark.parametrize("team, P", [([1, 1, -1], 6), ([1, -1, -1, 1, -1], 9),
                                     ([-1, 1, 1, -1, 1, -1, 1], 70)])
def test_parity_team_odd_sides(team, P):
    """Odd seat counts with unequal and interleaved sides (3, 5 and 7 seats;
    70 policies take the bucketed payoff reduction): returns, states, actions
    and the table against the oracle, every env."""
    wl = W.team_variant(len(team), d=64, P=P, n_envs=80, horizon=3, team=team,
                        dims=[64, 128, 128, 18])
    g = run_gpu(wl, snaps=[0, 2])
    check_parity(wl, g)


def test_parity_team_max_population():
    """The 4v4 game with 256 policies (8-bit policy ids, about four rows per
    policy, every tile ragged), every env against the oracle."""
    wl = W.make(5, P=256, n_envs=120, horizon=2)
    g = run_gpu(wl, snaps=[0, 1])
    check_parity(wl, g)


# ------------------------------------------------------------ largest population

def test_parity_max_population_pursuit():
    """256 policies, the most the ABI takes (every bit of the bucketing's
    8-bit policy id in use): bf16 pursuit with about two rows per policy, so
    nearly every tile is a ragged one."""
    wl = W.make(3, P=256, n_envs=300, horizon=20)
    g = run_gpu(wl, snaps=[0, 19])
    check_parity(wl, g)


def test_parity_max_population_iter_sampled():
    """256 fp32 policies, all 65536 ordered pairs once (one row per pair and
    seat: 32-row tiles of about 16 rows), sampled envs in lockstep."""
    wl = W.make(2, P=256, per_pair=1, horizon=4)
    g = run_gpu(wl, snaps=[0, 3])
    sel = np.concatenate([np.arange(0, wl.n_envs, 331), [wl.n_envs - 1]])
    check_parity(wl, g, sel)


def test_parity_max_population_matrix():
    """256 tabular policies, every ordered pair twice (131072 envs), all envs."""
    wl = W.make(1, P=256, per_pair=2)
    g = run_gpu(wl, snaps=[0])
    check_parity(wl, g)


def test_parity_maximum_batch_32_actions_sampled():
    """The largest batch the ABI takes (n_envs * n_agents = 2^26 slots) with
    32 actions: logit offsets slot * A reach 2^31, past 32-bit indexing.
    Sampled envs in lockstep (the first, the last, and across the range);
    the table against the fp64 reduction of every env's returns."""
    rng = np.random.default_rng([2106, 7551, 26])
    wl = W.make(1, P=4, per_pair=1 << 21)
    assert wl.n_envs * wl.n_agents == 1 << 26
    a = rng.uniform(-1.0, 1.0, (32, 32)).astype(np.float32)
    wl.A = np.triu(a, 1) - np.triu(a, 1).T
    wl.n_actions = 32
    wl.tab_logits = rng.normal(0.0, 1.0, (wl.P, 32)).astype(np.float32)
    g = run_gpu(wl, snaps=())
    sel = np.concatenate([[0], rng.choice(wl.n_envs, 254, replace=False), [wl.n_envs - 1]])
    check_parity(wl, g, np.unique(sel))
    assert g["table"]["counts"].sum() == wl.n_envs
