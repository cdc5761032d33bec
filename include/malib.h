/*
 * malib.h - C ABI of the MI355X (gfx950) payoff-table rollout library.
 *
 * The library fills the empirical payoff table of a policy population: it
 * simulates many episodes for every policy combination drawn from the
 * population and reduces their returns into a mean-return matrix with
 * per-cell counts.  In MALib (arXiv 2106.07551) this is the work of the
 * Actors and the Evaluator: each agent picks a policy from its pool to form a
 * combination Comb_t (Sec. 3.1, task graph), rollouts sample
 * X ~ P(s, a, s' | a ~ Comb_t) (Sec. 3.1, rollout equation), and the
 * Evaluator keeps a payoff table of the evaluation result of every policy
 * combination, on which e.g. PSRO solves for a meta-strategy (Sec. 3.2,
 * Actor-Evaluator-Learner).  The single-instance example (Appendix C.2) names
 * the pieces: PayoffManager, run_simulation_and_update_payoff, and per-agent
 * policy distributions Dict[AgentID, Dict[PolicyID, float]].
 *
 * Conventions shared by every call:
 *  - Device pointers are HIP device addresses (e.g. torch CUDA tensors'
 *    data_ptr()); host pointers are ordinary process memory.  Each argument
 *    says which it is.
 *  - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *    All device work is enqueued on it asynchronously; only malib_payoff_eval
 *    and malib_profile_read synchronize it.  Device buffers the caller passes
 *    in (pair assignments, environment parameters) must stay valid until the
 *    work on the stream has completed.
 *  - The caller owns every pointer it passes.  malib_pop_create copies and
 *    re-lays out the weights, so they may be freed after it returns (and after
 *    the stream has completed).
 *  - Host-detectable errors (bad sizes, null pointers, unsupported shapes,
 *    invalid meta-strategies) return a negative status before any device work
 *    is enqueued, and malib_last_error() gives a message (thread-local).
 *    Errors the device detects (a policy id outside [0, P), a NaN logit) set a
 *    flag on the population handle that the next malib_payoff_eval reports
 *    as MALIB_E_DEVICE.
 *  - Results depend only on (inputs, seed, env_offset + local env index):
 *    they are independent of launch geometry, batching and streams.
 *  - A handle must not be used from two threads at once.
 */
#ifndef MALIB_H
#define MALIB_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t malib_status;
enum {
    MALIB_OK = 0,
    MALIB_E_INVAL = -1,        /* invalid argument */
    MALIB_E_NOMEM = -2,        /* device or host allocation failed */
    MALIB_E_HIP = -3,          /* a HIP runtime call failed */
    MALIB_E_UNSUPPORTED = -4,  /* valid but not implemented shape/combination */
    MALIB_E_DEVICE = -5        /* the device flagged bad data (see above) */
};

/*
 * Allocation failures can be forced for tests of the error paths: while the
 * environment variable MALIB_FAULT_ALLOC is set to anything but "" or "0",
 * every device or pinned host allocation the library makes (handle creation
 * and extension, growth of a handle's batch buffers, the meta-samplers'
 * thresholds) fails without allocating and the call returns MALIB_E_NOMEM,
 * leaving handles as they were.  The variable is read at each allocation.
 */

/* ---------------------------------------------------------------- population */

enum {
    MALIB_POLICY_TABULAR = 0,  /* state-less logits per policy (one-step games) */
    MALIB_POLICY_MLP_F32 = 1,  /* fp32 MLP, fp32 arithmetic */
    MALIB_POLICY_MLP_BF16 = 2  /* bf16 MLP: bf16 inputs/weights/hidden, fp32 accumulation */
};

/*
 * A population of P policies shared by every seat (a policy pool that the
 * agents draw from, Sec. 3.1).  MLP policies have two
 * hidden ReLU layers: logits = W3 relu(W2 relu(W1 x + b1) + b2) + b3, with the
 * weight of layer l laid out [P][dims[l+1]][dims[l]] (row = output unit).
 *
 * Supported shapes:
 *  - TABULAR: n_layers = 0, tab_logits device fp32 [P][n_actions].
 *  - MLP_F32 and MLP_BF16: n_layers = 3, dims = {in, h1, h2, A} with
 *    1 <= in, h1, h2 <= 1024 and A = n_actions; `in` must be the
 *    environment's observation width (iterated game 8 * n_actions, pursuit
 *    75, feature games d).  bf16 populations have their fp32 weights rounded
 *    to bf16 (nearest, ties to even) when the handle is created.
 *    Specialized MFMA kernels run fp32 {24, h, h, 3} with h in {32, 64} and
 *    bf16 {in <= 512, h, h, A} with h in {64, 128, 256, 512}; every other
 *    shape runs a generic kernel (fp32 fused multiply-add chains over the
 *    inputs, same arithmetic per element, lower throughput).
 * 1 <= P <= 256, 1 <= n_actions <= 32.  Widths above 1024 return
 * MALIB_E_UNSUPPORTED before any device work.
 */
typedef struct {
    int32_t kind;                 /* MALIB_POLICY_* */
    int32_t n_policies;           /* P */
    int32_t n_actions;            /* A (= dims[n_layers] for MLPs) */
    int32_t n_layers;             /* 3 for MLPs, 0 for TABULAR */
    const int32_t* dims;          /* host [n_layers + 1] */
    const float* const* weights;  /* host array of n_layers device pointers (fp32) */
    const float* const* biases;   /* host array of n_layers device pointers
                                     fp32 [P][dims[l+1]], or NULL (all zero);
                                     individual entries may be NULL (zero) */
    const float* tab_logits;      /* TABULAR: device fp32 [P][n_actions] */
    const int64_t* policy_ids;    /* host [P] or NULL: the caller's ids of the policies
                                     (the PolicyID keys of the example API's per-agent
                                     distributions, Appendix C.2), distinct; NULL gives
                                     0 .. P-1.  Rows and columns of every table and
                                     every pair assignment use the index 0 .. P-1;
                                     malib_pop_policy_ids maps indices back to ids */
} malib_pop_desc;

typedef struct malib_pop* malib_pop_t;

/* Create a population handle: validates, allocates, packs the weights for the
 * policy kernels, allocates the P x P payoff accumulators (zeroed).  The
 * packing runs on `stream`, which is synchronized before returning, so the
 * caller's weight buffers may be released right away.  On error *out is set
 * to NULL. */
malib_status malib_pop_create(const malib_pop_desc* desc, void* stream, malib_pop_t* out);

/* Free a handle (synchronizes the device first).  NULL is ignored. */
void malib_pop_destroy(malib_pop_t pop);

/*
 * The caller's policy ids of a population (Sec. 3.1: agents draw policies from
 * pools keyed by policy id; Appendix C.2: distributions Dict[PolicyID, float]),
 * in index order: ids_out[i] is the id of the policy at row / column i of the
 * payoff table and of pair-assignment value i.  *n_out receives P.  ids_out
 * may be NULL (only the count is returned); otherwise it must hold
 * `capacity` >= P entries (MALIB_E_INVAL if not).  Host-only, no device work.
 */
malib_status malib_pop_policy_ids(malib_pop_t pop, int64_t* ids_out, int32_t capacity,
                                  int32_t* n_out);

/* --------------------------------------------------------------- environment */

enum {
    MALIB_ENV_MATRIX = 0,       /* one-step 2-player matrix game: r0 = A[a0][a1], r1 = -r0 */
    MALIB_ENV_ITER_MATRIX = 1,  /* repeated matrix game; obs = one-hot of the last 4 joint actions */
    MALIB_ENV_PURSUIT = 2,      /* 2-agent pursuit-evasion on a torus grid, capture ends the episode */
    MALIB_ENV_FEATURE = 3       /* s' = tanh(W s + sum_k emb[k][a_k]), r = u . s' (zero-sum teams) */
};

enum { MALIB_INIT_PER_ENV = 0, MALIB_INIT_SHARED = 1 };

/*
 * Environment family and parameters.  Rules (the paper specifies none; these
 * are the synthetic games used to exercise the rollout path):
 *  MATRIX / ITER_MATRIX: 2 seats, n_actions <= 3 for ITER_MATRIX, <= 32 for
 *    MATRIX.  ITER observation of seat k: for lag 1..4 (most recent first) the
 *    one-hot of its own action then of the opponent's, zeros before t = 0.
 *  PURSUIT: 2 seats (0 = pursuer, 1 = evader), n_actions = 5 (stay, up, down,
 *    left, right), grid = 8.  Capture (same cell after the move, or the two
 *    swapped cells) gives +1 / -1 and ends the episode; finished envs take no
 *    further actions and count no further frames.  Observation: egocentric
 *    5x5x3 window (pursuer, evader, self channels), 75 values.
 *  FEATURE: 2..8 seats, state fp32 [d] with d a multiple of 64, 64 <= d <= 512;
 *    the fp32 sums are formed in a fixed order (W s as a fused multiply-add
 *    chain over the input index, then the embeddings in seat order), tanh is
 *    the library's fixed tanh_ref and r = u . s' is a fused chain over the
 *    index; seats with team +1 receive r, the others -r.  Every seat observes
 *    bf16(s_t).
 */
typedef struct {
    int32_t kind;             /* MALIB_ENV_* */
    int32_t n_agents;         /* seats per env */
    int32_t n_actions;        /* must equal the population's */
    int32_t grid;             /* PURSUIT: torus side (8) */
    const int8_t* team;       /* host [n_agents]: +1 row side, -1 column side;
                                 NULL means {+1, -1} (two seats) */
    const float* A;           /* MATRIX / ITER_MATRIX: device fp32 [n_actions][n_actions] */
    int32_t d;                /* FEATURE: state dimension */
    int32_t init_mode;        /* MALIB_INIT_*: SHARED starts every env from the
                                 reset draw of global env 0 (for tests) */
    const float* W;           /* FEATURE: device fp32 [d][d] (row = output) */
    const float* emb;         /* FEATURE: device fp32 [n_agents][n_actions][d] */
    const float* u;           /* FEATURE: device fp32 [d] */
} malib_env_desc;

/* ---------------------------------------------------------------- rollouts */

/*
 * Optional parity trace.  Any pointer may be NULL.
 *  actions: device uint8 [horizon][n_envs * n_agents]; 255 where the env has
 *           already finished.
 *  snap_steps: host int32 [n_snap], steps in [0, horizon) to snapshot;
 *  logits: device fp32 [n_snap][n_envs * n_agents][n_actions], the logits of
 *          that step (slot order env * n_agents + seat);
 *  states: device [n_snap][...] the state before that step, in the format
 *          ITER_MATRIX: uint16 [n_envs] (4-bit joint action a0*3+a1 per lag,
 *          lag 1 in the low nibble, 15 = none); PURSUIT: uint8 [n_envs][3]
 *          (pursuer cell, evader cell, done), cell = 8*y + x; FEATURE: fp32
 *          [n_envs][d]; MATRIX: nothing.
 *  perm / offsets: device int32 [n_envs * n_agents] / [P + 1]: the slots sorted
 *          by policy id (stable) and the bucket boundaries (MLP policies only).
 */
typedef struct {
    uint8_t* actions;
    int32_t n_snap;
    const int32_t* snap_steps;
    float* logits;
    void* states;
    int32_t* perm;
    int32_t* offsets;
} malib_trace;

/*
 * Simulate n_envs episodes of `horizon` steps and add their returns to the
 * handle's payoff table (run_simulation_and_update_payoff, Appendix C.2).
 *  pair_assign: device int32 [n_envs][n_agents], the policy id of every seat
 *               (one policy combination per env, Sec. 3.1).
 *  seed, env_offset: the action noise, resets and everything random depend
 *               only on (seed, env_offset + e) for local env e.
 *  returns:     device fp32 [n_agents][n_envs] per-seat undiscounted returns,
 *               or NULL.
 *  trace:       NULL or a parity trace (above).
 * Every step runs: grouped policy forward (slots bucketed by policy id),
 * Gumbel-max action sampling on Philox4x64-10 noise, environment step with
 * return accumulation; after the last step the returns are reduced into the
 * P x P table: each (row-side seat a, column-side seat b) pair of an env adds
 * the return of seat a to cell (pid[a], pid[b]).
 * Limits: n_envs >= 1, n_envs * n_agents <= 2^26, 1 <= horizon <= 100000.
 * Device buffers of the batch (logits, state, bucketing tables) are the
 * handle's, grown with hipMalloc when a batch needs more than earlier ones.
 * On a stream that the caller is capturing into a HIP graph, a batch that
 * would grow them returns MALIB_E_INVAL before any device work (run one batch
 * of that size outside the capture first, or use
 * malib_rollout_batch_noalloc).
 */
malib_status malib_rollout_batch(malib_pop_t pop, const malib_env_desc* env,
                                 int64_t n_envs, const int32_t* pair_assign,
                                 uint64_t seed, int64_t env_offset, int32_t horizon,
                                 float* returns, const malib_trace* trace, void* stream);

/* ------------------------------------------------------ trajectory records */

/*
 * A device ring of per-step records for learners (the Actors' samples that
 * the paper's offline dataset server stores, Sec. 3.1 and Sec. 3.2; the
 * per-agent episode buffer of the example API, Appendix C.2).  One record per
 * (step t, env e) of a batch, at index (cursor + t * n_envs + e) mod capacity;
 * older records are overwritten once the ring wraps.  All buffers are
 * caller-owned device memory:
 *  actions:  uint8 [capacity][n_agents], each seat's action; 255 where the
 *            env had already finished (no action).
 *  rewards:  fp32 [capacity], the row side's (team +1) reward of the step;
 *            the column side receives its negation.
 *  flags:    uint8 [capacity]: bit 0 the episode terminated at this step
 *            (pursuit capture), bit 1 the last step of the horizon, bit 2
 *            the env had finished before this step.
 *  obs:      NULL or the state every seat observed before the step, in
 *            compact form: ITER_MATRIX uint16 [capacity] (the history as in
 *            malib_trace's states), PURSUIT uint8 [capacity][2] (pursuer and
 *            evader cell), FEATURE bf16 [capacity][d] (bf16_rne(s), exactly
 *            the policy input), MATRIX nothing (not written).
 *  cursor:   records written so far; malib_rollout_batch_traj advances it by
 *            horizon * n_envs.
 */
typedef struct {
    uint8_t* actions;
    float* rewards;
    uint8_t* flags;
    void* obs;
    int64_t capacity;
    int64_t cursor;
} malib_traj;

/*
 * malib_rollout_batch that also writes every step's records into `traj`
 * (written by the env-step kernels as they step; nothing else changes: the
 * same returns, table and random streams).
 */
malib_status malib_rollout_batch_traj(malib_pop_t pop, const malib_env_desc* env,
                                      int64_t n_envs, const int32_t* pair_assign, uint64_t seed,
                                      int64_t env_offset, int32_t horizon, float* returns,
                                      malib_traj* traj, void* stream);

/* ------------------------------------------------------- no allocation */

/*
 * malib_rollout_batch for callers that cannot allocate device memory: code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc.  Same batch, same kernels, same results bit for bit as
 * malib_rollout_batch with trace = NULL, but the batch's scratch (logits,
 * returns, environment state, bucketing tables) lives in one static device
 * array of the library, 64 MiB (67108864 bytes) per GPU, held from the first
 * malib_pop_create on that GPU until the process ends; the call makes no
 * hipMalloc / hipFree and records no HIP-event timing.  The caller still
 * passes the handle, inputs and outputs.  A batch whose scratch (each buffer
 * rounded up to 256 bytes) exceeds the array returns MALIB_E_INVAL before any
 * device work: e.g. the 4v4 game of 16384 envs x 8 seats at d = 256 needs
 * about 54 MB, the d = 512 feature game of 65536 envs does not fit.
 * Every call on one GPU shares that GPU's array and overwrites it (the
 * returns are cleared by the call itself): calls that overlap on one GPU, on
 * any streams or handles, race and must be serialized by the caller.
 */
malib_status malib_rollout_batch_noalloc(malib_pop_t pop, const malib_env_desc* env,
                                         int64_t n_envs, const int32_t* pair_assign,
                                         uint64_t seed, int64_t env_offset, int32_t horizon,
                                         float* returns, void* stream);

/* ------------------------------------------------------------- payoff table */

typedef struct {
    int64_t live_frames;   /* live agent-frames (env, seat, step) since the last reset */
    int64_t envs;          /* envs simulated since the last reset */
    int32_t device_flags;  /* bit 0: policy id out of range; bit 1: NaN logit */
} malib_eval_stats;

/*
 * The payoff table (the PayoffManager of Appendix C.2): synchronizes `stream`,
 * then writes, each optional,
 *  mean:   host fp64 [P][P], sum / count, NaN where count == 0;
 *  counts: host int64 [P][P];
 *  stderr_out: host fp64 [P][P], standard error of the mean (NaN if count < 2);
 *  stats:  host, see above.
 * Sums are kept in 64-bit fixed point (2^-32 units for returns, 2^-20 for
 * squares), so the table is exact and independent of reduction order.
 * reset != 0 zeroes the table afterwards.  Returns MALIB_E_DEVICE (after
 * writing the outputs and clearing the flags) if the device flagged bad data.
 */
malib_status malib_payoff_eval(malib_pop_t pop, void* stream, int32_t reset,
                               double* mean, int64_t* counts, double* stderr_out,
                               malib_eval_stats* stats);

/* ------------------------------------------------------- table expansion */

/*
 * Grow the population by add->n_policies policies (the auto-curriculum adds
 * policies to the pools, Sec. 3.1; extend_policy_pool of the example API,
 * Appendix C.2).  `add` describes only the new policies, with the kind, dims
 * and n_actions of the population; they take indices P0 .. P0 + k - 1 and
 * the caller ids add->policy_ids (NULL: ids P0 .. P0 + k - 1), which must be
 * distinct from each other and from the ids already present.  The
 * payoff table grows to (P0 + k)^2 cells: the P0 x P0 cells keep their sums
 * and counts, the new cells start empty, the live-frame counter and the error
 * flags carry over.  Synchronizes the device (the old buffers are freed); on
 * an error the population is unchanged.
 */
malib_status malib_pop_extend(malib_pop_t pop, const malib_pop_desc* add, void* stream);

/*
 * Policy ids of the batch that simulates only the new cells after a
 * population grew from first_new to n_policies policies
 * (run_simulation_and_update_payoff of the example API, Appendix C.2, on the
 * new combinations only): every cell (r, c) with r >= first_new or
 * c >= first_new, n_policies^2 - first_new^2 cells, taken in row-major order
 * of the grid; cell number q is played by envs q*per_pair .. (q+1)*per_pair-1.
 * In each env the row-side seats (team +1) take r, the others c.
 *  team: host [n_agents] of +1 / -1, or NULL for two seats (seat 0 row side).
 *  pair_assign_out: device int32 [(n_policies^2 - first_new^2) * per_pair]
 *                   [n_agents], caller-owned.
 * Rolling that batch out into the same population (malib_rollout_batch with
 * an env_offset past the envs already simulated) merges it into the table:
 * the accumulators only add.  Asynchronous on `stream`.
 */
malib_status malib_expansion_pairs(int32_t n_policies, int32_t first_new, int32_t per_pair,
                                   int32_t n_agents, const int8_t* team,
                                   int32_t* pair_assign_out, void* stream);

/* ------------------------------------------------------------ meta-strategy */

/*
 * Draw the policy id of every seat from a meta-strategy (the per-agent policy
 * distribution of Appendix C.2; Comb_{t+1} ~ G(...) in Sec. 3.1).
 *  sigma: host fp32 [n_sigma][n_policies], non-negative, finite, positive sum
 *         per row (rows need not be normalized); n_sigma is 1 (shared by all
 *         seats) or n_agents (row k for seat k).
 *  pair_assign_out: device int32 [n_envs][n_agents].
 * Seat k of global env g = env_offset + e takes pid = min{m : x < T_m}, where
 * x is the first 32-bit lane of the Philox block (g, 0, 2<<32 | k, 0) and T_m
 * = floor(2^32 * C_m) from the fp64 cumulative sum C of the normalized row
 * (T_{P-1} = 2^32).  Policies with zero mass are never drawn.  The
 * thresholds are computed on the host and uploaded on `stream`, which is
 * synchronized once before the sampling kernel is enqueued.
 */
malib_status malib_meta_sample(const float* sigma, int32_t n_sigma, int32_t n_policies,
                               int64_t n_envs, int32_t n_agents, uint64_t seed,
                               int64_t env_offset, int32_t* pair_assign_out, void* stream);

/* ------------------------------------------------------------- meta-solver */

/*
 * The payoff table as the meta-solver's game: M [P][P] fp64 on the device,
 * the mean of each cell as malib_payoff_eval computes it (sum / count), 0 for
 * cells with no simulations.  Asynchronous on `stream`; M is caller-owned.
 */
malib_status malib_payoff_matrix(malib_pop_t pop, double* M, void* stream);

/*
 * Fictitious play on the table (the meta-update Comb_{t+1} ~ G(Eval) of
 * Sec. 3.1 with the fictitious-play meta-solver of the PSRO experiments,
 * Sec. 4.2; get_equilibrium of the example API, Appendix C.2).  The game is
 * two-player zero-sum: the row side receives M[i][j], the column side
 * -M[i][j].  Each of `iterations` (1 .. 2^24) simultaneous steps plays the
 * first best response of each side to the other's empirical play so far:
 * i_t = first argmax of v = sum over s < t of M[:, j_s], j_t = first argmin
 * of w = sum over s < t of M[i_s, :], v and w kept in fp64 and grown by one
 * column / row per step.
 *  M:     device fp64 [P][P], finite (e.g. from malib_payoff_matrix).
 *  sigma: device fp32 [2][P]: the row side's and the column side's play
 *         counts, i.e. their average strategies times `iterations`, usable
 *         directly as weight rows of malib_meta_sample_device.
 *  gap:   device fp64 [1] or NULL: (max v - min w) / iterations, the
 *         exploitability of the two average strategies; NaN if a NaN entered
 *         v or w (the counts are then unspecified but still sum to
 *         `iterations` per side).
 * Asynchronous on `stream`; one wavefront (the solver is sequential in t),
 * with M in LDS for P <= 128.
 */
malib_status malib_solve_fp(const double* M, int32_t n_policies, int32_t iterations,
                            float* sigma, double* gap, void* stream);

/*
 * The LP meta-solver (named beside fictitious play and alpha-rank for the
 * PSRO experiments, Sec. 4.2): the exact equilibrium of the two-player
 * zero-sum game M (the row side receives M[i][j], the column side -M[i][j]),
 * its value v = max_x min_j (x^T M)_j = min_y max_i (M y)_i, by the primal
 * simplex method (Bland's rule, fp64) on the column side's problem after
 * shifting M to positive entries; the row side's strategy is the dual
 * solution.  Optimal strategies need not be unique; the value is.
 *  M:      device fp64 [P][P], finite (a NaN or infinite entry gives NaN
 *          value, x, y and sigma, and pivots = -1).
 *  work:   device fp64 [P+1][2P+1] workspace, needed for P > 96 (NULL
 *          allowed below: the tableau then lives in LDS).
 *  value:  device fp64 [1]; x, y: device fp64 [P] (row and column side).
 *  sigma:  device fp32 [2][P] or NULL: x and y as weight rows for
 *          malib_meta_sample_device.
 *  pivots: device int32 [1] or NULL: simplex pivots taken, -1 if the limit
 *          of 64 P + 256 pivots was reached (value, x and y are then NaN).
 * Asynchronous on `stream`; one workgroup.
 */
malib_status malib_solve_lp(const double* M, int32_t n_policies, double* work, double* value,
                            double* x, double* y, float* sigma, int32_t* pivots,
                            void* stream);

/*
 * alpha-rank on the table (the meta-solver named beside fictitious play and
 * the LP solver for the PSRO experiments, Sec. 4.2, Table 3), in its authors'
 * single-population form (Omidshafiei et al., 2019): the P policies are one
 * population, and two policies meet once on each side of the game (the row
 * side receives M[i][j], the column side -M[i][j]), so a mutant s in a
 * population of r has fitness advantage u = alpha (M[s][r] - M[r][s]).  Its
 * fixation probability in a population of m is rho(u) = (1 - e^-u) /
 * (1 - e^-(m u)), 1/m at u = 0; a mutation picks one of the other P - 1
 * policies uniformly, so the chain moves r -> s with probability
 * rho / (P - 1).  pi is the chain's stationary distribution (unique: every
 * rho > 0 for finite arguments), computed with the Grassmann-Taksar-Heyman
 * elimination in fp64 (no subtractions; small probabilities keep their
 * relative accuracy).
 *  M:      device fp64 [P][P], finite (e.g. from malib_payoff_matrix).
 *  alpha:  ranking intensity, finite, >= 0 (0: the uniform distribution).
 *  m:      population size, 1 .. 10^6.
 *  work:   device fp64 [P][P] workspace, needed for P > 128 (NULL allowed
 *          below: the chain then lives in LDS).
 *  pi:     device fp64 [P] output.
 *  sigma:  device fp32 [2][P] or NULL: pi in both weight rows, usable
 *          directly by malib_meta_sample_device.
 * A fitness gap so large that some rho underflows to 0 can make the chain
 * reducible; pi is then undefined (NaN or Inf entries).  Asynchronous on
 * `stream`; one workgroup.
 */
malib_status malib_solve_alpharank(const double* M, int32_t n_policies, double alpha,
                                   int32_t m, double* work, double* pi, float* sigma,
                                   void* stream);

/*
 * Aggregate payoffs of a meta-strategy pair on a game, for the PSRO
 * convergence judgement of the example API's main loop (Appendix C.2:
 * aggregate(equilibrium) and aggregate(equilibrium, brs), then the
 * evaluator's convergence test).
 *  M:      device fp64 [P][P] (e.g. from malib_payoff_matrix).
 *  sigma:  device fp32 [2][P] weight rows (e.g. malib_solve_fp's counts):
 *          x = sigma[0] / sum, y = sigma[1] / sum, in fp64.
 *  br_row, br_col: the sides' best-response (newly trained) policy ids, or
 *          -1 to leave that side out.
 *  out:    device fp64 [5]: {x^T M y (row side's equilibrium payoff),
 *          -x^T M y (column side's), (M y)[br_row], -(x^T M)[br_col],
 *          improvement = the larger of the sides' best-response gains over
 *          their equilibrium payoffs}; NaN for a side left out.  Sums are
 *          sequential in index order (u = M y row by row, then x^T u).
 *          A converged meta-game has improvement <= a caller's tolerance.
 * Weights are not checked: a row without positive finite mass gives NaN.
 * Asynchronous on `stream`; one workgroup.
 */
malib_status malib_aggregate(const double* M, int32_t n_policies, const float* sigma,
                             int32_t br_row, int32_t br_col, double* out, void* stream);

/*
 * malib_meta_sample with the weights on the device (e.g. from malib_solve_fp),
 * same draws and the same fp64 thresholds.
 *  sigma:    device fp32 [n_sigma][n_policies] weight rows.
 *  seat_row: host int32 [n_agents] or NULL.  With NULL, n_sigma is 1 or
 *            n_agents as for malib_meta_sample; otherwise seat k draws from
 *            row seat_row[k] (in [0, n_sigma), n_sigma <= 8), e.g. row 0 (the
 *            row side's counts from malib_solve_fp) for the seats of one team
 *            and row 1 for the other.
 * Weights are checked on the device: a row with a negative or non-finite
 * weight or no positive mass gives policy id -1 to its seats, which the next
 * malib_rollout_batch flags (reported by malib_payoff_eval as
 * MALIB_E_DEVICE).  Asynchronous on `stream`.
 */
malib_status malib_meta_sample_device(const float* sigma, int32_t n_sigma, int32_t n_policies,
                                      int64_t n_envs, int32_t n_agents,
                                      const int32_t* seat_row, uint64_t seed,
                                      int64_t env_offset, int32_t* pair_assign_out,
                                      void* stream);

/* Message for the last non-OK status returned on this thread. */
const char* malib_last_error(void);

/* ------------------------------------------------------------- graph mode */

/*
 * Graph mode of a handle (enable != 0; off at creation).  The paper names the
 * per-step overheads of its rollout workers (environment resets, data
 * concatenation, locks) as the main source of throughput noise (Sec. 4.1);
 * here the per-step cost outside the kernels is one launch per kernel, which
 * matters for small batches.  In graph mode, malib_rollout_batch and
 * malib_rollout_batch_traj record the batch's whole launch sequence (set-up,
 * `horizon` x (policy forward, env step), payoff reduction) into a HIP graph
 * and replay it with one launch; the handle keeps one executable graph and
 * updates it in place for the next batch with the same launch structure
 * (same population, environment kind, sizes and horizon), so repeated batches
 * pay the instantiation once.  Results are identical to the direct launches.
 * Calls with a parity trace, calls on a stream that is being captured by the
 * caller (the launches then join the caller's graph; the handle's host-side
 * counts of envs and of fixed-length frames count the capture, not the
 * replays) and malib_rollout_batch_noalloc launch directly.  HIP-event timing
 * (malib_profile_enable) does not see launches made in graph mode.
 */
malib_status malib_pop_set_graph(malib_pop_t pop, int32_t enable);

/* ---------------------------------------------------------------- profiling */

enum {
    MALIB_K_POLICY = 0,   /* grouped policy forward */
    MALIB_K_SAMPLE = 1,   /* Gumbel-max action sampling: runs inside the env
                             step (MALIB_K_ENV), so this class records no
                             launches */
    MALIB_K_ENV = 2,      /* environment step + return accumulation */
    MALIB_K_SETUP = 3,    /* bucketing + reset */
    MALIB_K_PAYOFF = 4,   /* payoff reduction */
    MALIB_K_COUNT = 5
};

/* HIP-event timing of the handle's kernel launches, on the stream each kernel
 * runs on.  mask: bit (1 << MALIB_K_x) enables class x (0 disables timing);
 * every: time one launch in `every` of each enabled class (>= 1), so that the
 * events' own cost stays small in long runs.  Each call clears the totals. */
malib_status malib_profile_enable(malib_pop_t pop, int32_t mask, int32_t every);

/* Total elapsed milliseconds and number of timed launches of one kernel class
 * since the profile was enabled; synchronizes the recorded events. */
malib_status malib_profile_read(malib_pop_t pop, int32_t kernel, double* total_ms,
                                int64_t* launches);

/* ------------------------------------------------------------- diagnostics */

/* y[i] = tanh_ref(x[i]) on the device: the fixed tanh of the feature
 * dynamics, exposed so it can be compared bit for bit.  x, y: device fp32 [n]. */
malib_status malib_debug_tanh_ref(const float* x, float* y, int64_t n, void* stream);

/* y[i] = bf16 bits of x[i] (round to nearest even) on the device, with the
 * conversion the policy kernels use for observations, weights and hidden
 * activations.  x: device fp32 [n], y: device uint16 [n], n even. */
malib_status malib_debug_bf16(const float* x, uint16_t* y, int64_t n, void* stream);

/* Philox4x64-10 blocks on the device: out[i] = philox(ctr[i], (key0, key1)).
 * ctr, out: device uint64 [n][4]. */
malib_status malib_debug_philox(const uint64_t* ctr, uint64_t key0, uint64_t key1,
                                uint64_t* out, int64_t n, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* MALIB_H */
