/*
 * CPU oracle for the population payoff-table rollout path.
 *
 * TEST INFRASTRUCTURE ONLY.  Only tests/, __graft_entry__.smoke() and the
 * cpu_baseline leg of bench.py may load this code.  It shares nothing with the
 * HIP library: no headers, no helpers, no constant tables.
 *
 * What it computes (MALib, arXiv 2106.07551):
 *   - each agent picks one policy from its pool, forming a combination
 *     (Sec. 3.1, task graph);
 *   - rollouts draw actions from that combination, X ~ P(s,a,s' | a ~ Comb_t)
 *     (Sec. 3.1, rollout equation);
 *   - the evaluator keeps a payoff table of per-combination evaluation results
 *     (Sec. 3.2, Actor-Evaluator-Learner), here the mean undiscounted return
 *     (the payoff mean itself is taken in numpy, oracle/__init__.py);
 *   - a meta-strategy (per-agent distribution over policy ids, Appendix C.2
 *     example) picks the policies of the next combinations.
 * The paper gives no game rules, encodings or random-number layout; the
 * readings used here are the ones the design document lists (random stream:
 * Philox4x64-10 keyed by (seed, 0), counter (global env, step,
 * purpose<<32|slot, block)).
 *
 * The code is deliberately plain: one env at a time, one seat at a time,
 * fp64 accumulation for policy forwards, fp32 where the definition of the
 * environment fixes fp32 (the feature dynamics and the returns).
 * Build: gcc -O2 -march=x86-64-v3 -ffp-contract=off -fPIC -shared (no fast-math).
 *
 * Parity pins: see tests/test_oracle_pins.py.  The semantic readings of the
 * synthetic games (rules, encodings) are pinned only against themselves
 * ("parity unpinned" against any external implementation, since none exists).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------ */
/* Philox4x64-10: Salmon, Moraes, Dror, Shaw, "Parallel Random Numbers: As    */
/* Easy as 1, 2, 3", SC'11.  Ten rounds of two 64x64->128 multiplies; the key */
/* is bumped by the Weyl constants between rounds.                            */
/* ------------------------------------------------------------------------ */
void ora_philox4x64_10(const uint64_t ctr[4], const uint64_t key[2], uint64_t out[4])
{
    uint64_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
    uint64_t k0 = key[0], k1 = key[1];
    for (int round = 0; round < 10; ++round) {
        unsigned __int128 p0 = (unsigned __int128)0xD2E7470EE14C6C93ULL * c0;
        unsigned __int128 p1 = (unsigned __int128)0xCA5A826395121157ULL * c2;
        uint64_t hi0 = (uint64_t)(p0 >> 64), lo0 = (uint64_t)p0;
        uint64_t hi1 = (uint64_t)(p1 >> 64), lo1 = (uint64_t)p1;
        uint64_t n0 = hi1 ^ c1 ^ k0;
        uint64_t n1 = lo1;
        uint64_t n2 = hi0 ^ c3 ^ k1;
        uint64_t n3 = lo0;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
        k0 += 0x9E3779B97F4A7C15ULL;
        k1 += 0xBB67AE8584CAA73BULL;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

enum { PURPOSE_ACTION = 0, PURPOSE_RESET = 1, PURPOSE_META = 2 };

/* The eight 32-bit lanes of one Philox block: lane 2w is the low half of word
 * w, lane 2w+1 its high half. */
static uint32_t lane_of(uint64_t seed, int64_t g, int64_t t, int purpose, int slot,
                        int64_t block, int lane)
{
    uint64_t ctr[4] = {(uint64_t)g, (uint64_t)t,
                       ((uint64_t)(uint32_t)purpose << 32) | (uint32_t)slot,
                       (uint64_t)block};
    uint64_t key[2] = {seed, 0};
    uint64_t out[4];
    ora_philox4x64_10(ctr, key, out);
    uint64_t w = out[lane / 2];
    return (lane & 1) ? (uint32_t)(w >> 32) : (uint32_t)w;
}

uint32_t ora_lane(uint64_t seed, int64_t g, int64_t t, int32_t purpose, int32_t slot,
                  int64_t block, int32_t lane)
{
    return lane_of(seed, g, t, purpose, slot, block, lane);
}

/* Uniform on the open interval (0,1): the odd integer 2*(x>>9)+1 < 2^24 scaled by
 * 2^-24, exact in fp32. */
float ora_uniform(uint32_t x)
{
    uint32_t odd = 2u * (x >> 9) + 1u;
    return (float)odd * 0x1p-24f;
}

/* Standard Gumbel draw from a uniform, in fp64. */
double ora_gumbel(float u)
{
    return -log(-log((double)u));
}

/* ------------------------------------------------------------------------ */
/* bfloat16: round to nearest, ties to even, to 8 significant bits.           */
/* Written from the definition: the two bf16 neighbours of x are its         */
/* truncation toward zero and the next value away from zero; pick the nearer  */
/* and on a tie the one with an even last kept bit.                          */
/* ------------------------------------------------------------------------ */
uint16_t ora_bf16_bits(float x)
{
    uint32_t b;
    memcpy(&b, &x, 4);
    if (isnan(x))
        return (uint16_t)(((b >> 16) & 0x8000u) | 0x7FC0u);
    uint32_t down = b & 0xFFFF0000u;           /* toward zero */
    uint32_t rest = b & 0x0000FFFFu;           /* discarded part */
    uint32_t up = down + 0x00010000u;          /* next magnitude (may reach inf) */
    uint32_t pick;
    if (rest < 0x8000u)
        pick = down;
    else if (rest > 0x8000u)
        pick = up;
    else
        pick = ((down >> 16) & 1u) ? up : down;
    return (uint16_t)(pick >> 16);
}

float ora_bf16_round(float x)
{
    uint32_t b = (uint32_t)ora_bf16_bits(x) << 16;
    float y;
    memcpy(&y, &b, 4);
    return y;
}

/* Hidden-unit ReLU of the bf16 policies: max(x, 0) rounded to bf16.  A NaN
 * (of either sign) stays NaN, so that it reaches the logits; zero and every
 * negative value (including -0 and -inf) give +0; a positive value gives its
 * bf16 rounding.  Rounding to nearest is monotone and keeps the sign, so this
 * equals the ReLU of the rounded value. */
float ora_bf16_relu(float x)
{
    if (isnan(x))
        return x;
    if (!(x > 0.0f))
        return 0.0f;
    return ora_bf16_round(x);
}

/* ------------------------------------------------------------------------ */
/* exp_ref / tanh_ref: the fixed fp32 definitions used by the feature         */
/* dynamics (the environment's tanh must be reproducible bit for bit).        */
/* exp_ref: Cody-Waite reduction x = n*ln2 + r (ln2 split in a high part with  */
/* trailing zeros and a low part), degree-7 Taylor polynomial of e^r in Horner */
/* form with fused multiply-adds, exact scaling by 2^n.                        */
/* tanh_ref: |x| < 0.55 -> odd Taylor series x + x^3*p(x^2) through x^19;      */
/* 0.55 <= |x| <= 9.01 -> 1 - 2/(exp_ref(2|x|)+1) with the sign of x;          */
/* |x| > 9.01 -> +-1; NaN and signed zeros are returned unchanged.             */
/* ------------------------------------------------------------------------ */
float ora_exp_ref(float x)
{
    const float log2e = 0x1.715476p+0f;
    const float ln2_hi = 0x1.62e4p-1f;
    const float ln2_lo = 0x1.7f7d1cp-20f;
    float n = rintf(x * log2e);
    float r = fmaf(-n, ln2_hi, x);
    r = fmaf(-n, ln2_lo, r);
    /* 1/k! for k = 7..0 */
    float p = 0x1.a01a02p-13f;
    p = fmaf(p, r, 0x1.6c16c2p-10f);
    p = fmaf(p, r, 0x1.111112p-7f);
    p = fmaf(p, r, 0x1.555556p-5f);
    p = fmaf(p, r, 0x1.555556p-3f);
    p = fmaf(p, r, 0x1p-1f);
    p = fmaf(p, r, 0x1p+0f);
    p = fmaf(p, r, 0x1p+0f);
    return ldexpf(p, (int)n);
}

float ora_tanh_ref(float x)
{
    if (isnan(x) || x == 0.0f)
        return x;
    float ax = fabsf(x);
    if (ax > 9.01f)
        return copysignf(1.0f, x);
    if (ax < 0.55f) {
        float y = x * x;
        /* Taylor coefficients of (tanh(x) - x)/x^3 in powers of y = x^2 */
        float p = -0x1.f57d78p-13f;          /* -443861162/1856156927625 */
        p = fmaf(p, y, 0x1.355824p-11f);     /*  6404582/10854718875 */
        p = fmaf(p, y, -0x1.7da364p-10f);    /* -929569/638512875 */
        p = fmaf(p, y, 0x1.d6d3dp-9f);       /*  21844/6081075 */
        p = fmaf(p, y, -0x1.226e36p-7f);     /* -1382/155925 */
        p = fmaf(p, y, 0x1.664f48p-6f);      /*  62/2835 */
        p = fmaf(p, y, -0x1.ba1ba2p-5f);     /* -17/315 */
        p = fmaf(p, y, 0x1.111112p-3f);      /*  2/15 */
        p = fmaf(p, y, -0x1.555556p-2f);     /* -1/3 */
        float x3 = x * y;
        return fmaf(x3, p, x);
    }
    float e = ora_exp_ref(2.0f * ax);
    float t = 1.0f - 2.0f / (e + 1.0f);
    return copysignf(t, x);
}

void ora_tanh_range(uint32_t first_bits, int64_t n, float* out)
{
    for (int64_t i = 0; i < n; ++i) {
        uint32_t b = first_bits + (uint32_t)i;
        float x;
        memcpy(&x, &b, 4);
        out[i] = ora_tanh_ref(x);
    }
}

/* Largest ulp error of tanh_ref against fp64 tanh over a range of bit patterns
 * (finite inputs only); also reports the worst input. */
double ora_tanh_max_ulp(uint32_t first_bits, int64_t n, uint32_t* worst)
{
    double best = 0.0;
    for (int64_t i = 0; i < n; ++i) {
        uint32_t b = first_bits + (uint32_t)i;
        float x;
        memcpy(&x, &b, 4);
        if (!isfinite(x))
            continue;
        double ref = tanh((double)x);
        float got = ora_tanh_ref(x);
        float rf = (float)ref;
        /* ulp of the exact value, measured at fp32 precision */
        double ulp;
        if (rf == 0.0f)
            ulp = 0x1p-149;
        else {
            int ex;
            frexp(fabs(ref), &ex);
            ulp = ldexp(1.0, ex - 24);
            if (ulp < 0x1p-149)
                ulp = 0x1p-149;
        }
        double err = fabs((double)got - ref) / ulp;
        if (err > best) {
            best = err;
            if (worst)
                *worst = b;
        }
    }
    return best;
}

/* ------------------------------------------------------------------------ */
/* Meta-strategy sampling (the per-agent policy distribution of the example */
/* API, Appendix C.2): thresholds T_k = floor(C_k * 2^32) from the fp64      */
/* cumulative sum of sigma, T_{P-1} = 2^32; pid = min{m : x < T_m} with x the */
/* first lane of the (env, seat) draw.                                        */
/* ------------------------------------------------------------------------ */
int ora_meta_sample(const float* sigma, int32_t n_sigma, int32_t P, int64_t n_envs,
                    int32_t n_agents, uint64_t seed, int64_t env_offset, int32_t* out)
{
    if (P <= 0 || n_envs < 0 || n_agents <= 0 || (n_sigma != 1 && n_sigma != n_agents))
        return -1;
    uint64_t* T = (uint64_t*)malloc(sizeof(uint64_t) * (size_t)P * (size_t)n_sigma);
    if (!T)
        return -2;
    for (int r = 0; r < n_sigma; ++r) {
        const float* s = sigma + (size_t)r * P;
        double total = 0.0;
        for (int m = 0; m < P; ++m) {
            if (!isfinite(s[m]) || s[m] < 0.0f) {
                free(T);
                return -1;
            }
            total += (double)s[m];
        }
        if (!(total > 0.0)) {
            free(T);
            return -1;
        }
        double run = 0.0;
        for (int m = 0; m < P; ++m) {
            run += (double)s[m];
            double c = floor(run / total * 4294967296.0);
            if (c > 4294967296.0)
                c = 4294967296.0;
            T[(size_t)r * P + m] = (uint64_t)c;
        }
        T[(size_t)r * P + P - 1] = 4294967296ULL;
    }
    for (int64_t e = 0; e < n_envs; ++e) {
        for (int k = 0; k < n_agents; ++k) {
            const uint64_t* Tr = T + (size_t)(n_sigma == 1 ? 0 : k) * P;
            uint32_t x = lane_of(seed, env_offset + e, 0, PURPOSE_META, k, 0, 0);
            int m = 0;
            while (!((uint64_t)x < Tr[m]))
                ++m;
            out[e * n_agents + k] = m;
        }
    }
    free(T);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Meta-solver on the payoff table: the meta-update Comb_{t+1} ~ G(...) of    */
/* Sec. 3.1 with a fictitious-play solver (the FP meta-solver of the PSRO     */
/* experiments, Sec. 4.2; get_equilibrium of the example API, Appendix C.2).  */
/* The table is a two-player zero-sum game: the row side receives M[i][j],   */
/* the column side -M[i][j].  Simultaneous fictitious play: at iteration t   */
/* each side best-responds to the other's empirical play so far,             */
/*   i_t = first argmax_i v_i,  v = sum over s < t of M[:, j_s],             */
/*   j_t = first argmin_j w_j,  w = sum over s < t of M[i_s, :],             */
/* (fp64, one column / row added per iteration in iteration order), then     */
/* both play counts are incremented.  The average strategies are cx/T and    */
/* cy/T; gap = (max_i v_i - min_j w_j) / T after the last update is their    */
/* exploitability (the sum of both sides' best-response gains).  M must be   */
/* finite.                                                                   */
/* ------------------------------------------------------------------------ */
int ora_solve_fp(const double* M, int32_t P, int32_t T, int32_t* cx, int32_t* cy, double* gap)
{
    if (P <= 0 || T <= 0)
        return -1;
    double* v = (double*)calloc((size_t)P, sizeof(double));
    double* w = (double*)calloc((size_t)P, sizeof(double));
    if (!v || !w) {
        free(v);
        free(w);
        return -2;
    }
    memset(cx, 0, sizeof(int32_t) * (size_t)P);
    memset(cy, 0, sizeof(int32_t) * (size_t)P);
    for (int32_t t = 0; t < T; ++t) {
        int i = 0, j = 0;
        for (int k = 1; k < P; ++k) {
            if (v[k] > v[i])
                i = k;
            if (w[k] < w[j])
                j = k;
        }
        cx[i] += 1;
        cy[j] += 1;
        for (int k = 0; k < P; ++k) {
            v[k] = v[k] + M[(size_t)k * P + j];
            w[k] = w[k] + M[(size_t)i * P + k];
        }
    }
    double vmax = v[0], wmin = w[0];
    for (int k = 1; k < P; ++k) {
        if (v[k] > vmax)
            vmax = v[k];
        if (w[k] < wmin)
            wmin = w[k];
    }
    *gap = (vmax - wmin) / (double)T;
    free(v);
    free(w);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Configuration                                                             */
/* ------------------------------------------------------------------------ */
enum { ENV_MATRIX = 0, ENV_ITER = 1, ENV_PURSUIT = 2, ENV_FEATURE = 3 };
enum { POL_TABULAR = 0, POL_MLP_F32 = 1, POL_MLP_BF16 = 2 };

typedef struct {
    int32_t env_kind;
    int32_t n_agents;
    int32_t n_actions;
    int32_t grid;
    const int8_t* team;   /* [n_agents] +1 row side, -1 column side */
    const float* A;       /* [n_actions][n_actions] */
    int32_t d;
    int32_t init_mode;    /* 0 per env, 1 every env starts from global env 0's draw */
    const float* W;       /* [d][d] */
    const float* emb;     /* [n_agents][n_actions][d] */
    const float* u;       /* [d] */
    int32_t pol_kind;
    int32_t P;
    int32_t n_layers;
    int32_t horizon;
    const int32_t* dims;  /* [n_layers+1] */
    const float* const* Wl;  /* n_layers pointers, [P][out][in] */
    const float* const* bl;  /* n_layers pointers, [P][out] (NULL entries = zero) */
    const float* tab;     /* [P][n_actions] */
    uint64_t seed;
    int64_t env_offset;
} ora_config;

/* Environment state of one env. */
typedef struct {
    int t;
    /* iterated matrix: joint actions at lags 1..4 (a0*3+a1), -1 = before start */
    int hist[4];
    /* pursuit */
    int pc, ec, done;
    /* feature */
    float* s;
} env_state;

/* ---- observations ------------------------------------------------------- */

/* Iterated matrix game: for lag 1..4 (most recent first) the one-hot of the
 * observer's own action, then of the opponent's; zeros before the start. */
static void obs_iter(const env_state* st, int seat, double* obs)
{
    for (int i = 0; i < 24; ++i)
        obs[i] = 0.0;
    for (int lag = 0; lag < 4; ++lag) {
        int j = st->hist[lag];
        if (j < 0)
            continue;
        int a0 = j / 3, a1 = j % 3;
        int own = seat == 0 ? a0 : a1;
        int other = seat == 0 ? a1 : a0;
        obs[lag * 6 + own] = 1.0;
        obs[lag * 6 + 3 + other] = 1.0;
    }
}

/* Pursuit: egocentric 5x5 window with wrap-around, offsets dy, dx in [-2, 2];
 * channel 0 pursuer present, 1 evader present, 2 the observer itself (the
 * centre cell).  Index ((dy+2)*5 + (dx+2))*3 + channel. */
static void obs_pursuit(const env_state* st, int seat, int grid, double* obs)
{
    for (int i = 0; i < 75; ++i)
        obs[i] = 0.0;
    int self = seat == 0 ? st->pc : st->ec;
    int sx = self % grid, sy = self / grid;
    for (int dy = -2; dy <= 2; ++dy) {
        for (int dx = -2; dx <= 2; ++dx) {
            int x = ((sx + dx) % grid + grid) % grid;
            int y = ((sy + dy) % grid + grid) % grid;
            int cell = y * grid + x;
            int base = ((dy + 2) * 5 + (dx + 2)) * 3;
            if (cell == st->pc)
                obs[base + 0] = 1.0;
            if (cell == st->ec)
                obs[base + 1] = 1.0;
            if (dx == 0 && dy == 0)
                obs[base + 2] = 1.0;
        }
    }
}

/* ---- policies ----------------------------------------------------------- */

static float bias_of(const ora_config* c, int l, int p, int j)
{
    if (!c->bl || !c->bl[l])
        return 0.0f;
    return c->bl[l][(size_t)p * c->dims[l + 1] + j];
}

/* fp32-weight MLP evaluated in fp64: h = relu(W x + b) per hidden layer, logits
 * = W x + b on the last one, rounded to fp32 at the end. */
static void mlp_f32(const ora_config* c, int p, const double* obs, float* logits)
{
    int L = c->n_layers;
    int maxw = 0;
    for (int l = 0; l <= L; ++l)
        if (c->dims[l] > maxw)
            maxw = c->dims[l];
    double* x = (double*)malloc(sizeof(double) * maxw);
    double* y = (double*)malloc(sizeof(double) * maxw);
    for (int i = 0; i < c->dims[0]; ++i)
        x[i] = obs[i];
    for (int l = 0; l < L; ++l) {
        int in = c->dims[l], out = c->dims[l + 1];
        const float* Wp = c->Wl[l] + (size_t)p * out * in;
        for (int j = 0; j < out; ++j) {
            double acc = 0.0;
            for (int k = 0; k < in; ++k)
                acc += (double)Wp[(size_t)j * in + k] * x[k];
            acc += (double)bias_of(c, l, p, j);
            if (l + 1 < L && acc < 0.0)
                acc = 0.0;
            y[j] = acc;
        }
        double* t = x; x = y; y = t;
    }
    for (int a = 0; a < c->dims[L]; ++a)
        logits[a] = (float)x[a];
    free(x);
    free(y);
}

/* bf16 MLP: the input and every hidden activation are rounded to bf16 (round to
 * nearest even); products of bf16 values are exact, the layer sum is formed in
 * fp64 and rounded to the fp32 accumulator, the fp32 bias is added in fp32;
 * hidden = ReLU of bf16(acc) (ora_bf16_relu); logits stay fp32. */
static void mlp_bf16(const ora_config* c, int p, const double* obs, float* logits)
{
    int L = c->n_layers;
    int maxw = 0;
    for (int l = 0; l <= L; ++l)
        if (c->dims[l] > maxw)
            maxw = c->dims[l];
    float* x = (float*)malloc(sizeof(float) * maxw);
    float* y = (float*)malloc(sizeof(float) * maxw);
    for (int i = 0; i < c->dims[0]; ++i)
        x[i] = ora_bf16_round((float)obs[i]);
    for (int l = 0; l < L; ++l) {
        int in = c->dims[l], out = c->dims[l + 1];
        const float* Wp = c->Wl[l] + (size_t)p * out * in;
        for (int j = 0; j < out; ++j) {
            double acc = 0.0;
            for (int k = 0; k < in; ++k)
                acc += (double)ora_bf16_round(Wp[(size_t)j * in + k]) * (double)x[k];
            float a32 = (float)acc + bias_of(c, l, p, j);
            if (l + 1 < L)
                y[j] = ora_bf16_relu(a32);
            else
                y[j] = a32;
        }
        float* t = x; x = y; y = t;
    }
    for (int a = 0; a < c->dims[L]; ++a)
        logits[a] = x[a];
    free(x);
    free(y);
}

static int obs_dim(const ora_config* c)
{
    switch (c->env_kind) {
    case ENV_ITER: return 24;
    case ENV_PURSUIT: return 75;
    case ENV_FEATURE: return c->d;
    default: return 0;
    }
}

static void make_obs(const ora_config* c, const env_state* st, int seat, double* obs)
{
    switch (c->env_kind) {
    case ENV_ITER: obs_iter(st, seat, obs); break;
    case ENV_PURSUIT: obs_pursuit(st, seat, c->grid, obs); break;
    case ENV_FEATURE:
        for (int k = 0; k < c->d; ++k)
            obs[k] = (double)st->s[k];
        break;
    default: break;
    }
}

static void policy_logits(const ora_config* c, int p, const double* obs, float* logits)
{
    if (c->pol_kind == POL_TABULAR) {
        for (int a = 0; a < c->n_actions; ++a)
            logits[a] = c->tab[(size_t)p * c->n_actions + a];
    } else if (c->pol_kind == POL_MLP_F32) {
        mlp_f32(c, p, obs, logits);
    } else {
        mlp_bf16(c, p, obs, logits);
    }
}

/* ---- environments ------------------------------------------------------- */

static void reset_env(const ora_config* c, int64_t g, env_state* st)
{
    st->t = 0;
    for (int i = 0; i < 4; ++i)
        st->hist[i] = -1;
    st->done = 0;
    int64_t gr = c->init_mode == 1 ? 0 : g;
    if (c->env_kind == ENV_PURSUIT) {
        /* G x G torus: pursuer floor(lane0 * G^2 / 2^32) (the top 6 bits of
         * lane 0 when G = 8), evader pursuer + 1 + floor(lane1 * (G^2 - 1) / 2^32)
         * mod G^2, so the two start on distinct cells */
        int cells = c->grid * c->grid;
        uint32_t x0 = lane_of(c->seed, gr, 0, PURPOSE_RESET, 0, 0, 0);
        uint32_t x1 = lane_of(c->seed, gr, 0, PURPOSE_RESET, 0, 0, 1);
        st->pc = (int)(((uint64_t)x0 * (uint64_t)cells) >> 32);
        uint32_t shift = (uint32_t)(((uint64_t)x1 * (uint64_t)(cells - 1)) >> 32);
        st->ec = (int)((st->pc + 1 + shift) % (uint32_t)cells);
    } else if (c->env_kind == ENV_FEATURE) {
        for (int k = 0; k < c->d; ++k) {
            uint32_t x = lane_of(c->seed, gr, 0, PURPOSE_RESET, 0, k / 8, k % 8);
            int32_t odd = (int32_t)(2u * (x >> 9) + 1u);
            st->s[k] = (float)(odd - (1 << 23)) * 0x1p-23f;
        }
    }
}

/* Torus move: 0 stay, 1 up (y-1), 2 down (y+1), 3 left (x-1), 4 right (x+1). */
static int move_cell(int cell, int a, int grid)
{
    int x = cell % grid, y = cell / grid;
    if (a == 1) y = (y + grid - 1) % grid;
    else if (a == 2) y = (y + 1) % grid;
    else if (a == 3) x = (x + grid - 1) % grid;
    else if (a == 4) x = (x + 1) % grid;
    return y * grid + x;
}

/* One environment step; writes the per-seat rewards (fp32). */
static void env_step(const ora_config* c, env_state* st, const int* act, float* r)
{
    int n = c->n_agents;
    for (int k = 0; k < n; ++k)
        r[k] = 0.0f;
    if (c->env_kind == ENV_MATRIX || c->env_kind == ENV_ITER) {
        float v = c->A[act[0] * c->n_actions + act[1]];
        r[0] = v;
        r[1] = -v;
        if (c->env_kind == ENV_ITER) {
            for (int i = 3; i > 0; --i)
                st->hist[i] = st->hist[i - 1];
            st->hist[0] = act[0] * 3 + act[1];
        }
    } else if (c->env_kind == ENV_PURSUIT) {
        if (st->done)
            return;
        int p0 = st->pc, e0 = st->ec;
        int p1 = move_cell(p0, act[0], c->grid);
        int e1 = move_cell(e0, act[1], c->grid);
        st->pc = p1;
        st->ec = e1;
        if (p1 == e1 || (p1 == e0 && e1 == p0)) {
            st->done = 1;
            r[0] = 1.0f;
            r[1] = -1.0f;
        }
    } else if (c->env_kind == ENV_FEATURE) {
        int d = c->d, A = c->n_actions;
        float* nxt = (float*)malloc(sizeof(float) * d);
        for (int k = 0; k < d; ++k) {
            float acc = 0.0f;
            for (int cc = 0; cc < d; ++cc)
                acc = fmaf(c->W[(size_t)k * d + cc], st->s[cc], acc);
            float pre = acc;
            for (int j = 0; j < n; ++j)
                pre = pre + c->emb[((size_t)j * A + act[j]) * d + k];
            nxt[k] = ora_tanh_ref(pre);
        }
        float rr = 0.0f;
        for (int k = 0; k < d; ++k)
            rr = fmaf(c->u[k], nxt[k], rr);
        memcpy(st->s, nxt, sizeof(float) * d);
        free(nxt);
        for (int j = 0; j < n; ++j)
            r[j] = c->team[j] > 0 ? rr : -rr;
    }
    st->t += 1;
}

static int live(const ora_config* c, const env_state* st)
{
    return !(c->env_kind == ENV_PURSUIT && st->done);
}

static void snapshot(const ora_config* c, const env_state* st, void* dst, int64_t i)
{
    if (c->env_kind == ENV_ITER) {
        uint16_t h = 0;
        for (int lag = 0; lag < 4; ++lag) {
            int j = st->hist[lag] < 0 ? 15 : st->hist[lag];
            h |= (uint16_t)(j << (4 * lag));
        }
        ((uint16_t*)dst)[i] = h;
    } else if (c->env_kind == ENV_PURSUIT) {
        uint8_t* b = (uint8_t*)dst + i * 3;
        b[0] = (uint8_t)st->pc;
        b[1] = (uint8_t)st->ec;
        b[2] = (uint8_t)st->done;
    } else if (c->env_kind == ENV_FEATURE) {
        memcpy((float*)dst + i * c->d, st->s, sizeof(float) * c->d);
    }
}

int64_t ora_state_elems(int32_t env_kind, int32_t d)
{
    switch (env_kind) {
    case ENV_ITER: return 1;      /* uint16 */
    case ENV_PURSUIT: return 3;   /* uint8 x3 */
    case ENV_FEATURE: return d;   /* float */
    default: return 0;
    }
}

/*
 * Roll out a list of envs.  For env index e (local to the batch, global g =
 * env_offset + e) the seats play policies pids[i][k].
 *
 * forced (optional) is the other implementation's action log [H][n_sel][n_agents].
 * At every live step the oracle draws its own action (Gumbel-max on fp64
 * perturbed logits z_a = l_a + g_a, lowest index on ties).  If a forced action
 * differs, the oracle's own top-two margin is compared with
 * tol * max(1, |z_top|): within it the step counts as a near-tie flip and the
 * forced action is adopted; otherwise the step is a failure (also adopted, so
 * that the rest of the run stays comparable) and the first one is recorded.
 * Steps whose margin is within the tolerance count as near ties either way.
 *
 * Outputs (each optional): returns [n_sel][n_agents] fp32 (summed in step
 * order), actions [H][n_sel][n_agents] (the actions taken; 255 where the env is
 * finished), logits [H][n_sel][n_agents][A] (0 where finished), states
 * [H][n_sel][...] (the state before step t).
 * stats[0] near ties, [1] flips, [2] failures, [3] live agent-frames,
 * [4..6] first failure (t, sel index, seat) or -1.
 * Returns 0, or -1 on bad input, -2 on a NaN logit.
 */
int ora_rollout(const ora_config* c, int64_t n_sel, const int64_t* env_idx,
                const int32_t* pids, const uint8_t* forced, double tol,
                float* returns, uint8_t* actions, float* logits, void* states,
                int64_t* stats, float* step_rewards)
{
    int n = c->n_agents, A = c->n_actions, H = c->horizon;
    if (n <= 0 || A <= 0 || A > 64 || H < 0 || (c->pol_kind != POL_TABULAR && c->dims[c->n_layers] != A))
        return -1;
    if (c->pol_kind != POL_TABULAR && c->dims[0] != obs_dim(c))
        return -1;
    for (int i = 0; i < 7; ++i)
        stats[i] = (i >= 4) ? -1 : 0;
    int od = obs_dim(c);
    double* obs = (double*)malloc(sizeof(double) * (od > 0 ? od : 1));
    float* l = (float*)malloc(sizeof(float) * A);
    int* act = (int*)malloc(sizeof(int) * n);
    float* r = (float*)malloc(sizeof(float) * n);
    env_state st;
    st.s = (float*)malloc(sizeof(float) * (c->d > 0 ? c->d : 1));
    int64_t se = ora_state_elems(c->env_kind, c->d);
    int rc = 0;
    for (int64_t i = 0; i < n_sel && rc == 0; ++i) {
        int64_t g = c->env_offset + env_idx[i];
        const int32_t* pp = pids + i * n;
        for (int k = 0; k < n; ++k) {
            if (pp[k] < 0 || pp[k] >= c->P) {
                rc = -1;
                break;
            }
        }
        if (rc)
            break;
        reset_env(c, g, &st);
        float* G = returns ? returns + i * n : NULL;
        if (G)
            for (int k = 0; k < n; ++k)
                G[k] = 0.0f;
        for (int t = 0; t < H; ++t) {
            if (states && se > 0) {
                int64_t idx = (int64_t)t * n_sel + i;
                snapshot(c, &st, states, idx);
            }
            int alive = live(c, &st);
            for (int k = 0; k < n; ++k) {
                size_t aidx = ((size_t)t * n_sel + i) * n + k;
                if (!alive) {
                    act[k] = 0;
                    if (actions)
                        actions[aidx] = 255;
                    if (logits)
                        for (int a = 0; a < A; ++a)
                            logits[aidx * A + a] = 0.0f;
                    continue;
                }
                stats[3] += 1;
                make_obs(c, &st, k, obs);
                policy_logits(c, pp[k], obs, l);
                double z1 = -INFINITY, z2 = -INFINITY;
                int best = 0;
                for (int a = 0; a < A; ++a) {
                    if (isnan(l[a])) {
                        rc = -2;
                        break;
                    }
                    uint32_t x = lane_of(c->seed, g, t, PURPOSE_ACTION, k, a / 8, a % 8);
                    double z = (double)l[a] + ora_gumbel(ora_uniform(x));
                    if (z > z1) {
                        z2 = z1;
                        z1 = z;
                        best = a;
                    } else if (z > z2) {
                        z2 = z;
                    }
                }
                if (rc)
                    break;
                double scale = fabs(z1) > 1.0 ? fabs(z1) : 1.0;
                int near = (z1 - z2) <= tol * scale;
                if (near)
                    stats[0] += 1;
                int chosen = best;
                if (forced) {
                    int fa = forced[aidx];
                    if (fa != best) {
                        if (near) {
                            stats[1] += 1;
                        } else {
                            stats[2] += 1;
                            if (stats[4] < 0) {
                                stats[4] = t;
                                stats[5] = i;
                                stats[6] = k;
                            }
                        }
                        if (fa >= 0 && fa < A)
                            chosen = fa;
                    }
                }
                act[k] = chosen;
                if (actions)
                    actions[aidx] = (uint8_t)chosen;
                if (logits)
                    for (int a = 0; a < A; ++a)
                        logits[aidx * A + a] = l[a];
            }
            if (rc)
                break;
            env_step(c, &st, act, r);
            if (G)
                for (int k = 0; k < n; ++k)
                    G[k] = G[k] + r[k];
            if (step_rewards)
                for (int k = 0; k < n; ++k)
                    step_rewards[((size_t)t * n_sel + i) * n + k] = r[k];
        }
    }
    free(obs);
    free(l);
    free(act);
    free(r);
    free(st.s);
    return rc;
}

/* ---- small pieces exposed for unit pins --------------------------------- */

void ora_obs_iter(const int32_t hist[4], int32_t seat, double* out)
{
    env_state st;
    for (int i = 0; i < 4; ++i)
        st.hist[i] = hist[i];
    obs_iter(&st, seat, out);
}

void ora_obs_pursuit(int32_t pc, int32_t ec, int32_t seat, int32_t grid, double* out)
{
    env_state st;
    st.pc = pc;
    st.ec = ec;
    st.done = 0;
    obs_pursuit(&st, seat, grid, out);
}

/* Pursuit step on explicit cells; returns 1 on capture. */
int ora_pursuit_step(int32_t* pc, int32_t* ec, int32_t a0, int32_t a1, int32_t grid)
{
    int p0 = *pc, e0 = *ec;
    int p1 = move_cell(p0, a0, grid), e1 = move_cell(e0, a1, grid);
    *pc = p1;
    *ec = e1;
    return (p1 == e1 || (p1 == e0 && e1 == p0)) ? 1 : 0;
}

void ora_pursuit_reset(uint64_t seed, int64_t g, int32_t grid, int32_t* pc, int32_t* ec)
{
    ora_config c;
    memset(&c, 0, sizeof(c));
    c.env_kind = ENV_PURSUIT;
    c.grid = grid;
    c.seed = seed;
    env_state st;
    reset_env(&c, g, &st);
    *pc = st.pc;
    *ec = st.ec;
}

void ora_feature_reset(uint64_t seed, int64_t g, int32_t d, float* s)
{
    ora_config c;
    memset(&c, 0, sizeof(c));
    c.env_kind = ENV_FEATURE;
    c.d = d;
    c.seed = seed;
    env_state st;
    st.s = s;
    reset_env(&c, g, &st);
}

/* Feature-dynamics step from an explicit state: s' = tanh_ref(W s + sum_j
 * emb[j][a_j]) with the fp32 sums in the fixed order, reward u . s'. */
float ora_feature_step(const ora_config* c, const float* s, const int32_t* act, float* s_out)
{
    env_state st;
    st.s = (float*)malloc(sizeof(float) * c->d);
    memcpy(st.s, s, sizeof(float) * c->d);
    st.t = 0;
    int* a = (int*)malloc(sizeof(int) * c->n_agents);
    float* r = (float*)malloc(sizeof(float) * c->n_agents);
    for (int j = 0; j < c->n_agents; ++j)
        a[j] = act[j];
    env_step(c, &st, a, r);
    memcpy(s_out, st.s, sizeof(float) * c->d);
    float out = 0.0f;
    for (int j = 0; j < c->n_agents; ++j)
        if (c->team[j] > 0) {
            out = r[j];
            break;
        }
    free(st.s);
    free(a);
    free(r);
    return out;
}

/* Policy logits for one observation (fp64 input). */
int ora_policy_logits(const ora_config* c, int32_t p, const double* obs, float* out)
{
    if (p < 0 || p >= c->P)
        return -1;
    policy_logits(c, p, obs, out);
    return 0;
}

/* bf16 bit patterns of a contiguous range of fp32 bit patterns (exhaustive pins). */
void ora_bf16_range(uint32_t first_bits, int64_t n, uint16_t* out)
{
    for (int64_t i = 0; i < n; ++i) {
        uint32_t b = first_bits + (uint32_t)i;
        float x;
        memcpy(&x, &b, 4);
        out[i] = ora_bf16_bits(x);
    }
}

/* Uniforms for a contiguous range of 32-bit lanes. */
void ora_uniform_range(uint32_t first, int64_t n, float* out)
{
    for (int64_t i = 0; i < n; ++i)
        out[i] = ora_uniform(first + (uint32_t)i);
}

/* exp_ref over an array (pins). */
void ora_exp_many(const float* x, int64_t n, float* out)
{
    for (int64_t i = 0; i < n; ++i)
        out[i] = ora_exp_ref(x[i]);
}

void ora_tanh_many(const float* x, int64_t n, float* out)
{
    for (int64_t i = 0; i < n; ++i)
        out[i] = ora_tanh_ref(x[i]);
}
