// Meta-solver on the payoff table and meta-strategy sampling from device
// weights: the meta-update Comb_{t+1} ~ G(...) of Sec. 3.1 with the
// fictitious-play solver of the PSRO experiments (Sec. 4.2), closed on the GPU
// (table -> game -> fictitious play -> sigma -> meta-sample -> next rollout).
#include "device.hpp"
#include "internal.hpp"

namespace malib {

// M[i][j] = the mean of cell (i, j), sum * 2^-32 / count as the table read-back
// computes it; 0 where the cell has no simulations.
__global__ void payoff_matrix_kernel(const unsigned long long* __restrict__ sum,
                                     const unsigned long long* __restrict__ cnt, int PP,
                                     double* __restrict__ M)
{
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= PP)
        return;
    const long long c = (long long)cnt[i];
    M[i] = c > 0 ? ldexp((double)(long long)sum[i], -32) / (double)c : 0.0;
}

hipError_t launch_payoff_matrix(const unsigned long long* sum, const unsigned long long* cnt,
                                int P, double* M, hipStream_t s)
{
    const int PP = P * P;
    payoff_matrix_kernel<<<(PP + 255) / 256, 256, 0, s>>>(sum, cnt, PP, M);
    return hipGetLastError();
}

constexpr int kSolveLdsP = 128;   // up to this P the game sits in LDS
static_assert(kMaxP <= 4 * 64, "the solver keeps at most 4 policies per lane");

// A lane's fp64 value moved across lanes by one DPP pattern (both halves).
// Only patterns that stay inside a 16-lane row are used, so every lane has a
// source.
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double x)
{
    const long long b = __double_as_longlong(x);
    const int lo = __builtin_amdgcn_mov_dpp((int)b, CTRL, 0xF, 0xF, false);
    const int hi = __builtin_amdgcn_mov_dpp((int)(b >> 32), CTRL, 0xF, 0xF, false);
    return __longlong_as_double(((long long)hi << 32) | (unsigned int)lo);
}

// The same across rows: lanes of the rows in ROWS take the pattern's source,
// the others keep their own value.
template <int CTRL, int ROWS>
__device__ __forceinline__ double dpp_f64_rows(double x)
{
    const long long b = __double_as_longlong(x);
    const int lo = __builtin_amdgcn_update_dpp((int)b, (int)b, CTRL, ROWS, 0xF, false);
    const int hi =
        __builtin_amdgcn_update_dpp((int)(b >> 32), (int)(b >> 32), CTRL, ROWS, 0xF, false);
    return __longlong_as_double(((long long)hi << 32) | (unsigned int)lo);
}

__device__ __forceinline__ double readlane_f64(double x, int l)
{
    const long long b = __double_as_longlong(x);
    const int lo = __builtin_amdgcn_readlane((int)b, l);
    const int hi = __builtin_amdgcn_readlane((int)(b >> 32), l);
    return __longlong_as_double(((long long)hi << 32) | (unsigned int)lo);
}

// DPP controls: swap neighbours, swap pairs in a quad, mirror each 8-lane
// half row, mirror each 16-lane row.  After the four steps every lane holds
// its row's result; two row broadcasts then combine the rows into lane 63.
constexpr int kDppQuadSwap1 = 0xB1;   // quad_perm [1, 0, 3, 2]
constexpr int kDppQuadSwap2 = 0x4E;   // quad_perm [2, 3, 0, 1]
constexpr int kDppHalfMirror = 0x141;
constexpr int kDppRowMirror = 0x140;
constexpr int kDppRowBcast15 = 0x142;   // lane 15 of each row to the next row
constexpr int kDppRowBcast31 = 0x143;   // lane 31 to the rows above it

// The largest of x and the smallest of y over the wavefront, the same in
// every lane; the two reductions interleave.  IEEE maxNum / minNum (one
// v_max_f64 / v_min_f64 each): a NaN never replaces a number, and which of
// +0 and -0 survives does not matter (the callers compare with ==, and take
// the winning policy's own sum afterwards).
__device__ __forceinline__ void wave_max_min(double& x, double& y)
{
    auto hi = [](double a, double b) { return __builtin_fmax(a, b); };
    auto lo = [](double a, double b) { return __builtin_fmin(a, b); };
    double dx = dpp_f64<kDppQuadSwap1>(x), dy = dpp_f64<kDppQuadSwap1>(y);
    x = hi(x, dx);
    y = lo(y, dy);
    dx = dpp_f64<kDppQuadSwap2>(x);
    dy = dpp_f64<kDppQuadSwap2>(y);
    x = hi(x, dx);
    y = lo(y, dy);
    dx = dpp_f64<kDppHalfMirror>(x);
    dy = dpp_f64<kDppHalfMirror>(y);
    x = hi(x, dx);
    y = lo(y, dy);
    dx = dpp_f64<kDppRowMirror>(x);
    dy = dpp_f64<kDppRowMirror>(y);
    x = hi(x, dx);
    y = lo(y, dy);
    // rows: lane 15 of rows 0 and 2 into rows 1 and 3, then lane 31 into
    // rows 2 and 3; lane 63 then holds the wavefront's result
    dx = dpp_f64_rows<kDppRowBcast15, 0xA>(x);
    dy = dpp_f64_rows<kDppRowBcast15, 0xA>(y);
    x = hi(x, dx);
    y = lo(y, dy);
    dx = dpp_f64_rows<kDppRowBcast31, 0xC>(x);
    dy = dpp_f64_rows<kDppRowBcast31, 0xC>(y);
    x = hi(x, dx);
    y = lo(y, dy);
    x = readlane_f64(x, 63);
    y = readlane_f64(y, 63);
}

// Simultaneous fictitious play on the zero-sum game with row payoff M
// (P x P, fp64; meant for finite entries, a NaN anywhere in v or w leaves the
// counts unspecified and sets gap to NaN): at iteration t, i_t = first argmax
// of v = sum over s < t of M[:, j_s] and j_t = first argmin of w = sum over
// s < t of M[i_s, :]; then both play counts are incremented and v, w gain
// column j_t and row i_t (one fp64 add per element per iteration, in
// iteration order).  One wavefront: lane l keeps policies k = l + 64 q,
// q < K, so an iteration needs no barrier.  The first argmax is the lowest k
// whose v equals the wavefront's maximum: the lowest q with a match, then the
// lowest lane (a ballot).  Writes sigma[0][k], sigma[1][k] = the play counts
// (weights for meta-sampling) and gap = (v[i] - w[j]) / T at the best
// responses i, j to the final sums.
template <int K, bool IN_LDS>
__global__ __launch_bounds__(64) void solve_fp_kernel(const double* __restrict__ M, int P, int T,
                                                      float* __restrict__ sigma,
                                                      double* __restrict__ gap)
{
    // the game with a padded row stride (column reads hit different banks)
    constexpr int LDS_DOUBLES = IN_LDS ? kSolveLdsP * (kSolveLdsP + 1) : 1;
    __shared__ double Ms[LDS_DOUBLES];
    const int lane = threadIdx.x;
    const int stride = IN_LDS ? P + 1 : P;
    const double* G = M;
    if constexpr (IN_LDS) {
        for (int e = lane; e < P * P; e += 64)
            Ms[(e / P) * stride + e % P] = M[e];
        __syncthreads();
        G = Ms;
    }
    double v[K], w[K];
    int cx[K], cy[K];
    bool mine[K];
    // slots past P start at -inf (v) and +inf (w) and keep adding finite
    // entries, so they never win a reduction and need no masking
#pragma unroll
    for (int q = 0; q < K; ++q) {
        mine[q] = lane + 64 * q < P;
        v[q] = mine[q] ? 0.0 : -INFINITY;
        w[q] = mine[q] ? 0.0 : INFINITY;
        cx[q] = 0;
        cy[q] = 0;
    }
    // first index of the best value (row side: largest v; column side:
    // smallest w); P - 1 when no policy matches (only NaN or infinite
    // entries can cause that, or a match past P)
    auto best = [&](int& i, int& j, double& vi, double& wj) {
        double lv = v[0], lw = w[0];
#pragma unroll
        for (int q = 1; q < K; ++q) {
            lv = __builtin_fmax(lv, v[q]);
            lw = __builtin_fmin(lw, w[q]);
        }
        wave_max_min(lv, lw);
        vi = lv;
        wj = lw;
        i = P - 1;
        j = P - 1;
        bool fi = false, fj = false;
#pragma unroll
        for (int q = 0; q < K; ++q) {
            const unsigned long long bi = __ballot(v[q] == vi);
            const unsigned long long bj = __ballot(w[q] == wj);
            if (!fi && bi) {
                i = 64 * q + __ffsll(bi) - 1;
                fi = true;
            }
            if (!fj && bj) {
                j = 64 * q + __ffsll(bj) - 1;
                fj = true;
            }
        }
        i = i < P ? i : P - 1;
        j = j < P ? j : P - 1;
    };
    for (int t = 0; t < T; ++t) {
        int i, j;
        double vi, wj;
        best(i, j, vi, wj);
        // every slot reads (a slot past P reads policy P - 1 and is never
        // looked at), so all loads issue before the first add waits
#pragma unroll
        for (int q = 0; q < K; ++q) {
            const int k = lane + 64 * q;
            const int kc = mine[q] ? k : P - 1;
            cx[q] += k == i;
            cy[q] += k == j;
            v[q] = v[q] + G[kc * stride + j];
            w[q] = w[q] + G[i * stride + kc];
        }
    }
#pragma unroll
    for (int q = 0; q < K; ++q) {
        if (mine[q]) {
            sigma[lane + 64 * q] = (float)cx[q];
            sigma[P + lane + 64 * q] = (float)cy[q];
        }
    }
    if (gap) {
        bool nan = false;
#pragma unroll
        for (int q = 0; q < K; ++q)
            nan = nan || (mine[q] && (__builtin_isnan(v[q]) || __builtin_isnan(w[q])));
        const bool any_nan = __ballot(nan) != 0ull;
        int i, j;
        double vi, wj;
        best(i, j, vi, wj);
        // the sums at the chosen indices themselves (of +0 and -0, the
        // reductions may keep either)
        double vs = v[0], ws = w[0];
#pragma unroll
        for (int q = 1; q < K; ++q) {
            vs = q == (i >> 6) ? v[q] : vs;
            ws = q == (j >> 6) ? w[q] : ws;
        }
        vi = __shfl(vs, i & 63);
        wj = __shfl(ws, j & 63);
        if (lane == 0)
            *gap = any_nan ? (double)NAN : (vi - wj) / (double)T;
    }
}

hipError_t launch_solve_fp(const double* M, int P, int T, float* sigma, double* gap,
                           hipStream_t s)
{
    if (P < 1 || P > kMaxP || T < 1)
        return hipErrorInvalidValue;
    if (P <= 64)
        solve_fp_kernel<1, true><<<1, 64, 0, s>>>(M, P, T, sigma, gap);
    else if (P <= kSolveLdsP)
        solve_fp_kernel<2, true><<<1, 64, 0, s>>>(M, P, T, sigma, gap);
    else
        solve_fp_kernel<4, false><<<1, 64, 0, s>>>(M, P, T, sigma, gap);
    return hipGetLastError();
}

// Aggregate payoffs of a meta-strategy pair (the PSRO convergence judgement):
// x, y = the weight rows sigma[0], sigma[1] normalized in fp64 (sequential
// sums); u = M y and v = x^T M, each entry a sequential fp64 sum of rounded
// products (thread k forms u[k] over row k and v[k] over column k); nash =
// x^T u (sequential).  out = {nash, -nash, u[br_row], -v[br_col],
// improvement}, where improvement is the larger best-response gain of the
// sides whose br is >= 0 (a side with br = -1 gives NaN).
__global__ __launch_bounds__(kMaxP) void aggregate_kernel(const double* __restrict__ M, int P,
                                                          const float* __restrict__ sigma,
                                                          int br_row, int br_col,
                                                          double* __restrict__ out)
{
    __shared__ double x[kMaxP], y[kMaxP], u[kMaxP];
    __shared__ double S[2], vbr;
    const int k = threadIdx.x;
    if (k == 0) {
        double a = 0.0, b = 0.0;
#pragma unroll 16
        for (int m = 0; m < P; ++m)
            a += (double)sigma[m];
#pragma unroll 16
        for (int m = 0; m < P; ++m)
            b += (double)sigma[P + m];
        S[0] = a;
        S[1] = b;
    }
    __syncthreads();
    if (k < P) {
        x[k] = (double)sigma[k] / S[0];
        y[k] = (double)sigma[P + k] / S[1];
    }
    __syncthreads();
    if (k < P) {
        // (unrolled so that the loads run ahead of the dependent adds)
        double acc = 0.0;
#pragma unroll 16
        for (int j = 0; j < P; ++j)
            acc = acc + M[(size_t)k * P + j] * y[j];
        u[k] = acc;
        double accv = 0.0;
#pragma unroll 16
        for (int i = 0; i < P; ++i)
            accv = accv + x[i] * M[(size_t)i * P + k];
        if (k == br_col)
            vbr = accv;
    }
    __syncthreads();
    if (k == 0) {
        double nash = 0.0;
#pragma unroll 16
        for (int i = 0; i < P; ++i)
            nash = nash + x[i] * u[i];
        const double wr = br_row >= 0 ? u[br_row] : (double)NAN;
        const double wc = br_col >= 0 ? -vbr : (double)NAN;
        double imp = (double)NAN;
        if (br_row >= 0)
            imp = wr - nash;
        if (br_col >= 0) {
            const double g = wc - (-nash);
            imp = (br_row < 0 || g > imp) ? g : imp;
        }
        out[0] = nash;
        out[1] = -nash;
        out[2] = wr;
        out[3] = wc;
        out[4] = imp;
    }
}

hipError_t launch_aggregate(const double* M, int P, const float* sigma, int br_row, int br_col,
                            double* out, hipStream_t s)
{
    aggregate_kernel<<<1, kMaxP, 0, s>>>(M, P, sigma, br_row, br_col, out);
    return hipGetLastError();
}

// ------------------------------------------------------------------ alpha-rank
//
// Single-population alpha-rank (Omidshafiei et al., 2019; the meta-solver the
// paper lists beside fictitious play for PSRO, Sec. 4.2, Table 3) on the
// table's game made symmetric by a meeting on each side: a mutant s in a
// population of r has fitness advantage u = alpha (M[s][r] - M[r][s]); its
// fixation probability in a population of m is rho(u) = (1 - e^-u) /
// (1 - e^-mu) (1/m at u = 0), and the chain moves r -> s with probability
// rho / (P - 1).  The stationary distribution comes from the
// Grassmann-Taksar-Heyman elimination, which uses only the off-diagonal
// transition probabilities and never subtracts, so small probabilities keep
// their relative accuracy: for n = P-1 .. 1, S = sum_{j<n} A[n][j],
// A[i][n] /= S and A[i][j] += A[i][n] A[n][j] for i, j < n; then pi_0 = 1,
// pi_j = sum_{i<j} pi_i A[i][j], normalized.  One workgroup of 1024 threads;
// the matrix in LDS for P <= kArLdsMax, else in the caller's workspace.

constexpr int kArThreads = 1024;
constexpr int kArLdsMax = 128;

__device__ __forceinline__ double ar_fixation(double u, int m)
{
    if (u == 0.0)
        return 1.0 / m;
    if (u > 0.0)
        return expm1(-u) / expm1(-m * u);
    // u < 0: e^((m-1) u) taken out, so that the ratio underflows gracefully
    const double v = -u;
    return exp(-(m - 1) * v) * (expm1(-v) / expm1(-m * v));
}

// Sum of one value per thread over the workgroup (fixed shuffle/LDS order).
__device__ __forceinline__ double ar_block_sum(double v, double* red)
{
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1)
        v += __shfl_xor(v, off, 64);
    __syncthreads();        // red is reused
    if (lane == 0)
        red[wave] = v;
    __syncthreads();
    double t = 0.0;
#pragma unroll
    for (int w = 0; w < kArThreads / 64; ++w)
        t += red[w];
    return t;
}

template <bool IN_LDS>
__global__ __launch_bounds__(kArThreads) void alpharank_kernel(const double* __restrict__ M,
                                                               int P, double alpha, int m,
                                                               double* __restrict__ work,
                                                               double* __restrict__ pi,
                                                               float* __restrict__ sigma)
{
    __shared__ double lds[IN_LDS ? kArLdsMax * (kArLdsMax + 1) : 1];
    __shared__ double red[kArThreads / 64];
    __shared__ double s_pi[kMaxP];
    double* A = IN_LDS ? lds : work;
    const int ld = IN_LDS ? P + 1 : P;      // odd stride in LDS: column reads spread over banks
    const int tid = threadIdx.x;
    // ---- the chain's off-diagonal transition probabilities
    const double mut = P > 1 ? 1.0 / (P - 1) : 0.0;
    for (int idx = tid; idx < P * P; idx += kArThreads) {
        const int r = idx / P, c = idx - r * P;
        double v = 0.0;
        if (r != c)
            v = ar_fixation(alpha * (M[(size_t)c * P + r] - M[(size_t)r * P + c]), m) * mut;
        A[(size_t)r * ld + c] = v;
    }
    __syncthreads();
    // ---- elimination, states P-1 .. 1; thread (ti, tj) of a 32 x 32 grid
    // updates A[i][j] for i = ti mod 32, j = tj mod 32
    const int ti = tid >> 5, tj = tid & 31;
    for (int n = P - 1; n >= 1; --n) {
        const double S = ar_block_sum(tid < n ? A[(size_t)n * ld + tid] : 0.0, red);
        for (int i = tid; i < n; i += kArThreads)
            A[(size_t)i * ld + n] /= S;
        __syncthreads();
        for (int i = ti; i < n; i += 32) {
            const double ain = A[(size_t)i * ld + n];
            for (int j = tj; j < n; j += 32)
                A[(size_t)i * ld + j] += ain * A[(size_t)n * ld + j];
        }
        __syncthreads();
    }
    // ---- back substitution, then normalization
    if (tid == 0)
        s_pi[0] = 1.0;
    __syncthreads();
    for (int j = 1; j < P; ++j) {
        const double v = ar_block_sum(tid < j ? s_pi[tid] * A[(size_t)tid * ld + j] : 0.0, red);
        if (tid == 0)
            s_pi[j] = v;
        __syncthreads();
    }
    const double total = ar_block_sum(tid < P ? s_pi[tid] : 0.0, red);
    if (tid < P) {
        const double x = s_pi[tid] / total;
        pi[tid] = x;
        if (sigma) {
            sigma[tid] = (float)x;
            sigma[P + tid] = (float)x;
        }
    }
}

bool alpharank_needs_work(int P)
{
    return P > kArLdsMax;
}

hipError_t launch_alpharank(const double* M, int P, double alpha, int m, double* work,
                            double* pi, float* sigma, hipStream_t s)
{
    if (P > kMaxP || P > kArThreads || (P > kArLdsMax && !work))
        return hipErrorInvalidValue;
    if (P <= kArLdsMax)
        alpharank_kernel<true><<<1, kArThreads, 0, s>>>(M, P, alpha, m, nullptr, pi, sigma);
    else
        alpharank_kernel<false><<<1, kArThreads, 0, s>>>(M, P, alpha, m, work, pi, sigma);
    return hipGetLastError();
}

// ------------------------------------------------------------------ LP solver
//
// The zero-sum meta-game's exact equilibrium (the LP solver of the PSRO
// experiments, Sec. 4.2) by the primal simplex method on the column side's
// problem after a shift that makes every payoff positive: with
// M' = M - min(M) + 1, maximize sum_j w_j subject to M' w <= 1, w >= 0.  The
// origin is feasible (slack basis).  At the optimum the column side's
// strategy is y = w / sum w, the row side's x = u / sum u with u the slack
// columns' reduced costs (the dual solution), and the value is
// 1 / sum w + min(M) - 1.  The entering column is the most negative reduced
// cost (Dantzig); after kLpDegenerate consecutive degenerate pivots (zero
// ratio) the solver switches to Bland's rule (the lowest entering column, the
// lowest basic variable among tied ratios), which cannot cycle, until a pivot
// makes progress again.  One workgroup:
// the tableau [P+1][2P+1] (fp64) in LDS for P <= kLpLdsMax, else in the
// caller's workspace; each pivot finds the entering column and the pivot row
// with block reductions, stages the column and the scaled pivot row in LDS
// and updates the other rows.

constexpr int kLpThreads = 1024;
constexpr int kLpLdsMax = 96;
constexpr double kLpEps = 1e-11;
constexpr int kLpDegenerate = 8;

__device__ __forceinline__ double lp_block_min(double v, double* red)
{
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1)
        v = fmin(v, __shfl_xor(v, off, 64));
    __syncthreads();
    if (lane == 0)
        red[wave] = v;
    __syncthreads();
    double t = red[0];
#pragma unroll
    for (int w = 1; w < kLpThreads / 64; ++w)
        t = fmin(t, red[w]);
    return t;
}

__device__ __forceinline__ int lp_block_min_int(int v, int* red)
{
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1)
        v = min(v, __shfl_xor(v, off, 64));
    __syncthreads();
    if (lane == 0)
        red[wave] = v;
    __syncthreads();
    int t = red[0];
#pragma unroll
    for (int w = 1; w < kLpThreads / 64; ++w)
        t = min(t, red[w]);
    return t;
}

template <bool IN_LDS>
__global__ __launch_bounds__(kLpThreads) void lp_kernel(const double* __restrict__ M, int P,
                                                        int max_pivots,
                                                        double* __restrict__ work,
                                                        double* __restrict__ value,
                                                        double* __restrict__ x,
                                                        double* __restrict__ y,
                                                        float* __restrict__ sigma,
                                                        int* __restrict__ pivots)
{
    constexpr int LDS_N = IN_LDS ? (kLpLdsMax + 1) * (2 * kLpLdsMax + 1) : 1;
    __shared__ double lds[LDS_N];
    __shared__ double col[kMaxP + 1];
    __shared__ double prow[2 * kMaxP + 1];
    __shared__ int basis[kMaxP];
    __shared__ double redd[kLpThreads / 64];
    __shared__ int redi[kLpThreads / 64];
    const int tid = threadIdx.x;
    const int W = 2 * P + 1;                 // columns: w (P), slacks (P), right-hand side
    double* T = IN_LDS ? lds : work;
    // ---- the shift: min(M); a NaN or infinite entry leaves no game to solve
    // (fmin would skip a NaN): every output is then NaN, pivots -1
    double mn = INFINITY, finite = 1.0;
    for (int i = tid; i < P * P; i += kLpThreads) {
        const double v = M[i];
        mn = fmin(mn, v);
        if (!isfinite(v))
            finite = 0.0;
    }
    mn = lp_block_min(mn, redd);
    if (lp_block_min(finite, redd) == 0.0) {
        for (int j = tid; j < P; j += kLpThreads) {
            x[j] = (double)NAN;
            y[j] = (double)NAN;
            if (sigma) {
                sigma[j] = NAN;
                sigma[P + j] = NAN;
            }
        }
        if (tid == 0) {
            *value = (double)NAN;
            if (pivots)
                *pivots = -1;
        }
        return;
    }
    // ---- the initial tableau (slack basis)
    for (int idx = tid; idx < (P + 1) * W; idx += kLpThreads) {
        const int i = idx / W, j = idx - i * W;
        double v;
        if (i < P)
            v = j < P ? M[(size_t)i * P + j] - mn + 1.0 : (j < 2 * P ? (j - P == i ? 1.0 : 0.0)
                                                                   : 1.0);
        else
            v = j < P ? -1.0 : 0.0;
        T[idx] = v;
    }
    if (tid < P)
        basis[tid] = P + tid;
    __syncthreads();
    int it = 0, degenerate = 0;
    bool done = false;
    for (; it < max_pivots; ++it) {
        // entering column: the most negative reduced cost (the lowest column
        // among equal ones), or under Bland's rule the lowest negative one
        const bool bland = degenerate >= kLpDegenerate;
        double best = INFINITY;
        if (!bland)
            for (int j = tid; j < 2 * P; j += kLpThreads)
                best = fmin(best, T[(size_t)P * W + j]);
        const double dmin = bland ? -INFINITY : lp_block_min(best, redd);
        int cand = INT_MAX;
        for (int j = tid; j < 2 * P; j += kLpThreads) {
            const double c = T[(size_t)P * W + j];
            if (c < -kLpEps && (bland || c == dmin))
                cand = min(cand, j);
        }
        const int e = lp_block_min_int(cand, redi);
        if (e == INT_MAX) {
            done = true;
            break;
        }
        for (int i = tid; i <= P; i += kLpThreads)
            col[i] = T[(size_t)i * W + e];
        __syncthreads();
        // ratio test: the smallest rhs / col over rows with col > 0, then the
        // lowest basic variable among the rows within rounding of it
        double ratio = INFINITY;
        for (int i = tid; i < P; i += kLpThreads)
            if (col[i] > kLpEps)
                ratio = T[(size_t)i * W + 2 * P] / col[i];
        const double rmin = lp_block_min(ratio, redd);
        if (!(rmin < INFINITY))
            break;                           // unbounded: not reachable for M' > 0
        int bcand = INT_MAX;
        for (int i = tid; i < P; i += kLpThreads)
            if (col[i] > kLpEps &&
                T[(size_t)i * W + 2 * P] / col[i] <= rmin + 1e-12 * fmax(1.0, rmin))
                bcand = min(bcand, basis[i] * 1024 + i);   // P <= 256 < 1024
        const int rb = lp_block_min_int(bcand, redi);
        const int r = rb & 1023;
        degenerate = rmin <= 0.0 ? degenerate + 1 : 0;
        // scaled pivot row, then every other row
        const double piv = col[r];
        for (int j = tid; j < W; j += kLpThreads) {
            const double v = T[(size_t)r * W + j] / piv;
            prow[j] = v;
            T[(size_t)r * W + j] = v;
        }
        __syncthreads();
        for (int idx = tid; idx < (P + 1) * W; idx += kLpThreads) {
            const int i = idx / W, j = idx - i * W;
            if (i != r)
                T[idx] -= col[i] * prow[j];
        }
        if (tid == 0)
            basis[r] = e;
        __syncthreads();
    }
    // ---- read the solution
    const double total = T[(size_t)P * W + 2 * P];      // sum of w = sum of u
    const bool ok = done && total > 0.0;
    for (int j = tid; j < P; j += kLpThreads) {
        y[j] = 0.0;
        x[j] = ok ? T[(size_t)P * W + P + j] / total : (double)NAN;
    }
    __syncthreads();
    for (int i = tid; i < P; i += kLpThreads) {
        if (basis[i] < P)
            y[basis[i]] = ok ? T[(size_t)i * W + 2 * P] / total : (double)NAN;
    }
    __syncthreads();
    if (!ok)
        for (int j = tid; j < P; j += kLpThreads)
            y[j] = (double)NAN;
    if (sigma) {
        __syncthreads();
        for (int j = tid; j < P; j += kLpThreads) {
            sigma[j] = (float)x[j];
            sigma[P + j] = (float)y[j];
        }
    }
    if (tid == 0) {
        *value = ok ? 1.0 / total + mn - 1.0 : (double)NAN;
        if (pivots)
            *pivots = done ? it : -1;
    }
}

bool lp_needs_work(int P)
{
    return P > kLpLdsMax;
}

hipError_t launch_lp(const double* M, int P, int max_pivots, double* work, double* value,
                     double* x, double* y, float* sigma, int* pivots, hipStream_t s)
{
    if (P > kMaxP || (P > kLpLdsMax && !work))
        return hipErrorInvalidValue;
    if (P <= kLpLdsMax)
        lp_kernel<true><<<1, kLpThreads, 0, s>>>(M, P, max_pivots, nullptr, value, x, y, sigma,
                                                  pivots);
    else
        lp_kernel<false><<<1, kLpThreads, 0, s>>>(M, P, max_pivots, work, value, x, y, sigma,
                                                   pivots);
    return hipGetLastError();
}

// Thresholds of meta-sampling from device weights, the same fp64 arithmetic as
// the host path: T_m = floor(C_m / C_{P-1} * 2^32) from the sequential fp64
// cumulative sum C of row r, T_{P-1} = 2^32.  A row with a negative or
// non-finite weight or no positive mass gets T = 0 everywhere, which the
// sampling kernel turns into policy id -1 (flagged by the next rollout).
__global__ __launch_bounds__(64) void thresholds_kernel(const float* __restrict__ sigma, int P,
                                                        unsigned long long* __restrict__ thr)
{
    // one wavefront per row: lane 0 forms the sequential fp64 cumulative sum
    // (the order of the host path), every lane then converts its share
    __shared__ double run[kMaxP];
    const int r = blockIdx.x, lane = threadIdx.x;
    const float* s = sigma + (size_t)r * P;
    unsigned long long* T = thr + (size_t)r * P;
    bool ok = true;
    for (int m = lane; m < P; m += 64) {
        const float x = s[m];
        ok = ok && __builtin_isfinite(x) && x >= 0.0f;
    }
    if (lane == 0) {
        double c = 0.0;
        for (int m = 0; m < P; ++m) {
            c += (double)s[m];
            run[m] = c;
        }
    }
    __syncthreads();
    const double total = run[P - 1];
    ok = !__syncthreads_or(!ok) && total > 0.0;
    for (int m = lane; m < P; m += 64) {
        double c = floor(run[m] / total * 4294967296.0);
        if (c > 4294967296.0)
            c = 4294967296.0;
        T[m] = !ok ? 0ull : m == P - 1 ? 4294967296ull : (unsigned long long)c;
    }
}

hipError_t launch_thresholds(const float* sigma, int n_sigma, int P, unsigned long long* thr,
                             hipStream_t s)
{
    thresholds_kernel<<<n_sigma, 64, 0, s>>>(sigma, P, thr);
    return hipGetLastError();
}

}  // namespace malib
