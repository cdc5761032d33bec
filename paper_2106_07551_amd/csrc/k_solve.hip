// Meta-solver on the payoff table and meta-strategy sampling from device
// weights: the meta-update Comb_{t+1} ~ G(...) of Sec. 3.1 with the
// fictitious-play solver of the PSRO experiments (Sec. 5), closed on the GPU
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

// (value, index) candidates of the best responses.  A beats B for the row side
// when its value is larger, or equal with a lower index; for the column side
// when smaller, or equal with a lower index.  For finite values these are
// strict total orders, so any reduction order finds the first argmax /
// argmin, the same choice as a sequential scan.
struct Cand {
    double v;
    int i;
};

__device__ __forceinline__ Cand shfl_xor_cand(Cand c, int m)
{
    Cand o;
    o.v = __shfl_xor(c.v, m);
    o.i = __shfl_xor(c.i, m);
    return o;
}

template <bool MAX>
__device__ __forceinline__ Cand better(Cand a, Cand b)
{
    const bool a_wins = MAX ? (a.v > b.v || (a.v == b.v && a.i < b.i))
                            : (a.v < b.v || (a.v == b.v && a.i < b.i));
    return a_wins ? a : b;
}

template <bool MAX>
__device__ __forceinline__ Cand wave_best(Cand c)
{
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1)
        c = better<MAX>(c, shfl_xor_cand(c, m));
    return c;
}

constexpr int kSolveThreads = kMaxP;           // one thread per policy
constexpr int kSolveWaves = kSolveThreads / 64;
constexpr int kSolveLdsP = 128;                // up to this P the game sits in LDS

// Simultaneous fictitious play on the zero-sum game with row payoff M
// (P x P, fp64; meant for finite entries, a NaN anywhere in v or w leaves the
// counts unspecified and sets gap to NaN): at iteration t, i_t = first argmax of v = sum over
// s < t of M[:, j_s] and j_t = first argmin of w = sum over s < t of M[i_s, :];
// then both play counts are incremented and v, w gain column j_t and row i_t
// (one fp64 add per element per iteration, in iteration order).  Thread k keeps
// v_k, w_k and both counts of policy k.  Writes sigma[0][k], sigma[1][k] = the
// play counts (weights for meta-sampling) and gap = (max v - min w) / T.
template <bool IN_LDS>
__global__ __launch_bounds__(kSolveThreads) void solve_fp_kernel(const double* __restrict__ M,
                                                                 int P, int T,
                                                                 float* __restrict__ sigma,
                                                                 double* __restrict__ gap)
{
    // the game with a padded row stride (column reads hit different banks)
    constexpr int LDS_DOUBLES = IN_LDS ? kSolveLdsP * (kSolveLdsP + 1) : 1;
    __shared__ double Ms[LDS_DOUBLES];
    __shared__ Cand red[2][2][kSolveWaves];    // [iteration parity][side][wave]
    const int k = threadIdx.x, lane = k & 63, wave = k >> 6;
    const int stride = IN_LDS ? P + 1 : P;
    const double* G = M;
    if constexpr (IN_LDS) {
        for (int e = k; e < P * P; e += kSolveThreads)
            Ms[(e / P) * stride + e % P] = M[e];
        __syncthreads();
        G = Ms;
    }
    const bool mine = k < P;
    double v = 0.0, w = 0.0;
    int cx = 0, cy = 0;
    for (int t = 0; t < T; ++t) {
        Cand a{mine ? v : -INFINITY, mine ? k : P};
        Cand b{mine ? w : INFINITY, mine ? k : P};
        a = wave_best<true>(a);
        b = wave_best<false>(b);
        const int par = t & 1;
        if (lane == 0) {
            red[par][0][wave] = a;
            red[par][1][wave] = b;
        }
        __syncthreads();   // (the other parity's slots are rewritten only after
                           // the next barrier, when every thread has read these)
        Cand ra = red[par][0][0], rb = red[par][1][0];
#pragma unroll
        for (int q = 1; q < kSolveWaves; ++q) {
            ra = better<true>(ra, red[par][0][q]);
            rb = better<false>(rb, red[par][1][q]);
        }
        // (an index of P is only possible when some value is NaN; clamping it
        // keeps every read inside the game, and the gap then reports NaN)
        const int i = ra.i < P ? ra.i : P - 1, j = rb.i < P ? rb.i : P - 1;
        if (mine) {
            cx += k == i;
            cy += k == j;
            v = v + G[k * stride + j];
            w = w + G[i * stride + k];
        }
    }
    if (mine) {
        sigma[k] = (float)cx;
        sigma[P + k] = (float)cy;
    }
    const bool bad = __syncthreads_or(mine && (__builtin_isnan(v) || __builtin_isnan(w)));
    if (gap) {
        Cand a{mine ? v : -INFINITY, mine ? k : P};
        Cand b{mine ? w : INFINITY, mine ? k : P};
        a = wave_best<true>(a);
        b = wave_best<false>(b);
        const int par = T & 1;
        __syncthreads();
        if (lane == 0) {
            red[par][0][wave] = a;
            red[par][1][wave] = b;
        }
        __syncthreads();
        if (k == 0) {
            Cand ra = red[par][0][0], rb = red[par][1][0];
            for (int q = 1; q < kSolveWaves; ++q) {
                ra = better<true>(ra, red[par][0][q]);
                rb = better<false>(rb, red[par][1][q]);
            }
            *gap = bad ? (double)NAN : (ra.v - rb.v) / (double)T;
        }
    }
}

hipError_t launch_solve_fp(const double* M, int P, int T, float* sigma, double* gap,
                           hipStream_t s)
{
    if (P < 1 || P > kSolveThreads || T < 1)
        return hipErrorInvalidValue;
    if (P <= kSolveLdsP)
        solve_fp_kernel<true><<<1, kSolveThreads, 0, s>>>(M, P, T, sigma, gap);
    else
        solve_fp_kernel<false><<<1, kSolveThreads, 0, s>>>(M, P, T, sigma, gap);
    return hipGetLastError();
}

// Thresholds of meta-sampling from device weights, the same fp64 arithmetic as
// the host path: T_m = floor(C_m / C_{P-1} * 2^32) from the sequential fp64
// cumulative sum C of row r, T_{P-1} = 2^32.  A row with a negative or
// non-finite weight or no positive mass gets T = 0 everywhere, which the
// sampling kernel turns into policy id -1 (flagged by the next rollout).
__global__ void thresholds_kernel(const float* __restrict__ sigma, int n_sigma, int P,
                                  unsigned long long* __restrict__ thr)
{
    const int r = blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= n_sigma)
        return;
    const float* s = sigma + (size_t)r * P;
    unsigned long long* T = thr + (size_t)r * P;
    double total = 0.0;
    bool ok = true;
    for (int m = 0; m < P; ++m) {
        const float x = s[m];
        ok = ok && __builtin_isfinite(x) && x >= 0.0f;
        total += (double)x;
    }
    ok = ok && total > 0.0;
    double run = 0.0;
    for (int m = 0; m < P; ++m) {
        run += (double)s[m];
        double c = floor(run / total * 4294967296.0);
        if (c > 4294967296.0)
            c = 4294967296.0;
        T[m] = ok ? (unsigned long long)c : 0ull;
    }
    if (ok)
        T[P - 1] = 4294967296ull;
}

hipError_t launch_thresholds(const float* sigma, int n_sigma, int P, unsigned long long* thr,
                             hipStream_t s)
{
    thresholds_kernel<<<(n_sigma + 63) / 64, 64, 0, s>>>(sigma, n_sigma, P, thr);
    return hipGetLastError();
}

}  // namespace malib
