// Incremental payoff-table expansion: when the population grows from P0 to P
// policies (Sec. 3.1's auto-curriculum adds policies to the pools; the example
// API extends a pool and then simulates only the new combinations, Appendix
// C.2), the table keeps its P0 x P0 cells and only the cells of the new rows
// and columns are simulated.
#include "device.hpp"
#include "internal.hpp"

namespace malib {

// Copies the three P0 x P0 accumulator arrays into the P x P layout (new cells
// zero) and the two trailing words (live frames, flags) after them.
__global__ void remap_table_kernel(const unsigned long long* __restrict__ src, int P0,
                                   unsigned long long* __restrict__ dst, int P)
{
    const int64_t PP = (int64_t)P * P, PP0 = (int64_t)P0 * P0;
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < 3 * PP) {
        const int64_t a = i / PP, c = i - a * PP;
        const int r = (int)(c / P), col = (int)(c - (int64_t)r * P);
        dst[i] = (r < P0 && col < P0) ? src[a * PP0 + (int64_t)r * P0 + col] : 0ull;
    } else if (i < 3 * PP + 2) {
        dst[i] = src[3 * PP0 + (i - 3 * PP)];
    }
}

hipError_t launch_remap_table(const unsigned long long* src, int P0, unsigned long long* dst,
                              int P, hipStream_t s)
{
    const int64_t n = 3 * (int64_t)P * P + 2;
    remap_table_kernel<<<(int)((n + 255) / 256), 256, 0, s>>>(src, P0, dst, P);
    return hipGetLastError();
}

// Policy ids of the expansion batch.  The cells with row or column >= first
// are taken in row-major order of the P x P grid: rows r < first contribute
// their columns first .. P-1, rows r >= first all P columns.  Cell c is
// played by envs c * per_pair .. (c + 1) * per_pair - 1; in each env the
// row-side seats take the cell's row policy, the column-side seats its column
// policy.
__global__ void expansion_pairs_kernel(int P, int first, int per_pair, int n_agents,
                                       uint32_t team_row, int64_t n_slots,
                                       int32_t* __restrict__ out)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n_slots)
        return;
    const int64_t e = i / n_agents;
    const int seat = (int)(i - e * n_agents);
    const int64_t c = e / per_pair;
    const int64_t head = (int64_t)first * (P - first);   // cells of the old rows
    int r, col;
    if (c < head) {
        r = (int)(c / (P - first));
        col = first + (int)(c - (int64_t)r * (P - first));
    } else {
        const int64_t d = c - head;
        r = first + (int)(d / P);
        col = (int)(d - (int64_t)(r - first) * P);
    }
    out[i] = ((team_row >> seat) & 1u) ? r : col;
}

hipError_t launch_expansion_pairs(int P, int first, int per_pair, int n_agents, uint32_t team_row,
                                  int64_t n_envs, int32_t* out, hipStream_t s)
{
    const int64_t n = n_envs * n_agents;
    if (n == 0)
        return hipSuccess;
    expansion_pairs_kernel<<<(int)((n + 255) / 256), 256, 0, s>>>(P, first, per_pair, n_agents,
                                                                  team_row, n, out);
    return hipGetLastError();
}

}  // namespace malib
