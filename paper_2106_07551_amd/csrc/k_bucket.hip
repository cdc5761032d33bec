// Bucketing of agent slots by policy id: a stable counting sort, so that the
// grouped policy forward can run each policy's rows as dense tiles with one
// set of weights.
//
//   bucket_hist    per-chunk histograms        hist[p][chunk]
//   bucket_scan    exclusive scan (pid-major)  base[p][chunk], offsets[P+1],
//                  tile table tile_off[P+1] (tiles of `tile_rows` rows per policy)
//   bucket_scatter stable scatter              perm[offsets[p] + rank] = slot
//
// Slots are processed in slot order inside each chunk (four waves over
// consecutive quarters; inside a wave, 64-slot segments in order, peeling one
// policy id per iteration with a ballot), so equal ids keep slot order.
#include "device.hpp"
#include "internal.hpp"

namespace malib {

constexpr int kBucketThreads = 256;
constexpr int kWaves = kBucketThreads / 64;
constexpr int kPerWave = kBucketChunk / kWaves;

__device__ __forceinline__ int load_pid(const int32_t* pids, int64_t i, int P, int* flags)
{
    int p = pids[i];
    if (p < 0 || p >= P) {
        atomicOr(flags, kErrPid);
        p = 0;
    }
    return p;
}

__global__ __launch_bounds__(kBucketThreads) void bucket_hist_kernel(
    const int32_t* __restrict__ pids, int64_t n_slots, int P, int n_chunks,
    int32_t* __restrict__ hist, int* flags)
{
    __shared__ int h[kMaxP];
    for (int p = threadIdx.x; p < P; p += kBucketThreads)
        h[p] = 0;
    __syncthreads();
    int64_t base = (int64_t)blockIdx.x * kBucketChunk;
    for (int j = threadIdx.x; j < kBucketChunk; j += kBucketThreads) {
        int64_t i = base + j;
        if (i < n_slots)
            atomicAdd(&h[load_pid(pids, i, P, flags)], 1);
    }
    __syncthreads();
    for (int p = threadIdx.x; p < P; p += kBucketThreads)
        hist[(int64_t)p * n_chunks + blockIdx.x] = h[p];
}

// Single workgroup of 1024 threads: exclusive scan of hist in pid-major order.
__global__ __launch_bounds__(1024) void bucket_scan_kernel(
    const int32_t* __restrict__ hist, int P, int n_chunks, int tile_rows,
    int32_t* __restrict__ base, int32_t* __restrict__ offsets, int32_t* __restrict__ tile_off)
{
    __shared__ int wsum[16];
    __shared__ int carry_s;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    if (tid == 0)
        carry_s = 0;
    __syncthreads();
    int64_t total = (int64_t)P * n_chunks;
    for (int64_t start = 0; start < total; start += 1024) {
        int64_t i = start + tid;
        int v = i < total ? hist[i] : 0;
        // inclusive scan inside the wave
        int x = v;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            int y = __shfl_up(x, off, 64);
            if (lane >= off)
                x += y;
        }
        if (lane == 63)
            wsum[wave] = x;
        __syncthreads();
        int wpre = 0;
        for (int w = 0; w < wave; ++w)
            wpre += wsum[w];
        int carry = carry_s;
        if (i < total)
            base[i] = carry + wpre + x - v;
        __syncthreads();
        if (tid == 1023)
            carry_s = carry + wpre + x;
        __syncthreads();
    }
    __syncthreads();
    // bucket bounds and the first tile of each policy: one thread per policy
    // (P <= 1024), tiles per policy scanned across the workgroup
    const int total_rows = carry_s;
    int start = 0, tiles = 0;
    if (tid < P) {
        start = base[(int64_t)tid * n_chunks];
        const int end = tid + 1 < P ? base[(int64_t)(tid + 1) * n_chunks] : total_rows;
        tiles = (end - start + tile_rows - 1) / tile_rows;
    }
    int x = tiles;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        int y = __shfl_up(x, off, 64);
        if (lane >= off)
            x += y;
    }
    __syncthreads();   // wsum is reused
    if (lane == 63)
        wsum[wave] = x;
    __syncthreads();
    int wpre = 0;
    for (int w = 0; w < wave; ++w)
        wpre += wsum[w];
    if (tid < P) {
        offsets[tid] = start;
        tile_off[tid] = wpre + x - tiles;
    }
    if (tid == P - 1) {
        offsets[P] = total_rows;
        tile_off[P] = wpre + x;
    }
}

__global__ __launch_bounds__(kBucketThreads) void bucket_scatter_kernel(
    const int32_t* __restrict__ pids, int64_t n_slots, int n_agents, int P, int n_chunks,
    const int32_t* __restrict__ base, int32_t* __restrict__ perm, int32_t* __restrict__ perm_env)
{
    __shared__ int wcnt[kWaves][kMaxP];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    for (int p = lane; p < P; p += 64)
        wcnt[wave][p] = 0;
    __syncthreads();
    const int64_t wbase = (int64_t)blockIdx.x * kBucketChunk + (int64_t)wave * kPerWave;
    // per-wave counts of its quarter
    for (int j = lane; j < kPerWave; j += 64) {
        int64_t i = wbase + j;
        if (i < n_slots) {
            int p = pids[i];
            p = (p < 0 || p >= P) ? 0 : p;
            atomicAdd(&wcnt[wave][p], 1);
        }
    }
    __syncthreads();
    // running destination of each policy for this wave
    __shared__ int run[kWaves][kMaxP];
    for (int p = tid; p < P; p += kBucketThreads) {
        int acc = base[(int64_t)p * n_chunks + blockIdx.x];
        for (int w = 0; w < kWaves; ++w) {
            run[w][p] = acc;
            acc += wcnt[w][p];
        }
    }
    __syncthreads();
    const unsigned long long lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    for (int seg = 0; seg < kPerWave; seg += 64) {
        const int64_t i = wbase + seg + lane;
        const bool valid = i < n_slots;
        int p = 0;
        if (valid) {
            p = pids[i];
            p = (p < 0 || p >= P) ? 0 : p;
        }
        // lanes holding the same policy id: intersect, bit by bit of the id
        // (P <= 256: 8 bits), the ballot of lanes that agree with this lane
        unsigned long long same = __ballot(valid);
#pragma unroll
        for (int b = 0; b < 8; ++b) {
            const unsigned long long ones = __ballot(valid && ((p >> b) & 1));
            same &= ((p >> b) & 1) ? ones : ~ones;
        }
        // the group's lowest lane takes the group's destination range; the
        // others rank themselves by lane (slot) order within it
        const int leader = __ffsll((unsigned long long)same) - 1;
        int dst0 = 0;
        if (valid && leader == lane)
            dst0 = atomicAdd(&run[wave][p], __popcll(same));
        dst0 = __shfl(dst0, leader < 0 ? 0 : leader, 64);
        if (valid) {
            const int rank = __popcll(same & lt_mask);
            perm[dst0 + rank] = (int32_t)i;
            perm_env[dst0 + rank] = (int32_t)(i / n_agents);
        }
    }
}

// One thread per table entry: the policy owning tile t (the last policy whose
// first tile is <= t, which skips empty buckets), its first row and row count.
// Plain layout: entry e holds tile e.  Striped layout (for a kernel whose
// workgroup b reads entry (b % 8) * (n_entries / 8) + b / 8, so that workgroups
// on one XCD read one segment): the n_entries (a multiple of 8) form 8 equal
// segments, segment x holds tiles [x T / 8, (x + 1) T / 8) of the T tiles in
// order, then padding, so every XCD gets the same number of real tiles.
__global__ void tile_table_kernel(const int32_t* __restrict__ offsets,
                                  const int32_t* __restrict__ tile_off, int P, int tile_rows,
                                  int n_entries, int striped, int4* __restrict__ info)
{
    const int e = blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= n_entries)
        return;
    const int T = tile_off[P];
    int t = e;
    if (striped) {
        const int per = n_entries / 8;
        const int x = e / per, j = e - x * per;
        const int lo = (int)((int64_t)x * T / 8), hi = (int)((int64_t)(x + 1) * T / 8);
        t = j < hi - lo ? lo + j : T;
    }
    if (t >= T) {
        info[e] = make_int4(-1, 0, 0, 0);
        return;
    }
    int lo = 0, hi = P - 1;
    while (lo < hi) {
        int mid = (lo + hi + 1) >> 1;
        if (tile_off[mid] <= t)
            lo = mid;
        else
            hi = mid - 1;
    }
    int r0 = offsets[lo] + (t - tile_off[lo]) * tile_rows;
    int rows = min(tile_rows, offsets[lo + 1] - r0);
    info[e] = make_int4(lo, r0, rows, 0);
}

hipError_t launch_bucket(const int32_t* pids, int64_t n_slots, int n_agents, int P,
                         int tile_rows, int n_entries, bool striped, int32_t* hist,
                         int32_t* base, int32_t* perm, int32_t* perm_env, int32_t* offsets,
                         int32_t* tile_off, int4* tile_info, int* flags, hipStream_t s)
{
    if (striped && n_entries % 8 != 0)
        return hipErrorInvalidValue;
    int n_chunks = (int)((n_slots + kBucketChunk - 1) / kBucketChunk);
    bucket_hist_kernel<<<n_chunks, kBucketThreads, 0, s>>>(pids, n_slots, P, n_chunks, hist,
                                                           flags);
    bucket_scan_kernel<<<1, 1024, 0, s>>>(hist, P, n_chunks, tile_rows, base, offsets,
                                          tile_off);
    bucket_scatter_kernel<<<n_chunks, kBucketThreads, 0, s>>>(pids, n_slots, n_agents, P,
                                                              n_chunks, base, perm, perm_env);
    tile_table_kernel<<<(n_entries + 255) / 256, 256, 0, s>>>(offsets, tile_off, P, tile_rows,
                                                             n_entries, striped ? 1 : 0,
                                                             tile_info);
    return hipGetLastError();
}

}  // namespace malib
