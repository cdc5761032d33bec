// Meta-strategy draws (policy id per env seat) on the Philox4x64-10 stream.
// (Gumbel-max action sampling runs inside the env-step kernels: gumbel_action.)
#include "device.hpp"
#include "internal.hpp"

namespace malib {

// One thread per (env, seat).  pid = min{m : x < T[m]} for the first lane x
// of block (g, 0, kPurposeMeta<<32 | seat, 0); T is non-decreasing with
// T[P-1] = 2^32, so the binary search always lands inside [0, P).
__global__ void meta_sample_kernel(const unsigned long long* __restrict__ thr, uint32_t seat_map,
                                   int P, int64_t n_envs, int n_agents, uint64_t seed,
                                   int64_t env_offset, int32_t* __restrict__ out)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    int64_t total = n_envs * n_agents;
    if (i >= total)
        return;
    int64_t e = i / n_agents;
    int seat = (int)(i - e * n_agents);
    u64x4 blk = stream_block(seed, (uint64_t)(env_offset + e), 0, kPurposeMeta, seat, 0);
    unsigned long long x = (uint32_t)blk.x;
    const unsigned long long* T = thr + (size_t)((seat_map >> (4 * seat)) & 0xFu) * P;
    if (T[P - 1] == 0ull) {   // an invalid weight row (device weights only)
        out[i] = -1;
        return;
    }
    int lo = 0, hi = P - 1;
    while (lo < hi) {
        int mid = (lo + hi) >> 1;
        if (x < T[mid])
            hi = mid;
        else
            lo = mid + 1;
    }
    out[i] = lo;
}

hipError_t launch_meta_sample(const unsigned long long* thr, uint32_t seat_map, int P,
                              int64_t n_envs, int n_agents, uint64_t seed, int64_t env_offset,
                              int32_t* out, hipStream_t s)
{
    int64_t total = n_envs * n_agents;
    int blocks = (int)((total + 255) / 256);
    meta_sample_kernel<<<blocks, 256, 0, s>>>(thr, seat_map, P, n_envs, n_agents, seed,
                                              env_offset, out);
    return hipGetLastError();
}

__global__ void debug_tanh_kernel(const float* __restrict__ x, float* __restrict__ y, int64_t n)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (; i < n; i += stride)
        y[i] = tanh_ref(x[i]);
}

hipError_t launch_debug_tanh(const float* x, float* y, int64_t n, hipStream_t s)
{
    int64_t blocks = (n + 255) / 256;
    if (blocks > 65536)
        blocks = 65536;
    if (blocks < 1)
        blocks = 1;
    debug_tanh_kernel<<<(int)blocks, 256, 0, s>>>(x, y, n);
    return hipGetLastError();
}

__global__ void debug_bf16_kernel(const float* __restrict__ x, uint32_t* __restrict__ y,
                                  int64_t n_pairs)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (; i < n_pairs; i += stride)
        y[i] = pack_bf16x2(x[2 * i], x[2 * i + 1]);
}

hipError_t launch_debug_bf16(const float* x, uint16_t* y, int64_t n, hipStream_t s)
{
    int64_t pairs = n / 2;
    int64_t blocks = (pairs + 255) / 256;
    blocks = blocks > 65536 ? 65536 : (blocks < 1 ? 1 : blocks);
    debug_bf16_kernel<<<(int)blocks, 256, 0, s>>>(x, (uint32_t*)y, pairs);
    return hipGetLastError();
}

__global__ void debug_philox_kernel(const uint64_t* __restrict__ ctr, uint64_t k0, uint64_t k1,
                                    uint64_t* __restrict__ out, int64_t n)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n)
        return;
    u64x4 c{ctr[4 * i], ctr[4 * i + 1], ctr[4 * i + 2], ctr[4 * i + 3]};
    u64x4 r = philox4x64_10(c, k0, k1);
    out[4 * i] = r.x;
    out[4 * i + 1] = r.y;
    out[4 * i + 2] = r.z;
    out[4 * i + 3] = r.w;
}

hipError_t launch_debug_philox(const uint64_t* ctr, uint64_t k0, uint64_t k1, uint64_t* out,
                               int64_t n, hipStream_t s)
{
    int blocks = (int)((n + 255) / 256);
    debug_philox_kernel<<<blocks, 256, 0, s>>>(ctr, k0, k1, out, n);
    return hipGetLastError();
}

}  // namespace malib
