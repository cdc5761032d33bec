// Environment kernels: reset, one step of each family with return
// accumulation, and the payoff-table reduction.
//
// State layouts (struct of arrays, coalesced per env index):
//   ITER_MATRIX  uint16 [n_envs]         joint action per lag in 4-bit fields,
//                                        lag 1 in the low nibble, 15 = none
//   PURSUIT      uint8  [2][n_envs]      pursuer cell, evader cell; done [n_envs]
//   FEATURE      fp32   [n_envs][d]      double-buffered between steps
// Returns: fp32 [n_agents][n_envs].
#include "device.hpp"
#include "internal.hpp"

namespace malib {

__device__ __forceinline__ int64_t traj_rec(const TrajArgs& tr, int t, int64_t n, int64_t e)
{
    return (tr.base + (int64_t)t * n + e) % tr.cap;
}


// ---------------------------------------------------------------- reset

// x[0..n) = 0 with a kernel rather than a memset node, so that a caller may
// capture the launch sequence in a HIP graph.
__global__ void zero_f32_kernel(float* __restrict__ x, int64_t n)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n)
        x[i] = 0.0f;
}

hipError_t launch_zero_f32(float* x, int64_t n, hipStream_t s)
{
    if (n > 0)
        zero_f32_kernel<<<(int)((n + 255) / 256), 256, 0, s>>>(x, n);
    return hipGetLastError();
}

__global__ void reset_iter_kernel(uint16_t* __restrict__ hist, int64_t n)
{
    int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e < n)
        hist[e] = 0xFFFF;
}

// G x G torus: pursuer cell = floor(lane0 * G^2 / 2^32) (the top 6 bits of
// lane 0 when G = 8); evader = pursuer + 1 + floor(lane1 * (G^2 - 1) / 2^32)
// mod G^2, so the two never start on the same cell.
__global__ void reset_pursuit_kernel(uint8_t* __restrict__ pos, uint8_t* __restrict__ done,
                                     int64_t n, int grid, uint64_t seed, int64_t env_offset,
                                     int shared)
{
    int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= n)
        return;
    uint64_t g = shared ? 0 : (uint64_t)(env_offset + e);
    u64x4 b = stream_block(seed, g, 0, kPurposeReset, 0, 0);
    uint32_t x0 = (uint32_t)b.x, x1 = (uint32_t)(b.x >> 32);
    uint32_t cells = (uint32_t)(grid * grid);
    uint32_t pc = (uint32_t)(((uint64_t)x0 * (uint64_t)cells) >> 32);
    uint32_t shift = (uint32_t)(((uint64_t)x1 * (uint64_t)(cells - 1)) >> 32);
    uint32_t ec = (pc + 1 + shift) % cells;
    pos[e] = (uint8_t)pc;
    pos[n + e] = (uint8_t)ec;
    done[e] = 0;
}

// s0[k] = (2*(x_k>>9)+1 - 2^23) * 2^-23 with x_k lane k%8 of block k/8.
// One thread per (env, block of 8 coordinates).
__global__ void reset_feature_kernel(float* __restrict__ s, uint16_t* __restrict__ obs, int64_t n,
                                     int d, uint64_t seed, int64_t env_offset, int shared)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    int nb = d / 8;
    if (i >= n * nb)
        return;
    int64_t e = i / nb;
    int blk = (int)(i - e * nb);
    uint64_t g = shared ? 0 : (uint64_t)(env_offset + e);
    u64x4 b = stream_block(seed, g, 0, kPurposeReset, 0, (uint64_t)blk);
    float v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        int32_t odd = (int32_t)(2u * (block_lane(b, j) >> 9) + 1u);
        v[j] = (float)(odd - (1 << 23)) * 0x1p-23f;
    }
    float4* dst = reinterpret_cast<float4*>(s + e * d + blk * 8);
    dst[0] = make_float4(v[0], v[1], v[2], v[3]);
    dst[1] = make_float4(v[4], v[5], v[6], v[7]);
    if (obs)
        *reinterpret_cast<uint4*>(obs + e * d + blk * 8) =
            make_uint4(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]),
                       pack_bf16x2(v[4], v[5]), pack_bf16x2(v[6], v[7]));
}

hipError_t launch_reset(const EnvArgs& e, int64_t n_envs, uint64_t seed, int64_t env_offset,
                        void* state, uint8_t* done, hipStream_t s)
{
    int shared = e.init_mode == MALIB_INIT_SHARED;
    if (e.kind == MALIB_ENV_ITER_MATRIX) {
        reset_iter_kernel<<<(int)((n_envs + 255) / 256), 256, 0, s>>>((uint16_t*)state, n_envs);
    } else if (e.kind == MALIB_ENV_PURSUIT) {
        reset_pursuit_kernel<<<(int)((n_envs + 255) / 256), 256, 0, s>>>(
            (uint8_t*)state, done, n_envs, e.grid, seed, env_offset, shared);
    } else if (e.kind == MALIB_ENV_FEATURE) {
        int64_t total = n_envs * (e.d / 8);
        reset_feature_kernel<<<(int)((total + 255) / 256), 256, 0, s>>>(
            (float*)state, e.obs, n_envs, e.d, seed, env_offset, shared);
    }
    return hipGetLastError();
}

__global__ void transpose_kernel(const float* __restrict__ W, float* __restrict__ WT, int d)
{
    __shared__ float tile[32][33];
    int bx = blockIdx.x * 32, by = blockIdx.y * 32;
    int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;   // 32 x 8
    for (int r = ty; r < 32; r += 8)
        tile[r][tx] = W[(int64_t)(by + r) * d + bx + tx];
    __syncthreads();
    for (int r = ty; r < 32; r += 8)
        WT[(int64_t)(bx + r) * d + by + tx] = tile[tx][r];
}

hipError_t launch_transpose(const float* W, float* WT, int d, hipStream_t s)
{
    dim3 grid(d / 32, d / 32);
    transpose_kernel<<<grid, 256, 0, s>>>(W, WT, d);
    return hipGetLastError();
}

// ---------------------------------------------------- matrix / iterated / pursuit

// The two seats' actions of env e (Gumbel-max over their logits, logged when
// asked); a NaN logit raises kErrNaN.
template <int AMAX>
__device__ __forceinline__ void sample_pair(const SampleArgs& sa, int A, int64_t e, int& a0,
                                            int& a1)
{
    bool n0, n1;
    const uint64_t g = (uint64_t)(sa.env_offset + e);
    a0 = gumbel_action<AMAX>(sa.logits + (2 * e) * A, A, sa.seed, g, sa.t, 0, n0);
    a1 = gumbel_action<AMAX>(sa.logits + (2 * e + 1) * A, A, sa.seed, g, sa.t, 1, n1);
    if (n0 || n1)
        atomicOr(sa.flags, kErrNaN);
    if (sa.log) {
        sa.log[2 * e] = (uint8_t)a0;
        sa.log[2 * e + 1] = (uint8_t)a1;
    }
}

// One thread per env: both seats' actions, then MATRIX and ITER_MATRIX:
// r0 = A[a0][a1], r1 = -r0; ITER also shifts the joint action into its history.
template <int AMAX>
__global__ void step_matrix_kernel(const float* __restrict__ Amat, int A, int iter, int64_t n,
                                   SampleArgs sa, TrajArgs tr, uint16_t* __restrict__ hist,
                                   float* __restrict__ ret)
{
    int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= n)
        return;
    int a0, a1;
    sample_pair<AMAX>(sa, A, e, a0, a1);
    float v = Amat[a0 * A + a1];
    ret[e] = ret[e] + v;
    ret[n + e] = ret[n + e] + (-v);
    const uint32_t h = iter ? hist[e] : 0u;
    if (iter)
        hist[e] = (uint16_t)(((h << 4) | (uint32_t)(a0 * 3 + a1)) & 0xFFFFu);
    if (tr.act) {
        const int64_t r = traj_rec(tr, sa.t, n, e);
        tr.act[2 * r] = (uint8_t)a0;
        tr.act[2 * r + 1] = (uint8_t)a1;
        tr.rew[r] = v;
        tr.flags[r] = sa.t == tr.horizon - 1 ? 2 : 0;
        if (iter && tr.obs)
            ((uint16_t*)tr.obs)[r] = (uint16_t)h;
    }
}

__device__ __forceinline__ uint32_t torus_move(uint32_t cell, int a, int grid)
{
    int x = (int)cell % grid, y = (int)cell / grid;
    if (a == 1)
        y = (y + grid - 1) % grid;
    else if (a == 2)
        y = (y + 1) % grid;
    else if (a == 3)
        x = (x + grid - 1) % grid;
    else if (a == 4)
        x = (x + 1) % grid;
    return (uint32_t)(y * grid + x);
}

// One thread per slot (lanes 2e and 2e+1: pursuer and evader of env e), all
// loads issued first: each lane samples its seat's action (5 actions), the
// pair exchange them, and the pursuer's lane makes the simultaneous moves;
// capture if the two land on the same cell or swap cells: pursuer +1, evader
// -1, env done.  Finished envs take no action (logged as 255).  Counts live
// agent-frames (two per live env) with one atomic per workgroup.
__global__ __launch_bounds__(256) void step_pursuit_kernel(
    int grid, int64_t n, SampleArgs sa, TrajArgs tr, uint8_t* __restrict__ pos,
    uint8_t* __restrict__ done, float* __restrict__ ret, unsigned long long* frames)
{
    __shared__ int live_s;
    if (threadIdx.x == 0)
        live_s = 0;
    __syncthreads();
    const int64_t slot = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t e = slot >> 1;
    const int seat = (int)(slot & 1);
    const bool valid = e < n;                 // both lanes of a pair agree
    const int64_t ec = valid ? e : 0;
    const bool dn = done[ec] != 0;
    const uint32_t p0 = pos[ec], q0 = pos[n + ec];
    bool nan = false;
    const int a = gumbel_action<8>(sa.logits + (valid ? slot : 0) * 5, 5, sa.seed,
                                   (uint64_t)(sa.env_offset + ec), sa.t, seat, nan);
    const int a_other = __shfl_xor(a, 1);
    const bool live = valid && !dn;
    if (live && nan)
        atomicOr(sa.flags, kErrNaN);
    if (valid && sa.log)
        sa.log[slot] = live ? (uint8_t)a : (uint8_t)255;
    bool caught = false;
    if (live && seat == 0) {
        const uint32_t p1 = torus_move(p0, a, grid);
        const uint32_t q1 = torus_move(q0, a_other, grid);
        pos[e] = (uint8_t)p1;
        pos[n + e] = (uint8_t)q1;
        if (p1 == q1 || (p1 == q0 && q1 == p0)) {
            caught = true;
            done[e] = 1;
            ret[e] = ret[e] + 1.0f;
            ret[n + e] = ret[n + e] + (-1.0f);
        }
    }
    if (valid && tr.act) {
        const int64_t r = traj_rec(tr, sa.t, n, e);
        tr.act[2 * r + seat] = live ? (uint8_t)a : (uint8_t)255;
        if (seat == 0) {
            tr.rew[r] = caught ? 1.0f : 0.0f;
            tr.flags[r] = (uint8_t)((caught ? 1 : 0) | (sa.t == tr.horizon - 1 ? 2 : 0) |
                                    (dn ? 4 : 0));
            if (tr.obs) {
                uint8_t* o = (uint8_t*)tr.obs + 2 * r;
                o[0] = (uint8_t)p0;
                o[1] = (uint8_t)q0;
            }
        }
    }
    const unsigned long long b = __ballot(live && seat == 0);
    if ((threadIdx.x & 63) == 0 && b)
        atomicAdd(&live_s, __popcll(b));
    __syncthreads();
    if (threadIdx.x == 0 && live_s)
        atomicAdd(frames, (unsigned long long)live_s * 2ull);
}

// ------------------------------------------------------------ feature dynamics

// One workgroup of kFeatWaves wavefronts owns kFeatWaves*EPT envs and all D
// outputs of each:
//   s'[e][k] = tanh_ref( fma-chain_{c=0..D-1}(W[k][c], s[e][c]) + emb[0][a_0][k]
//                        + emb[1][a_1][k] + ... )
// Thread (tx = tid%64, ty = tid/64) keeps the accumulators of envs
// ty*EPT..ty*EPT+EPT-1 and outputs g*64*GW + GW*tx + j (groups of GW <= 4
// consecutive outputs); the input index c runs in ascending order through
// LDS-staged chunks of WT (c-major) and of the state (so every accumulator
// sees exactly the sequential fused chain, no split of the sum).  The reward
// r = u . s' is then a sequential fused chain per env over the staged s'.
constexpr int kFeatKC = 32;
// Eight wavefronts per workgroup: the WT chunks staged through LDS serve twice
// as many envs as with four, and the grid has half as many workgroups to ramp
// up and drain (d=256: 50 vs 54 us per step of 16384 envs; d=512: -3%).
constexpr int kFeatWaves = 8, kFeatThreads = 64 * kFeatWaves;

// EPT envs per thread (8, 4, 2 or 1).
// GW consecutive floats (GW = 1, 2 or 4) as one load or store: outputs are
// mapped to threads in groups of GW consecutive indices, so the WT reads from
// LDS, the embedding loads and the state stores are single wide accesses.
template <int GW>
struct FVec;
template <>
struct FVec<1> {
    float v[1];
    __device__ __forceinline__ void load(const float* p) { v[0] = *p; }
    __device__ __forceinline__ void store(float* p) const { *p = v[0]; }
};
template <>
struct FVec<2> {
    float v[2];
    __device__ __forceinline__ void load(const float* p)
    {
        typedef float v2f __attribute__((ext_vector_type(2)));
        const v2f t = *reinterpret_cast<const v2f*>(p);
        v[0] = t.x;
        v[1] = t.y;
    }
    __device__ __forceinline__ void store(float* p) const
    {
        typedef float v2f __attribute__((ext_vector_type(2)));
        *reinterpret_cast<v2f*>(p) = v2f{v[0], v[1]};
    }
};
template <>
struct FVec<4> {
    float v[4];
    __device__ __forceinline__ void load(const float* p)
    {
        typedef float v4f __attribute__((ext_vector_type(4)));
        const v4f t = *reinterpret_cast<const v4f*>(p);
        v[0] = t.x;
        v[1] = t.y;
        v[2] = t.z;
        v[3] = t.w;
    }
    __device__ __forceinline__ void store(float* p) const
    {
        typedef float v4f __attribute__((ext_vector_type(4)));
        *reinterpret_cast<v4f*>(p) = v4f{v[0], v[1], v[2], v[3]};
    }
};

// bf16_rne of GW consecutive floats as one 2-, 4- or 8-byte store.
template <int GW>
__device__ __forceinline__ void store_bf16(uint16_t* p, const FVec<GW>& t)
{
    if constexpr (GW == 1) {
        *p = bf16_bits(t.v[0]);
    } else if constexpr (GW == 2) {
        *reinterpret_cast<uint32_t*>(p) = pack_bf16x2(t.v[0], t.v[1]);
    } else {
        *reinterpret_cast<uint2*>(p) =
            make_uint2(pack_bf16x2(t.v[0], t.v[1]), pack_bf16x2(t.v[2], t.v[3]));
    }
}

template <int D, int EPT>
__global__ __launch_bounds__(kFeatThreads) void step_feature_kernel(
    const float* __restrict__ WT, const float* __restrict__ emb, const float* __restrict__ u,
    EnvArgs ea, SampleArgs sa, int64_t n, const float* __restrict__ s_in,
    float* __restrict__ s_out, float* __restrict__ ret)
{
    constexpr int kFeatEnvs = kFeatWaves * EPT;
    constexpr int NJ = D / 64;                  // outputs per thread
    constexpr int GW = NJ < 4 ? NJ : 4;         // ... in groups of GW consecutive ones
    constexpr int NG = NJ / GW;                 // output k of (group g, j) = g*64*GW + GW*tx + j
    constexpr int SSTR = kFeatEnvs + 4;
    constexpr int SLD = D + 4;                  // row stride of s' in LDS (16-byte rows)
    constexpr int WS_FLOATS = kFeatKC * D > kFeatEnvs * SLD ? kFeatKC * D : kFeatEnvs * SLD;
    __shared__ __attribute__((aligned(16))) float Ws[WS_FLOATS];
    __shared__ __attribute__((aligned(16))) float Ss[kFeatKC * SSTR];
    // the reward weights u, staged once: the chain then reads both of its
    // operands from LDS (in-order returns, so its loads can run ahead)
    __shared__ __attribute__((aligned(16))) float Us[D];
    const int tid = threadIdx.x, tx = tid & 63, ty = tid >> 6;
    const int64_t e0 = (int64_t)blockIdx.x * kFeatEnvs;
    for (int k = tid; k < D; k += kFeatThreads)   // read after the main loop's barriers
        Us[k] = u[k];

    // Staging: chunk c0 of WT (KC x D floats, c-major) and of the state (32 envs
    // x KC) goes global -> registers -> LDS; the loads of chunk c0+KC are issued
    // before the FMAs of chunk c0 so their latency overlaps the arithmetic.
    constexpr int WQ = kFeatKC * D / 4 / kFeatThreads;   // float4 of WT per thread per chunk
    // state chunk: kFeatEnvs envs x KC columns = kFeatEnvs*8 float4; threads
    // beyond that re-load env 0's chunk and skip the LDS store
    const int el_ld = (tid >> 3) % kFeatEnvs, cq_ld = tid & 7;
    const bool s_owner = (tid >> 3) < kFeatEnvs;
    const int64_t e_ld = e0 + el_ld;
    typedef float v4f __attribute__((ext_vector_type(4)));
    const v4f* wsrc = reinterpret_cast<const v4f*>(WT) + tid;
    const float* ssrc = s_in + (e_ld < n ? e_ld : 0) * D + cq_ld * 4;
    v4f wreg[WQ];
    v4f sreg;
#pragma unroll
    for (int q = 0; q < WQ; ++q)
        wreg[q] = wsrc[q * kFeatThreads];
    sreg = *reinterpret_cast<const v4f*>(ssrc);

    // the actions of the workgroup's slots while the first chunk loads are in
    // flight: one thread per slot, Gumbel-max over its logits, or the action
    // the policy kernel sampled (envs past the end take action 0 and are never
    // stored)
    __shared__ __attribute__((aligned(8))) uint8_t act_s[kFeatEnvs * kMaxAgents];
    if (tid < kFeatEnvs * ea.n_agents) {
        const int el = tid / ea.n_agents, seat = tid - el * ea.n_agents;
        const int64_t e = e0 + el;
        int a = 0;
        if (e < n) {
            const int64_t slot = e * ea.n_agents + seat;
            if (sa.actions) {
                a = sa.actions[slot];   // sampled by the policy kernel
            } else {
                bool nan;
                a = gumbel_action<kMaxActions>(sa.logits + slot * ea.A, ea.A, sa.seed,
                                                (uint64_t)(sa.env_offset + e), sa.t, seat, nan);
                if (nan)
                    atomicOr(sa.flags, kErrNaN);
            }
            if (sa.log)
                sa.log[slot] = (uint8_t)a;
            if (ea.tr.act)
                ea.tr.act[traj_rec(ea.tr, sa.t, n, e) * ea.n_agents + seat] = (uint8_t)a;
        }
        act_s[el * kMaxAgents + seat] = (uint8_t)a;
    }
    __syncthreads();
    // the actions of this thread's envs, 8 bits per seat (bytes of seats
    // >= n_agents are never read)
    // (a wavefront's envs are the same for all its lanes: the action bytes, and
    // with them the embedding rows' addresses, are kept in scalar registers)
    uint64_t act_pk[EPT];
#pragma unroll
    for (int i = 0; i < EPT; ++i) {
        const uint64_t pk =
            *reinterpret_cast<const uint64_t*>(act_s + (ty * EPT + i) * kMaxAgents);
        act_pk[i] = (uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)pk) |
                    ((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(pk >> 32)) << 32);
    }

    float acc[EPT][NJ];
#pragma unroll
    for (int i = 0; i < EPT; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j)
            acc[i][j] = 0.0f;

    // trajectory observation of the step: bf16(s) of each env, written by the
    // threads that stage the state chunks
    uint16_t* obs_row = nullptr;
    if (ea.tr.obs && s_owner && e_ld < n)
        obs_row = (uint16_t*)ea.tr.obs + traj_rec(ea.tr, sa.t, n, e_ld) * D + cq_ld * 4;
    for (int c0 = 0; c0 < D; c0 += kFeatKC) {
        v4f* dst = reinterpret_cast<v4f*>(Ws);
#pragma unroll
        for (int q = 0; q < WQ; ++q)
            dst[q * kFeatThreads + tid] = wreg[q];
        if (e_ld >= n)
            sreg = v4f{0.f, 0.f, 0.f, 0.f};
        if (obs_row)
            *reinterpret_cast<uint2*>(obs_row + c0) =
                make_uint2(pack_bf16x2(sreg.x, sreg.y), pack_bf16x2(sreg.z, sreg.w));
        if (s_owner) {
            Ss[(cq_ld * 4 + 0) * SSTR + el_ld] = sreg.x;
            Ss[(cq_ld * 4 + 1) * SSTR + el_ld] = sreg.y;
            Ss[(cq_ld * 4 + 2) * SSTR + el_ld] = sreg.z;
            Ss[(cq_ld * 4 + 3) * SSTR + el_ld] = sreg.w;
        }
        __syncthreads();
        {
            // next chunk (the last iteration re-reads its own chunk, unused)
            const int cn = c0 + kFeatKC < D ? c0 + kFeatKC : c0;
            const v4f* wn = wsrc + cn * (D / 4);
#pragma unroll
            for (int q = 0; q < WQ; ++q)
                wreg[q] = wn[q * kFeatThreads];
            sreg = *reinterpret_cast<const v4f*>(ssrc + cn);
        }
#pragma unroll
        for (int c = 0; c < kFeatKC; ++c) {
            float w[NJ];
#pragma unroll
            for (int g = 0; g < NG; ++g) {
                FVec<GW> t;
                t.load(&Ws[c * D + g * 64 * GW + GW * tx]);
#pragma unroll
                for (int j = 0; j < GW; ++j)
                    w[g * GW + j] = t.v[j];
            }
            float sv[EPT];
            if constexpr (EPT % 4 == 0) {
                const v4f* sp = reinterpret_cast<const v4f*>(&Ss[c * SSTR + ty * EPT]);
#pragma unroll
                for (int q = 0; q < EPT / 4; ++q) {
                    v4f t4 = sp[q];
                    sv[4 * q + 0] = t4.x;
                    sv[4 * q + 1] = t4.y;
                    sv[4 * q + 2] = t4.z;
                    sv[4 * q + 3] = t4.w;
                }
            } else {
#pragma unroll
                for (int i = 0; i < EPT; ++i)
                    sv[i] = Ss[c * SSTR + ty * EPT + i];
            }
#pragma unroll
            for (int i = 0; i < EPT; ++i)
#pragma unroll
                for (int j = 0; j < NJ; ++j)
                    acc[i][j] = __builtin_fmaf(w[j], sv[i], acc[i][j]);
        }
        __syncthreads();
    }

    // epilogue: embeddings in seat order (seat-outer so that each seat's loads
    // for all of the thread's outputs are independent), tanh_ref, store s'
    float* Sl = Ws;   // [kFeatEnvs][SLD]
    float pre[EPT][NJ];
#pragma unroll
    for (int i = 0; i < EPT; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j)
            pre[i][j] = acc[i][j];
#pragma unroll
    for (int q = 0; q < kMaxAgents; ++q) {
        if (q < ea.n_agents) {
            int off[EPT];
#pragma unroll
            for (int i = 0; i < EPT; ++i) {
                const int a_q = (int)((act_pk[i] >> (8 * q)) & 0xFFu);
                off[i] = (q * ea.A + a_q) * D + GW * tx;
            }
#pragma unroll
            for (int i = 0; i < EPT; ++i)
#pragma unroll
                for (int g = 0; g < NG; ++g) {
                    FVec<GW> t;
                    t.load(emb + off[i] + g * 64 * GW);
#pragma unroll
                    for (int j = 0; j < GW; ++j)
                        pre[i][g * GW + j] = pre[i][g * GW + j] + t.v[j];
                }
        }
    }
#pragma unroll
    for (int i = 0; i < EPT; ++i) {
        const int el = ty * EPT + i;
        const int64_t e = e0 + el;
#pragma unroll
        for (int g = 0; g < NG; ++g) {
            const int k0 = g * 64 * GW + GW * tx;
            FVec<GW> t;
#pragma unroll
            for (int j = 0; j < GW; ++j)
                t.v[j] = tanh_ref(pre[i][g * GW + j]);
            if (e < n) {
                t.store(s_out + e * D + k0);
                if (ea.obs)
                    store_bf16<GW>(ea.obs + e * D + k0, t);
            }
            t.store(Sl + el * SLD + k0);
        }
    }
    // reward chain of the workgroup's envs (one lane each); the seats' running
    // returns are fetched before the chain so their latency overlaps it, and
    // the chain is unrolled so that its LDS loads run ahead of the dependent
    // FMAs
    const int64_t er = e0 + tid;
    const bool rlane = tid < kFeatEnvs && er < n;
    float rv[kMaxAgents];
#pragma unroll
    for (int q = 0; q < kMaxAgents; ++q)
        if (rlane && q < ea.n_agents)
            rv[q] = ret[(int64_t)q * n + er];
    __syncthreads();
    if (rlane) {
        float r = 0.0f;
        const float* row = Sl + tid * SLD;
        const float* u = Us;
#pragma unroll
        for (int k = 0; k < D; ++k)
            r = __builtin_fmaf(u[k], row[k], r);
#pragma unroll
        for (int q = 0; q < kMaxAgents; ++q)
            if (q < ea.n_agents)
                ret[(int64_t)q * n + er] = rv[q] + (((ea.team_row >> q) & 1u) ? r : -r);
        if (ea.tr.rew) {
            const int64_t rec = traj_rec(ea.tr, sa.t, n, er);
            ea.tr.rew[rec] = r;
            ea.tr.flags[rec] = sa.t == ea.tr.horizon - 1 ? 2 : 0;
        }
    }
}

hipError_t launch_env_step(const EnvArgs& e, const SampleArgs& sa, int64_t n_envs,
                           const void* state_in, void* state_out, uint8_t* done, float* ret,
                           unsigned long long* frames, hipStream_t s)
{
    int blocks = (int)((n_envs + 255) / 256);
    switch (e.kind) {
    case MALIB_ENV_MATRIX:
    case MALIB_ENV_ITER_MATRIX: {
        const int iter = e.kind == MALIB_ENV_ITER_MATRIX;
        uint16_t* hist = iter ? (uint16_t*)state_out : nullptr;
        if (e.A <= 8)
            step_matrix_kernel<8><<<blocks, 256, 0, s>>>(e.Amat, e.A, iter, n_envs, sa, e.tr, hist, ret);
        else if (e.A <= 16)
            step_matrix_kernel<16><<<blocks, 256, 0, s>>>(e.Amat, e.A, iter, n_envs, sa, e.tr, hist, ret);
        else if (e.A <= 24)
            step_matrix_kernel<24><<<blocks, 256, 0, s>>>(e.Amat, e.A, iter, n_envs, sa, e.tr, hist, ret);
        else if (e.A <= 32)
            step_matrix_kernel<32><<<blocks, 256, 0, s>>>(e.Amat, e.A, iter, n_envs, sa, e.tr, hist, ret);
        else
            return hipErrorInvalidValue;
        break;
    }
    case MALIB_ENV_PURSUIT:
        if (e.A != 5)
            return hipErrorInvalidValue;
        // one thread per slot
        step_pursuit_kernel<<<(int)((2 * n_envs + 255) / 256), 256, 0, s>>>(
            e.grid, n_envs, sa, e.tr, (uint8_t*)state_out, done, ret, frames);
        break;
    case MALIB_ENV_FEATURE: {
        const float* si = (const float*)state_in;
        float* so = (float*)state_out;
        if (e.A > kMaxActions)
            return hipErrorInvalidValue;
        // 8 envs per thread for d = 512 (64-env workgroups), 4 below (32 envs);
        // at d = 256 a batch too small for one such workgroup per CU takes 2 or
        // 1 env per thread instead (16- or 8-env workgroups): the step of a
        // small batch is latency-bound, and more workgroups shorten it (4v4
        // game: 4096 envs 28.9 -> 25.0 us with 2, 2048 envs 27.3 -> 20.9 us and
        // 257 envs 26.3 -> 19.0 us with 1; the sums are the same per output)
        const int64_t cus = e.n_cus > 0 ? e.n_cus : 256;
        const int fb8 = (int)((n_envs + 8 * kFeatWaves - 1) / (8 * kFeatWaves));
        const int fb4 = (int)((n_envs + 4 * kFeatWaves - 1) / (4 * kFeatWaves));
        const int fb2 = (int)((n_envs + 2 * kFeatWaves - 1) / (2 * kFeatWaves));
        const int fb1 = (int)((n_envs + kFeatWaves - 1) / kFeatWaves);
        if (e.d == 64)
            step_feature_kernel<64, 4><<<fb4, kFeatThreads, 0, s>>>(e.WT, e.emb, e.u, e, sa, n_envs, si, so, ret);
        else if (e.d == 128)
            step_feature_kernel<128, 4><<<fb4, kFeatThreads, 0, s>>>(e.WT, e.emb, e.u, e, sa, n_envs, si, so, ret);
        else if (e.d == 256 && n_envs >= 4 * kFeatWaves * cus)
            step_feature_kernel<256, 4><<<fb4, kFeatThreads, 0, s>>>(e.WT, e.emb, e.u, e, sa, n_envs, si, so, ret);
        else if (e.d == 256 && n_envs >= 2 * kFeatWaves * cus)
            step_feature_kernel<256, 2><<<fb2, kFeatThreads, 0, s>>>(e.WT, e.emb, e.u, e, sa, n_envs, si, so, ret);
        else if (e.d == 256)
            step_feature_kernel<256, 1><<<fb1, kFeatThreads, 0, s>>>(e.WT, e.emb, e.u, e, sa, n_envs, si, so, ret);
        else if (e.d == 512)
            step_feature_kernel<512, 8><<<fb8, kFeatThreads, 0, s>>>(e.WT, e.emb, e.u, e, sa, n_envs, si, so, ret);
        else
            return hipErrorInvalidValue;
        break;
    }
    default:
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

// PURSUIT snapshot in the trace format [n_envs][3] = (pursuer, evader, done).
__global__ void snapshot_pursuit_kernel(const uint8_t* __restrict__ pos,
                                        const uint8_t* __restrict__ done, int64_t n,
                                        uint8_t* __restrict__ out)
{
    int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= n)
        return;
    out[3 * e] = pos[e];
    out[3 * e + 1] = pos[n + e];
    out[3 * e + 2] = done[e];
}

hipError_t launch_snapshot_pursuit(const void* state, const uint8_t* done, int64_t n_envs,
                                   uint8_t* out, hipStream_t s)
{
    snapshot_pursuit_kernel<<<(int)((n_envs + 255) / 256), 256, 0, s>>>(
        (const uint8_t*)state, done, n_envs, out);
    return hipGetLastError();
}

// ------------------------------------------------------------ payoff reduction

// One thread per env.  Every (row-side seat a, column-side seat b) pair adds
// the fixed-point return of seat a (2^-32 units; squares in 2^-20 units) and a
// count to cell (pid[a], pid[b]).  When a whole wavefront targets one cell
// (blocked assignments), it reduces with shuffles and issues one set of
// atomics; otherwise each lane adds its own.
__device__ __forceinline__ long long wave_sum_i64(long long v)
{
#pragma unroll
    for (int off = 32; off > 0; off >>= 1)
        v += __shfl_xor(v, off, 64);
    return v;
}

__global__ __launch_bounds__(256) void payoff_kernel(
    const float* __restrict__ ret, const int32_t* __restrict__ pids, int64_t n, int n_agents,
    EnvArgs ea, int P, unsigned long long* __restrict__ sum,
    unsigned long long* __restrict__ sumsq, unsigned long long* __restrict__ cnt)
{
    int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    bool valid = e < n;
    for (int a = 0; a < n_agents; ++a) {
        if (!((ea.team_row >> a) & 1u))
            continue;
        long long fx = 0, fsq = 0;
        if (valid) {
            double g = (double)ret[(int64_t)a * n + e];
            fx = __double2ll_rn(g * 4294967296.0);
            fsq = __double2ll_rn(g * g * 1048576.0);
        }
        for (int b = 0; b < n_agents; ++b) {
            if (!((ea.team_col >> b) & 1u))
                continue;
            int cell = -1;
            if (valid) {
                int pa = pids[e * n_agents + a], pb = pids[e * n_agents + b];
                if (pa >= 0 && pa < P && pb >= 0 && pb < P)
                    cell = pa * P + pb;
            }
            int c0 = __shfl(cell, 0, 64);
            bool uniform = __ballot(cell != c0) == 0ull;
            if (uniform) {
                if (c0 >= 0) {
                    long long s1 = wave_sum_i64(fx), s2 = wave_sum_i64(fsq);
                    long long c = wave_sum_i64(cell >= 0 ? 1 : 0);
                    if ((threadIdx.x & 63) == 0) {
                        atomicAdd(&sum[c0], (unsigned long long)s1);
                        atomicAdd(&sumsq[c0], (unsigned long long)s2);
                        atomicAdd(&cnt[c0], (unsigned long long)c);
                    }
                }
            } else if (cell >= 0) {
                atomicAdd(&sum[cell], (unsigned long long)fx);
                atomicAdd(&sumsq[cell], (unsigned long long)fsq);
                atomicAdd(&cnt[cell], 1ull);
            }
        }
    }
}

// Small populations (P*P cells fit one workgroup's LDS): each workgroup walks
// a contiguous range of envs in env order (coalesced reads of the returns and
// ids) and reduces every incidence into a private copy of the whole table in
// LDS: one LDS atomic per incidence, or, where a whole wavefront targets one
// cell (blocked assignments), a shuffle reduction and one LDS atomic per
// wavefront.  The workgroup then adds each touched cell to the table with one
// set of global atomics.  64-bit integer atomics keep the sums exact and
// independent of the order.
__device__ __forceinline__ void lds_incidence(unsigned long long* s_sum,
                                              unsigned long long* s_sq, unsigned int* s_cnt,
                                              int cell, long long fx, long long fsq)
{
    const int c0 = __shfl(cell, 0, 64);
    if (__ballot(cell != c0) == 0ull) {
        if (c0 >= 0) {
            const long long s1 = wave_sum_i64(fx), s2 = wave_sum_i64(fsq);
            if ((threadIdx.x & 63) == 0) {
                atomicAdd(&s_sum[c0], (unsigned long long)s1);
                atomicAdd(&s_sq[c0], (unsigned long long)s2);
                atomicAdd(&s_cnt[c0], 64u);
            }
        }
    } else if (cell >= 0) {
        atomicAdd(&s_sum[cell], (unsigned long long)fx);
        atomicAdd(&s_sq[cell], (unsigned long long)fsq);
        atomicAdd(&s_cnt[cell], 1u);
    }
}

constexpr int kPayoffStreamThreads = 512;
constexpr int kPayoffStreamBatch = 2;     // envs per thread per iteration (loads in flight)

// The incidences of one env whose seats' returns and ids are in registers.
template <int NA>
__device__ __forceinline__ void stream_env(unsigned long long* s_sum, unsigned long long* s_sq,
                                           unsigned int* s_cnt, const float (&g)[NA],
                                           const int (&pid)[NA], uint32_t team_row,
                                           uint32_t team_col, int P)
{
#pragma unroll
    for (int a = 0; a < NA; ++a) {
        if (!((team_row >> a) & 1u))
            continue;
        const double gd = (double)g[a];
        const long long fx = __double2ll_rn(gd * 4294967296.0);
        const long long fsq = __double2ll_rn(gd * gd * 1048576.0);
#pragma unroll
        for (int b = 0; b < NA; ++b) {
            if (!((team_col >> b) & 1u))
                continue;
            // lanes past the range carry id -1, hence cell -1: a partial
            // wavefront never takes the shuffle path with them
            const int cell = (pid[a] >= 0 && pid[a] < P && pid[b] >= 0 && pid[b] < P)
                                 ? pid[a] * P + pid[b]
                                 : -1;
            lds_incidence(s_sum, s_sq, s_cnt, cell, fx, fsq);
        }
    }
}

// NA: seats per env known at compile time (2), or 0 (any count, one env per
// thread per iteration)
template <int CELLS, int NA>
__global__ __launch_bounds__(kPayoffStreamThreads) void payoff_stream_kernel(
    const float* __restrict__ ret, const int32_t* __restrict__ pids, int64_t n, int n_agents,
    uint32_t team_row, uint32_t team_col, int P, unsigned long long* __restrict__ sum,
    unsigned long long* __restrict__ sumsq, unsigned long long* __restrict__ cnt)
{
    __shared__ unsigned long long s_sum[CELLS], s_sq[CELLS];
    __shared__ unsigned int s_cnt[CELLS];
    const int cells = P * P;
    for (int c = threadIdx.x; c < cells; c += kPayoffStreamThreads) {
        s_sum[c] = 0;
        s_sq[c] = 0;
        s_cnt[c] = 0;
    }
    __syncthreads();
    const int64_t e0 = n * blockIdx.x / gridDim.x, e1 = n * (blockIdx.x + 1) / gridDim.x;
    if constexpr (NA > 0) {
        constexpr int kStep = kPayoffStreamThreads * kPayoffStreamBatch;
        // the loop bound is uniform over the workgroup (shuffles inside)
        for (int64_t base = e0; base < e1; base += kStep) {
            // every seat's return and id of this thread's envs first (all
            // loads in flight together), then the incidences
            float g[kPayoffStreamBatch][NA];
            int pid[kPayoffStreamBatch][NA];
#pragma unroll
            for (int k = 0; k < kPayoffStreamBatch; ++k) {
                const int64_t e = base + k * kPayoffStreamThreads + threadIdx.x;
                const bool valid = e < e1;
#pragma unroll
                for (int a = 0; a < NA; ++a) {
                    pid[k][a] = valid ? pids[e * NA + a] : -1;
                    g[k][a] = valid && ((team_row >> a) & 1u) ? ret[(int64_t)a * n + e] : 0.f;
                }
            }
#pragma unroll
            for (int k = 0; k < kPayoffStreamBatch; ++k)
                stream_env<NA>(s_sum, s_sq, s_cnt, g[k], pid[k], team_row, team_col, P);
        }
    } else {
        for (int64_t base = e0; base < e1; base += kPayoffStreamThreads) {
            const int64_t e = base + threadIdx.x;
            const bool valid = e < e1;
            for (int a = 0; a < n_agents; ++a) {
                if (!((team_row >> a) & 1u))
                    continue;
                long long fx = 0, fsq = 0;
                int pa = -1;
                if (valid) {
                    const double gd = (double)ret[(int64_t)a * n + e];
                    fx = __double2ll_rn(gd * 4294967296.0);
                    fsq = __double2ll_rn(gd * gd * 1048576.0);
                    pa = pids[e * n_agents + a];
                }
                for (int b = 0; b < n_agents; ++b) {
                    if (!((team_col >> b) & 1u))
                        continue;
                    const int pb = valid ? pids[e * n_agents + b] : -1;
                    const int cell =
                        (pa >= 0 && pa < P && pb >= 0 && pb < P) ? pa * P + pb : -1;
                    lds_incidence(s_sum, s_sq, s_cnt, cell, fx, fsq);
                }
            }
        }
    }
    __syncthreads();
    for (int c = threadIdx.x; c < cells; c += kPayoffStreamThreads) {
        const unsigned int k = s_cnt[c];
        if (k) {
            atomicAdd(&sum[c], s_sum[c]);
            atomicAdd(&sumsq[c], s_sq[c]);
            atomicAdd(&cnt[c], (unsigned long long)k);
        }
    }
}

// Larger populations: from the slots sorted by policy id (the bucketing of
// the policy forward).  The sorted slot list is cut into equal ranges, one
// per workgroup, so that a heavily played policy spreads over many
// workgroups; a range holds one or a few policy segments.  For each segment
// (row policy p) the row-side slots add their env's incidences (p, id of each
// column-side seat) into one row of P cells in LDS, which is then added to the
// table with one set of global atomics per touched cell.  Each thread keeps
// kPayoffBatch slots' loads in flight.  Slots whose id is out of range (the
// bucketing files them under policy 0) are skipped.
constexpr int kPayoffThreads = 256;
constexpr int kPayoffBatch = 4;

__global__ __launch_bounds__(kPayoffThreads) void payoff_bucketed_kernel(
    const float* __restrict__ ret, const int32_t* __restrict__ pids,
    const int32_t* __restrict__ perm, const int32_t* __restrict__ offsets, int64_t n,
    int n_agents, uint32_t team_row, uint32_t team_col, int P, int64_t rows_per_wg,
    unsigned long long* __restrict__ sum, unsigned long long* __restrict__ sumsq,
    unsigned long long* __restrict__ cnt)
{
    __shared__ unsigned long long s_sum[kMaxP], s_sq[kMaxP];
    __shared__ unsigned int s_cnt[kMaxP];
    __shared__ int s_off[kMaxP + 1];
    const int64_t ns = n * n_agents;
    const int64_t r0 = (int64_t)blockIdx.x * rows_per_wg;
    const int64_t r1 = r0 + rows_per_wg < ns ? r0 + rows_per_wg : ns;
    for (int c = threadIdx.x; c <= P; c += kPayoffThreads)
        s_off[c] = offsets[c];
    __syncthreads();
    // first policy whose segment reaches past r0 (offsets is non-decreasing,
    // offsets[0] = 0, offsets[P] = ns)
    int p = 0;
    {
        int lo = 0, hi = P - 1;
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (s_off[mid] <= r0)
                lo = mid;
            else
                hi = mid - 1;
        }
        p = lo;
    }
    for (; p < P && s_off[p] < r1; ++p) {
        const int64_t s0 = s_off[p] > r0 ? s_off[p] : r0;
        const int64_t s1 = s_off[p + 1] < r1 ? s_off[p + 1] : r1;
        if (s0 >= s1)
            continue;          // uniform over the workgroup
        for (int c = threadIdx.x; c < P; c += kPayoffThreads) {
            s_sum[c] = 0;
            s_sq[c] = 0;
            s_cnt[c] = 0;
        }
        __syncthreads();
        for (int64_t r = s0 + threadIdx.x; r < s1; r += (int64_t)kPayoffThreads * kPayoffBatch) {
            int slot[kPayoffBatch], pid[kPayoffBatch];
            float g[kPayoffBatch];
#pragma unroll
            for (int k = 0; k < kPayoffBatch; ++k) {
                const int64_t rk = r + (int64_t)k * kPayoffThreads;
                slot[k] = rk < s1 ? perm[rk] : -1;
            }
#pragma unroll
            for (int k = 0; k < kPayoffBatch; ++k) {
                pid[k] = -1;
                g[k] = 0.f;
                if (slot[k] >= 0) {
                    const int64_t e = slot[k] / n_agents, a = slot[k] - e * n_agents;
                    if ((team_row >> a) & 1u) {
                        pid[k] = pids[slot[k]];
                        g[k] = ret[a * n + e];
                    }
                }
            }
#pragma unroll
            for (int k = 0; k < kPayoffBatch; ++k) {
                if (pid[k] != p)
                    continue;
                const int64_t e = slot[k] / n_agents;
                const double gd = (double)g[k];
                const long long fx = __double2ll_rn(gd * 4294967296.0);
                const long long fsq = __double2ll_rn(gd * gd * 1048576.0);
                for (int b = 0; b < n_agents; ++b) {
                    if (!((team_col >> b) & 1u))
                        continue;
                    const int pb = pids[e * n_agents + b];
                    if (pb < 0 || pb >= P)
                        continue;
                    atomicAdd(&s_sum[pb], (unsigned long long)fx);
                    atomicAdd(&s_sq[pb], (unsigned long long)fsq);
                    atomicAdd(&s_cnt[pb], 1u);
                }
            }
        }
        __syncthreads();
        for (int c = threadIdx.x; c < P; c += kPayoffThreads) {
            const unsigned int k = s_cnt[c];
            if (k) {
                const int64_t cell = (int64_t)p * P + c;
                atomicAdd(&sum[cell], s_sum[c]);
                atomicAdd(&sumsq[cell], s_sq[c]);
                atomicAdd(&cnt[cell], (unsigned long long)k);
            }
        }
        __syncthreads();       // the row is cleared for the next segment
    }
}

hipError_t launch_payoff_bucketed(const float* ret, const int32_t* pids, const int32_t* perm,
                                  const int32_t* offsets, int64_t n_envs, int n_agents,
                                  uint32_t team_row, uint32_t team_col, int P, int n_cus,
                                  unsigned long long* sum, unsigned long long* sumsq,
                                  unsigned long long* cnt, hipStream_t s)
{
    const int64_t ns = n_envs * n_agents;
    // about four workgroups per CU, at least 256 slots each
    const int64_t want = std::max<int64_t>(1, std::min<int64_t>(4 * (int64_t)n_cus,
                                                                (ns + 255) / 256));
    const int64_t rows = (ns + want - 1) / want;
    const int grid = (int)((ns + rows - 1) / rows);
    payoff_bucketed_kernel<<<grid, kPayoffThreads, 0, s>>>(ret, pids, perm, offsets, n_envs,
                                                           n_agents, team_row, team_col, P,
                                                           rows, sum, sumsq, cnt);
    return hipGetLastError();
}

bool payoff_stream_fits(int P)
{
    return P * P <= kPayoffStreamMaxCells;
}

hipError_t launch_payoff_stream(const float* ret, const int32_t* pids, int64_t n_envs,
                                int n_agents, uint32_t team_row, uint32_t team_col, int P,
                                int n_cus, unsigned long long* sum, unsigned long long* sumsq,
                                unsigned long long* cnt, hipStream_t s)
{
    const int cells = P * P;
    // up to four workgroups per CU (two for the 80 KB table), at least 1024
    // envs each
    const int per_cu = cells <= 1024 ? 4 : 2;
    const int grid = (int)std::max<int64_t>(
        1, std::min<int64_t>((int64_t)per_cu * n_cus, (n_envs + 1023) / 1024));
    auto go = [&](auto cells_c) {
        constexpr int C = decltype(cells_c)::value;
        if (n_agents == 2)
            payoff_stream_kernel<C, 2><<<grid, kPayoffStreamThreads, 0, s>>>(
                ret, pids, n_envs, n_agents, team_row, team_col, P, sum, sumsq, cnt);
        else
            payoff_stream_kernel<C, 0><<<grid, kPayoffStreamThreads, 0, s>>>(
                ret, pids, n_envs, n_agents, team_row, team_col, P, sum, sumsq, cnt);
    };
    if (cells <= 256)
        go(std::integral_constant<int, 256>{});
    else if (cells <= 1024)
        go(std::integral_constant<int, 1024>{});
    else if (cells <= kPayoffStreamMaxCells)
        go(std::integral_constant<int, kPayoffStreamMaxCells>{});
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

hipError_t launch_payoff(const float* ret, const int32_t* pids, int64_t n_envs, int n_agents,
                         const int8_t* team, int P, unsigned long long* sum,
                         unsigned long long* sumsq, unsigned long long* cnt, hipStream_t s)
{
    EnvArgs ea{};
    for (int k = 0; k < n_agents; ++k) {
        if (team[k] > 0)
            ea.team_row |= 1u << k;
        else if (team[k] < 0)
            ea.team_col |= 1u << k;
    }
    payoff_kernel<<<(int)((n_envs + 255) / 256), 256, 0, s>>>(ret, pids, n_envs, n_agents, ea,
                                                              P, sum, sumsq, cnt);
    return hipGetLastError();
}

}  // namespace malib
