// Grouped policy forward: every agent slot is evaluated by the policy its
// seat plays (a heterogeneous policy combination per env, MALib Sec. 3.1).
// Slots are bucketed by policy id beforehand, so each workgroup (bf16) or
// wavefront (fp32) runs rows of a single policy with one set of weights.
//
//  tabular   logits = tab[pid]
//  mlp_f32   fp32 MLP, one row per lane; the policy is wave-uniform, so the
//            weights stream through the scalar cache as SGPR operands
//  mlp_bf16  bf16 MLP on v_mfma_f32_32x32x16_bf16: a 128-row tile per
//            workgroup; observations are built in LDS, hidden activations stay
//            in LDS, weights come pre-packed in MFMA fragment order
#include "device.hpp"
#include "internal.hpp"

namespace malib {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

// ------------------------------------------------------------------ packing

// Fragment layout of one layer (out rows padded to 32, in columns to 16):
//   frag[p][nt][ks][lane] = 8 bf16: W[p][nt*32 + lane%32][ks*16 + (lane/32)*8 + j]
// which is the A operand of v_mfma_f32_32x32x16_bf16 for output tile nt and
// k-step ks, so a wavefront loads it as 1 KiB contiguous.
__global__ void pack_bf16_kernel(const float* __restrict__ w, int P, int out, int in,
                                 int out_pad, int in_pad, uint4* __restrict__ dst)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    int nts = out_pad / 32, kss = in_pad / 16;
    int64_t total = (int64_t)P * nts * kss * 64;
    if (i >= total)
        return;
    int lane = (int)(i % 64);
    int64_t r = i / 64;
    int ks = (int)(r % kss);
    r /= kss;
    int nt = (int)(r % nts);
    int p = (int)(r / nts);
    int row = nt * 32 + (lane & 31);
    int col0 = ks * 16 + (lane >> 5) * 8;
    uint32_t v[4];
    for (int q = 0; q < 4; ++q) {
        float lo = 0.0f, hi = 0.0f;
        int c = col0 + 2 * q;
        if (row < out && c < in)
            lo = w[((int64_t)p * out + row) * in + c];
        if (row < out && c + 1 < in)
            hi = w[((int64_t)p * out + row) * in + c + 1];
        v[q] = pack_bf16x2(lo, hi);
    }
    dst[i] = make_uint4(v[0], v[1], v[2], v[3]);
}

hipError_t launch_pack_bf16(const float* w, int P, int out, int in, int out_pad, int in_pad,
                            void* dst, hipStream_t s)
{
    int64_t total = (int64_t)P * (out_pad / 32) * (in_pad / 16) * 64;
    pack_bf16_kernel<<<(int)((total + 255) / 256), 256, 0, s>>>(w, P, out, in, out_pad, in_pad,
                                                               (uint4*)dst);
    return hipGetLastError();
}

// ------------------------------------------------------------------ tabular

__global__ void tabular_kernel(const float* __restrict__ tab, const int32_t* __restrict__ pids,
                               int64_t n_slots, int A, int P, int* flags,
                               float* __restrict__ logits)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n_slots)
        return;
    int p = pids[i];
    if (p < 0 || p >= P) {
        atomicOr(flags, kErrPid);
        p = 0;
    }
    for (int a = 0; a < A; ++a)
        logits[i * A + a] = tab[p * A + a];
}

hipError_t launch_tabular(const float* tab, const int32_t* pids, int64_t n_slots, int A, int P,
                          int* flags, float* logits, hipStream_t s)
{
    tabular_kernel<<<(int)((n_slots + 255) / 256), 256, 0, s>>>(tab, pids, n_slots, A, P, flags,
                                                               logits);
    return hipGetLastError();
}

// ------------------------------------------------------------ tile lookup

// Tile t of the bucketed slots: the policy p with tile_off[p] <= t < tile_off[p+1]
// and its row range in perm.
__device__ __forceinline__ int tile_policy(const int32_t* __restrict__ tile_off, int P, int t)
{
    int lo = 0, hi = P - 1;
    while (lo < hi) {
        int mid = (lo + hi + 1) >> 1;
        if (tile_off[mid] <= t)
            lo = mid;
        else
            hi = mid - 1;
    }
    return lo;
}

// ------------------------------------------------------------------ fp32 MLP

// Iterated matrix game observation element c (0..8A-1) of a seat: lag c/(2A),
// own action block first.  hist holds 4-bit joint actions a0*3+a1, 15 = none.
__device__ __forceinline__ float iter_obs(uint32_t hist, int seat, int A, int c)
{
    int lag = c / (2 * A), r = c % (2 * A);
    uint32_t j = (hist >> (4 * lag)) & 15u;
    if (j == 15u)
        return 0.0f;
    int a0 = (int)j / 3, a1 = (int)j % 3;
    int own = seat == 0 ? a0 : a1, other = seat == 0 ? a1 : a0;
    return (r < A) ? (r == own ? 1.0f : 0.0f) : (r - A == other ? 1.0f : 0.0f);
}

struct MlpF32Args {
    const float* w1; const float* w2; const float* w3;
    const float* b1; const float* b2; const float* b3;
    const int32_t* perm; const int32_t* offsets; const int32_t* tile_off;
    const uint16_t* hist;
    float* logits;
    int P, A, IN, n_agents;
};

template <int HID, int IN, int AMAX>
__global__ __launch_bounds__(256) void mlp_f32_kernel(MlpF32Args a)
{
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int t = blockIdx.x * 4 + wave;
    if (t >= a.tile_off[a.P])
        return;
    int p = tile_policy(a.tile_off, a.P, t);
    p = __builtin_amdgcn_readfirstlane(p);
    const int r0 = a.offsets[p] + (t - a.tile_off[p]) * kF32TileRows;
    const int r1 = min(r0 + kF32TileRows, a.offsets[p + 1]);
    const int row = r0 + lane;
    const bool valid = row < r1;
    const int slot = a.perm[valid ? row : r0];
    const int env = slot / a.n_agents, seat = slot - env * a.n_agents;
    const uint32_t hist = a.hist[env];

    const float* W1 = a.w1 + (int64_t)p * HID * IN;
    const float* W2 = a.w2 + (int64_t)p * HID * HID;
    const float* W3 = a.w3 + (int64_t)p * a.A * HID;
    const float* B1 = a.b1 + p * HID;
    const float* B2 = a.b2 + p * HID;
    const float* B3 = a.b3 + p * a.A;

    float x[IN];
#pragma unroll
    for (int c = 0; c < IN; ++c)
        x[c] = iter_obs(hist, seat, a.A, c);
    float h1[HID];
#pragma unroll
    for (int j = 0; j < HID; ++j) {
        float acc = B1[j];
#pragma unroll
        for (int c = 0; c < IN; ++c)
            acc = __builtin_fmaf(W1[j * IN + c], x[c], acc);
        h1[j] = acc > 0.0f ? acc : 0.0f;
    }
    float h2[HID];
#pragma unroll
    for (int j = 0; j < HID; ++j) {
        float acc = B2[j];
#pragma unroll
        for (int k = 0; k < HID; ++k)
            acc = __builtin_fmaf(W2[j * HID + k], h1[k], acc);
        h2[j] = acc > 0.0f ? acc : 0.0f;
    }
    if (valid) {
        float* out = a.logits + (int64_t)slot * a.A;
#pragma unroll
        for (int o = 0; o < AMAX; ++o) {
            if (o < a.A) {
                float acc = B3[o];
#pragma unroll
                for (int k = 0; k < HID; ++k)
                    acc = __builtin_fmaf(W3[o * HID + k], h2[k], acc);
                out[o] = acc;
            }
        }
    }
}

hipError_t launch_mlp_f32(const Pop& pop, const int32_t* perm, const int32_t* offsets,
                          const int32_t* tile_off, int64_t n_slots, int n_agents,
                          const void* state, float* logits, hipStream_t s)
{
    MlpF32Args a;
    a.w1 = (const float*)pop.w[0];
    a.w2 = (const float*)pop.w[1];
    a.w3 = (const float*)pop.w[2];
    a.b1 = pop.b[0];
    a.b2 = pop.b[1];
    a.b3 = pop.b[2];
    a.perm = perm;
    a.offsets = offsets;
    a.tile_off = tile_off;
    a.hist = (const uint16_t*)state;
    a.logits = logits;
    a.P = pop.P;
    a.A = pop.A;
    a.IN = pop.in_dim;
    a.n_agents = n_agents;
    int64_t max_tiles = (n_slots + kF32TileRows - 1) / kF32TileRows + pop.P;
    int blocks = (int)((max_tiles + 3) / 4);
    if (pop.in_dim != 24 || pop.A > 3)
        return hipErrorInvalidValue;
    if (pop.hid == 32)
        mlp_f32_kernel<32, 24, 3><<<blocks, 256, 0, s>>>(a);
    else if (pop.hid == 64)
        mlp_f32_kernel<64, 24, 3><<<blocks, 256, 0, s>>>(a);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

// ------------------------------------------------------------------ bf16 MLP

enum { kObsFeature = 0, kObsPursuit = 1, kObsIter = 2 };

constexpr int kLdw = 520;           // LDS row stride (bf16): 512 + 8 to spread banks
constexpr int kMlpThreads = 512;    // 8 wavefronts

struct MlpBf16Args {
    const uint4* w1; const uint4* w2; const uint4* w3;
    const float* b1; const float* b2; const float* b3;
    const int32_t* perm; const int32_t* offsets; const int32_t* tile_off;
    const void* state;
    float* logits;
    int P, A, in_dim, in_pad, n_agents, grid, d;
    int64_t n_envs;
    int n_blocks;                   // launched workgroups (a multiple of 8)
};

// One MFMA layer of a wavefront: output tiles (n-tiles nt0.., row-tiles rt0..)
// = W[nt] (32 x 16 per k-step, from the packed fragments) x X^T[rt] (16 x 32,
// from LDS rows).  acc[nt][rt] register r, lane i holds output unit
// nt*32 + (r/4)*8 + (i/32)*4 + r%4 of tile row rt*32 + i%32.
template <int NT, int RT>
__device__ __forceinline__ void mfma_layer(const uint4* __restrict__ frag, int ksteps, int nt0,
                                           int rt0, const uint16_t* buf, int lane,
                                           f32x16 (&acc)[NT][RT])
{
#pragma unroll
    for (int n = 0; n < NT; ++n)
#pragma unroll
        for (int r = 0; r < RT; ++r)
            acc[n][r] = f32x16{};
    const int brow = lane & 31, bcol = (lane >> 5) * 8;
    uint4 a_cur[NT];
#pragma unroll
    for (int n = 0; n < NT; ++n)
        a_cur[n] = frag[((int64_t)(nt0 + n) * ksteps + 0) * 64 + lane];
    for (int ks = 0; ks < ksteps; ++ks) {
        uint4 a_nxt[NT];
        if (ks + 1 < ksteps) {
#pragma unroll
            for (int n = 0; n < NT; ++n)
                a_nxt[n] = frag[((int64_t)(nt0 + n) * ksteps + ks + 1) * 64 + lane];
        }
        uint4 b[RT];
#pragma unroll
        for (int r = 0; r < RT; ++r)
            b[r] = *reinterpret_cast<const uint4*>(buf + ((rt0 + r) * 32 + brow) * kLdw + ks * 16 + bcol);
#pragma unroll
        for (int n = 0; n < NT; ++n)
#pragma unroll
            for (int r = 0; r < RT; ++r)
                acc[n][r] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    __builtin_bit_cast(bf16x8, a_cur[n]), __builtin_bit_cast(bf16x8, b[r]),
                    acc[n][r], 0, 0, 0);
        if (ks + 1 < ksteps) {
#pragma unroll
            for (int n = 0; n < NT; ++n)
                a_cur[n] = a_nxt[n];
        }
    }
}

// bias + ReLU + bf16, written back as the next layer's input rows.
template <int NT, int RT>
__device__ __forceinline__ void hidden_epilogue(const f32x16 (&acc)[NT][RT], const float* bias,
                                                int nt0, int rt0, uint16_t* buf, int lane)
{
#pragma unroll
    for (int n = 0; n < NT; ++n) {
#pragma unroll
        for (int r = 0; r < RT; ++r) {
            int row = (rt0 + r) * 32 + (lane & 31);
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                int u0 = (nt0 + n) * 32 + g * 8 + (lane >> 5) * 4;
                float4 bb = *reinterpret_cast<const float4*>(bias + u0);
                float v0 = acc[n][r][g * 4 + 0] + bb.x;
                float v1 = acc[n][r][g * 4 + 1] + bb.y;
                float v2 = acc[n][r][g * 4 + 2] + bb.z;
                float v3 = acc[n][r][g * 4 + 3] + bb.w;
                v0 = v0 > 0.0f ? v0 : 0.0f;
                v1 = v1 > 0.0f ? v1 : 0.0f;
                v2 = v2 > 0.0f ? v2 : 0.0f;
                v3 = v3 > 0.0f ? v3 : 0.0f;
                uint2 pk = make_uint2(pack_bf16x2(v0, v1), pack_bf16x2(v2, v3));
                *reinterpret_cast<uint2*>(buf + row * kLdw + u0) = pk;
            }
        }
    }
}

template <int HID>
struct HidSplit {
    // wavefront grid for a HID-wide layer over the 4 row-tiles
    static constexpr int NT = HID >= 512 ? 2 : 1;
    static constexpr int RT = HID >= 256 ? 4 : (HID == 128 ? 2 : 1);
    static constexpr int NGROUPS = (HID / 32) / NT;
};

template <int HID, int OBS>
__global__ __launch_bounds__(kMlpThreads) void mlp_bf16_kernel(MlpBf16Args a)
{
    __shared__ __attribute__((aligned(16))) uint16_t buf[kTileRows * kLdw];
    __shared__ int row_slot[kTileRows];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

    // workgroups are dispatched round-robin over the 8 XCDs: give each XCD a
    // contiguous run of tiles so that a policy's tiles share one L2
    const int per = a.n_blocks / 8;
    const int t = (blockIdx.x & 7) * per + (blockIdx.x >> 3);
    const int total = a.tile_off[a.P];
    if (t >= total)
        return;
    const int p = tile_policy(a.tile_off, a.P, t);
    const int r0 = a.offsets[p] + (t - a.tile_off[p]) * kTileRows;
    const int nrows = min(kTileRows, a.offsets[p + 1] - r0);

    if (tid < kTileRows)
        row_slot[tid] = tid < nrows ? a.perm[r0 + tid] : -1;
    __syncthreads();

    // ---- observations -> LDS rows (bf16)
    if (OBS == kObsFeature) {
        const int q4 = a.in_pad / 4;
        const float* S = (const float*)a.state;
        for (int i = tid; i < kTileRows * q4; i += kMlpThreads) {
            int r = i / q4, c = (i - r * q4) * 4;
            int slot = row_slot[r];
            float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
            if (slot >= 0 && c < a.in_dim)
                v = *reinterpret_cast<const float4*>(S + (int64_t)(slot / a.n_agents) * a.d + c);
            uint2 pk = make_uint2(pack_bf16x2(v.x, v.y), pack_bf16x2(v.z, v.w));
            *reinterpret_cast<uint2*>(buf + r * kLdw + c) = pk;
        }
    } else if (OBS == kObsPursuit) {
        const uint8_t* pos = (const uint8_t*)a.state;
        for (int i = tid; i < kTileRows * a.in_pad; i += kMlpThreads) {
            int r = i / a.in_pad, c = i - r * a.in_pad;
            int slot = row_slot[r];
            float v = 0.0f;
            if (slot >= 0 && c < 75) {
                int64_t env = slot / a.n_agents;
                int seat = slot - (int)env * a.n_agents;
                int pc = pos[env], ec = pos[a.n_envs + env];
                int self = seat == 0 ? pc : ec;
                int o = c / 3, ch = c - o * 3;
                int dy = o / 5 - 2, dx = o % 5 - 2;
                int G = a.grid;
                int x = ((self % G) + dx + G) % G, y = ((self / G) + dy + G) % G;
                int cell = y * G + x;
                bool on = ch == 0 ? cell == pc : (ch == 1 ? cell == ec : (dx == 0 && dy == 0));
                v = on ? 1.0f : 0.0f;
            }
            buf[r * kLdw + c] = bf16_bits(v);
        }
    } else {
        const uint16_t* hist = (const uint16_t*)a.state;
        for (int i = tid; i < kTileRows * a.in_pad; i += kMlpThreads) {
            int r = i / a.in_pad, c = i - r * a.in_pad;
            int slot = row_slot[r];
            float v = 0.0f;
            if (slot >= 0 && c < a.in_dim) {
                int64_t env = slot / a.n_agents;
                int seat = slot - (int)env * a.n_agents;
                v = iter_obs(hist[env], seat, a.A, c);
            }
            buf[r * kLdw + c] = bf16_bits(v);
        }
    }
    __syncthreads();

    using S = HidSplit<HID>;
    const int nt0 = (wave % S::NGROUPS) * S::NT;
    const int rt0 = (wave / S::NGROUPS) * S::RT;
    f32x16 acc[S::NT][S::RT];

    // ---- layer 1: in_pad -> HID
    mfma_layer<S::NT, S::RT>(a.w1 + (int64_t)p * (HID / 32) * (a.in_pad / 16) * 64,
                             a.in_pad / 16, nt0, rt0, buf, lane, acc);
    __syncthreads();
    hidden_epilogue<S::NT, S::RT>(acc, a.b1 + p * HID, nt0, rt0, buf, lane);
    __syncthreads();
    // ---- layer 2: HID -> HID
    mfma_layer<S::NT, S::RT>(a.w2 + (int64_t)p * (HID / 32) * (HID / 16) * 64, HID / 16, nt0,
                             rt0, buf, lane, acc);
    __syncthreads();
    hidden_epilogue<S::NT, S::RT>(acc, a.b2 + p * HID, nt0, rt0, buf, lane);
    __syncthreads();
    // ---- layer 3: HID -> A (one 32-wide output tile; one row-tile per wave)
    if (wave < 4) {
        f32x16 o[1][1];
        mfma_layer<1, 1>(a.w3 + (int64_t)p * (HID / 16) * 64, HID / 16, 0, wave, buf, lane, o);
        int row = wave * 32 + (lane & 31);
        int slot = row < nrows ? row_slot[row] : -1;
        if (slot >= 0) {
            float* out = a.logits + (int64_t)slot * a.A;
            const float* b3 = a.b3 + p * a.A;
#pragma unroll
            for (int g = 0; g < 4; ++g)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    int u = g * 8 + (lane >> 5) * 4 + q;
                    if (u < a.A)
                        out[u] = o[0][0][g * 4 + q] + b3[u];
                }
        }
    }
}

hipError_t launch_mlp_bf16(const Pop& pop, int env_kind, int n_agents, int grid, int d,
                           const int32_t* perm, const int32_t* offsets, const int32_t* tile_off,
                           int64_t n_slots, const void* state, const uint8_t* done,
                           float* logits, hipStream_t s)
{
    (void)done;
    MlpBf16Args a;
    a.w1 = (const uint4*)pop.w[0];
    a.w2 = (const uint4*)pop.w[1];
    a.w3 = (const uint4*)pop.w[2];
    a.b1 = pop.b[0];
    a.b2 = pop.b[1];
    a.b3 = pop.b[2];
    a.perm = perm;
    a.offsets = offsets;
    a.tile_off = tile_off;
    a.state = state;
    a.logits = logits;
    a.P = pop.P;
    a.A = pop.A;
    a.in_dim = pop.in_dim;
    a.in_pad = pop.in_pad;
    a.n_agents = n_agents;
    a.grid = grid;
    a.d = d;
    a.n_envs = n_slots / n_agents;
    int64_t max_tiles = (n_slots + kTileRows - 1) / kTileRows + pop.P;
    int blocks = (int)((max_tiles + 7) / 8 * 8);
    a.n_blocks = blocks;
    int obs = env_kind == MALIB_ENV_FEATURE ? kObsFeature
              : env_kind == MALIB_ENV_PURSUIT ? kObsPursuit : kObsIter;
#define MALIB_MLP_CASE(H)                                                                   \
    if (pop.hid == H) {                                                                     \
        if (obs == kObsFeature)                                                             \
            mlp_bf16_kernel<H, kObsFeature><<<blocks, kMlpThreads, 0, s>>>(a);              \
        else if (obs == kObsPursuit)                                                        \
            mlp_bf16_kernel<H, kObsPursuit><<<blocks, kMlpThreads, 0, s>>>(a);              \
        else                                                                                \
            mlp_bf16_kernel<H, kObsIter><<<blocks, kMlpThreads, 0, s>>>(a);                 \
        return hipGetLastError();                                                           \
    }
    MALIB_MLP_CASE(64)
    MALIB_MLP_CASE(128)
    MALIB_MLP_CASE(256)
    MALIB_MLP_CASE(512)
#undef MALIB_MLP_CASE
    return hipErrorInvalidValue;
}

}  // namespace malib
