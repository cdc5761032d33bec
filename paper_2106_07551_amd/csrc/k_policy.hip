// Grouped policy forward: every agent slot is evaluated by the policy its
// seat plays (a heterogeneous policy combination per env, MALib Sec. 3.1).
// Slots are bucketed by policy id beforehand, so each workgroup (bf16) or
// wavefront (fp32) runs rows of a single policy with one set of weights.
//
//  tabular   logits = tab[pid]
//  mlp_f32   fp32 MLP on v_mfma_f32_32x32x2_f32: one wavefront per 32-row
//            tile, the hidden layer kept in registers (weights packed in the
//            accumulators' k order)
//  mlp_bf16  bf16 MLP on v_mfma_f32_32x32x16_bf16: a 64-row tile per
//            workgroup (or, for wide feature observations, a persistent
//            workgroup per CU over 128-row tiles); observations are built in
//            LDS, the first hidden layer stays in LDS, the second feeds the
//            output layer from the accumulators; weights come pre-packed in
//            MFMA fragment order
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
//
// With kperm set, the k order inside each 32-wide block of inputs follows the
// accumulator layout of the previous layer's MFMA (register g*4+q of lane i
// holds unit (g*8 + (i/32)*4 + q) of its 32-unit tile): k-step ks takes
// registers of groups g = 2(ks%2), 2(ks%2)+1 of tile ks/2, so that a
// wavefront can feed its own accumulators, converted to bf16, as the B operand
// without a trip through LDS.  Element j of lane i of k-step ks is input
//   (ks/2)*32 + (2(ks%2) + j/4)*8 + (i/32)*4 + j%4.
__global__ void pack_bf16_kernel(const float* __restrict__ w, int P, int out, int in,
                                 int out_pad, int in_pad, int kperm, uint4* __restrict__ dst)
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
        if (kperm)
            c = (ks >> 1) * 32 + (2 * (ks & 1) + (q >> 1)) * 8 + (lane >> 5) * 4 + (2 * q & 3);
        if (row < out && c < in)
            lo = w[((int64_t)p * out + row) * in + c];
        if (row < out && c + 1 < in)
            hi = w[((int64_t)p * out + row) * in + c + 1];
        v[q] = pack_bf16x2(lo, hi);
    }
    dst[i] = make_uint4(v[0], v[1], v[2], v[3]);
}

hipError_t launch_pack_bf16(const float* w, int P, int out, int in, int out_pad, int in_pad,
                            int kperm, void* dst, hipStream_t s)
{
    if (kperm && in_pad % 32 != 0)
        return hipErrorInvalidValue;
    int64_t total = (int64_t)P * (out_pad / 32) * (in_pad / 16) * 64;
    pack_bf16_kernel<<<(int)((total + 255) / 256), 256, 0, s>>>(w, P, out, in, out_pad, in_pad,
                                                               kperm, (uint4*)dst);
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
    const int32_t* perm; const int4* tile_info;
    const uint16_t* hist;
    float* logits;
    int P, A, IN, n_agents, max_tiles;
};

// fp32 MLP of the iterated game on v_mfma_f32_32x32x2_f32: one wavefront per
// 32-row tile, HID/32 n-tiles (32 rows keep both accumulator sets within 64
// registers; the weight stream is then 256 bytes per 2 MFMAs, far below the
// load path).
//
// MFMA 32x32x2 layouts: A (32 x 2) lane i holds A[i%32][i/32], B (2 x 32)
// lane i holds B[i/32][i%32], the accumulator register 4g+q of lane i holds
// C[8g + 4(i/32) + q][i%32].  So lane i always works on row (slot) i%32 of
// its row tiles; its half h = i/32 picks which units or inputs it holds.
//
//   layer 1: B = the observation, built in place per lane (input 2s+h at
//            k-step s); A = W1 in natural k order;
//   layer 2: B = the layer-1 accumulators after ReLU, register r of n-tile nt
//            at k-step 16nt+r, which holds unit u = 32nt + 8(r/4) + 4h + r%4:
//            W2 is packed in that k order (pack_f32_kernel), so the hidden
//            layer never leaves the registers;
//   layer 3: (A <= 3 logits) on the VALU from the layer-2 accumulators, each
//            half-wave summing its 16 NT units, the halves added by a shuffle.
// Sums run in a different order than a plain loop; fp32 policies are compared
// with a relative tolerance.
typedef float f32x16_t __attribute__((ext_vector_type(16)));

// Hidden ReLU of the fp32 policies: the IEEE 754-2019 maximum with +0, so a
// NaN of either sign propagates to the logits (and raises the NaN flag).
__device__ __forceinline__ float relu_f32(float x)
{
    return __builtin_elementwise_maximum(x, 0.0f);
}

template <int HID, int AMAX>
__global__ __launch_bounds__(256) void mlp_f32_kernel(MlpF32Args a)
{
    constexpr int NT = HID / 32, RT = 1, K1 = 12, K2 = HID / 2;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, h = lane >> 5, nn = lane & 31;
    // the observation build and the VALU output layer at a raised issue
    // priority, the MFMA layers at the normal one, so that the SIMD's other
    // wavefronts' MFMA loops yield issue slots to them (259.1 -> 256.8 us per
    // launch on the iterated game, four alternating runs)
    __builtin_amdgcn_s_setprio(2);
    const int t = blockIdx.x * 4 + wave;
    if (t >= a.max_tiles)
        return;
    const int4 ti = a.tile_info[t];
    const int p = __builtin_amdgcn_readfirstlane(ti.x);
    if (p < 0)
        return;
    const int r0 = __builtin_amdgcn_readfirstlane(ti.y);
    const int r1 = r0 + __builtin_amdgcn_readfirstlane(ti.z);

    int slot[RT];
    bool valid[RT];
    float xb[RT][K1];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
        const int row = r0 + 32 * rt + nn;
        valid[rt] = row < r1;
        slot[rt] = a.perm[valid[rt] ? row : r0];
        const int env = slot[rt] / a.n_agents, seat = slot[rt] - env * a.n_agents;
        const uint32_t hist = a.hist[env];
        // 24 inputs: 3 actions (constant divisors in iter_obs)
#pragma unroll
        for (int s = 0; s < K1; ++s)
            xb[rt][s] = iter_obs(hist, seat, 3, 2 * s + h);
    }
    // each lane's A operands are contiguous in the packed weights (16-byte loads)
    const float* W1 = a.w1 + (int64_t)p * HID * 24;
    float w1[NT][K1];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int s4 = 0; s4 < K1 / 4; ++s4) {
            const float4 v = *reinterpret_cast<const float4*>(W1 + (nt * 64 + lane) * K1 + 4 * s4);
            w1[nt][4 * s4 + 0] = v.x;
            w1[nt][4 * s4 + 1] = v.y;
            w1[nt][4 * s4 + 2] = v.z;
            w1[nt][4 * s4 + 3] = v.w;
        }

    // accumulators start from the bias of their units (32nt + 8g + 4h + q)
    auto bias16 = [&](const float* b, int nt) {
        f32x16_t v;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const float4 x = *reinterpret_cast<const float4*>(b + p * HID + 32 * nt + 8 * g + 4 * h);
            v[4 * g + 0] = x.x;
            v[4 * g + 1] = x.y;
            v[4 * g + 2] = x.z;
            v[4 * g + 3] = x.w;
        }
        return v;
    };
    f32x16_t acc[NT][RT], acc2[NT][RT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
            acc[nt][rt] = bias16(a.b1, nt);
    // ---- layer 1
    __builtin_amdgcn_s_setprio(0);
#pragma unroll
    for (int s = 0; s < K1; ++s)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
            for (int rt = 0; rt < RT; ++rt)
                acc[nt][rt] = __builtin_amdgcn_mfma_f32_32x32x2f32(w1[nt][s], xb[rt][s],
                                                                   acc[nt][rt], 0, 0, 0);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                acc[nt][rt][r] = relu_f32(acc[nt][rt][r]);
    // ---- layer 2 (k-step s2 = 16 nt + r takes register r of n-tile nt); the
    // weights stream through a ring DEPTH k-steps ahead
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
            acc2[nt][rt] = bias16(a.b2, nt);
    // A operands in groups of 4 k-steps (one 16-byte load per n-tile), the next
    // group loaded while the current one is used (a deeper ring measured slower)
    const float* W2 = a.w2 + (int64_t)p * HID * HID;
    constexpr int QDEPTH = 1, KQ = K2 / 4;
    float4 ring[QDEPTH][NT];
#pragma unroll
    for (int d = 0; d < QDEPTH; ++d)
#pragma unroll
        for (int ont = 0; ont < NT; ++ont)
            ring[d][ont] = *reinterpret_cast<const float4*>(W2 + (ont * 64 + lane) * K2 + 4 * d);
#pragma unroll
    for (int sq = 0; sq < KQ; ++sq) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int s2 = 4 * sq + j;
#pragma unroll
            for (int ont = 0; ont < NT; ++ont) {
                const float4 g4 = ring[sq % QDEPTH][ont];
                const float wv = j == 0 ? g4.x : j == 1 ? g4.y : j == 2 ? g4.z : g4.w;
#pragma unroll
                for (int rt = 0; rt < RT; ++rt)
                    acc2[ont][rt] = __builtin_amdgcn_mfma_f32_32x32x2f32(
                        wv, acc[s2 / 16][rt][s2 % 16], acc2[ont][rt], 0, 0, 0);
            }
        }
        if (sq + QDEPTH < KQ) {
#pragma unroll
            for (int ont = 0; ont < NT; ++ont)
                ring[sq % QDEPTH][ont] = *reinterpret_cast<const float4*>(
                    W2 + (ont * 64 + lane) * K2 + 4 * (sq + QDEPTH));
        }
        __builtin_amdgcn_sched_barrier(0);
    }
    __builtin_amdgcn_s_setprio(2);
    // ---- layer 3: W3 packed per (action, n-tile, half) as 16 floats
    const float* W3 = a.w3 + (int64_t)p * a.A * HID;
#pragma unroll
    for (int o = 0; o < AMAX; ++o) {
        if (o < a.A) {
            float w3[NT][16];
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const float4 v =
                        *reinterpret_cast<const float4*>(W3 + ((o * NT + nt) * 2 + h) * 16 + 4 * g);
                    w3[nt][4 * g + 0] = v.x;
                    w3[nt][4 * g + 1] = v.y;
                    w3[nt][4 * g + 2] = v.z;
                    w3[nt][4 * g + 3] = v.w;
                }
            const float bo = a.b3[p * a.A + o];
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) {
                float part = 0.0f;
#pragma unroll
                for (int nt = 0; nt < NT; ++nt)
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const float v = acc2[nt][rt][r];
                        part = __builtin_fmaf(w3[nt][r], relu_f32(v), part);
                    }
                const float tot = part + __shfl_xor(part, 32);
                if (h == 0 && valid[rt])
                    a.logits[(int64_t)slot[rt] * a.A + o] = bo + tot;
            }
        }
    }
}

// fp32 weights [P][out][in] -> the MFMA operand layouts of mlp_f32_kernel:
//   layer 0: [P][nt][lane][s] = W1[32nt + lane%32][2s + lane/32]        (s < 12)
//   layer 1: [P][ont][lane][s] = W2[32ont + lane%32][u(s, lane/32)]     (s < HID/2)
// (a lane's operands of consecutive k-steps are contiguous)
//            with u(s, h) = 32(s/16) + 8((s%16)/4) + 4h + s%4
//   layer 2: [P][o][nt][h][r] = W3[o][32nt + 8(r/4) + 4h + r%4]
__global__ void pack_f32_kernel(const float* __restrict__ w, int P, int layer, int hid, int A,
                                float* __restrict__ dst)
{
    const int per = layer == 0 ? hid * 24 : layer == 1 ? hid * hid : A * hid;
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (int64_t)P * per)
        return;
    const int p = (int)(i / per), e = (int)(i - (int64_t)p * per);
    int out, in, in_dim;
    if (layer == 0) {
        const int s = e % 12, lane = (e / 12) % 64, nt = e / (64 * 12);
        out = 32 * nt + lane % 32;
        in = 2 * s + lane / 32;
        in_dim = 24;
    } else if (layer == 1) {
        const int K2 = hid / 2;
        const int s = e % K2, lane = (e / K2) % 64, ont = e / (64 * K2);
        const int hh = lane / 32, r = s % 16;
        out = 32 * ont + lane % 32;
        in = 32 * (s / 16) + 8 * (r / 4) + 4 * hh + r % 4;
        in_dim = hid;
    } else {
        const int NT = hid / 32;
        const int r = e % 16, hh = (e / 16) % 2, nt = (e / 32) % NT, o = e / (32 * NT);
        out = o;
        in = 32 * nt + 8 * (r / 4) + 4 * hh + r % 4;
        in_dim = hid;
    }
    dst[i] = w[(int64_t)p * per + (int64_t)out * in_dim + in];
}

hipError_t launch_pack_f32(const float* w, int P, int layer, int hid, int A, float* dst,
                           hipStream_t s)
{
    const int per = layer == 0 ? hid * 24 : layer == 1 ? hid * hid : A * hid;
    const int64_t total = (int64_t)P * per;
    pack_f32_kernel<<<(int)((total + 255) / 256), 256, 0, s>>>(w, P, layer, hid, A, dst);
    return hipGetLastError();
}

hipError_t launch_mlp_f32(const Pop& pop, const int32_t* perm, const int4* tile_info,
                          int64_t n_slots, int n_agents, const void* state, float* logits,
                          hipStream_t s)
{
    MlpF32Args a;
    a.w1 = (const float*)pop.w[0];
    a.w2 = (const float*)pop.w[1];
    a.w3 = (const float*)pop.w[2];
    a.b1 = pop.b[0];
    a.b2 = pop.b[1];
    a.b3 = pop.b[2];
    a.perm = perm;
    a.tile_info = tile_info;
    a.hist = (const uint16_t*)state;
    a.logits = logits;
    a.P = pop.P;
    a.A = pop.A;
    a.IN = pop.in_dim;
    a.n_agents = n_agents;
    // tile_info holds max_tiles_for() entries; a wave past them would read out
    // of range, so the grid covers exactly that many wavefronts (rounded down
    // to whole workgroups plus one guarded workgroup)
    const int max_tiles = max_tiles_for(n_slots, pop.P, kF32TileRows);
    a.max_tiles = max_tiles;
    int blocks = (max_tiles + 3) / 4;
    if (pop.in_dim != 24 || pop.A != 3)
        return hipErrorInvalidValue;   // the iterated game: 3 actions, 8 x 3 inputs
    if (pop.hid == 32)
        mlp_f32_kernel<32, 3><<<blocks, 256, 0, s>>>(a);
    else if (pop.hid == 64)
        mlp_f32_kernel<64, 3><<<blocks, 256, 0, s>>>(a);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

// ------------------------------------------------------------------ bf16 MLP

enum { kObsFeature = 0, kObsPursuit = 1, kObsIter = 2 };

constexpr int kLdw = 520;           // LDS row stride (bf16): 512 + 8 to spread banks

struct MlpBf16Args {
    const uint4* w1; const uint4* w2; const uint4* w3;
    const float* b1; const float* b2; const float* b3;
    const int32_t* perm; const int32_t* perm_env; const int4* tile_info;
    // feature observations: bf16 rows [n_envs][d] (bf16_rne of the state) for
    // the 64-row kernel, the fp32 state for the persistent one; pursuit: the
    // env positions; iterated game: the action histories
    const void* state;
    float* logits;
    int P, A, in_dim, n_agents, grid, d;
    int64_t n_envs;
    int n_blocks;                   // launched workgroups (a multiple of 8)
    int max_tiles;                  // entries of tile_info
    const int32_t* tile_off;        // persistent kernel: tile_off[P] = number of tiles
    // Gumbel-max sampling inside the 64-row kernel (feature observations):
    // actions [n_slots] (null: the env step samples from the logits), the
    // Philox key, global env offset and step, and the device error flags
    uint8_t* actions;
    int* flags;
    uint64_t seed;
    int64_t env_offset;
    int t;
};

// Weight fragments of one layer of one policy, read through a buffer resource:
// the base address and size sit in scalar registers, each load takes the
// lane's byte offset (lane * 16, one VGPR for all loads) and the fragment's
// wave-uniform byte offset in a scalar register, so no 64-bit per-lane
// addresses are kept.  Loads beyond n_frags fragments return zero.
using Frags = __amdgpu_buffer_rsrc_t;

__device__ __forceinline__ Frags frag_src(const uint4* base, int n_frags)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint4*>(base), (short)0, n_frags * 1024,
                                             0x00020000);
}

__device__ __forceinline__ uint4 load_frag(Frags src, int idx, uint32_t loff)
{
    const auto v = __builtin_amdgcn_raw_buffer_load_b128(src, (int)loff, idx * 1024, 0);
    return make_uint4(v[0], v[1], v[2], v[3]);
}

// Ring of weight fragments of one layer: k-steps s, s+1, ... in flight, so a
// wavefront's weight loads are issued DEPTH-1 steps ahead of their MFMAs (and
// the first DEPTH steps of a layer before the preceding phase's LDS work).
template <int NT, int DEPTH>
struct WRing {
    uint4 a[DEPTH][NT];
};

template <int NT, int DEPTH>
__device__ __forceinline__ void ring_fill(WRing<NT, DEPTH>& ring, Frags frag,
                                          int ksteps, int nt0, int lane)
{
#pragma unroll
    for (int s = 0; s < DEPTH; ++s)
        if (s < ksteps)
#pragma unroll
            for (int n = 0; n < NT; ++n)
                ring.a[s][n] = load_frag(frag, (nt0 + n) * ksteps + s, lane * 16u);
}

// One MFMA layer of a wavefront: output tiles (n-tiles nt0.., row-tiles rt0..)
// = bias + W[nt] (32 x 16 per k-step, packed fragments) x X^T[rt] (16 x 32, LDS
// rows).  acc[nt][rt] register r, lane i holds output unit nt*32 + (r/4)*8 +
// (i/32)*4 + r%4 of tile row rt*32 + i%32.  The ring must hold k-steps
// 0..DEPTH-1.  (The fp32 sum order of a unit is the bias, then the k-steps.)
// PRIO: the wave runs the k-loop at the normal issue priority and returns to
// the raised one after it (see mlp_bf16_kernel).
template <int NT, int RT, int DEPTH, int LDW = kLdw, bool PRIO = false>
__device__ __forceinline__ void mfma_layer(WRing<NT, DEPTH>& ring, Frags frag, int ksteps,
                                           int nt0,
                                           int rt0, const uint16_t* buf, int lane,
                                           const float* __restrict__ bias, f32x16 (&acc)[NT][RT])
{
    // accumulators start from the bias of their output units
#pragma unroll
    for (int n = 0; n < NT; ++n) {
        f32x16 b0;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const float4 bb = *reinterpret_cast<const float4*>(
                bias + (nt0 + n) * 32 + g * 8 + (lane >> 5) * 4);
            b0[g * 4 + 0] = bb.x;
            b0[g * 4 + 1] = bb.y;
            b0[g * 4 + 2] = bb.z;
            b0[g * 4 + 3] = bb.w;
        }
#pragma unroll
        for (int r = 0; r < RT; ++r)
            acc[n][r] = b0;
    }
    const int brow = lane & 31, bcol = (lane >> 5) * 8;
    const uint16_t* bp[RT];
#pragma unroll
    for (int r = 0; r < RT; ++r)
        bp[r] = buf + ((rt0 + r) * 32 + brow) * LDW + bcol;
    uint4 b[2][RT];
#pragma unroll
    for (int r = 0; r < RT; ++r)
        b[0][r] = *reinterpret_cast<const uint4*>(bp[r]);

    if constexpr (PRIO)
        __builtin_amdgcn_s_setprio(0);
    for (int k0 = 0; k0 < ksteps; k0 += DEPTH) {
#pragma unroll
        for (int s = 0; s < DEPTH; ++s) {
            const int ks = k0 + s;
            if (ks < ksteps) {
                if (ks + 1 < ksteps) {
#pragma unroll
                    for (int r = 0; r < RT; ++r)
                        b[(ks + 1) & 1][r] = *reinterpret_cast<const uint4*>(bp[r] + (ks + 1) * 16);
                }
#pragma unroll
                for (int n = 0; n < NT; ++n)
#pragma unroll
                    for (int r = 0; r < RT; ++r)
                        acc[n][r] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                            __builtin_bit_cast(bf16x8, ring.a[s][n]),
                            __builtin_bit_cast(bf16x8, b[ks & 1][r]), acc[n][r], 0, 0, 0);
                if (ks + DEPTH < ksteps) {
#pragma unroll
                    for (int n = 0; n < NT; ++n)
                        ring.a[s][n] = load_frag(frag, (nt0 + n) * ksteps + ks + DEPTH, lane * 16u);
                }
                // keep each refill in its own k-step: left alone, the scheduler
                // may sink the loads next to their use and serialize the ring
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    }
    if constexpr (PRIO)
        __builtin_amdgcn_s_setprio(2);
}

// The same layer with one B buffer: row tile r of the next k-step is read
// from LDS as soon as this k-step's MFMAs on it are issued (row-tile-outer
// order), which saves RT x 4 VGPRs for the wider wave tiles.
template <int NT, int RT, int DEPTH, int LDW = kLdw>
__device__ __forceinline__ void mfma_layer_1b(WRing<NT, DEPTH>& ring, Frags frag, int ksteps,
                                              int nt0, int rt0, const uint16_t* buf, int lane,
                                              const float* __restrict__ bias,
                                              f32x16 (&acc)[NT][RT])
{
#pragma unroll
    for (int n = 0; n < NT; ++n) {
        f32x16 b0;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const float4 bb = *reinterpret_cast<const float4*>(
                bias + (nt0 + n) * 32 + g * 8 + (lane >> 5) * 4);
            b0[g * 4 + 0] = bb.x;
            b0[g * 4 + 1] = bb.y;
            b0[g * 4 + 2] = bb.z;
            b0[g * 4 + 3] = bb.w;
        }
#pragma unroll
        for (int r = 0; r < RT; ++r)
            acc[n][r] = b0;
    }
    const uint16_t* bp = buf + (rt0 * 32 + (lane & 31)) * LDW + (lane >> 5) * 8;
    uint4 b[RT];
#pragma unroll
    for (int r = 0; r < RT; ++r)
        b[r] = *reinterpret_cast<const uint4*>(bp + r * 32 * LDW);
    for (int k0 = 0; k0 < ksteps; k0 += DEPTH) {
#pragma unroll
        for (int s = 0; s < DEPTH; ++s) {
            const int ks = k0 + s;
            if (ks < ksteps) {
#pragma unroll
                for (int r = 0; r < RT; ++r) {
#pragma unroll
                    for (int n = 0; n < NT; ++n)
                        acc[n][r] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                            __builtin_bit_cast(bf16x8, ring.a[s][n]),
                            __builtin_bit_cast(bf16x8, b[r]), acc[n][r], 0, 0, 0);
                    if (ks + 1 < ksteps)
                        b[r] = *reinterpret_cast<const uint4*>(bp + r * 32 * LDW + (ks + 1) * 16);
                }
                if (ks + DEPTH < ksteps) {
#pragma unroll
                    for (int n = 0; n < NT; ++n)
                        ring.a[s][n] = load_frag(frag, (nt0 + n) * ksteps + ks + DEPTH, lane * 16u);
                }
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    }
}

// Hidden-unit ReLU on two accumulators: the IEEE 754-2019 maximum with +0
// (v_maximum3_f32: a NaN of either sign stays NaN, -0 becomes +0), then both
// rounded to bf16 with one v_cvt_pk_bf16_f32.  For non-NaN inputs this is
// bf16(max(x, 0)) = max(bf16(x), 0); a NaN reaches the next layer, so every
// logit of the row is NaN and the sampler raises the NaN flag.
__device__ __forceinline__ uint32_t relu_pack(float lo, float hi)
{
    return pack_bf16x2(relu_f32(lo), relu_f32(hi));
}

// ReLU + bf16, written back as the next layer's input rows.
template <int NT, int RT, int LDW = kLdw>
__device__ __forceinline__ void hidden_epilogue(const f32x16 (&acc)[NT][RT], int nt0, int rt0,
                                                uint16_t* buf, int lane)
{
#pragma unroll
    for (int n = 0; n < NT; ++n) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const int u0 = (nt0 + n) * 32 + g * 8 + (lane >> 5) * 4;
#pragma unroll
            for (int r = 0; r < RT; ++r) {
                const int row = (rt0 + r) * 32 + (lane & 31);
                uint2 pk = make_uint2(relu_pack(acc[n][r][g * 4 + 0], acc[n][r][g * 4 + 1]),
                                      relu_pack(acc[n][r][g * 4 + 2], acc[n][r][g * 4 + 3]));
                *reinterpret_cast<uint2*>(buf + row * LDW + u0) = pk;
            }
        }
    }
}

// ---- output layer fed from the layer-2 accumulators
//
// A wave holding layer-2 accumulators acc[n][r] (units (nt0+n)*32.., rows of
// row tile rt0+r) converts them with ReLU to bf16 B operands in place: k-step
// j of n-tile nt0+n takes registers 8j..8j+7 (see pack_bf16_kernel's kperm
// layout, in which the output weights are packed), so the output layer
// needs no trip of the second hidden layer through LDS.  Each wave produces
// partial logits over its own units; the partials of the NG waves sharing a
// row tile are summed in wave order by out_reduce.

template <int NT>
__device__ __forceinline__ void load_w3(uint4 (&w3)[NT][2], Frags W3, int nt0, int lane)
{
#pragma unroll
    for (int n = 0; n < NT; ++n)
#pragma unroll
        for (int j = 0; j < 2; ++j)
            w3[n][j] = load_frag(W3, (nt0 + n) * 2 + j, lane * 16u);
}

template <int NT, int RT>
__device__ __forceinline__ void out_from_acc(const f32x16 (&acc)[NT][RT],
                                             const uint4 (&w3)[NT][2], f32x16 (&o)[RT])
{
#pragma unroll
    for (int rr = 0; rr < RT; ++rr) {
        o[rr] = f32x16{};
#pragma unroll
        for (int n = 0; n < NT; ++n)
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const f32x16& c = acc[n][rr];
                const int g0 = 8 * j, g1 = 8 * j + 4;
                uint4 bq;
                bq.x = relu_pack(c[g0 + 0], c[g0 + 1]);
                bq.y = relu_pack(c[g0 + 2], c[g0 + 3]);
                bq.z = relu_pack(c[g1 + 0], c[g1 + 1]);
                bq.w = relu_pack(c[g1 + 2], c[g1 + 3]);
                o[rr] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    __builtin_bit_cast(bf16x8, w3[n][j]), __builtin_bit_cast(bf16x8, bq), o[rr],
                    0, 0, 0);
            }
    }
}

// Partials of wave group ng for row tiles rt0.. into red[NG][RTILES][G4][64]
// (registers of output groups g < G3 only: the real actions; G4 >= 4 G3 is
// 16 in general and 4 where at most 8 actions are known to be possible).
template <int RT, int RTILES, int G4 = 16, int RS = 64>
__device__ __forceinline__ void out_partials(float* red, const f32x16 (&o)[RT], int ng, int rt0,
                                             int G3, int lane)
{
#pragma unroll
    for (int rr = 0; rr < RT; ++rr)
#pragma unroll
        for (int g = 0; g < G4 / 4; ++g)
            if (g < G3)
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    red[((ng * RTILES + rt0 + rr) * G4 + g * 4 + q) * RS + lane] = o[rr][g * 4 + q];
}

// Logit (row, u) = sum over wave groups (in order) + bias; thread (row, u0)
// writes u0, u0+4, ... of its row.
template <int NG, int RTILES, int G4 = 16, int RS = 64>
__device__ __forceinline__ void out_reduce(const float* red, int row, int slot, int u0, int A,
                                           const float* b3, float* __restrict__ logits)
{
    if (slot < 0)
        return;
    float* out = logits + (int64_t)slot * A;
    for (int u = u0; u < A; u += 4) {
        const int lr = (row & 31) + 32 * ((u >> 2) & 1);
        const int reg = (u >> 3) * 4 + (u & 3);
        float v = 0.0f;
#pragma unroll
        for (int gq = 0; gq < NG; ++gq)
            v += red[((gq * RTILES + (row >> 5)) * G4 + reg) * RS + lr];
        out[u] = v + b3[u];
    }
}

// Row stride of the tile's Gumbel noise in LDS (gz): one float more than the
// largest action count, so that the rows start on different banks (with a
// stride of 32 floats every row's noise sat in the same banks).
constexpr int kGzStride = kMaxActions + 1;

// out_reduce that also samples the row's action (the four threads of a row,
// lanes 4r..4r+3, share it): z_u = logit_u + g_u with the Gumbel noise g of
// the row's slot staged in LDS (gz[row][u]), the first index of the largest z
// wins (each thread scans its own u in order, then the four bests are combined
// by two shuffles preferring the larger z, on equal z the lower index), as in
// gumbel_action.  A NaN logit raises kErrNaN and gives action 0.  Every lane
// takes part in the shuffles; padding rows (slot < 0) write nothing.  Logits
// are written when `logits` is not null.
template <int NG, int RTILES, int G4 = 16, int RS = 64>
__device__ __forceinline__ void out_reduce_sample(const float* red, const float* gz, int row,
                                                  int slot, int u0, int A, const float* b3,
                                                  float* __restrict__ logits,
                                                  uint8_t* __restrict__ actions, int* flags)
{
    float zbest = -__builtin_inff();
    int best = -1;
    bool bad = false;
    const bool live = slot >= 0;
    for (int u = u0; u < A; u += 4) {
        const int lr = (row & 31) + 32 * ((u >> 2) & 1);
        const int reg = (u >> 3) * 4 + (u & 3);
        float v = 0.0f;
#pragma unroll
        for (int gq = 0; gq < NG; ++gq)
            v += red[((gq * RTILES + (row >> 5)) * G4 + reg) * RS + lr];
        const float l = v + b3[u];
        if (live && logits)
            logits[(int64_t)slot * A + u] = l;
        bad |= __builtin_isnan(l);
        const float z = l + gz[row * kGzStride + u];
        if (best < 0 || z > zbest) {
            zbest = z;
            best = u;
        }
    }
#pragma unroll
    for (int m = 1; m <= 2; m <<= 1) {
        const float zo = __shfl_xor(zbest, m, 64);
        const int bo = __shfl_xor(best, m, 64);
        if (bo >= 0 && (best < 0 || zo > zbest || (zo == zbest && bo < best))) {
            zbest = zo;
            best = bo;
        }
        bad |= __shfl_xor((int)bad, m, 64) != 0;
    }
    if (live && u0 == 0) {
        actions[slot] = (uint8_t)(bad ? 0 : best);
        if (bad)
            atomicOr(flags, kErrNaN);
    }
}

// Wavefront grid of a HID-wide layer: WAVES wavefronts over (HID/32 n-tiles) x
// (RTILES row-tiles of 32); each wave owns NT n-tiles x RT row-tiles.
template <int HID, int WAVES, int RTILES>
struct HidSplit {
    static constexpr int NTT = HID / 32;
    static constexpr int NGROUPS = NTT >= WAVES ? WAVES : NTT;
    static constexpr int RGROUPS = WAVES / NGROUPS;
    static constexpr int NT = NTT / NGROUPS;
    static constexpr int RT = RTILES / RGROUPS;
    static constexpr int DEPTH = NT >= 4 ? 3 : 4;
    static_assert(NGROUPS * RGROUPS == WAVES && NT * NGROUPS == NTT && RT * RGROUPS == RTILES,
                  "wave split");
};

// Observation rows of the tile -> LDS (bf16).  KIN is the padded input width.
template <int OBS, int KIN, int MR, int THREADS, int LDW = kLdw>
__device__ __forceinline__ void build_obs(const MlpBf16Args& a, const int* row_slot,
                                          const int* row_env, uint16_t* buf, int tid)
{
    if constexpr (OBS == kObsFeature) {
        // KIN == d: bf16 rows of d, copied 8 columns (16 bytes) at a time;
        // thread t keeps columns 8 (t % (KIN/8)) ..
        constexpr int Q8 = KIN / 8;
        constexpr int ROWS_PER_PASS = THREADS / Q8;
        constexpr int PASSES = MR / ROWS_PER_PASS;
        static_assert(KIN % 8 == 0 && THREADS % Q8 == 0 && PASSES * ROWS_PER_PASS == MR,
                      "whole rows per pass");
        const int c = (tid % Q8) * 8, r0 = tid / Q8;
        constexpr int BATCH = PASSES < 16 ? PASSES : 16;
        const uint16_t* S = (const uint16_t*)a.state + c;
#pragma unroll
        for (int u0 = 0; u0 < PASSES; u0 += BATCH) {
            uint4 v[BATCH];
#pragma unroll
            for (int u = 0; u < BATCH; ++u) {
                // padding rows (env < 0) read env 0's row and drop it: a
                // conditional load here made the compiler spill
                const int env = row_env[r0 + (u0 + u) * ROWS_PER_PASS];
                const uint4 t =
                    *reinterpret_cast<const uint4*>(S + (uint32_t)max(env, 0) * (uint32_t)KIN);
                v[u] = env >= 0 ? t : make_uint4(0, 0, 0, 0);
            }
#pragma unroll
            for (int u = 0; u < BATCH; ++u)
                *reinterpret_cast<uint4*>(buf + (r0 + (u0 + u) * ROWS_PER_PASS) * LDW + c) = v[u];
        }
    } else if constexpr (OBS == kObsPursuit) {
        // each row's cells are fetched once (one thread per row), packed as
        // self x << 24 | self y << 16 | pursuer << 8 | evader (-1: padding
        // row); then one item per (row, window cell) writes its 3 channels
        __shared__ int cells[MR];
        static_assert(THREADS >= MR && KIN >= 75, "one thread per row, 75 inputs");
        const int G = a.grid;
        if (tid < MR) {
            const int env = row_env[tid];
            int cv = -1;
            if (env >= 0) {
                const uint8_t* pos = (const uint8_t*)a.state;
                const int seat = row_slot[tid] - env * a.n_agents;
                const int pc = pos[env], ec = pos[a.n_envs + env];
                const int self = seat == 0 ? pc : ec;
                cv = ((self % G) << 24) | ((self / G) << 16) | (pc << 8) | ec;
            }
            cells[tid] = cv;
        }
        __syncthreads();
        for (int it = tid; it < MR * 25; it += THREADS) {
            const int r = it / 25, o = it - r * 25;
            const int cv = cells[r];
            uint16_t* dst = buf + r * LDW + o * 3;
            if (cv < 0) {
                dst[0] = dst[1] = dst[2] = 0;
                continue;
            }
            const int dy = o / 5 - 2, dx = o - (o / 5) * 5 - 2;
            int x = (cv >> 24) + dx, y = ((cv >> 16) & 0xFF) + dy;   // |dx|, |dy| <= 2 < G
            x += x < 0 ? G : 0;
            x -= x >= G ? G : 0;
            y += y < 0 ? G : 0;
            y -= y >= G ? G : 0;
            const int cell = y * G + x;
            const uint16_t one = 0x3F80;   // bf16 1.0
            dst[0] = cell == ((cv >> 8) & 0xFF) ? one : 0;
            dst[1] = cell == (cv & 0xFF) ? one : 0;
            dst[2] = o == 12 ? one : 0;    // the centre cell: the agent itself
        }
        for (int it = tid; it < MR * (KIN - 75); it += THREADS) {
            const int r = it / (KIN - 75);
            buf[r * LDW + 75 + (it - r * (KIN - 75))] = 0;
        }
    } else {
        // each row's history is fetched once (one thread per row), packed as
        // seat << 16 | history (-1: padding row)
        __shared__ int hs[MR];
        static_assert(THREADS >= MR, "one thread per row");
        if (tid < MR) {
            const int env = row_env[tid];
            int hv = -1;
            if (env >= 0) {
                const uint16_t* hist = (const uint16_t*)a.state;
                hv = ((row_slot[tid] - env * a.n_agents) << 16) | hist[env];
            }
            hs[tid] = hv;
        }
        __syncthreads();
        for (int i = tid; i < MR * KIN; i += THREADS) {
            const int r = i / KIN, c = i - r * KIN;
            const int hv = hs[r];
            float v = 0.0f;
            if (hv >= 0 && c < a.in_dim)
                v = iter_obs((uint16_t)(hv & 0xFFFF), hv >> 16, a.A, c);
            buf[r * LDW + c] = bf16_bits(v);
        }
    }
}

// MR rows per tile (the library uses 64), two workgroups per CU; eight
// wavefronts per workgroup for hidden widths 128 and 256 (four per SIMD in
// all), four otherwise (bf16_tile_threads).
// Layers 1 and 2 run from LDS rows; the output layer is fed from the layer-2
// accumulators (out_from_acc), its partials summed through the row buffer.
template <int HID, int OBS, int KIN, int MR>
__global__ __launch_bounds__(bf16_tile_threads(HID), bf16_tile_waves_per_simd(HID)) void mlp_bf16_kernel(
    MlpBf16Args a)
{
    constexpr int THREADS = bf16_tile_threads(HID), WAVES = THREADS / 64, RTILES = MR / 32;
    // row stride: the wider of the input and hidden rows, + 8 to spread banks
    constexpr int LDW = (KIN > HID ? KIN : HID) + 8;
    // partial-logit registers kept per (wave group, row tile): pursuit (5
    // actions) and the iterated game (<= 3) need one accumulator group
    constexpr int G4 = OBS == kObsFeature ? 16 : 4;
    // partial logits at a row stride of 65 floats: the four threads of a row
    // then read different banks in out_reduce (at 64 they shared one)
    constexpr int RS = 65;
    constexpr int PART = HidSplit<HID, WAVES, RTILES>::NGROUPS * RTILES * G4 * RS * 2;   // in bf16
    constexpr int BUF = MR * LDW > PART ? MR * LDW : PART;
    __shared__ __attribute__((aligned(16))) uint16_t buf[BUF];
    __shared__ int row_slot[MR];
    __shared__ int row_env[MR];
    // the tile's hidden-layer biases, staged with the rows: the layers start
    // their accumulators from LDS instead of waiting on fresh global loads
    __shared__ __attribute__((aligned(16))) float bias[2][HID];
    // Gumbel noise of the rows' slots when the kernel samples the actions
    // (feature observations), [MR][kGzStride]
    constexpr int GZ = OBS == kObsFeature ? MR * kGzStride : 1;
    __shared__ float gz[GZ];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    // At hidden width 512 the waves run their latency-bound phases (row
    // indices, noise, gather, epilogue, output and sampling) at a raised issue
    // priority and their k-loops at the normal one, so that the CU's other
    // workgroup's k-loops yield issue slots to them (4v4 forward 104.8 ->
    // 103.8 us over six alternating runs; narrower widths measured slower).
    constexpr bool kPrio = HID >= 512;
    if constexpr (kPrio)
        __builtin_amdgcn_s_setprio(2);

    // workgroups are dispatched round-robin over the 8 XCDs: each XCD reads one
    // segment of the striped tile table, an equal share of the tiles in order,
    // so that a policy's tiles share one L2 and the XCDs get equal work
    const int per = a.n_blocks / 8;
    const int t = (blockIdx.x & 7) * per + (blockIdx.x >> 3);
    if (t >= a.max_tiles)
        return;
    const int4 ti = a.tile_info[t];
    const int p = __builtin_amdgcn_readfirstlane(ti.x);
    if (p < 0)
        return;
    const int r0 = ti.y;
    const int nrows = ti.z;

    using S = HidSplit<HID, WAVES, RTILES>;
    const int nt0 = (wave % S::NGROUPS) * S::NT;
    const int rt0 = (wave / S::NGROUPS) * S::RT;
    const Frags W1 = frag_src(a.w1 + (int64_t)p * (HID / 32) * (KIN / 16) * 64,
                              (HID / 32) * (KIN / 16));
    const Frags W2 = frag_src(a.w2 + (int64_t)p * (HID / 32) * (HID / 16) * 64,
                              (HID / 32) * (HID / 16));
    WRing<S::NT, S::DEPTH> ring;

    if (tid < MR) {
        row_slot[tid] = tid < nrows ? a.perm[r0 + tid] : -1;
        row_env[tid] = tid < nrows ? a.perm_env[r0 + tid] : -1;
    }
    for (int i = tid; i < HID; i += THREADS) {
        bias[0][i] = a.b1[p * HID + i];
        bias[1][i] = a.b2[p * HID + i];
    }
    __syncthreads();
    // the first weight fragments after the row indices (loads complete in
    // order, so issued earlier they would delay the indices' LDS stores);
    // they arrive during the noise and the observation gather
    ring_fill(ring, W1, KIN / 16, nt0, lane);
    if constexpr (OBS == kObsFeature) {
        // the rows' Gumbel noise while the observation rows are fetched: one
        // thread per (row, Philox block of 8 actions), the same stream and
        // transform as gumbel_action
        if (a.actions) {
            const int nb = (a.A + 7) >> 3;
            for (int i = tid; i < MR * nb; i += THREADS) {
                const int row = i / nb, blk = i - row * nb;
                const int slot = row_slot[row];
                if (slot >= 0) {
                    const int env = slot / a.n_agents, seat = slot - env * a.n_agents;
                    const u64x4 pb = stream_block(a.seed, (uint64_t)(a.env_offset + env),
                                                  (uint64_t)a.t, kPurposeAction,
                                                  (uint32_t)seat, (uint64_t)blk);
#pragma unroll
                    for (int j = 0; j < 8; ++j)
                        if (blk * 8 + j < a.A)
                            gz[row * kGzStride + blk * 8 + j] =
                                gumbel01(uniform01(block_lane(pb, j)));
                }
            }
        }
    }
    build_obs<OBS, KIN, MR, THREADS, LDW>(a, row_slot, row_env, buf, tid);
    __syncthreads();

    f32x16 acc[S::NT][S::RT];
    // ---- layer 1: KIN -> HID
    mfma_layer<S::NT, S::RT, S::DEPTH, LDW, kPrio>(ring, W1, KIN / 16, nt0, rt0, buf, lane,
                                                   bias[0], acc);
    ring_fill(ring, W2, HID / 16, nt0, lane);      // overlaps the epilogue
    // the output layer's weight fragments: in flight during layer 2 below
    // hidden width 512; at 512 their 32 registers live across layer 2 cost
    // more than the load's latency after it
    constexpr bool kW3Early = HID < 512;
    uint4 w3[S::NT][2];
    const Frags W3 = frag_src(a.w3 + (int64_t)p * (HID / 16) * 64, HID / 16);
    if constexpr (kW3Early)
        load_w3<S::NT>(w3, W3, nt0, lane);
    __syncthreads();
    hidden_epilogue<S::NT, S::RT, LDW>(acc, nt0, rt0, buf, lane);
    __syncthreads();
    // ---- layer 2: HID -> HID
    mfma_layer<S::NT, S::RT, S::DEPTH, LDW, kPrio>(ring, W2, HID / 16, nt0, rt0, buf, lane,
                                                   bias[1], acc);
    // ---- layer 3 from the accumulators, partial logits summed through LDS
    if constexpr (!kW3Early)
        load_w3<S::NT>(w3, W3, nt0, lane);
    f32x16 o[S::RT];
    out_from_acc<S::NT, S::RT>(acc, w3, o);
    __syncthreads();   // every wave is done reading the hidden rows: buf takes the partials
    float* red = reinterpret_cast<float*>(buf);
    out_partials<S::RT, RTILES, G4, RS>(red, o, wave % S::NGROUPS, rt0, (a.A + 7) >> 3, lane);
    __syncthreads();
    {
        const int row = tid >> 2;
        const int slot = row < nrows && row < MR ? row_slot[row] : -1;
        if constexpr (OBS == kObsFeature) {
            if (a.actions) {
                if (row < MR)
                    out_reduce_sample<S::NGROUPS, RTILES, G4, RS>(red, gz, row, slot, tid & 3, a.A,
                                                              a.b3 + p * a.A, a.logits,
                                                              a.actions, a.flags);
                return;
            }
        }
        out_reduce<S::NGROUPS, RTILES, G4, RS>(red, row, slot, tid & 3, a.A, a.b3 + p * a.A,
                                           a.logits);
    }
}

// ------------------------------------------------------------ generic MLP

// Any MLP the specialized kernels do not cover (input and hidden widths up to
// 1024 each, the two hidden widths free, fp32 policies on every environment):
// one workgroup per tile of kGenericTileRows rows of one policy; the rows'
// activations in LDS (fp32 values; bf16-rounded for bf16 policies), each
// thread forms output units tid, tid + 256, ... for every row with an fp32
// fused multiply-add chain over the inputs, then adds the bias, applies the
// hidden ReLU (IEEE maximum with +0: a NaN stays NaN) and, for bf16
// policies, rounds to bf16 (products of bf16 values are exact in fp32).
// Weights are kept as given, [P][out][in] (fp32, or bf16 bits rounded to
// nearest even at creation).  The logits go to the env step, which samples.

constexpr int kGenericThreads = 256;

struct MlpGenericArgs {
    const void* w[3];
    const float* b[3];
    int dims[4];
    int bf16;
    const int32_t* perm;
    const int32_t* perm_env;
    const int4* tile_info;
    int max_tiles;
    int env_kind;
    const void* state;      // iterated game: uint16 history; pursuit: uint8 [2][n]; feature: fp32 [n][d]
    int n_agents, grid, A;
    int64_t n_envs;
    float* logits;
};

// Observation element k of seat `seat` of env `env` (the encodings of the
// other policy kernels, element by element).
__device__ __forceinline__ float generic_obs(const MlpGenericArgs& a, int env, int seat, int k)
{
    if (a.env_kind == MALIB_ENV_FEATURE)
        return ((const float*)a.state)[(int64_t)env * a.dims[0] + k];
    if (a.env_kind == MALIB_ENV_PURSUIT) {
        const uint8_t* pos = (const uint8_t*)a.state;
        const int G = a.grid, pc = pos[env], ec = pos[a.n_envs + env];
        const int self = seat == 0 ? pc : ec;
        const int o = k / 3, c = k - 3 * o;
        const int dy = o / 5 - 2, dx = o - (o / 5) * 5 - 2;
        int x = self % G + dx, y = self / G + dy;     // |dx|, |dy| <= 2 < G
        x += x < 0 ? G : 0;
        x -= x >= G ? G : 0;
        y += y < 0 ? G : 0;
        y -= y >= G ? G : 0;
        const int cell = y * G + x;
        if (c == 0)
            return cell == pc ? 1.0f : 0.0f;
        if (c == 1)
            return cell == ec ? 1.0f : 0.0f;
        return o == 12 ? 1.0f : 0.0f;
    }
    const uint16_t* hist = (const uint16_t*)a.state;
    return iter_obs(hist[env], seat, a.A, k);
}

__device__ __forceinline__ float bf16_value(float x)
{
    return __uint_as_float((uint32_t)bf16_bits(x) << 16);
}

__device__ __forceinline__ float generic_weight(const MlpGenericArgs& a, int l, int64_t i)
{
    if (a.bf16)
        return __uint_as_float((uint32_t)((const uint16_t*)a.w[l])[i] << 16);
    return ((const float*)a.w[l])[i];
}

__global__ __launch_bounds__(kGenericThreads) void mlp_generic_kernel(MlpGenericArgs a)
{
    constexpr int R = kGenericTileRows, W = kGenericMaxWidth;
    __shared__ float xa[R * W];
    __shared__ float xb[R * W];
    __shared__ int row_slot[R], row_env[R];
    const int t = blockIdx.x, tid = threadIdx.x;
    if (t >= a.max_tiles)
        return;
    const int4 ti = a.tile_info[t];
    const int p = ti.x;
    if (p < 0)
        return;
    if (tid < R) {
        row_slot[tid] = tid < ti.z ? a.perm[ti.y + tid] : -1;
        row_env[tid] = tid < ti.z ? a.perm_env[ti.y + tid] : -1;
    }
    __syncthreads();
    const int in0 = a.dims[0];
    for (int i = tid; i < R * in0; i += kGenericThreads) {
        const int r = i / in0, k = i - r * in0;
        const int env = row_env[r];
        float v = 0.0f;
        if (env >= 0)
            v = generic_obs(a, env, row_slot[r] - env * a.n_agents, k);
        xa[r * W + k] = a.bf16 ? bf16_value(v) : v;
    }
    __syncthreads();
    float* x = xa;
    float* y = xb;
    for (int l = 0; l < 3; ++l) {
        const int in = a.dims[l], out = a.dims[l + 1];
        const int64_t wbase = (int64_t)p * out * in;
        for (int o = tid; o < out; o += kGenericThreads) {
            float acc[R];
#pragma unroll
            for (int r = 0; r < R; ++r)
                acc[r] = 0.0f;
            const int64_t wrow = wbase + (int64_t)o * in;
            for (int k = 0; k < in; ++k) {
                const float w = generic_weight(a, l, wrow + k);
#pragma unroll
                for (int r = 0; r < R; ++r)
                    acc[r] = __builtin_fmaf(w, x[r * W + k], acc[r]);
            }
            const float b = a.b[l][(int64_t)p * out + o];
#pragma unroll
            for (int r = 0; r < R; ++r) {
                float v = acc[r] + b;
                if (l < 2) {
                    v = relu_f32(v);
                    y[r * W + o] = a.bf16 ? bf16_value(v) : v;
                } else if (r < ti.z) {
                    a.logits[(int64_t)row_slot[r] * a.A + o] = v;
                }
            }
        }
        __syncthreads();
        float* tmp = x;
        x = y;
        y = tmp;
    }
}

hipError_t launch_mlp_generic(const Pop& pop, int env_kind, int n_agents, int grid,
                              const int32_t* perm, const int32_t* perm_env,
                              const int4* tile_info, int max_tiles, int64_t n_slots,
                              const void* state, float* logits, hipStream_t s)
{
    MlpGenericArgs a = {};
    for (int l = 0; l < 3; ++l) {
        a.w[l] = pop.w[l];
        a.b[l] = pop.b[l];
    }
    for (int l = 0; l < 4; ++l) {
        a.dims[l] = pop.dims[l];
        if (pop.dims[l] < 1 || pop.dims[l] > kGenericMaxWidth)
            return hipErrorInvalidValue;
    }
    a.bf16 = pop.kind == MALIB_POLICY_MLP_BF16;
    a.perm = perm;
    a.perm_env = perm_env;
    a.tile_info = tile_info;
    a.max_tiles = max_tiles;
    a.env_kind = env_kind;
    a.state = state;
    a.n_agents = n_agents;
    a.grid = grid;
    a.A = pop.A;
    a.n_envs = n_slots / n_agents;
    a.logits = logits;
    mlp_generic_kernel<<<max_tiles, kGenericThreads, 0, s>>>(a);
    return hipGetLastError();
}

// fp32 weights -> bf16 bits (round to nearest even), [n] elements.
__global__ void round_bf16_kernel(const float* __restrict__ w, int64_t n,
                                  uint16_t* __restrict__ out)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n)
        out[i] = bf16_bits(w[i]);
}

hipError_t launch_round_bf16(const float* w, int64_t n, uint16_t* out, hipStream_t s)
{
    if (n <= 0)
        return hipSuccess;
    round_bf16_kernel<<<(int)((n + 255) / 256), 256, 0, s>>>(w, n, out);
    return hipGetLastError();
}

// ------------------------------------------------------------ persistent bf16 MLP

// Feature observations, large batches: one persistent workgroup of eight
// wavefronts per CU walks a contiguous run of tiles of up to 128 rows (the
// tile table is built with 128-row tiles), so every weight fragment it streams
// serves 128 rows.  Runs are equal in tiles; run i of G goes to XCD i / (G/8)
// so that neighbouring runs (the same policies) share an L2.
//
// Per tile: observations (bf16, LDS) -> layer 1 -> ReLU/bf16 into LDS ->
// layer 2 -> output layer straight from the layer-2 accumulators (the output
// weights are packed in that k order, see pack_bf16_kernel) -> per-wave
// partial logits summed through LDS in wave order.  The next tile's table
// entry, row indices and output bias are fetched before layer 2, its first
// weight fragments and observation rows while the partial logits are summed.
template <int HID, int KIN>
__global__ __launch_bounds__(512, 1) void mlp_bf16_persist_kernel(MlpBf16Args a)
{
    constexpr int MR = kPersistRows, THREADS = 512, WAVES = 8, RTILES = 4;
    using S = HidSplit<HID, WAVES, RTILES>;
    constexpr int NT = S::NT, RT = S::RT, NG = S::NGROUPS;
    static_assert(NG * RTILES * 16 * 64 * 4 <= MR * kLdw * 2, "partials fit in the row buffer");
    __shared__ __attribute__((aligned(16))) uint16_t buf[MR * kLdw];
    __shared__ int row_slot[2][MR];
    __shared__ int row_env[2][MR];
    __shared__ float b3s[2][kMaxActions];
    float* red = reinterpret_cast<float*>(buf);   // [NG][RTILES][16][64] partial logits

    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int nt0 = (wave % NG) * NT, rt0 = (wave / NG) * RT, ng = wave % NG;

    const int T = a.tile_off[a.P];
    const int G = gridDim.x, ri = (blockIdx.x & 7) * (G >> 3) + (blockIdx.x >> 3);
    const int t0 = (int)((int64_t)ri * T / G), t1 = (int)((int64_t)(ri + 1) * T / G);
    if (t0 >= t1)
        return;

    constexpr int F1 = (HID / 32) * (KIN / 16), F2 = (HID / 32) * (HID / 16), F3 = HID / 16;
    constexpr int Q4 = KIN / 4, RPP = THREADS / Q4, PASSES = MR / RPP;
    // observation float4s per thread fetched ahead (more would spill)
    constexpr int PRE = PASSES < 8 ? PASSES : 8;
    typedef float v4f __attribute__((ext_vector_type(4)));
    const int G3 = (a.A + 7) >> 3;   // accumulator groups holding real actions

    int t = t0, cur = 0;
    int4 ti = a.tile_info[t];
    int p = __builtin_amdgcn_readfirstlane(ti.x), nrows = __builtin_amdgcn_readfirstlane(ti.z);
    {
        const int r0 = __builtin_amdgcn_readfirstlane(ti.y);
        if (tid < MR) {
            row_slot[0][tid] = tid < nrows ? a.perm[r0 + tid] : -1;
            row_env[0][tid] = tid < nrows ? a.perm_env[r0 + tid] : -1;
        }
        if (tid < a.A)
            b3s[0][tid] = a.b3[p * a.A + tid];
        __syncthreads();
        const int oc = (tid % Q4) * 4, orow = tid / Q4;
        const float* S0 = (const float*)a.state + oc;
        v4f ob[PASSES];
#pragma unroll
        for (int u = 0; u < PASSES; ++u) {
            const int env = row_env[0][orow + u * RPP];
            ob[u] = v4f{0.f, 0.f, 0.f, 0.f};
            if (env >= 0)
                ob[u] = *reinterpret_cast<const v4f*>(S0 + (uint32_t)env * (uint32_t)KIN);
        }
#pragma unroll
        for (int u = 0; u < PASSES; ++u)
            *reinterpret_cast<uint2*>(buf + (orow + u * RPP) * kLdw + oc) =
                make_uint2(pack_bf16x2(ob[u].x, ob[u].y), pack_bf16x2(ob[u].z, ob[u].w));
    }
    WRing<NT, S::DEPTH> ring;
    ring_fill(ring, frag_src(a.w1 + (int64_t)p * F1 * 64, F1), KIN / 16, nt0, tid & 63);
    __syncthreads();

    for (;;) {
        // per-lane values are recomputed every tile from an opaque copy of
        // the thread index: hoisted out of the loop they would stay live
        // across the MFMA layers and push the allocator into spills
        int tq = tid;
        asm volatile("" : "+v"(tq));
        const int ln = tq & 63;
        f32x16 acc[NT][RT];
        // ---- layer 1 (first fragments already in the ring)
        mfma_layer_1b<NT, RT, S::DEPTH>(ring, frag_src(a.w1 + (int64_t)p * F1 * 64, F1),
                                        KIN / 16, nt0, rt0, buf, ln, a.b1 + p * HID, acc);
        const Frags W2 = frag_src(a.w2 + (int64_t)p * F2 * 64, F2);
        ring_fill(ring, W2, HID / 16, nt0, ln);
        __syncthreads();
        hidden_epilogue<NT, RT>(acc, nt0, rt0, buf, ln);
        // next tile: table entry, row indices and output bias (into registers)
        const bool has_next = t + 1 < t1;
        int4 tin = make_int4(0, 0, 0, 0);
        if (has_next)
            tin = a.tile_info[t + 1];
        const int pn = __builtin_amdgcn_readfirstlane(tin.x);
        const int nn = __builtin_amdgcn_readfirstlane(tin.z);
        const int rn = __builtin_amdgcn_readfirstlane(tin.y);
        int slot_n = -1, env_n = -1;
        float b3_n = 0.0f;
        if (has_next) {
            if (tq < nn) {
                slot_n = a.perm[rn + tq];
                env_n = a.perm_env[rn + tq];
            }
            if (tq < a.A)
                b3_n = a.b3[pn * a.A + tq];
        }
        __syncthreads();
        // ---- layer 2
        mfma_layer_1b<NT, RT, S::DEPTH>(ring, W2, HID / 16, nt0, rt0, buf, ln, a.b2 + p * HID,
                                        acc);
        uint4 w3[NT][2];
        load_w3<NT>(w3, frag_src(a.w3 + (int64_t)p * F3 * 64, F3), nt0, ln);
        if (tq < MR) {
            row_slot[cur ^ 1][tq] = slot_n;
            row_env[cur ^ 1][tq] = env_n;
        }
        if (tq < kMaxActions)
            b3s[cur ^ 1][tq] = b3_n;

        // ---- layer 3 from the accumulators: partial logits over this wave's units
        f32x16 o[RT];
        out_from_acc<NT, RT>(acc, w3, o);
        __syncthreads();   // every wave is done reading the hidden rows
        out_partials<RT, RTILES>(red, o, ng, rt0, G3, ln);
        __builtin_amdgcn_sched_barrier(0);
        // next tile: first layer-1 fragments, observation rows -> registers
        // (issued now, consumed after the partial sums: nothing in between
        // waits on the vector memory counter)
        const int oc = (tq % Q4) * 4, orow = tq / Q4;
        v4f ob[PRE];
        const float* S0 = (const float*)a.state + oc;
        if (has_next) {
            ring_fill(ring, frag_src(a.w1 + (int64_t)pn * F1 * 64, F1), KIN / 16, nt0, ln);
#pragma unroll
            for (int u = 0; u < PRE; ++u) {
                const int env = row_env[cur ^ 1][orow + u * RPP];
                ob[u] = v4f{0.f, 0.f, 0.f, 0.f};
                if (env >= 0)
                    ob[u] = *reinterpret_cast<const v4f*>(S0 + (uint32_t)env * (uint32_t)KIN);
            }
        }
        __syncthreads();
        // logits: partials summed in wave order, then the bias
        out_reduce<NG, RTILES>(red, tq >> 2, row_slot[cur][tq >> 2], tq & 3, a.A, b3s[cur],
                               a.logits);
        if (!has_next)
            break;
        __syncthreads();   // partials consumed: the row buffer takes the next observations
#pragma unroll
        for (int u = 0; u < PRE; ++u)
            *reinterpret_cast<uint2*>(buf + (orow + u * RPP) * kLdw + oc) =
                make_uint2(pack_bf16x2(ob[u].x, ob[u].y), pack_bf16x2(ob[u].z, ob[u].w));
        // the remaining rows
#pragma unroll
        for (int u0 = PRE; u0 < PASSES; u0 += PRE) {
            v4f o2[PRE];
#pragma unroll
            for (int u = 0; u < PRE; ++u) {
                const int env = row_env[cur ^ 1][orow + (u0 + u) * RPP];
                o2[u] = v4f{0.f, 0.f, 0.f, 0.f};
                if (env >= 0)
                    o2[u] = *reinterpret_cast<const v4f*>(S0 + (uint32_t)env * (uint32_t)KIN);
            }
#pragma unroll
            for (int u = 0; u < PRE; ++u)
                *reinterpret_cast<uint2*>(buf + (orow + (u0 + u) * RPP) * kLdw + oc) =
                    make_uint2(pack_bf16x2(o2[u].x, o2[u].y), pack_bf16x2(o2[u].z, o2[u].w));
        }
        ++t;
        p = pn;
        nrows = nn;
        cur ^= 1;
        __syncthreads();
    }
}

template <int HID>
static hipError_t launch_persist_hid(const MlpBf16Args& a, int kin, int blocks, hipStream_t s)
{
    if (kin != 512)
        return hipErrorInvalidValue;
    mlp_bf16_persist_kernel<HID, 512><<<blocks, 512, 0, s>>>(a);
    return hipGetLastError();
}

hipError_t launch_mlp_bf16_persist(const Pop& pop, const int32_t* perm, const int32_t* perm_env,
                                   const int4* tile_info, const int32_t* tile_off,
                                   int64_t n_slots, int n_agents, const void* state,
                                   float* logits, hipStream_t s)
{
    if (pop.A > kMaxActions)
        return hipErrorInvalidValue;
    MlpBf16Args a = {};
    a.w1 = (const uint4*)pop.w[0];
    a.w2 = (const uint4*)pop.w[1];
    a.w3 = (const uint4*)pop.w[2];
    a.b1 = pop.b[0];
    a.b2 = pop.b[1];
    a.b3 = pop.b[2];
    a.perm = perm;
    a.perm_env = perm_env;
    a.tile_info = tile_info;
    a.tile_off = tile_off;
    a.state = state;
    a.logits = logits;
    a.P = pop.P;
    a.A = pop.A;
    a.in_dim = pop.in_dim;
    a.n_agents = n_agents;
    // one workgroup per CU (fewer for small batches: tiles are spread evenly
    // over the workgroups, a multiple of the 8 XCDs)
    const int64_t tiles = (n_slots + kPersistRows - 1) / kPersistRows + pop.P;
    int blocks = (int)std::min<int64_t>(tiles, pop.n_cus);
    blocks = std::max(8, (blocks + 7) / 8 * 8);
    switch (pop.hid) {
    case 64: return launch_persist_hid<64>(a, pop.in_pad, blocks, s);
    case 128: return launch_persist_hid<128>(a, pop.in_pad, blocks, s);
    case 256: return launch_persist_hid<256>(a, pop.in_pad, blocks, s);
    case 512: return launch_persist_hid<512>(a, pop.in_pad, blocks, s);
    default: return hipErrorInvalidValue;
    }
}

template <int HID, int OBS, int KIN>
static void launch_one(const MlpBf16Args& a, int rows, int blocks, hipStream_t s)
{
    (void)rows;   // kBf16TileRows
    mlp_bf16_kernel<HID, OBS, KIN, kBf16TileRows><<<blocks, bf16_tile_threads(HID), 0, s>>>(a);
}

template <int HID>
static hipError_t launch_hid(const MlpBf16Args& a, int obs, int in_pad, int rows, int blocks,
                             hipStream_t s)
{
    if (obs == kObsPursuit && in_pad == 80)
        launch_one<HID, kObsPursuit, 80>(a, rows, blocks, s);
    else if (obs == kObsIter && in_pad == 32)
        launch_one<HID, kObsIter, 32>(a, rows, blocks, s);
    else if (obs == kObsFeature && in_pad == 64)
        launch_one<HID, kObsFeature, 64>(a, rows, blocks, s);
    else if (obs == kObsFeature && in_pad == 128)
        launch_one<HID, kObsFeature, 128>(a, rows, blocks, s);
    else if (obs == kObsFeature && in_pad == 256)
        launch_one<HID, kObsFeature, 256>(a, rows, blocks, s);
    else if (obs == kObsFeature && in_pad == 512)
        launch_one<HID, kObsFeature, 512>(a, rows, blocks, s);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

hipError_t launch_mlp_bf16(const Pop& pop, int env_kind, int n_agents, int grid, int d,
                           int tile_rows, const int32_t* perm, const int32_t* perm_env,
                           const int4* tile_info, int64_t n_slots, const void* state,
                           float* logits, const KernelSample* ks, hipStream_t s)
{
    MlpBf16Args a = {};
    if (ks) {
        if (env_kind != MALIB_ENV_FEATURE)
            return hipErrorInvalidValue;
        a.actions = ks->actions;
        a.flags = ks->flags;
        a.seed = ks->seed;
        a.env_offset = ks->env_offset;
        a.t = ks->t;
    }
    a.w1 = (const uint4*)pop.w[0];
    a.w2 = (const uint4*)pop.w[1];
    a.w3 = (const uint4*)pop.w[2];
    a.b1 = pop.b[0];
    a.b2 = pop.b[1];
    a.b3 = pop.b[2];
    a.perm = perm;
    a.perm_env = perm_env;
    a.tile_info = tile_info;
    a.state = state;
    a.logits = logits;
    a.P = pop.P;
    a.A = pop.A;
    a.in_dim = pop.in_dim;
    a.n_agents = n_agents;
    a.grid = grid;
    a.d = d;
    a.n_envs = n_slots / n_agents;
    if (tile_rows != kBf16TileRows)
        return hipErrorInvalidValue;
    // one workgroup per entry of the striped tile table (a multiple of 8)
    const int blocks = striped_entries(n_slots, pop.P, tile_rows);
    a.n_blocks = blocks;
    a.max_tiles = blocks;
    int obs = env_kind == MALIB_ENV_FEATURE ? kObsFeature
              : env_kind == MALIB_ENV_PURSUIT ? kObsPursuit : kObsIter;
    if (pop.A > (obs == kObsFeature ? kMaxActions : 8))
        return hipErrorInvalidValue;   // the partial-logit layout holds one group of 8
    switch (pop.hid) {
    case 64: return launch_hid<64>(a, obs, pop.in_pad, tile_rows, blocks, s);
    case 128: return launch_hid<128>(a, obs, pop.in_pad, tile_rows, blocks, s);
    case 256: return launch_hid<256>(a, obs, pop.in_pad, tile_rows, blocks, s);
    case 512: return launch_hid<512>(a, obs, pop.in_pad, tile_rows, blocks, s);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace malib
