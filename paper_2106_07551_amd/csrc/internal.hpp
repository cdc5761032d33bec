// Internal interfaces of libmalib: the population handle and the kernel
// launchers (one translation unit per kernel family).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <string>
#include <vector>

#include "malib.h"

namespace malib {

constexpr int kMaxP = 256;
constexpr int kMaxActions = 32;
constexpr int kMaxAgents = 8;
constexpr int kF32TileRows = 32;   // rows per fp32 policy tile (one wavefront)
constexpr int kBucketChunk = 2048; // slots per bucketing workgroup

// Growable device buffer owned by a handle.
struct DevBuf {
    void* ptr = nullptr;
    size_t bytes = 0;
};

struct EventPair {
    hipEvent_t start, stop;
};

struct Profile {
    int mask = 0;                 // bit k: time kernel class k
    int every = 1;                // time one launch in `every` per class
    int64_t seen[MALIB_K_COUNT] = {0, 0, 0, 0, 0};
    std::vector<EventPair> pool;
    size_t used = 0;
    std::vector<int> kind;        // kernel class of each used pair
};

struct Pop {
    int kind = 0;
    int P = 0;
    int A = 0;
    int in_dim = 0, hid = 0;
    int in_pad = 0;               // bf16: input padded to a multiple of 16
    // generic MLP (shapes the specialized kernels do not take): weights kept
    // as [P][out][in] (fp32, or bf16 bits), dims = {in, h1, h2, A}
    bool generic = false;
    int dims[4] = {0, 0, 0, 0};
    int device = 0;
    int n_cus = 0;                // compute units of the device
    // packed weights
    // bf16: fragment layout (the output layer's k order follows the layer-2
    // accumulators, see pack_bf16_kernel); fp32: [P][out][in]
    void* w[3] = {nullptr, nullptr, nullptr};
    float* b[3] = {nullptr, nullptr, nullptr};  // fp32 [P][out] (zero-filled when absent)
    float* tab = nullptr;                       // fp32 [P][A]
    std::vector<int64_t> ids;                   // caller's policy id of each index
    // payoff accumulators, one allocation acc[3 P*P + 2] so that the table
    // comes back in one copy: sum, sumsq, cnt ([P*P] each), the live-frame
    // counter and the device error flags (the low half of the last word)
    unsigned long long* acc = nullptr;
    unsigned long long* sum = nullptr;   // int64 fixed point 2^-32 (two's complement)
    unsigned long long* sumsq = nullptr; // int64 fixed point 2^-20
    unsigned long long* cnt = nullptr;
    unsigned long long* dev_frames = nullptr;
    int* dev_flags = nullptr;
    unsigned long long* host_acc = nullptr;   // pinned copy of acc
    int64_t host_frames = 0;   // frames of env families with no early termination
    int64_t envs = 0;
    // scratch, grown on demand
    DevBuf perm, perm_env, tile_info, hist, base, offsets, tile_off, logits, ret, state0,
        state1, obs, wt, done, thresholds, actions;
    // device address of the library's static no-allocation scratch on this
    // handle's device (resolved at creation; null if that failed)
    void* scratch = nullptr;
    Profile prof;
    // graph mode: malib_rollout_batch records each batch's launch sequence
    // into a HIP graph and replays it through one executable graph, updated
    // in place for the next batch of the same shape
    int graph_mode = 0;
    hipGraphExec_t graph_exec = nullptr;
    hipEvent_t graph_done = nullptr;     // recorded after each replay
    hipStream_t graph_rec = nullptr;     // the (default-priority) stream recorded on
};

// Bucketing of slots by policy id (stable counting sort) + tile table:
// perm[r] = slot of sorted row r, perm_env[r] = its env, offsets[P+1] bucket
// bounds, tile_off[P+1] first tile of each policy, tile_info[n_entries]: the
// tiles (policy, first row, rows) and padding entries (-1, 0, 0).  Plain
// layout: entry t is tile t (padding from tile_off[P] on); striped layout
// (n_entries a multiple of 8): 8 equal segments, each holding an equal share
// of the tiles in order, then padding (see tile_table_kernel).
hipError_t launch_bucket(const int32_t* pids, int64_t n_slots, int n_agents, int P,
                         int tile_rows, int n_entries, bool striped, int32_t* hist,
                         int32_t* base, int32_t* perm, int32_t* perm_env, int32_t* offsets,
                         int32_t* tile_off, int4* tile_info, int* flags, hipStream_t s);
inline int max_tiles_for(int64_t n_slots, int P, int tile_rows)
{
    return (int)((n_slots + tile_rows - 1) / tile_rows + P);
}
// Entries of the striped table of the 64-row bf16 kernel: max_tiles_for
// rounded up to the 8 XCD segments (one workgroup per entry).
inline int striped_entries(int64_t n_slots, int P, int tile_rows)
{
    return (max_tiles_for(n_slots, P, tile_rows) + 7) / 8 * 8;
}

// Meta-solver: the table as a game, fictitious play, thresholds from device
// weights (k_solve.hip).
hipError_t launch_payoff_matrix(const unsigned long long* sum, const unsigned long long* cnt,
                                int P, double* M, hipStream_t s);
// LP solver (primal simplex, one workgroup); P > 96 needs a [P+1][2P+1] fp64
// workspace.
bool lp_needs_work(int P);
hipError_t launch_lp(const double* M, int P, int max_pivots, double* work, double* value,
                     double* x, double* y, float* sigma, int* pivots, hipStream_t s);
// alpha-rank: one workgroup; P > 128 needs a [P][P] fp64 workspace.
bool alpharank_needs_work(int P);
hipError_t launch_alpharank(const double* M, int P, double alpha, int m, double* work,
                            double* pi, float* sigma, hipStream_t s);
hipError_t launch_solve_fp(const double* M, int P, int T, float* sigma, double* gap,
                           hipStream_t s);
hipError_t launch_thresholds(const float* sigma, int n_sigma, int P, unsigned long long* thr,
                             hipStream_t s);
hipError_t launch_aggregate(const double* M, int P, const float* sigma, int br_row, int br_col,
                            double* out, hipStream_t s);

// Incremental table expansion (k_expand.hip): the P0 x P0 accumulators copied
// into a P x P table (new cells zero), and the policy ids of the batch that
// simulates every cell with row or column >= first (row-major over the grid,
// per_pair envs per cell; team_row: bit k set = seat k takes the row policy).
hipError_t launch_remap_table(const unsigned long long* src, int P0, unsigned long long* dst,
                              int P, hipStream_t s);
hipError_t launch_expansion_pairs(int P, int first, int per_pair, int n_agents, uint32_t team_row,
                                  int64_t n_envs, int32_t* out, hipStream_t s);

// Meta-strategy sampling from precomputed thresholds [n_sigma][P].
// seat_map: 4 bits per seat, the threshold row that seat draws from
hipError_t launch_meta_sample(const unsigned long long* thr, uint32_t seat_map, int P,
                              int64_t n_envs, int n_agents, uint64_t seed, int64_t env_offset,
                              int32_t* out, hipStream_t s);

// Gumbel-max action sampling, done by the env-step kernels for the slots of
// their envs (gumbel_action): the step's logits, the Philox key and counter
// parts, the optional action log [n_slots] (255 for finished envs) and the
// device error flags (kErrNaN).
struct SampleArgs {
    const float* logits;   // [n_slots][A]
    uint64_t seed;
    int64_t env_offset;
    int t;
    uint8_t* log;
    int* flags;
    // FEATURE: the actions the policy kernel already sampled [n_slots] (it
    // also raised the NaN flag), or null to sample here from the logits
    const uint8_t* actions = nullptr;
};

// Trajectory records written by the env-step kernels (all null: none).
// Record of step t of local env e: (base + t * n_envs + e) mod cap.
struct TrajArgs {
    uint8_t* act = nullptr;    // [cap][n_agents], 255 = no action (finished env)
    float* rew = nullptr;      // [cap] the row side's reward of the step
    uint8_t* flags = nullptr;  // [cap] bit 0 terminal, bit 1 last step, bit 2 finished before
    void* obs = nullptr;       // [cap][...] the state before the step, compact (or null)
    int64_t base = 0;
    int64_t cap = 1;
    int horizon = 0;
};

// Environment kernels.
struct EnvArgs {
    int kind, n_agents, A, grid, d, init_mode;
    uint32_t team_row;   // bit k set: seat k is on the row side (team +1)
    uint32_t team_col;   // bit k set: seat k is on the column side (team -1)
    const float* Amat;
    const float* W;
    const float* WT;     // transposed W (scratch)
    const float* emb;
    const float* u;
    // FEATURE with bf16 policies: the observation bf16_rne(s) of every env,
    // [n_envs][d], written by reset and by each step next to the fp32 state
    // (the policy forward gathers these rows: half the bytes, no conversion)
    uint16_t* obs;
    TrajArgs tr;
    int n_cus = 0;       // compute units of the device (workgroup sizing)
};
hipError_t launch_zero_f32(float* x, int64_t n, hipStream_t s);
hipError_t launch_reset(const EnvArgs& e, int64_t n_envs, uint64_t seed, int64_t env_offset,
                        void* state, uint8_t* done, hipStream_t s);
hipError_t launch_transpose(const float* W, float* WT, int d, hipStream_t s);
hipError_t launch_env_step(const EnvArgs& e, const SampleArgs& sa, int64_t n_envs,
                           const void* state_in, void* state_out, uint8_t* done, float* ret,
                           unsigned long long* frames, hipStream_t s);
hipError_t launch_snapshot_pursuit(const void* state, const uint8_t* done, int64_t n_envs,
                                   uint8_t* out, hipStream_t s);

// Payoff reduction (once per batch): for P*P <= kPayoffStreamMaxCells a
// private LDS copy of the whole table per workgroup over env ranges;
// otherwise from the policy bucketing (LDS rows, one set of global atomics per
// touched cell), or per env (global atomics, wave-combined where a wavefront
// shares a cell) when there is no bucketing (tabular policies).
constexpr int kPayoffStreamMaxCells = 4096;     // P <= 64: 80 KB of LDS
bool payoff_stream_fits(int P);
hipError_t launch_payoff_stream(const float* ret, const int32_t* pids, int64_t n_envs,
                                int n_agents, uint32_t team_row, uint32_t team_col, int P,
                                int n_cus, unsigned long long* sum, unsigned long long* sumsq,
                                unsigned long long* cnt, hipStream_t s);
hipError_t launch_payoff(const float* ret, const int32_t* pids, int64_t n_envs, int n_agents,
                         const int8_t* team, int P, unsigned long long* sum,
                         unsigned long long* sumsq, unsigned long long* cnt, hipStream_t s);
hipError_t launch_payoff_bucketed(const float* ret, const int32_t* pids, const int32_t* perm,
                                  const int32_t* offsets, int64_t n_envs, int n_agents,
                                  uint32_t team_row, uint32_t team_col, int P, int n_cus,
                                  unsigned long long* sum, unsigned long long* sumsq,
                                  unsigned long long* cnt, hipStream_t s);

// Policy forwards.
hipError_t launch_pack_bf16(const float* w, int P, int out, int in, int out_pad, int in_pad,
                            int kperm, void* dst, hipStream_t s);
hipError_t launch_pack_f32(const float* w, int P, int layer, int hid, int A, float* dst,
                           hipStream_t s);
hipError_t launch_tabular(const float* tab, const int32_t* pids, int64_t n_slots, int A, int P,
                          int* flags, float* logits, hipStream_t s);
hipError_t launch_mlp_f32(const Pop& pop, const int32_t* perm, const int4* tile_info,
                          int64_t n_slots, int n_agents, const void* state, float* logits,
                          hipStream_t s);
// bf16 policy tiles have 64 rows: two four-wave workgroups share a CU, so one
// workgroup's gather and epilogues overlap the other's MFMA loop.  (128-row
// tiles halve the weight traffic per row but leave one workgroup per CU; on
// the 4v4 and d=512 workloads they measured 12% and 3% slower.)
constexpr int kBf16TileRows = 64;
// Threads of a 64-row tile's workgroup: eight wavefronts for hidden widths 128
// and 256 (two workgroups per CU give four per SIMD to hide the
// weight-fragment latency; pursuit's forward measured 29.5 -> 23.7 us against
// four); four below, where eight would leave a wavefront no whole tile, and
// four at 512, where each wavefront then covers 128 output units (four
// fragment tiles for the same two row tiles: a quarter fewer operand bytes
// per MFMA, at two wavefronts per SIMD and ~200 registers; 4v4 forward 106.5
// -> 104.4 us).
constexpr int bf16_tile_threads(int hid) { return hid >= 128 && hid < 512 ? 512 : 256; }
// Wavefronts per SIMD the 64-row kernel is compiled for (two workgroups per CU)
constexpr int bf16_tile_waves_per_simd(int hid) { return hid >= 128 && hid < 512 ? 4 : 2; }
// Gumbel-max sampling done by the 64-row policy kernel itself (feature
// observations: no env finishes early): the sampled actions [n_slots], the
// error flags, the Philox key and the counter parts of the step.
struct KernelSample {
    uint8_t* actions;
    int* flags;
    uint64_t seed;
    int64_t env_offset;
    int t;
};
// ks: null = only the logits (the env step samples); logits may be null when
// ks is given and no one reads them.
hipError_t launch_mlp_bf16(const Pop& pop, int env_kind, int n_agents, int grid, int d,
                           int tile_rows, const int32_t* perm, const int32_t* perm_env,
                           const int4* tile_info, int64_t n_slots, const void* state,
                           float* logits, const KernelSample* ks, hipStream_t s);
// Generic MLP forward (k_policy.hip): tiles of kGenericTileRows rows, widths
// up to kGenericMaxWidth; logits for the env step to sample.
constexpr int kGenericTileRows = 8;
constexpr int kGenericMaxWidth = 1024;
hipError_t launch_mlp_generic(const Pop& pop, int env_kind, int n_agents, int grid,
                              const int32_t* perm, const int32_t* perm_env,
                              const int4* tile_info, int max_tiles, int64_t n_slots,
                              const void* state, float* logits, hipStream_t s);
hipError_t launch_round_bf16(const float* w, int64_t n, uint16_t* out, hipStream_t s);
// Feature observations of d = 512 with >= 256 slots per policy on average:
// persistent kernel over 128-row tiles (one eight-wave workgroup per CU, output
// layer fed from the layer-2 accumulators).  For narrower observations the
// 64-row kernel (two workgroups per CU, whose phases overlap) measured faster.
constexpr int kPersistRows = 128;
inline bool use_persist_kernel(int env_kind, int in_pad, int64_t n_slots, int P)
{
    return env_kind == MALIB_ENV_FEATURE && in_pad == 512 && n_slots >= 256 * (int64_t)P;
}
hipError_t launch_mlp_bf16_persist(const Pop& pop, const int32_t* perm, const int32_t* perm_env,
                                   const int4* tile_info, const int32_t* tile_off,
                                   int64_t n_slots, int n_agents, const void* state,
                                   float* logits, hipStream_t s);

// Diagnostics.
hipError_t launch_debug_bf16(const float* x, uint16_t* y, int64_t n, hipStream_t s);
hipError_t launch_debug_tanh(const float* x, float* y, int64_t n, hipStream_t s);
hipError_t launch_debug_philox(const uint64_t* ctr, uint64_t k0, uint64_t k1, uint64_t* out,
                               int64_t n, hipStream_t s);

}  // namespace malib
