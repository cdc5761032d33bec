// C ABI of libmalib: argument validation, device buffers, the rollout step
// loop and the payoff table.  Everything after validation is enqueued on the
// caller's stream.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <string>
#include <vector>

#include "device.hpp"
#include "internal.hpp"

#include <cmath>

using namespace malib;

struct malib_pop : public Pop {};

// Scratch of malib_rollout_batch_noalloc: one static device array per GPU the
// library runs on (held until the process ends).  Host code never passes the
// array's name to a kernel (on the host it is only a stand-in for the symbol):
// its device address is looked up once per device with hipGetSymbolAddress
// and kept in g_scratch_addr.
constexpr size_t kNoAllocScratchBytes = (size_t)64 << 20;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_addr[kMaxDevices];
hipError_t g_scratch_err[kMaxDevices];
}  // namespace

// The current device's address of `scratch` (looked up on the first call for
// that device, with the device current).  Null on failure (*err says why).
static void* scratch_address(int device, hipError_t* err)
{
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (device < 0 || device >= kMaxDevices) {
        *err = hipErrorInvalidDevice;
        return nullptr;
    }
    if (!g_scratch_addr[device] && g_scratch_err[device] == hipSuccess) {
        void* ptr = nullptr;
        const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e == hipSuccess && ptr)
            g_scratch_addr[device] = ptr;
        else
            g_scratch_err[device] = e == hipSuccess ? hipErrorInvalidSymbol : e;
    }
    *err = g_scratch_err[device];
    return g_scratch_addr[device];
}

namespace {

// fixed-size, so that reporting an error allocates nothing
thread_local char g_last_error[512];

malib_status fail(malib_status code, const char* fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
    va_end(ap);
    return code;
}

#define HIP_TRY(expr)                                                                     \
    do {                                                                                  \
        hipError_t e_ = (expr);                                                           \
        if (e_ != hipSuccess)                                                             \
            return fail(e_ == hipErrorOutOfMemory ? MALIB_E_NOMEM : MALIB_E_HIP,          \
                        "%s failed: %s", #expr, hipGetErrorString(e_));                   \
    } while (0)

// Allocation-failure hook for tests of the error paths: while the environment
// variable MALIB_FAULT_ALLOC is set to anything but "" or "0", every device
// or pinned host allocation of the library fails as out of memory without
// allocating.  Read at each allocation, so a test can turn it on and off.
bool fault_alloc()
{
    const char* v = getenv("MALIB_FAULT_ALLOC");
    return v && *v && strcmp(v, "0") != 0;
}

hipError_t dev_malloc(void** p, size_t bytes)
{
    return fault_alloc() ? hipErrorOutOfMemory : hipMalloc(p, bytes);
}

hipError_t host_malloc(void** p, size_t bytes)
{
    return fault_alloc() ? hipErrorOutOfMemory : hipHostMalloc(p, bytes, hipHostMallocDefault);
}

hipError_t dev_malloc_async(void** p, size_t bytes, hipStream_t s)
{
    return fault_alloc() ? hipErrorOutOfMemory : hipMallocAsync(p, bytes, s);
}

hipError_t ensure(DevBuf& b, size_t bytes)
{
    if (bytes <= b.bytes)
        return hipSuccess;
    if (b.ptr) {
        hipError_t e = hipDeviceSynchronize();
        if (e != hipSuccess)
            return e;
        e = hipFree(b.ptr);
        if (e != hipSuccess)
            return e;
        b.ptr = nullptr;
        b.bytes = 0;
    }
    size_t want = std::max(bytes, (size_t)256);
    hipError_t e = dev_malloc(&b.ptr, want);
    if (e == hipSuccess)
        b.bytes = want;
    return e;
}

void release(DevBuf& b)
{
    if (b.ptr)
        (void)hipFree(b.ptr);
    b.ptr = nullptr;
    b.bytes = 0;
}

int round_up(int x, int m) { return (x + m - 1) / m * m; }

// ---- profiling: one event pair per launch of a kernel class
int prof_begin(Pop& p, int kind, hipStream_t s)
{
    if (!((p.prof.mask >> kind) & 1))
        return -1;
    if (p.prof.seen[kind]++ % p.prof.every != 0)
        return -1;
    if (p.prof.used == p.prof.pool.size()) {
        EventPair ev;
        if (hipEventCreate(&ev.start) != hipSuccess || hipEventCreate(&ev.stop) != hipSuccess)
            return -1;
        p.prof.pool.push_back(ev);
    }
    int i = (int)p.prof.used++;
    p.prof.kind.push_back(kind);
    (void)hipEventRecord(p.prof.pool[i].start, s);
    return i;
}

void prof_end(Pop& p, int i, hipStream_t s)
{
    if (i >= 0)
        (void)hipEventRecord(p.prof.pool[i].stop, s);
}

int64_t state_bytes_per_env(int kind, int d)
{
    switch (kind) {
    case MALIB_ENV_ITER_MATRIX: return 2;
    case MALIB_ENV_PURSUIT: return 2;
    case MALIB_ENV_FEATURE: return 4 * (int64_t)d;
    default: return 0;
    }
}

int64_t snap_bytes_per_env(int kind, int d)
{
    switch (kind) {
    case MALIB_ENV_ITER_MATRIX: return 2;
    case MALIB_ENV_PURSUIT: return 3;
    case MALIB_ENV_FEATURE: return 4 * (int64_t)d;
    default: return 0;
    }
}

}  // namespace

extern "C" {

const char* malib_last_error(void) { return g_last_error; }

// ------------------------------------------------------------------- create

// Validates a population description; on success dims = {in, h1, h2, A}
// (zeros for tabular populations) and *generic tells whether the MLP needs
// the generic kernel (a shape the specialized kernels do not take).
static malib_status check_desc(const malib_pop_desc* desc, int (&dims)[4], bool* generic)
{
    const int P = desc->n_policies, A = desc->n_actions;
    if (P < 1 || P > kMaxP)
        return fail(MALIB_E_INVAL, "n_policies must be in [1, %d], got %d", kMaxP, P);
    if (A < 1 || A > kMaxActions)
        return fail(MALIB_E_INVAL, "n_actions must be in [1, %d], got %d", kMaxActions, A);
    for (int l = 0; l < 4; ++l)
        dims[l] = 0;
    *generic = false;
    if (desc->kind == MALIB_POLICY_TABULAR) {
        if (!desc->tab_logits)
            return fail(MALIB_E_INVAL, "tabular population needs tab_logits");
    } else if (desc->kind == MALIB_POLICY_MLP_F32 || desc->kind == MALIB_POLICY_MLP_BF16) {
        if (desc->n_layers != 3)
            return fail(MALIB_E_UNSUPPORTED, "MLP populations have 3 layers, got %d",
                        desc->n_layers);
        if (!desc->dims || !desc->weights)
            return fail(MALIB_E_INVAL, "MLP population needs dims and weights");
        for (int l = 0; l < 3; ++l)
            if (!desc->weights[l])
                return fail(MALIB_E_INVAL, "weights[%d] is NULL", l);
        for (int l = 0; l < 4; ++l)
            dims[l] = desc->dims[l];
        if (dims[3] != A)
            return fail(MALIB_E_INVAL, "dims[3] (%d) must equal n_actions (%d)", dims[3], A);
        for (int l = 0; l < 3; ++l)
            if (dims[l] < 1 || dims[l] > kGenericMaxWidth)
                return fail(MALIB_E_UNSUPPORTED, "MLP widths must be in [1, %d], got dims[%d] = %d",
                            kGenericMaxWidth, l, dims[l]);
        const int in = dims[0], h1 = dims[1], h2 = dims[2];
        bool special;
        if (desc->kind == MALIB_POLICY_MLP_F32)
            special = in == 24 && A == 3 && h1 == h2 && (h1 == 32 || h1 == 64);
        else
            special = h1 == h2 && (h1 == 64 || h1 == 128 || h1 == 256 || h1 == 512) && in <= 512;
        *generic = !special;
    } else {
        return fail(MALIB_E_INVAL, "unknown policy kind %d", desc->kind);
    }
    return MALIB_OK;
}

// Bytes of one policy's layer-l weights in the handle's layout.
static size_t weight_bytes(const Pop& p, int l)
{
    const int fi = p.dims[l], fo = p.dims[l + 1];
    if (p.generic)
        return (p.kind == MALIB_POLICY_MLP_F32 ? 4 : 2) * (size_t)fo * fi;
    if (p.kind == MALIB_POLICY_MLP_F32)
        return sizeof(float) * (size_t)fo * fi;
    const int ip = l == 0 ? p.in_pad : round_up(fi, 16);
    const int op = round_up(fo, 32);
    return (size_t)(op / 32) * (ip / 16) * 64 * 16;
}

// k policies' fp32 weights of layer l ([k][out][in], device) into the
// handle's layout at dst: the generic kernel's [k][out][in] (fp32, or bf16
// bits), or the specialized kernels' packed MFMA operand layouts.
static hipError_t store_weights(const Pop& p, int l, const float* src, int k, void* dst,
                                hipStream_t s)
{
    const int fi = p.dims[l], fo = p.dims[l + 1];
    if (p.generic) {
        const int64_t n = (int64_t)k * fo * fi;
        if (p.kind == MALIB_POLICY_MLP_F32)
            return hipMemcpyAsync(dst, src, sizeof(float) * n, hipMemcpyDeviceToDevice, s);
        return launch_round_bf16(src, n, (uint16_t*)dst, s);
    }
    if (p.kind == MALIB_POLICY_MLP_F32)
        return launch_pack_f32(src, k, l, p.hid, p.A, (float*)dst, s);
    const int ip = l == 0 ? p.in_pad : round_up(fi, 16);
    const int op = round_up(fo, 32);
    // the output layer in the k order of the layer-2 accumulators
    return launch_pack_bf16(src, k, fo, fi, op, ip, l == 2, dst, s);
}

// The caller ids of the policies a description adds at indices first ..
// first + P - 1 (desc->policy_ids, else the indices themselves), checked to be
// distinct from each other and from `existing`.
static malib_status read_ids(const malib_pop_desc* desc, int first,
                             const std::vector<int64_t>& existing, std::vector<int64_t>& out)
{
    const int P = desc->n_policies;
    out.clear();
    for (int i = 0; i < P; ++i)
        out.push_back(desc->policy_ids ? desc->policy_ids[i] : (int64_t)(first + i));
    std::vector<int64_t> all(existing);
    all.insert(all.end(), out.begin(), out.end());
    std::sort(all.begin(), all.end());
    for (size_t i = 1; i < all.size(); ++i)
        if (all[i] == all[i - 1])
            return fail(MALIB_E_INVAL, "policy id %lld appears twice", (long long)all[i]);
    return MALIB_OK;
}

malib_status malib_pop_create(const malib_pop_desc* desc, void* stream, malib_pop_t* out)
{
    if (!out)
        return fail(MALIB_E_INVAL, "out is NULL");
    *out = nullptr;
    if (!desc)
        return fail(MALIB_E_INVAL, "desc is NULL");
    hipStream_t s = (hipStream_t)stream;
    const int P = desc->n_policies, A = desc->n_actions;
    int dims[4];
    bool generic = false;
    {
        const malib_status st = check_desc(desc, dims, &generic);
        if (st != MALIB_OK)
            return st;
    }
    const int in = dims[0], hid = dims[1];
    std::vector<int64_t> ids;
    {
        const malib_status st = read_ids(desc, 0, {}, ids);
        if (st != MALIB_OK)
            return st;
    }

    malib_pop* p = new (std::nothrow) malib_pop();
    if (!p)
        return fail(MALIB_E_NOMEM, "host allocation failed");
    p->ids = std::move(ids);
    auto cleanup = [&](malib_status st) {
        malib_pop_destroy(p);
        return st;
    };
#define TRY(expr)                                                                         \
    do {                                                                                  \
        hipError_t e_ = (expr);                                                           \
        if (e_ != hipSuccess)                                                             \
            return cleanup(fail(e_ == hipErrorOutOfMemory ? MALIB_E_NOMEM : MALIB_E_HIP,  \
                                "%s failed: %s", #expr, hipGetErrorString(e_)));          \
    } while (0)
    TRY(hipGetDevice(&p->device));
    TRY(hipDeviceGetAttribute(&p->n_cus, hipDeviceAttributeMultiprocessorCount, p->device));
    {
        // set-up of the no-allocation entry point on this device
        hipError_t e = hipSuccess;
        p->scratch = scratch_address(p->device, &e);
    }
    p->kind = desc->kind;
    p->P = P;
    p->A = A;
    p->in_dim = in;
    p->hid = hid;
    p->generic = generic;
    for (int l = 0; l < 4; ++l)
        p->dims[l] = dims[l];
    if (desc->kind == MALIB_POLICY_TABULAR) {
        TRY(dev_malloc((void**)&p->tab, sizeof(float) * P * A));
        TRY(hipMemcpyAsync(p->tab, desc->tab_logits, sizeof(float) * P * A,
                           hipMemcpyDeviceToDevice, s));
    } else {
        p->in_pad = round_up(in, 16);
        for (int l = 0; l < 3; ++l) {
            const int fo = dims[l + 1];
            size_t nb = sizeof(float) * (size_t)P * fo;
            TRY(dev_malloc((void**)&p->b[l], nb));
            if (desc->biases && desc->biases[l])
                TRY(hipMemcpyAsync(p->b[l], desc->biases[l], nb, hipMemcpyDeviceToDevice, s));
            else
                TRY(hipMemsetAsync(p->b[l], 0, nb, s));
            TRY(dev_malloc(&p->w[l], weight_bytes(*p, l) * P));
            TRY(store_weights(*p, l, desc->weights[l], P, p->w[l], s));
        }
    }
    const size_t PP = (size_t)P * P, acc_bytes = sizeof(unsigned long long) * (3 * PP + 2);
    TRY(dev_malloc((void**)&p->acc, acc_bytes));
    TRY(host_malloc((void**)&p->host_acc, acc_bytes));
    p->sum = p->acc;
    p->sumsq = p->acc + PP;
    p->cnt = p->acc + 2 * PP;
    p->dev_frames = p->acc + 3 * PP;
    p->dev_flags = reinterpret_cast<int*>(p->acc + 3 * PP + 1);
    TRY(hipMemsetAsync(p->acc, 0, acc_bytes, s));
    TRY(hipStreamSynchronize(s));
#undef TRY
    *out = p;
    return MALIB_OK;
}

void malib_pop_destroy(malib_pop_t p)
{
    if (!p)
        return;
    (void)hipDeviceSynchronize();
    for (int l = 0; l < 3; ++l) {
        if (p->w[l])
            (void)hipFree(p->w[l]);
        if (p->b[l])
            (void)hipFree(p->b[l]);
    }
    if (p->tab)
        (void)hipFree(p->tab);
    if (p->acc)
        (void)hipFree(p->acc);
    if (p->host_acc)
        (void)hipHostFree(p->host_acc);
    for (DevBuf* b : {&p->perm, &p->perm_env, &p->tile_info, &p->hist, &p->base, &p->offsets, &p->tile_off, &p->logits,
                      &p->ret, &p->state0, &p->state1, &p->obs, &p->wt, &p->done,
                      &p->thresholds, &p->actions})
        release(*b);
    if (p->graph_exec)
        (void)hipGraphExecDestroy(p->graph_exec);
    if (p->graph_done)
        (void)hipEventDestroy(p->graph_done);
    if (p->graph_rec)
        (void)hipStreamDestroy(p->graph_rec);
    for (auto& ev : p->prof.pool) {
        (void)hipEventDestroy(ev.start);
        (void)hipEventDestroy(ev.stop);
    }
    delete p;
}

// ---------------------------------------------------------------- extend

malib_status malib_pop_extend(malib_pop_t pop, const malib_pop_desc* add, void* stream)
{
    if (!pop || !add)
        return fail(MALIB_E_INVAL, "pop and add must not be NULL");
    int dims[4];
    bool generic = false;
    {
        const malib_status st = check_desc(add, dims, &generic);
        if (st != MALIB_OK)
            return st;
    }
    if (add->kind != pop->kind)
        return fail(MALIB_E_INVAL, "policy kind %d differs from the population's (%d)",
                    add->kind, pop->kind);
    if (add->n_actions != pop->A)
        return fail(MALIB_E_INVAL, "n_actions %d differs from the population's (%d)",
                    add->n_actions, pop->A);
    for (int l = 0; l < 3; ++l)
        if (dims[l] != pop->dims[l])
            return fail(MALIB_E_INVAL, "dims {%d, %d, %d} differ from the population's "
                        "{%d, %d, %d}", dims[0], dims[1], dims[2], pop->dims[0],
                        pop->dims[1], pop->dims[2]);
    const int P0 = pop->P, k = add->n_policies, P = P0 + k, A = pop->A;
    if (P > kMaxP)
        return fail(MALIB_E_INVAL, "%d + %d policies exceed %d", P0, k, kMaxP);
    std::vector<int64_t> new_ids;
    {
        const malib_status st = read_ids(add, P0, pop->ids, new_ids);
        if (st != MALIB_OK)
            return st;
    }
    hipStream_t s = (hipStream_t)stream;
    // Everything new is built before the handle changes: on failure the
    // population is left as it was.
    void* w[3] = {nullptr, nullptr, nullptr};
    float* b[3] = {nullptr, nullptr, nullptr};
    float* tab = nullptr;
    unsigned long long* acc = nullptr;
    unsigned long long* host_acc = nullptr;
    auto drop = [&]() {
        (void)hipStreamSynchronize(s);
        for (int l = 0; l < 3; ++l) {
            if (w[l])
                (void)hipFree(w[l]);
            if (b[l])
                (void)hipFree(b[l]);
        }
        if (tab)
            (void)hipFree(tab);
        if (acc)
            (void)hipFree(acc);
        if (host_acc)
            (void)hipHostFree(host_acc);
    };
#define TRY(expr)                                                                         \
    do {                                                                                  \
        hipError_t e_ = (expr);                                                           \
        if (e_ != hipSuccess) {                                                           \
            drop();                                                                       \
            return fail(e_ == hipErrorOutOfMemory ? MALIB_E_NOMEM : MALIB_E_HIP,          \
                        "%s failed: %s", #expr, hipGetErrorString(e_));                   \
        }                                                                                 \
    } while (0)
    // work queued on any stream may still update the table (or read the
    // weights): let it finish before both are copied
    TRY(hipDeviceSynchronize());
    if (pop->kind == MALIB_POLICY_TABULAR) {
        const size_t per = sizeof(float) * A;
        TRY(dev_malloc((void**)&tab, per * P));
        TRY(hipMemcpyAsync(tab, pop->tab, per * P0, hipMemcpyDeviceToDevice, s));
        TRY(hipMemcpyAsync(tab + (size_t)P0 * A, add->tab_logits, per * k,
                           hipMemcpyDeviceToDevice, s));
    } else {
        for (int l = 0; l < 3; ++l) {
            const int fo = dims[l + 1];
            const size_t bper = sizeof(float) * fo;
            TRY(dev_malloc((void**)&b[l], bper * P));
            TRY(hipMemcpyAsync(b[l], pop->b[l], bper * P0, hipMemcpyDeviceToDevice, s));
            if (add->biases && add->biases[l])
                TRY(hipMemcpyAsync(b[l] + (size_t)P0 * fo, add->biases[l], bper * k,
                                   hipMemcpyDeviceToDevice, s));
            else
                TRY(hipMemsetAsync(b[l] + (size_t)P0 * fo, 0, bper * k, s));
            // every layout keeps each policy's weights contiguous, policy-major
            const size_t wper = weight_bytes(*pop, l);
            TRY(dev_malloc(&w[l], wper * P));
            TRY(hipMemcpyAsync(w[l], pop->w[l], wper * P0, hipMemcpyDeviceToDevice, s));
            TRY(store_weights(*pop, l, add->weights[l], k, (char*)w[l] + wper * P0, s));
        }
    }
    const size_t PP = (size_t)P * P, acc_bytes = sizeof(unsigned long long) * (3 * PP + 2);
    TRY(dev_malloc((void**)&acc, acc_bytes));
    TRY(host_malloc((void**)&host_acc, acc_bytes));
    TRY(launch_remap_table(pop->acc, P0, acc, P, s));
    // the copies and the remap read the old buffers
    TRY(hipDeviceSynchronize());
#undef TRY
    for (int l = 0; l < 3; ++l) {
        if (pop->w[l]) {
            (void)hipFree(pop->w[l]);
            pop->w[l] = w[l];
        }
        if (pop->b[l]) {
            (void)hipFree(pop->b[l]);
            pop->b[l] = b[l];
        }
    }
    if (pop->tab) {
        (void)hipFree(pop->tab);
        pop->tab = tab;
    }
    (void)hipFree(pop->acc);
    (void)hipHostFree(pop->host_acc);
    pop->acc = acc;
    pop->host_acc = host_acc;
    pop->sum = acc;
    pop->sumsq = acc + PP;
    pop->cnt = acc + 2 * PP;
    pop->dev_frames = acc + 3 * PP;
    pop->dev_flags = reinterpret_cast<int*>(acc + 3 * PP + 1);
    pop->P = P;
    pop->ids.insert(pop->ids.end(), new_ids.begin(), new_ids.end());
    return MALIB_OK;
}

malib_status malib_pop_policy_ids(malib_pop_t pop, int64_t* ids_out, int32_t capacity,
                                  int32_t* n_out)
{
    if (!pop)
        return fail(MALIB_E_INVAL, "pop is NULL");
    if (ids_out && capacity < pop->P)
        return fail(MALIB_E_INVAL, "capacity %d is below the population size %d", capacity,
                    pop->P);
    if (n_out)
        *n_out = pop->P;
    if (ids_out)
        std::copy(pop->ids.begin(), pop->ids.end(), ids_out);
    return MALIB_OK;
}

malib_status malib_expansion_pairs(int32_t n_policies, int32_t first_new, int32_t per_pair,
                                   int32_t n_agents, const int8_t* team, int32_t* out,
                                   void* stream)
{
    if (!out)
        return fail(MALIB_E_INVAL, "pair_assign_out is NULL");
    if (n_policies < 1 || n_policies > kMaxP)
        return fail(MALIB_E_INVAL, "n_policies must be in [1, %d]", kMaxP);
    if (first_new < 0 || first_new >= n_policies)
        return fail(MALIB_E_INVAL, "first_new must be in [0, n_policies)");
    if (per_pair < 1)
        return fail(MALIB_E_INVAL, "per_pair must be >= 1");
    if (n_agents < 2 || n_agents > kMaxAgents)
        return fail(MALIB_E_INVAL, "n_agents must be in [2, %d]", kMaxAgents);
    if (!team && n_agents != 2)
        return fail(MALIB_E_INVAL, "team may be NULL only for two seats");
    uint32_t row = 0, col = 0;
    for (int k = 0; k < n_agents; ++k) {
        const int t = team ? team[k] : (k == 0 ? 1 : -1);
        if (t != 1 && t != -1)
            return fail(MALIB_E_INVAL, "team entries must be +1 or -1");
        (t > 0 ? row : col) |= 1u << k;
    }
    if (row == 0 || col == 0)
        return fail(MALIB_E_INVAL, "both sides need at least one seat");
    const int64_t cells = (int64_t)n_policies * n_policies - (int64_t)first_new * first_new;
    const int64_t n_envs = cells * per_pair;
    if (n_envs * n_agents > ((int64_t)1 << 26))
        return fail(MALIB_E_INVAL, "the expansion batch exceeds 2^26 slots");
    HIP_TRY(launch_expansion_pairs(n_policies, first_new, per_pair, n_agents, row, n_envs, out,
                                   (hipStream_t)stream));
    return MALIB_OK;
}

// ------------------------------------------------------------------ rollout

// Everything a rollout batch needs besides its device buffers: the validated
// environment arguments and the shapes of the buffers.
struct RolloutPlan {
    EnvArgs ea{};
    int8_t team[kMaxAgents];
    int64_t ns = 0;               // agent slots
    bool mlp = false, persist = false, bf16_obs = false;
    bool kernel_sample = false;   // the 64-row policy kernel samples the actions
    bool striped = false;         // tile table in XCD segments (the 64-row kernel)
    int tile_rows = 0, max_tiles = 0, n_chunks = 0;
    int64_t state_bytes = 0;      // one state buffer (FEATURE has two)
};

// Device buffers of one rollout batch (from the handle, or carved from the
// no-allocation scratch).
struct RolloutBufs {
    float* logits = nullptr;
    float* ret = nullptr;
    void* state0 = nullptr;
    void* state1 = nullptr;
    uint8_t* done = nullptr;
    float* wt = nullptr;
    uint16_t* obs = nullptr;
    int32_t *perm = nullptr, *perm_env = nullptr, *hist = nullptr, *base = nullptr,
            *offsets = nullptr, *tile_off = nullptr;
    int4* tile_info = nullptr;
    uint8_t* actions = nullptr;   // actions sampled by the policy kernel
};

constexpr int kNumBufs = 15;

// Host-side validation of a batch (no device work) and its plan.
static malib_status plan_rollout(malib_pop_t pop, const malib_env_desc* env, int64_t n_envs,
                                 const int32_t* pair_assign, int64_t env_offset, int32_t horizon,
                                 RolloutPlan& plan)
{
    if (!pop)
        return fail(MALIB_E_INVAL, "pop is NULL");
    if (!env)
        return fail(MALIB_E_INVAL, "env is NULL");
    if (!pair_assign)
        return fail(MALIB_E_INVAL, "pair_assign is NULL");
    const int n_agents = env->n_agents;
    if (n_agents < 1 || n_agents > kMaxAgents)
        return fail(MALIB_E_INVAL, "n_agents must be in [1, %d]", kMaxAgents);
    if (env->n_actions != pop->A)
        return fail(MALIB_E_INVAL, "env n_actions (%d) differs from the population's (%d)",
                    env->n_actions, pop->A);
    if (n_envs < 1)
        return fail(MALIB_E_INVAL, "n_envs must be >= 1");
    if (n_envs > ((int64_t)1 << 26) / n_agents)
        return fail(MALIB_E_INVAL, "n_envs * n_agents exceeds 2^26");
    if (horizon < 1 || horizon > 100000)
        return fail(MALIB_E_INVAL, "horizon must be in [1, 100000]");
    if (env_offset < 0)
        return fail(MALIB_E_INVAL, "env_offset must be >= 0");
    if (env->init_mode != MALIB_INIT_PER_ENV && env->init_mode != MALIB_INIT_SHARED)
        return fail(MALIB_E_INVAL, "unknown init_mode %d", env->init_mode);
    int8_t* team = plan.team;
    if (env->team) {
        for (int k = 0; k < n_agents; ++k) {
            team[k] = env->team[k];
            if (team[k] != 1 && team[k] != -1)
                return fail(MALIB_E_INVAL, "team entries must be +1 or -1");
        }
    } else {
        if (n_agents != 2)
            return fail(MALIB_E_INVAL, "team may be NULL only for two seats");
        team[0] = 1;
        team[1] = -1;
    }
    EnvArgs& ea = plan.ea;
    ea.n_cus = pop->n_cus;
    ea.kind = env->kind;
    ea.n_agents = n_agents;
    ea.A = env->n_actions;
    ea.grid = env->grid;
    ea.d = env->d;
    ea.init_mode = env->init_mode;
    for (int k = 0; k < n_agents; ++k) {
        if (team[k] > 0)
            ea.team_row |= 1u << k;
        else
            ea.team_col |= 1u << k;
    }
    ea.Amat = env->A;
    ea.W = env->W;
    ea.emb = env->emb;
    ea.u = env->u;
    switch (env->kind) {
    case MALIB_ENV_MATRIX:
    case MALIB_ENV_ITER_MATRIX:
        if (n_agents != 2)
            return fail(MALIB_E_INVAL, "matrix games have two seats");
        if (!env->A)
            return fail(MALIB_E_INVAL, "matrix games need A");
        if (env->kind == MALIB_ENV_ITER_MATRIX && env->n_actions > 3)
            return fail(MALIB_E_UNSUPPORTED, "iterated matrix game supports <= 3 actions");
        if (env->kind == MALIB_ENV_ITER_MATRIX && pop->kind != MALIB_POLICY_TABULAR &&
            pop->in_dim != 8 * env->n_actions)
            return fail(MALIB_E_INVAL, "policy input width must be 8 * n_actions");
        if (env->kind == MALIB_ENV_MATRIX && pop->kind != MALIB_POLICY_TABULAR)
            return fail(MALIB_E_UNSUPPORTED, "the one-step matrix game has no observation; "
                                             "use tabular policies");
        break;
    case MALIB_ENV_PURSUIT:
        if (n_agents != 2 || env->n_actions != 5 || env->grid < 5 || env->grid > 16)
            return fail(MALIB_E_INVAL, "pursuit: 2 seats, 5 actions, 5 <= grid <= 16");
        if (pop->kind != MALIB_POLICY_TABULAR && pop->in_dim != 75)
            return fail(MALIB_E_INVAL, "pursuit observation has 75 inputs");
        break;
    case MALIB_ENV_FEATURE:
        if (!(env->d == 64 || env->d == 128 || env->d == 256 || env->d == 512))
            return fail(MALIB_E_UNSUPPORTED, "feature dimension must be 64/128/256/512");
        if (!env->W || !env->emb || !env->u)
            return fail(MALIB_E_INVAL, "feature dynamics need W, emb and u");
        if (pop->kind != MALIB_POLICY_TABULAR && pop->in_dim != env->d)
            return fail(MALIB_E_INVAL, "policy input width must equal d");
        break;
    default:
        return fail(MALIB_E_INVAL, "unknown environment kind %d", env->kind);
    }
    if (ea.team_row == 0 || ea.team_col == 0)
        return fail(MALIB_E_INVAL, "both sides need at least one seat");
    const int64_t ns = n_envs * n_agents;
    plan.ns = ns;
    plan.mlp = pop->kind != MALIB_POLICY_TABULAR;
    plan.persist = pop->kind == MALIB_POLICY_MLP_BF16 && !pop->generic &&
                   use_persist_kernel(env->kind, pop->in_pad, ns, pop->P);
    plan.tile_rows = pop->generic ? kGenericTileRows
                     : pop->kind == MALIB_POLICY_MLP_BF16
                         ? (plan.persist ? kPersistRows : kBf16TileRows)
                         : kF32TileRows;
    plan.striped = pop->kind == MALIB_POLICY_MLP_BF16 && !pop->generic && !plan.persist;
    plan.max_tiles = plan.striped ? striped_entries(ns, pop->P, plan.tile_rows)
                                  : max_tiles_for(ns, pop->P, plan.tile_rows);
    plan.n_chunks = (int)((ns + kBucketChunk - 1) / kBucketChunk);
    plan.state_bytes = state_bytes_per_env(env->kind, env->d) * n_envs;
    // bf16 observation rows for the 64-row policy kernel (its gather reads half
    // the bytes); the persistent kernel converts the fp32 state itself, since
    // at d = 512 the extra rows cost the env step more than they save
    plan.bf16_obs = env->kind == MALIB_ENV_FEATURE && pop->kind == MALIB_POLICY_MLP_BF16 &&
                    !pop->generic && !plan.persist;
    // feature games with the 64-row kernel: Gumbel-max sampling in the policy
    // kernel (its noise is drawn while the observation rows are fetched), so
    // the env step only reads one action byte per slot
    plan.kernel_sample = plan.bf16_obs;
    return MALIB_OK;
}

// Byte sizes of the batch's buffers, in the order of RolloutBufs (0 = unused).
static void buffer_sizes(const Pop& pop, const malib_env_desc* env, int64_t n_envs,
                         const RolloutPlan& plan, size_t (&sz)[kNumBufs])
{
    const int64_t ns = plan.ns;
    const bool feat = env->kind == MALIB_ENV_FEATURE;
    sz[0] = sizeof(float) * ns * pop.A;                                  // logits
    sz[1] = sizeof(float) * ns;                                          // ret
    sz[2] = plan.state_bytes;                                            // state0
    sz[3] = feat ? plan.state_bytes : 0;                                 // state1
    sz[4] = env->kind == MALIB_ENV_PURSUIT ? n_envs : 0;                 // done
    sz[5] = feat ? sizeof(float) * env->d * env->d : 0;                  // wt
    sz[6] = plan.bf16_obs ? sizeof(uint16_t) * env->d * n_envs : 0;     // obs
    const size_t pc = (size_t)pop.P * plan.n_chunks;
    sz[7] = plan.mlp ? sizeof(int32_t) * ns : 0;                         // perm
    sz[8] = plan.mlp ? sizeof(int32_t) * ns : 0;                         // perm_env
    sz[9] = plan.mlp ? sizeof(int32_t) * pc : 0;                         // hist
    sz[10] = plan.mlp ? sizeof(int32_t) * pc : 0;                        // base
    sz[11] = plan.mlp ? sizeof(int32_t) * (pop.P + 1) : 0;               // offsets
    sz[12] = plan.mlp ? sizeof(int32_t) * (pop.P + 1) : 0;               // tile_off
    sz[13] = plan.mlp ? sizeof(int4) * (size_t)plan.max_tiles : 0;       // tile_info
    sz[14] = plan.kernel_sample ? (size_t)ns : 0;                        // actions
}

static void assign_bufs(void* const (&ptr)[kNumBufs], RolloutBufs& b)
{
    b.logits = (float*)ptr[0];
    b.ret = (float*)ptr[1];
    b.state0 = ptr[2];
    b.state1 = ptr[3];
    b.done = (uint8_t*)ptr[4];
    b.wt = (float*)ptr[5];
    b.obs = (uint16_t*)ptr[6];
    b.perm = (int32_t*)ptr[7];
    b.perm_env = (int32_t*)ptr[8];
    b.hist = (int32_t*)ptr[9];
    b.base = (int32_t*)ptr[10];
    b.offsets = (int32_t*)ptr[11];
    b.tile_off = (int32_t*)ptr[12];
    b.tile_info = (int4*)ptr[13];
    b.actions = (uint8_t*)ptr[14];
}

// Whether the handle's growable buffers already hold the batch.
static bool handle_bufs_fit(const Pop& pop, const malib_env_desc* env, int64_t n_envs,
                            const RolloutPlan& plan)
{
    size_t sz[kNumBufs];
    buffer_sizes(pop, env, n_envs, plan, sz);
    const DevBuf* db[kNumBufs] = {&pop.logits, &pop.ret, &pop.state0, &pop.state1, &pop.done,
                                  &pop.wt, &pop.obs, &pop.perm, &pop.perm_env, &pop.hist,
                                  &pop.base, &pop.offsets, &pop.tile_off, &pop.tile_info,
                                  &pop.actions};
    for (int i = 0; i < kNumBufs; ++i)
        if (sz[i] > db[i]->bytes)
            return false;
    return true;
}

// The handle's growable buffers, enlarged as needed (may call hipMalloc).
static malib_status handle_bufs(malib_pop_t pop, const malib_env_desc* env, int64_t n_envs,
                                const RolloutPlan& plan, RolloutBufs& b)
{
    size_t sz[kNumBufs];
    buffer_sizes(*pop, env, n_envs, plan, sz);
    DevBuf* db[kNumBufs] = {&pop->logits, &pop->ret, &pop->state0, &pop->state1, &pop->done,
                      &pop->wt, &pop->obs, &pop->perm, &pop->perm_env, &pop->hist,
                      &pop->base, &pop->offsets, &pop->tile_off, &pop->tile_info,
                      &pop->actions};
    void* ptr[kNumBufs];
    for (int i = 0; i < kNumBufs; ++i) {
        ptr[i] = nullptr;
        if (sz[i]) {
            HIP_TRY(ensure(*db[i], sz[i]));
            ptr[i] = db[i]->ptr;
        }
    }
    assign_bufs(ptr, b);
    return MALIB_OK;
}

// The launch sequence of one batch on buffers `b`: set-up (returns cleared,
// bucketing, reset), `horizon` steps of policy forward -> env step (sampling
// inside), then the payoff reduction into the handle's table.  `snap_of`
// (host, [horizon], or NULL) maps a step to its trace snapshot; `prof`
// enables the handle's HIP-event timing.
static malib_status launch_rollout(malib_pop_t pop, const malib_env_desc* env, int64_t n_envs,
                                   const int32_t* pair_assign, uint64_t seed,
                                   int64_t env_offset, int32_t horizon, float* returns,
                                   const malib_trace* trace, const int* snap_of,
                                   const malib_traj* traj, RolloutPlan& plan,
                                   const RolloutBufs& b, bool prof, hipStream_t s)
{
    EnvArgs& ea = plan.ea;
    const int n_agents = env->n_agents;
    const int64_t ns = plan.ns;
    const bool mlp = plan.mlp, persist = plan.persist;
    ea.WT = b.wt;
    ea.obs = plan.bf16_obs ? b.obs : nullptr;
    if (traj) {
        ea.tr.act = traj->actions;
        ea.tr.rew = traj->rewards;
        ea.tr.flags = traj->flags;
        ea.tr.obs = env->kind == MALIB_ENV_MATRIX ? nullptr : traj->obs;
        ea.tr.base = traj->cursor % traj->capacity;
        ea.tr.cap = traj->capacity;
        ea.tr.horizon = horizon;
    }
    float* ret = b.ret;
    float* logits = b.logits;
    uint8_t* done = env->kind == MALIB_ENV_PURSUIT ? b.done : nullptr;
    void* cur = b.state0;
    void* nxt = env->kind == MALIB_ENV_FEATURE ? b.state1 : b.state0;
    auto pbeg = [&](int kind) { return prof ? prof_begin(*pop, kind, s) : -1; };
    auto pend = [&](int i) {
        if (prof)
            prof_end(*pop, i, s);
    };

    // ---- set-up: returns cleared (a fill kernel, no memset), bucketing, reset
    int pi = pbeg(MALIB_K_SETUP);
    HIP_TRY(launch_zero_f32(ret, ns, s));
    if (mlp)
        HIP_TRY(launch_bucket(pair_assign, ns, n_agents, pop->P, plan.tile_rows, plan.max_tiles,
                              plan.striped, b.hist, b.base, b.perm, b.perm_env, b.offsets,
                              b.tile_off, b.tile_info, pop->dev_flags, s));
    HIP_TRY(launch_reset(ea, n_envs, seed, env_offset, cur, done, s));
    if (env->kind == MALIB_ENV_FEATURE)
        HIP_TRY(launch_transpose(env->W, b.wt, env->d, s));
    pend(pi);
    if (trace && mlp) {
        if (trace->perm)
            HIP_TRY(hipMemcpyAsync(trace->perm, b.perm, sizeof(int32_t) * ns,
                                   hipMemcpyDeviceToDevice, s));
        if (trace->offsets)
            HIP_TRY(hipMemcpyAsync(trace->offsets, b.offsets, sizeof(int32_t) * (pop->P + 1),
                                   hipMemcpyDeviceToDevice, s));
    }

    // ---- the step loop
    const int64_t snap_b = snap_bytes_per_env(env->kind, env->d) * n_envs;
    for (int t = 0; t < horizon; ++t) {
        const int si = snap_of ? snap_of[t] : -1;
        if (si >= 0 && trace->states && snap_b > 0) {
            uint8_t* dst = (uint8_t*)trace->states + (int64_t)si * snap_b;
            if (env->kind == MALIB_ENV_PURSUIT)
                HIP_TRY(launch_snapshot_pursuit(cur, done, n_envs, dst, s));
            else
                HIP_TRY(hipMemcpyAsync(dst, cur, snap_b, hipMemcpyDeviceToDevice, s));
        }
        pi = pbeg(MALIB_K_POLICY);
        if (pop->kind == MALIB_POLICY_TABULAR)
            HIP_TRY(launch_tabular(pop->tab, pair_assign, ns, pop->A, pop->P, pop->dev_flags,
                                   logits, s));
        else if (pop->generic)
            HIP_TRY(launch_mlp_generic(*pop, env->kind, n_agents, env->grid, b.perm, b.perm_env,
                                       b.tile_info, plan.max_tiles, ns, cur, logits, s));
        else if (pop->kind == MALIB_POLICY_MLP_F32)
            HIP_TRY(launch_mlp_f32(*pop, b.perm, b.tile_info, ns, n_agents, cur, logits, s));
        else if (persist)
            HIP_TRY(launch_mlp_bf16_persist(*pop, b.perm, b.perm_env, b.tile_info, b.tile_off,
                                            ns, n_agents, cur, logits, s));
        else
        {
            KernelSample ks{b.actions, pop->dev_flags, seed, env_offset, t};
            // the logits are written only when a trace snapshot reads them
            float* lg = plan.kernel_sample && !(si >= 0 && trace->logits) ? nullptr : logits;
            HIP_TRY(launch_mlp_bf16(*pop, env->kind, n_agents, env->grid, env->d,
                                    plan.tile_rows, b.perm, b.perm_env, b.tile_info, ns,
                                    plan.bf16_obs ? (const void*)ea.obs : cur, lg,
                                    plan.kernel_sample ? &ks : nullptr, s));
        }
        pend(pi);
        if (si >= 0 && trace->logits)
            HIP_TRY(hipMemcpyAsync(trace->logits + (int64_t)si * ns * pop->A, logits,
                                   sizeof(float) * ns * pop->A, hipMemcpyDeviceToDevice, s));
        // action sampling happens inside the env step (one launch fewer per step)
        SampleArgs sa;
        sa.logits = logits;
        sa.seed = seed;
        sa.env_offset = env_offset;
        sa.t = t;
        sa.log = (trace && trace->actions) ? trace->actions + (int64_t)t * ns : nullptr;
        sa.flags = pop->dev_flags;
        sa.actions = plan.kernel_sample ? b.actions : nullptr;
        pi = pbeg(MALIB_K_ENV);
        HIP_TRY(launch_env_step(ea, sa, n_envs, cur, nxt, done, ret, pop->dev_frames, s));
        pend(pi);
        std::swap(cur, nxt);
        if (env->kind != MALIB_ENV_FEATURE)
            nxt = cur;
    }

    // ---- payoff reduction
    pi = pbeg(MALIB_K_PAYOFF);
    if (payoff_stream_fits(pop->P))
        HIP_TRY(launch_payoff_stream(ret, pair_assign, n_envs, n_agents, ea.team_row,
                                     ea.team_col, pop->P, pop->n_cus, pop->sum, pop->sumsq,
                                     pop->cnt, s));
    else if (mlp)
        HIP_TRY(launch_payoff_bucketed(ret, pair_assign, b.perm, b.offsets, n_envs, n_agents,
                                       ea.team_row, ea.team_col, pop->P, pop->n_cus, pop->sum,
                                       pop->sumsq, pop->cnt, s));
    else
        HIP_TRY(launch_payoff(ret, pair_assign, n_envs, n_agents, plan.team, pop->P, pop->sum,
                              pop->sumsq, pop->cnt, s));
    pend(pi);
    if (returns)
        HIP_TRY(hipMemcpyAsync(returns, ret, sizeof(float) * ns, hipMemcpyDeviceToDevice, s));
    if (env->kind != MALIB_ENV_PURSUIT)
        pop->host_frames += ns * (int64_t)horizon;
    pop->envs += n_envs;
    return MALIB_OK;
}

static malib_status rollout_impl(malib_pop_t pop, const malib_env_desc* env, int64_t n_envs,
                                 const int32_t* pair_assign, uint64_t seed, int64_t env_offset,
                                 int32_t horizon, float* returns, const malib_trace* trace,
                                 const malib_traj* traj, void* stream)
{
    RolloutPlan plan;
    {
        const malib_status st =
            plan_rollout(pop, env, n_envs, pair_assign, env_offset, horizon, plan);
        if (st != MALIB_OK)
            return st;
    }
    std::vector<int> snap_of;
    if (trace && trace->n_snap > 0) {
        if (!trace->snap_steps)
            return fail(MALIB_E_INVAL, "trace: snap_steps is NULL");
        snap_of.assign(horizon, -1);
        for (int i = 0; i < trace->n_snap; ++i) {
            int st = trace->snap_steps[i];
            if (st < 0 || st >= horizon)
                return fail(MALIB_E_INVAL, "trace: snapshot step %d outside [0, %d)", st,
                            horizon);
            snap_of[st] = i;
        }
    }
    hipStream_t s = (hipStream_t)stream;
    hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
    HIP_TRY(hipStreamIsCapturing(s, &cap));
    // growing a buffer synchronizes the device and frees memory, which a
    // capture in progress does not allow
    if (cap != hipStreamCaptureStatusNone && !handle_bufs_fit(*pop, env, n_envs, plan))
        return fail(MALIB_E_INVAL,
                    "the stream is being captured and this batch needs larger device buffers "
                    "than the handle holds: run a batch of this size outside the capture "
                    "first, or use malib_rollout_batch_noalloc");
    RolloutBufs b;
    {
        const malib_status st = handle_bufs(pop, env, n_envs, plan, b);
        if (st != MALIB_OK)
            return st;
    }
    if (!pop->graph_mode || trace || cap != hipStreamCaptureStatusNone)
        return launch_rollout(pop, env, n_envs, pair_assign, seed, env_offset, horizon, returns,
                              trace, snap_of.empty() ? nullptr : snap_of.data(), traj, plan, b,
                              true, s);
    // graph mode: record the batch (no HIP-event timing inside) on the
    // handle's own stream (recording runs nothing, and the caller's stream may
    // be the null stream, which cannot be captured), then replay it on the
    // caller's stream through the handle's executable graph, updated in place
    // when the batch has the same launch structure as the previous one
    if (!pop->graph_rec)
        HIP_TRY(hipStreamCreateWithFlags(&pop->graph_rec, hipStreamNonBlocking));
    HIP_TRY(hipStreamBeginCapture(pop->graph_rec, hipStreamCaptureModeThreadLocal));
    const malib_status st = launch_rollout(pop, env, n_envs, pair_assign, seed, env_offset,
                                           horizon, returns, nullptr, nullptr, traj, plan, b,
                                           false, pop->graph_rec);
    hipGraph_t graph = nullptr;
    const hipError_t ec = hipStreamEndCapture(pop->graph_rec, &graph);
    if (st != MALIB_OK) {
        if (graph)
            (void)hipGraphDestroy(graph);
        return st;
    }
    HIP_TRY(ec);
    bool updated = false;
    if (pop->graph_exec) {
        // an update rewrites the executable graph's kernel arguments: the
        // previous replay must have finished reading them
        if (pop->graph_done)
            HIP_TRY(hipEventSynchronize(pop->graph_done));
        hipGraphNode_t err_node = nullptr;
        hipGraphExecUpdateResult res;
        updated = hipGraphExecUpdate(pop->graph_exec, graph, &err_node, &res) == hipSuccess &&
                  res == hipGraphExecUpdateSuccess;
        if (!updated) {
            (void)hipGetLastError();
            (void)hipGraphExecDestroy(pop->graph_exec);
            pop->graph_exec = nullptr;
        }
    }
    hipError_t e = hipSuccess;
    if (!updated)
        e = hipGraphInstantiate(&pop->graph_exec, graph, nullptr, nullptr, 0);
    (void)hipGraphDestroy(graph);
    if (e != hipSuccess) {
        pop->graph_exec = nullptr;
        return fail(MALIB_E_HIP, "hipGraphInstantiate failed: %s", hipGetErrorString(e));
    }
    HIP_TRY(hipGraphLaunch(pop->graph_exec, s));
    if (!pop->graph_done)
        HIP_TRY(hipEventCreateWithFlags(&pop->graph_done, hipEventDisableTiming));
    HIP_TRY(hipEventRecord(pop->graph_done, s));
    return MALIB_OK;
}

malib_status malib_rollout_batch(malib_pop_t pop, const malib_env_desc* env, int64_t n_envs,
                                 const int32_t* pair_assign, uint64_t seed, int64_t env_offset,
                                 int32_t horizon, float* returns, const malib_trace* trace,
                                 void* stream)
{
    return rollout_impl(pop, env, n_envs, pair_assign, seed, env_offset, horizon, returns, trace,
                        nullptr, stream);
}

malib_status malib_rollout_batch_traj(malib_pop_t pop, const malib_env_desc* env,
                                      int64_t n_envs, const int32_t* pair_assign, uint64_t seed,
                                      int64_t env_offset, int32_t horizon, float* returns,
                                      malib_traj* traj, void* stream)
{
    if (!traj)
        return fail(MALIB_E_INVAL, "traj is NULL");
    if (!traj->actions || !traj->rewards || !traj->flags)
        return fail(MALIB_E_INVAL, "traj: actions, rewards and flags must not be NULL");
    if (traj->capacity < 1 || traj->cursor < 0)
        return fail(MALIB_E_INVAL, "traj: capacity must be >= 1 and cursor >= 0");
    const malib_status st = rollout_impl(pop, env, n_envs, pair_assign, seed, env_offset,
                                         horizon, returns, nullptr, traj, stream);
    if (st == MALIB_OK)
        traj->cursor += (int64_t)horizon * n_envs;
    return st;
}

// -------------------------------------------------------- no allocation

malib_status malib_rollout_batch_noalloc(malib_pop_t pop, const malib_env_desc* env,
                                         int64_t n_envs, const int32_t* pair_assign,
                                         uint64_t seed, int64_t env_offset, int32_t horizon,
                                         float* returns, void* stream)
{
    RolloutPlan plan;
    {
        const malib_status st =
            plan_rollout(pop, env, n_envs, pair_assign, env_offset, horizon, plan);
        if (st != MALIB_OK)
            return st;
    }
    if (!pop->scratch) {
        hipError_t e = hipSuccess;
        (void)scratch_address(pop->device, &e);
        return fail(MALIB_E_HIP, "the no-allocation scratch has no device address: %s",
                    hipGetErrorString(e));
    }
    size_t sz[kNumBufs];
    buffer_sizes(*pop, env, n_envs, plan, sz);
    void* ptr[kNumBufs];
    size_t off = 0;
    for (int i = 0; i < kNumBufs; ++i) {
        ptr[i] = nullptr;
        if (sz[i]) {
            ptr[i] = (unsigned char*)pop->scratch + off;
            off += (sz[i] + 255) / 256 * 256;
        }
    }
    if (off > kNoAllocScratchBytes)
        return fail(MALIB_E_INVAL,
                    "the batch needs %zu bytes of scratch, above the %zu bytes of "
                    "malib_rollout_batch_noalloc (use malib_rollout_batch)",
                    off, kNoAllocScratchBytes);
    RolloutBufs b;
    assign_bufs(ptr, b);
    return launch_rollout(pop, env, n_envs, pair_assign, seed, env_offset, horizon, returns,
                          nullptr, nullptr, nullptr, plan, b, false, (hipStream_t)stream);
}

// ------------------------------------------------------------------- payoff

malib_status malib_payoff_eval(malib_pop_t pop, void* stream, int32_t reset, double* mean,
                               int64_t* counts, double* stderr_out, malib_eval_stats* stats)
{
    if (!pop)
        return fail(MALIB_E_INVAL, "pop is NULL");
    hipStream_t s = (hipStream_t)stream;
    const size_t PP = (size_t)pop->P * pop->P;
    // the whole accumulator block in one copy (stream-ordered after the
    // batches), into the handle's pinned buffer
    HIP_TRY(hipMemcpyAsync(pop->host_acc, pop->acc, sizeof(unsigned long long) * (3 * PP + 2),
                           hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    const long long* sum = reinterpret_cast<const long long*>(pop->host_acc);
    const long long* sq = sum + PP;
    const long long* cnt = sum + 2 * PP;
    const unsigned long long frames = pop->host_acc[3 * PP];
    int flags;
    memcpy(&flags, pop->host_acc + 3 * PP + 1, sizeof(int));
    for (size_t i = 0; i < PP; ++i) {
        double n = (double)cnt[i];
        double m = cnt[i] > 0 ? ldexp((double)sum[i], -32) / n : NAN;
        if (mean)
            mean[i] = m;
        if (counts)
            counts[i] = cnt[i];
        if (stderr_out) {
            if (cnt[i] < 2) {
                stderr_out[i] = NAN;
            } else {
                double s2 = ldexp((double)sq[i], -20);
                double var = (s2 - n * m * m) / (n - 1.0);
                stderr_out[i] = sqrt(var > 0.0 ? var / n : 0.0);
            }
        }
    }
    if (stats) {
        stats->live_frames = pop->host_frames + (int64_t)frames;
        stats->envs = pop->envs;
        stats->device_flags = flags;
    }
    // clears are stream-ordered and complete before returning, so the next
    // batch may run on any stream
    if (reset) {
        HIP_TRY(hipMemsetAsync(pop->acc, 0, sizeof(unsigned long long) * (3 * PP + 1), s));
        pop->host_frames = 0;
        pop->envs = 0;
    }
    if (flags)
        HIP_TRY(hipMemsetAsync(pop->dev_flags, 0, sizeof(int), s));
    if (reset || flags)
        HIP_TRY(hipStreamSynchronize(s));
    if (flags)
        return fail(MALIB_E_DEVICE, "device flagged bad data (flags 0x%x:%s%s)", flags,
                    (flags & kErrPid) ? " policy id out of range" : "",
                    (flags & kErrNaN) ? " NaN logit" : "");
    return MALIB_OK;
}

// -------------------------------------------------------------- meta-sample

// Seat k draws from row 0 (one shared row) or row k (a row per seat).
static uint32_t default_seat_map(int n_sigma)
{
    return n_sigma == 1 ? 0u : 0x76543210u;
}

malib_status malib_meta_sample(const float* sigma, int32_t n_sigma, int32_t P, int64_t n_envs,
                               int32_t n_agents, uint64_t seed, int64_t env_offset,
                               int32_t* out, void* stream)
{
    if (!sigma || !out)
        return fail(MALIB_E_INVAL, "sigma and pair_assign_out must not be NULL");
    if (P < 1 || P > kMaxP)
        return fail(MALIB_E_INVAL, "n_policies must be in [1, %d]", kMaxP);
    if (n_agents < 1 || n_agents > kMaxAgents)
        return fail(MALIB_E_INVAL, "n_agents must be in [1, %d]", kMaxAgents);
    if (n_sigma != 1 && n_sigma != n_agents)
        return fail(MALIB_E_INVAL, "n_sigma must be 1 or n_agents");
    if (n_envs < 0 || n_envs > ((int64_t)1 << 26) / n_agents || env_offset < 0)
        return fail(MALIB_E_INVAL, "bad n_envs / env_offset");
    std::vector<unsigned long long> thr((size_t)n_sigma * P);
    for (int r = 0; r < n_sigma; ++r) {
        const float* row = sigma + (size_t)r * P;
        double total = 0.0;
        for (int m = 0; m < P; ++m) {
            if (!isfinite(row[m]) || row[m] < 0.0f)
                return fail(MALIB_E_INVAL, "sigma[%d][%d] is negative or not finite", r, m);
            total += (double)row[m];
        }
        if (!(total > 0.0))
            return fail(MALIB_E_INVAL, "sigma row %d has zero mass", r);
        double run = 0.0;
        for (int m = 0; m < P; ++m) {
            run += (double)row[m];
            double c = floor(run / total * 4294967296.0);
            thr[(size_t)r * P + m] = (unsigned long long)std::min(c, 4294967296.0);
        }
        thr[(size_t)r * P + P - 1] = 4294967296ull;
    }
    if (n_envs == 0)
        return MALIB_OK;
    hipStream_t s = (hipStream_t)stream;
    // Thresholds live in a device buffer that is freed in stream order; the
    // copy is staged synchronously from pageable memory before returning.
    unsigned long long* d_thr = nullptr;
    size_t nb = sizeof(unsigned long long) * thr.size();
    HIP_TRY(dev_malloc_async((void**)&d_thr, nb, s));
    HIP_TRY(hipMemcpyAsync(d_thr, thr.data(), nb, hipMemcpyHostToDevice, s));
    HIP_TRY(hipStreamSynchronize(s));
    HIP_TRY(launch_meta_sample(d_thr, default_seat_map(n_sigma), P, n_envs, n_agents, seed,
                               env_offset, out, s));
    HIP_TRY(hipFreeAsync(d_thr, s));
    return MALIB_OK;
}

// ---------------------------------------------------------------- meta-solver

malib_status malib_payoff_matrix(malib_pop_t pop, double* M, void* stream)
{
    if (!pop || !M)
        return fail(MALIB_E_INVAL, "pop and M must not be NULL");
    HIP_TRY(launch_payoff_matrix(pop->sum, pop->cnt, pop->P, M, (hipStream_t)stream));
    return MALIB_OK;
}

malib_status malib_solve_fp(const double* M, int32_t P, int32_t iterations, float* sigma,
                            double* gap, void* stream)
{
    if (!M || !sigma)
        return fail(MALIB_E_INVAL, "M and sigma must not be NULL");
    if (P < 1 || P > kMaxP)
        return fail(MALIB_E_INVAL, "n_policies must be in [1, %d]", kMaxP);
    if (iterations < 1 || iterations > (1 << 24))
        return fail(MALIB_E_INVAL, "iterations must be in [1, 2^24]");
    HIP_TRY(launch_solve_fp(M, P, iterations, sigma, gap, (hipStream_t)stream));
    return MALIB_OK;
}

malib_status malib_solve_alpharank(const double* M, int32_t P, double alpha, int32_t m,
                                   double* work, double* pi, float* sigma, void* stream)
{
    if (!M || !pi)
        return fail(MALIB_E_INVAL, "M and pi must not be NULL");
    if (P < 1 || P > kMaxP)
        return fail(MALIB_E_INVAL, "n_policies must be in [1, %d]", kMaxP);
    if (!(alpha >= 0.0) || !std::isfinite(alpha))
        return fail(MALIB_E_INVAL, "alpha must be finite and >= 0");
    if (m < 1 || m > 1000000)
        return fail(MALIB_E_INVAL, "population size m must be in [1, 10^6]");
    if (alpharank_needs_work(P) && !work)
        return fail(MALIB_E_INVAL, "n_policies > 128 needs a [P][P] fp64 workspace");
    HIP_TRY(launch_alpharank(M, P, alpha, m, work, pi, sigma, (hipStream_t)stream));
    return MALIB_OK;
}

malib_status malib_solve_lp(const double* M, int32_t P, double* work, double* value, double* x,
                            double* y, float* sigma, int32_t* pivots, void* stream)
{
    if (!M || !value || !x || !y)
        return fail(MALIB_E_INVAL, "M, value, x and y must not be NULL");
    if (P < 1 || P > kMaxP)
        return fail(MALIB_E_INVAL, "n_policies must be in [1, %d]", kMaxP);
    if (lp_needs_work(P) && !work)
        return fail(MALIB_E_INVAL, "n_policies > 96 needs a [P+1][2P+1] fp64 workspace");
    HIP_TRY(launch_lp(M, P, 64 * P + 256, work, value, x, y, sigma, pivots,
                      (hipStream_t)stream));
    return MALIB_OK;
}

malib_status malib_aggregate(const double* M, int32_t P, const float* sigma, int32_t br_row,
                             int32_t br_col, double* out, void* stream)
{
    if (!M || !sigma || !out)
        return fail(MALIB_E_INVAL, "M, sigma and out must not be NULL");
    if (P < 1 || P > kMaxP)
        return fail(MALIB_E_INVAL, "n_policies must be in [1, %d]", kMaxP);
    if (br_row < -1 || br_row >= P || br_col < -1 || br_col >= P)
        return fail(MALIB_E_INVAL, "best-response ids must be in [-1, n_policies)");
    HIP_TRY(launch_aggregate(M, P, sigma, br_row, br_col, out, (hipStream_t)stream));
    return MALIB_OK;
}

malib_status malib_meta_sample_device(const float* sigma, int32_t n_sigma, int32_t P,
                                      int64_t n_envs, int32_t n_agents, const int32_t* seat_row,
                                      uint64_t seed, int64_t env_offset, int32_t* out,
                                      void* stream)
{
    if (!sigma || !out)
        return fail(MALIB_E_INVAL, "sigma and pair_assign_out must not be NULL");
    if (P < 1 || P > kMaxP)
        return fail(MALIB_E_INVAL, "n_policies must be in [1, %d]", kMaxP);
    if (n_agents < 1 || n_agents > kMaxAgents)
        return fail(MALIB_E_INVAL, "n_agents must be in [1, %d]", kMaxAgents);
    uint32_t seat_map = 0;
    if (seat_row) {
        if (n_sigma < 1 || n_sigma > kMaxAgents)
            return fail(MALIB_E_INVAL, "n_sigma must be in [1, %d]", kMaxAgents);
        for (int k = 0; k < n_agents; ++k) {
            if (seat_row[k] < 0 || seat_row[k] >= n_sigma)
                return fail(MALIB_E_INVAL, "seat_row[%d] = %d is not a row of sigma", k,
                            seat_row[k]);
            seat_map |= (uint32_t)seat_row[k] << (4 * k);
        }
    } else {
        if (n_sigma != 1 && n_sigma != n_agents)
            return fail(MALIB_E_INVAL, "n_sigma must be 1 or n_agents");
        seat_map = default_seat_map(n_sigma);
    }
    if (n_envs < 0 || n_envs > ((int64_t)1 << 26) / n_agents || env_offset < 0)
        return fail(MALIB_E_INVAL, "bad n_envs / env_offset");
    if (n_envs == 0)
        return MALIB_OK;
    hipStream_t s = (hipStream_t)stream;
    unsigned long long* d_thr = nullptr;
    HIP_TRY(dev_malloc_async((void**)&d_thr, sizeof(unsigned long long) * (size_t)n_sigma * P,
                             s));
    HIP_TRY(launch_thresholds(sigma, n_sigma, P, d_thr, s));
    HIP_TRY(launch_meta_sample(d_thr, seat_map, P, n_envs, n_agents, seed, env_offset, out, s));
    HIP_TRY(hipFreeAsync(d_thr, s));
    return MALIB_OK;
}

// ---------------------------------------------------------------- profiling

malib_status malib_pop_set_graph(malib_pop_t pop, int32_t enable)
{
    if (!pop)
        return fail(MALIB_E_INVAL, "pop is NULL");
    pop->graph_mode = enable != 0;
    return MALIB_OK;
}

malib_status malib_profile_enable(malib_pop_t pop, int32_t mask, int32_t every)
{
    if (!pop)
        return fail(MALIB_E_INVAL, "pop is NULL");
    if (every < 1 || mask < 0 || mask >= (1 << MALIB_K_COUNT))
        return fail(MALIB_E_INVAL, "bad profile mask %d / every %d", mask, every);
    pop->prof.mask = mask;
    pop->prof.every = every;
    for (int k = 0; k < MALIB_K_COUNT; ++k)
        pop->prof.seen[k] = 0;
    pop->prof.used = 0;
    pop->prof.kind.clear();
    return MALIB_OK;
}

malib_status malib_profile_read(malib_pop_t pop, int32_t kernel, double* total_ms,
                                int64_t* launches)
{
    if (!pop)
        return fail(MALIB_E_INVAL, "pop is NULL");
    if (kernel < 0 || kernel >= MALIB_K_COUNT)
        return fail(MALIB_E_INVAL, "unknown kernel class %d", kernel);
    double ms = 0.0;
    int64_t n = 0;
    for (size_t i = 0; i < pop->prof.used; ++i) {
        if (pop->prof.kind[i] != kernel)
            continue;
        HIP_TRY(hipEventSynchronize(pop->prof.pool[i].stop));
        float e = 0.0f;
        HIP_TRY(hipEventElapsedTime(&e, pop->prof.pool[i].start, pop->prof.pool[i].stop));
        ms += e;
        ++n;
    }
    if (total_ms)
        *total_ms = ms;
    if (launches)
        *launches = n;
    return MALIB_OK;
}

// -------------------------------------------------------------- diagnostics

malib_status malib_debug_tanh_ref(const float* x, float* y, int64_t n, void* stream)
{
    if (!x || !y || n < 0)
        return fail(MALIB_E_INVAL, "bad arguments");
    if (n == 0)
        return MALIB_OK;
    HIP_TRY(launch_debug_tanh(x, y, n, (hipStream_t)stream));
    return MALIB_OK;
}

malib_status malib_debug_bf16(const float* x, uint16_t* y, int64_t n, void* stream)
{
    if (!x || !y || n < 0 || (n & 1))
        return fail(MALIB_E_INVAL, "bad arguments (n must be even)");
    if (n == 0)
        return MALIB_OK;
    HIP_TRY(launch_debug_bf16(x, y, n, (hipStream_t)stream));
    return MALIB_OK;
}

malib_status malib_debug_philox(const uint64_t* ctr, uint64_t key0, uint64_t key1,
                                uint64_t* out, int64_t n, void* stream)
{
    if (!ctr || !out || n < 0)
        return fail(MALIB_E_INVAL, "bad arguments");
    if (n == 0)
        return MALIB_OK;
    HIP_TRY(launch_debug_philox(ctr, key0, key1, out, n, (hipStream_t)stream));
    return MALIB_OK;
}

}  // extern "C"
