// engine.hip -- the C ABI of include/fgd.h: engine state, argument checks,
// stream-ordered topology upload and kernel launches.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "../../include/fgd.h"
#include "api.hpp"
#include "kernels.hpp"
#include "kernels_wg.hpp"
#include "topology.hpp"

namespace {

thread_local std::string g_last_error;

fgd_status fail(fgd_status st, const char *f, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, f);
    std::vsnprintf(buf, sizeof buf, f, ap);
    va_end(ap);
    g_last_error = buf;
    return st;
}

fgd_status hip_fail(hipError_t e, const char *what) {
    return fail(FGD_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// Makes a device current for one call and restores the caller's current
// device on every return path, so no call leaves the thread switched.
class DeviceGuard {
  public:
    DeviceGuard() = default;
    DeviceGuard(const DeviceGuard &) = delete;
    DeviceGuard &operator=(const DeviceGuard &) = delete;
    ~DeviceGuard() {
        if (switched_) (void)hipSetDevice(prev_);
    }
    hipError_t enter(int dev) {
        hipError_t err = hipGetDevice(&prev_);
        if (err != hipSuccess || prev_ == dev) return err;
        err = hipSetDevice(dev);
        switched_ = err == hipSuccess;
        return err;
    }

  private:
    int prev_ = 0;
    bool switched_ = false;
};

fgd_status from_topo(fgd::TopoStatus s, const std::string &err) {
    if (s == fgd::TopoStatus::ok) return FGD_OK;
    g_last_error = err;
    return s == fgd::TopoStatus::invalid_arg ? FGD_ERR_INVALID_ARG : FGD_ERR_TOPOLOGY;
}

int elem_size(int32_t dtype) { return dtype == FGD_BF16 ? 2 : 4; }

// Device copies of the packed topology tables.  A ring of slots, each with a
// pinned host staging buffer and an event recorded after the last kernel
// that read the slot, so a slot is refilled only once that kernel is done.
constexpr int kTopoRing = 8;
#ifndef FGD_MAX_BLOCKS_PER_CU
#define FGD_MAX_BLOCKS_PER_CU 8
#endif
constexpr int kMaxBlocksPerCu = FGD_MAX_BLOCKS_PER_CU;
constexpr int kTimingPool = 4096;
constexpr int64_t kMix1Chunks = 4096;  // chunks the Mix1 half's tiles are cut into (at most)
// LDS of a worker-group step block: two blocks share a compute unit's 160 KiB.
constexpr size_t kWgMaxLds = 80 * 1024;

}  // namespace

struct fgd_engine {
    fgd_config cfg{};
    bool host_only = true;
    fgd::MixTopology slot[2];   // [0] Mix1, [1] Mix2
    bool slot_set[2] = {false, false};
    std::vector<int64_t> subset;  // Mix2 subset segments, [n][2] (empty: Mix2 everywhere)
    uint64_t topo_version = 0;  // bumped by every fgd_set_topology and fgd_set_mix2_subset

    // Device side (absent for host-only engines).
    int num_cus = 0;
    size_t topo_capacity = 0;   // bytes per ring slot
    void *d_topo[kTopoRing] = {};
    void *h_topo[kTopoRing] = {};
    hipEvent_t topo_done[kTopoRing] = {};
    bool topo_pending[kTopoRing] = {};
    int topo_next = 0;
    int topo_current = -1;      // ring slot holding topo_version
    uint64_t topo_current_version = ~0ull;
    hipStream_t topo_stream = nullptr;
    double *d_partials = nullptr;
    size_t partials_capacity = 0;  // doubles, per step kernel
    double *d_chunk_partials = nullptr;  // Mix1 half: [kMix1Chunks][n_cd][M]
    int *d_counter = nullptr;            // Mix1 half: chunk counter

    // Kernel timing.
    bool timing = false;
    std::vector<hipEvent_t> ev_start, ev_stop;
    int64_t timed = 0;
};

namespace {

fgd_status check_engine(const fgd_engine *e) {
    if (!e) return fail(FGD_ERR_INVALID_ARG, "engine is NULL");
    return FGD_OK;
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Byte range [lo, hi) spanned by an [M][ld] array of element size es, P used.
void span(const void *p, int64_t M, int64_t ld, int64_t P, int es, uintptr_t &lo, uintptr_t &hi) {
    lo = reinterpret_cast<uintptr_t>(p);
    hi = lo + static_cast<uintptr_t>(((M - 1) * ld + P) * es);
}

bool overlap(uintptr_t a0, uintptr_t a1, uintptr_t b0, uintptr_t b1) { return a0 < b1 && b0 < a1; }

int32_t n_cd_rows(const fgd_engine *e) {
    return e->slot[1].effective_rounds() + 1 + e->slot[0].effective_rounds() + 1 + 1;
}

fgd::MixDev mix_dev(const fgd::MixTopology &t, const void *tables) {
    fgd::MixDev d{};
    d.kind = t.kind;
    d.rounds = t.rounds;
    d.width = t.width;
    d.table = static_cast<const int2 *>(tables);
    return d;
}

bool lookup_split(int M, int32_t dtype, int k1, int k2, bool subset, bool mix_state, fgd::SplitSet &ks) {
    return dtype == FGD_BF16 ? fgd::split_kernels_bf16(M, k1, k2, subset, mix_state, &ks)
                             : fgd::split_kernels_f32(M, k1, k2, subset, mix_state, &ks);
}

bool lookup(int M, int32_t dtype, int k1, int k2, bool mix_state, bool subset, fgd::KernelSet &ks) {
    if (mix_state)
        return dtype == FGD_BF16 ? fgd::kernels_bf16_ms(M, k1, k2, subset, &ks)
                                 : fgd::kernels_f32_ms(M, k1, k2, subset, &ks);
    return dtype == FGD_BF16 ? fgd::kernels_bf16(M, k1, k2, subset, &ks) : fgd::kernels_f32(M, k1, k2, subset, &ks);
}

// Byte offset of the subset segments in a ring slot (after both tables, 16-byte aligned).
size_t subset_offset(size_t tables_bytes) { return (tables_bytes + 15) & ~static_cast<size_t>(15); }

// Makes sure the device holds the current topology for `stream` and returns
// the ring slot.  Uploads (stream-ordered) when the topology changed or the
// stream differs from the one that received the last upload.
fgd_status ensure_topology(fgd_engine *e, hipStream_t stream, int &ring) {
    if (e->topo_current >= 0 && e->topo_current_version == e->topo_version && e->topo_stream == stream) {
        ring = e->topo_current;
        return FGD_OK;
    }
    std::vector<int32_t> t1, t2;
    e->slot[0].pack_tables(t1);
    e->slot[1].pack_tables(t2);
    const size_t b1 = t1.size() * sizeof(int32_t), b2 = t2.size() * sizeof(int32_t);
    const size_t so = subset_offset(b1 + b2), bs = e->subset.size() * sizeof(int64_t);
    if (so + bs > e->topo_capacity) return fail(FGD_ERR_UNSUPPORTED, "topology tables exceed the device slot");
    const int r = e->topo_next;
    e->topo_next = (e->topo_next + 1) % kTopoRing;
    if (e->topo_pending[r]) {
        hipError_t err = hipEventSynchronize(e->topo_done[r]);
        if (err != hipSuccess) return hip_fail(err, "waiting for a topology slot");
        e->topo_pending[r] = false;
    }
    char *h = static_cast<char *>(e->h_topo[r]);
    if (b1) std::memcpy(h, t1.data(), b1);
    if (b2) std::memcpy(h + b1, t2.data(), b2);
    if (bs) std::memcpy(h + so, e->subset.data(), bs);
    const size_t total = bs ? so + bs : b1 + b2;
    if (total) {
        hipError_t err = hipMemcpyAsync(e->d_topo[r], h, total, hipMemcpyHostToDevice, stream);
        if (err != hipSuccess) return hip_fail(err, "uploading the topology");
    }
    e->topo_current = r;
    e->topo_current_version = e->topo_version;
    e->topo_stream = stream;
    ring = r;
    return FGD_OK;
}

// Device addresses of the Mix1 and Mix2 tables and of the subset segments
// inside a ring slot.
void table_ptrs(const fgd_engine *e, int ring, const void *&t1, const void *&t2, const int64_t *&seg) {
    auto bytes = [&](const fgd::MixTopology &t) {
        return static_cast<size_t>(t.kind == 2 ? t.rounds * t.width : 0) * e->cfg.num_workers * 2 * sizeof(int32_t);
    };
    const size_t b1 = bytes(e->slot[0]), b2 = bytes(e->slot[1]);
    t1 = e->d_topo[ring];
    t2 = static_cast<const char *>(e->d_topo[ring]) + b1;
    seg = e->subset.empty() ? nullptr
                            : reinterpret_cast<const int64_t *>(static_cast<const char *>(e->d_topo[ring]) +
                                                                subset_offset(b1 + b2));
}

int64_t tiles_of(int64_t P, int v) {
    const int64_t per = static_cast<int64_t>(fgd::kBlock) * v;
    return (P + per - 1) / per;
}

// Resident blocks per CU of the standalone consensus kernel, a read-only
// stream of every row.  Up to 16 workers a lane already has a load of every
// row in flight and more blocks only add DRAM contention (8 x 1.1e9 bf16:
// 2.69 ms with 2 blocks, 2.72 with 4, 2.89 with 8, 4.32 with 1); with more
// workers a lane holds one parameter and the occupancy covers the latency
// (64 x 124M f32: 5.05 ms with 8, 5.16 with 2).
constexpr int consensus_blocks_per_cu(int num_workers) { return num_workers <= 16 ? 2 : 8; }

fgd_status grid_for_cus(int num_cus, const void *kernel, size_t lds, int64_t ntiles, int &grid,
                        int cap = kMaxBlocksPerCu) {
    int per_cu = 0;
    if (lds > 65536) {
        hipError_t err = hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
        if (err != hipSuccess) return hip_fail(err, "raising the kernel's LDS limit");
    }
    hipError_t err = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, fgd::kBlock, lds);
    if (err != hipSuccess) return hip_fail(err, "occupancy query");
    if (per_cu < 1) return fail(FGD_ERR_UNSUPPORTED, "kernel does not fit on a compute unit (LDS %zu bytes)", lds);
    per_cu = std::min(per_cu, std::min(cap, kMaxBlocksPerCu));
    const int64_t g = std::min<int64_t>(static_cast<int64_t>(per_cu) * num_cus, std::max<int64_t>(ntiles, 1));
    grid = static_cast<int>(g);
    return FGD_OK;
}

fgd_status grid_for(fgd_engine *e, const void *kernel, size_t lds, int64_t ntiles, int &grid, int cap = kMaxBlocksPerCu) {
    return grid_for_cus(e->num_cus, kernel, lds, ntiles, grid, cap);
}

fgd_status launch(const void *kernel, int grid, size_t lds, hipStream_t stream, void *arg) {
    void *args[] = {arg};
    if (lds > 65536) {
        hipError_t err = hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
        if (err != hipSuccess) return hip_fail(err, "raising the kernel's LDS limit");
    }
    hipError_t err = hipLaunchKernel(kernel, dim3(grid), dim3(fgd::kBlock), args, lds, stream);
    if (err != hipSuccess) return hip_fail(err, "kernel launch");
    return FGD_OK;
}

fgd_status launch_finalize(const double *partials, int nblocks, int n, double *out, hipStream_t stream) {
    hipLaunchKernelGGL(fgd::finalize_kernel, dim3(n), dim3(256), 0, stream, partials, nblocks, n, out);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return hip_fail(err, "finalize launch");
    return FGD_OK;
}

void release(fgd_engine *e) {
    for (int r = 0; r < kTopoRing; ++r) {
        if (e->d_topo[r]) (void)hipFree(e->d_topo[r]);
        if (e->h_topo[r]) (void)hipHostFree(e->h_topo[r]);
        if (e->topo_done[r]) (void)hipEventDestroy(e->topo_done[r]);
    }
    if (e->d_partials) (void)hipFree(e->d_partials);
    if (e->d_chunk_partials) (void)hipFree(e->d_chunk_partials);
    if (e->d_counter) (void)hipFree(e->d_counter);
    for (auto ev : e->ev_start) (void)hipEventDestroy(ev);
    for (auto ev : e->ev_stop) (void)hipEventDestroy(ev);
}

// Step parameters every kernel of a step shares.
void fill_common(const fgd_engine *e, int ring, int v, fgd::StepParams &p) {
    const fgd_config &c = e->cfg;
    p.P = c.num_params;
    p.ld = c.ld;
    p.ntiles = tiles_of(c.num_params, v);
    p.M = c.num_workers;
    p.lr = c.outer_lr;
    p.mu = c.momentum;
    p.nesterov = c.nesterov;
    const void *t1, *t2;
    const int64_t *seg;
    table_ptrs(e, ring, t1, t2, seg);
    p.mix1 = mix_dev(e->slot[0], t1);
    p.mix2 = mix_dev(e->slot[1], t2);
    p.n_seg = static_cast<int32_t>(e->subset.size() / 2);
    p.seg = seg;
}

// LDS rows for the table slots a kernel mixes with (use1 / use2: Mix1 / Mix2).
int32_t lds_rows_for(const fgd_engine *e, bool use1, bool use2) {
    const bool t1 = use1 && e->slot[0].kind == 2, t2 = use2 && e->slot[1].kind == 2;
    const bool padded = (t1 && e->slot[0].padded) || (t2 && e->slot[1].padded);
    return (t1 || t2) ? e->cfg.num_workers + (padded ? 1 : 0) : 0;
}

// Whether the 64-worker worker-group kernel serves this engine's step (a
// CSR Mix2, a CSR or global Mix1, sparse tables that fit in LDS beside the
// rows, no subset, no state mixing, per-lane row offsets below 2^32 bytes);
// if so its LDS bytes and rows per wave.
bool wg_step_fits(const fgd_engine *e, fgd::WgKernel &k, size_t &lds, int &wave_rows) {
    const fgd_config &c = e->cfg;
    const fgd::MixTopology &s1 = e->slot[0], &s2 = e->slot[1];
    if (c.num_workers != fgd::kWgWorkers || !e->subset.empty() || c.mix1_state) return false;
    if (s2.kind != 2 || s2.rounds > fgd::kWgR2 || s2.width > fgd::kWgMaxWidth) return false;
    if (s1.kind == 2 && (s1.rounds > fgd::kWgR1 || s1.width > fgd::kWgMaxWidth)) return false;
    if (!fgd::wg_kernel(c.param_dtype == FGD_BF16, s1.kind, s2.kind, &k)) return false;
    const int64_t es = elem_size(c.param_dtype);
    if ((3 * c.ld + fgd::kWgTile) * std::max<int64_t>(es, 4) + 64 > int64_t{0xFFFFFFFF}) return false;
    const bool padded = (s1.kind == 2 && s1.padded) || s2.padded;
    wave_rows = fgd::kWgWorkers + (padded ? 1 : 0);
    const size_t entries = static_cast<size_t>(s1.kind == 2 ? s1.rounds * s1.width : 0) * fgd::kWgWorkers +
                           static_cast<size_t>(s2.rounds) * s2.width * fgd::kWgWorkers;
    lds = static_cast<size_t>(fgd::kWavesPerBlock) * wave_rows * fgd::kWgRowBytes + entries * sizeof(int2);
    return lds <= kWgMaxLds;
}

// Checks a device [M][ld] array: non-NULL and 16-byte aligned.
bool bad_rows(const void *p) { return !p || !aligned16(p); }

// True when the [M][ld] spans of a (element size ea) and b (eb) overlap.
bool rows_overlap(const fgd_engine *e, const void *a, int ea, const void *b, int eb) {
    const fgd_config &c = e->cfg;
    if (c.num_params == 0) return false;
    uintptr_t a0, a1, b0, b1;
    span(a, c.num_workers, c.ld, c.num_params, ea, a0, a1);
    span(b, c.num_workers, c.ld, c.num_params, eb, b0, b1);
    return overlap(a0, a1, b0, b1);
}

}  // namespace

// ------------------------------------------- consensus without allocation
//
// fgd_consensus_distance_noalloc keeps its per-block partials in this array
// instead of engine memory: 2048 blocks (256 compute units x 8 resident
// blocks) x FGD_MAX_WORKERS doubles, 1 MiB on every device the library runs
// on, held until the process ends.  Host code never uses the name itself
// (on the host it is only a stand-in for the symbol): its device address is
// taken once per device with hipGetSymbolAddress and kept below.
namespace {
constexpr int kNoAllocBlocks = 2048;
constexpr int kNoAllocDoubles = kNoAllocBlocks * FGD_MAX_WORKERS;
constexpr int kNoAllocDevices = 64;
}  // namespace

static __device__ __align__(256) double scratch[kNoAllocDoubles];

namespace {

struct NoAllocDevice {
    bool ready = false;
    double *ptr = nullptr;  // device address of `scratch` on this device
    int num_cus = 0;
};
std::mutex g_noalloc_mutex;
NoAllocDevice g_noalloc[kNoAllocDevices];

// The scratch address and compute-unit count of the current device `dev`,
// resolved on the first call for that device (with it current).
fgd_status noalloc_device(int dev, double *&ptr, int &num_cus) {
    if (dev < 0 || dev >= kNoAllocDevices) return fail(FGD_ERR_UNSUPPORTED, "device %d is beyond %d", dev, kNoAllocDevices);
    std::lock_guard<std::mutex> lock(g_noalloc_mutex);
    NoAllocDevice &d = g_noalloc[dev];
    if (!d.ready) {
        void *p = nullptr;
        hipError_t err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (err != hipSuccess) return hip_fail(err, "resolving the static consensus scratch");
        int cus = 0;
        err = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
        if (err != hipSuccess) return hip_fail(err, "querying the compute-unit count");
        d.ptr = static_cast<double *>(p);
        d.num_cus = cus;
        d.ready = true;
    }
    ptr = d.ptr;
    num_cus = d.num_cus;
    return FGD_OK;
}

// Compute units of the current device (sizes persistent grids of the
// engine-free calls), queried once per device.
constexpr int kCuCacheDevices = 64;
std::mutex g_cu_mutex;
int g_cu_count[kCuCacheDevices] = {};
fgd_status current_device_cus(int &num_cus) {
    int dev = 0;
    hipError_t err = hipGetDevice(&dev);
    if (err != hipSuccess) return hip_fail(err, "querying the current device");
    if (dev < 0 || dev >= kCuCacheDevices) return fail(FGD_ERR_UNSUPPORTED, "device %d is beyond %d", dev, kCuCacheDevices);
    std::lock_guard<std::mutex> lock(g_cu_mutex);
    if (g_cu_count[dev] == 0) {
        int cus = 0;
        err = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
        if (err != hipSuccess) return hip_fail(err, "querying the compute-unit count");
        g_cu_count[dev] = cus > 0 ? cus : 1;
    }
    num_cus = g_cu_count[dev];
    return FGD_OK;
}

}  // namespace

namespace fgd {

fgd_status api_fail(fgd_status st, const char *f, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, f);
    std::vsnprintf(buf, sizeof buf, f, ap);
    va_end(ap);
    g_last_error = buf;
    return st;
}

void api_clear() { g_last_error.clear(); }

fgd_status api_device_cus(int &num_cus) { return current_device_cus(num_cus); }

}  // namespace fgd

extern "C" {

const char *fgd_status_string(int32_t s) {
    switch (s) {
        case FGD_OK: return "FGD_OK";
        case FGD_ERR_INVALID_ARG: return "FGD_ERR_INVALID_ARG";
        case FGD_ERR_TOPOLOGY: return "FGD_ERR_TOPOLOGY";
        case FGD_ERR_UNSUPPORTED: return "FGD_ERR_UNSUPPORTED";
        case FGD_ERR_OUT_OF_MEMORY: return "FGD_ERR_OUT_OF_MEMORY";
        case FGD_ERR_HIP: return "FGD_ERR_HIP";
        case FGD_ERR_STATE: return "FGD_ERR_STATE";
        default: return "FGD_UNKNOWN_STATUS";
    }
}

const char *fgd_last_error(void) { return g_last_error.c_str(); }

// Source hashes stamped in by the build (paper_2606_22768_amd/build.py).
#ifndef FGD_HASH_ALL
#define FGD_HASH_ALL "unstamped"
#endif
#ifndef FGD_HASH_STEP
#define FGD_HASH_STEP "unstamped"
#endif
#ifndef FGD_HASH_JS
#define FGD_HASH_JS "unstamped"
#endif

const char *fgd_source_hash(int32_t component) {
    switch (component) {
        case 0: return FGD_HASH_ALL;
        case 1: return FGD_HASH_STEP;
        case 2: return FGD_HASH_JS;
        default: return "";
    }
}

fgd_status fgd_create(const fgd_config *cfg, fgd_engine **out) {
    g_last_error.clear();
    if (!cfg || !out) return fail(FGD_ERR_INVALID_ARG, "cfg and out must not be NULL");
    *out = nullptr;
    if (cfg->struct_size != sizeof(fgd_config))
        return fail(FGD_ERR_INVALID_ARG, "struct_size %u does not match sizeof(fgd_config) %zu", cfg->struct_size,
                    sizeof(fgd_config));
    if (cfg->state_dtype != FGD_F32 && cfg->state_dtype != FGD_BF16)
        return fail(FGD_ERR_INVALID_ARG, "unknown state_dtype %d", cfg->state_dtype);
    if (cfg->state_dtype != FGD_F32) return fail(FGD_ERR_UNSUPPORTED, "the momentum is stored in float32 only");
    if (cfg->nesterov != 0 && cfg->nesterov != 1) return fail(FGD_ERR_INVALID_ARG, "nesterov must be 0 or 1");
    if (cfg->mix1_state != 0 && cfg->mix1_state != 1) return fail(FGD_ERR_INVALID_ARG, "mix1_state must be 0 or 1");
    if (cfg->reserved != 0) return fail(FGD_ERR_INVALID_ARG, "reserved must be 0");
    if (cfg->num_workers < 1 || cfg->num_workers > FGD_MAX_WORKERS)
        return fail(FGD_ERR_INVALID_ARG, "num_workers %d is outside [1, %d]", cfg->num_workers, FGD_MAX_WORKERS);
    if (cfg->num_params < 0) return fail(FGD_ERR_INVALID_ARG, "num_params is negative");
    if (cfg->param_dtype != FGD_F32 && cfg->param_dtype != FGD_BF16)
        return fail(FGD_ERR_INVALID_ARG, "unknown param_dtype %d", cfg->param_dtype);
    if (cfg->ld < cfg->num_params) return fail(FGD_ERR_INVALID_ARG, "ld < num_params");
    if ((cfg->ld * elem_size(cfg->param_dtype)) % 16 != 0 || cfg->ld % 4 != 0)
        return fail(FGD_ERR_INVALID_ARG, "rows must be 16-byte aligned: ld * elem_size and ld * 4 must be multiples of 16");
    if (!std::isfinite(cfg->outer_lr) || !std::isfinite(cfg->momentum))
        return fail(FGD_ERR_INVALID_ARG, "outer_lr and momentum must be finite");

    fgd_engine *e = new (std::nothrow) fgd_engine();
    if (!e) return fail(FGD_ERR_OUT_OF_MEMORY, "host allocation failed");
    e->cfg = *cfg;
    e->host_only = cfg->device < 0;
    if (!e->host_only) {
        DeviceGuard dg;
        hipError_t err = dg.enter(cfg->device);
        if (err != hipSuccess) {
            delete e;
            return hip_fail(err, "selecting the engine's device");
        }
        err = hipDeviceGetAttribute(&e->num_cus, hipDeviceAttributeMultiprocessorCount, cfg->device);
        if (err != hipSuccess) {
            delete e;
            return hip_fail(err, "querying the compute-unit count");
        }
        const size_t M = static_cast<size_t>(cfg->num_workers);
        // Largest packed tables (both slots, FGD_MAX_ROUNDS rounds, width M),
        // then the largest subset.
        e->topo_capacity = subset_offset(2 * static_cast<size_t>(FGD_MAX_ROUNDS) * M * M * 2 * sizeof(int32_t)) +
                           static_cast<size_t>(FGD_MAX_SUBSET_SEGMENTS) * 2 * sizeof(int64_t);
        const int n_cd_max = 2 * FGD_MAX_ROUNDS + 3;
        e->partials_capacity = static_cast<size_t>(e->num_cus) * kMaxBlocksPerCu * n_cd_max * M;
        for (int r = 0; r < kTopoRing && err == hipSuccess; ++r) {
            err = hipMalloc(&e->d_topo[r], e->topo_capacity);
            if (err == hipSuccess) err = hipHostMalloc(&e->h_topo[r], e->topo_capacity, hipHostMallocDefault);
            if (err == hipSuccess) err = hipEventCreateWithFlags(&e->topo_done[r], hipEventDisableTiming);
        }
        if (err == hipSuccess) err = hipMalloc(&e->d_partials, e->partials_capacity * sizeof(double));
        // The Mix1 half of split execution has its own consensus scratch and
        // counter: it may be enqueued on another stream.
        if (err == hipSuccess)
            err = hipMalloc(&e->d_chunk_partials,
                            static_cast<size_t>(kMix1Chunks) * (FGD_MAX_ROUNDS + 1) * M * sizeof(double));
        if (err == hipSuccess) err = hipMalloc(&e->d_counter, 64);
        if (err != hipSuccess) {
            release(e);
            delete e;
            return fail(err == hipErrorOutOfMemory ? FGD_ERR_OUT_OF_MEMORY : FGD_ERR_HIP, "device set-up: %s",
                        hipGetErrorString(err));
        }
    }
    *out = e;
    return FGD_OK;
}

fgd_status fgd_destroy(fgd_engine *e) {
    if (!e) return FGD_OK;
    if (!e->host_only) {
        DeviceGuard dg;
        (void)dg.enter(e->cfg.device);
        (void)hipDeviceSynchronize();
        release(e);
    }
    delete e;
    return FGD_OK;
}

fgd_status fgd_set_topology(fgd_engine *e, int32_t which, int32_t kind, const int32_t *row_ptr,
                            const int32_t *col_idx, const float *weights, int32_t num_rounds,
                            const uint8_t *edge_masks, int32_t reweight) {
    g_last_error.clear();
    if (fgd_status st = check_engine(e)) return st;
    if (which != FGD_MIX1 && which != FGD_MIX2) return fail(FGD_ERR_INVALID_ARG, "which must be FGD_MIX1 or FGD_MIX2");
    fgd::MixTopology t;
    std::string err;
    fgd::TopoStatus ts = fgd::build_mix_topology(e->cfg.num_workers, kind, row_ptr, col_idx, weights, num_rounds,
                                                 edge_masks, reweight, t, err);
    if (ts != fgd::TopoStatus::ok) return from_topo(ts, err);
    e->slot[which - 1] = std::move(t);
    e->slot_set[which - 1] = true;
    ++e->topo_version;
    return FGD_OK;
}

fgd_status fgd_set_mix2_subset(fgd_engine *e, const int64_t *segments, int32_t num_segments) {
    g_last_error.clear();
    if (fgd_status st = check_engine(e)) return st;
    if (num_segments < 0 || num_segments > FGD_MAX_SUBSET_SEGMENTS)
        return fail(FGD_ERR_INVALID_ARG, "num_segments %d is outside [0, %d]", num_segments, FGD_MAX_SUBSET_SEGMENTS);
    if (num_segments > 0 && !segments) return fail(FGD_ERR_INVALID_ARG, "segments is NULL");
    const int64_t P = e->cfg.num_params;
    int64_t prev_end = 0;
    for (int32_t i = 0; i < num_segments; ++i) {
        const int64_t b = segments[2 * i], en = segments[2 * i + 1];
        if (b < prev_end || en <= b || en > P)
            return fail(FGD_ERR_INVALID_ARG,
                        "segment %d [%lld, %lld) must be non-empty, inside [0, P) and after the previous one", i,
                        static_cast<long long>(b), static_cast<long long>(en));
        prev_end = en;
    }
    e->subset.assign(segments, segments + 2 * static_cast<size_t>(num_segments));
    ++e->topo_version;
    return FGD_OK;
}

fgd_status fgd_num_cd_rows(const fgd_engine *e, int32_t *n_rows) {
    if (fgd_status st = check_engine(e)) return st;
    if (!n_rows) return fail(FGD_ERR_INVALID_ARG, "n_rows is NULL");
    if (!e->slot_set[0] || !e->slot_set[1]) return fail(FGD_ERR_STATE, "both Mix slots must be set");
    *n_rows = n_cd_rows(e);
    return FGD_OK;
}

fgd_status fgd_get_effective_weights(const fgd_engine *e, int32_t which, int32_t round, float *out) {
    if (fgd_status st = check_engine(e)) return st;
    if (which != FGD_MIX1 && which != FGD_MIX2) return fail(FGD_ERR_INVALID_ARG, "which must be FGD_MIX1 or FGD_MIX2");
    if (!out) return fail(FGD_ERR_INVALID_ARG, "out is NULL");
    const fgd::MixTopology &t = e->slot[which - 1];
    if (!e->slot_set[which - 1]) return fail(FGD_ERR_STATE, "slot is not set");
    if (t.kind != 2) return fail(FGD_ERR_STATE, "slot is not a CSR topology");
    if (round < 0 || round >= t.rounds) return fail(FGD_ERR_INVALID_ARG, "round %d is outside [0, %d)", round, t.rounds);
    const size_t nnz = t.col_idx.size();
    std::memcpy(out, t.eff.data() + round * nnz, nnz * sizeof(float));
    return FGD_OK;
}

fgd_status fgd_effective_weights(int32_t num_workers, const int32_t *row_ptr, const int32_t *col_idx,
                                 const float *weights, const uint8_t *mask, int32_t reweight, float *out) {
    g_last_error.clear();
    if (reweight < 0 || reweight > 2) return fail(FGD_ERR_INVALID_ARG, "unknown reweighting %d", reweight);
    std::string err;
    return from_topo(fgd::effective_round_weights(num_workers, row_ptr, col_idx, weights, mask, reweight, out, err),
                     err);
}

fgd_status fgd_min_bytes_per_step(const fgd_engine *e, int64_t *bytes) {
    if (fgd_status st = check_engine(e)) return st;
    if (!bytes) return fail(FGD_ERR_INVALID_ARG, "bytes is NULL");
    *bytes = static_cast<int64_t>(e->cfg.num_workers) * e->cfg.num_params * (3 * elem_size(e->cfg.param_dtype) + 2 * 4);
    return FGD_OK;
}

fgd_status fgd_state_layout(const fgd_engine *e, int32_t spread, int32_t with_x, int64_t range_bytes,
                            int64_t *offsets, int64_t *total_bytes) {
    g_last_error.clear();
    if (fgd_status st = check_engine(e)) return st;
    if (!offsets || !total_bytes) return fail(FGD_ERR_INVALID_ARG, "offsets and total_bytes must not be NULL");
    if ((spread != 0 && spread != 1) || (with_x != 0 && with_x != 1))
        return fail(FGD_ERR_INVALID_ARG, "spread and with_x must be 0 or 1");
    constexpr int64_t kPage = int64_t{2} << 20;
    if (range_bytes < 0 || range_bytes % kPage != 0)
        return fail(FGD_ERR_INVALID_ARG, "range_bytes must be a non-negative multiple of 2 MiB");
    const fgd_config &c = e->cfg;
    // Every array is [M][ld]; the sizes below cannot overflow for any ld a
    // device can hold, but a corrupt ld is rejected rather than wrapped.
    if (c.ld > (int64_t{1} << 56) / c.num_workers) return fail(FGD_ERR_INVALID_ARG, "ld too large");
    auto up = [](int64_t b) { return (b + kPage - 1) / kPage * kPage; };
    const int64_t tb = up(c.num_workers * c.ld * elem_size(c.param_dtype));
    const int64_t vb = c.num_workers * c.ld * 4;
    int64_t end = 2 * tb;
    offsets[0] = 0;
    offsets[1] = tb;
    offsets[2] = with_x ? end : -1;
    if (with_x) end += tb;
    int64_t mom = end;
    if (spread) {
        int64_t range = range_bytes;
        if (range == 0) {
            if (e->host_only) return fail(FGD_ERR_STATE, "a host-only engine needs an explicit range_bytes");
            DeviceGuard dg;
            hipError_t err = dg.enter(c.device);
            size_t total = 0;
            if (err == hipSuccess) err = hipDeviceTotalMem(&total, c.device);
            if (err != hipSuccess) return hip_fail(err, "querying the device memory size");
            constexpr int64_t kGiB = int64_t{1} << 30;
            range = (static_cast<int64_t>(total / 3) + kGiB / 2) / kGiB * kGiB;
        }
        if (range >= end) mom = range;
        offsets[3] = mom;
        *total_bytes = mom + vb;
        // A buffer of up to 4/3 of a range is rounded up to exactly 4/3 of it
        // (128 GiB for 96 GiB ranges), a power of two the device allocator
        // hands out as one naturally aligned block that starts at 0 or at
        // 128 GiB of physical memory: in both cases offset 0 and the
        // momentum's offset lie in different ranges.
        const int64_t block = (range / 3 * 4 + kPage - 1) / kPage * kPage;
        if (mom == range && *total_bytes < block) *total_bytes = block;
        return FGD_OK;
    }
    offsets[3] = mom;
    *total_bytes = mom + vb;
    return FGD_OK;
}

fgd_status fgd_outer_step(fgd_engine *e, void *theta_prev, const void *theta_local, float *momentum,
                          double *cd_out, void *stream_handle) {
    g_last_error.clear();
    if (fgd_status st = check_engine(e)) return st;
    if (e->host_only) return fail(FGD_ERR_STATE, "host-only engine cannot run a step");
    if (!e->slot_set[0] || !e->slot_set[1]) return fail(FGD_ERR_STATE, "both Mix slots must be set before a step");
    const fgd_config &c = e->cfg;
    if (!theta_prev || !theta_local || !momentum) return fail(FGD_ERR_INVALID_ARG, "NULL device array");
    if (!aligned16(theta_prev) || !aligned16(theta_local) || !aligned16(momentum))
        return fail(FGD_ERR_INVALID_ARG, "device arrays must be 16-byte aligned");
    if (cd_out && (reinterpret_cast<uintptr_t>(cd_out) & 7u)) return fail(FGD_ERR_INVALID_ARG, "cd_out must be 8-byte aligned");
    const int es = elem_size(c.param_dtype);
    if (c.num_params > 0) {
        uintptr_t a0, a1, b0, b1, v0, v1;
        span(theta_prev, c.num_workers, c.ld, c.num_params, es, a0, a1);
        span(theta_local, c.num_workers, c.ld, c.num_params, es, b0, b1);
        span(momentum, c.num_workers, c.ld, c.num_params, 4, v0, v1);
        if (overlap(a0, a1, b0, b1) || overlap(b0, b1, v0, v1) || overlap(a0, a1, v0, v1))
            return fail(FGD_ERR_INVALID_ARG, "theta_prev, theta_local and momentum must not overlap");
    }
    hipStream_t stream = static_cast<hipStream_t>(stream_handle);
    if (!e->subset.empty() && e->slot[1].kind != 2)
        return fail(FGD_ERR_UNSUPPORTED, "a Mix2 subset needs a CSR Mix2");
    fgd::KernelSet ks;
    if (!lookup(c.num_workers, c.param_dtype, e->slot[0].kind, e->slot[1].kind, c.mix1_state != 0,
                !e->subset.empty(), ks))
        return fail(FGD_ERR_UNSUPPORTED, "no kernel for M=%d", c.num_workers);
    DeviceGuard dg;
    hipError_t herr = dg.enter(c.device);
    if (herr != hipSuccess) return hip_fail(herr, "selecting the engine's device");

    int ring = 0;
    if (fgd_status st = ensure_topology(e, stream, ring)) return st;

    fgd::StepParams p{};
    p.theta_prev = theta_prev;
    p.theta_out = theta_prev;
    p.theta_local = theta_local;
    p.mom = momentum;
    p.mom_out = momentum;
    p.P = c.num_params;
    p.ld = c.ld;
    p.ntiles = tiles_of(c.num_params, ks.v);
    p.M = c.num_workers;
    p.n_cd = n_cd_rows(e);
    p.lr = c.outer_lr;
    p.mu = c.momentum;
    p.nesterov = c.nesterov;
    const void *t1, *t2;
    const int64_t *seg;
    table_ptrs(e, ring, t1, t2, seg);
    p.mix1 = mix_dev(e->slot[0], t1);
    p.mix2 = mix_dev(e->slot[1], t2);
    p.n_seg = static_cast<int32_t>(e->subset.size() / 2);
    p.seg = seg;
    const bool tables = e->slot[0].kind == 2 || e->slot[1].kind == 2;
    const bool padded = (e->slot[0].kind == 2 && e->slot[0].padded) || (e->slot[1].kind == 2 && e->slot[1].padded);
    p.lds_rows = tables ? c.num_workers + (padded ? 1 : 0) : 0;
    size_t lds = static_cast<size_t>(p.lds_rows) * fgd::kBlock * ks.v * sizeof(float);
    if (cd_out) lds += static_cast<size_t>(p.n_cd) * fgd::kWavesPerBlock * ks.mmax * sizeof(double);

    // 64 workers on sparse tables: the worker-group kernel.
    fgd::WgKernel wk{};
    size_t wg_lds = 0;
    int wave_rows = 0;
    const bool wg = wg_step_fits(e, wk, wg_lds, wave_rows);
    fgd::WgParams wp{};
    const void *kernel = ks.step;
    void *args = &p;
    if (wg) {
        wp.theta_prev = theta_prev;
        wp.theta_out = theta_prev;
        wp.theta_local = theta_local;
        wp.mom = momentum;
        wp.mom_out = momentum;
        wp.P = c.num_params;
        wp.ld = c.ld;
        wp.ntiles = (c.num_params + fgd::kWgTile - 1) / fgd::kWgTile;
        wp.n_cd = p.n_cd;
        wp.wave_rows = wave_rows;
        wp.nesterov = c.nesterov;
        wp.lr = c.outer_lr;
        wp.mu = c.momentum;
        wp.rows_bytes = fgd::kWavesPerBlock * wave_rows * fgd::kWgRowBytes;
        const fgd::MixTopology &s1 = e->slot[0], &s2 = e->slot[1];
        wp.mix1 = fgd::WgMix{s1.kind, s1.rounds, s1.width, 0, static_cast<const int2 *>(t1)};
        wp.mix2 = fgd::WgMix{s2.kind, s2.rounds, s2.width, s1.kind == 2 ? s1.rounds * s1.width * fgd::kWgWorkers : 0,
                             static_cast<const int2 *>(t2)};
        kernel = wk.step;
        lds = wg_lds;
        args = &wp;
    }
    int grid = 0;
    if (fgd_status st = grid_for(e, kernel, lds, wg ? wp.ntiles : p.ntiles, grid, wg ? kMaxBlocksPerCu : ks.step_blocks_per_cu))
        return st;
    if (cd_out) {
        if (static_cast<size_t>(grid) * p.n_cd * c.num_workers > e->partials_capacity)
            return fail(FGD_ERR_UNSUPPORTED, "consensus scratch too small");
        p.cd_partials = e->d_partials;
        wp.cd_partials = e->d_partials;
    }

    const bool timed = e->timing && e->timed < kTimingPool;
    if (timed) {
        if (static_cast<int64_t>(e->ev_start.size()) <= e->timed) {
            hipEvent_t a, b;
            herr = hipEventCreate(&a);
            if (herr == hipSuccess) herr = hipEventCreate(&b);
            if (herr != hipSuccess) return hip_fail(herr, "creating timing events");
            e->ev_start.push_back(a);
            e->ev_stop.push_back(b);
        }
        herr = hipEventRecord(e->ev_start[e->timed], stream);
        if (herr != hipSuccess) return hip_fail(herr, "recording a timing event");
    }
    if (fgd_status st = launch(kernel, grid, lds, stream, args)) return st;
    if (timed) {
        herr = hipEventRecord(e->ev_stop[e->timed], stream);
        if (herr != hipSuccess) return hip_fail(herr, "recording a timing event");
        ++e->timed;
    }
    herr = hipEventRecord(e->topo_done[ring], stream);
    if (herr != hipSuccess) return hip_fail(herr, "recording the topology event");
    e->topo_pending[ring] = true;
    if (cd_out) return launch_finalize(e->d_partials, grid, p.n_cd * c.num_workers, cd_out, stream);
    return FGD_OK;
}

fgd_status fgd_step_variant(const fgd_engine *e, int32_t *variant) {
    if (fgd_status st = check_engine(e)) return st;
    if (!variant) return fail(FGD_ERR_INVALID_ARG, "variant is NULL");
    if (!e->slot_set[0] || !e->slot_set[1]) return fail(FGD_ERR_STATE, "both Mix slots must be set");
    fgd::WgKernel k{};
    size_t lds = 0;
    int rows = 0;
    *variant = wg_step_fits(e, k, lds, rows) ? FGD_STEP_WORKER_GROUPS : FGD_STEP_LANE_PER_PARAM;
    return FGD_OK;
}

fgd_status fgd_num_cd_rows_split(const fgd_engine *e, int32_t *mix1_rows, int32_t *blocking_rows) {
    if (fgd_status st = check_engine(e)) return st;
    if (!mix1_rows || !blocking_rows) return fail(FGD_ERR_INVALID_ARG, "NULL output");
    if (!e->slot_set[0] || !e->slot_set[1]) return fail(FGD_ERR_STATE, "both Mix slots must be set");
    *mix1_rows = e->slot[0].effective_rounds() + 1;
    *blocking_rows = e->slot[1].effective_rounds() + 2;
    return FGD_OK;
}

fgd_status fgd_min_bytes_split(const fgd_engine *e, int32_t write_local, int64_t *mix1_bytes,
                               int64_t *blocking_bytes) {
    if (fgd_status st = check_engine(e)) return st;
    if (!mix1_bytes || !blocking_bytes) return fail(FGD_ERR_INVALID_ARG, "NULL output");
    const int64_t n = static_cast<int64_t>(e->cfg.num_workers) * e->cfg.num_params;
    const int64_t ep = elem_size(e->cfg.param_dtype);
    *mix1_bytes = n * (2 * ep + (e->cfg.mix1_state ? 8 : 0));
    *blocking_bytes = n * (4 * ep + 8 + (write_local ? ep : 0));
    return FGD_OK;
}

fgd_status fgd_mix1(fgd_engine *e, const void *theta_prev, void *x_out, float *momentum, double *cd_out,
                    int32_t num_blocks, void *stream_handle) {
    g_last_error.clear();
    if (fgd_status st = check_engine(e)) return st;
    if (e->host_only) return fail(FGD_ERR_STATE, "host-only engine cannot run a step");
    if (!e->slot_set[0] || !e->slot_set[1]) return fail(FGD_ERR_STATE, "both Mix slots must be set before a step");
    const fgd_config &c = e->cfg;
    const int es = elem_size(c.param_dtype);
    if (bad_rows(theta_prev) || bad_rows(x_out))
        return fail(FGD_ERR_INVALID_ARG, "theta_prev and x_out must be non-NULL and 16-byte aligned");
    if (c.mix1_state && bad_rows(momentum))
        return fail(FGD_ERR_INVALID_ARG, "the state is mixed: momentum must be non-NULL and 16-byte aligned");
    if (cd_out && (reinterpret_cast<uintptr_t>(cd_out) & 7u)) return fail(FGD_ERR_INVALID_ARG, "cd_out must be 8-byte aligned");
    if (num_blocks < 0) return fail(FGD_ERR_INVALID_ARG, "num_blocks must be >= 0");
    if (rows_overlap(e, theta_prev, es, x_out, es) ||
        (c.mix1_state && (rows_overlap(e, momentum, 4, x_out, es) || rows_overlap(e, momentum, 4, theta_prev, es))))
        return fail(FGD_ERR_INVALID_ARG, "theta_prev, x_out and momentum must not overlap");
    hipStream_t stream = static_cast<hipStream_t>(stream_handle);
    fgd::SplitSet ks;
    if (!lookup_split(c.num_workers, c.param_dtype, e->slot[0].kind, e->slot[1].kind, false, c.mix1_state != 0, ks))
        return fail(FGD_ERR_UNSUPPORTED, "no kernel for M=%d", c.num_workers);
    DeviceGuard dg;
    hipError_t herr = dg.enter(c.device);
    if (herr != hipSuccess) return hip_fail(herr, "selecting the engine's device");
    int ring = 0;
    if (fgd_status st = ensure_topology(e, stream, ring)) return st;

    fgd::StepParams p{};
    fill_common(e, ring, ks.v, p);
    p.theta_prev = theta_prev;
    p.x_out = x_out;
    p.mom = momentum;
    p.mom_out = momentum;
    p.n_cd = e->slot[0].effective_rounds() + 1;
    p.lds_rows = lds_rows_for(e, true, false);
    size_t lds = static_cast<size_t>(p.lds_rows) * fgd::kBlock * ks.v * sizeof(float);
    if (cd_out) lds += static_cast<size_t>(p.n_cd) * fgd::kWavesPerBlock * ks.mmax * sizeof(double);
    int grid = 0;
    if (fgd_status st = grid_for(e, ks.mix1, lds, p.ntiles, grid, ks.blocks_per_cu)) return st;
    if (num_blocks > 0) grid = std::min(grid, num_blocks);
    p.chunk_tiles = std::max<int64_t>(1, (p.ntiles + kMix1Chunks - 1) / kMix1Chunks);
    p.nchunks = (p.ntiles + p.chunk_tiles - 1) / p.chunk_tiles;
    p.chunk_counter = e->d_counter;
    if (cd_out) p.cd_partials = e->d_chunk_partials;
    hipLaunchKernelGGL(fgd::counter_reset_kernel, dim3(1), dim3(64), 0, stream, e->d_counter);
    herr = hipGetLastError();
    if (herr != hipSuccess) return hip_fail(herr, "counter reset launch");
    if (fgd_status st = launch(ks.mix1, grid, lds, stream, &p)) return st;
    herr = hipEventRecord(e->topo_done[ring], stream);
    if (herr != hipSuccess) return hip_fail(herr, "recording the topology event");
    e->topo_pending[ring] = true;
    if (cd_out) return launch_finalize(e->d_chunk_partials, static_cast<int>(p.nchunks), p.n_cd * c.num_workers,
                                       cd_out, stream);
    return FGD_OK;
}

fgd_status fgd_outer_step_blocking(fgd_engine *e, const void *x, void *theta_prev, void *theta_local, float *momentum,
                                   double *cd_out, int32_t write_local, void *stream_handle) {
    g_last_error.clear();
    if (fgd_status st = check_engine(e)) return st;
    if (e->host_only) return fail(FGD_ERR_STATE, "host-only engine cannot run a step");
    if (!e->slot_set[0] || !e->slot_set[1]) return fail(FGD_ERR_STATE, "both Mix slots must be set before a step");
    const fgd_config &c = e->cfg;
    const int es = elem_size(c.param_dtype);
    if (write_local != 0 && write_local != 1) return fail(FGD_ERR_INVALID_ARG, "write_local must be 0 or 1");
    if (bad_rows(x) || bad_rows(theta_prev) || bad_rows(theta_local) || bad_rows(momentum))
        return fail(FGD_ERR_INVALID_ARG, "device arrays must be non-NULL and 16-byte aligned");
    if (cd_out && (reinterpret_cast<uintptr_t>(cd_out) & 7u)) return fail(FGD_ERR_INVALID_ARG, "cd_out must be 8-byte aligned");
    if (rows_overlap(e, x, es, theta_prev, es) || rows_overlap(e, x, es, theta_local, es) ||
        rows_overlap(e, x, es, momentum, 4) || rows_overlap(e, theta_prev, es, theta_local, es) ||
        rows_overlap(e, theta_prev, es, momentum, 4) || rows_overlap(e, theta_local, es, momentum, 4))
        return fail(FGD_ERR_INVALID_ARG, "x, theta_prev, theta_local and momentum must not overlap");
    if (!e->subset.empty() && e->slot[1].kind != 2) return fail(FGD_ERR_UNSUPPORTED, "a Mix2 subset needs a CSR Mix2");
    hipStream_t stream = static_cast<hipStream_t>(stream_handle);
    fgd::SplitSet ks;
    if (!lookup_split(c.num_workers, c.param_dtype, e->slot[0].kind, e->slot[1].kind, !e->subset.empty(), false, ks))
        return fail(FGD_ERR_UNSUPPORTED, "no kernel for M=%d", c.num_workers);
    DeviceGuard dg;
    hipError_t herr = dg.enter(c.device);
    if (herr != hipSuccess) return hip_fail(herr, "selecting the engine's device");
    int ring = 0;
    if (fgd_status st = ensure_topology(e, stream, ring)) return st;

    fgd::StepParams p{};
    fill_common(e, ring, ks.v, p);
    p.theta_prev = theta_prev;
    p.theta_out = theta_prev;
    p.theta_local = theta_local;
    p.mom = momentum;
    p.mom_out = momentum;
    p.x = x;
    p.local_out = write_local ? theta_local : nullptr;
    p.n_cd = e->slot[1].effective_rounds() + 2;
    p.lds_rows = lds_rows_for(e, false, true);
    size_t lds = static_cast<size_t>(p.lds_rows) * fgd::kBlock * ks.v * sizeof(float);
    if (cd_out) lds += static_cast<size_t>(p.n_cd) * fgd::kWavesPerBlock * ks.mmax * sizeof(double);
    int grid = 0;
    if (fgd_status st = grid_for(e, ks.blocking, lds, p.ntiles, grid, ks.blocks_per_cu)) return st;
    if (cd_out) {
        if (static_cast<size_t>(grid) * p.n_cd * c.num_workers > e->partials_capacity)
            return fail(FGD_ERR_UNSUPPORTED, "consensus scratch too small");
        p.cd_partials = e->d_partials;
    }
    if (fgd_status st = launch(ks.blocking, grid, lds, stream, &p)) return st;
    herr = hipEventRecord(e->topo_done[ring], stream);
    if (herr != hipSuccess) return hip_fail(herr, "recording the topology event");
    e->topo_pending[ring] = true;
    if (cd_out) return launch_finalize(e->d_partials, grid, p.n_cd * c.num_workers, cd_out, stream);
    return FGD_OK;
}

fgd_status fgd_consensus_distance(fgd_engine *e, const void *x, int32_t dtype, double *out, void *stream_handle) {
    g_last_error.clear();
    if (fgd_status st = check_engine(e)) return st;
    if (e->host_only) return fail(FGD_ERR_STATE, "host-only engine cannot run a kernel");
    if (!x || !out) return fail(FGD_ERR_INVALID_ARG, "NULL device array");
    if (dtype != FGD_F32 && dtype != FGD_BF16) return fail(FGD_ERR_INVALID_ARG, "unknown dtype %d", dtype);
    const fgd_config &c = e->cfg;
    if (!aligned16(x)) return fail(FGD_ERR_INVALID_ARG, "x must be 16-byte aligned");
    if ((c.ld * elem_size(dtype)) % 16 != 0) return fail(FGD_ERR_INVALID_ARG, "ld * elem_size must be a multiple of 16");
    if (reinterpret_cast<uintptr_t>(out) & 7u) return fail(FGD_ERR_INVALID_ARG, "out must be 8-byte aligned");
    fgd::KernelSet ks;
    if (!lookup(c.num_workers, dtype, 0, 0, false, false, ks)) return fail(FGD_ERR_UNSUPPORTED, "no kernel for M=%d", c.num_workers);
    DeviceGuard dg;
    hipError_t herr = dg.enter(c.device);
    if (herr != hipSuccess) return hip_fail(herr, "selecting the engine's device");
    hipStream_t stream = static_cast<hipStream_t>(stream_handle);
    fgd::ConsensusParams p{};
    p.x = x;
    p.P = c.num_params;
    p.ld = c.ld;
    p.ntiles = tiles_of(c.num_params, ks.v);
    p.M = c.num_workers;
    p.partials = e->d_partials;
    int grid = 0;
    if (fgd_status st = grid_for(e, ks.consensus, 0, p.ntiles, grid, consensus_blocks_per_cu(c.num_workers)))
        return st;
    if (static_cast<size_t>(grid) * c.num_workers > e->partials_capacity)
        return fail(FGD_ERR_UNSUPPORTED, "consensus scratch too small");
    if (fgd_status st = launch(ks.consensus, grid, 0, stream, &p)) return st;
    return launch_finalize(e->d_partials, grid, c.num_workers, out, stream);
}

fgd_status fgd_consensus_distance_noalloc(int32_t num_workers, int64_t num_params, int64_t ld, int32_t dtype,
                                          const void *x, double *out, void *stream_handle) {
    g_last_error.clear();
    if (num_workers < 1 || num_workers > FGD_MAX_WORKERS)
        return fail(FGD_ERR_INVALID_ARG, "num_workers %d is outside [1, %d] (the static scratch holds %d blocks of %d)",
                    num_workers, FGD_MAX_WORKERS, kNoAllocBlocks, FGD_MAX_WORKERS);
    if (num_params < 0 || ld < num_params) return fail(FGD_ERR_INVALID_ARG, "need 0 <= num_params <= ld");
    if (dtype != FGD_F32 && dtype != FGD_BF16) return fail(FGD_ERR_INVALID_ARG, "unknown dtype %d", dtype);
    if (!x || !out) return fail(FGD_ERR_INVALID_ARG, "NULL device array");
    if (!aligned16(x)) return fail(FGD_ERR_INVALID_ARG, "x must be 16-byte aligned");
    if ((ld * elem_size(dtype)) % 16 != 0) return fail(FGD_ERR_INVALID_ARG, "ld * elem_size must be a multiple of 16");
    if (reinterpret_cast<uintptr_t>(out) & 7u) return fail(FGD_ERR_INVALID_ARG, "out must be 8-byte aligned");
    fgd::KernelSet ks;
    if (!lookup(num_workers, dtype, 0, 0, false, false, ks)) return fail(FGD_ERR_UNSUPPORTED, "no kernel for M=%d", num_workers);
    int dev = 0;
    hipError_t herr = hipGetDevice(&dev);
    if (herr != hipSuccess) return hip_fail(herr, "querying the current device");
    double *partials = nullptr;
    int num_cus = 0;
    if (fgd_status st = noalloc_device(dev, partials, num_cus)) return st;
    fgd::ConsensusParams p{};
    p.x = x;
    p.P = num_params;
    p.ld = ld;
    p.ntiles = tiles_of(num_params, ks.v);
    p.M = num_workers;
    p.partials = partials;
    int grid = 0;
    if (fgd_status st = grid_for_cus(num_cus, ks.consensus, 0, p.ntiles, grid, consensus_blocks_per_cu(num_workers)))
        return st;
    // The grid of fgd_consensus_distance (so the same sums in the same
    // order), capped to the blocks the scratch holds on a larger device.
    grid = std::min(grid, kNoAllocDoubles / num_workers);
    hipStream_t stream = static_cast<hipStream_t>(stream_handle);
    if (fgd_status st = launch(ks.consensus, grid, 0, stream, &p)) return st;
    return launch_finalize(partials, grid, num_workers, out, stream);
}

fgd_status fgd_enable_timing(fgd_engine *e, int32_t enable) {
    if (fgd_status st = check_engine(e)) return st;
    e->timing = enable != 0;
    e->timed = 0;
    return FGD_OK;
}

fgd_status fgd_read_timing(fgd_engine *e, double *total_ms, int64_t *count) {
    if (fgd_status st = check_engine(e)) return st;
    if (!total_ms || !count) return fail(FGD_ERR_INVALID_ARG, "NULL output");
    double sum = 0.0;
    for (int64_t i = 0; i < e->timed; ++i) {
        hipError_t err = hipEventSynchronize(e->ev_stop[i]);
        if (err != hipSuccess) return hip_fail(err, "waiting for a timing event");
        float ms = 0.0f;
        err = hipEventElapsedTime(&ms, e->ev_start[i], e->ev_stop[i]);
        if (err != hipSuccess) return hip_fail(err, "reading a timing event");
        sum += ms;
    }
    *total_ms = sum;
    *count = e->timed;
    return FGD_OK;
}

fgd_status fgd_stream_step_pattern(fgd_engine *e, void *theta_prev, const void *theta_local, float *momentum,
                                   void *stream_handle) {
    g_last_error.clear();
    if (fgd_status st = check_engine(e)) return st;
    if (e->host_only) return fail(FGD_ERR_STATE, "host-only engine cannot run a kernel");
    const fgd_config &c = e->cfg;
    if (!theta_prev || !theta_local || !momentum) return fail(FGD_ERR_INVALID_ARG, "NULL device array");
    if (!aligned16(theta_prev) || !aligned16(theta_local) || !aligned16(momentum))
        return fail(FGD_ERR_INVALID_ARG, "device arrays must be 16-byte aligned");
    const int es = elem_size(c.param_dtype);
    if (rows_overlap(e, theta_prev, es, theta_local, es) || rows_overlap(e, theta_prev, es, momentum, 4) ||
        rows_overlap(e, theta_local, es, momentum, 4))
        return fail(FGD_ERR_INVALID_ARG, "theta_prev, theta_local and momentum must not overlap");
    const void *kernel = nullptr;
    int v = 0, bpc = 0;
    // The worker-group step's own layout when the current topology selects it.
    fgd::WgKernel wk{};
    size_t wg_lds = 0;
    int wave_rows = 0;
    const bool wg = e->slot_set[0] && e->slot_set[1] && wg_step_fits(e, wk, wg_lds, wave_rows);
    if (!wg && !fgd::pattern_kernel_for(c.num_workers, c.param_dtype == FGD_BF16, &kernel, &v, &bpc))
        return fail(FGD_ERR_UNSUPPORTED, "the pattern reference runs for M in {1, 2, 4, 8, 16, 32, 64}");
    if (c.num_params == 0) return FGD_OK;
    DeviceGuard dg;
    hipError_t herr = dg.enter(c.device);
    if (herr != hipSuccess) return hip_fail(herr, "selecting the engine's device");
    fgd::PatternParams p{};
    p.theta_prev = theta_prev;
    p.theta_out = theta_prev;
    p.theta_local = theta_local;
    p.mom = momentum;
    p.mom_out = momentum;
    p.P = c.num_params;
    p.ld = c.ld;
    p.mask = 0;
    int grid = 0;
    if (wg) {  // the step's grid: its occupancy with its LDS
        p.ntiles = (c.num_params + fgd::kWgTile - 1) / fgd::kWgTile;
        if (fgd_status st = grid_for(e, wk.step, wg_lds, p.ntiles, grid)) return st;
        return launch(wk.pattern, grid, 0, static_cast<hipStream_t>(stream_handle), &p);
    }
    p.ntiles = tiles_of(c.num_params, v);
    if (fgd_status st = grid_for(e, kernel, 0, p.ntiles, grid, bpc)) return st;
    return launch(kernel, grid, 0, static_cast<hipStream_t>(stream_handle), &p);
}

fgd_status fgd_stream_copy(void *dst, const void *src, int64_t bytes, void *stream_handle) {
    g_last_error.clear();
    if (!dst || !src || bytes < 0 || bytes % 16 != 0 || !aligned16(dst) || !aligned16(src))
        return fail(FGD_ERR_INVALID_ARG, "copy needs 16-byte aligned pointers and a size multiple of 16");
    if (bytes == 0) return FGD_OK;
    const int64_t n = bytes / 16;
    int dev = 0, cus = 0;
    hipError_t err = hipGetDevice(&dev);
    if (err == hipSuccess) err = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (err != hipSuccess) return hip_fail(err, "device query");
    const int64_t blocks = std::min<int64_t>((n + 1023) / 1024, static_cast<int64_t>(cus) * 8);
    hipLaunchKernelGGL(fgd::copy_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0,
                       static_cast<hipStream_t>(stream_handle), static_cast<const fgd::u32x4 *>(src),
                       static_cast<fgd::u32x4 *>(dst), n);
    err = hipGetLastError();
    if (err != hipSuccess) return hip_fail(err, "copy launch");
    return FGD_OK;
}

}  // extern "C"
