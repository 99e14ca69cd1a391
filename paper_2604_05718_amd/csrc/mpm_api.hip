// C ABI of the MPM library: argument validation (pure host code, run before
// anything touches the GPU), workspace carving and kernel launches.
#include <hip/hip_runtime.h>

#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include <atomic>
#include <mutex>


#include "../../include/mpm.h"
#include "mpm_launch.h"

namespace {

thread_local int g_last_hip_error = 0;

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

int hip_status(hipError_t e)
{
    if (e == hipSuccess) return MPM_OK;
    g_last_hip_error = static_cast<int>(e);
    return MPM_ERR_HIP;
}

// Fault injection for testing callers' error paths without a GPU: with the
// environment variable MPM_FAULT_INJECT=launch (read once, at the first call), every
// entry point that would launch a kernel returns MPM_ERR_HIP with
// hipErrorLaunchFailure recorded, after its argument checks and before any HIP call.
bool inject_launch_failure()
{
    static const bool on = [] {
        const char* v = getenv("MPM_FAULT_INJECT");
        return v != nullptr && strcmp(v, "launch") == 0;
    }();
    return on;
}

int injected_failure() { return hip_status(hipErrorLaunchFailure); }

#define MPM_LAUNCH_GATE()                                          \
    do {                                                           \
        if (inject_launch_failure()) return injected_failure();    \
    } while (0)

// Checked mode: with MPM_CHECKED=1 in the environment (read once, at the first call),
// every entry point validates the data-dependent preconditions it would otherwise take
// on trust, on the device, before launching its operation: packed offsets first (their
// verdict read back), then the values the operation indexes with. A failure returns
// MPM_ERR_INVALID_ARG with nothing of the operation launched. The verdict is one device
// word per GPU (a file-scope array: its address is looked up once per device, as for
// the allocation-free entry point's array); checked calls synchronise their stream and
// are serialised by a lock.
bool checked_mode()
{
    static const bool on = [] {
        const char* v = getenv("MPM_CHECKED");
        return v != nullptr && strcmp(v, "1") == 0;
    }();
    return on;
}

static __device__ __align__(16) int32_t check_verdict[4];

constexpr int kMaxCheckDevices = 64;
std::atomic<int32_t*> g_verdict_ptr[kMaxCheckDevices];
std::mutex g_check_mutex;  // held across a checked call's validation (one verdict word per GPU)

// Runs `launch_checks(verdict)` on `st` after clearing the verdict, reads it back and
// returns MPM_OK, MPM_ERR_INVALID_ARG or MPM_ERR_HIP. Called with g_check_mutex held.
template <class F>
int run_checks(hipStream_t st, F&& launch_checks)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_status(e);
    if (dev < 0 || dev >= kMaxCheckDevices) return hip_status(hipErrorInvalidDevice);
    int32_t* v = g_verdict_ptr[dev].load(std::memory_order_acquire);
    if (v == nullptr) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(check_verdict));
        if (e != hipSuccess) return hip_status(e);
        if (p == nullptr) return hip_status(hipErrorInvalidSymbol);
        v = static_cast<int32_t*>(p);
        g_verdict_ptr[dev].store(v, std::memory_order_release);
    }
    e = mpm::launch_zero_words(v, 1, st);
    if (e == hipSuccess) e = launch_checks(v);
    int32_t host = 0;
    if (e == hipSuccess) e = hipMemcpyAsync(&host, v, sizeof host, hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e != hipSuccess) return hip_status(e);
    return host == 0 ? MPM_OK : MPM_ERR_INVALID_ARG;
}

// Packed offsets of the rows of x (0 <= n_b <= N), then the rows themselves (finite),
// their given inverse norms (finite, positive) and grid positions (in range, rows
// non-decreasing), each where given.
int checked_rows(const void* x, const int32_t* x_off, const float* x_inv, const int32_t* pos, int grid_w, int32_t B,
                 int32_t N, int32_t D, int32_t dt, hipStream_t st)
{
    std::lock_guard<std::mutex> lock(g_check_mutex);
    int s = MPM_OK;
    if (x_off)
        s = run_checks(st, [&](int32_t* v) { return mpm::launch_check_offsets(x_off, B, N, 0, -1, nullptr, v, st); });
    if (s != MPM_OK) return s;
    return run_checks(st, [&](int32_t* v) {
        hipError_t e = mpm::launch_check_finite(x, x_off, B, N, D, dt, v, st);
        if (e == hipSuccess && x_inv) e = mpm::launch_check_inv(x_inv, x_off, B, N, v, st);
        if (e == hipSuccess && pos)
            e = mpm::launch_check_pos(pos, x_off, B, N, grid_w, (long)grid_w * MPM_MAX_N, v, st);
        return e;
    });
}

// Offsets (where given: x_off for the tokens, y_off for the merged rows, at most n_b of
// them and within the B*N rows of y), then the slot arrays: neighbours (nb), or the
// merged rows' sources (src, two per merged row, each below n_b).
int checked_pairs(const int32_t* x_off, const int32_t* nb, const int32_t* y_off, const int32_t* src, int32_t B,
                  int32_t N, hipStream_t st)
{
    std::lock_guard<std::mutex> lock(g_check_mutex);
    int s = run_checks(st, [&](int32_t* v) {
        hipError_t e = hipSuccess;
        if (x_off) e = mpm::launch_check_offsets(x_off, B, N, 0, -1, nullptr, v, st);
        if (e == hipSuccess && y_off) e = mpm::launch_check_offsets(y_off, B, N, 0, (long)B * N, x_off, v, st);
        return e;
    });
    if (s != MPM_OK) return s;
    return run_checks(st, [&](int32_t* v) {
        if (nb) return mpm::launch_check_nb(nb, x_off, B, N, v, st);
        return mpm::launch_check_slots(src, 2, y_off, 0, x_off, B, N, mpm::kCheckValues, v, st);
    });
}

// Offsets of the merged rows z (where given; at most rows_max rows per image), then
// maps: map_a in [-1, N) (it indexes map_b's slots, or z's rows when map_b is null) and
// map_b in [-1, n_z).
int checked_maps(const int32_t* z_off, int32_t rows_max, const int32_t* map_a, const int32_t* map_b, int32_t B,
                 int32_t N, hipStream_t st)
{
    std::lock_guard<std::mutex> lock(g_check_mutex);
    int s = MPM_OK;
    if (z_off)
        s = run_checks(st, [&](int32_t* v) { return mpm::launch_check_offsets(z_off, B, rows_max, 0, -1, nullptr, v, st); });
    if (s != MPM_OK || map_a == nullptr) return s;
    return run_checks(st, [&](int32_t* v) {
        hipError_t e = mpm::launch_check_slots(map_a, 1, nullptr, -1, map_b ? nullptr : z_off, B, N,
                                               mpm::kCheckValues, v, st);
        if (e == hipSuccess && map_b)
            e = mpm::launch_check_slots(map_b, 1, nullptr, -1, z_off, B, N, mpm::kCheckValues, v, st);
        return e;
    });
}

#define MPM_DATA_CHECK(expr)                                       \
    do {                                                           \
        if (checked_mode()) {                                      \
            const int mpm_checked_status_ = (expr);                \
            if (mpm_checked_status_ != MPM_OK) return mpm_checked_status_; \
        }                                                          \
    } while (0)

int check_shape(int32_t B, int32_t N)
{
    if (B < 1 || N < 1) return MPM_ERR_INVALID_ARG;
    if (B > MPM_MAX_B || N > MPM_MAX_N) return MPM_ERR_UNSUPPORTED;
    return MPM_OK;
}

int check_rows(int32_t B, int32_t N, int32_t D, int32_t dt)
{
    const int s = check_shape(B, N);
    if (s != MPM_OK) return s;
    if (dt != MPM_F32 && dt != MPM_BF16) return MPM_ERR_INVALID_ARG;
    if (D < 1) return MPM_ERR_INVALID_ARG;
    if (D % (dt == MPM_BF16 ? 8 : 4) != 0) return MPM_ERR_INVALID_ARG;  // 16-byte rows
    if (D > MPM_MAX_D) return MPM_ERR_UNSUPPORTED;
    return MPM_OK;
}

bool ok_rows_ptr(const void* p) { return p != nullptr && aligned(p, 16); }
bool ok_int_ptr(const void* p) { return p != nullptr && aligned(p, 4); }
bool ok_opt_int_ptr(const void* p) { return p == nullptr || aligned(p, 4); }

constexpr size_t kAlign = 256;
size_t round_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

// The sync region: one arrival counter per image plus the images-done counter, at
// the start of every workspace and of the same size for every shape.
constexpr size_t kSyncWords = (size_t)MPM_MAX_B + 1;

struct Workspace {
    int32_t* sync;
    int32_t* nb;
    int32_t* src;
    float* pv;
    int32_t* pi;
};

struct Offsets {
    size_t sync, nb, src, pv, pi, total;
};

Offsets workspace_offsets(int32_t B, int32_t N)
{
    const size_t slots = (size_t)B * (size_t)N;
    const size_t partial = slots * (size_t)mpm::partial_tiles(N);
    Offsets o;
    o.sync = 0;
    o.nb = o.sync + round_up(kSyncWords * sizeof(int32_t));
    o.src = o.nb + round_up(slots * sizeof(int32_t));
    o.pv = o.src + round_up(2 * slots * sizeof(int32_t));
    o.pi = o.pv + round_up(partial * sizeof(float));
    o.total = o.pi + round_up(partial * sizeof(int32_t));
    return o;
}

// Checks and carves the workspace; returns MPM_OK or an error status.
int carve(void* ws, size_t ws_bytes, int32_t B, int32_t N, Workspace* w)
{
    if (ws == nullptr || !aligned(ws, kAlign)) return MPM_ERR_INVALID_ARG;
    const Offsets o = workspace_offsets(B, N);
    if (ws_bytes < o.total) return MPM_ERR_WORKSPACE;
    char* p = static_cast<char*>(ws);
    w->sync = reinterpret_cast<int32_t*>(p + o.sync);
    w->nb = reinterpret_cast<int32_t*>(p + o.nb);
    w->src = reinterpret_cast<int32_t*>(p + o.src);
    w->pv = reinterpret_cast<float*>(p + o.pv);
    w->pi = reinterpret_cast<int32_t*>(p + o.pi);
    return MPM_OK;
}

hipStream_t as_stream(void* s) { return static_cast<hipStream_t>(s); }

// Shared checks of the affinity entry points.
int check_affinity(const void* x, const int32_t* x_off, const float* x_inv, int32_t B, int32_t N, int32_t D,
                   int32_t dt, int32_t schedule)
{
    const int s = check_rows(B, N, D, dt);
    if (s != MPM_OK) return s;
    if (!mpm::valid_schedule(schedule)) return MPM_ERR_INVALID_ARG;
    if (!ok_rows_ptr(x) || !ok_opt_int_ptr(x_off) || !ok_opt_int_ptr(x_inv)) return MPM_ERR_INVALID_ARG;
    if (x_inv && !mpm::affinity_takes_norms(D, dt)) return MPM_ERR_UNSUPPORTED;
    return MPM_OK;
}

// nb from the affinity partials, then mutual pairs, compact ids and offsets. With few
// candidate tiles the compaction kernel (one workgroup per image) reduces the
// partials itself; with more, that serial reduction dominates, so a fully
// parallel reduction writes nb first and the compaction reads it. A batch of a
// few images (as small as the 64 x 64 block schedule is for) leaves most of
// the device idle either way, and one launch fewer wins up to 16 tiles.
constexpr int kFusedReduceMaxTiles = 4;
constexpr int kFusedReduceMaxTilesFewImages = 16;
constexpr int kFewImages = 8;

// Compaction from partials of ct candidate rows each (reduced first by their own launch
// when an image has more tiles than the compaction reduces well itself).
hipError_t compact_partials_ct(const Workspace& w, const int32_t* x_off, int32_t B, int32_t N, int32_t D, int32_t dt,
                               int ct, int32_t* map, int32_t* y_off, hipStream_t st)
{
    const int T = mpm::partial_tiles(N);
    const int fused_max = B <= kFewImages ? kFusedReduceMaxTilesFewImages : kFusedReduceMaxTiles;
    if ((N + ct - 1) / ct <= fused_max)
        return mpm::launch_pair_compact_partials(w.pv, w.pi, T, ct, w.nb, x_off, B, N, map, w.src, y_off, w.sync, st);
    hipError_t e = mpm::launch_reduce_partials(w.pv, w.pi, ct, nullptr, x_off, B, N, D, dt, w.nb, nullptr, st);
    if (e == hipSuccess) e = mpm::launch_pair_compact(w.nb, x_off, B, N, map, w.src, y_off, w.sync, st);
    return e;
}

hipError_t compact_from_partials(const Workspace& w, const int32_t* x_off, int32_t B, int32_t N, int32_t D,
                                 int32_t dt, int32_t schedule, int32_t* map, int32_t* y_off, hipStream_t st)
{
    return compact_partials_ct(w, x_off, B, N, D, dt, mpm::partial_tile_width(B, D, dt, N, schedule), map, y_off, st);
}

// One insertion's affinity (events bound to its launches) and compaction into the carved workspace.
hipError_t affinity_compact(const void* x, const int32_t* x_off, const float* x_inv, int32_t B, int32_t N,
                            int32_t D, int32_t dt, int32_t schedule, int32_t* map, int32_t* y_off,
                            const Workspace& w, hipEvent_t start, hipEvent_t stop, hipStream_t st)
{
    hipError_t e = mpm::launch_affinity(x, x_off, B, N, D, dt, schedule, w.pv, w.pi, st, start, stop, x_inv);
    if (e == hipSuccess) e = compact_from_partials(w, x_off, B, N, D, dt, schedule, map, y_off, st);
    return e;
}

// ---- workspace of the allocation-free entry point --------------------------------
// A file-scope device array: each GPU the library runs on holds its own copy (at its
// own address) until the process ends. In host code `scratch` names a host-side
// stand-in, not device memory: its device address is looked up once per device with
// hipGetSymbolAddress and only that address is ever passed to kernels or copies.
constexpr size_t kScratchBytes = MPM_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch_ptr[kMaxDevices];  // device address of `scratch`, per device (set once)
std::mutex g_scratch_mutex;

// The device address of `scratch` on the current device. On the first call for a
// device (with that device current) it is looked up, and the array's sync region is
// cleared by a fill kernel on `st` (no memset node, so a first call under graph
// capture records a kernel).
hipError_t scratch_for_current_device(hipStream_t st, void** out)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
    if (p == nullptr) {
        std::lock_guard<std::mutex> lock(g_scratch_mutex);
        p = g_scratch_ptr[dev].load(std::memory_order_acquire);
        if (p == nullptr) {
            e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
            if (e != hipSuccess) return e;
            if (p == nullptr) return hipErrorInvalidSymbol;
            e = mpm::launch_zero_words(static_cast<int32_t*>(p), (long)kSyncWords, st);
            if (e != hipSuccess) return e;
            g_scratch_ptr[dev].store(p, std::memory_order_release);
        }
    }
    *out = p;
    return hipSuccess;
}

}  // namespace

extern "C" {

const char* mpm_version(void) { return "mpm 0.2.0 gfx950"; }

const char* mpm_status_string(int status)
{
    switch (status) {
    case MPM_OK: return "MPM_OK";
    case MPM_ERR_INVALID_ARG: return "MPM_ERR_INVALID_ARG";
    case MPM_ERR_UNSUPPORTED: return "MPM_ERR_UNSUPPORTED";
    case MPM_ERR_WORKSPACE: return "MPM_ERR_WORKSPACE";
    case MPM_ERR_HIP: return "MPM_ERR_HIP";
    default: return "MPM_UNKNOWN_STATUS";
    }
}

int mpm_last_hip_error(void) { return g_last_hip_error; }

size_t mpm_workspace_bytes(int32_t B, int32_t N)
{
    if (B < 1 || N < 1) return 0;
    return workspace_offsets(B, N).total;
}

int mpm_workspace_offsets(int32_t B, int32_t N, size_t* sync, size_t* nb, size_t* src, size_t* pv, size_t* pi)
{
    if (B < 1 || N < 1) return MPM_ERR_INVALID_ARG;
    const Offsets o = workspace_offsets(B, N);
    if (sync) *sync = o.sync;
    if (nb) *nb = o.nb;
    if (src) *src = o.src;
    if (pv) *pv = o.pv;
    if (pi) *pi = o.pi;
    return MPM_OK;
}

int mpm_workspace_init(void* ws, size_t ws_bytes, void* stream)
{
    if (ws == nullptr || !aligned(ws, kAlign)) return MPM_ERR_INVALID_ARG;
    if (ws_bytes < kSyncWords * sizeof(int32_t)) return MPM_ERR_WORKSPACE;
    MPM_LAUNCH_GATE();
    return hip_status(mpm::launch_zero_words(static_cast<int32_t*>(ws), (long)kSyncWords, as_stream(stream)));
}

int mpm_affinity(const void* x, const int32_t* x_off, const float* x_inv, int32_t B, int32_t N, int32_t D, int32_t dt,
                 int32_t schedule, void* ws, size_t ws_bytes, void* start_event, void* stop_event, void* stream)
{
    int s = check_affinity(x, x_off, x_inv, B, N, D, dt, schedule);
    if (s != MPM_OK) return s;
    Workspace w;
    if ((s = carve(ws, ws_bytes, B, N, &w)) != MPM_OK) return s;
    MPM_LAUNCH_GATE();
    MPM_DATA_CHECK(checked_rows(x, x_off, x_inv, nullptr, 1, B, N, D, dt, as_stream(stream)));
    return hip_status(mpm::launch_affinity(x, x_off, B, N, D, dt, schedule, w.pv, w.pi, as_stream(stream),
                                           static_cast<hipEvent_t>(start_event), static_cast<hipEvent_t>(stop_event),
                                           x_inv));
}

int mpm_affinity_compact(const void* x, const int32_t* x_off, const float* x_inv, int32_t B, int32_t N, int32_t D,
                         int32_t dt, int32_t schedule, int32_t* map, int32_t* y_off, void* ws, size_t ws_bytes,
                         void* start_event, void* stop_event, void* stream)
{
    int s = check_affinity(x, x_off, x_inv, B, N, D, dt, schedule);
    if (s != MPM_OK) return s;
    if (!ok_int_ptr(map) || !ok_int_ptr(y_off)) return MPM_ERR_INVALID_ARG;
    Workspace w;
    if ((s = carve(ws, ws_bytes, B, N, &w)) != MPM_OK) return s;
    MPM_LAUNCH_GATE();
    MPM_DATA_CHECK(checked_rows(x, x_off, x_inv, nullptr, 1, B, N, D, dt, as_stream(stream)));
    return hip_status(affinity_compact(x, x_off, x_inv, B, N, D, dt, schedule, map, y_off, w,
                                       static_cast<hipEvent_t>(start_event), static_cast<hipEvent_t>(stop_event),
                                       as_stream(stream)));
}

int mpm_affinity_schedule_used(int32_t B, int32_t N, int32_t D, int32_t dt, int32_t schedule, int32_t* used)
{
    const int s = check_rows(B, N, D, dt);
    if (s != MPM_OK) return s;
    if (!used || !mpm::valid_schedule(schedule)) return MPM_ERR_INVALID_ARG;
    int sc = 0;
    const int st = hip_status(mpm::affinity_schedule(B, N, D, dt, schedule, &sc));
    if (st == MPM_OK) *used = sc;
    return st;
}

int mpm_local_block_rows(int32_t B, int32_t N, int32_t D, int32_t dt, int32_t grid_w, int32_t window,
                         int32_t block_rows, int32_t* rows)
{
    const int s = check_rows(B, N, D, dt);
    if (s != MPM_OK) return s;
    if (!rows || grid_w < 1 || grid_w > MPM_MAX_N || window < 0 || !mpm::valid_local_block_rows(block_rows))
        return MPM_ERR_INVALID_ARG;
    int dev = 0;
    const int st = hip_status(hipGetDevice(&dev));
    if (st == MPM_OK) *rows = mpm::local_block_rows(B, N, D, dt, grid_w, window, block_rows);
    return st;
}

int mpm_argmax(const void* x, const int32_t* x_off, int32_t B, int32_t N, int32_t D, int32_t dt, int32_t schedule,
               int32_t* nb, float* best, void* ws, size_t ws_bytes, void* stream)
{
    int s = check_affinity(x, x_off, nullptr, B, N, D, dt, schedule);
    if (s != MPM_OK) return s;
    if (!ok_int_ptr(nb) || !ok_opt_int_ptr(best)) return MPM_ERR_INVALID_ARG;
    Workspace w;
    if ((s = carve(ws, ws_bytes, B, N, &w)) != MPM_OK) return s;
    MPM_LAUNCH_GATE();
    MPM_DATA_CHECK(checked_rows(x, x_off, nullptr, nullptr, 1, B, N, D, dt, as_stream(stream)));
    const hipStream_t st = as_stream(stream);
    hipError_t e = mpm::launch_affinity(x, x_off, B, N, D, dt, schedule, w.pv, w.pi, st, nullptr, nullptr, nullptr);
    if (e == hipSuccess)
        e = mpm::launch_reduce_partials(w.pv, w.pi, mpm::partial_tile_width(B, D, dt, N, schedule), x, x_off, B, N, D,
                                        dt, nb, best, st);
    return hip_status(e);
}

int mpm_pair_compact(const int32_t* nb, const int32_t* x_off, int32_t B, int32_t N, int32_t* map, int32_t* src,
                     int32_t* y_off, void* stream)
{
    const int s = check_shape(B, N);
    if (s != MPM_OK) return s;
    if (!ok_int_ptr(nb) || !ok_opt_int_ptr(x_off) || !ok_int_ptr(map) || !ok_int_ptr(src) || !ok_int_ptr(y_off))
        return MPM_ERR_INVALID_ARG;
    MPM_LAUNCH_GATE();
    MPM_DATA_CHECK(checked_pairs(x_off, nb, nullptr, nullptr, B, N, as_stream(stream)));
    return hip_status(mpm::launch_pair_compact(nb, x_off, B, N, map, src, y_off, nullptr, as_stream(stream)));
}

int mpm_pair_average(const void* x, const int32_t* x_off, const int32_t* src, const int32_t* y_off, int32_t B,
                     int32_t N, int32_t D, int32_t dt, void* y, float* y_inv, void* stream)
{
    const int s = check_rows(B, N, D, dt);
    if (s != MPM_OK) return s;
    if (!ok_rows_ptr(x) || !ok_opt_int_ptr(x_off) || !ok_int_ptr(src) || !ok_int_ptr(y_off) || !ok_rows_ptr(y) ||
        !ok_opt_int_ptr(y_inv))
        return MPM_ERR_INVALID_ARG;
    MPM_LAUNCH_GATE();
    MPM_DATA_CHECK(checked_pairs(x_off, nullptr, y_off, src, B, N, as_stream(stream)));
    return hip_status(mpm::launch_pair_average(x, x_off, src, y_off, B, N, D, dt, y, y_inv, as_stream(stream)));
}

int mpm_merge(const void* x, const int32_t* x_off, const float* x_inv, int32_t B, int32_t N, int32_t D, int32_t dt,
              int32_t schedule, void* y, int32_t* y_off, float* y_inv, int32_t* map, void* ws, size_t ws_bytes,
              void* stream)
{
    int s = check_affinity(x, x_off, x_inv, B, N, D, dt, schedule);
    if (s != MPM_OK) return s;
    if (!ok_rows_ptr(y) || !ok_int_ptr(y_off) || !ok_opt_int_ptr(y_inv) || !ok_int_ptr(map))
        return MPM_ERR_INVALID_ARG;
    Workspace w;
    if ((s = carve(ws, ws_bytes, B, N, &w)) != MPM_OK) return s;
    MPM_LAUNCH_GATE();
    MPM_DATA_CHECK(checked_rows(x, x_off, x_inv, nullptr, 1, B, N, D, dt, as_stream(stream)));
    const hipStream_t st = as_stream(stream);
    hipError_t e = affinity_compact(x, x_off, x_inv, B, N, D, dt, schedule, map, y_off, w, nullptr, nullptr, st);
    if (e == hipSuccess) e = mpm::launch_pair_average(x, x_off, w.src, y_off, B, N, D, dt, y, y_inv, st);
    return hip_status(e);
}

int mpm_merge_noalloc(const void* x, const int32_t* x_off, const float* x_inv, int32_t B, int32_t N, int32_t D,
                      int32_t dt, int32_t schedule, void* y, int32_t* y_off, float* y_inv, int32_t* map, void* stream)
{
    int s = check_affinity(x, x_off, x_inv, B, N, D, dt, schedule);
    if (s != MPM_OK) return s;
    if (!ok_rows_ptr(y) || !ok_int_ptr(y_off) || !ok_opt_int_ptr(y_inv) || !ok_int_ptr(map))
        return MPM_ERR_INVALID_ARG;
    if (workspace_offsets(B, N).total > kScratchBytes) return MPM_ERR_WORKSPACE;
    MPM_LAUNCH_GATE();
    MPM_DATA_CHECK(checked_rows(x, x_off, x_inv, nullptr, 1, B, N, D, dt, as_stream(stream)));
    const hipStream_t st = as_stream(stream);
    void* ws = nullptr;
    hipError_t e = scratch_for_current_device(st, &ws);
    if (e != hipSuccess) return hip_status(e);
    Workspace w;
    if ((s = carve(ws, kScratchBytes, B, N, &w)) != MPM_OK) return s;
    e = affinity_compact(x, x_off, x_inv, B, N, D, dt, schedule, map, y_off, w, nullptr, nullptr, st);
    if (e == hipSuccess) e = mpm::launch_pair_average(x, x_off, w.src, y_off, B, N, D, dt, y, y_inv, st);
    return hip_status(e);
}

int mpm_merge_local(const void* x, const int32_t* x_off, const float* x_inv, const int32_t* pos, int32_t B,
                    int32_t N, int32_t D, int32_t dt, int32_t grid_w, int32_t window, int32_t block_rows, void* y,
                    int32_t* y_off, float* y_inv, int32_t* y_pos, int32_t* map, void* ws, size_t ws_bytes,
                    void* start_event, void* stop_event, void* stream)
{
    int s = check_affinity(x, x_off, x_inv, B, N, D, dt, MPM_SCHEDULE_AUTO);
    if (s != MPM_OK) return s;
    if (!ok_opt_int_ptr(pos) || !ok_rows_ptr(y) || !ok_int_ptr(y_off) || !ok_opt_int_ptr(y_inv) ||
        !ok_int_ptr(y_pos) || !ok_int_ptr(map))
        return MPM_ERR_INVALID_ARG;
    if (grid_w < 1 || grid_w > MPM_MAX_N || window < 0 || !mpm::valid_local_block_rows(block_rows))
        return MPM_ERR_INVALID_ARG;
    Workspace w;
    if ((s = carve(ws, ws_bytes, B, N, &w)) != MPM_OK) return s;
    MPM_LAUNCH_GATE();
    MPM_DATA_CHECK(checked_rows(x, x_off, x_inv, pos, grid_w, B, N, D, dt, as_stream(stream)));
    const hipStream_t st = as_stream(stream);
    const int rows = mpm::local_block_rows(B, N, D, dt, grid_w, window, block_rows);
    hipError_t e = mpm::launch_affinity_local(x, x_off, x_inv, pos, grid_w, window, rows, B, N, D, dt, w.pv, w.pi, st,
                                              static_cast<hipEvent_t>(start_event),
                                              static_cast<hipEvent_t>(stop_event));
    if (e == hipSuccess)
        e = compact_partials_ct(w, x_off, B, N, D, dt, rows, map, y_off, st);
    if (e == hipSuccess)
        e = mpm::launch_pair_average(x, x_off, w.src, y_off, B, N, D, dt, y, y_inv, st, pos, y_pos);
    return hip_status(e);
}

int mpm_pad(const void* z, const int32_t* z_off, int32_t B, int32_t P, int32_t row_bytes, void* out, void* stream)
{
    if (B < 1 || P < 1 || row_bytes < 16 || row_bytes % 16 != 0) return MPM_ERR_INVALID_ARG;
    if (B > MPM_MAX_B || P > MPM_MAX_N || row_bytes > MPM_MAX_D * 4) return MPM_ERR_UNSUPPORTED;
    if (!ok_rows_ptr(z) || !ok_int_ptr(z_off) || !ok_rows_ptr(out)) return MPM_ERR_INVALID_ARG;
    MPM_LAUNCH_GATE();
    MPM_DATA_CHECK(checked_maps(z_off, INT32_MAX, nullptr, nullptr, B, P, as_stream(stream)));
    return hip_status(mpm::launch_pad(z, z_off, B, P, row_bytes, out, false, as_stream(stream)));
}

int mpm_unpad(const void* padded, const int32_t* z_off, int32_t B, int32_t P, int32_t row_bytes, void* z,
              void* stream)
{
    if (B < 1 || P < 1 || row_bytes < 16 || row_bytes % 16 != 0) return MPM_ERR_INVALID_ARG;
    if (B > MPM_MAX_B || P > MPM_MAX_N || row_bytes > MPM_MAX_D * 4) return MPM_ERR_UNSUPPORTED;
    if (!ok_rows_ptr(padded) || !ok_int_ptr(z_off) || !ok_rows_ptr(z)) return MPM_ERR_INVALID_ARG;
    MPM_LAUNCH_GATE();
    MPM_DATA_CHECK(checked_maps(z_off, INT32_MAX, nullptr, nullptr, B, P, as_stream(stream)));
    return hip_status(mpm::launch_pad(padded, z_off, B, P, row_bytes, z, true, as_stream(stream)));
}

int mpm_compose(const int32_t* map_a, const int32_t* map_b, int32_t B, int32_t N, int32_t* map_ab, void* stream)
{
    const int s = check_shape(B, N);
    if (s != MPM_OK) return s;
    if (!ok_int_ptr(map_a) || !ok_int_ptr(map_b) || !ok_int_ptr(map_ab)) return MPM_ERR_INVALID_ARG;
    MPM_LAUNCH_GATE();
    MPM_DATA_CHECK(checked_maps(nullptr, N, map_a, map_b, B, N, as_stream(stream)));
    return hip_status(mpm::launch_compose(map_a, map_b, B, N, map_ab, as_stream(stream)));
}

int mpm_compose_unmerge(const void* z, const int32_t* z_off, const int32_t* map_a, const int32_t* map_b,
                        int32_t* map_ab, const void* z_spec, int32_t E, int32_t B, int32_t N, int32_t D, int32_t dt,
                        void* out, void* stream)
{
    const int s = check_rows(B, N, D, dt);
    if (s != MPM_OK) return s;
    if (E < 0 || (E > 0 && !ok_rows_ptr(z_spec)) || (E == 0 && z_spec != nullptr && !aligned(z_spec, 16)))
        return MPM_ERR_INVALID_ARG;
    if ((long)E + N > MPM_MAX_N + (long)MPM_MAX_N) return MPM_ERR_UNSUPPORTED;
    if (!ok_rows_ptr(z) || !ok_opt_int_ptr(z_off) || !ok_int_ptr(map_a) || !ok_int_ptr(map_b) ||
        !ok_opt_int_ptr(map_ab) || !ok_rows_ptr(out))
        return MPM_ERR_INVALID_ARG;
    if (map_ab != nullptr && (map_ab == map_a || map_ab == map_b)) return MPM_ERR_INVALID_ARG;
    MPM_LAUNCH_GATE();
    MPM_DATA_CHECK(checked_maps(z_off, N, map_a, map_b, B, N, as_stream(stream)));
    return hip_status(mpm::launch_unmerge(z, z_off, map_a, z_spec, E, B, N, D, dt, out, as_stream(stream), map_b,
                                          map_ab));
}

int mpm_unmerge(const void* z, const int32_t* z_off, const int32_t* map, const void* z_spec, int32_t E, int32_t B,
                int32_t N, int32_t D, int32_t dt, void* out, void* stream)
{
    const int s = check_rows(B, N, D, dt);
    if (s != MPM_OK) return s;
    if (E < 0 || (E > 0 && !ok_rows_ptr(z_spec)) || (E == 0 && z_spec != nullptr && !aligned(z_spec, 16)))
        return MPM_ERR_INVALID_ARG;
    if ((long)E + N > MPM_MAX_N + (long)MPM_MAX_N) return MPM_ERR_UNSUPPORTED;
    if (!ok_rows_ptr(z) || !ok_opt_int_ptr(z_off) || !ok_int_ptr(map) || !ok_rows_ptr(out)) return MPM_ERR_INVALID_ARG;
    MPM_LAUNCH_GATE();
    MPM_DATA_CHECK(checked_maps(z_off, N, map, nullptr, B, N, as_stream(stream)));
    return hip_status(mpm::launch_unmerge(z, z_off, map, z_spec, E, B, N, D, dt, out, as_stream(stream)));
}

}  // extern "C"
