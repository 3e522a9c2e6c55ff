// Host side of the C ABI declared in include/gwtf_mcf.h: argument checks,
// workspace ownership, and the choice of solver pass: stage-pipelined
// register-resident (16 < n <= 64, S <= 32), LDS-resident (n <= 64, one workgroup per
// instance), grid-cooperative (64 < n <= 512, one instance over many
// workgroups), and the global-memory fallback pass (any n, or instances
// whose link costs or flow lists do not fit the faster passes).
#include "gwtf_mcf.h"
#include "mcf_grid.h"
#include "mcf_internal.h"
#include "mcf_pipe.h"
#include "mcf_small.h"

#include <algorithm>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>

using namespace gwtf;

namespace {

// Device buffers the passes write besides the caller's outputs: routes,
// flows, potentials and counters of every instance, the fallback pass's
// per-instance state, and the grid pass's label words, predecessors, path
// and control block.
struct Workspace {
    int32_t *route = nullptr, *node_flow = nullptr, *arc_flow = nullptr, *pot = nullptr;
    int64_t *stats = nullptr;
    unsigned char *state = nullptr;
    size_t state_stride = 0;
    int64_t fallback_slots = 0;
    // grid-cooperative pass (64 < n <= 512), when the device can hold its grid
    bool grid = false;
    int64_t grid_slots = 0;
    size_t grid_lds = 0;
    int grid_conc = 0; // instances per grid launch (buffers for that many)
    uint32_t *g_ex = nullptr, *g_en = nullptr, *g_ring = nullptr;
    unsigned long long *g_ring_key = nullptr;
    int32_t *g_pred = nullptr, *g_path = nullptr, *g_ctrl = nullptr;
};

// Device properties the pass choice depends on.
struct DeviceInfo {
    size_t lds_max = 0;
    int clock_khz = 0;
    int coop = 0;
    int cus = 0;
};

// Queries `device` (which must be current) and raises the kernels' dynamic
// LDS ceilings.  No allocation.
hipError_t query_device(int device, DeviceInfo &d)
{
    int lds = 0;
    hipError_t e = hipDeviceGetAttribute(&lds, hipDeviceAttributeMaxSharedMemoryPerBlock, device);
    if (e != hipSuccess) return e;
    d.lds_max = size_t(lds);
    if (hipDeviceGetAttribute(&d.clock_khz, hipDeviceAttributeWallClockRate, device) != hipSuccess) d.clock_khz = 0;
    if (hipDeviceGetAttribute(&d.coop, hipDeviceAttributeCooperativeLaunch, device) != hipSuccess) d.coop = 0;
    if (hipDeviceGetAttribute(&d.cus, hipDeviceAttributeMultiprocessorCount, device) != hipSuccess) d.cus = 0;
    (void)hipGetLastError();
    // Raising the per-kernel dynamic-LDS ceiling is not needed on every
    // runtime (some reject the attribute); failure is harmless, but its error
    // must not linger where a later launch check would read it.
    if (set_lds_limits(d.lds_max) != hipSuccess) (void)hipGetLastError();
    return hipSuccess;
}

// Sizes the workspace of up to B instances of S x n (pointers stay NULL):
// fallback state for the worst case (every exit vertex may need
// min(cap, n, supply) <= n flow-list entries), and the grid pass when its
// S * ceil(n / 128) workgroups can all be resident at once (cooperative
// launch, one per CU given their LDS), with buffers for as many instances
// per launch as can be resident together (at most B).  The grid pass serves
// 64 < n <= 512, and pipelines too long for the register pass with
// 16 < n <= 64 when the batch is small (grid_preferred).
void plan_workspace(Workspace &w, int S, int n, int B, const DeviceInfo &d)
{
    w.fallback_slots = int64_t(std::max(S - 1, 0)) * n * n;
    w.state_stride = align16(make_layout(S, n, w.fallback_slots, false).total);
    w.grid = false;
    if ((n > 64 || (n > 16 && !pipe_pass_fits(S, n))) && n <= kGridMaxNodes && S <= 1024 && d.coop && d.cus > 0) {
        const int64_t slots = grid_pass_list_slots(S, n, d.lds_max);
        if (slots >= 64) {
            const size_t lds = grid_pass_lds_bytes(S, n, slots);
            const int per_cu = grid_pass_blocks_per_cu(lds);
            const int64_t blocks = int64_t(S) * grid_pass_slices(n);
            if (per_cu >= 1 && blocks <= int64_t(per_cu) * d.cus && blocks <= kGridMaxBlocks) {
                w.grid = true;
                w.grid_slots = slots;
                w.grid_lds = lds;
                w.grid_conc = int(std::min<int64_t>({int64_t(per_cu) * d.cus / blocks, int64_t(std::max(B, 1)),
                                                     int64_t(kGridMaxConcurrent)}));
            }
        }
    }
}

// Long pipelines of narrow stages (16 < n <= 64, more stages than the
// register pass holds) run on the grid pass when the batch needs at most
// kDeepGridLaunches launches of it, on the LDS pass otherwise: an instance
// of 40 x 64 takes about 0.1 s on the grid pass (40 workgroups) and 1.9 s
// on the LDS pass (one workgroup), but the LDS pass solves a whole large
// batch at once (128 such instances: 1.85 s, against 2.13 s in 22 grid
// launches of six).
constexpr int kDeepGridLaunches = 8;
bool grid_preferred(const Workspace &w, int n, int B)
{
    return n > 64 || (B + w.grid_conc - 1) / w.grid_conc <= kDeepGridLaunches;
}

// Calls f(&buffer_pointer, bytes) for every workspace buffer of B instances
// (bytes may be 0: the buffer is not used).
template <class Fn>
void for_each_buffer(Workspace &w, int S, int n, int B, Fn f)
{
    const size_t SN = size_t(S) * n, V = 2 * SN + 3, na = size_t(std::max(S - 1, 0)) * n * n;
    const size_t gsn = w.grid ? SN : 0, gc = w.grid ? size_t(w.grid_conc) : 0;
    f((void **)&w.route, sizeof(int32_t) * B);
    f((void **)&w.node_flow, sizeof(int32_t) * SN * B);
    f((void **)&w.arc_flow, sizeof(int32_t) * std::max<size_t>(na, 1) * B);
    f((void **)&w.pot, sizeof(int32_t) * V * B);
    f((void **)&w.stats, sizeof(int64_t) * kStatsPerInstance * B);
    f((void **)&w.state, w.state_stride * B);
    f((void **)&w.g_ex, sizeof(uint32_t) * 2 * gsn * gc);
    f((void **)&w.g_en, sizeof(uint32_t) * 2 * gsn * gc);
    f((void **)&w.g_pred, sizeof(int32_t) * gsn * gc);
    f((void **)&w.g_path, sizeof(int32_t) * (2 * gsn + 8) * gc);
    f((void **)&w.g_ctrl, sizeof(int32_t) * kGridCtrlInts * gc);
    f((void **)&w.g_ring, sizeof(uint32_t) * kRingStride * grid_ring_slots(S) * gc);
    f((void **)&w.g_ring_key, sizeof(unsigned long long) * kRingKeyStride * grid_ring_slots(S) * gc);
}

} // namespace

struct gwtf_mcf {
    gwtf_mcf_shape_t shape;
    hipStream_t stream;
    std::string err;
    DeviceInfo dev;
    Workspace ws;
    int32_t *dense_arc = nullptr; // located batches: implied link delays, allocated on first use
    int32_t solved = 0; // batch size of the last successful solve (0 = none)
};

namespace {

// Last error of a call made without a handle (create, the no-allocation
// solve), per thread; a fixed buffer, so reporting allocates nothing.
thread_local char g_thread_err[256];

gwtf_status_t fail_thread(gwtf_status_t code, const char *what, hipError_t e = hipSuccess)
{
    if (e != hipSuccess) snprintf(g_thread_err, sizeof g_thread_err, "%s: %s", what, hipGetErrorString(e));
    else snprintf(g_thread_err, sizeof g_thread_err, "%s", what);
    return code;
}

gwtf_status_t fail(gwtf_mcf_t *h, gwtf_status_t code, const std::string &msg)
{
    if (h) h->err = msg;
    else fail_thread(code, msg.c_str());
    return code;
}

gwtf_status_t hip_fail(gwtf_mcf_t *h, hipError_t e, const char *what)
{
    return fail(h, GWTF_ERR_DEVICE, std::string(what) + ": " + hipGetErrorString(e));
}

// Narrow LDS state: flow-list capacity left once the node state and the
// scratch buffers are placed (0 if the node state alone does not fit).
int64_t lds_slots(int S, int n, int waves, size_t lds_max)
{
    if (n > 64) return 0;
    size_t fixed = make_layout(S, n, 0, true).total + scratch_bytes(waves, n) + 64;
    if (fixed >= lds_max) return 0;
    int64_t slots = int64_t((lds_max - fixed) / 9) - 16;
    int64_t worst = int64_t(std::max(S - 1, 0)) * n * n;
    slots = std::min<int64_t>(std::min<int64_t>(slots, worst), 65535);
    return std::max<int64_t>(slots, 0);
}

int lds_waves(int n) { return n <= 16 ? 1 : 4; }

void free_ws(gwtf_mcf_t *h)
{
    for_each_buffer(h->ws, h->shape.num_stages, h->shape.nodes_per_stage, h->shape.max_batch,
                    [](void **p, size_t) {
                        (void)hipFree(*p);
                        *p = nullptr;
                    });
    (void)hipFree(h->dense_arc);
    h->dense_arc = nullptr;
}

// Shape checks shared by gwtf_mcf_create and the no-allocation solve.
const char *check_shape(int S, int n, int B)
{
    if (S < 1 || n < 1 || B < 1) return "shape values must be >= 1";
    if (n > 32767) return "nodes_per_stage must be <= 32767";
    const int64_t V = 2 * int64_t(S) * n + 3;
    if (V > (int64_t(1) << 30) / 4) return "shape too large";
    return nullptr;
}

} // namespace

extern "C" gwtf_status_t gwtf_mcf_create(const gwtf_mcf_shape_t *shape, void *hip_stream, gwtf_mcf_t **out)
{
    if (!out) return fail_thread(GWTF_ERR_INVALID_ARG, "out is NULL");
    *out = nullptr;
    if (!shape) return fail_thread(GWTF_ERR_INVALID_ARG, "shape is NULL");
    const int S = shape->num_stages, n = shape->nodes_per_stage, B = shape->max_batch;
    if (const char *bad = check_shape(S, n, B)) return fail_thread(GWTF_ERR_INVALID_ARG, bad);
    int ndev = 0;
    hipError_t e = hipGetDeviceCount(&ndev);
    if (e != hipSuccess) return fail_thread(GWTF_ERR_DEVICE, "hipGetDeviceCount", e);
    if (shape->device < 0 || shape->device >= ndev) return fail_thread(GWTF_ERR_INVALID_ARG, "bad device ordinal");
    if ((e = hipSetDevice(shape->device)) != hipSuccess) return fail_thread(GWTF_ERR_DEVICE, "hipSetDevice", e);

    gwtf_mcf_t *h = new (std::nothrow) gwtf_mcf_t();
    if (!h) return fail_thread(GWTF_ERR_OUT_OF_MEMORY, "host allocation failed");
    h->shape = *shape;
    h->stream = static_cast<hipStream_t>(hip_stream);
    if ((e = query_device(shape->device, h->dev)) != hipSuccess) {
        delete h;
        return fail_thread(GWTF_ERR_DEVICE, "hipDeviceGetAttribute", e);
    }
    plan_workspace(h->ws, S, n, B, h->dev);
    hipError_t first = hipSuccess;
    for_each_buffer(h->ws, S, n, B, [&](void **p, size_t bytes) {
        if (bytes == 0 || first != hipSuccess) return;
        if ((e = hipMalloc(p, bytes)) != hipSuccess) {
            *p = nullptr;
            first = e;
        }
    });
    if (first != hipSuccess) {
        free_ws(h);
        delete h;
        return fail_thread(GWTF_ERR_OUT_OF_MEMORY, "hipMalloc workspace", first);
    }
    *out = h;
    return GWTF_OK;
}

namespace {

struct PassResult {
    gwtf_status_t code;
    const char *what; // failing step (code != GWTF_OK)
    hipError_t e;     // its HIP error (GWTF_ERR_DEVICE)
};

// Enqueues the solver passes for one batch (p describes it; loc/lat non-NULL
// selects the location-factored grid pass for shapes that use the grid),
// with workspace `w` and the properties `d` of the current device.
PassResult run_passes(const Workspace &w, const DeviceInfo &d, int S, int n, hipStream_t stream, SolveParams &p,
                      const int32_t *loc, const int32_t *lat, int32_t L)
{
    hipError_t e;
    p.route = w.route;
    p.node_flow = w.node_flow;
    p.arc_flow = w.arc_flow;
    p.pot = w.pot;
    p.stats = w.stats;
    p.state = w.state;
    p.state_stride = w.state_stride;
    p.clock_khz = d.clock_khz;

    const int64_t worst = int64_t(std::max(S - 1, 0)) * n * n;
    bool need_fallback = true;
    const int64_t pipe_slots = (n > 16 && pipe_pass_fits(S, n)) ? pipe_pass_slots(S, d.lds_max) : 0;
    const int waves = lds_waves(n);
    const int64_t slots = pipe_slots > 0 ? 0 : lds_slots(S, n, waves, d.lds_max);
    if (small_pass_fits(S, n)) {
        // Four instances per wave; instances outside the packed bounds go to
        // the fallback pass.
        p.list_slots = 0;
        p.route_all = 0;
        if ((e = launch_small_pass(p, stream)) != hipSuccess) return {GWTF_ERR_DEVICE, "packed solver launch", e};
        need_fallback = true;
    } else if (w.grid && grid_preferred(w, n, p.B)) {
        // Cooperative launches of up to grid_conc instances each; instances
        // whose link costs need more than 16 bits or whose flow lists outgrow
        // LDS go to the fallback pass.
        GridParams gp{};
        gp.base = p;
        gp.base.list_slots = w.grid_slots;
        gp.base.route_all = 0;
        gp.slices = grid_pass_slices(n);
        gp.list_slots = w.grid_slots;
        gp.big_bytes = grid_pass_big_bytes(S, n);
        gp.ex = w.g_ex;
        gp.en = w.g_en;
        gp.pred = w.g_pred;
        gp.path = w.g_path;
        gp.ctrl = w.g_ctrl;
        gp.ring = w.g_ring;
        gp.ring_key = w.g_ring_key;
        gp.ring_slots = grid_ring_slots(S);
        gp.loc = loc;
        gp.lat = lat;
        gp.L = L;
        for (int i = 0; i < p.B; i += w.grid_conc) {
            gp.instance = i;
            gp.count = std::min(w.grid_conc, p.B - i);
            if ((e = launch_grid_pass(gp, w.grid_lds, stream)) != hipSuccess)
                return {GWTF_ERR_DEVICE, "grid solver launch", e};
        }
        need_fallback = true;
    } else if (pipe_slots > 0) {
        // Stage-pipelined register pass; instances needing wider link costs
        // or more flow-list slots go to the fallback pass.
        p.list_slots = pipe_slots;
        p.route_all = 0;
        if ((e = launch_pipe_pass(p, stream)) != hipSuccess) return {GWTF_ERR_DEVICE, "pipelined solver launch", e};
        need_fallback = true;
    } else if (slots > 0) {
        p.list_slots = slots;
        p.route_all = 0;
        size_t lds = make_layout(S, n, slots, true).total + scratch_bytes(waves, n);
        if ((e = launch_lds_pass(p, waves, lds, stream)) != hipSuccess) return {GWTF_ERR_DEVICE, "LDS solver launch", e};
        // Worst-case list demand of an instance: (S-1) * n * min(n, cap, supply).
        need_fallback = slots < worst;
    } else {
        p.route_all = 1;
    }
    if (need_fallback) {
        p.list_slots = w.fallback_slots;
        size_t lds = scratch_bytes(fallback_waves(), n);
        if (lds > d.lds_max) return {GWTF_ERR_INVALID_ARG, "nodes_per_stage too large for LDS scratch", hipSuccess};
        if ((e = launch_fallback_pass(p, lds, stream)) != hipSuccess)
            return {GWTF_ERR_DEVICE, "fallback solver launch", e};
    }
    return {GWTF_OK, nullptr, hipSuccess};
}

// run_passes on a handle's workspace, with the outcome in the handle.
gwtf_status_t run_handle_passes(gwtf_mcf_t *h, SolveParams &p, const int32_t *loc, const int32_t *lat, int32_t L)
{
    h->solved = 0;
    const PassResult r = run_passes(h->ws, h->dev, h->shape.num_stages, h->shape.nodes_per_stage, h->stream, p,
                                    loc, lat, L);
    if (r.code == GWTF_ERR_DEVICE) return hip_fail(h, r.e, r.what);
    if (r.code != GWTF_OK) return fail(h, r.code, r.what);
    h->solved = p.B;
    h->err.clear();
    return GWTF_OK;
}

} // namespace

extern "C" gwtf_status_t gwtf_mcf_solve_batch(gwtf_mcf_t *h, const gwtf_mcf_batch_t *b)
{
    if (!h) return fail(nullptr, GWTF_ERR_INVALID_ARG, "handle is NULL");
    if (!b) return fail(h, GWTF_ERR_INVALID_ARG, "batch is NULL");
    const int S = h->shape.num_stages, n = h->shape.nodes_per_stage;
    if (b->batch < 1 || b->batch > h->shape.max_batch)
        return fail(h, GWTF_ERR_INVALID_ARG, "batch outside [1, max_batch]");
    if (!b->node_cap || !b->node_cost || !b->supply || !b->flow_value || !b->total_cost || !b->status)
        return fail(h, GWTF_ERR_INVALID_ARG, "required pointer is NULL");
    if ((S > 1) != (b->arc_cost != nullptr))
        return fail(h, GWTF_ERR_INVALID_ARG, "arc_cost must be non-NULL exactly when S > 1");
    hipError_t e = hipSetDevice(h->shape.device);
    if (e != hipSuccess) return hip_fail(h, e, "hipSetDevice");

    SolveParams p{};
    p.B = b->batch;
    p.S = S;
    p.n = n;
    p.cap = b->node_cap;
    p.ncost = b->node_cost;
    p.acost = b->arc_cost;
    p.src = b->src_cost;
    p.snk = b->snk_cost;
    p.supply = b->supply;
    p.F_out = b->flow_value;
    p.cost_out = b->total_cost;
    p.status_out = b->status;
    return run_handle_passes(h, p, nullptr, nullptr, 0);
}

// ---- Solve without allocation ----
//
extern "C" gwtf_status_t gwtf_mcf_calibrate_handoff(int32_t device, void *hip_stream, int32_t block_distance,
                                                    double *latency_ns)
{
    if (!latency_ns) return fail_thread(GWTF_ERR_INVALID_ARG, "latency_ns is NULL");
    if (block_distance < 1 || block_distance > 15 || block_distance == 8)
        return fail_thread(GWTF_ERR_INVALID_ARG, "block_distance outside [1, 15] or equal to 8");
    int ndev = 0;
    hipError_t e = hipGetDeviceCount(&ndev);
    if (e != hipSuccess) return fail_thread(GWTF_ERR_DEVICE, "hipGetDeviceCount", e);
    if (device < 0 || device >= ndev) return fail_thread(GWTF_ERR_INVALID_ARG, "bad device ordinal");
    if ((e = hipSetDevice(device)) != hipSuccess) return fail_thread(GWTF_ERR_DEVICE, "hipSetDevice", e);
    int clock_khz = 0;
    if (hipDeviceGetAttribute(&clock_khz, hipDeviceAttributeWallClockRate, device) != hipSuccess) clock_khz = 0;
    (void)hipGetLastError();
    double out[3];
    if ((e = run_handoff_calibration(static_cast<hipStream_t>(hip_stream), clock_khz, block_distance, out)) !=
        hipSuccess)
        return fail_thread(GWTF_ERR_DEVICE, "hand-off calibration", e);
    for (int q = 0; q < 3; ++q) latency_ns[q] = out[q];
    return GWTF_OK;
}

// Workspace of gwtf_mcf_solve_batch_noalloc: one array per device, held
// until the process ends.  In host code this name is only a host-side
// stand-in; the device address comes from hipGetSymbolAddress, once per
// device, and only that address is handed to kernels.
constexpr size_t kScratchBytes = size_t(64) << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

constexpr int kScratchMaxDevices = 64;
struct ScratchDevice {
    bool ready = false;
    unsigned char *ptr = nullptr; // device address of `scratch` on this device
    DeviceInfo dev;
};
ScratchDevice g_scratch[kScratchMaxDevices];
std::mutex g_scratch_lock;

} // namespace

extern "C" gwtf_status_t gwtf_mcf_solve_batch_noalloc(const gwtf_mcf_shape_t *shape, void *hip_stream,
                                                      const gwtf_mcf_batch_t *b)
{
    if (!shape) return fail_thread(GWTF_ERR_INVALID_ARG, "shape is NULL");
    if (!b) return fail_thread(GWTF_ERR_INVALID_ARG, "batch is NULL");
    const int S = shape->num_stages, n = shape->nodes_per_stage;
    if (const char *bad = check_shape(S, n, shape->max_batch)) return fail_thread(GWTF_ERR_INVALID_ARG, bad);
    if (b->batch < 1 || b->batch > shape->max_batch)
        return fail_thread(GWTF_ERR_INVALID_ARG, "batch outside [1, max_batch]");
    if (!b->node_cap || !b->node_cost || !b->supply || !b->flow_value || !b->total_cost || !b->status)
        return fail_thread(GWTF_ERR_INVALID_ARG, "required pointer is NULL");
    if ((S > 1) != (b->arc_cost != nullptr))
        return fail_thread(GWTF_ERR_INVALID_ARG, "arc_cost must be non-NULL exactly when S > 1");
    int ndev = 0;
    hipError_t e = hipGetDeviceCount(&ndev);
    if (e != hipSuccess) return fail_thread(GWTF_ERR_DEVICE, "hipGetDeviceCount", e);
    const int device = shape->device;
    if (device < 0 || device >= ndev || device >= kScratchMaxDevices)
        return fail_thread(GWTF_ERR_INVALID_ARG, "bad device ordinal");
    if ((e = hipSetDevice(device)) != hipSuccess) return fail_thread(GWTF_ERR_DEVICE, "hipSetDevice", e);

    DeviceInfo dev;
    unsigned char *base = nullptr;
    {
        std::lock_guard<std::mutex> lock(g_scratch_lock);
        ScratchDevice &sd = g_scratch[device];
        if (!sd.ready) {
            void *ptr = nullptr;
            if ((e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch))) != hipSuccess)
                return fail_thread(GWTF_ERR_DEVICE, "hipGetSymbolAddress(scratch)", e);
            if ((e = query_device(device, sd.dev)) != hipSuccess)
                return fail_thread(GWTF_ERR_DEVICE, "hipDeviceGetAttribute", e);
            sd.ptr = static_cast<unsigned char *>(ptr);
            sd.ready = true;
        }
        dev = sd.dev;
        base = sd.ptr;
    }

    // Lay the workspace of this batch out in the array (256-byte aligned
    // buffers), or refuse the batch if it does not fit.
    Workspace w;
    plan_workspace(w, S, n, b->batch, dev);
    size_t need = 0;
    for_each_buffer(w, S, n, b->batch, [&](void **, size_t bytes) {
        if (bytes) need = ((need + 255) & ~size_t(255)) + bytes;
    });
    if (need > kScratchBytes) {
        snprintf(g_thread_err, sizeof g_thread_err,
                 "batch needs %zu bytes of workspace, more than the %zu-byte scratch array; split it", need,
                 kScratchBytes);
        return GWTF_ERR_INVALID_ARG;
    }
    size_t off = 0;
    for_each_buffer(w, S, n, b->batch, [&](void **p, size_t bytes) {
        if (!bytes) return;
        off = (off + 255) & ~size_t(255);
        *p = base + off;
        off += bytes;
    });

    SolveParams p{};
    p.B = b->batch;
    p.S = S;
    p.n = n;
    p.cap = b->node_cap;
    p.ncost = b->node_cost;
    p.acost = b->arc_cost;
    p.src = b->src_cost;
    p.snk = b->snk_cost;
    p.supply = b->supply;
    p.F_out = b->flow_value;
    p.cost_out = b->total_cost;
    p.status_out = b->status;
    const PassResult r = run_passes(w, dev, S, n, static_cast<hipStream_t>(hip_stream), p, nullptr, nullptr, 0);
    if (r.code != GWTF_OK) return fail_thread(r.code, r.what, r.e);
    return GWTF_OK;
}

extern "C" gwtf_status_t gwtf_mcf_solve_located(gwtf_mcf_t *h, const gwtf_mcf_located_batch_t *b)
{
    if (!h) return fail(nullptr, GWTF_ERR_INVALID_ARG, "handle is NULL");
    if (!b) return fail(h, GWTF_ERR_INVALID_ARG, "batch is NULL");
    const int S = h->shape.num_stages, n = h->shape.nodes_per_stage, L = b->num_locations;
    if (b->batch < 1 || b->batch > h->shape.max_batch)
        return fail(h, GWTF_ERR_INVALID_ARG, "batch outside [1, max_batch]");
    if (L < 1 || L > kGridMaxLocations) return fail(h, GWTF_ERR_INVALID_ARG, "num_locations outside [1, 32]");
    if (!b->node_cap || !b->node_cost || !b->location || !b->latency || !b->supply || !b->flow_value ||
        !b->total_cost || !b->status)
        return fail(h, GWTF_ERR_INVALID_ARG, "required pointer is NULL");
    hipError_t e = hipSetDevice(h->shape.device);
    if (e != hipSuccess) return hip_fail(h, e, "hipSetDevice");
    const size_t na = size_t(std::max(S - 1, 0)) * n * n;
    if (S > 1 && !h->dense_arc) {
        if ((e = hipMalloc((void **)&h->dense_arc, sizeof(int32_t) * na * h->shape.max_batch)) != hipSuccess) {
            h->dense_arc = nullptr;
            return fail(h, GWTF_ERR_OUT_OF_MEMORY, std::string("hipMalloc located workspace: ") + hipGetErrorString(e));
        }
    }
    // The implied dense delays serve every pass but the factored grid pass
    // (the fallback pass included), so they are always written.
    if ((e = launch_located_expand(b->batch, S, n, L, b->location, b->latency, h->dense_arc, h->stream)) != hipSuccess)
        return hip_fail(h, e, "located expansion launch");

    SolveParams p{};
    p.B = b->batch;
    p.S = S;
    p.n = n;
    p.cap = b->node_cap;
    p.ncost = b->node_cost;
    p.acost = S > 1 ? h->dense_arc : nullptr;
    p.src = b->src_cost;
    p.snk = b->snk_cost;
    p.supply = b->supply;
    p.F_out = b->flow_value;
    p.cost_out = b->total_cost;
    p.status_out = b->status;
    return run_handle_passes(h, p, b->location, b->latency, L);
}

extern "C" gwtf_status_t gwtf_mcf_get_flows(gwtf_mcf_t *h, int32_t first, int32_t count, int32_t *node_flow,
                                            int32_t *arc_flow, int32_t *src_flow, int32_t *snk_flow,
                                            int32_t *potential)
{
    if (!h) return fail(nullptr, GWTF_ERR_INVALID_ARG, "handle is NULL");
    if (h->solved == 0) return fail(h, GWTF_ERR_NOT_SOLVED, "no successful solve on this handle");
    if (first < 0 || count < 0 || int64_t(first) + count > h->solved)
        return fail(h, GWTF_ERR_RANGE, "instance range outside the last solved batch");
    if (count == 0) return GWTF_OK;
    hipError_t e = hipSetDevice(h->shape.device);
    if (e != hipSuccess) return hip_fail(h, e, "hipSetDevice");
    const int S = h->shape.num_stages, n = h->shape.nodes_per_stage;
    const size_t SN = size_t(S) * n, V = 2 * SN + 3, na = size_t(std::max(S - 1, 0)) * n * n;
    auto copy = [&](void *dst, const void *src, size_t bytes) -> hipError_t {
        if (!dst || bytes == 0) return hipSuccess;
        return hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToDevice, h->stream);
    };
    if ((e = copy(node_flow, h->ws.node_flow + size_t(first) * SN, sizeof(int32_t) * SN * count)) != hipSuccess)
        return hip_fail(h, e, "copy node_flow");
    if ((e = copy(arc_flow, h->ws.arc_flow + size_t(first) * na, sizeof(int32_t) * na * count)) != hipSuccess)
        return hip_fail(h, e, "copy arc_flow");
    if ((e = copy(potential, h->ws.pot + size_t(first) * V, sizeof(int32_t) * V * count)) != hipSuccess)
        return hip_fail(h, e, "copy potential");
    if (src_flow || snk_flow) {
        if ((e = launch_export(h->ws.node_flow, S, n, first, count, src_flow, snk_flow, h->stream)) != hipSuccess)
            return hip_fail(h, e, "export launch");
    }
    return GWTF_OK;
}

extern "C" gwtf_status_t gwtf_mcf_get_stats(gwtf_mcf_t *h, int32_t first, int32_t count, int64_t *stats)
{
    if (!h) return fail(nullptr, GWTF_ERR_INVALID_ARG, "handle is NULL");
    if (!stats) return fail(h, GWTF_ERR_INVALID_ARG, "stats is NULL");
    if (h->solved == 0) return fail(h, GWTF_ERR_NOT_SOLVED, "no successful solve on this handle");
    if (first < 0 || count < 0 || int64_t(first) + count > h->solved)
        return fail(h, GWTF_ERR_RANGE, "instance range outside the last solved batch");
    if (count == 0) return GWTF_OK;
    hipError_t e = hipSetDevice(h->shape.device);
    if (e != hipSuccess) return hip_fail(h, e, "hipSetDevice");
    e = hipMemcpyAsync(stats, h->ws.stats + size_t(first) * kStatsPerInstance,
                       sizeof(int64_t) * kStatsPerInstance * count, hipMemcpyDeviceToDevice, h->stream);
    if (e != hipSuccess) return hip_fail(h, e, "copy stats");
    return GWTF_OK;
}

extern "C" gwtf_status_t gwtf_mcf_get_passes(gwtf_mcf_t *h, int32_t first, int32_t count, int32_t *pass)
{
    if (!h) return fail(nullptr, GWTF_ERR_INVALID_ARG, "handle is NULL");
    if (!pass) return fail(h, GWTF_ERR_INVALID_ARG, "pass is NULL");
    if (h->solved == 0) return fail(h, GWTF_ERR_NOT_SOLVED, "no successful solve on this handle");
    if (first < 0 || count < 0 || int64_t(first) + count > h->solved)
        return fail(h, GWTF_ERR_RANGE, "instance range outside the last solved batch");
    if (count == 0) return GWTF_OK;
    hipError_t e = hipSetDevice(h->shape.device);
    if (e != hipSuccess) return hip_fail(h, e, "hipSetDevice");
    e = hipMemcpyAsync(pass, h->ws.route + first, sizeof(int32_t) * count, hipMemcpyDeviceToDevice, h->stream);
    if (e != hipSuccess) return hip_fail(h, e, "copy pass");
    return GWTF_OK;
}

extern "C" void gwtf_mcf_destroy(gwtf_mcf_t *h)
{
    if (!h) return;
    if (hipSetDevice(h->shape.device) == hipSuccess) (void)hipStreamSynchronize(h->stream);
    free_ws(h);
    delete h;
}

extern "C" const char *gwtf_mcf_last_error(const gwtf_mcf_t *h)
{
    return h ? h->err.c_str() : g_thread_err;
}

namespace {

// S!/(S-m)! into *out; false when it does not fit in an int64.
bool placement_count(int32_t S, int32_t m, int64_t *out)
{
    int64_t c = 1;
    for (int32_t k = S - m + 1; k <= S; ++k) {
        if (c > INT64_MAX / k) return false;
        c *= k;
    }
    *out = c;
    return true;
}

} // namespace

extern "C" gwtf_status_t gwtf_whatif_count(int32_t num_stages, int32_t num_candidates, int64_t *count)
{
    if (!count) return fail(nullptr, GWTF_ERR_INVALID_ARG, "count is NULL");
    if (num_stages < 1 || num_candidates < 0 || num_candidates > num_stages)
        return fail(nullptr, GWTF_ERR_INVALID_ARG, "need S >= 1 and 0 <= m <= S");
    if (!placement_count(num_stages, num_candidates, count))
        return fail(nullptr, GWTF_ERR_INVALID_ARG, "S!/(S-m)! does not fit in an int64");
    return GWTF_OK;
}

extern "C" gwtf_status_t gwtf_mcf_whatif_expand(gwtf_mcf_t *h, const gwtf_mcf_batch_t *base,
                                                const gwtf_whatif_candidates_t *cand, int64_t first,
                                                int32_t count, const gwtf_mcf_instances_t *out)
{
    if (!h) return fail(nullptr, GWTF_ERR_INVALID_ARG, "handle is NULL");
    if (!base || !cand || !out) return fail(h, GWTF_ERR_INVALID_ARG, "base, cand or out is NULL");
    const int S = h->shape.num_stages, n = h->shape.nodes_per_stage, m = cand->num_candidates;
    if (S > kWhatifMaxStages) return fail(h, GWTF_ERR_INVALID_ARG, "what-if expansion needs S <= 1024");
    if (int64_t(S - 1) * n * n >= (int64_t(1) << 31) || int64_t(S) * n >= (int64_t(1) << 31))
        return fail(h, GWTF_ERR_INVALID_ARG, "instance too large for the what-if expansion");
    if (base->batch != 1) return fail(h, GWTF_ERR_INVALID_ARG, "base must hold exactly one instance");
    if (!base->node_cap || !base->node_cost || !base->supply)
        return fail(h, GWTF_ERR_INVALID_ARG, "base pointer is NULL");
    if ((S > 1) != (base->arc_cost != nullptr))
        return fail(h, GWTF_ERR_INVALID_ARG, "base arc_cost must be non-NULL exactly when S > 1");
    if (m < 0 || m > S) return fail(h, GWTF_ERR_INVALID_ARG, "num_candidates outside [0, S]");
    if (cand->slot < 0 || cand->slot >= n) return fail(h, GWTF_ERR_INVALID_ARG, "slot outside [0, n)");
    if ((m > 0) != (cand->cap != nullptr) || (m > 0) != (cand->cost != nullptr))
        return fail(h, GWTF_ERR_INVALID_ARG, "candidate cap and cost must be non-NULL exactly when m > 0");
    const bool links = S > 1 && m > 0;
    if (links != (cand->in_cost != nullptr) || links != (cand->out_cost != nullptr) ||
        links != (cand->link_cost != nullptr))
        return fail(h, GWTF_ERR_INVALID_ARG,
                    "candidate in_cost, out_cost and link_cost must be non-NULL exactly when S > 1 and m > 0");
    if (count < 0 || first < 0) return fail(h, GWTF_ERR_INVALID_ARG, "first and count must be >= 0");
    if (count > 0 && (!out->node_cap || !out->node_cost || !out->src_cost || !out->snk_cost || !out->supply))
        return fail(h, GWTF_ERR_INVALID_ARG, "output pointer is NULL");
    if (count > 0 && (S > 1) != (out->arc_cost != nullptr))
        return fail(h, GWTF_ERR_INVALID_ARG, "output arc_cost must be non-NULL exactly when S > 1");
    int64_t total = 0;
    if (!placement_count(S, m, &total))
        return fail(h, GWTF_ERR_INVALID_ARG, "S!/(S-m)! does not fit in an int64");
    if (first > total || count > total - first)
        return fail(h, GWTF_ERR_RANGE, "placement range outside [0, S!/(S-m)!)");
    if (count == 0) return GWTF_OK;
    hipError_t e = hipSetDevice(h->shape.device);
    if (e != hipSuccess) return hip_fail(h, e, "hipSetDevice");
    WhatifExpandParams p{};
    p.S = S;
    p.n = n;
    p.m = m;
    p.slot = cand->slot;
    p.first = first;
    p.cap = base->node_cap;
    p.cost = base->node_cost;
    p.arc = base->arc_cost;
    p.src = base->src_cost;
    p.snk = base->snk_cost;
    p.supply = base->supply;
    p.ccap = cand->cap;
    p.ccost = cand->cost;
    p.cin = cand->in_cost;
    p.cout = cand->out_cost;
    p.clink = cand->link_cost;
    p.csrc = cand->src_cost;
    p.csnk = cand->snk_cost;
    p.out_cap = out->node_cap;
    p.out_cost = out->node_cost;
    p.out_arc = out->arc_cost;
    p.out_src = out->src_cost;
    p.out_snk = out->snk_cost;
    p.out_supply = out->supply;
    if ((e = launch_whatif_expand(p, count, h->stream)) != hipSuccess) return hip_fail(h, e, "what-if expansion launch");
    return GWTF_OK;
}

extern "C" gwtf_status_t gwtf_mcf_whatif_best(gwtf_mcf_t *h, int32_t count, const int64_t *flow_value,
                                              const int64_t *total_cost, const int32_t *status, int64_t first,
                                              int32_t merge, int64_t *best)
{
    if (!h) return fail(nullptr, GWTF_ERR_INVALID_ARG, "handle is NULL");
    if (!best) return fail(h, GWTF_ERR_INVALID_ARG, "best is NULL");
    if (count < 0 || first < 0) return fail(h, GWTF_ERR_INVALID_ARG, "first and count must be >= 0");
    if (count > 0 && (!flow_value || !total_cost || !status))
        return fail(h, GWTF_ERR_INVALID_ARG, "flow_value, total_cost or status is NULL");
    hipError_t e = hipSetDevice(h->shape.device);
    if (e != hipSuccess) return hip_fail(h, e, "hipSetDevice");
    if ((e = launch_whatif_best(count, flow_value, total_cost, status, first, merge, best, h->stream)) != hipSuccess)
        return hip_fail(h, e, "what-if best launch");
    return GWTF_OK;
}

extern "C" gwtf_status_t gwtf_mcf_resolve_churn(gwtf_mcf_t *h, const gwtf_mcf_batch_t *b,
                                                const gwtf_mcf_flow_in_t *start,
                                                const gwtf_mcf_flow_out_t *out, int64_t *work)
{
    if (!h) return fail(nullptr, GWTF_ERR_INVALID_ARG, "handle is NULL");
    if (!b || !start) return fail(h, GWTF_ERR_INVALID_ARG, "batch or start flow is NULL");
    const int S = h->shape.num_stages, n = h->shape.nodes_per_stage;
    if (int64_t(S) * n > kChurnMaxNodes || int64_t(S - 1) * n * n > kChurnMaxLinks)
        return fail(h, GWTF_ERR_INVALID_ARG, "churn re-solve needs S*n <= 512 and (S-1)*n*n <= 4096");
    if (b->batch < 1 || b->batch > h->shape.max_batch)
        return fail(h, GWTF_ERR_INVALID_ARG, "batch outside [1, max_batch]");
    if (!b->node_cap || !b->node_cost || !b->supply || !b->flow_value || !b->total_cost || !b->status)
        return fail(h, GWTF_ERR_INVALID_ARG, "required pointer is NULL");
    if ((S > 1) != (b->arc_cost != nullptr))
        return fail(h, GWTF_ERR_INVALID_ARG, "arc_cost must be non-NULL exactly when S > 1");
    if (!start->node_flow || !start->src_flow || !start->snk_flow || (S > 1) != (start->arc_flow != nullptr))
        return fail(h, GWTF_ERR_INVALID_ARG,
                    "start flow needs node_flow, src_flow, snk_flow, and arc_flow exactly when S > 1");
    if (out && (!out->node_flow || !out->src_flow || !out->snk_flow || (S > 1) != (out->arc_flow != nullptr)))
        return fail(h, GWTF_ERR_INVALID_ARG,
                    "result flows need node_flow, src_flow, snk_flow, and arc_flow exactly when S > 1");
    hipError_t e = hipSetDevice(h->shape.device);
    if (e != hipSuccess) return hip_fail(h, e, "hipSetDevice");
    ChurnParams p{};
    p.B = b->batch;
    p.S = S;
    p.n = n;
    p.start_per_instance = start->per_instance != 0;
    p.cap = b->node_cap;
    p.ncost = b->node_cost;
    p.acost = b->arc_cost;
    p.src = b->src_cost;
    p.snk = b->snk_cost;
    p.supply = b->supply;
    p.nf0 = start->node_flow;
    p.af0 = start->arc_flow;
    p.sf0 = start->src_flow;
    p.tf0 = start->snk_flow;
    p.F_out = b->flow_value;
    p.cost_out = b->total_cost;
    p.status_out = b->status;
    if (out) {
        p.nf_out = out->node_flow;
        p.af_out = out->arc_flow;
        p.sf_out = out->src_flow;
        p.tf_out = out->snk_flow;
    }
    p.work = work;
    if ((e = launch_churn_resolve(p, h->stream)) != hipSuccess) return hip_fail(h, e, "churn re-solve launch");
    return GWTF_OK;
}

extern "C" gwtf_status_t gwtf_mcf_simulate_heuristic(gwtf_mcf_t *h, const gwtf_mcf_batch_t *b,
                                                     const gwtf_heur_config_t *cfg, const gwtf_heur_out_t *out)
{
    if (!h) return fail(nullptr, GWTF_ERR_INVALID_ARG, "handle is NULL");
    if (!b || !cfg) return fail(h, GWTF_ERR_INVALID_ARG, "batch or config is NULL");
    const int S = h->shape.num_stages, n = h->shape.nodes_per_stage;
    if (int64_t(S) * n > kHeurMaxNodes)
        return fail(h, GWTF_ERR_INVALID_ARG, "heuristic simulation needs S*n <= 64 (one lane per relay)");
    if (b->batch < 1 || b->batch > h->shape.max_batch)
        return fail(h, GWTF_ERR_INVALID_ARG, "batch outside [1, max_batch]");
    if (!b->node_cap || !b->node_cost || !b->supply || !b->flow_value || !b->total_cost || !b->status)
        return fail(h, GWTF_ERR_INVALID_ARG, "required pointer is NULL");
    if ((S > 1) != (b->arc_cost != nullptr))
        return fail(h, GWTF_ERR_INVALID_ARG, "arc_cost must be non-NULL exactly when S > 1");
    if (cfg->rounds < 0) return fail(h, GWTF_ERR_INVALID_ARG, "rounds must be >= 0");
    if (cfg->objective != GWTF_HEUR_SUM && cfg->objective != GWTF_HEUR_MAX)
        return fail(h, GWTF_ERR_INVALID_ARG, "objective must be GWTF_HEUR_SUM or GWTF_HEUR_MAX");
    if (!(cfg->t0 > 0.0) || !(cfg->t0 < 1e300) || !(cfg->alpha > 0.0) || !(cfg->alpha < 1e300))
        return fail(h, GWTF_ERR_INVALID_ARG, "t0 and alpha must be positive and finite");
    if (cfg->max_slots < 1 || cfg->max_slots > kHeurMaxSlots)
        return fail(h, GWTF_ERR_INVALID_ARG, "max_slots outside [1, 4096]");
    if (cfg->num_paths < 0 || (cfg->num_paths > 0) != (cfg->paths != nullptr))
        return fail(h, GWTF_ERR_INVALID_ARG, "paths must be non-NULL exactly when num_paths > 0");
    if (S == 1 && out && out->arc_flow)
        return fail(h, GWTF_ERR_INVALID_ARG, "arc_flow must be NULL when S == 1");
    hipError_t e = hipSetDevice(h->shape.device);
    if (e != hipSuccess) return hip_fail(h, e, "hipSetDevice");
    if (heuristic_lds_bytes(S, n, cfg->max_slots) > h->dev.lds_max)
        return fail(h, GWTF_ERR_INVALID_ARG, "max_slots too large for LDS");
    HeurParams p{};
    p.B = b->batch;
    p.S = S;
    p.n = n;
    p.rounds = cfg->rounds;
    p.objective = cfg->objective;
    p.max_slots = cfg->max_slots;
    p.num_paths = cfg->num_paths;
    p.t0 = cfg->t0;
    p.alpha = cfg->alpha;
    p.seed = cfg->seed;
    p.cap = b->node_cap;
    p.cost = b->node_cost;
    p.arc = b->arc_cost;
    p.src = b->src_cost;
    p.snk = b->snk_cost;
    p.supply = b->supply;
    p.paths = cfg->paths;
    p.F_out = b->flow_value;
    p.cost_out = b->total_cost;
    p.status_out = b->status;
    if (out) {
        p.node_flow = out->node_flow;
        p.arc_flow = out->arc_flow;
        p.used = out->used;
        p.accepted = out->accepted;
        p.temperature = out->temperature;
        p.counters = out->counters;
    }
    if ((e = launch_heuristic(p, h->stream)) != hipSuccess) return hip_fail(h, e, "heuristic simulation launch");
    return GWTF_OK;
}
