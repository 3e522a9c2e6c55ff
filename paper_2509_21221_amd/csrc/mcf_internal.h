// Internal interface between the host API (mcf_api.hip) and the solver
// kernels.  Not part of the public C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace gwtf {

// Sentinel label for "not reached"; every finite label stays below 2^29 in
// magnitude (the per-instance overflow check guarantees it), so sums of a
// finite label and a cost never reach kInf.
constexpr int32_t kInf = 0x3fffffff;
constexpr int64_t kLabelBound = int64_t(1) << 29;

// Route codes in the workspace: an instance waiting for the fallback pass,
// or the pass that finished it (the public GWTF_PASS_* values).
enum : int32_t { kRouteFallback = -1, kRouteReg = 1, kRouteLds = 2, kRouteGrid = 3, kRouteGlobal = 4, kRouteSmall = 5 };
// between the two launches of the pipelined pass only: the unscaled variant
// solves the instance
constexpr int32_t kRoutePipeWide = 6;

// Kernel arguments shared by both solver passes.
struct SolveParams {
    int32_t B, S, n;
    const int32_t *cap, *ncost, *acost, *src, *snk, *supply; // caller inputs
    int64_t *F_out, *cost_out;                                 // caller outputs [B]
    int32_t *status_out;                                       // [B]
    int32_t *route;       // [B] kRoute*
    int32_t *node_flow;   // [B][S][n]
    int32_t *arc_flow;    // [B][S-1][n][n]
    int32_t *pot;         // [B][2Sn+3]; entry potentials live here during the solve
    int64_t *stats;       // [B][kStatsPerInstance]
    unsigned char *state; // fallback pass: per-instance state, state_stride bytes each
    size_t state_stride;
    int64_t list_slots;   // flow-list capacity of one instance
    int32_t route_all;    // fallback pass: solve every instance, ignoring route[]
    int32_t clock_khz;    // device wall-clock rate, for the phase timers
};

// Per-instance counters written to SolveParams::stats: augmentations,
// label-correcting rounds, dense cost rows relaxed, flow-list relaxations,
// then nanoseconds spent in forward sweeps, backward sweeps, augmentation
// with the potential update, and the remainder (label reset, sink update),
// then executed forward and backward layer steps (register pass only).
constexpr int kStatsPerInstance = 10;

// Byte offsets of the per-instance solver state.  The LDS-resident pass uses
// narrow index types (n <= 64); the fallback pass keeps the state in global
// memory with wider ones.
struct StateLayout {
    size_t din, dout, pout, flow, cap, cost, pend, srcc, snkc;
    size_t prin, prout, loff, llen, lcost, lamt, lpart;
    size_t total;
};

__host__ __device__ inline size_t align16(size_t x) { return (x + 15) & ~size_t(15); }

__host__ __device__ inline StateLayout make_layout(int S, int n, int64_t slots, bool narrow)
{
    StateLayout L;
    size_t SN = size_t(S) * n, nw = (size_t(n) + 63) / 64, o = 0;
    auto take = [&](size_t bytes) { size_t at = o; o = align16(o + bytes); return at; };
    L.din = take(4 * SN);
    L.dout = take(4 * SN);
    L.pout = take(4 * SN);
    L.flow = take(4 * SN);
    L.cap = take(4 * SN);
    L.cost = take(4 * SN);
    L.pend = take(8 * size_t(S) * nw);
    L.srcc = take(4 * size_t(n));
    L.snkc = take(4 * size_t(n));
    L.prin = take((narrow ? 1 : 2) * SN);
    L.prout = take((narrow ? 1 : 2) * SN);
    L.loff = take((narrow ? 2 : 4) * SN);
    L.llen = take((narrow ? 1 : 2) * SN);
    // Lists carry 64 slots of slack so batched reads past the last list
    // stay inside the allocation.
    const size_t lslots = size_t(slots) + 64;
    L.lcost = take(4 * lslots);
    L.lamt = take(4 * lslots);
    L.lpart = take((narrow ? 1 : 2) * lslots);
    L.total = o;
    return L;
}

// LDS needed besides the state: per-wave partial minima and a scan buffer.
__host__ __device__ inline size_t scratch_bytes(int waves, int n)
{
    return align16(size_t(8) * waves * n) + align16(size_t(4) * waves * 64);
}

// Launchers (mcf_solver.hip).  Return the HIP launch status.
hipError_t launch_lds_pass(const SolveParams &p, int waves, size_t lds_bytes, hipStream_t s);
hipError_t launch_fallback_pass(const SolveParams &p, size_t lds_bytes, hipStream_t s);
hipError_t launch_export(const int32_t *node_flow_ws, int32_t S, int32_t n, int32_t first, int32_t count,
                         int32_t *src_flow, int32_t *snk_flow, hipStream_t s);
// What-if expansion (mcf_whatif.hip): the base instance, the candidates
// and the output batch, all device pointers in the canonical layouts.
constexpr int kWhatifMaxStages = 1024;
struct WhatifExpandParams {
    int32_t S, n, m, slot;
    int64_t first;
    const int32_t *cap, *cost, *arc, *src, *snk, *supply;                 // base [1][...]
    const int32_t *ccap, *ccost, *cin, *cout, *clink, *csrc, *csnk;       // candidates
    int32_t *out_cap, *out_cost, *out_arc, *out_src, *out_snk, *out_supply; // [count][...]
};
hipError_t launch_whatif_expand(const WhatifExpandParams &p, int32_t count, hipStream_t s);
hipError_t launch_whatif_best(int32_t count, const int64_t *F, const int64_t *cost, const int32_t *status,
                              int64_t first, int32_t merge, int64_t *best, hipStream_t s);
// Located instances (mcf_located.hip): the implied dense link delays
// arc[b][k][i][j] = lat[b][loc[b][k][i]][loc[b][k+1][j]], -2 where invalid.
hipError_t launch_located_expand(int32_t B, int32_t S, int32_t n, int32_t L, const int32_t *loc,
                                 const int32_t *lat, int32_t *arc, hipStream_t s);
int fallback_waves();
hipError_t set_lds_limits(size_t max_bytes);

// Warm-started re-solve of churn variants (mcf_churn.hip): one workgroup per
// instance with the instance in LDS, so S*n <= kChurnMaxNodes and
// (S-1)*n*n <= kChurnMaxLinks.
constexpr int kChurnMaxNodes = 512;
constexpr int kChurnMaxLinks = 4096;
struct ChurnParams {
    int32_t B, S, n, start_per_instance;
    const int32_t *cap, *ncost, *acost, *src, *snk, *supply; // caller inputs
    const int32_t *nf0, *af0, *sf0, *tf0;                    // start flow ([B] or [1])
    int64_t *F_out, *cost_out;                               // [B]
    int32_t *status_out;                                     // [B]
    int32_t *nf_out, *af_out, *sf_out, *tf_out;              // result flows, or all NULL
    int64_t *work;                                           // [B][4] or NULL
};
size_t churn_lds_bytes(int S, int n);
hipError_t launch_churn_resolve(const ChurnParams &p, hipStream_t stream);

// Simulation of the decentralized flow heuristic (mcf_heuristic.hip): one
// wave per instance, one lane per relay, so S*n <= kHeurMaxNodes; at most
// kHeurMaxSlots slots (units of capacity) per instance.
constexpr int kHeurMaxNodes = 64;
constexpr int kHeurMaxSlots = 4096;
struct HeurParams {
    int32_t B, S, n, rounds, objective, max_slots, num_paths;
    double t0, alpha;
    uint64_t seed;
    const int32_t *cap, *cost, *arc, *src, *snk, *supply; // caller inputs
    const int32_t *paths;                                 // [B][num_paths][S] or NULL
    int64_t *F_out, *cost_out;                            // [B]
    int32_t *status_out;                                  // [B]
    int32_t *node_flow, *arc_flow, *used, *accepted;      // optional outputs
    double *temperature;                                  // optional [B][S][n]
    int64_t *counters;                                    // optional [B][4]
};
size_t heuristic_lds_bytes(int S, int n, int max_slots);
hipError_t launch_heuristic(const HeurParams &p, hipStream_t stream);

// Hand-off latency calibration (mcf_calibrate.hip): one-way latencies in
// ns of an LDS hand-off between two waves, and of device-scope hand-offs
// between workgroups 0 and `neighbour` and between workgroups 0 and 8 of one
// cooperative launch; -1 where a bounded wait ran out.  Synchronises `s`.
hipError_t run_handoff_calibration(hipStream_t s, int clock_khz, int neighbour, double out_ns[3]);

} // namespace gwtf
