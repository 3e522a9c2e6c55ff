// Internal interface of the grid-cooperative pass (mcf_solver_grid.hip):
// each instance over S * ceil(n / 128) co-resident workgroups, as many
// instances per launch as fit at once, for 64 < n <= 512.  Not part of the
// public C ABI.
#pragma once

#include "mcf_internal.h"

namespace gwtf {

constexpr int kGridCtrlInts = 1280;    // control block: flags, barrier, per-iteration words, tied exits
constexpr int kGridMaxBlocks = 512;    // workgroups of one instance (the barrier's group counters)
constexpr int kGridMaxConcurrent = 64; // instances of one grid launch
// Ring slots and their sink keys sit 128 bytes apart: every workgroup adds
// its arrival to a slot each iteration, and atomics on one line serialize.
constexpr int kRingStride = 32, kRingKeyStride = 16;
constexpr int kGridMaxNodes = 512;     // a stage's labels are staged with one thread per node
constexpr size_t kGridStaticLds = 512; // static LDS of the grid kernel (upper bound)
struct GridParams {
    SolveParams base;
    int32_t instance;   // first instance solved by this launch
    int32_t count;      // instances solved by this launch, S * slices workgroups each
    int32_t slices;     // workgroups per stage
    int64_t list_slots; // flow-list capacity of one workgroup
    size_t big_bytes;   // leading LDS area: link-cost block or staged predecessors
    // per instance of the launch, one after another:
    uint32_t *ex, *en;  // [2][S*n] exit / entry labels << 2 | iteration tag, by iteration parity
    uint32_t *ring;     // [ring_slots * kRingStride] per-iteration arrivals (low 16 bits) and changed count
    unsigned long long *ring_key; // [ring_slots * kRingKeyStride] per-iteration minimum sink key
    int32_t ring_slots; // > S + 2: iterations in flight at once across the stages
    int32_t *pred;      // [S*n] entry predecessor (low 16 bits) and exit predecessor (high)
    int32_t *path;      // [2*S*n + 8] arc codes of the augmenting path
    int32_t *ctrl;      // [kGridCtrlInts], cleared before each launch
    // Location-factored links (NULL loc = dense link costs): the link from
    // node i of stage k to node j of stage k+1 costs
    // lat[loc[k][i]][loc[k+1][j]].
    const int32_t *loc; // [B][S][n] in [0, L)
    const int32_t *lat; // [B][L][L]
    int32_t L;          // 1 <= L <= kGridMaxLocations
};
constexpr int kGridMaxLocations = 32;
inline int grid_ring_slots(int S) { return S + 8; }
size_t grid_pass_big_bytes(int S, int n);
size_t grid_pass_lds_bytes(int S, int n, int64_t list_slots);
int64_t grid_pass_list_slots(int S, int n, size_t lds_max);
int grid_pass_slices(int n);
int grid_pass_blocks_per_cu(size_t lds_bytes);
hipError_t launch_grid_pass(const GridParams &gp, size_t lds_bytes, hipStream_t s);

} // namespace gwtf
