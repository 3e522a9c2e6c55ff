/*
 * gwtf_mcf.h -- C ABI of the batched min-cost max-flow solver for layered
 * pipeline-stage graphs, on AMD Instinct MI355X (gfx950).
 *
 * The problem (paper Sec. III system model, Sec. IV Eq. 1 and Sec. V-A
 * Eq. 2): a data node sends microbatches through S pipeline stages of n
 * relay nodes each and receives them back.  Node i holds at most cap_i
 * microbatches at a time (its memory, Sec. III) and costs c_i to run one;
 * sending from node i of stage k to node j of stage k+1 costs the delay
 * d(i, j).  One microbatch is one unit of flow (Sec. V-A).  The solver finds,
 * per instance, the most microbatches F the stages can carry
 * (capped by the data node's supply) and, among flows of that value, one of
 * minimum total cost sum f(i, j) * d(i, j) (Eq. 2).  Eq. 1's compute halves
 * summed along a microbatch's closed route equal the sum of the compute costs
 * of the nodes it visits, so each node's full compute cost is charged on the
 * node itself; a bandwidth term of Eq. 1 can be folded into arc_cost by the
 * caller.  The data node is both source and sink (Sec. V-A).
 *
 * All arrays passed to these calls are DEVICE pointers on the handle's GPU,
 * owned by the caller, C-contiguous, batch-major.  Integers only: int32
 * inputs, int64 flow value and cost.  All work is enqueued on the HIP stream
 * given to gwtf_mcf_create; calls return after enqueueing and outputs are
 * valid once the caller has synchronised that stream.  A handle serves one
 * stream and is not thread-safe; distinct handles are independent.
 */
#ifndef GWTF_MCF_H
#define GWTF_MCF_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct gwtf_mcf gwtf_mcf_t; /* opaque; owns its device workspace */

typedef enum {
    GWTF_OK = 0,
    GWTF_ERR_INVALID_ARG = 1,   /* bad pointer, shape or range; nothing enqueued */
    GWTF_ERR_OUT_OF_MEMORY = 2, /* workspace allocation failed */
    GWTF_ERR_DEVICE = 3,        /* a HIP runtime call failed; see gwtf_mcf_last_error */
    GWTF_ERR_NOT_SOLVED = 4,    /* gwtf_mcf_get_flows before any successful solve */
    GWTF_ERR_RANGE = 5          /* instance range outside the last solved batch */
} gwtf_status_t;

/* Per-instance status written to gwtf_mcf_batch_t.status. */
enum {
    GWTF_INST_OK = 0,
    GWTF_INST_BAD_INPUT = 1, /* a capacity, cost or supply < 0, or an arc cost < -1 */
    GWTF_INST_OVERFLOW = 2,  /* (2*S*n + 3) * max cost >= 2^29: labels could leave int32 */
    GWTF_INST_NOT_CONVERGED = 3 /* churn re-solve only: its final augmenting phase stopped at
                                   the safety limit of 2^20 label-correcting rounds (not
                                   expected on valid input) */
};

/* Solver pass that produced an instance's result (gwtf_mcf_get_passes). */
enum {
    GWTF_PASS_REGISTER = 1, /* one workgroup, link costs in registers: 16 < n <= 64, S <= 32 */
    GWTF_PASS_LDS = 2,      /* one workgroup, instance state in LDS: n <= 64 */
    GWTF_PASS_GRID = 3,     /* each instance over S * ceil(n/128) co-resident workgroups: 64 < n <= 512, or 16 < n <= 64 with S > 32 in small batches */
    GWTF_PASS_GLOBAL = 4,   /* one workgroup, instance state in device memory: any shape */
    GWTF_PASS_PACKED = 5    /* 1 to 8 instances per wave (8 only for n <= 8): S <= 8, supply <= 255, costs <= 2047 */
};

/* arc_cost entry meaning "these two nodes share no link". */
#define GWTF_NO_ARC (-1)

typedef struct {
    int32_t num_stages;      /* S >= 1 */
    int32_t nodes_per_stage; /* n >= 1 (a stage with fewer nodes pads with cap 0) */
    int32_t max_batch;       /* largest batch a solve may pass, >= 1 */
    int32_t device;          /* HIP device ordinal the handle works on */
} gwtf_mcf_shape_t;

typedef struct {
    int32_t batch;           /* B, 1 <= B <= max_batch */
    const int32_t *node_cap; /* [B][S][n] >= 0; 0 = node absent (crashed / left) */
    const int32_t *node_cost;/* [B][S][n] >= 0: compute cost c_i of one microbatch */
    const int32_t *arc_cost; /* [B][S-1][n][n]: [b][k][i][j] = delay from node i of stage k
                                to node j of stage k+1, >= 0 or GWTF_NO_ARC; NULL iff S == 1 */
    const int32_t *src_cost; /* [B][n] data node -> stage-0 node delay, >= 0; NULL = all 0 */
    const int32_t *snk_cost; /* [B][n] stage-(S-1) node -> data node delay, >= 0; NULL = all 0 */
    const int32_t *supply;   /* [B] >= 0: microbatches the data node injects */
    int64_t *flow_value;     /* [B] out: F */
    int64_t *total_cost;     /* [B] out: sum over arcs of flow * cost (Eq. 2) */
    int32_t *status;         /* [B] out: GWTF_INST_*; a bad instance reports F = cost = 0 */
} gwtf_mcf_batch_t;

/* Creates a solver for batches of `shape` on shape->device, enqueueing on
 * `hip_stream` (a hipStream_t; NULL = the device's null stream).  Allocates
 * the workspace (flows, potentials, fallback state) for shape->max_batch
 * instances.  *out receives the handle, or NULL on failure. */
gwtf_status_t gwtf_mcf_create(const gwtf_mcf_shape_t *shape, void *hip_stream, gwtf_mcf_t **out);

/* Solves every instance of the batch (paper Eq. 2 optimum per instance).
 * Argument errors return GWTF_ERR_INVALID_ARG with nothing enqueued; input
 * values are checked on the device and reported per instance in status.
 * Results are deterministic: the same inputs give the same flows. */
gwtf_status_t gwtf_mcf_solve_batch(gwtf_mcf_t *h, const gwtf_mcf_batch_t *b);

/* Copies the optimal flow of instances [first, first + count) of the last
 * solved batch into caller device buffers (any may be NULL):
 *   node_flow [count][S][n]        microbatches through each node
 *   arc_flow  [count][S-1][n][n]   microbatches on each inter-stage link
 *   src_flow  [count][n]           data node -> stage-0 node
 *   snk_flow  [count][n]           stage-(S-1) node -> data node
 *   potential [count][2*S*n + 3]   node potentials certifying optimality: every
 *       arc with spare capacity has cost + pi(tail) - pi(head) >= 0.  Vertex
 *       order: 0 = source root s0, 1 = data node as source s, 2 = data node as
 *       sink t, 3 + 2*(k*n + i) = node (k, i) entry, 4 + 2*(k*n + i) = its exit
 *       (the node's compute arc runs entry -> exit; the root s0 -> s arc holds
 *       the supply). */
gwtf_status_t gwtf_mcf_get_flows(gwtf_mcf_t *h, int32_t first, int32_t count,
                                 int32_t *node_flow, int32_t *arc_flow,
                                 int32_t *src_flow, int32_t *snk_flow, int32_t *potential);

/* Per-instance work counters of the last solve, into a caller device buffer
 * stats[count][10] (int64): augmenting paths, label-correcting rounds, cost
 * rows relaxed in the dense relaxation (each row is n arc relaxations),
 * flow-list (reverse-arc) relaxations, the nanoseconds the instance's
 * workgroup spent in forward sweeps, backward sweeps, augmentation with the
 * potential update, and the rest (label reset, sink update), then the
 * executed forward and backward layer steps (0 where not tracked).  For
 * instances of the grid pass (GWTF_PASS_GRID) the clocks are workgroup 0's:
 * label iterations, then 0, then the potential update with the path walks
 * and augmentations of a search (tied exits included), then the rest (label
 * resets, barriers); column 8 counts the shortest-path searches. */
gwtf_status_t gwtf_mcf_get_stats(gwtf_mcf_t *h, int32_t first, int32_t count, int64_t *stats);

/* Which solver pass produced each instance of the last solve, into a caller
 * device buffer pass[count] (int32, GWTF_PASS_*).  The pass follows from the
 * handle's shape, except that an instance whose link costs exceed 65534 or
 * whose flow lists outgrow LDS, or one outside GWTF_PASS_PACKED's bounds,
 * moves to GWTF_PASS_GLOBAL.  Enqueued on the
 * handle's stream; errors as for gwtf_mcf_get_stats. */
gwtf_status_t gwtf_mcf_get_passes(gwtf_mcf_t *h, int32_t first, int32_t count, int32_t *pass);

/* ---- Solve without allocation ----
 *
 * For callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.  The same
 * solve as gwtf_mcf_solve_batch (same passes, checks, per-instance status and
 * outputs), with no handle: every workspace buffer lives in one fixed array
 * of 64 MiB per device, declared in the library, that each device holds from
 * the first call on it until the process ends.  The call allocates nothing
 * (no hipMalloc, hipFree or other allocating routine).
 *
 * `shape` gives S, n and the device (max_batch bounds b->batch as for a
 * handle); the batch and its outputs are as for gwtf_mcf_solve_batch, on the
 * HIP stream `hip_stream` (NULL = the device's null stream).  A batch whose
 * workspace does not fit in the array gives GWTF_ERR_INVALID_ARG with nothing
 * enqueued, and gwtf_mcf_last_error(NULL) names the bytes it needs: about
 * 6,600 instances of 8 x 8 or 34 of 32 x 64 fit (larger batches are solved
 * in slices), and one 64 x 512 instance (about 223 MiB) does not.  Every call on a device shares that device's array and
 * leaves its contents behind: calls that overlap in time on one device (two
 * streams, or two host threads) race and give wrong results, so they must be
 * serialised by the caller.  Flows, stats and passes of these solves are
 * not kept (gwtf_mcf_get_flows needs a handle).  Errors are reported through
 * gwtf_mcf_last_error(NULL) of the calling thread. */
gwtf_status_t gwtf_mcf_solve_batch_noalloc(const gwtf_mcf_shape_t *shape, void *hip_stream,
                                           const gwtf_mcf_batch_t *b);

/* ---- Location-factored instances (paper Sec. VI testbed: every node sits at
 * one of a few geographic locations, and Eq. 1's link term is the latency
 * between the two nodes' locations) ----
 *
 * A located batch stands for the ordinary batch whose link from node i of
 * stage k to node j of stage k+1 has delay
 * latency[b][location[b][k][i]][location[b][k+1][j]]; the result is exactly
 * that batch's (gwtf_mcf_solve_batch semantics, every link present).  The
 * grid pass (64 < n <= 512) relaxes the links in factored form: per
 * location, the best label among the previous stage's nodes there, then per
 * node one candidate per location, L operations instead of n.  Other shapes
 * expand the delays into library workspace on the device and run the
 * ordinary passes. */
typedef struct {
    int32_t batch;            /* B, 1 <= B <= max_batch */
    int32_t num_locations;    /* L, 1 <= L <= 32 */
    const int32_t *node_cap;  /* [B][S][n] >= 0 */
    const int32_t *node_cost; /* [B][S][n] >= 0 */
    const int32_t *location;  /* [B][S][n] in [0, L) */
    const int32_t *latency;   /* [B][L][L] >= 0: [a][c] = delay from location a to location c */
    const int32_t *src_cost;  /* [B][n] or NULL = 0 */
    const int32_t *snk_cost;  /* [B][n] or NULL = 0 */
    const int32_t *supply;    /* [B] >= 0 */
    int64_t *flow_value;      /* [B] out */
    int64_t *total_cost;      /* [B] out */
    int32_t *status;          /* [B] out; with S > 1, a location outside [0, L) or a negative
                                 latency gives GWTF_INST_BAD_INPUT (S == 1 reads neither) */
} gwtf_mcf_located_batch_t;

/* Solves a located batch; argument errors and status as for
 * gwtf_mcf_solve_batch, and gwtf_mcf_get_flows / get_stats / get_passes then
 * refer to it (for instances of the factored grid pass, stats column 2
 * counts the factored relaxation operations divided by n).  The first call
 * on a handle with S > 1 allocates max_batch * (S-1) * n * n int32 of
 * workspace for the expanded delays, which every pass but the factored one
 * reads (GWTF_ERR_OUT_OF_MEMORY if that fails). */
gwtf_status_t gwtf_mcf_solve_located(gwtf_mcf_t *h, const gwtf_mcf_located_batch_t *b);

/* ---- What-if node addition (paper Sec. VI, handling joining nodes; the
 * joining example of Sec. V-B) ----
 *
 * The paper places joining nodes by solving the flow problem once for every
 * way of assigning the candidate nodes to stages and keeping the best
 * assignment.  These calls build that batch of instances on the device
 * (gwtf_mcf_whatif_expand), leave the solve to gwtf_mcf_solve_batch, and
 * reduce its results to the best placement (gwtf_mcf_whatif_best).
 *
 * A placement sends each of m candidates to a different stage (0 <= m <= S);
 * placements are numbered 0 .. S!/(S-m)! - 1 in lexicographic order of
 * (stage of candidate 0, stage of candidate 1, ...).  Placement p is the
 * base instance with, in every stage k that receives candidate c, node
 * position `slot` replaced by c: its capacity cap[c][k], compute cost
 * cost[c][k], links in_cost[c][k][i] from node i of stage k-1 and
 * out_cost[c][k][j] to node j of stage k+1, link_cost[c][d] to candidate d
 * when d sits in stage k+1, and src_cost[c] / snk_cost[c] to the data node
 * when k is 0 / S-1.  Stages without a candidate keep the base's node at
 * `slot` (an empty position has capacity 0). */
typedef struct {
    int32_t num_candidates;   /* m, 0 <= m <= S, with S!/(S-m)! < 2^63 */
    int32_t slot;             /* node position a candidate takes, 0 <= slot < n */
    const int32_t *cap;       /* [m][S] capacity if the candidate joins stage k (NULL iff m == 0) */
    const int32_t *cost;      /* [m][S] compute cost if it joins stage k (NULL iff m == 0) */
    const int32_t *in_cost;   /* [m][S][n] delay from node i of stage k-1 (row k = 0 unread);
                                 NULL iff S == 1 or m == 0 */
    const int32_t *out_cost;  /* [m][S][n] delay to node j of stage k+1 (row k = S-1 unread);
                                 NULL iff S == 1 or m == 0 */
    const int32_t *link_cost; /* [m][m] delay from candidate c to candidate d one stage later;
                                 NULL iff S == 1 or m == 0 */
    const int32_t *src_cost;  /* [m] data node -> candidate in stage 0; NULL = all 0 */
    const int32_t *snk_cost;  /* [m] candidate in stage S-1 -> data node; NULL = all 0 */
} gwtf_whatif_candidates_t;

/* Caller device buffers for `count` instances in the canonical layout
 * ([count][S][n] node_cap and node_cost, [count][S-1][n][n] arc_cost (NULL
 * iff S == 1), [count][n] src_cost and snk_cost, [count] supply). */
typedef struct {
    int32_t *node_cap, *node_cost, *arc_cost, *src_cost, *snk_cost, *supply;
} gwtf_mcf_instances_t;

/* Host-only: *count = S!/(S-m)!, the number of placements of m candidates
 * over S stages.  GWTF_ERR_INVALID_ARG if S < 1, m < 0, m > S, count is
 * NULL, or the number does not fit in an int64. */
gwtf_status_t gwtf_whatif_count(int32_t num_stages, int32_t num_candidates, int64_t *count);

/* Writes placements [first, first + count) into `out` (instance r of `out`
 * is placement first + r).  `base` is one instance in the batch layout of the
 * handle's shape (batch must be 1; src_cost / snk_cost may be NULL = 0; the
 * output fields flow_value, total_cost and status are not used).  Values are
 * copied as they are: an invalid value reaches the solve, which reports it in
 * that instance's status.  Requires S <= 1024 and count >= 0; first + count
 * must not exceed the placement count (GWTF_ERR_RANGE otherwise); with
 * count == 0 nothing is written and the `out` pointers may be NULL.  All other
 * argument errors give GWTF_ERR_INVALID_ARG with nothing enqueued.  Enqueued
 * on the handle's stream; `out` must not overlap any input. */
gwtf_status_t gwtf_mcf_whatif_expand(gwtf_mcf_t *h, const gwtf_mcf_batch_t *base,
                                     const gwtf_whatif_candidates_t *cand, int64_t first,
                                     int32_t count, const gwtf_mcf_instances_t *out);

/* Best placement among `count` solved instances (device arrays, as written
 * by gwtf_mcf_solve_batch for an expanded batch): among instances with status
 * GWTF_INST_OK, the largest flow value, then the smallest cost, then the
 * smallest index.  best (device, int64[3]) receives {first + index, F, cost},
 * or {-1, 0, 0} when no instance is OK.  With merge != 0 the call keeps the
 * better of that and what best already holds (same order; an entry with
 * index -1 loses), so chunks of one placement range can be reduced in turn.
 * count >= 0; errors as for gwtf_mcf_whatif_expand. */
gwtf_status_t gwtf_mcf_whatif_best(gwtf_mcf_t *h, int32_t count, const int64_t *flow_value,
                                   const int64_t *total_cost, const int32_t *status, int64_t first,
                                   int32_t merge, int64_t *best);

/* ---- Warm-started re-solve after churn (paper Sec. VI: nodes join and
 * leave between iterations; re-solving from the previous optimum instead of
 * from zero is this library's extension, the paper does not describe it) ----
 *
 * Solves every instance of `b` (same layout, checks and per-instance status
 * as gwtf_mcf_solve_batch; b->batch <= max_batch) starting from a feasible
 * flow of the same shape instead of from zero, typically the optimum of the
 * instance before the churn as returned by gwtf_mcf_get_flows.  The result
 * (F, cost) equals a cold solve's: the start flow loses whole source-to-sink
 * paths until it respects the new capacities, the missing links and the
 * supply; negative residual cycles are cancelled (the flow is then of least
 * cost for its value); shortest augmenting paths finish the solve.  Should
 * the cancelling stop at its safety limit of 2^20 label-correcting rounds,
 * the instance restarts from the zero flow, which is the cold solve.
 *
 * The start flow is in the layout of gwtf_mcf_get_flows: node_flow
 * [.][S][n], arc_flow [.][S-1][n][n] (NULL iff S == 1), src_flow and
 * snk_flow [.][n], with one entry for the whole batch when per_instance == 0
 * and one per instance otherwise.  It must be conserved (a node's flow equals
 * its inflow and its outflow; stage 0 is fed by src_flow, stage S-1 drains
 * into snk_flow) with every value in [0, 2^29) and a value (sum of src_flow)
 * below 2^29; otherwise the instance gets GWTF_INST_BAD_INPUT.  Its capacities and links need not match the new
 * instance. */
typedef struct {
    const int32_t *node_flow, *arc_flow, *src_flow, *snk_flow;
    int32_t per_instance;
} gwtf_mcf_flow_in_t;

/* Caller device buffers for result flows of `batch` instances, in the same
 * layout (arc_flow NULL iff S == 1). */
typedef struct {
    int32_t *node_flow, *arc_flow, *src_flow, *snk_flow;
} gwtf_mcf_flow_out_t;

/* One workgroup per instance holds the instance in LDS: requires S*n <= 512
 * and (S-1)*n*n <= 4096 (GWTF_ERR_INVALID_ARG otherwise, nothing enqueued).
 * `out` may be NULL (no flows written; an instance that is not OK gets zero
 * flows).  `work` (device int64 [batch][4], or NULL) receives per instance
 * the paths removed, cycles cancelled, augmentations and label-correcting
 * rounds.  Uses no handle workspace: gwtf_mcf_get_flows keeps referring to
 * the last gwtf_mcf_solve_batch.  Enqueued on the handle's stream. */
gwtf_status_t gwtf_mcf_resolve_churn(gwtf_mcf_t *h, const gwtf_mcf_batch_t *b,
                                     const gwtf_mcf_flow_in_t *start,
                                     const gwtf_mcf_flow_out_t *out, int64_t *work);

/* ---- Simulation of the decentralized flow heuristic (paper Sec. V-C:
 * Request Flow, Request Change and Request Redirect with simulated
 * annealing; Sec. VI setup: T0 = 1.7, alpha = 0.95) ----
 *
 * Runs the paper's decentralized routing heuristic on every instance of a
 * batch for a number of synchronous rounds, so that its result can be scored
 * against the exact optimum of gwtf_mcf_solve_batch on the same instances
 * (the flow ablation of Sec. VI).  Relay (k, i) holds cap[k][i] slots, one
 * per microbatch; each round:
 *   1. every relay computes, from the last stage to the first, the cost to
 *      the sink of each of its outflows (compute cost + link + the next
 *      hop's cost to the sink);
 *   2. Request Flow: a relay with no unpaired outflow and a free slot asks
 *      the next-stage relay whose unpaired outflow minimises (its cost to
 *      the sink + the link cost), lowest index on ties; a relay asked by
 *      several approves the lowest-index one, the data node as sink approves
 *      last-stage requesters in index order while it has flow left (it
 *      starts with `supply`), and the data node as source pairs first-stage
 *      unpaired outflows, cheapest first, while it has flow left;
 *   3. improvement: stages of even index, then odd ones, are shuffled and
 *      split into pairs; a proposer that made no request this round draws a
 *      Request Redirect (carrying one of its partner's paired flows itself,
 *      if it has a free slot) or a Request Change (swapping the next hops of
 *      one flow each) and takes it when exp((cost_cur - cost_new) / T) >
 *      U(0, 1); costs are the Eq. 1 costs of the changed links, summed
 *      (GWTF_HEUR_SUM, Eq. 2) or maximised (GWTF_HEUR_MAX, the local max
 *      objective of Sec. V-A); each accepted move multiplies the proposer's
 *      temperature by alpha.
 * Random numbers are Philox4x64-10 with key (seed, instance index) and
 * counter (round, stage, 0, block) for a stage's shuffle and (round, stage,
 * 1, pair) for a pair's four draws: the same inputs and seed give the same
 * result.
 *
 * Result: the complete paths (data node -> one relay per stage -> data node)
 * present after the last round.  b->flow_value receives their number,
 * b->total_cost their summed cost (Eq. 2, the exact solver's objective) and
 * b->status the instance status (GWTF_INST_BAD_INPUT as for the solver, or a
 * total capacity above max_slots, or an invalid initial path;
 * GWTF_INST_OVERFLOW when (2S + 2) * the largest cost >= 2^30).  Requires
 * S * n <= 64 (one lane per relay, one wave per instance); every input array
 * is a device pointer in the layout of gwtf_mcf_solve_batch.  Uses no handle
 * workspace; enqueued on the handle's stream. */
enum { GWTF_HEUR_SUM = 0, GWTF_HEUR_MAX = 1 };

typedef struct {
    int32_t rounds;        /* synchronous rounds, >= 0 (the paper runs at most 120) */
    int32_t objective;     /* GWTF_HEUR_SUM or GWTF_HEUR_MAX */
    double t0, alpha;      /* initial temperature and cooling factor, > 0 */
    uint64_t seed;         /* Philox key word 0 */
    int32_t max_slots;     /* bound on an instance's total capacity, 1..4096 (sizes LDS) */
    int32_t num_paths;     /* P >= 0: initial complete paths per instance */
    const int32_t *paths;  /* [B][P][S] device, node index per stage (rows starting
                              with -1 unused), NULL iff P == 0: the flow starts with
                              these paths, each node taking its lowest free slot */
} gwtf_heur_config_t;

/* Optional per-instance outputs (device pointers, any may be NULL). */
typedef struct {
    int32_t *node_flow;    /* [B][S][n] complete paths through each relay */
    int32_t *arc_flow;     /* [B][S-1][n][n] complete paths on each link (NULL iff S == 1) */
    int32_t *used;         /* [B][S][n] slots in use, incomplete chains included */
    int32_t *accepted;     /* [B][S][n] moves each relay proposed and had accepted */
    double *temperature;   /* [B][S][n] final temperature of each relay */
    int64_t *counters;     /* [B][4]: paths the data node paired, Request Flow approvals,
                              accepted moves, slots in incomplete chains */
} gwtf_heur_out_t;

gwtf_status_t gwtf_mcf_simulate_heuristic(gwtf_mcf_t *h, const gwtf_mcf_batch_t *b,
                                          const gwtf_heur_config_t *cfg, const gwtf_heur_out_t *out);

/* Frees the handle and its workspace after draining its stream; NULL-safe. */
/* ---- Hand-off latency calibration ----
 *
 * Measures on `device` the least time one hop of the stage pipelines can
 * take: the shortest paths of Sec. V-A are computed by passing labels from
 * each stage's owner to the next stage's owner, and the register and grid
 * passes each wait for such a hand-off per pipeline hop.  Runs three
 * ping-pongs of 2000 round trips each, with nothing else around them, and
 * writes the one-way latency in nanoseconds (half a round trip) to the HOST
 * array latency_ns[3]:
 *   [0] one wave to another of the same workgroup through LDS (the register
 *       pass's mailboxes);
 *   [1] workgroup 0 to workgroup `block_distance` of one launch of 16
 *       one-wave workgroups through device-scope atomic loads and stores (the grid pass's label
 *       words; its neighbouring stages are `ceil(n/128)` workgroups apart);
 *   [2] workgroup 0 to workgroup 8 (on the same XCD when workgroups are
 *       dealt round robin over 8 XCDs).
 * An entry is -1 if its bounded wait ran out.  Enqueued on hip_stream (NULL
 * = the null stream), which it synchronises before returning; it allocates
 * and frees 1 KB of device memory.  Errors: GWTF_ERR_INVALID_ARG for a NULL
 * array, a bad device ordinal or block_distance outside [1, 15] or equal to
 * 8; GWTF_ERR_DEVICE if a HIP call fails (text in gwtf_mcf_last_error(NULL)
 * of the calling thread). */
gwtf_status_t gwtf_mcf_calibrate_handoff(int32_t device, void *hip_stream, int32_t block_distance,
                                         double *latency_ns);

void gwtf_mcf_destroy(gwtf_mcf_t *h);

/* Text of the last error on this handle ("" if none); NULL handle gives the
 * last error of a call made without a handle (gwtf_mcf_create,
 * gwtf_mcf_solve_batch_noalloc, or one given a NULL handle) on the calling
 * thread. */
const char *gwtf_mcf_last_error(const gwtf_mcf_t *h);

#ifdef __cplusplus
}
#endif
#endif /* GWTF_MCF_H */
