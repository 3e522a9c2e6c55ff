/*
 * gwtf_heuristic.c -- reference CPU simulator of GWTF's decentralized flow
 * heuristic, for scoring it against the exact optimum.
 *
 * TEST INFRASTRUCTURE ONLY.  This is the plain, slow, obviously correct
 * simulator that the GPU simulator is checked against.  Only the test suite
 * and the benchmark's CPU-baseline leg may load it; the product path never
 * does.  It shares no code, header or table with the GPU library.
 *
 * The protocol (paper Sec. V-C, "Building Pipelines using Flow Requests"),
 * as read here; every point the paper leaves open is marked READING.
 *
 * Network: S stages of n relay nodes and one data node D that is both the
 * source and the sink of every microbatch (Sec. V-A).  Relay v = (k, i) has
 * capacity cap[k][i] (microbatches in memory, Sec. III) and compute cost
 * c[k][i]; the link from (k, i) to (k+1, j) costs arc[k][i][j] (-1 = no
 * link); D -> (0, i) costs src[i] and (S-1, i) -> D costs snk[i].
 *
 * State: relay v owns cap_v slots, one per microbatch it can hold.  A used
 * slot has an outflow (the next hop's slot, or D as sink) and, once paired,
 * an inflow (the previous hop's slot, or D as source).  A used slot without
 * inflow is an unpaired outflow (Sec. V-C: the node wants to receive).  A
 * slot's cost to the sink is its node's compute cost plus the link to the
 * next hop plus the next slot's cost to the sink, computed from the last
 * stage to the first (Sec. V-C).  D starts with `supply` unpaired flows on
 * each side (Sec. V-C: data nodes start with unpaired flows matching their
 * capacity).  Every used slot counts against capacity, paired or not (Sec.
 * V-C: sending outflow reduces capacity even if unpaired).
 *
 * READING (rounds): the simulation runs in synchronous rounds ("iterations"
 * of the algorithm, Sec. V-C and the flow ablation of Sec. VI).  Each round
 * has a Request Flow phase, then an improvement phase; every choice in a
 * phase reads the state at the start of that phase or step.
 *
 * Request Flow phase:
 *   - A relay with no unpaired outflow and a free slot is a requester
 *     (Sec. V-C: nodes with available capacity in a stable state; nodes at
 *     capacity make no request).  It picks, among the next stage's relays
 *     with an unpaired outflow and a link to them, the one minimising that
 *     outflow's cost to the sink plus the link cost (Sec. V-C); in the last
 *     stage the only candidate is D as sink, while D has unpaired flows left.
 *     READING: ties go to the lowest node index; a relay with no candidate
 *     is not a requester.
 *   - A relay asked by several requesters approves one (Sec. V-C: only one
 *     can connect to its single unpaired outflow; the others are rejected
 *     and retry).  READING: the lowest requester index wins.  D as sink
 *     approves last-stage requesters in index order while it has unpaired
 *     flows left.
 *   - D as source pairs its remaining unpaired flows with first-stage relays
 *     holding an unpaired outflow, cheapest first by source link plus cost
 *     to the sink (Sec. V-C: nodes with unpaired inflow look for unpaired
 *     outflow to the same data node).  READING: ties to the lowest index.
 *   - An approved requester takes its lowest free slot as a new unpaired
 *     outflow to the approved slot (or to D), which becomes paired.
 * Improvement phase (Sec. V-C, Request Change and Request Redirect, with
 * simulated annealing):
 *   - Relays that sent no Request Flow this round are improvers (Sec. V-C:
 *     a node with no peer to request flow from minimises its sending cost
 *     with its same-stage peers).
 *   - READING (pairing): stages of even index are processed first, in
 *     increasing order, then the odd ones.  A stage's relays are shuffled
 *     (Fisher-Yates) and taken in pairs (a, b) = (p[2m], p[2m+1]); a is the
 *     proposer and acts only if it is an improver.  Moves of different pairs
 *     then touch different slots, so the order within a step is immaterial.
 *   - Request Redirect (a has a free slot, b holds a paired flow
 *     u -> b -> w): a proposes to carry it as u -> a -> w; if accepted b's
 *     slot is freed and a takes its lowest free slot.  Request Change (both
 *     hold flow): a's outflow x and b's outflow y swap next hops when those
 *     differ (Sec. V-C example: 1 -> 2 and 3 -> 4 become 1 -> 4 and 3 -> 2).
 *     READING: if both are possible a random bit picks one; the flow moved is
 *     drawn uniformly among b's paired slots (Redirect) or among a's and b's
 *     used slots (Change); a move needing a missing link is dropped.
 *   - Objective of a move: the Eq. 1 cost of the links it changes, in
 *     doubled integer units E(x, y) = 2 * link(x, y) + c_x + c_y (c of D is
 *     0), either summed (Eq. 2, the objective of the flow ablation, Sec. VI)
 *     or maximised (the local max objective of Sec. V-A used in the Request
 *     Change example).  Its cost change is (cur - new) / 2.
 *   - Acceptance (Sec. V-C): a move is taken when
 *     exp((cost_cur - cost_new) / T) > U(0, 1) (so every move that does not
 *     raise the cost is taken); after each accepted move the proposer's
 *     temperature T is multiplied by alpha.  READING: each relay keeps its
 *     own T, starting at T0 (Sec. VI setup: T0 = 1.7, alpha = 0.95).  The
 *     decision is taken in IEEE double arithmetic.
 *
 * Random numbers: Philox4x64-10 (Salmon, Moraes, Dror, Shaw, "Parallel
 * random numbers: as easy as 1, 2, 3", SC 2011), key = (seed, instance),
 * counter = (round, stage, stream, index): stream 0 feeds the stage's
 * shuffle (index = block number, its four words used in turn; the draw for
 * position j picks r in [0, j] as ((w >> 32) * (j + 1)) >> 32), stream 1
 * feeds pair m (index = m; words: move kind bit, slot of a, slot of b or
 * the flow of b, and U = (w >> 11) * 2^-53).
 *
 * Result after `rounds` rounds: the complete paths (chains of slots from D
 * as source to D as sink) are the heuristic's routed microbatches: F is
 * their number and cost the sum of their path costs (src + compute costs +
 * links + snk), the same objective as the exact optimum, so the ratio of the
 * two scores the heuristic (Sec. VI flow ablation).  Dangling chains (slots
 * never paired from the source) hold capacity but carry nothing.
 *
 * Per-instance status: 0 ok; 1 bad input (negative capacity, cost or supply,
 * a link below -1, total capacity above max_slots, or an invalid initial
 * path); 2 overflow ((2S + 2) * largest cost >= 2^30).
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define HS_NONE (-1)
#define HS_DATA (-2)
#define HS_NO_ARC (-1)

enum { HS_OK = 0, HS_BAD_INPUT = 1, HS_OVERFLOW = 2 };

/* ---- Philox4x64-10, from the round function and key schedule published by
 * Salmon et al. (2011): each round multiplies counter words 0 and 2 by two
 * fixed 64-bit constants, and the key is bumped by two Weyl constants
 * between rounds. ---- */
static void philox4x64_10(const uint64_t ctr_in[4], const uint64_t key_in[2], uint64_t out[4])
{
    const uint64_t M0 = 0xD2E7470EE14C6C93ULL, M1 = 0xCA5A826395121157ULL;
    const uint64_t W0 = 0x9E3779B97F4A7C15ULL, W1 = 0xBB67AE8584CAA73BULL;
    uint64_t c0 = ctr_in[0], c1 = ctr_in[1], c2 = ctr_in[2], c3 = ctr_in[3];
    uint64_t k0 = key_in[0], k1 = key_in[1];
    for (int r = 0; r < 10; r++) {
        if (r > 0) {
            k0 += W0;
            k1 += W1;
        }
        unsigned __int128 p0 = (unsigned __int128)M0 * c0;
        unsigned __int128 p1 = (unsigned __int128)M1 * c2;
        uint64_t hi0 = (uint64_t)(p0 >> 64), lo0 = (uint64_t)p0;
        uint64_t hi1 = (uint64_t)(p1 >> 64), lo1 = (uint64_t)p1;
        c0 = hi1 ^ c1 ^ k0;
        c1 = lo1;
        c2 = hi0 ^ c3 ^ k1;
        c3 = lo0;
    }
    out[0] = c0;
    out[1] = c1;
    out[2] = c2;
    out[3] = c3;
}

/* Exported for the generator's own pin against an independent Philox. */
void heur_philox4x64_10(const uint64_t *ctr, const uint64_t *key, uint64_t *out)
{
    philox4x64_10(ctr, key, out);
}

static uint32_t bounded(uint64_t w, uint32_t m) { return (uint32_t)(((w >> 32) * (uint64_t)m) >> 32); }

typedef struct {
    int32_t S, n, V, nslots, supply;
    const int32_t *cap, *cost, *arc, *src, *snk;
    int32_t *base;   /* [V + 1] first slot of each relay */
    int32_t *owner;  /* [nslots] relay owning the slot */
    int32_t *in, *out;
    int64_t *cs;     /* cost to the sink of each used slot */
    double *T;       /* [V] temperature of each relay */
    int32_t *acc;    /* [V] accepted moves of each relay */
    int32_t *req;    /* [V] request target this round: HS_NONE, HS_DATA or a relay */
    int32_t *win;    /* [V] 1 if the request was approved */
    int32_t src_left, sink_left;
    uint64_t key[2];
} hs_state;

static int32_t stage_of(const hs_state *st, int32_t v) { return v / st->n; }
static int32_t index_of(const hs_state *st, int32_t v) { return v % st->n; }

/* Link cost from relay u (stage k) to relay v (stage k + 1). */
static int32_t link(const hs_state *st, int32_t u, int32_t v)
{
    int32_t k = stage_of(st, u);
    return st->arc[((int64_t)k * st->n + index_of(st, u)) * st->n + index_of(st, v)];
}

/* Node at the other end of a slot pointer (HS_DATA stays HS_DATA). */
static int32_t node_of(const hs_state *st, int32_t slot) { return slot == HS_DATA ? HS_DATA : st->owner[slot]; }

/* Link cost between x and y, where either end may be the data node D. */
static int32_t edge(const hs_state *st, int32_t x, int32_t y)
{
    if (x == HS_DATA) return st->src[index_of(st, y)];
    if (y == HS_DATA) return st->snk[index_of(st, x)];
    return link(st, x, y);
}

static int32_t ccost(const hs_state *st, int32_t v) { return v == HS_DATA ? 0 : st->cost[v]; }

/* Eq. 1 cost of the link x -> y in doubled units: 2 * link + c_x + c_y. */
static int64_t E(const hs_state *st, int32_t x, int32_t y)
{
    return 2 * (int64_t)edge(st, x, y) + ccost(st, x) + ccost(st, y);
}

static int32_t used(const hs_state *st, int32_t v)
{
    int32_t c = 0;
    for (int32_t s = st->base[v]; s < st->base[v + 1]; s++) c += st->out[s] != HS_NONE;
    return c;
}

static int32_t paired_count(const hs_state *st, int32_t v)
{
    int32_t c = 0;
    for (int32_t s = st->base[v]; s < st->base[v + 1]; s++) c += st->out[s] != HS_NONE && st->in[s] != HS_NONE;
    return c;
}

static int32_t unpaired(const hs_state *st, int32_t v)
{
    for (int32_t s = st->base[v]; s < st->base[v + 1]; s++)
        if (st->out[s] != HS_NONE && st->in[s] == HS_NONE) return s;
    return HS_NONE;
}

static int32_t free_slot(const hs_state *st, int32_t v)
{
    for (int32_t s = st->base[v]; s < st->base[v + 1]; s++)
        if (st->out[s] == HS_NONE) return s;
    return HS_NONE;
}

/* The q-th (from 0) slot of v that is used (paired_only = 0) or paired. */
static int32_t nth_slot(const hs_state *st, int32_t v, int32_t q, int paired_only)
{
    for (int32_t s = st->base[v]; s < st->base[v + 1]; s++) {
        if (st->out[s] == HS_NONE || (paired_only && st->in[s] == HS_NONE)) continue;
        if (q-- == 0) return s;
    }
    return HS_NONE;
}

/* Cost to the sink of every used slot, from the last stage to the first. */
static void costs_to_sink(hs_state *st)
{
    for (int32_t k = st->S - 1; k >= 0; k--)
        for (int32_t i = 0; i < st->n; i++) {
            int32_t v = k * st->n + i;
            for (int32_t s = st->base[v]; s < st->base[v + 1]; s++) {
                if (st->out[s] == HS_NONE) continue;
                int32_t o = st->out[s];
                st->cs[s] = st->cost[v] + (int64_t)edge(st, v, node_of(st, o)) + (o == HS_DATA ? 0 : st->cs[o]);
            }
        }
}

static void request_flow_phase(hs_state *st)
{
    const int32_t S = st->S, n = st->n, V = st->V;
    costs_to_sink(st);
    for (int32_t v = 0; v < V; v++) {
        st->req[v] = HS_NONE;
        st->win[v] = 0;
        if (unpaired(st, v) != HS_NONE || used(st, v) >= st->cap[v]) continue;
        int32_t k = stage_of(st, v);
        if (k == S - 1) {
            if (st->sink_left > 0) st->req[v] = HS_DATA;
            continue;
        }
        int64_t best = 0;
        for (int32_t j = 0; j < n; j++) {
            int32_t w = (k + 1) * n + j, u = unpaired(st, w);
            if (u == HS_NONE || link(st, v, w) == HS_NO_ARC) continue;
            int64_t score = st->cs[u] + link(st, v, w);
            if (st->req[v] == HS_NONE || score < best) {
                best = score;
                st->req[v] = w;
            }
        }
    }
    /* approvals: each relay target takes its lowest requester; D as sink
     * takes last-stage requesters in order while it has flows left */
    int32_t sink_room = st->sink_left;
    for (int32_t v = 0; v < V; v++) {
        if (st->req[v] == HS_NONE) continue;
        if (st->req[v] == HS_DATA) {
            if (sink_room > 0) {
                st->win[v] = 1;
                sink_room--;
            }
            continue;
        }
        int first = 1;
        for (int32_t q = 0; q < v; q++)
            if (st->req[q] == st->req[v]) first = 0;
        st->win[v] = first;
    }
    /* D as source pairs first-stage unpaired outflows, cheapest first */
    int32_t *order = malloc(sizeof(int32_t) * n), cnt = 0;
    for (int32_t j = 0; j < n; j++)
        if (unpaired(st, j) != HS_NONE) order[cnt++] = j;
    for (int32_t a = 0; a < cnt; a++) /* insertion sort by (src + cost to sink, index) */
        for (int32_t b = a; b > 0; b--) {
            int32_t x = order[b - 1], y = order[b];
            int64_t kx = st->src[x] + st->cs[unpaired(st, x)], ky = st->src[y] + st->cs[unpaired(st, y)];
            if (ky < kx) {
                order[b - 1] = y;
                order[b] = x;
            }
        }
    int32_t take = cnt < st->src_left ? cnt : st->src_left;
    for (int32_t a = 0; a < take; a++) st->in[unpaired(st, order[a])] = HS_DATA;
    st->src_left -= take;
    free(order);
    /* approved requesters open a new unpaired outflow */
    for (int32_t v = 0; v < V; v++) {
        if (!st->win[v]) continue;
        int32_t z = free_slot(st, v);
        if (st->req[v] == HS_DATA) {
            st->out[z] = HS_DATA;
            st->sink_left--;
        } else {
            int32_t u = unpaired(st, st->req[v]);
            st->out[z] = u;
            st->in[u] = z;
        }
        st->in[z] = HS_NONE;
    }
}

static int accept_move(int64_t cur, int64_t nxt, double T, uint64_t w)
{
    double U = (double)(w >> 11) * (1.0 / 9007199254740992.0);
    double delta = (double)(cur - nxt) * 0.5;
    return exp(delta / T) > U;
}

static void improvement_phase(hs_state *st, int32_t round, int32_t objective, double alpha)
{
    const int32_t S = st->S, n = st->n;
    int32_t *perm = malloc(sizeof(int32_t) * n);
    for (int32_t parity = 0; parity < 2; parity++)
        for (int32_t k = parity; k < S; k += 2) {
            /* shuffle the stage (stream 0) */
            for (int32_t j = 0; j < n; j++) perm[j] = j;
            uint64_t words[4];
            int32_t used_words = 4, block = 0;
            for (int32_t j = n - 1; j >= 1; j--) {
                if (used_words == 4) {
                    uint64_t ctr[4] = {(uint64_t)round, (uint64_t)k, 0, (uint64_t)block++};
                    philox4x64_10(ctr, st->key, words);
                    used_words = 0;
                }
                int32_t r = (int32_t)bounded(words[used_words++], (uint32_t)(j + 1));
                int32_t t = perm[j];
                perm[j] = perm[r];
                perm[r] = t;
            }
            /* pairs (stream 1) */
            for (int32_t m = 0; 2 * m + 1 < n; m++) {
                int32_t a = k * n + perm[2 * m], b = k * n + perm[2 * m + 1];
                if (st->req[a] != HS_NONE) continue; /* a sent a Request Flow this round */
                uint64_t w[4], ctr[4] = {(uint64_t)round, (uint64_t)k, 1, (uint64_t)m};
                philox4x64_10(ctr, st->key, w);
                int can_redirect = used(st, a) < st->cap[a] && paired_count(st, b) > 0;
                int can_change = used(st, a) > 0 && used(st, b) > 0;
                if (!can_redirect && !can_change) continue;
                int redirect = can_redirect && can_change ? (int)(w[0] & 1) : can_redirect;
                int64_t cur, nxt;
                if (redirect) {
                    int32_t y = nth_slot(st, b, (int32_t)bounded(w[1], (uint32_t)paired_count(st, b)), 1);
                    int32_t up = st->in[y], dn = st->out[y];
                    int32_t un = node_of(st, up), dw = node_of(st, dn);
                    if (edge(st, un, a) == HS_NO_ARC || edge(st, a, dw) == HS_NO_ARC) continue;
                    int64_t c0 = E(st, un, b), c1 = E(st, b, dw), n0 = E(st, un, a), n1 = E(st, a, dw);
                    cur = objective ? (c0 > c1 ? c0 : c1) : c0 + c1;
                    nxt = objective ? (n0 > n1 ? n0 : n1) : n0 + n1;
                    if (!accept_move(cur, nxt, st->T[a], w[3])) continue;
                    int32_t z = free_slot(st, a);
                    st->in[z] = up;
                    st->out[z] = dn;
                    if (up != HS_DATA) st->out[up] = z;
                    if (dn != HS_DATA) st->in[dn] = z;
                    st->in[y] = HS_NONE;
                    st->out[y] = HS_NONE;
                } else {
                    int32_t x = nth_slot(st, a, (int32_t)bounded(w[1], (uint32_t)used(st, a)), 0);
                    int32_t y = nth_slot(st, b, (int32_t)bounded(w[2], (uint32_t)used(st, b)), 0);
                    int32_t ox = st->out[x], oy = st->out[y];
                    int32_t nx = node_of(st, ox), ny = node_of(st, oy);
                    if (nx == ny) continue; /* same next hop: nothing to switch */
                    if (edge(st, a, ny) == HS_NO_ARC || edge(st, b, nx) == HS_NO_ARC) continue;
                    int64_t c0 = E(st, a, nx), c1 = E(st, b, ny), n0 = E(st, a, ny), n1 = E(st, b, nx);
                    cur = objective ? (c0 > c1 ? c0 : c1) : c0 + c1;
                    nxt = objective ? (n0 > n1 ? n0 : n1) : n0 + n1;
                    if (!accept_move(cur, nxt, st->T[a], w[3])) continue;
                    st->out[x] = oy;
                    st->out[y] = ox;
                    if (oy != HS_DATA) st->in[oy] = x;
                    if (ox != HS_DATA) st->in[ox] = y;
                }
                st->T[a] *= alpha;
                st->acc[a]++;
            }
        }
    free(perm);
}

typedef struct {
    int32_t B, S, n, P, rounds, objective, max_slots;
    double T0, alpha;
    uint64_t seed;
    const int32_t *cap, *cost, *arc, *src, *snk, *supply, *paths;
    int64_t *F, *total, *counters;
    int32_t *status, *node_flow, *arc_flow, *used, *acc;
    double *T;
    int32_t next;
} hs_job;

/* Validates instance b; 0 if it can run, else its status. */
static int32_t check_instance(const hs_job *jb, int32_t b)
{
    const int32_t S = jb->S, n = jb->n;
    const int64_t sn = (int64_t)S * n, ann = (int64_t)(S - 1) * n * n;
    int64_t total_cap = 0, maxc = 0;
    if (jb->supply[b] < 0) return HS_BAD_INPUT;
    for (int64_t q = 0; q < sn; q++) {
        int32_t c = jb->cap[b * sn + q], w = jb->cost[b * sn + q];
        if (c < 0 || w < 0) return HS_BAD_INPUT;
        total_cap += c;
        if (w > maxc) maxc = w;
    }
    for (int64_t q = 0; q < ann; q++) {
        int32_t w = jb->arc[b * ann + q];
        if (w < HS_NO_ARC) return HS_BAD_INPUT;
        if (w > maxc) maxc = w;
    }
    for (int32_t i = 0; i < n; i++) {
        int32_t a = jb->src ? jb->src[(int64_t)b * n + i] : 0, z = jb->snk ? jb->snk[(int64_t)b * n + i] : 0;
        if (a < 0 || z < 0) return HS_BAD_INPUT;
        if (a > maxc) maxc = a;
        if (z > maxc) maxc = z;
    }
    if (total_cap > jb->max_slots) return HS_BAD_INPUT;
    if ((int64_t)(2 * S + 2) * maxc >= ((int64_t)1 << 30)) return HS_OVERFLOW;
    return HS_OK;
}

/* Lays the initial complete paths of instance b into the slots (each path
 * node takes its lowest free slot, in path order); 0 on success. */
static int32_t place_paths(hs_state *st, const int32_t *paths, int32_t P)
{
    for (int32_t p = 0; p < P; p++) {
        const int32_t *path = paths + (int64_t)p * st->S;
        if (path[0] < 0) continue;
        if (st->src_left <= 0 || st->sink_left <= 0) return HS_BAD_INPUT;
        int32_t prev = HS_DATA;
        for (int32_t k = 0; k < st->S; k++) {
            if (path[k] < 0 || path[k] >= st->n) return HS_BAD_INPUT;
            int32_t v = k * st->n + path[k];
            if (prev != HS_DATA && link(st, st->owner[prev], v) == HS_NO_ARC) return HS_BAD_INPUT;
            int32_t z = free_slot(st, v);
            if (z == HS_NONE) return HS_BAD_INPUT;
            st->in[z] = prev;
            st->out[z] = HS_DATA; /* rewritten by the next hop */
            if (prev != HS_DATA) st->out[prev] = z;
            prev = z;
        }
        st->src_left--;
        st->sink_left--;
    }
    return HS_OK;
}

static void run_instance(const hs_job *jb, int32_t b)
{
    const int32_t S = jb->S, n = jb->n, V = S * n;
    const int64_t sn = (int64_t)S * n, ann = (int64_t)(S - 1) * n * n;
    int32_t status = check_instance(jb, b);
    int64_t F = 0, total = 0, counters[4] = {0, 0, 0, 0};
    int32_t *nf = jb->node_flow ? jb->node_flow + b * sn : NULL;
    int32_t *af = jb->arc_flow ? jb->arc_flow + b * ann : NULL;
    int32_t *us = jb->used ? jb->used + b * sn : NULL;
    int32_t *ac = jb->acc ? jb->acc + b * sn : NULL;
    double *Tout = jb->T ? jb->T + b * sn : NULL;
    if (nf) memset(nf, 0, sizeof(int32_t) * sn);
    if (af) memset(af, 0, sizeof(int32_t) * ann);
    if (us) memset(us, 0, sizeof(int32_t) * sn);
    if (ac) memset(ac, 0, sizeof(int32_t) * sn);
    if (Tout)
        for (int64_t q = 0; q < sn; q++) Tout[q] = jb->T0;
    int32_t *zeros = calloc(n, sizeof(int32_t));
    hs_state st;
    memset(&st, 0, sizeof st);
    if (status == HS_OK) {
        st.S = S;
        st.n = n;
        st.V = V;
        st.supply = jb->supply[b];
        st.cap = jb->cap + b * sn;
        st.cost = jb->cost + b * sn;
        st.arc = S > 1 ? jb->arc + b * ann : NULL;
        st.src = jb->src ? jb->src + (int64_t)b * n : zeros;
        st.snk = jb->snk ? jb->snk + (int64_t)b * n : zeros;
        st.base = malloc(sizeof(int32_t) * (V + 1));
        st.base[0] = 0;
        for (int32_t v = 0; v < V; v++) st.base[v + 1] = st.base[v] + st.cap[v];
        st.nslots = st.base[V];
        int32_t ns = st.nslots > 0 ? st.nslots : 1;
        st.owner = malloc(sizeof(int32_t) * ns);
        st.in = malloc(sizeof(int32_t) * ns);
        st.out = malloc(sizeof(int32_t) * ns);
        st.cs = calloc(ns, sizeof(int64_t));
        st.T = malloc(sizeof(double) * V);
        st.acc = calloc(V, sizeof(int32_t));
        st.req = malloc(sizeof(int32_t) * V);
        st.win = malloc(sizeof(int32_t) * V);
        for (int32_t v = 0; v < V; v++) {
            for (int32_t s = st.base[v]; s < st.base[v + 1]; s++) {
                st.owner[s] = v;
                st.in[s] = HS_NONE;
                st.out[s] = HS_NONE;
            }
            st.T[v] = jb->T0;
        }
        st.src_left = st.supply;
        st.sink_left = st.supply;
        st.key[0] = jb->seed;
        st.key[1] = (uint64_t)b;
        if (jb->paths) status = place_paths(&st, jb->paths + (int64_t)b * jb->P * S, jb->P);
    }
    if (status == HS_OK) {
        for (int32_t r = 0; r < jb->rounds; r++) {
            request_flow_phase(&st);
            for (int32_t v = 0; v < V; v++) counters[1] += st.win[v];
            improvement_phase(&st, r, jb->objective, jb->alpha);
        }
        for (int32_t v = 0; v < V; v++) counters[2] += st.acc[v];
        counters[0] = st.supply - st.src_left;
        /* complete paths: slots reached from D as source, stage by stage */
        int32_t *complete = calloc(st.nslots > 0 ? st.nslots : 1, sizeof(int32_t));
        for (int32_t k = 0; k < S; k++)
            for (int32_t i = 0; i < n; i++) {
                int32_t v = k * n + i;
                for (int32_t s = st.base[v]; s < st.base[v + 1]; s++) {
                    if (st.out[s] == HS_NONE) continue;
                    complete[s] = st.in[s] == HS_DATA || (st.in[s] >= 0 && complete[st.in[s]]);
                    if (!complete[s]) continue;
                    int32_t o = st.out[s];
                    total += st.cost[v] + (int64_t)edge(&st, v, node_of(&st, o));
                    if (k == 0) {
                        F++;
                        total += st.src[i];
                    }
                    if (nf) nf[v]++;
                    if (af && o != HS_DATA) af[(int64_t)v * n + index_of(&st, st.owner[o])]++;
                }
            }
        for (int32_t v = 0; v < V; v++) {
            if (us) us[v] = used(&st, v);
            if (ac) ac[v] = st.acc[v];
            if (Tout) Tout[v] = st.T[v];
        }
        int64_t dangling = 0;
        for (int32_t s = 0; s < st.nslots; s++) dangling += st.out[s] != HS_NONE && !complete[s];
        counters[3] = dangling;
        free(complete);
    }
    if (status != HS_OK) {
        F = 0;
        total = 0;
    }
    jb->F[b] = F;
    jb->total[b] = total;
    jb->status[b] = status;
    if (jb->counters)
        for (int q = 0; q < 4; q++) jb->counters[4 * (int64_t)b + q] = counters[q];
    free(st.base);
    free(st.owner);
    free(st.in);
    free(st.out);
    free(st.cs);
    free(st.T);
    free(st.acc);
    free(st.req);
    free(st.win);
    free(zeros);
}

static void *worker(void *arg)
{
    hs_job *jb = arg;
    for (;;) {
        int32_t b = __atomic_fetch_add(&jb->next, 1, __ATOMIC_RELAXED);
        if (b >= jb->B) break;
        run_instance(jb, b);
    }
    return NULL;
}

/* Simulates B independent instances (canonical batch layout: cap, cost
 * [B][S][n]; arc [B][S-1][n][n], NULL iff S == 1; src, snk [B][n] or NULL
 * = 0; supply [B]) for `rounds` rounds with objective 0 = sum, 1 = max.
 * paths (optional) gives initial complete paths [B][P][S] (node index per
 * stage; rows starting with -1 unused).  Outputs: F, total [B]; status [B];
 * optional node_flow [B][S][n] and arc_flow [B][S-1][n][n] of the complete
 * paths, used slots and accepted moves [B][S][n], final temperatures
 * [B][S][n], counters [B][4] = (paths paired by the data node, Request Flow
 * approvals, accepted moves, dangling slots).  Returns the threads used, or
 * -1 on a bad shape. */
int heur_simulate_batch(int32_t B, int32_t S, int32_t n, const int32_t *cap, const int32_t *cost,
                        const int32_t *arc, const int32_t *src, const int32_t *snk, const int32_t *supply,
                        const int32_t *paths, int32_t P, int32_t rounds, int32_t objective, double T0,
                        double alpha, uint64_t seed, int32_t max_slots, int64_t *F, int64_t *total,
                        int32_t *status, int32_t *node_flow, int32_t *arc_flow, int32_t *used_out,
                        int32_t *accepted, double *temperature, int64_t *counters, int32_t nthreads)
{
    if (B < 0 || S < 1 || n < 1 || !cap || !cost || !supply || !F || !total || !status) return -1;
    if ((S > 1) != (arc != NULL) || rounds < 0 || (paths && P < 0)) return -1;
    hs_job jb;
    memset(&jb, 0, sizeof jb);
    jb.B = B;
    jb.S = S;
    jb.n = n;
    jb.P = paths ? P : 0;
    jb.rounds = rounds;
    jb.objective = objective != 0;
    jb.max_slots = max_slots;
    jb.T0 = T0;
    jb.alpha = alpha;
    jb.seed = seed;
    jb.cap = cap;
    jb.cost = cost;
    jb.arc = arc;
    jb.src = src;
    jb.snk = snk;
    jb.supply = supply;
    jb.paths = paths;
    jb.F = F;
    jb.total = total;
    jb.status = status;
    jb.node_flow = node_flow;
    jb.arc_flow = arc_flow;
    jb.used = used_out;
    jb.acc = accepted;
    jb.T = temperature;
    jb.counters = counters;
    if (nthreads < 1) nthreads = 1;
    if (nthreads > B) nthreads = B > 0 ? B : 1;
    pthread_t *th = malloc(sizeof(pthread_t) * nthreads);
    int32_t started = 0;
    for (int32_t t = 1; t < nthreads; t++)
        if (pthread_create(&th[t], NULL, worker, &jb) == 0) started++;
        else break;
    worker(&jb);
    for (int32_t t = 1; t <= started; t++) pthread_join(th[t], NULL);
    free(th);
    return started + 1;
}
