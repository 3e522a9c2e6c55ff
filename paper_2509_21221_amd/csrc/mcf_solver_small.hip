// Packed pass for small instances: one to eight instances per wave, for at
// most 8 stages of at most 16 nodes (the node-addition batches of paper
// Sec. VI and the 4 x 4 / 8 x 8 presets).
//
// Same method as the other passes (successive shortest paths with Johnson
// potentials on the node-split stage graph, paper Sec. V-A Eq. 2); what
// differs is the mapping.  One wave = four 16-lane rows (the DPP row of
// CDNA), one instance per row (or per half row when n <= 8), lane j of a row
// = node j of every stage; a small batch leaves some rows of each wave empty
// so that it spreads over more waves:
//
//  * Keys.  A vertex label is kept as key = label << 5 | code, where code
//    names the predecessor arc: for an entry, 0..15 = the link from that
//    exit of the previous stage, 16 = the reverse compute arc, 17 = the
//    data node; for an exit, 0..15 = the reverse link from that entry of the
//    next stage, 16 = the compute arc.  Finite keys stay below 2^30 (labels
//    below 2^25); unreached vertices hold kKeyInf = 2^31 | 31, and a missing
//    link costs 2^30, so no sum or difference of a key and a cost wraps and
//    none that involves an unreached key or a missing link lands in the
//    finite range.  A key is replaced only by one with a strictly smaller
//    label, which keeps the predecessors a tree.
//  * Forward relaxation.  The incoming link costs of a stage sit in vector
//    registers (cost << 5, column j in lane j, one register per row); the
//    previous stage's exit keys reach lane j through DPP row broadcasts
//    fused into the adds, so a dense 16 x 16 relaxation is 16 broadcast-adds
//    and 8 three-way minima per stage.
//  * Reverse links (links carrying flow) are pulled at the exit's lane from
//    the next stage's entry keys, one partner per pass over the set bits of
//    the exit's 16-bit mask of links with flow (cross-lane read of the
//    partner's key, link cost from the exit's row of costs in LDS).
//  * Rounds: a forward sweep over the stages, then a backward sweep, until
//    a backward sweep changes nothing in any of the wave's instances.
//  * After each search: potentials (device workspace), then each row walks
//    its own path twice (bottleneck, then apply) over the node flows and the
//    per-link flows kept in LDS.
//
// Instances outside the pass's bounds (supply above 255, a cost above 2047,
// labels that could reach 2^25) are routed to the fallback pass.
#include "mcf_device.h"
#include "mcf_small.h"

namespace gwtf {
namespace {

using namespace dev;

constexpr uint32_t kKeyInf = 0x80000000u | 31u;
constexpr uint32_t kFiniteLimit = 0x40000000u; // keys at or above are unreached
constexpr uint32_t kNoLink = 0x40000000u;      // cost << 5 of a missing link
constexpr uint32_t kCodeSplit = 16, kCodeSrc = 17;
constexpr int kMaxCost = 2047;
constexpr int kMaxSupply = 255;
constexpr int64_t kSmallLabelLimit = (int64_t(1) << 25) - (int64_t(1) << 16);

// The largest key a strictly better candidate must stay below.
__device__ __forceinline__ uint32_t lim(uint32_t key) { return min(key & ~31u, kFiniteLimit); }

// Lane I of this lane's group of G lanes: for G = 16 one DPP row broadcast;
// for G = 8 the two halves of a row take lanes I and 8 + I through
// bank-masked broadcasts.
template <int G, int I> __device__ __forceinline__ uint32_t group_bcast(uint32_t x)
{
    if constexpr (G == 16) {
        return uint32_t(__builtin_amdgcn_update_dpp(0, int(x), 0x150 + I, 0xf, 0xf, false));
    } else {
        static_assert(G == 8, "groups of 8 or 16 lanes");
        // lanes 8-15 of each row are written by the second move, so the
        // first needs no old value
        const int lo = __builtin_amdgcn_mov_dpp(int(x), 0x150 + I, 0xf, 0x3, false);
        return uint32_t(__builtin_amdgcn_update_dpp(lo, int(x), 0x158 + I, 0xf, 0xc, false));
    }
}

// min over the G rows i of (key of exit i with code i) + cost(i -> this lane)
template <int G, int I> struct Relax {
    static __device__ __forceinline__ void run(uint32_t xr, const uint32_t (&c)[G], uint32_t &best)
    {
        best = min(best, group_bcast<G, I>(xr) + c[I]);
        Relax<G, I + 1>::run(xr, c, best);
    }
};
template <> struct Relax<16, 16> {
    static __device__ __forceinline__ void run(uint32_t, const uint32_t (&)[16], uint32_t &) {}
};
template <> struct Relax<8, 8> {
    static __device__ __forceinline__ void run(uint32_t, const uint32_t (&)[8], uint32_t &) {}
};

// min over the G lanes of a group, in every lane of the group
template <int G> __device__ __forceinline__ uint32_t group_min(uint32_t v)
{
    v = min(v, uint32_t(__builtin_amdgcn_update_dpp(0, int(v), 0xb1, 0xf, 0xf, false)));  // quad_perm [1,0,3,2]
    v = min(v, uint32_t(__builtin_amdgcn_update_dpp(0, int(v), 0x4e, 0xf, 0xf, false)));  // quad_perm [2,3,0,1]
    v = min(v, uint32_t(__builtin_amdgcn_update_dpp(0, int(v), 0x141, 0xf, 0xf, false))); // row_half_mirror
    if constexpr (G == 16)
        v = min(v, uint32_t(__builtin_amdgcn_update_dpp(0, int(v), 0x140, 0xf, 0xf, false))); // row_mirror
    return v;
}
template <int G> __device__ __forceinline__ int group_max(int v)
{
    v = max(v, __builtin_amdgcn_update_dpp(0, v, 0xb1, 0xf, 0xf, false));
    v = max(v, __builtin_amdgcn_update_dpp(0, v, 0x4e, 0xf, 0xf, false));
    v = max(v, __builtin_amdgcn_update_dpp(0, v, 0x141, 0xf, 0xf, false));
    if constexpr (G == 16) v = max(v, __builtin_amdgcn_update_dpp(0, v, 0x140, 0xf, 0xf, false));
    return v;
}

// LDS of one wave: node words (flow | capacity << 8 | compute cost << 16),
// per exit the mask of its links with flow (16 bits, two exits per word),
// per vertex its predecessor code and that arc's residual for the path walk
// (all laid out for the largest stage count, so their offsets are
// constants), then per link its flow and per exit its row of link costs
// (cost << 5), n x n per stage pair and row.
template <int MAXS, int ROWS> struct SmallLayout {
    static constexpr size_t node = 0;
    static constexpr size_t mask = node + 4 * MAXS * 64;     // 16 bits per exit
    static constexpr size_t walk = mask + 2 * MAXS * 64;     // per vertex: pred code | residual << 5
    static constexpr size_t lflow = walk + 2 * 2 * MAXS * 64;
    static __host__ __device__ size_t lcost(int n) { return lflow + align16(size_t(MAXS - 1) * ROWS * n * n); }
    static __host__ __device__ size_t total(int n) { return lcost(n) + align16(2 * size_t(MAXS - 1) * ROWS * n * n); }
};

template <int MAXS, int G, int R = 64 / G>
__global__ __launch_bounds__(64, 2) void solve_small_kernel(SolveParams p)
{
    constexpr int kRows = 64 / G; // instance rows per wave, the first R of them used
    const int S = p.S, n = p.n, SN = S * n, V = 2 * SN + 3;
    const int lane = threadIdx.x, g = lane / G, j = lane % G, gb = g * G; // gb: first lane of the group
    const int b = blockIdx.x * R + g;
    const bool inst = g < R && b < p.B; // this row holds an instance
    const bool node = inst && j < n; // this lane is a real node
    extern __shared__ __align__(16) unsigned char smem[];
    using Ly = SmallLayout<MAXS, kRows>;
    uint32_t *nodew = reinterpret_cast<uint32_t *>(smem + Ly::node);  // [S][64]
    uint32_t *lmask = reinterpret_cast<uint32_t *>(smem + Ly::mask);  // [S][32]: two exits' links with flow
    uint16_t *wstage = reinterpret_cast<uint16_t *>(smem + Ly::walk); // [S][2][64]: entry, exit
    uint8_t *lflow = smem + Ly::lflow;                                   // [S-1][4][n][n]: (k, i) -> (k+1, j)
    uint16_t *lcost = reinterpret_cast<uint16_t *>(smem + Ly::lcost(n)); // [S-1][4][n][n]
    auto lidx = [&](int k, int i, int jj) { return ((k * kRows + g) * n + i) * n + jj; };

    const int supply = inst ? p.supply[b] : 0;
    const int32_t *gcap = p.cap + size_t(b) * SN;
    const int32_t *gnc = p.ncost + size_t(b) * SN;
    const int32_t *gac = S > 1 ? p.acost + size_t(b) * (S - 1) * n * n : nullptr;
    int32_t *gpot = p.pot + size_t(b) * V;

    // ---------------- ingest + validate ----------------
    int bad = supply < 0, mx = 0;
    uint32_t cin[MAXS][G]; // [k][i]: cost << 5 of link (k-1, i) -> (k, j), k >= 1
#pragma unroll
    for (int k = 0; k < MAXS; ++k) {
#pragma unroll
        for (int r = 0; r < G; ++r) cin[k][r] = 0;
        if (k >= S) continue;
        const int q = k * n + j;
        const int cp = node ? gcap[q] : 0, w = node ? gnc[q] : 0;
        bad |= (cp < 0) | (w < 0);
        mx = max(mx, w);
        const int ec = min(max(cp, 0), max(supply, 0));
        nodew[k * 64 + lane] = uint32_t(min(ec, kMaxSupply)) << 8 | uint32_t(min(max(w, 0), kMaxCost)) << 16;
        if ((lane & 1) == 0) lmask[k * 32 + (lane >> 1)] = 0;
    }
    // link costs: each row's n x n block of a stage pair, read with
    // consecutive lanes on consecutive elements, into the row-major LDS copy
    for (int k = 0; k + 1 < S; ++k) {
        for (int e = j; e < n * n; e += G) {
            const int i = e / n, jj = e - i * n;
            const int a = inst ? gac[size_t(k) * n * n + size_t(e)] : 0;
            bad |= a < -1;
            mx = max(mx, a);
            // a missing link never carries flow, so its LDS copy is never read
            lcost[lidx(k, i, jj)] = a < 0 ? 0xffffu : uint16_t(uint32_t(min(a, kMaxCost)) << 5);
            lflow[lidx(k, i, jj)] = 0;
        }
    }
    __syncthreads();
    // columns into registers: lane j holds the costs of the links into node j
#pragma unroll
    for (int k = 1; k < MAXS; ++k) {
        if (k >= S) break;
#pragma unroll
        for (int r = 0; r < G; ++r) {
            // rows and columns beyond n are padding: cost 0, never improving
            // anything since those exits stay unreached
            const uint32_t c5 = (r < n && j < n) ? lcost[lidx(k - 1, r, j)] : 0u;
            cin[k][r] = c5 == 0xffffu ? kNoLink : c5;
        }
    }
    int srcc = node && p.src ? p.src[size_t(b) * n + j] : 0;
    int snkc = node && p.snk ? p.snk[size_t(b) * n + j] : 0;
    bad |= (srcc < 0) | (snkc < 0);
    mx = max(mx, max(srcc, snkc));
    bad = group_max<G>(bad);
    mx = group_max<G>(mx);
    int status = 0;
    if (bad) status = 1;
    else if (int64_t(V) * mx >= kLabelBound) status = 2;
    const bool fits = supply <= kMaxSupply && mx <= kMaxCost && int64_t(V) * mx < kSmallLabelLimit;
    const bool mine = inst && (status != 0 || fits); // this pass owns the instance
    if (inst && j == 0) p.route[b] = mine ? kRouteSmall : kRouteFallback;
    const uint32_t src5 = uint32_t(min(max(srcc, 0), kMaxCost)) << 5, snk5 = uint32_t(min(max(snkc, 0), kMaxCost)) << 5;

    // ---------------- successive shortest paths ----------------
    long long F = 0, cost = 0, augs = 0, rounds = 0, rows_relaxed = 0, pulls = 0;
    int pit = 0;
    bool active = mine && status == 0 && supply > 0; // this row still searches
    uint64_t tick = wall_clock64(), clk_fwd = 0, clk_bwd = 0, clk_aug = 0, clk_other = 0;
    uint32_t din[MAXS], dout[MAXS];
    int pin[MAXS], pout[MAXS]; // potentials of this lane's entries and exits
#pragma unroll
    for (int k = 0; k < MAXS; ++k) pin[k] = pout[k] = 0;
    while (__any(active)) {
        // labels of a fresh search
#pragma unroll
        for (int k = 0; k < MAXS; ++k) {
            din[k] = (k == 0 && active && j < n) ? (src5 | kCodeSrc) : kKeyInf;
            dout[k] = kKeyInf;
        }
        clk_other += lap(tick);
        int round_count = 0;
        bool fault = false;
        // Stages whose exit (entry) keys changed in some lane since the next
        // (previous) stage last read them: a relaxation or a pull whose input
        // is unchanged cannot improve anything and is skipped.
        uint32_t new_out = ~0u, new_in = ~0u;
        for (;;) {
            // -------- forward sweep --------
#pragma unroll
            for (int k = 0; k < MAXS; ++k) {
                if (k >= S) break;
                const uint32_t nw = nodew[k * 64 + lane];
                const uint32_t fl = nw & 255u, ec = (nw >> 8) & 255u, nc5 = ((nw >> 16) & 2047u) << 5;
                uint32_t di = din[k], dq = dout[k];
                if (k >= 1 && ((new_out >> (k - 1)) & 1u)) {
                    new_out &= ~(1u << (k - 1));
                    const uint32_t xr = (dout[k - 1] & ~31u) | uint32_t(j);
                    uint32_t best = kKeyInf;
                    Relax<G, 0>::run(xr, cin[k], best);
                    di = best < lim(di) ? best : di;
                    ++rows_relaxed;
                }
                if (fl > 0) {
                    const uint32_t cand = ((dq & ~31u) - nc5) | kCodeSplit;
                    di = cand < lim(di) ? cand : di;
                }
                if (fl < ec) {
                    const uint32_t cand = ((di & ~31u) + nc5) | kCodeSplit;
                    dq = cand < lim(dq) ? cand : dq;
                }
                if (__any(di != din[k])) new_in |= 1u << k;
                if (__any(dq != dout[k])) new_out |= 1u << k;
                din[k] = di;
                dout[k] = dq;
            }
            clk_fwd += lap(tick);
            // -------- backward sweep --------
            bool chg = false;
#pragma unroll
            for (int kk = MAXS - 1; kk >= 0; --kk) {
                if (kk >= S) continue;
                const int k = kk;
                const uint32_t nw = nodew[k * 64 + lane];
                const uint32_t fl = nw & 255u, nc5 = ((nw >> 16) & 2047u) << 5;
                uint32_t di = din[k], dq = dout[k];
                // links with flow out of this exit, read here each time (values
                // derived from it must not be kept live across the rounds)
                const uint32_t lm =
                    k + 1 < S ? (__hip_atomic_load(&lmask[k * 32 + (lane >> 1)], __ATOMIC_RELAXED,
                                                   __HIP_MEMORY_SCOPE_WORKGROUP) >> (16 * (lane & 1))) & 0xffffu
                              : 0u;
                if (k + 1 < S && ((new_in >> (k + 1)) & 1u) && __any(lm != 0u)) {
                    new_in &= ~(1u << (k + 1));
                    // one partner per pass: the lowest remaining link with flow
                    const uint32_t yr = (din[k + 1] & ~31u) | uint32_t(j);
                    uint32_t best = kKeyInf;
                    uint32_t rem = lm;
                    while (__any(rem != 0u)) {
                        const bool have = rem != 0u;
                        const int jj = have ? __builtin_ctz(rem) : 0;
                        rem &= rem - 1u;
                        const uint32_t yj = uint32_t(__shfl(int(yr), gb + jj));
                        // only a real exit with a partner reads its cost (rows of
                        // padding lanes lie outside the n x n block)
                        if (have) {
                            const uint32_t c5 =
                                __hip_atomic_load(&lcost[lidx(k, j, jj)], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
                            best = min(best, yj - c5);
                        }
                    }
                    pulls += __popc(lm);
                    dq = best < lim(dq) ? best : dq;
                }
                if (fl > 0) {
                    const uint32_t cand = ((dq & ~31u) - nc5) | kCodeSplit;
                    di = cand < lim(di) ? cand : di;
                }
                chg |= (di != din[k]) | (dq != dout[k]);
                if (__any(di != din[k])) new_in |= 1u << k;
                if (__any(dq != dout[k])) new_out |= 1u << k;
                din[k] = di;
                dout[k] = dq;
            }
            clk_bwd += lap(tick);
            ++rounds;
            if (!__any(chg)) break;
            // Bellman-Ford settles within |V| rounds without a negative cycle
            if (++round_count > V) {
                fault = true;
                break;
            }
        }
        if (fault) {
            if (active) status = kStatusInternal;
            active = false;
            break;
        }

        // -------- sink, potentials --------
        uint32_t tk = kKeyInf;
#pragma unroll
        for (int k = 0; k < MAXS; ++k)
            if (k == S - 1 && j < n) tk = ((dout[k] & ~31u) + snk5) | uint32_t(j);
        tk = group_min<G>(tk);
        const bool aug = active && tk < kFiniteLimit;
        if (active && !aug) active = false; // sink unreachable: the flow is maximum
        const int Dt = int(tk >> 5), predt = int(tk & 31u);
        if (aug && j < n) {
            const int dred = Dt - pit;
#pragma unroll
            for (int k = 0; k < MAXS; ++k) {
                const int li = din[k] < kFiniteLimit ? int(din[k] >> 5) : INT32_MAX;
                const int lo = dout[k] < kFiniteLimit ? int(dout[k] >> 5) : INT32_MAX;
                pin[k] = min(li, pin[k] + dred);
                pout[k] = min(lo, pout[k] + dred);
            }
        }

        // -------- path: bottleneck, then apply (each row its own) --------
        // Each vertex's predecessor code and the residual of that arc (255 =
        // unbounded or above the supply bound) go to LDS; one lane of the row
        // then needs a single read per step.
        if (__any(aug)) {
#pragma unroll
            for (int k = 0; k < MAXS; ++k) {
                if (k >= S) break;
                const uint32_t nw = nodew[k * 64 + lane];
                const uint32_t fl = nw & 255u, ec = (nw >> 8) & 255u;
                const uint32_t ci = din[k] & 31u, co = dout[k] & 31u;
                const uint32_t ri = ci == kCodeSplit ? fl : 255u;
                uint32_t ro = 255u;
                if (co == kCodeSplit) ro = ec - fl;
                else if (co < 16 && k + 1 < S && j < n) ro = lflow[lidx(k, j, int(co))];
                wstage[(2 * k) * 64 + lane] = uint16_t(ci | ri << 5);
                wstage[(2 * k + 1) * 64 + lane] = uint16_t(co | ro << 5);
            }
        }
        // The walk takes the bottleneck and records each arc (type | stage <<
        // 2 | node << 6 | other << 10) in lane step % 16 of the row: slot 0
        // takes the current block of 16 steps and the slots shift up after
        // each block.  Then all recorded arcs are applied at once.  A simple
        // path touches each node word and link byte once; the link masks of
        // an exit are updated atomically.
        constexpr int kSlots = (2 * MAXS * G + 5 + G - 1) / G;
        constexpr uint32_t kNoArcRec = ~0u;
        uint32_t rec[kSlots];
#pragma unroll
        for (int r = 0; r < kSlots; ++r) rec[r] = kNoArcRec;
        int delta = aug ? supply - int(F) : 0;
        bool bad_walk = false;
        int wave_steps = 0; // iterations of the walk loop (the same in every lane)
        {
            int k = S - 1, v = predt;
            bool at_exit = true, walking = aug && delta > 0;
            for (int steps = 0; __any(walking); ++steps) {
                wave_steps = steps + 1;
                if (walking) {
                    if (steps > 2 * S * G + 4) {
                        bad_walk = true;
                        walking = false;
                    }
                }
                uint32_t arc = ~0u; // type: 0 compute, 1 reverse compute, 2 link, 3 reverse link
                if (walking) {
                    const uint32_t w = wstage[(2 * k + (at_exit ? 1 : 0)) * 64 + gb + v];
                    const uint32_t code = w & 31u;
                    delta = min(delta, int(w >> 5));
                    if (at_exit) {
                        if (code == kCodeSplit) {
                            arc = 0u | uint32_t(k) << 2 | uint32_t(v) << 6;
                            at_exit = false;
                        } else if (code < 16 && k + 1 < S) {
                            arc = 3u | uint32_t(k) << 2 | uint32_t(v) << 6 | code << 10;
                            k = k + 1;
                            v = int(code);
                            at_exit = false;
                        } else {
                            bad_walk = true;
                            walking = false;
                        }
                    } else {
                        if (code == kCodeSrc && k == 0) {
                            walking = false;
                        } else if (code == kCodeSplit) {
                            arc = 1u | uint32_t(k) << 2 | uint32_t(v) << 6;
                            at_exit = true;
                        } else if (code < 16 && k >= 1) {
                            // link (k-1, code) -> (k, v): unbounded
                            arc = 2u | uint32_t(k - 1) << 2 | code << 6 | uint32_t(v) << 10;
                            k = k - 1;
                            v = int(code);
                            at_exit = true;
                        } else {
                            bad_walk = true;
                            walking = false;
                        }
                    }
                }
                if (arc != ~0u && j == steps % G) rec[0] = arc;
                if (steps % G == G - 1) { // steps is the same in every lane
#pragma unroll
                    for (int r = kSlots - 1; r > 0; --r) rec[r] = rec[r - 1];
                    rec[0] = kNoArcRec;
                }
            }
        }
        if (aug && !bad_walk && delta <= 0) bad_walk = true;
        if (bad_walk && active) status = kStatusInternal;
        if (bad_walk) active = false;
        {
            const bool apply = aug && !bad_walk;
            // the shifts run for the whole wave, after the record of steps
            // G - 1, 2G - 1, ...: every row's arcs sit in the first
            // floor(wave_steps / G) + 1 slots
            const int used = wave_steps / G + 1;
#pragma unroll
            for (int r = 0; r < kSlots; ++r) {
                if (r >= used) continue;
                const uint32_t arc = rec[r];
                if (!apply || arc == kNoArcRec) continue;
                const int type = int(arc & 3u), k = int((arc >> 2) & 15u), a = int((arc >> 6) & 15u),
                          c = int((arc >> 10) & 15u);
                if (type == 0) {
                    atomicAdd(&nodew[k * 64 + gb + a], uint32_t(delta));
                } else if (type == 1) {
                    atomicSub(&nodew[k * 64 + gb + a], uint32_t(delta));
                } else if (type == 2) {
                    const int e = lidx(k, a, c);
                    lflow[e] = uint8_t(lflow[e] + delta);
                    const int x = gb + a;
                    atomicOr(&lmask[k * 32 + (x >> 1)], 1u << (c + 16 * (x & 1)));
                } else {
                    const int e = lidx(k, a, c);
                    const int left = lflow[e] - delta;
                    lflow[e] = uint8_t(left);
                    const int x = gb + a;
                    if (left == 0) atomicAnd(&lmask[k * 32 + (x >> 1)], ~(1u << (c + 16 * (x & 1))));
                }
            }
        }
        if (aug && !bad_walk) {
            F += delta;
            cost += (long long)delta * Dt;
            ++augs;
            pit = Dt;
            if (F >= supply) active = false;
        }
        clk_aug += lap(tick);
    }

    // ---------------- export ----------------
    if (!mine) return; // the fallback pass writes this instance
    const bool ok = status == 0;
    const size_t na = size_t(S > 1 ? S - 1 : 0) * n * n;
    int32_t *nf = p.node_flow + size_t(b) * SN;
    int32_t *af = p.arc_flow + size_t(b) * na;
    if (j < n) {
#pragma unroll
        for (int k = 0; k < MAXS; ++k) {
            if (k >= S) break;
            const int q = k * n + j;
            nf[q] = ok ? int(nodew[k * 64 + lane] & 255u) : 0;
            gpot[3 + 2 * q] = ok ? pin[k] : 0;
            gpot[4 + 2 * q] = ok ? pout[k] : 0;
            if (k + 1 < S)
                for (int i = 0; i < n; ++i) af[size_t(k) * n * n + size_t(i) * n + j] = ok ? lflow[lidx(k, i, j)] : 0;
        }
    }
    if (j == 0) {
        gpot[0] = 0;
        gpot[1] = 0;
        gpot[2] = ok ? pit : 0;
        p.F_out[b] = ok ? F : 0;
        p.cost_out[b] = ok ? cost : 0;
        p.status_out[b] = status;
        int64_t *s = p.stats + size_t(b) * kStatsPerInstance;
        s[0] = augs;
        s[1] = rounds;
        s[2] = rows_relaxed * n; // relaxed stage blocks x n rows of n links
        s[3] = pulls;
        const double ns_per_tick = 1e6 / double(p.clock_khz > 0 ? p.clock_khz : 100000);
        s[4] = int64_t(double(clk_fwd) * ns_per_tick);
        s[5] = int64_t(double(clk_bwd) * ns_per_tick);
        s[6] = int64_t(double(clk_aug) * ns_per_tick);
        s[7] = int64_t(double(clk_other) * ns_per_tick);
        s[8] = 0;
        s[9] = 0;
    }
}

} // namespace

bool small_pass_fits(int S, int n) { return S >= 1 && S <= kSmallMaxStages && n <= 16; }

// A batch that gives at least kSmallFullWaves waves at eight instances per
// wave runs that way (n <= 8); otherwise each 16-lane row holds one instance,
// and a small batch uses only the first one or two rows of each wave while
// that keeps it within kSmallSpreadWaves waves, so that it spreads over more
// of the device (the 4 x 4 batch of 1,024 instances: 0.162 ms at eight per
// wave, 0.149 at four, 0.142 at two or one).
constexpr int kSmallFullWaves = 256, kSmallSpreadWaves = 512;

hipError_t launch_small_pass(const SolveParams &p, hipStream_t s)
{
    if (p.n <= 8 && (p.B + 7) / 8 >= kSmallFullWaves) {
        const size_t lds = SmallLayout<kSmallMaxStages, 8>::total(p.n);
        hipLaunchKernelGGL((solve_small_kernel<kSmallMaxStages, 8>), dim3(unsigned((p.B + 7) / 8)), dim3(64), lds, s,
                           p);
    } else {
        const size_t lds = SmallLayout<kSmallMaxStages, 4>::total(p.n);
        if (p.B <= kSmallSpreadWaves)
            hipLaunchKernelGGL((solve_small_kernel<kSmallMaxStages, 16, 1>), dim3(unsigned(p.B)), dim3(64), lds, s,
                               p);
        else if ((p.B + 1) / 2 <= kSmallSpreadWaves)
            hipLaunchKernelGGL((solve_small_kernel<kSmallMaxStages, 16, 2>), dim3(unsigned((p.B + 1) / 2)), dim3(64),
                               lds, s, p);
        else
            hipLaunchKernelGGL((solve_small_kernel<kSmallMaxStages, 16>), dim3(unsigned((p.B + 3) / 4)), dim3(64),
                               lds, s, p);
    }
    return hipGetLastError();
}

} // namespace gwtf
