// Batched simulation of GWTF's decentralized flow heuristic (paper Sec. V-C:
// Request Flow, Request Change, Request Redirect under simulated annealing;
// Sec. VI setup: T0 = 1.7, alpha = 0.95), for scoring it against the exact
// optimum the solver passes compute (Sec. VI flow ablation).
//
// One wave per instance, one lane per relay node (S * n <= 64).  The instance
// lives in LDS: link costs, node arrays, and one slot per unit of capacity
// (a slot holds one microbatch: its outflow to the next hop's slot or to the
// data node D, and its inflow from the previous hop's slot or from D).
// Rounds are synchronous:
//   1. cost to the sink of every used slot, from the last stage to the first;
//   2. Request Flow: every relay with no unpaired outflow and a free slot
//      asks the next-stage relay whose unpaired outflow minimises its cost to
//      the sink plus the link cost (lowest index on ties); a target approves
//      its lowest-index requester, D as sink its requesters in index order
//      while it has flow left; D as source pairs first-stage unpaired
//      outflows cheapest first (source link plus cost to the sink);
//   3. improvement: stages of even index, then odd ones, each shuffled and
//      split into pairs (proposer, partner); a proposer that sent no Request
//      Flow this round draws a Request Redirect (carry one of the partner's
//      paired flows itself) or a Request Change (swap next hops of one flow
//      each) and takes it when exp((cost_cur - cost_new) / T) > U(0, 1),
//      with Eq. 1 link costs summed or maximised; an accepted move cools the
//      proposer's T by alpha.
// Moves of different pairs touch disjoint slots, and a stage's moves touch
// only the in-links of the next stage's slots and the out-links of the
// previous stage's, so all pairs of all stages of one parity run at once.
// Random numbers: Philox4x64-10 (Salmon et al., SC 2011) with key (seed,
// instance) and counter (round, stage, stream, index): stream 0 drives the
// stage's Fisher-Yates shuffle, stream 1 pair m's four draws.  The result is
// the set of complete paths (slot chains from D back to D): their number F,
// their Eq. 2 cost, and their node and link flows.
#include "mcf_internal.h"

#include <math.h>

namespace gwtf {
namespace {

constexpr int32_t kSlotNone = -1; // free slot / no inflow yet
constexpr int32_t kData = -2;     // the data node, as source (inflow) or sink (outflow)
constexpr int32_t kNoLink = -1;

struct HeurLayout {
    size_t lk, src, snk, cost, cap, base, unp, req, key, perm, owner, sin, sout, cs, total;
};

__host__ __device__ inline HeurLayout heur_layout(int S, int n, int slots)
{
    HeurLayout L;
    const size_t V = size_t(S) * n, nl = size_t(S - 1) * n * n;
    size_t o = 0;
    auto take = [&](size_t bytes) { size_t at = o; o = align16(o + bytes); return at; };
    L.lk = take(4 * (nl > 0 ? nl : 1));
    L.src = take(4 * size_t(n));
    L.snk = take(4 * size_t(n));
    L.cost = take(4 * V);
    L.cap = take(4 * V);
    L.base = take(4 * (V + 1));
    L.unp = take(4 * V);
    L.req = take(4 * V);
    L.key = take(4 * V);
    L.perm = take(4 * V);
    L.owner = take(size_t(slots));
    L.sin = take(2 * size_t(slots));
    L.sout = take(2 * size_t(slots));
    L.cs = take(4 * size_t(slots));
    L.total = o;
    return L;
}

// Philox4x64-10: ten rounds of two 64 x 64 -> 128-bit products of counter
// words 0 and 2 with fixed multipliers, the key bumped by two Weyl constants
// between rounds.
__device__ inline void philox(uint64_t c0, uint64_t c1, uint64_t c2, uint64_t c3, uint64_t k0, uint64_t k1,
                              uint64_t out[4])
{
    const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
    const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
#pragma unroll 1 // rolled: the unrolled rounds cost a wave per SIMD in registers
    for (int r = 0; r < 10; ++r) {
        if (r > 0) {
            k0 += W0;
            k1 += W1;
        }
        const uint64_t hi0 = __umul64hi(M0, c0), lo0 = M0 * c0;
        const uint64_t hi1 = __umul64hi(M1, c2), lo1 = M1 * c2;
        const uint64_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
        c0 = n0;
        c1 = lo1;
        c2 = n2;
        c3 = lo0;
    }
    out[0] = c0;
    out[1] = c1;
    out[2] = c2;
    out[3] = c3;
}

// A draw in [0, m) from the high 32 bits of a word.
__device__ inline int32_t draw_below(uint64_t w, uint32_t m) { return int32_t(((w >> 32) * uint64_t(m)) >> 32); }

struct Inst {
    int S, n, V;
    int32_t *lk, *src, *snk, *cost, *cap, *base, *unp, *req, *key, *perm, *cs;
    uint8_t *owner;
    int16_t *sin, *sout;

    __device__ int stage(int v) const { return v / n; }
    __device__ int idx(int v) const { return v - (v / n) * n; }
    __device__ int node_at(int32_t slot) const { return slot == kData ? kData : int(owner[slot]); }
    // link cost x -> y (either end may be the data node)
    __device__ int32_t edge(int x, int y) const
    {
        if (x == kData) return src[idx(y)];
        if (y == kData) return snk[idx(x)];
        return lk[(stage(x) * n + idx(x)) * n + idx(y)];
    }
    __device__ int32_t ccost(int x) const { return x == kData ? 0 : cost[x]; }
    // Eq. 1 cost of the link x -> y, doubled: 2 * link + c_x + c_y
    __device__ int64_t E(int x, int y) const { return 2 * int64_t(edge(x, y)) + ccost(x) + ccost(y); }
    __device__ int lowest_free(int v) const
    {
        for (int s = base[v]; s < base[v + 1]; ++s)
            if (sout[s] == kSlotNone) return s;
        return kSlotNone;
    }
    // q-th (from 0) used slot of v, or q-th paired slot when paired_only
    __device__ int nth(int v, int q, bool paired_only) const
    {
        for (int s = base[v]; s < base[v + 1]; ++s) {
            if (sout[s] == kSlotNone || (paired_only && sin[s] == kSlotNone)) continue;
            if (q-- == 0) return s;
        }
        return kSlotNone;
    }
};

__device__ inline int wave_popc(uint64_t m) { return __popcll(m); }

__device__ inline int64_t wave_sum64(int64_t x)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
    return x;
}

__device__ inline int32_t wave_max32(int32_t x)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) x = max(x, __shfl_xor(x, o, 64));
    return x;
}

__global__ void __launch_bounds__(64) heuristic_kernel(HeurParams p)
{
    extern __shared__ __align__(16) unsigned char lds[];
    const int b = blockIdx.x, lane = threadIdx.x;
    const int S = p.S, n = p.n, V = S * n;
    const int64_t nl = int64_t(S - 1) * n * n;
    const HeurLayout L = heur_layout(S, n, p.max_slots);
    Inst I;
    I.S = S;
    I.n = n;
    I.V = V;
    I.lk = reinterpret_cast<int32_t *>(lds + L.lk);
    I.src = reinterpret_cast<int32_t *>(lds + L.src);
    I.snk = reinterpret_cast<int32_t *>(lds + L.snk);
    I.cost = reinterpret_cast<int32_t *>(lds + L.cost);
    I.cap = reinterpret_cast<int32_t *>(lds + L.cap);
    I.base = reinterpret_cast<int32_t *>(lds + L.base);
    I.unp = reinterpret_cast<int32_t *>(lds + L.unp);
    I.req = reinterpret_cast<int32_t *>(lds + L.req);
    I.key = reinterpret_cast<int32_t *>(lds + L.key);
    I.perm = reinterpret_cast<int32_t *>(lds + L.perm);
    I.owner = lds + L.owner;
    I.sin = reinterpret_cast<int16_t *>(lds + L.sin);
    I.sout = reinterpret_cast<int16_t *>(lds + L.sout);
    I.cs = reinterpret_cast<int32_t *>(lds + L.cs);

    const bool node = lane < V;
    const int v = lane, k = node ? lane / n : 0, i = node ? lane - k * n : 0;

    // ---- ingest and checks ----
    int32_t cap = node ? p.cap[int64_t(b) * V + v] : 0;
    int32_t cst = node ? p.cost[int64_t(b) * V + v] : 0;
    bool bad = node && (cap < 0 || cst < 0);
    int32_t maxc = cst;
    for (int64_t q = lane; q < nl; q += 64) {
        const int32_t w = p.arc[int64_t(b) * nl + q];
        I.lk[q] = w;
        bad |= w < kNoLink;
        maxc = max(maxc, w);
    }
    for (int q = lane; q < n; q += 64) {
        const int32_t a = p.src ? p.src[int64_t(b) * n + q] : 0, z = p.snk ? p.snk[int64_t(b) * n + q] : 0;
        I.src[q] = a;
        I.snk[q] = z;
        bad |= a < 0 || z < 0;
        maxc = max(maxc, max(a, z));
    }
    const int32_t supply = p.supply[b];
    // slot ranges: inclusive scan of the capacities over the lanes
    int64_t incl = node ? max(cap, 0) : 0;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int64_t t = __shfl_up(incl, o, 64);
        if (lane >= o) incl += t;
    }
    const int64_t total_cap = __shfl(incl, 63, 64);
    maxc = wave_max32(maxc);
    int32_t status = 0;
    if (__any(bad) || supply < 0 || total_cap > p.max_slots) status = 1;
    else if (int64_t(2 * S + 2) * maxc >= (int64_t(1) << 30)) status = 2;
    int src_left = supply, sink_left = supply;
    if (status == 0) {
        if (node) {
            I.cost[v] = cst;
            I.cap[v] = cap;
            I.base[v] = int32_t(incl - cap);
            for (int s = int(incl - cap); s < int(incl); ++s) {
                I.owner[s] = uint8_t(v);
                I.sin[s] = kSlotNone;
                I.sout[s] = kSlotNone;
            }
        }
        if (lane == 0) I.base[V] = int32_t(total_cap);
        __syncthreads();
        // initial complete paths, laid out in order by lane 0
        if (p.paths && p.num_paths > 0) {
            int32_t ok = 1;
            if (lane == 0) {
                for (int q = 0; q < p.num_paths && ok; ++q) {
                    const int32_t *path = p.paths + (int64_t(b) * p.num_paths + q) * S;
                    if (path[0] < 0) continue;
                    if (src_left <= 0 || sink_left <= 0) {
                        ok = 0;
                        break;
                    }
                    int32_t prev = kData;
                    for (int kk = 0; kk < S && ok; ++kk) {
                        const int32_t j = path[kk];
                        if (j < 0 || j >= n) {
                            ok = 0;
                            break;
                        }
                        const int w = kk * n + j;
                        if (prev != kData && I.edge(I.owner[prev], w) == kNoLink) {
                            ok = 0;
                            break;
                        }
                        const int z = I.lowest_free(w);
                        if (z == kSlotNone) {
                            ok = 0;
                            break;
                        }
                        I.sin[z] = int16_t(prev);
                        I.sout[z] = kData;
                        if (prev != kData) I.sout[prev] = int16_t(z);
                        prev = z;
                    }
                    if (ok) {
                        --src_left;
                        --sink_left;
                    }
                }
            }
            ok = __shfl(ok, 0, 64);
            src_left = __shfl(src_left, 0, 64);
            sink_left = __shfl(sink_left, 0, 64);
            if (!ok) status = 1;
            __syncthreads();
        }
    }

    double T = p.t0;
    int32_t acc = 0;
    int64_t approvals = 0;
    if (status == 0) {
        const uint64_t key0 = p.seed, key1 = uint64_t(b);
        for (int r = 0; r < p.rounds; ++r) {
            // ---- cost to the sink, last stage first; unpaired outflow and
            // used slots of each relay ----
            int32_t unp = kSlotNone, used = 0;
            for (int kk = S - 1; kk >= 0; --kk) {
                if (node && k == kk) {
                    for (int s = I.base[v]; s < I.base[v + 1]; ++s) {
                        const int32_t o = I.sout[s];
                        if (o == kSlotNone) continue;
                        ++used;
                        if (unp == kSlotNone && I.sin[s] == kSlotNone) unp = s;
                        I.cs[s] = cst + I.edge(v, I.node_at(o)) + (o == kData ? 0 : I.cs[o]);
                    }
                    I.unp[v] = unp;
                }
                __syncthreads();
            }
            // ---- Request Flow: choose targets ----
            int32_t req = kSlotNone;
            if (node && unp == kSlotNone && used < cap) {
                if (k == S - 1) {
                    if (sink_left > 0) req = kData;
                } else {
                    int32_t best = 0;
                    for (int j = 0; j < n; ++j) {
                        const int w = (k + 1) * n + j, u = I.unp[w];
                        const int32_t l = I.lk[(k * n + i) * n + j];
                        if (u == kSlotNone || l == kNoLink) continue;
                        const int32_t score = I.cs[u] + l;
                        if (req == kSlotNone || score < best) {
                            best = score;
                            req = w;
                        }
                    }
                }
            }
            if (node) {
                I.req[v] = req;
                I.key[v] = (k == 0 && unp != kSlotNone) ? I.src[i] + I.cs[unp] : 0;
            }
            __syncthreads();
            // approvals: lowest requester per relay target; D as sink in
            // index order while it has flow left
            const uint64_t sink_reqs = __ballot(node && req == kData);
            bool win = false;
            if (req >= 0) {
                win = true;
                for (int q = k * n; q < v; ++q)
                    if (I.req[q] == req) win = false;
            } else if (req == kData) {
                win = wave_popc(sink_reqs & ((uint64_t(1) << v) - 1)) < sink_left;
            }
            // D as source: first-stage unpaired outflows, cheapest first
            bool paired_by_data = false;
            if (node && k == 0 && unp != kSlotNone && src_left > 0) {
                const int32_t mine = I.key[v];
                int rank = 0;
                for (int j = 0; j < n; ++j) {
                    if (j == i || I.unp[j] == kSlotNone) continue;
                    const int32_t other = I.key[j];
                    rank += other < mine || (other == mine && j < i);
                }
                paired_by_data = rank < src_left;
            }
            const int data_pairs = wave_popc(__ballot(paired_by_data));
            const int sink_wins = wave_popc(__ballot(win && req == kData));
            approvals += wave_popc(__ballot(win));
            __syncthreads();
            if (paired_by_data) I.sin[unp] = kData;
            if (win) {
                const int z = I.lowest_free(v);
                if (req == kData) {
                    I.sout[z] = kData;
                } else {
                    const int u = I.unp[req];
                    I.sout[z] = int16_t(u);
                    I.sin[u] = int16_t(z);
                }
                I.sin[z] = kSlotNone;
            }
            src_left -= data_pairs;
            sink_left -= sink_wins;
            __syncthreads();

            // ---- improvement: even stages, then odd ones ----
            const bool improver = node && req == kSlotNone;
            for (int parity = 0; parity < 2; ++parity) {
                const bool active = node && (k & 1) == parity;
                if (active && i == 0) {
                    // Fisher-Yates shuffle of the stage (stream 0)
                    int32_t *pm = I.perm + k * n;
                    for (int j = 0; j < n; ++j) pm[j] = j;
                    uint64_t words[4];
                    int word = 4, block = 0;
                    for (int j = n - 1; j >= 1; --j) {
                        if (word == 4) {
                            philox(uint64_t(r), uint64_t(k), 0, uint64_t(block++), key0, key1, words);
                            word = 0;
                        }
                        const int t = draw_below(words[word++], uint32_t(j + 1));
                        const int32_t x = pm[j];
                        pm[j] = pm[t];
                        pm[t] = x;
                    }
                }
                __syncthreads();
                if (active && improver) {
                    const int32_t *pm = I.perm + k * n;
                    int pos = 0;
                    while (pos < n - 1 && pm[pos] != i) ++pos; // pm is a permutation of 0..n-1
                    if ((pos & 1) == 0 && pos + 1 < n) {
                        const int a = v, bn = k * n + pm[pos + 1], m = pos >> 1;
                        uint64_t w[4];
                        philox(uint64_t(r), uint64_t(k), 1, uint64_t(m), key0, key1, w);
                        int used_a = 0, used_b = 0, paired_b = 0;
                        for (int s = I.base[a]; s < I.base[a + 1]; ++s) used_a += I.sout[s] != kSlotNone;
                        for (int s = I.base[bn]; s < I.base[bn + 1]; ++s) {
                            used_b += I.sout[s] != kSlotNone;
                            paired_b += I.sout[s] != kSlotNone && I.sin[s] != kSlotNone;
                        }
                        const bool can_redirect = used_a < cap && paired_b > 0;
                        const bool can_change = used_a > 0 && used_b > 0;
                        if (can_redirect || can_change) {
                            const bool redirect = can_redirect && can_change ? (w[0] & 1) != 0 : can_redirect;
                            const double U = double(w[3] >> 11) * (1.0 / 9007199254740992.0);
                            if (redirect) {
                                const int y = I.nth(bn, draw_below(w[1], uint32_t(paired_b)), true);
                                const int32_t up = I.sin[y], dn = I.sout[y];
                                const int un = I.node_at(up), dw = I.node_at(dn);
                                if (I.edge(un, a) != kNoLink && I.edge(a, dw) != kNoLink) {
                                    const int64_t c0 = I.E(un, bn), c1 = I.E(bn, dw), n0 = I.E(un, a), n1 = I.E(a, dw);
                                    const int64_t cur = p.objective ? max(c0, c1) : c0 + c1;
                                    const int64_t nxt = p.objective ? max(n0, n1) : n0 + n1;
                                    if (exp(double(cur - nxt) * 0.5 / T) > U) {
                                        const int z = I.lowest_free(a);
                                        I.sin[z] = int16_t(up);
                                        I.sout[z] = int16_t(dn);
                                        if (up != kData) I.sout[up] = int16_t(z);
                                        if (dn != kData) I.sin[dn] = int16_t(z);
                                        I.sin[y] = kSlotNone;
                                        I.sout[y] = kSlotNone;
                                        T *= p.alpha;
                                        ++acc;
                                    }
                                }
                            } else {
                                const int x = I.nth(a, draw_below(w[1], uint32_t(used_a)), false);
                                const int y = I.nth(bn, draw_below(w[2], uint32_t(used_b)), false);
                                const int32_t ox = I.sout[x], oy = I.sout[y];
                                const int nx = I.node_at(ox), ny = I.node_at(oy);
                                if (nx != ny && I.edge(a, ny) != kNoLink && I.edge(bn, nx) != kNoLink) {
                                    const int64_t c0 = I.E(a, nx), c1 = I.E(bn, ny), n0 = I.E(a, ny), n1 = I.E(bn, nx);
                                    const int64_t cur = p.objective ? max(c0, c1) : c0 + c1;
                                    const int64_t nxt = p.objective ? max(n0, n1) : n0 + n1;
                                    if (exp(double(cur - nxt) * 0.5 / T) > U) {
                                        I.sout[x] = int16_t(oy);
                                        I.sout[y] = int16_t(ox);
                                        if (oy != kData) I.sin[oy] = int16_t(x);
                                        if (ox != kData) I.sin[ox] = int16_t(y);
                                        T *= p.alpha;
                                        ++acc;
                                    }
                                }
                            }
                        }
                    }
                }
                __syncthreads();
            }
        }
    }

    // ---- result: complete paths, stage by stage from the source ----
    int32_t nf = 0, used = 0;
    int64_t mycost = 0;
    if (status == 0) {
        int32_t *complete = I.cs; // cost to the sink is no longer needed
        for (int kk = 0; kk < S; ++kk) {
            if (node && k == kk) {
                for (int s = I.base[v]; s < I.base[v + 1]; ++s) {
                    const int32_t o = I.sout[s], in = I.sin[s];
                    int32_t c = 0;
                    if (o != kSlotNone) {
                        ++used;
                        c = in == kData || (in >= 0 && complete[in]);
                        if (c) {
                            ++nf;
                            mycost += cst + I.edge(v, I.node_at(o)) + (k == 0 ? I.src[i] : 0);
                        }
                    }
                    complete[s] = c;
                }
            }
            __syncthreads();
        }
    }
    const int64_t F = wave_sum64(node && k == 0 ? nf : 0);
    const int64_t cost = wave_sum64(mycost);
    const int64_t accepted = wave_sum64(acc);
    const int64_t dangling = wave_sum64(used - nf);
    if (lane == 0) {
        p.F_out[b] = status == 0 ? F : 0;
        p.cost_out[b] = status == 0 ? cost : 0;
        p.status_out[b] = status;
        if (p.counters) {
            int64_t *c = p.counters + int64_t(b) * 4;
            c[0] = status == 0 ? supply - src_left : 0;
            c[1] = status == 0 ? approvals : 0;
            c[2] = status == 0 ? accepted : 0;
            c[3] = status == 0 ? dangling : 0;
        }
    }
    if (node) {
        const int64_t at = int64_t(b) * V + v;
        if (p.node_flow) p.node_flow[at] = nf;
        if (p.used) p.used[at] = used;
        if (p.accepted) p.accepted[at] = acc;
        if (p.temperature) p.temperature[at] = T;
        if (p.arc_flow && k < S - 1) {
            int32_t *row = p.arc_flow + (int64_t(b) * (S - 1) + k) * n * n + int64_t(i) * n;
            for (int j = 0; j < n; ++j) {
                int32_t cnt = 0;
                if (status == 0)
                    for (int s = I.base[v]; s < I.base[v + 1]; ++s) {
                        const int32_t o = I.sout[s];
                        cnt += o >= 0 && I.cs[s] && I.idx(I.owner[o]) == j;
                    }
                row[j] = cnt;
            }
        }
    }
}

} // namespace

size_t heuristic_lds_bytes(int S, int n, int max_slots) { return heur_layout(S, n, max_slots).total; }

hipError_t launch_heuristic(const HeurParams &p, hipStream_t stream)
{
    const size_t lds = heuristic_lds_bytes(p.S, p.n, p.max_slots);
    if (hipFuncSetAttribute(reinterpret_cast<const void *>(heuristic_kernel),
                            hipFuncAttributeMaxDynamicSharedMemorySize, int(lds)) != hipSuccess)
        (void)hipGetLastError();
    hipLaunchKernelGGL(heuristic_kernel, dim3(unsigned(p.B)), dim3(64), lds, stream, p);
    return hipGetLastError();
}

} // namespace gwtf
