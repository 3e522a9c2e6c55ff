// Stage-pipelined register pass: one workgroup per instance, for pipelines of
// at most 32 stages of at most 64 nodes whose link costs fit in 16 bits.
//
// Same method as the other passes (successive shortest paths with Johnson
// potentials on the node-split stage graph, paper Sec. V-A Eq. 2), with the
// label-correcting step spread over the waves by stage instead of by row:
//
//  * Wave w owns P consecutive stages (k = w*P ...).  For each it keeps, in
//    vector registers, the 16-bit costs of every link into that stage (lane
//    j = receiving node, two rows per register: 32 registers per stage) and
//    the nodes' labels and predecessors (lane = node); capacities, compute
//    costs, node flows and the flow lists of the exits sit in LDS.
//  * Iteration t of stage k relaxes the links from stage k-1's exit labels
//    of the same iteration (only the rows whose label dropped since the stage
//    last saw them), applies its compute arcs in both directions and pulls
//    its reverse links from stage k+1's entry labels of iteration t-1.  A
//    wave sweeps its own stages in order, so a label crosses them within one
//    iteration; between waves the boundary stages' labels travel through LDS
//    mailboxes whose words carry the iteration's parity, and the reader waits
//    on the words themselves.  All waves run concurrently on different
//    stages, without workgroup barriers.
//  * Convergence travels with the labels: each exit-mailbox word of
//    iteration t also carries whether any stage up to that wave's last one
//    changed a label in iteration t, so the wave that owns the last stage
//    learns it for the whole pipeline and, when nothing changed, publishes
//    the sink's key and a stop word; the other waves leave on that word
//    while they wait for a mailbox.
//  * After convergence: potentials (kept in the device workspace), then lane
//    0 of wave 0 walks the path over predecessors staged in LDS and takes the
//    bottleneck from the LDS node flows and flow lists; every wave applies
//    the path to its own stages.
//
// Each mailbox is written by one wave and read by one other.  The reader of an
// exit mailbox (a wave's last-stage labels for iteration t) cannot be
// overtaken: the writer's iteration t+1 needs the reader's first-stage output
// of iteration t, which the reader publishes after its read, so a mailbox
// holds the awaited iteration or the one before it and one parity bit tells
// them apart.  The same holds for the entry mailboxes one iteration behind.
#include "mcf_device.h"
#include "mcf_pipe.h"

namespace gwtf {
namespace {

using namespace dev;

constexpr int kSpinLimit = 1 << 22;
constexpr uint32_t kNoArc16 = 0xffff;
constexpr int kBias = 1 << 30;
// Keyed relaxation: a link candidate is the key label * 64 + row, so one
// unsigned min keeps the smallest label and, among equal labels, the first
// row.  Link costs are then stored times 64 (at most kKeyMaxCost), and an
// unreached row broadcasts kKeyNone, which no real key reaches.
constexpr int kKeyMaxCost = 1023;
constexpr uint32_t kKeyNone = 0xffff0000u;
__host__ __device__ constexpr bool keyed_fits(int64_t V, int64_t maxc)
{
    return maxc <= kKeyMaxCost && (V + 1) * maxc * 64 + 63 < int64_t(kKeyNone);
}

enum : int { kArcSplitFwd = 0, kArcSplitRev = 1, kArcLinkFwd = 2, kArcLinkRev = 3 };

typedef uint32_t u32x32 __attribute__((ext_vector_type(32)));

__device__ __forceinline__ int key_label(uint64_t key) { return int(uint32_t(key >> 32)) - kBias; }

// The sink key of the wave: the smallest label and, among equal labels, the
// lowest lane; ~0 when no lane has one.
__device__ __forceinline__ uint64_t wave_min_key(bool has, int label)
{
    const uint32_t v = has ? uint32_t(label + kBias) : ~0u;
    const uint32_t m = wave_reduce_u32<false>(v);
    if (m == ~0u) return ~0ull;
    const int first = __builtin_ctzll(__ballot(v == m));
    return (uint64_t(m) << 32) | uint32_t(first);
}

// LDS accesses another wave may be racing with.
template <typename T> __device__ __forceinline__ T lds_ld(const T *p)
{
    return __hip_atomic_load(const_cast<T *>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
template <typename T> __device__ __forceinline__ void lds_st(T *p, T v)
{
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

__device__ __forceinline__ int arc_code(int type, int k, int i, int j)
{
    return type | (k << 2) | (i << 7) | (j << 13);
}

// Path-walk table: one word per vertex (entry 2q, exit 2q+1 of node q =
// k*64 + i, so below 4096): the vertex its predecessor arc comes from (13
// bits) and that arc's code (19 bits).
constexpr uint32_t kChainMask = 0x1fff;
constexpr uint32_t kChainDone = 0x1fff; // entry of stage 0 reached from the data node
constexpr uint32_t kChainBad = 0x1ffe;  // no usable predecessor
static_assert(2 * kPipeMaxStages * 64 <= 0x1ffe, "vertex ids below the markers");
__device__ __forceinline__ uint32_t chain_word(uint32_t next, int code) { return next | (uint32_t(code) << 13); }

// predecessors of one node, entry side in the low half, exit side in the high
__device__ __forceinline__ int pred_in(int pp) { return int(int16_t(pp & 0xffff)); }
__device__ __forceinline__ int pred_out(int pp) { return pp >> 16; }
__device__ __forceinline__ int pred_pack(int pi, int po) { return (pi & 0xffff) | (po << 16); }

struct PipeShared {
    unsigned long long final_key;
    int stop;  // iteration at which the search converged; 0 while it runs
    int fault; // a wait ran out, an iteration bound was exceeded, or a self-check failed
    int bad, wide, maxc;
    int plen, delta;
    int stage_tot[kPipeMaxStages];
    long long rows, pulls, steps;
};

// Waits until all 64 words of a mailbox carry parity `par` in bit 0; returns
// this lane's word.  Sets why to 1 if the search stopped meanwhile, 2 if the
// wait ran out.  A wave that has its input raises its issue priority: the
// work between a mailbox read and the next mailbox write is what the other
// waves wait for, so it goes ahead of the three other waves on its SIMD
// (which are polling or doing work nobody waits for yet); the wave drops back
// at the start of its next iteration.
__device__ __forceinline__ uint32_t mailbox_wait(const uint32_t *mb, uint32_t par, const int *stop, int &why)
{
    const int lane = threadIdx.x & 63;
    for (int spins = 0;; ++spins) {
        const uint32_t v = lds_ld(&mb[lane]);
        if (__all((v & 1u) == par)) {
            __builtin_amdgcn_s_setprio(3);
            return v;
        }
        if (lds_ld(stop) != 0) {
            why = 1;
            return ~0u;
        }
        if (spins > kSpinLimit) {
            why = 2;
            return ~0u;
        }
        __builtin_amdgcn_s_sleep(4);
    }
}

template <int W, int P, bool kKeyed>
__global__ __launch_bounds__(64 * W, 1) void solve_pipe_kernel(SolveParams p)
{
    constexpr int NT = 64 * W;
    const int b = blockIdx.x;
    // the unscaled variant runs after the keyed one, on the instances it passed on
    if (!kKeyed && p.route[b] != kRoutePipeWide) return;
    const int S = p.S, n = p.n, SN = S * n, V = 2 * SN + 3;
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int k0 = w * P;                 // this wave's first stage
    const int klast = min(S, k0 + P) - 1; // and last (k0 > klast for idle waves)
    const bool jv = lane < n;

    extern __shared__ __align__(16) unsigned char smem[];
    __shared__ PipeShared ps;
    const PipeLayout L = pipe_layout(S, W, p.list_slots);
    uint32_t *exmb = reinterpret_cast<uint32_t *>(smem + L.exmb); // [W][64] last-stage exit labels << 2 | changed << 1 | parity
    uint32_t *enmb = reinterpret_cast<uint32_t *>(smem + L.enmb); // [W][64] first-stage entry labels << 1 | parity
    int *nf = reinterpret_cast<int *>(smem + L.nf);               // [S][64] node flow
    int *capl = reinterpret_cast<int *>(smem + L.capl);           // [S][64] node capacity
    int *ncl = reinterpret_cast<int *>(smem + L.ncl);             // [S][64] node compute cost
    uint32_t *chain = reinterpret_cast<uint32_t *>(smem + L.chain); // [S][64][entry, exit]
    uint16_t *loff = reinterpret_cast<uint16_t *>(smem + L.loff); // [S][64]
    uint8_t *llen = reinterpret_cast<uint8_t *>(smem + L.llen);   // [S][64]
    int *path = reinterpret_cast<int *>(smem + L.path);           // [2*S*64 + 8]
    int *lamt = reinterpret_cast<int *>(smem + L.lamt);           // flow of each list entry
    uint32_t *lent = reinterpret_cast<uint32_t *>(smem + L.lent); // partner | cost << 8

    const int32_t *gcap = p.cap + size_t(b) * SN;
    const int32_t *gnc = p.ncost + size_t(b) * SN;
    const int32_t *gac = S > 1 ? p.acost + size_t(b) * (S - 1) * n * n : nullptr;
    int32_t *gpot = p.pot + size_t(b) * V;
    const int supply = p.supply[b];

    if (tid == 0) {
        ps.bad = supply < 0;
        ps.wide = 0;
        ps.maxc = 0;
        ps.fault = 0;
        ps.rows = ps.pulls = ps.steps = 0;
    }
    __syncthreads();

    // ---------------- ingest + validate ----------------
    u32x32 lw[P];
    int din[P], dout[P], pp[P], seen[P], seeny[P];
    uint32_t holes = 0; // bit s: some link into stage k0+s is missing
    int srcc = 0, snkc = 0;
    {
        int bad = 0, wide = 0, mx = 0;
#pragma unroll
        for (int s = 0; s < P; ++s) {
            const int k = k0 + s;
            const bool own = k <= klast;
            const int cp = (own && jv) ? gcap[k * n + lane] : 0;
            const int nc = (own && jv) ? gnc[k * n + lane] : 0;
            bad |= (cp < 0) | (nc < 0);
            mx = max(mx, nc);
            u32x32 v = (u32x32)(0xffffffffu);
            int hole = 0;
            if (own && k >= 1) {
                const int32_t *layer = gac + size_t(k - 1) * n * n;
#pragma unroll
                for (int r = 0; r < 32; ++r) {
                    const int a0 = (jv && 2 * r < n) ? layer[(2 * r) * n + lane] : -1;
                    const int a1 = (jv && 2 * r + 1 < n) ? layer[(2 * r + 1) * n + lane] : -1;
                    bad |= (a0 < -1) | (a1 < -1);
                    wide |= (a0 > 65534) | (a1 > 65534);
                    hole |= (jv & (2 * r < n) & (a0 < 0)) | (jv & (2 * r + 1 < n) & (a1 < 0));
                    mx = max(mx, max(a0, a1));
                    // keyed: costs above kKeyMaxCost send the instance on, so
                    // the clamp only keeps the stored word in range
                    const uint32_t c0 = a0 < 0 ? kNoArc16 : kKeyed ? uint32_t(min(a0, kKeyMaxCost)) << 6 : uint32_t(min(a0, 65535));
                    const uint32_t c1 = a1 < 0 ? kNoArc16 : kKeyed ? uint32_t(min(a1, kKeyMaxCost)) << 6 : uint32_t(min(a1, 65535));
                    v[r] = c0 | (c1 << 16);
                }
            }
            lw[s] = v;
            if (__any(hole)) holes |= 1u << s;
            if (own) {
                capl[k * 64 + lane] = cp;
                ncl[k * 64 + lane] = nc;
                nf[k * 64 + lane] = 0;
                if (jv) {
                    gpot[3 + 2 * (k * n + lane)] = 0;
                    gpot[4 + 2 * (k * n + lane)] = 0;
                }
            }
        }
        if (k0 == 0 && jv && p.src) srcc = p.src[size_t(b) * n + lane];
        if (klast == S - 1 && k0 <= klast && jv && p.snk) snkc = p.snk[size_t(b) * n + lane];
        bad |= (srcc < 0) | (snkc < 0);
        mx = max(mx, max(srcc, snkc));
        if (__any(bad)) atomicOr(&ps.bad, 1);
        if (__any(wide)) atomicOr(&ps.wide, 1);
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) mx = max(mx, __shfl_xor(mx, off));
        if (lane == 0) atomicMax(&ps.maxc, mx);
    }
    holes = __builtin_amdgcn_readfirstlane(holes);

    // flow-list capacity of each exit: min(cap, n, supply); none in the last stage
    {
        int base_of[P];
#pragma unroll
        for (int s = 0; s < P; ++s) {
            const int k = k0 + s;
            const bool own = k <= klast && k < S - 1;
            const int cp = own ? capl[k * 64 + lane] : 0;
            const int c = (own && jv && supply > 0 && cp > 0) ? min(min(cp, n), supply) : 0;
            int incl = c;
#pragma unroll
            for (int off = 1; off < 64; off <<= 1) {
                const int up = __shfl_up(incl, off);
                incl += lane >= off ? up : 0;
            }
            base_of[s] = incl - c;
            if (k <= klast && lane == 63) ps.stage_tot[k] = incl;
        }
        __syncthreads();
        long long before = 0;
        for (int kk = 0; kk < k0 && kk < S; ++kk) before += ps.stage_tot[kk];
#pragma unroll
        for (int s = 0; s < P; ++s) {
            const int k = k0 + s;
            if (k > klast) break;
            loff[k * 64 + lane] = uint16_t(min<long long>(before + base_of[s], 65535));
            llen[k * 64 + lane] = 0;
            before += ps.stage_tot[k];
        }
        if (klast == S - 1 && k0 <= klast && lane == 0 && before > p.list_slots) atomicOr(&ps.wide, 2);
    }
    if (tid == 0) {
        gpot[0] = 0;
        gpot[1] = 0;
        gpot[2] = 0;
    }
    __syncthreads();
    int status = 0;
    if (ps.bad) status = 1;
    else if (int64_t(V) * ps.maxc >= kLabelBound) status = 2;
    if (status == 0 && ps.wide) {
        // 16-bit link costs or LDS lists do not fit: the fallback pass
        // solves this instance.
        if (tid == 0) p.route[b] = kRouteFallback;
        return;
    }
    if (kKeyed && status == 0 && !keyed_fits(V, ps.maxc)) {
        // costs above kKeyMaxCost or labels too long for the keys: the
        // unscaled variant solves this instance
        if (tid == 0) p.route[b] = kRoutePipeWide;
        return;
    }

    long long F = 0, cost = 0, augs = 0, rounds = 0;
    int pit = 0;
    bool fault = false;
    uint64_t tick = wall_clock64(), clk_iter = 0, clk_aug = 0, clk_other = 0;

    if (status == 0) {
        while (F < supply) {
            // ---- labels of a fresh search; mailboxes hold iteration 0 ----
            // The flow lists change only between searches: each exit's list
            // and the wave's longest list per stage are read once here.
            int lst_lo[P], lst_len[P], lst_max[P];
#pragma unroll
            for (int s = 0; s < P; ++s) {
                const int q = (k0 + s) * 64 + lane;
                const bool own = k0 + s <= klast && k0 + s + 1 < S;
                lst_lo[s] = own ? int(loff[q]) : 0;
                lst_len[s] = own && jv ? int(llen[q]) : 0;
                lst_max[s] = int(wave_reduce_u32<true>(uint32_t(lst_len[s])));
            }
#pragma unroll
            for (int s = 0; s < P; ++s) {
                const int k = k0 + s;
                din[s] = (k == 0 && jv) ? srcc : kInf;
                dout[s] = kInf;
                pp[s] = pred_pack(k == 0 ? kPredSrc : kPredNone, kPredNone);
                seen[s] = kInf;
                seeny[s] = kInf;
            }
            if (k0 <= klast) {
                if (k0 >= 1) lds_st(&enmb[w * 64 + lane], uint32_t(din[0]) << 1);
                if (klast + 1 < S) lds_st(&exmb[w * 64 + lane], uint32_t(kInf) << 2);
            }
            if (tid == 0) {
                ps.stop = 0;
                ps.final_key = ~0ull;
            }
            __syncthreads();
            clk_other += lap(tick);

            // ---- (1) pipelined label-correcting iterations ----
            long long rows = 0, steps = 0;
            int pulls = 0;
            if (k0 <= klast) {
                for (int t = 1;; ++t) {
                    if (t > 4 * V + 8) {
                        if (lane == 0) atomicOr(&ps.fault, 1);
                        break;
                    }
                    const uint32_t par = uint32_t(t) & 1u;
                    __builtin_amdgcn_s_setprio(0);
                    int why = 0;
                    bool chg = false;
                    uint32_t upch = 0; // 2 if a stage before this wave's changed in iteration t
                    uint64_t skey = ~0ull;
#pragma unroll
                    for (int s = 0; s < P; ++s) {
                        const int k = k0 + s;
                        if (k > klast) break;
                        const int q = k * 64 + lane;
                        const int fl = nf[q], cp = capl[q], nc = ncl[q];
                        int di = din[s], dq = dout[s], pi = pred_in(pp[s]), po = pred_out(pp[s]);
                        const int di0 = di, dq0 = dq;
                        // links from stage k-1's exit labels X
                        auto relax = [&](const int X) {
                            const bool dr = X < seen[s];
                            seen[s] = dr ? X : seen[s];
                            const uint64_t mask = __ballot(dr);
                            rows += __popcll(mask);
                            // rows that dropped, two per cost register, in row order
                            if (mask && kKeyed) {
                                // every row of a group with a dropped row: a row
                                // that did not drop was relaxed with the same label
                                // before, so its key cannot beat the current label
                                const uint32_t xk = X < kInf ? (uint32_t(X) << 6) | uint32_t(lane) : kKeyNone;
                                uint32_t key = kKeyNone;
                                if (!((holes >> s) & 1u)) {
                                    const uint32_t mlo = uint32_t(mask), mhi = uint32_t(mask >> 32);
#pragma unroll
                                    for (int g = 0; g < 8; ++g) {
                                        const uint32_t half = g < 4 ? mlo : mhi;
                                        if (half & (0xffu << (8 * (g & 3)))) {
                                            // the group's eight keys first, so the reads overlap
                                            uint32_t xr[8], cand[8];
#pragma unroll
                                            for (int u = 0; u < 8; ++u) xr[u] = __builtin_amdgcn_readlane(xk, 8 * g + u);
#pragma unroll
                                            for (int u = 0; u < 8; u += 2) {
                                                const uint32_t wd = lw[s][(8 * g + u) >> 1];
                                                cand[u] = xr[u] + (wd & 0xffffu);
                                                cand[u + 1] = xr[u + 1] + (wd >> 16);
                                            }
                                            const uint32_t m0 = min(min(cand[0], cand[1]), cand[2]);
                                            const uint32_t m1 = min(min(cand[3], cand[4]), cand[5]);
                                            const uint32_t m2 = min(min(cand[6], cand[7]), key);
                                            key = min(min(m0, m1), m2);
                                        }
                                    }
                                } else {
                                    // some links are missing (cost 0xffff): skip them
                                    uint64_t m = mask;
                                    while (m) {
                                        const int r = __builtin_ctzll(m);
                                        m &= m - 1;
                                        const uint32_t c = (lw[s][r >> 1] >> (16 * (r & 1))) & 0xffffu;
                                        const uint32_t cand = __builtin_amdgcn_readlane(xk, r) + c;
                                        key = c != kNoArc16 ? min(key, cand) : key;
                                    }
                                }
                                if (key < kKeyNone && int(key >> 6) < di) {
                                    di = int(key >> 6);
                                    pi = int(key & 63u);
                                }
                            } else if (mask) {
                                if (!((holes >> s) & 1u)) {
                                    // one scalar test per group of 8 rows, then one
                                    // bit test per row of a group that has any
                                    const uint32_t mlo = uint32_t(mask), mhi = uint32_t(mask >> 32);
#pragma unroll
                                    for (int g = 0; g < 8; ++g) {
                                        const uint32_t half = g < 4 ? mlo : mhi;
                                        if (half & (0xffu << (8 * (g & 3)))) {
#pragma unroll
                                            for (int r = 8 * g; r < 8 * g + 8; ++r) {
                                                if (half & (1u << (r & 31))) {
                                                    const uint32_t wd = lw[s][r >> 1];
                                                    const int cand = __builtin_amdgcn_readlane(X, r) + int((r & 1) ? wd >> 16 : wd & 0xffffu);
                                                    pi = cand < di ? r : pi;
                                                    di = min(di, cand);
                                                }
                                            }
                                        }
                                    }
                                } else {
                                    // some links are missing (cost 0xffff): skip them
                                    uint64_t m = mask;
                                    while (m) {
                                        const int r = __builtin_ctzll(m);
                                        m &= m - 1;
                                        const uint32_t c = (lw[s][r >> 1] >> (16 * (r & 1))) & 0xffffu;
                                        const int cand = __builtin_amdgcn_readlane(X, r) + int(c);
                                        const bool take = (c != kNoArc16) & (cand < di);
                                        pi = take ? r : pi;
                                        di = take ? cand : di;
                                    }
                                }
                            }
                        };
                        // reverse links, only when some entry label of stage k+1 dropped
                        // since this stage last pulled (lists change only between
                        // searches): four list entries per pass, partner labels from
                        // the partner's lane (the loop runs to the wave's longest
                        // list so every cross-lane read has all lanes active)
                        auto pull = [&](const int Y) {
                            const bool ydr = Y < seeny[s];
                            seeny[s] = ydr ? Y : seeny[s];
                            if (k + 1 < S && __ballot(ydr) != 0) {
                                const int lo = lst_lo[s], len = lst_len[s], maxlen = lst_max[s];
                                for (int e = 0; e < maxlen; e += 4) {
                                    uint32_t ent[4];
#pragma unroll
                                    for (int u = 0; u < 4; ++u) ent[u] = lent[lo + e + u];
                                    // the four partner reads first, then the updates as
                                    // selects, so the reads are in flight together
                                    int dj[4];
#pragma unroll
                                    for (int u = 0; u < 4; ++u) dj[u] = __shfl(Y, e + u < len ? int(ent[u] & 255u) : 0);
#pragma unroll
                                    for (int u = 0; u < 4; ++u) {
                                        const int cand = dj[u] - int(ent[u] >> 8);
                                        const bool take = (e + u < len) & (dj[u] < kInf) & (cand < dq);
                                        dq = take ? cand : dq;
                                        po = take ? int(ent[u] & 255u) : po;
                                    }
                                }
                                pulls += len;
                            }
                        };
                        auto split_rev = [&]() {
                            if (fl > 0 && dq < kInf && dq - nc < di) {
                                di = dq - nc;
                                pi = kPredSplit;
                            }
                        };
                        auto split_fwd = [&]() {
                            if (di < kInf && fl < cp && di + nc < dq) {
                                dq = di + nc;
                                po = kPredSplit;
                            }
                        };
                        // The input held by this wave first (a wave's first stage
                        // pulls from its second's entry labels of iteration t-1,
                        // its second relaxes from its first's exit labels of
                        // iteration t), then the one another wave sends: the work
                        // between a mailbox read and the next mailbox write is
                        // what the waves pass to each other.
                        if (s < P - 1 && k + 1 < S) {
                            pull(din[s + 1]);
                            split_rev();
                        }
                        if (s > 0) relax(dout[s - 1]);
                        if (s == 0 && k >= 1) {
                            // exit labels of stage k-1, iteration t, from the previous wave
                            const uint32_t word = mailbox_wait(&exmb[(w - 1) * 64], par, &ps.stop, why);
                            if (why) break;
                            upch = __builtin_amdgcn_readfirstlane(word) & 2u;
                            relax(int(word >> 2));
                        }
                        split_rev();
                        split_fwd();
                        if (s == P - 1 && k + 1 < S) {
                            // entry labels of stage k+1, iteration t-1, from the next wave
                            const int Y = int(mailbox_wait(&enmb[(w + 1) * 64], par ^ 1u, &ps.stop, why) >> 1);
                            if (why) break;
                            pull(Y);
                            split_rev();
                        }
                        ++steps;
                        chg |= (di != di0) | (dq != dq0);
                        din[s] = di;
                        dout[s] = dq;
                        pp[s] = pred_pack(pi, po);
                        if (s == 0 && k >= 1) lds_st(&enmb[w * 64 + lane], (uint32_t(di) << 1) | par);
                        if (k == klast && k + 1 < S) {
                            const uint32_t ch = (upch | (__any(chg) ? 2u : 0u));
                            lds_st(&exmb[w * 64 + lane], (uint32_t(dq) << 2) | ch | par);
                        }
                        if (k == S - 1) {
                            skey = wave_min_key(jv && dq < kInf, dq + snkc);
                        }
                    }
                    if (why) {
                        if (why == 2 && lane == 0) atomicOr(&ps.fault, 1);
                        break;
                    }
                    // the wave of the last stage: no label changed anywhere in
                    // iteration t ends the search
                    if (klast == S - 1 && upch == 0 && !__any(chg)) {
                        if (lane == 0) {
                            ps.final_key = skey;
                            lds_st(&ps.stop, t);
                        }
                        break;
                    }
                }
            }
            __builtin_amdgcn_s_setprio(0);
#pragma unroll
            for (int off = 32; off > 0; off >>= 1) pulls += __shfl_xor(pulls, off);
            if (lane == 0) {
                atomicAdd(reinterpret_cast<unsigned long long *>(&ps.rows), (unsigned long long)rows);
                atomicAdd(reinterpret_cast<unsigned long long *>(&ps.steps), (unsigned long long)steps);
                atomicAdd(reinterpret_cast<unsigned long long *>(&ps.pulls), (unsigned long long)pulls);
            }
            __syncthreads();
            clk_iter += lap(tick);
            if (ps.fault) {
                fault = true;
                break;
            }
            const uint64_t fk = ps.final_key;
            rounds += ps.stop;
            if (fk == ~0ull) break; // sink unreachable: the flow is maximum

            // ---- (2) stage predecessors ----
            const int Dt = key_label(fk), predt = int(uint32_t(fk));
            const int dred = Dt - pit;
            // The lane index, opaque here so that the per-lane addresses and
            // words below are computed after each search rather than held in
            // registers across the label iterations (which would spill them).
            int ln = lane;
            __asm__ volatile("" : "+v"(ln));
#pragma unroll
            for (int s = 0; s < P; ++s) {
                const int k = k0 + s;
                if (k > klast) break;
                const int q = k * 64 + ln, pi = pred_in(pp[s]), po = pred_out(pp[s]);
                uint32_t ein, eout;
                if (pi == kPredSrc) ein = kChainDone;
                else if (pi == kPredSplit) ein = chain_word(2 * q + 1, arc_code(kArcSplitRev, k, ln, 0));
                else if (pi >= 0 && pi < n && k >= 1) ein = chain_word(2 * ((k - 1) * 64 + pi) + 1, arc_code(kArcLinkFwd, k - 1, pi, ln));
                else ein = kChainBad;
                if (po == kPredSplit) eout = chain_word(2 * q, arc_code(kArcSplitFwd, k, ln, 0));
                else if (po >= 0 && po < n && k + 1 < S) eout = chain_word(2 * ((k + 1) * 64 + po), arc_code(kArcLinkRev, k, ln, po));
                else eout = kChainBad;
                chain[2 * q] = ein;
                chain[2 * q + 1] = eout;
            }
            __syncthreads();
            // potentials of this wave's nodes (the other waves do theirs while
            // wave 0 walks; wave 0 after its walk)
            auto update_potentials = [&]() {
#pragma unroll
                for (int s = 0; s < P; ++s) {
                    const int k = k0 + s;
                    if (k <= klast && jv) {
                        int32_t *pin = gpot + 3 + 2 * (k * n + ln);
                        const int a = pin[0], c = pin[1];
                        pin[0] = min(din[s], a + dred);
                        pin[1] = min(dout[s], c + dred);
                    }
                }
            };
            if (w != 0) update_potentials();

            // ---- (3) wave 0 walks the predecessor chain, then the
            // whole wave takes the bottleneck over the recorded arcs ----
            if (w == 0) {
                // the whole wave follows the chain (uniform values)
                {
                    int len = 0;
                    bool okw = predt >= 0 && predt < n;
                    uint32_t v = 2 * ((S - 1) * 64 + predt) + 1;
                    // A node's two vertices are 2q and 2q+1, and a compute arc
                    // joins them: the partner's word is read with each vertex's
                    // own, so a compute arc and the arc after it take one round.
                    // Every lane writes the (uniform) path entries.
                    static_assert(kChainDone > kChainBad, "one compare finds both markers");
                    while (okw) {
                        // Most nodes are reached at their exit by the compute arc
                        // and at their entry by a link from an exit of the stage
                        // before: two entries and one read per node, with the
                        // tests in scalar arithmetic; anything else takes the
                        // general step below.
                        while (v & 1u) {
                            const uint64_t fb = *reinterpret_cast<const uint64_t *>(&chain[v - 1u]);
                            const uint32_t flo = __builtin_amdgcn_readfirstlane(uint32_t(fb));
                            const uint32_t fhi = __builtin_amdgcn_readfirstlane(uint32_t(fb >> 32));
                            const uint32_t fnx = flo & kChainMask;
                            // exit word leads to the entry, the entry's to an exit
                            // (odd, so no marker: both markers are 0x1ffe and up,
                            // and 0x1fff = done), room for two entries
                            if ((fhi & kChainMask) != v - 1u) break;
                            if ((fnx & 1u) == 0u || fnx == kChainDone) break;
                            if (len > 2 * SN + 2) break;
                            path[len] = int(fhi >> 13);
                            path[len + 1] = int(flo >> 13);
                            len += 2;
                            v = fnx;
                        }
                        // both words of the node in one 8-byte read
                        const uint64_t both = *reinterpret_cast<const uint64_t *>(&chain[v & ~1u]);
                        const uint32_t lo = __builtin_amdgcn_readfirstlane(uint32_t(both));
                        const uint32_t hi = __builtin_amdgcn_readfirstlane(uint32_t(both >> 32));
                        const uint32_t word = (v & 1u) ? hi : lo, part = (v & 1u) ? lo : hi;
                        uint32_t nx = word & kChainMask;
                        if (nx >= kChainBad) {
                            okw = nx == kChainDone;
                            break;
                        }
                        path[len++] = int(word >> 13);
                        if (nx == (v ^ 1u)) {
                            nx = part & kChainMask;
                            if (nx >= kChainBad) {
                                okw = nx == kChainDone;
                                break;
                            }
                            path[len++] = int(part >> 13);
                        }
                        okw = len <= 2 * SN + 4;
                        v = nx;
                    }
                    if (lane == 0) ps.plen = okw ? len : -1;
                }
                __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
                __builtin_amdgcn_wave_barrier();
                const int len = __builtin_amdgcn_readfirstlane(ps.plen);
                int r = supply - int(F);
                for (int e = lane; e < len; e += 64) {
                    const int code = path[e], type = code & 3, kk = (code >> 2) & 31;
                    const int i = (code >> 7) & 63, j = (code >> 13) & 63;
                    const int q = kk * 64 + i;
                    if (type == kArcSplitFwd) r = min(r, capl[q] - nf[q]);
                    else if (type == kArcSplitRev) r = min(r, nf[q]);
                    else if (type == kArcLinkRev) {
                        int amt = 0;
                        for (int x = loff[q]; x < loff[q] + llen[q]; ++x)
                            if (int(lent[x] & 255u) == j) amt = lamt[x];
                        r = min(r, amt);
                    }
                }
                r = int(wave_reduce_u32<false>(uint32_t(r)));
                if (lane == 0) ps.delta = r;
                update_potentials();
            }
            __syncthreads();
            const int len = ps.plen, delta = ps.delta;
            if (len < 0 || delta <= 0) {
                fault = true;
                break;
            }

            // ---- (4) each wave applies the path to its stages ----
            if (k0 <= klast) {
                for (int pass = 0; pass < 2; ++pass) {
                    for (int e = lane; e < len; e += 64) {
                        const int code = path[e], type = code & 3, kk = (code >> 2) & 31;
                        const int i = (code >> 7) & 63, j = (code >> 13) & 63;
                        if (kk < k0 || kk > klast) continue;
                        const int q = kk * 64 + i;
                        if (pass == 0) {
                            if (type == kArcSplitFwd) nf[q] += delta;
                            else if (type == kArcSplitRev) nf[q] -= delta;
                            else if (type == kArcLinkRev) {
                                const int lo = loff[q], hi = lo + llen[q];
                                int le = -1;
                                for (int x = lo; x < hi; ++x)
                                    if (int(lent[x] & 255u) == j) le = x;
                                if (le < 0 || lamt[le] < delta) {
                                    atomicOr(&ps.fault, 1);
                                } else if (lamt[le] == delta) { // the arc empties: move the last entry here
                                    lent[le] = lent[hi - 1];
                                    lamt[le] = lamt[hi - 1];
                                    llen[q] = uint8_t(hi - 1 - lo);
                                } else {
                                    lamt[le] -= delta;
                                }
                            }
                        } else if (type == kArcLinkFwd) {
                            const int lo = loff[q], hi = lo + llen[q];
                            int le = -1;
                            for (int x = lo; x < hi; ++x)
                                if (int(lent[x] & 255u) == j) le = x;
                            if (le >= 0) {
                                lamt[le] += delta;
                            } else if (hi - lo >= min(min(capl[q], n), supply)) {
                                atomicOr(&ps.fault, 1);
                            } else {
                                lent[hi] = uint32_t(j) | (uint32_t(gac[(size_t(kk) * n + i) * n + j]) << 8);
                                lamt[hi] = delta;
                                llen[q] = uint8_t(hi + 1 - lo);
                            }
                        }
                    }
                    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
                    __builtin_amdgcn_wave_barrier();
                }
            }
            F += delta;
            cost += (long long)delta * Dt;
            augs++;
            pit = Dt;
            __syncthreads();
            clk_aug += lap(tick);
            if (ps.fault) {
                fault = true;
                break;
            }
        }
    }

    // ---------------- export ----------------
    const bool ok = status == 0 && !fault;
    int32_t *nfo = p.node_flow + size_t(b) * SN;
    if (k0 <= klast && jv) {
#pragma unroll
        for (int s = 0; s < P; ++s) {
            const int k = k0 + s;
            if (k <= klast) {
                const int q = k * n + lane;
                nfo[q] = ok ? nf[k * 64 + lane] : 0;
                if (!ok) {
                    gpot[3 + 2 * q] = 0;
                    gpot[4 + 2 * q] = 0;
                }
            }
        }
    }
    const size_t na = size_t(S - 1) * n * n;
    int32_t *af = p.arc_flow + size_t(b) * na;
    for (size_t e = tid; e < na; e += NT) af[e] = 0;
    __syncthreads();
    if (ok) {
        for (int q = tid; q < (S - 1) * 64; q += NT) {
            const int k = q >> 6, i = q & 63;
            if (i >= n) continue;
            for (int e = loff[q]; e < loff[q] + llen[q]; ++e) af[(size_t(k) * n + i) * n + (lent[e] & 255u)] = lamt[e];
        }
    }
    if (tid == 0) {
        gpot[0] = 0;
        gpot[1] = 0;
        gpot[2] = ok ? pit : 0;
        p.F_out[b] = ok ? F : 0;
        p.cost_out[b] = ok ? cost : 0;
        p.status_out[b] = status != 0 ? status : (fault ? kStatusInternal : 0);
        p.route[b] = kRouteReg;
        int64_t *st = p.stats + size_t(b) * kStatsPerInstance;
        const double ns_per_tick = 1e6 / double(p.clock_khz > 0 ? p.clock_khz : 100000);
        st[0] = augs;
        st[1] = rounds;
        st[2] = ps.rows;
        st[3] = ps.pulls;
        st[4] = int64_t(double(clk_iter) * ns_per_tick);
        st[5] = 0;
        st[6] = int64_t(double(clk_aug) * ns_per_tick);
        st[7] = int64_t(double(clk_other) * ns_per_tick);
        st[8] = ps.steps;
        st[9] = 0;
    }
}

// Waves and stages per wave for a pipeline of S stages.
void pipe_shape(int S, int &W, int &P)
{
    if (S <= 8) {
        W = 8;
        P = 1;
    } else if (S <= 16) {
        W = 16;
        P = 1;
    } else {
        W = 16;
        P = 2;
    }
}

} // namespace

bool pipe_pass_fits(int S, int n) { return S >= 1 && S <= kPipeMaxStages && n >= 1 && n <= 64; }

int64_t pipe_pass_slots(int S, size_t lds_max)
{
    int W, P;
    pipe_shape(S, W, P);
    const size_t fixed = pipe_layout(S, W, 0).total + sizeof(PipeShared) + 256;
    if (fixed >= lds_max) return 0;
    return std::min<int64_t>(int64_t((lds_max - fixed) / 8), 65535);
}

hipError_t launch_pipe_pass(const SolveParams &p, hipStream_t s)
{
    int W, P;
    pipe_shape(p.S, W, P);
    const size_t lds = pipe_layout(p.S, W, p.list_slots).total;
    // keyed variant first; the unscaled one takes the instances it passed on
    if (W == 8) {
        hipLaunchKernelGGL((solve_pipe_kernel<8, 1, true>), dim3(p.B), dim3(512), lds, s, p);
        hipLaunchKernelGGL((solve_pipe_kernel<8, 1, false>), dim3(p.B), dim3(512), lds, s, p);
    } else if (P == 1) {
        hipLaunchKernelGGL((solve_pipe_kernel<16, 1, true>), dim3(p.B), dim3(1024), lds, s, p);
        hipLaunchKernelGGL((solve_pipe_kernel<16, 1, false>), dim3(p.B), dim3(1024), lds, s, p);
    } else {
        hipLaunchKernelGGL((solve_pipe_kernel<16, 2, true>), dim3(p.B), dim3(1024), lds, s, p);
        hipLaunchKernelGGL((solve_pipe_kernel<16, 2, false>), dim3(p.B), dim3(1024), lds, s, p);
    }
    return hipGetLastError();
}

} // namespace gwtf
