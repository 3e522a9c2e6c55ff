// Stage-pipelined register pass: one workgroup of 8 waves per instance, for
// pipelines of at most 32 stages of at most 64 nodes whose link costs fit in
// 16 bits.
//
// Same method as the other passes (successive shortest paths with Johnson
// potentials on the node-split stage graph, paper Sec. V-A Eq. 2), with the
// label-correcting step spread over the waves by stage instead of by row:
//
//  * Wave w owns P consecutive stages (k = w*P ...).  For each it keeps, in
//    vector registers, the 16-bit costs of every link into that stage (lane
//    j = receiving node, two rows per register: 32 registers per stage), and
//    the nodes' labels, predecessors, flows and potentials (lane = node).
//  * Iteration t of stage k relaxes the links from stage k-1's exit labels
//    of the same iteration (only the rows whose label dropped since the stage
//    last saw them), applies its compute arcs in both directions and pulls
//    its reverse links from stage k+1's entry labels of iteration t-1.  A
//    wave sweeps its own stages in order, so a label crosses them within one
//    iteration; between waves the boundary stages' labels travel through LDS
//    mailboxes whose words carry the iteration's parity, and the reader waits
//    on the words themselves.  All waves run concurrently on different
//    stages, without workgroup barriers.
//  * Convergence is counted per iteration on a ring of LDS counters: the last
//    wave to finish an iteration in which no label changed anywhere publishes
//    the sink's key and a stop word.
//  * After convergence: potentials, then lane 0 of wave 0 walks the path over
//    predecessors staged in LDS and takes the bottleneck from the LDS mirror
//    of node flows and the flow lists; every wave applies the path to its own
//    stages.
//
// Each mailbox is written by one wave and read by one other.  The reader of an
// exit mailbox (stage k's labels for iteration t) cannot be overtaken: the
// writer's iteration t+1 needs the reader's stage k+1 output of iteration t,
// which the reader publishes after its read, so a mailbox holds the awaited
// iteration or the one before it and one parity bit tells them apart.  The
// same holds for the entry mailboxes one iteration behind.
#include "mcf_device.h"
#include "mcf_pipe.h"

namespace gwtf {
namespace {

using namespace dev;

constexpr int kPipeWaves = 8;
constexpr int kPipeThreads = kPipeWaves * 64;
constexpr int kRing = 16; // iterations in flight across the waves: at most kPipeWaves
constexpr int kSpinLimit = 1 << 22;
constexpr uint32_t kNoArc16 = 0xffff;
constexpr int kBias = 1 << 30;

enum : int { kArcSplitFwd = 0, kArcSplitRev = 1, kArcLinkFwd = 2, kArcLinkRev = 3 };

typedef uint32_t u32x32 __attribute__((ext_vector_type(32)));

__device__ __forceinline__ uint64_t pack_key(int label, int idx)
{
    return (uint64_t(uint32_t(label + kBias)) << 32) | uint32_t(idx);
}
__device__ __forceinline__ int key_label(uint64_t key) { return int(uint32_t(key >> 32)) - kBias; }

__device__ __forceinline__ uint64_t wave_min_u64(uint64_t v)
{
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const uint32_t lo = __shfl_xor(uint32_t(v), off), hi = __shfl_xor(uint32_t(v >> 32), off);
        const uint64_t o = (uint64_t(hi) << 32) | lo;
        v = o < v ? o : v;
    }
    return v;
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

struct PipeShared {
    unsigned ring[kRing];
    unsigned long long ring_key[kRing];
    unsigned long long final_key;
    int stop;    // iteration at which the search converged; 0 while it runs
    int fault;   // a wait ran out, or an iteration bound was exceeded
    int bad, wide, maxc;
    int plen, delta;
    int stage_tot[kPipeMaxStages];
    long long rows, pulls, steps;
};

// Waits until all 64 words of a mailbox carry parity `par`; returns this
// lane's label.  Sets *why to 1 if the search stopped meanwhile, 2 if the
// wait ran out.
__device__ __forceinline__ int mailbox_wait(const uint32_t *mb, uint32_t par, const int *stop, int &why)
{
    const int lane = threadIdx.x & 63;
    for (int spins = 0;; ++spins) {
        const uint32_t v = lds_ld(&mb[lane]);
        if (__all((v & 1u) == par)) return int(v >> 1);
        if (lds_ld(stop) != 0) {
            why = 1;
            return kInf;
        }
        if (spins > kSpinLimit) {
            why = 2;
            return kInf;
        }
        __builtin_amdgcn_s_sleep(1);
    }
}

template <int P>
__global__ __launch_bounds__(kPipeThreads, 1) void solve_pipe_kernel(SolveParams p)
{
    const int b = blockIdx.x;
    const int S = p.S, n = p.n, SN = S * n, V = 2 * SN + 3;
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int nw = (S + P - 1) / P;         // waves that own stages
    const int k0 = w * P;                   // this wave's first stage
    const int klast = min(S, k0 + P) - 1;   // and last (k0 > klast for idle waves)
    const bool jv = lane < n;

    extern __shared__ __align__(16) unsigned char smem[];
    __shared__ PipeShared ps;
    const PipeLayout L = pipe_layout(S, p.list_slots);
    uint32_t *exmb = reinterpret_cast<uint32_t *>(smem + L.exmb); // [S][64] exit labels << 1 | parity
    uint32_t *enmb = reinterpret_cast<uint32_t *>(smem + L.enmb); // [S][64] entry labels << 1 | parity
    int *nf = reinterpret_cast<int *>(smem + L.nf);               // [S][64] node flow mirror
    int *capl = reinterpret_cast<int *>(smem + L.capl);           // [S][64]
    int8_t *prin8 = reinterpret_cast<int8_t *>(smem + L.prin);    // [S][64]
    int8_t *prout8 = reinterpret_cast<int8_t *>(smem + L.prout);  // [S][64]
    uint16_t *loff = reinterpret_cast<uint16_t *>(smem + L.loff); // [S][64]
    uint8_t *llen = reinterpret_cast<uint8_t *>(smem + L.llen);   // [S][64]
    int *path = reinterpret_cast<int *>(smem + L.path);           // [2*S*64 + 8]
    int *lamt = reinterpret_cast<int *>(smem + L.lamt);
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
    int capr[P], ncr[P], flow[P], din[P], dout[P], prin[P], prout[P], seen[P], potin[P], potout[P];
    int srcc = 0, snkc = 0;
    {
        int bad = 0, wide = 0, mx = 0;
#pragma unroll
        for (int s = 0; s < P; ++s) {
            const int k = k0 + s;
            const bool own = k <= klast;
            capr[s] = (own && jv) ? gcap[k * n + lane] : 0;
            ncr[s] = (own && jv) ? gnc[k * n + lane] : 0;
            bad |= (capr[s] < 0) | (ncr[s] < 0);
            mx = max(mx, ncr[s]);
            flow[s] = 0;
            potin[s] = potout[s] = 0;
            u32x32 v = (u32x32)(0xffffffffu);
            if (own && k >= 1) {
                const int32_t *layer = gac + size_t(k - 1) * n * n;
#pragma unroll
                for (int r = 0; r < 32; ++r) {
                    const int a0 = (jv && 2 * r < n) ? layer[(2 * r) * n + lane] : -1;
                    const int a1 = (jv && 2 * r + 1 < n) ? layer[(2 * r + 1) * n + lane] : -1;
                    bad |= (a0 < -1) | (a1 < -1);
                    wide |= (a0 > 65534) | (a1 > 65534);
                    mx = max(mx, max(a0, a1));
                    const uint32_t c0 = a0 < 0 ? kNoArc16 : uint32_t(min(a0, 65535));
                    const uint32_t c1 = a1 < 0 ? kNoArc16 : uint32_t(min(a1, 65535));
                    v[r] = c0 | (c1 << 16);
                }
            }
            lw[s] = v;
            if (own) {
                capl[k * 64 + lane] = capr[s];
                nf[k * 64 + lane] = 0;
            }
        }
        if (k0 == 0 && jv && p.src) srcc = p.src[size_t(b) * n + lane];
        if (klast == S - 1 && k0 <= klast && jv && p.snk) snkc = p.snk[size_t(b) * n + lane];
        bad |= (srcc < 0) | (snkc < 0);
        mx = max(mx, max(srcc, snkc));
        if (__any(bad)) atomicOr(&ps.bad, 1);
        if (__any(wide)) atomicOr(&ps.wide, 1);
        mx = max(mx, __shfl_xor(mx, 32));
        for (int off = 16; off > 0; off >>= 1) mx = max(mx, __shfl_xor(mx, off));
        if (lane == 0) atomicMax(&ps.maxc, mx);
    }

    // flow-list capacity of each exit: min(cap, n, supply); none in the last stage
    {
        int base_of[P];
#pragma unroll
        for (int s = 0; s < P; ++s) {
            const int k = k0 + s;
            const bool own = k <= klast && k < S - 1;
            const int c = (own && jv && supply > 0 && capr[s] > 0) ? (min(min(capr[s], n), supply) + 3) & ~3 : 0;
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

    long long F = 0, cost = 0, augs = 0, rounds = 0;
    int pit = 0;
    bool fault = false;
    uint64_t tick = wall_clock64(), clk_iter = 0, clk_aug = 0, clk_other = 0;

    if (status == 0) {
        while (F < supply) {
            // ---- labels of a fresh search; mailboxes hold iteration 0 ----
#pragma unroll
            for (int s = 0; s < P; ++s) {
                const int k = k0 + s;
                din[s] = (k == 0 && jv) ? srcc : kInf;
                dout[s] = kInf;
                prin[s] = k == 0 ? kPredSrc : kPredNone;
                prout[s] = kPredNone;
                seen[s] = kInf;
                if (k > klast) continue;
                if (s == 0 && k >= 1) lds_st(&enmb[k * 64 + lane], uint32_t(din[s]) << 1);
                if (k == klast && k + 1 < S) lds_st(&exmb[k * 64 + lane], uint32_t(kInf) << 1);
            }
            if (tid < kRing) {
                ps.ring[tid] = 0;
                ps.ring_key[tid] = ~0ull;
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
                    if (__builtin_amdgcn_readfirstlane(lds_ld(&ps.stop)) != 0) break;
                    const uint32_t par = uint32_t(t) & 1u;
                    int why = 0;
                    bool chg = false;
                    uint64_t skey = ~0ull;
#pragma unroll
                    for (int s = 0; s < P; ++s) {
                        const int k = k0 + s;
                        if (k > klast) break;
                        // forward input: exit labels of stage k-1, iteration t
                        int X = kInf;
                        if (k >= 1) X = s == 0 ? mailbox_wait(&exmb[(k - 1) * 64], par, &ps.stop, why) : dout[s - 1];
                        // backward input: entry labels of stage k+1, iteration t-1
                        int Y = kInf;
                        if (k + 1 < S && !why)
                            Y = k == klast ? mailbox_wait(&enmb[(k + 1) * 64], par ^ 1u, &ps.stop, why) : din[s + 1];
                        if (why) break;
                        ++steps;
                        int di = din[s], dq = dout[s], pi = prin[s], po = prout[s];
                        const int di0 = di, dq0 = dq;
                        if (k >= 1) {
                            const bool dr = X < seen[s];
                            seen[s] = dr ? X : seen[s];
                            const uint64_t mask = __ballot(dr);
                            rows += __popcll(mask);
                            // rows that dropped, two per cost register, in row order
                            auto relax = [&](int xr, uint32_t c, int r) {
                                const int cand = xr + int(c);
                                const bool take = (c != kNoArc16) & (cand < di);
                                di = take ? cand : di;
                                pi = take ? r : pi;
                            };
                            if (mask) {
#pragma unroll
                                for (int r2 = 0; r2 < 32; ++r2) {
                                    const uint32_t bits = uint32_t(mask >> (2 * r2)) & 3u;
                                    if (bits) {
                                        const uint32_t wd = lw[s][r2];
                                        if (bits & 1u) relax(__builtin_amdgcn_readlane(X, 2 * r2), wd & 0xffffu, 2 * r2);
                                        if (bits & 2u) relax(__builtin_amdgcn_readlane(X, 2 * r2 + 1), wd >> 16, 2 * r2 + 1);
                                    }
                                }
                            }
                        }
                        const int fl = flow[s], nc = ncr[s];
                        if (fl > 0 && dq < kInf && dq - nc < di) {
                            di = dq - nc;
                            pi = kPredSplit;
                        }
                        if (di < kInf && fl < capr[s] && di + nc < dq) {
                            dq = di + nc;
                            po = kPredSplit;
                        }
                        if (k + 1 < S) {
                            // reverse links: four list entries per read, partner
                            // labels from the partner's lane
                            // (the loop runs to the wave's longest list so that every
                            // cross-lane read happens with all lanes active)
                            const int lo = loff[k * 64 + lane], len = jv ? llen[k * 64 + lane] : 0;
                            int maxlen = len;
#pragma unroll
                            for (int off = 32; off > 0; off >>= 1) maxlen = max(maxlen, __shfl_xor(maxlen, off));
                            maxlen = __builtin_amdgcn_readfirstlane(maxlen);
                            for (int e = 0; e < maxlen; e += 4) {
                                const uint4 v4 = *reinterpret_cast<const uint4 *>(&lent[lo + e]);
                                const uint32_t ent[4] = {v4.x, v4.y, v4.z, v4.w};
#pragma unroll
                                for (int u = 0; u < 4; ++u) {
                                    const bool here = e + u < len;
                                    const int j = here ? int(ent[u] & 255u) : 0, c = int(ent[u] >> 8);
                                    const int dj = __shfl(Y, j);
                                    if (here && dj < kInf && dj - c < dq) {
                                        dq = dj - c;
                                        po = j;
                                    }
                                }
                            }
                            pulls += len;
                        }
                        if (fl > 0 && dq < kInf && dq - nc < di) {
                            di = dq - nc;
                            pi = kPredSplit;
                        }
                        chg |= (di != di0) | (dq != dq0);
                        din[s] = di;
                        dout[s] = dq;
                        prin[s] = pi;
                        prout[s] = po;
                        if (s == 0 && k >= 1) lds_st(&enmb[k * 64 + lane], (uint32_t(di) << 1) | par);
                        if (k == klast && k + 1 < S) lds_st(&exmb[k * 64 + lane], (uint32_t(dq) << 1) | par);
                        if (k == S - 1) {
                            const uint64_t key = (jv && dq < kInf) ? pack_key(dq + snkc, lane) : ~0ull;
                            skey = wave_min_u64(key);
                        }
                    }
                    if (why) {
                        if (why == 2 && lane == 0) atomicOr(&ps.fault, 1);
                        break;
                    }
                    // count this wave into iteration t
                    const bool anych = __any(chg);
                    if (lane == 0) {
                        const int slot = t & (kRing - 1);
                        if (skey != ~0ull) atomicMin(&ps.ring_key[slot], skey);
                        const unsigned mine = anych ? 0x101u : 1u;
                        const unsigned total = atomicAdd(&ps.ring[slot], mine) + mine;
                        if ((total & 0xffu) == unsigned(nw)) {
                            if ((total >> 8) == 0) {
                                ps.final_key = lds_ld(&ps.ring_key[slot]);
                                lds_st(&ps.stop, t);
                            } else {
                                lds_st(&ps.ring[slot], 0u);
                                lds_st(&ps.ring_key[slot], ~0ull);
                            }
                        }
                    }
                }
            }
            if (lane == 0) {
                atomicAdd(reinterpret_cast<unsigned long long *>(&ps.rows), (unsigned long long)rows);
                atomicAdd(reinterpret_cast<unsigned long long *>(&ps.steps), (unsigned long long)steps);
            }
#pragma unroll
            for (int off = 32; off > 0; off >>= 1) pulls += __shfl_xor(pulls, off);
            if (lane == 0) atomicAdd(reinterpret_cast<unsigned long long *>(&ps.pulls), (unsigned long long)pulls);
            __syncthreads();
            clk_iter += lap(tick);
            if (ps.fault) {
                fault = true;
                break;
            }
            const uint64_t fk = ps.final_key;
            rounds += ps.stop;
            if (fk == ~0ull) break; // sink unreachable: the flow is maximum

            // ---- (2) potentials; stage predecessors ----
            const int Dt = key_label(fk), predt = int(uint32_t(fk));
            const int dred = Dt - pit;
#pragma unroll
            for (int s = 0; s < P; ++s) {
                const int k = k0 + s;
                if (k > klast) break;
                if (jv) {
                    potin[s] = min(din[s], potin[s] + dred);
                    potout[s] = min(dout[s], potout[s] + dred);
                }
                prin8[k * 64 + lane] = int8_t(prin[s]);
                prout8[k * 64 + lane] = int8_t(prout[s]);
            }
            __syncthreads();

            // ---- (3) lane 0 of wave 0: walk, record, bottleneck ----
            if (tid == 0) {
                int kk = S - 1, i = predt, len = 0, delta = supply - int(F);
                bool at_exit = true, okw = predt >= 0 && predt < n;
                for (int steps_w = 0; okw; ++steps_w) {
                    if (steps_w > 2 * SN + 4) {
                        okw = false;
                        break;
                    }
                    const int q = kk * 64 + i;
                    if (at_exit) {
                        const int pr = prout8[q];
                        if (pr == kPredSplit) {
                            path[len++] = arc_code(kArcSplitFwd, kk, i, 0);
                            delta = min(delta, capl[q] - nf[q]);
                            at_exit = false;
                        } else if (pr >= 0 && pr < n && kk + 1 < S) {
                            int amt = 0;
                            for (int e = loff[q]; e < loff[q] + llen[q]; ++e)
                                if (int(lent[e] & 255u) == pr) amt = lamt[e];
                            path[len++] = arc_code(kArcLinkRev, kk, i, pr);
                            delta = min(delta, amt);
                            kk = kk + 1;
                            i = pr;
                            at_exit = false;
                        } else {
                            okw = false;
                        }
                    } else {
                        const int pr = prin8[q];
                        if (pr == kPredSrc) break;
                        if (pr == kPredSplit) {
                            path[len++] = arc_code(kArcSplitRev, kk, i, 0);
                            delta = min(delta, nf[q]);
                            at_exit = true;
                        } else if (pr >= 0 && pr < n && kk >= 1) {
                            path[len++] = arc_code(kArcLinkFwd, kk - 1, pr, i);
                            kk = kk - 1;
                            i = pr;
                            at_exit = true;
                        } else {
                            okw = false;
                        }
                    }
                }
                ps.plen = okw ? len : -1;
                ps.delta = delta;
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
#pragma unroll
                for (int s = 0; s < P; ++s) {
                    const int k = k0 + s;
                    if (k > klast) break;
                    flow[s] = nf[k * 64 + lane];
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
#pragma unroll
    for (int s = 0; s < P; ++s) {
        const int k = k0 + s;
        if (k <= klast && jv) {
            const int q = k * n + lane;
            nfo[q] = ok ? flow[s] : 0;
            gpot[3 + 2 * q] = ok ? potin[s] : 0;
            gpot[4 + 2 * q] = ok ? potout[s] : 0;
        }
    }
    const size_t na = size_t(S - 1) * n * n;
    int32_t *af = p.arc_flow + size_t(b) * na;
    for (size_t e = tid; e < na; e += kPipeThreads) af[e] = 0;
    __syncthreads();
    if (ok) {
        for (int q = tid; q < (S - 1) * 64; q += kPipeThreads) {
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

} // namespace

PipeLayout pipe_layout_host(int S, int64_t slots) { return pipe_layout(S, slots); }

bool pipe_pass_fits(int S, int n) { return S >= 1 && S <= kPipeMaxStages && n >= 1 && n <= 64; }

int64_t pipe_pass_slots(int S, size_t lds_max)
{
    const size_t fixed = pipe_layout(S, 0).total + sizeof(PipeShared) + 256;
    if (fixed >= lds_max) return 0;
    return std::min<int64_t>(int64_t((lds_max - fixed) / 8), 65535);
}

hipError_t launch_pipe_pass(const SolveParams &p, hipStream_t s)
{
    const size_t lds = pipe_layout(p.S, p.list_slots).total;
    const int P = (p.S + kPipeWaves - 1) / kPipeWaves;
    switch (P) {
    case 1: hipLaunchKernelGGL(solve_pipe_kernel<1>, dim3(p.B), dim3(kPipeThreads), lds, s, p); break;
    case 2: hipLaunchKernelGGL(solve_pipe_kernel<2>, dim3(p.B), dim3(kPipeThreads), lds, s, p); break;
    case 3: hipLaunchKernelGGL(solve_pipe_kernel<3>, dim3(p.B), dim3(kPipeThreads), lds, s, p); break;
    case 4: hipLaunchKernelGGL(solve_pipe_kernel<4>, dim3(p.B), dim3(kPipeThreads), lds, s, p); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

} // namespace gwtf
