// Register-resident solver pass for pipelines of at most 32 stages of at
// most 64 nodes whose link costs fit in 16 bits.
//
// Same method as mcf_solver.hip (successive shortest paths with Johnson
// potentials, stage-ordered Gauss-Seidel Bellman-Ford rounds, paper Sec. V-A
// Eq. 2 objective), laid out so that no step of the label-correcting loop
// waits on global memory:
//
//  * The dense link costs of the instance live in the vector registers of
//    the workgroup for the whole solve: thread (wave w, lane j) holds, for
//    every stage pair k, the costs from rows i = w, w+8, ..., w+56 of stage k
//    to node j of stage k+1, two 16-bit costs per register (124 registers for
//    31 stage pairs).  They are read from HBM once, at ingest.
//  * A forward step (exits of stage k-1 -> entries of stage k) costs one
//    workgroup barrier: each wave relaxes its rows for its lane's column and
//    posts a packed (label, row) 64-bit minimum with an LDS atomic min; after
//    the barrier every wave reads the 64 column minima and evaluates the
//    compute arcs of stage k itself, so all waves hold identical exit labels
//    and pending-row masks in registers for the next step (rows are broadcast
//    with readlane).  Three minimum buffers rotate over executed steps so a
//    buffer is cleared one barrier after its last read.
//  * The sink minimum is computed redundantly by every wave from registers.
//  * The backward sweep (reverse links from the flow lists, reverse compute
//    arcs) runs on wave 0 alone with wave-level ordering only, visiting a
//    stage only when the entry labels of the stage after it changed, with
//    partner labels fetched by cross-lane shuffles.
//  * The augmenting path is recorded once by lane 0 and applied by wave 0 in
//    parallel (decrements, then increments), while the other waves update the
//    potentials.
#include "mcf_device.h"

namespace gwtf {
namespace {

using namespace dev;

constexpr int kRegWaves = 8;
constexpr int kRegThreads = kRegWaves * 64;
constexpr int kRegMaxStages = 32;
constexpr int kRowsPerWave = 64 / kRegWaves;       // 8 source rows per wave and stage pair
constexpr int kWordsPerLayer = kRowsPerWave / 2;   // two 16-bit costs per register
constexpr uint32_t kNoArc16 = 0xffff;
constexpr int kBias = 1 << 30; // makes |label| < 2^29 positive inside a packed key
constexpr int kPathMax = 512;

enum : int { kArcSplitFwd = 0, kArcSplitRev = 1, kArcLinkFwd = 2, kArcLinkRev = 3 };


// The link costs of stage pair k sit in element k of four 32-element vector
// values (one per register word).  The pair index is wave-uniform, so
// reading or writing element k lowers to indirect register addressing
// rather than to memory or branches.
typedef uint32_t u32x32 __attribute__((ext_vector_type(32)));
static_assert(kRegMaxStages <= 32, "one vector element per stage pair");

__device__ __forceinline__ uint64_t pack_key(int label, int idx)
{
    return (uint64_t(uint32_t(label + kBias)) << 32) | uint32_t(idx);
}

__device__ __forceinline__ uint64_t rows_of_wave(int w)
{
    uint64_t m = 0;
#pragma unroll
    for (int r = 0; r < kRowsPerWave; ++r) m |= uint64_t(1) << (w + kRegWaves * r);
    return m;
}

__device__ __forceinline__ int key_label(uint64_t key) { return int(uint32_t(key >> 32)) - kBias; }

__device__ __forceinline__ uint64_t wave_min_u64(uint64_t v)
{
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        uint32_t lo = __shfl_xor(uint32_t(v), off);
        uint32_t hi = __shfl_xor(uint32_t(v >> 32), off);
        uint64_t o = (uint64_t(hi) << 32) | lo;
        v = o < v ? o : v;
    }
    return v;
}

__device__ __forceinline__ int wave_max_i32(int v)
{
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v = max(v, __shfl_xor(v, off));
    return v;
}

__device__ __forceinline__ int wave_min_i32(int v)
{
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v = min(v, __shfl_xor(v, off));
    return v;
}

__device__ __forceinline__ int arc_code(int type, int k, int i, int j)
{
    return type | (k << 2) | (i << 10) | (j << 18);
}

struct RegShared {
    int plen;
    int path[kPathMax];
};

__global__ __launch_bounds__(kRegThreads) void solve_reg_kernel(SolveParams p)
{
    constexpr int NT = kRegThreads;
    const int b = blockIdx.x;
    const int S = p.S, n = p.n, SN = S * n, V = 2 * SN + 3;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const bool jv = lane < n;

    extern __shared__ __align__(16) unsigned char smem[];
    __shared__ Shared sh;
    __shared__ RegShared rs;

    const StateLayout L = make_layout(S, n, p.list_slots, true);
    State<true> st;
    st.carve(smem, L);
    uint64_t *pk = reinterpret_cast<uint64_t *>(smem + L.total);      // [3][64] column minima
    int *scanbuf = reinterpret_cast<int *>(smem + L.total + 3 * 64 * 8); // [NT]

    const int32_t *gcap = p.cap + size_t(b) * SN;
    const int32_t *gnc = p.ncost + size_t(b) * SN;
    const int32_t *gac = S > 1 ? p.acost + size_t(b) * (S - 1) * n * n : nullptr;
    int32_t *gpot = p.pot + size_t(b) * V;
    const int supply = p.supply[b];

    // ---------------- ingest + validate ----------------
    if (tid == 0) {
        sh.bad = supply < 0;
        sh.maxc = 0;
        sh.slots = 0;
        sh.rows = sh.pulls = sh.rounds = sh.augs = 0;
        sh.any = 0; // reused: largest link cost
        sh.maxc_link_holes = 0;
        sh.kmax = 0;
    }
    __syncthreads();
    int bad = 0, mx = 0, mxlink = 0;
    bool any_hole = false;
    for (int q = tid; q < SN; q += NT) {
        int c = gcap[q], w = gnc[q];
        bad |= (c < 0) | (w < 0);
        mx = max(mx, w);
        st.cap[q] = c;
        st.cost[q] = w;
        st.flow[q] = 0;
        st.pout[q] = 0;
    }
    for (int j = tid; j < n; j += NT) {
        int a = p.src ? p.src[size_t(b) * n + j] : 0;
        int z = p.snk ? p.snk[size_t(b) * n + j] : 0;
        bad |= (a < 0) | (z < 0);
        mx = max(mx, max(a, z));
        st.srcc[j] = a;
        st.snkc[j] = z;
    }
    for (int k = tid; k < S; k += NT) st.pend[k] = 0;
    for (int e = tid; e < 3 * 64; e += NT) pk[e] = ~0ull;
    for (int q = tid; q < V; q += NT) gpot[q] = 0;

    // link costs -> registers (each link read exactly once by one thread)
    u32x32 lw0, lw1, lw2, lw3;
#pragma unroll
    for (int e = 0; e < 32; ++e) lw0[e] = lw1[e] = lw2[e] = lw3[e] = 0xffffffffu;
    for (int k = 0; k < S - 1; ++k) {
        uint32_t wv[kWordsPerLayer];
#pragma unroll
        for (int m = 0; m < kWordsPerLayer; ++m) {
            wv[m] = 0;
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int i = wave + kRegWaves * (2 * m + h);
                int a = -1;
                if (i < n && jv) a = gac[(size_t(k) * n + i) * n + lane];
                bad |= a < -1;
                mxlink = max(mxlink, a);
                const uint32_t c16 = (a < 0 || a > 65534) ? kNoArc16 : uint32_t(a);
                any_hole |= (i < n && jv && a == -1);
                wv[m] |= c16 << (16 * h);
            }
        }
        lw0[k] = wv[0];
        lw1[k] = wv[1];
        lw2[k] = wv[2];
        lw3[k] = wv[3];
    }
    if (bad) atomicOr(&sh.bad, 1);
    atomicMax(&sh.maxc, max(mx, mxlink));
    atomicMax(&sh.any, mxlink);
    if (any_hole) atomicOr(&sh.maxc_link_holes, 1);

    int mine = 0, kbig = 0;
    const int per = (SN + NT - 1) / NT, lo = min(SN, tid * per), hi = min(SN, lo + per);
    for (int q = lo; q < hi; ++q) {
        int c = gcap[q];
        int kq = (q < (S - 1) * n && c > 0 && supply > 0) ? min(min(c, n), supply) : 0;
        mine += kq;
        kbig = max(kbig, kq);
    }
    atomicMax(&sh.kmax, kbig);
    int total;
    int off0 = block_exclusive_scan<NT>(mine, scanbuf, total);
    for (int q = lo; q < hi; ++q) {
        int c = gcap[q];
        int kq = (q < (S - 1) * n && c > 0 && supply > 0) ? min(min(c, n), supply) : 0;
        st.loff[q] = off0;
        st.llen[q] = 0;
        off0 += kq;
    }
    if (tid == 0) {
        int status = 0;
        if (sh.bad) status = 1;
        else if (int64_t(V) * sh.maxc >= kLabelBound) status = 2;
        sh.status = status;
        sh.slots = total;
        sh.F = 0;
        sh.cost = 0;
        sh.pit = 0;
    }
    __syncthreads();
    if (sh.status == 0 && (sh.slots > p.list_slots || sh.any > 65534)) {
        if (tid == 0) p.route[b] = kRouteFallback;
        return;
    }
    if (tid == 0) p.route[b] = kRouteReg;

    long long my_pulls = 0, wave_rows = 0, fwd_steps = 0, bwd_steps = 0;
    const int lq = min(lane, n - 1);            // in-bounds stand-in index for lanes >= n
    const uint64_t myrows = rows_of_wave(wave); // rows i == wave (mod 8)
    const int kmax = __builtin_amdgcn_readfirstlane(sh.kmax);
    int cur = 0;                                 // column-minimum buffer of the next executed step
    uint64_t tick = 0, clk_fwd = 0, clk_bwd = 0, clk_aug = 0, clk_other = 0;
    const bool holes = __builtin_amdgcn_readfirstlane(sh.maxc_link_holes) != 0;

    if (sh.status == 0) {
        int pit = 0; // potential of the sink (uniform)
        while (sh.F < supply) {
            if (tid == 0) tick = wall_clock64();
            for (int q = tid; q < SN; q += NT) {
                st.din[q] = q < n ? st.srcc[q] : kInf;
                st.dout[q] = kInf;
                st.prin[q] = q < n ? kPredSrc : kPredNone;
                st.prout[q] = kPredNone;
            }
            __syncthreads();

            int Dt = kInf, predt = -1;
            uint32_t in_dirty = 0xffffffffu; // stages whose entry labels changed since their pull
            bool first = true;
            int round_count = 0;
            for (;;) {
                if (tid == 0) clk_other += lap(tick);
                // ------------- forward sweep (all waves) -------------
                const int dtred = __builtin_amdgcn_readfirstlane(Dt >= kInf ? kInf : Dt - pit);
                int dprev, pprev;
                uint64_t pend_prev;
                if (first) {
                    const int d = st.srcc[lq];
                    const int fl = st.flow[lq], cp = st.cap[lq], nc = st.cost[lq];
                    const bool chg = jv && fl < cp;
                    dprev = chg ? d + nc : kInf;
                    pend_prev = __ballot(chg);
                    if (wave == 0 && chg) {
                        st.dout[lane] = d + nc;
                        st.prout[lane] = kPredSplit;
                    }
                } else {
                    const int d = st.dout[lq];
                    dprev = jv ? d : kInf;
                    pend_prev = st.pend[0];
                }
                pprev = st.pout[lq];
                // stages whose exits were seeded by the last backward sweep
                const uint64_t seeded_stages = __ballot(lane > 0 && lane < S && st.pend[lane] != 0);
                for (int k = 1; k < S;) {
                    if (pend_prev == 0) {
                        // Nothing reaches stage k, so its pending exits are the
                        // seeded ones: jump to the next seeded stage m and
                        // continue with step m + 1 (or stop).
                        const uint64_t rest = seeded_stages & (~uint64_t(0) << k);
                        if (rest == 0) break;
                        const int m = __builtin_ctzll(rest);
                        const int qm = m * n + lq;
                        const int d = st.dout[qm];
                        dprev = jv ? d : kInf;
                        pprev = st.pout[qm];
                        pend_prev = st.pend[m];
                        k = m + 1;
                        continue;
                    }
                    const int qs = k * n + lq;
                    // stage-k state first: its LDS latency overlaps the relaxation
                    int din_k = st.din[qs], dout_k = st.dout[qs];
                    const int pout_k = st.pout[qs];
                    const int fl = st.flow[qs], cp = st.cap[qs], nc = st.cost[qs];
                    const uint64_t seeded = st.pend[k];
                    fwd_steps++;
                    // Row labels of stage k-1: kInf unless the exit is pending
                    // and below the pruning bound, so the row loop needs no
                    // per-row test; lanes are rows here.
                    const bool live = ((pend_prev >> lane) & 1) && (dtred >= kInf || dprev - pprev < dtred);
                    const int rowlab = live ? dprev : kInf;
                    const uint64_t mine = __ballot(live) & myrows;
                    int best = kInf, arg = -1;
                    if (mine) {
                        const int kk = __builtin_amdgcn_readfirstlane(k - 1);
                        const uint32_t wl[kWordsPerLayer] = {lw0[kk], lw1[kk], lw2[kk], lw3[kk]};
                        if (__popcll(mine) > 3) {
                            // many live rows: all of this wave's rows, no branches
#pragma unroll
                            for (int r = 0; r < kRowsPerWave; ++r) {
                                const int i = wave + kRegWaves * r;
                                const int d = __builtin_amdgcn_readlane(rowlab, i);
                                const uint32_t cw = wl[r / 2];
                                const uint32_t c = (r & 1) ? (cw >> 16) : (cw & 0xffffu);
                                int cand = d + int(c); // kInf + c stays below 2^31
                                if (holes && c == kNoArc16) cand = kInf;
                                const bool lt = cand < best;
                                best = lt ? cand : best;
                                arg = lt ? i : arg;
                            }
                        } else {
                            // few live rows: visit only those
                            uint64_t mm = mine;
                            while (mm) {
                                const int i = __builtin_ctzll(mm);
                                mm &= mm - 1;
                                const int r = i >> 3;
                                const int d = __builtin_amdgcn_readlane(rowlab, i);
                                const uint32_t cw = (r >> 1) == 0 ? wl[0] : (r >> 1) == 1 ? wl[1]
                                                  : (r >> 1) == 2 ? wl[2] : wl[3];
                                const uint32_t c = (cw >> (16 * (r & 1))) & 0xffffu;
                                int cand = d + int(c);
                                if (holes && c == kNoArc16) cand = kInf;
                                const bool lt = cand < best;
                                best = lt ? cand : best;
                                arg = lt ? i : arg;
                            }
                        }
                        wave_rows += __popcll(mine);
                    }
                    uint64_t *buf = pk + cur * 64;
                    if (jv && best < kInf)
                        atomicMin(reinterpret_cast<unsigned long long *>(buf + lane),
                                  (unsigned long long)pack_key(best, arg));
                    __syncthreads();
                    const uint64_t key = buf[lane];
                    const int v = key_label(key);
                    const bool in_imp = jv && key != ~0ull && v < din_k;
                    const int argk = int(uint32_t(key));
                    din_k = in_imp ? v : din_k;
                    const bool chg = jv && din_k < kInf && fl < cp && din_k + nc < dout_k;
                    dout_k = chg ? din_k + nc : dout_k;
                    const uint64_t m = __ballot(chg);
                    const uint64_t mi = __ballot(in_imp);
                    if (wave == 0) {
                        const int q = k * n + lane;
                        if (in_imp) {
                            st.din[q] = din_k;
                            st.prin[q] = int8_t(argk);
                        }
                        if (chg) {
                            st.dout[q] = dout_k;
                            st.prout[q] = kPredSplit;
                        }
                        // the buffer read two executed steps ago is free again
                        pk[(cur == 0 ? 2 : cur - 1) * 64 + lane] = ~0ull;
                    }
                    cur = cur == 2 ? 0 : cur + 1;
                    if (mi) in_dirty |= 1u << k;
                    pend_prev = seeded | m;
                    dprev = jv ? dout_k : kInf;
                    pprev = pout_k;
                    ++k;
                }
                // ------------- sink (every wave, from registers) -------------
                // (pend_prev refers to the last stage here, or is 0 after an early stop)
                if (pend_prev) {
                    int cand = kInf;
                    if (jv && ((pend_prev >> lane) & 1) && dprev < kInf) cand = dprev + st.snkc[lq];
                    uint64_t key = cand < kInf ? pack_key(cand, lane) : ~0ull;
                    key = wave_min_u64(key);
                    if (key != ~0ull) {
                        const int v = key_label(key);
                        if (v < Dt) {
                            Dt = v;
                            predt = int(uint32_t(key));
                        }
                    }
                    Dt = __builtin_amdgcn_readfirstlane(Dt); // identical in every lane
                    predt = __builtin_amdgcn_readfirstlane(predt);
                }
                if (tid == 0) clk_fwd += lap(tick);
                __syncthreads(); // every wave is done reading the forward-sweep state

                // ------------- backward sweep (wave 0) -------------
                if (wave == 0) {
                    if (lane < S) st.pend[lane] = 0;
                    wave_sync();
                    bool anyc = false;
                    int dnext = kInf;
                    int have = -1; // stage whose entry labels dnext holds
                    for (int k = S - 2; k >= 0; --k) {
                        if (!((in_dirty >> (k + 1)) & 1)) continue;
                        in_dirty &= ~(1u << (k + 1));
                        bwd_steps++;
                        const int qs = k * n + lq;
                        if (have != k + 1) {
                            const int d = st.din[qs + n];
                            dnext = jv ? d : kInf;
                        }
                        const int off = st.loff[qs];
                        const int len = jv ? int(st.llen[qs]) : 0;
                        int dout_k = st.dout[qs], din_k = st.din[qs];
                        const int fl = st.flow[qs], nc = st.cost[qs];
                        int best = kInf, arg = -1;
                        // Batches of 8 entries, loads first (the list arrays
                        // are padded so reads past a list stay in bounds).
                        for (int e0 = 0; e0 < kmax; e0 += 8) {
                            int part[8], lc[8], dj[8];
#pragma unroll
                            for (int u = 0; u < 8; ++u) {
                                part[u] = int(st.lpart[off + e0 + u]) & 63;
                                lc[u] = st.lcost[off + e0 + u];
                            }
#pragma unroll
                            for (int u = 0; u < 8; ++u) dj[u] = __shfl(dnext, part[u]);
#pragma unroll
                            for (int u = 0; u < 8; ++u) {
                                // branch-free (bitwise & instead of &&); ties keep the
                                // earlier list entry, deterministic for given inputs
                                const int cand = dj[u] - lc[u];
                                const bool take = (e0 + u < len) & (dj[u] < kInf) & (cand < best);
                                best = take ? cand : best;
                                arg = take ? part[u] : arg;
                            }
                        }
                        my_pulls += len;
                        const bool chg = best < dout_k;
                        bool ichg = false;
                        if (chg) {
                            const int q = k * n + lane;
                            dout_k = best;
                            st.dout[q] = best;
                            st.prout[q] = int8_t(arg);
                            if (fl > 0 && dout_k - nc < din_k) {
                                din_k = dout_k - nc;
                                st.din[q] = din_k;
                                st.prin[q] = kPredSplit;
                                ichg = true;
                            }
                        }
                        const uint64_t m = __ballot(chg);
                        if (m) {
                            anyc = true;
                            if (lane == 0) st.pend[k] = m;
                        }
                        if (__ballot(ichg)) in_dirty |= 1u << k;
                        dnext = jv ? din_k : kInf;
                        have = k;
                        // LDS operations of one wave complete in issue order, so the
                        // next step's cross-lane reads only need the compiler to
                        // keep them after these writes.
                        asm volatile("" ::: "memory");
                    }
                    if (lane == 0) sh.any = anyc;
                }
                if (tid == 0) clk_bwd += lap(tick);
                __syncthreads();
                if (tid == 0) sh.rounds++;
                first = false;
                in_dirty &= 0u; // every wave: all pulls done (only wave 0 reads it)
                if (!sh.any) break;
                if (++round_count > V) {
                    if (tid == 0) sh.status = kStatusInternal;
                    break;
                }
                __syncthreads();
            }
            __syncthreads();
            if (sh.status != 0 || Dt >= kInf) break;

            // ------------- augmentation (wave 0) + potentials (others) -------------
            const int dred = Dt - pit;
            if (wave == 0) {
                if (lane == 0) {
                    int k = S - 1, i = predt, len = 0;
                    bool at_exit = true, okw = predt >= 0 && predt < n;
                    for (int steps = 0; okw; ++steps) {
                        if (steps > 2 * SN + 4) {
                            okw = false;
                            break;
                        }
                        int code;
                        if (at_exit) {
                            const int pr = st.prout[k * n + i];
                            if (pr == kPredSplit) {
                                code = arc_code(kArcSplitFwd, k, i, 0);
                                at_exit = false;
                            } else if (pr >= 0 && k + 1 < S) {
                                code = arc_code(kArcLinkRev, k, i, pr);
                                k = k + 1;
                                i = pr;
                                at_exit = false;
                            } else {
                                okw = false;
                                break;
                            }
                        } else {
                            const int pr = st.prin[k * n + i];
                            if (pr == kPredSrc) break;
                            if (pr == kPredSplit) {
                                code = arc_code(kArcSplitRev, k, i, 0);
                                at_exit = true;
                            } else if (pr >= 0 && k >= 1) {
                                code = arc_code(kArcLinkFwd, k - 1, pr, i);
                                k = k - 1;
                                i = pr;
                                at_exit = true;
                            } else {
                                okw = false;
                                break;
                            }
                        }
                        if (len < kPathMax) rs.path[len] = code;
                        len++;
                    }
                    rs.plen = !okw ? -2 : (len > kPathMax ? -1 : len);
                }
                wave_sync();
                const int plen = rs.plen;
                int delta = -1;
                if (plen == -1) {
                    // longer than the path buffer: two serial walks
                    if (lane == 0) {
                        delta = walk_path<false>(st, gac, S, n, supply, predt, supply - int(sh.F));
                        if (delta <= 0 || walk_path<true>(st, gac, S, n, supply, predt, delta) < 0) delta = -1;
                    }
                    delta = __shfl(delta, 0);
                } else if (plen >= 0) {
                    int r = supply - int(sh.F);
                    for (int e = lane; e < plen; e += 64) {
                        const int code = rs.path[e], type = code & 3, k = (code >> 2) & 255,
                                  i = (code >> 10) & 255, j = (code >> 18) & 255, q = k * n + i;
                        if (type == kArcSplitFwd) r = min(r, st.cap[q] - st.flow[q]);
                        else if (type == kArcSplitRev) r = min(r, st.flow[q]);
                        else if (type == kArcLinkRev) {
                            const int le = list_find(st, q, j);
                            r = le < 0 ? -1 : min(r, st.lamt[le]);
                        }
                    }
                    delta = wave_min_i32(r);
                    if (delta > 0) {
                        bool fail = false;
                        for (int e = lane; e < plen; e += 64) {
                            const int code = rs.path[e], type = code & 3, k = (code >> 2) & 255,
                                      i = (code >> 10) & 255, j = (code >> 18) & 255, q = k * n + i;
                            if (type == kArcSplitFwd) st.flow[q] += delta;
                            else if (type == kArcSplitRev) st.flow[q] -= delta;
                            else if (type == kArcLinkRev) {
                                const int le = list_find(st, q, j);
                                const int left = st.lamt[le] - delta;
                                if (left == 0) {
                                    const int last = st.loff[q] + st.llen[q] - 1;
                                    st.lpart[le] = st.lpart[last];
                                    st.lamt[le] = st.lamt[last];
                                    st.lcost[le] = st.lcost[last];
                                    st.llen[q] = uint8_t(st.llen[q] - 1);
                                } else {
                                    st.lamt[le] = left;
                                }
                            }
                        }
                        wave_sync();
                        for (int e = lane; e < plen; e += 64) {
                            const int code = rs.path[e], type = code & 3, k = (code >> 2) & 255,
                                      i = (code >> 10) & 255, j = (code >> 18) & 255, q = k * n + i;
                            if (type != kArcLinkFwd) continue;
                            const int le = list_find(st, q, j);
                            if (le >= 0) {
                                st.lamt[le] += delta;
                            } else if (st.llen[q] >= min(min(st.cap[q], n), supply)) {
                                fail = true;
                            } else {
                                const int at = st.loff[q] + st.llen[q];
                                st.lpart[at] = uint8_t(j);
                                st.lamt[at] = delta;
                                st.lcost[at] = gac[size_t(q) * n + j];
                                st.llen[q] = uint8_t(st.llen[q] + 1);
                            }
                        }
                        if (__ballot(fail)) delta = -1;
                    }
                }
                if (lane == 0) {
                    if (delta <= 0) {
                        sh.status = kStatusInternal;
                    } else {
                        sh.F += delta;
                        sh.cost += (long long)delta * Dt;
                        sh.augs++;
                    }
                }
            } else {
                for (int q = tid - 64; q < SN; q += NT - 64) {
                    st.pout[q] = min(st.dout[q], st.pout[q] + dred);
                    int32_t *pi = gpot + 3 + 2 * q;
                    *pi = min(st.din[q], *pi + dred);
                }
            }
            __syncthreads();
            pit = Dt;
            if (tid == 0) {
                sh.pit = Dt;
                clk_aug += lap(tick);
            }
            if (sh.status != 0) break;
        }
    }

    // ---------------- export ----------------
    if (lane == 0) atomicAdd(reinterpret_cast<unsigned long long *>(&sh.rows), (unsigned long long)wave_rows);
    if (wave == 0) atomicAdd(reinterpret_cast<unsigned long long *>(&sh.pulls), (unsigned long long)my_pulls);
    const bool ok = sh.status == 0;
    int32_t *nf = p.node_flow + size_t(b) * SN;
    for (int q = tid; q < SN; q += NT) {
        nf[q] = ok ? st.flow[q] : 0;
        gpot[4 + 2 * q] = ok ? st.pout[q] : 0;
        if (!ok) gpot[3 + 2 * q] = 0;
    }
    const size_t na = size_t(S > 1 ? S - 1 : 0) * n * n;
    int32_t *af = p.arc_flow + size_t(b) * na;
    for (size_t e = tid; e < na; e += NT) af[e] = 0;
    __syncthreads();
    if (ok) {
        for (int q = tid; q < (S - 1) * n; q += NT) {
            const int off = st.loff[q], len = st.llen[q];
            for (int e = off; e < off + len; ++e) af[size_t(q) * n + st.lpart[e]] = st.lamt[e];
        }
    }
    if (tid == 0) {
        gpot[0] = 0;
        gpot[1] = 0;
        gpot[2] = ok ? sh.pit : 0;
        p.F_out[b] = ok ? sh.F : 0;
        p.cost_out[b] = ok ? sh.cost : 0;
        p.status_out[b] = sh.status;
        int64_t *s = p.stats + size_t(b) * kStatsPerInstance;
        s[0] = sh.augs;
        s[1] = sh.rounds;
        s[2] = sh.rows;
        s[3] = sh.pulls;
        const double ns_per_tick = 1e6 / double(p.clock_khz > 0 ? p.clock_khz : 100000);
        s[4] = int64_t(double(clk_fwd) * ns_per_tick);
        s[5] = int64_t(double(clk_bwd) * ns_per_tick);
        s[6] = int64_t(double(clk_aug) * ns_per_tick);
        s[7] = int64_t(double(clk_other) * ns_per_tick);
        s[8] = fwd_steps;
        s[9] = bwd_steps;
    }
}

} // namespace

size_t reg_pass_scratch_bytes() { return size_t(3) * 64 * 8 + size_t(4) * kRegThreads; }

bool reg_pass_fits(int S, int n) { return S >= 1 && S <= kRegMaxStages && n >= 1 && n <= 64; }

hipError_t launch_reg_pass(const SolveParams &p, size_t lds_bytes, hipStream_t s)
{
    hipLaunchKernelGGL(solve_reg_kernel, dim3(p.B), dim3(kRegThreads), lds_bytes, s, p);
    return hipGetLastError();
}

} // namespace gwtf
