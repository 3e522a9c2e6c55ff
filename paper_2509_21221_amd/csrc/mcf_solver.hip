// Batched min-cost max-flow on layered stage graphs: the solver kernels.
//
// Method (paper Sec. V-A, Eq. 2 objective): successive shortest paths with
// Johnson potentials.  Each instance is owned by one workgroup, which runs
// the whole loop on chip without host round trips:
//
//   repeat
//     label-correcting shortest paths from the source over the residual graph
//       (stage-ordered Gauss-Seidel Bellman-Ford rounds, see below)
//     stop when the sink is unreachable or the supply is exhausted
//     pi(v) <- min(D(v), pi(v) + d(t))        (potential update)
//     walk the predecessor chain from the sink, push the bottleneck delta
//     F += delta, cost += delta * D(t)
//
// Residual graph, kept implicitly (node splitting, paper Sec. III: a node's
// memory caps the microbatches it holds):
//   s -> entry(0,i)          cost src_i, unbounded
//   entry(k,i) -> exit(k,i)  cost c_ki, residual cap - flow   (compute arc)
//   exit(k,i) -> entry(k,i)  cost -c_ki, residual flow        (its reverse)
//   exit(k,i) -> entry(k+1,j) cost a_kij, unbounded           (link, dense)
//   entry(k+1,j) -> exit(k,i) cost -a_kij, residual flow(k,i,j) (reverse link)
//   exit(S-1,i) -> t         cost snk_i, unbounded
// Links form dense n x n matrices read straight from the caller's arc_cost
// (head implicit in the column, residual always unbounded), so only their
// reverse arcs -- the links that carry flow -- need storage: a short list per
// exit vertex (partner, cached cost, flow), at most min(cap, n, supply)
// entries because every partner carries at least one unit.
//
// Labels D are true path costs; the potentials pi make every residual
// reduced cost c + pi(u) - pi(v) >= 0.  Labels and potentials are int32 and
// the per-instance overflow check keeps them below 2^29 in magnitude.
//
// One round = forward sweep (stage 0 -> S-1: dense relaxation of the links
// out of exit vertices whose label changed, then the compute arcs) + sink
// update + backward sweep (stage S-1 -> 0: reverse links pulled from the
// flow lists, then reverse compute arcs).  Rounds repeat until the backward
// sweep changes no exit label.  A changed exit row whose reduced label
// already reaches the sink's reduced label is not relaxed (it cannot lie on
// a path shorter than the current sink label); every vertex whose true
// reduced distance is below d(t) still ends with an exact label, which is all
// the potential update needs.  Strict improvement keeps predecessors a tree.
#include "mcf_device.h"

namespace gwtf {
namespace {

using namespace dev;

template <int WAVES, bool NARROW>
__global__ __launch_bounds__(WAVES * 64) void solve_kernel(SolveParams p)
{
    constexpr int NT = WAVES * 64;
    const int b = blockIdx.x;
    const int S = p.S, n = p.n, SN = S * n, nw = (n + 63) >> 6, V = 2 * SN + 3;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    // Narrow state is the LDS pass (n <= 64): the sequential phases run on
    // wave 0 alone with wave-level syncs.  The wide fallback pass shares
    // every phase across the block.
    constexpr bool SINGLE = NARROW;
    if (!NARROW && !p.route_all && p.route[b] != kRouteFallback) return;

    extern __shared__ __align__(16) unsigned char smem[];
    __shared__ Shared sh;

    StateLayout L = make_layout(S, n, p.list_slots, NARROW);
    State<NARROW> st;
    unsigned char *scratch;
    if (NARROW) {
        st.carve(smem, L);
        scratch = smem + L.total;
    } else {
        st.carve(p.state + size_t(b) * p.state_stride, L);
        scratch = smem;
    }
    int32_t *pbest = reinterpret_cast<int32_t *>(scratch);
    int32_t *parg = pbest + WAVES * n;
    int *scanbuf = reinterpret_cast<int *>(scratch + align16(size_t(8) * WAVES * n));

    const int32_t *gcap = p.cap + size_t(b) * SN;
    const int32_t *gnc = p.ncost + size_t(b) * SN;
    const int32_t *gac = S > 1 ? p.acost + size_t(b) * (S - 1) * n * n : nullptr;
    int32_t *gpot = p.pot + size_t(b) * V;
    const int supply = p.supply[b];

    // ---- ingest + validate (all threads) ----
    if (tid == 0) {
        sh.bad = supply < 0;
        sh.maxc = 0;
        sh.rows = sh.pulls = sh.rounds = sh.augs = 0;
    }
    __syncthreads();
    int bad = 0, mx = 0;
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
    const size_t na = size_t(S > 1 ? S - 1 : 0) * n * n;
    for (size_t e = tid; e < na; e += NT) {
        int a = gac[e];
        bad |= a < -1;
        mx = max(mx, a);
    }
    for (int q = tid; q < V; q += NT) gpot[q] = 0;
    if (bad) atomicOr(&sh.bad, 1);
    atomicMax(&sh.maxc, mx);

    // flow-list capacity per exit vertex: min(cap, n, supply), none in the last stage
    int mine = 0;
    const int per = (SN + NT - 1) / NT, lo = min(SN, tid * per), hi = min(SN, lo + per);
    for (int q = lo; q < hi; ++q) {
        int c = gcap[q];
        mine += (q < (S - 1) * n && c > 0 && supply > 0) ? min(min(c, n), supply) : 0;
    }
    int total;
    int off = block_exclusive_scan<NT>(mine, scanbuf, total);
    for (int q = lo; q < hi; ++q) {
        int c = gcap[q];
        int kq = (q < (S - 1) * n && c > 0 && supply > 0) ? min(min(c, n), supply) : 0;
        st.loff[q] = off;
        st.llen[q] = 0;
        off += kq;
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
    if (NARROW && sh.status == 0 && sh.slots > p.list_slots) {
        if (tid == 0) p.route[b] = kRouteFallback;
        return;
    }
    if (tid == 0) p.route[b] = NARROW ? kRouteLds : kRouteGlobal;

    const uint64_t myrows = wave_rows<WAVES>(wave);
    long long my_rows = 0, my_pulls = 0;
    // Phase clocks (thread 0, wall-clock ticks): forward sweeps, backward
    // sweeps, augmentation + potentials, and the rest (label reset, sink).
    uint64_t tick = 0, clk_fwd = 0, clk_bwd = 0, clk_aug = 0, clk_other = 0;

    // ---- successive shortest paths ----
    if (sh.status == 0) {
        while (sh.F < supply) {
            if (tid == 0) tick = wall_clock64();
            for (int q = tid; q < SN; q += NT) {
                st.din[q] = kInf;
                st.dout[q] = kInf;
                st.prin[q] = kPredNone;
                st.prout[q] = kPredNone;
            }
            for (int w = tid; w < S * nw; w += NT) st.pend[w] = 0;
            __syncthreads();
            for (int j = tid; j < n; j += NT) {
                st.din[j] = st.srcc[j];
                st.prin[j] = kPredSrc;
            }
            if (tid == 0) {
                sh.Dt = kInf;
                sh.predt = -1;
            }
            __syncthreads();

            bool first = true;
            int round_count = 0;
            for (;;) {
                // -------- forward sweep --------
                if (tid == 0) clk_other += lap(tick);
                for (int k = 0; k < S; ++k) {
                    if (k > 0) {
                        bool has = false;
                        for (int w = 0; w < nw; ++w) has |= st.pend[(k - 1) * nw + w] != 0;
                        if (!has) continue; // uniform: nothing reaches stage k this sweep
                        const int dtred = sh.Dt >= kInf ? kInf : sh.Dt - sh.pit;
                        const int32_t *arow = gac + size_t(k - 1) * n * n;
                        for (int c = 0; c < nw; ++c) {
                            const int j = c * 64 + lane;
                            const bool jv = j < n;
                            int best = kInf, arg = -1;
                            for (int w = 0; w < nw; ++w) {
                                uint64_t m = st.pend[(k - 1) * nw + w] & myrows;
                                while (m) {
                                    constexpr int U = 8;
                                    int ri[U], dv[U], av[U];
                                    int cnt = 0;
#pragma unroll
                                    for (int u = 0; u < U; ++u) {
                                        ri[u] = -1;
                                        if (m) {
                                            int bit = __ffsll((unsigned long long)m) - 1;
                                            m &= m - 1;
                                            ri[u] = w * 64 + bit;
                                            cnt++;
                                        }
                                    }
#pragma unroll
                                    for (int u = 0; u < U; ++u) {
                                        dv[u] = kInf;
                                        av[u] = -1;
                                        if (ri[u] >= 0) {
                                            int qq = (k - 1) * n + ri[u];
                                            int d = st.dout[qq];
                                            if (d < kInf && (dtred >= kInf || d - st.pout[qq] < dtred)) {
                                                dv[u] = d;
                                                if (jv) av[u] = arow[size_t(ri[u]) * n + j];
                                            }
                                        }
                                    }
#pragma unroll
                                    for (int u = 0; u < U; ++u) {
                                        if (dv[u] < kInf && av[u] >= 0) {
                                            int cand = dv[u] + av[u];
                                            if (cand < best) {
                                                best = cand;
                                                arg = ri[u];
                                            }
                                        }
                                        if (c == 0 && lane == 0 && dv[u] < kInf) my_rows++;
                                    }
                                    (void)cnt;
                                }
                            }
                            if (jv) {
                                pbest[wave * n + j] = best;
                                parg[wave * n + j] = arg;
                            }
                        }
                        __syncthreads();
                        // combine partial minima, then the compute arcs of stage k
                        auto combine = [&](int j) {
                            int best = kInf, arg = -1;
                            for (int w = 0; w < WAVES; ++w) {
                                int v = pbest[w * n + j];
                                if (v < best) {
                                    best = v;
                                    arg = parg[w * n + j];
                                }
                            }
                            int q = k * n + j;
                            if (best < st.din[q]) {
                                st.din[q] = best;
                                st.prin[q] = arg;
                            }
                            int d = st.din[q];
                            bool chg = false;
                            if (d < kInf && st.flow[q] < st.cap[q] && d + st.cost[q] < st.dout[q]) {
                                st.dout[q] = d + st.cost[q];
                                st.prout[q] = kPredSplit;
                                chg = true;
                            }
                            return chg;
                        };
                        for (int base = wave * 64; base < n; base += NT) {
                            const int j = base + lane;
                            bool chg = j < n ? combine(j) : false;
                            uint64_t bal = __ballot(chg);
                            if (lane == 0 && bal) st.pend[k * nw + (base >> 6)] |= bal;
                        }
                        for (int w = tid; w < nw; w += NT) st.pend[(k - 1) * nw + w] = 0;
                        __syncthreads();
                    } else if (first) {
                        for (int base = wave * 64; base < n; base += NT) {
                            const int j = base + lane;
                            bool chg = false;
                            if (j < n) {
                                int d = st.din[j];
                                if (st.flow[j] < st.cap[j] && d + st.cost[j] < st.dout[j]) {
                                    st.dout[j] = d + st.cost[j];
                                    st.prout[j] = kPredSplit;
                                    chg = true;
                                }
                            }
                            uint64_t bal = __ballot(chg);
                            if (lane == 0 && bal) st.pend[base >> 6] |= bal;
                        }
                        __syncthreads();
                    }
                }
                // -------- sink --------
                if (tid == 0) clk_fwd += lap(tick);
                if (tid == 0) sh.tbest = ~0ull;
                __syncthreads();
                for (int j = tid; j < n; j += NT) {
                    int q = (S - 1) * n + j;
                    if ((st.pend[(S - 1) * nw + (j >> 6)] >> (j & 63)) & 1) {
                        int d = st.dout[q];
                        if (d < kInf) {
                            unsigned long long key =
                                (unsigned long long)(uint32_t)(d + st.snkc[j] + kInf) << 32 | uint32_t(j);
                            atomicMin(&sh.tbest, key);
                        }
                    }
                }
                __syncthreads();
                if (tid == 0) {
                    if (sh.tbest != ~0ull) {
                        int cand = int(uint32_t(sh.tbest >> 32)) - kInf;
                        if (cand < sh.Dt) {
                            sh.Dt = cand;
                            sh.predt = int(uint32_t(sh.tbest));
                        }
                    }
                    sh.any = 0;
                }
                for (int w = tid; w < nw; w += NT) st.pend[(S - 1) * nw + w] = 0;
                __syncthreads();

                // -------- backward sweep --------
                if (tid == 0) clk_other += lap(tick);
                auto back_node = [&](int k, int i, long long &pulls) {
                    int q = k * n + i;
                    bool chg = false;
                    if (k < S - 1) {
                        int off = st.loff[q], len = st.llen[q];
                        int best = kInf, arg = -1;
                        const int32_t *dnext = st.din + (k + 1) * n;
                        for (int e = off; e < off + len; ++e) {
                            int jj = st.lpart[e];
                            int d = dnext[jj];
                            if (d < kInf) {
                                int cand = d - st.lcost[e];
                                if (cand < best) {
                                    best = cand;
                                    arg = jj;
                                }
                            }
                        }
                        pulls += len;
                        if (best < st.dout[q]) {
                            st.dout[q] = best;
                            st.prout[q] = arg;
                            chg = true;
                        }
                    }
                    int d = st.dout[q];
                    if (st.flow[q] > 0 && d < kInf && d - st.cost[q] < st.din[q]) {
                        st.din[q] = d - st.cost[q];
                        st.prin[q] = kPredSplit;
                    }
                    return chg;
                };
                if (SINGLE) {
                    if (wave == 0) {
                        bool anyc = false;
                        for (int k = S - 1; k >= 0; --k) {
                            bool chg = lane < n ? back_node(k, lane, my_pulls) : false;
                            uint64_t bal = __ballot(chg);
                            if (bal) {
                                anyc = true;
                                if (lane == 0) st.pend[k * nw] |= bal;
                            }
                            wave_sync();
                        }
                        if (lane == 0 && anyc) sh.any = 1;
                    }
                } else {
                    bool anyc = false;
                    for (int k = S - 1; k >= 0; --k) {
                        for (int base = wave * 64; base < n; base += NT) {
                            const int i = base + lane;
                            bool chg = i < n ? back_node(k, i, my_pulls) : false;
                            uint64_t bal = __ballot(chg);
                            if (bal) {
                                anyc = true;
                                if (lane == 0) st.pend[k * nw + (base >> 6)] |= bal;
                            }
                        }
                        __syncthreads();
                    }
                    if (lane == 0 && anyc) atomicOr(&sh.any, 1);
                }
                __syncthreads();
                if (tid == 0) {
                    sh.rounds++;
                    clk_bwd += lap(tick);
                }
                first = false;
                if (!sh.any) break;
                // Bellman-Ford settles within |V| passes when the residual
                // graph has no negative cycle; more rounds mean a solver fault.
                if (++round_count > V) {
                    if (tid == 0) sh.status = kStatusInternal;
                    break;
                }
                __syncthreads();
            }
            __syncthreads();
            if (sh.status != 0 || sh.Dt >= kInf) break;

            // -------- potentials + augmentation --------
            const int dred = sh.Dt - sh.pit;
            if (tid == 0) {
                int delta = supply - int(sh.F);
                delta = walk_path<false>(st, gac, S, n, supply, sh.predt, delta);
                if (delta <= 0 || walk_path<true>(st, gac, S, n, supply, sh.predt, delta) < 0) {
                    sh.status = kStatusInternal;
                } else {
                    sh.F += delta;
                    sh.cost += (long long)delta * sh.Dt;
                    sh.augs++;
                }
            }
            for (int q = tid; q < SN; q += NT) {
                st.pout[q] = min(st.dout[q], st.pout[q] + dred);
                int32_t *pi = gpot + 3 + 2 * q;
                *pi = min(st.din[q], *pi + dred);
            }
            __syncthreads();
            if (tid == 0) {
                sh.pit = sh.Dt;
                clk_aug += lap(tick);
            }
            __syncthreads();
            if (sh.status != 0) break;
        }
    }

    // ---- export ----
    if (lane == 0) {
        atomicAdd(reinterpret_cast<unsigned long long *>(&sh.rows), (unsigned long long)my_rows);
    }
    atomicAdd(reinterpret_cast<unsigned long long *>(&sh.pulls), (unsigned long long)my_pulls);
    const bool ok = sh.status == 0;
    int32_t *nf = p.node_flow + size_t(b) * SN;
    for (int q = tid; q < SN; q += NT) {
        nf[q] = ok ? st.flow[q] : 0;
        gpot[4 + 2 * q] = ok ? st.pout[q] : 0;
        if (!ok) gpot[3 + 2 * q] = 0;
    }
    int32_t *af = p.arc_flow + size_t(b) * na;
    for (size_t e = tid; e < na; e += NT) af[e] = 0;
    __syncthreads();
    if (ok) {
        for (int q = tid; q < (S - 1) * n; q += NT) {
            int off = st.loff[q], len = st.llen[q];
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
        s[8] = 0; // step counts are kept by the register pass only
        s[9] = 0;
    }
}

__global__ void export_kernel(const int32_t *nf, int32_t S, int32_t n, int32_t first, int32_t count,
                              int32_t *src_flow, int32_t *snk_flow)
{
    size_t idx = size_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (idx >= size_t(count) * n) return;
    size_t b = idx / n, j = idx % n;
    const int32_t *f = nf + (size_t(first) + b) * S * n;
    if (src_flow) src_flow[idx] = f[j];
    if (snk_flow) snk_flow[idx] = f[size_t(S - 1) * n + j];
}

constexpr int kFallbackWaves = 16;

} // namespace

int fallback_waves() { return kFallbackWaves; }

hipError_t set_lds_limits(size_t max_bytes)
{
    hipError_t e = hipSuccess;
    e = hipFuncSetAttribute(reinterpret_cast<const void *>(solve_kernel<1, true>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, int(max_bytes));
    if (e != hipSuccess) return e;
    e = hipFuncSetAttribute(reinterpret_cast<const void *>(solve_kernel<4, true>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, int(max_bytes));
    if (e != hipSuccess) return e;
    return hipFuncSetAttribute(reinterpret_cast<const void *>(solve_kernel<kFallbackWaves, false>),
                               hipFuncAttributeMaxDynamicSharedMemorySize, int(max_bytes));
}

hipError_t launch_lds_pass(const SolveParams &p, int waves, size_t lds_bytes, hipStream_t s)
{
    if (waves == 1)
        hipLaunchKernelGGL((solve_kernel<1, true>), dim3(p.B), dim3(64), lds_bytes, s, p);
    else
        hipLaunchKernelGGL((solve_kernel<4, true>), dim3(p.B), dim3(256), lds_bytes, s, p);
    return hipGetLastError();
}

hipError_t launch_fallback_pass(const SolveParams &p, size_t lds_bytes, hipStream_t s)
{
    hipLaunchKernelGGL((solve_kernel<kFallbackWaves, false>), dim3(p.B), dim3(kFallbackWaves * 64),
                       lds_bytes, s, p);
    return hipGetLastError();
}

hipError_t launch_export(const int32_t *node_flow_ws, int32_t S, int32_t n, int32_t first, int32_t count,
                         int32_t *src_flow, int32_t *snk_flow, hipStream_t s)
{
    size_t total = size_t(count) * n;
    if (total == 0) return hipSuccess;
    unsigned blocks = unsigned((total + 255) / 256);
    hipLaunchKernelGGL(export_kernel, dim3(blocks), dim3(256), 0, s, node_flow_ws, S, n, first, count,
                       src_flow, snk_flow);
    return hipGetLastError();
}

} // namespace gwtf
