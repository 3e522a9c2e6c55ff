// Warm-started re-solve of churn variants.  The churn is the paper's (Sec.
// VI: nodes join and leave between iterations); re-solving the exact optimum
// from the previous one is this library's extension, not a method of the
// paper.  Each instance starts from a feasible flow of the same shape,
// typically the optimum of the instance before the churn, and reaches the
// same (F, cost) as a cold solve:
//
//   1. strip: remove whole source-to-sink paths of the start flow until no
//      node carries more than its new capacity, no missing link carries flow
//      and the value does not exceed the supply.  The flow stays feasible.
//   2. cancel: while the residual graph holds a negative cycle, push its
//      bottleneck around it.  A flow is of least cost for its value exactly
//      when no negative residual cycle is left (the cycle optimality
//      condition of min-cost flow).
//   3. augment: successive shortest paths from the data node's source side
//      to its sink side, each on exact distances, until the sink is
//      unreachable or the value equals the supply.  Augmenting a least-cost
//      flow along a shortest path keeps it least-cost, so the result is the
//      same optimum a cold solve reaches (Eq. 2).
//
// One workgroup per instance holds the whole instance in LDS.  Labels are
// corrected in place (stage order is not needed: the residual graph is no
// longer a DAG once cycles are cancelled) with one thread per vertex pulling
// over its incoming residual arcs.  A negative cycle is found in the
// predecessor graph: any cycle there is negative, and one exists once a label
// falls below -(V-1) * max cost, so the graph is checked every fourth round
// and at once when a label crosses that bound.  The check is pointer doubling:
// after ceil(log2 V) + 1 rounds every vertex's ancestor is either a root
// (never relabelled) or a vertex on a cycle.
#include "mcf_internal.h"

#include "gwtf_mcf.h"

namespace gwtf {

namespace {

constexpr int kChurnThreads = 256;
constexpr int32_t kResInf = 0x7fffffff;            // residual of an uncapacitated arc
constexpr int32_t kFlowMax = int32_t(1) << 29;     // bound on start-flow values
constexpr int64_t kChurnRoundCap = int64_t(1) << 20;

// Vertex numbering: 0 = source side s, 1 = sink side t, 2 + 2*nd = in of node
// nd = k*n + i, 3 + 2*nd = out of node nd.
__device__ inline int vin(int nd) { return 2 + 2 * nd; }
__device__ inline int vout(int nd) { return 3 + 2 * nd; }

struct Inst {
    // ac, af: link costs and flows, row r = k*n + i (exit i of stage k) at
    // r * ld, column j = entry j of stage k+1; ld = n + 1 is odd, so the
    // threads of a wave that read along rows or columns of different stages
    // fall on different LDS banks
    int32_t *ac, *af, *cap, *nc, *nf, *src, *snk, *sf, *tf, *d, *pred, *anc, *anc2;
    int S, n, V, ld;
    float inv_n; // 1 / n, for the stage of a node index without an integer division
};

// Stage of node nd: (nd + 1/2) / n is at least 1/(2n) >= 2^-10 away from
// every integer, and the float product is within S * 2^-23 <= 2^-14 of it
// (S * n <= kChurnMaxNodes), so truncation gives nd / n exactly.
__device__ inline int stage_of(const Inst &I, int nd) { return int((float(nd) + 0.5f) * I.inv_n); }

// Residual capacity of the residual arc u -> v (which must exist).
__device__ int32_t residual(const Inst &I, int u, int v)
{
    if (u == 0) return kResInf;
    if (v == 0) return I.sf[(u - 2) >> 1];
    if (v == 1) return kResInf;
    if (u == 1) return I.tf[((v - 3) >> 1) - (I.S - 1) * I.n];
    const int nu = (u - 2) >> 1, nv = (v - 2) >> 1;
    const bool uout = (u - 2) & 1;
    if (nu == nv) return uout ? I.nf[nu] : I.cap[nu] - I.nf[nu];
    if (uout) return kResInf;
    return I.af[nv * I.ld + nu % I.n];
}

// Push delta along the residual arc u -> v.
__device__ void push(Inst &I, int u, int v, int32_t delta)
{
    if (u == 0) I.sf[(v - 2) >> 1] += delta;
    else if (v == 0) I.sf[(u - 2) >> 1] -= delta;
    else if (v == 1) I.tf[((u - 3) >> 1) - (I.S - 1) * I.n] += delta;
    else if (u == 1) I.tf[((v - 3) >> 1) - (I.S - 1) * I.n] -= delta;
    else {
        const int nu = (u - 2) >> 1, nv = (v - 2) >> 1;
        const bool uout = (u - 2) & 1;
        if (nu == nv) I.nf[nu] += uout ? -delta : delta;
        else if (uout) I.af[nu * I.ld + nv % I.n] += delta;
        else I.af[nv * I.ld + nu % I.n] -= delta;
    }
}

// Best label of v over its incoming residual arcs; bp = the tail of the arc
// that improves on d[v], or -1 if none does.
__device__ void pull(const Inst &I, int v, int32_t &best, int &bp)
{
    const int S = I.S, n = I.n;
    const int32_t *d = I.d;
    best = d[v];
    bp = -1;
    auto take = [&](int u, int32_t c) {
        const int32_t du = d[u];
        if (du < kInf && du + c < best) {
            best = du + c;
            bp = u;
        }
    };
    if (v == 0) {
        for (int i = 0; i < n; ++i)
            if (I.sf[i] > 0) take(vin(i), -I.src[i]);
    } else if (v == 1) {
        for (int i = 0; i < n; ++i) take(vout((S - 1) * n + i), I.snk[i]);
    } else {
        const int nd = (v - 2) >> 1, k = stage_of(I, nd), i = nd - k * n;
        if (((v - 2) & 1) == 0) {
            if (k == 0) {
                take(0, I.src[i]);
            } else {
                const int32_t *col = I.ac + (k - 1) * n * I.ld + i;
                for (int j = 0; j < n; ++j) {
                    const int32_t a = col[j * I.ld];
                    if (a >= 0) take(vout((k - 1) * n + j), a);
                }
            }
            if (I.nf[nd] > 0) take(vout(nd), -I.nc[nd]);
        } else {
            if (I.nf[nd] < I.cap[nd]) take(vin(nd), I.nc[nd]);
            if (k < S - 1) {
                const int row = nd * I.ld;
                for (int j = 0; j < n; ++j)
                    if (I.af[row + j] > 0) take(vin((k + 1) * n + j), -I.ac[row + j]);
            } else if (I.tf[i] > 0) {
                take(1, -I.snk[i]);
            }
        }
    }
}

// Removes up to `want` units along one source-to-sink path of the current
// flow through node i0 of stage k0 and node i1 of stage k1 (k1 == k0, or
// k1 == k0 + 1 with flow on the link i0 -> i1).  Extends greedily over the
// lowest-index arc that carries flow; conservation guarantees one.  Returns
// the units removed (0 only if the flow is not conserved).  Thread 0 only.
__device__ int32_t strip_path(Inst &I, int k0, int i0, int k1, int i1, int32_t want)
{
    const int S = I.S, n = I.n;
    int32_t *P = I.anc;
    P[k0] = i0;
    P[k1] = i1;
    for (int k = k0; k > 0; --k) {
        int j = 0;
        while (j < n && I.af[((k - 1) * n + j) * I.ld + P[k]] <= 0) ++j;
        if (j == n) return 0;
        P[k - 1] = j;
    }
    for (int k = k1; k < S - 1; ++k) {
        int j = 0;
        while (j < n && I.af[(k * n + P[k]) * I.ld + j] <= 0) ++j;
        if (j == n) return 0;
        P[k + 1] = j;
    }
    int32_t delta = min(want, min(I.sf[P[0]], I.tf[P[S - 1]]));
    for (int k = 0; k < S; ++k) delta = min(delta, I.nf[k * n + P[k]]);
    for (int k = 0; k + 1 < S; ++k) delta = min(delta, I.af[(k * n + P[k]) * I.ld + P[k + 1]]);
    if (delta <= 0) return 0;
    I.sf[P[0]] -= delta;
    I.tf[P[S - 1]] -= delta;
    for (int k = 0; k < S; ++k) I.nf[k * n + P[k]] -= delta;
    for (int k = 0; k + 1 < S; ++k) I.af[(k * n + P[k]) * I.ld + P[k + 1]] -= delta;
    return delta;
}

struct Shared {
    int32_t flag[3];
    int32_t found, bad, strip_bad, err, mx;
    int32_t F;
    unsigned long long cost;
};

// Pointer doubling over the predecessor graph: true (uniformly) if it holds a
// cycle, with sh.found a vertex on one.
__device__ bool find_cycle(Inst &I, Shared &sh, int L)
{
    const int tid = threadIdx.x, nt = blockDim.x, V = I.V;
    for (int v = tid; v < V; v += nt) I.anc[v] = I.pred[v] < 0 ? v : I.pred[v];
    if (tid == 0) sh.found = V;
    __syncthreads();
    int32_t *a = I.anc, *a2 = I.anc2;
    for (int r = 0; r < L; ++r) {
        for (int v = tid; v < V; v += nt) a2[v] = a[a[v]];
        __syncthreads();
        int32_t *t = a;
        a = a2;
        a2 = t;
    }
    int low = V; // lowest vertex on a cycle among this thread's ancestors
    for (int v = tid; v < V; v += nt) {
        const int x = a[v];
        if (I.pred[x] >= 0) low = min(low, x);
    }
    for (int off = 32; off > 0; off >>= 1) low = min(low, __shfl_xor(low, off, 64));
    if (low < V && (tid & 63) == 0) atomicMin(&sh.found, low);
    __syncthreads();
    return sh.found < V;
}

// Label correction to a fixed point.  from_source: shortest distances from
// s (no negative cycle may exist); otherwise every label starts at 0 (a
// virtual root joined to all vertices) and the pass stops at the first
// predecessor cycle.  Returns 0 converged, 1 cycle found, 2 once `rounds`
// has grown by the round cap since `phase_start`.
__device__ int correct_labels(Inst &I, Shared &sh, bool from_source, int32_t bound, int L, int64_t &rounds,
                              int64_t phase_start)
{
    const int tid = threadIdx.x, nt = blockDim.x, V = I.V, Sn = I.S * I.n;
    for (int v = tid; v < V; v += nt) {
        I.d[v] = (!from_source || v == 0) ? 0 : kInf;
        I.pred[v] = -1;
    }
    if (tid == 0) sh.flag[0] = sh.flag[1] = sh.flag[2] = 0;
    __syncthreads();
    for (int it = 0;; ++it) {
        if (tid == 0) sh.flag[(it + 1) % 3] = 0;
        int f = 0;
        // all entry vertices first, then all exits, then s and t, so that a
        // wave pulls one kind of vertex at a time
        for (int q = tid; q < V; q += nt) {
            const int v = q < Sn ? 2 + 2 * q : (q < 2 * Sn ? 3 + 2 * (q - Sn) : q - 2 * Sn);
            int32_t best;
            int bp;
            pull(I, v, best, bp);
            if (bp >= 0) {
                I.d[v] = best;
                I.pred[v] = bp;
                f |= best < -bound ? 3 : 1;
            }
        }
        // one flag update per wave (the lanes' flags are ORed by ballot first)
        const int wf = (__ballot(f & 1) ? 1 : 0) | (__ballot(f & 2) ? 2 : 0);
        if (wf && (threadIdx.x & 63) == 0) atomicOr(&sh.flag[it % 3], wf);
        __syncthreads();
        const int fl = sh.flag[it % 3];
        ++rounds;
        if (!(fl & 1)) return 0;
        if (rounds - phase_start >= kChurnRoundCap) return 2;
        if (!from_source && ((fl & 2) || (it & 3) == 3) && find_cycle(I, sh, L)) return 1;
    }
}

__global__ void __launch_bounds__(kChurnThreads) churn_kernel(ChurnParams p)
{
    extern __shared__ int32_t lds[];
    __shared__ Shared sh;
    const int S = p.S, n = p.n, Sn = S * n, V = 2 * Sn + 2, links = (S - 1) * n * n;
    const int ld = n + 1, plinks = (S - 1) * n * ld; // padded rows in LDS
    const int tid = threadIdx.x, nt = blockDim.x;
    const int64_t b = blockIdx.x, s0 = p.start_per_instance ? b : 0;

    Inst I;
    I.S = S;
    I.n = n;
    I.V = V;
    I.ld = ld;
    I.inv_n = 1.0f / float(n);
    int32_t *q = lds;
    I.ac = q; q += plinks;
    I.af = q; q += plinks;
    I.cap = q; q += Sn;
    I.nc = q; q += Sn;
    I.nf = q; q += Sn;
    I.src = q; q += n;
    I.snk = q; q += n;
    I.sf = q; q += n;
    I.tf = q; q += n;
    I.d = q; q += V;
    I.pred = q; q += V;
    I.anc = q; q += V;
    I.anc2 = q;

    if (tid == 0) {
        sh.bad = 0;
        sh.strip_bad = 0;
        sh.err = 0;
        sh.mx = 0;
        sh.cost = 0;
    }
    __syncthreads();

    // Ingest the instance and its start flow, with the value checks of the
    // cold solve plus nonnegative start flows below 2^29.
    int bad = 0;
    int32_t mx = 0;
    for (int e = tid; e < links; e += nt) {
        const int32_t a = p.acost[b * links + e], f = p.af0[s0 * links + e];
        const int r = e / n, at = r * ld + (e - r * n);
        I.ac[at] = a;
        I.af[at] = f;
        bad |= (a < -1) | (f < 0) | (f >= kFlowMax);
        mx = max(mx, a);
    }
    for (int r = tid; r < (S - 1) * n; r += nt) {
        I.ac[r * ld + n] = -1; // the padding column: no link, no flow
        I.af[r * ld + n] = 0;
    }
    for (int e = tid; e < Sn; e += nt) {
        const int32_t c = p.cap[b * Sn + e], w = p.ncost[b * Sn + e], f = p.nf0[s0 * Sn + e];
        I.cap[e] = c;
        I.nc[e] = w;
        I.nf[e] = f;
        bad |= (c < 0) | (w < 0) | (f < 0) | (f >= kFlowMax);
        mx = max(mx, w);
    }
    for (int i = tid; i < n; i += nt) {
        const int32_t a = p.src ? p.src[b * n + i] : 0, z = p.snk ? p.snk[b * n + i] : 0;
        const int32_t f = p.sf0[s0 * n + i], g = p.tf0[s0 * n + i];
        I.src[i] = a;
        I.snk[i] = z;
        I.sf[i] = f;
        I.tf[i] = g;
        bad |= (a < 0) | (z < 0) | (f < 0) | (f >= kFlowMax) | (g < 0) | (g >= kFlowMax);
        mx = max(mx, max(a, z));
    }
    if (bad) atomicOr(&sh.bad, 1);
    atomicMax(&sh.mx, mx);
    __syncthreads();
    // Conservation of the start flow at every node.
    bad = 0;
    for (int nd = tid; nd < Sn; nd += nt) {
        const int k = nd / n, i = nd - k * n;
        int64_t in = 0, out = 0;
        if (k == 0) in = I.sf[i];
        else for (int j = 0; j < n; ++j) in += I.af[((k - 1) * n + j) * ld + i];
        if (k == S - 1) out = I.tf[i];
        else for (int j = 0; j < n; ++j) out += I.af[nd * ld + j];
        bad |= (in != I.nf[nd]) | (out != I.nf[nd]);
    }
    if (bad) atomicOr(&sh.bad, 1);
    __syncthreads();

    const int32_t supply = p.supply[b];
    int status = GWTF_INST_OK;
    if (sh.bad || supply < 0) status = GWTF_INST_BAD_INPUT;
    else if (int64_t(2 * Sn + 3) * sh.mx >= kLabelBound) status = GWTF_INST_OVERFLOW;

    int64_t removed = 0, cycles = 0, augs = 0, rounds = 0;
    if (status == GWTF_INST_OK) {
        // 1. strip
        if (tid == 0) {
            int64_t F = 0;
            for (int i = 0; i < n; ++i) F += I.sf[i];
            bool ok = F < kFlowMax;
            for (int nd = 0; ok && nd < Sn; ++nd) {
                const int k = nd / n, i = nd - k * n;
                while (ok && I.nf[nd] > I.cap[nd]) {
                    const int32_t r = strip_path(I, k, i, k, i, I.nf[nd] - I.cap[nd]);
                    ok = r > 0;
                    F -= r;
                    ++removed;
                }
            }
            for (int e = 0; ok && e < links; ++e) {
                const int k = e / (n * n), i = (e / n) % n, j = e % n, at = (k * n + i) * ld + j;
                while (ok && I.ac[at] < 0 && I.af[at] > 0) {
                    const int32_t r = strip_path(I, k, i, k + 1, j, I.af[at]);
                    ok = r > 0;
                    F -= r;
                    ++removed;
                }
            }
            while (ok && F > supply) {
                int i = 0;
                while (i < n && I.sf[i] <= 0) ++i;
                const int32_t r = i < n ? strip_path(I, 0, i, 0, i, int32_t(min<int64_t>(F - supply, kFlowMax))) : 0;
                ok = r > 0;
                F -= r;
                ++removed;
            }
            sh.F = int32_t(F);
            sh.strip_bad = ok ? 0 : 1;
        }
        __syncthreads();
        if (sh.strip_bad) status = GWTF_INST_BAD_INPUT;
    }

    const int32_t bound = int32_t((V - 1) * int64_t(sh.mx));
    const int L = 32 - __clz(V);
    // 2. cancel.  Should it stop at its round cap or meet a cycle it cannot
    // push (neither happens on valid input), the instance restarts from the
    // zero flow: step 3 alone is then the cold solve and reaches its result.
    bool restart = false;
    while (status == GWTF_INST_OK) {
        const int r = correct_labels(I, sh, false, bound, L, rounds, 0);
        if (r == 0) break;
        if (r == 2) {
            restart = true;
            break;
        }
        if (tid == 0) {
            const int c = sh.found;
            int32_t delta = kResInf;
            int x = c, steps = 0;
            do {
                const int u = I.pred[x];
                if (u < 0) break;
                delta = min(delta, residual(I, u, x));
                x = u;
            } while (x != c && ++steps <= V);
            if (x != c || delta <= 0 || delta == kResInf) {
                sh.err = 1;
            } else {
                do {
                    const int u = I.pred[x];
                    push(I, u, x, delta);
                    x = u;
                } while (x != c);
            }
        }
        __syncthreads();
        ++cycles;
        if (sh.err) {
            restart = true;
            break;
        }
    }
    if (restart) {
        for (int e = tid; e < plinks; e += nt) I.af[e] = 0;
        for (int e = tid; e < Sn; e += nt) I.nf[e] = 0;
        for (int i = tid; i < n; i += nt) I.sf[i] = I.tf[i] = 0;
        __syncthreads();
        if (tid == 0) {
            sh.F = 0;
            sh.err = 0;
        }
        __syncthreads();
    }
    const int64_t augment_start = rounds;
    // 3. augment
    while (status == GWTF_INST_OK && sh.F < supply) {
        if (correct_labels(I, sh, true, bound, L, rounds, augment_start) == 2) {
            status = GWTF_INST_NOT_CONVERGED;
            break;
        }
        if (I.d[1] >= kInf) break;
        if (tid == 0) {
            int32_t delta = supply - sh.F;
            int x = 1, steps = 0;
            while (x != 0 && steps++ <= V) {
                const int u = I.pred[x];
                if (u < 0) break;
                delta = min(delta, residual(I, u, x));
                x = u;
            }
            if (x != 0 || delta <= 0) {
                sh.err = 1;
            } else {
                for (x = 1; x != 0;) {
                    const int u = I.pred[x];
                    push(I, u, x, delta);
                    x = u;
                }
                sh.F += delta;
            }
        }
        __syncthreads();
        ++augs;
        if (sh.err) status = GWTF_INST_NOT_CONVERGED;
    }

    // Export: F, cost = sum of cost * flow over every arc (int64), flows.
    const bool ok = status == GWTF_INST_OK;
    int64_t part = 0;
    if (ok) {
        for (int e = tid; e < plinks; e += nt)
            if (I.af[e] > 0) part += int64_t(I.ac[e]) * I.af[e];
        for (int e = tid; e < Sn; e += nt) part += int64_t(I.nc[e]) * I.nf[e];
        for (int i = tid; i < n; i += nt) part += int64_t(I.src[i]) * I.sf[i] + int64_t(I.snk[i]) * I.tf[i];
        atomicAdd(&sh.cost, (unsigned long long)part);
    }
    __syncthreads();
    if (tid == 0) {
        p.F_out[b] = ok ? sh.F : 0;
        p.cost_out[b] = ok ? int64_t(sh.cost) : 0;
        p.status_out[b] = status;
        if (p.work) {
            p.work[4 * b + 0] = removed;
            p.work[4 * b + 1] = cycles;
            p.work[4 * b + 2] = augs;
            p.work[4 * b + 3] = rounds;
        }
    }
    if (p.nf_out) {
        for (int e = tid; e < links; e += nt) {
            const int r = e / n;
            p.af_out[b * links + e] = ok ? I.af[r * ld + (e - r * n)] : 0;
        }
        for (int e = tid; e < Sn; e += nt) p.nf_out[b * Sn + e] = ok ? I.nf[e] : 0;
        for (int i = tid; i < n; i += nt) {
            p.sf_out[b * n + i] = ok ? I.sf[i] : 0;
            p.tf_out[b * n + i] = ok ? I.tf[i] : 0;
        }
    }
}

} // namespace

size_t churn_lds_bytes(int S, int n)
{
    const size_t Sn = size_t(S) * n, V = 2 * Sn + 2;
    return sizeof(int32_t) * (2 * size_t(S - 1) * n * (n + 1) + 3 * Sn + 4 * size_t(n) + 4 * V);
}

hipError_t launch_churn_resolve(const ChurnParams &p, hipStream_t stream)
{
    // A single wave for small instances: its barriers cost next to nothing
    // and more instances share a CU.
    const int V = 2 * p.S * p.n + 2;
    const int threads = V <= 192 ? 64 : kChurnThreads;
    hipLaunchKernelGGL(churn_kernel, dim3(p.B), dim3(threads), churn_lds_bytes(p.S, p.n), stream, p);
    return hipGetLastError();
}

} // namespace gwtf
