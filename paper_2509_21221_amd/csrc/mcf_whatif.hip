// What-if node addition (paper Sec. VI, handling joining nodes): build the
// batch of instances that tries every assignment of the candidate nodes to
// stages, and reduce solved batches to the best assignment.
//
// Expansion is a pure copy with per-element selection: one workgroup per
// placement decodes the placement index into a stage -> candidate table in
// LDS, then its threads write the instance with consecutive lanes on
// consecutive elements (coalesced stores).  The base instance and the
// candidate arrays are small and shared by every workgroup, so they are
// served from L2; the kernel's HBM traffic is the instances it writes.
#include "mcf_internal.h"

namespace gwtf {

namespace {

constexpr int kExpandThreads = 256;
constexpr int kBestThreads = 1024;

__global__ void __launch_bounds__(kExpandThreads) whatif_expand_kernel(WhatifExpandParams p)
{
    __shared__ int32_t at_stage[kWhatifMaxStages];
    __shared__ uint64_t used[kWhatifMaxStages / 64];
    const int S = p.S, n = p.n, m = p.m, slot = p.slot;
    const int64_t r = p.first + blockIdx.x;

    for (int k = threadIdx.x; k < S; k += blockDim.x) at_stage[k] = -1;
    for (int w = threadIdx.x; w < kWhatifMaxStages / 64; w += blockDim.x) used[w] = 0;
    __syncthreads();
    if (threadIdx.x == 0) {
        // Mixed-radix digits of r: candidate c picks among the S - c stages
        // still free, and each choice is followed by P(S-c-1, m-c-1)
        // completions (the radix, built from the last candidate back).
        int64_t radix = 1;
        for (int c = m - 1; c > 0; --c) radix *= int64_t(S - c);
        int64_t rem = r;
        for (int c = 0; c < m; ++c) {
            int64_t d = rem / radix;
            rem -= d * radix;
            if (c + 1 < m) radix /= int64_t(S - c - 1);
            // stage = the d-th free stage (0-based) in increasing order; the
            // host guarantees r < S!/(S-m)!, so d < S - c free stages remain
            // and the search ends inside the last word at the latest.
            const int words = (S + 63) / 64;
            int w = 0;
            for (; w < words - 1; ++w) {
                const int64_t free_here = __popcll(~used[w]);
                if (d < free_here) break;
                d -= free_here;
            }
            uint64_t freebits = ~used[w];
            for (int64_t skip = 0; skip < d; ++skip) freebits &= freebits - 1;
            const int bit = __ffsll((unsigned long long)freebits) - 1;
            used[w] |= uint64_t(1) << bit;
            at_stage[64 * w + bit] = c;
        }
    }
    __syncthreads();

    // Sizes of one instance; the host keeps (S-1) n^2 below 2^31, so 32-bit
    // index arithmetic is exact.
    const uint32_t un = uint32_t(n), SN = uint32_t(S) * un, nn = un * un, na = uint32_t(S - 1) * nn;
    const size_t o = size_t(blockIdx.x);
    int32_t *cap = p.out_cap + o * size_t(SN), *ncost = p.out_cost + o * size_t(SN);
    for (uint32_t e = threadIdx.x; e < SN; e += blockDim.x) {
        const int k = int(e / un), i = int(e - uint32_t(k) * un);
        const int c = at_stage[k];
        const bool cand = (i == slot) && c >= 0;
        cap[e] = cand ? p.ccap[size_t(c) * S + k] : p.cap[e];
        ncost[e] = cand ? p.ccost[size_t(c) * S + k] : p.cost[e];
    }
    if (S > 1) {
        int32_t *arc = p.out_arc + o * size_t(na);
        for (uint32_t e = threadIdx.x; e < na; e += blockDim.x) {
            const int k = int(e / nn);
            const uint32_t q = e - uint32_t(k) * nn;
            const int i = int(q / un), j = int(q - uint32_t(i) * un);
            const int ci = (i == slot) ? at_stage[k] : -1;      // candidate sending
            const int cj = (j == slot) ? at_stage[k + 1] : -1;  // candidate receiving
            int32_t v;
            if (ci >= 0 && cj >= 0) v = p.clink[size_t(ci) * m + cj];
            else if (ci >= 0) v = p.cout[(size_t(ci) * S + k) * n + j];
            else if (cj >= 0) v = p.cin[(size_t(cj) * S + k + 1) * n + i];
            else v = p.arc[e];
            arc[e] = v;
        }
    }
    int32_t *src = p.out_src + o * n, *snk = p.out_snk + o * n;
    for (int i = threadIdx.x; i < n; i += blockDim.x) {
        const int c0 = (i == slot) ? at_stage[0] : -1, cl = (i == slot) ? at_stage[S - 1] : -1;
        src[i] = c0 >= 0 ? (p.csrc ? p.csrc[c0] : 0) : (p.src ? p.src[i] : 0);
        snk[i] = cl >= 0 ? (p.csnk ? p.csnk[cl] : 0) : (p.snk ? p.snk[i] : 0);
    }
    if (threadIdx.x == 0) p.out_supply[o] = p.supply[0];
}

// Candidate key: valid, larger F, smaller cost, smaller index wins.
struct Key {
    int64_t idx, F, cost; // idx < 0: no candidate
};

__device__ inline bool better(const Key &a, const Key &b)
{
    if (a.idx < 0) return false;
    if (b.idx < 0) return true;
    if (a.F != b.F) return a.F > b.F;
    if (a.cost != b.cost) return a.cost < b.cost;
    return a.idx < b.idx;
}

__global__ void __launch_bounds__(kBestThreads) whatif_best_kernel(int32_t count, const int64_t *F,
                                                                   const int64_t *cost, const int32_t *status,
                                                                   int64_t first, int32_t merge, int64_t *best)
{
    __shared__ Key part[kBestThreads / 64];
    Key k{-1, 0, 0};
    for (int i = threadIdx.x; i < count; i += blockDim.x) {
        if (status[i] != 0) continue;
        const Key c{first + i, F[i], cost[i]};
        if (better(c, k)) k = c;
    }
    for (int off = 32; off > 0; off >>= 1) {
        Key o;
        o.idx = __shfl_xor(k.idx, off);
        o.F = __shfl_xor(k.F, off);
        o.cost = __shfl_xor(k.cost, off);
        if (better(o, k)) k = o;
    }
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (lane == 0) part[wave] = k;
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int w = 1; w < int(blockDim.x >> 6); ++w)
            if (better(part[w], k)) k = part[w];
        if (merge) {
            const Key prev{best[0], best[1], best[2]};
            if (better(prev, k)) k = prev;
        }
        if (k.idx < 0) k = Key{-1, 0, 0};
        best[0] = k.idx;
        best[1] = k.F;
        best[2] = k.cost;
    }
}

} // namespace

hipError_t launch_whatif_expand(const WhatifExpandParams &p, int32_t count, hipStream_t s)
{
    if (count == 0) return hipSuccess;
    hipLaunchKernelGGL(whatif_expand_kernel, dim3(count), dim3(kExpandThreads), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_whatif_best(int32_t count, const int64_t *F, const int64_t *cost, const int32_t *status,
                              int64_t first, int32_t merge, int64_t *best, hipStream_t s)
{
    hipLaunchKernelGGL(whatif_best_kernel, dim3(1), dim3(kBestThreads), 0, s, count, F, cost, status, first,
                       merge, best);
    return hipGetLastError();
}

} // namespace gwtf
