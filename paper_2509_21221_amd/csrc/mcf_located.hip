// Location-factored instances (the paper's Sec. VI testbed places nodes at a
// few geographic locations; Eq. 1's link term is the latency between the two
// nodes' locations): expansion of the implied link delays into the ordinary
// dense layout, for the passes that read dense link costs.
//
// One workgroup writes one row of one stage pair, (b, k, i) -> the n delays
// from node i of stage k to every node of stage k+1: consecutive lanes write
// consecutive columns.  A location outside [0, L) or a negative latency
// turns the affected delays into -2, which the solver reports as
// GWTF_INST_BAD_INPUT; a negative latency that no link uses poisons the
// instance's first delay the same way.
#include "mcf_internal.h"

namespace gwtf {

namespace {

__global__ void located_expand_kernel(int32_t S, int32_t n, int32_t L, const int32_t *loc, const int32_t *lat,
                                      int32_t *arc)
{
    const int64_t row = blockIdx.x; // b * (S-1) * n + k * n + i
    const int64_t per_b = int64_t(S - 1) * n;
    const int64_t b = row / per_b;
    const int k = int((row - b * per_b) / n), i = int(row - b * per_b - int64_t(k) * n);
    const int32_t *lb = loc + b * int64_t(S) * n;
    const int32_t *tb = lat + b * int64_t(L) * L;
    int32_t *out = arc + row * n;
    const int a = lb[k * n + i];
    const bool aok = a >= 0 && a < L;
    for (int j = threadIdx.x; j < n; j += blockDim.x) {
        const int c = lb[(k + 1) * n + j];
        int32_t v = -2;
        if (aok && c >= 0 && c < L) {
            v = tb[a * L + c];
            if (v < 0) v = -2;
        }
        out[j] = v;
    }
    if (k == 0 && i == 0) {
        __shared__ int neg;
        if (threadIdx.x == 0) neg = 0;
        __syncthreads();
        for (int e = threadIdx.x; e < L * L; e += blockDim.x)
            if (tb[e] < 0) neg = 1;
        __syncthreads();
        if (threadIdx.x == 0 && neg) out[0] = -2;
    }
}

} // namespace

hipError_t launch_located_expand(int32_t B, int32_t S, int32_t n, int32_t L, const int32_t *loc,
                                 const int32_t *lat, int32_t *arc, hipStream_t s)
{
    if (S < 2) return hipSuccess;
    const int64_t rows = int64_t(B) * (S - 1) * n;
    const int threads = n >= 256 ? 256 : ((n + 63) / 64) * 64;
    hipLaunchKernelGGL(located_expand_kernel, dim3(unsigned(rows)), dim3(threads), 0, s, S, n, L, loc, lat, arc);
    return hipGetLastError();
}

} // namespace gwtf
