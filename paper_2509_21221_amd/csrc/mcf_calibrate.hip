// Hand-off latency calibration: the floor of the latency roofline that the
// stage-pipelined passes report.
//
// Both pipelined passes move labels from one stage's owner to the next one's
// and wait for them: the register pass between the waves of one workgroup
// through LDS mailboxes, the grid pass between workgroups on different CUs
// through device-scope atomic loads and stores.  One such hand-off, with no
// work around it, is the least a pipeline hop can cost.  These kernels
// measure it as half the round trip of a ping-pong repeated kHandoffRounds
// times:
//
//  * LDS: wave 0 and wave 1 of one workgroup, one word each way;
//  * device scope: two workgroups of one launch of 16 one-wave workgroups
//    (far fewer than the device's CUs, so all are placed at once; should one
//    not be, the other's bounded wait runs out), relaxed agent-scope atomics
//    as the grid pass uses, once for workgroups 0 and `neighbour` (a stage
//    and the next one in the grid pass, whose workgroup indices differ by
//    the stage's slices of 128 nodes: 4 at n = 512; workgroups are dealt
//    round robin to the 8 XCDs, so these sit on different XCDs) and once for
//    workgroups 0 and 8 (the same XCD).
//
// Every wait is bounded; a wait that runs out marks the result invalid
// instead of hanging.  Times come from the constant-rate wall clock.
#include "mcf_internal.h"

namespace gwtf {
namespace {

constexpr int kHandoffRounds = 2000;
constexpr int kHandoffSpin = 1 << 22;
constexpr int kDeviceBlocks = 16;

__global__ __launch_bounds__(128) void lds_handoff_kernel(long long *out)
{
    __shared__ int ping, pong;
    const int wave = threadIdx.x >> 6;
    if (threadIdx.x == 0) {
        ping = -1;
        pong = -1;
    }
    __syncthreads();
    int bad = 0;
    const long long t0 = wall_clock64();
    for (int i = 0; i < kHandoffRounds && !bad; ++i) {
        int *mine = wave == 0 ? &ping : &pong;
        int *theirs = wave == 0 ? &pong : &ping;
        if (wave == 0) __hip_atomic_store(mine, i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        int spins = 0;
        while (__hip_atomic_load(theirs, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) != i)
            if (++spins > kHandoffSpin) {
                bad = 1;
                break;
            }
        if (wave == 1) __hip_atomic_store(mine, i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    }
    const long long t1 = wall_clock64();
    if (threadIdx.x == 0) {
        out[0] = t1 - t0;
        out[1] = bad;
    }
}

// Blocks a and b ping-pong through flags[0] and flags[64] (separate cache
// lines); every other block returns at once.
__global__ __launch_bounds__(64) void device_handoff_kernel(int *flags, long long *out, int a, int b)
{
    const int g = blockIdx.x;
    if ((g != a && g != b) || threadIdx.x != 0) return;
    int *ping = flags, *pong = flags + 64;
    int bad = 0;
    const long long t0 = wall_clock64();
    for (int i = 1; i <= kHandoffRounds && !bad; ++i) {
        int *mine = g == a ? ping : pong;
        int *theirs = g == a ? pong : ping;
        if (g == a) __hip_atomic_store(mine, i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        int spins = 0;
        while (__hip_atomic_load(theirs, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != i)
            if (++spins > kHandoffSpin) {
                bad = 1;
                break;
            }
        if (g == b) __hip_atomic_store(mine, i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    const long long t1 = wall_clock64();
    if (g == a) {
        out[0] = t1 - t0;
        out[1] = bad;
    }
}

__global__ void clear_flags_kernel(int *flags, int count)
{
    for (int i = threadIdx.x; i < count; i += blockDim.x) flags[i] = 0;
}

} // namespace

hipError_t run_handoff_calibration(hipStream_t s, int clock_khz, int neighbour, double out_ns[3])
{
    int *flags = nullptr;
    long long *res = nullptr;
    hipError_t e = hipMalloc(&flags, 128 * sizeof(int));
    if (e != hipSuccess) return e;
    e = hipMalloc(&res, 6 * sizeof(long long));
    if (e != hipSuccess) {
        (void)hipFree(flags);
        return e;
    }
    long long host[6] = {0, 1, 0, 1, 0, 1};
    hipLaunchKernelGGL(lds_handoff_kernel, dim3(1), dim3(128), 0, s, res);
    e = hipGetLastError();
    const int pairs[2][2] = {{0, neighbour}, {0, 8}};
    for (int q = 0; q < 2 && e == hipSuccess; ++q) {
        hipLaunchKernelGGL(clear_flags_kernel, dim3(1), dim3(128), 0, s, flags, 128);
        e = hipGetLastError();
        if (e != hipSuccess) break;
        hipLaunchKernelGGL(device_handoff_kernel, dim3(kDeviceBlocks), dim3(64), 0, s, flags, res + 2 * (q + 1),
                           pairs[q][0], pairs[q][1]);
        e = hipGetLastError();
    }
    if (e == hipSuccess) e = hipMemcpyAsync(host, res, sizeof host, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    (void)hipFree(flags);
    (void)hipFree(res);
    if (e != hipSuccess) return e;
    const double ns_per_tick = 1e6 / double(clock_khz > 0 ? clock_khz : 100000);
    for (int q = 0; q < 3; ++q)
        out_ns[q] = host[2 * q + 1] ? -1.0 : double(host[2 * q]) * ns_per_tick / (2.0 * kHandoffRounds);
    return hipSuccess;
}

} // namespace gwtf
