// Internal interface of the stage-pipelined register pass
// (mcf_solver_pipe.hip): one workgroup of 8 waves per instance, S <= 32,
// n <= 64, link costs below 65535.  Not part of the public C ABI.
#pragma once

#include "mcf_internal.h"

namespace gwtf {

constexpr int kPipeMaxStages = 32;

// Dynamic LDS of one workgroup: mailboxes per wave, node arrays [S][64]
// (one row per stage), the path buffer and the flow lists.
struct PipeLayout {
    size_t exmb, enmb, nf, capl, ncl, chain, loff, llen, path, lamt, lent;
    size_t total;
};

__host__ __device__ inline PipeLayout pipe_layout(int S, int waves, int64_t slots)
{
    PipeLayout L;
    const size_t rows = size_t(S) * 64, lslots = size_t(slots) + 64;
    size_t o = 0;
    auto take = [&](size_t bytes) { size_t at = o; o = align16(o + bytes); return at; };
    L.exmb = take(4 * size_t(waves) * 64);
    L.enmb = take(4 * size_t(waves) * 64);
    L.nf = take(4 * rows);
    L.capl = take(4 * rows);
    L.ncl = take(4 * rows);
    L.chain = take(4 * 2 * rows); // per vertex: predecessor vertex | arc code << 13
    L.loff = take(2 * rows);
    L.llen = take(rows);
    L.path = take(4 * (2 * rows + 8));
    L.lamt = take(4 * lslots);
    L.lent = take(4 * lslots); // partner | cost << 8
    L.total = o;
    return L;
}

bool pipe_pass_fits(int S, int n);
int64_t pipe_pass_slots(int S, size_t lds_max); // flow-list slots that fit beside the rest
hipError_t launch_pipe_pass(const SolveParams &p, hipStream_t s);

} // namespace gwtf
