// Internal interface of the packed small-instance pass (mcf_solver_small.hip):
// one to eight instances per wave, for at most 8 stages of at most 16 nodes.
// Not part of the public C ABI.
#pragma once

#include "mcf_internal.h"

namespace gwtf {

constexpr int kSmallMaxStages = 8;
bool small_pass_fits(int S, int n);
hipError_t launch_small_pass(const SolveParams &p, hipStream_t s);

} // namespace gwtf
