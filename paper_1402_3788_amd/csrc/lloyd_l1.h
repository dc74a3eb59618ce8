// Assignment by the L1 distance (lloyd_l1.hip).
#pragma once

#include "lloyd.h"

namespace lloyd {

struct L1Plan {
    int waves;          // wavefronts per workgroup (0: the centres do not fit in LDS)
    int groups;         // persistent workgroups
    size_t lds_bytes;   // padded centres, then one tile slot per wave
};

L1Plan plan_l1(int64_t n, int M, int K);
// Labels (and optional distances) of a.X against a.C; early exit through
// a.ctl / a.t / a.fixed as the other assigning launches.
hipError_t launch_l1(const StepArgs &a, const L1Plan &plan, hipStream_t s);

}  // namespace lloyd
