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

// The L1 assignment fused with the accumulation of Eq. (1) in the direct-form
// lane kernel (lloyd_lane.hip), for shapes where its per-wave fp64 slabs leave
// enough waves per workgroup; waves = 0 in the plan when it is not used.
// The partials go where the other accumulating launches put theirs, for
// launch_centres with plan.groups.
AccumPlan plan_lane_l1(int64_t n, int M, int K);
hipError_t launch_lane_l1(const StepArgs &a, const AccumPlan &plan, hipStream_t s);

}  // namespace lloyd
