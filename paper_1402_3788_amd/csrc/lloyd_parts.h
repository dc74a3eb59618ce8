// The kernel files are compiled once per part of the feature-count range
// [1, kMaxM] (-DLLOYD_PART=p); each part defines launch_*_part_<p>, and part 0
// also defines the dispatchers, which pick the part from M.
#pragma once

#include "lloyd.h"

#ifndef LLOYD_PART
#define LLOYD_PART 0
#endif
#define LLOYD_PARTS 4
#define LLOYD_CAT2(a, b) a##_##b
#define LLOYD_CAT(a, b) LLOYD_CAT2(a, b)
#define LLOYD_PART_FN(name) LLOYD_CAT(name, LLOYD_PART)
#define LLOYD_PART_CASES LLOYD_CASE(0) LLOYD_CASE(1) LLOYD_CASE(2) LLOYD_CASE(3)

static_assert(lloyd::kMaxM % LLOYD_PARTS == 0, "parts split the feature counts evenly");

namespace lloyd {
hipError_t launch_tile_part_0(const StepArgs &, Mode, const AccumPlan &, hipStream_t);
hipError_t launch_tile_part_1(const StepArgs &, Mode, const AccumPlan &, hipStream_t);
hipError_t launch_tile_part_2(const StepArgs &, Mode, const AccumPlan &, hipStream_t);
hipError_t launch_tile_part_3(const StepArgs &, Mode, const AccumPlan &, hipStream_t);
hipError_t launch_lane_part_0(const StepArgs &, Mode, const AccumPlan &, hipStream_t);
hipError_t launch_lane_part_1(const StepArgs &, Mode, const AccumPlan &, hipStream_t);
hipError_t launch_lane_part_2(const StepArgs &, Mode, const AccumPlan &, hipStream_t);
hipError_t launch_lane_part_3(const StepArgs &, Mode, const AccumPlan &, hipStream_t);
hipError_t launch_lane_l1_part_0(const StepArgs &, const AccumPlan &, hipStream_t);
hipError_t launch_lane_l1_part_1(const StepArgs &, const AccumPlan &, hipStream_t);
hipError_t launch_lane_l1_part_2(const StepArgs &, const AccumPlan &, hipStream_t);
hipError_t launch_lane_l1_part_3(const StepArgs &, const AccumPlan &, hipStream_t);
hipError_t launch_lane_mfma_part_0(const StepArgs &, Mode, const AccumPlan &, hipStream_t);
hipError_t launch_lane_mfma_part_1(const StepArgs &, Mode, const AccumPlan &, hipStream_t);
hipError_t launch_lane_mfma_part_2(const StepArgs &, Mode, const AccumPlan &, hipStream_t);
hipError_t launch_lane_mfma_part_3(const StepArgs &, Mode, const AccumPlan &, hipStream_t);
}  // namespace lloyd
