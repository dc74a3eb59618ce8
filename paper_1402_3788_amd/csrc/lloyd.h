// Internal declarations shared by the kernel files and the C-ABI layer.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace lloyd {

constexpr int kWave = 64;            // CDNA wavefront width
constexpr int kMaxM = 64;            // features supported
constexpr int kMaxK = 1024;          // clusters supported
constexpr int kMaxKM = 16384;        // K * M supported
constexpr int kMaxLds = 160 * 1024;  // LDS bytes per workgroup on gfx950
constexpr int kCUs = 256;            // compute units the launch geometry is sized for

// Iteration control block, kept at the start of the caller's workspace.
//   changed[t & 1] : set by the centres launch of iteration t (each of its
//                    workgroups ORs in 1 when one of its centre coordinates
//                    differs bitwise from t-1's; the centres launch of t-1
//                    cleared it).
//   converged_at   : first t >= 2 whose centres were congruent with t-1's
//                    (0 = not yet); written by the launches of iteration t+1.
//   fallbacks      : objects whose label was re-decided in fp64 (diagnostic).
//   reruns         : wave tiles whose split-precision scores left a call too
//                    close, recomputed with fp32 products (diagnostic).
//   ring_stalls    : waves of the tile kernel's ring form whose wait for their
//                    turn gave up (never expected; the sums are then unordered
//                    and kmeans_run fails with KMEANS_EHIP).
struct Ctl {
    int32_t changed[2];
    int32_t converged_at;
    int32_t fallbacks;
    int32_t reruns;
    int32_t ring_stalls;
    int32_t pad[58];
};
static_assert(sizeof(Ctl) == 256, "control block is one 256-byte slot");

// Early exit of a launch that belongs to an iteration after convergence; the
// first such launch records the iteration count.
__device__ inline bool stop_before(Ctl *ctl, int t, int fixed)
{
    if (ctl == nullptr || fixed) return false;
    const bool stop =
        ctl->converged_at != 0 || ((t - 1 >= 2) && ctl->changed[(t - 1) & 1] == 0);
    if (stop && blockIdx.x == 0 && threadIdx.x == 0 && ctl->converged_at == 0)
        ctl->converged_at = t - 1;
    return stop;
}

// Early exit of a launch that accumulates from the labels another launch of
// the same iteration assigned (the L1 metric's second launch): once the run
// has converged, the assigning launch before it on the stream has evaluated
// the stop rule and recorded the iteration, so the value is settled here.
__device__ inline bool stop_after_assign(const Ctl *ctl, int fixed)
{
    return ctl != nullptr && !fixed && ctl->converged_at != 0;
}

// What a launch of the distance kernels does with the assignment.
enum Mode : int {
    kAssign = 0,        // labels (and optional min_d2) only
    kAssignAccum = 1,   // labels + per-workgroup partial sums/counts (fused)
    kAccumLabels = 2,   // partial sums/counts from caller-provided labels
};

// Distance paths: one object per lane with the direct form on the vector ALU
// (lloyd_lane.hip), one object per lane with the scores on the bf16 matrix
// cores (lloyd_lane_mfma.hip, K <= 16), or 64-object tiles on the matrix cores
// with a cross-lane argmin (lloyd_tile.hip, any K).
enum Path : int { kPathValu = 0, kPathTile = 1, kPathLaneMfma = 2 };

// Static LDS of a kernel (bytes), from the runtime's attributes; SIZE_MAX when
// they cannot be read. Launches check static + dynamic LDS against kMaxLds, so
// a plan that would not fit is refused on the host instead of dispatched.
inline size_t static_lds_bytes(const void *kernel)
{
    hipFuncAttributes attr{};
    if (hipFuncGetAttributes(&attr, kernel) != hipSuccess) return SIZE_MAX;
    return attr.sharedSizeBytes;
}

struct AccumPlan {
    Path path;
    int waves;          // wavefronts per workgroup
    int groups;         // workgroups (persistent, strided over 64-object tiles)
    int accum;          // accumulation form (kernel-specific code)
    size_t lds_bytes;   // dynamic LDS per workgroup
};

// Launch geometry for a problem shape (pure host code).
AccumPlan plan_lane(int64_t n, int M, int K, Mode mode);
AccumPlan plan_lane_mfma(int64_t n, int M, int K, Mode mode);
AccumPlan plan_tile(int64_t n, int M, int K, Mode mode);
// Whether the tile kernel's per-workgroup state (centre operands and fp64
// slab) fits in one workgroup's LDS for this shape.
bool tile_fits(int M, int K);
// Whether the one-object-per-lane matrix-core form supports this shape (its
// centre operands live in registers: K <= 16, M <= 32).
bool lane_mfma_fits(int M, int K);

struct StepArgs {
    const float *X;
    int64_t n;
    int M;
    const float *C;            // centres read by the assignment (previous centres)
    int K;
    int32_t *labels;           // out (modes 0/1)
    const int32_t *labels_in;  // in (mode 2)
    float *min_d2;             // optional out (mode 0)
    double *part_sums;         // [groups][K][M] (modes 1/2)
    int32_t *part_counts;      // [K][groups]
    float *centers_out;        // new centres (may alias C)
    int32_t *counts_out;       // [K]
    Ctl *ctl;                  // control block (modes 1/2)
    int t;                     // iteration number (1-based)
    int fixed;                 // no early stop
    int compare;               // record the change flag of iteration t
    int force64;               // decide every label with fp64 distances
    hipEvent_t ev_start;       // optional: stamped when the assigning launch's
    hipEvent_t ev_stop;        //   dispatch starts and ends (null: not timed)
};

hipError_t launch_lane(const StepArgs &a, Mode mode, const AccumPlan &plan, hipStream_t s);
hipError_t launch_lane_mfma(const StepArgs &a, Mode mode, const AccumPlan &plan, hipStream_t s);
hipError_t launch_tile(const StepArgs &a, Mode mode, const AccumPlan &plan, hipStream_t s);

hipError_t launch_ctl_reset(Ctl *ctl, hipStream_t s);

// Centres of gravity and change flag of iteration a.t from the partials of an
// accumulating launch with `groups` workgroups (lloyd_centres.hip).
hipError_t launch_centres(const StepArgs &a, int groups, hipStream_t s);

}  // namespace lloyd
