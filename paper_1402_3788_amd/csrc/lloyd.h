// Internal declarations shared by the kernel files and the C-ABI layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace lloyd {

constexpr int kWave = 64;          // CDNA wavefront width
constexpr int kMaxM = 64;          // features supported
constexpr int kMaxK = 1024;        // clusters supported
constexpr int kMaxKM = 16384;      // K * M supported
constexpr int kMaxLds = 160 * 1024;  // LDS bytes per workgroup on gfx950
constexpr int kMaxGroups = 1024;   // persistent workgroups of the accumulating launches

// Iteration control block, kept in the caller's workspace (device memory).
//   changed[t & 1]  : set (integer OR) by the finalise launch of iteration t when
//                     any centre coordinate differs bitwise from iteration t-1;
//                     cleared by iteration t's assign launch before that.
//   converged_at    : first t >= 2 whose centres were congruent with t-1's
//                     (0 = not yet); written by the finalise launch of t+1.
//   fallbacks       : objects whose label was re-decided in fp64 (diagnostic).
struct Ctl {
    int32_t changed[2];
    int32_t converged_at;
    int32_t fallbacks;
    int32_t pad[60];
};
static_assert(sizeof(Ctl) == 256, "control block is one 256-byte slot");

// What a launch of the distance kernels does with the assignment.
enum Mode : int {
    kAssign = 0,        // labels (and optional min_d2) only
    kAssignAccum = 1,   // labels + per-workgroup partial sums/counts (fused)
    kAccumLabels = 2,   // partial sums/counts from caller-provided labels
};

struct AccumPlan {
    int waves;          // wavefronts per workgroup
    int groups;         // workgroups (persistent, strided over 64-object tiles)
    size_t lds_bytes;   // dynamic LDS per workgroup
};

// Launch geometry of the vector-ALU kernel for a problem shape (pure host code).
AccumPlan plan_valu(int64_t n, int M, int K, Mode mode);

struct StepArgs {
    const float *X;
    int64_t n;
    int M;
    const float *C;          // centres read by the assignment
    int K;
    int32_t *labels;         // out (modes 0/1)
    const int32_t *labels_in;  // in (mode 2)
    float *min_d2;           // optional out (mode 0)
    double *part_sums;       // [groups][K][M] (modes 1/2)
    int32_t *part_counts;    // [groups][K]
    Ctl *ctl;                // iteration control (mode 1 in a run), else null
    int t;                   // iteration number (1-based) for the control block
    int fixed;               // no early stop
};

hipError_t launch_valu(const StepArgs &a, Mode mode, const AccumPlan &plan, hipStream_t s);

// Reduce the per-workgroup partials in fixed order, form fp32 centres (Eq. (1)),
// write counts, and (compare != 0) flag a change against prev for iteration t.
hipError_t launch_finalize(const double *part_sums, const int32_t *part_counts, int groups,
                           int K, int M, const float *prev, float *centers, int32_t *counts,
                           Ctl *ctl, int t, int fixed, int compare, hipStream_t s);

hipError_t launch_ctl_reset(Ctl *ctl, hipStream_t s);

}  // namespace lloyd
