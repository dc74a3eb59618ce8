// Centres of gravity (Eq. (1)) and the congruence test of Algorithm 1 steps
// 6-7, from the per-workgroup partials that an accumulating launch leaves in
// the workspace.
//
// Workgroup g (of G <= 256) of the accumulating launch wrote a row of K*M fp64
// feature sums and a column of K int32 counts (a [K][G] table, so the G counts
// of a cluster are consecutive). One wavefront forms eight coordinates
// j = 8b .. 8b+7 of centre k: lane (r, f) = (lane / 8, lane % 8) reads
// coordinate 8b + f of rows r, r + 8, r + 16, ... (eight consecutive
// coordinates of eight rows per load instruction) and adds them in four
// interleaved running sums (rows r + 8u with u = 0, 4, 8, ... into the first,
// u = 1, 5, ... into the second, and so on) that are then added pairwise; the
// eight lanes of a coordinate are combined by a butterfly over r (partner
// lane l ^ 32, then l ^ 16, then l ^ 8). fp64 addition is commutative, so
// both lanes of a pair form the same value, and the order of every addition
// depends only on G. The count of cluster k is formed in every wave the same
// way (integers: order-free). Every load is issued before the first addition,
// so a wave waits on one round trip to memory. The new coordinate is
// fp32(sum / count), or the previous one for an empty cluster (count 0). A
// wave any of whose coordinates changed bitwise ORs 1 into the iteration's
// change flag; the wave of (0, 0) clears the flag the next iteration will use.
#include "lloyd.h"

namespace lloyd {

namespace {

constexpr int kMaxRows = 256;                 // workgroup partials (G)
constexpr int kFeat = 8;                      // coordinates per wave
constexpr int kRowLanes = kWave / kFeat;      // 8 rows per load instruction
constexpr int kRowSteps = kMaxRows / kRowLanes;   // 32 loads per lane
static_assert(kMaxRows >= kCUs, "every accumulating launch has at most kCUs workgroups");

__global__ void __launch_bounds__(kWave)
centres_kernel(const double *__restrict__ part_sums, const int32_t *__restrict__ part_counts,
               int G, int K, int M, const float *prev, float *centers, int32_t *counts, Ctl *ctl,
               int t, int fixed, int compare)
{
    // Iterations past convergence: the assign launch of this iteration found
    // the centres congruent and recorded converged_at (its first workgroup);
    // that launch has finished, so the value is settled here. (The change
    // flags are not read: wave (0, 0) of this launch clears one of them.)
    // The test waits until the loads below are in flight.
    const bool skip = !fixed && ctl != nullptr && ctl->converged_at != 0;
    const int nb = (M + kFeat - 1) / kFeat;
    const int k = blockIdx.x / nb, b = blockIdx.x % nb;
    const int lane = threadIdx.x;
    const int r = lane / kFeat, f = lane % kFeat;
    const int e = kFeat * b + f;
    const bool live = e < M;
    const int64_t KM = (int64_t)K * M;
    const double *col = part_sums + (int64_t)k * M + (live ? e : 0);

    const float old = live ? prev[(int64_t)k * M + e] : 0.f;
    double v[kRowSteps];
#pragma unroll
    for (int u = 0; u < kRowSteps; ++u) {
        const int g = r + kRowLanes * u;
        v[u] = (live && g < G) ? col[(int64_t)g * KM] : 0.0;
    }
    int32_t c[kMaxRows / kWave];
#pragma unroll
    for (int u = 0; u < kMaxRows / kWave; ++u) {
        const int g = lane + kWave * u;
        c[u] = g < G ? part_counts[(int64_t)k * G + g] : 0;
    }
    int32_t n = 0;
#pragma unroll
    for (int u = 0; u < kMaxRows / kWave; ++u) n += c[u];
#pragma unroll
    for (int m = kWave / 2; m >= 1; m /= 2) n += __shfl_xor(n, m, kWave);

    // rows past G hold zeros here, which leave a running sum unchanged
    // (partial sums are never -0.0: they start from +0.0)
    double a[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) a[i] = v[i];
#pragma unroll
    for (int u = 4; u < kRowSteps; ++u) a[u % 4] = a[u % 4] + v[u];
    double s = (a[0] + a[1]) + (a[2] + a[3]);
#pragma unroll
    for (int m = kWave / 2; m >= kFeat; m /= 2) s = s + __shfl_xor(s, m, kWave);

    if (skip) return;                           // uniform: every lane read the same value
    int changed = 0;
    if (r == 0 && live) {
        const float nv = n > 0 ? (float)(s / (double)n) : old;
        centers[(int64_t)k * M + e] = nv;
        changed = __float_as_uint(nv) != __float_as_uint(old);
    }
    const bool any = __ballot(changed) != 0;
    if (lane != 0) return;
    if (b == 0) counts[k] = n;
    if (compare && ctl != nullptr) {
        if (any) atomicOr(&ctl->changed[t & 1], 1);
        // the flag of iteration t + 1 was last read by the launch of
        // iteration t (which has finished); clear it for the next reduction
        if (k == 0 && b == 0) ctl->changed[(t + 1) & 1] = 0;
    }
}

}  // namespace

hipError_t launch_centres(const StepArgs &a, int groups, hipStream_t s)
{
    if (groups < 1 || groups > kMaxRows || a.M < 1 || a.M > kMaxM) return hipErrorInvalidValue;
    const int nb = (a.M + kFeat - 1) / kFeat;
    hipLaunchKernelGGL(centres_kernel, dim3(a.K * nb), dim3(kWave), 0, s, a.part_sums,
                       a.part_counts, groups, a.K, a.M, a.C, a.centers_out, a.counts_out, a.ctl,
                       a.t, a.fixed, a.compare);
    return hipGetLastError();
}

}  // namespace lloyd
