// Centres of gravity (Eq. (1)) and the congruence test of Algorithm 1 steps
// 6-7, from the per-workgroup partials that an accumulating launch leaves in
// the workspace.
//
// One workgroup per cluster k. Workgroup g of the accumulating launch wrote a
// row of K*M fp64 feature sums and K int32 counts. The sums of every (k, j)
// entry are added in an order that depends only on the number of workgroups G:
// the rows of each group of kGroup consecutive workgroups in ascending order,
// then the group sums in ascending group order. One thread per (entry, group)
// issues its kGroup loads together, so the whole reduction is one round trip
// of loads and one LDS pass. The new centre is fp32(sum / count), or the
// previous centre for an empty cluster (count 0). Each workgroup ORs into the
// iteration's change flag whether any of its centre values changed bitwise;
// workgroup 0 clears the flag the next iteration will use.
#include "lloyd.h"

namespace lloyd {

namespace {

constexpr int kGroup = 16;   // workgroup rows per first-level group
constexpr int kThreads = 1024;

__global__ void __launch_bounds__(kThreads)
centres_kernel(const double *__restrict__ part_sums, const int32_t *__restrict__ part_counts,
               int G, int K, int M, const float *prev, float *centers, int32_t *counts, Ctl *ctl,
               int t, int fixed, int compare)
{
    // Iterations past convergence: the assign launch of this iteration found
    // the centres congruent and recorded converged_at (its first workgroup);
    // that launch has finished, so the value is settled here. (The change
    // flags are not read: workgroup 0 of this launch clears one of them.)
    // The test waits until the loads below are in flight.
    const bool skip = !fixed && ctl != nullptr && ctl->converged_at != 0;
    extern __shared__ __align__(16) unsigned char smem[];
    const int k = blockIdx.x;
    const int MW = M + 1;                       // M sums, then the count
    const int NG = (G + kGroup - 1) / kGroup;
    const int64_t KM = (int64_t)K * M;
    double *sub = reinterpret_cast<double *>(smem);           // [MW][NG] group sums
    int32_t *s_changed = reinterpret_cast<int32_t *>(sub + (size_t)MW * NG);

    // this workgroup's previous centre (threads 0 .. M-1; blockDim.x > M)
    const float old = threadIdx.x < M ? prev[(int64_t)k * M + threadIdx.x] : 0.f;
    if (threadIdx.x == 0) *s_changed = 0;
    for (int it = threadIdx.x; it < MW * NG; it += blockDim.x) {
        const int e = it % MW, q = it / MW;
        const int g0 = q * kGroup;
        const int ng = G - g0 < kGroup ? G - g0 : kGroup;
        double s;
        if (e < M) {
            const double *p = part_sums + (int64_t)g0 * KM + (int64_t)k * M + e;
            double v[kGroup];
#pragma unroll
            for (int u = 0; u < kGroup; ++u) v[u] = u < ng ? p[(int64_t)u * KM] : 0.0;
            s = v[0];
#pragma unroll
            for (int u = 1; u < kGroup; ++u)
                if (u < ng) s = s + v[u];
        } else {
            const int32_t *p = part_counts + (int64_t)g0 * K + k;
            int32_t c = 0;
#pragma unroll
            for (int u = 0; u < kGroup; ++u)
                if (u < ng) c += p[(int64_t)u * K];
            s = (double)c;                      // exact: c < 2^31
        }
        sub[e * NG + q] = s;
    }
    __syncthreads();
    if (skip) return;                           // uniform: every thread read the same value

    int32_t c = 0;
    for (int q = 0; q < NG; ++q) c += (int32_t)sub[M * NG + q];
    int changed = 0;
    if (threadIdx.x < M) {
        const int e = threadIdx.x;
        double s = sub[e * NG];
        for (int q = 1; q < NG; ++q) s = s + sub[e * NG + q];
        const float nv = c > 0 ? (float)(s / (double)c) : old;
        changed = (__float_as_uint(nv) != __float_as_uint(old)) ? 1 : 0;
        centers[(int64_t)k * M + e] = nv;
    }
    if (threadIdx.x == 0) counts[k] = c;
    if (changed) *s_changed = 1;
    __syncthreads();
    if (threadIdx.x == 0 && compare && ctl != nullptr) {
        if (*s_changed) atomicOr(&ctl->changed[t & 1], 1);
        // the flag of iteration t + 1 was last read by the launch of
        // iteration t (which has finished); clear it for the next reduction
        if (k == 0) ctl->changed[(t + 1) & 1] = 0;
    }
}

}  // namespace

size_t centres_lds_bytes(int M, int groups)
{
    const int NG = (groups + kGroup - 1) / kGroup;
    return (size_t)(M + 1) * NG * sizeof(double) + 16;
}

hipError_t launch_centres(const StepArgs &a, int groups, hipStream_t s)
{
    if (groups < 1 || groups > kGroup * kGroup) return hipErrorInvalidValue;
    const int NG = (groups + kGroup - 1) / kGroup;
    const int items = (a.M + 1) * NG;
    int threads = (items + kWave - 1) / kWave * kWave;
    if (threads > kThreads) threads = kThreads;
    hipLaunchKernelGGL(centres_kernel, dim3(a.K), dim3(threads), centres_lds_bytes(a.M, groups), s,
                       a.part_sums, a.part_counts, groups, a.K, a.M, a.C, a.centers_out,
                       a.counts_out, a.ctl, a.t, a.fixed, a.compare);
    return hipGetLastError();
}

}  // namespace lloyd
