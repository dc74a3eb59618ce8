// Centres of gravity (Eq. (1)) from the per-workgroup partials, and the
// congruence test of Algorithm 1 steps 6-7, in one launch.
//
// Stage 1 (every workgroup): a workgroup owns 64 consecutive entries of the
// flattened [K][M] sums (or of the [K] counts). Its 16 wavefronts each add a
// contiguous 1/16 of the G partials for those entries (lane = entry, so every
// load of a wavefront is one 512-byte contiguous row), and wavefront 0 adds the
// 16 wavefront sums in order. The totals go to the workspace.
// Stage 2 (the last workgroup to finish, found with an integer ticket): for
// every (k, j), centre = fp32(total / count) in fp64, or the previous centre
// when the count is 0; counts are written; any bitwise difference from the
// previous centre sets the iteration's change flag.
//
// Every addition happens in an order fixed by the problem shape, so the result
// is deterministic. The ticket is the only atomic; workgroups publish their
// totals with a device-scope release and the last one reads them after a
// device-scope acquire.
#include "lloyd.h"

namespace lloyd {

namespace {

constexpr int kFinWaves = 16;
constexpr int kFinThreads = kFinWaves * kWave;

__global__ void __launch_bounds__(kFinThreads)
lloyd_finalize_kernel(const double *__restrict__ part_sums, const int32_t *__restrict__ part_counts,
                      int G, int K, int M, const float *prev, float *centers,
                      int32_t *__restrict__ counts, double *__restrict__ tot_sums,
                      int32_t *__restrict__ tot_counts, uint32_t *__restrict__ ticket, Ctl *ctl,
                      int t, int fixed, int compare)
{
    const int tid = threadIdx.x;
    const int wave = tid / kWave, lane = tid % kWave;
    if (ctl != nullptr && !fixed) {
        const bool stop =
            ctl->converged_at != 0 || ((t - 1 >= 2) && ctl->changed[(t - 1) & 1] == 0);
        if (stop) {
            if (blockIdx.x == 0 && tid == 0 && ctl->converged_at == 0) ctl->converged_at = t - 1;
            return;
        }
    }
    __shared__ double sred[kFinWaves][kWave];
    __shared__ int32_t cred[kFinWaves][kWave];
    __shared__ uint32_t s_ticket;

    const int KM = K * M;
    const int nsum_blocks = (KM + kWave - 1) / kWave;
    const int per = (G + kFinWaves - 1) / kFinWaves;
    const int g0 = wave * per;
    const int g1 = (g0 + per < G) ? g0 + per : G;

    if ((int)blockIdx.x < nsum_blocks) {
        const int e = blockIdx.x * kWave + lane;
        double acc = 0.0;
        if (e < KM) {
            const double *p = part_sums + e;
            int g = g0;
            for (; g + 8 <= g1; g += 8) {
                double v[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) v[u] = p[(int64_t)(g + u) * KM];
#pragma unroll
                for (int u = 0; u < 8; ++u) acc = acc + v[u];
            }
            for (; g < g1; ++g) acc = acc + p[(int64_t)g * KM];
        }
        sred[wave][lane] = acc;
        __syncthreads();
        if (wave == 0 && e < KM) {
            double s = 0.0;
            for (int w = 0; w < kFinWaves; ++w) s = s + sred[w][lane];
            tot_sums[e] = s;
        }
    } else {
        const int k = (blockIdx.x - nsum_blocks) * kWave + lane;
        int32_t c = 0;
        if (k < K)
            for (int g = g0; g < g1; ++g) c += part_counts[(int64_t)g * K + k];
        cred[wave][lane] = c;
        __syncthreads();
        if (wave == 0 && k < K) {
            int32_t s = 0;
            for (int w = 0; w < kFinWaves; ++w) s += cred[w][lane];
            tot_counts[k] = s;
        }
    }

    // publish, then take a ticket; the last workgroup forms the centres
    __threadfence();
    __syncthreads();
    if (tid == 0) s_ticket = atomicAdd(ticket, 1u);
    __syncthreads();
    if (s_ticket != gridDim.x - 1) return;
    __threadfence();

    int changed = 0;
    for (int e = tid; e < KM; e += kFinThreads) {
        const int k = e / M;
        const int32_t cnt = __hip_atomic_load(&tot_counts[k], __ATOMIC_RELAXED,
                                              __HIP_MEMORY_SCOPE_AGENT);
        const double tot = __hip_atomic_load(&tot_sums[e], __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT);
        const float old = prev[e];
        const float nv = cnt > 0 ? (float)(tot / (double)cnt) : old;
        changed |= (__float_as_uint(nv) != __float_as_uint(old)) ? 1 : 0;
        centers[e] = nv;
    }
    for (int k = tid; k < K; k += kFinThreads)
        counts[k] = __hip_atomic_load(&tot_counts[k], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const int any = __syncthreads_or(changed);
    if (tid == 0) {
        if (compare && ctl != nullptr && any) ctl->changed[t & 1] = 1;
        *ticket = 0;            // ready for the next launch (stream-ordered)
    }
}

__global__ void ctl_reset_kernel(Ctl *ctl)
{
    int32_t *p = reinterpret_cast<int32_t *>(ctl);
    const int i = threadIdx.x;
    if (i < (int)(sizeof(Ctl) / sizeof(int32_t))) p[i] = 0;
}

}  // namespace

int finalize_blocks(int K, int M)
{
    return (K * M + kWave - 1) / kWave + (K + kWave - 1) / kWave;
}

hipError_t launch_finalize(const FinalizeArgs &f, const float *prev, float *centers,
                           int32_t *counts, Ctl *ctl, int t, int fixed, int compare, hipStream_t s)
{
    hipLaunchKernelGGL(lloyd_finalize_kernel, dim3(finalize_blocks(f.K, f.M)), dim3(kFinThreads), 0,
                       s, f.part_sums, f.part_counts, f.groups, f.K, f.M, prev, centers, counts,
                       f.tot_sums, f.tot_counts, f.ticket, ctl, t, fixed, compare);
    return hipGetLastError();
}

hipError_t launch_ctl_reset(Ctl *ctl, hipStream_t s)
{
    hipLaunchKernelGGL(ctl_reset_kernel, dim3(1), dim3(64), 0, s, ctl);
    return hipGetLastError();
}

}  // namespace lloyd
