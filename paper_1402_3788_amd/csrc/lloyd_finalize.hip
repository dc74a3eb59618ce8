// Centres of gravity (Eq. (1)) from the per-workgroup partials, and the
// congruence test of Algorithm 1 steps 6-7.
//
// One workgroup per cluster k. The fp64 partial sums of the G workgroups are
// added in a fixed order (stripe s of feature j takes workgroups s, s+S, ...,
// then the S stripe sums are added in stripe order), so the result depends only
// on the problem shape. The centre is the fp64 sum divided by the count in fp64
// and rounded once to fp32; an empty cluster keeps its previous centre. The
// new centre is compared bitwise with the previous one and any difference is
// OR-ed (integer atomic) into the control block's flag for iteration t.
#include "lloyd.h"

namespace lloyd {

namespace {

__global__ void __launch_bounds__(256)
lloyd_finalize_kernel(const double *__restrict__ part_sums, const int32_t *__restrict__ part_counts,
                      int G, int K, int M, const float *prev, float *centers,
                      int32_t *__restrict__ counts, Ctl *ctl, int t, int fixed, int compare)
{
    const int k = blockIdx.x;
    const int tid = threadIdx.x;
    if (ctl != nullptr && !fixed) {
        bool stop = ctl->converged_at != 0 || ((t - 1 >= 2) && ctl->changed[(t - 1) & 1] == 0);
        if (stop) {
            if (k == 0 && tid == 0 && ctl->converged_at == 0) ctl->converged_at = t - 1;
            return;
        }
    }
    __shared__ double sred[256];
    __shared__ int32_t cred[256];

    int32_t c = 0;
    for (int g = tid; g < G; g += 256) c += part_counts[(int64_t)g * K + k];
    cred[tid] = c;

    const int S = 256 / M;                 // stripes per feature (M <= 64, so S >= 4)
    double acc = 0.0;
    if (tid < S * M) {
        const int j = tid % M, s = tid / M;
        for (int g = s; g < G; g += S) acc = acc + part_sums[((int64_t)g * K + k) * M + j];
    }
    sred[tid] = acc;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if (tid < w) cred[tid] += cred[tid + w];
        __syncthreads();
    }
    const int32_t cnt = cred[0];

    int changed = 0;
    if (tid < M) {
        double tot = 0.0;
        for (int s = 0; s < S; ++s) tot = tot + sred[s * M + tid];
        const float old = prev[(int64_t)k * M + tid];
        const float nv = cnt > 0 ? (float)(tot / (double)cnt) : old;
        changed = __float_as_uint(nv) != __float_as_uint(old);
        centers[(int64_t)k * M + tid] = nv;
    }
    if (tid == 0) counts[k] = cnt;
    const int any = __syncthreads_or(changed);
    if (compare && ctl != nullptr && tid == 0 && any) atomicOr(&ctl->changed[t & 1], 1);
}

__global__ void ctl_reset_kernel(Ctl *ctl)
{
    int32_t *p = reinterpret_cast<int32_t *>(ctl);
    const int i = threadIdx.x;
    if (i < (int)(sizeof(Ctl) / sizeof(int32_t))) p[i] = 0;
}

}  // namespace

hipError_t launch_finalize(const double *part_sums, const int32_t *part_counts, int groups, int K,
                           int M, const float *prev, float *centers, int32_t *counts, Ctl *ctl,
                           int t, int fixed, int compare, hipStream_t s)
{
    hipLaunchKernelGGL(lloyd_finalize_kernel, dim3(K), dim3(256), 0, s, part_sums, part_counts,
                       groups, K, M, prev, centers, counts, ctl, t, fixed, compare);
    return hipGetLastError();
}

hipError_t launch_ctl_reset(Ctl *ctl, hipStream_t s)
{
    hipLaunchKernelGGL(ctl_reset_kernel, dim3(1), dim3(64), 0, s, ctl);
    return hipGetLastError();
}

}  // namespace lloyd
