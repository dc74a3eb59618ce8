// Reset of the iteration control block at the start of a library call.
#include "lloyd.h"

namespace lloyd {

namespace {

__global__ void ctl_reset_kernel(Ctl *ctl)
{
    int32_t *p = reinterpret_cast<int32_t *>(ctl);
    const int i = threadIdx.x;
    if (i < (int)(sizeof(Ctl) / sizeof(int32_t))) p[i] = 0;
}

}  // namespace

hipError_t launch_ctl_reset(Ctl *ctl, hipStream_t s)
{
    hipLaunchKernelGGL(ctl_reset_kernel, dim3(1), dim3(64), 0, s, ctl);
    return hipGetLastError();
}

}  // namespace lloyd
