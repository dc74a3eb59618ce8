// Cross-workgroup reduction that ends the fused assign/accumulate launch:
// centres of gravity (Eq. (1)) from the per-workgroup partials and the
// congruence test of Algorithm 1 steps 6-7.
//
// Every workgroup writes its fp64 partial sums [K][M] and counts [K], then takes
// a ticket in its group of kGroup workgroups. The last workgroup of a group to
// arrive adds the group's partials in workgroup order into a group partial and
// takes a ticket at the top level; the last group reducer adds the group
// partials in group order, forms every centre as fp32(sum / count) (the previous
// centre when the count is 0), writes the counts, and records whether any centre
// changed bitwise. The order of every addition is fixed by the problem shape,
// not by which workgroup arrives last, so the result is deterministic. The
// tickets are the only atomics (integer); partials are published with a
// device-scope release fence and read after a device-scope acquire fence.
// There are at most kGroup groups (at most kGroup * kGroup workgroups).
// No workgroup ever waits for another.
#pragma once

#include "lloyd.h"

namespace lloyd {

constexpr int kGroup = 16;   // workgroups per first-level group
static_assert(kCUs <= kGroup * kGroup, "two reduction levels cover every workgroup");

struct TreeArgs {
    double *part_sums;       // [G][K][M]
    int32_t *part_counts;    // [G][K]
    double *grp_sums;        // [NG][K][M]
    int32_t *grp_counts;     // [NG][K]
    uint32_t *tickets;       // [NG + 1], zero between launches
    int G, K, M;
    const float *prev;       // previous centres (may alias centers)
    float *centers;
    int32_t *counts;
    Ctl *ctl;                // change flag of iteration t (may be null)
    int t;
    int compare;
};

// Must be called by every thread of every workgroup after the workgroup's
// partial has been written; s_scratch needs 4 + 4*K bytes of LDS.
__device__ inline void tree_finalize(const TreeArgs &r, uint32_t *s_scratch)
{
    const int tid = threadIdx.x, nthr = blockDim.x;
    const int KM = r.K * r.M;
    const int NG = (r.G + kGroup - 1) / kGroup;
    const int q = blockIdx.x / kGroup;
    const int g0 = q * kGroup;
    const int g1 = (g0 + kGroup < r.G) ? g0 + kGroup : r.G;

    // ---- first level: the last workgroup of group q
    // The barrier completes every wave's stores (workgroup release); one
    // device-scope release fence per workgroup then publishes them, and only
    // the last arrival takes a device-scope acquire (a full fence would also
    // invalidate the caches in every workgroup).
    __syncthreads();
    if (tid == 0) {
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
        s_scratch[0] = atomicAdd(&r.tickets[q], 1u);
        if (s_scratch[0] == (uint32_t)(g1 - g0 - 1)) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    }
    __syncthreads();
    if (s_scratch[0] != (uint32_t)(g1 - g0 - 1)) return;
    // (plain loads: the acquire above invalidated this compute unit's caches)
    for (int e = tid; e < KM; e += nthr) {
        double v[kGroup];
#pragma unroll
        for (int u = 0; u < kGroup; ++u)
            v[u] = (g0 + u < g1) ? r.part_sums[(int64_t)(g0 + u) * KM + e] : 0.0;
        double s = v[0];
#pragma unroll
        for (int u = 1; u < kGroup; ++u)
            if (g0 + u < g1) s = s + v[u];
        r.grp_sums[(int64_t)q * KM + e] = s;
    }
    for (int k = tid; k < r.K; k += nthr) {
        int32_t c = 0;
#pragma unroll
        for (int u = 0; u < kGroup; ++u)
            if (g0 + u < g1) c += r.part_counts[(int64_t)(g0 + u) * r.K + k];
        r.grp_counts[(int64_t)q * r.K + k] = c;
    }
    if (tid == 0) r.tickets[q] = 0;      // ready for the next launch

    // ---- second level: the last group reducer
    __syncthreads();
    if (tid == 0) {
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
        s_scratch[0] = atomicAdd(&r.tickets[NG], 1u);
        if (s_scratch[0] == (uint32_t)(NG - 1)) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    }
    __syncthreads();
    if (s_scratch[0] != (uint32_t)(NG - 1)) return;
    int32_t *s_cnt = reinterpret_cast<int32_t *>(s_scratch + 1);
    for (int k = tid; k < r.K; k += nthr) {
        int32_t c = 0;
#pragma unroll 16
        for (int gq = 0; gq < NG; ++gq) c += r.grp_counts[(int64_t)gq * r.K + k];
        s_cnt[k] = c;
        r.counts[k] = c;
    }
    __syncthreads();                 // every thread has read the ticket; counts are in LDS
    if (tid == 0) s_scratch[0] = 0;  // reused as the "some centre changed" flag
    __syncthreads();
    int changed = 0;
    for (int e = tid; e < KM; e += nthr) {
        double v[kGroup];
#pragma unroll
        for (int u = 0; u < kGroup; ++u) v[u] = (u < NG) ? r.grp_sums[(int64_t)u * KM + e] : 0.0;
        double s = v[0];
#pragma unroll
        for (int u = 1; u < kGroup; ++u)
            if (u < NG) s = s + v[u];
        const int32_t c = s_cnt[e / r.M];
        const float old = r.prev[e];
        const float nv = c > 0 ? (float)(s / (double)c) : old;
        changed |= (__float_as_uint(nv) != __float_as_uint(old)) ? 1 : 0;
        r.centers[e] = nv;
    }
    // (an explicit LDS flag rather than __syncthreads_or, which takes static LDS)
    if (changed) s_scratch[0] = 1;
    __syncthreads();
    const int any = (int)s_scratch[0];
    if (tid == 0) {
        if (r.compare && r.ctl != nullptr) r.ctl->changed[r.t & 1] = any ? 1 : 0;
        r.tickets[NG] = 0;
    }
}

}  // namespace lloyd
