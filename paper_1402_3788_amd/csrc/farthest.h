// Farthest-point initial centres (farthest.hip).
#pragma once

#include "lloyd.h"

namespace lloyd {

struct FarthestPlan {
    int waves;          // wavefronts per workgroup
    int groups;         // persistent workgroups of each pass
    size_t lds_bytes;   // dynamic LDS per workgroup (one tile slot per wave)
};

struct FarthestArgs {
    const float *X;
    int64_t n;
    int M;
    int K;              // 1 <= K <= n
    double *nearest;    // [n] fp64 nearest-centre distances (-1 = chosen)
    double *cand_v;     // [2][groups] farthest distance per workgroup and pass parity
    int32_t *cand_i;    // [2][groups] its object index
    int32_t *idx;       // out: [K] chosen objects
    float *centers;     // out: [K][M] their rows
    const int32_t *seeds;  // [nseeds] device seeds, or null: one seed, object 0
    int nseeds;            // 1 <= nseeds <= K
};

FarthestPlan plan_farthest(int64_t n, int M);

// Enqueues the K launches of the traversal on s.
hipError_t launch_farthest(const FarthestArgs &a, const FarthestPlan &plan, hipStream_t s);

}  // namespace lloyd
