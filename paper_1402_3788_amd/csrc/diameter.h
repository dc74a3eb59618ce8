// Centre of gravity of the whole set and the diameter of Eq. (3) (diameter.hip).
#pragma once

#include "lloyd.h"

namespace lloyd {

struct CentroidPlan {
    int threads;        // per workgroup, a multiple of M
    int groups;         // workgroups (rows of fp64 partial sums)
};

struct DiameterPlan {
    int ks;             // 32-feature steps of the operands: ceil((M + 2) / 32)
    int64_t npad;       // objects the operand arrays hold (zero rows past n)
    int64_t row_blocks; // items per column chunk
    int64_t chunks;     // column chunks
};

// Best pair of one work item: largest fp64 squared distance, then lowest k, l.
struct DiamBest {
    double d;
    int32_t k, l;
};

struct DiameterArgs {
    const float *X;
    int64_t n;
    int M;
    float *centroid_ws;       // [M] centre of gravity (written by launch_centroid)
    uint4 *ah, *al, *bh, *bl; // [npad][4 ks] split operands
    uint32_t *counters;       // [0] largest |y|^2 (fp32 bits), [1] key of the pass-1 maximum,
                              // [2] nonzero if X holds a NaN or an infinity
    DiamBest *slots;          // [row_blocks * chunks]
    double *d2;               // out: squared diameter
    int32_t *pair;            // out: [2] the pair
};

CentroidPlan plan_centroid(int64_t n, int M);
// Two launches: fp64 partial sums per workgroup, then the fp32 centroid
// (written to centroid_ws and/or centroid_out, either may be null) and, when
// counters is not null, the reset of the diameter counters.
hipError_t launch_centroid(const float *X, int64_t n, int M, double *part, float *centroid_ws,
                           float *centroid_out, uint32_t *counters, const CentroidPlan &pl,
                           hipStream_t s);
DiameterPlan plan_diameter(int64_t n, int M);
// Four launches after launch_centroid: operands, pass 1, pass 2, final.
hipError_t launch_diameter(const DiameterArgs &a, const DiameterPlan &pl, hipStream_t s);

}  // namespace lloyd
