// Device helpers shared by the distance kernels: streaming a 64-object tile of
// X through registers into LDS, and the fp64 re-decision of close calls.
#pragma once

#include "lloyd.h"

#include <math.h>

namespace lloyd {

template <int M>
struct TileGeom {
    static constexpr int kFloats = kWave * M;          // floats per 64-object tile
    static constexpr int kVec = kFloats / 4;           // float4s per tile (64*M divisible by 4)
    static constexpr int kVecPerLane = (kVec + kWave - 1) / kWave;
};

// Issue the loads of tile q (objects 64q .. 64q+63) into registers.
template <int M>
__device__ inline void load_tile(const float *__restrict__ X, int64_t n, int64_t q, int lane,
                                 float4 (&buf)[TileGeom<M>::kVecPerLane])
{
    using G = TileGeom<M>;
    const int64_t f0 = q * (int64_t)G::kFloats;
    const int64_t total = n * (int64_t)M;
    const int64_t left = total - f0;
    const int nf = left < G::kFloats ? (int)left : G::kFloats;   // floats present
    const float4 *src = reinterpret_cast<const float4 *>(X + f0);
    if (nf == G::kFloats) {             // every tile but possibly the last
#pragma unroll
        for (int v = 0; v < G::kVecPerLane; ++v) {
            const int idx = lane + kWave * v;
            if (idx < G::kVec) buf[v] = src[idx];
        }
        return;
    }
#pragma unroll
    for (int v = 0; v < G::kVecPerLane; ++v) {
        const int idx = lane + kWave * v;
        if (idx < G::kVec) {
            if (4 * idx + 3 < nf) {
                buf[v] = src[idx];
            } else {
                const float *s = X + f0 + 4 * idx;
                float4 r = make_float4(0.f, 0.f, 0.f, 0.f);
                if (4 * idx + 0 < nf) r.x = s[0];
                if (4 * idx + 1 < nf) r.y = s[1];
                if (4 * idx + 2 < nf) r.z = s[2];
                buf[v] = r;
            }
        }
    }
}

template <int M>
__device__ inline void store_tile(float *tile, int lane,
                                  const float4 (&buf)[TileGeom<M>::kVecPerLane])
{
    using G = TileGeom<M>;
    float4 *dst = reinterpret_cast<float4 *>(tile);
#pragma unroll
    for (int v = 0; v < G::kVecPerLane; ++v) {
        const int idx = lane + kWave * v;
        if (idx < G::kVec) dst[idx] = buf[v];
    }
}

// fp64 squared distance in the reference operation order: for j ascending,
// e = x_j - c_j, then d = d + e*e, every operation rounded on its own (this file
// is compiled with -ffp-contract=off, so nothing is fused).
template <int M>
__device__ inline int argmin_fp64(const float (&x)[M], const float *__restrict__ C, int K,
                                  double &best_out)
{
    double best = INFINITY;
    int lab = 0;
    for (int k = 0; k < K; ++k) {
        const float *c = C + k * M;
        double d = 0.0;
#pragma unroll
        for (int j = 0; j < M; ++j) {
            const double e = (double)x[j] - (double)c[j];
            const double sq = e * e;
            d = d + sq;
        }
        if (d < best) {
            best = d;
            lab = k;
        }
    }
    best_out = best;
    return lab;
}

}  // namespace lloyd

namespace lloyd {

// Accumulation layout: a wavefront adds up to P members of one cluster per step,
// one member per group of MW = M + 1 lanes (lane = slot * MW + column); columns
// 0..M-1 carry the features and column M carries the member count (adding 1.0
// per member, exact in fp64).
template <int M>
struct Slots {
    static constexpr int MW = M + 1;
    static constexpr int P = (kWave / MW >= 4) ? 4 : ((kWave / MW >= 2) ? 2 : 1);
    // floats per wave tile slot: 64 objects, then zeros (one full row, and at
    // least 4 floats for the matrix-core operand reads that run past a row)
    static constexpr int kTileFloats = (kWave * M + (M > 4 ? M : 4) + 3) / 4 * 4;
};


// Add the members of one 64-object tile into the wave's private fp64 slab
// slab[k][0..M] (feature sums and the count of cluster k: the numerator and
// denominator of Eq. (1)).
//
// lab is this lane's object label (-1: no object). tile holds the 64 objects'
// features, object-major, followed by at least one row of zeros; ones[0..63] = 1
// and ones[64] = 0. For each cluster present in the tile a ballot lists its
// members; member m (in ascending lane order) goes to slot m % P, each slot
// adds its members in order in fp64, the P slot sums are combined in a fixed
// tree and added once to the slab. Absent members read the zero row, so the
// loop has no branches. The order of every addition depends only on the labels.
template <int M>
__device__ inline void wave_accumulate(int lab, const float *tile, const float *ones,
                                       double *slab, int K, int lane)
{
    constexpr int MW = Slots<M>::MW, P = Slots<M>::P;
    const int s = lane / MW, j = lane - (lane / MW) * MW;
    // Value of member p for this lane: *(base + p * stride) (bytes). Lanes of
    // slot u take the position p_u of their step; the per-slot strides are zero
    // for the other slots, so the address is base + sum_u p_u * stride_u with
    // one multiply-add per slot and no selects. Lanes outside every slot read
    // row 0 and their sums are never used.
    const char *base = (j < M) ? reinterpret_cast<const char *>(tile + j)
                               : reinterpret_cast<const char *>(ones);
    const uint32_t stride = (j < M) ? M * 4 : 4;
    uint32_t st[P];
#pragma unroll
    for (int u = 0; u < P; ++u) st[u] = (s == u) ? stride : 0u;
    for (int k = 0; k < K; ++k) {
        uint64_t mask = __ballot(lab == k);
        if (mask == 0) continue;
        const int members = __popcll(mask);
        const double old = (lane < MW) ? slab[k * MW + lane] : 0.0;
        double acc = 0.0;
        do {
            uint32_t offa = 0, offb = 0;
#pragma unroll
            for (int u = 0; u < P; ++u) {          // positions off the mask, in order
                const uint32_t p = mask ? (uint32_t)__builtin_ctzll(mask) : (uint32_t)kWave;
                mask &= ~(1ull << (p & 63));
                offa += p * st[u];
            }
#pragma unroll
            for (int u = 0; u < P; ++u) {
                const uint32_t p = mask ? (uint32_t)__builtin_ctzll(mask) : (uint32_t)kWave;
                mask &= ~(1ull << (p & 63));
                offb += p * st[u];
            }
            const float va = *reinterpret_cast<const float *>(base + offa);
            const float vb = *reinterpret_cast<const float *>(base + offb);
            acc = acc + (double)va;
            acc = acc + (double)vb;
        } while (mask);
        double t = acc;
        if (P >= 2) t = t + __shfl_down(t, MW, kWave);        // slots (0,1) and (2,3)
        if (P >= 4) t = t + __shfl_down(t, 2 * MW, kWave);    // then the two pairs
        if (lane < MW) slab[k * MW + lane] = old + t;
        if (MW > kWave && lane == 0)                          // M = 64: no lane for the count
            slab[k * MW + M] = slab[k * MW + M] + (double)members;
    }
}

}  // namespace lloyd
