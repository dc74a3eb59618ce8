// Fused assign + accumulate on the vector ALU (small K).
//
// One wavefront owns a 64-object tile at a time (one object per lane) and walks
// its tiles with a fixed stride, so every sum below is formed in an order that
// depends only on the problem shape:
//   1. the tile's 64*M fp32 values are streamed from HBM with 16-byte loads into
//      the wave's LDS slot (the next tile's loads are issued before the current
//      tile is processed) and each lane reads its own object's M features;
//   2. assignment (Algorithm 1 steps 2/4, Eq. (2)): the squared distance to every
//      centre in fp32 (centres are wave-uniform and come through scalar loads),
//      keeping the best and second-best; if the two are closer than the fp32
//      error bound allows to call, the lane recomputes all K distances in fp64
//      in a fixed operation order and takes the lowest-index minimum, so the
//      label is the exact-arithmetic argmin;
//   3. accumulation (the numerator and denominator of Eq. (1)): for each cluster,
//      a ballot gives the lanes holding its members; lanes then act as feature
//      columns and add the members' features (read back from the LDS tile) into
//      an fp64 running sum, two members per step (one per half-wave), and the
//      sum is added to the wave's private fp64 slab. No atomics are involved.
//   4. at the end the workgroup adds its waves' slabs in wave order and writes
//      one fp64 partial per (cluster, feature) plus one count per cluster.
#include "lloyd.h"

#include <math.h>

namespace lloyd {

namespace {

__device__ inline bool stop_before(const Ctl *ctl, int t, int fixed)
{
    if (ctl == nullptr || fixed) return false;
    if (ctl->converged_at != 0) return true;
    return (t - 1 >= 2) && ctl->changed[(t - 1) & 1] == 0;
}

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

template <int M, int MODE>
__global__ void __launch_bounds__(256)
lloyd_valu_kernel(const float *__restrict__ X, int64_t n, const float *__restrict__ C, int K,
                  int32_t *__restrict__ labels, const int32_t *__restrict__ labels_in,
                  float *__restrict__ min_d2, double *__restrict__ part_sums,
                  int32_t *__restrict__ part_counts, Ctl *__restrict__ ctl, int t, int fixed)
{
    using G = TileGeom<M>;
    extern __shared__ __align__(16) unsigned char smem[];
    const int W = blockDim.x / kWave;
    const int wave = threadIdx.x / kWave;
    const int lane = threadIdx.x % kWave;

    if (MODE == kAssignAccum) {
        if (stop_before(ctl, t, fixed)) return;
        if (ctl != nullptr && blockIdx.x == 0 && threadIdx.x == 0) ctl->changed[t & 1] = 0;
    }

    float *tile = reinterpret_cast<float *>(smem) + wave * G::kFloats;
    double *slab = reinterpret_cast<double *>(smem + (size_t)W * G::kFloats * 4) +
                   (size_t)wave * K * M;
    int32_t *cnt = reinterpret_cast<int32_t *>(smem + (size_t)W * G::kFloats * 4 +
                                               (size_t)W * K * M * 8) + wave * K;
    if (MODE != kAssign) {
        for (int i = lane; i < K * M; i += kWave) slab[i] = 0.0;
        for (int i = lane; i < K; i += kWave) cnt[i] = 0;
    }

    // Bound on the relative error of an fp32 squared distance (M products and
    // M-1 sums, each rounded): |d_fp32 - d| <= gamma_{M+1} d. Two candidates are
    // called in fp32 only if their gap exceeds twice that with a 2x margin.
    constexpr float kTau = 4.0f * (float)(M + 2) * 5.9604645e-8f;

    const int64_t nq = (n + kWave - 1) / kWave;
    const int64_t stride = (int64_t)gridDim.x * W;
    int64_t q = (int64_t)blockIdx.x * W + wave;

    float4 buf[G::kVecPerLane];
    if (q < nq) load_tile<M>(X, n, q, lane, buf);
    int nfallback = 0;

    for (; q < nq; q += stride) {
        store_tile<M>(tile, lane, buf);
        __builtin_amdgcn_wave_barrier();
        if (q + stride < nq) load_tile<M>(X, n, q + stride, lane, buf);

        const int64_t i = q * kWave + lane;
        const bool valid = i < n;
        float x[M];
#pragma unroll
        for (int j = 0; j < M; ++j) x[j] = tile[lane * M + j];

        int lab;
        if (MODE == kAccumLabels) {
            lab = valid ? labels_in[i] : -1;
            if (lab < 0 || lab >= K) lab = -1;
        } else {
            float b1 = INFINITY, b2 = INFINITY;
            lab = 0;
            // centres are wave-uniform: scalar loads, the next centre's issued
            // before the current one is used
            float cc[M];
#pragma unroll
            for (int j = 0; j < M; ++j) cc[j] = C[j];
            for (int k = 0; k < K; ++k) {
                const int kn = (k + 1 < K) ? k + 1 : k;
                float cn[M];
#pragma unroll
                for (int j = 0; j < M; ++j) cn[j] = C[kn * M + j];
                float d = 0.f;
#pragma unroll
                for (int j = 0; j < M; ++j) {
                    const float e = x[j] - cc[j];
                    d = __builtin_fmaf(e, e, d);
                }
                // top-2: with b1 <= b2, the new second-best is the median of
                // (b1, b2, d) and the new best is min(b1, d)
                const bool lt = d < b1;
                b2 = __builtin_amdgcn_fmed3f(b1, b2, d);
                b1 = lt ? d : b1;
                lab = lt ? k : lab;
#pragma unroll
                for (int j = 0; j < M; ++j) cc[j] = cn[j];
            }
            const bool ok = (K == 1) || ((b2 - b1) > kTau * b2 && b2 >= 1e-30f);
            float dmin = b1;
            if (valid && !ok) {
                double bd;
                lab = argmin_fp64<M>(x, C, K, bd);
                dmin = (float)bd;
            }
            if (ctl != nullptr) {
                const uint64_t fb = __ballot(valid && !ok);
                nfallback += __popcll(fb);
            }
            if (valid) {
                labels[i] = lab;
                if (MODE == kAssign && min_d2 != nullptr) min_d2[i] = dmin;
            }
            if (!valid) lab = -1;
        }

        if (MODE != kAssign) {
            const bool hi = lane >= 32;
            const int jl = (M <= 32) ? (lane & 31) : lane;
            for (int k = 0; k < K; ++k) {
                uint64_t mask = __ballot(lab == k);
                if (mask == 0) continue;
                if (lane == 0) cnt[k] += __popcll(mask);
                double acc = 0.0;
                if (M <= 32) {
                    // two members per step: the lower half-wave takes the
                    // first, the upper half-wave the second
                    while (mask) {
                        const int p0 = __ffsll((unsigned long long)mask) - 1;
                        mask &= mask - 1;
                        int p1 = -1;
                        if (mask) {
                            p1 = __ffsll((unsigned long long)mask) - 1;
                            mask &= mask - 1;
                        }
                        const int pp = hi ? p1 : p0;
                        if (jl < M && pp >= 0) acc = acc + (double)tile[pp * M + jl];
                    }
                    const double upper = __shfl_down(acc, 32, kWave);
                    if (lane < M) slab[k * M + lane] = slab[k * M + lane] + (acc + upper);
                } else {
                    while (mask) {
                        const int p0 = __ffsll((unsigned long long)mask) - 1;
                        mask &= mask - 1;
                        if (lane < M) acc = acc + (double)tile[p0 * M + lane];
                    }
                    if (lane < M) slab[k * M + lane] = slab[k * M + lane] + acc;
                }
            }
        }
        __builtin_amdgcn_wave_barrier();
    }

    if (ctl != nullptr && lane == 0 && nfallback > 0) atomicAdd(&ctl->fallbacks, nfallback);

    if (MODE != kAssign) {
        __syncthreads();
        const double *slabs = reinterpret_cast<const double *>(smem + (size_t)W * G::kFloats * 4);
        const int32_t *cnts = reinterpret_cast<const int32_t *>(
            smem + (size_t)W * G::kFloats * 4 + (size_t)W * K * M * 8);
        double *out = part_sums + (int64_t)blockIdx.x * K * M;
        for (int idx = threadIdx.x; idx < K * M; idx += blockDim.x) {
            double s = slabs[idx];
            for (int w = 1; w < W; ++w) s = s + slabs[(size_t)w * K * M + idx];
            out[idx] = s;
        }
        for (int k = threadIdx.x; k < K; k += blockDim.x) {
            int32_t c = cnts[k];
            for (int w = 1; w < W; ++w) c += cnts[w * K + k];
            part_counts[(int64_t)blockIdx.x * K + k] = c;
        }
    }
}

template <int M>
hipError_t launch_m(const StepArgs &a, Mode mode, const AccumPlan &p, hipStream_t s)
{
    const dim3 grid(p.groups), block(p.waves * kWave);
    switch (mode) {
    case kAssign:
        hipLaunchKernelGGL((lloyd_valu_kernel<M, kAssign>), grid, block, p.lds_bytes, s, a.X,
                           a.n, a.C, a.K, a.labels, a.labels_in, a.min_d2, a.part_sums,
                           a.part_counts, a.ctl, a.t, a.fixed);
        break;
    case kAssignAccum:
        hipLaunchKernelGGL((lloyd_valu_kernel<M, kAssignAccum>), grid, block, p.lds_bytes, s,
                           a.X, a.n, a.C, a.K, a.labels, a.labels_in, a.min_d2, a.part_sums,
                           a.part_counts, a.ctl, a.t, a.fixed);
        break;
    case kAccumLabels:
        hipLaunchKernelGGL((lloyd_valu_kernel<M, kAccumLabels>), grid, block, p.lds_bytes, s,
                           a.X, a.n, a.C, a.K, a.labels, a.labels_in, a.min_d2, a.part_sums,
                           a.part_counts, a.ctl, a.t, a.fixed);
        break;
    }
    return hipGetLastError();
}

using LaunchFn = hipError_t (*)(const StepArgs &, Mode, const AccumPlan &, hipStream_t);

template <int... Ms>
struct LaunchTable {
    static constexpr LaunchFn fns[sizeof...(Ms)] = {&launch_m<Ms + 1>...};
};

template <int... Is>
constexpr auto make_table(std::integer_sequence<int, Is...>)
{
    return LaunchTable<Is...>{};
}

}  // namespace

AccumPlan plan_valu(int64_t n, int M, int K, Mode mode)
{
    AccumPlan p{};
    const size_t tile = (size_t)kWave * M * 4;
    const size_t per_wave = tile + (mode == kAssign ? 0 : (size_t)K * M * 8 + (size_t)K * 4);
    int W = 4;
    while (W > 1 && (size_t)W * per_wave > (size_t)kMaxLds) W /= 2;
    const int64_t nq = (n + kWave - 1) / kWave;
    int64_t groups = (nq + W - 1) / W;
    const int64_t cap = mode == kAssign ? 8192 : kMaxGroups;
    if (groups > cap) groups = cap;
    p.waves = W;
    p.groups = (int)groups;
    p.lds_bytes = (size_t)W * per_wave;
    return p;
}

hipError_t launch_valu(const StepArgs &a, Mode mode, const AccumPlan &plan, hipStream_t s)
{
    static constexpr auto table = make_table(std::make_integer_sequence<int, kMaxM>{});
    if (a.M < 1 || a.M > kMaxM) return hipErrorInvalidValue;
    return decltype(table)::fns[a.M - 1](a, mode, plan, s);
}

}  // namespace lloyd
