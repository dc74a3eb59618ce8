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
//      a ballot gives the lanes holding its members; lanes then act as (slot,
//      feature) pairs and add the members' features (read back from the LDS
//      tile) into fp64 running sums, and the sum is added to the wave's private
//      fp64 slab (wave_accumulate). No atomics are involved.
//   4. at the end the workgroup adds its waves' slabs in wave order and writes
//      one fp64 partial per (cluster, feature) plus one count per cluster.
#include "lloyd.h"
#include "lloyd_device.h"
#include "lloyd_reduce.h"

#include <math.h>

#include <array>
#include <utility>

#include "lloyd_parts.h"

namespace lloyd {

namespace {

template <int M, int MODE>
__global__ void __launch_bounds__(1024)
lloyd_valu_kernel(const float *__restrict__ X, int64_t n, const float *__restrict__ C, int K,
                  int32_t *__restrict__ labels, const int32_t *__restrict__ labels_in,
                  float *__restrict__ min_d2, double *__restrict__ part_sums,
                  int32_t *__restrict__ part_counts, Ctl *__restrict__ ctl, int t, int fixed,
                  TreeArgs tree)
{
    using G = TileGeom<M>;
    extern __shared__ __align__(16) unsigned char smem[];
    const int W = blockDim.x / kWave;
    const int wave = threadIdx.x / kWave;
    const int lane = threadIdx.x % kWave;

    if (MODE == kAssignAccum && stop_before(ctl, t, fixed)) return;

    using S = Slots<M>;
    constexpr int MW = S::MW;
    // LDS: [ones: 68 floats] [W tiles of kTileFloats] [W slabs of K*(M+1) fp64]
    float *ones = reinterpret_cast<float *>(smem);
    float *tile = ones + 68 + wave * S::kTileFloats;
    const size_t slab_off = (68 + (size_t)W * S::kTileFloats) * 4;
    double *slab = reinterpret_cast<double *>(smem + slab_off) + (size_t)wave * K * MW;
    for (int i = lane; i < S::kTileFloats - kWave * M; i += kWave) tile[kWave * M + i] = 0.f;
    if (MODE != kAssign) {
        for (int i = lane; i < K * MW; i += kWave) slab[i] = 0.0;
        if (wave == 0)
            for (int i = lane; i < 68; i += kWave) ones[i] = i < kWave ? 1.f : 0.f;
        __syncthreads();
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

        if (MODE != kAssign) wave_accumulate<M>(lab, tile, ones, slab, K, lane);
        __builtin_amdgcn_wave_barrier();
    }

    if (ctl != nullptr && lane == 0 && nfallback > 0) atomicAdd(&ctl->fallbacks, nfallback);

    if (MODE != kAssign) {
        __syncthreads();
        const double *slabs = reinterpret_cast<const double *>(smem + slab_off);
        double *out = part_sums + (int64_t)blockIdx.x * K * M;
        for (int e = threadIdx.x; e < K * M; e += blockDim.x) {
            const int k = e / M, j = e - (e / M) * M;
            double s = slabs[k * MW + j];
            for (int w = 1; w < W; ++w) s = s + slabs[(size_t)w * K * MW + k * MW + j];
            out[e] = s;
        }
        for (int k = threadIdx.x; k < K; k += blockDim.x) {
            double c = 0.0;
            for (int w = 0; w < W; ++w) c = c + slabs[(size_t)w * K * MW + k * MW + M];
            part_counts[(int64_t)blockIdx.x * K + k] = (int32_t)c;
        }
        tree_finalize(tree, reinterpret_cast<uint32_t *>(const_cast<double *>(slabs)));
    }
}

TreeArgs tree_args(const StepArgs &a, int groups)
{
    TreeArgs r{};
    r.part_sums = a.part_sums;
    r.part_counts = a.part_counts;
    r.grp_sums = a.grp_sums;
    r.grp_counts = a.grp_counts;
    r.tickets = a.ctl != nullptr ? a.ctl->tickets : nullptr;
    r.G = groups;
    r.K = a.K;
    r.M = a.M;
    r.prev = a.C;
    r.centers = a.centers_out;
    r.counts = a.counts_out;
    r.ctl = a.ctl;
    r.t = a.t;
    r.compare = a.compare;
    return r;
}

template <int M>
hipError_t launch_m(const StepArgs &a, Mode mode, const AccumPlan &p, hipStream_t s)
{
    const dim3 grid(p.groups), block(p.waves * kWave);
    const TreeArgs tr = tree_args(a, p.groups);
#define LLOYD_VALU_LAUNCH(MD)                                                                  \
    hipLaunchKernelGGL((lloyd_valu_kernel<M, MD>), grid, block, p.lds_bytes, s, a.X, a.n, a.C,  \
                       a.K, a.labels, a.labels_in, a.min_d2, a.part_sums, a.part_counts, a.ctl, \
                       a.t, a.fixed, tr)
    switch (mode) {
    case kAssign: LLOYD_VALU_LAUNCH(kAssign); break;
    case kAssignAccum: LLOYD_VALU_LAUNCH(kAssignAccum); break;
    case kAccumLabels: LLOYD_VALU_LAUNCH(kAccumLabels); break;
    }
#undef LLOYD_VALU_LAUNCH
    return hipGetLastError();
}

using LaunchFn = hipError_t (*)(const StepArgs &, Mode, const AccumPlan &, hipStream_t);

// This translation unit instantiates the kernels for the feature counts of
// one part of [1, kMaxM] (the build compiles it once per part, in parallel).
constexpr int kPartLo = LLOYD_PART * kMaxM / LLOYD_PARTS + 1;
constexpr int kPartN = kMaxM / LLOYD_PARTS;

template <int... Is>
constexpr auto make_table(std::integer_sequence<int, Is...>)
{
    return std::array<LaunchFn, sizeof...(Is)>{&launch_m<kPartLo + Is>...};
}

}  // namespace

hipError_t LLOYD_PART_FN(launch_valu_part)(const StepArgs &a, Mode mode, const AccumPlan &plan,
                                           hipStream_t s)
{
    static constexpr auto table = make_table(std::make_integer_sequence<int, kPartN>{});
    if (a.M < kPartLo || a.M >= kPartLo + kPartN) return hipErrorInvalidValue;
    return table[a.M - kPartLo](a, mode, plan, s);
}

#if LLOYD_PART == 0
AccumPlan plan_valu(int64_t n, int M, int K, Mode mode)
{
    AccumPlan p{};
    p.path = kPathValu;
    const size_t tile = (size_t)((kWave * M + (M > 4 ? M : 4) + 3) / 4 * 4) * 4;
    const size_t per_wave =
        tile + (mode == kAssign ? 0 : (size_t)K * (M + 1) * 8);
    int W = 16;
    while (W > 1 && 68 * 4 + (size_t)W * per_wave > (size_t)kMaxLds) W -= (W > 8 ? 1 : W / 2);
    const int64_t nq = (n + kWave - 1) / kWave;
    while (W > 1 && W / 2 >= nq) W /= 2;
    int64_t groups = (nq + W - 1) / W;
    if (groups > kCUs) groups = kCUs;       // one persistent workgroup per compute unit
    p.waves = W;
    p.groups = (int)groups;
    p.accum = 1;
    p.lds_bytes = 68 * 4 + (size_t)W * per_wave;
    return p;
}

hipError_t launch_valu(const StepArgs &a, Mode mode, const AccumPlan &plan, hipStream_t s)
{
    if (a.M < 1 || a.M > kMaxM) return hipErrorInvalidValue;
    switch ((a.M - 1) / (kMaxM / LLOYD_PARTS)) {
#define LLOYD_CASE(P) case P: return launch_valu_part_##P(a, mode, plan, s);
        LLOYD_PART_CASES
#undef LLOYD_CASE
    }
    return hipErrorInvalidValue;
}
#endif

}  // namespace lloyd
