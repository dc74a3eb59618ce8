// Fused assign + accumulate with one object per lane, the distances in the
// direct form on the vector ALU (small K, or on request).
//
// One wavefront owns a 64-object tile at a time (object l of the tile in lane
// l) and walks its tiles with a fixed stride, so every sum below is formed in an
// order that depends only on the problem shape:
//   1. the tile's 64*M fp32 values are streamed from HBM with 16-byte loads into
//      the wave's LDS slot (the loads of the tile two strides ahead are issued
//      before the current tile is processed);
//   2. assignment (Algorithm 1 steps 2/4, Eq. (2)): each lane reads its own
//      object's M features into registers and evaluates |x - c|^2 for every
//      centre on the vector ALU (centres are wave-uniform and come through
//      scalar loads); its fp32 error is at most gamma_{M+1} |x - c|^2, so the
//      two best distances are called in fp32 only when their gap exceeds
//      4 gamma_{M+2} of the second; a lane whose call is too close recomputes
//      all K distances in fp64 in the oracle's operation order and takes the
//      lowest-index minimum, so the label is the exact-arithmetic argmin;
//   3. accumulation (the numerator and denominator of Eq. (1)) into the wave's
//      private fp64 slabs (accumulate_tile), no barriers;
//   4. at the end the workgroup adds its waves' slabs in a fixed order and
//      writes one fp64 partial per (cluster, feature) plus one count per
//      cluster; a second launch forms the centres (lloyd_centres.hip).
//
// The same kernel also assigns by the L1 distance (the other metric the paper
// allows in place of Eq. (2)) fused with the same accumulation: the distance
// is sum_j |x_j - c_j| in fp32, features ascending, within gamma_M of the
// exact one, so a label is accepted when the two best differ by more than
// 2.02 gamma_M (d1 + d2); otherwise all K distances are formed again in fp64
// in the oracle's order (e = x_j - c_j, d = d + |e|) and the lowest-index
// minimum is taken.
#include "lloyd.h"
#include "lloyd_device.h"
#include "lloyd_l1.h"

#include <math.h>

#include <array>
#include <type_traits>
#include <utility>

#include "lloyd_parts.h"

namespace lloyd {

namespace {

constexpr int kMaxWaves = 12;
constexpr int kMinWavesPerSimd = 3;   // caps registers at 168 per lane
constexpr int kSqEuclid = 0;          // metrics of the assignment
constexpr int kL1 = 1;
// Where the fused L1 form is used: at least this many waves per workgroup
// (fewer leave SIMDs idle) and at most this many centres. Its distance loop
// (centres as scalar operands, three waves per SIMD) costs more per centre
// than the L1 kernel's (centres broadcast from LDS, four waves per SIMD); the
// fused form saves the accumulate launch's second read of X. Measured at
// M = 25: K = 16, n = 2e6: 75.2 us per L1 iteration against 103.4 for the
// two-launch form; K = 64, n = 2e7: 2,110 against 1,954.
constexpr int kL1FusedMinWaves = 8;
constexpr int kL1FusedMaxK = 32;

// Per-wave tile slot: the 64 objects plus slack.
__host__ __device__ inline size_t lane_tile_bytes(int M)
{
    return (size_t)((kWave * M + (M > 4 ? M : 4) + 3) / 4 * 4) * 4;
}

// Objects per accumulation step: the most the lanes allow (pa = 0) or one (pa = 1).
[[maybe_unused]] __host__ __device__ inline int lane_acc_p(int M, int pa)
{
    if (pa == 1) return 1;
    const int lw = (M + 1 <= 2) ? 2 : (M + 1 <= 4) ? 4 : (M + 1 <= 8) ? 8
                 : (M + 1 <= 16) ? 16 : (M + 1 <= 32) ? 32 : 64;
    return kWave / lw;
}

// LDS carve-up: [W tile slots] [W x 64 ints of slab offsets] [W x P slabs].
__host__ __device__ inline size_t lane_slab_off(int M, int W)
{
    return (size_t)W * (lane_tile_bytes(M) + kWave * 4);
}

// L1 label of one object in fp64, the oracle's operation order, lowest index
// on ties (a NaN distance never wins: such an object keeps label 0)
template <int M>
__device__ inline int argmin_l1_fp64(const float *xs, const float *__restrict__ C, int K,
                                     double &bd)
{
    bd = INFINITY;
    int lab = 0;
    for (int k = 0; k < K; ++k) {
        const float *c = C + (int64_t)k * M;
        double d = 0.0;
        for (int j = 0; j < M; ++j) {
            const double e = (double)xs[j] - (double)c[j];
            d = d + fabs(e);
        }
        if (d < bd) {
            bd = d;
            lab = k;
        }
    }
    return lab;
}

template <int M, int MODE, int PA, int METRIC>
__global__ void __launch_bounds__(kMaxWaves * kWave, kMinWavesPerSimd)
lloyd_lane_kernel(const float *__restrict__ X, int64_t n, const float *__restrict__ C, int K,
                  int32_t *__restrict__ labels, const int32_t *__restrict__ labels_in,
                  float *__restrict__ min_d2, double *__restrict__ part_sums,
                  int32_t *__restrict__ part_counts, Ctl *__restrict__ ctl, int t, int fixed,
                  int force64)
{
    using G = TileGeom<M>;
    constexpr int V = G::kVecPerLane;
    constexpr int kP = WaveAcc<M, PA>::P;
    extern __shared__ __align__(16) unsigned char smem[];
    const int W = blockDim.x / kWave;
    const int wave = threadIdx.x / kWave;
    const int lane = threadIdx.x % kWave;

    if (MODE == kAssignAccum && stop_before(ctl, t, fixed)) return;
    if (MODE == kAccumLabels && stop_after_assign(ctl, fixed)) return;

    float *tile = reinterpret_cast<float *>(smem) + wave * G::kSlot;
    int32_t *offs = reinterpret_cast<int32_t *>(smem + (size_t)W * G::kSlot * 4) + wave * kWave;
    double *slabs_all = reinterpret_cast<double *>(smem + lane_slab_off(M, W));
    double *slabs = slabs_all + (size_t)wave * kP * K * (M + 1);

    // Full tiles (all 64 objects present) are streamed in the main loop; the
    // last, partial tile (if n is not a multiple of 64) is handled after it.
    // Wave w of workgroup b takes tiles w*G + b, then every G*W-th: the
    // waves with one tile more than the others are then waves 0, 1, ... of
    // every workgroup, which sit on different SIMDs, rather than every wave
    // of the first workgroups.
    const int64_t nfull = n / kWave;
    const int64_t stride = (int64_t)gridDim.x * W;
    const int64_t q0 = (int64_t)wave * gridDim.x + blockIdx.x;

    float4 buf[2][V];   // register buffers (two tiles ahead), selected by compile-time index
    if (q0 < nfull) load_tile<M>(X, q0, lane, buf[0]);
    if (q0 + stride < nfull) load_tile<M>(X, q0 + stride, lane, buf[1]);

    for (int i = lane; i < G::kSlot - kWave * M; i += kWave) tile[kWave * M + i] = 0.f;
    if (MODE != kAssign) {
        for (int i = lane; i < kP * K * (M + 1); i += kWave) slabs[i] = 0.0;
    }

    // call thresholds in fp32 (see the header comment)
    constexpr float kTau = 4.0f * (float)(M + 2) * 5.9604645e-8f;
    constexpr double kU = 5.9604644775390625e-8;
    constexpr float kTauL1 = (float)(2.02 * (M * kU / (1.0 - M * kU)));
    int nfallback = 0;

    // A tile's labels (and distances) are stored at the start of the next step,
    // after that step's tile has arrived and before its successor's loads are
    // issued: the wait for those loads then never waits on a store issued
    // just before it.
    int64_t pend_i = -1;      // this lane's object whose label waits to be stored
    int pend_lab = 0;
    float pend_d2 = 0.f;
    auto flush = [&]() {
        if (pend_i >= 0) {
            labels[pend_i] = pend_lab;
            if (MODE == kAssign && min_d2 != nullptr) min_d2[pend_i] = pend_d2;
        }
    };

    // full: a tile of the main loop (all 64 objects present; the loads of the
    // tile two strides ahead are issued here) rather than the partial last one
    auto step = [&](int64_t qq_, auto bi, auto full) {
        constexpr bool kFullTile = decltype(full)::value;
        float4 (&bb)[V] = buf[decltype(bi)::value];
        store_tile<M>(tile, lane, bb);
        __builtin_amdgcn_wave_barrier();
        if (MODE != kAccumLabels) flush();
        if (kFullTile && qq_ + 2 * stride < nfull) load_tile<M>(X, qq_ + 2 * stride, lane, bb);

        const int64_t i = qq_ * kWave + lane;
        const bool valid = kFullTile || i < n;
        int lab;
        if (MODE == kAccumLabels) {
            lab = valid ? labels_in[i] : -1;
            if (lab < 0 || lab >= K) lab = -1;
        } else {
            float b1 = INFINITY, b2 = INFINITY;
            lab = 0;
            float x[M];
#pragma unroll
            for (int j = 0; j < M; ++j) x[j] = tile[lane * M + j];
            for (int k = 0; k < K; ++k) {
                float d = 0.f;
#pragma unroll
                for (int j = 0; j < M; ++j) {
                    const float e = x[j] - C[k * M + j];
                    if constexpr (METRIC == kL1) d = d + fabsf(e);
                    else d = __builtin_fmaf(e, e, d);
                }
                if constexpr (METRIC == kL1) {
                    // a NaN distance changes neither
                    if (d < b1) {
                        b2 = b1;
                        b1 = d;
                        lab = k;
                    } else if (d < b2) {
                        b2 = d;
                    }
                } else {
                    // top-2: with b1 <= b2, the new second-best is the median
                    // of (b1, b2, d) and the new best is min(b1, d)
                    const bool lt = d < b1;
                    b2 = __builtin_amdgcn_fmed3f(b1, b2, d);
                    b1 = lt ? d : b1;
                    lab = lt ? k : lab;
                }
            }
            bool ok;
            if constexpr (METRIC == kL1)
                // every fp32 distance overflowed or is NaN (b1 never set): the
                // fp64 distances may still tell the centres apart
                ok = !force64 && b1 < INFINITY && (b2 == INFINITY || b2 - b1 > kTauL1 * (b1 + b2));
            else
                ok = !force64 && ((K == 1) || ((b2 - b1) > kTau * b2 && b2 >= 1e-30f));
            float dmin = b1;
            if (valid && !ok) {
                double bd;
                if constexpr (METRIC == kL1) lab = argmin_l1_fp64<M>(X + i * M, C, K, bd);
                else lab = argmin_fp64<M>(X + i * M, C, K, bd);
                dmin = (float)bd;
            }
            if (ctl != nullptr) nfallback += __popcll(__ballot(valid && !ok));
            pend_i = valid ? i : -1;
            pend_lab = lab;
            pend_d2 = dmin;
            if (!valid) lab = -1;
        }

        if (MODE != kAssign) {
            // (labels read back may be out of range even in a full tile)
            accumulate_tile<M, PA, kFullTile && MODE != kAccumLabels>(lab, tile, offs, slabs, K,
                                                                     lane);
        }
    };

    for (int64_t q = q0; q < nfull; q += 2 * stride) {
        step(q, std::integral_constant<int, 0>{}, std::true_type{});
        if (q + stride < nfull) step(q + stride, std::integral_constant<int, 1>{}, std::true_type{});
    }
    if (nfull * kWave < n && nfull >= q0 && (nfull - q0) % stride == 0) {
        load_tail_tile<M>(X, n, nfull, lane, buf[0]);
        step(nfull, std::integral_constant<int, 0>{}, std::false_type{});
    }
    if (MODE != kAccumLabels) flush();

    if (ctl != nullptr && lane == 0 && nfallback > 0) atomicAdd(&ctl->fallbacks, nfallback);

    if (MODE != kAssign) {
        __syncthreads();
        write_wave_partials<M, PA>(slabs_all, W, K, part_sums + (int64_t)blockIdx.x * K * M,
                                   part_counts + blockIdx.x, gridDim.x);
    }
}

template <int M>
hipError_t launch_m(const StepArgs &a, Mode mode, const AccumPlan &p, hipStream_t s)
{
    const dim3 grid(p.groups), block(p.waves * kWave);
#define LLOYD_LANE_LAUNCH(MD, PA)                                                              \
    do {                                                                                       \
        auto kern = lloyd_lane_kernel<M, MD, PA, kSqEuclid>;                                   \
        static const size_t st = static_lds_bytes(reinterpret_cast<const void *>(kern));       \
        if (st > (size_t)kMaxLds || st + p.lds_bytes > (size_t)kMaxLds)                        \
            return hipErrorInvalidConfiguration;                                               \
        hipExtLaunchKernelGGL(kern, grid, block, p.lds_bytes, s, a.ev_start, a.ev_stop, 0,     \
                              a.X, a.n, a.C, a.K, a.labels, a.labels_in, a.min_d2,            \
                              a.part_sums, a.part_counts, a.ctl, a.t, a.fixed, a.force64);    \
    } while (0)
    const bool one = p.accum == 1;
    switch (mode) {
    case kAssign: LLOYD_LANE_LAUNCH(kAssign, 0); break;
    case kAssignAccum:
        if (one) LLOYD_LANE_LAUNCH(kAssignAccum, 1);
        else LLOYD_LANE_LAUNCH(kAssignAccum, 0);
        break;
    case kAccumLabels:
        if (one) LLOYD_LANE_LAUNCH(kAccumLabels, 1);
        else LLOYD_LANE_LAUNCH(kAccumLabels, 0);
        break;
    }
#undef LLOYD_LANE_LAUNCH
    return hipGetLastError();
}

// the fused L1 assign + accumulate launch
template <int M>
hipError_t launch_l1_m(const StepArgs &a, const AccumPlan &p, hipStream_t s)
{
    auto kern = p.accum == 1 ? lloyd_lane_kernel<M, kAssignAccum, 1, kL1>
                             : lloyd_lane_kernel<M, kAssignAccum, 0, kL1>;
    static const size_t st0 =
        static_lds_bytes(reinterpret_cast<const void *>(lloyd_lane_kernel<M, kAssignAccum, 0, kL1>));
    static const size_t st1 =
        static_lds_bytes(reinterpret_cast<const void *>(lloyd_lane_kernel<M, kAssignAccum, 1, kL1>));
    const size_t st = p.accum == 1 ? st1 : st0;
    if (st > (size_t)kMaxLds || st + p.lds_bytes > (size_t)kMaxLds)
        return hipErrorInvalidConfiguration;
    hipExtLaunchKernelGGL(kern, dim3(p.groups), dim3(p.waves * kWave), p.lds_bytes, s, a.ev_start,
                          a.ev_stop, 0, a.X, a.n, a.C, a.K, a.labels, a.labels_in, a.min_d2,
                          a.part_sums, a.part_counts, a.ctl, a.t, a.fixed, a.force64);
    return hipGetLastError();
}

using LaunchFn = hipError_t (*)(const StepArgs &, Mode, const AccumPlan &, hipStream_t);
using LaunchL1Fn = hipError_t (*)(const StepArgs &, const AccumPlan &, hipStream_t);

// This translation unit instantiates the kernels for the feature counts of
// one part of [1, kMaxM] (the build compiles it once per part, in parallel).
constexpr int kPartLo = LLOYD_PART * kMaxM / LLOYD_PARTS + 1;
constexpr int kPartN = kMaxM / LLOYD_PARTS;

template <int M>
constexpr LaunchFn entry()
{
#ifdef LLOYD_ONLY_M
    if constexpr (M != LLOYD_ONLY_M) return nullptr;
    else
#endif
    return &launch_m<M>;
}

template <int... Is>
constexpr auto make_table(std::integer_sequence<int, Is...>)
{
    return std::array<LaunchFn, sizeof...(Is)>{entry<kPartLo + Is>()...};
}

template <int M>
constexpr LaunchL1Fn entry_l1()
{
#ifdef LLOYD_ONLY_M
    if constexpr (M != LLOYD_ONLY_M) return nullptr;
    else
#endif
    return &launch_l1_m<M>;
}

template <int... Is>
constexpr auto make_l1_table(std::integer_sequence<int, Is...>)
{
    return std::array<LaunchL1Fn, sizeof...(Is)>{entry_l1<kPartLo + Is>()...};
}

}  // namespace

hipError_t LLOYD_PART_FN(launch_lane_part)(const StepArgs &a, Mode mode, const AccumPlan &plan,
                                           hipStream_t s)
{
    static constexpr auto table = make_table(std::make_integer_sequence<int, kPartN>{});
    if (a.M < kPartLo || a.M >= kPartLo + kPartN) return hipErrorInvalidValue;
    const LaunchFn fn = table[a.M - kPartLo];
    return fn ? fn(a, mode, plan, s) : hipErrorInvalidValue;
}

hipError_t LLOYD_PART_FN(launch_lane_l1_part)(const StepArgs &a, const AccumPlan &plan,
                                              hipStream_t s)
{
    static constexpr auto table = make_l1_table(std::make_integer_sequence<int, kPartN>{});
    if (a.M < kPartLo || a.M >= kPartLo + kPartN) return hipErrorInvalidValue;
    const LaunchL1Fn fn = table[a.M - kPartLo];
    return fn ? fn(a, plan, s) : hipErrorInvalidValue;
}

#if LLOYD_PART == 0
AccumPlan plan_lane(int64_t n, int M, int K, Mode mode)
{
    AccumPlan p{};
    p.path = kPathValu;
    auto bytes = [&](int W, int pa) {
        size_t b = lane_slab_off(M, W);
        if (mode != kAssign) b += (size_t)W * lane_acc_p(M, pa) * K * (M + 1) * 8;
        return b;
    };
    auto most_waves = [&](int pa) {
        int w = kMaxWaves;
        while (w > 0 && bytes(w, pa) > (size_t)kMaxLds) --w;
        return w;
    };
    // slabs with the most objects per step unless one object per step leaves
    // more waves
    int pa = 0, W = most_waves(0);
    if (mode != kAssign && most_waves(1) > W) {
        pa = 1;
        W = most_waves(1);
    }
    const int64_t nq = (n + kWave - 1) / kWave;
    while (W > 1 && W / 2 >= nq) W /= 2;
    int64_t groups = (nq + W - 1) / W;
    if (groups > kCUs) groups = kCUs;       // one persistent workgroup per compute unit
    p.waves = W;
    p.groups = (int)groups;
    p.accum = pa;
    p.lds_bytes = bytes(W, pa);
    return p;
}

AccumPlan plan_lane_l1(int64_t n, int M, int K)
{
    AccumPlan p = plan_lane(n, M, K, kAssignAccum);
    if (K > kL1FusedMaxK || (p.waves < kL1FusedMinWaves && p.groups >= kCUs))
        p.waves = 0;   // not used
    return p;
}

hipError_t launch_lane_l1(const StepArgs &a, const AccumPlan &plan, hipStream_t s)
{
    if (a.M < 1 || a.M > kMaxM || plan.waves < 1 || plan.groups < 1) return hipErrorInvalidValue;
    switch ((a.M - 1) / (kMaxM / LLOYD_PARTS)) {
#define LLOYD_CASE(P) case P: return launch_lane_l1_part_##P(a, plan, s);
        LLOYD_PART_CASES
#undef LLOYD_CASE
    }
    return hipErrorInvalidValue;
}

hipError_t launch_lane(const StepArgs &a, Mode mode, const AccumPlan &plan, hipStream_t s)
{
    if (a.M < 1 || a.M > kMaxM) return hipErrorInvalidValue;
    switch ((a.M - 1) / (kMaxM / LLOYD_PARTS)) {
#define LLOYD_CASE(P) case P: return launch_lane_part_##P(a, mode, plan, s);
        LLOYD_PART_CASES
#undef LLOYD_CASE
    }
    return hipErrorInvalidValue;
}
#endif

}  // namespace lloyd
