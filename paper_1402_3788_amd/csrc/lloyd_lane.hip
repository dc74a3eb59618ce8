// Fused assign + accumulate with one object per lane (small K).
//
// One wavefront owns a 64-object tile at a time (object l of the tile in lane
// l) and walks its tiles with a fixed stride, so every sum below is formed in an
// order that depends only on the problem shape:
//   1. the tile's 64*M fp32 values are streamed from HBM with 16-byte loads into
//      the wave's LDS slot (the loads of the tile one or two strides ahead are
//      issued before the current tile is processed);
//   2. assignment (Algorithm 1 steps 2/4, Eq. (2)), in one of two forms:
//        DIST = kDistValu: each lane reads its own object's M features into
//          registers and evaluates the direct form |x - c|^2 on the vector
//          ALU (centres are wave-uniform and come through scalar loads); its
//          fp32 error is at most gamma_{M+1} |x - c|^2, so the two best
//          distances are called in fp32 only when their gap exceeds
//          4 gamma_{M+2} of the second;
//        DIST = kDistMfma: the expanded form score = |c|^2 - 2 x.c on the
//          bf16 matrix cores (v_mfma_f32_16x16x32_bf16) in split precision:
//          A = -2C for 16 centres by 32 features and B = 32 features of 16
//          objects (read from the tile), each split into bf16 hi and lo
//          parts rounded to nearest, three products per 16-object block
//          (lo(A) hi(B) + hi(A) lo(B) + hi(A) hi(B)) on top of |c|^2; A and
//          |c|^2 stay in registers for the whole launch (K <= 16). Each lane
//          ends with 4 scores of one object; they go back into the slot
//          (which is no longer needed) as one row of 16 scores per object, so
//          that each lane again scans the K scores of its own object with no
//          cross-lane merge. A score is within E (3|c|^2 + |x|^2) of the
//          exact one, E = 3.02 * 2^-16 + 1.03 gamma_98, so a label is
//          accepted only if the two best scores differ by more than 2.02 E
//          (3 max|c|^2 + |x|^2);
//      either way, a lane whose call is too close recomputes all K distances
//      in fp64 in the oracle's operation order and takes the lowest-index
//      minimum, so the label is the exact-arithmetic argmin;
//   3. accumulation (the numerator and denominator of Eq. (1)) into the wave's
//      private fp64 slabs (accumulate_tile), no barriers;
//   4. at the end the workgroup adds its waves' slabs in a fixed order and
//      writes one fp64 partial per (cluster, feature) plus one count per
//      cluster; a second launch forms the centres (lloyd_centres.hip).
#include "lloyd.h"
#include "lloyd_device.h"

#include <math.h>

#include <array>
#include <type_traits>
#include <utility>

#include "lloyd_parts.h"

namespace lloyd {

namespace {

typedef float f4v __attribute__((ext_vector_type(4)));

constexpr int kMaxWaves = 12;
constexpr int kMinWavesPerSimd = 3;   // caps registers at 168 per lane
constexpr int kDistValu = 0;
constexpr int kDistMfma = 1;
constexpr int kLaneMfmaMaxK = 16;     // four 4-centre operand columns
constexpr int kLaneMfmaMaxM = 27;

// LDS carve-up: [operand table] [W tile slots] [W x 64 ints of slab offsets]
// [W x P slabs]. The operand table (matrix-core form only) holds, for centre
// quad qq and lane group r = lane % 4, the row -2 c_{4qq+r, 0..M-1}, |c|^2,
// zero-padded to a multiple of 4 floats.
// Scores written back per object by the matrix-core form: 16 centre scores
// and the four partial |x|^2 of the lanes that held its features.
constexpr int kScoreRow = 20;

// Per-wave tile slot: the 64 objects plus slack; in the matrix-core form at
// least 64 score rows, which reuse the slot once the tile has been read.
__host__ __device__ inline size_t lane_tile_bytes(int M, bool mfma)
{
    const size_t tile = (size_t)((kWave * M + (M > 4 ? M : 4) + 3) / 4 * 4) * 4;
    const size_t scores = (size_t)kWave * kScoreRow * 4;
    return mfma && scores > tile ? scores : tile;
}

__host__ __device__ inline int lane_atab_row(int M) { return (M + 1 + 3) / 4 * 4; }

__host__ __device__ inline size_t lane_atab_bytes(int M, bool mfma)
{
    return mfma ? (size_t)(kLaneMfmaMaxK / 4) * 4 * lane_atab_row(M) * 4 : 0;
}

// Objects per accumulation step: the most the lanes allow (pa = 0) or one (pa = 1).
[[maybe_unused]] __host__ __device__ inline int lane_acc_p(int M, int pa)
{
    if (pa == 1) return 1;
    const int lw = (M + 1 <= 2) ? 2 : (M + 1 <= 4) ? 4 : (M + 1 <= 8) ? 8
                 : (M + 1 <= 16) ? 16 : (M + 1 <= 32) ? 32 : 64;
    return kWave / lw;
}

__host__ __device__ inline size_t lane_slab_off(int M, int W, bool mfma)
{
    return lane_atab_bytes(M, mfma) + (size_t)W * (lane_tile_bytes(M, mfma) + kWave * 4);
}

template <int M, int MODE, int PA, int DIST>
__global__ void __launch_bounds__(kMaxWaves * kWave, kMinWavesPerSimd)
lloyd_lane_kernel(const float *__restrict__ X, int64_t n, const float *__restrict__ C, int K,
                  int32_t *__restrict__ labels, const int32_t *__restrict__ labels_in,
                  float *__restrict__ min_d2, double *__restrict__ part_sums,
                  int32_t *__restrict__ part_counts, Ctl *__restrict__ ctl, int t, int fixed)
{
    using G = TileGeom<M>;
    constexpr int V = G::kVecPerLane;
    constexpr int kP = WaveAcc<M, PA>::P;
    constexpr bool kMfma = DIST == kDistMfma;
    constexpr int KQ = kMfma ? kLaneMfmaMaxK / 4 : 1;    // centre quads held in registers
    extern __shared__ __align__(16) unsigned char smem[];
    const int W = blockDim.x / kWave;
    const int wave = threadIdx.x / kWave;
    const int lane = threadIdx.x % kWave;

    if (MODE == kAssignAccum && stop_before(ctl, t, fixed)) return;

    constexpr int FP = (M + 1 + 3) / 4 * 4;               // operand table row (lane_atab_row)
    constexpr size_t kAtab = kMfma ? (size_t)KQ * 4 * FP * 4 : 0;   // lane_atab_bytes
    float *atab = reinterpret_cast<float *>(smem);
    // tile slot in floats (lane_tile_bytes / 4)
    constexpr int kSlotL = kMfma && kWave * kScoreRow > G::kSlot ? kWave * kScoreRow : G::kSlot;
    float *tile = reinterpret_cast<float *>(smem + kAtab) + wave * kSlotL;
    int32_t *offs = reinterpret_cast<int32_t *>(smem + kAtab + (size_t)W * kSlotL * 4) + wave * kWave;
    double *slabs_all = reinterpret_cast<double *>(smem + lane_slab_off(M, W, kMfma));
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

    // tiles in flight per wave: two ahead, or one where the matrix-core
    // operands take the registers
    constexpr int kDepth = kMfma ? 1 : 2;
    float4 buf[2][V];   // register buffers, selected by compile-time index
    if (q0 < nfull) load_tile<M>(X, q0, lane, buf[0]);
    if (kDepth == 2 && q0 + stride < nfull) load_tile<M>(X, q0 + stride, lane, buf[1]);

    for (int i = lane; i < G::kSlot - kWave * M; i += kWave) tile[kWave * M + i] = 0.f;
    if (MODE != kAssign) {
        for (int i = lane; i < kP * K * (M + 1); i += kWave) slabs[i] = 0.0;
    }

    // Matrix-core operand table (see lane_atab_bytes): -2c (exact), then |c|^2
    // in fp32 with the features in order (+inf for centres past K, so they
    // never win), then zeros; and cmax = the largest |c|^2.
    float cmax = 0.f;
    if (kMfma && MODE != kAccumLabels) {
        if (threadIdx.x < KQ * 4) {
            const int k = threadIdx.x;                 // row qq * 4 + r holds centre k
            float *row = atab + k * FP;
            float nk = 0.f;
            for (int f = 0; f < M; ++f) {
                const float c = k < K ? C[(int64_t)k * M + f] : 0.f;
                row[f] = -2.0f * c;
                nk = __builtin_fmaf(c, c, nk);
            }
            row[M] = k < K ? nk : INFINITY;
            for (int f = M + 1; f < FP; ++f) row[f] = 0.f;
        }
        __syncthreads();
        for (int k = 0; k < K; ++k) cmax = fmaxf(cmax, atab[k * FP + M]);
    }
    // A operands of the bf16 products for the whole launch: lane l holds
    // features 8(l/16) .. 8(l/16)+7 of centre l % 16 (-2c, zero past M),
    // split into bf16 hi and lo, and the |c|^2 seeds of centres
    // 4(l/16) .. 4(l/16)+3 (the rows of the result it holds).
    uint32_t ah[4], al[4];
    f4v cseed;
    {
        float a[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int f = 8 * (lane / 16) + e;
            a[e] = (kMfma && MODE != kAccumLabels && f < M) ? atab[(lane % 16) * FP + f] : 0.f;
        }
        split_bf16x8(a, ah, al);
#pragma unroll
        for (int r = 0; r < 4; ++r)
            cseed[r] = (kMfma && MODE != kAccumLabels) ? atab[(4 * (lane / 16) + r) * FP + M] : 0.f;
    }

    // call thresholds (see the header comment): the direct form in fp32; the
    // split-precision scores, within E (|x|^2 + 3|c|^2) of the exact ones with
    // E = 3.02 * 2^-16 + 1.03 gamma_98 (the bf16 split of both operands, the
    // fp32 sums of 96 exact products and |c|^2, and |c|^2 itself in fp32)
    constexpr float kTau = 4.0f * (float)(M + 2) * 5.9604645e-8f;
    constexpr float kE1 = 3.02f * 1.5258789e-05f + 1.03f * 98.0f * 5.9604645e-8f;
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
    // tile kDepth strides ahead are issued here) rather than the partial last one
    auto step = [&](int64_t qq_, auto bi, auto full) {
        constexpr bool kFullTile = decltype(full)::value;
        float4 (&bb)[V] = buf[decltype(bi)::value];
        store_tile<M>(tile, lane, bb);
        __builtin_amdgcn_wave_barrier();
        if (MODE != kAccumLabels) flush();
        if (kFullTile && qq_ + kDepth * stride < nfull)
            load_tile<M>(X, qq_ + kDepth * stride, lane, bb);

        const int64_t i = qq_ * kWave + lane;
        const bool valid = kFullTile || i < n;
        // the accumulation's feature reads go out now and wait in registers
        // (matrix-core form, where the registers are there)
        constexpr bool kEarly = kMfma && WaveAcc<M, PA>::kSteps <= 32;
        static_assert(!kMfma || MODE != kAssignAccum || kEarly,
                      "the matrix-core form reads the accumulation values before the scores overwrite the tile");
        AccFetch<M, PA> af;
        if (MODE != kAssign && kEarly) accumulate_fetch<M, PA>(tile, lane, af);
        int lab;
        if (MODE == kAccumLabels) {
            lab = valid ? labels_in[i] : -1;
            if (lab < 0 || lab >= K) lab = -1;
        } else {
            float b1 = INFINITY, b2 = INFINITY;
            lab = 0;
            bool ok;
            if constexpr (kMfma) {
                // Split-precision products on the bf16 matrix cores
                // (v_mfma_f32_16x16x32_bf16) for four blocks of 16 objects:
                // A = -2C (16 centres x 32 features, in ah / al), B = features
                // 8(l/16) .. 8(l/16)+7 of object 16b + l%16 read from the tile
                // (zero past M; the reads stay inside the wave's slot) and split
                // likewise; per block lo(A) hi(B) + hi(A) lo(B) + hi(A) hi(B)
                // on top of |c|^2. Lane l ends with the scores of centres
                // 4(l/16) .. 4(l/16)+3 for object 16b + l%16 of block b; it
                // also sums the squares of the features it read (a quarter
                // of |x|^2). The four blocks are four independent chains.
                const int g = lane / 16, o16 = lane % 16;
                f4v d[4];
                float xp[4];
                uint32_t bh[4][4], bl[4][4];
#pragma unroll
                for (int b = 0; b < 4; ++b) {
                    const float *row = tile + (16 * b + o16) * M + 8 * g;
                    float v[8];
                    float acc = 0.f;
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        // every read is made (in range for every lane group
                        // where 24 + e < M), and the bits past M are masked
                        const bool always = 24 + e < M;
                        const uint32_t keep = (always || 8 * g + e < M) ? ~0u : 0u;
                        v[e] = __uint_as_float(__float_as_uint(row[e]) & keep);
                        acc = __builtin_fmaf(v[e], v[e], acc);
                    }
                    xp[b] = acc;
                    split_bf16x8(v, bh[b], bl[b]);
                }
#pragma unroll
                for (int b = 0; b < 4; ++b) d[b] = cseed;
#pragma unroll
                for (int b = 0; b < 4; ++b)
                    d[b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf8(al), as_bf8(bh[b]), d[b], 0, 0, 0);
#pragma unroll
                for (int b = 0; b < 4; ++b)
                    d[b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf8(ah), as_bf8(bl[b]), d[b], 0, 0, 0);
#pragma unroll
                for (int b = 0; b < 4; ++b)
                    d[b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf8(ah), as_bf8(bh[b]), d[b], 0, 0, 0);
                // every read of the tile (features above, accumulation values
                // before) precedes these writes in program order, and a wave's
                // LDS operations complete in order: the score rows may reuse
                // the slot. Row o: 16 scores, then the 4 partial |x|^2.
#pragma unroll
                for (int b = 0; b < 4; ++b) {
                    float *row = tile + (16 * b + o16) * kScoreRow;
                    *reinterpret_cast<f4v *>(row + 4 * g) = d[b];
                    row[16 + g] = xp[b];
                }
                __builtin_amdgcn_wave_barrier();
                f4v sc[4];
#pragma unroll
                for (int qq = 0; qq < 4; ++qq)
                    sc[qq] = *reinterpret_cast<const f4v *>(tile + lane * kScoreRow + 4 * qq);
                const f4v pp = *reinterpret_cast<const f4v *>(tile + lane * kScoreRow + 16);
                const float xsq = ((pp[0] + pp[1]) + pp[2]) + pp[3];
#pragma unroll
                for (int qq = 0; qq < 4; ++qq) {
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const float v = sc[qq][r];
                        const bool lt = v < b1;
                        b2 = __builtin_amdgcn_fmed3f(b1, b2, v);
                        b1 = lt ? v : b1;
                        lab = lt ? 4 * qq + r : lab;
                    }
                }
                const float thr = 2.02f * kE1 * (3.02f * cmax + 1.0001f * xsq) + 1e-30f;
                ok = (K == 1) || (b2 - b1 > thr);
            } else {
                float x[M];
#pragma unroll
                for (int j = 0; j < M; ++j) x[j] = tile[lane * M + j];
                for (int k = 0; k < K; ++k) {
                    float d = 0.f;
#pragma unroll
                    for (int j = 0; j < M; ++j) {
                        const float e = x[j] - C[k * M + j];
                        d = __builtin_fmaf(e, e, d);
                    }
                    // top-2: with b1 <= b2, the new second-best is the median of
                    // (b1, b2, d) and the new best is min(b1, d)
                    const bool lt = d < b1;
                    b2 = __builtin_amdgcn_fmed3f(b1, b2, d);
                    b1 = lt ? d : b1;
                    lab = lt ? k : lab;
                }
                ok = (K == 1) || ((b2 - b1) > kTau * b2 && b2 >= 1e-30f);
            }
            // the object's features from X: in the matrix-core form the slot
            // now holds scores (both uses are off the common path)
            float dmin = kMfma ? 0.f : b1;
            if (valid && !ok) {
                double bd;
                lab = argmin_fp64<M>(X + i * M, C, K, bd);
                dmin = (float)bd;
            } else if (kMfma && valid && MODE == kAssign && min_d2 != nullptr) {
                const float *xg = X + i * M;
                const float *c = C + (int64_t)lab * M;
                float d = 0.f;
#pragma unroll
                for (int j = 0; j < M; ++j) {
                    const float e = xg[j] - c[j];
                    d = __builtin_fmaf(e, e, d);
                }
                dmin = d;
            }
            if (ctl != nullptr) nfallback += __popcll(__ballot(valid && !ok));
            pend_i = valid ? i : -1;
            pend_lab = lab;
            pend_d2 = dmin;
            if (!valid) lab = -1;
        }

        if (MODE != kAssign) {
            // (labels read back may be out of range even in a full tile)
            if (kEarly) accumulate_commit<M, PA, kFullTile && MODE != kAccumLabels>(lab, af, offs, slabs, K, lane);
            else accumulate_tile<M, PA>(lab, tile, offs, slabs, K, lane);
        }
    };

    if (kDepth == 1) {
        for (int64_t q = q0; q < nfull; q += stride) step(q, std::integral_constant<int, 0>{}, std::true_type{});
    } else {
        for (int64_t q = q0; q < nfull; q += 2 * stride) {
            step(q, std::integral_constant<int, 0>{}, std::true_type{});
            if (q + stride < nfull) step(q + stride, std::integral_constant<int, 1>{}, std::true_type{});
        }
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
                                   part_counts + (int64_t)blockIdx.x * K);
    }
}

template <int M, int DIST>
hipError_t launch_m(const StepArgs &a, Mode mode, const AccumPlan &p, hipStream_t s)
{
    const dim3 grid(p.groups), block(p.waves * kWave);
#define LLOYD_LANE_LAUNCH(MD, PA)                                                              \
    do {                                                                                       \
        auto kern = lloyd_lane_kernel<M, MD, PA, DIST>;                                        \
        static const size_t st = static_lds_bytes(reinterpret_cast<const void *>(kern));       \
        if (st > (size_t)kMaxLds || st + p.lds_bytes > (size_t)kMaxLds)                        \
            return hipErrorInvalidConfiguration;                                               \
        hipLaunchKernelGGL(kern, grid, block, p.lds_bytes, s, a.X, a.n, a.C, a.K, a.labels,    \
                           a.labels_in, a.min_d2, a.part_sums, a.part_counts, a.ctl, a.t,      \
                           a.fixed);                                                           \
    } while (0)
    const bool one = p.accum == 1;
    switch (mode) {
    case kAssign: LLOYD_LANE_LAUNCH(kAssign, 0); break;
    case kAssignAccum:
        if constexpr (DIST == kDistMfma) {
            if (one) return hipErrorInvalidConfiguration;   // plan_lane never asks for it
            LLOYD_LANE_LAUNCH(kAssignAccum, 0);
        } else {
            if (one) LLOYD_LANE_LAUNCH(kAssignAccum, 1);
            else LLOYD_LANE_LAUNCH(kAssignAccum, 0);
        }
        break;
    case kAccumLabels:
        if (one) LLOYD_LANE_LAUNCH(kAccumLabels, 1);
        else LLOYD_LANE_LAUNCH(kAccumLabels, 0);
        break;
    }
#undef LLOYD_LANE_LAUNCH
    return hipGetLastError();
}

using LaunchFn = hipError_t (*)(const StepArgs &, Mode, const AccumPlan &, hipStream_t);

// This translation unit instantiates the kernels for the feature counts of
// one part of [1, kMaxM] (the build compiles it once per part, in parallel);
// the matrix-core form only up to kLaneMfmaMaxM features.
constexpr int kPartLo = LLOYD_PART * kMaxM / LLOYD_PARTS + 1;
constexpr int kPartN = kMaxM / LLOYD_PARTS;

template <int M>
constexpr LaunchFn mfma_entry()
{
    if constexpr (M <= kLaneMfmaMaxM) return &launch_m<M, kDistMfma>;
    else return nullptr;
}

template <int... Is>
constexpr auto make_table(std::integer_sequence<int, Is...>)
{
    return std::array<LaunchFn, 2 * sizeof...(Is)>{&launch_m<kPartLo + Is, kDistValu>...,
                                                   mfma_entry<kPartLo + Is>()...};
}

}  // namespace

hipError_t LLOYD_PART_FN(launch_lane_part)(const StepArgs &a, Mode mode, const AccumPlan &plan,
                                           hipStream_t s)
{
    static constexpr auto table = make_table(std::make_integer_sequence<int, kPartN>{});
    if (a.M < kPartLo || a.M >= kPartLo + kPartN) return hipErrorInvalidValue;
    const LaunchFn fn = table[(plan.path == kPathLaneMfma ? kPartN : 0) + a.M - kPartLo];
    return fn ? fn(a, mode, plan, s) : hipErrorInvalidValue;
}

#if LLOYD_PART == 0
bool lane_mfma_fits(int M, int K) { return K <= kLaneMfmaMaxK && M <= kLaneMfmaMaxM; }

AccumPlan plan_lane(int64_t n, int M, int K, Mode mode, bool mfma)
{
    AccumPlan p{};
    p.path = mfma ? kPathLaneMfma : kPathValu;
    auto bytes = [&](int W, int pa) {
        size_t b = lane_slab_off(M, W, mfma);
        if (mode != kAssign) b += (size_t)W * lane_acc_p(M, pa) * K * (M + 1) * 8;
        return b;
    };
    auto most_waves = [&](int pa) {
        int w = kMaxWaves;
        while (w > 0 && bytes(w, pa) > (size_t)kMaxLds) --w;
        return w;
    };
    // slabs with the most objects per step unless one object per step leaves
    // more waves (not in the matrix-core form, whose accumulation reads the
    // tile before the score rows overwrite it, which needs at most 32 steps)
    int pa = 0, W = most_waves(0);
    if (mode != kAssign && !mfma && most_waves(1) > W) {
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
