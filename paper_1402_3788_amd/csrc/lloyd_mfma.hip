// Fused assign + accumulate with the distances on the matrix cores.
//
// Expanded form of the squared distance of Eq. (2): for object x and centre c,
//     |x - c|^2 = |x|^2 + score,   score = |c|^2 - 2 x.c,
// and |x|^2 is the same for every centre, so the nearest centre is the one with
// the smallest score. For 16 centres and 16 objects the scores are one
// v_mfma_f32_16x16x4f32 chain over the features (4 per step, zero-padded):
//     D[centre][object] = |c|^2 + sum_j (-2 c_j) x_j,
// with A = -2C (16 x 4 per step, built once per workgroup in LDS, already in
// the lane order the instruction wants), B = X^T (4 x 16 per step, read from
// the LDS tile) and the accumulator seeded with |c|^2.
//
// Layout of v_mfma_f32_16x16x4f32 (64 lanes): A[i][k] is in lane i + 16k,
// B[k][j] in lane j + 16k, and D[i][j] in lane j + 16(i/4), register i%4. So
// after a chain every lane holds the scores of 4 centres for one object; a lane
// keeps a running best / second-best over its centres, and two xor-shuffles
// (16, 32) merge the four lanes that share an object.
//
// The expanded form cancels: its fp32 error is bounded by
// gamma_{M+2} (3|c|^2 + |x|^2), so a label is accepted only if the two best
// scores differ by more than 2.5 times that bound (with |c|^2 bounded by the
// largest centre norm). Other objects are re-decided with fp64 distances in the
// fixed operation order, over all centres, lowest index on ties.
//
// Accumulation (the sums of Eq. (1)) has two forms, both free of atomics and
// with every addition in an order fixed by the problem shape:
//   wave    -- each wavefront adds its own tiles into a private fp64 slab (no
//              barriers); at the end the workgroup adds the slabs in wave order.
//              Used while W private slabs fit in LDS (small K*M).
//   block   -- one fp64 slab per workgroup: after a barrier, wave w owns the
//              clusters k = w, w+W, ...; for each it lists the workgroup tile's
//              members in ascending object order (ballot + prefix count) and
//              adds them. Used for large K*M.
#include "lloyd.h"
#include "lloyd_device.h"
#include "lloyd_reduce.h"

#include <math.h>

#include <array>
#include <utility>

#include "lloyd_parts.h"

namespace lloyd {

namespace {

typedef float f4v __attribute__((ext_vector_type(4)));

constexpr int kCols = 4;      // 16-object columns per wave tile (64 objects)
constexpr int kAccWave = 1;
constexpr int kAccBlock = 2;
constexpr int kMaxWaves = 16;

// LDS carve-up of a workgroup (dynamic shared memory).
struct MfmaLds {
    size_t ones, tiles, aswz, cnorm, misc, labs, members, scratch, slab, cnt, total;
    int tile_floats;
};

__host__ __device__ inline size_t al16(size_t v) { return (v + 15) & ~size_t(15); }

__host__ __device__ inline MfmaLds mfma_lds(int M, int K, int W, int acc)
{
    const int KS = (M + 3) / 4, KT = (K + 15) / 16;
    MfmaLds L{};
    L.tile_floats = (kWave * M + (M > 4 ? M : 4) + 3) / 4 * 4;    // tile + zero slack
    size_t o = 0;
    L.ones = o;    o = al16(o + 68 * 4);
    L.tiles = o;   o = al16(o + (size_t)W * L.tile_floats * 4);
    L.aswz = o;    o = al16(o + (size_t)KT * KS * kWave * 4);
    L.cnorm = o;   o = al16(o + (size_t)KT * 16 * 4);
    L.misc = o;    o = al16(o + 16);
    if (acc == kAccWave) {
        L.slab = o;    o = al16(o + (size_t)W * K * (M + 1) * 8);
    } else if (acc == kAccBlock) {
        L.labs = o;    o = al16(o + (size_t)W * kWave * 4);
        L.members = o; o = al16(o + (size_t)W * W * kWave * 4);
        L.scratch = o; o = al16(o + (size_t)W * kWave * 8);
        L.slab = o;    o = al16(o + (size_t)K * M * 8);
        L.cnt = o;     o = al16(o + (size_t)K * 4);
    }
    L.total = o;
    return L;
}

template <int M, int MODE, int ACC>
__global__ void __launch_bounds__(kMaxWaves * kWave)
lloyd_mfma_kernel(const float *__restrict__ X, int64_t n, const float *__restrict__ C, int K,
                  int32_t *__restrict__ labels, const int32_t *__restrict__ labels_in,
                  float *__restrict__ min_d2, double *__restrict__ part_sums,
                  int32_t *__restrict__ part_counts, Ctl *__restrict__ ctl, int t, int fixed,
                  TreeArgs tree)
{
    using TG = TileGeom<M>;
    constexpr int KS = (M + 3) / 4;
    constexpr int kTilePad = Slots<M>::kTileFloats;   // floats per wave tile slot
    constexpr int MW = Slots<M>::MW;
    constexpr bool kAccum = MODE != kAssign;
    constexpr int kAcc = kAccum ? ACC : 0;
    extern __shared__ __align__(16) unsigned char smem[];
    const int W = blockDim.x / kWave;
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int tid = threadIdx.x;
    const int KT = (K + 15) / 16;

    if (MODE == kAssignAccum && stop_before(ctl, t, fixed)) return;

    const MfmaLds L = mfma_lds(M, K, W, kAcc);
    float *ones = reinterpret_cast<float *>(smem + L.ones);
    float *tiles = reinterpret_cast<float *>(smem + L.tiles);
    float *tile = tiles + wave * kTilePad;
    float *aswz = reinterpret_cast<float *>(smem + L.aswz);
    float *cnorm = reinterpret_cast<float *>(smem + L.cnorm);
    float *s_cmax = reinterpret_cast<float *>(smem + L.misc);

    const int64_t nq = (n + kWave - 1) / kWave;
    const int64_t nbt = (nq + W - 1) / W;

    // first tile's loads go out before the prologue
    float4 buf[TG::kVecPerLane];
    int64_t bt = blockIdx.x;
    if (bt < nbt && bt * W + wave < nq) load_tile<M>(X, n, bt * W + wave, lane, buf);

    // ---- prologue: A operands (-2C in lane order), centre norms, slabs
    if (MODE != kAccumLabels) {
        for (int idx = tid; idx < KT * KS * kWave; idx += blockDim.x) {
            const int tt = idx / (KS * kWave), s = (idx / kWave) % KS, l = idx % kWave;
            const int k = tt * 16 + (l & 15), j = 4 * s + (l >> 4);
            aswz[idx] = (k < K && j < M) ? -2.0f * C[(int64_t)k * M + j] : 0.0f;
        }
    }
    {
        constexpr int kSlack = kTilePad - kWave * M;     // zeros after each tile
        for (int i = tid; i < W * kSlack; i += blockDim.x)
            tiles[(i / kSlack) * kTilePad + kWave * M + (i % kSlack)] = 0.f;
    }
    if (kAcc == kAccWave) {
        double *slabs = reinterpret_cast<double *>(smem + L.slab);
        for (int i = tid; i < W * K * MW; i += blockDim.x) slabs[i] = 0.0;
        for (int i = tid; i < 68; i += blockDim.x) ones[i] = i < kWave ? 1.f : 0.f;
    } else if (kAcc == kAccBlock) {
        double *slab = reinterpret_cast<double *>(smem + L.slab);
        int32_t *cnt = reinterpret_cast<int32_t *>(smem + L.cnt);
        for (int i = tid; i < K * M; i += blockDim.x) slab[i] = 0.0;
        for (int i = tid; i < K; i += blockDim.x) cnt[i] = 0;
    }
    __syncthreads();
    if (MODE != kAccumLabels) {
        // |c_k|^2 in fp32, features in order, from c = -a/2 (exact)
        for (int k = tid; k < KT * 16; k += blockDim.x) {
            float nk = INFINITY;
            if (k < K) {
                const int tt = k / 16, i16 = k % 16;
                nk = 0.f;
#pragma unroll
                for (int j = 0; j < M; ++j) {
                    const float c = -0.5f * aswz[(tt * KS + j / 4) * kWave + i16 + 16 * (j % 4)];
                    nk = __builtin_fmaf(c, c, nk);
                }
            }
            cnorm[k] = nk;
        }
        __syncthreads();
        if (wave == 0) {
            float m = 0.f;
            for (int k = lane; k < K; k += kWave) m = fmaxf(m, cnorm[k]);
            for (int off = 32; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off, kWave));
            if (lane == 0) *s_cmax = m;
        }
        __syncthreads();
    }
    const float cmax = (MODE != kAccumLabels) ? *s_cmax : 0.f;
    // fp32 error bound of a score, relative to (3|c|^2 + |x|^2), with margins
    constexpr float kGuard = 2.5f * 1.01f * (float)(M + 2) * 5.9604645e-8f;

    const int g = lane >> 4, l16 = lane & 15;
    int nfallback = 0;

    for (; bt < nbt; bt += gridDim.x) {
        const int64_t q = bt * W + wave;
        const bool have = q < nq;
        if (kAcc != kAccBlock && !have) break;      // no barriers inside: a wave may stop
        if (have) store_tile<M>(tile, lane, buf);
        __builtin_amdgcn_wave_barrier();
        {
            const int64_t qn = (bt + gridDim.x) * W + wave;
            if (bt + gridDim.x < nbt && qn < nq) load_tile<M>(X, n, qn, lane, buf);
        }
        const int64_t i = q * kWave + lane;
        const bool valid = have && i < n;
        int my_lab = -1;

        if (have && MODE == kAccumLabels) {
            if (valid) {
                my_lab = labels_in[i];
                if (my_lab < 0 || my_lab >= K) my_lab = -1;
            }
        } else if (have) {
            // B operands: object 16c + l16, features 4s + g
            float b[kCols][KS];
            float xsq[kCols];
#pragma unroll
            for (int c = 0; c < kCols; ++c) {
                const float *row = tile + (16 * c + l16) * M + g;
                float acc = 0.f;
#pragma unroll
                for (int s = 0; s < KS; ++s) {
                    float v = row[4 * s];
                    if ((M % 4) != 0 && s == KS - 1 && 4 * s + g >= M) v = 0.f;
                    b[c][s] = v;
                    acc = __builtin_fmaf(v, v, acc);
                }
                acc += __shfl_xor(acc, 16, kWave);
                acc += __shfl_xor(acc, 32, kWave);
                xsq[c] = acc;
            }
            float b1[kCols], b2[kCols];
            int lb[kCols];
#pragma unroll
            for (int c = 0; c < kCols; ++c) {
                b1[c] = INFINITY;
                b2[c] = INFINITY;
                lb[c] = 0;
            }
            for (int tt = 0; tt < KT; ++tt) {
                float a[KS];
#pragma unroll
                for (int s = 0; s < KS; ++s) a[s] = aswz[(tt * KS + s) * kWave + lane];
                f4v d[kCols];
                const f4v cinit = *reinterpret_cast<const f4v *>(cnorm + tt * 16 + 4 * g);
#pragma unroll
                for (int c = 0; c < kCols; ++c) d[c] = cinit;
#pragma unroll
                for (int s = 0; s < KS; ++s)
#pragma unroll
                    for (int c = 0; c < kCols; ++c)
                        d[c] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[s], b[c][s], d[c], 0, 0, 0);
                const int kb = tt * 16 + 4 * g;
#pragma unroll
                for (int c = 0; c < kCols; ++c)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const float sc = d[c][r];
                        const bool lt = sc < b1[c];
                        b2[c] = __builtin_amdgcn_fmed3f(b1[c], b2[c], sc);
                        b1[c] = lt ? sc : b1[c];
                        lb[c] = lt ? kb + r : lb[c];
                    }
            }
            // merge the four lanes that hold the same object (no branches: the
            // second best of two (best, second) pairs is the median of
            // (b1, pb1, min(b2, pb2)) when b1 <= b2 and pb1 <= pb2)
#pragma unroll
            for (int c = 0; c < kCols; ++c)
#pragma unroll
                for (int off = 16; off <= 32; off <<= 1) {
                    const float pb1 = __shfl_xor(b1[c], off, kWave);
                    const float pb2 = __shfl_xor(b2[c], off, kWave);
                    const int pl = __shfl_xor(lb[c], off, kWave);
                    const float m2 = __builtin_amdgcn_fmed3f(b2[c], pb2, -INFINITY);
                    const float nb2 = __builtin_amdgcn_fmed3f(b1[c], pb1, m2);
                    const bool take = (pb1 < b1[c]) | ((pb1 == b1[c]) & (pl < lb[c]));
                    b1[c] = take ? pb1 : b1[c];
                    lb[c] = take ? pl : lb[c];
                    b2[c] = nb2;
                }
            // lane l reports object l, which sits in column c = l / 16 = g
            float mb1 = b1[0], mb2 = b2[0], mx = xsq[0];
            int ml = lb[0];
#pragma unroll
            for (int c = 1; c < kCols; ++c)
                if (g == c) {
                    mb1 = b1[c];
                    mb2 = b2[c];
                    mx = xsq[c];
                    ml = lb[c];
                }
            const float thr = kGuard * (3.02f * cmax + 1.0001f * mx) + 1e-30f;
            const bool ok = (K == 1) || (mb2 - mb1 > thr);
            float dmin = 0.f;
            if (valid && !ok) {
                float x[M];
#pragma unroll
                for (int j = 0; j < M; ++j) x[j] = tile[lane * M + j];
                double bd;
                ml = argmin_fp64<M>(x, C, K, bd);
                dmin = (float)bd;
            } else if (valid && MODE == kAssign && min_d2 != nullptr) {
                const float *c = C + (int64_t)ml * M;
                float d = 0.f;
#pragma unroll
                for (int j = 0; j < M; ++j) {
                    const float e = tile[lane * M + j] - c[j];
                    d = __builtin_fmaf(e, e, d);
                }
                dmin = d;
            }
            if (ctl != nullptr) nfallback += __popcll(__ballot(valid && !ok));
            if (valid) {
                labels[i] = ml;
                if (MODE == kAssign && min_d2 != nullptr) min_d2[i] = dmin;
                my_lab = ml;
            }
        }

        if (kAcc == kAccWave) {
            double *slab = reinterpret_cast<double *>(smem + L.slab) + (size_t)wave * K * MW;
            wave_accumulate<M>(valid ? my_lab : -1, tile, ones, slab, K, lane);
            __builtin_amdgcn_wave_barrier();
        } else if (kAcc == kAccBlock) {
            int32_t *labs = reinterpret_cast<int32_t *>(smem + L.labs);
            int32_t *members = reinterpret_cast<int32_t *>(smem + L.members) + wave * W * kWave;
            double *scratch = reinterpret_cast<double *>(smem + L.scratch) + wave * kWave;
            double *slab = reinterpret_cast<double *>(smem + L.slab);
            int32_t *cnt = reinterpret_cast<int32_t *>(smem + L.cnt);
            constexpr int P = kWave / M;
            labs[wave * kWave + lane] = valid ? my_lab : -1;
            __syncthreads();
            const int s = lane / M, j = lane % M;
            for (int k = wave; k < K; k += W) {
                int cnt_k = 0;
                for (int v = 0; v < W; ++v) {
                    const bool mine = labs[v * kWave + lane] == k;
                    const uint64_t mask = __ballot(mine);
                    const int rank = __builtin_amdgcn_mbcnt_hi(
                        (uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
                    if (mine) members[cnt_k + rank] = v * kTilePad + lane * M;
                    cnt_k += __popcll(mask);
                }
                if (cnt_k == 0) continue;
                __builtin_amdgcn_wave_barrier();
                double acc = 0.0;
                if (s < P) {
                    for (int base = 0; base < cnt_k; base += P) {
                        const int idx = base + s;
                        if (idx < cnt_k) acc = acc + (double)tiles[members[idx] + j];
                    }
                }
                scratch[lane] = acc;
                __builtin_amdgcn_wave_barrier();
                if (lane < M) {
                    double tsum = 0.0;
                    for (int u = 0; u < P; ++u) tsum = tsum + scratch[u * M + lane];
                    slab[k * M + lane] = slab[k * M + lane] + tsum;
                }
                if (lane == 0) cnt[k] += cnt_k;
                __builtin_amdgcn_wave_barrier();
            }
            __syncthreads();
        }
    }

    if (ctl != nullptr && lane == 0 && nfallback > 0) atomicAdd(&ctl->fallbacks, nfallback);

    if (kAcc == kAccWave) {
        __syncthreads();
        const double *slabs = reinterpret_cast<const double *>(smem + L.slab);
        double *out = part_sums + (int64_t)blockIdx.x * K * M;
        for (int e = tid; e < K * M; e += blockDim.x) {
            const int k = e / M, j = e - (e / M) * M;
            double s = slabs[k * MW + j];
            for (int w = 1; w < W; ++w) s = s + slabs[(size_t)w * K * MW + k * MW + j];
            out[e] = s;
        }
        for (int k = tid; k < K; k += blockDim.x) {
            double c = 0.0;
            for (int w = 0; w < W; ++w) c = c + slabs[(size_t)w * K * MW + k * MW + M];
            part_counts[(int64_t)blockIdx.x * K + k] = (int32_t)c;
        }
    } else if (kAcc == kAccBlock) {
        const double *slab = reinterpret_cast<const double *>(smem + L.slab);
        const int32_t *cnt = reinterpret_cast<const int32_t *>(smem + L.cnt);
        double *out = part_sums + (int64_t)blockIdx.x * K * M;
        for (int e = tid; e < K * M; e += blockDim.x) out[e] = slab[e];
        for (int k = tid; k < K; k += blockDim.x) part_counts[(int64_t)blockIdx.x * K + k] = cnt[k];
    }
    if (kAccum) tree_finalize(tree, reinterpret_cast<uint32_t *>(smem + L.slab));
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
#define LLOYD_MFMA_LAUNCH(MD, AC)                                                              \
    hipLaunchKernelGGL((lloyd_mfma_kernel<M, MD, AC>), grid, block, p.lds_bytes, s, a.X, a.n,   \
                       a.C, a.K, a.labels, a.labels_in, a.min_d2, a.part_sums, a.part_counts,  \
                       a.ctl, a.t, a.fixed, tr)
    const bool wave_acc = p.accum == kAccWave;
    switch (mode) {
    case kAssign: LLOYD_MFMA_LAUNCH(kAssign, kAccWave); break;
    case kAssignAccum:
        if (wave_acc) LLOYD_MFMA_LAUNCH(kAssignAccum, kAccWave);
        else LLOYD_MFMA_LAUNCH(kAssignAccum, kAccBlock);
        break;
    case kAccumLabels:
        if (wave_acc) LLOYD_MFMA_LAUNCH(kAccumLabels, kAccWave);
        else LLOYD_MFMA_LAUNCH(kAccumLabels, kAccBlock);
        break;
    }
#undef LLOYD_MFMA_LAUNCH
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

hipError_t LLOYD_PART_FN(launch_mfma_part)(const StepArgs &a, Mode mode, const AccumPlan &plan, hipStream_t s)
{
    static constexpr auto table = make_table(std::make_integer_sequence<int, kPartN>{});
    if (a.M < kPartLo || a.M >= kPartLo + kPartN) return hipErrorInvalidValue;
    return table[a.M - kPartLo](a, mode, plan, s);
}

#if LLOYD_PART == 0
AccumPlan plan_mfma(int64_t n, int M, int K, Mode mode)
{
    AccumPlan p{};
    p.path = kPathMfma;
    const int64_t nq = (n + kWave - 1) / kWave;
    auto fits = [&](int W, int acc) { return mfma_lds(M, K, W, acc).total <= (size_t)kMaxLds; };
    int W = kMaxWaves, acc = 0;
    if (mode == kAssign) {
        while (W > 1 && !fits(W, 0)) W /= 2;
    } else {
        // private slabs while at least 8 waves fit, else one shared slab
        acc = kAccWave;
        while (W > 8 && !fits(W, kAccWave)) --W;
        if (!fits(W, kAccWave)) {
            acc = kAccBlock;
            W = kMaxWaves;
            while (W > 1 && !fits(W, kAccBlock)) W /= 2;
        }
    }
    // no more waves than there are 64-object tiles
    while (W > 1 && W / 2 >= nq) W /= 2;
    int64_t groups = (nq + W - 1) / W;
    if (groups > kCUs) groups = kCUs;       // one persistent workgroup per compute unit
    p.waves = W;
    p.groups = (int)groups;
    p.accum = acc;
    p.lds_bytes = mfma_lds(M, K, W, acc).total;
    return p;
}

bool mfma_fits(int M, int K)
{
    return mfma_lds(M, K, 1, kAccBlock).total <= (size_t)kMaxLds;
}

hipError_t launch_mfma(const StepArgs &a, Mode mode, const AccumPlan &plan, hipStream_t s)
{
    if (a.M < 1 || a.M > kMaxM) return hipErrorInvalidValue;
    switch ((a.M - 1) / (kMaxM / LLOYD_PARTS)) {
#define LLOYD_CASE(P) case P: return launch_mfma_part_##P(a, mode, plan, s);
        LLOYD_PART_CASES
#undef LLOYD_CASE
    }
    return hipErrorInvalidValue;
}
#endif

}  // namespace lloyd
