// Initial centres of Algorithm 1 step 1 (K objects lying far apart,
// method left open), taken as farthest-point traversal from object 0:
//   idx[0] = 0, and idx[m] = the not-yet-chosen object whose smallest squared
//   distance (Eq. (2)) to the objects idx[0..m-1] is largest, lowest index on
//   ties.
// The choice is an argmax decided by fp64 distances formed in the fixed
// operation order of the library's exact re-decisions (e = x_j - c_j, then
// d = d + e*e, features ascending, each operation rounded on its own), so the
// chosen indices are exactly those of that definition.
//
// One launch per pass p = 1 .. K-1, each a stream over X:
//   - every workgroup first reduces the per-workgroup candidates of pass p-1
//     (G pairs, a few KB from L2) to the newest centre c = idx[p-1] (object 0
//     when p = 1); workgroup 0 records idx[p-1] and copies row X[c] into the
//     centres;
//   - each object's nearest distance becomes min(nearest, |x - X[c]|^2), and
//     object c itself is marked chosen with -1, which no later minimum with a
//     distance (>= 0) undoes; the last pass keeps nothing;
//   - each workgroup writes its farthest (distance, lowest index) pair to the
//     half of the candidate buffer that pass p owns (pass p+1 reads it, pass
//     p+2 overwrites it, so no launch reads what it writes).
// A last one-workgroup launch (p = K) only records idx[K-1]. With K = 1 that
// launch is the only one and records object 0.
//
// The traversal may also start from S given seed objects (device array, e.g.
// the two ends of the diameter): passes p <= S take seed p-1 as the newest
// centre instead of the previous pass's farthest object.
//
// Streaming follows the distance kernels: 64-object tiles, each wave's next
// tile in flight in registers while the current one is read from its LDS slot,
// the ragged last tile handled after the loop by the one wave whose sequence
// reaches it.
#include "lloyd_device.h"
#include "farthest.h"

#include <array>
#include <climits>
#include <utility>

namespace lloyd {

namespace {

constexpr int kFarMaxWaves = 16;
constexpr size_t kFarMaxDynLds = 150 * 1024;

// Candidates ordered by distance, then by the lower index: the maximum is the
// farthest object with the lowest index on ties, whatever order pairs meet in.
__device__ inline void far_merge(double &v, int &i, double v2, int i2)
{
    if (v2 > v || (v2 == v && i2 < i)) {
        v = v2;
        i = i2;
    }
}

// Workgroup-wide maximum; every thread receives it.
__device__ inline void far_block_max(double &v, int &i, double *sv, int *si)
{
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) {
        const double v2 = __shfl_xor(v, off);
        const int i2 = __shfl_xor(i, off);
        far_merge(v, i, v2, i2);
    }
    const int w = threadIdx.x / kWave, W = blockDim.x / kWave;
    __syncthreads();                      // sv / si of an earlier call are read
    if (threadIdx.x % kWave == 0) {
        sv[w] = v;
        si[w] = i;
    }
    __syncthreads();
    v = -INFINITY;
    i = INT_MAX;
    for (int k = 0; k < W; ++k) far_merge(v, i, sv[k], si[k]);
}

template <int M>
__global__ void __launch_bounds__(kFarMaxWaves * kWave)
farthest_pass_kernel(const float *__restrict__ X, int64_t n, int K, int p,
                     double *__restrict__ nearest, double *__restrict__ cand_v,
                     int32_t *__restrict__ cand_i, int groups, int32_t *__restrict__ idx_out,
                     float *__restrict__ centers_out, const int32_t *__restrict__ seeds,
                     int nseeds)
{
    using G = TileGeom<M>;
    constexpr int V = G::kVecPerLane;
    extern __shared__ float far_lds[];
    __shared__ double sv[kFarMaxWaves];
    __shared__ int si[kFarMaxWaves];
    __shared__ double cd[M];                  // the newest centre, in fp64
    const int lane = threadIdx.x % kWave, w = threadIdx.x / kWave, W = blockDim.x / kWave;

    // the newest centre: a seed (object 0 without seeds), or the farthest
    // object of the previous pass
    int c = 0;
    if (p <= nseeds) {
        if (seeds != nullptr) {
            c = seeds[p - 1];
            if (c < 0 || (int64_t)c >= n) c = 0;          // refused on the host; reads stay in bounds
        }
    } else {
        const int half = ((p - 1) & 1) * groups;
        double v = -INFINITY;
        int i = INT_MAX;
        for (int g = threadIdx.x; g < groups; g += blockDim.x)
            far_merge(v, i, cand_v[half + g], cand_i[half + g]);
        far_block_max(v, i, sv, si);
        // with finite inputs the maximum is an unchosen object's distance
        // (>= 0); the clamp only keeps non-finite inputs' reads in bounds
        c = (i >= 0 && (int64_t)i < n) ? i : 0;
    }
    c = __builtin_amdgcn_readfirstlane(c);
    const float *crow = X + (int64_t)c * M;
    if (blockIdx.x == 0) {
        if (threadIdx.x == 0) idx_out[p - 1] = c;
        for (int j = threadIdx.x; j < M; j += blockDim.x)
            centers_out[(int64_t)(p - 1) * M + j] = crow[j];
    }
    if (p >= K) return;

    for (int j = threadIdx.x; j < M; j += blockDim.x) cd[j] = (double)crow[j];
    __syncthreads();

    float *slot = far_lds + w * G::kSlot;
    const int64_t nfull = n / kWave;
    const int64_t stride = (int64_t)groups * W;
    const bool keep = p + 1 < K;              // a later pass reads the distances
    double bv = -INFINITY;
    int bi = INT_MAX;

    auto pass_tile = [&](int64_t q, bool full) {
        const int64_t i = q * kWave + lane;
        const bool valid = full || i < n;
        const double old = (p > 1 && valid) ? nearest[i] : INFINITY;
        const float *x = slot + lane * M;
        double d = 0.0;
#pragma unroll
        for (int j = 0; j < M; ++j) {
            const double e = (double)x[j] - cd[j];
            const double sq = e * e;
            d = d + sq;
        }
        double nv = d < old ? d : old;
        if (i == c) nv = -1.0;
        if (valid) {
            if (keep) nearest[i] = nv;
            far_merge(bv, bi, nv, (int)i);
        }
    };

    int64_t q = (int64_t)w * groups + blockIdx.x;
    float4 buf[V];
    if (q < nfull) load_tile<M>(X, q, lane, buf);
    for (; q < nfull; q += stride) {
        store_tile<M>(slot, lane, buf);
        __builtin_amdgcn_wave_barrier();
        if (q + stride < nfull) load_tile<M>(X, q + stride, lane, buf);
        pass_tile(q, true);
    }
    // exactly one wave's sequence reaches the partial last tile
    if (q == nfull && nfull * kWave < n) {
        load_tail_tile<M>(X, n, q, lane, buf);
        store_tile<M>(slot, lane, buf);
        __builtin_amdgcn_wave_barrier();
        pass_tile(q, false);
    }

    far_block_max(bv, bi, sv, si);
    if (threadIdx.x == 0) {
        cand_v[(p & 1) * groups + blockIdx.x] = bv;
        cand_i[(p & 1) * groups + blockIdx.x] = bi;
    }
}

template <int M>
hipError_t farthest_m(const FarthestArgs &a, const FarthestPlan &pl, hipStream_t s)
{
    auto kern = farthest_pass_kernel<M>;
    static const size_t st = static_lds_bytes(reinterpret_cast<const void *>(kern));
    if (st > (size_t)kMaxLds || st + pl.lds_bytes > (size_t)kMaxLds)
        return hipErrorInvalidConfiguration;
    for (int p = 1; p <= a.K; ++p) {
        const dim3 grid(p < a.K ? pl.groups : 1), block(pl.waves * kWave);
        hipLaunchKernelGGL(kern, grid, block, pl.lds_bytes, s, a.X, a.n, a.K, p, a.nearest,
                           a.cand_v, a.cand_i, pl.groups, a.idx, a.centers, a.seeds,
                           a.nseeds);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

using FarFn = hipError_t (*)(const FarthestArgs &, const FarthestPlan &, hipStream_t);

template <int... Is>
constexpr auto far_table(std::integer_sequence<int, Is...>)
{
    return std::array<FarFn, sizeof...(Is)>{&farthest_m<Is + 1>...};
}

}  // namespace

FarthestPlan plan_farthest(int64_t n, int M)
{
    FarthestPlan pl{};
    const size_t slot = (size_t)((kWave * M + (M > 4 ? M : 4) + 3) / 4 * 4) * sizeof(float);
    int W = (int)(kFarMaxDynLds / slot);
    if (W > kFarMaxWaves) W = kFarMaxWaves;
    const int64_t nq = (n + kWave - 1) / kWave;
    while (W > 1 && W / 2 >= nq) W /= 2;
    int64_t groups = (nq + W - 1) / W;
    if (groups > kCUs) groups = kCUs;
    pl.waves = W;
    pl.groups = (int)groups;
    pl.lds_bytes = (size_t)W * slot;
    return pl;
}

hipError_t launch_farthest(const FarthestArgs &a, const FarthestPlan &pl, hipStream_t s)
{
    static constexpr auto table = far_table(std::make_integer_sequence<int, kMaxM>{});
    if (a.M < 1 || a.M > kMaxM || a.K < 1 || (int64_t)a.K > a.n || a.nseeds < 1 ||
        a.nseeds > a.K || (a.seeds == nullptr && a.nseeds != 1))
        return hipErrorInvalidValue;
    return table[a.M - 1](a, pl, s);
}

}  // namespace lloyd
