// Assignment by the L1 (city-block) distance, the other metric the paper
// allows in place of Eq. (2): label = argmin_k sum_j |x_j - c_kj|, lowest k on
// ties. Only the assignment changes; the sums of Eq. (1) and the centres are
// formed by the accumulate-from-labels and centres launches shared with the
// Euclidean path. This kernel serves the assign-only call and the iterations
// with K > 32; below that an iteration assigns and accumulates in one launch
// of the direct-form lane kernel (lloyd_lane.hip).
//
// One object per lane, on the vector ALU (the L1 distance is no contraction,
// so there is nothing for the matrix cores). The kernel is compiled for each
// feature count M. The centres sit in LDS, each padded with zeros to a
// multiple of 4 features, and are read with uniform (broadcast) 16-byte
// reads. Each lane holds its object's M features in registers, read from its
// wave's LDS tile slot. Only the M real features enter a distance.
//
// fp32 error: each term |fl(x_j - c_j)| is within u of |x_j - c_j| and the
// recursive sum of M non-negative terms adds gamma_{M-1}, so every computed
// distance is within gamma_M of the exact one (u = 2^-24, gamma_m =
// m u / (1 - m u)). A label is accepted when the two best computed distances
// differ by more than 2.02 gamma_M (d1 + d2); otherwise the object is
// re-decided with fp64 distances in the fixed order e = x_j - c_j,
// d = d + |e| (features ascending, each operation rounded), over all centres.
#include "lloyd_l1.h"

#include <math.h>

#include <utility>

namespace lloyd {

namespace {

constexpr int kL1MaxWaves = 8;
constexpr size_t kL1MaxLds = 150 * 1024;

typedef float f4v __attribute__((ext_vector_type(4)));

// features per centre row in LDS: M rounded up to a multiple of 4
__host__ __device__ constexpr int l1_row(int M) { return (M + 3) / 4 * 4; }

template <int M>
__global__ void __launch_bounds__(kL1MaxWaves * kWave)
lloyd_l1_kernel(const float *__restrict__ X, int64_t n, const float *__restrict__ C, int K,
                int32_t *__restrict__ labels, float *__restrict__ min_d, Ctl *__restrict__ ctl,
                int t, int fixed, int force64)
{
    constexpr int MB = l1_row(M);
    if (stop_before(ctl, t, fixed)) return;
    extern __shared__ __align__(16) float l1_lds[];
    const int lane = threadIdx.x % kWave, w = threadIdx.x / kWave, W = blockDim.x / kWave;
    f4v *cen = reinterpret_cast<f4v *>(l1_lds);               // [K][MB / 4]
    float *slot = l1_lds + (size_t)K * MB + (size_t)w * kWave * M;   // 16-byte aligned: K*MB, 64*M multiples of 4

    for (int e = threadIdx.x; e < K * MB; e += blockDim.x) {
        const int k = e / MB, j = e % MB;
        l1_lds[e] = j < M ? C[(int64_t)k * M + j] : 0.f;
    }
    __syncthreads();

    const double u = 5.9604644775390625e-8;
    const float tau = (float)(2.02 * (M * u / (1.0 - M * u)));
    const int64_t ntiles = (n + kWave - 1) / kWave;
    const int64_t stride = (int64_t)gridDim.x * W;
    int nfallback = 0;

    for (int64_t q = (int64_t)w * gridDim.x + blockIdx.x; q < ntiles; q += stride) {
        // stage the tile (64 objects, M features each): a full tile is 16 M
        // aligned float4s (X is 16-byte aligned and 64 M floats a multiple of
        // 4), read with 16-byte loads; the last, partial tile element by
        // element with zeros past n
        const int64_t base = q * kWave * (int64_t)M;
        if ((q + 1) * kWave <= n) {
            const f4v *src = reinterpret_cast<const f4v *>(X + base);
            f4v *dst = reinterpret_cast<f4v *>(slot);
            for (int v = lane; v < 16 * M; v += kWave) dst[v] = src[v];
        } else {
            const int64_t total = n * (int64_t)M;
            for (int e = lane; e < kWave * M; e += kWave)
                slot[e] = base + e < total ? X[base + e] : 0.f;
        }
        __builtin_amdgcn_wave_barrier();
        const int64_t i = q * kWave + lane;

        // the object's features stay in registers
        float x[M];
#pragma unroll
        for (int j = 0; j < M; ++j) {
            x[j] = slot[lane * M + j];
            asm volatile("" : "+v"(x[j]));            // keep it in a register: no re-read per centre
        }

        float b1 = INFINITY, b2 = INFINITY;
        int lab = 0;
        for (int k = 0; k < K; ++k) {
            float d = 0.f;
#pragma unroll
            for (int j4 = 0; j4 < MB / 4; ++j4) {
                const f4v c = cen[k * (MB / 4) + j4];
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (4 * j4 + e < M) d = d + fabsf(x[4 * j4 + e] - c[e]);
            }
            if (d < b1) {
                b2 = b1;
                b1 = d;
                lab = k;
            } else if (d < b2) {
                b2 = d;
            }
        }
        float best = b1;
        // every fp32 distance overflowed or is NaN (b1 never set): the fp64
        // distances may still tell the centres apart
        const bool close = force64 || !(b1 < INFINITY) ||
                           (b2 != INFINITY && !(b2 - b1 > tau * (b1 + b2)));
        if (close && i < n) {
            // too close to call in fp32: every centre again in fp64
            double bd = INFINITY;
            lab = 0;
            for (int k = 0; k < K; ++k) {
                const float *c = C + (int64_t)k * M;
                double d = 0.0;
                for (int j = 0; j < M; ++j) {
                    const double e = (double)slot[lane * M + j] - (double)c[j];
                    d = d + fabs(e);
                }
                if (d < bd) {
                    bd = d;
                    lab = k;
                }
            }
            best = (float)bd;
            ++nfallback;
        }
        if (i < n) {
            labels[i] = lab;
            if (min_d) min_d[i] = best;
        }
        __builtin_amdgcn_wave_barrier();              // the slot's reads are done
    }
    if (ctl) {
        int s = nfallback;
#pragma unroll
        for (int off = kWave / 2; off > 0; off >>= 1) s += __shfl_xor(s, off);
        if (lane == 0 && s) atomicAdd(&ctl->fallbacks, s);
    }
}

template <int M>
hipError_t l1_launch_m(const StepArgs &a, const L1Plan &pl, hipStream_t s)
{
    auto kern = lloyd_l1_kernel<M>;
    static const size_t st = static_lds_bytes(reinterpret_cast<const void *>(kern));
    if (st > (size_t)kMaxLds || st + pl.lds_bytes > (size_t)kMaxLds)
        return hipErrorInvalidConfiguration;
    hipExtLaunchKernelGGL(kern, dim3(pl.groups), dim3(pl.waves * kWave), pl.lds_bytes, s,
                          a.ev_start, a.ev_stop, 0, a.X, a.n, a.C, a.K, a.labels, a.min_d2, a.ctl,
                          a.t, a.fixed, a.force64);
    return hipGetLastError();
}

// the instance for M = a.M (1 .. kMaxM)
template <int... Ms>
hipError_t l1_dispatch(std::integer_sequence<int, Ms...>, const StepArgs &a, const L1Plan &pl,
                       hipStream_t s)
{
    hipError_t r = hipErrorInvalidValue;
    (void)((a.M == Ms + 1 ? (r = l1_launch_m<Ms + 1>(a, pl, s), true) : false) || ...);
    return r;
}

}  // namespace

L1Plan plan_l1(int64_t n, int M, int K)
{
    L1Plan pl{};
    const size_t cen = (size_t)K * l1_row(M) * sizeof(float);
    const size_t slot = (size_t)kWave * M * sizeof(float);
    int W = cen + slot > kL1MaxLds ? 0 : (int)((kL1MaxLds - cen) / slot);
    if (W > kL1MaxWaves) W = kL1MaxWaves;
    const int64_t nq = (n + kWave - 1) / kWave;
    while (W > 1 && W / 2 >= nq) W /= 2;
    // up to four workgroups per compute unit: the per-centre loop waits on its
    // LDS reads, and more resident waves hide that wait
    int64_t groups = W > 0 ? (nq + W - 1) / W : 0;
    if (groups > 4 * kCUs) groups = 4 * kCUs;
    pl.waves = W;
    pl.groups = (int)groups;
    pl.lds_bytes = cen + (size_t)W * slot;
    return pl;
}

hipError_t launch_l1(const StepArgs &a, const L1Plan &pl, hipStream_t s)
{
    if (pl.waves < 1 || pl.groups < 1) return hipErrorInvalidConfiguration;
    if (a.M < 1 || a.M > kMaxM) return hipErrorInvalidValue;
    return l1_dispatch(std::make_integer_sequence<int, kMaxM>{}, a, pl, s);
}

}  // namespace lloyd
