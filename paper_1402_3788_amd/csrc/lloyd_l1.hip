// Assignment by the L1 (city-block) distance, the other metric the paper
// allows in place of Eq. (2): label = argmin_k sum_j |x_j - c_kj|, lowest k on
// ties. Only the assignment changes; the sums of Eq. (1) and the centres are
// formed by the accumulate-from-labels and centres launches shared with the
// Euclidean path.
//
// One object per lane, on the vector ALU (the L1 distance is no contraction,
// so there is nothing for the matrix cores). The centres sit in LDS padded to
// MB = 4, 8, 16, 32 or 64 features with zeros and are read with uniform
// (broadcast) 16-byte reads; each lane holds its object's features in
// registers, zero past M, read from its wave's LDS tile slot. Padding adds
// |0 - 0| = 0 exactly, so the fp32 sum is the sum over the M real features.
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

namespace lloyd {

namespace {

constexpr int kL1MaxWaves = 8;
constexpr size_t kL1MaxLds = 150 * 1024;

typedef float f4v __attribute__((ext_vector_type(4)));

int l1_padded(int M) { return M <= 4 ? 4 : M <= 8 ? 8 : M <= 16 ? 16 : M <= 32 ? 32 : 64; }

template <int MB>
__global__ void __launch_bounds__(kL1MaxWaves * kWave)
lloyd_l1_kernel(const float *__restrict__ X, int64_t n, int M, const float *__restrict__ C,
                int K, int32_t *__restrict__ labels, float *__restrict__ min_d,
                Ctl *__restrict__ ctl, int t, int fixed, int force64)
{
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

        // every lane reads every feature (the index clamped to the row, the
        // value zeroed past M), so the features stay in registers, branch-free
        float x[MB];
#pragma unroll
        for (int j = 0; j < MB; ++j) {
            const float v = slot[lane * M + (j < M ? j : M - 1)];
            x[j] = j < M ? v : 0.f;
            asm volatile("" : "+v"(x[j]));            // keep it in a register: no re-read per centre
        }

        float b1 = INFINITY, b2 = INFINITY;
        int lab = 0;
        for (int k = 0; k < K; ++k) {
            float d = 0.f;
#pragma unroll
            for (int j4 = 0; j4 < MB / 4; ++j4) {
                const f4v c = cen[k * (MB / 4) + j4];
                d = d + fabsf(x[4 * j4 + 0] - c[0]);
                d = d + fabsf(x[4 * j4 + 1] - c[1]);
                d = d + fabsf(x[4 * j4 + 2] - c[2]);
                d = d + fabsf(x[4 * j4 + 3] - c[3]);
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

template <int MB>
hipError_t l1_launch_mb(const StepArgs &a, const L1Plan &pl, hipStream_t s)
{
    auto kern = lloyd_l1_kernel<MB>;
    static const size_t st = static_lds_bytes(reinterpret_cast<const void *>(kern));
    if (st > (size_t)kMaxLds || st + pl.lds_bytes > (size_t)kMaxLds)
        return hipErrorInvalidConfiguration;
    hipExtLaunchKernelGGL(kern, dim3(pl.groups), dim3(pl.waves * kWave), pl.lds_bytes, s,
                          a.ev_start, a.ev_stop, 0, a.X, a.n, a.M, a.C, a.K, a.labels, a.min_d2,
                          a.ctl, a.t, a.fixed, a.force64);
    return hipGetLastError();
}

}  // namespace

L1Plan plan_l1(int64_t n, int M, int K)
{
    L1Plan pl{};
    const size_t cen = (size_t)K * l1_padded(M) * sizeof(float);
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
    switch (l1_padded(a.M)) {
    case 4: return l1_launch_mb<4>(a, pl, s);
    case 8: return l1_launch_mb<8>(a, pl, s);
    case 16: return l1_launch_mb<16>(a, pl, s);
    case 32: return l1_launch_mb<32>(a, pl, s);
    case 64: return l1_launch_mb<64>(a, pl, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace lloyd
