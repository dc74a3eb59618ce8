// Algorithm 2 steps 1-2 (the two steps the paper's GPU regime, Algorithm 4,
// sends to the GPU): the centre of gravity C of the whole set, and the
// diameter of Eq. (3) -- the pair of objects with the largest distance.
//
// Centre of gravity: X read as a flat array of n*M floats by G workgroups of
// T threads, T a multiple of M, so that thread t always meets feature t mod M;
// each thread keeps one fp64 sum, each workgroup adds its threads' sums per
// feature in ascending thread order, and one workgroup adds the G rows in
// ascending order and rounds fp32(sum / n). Every addition's order depends
// only on the shape.
//
// Diameter, squared: D2 = max over pairs k < l of |x_k - x_l|^2, with the
// lexicographically smallest pair reaching it. The all-pairs distances are a
// Gram matrix (a dense contraction over the features), formed on the bf16
// matrix cores in split precision, then made exact:
//   prep    y_i = fl(x_i - C) (centring keeps the norms, and so the error
//           bound, small against D2), n_i = fl(|y_i|^2); operand rows
//             a_i = [-2 y_i, 1, n_i, 0 ...],  b_j = [y_j, n_j, 1, 0 ...]
//           (P = 32 ceil((M+2)/32) features) so that a_i . b_j =
//           n_i + n_j - 2 y_i.y_j ~ |x_i - x_j|^2 with no epilogue
//           arithmetic; each operand value v is split into bf16 hi = bf16(v)
//           and lo = bf16(v - hi), both rounded to nearest, and stored in the
//           matrix instruction's lane order;
//   pass 1  every pair block is three v_mfma_f32_16x16x32_bf16 per 32
//           features (lo.hi, hi.lo, hi.hi), exact products summed in fp32;
//           the maximum approximate value d~* over all pairs is kept (integer
//           atomic max of an order-preserving key: order-free), and each
//           work item's own maximum goes to its result slot;
//   pass 2  items whose maximum is below the threshold d~* - 2B write an
//           empty result at once; the others form the same products again,
//           and every pair k < l with d~ >= d~* - 2B is re-evaluated in fp64
//           in the fixed operation order
//           e = x_j - c_j, d = d + e*e (features ascending, each operation
//           rounded) and the lexicographic best (largest d, then lowest k,
//           then lowest l) is kept.
// B bounds |d~ - d| for every pair: with u = 2^-24, gamma_m = m u / (1 - m u)
// for this code's own round-to-nearest fp32 arithmetic and
// phi_m = 2 m u / (1 - 2 m u) for the matrix core's additions (assumed only
// faithful: each within 2^-23 relative, in any order or direction),
//   |d~ - d| <= E (|y_k|^2 + |y_l|^2),
//   E = 4.01 u (centring) + 4.03 * 2^-16 (dropped split terms, three per
//       feature at most 3.02 * 2^-16 |a b|, and 2^-16 for each norm operand)
//       + 1.01 gamma_M (the fp32 norms) + 2.02 phi_{3P+2} (the sums),
// so B = 1.25 * 2.02 * E * max_i n_i covers every pair (1.25: margin). The
// true pair has d~ >= D2 - B >= d~* - 2B, so it is always re-evaluated, and
// the result is exact whatever the split products round to.
//
// Work: pass items are (row block of 512 objects, column chunk of 16384);
// items wholly below the diagonal return at once, and within the diagonal
// chunk the column steps start at the row block. Each of 8 waves holds the A
// operands of 64 rows in registers; the workgroup stages 64 columns of B at a
// time in LDS (row stride padded by 16 bytes so the 16-byte reads of a
// 16-object column block spread over the banks), and each wave forms 4 x 4
// blocks of 16 x 16 pairs per step. The next step's operands are loaded into
// registers while the current step is computed, and written to the other of
// two LDS buffers after it: one barrier per step.
#include "lloyd_device.h"
#include "diameter.h"

#include <cfloat>
#include <climits>

namespace lloyd {

namespace {

typedef float f4v __attribute__((ext_vector_type(4)));

constexpr int kDiamWaves = 8;
constexpr int kDiamThreads = kDiamWaves * kWave;
constexpr int kRowBlock = kDiamWaves * 64;       // objects per item's row block
constexpr int kChunkSteps = 256;                 // 64-column steps per item
constexpr int kChunk = kChunkSteps * 64;         // columns per item
constexpr int kCentroidGroups = 256;

// Order-preserving key of an fp32 value (larger value, larger key).
__device__ inline uint32_t float_key(float v)
{
    const uint32_t b = __float_as_uint(v);
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

__device__ inline float key_float(uint32_t k)
{
    return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}

// ---------------------------------------------------------------------------
// Centre of gravity (Algorithm 2 step 2).

__global__ void __launch_bounds__(1024)
centroid_partial_kernel(const float *__restrict__ X, int64_t total, int M,
                        double *__restrict__ part)
{
    extern __shared__ double csum[];                  // [blockDim.x]
    const int T = blockDim.x;                         // a multiple of M
    const int64_t S = (int64_t)gridDim.x * T;
    double s = 0.0;
    for (int64_t e = (int64_t)blockIdx.x * T + threadIdx.x; e < total; e += S)
        s = s + (double)X[e];
    csum[threadIdx.x] = s;
    __syncthreads();
    if (threadIdx.x < M) {
        double r = 0.0;
        for (int t = threadIdx.x; t < T; t += M) r = r + csum[t];
        part[(int64_t)blockIdx.x * M + threadIdx.x] = r;
    }
}

// Reads the G partial rows; writes the centroid (fp32) and resets the
// counters of the diameter passes.
__global__ void centroid_final_kernel(const double *__restrict__ part, int G, int M, int64_t n,
                                      float *__restrict__ centroid_ws, float *__restrict__ centroid_out,
                                      uint32_t *__restrict__ counters)
{
    for (int j = threadIdx.x; j < M; j += blockDim.x) {
        double s = 0.0;
        for (int g = 0; g < G; ++g) s = s + part[(int64_t)g * M + j];
        const float c = (float)(s / (double)n);
        if (centroid_ws) centroid_ws[j] = c;
        if (centroid_out) centroid_out[j] = c;
    }
    // max norm, key of d~*, non-finite coordinate seen
    if (counters && threadIdx.x < 3) counters[threadIdx.x] = 0;
}

// ---------------------------------------------------------------------------
// Split-precision operands.

template <int KS>
__global__ void __launch_bounds__(256)
diam_prep_kernel(const float *__restrict__ X, int64_t n, int64_t npad, int M,
                 const float *__restrict__ C, uint4 *__restrict__ ah, uint4 *__restrict__ al,
                 uint4 *__restrict__ bh, uint4 *__restrict__ bl, uint32_t *__restrict__ counters)
{
    constexpr int P = 32 * KS;
    __shared__ float smax[256 / kWave];
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    float y[P];
    float nrm = 0.f;
    const bool real = i < n;
    bool finite = true;
#pragma unroll
    for (int f = 0; f < P; ++f) {
        const float x = (real && f < M) ? X[i * M + f] : 0.f;
        finite = finite && fabsf(x) < INFINITY;
        y[f] = (real && f < M) ? x - C[f] : 0.f;
        nrm = nrm + y[f] * y[f];
    }
    // a NaN or an infinite coordinate leaves the diameter undefined: the
    // passes return at once and the result is NaN with the pair (-1, -1)
    if (__ballot(!finite) != 0ull && threadIdx.x % kWave == 0) atomicOr(&counters[2], 1u);
    if (i < npad) {
#pragma unroll
        for (int g = 0; g < 4 * KS; ++g) {
            float av[8], bv[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int f = 8 * g + e;
                float a = -2.0f * y[f], b = y[f];
                if (f == M) { a = 1.0f; b = nrm; }
                if (f == M + 1) { a = nrm; b = 1.0f; }
                if (!real) { a = 0.f; b = 0.f; }
                av[e] = a;
                bv[e] = b;
            }
            uint32_t h[4], l[4];
            split_bf16x8(av, h, l);
            ah[i * (4 * KS) + g] = make_uint4(h[0], h[1], h[2], h[3]);
            al[i * (4 * KS) + g] = make_uint4(l[0], l[1], l[2], l[3]);
            split_bf16x8(bv, h, l);
            bh[i * (4 * KS) + g] = make_uint4(h[0], h[1], h[2], h[3]);
            bl[i * (4 * KS) + g] = make_uint4(l[0], l[1], l[2], l[3]);
        }
    }
    // largest norm of the workgroup, then one order-free atomic max
    float m = nrm;
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
    if (threadIdx.x % kWave == 0) smax[threadIdx.x / kWave] = m;
    __syncthreads();
    if (threadIdx.x == 0) {
        float r = smax[0];
        for (int w = 1; w < (int)(blockDim.x / kWave); ++w) r = fmaxf(r, smax[w]);
        atomicMax(&counters[0], __float_as_uint(r));          // r >= 0: bits order like values
    }
}

// ---------------------------------------------------------------------------
// The two all-pairs passes.

__device__ inline bool diam_better(double d, int k, int l, double bd, int bk, int bl_)
{
    return d > bd || (d == bd && (k < bk || (k == bk && l < bl_)));
}

// Threshold of pass 2: d~* - 2B, rounded down to fp32; minus infinity (every
// pair re-evaluated in fp64) when the largest norm is so large that an fp32
// pair value may overflow (a value is at most 4 max n_i), where the bound no
// longer holds.
template <int KS>
__device__ inline float diam_threshold(const uint32_t *counters, int M)
{
    constexpr int P = 32 * KS;
    const double u = 5.9604644775390625e-8;           // 2^-24
    auto gamma = [&](int m) { return m * u / (1.0 - m * u); };
    auto phi = [&](int m) { return 2.0 * m * u / (1.0 - 2.0 * m * u); };
    const double E = 4.01 * u + 4.03 * 1.52587890625e-05 + 1.01 * gamma(M) + 2.02 * phi(3 * P + 2);
    const double maxn = (double)__uint_as_float(counters[0]);
    if (!(4.0 * maxn < (double)FLT_MAX)) return -INFINITY;
    const double B = 1.25 * 2.02 * E * maxn;
    const double thr = (double)key_float(counters[1]) - 2.0 * B;
    float t = (float)thr;
    if ((double)t > thr) t = nextafterf(t, -INFINITY);
    return t;
}

// fp64 squared distance of objects i and j in the fixed operation order (the
// rare exact re-evaluation of pass 2, kept out of line so that the matrix
// loop's registers are not sized for it).
__device__ __attribute__((noinline)) double diam_exact_d2(const float *__restrict__ X, int M,
                                                          int64_t i, int64_t j)
{
    const float *xi = X + i * M, *xj = X + j * M;
    double d = 0.0;
    for (int f = 0; f < M; ++f) {
        const double e = (double)xi[f] - (double)xj[f];
        const double sq = e * e;
        d = d + sq;
    }
    return d;
}

template <int KS, bool kExact>
__device__ __forceinline__ void
diam_pass_body(const uint4 *__restrict__ ah, const uint4 *__restrict__ al,
               const uint4 *__restrict__ bh, const uint4 *__restrict__ bl, int64_t n,
               int64_t nsteps_total, const float *__restrict__ X, int M,
               uint32_t *__restrict__ counters, DiamBest *__restrict__ slots)
{
    constexpr int G4 = 4 * KS;                        // 16-byte groups per operand row
    constexpr int kLdsRow = G4 + 1;                   // uint4 per LDS row (16 bytes padding)
    constexpr int kQuads = 64 * G4;                   // 16-byte groups per step and array
    constexpr int kPer = 2 * kQuads / kDiamThreads;   // groups each thread copies (= KS)
    static_assert(2 * kQuads == kPer * kDiamThreads, "copy split");
    // two buffers (the step computed and the step being staged), hi and lo
    __shared__ uint4 sb[2][2][64 * kLdsRow];
    __shared__ float wmax[kDiamWaves];
    __shared__ DiamBest wbest[kDiamWaves];

    if (counters[2] != 0u) return;                    // non-finite input (uniform)
    const int lane = threadIdx.x % kWave, w = threadIdx.x / kWave;
    const int64_t I0 = (int64_t)blockIdx.x * kRowBlock;
    const int64_t J0 = (int64_t)blockIdx.y * kChunk;
    const int64_t slot = (int64_t)blockIdx.y * gridDim.x + blockIdx.x;
    const int64_t s_lo = (J0 > I0 ? J0 : I0) / 64;    // first 64-column step
    int64_t s_hi = (J0 + kChunk) / 64;
    if (s_hi > nsteps_total) s_hi = nsteps_total;
    if (s_lo >= s_hi) {                               // wholly below the diagonal or past n
        if (threadIdx.x == 0) slots[slot] = DiamBest{kExact ? -1.0 : -INFINITY, INT_MAX, INT_MAX};
        return;
    }

    float thr = 0.f;
    if constexpr (kExact) {
        // pass 1 left this item's largest value in its slot: an item with no
        // value at the threshold has no candidate pair
        thr = diam_threshold<KS>(counters, M);
        if (!(slots[slot].d >= (double)thr)) {
            __syncthreads();                          // every thread has read the slot
            if (threadIdx.x == 0) slots[slot] = DiamBest{-1.0, INT_MAX, INT_MAX};
            return;
        }
    }

    // A operands of this wave's 64 rows: 4 row blocks x KS steps of 32 features
    uint32_t a_hi[4][KS][4], a_lo[4][KS][4];
    const int64_t r0 = I0 + 64 * w;
#pragma unroll
    for (int rb = 0; rb < 4; ++rb)
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            const int64_t row = r0 + 16 * rb + lane % 16;
            const uint4 h = ah[row * G4 + ks * 4 + lane / 16];
            const uint4 l = al[row * G4 + ks * 4 + lane / 16];
            a_hi[rb][ks][0] = h.x; a_hi[rb][ks][1] = h.y; a_hi[rb][ks][2] = h.z; a_hi[rb][ks][3] = h.w;
            a_lo[rb][ks][0] = l.x; a_lo[rb][ks][1] = l.y; a_lo[rb][ks][2] = l.z; a_lo[rb][ks][3] = l.w;
        }

    // staging: thread t copies groups q = t + 512 u of the hi array, then the lo array
    uint4 pf[kPer];
    auto fetch = [&](int64_t s) {
#pragma unroll
        for (int u = 0; u < kPer; ++u) {
            const int q = threadIdx.x + kDiamThreads * u;
            const int qq = q < kQuads ? q : q - kQuads;
            pf[u] = (q < kQuads ? bh : bl)[(s * 64 + qq / G4) * G4 + qq % G4];
        }
    };
    auto stage = [&](int buf) {
#pragma unroll
        for (int u = 0; u < kPer; ++u) {
            const int q = threadIdx.x + kDiamThreads * u;
            const int qq = q < kQuads ? q : q - kQuads;
            sb[buf][q < kQuads ? 0 : 1][(qq / G4) * kLdsRow + qq % G4] = pf[u];
        }
    };

    float vmax = -INFINITY;
    double bd = -1.0;
    int bk = INT_MAX, bl_ = INT_MAX;

    fetch(s_lo);
    stage(0);
    __syncthreads();
    for (int64_t s = s_lo; s < s_hi; ++s) {
        const int buf = (int)((s - s_lo) & 1);
        const bool more = s + 1 < s_hi;
        if (more) fetch(s + 1);                       // in flight during this step
        const uint4 *lh = sb[buf][0], *ll = sb[buf][1];

        // the step's 64 columns in two halves of 32 (2 column blocks): with 32
        // accumulator registers per half, 32 features fit 4 waves per SIMD
        // (two workgroups per compute unit)
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            f4v acc[4][2];
#pragma unroll
            for (int rb = 0; rb < 4; ++rb)
#pragma unroll
                for (int cc = 0; cc < 2; ++cc) acc[rb][cc] = f4v{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                // one operand set at a time: the hi parts of B with both parts
                // of A, then the lo parts of B with hi(A)
                uint32_t b[2][4];
#pragma unroll
                for (int cc = 0; cc < 2; ++cc) {
                    const int o = 16 * (2 * half + cc) + lane % 16;
                    const uint4 h = lh[o * kLdsRow + ks * 4 + lane / 16];
                    b[cc][0] = h.x; b[cc][1] = h.y; b[cc][2] = h.z; b[cc][3] = h.w;
                }
#pragma unroll
                for (int rb = 0; rb < 4; ++rb)
#pragma unroll
                    for (int cc = 0; cc < 2; ++cc)
                        acc[rb][cc] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                            as_bf8(a_lo[rb][ks]), as_bf8(b[cc]), acc[rb][cc], 0, 0, 0);
#pragma unroll
                for (int rb = 0; rb < 4; ++rb)
#pragma unroll
                    for (int cc = 0; cc < 2; ++cc)
                        acc[rb][cc] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                            as_bf8(a_hi[rb][ks]), as_bf8(b[cc]), acc[rb][cc], 0, 0, 0);
#pragma unroll
                for (int cc = 0; cc < 2; ++cc) {
                    const int o = 16 * (2 * half + cc) + lane % 16;
                    const uint4 l = ll[o * kLdsRow + ks * 4 + lane / 16];
                    b[cc][0] = l.x; b[cc][1] = l.y; b[cc][2] = l.z; b[cc][3] = l.w;
                }
#pragma unroll
                for (int rb = 0; rb < 4; ++rb)
#pragma unroll
                    for (int cc = 0; cc < 2; ++cc)
                        acc[rb][cc] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                            as_bf8(a_hi[rb][ks]), as_bf8(b[cc]), acc[rb][cc], 0, 0, 0);
            }

            // the largest value of the half in this lane (padding rows and
            // columns give exactly 0, never above a real pair's value by more
            // than the bound; pairs i >= j repeat pairs i < j)
            float smax = -INFINITY;
#pragma unroll
            for (int rb = 0; rb < 4; ++rb)
#pragma unroll
                for (int cc = 0; cc < 2; ++cc)
                    smax = fmaxf(fmaxf(smax, fmaxf(acc[rb][cc][0], acc[rb][cc][1])),
                                 fmaxf(acc[rb][cc][2], acc[rb][cc][3]));
            if constexpr (!kExact) {
                vmax = fmaxf(vmax, smax);
            } else if (__builtin_amdgcn_ballot_w64(!(smax < thr)) != 0) {
                // rare: some pair of this wave's half step reaches the threshold
                const int64_t c0 = s * 64 + 32 * half;
#pragma unroll
                for (int rb = 0; rb < 4; ++rb)
#pragma unroll
                    for (int cc = 0; cc < 2; ++cc)
#pragma unroll
                        for (int r = 0; r < 4; ++r) {
                            const int64_t i = r0 + 16 * rb + 4 * (lane / 16) + r;
                            const int64_t j = c0 + 16 * cc + lane % 16;
                            // (a NaN value, possible only when thr is minus
                            // infinity, is re-evaluated too)
                            if (!(acc[rb][cc][r] < thr) && i < j && j < n) {
                                const double d = diam_exact_d2(X, M, i, j);
                                if (diam_better(d, (int)i, (int)j, bd, bk, bl_)) {
                                    bd = d;
                                    bk = (int)i;
                                    bl_ = (int)j;
                                }
                            }
                        }
            }
        }

        if (more) stage(buf ^ 1);                     // the other buffer: nobody reads it now
        __syncthreads();
    }

    if constexpr (!kExact) {
#pragma unroll
        for (int off = kWave / 2; off > 0; off >>= 1) vmax = fmaxf(vmax, __shfl_xor(vmax, off));
        if (lane == 0) wmax[w] = vmax;
        __syncthreads();
        if (threadIdx.x == 0) {
            float m = wmax[0];
            for (int k = 1; k < kDiamWaves; ++k) m = fmaxf(m, wmax[k]);
            atomicMax(&counters[1], float_key(m));
            slots[slot] = DiamBest{(double)m, INT_MAX, INT_MAX};   // read by pass 2
        }
    } else {
#pragma unroll
        for (int off = kWave / 2; off > 0; off >>= 1) {
            const double d2 = __shfl_xor(bd, off);
            const int k2 = __shfl_xor(bk, off), l2 = __shfl_xor(bl_, off);
            if (diam_better(d2, k2, l2, bd, bk, bl_)) {
                bd = d2;
                bk = k2;
                bl_ = l2;
            }
        }
        if (lane == 0) wbest[w] = DiamBest{bd, bk, bl_};
        __syncthreads();
        if (threadIdx.x == 0) {
            DiamBest b = wbest[0];
            for (int k = 1; k < kDiamWaves; ++k)
                if (diam_better(wbest[k].d, wbest[k].k, wbest[k].l, b.d, b.k, b.l)) b = wbest[k];
            slots[slot] = b;
        }
    }
}

template <int KS, bool kExact>
__global__ void __launch_bounds__(kDiamThreads)
diam_pass_kernel(const uint4 *__restrict__ ah, const uint4 *__restrict__ al,
                 const uint4 *__restrict__ bh, const uint4 *__restrict__ bl, int64_t n,
                 int64_t nsteps_total, const float *__restrict__ X, int M,
                 uint32_t *__restrict__ counters, DiamBest *__restrict__ slots)
{
    diam_pass_body<KS, kExact>(ah, al, bh, bl, n, nsteps_total, X, M, counters, slots);
}

// The lexicographic best of all item slots. With n = 1 there is no pair:
// (0, 0, 0); with a non-finite coordinate in X: (NaN, -1, -1).
__global__ void __launch_bounds__(1024)
diam_final_kernel(const DiamBest *__restrict__ slots, int64_t nslots, int64_t n,
                  const uint32_t *__restrict__ counters, double *__restrict__ d2_out,
                  int32_t *__restrict__ pair_out)
{
    if (counters[2] != 0u) {
        if (threadIdx.x == 0) {
            *d2_out = __builtin_nan("");
            pair_out[0] = -1;
            pair_out[1] = -1;
        }
        return;
    }
    __shared__ DiamBest wb[1024 / kWave];
    double bd = -1.0;
    int bk = INT_MAX, bl_ = INT_MAX;
    for (int64_t s = threadIdx.x; s < nslots; s += blockDim.x) {
        const DiamBest b = slots[s];
        if (diam_better(b.d, b.k, b.l, bd, bk, bl_)) {
            bd = b.d;
            bk = b.k;
            bl_ = b.l;
        }
    }
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) {
        const double d2 = __shfl_xor(bd, off);
        const int k2 = __shfl_xor(bk, off), l2 = __shfl_xor(bl_, off);
        if (diam_better(d2, k2, l2, bd, bk, bl_)) {
            bd = d2;
            bk = k2;
            bl_ = l2;
        }
    }
    const int lane = threadIdx.x % kWave, w = threadIdx.x / kWave;
    if (lane == 0) wb[w] = DiamBest{bd, bk, bl_};
    __syncthreads();
    if (threadIdx.x == 0) {
        DiamBest b = wb[0];
        for (int k = 1; k < (int)(blockDim.x / kWave); ++k)
            if (diam_better(wb[k].d, wb[k].k, wb[k].l, b.d, b.k, b.l)) b = wb[k];
        if (n < 2 || b.d < 0.0) b = DiamBest{0.0, 0, n > 1 ? 1 : 0};
        *d2_out = b.d;
        pair_out[0] = b.k;
        pair_out[1] = b.l;
    }
}

template <int KS>
hipError_t diam_launch_ks(const DiameterArgs &a, const DiameterPlan &pl, hipStream_t s)
{
    const dim3 gprep((unsigned)((pl.npad + 255) / 256));
    hipLaunchKernelGGL(diam_prep_kernel<KS>, gprep, dim3(256), 0, s, a.X, a.n, pl.npad, a.M,
                       a.centroid_ws, a.ah, a.al, a.bh, a.bl, a.counters);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const dim3 grid((unsigned)pl.row_blocks, (unsigned)pl.chunks);
    const int64_t nsteps = pl.npad / 64;
    auto pass1 = diam_pass_kernel<KS, false>;
    auto pass2 = diam_pass_kernel<KS, true>;
    hipLaunchKernelGGL(pass1, grid, dim3(kDiamThreads), 0, s, a.ah, a.al, a.bh, a.bl, a.n,
                       nsteps, a.X, a.M, a.counters, a.slots);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(pass2, grid, dim3(kDiamThreads), 0, s, a.ah, a.al, a.bh, a.bl, a.n,
                       nsteps, a.X, a.M, a.counters, a.slots);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(diam_final_kernel, dim3(1), dim3(1024), 0, s, a.slots,
                       (int64_t)pl.row_blocks * pl.chunks, a.n, a.counters, a.d2, a.pair);
    return hipGetLastError();
}

}  // namespace

CentroidPlan plan_centroid(int64_t n, int M)
{
    CentroidPlan pl{};
    pl.threads = (1024 / M) * M;
    const int64_t total = n * M;
    int64_t g = (total + pl.threads - 1) / pl.threads;
    pl.groups = (int)(g < kCentroidGroups ? g : kCentroidGroups);
    return pl;
}

hipError_t launch_centroid(const float *X, int64_t n, int M, double *part, float *centroid_ws,
                           float *centroid_out, uint32_t *counters, const CentroidPlan &pl,
                           hipStream_t s)
{
    hipLaunchKernelGGL(centroid_partial_kernel, dim3(pl.groups), dim3(pl.threads),
                       (size_t)pl.threads * sizeof(double), s, X, n * M, M, part);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(centroid_final_kernel, dim3(1), dim3(64), 0, s, part, pl.groups, M, n,
                       centroid_ws, centroid_out, counters);
    return hipGetLastError();
}

DiameterPlan plan_diameter(int64_t n, int M)
{
    DiameterPlan pl{};
    pl.ks = (M + 2 + 31) / 32;
    pl.npad = (n + kChunk - 1) / kChunk * kChunk;
    pl.row_blocks = (n + kRowBlock - 1) / kRowBlock;
    pl.chunks = pl.npad / kChunk;
    return pl;
}

hipError_t launch_diameter(const DiameterArgs &a, const DiameterPlan &pl, hipStream_t s)
{
    switch (pl.ks) {
    case 1: return diam_launch_ks<1>(a, pl, s);
    case 2: return diam_launch_ks<2>(a, pl, s);
    case 3: return diam_launch_ks<3>(a, pl, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace lloyd
