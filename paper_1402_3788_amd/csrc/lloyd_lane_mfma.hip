// Fused assign + accumulate for K <= 64, M <= 32: one 64-object tile per
// wavefront at a time, the scores on the bf16 matrix cores in one, two or four
// 16-centre blocks (KB), and every tile read from global memory twice -- once
// in the matrix operand layout and once in the accumulation layout -- so that
// the cache does the transpose and LDS holds nothing but the fp64 sums (and,
// for KB > 1, the centre operands).
//
// Per tile q (objects 64q .. 64q+63) a wave does:
//   1. operand loads (issued one tile ahead): lane (g, o) = (lane / 16,
//      lane % 16) reads features 8g .. 8g+7 of object 16b + o of the tile for
//      each 16-object block b = 0..3 -- two 16-byte loads per block, each
//      starting at any float of a row (rows of M floats) and reading at most
//      three floats into the next row, which the zero A operands past M ignore;
//   2. accumulation loads, issued right after the operand loads of the same
//      tile so that both meet the same cache lines in flight (X crosses HBM
//      and L2 once): lane (h, j) = (lane / 32, lane % 32) reads feature j of
//      32 objects of the tile (s + 32h with two slabs, 2s + h with one);
//   3. scores (Algorithm 1 steps 2/4, Eq. (2) in the expanded form
//      score = |c|^2 - 2 x.c, |x|^2 being common to all centres): per centre
//      block A = -2C (16 centres x 32 features, zero past K and M) and B = X^T,
//      both split into bf16 hi and lo parts rounded to nearest, three
//      v_mfma_f32_16x16x32_bf16 per object block (lo(A) hi(B) + hi(A) lo(B) +
//      hi(A) hi(B)) on top of |c|^2; lane (g, o) gets the scores of centres
//      16cb + 4g .. 16cb + 4g + 3 for object o of every object block;
//   4. the label: each score becomes a packed key (its low 4, 5 or 6 bits
//      replaced by the centre's index), each lane keeps the best and
//      second-best key of each object block over the centre blocks, and two
//      rounds of row swaps (v_permlane32_swap, then v_permlane16_swap) leave
//      lane l with the two best keys of object l; a label is accepted when the
//      two differ by more than twice the proven error bound thr/2. Otherwise
//      (a close call) the keys of the object's column are formed again from
//      the same split operands, every centre whose key is within thr of the
//      best becomes a candidate (no other centre can be the nearest), and the
//      object is decided among its candidates with fp64 distances in the
//      reference operation order (lowest index on ties): one close object at
//      a time, its features made wave-uniform, lane k computing the distance
//      to centre k from an LDS copy of the centres, so that no memory read
//      of the close path waits behind the next tile's loads. Every label is
//      the exact-arithmetic argmin;
//   5. accumulation (the numerator and denominator of Eq. (1)): lane l
//      writes the slab row offset of object l to the wave's offset table;
//      lanes (h, .) read the offsets of their 32 objects back with broadcast
//      16-byte reads, and in step s lane (h, j) adds feature j of its object
//      of the step with an LDS fp64 add. With two slabs per wave (KB <= 2) the
//      halves of a tile add to different slabs and the lanes of a half to
//      different columns, so no two lanes of one add meet on an address; with
//      one slab (KB = 4, whose eight waves' slabs would not fit twice) the
//      objects 2s and 2s + 1 of a step meet on an address when they share a
//      cluster, and the LDS applies the lanes of an add in ascending order. So
//      every sum is formed in a fixed order: objects of the wave's tiles in
//      ascending order per slab. Counts are integer LDS adds (order-free).
// At the end the workgroup adds its slabs in a fixed order (waves, then
// slabs) and writes one fp64 partial per (cluster, feature) and one count per
// cluster; a second launch forms the centres (lloyd_centres.hip).
//
// Error bound of a score (why the label test is safe): with a = -2c_j and
// b = x_j split as a = ah + al + ea (|ea| <= 2^-16 |a|, |al| <= 2^-8 (1+2^-8)|a|)
// and likewise b, the dropped terms ah eb + al bl + ea b are below
// 3.02 * 2^-16 |a b| per feature, and sum_j |a_j b_j| <= |c|^2 + |x|^2. The
// bf16 products are exact in fp32. The matrix core adds the 96 products and
// the |c|^2 seed in some order with at most 98 roundings; the bound assumes
// only that each rounding is faithful (error below one unit in the last place,
// 2^-23 relative), whatever the order or rounding direction, so the sums err by
// at most 1.01 * 98 * 2^-23 of (|c|^2 + sum |a b|) <= (3|c|^2 + |x|^2). The
// fp32 |c|^2 (eight fused multiply-adds in each of the centre's four lanes,
// then two additions across them) errs by at most 10 * 2^-23 |c|^2.
// A packed key with b index bits moves its score by less than 2^(b-23) of
// the score's magnitude, itself below (1 + E)(3|c|^2 + |x|^2). Together every
// key is within E (3 max|c|^2 + |x|^2) of the exact score with
//     E = 3.02 * 2^-16 + 104 * 2^-23 + 1.01 * 2^(b-23),
// and a label is accepted when the two best keys differ by more than
// 2.02 E (3.02 max|c|^2 + 1.0001 |x|^2) + 1e-30 (the fp32 |x|^2 and max|c|^2
// are themselves within the margins; 1e-30 covers bf16 parts below the normal
// range). |x|^2 here sums the squares of every value the lane group read,
// including the up to seven floats past the object's M features: an upper
// bound, which only widens the band (and makes an object whose neighbour holds
// an infinity or a NaN go to the fp64 path). The same bound makes a close
// call's candidate set complete: a centre whose key exceeds the best key b1 by
// more than thr has an exact score above b1 + thr - e >= b1 + e (e the error
// bound of one key, thr >= 2.02 e), while the best key's centre scores at most
// b1 + e; the 1 % margin keeps that gap far above fp64 rounding, so the fp64
// distances order the candidates as they order all centres.
#include "lloyd.h"
#include "lloyd_device.h"

#include <float.h>
#include <math.h>

#include <array>
#include <type_traits>
#include <utility>

#include "lloyd_parts.h"

namespace lloyd {

namespace {

typedef float f4v __attribute__((ext_vector_type(4)));
// Four floats at any 4-byte-aligned address: rows of X start on any float.
typedef float f4u __attribute__((ext_vector_type(4), aligned(4)));

// Waves per workgroup: two per SIMD. The two register sets of the tile loads
// in flight (operands and accumulation values, 64 registers each) take what a
// third wave would need; measured at K = 16, M = 25, n = 2e6, two waves with
// both loads in flight beat three with the accumulation loads issued a tile
// later (whose lines have by then left the cache).
constexpr int kWaves = 8;
constexpr int kMinWavesPerSimd = 2;   // caps registers at 256 per lane
constexpr int kMaxMLane = 32;         // features: four lane groups of eight
[[maybe_unused]] constexpr int kMaxKLane = 64;   // centres: up to four 16-row A operands

// 16-centre blocks of a launch (1, 2 or 4) and the index bits of its keys.
__host__ __device__ constexpr int lane_blocks(int K) { return K <= 16 ? 1 : K <= 32 ? 2 : 4; }
[[maybe_unused]] __host__ __device__ constexpr int key_bits_of(int KB) { return KB == 1 ? 4 : KB == 2 ? 5 : 6; }
// fp64 slabs per wave: two (the halves of a tile; no two lanes of one add
// meet) while eight waves' worth fit; one for four blocks (the two objects of
// a step then share it, the LDS applying the lanes of one add in order).
__host__ __device__ constexpr int lane_slabs(int KB) { return KB == 4 ? 1 : 2; }

// With more than one 16-centre block the A operands and seeds of the blocks
// (48 bytes per lane and block) live in LDS, read again for every tile,
// instead of in registers.
__host__ __device__ constexpr bool lane_a_in_lds(int KB) { return KB > 1; }

// LDS of a workgroup: with accumulation [W][S][K][M] fp64 slabs, [W][K] int32
// counts and [W][64] int32 slab offsets of the objects of the current tile
// (rounded up to 16 bytes); with distances, the A table [3][KB][64] x 16 bytes
// when there is more than one block, then the centres [K][M] in fp32 (one copy
// per wave with one block, which needs no workgroup barrier, else one for the
// workgroup; read by the fp64 decisions of close calls).
[[maybe_unused]] __host__ __device__ inline size_t lane_acc_bytes(int M, int K, int W)
{
    const int S = lane_slabs(lane_blocks(K));
    return ((size_t)W * S * K * M * 8 + (size_t)W * K * 4 + (size_t)W * kWave * 4 + 15) & ~size_t(15);
}
[[maybe_unused]] __host__ __device__ inline size_t lane_tab_bytes(int K, Mode mode)
{
    const int KB = lane_blocks(K);
    return (mode != kAccumLabels && lane_a_in_lds(KB)) ? (size_t)3 * KB * kWave * 16 : 0;
}
[[maybe_unused]] __host__ __device__ inline size_t lane_lds_bytes(int M, int K, int W, Mode mode)
{
    const size_t acc = mode == kAssign ? 0 : lane_acc_bytes(M, K, W);
    const size_t ctab = mode != kAccumLabels ? (size_t)(lane_blocks(K) == 1 ? W : 1) * K * M * 4 : 0;
    return acc + lane_tab_bytes(K, mode) + ctab;
}

// Object rows after the last row of a tile that the operand loads may touch
// (up to three floats past a row): tiles whose rows have that many successors
// in X take the unguarded loads.
[[maybe_unused]] __host__ __device__ inline int64_t rows_after(int M) { return (3 + M - 1) / M; }

// Comparisons of packed keys (a key is a float whose low bits were replaced by
// an index). Plain floating-point minimum, maximum and median instructions, in
// compiler-visible form: the compiler then also keeps the wait states that a
// matrix instruction still reading an operand register needs before the
// register is overwritten (it cannot do so for inline assembly). Keys of
// finite scores are finite; a score that overflowed sends its object to the
// fp64 path (its |x|^2 bound is infinite), whatever these return for it.
[[maybe_unused]] __device__ inline float key_min(float a, float b) { return __builtin_fminf(a, b); }
[[maybe_unused]] __device__ inline float key_max(float a, float b) { return __builtin_fmaxf(a, b); }
[[maybe_unused]] __device__ inline float key_min3(float a, float b, float c)
{
    return __builtin_fminf(__builtin_fminf(a, b), c);
}
[[maybe_unused]] __device__ inline float key_med3(float a, float b, float c)
{
    return __builtin_amdgcn_fmed3f(a, b, c);
}

// Best and second best of two (best, second) key pairs.
[[maybe_unused]] __device__ inline void key_merge(float a1, float a2, float b1, float b2, float &m1, float &m2)
{
    m1 = key_min(a1, b1);
    m2 = key_med3(a1, b1, key_min(a2, b2));
}

// The row swaps below exchange two registers at once: v_permlane32_swap(x, y)
// gives lanes 0-31 the y of lane l+32 in place of their y, and lanes 32-63 the
// x of lane l-32 in place of their x; v_permlane16_swap does the same between
// even and odd 16-lane rows. With x = column c and y = column c + 2 (c + 1),
// each lane ends with both lanes' values of the one column it keeps: the
// lower half (even rows) column c, the upper half (odd rows) column c + 2
// (c + 1), one in x and one in y.
[[maybe_unused]] __device__ inline void swap32(float &x, float &y)
{
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(y),
                                                    false, false);
    x = __uint_as_float(r[0]);
    y = __uint_as_float(r[1]);
}
[[maybe_unused]] __device__ inline void swap16(float &x, float &y)
{
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(y),
                                                    false, false);
    x = __uint_as_float(r[0]);
    y = __uint_as_float(r[1]);
}

// (best, second) keys of object `lane` from the per-block keys (k1[b], k2[b])
// of the four lanes l16 + 16g that hold its centre rows (lane 16b + l16 owns
// object 16b + l16 of the tile): a swap with lane l ^ 32 and a merge keep
// blocks {0, 1} in the lower half and {2, 3} in the upper half, then a swap
// with lane l ^ 16 and a merge keep the lane's own block. Keys of different
// centres never compare equal, so the merge order does not matter.
[[maybe_unused]] __device__ inline void own_block_keys(float (&k1)[4], float (&k2)[4], float &b1, float &b2)
{
    float m1[2], m2[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        swap32(k1[i], k1[2 + i]);
        swap32(k2[i], k2[2 + i]);
        key_merge(k1[i], k2[i], k1[2 + i], k2[2 + i], m1[i], m2[i]);
    }
    swap16(m1[0], m1[1]);
    swap16(m2[0], m2[1]);
    key_merge(m1[0], m2[0], m1[1], m2[1], b1, b2);
}

// The same exchange for the per-block partial sums of |x|^2 (fp32 addition
// is commutative, so both lanes of a pair form the same sums).
[[maybe_unused]] __device__ inline float own_block_sum(float (&p)[4])
{
    swap32(p[0], p[2]);
    swap32(p[1], p[3]);
    float m0 = p[0] + p[2], m1 = p[1] + p[3];
    swap16(m0, m1);
    return m0 + m1;
}

// Bitwise or of x over the four lanes l16 + 16g (g = 0..3), in each of them:
// a row swap returns, in every lane, the values of both lanes of its pair.
[[maybe_unused]] __device__ inline uint32_t or_rows(uint32_t x)
{
    const auto a = __builtin_amdgcn_permlane32_swap(x, x, false, false);
    x = a[0] | a[1];
    const auto b = __builtin_amdgcn_permlane16_swap(x, x, false, false);
    return b[0] | b[1];
}

template <int M, int MODE, int KB>
__global__ void __launch_bounds__(kWaves * kWave, kMinWavesPerSimd)
lane_mfma_kernel(const float *__restrict__ X, int64_t n, const float *__restrict__ C, int K,
                 int32_t *__restrict__ labels, const int32_t *__restrict__ labels_in,
                 float *__restrict__ min_d2, double *__restrict__ part_sums,
                 int32_t *__restrict__ part_counts, Ctl *__restrict__ ctl, int t, int fixed,
                 int force64)
{
    static_assert(M >= 1 && M <= kMaxMLane, "feature count");
    static_assert(KB == 1 || KB == 2 || KB == 4, "centre blocks");
    constexpr bool kAcc = MODE != kAssign;
    constexpr bool kDist = MODE != kAccumLabels;
    constexpr int S = lane_slabs(KB);          // fp64 slabs per wave
    constexpr int kBits = key_bits_of(KB);     // index bits of a packed key
    // With more than one block the operand loads of the next tile go into the
    // registers of the current one once it is split (one register set), which
    // leaves room for the A operands of the other blocks.
    constexpr bool kOneOpSet = KB > 1;
    // With four blocks a tile's distance work is long enough to cover a read
    // that hits the cache: the accumulation values of a tile are loaded at the
    // start of its own step, before the next tile's operand loads (so waiting
    // for them does not wait for those), in one register set instead of two.
    constexpr bool kLateAcc = KB == 4 && MODE == kAssignAccum;
    extern __shared__ __align__(16) unsigned char smem[];
    const int W = blockDim.x / kWave;
    // wave-uniform (scalar) wave index, so that tile addresses are scalar
    // bases with 32-bit lane offsets
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int lane = threadIdx.x % kWave;
    const int g = lane >> 4, o16 = lane & 15;     // matrix layout
    const int h = lane >> 5, j = lane & 31;       // accumulation layout

    if (MODE == kAssignAccum && stop_before(ctl, t, fixed)) return;
    if (MODE == kAccumLabels && stop_after_assign(ctl, fixed)) return;

    double *slabs = reinterpret_cast<double *>(smem) + (size_t)wave * S * K * M;
    int32_t *cnts = reinterpret_cast<int32_t *>(reinterpret_cast<double *>(smem) +
                                                (size_t)W * S * K * M) + wave * K;
    int32_t *offs = reinterpret_cast<int32_t *>(reinterpret_cast<double *>(smem) +
                                                (size_t)W * S * K * M) + W * K + wave * kWave;
    if (kAcc) {
        for (int i = lane; i < S * K * M; i += kWave) slabs[i] = 0.0;
        for (int i = lane; i < K; i += kWave) cnts[i] = 0;
    }

    // A operands for the whole launch: for block cb, lane (g, o) holds
    // -2 c_{16cb+o}, features 8g .. 8g+7 (zero past K and M), split into bf16
    // hi and lo, and the accumulator seeds |c_k|^2 of centres k = 16cb + 4g ..
    // 16cb + 4g + 3 (the largest finite float past K, so padding centres never
    // win and their keys stay finite). The centre values are loaded first and
    // the first tile's loads right after them, so that both are in flight
    // together; |c|^2 is formed from the same registers (eight fused
    // multiply-adds per lane, then the four lanes of a centre added pairwise).
    constexpr bool kALds = kDist && lane_a_in_lds(KB);
    uint32_t ah[KB][4], al[KB][4];
    f4v cseed[KB];
    float cmax = 0.f;
    float craw[KB][8];
    if (kDist) {
#pragma unroll
        for (int cb = 0; cb < KB; ++cb) {
            const int ko = 16 * cb + o16;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int f = 8 * g + e;
                craw[cb][e] = (ko < K && f < M) ? C[ko * M + f] : 0.f;
            }
        }
    }
    const int64_t nt = (n + kWave - 1) / kWave;                    // tiles
    int64_t nsafe = (n - rows_after(M)) / kWave;                   // unguarded tiles
    if (nsafe < 0) nsafe = 0;
    const int64_t stride = (int64_t)gridDim.x * W;
    const int64_t q0 = (int64_t)wave * gridDim.x + blockIdx.x;

    // operand loads of tile q (unguarded: q < nsafe). Chunk starts are
    // clamped into the row, so a lane group with fewer than eight features
    // left reads some of them twice (harmless: A is zero there, and |x|^2 is
    // an upper bound).
    const int c0 = 8 * g < M ? 8 * g : 0;
    const int c1 = 8 * g + 4 < M ? 8 * g + 4 : c0;
    auto load_ops = [&](int64_t q, f4v (&xb)[4][2]) {
        const float *tb = X + q * (kWave * M);                 // scalar
        const int r0 = o16 * M;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            xb[b][0] = *reinterpret_cast<const f4u *>(tb + (r0 + 16 * b * M + c0));
            xb[b][1] = *reinterpret_cast<const f4u *>(tb + (r0 + 16 * b * M + c1));
        }
    };
    // guarded form for the last tiles: zero past n and past M
    auto load_ops_tail = [&](int64_t q, f4v (&xb)[4][2]) {
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            const int64_t r = q * kWave + 16 * b + o16;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int f = 8 * g + e;
                xb[b][e / 4][e % 4] = (r < n && f < M) ? X[r * M + f] : 0.f;
            }
        }
    };
    const int jr = j < M ? j : M - 1;

    // Accumulation layout: in step s lane (h, j) adds feature j of object
    // s + 32h of the tile into slab h (two slabs), or of object 2s + h (one
    // slab: objects in ascending order, the two of a step meeting on an
    // address only in the LDS's lane order).
    // accumulation values of tile q (the guarded form reads zeros past n)
    auto load_acc = [&](int64_t q, float (&xa)[32], auto tail) {
        constexpr bool kTail = decltype(tail)::value;
        const float *tb = X + q * (kWave * M);                 // scalar
        const int c = (S == 2 ? 32 * h : h) * M + jr;
        constexpr int kObjStride = S == 2 ? 1 : 2;
#pragma unroll
        for (int s = 0; s < 32; ++s) {
            if (kTail) xa[s] = (q * kWave + (S == 2 ? 32 * h : h) + kObjStride * s < n)
                                   ? tb[c + kObjStride * s * M] : 0.f;
            else xa[s] = tb[c + kObjStride * s * M];
        }
    };

    // the first tile's loads, in flight while the centre operands are formed
    constexpr int kOpSets = kOneOpSet ? 1 : 2;
    f4v xb[kOpSets][4][2];
    float xa[kLateAcc ? 1 : 2][32];
    int64_t q = q0;
    if (q < nsafe) {
        if (kDist) load_ops(q, xb[0]);
        if (kAcc && !kLateAcc) load_acc(q, xa[0], std::false_type{});
    }

    // the A table in LDS: [hi | lo | seeds][KB][64 lanes], 16 bytes each; then
    // the centres, [K][M] fp32 (the wave's own copy with one block)
    uint4 *atab = reinterpret_cast<uint4 *>(smem + (kAcc ? lane_acc_bytes(M, K, W) : 0));
    float *ctab_w = reinterpret_cast<float *>(smem + (kAcc ? lane_acc_bytes(M, K, W) : 0) +
                                              lane_tab_bytes(K, (Mode)MODE)) +
                    (kALds ? 0 : wave * K * M);
    if (kDist) {
#pragma unroll
        for (int cb = 0; cb < KB; ++cb) {
            float a[8];
            float nrm = 0.f;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                a[e] = -2.0f * craw[cb][e];
                nrm = __builtin_fmaf(craw[cb][e], craw[cb][e], nrm);
            }
            split_bf16x8(a, ah[cb], al[cb]);
            // |c_{16cb+o}|^2 in every lane (g, o): (p0 + p1) + (p2 + p3)
            nrm = nrm + __shfl_xor(nrm, 16, kWave);
            nrm = nrm + __shfl_xor(nrm, 32, kWave);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int k = 16 * cb + 4 * g + r;
                const float nk = __shfl(nrm, 4 * g + r, kWave);
                cseed[cb][r] = k < K ? nk : FLT_MAX;
                if (k < K) cmax = fmaxf(cmax, nk);
            }
            if (!kALds || wave == 0) {
                const int ko = 16 * cb + o16;
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    if (ko < K && 8 * g + e < M) ctab_w[ko * M + 8 * g + e] = craw[cb][e];
            }
            if (kALds && wave == 0) {
                atab[(0 * KB + cb) * kWave + lane] = make_uint4(ah[cb][0], ah[cb][1], ah[cb][2], ah[cb][3]);
                atab[(1 * KB + cb) * kWave + lane] = make_uint4(al[cb][0], al[cb][1], al[cb][2], al[cb][3]);
                atab[(2 * KB + cb) * kWave + lane] =
                    make_uint4(__float_as_uint(cseed[cb][0]), __float_as_uint(cseed[cb][1]),
                               __float_as_uint(cseed[cb][2]), __float_as_uint(cseed[cb][3]));
            }
        }
        cmax = fmaxf(cmax, __shfl_xor(cmax, 16, kWave));
        cmax = fmaxf(cmax, __shfl_xor(cmax, 32, kWave));
        // the tables are read by other lanes (and, for the shared ones, other
        // waves) from here on
        if (kALds) __syncthreads();
        else __builtin_amdgcn_wave_barrier();
    }
    // block cb's operands and seeds: registers, or the LDS table
    auto a_ops = [&](int cb, uint32_t (&h4)[4], uint32_t (&l4)[4], f4v &seed) {
        if (kALds) {
            const uint4 u = atab[(0 * KB + cb) * kWave + lane];
            const uint4 v = atab[(1 * KB + cb) * kWave + lane];
            const uint4 w = atab[(2 * KB + cb) * kWave + lane];
            h4[0] = u.x; h4[1] = u.y; h4[2] = u.z; h4[3] = u.w;
            l4[0] = v.x; l4[1] = v.y; l4[2] = v.z; l4[3] = v.w;
            seed[0] = __uint_as_float(w.x); seed[1] = __uint_as_float(w.y);
            seed[2] = __uint_as_float(w.z); seed[3] = __uint_as_float(w.w);
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                h4[e] = ah[cb][e];
                l4[e] = al[cb][e];
            }
            seed = cseed[cb];
        }
    };
    // error bound of a key relative to (3|c|^2 + |x|^2); the last term is the
    // packing of a kBits-bit index into the low bits
    constexpr float kKeyRel = kBits == 4 ? 1.9073486e-06f : kBits == 5 ? 3.8146973e-06f : 7.6293945e-06f;
    constexpr float kE = 3.02f * 1.5258789e-05f + 104.0f * 1.1920929e-07f + 1.01f * kKeyRel;
    constexpr uint32_t kIdxMask = (1u << kBits) - 1u;
    constexpr uint32_t kKeyMask = ~kIdxMask;

    int nfallback = 0;

    // One tile (kTail: the guarded loads and validity tests): xb / xa hold its
    // operand and accumulation values (loaded one tile earlier); the loads of
    // tile qn go into nxt / xan (unguarded form only; with one operand set,
    // nxt is xb itself, loaded once it is split). Every load is unconditional,
    // so the waits count them exactly.
    auto step = [&](int64_t q, f4v (&xb)[4][2], float (&xa)[32], f4v (&nxt)[4][2],
                    float (&xan)[32], int64_t qn, auto tail) {
        constexpr bool kTail = decltype(tail)::value;
        const int64_t i = q * kWave + lane;           // this lane's object
        const bool valid = !kTail || i < n;
        if (!kTail) {
            if (kDist && !kOneOpSet) load_ops(qn, nxt);
            if (kAcc && kLateAcc) load_acc(q, xa, std::false_type{});
            else if (kAcc) load_acc(qn, xan, std::false_type{});
        }
        int lab = 0;
        if (kDist) {
            uint32_t bh[4][4], bl[4][4];
            float xp[4];
#pragma unroll
            for (int b = 0; b < 4; ++b) {
                float v[8];
                float acc = 0.f;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    v[e] = xb[b][e / 4][e % 4];
                    acc = __builtin_fmaf(v[e], v[e], acc);
                }
                xp[b] = acc;
                split_bf16x8(v, bh[b], bl[b]);
            }
            if (kOneOpSet && !kTail && kDist) load_ops(qn, nxt);
            // per block: three products per 16-object column, then packed
            // keys (low kBits bits replaced by the centre index) folded into
            // the lane's best and second-best key of each column
            float k1[4], k2[4];
            const uint32_t i0 = (uint32_t)(4 * g);
#pragma unroll
            for (int cb = 0; cb < KB; ++cb) {
                uint32_t h4[4], l4[4];
                f4v seed;
                a_ops(cb, h4, l4, seed);
                f4v d[4];
#pragma unroll
                for (int b = 0; b < 4; ++b) d[b] = seed;
#pragma unroll
                for (int b = 0; b < 4; ++b)
                    d[b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf8(l4), as_bf8(bh[b]), d[b], 0, 0, 0);
#pragma unroll
                for (int b = 0; b < 4; ++b)
                    d[b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf8(h4), as_bf8(bl[b]), d[b], 0, 0, 0);
#pragma unroll
                for (int b = 0; b < 4; ++b)
                    d[b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf8(h4), as_bf8(bh[b]), d[b], 0, 0, 0);
#pragma unroll
                for (int b = 0; b < 4; ++b) {
                    float s[4];
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        s[r] = __uint_as_float((__float_as_uint(d[b][r]) & kKeyMask) |
                                               (i0 + (uint32_t)(16 * cb + r)));
                    if (cb == 0) {
                        const float lo01 = key_min(s[0], s[1]), hi01 = key_max(s[0], s[1]);
                        k2[b] = key_min(hi01, key_med3(lo01, s[2], s[3]));
                        k1[b] = key_min3(lo01, s[2], s[3]);
                    } else {
                        // two keys at a time: the second best of the running
                        // pair and the two is min(second, med3(best, a, b))
#pragma unroll
                        for (int r = 0; r < 4; r += 2) {
                            const float n2 = key_min(k2[b], key_med3(k1[b], s[r], s[r + 1]));
                            k1[b] = key_min3(k1[b], s[r], s[r + 1]);
                            k2[b] = n2;
                        }
                    }
                }
            }
            float b1, b2;
            own_block_keys(k1, k2, b1, b2);
            const float xsq = own_block_sum(xp);
            lab = (int)(__float_as_uint(b1) & kIdxMask);
            lab = lab < K ? lab : K - 1;
            const float thr = 2.02f * kE * (3.02f * cmax + 1.0001f * xsq) + 1e-30f;
            const bool ok = !force64 && ((K == 1) || (b2 - b1 > thr));
            float dmin = 0.f;
            const bool close = valid && !ok;
            const uint64_t cmask = __ballot(close);
            if (cmask != 0ull) {
                if (force64) {
                    if (valid) {
                        double bd;
                        lab = argmin_fp64<M>(X + i * M, C, K, bd);
                        dmin = (float)bd;
                    }
                } else {
                    // Close calls: only centres whose key is within thr of the
                    // best key can be the nearest (a key errs by at most half
                    // of thr, so any other centre's exact score exceeds the
                    // best centre's). For each column that holds a close call
                    // the keys are formed again exactly as above from the same
                    // split operands, each lane marks its candidates for the
                    // object of the column, and the four lanes of an object
                    // combine their marks; then the objects are decided one at
                    // a time with fp64 distances (below).
                    const float lim_own = close ? b1 + thr : -INFINITY;
                    // the limits of the four lanes o16 + 16b (b = 0..3) in
                    // every lane: a 32-lane swap leaves rows r and r + 2 in
                    // the lanes of rows r and r + 2 (r = 0, 1), two 16-lane
                    // swaps then rows 0 and 1, and rows 2 and 3
                    float lim4[4];
                    {
                        float lo = lim_own, hi = lim_own;
                        swap32(lo, hi);
                        float r0 = lo, r1 = lo, r2 = hi, r3 = hi;
                        swap16(r0, r1);
                        swap16(r2, r3);
                        lim4[0] = r0;
                        lim4[1] = r1;
                        lim4[2] = r2;
                        lim4[3] = r3;
                    }
                    uint32_t clo = 0u, chi = 0u;
#pragma unroll
                    for (int b = 0; b < 4; ++b) {
                        if (((cmask >> (16 * b)) & 0xffffull) == 0ull) continue;   // uniform
                        const float lim = lim4[b];
                        uint32_t mlo = 0u, mhi = 0u;
#pragma unroll
                        for (int cb = 0; cb < KB; ++cb) {
                            uint32_t h4[4], l4[4];
                            f4v d;
                            a_ops(cb, h4, l4, d);
                            d = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf8(l4), as_bf8(bh[b]), d, 0, 0, 0);
                            d = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf8(h4), as_bf8(bl[b]), d, 0, 0, 0);
                            d = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf8(h4), as_bf8(bh[b]), d, 0, 0, 0);
#pragma unroll
                            for (int r = 0; r < 4; ++r) {
                                const uint32_t idx = i0 + (uint32_t)(16 * cb + r);
                                const float key =
                                    __uint_as_float((__float_as_uint(d[r]) & kKeyMask) | idx);
                                // bit idx - i0 of the word (an immediate), shifted by
                                // i0 below; a centre is ruled out only by a key
                                // above the limit, so a NaN key (a score that
                                // overflowed, or values read past the object's
                                // features that hold an infinity or a NaN) or a NaN
                                // limit keeps every such centre a candidate
                                const uint32_t bit = !(key > lim) ? 1u << (16 * (cb & 1) + r) : 0u;
                                if (cb < 2) mlo |= bit;
                                else mhi |= bit;
                            }
                        }
                        mlo <<= i0;
                        mhi <<= i0;
                        // lane l16 + 16b keeps the marks of its own object
                        mlo = or_rows(mlo);
                        if (KB == 4) mhi = or_rows(mhi);
                        clo = g == b ? mlo : clo;
                        chi = g == b ? mhi : chi;
                    }
                    if (K < 32) clo &= (1u << K) - 1u;      // padding centres never count
                    if (K > 32 && K < 64) chi &= (1u << (K - 32)) - 1u;
                    // The fp64 decisions, one close object at a time: its
                    // features are made wave-uniform (scalars), lane k
                    // computes the distance to centre k if that is one of the
                    // object's candidates (the fp64 sum in the reference
                    // order), and a butterfly over the lanes keeps the
                    // smallest distance, the lowest index on ties. A distance
                    // that is not below infinity (overflow, NaN) never wins,
                    // and with no finite distance the label is 0: what the
                    // ascending scan with a strict comparison gives.
                    uint64_t rem = cmask;
                    while (rem != 0ull) {
                        const int l = (int)__builtin_ctzll(rem);     // uniform
                        rem &= rem - 1ull;
                        float xr[M];
                        if constexpr (kAcc) {
                            // the tile's accumulation registers hold the
                            // object's features (feature f of object l in lane
                            // 32h + f, register s): the register is picked by
                            // selects and read out lane by lane, so that no
                            // memory read waits behind the next tile's loads
                            const int sl = S == 2 ? (l & 31) : (l >> 1);
                            const int hl = S == 2 ? (l >> 5) : (l & 1);
                            float v = xa[0];
#pragma unroll
                            for (int u = 1; u < 32; ++u) v = sl == u ? xa[u] : v;
#pragma unroll
                            for (int f = 0; f < M; ++f)
                                xr[f] = __int_as_float(
                                    __builtin_amdgcn_readlane(__float_as_int(v), 32 * hl + f));
                        } else {
                            const float *xs = X + (q * kWave + l) * M;   // uniform address
#pragma unroll
                            for (int f = 0; f < M; ++f) xr[f] = xs[f];
                        }
                        const uint64_t cand =
                            ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)chi, l) << 32) |
                            (uint32_t)__builtin_amdgcn_readlane((int)clo, l);
                        double dk = INFINITY;
                        if ((cand >> lane) & 1ull) {
                            const double dd = dist_fp64<M>(xr, ctab_w + lane * M);
                            dk = dd < INFINITY ? dd : INFINITY;
                        }
                        int kk = lane;
#pragma unroll
                        for (int m = 1; m < kWave; m <<= 1) {
                            const double od = __shfl_xor(dk, m, kWave);
                            const int ok2 = __shfl_xor(kk, m, kWave);
                            if (od < dk || (od == dk && ok2 < kk)) {
                                dk = od;
                                kk = ok2;
                            }
                        }
                        if (lane == l) {
                            lab = kk;
                            dmin = (float)dk;
                        }
                    }
                }
                if (ctl != nullptr) nfallback += __popcll(cmask);
            }
            if (MODE == kAssign && min_d2 != nullptr && valid && ok) {
                const float *xg = X + i * M;
                const float *c = C + (int64_t)lab * M;
                float dd = 0.f;
#pragma unroll
                for (int f = 0; f < M; ++f) {
                    const float e = xg[f] - c[f];
                    dd = __builtin_fmaf(e, e, dd);
                }
                dmin = dd;
            }
            if (valid) {
                labels[i] = lab;
                if (MODE == kAssign && min_d2 != nullptr) min_d2[i] = dmin;
            }
        } else {
            lab = valid ? labels_in[i] : -1;
            if (lab >= K) lab = -1;
        }
        if (kAcc) {
            const bool adds = valid && lab >= 0;
            // slab row of object `lane`, -1: none; stored where the lanes
            // that add the object read it (entry 32h + s for the object of
            // lane (h, .) in step s)
            const int my_off = adds ? ((S == 2 ? (lane >> 5) : 0) * K + lab) * M : -1;
            const int my_pos = S == 2 ? lane : (lane & 1) * 32 + (lane >> 1);
            if (adds) atomicAdd(cnts + lab, 1);
            // all 32 offsets first (8 broadcast reads), then the adds (each
            // add waits for its broadcast; issued in between they would wait
            // one by one)
            int o[32];
            offs[my_pos] = my_off;
            __builtin_amdgcn_wave_barrier();
            {
                const int4 *src = reinterpret_cast<const int4 *>(offs + 32 * h);
#pragma unroll
                for (int r = 0; r < 8; ++r) {
                    const int4 v = src[r];
                    o[4 * r] = v.x; o[4 * r + 1] = v.y; o[4 * r + 2] = v.z; o[4 * r + 3] = v.w;
                }
            }
            if (j < M) {
#pragma unroll
                for (int s = 0; s < 32; ++s)
                    if ((!kTail && MODE != kAccumLabels) || o[s] >= 0)
                        __hip_atomic_fetch_add(slabs + o[s] + j, (double)xa[s], __ATOMIC_RELAXED,
                                               __HIP_MEMORY_SCOPE_WAVEFRONT);
            }
        }
    };

    // Main loop over the unguarded tiles, the next tile's loads in flight in
    // the other register set (accumulation values; operands too with one
    // block); then the guarded tail tiles.
    // (The prefetch past a wave's last unguarded tile reloads tile nsafe - 1.)
    auto next = [&](int64_t qq) { return qq < nsafe ? qq : nsafe - 1; };
    for (; q < nsafe; q += 2 * stride) {
        step(q, xb[0], xa[0], xb[kOpSets - 1], xa[kLateAcc ? 0 : 1], next(q + stride), std::false_type{});
        if (q + stride >= nsafe) {
            q += stride;
            break;
        }
        step(q + stride, xb[kOpSets - 1], xa[kLateAcc ? 0 : 1], xb[0], xa[0], next(q + 2 * stride),
             std::false_type{});
    }
    for (; q < nt; q += stride) {
        if (kDist) load_ops_tail(q, xb[0]);
        if (kAcc) load_acc(q, xa[0], std::true_type{});
        step(q, xb[0], xa[0], xb[kOpSets - 1], xa[kLateAcc ? 0 : 1], q, std::true_type{});
    }

    if (ctl != nullptr && lane == 0 && nfallback > 0) atomicAdd(&ctl->fallbacks, nfallback);

    if (kAcc) {
        __syncthreads();
        const double *all = reinterpret_cast<const double *>(smem);
        const int32_t *allc = reinterpret_cast<const int32_t *>(all + (size_t)W * S * K * M);
        double *ps = part_sums + (int64_t)blockIdx.x * K * M;
        for (int e = threadIdx.x; e < K * M; e += blockDim.x) {
            double s = 0.0;
            for (int r = 0; r < S * W; ++r) s = s + all[(size_t)r * K * M + e];
            ps[e] = s;
        }
        for (int k = threadIdx.x; k < K; k += blockDim.x) {
            int32_t c = 0;
            for (int w = 0; w < W; ++w) c += allc[w * K + k];
            part_counts[(int64_t)k * gridDim.x + blockIdx.x] = c;
        }
    }
}

template <int M, int KB>
hipError_t launch_mb(const StepArgs &a, Mode mode, const AccumPlan &p, hipStream_t s)
{
    const dim3 grid(p.groups), block(p.waves * kWave);
#define LANE_MFMA_LAUNCH(MD)                                                                   \
    do {                                                                                       \
        auto kern = lane_mfma_kernel<M, MD, KB>;                                               \
        if (p.lds_bytes > (size_t)kMaxLds) return hipErrorInvalidConfiguration;                \
        hipExtLaunchKernelGGL(kern, grid, block, p.lds_bytes, s, a.ev_start, a.ev_stop, 0,     \
                              a.X, a.n, a.C, a.K, a.labels, a.labels_in, a.min_d2,            \
                              a.part_sums, a.part_counts, a.ctl, a.t, a.fixed, a.force64);    \
    } while (0)
    switch (mode) {
    case kAssign: LANE_MFMA_LAUNCH(kAssign); break;
    case kAssignAccum: LANE_MFMA_LAUNCH(kAssignAccum); break;
    case kAccumLabels: LANE_MFMA_LAUNCH(kAccumLabels); break;
    }
#undef LANE_MFMA_LAUNCH
    return hipGetLastError();
}

template <int M>
hipError_t launch_m(const StepArgs &a, Mode mode, const AccumPlan &p, hipStream_t s)
{
    switch (lane_blocks(a.K)) {
    case 1: return launch_mb<M, 1>(a, mode, p, s);
    case 2: return launch_mb<M, 2>(a, mode, p, s);
    default: return launch_mb<M, 4>(a, mode, p, s);
    }
}

using LaunchFn = hipError_t (*)(const StepArgs &, Mode, const AccumPlan &, hipStream_t);

// This translation unit instantiates the kernel for the feature counts of one
// part of [1, kMaxM] that are at most kMaxMLane.
constexpr int kPartLo = LLOYD_PART * kMaxM / LLOYD_PARTS + 1;
constexpr int kPartN = kMaxM / LLOYD_PARTS;

template <int M>
constexpr LaunchFn entry()
{
#ifdef LLOYD_ONLY_M
    if constexpr (M != LLOYD_ONLY_M) return nullptr;
    else
#endif
    if constexpr (M <= kMaxMLane) return &launch_m<M>;
    else return nullptr;
}

template <int... Is>
constexpr auto make_table(std::integer_sequence<int, Is...>)
{
    return std::array<LaunchFn, sizeof...(Is)>{entry<kPartLo + Is>()...};
}

}  // namespace

hipError_t LLOYD_PART_FN(launch_lane_mfma_part)(const StepArgs &a, Mode mode, const AccumPlan &plan,
                                                hipStream_t s)
{
    static constexpr auto table = make_table(std::make_integer_sequence<int, kPartN>{});
    if (a.M < kPartLo || a.M >= kPartLo + kPartN) return hipErrorInvalidValue;
    const LaunchFn fn = table[a.M - kPartLo];
    return fn ? fn(a, mode, plan, s) : hipErrorInvalidValue;
}

#if LLOYD_PART == 0
bool lane_mfma_fits(int M, int K)
{
    return K <= kMaxKLane && M <= kMaxMLane &&
           lane_lds_bytes(M, K, kWaves, kAssignAccum) <= (size_t)kMaxLds;
}

AccumPlan plan_lane_mfma(int64_t n, int M, int K, Mode mode)
{
    AccumPlan p{};
    p.path = kPathLaneMfma;
    int W = kWaves;
    const int64_t nq = (n + kWave - 1) / kWave;
    while (W > 1 && W / 2 >= nq) W /= 2;
    int64_t groups = (nq + W - 1) / W;
    if (groups > kCUs) groups = kCUs;       // one persistent workgroup per compute unit
    p.waves = W;
    p.groups = (int)groups;
    p.accum = 0;
    p.lds_bytes = lane_lds_bytes(M, K, W, mode);
    return p;
}

hipError_t launch_lane_mfma(const StepArgs &a, Mode mode, const AccumPlan &plan, hipStream_t s)
{
    if (a.M < 1 || a.M > kMaxMLane || a.K > kMaxKLane) return hipErrorInvalidValue;
    switch ((a.M - 1) / (kMaxM / LLOYD_PARTS)) {
#define LLOYD_CASE(P) case P: return launch_lane_mfma_part_##P(a, mode, plan, s);
        LLOYD_PART_CASES
#undef LLOYD_CASE
    }
    return hipErrorInvalidValue;
}
#endif

}  // namespace lloyd
