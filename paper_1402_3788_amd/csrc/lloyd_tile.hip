// Fused assign + accumulate with the distances on the matrix cores, 64-object
// tiles against 16-centre blocks (any K).
//
// Expanded form of the squared distance of Eq. (2): for object x and centre c,
//     |x - c|^2 = |x|^2 + score,   score = |c|^2 - 2 x.c,
// and |x|^2 is the same for every centre, so the nearest centre is the one with
// the smallest score. For 16 centres and 16 objects the scores are one matrix
// product D[centre][object] = |c|^2 + sum_j (-2 c_j) x_j with A = -2C (built
// once per workgroup in LDS, in the lane order the instruction wants), B = X^T
// (read from the LDS tile) and the accumulator seeded with |c|^2, in up to
// three stages:
//   pass 1 (every tile): split precision on the bf16 matrix cores, three
//     v_mfma_f32_16x16x32_bf16 per block on operands split into bf16 hi and
//     lo parts rounded to nearest; each score is within E (3|c|^2 + |x|^2) of
//     the exact one (E = 3.02 * 2^-16 + 1.01 (96 ceil(M/32) + 2 + M/6) 2^-23,
//     assuming only that the matrix core rounds each addition faithfully); the
//     scores are scanned as packed (score, index) keys, and a label is
//     accepted when the two best keys differ by more than twice that bound
//     plus the keys' truncation (with |c|^2 bounded by the largest centre
//     norm and margins);
//   pass 2 (tiles with a call too close for pass 1): fp32 products, a
//     v_mfma_f32_16x16x4f32 chain over the features, whose error is bounded by
//     1.01 (4 ceil(M/4) + 3 + M/6) 2^-23 (3|c|^2 + |x|^2) under the same
//     assumption (each product and each addition rounded faithfully); a label
//     is accepted at 2.02 times that;
//   the objects still too close are re-decided with fp64 distances in the
//   fixed operation order, over all centres, lowest index on ties.
//
// Layout of the 16x16 products (64 lanes): D[i][j] is in lane j + 16(i/4),
// register i%4; A[i][k] in lane i + 16k (16x16x4) or lane i + 16(k/8), element
// k%8 (16x16x32), and B[k][j] likewise with j. So every lane holds the scores
// of 4 centres for the four objects it sees in the tile's four 16-object
// columns, and the four lanes that hold an object's centre rows exchange their
// results with row swaps (v_permlane16_swap, v_permlane32_swap).
//
// Each wavefront streams 64-object tiles (in wave-major rounds of the grid):
// the next two tiles' loads are in flight in registers while the current tile
// is staged in the wave's LDS slot; the round with the ragged last tile (n not
// a multiple of 64) is handled after the loop.
//
// Accumulation (the sums of Eq. (1)) has two forms, both with every addition in
// an order fixed by the problem shape (and the hardware's lane order):
//   wave    -- each wavefront adds its own tiles into private fp64 slabs
//              (accumulate_tile: LDS fp64 adds in program order, no barriers),
//              one slab per object of a step, or (when that leaves fewer
//              waves) one slab that the objects of a step share, the LDS
//              applying the lanes of one add in a fixed order; at the end the
//              workgroup adds the slabs in a fixed order. Used while W >= 4
//              waves' private slabs fit in LDS (small K*M).
//   ring    -- one fp64 slab per workgroup that the waves take turns to add
//              their tiles into, in the fixed cyclic order wave 0, 1, ..., W-1
//              of every step (a turn counter in LDS; no barriers): one lane per
//              object, one LDS fp64 add per feature, the LDS applying the lanes
//              of one add in a fixed order. A wave's turn overlaps the other
//              waves' distance work. Used for large K*M.
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

constexpr int kCols = 4;      // 16-object columns per wave tile (64 objects)
// Index bits of a packed key: enough for the (padded) centres, at most 8;
// a group of 2^bits centres shares one running best / second best.
__host__ __device__ inline int key_bits(int KT)
{
    return KT <= 2 ? 5 : KT <= 4 ? 6 : KT <= 8 ? 7 : 8;
}
constexpr int kAccWave = 1;    // per-wave slabs, WaveAcc<M>::Pmax objects per step
constexpr int kAccRing = 2;    // one slab per workgroup, waves add in turn
constexpr int kAccWave1 = 3;   // one slab per wave, WaveAcc<M>::Pmax objects per step (less LDS)
constexpr int kMaxWaves = 8;
[[maybe_unused]] constexpr int kMinWaveForm = 4;   // fewest waves the wave form is used with

// LDS carve-up of a workgroup (dynamic shared memory).
struct MfmaLds {
    size_t abf, cnorm, misc, tiles, offs, slab, total;
    int tile_floats;
};

__host__ __device__ inline size_t al16(size_t v) { return (v + 15) & ~size_t(15); }

// Objects added per accumulation step of a wave form (WaveAcc<M, P>::P).
// Slabs per wave of a wave form.
__host__ __device__ inline int wave_acc_p(int M, int acc)
{
    if (acc == kAccWave1) return 1;
    const int lw = (M + 1 <= 2) ? 2 : (M + 1 <= 4) ? 4 : (M + 1 <= 8) ? 8
                 : (M + 1 <= 16) ? 16 : (M + 1 <= 32) ? 32 : 64;
    return kWave / lw;
}

// Row stride (doubles) of the ring form's slab: the M sums and the count,
// rounded up to an odd count, so that rows of different clusters start on
// different LDS banks (lanes of one add hit rows of arbitrary clusters).
__host__ __device__ constexpr int ring_row(int M) { return (M + 1) | 1; }

// 16-centre blocks, rounded up to an even count (the assignment loop works on
// pairs of blocks; the padding centres score +inf).
__host__ __device__ inline int centre_blocks(int K) { return ((K + 15) / 16 + 1) / 2 * 2; }

__host__ __device__ inline MfmaLds mfma_lds(int M, int K, int W, int acc)
{
    const int KC = (M + 31) / 32, KT = centre_blocks(K);
    MfmaLds L{};
    L.tile_floats = (kWave * M + (M > 4 ? M : 4) + 3) / 4 * 4;    // TileGeom<M>::kSlot
    size_t o = 0;
    L.abf = o;     o = al16(o + (size_t)KT * KC * kWave * 32);
    L.cnorm = o;   o = al16(o + (size_t)KT * 16 * 4);
    L.misc = o;    o = al16(o + 16);
    L.tiles = o;   o = al16(o + (size_t)W * L.tile_floats * 4);
    if (acc == kAccWave || acc == kAccWave1) {
        L.offs = o;    o = al16(o + (size_t)W * kWave * 4);
        L.slab = o;    o = al16(o + (size_t)W * wave_acc_p(M, acc) * K * (M + 1) * 8);
    } else if (acc == kAccRing) {
        L.slab = o;    o = al16(o + (size_t)K * ring_row(M) * 8);
    }
    L.total = o;
    return L;
}

// Turns of the ring form. The counter in LDS holds the number of turns taken
// in the workgroup; wave w's turn of step s is number s*W + w. A wave waits for
// its number with a bounded number of polls (so that every wave finishes even
// if the order were ever broken; the caller reports a wait that gave up), and
// passes the turn on once its LDS adds have completed.
constexpr int kRingPolls = 1 << 22;

__device__ inline bool ring_wait(const uint32_t *turn, uint32_t want)
{
    for (int p = 0; p < kRingPolls; ++p) {
        const uint32_t now = __hip_atomic_load(turn, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        if (__builtin_amdgcn_readfirstlane(now) == want) {
            __atomic_signal_fence(__ATOMIC_SEQ_CST);   // the adds stay after the wait
            return true;
        }
        __builtin_amdgcn_s_sleep(1);
    }
    return false;
}

__device__ inline void ring_pass(uint32_t *turn, uint32_t next)
{
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_waitcnt(0xC07F);        // lgkmcnt(0): this wave's LDS adds are done
    __hip_atomic_store(turn, next, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

template <int M, int MODE, int ACC>
__global__ void __launch_bounds__(kMaxWaves * kWave)
lloyd_tile_kernel(const float *__restrict__ X, int64_t n, const float *__restrict__ C, int K,
                  int32_t *__restrict__ labels, const int32_t *__restrict__ labels_in,
                  float *__restrict__ min_d2, double *__restrict__ part_sums,
                  int32_t *__restrict__ part_counts, Ctl *__restrict__ ctl, int t, int fixed,
                  int force64)
{
    using TG = TileGeom<M>;
    constexpr int KS = (M + 3) / 4;          // 4-feature steps of the fp32 products
    constexpr int KC = (M + 31) / 32;        // 32-feature chunks of the bf16 products
    constexpr int kSlot = TG::kSlot;
    constexpr int V = TG::kVecPerLane;
    constexpr bool kAccum = MODE != kAssign;
    constexpr int kAcc = kAccum ? ACC : 0;
    constexpr bool kWaveForm = kAcc == kAccWave || kAcc == kAccWave1;
    constexpr int PA = 0;                                // most objects per step
    constexpr bool kShared = kAcc == kAccWave1;          // ... into one slab per wave
    constexpr int kP = kShared ? 1 : WaveAcc<M, PA>::P;  // slabs per wave
    extern __shared__ __align__(16) unsigned char smem[];
    const int W = blockDim.x / kWave;
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int tid = threadIdx.x;
    const int KT = centre_blocks(K);       // even
    const int kbits = key_bits(KT);        // index bits of the packed keys

    if (MODE == kAssignAccum && stop_before(ctl, t, fixed)) return;
    if (MODE == kAccumLabels && stop_after_assign(ctl, fixed)) return;

    const MfmaLds L = mfma_lds(M, K, W, kAcc);
    float *tiles = reinterpret_cast<float *>(smem + L.tiles);
    float *tile = tiles + wave * kSlot;
    int32_t *offs = reinterpret_cast<int32_t *>(smem + L.offs) + wave * kWave;
    uint32_t *abf = reinterpret_cast<uint32_t *>(smem + L.abf);
    float *cnorm = reinterpret_cast<float *>(smem + L.cnorm);
    float *s_cmax = reinterpret_cast<float *>(smem + L.misc);
    uint32_t *turn = reinterpret_cast<uint32_t *>(smem + L.misc + 4);
    double *wslabs = reinterpret_cast<double *>(smem + L.slab) + (size_t)wave * kP * K * (M + 1);

    // The grid works in rounds of G*W wave tiles; in round r, wave w of
    // workgroup b takes tile r*G*W + w*G + b. Rounds whose tiles are all full
    // (64 objects present) are streamed in the main loop; the one round after
    // them (the remaining tiles, fewer than G*W, the ragged one included) is
    // handled after it, its tiles going to waves 0, 1, ... of every
    // workgroup. Every workgroup runs the same rounds.
    const int64_t nq = (n + kWave - 1) / kWave;
    const int64_t nfull = n / kWave;
    const int64_t G = gridDim.x;
    const int64_t R = G * W;                   // tiles per round
    const int64_t nr_main = nfull / R;
    const int64_t qw = (int64_t)wave * G + blockIdx.x;   // this wave's tile in round 0

    // the first two tiles' loads go out before the prologue
    float4 buf[2][V];   // register buffers, selected by compile-time index
    if (nr_main > 0) load_tile<M>(X, qw, lane, buf[0]);
    if (nr_main > 1) load_tile<M>(X, R + qw, lane, buf[1]);

    // ---- prologue: split A operands (-2C, bf16 hi and lo, in lane order),
    // centre norms, slabs
    if (MODE != kAccumLabels) {
        for (int idx = tid; idx < KT * KC * kWave; idx += blockDim.x) {
            const int tt = idx / (KC * kWave), qc = (idx / kWave) % KC, l = idx % kWave;
            const int k = tt * 16 + (l & 15), j0 = 32 * qc + 8 * (l >> 4);
            float a[8];
#pragma unroll
            for (int e = 0; e < 8; ++e)
                a[e] = (k < K && j0 + e < M) ? -2.0f * C[(int64_t)k * M + j0 + e] : 0.0f;
            uint32_t hi[4], lo[4];
            split_bf16x8(a, hi, lo);
            uint32_t *dst = abf + (size_t)idx * 8;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                dst[e] = hi[e];
                dst[4 + e] = lo[e];
            }
        }
    }
    {
        constexpr int kSlack = kSlot - kWave * M;     // zeros after each tile
        for (int i = tid; i < W * kSlack; i += blockDim.x)
            tiles[(i / kSlack) * kSlot + kWave * M + (i % kSlack)] = 0.f;
    }
    if (kWaveForm) {
        double *slabs = reinterpret_cast<double *>(smem + L.slab);
        for (int i = tid; i < W * kP * K * (M + 1); i += blockDim.x) slabs[i] = 0.0;
    } else if (kAcc == kAccRing) {
        double *slab = reinterpret_cast<double *>(smem + L.slab);
        for (int i = tid; i < K * ring_row(M); i += blockDim.x) slab[i] = 0.0;
        if (tid == 0) *turn = 0u;
    }
    __syncthreads();
    if (MODE != kAccumLabels) {
        // |c_k|^2 in fp32, features in order
        // padding centres (k >= K) get the largest finite norm: their scores
        // stay finite (a packed key of an infinite score would be a NaN)
        for (int k = tid; k < KT * 16; k += blockDim.x) {
            float nk = FLT_MAX;
            if (k < K) {
                nk = 0.f;
#pragma unroll
                for (int j = 0; j < M; ++j) {
                    const float c = C[(int64_t)k * M + j];
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
    // fp32 error bound of a pass-2 score, relative to (3|c|^2 + |x|^2): 4 KS
    // products and 4 KS + 2 additions on the matrix core, each rounded
    // faithfully (within 2^-23 relative, in any order and direction), and the
    // fp32 |c|^2 (M fused multiply-adds, 2^-24 each, against 3|c|^2); twice
    // that (two scores) with margins
    constexpr float kGuard = 2.02f * 1.01f * ((float)(4 * KS + 3) + (float)M / 6.0f) * 1.1920929e-07f;

    const int g = lane >> 4, l16 = lane & 15;
    int nfallback = 0;
    int nrerun = 0;     // wave tiles that needed the fp32 pass
    uint32_t ring_seq = 0;   // steps taken (ring form)
    bool ring_ok = true;     // every turn wait of this wave succeeded

    // One wave tile: stage it in LDS, put the loads of the tile two strides
    // ahead in flight in the same registers, assign, accumulate.
    // full: a round of the main loop (every wave tile present and full; the
    // loads two rounds ahead are issued here) rather than the last one
    auto step = [&](int64_t r, auto bi, auto full) {
        constexpr bool kFullTile = decltype(full)::value;
        constexpr bool prefetch = kFullTile;
        float4 (&bb)[V] = buf[decltype(bi)::value];
        const int64_t q = r * R + qw;
        const bool have = kFullTile || q < nq;
        if (have) store_tile<M>(tile, lane, bb);
        __builtin_amdgcn_wave_barrier();
        if (prefetch && r + 2 < nr_main) load_tile<M>(X, q + 2 * R, lane, bb);
        const int64_t i = q * kWave + lane;
        const bool valid = kFullTile || (have && i < n);
        int my_lab = -1;

        if (have && MODE == kAccumLabels) {
            if (valid) {
                my_lab = labels_in[i];
                if (my_lab < 0 || my_lab >= K) my_lab = -1;
            }
        } else if (have) {
            // Running best / second best / label of the lane's 4 centres of
            // each column, over the centre blocks; then the four lanes that
            // hold the same object merged (rows r, r^1, r^2), and lane l keeps
            // column l / 16, i.e. object l.
            float b1[kCols], b2[kCols];
            int lb[kCols];
            auto reset = [&]() {
#pragma unroll
                for (int c = 0; c < kCols; ++c) {
                    b1[c] = INFINITY;
                    b2[c] = INFINITY;
                    lb[c] = 0;
                }
            };
            auto scan = [&](int tt, const f4v (&d)[kCols]) {
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
            };
            float mb1, mb2, mx;
            int ml;
            auto finish = [&]() {
#pragma unroll
                for (int c = 0; c < kCols; ++c) {
                    merge_rows<16>(b1[c], b2[c], lb[c]);
                    merge_rows<32>(b1[c], b2[c], lb[c]);
                }
                mb1 = b1[0];
                mb2 = b2[0];
                ml = lb[0];
#pragma unroll
                for (int c = 1; c < kCols; ++c) {
                    const bool mine = g == c;
                    mb1 = mine ? b1[c] : mb1;
                    mb2 = mine ? b2[c] : mb2;
                    ml = mine ? lb[c] : ml;
                }
            };
            // |x|^2 of the lane's own object (row `lane` of the tile), features
            // in order; it enters only the guard bands, whose margins cover its
            // fp32 rounding
            mx = 0.f;
#pragma unroll
            for (int j = 0; j < M; ++j) {
                const float v = tile[lane * M + j];
                mx = __builtin_fmaf(v, v, mx);
            }
            // Both passes keep two accumulator sets and two operand sets: the
            // matrix cores compute one centre block while the vector ALU scans
            // the previous one and the next block's operands arrive.
            // Blocks t0 .. t1-1 (an even count).
            auto blocks = [&](int t0, int t1, auto &oA, auto &oB, auto load_ops, auto chain,
                              auto scan_fn) {
                f4v dA[kCols], dB[kCols];
                load_ops(t0, oA);
                load_ops(t0 + 1, oB);
                chain(oA, dA);
                int tt = t0;
                for (; tt + 2 < t1; tt += 2) {
                    load_ops(tt + 2, oA);
                    chain(oB, dB);
                    scan_fn(tt, dA);
                    load_ops(tt + 3, oB);
                    chain(oA, dA);
                    scan_fn(tt + 1, dB);
                }
                chain(oB, dB);
                scan_fn(tt, dA);
                scan_fn(tt + 1, dB);
            };

            // ---- pass 1: split-precision products on the bf16 matrix cores.
            // B operands: object 16c + l16, features 32q + 8g .. 32q + 8g + 7,
            // split into bf16 hi and lo; A likewise (table in LDS, zero past M).
            // Each centre block is three products per column,
            // lo(A) hi(B) + hi(A) lo(B) + hi(A) hi(B), on top of |c|^2.
            // Past M the A operands are zero, so the B values there only need
            // to be finite: with M >= 16 the tile's zero slack covers the last
            // row's reads past M and the rows are read straight through (the
            // next object's features), else the reads are clamped to the row.
            {
                constexpr bool kClampReads = M < 16;
                uint32_t bh[kCols][KC][4], bl[kCols][KC][4];
#pragma unroll
                for (int c = 0; c < kCols; ++c) {
                    const float *row = tile + (16 * c + l16) * M;
#pragma unroll
                    for (int qc = 0; qc < KC; ++qc) {
                        float v[8];
#pragma unroll
                        for (int e = 0; e < 8; ++e) {
                            const int f = 32 * qc + 8 * g + e;
                            v[e] = kClampReads ? row[f < M ? f : M - 1] : row[f];
                        }
                        split_bf16x8(v, bh[c][qc], bl[c][qc]);
                    }
                }
                struct OpsH {
                    uint32_t ah[KC][4], al[KC][4];
                    f4v c0;
                };
                auto load_h = [&](int tt, OpsH &o) {
#pragma unroll
                    for (int qc = 0; qc < KC; ++qc) {
                        const uint32_t *src = abf + ((size_t)(tt * KC + qc) * kWave + lane) * 8;
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            o.ah[qc][e] = src[e];
                            o.al[qc][e] = src[4 + e];
                        }
                    }
                    o.c0 = *reinterpret_cast<const f4v *>(cnorm + tt * 16 + 4 * g);
                };
                auto chain_h = [&](const OpsH &o, f4v (&d)[kCols]) {
#pragma unroll
                    for (int c = 0; c < kCols; ++c) d[c] = o.c0;
#pragma unroll
                    for (int qc = 0; qc < KC; ++qc) {
#pragma unroll
                        for (int c = 0; c < kCols; ++c)
                            d[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                as_bf8(o.al[qc]), as_bf8(bh[c][qc]), d[c], 0, 0, 0);
#pragma unroll
                        for (int c = 0; c < kCols; ++c)
                            d[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                as_bf8(o.ah[qc]), as_bf8(bl[c][qc]), d[c], 0, 0, 0);
#pragma unroll
                        for (int c = 0; c < kCols; ++c)
                            d[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                as_bf8(o.ah[qc]), as_bf8(bh[c][qc]), d[c], 0, 0, 0);
                    }
                };
                // Scan with packed keys: a score with its low `bits` bits
                // replaced by the centre's index within its group of 2^bits
                // centres, so that min / med3 / min keep the best and second
                // best keys and the label comes with the best one. Per group
                // each lane gathers the keys of its own object from the four
                // lanes that hold its centre rows, and the group folds into
                // the lane's running (best, second, label).
                const int gblocks = (1 << kbits) / 16;            // even
                const uint32_t kmask = ~((1u << kbits) - 1u);
                float g1 = INFINITY, g2 = INFINITY;
                int gl = 0;
                float k1[kCols], k2[kCols];
                int kt0 = 0;
                auto scan_key = [&](int tt, const f4v (&d)[kCols]) {
                    // the four index values of the lane's centre rows, shared
                    // by the four columns; one and-or per key, and per column
                    // two (med3, min3) pairs and a min3 for the running second
                    // best
                    const uint32_t i0 = (uint32_t)((tt - kt0) * 16 + 4 * g);
                    const uint32_t iv[4] = {i0, i0 + 1, i0 + 2, i0 + 3};
#pragma unroll
                    for (int c = 0; c < kCols; ++c) {
                        float sk[4];
#pragma unroll
                        for (int r = 0; r < 4; ++r)
                            sk[r] = __uint_as_float((__float_as_uint(d[c][r]) & kmask) | iv[r]);
                        const float ma = __builtin_amdgcn_fmed3f(k1[c], sk[0], sk[1]);
                        const float b1 = fminf(fminf(k1[c], sk[0]), sk[1]);
                        const float mb = __builtin_amdgcn_fmed3f(b1, sk[2], sk[3]);
                        k1[c] = fminf(fminf(b1, sk[2]), sk[3]);
                        k2[c] = fminf(fminf(k2[c], ma), mb);
                    }
                };
                OpsH oA, oB;
                for (; kt0 < KT; kt0 += gblocks) {
                    const int kt1 = KT - kt0 < gblocks ? KT : kt0 + gblocks;
#pragma unroll
                    for (int c = 0; c < kCols; ++c) {
                        k1[c] = INFINITY;
                        k2[c] = INFINITY;
                    }
                    blocks(kt0, kt1, oA, oB, load_h, chain_h, scan_key);
                    float b1, b2;
                    own_column_keys(k1, k2, lane, b1, b2);
                    const int lab = kt0 * 16 + (int)(__float_as_uint(b1) & ~kmask);
                    const bool take = b1 < g1;
                    g2 = second_of(g1, g2, b1, b2);
                    g1 = take ? b1 : g1;
                    gl = take ? lab : gl;
                }
                mb1 = g1;
                mb2 = g2;
                ml = gl;
            }
            // Error of a pass-1 score against the exact score |c|^2 - 2 x.c:
            // with a = ah + al + ea, b = bh + bl + eb (|ea| <= 2^-16 |a|, |al|
            // <= 2^-8 (1 + 2^-8) |a|, likewise b) the dropped terms
            // (a - ea) eb + al bl + ea b are below 3.02 * 2^-16 |a b| per
            // feature; the products are exact in fp32 and their sums with |c|^2
            // take at most 96 KC + 2 roundings on the matrix core, each assumed
            // only faithful (within 2^-23 relative, any order or direction), so
            // they add (96 KC + 2) 2^-23 of the terms' magnitudes; |c|^2 in fp32
            // adds M 2^-24 |c|^2. With 2|c_j x_j| <= c_j^2 + x_j^2 each score is
            // within E (|x|^2 + 3|c|^2), E = 3.02 * 2^-16 + 1.01 (96 KC + 2 + M/6) 2^-23.
            // A packed key moves its score by less than 2^(bits - 23) of the
            // score's magnitude, itself below (1 + E)(|x|^2 + 3|c|^2). So the
            // label stands when the two best keys differ by more than twice
            // E + 1.01 * 2^(bits - 23) (with margins).
            const float key_rel = __uint_as_float((uint32_t)(127 - 23 + kbits) << 23);   // 2^(bits-23)
            const float e1 = 3.02f * 1.5258789e-05f +
                             1.01f * ((float)(96 * KC + 2) + (float)M / 6.0f) * 1.1920929e-07f +
                             1.01f * key_rel;
            const float thr1 = 2.02f * e1 * (3.02f * cmax + 1.0001f * mx) + 1e-30f;
            bool ok = !force64 && ((K == 1) || (mb2 - mb1 > thr1));

            // ---- pass 2 (tiles with a call too close for pass 1): the fp32
            // products, A = -2C read from C, B = X^T from the tile.
            if (!force64 && __ballot(valid && !ok) != 0) {
                float bop[kCols][KS];
#pragma unroll
                for (int c = 0; c < kCols; ++c) {
                    const float *row = tile + (16 * c + l16) * M + g;
#pragma unroll
                    for (int s = 0; s < KS; ++s) {
                        float v = row[4 * s];
                        if ((M % 4) != 0 && s == KS - 1 && 4 * s + g >= M) v = 0.f;
                        bop[c][s] = v;
                    }
                }
                struct Ops {
                    float a[KS];
                    f4v c0;
                };
                auto load_ops = [&](int tt, Ops &o) {
                    const int k = tt * 16 + l16;
#pragma unroll
                    for (int s = 0; s < KS; ++s) {
                        const int j = 4 * s + g;
                        o.a[s] = (k < K && j < M) ? -2.0f * C[(int64_t)k * M + j] : 0.0f;
                    }
                    o.c0 = *reinterpret_cast<const f4v *>(cnorm + tt * 16 + 4 * g);
                };
                auto chain = [&](const Ops &o, f4v (&d)[kCols]) {
#pragma unroll
                    for (int c = 0; c < kCols; ++c) d[c] = o.c0;
#pragma unroll
                    for (int s = 0; s < KS; ++s)
#pragma unroll
                        for (int c = 0; c < kCols; ++c)
                            d[c] = __builtin_amdgcn_mfma_f32_16x16x4f32(o.a[s], bop[c][s], d[c], 0, 0, 0);
                };
                Ops oA, oB;
                reset();
                blocks(0, KT, oA, oB, load_ops, chain, scan);
                finish();
                const float thr = kGuard * (3.02f * cmax + 1.0001f * mx) + 1e-30f;
                ok = (K == 1) || (mb2 - mb1 > thr);
                if (ctl != nullptr && lane == 0) ++nrerun;
            }
            // a padding centre (index >= K, |c|^2 = FLT_MAX) wins only when
            // every real score overflows; keep such a label in range
            ml = ml < K ? ml : K - 1;
            float dmin = 0.f;
            if (valid && !ok) {
                double bd;
                ml = argmin_fp64<M>(tile + lane * M, C, K, bd);
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

        if (kWaveForm) {
            // (labels read back may be out of range even in a full tile)
            if (have)
                accumulate_tile<M, PA, kFullTile && MODE != kAccumLabels, kShared>(
                    valid ? my_lab : -1, tile, offs, wslabs, K, lane);
        } else if (kAcc == kAccRing) {
            // This wave's turn of the step (every wave takes it, with or
            // without objects): lane l adds object l's features and count to
            // its cluster's row of the workgroup slab. The features are read
            // from the wave's own tile before the wait.
            const bool adds = valid && my_lab >= 0;
            float xv[M];
#pragma unroll
            for (int j = 0; j < M; ++j) xv[j] = tile[lane * M + j];
            const uint32_t want =
                __builtin_amdgcn_readfirstlane(ring_seq * (uint32_t)W + (uint32_t)wave);
            if (ring_ok) ring_ok = ring_wait(turn, want);
            if (adds) {
                constexpr int RS = ring_row(M);
                double *row = reinterpret_cast<double *>(smem + L.slab) + (int64_t)my_lab * RS;
#pragma unroll
                for (int j = 0; j < M; ++j)
                    __hip_atomic_fetch_add(row + j, (double)xv[j], __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_WORKGROUP);
                __hip_atomic_fetch_add(row + M, 1.0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            }
            ring_pass(turn, want + 1);
            ++ring_seq;
        }
    };

    // The register buffers alternate between rounds. Every wave of a
    // workgroup runs the same steps (the ring form needs every wave's turn in
    // every step).
    for (int64_t r = 0; r < nr_main; r += 2) {
        step(r, std::integral_constant<int, 0>{}, std::true_type{});
        if (r + 1 < nr_main) step(r + 1, std::integral_constant<int, 1>{}, std::true_type{});
    }
    if (nr_main * R < nq) {
        const int64_t q = nr_main * R + qw;
        if (q < nfull) load_tile<M>(X, q, lane, buf[0]);
        else if (q < nq) load_tail_tile<M>(X, n, q, lane, buf[0]);
        step(nr_main, std::integral_constant<int, 0>{}, std::false_type{});
    }

    if (ctl != nullptr && lane == 0 && nfallback > 0) atomicAdd(&ctl->fallbacks, nfallback);
    if (ctl != nullptr && lane == 0 && nrerun > 0) atomicAdd(&ctl->reruns, nrerun);
    if (kAcc == kAccRing && ctl != nullptr && lane == 0 && !ring_ok) atomicAdd(&ctl->ring_stalls, 1);

    if (kWaveForm) {
        __syncthreads();
        write_wave_partials<M, PA, kShared>(reinterpret_cast<const double *>(smem + L.slab), W, K,
                               part_sums + (int64_t)blockIdx.x * K * M,
                               part_counts + blockIdx.x, gridDim.x);
    } else if (kAcc == kAccRing) {
        __syncthreads();
        constexpr int RS = ring_row(M);
        const double *slab = reinterpret_cast<const double *>(smem + L.slab);
        double *out = part_sums + (int64_t)blockIdx.x * K * M;
        for (int e = tid; e < K * (M + 1); e += blockDim.x) {
            const int k = e / (M + 1), j = e % (M + 1);
            const double v = slab[k * RS + j];
            if (j < M) out[(int64_t)k * M + j] = v;
            else part_counts[(int64_t)k * gridDim.x + blockIdx.x] = (int32_t)v;
        }
    }
}

template <int M>
hipError_t launch_m(const StepArgs &a, Mode mode, const AccumPlan &p, hipStream_t s)
{
    const dim3 grid(p.groups), block(p.waves * kWave);
#define LLOYD_MFMA_LAUNCH(MD, AC)                                                              \
    do {                                                                                       \
        auto kern = lloyd_tile_kernel<M, MD, AC>;                                              \
        static const size_t st = static_lds_bytes(reinterpret_cast<const void *>(kern));       \
        if (st > (size_t)kMaxLds || st + p.lds_bytes > (size_t)kMaxLds)                        \
            return hipErrorInvalidConfiguration;                                               \
        hipExtLaunchKernelGGL(kern, grid, block, p.lds_bytes, s, a.ev_start, a.ev_stop, 0,     \
                              a.X, a.n, a.C, a.K, a.labels, a.labels_in, a.min_d2,            \
                              a.part_sums, a.part_counts, a.ctl, a.t, a.fixed, a.force64);    \
    } while (0)
    switch (mode) {
    case kAssign: LLOYD_MFMA_LAUNCH(kAssign, 0); break;
    case kAssignAccum:
        if (p.accum == kAccWave) LLOYD_MFMA_LAUNCH(kAssignAccum, kAccWave);
        else if (p.accum == kAccWave1) LLOYD_MFMA_LAUNCH(kAssignAccum, kAccWave1);
        else LLOYD_MFMA_LAUNCH(kAssignAccum, kAccRing);
        break;
    case kAccumLabels:
        if (p.accum == kAccWave) LLOYD_MFMA_LAUNCH(kAccumLabels, kAccWave);
        else if (p.accum == kAccWave1) LLOYD_MFMA_LAUNCH(kAccumLabels, kAccWave1);
        else LLOYD_MFMA_LAUNCH(kAccumLabels, kAccRing);
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

hipError_t LLOYD_PART_FN(launch_tile_part)(const StepArgs &a, Mode mode, const AccumPlan &plan, hipStream_t s)
{
    static constexpr auto table = make_table(std::make_integer_sequence<int, kPartN>{});
    if (a.M < kPartLo || a.M >= kPartLo + kPartN) return hipErrorInvalidValue;
    return table[a.M - kPartLo](a, mode, plan, s);
}

#if LLOYD_PART == 0
AccumPlan plan_tile(int64_t n, int M, int K, Mode mode)
{
    AccumPlan p{};
    p.path = kPathTile;
    const int64_t nq = (n + kWave - 1) / kWave;
    auto fits = [&](int W, int acc) { return mfma_lds(M, K, W, acc).total <= (size_t)kMaxLds; };
    auto most_waves = [&](int acc) {      // 0 when not even one wave fits
        int w = kMaxWaves;
        while (w > 0 && !fits(w, acc)) --w;
        return w;
    };
    int W = kMaxWaves, acc = 0;
    if (mode == kAssign) {
        W = most_waves(0);
    } else {
        // private slabs (the most objects per step that leaves the most waves)
        // while at least kMinWaveForm waves fit, else one shared slab
        const int w_p = most_waves(kAccWave), w_1 = most_waves(kAccWave1);
        if (w_p >= kMinWaveForm && w_p >= w_1) {
            acc = kAccWave;
            W = w_p;
        } else if (w_1 >= kMinWaveForm) {
            acc = kAccWave1;
            W = w_1;
        } else {
            acc = kAccRing;
            W = most_waves(kAccRing);
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

bool tile_fits(int M, int K)
{
    return mfma_lds(M, K, 1, kAccRing).total <= (size_t)kMaxLds;
}

hipError_t launch_tile(const StepArgs &a, Mode mode, const AccumPlan &plan, hipStream_t s)
{
    if (a.M < 1 || a.M > kMaxM) return hipErrorInvalidValue;
    switch ((a.M - 1) / (kMaxM / LLOYD_PARTS)) {
#define LLOYD_CASE(P) case P: return launch_tile_part_##P(a, mode, plan, s);
        LLOYD_PART_CASES
#undef LLOYD_CASE
    }
    return hipErrorInvalidValue;
}
#endif

}  // namespace lloyd
