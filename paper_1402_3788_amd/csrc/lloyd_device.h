// Device helpers shared by the distance kernels: bf16 operand splitting,
// streaming a 64-object tile of X through registers into LDS, the per-wave
// fp64 accumulation of Eq. (1)'s sums, and the fp64 re-decision of close
// calls.
#pragma once

#include "lloyd.h"

#include <math.h>

namespace lloyd {

// ---------------------------------------------------------------------------
// Split-precision operands of the bf16 matrix products (both distance kernels).

typedef __bf16 bf2v __attribute__((ext_vector_type(2)));
typedef float f2v __attribute__((ext_vector_type(2)));

// Two fp32 values rounded to nearest-even bf16 (v_cvt_pk_bf16_f32), packed
// with the first in the low half.
__device__ inline uint32_t bf16x2_rne(float a, float b)
{
    const f2v v = {a, b};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf2v));
}

// Split eight fp32 values v into bf16 parts rounded to nearest: hi = bf16(v),
// lo = bf16(v - hi), the remainder being exact (hi is within a factor 2 of v).
// With the bf16 unit roundoff 2^-8, |v - hi| <= 2^-8 |v| and
// |v - hi - lo| <= 2^-16 |v| (v finite and below the bf16 overflow
// threshold). Parts are packed two per dword, element 2e in the low half of
// dword e, as the bf16 operands of v_mfma_f32_16x16x32_bf16 expect.
__device__ inline void split_bf16x8(const float (&v)[8], uint32_t (&hi)[4], uint32_t (&lo)[4])
{
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const uint32_t h = bf16x2_rne(v[2 * e], v[2 * e + 1]);
        hi[e] = h;
        lo[e] = bf16x2_rne(v[2 * e] - __uint_as_float(h << 16),
                           v[2 * e + 1] - __uint_as_float(h & 0xFFFF0000u));
    }
}

typedef __bf16 bf8v __attribute__((ext_vector_type(8)));

// Four packed dwords as the eight bf16 of a matrix operand.
__device__ inline bf8v as_bf8(const uint32_t (&u)[4])
{
    typedef uint32_t u4v __attribute__((ext_vector_type(4)));
    const u4v w = {u[0], u[1], u[2], u[3]};
    return __builtin_bit_cast(bf8v, w);
}

template <int M>
struct TileGeom {
    static constexpr int kFloats = kWave * M;          // floats per 64-object tile
    static constexpr int kVec = kFloats / 4;           // float4s per tile (64*M divisible by 4)
    static constexpr int kVecPerLane = (kVec + kWave - 1) / kWave;
    // floats per LDS tile slot: the 64 objects, then zeros (at least one full
    // row, and at least 4 floats for the matrix-core operand reads that run
    // past a row)
    static constexpr int kSlot = (kWave * M + (M > 4 ? M : 4) + 3) / 4 * 4;
};

// Issue the loads of full tile q (objects 64q .. 64q+63, all < n) into
// registers: a fixed number of 16-byte loads with no branches, so the compiler
// can count them when it waits for them.
template <int M>
__device__ inline void load_tile(const float *__restrict__ X, int64_t q, int lane,
                                 float4 (&buf)[TileGeom<M>::kVecPerLane])
{
    using G = TileGeom<M>;
    const float4 *src = reinterpret_cast<const float4 *>(X + q * (int64_t)G::kFloats);
#pragma unroll
    for (int v = 0; v < G::kVecPerLane; ++v) {
        // lanes past the tile's last float4 reload it (in bounds; store_tile
        // drops them), so every lane issues every load
        const int idx = lane + kWave * v;
        buf[v] = src[idx < G::kVec ? idx : G::kVec - 1];
    }
}

// Loads of the last, partial tile q (objects 64q .. n-1): floats past the end of
// X read as zero. Used once per launch, outside the streaming loop.
template <int M>
__device__ inline void load_tail_tile(const float *__restrict__ X, int64_t n, int64_t q, int lane,
                                      float4 (&buf)[TileGeom<M>::kVecPerLane])
{
    using G = TileGeom<M>;
    const int64_t f0 = q * (int64_t)G::kFloats;
    const int nf = (int)(n * (int64_t)M - f0);          // floats present, < kFloats
#pragma unroll
    for (int v = 0; v < G::kVecPerLane; ++v) {
        // lanes past the tile's last float4 read that one again, as in load_tile
        const int idx0 = lane + kWave * v;
        const int idx = idx0 < G::kVec ? idx0 : G::kVec - 1;
        float4 r = make_float4(0.f, 0.f, 0.f, 0.f);
        const float *s = X + f0 + 4 * idx;
        if (4 * idx + 0 < nf) r.x = s[0];
        if (4 * idx + 1 < nf) r.y = s[1];
        if (4 * idx + 2 < nf) r.z = s[2];
        if (4 * idx + 3 < nf) r.w = s[3];
        buf[v] = r;
    }
}

// Lanes past the tile's last float4 hold a copy of it (load_tile clamps their
// index) and write it to the same place: every lane stores, with no branch, so
// every load is waited for on every path (a masked store would leave the last
// load's wait to a later, coarser one).
template <int M>
__device__ inline void store_tile(float *tile, int lane,
                                  const float4 (&buf)[TileGeom<M>::kVecPerLane])
{
    using G = TileGeom<M>;
    float4 *dst = reinterpret_cast<float4 *>(tile);
#pragma unroll
    for (int v = 0; v < G::kVecPerLane; ++v) {
        const int idx = lane + kWave * v;
        dst[idx < G::kVec ? idx : G::kVec - 1] = buf[v];
    }
}

// fp64 squared distance in the reference operation order: for j ascending,
// e = x_j - c_j, then d = d + e*e, every operation rounded on its own (this file
// is compiled with -ffp-contract=off, so nothing is fused). xs: the object's M
// features; read per centre so the rare re-decision holds no fp64 copy of the
// object in registers.
template <int M>
__device__ inline double dist_fp64(const float *xs, const float *c)
{
    double d = 0.0;
#pragma unroll
    for (int j = 0; j < M; ++j) {
        const double e = (double)xs[j] - (double)c[j];
        const double sq = e * e;
        d = d + sq;
    }
    return d;
}

// Nearest centre by dist_fp64 over all K centres, lowest index on ties.
template <int M>
__device__ inline int argmin_fp64(const float *xs, const float *__restrict__ C, int K,
                                  double &best_out)
{
    double best = INFINITY;
    int lab = 0;
    for (int k = 0; k < K; ++k) {
        const double d = dist_fp64<M>(xs, C + k * M);
        if (d < best) {
            best = d;
            lab = k;
        }
    }
    best_out = best;
    return lab;
}

// ---------------------------------------------------------------------------
// Cross-lane merges of the matrix-core layouts (both distance kernels). In a
// 16x16 product D[i][j] sits in lane j + 16(i/4), register i%4, so the four
// lanes l16 + 16g (g = 0..3) hold different centre rows of the same objects.

// Second-best of two (best, second) pairs, b1 <= b2 and p1 <= p2:
// min(max(b1, p1), min(b2, p2)).
__device__ inline float second_of(float b1, float b2, float p1, float p2)
{
    return __builtin_amdgcn_fmed3f(b1, p1, fminf(b2, p2));
}

// Merge the (best, second, label) triples of lanes l and l ^ 16 (ROW = 16) or
// l and l ^ 32 (ROW = 32): the row swap returns, in every lane, the triples of
// both lanes of its pair; the merge keeps the lower label on equal scores.
template <int ROW>
__device__ inline void merge_rows(float &b1, float &b2, int &lb)
{
    auto swap = [](uint32_t v) {
        if (ROW == 16) return __builtin_amdgcn_permlane16_swap(v, v, false, false);
        return __builtin_amdgcn_permlane32_swap(v, v, false, false);
    };
    const auto s1 = swap(__float_as_uint(b1));
    const auto s2 = swap(__float_as_uint(b2));
    const auto sl = swap((uint32_t)lb);
    const float f1 = __uint_as_float(s1[0]), g1 = __uint_as_float(s1[1]);
    const float f2 = __uint_as_float(s2[0]), g2 = __uint_as_float(s2[1]);
    const int fl = (int)sl[0], gl = (int)sl[1];
    const bool take = (g1 < f1) | ((g1 == f1) & (gl < fl));
    b2 = second_of(f1, f2, g1, g2);
    b1 = take ? g1 : f1;
    lb = take ? gl : fl;
}

template <int ROW>
__device__ inline float sum_rows(float v)
{
    uint32_t u = __float_as_uint(v);
    const auto s = (ROW == 16) ? __builtin_amdgcn_permlane16_swap(u, u, false, false)
                               : __builtin_amdgcn_permlane32_swap(u, u, false, false);
    return __uint_as_float(s[0]) + __uint_as_float(s[1]);
}

// Packed (best, second) keys of object `lane` (column lane / 16 of the tile's
// 16-object columns) from the per-column keys (k1[c], k2[c]) of the four lanes
// l16 + 16 g' that hold its centre rows. Two exchange stages: with lane l ^ 32
// (the lower half keeps columns 0, 1 and sends 2, 3; the upper half the
// reverse), then with lane l ^ 16 (a lane keeps its own column and sends the
// other); each received pair is merged into the kept one. Keys of different
// centres never compare equal, so the order of a merge does not matter.
__device__ inline void own_column_keys(const float (&k1)[4], const float (&k2)[4], int lane,
                                       float &b1, float &b2)
{
    const bool up = lane >= 32;
    const bool odd = (lane >> 4) & 1;
    // the partner's value out of a swap's pair (see merge_rows)
    auto other32 = [up](uint32_t v) {
        const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
        return __uint_as_float(up ? r[0] : r[1]);
    };
    auto other16 = [odd](uint32_t v) {
        const auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
        return __uint_as_float(odd ? r[0] : r[1]);
    };
    float m1[2], m2[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const float o1 = up ? k1[2 + i] : k1[i], o2 = up ? k2[2 + i] : k2[i];   // kept
        const float s1 = up ? k1[i] : k1[2 + i], s2 = up ? k2[i] : k2[2 + i];   // sent
        const float p1 = other32(__float_as_uint(s1)), p2 = other32(__float_as_uint(s2));
        m2[i] = second_of(o1, o2, p1, p2);
        m1[i] = fminf(o1, p1);
    }
    const float o1 = odd ? m1[1] : m1[0], o2 = odd ? m2[1] : m2[0];
    const float s1 = odd ? m1[0] : m1[1], s2 = odd ? m2[0] : m2[1];
    const float p1 = other16(__float_as_uint(s1)), p2 = other16(__float_as_uint(s2));
    b2 = second_of(o1, o2, p1, p2);
    b1 = fminf(o1, p1);
}


// ---------------------------------------------------------------------------
// Per-wave accumulation of the numerator and denominator of Eq. (1).
//
// A wave owns P fp64 slabs of K rows x (M+1) columns: columns 0..M-1 hold the
// feature sums of a cluster's members and column M their count (adding 1.0
// per member is exact in fp64). The wave's lanes are split into P groups of
// LW = 64 / P >= M+1 lanes; in step s, lane (h, j) adds
// feature j of the tile's object s*P + h into slab h, row label(object). So slab
// h receives the members at tile positions h, h+P, h+2P, ... in ascending
// order, every addition is an LDS fp64 add done in program order, and no two
// lanes of one instruction touch the same address: the sums are deterministic
// and need no barriers.
template <int M, int P_ = 0>
struct WaveAcc {
    static constexpr int MW = M + 1;
    static constexpr int LWmin = (M + 1 <= 2) ? 2 : (M + 1 <= 4) ? 4 : (M + 1 <= 8) ? 8
                               : (M + 1 <= 16) ? 16 : (M + 1 <= 32) ? 32 : 64;
    static constexpr int Pmax = kWave / LWmin;
    static constexpr int P = P_ == 0 ? Pmax : P_;   // objects added per step
    static constexpr int LW = kWave / P;            // lanes per object
    static constexpr int kSteps = kWave / P;
    static_assert(P >= 1 && P <= Pmax && (kWave % P) == 0, "slab count");
};

// P (a power of two, at most 64 / (M+1) rounded down to a power of two; 0 =
// that maximum) trades LDS for steps: P slabs, 64 / P steps per tile.
// lab: this lane's object label (-1: no object). tile: the wave's LDS tile
// (object-major, with at least one float of slack after the 64 rows). offs: 64
// ints of wave-private LDS. slabs: the wave's P slabs (P*K*(M+1) doubles).
// kFull: every object of the tile is present (lab >= 0 in every lane): the
// per-step validity test drops out and the lanes past the count column are
// masked once for the whole tile.
// kShared: the P objects of a step add into one slab instead of P. Two lanes
// of one instruction then meet on a row when their objects share a cluster;
// the slab is the wave's own and the LDS applies the lanes of one instruction
// in a fixed order, so the sums are still reproducible, with 1/P of the LDS.
template <int M, int P_, bool kFull = false, bool kShared = false>
__device__ inline void accumulate_tile(int lab, const float *tile, int32_t *offs, double *slabs,
                                       int K, int lane)
{
    using A = WaveAcc<M, P_>;
    constexpr int MW = A::MW, LW = A::LW, P = A::P;
    // row offset (in doubles) of this lane's object in its slab
    const int slab_of = kShared ? 0 : lane % P;
    offs[lane] = (kFull || lab >= 0) ? (slab_of * K + lab) * MW : -1;
    __builtin_amdgcn_wave_barrier();
    const int h = lane / LW, j = lane % LW;
    const int jr = j < M ? j : M;              // count lanes read a value they ignore
    const float *xp = tile + h * M + jr;
    const int32_t *op = offs + h;
    const bool feat = j < M;
    const bool used = j <= M;
    // Batches of steps: all LDS reads of a batch first, then its adds back to
    // back (an add cannot be hoisted above a read the compiler cannot prove
    // disjoint, so interleaving them would serialise every step on LDS latency).
    constexpr int B = A::kSteps < 16 ? A::kSteps : 16;
    if constexpr (kFull && M + 1 <= kWave) {
        if (used) {
            double *col = slabs + j;
            // 1.0f the optimiser cannot see through (see accumulate_commit)
            float one;
            asm("v_mov_b32 %0, 1.0" : "=v"(one));
#pragma unroll
            for (int s0 = 0; s0 < A::kSteps; s0 += B) {
                int o[B];
                float x[B];
#pragma unroll
                for (int b = 0; b < B; ++b) {
                    o[b] = op[(s0 + b) * P];
                    x[b] = xp[(s0 + b) * P * M];
                }
#pragma unroll
                for (int b = 0; b < B; ++b) {
                    const float v = feat ? x[b] : one;   // the count column adds 1
                    __hip_atomic_fetch_add(col + o[b], (double)v, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_WAVEFRONT);
                }
            }
        }
    } else {
#pragma unroll
        for (int s0 = 0; s0 < A::kSteps; s0 += B) {
            int o[B];
            float x[B];
#pragma unroll
            for (int b = 0; b < B; ++b) {
                o[b] = op[(s0 + b) * P];
                x[b] = xp[(s0 + b) * P * M];
            }
#pragma unroll
            for (int b = 0; b < B; ++b) {
                const double v = (double)(feat ? x[b] : 1.0f);
                if (used && o[b] >= 0)
                    __hip_atomic_fetch_add(slabs + o[b] + j, v, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_WAVEFRONT);
                if (M + 1 > kWave && lane == 0 && o[b] >= 0)   // M = 64: no lane left for the count
                    __hip_atomic_fetch_add(slabs + o[b] + M, 1.0, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_WAVEFRONT);
            }
        }
    }
    __builtin_amdgcn_wave_barrier();
}

// The same accumulation in two parts, so the tile's feature reads (which do
// not depend on the labels) can be issued before the assignment and wait in
// registers: accumulate_fetch reads every step's value for this lane,
// accumulate_commit adds them once the labels are known.
template <int M, int P_>
struct AccFetch {
    float x[WaveAcc<M, P_>::kSteps];
};

template <int M, int P_>
__device__ inline void accumulate_fetch(const float *tile, int lane, AccFetch<M, P_> &f)
{
    using A = WaveAcc<M, P_>;
    constexpr int LW = A::LW, P = A::P;
    const int h = lane / LW, j = lane % LW;
    const float *xp = tile + h * M + (j < M ? j : M);
#pragma unroll
    for (int s = 0; s < A::kSteps; ++s) f.x[s] = xp[s * P * M];
}

// kFull: every object of the tile is present (lab >= 0 in every lane), so the
// per-step validity test drops out and the lanes past the count column are
// masked once for the whole tile.
template <int M, int P_, bool kFull = false>
__device__ inline void accumulate_commit(int lab, const AccFetch<M, P_> &f, int32_t *offs,
                                         double *slabs, int K, int lane)
{
    using A = WaveAcc<M, P_>;
    constexpr int MW = A::MW, LW = A::LW, P = A::P;
    offs[lane] = (kFull || lab >= 0) ? ((lane % P) * K + lab) * MW : -1;
    __builtin_amdgcn_wave_barrier();
    const int h = lane / LW, j = lane % LW;
    const int32_t *op = offs + h;
    const bool feat = j < M;
    const bool used = j <= M;
    constexpr int B = A::kSteps < 16 ? A::kSteps : 16;
    if constexpr (kFull && M + 1 <= kWave) {
        if (used) {
            double *col = slabs + j;
            // 1.0f the optimiser cannot see through, so the count lane's select
            // stays one 32-bit select ahead of the conversion instead of two
            // 32-bit selects on the converted double
            float one;
            asm("v_mov_b32 %0, 1.0" : "=v"(one));
#pragma unroll
            for (int s0 = 0; s0 < A::kSteps; s0 += B) {
                int o[B];
#pragma unroll
                for (int b = 0; b < B; ++b) o[b] = op[(s0 + b) * P];
#pragma unroll
                for (int b = 0; b < B; ++b) {
                    // the count column adds 1 (exact in fp64)
                    const float x = feat ? f.x[s0 + b] : one;
                    __hip_atomic_fetch_add(col + o[b], (double)x, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_WAVEFRONT);
                }
            }
        }
    } else {
#pragma unroll
        for (int s0 = 0; s0 < A::kSteps; s0 += B) {
            int o[B];
#pragma unroll
            for (int b = 0; b < B; ++b) o[b] = op[(s0 + b) * P];
#pragma unroll
            for (int b = 0; b < B; ++b) {
                const double v = feat ? (double)f.x[s0 + b] : 1.0;
                if (used && o[b] >= 0)
                    __hip_atomic_fetch_add(slabs + o[b] + j, v, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_WAVEFRONT);
                if (M + 1 > kWave && lane == 0 && o[b] >= 0)   // M = 64: no lane left for the count
                    __hip_atomic_fetch_add(slabs + o[b] + M, 1.0, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_WAVEFRONT);
            }
        }
    }
    __builtin_amdgcn_wave_barrier();
}

// Workgroup partial of the wave-accumulation form: for every (cluster, feature)
// the sum over waves w and slabs h (w, then h, ascending) written to
// part_sums[K][M], and the count of cluster k to counts_col[k * cstride] (the
// workgroup's column of the [K][G] count table). Call after a barrier.
// kShared: one slab per wave (see accumulate_tile).
template <int M, int P_, bool kShared = false>
__device__ inline void write_wave_partials(const double *slabs, int W, int K,
                                           double *__restrict__ part_sums,
                                           int32_t *__restrict__ counts_col, int cstride)
{
    using A = WaveAcc<M, P_>;
    constexpr int MW = A::MW, P = kShared ? 1 : A::P;
    const int tid = threadIdx.x, nthr = blockDim.x;
    const size_t rows = (size_t)W * P;          // slabs in the workgroup
    for (int e = tid; e < K * MW; e += nthr) {
        const int k = e / MW, j = e - (e / MW) * MW;
        double s = 0.0;
        for (size_t r = 0; r < rows; ++r) s = s + slabs[(r * K + k) * MW + j];
        if (j < M) part_sums[(int64_t)k * M + j] = s;
        else counts_col[(int64_t)k * cstride] = (int32_t)s;
    }
}

}  // namespace lloyd
