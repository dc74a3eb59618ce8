// C ABI of the Lloyd-iteration library: argument validation, workspace layout,
// the initial centres of Algorithm 1 step 1 and the iteration control of its
// steps 2-7. See include/kmeans.h.
#include "../../include/kmeans.h"
#include "lloyd.h"
#include "lloyd_l1.h"
#include "farthest.h"
#include "diameter.h"

#include <mutex>


using namespace lloyd;

namespace {

constexpr uint32_t kKnownFlags = KMEANS_FIXED_ITERS | KMEANS_PATH_DIRECT | KMEANS_PATH_MFMA |
                                  KMEANS_PATH_TILES | KMEANS_METRIC_L1 | KMEANS_FORCE_FP64;

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

int check_shape(int64_t n, int32_t M, int32_t K)
{
    if (n < 1 || M < 1 || K < 1) return KMEANS_EINVAL;
    if (n > INT32_MAX) return KMEANS_EUNSUPPORTED;
    if (M > kMaxM || K > kMaxK || (int64_t)K * M > kMaxKM) return KMEANS_EUNSUPPORTED;
    return KMEANS_OK;
}

int check_flags(uint32_t flags)
{
    if (flags & ~kKnownFlags) return KMEANS_EINVAL;
    const uint32_t paths = flags & (KMEANS_PATH_DIRECT | KMEANS_PATH_MFMA | KMEANS_PATH_TILES);
    if (paths & (paths - 1)) return KMEANS_EINVAL;          // at most one path flag
    if ((flags & KMEANS_METRIC_L1) && paths) return KMEANS_EINVAL;   // L1 has one form
    return KMEANS_OK;
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Distance path. KMEANS_PATH_DIRECT: the vector ALU. KMEANS_PATH_TILES: the
// 64-object tiles (-1 when their workgroup state does not fit in LDS).
// KMEANS_PATH_MFMA: the
// matrix cores, one object per lane when the centre operands fit in registers
// (K <= 16, M <= 32), else 64-object tiles when their workgroup state fits in
// LDS, else -1 (refused). No flag: tiles for K > 16, one object per lane on the
// matrix cores for 5 <= K <= 16, the vector ALU otherwise (and wherever the
// matrix-core forms do not fit).
int select_path(int32_t M, int32_t K, uint32_t flags)
{
    if (flags & KMEANS_PATH_DIRECT) return kPathValu;
    const bool lane = lane_mfma_fits(M, K), tile = tile_fits(M, K);
    if (flags & KMEANS_PATH_TILES) return tile ? kPathTile : -1;
    if (flags & KMEANS_PATH_MFMA) return lane ? kPathLaneMfma : tile ? kPathTile : -1;
    if (lane && K >= 5) return kPathLaneMfma;
    return (K > 16 && tile) ? kPathTile : kPathValu;
}

AccumPlan plan_for(int p, int64_t n, int32_t M, int32_t K, Mode mode)
{
    if (p == kPathTile) return plan_tile(n, M, K, mode);
    if (p == kPathLaneMfma) return plan_lane_mfma(n, M, K, mode);
    return plan_lane(n, M, K, mode);
}

hipError_t launch_step(const StepArgs &a, Mode mode, const AccumPlan &plan, hipStream_t s)
{
    if (plan.path == kPathTile) return launch_tile(a, mode, plan, s);
    if (plan.path == kPathLaneMfma) return launch_lane_mfma(a, mode, plan, s);
    return launch_lane(a, mode, plan, s);
}

// Per-thread, per-device state of kmeans_run that outlives a call: HIP events
// for its optional timing (created on first use, kept) and a pinned host copy
// of the control block (the read at the end of a call needs no staging).
// Neither is ever released; a thread holds at most a few events per device and
// 256 bytes of pinned memory.
struct RunCache {
    int device = -1;
    hipEvent_t ev[2 + 2 * 64];   // kMaxSamples sampled launches
    int nev = 0;
    Ctl *pinned = nullptr;
};

RunCache &run_cache()
{
    static thread_local RunCache caches[16];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) dev = 0;
    RunCache &c = caches[dev % 16];
    if (c.device != dev) {
        c = RunCache{};
        c.device = dev;
    }
    return c;
}

// Workspace: [Ctl (256 B)] [fp64 workgroup partials G*K*M] [int32 workgroup
// counts G*K], with G the persistent workgroups of the accumulating launch.
struct Layout {
    AccumPlan plan;
    bool l1_fused;   // L1 runs assign and accumulate in one launch (plan is its plan)
    size_t sums_off, counts_off, total;
};

Layout layout(int64_t n, int32_t M, int32_t K, uint32_t flags)
{
    Layout L{};
    if (flags & KMEANS_METRIC_L1) {
        const AccumPlan f = plan_lane_l1(n, M, K);
        L.l1_fused = f.waves > 0;
        if (L.l1_fused) L.plan = f;
    }
    if (!L.l1_fused) L.plan = plan_for(select_path(M, K, flags), n, M, K, kAssignAccum);
    const size_t km = (size_t)K * M;
    L.sums_off = align_up(sizeof(Ctl), 256);
    L.counts_off = align_up(L.sums_off + (size_t)L.plan.groups * km * sizeof(double), 256);
    L.total = align_up(L.counts_off + (size_t)L.plan.groups * K * sizeof(int32_t), 256);
    return L;
}

void bind_workspace(StepArgs &a, const Layout &L, char *ws)
{
    a.part_sums = reinterpret_cast<double *>(ws + L.sums_off);
    a.part_counts = reinterpret_cast<int32_t *>(ws + L.counts_off);
    a.ctl = reinterpret_cast<Ctl *>(ws);
}

int hip_status(hipError_t e) { return e == hipSuccess ? KMEANS_OK : KMEANS_EHIP; }

// Workspace of the farthest-point traversal: [fp64 nearest distance per
// object] [fp64 candidate distance 2*G] [int32 candidate index 2*G].
struct InitLayout {
    FarthestPlan plan;
    size_t cand_v_off, cand_i_off, total;
};

InitLayout init_layout(int64_t n, int32_t M)
{
    InitLayout L{};
    L.plan = plan_farthest(n, M);
    L.cand_v_off = align_up((size_t)n * sizeof(double), 256);
    L.cand_i_off = align_up(L.cand_v_off + 2 * (size_t)L.plan.groups * sizeof(double), 256);
    L.total = align_up(L.cand_i_off + 2 * (size_t)L.plan.groups * sizeof(int32_t), 256);
    return L;
}

// Workspace of the centroid and diameter launches: [counters 256 B]
// [fp32 centroid, M] [fp64 partials G*M] then, for the diameter, the four
// split operand arrays [npad][4 ks] x 16 B and the item slots.
struct DiamLayout {
    CentroidPlan cplan;
    DiameterPlan dplan;
    size_t centroid_off, part_off, ops_off, ops_bytes, slots_off, total;
};

DiamLayout diam_layout(int64_t n, int32_t M, bool diameter)
{
    DiamLayout L{};
    L.cplan = plan_centroid(n, M);
    L.centroid_off = 256;
    L.part_off = align_up(L.centroid_off + (size_t)M * sizeof(float), 256);
    L.ops_off = align_up(L.part_off + (size_t)L.cplan.groups * M * sizeof(double), 256);
    L.total = L.ops_off;
    if (diameter) {
        L.dplan = plan_diameter(n, M);
        L.ops_bytes = align_up((size_t)L.dplan.npad * 4 * L.dplan.ks * 16, 256);
        L.slots_off = L.ops_off + 4 * L.ops_bytes;
        L.total = align_up(L.slots_off + (size_t)L.dplan.row_blocks * L.dplan.chunks *
                                             sizeof(DiamBest), 256);
    }
    return L;
}

// Grid limits of the diameter passes (row blocks in x, column chunks in y).
bool diameter_fits(int64_t n, int32_t M)
{
    const DiameterPlan p = plan_diameter(n, M);
    return p.chunks <= 65535 && p.row_blocks <= INT32_MAX;
}


// Workspace of kmeans_run_noalloc: one array per GPU, allocated with the code
// object when the library is loaded on a device and kept until the process
// ends. In host code `scratch` names a host-side stand-in, not the device
// array: its device address, which differs from GPU to GPU, comes from
// hipGetSymbolAddress with the device current, once per device, and only that
// address is ever handed to kernels or copies.
constexpr size_t kScratchBytes = KMEANS_NOALLOC_MAX_WORKSPACE;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

int scratch_on_current_device(char **out)
{
    constexpr int kMaxDevices = 64;
    static std::mutex mu;
    static char *addr[kMaxDevices] = {};
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return KMEANS_EHIP;
    std::lock_guard<std::mutex> lock(mu);
    if (addr[dev] == nullptr) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr)
            return KMEANS_EHIP;
        addr[dev] = static_cast<char *>(p);
    }
    *out = addr[dev];
    return KMEANS_OK;
}

// Arguments of kmeans_run that need no workspace (the shared validation).
int check_run(const float *X, int64_t n, int32_t M, int32_t K, const float *init_centers,
              int32_t max_iter, uint32_t flags, const int32_t *labels, const float *centers,
              const int32_t *counts, const int32_t *iterations)
{
    if (!X || !init_centers || !labels || !centers || !counts || !iterations) return KMEANS_EINVAL;
    int rc = check_shape(n, M, K);
    if (rc) return rc;
    if (max_iter < 1) return KMEANS_EINVAL;
    if ((rc = check_flags(flags))) return rc;
    if (!aligned16(X)) return KMEANS_EINVAL;
    if (select_path(M, K, flags) < 0) return KMEANS_EUNSUPPORTED;
    return KMEANS_OK;
}

// The Lloyd loop on a validated call; ws holds L.total bytes. With
// may_allocate false nothing is allocated: no events (timing must be null) and
// the control block is read back into pageable host memory.
int run_impl(const float *X, int64_t n, int32_t M, int32_t K, const float *init_centers,
             int32_t max_iter, uint32_t flags, int32_t *labels, float *centers, int32_t *counts,
             int32_t *iterations, const Layout &L, char *ws, hipStream_t s,
             kmeans_timing_t *timing, bool may_allocate)
{
    int rc = KMEANS_OK;
    const int fixed = (flags & KMEANS_FIXED_ITERS) ? 1 : 0;
    const bool l1 = (flags & KMEANS_METRIC_L1) != 0;
    const L1Plan p1 = l1 && !L.l1_fused ? plan_l1(n, M, K) : L1Plan{};
    if (l1 && !L.l1_fused && p1.waves < 1) return KMEANS_EUNSUPPORTED;
    const int every = timing == nullptr ? 0 : (timing->sample_every > 0 ? timing->sample_every : 16);
    // events: one before the first launch, one after the last, and a pair
    // stamped with the start and end of each sampled assigning launch
    constexpr int kMaxSamples = 64;
    int nsampled = every > 0 ? (max_iter + every - 1) / every : 0;
    if (nsampled > kMaxSamples) nsampled = kMaxSamples;

    RunCache &cache = run_cache();
    if (timing && !may_allocate) return KMEANS_EINVAL;
    if (timing) {
        while (cache.nev < 2 + 2 * nsampled) {
            if (hipEventCreate(&cache.ev[cache.nev]) != hipSuccess) return KMEANS_EHIP;
            ++cache.nev;
        }
    }
    if (may_allocate && cache.pinned == nullptr) {
        void *p = nullptr;
        if (hipHostMalloc(&p, sizeof(Ctl), hipHostMallocDefault) == hipSuccess)
            cache.pinned = static_cast<Ctl *>(p);
    }
    Ctl pageable{};
    Ctl *host = (may_allocate && cache.pinned != nullptr) ? cache.pinned : &pageable;

    StepArgs a{};
    a.X = X; a.n = n; a.M = M; a.K = K;
    a.labels = labels;
    a.centers_out = centers;     // centres are updated in place, iteration by iteration
    a.counts_out = counts;
    bind_workspace(a, L, ws);
    a.fixed = fixed;
    a.compare = 1;
    a.force64 = (flags & KMEANS_FORCE_FP64) ? 1 : 0;
    a.labels_in = labels;        // the L1 form accumulates from the labels it wrote
    Ctl *ctl = a.ctl;

    if ((rc = hip_status(launch_ctl_reset(ctl, s)))) return rc;

    int nev = 0;
    auto mark = [&]() -> int {
        if (!timing) return KMEANS_OK;
        return hip_status(hipEventRecord(cache.ev[nev++], s));
    };

    // Two launches per iteration: assign + accumulate (fused), then the centres
    // and the congruence test from the workgroup partials. Iteration t assigns
    // with the centres of iteration t - 1: the caller's initial centres for
    // t = 1 (read in place; nothing is copied), `centers` afterwards, which
    // every centres launch writes whole.
    // Enqueue iterations in chunks; between chunks (early-stop mode only) read
    // the control block to learn whether the centres have become congruent.
    // Launches past convergence return at their first instruction.
    int t = 1, chunk = 3, launched = 0;
    rc = mark();
    while (!rc && t <= max_iter) {
        // fixed-count runs enqueue everything at once; otherwise chunks grow 3, 6, 12, ...
        const int end = (fixed || t + chunk - 1 >= max_iter) ? max_iter : t + chunk - 1;
        for (int tt = t; tt <= end && !rc; ++tt) {
            a.t = tt;
            a.C = tt == 1 ? init_centers : centers;
            const bool sampled =
                every > 0 && (tt - 1) % every == 0 && (tt - 1) / every < kMaxSamples;
            if (sampled) {
                // the pair is stamped by the assigning dispatch itself
                a.ev_start = cache.ev[nev++];
                a.ev_stop = cache.ev[nev++];
            }
            if (l1 && L.l1_fused) {
                // L1 assignment fused with the sums of Eq. (1)
                rc = hip_status(launch_lane_l1(a, L.plan, s));
                a.ev_start = a.ev_stop = nullptr;
            } else if (l1) {
                // L1: assign, then the sums of Eq. (1) from those labels
                rc = hip_status(launch_l1(a, p1, s));
                a.ev_start = a.ev_stop = nullptr;
                if (!rc) rc = hip_status(launch_step(a, kAccumLabels, L.plan, s));
            } else {
                rc = hip_status(launch_step(a, kAssignAccum, L.plan, s));
                a.ev_start = a.ev_stop = nullptr;
            }
            if (!rc) rc = hip_status(launch_centres(a, L.plan.groups, s));
            ++launched;
        }
        t = end + 1;
        if (rc || t > max_iter) break;
        rc = hip_status(hipMemcpyAsync(host, ctl, sizeof(Ctl), hipMemcpyDeviceToHost, s));
        if (!rc) rc = hip_status(hipStreamSynchronize(s));
        if (rc || host->converged_at != 0) break;
        chunk = chunk * 2 < 64 ? chunk * 2 : 64;
    }
    if (!rc) rc = mark();
    if (!rc) rc = hip_status(hipMemcpyAsync(host, ctl, sizeof(Ctl), hipMemcpyDeviceToHost, s));
    if (!rc) rc = hip_status(hipStreamSynchronize(s));
    if (rc) return rc;
    *iterations = host->converged_at != 0 ? host->converged_at : max_iter;
    if (host->ring_stalls != 0) rc = KMEANS_EHIP;

    if (timing) {
        timing->step_ms = 0.0;
        timing->assign_ms = 0.0;
        timing->step_launches = launched;
        timing->assign_samples = 0;
        timing->reserved = 0;
        float ms = 0.f;
        if (nev < 2 || hipEventElapsedTime(&ms, cache.ev[0], cache.ev[nev - 1]) != hipSuccess)
            return KMEANS_EHIP;
        timing->step_ms = ms;
        for (int e = 1; e + 2 < nev; e += 2) {
            if (hipEventElapsedTime(&ms, cache.ev[e], cache.ev[e + 1]) != hipSuccess)
                return KMEANS_EHIP;
            timing->assign_ms += ms;
            timing->assign_samples++;
        }
    }
    return rc;
}

}  // namespace

extern "C" {

const char *kmeans_strerror(int status)
{
    switch (status) {
    case KMEANS_OK: return "ok";
    case KMEANS_EINVAL: return "invalid argument";
    case KMEANS_EUNSUPPORTED: return "shape or option outside the supported envelope";
    case KMEANS_EWORKSPACE: return "workspace missing or too small";
    case KMEANS_EHIP: return "HIP runtime or kernel launch failure";
    default: return "unknown status";
    }
}

size_t kmeans_workspace_bytes(int64_t n, int32_t M, int32_t K, uint32_t flags)
{
    if (check_shape(n, M, K) != KMEANS_OK || (flags & ~kKnownFlags)) return 0;
    if (check_flags(flags) != KMEANS_OK || select_path(M, K, flags) < 0) return 0;
    return layout(n, M, K, flags).total;
}

size_t kmeans_init_workspace_bytes(int64_t n, int32_t M, int32_t K)
{
    if (check_shape(n, M, K) != KMEANS_OK || (int64_t)K > n) return 0;
    return init_layout(n, M).total;
}

int kmeans_init_farthest(const float *X, int64_t n, int32_t M, int32_t K, int32_t *init_idx,
                         float *centers, void *workspace, size_t workspace_bytes, void *stream)
{
    return kmeans_init_farthest_from(X, n, M, K, nullptr, 1, init_idx, centers, workspace,
                                     workspace_bytes, stream);
}

int kmeans_init_farthest_from(const float *X, int64_t n, int32_t M, int32_t K,
                              const int32_t *seeds, int32_t nseeds, int32_t *init_idx,
                              float *centers, void *workspace, size_t workspace_bytes,
                              void *stream)
{
    if (!X || !init_idx || !centers) return KMEANS_EINVAL;
    if (nseeds < 1 || nseeds > K || (!seeds && nseeds != 1)) return KMEANS_EINVAL;
    int rc = check_shape(n, M, K);
    if (rc) return rc;
    if ((int64_t)K > n || !aligned16(X)) return KMEANS_EINVAL;
    const InitLayout L = init_layout(n, M);
    if (!workspace || workspace_bytes < L.total) return KMEANS_EWORKSPACE;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (seeds != nullptr) {
        // the seeds live in device memory (often written by kmeans_diameter on
        // the same stream): read them back once, after the work that writes
        // them, and refuse any outside [0, n) before anything is enqueued
        int32_t host[kMaxK];
        if (hipMemcpyAsync(host, seeds, sizeof(int32_t) * (size_t)nseeds, hipMemcpyDeviceToHost,
                           s) != hipSuccess ||
            hipStreamSynchronize(s) != hipSuccess)
            return KMEANS_EHIP;
        for (int i = 0; i < nseeds; ++i)
            if (host[i] < 0 || (int64_t)host[i] >= n) return KMEANS_EINVAL;
    }
    char *ws = static_cast<char *>(workspace);
    FarthestArgs a{};
    a.X = X; a.n = n; a.M = M; a.K = K;
    a.nearest = reinterpret_cast<double *>(ws);
    a.cand_v = reinterpret_cast<double *>(ws + L.cand_v_off);
    a.cand_i = reinterpret_cast<int32_t *>(ws + L.cand_i_off);
    a.idx = init_idx;
    a.centers = centers;
    a.seeds = seeds;
    a.nseeds = nseeds;
    return hip_status(launch_farthest(a, L.plan, s));
}

size_t kmeans_centroid_workspace_bytes(int64_t n, int32_t M)
{
    if (check_shape(n, M, 1) != KMEANS_OK) return 0;
    return diam_layout(n, M, false).total;
}

int kmeans_centroid(const float *X, int64_t n, int32_t M, float *centroid, void *workspace,
                    size_t workspace_bytes, void *stream)
{
    if (!X || !centroid) return KMEANS_EINVAL;
    int rc = check_shape(n, M, 1);
    if (rc) return rc;
    if (!aligned16(X)) return KMEANS_EINVAL;
    const DiamLayout L = diam_layout(n, M, false);
    if (!workspace || workspace_bytes < L.total) return KMEANS_EWORKSPACE;
    char *ws = static_cast<char *>(workspace);
    return hip_status(launch_centroid(X, n, M, reinterpret_cast<double *>(ws + L.part_off),
                                      nullptr, centroid, nullptr, L.cplan,
                                      static_cast<hipStream_t>(stream)));
}

size_t kmeans_diameter_workspace_bytes(int64_t n, int32_t M)
{
    if (check_shape(n, M, 1) != KMEANS_OK || !diameter_fits(n, M)) return 0;
    return diam_layout(n, M, true).total;
}

int kmeans_diameter(const float *X, int64_t n, int32_t M, double *d2, int32_t *pair,
                    float *centroid, void *workspace, size_t workspace_bytes, void *stream)
{
    if (!X || !d2 || !pair) return KMEANS_EINVAL;
    int rc = check_shape(n, M, 1);
    if (rc) return rc;
    if (!aligned16(X)) return KMEANS_EINVAL;
    if (!diameter_fits(n, M)) return KMEANS_EUNSUPPORTED;
    const DiamLayout L = diam_layout(n, M, true);
    if (!workspace || workspace_bytes < L.total) return KMEANS_EWORKSPACE;
    char *ws = static_cast<char *>(workspace);
    hipStream_t s = static_cast<hipStream_t>(stream);
    DiameterArgs a{};
    a.X = X; a.n = n; a.M = M;
    a.counters = reinterpret_cast<uint32_t *>(ws);
    a.centroid_ws = reinterpret_cast<float *>(ws + L.centroid_off);
    a.ah = reinterpret_cast<uint4 *>(ws + L.ops_off);
    a.al = reinterpret_cast<uint4 *>(ws + L.ops_off + L.ops_bytes);
    a.bh = reinterpret_cast<uint4 *>(ws + L.ops_off + 2 * L.ops_bytes);
    a.bl = reinterpret_cast<uint4 *>(ws + L.ops_off + 3 * L.ops_bytes);
    a.slots = reinterpret_cast<DiamBest *>(ws + L.slots_off);
    a.d2 = d2;
    a.pair = pair;
    rc = hip_status(launch_centroid(X, n, M, reinterpret_cast<double *>(ws + L.part_off),
                                    a.centroid_ws, centroid, a.counters, L.cplan, s));
    if (rc) return rc;
    return hip_status(launch_diameter(a, L.dplan, s));
}

int kmeans_assign(const float *X, int64_t n, int32_t M, const float *centers, int32_t K,
                  int32_t *labels, float *min_d2, uint32_t flags, void *stream)
{
    if (!X || !centers || !labels) return KMEANS_EINVAL;
    int rc = check_shape(n, M, K);
    if (rc) return rc;
    if ((rc = check_flags(flags)) || (flags & KMEANS_FIXED_ITERS)) return rc ? rc : KMEANS_EINVAL;
    if (!aligned16(X)) return KMEANS_EINVAL;
    hipStream_t s = static_cast<hipStream_t>(stream);
    StepArgs a{};
    a.X = X; a.n = n; a.M = M; a.C = centers; a.K = K;
    a.labels = labels; a.min_d2 = min_d2;
    a.force64 = (flags & KMEANS_FORCE_FP64) ? 1 : 0;
    if (flags & KMEANS_METRIC_L1) {
        const L1Plan p1 = plan_l1(n, M, K);
        if (p1.waves < 1) return KMEANS_EUNSUPPORTED;
        return hip_status(launch_l1(a, p1, s));
    }
    if (select_path(M, K, flags) < 0) return KMEANS_EUNSUPPORTED;
    const AccumPlan plan = plan_for(select_path(M, K, flags), n, M, K, kAssign);
    return hip_status(launch_step(a, kAssign, plan, s));
}

int kmeans_update(const float *X, int64_t n, int32_t M, const int32_t *labels, int32_t K,
                  const float *prev_centers, float *centers, int32_t *counts, void *workspace,
                  size_t workspace_bytes, void *stream)
{
    if (!X || !labels || !prev_centers || !centers || !counts) return KMEANS_EINVAL;
    int rc = check_shape(n, M, K);
    if (rc) return rc;
    if (!aligned16(X)) return KMEANS_EINVAL;
    const Layout L = layout(n, M, K, 0);
    if (!workspace || workspace_bytes < L.total) return KMEANS_EWORKSPACE;
    hipStream_t s = static_cast<hipStream_t>(stream);
    StepArgs a{};
    a.X = X; a.n = n; a.M = M; a.C = prev_centers; a.K = K;
    a.labels_in = labels;
    a.centers_out = centers;
    a.counts_out = counts;
    bind_workspace(a, L, static_cast<char *>(workspace));
    a.fixed = 1;
    a.compare = 0;
    if ((rc = hip_status(launch_ctl_reset(a.ctl, s)))) return rc;
    if ((rc = hip_status(launch_step(a, kAccumLabels, L.plan, s)))) return rc;
    return hip_status(launch_centres(a, L.plan.groups, s));
}

int kmeans_run(const float *X, int64_t n, int32_t M, int32_t K, const float *init_centers,
               int32_t max_iter, uint32_t flags, int32_t *labels, float *centers, int32_t *counts,
               int32_t *iterations, void *workspace, size_t workspace_bytes, void *stream,
               kmeans_timing_t *timing)
{
    int rc = check_run(X, n, M, K, init_centers, max_iter, flags, labels, centers, counts,
                       iterations);
    if (rc) return rc;
    const Layout L = layout(n, M, K, flags);
    if (!workspace || workspace_bytes < L.total) return KMEANS_EWORKSPACE;
    return run_impl(X, n, M, K, init_centers, max_iter, flags, labels, centers, counts,
                    iterations, L, static_cast<char *>(workspace),
                    static_cast<hipStream_t>(stream), timing, true);
}

int kmeans_run_noalloc(const float *X, int64_t n, int32_t M, int32_t K, const float *init_centers,
                       int32_t max_iter, uint32_t flags, int32_t *labels, float *centers,
                       int32_t *counts, int32_t *iterations, void *stream)
{
    int rc = check_run(X, n, M, K, init_centers, max_iter, flags, labels, centers, counts,
                       iterations);
    if (rc) return rc;
    const Layout L = layout(n, M, K, flags);
    if (L.total > kScratchBytes) return KMEANS_EWORKSPACE;
    char *ws = nullptr;
    if ((rc = scratch_on_current_device(&ws))) return rc;
    return run_impl(X, n, M, K, init_centers, max_iter, flags, labels, centers, counts,
                    iterations, L, ws, static_cast<hipStream_t>(stream), nullptr, false);
}

}  // extern "C"
