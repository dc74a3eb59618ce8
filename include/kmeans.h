/*
 * kmeans.h -- C ABI of the MI355X (gfx950) Lloyd-iteration library.
 *
 * The library runs the data-parallel part of K-means as described in
 * Algorithm 1 of Litvinenko, "Using of GPUs for cluster analysis of large data
 * by K-means method": assign every object to the nearest centre (steps 2 and
 * 4, Euclidean distance of Eq. (2)), recompute each cluster's centre of gravity
 * (steps 3 and 5, Eq. (1)), and stop when the centres of the last two
 * iterations are congruent (steps 6 and 7). It also picks the K initial
 * centres of step 1 by farthest-point traversal, and computes the diameter
 * (Eq. (3)) and the centre of gravity of the whole set (Algorithm 2 steps
 * 1-2).
 *
 * Conventions shared by every entry point
 *   - Array arguments are DEVICE pointers (hipMalloc'd or equivalent), owned by
 *     the caller; the library never allocates, frees or retains device memory
 *     beyond a call. Row-major layouts: X is [n][M] fp32 (object-major, each
 *     object's M features contiguous), centres are [K][M] fp32.
 *   - X must be 16-byte aligned (every hipMalloc'd buffer is).
 *   - `stream` is a hipStream_t (NULL = the default stream). Work is enqueued on
 *     it; kmeans_assign and kmeans_update return without waiting, kmeans_run
 *     waits for its own work before returning.
 *   - The return value is KMEANS_OK (0) or a negative KMEANS_E* code. Arguments
 *     are validated on the host before anything is enqueued: on a validation
 *     error nothing is enqueued and no output is touched. kmeans_strerror()
 *     names a code. No C++ exception crosses this interface.
 *   - Envelope: 1 <= n <= 2^31-1, 1 <= M <= 64, 1 <= K <= 1024, K*M <= 16384.
 *     Shapes outside it return KMEANS_EUNSUPPORTED.
 *   - Results are deterministic: the same inputs on the same device give
 *     bitwise-identical labels, centres, counts and iteration counts (sums are
 *     formed in fp64 in a fixed order; no floating-point atomics).
 *   - Arithmetic (the readings taken where the paper is silent): distances are
 *     compared squared; ties go to the lowest centre index; centres are the
 *     fp64 mean of the members rounded once to fp32; a cluster with no members
 *     keeps its previous centre and has count 0. A label is the exact-arithmetic
 *     argmin: points whose fp32 distances are too close to call are re-decided
 *     with fp64 distances. Inputs containing NaN or Inf give unspecified labels.
 */
#ifndef KMEANS_MI355X_H
#define KMEANS_MI355X_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
#define KMEANS_OK             0
#define KMEANS_EINVAL        -1   /* NULL pointer, non-positive size, misaligned X, bad flags */
#define KMEANS_EUNSUPPORTED  -2   /* shape outside the envelope above                        */
#define KMEANS_EWORKSPACE    -3   /* workspace missing or smaller than kmeans_workspace_bytes */
#define KMEANS_EHIP          -4   /* a HIP runtime call or kernel launch failed, or a kernel  */
                                  /* reported that its ordered accumulation broke down      */

/* Flags (bitwise OR). */
#define KMEANS_FIXED_ITERS  (1u << 0) /* kmeans_run: run exactly max_iter iterations, no early stop */
#define KMEANS_PATH_DIRECT  (1u << 1) /* force the vector-ALU distance path                          */
#define KMEANS_PATH_MFMA    (1u << 2) /* force a matrix-core (expanded-form) distance path: one      */
                                      /* object per lane for K <= 64 and M <= 32, else 64-object      */
                                      /* tiles; KMEANS_EUNSUPPORTED when the tiles' per-workgroup     */
                                      /* state (centre operands, fp64 sums) does not fit in LDS       */
#define KMEANS_PATH_TILES   (1u << 3) /* force the 64-object-tile matrix-core path (any K)           */
#define KMEANS_METRIC_L1    (1u << 4) /* assign by the L1 (city-block) distance sum_j |x_j - c_j|      */
                                      /* instead of Eq. (2) -- the paper allows another metric; the   */
                                      /* centres stay the centres of gravity of Eq. (1). One form (one */
                                      /* object per lane on the vector ALU): no path flag with it.     */
#define KMEANS_FORCE_FP64   (1u << 5) /* decide every label from fp64 distances in the fixed          */
                                      /* operation order (the path every close call takes anyway),    */
                                      /* skipping the faster screening: slower, same results; for     */
                                      /* checking that the screening changes no label.                 */
/* Without a path flag: one object per lane on the matrix cores for
 * 5 <= K <= 64 (M <= 32), 64-object tiles on the matrix cores for other
 * K > 16, the vector ALU otherwise. Every path gives the same labels and
 * counts, and centres equal to within the rounding of fp64 sums (each path
 * sums in its own fixed order). */

/* Optional per-call timing for kmeans_run (pass NULL for none). Each
 * iteration is two launches on `stream`: assign + accumulate (Algorithm 1
 * steps 2/4 and the sums of Eq. (1)), then the centres and the congruence test
 * (Eq. (1), steps 6-7). HIP events are recorded on `stream` before the first
 * and after the last launch of the call (step_ms). The assigning launch of
 * every sample_every-th iteration (for the L1 metric with K > 32 the L1 assign
 * launch, else the fused assign + accumulate launch) is made with
 * hipExtLaunchKernel and a
 * pair of events that its dispatch stamps at its start and end (assign_ms: the
 * kernel's own duration, nothing between launches). In early-stop mode step_ms
 * also contains the host's convergence polls; timing is meant for
 * KMEANS_FIXED_ITERS runs.
 *   in:  sample_every  (0 = every 16th iteration, 1 = every iteration)
 *   out: the other fields */
typedef struct kmeans_timing {
    double  step_ms;          /* device time of the whole call's iterations    */
    double  assign_ms;        /* summed duration of the sampled assign launches */
    int32_t step_launches;    /* iterations covered by step_ms                 */
    int32_t assign_samples;   /* launches summed in assign_ms                  */
    int32_t sample_every;     /* in: sampling stride of the assign launches    */
    int32_t reserved;
} kmeans_timing_t;

/* Bytes of device workspace that kmeans_update and kmeans_run need for a problem
 * of this shape and these flags (per-workgroup fp64 partial sums and counts,
 * their totals, and a 256-byte control block at the start). kmeans_assign needs
 * none. Returns 0 for shapes or flags the library refuses. Pure host
 * computation. After kmeans_run, bytes 12..15 of the workspace hold (int32)
 * the number of objects whose label was re-decided with fp64 distances during
 * the run -- a diagnostic, not part of the result. */
size_t kmeans_workspace_bytes(int64_t n, int32_t M, int32_t K, uint32_t flags);

/* Human-readable name of a status code (static storage). */
const char *kmeans_strerror(int status);

/* Bytes of device workspace that kmeans_init_farthest needs for this shape
 * (one fp64 distance per object, n * 8 bytes plus a few KB). Returns 0 for
 * shapes the library refuses, K > n included. Pure host computation. */
size_t kmeans_init_workspace_bytes(int64_t n, int32_t M, int32_t K);

/*
 * Initial centres, Algorithm 1 step 1 (K objects lying far apart;
 * the paper leaves the method open), read as farthest-point traversal from
 * object 0:
 *   init_idx[0] = 0;
 *   init_idx[m] = the object not among init_idx[0..m-1] whose smallest squared
 *                 distance (Eq. (2)) to those objects is largest, the lowest
 *                 such index on ties;
 *   centers[m]  = X[init_idx[m]] (fp32 [K][M], copied bit for bit).
 * The distances are formed in fp64 in the fixed order e = x_j - c_j,
 * d = d + e*e (features ascending, each operation rounded), so the indices are
 * exactly the ones that definition gives. Needs 1 <= K <= n (K > n:
 * KMEANS_EINVAL). init_idx is an int32 [K] DEVICE array. Asynchronous on
 * `stream`: K launches, each one pass over X (n * (4M + 16) bytes).
 */
int kmeans_init_farthest(const float *X, int64_t n, int32_t M, int32_t K, int32_t *init_idx,
                         float *centers, void *workspace, size_t workspace_bytes, void *stream);

/*
 * The same traversal from nseeds given seed objects (another reading of
 * Algorithm 2 step 3, e.g. the two ends of the diameter that kmeans_diameter
 * leaves in device memory):
 *   init_idx[m] = seeds[m] for m < nseeds (as given; repeats allowed);
 *   init_idx[m] = the object not among init_idx[0..m-1] farthest from them
 *                 (as above), for nseeds <= m < K.
 * seeds is an int32 [nseeds] DEVICE array; the call reads it back (one small
 * copy on `stream`, so it waits for the work that wrote the seeds) and returns
 * KMEANS_EINVAL, with nothing enqueued, if a seed lies outside [0, n).
 * 1 <= nseeds <= K <= n, else KMEANS_EINVAL. Workspace as
 * kmeans_init_workspace_bytes. kmeans_init_farthest is this call with the one
 * seed 0 (which needs no read-back). Otherwise asynchronous on `stream`.
 */
int kmeans_init_farthest_from(const float *X, int64_t n, int32_t M, int32_t K,
                              const int32_t *seeds, int32_t nseeds, int32_t *init_idx,
                              float *centers, void *workspace, size_t workspace_bytes,
                              void *stream);

/* Bytes of device workspace that kmeans_centroid needs (one fp64 row of
 * partial sums per workgroup, a few KB). 0 for refused shapes. Pure host. */
size_t kmeans_centroid_workspace_bytes(int64_t n, int32_t M);

/*
 * Centre of gravity of the whole set, Algorithm 2 step 2 (and Algorithm 4's
 * coordinate sums): centroid[j] = fp32(fp64 sum of x_ij over all i / n),
 * fp32 [M] DEVICE array. The sums are formed in an order fixed by the shape
 * (deterministic). Asynchronous on `stream`: two launches, one pass over X.
 */
int kmeans_centroid(const float *X, int64_t n, int32_t M, float *centroid, void *workspace,
                    size_t workspace_bytes, void *stream);

/* Bytes of device workspace that kmeans_diameter needs: the centre of gravity
 * and its partials, four bf16 operand arrays of n * 32 ceil((M+2)/32) values
 * each (n rounded up to 16384), and 16 bytes per (512-object block, 16384-object
 * chunk) pair. 0 for refused shapes (also when n needs more than 65535 column
 * chunks). Pure host computation. */
size_t kmeans_diameter_workspace_bytes(int64_t n, int32_t M);

/*
 * Diameter of the set, Eq. (3) (Algorithm 2 step 1: the pair of objects that
 * lie farthest apart), squared:
 *   *d2     = max over pairs k < l of |x_k - x_l|^2 (DEVICE fp64 [1]), the
 *             fp64 value formed as e = x_j - c_j, d = d + e*e (features
 *             ascending, each operation rounded), so exactly that pair's value;
 *   pair    = (k, l), the lexicographically smallest pair reaching it
 *             (DEVICE int32 [2]);
 *   centroid (may be NULL) = the centre of gravity, as kmeans_centroid.
 * With n = 1 there is no pair: *d2 = 0 and pair = (0, 0). If X holds a NaN
 * or an infinity the diameter is not defined: *d2 = NaN and pair = (-1, -1)
 * (kmeans_init_farthest_from refuses such seeds). The diameter is
 * sqrt(*d2). The pairs are screened with split-precision bf16 matrix
 * products under a proven error bound and the close ones re-evaluated in
 * fp64, so the result is exact; the cost is two passes over all n(n-1)/2
 * pairs (O(n^2 M): about half a second per pass at n = 2*10^6, M = 25).
 * Asynchronous on `stream`.
 */
int kmeans_diameter(const float *X, int64_t n, int32_t M, double *d2, int32_t *pair,
                    float *centroid, void *workspace, size_t workspace_bytes, void *stream);

/*
 * Assignment, Algorithm 1 steps 2 and 4, distance of Eq. (2):
 *   labels[i] = argmin_k |X_i - centers_k|^2  (lowest k on ties), int32 [n].
 * min_d2 (may be NULL) receives fp32 [n] squared distances to the chosen centre
 * (with KMEANS_METRIC_L1: the labels are by the L1 distance and min_d2 holds it).
 * flags: KMEANS_PATH_* or KMEANS_METRIC_L1. Asynchronous on `stream`.
 */
int kmeans_assign(const float *X, int64_t n, int32_t M, const float *centers, int32_t K,
                  int32_t *labels, float *min_d2, uint32_t flags, void *stream);

/*
 * Centres of gravity, Eq. (1) (Algorithm 1 steps 3 and 5):
 *   counts[k]  = number of objects with labels[i] == k                 (int32 [K]),
 *   centers[k] = fp32(fp64 mean of those objects), or prev_centers[k] when the
 *                cluster has no member                                 (fp32 [K][M]).
 * labels must lie in [0, K); objects with other labels are not counted.
 * centers may alias prev_centers. Asynchronous on `stream`.
 */
int kmeans_update(const float *X, int64_t n, int32_t M, const int32_t *labels, int32_t K,
                  const float *prev_centers, float *centers, int32_t *counts,
                  void *workspace, size_t workspace_bytes, void *stream);

/*
 * The Lloyd loop, Algorithm 1 steps 2-7, from the given initial centres:
 *   for t = 1..max_iter: labels_t = assign(C_{t-1}); C_t = update(labels_t);
 *                        stop when t >= 2 and C_t is bitwise equal to C_{t-1}
 *                        (unless KMEANS_FIXED_ITERS).
 * Outputs: labels of the last assignment pass (int32 [n]), the centres of
 * gravity of those labels (fp32 [K][M]), their counts (int32 [K]), and in
 * *iterations (a HOST int32) the number of assignment passes executed.
 * init_centers may alias centers. Synchronous: returns once the work is done.
 * timing may be NULL.
 */
int kmeans_run(const float *X, int64_t n, int32_t M, int32_t K, const float *init_centers,
               int32_t max_iter, uint32_t flags, int32_t *labels, float *centers,
               int32_t *counts, int32_t *iterations, void *workspace,
               size_t workspace_bytes, void *stream, kmeans_timing_t *timing);

/*
 * kmeans_run without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid allocation). Same arguments, results and behaviour as
 * kmeans_run with timing == NULL, except:
 *   - the workspace is a static array the library holds on each GPU it runs
 *     on (KMEANS_NOALLOC_MAX_WORKSPACE bytes, reserved when the library is
 *     loaded on the device and kept until the process ends); a shape whose
 *     kmeans_workspace_bytes(n, M, K, flags) exceeds it returns
 *     KMEANS_EWORKSPACE with nothing enqueued;
 *   - the call allocates nothing: no device or pinned host memory, no events
 *     (the control block is read back into host stack memory);
 *   - every call on one GPU uses that GPU's one array: calls that overlap on
 *     a GPU (other host threads, or other streams) race and give undefined
 *     results. Each call starts by clearing what must start at zero, so
 *     consecutive calls need nothing in between.
 * The current HIP device selects the array; `stream` must belong to it.
 * Synchronous, like kmeans_run.
 */
#define KMEANS_NOALLOC_MAX_WORKSPACE ((size_t)16 << 20)
int kmeans_run_noalloc(const float *X, int64_t n, int32_t M, int32_t K, const float *init_centers,
                       int32_t max_iter, uint32_t flags, int32_t *labels, float *centers,
                       int32_t *counts, int32_t *iterations, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* KMEANS_MI355X_H */
