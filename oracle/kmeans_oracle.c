/*
 * CPU oracle for the Lloyd iteration of K-means (Algorithm 1 of Litvinenko,
 * "Using of GPUs for cluster analysis of large data by K-means method").
 *
 * TEST INFRASTRUCTURE ONLY. This file is the plain, slow, single-threaded
 * statement of what the GPU library must compute; only the test suite, the
 * smoke check and the benchmark's CPU-baseline leg may load it. It shares no
 * code, header or constant with the GPU library.
 *
 * It follows the single-threaded regime (Algorithm 2, steps 4-8, which is
 * Algorithm 1 steps 2-7 with given initial centres):
 *   assign   : every object goes to the cluster whose centre is closest
 *              (Algorithm 1 steps 2 and 4, distance of Eq. (2));
 *   update   : each cluster's centre of gravity, Eq. (1)
 *              (Algorithm 1 steps 3 and 5);
 *   compare  : stop when the centres of the last two iterations are congruent
 *              (Algorithm 1 steps 6 and 7).
 *
 * Readings where the paper is silent (each is listed with its reason in the
 * design notes of the repository):
 *   - distances are compared squared (same argmin as Eq. (2), no sqrt);
 *   - arithmetic is fp64; inputs and stored centres are fp32; for every
 *     object and centre the squared distance is accumulated as
 *         e = (double)x_j - (double)c_j ;  d = d + e*e
 *     for j ascending, each operation rounded separately (no fused
 *     multiply-add; build with -ffp-contract=off);
 *   - ties go to the lowest cluster index (strict '<' while scanning k up);
 *   - a cluster with no members keeps its previous centre, count 0;
 *   - "congruent" means bitwise-identical fp32 centres; the first comparison
 *     is after the second update (t = 2), so the earliest stop is t = 2;
 *   - iterations = number of assignment passes executed; the returned labels
 *     are those of the last pass and the returned centres are the centres of
 *     gravity of those labels.
 *
 * Build: gcc -std=c99 -O2 -ffp-contract=off -fPIC -shared
 * All pointers are host pointers; arrays are row-major; return 0 or -1.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <math.h>

#define ORACLE_EINVAL (-1)
#define ORACLE_ENOMEM (-2)

/* Squared distance of Eq. (2) between object x and centre c, in the
 * normative operation order described above. */
static double sqdist(const float *x, const float *c, int32_t M)
{
    double d = 0.0;
    for (int32_t j = 0; j < M; ++j) {
        double e = (double)x[j] - (double)c[j];
        double sq = e * e;
        d = d + sq;
    }
    return d;
}

/*
 * Assignment, Algorithm 1 steps 2 and 4: labels[i] = argmin_k |x_i - c_k|^2,
 * lowest k on ties. Optionally reports, per object, the best squared distance
 * d1[i] and the smallest squared distance to any other centre d2[i]
 * (+infinity when K == 1); both may be NULL.
 */
int oracle_assign(const float *X, int64_t n, int32_t M, const float *C, int32_t K,
                  int32_t *labels, double *d1, double *d2)
{
    if (!X || !C || !labels || n < 0 || M < 1 || K < 1)
        return ORACLE_EINVAL;
    for (int64_t i = 0; i < n; ++i) {
        const float *x = X + i * (int64_t)M;
        double best = INFINITY, second = INFINITY;
        int32_t lab = 0;
        for (int32_t k = 0; k < K; ++k) {
            double d = sqdist(x, C + (int64_t)k * M, M);
            if (d < best) {
                second = best;
                best = d;
                lab = k;
            } else if (d < second) {
                second = d;
            }
        }
        labels[i] = lab;
        if (d1) d1[i] = best;
        if (d2) d2[i] = second;
    }
    return 0;
}

/*
 * Centres of gravity, Eq. (1) (Algorithm 1 steps 3 and 5):
 *   counts[k]  = n_k = number of objects with label k,
 *   centers[k] = fp32( (sum over those objects of x, in fp64, i ascending) / n_k )
 * and a cluster with n_k = 0 keeps prev[k]. centers may alias prev.
 * Labels outside [0, K) are an error.
 */
int oracle_update(const float *X, int64_t n, int32_t M, const int32_t *labels,
                  int32_t K, const float *prev, float *centers, int32_t *counts)
{
    if (!X || !labels || !prev || !centers || !counts || n < 0 || M < 1 || K < 1)
        return ORACLE_EINVAL;
    double *S = (double *)calloc((size_t)K * (size_t)M, sizeof(double));
    int64_t *cnt = (int64_t *)calloc((size_t)K, sizeof(int64_t));
    if (!S || !cnt) {
        free(S);
        free(cnt);
        return ORACLE_ENOMEM;
    }
    for (int64_t i = 0; i < n; ++i) {
        int32_t l = labels[i];
        if (l < 0 || l >= K) {
            free(S);
            free(cnt);
            return ORACLE_EINVAL;
        }
        const float *x = X + i * (int64_t)M;
        double *s = S + (int64_t)l * M;
        for (int32_t j = 0; j < M; ++j)
            s[j] = s[j] + (double)x[j];
        cnt[l] += 1;
    }
    for (int32_t k = 0; k < K; ++k) {
        for (int32_t j = 0; j < M; ++j) {
            int64_t o = (int64_t)k * M + j;
            if (cnt[k] > 0)
                centers[o] = (float)(S[o] / (double)cnt[k]);
            else
                centers[o] = prev[o];
        }
        counts[k] = (int32_t)cnt[k];
    }
    free(S);
    free(cnt);
    return 0;
}

/* Steps 6-7: are two sets of K*M fp32 centres congruent (bitwise equal)? */
static int congruent(const float *a, const float *b, int64_t count)
{
    return memcmp(a, b, (size_t)count * sizeof(float)) == 0;
}

/*
 * Another metric for the assignment (the paper allows one in place of
 * Eq. (2)): the L1 (city-block) distance sum_j |x_j - c_j|, in fp64 as
 *     e = (double)x_j - (double)c_j ;  d = d + |e|
 * for j ascending, each operation rounded. Only the assignment changes; the
 * centres stay the centres of gravity of Eq. (1).
 */
static double l1dist(const float *x, const float *c, int32_t M)
{
    double sum = 0.0;
    for (int32_t f = 0; f < M; ++f) {
        double diff = (double)x[f] - (double)c[f];
        sum = sum + fabs(diff);
    }
    return sum;
}

/* Assignment by the L1 distance: the same rule as oracle_assign (lowest k on
 * ties, optional best and second-best distances). */
int oracle_assign_l1(const float *X, int64_t n, int32_t M, const float *C, int32_t K,
                     int32_t *labels, double *d1, double *d2)
{
    if (!X || !C || !labels || n < 0 || M < 1 || K < 1)
        return ORACLE_EINVAL;
    for (int64_t obj = 0; obj < n; ++obj) {
        const float *row = X + obj * (int64_t)M;
        double nearest = INFINITY, runner_up = INFINITY;
        int32_t choice = 0;
        for (int32_t k = 0; k < K; ++k) {
            double dk = l1dist(row, C + (int64_t)k * M, M);
            if (dk < nearest) {
                runner_up = nearest;
                nearest = dk;
                choice = k;
            } else if (dk < runner_up) {
                runner_up = dk;
            }
        }
        labels[obj] = choice;
        if (d1) d1[obj] = nearest;
        if (d2) d2[obj] = runner_up;
    }
    return 0;
}

/*
 * The whole loop, Algorithm 1 steps 2-7 from the given initial centres:
 *   for t = 1 .. max_iter:
 *     labels_t = assign(C_{t-1});  C_t = update(labels_t, C_{t-1});
 *     if !fixed and t >= 2 and C_t congruent to C_{t-1}: stop.
 * Outputs the last labels, the last centres, their counts, and the number of
 * assignment passes executed. d1/d2 (nullable) receive the final pass's best
 * and second-best squared distances per object.
 */
static int run_loop(const float *X, int64_t n, int32_t M, int32_t K, const float *init,
                    int32_t max_iter, int32_t fixed, int32_t l1, int32_t *labels,
                    float *centers, int32_t *counts, int32_t *iterations, double *d1,
                    double *d2)
{
    if (!X || !init || !labels || !centers || !counts || !iterations || n < 0 ||
        M < 1 || K < 1 || max_iter < 1)
        return ORACLE_EINVAL;
    int64_t km = (int64_t)K * M;
    float *prev = (float *)malloc((size_t)km * sizeof(float));
    float *cur = (float *)malloc((size_t)km * sizeof(float));
    if (!prev || !cur) {
        free(prev);
        free(cur);
        return ORACLE_ENOMEM;
    }
    memcpy(prev, init, (size_t)km * sizeof(float));
    int32_t t = 0;
    int rc = 0;
    for (t = 1; t <= max_iter; ++t) {
        if (l1)
            rc = oracle_assign_l1(X, n, M, prev, K, labels, d1, d2);
        else
            rc = oracle_assign(X, n, M, prev, K, labels, d1, d2);
        if (rc) break;
        rc = oracle_update(X, n, M, labels, K, prev, cur, counts);
        if (rc) break;
        int stop = !fixed && t >= 2 && congruent(cur, prev, km);
        memcpy(prev, cur, (size_t)km * sizeof(float));
        if (stop) break;
    }
    if (t > max_iter) t = max_iter;
    if (!rc) {
        memcpy(centers, prev, (size_t)km * sizeof(float));
        *iterations = t;
    }
    free(prev);
    free(cur);
    return rc;
}

int oracle_run(const float *X, int64_t n, int32_t M, int32_t K, const float *init,
               int32_t max_iter, int32_t fixed, int32_t *labels, float *centers,
               int32_t *counts, int32_t *iterations, double *d1, double *d2)
{
    return run_loop(X, n, M, K, init, max_iter, fixed, 0, labels, centers, counts, iterations,
                    d1, d2);
}

/* The same loop with the L1 assignment. */
int oracle_run_l1(const float *X, int64_t n, int32_t M, int32_t K, const float *init,
                  int32_t max_iter, int32_t fixed, int32_t *labels, float *centers,
                  int32_t *counts, int32_t *iterations, double *d1, double *d2)
{
    return run_loop(X, n, M, K, init, max_iter, fixed, 1, labels, centers, counts, iterations,
                    d1, d2);
}

/* Objective sum_i |x_i - c_{label_i}|^2 in fp64 (used by the invariant tests). */
double oracle_sse(const float *X, int64_t n, int32_t M, const int32_t *labels,
                  const float *C, int32_t K)
{
    double s = 0.0;
    for (int64_t i = 0; i < n; ++i) {
        int32_t l = labels[i];
        if (l < 0 || l >= K) return NAN;
        s = s + sqdist(X + i * (int64_t)M, C + (int64_t)l * M, M);
    }
    return s;
}

/*
 * Initial centres, Algorithm 1 step 1 (K objects lying far apart;
 * the paper leaves the method open). Reading: farthest-point traversal from
 * object 0 --
 *   idx[0] = 0;
 *   idx[m] = the object i not among idx[0..m-1] whose smallest squared
 *            distance (Eq. (2), normative fp64 order above) to the objects
 *            idx[0..m-1] is largest, the lowest such i on ties.
 * The centres are the rows X[idx[m]]. Requires 1 <= K <= n.
 */
int oracle_init_farthest(const float *X, int64_t n, int32_t M, int32_t K, int32_t *idx)
{
    if (!X || !idx || n < 1 || M < 1 || K < 1 || (int64_t)K > n)
        return ORACLE_EINVAL;
    double *nearest = (double *)malloc((size_t)n * sizeof(double));
    unsigned char *chosen = (unsigned char *)calloc((size_t)n, 1);
    if (!nearest || !chosen) {
        free(nearest);
        free(chosen);
        return ORACLE_ENOMEM;
    }
    for (int64_t i = 0; i < n; ++i)
        nearest[i] = INFINITY;
    idx[0] = 0;
    chosen[0] = 1;
    for (int32_t m = 1; m < K; ++m) {
        /* fold the newest centre into every object's nearest distance */
        const float *c = X + (int64_t)idx[m - 1] * M;
        for (int64_t i = 0; i < n; ++i) {
            double d = sqdist(X + i * (int64_t)M, c, M);
            if (d < nearest[i])
                nearest[i] = d;
        }
        /* the farthest object not yet chosen, lowest index on ties */
        int64_t far = -1;
        for (int64_t i = 0; i < n; ++i) {
            if (chosen[i])
                continue;
            if (far < 0 || nearest[i] > nearest[far])
                far = i;
        }
        idx[m] = (int32_t)far;
        chosen[far] = 1;
    }
    free(nearest);
    free(chosen);
    return 0;
}

/*
 * Centre of gravity of the whole set (Algorithm 2 step 2):
 *   centroid[j] = fp32( (sum over i ascending of (double)x_ij) / n ).
 */
int oracle_centroid(const float *X, int64_t n, int32_t M, float *centroid)
{
    if (!X || !centroid || n < 1 || M < 1)
        return ORACLE_EINVAL;
    for (int32_t j = 0; j < M; ++j) {
        double s = 0.0;
        for (int64_t i = 0; i < n; ++i)
            s = s + (double)X[i * (int64_t)M + j];
        centroid[j] = (float)(s / (double)n);
    }
    return 0;
}

/*
 * Diameter of the set, Eq. (3) (Algorithm 2 step 1: the pair of objects that
 * lie farthest apart), squared:
 *   d2 = max over pairs k < l of |x_k - x_l|^2 (normative fp64 order above),
 *   (k, l) = the lexicographically smallest pair reaching it.
 * With n = 1 there is no pair: d2 = 0 and k = l = 0. The diameter is sqrt(d2).
 */
int oracle_diameter(const float *X, int64_t n, int32_t M, double *d2, int32_t *k_out,
                    int32_t *l_out)
{
    if (!X || !d2 || !k_out || !l_out || n < 1 || M < 1)
        return ORACLE_EINVAL;
    /* A coordinate that is NaN or infinite leaves the diameter undefined (the
     * paper defines it for real vectors): NaN and the pair (-1, -1). */
    for (int64_t e = 0; e < n * (int64_t)M; ++e) {
        if (!isfinite(X[e])) {
            *d2 = NAN;
            *k_out = -1;
            *l_out = -1;
            return 0;
        }
    }
    double best = 0.0;
    int64_t bk = 0, bl = n > 1 ? 1 : 0;
    int have = 0;
    for (int64_t k = 0; k < n; ++k) {
        for (int64_t l = k + 1; l < n; ++l) {
            double d = sqdist(X + k * (int64_t)M, X + l * (int64_t)M, M);
            if (!have || d > best) {
                best = d;
                bk = k;
                bl = l;
                have = 1;
            }
        }
    }
    *d2 = best;
    *k_out = (int32_t)bk;
    *l_out = (int32_t)bl;
    return 0;
}

/*
 * Farthest-point traversal from S given seed objects (another reading of
 * Algorithm 2 step 3, e.g. the two ends of the diameter of step 1):
 *   idx[m] = seeds[m] for m < S (as given, repeats allowed);
 *   idx[m] = the object not among idx[0..m-1] whose smallest squared distance
 *            to idx[0..m-1] is largest, lowest index on ties, for S <= m < K.
 * Requires 1 <= S <= K <= n and seeds in [0, n). With S = 1 and seed 0 it is
 * oracle_init_farthest.
 */
int oracle_init_farthest_from(const float *X, int64_t n, int32_t M, int32_t K,
                              const int32_t *seeds, int32_t S, int32_t *idx)
{
    if (!X || !idx || !seeds || n < 1 || M < 1 || K < 1 || (int64_t)K > n || S < 1 || S > K)
        return ORACLE_EINVAL;
    for (int32_t s = 0; s < S; ++s)
        if (seeds[s] < 0 || (int64_t)seeds[s] >= n)
            return ORACLE_EINVAL;
    double *closest = (double *)malloc((size_t)n * sizeof(double));
    unsigned char *taken = (unsigned char *)calloc((size_t)n, 1);
    if (!closest || !taken) {
        free(closest);
        free(taken);
        return ORACLE_ENOMEM;
    }
    for (int64_t obj = 0; obj < n; ++obj)
        closest[obj] = INFINITY;
    idx[0] = seeds[0];
    taken[seeds[0]] = 1;
    for (int32_t m = 1; m < K; ++m) {
        const float *newest = X + (int64_t)idx[m - 1] * M;
        for (int64_t obj = 0; obj < n; ++obj) {
            double dd = sqdist(X + obj * (int64_t)M, newest, M);
            if (dd < closest[obj])
                closest[obj] = dd;
        }
        if (m < S) {
            idx[m] = seeds[m];
        } else {
            int64_t pick = -1;
            for (int64_t obj = 0; obj < n; ++obj) {
                if (taken[obj])
                    continue;
                if (pick < 0 || closest[obj] > closest[pick])
                    pick = obj;
            }
            idx[m] = (int32_t)pick;
        }
        taken[idx[m]] = 1;
    }
    free(closest);
    free(taken);
    return 0;
}
