/*
 * Multi-threaded CPU regime of the Lloyd iteration: Algorithm 3 of
 * Litvinenko, "Using of GPUs for cluster analysis of large data by K-means
 * method", steps 4-9 (with given initial centres).
 *
 * CPU BASELINE, TEST INFRASTRUCTURE ONLY: the benchmark times it beside the
 * GPU library as the paper's own multi-threaded regime, and the tests check
 * it against the single-threaded oracle. It shares no code with the GPU
 * library.
 *
 * As Algorithm 3 states it, each of N threads handles a contiguous 1/N of the
 * objects: it assigns them to the nearest centre (steps 4 and 6) and forms
 * their per-cluster coordinate sums and counts (steps 5 and 7); when all
 * threads have finished, the partial sums are added in thread order and
 * divided by the counts; the centres of the last two iterations are then
 * compared by one thread (step 8), and the loop repeats until they are
 * congruent (step 9).
 *
 * Arithmetic follows the oracle's readings: squared distances in fp64 formed
 * as e = (double)x_j - (double)c_j, d = d + e*e (features ascending, no fused
 * multiply-add), lowest index on ties, fp64 sums, centres = fp32(sum / count),
 * an empty cluster keeps its centre, congruent = bitwise equal, earliest stop
 * at t = 2. The labels are therefore the oracle's for the same centres; the
 * sums are added in another order (per thread, then across threads), so a
 * centre can differ from the oracle's in its last fp32 bit.
 *
 * Build: gcc -std=c99 -O3 -fopenmp -ffp-contract=off -fPIC -shared
 */
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <math.h>

#define ALG3_EINVAL (-1)
#define ALG3_ENOMEM (-2)

static int nearest_centre(const float *x, const float *C, int32_t M, int32_t K)
{
    double best = INFINITY;
    int lab = 0;
    for (int32_t k = 0; k < K; ++k) {
        const float *c = C + (int64_t)k * M;
        double d = 0.0;
        for (int32_t j = 0; j < M; ++j) {
            double e = (double)x[j] - (double)c[j];
            double sq = e * e;
            d = d + sq;
        }
        if (d < best) {
            best = d;
            lab = k;
        }
    }
    return lab;
}

/*
 * Steps 4-9 of Algorithm 3 with `threads` threads (0 = OpenMP's default).
 * Same outputs as the oracle's run: the last labels, the centres of gravity
 * of those labels, their counts, and the number of assignment passes.
 * Returns 0, or a negative code.
 */
int alg3_run(const float *X, int64_t n, int32_t M, int32_t K, const float *init,
             int32_t max_iter, int32_t fixed, int32_t threads, int32_t *labels,
             float *centers, int32_t *counts, int32_t *iterations, int32_t *threads_used)
{
    if (!X || !init || !labels || !centers || !counts || !iterations || n < 1 || M < 1 ||
        K < 1 || max_iter < 1)
        return ALG3_EINVAL;
    const int N = threads > 0 ? threads : omp_get_max_threads();
    const int64_t km = (int64_t)K * M;
    float *prev = (float *)malloc((size_t)km * sizeof(float));
    float *cur = (float *)malloc((size_t)km * sizeof(float));
    double *S = (double *)malloc((size_t)N * km * sizeof(double));       /* per thread */
    int64_t *cnt = (int64_t *)malloc((size_t)N * K * sizeof(int64_t));
    if (!prev || !cur || !S || !cnt) {
        free(prev);
        free(cur);
        free(S);
        free(cnt);
        return ALG3_ENOMEM;
    }
    memcpy(prev, init, (size_t)km * sizeof(float));
    int32_t t;
    for (t = 1; t <= max_iter; ++t) {
        /* assignment and per-thread sums, each thread on its 1/N of the objects */
#pragma omp parallel num_threads(N)
        {
            const int id = omp_get_thread_num();
            const int nt = omp_get_num_threads();
            const int64_t lo = n * id / nt, hi = n * (id + 1) / nt;
            double *s = S + (int64_t)id * km;
            int64_t *c = cnt + (int64_t)id * K;
            memset(s, 0, (size_t)km * sizeof(double));
            memset(c, 0, (size_t)K * sizeof(int64_t));
            for (int64_t i = lo; i < hi; ++i) {
                const float *x = X + i * (int64_t)M;
                const int l = nearest_centre(x, prev, M, K);
                labels[i] = l;
                double *sl = s + (int64_t)l * M;
                for (int32_t j = 0; j < M; ++j)
                    sl[j] = sl[j] + (double)x[j];
                c[l] += 1;
            }
        }
        /* when all threads have finished: totals in thread order, centres */
        for (int32_t k = 0; k < K; ++k) {
            int64_t total = 0;
            for (int th = 0; th < N; ++th)
                total += cnt[(int64_t)th * K + k];
            for (int32_t j = 0; j < M; ++j) {
                const int64_t o = (int64_t)k * M + j;
                double sum = 0.0;
                for (int th = 0; th < N; ++th)
                    sum = sum + S[(int64_t)th * km + o];
                cur[o] = total > 0 ? (float)(sum / (double)total) : prev[o];
            }
            counts[k] = (int32_t)total;
        }
        /* step 8, one thread: congruent centres end the loop (from t = 2) */
        const int stop = !fixed && t >= 2 && memcmp(cur, prev, (size_t)km * sizeof(float)) == 0;
        memcpy(prev, cur, (size_t)km * sizeof(float));
        if (stop)
            break;
    }
    if (t > max_iter)
        t = max_iter;
    memcpy(centers, prev, (size_t)km * sizeof(float));
    *iterations = t;
    if (threads_used)
        *threads_used = N;
    free(prev);
    free(cur);
    free(S);
    free(cnt);
    return 0;
}
