/*
 * A plain C consumer of the library's C ABI (include/kmeans.h), built with gcc
 * and linked against libkmeans_mi355x.so by tests/test_abi.py. It calls only
 * what runs on the host: the workspace sizing functions, kmeans_strerror, and
 * every entry point with arguments that validation refuses before any HIP
 * call. Prints one line per check and exits with the number of failures.
 */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "kmeans.h"

static int failures = 0;

static void check(int ok, const char *what)
{
    printf("%s %s\n", ok ? "ok  " : "FAIL", what);
    if (!ok) ++failures;
}

int main(void)
{
    float *fake = (float *)(uintptr_t)0x10000;        /* never dereferenced */
    int32_t *ifake = (int32_t *)(uintptr_t)0x10000;
    double *dfake = (double *)(uintptr_t)0x10000;
    int32_t iters = 0;

    check(kmeans_workspace_bytes(2000000, 25, 16, 0) > 0, "workspace for 2e6 x 25, K = 16");
    check(kmeans_workspace_bytes(10, 65, 4, 0) == 0, "workspace refuses M = 65");
    check(kmeans_workspace_bytes(10, 4, 4, KMEANS_METRIC_L1 | KMEANS_PATH_MFMA) == 0,
          "workspace refuses L1 with a path flag");
    check(kmeans_init_workspace_bytes(100, 4, 101) == 0, "init workspace refuses K > n");
    check(kmeans_init_workspace_bytes(100, 4, 100) >= 100 * sizeof(double), "init workspace");
    check(kmeans_centroid_workspace_bytes(1000, 3) > 0, "centroid workspace");
    check(kmeans_diameter_workspace_bytes(1000, 3) > 0, "diameter workspace");
    check(strcmp(kmeans_strerror(KMEANS_OK), "ok") == 0, "strerror(KMEANS_OK)");
    check(strcmp(kmeans_strerror(-99), "unknown status") == 0, "strerror(unknown)");

    check(kmeans_assign(NULL, 100, 4, fake, 3, ifake, NULL, 0, NULL) == KMEANS_EINVAL,
          "assign: NULL X");
    check(kmeans_assign(fake, 100, 4, fake, 3, ifake, NULL, 1u << 7, NULL) == KMEANS_EINVAL,
          "assign: unknown flag");
    check(kmeans_update(fake, 100, 4, ifake, 3, fake, fake, ifake, NULL, 0, NULL) ==
              KMEANS_EWORKSPACE, "update: no workspace");
    check(kmeans_run(fake, 100, 4, 3, fake, 0, 0, ifake, fake, ifake, &iters, fake,
                     1 << 20, NULL, NULL) == KMEANS_EINVAL, "run: max_iter = 0");
    check(kmeans_run(fake, 100, 4, 2000, fake, 5, 0, ifake, fake, ifake, &iters, fake,
                     1 << 20, NULL, NULL) == KMEANS_EUNSUPPORTED, "run: K = 2000");
    check(kmeans_init_farthest(fake, 5, 2, 6, ifake, fake, fake, 1 << 20, NULL) ==
              KMEANS_EINVAL, "init: K > n");
    check(kmeans_centroid(fake, 100, 65, fake, fake, 1 << 20, NULL) == KMEANS_EUNSUPPORTED,
          "centroid: M = 65");
    check(kmeans_diameter(fake, 100, 4, NULL, ifake, NULL, fake, 1 << 20, NULL) ==
              KMEANS_EINVAL, "diameter: NULL d2");
    check(kmeans_diameter(fake, 100, 4, dfake, ifake, NULL, fake, 16, NULL) ==
              KMEANS_EWORKSPACE, "diameter: small workspace");
    return failures;
}
