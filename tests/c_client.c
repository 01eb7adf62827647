/*
 * c_client.c -- a plain C program that uses the library through include/tree_ens.h only (no
 * Python, no torch): the hand-worked three-tree ensemble of tests/golden/hand_ensemble.txt,
 * whose scores under the paper's tie rule (right iff x >= theta, Section 3) are exact sums
 * worked out by hand.
 *
 *   c_client errors   model and argument errors, reported before any device call (no GPU needed)
 *   c_client gpu      device buffers from the HIP runtime, predict / predict_leaves / info on a
 *                     stream of its own, results compared exactly with the hand-worked values
 *
 * Exit status 0 when every check passes; the first failed check is printed.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "tree_ens.h"

#define CHECK(cond, ...)                                                                     \
    do {                                                                                     \
        if (!(cond)) {                                                                       \
            fprintf(stderr, "c_client: check failed at line %d: ", __LINE__);               \
            fprintf(stderr, __VA_ARGS__);                                                    \
            fprintf(stderr, " (last error: %s)\n", tree_ens_last_error());                   \
            return 1;                                                                        \
        }                                                                                    \
    } while (0)

/* the hand-worked ensemble (tree-local node ids, not breadth-first) */
static const int64_t kOffsets[4] = {0, 3, 10, 11};
static const int32_t kFeature[11] = {0, -1, -1, 1, 0, -1, 2, -1, -1, -1, -1};
static const float kThreshold[11] = {0.5f, 0, 0, 0.0f, 0.75f, 0, 1.0f, 0, 0, 0, 0};
static const int32_t kLeft[11] = {2, -1, -1, 5, 4, -1, 6, -1, -1, -1, -1};
static const int32_t kRight[11] = {1, -1, -1, 3, 2, -1, 1, -1, -1, -1, -1};
static const float kValue[11] = {0, 2.0f, 1.0f, 0, 0, 8.0f, 0, 4.0f, -0.5f, 0.25f, 0.125f};
#define N_DOCS 7
#define N_FEAT 3
/* tree 1 above: root 0 (feature 1 at 0.0) -> left 5 (-0.5), right 3; node 3 (feature 2 at 1.0)
 * -> left 6 (0.25), right 1; node 1 (feature 0 at 0.75) -> left 4 (4.0), right 2 (8.0). Its
 * flat arrays are listed by node id 0..6. */

static int errors_mode(void) {
    tree_ens_t *h = (tree_ens_t *)0x1;
    int rc = tree_ens_create(NULL, 3, kOffsets, kFeature, kThreshold, kLeft, kRight, kValue, 0);
    CHECK(rc == TREE_ENS_E_ARG, "NULL out gives %d", rc);
    int32_t left[11];
    memcpy(left, kLeft, sizeof left);
    left[3] = 0; /* tree 1's root names itself as its left child */
    rc = tree_ens_create(&h, 3, kOffsets, kFeature, kThreshold, left, kRight, kValue, 0);
    CHECK(rc == TREE_ENS_E_MODEL && h == NULL, "a child naming the root gives %d", rc);
    CHECK(strstr(tree_ens_last_error(), "root") != NULL, "message names the root");
    rc = tree_ens_create(&h, 3, kOffsets, kFeature, kThreshold, kLeft, kRight, kValue, 8u);
    CHECK(rc == TREE_ENS_E_ARG, "unknown flag bits give %d", rc);
    rc = tree_ens_create_multi(&h, 3, kOffsets, kFeature, kThreshold, kLeft, kRight, kValue, 1, 0, 0);
    CHECK(rc == TREE_ENS_E_ARG, "zero bags give %d", rc);
    rc = tree_ens_predict(NULL, NULL, NULL, 1, N_FEAT, NULL);
    CHECK(rc == TREE_ENS_E_ARG, "NULL handle gives %d", rc);
    tree_ens_destroy(NULL);
    printf("c_client errors: ok\n");
    return 0;
}

static int gpu_mode(void) {
    /* documents d0..d6 of the golden file and their hand-worked scores and leaf ids */
    const float X[N_DOCS][N_FEAT] = {
        {0.5f, 0.0f, 1.0f},          {0.25f, -0.0f, 0.5f},          {NAN, NAN, NAN},
        {INFINITY, -1e-30f, INFINITY}, {0.75f, 1e-45f, 2.0f},       {-INFINITY, -INFINITY, -INFINITY},
        {0x1.fffffep-2f, 0.0f, 0x1.fffffep-1f}};
    const float expect[N_DOCS] = {6.125f, 1.375f, 0.625f, 1.625f, 10.125f, 0.625f, 1.375f};
    const int32_t expect_leaf[N_DOCS][3] = {{1, 4, 0}, {2, 6, 0}, {2, 5, 0}, {1, 5, 0},
                                            {1, 2, 0}, {2, 5, 0}, {2, 6, 0}};
    hipStream_t stream = NULL;
    float *dX = NULL, *dS = NULL;
    int32_t *dL = NULL;
    CHECK(hipStreamCreate(&stream) == hipSuccess, "hipStreamCreate");
    CHECK(hipMalloc((void **)&dX, sizeof X) == hipSuccess, "hipMalloc X");
    CHECK(hipMalloc((void **)&dS, N_DOCS * sizeof(float)) == hipSuccess, "hipMalloc scores");
    CHECK(hipMalloc((void **)&dL, N_DOCS * 3 * sizeof(int32_t)) == hipSuccess, "hipMalloc leaves");
    CHECK(hipMemcpy(dX, X, sizeof X, hipMemcpyHostToDevice) == hipSuccess, "copy X");

    tree_ens_t *h = NULL;
    int rc = tree_ens_create(&h, 3, kOffsets, kFeature, kThreshold, kLeft, kRight, kValue,
                             TREE_ENS_RIGHT_IF_GE);
    CHECK(rc == TREE_ENS_OK && h != NULL, "create gives %d", rc);
    int32_t n_trees = 0, min_features = 0, max_depth = 0, n_tiles = 0, dpb = 0;
    int64_t packed = 0;
    rc = tree_ens_info(h, &n_trees, &min_features, &max_depth, &packed, &n_tiles, &dpb);
    CHECK(rc == TREE_ENS_OK && n_trees == 3 && min_features == 3 && max_depth == 3 && packed == 88,
          "info: %d trees, %d features, depth %d, %lld bytes", n_trees, min_features, max_depth,
          (long long)packed);
    rc = tree_ens_predict(h, stream, dX, N_DOCS, N_FEAT, dS);
    CHECK(rc == TREE_ENS_OK, "predict gives %d", rc);
    rc = tree_ens_predict_leaves(h, stream, dX, N_DOCS, N_FEAT, dL);
    CHECK(rc == TREE_ENS_OK, "predict_leaves gives %d", rc);
    rc = tree_ens_predict(h, stream, dX, 0, N_FEAT, NULL);
    CHECK(rc == TREE_ENS_OK, "zero documents give %d", rc);
    rc = tree_ens_predict(h, stream, dX, N_DOCS, 2, dS);
    CHECK(rc == TREE_ENS_E_SHAPE, "two features give %d", rc);
    CHECK(hipStreamSynchronize(stream) == hipSuccess, "stream synchronize");

    float scores[N_DOCS];
    int32_t leaves[N_DOCS][3];
    CHECK(hipMemcpy(scores, dS, sizeof scores, hipMemcpyDeviceToHost) == hipSuccess, "copy scores");
    CHECK(hipMemcpy(leaves, dL, sizeof leaves, hipMemcpyDeviceToHost) == hipSuccess, "copy leaves");
    for (int d = 0; d < N_DOCS; d++) {
        CHECK(scores[d] == expect[d], "doc %d: score %.9g, expected %.9g", d, scores[d], expect[d]);
        for (int t = 0; t < 3; t++)
            CHECK(leaves[d][t] == expect_leaf[d][t], "doc %d tree %d: leaf %d, expected %d", d, t,
                  leaves[d][t], expect_leaf[d][t]);
    }
    tree_ens_destroy(h);
    (void)hipFree(dX);
    (void)hipFree(dS);
    (void)hipFree(dL);
    (void)hipStreamDestroy(stream);
    printf("c_client gpu: ok (%d documents, scores and leaf ids exact)\n", N_DOCS);
    return 0;
}

int main(int argc, char **argv) {
    if (argc == 2 && strcmp(argv[1], "errors") == 0)
        return errors_mode();
    if (argc == 2 && strcmp(argv[1], "gpu") == 0)
        return gpu_mode();
    fprintf(stderr, "usage: c_client errors|gpu\n");
    return 2;
}
