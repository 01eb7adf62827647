/*
 * oracle.c -- plain, slow, obviously correct CPU scorer for regression-tree ensembles.
 *
 * TEST INFRASTRUCTURE ONLY. Only the tests, the smoke check and the bench's CPU-baseline leg
 * load this library. It shares no code, header, table or helper with the GPU library; it
 * reads the caller's flat creation-order arrays directly and never a packed layout.
 *
 * What it computes (Section 3 of the paper, first paragraphs): a tree is walked from its
 * root; at an internal node holding feature id f and threshold theta the walk goes left when
 * x[f] < theta and right otherwise, until it reaches a leaf. The feature vector is a dense
 * float array indexed by feature id (Section 3, dense-vector assumption). An ensemble's score
 * is the sum over its trees of the reached leaves' values (Section 5.3: an outer loop over the
 * trees). Scores are summed in double precision in tree order.
 *
 * rule 0 (paper): right iff x[f] >= theta.   rule 1: right iff x[f] > theta.
 * Under IEEE comparison a NaN feature value is never >= (nor >) a threshold, so it goes left.
 *
 * Three independent walks reach the leaf:
 *   walk 0 -- branching walk over explicit left/right links (the Struct form, Section 3);
 *   walk 1 -- predicated walk: the comparison result, 0 or 1, indexes the pair
 *             {left, right} (the branch-free step of the Pred form, Section 3, with explicit
 *             children);
 *   oracle_score_padded -- the literal Pred form: the tree is padded with dummy nodes to a
 *             complete tree of its depth d, laid out breadth-first (children of i at 2i+1 and
 *             2i+2), and walked with exactly d steps i = 2i + 1 + bit. A dummy node's two
 *             subtrees both end at the original leaf it replaces, so padding does not change
 *             the prediction (Section 3, end of Pred; Section 6 on unbalanced trees).
 *
 * oracle_score_multi sums vector-valued leaves component by component and averages bagged
 * ensembles. oracle_feature_usage traces the branching walk and records the distinct feature ids each
 * document's walks compare over the whole ensemble (the fraction of features a prediction
 * reads, Section 6 and its Table 4).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

#define ORACLE_OK 0
#define ORACLE_E_MODEL 1 /* a child id out of range or a walk longer than the tree */
#define ORACLE_E_ARG 2
#define ORACLE_E_NOMEM 3

static int goes_right(float x, float theta, int rule)
{
    if (rule == 0)
        return x >= theta;
    return x > theta;
}

/* Branching (walk 0) or predicated (walk 1) walk of one tree for one document. Returns the
 * tree-local leaf id, or -1 when the tree is malformed. *steps receives the number of internal
 * nodes visited (the comparisons made). */
static int32_t walk_tree(int64_t n_nodes, const int32_t *feature, const float *threshold,
                         const int32_t *left, const int32_t *right, const float *x,
                         int32_t n_features, int rule, int walk, int64_t *steps)
{
    int64_t n = 0;
    int64_t k = 0;
    while (feature[n] >= 0) {
        int32_t f = feature[n];
        if (f >= n_features || k >= n_nodes)
            return -1;
        int32_t next;
        if (walk == 0) {
            if (goes_right(x[f], threshold[n], rule))
                next = right[n];
            else
                next = left[n];
        } else {
            int32_t kids[2];
            kids[0] = left[n];
            kids[1] = right[n];
            next = kids[goes_right(x[f], threshold[n], rule)];
        }
        if (next < 0 || next >= n_nodes)
            return -1;
        n = next;
        k++;
    }
    *steps = k;
    return (int32_t)n;
}

/*
 * Score n_docs documents (row-major X[n_docs][n_features]) with the ensemble.
 *   scores   [n_docs] doubles, or NULL
 *   leaf_ids [n_docs][n_trees] tree-local leaf ids, or NULL
 *   visits   total number of internal nodes visited over all (document, tree) pairs, or NULL
 * Returns ORACLE_OK or an error code.
 */
int oracle_score(int32_t n_trees, const int64_t *tree_offsets, const int32_t *feature,
                 const float *threshold, const int32_t *left, const int32_t *right,
                 const float *value, const float *X, int64_t n_docs, int32_t n_features,
                 int32_t rule, int32_t walk, int32_t n_threads, double *scores,
                 int32_t *leaf_ids, int64_t *visits)
{
    if (n_trees < 0 || n_docs < 0 || n_features < 0 || (n_trees > 0 && !tree_offsets))
        return ORACLE_E_ARG;
    int err = ORACLE_OK;
    int64_t total_steps = 0;
#ifdef _OPENMP
    if (n_threads > 0)
        omp_set_num_threads(n_threads);
#endif
#pragma omp parallel for schedule(dynamic, 16) reduction(+ : total_steps)
    for (int64_t d = 0; d < n_docs; d++) {
        const float *x = X + d * (int64_t)n_features;
        double s = 0.0;
        for (int32_t t = 0; t < n_trees; t++) {
            int64_t a = tree_offsets[t];
            int64_t nn = tree_offsets[t + 1] - a;
            int64_t steps = 0;
            int32_t leaf = -1;
            if (nn > 0)
                leaf = walk_tree(nn, feature + a, threshold + a, left + a, right + a, x, n_features,
                                 rule, walk, &steps);
            if (leaf < 0) {
#pragma omp atomic write
                err = ORACLE_E_MODEL;
                continue;
            }
            s += (double)value[a + leaf];
            total_steps += steps;
            if (leaf_ids)
                leaf_ids[d * (int64_t)n_trees + t] = leaf;
        }
        if (scores)
            scores[d] = s;
    }
    if (visits)
        *visits = total_steps;
    return err;
}

/*
 * Vector-valued leaves and bagged ensembles (Section 3: the leaf predictor may be a class, a
 * real or another model; Section 5.3: an ensemble made of several bagged boosted ensembles).
 * Every leaf holds n_outputs values (value[node * n_outputs + c]); output c of a document is
 * the sum over the trees, in tree order and in double precision, of component c of the leaves
 * reached, divided by n_bags: the trees are the concatenation of n_bags ensembles whose scores
 * are averaged, and the mean of the bags' sums is the sum over all trees over n_bags.
 *   scores [n_docs][n_outputs] doubles
 * Returns ORACLE_OK or an error code.
 */
int oracle_score_multi(int32_t n_trees, const int64_t *tree_offsets, const int32_t *feature,
                       const float *threshold, const int32_t *left, const int32_t *right,
                       const float *value, int32_t n_outputs, int32_t n_bags, const float *X,
                       int64_t n_docs, int32_t n_features, int32_t rule, int32_t n_threads,
                       double *scores)
{
    if (n_trees < 0 || n_docs < 0 || n_features < 0 || n_outputs < 1 || n_bags < 1 ||
        (n_trees > 0 && !tree_offsets) || !scores)
        return ORACLE_E_ARG;
    int err = ORACLE_OK;
#ifdef _OPENMP
    if (n_threads > 0)
        omp_set_num_threads(n_threads);
#endif
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t d = 0; d < n_docs; d++) {
        const float *x = X + d * (int64_t)n_features;
        double *out = scores + d * (int64_t)n_outputs;
        for (int32_t c = 0; c < n_outputs; c++)
            out[c] = 0.0;
        for (int32_t t = 0; t < n_trees; t++) {
            const int64_t a = tree_offsets[t];
            const int64_t nn = tree_offsets[t + 1] - a;
            int64_t steps = 0;
            int32_t leaf = -1;
            if (nn > 0)
                leaf = walk_tree(nn, feature + a, threshold + a, left + a, right + a, x, n_features,
                                 rule, 0, &steps);
            if (leaf < 0) {
#pragma omp atomic write
                err = ORACLE_E_MODEL;
                continue;
            }
            const float *v = value + (a + leaf) * (int64_t)n_outputs;
            for (int32_t c = 0; c < n_outputs; c++)
                out[c] += (double)v[c];
        }
        for (int32_t c = 0; c < n_outputs; c++)
            out[c] /= (double)n_bags;
    }
    return err;
}

/*
 * Features examined (Section 6 and its Table 4: the fraction of features a prediction reads).
 * For each document, the set of distinct feature ids compared at the internal nodes its walks
 * pass through, over all trees (branching walk, the same rule as oracle_score).
 *   counts [n_docs] int32: the size of the set, or NULL
 *   masks  [n_docs][(n_features + 31) / 32] uint32: bit (f % 32) of word f / 32 is set when
 *          feature f is examined, or NULL
 * Returns ORACLE_OK or an error code.
 */
int oracle_feature_usage(int32_t n_trees, const int64_t *tree_offsets, const int32_t *feature,
                         const float *threshold, const int32_t *left, const int32_t *right,
                         const float *X, int64_t n_docs, int32_t n_features, int32_t rule,
                         int32_t n_threads, int32_t *counts, uint32_t *masks)
{
    if (n_trees < 0 || n_docs < 0 || n_features < 1 || (n_trees > 0 && !tree_offsets))
        return ORACLE_E_ARG;
    const int64_t words = ((int64_t)n_features + 31) / 32;
    int err = ORACLE_OK;
#ifdef _OPENMP
    if (n_threads > 0)
        omp_set_num_threads(n_threads);
#endif
#pragma omp parallel
    {
        uint32_t *seen = (uint32_t *)calloc((size_t)words, sizeof(uint32_t));
        if (!seen) {
#pragma omp atomic write
            err = ORACLE_E_NOMEM;
        }
#pragma omp for schedule(dynamic, 16)
        for (int64_t d = 0; d < n_docs; d++) {
            if (!seen)
                continue;
            const float *x = X + d * (int64_t)n_features;
            memset(seen, 0, (size_t)words * sizeof(uint32_t));
            for (int32_t t = 0; t < n_trees; t++) {
                const int64_t a = tree_offsets[t];
                const int64_t nn = tree_offsets[t + 1] - a;
                int64_t n = 0, k = 0;
                while (nn > 0 && feature[a + n] >= 0) {
                    const int32_t f = feature[a + n];
                    if (f >= n_features || k >= nn) {
#pragma omp atomic write
                        err = ORACLE_E_MODEL;
                        break;
                    }
                    seen[f / 32] |= (uint32_t)1 << (f % 32);
                    n = goes_right(x[f], threshold[a + n], rule) ? right[a + n] : left[a + n];
                    if (n < 0 || n >= nn) {
#pragma omp atomic write
                        err = ORACLE_E_MODEL;
                        break;
                    }
                    k++;
                }
            }
            int32_t c = 0;
            for (int64_t w = 0; w < words; w++) {
                for (int b = 0; b < 32; b++)
                    c += (seen[w] >> b) & 1u;
                if (masks)
                    masks[d * words + w] = seen[w];
            }
            if (counts)
                counts[d] = c;
        }
        free(seen);
    }
    return err;
}

/* Depth (edges on the longest root-to-leaf path) of a tree, or -1 if malformed. */
static int32_t tree_depth(int64_t n_nodes, const int32_t *feature, const int32_t *left,
                          const int32_t *right)
{
    /* iterative DFS with an explicit stack of (node, depth) */
    int64_t *stack = (int64_t *)malloc(sizeof(int64_t) * 2 * (size_t)(n_nodes + 1));
    if (!stack)
        return -1;
    int64_t top = 0, visited = 0;
    int32_t best = 0;
    stack[0] = 0;
    stack[1] = 0;
    top = 1;
    while (top > 0) {
        top--;
        int64_t n = stack[2 * top], dep = stack[2 * top + 1];
        if (++visited > n_nodes || n < 0 || n >= n_nodes) {
            free(stack);
            return -1;
        }
        if (dep > best)
            best = (int32_t)dep;
        if (feature[n] >= 0) {
            stack[2 * top] = left[n];
            stack[2 * top + 1] = dep + 1;
            top++;
            stack[2 * top] = right[n];
            stack[2 * top + 1] = dep + 1;
            top++;
        }
    }
    free(stack);
    return best;
}

/* Fill the padded breadth-first arrays of a complete tree of depth `depth`: slot `slot` at
 * level `level` holds original node `node`. A leaf met above the last level becomes a dummy
 * node (feature 0, threshold 0) whose two subtrees both carry that leaf. */
static void pad_fill(int64_t slot, int32_t node, int32_t level, int32_t depth,
                     const int32_t *feature, const float *threshold, const int32_t *left,
                     const int32_t *right, int32_t *pfid, float *pthr, int32_t *pleaf)
{
    int64_t n_internal = ((int64_t)1 << depth) - 1;
    if (level == depth) {
        pleaf[slot - n_internal] = node;
        return;
    }
    if (feature[node] >= 0) {
        pfid[slot] = feature[node];
        pthr[slot] = threshold[node];
        pad_fill(2 * slot + 1, left[node], level + 1, depth, feature, threshold, left, right, pfid,
                 pthr, pleaf);
        pad_fill(2 * slot + 2, right[node], level + 1, depth, feature, threshold, left, right, pfid,
                 pthr, pleaf);
    } else {
        pfid[slot] = 0;
        pthr[slot] = 0.0f;
        pad_fill(2 * slot + 1, node, level + 1, depth, feature, threshold, left, right, pfid, pthr,
                 pleaf);
        pad_fill(2 * slot + 2, node, level + 1, depth, feature, threshold, left, right, pfid, pthr,
                 pleaf);
    }
}

/*
 * Same outputs as oracle_score, reached by the literal padded Pred walk. Trees deeper than
 * max_depth (at most 24) are rejected with ORACLE_E_ARG, since the padded array has 2^(d+1)-1
 * slots. Needs n_features >= 1 when any tree is padded (dummy nodes read feature 0).
 */
int oracle_score_padded(int32_t n_trees, const int64_t *tree_offsets, const int32_t *feature,
                        const float *threshold, const int32_t *left, const int32_t *right,
                        const float *value, const float *X, int64_t n_docs, int32_t n_features,
                        int32_t rule, int32_t max_depth, double *scores, int32_t *leaf_ids)
{
    if (n_trees < 0 || n_docs < 0 || max_depth > 24)
        return ORACLE_E_ARG;
    int32_t **pfid = (int32_t **)calloc((size_t)n_trees + 1, sizeof(int32_t *));
    float **pthr = (float **)calloc((size_t)n_trees + 1, sizeof(float *));
    int32_t **pleaf = (int32_t **)calloc((size_t)n_trees + 1, sizeof(int32_t *));
    int32_t *depth = (int32_t *)calloc((size_t)n_trees + 1, sizeof(int32_t));
    int err = ORACLE_OK;
    if (!pfid || !pthr || !pleaf || !depth)
        err = ORACLE_E_NOMEM;
    for (int32_t t = 0; t < n_trees && err == ORACLE_OK; t++) {
        int64_t a = tree_offsets[t];
        int64_t nn = tree_offsets[t + 1] - a;
        int32_t d = nn > 0 ? tree_depth(nn, feature + a, left + a, right + a) : -1;
        if (d < 0) {
            err = ORACLE_E_MODEL;
            break;
        }
        if (d > max_depth || (d > 0 && n_features < 1)) {
            err = ORACLE_E_ARG;
            break;
        }
        depth[t] = d;
        int64_t n_int = ((int64_t)1 << d) - 1;
        pfid[t] = (int32_t *)malloc(sizeof(int32_t) * (size_t)(n_int + 1));
        pthr[t] = (float *)malloc(sizeof(float) * (size_t)(n_int + 1));
        pleaf[t] = (int32_t *)malloc(sizeof(int32_t) * (size_t)(n_int + 1));
        if (!pfid[t] || !pthr[t] || !pleaf[t]) {
            err = ORACLE_E_NOMEM;
            break;
        }
        pad_fill(0, 0, 0, d, feature + a, threshold + a, left + a, right + a, pfid[t], pthr[t],
                 pleaf[t]);
    }
    if (err == ORACLE_OK) {
        for (int64_t doc = 0; doc < n_docs; doc++) {
            const float *x = X + doc * (int64_t)n_features;
            double s = 0.0;
            for (int32_t t = 0; t < n_trees; t++) {
                int64_t i = 0;
                for (int32_t k = 0; k < depth[t]; k++)
                    i = (i << 1) + 1 + goes_right(x[pfid[t][i]], pthr[t][i], rule);
                int32_t leaf = pleaf[t][i - (((int64_t)1 << depth[t]) - 1)];
                s += (double)value[tree_offsets[t] + leaf];
                if (leaf_ids)
                    leaf_ids[doc * (int64_t)n_trees + t] = leaf;
            }
            if (scores)
                scores[doc] = s;
        }
    }
    for (int32_t t = 0; t < n_trees; t++) {
        if (pfid)
            free(pfid[t]);
        if (pthr)
            free(pthr[t]);
        if (pleaf)
            free(pleaf[t]);
    }
    free(pfid);
    free(pthr);
    free(pleaf);
    free(depth);
    return err;
}

/* Number of OpenMP threads a parallel region would use (1 without OpenMP). */
int oracle_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
