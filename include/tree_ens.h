/*
 * tree_ens.h -- C ABI of the MI355X (gfx950) tree-ensemble scorer.
 *
 * The operation (paper, Section 3 and Section 5.3): a model is an ensemble of binary
 * regression trees. Each internal node holds a feature id f and a threshold theta; a document's
 * walk goes left when x[f] < theta and right otherwise (the Pred form writes the test as
 * x[f] >= theta), until it reaches a leaf, which holds a regression value. A document is a
 * dense float vector indexed by feature id (Section 3). The ensemble score of a document is the
 * sum of the reached leaves' values over all trees (Section 5.3: an outer loop over the trees).
 *
 * No HIP or framework header is needed to include this file. Device pointers are plain
 * pointers into memory of the device that was current when the model was created (for example
 * a torch tensor's data_ptr()). Streams are passed as void* and are hipStream_t values
 * (0 = the null stream).
 *
 * Every function returns TREE_ENS_OK (0) or a negative status; on failure
 * tree_ens_last_error() returns a message for the calling thread. No function throws.
 */
#ifndef TREE_ENS_H
#define TREE_ENS_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct tree_ens tree_ens_t;

/* status codes */
#define TREE_ENS_OK 0
#define TREE_ENS_E_ARG (-1)    /* a null pointer where one is required, a negative count, a
                                  misaligned pointer, or unknown flag bits */
#define TREE_ENS_E_MODEL (-2)  /* the flat arrays do not describe an ensemble of trees (see
                                  tree_ens_create), or a tree has more than 65,535 nodes */
#define TREE_ENS_E_SHAPE (-3)  /* the documents carry fewer features than the model reads */
#define TREE_ENS_E_DEVICE (-4) /* a HIP call failed (no device, launch or copy error) */
#define TREE_ENS_E_NOMEM (-5)  /* host or device allocation failed */

/* create-time flags */
#define TREE_ENS_RIGHT_IF_GE 0u /* right iff x[f] >= theta: the paper's rule (default) */
#define TREE_ENS_RIGHT_IF_GT 1u /* right iff x[f] >  theta: the other tie convention */
/* Also compile, at create time, a scoring kernel specialised for the model (the CodeGen form of
 * Section 3: the trees as nested if/else blocks with constant feature ids, thresholds and leaf
 * values; one document per thread, features read in place) with hiprtc; tree_ens_predict then
 * runs it. Other entry points keep the generic kernels. Models of at most 65,536 nodes and
 * depth 64, one value per leaf (else TREE_ENS_E_MODEL / TREE_ENS_E_ARG); a compiler failure is
 * TREE_ENS_E_DEVICE with the compiler log in the message. Compiling takes about 6 s per
 * 15,000 nodes (this call returns when it is done). This is the paper's comparison form, kept
 * for that comparison: on MI355X it only ties the generic kernel on tiny models (10 trees of 8
 * leaves, where both are bound by the launch) and is 15x slower at 200 trees of 32 leaves and
 * 55x slower at 1,000 trees of depth 3 (one document per thread follows the union of its
 * wave's branch paths and reads features from global memory); do not use it for throughput. */
#define TREE_ENS_CODEGEN 2u

/*
 * tree_ens_create -- validate an ensemble given as flat host arrays, pack it for the GPU and
 * upload it to the current device (the model representation of Section 3: per node a feature
 * id and a threshold, explicit left/right links as in the Struct and Struct+ forms, and leaf
 * values).
 *
 *   out           receives the handle; set to NULL on failure.
 *   n_trees       number of trees, >= 0 (0 gives all-zero scores).
 *   tree_offsets  [n_trees+1] int64: tree t owns flat nodes [tree_offsets[t], tree_offsets[t+1]);
 *                 tree_offsets[0] == 0, every tree has at least one node.
 *   feature       [n_nodes] int32: feature id (>= 0) of an internal node, -1 for a leaf.
 *   threshold     [n_nodes] float: threshold of an internal node (NaN rejected); ignored for
 *                 leaves.
 *   left, right   [n_nodes] int32: tree-local child ids of an internal node; ignored for leaves.
 *                 Node 0 of every tree is its root.
 *   value         [n_nodes] float: leaf values; ignored for internal nodes.
 *   flags         TREE_ENS_RIGHT_IF_GE or TREE_ENS_RIGHT_IF_GT, optionally | TREE_ENS_CODEGEN.
 *
 * All arrays are host memory, read during the call only; the caller keeps ownership. Node ids
 * need not be in any particular order. TREE_ENS_E_MODEL is returned when a child id is out of
 * range or names the root, a node has two parents, a node is unreachable from the root, a
 * threshold is NaN, a feature id is below -1, a tree has more than 65,535 nodes (32,768
 * leaves), or a feature id exceeds the LDS document-tile limit. Trees too large for one LDS
 * tile (a few thousand leaves, depending on the feature count) are accepted: they are walked
 * from device memory (their records stay in L2) instead of being staged in LDS, more slowly. Validation
 * happens before any HIP call, so model errors are reported on a host without a GPU. The
 * handle owns the device copy and is immutable; it may be used from several streams at once.
 */
int tree_ens_create(tree_ens_t **out, int32_t n_trees, const int64_t *tree_offsets,
                    const int32_t *feature, const float *threshold, const int32_t *left,
                    const int32_t *right, const float *value, uint32_t flags);

/*
 * tree_ens_create_multi -- tree_ens_create for vector-valued leaves and bagged ensembles
 * (Section 3: the predictor at a leaf may be a class, a real or another model; Section 5.3:
 * several boosted ensembles, each trained on a bootstrap sample, whose scores are averaged).
 *
 *   value      [n_nodes][n_outputs] float, row-major: the n_outputs values of each leaf (rows
 *              of internal nodes are ignored). One output per class with one tree per class
 *              and round is the multi-class boosting layout (zeros in the other columns).
 *   n_outputs  1 .. 256. tree_ens_predict then writes n_outputs scores per document.
 *   n_bags     >= 1: the trees are the concatenation of n_bags ensembles and every score is
 *              the mean of their sums, i.e. the sum over all trees divided by n_bags.
 * Other arguments, ownership and errors as tree_ens_create (tree_ens_create is this call with
 * n_outputs = n_bags = 1). With n_outputs > 1 the leaf rows live in a device table of
 * n_nodes + 1 rows of ceil(n_outputs / 4) * 4 floats, and a predict makes one pass over the
 * trees per four outputs.
 */
int tree_ens_create_multi(tree_ens_t **out, int32_t n_trees, const int64_t *tree_offsets,
                          const int32_t *feature, const float *threshold, const int32_t *left,
                          const int32_t *right, const float *value, int32_t n_outputs,
                          int32_t n_bags, uint32_t flags);

/*
 * tree_ens_predict -- score n_docs documents (the ensemble sum of Section 5.3).
 *
 *   h           a handle from tree_ens_create.
 *   stream      hipStream_t the work is enqueued on (0 = null stream). The call returns without
 *               waiting; scores are valid once the stream reaches this point, and X must stay
 *               unchanged until then.
 *   X           device, row-major float [n_docs][n_features], 4-byte aligned (rows contiguous,
 *               row stride n_features).
 *   n_docs      >= 0; 0 returns TREE_ENS_OK without a launch.
 *   n_features  row length; must be >= 1 + the largest feature id of the model (else
 *               TREE_ENS_E_SHAPE). Columns beyond the ones the model reads are never read.
 *   scores      device, float [n_docs][n_outputs] (n_outputs = 1 unless the handle comes from
 *               tree_ens_create_multi): per output, the sum of the reached leaves' values,
 *               accumulated in double precision, divided by n_bags and rounded once to float.
 *
 * Kernel faults surface at the caller's next synchronisation with the stream. When the launch
 * splits document blocks over several workgroups (small batches, and the blocks of a last,
 * partial round of workgroups) their fp64 partial sums go to a 1 MiB scratch buffer owned by
 * the handle (calls on different streams are ordered by an event while they share it), or, if
 * larger, to a stream-ordered allocation (hipMallocAsync / hipFreeAsync on `stream`). Models
 * with threshold-coded features also take a stream-ordered buffer of n_docs x min_features
 * 16-bit codes for the duration of the call. A call made while `stream` is being captured into
 * a HIP graph takes neither: it gets a device buffer of its own for its partial sums and codes,
 * allocated when it is captured and kept by the handle until tree_ens_destroy, so the graph's
 * replays never share scratch with other calls of the handle, eager or captured.
 */
int tree_ens_predict(const tree_ens_t *h, void *stream, const float *X, int64_t n_docs,
                     int32_t n_features, float *scores);

/*
 * tree_ens_predict_noalloc -- tree_ens_predict for callers that cannot allocate device memory
 * during the call (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc). Arguments, results and errors as tree_ens_predict; the same kernels run.
 *
 * The call allocates nothing: no hipMalloc, hipMallocAsync or hipFree, no allocating library
 * routine. Its scratch (the fp64 partial sums of document blocks split over several workgroups,
 * and the 16-bit threshold codes of coded models) lives in one static device array of 16 MiB
 * that the library holds on each device it runs on until the process ends. A batch whose split
 * partial sums would not fit is launched without splits (every workgroup walks all trees of its
 * block; the scores are the same within the documented tolerance); a batch whose threshold
 * codes (n_docs x min_features x 2 bytes) exceed 16 MiB is refused with TREE_ENS_E_ARG.
 * Every call on a device shares that device's array and leaves its contents behind: calls of
 * this function that overlap in time on one device (different streams, or graph replays next to
 * eager calls) race on it and must be ordered by the caller.
 */
int tree_ens_predict_noalloc(const tree_ens_t *h, void *stream, const float *X, int64_t n_docs,
                             int32_t n_features, float *scores);

/*
 * tree_ens_predict_leaves -- the leaf each (document, tree) pair reaches, by the same walk.
 *
 *   leaf_ids  device, int32 [n_docs][n_trees] row-major: the tree-local id, in the caller's
 *             input numbering, of the leaf that document d reaches in tree t.
 * Other arguments and behaviour as tree_ens_predict.
 */
int tree_ens_predict_leaves(const tree_ens_t *h, void *stream, const float *X, int64_t n_docs,
                            int32_t n_features, int32_t *leaf_ids);

/*
 * tree_ens_feature_usage -- feature-access trace (Section 6 and its Table 4: how many of the
 * features a prediction actually reads). For each document, the set of distinct feature ids
 * compared at the internal nodes its walks pass through, over all trees, by the same walk as
 * tree_ens_predict (same tie rule, same flags).
 *
 *   counts    device, int32 [n_docs]: the size of document d's set.
 *   masks     device, uint32 [n_docs][(n_features + 31) / 32] row-major, or NULL: bit (f % 32)
 *             of word f / 32 is set when feature f is in the set; bits of features the model
 *             never reads are 0.
 * Other arguments, errors and behaviour as tree_ens_predict. One workgroup walks every tree for
 * its block of documents, holding the block's bitmasks in LDS.
 */
int tree_ens_feature_usage(const tree_ens_t *h, void *stream, const float *X, int64_t n_docs,
                           int32_t n_features, int32_t *counts, uint32_t *masks);

/*
 * tree_ens_topk -- per-query top-k reranking of scores (Section 6: a query's candidate
 * documents, e.g. 200 of them, are scored and reranked into the final list of the best 20).
 *
 *   stream        hipStream_t the work is enqueued on (0 = null stream); returns without waiting.
 *   scores        device, float [n_docs].
 *   n_docs        >= 0 and <= INT32_MAX (indices are int32).
 *   group_offsets device, int64 [n_groups+1]: query g owns documents [off[g], off[g+1]).
 *                 Offsets are clamped into [0, n_docs] and a group ending before it starts is
 *                 empty, so ill-formed offsets never read outside `scores`.
 *   n_groups      >= 0; 0 returns TREE_ENS_OK without a launch.
 *   k             1 <= k <= 1024.
 *   top_idx       device, int32 [n_groups][k] row-major: the k first documents of each group
 *                 (absolute document indices). Order: higher score first; equal scores
 *                 (-0.0 equals +0.0) by increasing document index; NaN scores after every
 *                 number. Positions past a group's size hold -1.
 *   top_scores    device, float [n_groups][k], or NULL: the scores of top_idx (NaN past a
 *                 group's size).
 * Returns TREE_ENS_E_ARG for a count or k out of range or a NULL required pointer.
 */
int tree_ens_topk(void *stream, const float *scores, int64_t n_docs, const int64_t *group_offsets,
                  int64_t n_groups, int32_t k, int32_t *top_idx, float *top_scores);

/*
 * tree_ens_predict_topk -- tree_ens_predict into `scores` followed by tree_ens_topk over it
 * (handles with one output only; TREE_ENS_E_ARG otherwise),
 * both enqueued on `stream` (scoring and reranking of query candidates in one call). Arguments
 * as for those two functions; `scores` is a device buffer of n_docs floats the caller owns
 * (it receives the scores).
 */
int tree_ens_predict_topk(const tree_ens_t *h, void *stream, const float *X, int64_t n_docs,
                          int32_t n_features, const int64_t *group_offsets, int64_t n_groups,
                          int32_t k, float *scores, int32_t *top_idx, float *top_scores);

/*
 * tree_ens_info -- facts about a packed model; every output pointer may be NULL.
 *   n_trees        number of trees.
 *   min_features   1 + the largest feature id any node reads (0 if there is none).
 *   max_depth      edges on the longest root-to-leaf path over all trees.
 *   packed_bytes   bytes of node records (8 per node); the device also holds the tile images
 *                  built from them (one set per tiling granularity) and, for models whose
 *                  groups of trees fit, the per-wave packets (one more copy of the records;
 *                  for threshold-coded models of trees up to 511 nodes, compact packets of
 *                  4-byte records with two 4-byte arrays of leaf values and node ids of the
 *                  same shape).
 *   n_tiles        LDS tiles the tiled trees are streamed in for a large batch (trees too
 *                  large for one tile are walked from device memory and not counted).
 *   docs_per_block documents a workgroup stages in LDS (a power of two from 8 to 64).
 */
int tree_ens_info(const tree_ens_t *h, int32_t *n_trees, int32_t *min_features,
                  int32_t *max_depth, int64_t *packed_bytes, int32_t *n_tiles,
                  int32_t *docs_per_block);

/*
 * tree_ens_codegen_source -- the HIP source that TREE_ENS_CODEGEN compiles for a model (for
 * inspection or offline compilation; its entry point is `tree_ens_cg(const float *X,
 * long long n_docs, int n_features, float *scores, double scale)`, one document per thread in
 * blocks of 256). Model arguments and validation as tree_ens_create; host only.
 *   buf, buf_size  receives the source, truncated to buf_size - 1 characters and NUL-terminated
 *                  (buf may be NULL when buf_size is 0).
 *   src_len        receives the full length without the NUL (may be NULL).
 */
int tree_ens_codegen_source(int32_t n_trees, const int64_t *tree_offsets, const int32_t *feature,
                            const float *threshold, const int32_t *left, const int32_t *right,
                            const float *value, uint32_t flags, char *buf, int64_t buf_size,
                            int64_t *src_len);

/* tree_ens_outputs -- the handle's outputs per document and bag count (either pointer may be
 * NULL). */
int tree_ens_outputs(const tree_ens_t *h, int32_t *n_outputs, int32_t *n_bags);

/*
 * tree_ens_kernel_timing -- measurement aid: time the scoring kernel of later predict calls with
 * HIP events (the paper reports its timings as means over repeated trials, Section 4). enable !=
 * 0 starts a new record: every later eager predict call of h (every mode; calls captured into a
 * HIP graph are not timed) records an event on its stream right before and right after each
 * launch of the scoring kernel, for the first 1,024 such launches; enable == 0 stops recording.
 * The events are created on the handle's device by the first enabling call (no device memory is
 * allocated) and live until destroy. Returns TREE_ENS_E_ARG for a NULL handle,
 * TREE_ENS_E_DEVICE if an event cannot be created.
 *
 * tree_ens_kernel_time -- waits for the recorded events (a host wait on them, so the predicts
 * must have been enqueued) and gives the sum of the timed launches' durations in milliseconds
 * and their number (either pointer may be NULL). Neither call may run concurrently with a
 * predict of h on another thread.
 */
int tree_ens_kernel_timing(const tree_ens_t *h, int32_t enable);
int tree_ens_kernel_time(const tree_ens_t *h, double *total_ms, int32_t *launches);

/* tree_ens_destroy -- free the handle and its device memory. NULL is accepted. The caller must
 * ensure no enqueued predict that uses h is still pending. */
void tree_ens_destroy(tree_ens_t *h);

/* tree_ens_last_error -- message for the last failure on the calling thread ("" if none). The
 * pointer stays valid until the next call into the library on this thread. */
const char *tree_ens_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* TREE_ENS_H */
